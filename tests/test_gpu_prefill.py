"""Parity of the prefix stage, vla_prefix_prefill (the backbone's bidirectional
prefill, Algorithm 1's VLM-Prefix), against the fp64 oracle, and of the whole
observation path prefill -> vla_prefix_kv_build -> vla_denoise.

Tolerances on the hidden states (unit RMS after the final norm) come from a
CPU study of the oracle with the kernels' bf16 storage points emulated (GEMM
inputs, Q, K, V, attention output; u and the MLP hidden stay fp32 in the
W2A8 backbone): 2 Gemma-width layers move the hidden by max 2.3e-2 / mean
3.6e-3, 18 layers by 7.6e-2 / 1.1e-2; one BitNet-width W2A8 layer by
0.10 / 1.3e-2 and 30 layers with W_o and W_d scales at 0.1x by 0.21 /
3.3e-2 (bf16 Q/K/V flip int8 codes of the O-projection input).  The tests
allow about three times those.  The hidden output itself is bf16 (2^-9
relative).  The end-to-end chunk is held to the 2e-2 bar.
"""
import numpy as np
import pytest

import workloads as wl
from oracle import vla_oracle as O

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch as t
    if not t.cuda.is_available():
        pytest.skip("no GPU")
    return t


def _prefill(bcfg, W, e):
    from vla_testlib import Prefill
    pre = Prefill(bcfg, W, e)
    try:
        return pre.run().float().cpu().numpy().astype(np.float64)
    finally:
        pre.close()


def _cmp(name, got, ref, max_tol, mean_tol):
    d = np.abs(got - ref)
    print(f"{name}: max|d| = {d.max():.3e} (tol {max_tol}), mean|d| = {d.mean():.3e} (tol {mean_tol}), "
          f"rms ref {np.sqrt(np.mean(ref ** 2)):.3f}", flush=True)
    assert np.all(np.isfinite(got))
    assert d.max() <= max_tol and d.mean() <= mean_tol


SMALL = wl.PI0_VLM_BF16.with_(name="vlm_small", n_layers=2, d_model=512, n_heads=4, head_dim=128, n_kv_heads=2,
                              d_ff=1536, prefix_len=100, seed_base=8100)

CASES = {
    "geglu_rope_ragged": SMALL,
    "swiglu_norope_hd64": SMALL.with_(name="s2", mlp="swiglu", rope_base=0.0, head_dim=64, n_heads=8,
                                      n_kv_heads=8, prefix_len=77, seed_base=8200),
    "gelu_mqa_hd256": SMALL.with_(name="s3", mlp="gelu", head_dim=256, n_heads=4, n_kv_heads=1, prefix_len=130,
                                  seed_base=8300),
}


@pytest.mark.parametrize("case", sorted(CASES))
def test_prefill_small_batched(torch, case):
    """Two-layer backbones at small widths, B = 2 requests with a ragged
    prefix length (tiles with partial tails), GeGLU / SwiGLU / GELU MLPs,
    RoPE on and off, grouped and multi-query K/V heads."""
    bcfg = CASES[case]
    W = wl.make_backbone_weights(bcfg)
    e = wl.make_prefix_embeds(bcfg, 2)
    got = _prefill(bcfg, W, e)
    ref = O.prefix_prefill(bcfg, W, e)
    _cmp(case, got, ref, 8e-2, 1.2e-2)


def test_prefill_gemma_width_two_layers(torch):
    """Two layers at the Gemma-2B-shaped widths (d 2048, 8 x 256 heads over one
    K/V head, GeGLU 16384) over the 816-row prefix."""
    bcfg = wl.PI0_VLM_BF16.with_(n_layers=2)
    W = wl.make_backbone_weights(bcfg)
    e = wl.make_prefix_embeds(bcfg, 1)
    got = _prefill(bcfg, W, e)
    ref = O.prefix_prefill(bcfg, W, e)
    _cmp("gemma-width 2 layers", got, ref, 8e-2, 1.2e-2)


def test_prefill_is_bidirectional_on_gpu(torch):
    """The kernels' attention over the prefix is bidirectional: changing the
    last row's embedding changes the first row's hidden state (by far more
    than the bf16 noise), as the oracle says."""
    bcfg = SMALL
    W = wl.make_backbone_weights(bcfg)
    e = wl.make_prefix_embeds(bcfg, 1)
    e2 = e.copy()
    e2[0, -1] = wl.round_bf16(e2[0, -1] + 1.0)
    a, b = _prefill(bcfg, W, e), _prefill(bcfg, W, e2)
    ra, rb = O.prefix_prefill(bcfg, W, e), O.prefix_prefill(bcfg, W, e2)
    moved, moved_ref = np.abs(b[0, 0] - a[0, 0]).max(), np.abs(rb[0, 0] - ra[0, 0]).max()
    print(f"row 0 moved by {moved:.3e} on the GPU, {moved_ref:.3e} in the oracle")
    assert moved > 0.5 * moved_ref > 1e-3


@pytest.mark.timeout(1200)
def test_pi0_observation_path_full(torch):
    """The pi0-shaped observation path at full size: the Gemma-2B-shaped
    18-layer prefill over 816 rows, its hidden states projected by the
    pi0-shaped expert's vla_prefix_kv_build, then vla_denoise at T = 10; the
    hidden states against the oracle's prefill, the chunk against the oracle's
    chain (prefill -> cross K/V -> Euler) at the 2e-2 bar."""
    from vla_testlib import Pipeline, Prefill
    bcfg = wl.PI0_VLM_BF16
    cfg = wl.PI0_BF16
    print("generating the backbone's weights ...", flush=True)
    Wb = wl.make_backbone_weights(bcfg)
    e = wl.make_prefix_embeds(bcfg, 1)
    W = wl.make_weights(cfg)
    inp = wl.make_batch(cfg, 1)
    tau = wl.uniform_schedule(cfg.n_steps)
    pre = Prefill(bcfg, Wb, e)
    try:
        hidden = pre.run()
        pipe = Pipeline(cfg, W, inp)
        try:
            pipe.model.prefix_kv_build(hidden, 1, bcfg.prefix_len, pipe.cache, pipe.cache_bytes)
            chunk = pipe.denoise(tau).cpu().numpy().astype(np.float64)
        finally:
            pipe.close()
        h_got = hidden.float().cpu().numpy().astype(np.float64)
    finally:
        pre.close()
    print("GPU done; oracle prefill (about a minute) ...", flush=True)
    h_ref = O.prefix_prefill(bcfg, Wb, e)
    _cmp("pi0 18-layer prefill", h_got, h_ref, 0.25, 3.5e-2)
    print("oracle expert ...", flush=True)
    cache = O.prefix_kv_build(cfg, W, h_ref)
    ref = O.denoise(cfg, W, cache, inp["noise"], inp["state"], tau)
    err = np.abs(chunk - ref).max()
    print(f"pi0 observation path (prefill + cross K/V + 10 Euler steps): max|d| = {err:.3e}")
    assert np.all(np.isfinite(chunk)) and err <= 2e-2


def _tern(n_layers, **scale_of):
    bcfg = wl.BITNET_W2A8.with_(n_layers=n_layers)
    W = wl.make_backbone_weights(bcfg)
    for l in range(n_layers):
        for n, f in scale_of.items():
            W[f"B{l}.{n}.scale"] = np.float32(W[f"B{l}.{n}.scale"] * f)
    return bcfg, W, wl.make_prefix_embeds(bcfg, 1)


@pytest.mark.parametrize("P,B,seed", [(77, 2, 9300), (50, 1, 9400), (200, 1, 9500)])
def test_ternary_prefill_small_batched(torch, P, B, seed):
    """Two W2A8 layers at small widths (d 512, 4 x 128 heads over 2 K/V heads,
    ReLU^2-GLU 1536), both branches on: 154 rows of two requests (the tiled
    W2A8 kernel with a ragged last row tile), 50 rows (the few-row kernel) and
    200 rows.  The CPU study with the kernels' bf16 storage points emulated
    gives max 9.6e-3 / mean 1.4e-3 on these cases; the bf16 output adds up to
    2^-9 relative.  The layers move the hidden states by mean 0.10."""
    bcfg = wl.BITNET_W2A8.with_(name="tern_small", n_layers=2, d_model=512, n_heads=4, head_dim=128,
                                n_kv_heads=2, d_ff=1536, prefix_len=P, seed_base=seed)
    W = wl.make_backbone_weights(bcfg)
    e = wl.make_prefix_embeds(bcfg, B)
    got = _prefill(bcfg, W, e)
    ref = O.prefix_prefill(bcfg, W, e)
    _cmp(f"ternary small P={P} B={B}", got, ref, 4e-2, 6e-3)
    W0 = dict(W)
    for l in range(2):
        W0[f"B{l}.W_o.scale"] = np.float32(0.0)
        W0[f"B{l}.W_d.scale"] = np.float32(0.0)
    assert np.abs(ref - O.prefix_prefill(bcfg, W0, e)).mean() > 0.05


def test_ternary_prefill_mlp_branch(torch):
    """One BitNet-width W2A8 layer (d 2560, 20 x 128 heads over 5 K/V heads,
    ReLU^2-GLU 6912, 512 rows) with the attention branch off (W_o scale 0):
    every quantiser input of the MLP branch is fp32 on both sides, so only
    rounding-level differences (fp32 against fp64 sums) move a code, at a .5
    boundary.  A CPU study of the oracle with 1e-7 relative jitter on its
    quantiser inputs puts that at max 2.5e-2, mean 6e-5; the bf16 output
    adds up to 2^-9 relative (mean about 8e-4 on unit-RMS values)."""
    bcfg, W, e = _tern(1, W_o=0.0)
    got = _prefill(bcfg, W, e)
    ref = O.prefix_prefill(bcfg, W, e)
    _cmp("ternary MLP branch", got, ref, 6e-2, 3e-3)


def test_ternary_prefill_one_layer(torch):
    """One BitNet-width W2A8 layer with both branches on."""
    bcfg, W, e = _tern(1)
    got = _prefill(bcfg, W, e)
    ref = O.prefix_prefill(bcfg, W, e)
    _cmp("ternary 1 layer", got, ref, 0.3, 4e-2)


@pytest.mark.timeout(900)
def test_ternary_prefill_full_depth(torch):
    """The paper's 30-layer W2A8 prefill at BitNet widths, 512 rows, with the
    W_o and W_d scales at 0.1x (so that one flipped code does not cascade);
    the layers still move the hidden states by far more than the tolerance."""
    bcfg, W, e = _tern(30, W_o=0.1, W_d=0.1)
    got = _prefill(bcfg, W, e)
    print("GPU done; oracle (about 30 s) ...", flush=True)
    ref = O.prefix_prefill(bcfg, W, e)
    _cmp("ternary 30 layers", got, ref, 0.6, 0.1)
    W0 = dict(W)
    for l in range(30):
        W0[f"B{l}.W_o.scale"] = np.float32(0.0)
        W0[f"B{l}.W_d.scale"] = np.float32(0.0)
    assert np.abs(ref - O.prefix_prefill(bcfg, W0, e)).mean() > 0.3


@pytest.mark.parametrize("wtype", ["bf16", "ternary"])
def test_prefill_single_prefix_row(torch, wtype):
    """A prefix of one row per request (two requests): attention over a single
    key (weight 1), RoPE at position 0 only, every GEMM with M = 2."""
    if wtype == "bf16":
        bcfg = SMALL.with_(name="one_row", prefix_len=1, seed_base=8500)
        tol = (8e-2, 1.2e-2)
    else:
        bcfg = wl.BITNET_W2A8.with_(name="one_row_tern", n_layers=2, d_model=512, n_heads=4, head_dim=128,
                                    n_kv_heads=2, d_ff=1536, prefix_len=1, seed_base=8600)
        tol = (4e-2, 6e-3)
    W = wl.make_backbone_weights(bcfg)
    e = wl.make_prefix_embeds(bcfg, 2)
    got = _prefill(bcfg, W, e)
    ref = O.prefix_prefill(bcfg, W, e)
    _cmp(f"one prefix row ({wtype})", got, ref, *tol)
