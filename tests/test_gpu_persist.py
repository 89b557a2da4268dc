"""Parity of the persistent step-loop driver (loop mode 2: one kernel of
co-resident workgroups runs every solver step) against the fp64 oracle, against the
launch-per-phase graph driver, and run-to-run determinism.

The driver covers batch-1 bf16 experts with joint attention whose shape fits
its team layout (8 teams of 32 workgroups: query heads and MLP columns split
over the teams).  Cases span one and two heads per team, grouped K/V heads,
GeGLU / SwiGLU / GELU MLPs, ragged prefix and chunk lengths (prefix blocks and
chunk blocks with partial 32-key tails, 16-row query tiles with a ragged last
tile) and T = 1 .. 10.  Tolerance on the final chunk: max|d| <= 2e-2 (bf16).
"""
import numpy as np
import pytest

import workloads as wl
from oracle import vla_oracle as O

pytestmark = pytest.mark.gpu

TOL = 2e-2

SMALL = wl.PI0_BF16.with_(name="pi0_small", n_layers=2, d_model=512, head_dim=64, d_ff=2048, d_prefix=512,
                          prefix_len=100, n_steps=3, seed_base=6000)

CASES = {
    "small_geglu": SMALL,
    "small_gelu_ragged": SMALL.with_(name="small_gelu", mlp="gelu", n_action=20, prefix_len=37, n_steps=4,
                                     seed_base=6100),
    "two_heads_per_team_swiglu": SMALL.with_(name="h16", n_heads=16, n_kv_heads=2, mlp="swiglu", n_action=9,
                                             prefix_len=70, d_action=7, d_state=7, n_steps=2, seed_base=6200),
    "d1024_hd128_t1": SMALL.with_(name="d1024", d_model=1024, head_dim=128, d_ff=4096, d_prefix=1024,
                                  n_action=33, prefix_len=129, n_steps=1, seed_base=6300),
    # chunks of up to 50 rows fold rows 48-49 of the GEMM phases' operand into
    # one load per wave; longer chunks (51..64 rows) take the unfolded form
    "chunk49_one_tail_row": SMALL.with_(name="n49", n_action=49, prefix_len=64, n_steps=2, seed_base=6400),
    "chunk61_unfolded": SMALL.with_(name="n61", n_action=61, prefix_len=45, n_steps=2, seed_base=6500),
    "chunk64_unfolded_d1024": SMALL.with_(name="n64", d_model=1024, head_dim=128, d_ff=4096, d_prefix=1024,
                                          n_action=64, prefix_len=90, n_steps=1, seed_base=6600),
}


@pytest.fixture(scope="module")
def torch():
    import torch as t
    if not t.cuda.is_available():
        pytest.skip("no GPU")
    return t


def _run(cfg, W, inp, tau, loop_mode, reps=1, expect_persist=True):
    from vla_testlib import Pipeline
    pipe = Pipeline(cfg, W, inp, loop_mode)
    import torch
    try:
        pipe.build_cache()
        if loop_mode == 2:
            pipe.model.set_trace(1)   # the persistent kernel's marks show that it ran
        outs = []
        for _ in range(reps):
            out = pipe.denoise(tau)
            torch.cuda.synchronize()
            outs.append(out.cpu().numpy().astype(np.float64).copy())
        if loop_mode == 2:
            tr = pipe.model.trace_read()
            ran = tr is not None and bool(tr.any())
            assert ran == expect_persist, f"persistent kernel ran: {ran}, expected {expect_persist}"
        return outs
    finally:
        pipe.close()


@pytest.mark.parametrize("case", sorted(CASES))
def test_persist_matches_oracle_and_graph(torch, case):
    cfg = CASES[case]
    W = wl.make_weights(cfg)
    inp = wl.make_batch(cfg, 1)
    tau = wl.uniform_schedule(cfg.n_steps)
    cache = O.prefix_kv_build(cfg, W, inp["prefix"])
    ref = O.denoise(cfg, W, cache, inp["noise"], inp["state"], tau)
    got = _run(cfg, W, inp, tau, loop_mode=2, reps=2)
    graph = _run(cfg, W, inp, tau, loop_mode=1)[0]
    err = np.abs(got[0] - ref).max()
    dg = np.abs(got[0] - graph).max()
    print(f"{case}: persistent vs oracle max|d| = {err:.3e}, vs graph driver {dg:.3e}")
    assert np.all(np.isfinite(got[0]))
    assert err <= TOL, f"{case}: max|d| {err}"
    assert dg <= TOL
    assert np.array_equal(got[0], got[1]), "persistent driver is not deterministic"


def test_persist_pi0_full(torch):
    """The full pi0-shaped workload (18 layers, 816 prefix rows, T = 10) with
    denormalisation statistics."""
    from vla_testlib import Pipeline, to_device, workload
    cfg, W, inp = workload("pi0_bf16", 1)
    tau = wl.uniform_schedule(cfg.n_steps)
    mean = np.linspace(-0.5, 0.5, cfg.d_action).astype(np.float32)
    std = np.linspace(0.5, 2.0, cfg.d_action).astype(np.float32)
    cache = O.prefix_kv_build(cfg, W, inp["prefix"])
    ref = O.denoise(cfg, W, cache, inp["noise"], inp["state"], tau, mean, std)
    pipe = Pipeline(cfg, W, inp, loop_mode=2)
    try:
        pipe.build_cache()
        got = pipe.denoise(tau, to_device(mean), to_device(std)).cpu().numpy().astype(np.float64)
    finally:
        pipe.close()
    err = np.abs(got - ref).max()
    print(f"pi0_bf16 persistent: max|d| = {err:.3e}")
    assert err <= TOL


def test_ineligible_model_falls_back(torch):
    """Loop mode 2 on a model the persistent kernel does not cover (fp32,
    self + cross attention) runs the graph driver: identical output."""
    cfg = wl.TINY_F32
    W = wl.make_weights(cfg)
    inp = wl.make_batch(cfg, 2)
    tau = wl.uniform_schedule(cfg.n_steps)
    a = _run(cfg, W, inp, tau, loop_mode=2, expect_persist=False)[0]
    b = _run(cfg, W, inp, tau, loop_mode=1)[0]
    assert np.array_equal(a, b)


def test_persist_barrier_timeout_is_reported(torch):
    """The failure path, forced from the host: with a spin limit of 0 every
    barrier wait that is not satisfied at its first look gives up, so every
    workgroup leaves early (each wait is bounded: no kernel hangs).  The
    call's chunk is NaN; vla_model_check then reports VLA_E_DEVICE once; the
    next call (default limit) starts from a cleared error word and matches
    the oracle.  A failure that has completed before the next vla_denoise is
    reported by that call, before it enqueues anything."""
    from paper_2606_08094_amd.vla import VlaError
    from vla_testlib import Pipeline
    cfg = CASES["small_geglu"]
    W = wl.make_weights(cfg)
    inp = wl.make_batch(cfg, 1)
    tau = wl.uniform_schedule(cfg.n_steps)
    ref = O.denoise(cfg, W, O.prefix_kv_build(cfg, W, inp["prefix"]), inp["noise"], inp["state"], tau)
    pipe = Pipeline(cfg, W, inp, loop_mode=2)
    try:
        pipe.build_cache()
        pipe.model.set_spin_limit(0)
        bad = pipe.denoise(tau).cpu().numpy()
        with pytest.raises(VlaError, match="VLA_E_DEVICE"):
            pipe.model.check()
        assert np.isnan(bad).all()
        pipe.model.check()                      # reported once
        pipe.model.set_spin_limit(-1)
        good = pipe.denoise(tau).cpu().numpy().astype(np.float64)
        pipe.model.check()
        assert np.abs(good - ref).max() <= TOL
        # a completed failure is reported by the next denoise call itself
        pipe.model.set_spin_limit(0)
        pipe.denoise(tau)
        torch.cuda.synchronize()
        pipe.model.set_spin_limit(-1)
        with pytest.raises(VlaError, match="VLA_E_DEVICE"):
            pipe.denoise(tau)
        again = pipe.denoise(tau).cpu().numpy().astype(np.float64)
        pipe.model.check()
        assert np.array_equal(again, good)
    finally:
        pipe.close()
