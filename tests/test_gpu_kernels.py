"""Kernel-level parity of the HIP path against the fp64 oracle, through the
C ABI (include/vla.h, include/vla_test.h), on seeded inputs at the
workloads' real shapes plus ragged ones (M, N, K not multiples of the tiles)."""
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


def _vla():
    from paper_2606_08094_amd import vla
    return vla


def _dev(torch, arr, bf16=False):
    from vla_testlib import to_device
    return to_device(arr, bf16)


def _fp32_bound(x, w):
    """Rigorous fp32-accumulation bound for x w^T: K * 2^-24 * |x| |w|^T (+ slack)."""
    K = x.shape[1]
    return (K * 2.0 ** -24 + 1e-7) * (np.abs(x) @ np.abs(w).T) + 1e-30


GEMM_SHAPES = [
    # (M, N, K)  pi0 / SmolVLA / tiny shapes, ragged edges, large M
    (50, 2560, 1024), (50, 1024, 2048), (50, 1024, 4096), (50, 32, 1024),
    (50, 1600, 720), (50, 720, 2048), (50, 6, 720),
    (8, 384, 256), (8, 7, 256), (1, 5, 8), (17, 33, 136), (100, 2560, 1024),
    (816, 512, 2048), (10, 6144, 1024), (128, 1024, 4096), (129, 64, 64), (50, 1024, 8192),
    # split-K with four W subtiles per workgroup (variant 4), ragged in M, N and the last K split
    (100, 1024, 4096), (90, 1000, 4096), (120, 1536, 3072),
    # large M (batched requests, prefix K/V build): the tiled kernel, ragged in M, N and K
    (400, 1024, 4096), (1600, 2560, 1024), (257, 136, 72), (300, 100, 200), (520, 200, 640),
]

# 0 runtime choice, 1 wide, 2 skinny, 3 tiled (runtime tile), 4 split-K partials (the residual
# projections' launch) summed by the library, 10..14 tiled with a fixed tile (14: 256 x 256, eight waves)
GEMM_VARIANTS = (0, 1, 2, 3, 4, 10, 11, 12, 13, 14)


@pytest.mark.parametrize("elem", [1, 0])
@pytest.mark.parametrize("M,N,K", GEMM_SHAPES)
def test_gemm_parity(torch, elem, M, N, K):
    if elem == 0 and K % 4:
        pytest.skip("fp32 needs K % 4 == 0")
    bf = elem == 1
    seed = 1000 * M + N + K
    x = wl.random_matrix((M, K), seed, 1.0, bf16=bf)
    w = wl.random_matrix((N, K), seed + 1, 0.05, bf16=bf)
    ref = O.linear(x, w)
    bound = _fp32_bound(x.astype(np.float64), w.astype(np.float64))
    vla = _vla()
    for variant in GEMM_VARIANTS:
        y = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
        try:
            vla.test_gemm(elem, _dev(torch, x, bf), _dev(torch, w, bf), M, N, K, y, variant=variant)
        except vla.VlaError as e:
            # shape outside the skinny kernel, or not a bf16 GEMM with M > 128 for the tiled one
            assert e.status == 3 and (variant == 2 or (variant == 4 and not bf and M > 128)
                                      or (variant == 3 or variant >= 10) and (not bf or M <= 128)
                                      or variant == 14 and K % 64), e
            continue
        got = y.cpu().numpy().astype(np.float64)
        err = np.abs(got - ref)
        assert np.all(err <= bound), f"variant={variant} max err {err.max()} worst ratio {(err / bound).max()}"


ATTN_CASES = [
    # (elem, mode, B, n, P, H, G, hd)
    (1, 2, 1, 50, 816, 8, 1, 256),     # pi0 joint
    (1, 1, 1, 50, 241, 15, 5, 64),     # SmolVLA cross
    (1, 0, 1, 50, 0, 15, 5, 64),       # SmolVLA self
    (1, 2, 1, 8, 512, 20, 5, 128),     # ternary workload joint
    (1, 2, 2, 100, 300, 8, 1, 256),    # batched requests
    (1, 1, 1, 3, 1, 4, 2, 64),         # single prefix key
    (0, 0, 1, 8, 0, 4, 1, 64),         # tiny fp32 self
    (0, 1, 1, 8, 64, 4, 1, 64),        # tiny fp32 cross
    (0, 2, 2, 19, 45, 6, 3, 128),      # ragged fp32 joint
    (1, 2, 3, 100, 2048, 8, 1, 256),   # stress shape: 68 key blocks, looped in chunks
]


@pytest.mark.parametrize("case", ATTN_CASES, ids=[str(c) for c in ATTN_CASES])
@pytest.mark.parametrize("kv_split", [0, 1, 3, 201, 403, 800, 1000, 1001, 1005])
def test_attention_parity(torch, case, kv_split):
    """kv_split: key splits (% 100) and query-head groups per K/V head (// 100);
    1000 + s: the 128-row tiled kernel with s splits of 64-key blocks."""
    elem, mode, B, n, P, H, G, hd = case
    if kv_split >= 1000 and elem != 1:
        pytest.skip("the tiled kernel is bf16 only")
    if kv_split < 1000 and kv_split // 100 and (H // G) % (kv_split // 100):
        pytest.skip("head groups must divide the heads per K/V head")
    bf = elem == 1
    s = 7 * n + P + H + hd + mode
    q = wl.random_matrix((B * n, H * hd), s, 1.0, bf16=bf)
    ks = wl.random_matrix((B * n, G * hd), s + 1, 1.0, bf16=bf)
    vs = wl.random_matrix((B * n, G * hd), s + 2, 1.0, bf16=bf)
    kc = wl.random_matrix((B, G, max(P, 1), hd), s + 3, 1.0, bf16=bf)
    vc = wl.random_matrix((B, G, max(P, 1), hd), s + 4, 1.0, bf16=bf)
    o = torch.full((B * n, H * hd), float("nan"), dtype=torch.bfloat16 if bf else torch.float32, device="cuda")
    _vla().test_attention(elem, mode, _dev(torch, q, bf), _dev(torch, ks, bf), _dev(torch, vs, bf),
                          _dev(torch, kc, bf), _dev(torch, vc, bf), B, n, P, H, G, hd, o, kv_split=kv_split)
    got = o.float().cpu().numpy().astype(np.float64)
    for b in range(B):
        rows = slice(b * n, (b + 1) * n)
        kself = ks[rows].reshape(n, G, hd).transpose(1, 0, 2)
        vself = vs[rows].reshape(n, G, hd).transpose(1, 0, 2)
        if mode == 0:
            kk, vv = kself, vself
        elif mode == 1:
            kk, vv = kc[b], vc[b]
        else:
            kk, vv = np.concatenate([kc[b], kself], 1), np.concatenate([vc[b], vself], 1)
        ref = O.attention(q[rows], kk, vv, H, G, hd)
        # bf16: probabilities and the output are rounded to bf16 (relative 2^-8 each)
        tol = 1.2e-2 * np.abs(vv).max() if bf else 2e-5
        err = np.abs(got[rows] - ref).max()
        assert err <= tol, f"request {b}: max err {err} > {tol}"


CAUSAL_CASES = [
    # (elem, mode, B, n, P, H, G, hd): self and joint only
    (1, 2, 1, 50, 816, 8, 1, 256),     # pi0 joint
    (1, 0, 1, 50, 0, 15, 5, 64),       # SmolVLA self
    (1, 2, 2, 100, 300, 8, 1, 256),    # batched requests, several action-key blocks
    (0, 0, 1, 8, 0, 4, 1, 64),         # tiny fp32 self
    (1, 2, 4, 70, 64, 16, 2, 128),     # tiled-kernel sizes, ragged blocks
]


@pytest.mark.parametrize("case", CAUSAL_CASES, ids=[str(c) for c in CAUSAL_CASES])
@pytest.mark.parametrize("kv_split", [0, 1, 3, 1000, 1005])
def test_attention_causal_parity(torch, case, kv_split):
    """The causal action-token variant (mode + 4): query t sees every prefix
    row and the action keys 0 .. t; compared with the oracle's masked routine
    (whole splits can be masked for the first queries)."""
    elem, mode, B, n, P, H, G, hd = case
    if kv_split >= 1000 and elem != 1:
        pytest.skip("the tiled kernel is bf16 only")
    bf = elem == 1
    s = 11 * n + P + H + hd + mode
    q = wl.random_matrix((B * n, H * hd), s, 1.0, bf16=bf)
    ks = wl.random_matrix((B * n, G * hd), s + 1, 1.0, bf16=bf)
    vs = wl.random_matrix((B * n, G * hd), s + 2, 1.0, bf16=bf)
    kc = wl.random_matrix((B, G, max(P, 1), hd), s + 3, 1.0, bf16=bf)
    vc = wl.random_matrix((B, G, max(P, 1), hd), s + 4, 1.0, bf16=bf)
    o = torch.full((B * n, H * hd), float("nan"), dtype=torch.bfloat16 if bf else torch.float32, device="cuda")
    _vla().test_attention(elem, mode + 4, _dev(torch, q, bf), _dev(torch, ks, bf), _dev(torch, vs, bf),
                          _dev(torch, kc, bf), _dev(torch, vc, bf), B, n, P, H, G, hd, o, kv_split=kv_split)
    got = o.float().cpu().numpy().astype(np.float64)
    for b in range(B):
        rows = slice(b * n, (b + 1) * n)
        kself = ks[rows].reshape(n, G, hd).transpose(1, 0, 2)
        vself = vs[rows].reshape(n, G, hd).transpose(1, 0, 2)
        if mode == 0:
            kk, vv, c = kself, vself, 0
        else:
            kk, vv, c = np.concatenate([kc[b], kself], 1), np.concatenate([vc[b], vself], 1), P
        ref = O.attention(q[rows], kk, vv, H, G, hd, causal_from=c)
        tol = 1.2e-2 * np.abs(vv).max() if bf else 2e-5
        err = np.abs(got[rows] - ref).max()
        assert np.isfinite(got[rows]).all() and err <= tol, f"request {b}: max err {err} > {tol}"
        # the kernel applied the mask: it is much closer to the masked result than
        # the unmasked result is (with a long prefix the mask moves little)
        eff = np.abs(ref - O.attention(q[rows], kk, vv, H, G, hd)).max()
        assert err < 0.5 * eff, f"request {b}: err {err} vs mask effect {eff}"


@pytest.mark.parametrize("elem,u_f32,M,d,nsplit", [
    (1, 0, 50, 1024, 4),    # pi0 width, bf16 u, four split-K partials
    (1, 0, 50, 720, 0),     # SmolVLA width (d % 1024 != 0), no residual update
    (0, 1, 8, 256, 3),      # tiny fp32 expert
    (1, 1, 8, 2560, 2),     # ternary width: fp32 u for the int8 quantiser
    (1, 0, 3, 4096, 1),     # widest row the kernel takes, ragged row count
])
def test_adarms_parity(torch, elem, u_f32, M, d, nsplit):
    """Residual finish + adaRMS row kernel against the oracle's ada_rms on the
    updated residual x + alpha * sum of the partials.  x is fp32 throughout;
    u is compared after the kernel's own rounding of its output (bf16: 2^-8
    relative), fp32 u at 1e-5 relative."""
    rng = np.random.default_rng(100 + d + nsplit)
    x = (rng.standard_normal((M, d)) * 3.0).astype(np.float32)
    part = rng.standard_normal((max(nsplit, 1), M, d)).astype(np.float32)
    alpha = rng.uniform(-1.0, 1.0, d).astype(np.float32)
    gamma = (0.3 * rng.standard_normal(d)).astype(np.float32)
    beta = (0.3 * rng.standard_normal(d)).astype(np.float32)
    eps = 1e-6
    xd = torch.from_numpy(x).cuda()
    dev = {k: torch.from_numpy(v).cuda() for k, v in dict(part=part, alpha=alpha, gamma=gamma, beta=beta).items()}
    u = torch.empty((M, d), dtype=torch.float32 if u_f32 or elem == 0 else torch.bfloat16, device="cuda")
    _vla().test_adarms(elem, xd, dev["part"] if nsplit else None, nsplit, dev["alpha"] if nsplit else None,
                       dev["gamma"], dev["beta"], M, d, eps, u, bool(u_f32))
    x_ref = x.astype(np.float64)
    if nsplit:
        x_ref = x_ref + alpha.astype(np.float64) * part[:nsplit].astype(np.float64).sum(0)
    u_ref = O.ada_rms(x_ref, gamma, beta, eps)
    x_got = xd.cpu().numpy().astype(np.float64)
    u_got = u.float().cpu().numpy().astype(np.float64)
    assert np.abs(x_got - x_ref).max() <= 1e-5 * max(1.0, np.abs(x_ref).max())
    rel = 2.0 ** -8 if (elem == 1 and not u_f32) else 1e-5
    assert np.all(np.abs(u_got - u_ref) <= rel * np.abs(u_ref) + 1e-5), np.abs(u_got - u_ref).max()


@pytest.mark.parametrize("name", ["tiny_f32", "pi0_bf16", "smolvla_bf16"])
def test_time_cond_parity(torch, name):
    """Time-conditioning precompute (sinusoid, time MLP, every layer's W_mod and
    W_fm) for a non-uniform schedule: (1) against the oracle's primitives
    rounded to bf16 exactly where the kernels store bf16 (the embedding,
    SiLU(W_t1 e + b_t1) and SiLU(c)), leaving fp32 accumulation order; (2)
    against the plain oracle's modulation() within the bound those bf16 stores
    can produce (fp32 models: within fp32 accumulation)."""
    from vla_testlib import device_weights
    cfg = wl.CONFIGS[name]
    W = wl.make_weights(cfg)
    tau = np.array([1.0, 0.83, 0.51, 0.5, 0.12, 0.0], np.float32)
    T, d = len(tau) - 1, cfg.d_model
    vla = _vla()
    model = vla.Model(cfg, device_weights(cfg, W))
    try:
        rows = cfg.n_layers * 3 * cfg.n_sub * d
        mods = torch.empty((T, rows), dtype=torch.float32, device="cuda")
        modf = torch.empty((T, 2 * d), dtype=torch.float32, device="cuda")
        vla.test_time_cond(model, list(tau), mods, modf)
        got_m = mods.cpu().numpy().astype(np.float64)
        got_f = modf.cpu().numpy().astype(np.float64)
    finally:
        model.close()
    bf = cfg.wtype != "f32"
    st = O.round_to_bf16 if bf else (lambda v: v)
    W_mod = np.concatenate([W[f"L{l}.W_mod"] for l in range(cfg.n_layers)], 0)
    b_mod = np.concatenate([W[f"L{l}.b_mod"] for l in range(cfg.n_layers)], 0)
    for k in range(T):
        e = st(O.time_embedding(float(tau[k]), d))
        h1 = st(O.silu(O.linear(e, W["W_t1"], W["b_t1"])))
        sc = st(O.silu(O.linear(h1, W["W_t2"], W["b_t2"])))
        ref_m = O.linear(sc, W_mod, b_mod)
        ref_f = O.linear(sc, W["W_fm"], W["b_fm"])
        # fp32: accumulation order only.  bf16: a stored value that lies at a
        # bf16 rounding boundary may round the other way on one side (one ulp,
        # 2^-8 relative, of an element of |x| <= 1, weighted by |w| ~ 0.02)
        tol = 1e-3 if bf else 1e-5
        assert np.abs(got_m[k] - ref_m).max() <= tol, (k, np.abs(got_m[k] - ref_m).max())
        assert np.abs(got_f[k] - ref_f).max() <= tol, (k, np.abs(got_f[k] - ref_f).max())
        mods_o, fin_o = O.modulation(cfg, W, float(tau[k]))
        flat = np.concatenate([np.concatenate([np.concatenate(gba) for gba in ml]) for ml in mods_o])
        flat_f = np.concatenate(fin_o)
        if not bf:  # fp32 models: the whole chain against the oracle's own modulation()
            assert np.abs(got_m[k] - flat).max() <= 1e-4
            assert np.abs(got_f[k] - flat_f).max() <= 1e-4
        else:
            # bf16 models against the plain oracle: each of the kernels' three
            # bf16 stores (e, SiLU(W_t1 e + b_t1), SiLU(c)) moves a value v by
            # an independent error of at most 2^-9 |v| (variance (2^-9 v)^2 / 3
            # if uniform); propagated through W^2 with |SiLU'| <= 1.1, six
            # standard deviations of the result bound the difference, plus
            # fp32 accumulation
            e64 = O.time_embedding(float(tau[k]), d)
            h64 = O.silu(O.linear(e64, W["W_t1"], W["b_t1"]))
            sc64 = O.silu(O.linear(h64, W["W_t2"], W["b_t2"]))
            u = 2.0 ** -9
            vh = 1.21 * (W["W_t1"].astype(np.float64) ** 2 @ ((u * e64) ** 2 / 3)) + (u * h64) ** 2 / 3
            vsc = 1.21 * (W["W_t2"].astype(np.float64) ** 2 @ vh) + (u * sc64) ** 2 / 3
            bm = 6.0 * np.sqrt(W_mod.astype(np.float64) ** 2 @ vsc) + 1e-5
            bfm = 6.0 * np.sqrt(W["W_fm"].astype(np.float64) ** 2 @ vsc) + 1e-5
            assert np.all(np.abs(got_m[k] - flat) <= bm), np.abs(got_m[k] - flat).max()
            assert np.all(np.abs(got_f[k] - flat_f) <= bfm), np.abs(got_f[k] - flat_f).max()


def _tie_rows():
    import os
    rows = []
    for line in open(os.path.join(os.path.dirname(__file__), "golden", "quantizer_ties.txt")):
        if line.startswith("row:"):
            rows.append([float(v) for v in line.split()[1:]])
    return rows


@pytest.mark.parametrize("K", [300, 301])   # whole 16-byte vectors / a ragged row (looping kernel)
def test_quantize_i8_bit_exact(torch, K):
    rows = _tie_rows()
    x = wl.random_matrix((37, K), 5, 3.0)
    for i, r in enumerate(rows):
        x[i, :] = 0
        x[i, :len(r)] = r
    x[len(rows), :] = 0.0
    qd = torch.empty((37, K), dtype=torch.int8, device="cuda")
    rd = torch.empty(37, dtype=torch.float32, device="cuda")
    _vla().test_quantize_i8(_dev(torch, x), 37, K, qd, rd)
    q_ref, r_ref = O.quantize_int8_rows(x)
    assert np.array_equal(qd.cpu().numpy(), q_ref)
    assert np.array_equal(rd.cpu().numpy(), r_ref)


# (M, K, row pitch): the W2A8 expert's O / down inputs, the largest row, a
# pitched row, and rows the register-resident kernel does not take (K or the
# pitch not a multiple of 8 values)
@pytest.mark.parametrize("M,K,ldx", [(8, 2560, 2560), (8, 6912, 6912), (37, 16384, 16384), (512, 6912, 6912),
                                     (9, 256, 264), (5, 130, 130), (3, 136, 140)])
def test_quantize_bf16_rows_bit_exact(torch, M, K, ldx):
    """bf16 rows (the attention output and the GLU output of the W2A8 path)
    quantise to the oracle's codes and scales exactly: the bf16 values are
    exact in fp32, so both sides quantise the same numbers."""
    x = wl.random_matrix((M, ldx), 17 + K, 2.0)
    rows = _tie_rows()
    for i, r in enumerate(rows[:max(0, M - 1)]):
        x[i, :] = 0
        x[i, :min(len(r), K)] = r[:K]
    if M > len(rows):
        x[len(rows), :] = 0.0
    xb = wl.round_bf16(x)
    qd = torch.empty((M, K), dtype=torch.int8, device="cuda")
    rd = torch.empty(M, dtype=torch.float32, device="cuda")
    _vla().test_quantize_bf16(_dev(torch, xb, bf16=True), M, K, ldx, qd, rd)
    q_ref, r_ref = O.quantize_int8_rows(np.ascontiguousarray(xb[:, :K]))
    assert np.array_equal(qd.cpu().numpy(), q_ref)
    assert np.array_equal(rd.cpu().numpy(), r_ref)


TERN_SHAPES = [(8, 3840, 2560), (8, 2560, 2560), (8, 13824, 2560), (8, 2560, 6912), (56, 2560, 6912),
               (512, 1280, 2560), (512, 3840, 2560), (512, 13824, 2560), (512, 2560, 6912), (300, 200, 640),
               (3, 17, 64), (20, 100, 192), (5, 7, 68), (2, 3, 4)]


@pytest.mark.parametrize("M,N,K", TERN_SHAPES)
def test_ternary_gemm_bit_exact(torch, M, N, K):
    x = wl.random_int8((M, K), M + N)
    w = wl.random_ternary((N, K), K + N)
    # include the extreme rows: all -128 and all 127
    x[0, :] = -128
    if M > 1:
        x[1, :] = 127
    packed = wl.pack_ternary(w)
    out = torch.full((M, N), 12345, dtype=torch.int32, device="cuda")
    _vla().ternary_gemm(torch.from_numpy(x).cuda(), torch.from_numpy(packed).cuda(), M, N, K, out)
    assert np.array_equal(out.cpu().numpy().astype(np.int64), O.ternary_gemm(x, packed, K))


def test_ternary_gemm_empty(torch):
    out = torch.zeros(1, dtype=torch.int32, device="cuda")
    x = torch.zeros(16, dtype=torch.int8, device="cuda")
    w = torch.zeros(16, dtype=torch.uint8, device="cuda")
    _vla().ternary_gemm(x, w, 0, 5, 64, out)
    _vla().ternary_gemm(x, w, 3, 0, 64, out)
    assert int(out.cpu()[0]) == 0


@pytest.mark.parametrize("elem,rows,rpr,nheads,hd,col0,ld,pos0", [
    (1, 100, 50, 8, 256, 0, 2560, 816),     # pi0 queries of 2 requests after an 816-row prefix
    (1, 100, 50, 1, 256, 2048, 2560, 816),  # their keys (columns after the 2048 query columns)
    (1, 3 * 241, 241, 1, 64, 0, 64, 0),     # cached prefix keys, positions 0 .. P-1
    (0, 16, 8, 4, 64, 0, 256, 0),           # fp32 self attention
])
def test_rope_kernel(torch, elem, rows, rpr, nheads, hd, col0, ld, pos0):
    """The RoPE kernel against the oracle's rotation on the same (bf16 or
    fp32) inputs: columns outside the heads stay untouched."""
    bf = elem == 1
    x = wl.random_matrix((rows, ld), 60 + rows + hd, 1.0, bf16=bf)
    base = 10000.0
    pos = pos0 + np.arange(rows) % rpr
    ref = x.astype(np.float64).copy()
    ref[:, col0:col0 + nheads * hd] = O.rope(x[:, col0:col0 + nheads * hd], pos, nheads, hd, base)
    xd = _dev(torch, x, bf)
    _vla().test_rope(elem, xd, rows, rpr, ld, col0, nheads, hd, pos0, base)
    got = xd.float().cpu().numpy().astype(np.float64)
    # bf16: one rounding of the stored result (2^-9 relative) on values of norm <= |x|;
    # fp32 angles lose about 1e-7 relative at positions up to ~1000
    tol = 8e-3 * np.abs(x).max() if bf else 2e-4 * np.abs(x).max()
    err = np.abs(got - ref).max()
    assert err <= tol, f"max err {err} > {tol}"
    outside = np.ones(ld, bool)
    outside[col0:col0 + nheads * hd] = False
    assert np.array_equal(got[:, outside], x[:, outside].astype(np.float64))


# The ternary model's projections (scope row a11) at M = 8 and the alternative M = 56, plus
# ragged shapes: more token rows than one pass of the dot4 kernel, N not a multiple of 16, and
# K over two 4096-wide slices.
TERN_GEMM_SHAPES = [(8, 3840, 2560), (8, 2560, 2560), (8, 13824, 2560), (8, 2560, 6912),
                    (56, 2560, 6912), (17, 100, 320), (70, 33, 128), (1, 16, 64), (33, 4100, 8192)]


@pytest.mark.parametrize("M,N,K", TERN_GEMM_SHAPES)
def test_ternary_gemm_dot4_matches_mfma(torch, M, N, K):
    """The VALU sdot4 kernel and the int8-MFMA launch on the same int8 codes and
    packed weights: both sums are exact int32, so the dequantised outputs are
    identical, and they match the oracle's exact sum to fp32 rounding."""
    x = wl.random_matrix((M, K), 5 + M + K, 1.0)
    q, r = O.quantize_int8_rows(x)
    w = wl.random_ternary((N, K), 6 + N)
    wp = wl.pack_ternary(w)
    wscale = (0.01 + 0.02 * (np.arange(N) % 7) / 7.0).astype(np.float32)
    acc = O.ternary_gemm(q, wp, K)
    ref = acc.astype(np.float64) * (wscale.astype(np.float64)[None, :] * r.astype(np.float64)[:, None] / 127.0)
    qd = torch.from_numpy(np.ascontiguousarray(q)).cuda()
    rd = torch.from_numpy(r).cuda()
    wd = torch.from_numpy(wp).cuda()
    sd = torch.from_numpy(wscale).cuda()
    ys = []
    for variant in (0, 1):
        y = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
        _vla().test_ternary_gemm(qd, rd, wd, sd, M, N, K, variant, y)
        ys.append(y.cpu().numpy())
    assert np.array_equal(ys[0], ys[1])
    np.testing.assert_allclose(ys[1], ref, rtol=1e-6, atol=1e-7)


TILE_VARIANTS = {2: "32-row tiles", 3: "64-row tiles", 4: "128-row tiles", 5: "64 x 256 tiles (eight waves)",
                 6: "128 x 256 tiles (eight waves)", 7: "32-row tiles, two K groups", 8: "64-row tiles, two K groups",
                 9: "128-row tiles, two K groups"}


@pytest.mark.parametrize("M,N,K", [(512, 2560, 2560), (512, 2560, 6912), (512, 3840, 2560), (300, 200, 640),
                                   (129, 130, 128), (160, 1000, 384)])
def test_ternary_tile_configurations_identical(torch, M, N, K):
    """Every row-tile height of the many-row tiled kernel (ragged row and
    column tiles included) gives the library launch's
    dequantised outputs bit for bit (exact int32 sums), and those match the
    oracle's exact sum to fp32 rounding."""
    x = wl.random_matrix((M, K), 7 + M + K, 1.0)
    q, r = O.quantize_int8_rows(x)
    q[0, :] = -128
    w = wl.random_ternary((N, K), 8 + N)
    wp = wl.pack_ternary(w)
    wscale = (0.01 + 0.02 * (np.arange(N) % 5) / 5.0).astype(np.float32)
    acc = O.ternary_gemm(q, wp, K)
    ref = acc.astype(np.float64) * (wscale.astype(np.float64)[None, :] * r.astype(np.float64)[:, None] / 127.0)
    qd = torch.from_numpy(np.ascontiguousarray(q)).cuda()
    rd = torch.from_numpy(r).cuda()
    wd = torch.from_numpy(wp).cuda()
    sd = torch.from_numpy(wscale).cuda()
    ys = {}
    for variant in [0] + sorted(TILE_VARIANTS):
        y = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
        _vla().test_ternary_gemm(qd, rd, wd, sd, M, N, K, variant, y)
        ys[variant] = y.cpu().numpy()
    np.testing.assert_allclose(ys[0], ref, rtol=1e-6, atol=1e-7)
    for v in TILE_VARIANTS:
        assert np.array_equal(ys[v], ys[0]), TILE_VARIANTS[v]


@pytest.mark.parametrize("M,N,K", [(8, 3840, 2560), (8, 2560, 6912), (512, 1280, 2560), (13, 70, 128),
                                   (56, 2560, 2560), (20, 512, 6912), (40, 200, 320), (64, 48, 64),
                                   (512, 13824, 2560), (512, 2560, 6912), (300, 200, 640), (129, 130, 128)])
def test_ternary_linear(torch, M, N, K):
    x = wl.random_matrix((M, K), 3 + M, 1.0)
    w = wl.random_ternary((N, K), 4 + N)
    scale = np.float32(0.0244)
    y = torch.empty((M, N), dtype=torch.float32, device="cuda")
    _vla().test_ternary_linear(_dev(torch, x), torch.from_numpy(wl.pack_ternary(w)).cuda(), M, N, K, float(scale), y)
    ref = O.ternary_linear(x, w, scale)
    # identical int8 codes and int32 sums; only the fp32 dequantisation rounds
    np.testing.assert_allclose(y.cpu().numpy(), ref, rtol=1e-6, atol=1e-7)


def test_ternary_layer_quantiser_codes_differ_by_one(torch):
    """One W2A8 attention branch of the ternary expert's first layer (full
    widths: d 2560, 20 x 128 query heads, 5 K/V heads, 512 cached prefix rows),
    both sides starting from the same float32 sublayer input u: the kernels
    project Q, K, V (W2A8, stored bf16 as the expert stores them), run joint
    attention over the bf16 cache built by vla_prefix_kv_build, and quantise
    the attention output for W_o; the oracle does the same in float64.  The
    quantiser codes of u itself are identical (both quantise the same float32
    values).  At the O-projection input the two sides' values differ by the
    kernel's bf16 storage and fp32 sums, so some codes differ: each by exactly
    one, each explained by a rounding boundary lying between the two sides'
    scaled values, and at most 15% of them (the bf16 steps are 2^-9 relative
    against a quantiser step of max|o| / 127)."""
    from vla_testlib import Pipeline, device_weights
    vla = _vla()
    cfg = wl.TERNARY_W2A8.with_(n_layers=1)
    W = wl.make_weights(cfg)
    inp = wl.make_batch(cfg, 1)
    d, H, G, hd, n, P = cfg.d_model, cfg.n_heads, cfg.n_kv_heads, cfg.head_dim, cfg.n_action, cfg.prefix_len
    mods, _ = O.modulation(cfg, W, 0.0)
    gamma, beta, _ = mods[0][0]
    x0 = O.input_embedding(cfg, W, inp["noise"][0], inp["state"][0])
    u = O.ada_rms(x0, gamma, beta, cfg.rms_eps).astype(np.float32)
    # codes of the sublayer input: same float32 values on both sides
    qd = torch.empty((n, d), dtype=torch.int8, device="cuda")
    rd = torch.empty(n, dtype=torch.float32, device="cuda")
    vla.test_quantize_i8(_dev(torch, u), n, d, qd, rd)
    q_u, r_u = O.quantize_int8_rows(u)
    assert np.array_equal(qd.cpu().numpy(), q_u) and np.array_equal(rd.cpu().numpy(), r_u)
    # oracle branch in float64
    cache = O.prefix_kv_build(cfg, W, inp["prefix"])
    q_ref = O._lin(cfg, W, "L0.W_q", u)
    k_ref = O.split_heads(O._lin(cfg, W, "L0.W_k", u), G, hd)
    v_ref = O.split_heads(O._lin(cfg, W, "L0.W_v", u), G, hd)
    o_ref = O.attention(q_ref, np.concatenate([cache[0, 0, 0], k_ref], 1),
                        np.concatenate([cache[0, 1, 0], v_ref], 1), H, G, hd)
    # kernel branch: W2A8 projections from u, bf16 stores, the library's cache
    dw = device_weights(cfg, W)
    ud = _dev(torch, u)
    proj = {}
    for name, N in (("W_q", H * hd), ("W_k", G * hd), ("W_v", G * hd)):
        y = torch.empty((n, N), dtype=torch.float32, device="cuda")
        vla.test_ternary_linear(ud, dw["L0." + name], n, N, d, float(W["L0." + name + ".scale"]), y)
        proj[name] = y.to(torch.bfloat16).contiguous()
    pipe = Pipeline(cfg, W, inp)
    try:
        pipe.build_cache()
        c = pipe.cache.view(torch.bfloat16).view(1, 2, 1, G, P, hd)
        kc, vc = c[0, 0].contiguous(), c[0, 1].contiguous()
        o = torch.empty((n, H * hd), dtype=torch.bfloat16, device="cuda")
        vla.test_attention(1, 2, proj["W_q"], proj["W_k"], proj["W_v"], kc, vc, 1, n, P, H, G, hd, o)
        of = o.float().contiguous()
        qo = torch.empty((n, H * hd), dtype=torch.int8, device="cuda")
        ro = torch.empty(n, dtype=torch.float32, device="cuda")
        vla.test_quantize_i8(of, n, H * hd, qo, ro)
        torch.cuda.synchronize()
        o_got = of.cpu().numpy()
        c_got, r_got = qo.cpu().numpy().astype(np.int64), ro.cpu().numpy()
    finally:
        pipe.close()
    c_ref, r_ref = O.quantize_int8_rows(o_ref.astype(np.float32))
    c_ref = c_ref.astype(np.int64)
    diff = c_got != c_ref
    frac = float(diff.mean())
    s_ref = o_ref * (127.0 / r_ref.astype(np.float64))[:, None]
    s_got = o_got.astype(np.float64) * (127.0 / r_got.astype(np.float64))[:, None]
    print(f"W2A8 layer 0: O-projection codes differing from the oracle: {int(diff.sum())} of {diff.size} "
          f"({100 * frac:.2f}%), max |d o| = {np.abs(o_got - o_ref).max():.2e}")
    assert np.all(np.abs(c_got - c_ref) <= 1)
    bnd = 0.5 * (c_got + c_ref)                      # the boundary the two values straddle
    lo, hi = np.minimum(s_ref, s_got), np.maximum(s_ref, s_got)
    slack = 1e-5 * (1.0 + np.abs(bnd))
    assert np.all((bnd[diff] >= lo[diff] - slack[diff]) & (bnd[diff] <= hi[diff] + slack[diff]))
    assert frac <= 0.15
