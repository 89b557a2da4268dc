"""Pins of the fp64 oracle against facts fixed outside it: closed forms,
invariants, special cases that reduce to textbook definitions, hand-derived
fixtures (tests/golden/) and brute force on tiny inputs.

Each test names the plausible oracle mistake it would catch.
"""
import itertools
import math
import os

import numpy as np
import pytest

import workloads as wl
from oracle import vla_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")

TINY = wl.ExpertConfig(
    name="pin_tiny", n_layers=2, d_model=8, n_heads=2, head_dim=4, n_kv_heads=1,
    d_ff=16, d_prefix=6, n_action=3, d_action=2, d_state=3,
    pattern="self_cross", mlp="gelu", wtype="f32", prefix_len=3, n_steps=3, seed_base=77)


def _rng(seed=0):
    return np.random.default_rng(seed)


# --- brute-force evaluators (pure-Python loops, tiny shapes only) ------------

def bf_linear(u, W):
    n, k = len(u), len(u[0])
    return [[sum(float(u[i][j]) * float(W[o][j]) for j in range(k)) for o in range(len(W))]
            for i in range(n)]


def bf_attention(q, k, v, H, G, hd):
    """Textbook softmax attention per head; head i uses K/V head i // (H/G)."""
    n = len(q)
    per = H // G
    out = [[0.0] * (H * hd) for _ in range(n)]
    for i in range(H):
        g = i // per
        for r in range(n):
            scores = []
            for key in range(len(k[g])):
                s = sum(float(q[r][i * hd + c]) * float(k[g][key][c]) for c in range(hd))
                scores.append(s / math.sqrt(hd))
            mx = max(scores)
            w = [math.exp(s - mx) for s in scores]
            z = sum(w)
            for c in range(hd):
                out[r][i * hd + c] = sum(w[key] * float(v[g][key][c]) for key in range(len(w))) / z
    return np.array(out)


# --- Euler integrator (explicit Euler, t = 1 -> 0) -------------------------

SCHED = np.array([1.0, 0.7, 0.45, 0.1, 0.0])   # non-uniform, decreasing


def test_euler_zero_field_returns_noise():
    """v = 0 must leave a0 untouched (catches a stray additive term)."""
    a0 = _rng(1).standard_normal((5, 3))
    out = O.euler_integrate(lambda a, k, t: np.zeros_like(a), a0, SCHED)
    assert np.array_equal(out, a0)


def test_euler_constant_field_endpoint():
    """v = c gives a_T = a0 + (tau_T - tau_0) c exactly up to rounding
    (catches a wrong sign of the step or a missing step)."""
    a0 = _rng(2).standard_normal((5, 3))
    c = _rng(3).standard_normal((5, 3))
    out = O.euler_integrate(lambda a, k, t: c, a0, SCHED)
    np.testing.assert_allclose(out, a0 + (SCHED[-1] - SCHED[0]) * c, rtol=0, atol=1e-14)


def test_euler_linear_field_product():
    """v = lam a gives a_T = prod_k (1 + lam dt_k) a0 (catches evaluating v at
    the end of the interval instead of the start)."""
    a0 = _rng(4).standard_normal((4, 2))
    lam = -0.8
    out = O.euler_integrate(lambda a, k, t: lam * a, a0, SCHED)
    fac = np.prod([1 + lam * (SCHED[i + 1] - SCHED[i]) for i in range(len(SCHED) - 1)])
    np.testing.assert_allclose(out, fac * a0, rtol=1e-14)


def test_euler_time_argument_is_interval_start():
    """v = t: a_T - a0 = sum_k dt_k tau_k (left Riemann sum)."""
    a0 = np.zeros((1, 1))
    out = O.euler_integrate(lambda a, k, t: np.full_like(a, t), a0, SCHED)
    expect = sum((SCHED[i + 1] - SCHED[i]) * SCHED[i] for i in range(len(SCHED) - 1))
    assert abs(out[0, 0] - expect) < 1e-15


# --- time embedding --------------------------------------------------------------

def test_time_embedding_golden():
    """Hand-derived d = 4 values (catches a swapped sin/cos half or wrong periods)."""
    rows = np.loadtxt(os.path.join(GOLDEN, "time_embedding.txt"))
    for t, *e in rows:
        np.testing.assert_allclose(O.time_embedding(t, 4), e, atol=1e-12)


def test_time_embedding_zero_and_norm():
    d = 1024
    e0 = O.time_embedding(0.0, d)
    assert np.array_equal(e0, np.concatenate([np.zeros(d // 2), np.ones(d // 2)]))
    for t in (0.1, 0.37, 0.9, 1.0):
        assert abs(np.sum(O.time_embedding(t, d) ** 2) - d / 2) < 1e-9


def test_time_embedding_period_endpoints():
    """First pair uses period 4e-3, last pair period 4 (geometric ends)."""
    d, t = 16, 0.3
    e = O.time_embedding(t, d)
    assert abs(e[0] - math.sin(2 * math.pi * t / 4e-3)) < 1e-9
    assert abs(e[d // 2 - 1] - math.sin(2 * math.pi * t / 4.0)) < 1e-12
    assert abs(e[d - 1] - math.cos(2 * math.pi * t / 4.0)) < 1e-12


# --- adaRMS -------------------------------------------------------------------------

def test_adarms_unit_mean_square():
    """gamma = beta = 0: mean(u^2) = m / (m + eps), m = mean(x^2)."""
    x = _rng(5).standard_normal((6, 32))
    eps = 1e-3
    u = O.ada_rms(x, np.zeros(32), np.zeros(32), eps)
    m = np.mean(x * x, axis=-1)
    np.testing.assert_allclose(np.mean(u * u, axis=-1), m / (m + eps), rtol=1e-13)


def test_adarms_scale_invariance_and_affine():
    """u(kx) = u(x) at eps = 0, and gamma, beta enter as (1+gamma) and +beta."""
    x = _rng(6).standard_normal((3, 16))
    g, b = np.zeros(16), np.zeros(16)
    base = O.ada_rms(x, g, b, 0.0)
    np.testing.assert_allclose(O.ada_rms(7.5 * x, g, b, 0.0), base, rtol=1e-13)
    np.testing.assert_allclose(O.ada_rms(x, np.ones(16), np.full(16, 0.5), 0.0), 2 * base + 0.5,
                               rtol=1e-13)


# --- activations ---------------------------------------------------------------------

def test_activations_closed_forms():
    from scipy.special import erf
    x = np.linspace(-6, 6, 241)
    exact_gelu = 0.5 * x * (1 + erf(x / np.sqrt(2)))
    # the tanh form stays within 1e-3 of the erf form everywhere
    assert np.max(np.abs(O.gelu_tanh(x) - exact_gelu)) < 1e-3
    assert O.gelu_tanh(0.0) == 0.0
    assert abs(O.silu(1.0) - 1.0 / (1.0 + math.exp(-1.0))) < 1e-15
    assert O.silu(0.0) == 0.0
    # gate vs up roles: the activation applies to the gate only
    assert O.mlp_activation("geglu", 0.0, 5.0) == 0.0
    assert O.mlp_activation("swiglu", 0.0, 5.0) == 0.0
    assert O.mlp_activation("relu2glu", -1.0, 3.0) == 0.0
    assert O.mlp_activation("relu2glu", 2.0, 3.0) == 12.0
    assert abs(O.mlp_activation("swiglu", 1.0, 2.0) - 2.0 / (1.0 + math.exp(-1.0))) < 1e-15


# --- linear / attention -----------------------------------------------------------

def test_linear_bruteforce():
    """[out][in] convention: y = u W^T (catches a transposed operand)."""
    u = _rng(7).standard_normal((3, 5))
    W = _rng(8).standard_normal((4, 5))
    np.testing.assert_allclose(O.linear(u, W), bf_linear(u, W), rtol=1e-13)


def test_softmax_rows_sum_to_one():
    s = _rng(9).standard_normal((7, 40)) * 30
    p = O.softmax_rows(s)
    assert np.max(np.abs(p.sum(-1) - 1)) < 1e-15 * 40
    assert np.all(p >= 0)


@pytest.mark.parametrize("H,G", [(2, 1), (4, 2), (6, 3), (3, 3)])
def test_attention_bruteforce_gqa(H, G):
    """Grouped K/V heads: consecutive query heads share one K/V head."""
    hd, n, keys = 4, 3, 5
    r = _rng(10 + H + G)
    q = r.standard_normal((n, H * hd))
    k = r.standard_normal((G, keys, hd))
    v = r.standard_normal((G, keys, hd))
    np.testing.assert_allclose(O.attention(q, k, v, H, G, hd), bf_attention(q, k, v, H, G, hd),
                               rtol=1e-12, atol=1e-14)


def test_attention_single_key_returns_v():
    r = _rng(11)
    q = r.standard_normal((4, 2 * 8))
    k = r.standard_normal((1, 1, 8))
    v = r.standard_normal((1, 1, 8))
    out = O.attention(q, k, v, 2, 1, 8)
    for i in range(2):
        np.testing.assert_allclose(out[:, i * 8:(i + 1) * 8], np.repeat(v[0], 4, axis=0), rtol=1e-15)


def test_attention_zero_query_is_mean_of_values():
    r = _rng(12)
    k = r.standard_normal((2, 9, 4))
    v = r.standard_normal((2, 9, 4))
    out = O.attention(np.zeros((3, 4 * 4)), k, v, 4, 2, 4)
    for i in range(4):
        np.testing.assert_allclose(out[:, i * 4:(i + 1) * 4],
                                   np.repeat(v[i // 2].mean(0, keepdims=True), 3, 0), rtol=1e-13)


def test_attention_key_permutation_invariance():
    r = _rng(13)
    q = r.standard_normal((5, 8))
    k = r.standard_normal((1, 11, 4))
    v = r.standard_normal((1, 11, 4))
    perm = r.permutation(11)
    np.testing.assert_allclose(O.attention(q, k[:, perm], v[:, perm], 2, 1, 4),
                               O.attention(q, k, v, 2, 1, 4), rtol=1e-12)


def test_attention_query_permutation_equivariance():
    r = _rng(14)
    q = r.standard_normal((6, 8))
    k = r.standard_normal((2, 6, 4))
    v = r.standard_normal((2, 6, 4))
    perm = r.permutation(6)
    np.testing.assert_allclose(O.attention(q[perm], k, v, 2, 2, 4),
                               O.attention(q, k, v, 2, 2, 4)[perm], rtol=1e-12)


@pytest.mark.parametrize("c", [0, 3])
def test_attention_causal_rows_equal_truncated_unmasked(c):
    """Causal action-token variant: query i sees keys 0 .. c+i (c keys before
    the action tokens), i.e. the unmasked routine (here the brute-force one)
    over the truncated key set."""
    H, G, hd, n = 4, 2, 4, 5
    r = _rng(40 + c)
    q = r.standard_normal((n, H * hd))
    k = r.standard_normal((G, c + n, hd))
    v = r.standard_normal((G, c + n, hd))
    out = O.attention(q, k, v, H, G, hd, causal_from=c)
    for i in range(n):
        ref = bf_attention(q[i:i + 1], k[:, :c + i + 1], v[:, :c + i + 1], H, G, hd)
        np.testing.assert_allclose(out[i:i + 1], ref, rtol=1e-12, atol=1e-14)


def test_attention_causal_first_and_last_query():
    """Self attention with the causal mask: token 0 sees only key 0 (its value
    comes back exactly); the last token sees every key (unmasked result)."""
    r = _rng(42)
    q = r.standard_normal((6, 2 * 4))
    k = r.standard_normal((1, 6, 4))
    v = r.standard_normal((1, 6, 4))
    out = O.attention(q, k, v, 2, 1, 4, causal_from=0)
    for h in range(2):
        np.testing.assert_allclose(out[0, h * 4:(h + 1) * 4], v[0, 0], rtol=1e-15)
    np.testing.assert_allclose(out[5], O.attention(q, k, v, 2, 1, 4)[5], rtol=1e-12)


@pytest.mark.parametrize("pattern", ["self_cross", "joint"])
def test_causal_expert_earlier_tokens_ignore_later_ones(pattern):
    """With the causal variant, action token i of the chunk depends only on the
    prefix and tokens 0 .. i: changing the noise of the last token leaves every
    other row of the chunk unchanged.  Bidirectional attention (the default)
    spreads the change to every row."""
    for causal in (True, False):
        cfg = TINY.with_(pattern=pattern, causal_self=causal)
        W, inp, cache = _tiny_setup(cfg)
        tau = wl.uniform_schedule(cfg.n_steps)
        a = O.denoise(cfg, W, cache, inp["noise"], inp["state"], tau)
        noise2 = inp["noise"].copy()
        noise2[:, -1] += 0.5
        b = O.denoise(cfg, W, cache, noise2, inp["state"], tau)
        moved = np.abs(a - b).max(axis=-1)[0]   # per action row of request 0
        assert moved[-1] > 1e-3
        if causal:
            assert np.all(moved[:-1] == 0.0)
        else:
            assert np.all(moved[:-1] > 1e-9)


def test_cross_only_pattern_tokens_interact_only_through_prefix():
    """Cross-attention-only layers (Evo-1's DiT head): the action tokens never
    attend to one another, so changing one token's noise leaves every other
    row of the chunk unchanged; the prefix still reaches every row."""
    cfg = TINY.with_(pattern="cross")
    assert cfg.sublayers(0) == ["cross", "mlp"] and cfg.sublayers(1) == ["cross", "mlp"]
    W, inp, cache = _tiny_setup(cfg)
    tau = wl.uniform_schedule(cfg.n_steps)
    a = O.denoise(cfg, W, cache, inp["noise"], inp["state"], tau)
    noise2 = inp["noise"].copy()
    noise2[:, 2] += 0.5
    b = O.denoise(cfg, W, cache, noise2, inp["state"], tau)
    moved = np.abs(a - b).max(axis=-1)[0]
    assert moved[2] > 1e-3 and np.all(np.delete(moved, 2) == 0.0)
    cache2 = O.prefix_kv_build(cfg, W, inp["prefix"] * 1.5)
    c = O.denoise(cfg, W, cache2, inp["noise"], inp["state"], tau)
    assert np.all(np.abs(a - c).max(axis=-1)[0] > 1e-6)


def test_rope_two_dims_is_plane_rotation():
    """head_dim 2: w_0 = 1, so position p turns (x0, x1) by p radians."""
    r = _rng(50)
    x = r.standard_normal((5, 2 * 3))   # 3 heads of 2 dims
    pos = np.array([0.0, 1.0, 2.5, -3.0, 7.0])
    y = O.rope(x, pos, 3, 2, 10000.0)
    for i, p in enumerate(pos):
        rot = np.array([[np.cos(p), -np.sin(p)], [np.sin(p), np.cos(p)]])
        for h in range(3):
            np.testing.assert_allclose(y[i, 2 * h:2 * h + 2], rot @ x[i, 2 * h:2 * h + 2], rtol=1e-13, atol=1e-15)


def test_rope_identity_norms_and_relative_positions():
    """Position 0 is the identity; every rotated pair keeps its norm; scores of
    rotated queries and keys depend only on the position difference."""
    r = _rng(51)
    hd, base = 8, 10000.0
    q = r.standard_normal((4, hd))
    k = r.standard_normal((4, hd))
    np.testing.assert_array_equal(O.rope(q, np.zeros(4), 1, hd, base), q)
    y = O.rope(q, np.arange(4) * 3.0, 1, hd, base)
    h = hd // 2
    np.testing.assert_allclose(y[:, :h] ** 2 + y[:, h:] ** 2, q[:, :h] ** 2 + q[:, h:] ** 2, rtol=1e-12)
    pm, pn = np.array([5.0, 9.0, 2.0, 0.0]), np.array([1.0, 4.0, 8.0, 3.0])
    s1 = np.sum(O.rope(q, pm, 1, hd, base) * O.rope(k, pn, 1, hd, base), axis=1)
    s2 = np.sum(O.rope(q, pm + 11, 1, hd, base) * O.rope(k, pn + 11, 1, hd, base), axis=1)
    np.testing.assert_allclose(s1, s2, rtol=1e-10, atol=1e-12)


def test_rope_variant_joint_positions_follow_the_prefix():
    """RoPE on the joint sequence: rotating every key and query by one extra
    position (prefix and action rows alike) leaves the chunk unchanged, since
    only position differences enter the scores."""
    cfg = TINY.with_(pattern="joint", rope_base=10000.0)
    W, inp, cache = _tiny_setup(cfg)
    tau = wl.uniform_schedule(cfg.n_steps)
    a = O.denoise(cfg, W, cache, inp["noise"], inp["state"], tau)
    b0 = O.denoise(cfg.with_(rope_base=0.0), W, O.prefix_kv_build(cfg.with_(rope_base=0.0), W, inp["prefix"]),
                   inp["noise"], inp["state"], tau)
    # the positions matter (small weights keep the effect small, 5e-8 here); the
    # shift check below resolves far less than that
    assert np.abs(a - b0).max() > 1e-8
    real_rope = O.rope
    try:
        O.rope = lambda x, pos, nh, hd, base: real_rope(x, np.asarray(pos) + 1.0, nh, hd, base)
        cache1 = O.prefix_kv_build(cfg, W, inp["prefix"])
        c = O.denoise(cfg, W, cache1, inp["noise"], inp["state"], tau)
    finally:
        O.rope = real_rope
    np.testing.assert_allclose(c, a, rtol=1e-11, atol=1e-13)


@pytest.mark.parametrize("pattern", ["self_cross", "joint"])
def test_state_token_variant(pattern):
    """State as its own token: with zero state weights and bias, the state
    token is a zero row that still takes part in attention (so the chunk
    differs from the added-state model); in a cross-only expert the action
    rows never see it, and the chunk equals the added-state model with a zero
    state contribution."""
    cfg = TINY.with_(pattern=pattern, state_token=True)
    W, inp, cache = _tiny_setup(cfg)
    tau = wl.uniform_schedule(cfg.n_steps)
    W0 = dict(W)
    W0["W_s"] = np.zeros_like(W["W_s"])
    W0["b_s"] = np.zeros_like(W["b_s"])
    a = O.denoise(cfg, W0, cache, inp["noise"], inp["state"], tau)
    b = O.denoise(cfg.with_(state_token=False), W0, cache, inp["noise"], inp["state"], tau)
    assert a.shape == b.shape and np.abs(a - b).max() > 1e-9
    cfgc = TINY.with_(pattern="cross", state_token=True)
    Wc, inpc, cachec = _tiny_setup(cfgc)
    Wc0 = dict(Wc)
    Wc0["W_s"] = np.zeros_like(Wc["W_s"])
    Wc0["b_s"] = np.zeros_like(Wc["b_s"])
    c = O.denoise(cfgc, Wc0, cachec, inpc["noise"], inpc["state"], tau)
    d = O.denoise(cfgc.with_(state_token=False), Wc0, cachec, inpc["noise"], inpc["state"], tau)
    np.testing.assert_allclose(c, d, rtol=1e-13, atol=1e-15)


# --- ternary / quantiser ------------------------------------------------------------

def test_pack_golden_and_unpack_roundtrip():
    rows = np.loadtxt(os.path.join(GOLDEN, "ternary_pack.txt"), dtype=np.int64)
    w = rows[:, :4]
    packed = wl.pack_ternary(w)
    assert packed[:, 0].tolist() == rows[:, 4].tolist()
    assert np.array_equal(O.unpack_ternary(packed, 4), w)
    big = wl.random_ternary((7, 64), 3)
    assert np.array_equal(O.unpack_ternary(wl.pack_ternary(big), 64), big)


def test_ternary_gemm_bruteforce_and_special_cases():
    x = wl.random_int8((5, 32), 1)
    w = wl.random_ternary((6, 32), 2)
    acc = O.ternary_gemm(x, wl.pack_ternary(w), 32)
    bf = [[sum(int(x[m, k]) * int(w[n, k]) for k in range(32)) for n in range(6)] for m in range(5)]
    assert acc.tolist() == bf
    ones = np.ones((3, 32), np.int8)
    assert np.array_equal(O.ternary_gemm(x, wl.pack_ternary(0 * ones), 32), np.zeros((5, 3)))
    assert np.array_equal(O.ternary_gemm(x, wl.pack_ternary(ones), 32)[:, 0], x.astype(np.int64).sum(1))
    assert np.array_equal(O.ternary_gemm(x, wl.pack_ternary(-ones), 32)[:, 2], -x.astype(np.int64).sum(1))
    onehot = np.zeros((2, 32), np.int8)
    onehot[0, 5] = 1
    onehot[1, 31] = -1
    acc = O.ternary_gemm(x, wl.pack_ternary(onehot), 32)
    assert np.array_equal(acc[:, 0], x[:, 5]) and np.array_equal(acc[:, 1], -x[:, 31].astype(np.int64))


def test_ternary_gemm_extreme_fits_int32():
    k = 6912
    x = np.full((2, k), -128, np.int8)
    w = np.ones((1, k), np.int8)
    assert O.ternary_gemm(x, wl.pack_ternary(w), k)[0, 0] == -128 * k


def _read_quant_golden():
    rows, codes = [], []
    for line in open(os.path.join(GOLDEN, "quantizer_ties.txt")):
        if line.startswith("row:"):
            rows.append([float(v) for v in line.split()[1:]])
        elif line.startswith("codes:"):
            codes.append([int(v) for v in line.split()[1:]])
    return rows, codes


def test_quantizer_golden_ties_floor_zero_row():
    for row, code in zip(*_read_quant_golden()):
        q, r = O.quantize_int8_rows(np.array([row], np.float32))
        assert q[0].tolist() == code


def test_quantizer_single_value_and_range():
    u = np.zeros((2, 10), np.float32)
    u[0, 3] = 0.37
    u[1, 7] = -5.0
    q, r = O.quantize_int8_rows(u)
    assert q[0, 3] == 127 and q[1, 7] == -127 and np.count_nonzero(q) == 2
    big = wl.random_matrix((50, 300), 5)
    q, _ = O.quantize_int8_rows(big)
    assert q.min() >= -127 and q.max() == 127


def test_ternary_linear_integer_rows():
    """A row whose absmax is 127 and whose values are integers quantises to
    itself, so y = s_w * (u . w) exactly (catches a wrong dequant scale)."""
    u = np.zeros((1, 8), np.float32)
    u[0, :] = [127, -3, 5, 0, 2, -127, 1, 1]
    w = wl.random_ternary((3, 8), 4)
    y = O.ternary_linear(u, w, np.float32(0.5))
    np.testing.assert_allclose(y, 0.5 * (u.astype(np.float64) @ w.T.astype(np.float64)), rtol=1e-15)


# --- denormalise -------------------------------------------------------------------------

def test_denormalize_identity_and_affine():
    a = _rng(15).standard_normal((4, 3))
    assert np.array_equal(O.denormalize(a), a)
    np.testing.assert_allclose(O.denormalize(a, np.ones(3), 2 * np.ones(3)), 2 * a + 1, rtol=1e-15)


# --- whole-expert special cases ------------------------------------------------------

def _tiny_setup(cfg=TINY, B=1):
    W = wl.make_weights(cfg)
    inp = wl.make_batch(cfg, B)
    cache = O.prefix_kv_build(cfg, W, inp["prefix"])
    return W, inp, cache


def test_prefix_kv_build_bruteforce_entries():
    """cache[c][0|1][b][g][p][:] is head g's slice of X_p W^T (catches a
    transposed projection or a wrong head split)."""
    cfg = TINY.with_(n_kv_heads=2, n_heads=2)
    W, inp, cache = _tiny_setup(cfg, B=2)
    for c, l in enumerate([l for l in range(cfg.n_layers) if cfg.has_prefix(l)]):
        for b, g, p in itertools.product(range(2), range(2), range(cfg.prefix_len)):
            for kv, name in ((0, "W_kc"), (1, "W_vc")):
                Wm = W[f"L{l}.{name}"]
                rows = Wm[g * cfg.head_dim:(g + 1) * cfg.head_dim]
                bf = bf_linear([inp["prefix"][b, p]], rows)[0]
                np.testing.assert_allclose(cache[c, kv, b, g, p], bf, rtol=1e-12)


def test_zero_velocity_end_to_end():
    """W_out = 0, b_out = 0: the expert's velocity vanishes, output = noise."""
    W, inp, cache = _tiny_setup()
    W["W_out"] = np.zeros_like(W["W_out"])
    W["b_out"] = np.zeros_like(W["b_out"])
    tau = wl.uniform_schedule(TINY.n_steps)
    out = O.denoise(TINY, W, cache, inp["noise"], inp["state"], tau)
    assert np.array_equal(out, inp["noise"].astype(np.float64))


def test_constant_velocity_end_to_end():
    """W_out = 0, b_out = c: exact Euler endpoint noise + (tau_T - tau_0) c,
    then denormalised."""
    W, inp, cache = _tiny_setup()
    c = np.array([0.3, -1.1])
    W["W_out"] = np.zeros_like(W["W_out"])
    W["b_out"] = c.astype(np.float32)
    tau = np.array([1.0, 0.6, 0.25, 0.0], np.float32)
    mean, std = np.array([1.0, -2.0]), np.array([0.5, 3.0])
    out = O.denoise(TINY, W, cache, inp["noise"], inp["state"], tau, mean, std)
    expect = (inp["noise"][0] + (0.0 - 1.0) * c.astype(np.float32).astype(np.float64)) * std + mean
    np.testing.assert_allclose(out[0], expect, rtol=1e-14)


def test_regression_head_is_single_pass():
    """head_regression: the output is the head's value, not a + dt v."""
    cfg = TINY.with_(head_regression=True, n_steps=1)
    W, inp, cache = _tiny_setup(cfg)
    W["W_out"] = np.zeros_like(W["W_out"])
    W["b_out"] = np.array([0.25, -0.5], np.float32)
    out = O.denoise(cfg, W, cache, inp["noise"], inp["state"], wl.uniform_schedule(1))
    assert np.array_equal(out[0], np.tile([0.25, -0.5], (cfg.n_action, 1)))


@pytest.mark.parametrize("pattern", ["self_cross", "joint", "alt"])
def test_zero_gates_equal_zero_layers(pattern):
    """All residual gates alpha = 0: every layer is skipped, so the forward
    equals the same expert with no layers (catches an ungated residual)."""
    cfg = TINY.with_(pattern=pattern, mlp="swiglu")
    W, inp, cache = _tiny_setup(cfg)
    d, ns = cfg.d_model, cfg.n_sub
    for l in range(cfg.n_layers):
        for j in range(ns):
            W[f"L{l}.W_mod"][(3 * j + 2) * d:(3 * j + 3) * d] = 0
            W[f"L{l}.b_mod"][(3 * j + 2) * d:(3 * j + 3) * d] = 0
    a = inp["noise"][0].astype(np.float64)
    cb = cache[:, :, 0]
    full = O.expert_forward(cfg, W, cb, a, inp["state"][0], 0.4)
    empty = O.expert_forward(cfg.with_(n_layers=0), W, None, a, inp["state"][0], 0.4)
    np.testing.assert_allclose(full, empty, rtol=1e-13)


@pytest.mark.parametrize("pattern", ["self_cross", "joint", "alt"])
def test_cache_reuse_equals_recompute(pattern):
    """The cached cross K/V and K/V recomputed at every solver step agree
    bitwise in fp64."""
    cfg = TINY.with_(pattern=pattern)
    W, inp, cache = _tiny_setup(cfg, B=2)
    tau = wl.uniform_schedule(cfg.n_steps)
    a = O.denoise(cfg, W, cache, inp["noise"], inp["state"], tau)
    b = O.denoise(cfg, W, None, inp["noise"], inp["state"], tau, prefix_hidden=inp["prefix"])
    assert np.array_equal(a, b)


def test_prefix_row_permutation_invariance():
    """The expert attends to every prefix row without a mask or positions,
    so permuting prefix rows leaves the chunk unchanged."""
    cfg = TINY.with_(pattern="joint")
    W, inp, cache = _tiny_setup(cfg)
    tau = wl.uniform_schedule(cfg.n_steps)
    perm = _rng(16).permutation(cfg.prefix_len)
    cache_p = O.prefix_kv_build(cfg, W, inp["prefix"][:, perm])
    a = O.denoise(cfg, W, cache, inp["noise"], inp["state"], tau)
    b = O.denoise(cfg, W, cache_p, inp["noise"], inp["state"], tau)
    np.testing.assert_allclose(a, b, rtol=1e-12, atol=1e-14)


def test_batch_requests_independent():
    W, inp, cache = _tiny_setup(B=3)
    tau = wl.uniform_schedule(TINY.n_steps)
    allb = O.denoise(TINY, W, cache, inp["noise"], inp["state"], tau)
    one = O.denoise(TINY, W, cache, inp["noise"], inp["state"], tau, requests=[1])
    assert np.array_equal(allb[1], one[0])
    assert not np.allclose(allb[0], allb[1])


def test_ternary_expert_runs_and_uses_w2a8():
    """Ternary matrices go through the W2A8 linear: scaling every ternary
    scale by 2 scales every projection by 2 exactly."""
    cfg = TINY.with_(wtype="ternary", head_regression=True, n_steps=1, mlp="relu2glu", pattern="joint")
    W, inp, cache = _tiny_setup(cfg)
    u = wl.random_matrix((3, cfg.d_model), 9)
    y1 = O._lin(cfg, W, "L0.W_q", u)
    W2 = dict(W)
    W2["L0.W_q.scale"] = np.float32(2 * W["L0.W_q.scale"])
    np.testing.assert_allclose(O._lin(cfg, W2, "L0.W_q", u), 2 * y1, rtol=1e-15)
    q, r = O.quantize_int8_rows(u)
    acc = q.astype(np.int64) @ W["L0.W_q"].astype(np.int64).T
    np.testing.assert_allclose(y1, acc * (float(W["L0.W_q.scale"]) * r[:, None].astype(np.float64) / 127),
                               rtol=1e-15)


def test_final_modulation_slot_order():
    """(gamma_f, beta_f) = first and second half of W_fm SiLU(c) + b_fm: with
    W_fm = 0, b_fm = [1...; 0.5...], gated-off layers and W_in = W_s = 0 the
    velocity is (2 x0/rms(x0) + 0.5) W_out^T + b_out with x0 = b_in + b_s + E_pos."""
    cfg = TINY
    W, inp, cache = _tiny_setup(cfg)
    d = cfg.d_model
    W["W_fm"] = np.zeros_like(W["W_fm"])
    W["b_fm"] = np.concatenate([np.ones(d), np.full(d, 0.5)]).astype(np.float32)
    W["W_in"] = np.zeros_like(W["W_in"])
    W["W_s"] = np.zeros_like(W["W_s"])
    for l in range(cfg.n_layers):
        for j in range(cfg.n_sub):
            W[f"L{l}.W_mod"][(3 * j + 2) * d:(3 * j + 3) * d] = 0
            W[f"L{l}.b_mod"][(3 * j + 2) * d:(3 * j + 3) * d] = 0
    x0 = (W["b_in"].astype(np.float64) + W["b_s"] + W["E_pos"])
    rms = np.sqrt(np.mean(x0 * x0, axis=-1, keepdims=True) + cfg.rms_eps)
    expect = (2 * x0 / rms + 0.5) @ W["W_out"].T.astype(np.float64) + W["b_out"]
    v = O.expert_forward(cfg, W, cache[:, :, 0], inp["noise"][0], inp["state"][0], 0.7)
    np.testing.assert_allclose(v, expect, rtol=1e-13)


# --- storage rounding ---------------------------------------------------------------

def test_round_to_bf16_golden():
    """Hand-derived cases (tests/golden/bf16_rounding.txt): float32 first, then
    nearest-even bf16 (catches truncation, ties away from zero, rounding the
    float64 value directly, a lost carry into the exponent, a lost sign)."""
    n = 0
    with open(os.path.join(GOLDEN, "bf16_rounding.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            a, b = line.split()[:2]
            x = float.fromhex(a)
            want = math.inf if b == "inf" else float.fromhex(b)
            got = float(O.round_to_bf16(np.array([x]))[0])
            assert got == want and math.copysign(1.0, got) == math.copysign(1.0, want), (a, got, b)
            n += 1
    assert n >= 15


# --- time-conditioning chain and modulation slots ------------------------------------

def _silu_s(v):
    return v / (1.0 + math.exp(-v))


def _gelu_s(v):
    return 0.5 * v * (1.0 + math.tanh(math.sqrt(2.0 / math.pi) * (v + 0.044715 * v ** 3)))


@pytest.mark.parametrize("case", ["t1_zero", "t1_t2_zero", "identity"])
def test_time_mlp_chain_closed_forms(case):
    """The time MLP c = W_t2 SiLU(W_t1 e + b_t1) + b_t2 and the modulation
    m^l = W_mod^l SiLU(c) + b_mod^l, (gamma_f, beta_f) = W_fm SiLU(c) + b_fm,
    evaluated by scalar loops in three closed forms:
      W_t1 = 0            -> c = W_t2 SiLU(b_t1) + b_t2;
      W_t1 = W_t2 = 0     -> c = b_t2;
      W_t1 = W_t2 = I, b_t1 = b_t2 = 0 -> c = SiLU(e(t)).
    Catches a dropped SiLU (before W_t2 or before W_mod / W_fm), W_t1 and W_t2
    applied in the wrong order, a missing bias, and a time embedding that
    never reaches the chain."""
    cfg = TINY
    W = wl.make_weights(cfg)
    d, t = cfg.d_model, 0.37
    if case in ("t1_zero", "t1_t2_zero"):
        W["W_t1"] = np.zeros_like(W["W_t1"])
    if case == "t1_t2_zero":
        W["W_t2"] = np.zeros_like(W["W_t2"])
    if case == "identity":
        W["W_t1"] = np.eye(d, dtype=np.float32)
        W["W_t2"] = np.eye(d, dtype=np.float32)
        W["b_t1"] = np.zeros(d, np.float32)
        W["b_t2"] = np.zeros(d, np.float32)
    bt1 = [float(v) for v in W["b_t1"]]
    bt2 = [float(v) for v in W["b_t2"]]
    if case == "t1_zero":
        h = [_silu_s(v) for v in bt1]
        c = [a + b for a, b in zip(bf_linear([h], W["W_t2"])[0], bt2)]
    elif case == "t1_t2_zero":
        c = bt2
    else:
        c = [_silu_s(float(v)) for v in O.time_embedding(t, d)]   # e(t) is pinned above
    sc = [_silu_s(v) for v in c]
    mods, (gf, bfin) = O.modulation(cfg, W, t)
    for l in range(cfg.n_layers):
        m = [a + float(b) for a, b in zip(bf_linear([sc], W[f"L{l}.W_mod"])[0], W[f"L{l}.b_mod"])]
        for j in range(cfg.n_sub):
            for s in range(3):
                np.testing.assert_allclose(mods[l][j][s], m[(3 * j + s) * d:(3 * j + s + 1) * d],
                                           rtol=1e-12, atol=1e-15)
    fin = [a + float(b) for a, b in zip(bf_linear([sc], W["W_fm"])[0], W["b_fm"])]
    np.testing.assert_allclose(gf, fin[:d], rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(bfin, fin[d:], rtol=1e-12, atol=1e-15)


def _bf_rows_rms(x, eps):
    return [math.sqrt(sum(v * v for v in row) / len(row) + eps) for row in x]


def _bf_one_sublayer(cfg, W, kind, x0, prefix, alpha):
    """Brute-force velocity of a one-layer expert in which only sublayer `kind`
    is gated on (alpha) with gamma = 1, beta = 0.5, and the final modulation is
    zero: v = (x1 / rms(x1)) W_out^T + b_out, x1 = x0 + alpha * y(u),
    u = 2 x0 / rms(x0) + 0.5."""
    eps, H, G, hd = cfg.rms_eps, cfg.n_heads, cfg.n_kv_heads, cfg.head_dim
    r0 = _bf_rows_rms(x0, eps)
    u = [[2.0 * v / r0[i] + 0.5 for v in row] for i, row in enumerate(x0)]
    if kind == "mlp":
        hid = [[_gelu_s(v) for v in row] for row in bf_linear(u, W["L0.W1"])]
        y = bf_linear(hid, W["L0.W2"])
    else:
        q = bf_linear(u, W["L0.W_q"])

        def heads(rows):
            return [[r[g * hd:(g + 1) * hd] for r in rows] for g in range(G)]
        if kind == "cross":
            k = heads(bf_linear(prefix, W["L0.W_kc"]))
            v = heads(bf_linear(prefix, W["L0.W_vc"]))
        else:
            k = heads(bf_linear(u, W["L0.W_k"]))
            v = heads(bf_linear(u, W["L0.W_v"]))
            if kind == "joint":      # prefix rows first, one softmax
                kc = heads(bf_linear(prefix, W["L0.W_kc"]))
                vc = heads(bf_linear(prefix, W["L0.W_vc"]))
                k = [kc[g] + k[g] for g in range(G)]
                v = [vc[g] + v[g] for g in range(G)]
        o = bf_attention(q, k, v, H, G, hd).tolist()
        y = bf_linear(o, W["L0.W_o"])
    x1 = [[x0[i][c] + float(alpha[c]) * y[i][c] for c in range(len(x0[0]))] for i in range(len(x0))]
    r1 = _bf_rows_rms(x1, eps)
    xn = [[v / r1[i] for v in row] for i, row in enumerate(x1)]
    return np.array(bf_linear(xn, W["W_out"])) + W["b_out"].astype(np.float64)


@pytest.mark.parametrize("pattern,j", [("self_cross", 0), ("self_cross", 1), ("self_cross", 2),
                                       ("joint", 0), ("joint", 1), ("alt", 0), ("alt", 1), ("cross", 0)])
def test_sublayer_slot_order_single_active_sublayer(pattern, j):
    """W_mod = 0 and b_mod = (gamma, beta, alpha) = (1, 0.5, a) in sublayer j
    of the layer, alpha = 0 in every other sublayer, zero final modulation:
    the expert's velocity equals a brute-force evaluation of that one sublayer
    on u = 2 x0 / rms(x0) + 0.5.  Catches gamma and beta (or alpha) swapped
    within a sublayer's slots, one sublayer reading another's slots, and a
    sublayer of another kind run at position j."""
    cfg = TINY.with_(pattern=pattern, n_layers=1)
    W, inp, cache = _tiny_setup(cfg)
    d = cfg.d_model
    W["L0.W_mod"] = np.zeros_like(W["L0.W_mod"])
    bm = np.zeros_like(W["L0.b_mod"])
    bm[(3 * j) * d:(3 * j + 1) * d] = 1.0
    bm[(3 * j + 1) * d:(3 * j + 2) * d] = 0.5
    alpha = _rng(60 + j).uniform(0.5, 1.5, d).astype(np.float32)
    bm[(3 * j + 2) * d:(3 * j + 3) * d] = alpha
    W["L0.b_mod"] = bm
    W["W_fm"] = np.zeros_like(W["W_fm"])
    W["b_fm"] = np.zeros_like(W["b_fm"])
    a, s = inp["noise"][0].astype(np.float64), inp["state"][0].astype(np.float64)
    x0 = [[sum(a[i][k] * float(W["W_in"][c][k]) for k in range(cfg.d_action)) + float(W["b_in"][c]) +
           sum(s[k] * float(W["W_s"][c][k]) for k in range(cfg.d_state)) + float(W["b_s"][c]) +
           float(W["E_pos"][i][c]) for c in range(d)] for i in range(cfg.n_action)]
    prefix = inp["prefix"][0].astype(np.float64).tolist()
    kind = cfg.sublayers(0)[j]
    want = _bf_one_sublayer(cfg, W, kind, x0, prefix, alpha)
    got = O.expert_forward(cfg, W, cache[:, :, 0], a, s, 0.6)
    np.testing.assert_allclose(got, want, rtol=1e-11, atol=1e-13)
    # the gated-on sublayer matters: without it the velocity moves by far more
    # than the tolerance above
    bm[(3 * j + 2) * d:(3 * j + 3) * d] = 0.0
    assert np.abs(O.expert_forward(cfg, W, cache[:, :, 0], a, s, 0.6) - got).max() > 1e-5


# --- the prefix stage: backbone prefill ----------------------------------------------

BB_TINY = wl.BackboneConfig(name="bb_tiny", n_layers=1, d_model=8, n_heads=2, head_dim=4, n_kv_heads=1,
                            d_ff=12, mlp="geglu", wtype="bf16", rope_base=0.0, prefix_len=5, seed_base=91)


def _bf_norm(rows, g, eps):
    r = _bf_rows_rms(rows, eps)
    return [[v / r[i] * (1.0 + float(g[c])) for c, v in enumerate(row)] for i, row in enumerate(rows)]


def _bf_backbone(bcfg, W, x, rotate=False):
    """Brute-force prefill of a one-layer bf16 backbone over rows x: norm,
    bidirectional GQA attention (q, k optionally rotated to positions
    0 .. P-1 by the pinned rope), residual, norm, GeGLU MLP, residual, final
    norm."""
    eps, H, G, hd = bcfg.rms_eps, bcfg.n_heads, bcfg.n_kv_heads, bcfg.head_dim
    P = len(x)
    u = _bf_norm(x, W["B0.g_att"], eps)
    q, k, v = bf_linear(u, W["B0.W_q"]), bf_linear(u, W["B0.W_k"]), bf_linear(u, W["B0.W_v"])
    if rotate:
        q = O.rope(np.array(q), np.arange(P), H, hd, bcfg.rope_base).tolist()
        k = O.rope(np.array(k), np.arange(P), G, hd, bcfg.rope_base).tolist()

    def heads(rows):
        return [[r[g * hd:(g + 1) * hd] for r in rows] for g in range(G)]
    o = bf_attention(q, heads(k), heads(v), H, G, hd).tolist()
    y = bf_linear(o, W["B0.W_o"])
    x1 = [[x[i][c] + y[i][c] for c in range(len(x[0]))] for i in range(P)]
    u2 = _bf_norm(x1, W["B0.g_mlp"], eps)
    gt, up = bf_linear(u2, W["B0.W_g"]), bf_linear(u2, W["B0.W_u"])
    h = [[_gelu_s(gt[i][f]) * up[i][f] for f in range(len(gt[0]))] for i in range(P)]
    y2 = bf_linear(h, W["B0.W_d"])
    x2 = [[x1[i][c] + y2[i][c] for c in range(len(x[0]))] for i in range(P)]
    return np.array(_bf_norm(x2, W["g_f"], eps))


@pytest.mark.parametrize("rotate", [False, True])
def test_prefill_one_layer_bruteforce(rotate):
    """One backbone layer by scalar loops (catches a missing residual, the norm
    gain applied as g instead of 1 + g, a transposed projection, the gate and
    up roles swapped, RoPE applied to the values or at wrong positions)."""
    bcfg = BB_TINY.with_(rope_base=10000.0 if rotate else 0.0)
    W = wl.make_backbone_weights(bcfg)
    e = wl.make_prefix_embeds(bcfg, 2)
    got = O.prefix_prefill(bcfg, W, e)
    for b in range(2):
        want = _bf_backbone(bcfg, W, e[b].astype(np.float64).tolist(), rotate)
        np.testing.assert_allclose(got[b], want, rtol=1e-11, atol=1e-12)


def test_prefill_zero_layers_and_zero_branches_are_the_final_norm():
    """No layers, or every W_o and W_d zero: the prefill returns the final
    norm of the embeddings, x / rms(x) (1 + g_f) (catches an extra term on the
    residual stream)."""
    bcfg = BB_TINY.with_(n_layers=2)
    W = wl.make_backbone_weights(bcfg)
    e = wl.make_prefix_embeds(bcfg, 1)
    want = np.array(_bf_norm(e[0].astype(np.float64).tolist(), W["g_f"], bcfg.rms_eps))
    np.testing.assert_allclose(O.prefix_prefill(bcfg.with_(n_layers=0), W, e)[0], want, rtol=1e-13)
    for l in range(2):
        W[f"B{l}.W_o"] = np.zeros_like(W[f"B{l}.W_o"])
        W[f"B{l}.W_d"] = np.zeros_like(W[f"B{l}.W_d"])
    np.testing.assert_allclose(O.prefix_prefill(bcfg, W, e)[0], want, rtol=1e-13)


def test_prefill_is_bidirectional():
    """Without positions the prefill is permutation-equivariant over the
    prefix rows, and the first row's output depends on the last row's input
    (a causal mask, the failure the paper's bidirectional prefix avoids,
    breaks both)."""
    bcfg = BB_TINY.with_(n_layers=2)
    W = wl.make_backbone_weights(bcfg)
    e = wl.make_prefix_embeds(bcfg, 1)
    perm = _rng(70).permutation(bcfg.prefix_len)
    a = O.prefix_prefill(bcfg, W, e)
    np.testing.assert_allclose(O.prefix_prefill(bcfg, W, e[:, perm]), a[:, perm], rtol=1e-12, atol=1e-13)
    e2 = e.copy()
    e2[0, -1] += 1.0
    assert np.abs(O.prefix_prefill(bcfg, W, e2)[0, 0] - a[0, 0]).max() > 1e-6
    # with RoPE the rows carry positions: permuting them changes the result
    r = bcfg.with_(rope_base=10000.0)
    assert np.abs(O.prefix_prefill(r, W, e[:, perm]) - O.prefix_prefill(r, W, e)[:, perm]).max() > 1e-6


def test_prefill_ternary_projections_use_their_scales():
    """Ternary backbone: with the W_o and W_d scales at 0 every residual
    branch vanishes (each projection is the W2A8 linear times its per-tensor
    scale), leaving the final norm of the embeddings."""
    bcfg = BB_TINY.with_(n_layers=2, wtype="ternary", mlp="relu2glu", d_model=16, d_ff=16)
    W = wl.make_backbone_weights(bcfg)
    e = wl.make_prefix_embeds(bcfg, 1)
    assert W["B0.W_q"].dtype == np.int8 and "B0.W_q.scale" in W
    full = O.prefix_prefill(bcfg, W, e)
    for l in range(2):
        W[f"B{l}.W_o.scale"] = np.float32(0.0)
        W[f"B{l}.W_d.scale"] = np.float32(0.0)
    want = np.array(_bf_norm(e[0].astype(np.float64).tolist(), W["g_f"], bcfg.rms_eps))
    np.testing.assert_allclose(O.prefix_prefill(bcfg, W, e)[0], want, rtol=1e-13)
    assert np.abs(full[0] - want).max() > 1e-4
