"""fp64 CPU oracle of the flow-matching action-expert denoise loop.

TEST INFRASTRUCTURE ONLY.  Only tests/, __graft_entry__.smoke() and the
cpu_baseline leg of bench.py may import this module.  The HIP library never
calls it and shares no code with it.

What it computes follows the paper's canonical inference loop (Sec. 3.3,
Algorithm 1): the prefix hidden states are projected once into a per-layer
cross-attention K/V cache (Appendix A.2, item 3), a0 is the noise chunk, T
solver steps each run the action head over the chunk conditioned on the
cached prefix and the solver time, and the result is denormalised with the
bundle statistics.  The paper gives no equations for the head itself; the
readings taken here (explicit Euler from t=1 to t=0, sinusoidal time
embedding, adaRMS modulation with residual gates, GQA attention without
masks, tanh-GELU, ternary W2A8 linear with per-token absmax int8
activations) are listed with their reasons in the design doc.

Everything is float64 except the int8 activation quantiser, which the method
fixes in IEEE float32 so that a GPU and this oracle reach identical codes
from identical float32 inputs.  Matrix products use numpy's matmul as a
library primitive; nothing is blocked, fused or reordered beyond the
definitions below.

Parity status: every function here is pinned by tests/test_oracle_pins.py
(closed forms, invariants, hand-derived fixtures in tests/golden/, brute
force on tiny inputs).  The full expert forward on random weights has no
closed form: it is pinned through its components, the one-sublayer
brute-force evaluations and the closed-form end-to-end special cases
(zero / constant velocity field, zero residual gates).
"""
from __future__ import annotations

from typing import Callable, Dict, List, Optional

import numpy as np

F64 = np.float64

# Time-embedding periods (geometric from P_MIN to P_MAX).
P_MIN = 4e-3
P_MAX = 4.0
# Floor of the per-token absmax in the int8 activation quantiser.
ABSMAX_FLOOR = np.float32(1e-5)


# --- storage precision ------------------------------------------------------

def round_to_bf16(x):
    """Nearest-even bf16 value of float32(x), as float64 (float32 first, then
    bf16: the value a bf16 store of a float32 result holds).  The expert below
    never calls it; kernel-level tests use it to state what a bf16 store may
    change."""
    f = np.ascontiguousarray(np.asarray(x, dtype=F64).astype(np.float32))
    u = f.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32).astype(F64)


# --- elementwise pieces -----------------------------------------------------

def silu(x):
    """SiLU(x) = x * sigmoid(x)."""
    x = np.asarray(x, dtype=F64)
    return x / (1.0 + np.exp(-x))


def gelu_tanh(x):
    """tanh form of GELU: 0.5 x (1 + tanh(sqrt(2/pi) (x + 0.044715 x^3)))."""
    x = np.asarray(x, dtype=F64)
    return 0.5 * x * (1.0 + np.tanh(np.sqrt(2.0 / np.pi) * (x + 0.044715 * x ** 3)))


def mlp_activation(kind: str, g, u=None):
    """Hidden activation of the expert MLP.

    gelu: GELU(g); geglu: GELU(g)*u; swiglu: SiLU(g)*u; relu2glu: relu(g)^2*u.
    """
    if kind == "gelu":
        return gelu_tanh(g)
    if kind == "geglu":
        return gelu_tanh(g) * u
    if kind == "swiglu":
        return silu(g) * u
    if kind == "relu2glu":
        return np.maximum(np.asarray(g, dtype=F64), 0.0) ** 2 * u
    raise ValueError(kind)


def time_embedding(t: float, d: int) -> np.ndarray:
    """Sinusoidal embedding of the solver time t (width d, d even).

    For j < d/2 the period is p_j = P_MIN * (P_MAX/P_MIN)^(j/(d/2-1));
    e_j = sin(2 pi t / p_j) and e_{j+d/2} = cos(2 pi t / p_j).
    """
    half = d // 2
    frac = np.arange(half, dtype=F64) / max(half - 1, 1)
    period = P_MIN * (P_MAX / P_MIN) ** frac
    ang = 2.0 * np.pi * float(t) / period
    return np.concatenate([np.sin(ang), np.cos(ang)])


def ada_rms(x, gamma, beta, eps):
    """adaRMS: x / sqrt(mean(x^2) + eps) * (1 + gamma) + beta, per row."""
    x = np.asarray(x, dtype=F64)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * (1.0 + np.asarray(gamma, F64)) + np.asarray(beta, F64)


def linear(u, W, b=None):
    """y = u W^T (+ b), with W stored [out][in]."""
    y = np.asarray(u, dtype=F64) @ np.asarray(W, dtype=F64).T
    if b is not None:
        y = y + np.asarray(b, dtype=F64)
    return y


# --- attention ----------------------------------------------------------------

def softmax_rows(s):
    """Max-subtracted softmax over the last axis."""
    s = np.asarray(s, dtype=F64)
    e = np.exp(s - np.max(s, axis=-1, keepdims=True))
    return e / np.sum(e, axis=-1, keepdims=True)


def attention(q, k, v, n_heads: int, n_kv_heads: int, head_dim: int, causal_from=None):
    """Multi-head attention with grouped K/V heads.

    q: [n][H*hd]; k, v: [G][keys][hd].  Head i reads K/V head floor(i*G/H).
    Returns [n][H*hd] with head i in columns i*hd .. i*hd+hd-1.
    Unmasked by default.  causal_from = c (the causal action-token variant):
    keys c, c+1, ... are the n action tokens in order, and query i sees every
    key before c and the action keys c .. c+i; the other scores get weight 0.
    """
    q = np.asarray(q, dtype=F64)
    n = q.shape[0]
    out = np.zeros((n, n_heads * head_dim), dtype=F64)
    scale = 1.0 / np.sqrt(head_dim)
    mask = None
    if causal_from is not None:
        keys = np.asarray(k).shape[1]
        j = np.arange(keys)[None, :]
        i = np.arange(n)[:, None]
        mask = (j >= causal_from) & (j - causal_from > i)
    for i in range(n_heads):
        g = (i * n_kv_heads) // n_heads
        qi = q[:, i * head_dim:(i + 1) * head_dim]
        s = qi @ np.asarray(k[g], F64).T * scale
        if mask is not None:
            s = np.where(mask, -np.inf, s)
        p = softmax_rows(s)
        out[:, i * head_dim:(i + 1) * head_dim] = p @ np.asarray(v[g], F64)
    return out


def rope(x, positions, n_heads: int, head_dim: int, base: float):
    """Rotary position embedding, rotate-half form, of every head of x
    [rows][n_heads*hd]: with h = hd/2 and w_i = base^(-2i/hd), the pair
    (x_i, x_{i+h}) of a row at position p turns by the angle p*w_i:
    x_i' = x_i cos - x_{i+h} sin, x_{i+h}' = x_{i+h} cos + x_i sin."""
    x = np.array(x, dtype=F64)
    half = head_dim // 2
    w = float(base) ** (-2.0 * np.arange(half, dtype=F64) / head_dim)
    ang = np.asarray(positions, dtype=F64)[:, None] * w[None, :]
    c, s = np.cos(ang), np.sin(ang)
    for h in range(n_heads):
        lo = x[:, h * head_dim:h * head_dim + half].copy()
        hi = x[:, h * head_dim + half:(h + 1) * head_dim].copy()
        x[:, h * head_dim:h * head_dim + half] = lo * c - hi * s
        x[:, h * head_dim + half:(h + 1) * head_dim] = hi * c + lo * s
    return x


def split_heads(x, n_kv_heads: int, head_dim: int):
    """[rows][G*hd] -> [G][rows][hd]."""
    x = np.asarray(x, dtype=F64)
    return x.reshape(x.shape[0], n_kv_heads, head_dim).transpose(1, 0, 2)


# --- ternary W2A8 -------------------------------------------------------------

def quantize_int8_rows(u):
    """Per-token absmax int8 quantiser, evaluated in IEEE float32.

    r_m = max(max_k |u_mk|, 1e-5); q_mk = clamp(round_half_even(u_mk * (127/r_m)), -128, 127).
    127/r_m is a correctly rounded float32 divide, the product a float32 multiply.
    Returns (codes int8 [M][K], r float32 [M]).
    """
    u = np.asarray(u, dtype=np.float32)
    r = np.maximum(np.max(np.abs(u), axis=-1), ABSMAX_FLOOR).astype(np.float32)
    inv = (np.float32(127.0) / r).astype(np.float32)
    prod = (u * inv[:, None]).astype(np.float32)
    q = np.clip(np.rint(prod), -128, 127).astype(np.int8)
    return q, r


def unpack_ternary(packed, k: int):
    """Inverse of the 2-bit layout: byte j of row n holds w[n][4j+i] + 1 in bits 2i..2i+1."""
    packed = np.asarray(packed, dtype=np.uint8)
    n = packed.shape[0]
    w = np.zeros((n, k), dtype=np.int64)
    for i in range(4):
        code = (packed >> (2 * i)) & 3
        if np.any(code == 3):
            raise ValueError("invalid ternary code 3")
        w[:, i::4] = code.astype(np.int64) - 1
    return w


def ternary_gemm(x_int8, w_packed, k: int):
    """acc[m][n] = sum_k x[m][k] * w[n][k], exact in int64, checked to fit int32."""
    x = np.asarray(x_int8, dtype=np.int64)
    w = unpack_ternary(w_packed, k)
    acc = x @ w.T
    if acc.size and (acc.max() > np.iinfo(np.int32).max or acc.min() < np.iinfo(np.int32).min):
        raise OverflowError("accumulator exceeds int32")
    return acc


def ternary_linear(u, w_codes, scale):
    """W2A8 linear: int8 activations (float32 quantiser) times ternary weights,
    int64 sum, then y = acc * (s_w * r_m / 127)."""
    q, r = quantize_int8_rows(np.asarray(u, dtype=F64).astype(np.float32))
    # Integer-valued float64 operands: every product and partial sum is an
    # integer below 2^53 in magnitude (|acc| <= 128 * K), so the float64
    # matmul returns the exact integer sum.
    acc = q.astype(F64) @ np.asarray(w_codes, dtype=F64).T
    return acc * (F64(scale) * r.astype(F64)[:, None] / 127.0)


# --- the expert -------------------------------------------------------------------

def _lin(cfg, W, name, u):
    """Projection through a named weight: dense fp64, or W2A8 for ternary matrices."""
    if cfg.wtype == "ternary" and (name + ".scale") in W:
        return ternary_linear(u, W[name], W[name + ".scale"])
    return linear(u, W[name])


def prefix_kv_build(cfg, W: Dict[str, np.ndarray], prefix_hidden) -> np.ndarray:
    """Cross-attention K/V cache from the final-layer prefix hidden states.

    For every layer with a cross or joint sublayer (in layer order):
    Kc = X_p W_kc^T, Vc = X_p W_vc^T, no norm, bias or position encoding (in the
    RoPE variant the joint layers' Kc rows are rotated to positions 0 .. P-1).
    prefix_hidden: [B][P][d_p].  Returns [Lc][2][B][G][P][hd] float64.
    """
    xp = np.asarray(prefix_hidden, dtype=F64)
    B, P = xp.shape[0], xp.shape[1]
    layers = [l for l in range(cfg.n_layers) if cfg.has_prefix(l)]
    cache = np.zeros((len(layers), 2, B, cfg.n_kv_heads, P, cfg.head_dim), dtype=F64)
    base = getattr(cfg, "rope_base", 0.0)
    for c, l in enumerate(layers):
        for b in range(B):
            kc = _lin(cfg, W, f"L{l}.W_kc", xp[b])
            vc = _lin(cfg, W, f"L{l}.W_vc", xp[b])
            if base > 0 and "joint" in cfg.sublayers(l):
                # RoPE variant: prefix rows hold positions 0 .. P-1 of the joint sequence
                kc = rope(kc, np.arange(P), cfg.n_kv_heads, cfg.head_dim, base)
            cache[c, 0, b] = split_heads(kc, cfg.n_kv_heads, cfg.head_dim)
            cache[c, 1, b] = split_heads(vc, cfg.n_kv_heads, cfg.head_dim)
    return cache


def modulation(cfg, W: Dict[str, np.ndarray], t: float):
    """Per-layer (gamma, beta, alpha) for each sublayer and the final (gamma_f, beta_f).

    Time-conditioned heads: e = time_embedding(t); c = W_t2 SiLU(W_t1 e + b_t1) + b_t2;
    m^l = W_mod^l SiLU(c) + b_mod^l split in sublayer order into (gamma, beta, alpha);
    (gamma_f, beta_f) = W_fm SiLU(c) + b_fm.
    The regression head has no time input and reads static tables instead.
    Returns (mods[l][j] = (gamma, beta, alpha), (gamma_f, beta_f)).
    """
    d, ns = cfg.d_model, cfg.n_sub
    if cfg.head_regression:
        rows = [np.asarray(W[f"L{l}.mod"], F64) for l in range(cfg.n_layers)]
        fin = np.asarray(W["mod_f"], F64)
    else:
        e = time_embedding(t, d)
        c = linear(silu(linear(e, W["W_t1"], W["b_t1"])), W["W_t2"], W["b_t2"])
        sc = silu(c)
        rows = [linear(sc, W[f"L{l}.W_mod"], W[f"L{l}.b_mod"]) for l in range(cfg.n_layers)]
        fin = linear(sc, W["W_fm"], W["b_fm"])
    mods = []
    for m in rows:
        mods.append([(m[(3 * j) * d:(3 * j + 1) * d],
                      m[(3 * j + 1) * d:(3 * j + 2) * d],
                      m[(3 * j + 2) * d:(3 * j + 3) * d]) for j in range(ns)])
    return mods, (fin[:d], fin[d:])


def input_embedding(cfg, W, a, s):
    """x = a W_in^T + b_in + (s W_s^T + b_s) on every token + E_pos.

    State-token variant: row 0 is s W_s^T + b_s alone and rows 1 .. n are
    a W_in^T + b_in + E_pos (n + 1 rows)."""
    xs = linear(np.asarray(s, F64)[None, :], W["W_s"], W["b_s"])
    xa = linear(a, W["W_in"], W["b_in"]) + np.asarray(W["E_pos"], F64)
    if getattr(cfg, "state_token", False):
        return np.concatenate([xs, xa], axis=0)
    return xa + xs


def expert_forward(cfg, W, cache_b, a, s, t: float, prefix_b=None) -> np.ndarray:
    """One pass of the action head over the chunk a [n][A]: returns the velocity
    (or, for the regression head, the action chunk) v [n][A].

    cache_b: [Lc][2][G][P][hd] for this request.  If prefix_b is given the
    cross K/V are recomputed from it here instead of being read from cache_b
    (used to check that caching changes nothing).
    Every value between the operations is kept in float64.
    """
    mods, (gf, bf) = modulation(cfg, W, t)
    x = input_embedding(cfg, W, a, s)
    H, G, hd, eps = cfg.n_heads, cfg.n_kv_heads, cfg.head_dim, cfg.rms_eps
    c = 0
    for l in range(cfg.n_layers):
        p = f"L{l}."
        if cfg.has_prefix(l):
            if prefix_b is None:
                kc, vc = cache_b[c, 0], cache_b[c, 1]
            else:
                kc = split_heads(_lin(cfg, W, p + "W_kc", prefix_b), G, hd)
                vc = split_heads(_lin(cfg, W, p + "W_vc", prefix_b), G, hd)
            c += 1
        for j, kind in enumerate(cfg.sublayers(l)):
            gamma, beta, alpha = mods[l][j]
            u = ada_rms(x, gamma, beta, eps)
            if kind == "mlp":
                if cfg.mlp == "gelu":
                    y = _lin(cfg, W, p + "W2", mlp_activation("gelu", _lin(cfg, W, p + "W1", u)))
                else:
                    h = mlp_activation(cfg.mlp, _lin(cfg, W, p + "W_g", u), _lin(cfg, W, p + "W_u", u))
                    y = _lin(cfg, W, p + "W_d", h)
            else:
                q = _lin(cfg, W, p + "W_q", u)
                if kind in ("self", "joint"):
                    k2 = _lin(cfg, W, p + "W_k", u)
                    base = getattr(cfg, "rope_base", 0.0)
                    if base > 0:
                        # RoPE variant: action token i at position i (self) or P + i
                        # (joint, after the prefix rows)
                        pos = np.arange(q.shape[0]) + (kc.shape[1] if kind == "joint" else 0)
                        q = rope(q, pos, H, hd, base)
                        k2 = rope(k2, pos, G, hd, base)
                    ks = split_heads(k2, G, hd)
                    vs = split_heads(_lin(cfg, W, p + "W_v", u), G, hd)
                causal = getattr(cfg, "causal_self", False)
                cfrom = None
                if kind == "self":
                    k_all, v_all = ks, vs
                    cfrom = 0 if causal else None
                elif kind == "cross":
                    k_all, v_all = kc, vc
                else:   # joint: one softmax over [prefix rows ; action rows]
                    k_all = np.concatenate([kc, ks], axis=1)
                    v_all = np.concatenate([vc, vs], axis=1)
                    cfrom = kc.shape[1] if causal else None
                o = attention(q, k_all, v_all, H, G, hd, causal_from=cfrom)
                y = _lin(cfg, W, p + "W_o", o)
            x = x + np.asarray(alpha, F64) * y
    if getattr(cfg, "state_token", False):
        x = x[1:]           # the state token has no action output
    return linear(ada_rms(x, gf, bf, eps), W["W_out"], W["b_out"])


# --- the prefix stage: backbone prefill -------------------------------------------

def backbone_layer(bcfg, Wb, l: int, x):
    """One pre-norm backbone layer over the P prefix rows x [P][d]: the
    attention sublayer, then the MLP sublayer, each added to the residual
    stream.  Attention is bidirectional (every prefix row attends to every
    other, no mask) with grouped K/V heads; with rope_base > 0 the queries and
    keys of row i are rotated to position i.  Norms scale by (1 + g) with the
    layer's learned gains g."""
    p = f"B{l}."
    P = x.shape[0]
    H, G, hd, eps = bcfg.n_heads, bcfg.n_kv_heads, bcfg.head_dim, bcfg.rms_eps
    u = ada_rms(x, Wb[p + "g_att"], 0.0, eps)
    q = _lin(bcfg, Wb, p + "W_q", u)
    k = _lin(bcfg, Wb, p + "W_k", u)
    v = _lin(bcfg, Wb, p + "W_v", u)
    if bcfg.rope_base > 0:
        q = rope(q, np.arange(P), H, hd, bcfg.rope_base)
        k = rope(k, np.arange(P), G, hd, bcfg.rope_base)
    o = attention(q, split_heads(k, G, hd), split_heads(v, G, hd), H, G, hd)
    x = x + _lin(bcfg, Wb, p + "W_o", o)
    u = ada_rms(x, Wb[p + "g_mlp"], 0.0, eps)
    if bcfg.mlp == "gelu":
        y = _lin(bcfg, Wb, p + "W2", mlp_activation("gelu", _lin(bcfg, Wb, p + "W1", u)))
    else:
        h = mlp_activation(bcfg.mlp, _lin(bcfg, Wb, p + "W_g", u), _lin(bcfg, Wb, p + "W_u", u))
        y = _lin(bcfg, Wb, p + "W_d", h)
    return x + y


def prefix_prefill(bcfg, Wb, embeds) -> np.ndarray:
    """The prefix stage (Algorithm 1, h = VLM-Prefix(...), bidirectional): the
    prefix token embeddings [B][P][d] pass through every backbone layer, and
    the final-layer hidden states, after the final norm (the tensor a language
    model feeds its output projection), are returned [B][P][d] in float64.
    They are the cross-attention source of prefix_kv_build."""
    e = np.asarray(embeds, dtype=F64)
    out = np.zeros_like(e)
    for b in range(e.shape[0]):
        x = e[b]
        for l in range(bcfg.n_layers):
            x = backbone_layer(bcfg, Wb, l, x)
        out[b] = ada_rms(x, Wb["g_f"], 0.0, bcfg.rms_eps)
    return out


def euler_integrate(velocity: Callable[[np.ndarray, int, float], np.ndarray], a0, tau) -> np.ndarray:
    """Explicit Euler from tau_0 to tau_T: a_{k+1} = a_k + (tau_{k+1} - tau_k) v(a_k, k, tau_k)."""
    a = np.asarray(a0, dtype=F64).copy()
    tau = np.asarray(tau, dtype=F64)
    for k in range(len(tau) - 1):
        a = a + (tau[k + 1] - tau[k]) * velocity(a, k, float(tau[k]))
    return a


def denormalize(a, mean=None, std=None):
    """a * std + mean per action dim (identity when the statistics are absent)."""
    a = np.asarray(a, dtype=F64)
    if std is not None:
        a = a * np.asarray(std, F64)
    if mean is not None:
        a = a + np.asarray(mean, F64)
    return a


def denoise(cfg, W, cache, noise, state, tau, act_mean=None, act_std=None,
            prefix_hidden=None, requests: Optional[List[int]] = None) -> np.ndarray:
    """The whole chunk for every request: Euler over T solver steps (the
    regression head takes one pass and returns its output), then denormalise.

    cache [Lc][2][B][G][P][hd]; noise [B][n][A]; state [B][S]; tau [T+1].
    With prefix_hidden given, cross K/V are recomputed at every step instead of
    read from the cache.  requests restricts the evaluation to some of the B.
    """
    noise = np.asarray(noise, F64)
    B = noise.shape[0]
    reqs = range(B) if requests is None else requests
    out = np.zeros((len(reqs),) + noise.shape[1:], dtype=F64)
    for i, b in enumerate(reqs):
        cb = None if cache is None else np.asarray(cache)[:, :, b]
        pb = None if prefix_hidden is None else np.asarray(prefix_hidden, F64)[b]

        def vel(a, k, t, cb=cb, pb=pb, b=b):
            return expert_forward(cfg, W, cb, a, state[b], t, prefix_b=pb)

        if cfg.head_regression:
            a = vel(noise[b], 0, float(tau[0]))
        else:
            a = euler_integrate(vel, noise[b], tau)
        out[i] = denormalize(a, act_mean, act_std)
    return out
