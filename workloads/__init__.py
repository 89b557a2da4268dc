"""Seeded synthetic workloads for the action-expert denoise loop.

This module is the only code shared by the HIP path's callers (tests, bench,
smoke) and the CPU oracle.  It holds configuration records and seeded input
generators only: shapes, random draws, bf16 rounding of the drawn values and
the 2-bit packing of ternary codes.  None of the method's arithmetic lives here.

The five workloads stand in for the paper's deployment shapes (the pi0,
SmolVLA and BitVLA rows of the served-architecture table, Appendix A); the
paper's LIBERO suites and trained checkpoints are not used.  Every weight and
bias is N(0, 0.02^2), prefix hidden states and noise are N(0, 1) (the
diffusion-style GR00T-shaped head starts from U(-1, 1) noise instead), the
proprioceptive state is U(-1, 1) and the solver schedule is uniform from
t = 1 down to t = 0.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List

import numpy as np

PATTERNS = ("self_cross", "joint", "alt")
MLPS = ("gelu", "geglu", "swiglu", "relu2glu")
WTYPES = ("f32", "bf16", "ternary")


@dataclasses.dataclass(frozen=True)
class ExpertConfig:
    """Architecture of the action expert plus the workload it runs on."""
    name: str
    n_layers: int
    d_model: int
    n_heads: int
    head_dim: int
    n_kv_heads: int
    d_ff: int
    d_prefix: int
    n_action: int          # chunk length n (action tokens)
    d_action: int          # action dim A
    d_state: int           # proprio state dim S
    pattern: str           # "self_cross" | "joint" | "alt" | "cross"
    mlp: str               # "gelu" | "geglu" | "swiglu" | "relu2glu"
    wtype: str             # "f32" | "bf16" | "ternary"
    head_regression: bool = False
    # variant: action token i attends only to action tokens j <= i in self and
    # joint attention (every prefix row stays visible); default bidirectional
    causal_self: bool = False
    # variant: rotary position embedding (rotate-half form, this base; 0 = none)
    # on the queries and keys of self and joint attention
    rope_base: float = 0.0
    # variant: the state enters as its own token ahead of the n action tokens
    # (pi0-style) instead of being added to every action token
    state_token: bool = False
    # the chunk's starting draw a_0: "normal" N(0, I) for flow-matching heads,
    # "uniform" U(-1, 1) per element for the diffusion head (Algorithm 1)
    start: str = "normal"
    rms_eps: float = 1e-6
    # workload
    prefix_len: int = 64
    n_steps: int = 4
    batch: int = 1
    seed_base: int = 1000

    @property
    def d_q(self) -> int:
        return self.n_heads * self.head_dim

    @property
    def d_kv(self) -> int:
        return self.n_kv_heads * self.head_dim

    def sublayers(self, layer: int) -> List[str]:
        """Sublayer kinds of one layer, in execution order."""
        if self.pattern == "self_cross":
            return ["self", "cross", "mlp"]
        if self.pattern == "joint":
            return ["joint", "mlp"]
        if self.pattern == "alt":
            return ["cross", "mlp"] if layer % 2 == 0 else ["self", "mlp"]
        if self.pattern == "cross":
            return ["cross", "mlp"]
        raise ValueError(self.pattern)

    @property
    def n_sub(self) -> int:
        return len(self.sublayers(0))

    def has_prefix(self, layer: int) -> bool:
        return any(k in ("cross", "joint") for k in self.sublayers(layer))

    def has_self_kv(self, layer: int) -> bool:
        return any(k in ("self", "joint") for k in self.sublayers(layer))

    @property
    def n_cache_layers(self) -> int:
        return sum(self.has_prefix(l) for l in range(self.n_layers))

    def with_(self, **kw) -> "ExpertConfig":
        return dataclasses.replace(self, **kw)


# --- the five workloads -----------------------------------------------------

TINY_F32 = ExpertConfig(
    name="tiny_f32", n_layers=2, d_model=256, n_heads=4, head_dim=64, n_kv_heads=1,
    d_ff=1024, d_prefix=256, n_action=8, d_action=7, d_state=7,
    pattern="self_cross", mlp="gelu", wtype="f32",
    prefix_len=64, n_steps=4, seed_base=1000)

PI0_BF16 = ExpertConfig(
    name="pi0_bf16", n_layers=18, d_model=1024, n_heads=8, head_dim=256, n_kv_heads=1,
    d_ff=4096, d_prefix=2048, n_action=50, d_action=32, d_state=32,
    pattern="joint", mlp="geglu", wtype="bf16",
    prefix_len=816, n_steps=10, seed_base=2000)

SMOLVLA_BF16 = ExpertConfig(
    name="smolvla_bf16", n_layers=16, d_model=720, n_heads=15, head_dim=64, n_kv_heads=5,
    d_ff=2048, d_prefix=960, n_action=50, d_action=6, d_state=6,
    pattern="alt", mlp="swiglu", wtype="bf16",
    prefix_len=241, n_steps=10, seed_base=3000)

TERNARY_W2A8 = ExpertConfig(
    name="ternary_w2a8", n_layers=24, d_model=2560, n_heads=20, head_dim=128, n_kv_heads=5,
    d_ff=6912, d_prefix=2560, n_action=8, d_action=7, d_state=7,
    pattern="joint", mlp="relu2glu", wtype="ternary", head_regression=True,
    prefix_len=512, n_steps=1, seed_base=4000)

STRESS_PI0 = PI0_BF16.with_(name="stress_pi0", n_action=100, prefix_len=2048, n_steps=20,
                            seed_base=5000)

# DiT-style heads (the paper's Table of served architectures gives their layer pattern, solver
# steps and chunk length; widths are not given and are stand-ins of the same order):
#   GR00T-series alternating DiT: cross-attention to the VL prefix and self-attention in turn,
#   T = 4, 16 action tokens, multi-head attention, GELU MLP;
#   Evo-1 cross-attention DiT: cross-attention in every layer, T = 32, 8 action tokens.
GR00T_ALT_BF16 = ExpertConfig(
    name="gr00t_alt_bf16", n_layers=32, d_model=1024, n_heads=16, head_dim=64, n_kv_heads=16,
    d_ff=4096, d_prefix=2048, n_action=16, d_action=32, d_state=32,
    pattern="alt", mlp="gelu", wtype="bf16", start="uniform",
    prefix_len=200, n_steps=4, seed_base=6000)

EVO1_CROSS_BF16 = ExpertConfig(
    name="evo1_cross_bf16", n_layers=8, d_model=896, n_heads=14, head_dim=64, n_kv_heads=2,
    d_ff=3584, d_prefix=896, n_action=8, d_action=7, d_state=8,
    pattern="cross", mlp="swiglu", wtype="bf16",
    prefix_len=256, n_steps=32, seed_base=7000)

CONFIGS: Dict[str, ExpertConfig] = {
    c.name: c for c in (TINY_F32, PI0_BF16, SMOLVLA_BF16, TERNARY_W2A8, STRESS_PI0, GR00T_ALT_BF16,
                        EVO1_CROSS_BF16)}

# Prefix segment structure of the pi0-shaped workloads (camera patches + text).
# The expert attends to every prefix row, so the segments do not change the
# computation; rows are drawn i.i.d.
PREFIX_SEGMENTS = {"pi0_bf16": [256, 256, 256, 48],
                   "stress_pi0": [320] * 6 + [128]}

TERNARY_P0 = 0.33                      # probability of a zero weight
TERNARY_SCALE = np.float32(0.02 / np.sqrt(0.67))   # effective weight std 0.02


# --- value helpers (input preparation only) --------------------------------

def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bf16 (ties to even); returns float32."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    r = (u + np.uint32(0x7FFF) + lsb) & np.uint32(0xFFFF0000)   # finite inputs: no wrap
    return r.view(np.float32)


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """uint16 bit patterns of float32 values that are already bf16-representable."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    if np.any(u & 0xFFFF):
        raise ValueError("values are not bf16-representable")
    return (u >> 16).astype(np.uint16)


def pack_ternary(codes: np.ndarray) -> np.ndarray:
    """Pack ternary weights w in {-1,0,+1}, shape [N][K] (K % 4 == 0), into
    bytes [N][K/4]: byte j of row n holds the 2-bit code w[n][4j+i] + 1 in bits
    2i..2i+1.  Code 3 never occurs."""
    codes = np.asarray(codes, dtype=np.int64)
    n, k = codes.shape
    if k % 4:
        raise ValueError("K must be a multiple of 4")
    c = (codes + 1).astype(np.uint8).reshape(n, k // 4, 4)
    return (c[..., 0] | (c[..., 1] << 2) | (c[..., 2] << 4) | (c[..., 3] << 6)).astype(np.uint8)


def uniform_schedule(n_steps: int) -> np.ndarray:
    """tau_k = 1 - k/T, k = 0..T, as float32."""
    return (1.0 - np.arange(n_steps + 1, dtype=np.float64) / n_steps).astype(np.float32)


# --- seeded generation ------------------------------------------------------

def _normal(rng, shape, std):
    return (rng.standard_normal(size=shape) * std).astype(np.float32)


def _wcast(cfg: ExpertConfig, x: np.ndarray) -> np.ndarray:
    return x if cfg.wtype == "f32" else round_bf16(x)


def _ternary(rng, shape):
    u = rng.random(size=shape)
    w = np.zeros(shape, dtype=np.int8)
    p_pm = (1.0 - TERNARY_P0) / 2.0
    w[u < p_pm] = -1
    w[(u >= p_pm) & (u < 2 * p_pm)] = 1
    return w


def weight_names(cfg: ExpertConfig) -> List[str]:
    """Every weight/bias name in the order of the C-ABI weight table."""
    names = ["W_in", "b_in", "W_s", "b_s", "E_pos"]
    if cfg.head_regression:
        names += ["mod_f"]
    else:
        names += ["W_t1", "b_t1", "W_t2", "b_t2", "W_fm", "b_fm"]
    names += ["W_out", "b_out"]
    for l in range(cfg.n_layers):
        p = f"L{l}."
        names += [p + "mod"] if cfg.head_regression else [p + "W_mod", p + "b_mod"]
        for kind in cfg.sublayers(l):
            if kind == "mlp":
                mats = ["W1", "W2"] if cfg.mlp == "gelu" else ["W_g", "W_u", "W_d"]
                names += [p + m for m in mats]
            else:
                names += [p + "W_q"]
                if kind in ("self", "joint"):
                    names += [p + "W_k", p + "W_v"]
                if kind in ("cross", "joint"):
                    names += [p + "W_kc", p + "W_vc"]
                names += [p + "W_o"]
    return names


def weight_shape(cfg: ExpertConfig, name: str):
    d, A, S, n = cfg.d_model, cfg.d_action, cfg.d_state, cfg.n_action
    short = name.split(".")[-1]
    table = {
        "W_in": (d, A), "b_in": (d,), "W_s": (d, S), "b_s": (d,), "E_pos": (n, d),
        "W_t1": (d, d), "b_t1": (d,), "W_t2": (d, d), "b_t2": (d,),
        "W_fm": (2 * d, d), "b_fm": (2 * d,), "mod_f": (2 * d,),
        "W_out": (A, d), "b_out": (A,),
        "W_mod": (3 * cfg.n_sub * d, d), "b_mod": (3 * cfg.n_sub * d,), "mod": (3 * cfg.n_sub * d,),
        "W_q": (cfg.d_q, d), "W_k": (cfg.d_kv, d), "W_v": (cfg.d_kv, d),
        "W_kc": (cfg.d_kv, cfg.d_prefix), "W_vc": (cfg.d_kv, cfg.d_prefix),
        "W_o": (d, cfg.d_q),
        "W1": (cfg.d_ff, d), "W2": (d, cfg.d_ff),
        "W_g": (cfg.d_ff, d), "W_u": (cfg.d_ff, d), "W_d": (d, cfg.d_ff),
    }
    return table[short]


TERNARY_MATS = ("W_q", "W_k", "W_v", "W_kc", "W_vc", "W_o", "W_g", "W_u", "W_d", "W1", "W2")


def is_ternary_matrix(cfg: ExpertConfig, name: str) -> bool:
    return cfg.wtype == "ternary" and name.split(".")[-1] in TERNARY_MATS


def make_weights(cfg: ExpertConfig, seed: int | None = None) -> Dict[str, np.ndarray]:
    """Seeded random-init weights.

    Dense matrices are float32 arrays (bf16-representable unless wtype is f32).
    Ternary matrices are int8 codes in {-1,0,+1} under the name itself plus a
    float32 scalar under name + ".scale".  Biases and the static modulation
    tables of regression mode are float32.
    """
    rng = np.random.default_rng(cfg.seed_base + 1 if seed is None else seed)
    out: Dict[str, np.ndarray] = {}
    for name in weight_names(cfg):
        shape = weight_shape(cfg, name)
        short = name.split(".")[-1]
        if is_ternary_matrix(cfg, name):
            out[name] = _ternary(rng, shape)
            out[name + ".scale"] = np.float32(TERNARY_SCALE)
        elif short.startswith("b_") or short in ("mod", "mod_f"):
            out[name] = _normal(rng, shape, 0.02)
        else:
            out[name] = _wcast(cfg, _normal(rng, shape, 0.02))
    return out


def make_inputs(cfg: ExpertConfig, request: int = 0) -> Dict[str, np.ndarray]:
    """Seeded per-request inputs: prefix hidden states, noise and state.

    Request r of a batch adds 10*r to each seed.  bf16 and ternary workloads
    carry bf16-representable prefix hidden states.
    """
    sb = cfg.seed_base + 10 * request
    rp = np.random.default_rng(sb + 2)
    rn = np.random.default_rng(sb + 3)
    rs = np.random.default_rng(sb + 4)
    prefix = rp.standard_normal(size=(cfg.prefix_len, cfg.d_prefix)).astype(np.float32)
    if cfg.wtype != "f32":
        prefix = round_bf16(prefix)
    if cfg.start == "uniform":
        noise = rn.uniform(-1.0, 1.0, size=(cfg.n_action, cfg.d_action)).astype(np.float32)
    else:
        noise = rn.standard_normal(size=(cfg.n_action, cfg.d_action)).astype(np.float32)
    if cfg.head_regression:
        noise[:] = 0.0      # the single-pass regression head has no noise input
    state = rs.uniform(-1.0, 1.0, size=(cfg.d_state,)).astype(np.float32)
    return {"prefix": prefix, "noise": noise, "state": state}


def make_batch(cfg: ExpertConfig, batch: int | None = None) -> Dict[str, np.ndarray]:
    """Stack make_inputs over requests 0..B-1 along a leading batch axis."""
    b = cfg.batch if batch is None else batch
    reqs = [make_inputs(cfg, r) for r in range(b)]
    return {k: np.stack([r[k] for r in reqs]) for k in reqs[0]}


def random_matrix(shape, seed: int, std: float = 1.0, bf16: bool = False) -> np.ndarray:
    """A seeded N(0, std^2) float32 array, optionally rounded to bf16."""
    x = _normal(np.random.default_rng(seed), shape, std)
    return round_bf16(x) if bf16 else x


def random_ternary(shape, seed: int) -> np.ndarray:
    return _ternary(np.random.default_rng(seed), shape)


def random_int8(shape, seed: int) -> np.ndarray:
    return np.random.default_rng(seed).integers(-128, 128, size=shape, dtype=np.int64).astype(np.int8)


# --- the vision-language backbone of the prefix (prefill) ---------------------

@dataclasses.dataclass(frozen=True)
class BackboneConfig:
    """Language-model backbone that encodes the prefix tokens in one
    bidirectional pass (the prefix stage of the paper's inference loop), plus
    the workload it runs on."""
    name: str
    n_layers: int
    d_model: int
    n_heads: int
    head_dim: int
    n_kv_heads: int
    d_ff: int
    mlp: str               # "gelu" | "geglu" | "swiglu" | "relu2glu"
    wtype: str             # "bf16" | "ternary"
    rope_base: float = 10000.0   # rotary position embedding of q and k (0 = none)
    rms_eps: float = 1e-6
    prefix_len: int = 512
    batch: int = 1
    seed_base: int = 8000

    @property
    def d_q(self) -> int:
        return self.n_heads * self.head_dim

    @property
    def d_kv(self) -> int:
        return self.n_kv_heads * self.head_dim

    def with_(self, **kw) -> "BackboneConfig":
        return dataclasses.replace(self, **kw)


# Gemma-2B-shaped bf16 backbone of the pi0-shaped workload (its 816 prefix
# tokens: 3 x 256 image patches + 48 text tokens); width 2048 is the expert's d_p.
PI0_VLM_BF16 = BackboneConfig(
    name="pi0_vlm_bf16", n_layers=18, d_model=2048, n_heads=8, head_dim=256, n_kv_heads=1,
    d_ff=16384, mlp="geglu", wtype="bf16", prefix_len=816, seed_base=8000)

# BitNet-2B-shaped ternary backbone of the BitVLA-shaped workload: the paper's
# 30-layer one-shot prefill, at the ternary expert's widths, over its 512-token prefix.
BITNET_W2A8 = BackboneConfig(
    name="bitnet_w2a8", n_layers=30, d_model=2560, n_heads=20, head_dim=128, n_kv_heads=5,
    d_ff=6912, mlp="relu2glu", wtype="ternary", prefix_len=512, seed_base=9000)

BACKBONES: Dict[str, BackboneConfig] = {c.name: c for c in (PI0_VLM_BF16, BITNET_W2A8)}


def backbone_weight_names(bcfg: BackboneConfig) -> List[str]:
    """Backbone weight names in the order of the C-ABI weight table."""
    names = ["g_f"]
    mats = ["W1", "W2"] if bcfg.mlp == "gelu" else ["W_g", "W_u", "W_d"]
    for l in range(bcfg.n_layers):
        p = f"B{l}."
        names += [p + "g_att", p + "W_q", p + "W_k", p + "W_v", p + "W_o", p + "g_mlp"] + [p + m for m in mats]
    return names


def backbone_weight_shape(bcfg: BackboneConfig, name: str):
    d, F = bcfg.d_model, bcfg.d_ff
    return {"g_f": (d,), "g_att": (d,), "g_mlp": (d,),
            "W_q": (bcfg.d_q, d), "W_k": (bcfg.d_kv, d), "W_v": (bcfg.d_kv, d), "W_o": (d, bcfg.d_q),
            "W1": (F, d), "W2": (d, F), "W_g": (F, d), "W_u": (F, d), "W_d": (d, F)}[name.split(".")[-1]]


def is_backbone_ternary(bcfg: BackboneConfig, name: str) -> bool:
    return bcfg.wtype == "ternary" and name.split(".")[-1] in TERNARY_MATS


def make_backbone_weights(bcfg: BackboneConfig, seed: int | None = None) -> Dict[str, np.ndarray]:
    """Seeded random-init backbone weights: norm gains g N(0, 0.02^2) (the
    norm scales by 1 + g), matrices N(0, 0.02^2) rounded to bf16, or ternary
    codes with the per-tensor scale under name + ".scale"."""
    rng = np.random.default_rng(bcfg.seed_base + 1 if seed is None else seed)
    out: Dict[str, np.ndarray] = {}
    for name in backbone_weight_names(bcfg):
        shape = backbone_weight_shape(bcfg, name)
        if is_backbone_ternary(bcfg, name):
            out[name] = _ternary(rng, shape)
            out[name + ".scale"] = np.float32(TERNARY_SCALE)
        else:
            # float32 draws: the Gemma-shaped backbone has two billion weights
            x = rng.standard_normal(size=shape, dtype=np.float32) * np.float32(0.02)
            out[name] = x if len(shape) == 1 else round_bf16(x)
    return out


def make_prefix_embeds(bcfg: BackboneConfig, batch: int | None = None) -> np.ndarray:
    """Seeded prefix token embeddings [B][P][d], N(0, 1) rounded to bf16: the
    stand-in for the vision encoder's patch tokens and the text embeddings.
    Request r draws from seed_base + 2 + 10 r."""
    b = bcfg.batch if batch is None else batch
    rows = [np.random.default_rng(bcfg.seed_base + 2 + 10 * r).standard_normal(
        size=(bcfg.prefix_len, bcfg.d_model)).astype(np.float32) for r in range(b)]
    return round_bf16(np.stack(rows))
