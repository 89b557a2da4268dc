"""ctypes binding of libvla (include/vla.h, include/vla_test.h).

Argument marshalling only: every step of the denoise loop runs in the HIP
library.  Device buffers are passed as torch tensors (their data pointers) or
as raw integer addresses; streams as torch.cuda.Stream, an integer handle, or
None for torch's current stream.  If libvla.so is missing or fails to load,
every call raises: there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, List, Optional, Sequence

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libvla.so")

PATTERNS = {"self_cross": 0, "joint": 1, "alt": 2, "cross": 3}
MLPS = {"gelu": 0, "geglu": 1, "swiglu": 2, "relu2glu": 3}
WTYPES = {"f32": 0, "bf16": 1, "ternary": 2}
STATUS = {0: "VLA_OK", 1: "VLA_E_ARG", 2: "VLA_E_SHAPE", 3: "VLA_E_UNSUPPORTED", 4: "VLA_E_NOMEM",
          5: "VLA_E_DEVICE", 6: "VLA_E_NONFINITE"}
VLA_OPT_LOOP_MODE = 0
VLA_OPT_PROFILE = 1
VLA_OPT_TRACE = 2
VLA_OPT_ATTN_SPLITS = 3
VLA_OPT_CAUSAL_SELF = 4
VLA_OPT_ROPE_BASE = 5
VLA_OPT_STATE_TOKEN = 6
VLA_OPT_PERSIST_SPIN_LIMIT = 7
PERSIST_TRACE_MAX = 8192
OP_KINDS = {0: "gemm", 1: "gemm_glu", 2: "attention", 3: "ternary_gemm", 4: "quantize", 5: "small",
            6: "attn_merge", 7: "persist"}

# Every symbol the headers declare.
EXPORTS = ["vla_weight_count", "vla_model_create", "vla_model_destroy", "vla_model_check", "vla_kv_cache_bytes",
           "vla_prefix_kv_build", "vla_prefix_kv_build_noalloc", "vla_denoise", "vla_ternary_gemm", "vla_model_set_option",
           "vla_last_error", "vla_status_string", "vla_profile_read",
           "vla_test_gemm", "vla_test_attention", "vla_test_quantize_i8", "vla_test_quantize_bf16", "vla_test_ternary_linear",
           "vla_test_ternary_gemm", "vla_test_rope",
           "vla_test_adarms", "vla_test_time_cond", "vla_test_persist_trace",
           "vla_backbone_weight_count", "vla_backbone_create", "vla_backbone_destroy", "vla_prefix_prefill"]


class VlaError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS.get(status, status)}: {msg}")
        self.status = status


class VlaConfig(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "n_layers", "d_model", "n_heads", "head_dim", "n_kv_heads", "d_ff", "d_prefix",
        "n_action", "d_action", "d_state", "pattern", "mlp", "wtype", "head_regression")] + [
        ("rms_eps", ctypes.c_float)]


class VlaBackboneConfig(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "n_layers", "d_model", "n_heads", "head_dim", "n_kv_heads", "d_ff", "mlp", "wtype")] + [
        ("rope_base", ctypes.c_float), ("rms_eps", ctypes.c_float)]


class VlaOpTime(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("M", ctypes.c_int32), ("N", ctypes.c_int32), ("K", ctypes.c_int32),
                ("bytes", ctypes.c_double), ("flops", ctypes.c_double), ("ms", ctypes.c_float)]


_lib = None


def lib():
    """Load libvla.so once; raise if it is absent."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with python -m paper_2606_08094_amd.build")
    L = ctypes.CDLL(LIB_PATH)
    vp, i32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
    sig = {
        "vla_weight_count": (i32, [ctypes.POINTER(VlaConfig)]),
        "vla_model_create": (i32, [ctypes.POINTER(VlaConfig), ctypes.POINTER(vp), i32, ctypes.POINTER(vp)]),
        "vla_model_destroy": (None, [vp]),
        "vla_model_check": (i32, [vp, vp]),
        "vla_kv_cache_bytes": (sz, [vp, i32, i32]),
        "vla_prefix_kv_build": (i32, [vp, vp, i32, i32, vp, sz, vp]),
        "vla_prefix_kv_build_noalloc": (i32, [vp, vp, i32, i32, vp, sz, vp]),
        "vla_denoise": (i32, [vp, vp, sz, i32, i32, vp, vp, ctypes.POINTER(ctypes.c_float), i32, vp, vp, vp, vp]),
        "vla_ternary_gemm": (i32, [vp, vp, i32, i32, i32, vp, vp]),
        "vla_model_set_option": (i32, [vp, i32, i32]),
        "vla_last_error": (ctypes.c_char_p, []),
        "vla_status_string": (ctypes.c_char_p, [i32]),
        "vla_profile_read": (i32, [vp, ctypes.POINTER(VlaOpTime), i32]),
        "vla_test_gemm": (i32, [i32, vp, vp, i32, i32, i32, i32, vp, vp]),
        "vla_test_attention": (i32, [i32, i32, vp, vp, vp, vp, vp, i32, i32, i32, i32, i32, i32, i32, vp, vp]),
        "vla_test_quantize_i8": (i32, [vp, i32, i32, vp, vp, vp]),
        "vla_test_quantize_bf16": (i32, [vp, i32, i32, i32, vp, vp, vp]),
        "vla_test_adarms": (i32, [i32, vp, vp, i32, vp, vp, vp, i32, i32, ctypes.c_float, vp, i32, vp]),
        "vla_test_time_cond": (i32, [vp, ctypes.POINTER(ctypes.c_float), i32, vp, vp, vp]),
        "vla_test_ternary_linear": (i32, [vp, vp, i32, i32, i32, ctypes.c_float, vp, vp]),
        "vla_test_rope": (i32, [i32, vp, i32, i32, i32, i32, i32, i32, i32, ctypes.c_float, vp]),
        "vla_test_ternary_gemm": (i32, [vp, vp, vp, vp, i32, i32, i32, i32, i32, vp,
                                        ctypes.POINTER(ctypes.c_float), vp]),
        "vla_test_persist_trace": (i32, [vp, ctypes.POINTER(ctypes.c_uint64), i32]),
        "vla_backbone_weight_count": (i32, [ctypes.POINTER(VlaBackboneConfig)]),
        "vla_backbone_create": (i32, [ctypes.POINTER(VlaBackboneConfig), ctypes.POINTER(vp), i32,
                                      ctypes.POINTER(vp)]),
        "vla_backbone_destroy": (None, [vp]),
        "vla_prefix_prefill": (i32, [vp, vp, i32, i32, vp, vp]),
    }
    for name, (res, args) in sig.items():
        f = getattr(L, name)
        f.restype = res
        f.argtypes = args
    _lib = L
    return L


def _check(status: int):
    if status != 0:
        raise VlaError(status, lib().vla_last_error().decode())


def _ptr(x) -> Optional[int]:
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(s) -> Optional[int]:
    if s is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(s, int):
        return s
    return s.cuda_stream


def make_config(cfg) -> VlaConfig:
    """vla_config from any object with the expert's attributes (string enums)."""
    return VlaConfig(
        n_layers=cfg.n_layers, d_model=cfg.d_model, n_heads=cfg.n_heads, head_dim=cfg.head_dim,
        n_kv_heads=cfg.n_kv_heads, d_ff=cfg.d_ff, d_prefix=cfg.d_prefix, n_action=cfg.n_action,
        d_action=cfg.d_action, d_state=cfg.d_state, pattern=PATTERNS[cfg.pattern], mlp=MLPS[cfg.mlp],
        wtype=WTYPES[cfg.wtype], head_regression=int(bool(cfg.head_regression)), rms_eps=float(cfg.rms_eps))


def weight_order(cfg) -> List[str]:
    """Names of the weight-table entries in the order vla.h documents.
    Ternary matrices are followed by '<name>.scale'."""
    tern = cfg.wtype == "ternary"

    def mat(name):
        return [name, name + ".scale"] if tern else [name]

    names = ["W_in", "b_in", "W_s", "b_s", "E_pos"]
    names += ["mod_f"] if cfg.head_regression else ["W_t1", "b_t1", "W_t2", "b_t2", "W_fm", "b_fm"]
    names += ["W_out", "b_out"]
    for l in range(cfg.n_layers):
        p = f"L{l}."
        names += [p + "mod"] if cfg.head_regression else [p + "W_mod", p + "b_mod"]
        if cfg.pattern == "self_cross":
            kinds = ["self", "cross", "mlp"]
        elif cfg.pattern == "joint":
            kinds = ["joint", "mlp"]
        elif cfg.pattern == "cross":
            kinds = ["cross", "mlp"]
        else:
            kinds = ["cross", "mlp"] if l % 2 == 0 else ["self", "mlp"]
        for k in kinds:
            if k == "mlp":
                for w in (["W1", "W2"] if cfg.mlp == "gelu" else ["W_g", "W_u", "W_d"]):
                    names += mat(p + w)
            else:
                names += mat(p + "W_q")
                if k in ("self", "joint"):
                    names += mat(p + "W_k") + mat(p + "W_v")
                if k in ("cross", "joint"):
                    names += mat(p + "W_kc") + mat(p + "W_vc")
                names += mat(p + "W_o")
    return names


class Model:
    """A vla_model created from device tensors keyed by weight-table name."""

    def __init__(self, cfg, device_weights: Dict[str, object]):
        self.cfg = cfg
        self._c = make_config(cfg)
        names = weight_order(cfg)
        want = lib().vla_weight_count(ctypes.byref(self._c))
        if want != len(names):
            raise VlaError(1, f"weight table length mismatch ({want} vs {len(names)})")
        table = (ctypes.c_void_p * len(names))(*[_ptr(device_weights[n]) for n in names])
        h = ctypes.c_void_p()
        _check(lib().vla_model_create(ctypes.byref(self._c), table, len(names), ctypes.byref(h)))
        self.handle = h

    def close(self):
        if getattr(self, "handle", None):
            lib().vla_model_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def kv_cache_bytes(self, batch: int, prefix_len: int) -> int:
        return lib().vla_kv_cache_bytes(self.handle, batch, prefix_len)

    def set_loop_mode(self, mode: int):
        _check(lib().vla_model_set_option(self.handle, VLA_OPT_LOOP_MODE, mode))

    def set_profile(self, reps: int):
        """0 = off; R >= 1 = time each launch of the next denoise calls as the
        mean of R back-to-back repetitions (R > 1 is for timing only)."""
        _check(lib().vla_model_set_option(self.handle, VLA_OPT_PROFILE, int(reps)))

    def set_attn_splits(self, splits: int):
        """Key splits of the launch-per-phase attention (0 = automatic)."""
        _check(lib().vla_model_set_option(self.handle, VLA_OPT_ATTN_SPLITS, int(splits)))

    def set_causal_self(self, on: bool):
        """Causal action-token attention (self and joint sublayers): token i sees
        action tokens 0 .. i and every prefix row.  Discards cached plans."""
        _check(lib().vla_model_set_option(self.handle, VLA_OPT_CAUSAL_SELF, int(bool(on))))

    def set_state_token(self, on: bool):
        """The pi0-style embedding: the state as its own leading token."""
        _check(lib().vla_model_set_option(self.handle, VLA_OPT_STATE_TOKEN, 1 if on else 0))

    def set_rope_base(self, base: float):
        """Rotary position embedding of self / joint queries and keys (0 = none).
        Discards cached plans; build the prefix cache after setting it."""
        _check(lib().vla_model_set_option(self.handle, VLA_OPT_ROPE_BASE, int(base)))

    def set_spin_limit(self, polls: int):
        """Polls of one barrier wait of the persistent step kernel before it
        gives up (-1 = the library default); small values force the failure path."""
        _check(lib().vla_model_set_option(self.handle, VLA_OPT_PERSIST_SPIN_LIMIT, int(polls)))

    def check(self, stream=None):
        """Synchronise the stream; raise VlaError(VLA_E_DEVICE) if an earlier
        denoise call of this model failed on the device."""
        _check(lib().vla_model_check(self.handle, _stream(stream)))

    def set_trace(self, mode):
        """Record the persistent kernel's phase timeline on the next calls:
        0 off, 1 one workgroup per team, 2 every workgroup (first 256 marks)."""
        _check(lib().vla_model_set_option(self.handle, VLA_OPT_TRACE, int(mode)))

    def trace_read(self, all_workgroups: bool = False):
        """uint64 clock values (100 MHz) of the last traced persistent call:
        [8][PERSIST_TRACE_MAX] (mode 1) or [256][256] (mode 2); None if none."""
        import numpy as np
        shape = (256, 256) if all_workgroups else (8, PERSIST_TRACE_MAX)
        out = np.zeros(shape, np.uint64)
        n = lib().vla_test_persist_trace(self.handle, out.ctypes.data_as(ctypes.POINTER(ctypes.c_uint64)),
                                         shape[1])
        return None if n < 0 else out

    def profile_read(self) -> List[dict]:
        """Per-launch timings of the last profiled denoise call."""
        n = lib().vla_profile_read(self.handle, None, 0)
        if n < 0:
            return []
        buf = (VlaOpTime * n)()
        lib().vla_profile_read(self.handle, buf, n)
        return [dict(kind=OP_KINDS.get(o.kind, str(o.kind)), M=o.M, N=o.N, K=o.K, bytes=o.bytes,
                     flops=o.flops, ms=o.ms) for o in buf]

    def prefix_kv_build(self, prefix_hidden, batch: int, prefix_len: int, kv_cache, kv_cache_bytes: int,
                        stream=None):
        _check(lib().vla_prefix_kv_build(self.handle, _ptr(prefix_hidden), batch, prefix_len, _ptr(kv_cache),
                                         kv_cache_bytes, _stream(stream)))

    def prefix_kv_build_noalloc(self, prefix_hidden, batch: int, prefix_len: int, kv_cache, kv_cache_bytes: int,
                                stream=None):
        """vla_prefix_kv_build with its scratch in the library's static device array."""
        _check(lib().vla_prefix_kv_build_noalloc(self.handle, _ptr(prefix_hidden), batch, prefix_len,
                                                 _ptr(kv_cache), kv_cache_bytes, _stream(stream)))

    def denoise(self, kv_cache, kv_cache_bytes: int, batch: int, prefix_len: int, noise, state,
                t_schedule: Sequence[float], act_mean=None, act_std=None, actions_out=None, stream=None):
        n_steps = len(t_schedule) - 1
        sched = (ctypes.c_float * len(t_schedule))(*[float(t) for t in t_schedule])
        _check(lib().vla_denoise(self.handle, _ptr(kv_cache), kv_cache_bytes, batch, prefix_len, _ptr(noise),
                                 _ptr(state), sched, n_steps, _ptr(act_mean), _ptr(act_std), _ptr(actions_out),
                                 _stream(stream)))


def weight_count(cfg) -> int:
    c = make_config(cfg)
    return lib().vla_weight_count(ctypes.byref(c))


def ternary_gemm(x, w_packed, M: int, N: int, K: int, acc_out, stream=None):
    _check(lib().vla_ternary_gemm(_ptr(x), _ptr(w_packed), M, N, K, _ptr(acc_out), _stream(stream)))


# ---- test-only per-kernel entries (include/vla_test.h) ---------------------

def test_gemm(elem: int, x, w, M: int, N: int, K: int, y, variant: int = 0, stream=None):
    _check(lib().vla_test_gemm(elem, _ptr(x), _ptr(w), M, N, K, variant, _ptr(y), _stream(stream)))


def test_attention(elem: int, mode: int, q, k_self, v_self, k_cache, v_cache, B: int, n: int, P: int, H: int,
                   G: int, hd: int, o, kv_split: int = 0, stream=None):
    _check(lib().vla_test_attention(elem, mode, _ptr(q), _ptr(k_self), _ptr(v_self), _ptr(k_cache),
                                    _ptr(v_cache), B, n, P, H, G, hd, kv_split, _ptr(o), _stream(stream)))


def test_adarms(elem: int, x, part, nsplit: int, alpha, gamma, beta, M: int, d: int, eps: float, u,
                u_f32: bool, stream=None):
    _check(lib().vla_test_adarms(elem, _ptr(x), _ptr(part), nsplit, _ptr(alpha), _ptr(gamma), _ptr(beta), M, d,
                                 eps, _ptr(u), int(bool(u_f32)), _stream(stream)))


def test_time_cond(model: "Model", t_schedule: Sequence[float], mods, modf, stream=None):
    tau = (ctypes.c_float * len(t_schedule))(*[float(t) for t in t_schedule])
    _check(lib().vla_test_time_cond(model.handle, tau, len(t_schedule) - 1, _ptr(mods), _ptr(modf),
                                    _stream(stream)))


def test_quantize_i8(x, M: int, K: int, q, r, stream=None):
    _check(lib().vla_test_quantize_i8(_ptr(x), M, K, _ptr(q), _ptr(r), _stream(stream)))


def test_quantize_bf16(x, M: int, K: int, ldx: int, q, r, stream=None):
    _check(lib().vla_test_quantize_bf16(_ptr(x), M, K, ldx, _ptr(q), _ptr(r), _stream(stream)))


def test_ternary_linear(x, w_packed, M: int, N: int, K: int, scale: float, y, stream=None):
    _check(lib().vla_test_ternary_linear(_ptr(x), _ptr(w_packed), M, N, K, float(scale), _ptr(y), _stream(stream)))


def test_ternary_gemm(q, r, w_packed, wscale, M: int, N: int, K: int, variant: int, y, iters: int = 1,
                      stream=None) -> float:
    """The W2A8 GEMM alone on int8 codes: variant 0 the int8-MFMA launch, 1 the
    VALU sdot4 kernel, 2 / 3 / 4 the many-row tiled kernel with 32- / 64- /
    128-row tiles of 128 columns, 5 / 6 with 64- / 128-row tiles of 256 columns
    (eight waves), 7 / 8 / 9 with 32- / 64- / 128-row tiles of 128 columns on
    eight waves in two K-slice groups.  Returns the mean microseconds of one of
    `iters` launches."""
    us = ctypes.c_float(0.0)
    _check(lib().vla_test_ternary_gemm(_ptr(q), _ptr(r), _ptr(w_packed), _ptr(wscale), M, N, K, variant, iters,
                                       _ptr(y), ctypes.byref(us), _stream(stream)))
    return float(us.value)


def test_rope(elem: int, x, rows: int, rows_per_request: int, ld: int, col0: int, nheads: int, hd: int, pos0: int,
              base: float, stream=None):
    """Rotary position embedding in place on x (the RoPE variant's kernel)."""
    _check(lib().vla_test_rope(elem, _ptr(x), rows, rows_per_request, ld, col0, nheads, hd, pos0, float(base),
                               _stream(stream)))


# ---- the prefix stage: backbone prefill -------------------------------------

def make_backbone_config(bcfg) -> VlaBackboneConfig:
    """vla_backbone_config from an object with the backbone's attributes."""
    return VlaBackboneConfig(
        n_layers=bcfg.n_layers, d_model=bcfg.d_model, n_heads=bcfg.n_heads, head_dim=bcfg.head_dim,
        n_kv_heads=bcfg.n_kv_heads, d_ff=bcfg.d_ff, mlp=MLPS[bcfg.mlp], wtype=WTYPES[bcfg.wtype],
        rope_base=float(bcfg.rope_base), rms_eps=float(bcfg.rms_eps))


def backbone_weight_order(bcfg) -> List[str]:
    """Backbone weight-table names in the order vla.h documents (ternary
    matrices followed by '<name>.scale')."""
    tern = bcfg.wtype == "ternary"
    mats = ["W1", "W2"] if bcfg.mlp == "gelu" else ["W_g", "W_u", "W_d"]
    names = ["g_f"]
    for l in range(bcfg.n_layers):
        p = f"B{l}."
        for n in ["g_att", "W_q", "W_k", "W_v", "W_o", "g_mlp"] + mats:
            names.append(p + n)
            if tern and n.startswith("W"):
                names.append(p + n + ".scale")
    return names


class Backbone:
    """A vla_backbone created from device tensors keyed by weight-table name."""

    def __init__(self, bcfg, device_weights: Dict[str, object]):
        self.cfg = bcfg
        self._c = make_backbone_config(bcfg)
        names = backbone_weight_order(bcfg)
        want = lib().vla_backbone_weight_count(ctypes.byref(self._c))
        if want != len(names):
            raise VlaError(1, f"backbone weight table length mismatch ({want} vs {len(names)})")
        table = (ctypes.c_void_p * len(names))(*[_ptr(device_weights[n]) for n in names])
        h = ctypes.c_void_p()
        _check(lib().vla_backbone_create(ctypes.byref(self._c), table, len(names), ctypes.byref(h)))
        self.handle = h

    def close(self):
        if getattr(self, "handle", None):
            lib().vla_backbone_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def prefill(self, embeds, batch: int, prefix_len: int, hidden_out, stream=None):
        _check(lib().vla_prefix_prefill(self.handle, _ptr(embeds), batch, prefix_len, _ptr(hidden_out),
                                        _stream(stream)))
