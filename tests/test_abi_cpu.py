"""C-ABI checks that need no GPU: the library loads, exports every function
include/*.h declares, and rejects bad arguments on the host before touching
a device."""
import ctypes
import os
import re

import pytest

import workloads as wl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _vla():
    from paper_2606_08094_amd import vla
    if not os.path.exists(vla.LIB_PATH):
        pytest.skip("libvla.so not built")
    return vla


def declared_functions():
    names = set()
    for h in ("vla.h", "vla_test.h"):
        text = open(os.path.join(ROOT, "include", h)).read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        names |= set(re.findall(r"\b(vla_[a-z0-9_]+)\s*\(", text))
    return names


def test_exports_every_declared_symbol():
    vla = _vla()
    lib = ctypes.CDLL(vla.LIB_PATH)
    decl = declared_functions()
    assert decl >= {"vla_prefix_kv_build", "vla_denoise", "vla_ternary_gemm"}
    for name in decl:
        assert hasattr(lib, name), f"{name} declared but not exported"
    assert decl == set(vla.EXPORTS)


@pytest.mark.parametrize("name", list(wl.CONFIGS))
def test_binding_weight_order_matches_generator(name):
    """The binding's weight-table order is the generator's name order, with
    each ternary matrix followed by its scale."""
    vla = _vla()
    cfg = wl.CONFIGS[name]
    assert vla.weight_count(cfg) == len(vla.weight_order(cfg))
    gen = []
    for n in wl.weight_names(cfg):
        gen += [n, n + ".scale"] if wl.is_ternary_matrix(cfg, n) else [n]
    assert gen == vla.weight_order(cfg)


@pytest.mark.parametrize("bad,status", [
    (dict(n_kv_heads=3), "VLA_E_SHAPE"),          # H % G != 0
    (dict(d_model=255), "VLA_E_SHAPE"),           # odd width
    (dict(head_dim=96), "VLA_E_UNSUPPORTED"),
    (dict(d_ff=1000), "VLA_E_SHAPE"),             # not a multiple of 16
    (dict(n_layers=0), "VLA_E_SHAPE"),
    (dict(rms_eps=0.0), "VLA_E_ARG"),
])
def test_config_validation(bad, status):
    vla = _vla()
    cfg = wl.TINY_F32.with_(**bad)
    c = vla.make_config(cfg)
    h = ctypes.c_void_p()
    table = (ctypes.c_void_p * 1)()
    st = vla.lib().vla_model_create(ctypes.byref(c), table, 1, ctypes.byref(h))
    assert vla.STATUS[st] == status, vla.lib().vla_last_error()
    assert h.value is None
    assert vla.lib().vla_weight_count(ctypes.byref(c)) == -1


@pytest.mark.parametrize("name", sorted(wl.CONFIGS))
def test_weight_count_matches_table_order(name):
    """Every layer pattern (self_cross, joint, alt, cross) and weight type: the
    library's weight table length equals the binding's name list."""
    vla = _vla()
    cfg = wl.CONFIGS[name]
    c = vla.make_config(cfg)
    assert vla.lib().vla_weight_count(ctypes.byref(c)) == len(vla.weight_order(cfg))


def test_pattern_out_of_range_rejected():
    vla = _vla()
    c = vla.make_config(wl.TINY_F32.with_(pattern="cross"))
    assert vla.lib().vla_weight_count(ctypes.byref(c)) > 0
    c.pattern = 4
    assert vla.lib().vla_weight_count(ctypes.byref(c)) == -1


def test_null_table_entries_rejected_before_device_use():
    vla = _vla()
    cfg = wl.TINY_F32
    c = vla.make_config(cfg)
    n = vla.weight_count(cfg)
    table = (ctypes.c_void_p * n)()
    h = ctypes.c_void_p()
    assert vla.lib().vla_model_create(ctypes.byref(c), table, n, ctypes.byref(h)) == 1
    assert b"NULL" in vla.lib().vla_last_error()
    assert vla.lib().vla_model_create(ctypes.byref(c), table, n - 1, ctypes.byref(h)) == 1
    assert b"expected" in vla.lib().vla_last_error()


def test_call_validation_without_device():
    vla = _vla()
    L = vla.lib()
    f = (ctypes.c_float * 3)(1.0, 0.5, 0.0)
    assert L.vla_denoise(None, 16, 0, 1, 1, 16, 16, f, 2, None, None, 16, None) == 1
    assert L.vla_prefix_kv_build(None, 16, 1, 1, 16, 0, None) == 1
    assert L.vla_kv_cache_bytes(None, 1, 1) == 0
    assert vla.STATUS[L.vla_model_check(None, None)] == "VLA_E_ARG"
    assert vla.STATUS[L.vla_model_set_option(None, 7, 0)] == "VLA_E_ARG"
    # ternary GEMM: K % 4, negative sizes, NULL, misaligned
    assert vla.STATUS[L.vla_ternary_gemm(16, 16, 2, 2, 6, 16, None)] == "VLA_E_SHAPE"
    assert vla.STATUS[L.vla_ternary_gemm(16, 16, -1, 2, 8, 16, None)] == "VLA_E_SHAPE"
    assert vla.STATUS[L.vla_ternary_gemm(None, 16, 2, 2, 8, 16, None)] == "VLA_E_ARG"
    assert vla.STATUS[L.vla_ternary_gemm(17, 16, 2, 2, 8, 16, None)] == "VLA_E_ARG"
    assert vla.STATUS[L.vla_ternary_gemm(16, 16, 2, 2, 1 << 20, 16, None)] == "VLA_E_SHAPE"
    # empty problem: nothing to do, nothing touched
    assert L.vla_ternary_gemm(None, None, 0, 5, 8, 16, None) == 0
    assert L.vla_status_string(6) == b"VLA_E_NONFINITE"
    # test entries validate too
    assert vla.STATUS[L.vla_test_gemm(2, 16, 16, 1, 1, 8, 0, 16, None)] == "VLA_E_ARG"
    assert vla.STATUS[L.vla_test_gemm(1, 16, 16, 1, 1, 8, 5, 16, None)] == "VLA_E_ARG"
    assert vla.STATUS[L.vla_test_gemm(1, 16, 16, 1, 1, 8, 15, 16, None)] == "VLA_E_ARG"
    # the tiled kernel takes bf16 with M > 128 only, refused before any device work
    assert vla.STATUS[L.vla_test_gemm(1, 16, 16, 1, 1, 8, 3, 16, None)] == "VLA_E_UNSUPPORTED"
    assert vla.STATUS[L.vla_test_gemm(0, 16, 16, 200, 1, 8, 12, 16, None)] == "VLA_E_UNSUPPORTED"
    assert vla.STATUS[L.vla_test_gemm(1, 16, 16, 1, 1, 7, 0, 16, None)] == "VLA_E_SHAPE"
    assert vla.STATUS[L.vla_test_attention(1, 2, 16, 16, 16, 16, 16, 1, 4, 4, 6, 4, 64, 0, 16, None)] == "VLA_E_SHAPE"


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    from paper_2606_08094_amd import vla
    monkeypatch.setattr(vla, "LIB_PATH", str(tmp_path / "nope.so"))
    monkeypatch.setattr(vla, "_lib", None)
    with pytest.raises(RuntimeError, match="missing"):
        vla.lib()


@pytest.mark.parametrize("name", sorted(wl.BACKBONES))
def test_backbone_weight_count_matches_binding_order(name):
    """The library's backbone table length equals the binding's name list,
    which follows the generator's names (ternary matrices plus scales)."""
    vla = _vla()
    bcfg = wl.BACKBONES[name]
    c = vla.make_backbone_config(bcfg)
    order = vla.backbone_weight_order(bcfg)
    assert vla.lib().vla_backbone_weight_count(ctypes.byref(c)) == len(order)
    gen = []
    for n in wl.backbone_weight_names(bcfg):
        gen += [n, n + ".scale"] if wl.is_backbone_ternary(bcfg, n) else [n]
    assert gen == order


@pytest.mark.parametrize("bad,status", [
    (dict(wtype="f32"), "VLA_E_UNSUPPORTED"),
    (dict(n_kv_heads=3), "VLA_E_SHAPE"),
    (dict(head_dim=96), "VLA_E_UNSUPPORTED"),
    (dict(d_model=8192), "VLA_E_UNSUPPORTED"),
    (dict(rope_base=0.5), "VLA_E_ARG"),
    (dict(rms_eps=0.0), "VLA_E_ARG"),
    (dict(n_layers=0), "VLA_E_SHAPE"),
])
def test_backbone_config_validation(bad, status):
    vla = _vla()
    c = vla.make_backbone_config(wl.PI0_VLM_BF16.with_(**bad))
    h = ctypes.c_void_p()
    table = (ctypes.c_void_p * 1)()
    st = vla.lib().vla_backbone_create(ctypes.byref(c), table, 1, ctypes.byref(h))
    assert vla.STATUS[st] == status, vla.lib().vla_last_error()
    assert h.value is None
    assert vla.lib().vla_backbone_weight_count(ctypes.byref(c)) == -1


def test_backbone_calls_rejected_before_device_use():
    vla = _vla()
    L = vla.lib()
    c = vla.make_backbone_config(wl.PI0_VLM_BF16)
    n = L.vla_backbone_weight_count(ctypes.byref(c))
    h = ctypes.c_void_p()
    table = (ctypes.c_void_p * n)()
    assert vla.STATUS[L.vla_backbone_create(ctypes.byref(c), table, n, ctypes.byref(h))] == "VLA_E_ARG"
    assert b"NULL" in L.vla_last_error()
    assert vla.STATUS[L.vla_backbone_create(ctypes.byref(c), table, n - 1, ctypes.byref(h))] == "VLA_E_ARG"
    assert vla.STATUS[L.vla_prefix_prefill(None, 16, 1, 1, 16, None)] == "VLA_E_ARG"
    assert vla.STATUS[L.vla_prefix_kv_build_noalloc(None, 16, 1, 1, 16, 0, None)] == "VLA_E_ARG"


def test_diffusion_head_starts_from_uniform_noise():
    """Algorithm 1 draws the chunk's start a_0 from N(0, I), or uniformly for a
    diffusion head: the GR00T-shaped workload (diffusion-transformer head)
    draws U(-1, 1) per element, the flow-matching workloads N(0, 1)."""
    import numpy as np
    g = wl.make_batch(wl.CONFIGS["gr00t_alt_bf16"], 4)["noise"]
    assert g.shape == (4, 16, 32)
    assert g.min() >= -1.0 and g.max() < 1.0
    assert abs(float(g.mean())) < 0.05 and abs(float(g.var()) - 1.0 / 3.0) < 0.03
    p = wl.make_batch(wl.CONFIGS["pi0_bf16"], 1)["noise"]
    assert np.abs(p).max() > 2.0 and abs(float(p.var()) - 1.0) < 0.1
