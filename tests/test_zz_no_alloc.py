"""The no-allocation prefix build (vla_prefix_kv_build_noalloc, for callers
that cannot allocate device memory) against vla_prefix_kv_build: the same
cache, bit for bit, on two calls in a row, the second with a smaller input
(the shared scratch keeps the first call's contents); sizes beyond the
scratch are refused before any work."""
import ctypes

import numpy as np
import pytest

import workloads as wl

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch as t
    if not t.cuda.is_available():
        pytest.skip("no GPU")
    return t


@pytest.mark.parametrize("name", ["ternary_w2a8", "smolvla_bf16"])
def test_noalloc_prefix_build_matches_allocating_entry(torch, name):
    """W2A8 (its scratch holds the prefix rows' int8 codes and row scales)
    and bf16 (no scratch): B = 2 at the workload's prefix length, then B = 1
    at a shorter, ragged one."""
    from paper_2606_08094_amd import vla
    from vla_testlib import device_weights, to_device
    cfg = wl.CONFIGS[name]
    W = wl.make_weights(cfg)
    model = vla.Model(cfg, device_weights(cfg, W))
    try:
        for i, (B, P) in enumerate([(2, cfg.prefix_len), (1, cfg.prefix_len // 2 + 3)]):
            prefix = wl.random_matrix((B, P, cfg.d_prefix), 100 + i, 1.0, bf16=True)
            pd = to_device(prefix, bf16=True)
            nbytes = model.kv_cache_bytes(B, P)
            ref = torch.zeros(nbytes, dtype=torch.uint8, device="cuda")
            got = torch.full((nbytes,), 0xA5, dtype=torch.uint8, device="cuda")
            model.prefix_kv_build(pd, B, P, ref, nbytes)
            model.prefix_kv_build_noalloc(pd, B, P, got, nbytes)
            torch.cuda.synchronize()
            same = bool(torch.equal(ref, got))
            print(f"{name} call {i} (B={B}, P={P}): caches identical: {same}", flush=True)
            assert same
    finally:
        model.close()


def test_noalloc_prefix_build_refuses_oversized_input(torch):
    """A W2A8 prefix whose codes do not fit the 16 MiB scratch is refused with
    VLA_E_UNSUPPORTED before anything is enqueued (the cache pointer is never
    touched, so a small stand-in buffer is passed)."""
    from paper_2606_08094_amd import vla
    from vla_testlib import device_weights
    cfg = wl.TERNARY_W2A8.with_(n_layers=1)
    model = vla.Model(cfg, device_weights(cfg, wl.make_weights(cfg)))
    try:
        B, P = 8, 1024                      # 8192 rows x (2560 + 4) bytes > 16 MiB
        stand_in = torch.zeros(64, dtype=torch.uint8, device="cuda")
        st = vla.lib().vla_prefix_kv_build_noalloc(model.handle, vla._ptr(stand_in), B, P, vla._ptr(stand_in),
                                                   model.kv_cache_bytes(B, P), None)
        assert vla.STATUS[st] == "VLA_E_UNSUPPORTED", vla.lib().vla_last_error()
        assert b"scratch" in vla.lib().vla_last_error()
        torch.cuda.synchronize()
    finally:
        model.close()
