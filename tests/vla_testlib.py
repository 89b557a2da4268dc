"""Helpers shared by the GPU tests, smoke() and bench.py: upload seeded
workloads to the device and run the library through its C ABI."""
from __future__ import annotations

import functools
import os
import sys
from typing import Dict

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import workloads as wl  # noqa: E402


def torch_mod():
    import torch
    return torch


def to_device(arr: np.ndarray, bf16: bool = False):
    """numpy -> CUDA tensor; bf16=True expects bf16-representable float32 values."""
    torch = torch_mod()
    if bf16:
        bits = wl.bf16_bits(arr).astype(np.int16)
        return torch.from_numpy(bits).cuda().view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(arr)).cuda()


def device_weights(cfg: wl.ExpertConfig, W: Dict[str, np.ndarray]):
    """Weight-table tensors on the GPU, keyed as the binding expects."""
    torch = torch_mod()
    out = {}
    for name, arr in W.items():
        if name.endswith(".scale"):
            out[name] = torch.tensor([float(arr)], dtype=torch.float32, device="cuda")
        elif wl.is_ternary_matrix(cfg, name):
            out[name] = torch.from_numpy(wl.pack_ternary(arr)).cuda()
        elif arr.ndim == 2 and cfg.wtype != "f32":
            out[name] = to_device(arr, bf16=True)
        else:
            out[name] = to_device(np.asarray(arr, np.float32))
    return out


@functools.lru_cache(maxsize=4)
def workload(name: str, batch: int = 1):
    """(cfg, numpy weights, numpy inputs) for a named workload, cached."""
    cfg = wl.CONFIGS[name].with_(batch=batch)
    return cfg, wl.make_weights(cfg), wl.make_batch(cfg, batch)


class Pipeline:
    """A model plus device buffers for one (batch, prefix_len) shape."""

    def __init__(self, cfg, W, inputs, loop_mode: int = 1):
        from paper_2606_08094_amd import vla
        torch = torch_mod()
        self.cfg = cfg
        self.dw = device_weights(cfg, W)
        self.model = vla.Model(cfg, self.dw)
        self.model.set_loop_mode(loop_mode)
        if getattr(cfg, "causal_self", False):
            self.model.set_causal_self(True)
        if getattr(cfg, "rope_base", 0.0) > 0:
            self.model.set_rope_base(cfg.rope_base)
        if getattr(cfg, "state_token", False):
            self.model.set_state_token(True)
        B = inputs["noise"].shape[0]
        self.B, self.P = B, cfg.prefix_len
        self.prefix = to_device(inputs["prefix"], bf16=cfg.wtype != "f32")
        self.noise = to_device(inputs["noise"].astype(np.float32))
        self.state = to_device(inputs["state"].astype(np.float32))
        self.cache_bytes = self.model.kv_cache_bytes(B, self.P)
        self.cache = torch.empty(self.cache_bytes, dtype=torch.uint8, device="cuda")
        self.out = torch.empty_like(self.noise)

    def build_cache(self):
        self.model.prefix_kv_build(self.prefix, self.B, self.P, self.cache, self.cache_bytes)

    def denoise(self, tau, mean=None, std=None, out=None):
        out = self.out if out is None else out
        self.model.denoise(self.cache, self.cache_bytes, self.B, self.P, self.noise, self.state, list(tau),
                           mean, std, out)
        return out

    def cache_array(self) -> np.ndarray:
        """The cache as float64 [Lc][2][B][G][P][hd]."""
        torch = torch_mod()
        c = self.cfg
        shape = (c.n_cache_layers, 2, self.B, c.n_kv_heads, self.P, c.head_dim)
        t = self.cache.view(torch.float32 if c.wtype == "f32" else torch.bfloat16)
        return t.float().cpu().numpy().astype(np.float64).reshape(shape)

    def close(self):
        self.model.close()


def device_backbone_weights(bcfg: wl.BackboneConfig, Wb: Dict[str, np.ndarray]):
    """Backbone weight-table tensors on the GPU, keyed as the binding expects."""
    torch = torch_mod()
    out = {}
    for name, arr in Wb.items():
        if name.endswith(".scale"):
            out[name] = torch.tensor([float(arr)], dtype=torch.float32, device="cuda")
        elif wl.is_backbone_ternary(bcfg, name):
            out[name] = torch.from_numpy(wl.pack_ternary(arr)).cuda()
        elif arr.ndim == 2:
            out[name] = to_device(arr, bf16=True)
        else:
            out[name] = to_device(np.asarray(arr, np.float32))
    return out


class Prefill:
    """A backbone plus device buffers for one (batch, prefix_len) shape."""

    def __init__(self, bcfg, Wb, embeds: np.ndarray):
        from paper_2606_08094_amd import vla
        torch = torch_mod()
        self.cfg = bcfg
        self.dw = device_backbone_weights(bcfg, Wb)
        self.bb = vla.Backbone(bcfg, self.dw)
        self.B, self.P = embeds.shape[0], embeds.shape[1]
        self.embeds = to_device(embeds, bf16=True)
        self.hidden = torch.empty((self.B, self.P, bcfg.d_model), dtype=torch.bfloat16, device="cuda")

    def run(self, stream=None):
        self.bb.prefill(self.embeds, self.B, self.P, self.hidden, stream)
        return self.hidden

    def close(self):
        self.bb.close()
