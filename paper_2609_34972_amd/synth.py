"""Seeded synthetic inputs shared by the GPU path, the oracle and the benchmark.

This module draws random numbers and nothing else: it holds none of the
method's arithmetic. Every tensor is drawn in fp32 from
``numpy.random.default_rng(SeedSequence([seed, tensor_id, layer]))`` so that any
single layer of any weight can be regenerated on its own, then rounded to the
workload dtype (bf16 by round-to-nearest-even). The GPU and the oracle both
consume exactly these bytes (the oracle widens them to fp64).

Distributions (weights N(0, 1/fan_in), activations N(0, 1)):
  E      [B*Nv, d]        N(0,1), optional outlier channels multiplied by a scale
  Dw     [L, r, d]        N(0, 1/d)   down-projection D_l stored out x in
  Uw     [L, d, r]        N(0, 1/r)   up-projection U_l stored out x in
  gamma  [L, d]           1 + 0.1 N(0,1)  frozen RMSNorm weight of each layer
  Wk, Wv [L, Hkv*hd, d]   N(0, 1/d)   frozen key / value projections
  Q      [L, B, Nq, Hq, hd]    N(0,1)  text queries of each layer
  Kt, Vt [L, B, Hkv, Nkt, hd]  N(0,1)  text key / value cache of each layer
  Kv, Vv [L, B, Hkv, Nv, hd]   N(0,1)  cached visual K/V (decode workload only)
  k_bias, v_bias [L, Hkv*hd]   0.05 N(0,1)      backbone projection biases
  k_norm [L, hd]               1 + 0.1 N(0,1)   backbone per-head key norm weight
  delta-rule inputs            k [B,Hk,N,dk] unit rows (as the backbone normalises its keys),
                               v [B,Hv,N,dv] N(0,1), alpha = exp(-0.1 softplus(N(0,1))),
                               beta = sigmoid(N(0,1)), initial state S [B,Hv,dk,dv] 0.1 N(0,1)
  positions [B, 3, Nv] int32   position ids of the visual tokens: p0 + i on every axis for a
                               single image, or (p0 + frame, p0 + row, p0 + column) for a video
                               grid (a multimodal rotary embedding's three axes)
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from typing import Dict, Iterable, Optional, Sequence

import numpy as np
import torch

from .configs import Workload

TENSOR_IDS = {"E": 1, "Dw": 2, "Uw": 3, "gamma": 4, "Wk": 5, "Wv": 6, "Q": 7, "Kt": 8,
              "Vt": 9, "Kv": 10, "Vv": 11, "k_bias": 12, "v_bias": 13, "k_norm": 14,
              "dr_k": 15, "dr_v": 16, "dr_alpha": 17, "dr_beta": 18, "dr_S": 19}

_THREADS = max(1, min(16, os.cpu_count() or 1))


def normal(seed: int, name: str, layer: int, shape: Sequence[int]) -> np.ndarray:
    """Standard normal fp32 array for (seed, tensor, layer)."""
    rng = np.random.default_rng(np.random.SeedSequence([seed, TENSOR_IDS[name], layer]))
    return rng.standard_normal(tuple(shape), dtype=np.float32)


def torch_dtype(w: Workload) -> torch.dtype:
    return torch.float32 if w.dtype == "f32" else torch.bfloat16


def _to_dtype(a: np.ndarray, dt: torch.dtype) -> torch.Tensor:
    return torch.from_numpy(a).to(dt)


def _per_layer(seed: int, name: str, layers: Sequence[int], shape: Sequence[int], std: float,
               shift: float, dt: torch.dtype) -> torch.Tensor:
    def one(l: int) -> torch.Tensor:
        a = normal(seed, name, l, shape)
        if std != 1.0:
            a *= np.float32(std)
        if shift != 0.0:
            a += np.float32(shift)
        return _to_dtype(a, dt)

    if len(layers) == 1:
        return one(layers[0]).unsqueeze(0)
    with ThreadPoolExecutor(_THREADS) as ex:
        parts = list(ex.map(one, layers))
    return torch.stack(parts, 0)


def make_E(w: Workload, seed: int = 0) -> torch.Tensor:
    a = normal(seed, "E", 0, (w.T, w.d))
    if w.outlier_channels:
        a[:, list(w.outlier_channels)] *= np.float32(w.outlier_scale)
    return _to_dtype(a, torch_dtype(w))


def make_build_weights(w: Workload, seed: int = 0,
                       layers: Optional[Iterable[int]] = None) -> Dict[str, torch.Tensor]:
    """Adapter and frozen K/V weights for the requested layers (default: all)."""
    ls = list(range(w.L)) if layers is None else list(layers)
    dt = torch_dtype(w)
    return {
        "Dw": _per_layer(seed, "Dw", ls, (w.r, w.d), w.d ** -0.5, 0.0, dt),
        "Uw": _per_layer(seed, "Uw", ls, (w.d, w.r), w.r ** -0.5, 0.0, dt),
        "gamma": _per_layer(seed, "gamma", ls, (w.d,), 0.1, 1.0, dt),
        "Wk": _per_layer(seed, "Wk", ls, (w.kv, w.d), w.d ** -0.5, 0.0, dt),
        "Wv": _per_layer(seed, "Wv", ls, (w.kv, w.d), w.d ** -0.5, 0.0, dt),
    }


def make_text(w: Workload, seed: int = 0,
              layers: Optional[Iterable[int]] = None) -> Dict[str, torch.Tensor]:
    """Text queries and text K/V cache for the requested layers."""
    ls = list(range(w.L)) if layers is None else list(layers)
    dt = torch_dtype(w)
    return {
        "Q": _per_layer(seed, "Q", ls, (w.B, w.Nq, w.Hq, w.hd), 1.0, 0.0, dt),
        "Kt": _per_layer(seed, "Kt", ls, (w.B, w.Hkv, w.Nkt, w.hd), 1.0, 0.0, dt),
        "Vt": _per_layer(seed, "Vt", ls, (w.B, w.Hkv, w.Nkt, w.hd), 1.0, 0.0, dt),
    }


def make_visual_cache(w: Workload, seed: int = 0,
                      layers: Optional[Iterable[int]] = None) -> Dict[str, torch.Tensor]:
    """Cached visual K/V drawn directly (used where attention is tested alone)."""
    ls = list(range(w.L)) if layers is None else list(layers)
    dt = torch_dtype(w)
    return {
        "Kv": _per_layer(seed, "Kv", ls, (w.B, w.Hkv, w.Nv, w.hd), 1.0, 0.0, dt),
        "Vv": _per_layer(seed, "Vv", ls, (w.B, w.Hkv, w.Nv, w.hd), 1.0, 0.0, dt),
    }


def make_epilogue_weights(w: Workload, seed: int = 0,
                          layers: Optional[Iterable[int]] = None) -> Dict[str, torch.Tensor]:
    """Backbone K/V projection biases and per-head key norm weights."""
    ls = list(range(w.L)) if layers is None else list(layers)
    dt = torch_dtype(w)
    return {
        "k_bias": _per_layer(seed, "k_bias", ls, (w.kv,), 0.05, 0.0, dt),
        "v_bias": _per_layer(seed, "v_bias", ls, (w.kv,), 0.05, 0.0, dt),
        "k_norm": _per_layer(seed, "k_norm", ls, (w.hd,), 0.1, 1.0, dt),
    }


def image_positions(B: int, Nv: int, p0: int = 0) -> torch.Tensor:
    """Positions p0 + i of Nv consecutive visual tokens, repeated on the three axes."""
    p = torch.arange(Nv, dtype=torch.int32) + p0
    return p.view(1, 1, Nv).expand(B, 3, Nv).contiguous()


def video_positions(B: int, frames: int, rows: int, cols: int, p0: int = 0) -> torch.Tensor:
    """(p0 + frame, p0 + row, p0 + column) of a frames x rows x cols token grid (row-major)."""
    f, r, c = torch.meshgrid(torch.arange(frames), torch.arange(rows), torch.arange(cols),
                             indexing="ij")
    p = torch.stack([f.reshape(-1), r.reshape(-1), c.reshape(-1)], 0).to(torch.int32) + p0
    return p.unsqueeze(0).expand(B, 3, frames * rows * cols).contiguous()


def make_delta_inputs(w, seed: int = 0) -> Dict[str, torch.Tensor]:
    """Inputs of the gated delta-rule write of a DeltaWorkload (see the module docstring)."""
    dt = torch.float32 if w.dtype == "f32" else torch.bfloat16
    k = normal(seed, "dr_k", 0, (w.B, w.Hk, w.N, w.dk))
    k /= np.linalg.norm(k, axis=-1, keepdims=True)
    z = normal(seed, "dr_alpha", 0, (w.B, w.Hv, w.N)).astype(np.float64)
    alpha = np.exp(-0.1 * np.logaddexp(0.0, z)).astype(np.float32)
    beta = (1.0 / (1.0 + np.exp(-normal(seed, "dr_beta", 0, (w.B, w.Hv, w.N))))).astype(np.float32)
    return {
        "k": _to_dtype(k, dt),
        "v": _to_dtype(normal(seed, "dr_v", 0, (w.B, w.Hv, w.N, w.dv)), dt),
        "alpha": torch.from_numpy(alpha),
        "beta": torch.from_numpy(beta),
        "S": torch.from_numpy(0.1 * normal(seed, "dr_S", 0, (w.B, w.Hv, w.dk, w.dv))),
    }


def as_f64(t: torch.Tensor) -> np.ndarray:
    """The exact values a tensor holds, widened to fp64 for the oracle."""
    return t.detach().to("cpu").to(torch.float64).numpy()


def make_on_device(w: Workload, device, seed: int = 0) -> Dict[str, torch.Tensor]:
    """E, the build weights and the text tensors of every layer drawn on the GPU, with the same
    distributions as make_E / make_build_weights / make_text (torch's device generator instead
    of numpy's, so the values differ). Used where the numpy draw of a large workload would take
    minutes; operand statistics matter for timing because the chip's clock depends on them."""
    dt = torch_dtype(w)
    gen = torch.Generator(device=device)
    gen.manual_seed(seed)

    def normal_(shape, std=1.0, shift=0.0):
        a = torch.randn(*shape, generator=gen, device=device, dtype=torch.float32)
        if std != 1.0:
            a.mul_(std)
        if shift != 0.0:
            a.add_(shift)
        return a.to(dt)

    def stack(shape, std=1.0, shift=0.0, L=None):
        return torch.stack([normal_(shape, std, shift) for _ in range(w.L if L is None else L)], 0)

    E = torch.randn(w.T, w.d, generator=gen, device=device, dtype=torch.float32)
    if w.outlier_channels:
        E[:, list(w.outlier_channels)] *= w.outlier_scale
    return {
        "E": E.to(dt),
        "Dw": stack((w.r, w.d), w.d ** -0.5),
        "Uw": stack((w.d, w.r), w.r ** -0.5),
        "gamma": stack((w.d,), 0.1, 1.0),
        "Wk": stack((w.kv, w.d), w.d ** -0.5),
        "Wv": stack((w.kv, w.d), w.d ** -0.5),
        "Q": stack((w.B, w.Nq, w.Hq, w.hd)),
        "Kt": stack((w.B, w.Hkv, w.Nkt, w.hd)),
        "Vt": stack((w.B, w.Hkv, w.Nkt, w.hd)),
    }
