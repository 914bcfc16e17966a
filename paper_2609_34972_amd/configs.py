"""Workload shapes for the visual-memory path.

Each workload fixes the sizes of the layer-wise visual-memory build
(Section 3.1, Eq. 4-5), the visual K/V projection (Section 3.2, Eq. 7) and the
text-query attention over [visual; text] keys (Section 3.2, Eq. 9).

The four prefill workloads are shaped like LLaVA-1.5-7B, LLaVA-NeXT-7B (5 image
tiles) and Qwen2.5-VL-7B on a 64-frame video; the decode workload is one new
text token per sequence reading cached LLaVA-7B-shaped visual and text K/V.
Nothing here performs any arithmetic of the method.
"""
from __future__ import annotations

from dataclasses import dataclass, replace
from typing import Optional, Tuple

ACT_SILU = 0      # the paper's activation (Section 3.1)
ACT_GELU = 1      # exact erf GELU, used by the small fp32 workload


@dataclass(frozen=True)
class Workload:
    name: str
    dtype: str            # "f32" or "bf16": the arithmetic type of every tensor
    d: int                # hidden size of the language model
    L: int                # number of layers with a visual memory
    r: int                # adapter bottleneck rank
    Hq: int               # query heads
    Hkv: int              # key/value heads (GQA when Hkv < Hq)
    hd: int               # head dimension
    Nv: int               # visual tokens per sequence
    Nt: int               # text tokens per sequence (queries in prefill)
    B: int                # sequences in the batch
    act: int = ACT_SILU
    eps: float = 1e-5     # RMSNorm epsilon
    outlier_channels: Tuple[int, ...] = ()
    outlier_scale: float = 1.0
    # decode-only: one query per sequence at text position q_pos0, attending
    # all Nv visual keys and text keys 0..q_pos0 (its own key included).
    decode: bool = False
    q_pos0: int = 0

    @property
    def T(self) -> int:
        return self.B * self.Nv

    @property
    def kv(self) -> int:
        return self.Hkv * self.hd

    @property
    def G(self) -> int:
        return self.Hq // self.Hkv

    @property
    def Nq(self) -> int:
        return 1 if self.decode else self.Nt

    @property
    def Nkt(self) -> int:
        return self.q_pos0 + 1 if self.decode else self.Nt

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


TINY = Workload("tiny", "f32", d=256, L=4, r=16, Hq=4, Hkv=4, hd=64, Nv=64, Nt=16, B=1,
                act=ACT_GELU, eps=1e-5)

LLAVA7B = Workload("llava7b", "bf16", d=4096, L=32, r=256, Hq=32, Hkv=32, hd=128, Nv=576, Nt=64,
                   B=4, eps=1e-5, outlier_channels=tuple(512 * k + 211 for k in range(8)),
                   outlier_scale=20.0)

LLAVA_NEXT = Workload("llava_next", "bf16", d=4096, L=32, r=256, Hq=32, Hkv=32, hd=128, Nv=2880,
                      Nt=128, B=8, eps=1e-5)

QWEN25VL_VIDEO = Workload("qwen25vl_video", "bf16", d=3584, L=28, r=512, Hq=28, Hkv=4, hd=128,
                          Nv=16384, Nt=128, B=1, eps=1e-6)

DECODE = Workload("decode", "bf16", d=4096, L=32, r=256, Hq=32, Hkv=32, hd=128, Nv=576, Nt=513,
                  B=64, eps=1e-5, decode=True, q_pos0=512)

ALL = {w.name: w for w in (TINY, LLAVA7B, LLAVA_NEXT, QWEN25VL_VIDEO, DECODE)}


def get(name: str) -> Workload:
    return ALL[name]


def flops_build_kv(w: Workload, layers: Optional[int] = None) -> float:
    """Algorithmic FLOPs of Eq. 4-5 and Eq. 7 (2 per multiply-add)."""
    L = w.L if layers is None else layers
    per_token_layer = 2 * w.d * w.r + 2 * w.r * w.d + 2 * w.d * 2 * w.kv
    return float(per_token_layer) * w.T * L


def attention_pairs(w: Workload) -> int:
    """Unmasked (query row, key) pairs per layer, summed over batch and q heads."""
    if w.decode:
        per_q = w.Nv + w.q_pos0 + 1
        return w.B * w.Hq * per_q
    text = sum(w.q_pos0 + i + 1 for i in range(w.Nq))
    return w.B * w.Hq * (w.Nq * w.Nv + text)


def flops_attention(w: Workload, layers: Optional[int] = None) -> float:
    """Algorithmic FLOPs of Eq. 9: QK^T and PV over unmasked pairs."""
    L = w.L if layers is None else layers
    return float(attention_pairs(w)) * 4 * w.hd * L


def bytes_attention(w: Workload, layers: Optional[int] = None) -> float:
    """Algorithmic HBM bytes of Eq. 9: Q, K, V (visual + text) read once, O written once."""
    L = w.L if layers is None else layers
    e = w.elem_bytes
    q = w.B * w.Nq * w.Hq * w.hd
    kv = 2 * w.B * w.Hkv * (w.Nv + w.Nkt) * w.hd
    return float((2 * q + kv) * e) * L


@dataclass(frozen=True)
class DeltaWorkload:
    """Visual write into the linear-attention layers of a hybrid Gated DeltaNet backbone
    (appendix on linear attention): N visual tokens of B sequences written into the state of
    Hv value heads (key heads Hk) in each of `layers` linear-attention layers."""
    name: str
    dtype: str
    B: int
    Hk: int
    Hv: int
    N: int
    dk: int
    dv: int
    layers: int

    def with_(self, **kw) -> "DeltaWorkload":
        return replace(self, **kw)


# 24 linear-attention layers with 16 key / 32 value heads of 128 channels (a 4B-class hybrid
# backbone with 8 full-attention layers); a 576-token image batch and a 16384-token video.
GDN_IMAGE = DeltaWorkload("gdn_image", "bf16", B=4, Hk=16, Hv=32, N=576, dk=128, dv=128, layers=24)
GDN_VIDEO = DeltaWorkload("gdn_video", "bf16", B=1, Hk=16, Hv=32, N=16384, dk=128, dv=128,
                          layers=24)


def bytes_delta_write(w: DeltaWorkload) -> float:
    """Bytes read once and written once by the visual write of one layer: k, v, the gates and
    the fp32 state in and out."""
    e = 2 if w.dtype == "bf16" else 4
    return (w.B * w.N * (w.Hk * w.dk + w.Hv * w.dv) * e + 2 * w.B * w.Hv * w.N * 4
            + 2 * w.B * w.Hv * w.dk * w.dv * 4)


def flops_delta_write(w: DeltaWorkload) -> float:
    """Arithmetic of the token-by-token recurrence for one layer: per token and value head, the
    decay (dk dv), the read-out S^T k (2 dk dv) and the rank-one update (3 dk dv)."""
    return 6.0 * w.B * w.Hv * w.N * w.dk * w.dv
