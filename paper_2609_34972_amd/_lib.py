"""Python binding of ``libdeltavision.so``: argument marshalling only.

Every function takes torch tensors that live in device memory, derives the
sizes the C ABI expects from their shapes, passes raw device pointers and the
current HIP stream, and raises on a non-zero status. All arithmetic happens in
the library's gfx950 kernels; there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
import threading
from dataclasses import dataclass
from typing import Optional, Tuple

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libdeltavision.so")

DV_F32, DV_BF16 = 0, 1
ACT_SILU, ACT_GELU = 0, 1

# Every symbol declared by include/deltavision.h.
EXPORTS = (
    "dv_build_visual_memory",
    "dv_project_visual_kv_workspace",
    "dv_project_visual_kv",
    "dv_project_visual_kv_fused",
    "dv_set_fused_kv",
    "dv_set_up_kernel",
    "dv_project_visual_kv_up_kernel",
    "dv_text_visual_attention_workspace",
    "dv_text_visual_attention",
    "dv_text_visual_attention_noalloc",
    "dv_status_string",
    "dv_last_error",
    "dv_abi_version",
    "dv_probe_mfma",
    "dv_time_kernel",
    "dv_recurrent_visual_kv_workspace",
    "dv_recurrent_visual_kv",
    "dv_kept_visual_kv_workspace",
    "dv_kept_visual_kv",
    "dv_project_visual_kv_ex_workspace",
    "dv_project_visual_kv_ex",
    "dv_delta_rule_workspace",
    "dv_delta_rule_write",
)


class _KvEpilogue(ctypes.Structure):
    """Mirror of dv_kv_epilogue."""
    _fields_ = [("k_bias", ctypes.c_void_p), ("v_bias", ctypes.c_void_p),
                ("k_norm", ctypes.c_void_p), ("k_norm_eps", ctypes.c_float),
                ("positions", ctypes.c_void_p), ("rope_sections", ctypes.c_int32 * 3),
                ("rope_theta", ctypes.c_float)]


@dataclass
class KVEpilogue:
    """Backbone epilogue of the visual K/V: projection bias [L, Hkv*hd], per-head key RMSNorm
    weight [L, hd] (call dtype), and rotary embedding at int32 positions [B, 3, Nv] (axes of a
    multimodal rotary embedding; sections default to (hd/2, 0, 0), the 1-D rotation)."""
    k_bias: Optional[torch.Tensor] = None
    v_bias: Optional[torch.Tensor] = None
    k_norm: Optional[torch.Tensor] = None
    k_norm_eps: float = 1e-6
    positions: Optional[torch.Tensor] = None
    rope_sections: Optional[Tuple[int, int, int]] = None
    rope_theta: float = 10000.0

KERNEL_DOWN, KERNEL_UP, KERNEL_KV, KERNEL_ATTENTION = 0, 1, 2, 3
KERNEL_DELTA_PREP, KERNEL_DELTA_SCAN = 4, 5

_lock = threading.Lock()
_lib = None


class DeltaVisionError(RuntimeError):
    def __init__(self, status: int, name: str, detail: str):
        super().__init__(f"{name}: {detail}" if detail else name)
        self.status = status
        self.name = name


def load() -> ctypes.CDLL:
    """Load the built library (raises if it has not been built)."""
    global _lib
    with _lock:
        if _lib is not None:
            return _lib
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is missing: build it with `python -m paper_2609_34972_amd.build`; "
                "there is no non-HIP implementation")
        lib = ctypes.CDLL(LIB_PATH)
        vp, i32, i64, f32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_size_t
        lib.dv_build_visual_memory.argtypes = [vp, vp, vp, i64, i32, i32, i32, i32, i32, vp]
        lib.dv_build_visual_memory.restype = i32
        lib.dv_project_visual_kv_workspace.argtypes = [i64, i32, i32, i32]
        lib.dv_project_visual_kv_workspace.restype = sz
        lib.dv_project_visual_kv.argtypes = [vp] * 8 + [i32] * 9 + [f32, i32, vp, sz, vp]
        lib.dv_project_visual_kv.restype = i32
        lib.dv_project_visual_kv_fused.argtypes = [i32] * 5
        lib.dv_project_visual_kv_fused.restype = i32
        lib.dv_set_fused_kv.argtypes = [i32]
        lib.dv_set_fused_kv.restype = i32
        lib.dv_set_up_kernel.argtypes = [i32]
        lib.dv_set_up_kernel.restype = i32
        lib.dv_project_visual_kv_up_kernel.argtypes = [i64, i32, i32, i32, i32]
        lib.dv_project_visual_kv_up_kernel.restype = i32
        lib.dv_project_visual_kv_ex_workspace.argtypes = [i64, i32, i32, i32, i32]
        lib.dv_project_visual_kv_ex_workspace.restype = sz
        lib.dv_project_visual_kv_ex.argtypes = ([vp] * 8 + [i32] * 9 + [f32, ctypes.POINTER(_KvEpilogue), i32, vp, sz, vp])
        lib.dv_project_visual_kv_ex.restype = i32
        lib.dv_delta_rule_workspace.argtypes = [i32] * 6
        lib.dv_delta_rule_workspace.restype = sz
        lib.dv_delta_rule_write.argtypes = [vp] * 5 + [i32] * 7 + [vp, sz, vp]
        lib.dv_delta_rule_write.restype = i32
        lib.dv_text_visual_attention_workspace.argtypes = [i32] * 7
        lib.dv_text_visual_attention_workspace.restype = sz
        lib.dv_text_visual_attention.argtypes = [vp] * 6 + [i32] * 8 + [f32, i32, vp, sz, vp]
        lib.dv_text_visual_attention.restype = i32
        lib.dv_text_visual_attention_noalloc.argtypes = [vp] * 6 + [i32] * 8 + [f32, i32, vp]
        lib.dv_text_visual_attention_noalloc.restype = i32
        lib.dv_status_string.argtypes = [i32]
        lib.dv_status_string.restype = ctypes.c_char_p
        lib.dv_last_error.argtypes = []
        lib.dv_last_error.restype = ctypes.c_char_p
        lib.dv_abi_version.argtypes = []
        lib.dv_abi_version.restype = i32
        lib.dv_time_kernel.argtypes = [i32, vp, vp]
        lib.dv_time_kernel.restype = i32
        lib.dv_probe_mfma.argtypes = [i32, i32, vp, vp]
        lib.dv_probe_mfma.restype = i32
        lib.dv_recurrent_visual_kv_workspace.argtypes = [i64, i32, i32, i32, i32]
        lib.dv_recurrent_visual_kv_workspace.restype = sz
        lib.dv_recurrent_visual_kv.argtypes = [vp] * 8 + [i32] * 8 + [f32, i32, vp, sz, vp]
        lib.dv_recurrent_visual_kv.restype = i32
        lib.dv_kept_visual_kv_workspace.argtypes = [ctypes.c_int64, i32, i32, i32, i32]
        lib.dv_kept_visual_kv_workspace.restype = sz
        lib.dv_kept_visual_kv.argtypes = [vp] * 9 + [i32] * 8 + [f32, i32, vp, sz, vp]
        lib.dv_kept_visual_kv.restype = i32
        _lib = lib
        return lib


def _check(status: int) -> None:
    if status != 0:
        lib = load()
        raise DeltaVisionError(status, lib.dv_status_string(status).decode(),
                               lib.dv_last_error().decode())


def _dtype_code(*ts: torch.Tensor) -> int:
    dt = ts[0].dtype
    for t in ts:
        if t.dtype != dt:
            raise TypeError(f"all tensors of a call must share one dtype ({t.dtype} vs {dt})")
    if dt == torch.bfloat16:
        return DV_BF16
    if dt == torch.float32:
        return DV_F32
    raise TypeError(f"unsupported dtype {dt}")


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("tensors must be in device memory")
    if not t.is_contiguous():
        raise ValueError("tensors must be contiguous")
    return t.data_ptr()


def _stream(device: torch.device, stream=None) -> int:
    s = stream if stream is not None else torch.cuda.current_stream(device)
    return s.cuda_stream


def _workspace(nbytes: int, device: torch.device, stream=None) -> torch.Tensor:
    """A temporary workspace for one call. The caching allocator ties a block to the stream it
    was allocated on; when the work runs on another stream, record that stream so the block is
    not handed out again before the enqueued kernels are done with it."""
    ws = torch.empty(max(int(nbytes), 16), dtype=torch.uint8, device=device)
    if stream is not None:
        ws.record_stream(stream)
    return ws


def time_kernel(kernel: int, begin: Optional[int] = None, end: Optional[int] = None) -> None:
    """Bracket every later launch of `kernel` on this thread with two hipEvent_t handles
    (raw integers, e.g. from hipEventCreate); time_kernel(kernel) switches the hook off."""
    _check(load().dv_time_kernel(kernel, begin, end))


PROBE_BLOCKS = 1024
PROBE_FLOP_PER_ITER = 1024 * 8 * 32 * 2 * 16 * 16 * 32  # blocks x waves x MFMAs x FLOP per MFMA


def probe_mfma(random: bool, iters: int, sink: torch.Tensor, stream=None) -> None:
    """Enqueue the MFMA-rate probe (iters x PROBE_FLOP_PER_ITER FLOP on register operands);
    sink is a float32 CUDA tensor of at least PROBE_BLOCKS elements."""
    if sink.dtype != torch.float32 or sink.numel() < PROBE_BLOCKS or not sink.is_cuda:
        raise ValueError("sink must be a float32 CUDA tensor of at least 1024 elements")
    _check(load().dv_probe_mfma(1 if random else 0, iters, _ptr(sink), _stream(sink.device, stream)))


def build_visual_memory(E: torch.Tensor, Dw: torch.Tensor, Z: torch.Tensor, act: int = ACT_SILU,
                        stream=None) -> torch.Tensor:
    """Z[l] = phi(E D_l) for every layer. E [T,d], Dw [L,r,d], Z [L,T,r]."""
    T, d = E.shape
    L, r, d2 = Dw.shape
    if d2 != d or tuple(Z.shape) != (L, T, r):
        raise ValueError(f"shape mismatch: E {tuple(E.shape)} Dw {tuple(Dw.shape)} Z {tuple(Z.shape)}")
    code = _dtype_code(E, Dw, Z)
    _check(load().dv_build_visual_memory(_ptr(E), _ptr(Dw), _ptr(Z), T, d, L, r, act, code,
                                         _stream(E.device, stream)))
    return Z


def project_visual_kv_workspace(T: int, d: int, nl: int, dtype: torch.dtype) -> int:
    code = DV_BF16 if dtype == torch.bfloat16 else DV_F32
    return int(load().dv_project_visual_kv_workspace(T, d, nl, code))


def project_visual_kv_fused(d: int, r: int, Hkv: int, hd: int, dtype: torch.dtype) -> bool:
    """Whether project_visual_kv (no epilogue) takes the fused up + norm + K/V kernel now."""
    code = DV_BF16 if dtype == torch.bfloat16 else DV_F32
    return bool(load().dv_project_visual_kv_fused(d, r, Hkv, hd, code))


def set_up_kernel(mode: int) -> None:
    """Kernel for M * gamma and the row sums of squares in the bf16 projection: 0 by shape, 1 the
    tiled kernel, 2 the Z-resident kernel where it applies (process-wide)."""
    _check(load().dv_set_up_kernel(int(mode)))


def project_visual_kv_up_kernel(T: int, d: int, r: int, nl: int, dtype: torch.dtype) -> int:
    """The kernel (1 tiled, 2 Z-resident) a projection call with these sizes takes now."""
    code = DV_BF16 if dtype == torch.bfloat16 else DV_F32
    return int(load().dv_project_visual_kv_up_kernel(int(T), int(d), int(r), int(nl), code))


def set_fused_kv(on: bool) -> None:
    """Switch the fused up + norm + K/V kernel on or off for the sizes it covers (process-wide;
    off by default)."""
    _check(load().dv_set_fused_kv(1 if on else 0))


def project_visual_kv_ex_workspace(T: int, d: int, nl: int, hd: int, dtype: torch.dtype) -> int:
    code = DV_BF16 if dtype == torch.bfloat16 else DV_F32
    return int(load().dv_project_visual_kv_ex_workspace(T, d, nl, hd, code))


def _epilogue_struct(epi: KVEpilogue, L: int, B: int, Nv: int, Hkv: int, hd: int, dtype):
    def tensor(t, shape, dt, name):
        if t is None:
            return None
        if tuple(t.shape) != shape or t.dtype != dt or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous {dt} tensor of shape {shape}")
        return t.data_ptr()
    st = _KvEpilogue()
    st.k_bias = tensor(epi.k_bias, (L, Hkv * hd), dtype, "k_bias")
    st.v_bias = tensor(epi.v_bias, (L, Hkv * hd), dtype, "v_bias")
    st.k_norm = tensor(epi.k_norm, (L, hd), dtype, "k_norm")
    st.k_norm_eps = float(epi.k_norm_eps)
    st.positions = tensor(epi.positions, (B, 3, Nv), torch.int32, "positions")
    sec = epi.rope_sections if epi.rope_sections is not None else (hd // 2, 0, 0)
    st.rope_sections = (ctypes.c_int32 * 3)(*[int(x) for x in sec])
    st.rope_theta = float(epi.rope_theta)
    return st


def project_visual_kv(E, Z, Uw, gamma, Wk, Wv, Kv, Vv, eps: float, l0: int = 0,
                      nl: Optional[int] = None, ws: Optional[torch.Tensor] = None, stream=None,
                      epilogue: Optional[KVEpilogue] = None):
    """Memories, RMSNorm and visual K/V of layers l0..l0+nl-1 into Kv, Vv [L,B,Hkv,Nv,hd],
    optionally followed by the backbone epilogue (bias, key norm, rotary embedding)."""
    L, B, Hkv, Nv, hd = Kv.shape
    T, d = E.shape
    r = Z.shape[2]
    if nl is None:
        nl = L - l0
    if (T != B * Nv or tuple(Z.shape) != (L, T, r) or tuple(Uw.shape) != (L, d, r)
            or tuple(gamma.shape) != (L, d) or tuple(Wk.shape) != (L, Hkv * hd, d)
            or Wv.shape != Wk.shape or Vv.shape != Kv.shape):
        raise ValueError("shape mismatch in project_visual_kv")
    code = _dtype_code(E, Z, Uw, gamma, Wk, Wv, Kv, Vv)
    lib = load()
    if epilogue is None:
        if ws is None:
            ws = _workspace(project_visual_kv_workspace(T, d, nl, E.dtype), E.device, stream)
        _check(lib.dv_project_visual_kv(_ptr(E), _ptr(Z), _ptr(Uw), _ptr(gamma), _ptr(Wk),
                                        _ptr(Wv), _ptr(Kv), _ptr(Vv), B, Nv, d, L, r, Hkv, hd, l0,
                                        nl, float(eps), code, _ptr(ws), ws.numel(),
                                        _stream(E.device, stream)))
        return Kv, Vv
    st = _epilogue_struct(epilogue, L, B, Nv, Hkv, hd, E.dtype)
    if ws is None:
        ws = _workspace(project_visual_kv_ex_workspace(T, d, nl, hd, E.dtype), E.device, stream)
    _check(lib.dv_project_visual_kv_ex(_ptr(E), _ptr(Z), _ptr(Uw), _ptr(gamma), _ptr(Wk), _ptr(Wv),
                                       _ptr(Kv), _ptr(Vv), B, Nv, d, L, r, Hkv, hd, l0, nl,
                                       float(eps), ctypes.byref(st), code, _ptr(ws), ws.numel(),
                                       _stream(E.device, stream)))
    return Kv, Vv


def recurrent_visual_kv_workspace(T: int, d: int, L: int, r: int, dtype: torch.dtype) -> int:
    code = DV_BF16 if dtype == torch.bfloat16 else DV_F32
    return int(load().dv_recurrent_visual_kv_workspace(T, d, L, r, code))


def recurrent_visual_kv(E, Dw, Uw, gamma, Wk, Wv, Kv, Vv, eps: float, act: int = ACT_SILU,
                        ws: Optional[torch.Tensor] = None, stream=None):
    """Recurrent adapter (Eq. 6) and K/V of every layer into Kv, Vv [L,B,Hkv,Nv,hd]."""
    L, B, Hkv, Nv, hd = Kv.shape
    T, d = E.shape
    r = Dw.shape[1]
    if (T != B * Nv or tuple(Dw.shape) != (L, r, d) or tuple(Uw.shape) != (L, d, r)
            or tuple(gamma.shape) != (L, d) or tuple(Wk.shape) != (L, Hkv * hd, d)
            or Wv.shape != Wk.shape or Vv.shape != Kv.shape):
        raise ValueError("shape mismatch in recurrent_visual_kv")
    code = _dtype_code(E, Dw, Uw, gamma, Wk, Wv, Kv, Vv)
    if ws is None:
        ws = _workspace(recurrent_visual_kv_workspace(T, d, L, r, E.dtype), E.device, stream)
    _check(load().dv_recurrent_visual_kv(_ptr(E), _ptr(Dw), _ptr(Uw), _ptr(gamma), _ptr(Wk),
                                         _ptr(Wv), _ptr(Kv), _ptr(Vv), B, Nv, d, L, r, Hkv, hd, act,
                                         float(eps), code, _ptr(ws), ws.numel(),
                                         _stream(E.device, stream)))
    return Kv, Vv


def kept_visual_kv_workspace(T: int, d: int, r: int, nkeep: int, dtype: torch.dtype) -> int:
    code = DV_BF16 if dtype == torch.bfloat16 else DV_F32
    return int(load().dv_kept_visual_kv_workspace(T, d, r, nkeep, code))


def kept_visual_kv(E, Dw, Uw, gamma, Wk, Wv, keep, Kv, Vv, eps: float, act: int = ACT_SILU,
                   ws: Optional[torch.Tensor] = None, stream=None):
    """Adapters and K/V only for the layers with keep[l] true; Kv, Vv [nkeep,B,Hkv,Nv,hd]
    hold the kept layers in order (layer-wise adapter skipping)."""
    L, r, d = Dw.shape
    flags = bytes(1 if k else 0 for k in keep)
    if len(flags) != L:
        raise ValueError(f"keep has {len(flags)} entries for {L} layers")
    nkeep = sum(flags)
    T = E.shape[0]
    if nkeep == 0:
        if Kv is not None and Kv.numel() or Vv is not None and Vv.numel():
            raise ValueError("no layer is kept but Kv/Vv are not empty")
        return Kv, Vv
    nk, B, Hkv, Nv, hd = Kv.shape
    if (nk != nkeep or T != B * Nv or E.shape[1] != d or tuple(Uw.shape) != (L, d, r)
            or tuple(gamma.shape) != (L, d) or tuple(Wk.shape) != (L, Hkv * hd, d)
            or Wv.shape != Wk.shape or Vv.shape != Kv.shape):
        raise ValueError("shape mismatch in kept_visual_kv")
    code = _dtype_code(E, Dw, Uw, gamma, Wk, Wv, Kv, Vv)
    if ws is None:
        ws = _workspace(kept_visual_kv_workspace(T, d, r, nkeep, E.dtype), E.device, stream)
    keep_arr = (ctypes.c_uint8 * L).from_buffer_copy(flags)
    _check(load().dv_kept_visual_kv(_ptr(E), _ptr(Dw), _ptr(Uw), _ptr(gamma), _ptr(Wk), _ptr(Wv),
                                    ctypes.cast(keep_arr, ctypes.c_void_p), _ptr(Kv), _ptr(Vv), B,
                                    Nv, d, L, r, Hkv, hd, act, float(eps), code, _ptr(ws),
                                    ws.numel(), _stream(E.device, stream)))
    return Kv, Vv


def delta_rule_workspace(B: int, Hv: int, N: int, dk: int, dv: int, dtype: torch.dtype) -> int:
    code = DV_BF16 if dtype == torch.bfloat16 else DV_F32
    return int(load().dv_delta_rule_workspace(B, Hv, N, dk, dv, code))


def delta_rule_write(k, v, alpha, beta, S, ws: Optional[torch.Tensor] = None, stream=None):
    """Gated delta-rule write of N tokens into the fp32 state S [B,Hv,dk,dv] in place.
    k [B,Hk,N,dk], v [B,Hv,N,dv] (call dtype); alpha, beta [B,Hv,N] fp32."""
    B, Hk, N, dk = k.shape
    Hv, dv = v.shape[1], v.shape[3]
    if (tuple(v.shape) != (B, Hv, N, dv) or tuple(alpha.shape) != (B, Hv, N)
            or beta.shape != alpha.shape or tuple(S.shape) != (B, Hv, dk, dv)):
        raise ValueError("shape mismatch in delta_rule_write")
    if alpha.dtype != torch.float32 or beta.dtype != torch.float32 or S.dtype != torch.float32:
        raise ValueError("alpha, beta and S must be float32")
    for t in (alpha, beta, S):
        if not t.is_contiguous() or t.device.type != "cuda":
            raise ValueError("alpha, beta and S must be contiguous device tensors")
    code = _dtype_code(k, v)
    if ws is None:
        ws = _workspace(delta_rule_workspace(B, Hv, N, dk, dv, k.dtype), k.device, stream)
    _check(load().dv_delta_rule_write(_ptr(k), _ptr(v), alpha.data_ptr(), beta.data_ptr(),
                                      S.data_ptr(), B, Hk, Hv, N, dk, dv, code, _ptr(ws),
                                      ws.numel(), _stream(k.device, stream)))
    return S


def text_visual_attention_workspace(B: int, Hq: int, Hkv: int, hd: int, Nv: int, Nq: int,
                                    Nkt: int) -> int:
    return int(load().dv_text_visual_attention_workspace(B, Hq, Hkv, hd, Nv, Nq, Nkt))


def text_visual_attention(Q, Kv, Vv, Kt, Vt, O, q_pos0: int = 0, scale: Optional[float] = None,
                          ws: Optional[torch.Tensor] = None, stream=None):
    """One layer of Eq. 9. Q, O [B,Nq,Hq,hd]; Kv, Vv [B,Hkv,Nv,hd]; Kt, Vt [B,Hkv,Nkt,hd]."""
    B, Nq, Hq, hd = Q.shape
    _, Hkv, Nkt, _ = Kt.shape
    if Kv is None or Vv is None:  # a layer without visual keys (skipped adapter)
        if Kv is not None or Vv is not None:
            raise ValueError("Kv and Vv must both be given or both be None")
        Kv = Vv = Q.new_empty((B, Hkv, 0, hd))
    Nv = Kv.shape[2]
    if (tuple(Kv.shape) != (B, Hkv, Nv, hd) or Vv.shape != Kv.shape or Vt.shape != Kt.shape
            or Kt.shape[0] != B or Kt.shape[3] != hd or O.shape != Q.shape):
        raise ValueError("shape mismatch in text_visual_attention")
    code = _dtype_code(Q, Kv, Vv, Kt, Vt, O)
    if scale is None:
        scale = hd ** -0.5
    if ws is None:
        n = text_visual_attention_workspace(B, Hq, Hkv, hd, Nv, Nq, Nkt)
        ws = _workspace(n, Q.device, stream) if n else None
    kvp = _ptr(Kv) if Nv > 0 else None
    vvp = _ptr(Vv) if Nv > 0 else None
    _check(load().dv_text_visual_attention(_ptr(Q), kvp, vvp, _ptr(Kt), _ptr(Vt), _ptr(O), B, Hq,
                                           Hkv, hd, Nv, Nq, Nkt, q_pos0, float(scale), code,
                                           _ptr(ws) if ws is not None else None,
                                           ws.numel() if ws is not None else 0,
                                           _stream(Q.device, stream)))
    return O


ATTENTION_SCRATCH_BYTES = 32 << 20  # DV_ATTENTION_SCRATCH_BYTES


def text_visual_attention_noalloc(Q, Kv, Vv, Kt, Vt, O, q_pos0: int = 0,
                                  scale: Optional[float] = None, stream=None):
    """text_visual_attention without a workspace: the key-split partials live in the library's
    static per-GPU scratch, so the call allocates nothing. Calls that may overlap on one GPU
    share that scratch and must be serialised by the caller."""
    B, Nq, Hq, hd = Q.shape
    _, Hkv, Nkt, _ = Kt.shape
    if Kv is None or Vv is None:
        if Kv is not None or Vv is not None:
            raise ValueError("Kv and Vv must both be given or both be None")
        Nv = 0
    else:
        Nv = Kv.shape[2]
        if tuple(Kv.shape) != (B, Hkv, Nv, hd) or Vv.shape != Kv.shape:
            raise ValueError("shape mismatch in text_visual_attention_noalloc")
    if (Vt.shape != Kt.shape or Kt.shape[0] != B or Kt.shape[3] != hd or O.shape != Q.shape):
        raise ValueError("shape mismatch in text_visual_attention_noalloc")
    code = _dtype_code(*[t for t in (Q, Kv, Vv, Kt, Vt, O) if t is not None])
    if scale is None:
        scale = hd ** -0.5
    _check(load().dv_text_visual_attention_noalloc(
        _ptr(Q), _ptr(Kv) if Nv > 0 else None, _ptr(Vv) if Nv > 0 else None, _ptr(Kt), _ptr(Vt),
        _ptr(O), B, Hq, Hkv, hd, Nv, Nq, Nkt, q_pos0, float(scale), code,
        _stream(Q.device, stream)))
    return O
