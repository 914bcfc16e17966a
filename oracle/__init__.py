"""Oracle of the visual-memory path (TEST INFRASTRUCTURE ONLY).

Plain fp64 CPU implementation of the paper's definitions (Section 3.1 Eq. 4-6,
Section 3.2 Eq. 7 and Eq. 9), in C (``dvref.c``) behind thin numpy wrappers,
plus a numpy brute-force full-layer evaluator (``brute.py``) used to pin it.
Only the tests, the smoke check and the benchmark's CPU-baseline leg may import
this package; the GPU library never does, and the two share no code.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "dvref.c")
_LIB_PATH = os.path.join(_HERE, "libdvref.so")
_lock = threading.Lock()
_lib = None

ACT_SILU = 0
ACT_GELU = 1


def build(force: bool = True) -> str:
    """Compile the C oracle with gcc (fp64, -O2, OpenMP over independent outputs)."""
    if not force and os.path.exists(_LIB_PATH) and os.path.getmtime(_LIB_PATH) >= os.path.getmtime(_SRC):
        return _LIB_PATH
    tmp = _LIB_PATH + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-O2", "-fno-fast-math", "-ffp-contract=off", "-fopenmp", "-shared", "-fPIC",
           "-std=c11", _SRC, "-o", tmp, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    with _lock:
        if _lib is not None:
            return _lib
        build(force=False)
        lib = ctypes.CDLL(_LIB_PATH)
        P = ctypes.POINTER(ctypes.c_double)
        i64, i32, f64 = ctypes.c_int64, ctypes.c_int, ctypes.c_double
        lib.dvref_act.argtypes = [f64, i32]
        lib.dvref_act.restype = f64
        lib.dvref_down.argtypes = [P, P, i64, i32, i32, i32, i32, P]
        lib.dvref_memory.argtypes = [P, P, P, i64, i32, i32, i32, P]
        lib.dvref_memory_recurrent.argtypes = [P, P, P, i64, i32, i32, i32, i32, P]
        lib.dvref_rmsnorm.argtypes = [P, P, i32, f64, P]
        lib.dvref_visual_kv.argtypes = [P, P, P, P, i32, i32, i32, i32, i32, i32, f64, P, P]
        lib.dvref_text_visual_attention.argtypes = [P, P, P, P, P, P] + [i32] * 8 + [f64]
        lib.dvref_text_visual_attention.restype = i32
        lib.dvref_kv_epilogue.argtypes = [P, P] + [i32] * 5 + [P, P, P, f64, ctypes.c_void_p] + [i32] * 3 + [f64]
        lib.dvref_kv_epilogue.restype = i32
        lib.dvref_delta_rule.argtypes = [P, P, P, P, P] + [i32] * 6
        lib.dvref_delta_rule.restype = i32
        _lib = lib
        return lib


def _c(a: np.ndarray) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float64)


def _p(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def act(x: float, kind: int) -> float:
    """phi of Eq. 4 (SiLU; exact erf GELU as the alternative)."""
    return _load().dvref_act(float(x), int(kind))


def down(X: np.ndarray, Dw: np.ndarray, act_kind: int) -> np.ndarray:
    """Eq. 4 down half for every layer: Z[l] = phi(X D_l), D_l = Dw[l]^T. X [T,d], Dw [L,r,d]."""
    X, Dw = _c(X), _c(Dw)
    T, d = X.shape
    L, r, d2 = Dw.shape
    assert d2 == d
    Z = np.empty((L, T, r))
    _load().dvref_down(_p(X), _p(Dw), T, d, L, r, int(act_kind), _p(Z))
    return Z


def memory(E: np.ndarray, Z: np.ndarray, Uw: np.ndarray) -> np.ndarray:
    """Eq. 4-5 embedding adapter: M_l = E + Z_l U_l, U_l = Uw[l]^T. Returns M [L,T,d]."""
    E, Z, Uw = _c(E), _c(Z), _c(Uw)
    T, d = E.shape
    L, T2, r = Z.shape
    assert T2 == T and Uw.shape == (L, d, r)
    M = np.empty((L, T, d))
    _load().dvref_memory(_p(E), _p(Z), _p(Uw), T, d, L, r, _p(M))
    return M


def memory_recurrent(E: np.ndarray, Dw: np.ndarray, Uw: np.ndarray, act_kind: int) -> np.ndarray:
    """Eq. 6 recurrent adapter: M_l = M_{l-1} + phi(M_{l-1} D_l) U_l with M_{-1} = E."""
    E, Dw, Uw = _c(E), _c(Dw), _c(Uw)
    T, d = E.shape
    L, r, _ = Dw.shape
    M = np.empty((L, T, d))
    _load().dvref_memory_recurrent(_p(E), _p(Dw), _p(Uw), T, d, L, r, int(act_kind), _p(M))
    return M


def rmsnorm(x: np.ndarray, gamma: np.ndarray, eps: float) -> np.ndarray:
    """LN_l read as RMSNorm, applied to each row of x [n,d]."""
    x, gamma = _c(np.atleast_2d(x)), _c(gamma)
    out = np.empty_like(x)
    lib = _load()
    for t in range(x.shape[0]):
        row = np.ascontiguousarray(x[t])
        o = np.empty_like(row)
        lib.dvref_rmsnorm(_p(row), _p(gamma), x.shape[1], float(eps), _p(o))
        out[t] = o
    return out


def visual_kv(M: np.ndarray, gamma: np.ndarray, Wk: np.ndarray, Wv: np.ndarray, B: int, Nv: int,
              Hkv: int, hd: int, eps: float):
    """Eq. 7: head-major Kv, Vv [L,B,Hkv,Nv,hd] from memories M [L,B*Nv,d]."""
    M, gamma, Wk, Wv = _c(M), _c(gamma), _c(Wk), _c(Wv)
    L, T, d = M.shape
    assert T == B * Nv and Wk.shape == (L, Hkv * hd, d) and Wv.shape == Wk.shape
    assert gamma.shape == (L, d)
    Kv = np.empty((L, B, Hkv, Nv, hd))
    Vv = np.empty((L, B, Hkv, Nv, hd))
    _load().dvref_visual_kv(_p(M), _p(gamma), _p(Wk), _p(Wv), B, Nv, d, L, Hkv, hd, float(eps),
                            _p(Kv), _p(Vv))
    return Kv, Vv


def text_visual_attention(Q: np.ndarray, Kv: np.ndarray, Vv: np.ndarray, Kt: np.ndarray,
                          Vt: np.ndarray, q_pos0: int, scale: Optional[float] = None) -> np.ndarray:
    """Eq. 9 for one layer. Q [B,Nq,Hq,hd], Kv/Vv [B,Hkv,Nv,hd], Kt/Vt [B,Hkv,Nkt,hd]."""
    Q, Kv, Vv, Kt, Vt = map(_c, (Q, Kv, Vv, Kt, Vt))
    B, Nq, Hq, hd = Q.shape
    _, Hkv, Nv, _ = Kv.shape
    Nkt = Kt.shape[2]
    if scale is None:
        scale = hd ** -0.5
    O = np.empty_like(Q)
    rc = _load().dvref_text_visual_attention(_p(Q), _p(Kv), _p(Vv), _p(Kt), _p(Vt), _p(O), B, Hq,
                                             Hkv, hd, Nv, Nq, Nkt, int(q_pos0), float(scale))
    if rc != 0:
        raise ValueError("invalid attention shape")
    return O


def kv_epilogue(Kv, Vv, k_bias=None, v_bias=None, k_norm=None, kn_eps: float = 1e-6, pos=None,
                sections=None, theta: float = 10000.0):
    """Backbone epilogue on visual K/V [L,B,Hkv,Nv,hd]: projection bias, per-head key RMSNorm
    and rotary embedding at the tokens' positions pos [B,3,Nv] with multimodal sections (the
    paper keeps visual positions unchanged, so the backbone's key treatment applies to them).
    Returns new arrays; None skips a step."""
    Kv, Vv = _c(Kv).copy(), _c(Vv).copy()
    L, B, Hkv, Nv, hd = Kv.shape
    sections = (hd // 2, 0, 0) if sections is None else tuple(int(x) for x in sections)
    posa = None
    if pos is not None:
        posa = np.ascontiguousarray(pos, dtype=np.int32)
        if posa.shape != (B, 3, Nv):
            raise ValueError("pos must be [B, 3, Nv]")
    extra = [None if a is None else _c(a) for a in (k_bias, v_bias, k_norm)]
    rc = _load().dvref_kv_epilogue(_p(Kv), _p(Vv), L, B, Hkv, Nv, hd,
                                   *[None if a is None else _p(a) for a in extra], float(kn_eps),
                                   None if posa is None else posa.ctypes.data, *sections,
                                   float(theta))
    if rc != 0:
        raise ValueError("rotary sections must add up to hd/2")
    return Kv, Vv


def delta_rule(k, v, alpha, beta, S):
    """Gated delta-rule write (appendix on linear attention, Eq. 15-16), token by token:
    S <- alpha_t S, then S <- S + beta_t k_t (v_t - S^T k_t)^T. k [B,Hk,N,dk], v [B,Hv,N,dv],
    alpha, beta [B,Hv,N], S [B,Hv,dk,dv]; value head h reads key head h // (Hv/Hk).
    Returns the final state (a new array)."""
    k, v, alpha, beta = _c(k), _c(v), _c(alpha), _c(beta)
    S = _c(S).copy()
    B, Hk, N, dk = k.shape
    Hv, dv = v.shape[1], v.shape[3]
    assert v.shape == (B, Hv, N, dv) and alpha.shape == (B, Hv, N) and beta.shape == alpha.shape
    assert S.shape == (B, Hv, dk, dv)
    if _load().dvref_delta_rule(_p(k), _p(v), _p(alpha), _p(beta), _p(S), B, Hk, Hv, N, dk, dv) != 0:
        raise ValueError("Hv must be a multiple of Hk")
    return S


def project_visual_kv(E, Z, Uw, gamma, Wk, Wv, B: int, Nv: int, Hkv: int, hd: int, eps: float):
    """Eq. 4-5 up half followed by Eq. 7, for every layer of the given weights."""
    M = memory(E, Z, Uw)
    return visual_kv(M, gamma, Wk, Wv, B, Nv, Hkv, hd, eps)


def pipeline(E, Dw, Uw, gamma, Wk, Wv, Q, Kt, Vt, B: int, Nv: int, Hkv: int, hd: int, eps: float,
             act_kind: int, q_pos0: int = 0, scale: Optional[float] = None, recurrent: bool = False,
             keep=None):
    """The whole path: memories (Eq. 5 or 6) -> visual K/V (Eq. 7) -> text attention (Eq. 9).

    Q, Kt, Vt carry a leading layer axis. Returns (Z or None, Kv, Vv, O).

    keep: optional per-layer flags for layer-wise adapter skipping (appendix on adapter
    skipping, Tables 14-15; defined there for the embedding adapter). A skipped layer has no
    visual memory, so its text queries attend to text keys only (Eq. 18). Z, Kv and Vv then
    hold the kept layers in layer order; O still has every layer."""
    L = Dw.shape[0]
    if keep is None:
        kept = list(range(L))
    else:
        if recurrent:
            raise ValueError("adapter skipping is defined for the embedding adapter only")
        if len(keep) != L:
            raise ValueError("keep needs one flag per layer")
        kept = [l for l in range(L) if keep[l]]
    if recurrent:
        Z = None
        M = memory_recurrent(E, Dw, Uw, act_kind)
    elif kept:
        Z = down(E, Dw[kept], act_kind)
        M = memory(E, Z, Uw[kept])
    else:
        Z = np.empty((0, E.shape[0], Dw.shape[1]))
        M = np.empty((0,) + E.shape)
    if kept:
        Kv, Vv = visual_kv(M, gamma[kept], Wk[kept], Wv[kept], B, Nv, Hkv, hd, eps)
    else:
        Kv = Vv = np.empty((0, B, Hkv, Nv, hd))
    slot = {l: j for j, l in enumerate(kept)}
    none = np.empty((B, Hkv, 0, hd))
    O = np.stack([text_visual_attention(Q[l], Kv[slot[l]] if l in slot else none,
                                        Vv[slot[l]] if l in slot else none, Kt[l], Vt[l], q_pos0,
                                        scale)
                  for l in range(L)])
    return Z, Kv, Vv, O
