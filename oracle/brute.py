"""Brute-force references used to pin the oracle (TEST INFRASTRUCTURE ONLY).

These evaluate the *vanilla* decoder layer the method starts from (Section 2,
Eq. 2: hidden states [V_l; T_l], visual first) with textbook numpy
expressions, independent of ``dvref.c``:

* ``full_layer_attention``: every position of [visual; text] is a query of
  ordinary causal self-attention over the whole sequence, with RMSNorm and the
  Q/K/V projections of one layer. With a zero up-projection (U_l = 0, the
  identity initialisation of Section 3.1) the method's memory equals E, so the
  text rows of this vanilla first layer must equal the method's Eq. 9 output.
* ``rank`` helpers for the low-rank property stated after Eq. 4.
"""
from __future__ import annotations

import numpy as np


def rms_normalize(X: np.ndarray, gamma: np.ndarray, eps: float) -> np.ndarray:
    ms = np.mean(X * X, axis=-1, keepdims=True)
    return X / np.sqrt(ms + eps) * gamma


def full_layer_attention(X: np.ndarray, gamma: np.ndarray, Wq: np.ndarray, Wk: np.ndarray,
                         Wv: np.ndarray, Hq: int, Hkv: int, hd: int, eps: float,
                         scale: float) -> np.ndarray:
    """Causal self-attention of a whole [visual; text] sequence.

    X [B,N,d]; Wq [Hq*hd,d]; Wk, Wv [Hkv*hd,d]. Returns the attention output of
    every position, [B,N,Hq,hd]. Query head h uses key/value head h // (Hq/Hkv)."""
    B, N, d = X.shape
    G = Hq // Hkv
    Xn = rms_normalize(X, gamma, eps)
    q = (Xn @ Wq.T).reshape(B, N, Hq, hd)
    k = (Xn @ Wk.T).reshape(B, N, Hkv, hd)
    v = (Xn @ Wv.T).reshape(B, N, Hkv, hd)
    future = np.triu(np.ones((N, N), dtype=bool), k=1)
    out = np.empty((B, N, Hq, hd))
    for b in range(B):
        for h in range(Hq):
            g = h // G
            s = (q[b, :, h, :] @ k[b, :, g, :].T) * scale
            s[future] = -np.inf
            s = s - s.max(axis=1, keepdims=True)
            p = np.exp(s)
            p /= p.sum(axis=1, keepdims=True)
            out[b, :, h, :] = p @ v[b, :, g, :]
    return out


def singular_values(A: np.ndarray) -> np.ndarray:
    return np.linalg.svd(np.asarray(A, dtype=np.float64), compute_uv=False)


def row_space_residual(Delta: np.ndarray, U: np.ndarray) -> float:
    """max |Delta - Delta P| where P projects onto the row space of U ([r,d])."""
    P = np.linalg.pinv(U) @ U
    return float(np.max(np.abs(Delta - Delta @ P)))
