"""GPU parity at the full workload sizes, in the launch configuration the benchmark times.

The whole batch runs on the GPU exactly as in the benchmark (all layers in one
call, the recommended workspace); the oracle then recomputes seeded samples of
the outputs one row or one (batch, kv-head) group at a time. Every output row
depends only on its own token (build) or its own group (attention), so the
sampled rows are complete checks of those outputs.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_34972_amd as dvl
from paper_2609_34972_amd import configs, synth
from tests.gpu_helpers import assert_close, cuda, f64, say

pytestmark = pytest.mark.gpu

BUILD_FULL = [configs.LLAVA7B, configs.QWEN25VL_VIDEO, configs.LLAVA_NEXT,
              # 8241 tokens: the down projection's 256 x 256 tiles with a ragged last row tile
              configs.LLAVA_NEXT.with_(name="next_ragged_tokens", B=3, Nv=2747)]
ATTN_FULL = [configs.LLAVA7B, configs.QWEN25VL_VIDEO, configs.LLAVA_NEXT, configs.DECODE]


_CACHE = {}


def build_inputs(w):
    """Seeded inputs of a workload; the LLaVA-7B ones are kept for the chained check."""
    if w.name in _CACHE:
        return _CACHE[w.name]
    E, wts = synth.make_E(w), synth.make_build_weights(w)
    if w.name == configs.LLAVA7B.name:
        _CACHE[w.name] = (E, wts)
    return E, wts


@pytest.mark.parametrize("w", BUILD_FULL, ids=lambda w: w.name)
def test_full_build_sampled(w):
    say(f"[full build {w.name}] generating inputs")
    E, wts = build_inputs(w)
    Eg = cuda(E)
    wg = {k: cuda(v) for k, v in wts.items()}
    dt = Eg.dtype
    say(f"[full build {w.name}] running on GPU")
    Z = torch.empty(w.L, w.T, w.r, dtype=dt, device="cuda:0")
    dvl.build_visual_memory(Eg, wg["Dw"], Z, act=w.act)
    Kv = torch.empty(w.L, w.B, w.Hkv, w.Nv, w.hd, dtype=dt, device="cuda:0")
    Vv = torch.empty_like(Kv)
    ws = torch.empty(dvl.project_visual_kv_workspace(w.T, w.d, w.L, dt), dtype=torch.uint8,
                     device="cuda:0")
    dvl.project_visual_kv(Eg, Z, wg["Uw"], wg["gamma"], wg["Wk"], wg["Wv"], Kv, Vv, eps=w.eps, ws=ws)
    torch.cuda.synchronize()
    del ws, wg
    rng = np.random.default_rng(1234)
    # Z: 256 sampled tokens and the last 8, every layer.
    rows = np.union1d(rng.choice(w.T, 256, replace=False), np.arange(w.T - 8, w.T))
    E64 = f64(E[torch.from_numpy(rows)])
    Zr = oracle.down(E64, f64(wts["Dw"]), w.act)
    Zg = f64(Z[:, torch.from_numpy(rows)])
    for l in range(w.L):
        assert_close(Zg[l], Zr[l], w.dtype, f"Z layer {l}")
    # Kv / Vv: 64 sampled tokens, layers 0, L-1 and two random ones.
    layers = sorted({0, w.L - 1, *rng.choice(np.arange(1, w.L - 1), 2, replace=False).tolist()})
    rows = np.union1d(rng.choice(w.T, 64, replace=False), np.arange(w.T - 4, w.T))
    E64 = f64(E[torch.from_numpy(rows)])
    li = torch.tensor(layers)
    say(f"[full build {w.name}] oracle on {len(rows)} rows x layers {layers}")
    Zl = oracle.down(E64, f64(wts["Dw"][li]), w.act)
    Kr, Vr = oracle.project_visual_kv(E64, Zl, f64(wts["Uw"][li]), f64(wts["gamma"][li]),
                                      f64(wts["Wk"][li]), f64(wts["Wv"][li]), 1, len(rows), w.Hkv,
                                      w.hd, w.eps)
    b_idx = torch.from_numpy(rows // w.Nv)
    i_idx = torch.from_numpy(rows % w.Nv)
    for n, l in enumerate(layers):
        kg = f64(Kv[l][b_idx, :, i_idx, :])   # [rows, Hkv, hd]
        vg = f64(Vv[l][b_idx, :, i_idx, :])
        ek = assert_close(kg, Kr[n, 0].transpose(1, 0, 2), w.dtype, f"Kv layer {l}")
        ev = assert_close(vg, Vr[n, 0].transpose(1, 0, 2), w.dtype, f"Vv layer {l}")
        say(f"  layer {l}: Kv {ek:.2e} Vv {ev:.2e}")


@pytest.mark.parametrize("w", ATTN_FULL, ids=lambda w: w.name)
def test_full_attention_sampled(w):
    say(f"[full attention {w.name}] generating inputs")
    tx = synth.make_text(w, layers=[0])
    vc = synth.make_visual_cache(w, layers=[0])
    x = {k: v[0] for k, v in {**tx, **vc}.items()}
    xg = {k: cuda(v) for k, v in x.items()}
    O = torch.empty_like(xg["Q"])
    n = dvl.text_visual_attention_workspace(w.B, w.Hq, w.Hkv, w.hd, w.Nv, w.Nq, w.Nkt)
    ws = torch.empty(max(n, 16), dtype=torch.uint8, device="cuda:0")
    say(f"[full attention {w.name}] running on GPU")
    dvl.text_visual_attention(xg["Q"], xg["Kv"], xg["Vv"], xg["Kt"], xg["Vt"], O, q_pos0=w.q_pos0,
                              ws=ws)
    torch.cuda.synchronize()
    rng = np.random.default_rng(99)
    G = w.G
    groups = [(int(b), int(g)) for b, g in zip(rng.integers(0, w.B, 4), rng.integers(0, w.Hkv, 4))]
    for b, g in groups:
        hs = slice(g * G, (g + 1) * G)
        ref = oracle.text_visual_attention(
            f64(x["Q"][b:b + 1, :, hs]), f64(x["Kv"][b:b + 1, g:g + 1]), f64(x["Vv"][b:b + 1, g:g + 1]),
            f64(x["Kt"][b:b + 1, g:g + 1]), f64(x["Vt"][b:b + 1, g:g + 1]), w.q_pos0)
        e = assert_close(f64(O[b:b + 1, :, hs]), ref, w.dtype, f"O batch {b} kv-head {g}")
        say(f"  (b={b}, g={g}): {e:.2e}")


def test_full_chain_llava7b():
    """The whole step at the LLaVA-7B size in the benchmark's launch configuration (all 32
    layers built and projected in one call each, then attention per layer), checked end to end:
    for 2 layers x 4 (batch, kv-head) groups the GPU's attention output is compared with the
    oracle's attention over the GPU's own visual K/V (the attention alone), and with the
    oracle's whole chain (memory, norm and K/V of that batch entry and head recomputed from E,
    then attention)."""
    w = configs.LLAVA7B
    say("[full chain llava7b] generating inputs")
    E, wts = build_inputs(w)
    layers = [0, w.L - 1]
    tx = synth.make_text(w, layers=layers)
    Eg = cuda(E)
    wg = {k: cuda(v) for k, v in wts.items()}
    dt = Eg.dtype
    say("[full chain llava7b] running on GPU")
    Z = torch.empty(w.L, w.T, w.r, dtype=dt, device="cuda:0")
    dvl.build_visual_memory(Eg, wg["Dw"], Z, act=w.act)
    Kv = torch.empty(w.L, w.B, w.Hkv, w.Nv, w.hd, dtype=dt, device="cuda:0")
    Vv = torch.empty_like(Kv)
    ws = torch.empty(dvl.project_visual_kv_workspace(w.T, w.d, w.L, dt), dtype=torch.uint8,
                     device="cuda:0")
    dvl.project_visual_kv(Eg, Z, wg["Uw"], wg["gamma"], wg["Wk"], wg["Wv"], Kv, Vv, eps=w.eps, ws=ws)
    n = dvl.text_visual_attention_workspace(w.B, w.Hq, w.Hkv, w.hd, w.Nv, w.Nq, w.Nkt)
    wsa = torch.empty(max(n, 16), dtype=torch.uint8, device="cuda:0")
    O = []
    for j, l in enumerate(layers):
        o = torch.empty(w.B, w.Nq, w.Hq, w.hd, dtype=dt, device="cuda:0")
        dvl.text_visual_attention(cuda(tx["Q"][j]), Kv[l], Vv[l], cuda(tx["Kt"][j]),
                                  cuda(tx["Vt"][j]), o, q_pos0=w.q_pos0, ws=wsa)
        O.append(o)
    torch.cuda.synchronize()
    del ws, wg, Z
    rng = np.random.default_rng(77)
    groups = [(int(b), int(g)) for b, g in zip(rng.integers(0, w.B, 4), rng.integers(0, w.Hkv, 4))]
    for j, l in enumerate(layers):
        for b, g in groups:
            hs, ks = slice(g * w.G, (g + 1) * w.G), slice(g * w.hd, (g + 1) * w.hd)
            Q64 = f64(tx["Q"][j][b:b + 1, :, hs])
            Kt64, Vt64 = f64(tx["Kt"][j][b:b + 1, g:g + 1]), f64(tx["Vt"][j][b:b + 1, g:g + 1])
            got = f64(O[j][b:b + 1, :, hs])
            iso = oracle.text_visual_attention(Q64, f64(Kv[l][b:b + 1, g:g + 1]),
                                               f64(Vv[l][b:b + 1, g:g + 1]), Kt64, Vt64, w.q_pos0)
            e1 = assert_close(got, iso, w.dtype, f"O layer {l} (b={b}, g={g}) on the GPU's K/V")
            E64 = f64(E[b * w.Nv:(b + 1) * w.Nv])
            Zr = oracle.down(E64, f64(wts["Dw"][l:l + 1]), w.act)
            Kr, Vr = oracle.project_visual_kv(E64, Zr, f64(wts["Uw"][l:l + 1]),
                                              f64(wts["gamma"][l:l + 1]),
                                              f64(wts["Wk"][l:l + 1, ks]),
                                              f64(wts["Wv"][l:l + 1, ks]), 1, w.Nv, 1, w.hd, w.eps)
            chain = oracle.text_visual_attention(Q64, Kr[0], Vr[0], Kt64, Vt64, w.q_pos0)
            e2 = assert_close(got, chain, w.dtype, f"O layer {l} (b={b}, g={g}) whole chain")
            say(f"  layer {l} (b={b}, g={g}): attention {e1:.2e}, chain {e2:.2e}")
    _CACHE.clear()
