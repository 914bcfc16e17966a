"""GPU parity of the recurrent adapter (Section 3.1, Eq. 6) followed by Eq. 7, through the C ABI.

The oracle runs the recurrence in fp64 (dvref_memory_recurrent) and projects every layer's memory
to K/V. Tokens are independent along the recurrence, so full-size checks recompute sampled tokens
through all layers.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_34972_amd as dvl
from paper_2609_34972_amd import configs, synth
from tests.gpu_helpers import assert_close, cuda, f64, say

pytestmark = pytest.mark.gpu


def run_rec(w, E, wts):
    Eg, wg = cuda(E), {k: cuda(v) for k, v in wts.items()}
    Kv = torch.empty(w.L, w.B, w.Hkv, w.Nv, w.hd, dtype=Eg.dtype, device="cuda:0")
    Vv = torch.empty_like(Kv)
    dvl.recurrent_visual_kv(Eg, wg["Dw"], wg["Uw"], wg["gamma"], wg["Wk"], wg["Wv"], Kv, Vv,
                            eps=w.eps, act=w.act)
    torch.cuda.synchronize()
    return Kv, Vv


CASES = [
    configs.TINY,
    configs.TINY.with_(name="tiny_silu", act=configs.ACT_SILU),
    configs.LLAVA7B.with_(name="rec_mid_llava", L=4, B=3, Nv=100),
    configs.QWEN25VL_VIDEO.with_(name="rec_mid_gqa_hd64", d=960, L=3, r=64, Hq=8, Hkv=2, hd=64,
                                 B=3, Nv=37),
]


@pytest.mark.parametrize("w", CASES, ids=lambda w: w.name)
def test_recurrent_full_compare(w):
    say(f"[recurrent {w.name}]")
    E, wts = synth.make_E(w, 5), synth.make_build_weights(w, 5)
    Kv, Vv = run_rec(w, E, wts)
    M = oracle.memory_recurrent(f64(E), f64(wts["Dw"]), f64(wts["Uw"]), w.act)
    Kr, Vr = oracle.visual_kv(M, f64(wts["gamma"]), f64(wts["Wk"]), f64(wts["Wv"]), w.B, w.Nv,
                              w.Hkv, w.hd, w.eps)
    for l in range(w.L):
        ek = assert_close(f64(Kv[l]), Kr[l], w.dtype, f"Kv layer {l}")
        ev = assert_close(f64(Vv[l]), Vr[l], w.dtype, f"Vv layer {l}")
        say(f"  layer {l}: Kv {ek:.2e} Vv {ev:.2e}")


def test_recurrent_first_layer_equals_embedding():
    """Eq. 5 and Eq. 6 give the same first-layer memory, hence the same layer-0 K/V."""
    w = CASES[2]
    E, wts = synth.make_E(w, 6), synth.make_build_weights(w, 6)
    Kr, Vr = run_rec(w, E, wts)
    Eg, wg = cuda(E), {k: cuda(v) for k, v in wts.items()}
    Z = torch.empty(w.L, w.T, w.r, dtype=Eg.dtype, device="cuda:0")
    dvl.build_visual_memory(Eg, wg["Dw"], Z, act=w.act)
    Ke = torch.empty_like(Kr)
    Ve = torch.empty_like(Vr)
    dvl.project_visual_kv(Eg, Z, wg["Uw"], wg["gamma"], wg["Wk"], wg["Wv"], Ke, Ve, eps=w.eps)
    torch.cuda.synchronize()
    assert_close(f64(Kr[0]), f64(Ke[0]), "bf16", "layer-0 K, recurrent vs embedding")
    assert float((Kr[1].float() - Ke[1].float()).abs().max()) > 1e-2  # they differ afterwards


def test_recurrent_full_llava7b_sampled():
    w = configs.LLAVA7B
    say("[recurrent llava7b full] generating inputs")
    E, wts = synth.make_E(w), synth.make_build_weights(w)
    Kv, Vv = run_rec(w, E, wts)
    rng = np.random.default_rng(77)
    rows = np.sort(rng.choice(w.T, 32, replace=False))
    M = oracle.memory_recurrent(f64(E[torch.from_numpy(rows)]), f64(wts["Dw"]), f64(wts["Uw"]),
                                w.act)
    layers = [0, 7, 19, w.L - 1]
    li = torch.tensor(layers)
    Kr, Vr = oracle.visual_kv(M[layers], f64(wts["gamma"][li]), f64(wts["Wk"][li]),
                              f64(wts["Wv"][li]), 1, len(rows), w.Hkv, w.hd, w.eps)
    b_idx, i_idx = torch.from_numpy(rows // w.Nv), torch.from_numpy(rows % w.Nv)
    for n, l in enumerate(layers):
        ek = assert_close(f64(Kv[l][b_idx, :, i_idx, :]), Kr[n, 0].transpose(1, 0, 2), "bf16", f"Kv {l}")
        ev = assert_close(f64(Vv[l][b_idx, :, i_idx, :]), Vr[n, 0].transpose(1, 0, 2), "bf16", f"Vv {l}")
        say(f"  layer {l}: Kv {ek:.2e} Vv {ev:.2e}")
