"""GPU parity of layer-wise adapter skipping (appendix on adapter skipping, Tables 14-15).

Kept layers run Eq. 4-5 and Eq. 7 into caches packed in layer order; skipped layers have no
visual keys and their attention is text-only (Eq. 18). Checked against the fp64 oracle with the
same keep mask, and bit for bit against the unskipped entry points on the kept layers.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_34972_amd as dvl
from paper_2609_34972_amd import configs, synth
from tests.gpu_helpers import assert_close, cuda, f64, say

pytestmark = pytest.mark.gpu


def run_kept(w, E, wts, keep):
    nk = sum(bool(k) for k in keep)
    Eg, wg = cuda(E), {k: cuda(v) for k, v in wts.items()}
    Kv = torch.empty(nk, w.B, w.Hkv, w.Nv, w.hd, dtype=Eg.dtype, device="cuda:0")
    Vv = torch.empty_like(Kv)
    dvl.kept_visual_kv(Eg, wg["Dw"], wg["Uw"], wg["gamma"], wg["Wk"], wg["Wv"], keep, Kv, Vv,
                       eps=w.eps, act=w.act)
    torch.cuda.synchronize()
    return Kv, Vv


def run_full(w, E, wts):
    Eg, wg = cuda(E), {k: cuda(v) for k, v in wts.items()}
    Z = torch.empty(w.L, w.T, w.r, dtype=Eg.dtype, device="cuda:0")
    dvl.build_visual_memory(Eg, wg["Dw"], Z, act=w.act)
    Kv = torch.empty(w.L, w.B, w.Hkv, w.Nv, w.hd, dtype=Eg.dtype, device="cuda:0")
    Vv = torch.empty_like(Kv)
    dvl.project_visual_kv(Eg, Z, wg["Uw"], wg["gamma"], wg["Wk"], wg["Wv"], Kv, Vv, eps=w.eps)
    torch.cuda.synchronize()
    return Kv, Vv


CASES = [
    (configs.TINY, (1, 0, 1, 1)),
    (configs.TINY.with_(name="tiny_silu", act=configs.ACT_SILU), (0, 1, 1, 0)),
    (configs.LLAVA7B.with_(name="skip_mid_llava", L=6, B=2, Nv=90), (0, 1, 1, 0, 1, 0)),
    (configs.QWEN25VL_VIDEO.with_(name="skip_mid_gqa", d=896, L=5, r=32, Hq=8, Hkv=2, hd=64, B=1,
                                  Nv=200, Nt=24), (1, 1, 0, 0, 1)),
]


@pytest.mark.parametrize("w,keep", CASES, ids=[c[0].name for c in CASES])
def test_skip_pipeline_against_oracle(w, keep):
    say(f"[skip {w.name} keep={keep}]")
    E, wts, tx = synth.make_E(w, 3), synth.make_build_weights(w, 3), synth.make_text(w, 3)
    Kv, Vv = run_kept(w, E, wts, keep)
    txg = {k: cuda(v) for k, v in tx.items()}
    slot = {l: j for j, l in enumerate(l for l in range(w.L) if keep[l])}
    O = torch.empty_like(txg["Q"])
    for l in range(w.L):
        j = slot.get(l)
        dvl.text_visual_attention(txg["Q"][l], Kv[j] if j is not None else None,
                                  Vv[j] if j is not None else None, txg["Kt"][l], txg["Vt"][l],
                                  O[l])
    torch.cuda.synchronize()
    _, Kr, Vr, Or = oracle.pipeline(f64(E), f64(wts["Dw"]), f64(wts["Uw"]), f64(wts["gamma"]),
                                    f64(wts["Wk"]), f64(wts["Wv"]), f64(tx["Q"]), f64(tx["Kt"]),
                                    f64(tx["Vt"]), w.B, w.Nv, w.Hkv, w.hd, w.eps, w.act, keep=keep)
    for j in range(len(slot)):
        assert_close(f64(Kv[j]), Kr[j], w.dtype, f"Kv slot {j}")
        assert_close(f64(Vv[j]), Vr[j], w.dtype, f"Vv slot {j}")
    for l in range(w.L):
        e = assert_close(f64(O[l]), Or[l], w.dtype, f"O layer {l}")
        say(f"  layer {l} {'kept' if l in slot else 'skipped'}: O err {e:.2e}")


@pytest.mark.parametrize("w,keep", CASES[2:], ids=[c[0].name for c in CASES[2:]])
def test_kept_layers_bit_identical_to_full_path(w, keep):
    E, wts = synth.make_E(w, 4), synth.make_build_weights(w, 4)
    Kv, Vv = run_kept(w, E, wts, keep)
    Kf, Vf = run_full(w, E, wts)
    kept = [l for l in range(w.L) if keep[l]]
    assert torch.equal(Kv, Kf[kept]) and torch.equal(Vv, Vf[kept])


def test_small_workspace_groups_layers_identically():
    w, keep = CASES[2]
    E, wts = synth.make_E(w, 8), synth.make_build_weights(w, 8)
    Kv, Vv = run_kept(w, E, wts, keep)
    Eg, wg = cuda(E), {k: cuda(v) for k, v in wts.items()}
    ws = torch.empty(dvl.kept_visual_kv_workspace(w.T, w.d, w.r, 1, Eg.dtype) + 3 * w.T * w.r * 2,
                     dtype=torch.uint8, device="cuda:0")  # Z for 3 layers + one projection slot
    K1, V1 = torch.empty_like(Kv), torch.empty_like(Vv)
    dvl.kept_visual_kv(Eg, wg["Dw"], wg["Uw"], wg["gamma"], wg["Wk"], wg["Wv"], keep, K1, V1,
                       eps=w.eps, act=w.act, ws=ws)
    torch.cuda.synchronize()
    assert torch.equal(K1, Kv) and torch.equal(V1, Vv)


def test_nothing_kept_and_everything_kept():
    w = CASES[2][0]
    E, wts = synth.make_E(w, 9), synth.make_build_weights(w, 9)
    assert dvl.kept_visual_kv(cuda(E), *[cuda(wts[k]) for k in ("Dw", "Uw", "gamma", "Wk", "Wv")],
                              [0] * w.L, None, None, eps=w.eps) == (None, None)
    Kv, Vv = run_kept(w, E, wts, [1] * w.L)
    Kf, Vf = run_full(w, E, wts)
    assert torch.equal(Kv, Kf) and torch.equal(Vv, Vf)


def test_skip_full_qwen_sampled():
    """The full video workload with the first 5 and last 10 adapters skipped (13 of 28 kept)."""
    w = configs.QWEN25VL_VIDEO
    keep = [0] * 5 + [1] * (w.L - 15) + [0] * 10
    say("[skip qwen full] generating inputs")
    E, wts = synth.make_E(w), synth.make_build_weights(w)
    Kv, Vv = run_kept(w, E, wts, keep)
    kept = [l for l in range(w.L) if keep[l]]
    rng = np.random.default_rng(41)
    rows = np.sort(rng.choice(w.T, 48, replace=False))
    for j in (0, len(kept) - 1):
        l = kept[j]
        Ef = f64(E[torch.from_numpy(rows)])
        Z = oracle.down(Ef, f64(wts["Dw"][l:l + 1]), w.act)
        M = oracle.memory(Ef, Z, f64(wts["Uw"][l:l + 1]))
        Kr, Vr = oracle.visual_kv(M, f64(wts["gamma"][l:l + 1]), f64(wts["Wk"][l:l + 1]),
                                  f64(wts["Wv"][l:l + 1]), 1, len(rows), w.Hkv, w.hd, w.eps)
        i_idx = torch.from_numpy(rows)  # B = 1
        ek = assert_close(f64(Kv[j][0][:, i_idx, :]), Kr[0, 0], "bf16", f"Kv layer {l}")
        ev = assert_close(f64(Vv[j][0][:, i_idx, :]), Vr[0, 0], "bf16", f"Vv layer {l}")
        say(f"  layer {l} (slot {j}): Kv {ek:.2e} Vv {ev:.2e}")
