"""The two kernels for M_l * gamma_l and the row sums of squares (Eq. 5 and the RMSNorm of
Eq. 7): the tiled one and the one that keeps a 128-row tile of Z_l in registers and walks all of
d. Both form the same products in the same order, so M_l * gamma_l must agree to the bit; the
row sums of squares are added up in another order, so K/V agree to rounding, and both meet the
oracle. Shapes cover ragged row tiles (T not a multiple of 128), a hidden size with a half column
tile (d = 960) and both ranks the Z-resident kernel takes."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_34972_amd as dvl
from paper_2609_34972_amd import configs, synth
from tests.gpu_helpers import assert_close, cuda, f64, say

pytestmark = pytest.mark.gpu

SHAPES = [
    configs.LLAVA7B.with_(name="r256_T300_d960", d=960, L=2, r=256, Hq=4, Hkv=2, hd=128, B=3,
                          Nv=100, outlier_channels=(211, 723)),
    configs.QWEN25VL_VIDEO.with_(name="r512_T129_d1024", d=1024, L=3, r=512, Hq=8, Hkv=4, hd=64,
                                 B=1, Nv=129, Nt=16),
]


def _run(w, Eg, Z, wg, mode):
    dvl.set_up_kernel(mode)
    assert dvl.project_visual_kv_up_kernel(w.T, w.d, w.r, w.L, torch.bfloat16) == mode
    Kv = torch.empty(w.L, w.B, w.Hkv, w.Nv, w.hd, dtype=torch.bfloat16, device="cuda:0")
    Vv = torch.empty_like(Kv)
    nbytes = dvl.project_visual_kv_workspace(w.T, w.d, w.L, torch.bfloat16)
    ws = torch.full((nbytes,), 0x7F, dtype=torch.uint8, device="cuda:0")
    dvl.project_visual_kv(Eg, Z, wg["Uw"], wg["gamma"], wg["Wk"], wg["Wv"], Kv, Vv, eps=w.eps,
                          ws=ws)
    torch.cuda.synchronize()
    Mg = ws[: w.L * w.T * w.d * 2].clone()  # M * gamma of every layer (one group)
    return Mg, Kv, Vv


@pytest.mark.parametrize("w", SHAPES, ids=lambda w: w.name)
def test_up_kernels_agree(w):
    say(f"[up kernels {w.name}]")
    E, wts = synth.make_E(w, 5), synth.make_build_weights(w, 5)
    Eg, wg = cuda(E), {k: cuda(v) for k, v in wts.items()}
    Z = torch.empty(w.L, w.T, w.r, dtype=torch.bfloat16, device="cuda:0")
    dvl.build_visual_memory(Eg, wg["Dw"], Z, act=w.act)
    try:
        Mt, Kt, Vt = _run(w, Eg, Z, wg, 1)
        Mz, Kz, Vz = _run(w, Eg, Z, wg, 2)
        Mz2, Kz2, _ = _run(w, Eg, Z, wg, 2)
    finally:
        dvl.set_up_kernel(0)
    assert torch.equal(Mz, Mt), "M * gamma differs between the kernels"
    assert torch.equal(Mz2, Mz) and torch.equal(Kz2, Kz), "Z-resident kernel not deterministic"
    Zr = oracle.down(f64(E), f64(wts["Dw"]), w.act)
    Kr, Vr = oracle.project_visual_kv(f64(E), f64(Z.cpu()), f64(wts["Uw"]), f64(wts["gamma"]),
                                      f64(wts["Wk"]), f64(wts["Wv"]), w.B, w.Nv, w.Hkv, w.hd, w.eps)
    assert_close(f64(Z), Zr, "bf16", "Z")
    for l in range(w.L):
        ek = assert_close(f64(Kz[l]), Kr[l], "bf16", f"Kv layer {l} (Z-resident)")
        ev = assert_close(f64(Vz[l]), Vr[l], "bf16", f"Vv layer {l} (Z-resident)")
        assert_close(f64(Kt[l]), Kr[l], "bf16", f"Kv layer {l} (tiled)")
        # the same M * gamma; only the order of the row sum of squares differs
        dk = float((Kz[l].float() - Kt[l].float()).abs().max() / Kt[l].float().abs().max())
        assert dk <= 1e-2, f"Kv layer {l}: kernels differ by {dk:.2e}"
        say(f"  layer {l}: Kv {ek:.2e} Vv {ev:.2e} kernels {dk:.1e}")
