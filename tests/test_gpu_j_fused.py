"""GPU parity of the fused up + RMSNorm + K/V kernel (Section 3.1 Eq. 4-5 with Section 3.2 Eq. 7).

With the kernel switched on, bf16 projections whose K/V width 2 Hkv hd is 1024 (the Qwen2.5-VL
shape: 4 K/V heads of 128) and whose rank is 128, 256 or 512 compute M_l on chip, 64 tokens per
block, and never write it out. Every case checks that the library reports the fused path for
its sizes and compares every output element with the fp64 oracle: row tiles with ragged tails,
a single partial tile, hidden sizes that are not multiples of 128, head dims 64 and 128,
outlier channels in E, layer sub-ranges, layer groups and the layer-skipping entry point. The
switch is restored to its default (off) after every test.
"""
import pytest
import torch

import oracle
import paper_2609_34972_amd as dvl
from paper_2609_34972_amd import configs, synth
from tests.gpu_helpers import assert_close, cuda, f64, say

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def fused_on():
    dvl.set_fused_kv(True)
    try:
        yield
    finally:
        dvl.set_fused_kv(False)


Q = configs.QWEN25VL_VIDEO
FUSED = [
    # rank 512 as in the Qwen video workload; 4 row tiles, the last with 8 tokens
    Q.with_(name="f_r512_hd128", d=512, L=3, r=512, B=2, Nv=100),
    # rank 512 with E's outlier channels scaled by 20 (the row norms then vary widely)
    Q.with_(name="f_r512_outliers", d=448, L=2, r=512, B=1, Nv=150, outlier_channels=(3, 77, 200),
            outlier_scale=20.0),
    # head dim 64 (8 K/V heads), rank 256, d = 6 chunks of 64
    Q.with_(name="f_r256_hd64", d=384, L=2, r=256, Hq=16, Hkv=8, hd=64, B=1, Nv=130),
    # rank 128, d = 3 chunks (not a multiple of 128), 63 tokens: one partial row tile
    Q.with_(name="f_r128_T63", d=192, L=2, r=128, B=3, Nv=21),
    # exactly one full row tile, GELU adapter
    Q.with_(name="f_r256_T64", d=256, L=2, r=256, B=1, Nv=64, act=configs.ACT_GELU),
]


def build(w, seed):
    E, wts = synth.make_E(w, seed), synth.make_build_weights(w, seed)
    Eg, wg = cuda(E), {k: cuda(v) for k, v in wts.items()}
    Z = torch.empty(w.L, w.T, w.r, dtype=Eg.dtype, device="cuda:0")
    dvl.build_visual_memory(Eg, wg["Dw"], Z, act=w.act)
    return E, wts, Eg, wg, Z


def project(w, Eg, wg, Z, l0=0, nl=None, ws_layers=None):
    nl = w.L if nl is None else nl
    Kv = torch.zeros(w.L, w.B, w.Hkv, w.Nv, w.hd, dtype=Eg.dtype, device="cuda:0")
    Vv = torch.zeros_like(Kv)
    ws = torch.empty(dvl.project_visual_kv_workspace(w.T, w.d, ws_layers or nl, Eg.dtype),
                     dtype=torch.uint8, device="cuda:0")
    dvl.project_visual_kv(Eg, Z, wg["Uw"], wg["gamma"], wg["Wk"], wg["Wv"], Kv, Vv, eps=w.eps,
                          l0=l0, nl=nl, ws=ws)
    return Kv, Vv


@pytest.mark.parametrize("w", FUSED, ids=lambda w: w.name)
def test_fused_projection_matches_oracle(w):
    say(f"[fused {w.name}]")
    assert dvl.project_visual_kv_fused(w.d, w.r, w.Hkv, w.hd, torch.bfloat16)
    E, wts, Eg, wg, Z = build(w, 4)
    Kv, Vv = project(w, Eg, wg, Z)
    torch.cuda.synchronize()
    Zr = oracle.down(f64(E), f64(wts["Dw"]), w.act)
    assert_close(f64(Z), Zr, "bf16", "Z")
    Kr, Vr = oracle.project_visual_kv(f64(E), Zr, f64(wts["Uw"]), f64(wts["gamma"]),
                                      f64(wts["Wk"]), f64(wts["Wv"]), w.B, w.Nv, w.Hkv, w.hd,
                                      w.eps)
    for l in range(w.L):
        ek = assert_close(f64(Kv[l]), Kr[l], "bf16", f"Kv layer {l}")
        ev = assert_close(f64(Vv[l]), Vr[l], "bf16", f"Vv layer {l}")
        say(f"  layer {l}: Kv {ek:.2e} Vv {ev:.2e}")


def test_fused_layer_ranges_and_groups():
    """A layer sub-range writes only its slots, with the bytes of the all-layer call; a workspace
    of one layer (layers in groups) gives the same bytes too."""
    w = FUSED[0]
    say(f"[fused ranges {w.name}]")
    _, _, Eg, wg, Z = build(w, 6)
    Kv, Vv = project(w, Eg, wg, Z)
    Kg, Vg = project(w, Eg, wg, Z, ws_layers=1)
    K1, V1 = project(w, Eg, wg, Z, l0=1, nl=2)
    torch.cuda.synchronize()
    assert torch.equal(Kv, Kg) and torch.equal(Vv, Vg)
    assert torch.equal(K1[1:], Kv[1:]) and torch.equal(V1[1:], Vv[1:])
    assert not K1[0].any() and not V1[0].any(), "a layer outside the range was written"


def test_fused_kept_layers_match_projection():
    """Layer skipping runs the same kernel on the kept layers: bit-identical K/V."""
    w = FUSED[2].with_(L=4)
    say(f"[fused kept {w.name}]")
    _, _, Eg, wg, Z = build(w, 8)
    Kv, Vv = project(w, Eg, wg, Z)
    keep = [1, 0, 1, 1]
    Kk = torch.empty(3, w.B, w.Hkv, w.Nv, w.hd, dtype=Eg.dtype, device="cuda:0")
    Vk = torch.empty_like(Kk)
    ws = torch.empty(dvl.kept_visual_kv_workspace(w.T, w.d, w.r, 3, Eg.dtype), dtype=torch.uint8,
                     device="cuda:0")
    dvl.kept_visual_kv(Eg, wg["Dw"], wg["Uw"], wg["gamma"], wg["Wk"], wg["Wv"], keep, Kk, Vk,
                       eps=w.eps, act=w.act, ws=ws)
    torch.cuda.synchronize()
    for j, l in enumerate([0, 2, 3]):
        assert torch.equal(Kk[j], Kv[l]) and torch.equal(Vk[j], Vv[l]), f"kept layer {l}"


def test_fused_and_two_kernel_paths_agree():
    """The same inputs through both paths: each matches the oracle, and they differ only by the
    rounding of their different summation orders."""
    w = FUSED[0].with_(L=2)
    say(f"[fused vs two-kernel {w.name}]")
    E, wts, Eg, wg, Z = build(w, 9)
    Kf, Vf = project(w, Eg, wg, Z)
    dvl.set_fused_kv(False)
    assert not dvl.project_visual_kv_fused(w.d, w.r, w.Hkv, w.hd, torch.bfloat16)
    Km, Vm = project(w, Eg, wg, Z)
    torch.cuda.synchronize()
    Kr, Vr = oracle.project_visual_kv(f64(E), oracle.down(f64(E), f64(wts["Dw"]), w.act),
                                      f64(wts["Uw"]), f64(wts["gamma"]), f64(wts["Wk"]),
                                      f64(wts["Wv"]), w.B, w.Nv, w.Hkv, w.hd, w.eps)
    for l in range(w.L):
        for x, ref, n in ((Kf, Kr, "fused Kv"), (Vf, Vr, "fused Vv"), (Km, Kr, "two-kernel Kv"),
                          (Vm, Vr, "two-kernel Vv")):
            assert_close(f64(x[l]), ref[l], "bf16", f"{n} layer {l}")
        assert_close(f64(Kf[l]), f64(Km[l]), "bf16", f"fused vs two-kernel Kv layer {l}")
