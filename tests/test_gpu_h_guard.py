"""Canary guards around every output and workspace of the C ABI.

Each output, in/out state and workspace lives in the middle of a larger device buffer whose two
4 KiB margins hold a seeded random byte pattern; the workspaces are exactly the size the library
asks for and start out filled with random bytes (so a kernel that relied on cleared scratch would
show it). The calls run on ragged shapes (token counts and key counts that leave partial tiles),
then the margins must hold their pattern byte for byte and the outputs must still match the
oracle: no kernel stores outside the extent the boundary declares.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2609_34972_amd as dvl
from paper_2609_34972_amd import configs, synth
from tests.gpu_helpers import assert_close, cuda, f64, say

pytestmark = pytest.mark.gpu

MARGIN = 4096  # bytes on each side; keeps the tensor 256-byte aligned


class Guarded:
    """A device tensor of `shape`/`dtype` between two margins of random bytes."""

    def __init__(self, shape, dtype, seed, init=None):
        esize = torch.empty(0, dtype=dtype).element_size()
        self.nbytes = int(math.prod(shape)) * esize
        total = 2 * MARGIN + (self.nbytes + 255) // 256 * 256
        g = torch.Generator().manual_seed(seed)
        self.pattern = torch.randint(0, 256, (total,), generator=g, dtype=torch.uint8)
        self.buf = self.pattern.to("cuda:0")
        self.t = self.buf[MARGIN:MARGIN + self.nbytes].view(dtype).view(*shape)
        if init is not None:
            self.t.copy_(init.to(self.t.device))

    def check(self, what):
        host = self.buf.cpu()
        lo = torch.equal(host[:MARGIN], self.pattern[:MARGIN])
        hi = torch.equal(host[MARGIN + self.nbytes:], self.pattern[MARGIN + self.nbytes:])
        assert lo and hi, f"{what}: a store landed outside the tensor ({'before' if not lo else 'after'} it)"


def guarded_ws(nbytes, seed):
    return Guarded((max(int(nbytes), 16),), torch.uint8, seed)


BUILD = [
    # one ragged row tile of tokens (T = 100), LLaVA dimensions
    configs.LLAVA7B.with_(name="g_llava_T100", L=2, B=1, Nv=100, outlier_channels=()),
    # GQA, hd 64, d not a multiple of the column tile, 3 x 37 tokens
    configs.QWEN25VL_VIDEO.with_(name="g_gqa_hd64", d=960, L=3, r=64, Hq=8, Hkv=2, hd=64, B=3,
                                 Nv=37, Nt=16),
    # K/V width 1024, rank 128, 100 tokens: ragged row tiles (run with the fused kernel too)
    configs.QWEN25VL_VIDEO.with_(name="g_fused_r128", d=320, L=2, r=128, B=1, Nv=100),
    # fp32 engine
    configs.TINY.with_(name="g_f32", d=320, L=3, r=48, Hq=6, Hkv=3, hd=128, B=2, Nv=35,
                       act=configs.ACT_SILU),
    # the Z-resident up projection (forced): ragged rows, a half column tile (d = 960), r = 256
    # and r = 512
    configs.LLAVA7B.with_(name="g_zr_r256", d=960, L=2, r=256, Hq=4, Hkv=2, hd=128, B=1, Nv=100,
                          outlier_channels=(211, 723)),
    configs.QWEN25VL_VIDEO.with_(name="g_zr_r512", d=1024, L=2, r=512, Hq=8, Hkv=4, hd=64, B=3,
                                 Nv=37, Nt=16),
]


@pytest.mark.parametrize("w", BUILD, ids=lambda w: w.name)
def test_build_and_projection_stay_inside(w):
    say(f"[guard build {w.name}]")
    fused = w.name.startswith("g_fused")
    dvl.set_fused_kv(fused)
    dvl.set_up_kernel(2 if w.name.startswith("g_zr") else 0)
    try:
        if w.name.startswith("g_zr"):
            assert dvl.project_visual_kv_up_kernel(w.T, w.d, w.r, w.L, torch.bfloat16) == 2
        _build_and_projection(w)
    finally:
        dvl.set_fused_kv(False)
        dvl.set_up_kernel(0)


def _build_and_projection(w):
    E, wts = synth.make_E(w, 9), synth.make_build_weights(w, 9)
    Eg, wg = cuda(E), {k: cuda(v) for k, v in wts.items()}
    dt = Eg.dtype
    Z = Guarded((w.L, w.T, w.r), dt, 1)
    Kv, Vv = Guarded((w.L, w.B, w.Hkv, w.Nv, w.hd), dt, 2), Guarded((w.L, w.B, w.Hkv, w.Nv, w.hd), dt, 3)
    ws = guarded_ws(dvl.project_visual_kv_workspace(w.T, w.d, w.L, dt), 4)
    dvl.build_visual_memory(Eg, wg["Dw"], Z.t, act=w.act)
    dvl.project_visual_kv(Eg, Z.t, wg["Uw"], wg["gamma"], wg["Wk"], wg["Wv"], Kv.t, Vv.t, eps=w.eps,
                          ws=ws.t)
    torch.cuda.synchronize()
    for g, n in ((Z, "Z"), (Kv, "Kv"), (Vv, "Vv"), (ws, "projection workspace")):
        g.check(n)
    Zr = oracle.down(f64(E), f64(wts["Dw"]), w.act)
    Kr, Vr = oracle.project_visual_kv(f64(E), Zr, f64(wts["Uw"]), f64(wts["gamma"]), f64(wts["Wk"]),
                                      f64(wts["Wv"]), w.B, w.Nv, w.Hkv, w.hd, w.eps)
    for l in range(w.L):
        assert_close(f64(Z.t[l]), Zr[l], w.dtype, f"Z layer {l}")
        assert_close(f64(Kv.t[l]), Kr[l], w.dtype, f"Kv layer {l}")
        assert_close(f64(Vv.t[l]), Vr[l], w.dtype, f"Vv layer {l}")


def test_epilogue_recurrent_and_kept_stay_inside():
    w = BUILD[1]
    say(f"[guard epilogue / recurrent / kept {w.name}]")
    E, wts = synth.make_E(w, 10), synth.make_build_weights(w, 10)
    Eg, wg = cuda(E), {k: cuda(v) for k, v in wts.items()}
    dt = Eg.dtype
    shape = (w.L, w.B, w.Hkv, w.Nv, w.hd)
    # projection with the backbone epilogue (its workspace also holds the rotary table)
    ew = {k: cuda(v) for k, v in synth.make_epilogue_weights(w, 10).items()}
    epi = dvl.KVEpilogue(k_bias=ew["k_bias"], v_bias=ew["v_bias"], k_norm=ew["k_norm"],
                         positions=cuda(synth.image_positions(w.B, w.Nv, 3)))
    Z = torch.empty(w.L, w.T, w.r, dtype=dt, device="cuda:0")
    dvl.build_visual_memory(Eg, wg["Dw"], Z, act=w.act)
    Kv, Vv = Guarded(shape, dt, 11), Guarded(shape, dt, 12)
    ws = guarded_ws(dvl.project_visual_kv_ex_workspace(w.T, w.d, w.L, w.hd, dt), 13)
    dvl.project_visual_kv(Eg, Z, wg["Uw"], wg["gamma"], wg["Wk"], wg["Wv"], Kv.t, Vv.t, eps=w.eps,
                          ws=ws.t, epilogue=epi)
    torch.cuda.synchronize()
    for g, n in ((Kv, "Kv (epilogue)"), (Vv, "Vv (epilogue)"), (ws, "epilogue workspace")):
        g.check(n)
    # recurrent adapter
    Kv, Vv = Guarded(shape, dt, 14), Guarded(shape, dt, 15)
    ws = guarded_ws(dvl.recurrent_visual_kv_workspace(w.T, w.d, w.L, w.r, dt), 16)
    dvl.recurrent_visual_kv(Eg, wg["Dw"], wg["Uw"], wg["gamma"], wg["Wk"], wg["Wv"], Kv.t, Vv.t,
                            eps=w.eps, act=w.act, ws=ws.t)
    torch.cuda.synchronize()
    for g, n in ((Kv, "Kv (recurrent)"), (Vv, "Vv (recurrent)"), (ws, "recurrent workspace")):
        g.check(n)
    M = oracle.memory_recurrent(f64(E), f64(wts["Dw"]), f64(wts["Uw"]), w.act)
    Kr, _ = oracle.visual_kv(M, f64(wts["gamma"]), f64(wts["Wk"]), f64(wts["Wv"]), w.B, w.Nv,
                             w.Hkv, w.hd, w.eps)
    for l in range(w.L):
        assert_close(f64(Kv.t[l]), Kr[l], w.dtype, f"recurrent Kv layer {l}")
    # layer skipping (layers 0 and 2 kept)
    keep = [1, 0, 1]
    kshape = (2, w.B, w.Hkv, w.Nv, w.hd)
    Kv, Vv = Guarded(kshape, dt, 17), Guarded(kshape, dt, 18)
    ws = guarded_ws(dvl.kept_visual_kv_workspace(w.T, w.d, w.r, 2, dt), 19)
    dvl.kept_visual_kv(Eg, wg["Dw"], wg["Uw"], wg["gamma"], wg["Wk"], wg["Wv"], keep, Kv.t, Vv.t,
                       eps=w.eps, act=w.act, ws=ws.t)
    torch.cuda.synchronize()
    for g, n in ((Kv, "Kv (kept)"), (Vv, "Vv (kept)"), (ws, "kept workspace")):
        g.check(n)


ATTN = [
    # name, dtype, B, Hq, Hkv, hd, Nv, Nq, Nkt, q_pos0
    ("hd64_bf16", "bf16", 2, 8, 2, 64, 577, 7, 20, 13),
    ("hd128_ksplit", "bf16", 3, 4, 4, 128, 577, 16, 16, 0),
    ("hd128_stream", "bf16", 1, 28, 4, 128, 577, 33, 40, 7),
    ("decode_bf16", "bf16", 5, 8, 8, 128, 577, 1, 33, 32),
    ("hd64_f32", "f32", 2, 6, 3, 64, 577, 5, 9, 4),
]


@pytest.mark.parametrize("spec", ATTN, ids=[a[0] for a in ATTN])
def test_attention_stays_inside(spec):
    name, dt, B, Hq, Hkv, hd, Nv, Nq, Nkt, q0 = spec
    say(f"[guard attention {name}]")
    tdt = torch.float32 if dt == "f32" else torch.bfloat16
    g = torch.Generator().manual_seed(21)
    mk = lambda *s: torch.randn(*s, generator=g).to(tdt)
    x = dict(Q=mk(B, Nq, Hq, hd), Kv=mk(B, Hkv, Nv, hd), Vv=mk(B, Hkv, Nv, hd),
             Kt=mk(B, Hkv, Nkt, hd), Vt=mk(B, Hkv, Nkt, hd))
    xg = {k: cuda(v) for k, v in x.items()}
    ref = oracle.text_visual_attention(*(f64(x[k]) for k in ("Q", "Kv", "Vv", "Kt", "Vt")), q0)
    n = dvl.text_visual_attention_workspace(B, Hq, Hkv, hd, Nv, Nq, Nkt)
    for split in (True, False):
        O = Guarded((B, Nq, Hq, hd), tdt, 22)
        ws = guarded_ws(n if split else 16, 23)
        dvl.text_visual_attention(xg["Q"], xg["Kv"], xg["Vv"], xg["Kt"], xg["Vt"], O.t, q_pos0=q0,
                                  ws=ws.t)
        torch.cuda.synchronize()
        O.check(f"O split={split}")
        ws.check(f"attention workspace split={split}")
        assert_close(f64(O.t), ref, dt, f"O {name} split={split}")


def test_delta_rule_stays_inside():
    w = configs.GDN_IMAGE.with_(name="g_delta", B=2, Hk=2, Hv=4, N=700)
    say(f"[guard delta rule {w.name}]")
    x = synth.make_delta_inputs(w, 3)
    xg = {k: cuda(v) for k, v in x.items()}
    S = Guarded(tuple(x["S"].shape), torch.float32, 31, init=x["S"])
    ws = guarded_ws(dvl.delta_rule_workspace(w.B, w.Hv, w.N, w.dk, w.dv, xg["k"].dtype), 32)
    dvl.delta_rule_write(xg["k"], xg["v"], xg["alpha"], xg["beta"], S.t, ws=ws.t)
    torch.cuda.synchronize()
    S.check("S")
    ws.check("delta-rule workspace")
    ref = oracle.delta_rule(f64(x["k"]), f64(x["v"]), f64(x["alpha"]), f64(x["beta"]), f64(x["S"]))
    assert_close(f64(S.t), ref, "bf16", "S")
