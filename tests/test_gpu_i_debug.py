"""DV_DEBUG: with the variable set, every call waits for its kernels and checks them; results
are the same bits as without it (through the C ABI, every entry point with kernels)."""
import pytest
import torch

import paper_2609_34972_amd as dvl
from paper_2609_34972_amd import configs, synth
from tests.gpu_helpers import cuda, say

pytestmark = pytest.mark.gpu


def run_all():
    w = configs.LLAVA7B.with_(name="dbg", L=2, B=1, Nv=100, Nt=16, outlier_channels=())
    E, wts, tx = synth.make_E(w, 4), synth.make_build_weights(w, 4), synth.make_text(w, 4)
    Eg, wg, tg = cuda(E), {k: cuda(v) for k, v in wts.items()}, {k: cuda(v) for k, v in tx.items()}
    out = {}
    Z = torch.empty(w.L, w.T, w.r, dtype=Eg.dtype, device="cuda:0")
    dvl.build_visual_memory(Eg, wg["Dw"], Z, act=w.act)
    Kv = torch.empty(w.L, w.B, w.Hkv, w.Nv, w.hd, dtype=Eg.dtype, device="cuda:0")
    Vv = torch.empty_like(Kv)
    dvl.project_visual_kv(Eg, Z, wg["Uw"], wg["gamma"], wg["Wk"], wg["Wv"], Kv, Vv, eps=w.eps)
    O = torch.empty_like(tg["Q"][0])
    dvl.text_visual_attention(tg["Q"][0], Kv[0], Vv[0], tg["Kt"][0], tg["Vt"][0], O)
    O2 = torch.empty_like(O)
    dvl.text_visual_attention_noalloc(tg["Q"][1], Kv[1], Vv[1], tg["Kt"][1], tg["Vt"][1], O2)
    Kr, Vr = torch.empty_like(Kv), torch.empty_like(Vv)
    dvl.recurrent_visual_kv(Eg, wg["Dw"], wg["Uw"], wg["gamma"], wg["Wk"], wg["Wv"], Kr, Vr,
                            eps=w.eps, act=w.act)
    Kk, Vk = torch.empty_like(Kv[:1]), torch.empty_like(Vv[:1])
    dvl.kept_visual_kv(Eg, wg["Dw"], wg["Uw"], wg["gamma"], wg["Wk"], wg["Wv"], [0, 1], Kk, Vk,
                       eps=w.eps, act=w.act)
    dw = configs.GDN_IMAGE.with_(name="dbg_delta", B=1, Hk=2, Hv=4, N=130)
    x = {k: cuda(v) for k, v in synth.make_delta_inputs(dw, 2).items()}
    S = x["S"].clone()
    dvl.delta_rule_write(x["k"], x["v"], x["alpha"], x["beta"], S)
    torch.cuda.synchronize()
    return dict(Z=Z, Kv=Kv, Vv=Vv, O=O, O2=O2, Kr=Kr, Vr=Vr, Kk=Kk, Vk=Vk, S=S)


def test_debug_mode_gives_the_same_bits(monkeypatch):
    monkeypatch.delenv("DV_DEBUG", raising=False)
    ref = run_all()
    monkeypatch.setenv("DV_DEBUG", "1")
    say("[DV_DEBUG=1]")
    got = run_all()
    for k in ref:
        assert torch.equal(ref[k], got[k]), k
