"""GPU parity at sizes the oracle computes in full (every output element compared).

Shapes span several tiles with ragged tails; every call goes through the C ABI
of libdeltavision.so via the ctypes binding.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_34972_amd as dvl
from paper_2609_34972_amd import configs, synth
from tests.gpu_helpers import assert_close, cuda, f64, say

pytestmark = pytest.mark.gpu


def run_build(w, E, wts, act, ws_layers=None):
    T, L = w.T, w.L
    dt = E.dtype
    Z = torch.empty(L, T, w.r, dtype=dt, device="cuda:0")
    dvl.build_visual_memory(E, wts["Dw"], Z, act=act)
    Kv = torch.empty(L, w.B, w.Hkv, w.Nv, w.hd, dtype=dt, device="cuda:0")
    Vv = torch.empty_like(Kv)
    nl = L if ws_layers is None else ws_layers
    ws = torch.empty(dvl.project_visual_kv_workspace(T, w.d, nl, dt), dtype=torch.uint8,
                     device="cuda:0")
    dvl.project_visual_kv(E, Z, wts["Uw"], wts["gamma"], wts["Wk"], wts["Wv"], Kv, Vv, eps=w.eps,
                          ws=ws)
    return Z, Kv, Vv


def gen_build(w, seed=0):
    E = synth.make_E(w, seed)
    wts = synth.make_build_weights(w, seed)
    return E, wts


@pytest.mark.parametrize("act", [configs.ACT_GELU, configs.ACT_SILU])
def test_tiny_pipeline_f32(act):
    w = configs.TINY.with_(act=act)
    say(f"[tiny f32 act={act}]")
    E, wts = gen_build(w)
    tx = synth.make_text(w)
    Eg, wg, tg = cuda(E), {k: cuda(v) for k, v in wts.items()}, {k: cuda(v) for k, v in tx.items()}
    Z, Kv, Vv = run_build(w, Eg, wg, act)
    O = torch.empty_like(tg["Q"])
    for l in range(w.L):
        dvl.text_visual_attention(tg["Q"][l], Kv[l], Vv[l], tg["Kt"][l], tg["Vt"][l], O[l])
    torch.cuda.synchronize()
    Zr, Kr, Vr, Or = oracle.pipeline(f64(E), f64(wts["Dw"]), f64(wts["Uw"]), f64(wts["gamma"]),
                                     f64(wts["Wk"]), f64(wts["Wv"]), f64(tx["Q"]), f64(tx["Kt"]),
                                     f64(tx["Vt"]), w.B, w.Nv, w.Hkv, w.hd, w.eps, act)
    for l in range(w.L):
        assert_close(f64(Z[l]), Zr[l], "f32", f"Z layer {l}")
        assert_close(f64(Kv[l]), Kr[l], "f32", f"Kv layer {l}")
        assert_close(f64(Vv[l]), Vr[l], "f32", f"Vv layer {l}")
        assert_close(f64(O[l]), Or[l], "f32", f"O layer {l}")


MID = [
    # LLaVA-7B dims, 2 layers; T below one row tile and across three ragged tiles
    configs.LLAVA7B.with_(name="mid_llava_T100", L=2, B=1, Nv=100, outlier_channels=()),
    configs.LLAVA7B.with_(name="mid_llava_T300", L=2, B=3, Nv=100),
    # GQA, hd = 64, a hidden size that is not a multiple of the 128-column tile
    configs.QWEN25VL_VIDEO.with_(name="mid_gqa_hd64", d=960, L=3, r=64, Hq=8, Hkv=2, hd=64, B=3,
                                 Nv=37, Nt=16),
    # Few column tiles (2 kv x 4 heads x 128 = 4 tiles of 256) and many more rows than columns: the
    # projection deals its row tiles out to the XCDs; 12 row tiles, 4 of them past the first 8
    configs.QWEN25VL_VIDEO.with_(name="mid_rows_dealt", d=256, L=2, r=64, B=3, Nv=1000, Nt=16),
    # fp32 with several tiles in every dimension
    configs.TINY.with_(name="mid_f32", d=320, L=5, r=48, Hq=6, Hkv=3, hd=128, B=2, Nv=70,
                       act=configs.ACT_SILU),
]


@pytest.mark.parametrize("w", MID, ids=lambda w: w.name)
def test_mid_build(w):
    say(f"[mid build {w.name}]")
    E, wts = gen_build(w, seed=3)
    Eg, wg = cuda(E), {k: cuda(v) for k, v in wts.items()}
    Z, Kv, Vv = run_build(w, Eg, wg, w.act)
    torch.cuda.synchronize()
    Zr = oracle.down(f64(E), f64(wts["Dw"]), w.act)
    Kr, Vr = oracle.project_visual_kv(f64(E), Zr, f64(wts["Uw"]), f64(wts["gamma"]), f64(wts["Wk"]),
                                      f64(wts["Wv"]), w.B, w.Nv, w.Hkv, w.hd, w.eps)
    for l in range(w.L):
        assert_close(f64(Z[l]), Zr[l], w.dtype, f"Z layer {l}")
        ek = assert_close(f64(Kv[l]), Kr[l], w.dtype, f"Kv layer {l}")
        ev = assert_close(f64(Vv[l]), Vr[l], w.dtype, f"Vv layer {l}")
        say(f"  layer {l}: Kv {ek:.2e} Vv {ev:.2e}")


def test_project_kv_layer_groups_match_all_layers():
    """A workspace holding one layer (processed in groups) and a sub-range of layers give the
    same bytes as the all-layer call."""
    w = MID[1]
    E, wts = gen_build(w, seed=5)
    Eg, wg = cuda(E), {k: cuda(v) for k, v in wts.items()}
    Z, Kv, Vv = run_build(w, Eg, wg, w.act)
    _, Kv1, Vv1 = run_build(w, Eg, wg, w.act, ws_layers=1)
    Kv2 = torch.zeros_like(Kv)
    Vv2 = torch.zeros_like(Vv)
    ws = torch.empty(dvl.project_visual_kv_workspace(w.T, w.d, 1, Eg.dtype), dtype=torch.uint8,
                     device="cuda:0")
    dvl.project_visual_kv(Eg, Z, wg["Uw"], wg["gamma"], wg["Wk"], wg["Wv"], Kv2, Vv2, eps=w.eps,
                          l0=1, nl=1, ws=ws)
    torch.cuda.synchronize()
    assert torch.equal(Kv, Kv1) and torch.equal(Vv, Vv1)
    assert torch.equal(Kv2[1], Kv[1]) and torch.equal(Vv2[1], Vv[1])
    assert torch.count_nonzero(Kv2[0]) == 0  # layers outside the range are untouched


def test_down_192_row_tiles_ragged():
    """T = 2100 tokens against L * r = 4096 columns: 352 tiles of 192 x 128 fill one round of the
    512 two-per-CU slots, where 128 x 128 tiles would need two and 256 x 256 tiles two of 256,
    so the launch takes the 192-row tiles; the last row tile holds 180 rows."""
    w = configs.LLAVA7B.with_(name="mid_down192", d=256, L=16, r=256, Hq=2, Hkv=2, hd=64, B=3,
                              Nv=700, Nt=8, outlier_channels=(3, 200))
    say(f"[down 192-row tiles {w.name}: T {w.T} x N {w.L * w.r} x d {w.d}]")
    E, wts = gen_build(w, seed=13)
    Eg, Dg = cuda(E), cuda(wts["Dw"])
    Z = torch.empty(w.L, w.T, w.r, dtype=Eg.dtype, device="cuda:0")
    dvl.build_visual_memory(Eg, Dg, Z, act=w.act)
    torch.cuda.synchronize()
    Zr = oracle.down(f64(E), f64(wts["Dw"]), w.act)
    for l in range(w.L):
        assert_close(f64(Z[l]), Zr[l], w.dtype, f"Z layer {l}")


def test_project_kv_eleven_layers_in_runs_of_eight():
    """The tiled up projection takes up to eight layers per block: 11 layers run as blocks of 8
    and 3, the sub-range l0 = 2, nl = 9 as 8 and 1, and a one-layer workspace as single layers.
    All three give the same bytes, and the all-layer call matches the oracle layer by layer."""
    w = configs.LLAVA7B.with_(name="mid_eleven_layers", d=512, L=11, r=64, Hq=4, Hkv=4, hd=128,
                              B=2, Nv=150, Nt=8, outlier_channels=(7, 311))
    say(f"[eleven layers {w.name}: T {w.T}, d {w.d}, r {w.r}]")
    E, wts = gen_build(w, seed=9)
    Eg, wg = cuda(E), {k: cuda(v) for k, v in wts.items()}
    Z, Kv, Vv = run_build(w, Eg, wg, w.act)
    _, Kv1, Vv1 = run_build(w, Eg, wg, w.act, ws_layers=1)
    Kv2 = torch.zeros_like(Kv)
    Vv2 = torch.zeros_like(Vv)
    ws = torch.empty(dvl.project_visual_kv_workspace(w.T, w.d, 9, Eg.dtype), dtype=torch.uint8,
                     device="cuda:0")
    dvl.project_visual_kv(Eg, Z, wg["Uw"], wg["gamma"], wg["Wk"], wg["Wv"], Kv2, Vv2, eps=w.eps,
                          l0=2, nl=9, ws=ws)
    torch.cuda.synchronize()
    assert torch.equal(Kv, Kv1) and torch.equal(Vv, Vv1)
    assert torch.equal(Kv2[2:], Kv[2:]) and torch.equal(Vv2[2:], Vv[2:])
    assert torch.count_nonzero(Kv2[:2]) == 0 and torch.count_nonzero(Vv2[:2]) == 0
    Zr = oracle.down(f64(E), f64(wts["Dw"]), w.act)
    Kr, Vr = oracle.project_visual_kv(f64(E), Zr, f64(wts["Uw"]), f64(wts["gamma"]), f64(wts["Wk"]),
                                      f64(wts["Wv"]), w.B, w.Nv, w.Hkv, w.hd, w.eps)
    for l in range(w.L):
        assert_close(f64(Z[l]), Zr[l], w.dtype, f"Z layer {l}")
        assert_close(f64(Kv[l]), Kr[l], w.dtype, f"Kv layer {l}")
        assert_close(f64(Vv[l]), Vr[l], w.dtype, f"Vv layer {l}")


ATTN = [
    # name, dtype, B, Hq, Hkv, hd, Nv, Nq, Nkt, q_pos0
    ("llava_mha", "bf16", 2, 8, 8, 128, 577, 64, 64, 0),
    ("qwen_gqa", "bf16", 1, 28, 4, 128, 1000, 128, 128, 0),
    # 97-128 rows per kv-head: one ping-pong block (eight waves) per kv-head, non-temporal tiles
    ("next_mha_rows128", "bf16", 2, 8, 8, 128, 700, 128, 128, 0),
    ("ragged_rows100", "bf16", 2, 4, 2, 128, 333, 50, 50, 0),
    ("decode_mha", "bf16", 4, 32, 32, 128, 576, 1, 513, 512),
    ("decode_gqa", "bf16", 3, 28, 4, 128, 300, 1, 40, 39),
    ("chunked_hd64", "bf16", 2, 8, 2, 64, 130, 7, 20, 13),
    ("no_visual", "bf16", 2, 4, 4, 128, 0, 33, 33, 0),
    ("single_query_g16", "bf16", 2, 16, 1, 64, 200, 1, 10, 9),
    ("tiny_f32", "f32", 1, 4, 4, 64, 64, 16, 16, 0),
    ("gqa_f32_hd128", "f32", 2, 6, 2, 128, 90, 9, 12, 3),
    ("decode_f32", "f32", 5, 4, 4, 64, 33, 1, 7, 6),
]


def attn_inputs(spec, seed=11):
    name, dt, B, Hq, Hkv, hd, Nv, Nq, Nkt, q0 = spec
    g = torch.Generator().manual_seed(seed)
    tdt = torch.float32 if dt == "f32" else torch.bfloat16
    mk = lambda *s: torch.randn(*s, generator=g).to(tdt)
    return dict(Q=mk(B, Nq, Hq, hd), Kv=mk(B, Hkv, Nv, hd), Vv=mk(B, Hkv, Nv, hd),
                Kt=mk(B, Hkv, Nkt, hd), Vt=mk(B, Hkv, Nkt, hd))


@pytest.mark.parametrize("spec", ATTN, ids=[a[0] for a in ATTN])
@pytest.mark.parametrize("split", [True, False], ids=["ws", "nows"])
def test_attention(spec, split):
    name, dt, B, Hq, Hkv, hd, Nv, Nq, Nkt, q0 = spec
    say(f"[attention {name} split={split}]")
    x = attn_inputs(spec)
    xg = {k: cuda(v) for k, v in x.items()}
    O = torch.empty_like(xg["Q"])
    ws = None
    if split:
        n = dvl.text_visual_attention_workspace(B, Hq, Hkv, hd, Nv, Nq, Nkt)
        ws = torch.empty(max(n, 16), dtype=torch.uint8, device="cuda:0")
    else:
        ws = torch.empty(16, dtype=torch.uint8, device="cuda:0")  # too small: no split
    dvl.text_visual_attention(xg["Q"], xg["Kv"], xg["Vv"], xg["Kt"], xg["Vt"], O, q_pos0=q0, ws=ws)
    torch.cuda.synchronize()
    ref = oracle.text_visual_attention(f64(x["Q"]), f64(x["Kv"]), f64(x["Vv"]), f64(x["Kt"]),
                                       f64(x["Vt"]), q0)
    e = assert_close(f64(O), ref, dt, f"O {name}")
    say(f"  err {e:.2e}")


def test_decode_matches_prefill_row():
    """The decode path at text position p returns prefill row p (same caches)."""
    B, Hq, Hkv, hd, Nv, Nt = 4, 32, 32, 128, 576, 24
    x = attn_inputs(("p", "bf16", B, Hq, Hkv, hd, Nv, Nt, Nt, 0), seed=21)
    xg = {k: cuda(v) for k, v in x.items()}
    O = torch.empty_like(xg["Q"])
    dvl.text_visual_attention(xg["Q"], xg["Kv"], xg["Vv"], xg["Kt"], xg["Vt"], O)
    for p in (0, 7, Nt - 1):
        Od = torch.empty_like(xg["Q"][:, p:p + 1]).contiguous()
        dvl.text_visual_attention(xg["Q"][:, p:p + 1].contiguous(), xg["Kv"], xg["Vv"],
                                  xg["Kt"][:, :, :p + 1].contiguous(),
                                  xg["Vt"][:, :, :p + 1].contiguous(), Od, q_pos0=p)
        torch.cuda.synchronize()
        assert_close(f64(Od[:, 0]), f64(O[:, p]), "bf16", f"decode row {p}")


def test_visual_permutation_invariance():
    """No positional term touches the visual keys: permuting them leaves O unchanged."""
    spec = ("perm", "f32", 2, 8, 2, 128, 200, 16, 16, 0)
    x = attn_inputs(spec, seed=31)
    perm = torch.randperm(200, generator=torch.Generator().manual_seed(5))
    xg = {k: cuda(v) for k, v in x.items()}
    O1, O2 = torch.empty_like(xg["Q"]), torch.empty_like(xg["Q"])
    dvl.text_visual_attention(xg["Q"], xg["Kv"], xg["Vv"], xg["Kt"], xg["Vt"], O1)
    dvl.text_visual_attention(xg["Q"], xg["Kv"][:, :, perm].contiguous(),
                              xg["Vv"][:, :, perm].contiguous(), xg["Kt"], xg["Vt"], O2)
    torch.cuda.synchronize()
    assert_close(f64(O2), f64(O1), "f32", "permuted visual keys")


def test_bitwise_determinism():
    w = MID[0]
    E, wts = gen_build(w, seed=7)
    Eg, wg = cuda(E), {k: cuda(v) for k, v in wts.items()}
    r1 = run_build(w, Eg, wg, w.act)
    r2 = run_build(w, Eg, wg, w.act)
    spec = ATTN[1]
    xg = {k: cuda(v) for k, v in attn_inputs(spec).items()}
    outs = []
    for _ in range(2):
        O = torch.empty_like(xg["Q"])
        dvl.text_visual_attention(xg["Q"], xg["Kv"], xg["Vv"], xg["Kt"], xg["Vt"], O)
        outs.append(O)
    torch.cuda.synchronize()
    for a, b in zip(r1, r2):
        assert torch.equal(a, b)
    assert torch.equal(outs[0], outs[1])


def test_rejects_bad_shapes_without_writing():
    spec = ATTN[0]
    xg = {k: cuda(v) for k, v in attn_inputs(spec).items()}
    O = torch.full_like(xg["Q"], 7.0)
    with pytest.raises(dvl.DeltaVisionError) as ei:
        dvl.text_visual_attention(xg["Q"], xg["Kv"], xg["Vv"], xg["Kt"], xg["Vt"], O, q_pos0=5)
    assert ei.value.name == "DV_ERR_SHAPE"
    torch.cuda.synchronize()
    assert bool(torch.all(O == 7.0))


def test_mfma_probe():
    """The measurement probe runs the MFMAs it is timed for: with constant operands (bf16 1.0)
    every accumulator gains 32 per MFMA, so block sinks read 32 fragments x 4 lanes' items x
    32 x iters."""
    say("[mfma probe]")
    sink = torch.full((dvl.PROBE_BLOCKS,), float("nan"), dtype=torch.float32, device="cuda:0")
    dvl.probe_mfma(False, 5, sink)
    torch.cuda.synchronize()
    assert torch.all(sink == 32 * 4 * 32 * 5)
    sink.fill_(float("nan"))
    dvl.probe_mfma(True, 5, sink)
    torch.cuda.synchronize()
    assert torch.all(torch.isfinite(sink))
