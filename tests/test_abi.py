"""C-ABI boundary checks that need no GPU.

The library must load, export every function that include/deltavision.h
declares, and reject invalid arguments on the host (before any HIP call) with
the documented status codes. Only NULL or fake pointers are passed: every case
here fails validation, so nothing is ever launched.
"""
import ctypes
import os
import re

import pytest

from paper_2609_34972_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "deltavision.h")

OK, NULL, SHAPE, UNSUP, ALIGN, WS = 0, 1, 2, 3, 4, 5
F32, BF16 = 0, 1
FAKE = 0x10000  # a 16-byte aligned non-NULL address; never dereferenced (validation fails first)


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(dv_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(_lib.LIB_PATH):
        from paper_2609_34972_amd import build
        build.build()
    return _lib.load()


def test_every_declared_symbol_is_exported(lib):
    names = declared_functions()
    assert set(names) == set(_lib.EXPORTS), names
    for n in names:
        assert hasattr(lib, n), n
        assert ctypes.cast(getattr(lib, n), ctypes.c_void_p).value


def test_version_and_status_strings(lib):
    assert lib.dv_abi_version() == 1
    for code, name in [(0, b"DV_OK"), (1, b"DV_ERR_NULL"), (2, b"DV_ERR_SHAPE"),
                       (3, b"DV_ERR_UNSUPPORTED"), (4, b"DV_ERR_ALIGN"), (5, b"DV_ERR_WORKSPACE"),
                       (6, b"DV_ERR_HIP"), (7, b"DV_ERR_INTERNAL"), (99, b"DV_UNKNOWN_STATUS")]:
        assert lib.dv_status_string(code) == name


def build_call(lib, E=FAKE, Dw=FAKE, Z=FAKE, T=64, d=256, L=4, r=16, act=0, dt=F32):
    return lib.dv_build_visual_memory(E, Dw, Z, T, d, L, r, act, dt, None)


@pytest.mark.parametrize("kw,code", [
    (dict(E=None), NULL), (dict(Dw=None), NULL), (dict(Z=None), NULL),
    (dict(E=FAKE + 4), ALIGN), (dict(Z=FAKE + 8), ALIGN),
    (dict(T=0), SHAPE), (dict(T=-5), SHAPE), (dict(d=0), SHAPE), (dict(L=0), SHAPE), (dict(r=0), SHAPE),
    (dict(T=65535 * 64 + 1), SHAPE),
    (dict(d=100), UNSUP), (dict(r=24), UNSUP), (dict(act=7), UNSUP), (dict(dt=5), UNSUP),
])
def test_build_visual_memory_rejects(lib, kw, code):
    assert build_call(lib, **kw) == code
    assert lib.dv_last_error() != b""


def kv_call(lib, ws=FAKE, ws_bytes=None, **over):
    a = dict(E=FAKE, Z=FAKE, Uw=FAKE, g=FAKE, Wk=FAKE, Wv=FAKE, Kv=FAKE, Vv=FAKE, B=1, Nv=64, d=256,
             L=4, r=16, Hkv=4, hd=64, l0=0, nl=4, eps=1e-5, dt=F32)
    a.update(over)
    if ws_bytes is None:
        ws_bytes = lib.dv_project_visual_kv_workspace(a["B"] * a["Nv"], a["d"], a["nl"], a["dt"])
    return lib.dv_project_visual_kv(a["E"], a["Z"], a["Uw"], a["g"], a["Wk"], a["Wv"], a["Kv"],
                                    a["Vv"], a["B"], a["Nv"], a["d"], a["L"], a["r"], a["Hkv"],
                                    a["hd"], a["l0"], a["nl"], a["eps"], a["dt"], ws, ws_bytes,
                                    None)


@pytest.mark.parametrize("kw,code", [
    (dict(E=None), NULL), (dict(Wv=None), NULL), (dict(Kv=None), NULL), (dict(g=None), NULL),
    (dict(Wk=FAKE + 2), ALIGN),
    (dict(B=0), SHAPE), (dict(Nv=0), SHAPE), (dict(l0=-1), SHAPE), (dict(nl=0), SHAPE),
    (dict(l0=2, nl=3), SHAPE), (dict(eps=-1.0), SHAPE), (dict(eps=float("nan")), SHAPE),
    (dict(hd=96), UNSUP), (dict(d=96), UNSUP), (dict(r=8), UNSUP), (dict(dt=2), UNSUP),
])
def test_project_visual_kv_rejects(lib, kw, code):
    assert kv_call(lib, **kw) == code


def test_project_visual_kv_workspace_rules(lib):
    one = lib.dv_project_visual_kv_workspace(64, 256, 1, F32)
    four = lib.dv_project_visual_kv_workspace(64, 256, 4, F32)
    assert one > 64 * 256 * 4 and four == 4 * one
    assert lib.dv_project_visual_kv_workspace(64, 256, 1, BF16) < one
    assert lib.dv_project_visual_kv_workspace(0, 256, 1, F32) == 0
    assert lib.dv_project_visual_kv_workspace(64, 256, 1, 9) == 0
    assert kv_call(lib, ws=None) == WS
    assert kv_call(lib, ws_bytes=one - 1) == WS
    assert kv_call(lib, ws=FAKE + 4, ws_bytes=one) == ALIGN


def attn_call(lib, ws=None, ws_bytes=0, **over):
    a = dict(Q=FAKE, Kv=FAKE, Vv=FAKE, Kt=FAKE, Vt=FAKE, O=FAKE, B=1, Hq=4, Hkv=4, hd=64, Nv=64,
             Nq=16, Nkt=16, q0=0, scale=0.125, dt=F32)
    a.update(over)
    return lib.dv_text_visual_attention(a["Q"], a["Kv"], a["Vv"], a["Kt"], a["Vt"], a["O"], a["B"],
                                        a["Hq"], a["Hkv"], a["hd"], a["Nv"], a["Nq"], a["Nkt"],
                                        a["q0"], a["scale"], a["dt"], ws, ws_bytes, None)


def test_project_visual_kv_fused_rule(lib):
    """The fused up + norm + K/V kernel covers bf16 with 2 Hkv hd = 1024, r in {128, 256, 512}
    and d a multiple of 64, and is taken only while switched on."""
    eligible = [(3584, 512, 4, 128, BF16), (384, 256, 8, 64, BF16), (192, 128, 4, 128, BF16)]
    other = [(3584, 512, 4, 128, F32),        # fp32
             (4096, 256, 32, 128, BF16),      # K/V width 8192
             (3584, 384, 4, 128, BF16),       # rank 384
             (3584, 64, 4, 128, BF16),        # rank 64
             (3552, 512, 4, 128, BF16),       # d % 64 != 0
             (0, 512, 4, 128, BF16), (3584, 512, 1 << 30, 128, BF16), (3584, 512, 4, 128, 9)]
    assert all(lib.dv_project_visual_kv_fused(*a) == 0 for a in eligible + other)  # off at load
    assert lib.dv_set_fused_kv(2) == SHAPE
    try:
        assert lib.dv_set_fused_kv(1) == 0
        assert all(lib.dv_project_visual_kv_fused(*a) == 1 for a in eligible)
        assert all(lib.dv_project_visual_kv_fused(*a) == 0 for a in other)
    finally:
        assert lib.dv_set_fused_kv(0) == 0
    assert all(lib.dv_project_visual_kv_fused(*a) == 0 for a in eligible)


def test_up_kernel_rule(lib):
    """By shape the Z-resident up kernel takes r = 256 with at least 2048 blocks (128-row tiles
    times layers); forced (mode 2) it takes r = 256 or 512; mode 1 always the tiled kernel."""
    next_shape = (8 * 2880, 4096, 256, 32, BF16)     # LLaVA-NeXT: 180 x 32 blocks
    llava = (4 * 576, 4096, 256, 32, BF16)           # LLaVA-7B: 18 x 32 blocks
    qwen = (16384, 3584, 512, 28, BF16)               # Qwen2.5-VL video: r = 512
    others = [(16384, 3584, 128, 28, BF16),           # rank 128
              (16384, 3584, 256, 28, F32),            # fp32
              (1 << 21, 4096, 256, 32, BF16),         # E beyond 2^31 bytes
              (0, 4096, 256, 32, BF16)]
    assert lib.dv_project_visual_kv_up_kernel(*next_shape) == 2
    assert lib.dv_project_visual_kv_up_kernel(*llava) == 1
    assert lib.dv_project_visual_kv_up_kernel(*qwen) == 1
    assert all(lib.dv_project_visual_kv_up_kernel(*a) == 1 for a in others)
    assert lib.dv_set_up_kernel(3) == SHAPE and lib.dv_set_up_kernel(-1) == SHAPE
    try:
        assert lib.dv_set_up_kernel(2) == 0
        assert all(lib.dv_project_visual_kv_up_kernel(*a) == 2 for a in (next_shape, llava, qwen))
        assert all(lib.dv_project_visual_kv_up_kernel(*a) == 1 for a in others)
        assert lib.dv_set_up_kernel(1) == 0
        assert all(lib.dv_project_visual_kv_up_kernel(*a) == 1 for a in (next_shape, llava, qwen))
    finally:
        assert lib.dv_set_up_kernel(0) == 0
    assert lib.dv_project_visual_kv_up_kernel(*next_shape) == 2


@pytest.mark.parametrize("kw,code", [
    (dict(Q=None), NULL), (dict(Kt=None), NULL), (dict(O=None), NULL), (dict(Kv=None), NULL),
    (dict(Vt=FAKE + 4), ALIGN),
    (dict(B=0), SHAPE), (dict(Nq=0), SHAPE), (dict(Nv=-1), SHAPE), (dict(q0=-1), SHAPE),
    (dict(Hq=6, Hkv=4), SHAPE), (dict(q0=1), SHAPE), (dict(Nkt=15), SHAPE),
    (dict(scale=float("inf")), SHAPE), (dict(scale=0.0), SHAPE), (dict(scale=-0.5), SHAPE),
    (dict(B=70000, Hkv=1, Hq=1), SHAPE),
    (dict(hd=32), UNSUP), (dict(hd=256), UNSUP), (dict(dt=3), UNSUP),
])
def test_text_visual_attention_rejects(lib, kw, code):
    assert attn_call(lib, **kw) == code


def test_attention_misaligned_workspace_rejected(lib):
    assert attn_call(lib, ws=FAKE + 4, ws_bytes=1 << 20) == ALIGN


def test_attention_workspace_query(lib):
    # Few (batch, head) units with many keys want a key split, hence a workspace.
    n = lib.dv_text_visual_attention_workspace(1, 28, 4, 128, 16384, 128, 128)
    assert n > 0 and n % (1 * 128 * 28 * (128 + 2) * 4) == 0
    # Decode over 2048 (batch, head) streams fills the chip without a split.
    assert lib.dv_text_visual_attention_workspace(64, 32, 32, 128, 576, 1, 513) == 0
    assert lib.dv_text_visual_attention_workspace(1, 6, 4, 128, 10, 4, 4) == 0  # invalid GQA


def rec_call(lib, ws=FAKE, ws_bytes=None, **over):
    a = dict(E=FAKE, Dw=FAKE, Uw=FAKE, g=FAKE, Wk=FAKE, Wv=FAKE, Kv=FAKE, Vv=FAKE, B=1, Nv=64,
             d=256, L=4, r=16, Hkv=4, hd=64, act=0, eps=1e-5, dt=F32)
    a.update(over)
    if ws_bytes is None:
        ws_bytes = lib.dv_recurrent_visual_kv_workspace(a["B"] * a["Nv"], a["d"], a["L"], a["r"], a["dt"])
    return lib.dv_recurrent_visual_kv(a["E"], a["Dw"], a["Uw"], a["g"], a["Wk"], a["Wv"], a["Kv"],
                                      a["Vv"], a["B"], a["Nv"], a["d"], a["L"], a["r"], a["Hkv"],
                                      a["hd"], a["act"], a["eps"], a["dt"], ws, ws_bytes, None)


@pytest.mark.parametrize("kw,code", [
    (dict(E=None), NULL), (dict(Dw=None), NULL), (dict(Vv=None), NULL), (dict(Uw=FAKE + 2), ALIGN),
    (dict(B=0), SHAPE), (dict(L=0), SHAPE), (dict(eps=-1.0), SHAPE),
    (dict(hd=32), UNSUP), (dict(d=100), UNSUP), (dict(r=12), UNSUP), (dict(act=3), UNSUP),
    (dict(dt=4), UNSUP), (dict(ws=None), WS), (dict(ws_bytes=1024), WS), (dict(ws=FAKE + 8), ALIGN),
])
def test_recurrent_visual_kv_rejects(lib, kw, code):
    assert rec_call(lib, **kw) == code


def test_recurrent_workspace_grows_with_layers(lib):
    a = lib.dv_recurrent_visual_kv_workspace(2304, 4096, 8, 256, BF16)
    b = lib.dv_recurrent_visual_kv_workspace(2304, 4096, 32, 256, BF16)
    assert 0 < a < b and lib.dv_recurrent_visual_kv_workspace(0, 4096, 8, 256, BF16) == 0


def kept_call(lib, keep=(1, 0, 1, 1), ws=FAKE, ws_bytes=None, **over):
    a = dict(E=FAKE, Dw=FAKE, Uw=FAKE, g=FAKE, Wk=FAKE, Wv=FAKE, Kv=FAKE, Vv=FAKE, B=1, Nv=64,
             d=256, L=4, r=16, Hkv=4, hd=64, act=0, eps=1e-5, dt=F32)
    a.update(over)
    karr = None if keep is None else (ctypes.c_uint8 * len(keep))(*keep)
    if ws_bytes is None:
        ws_bytes = lib.dv_kept_visual_kv_workspace(a["B"] * a["Nv"], a["d"], a["r"],
                                                   max(1, sum(keep or ())), a["dt"])
    return lib.dv_kept_visual_kv(a["E"], a["Dw"], a["Uw"], a["g"], a["Wk"], a["Wv"],
                                 ctypes.cast(karr, ctypes.c_void_p) if karr else None, a["Kv"],
                                 a["Vv"], a["B"], a["Nv"], a["d"], a["L"], a["r"], a["Hkv"], a["hd"],
                                 a["act"], a["eps"], a["dt"], ws, ws_bytes, None)


@pytest.mark.parametrize("kw,code", [
    (dict(keep=None), NULL), (dict(E=None), NULL), (dict(Kv=None), NULL), (dict(Wk=FAKE + 2), ALIGN),
    (dict(B=0), SHAPE), (dict(L=0), SHAPE), (dict(eps=float("inf")), SHAPE),
    (dict(hd=48), UNSUP), (dict(d=96), UNSUP), (dict(r=20), UNSUP), (dict(act=5), UNSUP),
    (dict(dt=7), UNSUP), (dict(ws=None), WS), (dict(ws_bytes=4096), WS), (dict(ws=FAKE + 8), ALIGN),
])
def test_kept_visual_kv_rejects(lib, kw, code):
    assert kept_call(lib, **kw) == code


def test_kept_visual_kv_nothing_kept_is_a_no_op(lib):
    # Every layer skipped: valid, launches nothing, needs no caches and no workspace.
    assert kept_call(lib, keep=(0, 0, 0, 0), Kv=None, Vv=None, ws=None, ws_bytes=0) == OK


def test_kept_workspace_rules(lib):
    one = lib.dv_kept_visual_kv_workspace(2304, 4096, 256, 1, BF16)
    many = lib.dv_kept_visual_kv_workspace(2304, 4096, 256, 17, BF16)
    proj = lib.dv_project_visual_kv_workspace(2304, 4096, 1, BF16)
    assert one == proj + 2304 * 256 * 2 and many == 17 * one
    assert lib.dv_kept_visual_kv_workspace(2304, 4096, 256, 0, BF16) == 0


def ex_call(lib, epi=None, ws=FAKE, ws_bytes=None, **over):
    a = dict(E=FAKE, Z=FAKE, Uw=FAKE, g=FAKE, Wk=FAKE, Wv=FAKE, Kv=FAKE, Vv=FAKE, B=1, Nv=64, d=256,
             L=4, r=16, Hkv=4, hd=64, l0=0, nl=4, eps=1e-5, dt=F32)
    a.update(over)
    if ws_bytes is None:
        ws_bytes = lib.dv_project_visual_kv_ex_workspace(a["B"] * a["Nv"], a["d"], a["nl"], a["hd"],
                                                         a["dt"])
    return lib.dv_project_visual_kv_ex(a["E"], a["Z"], a["Uw"], a["g"], a["Wk"], a["Wv"], a["Kv"],
                                       a["Vv"], a["B"], a["Nv"], a["d"], a["L"], a["r"], a["Hkv"],
                                       a["hd"], a["l0"], a["nl"], a["eps"],
                                       ctypes.byref(epi) if epi is not None else None, a["dt"], ws,
                                       ws_bytes, None)


def epi(**kw):
    e = _lib._KvEpilogue()
    e.k_norm_eps, e.rope_theta = 1e-6, 10000.0
    e.rope_sections = (ctypes.c_int32 * 3)(32, 0, 0)
    for k, v in kw.items():
        if k == "sections":
            e.rope_sections = (ctypes.c_int32 * 3)(*v)
        else:
            setattr(e, k, v)
    return e


@pytest.mark.parametrize("kw,code", [
    (dict(positions=FAKE, sections=(16, 8, 4)), SHAPE),
    (dict(positions=FAKE, sections=(40, -8, 0)), SHAPE),
    (dict(positions=FAKE, rope_theta=0.0), SHAPE),
    (dict(positions=FAKE, rope_theta=float("inf")), SHAPE),
    (dict(positions=FAKE + 2), ALIGN),
    (dict(k_norm=FAKE, k_norm_eps=-1.0), SHAPE),
    (dict(k_norm=FAKE + 4), ALIGN),
    (dict(k_bias=FAKE + 8), ALIGN),
    (dict(v_bias=FAKE + 2), ALIGN),
])
def test_project_ex_rejects_bad_epilogue(lib, kw, code):
    assert ex_call(lib, epi(**kw)) == code


def test_project_ex_rejects_like_plain(lib):
    assert ex_call(lib, epi(), hd=96) == UNSUP
    assert ex_call(lib, epi(), E=None) == NULL
    assert ex_call(lib, None, nl=5) == SHAPE


def test_project_ex_workspace_includes_rope_table(lib):
    one = lib.dv_project_visual_kv_ex_workspace(64, 256, 1, 64, F32)
    assert one == lib.dv_project_visual_kv_workspace(64, 256, 1, F32) + 64 * 64 * 4
    assert lib.dv_project_visual_kv_ex_workspace(64, 256, 1, 96, F32) == 0
    # with rotation the table must fit next to one layer slot
    assert ex_call(lib, epi(positions=FAKE), ws_bytes=one - 1, nl=1) == WS


def dr_call(lib, ws=FAKE, ws_bytes=None, **over):
    a = dict(k=FAKE, v=FAKE, alpha=FAKE, beta=FAKE, S=FAKE, B=1, Hk=2, Hv=4, N=100, dk=64, dv=64,
             dt=F32)
    a.update(over)
    if ws_bytes is None:
        ws_bytes = lib.dv_delta_rule_workspace(a["B"], a["Hv"], max(a["N"], 1), a["dk"], a["dv"],
                                               a["dt"])
    return lib.dv_delta_rule_write(a["k"], a["v"], a["alpha"], a["beta"], a["S"], a["B"], a["Hk"],
                                   a["Hv"], a["N"], a["dk"], a["dv"], a["dt"], ws, ws_bytes, None)


@pytest.mark.parametrize("kw,code", [
    (dict(k=None), NULL), (dict(v=None), NULL), (dict(alpha=None), NULL), (dict(S=None), NULL),
    (dict(S=FAKE + 4), ALIGN), (dict(beta=FAKE + 2), ALIGN), (dict(k=FAKE + 8), ALIGN),
    (dict(B=0), SHAPE), (dict(Hk=0), SHAPE), (dict(N=-1), SHAPE), (dict(Hk=3), SHAPE),
    (dict(dk=96), UNSUP), (dict(dv=32), UNSUP), (dict(dt=2), UNSUP),
    (dict(ws=None), WS), (dict(ws_bytes=256), WS), (dict(ws=FAKE + 8), ALIGN),
])
def test_delta_rule_rejects(lib, kw, code):
    assert dr_call(lib, **kw) == code


def test_delta_rule_without_tokens_is_a_no_op(lib):
    assert dr_call(lib, N=0, k=None, v=None, alpha=None, beta=None, ws=None, ws_bytes=0) == OK


def test_delta_rule_workspace_scales_with_chunks(lib):
    one = lib.dv_delta_rule_workspace(1, 32, 64, 128, 128, BF16)
    assert one >= 32 * (64 * 128 * 3 * 2 + 4)
    assert lib.dv_delta_rule_workspace(1, 32, 65, 128, 128, BF16) > one  # a second chunk
    assert lib.dv_delta_rule_workspace(1, 32, 64, 96, 128, BF16) == 0


@pytest.mark.parametrize("sink,iters,code", [
    (None, 16, NULL), (FAKE + 4, 16, ALIGN), (FAKE, 0, SHAPE), (FAKE, -1, SHAPE),
    (FAKE, (1 << 20) + 1, SHAPE),
])
def test_probe_mfma_rejects(lib, sink, iters, code):
    assert lib.dv_probe_mfma(1, iters, sink, None) == code
    assert lib.dv_last_error() != b""


def noalloc_call(lib, Q=FAKE, Kv=FAKE, Vv=FAKE, Kt=FAKE, Vt=FAKE, O=FAKE, B=2, Hq=8, Hkv=2, hd=64,
                 Nv=300, Nq=9, Nkt=20, q0=11, scale=0.125, dt=BF16):
    return lib.dv_text_visual_attention_noalloc(Q, Kv, Vv, Kt, Vt, O, B, Hq, Hkv, hd, Nv, Nq, Nkt,
                                                q0, scale, dt, None)


@pytest.mark.parametrize("kw,code", [
    (dict(Q=None), NULL), (dict(O=None), NULL), (dict(Kv=None), NULL), (dict(O=FAKE + 2), ALIGN),
    (dict(Hq=7), SHAPE), (dict(q0=12), SHAPE), (dict(scale=0.0), SHAPE), (dict(hd=96), UNSUP),
    (dict(dt=3), UNSUP),
    # fp32 prefill with 64 GQA streams (8 query heads per key head, 128 text rows): the planner
    # splits the 4096 keys 8 ways, whose partials need more than the static scratch holds, so
    # the call is refused on the host
    (dict(B=1, Hq=64, Hkv=8, hd=128, Nv=4096, Nq=128, Nkt=128, q0=0, dt=F32), WS),
])
def test_noalloc_attention_rejects(lib, kw, code):
    assert noalloc_call(lib, **kw) == code
    assert lib.dv_last_error() != b""
