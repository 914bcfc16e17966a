"""The allocation-free attention entry point (dv_text_visual_attention_noalloc) against the
workspace entry point, through the C ABI.

Two calls in a row share the library's static scratch: a larger key-split call, then a smaller
one that finds the first call's partials still in the array. Each must equal the workspace entry
point with its recommended workspace (the same split, so the same bits) and meet the parity bar
against the oracle. A call whose split would need more partials than the scratch holds is
refused before anything is launched.
"""
import pytest
import torch

import oracle
import paper_2609_34972_amd as dvl
from tests.gpu_helpers import assert_close, cuda, f64, say

pytestmark = pytest.mark.gpu

CALLS = [
    # name, dtype, B, Hq, Hkv, hd, Nv, Nq, Nkt, q_pos0 -- in call order, larger first
    ("qwen_video_prefill", "bf16", 1, 28, 4, 128, 16384, 128, 128, 0),
    ("small_gqa_hd64", "bf16", 2, 8, 2, 64, 300, 9, 20, 11),
    ("decode_mha", "bf16", 4, 32, 32, 128, 576, 1, 600, 512),
]


def inputs(spec, seed):
    name, dt, B, Hq, Hkv, hd, Nv, Nq, Nkt, q0 = spec
    tdt = torch.float32 if dt == "f32" else torch.bfloat16
    g = torch.Generator().manual_seed(seed)
    mk = lambda *s: torch.randn(*s, generator=g).to(tdt)
    return dict(Q=mk(B, Nq, Hq, hd), Kv=mk(B, Hkv, Nv, hd), Vv=mk(B, Hkv, Nv, hd),
                Kt=mk(B, Hkv, Nkt, hd), Vt=mk(B, Hkv, Nkt, hd))


def test_noalloc_matches_workspace_entry_point():
    for n, spec in enumerate(CALLS):
        name, dt, B, Hq, Hkv, hd, Nv, Nq, Nkt, q0 = spec
        say(f"[noalloc call {n}: {name}]")
        x = inputs(spec, 40 + n)
        xg = {k: cuda(v) for k, v in x.items()}
        need = dvl.text_visual_attention_workspace(B, Hq, Hkv, hd, Nv, Nq, Nkt)
        assert need > 0  # the call splits its keys
        ws = torch.empty(need, dtype=torch.uint8, device="cuda:0")
        O_ws = torch.empty_like(xg["Q"])
        dvl.text_visual_attention(xg["Q"], xg["Kv"], xg["Vv"], xg["Kt"], xg["Vt"], O_ws, q_pos0=q0,
                                  ws=ws)
        O = torch.full_like(xg["Q"], float("nan"))
        dvl.text_visual_attention_noalloc(xg["Q"], xg["Kv"], xg["Vv"], xg["Kt"], xg["Vt"], O,
                                          q_pos0=q0)
        torch.cuda.synchronize()
        e = assert_close(f64(O), f64(O_ws), dt, f"{name}: no-alloc vs workspace entry point")
        assert torch.equal(O, O_ws), f"{name}: the two entry points differ in the bits"
        ref = oracle.text_visual_attention(*(f64(x[k]) for k in ("Q", "Kv", "Vv", "Kt", "Vt")), q0)
        e2 = assert_close(f64(O), ref, dt, f"{name}: no-alloc vs oracle")
        say(f"  vs workspace entry point {e:.1e}, vs oracle {e2:.2e}")


def test_noalloc_refuses_split_beyond_scratch():
    # fp32 GQA prefill with 64 (kv-head, row block) streams: its preferred split fills 512 blocks
    # of 128 rows, whose fp32 partials need more than the scratch holds
    B, Hq, Hkv, hd, Nv, Nq = 1, 64, 8, 128, 4096, 128
    assert dvl.text_visual_attention_workspace(B, Hq, Hkv, hd, Nv, Nq, Nq) > dvl.ATTENTION_SCRATCH_BYTES
    mk = lambda *s: torch.zeros(*s, dtype=torch.float32, device="cuda:0")
    Q, Kv, Vv, Kt, Vt = mk(B, Nq, Hq, hd), mk(B, Hkv, Nv, hd), mk(B, Hkv, Nv, hd), mk(B, Hkv, Nq, hd), mk(B, Hkv, Nq, hd)
    O = torch.full_like(Q, 7.0)
    with pytest.raises(dvl.DeltaVisionError) as ei:
        dvl.text_visual_attention_noalloc(Q, Kv, Vv, Kt, Vt, O)
    assert ei.value.name == "DV_ERR_WORKSPACE"
    torch.cuda.synchronize()
    assert bool(torch.all(O == 7.0))
