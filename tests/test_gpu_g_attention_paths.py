"""GPU parity of attention paths that ordinary random inputs leave out (Section 3.2, Eq. 9).

* The online softmax raises its running maximum lazily: only when some row of a wave grows by
  more than 8 (log2 units) after its first key tile, and only then rescales the running sum and
  the output accumulators. With N(0, 1) queries and keys that never happens after the first
  tile. Here the keys ramp along a direction shared with the queries, so every row's maximum
  grows by far more than that on every key tile (checked on the inputs themselves), and the
  rescale runs in every wave whatever the key split.
* Text caches longer than the queries' positions (a preallocated decode cache, a chunk of a
  longer prompt): the free slots past q_pos0 + Nq - 1 hold NaN, so a kernel that read any of
  them would return NaN.

Every case is compared element by element with the fp64 oracle at the parity bar.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_34972_amd as dvl
from tests.gpu_helpers import assert_close, cuda, f64, say

pytestmark = pytest.mark.gpu

LOG2E = 1.4426950408889634


def _ws(split, B, Hq, Hkv, hd, Nv, Nq, Nkt):
    if split:
        n = dvl.text_visual_attention_workspace(B, Hq, Hkv, hd, Nv, Nq, Nkt)
        return torch.empty(max(n, 16), dtype=torch.uint8, device="cuda:0")
    return torch.empty(16, dtype=torch.uint8, device="cuda:0")  # too small: no split


def ramp_inputs(B, Hq, Hkv, hd, Nv, Nq, Nkt, seed):
    """Queries and keys share a unit direction u. Keys are grouped in blocks of 32 in the order
    the kernels walk them (visual keys from 0, then text keys from 0); every key of block n
    carries c_n = 1 + n * step along u, so every block scores about 24 (natural-log units) above
    the one before it for every query, whatever part of a text block the causal mask leaves.
    The queries carry a 12 u component plus N(0, 1) noise, the keys N(0, 1) noise."""
    g = torch.Generator().manual_seed(seed)
    u = torch.randn(hd, generator=g)
    u /= u.norm()
    a, scale = 12.0, hd ** -0.5
    step = 24.0 / (a * scale)
    nvb = (Nv + 31) // 32
    level = torch.cat([torch.arange(Nv) // 32, nvb + torch.arange(Nkt) // 32]).float()
    cj = 1.0 + step * level
    Q = a * u + torch.randn(B, Nq, Hq, hd, generator=g)
    Kall = cj.view(1, 1, -1, 1) * u + torch.randn(B, Hkv, Nv + Nkt, hd, generator=g)
    Vall = torch.randn(B, Hkv, Nv + Nkt, hd, generator=g)
    bf = lambda t: t.to(torch.bfloat16)
    return dict(Q=bf(Q), Kv=bf(Kall[:, :, :Nv].contiguous()), Vv=bf(Vall[:, :, :Nv].contiguous()),
                Kt=bf(Kall[:, :, Nv:].contiguous()), Vt=bf(Vall[:, :, Nv:].contiguous()))


def tile_maxima(x, q_pos0, tile):
    """Per (b, query, head) the maximum scaled score (log2 units) of each key tile, in the kernels'
    key order (visual tiles, then text tiles); masked keys are left out."""
    Q, Kv, Kt = f64(x["Q"]), f64(x["Kv"]), f64(x["Kt"])
    B, Nq, Hq, hd = Q.shape
    Hkv, Nv = Kv.shape[1], Kv.shape[2]
    G = Hq // Hkv
    K = np.repeat(np.concatenate([Kv, Kt], axis=2), G, axis=1)           # [B, Hq, keys, hd]
    s = np.einsum("bihc,bhjc->bihj", Q, K) * hd ** -0.5 * LOG2E
    nt = Nv + q_pos0 + Nq
    s = s[..., :nt]
    for i in range(Nq):
        s[:, i, :, Nv + q_pos0 + i + 1:] = -np.inf
    out = []
    for k0 in list(range(0, Nv, tile)) + [Nv + t for t in range(0, q_pos0 + Nq, tile)]:
        k1 = min(k0 + tile, Nv) if k0 < Nv else min(k0 + tile, nt)
        out.append(s[..., k0:k1].max(axis=-1))
    return np.stack(out, axis=-1)                                           # [B, Nq, Hq, tiles]


LAZY = [
    # name, B, Hq, Hkv, hd, Nv, Nq, Nkt: bf16 hd 128 takes the key-group kernel for up to 64
    # (query, head) rows per kv-head, the two-wave streaming kernel for 65-96 and the ping-pong
    # kernel above that
    ("ksplit_mha", 2, 8, 8, 128, 577, 64, 64),
    ("pp_gqa", 1, 28, 4, 128, 1000, 128, 128),
    ("stream_mha_96rows", 2, 6, 2, 128, 700, 32, 32),
    ("pp_mha_128rows", 2, 8, 8, 128, 700, 128, 128),
]


@pytest.mark.parametrize("spec", LAZY, ids=[c[0] for c in LAZY])
@pytest.mark.parametrize("split", [True, False], ids=["ws", "nows"])
def test_running_max_rescale(spec, split):
    name, B, Hq, Hkv, hd, Nv, Nq, Nkt = spec
    say(f"[rescale {name} split={split}]")
    x = ramp_inputs(B, Hq, Hkv, hd, Nv, Nq, Nkt, seed=5)
    # Premise: in every row each 32-key tile beats the best score of all earlier tiles by more
    # than 8 (log2 units), so any wave that computes two or more tiles rescales mid-stream.
    tm = tile_maxima(x, 0, 32)
    best_before = np.maximum.accumulate(tm, axis=-1)[..., :-1]
    valid = np.isfinite(tm[..., 1:])
    assert np.all((tm[..., 1:] > best_before + 8.0) | ~valid), "inputs do not force the rescale"
    xg = {k: cuda(v) for k, v in x.items()}
    O = torch.empty_like(xg["Q"])
    ws = _ws(split, B, Hq, Hkv, hd, Nv, Nq, Nkt)
    dvl.text_visual_attention(xg["Q"], xg["Kv"], xg["Vv"], xg["Kt"], xg["Vt"], O, ws=ws)
    torch.cuda.synchronize()
    ref = oracle.text_visual_attention(f64(x["Q"]), f64(x["Kv"]), f64(x["Vv"]), f64(x["Kt"]),
                                       f64(x["Vt"]), 0)
    e = assert_close(f64(O), ref, "bf16", f"O {name}")
    say(f"  err {e:.2e}")


def test_running_max_rescale_growing_key_norms():
    """A milder form: queries scaled by 12 and visual key norms growing from 1 to 4 along the key
    index, plus text keys 3x larger (their tiles come last)."""
    B, Hq, Hkv, hd, Nv, Nq = 2, 8, 8, 128, 577, 64
    g = torch.Generator().manual_seed(8)
    grow = (1.0 + 3.0 * torch.arange(Nv) / Nv).view(1, 1, Nv, 1)
    x = dict(Q=12.0 * torch.randn(B, Nq, Hq, hd, generator=g),
             Kv=grow * torch.randn(B, Hkv, Nv, hd, generator=g),
             Vv=torch.randn(B, Hkv, Nv, hd, generator=g),
             Kt=3.0 * torch.randn(B, Hkv, Nq, hd, generator=g),
             Vt=torch.randn(B, Hkv, Nq, hd, generator=g))
    x = {k: v.to(torch.bfloat16) for k, v in x.items()}
    tm = tile_maxima(x, 0, 32)
    first = tm[..., 0:1]
    assert np.mean(np.max(tm[..., 4:], axis=-1) > first[..., 0] + 8.0) > 0.9
    xg = {k: cuda(v) for k, v in x.items()}
    for split in (False, True):
        O = torch.empty_like(xg["Q"])
        dvl.text_visual_attention(xg["Q"], xg["Kv"], xg["Vv"], xg["Kt"], xg["Vt"], O,
                                  ws=_ws(split, B, Hq, Hkv, hd, Nv, Nq, Nq))
        torch.cuda.synchronize()
        ref = oracle.text_visual_attention(f64(x["Q"]), f64(x["Kv"]), f64(x["Vv"]), f64(x["Kt"]),
                                           f64(x["Vt"]), 0)
        e = assert_close(f64(O), ref, "bf16", f"O split={split}")
        say(f"  split={split}: err {e:.2e}")


LONG = [
    # name, dtype, B, Hq, Hkv, hd, Nv, Nq, Nkt, q_pos0: text keys q_pos0 + Nq .. Nkt - 1 unused
    ("ksplit_chunk", "bf16", 2, 8, 8, 128, 577, 64, 1024, 512),
    ("pp_chunk", "bf16", 1, 28, 4, 128, 1000, 128, 1024, 512),
    ("stream_chunk_96rows", "bf16", 2, 6, 2, 128, 700, 32, 600, 300),
    ("decode_mha", "bf16", 4, 32, 32, 128, 576, 1, 1024, 512),
    ("decode_gqa", "bf16", 2, 28, 4, 128, 300, 1, 1024, 700),
    ("prefill_bf16_hd64", "bf16", 2, 8, 2, 64, 130, 7, 100, 13),
    ("prefill_f32", "f32", 2, 6, 2, 128, 90, 9, 40, 3),
    ("decode_f32_hd64", "f32", 3, 4, 4, 64, 33, 1, 50, 6),
]


@pytest.mark.parametrize("spec", LONG, ids=[c[0] for c in LONG])
@pytest.mark.parametrize("split", [True, False], ids=["ws", "nows"])
def test_text_cache_longer_than_queries(spec, split):
    name, dt, B, Hq, Hkv, hd, Nv, Nq, Nkt, q0 = spec
    say(f"[long text cache {name} split={split}]")
    tdt = torch.float32 if dt == "f32" else torch.bfloat16
    g = torch.Generator().manual_seed(13)
    mk = lambda *s: torch.randn(*s, generator=g).to(tdt)
    x = dict(Q=mk(B, Nq, Hq, hd), Kv=mk(B, Hkv, Nv, hd), Vv=mk(B, Hkv, Nv, hd),
             Kt=mk(B, Hkv, Nkt, hd), Vt=mk(B, Hkv, Nkt, hd))
    used = q0 + Nq
    x["Kt"][:, :, used:] = float("nan")
    x["Vt"][:, :, used:] = float("nan")
    xg = {k: cuda(v) for k, v in x.items()}
    O = torch.empty_like(xg["Q"])
    dvl.text_visual_attention(xg["Q"], xg["Kv"], xg["Vv"], xg["Kt"], xg["Vt"], O, q_pos0=q0,
                              ws=_ws(split, B, Hq, Hkv, hd, Nv, Nq, Nkt))
    torch.cuda.synchronize()
    ref = oracle.text_visual_attention(f64(x["Q"]), f64(x["Kv"]), f64(x["Vv"]), f64(x["Kt"]),
                                       f64(x["Vt"]), q0)
    assert np.all(np.isfinite(ref))
    e = assert_close(f64(O), ref, dt, f"O {name}")
    # the same call on the cache cut to the used slots gives the same bits
    O2 = torch.empty_like(O)
    dvl.text_visual_attention(xg["Q"], xg["Kv"], xg["Vv"], xg["Kt"][:, :, :used].contiguous(),
                              xg["Vt"][:, :, :used].contiguous(), O2, q_pos0=q0,
                              ws=_ws(split, B, Hq, Hkv, hd, Nv, Nq, used))
    torch.cuda.synchronize()
    say(f"  err {e:.2e}")
    assert torch.equal(O, O2), "the unused cache slots changed the result"


GRAPH = [
    # name, B, Hq, Hkv, hd, Nv, Nq: both take a key split with the workspace, so the graph holds
    # the attention kernel and the merge kernel
    ("ksplit_mha", 1, 4, 4, 128, 577, 64),
    ("pp_gqa", 1, 28, 4, 128, 1000, 128),
]


@pytest.mark.parametrize("spec", GRAPH, ids=[c[0] for c in GRAPH])
def test_attention_graph_replays(spec):
    """A captured HIP graph of an attention call with its key split (the attention kernel, then
    the merge of the partials in the workspace) replays with eager work in between: every
    replay, and every eager call after it, gives the bits of the first eager call, which meets
    the parity bar against the oracle. The workspace starts out filled with a byte pattern."""
    name, B, Hq, Hkv, hd, Nv, Nq = spec
    say(f"[graph replays {name}]")
    n = dvl.text_visual_attention_workspace(B, Hq, Hkv, hd, Nv, Nq, Nq)
    assert n > 0, "the case must take a key split"
    g = torch.Generator().manual_seed(29)
    mk = lambda *s: torch.randn(*s, generator=g).to(torch.bfloat16)
    x = dict(Q=mk(B, Nq, Hq, hd), Kv=mk(B, Hkv, Nv, hd), Vv=mk(B, Hkv, Nv, hd),
             Kt=mk(B, Hkv, Nq, hd), Vt=mk(B, Hkv, Nq, hd))
    xg = {k: cuda(v) for k, v in x.items()}
    ws = torch.full((n,), 0xA5, dtype=torch.uint8, device="cuda:0")
    args = (xg["Q"], xg["Kv"], xg["Vv"], xg["Kt"], xg["Vt"])
    O_ref = torch.empty_like(xg["Q"])
    dvl.text_visual_attention(*args, O_ref, ws=ws)
    torch.cuda.synchronize()
    ref = oracle.text_visual_attention(f64(x["Q"]), f64(x["Kv"]), f64(x["Vv"]), f64(x["Kt"]),
                                       f64(x["Vt"]), 0)
    assert_close(f64(O_ref), ref, "bf16", f"eager {name}")
    O = torch.empty_like(O_ref)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        dvl.text_visual_attention(*args, O, ws=ws)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        dvl.text_visual_attention(*args, O, ws=ws)
    for r in range(4):
        O.fill_(float("nan"))
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(O, O_ref), f"replay {r} differs from the eager call"
        O2 = torch.empty_like(O)
        dvl.text_visual_attention(*args, O2, ws=ws)
        torch.cuda.synchronize()
        assert torch.equal(O2, O_ref), f"eager call after replay {r} differs"
    say("  4 replays and 4 eager calls equal the first eager call")
