"""GPU parity of the gated delta-rule visual write (appendix on linear attention, Eq. 15-16)
through dv_delta_rule_write, against the fp64 oracle's token-by-token recurrence."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_34972_amd as dvl
from paper_2609_34972_amd import configs, synth
from tests.gpu_helpers import assert_close, cuda, f64, say

pytestmark = pytest.mark.gpu

SMALL = configs.DeltaWorkload("dr_small", "f32", B=1, Hk=1, Hv=2, N=150, dk=64, dv=64, layers=1)
CASES = [
    SMALL,
    SMALL.with_(name="dr_f32_gqa_128", B=2, Hk=2, Hv=4, N=64, dk=128, dv=128),
    SMALL.with_(name="dr_f32_dk128_dv64", Hk=1, Hv=3, N=97, dk=128, dv=64),
    SMALL.with_(name="dr_f32_one_token", N=1),
    configs.GDN_IMAGE.with_(name="dr_bf16_ragged", B=2, Hk=4, Hv=8, N=700),
    configs.GDN_IMAGE.with_(name="dr_bf16_dk64_dv128", B=1, Hk=2, Hv=2, N=333, dk=64, dv=128),
    configs.GDN_IMAGE.with_(name="dr_bf16_image", B=4, Hk=4, Hv=8),
    # long sequences at dk = dv = 128 take the two-level scan (segments of the affine chunk
    # map, then the segments in order)
    SMALL.with_(name="dr_f32_segmented", B=1, Hk=1, Hv=2, N=4000, dk=128, dv=128),
    configs.GDN_IMAGE.with_(name="dr_bf16_segmented", B=2, Hk=2, Hv=4, N=4096),
    SMALL.with_(name="dr_f32_dk64_segmented", B=1, Hk=1, Hv=2, N=4096),
    configs.GDN_IMAGE.with_(name="dr_bf16_dk64_dv128_segmented", B=1, Hk=1, Hv=2, N=4100, dk=64, dv=128),
]


def run(w, x):
    xg = {k: cuda(v) for k, v in x.items()}
    S = xg["S"].clone()
    dvl.delta_rule_write(xg["k"], xg["v"], xg["alpha"], xg["beta"], S)
    torch.cuda.synchronize()
    return S


@pytest.mark.parametrize("w", CASES, ids=lambda w: w.name)
def test_delta_rule_against_oracle(w):
    say(f"[delta rule {w.name}]")
    x = synth.make_delta_inputs(w, 1)
    S = run(w, x)
    ref = oracle.delta_rule(f64(x["k"]), f64(x["v"]), f64(x["alpha"]), f64(x["beta"]), f64(x["S"]))
    for b in range(w.B):
        for h in range(w.Hv):
            assert_close(f64(S[b, h]), ref[b, h], w.dtype, f"S[{b},{h}]")
    say(f"  max err {max(np.abs(f64(S) - ref).max() / np.abs(ref).max(), 0):.2e}")


def test_strong_decay_and_zero_strength():
    """alpha near 0 (the state is almost reset at every token) and beta = 0 on half the tokens."""
    w = SMALL.with_(name="dr_decay", N=200)
    x = synth.make_delta_inputs(w, 2)
    x["alpha"] = torch.full_like(x["alpha"], 0.05)
    x["beta"][..., ::2] = 0
    S = run(w, x)
    ref = oracle.delta_rule(f64(x["k"]), f64(x["v"]), f64(x["alpha"]), f64(x["beta"]), f64(x["S"]))
    assert_close(f64(S), ref, "f32", "S strong decay")


def test_no_tokens_leaves_state_untouched():
    w = SMALL.with_(name="dr_empty", N=0)
    x = synth.make_delta_inputs(w.with_(N=1), 3)
    xg = {k: cuda(v) for k, v in x.items()}
    S = xg["S"].clone()
    dvl.delta_rule_write(xg["k"][:, :, :0].contiguous(), xg["v"][:, :, :0].contiguous(),
                         xg["alpha"][:, :, :0].contiguous(), xg["beta"][:, :, :0].contiguous(), S)
    torch.cuda.synchronize()
    assert torch.equal(S, xg["S"])


def test_split_write_equals_one_write():
    """Writing the tokens in two calls (the state carries over) equals one call: chunk
    boundaries of the second call fall at different tokens."""
    w = configs.GDN_IMAGE.with_(name="dr_split", B=1, Hk=2, Hv=4, N=300)
    x = synth.make_delta_inputs(w, 4)
    xg = {k: cuda(v) for k, v in x.items()}
    S1 = xg["S"].clone()
    dvl.delta_rule_write(xg["k"], xg["v"], xg["alpha"], xg["beta"], S1)
    S2 = xg["S"].clone()
    for a, b in ((0, 100), (100, 300)):
        dvl.delta_rule_write(xg["k"][:, :, a:b].contiguous(), xg["v"][:, :, a:b].contiguous(),
                             xg["alpha"][:, :, a:b].contiguous(), xg["beta"][:, :, a:b].contiguous(),
                             S2)
    torch.cuda.synchronize()
    ref = oracle.delta_rule(f64(x["k"]), f64(x["v"]), f64(x["alpha"]), f64(x["beta"]), f64(x["S"]))
    assert_close(f64(S1), ref, "bf16", "one call")
    assert_close(f64(S2), ref, "bf16", "two calls")


def test_full_video_write_sampled_heads():
    """The 16384-token video write of one layer (16 key / 32 value heads); the oracle replays
    four complete value heads token by token."""
    w = configs.GDN_VIDEO
    say("[delta rule video] generating inputs")
    x = synth.make_delta_inputs(w, 5)
    S = run(w, x)
    G = w.Hv // w.Hk
    for h in (0, 7, 18, 31):
        sl = slice(h, h + 1)
        ref = oracle.delta_rule(f64(x["k"][:, h // G:h // G + 1]), f64(x["v"][:, sl]),
                                f64(x["alpha"][:, sl]), f64(x["beta"][:, sl]), f64(x["S"][:, sl]))
        e = assert_close(f64(S[:, sl]), ref, "bf16", f"S head {h}")
        say(f"  head {h}: {e:.2e}")
