"""attn_decode_noalloc (the decode entry point that allocates nothing, its
workspace built into the library) against attn_decode with a caller's
workspace: the same kernels and cut, so O and LSE must be bit-identical.
Two calls in a row, the second with a smaller input, so the second reuses
the built-in buffer that the first filled; then a cut whose workspace
exceeds the built-in buffer is refused with ATTN_ENOSPACE before any launch."""
import pytest
import torch

import paper_2609_33586_amd as pkg
from paper_2609_33586_amd import synth
from parity_helpers import BF16, EXACT, FP8, H15, dev_tensors, say, scale_of

pytestmark = pytest.mark.gpu

# (B, Hq, Hkv, Sq, Sk, d, dtype, causal, mode, split_keys): the second case is
# smaller than the first in every dimension that sizes the workspace
CASES = [
    (2, 32, 8, 4, 6000, 128, BF16, True, H15, 512),
    (1, 8, 2, 1, 1700, 64, BF16, False, EXACT, 256),
    (2, 16, 4, 2, 5000, 128, FP8, True, H15, 384),
    (1, 4, 4, 1, 900, 128, FP8, False, EXACT, 128),
]


def run_pair(case, seed):
    B, Hq, Hkv, Sq, Sk, d, dt, causal, mode, split = case
    say(f"noalloc B={B} Hq={Hq} Hkv={Hkv} Sq={Sq} Sk={Sk} d={d} dtype={dt} causal={causal} mode={mode} split={split}")
    inp = synth.make_decode_inputs(B, Hq, Hkv, Sq, Sk, d, dt, sharp=True, seed=seed)
    q, k, v = dev_tensors(inp)
    assert pkg.attn_decode_workspace_bytes(B, Hq, Sq, Sk, d, split) > 0  # several parts
    sc = scale_of(d)
    o_ref, l_ref = pkg.attn_decode(q, k, v, causal=causal, scale=sc, exp_mode=mode, split_keys=split,
                                   descale=inp.descale)
    o = torch.full_like(o_ref, float("nan"))
    lse = torch.full_like(l_ref, float("nan"))
    pkg.attn_decode_noalloc(q, k, v, causal=causal, scale=sc, exp_mode=mode, split_keys=split, descale=inp.descale,
                            out=o, lse=lse)
    torch.cuda.synchronize()
    assert torch.equal(o.view(torch.int16), o_ref.view(torch.int16))
    assert torch.equal(lse, l_ref)
    # the same on a side stream of the current device
    st = torch.cuda.Stream()
    o2 = torch.full_like(o_ref, float("nan"))
    lse2 = torch.full_like(l_ref, float("nan"))
    torch.cuda.synchronize()
    with torch.cuda.stream(st):
        pkg.attn_decode_noalloc(q, k, v, causal=causal, scale=sc, exp_mode=mode, split_keys=split,
                                descale=inp.descale, stream=st, out=o2, lse=lse2)
    st.synchronize()
    torch.cuda.synchronize()
    assert torch.equal(o2.view(torch.int16), o_ref.view(torch.int16))
    assert torch.equal(lse2, l_ref)


@pytest.mark.parametrize("first,second", [(0, 1), (2, 3)])
def test_noalloc_matches_decode_twice(first, second):
    run_pair(CASES[first], seed=900 + first)
    run_pair(CASES[second], seed=900 + second)


def test_noalloc_refuses_beyond_its_buffer():
    # 4 x 64 rows x 128 parts x (128 + 2) floats: 17.0 MB of partial results
    B, Hq, Hkv, Sq, Sk, d = 4, 64, 8, 1, 16384, 128
    split = 128
    assert pkg.attn_decode_workspace_bytes(B, Hq, Sq, Sk, d, split) > 16 << 20
    dev = torch.device("cuda:0")
    q = torch.zeros((B, Hq, Sq, d), dtype=torch.bfloat16, device=dev)
    k = torch.zeros((B, Hkv, Sk, d), dtype=torch.bfloat16, device=dev)
    v = torch.zeros_like(k)
    o = torch.full((B, Hq, Sq, d), 7.0, dtype=torch.bfloat16, device=dev)
    with pytest.raises(pkg.AttnError) as e:
        pkg.attn_decode_noalloc(q, k, v, causal=True, scale=0.1, exp_mode=H15, split_keys=split, out=o)
    assert e.value.code == pkg.ATTN_ENOSPACE
    torch.cuda.synchronize()
    assert bool((o == 7.0).all())  # nothing launched, nothing written
