"""The forward and the allocation-free decode under HIP graph capture: both
launch only kernels on the caller's stream (no allocation, no memset), so a
captured graph replays them; every replay, with eager work between the
replays, must give the eager results bit for bit."""
import pytest
import torch

import paper_2609_33586_amd as pkg
from paper_2609_33586_amd import synth
from parity_helpers import FP8, H15, dev_tensors, say, scale_of

pytestmark = pytest.mark.gpu


def test_forward_and_noalloc_decode_replay_in_a_graph():
    dev = torch.device("cuda:0")
    sc = scale_of(128)
    inp = synth.make_inputs(1, 8, 2, 700, 128, FP8, sharp=True, seed=1900)
    q, k, v = dev_tensors(inp)
    o = torch.empty((1, 8, 700, 128), dtype=torch.bfloat16, device=dev)
    lse = torch.empty((1, 8, 700), dtype=torch.float32, device=dev)
    o_ref, l_ref = pkg.attn_fwd_ex(q, k, v, causal=True, scale=sc, exp_mode=H15, descale=inp.descale)

    dinp = synth.make_decode_inputs(2, 8, 2, 1, 1500, 128, FP8, sharp=True, seed=1901)
    dq, dk, dv = dev_tensors(dinp)
    split = 512  # three parts: the parts kernel and the merge
    od = torch.empty((2, 8, 1, 128), dtype=torch.bfloat16, device=dev)
    ld = torch.empty((2, 8, 1), dtype=torch.float32, device=dev)
    od_ref, ld_ref = pkg.attn_decode(dq, dk, dv, causal=True, scale=sc, exp_mode=H15, split_keys=split,
                                     descale=dinp.descale)
    # eager first call: the built-in workspace's address is looked up here
    pkg.attn_decode_noalloc(dq, dk, dv, causal=True, scale=sc, exp_mode=H15, split_keys=split,
                            descale=dinp.descale, out=od, lse=ld)
    torch.cuda.synchronize()

    say("graph capture: forward + allocation-free decode")
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        pkg.attn_fwd_ex(q, k, v, causal=True, scale=sc, exp_mode=H15, descale=inp.descale, out=o, lse=lse)
        pkg.attn_decode_noalloc(dq, dk, dv, causal=True, scale=sc, exp_mode=H15, split_keys=split,
                                descale=dinp.descale, out=od, lse=ld)
    for r in range(3):
        say(f"graph replay {r}")
        for t in (o, lse, od, ld):
            t.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(o.view(torch.int16), o_ref.view(torch.int16)) and torch.equal(lse, l_ref)
        assert torch.equal(od.view(torch.int16), od_ref.view(torch.int16)) and torch.equal(ld, ld_ref)
        # eager work between the replays, on the same buffers
        pkg.attn_fwd_ex(q, k, v, causal=False, scale=sc, exp_mode=H15, descale=inp.descale, out=o, lse=lse)
        torch.cuda.synchronize()
