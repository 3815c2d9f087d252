"""The layer captured in a HIP graph (no host launch cost per step): every
replay equals the eager call bit for bit, with eager work and host
synchronisation between replays.  Nothing in the layer records a memset."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_05228_amd as ace
import synth
from gpu_helpers import DEV, device_layer

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("T", [1, 8, 40, 300])
def test_graph_replay_matches_eager(T):
    L = synth.make_layer(synth.config("prefill_4096", T=T, d=256, N=32, k=8, m=128, seed=23))
    tb = oracle.tables.build_tables(L)
    D = device_layer(L)
    ag = torch.from_numpy(tb["a_gsp"]).to(DEV)
    ar = torch.from_numpy(tb["a_rcr"]).to(DEV)
    k, m, N, d = 8, 128, 32, 256
    out = {"y": torch.empty((T, d), dtype=torch.bfloat16, device=DEV),
           "topk_idx": torch.empty((T, k), dtype=torch.int32, device=DEV),
           "keep": torch.empty((T, k), dtype=torch.uint8, device=DEV),
           "gates": torch.empty((T, k), dtype=torch.float32, device=DEV),
           "counts": torch.empty((N,), dtype=torch.int32, device=DEV),
           "offsets": torch.empty((N + 1,), dtype=torch.int32, device=DEV),
           "perm": torch.empty((T * k,), dtype=torch.int32, device=DEV)}
    desc = ace.make_desc(T, d, N, k, m, torch.bfloat16, 0.12)
    ws = torch.empty(ace.workspace_size(desc), dtype=torch.uint8, device=DEV)

    def step():
        ace.moe_forward(D["x"], D, ag, ar, k=k, tau=0.12, out=out, ws=ws, want_plan=True)

    step()
    torch.cuda.synchronize()
    want = {key: v.clone() for key, v in out.items()}
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()  # warm-up on the capture stream
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    for rep in range(4):
        for v in out.values():
            v.fill_(0)              # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        n = int(want["offsets"][-1].item())
        for key in ("y", "topk_idx", "keep", "gates", "counts", "offsets"):
            assert torch.equal(out[key], want[key]), (rep, key)
        assert torch.equal(out["perm"][:n], want["perm"][:n]), rep


@pytest.mark.parametrize("T", [1, 33])
def test_prepared_forward_matches_moe_forward(T):
    """A prepared call (arguments marshalled once) gives the eager call's outputs
    bit for bit, also after new tokens are written into x in place, and it can be
    captured in a graph on another stream."""
    L = synth.make_layer(synth.config("prefill_4096", T=T, d=256, N=32, k=8, m=128, seed=29))
    tb = oracle.tables.build_tables(L)
    D = device_layer(L)
    ag = torch.from_numpy(tb["a_gsp"]).to(DEV)
    ar = torch.from_numpy(tb["a_rcr"]).to(DEV)
    x = D["x"].clone()
    fn = ace.prepare_forward(x, D, ag, ar, k=8, tau=0.12, want_plan=True)
    x2 = torch.from_numpy(synth.decode_inputs(L["cfg"], T, step=5)).to(DEV).to(torch.bfloat16)
    for src in (D["x"], x2):
        x.copy_(src)
        got = {key: v.clone() for key, v in fn().items()}
        want = ace.moe_forward(src, D, ag, ar, k=8, tau=0.12, want_plan=True)
        torch.cuda.synchronize()
        n = int(want["offsets"][-1].item())
        for key in ("y", "topk_idx", "keep", "gates", "counts", "offsets"):
            assert torch.equal(got[key], want[key]), key
        assert torch.equal(got["perm"][:n], want["perm"][:n])
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        fn()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    ref = fn.out["y"].clone()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn()
    fn.out["y"].fill_(0)
    torch.cuda.synchronize()
    g.replay()
    torch.cuda.synchronize()
    assert torch.equal(fn.out["y"], ref)
