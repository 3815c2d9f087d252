"""The no-allocation entry point against the workspace entry point, through the C ABI.

ace_moe_forward_noalloc runs the same kernels as ace_moe_forward in a static
per-device scratch array instead of a caller workspace, so on the same inputs
its outputs must be bit-identical.  Calls follow each other on one stream,
each later one on a smaller layer than the one before (the array keeps the
previous call's contents, which no call may depend on); a layer past the
array's size is refused on the host before any launch."""
import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_helpers import DEV, device_layer
from paper_2609_05228_amd import _lib
from paper_2609_05228_amd.layer import _marshal

pytestmark = pytest.mark.gpu

KEYS = ("y", "topk_idx", "keep", "gates", "scores", "counts", "offsets")


def _tables(L):
    tb = oracle.tables.build_tables(L)
    return (torch.from_numpy(tb["a_gsp"]).to(DEV), torch.from_numpy(tb["a_rcr"]).to(DEV))


def _call(L, D, tabs, tau, noalloc):
    """One layer call through the C ABI; returns host copies of every output."""
    k = L["cfg"].k
    ws = torch.empty(1, dtype=torch.uint8, device=DEV) if noalloc else None
    desc, W, O, o, ws = _marshal(D["x"], D, tabs[0], tabs[1], k, tau, 1, 1e-6, 1e-6, False, True, True, None, ws,
                                 "max")
    for v in o.values():  # poison every output: each must be written by the call
        if v.dtype.is_floating_point:
            v.fill_(float("nan"))
        else:
            v.fill_(-1 if v.dtype != torch.uint8 else 255)
    stream = torch.cuda.current_stream(DEV).cuda_stream
    if noalloc:
        st = _lib.forward_noalloc_raw(desc, D["x"].data_ptr(), W, O, stream)
    else:
        st = _lib.forward_raw(desc, D["x"].data_ptr(), W, O, ws.data_ptr(), ws.numel(), stream)
    assert st == _lib.ACE_OK, _lib.status_string(st)
    torch.cuda.synchronize()
    res = {key: o[key].view(torch.int16 if o[key].dtype == torch.bfloat16 else o[key].dtype).cpu().numpy()
           for key in KEYS}
    n = int(res["offsets"][-1])
    res["perm"] = o["perm"][:n].cpu().numpy()
    return res


def _same(a, b, name):
    for key in a:
        assert a[key].dtype == b[key].dtype and a[key].shape == b[key].shape, (name, key)
        assert np.array_equal(a[key].view(np.uint8), b[key].view(np.uint8)), f"{name}: {key} differs"


def _layer(cfg):
    L = synth.make_layer(cfg)
    tabs = _tables(L)
    base = oracle.forward.moe_forward(L, cfg.k, tabs[0].cpu().numpy(), tabs[1].cpu().numpy(), tau=0.0, tokens=[])
    tau = float(np.float32(oracle.tau.tau_table([base["c"]], 1, [0.5])[0.5]))
    return L, device_layer(L), tabs, tau


CASES = [
    # a multi-chunk bf16 layer (grouped GEMMs, plan kernel) with a shared expert and Zipf router
    synth.config("zipf_256", T=300, d=256, N=32, k=4, m=128, m_shared=128, seed=3),
    # a smaller bf16 batch (the small-batch GEMMs, self-planned)
    synth.config("prefill_4096", T=37, d=256, N=32, k=4, m=128, seed=4),
    # a one-chunk fp32 batch, smaller again
    synth.config("tiny_f32", T=9, d=256, N=8, k=2, m=128, seed=5),
]


def test_noalloc_matches_workspace_entry_point():
    for i, cfg in enumerate(CASES):
        L, D, tabs, tau = _layer(cfg)
        ref = _call(L, D, tabs, tau, noalloc=False)
        got = _call(L, D, tabs, tau, noalloc=True)
        _same(ref, got, f"call {i} ({cfg.name}, T={cfg.T})")
        assert ref["keep"].min() == 0 and ref["keep"][:, 0].all(), "some slots skipped, top-1 kept"
        print(f"[noalloc] call {i}: {cfg.name} T={cfg.T} identical to ace_moe_forward "
              f"(skip {1 - ref['keep'].mean():.3f})", flush=True)


def test_noalloc_refuses_a_layer_past_its_scratch():
    cfg = synth.config("prefill_4096", T=8, d=256, N=16, k=4, m=128, seed=6)
    L, D, tabs, tau = _layer(cfg)
    # the same tensors, described as a 4096-token layer of the 2048-hidden shape, need
    # ~200 MB of scratch: refused on the host, before any launch
    desc = _lib.Desc(4096, 2048, 128, 8, 768, 0, 0, _lib.ACE_BF16, 1, tau, 1e-6, 1e-6, 0)
    assert _lib.workspace_size(desc) > _lib.NOALLOC_SCRATCH_BYTES
    _, W, O, o, _ = _marshal(D["x"], D, tabs[0], tabs[1], cfg.k, tau, 1, 1e-6, 1e-6, False, False, True, None,
                             torch.empty(1, dtype=torch.uint8, device=DEV), "max")
    o["y"].fill_(7.0)
    torch.cuda.synchronize()
    st = _lib.forward_noalloc_raw(desc, D["x"].data_ptr(), W, O, torch.cuda.current_stream(DEV).cuda_stream)
    assert st == _lib.ACE_ERR_SCRATCH_LIMIT
    assert "SCRATCH_LIMIT" in _lib.status_string(st)
    torch.cuda.synchronize()
    assert bool((o["y"] == 7.0).all()), "a refused call must enqueue nothing"
    # and the largest layer that fits is accepted by the size rule
    ok = _lib.Desc(1361, 2048, 128, 8, 768, 0, 0, _lib.ACE_BF16, 1, tau, 1e-6, 1e-6, 0)
    assert _lib.workspace_size(ok) <= _lib.NOALLOC_SCRATCH_BYTES
