"""Dispatch plan on the GPU across the shapes that select its kernels (and the
small bf16 batches whose gate/up waves derive it themselves).

Batches above 16 router chunks get their plan from plan_kernel when the
[chunks, experts] count matrix is at most 128 KB and the expert count is a
multiple of 4 (16-byte rows when a multiple of 16, else 4-byte rows), and from
expert_scan + scatter otherwise.  Each case checks every routing decision and
the whole plan against the oracle (counts, offsets, the permutation in
(expert, token) order, slot rows), and outputs on a token sample."""
import pytest

import oracle
import synth
from gpu_helpers import device_layer, full_check

pytestmark = pytest.mark.gpu

CASES = [
    # (T, N, k): kernel taken
    (600, 64, 8),      # one kernel, 16-byte rows
    (1000, 36, 4),     # one kernel, 4-byte rows
    (700, 30, 4),      # two kernels: N not a multiple of 4
    (8192, 256, 2),    # one kernel at the 128 KB limit (512 chunks x 256 experts)
    (8208, 256, 2),    # two kernels: one chunk past it
    (4097, 128, 8),    # one kernel, ragged last chunk (one token)
    (4200, 16, 2),     # router: chunk pairs with one 16-expert tile (all experts per wave)
    (4200, 30, 4),     # router: chunk pairs with two expert tiles (one per wave); two plan kernels
]


@pytest.mark.parametrize("T,N,k", CASES, ids=[f"T{t}_N{n}_k{k}" for t, n, k in CASES])
def test_plan_kernels(T, N, k):
    L = synth.make_layer(synth.config("prefill_4096", T=T, d=128, N=N, k=k, m=64, seed=50 + N))
    tb = oracle.tables.build_tables(L)
    base = oracle.forward.moe_forward(L, k, tb["a_gsp"], tb["a_rcr"], tau=0.0, tokens=[])
    tau = float(oracle.tau.tau_table([base["c"]], 1, [0.5])[0.5])
    r = full_check(L, device_layer(L), tb["a_gsp"], tb["a_rcr"], tau, tokens=range(0, T, 37))
    print(f"[plan T={T} N={N} k={k}] skip={1 - r['gpu']['keep'].mean():.3f} rel_l2={r['rel_l2']:.2e} "
          f"tied={len(r['ties']['tied'])}", flush=True)


SELF_PLAN = [
    # (T, N, k, m_min, skip_disable): bf16 batches of 2-4 router chunks, planned by the gate/up waves
    (17, 64, 8, 1, False),     # two chunks, one token in the second
    (31, 36, 4, 2, False),     # N not a multiple of 4 (byte-wise counts), m_min restore
    (48, 128, 8, 1, True),     # plain top-k: every slot kept
    (64, 256, 8, 3, False),    # four chunks, 256 experts (all 64 lanes hold experts)
    (40, 12, 1, 1, False),     # top-1 only
]


@pytest.mark.parametrize("T,N,k,m_min,sd", SELF_PLAN, ids=[f"T{t}_N{n}_k{k}_mmin{mm}{'_topk' if sd else ''}"
                                                          for t, n, k, mm, sd in SELF_PLAN])
def test_self_planned_small_batches(T, N, k, m_min, sd):
    """Small bf16 batches whose skinny gate/up waves derive the plan themselves:
    routing, masks, counts, offsets and the permutation against the oracle, and
    every output row."""
    L = synth.make_layer(synth.config("prefill_4096", T=T, d=256, N=N, k=k, m=128, seed=70 + T))
    tb = oracle.tables.build_tables(L)
    base = oracle.forward.moe_forward(L, k, tb["a_gsp"], tb["a_rcr"], tau=0.0, m_min=m_min, tokens=[])
    tau = float(oracle.tau.tau_table([base["c"]], m_min, [0.5])[0.5])
    r = full_check(L, device_layer(L), tb["a_gsp"], tb["a_rcr"], tau, m_min=m_min, skip_disable=sd)
    keep = r["gpu"]["keep"].astype(bool)
    assert keep[:, 0].all() and (keep.sum(axis=1) >= m_min).all()
    if sd:
        assert keep.all()
    print(f"[self-plan T={T} N={N} k={k} m_min={m_min}] skip={1 - keep.mean():.3f} rel_l2={r['rel_l2']:.2e}",
          flush=True)
