"""Dispatch plan on the GPU across the shapes that select its kernels.

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
