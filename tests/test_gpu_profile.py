"""The measurement hook of the C ABI on the GPU (ace_profile_begin / _begin_span /
_end), which the benchmark's timings come from: per-call stage times in the staged
mode, one span per call in the span mode, calls past the capacity not recorded,
one profile open at a time."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_05228_amd as ace
import synth
from gpu_helpers import DEV, device_layer

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def step():
    L = synth.make_layer(synth.config("prefill_4096", T=300, d=256, N=16, k=4, m=192, seed=11))
    tb = oracle.tables.build_tables(L)
    D = device_layer(L)
    ag = torch.from_numpy(np.asarray(tb["a_gsp"], np.float32)).to(DEV)
    ar = torch.from_numpy(np.asarray(tb["a_rcr"], np.float32)).to(DEV)
    fn = ace.prepare_forward(D["x"], D, ag, ar, k=4, tau=0.1)
    fn()
    torch.cuda.synchronize()
    return fn


def test_staged_profile(step):
    ace.profile_begin(3)
    try:
        for _ in range(4):  # one call past the capacity: not recorded
            step()
    finally:
        tot, n, calls = ace.profile_end(3)
    torch.cuda.synchronize()
    assert n == 3 and len(calls) == 3
    for c in calls:
        for s in ("route", "plan", "gateup", "down", "combine"):
            assert c[s] > 0, (s, c)
        assert c["shared"] == 0  # no shared expert: the stage enqueues nothing
    for s in tot:
        assert tot[s] == pytest.approx(sum(c[s] for c in calls), rel=1e-9, abs=1e-12)


def test_span_profile(step):
    ace.profile_begin(3, span=True)
    try:
        for _ in range(3):
            step()
    finally:
        _, n, calls = ace.profile_end(3)
    torch.cuda.synchronize()
    assert n == 3
    for c in calls:
        assert c["combine"] > 0  # the whole call, from before the first stage to after the last
        assert all(c[s] == 0 for s in ("route", "plan", "gateup", "down", "shared")), c


def test_one_profile_at_a_time(step):
    ace.profile_begin(1)
    try:
        with pytest.raises(ace.AceError):
            ace.profile_begin(1, span=True)
    finally:
        ace.profile_end(0)
    with pytest.raises(ace.AceError):
        ace.profile_end(0)  # nothing open
