"""gdn_tail_replay_noalloc against gdn_tail_replay (needs an MI355X).

The entry point that allocates nothing takes its workspace from the library's
own device array; its states must equal those of gdn_tail_replay, which uses a
caller-owned workspace and the same kernels, bit for bit.  Two calls in a
row, the second with a smaller input (the array keeps the first call's
records, which the second must not read), the first long enough to run the
split tail replay; both also checked against the fp64 oracle.
"""
import numpy as np
import pytest
import torch

import paper_2608_30310_amd as gdn
import synth
from tests.gpu_util import STATE_TOL, device_inputs, oracle_run, state_err, to_f64

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    gdn.load_library()


def _case(seed, lens, shape):
    p = synth.pack([synth.tokens(500 + seed, 0, i, 0, n, shape) for i, n in enumerate(lens)])
    return p, device_inputs(p)


def test_noalloc_matches_tail_replay_twice():
    shape = synth.Shape(hk=16, hv=32, dk=128, dv=128, dtype="bf16")
    for seed, lens in ((0, [3277]), (1, [5, 200, 64])):
        p, x = _case(seed, lens, shape)
        n = len(lens)
        print(f"[noalloc] call with lengths {lens}", flush=True)
        want = gdn.tail_replay(x["k"], x["v"], x["g"], x["beta"], x["cu"], x["cu_host"])
        got = torch.full((n, shape.hv, shape.dk, shape.dv), float("nan"), device="cuda:0")
        gdn.tail_replay_noalloc(x["k"], x["v"], x["g"], x["beta"], x["cu"], x["cu_host"], got)
        torch.cuda.synchronize()
        assert torch.equal(got, want), f"lengths {lens}: states differ from gdn_tail_replay"
        _, w = oracle_run(p)
        e = state_err(to_f64(got), w)
        print(f"[noalloc] lengths {lens}: equal to gdn_tail_replay, oracle error {e:.2e}", flush=True)
        assert e <= STATE_TOL


def test_noalloc_rejects_oversized_input():
    shape = synth.Shape(hk=16, hv=32, dk=128, dv=128, dtype="bf16")
    T = 60000
    k = torch.zeros((T, 16, 128), dtype=torch.bfloat16, device="cuda:0")
    v = torch.zeros((T, 32, 128), dtype=torch.bfloat16, device="cuda:0")
    g = torch.zeros((T, 32), dtype=torch.float32, device="cuda:0")
    cu = torch.tensor([0, T], dtype=torch.int32)
    st = torch.zeros((1, 32, 128, 128), dtype=torch.float32, device="cuda:0")
    with pytest.raises(gdn.GDNError) as ei:
        gdn.tail_replay_noalloc(k, v, g, g, cu.cuda(), cu, st)
    assert ei.value.status == 5
    assert torch.count_nonzero(st).item() == 0
