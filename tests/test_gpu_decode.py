"""Decode step (one token per sequence from a given state) vs the fp64 oracle.

The oracle runs Eq. 1 over N one-token sequences from the same state.  The
kernel computes in fp32 throughout: each state element takes part in two dot
products of length d_k <= 128, accumulated in fp32, so the relative error of
states and fp32 outputs stays below d_k * 2^-24 ~ 1e-5 (asserted), far inside
the 2e-3 / 5e-3 bar; bf16 outputs carry one bf16 rounding (2^-9 relative) and
are held to the 5e-3 output bar.
"""
import numpy as np
import pytest
import torch

import paper_2608_30310_amd as gdn
import synth
from tests.gpu_util import (OUTPUT_TOL, STATE_TOL, device_inputs, oracle_run, output_err,
                            state_err, to_f64)

pytestmark = pytest.mark.gpu

FP32_TOL = 1e-5


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    gdn.load_library()


def _report(name, **errs):
    print(f"[decode] {name}: " + ", ".join(f"{k}={v:.3e}" for k, v in errs.items()), flush=True)


def _batch(workload, n, shape, pos=0):
    """n sequences, token `pos` of each (one token per sequence)."""
    return synth.pack([synth.tokens(workload, 0, i, pos, pos + 1, shape) for i in range(n)])


def _state(seed, n, shape):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((n, shape.hv, shape.dk, shape.dv)) * 0.3).astype(np.float32)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("dk,dv", [(64, 64), (128, 128), (64, 128), (128, 64)])
@pytest.mark.parametrize("grp", [1, 2])
def test_decode_step_parity(dtype, dk, dv, grp):
    shape = synth.Shape(hk=2, hv=2 * grp, dk=dk, dv=dv, dtype=dtype)
    n = 5
    p = _batch(120, n, shape)
    x = device_inputs(p)
    s0 = _state(9, n, shape)
    o, st = gdn.decode_step(x["q"], x["k"], x["v"], x["g"], x["beta"],
                            state_in=torch.from_numpy(s0).cuda(), scale=0.6)
    wo, ws = oracle_run(p, state_in=s0.astype(np.float64), outputs=True, scale=0.6)
    e_st = state_err(to_f64(st), ws)
    e_o = output_err(to_f64(o), wo, p.cu_seqlens)
    _report(f"{dtype} dk={dk} dv={dv} grp={grp}", state=e_st, out=e_o)
    assert e_st <= FP32_TOL
    assert e_o <= (FP32_TOL if dtype == "f32" else OUTPUT_TOL)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_decode_in_place_and_zero_state(dtype):
    shape = synth.Shape(hk=2, hv=4, dk=128, dv=128, dtype=dtype)
    n = 3
    p = _batch(121, n, shape)
    x = device_inputs(p)
    s0 = torch.from_numpy(_state(10, n, shape)).cuda()
    o_a, st_a = gdn.decode_step(x["q"], x["k"], x["v"], x["g"], x["beta"], state_in=s0, scale=0.5)
    s_in = s0.clone()
    o_b, st_b = gdn.decode_step(x["q"], x["k"], x["v"], x["g"], x["beta"], state_in=s_in,
                                state_out=s_in, scale=0.5)
    torch.cuda.synchronize()
    assert st_b.data_ptr() == s_in.data_ptr()
    assert torch.equal(st_a, st_b) and torch.equal(o_a, o_b), "in-place update must be bitwise the same"
    # zero state: M1 = k (beta v)^T, o = scale beta v (k . q)
    o_z, st_z = gdn.decode_step(x["q"], x["k"], x["v"], x["g"], x["beta"], state_in=None, scale=0.5)
    wo, ws = oracle_run(p, state_in=None, outputs=True, scale=0.5)
    e_st = state_err(to_f64(st_z), ws)
    e_o = output_err(to_f64(o_z), wo, p.cu_seqlens)
    _report(f"zero state {dtype}", state=e_st, out=e_o)
    assert e_st <= FP32_TOL and e_o <= (FP32_TOL if dtype == "f32" else OUTPUT_TOL)


def test_decode_steps_continue_the_chunked_forward():
    """Replay a tail, then six decode steps, equals the oracle over tail + 6 tokens."""
    shape = synth.Shape(hk=2, hv=4, dk=128, dv=128, dtype="bf16")
    n, tail, steps = 3, 150, 6
    seqs = [synth.tokens(122, 0, i, 0, tail + steps, shape) for i in range(n)]
    full = synth.pack(seqs)
    tail_p = synth.pack([synth.tokens(122, 0, i, 0, tail, shape) for i in range(n)])
    xt = device_inputs(tail_p)
    st = gdn.tail_replay(xt["k"], xt["v"], xt["g"], xt["beta"], xt["cu"], xt["cu_host"])
    outs = []
    for j in range(steps):
        xj = device_inputs(synth.pack([synth.tokens(122, 0, i, tail + j, tail + j + 1, shape)
                                       for i in range(n)]))
        o, st = gdn.decode_step(xj["q"], xj["k"], xj["v"], xj["g"], xj["beta"], state_in=st,
                                state_out=st, scale=0.4)
        outs.append(to_f64(o))
    wo, ws = oracle_run(full, outputs=True, scale=0.4)
    e_st = state_err(to_f64(st), ws)
    got = np.stack(outs, axis=1)                       # [n, steps, hv, dv]
    cu = full.cu_seqlens
    want = np.stack([wo[cu[i] + tail:cu[i] + tail + steps] for i in range(n)])
    e_o = max(np.linalg.norm(got[i, :, h] - want[i, :, h]) / np.linalg.norm(want[i, :, h])
              for i in range(n) for h in range(shape.hv))
    _report("replay + 6 decode steps", state=e_st, out=e_o)
    assert e_st <= STATE_TOL and e_o <= OUTPUT_TOL


def test_decode_batch_at_one_layer_shape():
    """64 sequences at Hk = 16, Hv = 32, d_k = d_v = 128, bf16: the batched
    decode the benchmark times."""
    shape = synth.Shape(hk=16, hv=32, dk=128, dv=128, dtype="bf16")
    n = 64
    p = _batch(123, n, shape)
    x = device_inputs(p)
    s0 = _state(11, n, shape)
    o, st = gdn.decode_step(x["q"], x["k"], x["v"], x["g"], x["beta"],
                            state_in=torch.from_numpy(s0).cuda(), scale=128 ** -0.5)
    wo, ws = oracle_run(p, state_in=s0.astype(np.float64), outputs=True, scale=128 ** -0.5)
    e_st = state_err(to_f64(st), ws)
    e_o = output_err(to_f64(o), wo, p.cu_seqlens)
    _report("batch 64 x 32 heads", state=e_st, out=e_o)
    assert e_st <= FP32_TOL and e_o <= OUTPUT_TOL
