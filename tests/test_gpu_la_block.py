"""Linear-attention layer block replay (projections, conv, norms, gates and the
recurrence) vs the fp64 layer-block oracle, through the C ABI.

Both sides see the same stored values: bf16 hiddens and projection weights,
fp32 conv taps, gate parameters and norm weights (synth.layer).

Tolerances.  With fp32 intermediates the block adds one rounding to the
recurrence's inputs' path (none: the in-projection multiplies exact bf16
values with fp32 accumulation) and the recurrence runs its fp32 path, so the
states are held to the recurrence's bar (2e-3 max relative Frobenius per
(sequence, head)); the output passes through two bf16 roundings (y, the
out-projection's operand, and out itself), 2^-9 relative each, and is held to
the 5e-3 output bar per sequence.  With bf16 intermediates four more
roundings sit on the path (P, q/k/v, o, y); each is 2^-9 relative at most,
about 1.1e-3 rms, and k enters the delta rule twice, so the state error is
expected near 3-4e-3 (an fp64 simulation of exactly these roundings at the
full layer shape gives 4.1e-3); those runs are held to 1e-2.  Their outputs
are held to 1e-2 per sequence of at least 16 tokens and over the whole batch:
a sequence of one token outputs scale beta v (k . q), a single dot product of
bf16-rounded unit vectors whose relative error grows as 1 / |k . q| (1.3e-2
measured for one such token), and the gated RMS norm carries that relative
error into y unchanged; longer sequences average it out.

Beside the oracle, each case is compared with the oracle's steps carrying
the block's bf16 stores (tests/la_block_model.py): the GPU path and that
model see the same rounded values, so their states are held to the
recurrence's 2e-3 bar and every sequence's outputs, one-token sequences
included, to the 5e-3 output bar, with either intermediate type.
"""
import numpy as np
import pytest
import torch

import paper_2608_30310_amd as gdn
from oracle import la_block as lb
from synth.layer import LayerDims, exact_weights, hiddens, layer_weights, pack_hiddens
from tests.gpu_util import OUTPUT_TOL, STATE_TOL, state_err, to_f64
from tests.la_block_model import la_block_rounded

pytestmark = pytest.mark.gpu

BF16_ACT_TOL = 1e-2


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    gdn.load_library()


def _bf16_dev(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


def _dev_weights(w):
    return {k: (_bf16_dev(a) if a.dtype == np.uint16 else torch.from_numpy(a).cuda()) for k, a in w.items()}


def _x_exact(bits):
    from synth import bf16_bits_to_f32
    return bf16_bits_to_f32(bits).astype(np.float64)


def _case(workload, dims, lens, layer=0):
    x, cu = pack_hiddens([hiddens(workload, layer, i, 0, n, dims.hidden) for i, n in enumerate(lens)],
                         dims.hidden)
    return x, cu, layer_weights(workload, layer, dims)


def _oracle(x, cu, w, dims, scale, outputs):
    we = exact_weights(w)
    return lb.la_block(_x_exact(x), we["w_in"], we["conv_w"], we["a_log"], we["dt_bias"], we["norm_w"],
                       we["w_out"], cu.astype(np.int64), dims.hk, dims.hv, dims.dk, dims.dv, scale,
                       outputs=outputs)


def _gpu_run(x, cu, w, dims, scale, outputs, act, out=None):
    xd = _bf16_dev(x)
    st, o = gdn.la_block_replay(xd, _dev_weights(w), torch.from_numpy(cu).cuda(), dims.hk, dims.hv,
                                dims.dk, dims.dv, scale, cu_seqlens_host=torch.from_numpy(cu.copy()),
                                outputs=outputs, act_dtype=act, out=out)
    torch.cuda.synchronize()
    return st, o


def out_err(got, want, cu, min_len=1):
    """max over sequences (of at least min_len tokens) of ||got - want||_F /
    ||want||_F over the [len, D] block."""
    worst = 0.0
    for n in range(len(cu) - 1):
        a, b = int(cu[n]), int(cu[n + 1])
        if b - a < min_len:
            continue
        den = np.linalg.norm(want[a:b])
        worst = max(worst, np.linalg.norm(got[a:b] - want[a:b]) / den)
    return worst


def _model(x, cu, w, dims, scale, outputs, act):
    we = exact_weights(w)
    return la_block_rounded(_x_exact(x), we["w_in"], we["conv_w"], we["a_log"], we["dt_bias"], we["norm_w"],
                            we["w_out"], cu.astype(np.int64), dims.hk, dims.hv, dims.dk, dims.dv, scale,
                            act, outputs=outputs)


def _check(name, x, cu, w, dims, scale, outputs, act):
    st, o = _gpu_run(x, cu, w, dims, scale, outputs, act)
    ws, wo, _ = _oracle(x, cu, w, dims, scale, outputs)
    e_st = state_err(to_f64(st), ws)
    tol_s = STATE_TOL if act == "f32" else BF16_ACT_TOL
    # against the same steps with the block's bf16 stores: the recurrence's bars
    ms, mo = _model(x, cu, w, dims, scale, outputs, act)
    e_st_m = state_err(to_f64(st), ms)
    assert e_st_m <= STATE_TOL, f"state vs the rounded model {e_st_m:.3e}"
    if outputs:
        e_o_m = out_err(to_f64(o), mo, cu)
        assert e_o_m <= OUTPUT_TOL, f"outputs vs the rounded model {e_o_m:.3e}"
    msg = f"[la_block] {name} act={act} outputs={outputs}: state={e_st:.3e} (rounded model {e_st_m:.3e}" + \
        (f", outputs {e_o_m:.3e})" if outputs else ")")
    if outputs:
        got = to_f64(o)
        if act == "f32":
            e_o = out_err(got, wo, cu)
        else:
            e_o = max(out_err(got, wo, cu, min_len=16),
                      np.linalg.norm(got - wo) / np.linalg.norm(wo) if len(wo) else 0.0)
        msg += f" out={e_o:.3e} (all sequences: {out_err(got, wo, cu):.3e})"
    print(msg, flush=True)
    assert e_st <= tol_s
    if outputs:
        assert e_o <= (OUTPUT_TOL if act == "f32" else BF16_ACT_TOL)
        assert np.all(np.isfinite(to_f64(o)))
    else:
        assert o is None


@pytest.mark.parametrize("act", ["f32", "bf16"])
@pytest.mark.parametrize("outputs", [True, False])
@pytest.mark.parametrize("dk,dv", [(64, 64), (128, 128), (64, 128), (128, 64)])
def test_block_parity_ragged(act, outputs, dk, dv):
    """Five sequences, one empty and one of a single token, lengths that end
    mid-chunk and mid token-block of the prep kernel."""
    dims = LayerDims(hidden=256, hk=2, hv=4, dk=dk, dv=dv)
    x, cu, w = _case(200, dims, [37, 0, 150, 93, 1])
    _check(f"ragged dk={dk} dv={dv}", x, cu, w, dims, dk ** -0.5, outputs, act)


@pytest.mark.parametrize("act", ["f32", "bf16"])
@pytest.mark.parametrize("outputs", [True, False])
def test_block_parity_layer_shape(act, outputs):
    """The benchmark's layer: D = 2048, Hk = 16, Hv = 32, d_k = d_v = 128, one
    replayed tail of 819 tokens (10% of an 8192-token prefix)."""
    dims = LayerDims(hidden=2048, hk=16, hv=32, dk=128, dv=128)
    x, cu, w = _case(201, dims, [819])
    _check("layer shape, tail 819", x, cu, w, dims, 128 ** -0.5, outputs, act)


@pytest.mark.parametrize("act", ["f32", "bf16"])
@pytest.mark.parametrize("outputs", [True, False])
def test_block_prep_four_tokens_per_thread(act, outputs):
    """Enough tokens that the prep kernel takes four consecutive tokens per
    thread (one-token units would fill its grid four times over): sequences
    of 1, 2 and 3 tokens put sequence starts inside a thread's four tokens."""
    dims = LayerDims(hidden=256, hk=2, hv=4, dk=128, dv=128)
    lens = [6001, 1, 2, 3, 5, 7000, 130]
    assert sum(lens) // 8 * 5 >= 4 * 2048   # 5 prep slabs at this shape
    x, cu, w = _case(207, dims, lens)
    _check("four tokens per prep thread", x, cu, w, dims, 0.1, outputs, act)


def test_block_parity_several_tails_layer_shape():
    dims = LayerDims(hidden=2048, hk=16, hv=32, dk=128, dv=128)
    x, cu, w = _case(202, dims, [410, 64, 129, 7])
    _check("layer shape, 4 tails", x, cu, w, dims, 128 ** -0.5, True, "bf16")


@pytest.mark.parametrize("act", ["f32", "bf16"])
def test_block_out_may_alias_x(act):
    dims = LayerDims(hidden=256, hk=2, hv=4, dk=128, dv=128)
    x, cu, w = _case(203, dims, [70, 100])
    st_a, o_a = _gpu_run(x, cu, w, dims, 0.1, True, act)
    xd = _bf16_dev(x)
    st_b, o_b = gdn.la_block_replay(xd, _dev_weights(w), torch.from_numpy(cu).cuda(), dims.hk, dims.hv,
                                    dims.dk, dims.dv, 0.1, outputs=True, act_dtype=act, out=xd)
    torch.cuda.synchronize()
    assert o_b.data_ptr() == xd.data_ptr()
    assert torch.equal(st_a, st_b) and torch.equal(o_a, o_b)


def test_block_with_no_tokens():
    dims = LayerDims(hidden=256, hk=2, hv=4, dk=64, dv=64)
    x, cu, w = _case(204, dims, [0, 0, 0])
    for outputs in (True, False):
        st, o = _gpu_run(x, cu, w, dims, 0.1, outputs, "bf16")
        assert st.shape == (3, 4, 64, 64) and torch.count_nonzero(st) == 0
        if outputs:
            assert o.shape == (0, 256)
    x, cu, w = _case(204, dims, [])
    st, o = _gpu_run(x, cu, w, dims, 0.1, True, "f32")
    assert st.shape[0] == 0 and o.shape == (0, 256)


def test_two_layer_chain():
    """A group's replay without its feed-forward blocks: layer 0 with outputs
    feeds layer 1, which only rebuilds its state.  Both layers' states vs the
    oracle run on the oracle's own layer-0 output rounded to bf16 (the stored
    type of a hidden): the chain's inputs are compared, not assumed."""
    dims = LayerDims(hidden=512, hk=4, hv=8, dk=128, dv=128)
    x, cu, w0 = _case(205, dims, [300, 45])
    w1 = layer_weights(205, 1, dims)
    st0, o0 = _gpu_run(x, cu, w0, dims, 0.1, True, "f32")
    x1 = o0.contiguous()
    st1, _ = gdn.la_block_replay(x1, _dev_weights(w1), torch.from_numpy(cu).cuda(), dims.hk, dims.hv,
                                 dims.dk, dims.dv, 0.1, outputs=False, act_dtype="f32")
    torch.cuda.synchronize()
    ws0, wo0, _ = _oracle(x, cu, w0, dims, 0.1, True)
    from synth import f32_to_bf16_bits
    x1_oracle = f32_to_bf16_bits(wo0.astype(np.float32))
    ws1, _, _ = _oracle(x1_oracle, cu, w1, dims, 0.1, False)
    e0 = state_err(to_f64(st0), ws0)
    e1 = state_err(to_f64(st1), ws1)
    # layer 1 against the oracle on the GPU's own layer-0 output: the same
    # input on both sides, so the recurrence's bar
    x1_gpu = o0.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
    ws1g, _, _ = _oracle(x1_gpu, cu, w1, dims, 0.1, False)
    e1g = state_err(to_f64(st1), ws1g)
    print(f"[la_block] chain: layer0 state={e0:.3e} layer1 state={e1:.3e} (on the GPU's layer-0 output "
          f"{e1g:.3e})", flush=True)
    assert e0 <= STATE_TOL
    assert e1g <= STATE_TOL
    # against the oracle's own chain, layer 1's input differs by the bf16
    # rounding of out on each side (5e-3 bar)
    assert e1 <= BF16_ACT_TOL


@pytest.mark.parametrize("outputs", [True, False])
def test_block_in_a_graph(outputs):
    """The whole call captured in a HIP graph (after one eager call has set up
    the projections) replays bitwise like the eager call, three times, with
    other eager work on the stream between the replays."""
    dims = LayerDims(hidden=512, hk=4, hv=8, dk=128, dv=128)
    # 21 chunks: without outputs the recurrence runs as two halves and a combine
    x, cu, w = _case(206, dims, [1300, 70])
    xd, wd = _bf16_dev(x), _dev_weights(w)
    cu_d, cu_h = torch.from_numpy(cu).cuda(), torch.from_numpy(cu.copy())
    n, T = len(cu) - 1, int(cu[-1])
    st = torch.empty((n, dims.hv, dims.dk, dims.dv), dtype=torch.float32, device="cuda")
    out = torch.empty((T, dims.hidden), dtype=torch.bfloat16, device="cuda") if outputs else None
    ws = torch.empty(gdn.la_block_workspace_size(dims.hidden, dims.hk, dims.hv, dims.dk, dims.dv,
                                                 cu.tolist(), outputs, "bf16") + 256,
                     dtype=torch.uint8, device="cuda")
    call = lambda: gdn.la_block_replay(xd, wd, cu_d, dims.hk, dims.hv, dims.dk, dims.dv, 0.1,
                                       cu_seqlens_host=cu_h, outputs=outputs, act_dtype="bf16",
                                       state_out=st, out=out, workspace=ws)
    call()
    torch.cuda.synchronize()
    st_ref = st.clone()
    out_ref = out.clone() if outputs else None
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        call()
    torch.cuda.current_stream().wait_stream(side)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        call()
    for rep in range(3):
        st.zero_()
        if outputs:
            out.zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(st, st_ref), f"replay {rep}: state differs"
        if outputs:
            assert torch.equal(out, out_ref), f"replay {rep}: output differs"
        junk = torch.randn(1 << 20, device="cuda").sum()   # eager work between replays
        torch.cuda.synchronize()
        del junk
