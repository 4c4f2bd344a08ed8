"""Properties of the HIP path that hold at any size (needs an MI355X).

Bitwise: replaying the whole prefix equals the forward's final state (Eq. 2
with k = m), a varlen batch equals per-sequence calls, grouped heads equal the
matching single-head problem, repeated runs are identical, an empty replay is
exactly zero (the zero-only baseline), in-place state update equals the
out-of-place one.  Within tolerance: splitting a sequence at any token and
handing the state over equals one call.
"""
import numpy as np
import pytest
import torch

import paper_2608_30310_amd as gdn
import synth
from tests.gpu_util import STATE_TOL, OUTPUT_TOL, device_inputs, oracle_run, state_err, to_f64

pytestmark = pytest.mark.gpu

SHAPE = synth.Shape(hk=2, hv=4, dk=128, dv=128, dtype="bf16")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    gdn.load_library()


def _seq(seq, n, start=0, shape=SHAPE, gate_scale=0.1):
    return synth.tokens(200, 0, seq, start, start + n, shape, gate_scale)


def test_replay_of_whole_prefix_is_full_prefill_bitwise():
    # below 20 chunks tail replay runs one chain, as the forward does
    p = synth.pack([_seq(0, 333)])
    x = device_inputs(p)
    st = gdn.tail_replay(x["k"], x["v"], x["g"], x["beta"], x["cu"], x["cu_host"])
    _, st_f = gdn.chunk_forward(x["q"], x["k"], x["v"], x["g"], x["beta"], x["cu"], x["cu_host"])
    assert torch.equal(st, st_f)


def test_varlen_batch_equals_separate_calls_bitwise():
    lens = [130, 0, 64, 1, 257]
    seqs = [_seq(i, n) for i, n in enumerate(lens)]
    p = synth.pack(seqs)
    x = device_inputs(p)
    st = gdn.tail_replay(x["k"], x["v"], x["g"], x["beta"], x["cu"], x["cu_host"])
    o, st_f = gdn.chunk_forward(x["q"], x["k"], x["v"], x["g"], x["beta"], x["cu"], x["cu_host"],
                                state_in=st)
    for i, s in enumerate(seqs):
        xi = device_inputs(synth.pack([s]))
        sti = gdn.tail_replay(xi["k"], xi["v"], xi["g"], xi["beta"], xi["cu"], xi["cu_host"])
        assert torch.equal(st[i], sti[0])
        oi, sfi = gdn.chunk_forward(xi["q"], xi["k"], xi["v"], xi["g"], xi["beta"], xi["cu"],
                                    xi["cu_host"], state_in=sti)
        a, b = int(p.cu_seqlens[i]), int(p.cu_seqlens[i + 1])
        assert torch.equal(o[a:b], oi)
        assert torch.equal(st_f[i], sfi[0])


def test_grouped_heads_equal_single_head_problems_bitwise():
    p = synth.pack([_seq(0, 200)])
    x = device_inputs(p)
    st = gdn.tail_replay(x["k"], x["v"], x["g"], x["beta"], x["cu"], x["cu_host"])
    o, _ = gdn.chunk_forward(x["q"], x["k"], x["v"], x["g"], x["beta"], x["cu"], x["cu_host"])
    grp = SHAPE.hv // SHAPE.hk
    for h in range(SHAPE.hv):
        kh = h // grp
        sl = lambda t, a: t[:, a:a + 1].contiguous()
        sth = gdn.tail_replay(sl(x["k"], kh), sl(x["v"], h), sl(x["g"], h), sl(x["beta"], h),
                              x["cu"], x["cu_host"])
        oh, _ = gdn.chunk_forward(sl(x["q"], kh), sl(x["k"], kh), sl(x["v"], h), sl(x["g"], h),
                                  sl(x["beta"], h), x["cu"], x["cu_host"])
        assert torch.equal(st[:, h], sth[:, 0])
        assert torch.equal(o[:, h], oh[:, 0])


def test_repeated_runs_are_identical():
    p = synth.pack([_seq(0, 700), _seq(1, 90)])
    x = device_inputs(p)
    ref_st = gdn.tail_replay(x["k"], x["v"], x["g"], x["beta"], x["cu"], x["cu_host"]).clone()
    ref_o, _ = gdn.chunk_forward(x["q"], x["k"], x["v"], x["g"], x["beta"], x["cu"],
                                 x["cu_host"], state_in=ref_st)
    ref_o = ref_o.clone()
    for _ in range(10):
        st = gdn.tail_replay(x["k"], x["v"], x["g"], x["beta"], x["cu"], x["cu_host"])
        o, _ = gdn.chunk_forward(x["q"], x["k"], x["v"], x["g"], x["beta"], x["cu"],
                                 x["cu_host"], state_in=st)
        assert torch.equal(st, ref_st) and torch.equal(o, ref_o)


def test_zero_length_replay_is_the_zero_only_baseline():
    p = synth.pack([_seq(0, 0), _seq(1, 0)], SHAPE)
    x = device_inputs(p)
    st = gdn.tail_replay(x["k"], x["v"], x["g"], x["beta"], x["cu"], x["cu_host"])
    assert st.shape == (2, SHAPE.hv, SHAPE.dk, SHAPE.dv)
    assert torch.count_nonzero(st).item() == 0
    s0 = torch.randn_like(st)
    o, s1 = gdn.chunk_forward(x["q"], x["k"], x["v"], x["g"], x["beta"], x["cu"], x["cu_host"],
                              state_in=s0)
    assert o.numel() == 0 and torch.equal(s1, s0)


def test_no_sequences_is_a_no_op():
    p = synth.pack([], SHAPE)
    x = device_inputs(p)
    st = gdn.tail_replay(x["k"], x["v"], x["g"], x["beta"], x["cu"], x["cu_host"])
    assert st.shape == (0, SHAPE.hv, SHAPE.dk, SHAPE.dv)


def test_in_place_state_update_matches_out_of_place():
    p = synth.pack([_seq(0, 150), _seq(1, 70)])
    x = device_inputs(p)
    s0 = torch.randn(2, SHAPE.hv, SHAPE.dk, SHAPE.dv, device="cuda") * 0.2
    o1, s1 = gdn.chunk_forward(x["q"], x["k"], x["v"], x["g"], x["beta"], x["cu"], x["cu_host"],
                               state_in=s0)
    s_inplace = s0.clone()
    o2, s2 = gdn.chunk_forward(x["q"], x["k"], x["v"], x["g"], x["beta"], x["cu"], x["cu_host"],
                               state_in=s_inplace, state_out=s_inplace)
    assert s2.data_ptr() == s_inplace.data_ptr()
    assert torch.equal(o1, o2) and torch.equal(s1, s2)


@pytest.mark.parametrize("split", [1, 37, 64, 100, 191])
def test_state_hand_off_at_any_token(split):
    n = 256
    whole = synth.pack([_seq(0, n)])
    head = synth.pack([_seq(0, split)])
    rest = synth.pack([_seq(0, n - split, start=split)])
    xw, xh, xr = device_inputs(whole), device_inputs(head), device_inputs(rest)
    o, s = gdn.chunk_forward(xw["q"], xw["k"], xw["v"], xw["g"], xw["beta"], xw["cu"],
                             xw["cu_host"])
    oh, sh = gdn.chunk_forward(xh["q"], xh["k"], xh["v"], xh["g"], xh["beta"], xh["cu"],
                               xh["cu_host"])
    orr, sr = gdn.chunk_forward(xr["q"], xr["k"], xr["v"], xr["g"], xr["beta"], xr["cu"],
                                xr["cu_host"], state_in=sh)
    assert state_err(to_f64(sr), to_f64(s)) <= STATE_TOL / 10
    o_cat = torch.cat([oh, orr])
    rel = (o_cat.float() - o.float()).norm() / o.float().norm()
    assert rel.item() <= OUTPUT_TOL / 5
    # and both agree with the oracle
    _, want = oracle_run(whole)
    assert state_err(to_f64(sr), want) <= STATE_TOL


@pytest.mark.parametrize("gate_scale", [0.02, 0.5, 2.0])
def test_gate_scales(gate_scale):
    p = synth.pack([_seq(0, 300, gate_scale=gate_scale)])
    x = device_inputs(p)
    st = gdn.tail_replay(x["k"], x["v"], x["g"], x["beta"], x["cu"], x["cu_host"])
    _, want = oracle_run(p)
    assert state_err(to_f64(st), want) <= STATE_TOL


def test_adversarial_repeated_keys():
    """Identical keys in a chunk (A has all-equal entries): the triangular solve
    must stay accurate."""
    shape = synth.Shape(hk=1, hv=1, dk=64, dv=64, dtype="f32")
    t = synth.tokens(201, 0, 0, 0, 192, shape)
    t.k[:] = t.k[0]
    t.beta[:] = 0.999
    t.g[:] = -1e-4
    p = synth.pack([t])
    x = device_inputs(p)
    st = gdn.tail_replay(x["k"], x["v"], x["g"], x["beta"], x["cu"], x["cu_host"])
    _, want = oracle_run(p)
    assert state_err(to_f64(st), want) <= STATE_TOL


def test_whole_head_and_column_kernels_agree():
    # 72 sequences x 4 heads exceed the chip with the column-split scan (one
    # workgroup per 32 columns), so the batch's tail replay runs on the wide
    # column scan (two tiles per wave) and its forward on the whole-head
    # kernel; single sequences run on the 32-wide column scan (one tile per
    # wave).  Same products in the same order: the replayed states agree bit
    # for bit.
    lens = [1 + (37 * i) % 200 for i in range(72)]
    seqs = [_seq(i, n) for i, n in enumerate(lens)]
    x = device_inputs(synth.pack(seqs))
    st = gdn.tail_replay(x["k"], x["v"], x["g"], x["beta"], x["cu"], x["cu_host"])
    o, _ = gdn.chunk_forward(x["q"], x["k"], x["v"], x["g"], x["beta"], x["cu"], x["cu_host"],
                             state_in=st)
    cu = synth.pack(seqs).cu_seqlens
    for i in (0, 5, 71):
        xi = device_inputs(synth.pack([seqs[i]]))
        sti = gdn.tail_replay(xi["k"], xi["v"], xi["g"], xi["beta"], xi["cu"], xi["cu_host"])
        oi, _ = gdn.chunk_forward(xi["q"], xi["k"], xi["v"], xi["g"], xi["beta"], xi["cu"],
                                  xi["cu_host"], state_in=sti)
        assert torch.equal(st[i:i + 1], sti), f"sequence {i}: wide and 32-wide replays differ"
        a, b = int(cu[i]), int(cu[i + 1])
        rel = (o[a:b].float() - oi.float()).norm() / oi.float().norm()
        assert rel.item() <= 1e-3   # bf16 outputs: one rounding step apart at most


@pytest.mark.parametrize("nseq", [3, 12, 36])
def test_one_tile_and_wide_batches_bitwise(nseq):
    # 3 and 12 sequences at 32 value heads run in the 64-column one-tile scan
    # (at most three rounds of MI355X's 256 CUs); 36 run wide (1152
    # workgroups, two per CU), whose last round would be a quarter full, so
    # the four shortest run in the one-tile scan after it.  Every sequence's
    # state must be bitwise that of its own call (the one-tile, two-tile and
    # 32-column chains run the same products).
    shape = synth.Shape(hk=16, hv=32, dk=128, dv=128, dtype="bf16")
    lens = [64 + (37 * i) % 200 for i in range(nseq)]
    seqs = [_seq(i, n, shape=shape) for i, n in enumerate(lens)]
    x = device_inputs(synth.pack(seqs))
    st = gdn.tail_replay(x["k"], x["v"], x["g"], x["beta"], x["cu"], x["cu_host"])
    for i in range(len(seqs)):
        xi = device_inputs(synth.pack([seqs[i]]))
        sti = gdn.tail_replay(xi["k"], xi["v"], xi["g"], xi["beta"], xi["cu"], xi["cu_host"])
        assert torch.equal(st[i:i + 1], sti), f"sequence {i} (length {lens[i]})"


@pytest.mark.parametrize("nseq,d", [(12, 128), (36, 128), (12, 64)])
def test_forward_batches_with_a_peeled_last_round(nseq, d):
    # 12 and 36 sequences at 32 value heads run the forward on the whole-head
    # kernel (384 and 1152 workgroups, one per CU); the last round would hold
    # 128 of 256, so the four shortest sequences run in the 32-column scan
    # with output waves after it.  States agree bit for bit with each
    # sequence's own call (same products, same order); outputs to within one
    # bf16 rounding (the whole-head kernel sums the output's two terms in
    # another order).  At d = 64 the same holds with two 32-column groups per
    # head.
    shape = synth.Shape(hk=16, hv=32, dk=d, dv=d, dtype="bf16")
    lens = [64 + (37 * i) % 200 for i in range(nseq)]
    seqs = [_seq(i, n, shape=shape) for i, n in enumerate(lens)]
    p = synth.pack(seqs)
    x = device_inputs(p)
    st = gdn.tail_replay(x["k"], x["v"], x["g"], x["beta"], x["cu"], x["cu_host"])
    o, st_f = gdn.chunk_forward(x["q"], x["k"], x["v"], x["g"], x["beta"], x["cu"], x["cu_host"],
                                state_in=st)
    for i in range(nseq):
        xi = device_inputs(synth.pack([seqs[i]]))
        oi, sfi = gdn.chunk_forward(xi["q"], xi["k"], xi["v"], xi["g"], xi["beta"], xi["cu"],
                                    xi["cu_host"], state_in=st[i:i + 1].contiguous())
        assert torch.equal(st_f[i:i + 1], sfi), f"sequence {i} (length {lens[i]})"
        a, b = int(p.cu_seqlens[i]), int(p.cu_seqlens[i + 1])
        rel = (o[a:b].float() - oi.float()).norm() / oi.float().norm()
        assert rel.item() <= 1e-3, f"sequence {i} (length {lens[i]})"


def test_fp32_forward_beyond_the_chip_bitwise():
    # fp32 inputs with outputs: 72 varlen sequences x 4 heads need 1152
    # 32-column workgroups, more than the chip holds, and run in that form over
    # several rounds, longest first; single sequences fit and run the same
    # body.  States and outputs agree bit for bit.
    shape = synth.Shape(hk=2, hv=4, dk=128, dv=128, dtype="f32")
    lens = [1 + (37 * i) % 200 for i in range(72)]
    seqs = [_seq(i, n, shape=shape) for i, n in enumerate(lens)]
    p = synth.pack(seqs)
    x = device_inputs(p)
    st = gdn.tail_replay(x["k"], x["v"], x["g"], x["beta"], x["cu"], x["cu_host"])
    o, st_f = gdn.chunk_forward(x["q"], x["k"], x["v"], x["g"], x["beta"], x["cu"], x["cu_host"],
                                state_in=st)
    for i in (0, 5, 40, 71):
        xi = device_inputs(synth.pack([seqs[i]]))
        oi, sfi = gdn.chunk_forward(xi["q"], xi["k"], xi["v"], xi["g"], xi["beta"], xi["cu"],
                                    xi["cu_host"], state_in=st[i:i + 1].contiguous())
        a, b = int(p.cu_seqlens[i]), int(p.cu_seqlens[i + 1])
        assert torch.equal(o[a:b], oi), f"sequence {i} (length {lens[i]})"
        assert torch.equal(st_f[i:i + 1], sfi), f"sequence {i} (length {lens[i]})"


def test_two_heads_per_preparation_workgroup_bitwise():
    # 64 sequences at 32 value heads (two per key head): the tail's chunk
    # preparation grid exceeds one round of the chip, so each workgroup
    # prepares both value heads of a key head; single sequences prepare one
    # head per workgroup.  The per-head arithmetic is the same, and the wide
    # and 32-wide scans agree bit for bit, so the states do too.
    shape = synth.Shape(hk=16, hv=32, dk=128, dv=128, dtype="bf16")
    lens = [1 + (97 * i) % 300 for i in range(64)]
    seqs = [_seq(i, n, shape=shape) for i, n in enumerate(lens)]
    x = device_inputs(synth.pack(seqs))
    st = gdn.tail_replay(x["k"], x["v"], x["g"], x["beta"], x["cu"], x["cu_host"])
    for i in (0, 17, 63):
        xi = device_inputs(synth.pack([seqs[i]]))
        sti = gdn.tail_replay(xi["k"], xi["v"], xi["g"], xi["beta"], xi["cu"], xi["cu_host"])
        assert torch.equal(st[i:i + 1], sti), f"sequence {i} (length {lens[i]})"


@pytest.mark.parametrize("case", ["one", "ragged", "wide", "ragged_d64", "ragged_dk64", "ragged_dv64", "split",
                                  "split_no_suffix"])
def test_replay_forward_equals_the_two_calls_bitwise(case):
    # the fused call runs the same kernels (the suffix's chunk preparation
    # beside the tail scan), so it must reproduce tail_replay + chunk_forward
    # "ragged*" covers an empty tail and an empty suffix at every (d_k, d_v)
    # the kernels are built for; "wide" runs the whole-head scan kernel;
    # "split*": a 21-chunk tail at 32 heads, which both run in two halves (the
    # fused call with the suffix's preparation beside the split scan, or with
    # no suffix at all)
    shape = {"ragged_d64": synth.Shape(hk=2, hv=4, dk=64, dv=64, dtype="bf16"),
             "ragged_dk64": synth.Shape(hk=2, hv=4, dk=64, dv=128, dtype="bf16"),
             "ragged_dv64": synth.Shape(hk=2, hv=4, dk=128, dv=64, dtype="bf16"),
             "split": synth.Shape(hk=16, hv=32, dk=128, dv=128, dtype="bf16"),
             "split_no_suffix": synth.Shape(hk=16, hv=32, dk=128, dv=128, dtype="bf16")}.get(case, SHAPE)
    if case == "one":
        rs, ss = [333], [200]
    elif case == "split":
        rs, ss = [1300], [200]
    elif case == "split_no_suffix":
        rs, ss = [1300], [0]
    elif case.startswith("ragged"):
        rs, ss = [0, 1, 64, 130, 257], [65, 0, 1, 200, 64]
    else:   # enough heads that the whole-head scan kernel runs
        rs = [1 + (37 * i) % 150 for i in range(72)]
        ss = [1 + (53 * i) % 120 for i in range(72)]
    tails = synth.pack([_seq(i, r, start=0, shape=shape) for i, r in enumerate(rs)])
    sufs = synth.pack([_seq(i, s, start=r, shape=shape) for i, (r, s) in enumerate(zip(rs, ss))])
    xt, xs = device_inputs(tails), device_inputs(sufs)
    st = gdn.tail_replay(xt["k"], xt["v"], xt["g"], xt["beta"], xt["cu"], xt["cu_host"])
    o, st2 = gdn.chunk_forward(xs["q"], xs["k"], xs["v"], xs["g"], xs["beta"], xs["cu"],
                               xs["cu_host"], state_in=st, scale=0.7)
    of, mid, stf = gdn.replay_forward(xt["k"], xt["v"], xt["g"], xt["beta"], xt["cu"],
                                      xs["q"], xs["k"], xs["v"], xs["g"], xs["beta"], xs["cu"],
                                      cu_tail_host=xt["cu_host"], cu_suf_host=xs["cu_host"],
                                      scale=0.7)
    assert torch.equal(mid, st)
    assert torch.equal(of, o)
    assert torch.equal(stf, st2)


@pytest.mark.parametrize("r,slow", [(1300, True), (1638, False), (2000, True), (3277, True), (3277, False)])
def test_split_replay_agrees_with_one_chain(r, slow):
    """One sequence at 32 heads replays in two halves (the first half's state,
    the second half's from zero and its transition, combined), and so does the
    fused call's tail (bit for bit); the same sequence in a batch of two
    exceeds the split grid and runs one chain.  The two forms differ by
    rounding order only.
    `slow`: gates that decay slowly (scale 0.002, beta x 0.1), so the first
    half's share of the state is large and the combine is exercised."""
    import dataclasses
    shape = synth.Shape(hk=16, hv=32, dk=128, dv=128, dtype="bf16")
    s = synth.tokens(207, 0, 0, 0, r, shape, gate_scale=0.002 if slow else 0.1)
    if slow:
        s = dataclasses.replace(s, beta=(s.beta * 0.1).astype(np.float32))
    x1, x2 = device_inputs(synth.pack([s])), device_inputs(synth.pack([s, s]))
    split = gdn.tail_replay(x1["k"], x1["v"], x1["g"], x1["beta"], x1["cu"], x1["cu_host"])
    chain = gdn.tail_replay(x2["k"], x2["v"], x2["g"], x2["beta"], x2["cu"], x2["cu_host"])
    assert torch.equal(chain[0], chain[1])
    e = state_err(to_f64(split), to_f64(chain[:1]))
    xs = device_inputs(synth.pack([synth.tokens(207, 0, 0, r, r + 64, shape)]))
    # (the suffix only completes the fused call; its outputs are not compared)
    _, mid, _ = gdn.replay_forward(x1["k"], x1["v"], x1["g"], x1["beta"], x1["cu"],
                                   xs["q"], xs["k"], xs["v"], xs["g"], xs["beta"], xs["cu"],
                                   cu_tail_host=x1["cu_host"], cu_suf_host=xs["cu_host"])
    e_mid = state_err(to_f64(mid), to_f64(split))
    print(f"[split] r={r}: split vs one chain {e:.2e}, fused tail vs split {e_mid:.2e}", flush=True)
    # each form is within ~5e-4 of the exact state (bf16 inputs: hi(T) alone in
    # T R), and the two round differently, so they differ by at most 1e-3
    assert e <= 1e-3
    assert torch.equal(mid, split)


def test_varlen_graph_with_longest_first_order():
    """An unsorted varlen batch whose scan grids exceed the chip (wide tail
    scan, whole-head forward): both run in longest-first order, which travels
    in the kernels' arguments.  Tail replay and forward captured in one HIP
    graph replay bitwise like the eager calls, three times, with other eager
    work between the replays."""
    shape = synth.Shape(hk=8, hv=16, dk=128, dv=128, dtype="bf16")
    lens = [70, 700, 3, 300, 1000, 64]          # 6 x 16 x 4 = 384 column groups > 256 CUs
    p = synth.pack([_seq(i, n, shape=shape) for i, n in enumerate(lens)])
    x = device_inputs(p)
    n = len(lens)
    st = torch.empty((n, shape.hv, shape.dk, shape.dv), dtype=torch.float32, device="cuda")
    st2 = torch.empty_like(st)
    o = torch.empty_like(x["v"])
    ws_t = torch.empty(gdn.workspace_size(n, shape.hk, shape.hv, shape.dk, shape.dv, p.cu_seqlens.tolist()) + 256,
                       dtype=torch.uint8, device="cuda")
    ws_f = torch.empty(gdn.workspace_size(n, shape.hk, shape.hv, shape.dk, shape.dv, p.cu_seqlens.tolist(),
                                          with_outputs=True) + 256, dtype=torch.uint8, device="cuda")

    def calls():
        gdn.tail_replay(x["k"], x["v"], x["g"], x["beta"], x["cu"], x["cu_host"], state_out=st, workspace=ws_t)
        gdn.chunk_forward(x["q"], x["k"], x["v"], x["g"], x["beta"], x["cu"], x["cu_host"], state_in=st,
                          o=o, state_out=st2, workspace=ws_f, scale=0.5)

    calls()
    torch.cuda.synchronize()
    ref = (st.clone(), st2.clone(), o.clone())
    # each sequence as its own call: the order only moves work between workgroups
    for i, s in enumerate(lens):
        xi = device_inputs(synth.pack([_seq(i, s, shape=shape)]))
        sti = gdn.tail_replay(xi["k"], xi["v"], xi["g"], xi["beta"], xi["cu"], xi["cu_host"])
        assert state_err(to_f64(ref[0][i:i + 1]), to_f64(sti)) <= 1e-5
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        calls()
    torch.cuda.current_stream().wait_stream(side)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        calls()
    for rep in range(3):
        st.zero_()
        st2.zero_()
        o.zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(st, ref[0]) and torch.equal(st2, ref[1]) and torch.equal(o, ref[2]), f"replay {rep}"
        junk = torch.randn(1 << 20, device="cuda").sum()
        torch.cuda.synchronize()
        del junk
