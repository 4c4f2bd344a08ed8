"""The transfer beside the replay changes no result (paper Section 3, "Replay
efficiency": the full-attention KV moves on a copy stream while the
linear-attention layers replay, and is joined before the query forward;
Table 2, H2D-SER against H2D-OVL).  Needs an MI355X.

The copied region carries, behind a block of filler bytes the size of a
matched prefix's full-attention KV, the suffix inputs (q, k, v, g, beta) of
every layer, and the suffix forwards read them from the copy's destination,
which is cleared before each run.  So a suffix forward that ran before the
copy had landed would read cleared inputs, and its outputs would differ from
the serial order's.  Checked: states and outputs of the overlapped order
equal the serial order's bit for bit on three runs, the copied bytes equal
the source, and the serial results match the fp64 oracle.
"""
import numpy as np
import pytest
import torch

import paper_2608_30310_amd as gdn
import synth
from paper_2608_30310_amd import transfer
from tests.gpu_util import (OUTPUT_TOL, STATE_TOL, device_inputs, oracle_run, output_err,
                            state_err, to_f64)

pytestmark = pytest.mark.gpu

LAYERS, R, S = 4, 819, 512
FILLER = 96 << 20          # bytes of stand-in full-attention KV in front of the suffix inputs


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    gdn.load_library()


def _bytes_of(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a).view(np.uint8).reshape(-1))


def test_overlapped_transfer_matches_serial():
    shape = synth.Shape(hk=16, hv=32, dk=128, dv=128, dtype="bf16")
    m = 8192
    tails = [synth.pack([synth.tokens(120, l, 0, m - R, m, shape)]) for l in range(LAYERS)]
    sufs = [synth.pack([synth.tokens(120, l, 0, m, m + S, shape)]) for l in range(LAYERS)]
    xt = [device_inputs(p) for p in tails]

    # host image of the transfer: filler, then each layer's suffix q, k, v, g, beta
    parts, spans, off = [torch.from_numpy(np.random.default_rng(5).integers(0, 256, FILLER, dtype=np.uint8))], [], FILLER
    for p in sufs:
        layer = {}
        for name in ("q", "k", "v", "g", "beta"):
            b = _bytes_of(getattr(p, name))
            assert b.numel() % 16 == 0
            layer[name] = (off, b.numel(), getattr(p, name).shape)
            parts.append(b)
            off += b.numel()
        spans.append(layer)
    host = torch.empty(off, dtype=torch.uint8, pin_memory=True)
    torch.cat(parts, out=host)
    dev = torch.empty(off, dtype=torch.uint8, device="cuda:0")

    def view(layer, name):
        o, n, shp = spans[layer][name]
        dt = torch.float32 if name in ("g", "beta") else torch.bfloat16
        return dev[o:o + n].view(dt).view(shp)

    cu_s = torch.tensor([0, S], dtype=torch.int32, device="cuda:0")
    cu_s_host = torch.tensor([0, S], dtype=torch.int32)
    mids = [torch.empty((1, 32, 128, 128), dtype=torch.float32, device="cuda:0") for _ in range(LAYERS)]
    fins = [torch.empty_like(mids[0]) for _ in range(LAYERS)]
    outs = [torch.empty((S, 32, 128), dtype=torch.bfloat16, device="cuda:0") for _ in range(LAYERS)]

    def replay():
        for l in range(LAYERS):
            x = xt[l]
            gdn.tail_replay(x["k"], x["v"], x["g"], x["beta"], x["cu"], x["cu_host"], state_out=mids[l])

    def forward():
        for l in range(LAYERS):
            gdn.chunk_forward(view(l, "q"), view(l, "k"), view(l, "v"), view(l, "g"), view(l, "beta"), cu_s,
                              cu_s_host, state_in=mids[l], o=outs[l], state_out=fins[l])

    def clear():
        dev.zero_()
        for t in mids + fins + outs:
            t.zero_()

    clear()
    transfer.rebuild_serial(host, dev, replay, forward)
    torch.cuda.synchronize()
    want = [(m_.clone(), f.clone(), o.clone()) for m_, f, o in zip(mids, fins, outs)]
    assert torch.equal(dev.cpu(), host)

    # the serial order itself against the oracle (layer 0, all heads)
    _, w_mid = oracle_run(tails[0])
    w_o, w_fin = oracle_run(sufs[0], state_in=w_mid, outputs=True)
    e = (state_err(to_f64(want[0][0]), w_mid), state_err(to_f64(want[0][1]), w_fin),
         output_err(to_f64(want[0][2]), w_o, sufs[0].cu_seqlens))
    print(f"[overlap] serial vs oracle: mid={e[0]:.3e} fin={e[1]:.3e} out={e[2]:.3e}", flush=True)
    assert e[0] <= STATE_TOL and e[1] <= STATE_TOL and e[2] <= OUTPUT_TOL

    copy_stream = torch.cuda.Stream()
    for run in range(3):
        clear()
        transfer.rebuild_overlapped(host, dev, replay, forward, copy_stream)
        torch.cuda.synchronize()
        assert torch.equal(dev.cpu(), host), f"run {run}: copied bytes differ"
        for l in range(LAYERS):
            assert torch.equal(mids[l], want[l][0]), f"run {run} layer {l}: rebuilt state differs"
            assert torch.equal(fins[l], want[l][1]), f"run {run} layer {l}: final state differs"
            assert torch.equal(outs[l], want[l][2]), f"run {run} layer {l}: outputs differ"
        # eager work on the compute stream between runs
        replay()
        torch.cuda.synchronize()
