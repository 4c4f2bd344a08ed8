"""The seeded input generator: reproducibility, distributions, bf16 rounding."""
from fractions import Fraction

import numpy as np
import torch

import synth
from synth import workloads


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(100000).astype(np.float32),
                        np.array([1.0, -1.0, 0.0, 1.00390625, 1.01171875,
                                  3.3895314e38, 1e-40], np.float32)])
    # ties: 1 + 2^-8 rounds to even (1.0), 1 + 3*2^-8 rounds up
    ours = synth.f32_to_bf16_bits(x)
    theirs = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, theirs)
    back = synth.bf16_bits_to_f32(ours)
    assert np.array_equal(back, torch.from_numpy(ours.view(np.int16)).view(torch.bfloat16).float().numpy())


def test_tail_is_a_slice_of_the_prefix():
    shape = synth.Shape(2, 4, 16, 8, "bf16")
    full = synth.tokens(9, 1, 2, 0, 300, shape)
    tail = synth.tokens(9, 1, 2, 171, 300, shape)
    for name in ("q", "k", "v", "g", "beta"):
        assert np.array_equal(getattr(full, name)[171:], getattr(tail, name))
    other = synth.tokens(9, 2, 2, 171, 300, shape)
    assert not np.array_equal(other.k, tail.k)


def test_distributions():
    shape = synth.Shape(2, 4, 64, 32, "f32")
    t = synth.tokens(1, 0, 0, 0, 640, shape, gate_scale=0.1)
    assert np.allclose(np.linalg.norm(t.k.astype(np.float64), axis=-1), 1.0, atol=1e-6)
    assert np.allclose(np.linalg.norm(t.q.astype(np.float64), axis=-1), 1.0, atol=1e-6)
    assert np.all(t.g < 0) and np.all(t.g > -2.0)
    assert np.all((t.beta > 0) & (t.beta < 1))
    # mean softplus(N(0,1)) ~ 0.806
    assert abs(float(-t.g.mean()) / 0.1 - 0.806) < 0.05
    assert abs(float(t.v.std()) - 1.0) < 0.05


def test_pack_offsets_and_exact_values():
    shape = synth.Shape(1, 2, 8, 8, "bf16")
    seqs = [synth.tokens(5, 0, i, 0, n, shape) for i, n in enumerate([3, 0, 65])]
    p = synth.pack(seqs)
    assert p.cu_seqlens.tolist() == [0, 3, 3, 68]
    assert p.cu_seqlens.dtype == np.int32
    ex = p.exact()
    assert ex["k"].dtype == np.float64
    assert np.array_equal(ex["k"].astype(np.float32), synth.bf16_bits_to_f32(p.k))


def test_workload3_draw_is_fixed():
    d = workloads.workload3_draw()
    assert len(d) == 16
    assert all(m in (8192, 16384, 32768) for m, _, _ in d)
    assert all(Fraction(1, 20) <= r <= Fraction(1, 10) for _, r, _ in d)
    assert all(128 <= s <= 2048 for _, _, s in d)
    assert d == workloads.workload3_draw()


def test_layer_hiddens_tail_is_a_slice_and_weights_are_fixed():
    from synth.layer import LayerDims, exact_weights, hiddens, layer_weights, pack_hiddens
    full = hiddens(5, 0, 3, 0, 200, 64)
    tail = hiddens(5, 0, 3, 130, 200, 64)
    assert full.dtype == np.uint16 and np.array_equal(full[130:], tail)
    assert not np.array_equal(hiddens(5, 1, 3, 130, 200, 64), tail)   # another layer
    dims = LayerDims(hidden=64, hk=2, hv=4, dk=16, dv=8)
    w1, w2 = layer_weights(5, 0, dims), layer_weights(5, 0, dims)
    for name in w1:
        assert np.array_equal(w1[name], w2[name])
    assert w1["w_in"].shape == (dims.in_rows, 64) and w1["w_in"].dtype == np.uint16
    assert w1["w_out"].shape == (64, dims.cv) and w1["conv_w"].shape == (2 * dims.cq + dims.cv, 4)
    ex = exact_weights(w1)
    # the gate parameters land where the recipe puts them: A = exp(A_log) in [1, 16],
    # softplus(dt_bias) = dt in [1e-3, 1e-1]
    assert np.all((np.exp(ex["a_log"]) >= 1 - 1e-6) & (np.exp(ex["a_log"]) <= 16 + 1e-5))
    dt = np.logaddexp(0.0, ex["dt_bias"])
    assert np.all((dt > 0.99e-3) & (dt < 1.01e-1))
    x, cu = pack_hiddens([hiddens(5, 0, i, 0, n, 64) for i, n in enumerate([3, 0, 70])], 64)
    assert list(cu) == [0, 3, 3, 73] and x.shape == (73, 64)


def test_threaded_draw_equals_one_by_one():
    shape = synth.Shape(2, 4, 16, 8, "bf16")
    hits = [workloads.Hit(9, l, 0, 300, 70, 40) for l in range(5)]
    got = workloads.draw_hits(hits, shape, threads=4)
    for h, (t, s) in zip(hits, got):
        want_t, want_s = h.tail(shape), h.suffix(shape)
        for name in ("q", "k", "v", "g", "beta"):
            assert np.array_equal(getattr(t, name), getattr(want_t, name))
            assert np.array_equal(getattr(s, name), getattr(want_s, name))
