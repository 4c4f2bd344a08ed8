"""The layer-block C ABI on the host (no GPU): workspace plan, validation.

As in test_abi_cpu.py, every call that takes device pointers carries at least
one invalid argument, so the library rejects it before touching a device;
those cases are skipped where a GPU is visible.
"""
import ctypes

import pytest
import torch

import paper_2608_30310_amd as gdn
from paper_2608_30310_amd import binding

FAKE = ctypes.c_void_p(0x1000)
GEMM_WS = 32 << 20


def _shape(**kw):
    base = dict(num_seqs=1, hidden=2048, num_k_heads=16, num_v_heads=32, d_k=128, d_v=128,
                conv_taps=4, act_dtype=binding.GDN_F32, scale=0.1, l2_eps=1e-6, norm_eps=1e-6)
    base.update(kw)
    return binding.LAShape(**base)


def _cu(vals):
    return (ctypes.c_int32 * len(vals))(*vals)


def _ws(shape, cu, outputs):
    out = ctypes.c_size_t(0)
    st = gdn.load_library().gdn_la_block_workspace_size(
        ctypes.byref(shape) if shape is not None else None,
        ctypes.cast(cu, ctypes.c_void_p) if cu is not None else None, int(outputs), ctypes.byref(out))
    return st, out.value


def _up(n):
    return (n + 255) // 256 * 256


@pytest.mark.parametrize("act,es", [(binding.GDN_F32, 4), (binding.GDN_BF16, 2)])
def test_workspace_is_the_sum_of_its_regions(act, es):
    T, hk, hv, dk, dv = 819, 16, 32, 128, 128
    cq, cv = hk * dk, hv * dv
    scan_dtype = torch.float32 if act == binding.GDN_F32 else torch.bfloat16
    for outputs in (True, False):
        rows = 2 * cq + 2 * cv + 2 * hv if outputs else cq + cv + 2 * hv
        scan = gdn.workspace_size(1, hk, hv, dk, dv, [0, T], dtype=scan_dtype, with_outputs=outputs)
        regions = [T * rows * es] + ([T * cq * es] if outputs else []) + [T * cq * es, T * cv * es,
                                                                          T * hv * 4, T * hv * 4]
        regions += ([T * cv * es] if outputs else []) + [scan, GEMM_WS]
        want = sum(_up(r) for r in regions[:-1]) + _up(GEMM_WS)
        st, got = _ws(_shape(act_dtype=act), _cu([0, T]), outputs)
        assert st == 0 and got == want
        assert gdn.la_block_workspace_size(2048, hk, hv, dk, dv, [0, T], outputs,
                                           "f32" if act == binding.GDN_F32 else "bf16") == want


@pytest.mark.parametrize("kw,status", [
    (dict(hidden=0), 2), (dict(hidden=100), 4), (dict(num_v_heads=48, num_k_heads=24), 0),
    (dict(num_v_heads=6, num_k_heads=3), 4), (dict(num_k_heads=5), 2), (dict(conv_taps=3), 4),
    (dict(act_dtype=5), 4), (dict(d_k=96), 4), (dict(l2_eps=-1.0), 2), (dict(norm_eps=float("inf")), 2),
    (dict(scale=float("nan")), 2), (dict(num_seqs=-1), 2),
])
def test_workspace_size_validates_the_shape(kw, status):
    cu = [0] if kw.get("num_seqs") == -1 else [0, 64]
    st, _ = _ws(_shape(**kw), _cu(cu), True)
    assert st == status, gdn.load_library().gdn_last_error().decode()


def test_workspace_size_null_args():
    assert _ws(None, _cu([0, 1]), True)[0] == 1
    assert _ws(_shape(), None, True)[0] == 1


def test_stage_names():
    assert gdn.la_block_stage_names(True) == ["in-projection", "prep", "recurrence", "gated norm",
                                              "out-projection"]
    assert gdn.la_block_stage_names(False) == ["in-projection", "prep", "recurrence"]
    assert gdn.load_library().gdn_la_block_stage_name(1, 5) == b""


needs_no_gpu = pytest.mark.skipif(torch.cuda.is_available(),
                                  reason="placeholder pointers are only used without a GPU")

CASES = {"null_weights": 1, "null_w_in": 1, "null_w_out": 1, "null_state": 1, "null_x": 1, "null_cu": 1,
         "misaligned_x": 4, "misaligned_conv_w": 4, "misaligned_norm_w": 4, "misaligned_out": 4, "small_ws": 5, "null_ws": 5,
         "misaligned_ws": 5, "bad_hidden": 4, "bad_events": 2}


@needs_no_gpu
@pytest.mark.parametrize("case", sorted(CASES))
def test_block_rejects_before_launch(case):
    lib = gdn.load_library()
    shape = _shape(hidden=100) if case == "bad_hidden" else _shape()
    cu = _cu([0, 100])
    _, need = _ws(_shape(), cu, True)
    w = binding.LAWeights(FAKE.value, FAKE.value, FAKE.value, FAKE.value, FAKE.value, FAKE.value)
    if case == "null_w_in":
        w.w_in = None
    if case == "null_w_out":
        w.w_out = None
    if case == "misaligned_conv_w":
        w.conv_w = 0x1004
    if case == "misaligned_norm_w":
        w.norm_w = 0x1008
    x = None if case == "null_x" else (ctypes.c_void_p(0x1008) if case == "misaligned_x" else FAKE)
    out = ctypes.c_void_p(0x1002) if case == "misaligned_out" else FAKE
    ws = None if case == "null_ws" else ctypes.c_void_p(0x20000 + (16 if case == "misaligned_ws" else 0))
    args = [ctypes.byref(shape), None if case == "null_weights" else ctypes.byref(w),
            ctypes.cast(cu, ctypes.c_void_p), None if case == "null_cu" else FAKE, x,
            None if case == "null_state" else FAKE, out, ws, need - 256 if case == "small_ws" else need, None]
    if case == "bad_events":
        ev = (ctypes.c_void_p * 3)(FAKE, FAKE, FAKE)
        st = lib.gdn_la_block_replay_profiled(*args, ctypes.cast(ev, ctypes.c_void_p), 3)
    else:
        st = lib.gdn_la_block_replay(*args)
    assert st == CASES[case], lib.gdn_last_error().decode()


def test_block_with_no_sequences_does_nothing():
    # N = 0: every stage has nothing to do, so nothing touches a device
    lib = gdn.load_library()
    shape = _shape(num_seqs=0)
    st, need = _ws(shape, _cu([0]), True)
    assert st == 0 and need >= GEMM_WS
    w = binding.LAWeights(FAKE.value, FAKE.value, FAKE.value, FAKE.value, FAKE.value, FAKE.value)
    st = lib.gdn_la_block_replay(ctypes.byref(shape), ctypes.byref(w), ctypes.cast(_cu([0]), ctypes.c_void_p),
                                 None, None, None, FAKE, ctypes.c_void_p(0x20000), need, None)
    assert st == 0, lib.gdn_last_error().decode()
