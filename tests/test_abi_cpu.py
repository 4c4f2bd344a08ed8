"""The C ABI on the host: symbols, validation paths, replay-length rule (no GPU).

Calls here only take paths that the library rejects on the host before it
touches a device: every case carries at least one invalid argument.  Device
pointers are placeholders that are never dereferenced; on a machine with a GPU
these cases are skipped so no placeholder can ever reach a kernel.
"""
import ctypes
import glob
import os
import re

import pytest
import torch

import oracle
import paper_2608_30310_amd as gdn
from paper_2608_30310_amd import binding

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = sorted(glob.glob(os.path.join(ROOT, "include", "*.h")))

FAKE = ctypes.c_void_p(0x1000)   # never dereferenced: validation fails first


def declared_functions():
    text = "".join(open(h).read() for h in HEADERS)
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(gdn_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for want in ("gdn_tail_replay", "gdn_chunk_forward", "gdn_workspace_size",
                 "gdn_replay_forward", "gdn_replay_forward_workspace_size",
                 "gdn_replay_len", "gdn_status_string", "gdn_last_error", "gdn_decode_step",
                 "gdn_la_block_replay", "gdn_la_block_workspace_size"):
        assert want in names


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(binding.LIB_PATH)
    for name in declared_functions():
        assert hasattr(lib, name), f"{name} declared in the header but not exported"


def _shape(**kw):
    base = dict(num_seqs=1, num_k_heads=16, num_v_heads=32, d_k=128, d_v=128,
                qkv_dtype=binding.GDN_BF16, scale=1.0)
    base.update(kw)
    return binding.GDNShape(**base)


def _cu(vals):
    arr = (ctypes.c_int32 * len(vals))(*vals)
    return arr


def _ws_size(shape, cu, fwd=0):
    lib = gdn.load_library()
    out = ctypes.c_size_t(0)
    st = lib.gdn_workspace_size(ctypes.byref(shape) if shape is not None else None,
                                ctypes.cast(cu, ctypes.c_void_p) if cu is not None else None,
                                fwd, ctypes.byref(out))
    return st, out.value


@pytest.mark.parametrize("kw,cu,status", [
    (dict(num_k_heads=3), [0, 10], 2),              # Hv % Hk != 0
    (dict(num_k_heads=0), [0, 10], 2),
    (dict(num_seqs=-1), [0], 2),
    (dict(d_k=96), [0, 10], 4),                     # unsupported head dim
    (dict(d_v=256), [0, 10], 4),
    (dict(qkv_dtype=7), [0, 10], 4),
    (dict(scale=float("nan")), [0, 10], 2),
    (dict(), [1, 10], 3),                           # does not start at 0
    (dict(num_seqs=2), [0, 10, 5], 3),              # decreasing
])
def test_workspace_size_rejects(kw, cu, status):
    st, _ = _ws_size(_shape(**kw), _cu(cu))
    assert st == status
    assert gdn.load_library().gdn_last_error().decode()


def test_workspace_size_null_args():
    assert _ws_size(None, _cu([0, 1]))[0] == 1
    assert _ws_size(_shape(), None)[0] == 1


def test_workspace_size_values():
    # 819 tokens -> 13 chunk slots.  Per (slot, value head): T as 6 fragments,
    # hi only for bf16 inputs (6 KiB; hi and lo for fp32, 12 KiB) + 5 rows of
    # 64 fp32 scalars; outputs add P, split (12 KiB).  Per (slot, key head),
    # fp32 inputs only: the K record, K [and Q] as 4 x d_k / 32 1 KiB
    # fragments each, hi and lo parts (the scan fetches bf16 key and query
    # rows themselves).
    t_rec, s_rec, frag = 6 * 1024, 5 * 64 * 4, 1024
    p_rec = 6 * 2 * 1024

    def krec(dk=128, outputs=False, split=False):
        return 4 * (dk // 32) * (2 if outputs else 1) * 2 * frag if split else 0

    records = 13 * 32 * (t_rec + s_rec) + 13 * 16 * krec()
    st, n = _ws_size(_shape(), _cu([0, 819]))
    assert st == 0 and n == records
    st, nf = _ws_size(_shape(), _cu([0, 819]), 1)
    assert st == 0 and nf == 13 * 32 * (t_rec + p_rec + s_rec) + 13 * 16 * krec(outputs=True)
    st, n32 = _ws_size(_shape(qkv_dtype=binding.GDN_F32), _cu([0, 819]))
    assert st == 0 and n32 == 13 * 32 * (2 * t_rec + s_rec) + 13 * 16 * krec(split=True)
    st, n64 = _ws_size(_shape(d_k=64), _cu([0, 819]))
    assert st == 0 and n64 == 13 * 32 * (t_rec + s_rec) + 13 * 16 * krec(dk=64)
    # two sequences: slots cu[n]/64 + n + j, the last ends at 100/64 + 1 + 1 = 3
    st, n2 = _ws_size(_shape(num_seqs=2), _cu([0, 100, 130]))
    assert st == 0 and n2 == 3 * 32 * (t_rec + s_rec) + 3 * 16 * krec()
    # the longest-first order travels in the kernels' arguments: no region
    st, n2u = _ws_size(_shape(num_seqs=2), _cu([0, 30, 130]))
    assert st == 0 and n2u == 3 * 32 * (t_rec + s_rec) + 3 * 16 * krec()
    # Tail replay of bf16 inputs that may run in two halves (at least 20
    # chunks, N x Hv x (d_v / 32 + (d_v + d_k) / 64) <= 256 workgroups) adds
    # the second half's fp32 state [N, Hv, d_k, d_v] and transition [N, Hv,
    # d_k, d_k]: 1300 tokens -> 21 slots
    st, nl = _ws_size(_shape(), _cu([0, 1300]))
    assert st == 0 and nl == 21 * 32 * (t_rec + s_rec) + 21 * 16 * krec() + 32 * 128 * 128 * 4 * 2
    st, nl64 = _ws_size(_shape(d_k=64), _cu([0, 1300]))
    assert st == 0 and nl64 == (21 * 32 * (t_rec + s_rec) + 21 * 16 * krec(dk=64)
                                + 32 * 64 * 128 * 4 + 32 * 64 * 64 * 4)
    # with outputs, fp32 inputs, or two sequences at 32 heads (512 split
    # workgroups, more than the chip): no split regions
    st, nlf = _ws_size(_shape(), _cu([0, 1300]), 1)
    assert st == 0 and nlf == 21 * 32 * (t_rec + p_rec + s_rec) + 21 * 16 * krec(outputs=True)
    st, nl32 = _ws_size(_shape(qkv_dtype=binding.GDN_F32), _cu([0, 1300]))
    assert st == 0 and nl32 == 21 * 32 * (2 * t_rec + s_rec) + 21 * 16 * krec(split=True)
    # slots 0..20, then 1300/64 + 1 = 21 .. 41
    st, n2l = _ws_size(_shape(num_seqs=2), _cu([0, 1300, 2600]))
    assert st == 0 and n2l == 42 * 32 * (t_rec + s_rec) + 42 * 16 * krec()
    st, z = _ws_size(_shape(num_seqs=0), _cu([0]))
    assert st == 0 and z < 1024
    assert gdn.workspace_size(1, 16, 32, 128, 128, [0, 819]) == n


needs_no_gpu = pytest.mark.skipif(torch.cuda.is_available(),
                                  reason="placeholder pointers are only used without a GPU")


@needs_no_gpu
@pytest.mark.parametrize("case", ["null_k", "null_state", "small_ws", "null_ws", "misaligned_ws",
                                  "bad_seqlens", "null_cu_dev", "bad_heads"])
def test_tail_replay_rejects_before_launch(case):
    lib = gdn.load_library()
    shape = _shape(num_k_heads=3) if case == "bad_heads" else _shape()
    cu_host = _cu([0, 5, 3] if case == "bad_seqlens" else [0, 100])
    if case == "bad_seqlens":
        shape = _shape(num_seqs=2)
    _, need = _ws_size(_shape(), _cu([0, 100]))
    ws = None if case == "null_ws" else ctypes.c_void_p(0x10000 + (8 if case == "misaligned_ws" else 0))
    ws_bytes = need - 1 if case == "small_ws" else need
    st = lib.gdn_tail_replay(ctypes.byref(shape), ctypes.cast(cu_host, ctypes.c_void_p),
                             None if case == "null_cu_dev" else FAKE,
                             None if case == "null_k" else FAKE, FAKE, FAKE, FAKE,
                             None if case == "null_state" else FAKE, ws, ws_bytes, None)
    want = {"null_k": 1, "null_state": 1, "small_ws": 5, "null_ws": 5, "misaligned_ws": 5,
            "bad_seqlens": 3, "null_cu_dev": 1, "bad_heads": 2}[case]
    assert st == want, lib.gdn_last_error().decode()


@needs_no_gpu
@pytest.mark.parametrize("case", ["null_q", "null_o", "overlap", "small_ws", "misaligned_o"])
def test_chunk_forward_rejects_before_launch(case):
    lib = gdn.load_library()
    shape = _shape(num_seqs=2)
    cu_host = _cu([0, 50, 100])
    _, need = _ws_size(shape, cu_host, 1)
    state_bytes = 2 * 32 * 128 * 128 * 4
    s_in = ctypes.c_void_p(0x100000)
    s_out = ctypes.c_void_p(0x100000 + (state_bytes // 2 if case == "overlap" else 2 * state_bytes))
    st = lib.gdn_chunk_forward(ctypes.byref(shape), ctypes.cast(cu_host, ctypes.c_void_p), FAKE,
                               None if case == "null_q" else FAKE, FAKE, FAKE, FAKE, FAKE,
                               s_in, None if case == "null_o" else
                               (ctypes.c_void_p(0x1008) if case == "misaligned_o" else FAKE), s_out,
                               ctypes.c_void_p(0x20000),
                               need - 256 if case == "small_ws" else need, None)
    want = {"null_q": 1, "null_o": 1, "overlap": 2, "small_ws": 5, "misaligned_o": 4}[case]
    assert st == want, lib.gdn_last_error().decode()


@needs_no_gpu
@pytest.mark.parametrize("case", ["null_q", "null_o", "null_state_out", "overlap", "misaligned_state",
                                  "misaligned_v", "bad_dk", "bad_dtype", "bad_heads"])
def test_decode_step_rejects_before_launch(case):
    lib = gdn.load_library()
    kw = {"bad_dk": dict(d_k=96), "bad_dtype": dict(qkv_dtype=7), "bad_heads": dict(num_k_heads=3)}
    shape = _shape(num_seqs=2, **kw.get(case, {}))
    state_bytes = 2 * 32 * 128 * 128 * 4
    s_in = ctypes.c_void_p(0x100000 + (4 if case == "misaligned_state" else 0))
    s_out = ctypes.c_void_p(0x100000 + (state_bytes // 2 if case == "overlap" else 2 * state_bytes))
    st = lib.gdn_decode_step(ctypes.byref(shape), None if case == "null_q" else FAKE, FAKE,
                             ctypes.c_void_p(0x1008) if case == "misaligned_v" else FAKE, FAKE, FAKE,
                             s_in, None if case == "null_o" else FAKE,
                             None if case == "null_state_out" else s_out, None)
    want = {"null_q": 1, "null_o": 1, "null_state_out": 1, "overlap": 2, "misaligned_state": 4,
            "misaligned_v": 4, "bad_dk": 4, "bad_dtype": 4, "bad_heads": 2}[case]
    assert st == want, lib.gdn_last_error().decode()


def test_decode_step_with_no_sequences_does_nothing():
    lib = gdn.load_library()
    assert lib.gdn_decode_step(ctypes.byref(_shape(num_seqs=0)), None, None, None, None, None,
                               None, None, None, None) == 0


def test_status_strings():
    lib = gdn.load_library()
    for code in range(7):
        assert lib.gdn_status_string(code).decode().startswith("GDN_")


def test_replay_len_matches_the_oracle():
    lib = gdn.load_library()
    for m in (0, 1, 63, 2048, 8192, 16384, 32768, 31366, 31847):
        for ratio in ("0.05", "0.1", "1/3", "0.0723", "1"):
            assert gdn.replay_len(m, ratio) == oracle.replay_len(m, ratio)
    assert gdn.replay_len(8192, "0.1") == 820     # the paper's ceiling
    assert lib.gdn_replay_len(-1, 1, 10) == -1
    assert lib.gdn_replay_len(10, 1, 0) == -1
    assert lib.gdn_replay_len(2 ** 62, 4, 1) == -1
    with pytest.raises(TypeError):
        gdn.replay_len(10, 0.1)


def test_binding_raises_gdn_error():
    with pytest.raises(gdn.GDNError):
        binding._check(2)


def test_replay_forward_workspace_is_both_plans():
    # the fused call holds the tail plan (256-byte aligned) then the suffix plan
    lib = gdn.load_library()
    shape = _shape(num_seqs=2)
    ct, cs = [0, 819, 1230], [0, 512, 600]
    _, nt = _ws_size(shape, _cu(ct), 0)
    _, ns = _ws_size(shape, _cu(cs), 1)
    out = ctypes.c_size_t(0)
    st = lib.gdn_replay_forward_workspace_size(ctypes.byref(shape), ctypes.cast(_cu(ct), ctypes.c_void_p),
                                               ctypes.cast(_cu(cs), ctypes.c_void_p), ctypes.byref(out))
    assert st == 0 and out.value == (nt + 255) // 256 * 256 + ns
    assert gdn.replay_forward_workspace_size(2, 16, 32, 128, 128, ct, cs) == out.value
    assert gdn.replay_forward_stage_names() == ["tail intra", "tail scan (+ suffix intra)",
                                                "combine (+ suffix intra)", "suffix scan"]
    assert gdn.stage_names(False) == ["intra", "scan", "combine"]
    assert gdn.stage_names(True) == ["intra", "scan"]
    assert lib.gdn_stage_name(0, 3) == b"" and lib.gdn_stage_name(1, 2) == b""
    # sequence counts must agree
    st = lib.gdn_replay_forward_workspace_size(ctypes.byref(_shape(num_seqs=2)),
                                               ctypes.cast(_cu(ct), ctypes.c_void_p),
                                               ctypes.cast(_cu([0, 5, 3]), ctypes.c_void_p),
                                               ctypes.byref(out))
    assert st == 3


@needs_no_gpu
@pytest.mark.parametrize("case", ["null_mid", "null_o", "misaligned_k_tail", "small_ws", "overlap"])
def test_replay_forward_rejects_before_launch(case):
    lib = gdn.load_library()
    shape = _shape(num_seqs=1)
    ct, cs = _cu([0, 100]), _cu([0, 50])
    out = ctypes.c_size_t(0)
    assert lib.gdn_replay_forward_workspace_size(ctypes.byref(shape), ctypes.cast(ct, ctypes.c_void_p),
                                                 ctypes.cast(cs, ctypes.c_void_p), ctypes.byref(out)) == 0
    n_state = 32 * 128 * 128 * 4
    mid = ctypes.c_void_p(0x100000)
    fin = ctypes.c_void_p(0x100000 + (n_state // 2 if case == "overlap" else 2 * n_state))
    kt = ctypes.c_void_p(0x1008) if case == "misaligned_k_tail" else FAKE
    st = lib.gdn_replay_forward(ctypes.byref(shape), ctypes.cast(ct, ctypes.c_void_p), FAKE, kt, FAKE,
                                FAKE, FAKE, ctypes.cast(cs, ctypes.c_void_p), FAKE, FAKE, FAKE, FAKE,
                                FAKE, FAKE, None if case == "null_mid" else mid,
                                None if case == "null_o" else FAKE, fin, ctypes.c_void_p(0x20000),
                                out.value - (256 if case == "small_ws" else 0), None)
    want = {"null_mid": 1, "null_o": 1, "misaligned_k_tail": 4, "small_ws": 5, "overlap": 2}[case]
    assert st == want, lib.gdn_last_error().decode()


def test_noalloc_rejects_input_beyond_its_scratch_before_any_device_call():
    # the plan comes first: an input whose workspace exceeds the library's
    # scratch array returns GDN_ERR_WORKSPACE without touching the device
    lib = gdn.load_library()
    assert lib.gdn_noalloc_scratch_bytes() == 64 << 20 == gdn.noalloc_scratch_bytes()
    shape = _shape(num_seqs=1)
    big = _cu([0, 60000])          # ~0.5 GiB of records at 32 heads
    _, need = _ws_size(shape, big)
    assert need > 64 << 20
    st = lib.gdn_tail_replay_noalloc(ctypes.byref(shape), ctypes.cast(big, ctypes.c_void_p), FAKE, FAKE, FAKE,
                                     FAKE, FAKE, FAKE, None)
    assert st == 5 and b"scratch" in lib.gdn_last_error()
    # and the ordinary validation still applies
    st = lib.gdn_tail_replay_noalloc(ctypes.byref(_shape(num_seqs=2)), ctypes.cast(_cu([0, 10, 5]), ctypes.c_void_p),
                                     FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None)
    assert st == 3
