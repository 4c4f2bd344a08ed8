"""ctypes binding of libgdn_tailreplay.so: argument marshalling only.

Every step of the path runs in the library's HIP kernels; this module checks
tensor dtypes/devices/shapes, keeps a cached workspace per (device, stream),
passes raw pointers and torch's current stream, and raises ``GDNError`` on a
non-zero status.  It never computes any part of the method itself, and it has
no fallback: when the library is missing every call raises.
"""
from __future__ import annotations

import ctypes
import os
from fractions import Fraction
from typing import Optional, Sequence, Union

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libgdn_tailreplay.so")

GDN_F32 = 0
GDN_BF16 = 1


class GDNError(RuntimeError):
    """A gdn_* call returned a non-zero gdn_status."""

    def __init__(self, status: int, message: str):
        super().__init__(message)
        self.status = status


class GDNShape(ctypes.Structure):
    _fields_ = [("num_seqs", ctypes.c_int32), ("num_k_heads", ctypes.c_int32),
                ("num_v_heads", ctypes.c_int32), ("d_k", ctypes.c_int32),
                ("d_v", ctypes.c_int32), ("qkv_dtype", ctypes.c_int32),
                ("scale", ctypes.c_float)]


class LAShape(ctypes.Structure):
    _fields_ = [("num_seqs", ctypes.c_int32), ("hidden", ctypes.c_int32),
                ("num_k_heads", ctypes.c_int32), ("num_v_heads", ctypes.c_int32),
                ("d_k", ctypes.c_int32), ("d_v", ctypes.c_int32), ("conv_taps", ctypes.c_int32),
                ("act_dtype", ctypes.c_int32), ("scale", ctypes.c_float),
                ("l2_eps", ctypes.c_float), ("norm_eps", ctypes.c_float)]


class LAWeights(ctypes.Structure):
    _fields_ = [("w_in", ctypes.c_void_p), ("conv_w", ctypes.c_void_p), ("a_log", ctypes.c_void_p),
                ("dt_bias", ctypes.c_void_p), ("norm_w", ctypes.c_void_p), ("w_out", ctypes.c_void_p)]


_lib = None


def load_library():
    """Loads the HIP library (raises ``ImportError`` if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is missing: build it with `python -m paper_2608_30310_amd.build` "
            "(or __graft_entry__.build()); there is no fallback path")
    lib = ctypes.CDLL(LIB_PATH)
    P = ctypes.c_void_p
    SP = ctypes.POINTER(GDNShape)
    lib.gdn_workspace_size.argtypes = [SP, P, ctypes.c_int32, ctypes.POINTER(ctypes.c_size_t)]
    lib.gdn_workspace_size.restype = ctypes.c_int
    lib.gdn_tail_replay.argtypes = [SP, P, P, P, P, P, P, P, P, ctypes.c_size_t, P]
    lib.gdn_tail_replay.restype = ctypes.c_int
    lib.gdn_chunk_forward.argtypes = [SP, P, P, P, P, P, P, P, P, P, P, P, ctypes.c_size_t, P]
    lib.gdn_chunk_forward.restype = ctypes.c_int
    lib.gdn_tail_replay_profiled.argtypes = lib.gdn_tail_replay.argtypes + [P, ctypes.c_int32]
    lib.gdn_tail_replay_profiled.restype = ctypes.c_int
    lib.gdn_chunk_forward_profiled.argtypes = lib.gdn_chunk_forward.argtypes + [P, ctypes.c_int32]
    lib.gdn_chunk_forward_profiled.restype = ctypes.c_int
    lib.gdn_replay_forward_workspace_size.argtypes = [SP, P, P, ctypes.POINTER(ctypes.c_size_t)]
    lib.gdn_replay_forward_workspace_size.restype = ctypes.c_int
    lib.gdn_replay_forward.argtypes = [SP, P, P, P, P, P, P, P, P, P, P, P, P, P, P, P, P, P, ctypes.c_size_t, P]
    lib.gdn_replay_forward.restype = ctypes.c_int
    lib.gdn_replay_forward_profiled.argtypes = lib.gdn_replay_forward.argtypes + [P, ctypes.c_int32]
    lib.gdn_replay_forward_profiled.restype = ctypes.c_int
    lib.gdn_replay_forward_num_stages.argtypes = []
    lib.gdn_replay_forward_num_stages.restype = ctypes.c_int32
    lib.gdn_replay_forward_stage_name.argtypes = [ctypes.c_int32]
    lib.gdn_replay_forward_stage_name.restype = ctypes.c_char_p
    lib.gdn_num_stages.argtypes = [ctypes.c_int32]
    lib.gdn_num_stages.restype = ctypes.c_int32
    lib.gdn_stage_name.argtypes = [ctypes.c_int32, ctypes.c_int32]
    lib.gdn_stage_name.restype = ctypes.c_char_p
    lib.gdn_tail_replay_noalloc.argtypes = [SP, P, P, P, P, P, P, P, P]
    lib.gdn_tail_replay_noalloc.restype = ctypes.c_int
    lib.gdn_noalloc_scratch_bytes.argtypes = []
    lib.gdn_noalloc_scratch_bytes.restype = ctypes.c_size_t
    lib.gdn_decode_step.argtypes = [SP, P, P, P, P, P, P, P, P, P]
    lib.gdn_decode_step.restype = ctypes.c_int
    LP = ctypes.POINTER(LAShape)
    WP = ctypes.POINTER(LAWeights)
    lib.gdn_la_block_workspace_size.argtypes = [LP, P, ctypes.c_int32, ctypes.POINTER(ctypes.c_size_t)]
    lib.gdn_la_block_workspace_size.restype = ctypes.c_int
    lib.gdn_la_block_replay.argtypes = [LP, WP, P, P, P, P, P, P, ctypes.c_size_t, P]
    lib.gdn_la_block_replay.restype = ctypes.c_int
    lib.gdn_la_block_replay_profiled.argtypes = lib.gdn_la_block_replay.argtypes + [P, ctypes.c_int32]
    lib.gdn_la_block_replay_profiled.restype = ctypes.c_int
    lib.gdn_la_block_num_stages.argtypes = [ctypes.c_int32]
    lib.gdn_la_block_num_stages.restype = ctypes.c_int32
    lib.gdn_la_block_stage_name.argtypes = [ctypes.c_int32, ctypes.c_int32]
    lib.gdn_la_block_stage_name.restype = ctypes.c_char_p
    lib.gdn_replay_len.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_int64]
    lib.gdn_replay_len.restype = ctypes.c_int64
    lib.gdn_status_string.argtypes = [ctypes.c_int]
    lib.gdn_status_string.restype = ctypes.c_char_p
    lib.gdn_last_error.argtypes = []
    lib.gdn_last_error.restype = ctypes.c_char_p
    _lib = lib
    return lib


def _check(status: int):
    if status != 0:
        lib = load_library()
        msg = lib.gdn_status_string(status).decode()
        detail = lib.gdn_last_error().decode()
        raise GDNError(status, f"{msg}: {detail}" if detail else msg)


def replay_len(m: int, ratio: Union[Fraction, int, str]) -> int:
    """Replay budget k = ceil(r * m) (paper Section 3), via ``gdn_replay_len``."""
    if isinstance(ratio, float):
        raise TypeError("pass the ratio as a Fraction or decimal string, not a float")
    r = Fraction(ratio)
    out = load_library().gdn_replay_len(int(m), r.numerator, r.denominator)
    if out < 0:
        raise ValueError("invalid replay length arguments")
    return int(out)


def stage_names(with_outputs: bool):
    """Names of the kernel stages a call enqueues, in order."""
    lib = load_library()
    n = lib.gdn_num_stages(int(with_outputs))
    return [lib.gdn_stage_name(int(with_outputs), i).decode() for i in range(n)]


def replay_forward_stage_names():
    """Names of the kernel stages ``replay_forward`` enqueues, in order."""
    lib = load_library()
    return [lib.gdn_replay_forward_stage_name(i).decode()
            for i in range(lib.gdn_replay_forward_num_stages())]


def _event_array(events, with_outputs, fused=False):
    """torch.cuda.Event list -> (void*[n], n) for the *_profiled entry points."""
    lib = load_library()
    n = (lib.gdn_replay_forward_num_stages() if fused else lib.gdn_num_stages(int(with_outputs))) + 1
    if len(events) != n:
        raise ValueError(f"need {n} events (one per stage boundary)")
    handles = []
    for ev in events:
        if ev.cuda_event == 0:          # torch creates the HIP event on first record
            ev.record()
        handles.append(ev.cuda_event)
    arr = (ctypes.c_void_p * n)(*handles)
    return arr, n


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _seqlens(cu_seqlens, cu_seqlens_host, device):
    if cu_seqlens_host is None:
        if isinstance(cu_seqlens, torch.Tensor):
            cu_seqlens_host = cu_seqlens.detach().to("cpu", torch.int32)
        else:
            cu_seqlens_host = torch.tensor(list(cu_seqlens), dtype=torch.int32)
    elif not isinstance(cu_seqlens_host, torch.Tensor):
        cu_seqlens_host = torch.tensor(list(cu_seqlens_host), dtype=torch.int32)
    cu_seqlens_host = cu_seqlens_host.to(torch.int32).contiguous()
    if cu_seqlens_host.device.type != "cpu":
        raise ValueError("cu_seqlens_host must live in host memory")
    if isinstance(cu_seqlens, torch.Tensor) and cu_seqlens.device == device:
        cu_dev = cu_seqlens
    else:
        cu_dev = cu_seqlens_host.to(device, non_blocking=False)
    if cu_dev.dtype != torch.int32 or not cu_dev.is_contiguous():
        raise ValueError("cu_seqlens must be a contiguous int32 tensor")
    if cu_dev.numel() != cu_seqlens_host.numel() or cu_dev.numel() < 1:
        raise ValueError("cu_seqlens and cu_seqlens_host must both hold N + 1 offsets")
    return cu_dev, cu_seqlens_host


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return GDN_BF16
    if t.dtype == torch.float32:
        return GDN_F32
    raise ValueError(f"q/k/v must be bfloat16 or float32, got {t.dtype}")


def _need(t, name, dtype, device, ndim):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device != device:
        raise ValueError(f"{name} must live on {device}")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if t.dim() != ndim:
        raise ValueError(f"{name} must have {ndim} dimensions")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


_WORKSPACES = {}


def _workspace(nbytes: int, device: torch.device, stream) -> torch.Tensor:
    key = (device.index, stream.cuda_stream)
    ws = _WORKSPACES.get(key)
    if ws is None or ws.numel() < nbytes:
        ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)
        _WORKSPACES[key] = ws
    if ws.data_ptr() % 256:
        raise RuntimeError("workspace allocation is not 256-byte aligned")
    return ws


def _shape(num_seqs, hk, hv, dk, dv, dtype_code, scale):
    return GDNShape(num_seqs, hk, hv, dk, dv, dtype_code, float(scale))


def workspace_size(num_seqs: int, num_k_heads: int, num_v_heads: int, d_k: int, d_v: int,
                   cu_seqlens_host: Sequence[int], dtype=torch.bfloat16,
                   with_outputs: bool = False) -> int:
    lib = load_library()
    cu = torch.tensor(list(cu_seqlens_host), dtype=torch.int32)
    shp = _shape(num_seqs, num_k_heads, num_v_heads, d_k, d_v,
                 GDN_BF16 if dtype == torch.bfloat16 else GDN_F32, 1.0)
    out = ctypes.c_size_t(0)
    _check(lib.gdn_workspace_size(ctypes.byref(shp), _ptr(cu), int(with_outputs),
                                  ctypes.byref(out)))
    return int(out.value)


def tail_replay(k: torch.Tensor, v: torch.Tensor, g: torch.Tensor, beta: torch.Tensor,
                cu_seqlens, cu_seqlens_host=None, state_out: Optional[torch.Tensor] = None,
                workspace: Optional[torch.Tensor] = None, events=None) -> torch.Tensor:
    """Independent Tail-Replay (paper Section 3, Eq. 2) on torch's current stream.

    k [T,Hk,d_k], v [T,Hv,d_v] (bf16 or fp32), g/beta [T,Hv] fp32, packed by
    ``cu_seqlens`` (N + 1 int32 offsets).  Returns the rebuilt states
    [N, Hv, d_k, d_v] fp32 (M = S^T), each started from zero at its tail's
    first token.  ``events``: optional torch.cuda.Event list, one per stage
    boundary, recorded by the library between its kernel stages.
    """
    lib = load_library()
    device = k.device
    dt = k.dtype
    _need(k, "k", dt, device, 3)
    _need(v, "v", dt, device, 3)
    T, hk, dk = k.shape
    hv, dv = v.shape[1], v.shape[2]
    if v.shape[0] != T:
        raise ValueError("k and v must hold the same tokens")
    _need(g, "g", torch.float32, device, 2)
    _need(beta, "beta", torch.float32, device, 2)
    if tuple(g.shape) != (T, hv) or tuple(beta.shape) != (T, hv):
        raise ValueError("g and beta must be [T, Hv]")
    cu_dev, cu_host = _seqlens(cu_seqlens, cu_seqlens_host, device)
    n = cu_host.numel() - 1
    if state_out is None:
        state_out = torch.empty((n, hv, dk, dv), dtype=torch.float32, device=device)
    _need(state_out, "state_out", torch.float32, device, 4)
    if tuple(state_out.shape) != (n, hv, dk, dv):
        raise ValueError("state_out must be [N, Hv, d_k, d_v]")
    shp = _shape(n, hk, hv, dk, dv, _dtype_code(k), 1.0)
    stream = torch.cuda.current_stream(device)
    need = ctypes.c_size_t(0)
    _check(lib.gdn_workspace_size(ctypes.byref(shp), _ptr(cu_host), 0, ctypes.byref(need)))
    ws = workspace if workspace is not None else _workspace(need.value, device, stream)
    args = [ctypes.byref(shp), _ptr(cu_host), _ptr(cu_dev), _ptr(k), _ptr(v), _ptr(g),
            _ptr(beta), _ptr(state_out), _ptr(ws), ws.numel() * ws.element_size(),
            ctypes.c_void_p(stream.cuda_stream)]
    if events is None:
        _check(lib.gdn_tail_replay(*args))
    else:
        arr, n = _event_array(events, False)
        _check(lib.gdn_tail_replay_profiled(*args, ctypes.cast(arr, ctypes.c_void_p), n))
    return state_out


def noalloc_scratch_bytes() -> int:
    """Size of the device array ``tail_replay_noalloc`` uses as its workspace."""
    return int(load_library().gdn_noalloc_scratch_bytes())


def tail_replay_noalloc(k: torch.Tensor, v: torch.Tensor, g: torch.Tensor, beta: torch.Tensor,
                        cu_seqlens, cu_seqlens_host, state_out: torch.Tensor) -> torch.Tensor:
    """``tail_replay`` through ``gdn_tail_replay_noalloc``: the library takes
    its workspace from a device array of its own and allocates nothing; the
    caller passes every tensor, including ``state_out`` [N, Hv, d_k, d_v] fp32
    and the device and host copies of ``cu_seqlens``.  Calls that may overlap
    on one GPU share that array and must be ordered on one stream."""
    lib = load_library()
    device = k.device
    dt = k.dtype
    _need(k, "k", dt, device, 3)
    _need(v, "v", dt, device, 3)
    T, hk, dk = k.shape
    hv, dv = v.shape[1], v.shape[2]
    if v.shape[0] != T:
        raise ValueError("k and v must hold the same tokens")
    _need(g, "g", torch.float32, device, 2)
    _need(beta, "beta", torch.float32, device, 2)
    if tuple(g.shape) != (T, hv) or tuple(beta.shape) != (T, hv):
        raise ValueError("g and beta must be [T, Hv]")
    if not isinstance(cu_seqlens, torch.Tensor) or cu_seqlens.device != device:
        raise ValueError("cu_seqlens must be a device tensor (nothing is copied here)")
    if not isinstance(cu_seqlens_host, torch.Tensor):
        raise ValueError("cu_seqlens_host must be a host tensor")
    cu_dev, cu_host = _seqlens(cu_seqlens, cu_seqlens_host, device)
    n = cu_host.numel() - 1
    _need(state_out, "state_out", torch.float32, device, 4)
    if tuple(state_out.shape) != (n, hv, dk, dv):
        raise ValueError("state_out must be [N, Hv, d_k, d_v]")
    shp = _shape(n, hk, hv, dk, dv, _dtype_code(k), 1.0)
    stream = torch.cuda.current_stream(device)
    _check(lib.gdn_tail_replay_noalloc(ctypes.byref(shp), _ptr(cu_host), _ptr(cu_dev), _ptr(k), _ptr(v),
                                       _ptr(g), _ptr(beta), _ptr(state_out),
                                       ctypes.c_void_p(stream.cuda_stream)))
    return state_out


def chunk_forward(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, g: torch.Tensor,
                  beta: torch.Tensor, cu_seqlens, cu_seqlens_host=None,
                  state_in: Optional[torch.Tensor] = None, scale: float = 1.0,
                  o: Optional[torch.Tensor] = None, state_out: Optional[torch.Tensor] = None,
                  write_state: bool = True, workspace: Optional[torch.Tensor] = None,
                  events=None):
    """Chunked GDN forward from ``state_in`` (None = zero) on torch's current stream.

    Returns ``(o [T,Hv,d_v] in q's dtype, state_out [N,Hv,d_k,d_v] fp32 or None)``.
    ``state_out`` may be ``state_in`` (in-place update).
    """
    lib = load_library()
    device = q.device
    dt = q.dtype
    _need(q, "q", dt, device, 3)
    _need(k, "k", dt, device, 3)
    _need(v, "v", dt, device, 3)
    T, hk, dk = q.shape
    if tuple(k.shape) != (T, hk, dk):
        raise ValueError("q and k must have the same shape")
    hv, dv = v.shape[1], v.shape[2]
    if v.shape[0] != T:
        raise ValueError("v must hold the same tokens as q and k")
    _need(g, "g", torch.float32, device, 2)
    _need(beta, "beta", torch.float32, device, 2)
    if tuple(g.shape) != (T, hv) or tuple(beta.shape) != (T, hv):
        raise ValueError("g and beta must be [T, Hv]")
    cu_dev, cu_host = _seqlens(cu_seqlens, cu_seqlens_host, device)
    n = cu_host.numel() - 1
    if state_in is not None:
        _need(state_in, "state_in", torch.float32, device, 4)
        if tuple(state_in.shape) != (n, hv, dk, dv):
            raise ValueError("state_in must be [N, Hv, d_k, d_v]")
    if o is None:
        o = torch.empty((T, hv, dv), dtype=dt, device=device)
    _need(o, "o", dt, device, 3)
    if tuple(o.shape) != (T, hv, dv):
        raise ValueError("o must be [T, Hv, d_v]")
    if write_state and state_out is None:
        state_out = torch.empty((n, hv, dk, dv), dtype=torch.float32, device=device)
    if state_out is not None:
        _need(state_out, "state_out", torch.float32, device, 4)
        if tuple(state_out.shape) != (n, hv, dk, dv):
            raise ValueError("state_out must be [N, Hv, d_k, d_v]")
    shp = _shape(n, hk, hv, dk, dv, _dtype_code(q), scale)
    stream = torch.cuda.current_stream(device)
    need = ctypes.c_size_t(0)
    _check(lib.gdn_workspace_size(ctypes.byref(shp), _ptr(cu_host), 1, ctypes.byref(need)))
    ws = workspace if workspace is not None else _workspace(need.value, device, stream)
    args = [ctypes.byref(shp), _ptr(cu_host), _ptr(cu_dev), _ptr(q), _ptr(k), _ptr(v), _ptr(g),
            _ptr(beta), _ptr(state_in), _ptr(o), _ptr(state_out), _ptr(ws),
            ws.numel() * ws.element_size(), ctypes.c_void_p(stream.cuda_stream)]
    if events is None:
        _check(lib.gdn_chunk_forward(*args))
    else:
        arr, n = _event_array(events, True)
        _check(lib.gdn_chunk_forward_profiled(*args, ctypes.cast(arr, ctypes.c_void_p), n))
    return o, state_out


def replay_forward_workspace_size(num_seqs: int, num_k_heads: int, num_v_heads: int, d_k: int,
                                  d_v: int, cu_tail_host: Sequence[int], cu_suf_host: Sequence[int],
                                  dtype=torch.bfloat16) -> int:
    lib = load_library()
    ct = torch.tensor(list(cu_tail_host), dtype=torch.int32)
    cs = torch.tensor(list(cu_suf_host), dtype=torch.int32)
    shp = _shape(num_seqs, num_k_heads, num_v_heads, d_k, d_v,
                 GDN_BF16 if dtype == torch.bfloat16 else GDN_F32, 1.0)
    out = ctypes.c_size_t(0)
    _check(lib.gdn_replay_forward_workspace_size(ctypes.byref(shp), _ptr(ct), _ptr(cs),
                                                 ctypes.byref(out)))
    return int(out.value)


def replay_forward(k_tail: torch.Tensor, v_tail: torch.Tensor, g_tail: torch.Tensor,
                   beta_tail: torch.Tensor, cu_tail, q: torch.Tensor, k: torch.Tensor,
                   v: torch.Tensor, g: torch.Tensor, beta: torch.Tensor, cu_suf,
                   cu_tail_host=None, cu_suf_host=None, scale: float = 1.0,
                   state_mid: Optional[torch.Tensor] = None, o: Optional[torch.Tensor] = None,
                   state_out: Optional[torch.Tensor] = None, write_state: bool = True,
                   workspace: Optional[torch.Tensor] = None, events=None):
    """Tail replay (paper Section 3, Eq. 2), then the forward over each
    sequence's new suffix from the rebuilt state, in one call on torch's
    current stream (same results as ``tail_replay`` then ``chunk_forward``).

    Returns ``(o [Ts,Hv,d_v], state_mid [N,Hv,d_k,d_v], state_out or None)``.
    """
    lib = load_library()
    device = q.device
    dt = q.dtype
    for name, t in (("k_tail", k_tail), ("v_tail", v_tail), ("q", q), ("k", k), ("v", v)):
        _need(t, name, dt, device, 3)
    Tt, hk, dk = k_tail.shape
    Ts = q.shape[0]
    hv, dv = v.shape[1], v.shape[2]
    if tuple(v_tail.shape) != (Tt, hv, dv) or tuple(k.shape) != (Ts, hk, dk) or \
            tuple(q.shape) != (Ts, hk, dk) or v.shape[0] != Ts:
        raise ValueError("inconsistent tail/suffix shapes")
    for name, t, T in (("g_tail", g_tail, Tt), ("beta_tail", beta_tail, Tt), ("g", g, Ts),
                       ("beta", beta, Ts)):
        _need(t, name, torch.float32, device, 2)
        if tuple(t.shape) != (T, hv):
            raise ValueError(f"{name} must be [T, Hv]")
    cu_t, cu_t_host = _seqlens(cu_tail, cu_tail_host, device)
    cu_s, cu_s_host = _seqlens(cu_suf, cu_suf_host, device)
    n = cu_t_host.numel() - 1
    if cu_s_host.numel() - 1 != n:
        raise ValueError("tail and suffix must pack the same number of sequences")
    if state_mid is None:
        state_mid = torch.empty((n, hv, dk, dv), dtype=torch.float32, device=device)
    if o is None:
        o = torch.empty((Ts, hv, dv), dtype=dt, device=device)
    if write_state and state_out is None:
        state_out = torch.empty((n, hv, dk, dv), dtype=torch.float32, device=device)
    for name, t in (("state_mid", state_mid), ("state_out", state_out)):
        if t is not None:
            _need(t, name, torch.float32, device, 4)
            if tuple(t.shape) != (n, hv, dk, dv):
                raise ValueError(f"{name} must be [N, Hv, d_k, d_v]")
    _need(o, "o", dt, device, 3)
    if tuple(o.shape) != (Ts, hv, dv):
        raise ValueError("o must be [Ts, Hv, d_v]")
    shp = _shape(n, hk, hv, dk, dv, _dtype_code(q), scale)
    stream = torch.cuda.current_stream(device)
    need = ctypes.c_size_t(0)
    _check(lib.gdn_replay_forward_workspace_size(ctypes.byref(shp), _ptr(cu_t_host), _ptr(cu_s_host),
                                                 ctypes.byref(need)))
    ws = workspace if workspace is not None else _workspace(need.value, device, stream)
    args = [ctypes.byref(shp), _ptr(cu_t_host), _ptr(cu_t), _ptr(k_tail), _ptr(v_tail),
            _ptr(g_tail), _ptr(beta_tail), _ptr(cu_s_host), _ptr(cu_s), _ptr(q), _ptr(k), _ptr(v),
            _ptr(g), _ptr(beta), _ptr(state_mid), _ptr(o), _ptr(state_out), _ptr(ws),
            ws.numel() * ws.element_size(), ctypes.c_void_p(stream.cuda_stream)]
    if events is None:
        _check(lib.gdn_replay_forward(*args))
    else:
        arr, ne = _event_array(events, True, fused=True)
        _check(lib.gdn_replay_forward_profiled(*args, ctypes.cast(arr, ctypes.c_void_p), ne))
    return o, state_mid, state_out


def decode_step(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, g: torch.Tensor,
                beta: torch.Tensor, state_in: Optional[torch.Tensor] = None, scale: float = 1.0,
                o: Optional[torch.Tensor] = None, state_out: Optional[torch.Tensor] = None):
    """One decode step (paper Section 2, Eq. 1 for a single token per sequence)
    on torch's current stream.

    q, k [N,Hk,d_k], v [N,Hv,d_v] (bf16 or fp32), g/beta [N,Hv] fp32,
    state_in [N,Hv,d_k,d_v] fp32 (None = zero state).  Returns
    ``(o [N,Hv,d_v], state_out)``; pass ``state_out=state_in`` to update in place.
    """
    lib = load_library()
    device = q.device
    dt = q.dtype
    _need(q, "q", dt, device, 3)
    _need(k, "k", dt, device, 3)
    _need(v, "v", dt, device, 3)
    n, hk, dk = q.shape
    if tuple(k.shape) != (n, hk, dk):
        raise ValueError("q and k must have the same shape")
    hv, dv = v.shape[1], v.shape[2]
    if v.shape[0] != n:
        raise ValueError("v must hold one token per sequence, like q and k")
    _need(g, "g", torch.float32, device, 2)
    _need(beta, "beta", torch.float32, device, 2)
    if tuple(g.shape) != (n, hv) or tuple(beta.shape) != (n, hv):
        raise ValueError("g and beta must be [N, Hv]")
    if state_in is not None:
        _need(state_in, "state_in", torch.float32, device, 4)
        if tuple(state_in.shape) != (n, hv, dk, dv):
            raise ValueError("state_in must be [N, Hv, d_k, d_v]")
    if state_out is None:
        state_out = torch.empty((n, hv, dk, dv), dtype=torch.float32, device=device)
    _need(state_out, "state_out", torch.float32, device, 4)
    if tuple(state_out.shape) != (n, hv, dk, dv):
        raise ValueError("state_out must be [N, Hv, d_k, d_v]")
    if o is None:
        o = torch.empty((n, hv, dv), dtype=dt, device=device)
    _need(o, "o", dt, device, 3)
    if tuple(o.shape) != (n, hv, dv):
        raise ValueError("o must be [N, Hv, d_v]")
    shp = _shape(n, hk, hv, dk, dv, _dtype_code(q), scale)
    stream = torch.cuda.current_stream(device)
    _check(lib.gdn_decode_step(ctypes.byref(shp), _ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta),
                               _ptr(state_in), _ptr(o), _ptr(state_out),
                               ctypes.c_void_p(stream.cuda_stream)))
    return o, state_out


# ---------------------------------------------------------------- layer block

LA_WEIGHT_NAMES = ("w_in", "conv_w", "a_log", "dt_bias", "norm_w", "w_out")


def la_block_stage_names(with_outputs: bool):
    """Names of the stages ``la_block_replay`` enqueues, in order."""
    lib = load_library()
    n = lib.gdn_la_block_num_stages(int(with_outputs))
    return [lib.gdn_la_block_stage_name(int(with_outputs), i).decode() for i in range(n)]


def _la_shape(n, hidden, hk, hv, dk, dv, act_dtype, scale, l2_eps, norm_eps):
    code = {"f32": GDN_F32, "bf16": GDN_BF16}.get(act_dtype)
    if code is None:
        raise ValueError("act_dtype must be 'f32' or 'bf16'")
    return LAShape(n, hidden, hk, hv, dk, dv, 4, code, float(scale), float(l2_eps), float(norm_eps))


def la_block_workspace_size(hidden: int, num_k_heads: int, num_v_heads: int, d_k: int, d_v: int,
                            cu_seqlens_host: Sequence[int], with_outputs: bool = True,
                            act_dtype: str = "f32") -> int:
    lib = load_library()
    cu = torch.tensor(list(cu_seqlens_host), dtype=torch.int32)
    shp = _la_shape(cu.numel() - 1, hidden, num_k_heads, num_v_heads, d_k, d_v, act_dtype, 1.0, 0.0, 0.0)
    out = ctypes.c_size_t(0)
    _check(lib.gdn_la_block_workspace_size(ctypes.byref(shp), _ptr(cu), int(with_outputs),
                                           ctypes.byref(out)))
    return int(out.value)


def la_block_replay(x: torch.Tensor, weights, cu_seqlens, num_k_heads: int, num_v_heads: int,
                    d_k: int, d_v: int, scale: float, cu_seqlens_host=None, outputs: bool = True,
                    act_dtype: str = "f32", l2_eps: float = 1e-6, norm_eps: float = 1e-6,
                    state_out: Optional[torch.Tensor] = None, out: Optional[torch.Tensor] = None,
                    workspace: Optional[torch.Tensor] = None, events=None):
    """Replay of one linear-attention layer over packed tails (paper Section 3,
    Eq. 2 behind the layer's projections) on torch's current stream.

    x [T, D] bf16: the cached hiddens; ``weights``: mapping with w_in bf16
    [2cq+2cv+2Hv, D] (rows q|k|v|a|b|z), conv_w fp32 [2cq+cv, 4], a_log and
    dt_bias fp32 [Hv], norm_w fp32 [d_v], w_out bf16 [D, cv] (the last two
    unused when ``outputs`` is False).  Returns ``(state_out [N,Hv,d_k,d_v]
    fp32, out [T, D] bf16 or None)``.
    """
    lib = load_library()
    device = x.device
    _need(x, "x", torch.bfloat16, device, 2)
    T, D = x.shape
    cq, cv = num_k_heads * d_k, num_v_heads * d_v
    specs = {"w_in": (torch.bfloat16, (2 * cq + 2 * cv + 2 * num_v_heads, D)),
             "conv_w": (torch.float32, (2 * cq + cv, 4)),
             "a_log": (torch.float32, (num_v_heads,)), "dt_bias": (torch.float32, (num_v_heads,)),
             "norm_w": (torch.float32, (d_v,)), "w_out": (torch.bfloat16, (D, cv))}
    ptrs = {}
    for name in LA_WEIGHT_NAMES:
        t = weights.get(name)
        if t is None and not outputs and name in ("norm_w", "w_out"):
            ptrs[name] = None
            continue
        dt, shp = specs[name]
        _need(t, name, dt, device, len(shp))
        if tuple(t.shape) != shp:
            raise ValueError(f"{name} must be {list(shp)}, got {list(t.shape)}")
        ptrs[name] = t.data_ptr()
    w = LAWeights(*(ptrs[n] for n in LA_WEIGHT_NAMES))
    cu_dev, cu_host = _seqlens(cu_seqlens, cu_seqlens_host, device)
    n = cu_host.numel() - 1
    if state_out is None:
        state_out = torch.empty((n, num_v_heads, d_k, d_v), dtype=torch.float32, device=device)
    _need(state_out, "state_out", torch.float32, device, 4)
    if tuple(state_out.shape) != (n, num_v_heads, d_k, d_v):
        raise ValueError("state_out must be [N, Hv, d_k, d_v]")
    if outputs:
        if out is None:
            out = torch.empty((T, D), dtype=torch.bfloat16, device=device)
        _need(out, "out", torch.bfloat16, device, 2)
        if tuple(out.shape) != (T, D):
            raise ValueError("out must be [T, D]")
    else:
        out = None
    shp = _la_shape(n, D, num_k_heads, num_v_heads, d_k, d_v, act_dtype, scale, l2_eps, norm_eps)
    stream = torch.cuda.current_stream(device)
    need = ctypes.c_size_t(0)
    _check(lib.gdn_la_block_workspace_size(ctypes.byref(shp), _ptr(cu_host), int(outputs),
                                           ctypes.byref(need)))
    ws = workspace if workspace is not None else _workspace(need.value, device, stream)
    args = [ctypes.byref(shp), ctypes.byref(w), _ptr(cu_host), _ptr(cu_dev), _ptr(x), _ptr(state_out),
            _ptr(out), _ptr(ws), ws.numel() * ws.element_size(), ctypes.c_void_p(stream.cuda_stream)]
    if events is None:
        _check(lib.gdn_la_block_replay(*args))
    else:
        ne = lib.gdn_la_block_num_stages(int(outputs)) + 1
        if len(events) != ne:
            raise ValueError(f"need {ne} events (one per stage boundary)")
        handles = []
        for ev in events:
            if ev.cuda_event == 0:
                ev.record()
            handles.append(ev.cuda_event)
        arr = (ctypes.c_void_p * ne)(*handles)
        _check(lib.gdn_la_block_replay_profiled(*args, ctypes.cast(arr, ctypes.c_void_p), ne))
    return state_out, out

