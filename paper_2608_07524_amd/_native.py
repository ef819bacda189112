"""ctypes binding of libdcp (the C ABI in include/dcp.h).

Argument marshalling only: every step of attention, profiling and planning
runs inside libdcp.  PyTorch supplies device memory and the current stream.
The library must be built (``python -m paper_2608_07524_amd.build``); there
is no fallback.
"""

from __future__ import annotations

import ctypes as C
import math
import os
from dataclasses import dataclass, field
from typing import List, Optional, Sequence

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libdcp.so")

DCP_OK = 0
DCP_ERR_INVALID = -1
DCP_ERR_UNSUPPORTED = -2
DCP_ERR_HIP = -3
DCP_ERR_WORKSPACE = -4
DCP_ERR_INFEASIBLE = -5
DCP_ERR_TABLE = -6

PLAN_INTER = 0
PLAN_INTRA = 1
PLAN_FLAG_MIN_TIME = 1
PLAN_FLAG_NO_HEAD_FILTER = 2


class DCPError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"libdcp error {code}: {msg}")
        self.code = code


class AttnDesc(C.Structure):
    _fields_ = [("n_seqs", C.c_int32), ("cu_seqlens_host", C.POINTER(C.c_int32)), ("total_tokens", C.c_int64),
                ("n_heads", C.c_int32), ("head_dim", C.c_int32), ("scale", C.c_float), ("causal", C.c_int32)]


class CostRow(C.Structure):
    _fields_ = [("seq_len", C.c_int64), ("t_f_ns", C.c_int64), ("t_b_ns", C.c_int64), ("m_bytes", C.c_int64),
                ("m_inp_bytes", C.c_int64)]


class ProfileOpts(C.Structure):
    _fields_ = [("n_heads", C.c_int32), ("head_dim", C.c_int32), ("causal", C.c_int32), ("scale", C.c_float),
                ("warmup", C.c_int32), ("reps", C.c_int32), ("lin_f_ps_per_token", C.c_int64),
                ("lin_b_ps_per_token", C.c_int64), ("act_bytes_per_token", C.c_int64),
                ("inp_bytes_per_token", C.c_int64)]


class CostTableC(C.Structure):
    _fields_ = [("rows", C.POINTER(CostRow)), ("n_rows", C.c_int32), ("n_layers", C.c_int32),
                ("T_C_ns", C.c_int64), ("M_C_bytes", C.c_int64)]


class PlanOptsC(C.Structure):
    _fields_ = [("sp_cands", C.POINTER(C.c_int32)), ("n_sp", C.c_int32), ("b_max", C.c_int32),
                ("n_heads", C.c_int32), ("hidden", C.c_int64), ("a2a_alpha_ns", C.c_int64),
                ("link_bytes_per_ns", C.c_int64), ("g_min", C.c_int32), ("g_max", C.c_int32),
                ("mode", C.c_int32), ("flags", C.c_int32)]


class PlanOutC(C.Structure):
    _fields_ = [("sp_size", C.POINTER(C.c_int32)), ("micro_batch", C.POINTER(C.c_int32)),
                ("grad_accum", C.POINTER(C.c_int32)), ("recompute_layers", C.POINTER(C.c_int32)),
                ("recompute_flags", C.POINTER(C.c_uint8)), ("step_time_ns", C.POINTER(C.c_int64)),
                ("mem_bytes", C.POINTER(C.c_int64)), ("idle_ns", C.c_int64), ("makespan_ns", C.c_int64)]


class SimOptsC(C.Structure):
    _fields_ = [("n_devices", C.c_int32), ("bucket_sp", C.c_int32), ("iter_sync_ns", C.c_int64)]


class SimResultC(C.Structure):
    _fields_ = [("iterations", C.c_int64), ("makespan_ns", C.c_int64), ("time_ns", C.c_int64),
                ("busy_device_ns", C.c_int64), ("tokens", C.c_int64), ("bucket_sp", C.c_int32)]


class LayerDescC(C.Structure):
    _fields_ = [("attn", C.POINTER(AttnDesc)), ("eps", C.c_float)]


class LayerWeightsC(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in ("norm1", "wq", "wk", "wv", "wo", "norm2", "w_up", "w_down")]


LAYER_PARAMS = ("norm1", "wq", "wk", "wv", "wo", "norm2", "w_up", "w_down")

_lib = None


def load() -> C.CDLL:
    """Load libdcp.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2608_07524_amd.build`")
    lib = C.CDLL(LIB_PATH)
    vp, sz = C.c_void_p, C.c_size_t
    sig = {
        "dcp_last_error": ([], C.c_char_p),
        "dcp_version": ([], C.c_char_p),
        "dcp_varlen_attn_fwd_workspace_size": ([C.POINTER(AttnDesc), C.POINTER(sz)], C.c_int),
        "dcp_varlen_attn_bwd_workspace_size": ([C.POINTER(AttnDesc), C.POINTER(sz)], C.c_int),
        "dcp_varlen_attn_fwd": ([C.POINTER(AttnDesc), vp, vp, vp, vp, vp, vp, sz, vp], C.c_int),
        "dcp_varlen_attn_bwd": ([C.POINTER(AttnDesc), vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp], C.c_int),
        "dcp_set_kernel_events": ([vp, vp], C.c_int),
        "dcp_device_info": ([C.POINTER(C.c_int32), C.POINTER(C.c_int32)], C.c_int),
        "dcp_varlen_attn_fwd_noalloc": ([C.POINTER(AttnDesc), vp, vp, vp, vp, vp, vp], C.c_int),
        "dcp_batch_create": ([C.POINTER(AttnDesc), C.POINTER(vp)], C.c_int),
        "dcp_batch_workspace_size": ([vp, C.POINTER(sz)], C.c_int),
        "dcp_batch_upload": ([vp, vp, sz, vp], C.c_int),
        "dcp_batch_fwd": ([vp, vp, vp, vp, vp, vp, vp, sz, vp], C.c_int),
        "dcp_batch_bwd": ([vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp], C.c_int),
        "dcp_batch_destroy": ([vp], None),
        "dcp_work_list": ([C.POINTER(AttnDesc), C.c_int32, C.POINTER(C.c_int32), sz, C.POINTER(sz), C.POINTER(sz),
                           C.POINTER(C.c_uint64), sz, C.POINTER(sz)], C.c_int),
        "dcp_profile_workspace_size": ([C.c_int64, C.POINTER(ProfileOpts), C.POINTER(sz)], C.c_int),
        "dcp_profile_cost": ([C.POINTER(C.c_int64), C.c_int32, C.POINTER(ProfileOpts), vp, sz, vp,
                              C.POINTER(CostRow)], C.c_int),
        "dcp_plan_opts_default": ([C.POINTER(PlanOptsC)], None),
        "dcp_plan": ([C.POINTER(C.c_int64), C.c_int32, C.POINTER(C.c_int32), C.c_int32, C.POINTER(CostTableC),
                      C.c_int64, C.POINTER(PlanOptsC), C.POINTER(PlanOutC)], C.c_int),
        "dcp_layer_sizes": ([C.POINTER(LayerDescC), C.POINTER(sz), C.POINTER(sz), C.POINTER(sz)], C.c_int),
        "dcp_layer_fwd": ([C.POINTER(LayerDescC), C.POINTER(LayerWeightsC), vp, vp, vp, vp, sz, vp], C.c_int),
        "dcp_layer_bwd": ([C.POINTER(LayerDescC), C.POINTER(LayerWeightsC), vp, vp, vp, C.POINTER(LayerWeightsC), vp,
                           vp, sz, vp], C.c_int),
        "dcp_simulate": ([C.POINTER(C.c_int64), C.c_int32, C.POINTER(C.c_int32), C.c_int32, C.POINTER(CostTableC),
                          C.c_int64, C.POINTER(PlanOptsC), C.POINTER(SimOptsC), C.POINTER(SimResultC),
                          C.POINTER(SimResultC)], C.c_int),
    }
    for name, (args, res) in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    _lib = lib
    return lib


def last_error() -> str:
    return load().dcp_last_error().decode()


def _check(status: int):
    if status != DCP_OK:
        raise DCPError(status, last_error())


# ---------------------------------------------------------------------------
# attention

class _Desc:
    """Keeps a dcp_attn_desc and the host cu_seqlens array it points to alive."""

    def __init__(self, cu_seqlens, total_tokens: int, n_heads: int, head_dim: int, scale: float, causal: bool):
        self.cu = np.ascontiguousarray(np.asarray(cu_seqlens, dtype=np.int32))
        self.desc = AttnDesc(int(self.cu.size - 1), self.cu.ctypes.data_as(C.POINTER(C.c_int32)), int(total_tokens),
                             int(n_heads), int(head_dim), float(scale), int(bool(causal)))

    @property
    def ref(self):
        return C.byref(self.desc)


def _host_cu(cu_seqlens):
    """cu_seqlens as a host int32 array; raises on values int32 cannot hold
    (the C ABI reads int32) or on non-integer input."""
    if hasattr(cu_seqlens, "detach"):
        cu_seqlens = cu_seqlens.detach().cpu().numpy()
    a = np.asarray(cu_seqlens)
    if a.ndim != 1 or a.size < 2:
        raise ValueError("cu_seqlens must be a 1-D sequence of at least two offsets")
    if a.dtype.kind not in "iu":
        if a.dtype.kind == "f" and np.all(np.floor(a) == a):
            a = a.astype(np.int64)
        else:
            raise ValueError("cu_seqlens must hold integers")
    if int(a.min()) < 0 or int(a.max()) > np.iinfo(np.int32).max:
        raise ValueError("cu_seqlens values must lie in [0, 2^31 - 1]")
    return np.ascontiguousarray(a, dtype=np.int32)


def _stream_ptr(torch, device):
    return C.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def fwd_workspace_size(cu_seqlens, total_tokens, n_heads, head_dim, scale=1.0, causal=False) -> int:
    d = _Desc(_host_cu(cu_seqlens), total_tokens, n_heads, head_dim, scale, causal)
    n = C.c_size_t()
    _check(load().dcp_varlen_attn_fwd_workspace_size(d.ref, C.byref(n)))
    return n.value


def bwd_workspace_size(cu_seqlens, total_tokens, n_heads, head_dim, scale=1.0, causal=False) -> int:
    d = _Desc(_host_cu(cu_seqlens), total_tokens, n_heads, head_dim, scale, causal)
    n = C.c_size_t()
    _check(load().dcp_varlen_attn_bwd_workspace_size(d.ref, C.byref(n)))
    return n.value


def _check_attn(torch, q, others=(), lse=None, workspace=None):
    """Checks, before any library call, everything the C ABI cannot see
    behind its raw pointers: q is a contiguous bf16 [T, H, D] tensor; every
    tensor in ``others`` (name, tensor) has q's shape, dtype and device and is
    contiguous; ``lse`` is contiguous fp32 [H, T] on that device; the
    workspace is contiguous on that device.  Shapes and dtypes are checked
    before the device, so a mismatch is reported as such on any device.
    Returns (T, H, D)."""
    if not hasattr(q, "dim") or q.dim() != 3:
        raise ValueError("q must be a tensor of shape [T, H, D]")
    if q.dtype != torch.bfloat16 or not q.is_contiguous():
        raise ValueError("q must be a contiguous bf16 tensor")
    for name, t in others:
        if tuple(t.shape) != tuple(q.shape):
            raise ValueError(f"{name} has shape {tuple(t.shape)}, q has {tuple(q.shape)}")
        if t.dtype != torch.bfloat16 or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous bf16 tensor")
    T, H, D = (int(x) for x in q.shape)
    if lse is not None:
        if tuple(lse.shape) != (H, T) or lse.dtype != torch.float32 or not lse.is_contiguous():
            raise ValueError(f"lse must be a contiguous float32 tensor of shape ({H}, {T})")
    if workspace is not None and not workspace.is_contiguous():
        raise ValueError("workspace must be contiguous")
    if not q.is_cuda:
        raise ValueError("tensors must be on a CUDA (HIP) device")
    for name, t in list(others) + [("lse", lse), ("workspace", workspace)]:
        if t is not None and t.device != q.device:
            raise ValueError(f"{name} is on {t.device}, q on {q.device}")
    return T, H, D


def _nbytes(t) -> int:
    return int(t.numel()) * int(t.element_size())


def varlen_attn_fwd(q, k, v, cu_seqlens, scale: Optional[float] = None, causal: bool = False,
                    out=None, lse=None, workspace=None):
    """O, LSE = attention over packed sequences (see dcp_varlen_attn_fwd)."""
    import torch
    given = [("k", k), ("v", v)] + ([("out", out)] if out is not None else [])
    T, H, D = _check_attn(torch, q, given, lse, workspace)
    scale = 1.0 / math.sqrt(D) if scale is None else scale
    d = _Desc(_host_cu(cu_seqlens), T, H, D, scale, causal)
    lib = load()
    n = C.c_size_t()
    _check(lib.dcp_varlen_attn_fwd_workspace_size(d.ref, C.byref(n)))
    o = torch.empty_like(q) if out is None else out
    lse = torch.empty((H, T), dtype=torch.float32, device=q.device) if lse is None else lse
    ws = torch.empty(n.value, dtype=torch.uint8, device=q.device) if workspace is None else workspace
    _check(lib.dcp_varlen_attn_fwd(d.ref, q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), lse.data_ptr(),
                                   ws.data_ptr(), _nbytes(ws), _stream_ptr(torch, q.device)))
    return o, lse


def varlen_attn_fwd_noalloc(q, k, v, cu_seqlens, scale: Optional[float] = None, causal: bool = False,
                            out=None, lse=None):
    """O, LSE through dcp_varlen_attn_fwd_noalloc (the library's fixed
    scratch instead of a workspace; pass ``out`` and ``lse`` to allocate
    nothing here either)."""
    import torch
    given = [("k", k), ("v", v)] + ([("out", out)] if out is not None else [])
    T, H, D = _check_attn(torch, q, given, lse)
    scale = 1.0 / math.sqrt(D) if scale is None else scale
    d = _Desc(_host_cu(cu_seqlens), T, H, D, scale, causal)
    o = torch.empty_like(q) if out is None else out
    lse = torch.empty((H, T), dtype=torch.float32, device=q.device) if lse is None else lse
    _check(load().dcp_varlen_attn_fwd_noalloc(d.ref, q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(),
                                              lse.data_ptr(), _stream_ptr(torch, q.device)))
    return o, lse


def varlen_attn_bwd(dout, o, lse, q, k, v, cu_seqlens, scale: Optional[float] = None, causal: bool = False,
                    dq=None, dk=None, dv=None, workspace=None):
    """dQ, dK, dV of the loss <dO, O> (see dcp_varlen_attn_bwd)."""
    import torch
    given = [("k", k), ("v", v), ("dout", dout), ("o", o)]
    given += [(n_, t) for n_, t in (("dq", dq), ("dk", dk), ("dv", dv)) if t is not None]
    T, H, D = _check_attn(torch, q, given, lse, workspace)
    scale = 1.0 / math.sqrt(D) if scale is None else scale
    d = _Desc(_host_cu(cu_seqlens), T, H, D, scale, causal)
    lib = load()
    n = C.c_size_t()
    _check(lib.dcp_varlen_attn_bwd_workspace_size(d.ref, C.byref(n)))
    dq = torch.empty_like(q) if dq is None else dq
    dk = torch.empty_like(k) if dk is None else dk
    dv = torch.empty_like(v) if dv is None else dv
    ws = torch.empty(n.value, dtype=torch.uint8, device=q.device) if workspace is None else workspace
    _check(lib.dcp_varlen_attn_bwd(d.ref, dout.data_ptr(), o.data_ptr(), lse.data_ptr(), q.data_ptr(),
                                   k.data_ptr(), v.data_ptr(), dq.data_ptr(), dk.data_ptr(), dv.data_ptr(),
                                   ws.data_ptr(), _nbytes(ws), _stream_ptr(torch, q.device)))
    return dq, dk, dv


class PreparedAttention:
    """Forward + backward calls on fixed buffers over one prepared batch
    (dcp_batch_create / dcp_batch_upload): the work lists are built and
    copied to the device once, so each later call only launches kernels."""

    def __init__(self, q, k, v, dout, cu_seqlens, scale: Optional[float] = None, causal: bool = False):
        import torch
        T, H, D = _check_attn(torch, q, [("k", k), ("v", v), ("dout", dout)])
        self.torch = torch
        self.scale = 1.0 / math.sqrt(D) if scale is None else scale
        self.d = _Desc(_host_cu(cu_seqlens), T, H, D, self.scale, causal)
        lib = self.lib = load()
        self.batch = None
        h = C.c_void_p()
        _check(lib.dcp_batch_create(self.d.ref, C.byref(h)))
        self.batch = h
        n = C.c_size_t()
        _check(lib.dcp_batch_workspace_size(self.batch, C.byref(n)))
        self.q, self.k, self.v, self.dout = q, k, v, dout
        self.o = torch.empty_like(q)
        self.lse = torch.empty((H, T), dtype=torch.float32, device=q.device)
        self.dq, self.dk, self.dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
        self.ws = torch.empty(max(1, n.value), dtype=torch.uint8, device=q.device)
        self.stream = _stream_ptr(torch, q.device)
        _check(lib.dcp_batch_upload(self.batch, self.ws.data_ptr(), self.ws.numel(), self.stream))

    def fwd(self):
        _check(self.lib.dcp_batch_fwd(self.batch, self.q.data_ptr(), self.k.data_ptr(), self.v.data_ptr(),
                                      self.o.data_ptr(), self.lse.data_ptr(), self.ws.data_ptr(), self.ws.numel(),
                                      self.stream))

    def bwd(self):
        _check(self.lib.dcp_batch_bwd(self.batch, self.dout.data_ptr(), self.o.data_ptr(), self.lse.data_ptr(),
                                      self.q.data_ptr(), self.k.data_ptr(), self.v.data_ptr(), self.dq.data_ptr(),
                                      self.dk.data_ptr(), self.dv.data_ptr(), self.ws.data_ptr(), self.ws.numel(),
                                      self.stream))

    def step(self):
        self.fwd()
        self.bwd()

    def __del__(self):
        if getattr(self, "batch", None):
            self.lib.dcp_batch_destroy(self.batch)
            self.batch = None


def device_info() -> dict:
    """Compute units and peak engine clock of the current device (see
    dcp_device_info)."""
    cus, khz = C.c_int32(), C.c_int32()
    _check(load().dcp_device_info(C.byref(cus), C.byref(khz)))
    return {"compute_units": cus.value, "clock_mhz": khz.value / 1000.0}


def set_kernel_events(begin=None, end=None):
    """Record the hipEvent_t handles ``begin``/``end`` (ints) around each
    following call's main attention kernel; ``None`` clears the hook (see
    dcp_set_kernel_events)."""
    _check(load().dcp_set_kernel_events(None if begin is None else C.c_void_p(begin),
                                        None if end is None else C.c_void_p(end)))


def work_list(cu_seqlens, n_heads: int, head_dim: int, causal: bool, pass_: int):
    """The tile list one kernel pass runs (0 forward, 1 dK/dV, 2 dQ; see
    dcp_work_list): (units int32 [n, 5] = row0, seq0, seqlen, rows, head;
    n_tiles, the count of sequence-tile units before the packed windows;
    window_starts uint64 [n_windows, 4])."""
    cu = _host_cu(cu_seqlens)
    d = _Desc(cu, int(cu[-1]), n_heads, head_dim, 1.0, causal)
    lib = load()
    n, nt, nw = C.c_size_t(), C.c_size_t(), C.c_size_t()
    _check(lib.dcp_work_list(C.byref(d.desc), int(pass_), None, 0, C.byref(n), C.byref(nt), None, 0, C.byref(nw)))
    units = np.zeros((max(n.value, 1), 5), dtype=np.int32)
    starts = np.zeros((max(nw.value, 1), 4), dtype=np.uint64)
    _check(lib.dcp_work_list(C.byref(d.desc), int(pass_), units.ctypes.data_as(C.POINTER(C.c_int32)), n.value,
                             C.byref(n), C.byref(nt), starts.ctypes.data_as(C.POINTER(C.c_uint64)), nw.value,
                             C.byref(nw)))
    return units[:n.value], nt.value, starts[:nw.value]


# ---------------------------------------------------------------------------
# profiling

def profile_cost(lengths: Sequence[int], n_heads: int, head_dim: int, causal: bool = False,
                 scale: float = 0.0, warmup: int = 3, reps: int = 10, lin_f_ps_per_token: int = 0,
                 lin_b_ps_per_token: int = 0, act_bytes_per_token: int = 0, inp_bytes_per_token: int = 0,
                 device=None) -> List[CostRow]:
    """Measured per-length cost rows (see dcp_profile_cost)."""
    import torch
    lib = load()
    opts = ProfileOpts(n_heads, head_dim, int(causal), scale, warmup, reps, lin_f_ps_per_token,
                       lin_b_ps_per_token, act_bytes_per_token, inp_bytes_per_token)
    lens = np.ascontiguousarray(np.asarray(lengths, dtype=np.int64))
    n = C.c_size_t()
    _check(lib.dcp_profile_workspace_size(int(lens.max()), C.byref(opts), C.byref(n)))
    dev = torch.device("cuda") if device is None else device
    ws = torch.empty(n.value, dtype=torch.uint8, device=dev)
    out = (CostRow * lens.size)()
    _check(lib.dcp_profile_cost(lens.ctypes.data_as(C.POINTER(C.c_int64)), int(lens.size), C.byref(opts),
                                ws.data_ptr(), ws.numel(), _stream_ptr(torch, dev), out))
    return [CostRow(r.seq_len, r.t_f_ns, r.t_b_ns, r.m_bytes, r.m_inp_bytes) for r in out]


# ---------------------------------------------------------------------------
# planner

@dataclass
class Plan:
    sp_size: List[int] = field(default_factory=list)
    micro_batch: List[int] = field(default_factory=list)
    grad_accum: List[int] = field(default_factory=list)
    recompute_layers: List[int] = field(default_factory=list)
    recompute_flags: List[int] = field(default_factory=list)
    step_time_ns: List[int] = field(default_factory=list)
    mem_bytes: List[int] = field(default_factory=list)
    idle_ns: int = 0
    makespan_ns: int = 0


def default_plan_opts() -> dict:
    o = PlanOptsC()
    load().dcp_plan_opts_default(C.byref(o))
    return dict(sp_cands=tuple(o.sp_cands[i] for i in range(o.n_sp)), b_max=o.b_max, n_heads=o.n_heads,
                hidden=o.hidden, a2a_alpha_ns=o.a2a_alpha_ns, link_bytes_per_ns=o.link_bytes_per_ns,
                g_min=o.g_min, g_max=o.g_max, mode=o.mode, flags=o.flags)


def _plan_opts(lib, opts):
    """dcp_plan_opts from the defaults with ``opts`` overrides; returns the
    struct and the arrays it points to (kept alive by the caller)."""
    o = PlanOptsC()
    lib.dcp_plan_opts_default(C.byref(o))
    keep = []
    for key, val in opts.items():
        if key == "sp_cands":
            sp = np.ascontiguousarray(np.asarray(val, dtype=np.int32))
            keep.append(sp)
            o.sp_cands = sp.ctypes.data_as(C.POINTER(C.c_int32))
            o.n_sp = int(sp.size)
        elif hasattr(o, key):
            setattr(o, key, int(val))
        else:
            raise TypeError(f"unknown planner option {key}")
    return o, keep


def _cost_table(rows, n_layers, T_C_ns, M_C_bytes):
    crow = (CostRow * len(rows))()
    for i, r in enumerate(rows):
        vals = (r.seq_len, r.t_f_ns, r.t_b_ns, r.m_bytes, r.m_inp_bytes) if hasattr(r, "seq_len") else tuple(r)
        crow[i] = CostRow(*[int(x) for x in vals])
    return CostTableC(crow, len(rows), int(n_layers), int(T_C_ns), int(M_C_bytes)), crow


def _batches(seq_lens, batch_offsets, n_batches):
    lens = np.ascontiguousarray(np.asarray(seq_lens, dtype=np.int64))
    offs = None
    if batch_offsets is not None:
        offs = np.ascontiguousarray(np.asarray(batch_offsets, dtype=np.int32))
        nb = int(offs.size - 1) if n_batches is None else int(n_batches)
    else:
        nb = int(lens.size) if n_batches is None else int(n_batches)
    return lens, offs, nb


def plan(seq_lens: Sequence[int], rows: Sequence, n_layers: int, T_C_ns: int, M_C_bytes: int, hbm_budget: int,
         batch_offsets: Optional[Sequence[int]] = None, n_batches: Optional[int] = None, **opts) -> Plan:
    """Plan one iteration (see dcp_plan).  ``rows``: (seq_len, t_f, t_b, m, m_inp)
    tuples or CostRow objects; ``opts`` override dcp_plan_opts_default."""
    lib = load()
    o, _keep = _plan_opts(lib, opts)
    table, _rows = _cost_table(rows, n_layers, T_C_ns, M_C_bytes)
    lens, offs, nb = _batches(seq_lens, batch_offsets, n_batches)
    nb_alloc = max(nb, 1)
    i32 = lambda: (C.c_int32 * nb_alloc)()
    i64 = lambda: (C.c_int64 * nb_alloc)()
    sp_o, mb_o, ga_o, rl_o = i32(), i32(), i32(), i32()
    fl_o = (C.c_uint8 * max(1, nb_alloc * max(1, int(n_layers))))()
    st_o, mem_o = i64(), i64()
    out = PlanOutC(sp_o, mb_o, ga_o, rl_o, fl_o, st_o, mem_o, 0, 0)
    _check(lib.dcp_plan(lens.ctypes.data_as(C.POINTER(C.c_int64)), int(lens.size),
                        None if offs is None else offs.ctypes.data_as(C.POINTER(C.c_int32)), nb, C.byref(table),
                        int(hbm_budget), C.byref(o), C.byref(out)))
    L = int(n_layers)
    return Plan(list(sp_o[:nb]), list(mb_o[:nb]), list(ga_o[:nb]), list(rl_o[:nb]), list(fl_o[:nb * L]),
                list(st_o[:nb]), list(mem_o[:nb]), out.idle_ns, out.makespan_ns)


def simulate(seq_lens: Sequence[int], rows: Sequence, n_layers: int, T_C_ns: int, M_C_bytes: int, hbm_budget: int,
             n_devices: int, bucket_sp: int = 0, iter_sync_ns: int = 0,
             batch_offsets: Optional[Sequence[int]] = None, n_batches: Optional[int] = None, **opts):
    """Replay a stream of batches under DCP and under bucket parallelism (see
    dcp_simulate).  Returns two dicts of totals (iterations, makespan_ns,
    time_ns, busy_device_ns, tokens, bucket_sp), DCP's first."""
    lib = load()
    o, _keep = _plan_opts(lib, opts)
    table, _rows = _cost_table(rows, n_layers, T_C_ns, M_C_bytes)
    lens, offs, nb = _batches(seq_lens, batch_offsets, n_batches)
    sim = SimOptsC(int(n_devices), int(bucket_sp), int(iter_sync_ns))
    a, b = SimResultC(), SimResultC()
    _check(lib.dcp_simulate(lens.ctypes.data_as(C.POINTER(C.c_int64)), int(lens.size),
                            None if offs is None else offs.ctypes.data_as(C.POINTER(C.c_int32)), nb,
                            C.byref(table), int(hbm_budget), C.byref(o), C.byref(sim), C.byref(a), C.byref(b)))
    as_dict = lambda r: {k: int(getattr(r, k)) for k, _ in SimResultC._fields_}
    return as_dict(a), as_dict(b)


# ---------------------------------------------------------------------------
# transformer layer

def layer_param_shapes(hidden: int):
    """Shapes of the layer parameters (row-major [in, out] matrices)."""
    h = int(hidden)
    return {"norm1": (h,), "wq": (h, h), "wk": (h, h), "wv": (h, h), "wo": (h, h), "norm2": (h,),
            "w_up": (h, 4 * h), "w_down": (4 * h, h)}


class Layer:
    """One transformer layer over a fixed packed batch (see dcp_layer_fwd /
    dcp_layer_bwd): ``weights`` bf16 and ``grads`` fp32 device tensors keyed
    by LAYER_PARAMS.  ``fwd(x, keep)`` returns the output and keeps the
    activation stash when ``keep``; ``bwd(x, dout)`` returns dx, adding the
    weight gradients into ``grads`` and recomputing the forward first when
    no stash was kept."""

    def __init__(self, weights, grads, cu_seqlens, n_heads: int, head_dim: int, causal: bool = False,
                 scale: Optional[float] = None, eps: float = 1e-6, workspace=None):
        import torch
        self.torch = torch
        self.weights, self.grads = weights, grads
        cu = _host_cu(cu_seqlens)
        T = int(cu[-1])
        self.T, self.hidden = T, n_heads * head_dim
        self.scale = 1.0 / math.sqrt(head_dim) if scale is None else scale
        self.d = _Desc(cu, T, n_heads, head_dim, self.scale, causal)
        self.desc = LayerDescC(C.pointer(self.d.desc), float(eps))
        lib = self.lib = load()
        s, f, b = C.c_size_t(), C.c_size_t(), C.c_size_t()
        _check(lib.dcp_layer_sizes(C.byref(self.desc), C.byref(s), C.byref(f), C.byref(b)))
        self.stash_bytes, self.fwd_ws_bytes, self.bwd_ws_bytes = s.value, f.value, b.value
        dev = weights["wq"].device
        self.w = LayerWeightsC(*[weights[n].data_ptr() for n in LAYER_PARAMS])
        self.g = LayerWeightsC(*[grads[n].data_ptr() for n in LAYER_PARAMS])
        need = max(self.fwd_ws_bytes, self.bwd_ws_bytes)
        if workspace is not None and workspace.numel() < need:
            raise ValueError(f"layer workspace needs {need} bytes")
        # (several layers of one shape may share one workspace: calls on a stream run in order)
        self.ws = torch.empty(need, dtype=torch.uint8, device=dev) if workspace is None else workspace
        self.stream = _stream_ptr(torch, dev)
        self.stash = None

    def fwd(self, x, keep: bool = True, out=None, stash=None):
        """``stash``: a preallocated buffer of stash_bytes to keep into."""
        t = self.torch
        out = t.empty_like(x) if out is None else out
        if keep:
            self.stash = t.empty(self.stash_bytes, dtype=t.uint8, device=x.device) if stash is None else stash
        else:
            self.stash = None
        _check(self.lib.dcp_layer_fwd(C.byref(self.desc), C.byref(self.w), x.data_ptr(), out.data_ptr(),
                                      None if self.stash is None else self.stash.data_ptr(), self.ws.data_ptr(),
                                      _nbytes(self.ws), self.stream))
        return out

    def bwd(self, x, dout, dx=None):
        t = self.torch
        dx = t.empty_like(x) if dx is None else dx
        _check(self.lib.dcp_layer_bwd(C.byref(self.desc), C.byref(self.w), x.data_ptr(), dout.data_ptr(),
                                      dx.data_ptr(), C.byref(self.g),
                                      None if self.stash is None else self.stash.data_ptr(), self.ws.data_ptr(),
                                      _nbytes(self.ws), self.stream))
        self.stash = None
        return dx
