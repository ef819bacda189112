"""The C ABI on the CPU: every declared symbol is exported, and argument
errors are reported with the documented status before any device call."""

import ctypes as C
import os
import re

import numpy as np
import pytest

import paper_2608_07524_amd as P
from paper_2608_07524_amd import _native as N

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    names = set()
    for fn in os.listdir(os.path.join(ROOT, "include")):
        if fn.endswith(".h"):
            src = open(os.path.join(ROOT, "include", fn)).read()
            src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
            names |= set(re.findall(r"\b(dcp_[a-z0-9_]+)\s*\(", src))
    return names


def test_library_exports_every_declared_symbol():
    lib = C.CDLL(N.LIB_PATH)
    names = _declared_functions()
    assert {"dcp_varlen_attn_fwd", "dcp_varlen_attn_bwd", "dcp_profile_cost", "dcp_plan"} <= names
    for name in sorted(names):
        assert hasattr(lib, name), name


def _desc(cu, T, H=2, D=64, scale=0.125, causal=0):
    cu = np.asarray(cu, dtype=np.int32)
    d = N.AttnDesc(cu.size - 1, cu.ctypes.data_as(C.POINTER(C.c_int32)), T, H, D, scale, causal)
    return d, cu


@pytest.mark.parametrize("kw,code", [
    (dict(cu=[1, 5], T=5), N.DCP_ERR_INVALID),        # cu[0] != 0
    (dict(cu=[0, 5, 3], T=5), N.DCP_ERR_INVALID),     # decreasing
    (dict(cu=[0, 9], T=5), N.DCP_ERR_INVALID),        # beyond total_tokens
    (dict(cu=[0, 5], T=5, H=0), N.DCP_ERR_INVALID),
    (dict(cu=[0, 5], T=5, H=65536), N.DCP_ERR_INVALID),  # heads travel as uint16 in the work lists
    (dict(cu=[0, 5], T=5, D=96), N.DCP_ERR_UNSUPPORTED),
    (dict(cu=[0, 5], T=5, scale=0.0), N.DCP_ERR_INVALID),
    (dict(cu=[0, 5], T=5, scale=float("nan")), N.DCP_ERR_INVALID),
    (dict(cu=[0, 5], T=5, causal=2), N.DCP_ERR_INVALID),
    (dict(cu=[0, 5], T=1 << 31), N.DCP_ERR_INVALID),
])
def test_descriptor_validation(kw, code):
    lib = P.load()
    d, keep = _desc(**kw)
    n = C.c_size_t()
    assert lib.dcp_varlen_attn_fwd_workspace_size(C.byref(d), C.byref(n)) == code
    assert lib.dcp_varlen_attn_bwd_workspace_size(C.byref(d), C.byref(n)) == code
    assert lib.dcp_last_error()


def test_pointer_workspace_and_device_errors():
    lib = P.load()
    d, keep = _desc([0, 37, 101], 101)
    n = C.c_size_t()
    assert lib.dcp_varlen_attn_fwd_workspace_size(C.byref(d), C.byref(n)) == 0 and n.value > 0
    fake = 1 << 20  # 16-byte aligned host address, never dereferenced
    # null / misaligned tensors
    assert lib.dcp_varlen_attn_fwd(C.byref(d), None, fake, fake, fake, fake, fake, n.value, None) == N.DCP_ERR_INVALID
    assert lib.dcp_varlen_attn_fwd(C.byref(d), fake + 2, fake, fake, fake, fake, fake, n.value, None) \
        == N.DCP_ERR_INVALID
    # workspace too small
    assert lib.dcp_varlen_attn_fwd(C.byref(d), fake, fake, fake, fake, fake, fake, n.value - 1, None) \
        == N.DCP_ERR_WORKSPACE
    assert "workspace" in P.last_error()
    nb = C.c_size_t()
    assert lib.dcp_varlen_attn_bwd_workspace_size(C.byref(d), C.byref(nb)) == 0
    assert nb.value >= 4 * 101 * 2  # rowsum(dO o O) per (row, head)
    assert lib.dcp_varlen_attn_bwd(C.byref(d), *([fake] * 9), fake, nb.value - 1, None) == N.DCP_ERR_WORKSPACE
    # valid arguments but no gfx950 device in this process
    import torch
    if not torch.cuda.is_available():
        assert lib.dcp_varlen_attn_fwd(C.byref(d), fake, fake, fake, fake, fake, fake, n.value, None) \
            == N.DCP_ERR_HIP
        cus, khz = C.c_int32(-1), C.c_int32(-1)
        assert lib.dcp_device_info(C.byref(cus), C.byref(khz)) == N.DCP_ERR_HIP and cus.value == -1
    assert lib.dcp_device_info(None, None) == N.DCP_ERR_INVALID


def test_profile_validation():
    lib = P.load()
    o = N.ProfileOpts(2, 128, 0, 0.0, 1, 3, 0, 0, 0, 0)
    n = C.c_size_t()
    assert lib.dcp_profile_workspace_size(1024, C.byref(o), C.byref(n)) == 0 and n.value > 8 * 1024 * 2 * 128 * 2
    bad = N.ProfileOpts(2, 80, 0, 0.0, 1, 3, 0, 0, 0, 0)
    assert lib.dcp_profile_workspace_size(1024, C.byref(bad), C.byref(n)) == N.DCP_ERR_UNSUPPORTED
    bad = N.ProfileOpts(2, 128, 0, 0.0, 1, 0, 0, 0, 0, 0)
    assert lib.dcp_profile_workspace_size(1024, C.byref(bad), C.byref(n)) == N.DCP_ERR_INVALID
    lens = np.array([64, 0], dtype=np.int64)
    rows = (N.CostRow * 2)()
    assert lib.dcp_profile_cost(lens.ctypes.data_as(C.POINTER(C.c_int64)), 2, C.byref(o), 1 << 20, n.value, None,
                                rows) == N.DCP_ERR_INVALID


def test_layer_validation():
    """Layer calls reject bad descriptors, pointers and workspaces on the host."""
    lib = P.load()
    fake = 1 << 20

    def layer_desc(cu, T, H, D, eps=1e-6):
        d, keep = _desc(cu, T, H=H, D=D)
        L = N.LayerDescC(C.pointer(d), eps)
        return L, (d, keep)

    s, f, b = C.c_size_t(), C.c_size_t(), C.c_size_t()
    L, keep = layer_desc([0, 30, 64], 64, 2, 64)
    assert lib.dcp_layer_sizes(C.byref(L), C.byref(s), C.byref(f), C.byref(b)) == 0
    assert s.value >= 30 * 128 * 64 and f.value > s.value and b.value > s.value
    # hidden = 64 * 128 = 8192 > 4096
    L2, keep2 = layer_desc([0, 64], 64, 64, 128)
    assert lib.dcp_layer_sizes(C.byref(L2), C.byref(s), C.byref(f), C.byref(b)) == N.DCP_ERR_UNSUPPORTED
    # rows outside every sequence
    L3, keep3 = layer_desc([0, 60], 64, 2, 64)
    assert lib.dcp_layer_sizes(C.byref(L3), C.byref(s), C.byref(f), C.byref(b)) == N.DCP_ERR_INVALID
    L4, keep4 = layer_desc([0, 64], 64, 2, 64, eps=-1.0)
    assert lib.dcp_layer_sizes(C.byref(L4), C.byref(s), C.byref(f), C.byref(b)) == N.DCP_ERR_INVALID
    # null weights, misaligned input, short workspace: rejected before any device work
    lib.dcp_layer_sizes(C.byref(L), C.byref(s), C.byref(f), C.byref(b))
    w = N.LayerWeightsC(*([fake] * 8))
    w_null = N.LayerWeightsC(*([fake] * 7 + [None]))
    assert lib.dcp_layer_fwd(C.byref(L), C.byref(w_null), fake, fake, None, fake, f.value, None) == N.DCP_ERR_INVALID
    assert lib.dcp_layer_fwd(C.byref(L), C.byref(w), fake + 8, fake, None, fake, f.value, None) == N.DCP_ERR_INVALID
    assert lib.dcp_layer_fwd(C.byref(L), C.byref(w), fake, fake, None, fake, f.value - 1, None) == N.DCP_ERR_WORKSPACE
    assert lib.dcp_layer_bwd(C.byref(L), C.byref(w), fake, fake, fake, C.byref(w), None, fake, b.value - 1, None) \
        == N.DCP_ERR_WORKSPACE


# ---------------------------------------------------------------------------
# the Python binding checks what the C ABI cannot see behind raw pointers

def _bf(*shape):
    import torch
    return torch.zeros(shape, dtype=torch.bfloat16)


def test_binding_rejects_mismatched_tensors_before_any_call():
    import torch
    q = _bf(16, 2, 64)
    cu = [0, 16]
    cases = [
        dict(k=_bf(8, 2, 64)),                         # shorter k: the kernels would read past it
        dict(v=_bf(16, 2, 72)),
        dict(k=torch.zeros(16, 2, 64, dtype=torch.float16)),
        dict(v=_bf(16, 64, 2).transpose(1, 2)),        # non-contiguous
        dict(out=_bf(16, 1, 64)),
        dict(lse=torch.zeros(16, 2, dtype=torch.float32)),   # [T, H] instead of [H, T]
        dict(lse=torch.zeros(2, 16, dtype=torch.bfloat16)),
    ]
    for kw in cases:
        args = dict(k=_bf(16, 2, 64), v=_bf(16, 2, 64))
        args.update(kw)
        with pytest.raises(ValueError) as e:
            P.varlen_attn_fwd(q, args.pop("k"), args.pop("v"), cu, 0.125, **args)
        assert "device" not in str(e.value), kw
    bwd_cases = [dict(dout=_bf(16, 2, 32)), dict(o=_bf(15, 2, 64)), dict(dq=_bf(16, 2, 64)[:, :1]),
                 dict(dk=_bf(17, 2, 64)), dict(lse=torch.zeros(2, 15, dtype=torch.float32))]
    for kw in bwd_cases:
        args = dict(dout=_bf(16, 2, 64), o=_bf(16, 2, 64), lse=torch.zeros(2, 16, dtype=torch.float32))
        args.update(kw)
        with pytest.raises(ValueError) as e:
            P.varlen_attn_bwd(args.pop("dout"), args.pop("o"), args.pop("lse"), q, _bf(16, 2, 64), _bf(16, 2, 64),
                              cu, 0.125, **args)
        assert "device" not in str(e.value), kw
    # well-formed host tensors are refused for their device, still before any call
    with pytest.raises(ValueError, match="device"):
        P.varlen_attn_fwd(q, _bf(16, 2, 64), _bf(16, 2, 64), cu, 0.125)


@pytest.mark.parametrize("cu", [[0, 1 << 31], [0, -1, 4], [0.5, 4], [[0, 4]]])
def test_binding_rejects_cu_seqlens_outside_int32(cu):
    from paper_2608_07524_amd._native import _host_cu
    with pytest.raises(ValueError):
        _host_cu(cu)


def test_batch_handle_on_the_host():
    """dcp_batch_create validates like the per-call API and sizes its buffer
    (constants, three lists, the backward's 8*H*T bytes of scratch); a call
    on a buffer that was never uploaded is refused before any device work."""
    lib = P.load()
    h = C.c_void_p()
    d, keep = _desc([0, 5, 3], 5)
    assert lib.dcp_batch_create(C.byref(d), C.byref(h)) == N.DCP_ERR_INVALID and not h.value
    d, keep = _desc([0, 300, 1000], 1000, H=3, D=72, causal=1)
    assert lib.dcp_batch_create(C.byref(d), C.byref(h)) == N.DCP_OK and h.value
    n = C.c_size_t()
    assert lib.dcp_batch_workspace_size(h, C.byref(n)) == N.DCP_OK
    assert n.value >= 256 + 8 * 3 * 1000 and n.value % 256 == 0
    assert lib.dcp_batch_fwd(h, 16, 16, 16, 16, 16, None, 0, None) == N.DCP_ERR_WORKSPACE
    assert lib.dcp_batch_fwd(h, 16, 16, 16, 16, 16, 4096, n.value, None) == N.DCP_ERR_INVALID
    assert "dcp_batch_upload" in N.last_error()
    assert lib.dcp_batch_bwd(h, 16, 16, 16, 16, 16, 16, 16, 16, 16, 4096, n.value, None) == N.DCP_ERR_INVALID
    assert lib.dcp_batch_upload(h, 4096 + 16, n.value, None) == N.DCP_ERR_INVALID  # alignment
    lib.dcp_batch_destroy(h)
    lib.dcp_batch_destroy(None)


def test_noalloc_forward_rejects_oversize_lists_on_the_host():
    """dcp_varlen_attn_fwd_noalloc refuses a batch whose tile list exceeds
    its fixed 8 MiB scratch before any device call (65,535 heads x 16 tiles
    of 256 rows = 1,048,560 tiles x 16 bytes)."""
    lib = P.load()
    d, keep = _desc([0, 4096], 4096, H=65535, D=128)
    st = lib.dcp_varlen_attn_fwd_noalloc(C.byref(d), 16, 16, 16, 16, 16, None)
    assert st == N.DCP_ERR_WORKSPACE and "8388608" in N.last_error()
    d, keep = _desc([0, 5, 3], 5)
    assert lib.dcp_varlen_attn_fwd_noalloc(C.byref(d), 16, 16, 16, 16, 16, None) == N.DCP_ERR_INVALID
    d, keep = _desc([0, 5], 5)
    assert lib.dcp_varlen_attn_fwd_noalloc(C.byref(d), None, 16, 16, 16, 16, None) == N.DCP_ERR_INVALID
