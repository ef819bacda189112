"""The no-allocation forward (dcp_varlen_attn_fwd_noalloc, scratch in the
library's fixed device array) against dcp_varlen_attn_fwd (caller
workspace), called through the C ABI: bitwise-equal O and LSE on two calls in
a row, the second with a smaller batch (the array keeps the first call's
contents, which the second must not depend on)."""

import ctypes as C
import math

import numpy as np
import pytest

from paper_2608_07524_amd import inputs as I

from gpu_util import to_bits, to_device

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    t = pytest.importorskip("torch")
    if not t.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2608_07524_amd as P
    P.load()
    return t


def _desc(cu, T, H, D, causal):
    from paper_2608_07524_amd import _native as N
    cu = np.ascontiguousarray(cu, dtype=np.int32)
    return N.AttnDesc(cu.size - 1, cu.ctypes.data_as(C.POINTER(C.c_int32)), T, H, D, 1.0 / math.sqrt(D),
                      int(causal)), cu


def _both(torch, lengths, H, D, causal, seed):
    from paper_2608_07524_amd import _native as N
    lib = N.load()
    cu = I.cu_from_lengths(lengths)
    T = int(cu[-1])
    bits = I.tensors(np.random.default_rng(seed), T, H, D, n=3)
    q, k, v = (to_device(torch, b) for b in bits)
    d, keep = _desc(cu, T, H, D, causal)
    stream = C.c_void_p(torch.cuda.current_stream().cuda_stream)
    n = C.c_size_t()
    assert lib.dcp_varlen_attn_fwd_workspace_size(C.byref(d), C.byref(n)) == 0
    ws = torch.empty(max(1, n.value), dtype=torch.uint8, device="cuda")
    o_ref, o = torch.full_like(q, 7.0), torch.full_like(q, -7.0)
    l_ref = torch.full((H, T), 3.0, dtype=torch.float32, device="cuda")
    l = torch.full((H, T), -3.0, dtype=torch.float32, device="cuda")
    assert lib.dcp_varlen_attn_fwd(C.byref(d), q.data_ptr(), k.data_ptr(), v.data_ptr(), o_ref.data_ptr(),
                                   l_ref.data_ptr(), ws.data_ptr(), ws.numel(), stream) == 0, N.last_error()
    assert lib.dcp_varlen_attn_fwd_noalloc(C.byref(d), q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(),
                                           l.data_ptr(), stream) == 0, N.last_error()
    torch.cuda.synchronize()
    rows = int(cu[-1])
    assert np.array_equal(to_bits(o)[:rows], to_bits(o_ref)[:rows])
    assert np.array_equal(l.cpu().numpy()[:, :rows], l_ref.cpu().numpy()[:, :rows])
    print(f"no-alloc forward: {len(lengths)} sequences, {T} tokens, H{H} D{D} causal={causal}: bitwise equal",
          flush=True)


def test_noalloc_forward_matches_workspace_forward_twice(torch):
    # a large pack (tiles and packed windows), then a smaller one
    _both(torch, [5, 17, 40, 3, 700, 60, 60, 1, 0, 9, 127, 2049, 300, 4096], 8, 128, True, 1)
    _both(torch, [300, 40, 3, 1], 2, 72, False, 2)
