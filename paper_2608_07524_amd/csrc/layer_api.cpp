// C ABI of one transformer layer around the packed attention kernels: the
// unit whose forward time t_f, backward time t_b and stashed activations m
// the profiling of Sec. 3.5 measures, and whose forward is run again in the
// backward when the layer is recomputed (Eqs. (4)-(6)).
//
// Pre-norm block, bf16 storage, fp32 accumulation:
//   y1 = RMSNorm(x; g1), q = y1 Wq, k = y1 Wk, v = y1 Wv (each [T, H*D]),
//   o  = attention(q, k, v) per sequence (the HIP kernels of this library),
//   h  = x + o Wo,  y2 = RMSNorm(h; g2),  u = y2 Wup ([T, 4 hidden]),
//   a  = GELU(u),   out = h + a Wdown.
// GEMMs are plain library GEMMs (rocBLAS, bf16 inputs, fp32 compute); the
// norms and the activation are the kernels of layer.hip.  A forward with a
// stash keeps every activation the backward needs; with no stash it keeps
// nothing and the backward runs the forward again first (recomputation).
#include <hip/hip_runtime.h>
#include <rocblas/rocblas.h>

#include <cmath>
#include <cstdint>
#include <initializer_list>

#include "dcp_internal.h"
#include "layer_launch.h"

namespace dcp {
namespace {

constexpr size_t kAlign = 256;
inline size_t up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }
constexpr size_t kGemmWorkspace = size_t(64) << 20;  // rocBLAS scratch, carved from the caller's workspace

constexpr int kMaxHidden = 4096;

struct Dims {
  int64_t T, H, D, h;
};

// Activations kept from forward to backward (byte offsets).
struct Stash {
  size_t rstd1, y1, q, k, v, o, lse, hres, rstd2, y2, u, a, total;
};
Stash stash_layout(const Dims& d) {
  Stash s{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off += up(bytes);
    return at;
  };
  const size_t Th = size_t(d.T) * size_t(d.h);
  s.rstd1 = take(4 * size_t(d.T));
  s.y1 = take(2 * Th);
  s.q = take(2 * Th);
  s.k = take(2 * Th);
  s.v = take(2 * Th);
  s.o = take(2 * Th);
  s.lse = take(4 * size_t(d.H) * size_t(d.T));
  s.hres = take(2 * Th);
  s.rstd2 = take(4 * size_t(d.T));
  s.y2 = take(2 * Th);
  s.u = take(8 * Th);
  s.a = take(8 * Th);
  s.total = off;
  return s;
}

// Workspaces: rocBLAS scratch | attention workspace(s) | a stash (used when
// the caller passes none) | backward temporaries.
struct FwdWs {
  size_t gemm, attn, stash, total;
};
struct BwdWs {
  size_t gemm, attn_f, attn_b, stash, da, dy2, dh, dout_recomputed, dq, dk, dv, dy1, partial, total;
};

int dims_of(const dcp_layer_desc* L, Dims* d) {
  if (!L || !L->attn) return fail(DCP_ERR_INVALID, "layer desc or its attention desc is null");
  size_t n = 0;
  int st = dcp_varlen_attn_fwd_workspace_size(L->attn, &n);  // validates the attention desc
  if (st) return st;
  const dcp_attn_desc* a = L->attn;
  if (a->cu_seqlens_host[a->n_seqs] != a->total_tokens)
    return fail(DCP_ERR_INVALID, "a layer processes every row: cu_seqlens[n] must equal total_tokens");
  if (!(std::isfinite(L->eps) && L->eps >= 0.f)) return fail(DCP_ERR_INVALID, "eps must be finite and >= 0");
  d->T = a->total_tokens;
  d->H = a->n_heads;
  d->D = a->head_dim;
  d->h = d->H * d->D;
  // the RMSNorm backward keeps four fp32 rows of gain partials in LDS (<= 64 KB)
  if (d->h > kMaxHidden) return fail(DCP_ERR_UNSUPPORTED, "hidden size %lld exceeds %d", (long long)d->h, kMaxHidden);
  return DCP_OK;
}

int fwd_ws(const dcp_layer_desc* L, const Dims& d, FwdWs* w) {
  size_t na = 0;
  int st = dcp_varlen_attn_fwd_workspace_size(L->attn, &na);
  if (st) return st;
  w->gemm = 0;
  w->attn = up(kGemmWorkspace);
  w->stash = w->attn + up(na);
  w->total = w->stash + stash_layout(d).total;
  return DCP_OK;
}

int bwd_ws(const dcp_layer_desc* L, const Dims& d, BwdWs* w) {
  size_t na = 0, nb = 0;
  int st = dcp_varlen_attn_fwd_workspace_size(L->attn, &na);
  if (st) return st;
  st = dcp_varlen_attn_bwd_workspace_size(L->attn, &nb);
  if (st) return st;
  const size_t Th = size_t(d.T) * size_t(d.h);
  size_t off = up(kGemmWorkspace);
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off += up(bytes);
    return at;
  };
  w->gemm = 0;
  w->attn_f = take(na);
  w->attn_b = take(nb);
  w->stash = take(stash_layout(d).total);
  w->da = take(8 * Th);  // dA, then dU in place
  w->dy2 = take(4 * Th);
  w->dh = take(2 * Th);
  w->dout_recomputed = take(2 * Th);
  w->dq = take(2 * Th);
  w->dk = take(2 * Th);
  w->dv = take(2 * Th);
  w->dy1 = take(4 * Th);
  w->partial = take(4 * size_t(rmsnorm_bwd_blocks(d.T)) * size_t(d.h));
  w->total = off;
  return DCP_OK;
}

// One rocBLAS handle per thread and device, on the call's stream, with its
// scratch in the caller's workspace.
int blas(hipStream_t stream, void* scratch, rocblas_handle* out) {
  struct Handle {
    int dev = -1;
    rocblas_handle h = nullptr;
    ~Handle() {
      if (h) rocblas_destroy_handle(h);
    }
  };
  thread_local Handle th;
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return fail(DCP_ERR_HIP, "no HIP device");
  if (th.h == nullptr || th.dev != dev) {
    if (th.h) rocblas_destroy_handle(th.h);
    th.h = nullptr;
    if (rocblas_create_handle(&th.h) != rocblas_status_success) return fail(DCP_ERR_HIP, "rocblas_create_handle failed");
    th.dev = dev;
    // no split-K atomics: every GEMM, hence every layer output, is bitwise reproducible
    if (rocblas_set_atomics_mode(th.h, rocblas_atomics_not_allowed) != rocblas_status_success)
      return fail(DCP_ERR_HIP, "rocblas_set_atomics_mode failed");
  }
  if (rocblas_set_stream(th.h, stream) != rocblas_status_success ||
      rocblas_set_workspace(th.h, scratch, kGemmWorkspace) != rocblas_status_success)
    return fail(DCP_ERR_HIP, "rocBLAS stream or workspace setup failed");
  *out = th.h;
  return DCP_OK;
}

// Row-major C[M, N] = op(A)[M, K] op(B)[K, N] + beta C, A and B bf16 (A
// stored [M, K], or [K, M] when ta; B stored [K, N], or [N, K] when tb),
// C bf16 or fp32; the result goes to Dst (C itself, or another buffer of
// C's layout and type).
int gemm(rocblas_handle hd, bool ta, bool tb, int64_t M, int64_t N, int64_t K, const void* A, const void* B,
         float beta, const void* C, void* Dst, bool c_f32) {
  // column-major view: C^T[N, M] = op(B)^T[N, K] op(A)^T[K, M]
  const float alpha = 1.f;
  const rocblas_datatype ct = c_f32 ? rocblas_datatype_f32_r : rocblas_datatype_bf16_r;
  const rocblas_status s = rocblas_gemm_ex(
      hd, tb ? rocblas_operation_transpose : rocblas_operation_none,
      ta ? rocblas_operation_transpose : rocblas_operation_none, rocblas_int(N), rocblas_int(M), rocblas_int(K), &alpha,
      B, rocblas_datatype_bf16_r, rocblas_int(tb ? K : N), A, rocblas_datatype_bf16_r, rocblas_int(ta ? M : K), &beta,
      C, ct, rocblas_int(N), Dst, ct, rocblas_int(N), rocblas_datatype_f32_r, rocblas_gemm_algo_standard, 0, 0);
  if (s != rocblas_status_success) return fail(DCP_ERR_HIP, "rocblas_gemm_ex failed (status %d)", int(s));
  return DCP_OK;
}

int check_ptrs(std::initializer_list<const void*> ps, const char* what) {
  for (const void* p : ps)
    if (!p || reinterpret_cast<uintptr_t>(p) % 16) return fail(DCP_ERR_INVALID, "%s: null or not 16-byte aligned", what);
  return DCP_OK;
}

inline char* at(void* base, size_t off) { return static_cast<char*>(base) + off; }

#define DCP_TRY(x)          \
  do {                      \
    int st_ = (x);          \
    if (st_) return st_;    \
  } while (0)
#define DCP_HIP(x)                                                                          \
  do {                                                                                      \
    hipError_t e_ = (x);                                                                    \
    if (e_ != hipSuccess) return fail(DCP_ERR_HIP, "layer kernel: %s", hipGetErrorString(e_)); \
  } while (0)

// The forward into stash buffers `s` (offsets from `sb`), output `out`.
int forward(const dcp_layer_desc* L, const Dims& d, const dcp_layer_weights* w, const void* x, void* out, void* sb,
            const Stash& s, void* attn_ws, size_t attn_ws_bytes, rocblas_handle hd, hipStream_t st) {
  const int64_t T = d.T, h = d.h;
  DCP_HIP(launch_rmsnorm_fwd(x, w->norm1, at(sb, s.y1), reinterpret_cast<float*>(at(sb, s.rstd1)), T, int(h), L->eps, st));
  DCP_TRY(gemm(hd, false, false, T, h, h, at(sb, s.y1), w->wq, 0.f, at(sb, s.q), at(sb, s.q), false));
  DCP_TRY(gemm(hd, false, false, T, h, h, at(sb, s.y1), w->wk, 0.f, at(sb, s.k), at(sb, s.k), false));
  DCP_TRY(gemm(hd, false, false, T, h, h, at(sb, s.y1), w->wv, 0.f, at(sb, s.v), at(sb, s.v), false));
  DCP_TRY(dcp_varlen_attn_fwd(L->attn, at(sb, s.q), at(sb, s.k), at(sb, s.v), at(sb, s.o),
                              reinterpret_cast<float*>(at(sb, s.lse)), attn_ws, attn_ws_bytes, st));
  DCP_TRY(gemm(hd, false, false, T, h, h, at(sb, s.o), w->wo, 1.f, x, at(sb, s.hres), false));
  DCP_HIP(launch_rmsnorm_fwd(at(sb, s.hres), w->norm2, at(sb, s.y2), reinterpret_cast<float*>(at(sb, s.rstd2)), T,
                             int(h), L->eps, st));
  DCP_TRY(gemm(hd, false, false, T, 4 * h, h, at(sb, s.y2), w->w_up, 0.f, at(sb, s.u), at(sb, s.u), false));
  DCP_HIP(launch_gelu_fwd(at(sb, s.u), at(sb, s.a), T * 4 * h, st));
  DCP_TRY(gemm(hd, false, false, T, h, 4 * h, at(sb, s.a), w->w_down, 1.f, at(sb, s.hres), out, false));
  return DCP_OK;
}

int check_weights(const dcp_layer_weights* w) {
  if (!w) return fail(DCP_ERR_INVALID, "weights are null");
  return check_ptrs({w->norm1, w->wq, w->wk, w->wv, w->wo, w->norm2, w->w_up, w->w_down}, "weights");
}

}  // namespace
}  // namespace dcp

using namespace dcp;

extern "C" int dcp_layer_sizes(const dcp_layer_desc* L, size_t* stash_bytes, size_t* fwd_workspace_bytes,
                               size_t* bwd_workspace_bytes) {
  clear_error();
  Dims d;
  DCP_TRY(dims_of(L, &d));
  FwdWs f;
  BwdWs b;
  DCP_TRY(fwd_ws(L, d, &f));
  DCP_TRY(bwd_ws(L, d, &b));
  if (stash_bytes) *stash_bytes = stash_layout(d).total;
  if (fwd_workspace_bytes) *fwd_workspace_bytes = f.total;
  if (bwd_workspace_bytes) *bwd_workspace_bytes = b.total;
  return DCP_OK;
}

extern "C" int dcp_layer_fwd(const dcp_layer_desc* L, const dcp_layer_weights* w, const void* x, void* out,
                             void* stash, void* workspace, size_t workspace_bytes, void* stream) {
  clear_error();
  Dims d;
  DCP_TRY(dims_of(L, &d));
  DCP_TRY(check_weights(w));
  DCP_TRY(check_ptrs({x, out}, "x and out"));
  FwdWs f;
  DCP_TRY(fwd_ws(L, d, &f));
  if (!workspace || workspace_bytes < f.total || reinterpret_cast<uintptr_t>(workspace) % kAlign)
    return fail(DCP_ERR_WORKSPACE, "layer forward workspace needs %zu bytes (256-byte aligned), got %zu", f.total,
                workspace_bytes);
  if (stash && reinterpret_cast<uintptr_t>(stash) % kAlign) return fail(DCP_ERR_INVALID, "stash must be 256-byte aligned");
  hipStream_t st = static_cast<hipStream_t>(stream);
  rocblas_handle hd;
  DCP_TRY(blas(st, at(workspace, f.gemm), &hd));
  void* sb = stash ? stash : at(workspace, f.stash);
  return forward(L, d, w, x, out, sb, stash_layout(d), at(workspace, f.attn), f.stash - f.attn, hd, st);
}

extern "C" int dcp_layer_bwd(const dcp_layer_desc* L, const dcp_layer_weights* w, const void* x, const void* dout,
                             void* dx, const dcp_layer_grads* g, void* stash, void* workspace, size_t workspace_bytes,
                             void* stream) {
  clear_error();
  Dims d;
  DCP_TRY(dims_of(L, &d));
  DCP_TRY(check_weights(w));
  DCP_TRY(check_ptrs({x, dout, dx}, "x, dout and dx"));
  if (!g) return fail(DCP_ERR_INVALID, "grads are null");
  DCP_TRY(check_ptrs({g->norm1, g->wq, g->wk, g->wv, g->wo, g->norm2, g->w_up, g->w_down}, "grads"));
  BwdWs b;
  DCP_TRY(bwd_ws(L, d, &b));
  if (!workspace || workspace_bytes < b.total || reinterpret_cast<uintptr_t>(workspace) % kAlign)
    return fail(DCP_ERR_WORKSPACE, "layer backward workspace needs %zu bytes (256-byte aligned), got %zu", b.total,
                workspace_bytes);
  if (stash && reinterpret_cast<uintptr_t>(stash) % kAlign) return fail(DCP_ERR_INVALID, "stash must be 256-byte aligned");
  hipStream_t st = static_cast<hipStream_t>(stream);
  rocblas_handle hd;
  DCP_TRY(blas(st, at(workspace, b.gemm), &hd));
  const Stash s = stash_layout(d);
  void* sb = stash;
  if (!sb) {  // recomputation: the forward again, its output discarded
    sb = at(workspace, b.stash);
    DCP_TRY(forward(L, d, w, x, at(workspace, b.dout_recomputed), sb, s, at(workspace, b.attn_f), b.attn_b - b.attn_f,
                    hd, st));
  }
  const int64_t T = d.T, h = d.h;
  float* partial = reinterpret_cast<float*>(at(workspace, b.partial));
  // MLP: dA = dout Wdown^T; dWdown += A^T dout; dU = dA * GELU'(U) (in place)
  DCP_TRY(gemm(hd, false, true, T, 4 * h, h, dout, w->w_down, 0.f, at(workspace, b.da), at(workspace, b.da), false));
  DCP_TRY(gemm(hd, true, false, 4 * h, h, T, at(sb, s.a), dout, 1.f, g->w_down, g->w_down, true));
  DCP_HIP(launch_gelu_bwd(at(sb, s.u), at(workspace, b.da), at(workspace, b.da), T * 4 * h, st));
  // dY2 = dU Wup^T (fp32); dWup += Y2^T dU; dH = dout + RMSNorm backward
  DCP_TRY(gemm(hd, false, true, T, h, 4 * h, at(workspace, b.da), w->w_up, 0.f, at(workspace, b.dy2),
               at(workspace, b.dy2), true));
  DCP_TRY(gemm(hd, true, false, h, 4 * h, T, at(sb, s.y2), at(workspace, b.da), 1.f, g->w_up, g->w_up, true));
  DCP_HIP(launch_rmsnorm_bwd(reinterpret_cast<float*>(at(workspace, b.dy2)), at(sb, s.hres), w->norm2,
                             reinterpret_cast<float*>(at(sb, s.rstd2)), dout, at(workspace, b.dh), partial, g->norm2, T,
                             int(h), st));
  // attention block: dO = dH Wo^T; dWo += O^T dH; attention backward
  void* dO = at(workspace, b.dy1);  // dY1 is not needed yet: its space holds dO (bf16) first
  DCP_TRY(gemm(hd, false, true, T, h, h, at(workspace, b.dh), w->wo, 0.f, dO, dO, false));
  DCP_TRY(gemm(hd, true, false, h, h, T, at(sb, s.o), at(workspace, b.dh), 1.f, g->wo, g->wo, true));
  DCP_TRY(dcp_varlen_attn_bwd(L->attn, dO, at(sb, s.o), reinterpret_cast<const float*>(at(sb, s.lse)), at(sb, s.q),
                              at(sb, s.k), at(sb, s.v), at(workspace, b.dq), at(workspace, b.dk), at(workspace, b.dv),
                              at(workspace, b.attn_b), b.stash - b.attn_b, st));
  // dY1 = dQ Wq^T + dK Wk^T + dV Wv^T (fp32); dW{q,k,v} += Y1^T d{Q,K,V}
  void* dY1 = at(workspace, b.dy1);
  DCP_TRY(gemm(hd, false, true, T, h, h, at(workspace, b.dq), w->wq, 0.f, dY1, dY1, true));
  DCP_TRY(gemm(hd, false, true, T, h, h, at(workspace, b.dk), w->wk, 1.f, dY1, dY1, true));
  DCP_TRY(gemm(hd, false, true, T, h, h, at(workspace, b.dv), w->wv, 1.f, dY1, dY1, true));
  DCP_TRY(gemm(hd, true, false, h, h, T, at(sb, s.y1), at(workspace, b.dq), 1.f, g->wq, g->wq, true));
  DCP_TRY(gemm(hd, true, false, h, h, T, at(sb, s.y1), at(workspace, b.dk), 1.f, g->wk, g->wk, true));
  DCP_TRY(gemm(hd, true, false, h, h, T, at(sb, s.y1), at(workspace, b.dv), 1.f, g->wv, g->wv, true));
  // dX = dH + RMSNorm backward of dY1
  DCP_HIP(launch_rmsnorm_bwd(reinterpret_cast<float*>(dY1), x, w->norm1, reinterpret_cast<float*>(at(sb, s.rstd1)),
                             at(workspace, b.dh), dx, partial, g->norm1, T, int(h), st));
  return DCP_OK;
}
