// Varlen attention backward on CDNA4 for the loss <dO, O>.
//
// Three launches:
//   1. bwd_pre:    Delta = rowsum(dO o O) per (row, head) in fp32 and the
//                  fp32 dQ accumulator zeroed (rows of sequences only).
//   2. bwd_main:   one workgroup per (key tile of kBwdBN rows, head); each of
//                  the four wavefronts keeps 32 keys' K and V fragments and
//                  their dK, dV accumulators in registers and walks the
//                  query tiles of the same sequence (only those on or below
//                  the diagonal when causal):
//                    S  = Q K^T,  dP = dO V^T        (A from LDS, B in regs)
//                    P  = exp2(S*scale*log2e - LSE*log2e)   (recomputed)
//                    dS = P o (dP - Delta)
//                    dV += P^T dO,  dK += dS^T Q      (B via transposing
//                                                      LDS reads)
//                  dS is staged in LDS; the workgroup then forms
//                  dQ_tile = dS K over all its keys and adds it to the fp32
//                  accumulator with one atomic per element.
//   3. bwd_post:   dQ = bf16(scale * accumulator).
// In the S / dP accumulators a lane holds one key and 16 queries, which is
// exactly the A-operand layout P^T and dS^T need for dV and dK.
#include "attn_common.h"
#include "attn_launch.h"

namespace dcp {
namespace {

// ---------------------------------------------------------------------------
// 1. Delta = rowsum(dO o O); zero the dQ accumulator.
// 16 lanes per (row, head); lane c covers elements 8c .. 8c+7.
template <int D>
__global__ __launch_bounds__(256) void bwd_pre_kernel(const __bf16* __restrict__ dout, const __bf16* __restrict__ o,
                                                      float* __restrict__ delta, float* __restrict__ dq_acc,
                                                      int rows_end, int H, int T) {
  constexpr int CPR = D / 8;
  const int64_t pair = (int64_t(blockIdx.x) * blockDim.x + threadIdx.x) >> 4;
  const int c = threadIdx.x & 15;
  const int64_t n_pairs = int64_t(rows_end) * H;
  float part = 0.f;
  if (pair < n_pairs && c < CPR) {
    const int64_t off = pair * D + 8 * c;
    const bf16x8 a = *reinterpret_cast<const bf16x8*>(dout + off);
    const bf16x8 b = *reinterpret_cast<const bf16x8*>(o + off);
#pragma unroll
    for (int e = 0; e < 8; ++e) part = fmaf(float(a[e]), float(b[e]), part);
    *reinterpret_cast<f32x4*>(dq_acc + off) = f32x4{};
    *reinterpret_cast<f32x4*>(dq_acc + off + 4) = f32x4{};
  }
  part += __shfl_xor(part, 8, 16);
  part += __shfl_xor(part, 4, 16);
  part += __shfl_xor(part, 2, 16);
  part += __shfl_xor(part, 1, 16);
  if (pair < n_pairs && c == 0) {
    const int64_t row = pair / H;
    const int hh = int(pair % H);
    delta[int64_t(hh) * T + row] = part;
  }
}

// ---------------------------------------------------------------------------
// 3. dQ = bf16(scale * accumulator), 8 elements per thread.
__global__ __launch_bounds__(256) void bwd_post_kernel(const float* __restrict__ dq_acc, __bf16* __restrict__ dq,
                                                       int64_t n8, float scale) {
  const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i >= n8) return;
  const f32x4 a = *reinterpret_cast<const f32x4*>(dq_acc + 8 * i);
  const f32x4 b = *reinterpret_cast<const f32x4*>(dq_acc + 8 * i + 4);
  bf16x8 w;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    w[e] = __bf16(a[e] * scale);
    w[4 + e] = __bf16(b[e] * scale);
  }
  *reinterpret_cast<bf16x8*>(dq + 8 * i) = w;
}

// ---------------------------------------------------------------------------
// 2. Main backward kernel.
template <int D, bool CAUSAL>
__global__ __launch_bounds__(256) void attn_bwd_kernel(const __bf16* __restrict__ q, const __bf16* __restrict__ k,
                                                       const __bf16* __restrict__ v,
                                                       const __bf16* __restrict__ dout,
                                                       const float* __restrict__ lse,
                                                       const float* __restrict__ delta,
                                                       float* __restrict__ dq_acc, __bf16* __restrict__ dk,
                                                       __bf16* __restrict__ dv,
                                                       const WorkUnit* __restrict__ units, int H, int T,
                                                       float scale, float scale_log2) {
  constexpr int DP = (D + 15) / 16 * 16;
  constexpr int NKD = DP / 16;
  constexpr int NDB = (D + 31) / 32;
  constexpr int BN = kBwdBN;  // keys per workgroup (32 per wavefront)
  constexpr int BM = kBwdBM;  // queries per step
  constexpr int KSTR = NDB * 32 + 16;
  constexpr int QW = (DP + 8 > NDB * 32 + 8) ? DP + 8 : NDB * 32 + 8;
  constexpr int QSTR = (QW % 16 == 8) ? QW : QW + 8;  // keeps the row stride an odd multiple of 16 bytes
  constexpr int DSTR = BM + 8;
  constexpr int CPR = D / 8;
  constexpr int NCHQ = BM * CPR;  // 16-byte chunks per Q (or dO) tile
  constexpr int CPTQ = (NCHQ + 255) / 256;
  constexpr int NCHK = BN * CPR;
  constexpr int CPTK = (NCHK + 255) / 256;

  __shared__ __attribute__((aligned(16))) __bf16 Ks[BN * KSTR];
  __shared__ __attribute__((aligned(16))) __bf16 Qs[BM * QSTR];
  __shared__ __attribute__((aligned(16))) __bf16 dOs[BM * QSTR];
  __shared__ __attribute__((aligned(16))) __bf16 dSs[BN * DSTR];
  __shared__ __attribute__((aligned(16))) float lse_s[BM];
  __shared__ __attribute__((aligned(16))) float dlt_s[BM];

  const WorkUnit u = units[blockIdx.x];
  const int h = blockIdx.y;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int g = lane >> 5;
  const int j = lane & 31;
  const int64_t ts = int64_t(H) * D;
  const int seqlen = u.seqlen;
  const int key_t0 = u.row0 - u.seq0;  // first key of the workgroup, sequence-relative

  const __bf16* qh = q + int64_t(u.seq0) * ts + int64_t(h) * D;
  const __bf16* kh = k + int64_t(u.seq0) * ts + int64_t(h) * D;
  const __bf16* vh = v + int64_t(u.seq0) * ts + int64_t(h) * D;
  const __bf16* doh = dout + int64_t(u.seq0) * ts + int64_t(h) * D;
  const float* lseh = lse + int64_t(h) * T + u.seq0;
  const float* dlth = delta + int64_t(h) * T + u.seq0;
  float* dqh = dq_acc + int64_t(u.seq0) * ts + int64_t(h) * D;

  // Zero pad columns (tile loads never write them).
  for (int i = tid; i < BN * (KSTR - D); i += 256) Ks[(i / (KSTR - D)) * KSTR + D + i % (KSTR - D)] = __bf16(0.f);
  for (int i = tid; i < BM * (QSTR - D); i += 256) {
    Qs[(i / (QSTR - D)) * QSTR + D + i % (QSTR - D)] = __bf16(0.f);
    dOs[(i / (QSTR - D)) * QSTR + D + i % (QSTR - D)] = __bf16(0.f);
  }
  // K tile -> LDS (rows past the sequence end are zero).
#pragma unroll
  for (int c = 0; c < CPTK; ++c) {
    const int ch = tid + 256 * c;
    if (NCHK % 256 == 0 || ch < NCHK) {
      const int r = ch / CPR, cc = ch % CPR;
      u32x4 val = u32x4{0, 0, 0, 0};
      if (r < u.rows) val = *reinterpret_cast<const u32x4*>(kh + int64_t(key_t0 + r) * ts + cc * 8);
      *reinterpret_cast<u32x4*>(&Ks[r * KSTR + cc * 8]) = val;
    }
  }
  // V fragments (B operand of dP = dO V^T): lane (g, j) holds key j of this
  // wavefront, columns 16*kd + 8*g .. +7.
  const int my_key = 32 * wave + j;  // tile-relative
  bf16x8 vf[NKD];
#pragma unroll
  for (int kd = 0; kd < NKD; ++kd) {
    const int col = 16 * kd + 8 * g;
    if (my_key < u.rows && col < D) {
      vf[kd] = *reinterpret_cast<const bf16x8*>(vh + int64_t(key_t0 + my_key) * ts + col);
    } else {
      vf[kd] = bf16x8{};
    }
  }

  const int q_begin = CAUSAL ? (key_t0 / BM) * BM : 0;
  const int n_qt = (seqlen - q_begin + BM - 1) / BM;

  u32x4 qreg[CPTQ], doreg[CPTQ];
  float lse_reg = INFINITY, dlt_reg = 0.f;
  auto load_q_tile = [&](int q0) {
#pragma unroll
    for (int c = 0; c < CPTQ; ++c) {
      const int ch = tid + 256 * c;
      if (NCHQ % 256 == 0 || ch < NCHQ) {
        const int r = ch / CPR, cc = ch % CPR;
        if (q0 + r < seqlen) {
          qreg[c] = *reinterpret_cast<const u32x4*>(qh + int64_t(q0 + r) * ts + cc * 8);
          doreg[c] = *reinterpret_cast<const u32x4*>(doh + int64_t(q0 + r) * ts + cc * 8);
        } else {
          qreg[c] = u32x4{0, 0, 0, 0};
          doreg[c] = u32x4{0, 0, 0, 0};
        }
      }
    }
    if (tid < BM) {
      // A query past the sequence end gets LSE = +inf, so its P is exactly 0.
      const bool ok = q0 + tid < seqlen;
      lse_reg = ok ? lseh[q0 + tid] * kLog2e : INFINITY;
      dlt_reg = ok ? dlth[q0 + tid] : 0.f;
    }
  };
  auto store_q_tile = [&]() {
#pragma unroll
    for (int c = 0; c < CPTQ; ++c) {
      const int ch = tid + 256 * c;
      if (NCHQ % 256 == 0 || ch < NCHQ) {
        const int r = ch / CPR, cc = ch % CPR;
        *reinterpret_cast<u32x4*>(&Qs[r * QSTR + cc * 8]) = qreg[c];
        *reinterpret_cast<u32x4*>(&dOs[r * QSTR + cc * 8]) = doreg[c];
      }
    }
    if (tid < BM) {
      lse_s[tid] = lse_reg;
      dlt_s[tid] = dlt_reg;
    }
  };

  f32x16 dk_acc[NDB], dv_acc[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) {
    dk_acc[db] = f32x16{};
    dv_acc[db] = f32x16{};
  }

  if (n_qt > 0) load_q_tile(q_begin);
  __syncthreads();  // K tile and pads visible
  // K fragments (B operand of S = Q K^T), same layout as vf.
  bf16x8 kf[NKD];
#pragma unroll
  for (int kd = 0; kd < NKD; ++kd) kf[kd] = lds_read_b128(&Ks[my_key * KSTR + 16 * kd + 8 * g]);

  const int tr_row = (lane & 15) >> 2;
  const int tr_col = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
  const int key_seq = key_t0 + my_key;  // this lane's key, sequence-relative
  const bool key_ok = my_key < u.rows;

  for (int it = 0; it < n_qt; ++it) {
    const int q0 = q_begin + it * BM;
    store_q_tile();
    __syncthreads();
    if (it + 1 < n_qt) load_q_tile(q0 + BM);

#pragma unroll
    for (int qb = 0; qb < BM / 32; ++qb) {
      f32x16 s = f32x16{}, dp = f32x16{};
#pragma unroll
      for (int kd = 0; kd < NKD; ++kd) {
        const bf16x8 aq = lds_read_b128(&Qs[(32 * qb + j) * QSTR + 16 * kd + 8 * g]);
        s = mfma32(aq, kf[kd], s);
        const bf16x8 ado = lds_read_b128(&dOs[(32 * qb + j) * QSTR + 16 * kd + 8 * g]);
        dp = mfma32(ado, vf[kd], dp);
      }
      // Row statistics for the 16 queries this lane holds: 32qb + 8b + 4g + c.
      float pv[16], dsv[16];
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        const f32x4 l4 = *reinterpret_cast<const f32x4*>(&lse_s[32 * qb + 8 * b + 4 * g]);
        const f32x4 d4 = *reinterpret_cast<const f32x4*>(&dlt_s[32 * qb + 8 * b + 4 * g]);
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          const int r = 4 * b + c;
          float p = exp2f(fmaf(s[r], scale_log2, -l4[c]));
          if (CAUSAL) {
            const int qi = q0 + 32 * qb + 8 * b + 4 * g + c;
            if (key_seq > qi) p = 0.f;
          }
          if (!key_ok) p = 0.f;
          pv[r] = p;
          dsv[r] = p * (dp[r] - d4[c]);
        }
      }
      bf16x8 pa[2], da[2];
#pragma unroll
      for (int hh = 0; hh < 2; ++hh)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          pa[hh][e] = __bf16(pv[8 * hh + e]);
          da[hh][e] = __bf16(dsv[8 * hh + e]);
        }
      // dV += P^T dO and dK += dS^T Q; B = rows (queries) x columns (d)
      // fetched column-wise with transposing reads.
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
          const int off = (32 * qb + 16 * hh + 4 * g + tr_row) * QSTR + 32 * db + tr_col;
          const bf16x8 bdo = cat(lds_read_tr(&dOs[off]), lds_read_tr(&dOs[off + 8 * QSTR]));
          dv_acc[db] = mfma32(pa[hh], bdo, dv_acc[db]);
          const bf16x8 bq = cat(lds_read_tr(&Qs[off]), lds_read_tr(&Qs[off + 8 * QSTR]));
          dk_acc[db] = mfma32(da[hh], bq, dk_acc[db]);
        }
      }
      // Stage dS as [key][query] for the dQ product.
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        bf16x4 w;
#pragma unroll
        for (int c = 0; c < 4; ++c) w[c] = da[b >> 1][4 * (b & 1) + c];
        *reinterpret_cast<bf16x4*>(&dSs[my_key * DSTR + 32 * qb + 8 * b + 4 * g]) = w;
      }
    }
    __syncthreads();

    // dQ_tile = dS K over the workgroup's BN keys; (query block, d block)
    // jobs are spread over the wavefronts.
    for (int job = wave; job < (BM / 32) * NDB; job += 4) {
      const int qb = job / NDB, db = job % NDB;
      f32x16 acc = f32x16{};
#pragma unroll
      for (int kk = 0; kk < BN / 16; ++kk) {
        const int arow = 16 * kk + 4 * g + tr_row;
        const __bf16* pa_ = &dSs[arow * DSTR + 32 * qb + tr_col];
        const bf16x8 a = cat(lds_read_tr(pa_), lds_read_tr(pa_ + 8 * DSTR));
        const __bf16* pb_ = &Ks[arow * KSTR + 32 * db + tr_col];
        const bf16x8 b = cat(lds_read_tr(pb_), lds_read_tr(pb_ + 8 * KSTR));
        acc = mfma32(a, b, acc);
      }
      const int d = 32 * db + j;
      if (d < D) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int qi = q0 + 32 * qb + 8 * (r >> 2) + 4 * g + (r & 3);
          if (qi < seqlen) atomic_add_f32(dqh + int64_t(qi) * ts + d, acc[r]);
        }
      }
    }
    __syncthreads();
  }

  // Epilogue: lane (g, j) holds column 32*db + j of keys 8*(r/4) + 4*g + r%4.
#pragma unroll
  for (int db = 0; db < NDB; ++db) {
    const int d = 32 * db + j;
    if (d < D) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = 32 * wave + 8 * (r >> 2) + 4 * g + (r & 3);
        if (key < u.rows) {
          const int64_t off = int64_t(u.row0 + key) * ts + int64_t(h) * D + d;
          dk[off] = __bf16(dk_acc[db][r] * scale);
          dv[off] = __bf16(dv_acc[db][r]);
        }
      }
    }
  }
}

template <int D, bool CAUSAL>
hipError_t launch_bwd_t(const BwdArgs& a) {
  const int64_t n_pairs = int64_t(a.rows_end) * a.n_heads;
  if (n_pairs > 0) {
    const int64_t blocks = (n_pairs * 16 + 255) / 256;
    hipLaunchKernelGGL((bwd_pre_kernel<D>), dim3(unsigned(blocks)), dim3(256), 0, a.stream,
                       static_cast<const __bf16*>(a.dout), static_cast<const __bf16*>(a.o), a.delta, a.dq_acc,
                       a.rows_end, a.n_heads, a.total_tokens);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (a.n_units > 0) {
    hipLaunchKernelGGL((attn_bwd_kernel<D, CAUSAL>), dim3(a.n_units, a.n_heads), dim3(256), 0, a.stream,
                       static_cast<const __bf16*>(a.q), static_cast<const __bf16*>(a.k),
                       static_cast<const __bf16*>(a.v), static_cast<const __bf16*>(a.dout), a.lse, a.delta,
                       a.dq_acc, static_cast<__bf16*>(a.dk), static_cast<__bf16*>(a.dv),
                       static_cast<const WorkUnit*>(a.units), a.n_heads, a.total_tokens, a.scale,
                       a.scale * kLog2e);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  const int64_t n8 = n_pairs * D / 8;
  if (n8 > 0) {
    hipLaunchKernelGGL(bwd_post_kernel, dim3(unsigned((n8 + 255) / 256)), dim3(256), 0, a.stream, a.dq_acc,
                       static_cast<__bf16*>(a.dq), n8, a.scale);
    return hipGetLastError();
  }
  return hipSuccess;
}

// Deterministic fill for profiling inputs: a 32-bit integer hash mapped to
// [-1, 1) and rounded to bf16.
__global__ void fill_bf16_kernel(__bf16* p, int64_t n, uint32_t seed) {
  const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i >= n) return;
  uint32_t x = uint32_t(i) * 0x9E3779B1u ^ seed ^ uint32_t(i >> 32) * 0x85EBCA77u;
  x ^= x >> 16;
  x *= 0x7FEB352Du;
  x ^= x >> 15;
  x *= 0x846CA68Bu;
  x ^= x >> 16;
  p[i] = __bf16(float(int32_t(x)) * (1.0f / 2147483648.0f));
}

}  // namespace

hipError_t launch_bwd(const BwdArgs& a) {
  switch (a.head_dim) {
    case 64: return a.causal ? launch_bwd_t<64, true>(a) : launch_bwd_t<64, false>(a);
    case 72: return a.causal ? launch_bwd_t<72, true>(a) : launch_bwd_t<72, false>(a);
    case 128: return a.causal ? launch_bwd_t<128, true>(a) : launch_bwd_t<128, false>(a);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_fill_bf16(void* p, int64_t n, uint32_t seed, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(fill_bf16_kernel, dim3(unsigned((n + 255) / 256)), dim3(256), 0, stream,
                     static_cast<__bf16*>(p), n, seed);
  return hipGetLastError();
}

}  // namespace dcp
