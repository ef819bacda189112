// Varlen attention forward on CDNA4: bf16 matrix-core products with an fp32
// online softmax (exact attention, as used for every run of the paper,
// Sec. 4.1; packed block-diagonal layout of Sec. 1).
//
// Work decomposition: one workgroup per (query tile, head).  A query tile
// never straddles two sequences, and the key loop runs over the tile's own
// sequence only, so no off-diagonal (cross-sequence) block is ever touched.
// Four wavefronts per workgroup, each owning 32*NQB query rows.
//
// Per key tile of BN = 64 keys (staged in LDS, next tile prefetched into
// registers while the current one is consumed):
//   S^T = K Q^T      A = K rows from LDS, B = Q rows kept in registers;
//                    each lane ends up holding one query and 16 keys.
//   m, l, P          row max: in-lane over 32 keys + one cross-half swap;
//                    P = exp2(S*scale*log2e - m) stays in registers.
//   O^T += V^T P^T   A = V^T via transposing LDS reads of the row-major V
//                    tile, B = P^T straight from the S^T accumulator layout.
// Epilogue: O = O^T / l (bf16), LSE = (m + log2 l) * ln 2.
#include "attn_common.h"
#include "attn_launch.h"

namespace dcp {
namespace {

constexpr int kFwdBN = 64;

template <int D, int NQB, bool CAUSAL>
__global__ __launch_bounds__(256) void attn_fwd_kernel(const __bf16* __restrict__ q, const __bf16* __restrict__ k,
                                                       const __bf16* __restrict__ v, __bf16* __restrict__ o,
                                                       float* __restrict__ lse, const WorkUnit* __restrict__ units,
                                                       int H, int T, float scale_log2) {
  constexpr int DP = (D + 15) / 16 * 16;  // contraction width (zero padded)
  constexpr int NKD = DP / 16;
  constexpr int NDB = (D + 31) / 32;  // 32-row blocks of O^T
  constexpr int BN = kFwdBN;
  constexpr int KSTR = DP + 8;         // K tile row stride (elements)
  constexpr int VSTR = NDB * 32 + 16;  // V tile row stride (elements)
  constexpr int QPW = 32 * NQB;
  constexpr int CPR = D / 8;  // 16-byte chunks per row
  constexpr int NCH = BN * CPR;
  constexpr int CPT = (NCH + 255) / 256;

  __shared__ __attribute__((aligned(16))) __bf16 Ks[BN * KSTR];
  __shared__ __attribute__((aligned(16))) __bf16 Vs[BN * VSTR];

  const WorkUnit u = units[blockIdx.x];
  const int h = blockIdx.y;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int g = lane >> 5;
  const int j = lane & 31;
  const int64_t ts = int64_t(H) * D;  // token stride

  const __bf16* qh = q + int64_t(u.seq0) * ts + int64_t(h) * D;
  const __bf16* kh = k + int64_t(u.seq0) * ts + int64_t(h) * D;
  const __bf16* vh = v + int64_t(u.seq0) * ts + int64_t(h) * D;

  // Pad columns are never written by tile loads: zero them once.
  for (int i = tid; i < BN * (KSTR - D); i += 256) Ks[(i / (KSTR - D)) * KSTR + D + i % (KSTR - D)] = __bf16(0.f);
  for (int i = tid; i < BN * (VSTR - D); i += 256) Vs[(i / (VSTR - D)) * VSTR + D + i % (VSTR - D)] = __bf16(0.f);

  const int tile_q0 = u.row0 - u.seq0;      // first query of the tile, sequence-relative
  const int wave_q0 = tile_q0 + wave * QPW;  // first query of this wave
  const int seqlen = u.seqlen;

  // Q fragments (B operand of S^T): lane (g, j) holds query j of each
  // 32-row block, columns 16*kd + 8*g .. +7.
  bf16x8 qf[NQB][NKD];
#pragma unroll
  for (int qb = 0; qb < NQB; ++qb) {
    const int qrel = wave * QPW + 32 * qb + j;  // row within the tile
#pragma unroll
    for (int kd = 0; kd < NKD; ++kd) {
      const int col = 16 * kd + 8 * g;
      if (qrel < u.rows && col < D) {
        qf[qb][kd] = *reinterpret_cast<const bf16x8*>(qh + int64_t(tile_q0 + qrel) * ts + col);
      } else {
        qf[qb][kd] = bf16x8{};
      }
    }
  }

  const int key_end = CAUSAL ? min(seqlen, tile_q0 + u.rows) : seqlen;
  const int n_tiles = (key_end + BN - 1) / BN;

  u32x4 kreg[CPT], vreg[CPT];
  auto load_tile = [&](int kt) {
#pragma unroll
    for (int c = 0; c < CPT; ++c) {
      const int ch = tid + 256 * c;
      if (NCH % 256 == 0 || ch < NCH) {
        const int r = ch / CPR, cc = ch % CPR;
        const int key = kt * BN + r;
        if (key < seqlen) {
          kreg[c] = *reinterpret_cast<const u32x4*>(kh + int64_t(key) * ts + cc * 8);
          vreg[c] = *reinterpret_cast<const u32x4*>(vh + int64_t(key) * ts + cc * 8);
        } else {
          kreg[c] = u32x4{0, 0, 0, 0};
          vreg[c] = u32x4{0, 0, 0, 0};
        }
      }
    }
  };
  auto store_tile = [&]() {
#pragma unroll
    for (int c = 0; c < CPT; ++c) {
      const int ch = tid + 256 * c;
      if (NCH % 256 == 0 || ch < NCH) {
        const int r = ch / CPR, cc = ch % CPR;
        *reinterpret_cast<u32x4*>(&Ks[r * KSTR + cc * 8]) = kreg[c];
        *reinterpret_cast<u32x4*>(&Vs[r * VSTR + cc * 8]) = vreg[c];
      }
    }
  };

  float m_run[NQB], l_run[NQB];
  f32x16 oacc[NQB][NDB];
#pragma unroll
  for (int qb = 0; qb < NQB; ++qb) {
    m_run[qb] = -INFINITY;
    l_run[qb] = 0.f;
#pragma unroll
    for (int db = 0; db < NDB; ++db) oacc[qb][db] = f32x16{};
  }

  if (n_tiles > 0) {
    load_tile(0);
    store_tile();
  }
  __syncthreads();

  const int wave_last_q = wave_q0 + QPW - 1;
  // transposing-read addressing (see lds_read_tr): row and column offsets
  const int tr_row = (lane & 15) >> 2;
  const int tr_col = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);

  for (int kt = 0; kt < n_tiles; ++kt) {
    if (kt + 1 < n_tiles) load_tile(kt + 1);
    const int k0 = kt * BN;
    const bool active = !CAUSAL || k0 <= wave_last_q;
    if (active) {
      f32x16 s[2][NQB];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int qb = 0; qb < NQB; ++qb) s[kb][qb] = f32x16{};
#pragma unroll
      for (int kd = 0; kd < NKD; ++kd) {
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
          const bf16x8 a = lds_read_b128(&Ks[(32 * kb + j) * KSTR + 16 * kd + 8 * g]);
#pragma unroll
          for (int qb = 0; qb < NQB; ++qb) s[kb][qb] = mfma32(a, qf[qb][kd], s[kb][qb]);
        }
      }
      const bool need_mask = (k0 + BN > seqlen) || (CAUSAL && k0 + BN - 1 > wave_q0);
      if (need_mask) {
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int qb = 0; qb < NQB; ++qb) {
            const int qi = wave_q0 + 32 * qb + j;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
              const int key = k0 + 32 * kb + 8 * (r >> 2) + 4 * g + (r & 3);
              if (key >= seqlen || (CAUSAL && key > qi)) s[kb][qb][r] = -INFINITY;
            }
          }
      }
      bf16x8 pb[2][2][NQB];
#pragma unroll
      for (int qb = 0; qb < NQB; ++qb) {
        float mx = -INFINITY;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[kb][qb][r]);
        mx = half_swap_max(mx);
        const float m_new = fmaxf(m_run[qb], mx * scale_log2);
        const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
        const float alpha = exp2f(m_run[qb] - m_use);
        m_run[qb] = m_new;
        l_run[qb] *= alpha;
#pragma unroll
        for (int db = 0; db < NDB; ++db) oacc[qb][db] *= alpha;
        float lsum = 0.f;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const float p = exp2f(fmaf(s[kb][qb][r], scale_log2, -m_use));
            s[kb][qb][r] = p;
            lsum += p;
          }
        l_run[qb] += lsum;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int hh = 0; hh < 2; ++hh)
#pragma unroll
            for (int e = 0; e < 8; ++e) pb[kb][hh][qb][e] = __bf16(s[kb][qb][8 * hh + e]);
      }
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
          for (int hh = 0; hh < 2; ++hh) {
            // keys 32kb + 16hh + 4g + {0..3} and + 8 + {0..3}; column 32db + (lane % 32)
            const __bf16* p = &Vs[(32 * kb + 16 * hh + 4 * g + tr_row) * VSTR + 32 * db + tr_col];
            const bf16x8 a = cat(lds_read_tr(p), lds_read_tr(p + 8 * VSTR));
#pragma unroll
            for (int qb = 0; qb < NQB; ++qb) oacc[qb][db] = mfma32(a, pb[kb][hh][qb], oacc[qb][db]);
          }
        }
      }
    }
    if (kt + 1 < n_tiles) {
      __syncthreads();
      store_tile();
      __syncthreads();
    }
  }

  // Epilogue.
#pragma unroll
  for (int qb = 0; qb < NQB; ++qb) {
    const float l_tot = half_swap_sum(l_run[qb]);
    const float inv = 1.f / l_tot;
    const int qrel = wave * QPW + 32 * qb + j;
    if (qrel < u.rows) {
      const int64_t row = int64_t(u.row0) + qrel;
      __bf16* orow = o + row * ts + int64_t(h) * D;
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int rb = 0; rb < 4; ++rb) {
          const int d0 = 32 * db + 8 * rb + 4 * g;
          if (d0 < D) {
            bf16x4 w;
#pragma unroll
            for (int c = 0; c < 4; ++c) w[c] = __bf16(oacc[qb][db][4 * rb + c] * inv);
            *reinterpret_cast<bf16x4*>(orow + d0) = w;
          }
        }
      if (g == 0) lse[int64_t(h) * T + row] = (m_run[qb] + log2f(l_tot)) * kLn2;
    }
  }
}

template <int D, int NQB, bool CAUSAL>
hipError_t launch_fwd_t(const FwdArgs& a) {
  dim3 grid(a.n_units, a.n_heads);
  hipLaunchKernelGGL((attn_fwd_kernel<D, NQB, CAUSAL>), grid, dim3(256), 0, a.stream,
                     static_cast<const __bf16*>(a.q), static_cast<const __bf16*>(a.k),
                     static_cast<const __bf16*>(a.v), static_cast<__bf16*>(a.o), a.lse,
                     static_cast<const WorkUnit*>(a.units), a.n_heads, a.total_tokens, a.scale * kLog2e);
  return hipGetLastError();
}

}  // namespace

int fwd_tile_rows(int head_dim) { return 4 * 32 * kFwdNQB; }

hipError_t launch_fwd(const FwdArgs& a) {
  if (a.n_units == 0) return hipSuccess;
  switch (a.head_dim) {
    case 64: return a.causal ? launch_fwd_t<64, kFwdNQB, true>(a) : launch_fwd_t<64, kFwdNQB, false>(a);
    case 72: return a.causal ? launch_fwd_t<72, kFwdNQB, true>(a) : launch_fwd_t<72, kFwdNQB, false>(a);
    case 128: return a.causal ? launch_fwd_t<128, kFwdNQB, true>(a) : launch_fwd_t<128, kFwdNQB, false>(a);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace dcp
