// Varlen attention forward on CDNA4: bf16 matrix-core products with an fp32
// online softmax (exact attention, as used for every run of the paper,
// Sec. 4.1; packed block-diagonal layout of Sec. 1).
//
// Work decomposition: one workgroup per (query tile, head).  A query tile
// never straddles two sequences, and the key loop runs over the tile's own
// sequence only, so no off-diagonal (cross-sequence) block is ever touched.
// NW wavefronts per workgroup, each owning 32*NQB query rows.
//
// Per key tile of BN = 64 keys (double-buffered in LDS; the next tile is
// prefetched into registers while the current one is consumed, so there is
// one barrier per tile):
//   S^T = K Q^T      A = K rows from LDS, B = Q rows kept in registers;
//                    each lane ends up holding one query and 16 keys.
//   m, P             row max: in-lane over 32 keys + one cross-half swap;
//                    P = exp2(S*scale*log2e - m) stays in registers.
//   O^T += V^T P^T   A = V^T via transposing LDS reads of the row-major V
//                    tile, B = P^T straight from the S^T accumulator layout.
// Rescaling is lazy: the running max m used in the exponent is only moved
// when some row's true max exceeds it by more than 2^8, so P <= 256 and the
// accumulators stay far from fp32 limits; the result O = acc / l does not
// depend on which m was used.  When the head width leaves a spare padded
// row in the last 32-row block of O^T (D = 72), a column of ones appended to
// V makes the matrix cores produce the row sum l = sum_j P_ij as well.
// Epilogue: O = O^T / l (bf16), LSE = (m + log2 l) * ln 2.
#include "attn_common.h"
#include "attn_launch.h"

namespace dcp {
namespace {

constexpr int kFwdBN = 64;
constexpr float kRescaleSlack = 8.0f;  // log2 units

template <int D>
struct FwdShape {
  static constexpr int DP = (D + 15) / 16 * 16;  // contraction width (zero padded)
  static constexpr int NKD = DP / 16;
  static constexpr int NDB = (D + 31) / 32;  // 32-row blocks of O^T
  static constexpr bool ONES_ROW = NDB * 32 > D;  // spare padded row carries l
  // K rows are read 16 B per lane: an odd multiple of 16 bytes avoids bank
  // conflicts.  V rows are read by transposing 8-byte reads, 4 rows x 64 B
  // per half-wavefront: a stride of 64 mod 128 bytes avoids conflicts.
  static constexpr int KSTR = DP + 8;
  static constexpr int VW = NDB * 32;
  static constexpr int VSTR = (VW % 64 == 32) ? VW : VW + 32;
  static constexpr int CPR = D / 8;  // 16-byte chunks per row
};

template <int D, int NQB, int NW, bool CAUSAL>
__global__ __launch_bounds__(64 * NW) void attn_fwd_kernel(const __bf16* __restrict__ q,
                                                           const __bf16* __restrict__ k,
                                                           const __bf16* __restrict__ v, __bf16* __restrict__ o,
                                                           float* __restrict__ lse,
                                                           const WorkUnit* __restrict__ units, int H, int T,
                                                           float scale_log2) {
  using S = FwdShape<D>;
  constexpr int NKD = S::NKD, NDB = S::NDB, KSTR = S::KSTR, VSTR = S::VSTR, CPR = S::CPR;
  constexpr int BN = kFwdBN;
  constexpr int NT = 64 * NW;  // threads
  constexpr int QPW = 32 * NQB;
  constexpr int NCH = BN * CPR;
  constexpr int CPT = (NCH + NT - 1) / NT;
  constexpr int KBUF = BN * KSTR, VBUF = BN * VSTR;

  __shared__ __attribute__((aligned(16))) __bf16 Ks[2 * KBUF];
  __shared__ __attribute__((aligned(16))) __bf16 Vs[2 * VBUF];

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

  // Columns past D are never written by tile loads.  K pads must be zero
  // (they enter the contraction); V pads are zero except column D, which
  // holds ones when it is the row-sum column.
  for (int i = tid; i < 2 * BN * (KSTR - D); i += NT) {
    const int r = i / (KSTR - D), c = D + i % (KSTR - D);
    Ks[r * KSTR + c] = __bf16(0.f);
  }
  for (int i = tid; i < 2 * BN * (VSTR - D); i += NT) {
    const int r = i / (VSTR - D), c = D + i % (VSTR - D);
    Vs[r * VSTR + c] = __bf16((S::ONES_ROW && c == D) ? 1.f : 0.f);
  }

  const int tile_q0 = u.row0 - u.seq0;       // first query of the tile, sequence-relative
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
      const int ch = tid + NT * c;
      if (NCH % NT == 0 || ch < NCH) {
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
  auto store_tile = [&](int buf) {
#pragma unroll
    for (int c = 0; c < CPT; ++c) {
      const int ch = tid + NT * c;
      if (NCH % NT == 0 || ch < NCH) {
        const int r = ch / CPR, cc = ch % CPR;
        *reinterpret_cast<u32x4*>(&Ks[buf * KBUF + r * KSTR + cc * 8]) = kreg[c];
        *reinterpret_cast<u32x4*>(&Vs[buf * VBUF + r * VSTR + cc * 8]) = vreg[c];
      }
    }
  };

  float m_use[NQB], l_run[NQB];
  f32x16 oacc[NQB][NDB];
#pragma unroll
  for (int qb = 0; qb < NQB; ++qb) {
    m_use[qb] = -INFINITY;
    l_run[qb] = 0.f;
#pragma unroll
    for (int db = 0; db < NDB; ++db) oacc[qb][db] = f32x16{};
  }

  if (n_tiles > 0) {
    load_tile(0);
    store_tile(0);
  }
  __syncthreads();

  const int wave_last_q = wave_q0 + QPW - 1;
  // transposing-read addressing (see lds_read_tr): row and column offsets
  const int tr_row = (lane & 15) >> 2;
  const int tr_col = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);

  for (int kt = 0; kt < n_tiles; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < n_tiles) load_tile(kt + 1);
    const int k0 = kt * BN;
    const bool active = !CAUSAL || k0 <= wave_last_q;
    if (active) {
      const __bf16* Kb = &Ks[buf * KBUF];
      const __bf16* Vb = &Vs[buf * VBUF];
      f32x16 s[2][NQB];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int qb = 0; qb < NQB; ++qb) s[kb][qb] = f32x16{};
#pragma unroll
      for (int kd = 0; kd < NKD; ++kd) {
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
          const bf16x8 a = lds_read_b128(&Kb[(32 * kb + j) * KSTR + 16 * kd + 8 * g]);
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
      // Lazy rescale: move m only when a row's max outgrows it by > 2^8.
      float mx[NQB];
      bool grow = false;
#pragma unroll
      for (int qb = 0; qb < NQB; ++qb) {
        float t = -INFINITY;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int r = 0; r < 16; ++r) t = fmaxf(t, s[kb][qb][r]);
        mx[qb] = half_swap_max(t) * scale_log2;
        grow |= mx[qb] > m_use[qb] + kRescaleSlack;
      }
      if (__builtin_amdgcn_ballot_w64(grow)) {
#pragma unroll
        for (int qb = 0; qb < NQB; ++qb) {
          const float m_new = fmaxf(m_use[qb], mx[qb]);
          const float alpha = __builtin_amdgcn_exp2f(m_use[qb] - m_new);  // 0 on the first tile
          m_use[qb] = m_new;
          l_run[qb] *= alpha;
#pragma unroll
          for (int db = 0; db < NDB; ++db) oacc[qb][db] *= alpha;
        }
      }
      bf16x8 pb[2][2][NQB];
#pragma unroll
      for (int qb = 0; qb < NQB; ++qb) {
        // every row has a finite max after its first tile (key 0 is visible)
        const float mneg = -m_use[qb];
        float lsum = 0.f;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const float p = __builtin_amdgcn_exp2f(fmaf(s[kb][qb][r], scale_log2, mneg));
            s[kb][qb][r] = p;
            if (!S::ONES_ROW) lsum += p;
          }
        if (!S::ONES_ROW) l_run[qb] += lsum;
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
            const __bf16* p = &Vb[(32 * kb + 16 * hh + 4 * g + tr_row) * VSTR + 32 * db + tr_col];
            const bf16x8 a = cat(lds_read_tr(p), lds_read_tr(p + 8 * VSTR));
#pragma unroll
            for (int qb = 0; qb < NQB; ++qb) oacc[qb][db] = mfma32(a, pb[kb][hh][qb], oacc[qb][db]);
          }
        }
      }
    }
    if (kt + 1 < n_tiles) store_tile(buf ^ 1);
    __syncthreads();
  }

  // Epilogue.
#pragma unroll
  for (int qb = 0; qb < NQB; ++qb) {
    float l_tot;
    if (S::ONES_ROW) {
      // row D of O^T: block NDB-1, in-block row D - 32*(NDB-1), held by g = 0 lanes
      constexpr int rr = D - 32 * (NDB - 1);
      constexpr int reg = 4 * (rr / 8) + (rr % 4);
      static_assert((rr % 8) < 4, "row-sum row must sit in the g = 0 half");
      const float mine = oacc[qb][NDB - 1][reg];
      auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mine), __float_as_uint(mine), false, false);
      l_tot = __uint_as_float(sw[0]);  // lanes < 32 keep their own, lanes >= 32 get lane - 32
    } else {
      l_tot = half_swap_sum(l_run[qb]);
    }
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
      if (g == 0) lse[int64_t(h) * T + row] = (m_use[qb] + __log2f(l_tot)) * kLn2;
    }
  }
}

template <int D, int NQB, int NW, bool CAUSAL>
hipError_t launch_fwd_t(const FwdArgs& a) {
  dim3 grid(a.n_units, a.n_heads);
  const KernelEvents& ev = kernel_events();
  if (ev.begin) (void)hipEventRecord(ev.begin, a.stream);
  hipLaunchKernelGGL((attn_fwd_kernel<D, NQB, NW, CAUSAL>), grid, dim3(64 * NW), 0, a.stream,
                     static_cast<const __bf16*>(a.q), static_cast<const __bf16*>(a.k),
                     static_cast<const __bf16*>(a.v), static_cast<__bf16*>(a.o), a.lse,
                     static_cast<const WorkUnit*>(a.units), a.n_heads, a.total_tokens, a.scale * kLog2e);
  hipError_t e = hipGetLastError();
  if (ev.end) (void)hipEventRecord(ev.end, a.stream);
  return e;
}

}  // namespace

int fwd_tile_rows(int head_dim) { return kFwdWaves * 32 * kFwdNQB; }

hipError_t launch_fwd(const FwdArgs& a) {
  if (a.n_units == 0) return hipSuccess;
  constexpr int Q = kFwdNQB, W = kFwdWaves;
  switch (a.head_dim) {
    case 64: return a.causal ? launch_fwd_t<64, Q, W, true>(a) : launch_fwd_t<64, Q, W, false>(a);
    case 72: return a.causal ? launch_fwd_t<72, Q, W, true>(a) : launch_fwd_t<72, Q, W, false>(a);
    case 128: return a.causal ? launch_fwd_t<128, Q, W, true>(a) : launch_fwd_t<128, Q, W, false>(a);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace dcp
