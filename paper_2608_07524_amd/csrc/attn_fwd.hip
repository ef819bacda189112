// Varlen attention forward on CDNA4: bf16 matrix-core products with an fp32
// online softmax (exact attention, as used for every run of the paper,
// Sec. 4.1; packed block-diagonal layout of Sec. 1).
//
// Work decomposition: one workgroup per (query tile, head).  A query tile
// never straddles two sequences, and the key loop runs over the tile's own
// sequence only, so no off-diagonal (cross-sequence) block is ever touched.
// NW wavefronts per workgroup, each owning 32*NQB query rows.
//
// Per key tile of BN = 64 keys (a three-stage LDS ring filled by direct
// global-to-LDS copies two tiles ahead; one barrier per tile):
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
#include <type_traits>

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
                                                           const __bf16* __restrict__ consts,
                                                           const WorkUnit* __restrict__ units, int per_xcd, int H, int T,
                                                           float scale_log2) {
  using S = FwdShape<D>;
  constexpr int NKD = S::NKD, NDB = S::NDB, KSTR = S::KSTR, VSTR = S::VSTR, CPR = S::CPR;
  constexpr int BN = kFwdBN;
  constexpr int NT = 64 * NW;  // threads
  constexpr int QPW = 32 * NQB;
  constexpr int KBUF = BN * KSTR, VBUF = BN * VSTR;
  using DK = DmaTile<BN, KSTR / 8, CPR, NW>;
  using DV = DmaTile<BN, VSTR / 8, CPR, NW>;
  constexpr int NI = DK::NI + DV::NI;  // copies per wavefront per tile

  // Three-stage ring: tile kt+2 streams in while tile kt is consumed.
  __shared__ __attribute__((aligned(16))) __bf16 Ks[3 * KBUF];
  __shared__ __attribute__((aligned(16))) __bf16 Vs[3 * VBUF];

  const WorkUnit u = unit_for_block(units, per_xcd);
  if (u.rows == 0) return;
  const int h = u.head;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: scalar branches on it
  const int g = lane >> 5;
  const int j = lane & 31;
  const int64_t ts = int64_t(H) * D;  // token stride

  const __bf16* qh = q + int64_t(u.seq0) * ts + int64_t(h) * D;
  const __bf16* kh = k + int64_t(u.seq0) * ts + int64_t(h) * D;
  const __bf16* vh = v + int64_t(u.seq0) * ts + int64_t(h) * D;
  const __bf16* zero = consts + kConstZero;
  // K pad columns must be zero (they enter the contraction); V's first pad
  // column holds ones when it is the row-sum column.
  const __bf16* v_pad = S::ONES_ROW ? consts + kConstOnes : zero;

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

  // Settle the Q loads here: the tile copies below are invisible to the
  // compiler's wait tracking, so no later compiler-inserted wait may stand
  // for these loads inside the tile loop.
  wait_vmcnt<0>();

  const int key_end = CAUSAL ? min(seqlen, tile_q0 + u.rows) : seqlen;
  const int n_tiles = (key_end + BN - 1) / BN;

  auto issue_tile = [&](int kt) {
    const unsigned st = unsigned(kt) % 3;
    const int valid = min(BN, seqlen - kt * BN);
    DK::issue(&Ks[st * KBUF], kh + int64_t(kt) * BN * ts, ts, valid, zero, zero, wave, lane);
    DV::issue(&Vs[st * VBUF], vh + int64_t(kt) * BN * ts, ts, valid, zero, v_pad, wave, lane);
  };
  // Before the barrier that ends tile kt: tile kt+1 must have landed; only
  // tile kt+2's copies (issued this iteration) may still be in flight.
  auto wait_next = [&](int kt) {
    if (kt + 2 < n_tiles) {
      wait_vmcnt<NI>();
    } else {
      wait_vmcnt<0>();
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

  if (n_tiles > 0) issue_tile(0);
  if (n_tiles > 1) issue_tile(1);
  wait_next(-1);
  __syncthreads();

  const int wave_last_q = wave_q0 + QPW - 1;
  // transposing-read addressing (see lds_read_tr): this lane's element
  // offset inside a V tile; every other term is a compile-time constant
  const unsigned tr_off = (4 * g + ((lane & 15) >> 2)) * VSTR + 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
  // and the 16-byte read offset inside a K tile
  const unsigned kr_off = j * KSTR + 8 * g;
  const lds_bf16* Ks3 = lds_ptr(Ks);
  const lds_bf16* Vs3 = lds_ptr(Vs);

  // One key tile.  MASK selects the variant for tiles that reach past the
  // sequence end or cross the causal diagonal; it is a compile-time flag so
  // the common unmasked tiles carry no per-element compare and select.
  auto process_tile = [&](unsigned st, int k0, auto mask_tag) {
    constexpr bool MASK = decltype(mask_tag)::value;
    unsigned kb0 = st * KBUF + kr_off;
    unsigned vb0 = st * VBUF + tr_off;
    asm("" : "+v"(kb0), "+v"(vb0));  // keeps the constant terms in the offset fields
    f32x16 s[2][NQB];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int qb = 0; qb < NQB; ++qb) s[kb][qb] = f32x16{};
#pragma unroll
    for (int kd = 0; kd < NKD; ++kd) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        const bf16x8 a = lds_read_b128(Ks3 + kb0 + 32 * kb * KSTR + 16 * kd);
#pragma unroll
        for (int qb = 0; qb < NQB; ++qb) s[kb][qb] = mfma32(a, qf[qb][kd], s[kb][qb]);
      }
    }
    if constexpr (MASK) {
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
          const lds_bf16* p = Vs3 + vb0 + (32 * kb + 16 * hh) * VSTR + 32 * db;
          const bf16x8 a = cat(lds_read_tr(p), lds_read_tr(p + 8 * VSTR));
#pragma unroll
          for (int qb = 0; qb < NQB; ++qb) oacc[qb][db] = mfma32(a, pb[kb][hh][qb], oacc[qb][db]);
        }
      }
    }
  };

  // Each wavefront walks the key tiles in up to three phases: tiles that
  // need no mask, the (at most two) tiles crossing the sequence end or its
  // causal diagonal, and, when causal, tiles entirely above its queries.
  // Every phase runs the same copy / wait / barrier sequence, so all
  // wavefronts meet the same number of barriers.
  const int n_full = seqlen / BN;  // tiles lying entirely inside the sequence
  int t_mask = min(n_tiles, n_full);
  int t_idle = n_tiles;
  if (CAUSAL) {
    t_mask = min(t_mask, (wave_q0 + 1) / BN);  // tiles whose last key is <= the wave's first query
    t_idle = min(n_tiles, wave_last_q / BN + 1);
  }
  auto run = [&](int kt0, int kt1, auto mode_tag) {
    constexpr int MODE = decltype(mode_tag)::value;  // 0 unmasked, 1 masked, 2 idle
    for (int kt = kt0; kt < kt1; ++kt) {
      const unsigned st = unsigned(kt) % 3;
      if (kt + 2 < n_tiles) issue_tile(kt + 2);
      if constexpr (MODE == 0) process_tile(st, kt * BN, std::false_type{});
      if constexpr (MODE == 1) process_tile(st, kt * BN, std::true_type{});
      wait_next(kt);
      __syncthreads();
    }
  };
  run(0, t_mask, std::integral_constant<int, 0>{});
  run(t_mask, t_idle, std::integral_constant<int, 1>{});
  if (CAUSAL) run(t_idle, n_tiles, std::integral_constant<int, 2>{});

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
  dim3 grid(a.n_units);
  const KernelEvents& ev = kernel_events();
  if (ev.begin) (void)hipEventRecord(ev.begin, a.stream);
  hipLaunchKernelGGL((attn_fwd_kernel<D, NQB, NW, CAUSAL>), grid, dim3(64 * NW), 0, a.stream,
                     static_cast<const __bf16*>(a.q), static_cast<const __bf16*>(a.k),
                     static_cast<const __bf16*>(a.v), static_cast<__bf16*>(a.o), a.lse,
                     static_cast<const __bf16*>(a.consts), static_cast<const WorkUnit*>(a.units),
                     a.n_units / kNumXcd, a.n_heads, a.total_tokens,
                     a.scale * kLog2e);
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
