// Varlen attention forward on CDNA4: bf16 matrix-core products with an fp32
// online softmax (exact attention, as used for every run of the paper,
// Sec. 4.1; packed block-diagonal layout of Sec. 1).
//
// Work decomposition: one workgroup per (query tile, head).  A query tile
// never straddles two sequences, and the key loop runs over the tile's own
// sequence only, so no off-diagonal (cross-sequence) block is ever touched.
// NW wavefronts per workgroup, each owning 32 query rows.
//
// Keys arrive in tiles of BN = 64 rows through a four-stage LDS ring filled
// by direct global-to-LDS copies three tiles ahead (one barrier per tile).
// Each wavefront walks its keys in blocks of 32 and software-pipelines them:
// while the exponentials of block b run on the vector ALUs, the matrix cores
// compute the scores of block b + 1, and while block b's probabilities are
// multiplied into O, the vector ALUs take block b + 1's row maximum.
//   S^T = K Q^T      A = K rows from LDS, B = Q rows kept in registers;
//                    each lane holds one query and 16 keys of the block.
//   m, P             row max: in-lane over 16 keys + one cross-half swap;
//                    P = exp2(S*scale*log2e - m) stays in registers.
//   O^T += V^T P^T   A = V^T via transposing LDS reads of the row-major V
//                    tile, B = P^T straight from the S^T accumulator layout.
// Rescaling is lazy: the running max m used in the exponent is only moved
// when some row's true max exceeds it by more than 2^8, so P <= 256 and the
// accumulators stay far from fp32 limits; the result O = acc / l does not
// depend on which m was used.  When the head width leaves a spare padded
// row in the last 32-row block of O^T (D = 72), a column of ones appended to
// V makes the matrix cores produce the row sum l = sum_j P_ij as well, and
// each block's row max decides the move.  Otherwise (D = 64, 128) the row
// sum is formed on the vector ALUs anyway, and it replaces the row max: a
// lane's 16 weights of a block sum to at most 2^8 unless one of them may
// exceed 2^8, so only a block whose sum passes 2^8 (rarely; in a packed
// window also a row's first block with keys of its own, where the weights
// against the initial m overflow) takes its row max, moves m and forms its
// weights again.
// Epilogue: O = O^T / l (bf16), LSE = (m + log2 l) * ln 2.
#include <type_traits>

#include "attn_common.h"
#include "attn_launch.h"

namespace dcp {
namespace {

constexpr int kFwdBN = 64;
// Ring depth: tile kt + kFwdStages - 1 streams in while tile kt is consumed.
constexpr int kFwdStages = 4;
static_assert(kFwdStages >= 3 && kWinFwdStages >= 3, "tiles kt and kt + 1 are read while kt + 2 lands");
constexpr float kRescaleSlack = 8.0f;  // log2 units
constexpr float kNoMax = -1e30f;       // running max before any key
constexpr float kSumBound = 256.0f;    // 2^kRescaleSlack

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
  // When 16-row blocks cover D plus the row-sum row with fewer padded rows
  // than 32-row blocks do (D = 72: 80 rows instead of 96), O^T is built
  // from 16x16x32 products instead.
  static constexpr int NMB = (D + 1 + 15) / 16;
  static constexpr bool PV16 = ONES_ROW && NMB * 16 < NDB * 32;
  // With 16x16x32 products a half-wavefront's transposing reads cover rows
  // 0..3 and 16..19 of a 32-key block, which any row stride puts on the
  // same banks (16 rows x 64 mod 128 bytes = 0 mod 256); starting every
  // 16-row group of the V tile 32 bytes further on moves the second set of
  // rows onto the other half of each bank run.
  static constexpr int VSKEW = PV16 ? 16 : 0;
};

template <int D, int NW, bool CAUSAL, bool PACKED, int STAGES>
__global__ __launch_bounds__(64 * NW) void attn_fwd_kernel(const __bf16* __restrict__ q,
                                                           const __bf16* __restrict__ k,
                                                           const __bf16* __restrict__ v, __bf16* __restrict__ o,
                                                           float* __restrict__ lse,
                                                           const __bf16* __restrict__ consts,
                                                           const WorkUnit* __restrict__ units,
                                                           const uint64_t* __restrict__ window_starts, int per_xcd,
                                                           int H, int T, float scale_log2) {
  using S = FwdShape<D>;
  constexpr int NKD = S::NKD, NDB = S::NDB, KSTR = S::KSTR, VSTR = S::VSTR, CPR = S::CPR;
  constexpr int BN = kFwdBN;
  constexpr int KBUF = BN * KSTR;
  using DK = DmaTile<BN, KSTR / 8, CPR, NW>;
  using DV = DmaTile<BN, VSTR / 8, CPR, NW, S::VSKEW>;
  constexpr int VBUF = DV::ELEMS;
  // as deep as asked, within the 160 KB of LDS
  constexpr int NST = STAGES * 2 * (KBUF + VBUF) <= 163840 ? STAGES : 163840 / (2 * (KBUF + VBUF));
  static_assert(NST >= 3, "ring too shallow");
  constexpr int NI = DK::NI + DV::NI;  // copies per wavefront per tile

  __shared__ __attribute__((aligned(16))) __bf16 Ks[NST * KBUF];
  __shared__ __attribute__((aligned(16))) __bf16 Vs[NST * VBUF];

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

  const int tile_q0 = u.row0 - u.seq0;  // first query of the tile, sequence-relative
  const int wave_q0 = tile_q0 + wave * 32;
  constexpr bool packed = PACKED;  // a list of packed windows only
  const int seqlen = packed ? int(u.rows) : u.seqlen;  // (window-relative offsets when packed)
  const int qi = wave_q0 + j;  // this lane's query
  // keys of this lane's sequence: [k_lo, k_hi)
  int k_lo = 0, k_hi = seqlen;
  if (packed) window_bounds(window_starts + kWindowWords * (-u.seqlen - 1), min(qi, seqlen - 1), seqlen, k_lo, k_hi);

  // Q fragments (B operand of S^T): lane (g, j) holds query j,
  // columns 16*kd + 8*g .. +7.
  bf16x8 qf[NKD];
#pragma unroll
  for (int kd = 0; kd < NKD; ++kd) {
    const int col = 16 * kd + 8 * g;
    if (wave * 32 + j < u.rows && col < D) {
      qf[kd] = *reinterpret_cast<const bf16x8*>(qh + int64_t(qi) * ts + col);
    } else {
      qf[kd] = bf16x8{};
    }
  }

  // Settle the Q loads here: the tile copies below are invisible to the
  // compiler's wait tracking, so no later compiler-inserted wait may stand
  // for these loads inside the tile loop.
  wait_vmcnt<0>();

  const int key_end = CAUSAL ? min(seqlen, tile_q0 + u.rows) : seqlen;
  const int n_tiles = (key_end + BN - 1) / BN;
  // This wavefront's 32-key blocks.  Blocks from b_mask on cross the
  // sequence end or the causal diagonal (only ever the last one or two);
  // blocks before it need no mask.  The wavefront works through whole
  // tiles: t_plain tiles whose blocks and successors are all unmasked, then
  // up to t_work tiles with masking on (a block past the wavefront's keys is
  // simply fully masked), then idles to n_tiles so that every wavefront
  // meets the same barriers.  A wavefront holding no query of the tile
  // (the last tile of a sequence) only copies and idles.  In a packed
  // window every block is masked, and the wavefront first idles through
  // the tiles before its first query's sequence (t_first).
  const bool live = wave * 32 < u.rows;
  const int last = min(31, int(u.rows) - 1 - wave * 32);  // lane of the wavefront's last query
  const int wave_keys = packed ? min(__builtin_amdgcn_readlane(k_hi, max(last, 0)), CAUSAL ? wave_q0 + 32 : seqlen)
                               : (CAUSAL ? min(seqlen, wave_q0 + 32) : seqlen);
  const int t_first = packed && live ? __builtin_amdgcn_readfirstlane(k_lo) / BN : 0;
  const int b_first = 2 * t_first;
  const int nb = live ? min((wave_keys + 31) / 32, 2 * n_tiles) : 0;
  const int b_mask = packed ? 0 : min(nb, CAUSAL ? min(seqlen / 32, (wave_q0 + 1) / 32) : seqlen / 32);
  const int t_work = (nb + 1) / 2;
  const int t_plain = b_mask >= 1 ? (b_mask - 1) / 2 : 0;  // tiles kt with 2kt + 2 < b_mask

  // Full tiles take the scalar-base copies.  When V's first pad column
  // carries the ones of the row-sum row, that column is written once per
  // ring stage here and full-tile copies leave it alone (partial tiles
  // rewrite it with the same ones).
  const typename DK::FullOffsets fo_k = DK::full_offsets(ts, wave, lane);
  const typename DV::FullOffsets fo_v = DV::full_offsets(ts, wave, lane);
  const auto vskip = DV::template skip_masks<CPR>(wave, lane);
  if constexpr (S::ONES_ROW) {
    for (int idx = tid; idx < NST * BN; idx += 64 * NW) {
      const int st = idx / BN, r = idx % BN;
      *reinterpret_cast<bf16x8*>(&Vs[st * VBUF + r * VSTR + S::VSKEW * (r / 16) + 8 * CPR]) =
          bf16x8{__bf16(1.f), __bf16(0.f), __bf16(0.f), __bf16(0.f), __bf16(0.f), __bf16(0.f), __bf16(0.f), __bf16(0.f)};
    }
  }
  auto issue_tile = [&](int kt) DCP_INLINE {
    const unsigned st = unsigned(kt) % NST;
    const int valid = min(BN, seqlen - kt * BN);
    if (valid == BN) {
      DK::issue_full(&Ks[st * KBUF], kh + int64_t(kt) * BN * ts, fo_k, wave);
      if constexpr (S::ONES_ROW) {
        DV::issue_full_skip(&Vs[st * VBUF], vh + int64_t(kt) * BN * ts, fo_v, vskip, wave);
      } else {
        DV::issue_full(&Vs[st * VBUF], vh + int64_t(kt) * BN * ts, fo_v, wave);
      }
    } else {
      DK::issue(&Ks[st * KBUF], kh + int64_t(kt) * BN * ts, ts, valid, zero, zero, wave, lane);
      DV::issue(&Vs[st * VBUF], vh + int64_t(kt) * BN * ts, ts, valid, zero, v_pad, wave, lane);
    }
  };
  // Before tile kt is consumed, tiles kt and kt + 1 must have landed (the
  // scores of tile kt + 1's first block are computed while tile kt is
  // processed); copies of the tiles after them may still be in flight.
  constexpr int PD = NST - 1;  // prefetch distance in tiles
  auto wait_for = [&](int kt) DCP_INLINE {
    const int ahead = min(PD - 2, n_tiles - kt - 2);  // tiles issued beyond kt + 1
    if (PD >= 4 && ahead >= 2) {
      wait_vmcnt<(PD >= 4 ? 2 * NI : 0)>();
    } else if (PD >= 3 && ahead >= 1) {
      wait_vmcnt<NI>();
    } else {
      wait_vmcnt<0>();
    }
  };

  // transposing-read addressing (see lds_read_tr): this lane's element
  // offset inside a V tile; every other term is a compile-time constant
  const unsigned tr_off = (4 * g + ((lane & 15) >> 2)) * VSTR + 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
  // (16x16x32 products: lane group g4 = lane / 16 reads the key runs
  // starting at 0, 16, 4, 20 and 8 further, see pv_product)
  const int g4 = lane >> 4;
  const unsigned tr16_off =
      (16 * (g4 & 1) + 4 * (g4 >> 1) + ((lane & 15) >> 2)) * VSTR + S::VSKEW * (g4 & 1) + 4 * (lane & 3);
  const unsigned tr_lane = S::PV16 ? tr16_off : tr_off;
  // and the 16-byte read offset inside a K tile
  const unsigned kr_off = j * KSTR + 8 * g;
  const lds_bf16* Ks3 = lds_ptr(Ks);
  const lds_bf16* Vs3 = lds_ptr(Vs);

  // Finite start: a row whose first blocks are all masked (packed windows)
  // then gets exp2(-inf + kNoMax) = 0 there, not NaN; its first key moves
  // m with a factor exp2(kNoMax - m) = 0 on the empty accumulators.
  float m_use = kNoMax, l_run = 0.f;
  f32x16 oacc[NDB];  // O^T in 32-row blocks (lane (g, j): query j)
#pragma unroll
  for (int db = 0; db < NDB; ++db) oacc[db] = f32x16{};
  // or, when PV16, in 16x16 blocks: [d block][query block]; lane (g4, n)
  // holds query 16 * qb + n, rows 16 * mb + 4 * g4 + {0..3}
  constexpr int NMB = S::NMB;
  f32x4 oacc16[NMB][2];
#pragma unroll
  for (int mb = 0; mb < NMB; ++mb) oacc16[mb][0] = oacc16[mb][1] = f32x4{};

  // K fragments (A operand of S^T) of one 32-key block whose K rows start
  // at LDS element kbase, and S^T from fragments held in registers.  The
  // fragments of the next block are read one step ahead, so the score
  // products never wait on their LDS reads.
  auto load_k = [&](unsigned kbase, bf16x8 (&kf)[NKD]) DCP_INLINE {
#pragma unroll
    for (int kd = 0; kd < NKD; ++kd) kf[kd] = lds_read_b128(Ks3 + kbase + 16 * kd);
  };
  auto scores = [&](const bf16x8 (&kf)[NKD]) DCP_INLINE {
    f32x16 s = f32x16{};
#pragma unroll
    for (int kd = 0; kd < NKD; ++kd) s = mfma32(kf[kd], qf[kd], s);
    return s;
  };
  auto apply_mask = [&](f32x16& s, int b) DCP_INLINE {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int key = 32 * b + 8 * (r >> 2) + 4 * g + (r & 3);
      if (unsigned(key - k_lo) >= unsigned(k_hi - k_lo) || (CAUSAL && key > qi)) s[r] = -INFINITY;
    }
  };
  auto row_max = [&](const f32x16& s) DCP_INLINE {
    float t = -INFINITY;  // a sequential chain lowers to v_max3
#pragma unroll
    for (int r = 0; r < 16; ++r) t = fmaxf(t, s[r]);
    return half_swap_max(t) * scale_log2;
  };
  // Lazy rescale: move m only when the row max outgrows it by > 2^8.
  auto rescale = [&](float mx, bool valid) DCP_INLINE {
    if (__builtin_amdgcn_ballot_w64(valid && mx > m_use + kRescaleSlack)) {
      const float m_new = fmaxf(m_use, mx);
      const float alpha = __builtin_amdgcn_exp2f(m_use - m_new);  // 0 on the first block
      m_use = m_new;
      l_run *= alpha;
      if constexpr (S::PV16) {
        // alpha of queries n and 16 + n for lane (g4, n)
        auto sw = __builtin_amdgcn_permlane16_swap(__float_as_uint(alpha), __float_as_uint(alpha), false, false);
        const float a0 = __uint_as_float(sw[0]), a1 = __uint_as_float(sw[1]);
#pragma unroll
        for (int mb = 0; mb < NMB; ++mb) {
          oacc16[mb][0] *= a0;
          oacc16[mb][1] *= a1;
        }
      } else {
#pragma unroll
        for (int db = 0; db < NDB; ++db) oacc[db] *= alpha;
      }
    }
  };

  // Unconditional move of m to the larger of m and mx (a wave-uniform
  // branch has already been taken).
  auto move_max = [&](float mx) DCP_INLINE {
    const float m_new = fmaxf(m_use, mx);
    const float alpha = __builtin_amdgcn_exp2f(m_use - m_new);
    m_use = m_new;
    l_run *= alpha;
#pragma unroll
    for (int db = 0; db < NDB; ++db) oacc[db] *= alpha;
  };

  // O^T += V^T P^T for the current block (V rows at vcur, this lane's
  // transposing-read offset included).  32x32 blocks: A = V^T rows
  // 32db + (lane % 32) over keys 16hh + 4g + {0..3, 8..11}, B = pb[hh]
  // as it is.  16x16 blocks: two lane-row swaps turn pb into the B
  // operands of queries 0..15 and 16..31, lane group g4 then holding keys
  // {0..3, 8..11}, {16..19, 24..27}, {4..7, 12..15}, {20..23, 28..31} for
  // g4 = 0..3, and the A operand of each 16-row block of V^T (two
  // transposing reads of those key runs) feeds both query blocks.
  auto pv_product = [&](const bf16x8 (&pb)[2], unsigned vcur) {
    if constexpr (S::PV16) {
      u32x4 x = __builtin_bit_cast(u32x4, pb[0]), y = __builtin_bit_cast(u32x4, pb[1]);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        auto sw = __builtin_amdgcn_permlane16_swap(x[i], y[i], false, false);
        x[i] = sw[0];
        y[i] = sw[1];
      }
      const bf16x8 b0 = __builtin_bit_cast(bf16x8, x), b1 = __builtin_bit_cast(bf16x8, y);
#pragma unroll
      for (int mb = 0; mb < NMB; ++mb) {
        const lds_bf16* p = Vs3 + vcur + 16 * mb;
        const bf16x8 a = cat(lds_read_tr(p), lds_read_tr(p + 8 * VSTR));
        oacc16[mb][0] = mfma16(a, b0, oacc16[mb][0]);
        oacc16[mb][1] = mfma16(a, b1, oacc16[mb][1]);
      }
    } else {
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
          const lds_bf16* p = Vs3 + vcur + 16 * hh * VSTR + 32 * db;
          oacc[db] = mfma32(cat(lds_read_tr(p), lds_read_tr(p + 8 * VSTR)), pb[hh], oacc[db]);
        }
    }
  };

#pragma unroll
  for (int t = 0; t < PD; ++t)
    if (t < n_tiles) issue_tile(t);
  wait_for(0);
  __syncthreads();

  // A tile this wavefront has no work in: its copies, wait and barrier.
  auto idle = [&](int kt) DCP_INLINE {
    if (kt + PD < n_tiles) issue_tile(kt + PD);
    wait_for(kt + 1);
    __syncthreads();
  };
  int kt = 0;
  for (; kt < t_first; ++kt) idle(kt);

  f32x16 sc{};  // S^T of the current block, masked, not yet exponentiated
  bf16x8 kn[NKD];  // K fragments of the block after it
  if (nb > b_first) {
    unsigned kb0 = (unsigned(t_first) % NST) * KBUF + kr_off;
    asm("" : "+v"(kb0));
    load_k(kb0, kn);
    sc = scores(kn);
    load_k(kb0 + 32 * KSTR, kn);
    if (b_mask <= b_first) apply_mask(sc, b_first);
    rescale(row_max(sc), true);
  }

  // One pipelined step: P and O for the current block (V rows at vcur)
  // while the scores of block bn (K fragments already in kn) are computed,
  // masked when MASK, and (D = 72) their row max taken; kn then receives
  // the K fragments of block bn + 1 (K rows at kafter).  On a wavefront's last
  // block the successor's scores are computed but not used (valid_next
  // false), and the reads ahead stay inside the ring.
  auto step = [&](int bn, unsigned kafter, unsigned vcur, bool valid_next, auto mask_tag) DCP_INLINE {
    constexpr bool MASK = decltype(mask_tag)::value;
    f32x16 sn = scores(kn);
    load_k(kafter, kn);
    // P = exp2(S*scale*log2e - m) as bf16 (B operand of the PV product)
    bf16x8 pb[2];
    auto exps = [&]() DCP_INLINE {
      const float mneg = -m_use;
#pragma unroll
      for (int hh = 0; hh < 2; ++hh)
#pragma unroll
        for (int e = 0; e < 8; ++e) pb[hh][e] = __bf16(__builtin_amdgcn_exp2f(fmaf(sc[8 * hh + e], scale_log2, mneg)));
    };
    exps();
    if constexpr (!S::ONES_ROW) {
      // the row sum over the same bf16 weights the PV product uses, so that
      // O = sum_j w_j v_j / sum_j w_j is an exact weighted mean of V rows
      // (pairwise dot products with (1, 1), one accumulator per half)
      auto psum = [&]() DCP_INLINE {
        const bf16x2 one = {__bf16(1.f), __bf16(1.f)};
        float lh[2] = {0.f, 0.f};
#pragma unroll
        for (int hh = 0; hh < 2; ++hh)
#pragma unroll
          for (int i = 0; i < 4; ++i)
            lh[hh] = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{pb[hh][2 * i], pb[hh][2 * i + 1]}, one, lh[hh], false);
        return lh[0] + lh[1];
      };
      // The lane's 16 weights sum to at most 2^8 unless one of them may
      // exceed 2^8 (or overflowed): only then is the block's row max taken,
      // m moved to it and the weights formed again (at most 1 each).
      float ls = psum();
      if (__builtin_amdgcn_ballot_w64(!(ls <= kSumBound))) {
        move_max(row_max(sc));
        exps();
        ls = psum();
      }
      l_run += ls;
    }
    if constexpr (MASK) apply_mask(sn, bn);
    pv_product(pb, vcur);
    if constexpr (S::ONES_ROW) rescale(row_max(sn), valid_next);
    sc = sn;
  };

  // Tile kt: blocks 2kt and 2kt + 1; the successor of the second block is
  // the first block of tile kt + 1, and the reads ahead take the two blocks
  // of tile kt + 1 (landed before tile kt began).
  auto tile = [&](int kt, auto mask_tag) DCP_INLINE {
    if (kt + PD < n_tiles) issue_tile(kt + PD);
    unsigned kb0 = (unsigned(kt) % NST) * KBUF + kr_off;
    unsigned kb1 = (unsigned(kt + 1) % NST) * KBUF + kr_off;
    unsigned vb0 = (unsigned(kt) % NST) * VBUF + tr_lane;
    asm("" : "+v"(kb0), "+v"(kb1), "+v"(vb0));  // keeps the constant terms in the offset fields
    step(2 * kt + 1, kb1, vb0, 2 * kt + 1 < 2 * t_work, mask_tag);
    step(2 * kt + 2, kb1 + 32 * KSTR, vb0 + 32 * VSTR + 2 * S::VSKEW, 2 * kt + 2 < 2 * t_work, mask_tag);
    wait_for(kt + 1);
    __syncthreads();
  };
  for (; kt < t_plain; ++kt) tile(kt, std::false_type{});
  for (; kt < t_work; ++kt) tile(kt, std::true_type{});
  for (; kt < n_tiles; ++kt) idle(kt);

  // Epilogue.
  if constexpr (S::PV16) {
    // the row-sum row D sits in block NMB-1, row D % 16: lane group
    // (D % 16) / 4, register D % 4, of the lanes holding queries n, 16 + n
    constexpr int rg = (D % 16) / 4, rr = D % 4;
    const int src = 16 * rg + (lane & 15);
    const float l0 = __shfl(oacc16[NMB - 1][0][rr], src);
    const float l1 = __shfl(oacc16[NMB - 1][1][rr], src);
    const float inv[2] = {1.f / l0, 1.f / l1};
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
      const int qrel = wave * 32 + 16 * qb + (lane & 15);
      if (qrel < u.rows) {
        __bf16* orow = o + (int64_t(u.row0) + qrel) * ts + int64_t(h) * D;
#pragma unroll
        for (int mb = 0; mb < NMB; ++mb) {
          const int d0 = 16 * mb + 4 * g4;
          if (d0 < D) {
            bf16x4 w;
#pragma unroll
            for (int c = 0; c < 4; ++c) w[c] = __bf16(oacc16[mb][qb][c] * inv[qb]);
            *reinterpret_cast<bf16x4*>(orow + d0) = w;
          }
        }
      }
    }
    const int qrel = wave * 32 + j;
    if (g == 0 && qrel < u.rows)
      lse[int64_t(h) * T + u.row0 + qrel] = (m_use + __log2f((j & 16) ? l1 : l0)) * kLn2;
    return;
  }
  float l_tot;
  if (S::ONES_ROW) {
    // row D of O^T: block NDB-1, in-block row D - 32*(NDB-1), held by g = 0 lanes
    constexpr int rr = D - 32 * (NDB - 1);
    constexpr int reg = 4 * (rr / 8) + (rr % 4);
    static_assert((rr % 8) < 4, "row-sum row must sit in the g = 0 half");
    const float mine = oacc[NDB - 1][reg];
    auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mine), __float_as_uint(mine), false, false);
    l_tot = __uint_as_float(sw[0]);  // lanes < 32 keep their own, lanes >= 32 get lane - 32
  } else {
    l_tot = half_swap_sum(l_run);
  }
  const float inv = 1.f / l_tot;
  const int qrel = wave * 32 + j;
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
          for (int c = 0; c < 4; ++c) w[c] = __bf16(oacc[db][4 * rb + c] * inv);
          *reinterpret_cast<bf16x4*>(orow + d0) = w;
        }
      }
    if (g == 0) lse[int64_t(h) * T + row] = (m_use + __log2f(l_tot)) * kLn2;
  }
}

template <int D, int NW, bool CAUSAL, bool PACKED, int STAGES>
hipError_t launch_fwd_list(const FwdArgs& a, const WorkUnit* units, int n_units) {
  hipLaunchKernelGGL((attn_fwd_kernel<D, NW, CAUSAL, PACKED, STAGES>), dim3(n_units), dim3(64 * NW), 0, a.stream,
                     static_cast<const __bf16*>(a.q), static_cast<const __bf16*>(a.k),
                     static_cast<const __bf16*>(a.v), static_cast<__bf16*>(a.o), a.lse,
                     static_cast<const __bf16*>(a.consts), units, static_cast<const uint64_t*>(a.window_starts),
                     n_units / kNumXcd, a.n_heads, a.total_tokens, a.scale * kLog2e);
  return hipGetLastError();
}

// Sequence tiles, then packed windows: one launch per non-empty list.
template <int D, int NW, bool CAUSAL>
hipError_t launch_fwd_t(const FwdArgs& a) {
  const KernelEvents& ev = kernel_events();
  const WorkUnit* units = static_cast<const WorkUnit*>(a.units);
  if (ev.begin) (void)hipEventRecord(ev.begin, a.stream);
  hipError_t e = hipSuccess;
  if (a.n_units > 0) e = launch_fwd_list<D, NW, CAUSAL, false, kFwdStages>(a, units, a.n_units);
  if (e == hipSuccess && a.n_wunits > 0)
    e = launch_fwd_list<D, kWinFwdWaves, CAUSAL, true, kWinFwdStages>(a, units + a.n_units, a.n_wunits);
  if (ev.end) (void)hipEventRecord(ev.end, a.stream);
  return e;
}

}  // namespace

hipError_t launch_fwd(const FwdArgs& a) {
  if (a.n_units == 0 && a.n_wunits == 0) return hipSuccess;
  constexpr int W = kFwdWaves;
  switch (a.head_dim) {
    case 64: return a.causal ? launch_fwd_t<64, W, true>(a) : launch_fwd_t<64, W, false>(a);
    case 72: return a.causal ? launch_fwd_t<72, W, true>(a) : launch_fwd_t<72, W, false>(a);
    case 128: return a.causal ? launch_fwd_t<128, W, true>(a) : launch_fwd_t<128, W, false>(a);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace dcp
