// Varlen attention backward on CDNA4 for the loss <dO, O> (gradients of the
// exact attention the paper trains with, Sec. 4.1; block diagonal over the
// packed sequences of Sec. 1).
//
// Three launches, no atomics, bitwise deterministic:
//   1. bwd_delta:  -Delta = -rowsum(dO o O) and LSE*log2e per (row, head),
//                  fp32.
//   2. bwd_dkdv:   key-stationary.  One workgroup per (key tile, head);
//                  each wavefront keeps the K and V fragments of 32 keys
//                  (at head width 128 V comes from an LDS copy instead, so
//                  that two wavefronts fit per SIMD) and their dK, dV
//                  accumulators in registers and walks
//                  the query tiles of its own sequence (on or below the
//                  diagonal when causal), Q / dO tiles streaming through an
//                  LDS ring:
//                    S  = Q K^T,  dP = dO V^T         (A from LDS, B in regs)
//                    P  = exp2(S*scale*log2e - LSE*log2e)
//                    dS = P o (dP - Delta)
//                    dV += P^T dO,  dK += dS^T Q       (B via transposing reads)
//                  In the S / dP accumulators a lane holds one key and 16
//                  queries: exactly the A-operand layout P^T and dS^T need.
//   3. bwd_dq:     query-stationary, shaped like the forward.  One workgroup
//                  per (query tile of 32*NW rows, head); each wavefront keeps
//                  32 queries' Q and dO fragments, LSE, Delta and its dQ^T
//                  accumulator in registers while K / V tiles stream through
//                  LDS:
//                    S^T = K Q^T,  dP^T = V dO^T       (A from LDS, B in regs)
//                    dS^T = exp2(S^T*c - LSE*log2e) o (dP^T - Delta)
//                    dQ^T += K^T dS^T                  (A via transposing reads,
//                                                       B = dS^T from registers)
// The dQ pass recomputes S and dP (two extra products) instead of adding
// per-key-tile partial dQ into an fp32 accumulator with atomics.
#include <type_traits>

#include "attn_common.h"
#include "attn_launch.h"



namespace dcp {
namespace {

template <int D>
struct BwdShape {
  static constexpr int DP = (D + 15) / 16 * 16;  // contraction width (zero padded)
  static constexpr int NKD = DP / 16;
  static constexpr int NDB = (D + 31) / 32;  // 32-column blocks of dK, dV, dQ
  static constexpr int CPR = D / 8;          // 16-byte chunks per row
  // Row strides (elements).  Rows read 16 B per lane want an odd multiple
  // of 16 bytes; rows read by transposing 8-byte reads (4 rows x 64 B per
  // half-wavefront) want 64 mod 128 bytes.  Tiles read both ways take the
  // first and cover NDB*32 columns.
  static constexpr int W = (DP > NDB * 32) ? DP : NDB * 32;
  static constexpr int RSTR = W + 8;                                  // both ways
  static constexpr int TSTR = (NDB * 32 % 64 == 32) ? NDB * 32 : NDB * 32 + 32;  // transposing only
  // dK and dV from 16x16x32 products when 16-column blocks cover D with
  // fewer padded columns than 32-column blocks (D = 72: 80 instead of 96).
  static constexpr int NMB = (D + 15) / 16;
  static constexpr bool KV16 = NMB * 16 < NDB * 32;
  // Stride of a tile held once and read both ways.  An odd number of
  // 16-byte chunks keeps the 16-byte row reads conflict-free (16 lanes, 16
  // rows: 64 banks).  The transposing reads of a half-wavefront cover 4
  // consecutive rows (KV16: 8 bank-wide runs of 32 bytes; else 16-bank runs
  // of 64 bytes), so the row starts should spread over the banks: at D = 72,
  // 104 elements puts them 12 banks apart and every run lands on its own
  // banks (only the two row groups 16 apart, always on the same banks,
  // meet); at D = 128, 152 elements leaves two-way overlaps where the
  // minimal 136 stacks four.
  static constexpr int OSTR = D == 72 ? 104 : D == 128 ? 152 : DP + 8;
  static_assert(OSTR % 16 == 8 && OSTR >= (KV16 ? NMB * 16 : NDB * 32), "one-copy stride");
};

// ---------------------------------------------------------------------------
// 1. -Delta = -rowsum(dO o O) and LSE*log2e per (row, head), fp32 [H, T].
// A workgroup takes kDeltaRows rows x up to kDeltaHeads heads: 16 lanes per
// (row, head) pair, lane c covering columns 8c..8c+7.  Pairs are taken
// row-major, so the heads of one token -- adjacent in memory -- are read
// together and the bf16 rows arrive as whole cache lines; the sums meet in
// LDS and leave head-major, kDeltaRows consecutive fp32 values (128 bytes)
// per head.  1024 threads: each 16-lane group takes 8 pairs, all loads in
// flight at once (short sequences give few workgroups, so the per-workgroup
// latency is the pass's).
constexpr int kDeltaRows = 32, kDeltaHeads = 16, kDeltaThreads = 1024;
template <int D>
__global__ __launch_bounds__(kDeltaThreads) void bwd_delta_kernel(const __bf16* __restrict__ dout,
                                                        const __bf16* __restrict__ o,
                                                        const float* __restrict__ lse, float* __restrict__ ndelta,
                                                        float* __restrict__ lse2, int rows_end, int H, int T) {
  constexpr int CPR = D / 8;
  constexpr int NPAIR = kDeltaRows * kDeltaHeads;
  __shared__ float nd_lds[kDeltaHeads][kDeltaRows + 1];
  const int r0 = blockIdx.x * kDeltaRows;
  const int h0 = blockIdx.y * kDeltaHeads;
  const int hc = min(kDeltaHeads, H - h0);
  const int rows = min(kDeltaRows, rows_end - r0);
  const int n_pairs = rows * hc;
  const int c = threadIdx.x & 15;
  // (every lane runs every step: the 16-lane reductions need all of them)
#pragma unroll
  for (int p = threadIdx.x >> 4; p < NPAIR; p += kDeltaThreads / 16) {
    const int r = p / hc, hh = p - r * hc;
    float part = 0.f;
    if (p < n_pairs && c < CPR) {
      const int64_t off = (int64_t(r0 + r) * H + h0 + hh) * D + 8 * c;
      const bf16x8 x = *reinterpret_cast<const bf16x8*>(dout + off);
      const bf16x8 y = *reinterpret_cast<const bf16x8*>(o + off);
#pragma unroll
      for (int e = 0; e < 8; ++e) part = fmaf(float(x[e]), float(y[e]), part);
    }
    part += __shfl_xor(part, 8, 16);
    part += __shfl_xor(part, 4, 16);
    part += __shfl_xor(part, 2, 16);
    part += __shfl_xor(part, 1, 16);
    if (p < n_pairs && c == 0) nd_lds[hh][r] = -part;
  }
  __syncthreads();
  for (int e = threadIdx.x; e < NPAIR; e += kDeltaThreads) {
    const int hh = e / kDeltaRows, r = e % kDeltaRows;
    if (hh < hc && r < rows) {
      const int64_t i = int64_t(h0 + hh) * T + r0 + r;
      ndelta[i] = nd_lds[hh][r];
      lse2[i] = lse[i] * kLog2e;
    }
  }
}

// Writes a wavefront's 32 x D fp32 accumulator block (C layout: lane (g, j)
// holds column 32*db + j of rows 8*(r/4) + 4*g + r%4) as bf16 rows through
// an LDS staging area of 32 rows x stride `st`, with 16-byte global stores.
// Orders this wavefront's LDS accesses: everything issued before has
// completed before anything after is issued.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");
  __builtin_amdgcn_wave_barrier();
}

template <int D, int NDB>
__device__ __forceinline__ void store_rows_bf16(const f32x16 (&acc)[NDB], float mul, __bf16* stage, int st,
                                                __bf16* __restrict__ base, int64_t row_stride, int n_rows,
                                                int lane) {
  const int g = lane >> 5, j = lane & 31;
  wave_lds_sync();
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = 8 * (r >> 2) + 4 * g + (r & 3);
      stage[row * st + 32 * db + j] = __bf16(acc[db][r] * mul);
    }
  wave_lds_sync();
  constexpr int CPR = D / 8;
  for (int ch = lane; ch < 32 * CPR; ch += 64) {
    const int row = ch / CPR, cc = ch % CPR;
    if (row < n_rows)
      *reinterpret_cast<u32x4*>(base + int64_t(row) * row_stride + cc * 8) =
          *reinterpret_cast<const u32x4*>(&stage[row * st + cc * 8]);
  }
  wave_lds_sync();
}

// The same for accumulators in 16x16 blocks [key block][column block]
// (C layout of v_mfma_f32_16x16x32: lane (g4, n) holds column 16*nb + n of
// rows 16*mb + 4*g4 + r).
template <int D, int NMB>
__device__ __forceinline__ void store_rows16_bf16(const f32x4 (&acc)[2][NMB], float mul, __bf16* stage, int st,
                                                  __bf16* __restrict__ base, int64_t row_stride, int n_rows,
                                                  int lane) {
  const int g4 = lane >> 4, n = lane & 15;
  wave_lds_sync();
#pragma unroll
  for (int mb = 0; mb < 2; ++mb)
#pragma unroll
    for (int nb = 0; nb < NMB; ++nb)
#pragma unroll
      for (int r = 0; r < 4; ++r) stage[(16 * mb + 4 * g4 + r) * st + 16 * nb + n] = __bf16(acc[mb][nb][r] * mul);
  wave_lds_sync();
  constexpr int CPR = D / 8;
  for (int ch = lane; ch < 32 * CPR; ch += 64) {
    const int row = ch / CPR, cc = ch % CPR;
    if (row < n_rows)
      *reinterpret_cast<u32x4*>(base + int64_t(row) * row_stride + cc * 8) =
          *reinterpret_cast<const u32x4*>(&stage[row * st + cc * 8]);
  }
  wave_lds_sync();
}

// Moves the two halves of a 32x32 accumulator-layout operand (lane (g, j):
// index j, contraction values {8b + 4g + c}, b in {0,1} in x and {2,3} in
// y) into the 16x16x32 layout: x becomes the operand of indices 0..15 and
// y that of indices 16..31, lane group g4 = lane / 16 then holding the
// contraction values {0..3, 8..11}, {16..19, 24..27}, {4..7, 12..15},
// {20..23, 28..31} for g4 = 0..3 (v_permlane16_swap exchanges the odd
// 16-lane rows of x with the even rows of y).
__device__ __forceinline__ void to_mfma16_layout(bf16x8& xv, bf16x8& yv) {
  u32x4 x = __builtin_bit_cast(u32x4, xv), y = __builtin_bit_cast(u32x4, yv);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    auto sw = __builtin_amdgcn_permlane16_swap(x[i], y[i], false, false);
    x[i] = sw[0];
    y[i] = sw[1];
  }
  xv = __builtin_bit_cast(bf16x8, x);
  yv = __builtin_bit_cast(bf16x8, y);
}

// ---------------------------------------------------------------------------
// 2. dK, dV (key-stationary).
//
// Each wavefront owns 32*KB keys: their K and V fragments (B operands of
// S = Q K^T and dP = dO V^T) and their dK, dV accumulators stay in
// registers for the whole query loop.  Query tiles of BM rows stream
// through an NSTAGE-deep LDS ring filled by direct global-to-LDS copies
// NSTAGE - 1 tiles ahead, one barrier per tile: Q and dO twice each (rows
// read 16 B per lane for the A operands of S and dP, rows read by
// transposing reads for the B operands of dV and dK, each copy at its
// conflict-free stride), plus LSE*log2e and -Delta of the tile's queries.
// -Delta is the initial value of the dP accumulator, so the products yield
// dP - Delta directly.  With KB = 2 every operand fetched from LDS feeds
// two matrix products, and the exponentials of one key block can overlap
// the products of the other.
//
// FUSED (packed windows, 32-query tiles, one 32-key block per wavefront):
// the workgroup holds every key of the queries it visits, so it also
// computes dQ = scale * dS K.  Each wavefront writes its bf16 dS^T block
// (32 keys x the tile's 32 queries) into an LDS matrix of the window's keys
// x 32 queries (two buffers, alternating per tile); after the tile's
// barrier the wavefronts split the tile's 16x16 dQ output blocks, reading dS
// and a copy of the window's K (both by transposing reads) from LDS.  To
// fit two workgroups per CU the ring then holds Q and dO once, at the
// row-read stride, and the transposing reads of dV and dK use that copy.
template <int D, int KB, int NW, int BM, int NSTAGE, int WPE, bool CAUSAL, bool PACKED, bool FUSED, bool ONECOPY,
          bool VLDS>
__global__ __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(WPE))) void attn_bwd_dkdv_kernel(
    const __bf16* __restrict__ q, const __bf16* __restrict__ k, const __bf16* __restrict__ v,
    const __bf16* __restrict__ dout, const float* __restrict__ lse2, const float* __restrict__ ndelta,
    __bf16* __restrict__ dk, __bf16* __restrict__ dv, __bf16* __restrict__ dq, const __bf16* __restrict__ consts,
    const WorkUnit* __restrict__ units, const uint64_t* __restrict__ window_starts, int per_xcd, int H, int T,
    float scale, float scale_log2) {
  using S = BwdShape<D>;
  constexpr int NKD = S::NKD, NDB = S::NDB, CPR = S::CPR;
  // an odd number of 16-byte chunks (one copy outside packed windows: the
  // stride that also spreads the transposing reads; the fused window launch
  // keeps the minimal one to fit two workgroups per CU)
  constexpr int RSTR = (ONECOPY && !FUSED) ? S::OSTR : S::DP + 8;
  constexpr int TSTR = ONECOPY ? RSTR : S::TSTR;  // (one copy: it serves both reads)
  static_assert(BM % 32 == 0, "whole 32-query blocks per tile");
  static_assert(!FUSED || (PACKED && KB == 1 && BM == 32 && ONECOPY),
                "fused dQ: packed windows, 32-query tiles, KB 1, one ring copy");
  static_assert(!VLDS || (KB == 1 && !FUSED && !BwdShape<D>::KV16), "V from LDS: one key block, 32x32 products");
  using DR = DmaTile<BM, RSTR / 8, CPR, NW>;
  using DT = DmaTile<BM, TSTR / 8, CPR, NW>;
  using DL = DmaVecPair<BM, NW>;
  constexpr int NI = ONECOPY ? 2 * DR::NI + DL::NI : 2 * DR::NI + 2 * DT::NI + DL::NI;  // copies per wavefront per tile
  constexpr int RBUF = DR::ELEMS, TBUF = ONECOPY ? 0 : DT::ELEMS;
  constexpr int SSTR = S::RSTR;  // epilogue staging stride
  // fused dQ: the window's K rows for transposing reads, and dS^T
  constexpr int NKEY = 32 * NW;
  constexpr int KTSTR = S::TSTR;  // 64 mod 128 bytes
  using DKT = DmaTile<NKEY, KTSTR / 8, CPR, NW>;
  constexpr int KTBUF = FUSED ? DKT::ELEMS : 0;
  constexpr int DSBUF = FUSED ? NKEY * BM : 0;  // one buffer: [key][query], rows of 64 bytes
  constexpr int NMQ = (D + 15) / 16;            // 16-column blocks of dQ
  __shared__ __attribute__((aligned(16))) __bf16 Qr[NSTAGE * RBUF];
  __shared__ __attribute__((aligned(16))) __bf16 dOr[NSTAGE * RBUF];
  __shared__ __attribute__((aligned(16))) __bf16 Qt[ONECOPY ? 8 : NSTAGE * TBUF];
  __shared__ __attribute__((aligned(16))) __bf16 dOt[ONECOPY ? 8 : NSTAGE * TBUF];
  __shared__ __attribute__((aligned(16))) float LV[NSTAGE * 2 * BM];  // LSE*log2e | -Delta
  __shared__ __attribute__((aligned(16))) __bf16 Kt[FUSED ? KTBUF : 8];
  __shared__ __attribute__((aligned(16))) __bf16 dSt[FUSED ? 2 * DSBUF : 8];
  // (VLDS) the tile's V rows, read 16 bytes per lane as B operands (an odd
  // number of 16-byte chunks per row: conflict-free); rows past the tile's
  // keys are zero
  constexpr int VLSTR = S::DP + 8;
  using DVL = DmaTile<32 * KB * NW, VLSTR / 8, CPR, NW>;
  __shared__ __attribute__((aligned(16))) __bf16 Vl[VLDS ? DVL::ELEMS : 8];
  constexpr int NSB = NW * KB;  // 32-key blocks per workgroup
  static_assert(NSB % 2 == 0 && NSTAGE * RBUF >= NSB / 2 * 32 * SSTR, "staging area too small");
  static_assert(NSTAGE >= 2 && NSTAGE <= 4, "ring depth");
  static_assert(2 * NI < 64, "vmcnt range");

  const WorkUnit u = unit_for_block(units, per_xcd);
  if (u.rows == 0) return;
  const int h = u.head;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: scalar branches on it
  const int g = lane >> 5;
  const int j = lane & 31;
  const int64_t ts = int64_t(H) * D;
  constexpr bool packed = PACKED;  // a list of packed windows only
  const int seqlen = packed ? int(u.rows) : u.seqlen;  // (window-relative offsets when packed)
  const int key_t0 = u.row0 - u.seq0;  // first key of the workgroup, sequence-relative
  const __bf16* zero = consts + kConstZero;
  const float* fzero = reinterpret_cast<const float*>(consts + kConstZero);
  const float* finf = reinterpret_cast<const float*>(consts + kConstInf);

  const __bf16* qh = q + int64_t(u.seq0) * ts + int64_t(h) * D;
  const __bf16* kh = k + int64_t(u.seq0) * ts + int64_t(h) * D;
  const __bf16* vh = v + int64_t(u.seq0) * ts + int64_t(h) * D;
  const __bf16* doh = dout + int64_t(u.seq0) * ts + int64_t(h) * D;
  const float* lseh = lse2 + int64_t(h) * T + u.seq0;
  const float* ndh = ndelta + int64_t(h) * T + u.seq0;

  // K and V fragments: lane (g, j) of key block kb holds key 32*(KB*wave +
  // kb) + j of the tile, columns 16*kd + 8*g .. +7.  Keys past the sequence
  // end are zero; their dK, dV rows are never stored.
  bf16x8 kf[KB][NKD], vf[KB][NKD];
#pragma unroll
  for (int kb = 0; kb < KB; ++kb) {
    const int key = 32 * (KB * wave + kb) + j;
    const bool ok = key < u.rows;
#pragma unroll
    for (int kd = 0; kd < NKD; ++kd) {
      const int col = 16 * kd + 8 * g;
      if (ok && col < D) {
        kf[kb][kd] = *reinterpret_cast<const bf16x8*>(kh + int64_t(key_t0 + key) * ts + col);
        if constexpr (!VLDS) vf[kb][kd] = *reinterpret_cast<const bf16x8*>(vh + int64_t(key_t0 + key) * ts + col);
      } else {
        kf[kb][kd] = bf16x8{};
        if constexpr (!VLDS) vf[kb][kd] = bf16x8{};
      }
    }
  }
  wait_vmcnt<0>();  // settle the fragment loads before the first copy
  // (fused) the window's keys, rows past its end zero; issued before the
  // first ring tile, so the first ring wait covers it
  if constexpr (FUSED) DKT::issue(Kt, kh + int64_t(key_t0) * ts, ts, u.rows, zero, zero, wave, lane);
  // (VLDS) likewise the tile's V rows
  if constexpr (VLDS) DVL::issue(Vl, vh + int64_t(key_t0) * ts, ts, u.rows, zero, zero, wave, lane);

  const int wave_key_lo = key_t0 + 32 * KB * wave;  // smallest key of this wavefront
  // queries of each key's sequence: [q_lo, q_hi)
  int q_lo[KB], q_hi[KB];
#pragma unroll
  for (int kb = 0; kb < KB; ++kb) {
    q_lo[kb] = 0;
    q_hi[kb] = seqlen;
    if (packed)
      window_bounds(window_starts + kWindowWords * (-u.seqlen - 1), min(wave_key_lo + 32 * kb + j, seqlen - 1),
                    seqlen, q_lo[kb], q_hi[kb]);
  }
  const int q_begin = CAUSAL ? (key_t0 / BM) * BM : 0;
  const int n_qt = (seqlen - q_begin + BM - 1) / BM;
  // Causal sequence tiles walk their query tiles from the sequence end back
  // to the diagonal: the key workgroups of one sequence and head, which run
  // side by side on one die, then read the same Q and dO rows at about the
  // same time and share them in its L2.  Step it of the walk takes query
  // tile tile_of(it).
  constexpr bool REV = CAUSAL && !PACKED;
  auto tile_of = [&](int it) DCP_INLINE { return REV ? n_qt - 1 - it : it; };

  // Full query tiles take the scalar-base copies, except in the causal
  // one-wavefront-per-SIMD variant: its resident state leaves no registers
  // for the precomputed offsets (holding them pushes values into scratch).
  constexpr bool kFullCopies = !(CAUSAL && WPE == 1);
  const typename DR::FullOffsets fo_r = DR::full_offsets(ts, wave, lane);
  const typename DT::FullOffsets fo_t = DT::full_offsets(ts, wave, lane);
  auto issue_tile = [&](int it) DCP_INLINE {
    const unsigned st = unsigned(it) % NSTAGE;
    const int q0 = q_begin + tile_of(it) * BM;
    const int valid = seqlen - q0;
    const __bf16* qs = qh + int64_t(q0) * ts;
    const __bf16* ds = doh + int64_t(q0) * ts;
    if (kFullCopies && valid >= BM) {
      DR::issue_full(&Qr[st * RBUF], qs, fo_r, wave);
      if constexpr (!ONECOPY) DT::issue_full(&Qt[st * TBUF], qs, fo_t, wave);
      DR::issue_full(&dOr[st * RBUF], ds, fo_r, wave);
      if constexpr (!ONECOPY) DT::issue_full(&dOt[st * TBUF], ds, fo_t, wave);
    } else {
      DR::issue(&Qr[st * RBUF], qs, ts, valid, zero, zero, wave, lane);
      if constexpr (!ONECOPY) DT::issue(&Qt[st * TBUF], qs, ts, valid, zero, zero, wave, lane);
      DR::issue(&dOr[st * RBUF], ds, ts, valid, zero, zero, wave, lane);
      if constexpr (!ONECOPY) DT::issue(&dOt[st * TBUF], ds, ts, valid, zero, zero, wave, lane);
    }
    // A query past the sequence end gets LSE = +inf, so its P is exactly 0.
    DL::issue(&LV[st * 2 * BM], lseh + q0, ndh + q0, valid, finf, fzero, wave, lane);
  };
  // Waits until tile it+1 has landed (the tiles after it may stay in flight).
  auto wait_next = [&](int it) DCP_INLINE {
    if (NSTAGE >= 4 && it + 3 < n_qt)
      wait_vmcnt<2 * NI>();
    else if (NSTAGE >= 3 && it + 2 < n_qt)
      wait_vmcnt<NI>();
    else
      wait_vmcnt<0>();
  };

  f32x16 dk_acc[KB][NDB], dv_acc[KB][NDB];
#pragma unroll
  for (int kb = 0; kb < KB; ++kb)
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      dk_acc[kb][db] = f32x16{};
      dv_acc[kb][db] = f32x16{};
    }
  // KV16: [key block][16-key half][16-column block]
  constexpr int NMB = S::NMB;
  f32x4 dk16[KB][2][NMB], dv16[KB][2][NMB];
#pragma unroll
  for (int kb = 0; kb < KB; ++kb)
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
      for (int nb = 0; nb < NMB; ++nb) dk16[kb][mb][nb] = dv16[kb][mb][nb] = f32x4{};

  for (int i = 0; i < NSTAGE - 1 && i < n_qt; ++i) issue_tile(i);
  wait_next(-1);
  __syncthreads();

  // This lane's element offsets inside a tile: 16-byte row reads (A
  // operands) and transposing reads (see lds_read_tr); every other term is
  // a compile-time constant.
  const unsigned ar_off = j * RSTR + 8 * g;
  // (KV16: lane group g4 reads the query runs starting at 0, 16, 4, 20
  // and 8 further, matching to_mfma16_layout)
  const int g4 = lane >> 4;
  const unsigned tr_off =
      S::KV16 ? (16 * (g4 & 1) + 4 * (g4 >> 1) + ((lane & 15) >> 2)) * TSTR + 4 * (lane & 3)
              : (4 * g + ((lane & 15) >> 2)) * TSTR + 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
  const lds_bf16* Qr3 = lds_ptr(Qr);
  const lds_bf16* dOr3 = lds_ptr(dOr);
  const lds_bf16* Qt3 = ONECOPY ? Qr3 : lds_ptr(Qt);
  const lds_bf16* dOt3 = ONECOPY ? dOr3 : lds_ptr(dOt);
  const lds_f32* LV3 = lds_ptr(LV);
  const lds_bf16* Vl3 = lds_ptr(Vl);
  // (VLDS) lane (g, j) reads key 32*(KB*wave + kb) + j, columns 16*kd + 8*g
  const unsigned vl_off = (32 * KB * wave + j) * VLSTR + 8 * g;
  constexpr unsigned TBUF_R = ONECOPY ? RBUF : TBUF;  // stage size of the transposing-read copies

  // (fused) this lane's four 8-byte slots of the dS^T buffer of tile it:
  // key 32*wave + j, queries 8b + 4g .. +3 for b = 0..3 at bf16x4 index 2b
  typedef DCP_LDS bf16x4 lds_bf16x4;
  auto ds_slots = [&](int it) DCP_INLINE {
    return (lds_bf16x4*)(lds_ptr(dSt) + (unsigned(it) & 1u) * DSBUF + (32 * wave + j) * BM + 4 * g);
  };
  // (fused) a wavefront with no work in tile it still owns its rows of dS^T
  auto zero_ds = [&](int it) DCP_INLINE {
    if constexpr (FUSED) {
      lds_bf16x4* row = ds_slots(it);
#pragma unroll
      for (int b = 0; b < 4; ++b) row[2 * b] = bf16x4{};
    }
  };
  // (fused) dQ of tile it once every wavefront's dS^T is in LDS, as dQ^T =
  // K^T dS^T in 16x16 blocks: block x = (16-column block nd, 16-query half
  // mq) goes to wavefront x % NW.  A = K^T (columns x keys) and B = dS^T
  // (keys x queries) both come from transposing reads of key-major rows,
  // with the contraction index of lane group g4 = keys 32*ks + 8*g4 .. +7
  // on both sides; lane (g4, i) ends with query 16*mq + i, columns
  // 16*nd + 4*g4 .. +3 (one 8-byte store).
  __bf16* dqh = dq + int64_t(u.seq0) * ts + int64_t(h) * D;
  auto dq_phase = [&](int it) DCP_INLINE {
    if constexpr (FUSED) {
      const int q0 = q_begin + it * BM;
      const int l16 = lane & 15, g4q = lane >> 4;
      const lds_bf16* ds3 = lds_ptr(dSt) + (unsigned(it) & 1u) * DSBUF + (8 * g4q + (l16 >> 2)) * BM + 4 * (l16 & 3);
      const lds_bf16* kt3 = lds_ptr(Kt) + (8 * g4q + (l16 >> 2)) * KTSTR + 4 * (l16 & 3);
      for (int x = wave; x < 2 * NMQ; x += NW) {
        const int nd = x >> 1, mq = x & 1;
        f32x4 acc = {};
#pragma unroll
        for (int ks = 0; ks < NW; ++ks) {
          const lds_bf16* pk = kt3 + 32 * ks * KTSTR + 16 * nd;
          const lds_bf16* pd = ds3 + 32 * ks * BM + 16 * mq;
          acc = mfma16(cat(lds_read_tr(pk), lds_read_tr(pk + 4 * KTSTR)), cat(lds_read_tr(pd), lds_read_tr(pd + 4 * BM)),
                       acc);
        }
        const int qq = q0 + 16 * mq + l16;
        const int d0 = 16 * nd + 4 * g4q;
        if (qq < seqlen && d0 < D) {
          bf16x4 w;
#pragma unroll
          for (int r = 0; r < 4; ++r) w[r] = __bf16(acc[r] * scale);
          *reinterpret_cast<bf16x4*>(dqh + int64_t(qq) * ts + d0) = w;
        }
      }
    }
  };
  int ds_it = 0;  // (fused) the tile whose dS^T process_block writes

  // One 32-query block (first query qa, sequence-relative) of stage st
  // against this wavefront's 32*KB keys.  MASK 1 applies the causal mask,
  // 2 also each key's sequence bounds (packed windows).
  auto process_block = [&](unsigned st, int qb, int qa, auto mask_tag) DCP_INLINE {
    constexpr int MASK = decltype(mask_tag)::value;
    unsigned rb = st * RBUF + 32 * qb * RSTR + ar_off;
    unsigned tb = st * TBUF_R + 32 * qb * TSTR + tr_off;
    unsigned lb = st * 2 * BM + 32 * qb + 4 * g;
    unsigned vb = vl_off;
    // Opaque to the optimizer: each read below is then one of these bases
    // plus a constant, which folds into the instruction's offset field
    // (otherwise every read's address is rebuilt with vector arithmetic).
    asm("" : "+v"(rb), "+v"(tb), "+v"(lb), "+v"(vb));
    if constexpr (VLDS) {
      // Two wavefronts per SIMD: besides the dK, dV accumulators and the K
      // fragments only S, dP and the operands of the current 16-column step
      // stay live (V, Q and dO fragments are read where they are used, LSE
      // per 4-query group).
      // (no issue-priority raise here: with two wavefronts per SIMD it cost
      // about 1 % of the pass)
      // the dP accumulator starts at -Delta (the registers dP needs anyway)
      f32x16 sv = f32x16{}, dpv;
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        const f32x4 t = lds_read_f32x4(LV3 + lb + BM + 8 * b);
#pragma unroll
        for (int c = 0; c < 4; ++c) dpv[4 * b + c] = t[c];
      }
      // The Q, dO and V fragments of step kd + 1 are read while step kd's
      // products run (held in that order by scheduling fences).
      bf16x8 fq[NKD], fo[NKD], fv[NKD];
      auto fetch = [&](int kd) DCP_INLINE {
        fq[kd] = lds_read_b128(Qr3 + rb + 16 * kd);
        fo[kd] = lds_read_b128(dOr3 + rb + 16 * kd);
        fv[kd] = lds_read_b128(Vl3 + vb + 16 * kd);
      };
      fetch(0);
#pragma unroll
      for (int kd = 0; kd < NKD; ++kd) {
        if (kd + 1 < NKD) fetch(kd + 1);
        __builtin_amdgcn_sched_barrier(0);
        sv = mfma32(fq[kd], kf[0][kd], sv);
        dpv = mfma32(fo[kd], fv[kd], dpv);
        __builtin_amdgcn_sched_barrier(0);
      }
      const int key = wave_key_lo + j;
      bf16x8 pa2[2], da2[2];
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        const f32x4 l = lds_read_f32x4(LV3 + lb + 8 * b);
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          const int r = 4 * b + c;
          float p = __builtin_amdgcn_exp2f(fmaf(sv[r], scale_log2, -l[c]));
          const int qq = qa + 8 * b + 4 * g + c;
          if (MASK == 1 && key > qq) p = 0.f;
          if (MASK == 2 && (unsigned(qq - q_lo[0]) >= unsigned(q_hi[0] - q_lo[0]) || (CAUSAL && key > qq))) p = 0.f;
          pa2[b >> 1][4 * (b & 1) + c] = __bf16(p);
          da2[b >> 1][4 * (b & 1) + c] = __bf16(p * dpv[r]);
        }
      }
      mfma_prio_hi();
      // The transposed operands are read one product ahead: Q's for step n
      // while dV's product of step n runs, dO's for step n + 1 while dK's
      // product of step n runs (steps n = (db, hh)).
      auto operand = [&](const lds_bf16* t3, int n) DCP_INLINE {
        const unsigned o = tb + 16 * (n & 1) * TSTR + 32 * (n >> 1);
        return cat(lds_read_tr(t3 + o), lds_read_tr(t3 + o + 8 * TSTR));
      };
      // (scheduling fences keep this order: left alone, the compiler issues
      // each product right behind its own reads and waits on them)
      bf16x8 bd = operand(dOt3, 0);
#pragma unroll
      for (int n = 0; n < 2 * NDB; ++n) {
        const int db = n >> 1, hh = n & 1;
        const bf16x8 bq = operand(Qt3, n);
        __builtin_amdgcn_sched_barrier(0);
        dv_acc[0][db] = mfma32(pa2[hh], bd, dv_acc[0][db]);
        if (n + 1 < 2 * NDB) bd = operand(dOt3, n + 1);
        __builtin_amdgcn_sched_barrier(0);
        dk_acc[0][db] = mfma32(da2[hh], bq, dk_acc[0][db]);
      }
      mfma_prio_lo();
      return;
    }
    bf16x8 aq[NKD], ado[NKD];
#pragma unroll
    for (int kd = 0; kd < NKD; ++kd) {
      aq[kd] = lds_read_b128(Qr3 + rb + 16 * kd);
      ado[kd] = lds_read_b128(dOr3 + rb + 16 * kd);
    }
    // Lane (g, j) of an S / dP accumulator holds key j of its key block
    // against queries qa + 8b + 4g + c (register 4b + c).
    f32x16 nd;
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const f32x4 t = lds_read_f32x4(LV3 + lb + BM + 8 * b);
#pragma unroll
      for (int c = 0; c < 4; ++c) nd[4 * b + c] = t[c];
    }
    f32x16 s[KB], dp[KB];
    mfma_prio_hi();
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      s[kb] = f32x16{};
#pragma unroll
      for (int kd = 0; kd < NKD; ++kd) s[kb] = mfma32(aq[kd], kf[kb][kd], s[kb]);
      dp[kb] = nd;
#pragma unroll
      for (int kd = 0; kd < NKD; ++kd)
        dp[kb] = mfma32(ado[kd], VLDS ? lds_read_b128(Vl3 + vb + 32 * kb * VLSTR + 16 * kd) : vf[kb][kd], dp[kb]);
    }
    mfma_prio_lo();
    f32x4 l4[4];
#pragma unroll
    for (int b = 0; b < 4; ++b) l4[b] = lds_read_f32x4(LV3 + lb + 8 * b);
    bf16x8 pa[KB][2], da[KB][2];
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      const int key = wave_key_lo + 32 * kb + j;
#pragma unroll
      for (int b = 0; b < 4; ++b)
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          const int r = 4 * b + c;
          float p = __builtin_amdgcn_exp2f(fmaf(s[kb][r], scale_log2, -l4[b][c]));
          const int qq = qa + 8 * b + 4 * g + c;
          if (MASK == 1 && key > qq) p = 0.f;
          if (MASK == 2 && (unsigned(qq - q_lo[kb]) >= unsigned(q_hi[kb] - q_lo[kb]) || (CAUSAL && key > qq)))
            p = 0.f;
          pa[kb][b >> 1][4 * (b & 1) + c] = __bf16(p);
          da[kb][b >> 1][4 * (b & 1) + c] = __bf16(p * dp[kb][r]);
        }
    }
    if constexpr (FUSED) {
      lds_bf16x4* row = ds_slots(ds_it);
#pragma unroll
      for (int b = 0; b < 4; ++b)
        row[2 * b] = bf16x4{da[0][b >> 1][4 * (b & 1)], da[0][b >> 1][4 * (b & 1) + 1], da[0][b >> 1][4 * (b & 1) + 2],
                            da[0][b >> 1][4 * (b & 1) + 3]};
    }
    if constexpr (S::KV16) {
      // dV += P^T dO and dK += dS^T Q in 16x16 blocks: each B fragment (16
      // columns of dO or Q over the block's 32 queries) feeds both 16-key
      // halves.
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) {
        to_mfma16_layout(pa[kb][0], pa[kb][1]);
        to_mfma16_layout(da[kb][0], da[kb][1]);
      }
      mfma_prio_hi();
#pragma unroll
      for (int nb = 0; nb < NMB; ++nb) {
        const unsigned o = tb + 16 * nb;
        const bf16x8 bd = cat(lds_read_tr(dOt3 + o), lds_read_tr(dOt3 + o + 8 * TSTR));
        const bf16x8 bqq = cat(lds_read_tr(Qt3 + o), lds_read_tr(Qt3 + o + 8 * TSTR));
#pragma unroll
        for (int kb = 0; kb < KB; ++kb)
#pragma unroll
          for (int mb = 0; mb < 2; ++mb) {
            dv16[kb][mb][nb] = mfma16(pa[kb][mb], bd, dv16[kb][mb][nb]);
            dk16[kb][mb][nb] = mfma16(da[kb][mb], bqq, dk16[kb][mb][nb]);
          }
      }
      mfma_prio_lo();
      return;
    }
    // dV += P^T dO and dK += dS^T Q: B = rows (queries) x columns (d),
    // fetched column-wise with transposing reads, shared by the key blocks.
    bf16x8 bdo[NDB][2], bq[NDB][2];
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        const unsigned o = tb + 16 * hh * TSTR + 32 * db;
        bdo[db][hh] = cat(lds_read_tr(dOt3 + o), lds_read_tr(dOt3 + o + 8 * TSTR));
        bq[db][hh] = cat(lds_read_tr(Qt3 + o), lds_read_tr(Qt3 + o + 8 * TSTR));
      }
    mfma_prio_hi();
#pragma unroll
    for (int kb = 0; kb < KB; ++kb)
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
          dv_acc[kb][db] = mfma32(pa[kb][hh], bdo[db][hh], dv_acc[kb][db]);
          dk_acc[kb][db] = mfma32(da[kb][hh], bq[db][hh], dk_acc[kb][db]);
        }
    mfma_prio_lo();
  };

  // Query tiles are walked in two phases per wavefront: (causal, from the
  // sequence end) those needing no mask, then those reaching its keys,
  // where 32-query blocks entirely before its keys are skipped and blocks
  // crossing them masked.  Every iteration runs the same copy / wait /
  // barrier sequence.
  // (packed windows: the queries of this wavefront's keys' sequences)
  const int last_key = min(32 * KB - 1, int(u.rows) - 1 - 32 * KB * wave);  // of the wavefront, tile-relative
  const int wq_lo = packed ? (CAUSAL ? wave_key_lo : __builtin_amdgcn_readfirstlane(q_lo[0])) : 0;
  const int wq_hi = packed ? __builtin_amdgcn_readlane(q_hi[KB - 1], max(last_key, 0) % 32) : seqlen;
  auto run = [&](int it0, int it1, auto mask_tag) DCP_INLINE {
    constexpr int MASK = decltype(mask_tag)::value;
    for (int it = it0; it < it1; ++it) {
      if (it + NSTAGE - 1 < n_qt) issue_tile(it + NSTAGE - 1);
      const unsigned st = unsigned(it) % NSTAGE;
      const int q0 = q_begin + tile_of(it) * BM;
      ds_it = it;
#pragma unroll
      for (int qb = 0; qb < BM / 32; ++qb) {
        const int qa = q0 + 32 * qb;
        if (qa >= seqlen) {  // padding rows of the last tile
          zero_ds(it);
          continue;
        }
        if (MASK == 1) {
          if (qa + 31 < wave_key_lo) continue;  // every query precedes every key
          // (V from LDS: one block body per loop keeps the accumulators in
          // place; the mask costs a compare per element on these few tiles)
          if (!VLDS && qa >= wave_key_lo + 32 * KB - 1) {
            process_block(st, qb, qa, std::integral_constant<int, 0>{});
            continue;
          }
        }
        if (MASK == 2 && (qa + 31 < wq_lo || qa >= wq_hi)) {  // no query of these keys' sequences
          zero_ds(it);
          continue;
        }
        process_block(st, qb, qa, std::integral_constant<int, MASK>{});
      }
      wait_next(it);
      __syncthreads();
      dq_phase(it);
    }
  };
  // no key of this wavefront in the tile: copies and barriers only (and,
  // fused, zero dS^T rows and a share of the tile's dQ)
  auto idle = [&](int it0, int it1) DCP_INLINE {
    for (int it = it0; it < it1; ++it) {
      if (it + NSTAGE - 1 < n_qt) issue_tile(it + NSTAGE - 1);
      zero_ds(it);
      wait_next(it);
      __syncthreads();
      dq_phase(it);
    }
  };
  if (32 * KB * wave < u.rows) {
    if constexpr (packed) {
      const int it_lo = (wq_lo - q_begin) / BM;
      const int it_hi = min(n_qt, (wq_hi - q_begin + BM - 1) / BM);
      idle(0, it_lo);
      run(it_lo, it_hi, std::integral_constant<int, 2>{});
      idle(it_hi, n_qt);
    } else {
      if (CAUSAL) {
        // the tiles whose queries all follow all of this wavefront's keys
        // (from the end), then those crossing or preceding them
        const int t_plain = min(n_qt, max(0, (wave_key_lo + 32 * KB - 1 - q_begin + BM - 1) / BM));
        run(0, n_qt - t_plain, std::integral_constant<int, 0>{});
        run(n_qt - t_plain, n_qt, std::integral_constant<int, 1>{});
      } else {
        run(0, n_qt, std::integral_constant<int, 0>{});
      }
    }
  } else {
    idle(0, n_qt);  // no key of the tile (the last tile of a sequence)
  }


  // Epilogue through LDS (the ring is idle now): the workgroup's first half
  // of 32-key blocks is staged in the Q buffers, the second in the dO
  // buffers, dK first, then dV.
#pragma unroll
  for (int kb = 0; kb < KB; ++kb) {
    const int sb = KB * wave + kb;
    const int key0 = 32 * sb;
    __bf16* stage = sb < NSB / 2 ? Qr + sb * 32 * SSTR : dOr + (sb - NSB / 2) * 32 * SSTR;
    const int n_rows = max(0, min(32, u.rows - key0));
    __bf16* dk_base = dk + int64_t(u.row0 + key0) * ts + int64_t(h) * D;
    __bf16* dv_base = dv + int64_t(u.row0 + key0) * ts + int64_t(h) * D;
    if constexpr (S::KV16) {
      store_rows16_bf16<D, NMB>(dk16[kb], scale, stage, SSTR, dk_base, ts, n_rows, lane);
      store_rows16_bf16<D, NMB>(dv16[kb], 1.f, stage, SSTR, dv_base, ts, n_rows, lane);
    } else {
      store_rows_bf16<D, NDB>(dk_acc[kb], scale, stage, SSTR, dk_base, ts, n_rows, lane);
      store_rows_bf16<D, NDB>(dv_acc[kb], 1.f, stage, SSTR, dv_base, ts, n_rows, lane);
    }
  }
}

// ---------------------------------------------------------------------------
// 3. dQ (query-stationary).
//
// Each wavefront keeps 32 queries' Q and dO fragments (B operands), their
// LSE*log2e and -Delta in registers while key tiles of BN rows stream
// through an NSTAGE-deep LDS ring filled by direct global-to-LDS copies
// NSTAGE - 1 tiles ahead (K twice: rows read 16 B per lane for S^T, rows
// read by transposing reads for dQ^T; V once), one barrier per tile.  With
// ONECOPY, K is held once, at the row-read stride, and the transposing
// reads use that copy.
template <int D, int NW, int NSTAGE, bool CAUSAL, bool PACKED, bool ONECOPY>
__global__ __launch_bounds__(64 * NW) void attn_bwd_dq_kernel(
    const __bf16* __restrict__ q, const __bf16* __restrict__ k, const __bf16* __restrict__ v,
    const __bf16* __restrict__ dout, const float* __restrict__ lse2, const float* __restrict__ ndelta,
    __bf16* __restrict__ dq, const __bf16* __restrict__ consts, const WorkUnit* __restrict__ units,
    const uint64_t* __restrict__ window_starts, int per_xcd, int H, int T, float scale, float scale_log2) {
  using S = BwdShape<D>;
  constexpr int NKD = S::NKD, NDB = S::NDB, CPR = S::CPR;
  constexpr int KSTR = ONECOPY ? S::OSTR : S::DP + 8;  // K and V rows read 16 B per lane (and K transposed)
  constexpr int TSTR = ONECOPY ? KSTR : S::TSTR;  // (second copy of K for transposing reads)
  constexpr int BN = kBwdDqBN;
  constexpr int KBUF = BN * KSTR, TBUF = ONECOPY ? 0 : BN * TSTR;
  using DK = DmaTile<BN, KSTR / 8, CPR, NW>;
  using DT = DmaTile<BN, TSTR / 8, CPR, NW>;
  constexpr int NI = ONECOPY ? 2 * DK::NI : 2 * DK::NI + DT::NI;  // copies per wavefront per tile

  __shared__ __attribute__((aligned(16))) __bf16 Ks[NSTAGE * KBUF];
  __shared__ __attribute__((aligned(16))) __bf16 Vs[NSTAGE * KBUF];
  __shared__ __attribute__((aligned(16))) __bf16 Kt[ONECOPY ? 8 : NSTAGE * TBUF];
  static_assert(NSTAGE >= 2 && NSTAGE <= 4, "ring depth");
  static_assert(2 * NI < 64, "vmcnt range");

  const WorkUnit u = unit_for_block(units, per_xcd);
  if (u.rows == 0) return;
  const int h = u.head;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: scalar branches on it
  const int g = lane >> 5;
  const int j = lane & 31;
  const int64_t ts = int64_t(H) * D;
  constexpr bool packed = PACKED;  // a list of packed windows only
  const int seqlen = packed ? int(u.rows) : u.seqlen;  // (window-relative offsets when packed)
  const int tile_q0 = u.row0 - u.seq0;
  const int wave_q0 = tile_q0 + 32 * wave;
  const __bf16* zero = consts + kConstZero;

  const __bf16* qh = q + int64_t(u.seq0) * ts + int64_t(h) * D;
  const __bf16* kh = k + int64_t(u.seq0) * ts + int64_t(h) * D;
  const __bf16* vh = v + int64_t(u.seq0) * ts + int64_t(h) * D;
  const __bf16* doh = dout + int64_t(u.seq0) * ts + int64_t(h) * D;

  // Per-lane query state: Q and dO fragments (B operands), LSE, -Delta.
  const int qrel = 32 * wave + j;
  const bool q_ok = qrel < u.rows;
  const int my_q = tile_q0 + qrel;  // sequence-relative
  // keys of this lane's sequence: [k_lo, k_hi)
  int k_lo = 0, k_hi = seqlen;
  if (packed)
    window_bounds(window_starts + kWindowWords * (-u.seqlen - 1), min(my_q, seqlen - 1), seqlen, k_lo, k_hi);
  bf16x8 qf[NKD], df[NKD];
#pragma unroll
  for (int kd = 0; kd < NKD; ++kd) {
    const int col = 16 * kd + 8 * g;
    if (q_ok && col < D) {
      qf[kd] = *reinterpret_cast<const bf16x8*>(qh + int64_t(my_q) * ts + col);
      df[kd] = *reinterpret_cast<const bf16x8*>(doh + int64_t(my_q) * ts + col);
    } else {
      qf[kd] = bf16x8{};
      df[kd] = bf16x8{};
    }
  }
  const float lse_l2 = q_ok ? lse2[int64_t(h) * T + u.seq0 + my_q] : INFINITY;
  const float ndlt = q_ok ? ndelta[int64_t(h) * T + u.seq0 + my_q] : 0.f;
  // -Delta as the initial dP^T accumulator, so the products yield
  // dP^T - Delta (at head width 128 the 16 registers it takes are not
  // spare: there the difference is taken per element instead).
  constexpr bool FOLD = D <= 96;
  f32x16 nd_init;
#pragma unroll
  for (int r = 0; r < 16; ++r) nd_init[r] = FOLD ? ndlt : 0.f;
  wait_vmcnt<0>();  // settle the fragment loads before the first copy

  const int key_end = CAUSAL ? min(seqlen, tile_q0 + u.rows) : seqlen;
  const int n_tiles = (key_end + BN - 1) / BN;

  const typename DK::FullOffsets fo_k = DK::full_offsets(ts, wave, lane);
  const typename DT::FullOffsets fo_t = DT::full_offsets(ts, wave, lane);
  auto issue_tile = [&](int kt) DCP_INLINE {
    const unsigned st = unsigned(kt) % NSTAGE;
    const int valid = seqlen - kt * BN;
    const __bf16* ks = kh + int64_t(kt) * BN * ts;
    if (valid >= BN) {
      DK::issue_full(&Ks[st * KBUF], ks, fo_k, wave);
      DK::issue_full(&Vs[st * KBUF], vh + int64_t(kt) * BN * ts, fo_k, wave);
      if constexpr (!ONECOPY) DT::issue_full(&Kt[st * TBUF], ks, fo_t, wave);
    } else {
      DK::issue(&Ks[st * KBUF], ks, ts, valid, zero, zero, wave, lane);
      DK::issue(&Vs[st * KBUF], vh + int64_t(kt) * BN * ts, ts, valid, zero, zero, wave, lane);
      if constexpr (!ONECOPY) DT::issue(&Kt[st * TBUF], ks, ts, valid, zero, zero, wave, lane);
    }
  };
  // Before the barrier that ends tile kt: tile kt+1 must have landed; the
  // later tiles' copies may still be in flight.
  auto wait_next = [&](int kt) DCP_INLINE {
    if (NSTAGE >= 4 && kt + 3 < n_tiles)
      wait_vmcnt<2 * NI>();
    else if (NSTAGE >= 3 && kt + 2 < n_tiles)
      wait_vmcnt<NI>();
    else
      wait_vmcnt<0>();
  };

  f32x16 acc[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) acc[db] = f32x16{};
  // KV16: dQ^T in 16x16 blocks [d block][query block]; lane (g4, n) holds
  // query 16 * qb + n, columns 16 * mb + 4 * g4 + {0..3}
  constexpr int NMB = S::NMB;
  f32x4 acc16[NMB][2];
#pragma unroll
  for (int mb = 0; mb < NMB; ++mb) acc16[mb][0] = acc16[mb][1] = f32x4{};

  for (int i = 0; i < NSTAGE - 1 && i < n_tiles; ++i) issue_tile(i);
  wait_next(-1);
  __syncthreads();

  const unsigned ar_off = j * KSTR + 8 * g;
  // (KV16: lane group g4 reads the key runs starting at 0, 16, 4, 20 and 8
  // further, matching to_mfma16_layout)
  const int g4 = lane >> 4;
  const unsigned tr_off =
      S::KV16 ? (16 * (g4 & 1) + 4 * (g4 >> 1) + ((lane & 15) >> 2)) * TSTR + 4 * (lane & 3)
              : (4 * g + ((lane & 15) >> 2)) * TSTR + 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
  const lds_bf16* Ks3 = lds_ptr(Ks);
  const lds_bf16* Vs3 = lds_ptr(Vs);
  const lds_bf16* Kt3 = ONECOPY ? Ks3 : lds_ptr(Kt);
  constexpr unsigned TBUF_R = ONECOPY ? KBUF : TBUF;  // stage size of the transposing-read copy
  const int wave_last_q = wave_q0 + 31;

  // One key tile against this wavefront's 32 queries.  MASK covers tiles
  // crossing the sequence end or the causal diagonal.
  auto process_tile = [&](unsigned st, int k0, auto mask_tag) DCP_INLINE {
    constexpr bool MASK = decltype(mask_tag)::value;
    unsigned rb = st * KBUF + ar_off;
    unsigned tb = st * TBUF_R + tr_off;
    asm("" : "+v"(rb), "+v"(tb));  // keeps the constant terms in the offset fields
    f32x16 s[BN / 32], dp[BN / 32];
#pragma unroll
    for (int kb = 0; kb < BN / 32; ++kb) {
      s[kb] = f32x16{};
      dp[kb] = FOLD ? nd_init : f32x16{};
    }
    mfma_prio_hi();
    // The K and V fragments of step kd + 1 are read while step kd's products
    // run (held in that order by scheduling fences).
    bf16x8 fk[NKD][BN / 32], fv[NKD][BN / 32];
    auto fetch = [&](int kd) DCP_INLINE {
#pragma unroll
      for (int kb = 0; kb < BN / 32; ++kb) {
        fk[kd][kb] = lds_read_b128(Ks3 + rb + 32 * kb * KSTR + 16 * kd);
        fv[kd][kb] = lds_read_b128(Vs3 + rb + 32 * kb * KSTR + 16 * kd);
      }
    };
    fetch(0);
#pragma unroll
    for (int kd = 0; kd < NKD; ++kd) {
      if (kd + 1 < NKD) fetch(kd + 1);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int kb = 0; kb < BN / 32; ++kb) {
        s[kb] = mfma32(fk[kd][kb], qf[kd], s[kb]);
        dp[kb] = mfma32(fv[kd][kb], df[kd], dp[kb]);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    mfma_prio_lo();
    // Lane (g, j) holds query j against keys k0 + 32kb + 8(r/4) + 4g + r%4.
    bf16x8 dsb[BN / 32][2];
#pragma unroll
    for (int kb = 0; kb < BN / 32; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float p = __builtin_amdgcn_exp2f(fmaf(s[kb][r], scale_log2, -lse_l2));
        if constexpr (MASK) {
          const int key = k0 + 32 * kb + 8 * (r >> 2) + 4 * g + (r & 3);
          if (unsigned(key - k_lo) >= unsigned(k_hi - k_lo) || (CAUSAL && key > my_q)) p = 0.f;
        }
        dsb[kb][r >> 3][r & 7] = __bf16(p * (FOLD ? dp[kb][r] : dp[kb][r] + ndlt));
      }
    if constexpr (S::KV16) {
      // dQ^T += K^T dS^T in 16x16 blocks: each A fragment (16 rows of K^T
      // over the block's 32 keys) feeds both 16-query halves.
#pragma unroll
      for (int kb = 0; kb < BN / 32; ++kb) to_mfma16_layout(dsb[kb][0], dsb[kb][1]);
      mfma_prio_hi();
#pragma unroll
      for (int kb = 0; kb < BN / 32; ++kb)
#pragma unroll
        for (int mb = 0; mb < NMB; ++mb) {
          const unsigned o = tb + 32 * kb * TSTR + 16 * mb;
          const bf16x8 a = cat(lds_read_tr(Kt3 + o), lds_read_tr(Kt3 + o + 8 * TSTR));
          acc16[mb][0] = mfma16(a, dsb[kb][0], acc16[mb][0]);
          acc16[mb][1] = mfma16(a, dsb[kb][1], acc16[mb][1]);
        }
      mfma_prio_lo();
      return;
    }
    // dQ^T += K^T dS^T: A = K^T (rows d, keys 32kb + 16hh + 4g + {0..3, 8..11}).
    mfma_prio_hi();
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int kb = 0; kb < BN / 32; ++kb)
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
          const unsigned o = tb + (32 * kb + 16 * hh) * TSTR + 32 * db;
          const bf16x8 a = cat(lds_read_tr(Kt3 + o), lds_read_tr(Kt3 + o + 8 * TSTR));
          acc[db] = mfma32(a, dsb[kb][hh], acc[db]);
        }
    mfma_prio_lo();
  };

  // Key tiles in up to three phases per wavefront (unmasked, masked, idle),
  // each with the same copy / wait / barrier sequence.  A wavefront holding
  // no query of the tile (the last tile of a sequence) only idles.  In a
  // packed window every tile is masked, and the tiles before the first
  // query's sequence (t_lead) and after the last one's are idle.
  int t_lead = 0;
  int t_mask = min(n_tiles, seqlen / BN);
  int t_idle = n_tiles;
  if (CAUSAL) {
    t_mask = min(t_mask, (wave_q0 + 1) / BN);
    t_idle = min(n_tiles, wave_last_q / BN + 1);
  }
  if constexpr (packed) {
    const int last = min(31, int(u.rows) - 1 - 32 * wave);  // lane of the wavefront's last query
    const int keys_end = min(__builtin_amdgcn_readlane(k_hi, max(last, 0)), CAUSAL ? wave_q0 + 32 : seqlen);
    t_lead = t_mask = __builtin_amdgcn_readfirstlane(k_lo) / BN;
    t_idle = min(n_tiles, (keys_end + BN - 1) / BN);
  }
  if (32 * wave >= u.rows) t_lead = t_mask = t_idle = 0;
  auto run = [&](int kt0, int kt1, auto mode_tag) DCP_INLINE {
    constexpr int MODE = decltype(mode_tag)::value;  // 0 unmasked, 1 masked, 2 idle
    for (int kt = kt0; kt < kt1; ++kt) {
      if (kt + NSTAGE - 1 < n_tiles) issue_tile(kt + NSTAGE - 1);
      const unsigned st = unsigned(kt) % NSTAGE;
      if constexpr (MODE == 0) process_tile(st, kt * BN, std::false_type{});
      if constexpr (MODE == 1) process_tile(st, kt * BN, std::true_type{});
      wait_next(kt);
      __syncthreads();
    }
  };
  run(0, t_lead, std::integral_constant<int, 2>{});
  run(t_lead, t_mask, std::integral_constant<int, 0>{});
  run(t_mask, t_idle, std::integral_constant<int, 1>{});
  run(t_idle, n_tiles, std::integral_constant<int, 2>{});

  if constexpr (S::KV16) {
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
      const int qr = 32 * wave + 16 * qb + (lane & 15);
      if (qr < u.rows) {
        __bf16* qrow = dq + int64_t(u.row0 + qr) * ts + int64_t(h) * D;
#pragma unroll
        for (int mb = 0; mb < NMB; ++mb) {
          const int d0 = 16 * mb + 4 * g4;
          if (d0 < D) {
            bf16x4 w;
#pragma unroll
            for (int c = 0; c < 4; ++c) w[c] = __bf16(acc16[mb][qb][c] * scale);
            *reinterpret_cast<bf16x4*>(qrow + d0) = w;
          }
        }
      }
    }
    return;
  }
  // Epilogue: lane (g, j) holds query j, columns 32db + 8rb + 4g + {0..3}.
  if (q_ok) {
    __bf16* qrow = dq + int64_t(u.seq0 + my_q) * ts + int64_t(h) * D;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int rb = 0; rb < 4; ++rb) {
        const int d0 = 32 * db + 8 * rb + 4 * g;
        if (d0 < D) {
          bf16x4 w;
#pragma unroll
          for (int c = 0; c < 4; ++c) w[c] = __bf16(acc[db][4 * rb + c] * scale);
          *reinterpret_cast<bf16x4*>(qrow + d0) = w;
        }
      }
  }
}

template <int D, bool CAUSAL, bool PACKED, bool FUSED = false>
hipError_t launch_dkdv_list(const BwdArgs& a, const WorkUnit* units, int n_units) {
  constexpr DkdvShape sh = PACKED ? bwd_dkdv_window_shape(D) : bwd_dkdv_shape(D);
  hipLaunchKernelGGL(
      (attn_bwd_dkdv_kernel<D, sh.kb, sh.waves, sh.bm, sh.stages, sh.waves_per_eu, CAUSAL, PACKED, FUSED,
                            FUSED || sh.onecopy, sh.vlds>),
                     dim3(n_units), dim3(64 * sh.waves), 0, a.stream, static_cast<const __bf16*>(a.q),
                     static_cast<const __bf16*>(a.k), static_cast<const __bf16*>(a.v),
                     static_cast<const __bf16*>(a.dout), a.lse2, a.ndelta, static_cast<__bf16*>(a.dk),
                     static_cast<__bf16*>(a.dv), static_cast<__bf16*>(a.dq), static_cast<const __bf16*>(a.consts), units,
                     static_cast<const uint64_t*>(a.window_starts), n_units / kNumXcd, a.n_heads, a.total_tokens,
                     a.scale, a.scale * kLog2e);
  return hipGetLastError();
}

template <int D, bool CAUSAL, bool PACKED>
hipError_t launch_dq_list(const BwdArgs& a, const WorkUnit* units, int n_units) {
  constexpr int NW = PACKED ? kWinDqWaves : kBwdDqWaves;
  constexpr int NS = D > 96 ? kBwdDqStagesD128 : (PACKED ? kWinDqStages : kBwdDqStages);
  hipLaunchKernelGGL((attn_bwd_dq_kernel<D, NW, NS, CAUSAL, PACKED, kBwdDqOneCopy>), dim3(n_units), dim3(64 * NW), 0, a.stream, static_cast<const __bf16*>(a.q),
                     static_cast<const __bf16*>(a.k), static_cast<const __bf16*>(a.v),
                     static_cast<const __bf16*>(a.dout), a.lse2, a.ndelta, static_cast<__bf16*>(a.dq),
                     static_cast<const __bf16*>(a.consts), units, static_cast<const uint64_t*>(a.qwindow_starts),
                     n_units / kNumXcd, a.n_heads, a.total_tokens, a.scale, a.scale * kLog2e);
  return hipGetLastError();
}

// Delta, then the dK/dV pass and the dQ pass, each over its sequence tiles
// and then its packed windows (one launch per non-empty list).
template <int D, bool CAUSAL>
hipError_t launch_bwd_t(const BwdArgs& a) {
  if (a.rows_end > 0) {
    const dim3 grid(unsigned((a.rows_end + kDeltaRows - 1) / kDeltaRows),
                    unsigned((a.n_heads + kDeltaHeads - 1) / kDeltaHeads));
    hipLaunchKernelGGL((bwd_delta_kernel<D>), grid, dim3(kDeltaThreads), 0, a.stream,
                       static_cast<const __bf16*>(a.dout), static_cast<const __bf16*>(a.o), a.lse, a.ndelta,
                       a.lse2, a.rows_end, a.n_heads, a.total_tokens);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  const KernelEvents& ev = kernel_events();
  const WorkUnit* units = static_cast<const WorkUnit*>(a.units);
  const WorkUnit* qunits = static_cast<const WorkUnit*>(a.qunits);
  hipError_t e = hipSuccess;
  if (a.n_units + a.n_wunits > 0) {
    if (ev.begin) (void)hipEventRecord(ev.begin, a.stream);
    if (a.n_units > 0) e = launch_dkdv_list<D, CAUSAL, false>(a, units, a.n_units);
    if (e == hipSuccess && a.n_wunits > 0)
      e = launch_dkdv_list<D, CAUSAL, true, bwd_window_fused(D)>(a, units + a.n_units, a.n_wunits);
    if (ev.end) (void)hipEventRecord(ev.end, a.stream);
    if (e != hipSuccess) return e;
  }
  if (a.n_qunits > 0) e = launch_dq_list<D, CAUSAL, false>(a, qunits, a.n_qunits);
  // (windows with fused dQ: their dQ rows were written by the dK/dV pass)
  if (e == hipSuccess && a.n_wqunits > 0 && !bwd_window_fused(D))
    e = launch_dq_list<D, CAUSAL, true>(a, qunits + a.n_qunits, a.n_wqunits);
  return e;
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
