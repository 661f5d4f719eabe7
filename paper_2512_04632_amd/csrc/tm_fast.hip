// bf16 matrix-core path of the Turbo-Muon orthogonalizer for gfx950 (MI355X).
//
// Every matrix is processed in a zero-padded workspace layout whose dims are
// multiples of the square tile T (256, 128 or 64), so every tile is full: the
// main loops carry no bounds checks and zero padding is preserved by the
// iteration (padded rows and columns of Y, A and B stay zero).  A wide matrix
// that needs no padding is read in place by the first iteration.
//
// Phases (one launch each over the tiles of all matrices of a call):
//   k_load_in     W1 = X (wide) or X^T (tall), zero padded
//   k_gram_fast   A = Y Y^T, upper tiles, mirrored bf16 store; at iteration 1
//                 the fp32 accumulators of the upper tiles are stored instead
//                 (A0 is rescaled before rounding) and the epilogue emits the
//                 AOL row sums sum_j |A0_ij| (eq. (aol))
//   k_apply_s     A1 = diag(s) A0 diag(s), rounded once to bf16, from the
//                 upper tiles of A0 (for k <= 1024 it also sums the AOL
//                 vector s from the row partials, in place of a separate
//                 launch)
//   k_poly_fast   B~ = b A + c A A + a I, upper tiles, mirrored store; at
//                 iteration 1 it stores C = B~ diag(s) instead, so that X1 =
//                 diag(s) X0 is never formed: B~ X1 = C X0
//   k_update_fast Y' = B~ Y = a Y + B Y: the axpy of the update rides on B~'s
//                 diagonal, so the update is a single product with no second
//                 read of Y (iteration 1: Y' = C X0)
//
// Main loop: the 256 x 256 tile runs 8 wave64s (two per SIMD, so one wave's
// barrier or DMA issue can hide behind the other's MFMAs) in a 2 x 4 grid of
// 128 x 64 blocks; smaller tiles run 4 compute waves in a 2 x 2 grid (the 32
// tile one), plus producer waves for the Gram and polynomial.  Each wave
// accumulates 16 x 16 blocks with v_mfma_f32_16x16x32_bf16, which carries half
// the accumulator traffic per flop of the 32 x 32 x 16 form and, on random
// bf16 data, keeps the power-limited clock about 14% higher; every tile size
// uses it, so all of them add the same products in the same order.  The 256
// tile's waves multiply a whole 64-wide K stage (96 operand registers next to
// the 128 accumulators) between two barriers.  Operands reach LDS
// through global_load_lds_dwordx4 (direct to LDS, no VGPR staging) into a
// ring of five operand slots of 64 K elements for the 256 tile, three or
// four stages of 32, 64 or 128 for the smaller tiles.  K-contiguous operands
// are stored as rows of 2 BK bytes whose 16-byte chunks are XOR-swizzled by
// row group; the update's Y operand is staged in its row-major layout (BK rows
// of T bf16) with 32-byte chunks XOR-swizzled per row and read with
// ds_read_b64_tr_b16, which hands each lane 4 consecutive K values of one
// column.  Both layouts are free of LDS bank conflicts for the main-loop
// reads.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "tm_internal.h"

namespace tmk {
namespace fast {

// K elements per ring stage of the 8-wave (256) tile: rows of 128 bytes.
constexpr int kPingPongBK = 64;

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef short s16x4_t __attribute__((ext_vector_type(4)));

// Tile T x T computed by NW wave64s in a WGM x WGN grid (2 x 4, 2 x 2, or a
// single wave for the 32 tile); each wave owns TWM x TWN of the output as
// FM x FN blocks of 16 x 16, each accumulated by v_mfma_f32_16x16x32_bf16 (a
// 16 x 16 fp32 block, 4 registers per lane, 32 K values per instruction).
// The smaller tiles' Gram and polynomial add NP producer waves that only
// issue the ring's DMA (mainloop_pc); they leave after the main loop, so the
// epilogues run on the NT threads of the NW compute waves.  (The update's
// smaller tiles keep the DMA in their compute waves: producer waves made
// them slower.)
template <int T>
struct Tile {
  static constexpr int NW = T == 256 ? 8 : (T == 32 ? 1 : 4);   // 2 waves per SIMD for 256
  static constexpr int WGM = NW == 1 ? 1 : 2, WGN = NW / WGM;
  static constexpr int NT = 64 * NW;            // threads of the compute waves
  static constexpr int NP = T == 256 ? 0 : (T == 32 ? 1 : 2);   // producer waves
  static constexpr int NTT = 64 * (NW + NP);    // threads per workgroup
  static constexpr int TWM = T / WGM, TWN = T / WGN;
  static constexpr int FM = TWM / 16, FN = TWN / 16;
};

// The fp32 accumulators of one wave: block (fm, fn), lane L, element v holds
// output row 16 fm + 4 (L / 16) + v, column 16 fn + L % 16 of the wave's part
// (the operands fed the other way round, as the update does, give the
// transposed block: row 16 fm + L % 16, columns 16 fn + 4 (L / 16) + v).
template <int T>
using AccT = f32x4_t[Tile<T>::FM][Tile<T>::FN];

// LDS ring of one main loop: NSTAGE stages of BK K-elements of both operands
// (the 128 tile's 32-wide ring is 3 deep, 48 KB, so that three blocks share a
// compute unit in many-block launches).
// A K-contiguous operand row of a stage is RB = 2 BK bytes, stored as CPR
// 16-byte chunks; logical chunk c of row r lives at chunk c ^ ((r / RPB) %
// CPR), RPB being the rows that span the 64 banks once, so that the 16 lanes
// of a ds_read_b128 pass (16 rows, one chunk) hit every bank once.
template <int T, int BK>
struct Ring {
  static constexpr int NSTAGE = BK == 32 ? (T == 128 ? 3 : 4) : (T == 256 ? 2 : 3);
  static constexpr int RB = 2 * BK;
  static constexpr int CPR = RB / 16;
  static constexpr int RPB = 256 / RB;
  static constexpr int A_BYTES = T * RB;         // one operand stage
  static constexpr int STAGE = 2 * A_BYTES;
  // the 256 tile keeps five operand slots of A_BYTES (mainloop_pp_kc5)
  static constexpr int LDS = T == 256 ? 5 * A_BYTES : NSTAGE * STAGE;
  static constexpr int DMA_OP = T * BK / 512 / Tile<T>::NW;   // 1 KB DMAs per wave per operand
  static constexpr int PER_STAGE = 2 * DMA_OP;
  static_assert(T * BK % (512 * Tile<T>::NW) == 0, "whole DMA instructions per wave");
  static_assert(LDS <= 160 * 1024, "gfx950 LDS is 160 KB per workgroup");
};

__device__ inline float bf2f(uint16_t v) { return __uint_as_float(uint32_t(v) << 16); }
__device__ inline uint16_t f2bf(float f) {     // v_cvt_pk_bf16_f32: round to nearest even
  __bf16 h = static_cast<__bf16>(f);
  return __builtin_bit_cast(uint16_t, h);
}

__device__ inline uint32_t lds_addr(const void* p) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>(p));
}

// One 16-byte-per-lane direct global -> LDS load: lane i writes LDS bytes
// [lds + 16 i, lds + 16 i + 16).  Issued through inline assembly so that the
// compiler does not serialise the LDS reads of other stages behind it; the
// ring's own s_waitcnt/s_barrier pairs order it.
__device__ inline void dma16(const void* base, uint32_t voff, uint32_t lds) {
  asm volatile(
      "s_mov_b32 m0, %2\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %0, %1\n"
      :
      : "v"(voff), "s"(base), "s"(lds)
      : "memory", "m0");
}

// Wait until at most `pending` DMA instructions of this wave are in flight and
// all of its LDS reads are done, then join the workgroup barrier.  The LDS
// wait goes through the builtin so that the compiler knows the reads are
// complete; the DMA wait and the barrier are assembly, since the compiler does
// not see the DMA loads.
template <int PENDING>
__device__ inline void ring_sync_dma() {
  if constexpr (PENDING == 0) asm volatile("s_waitcnt vmcnt(0)\n\ts_barrier" ::: "memory");
  else if constexpr (PENDING == 2) asm volatile("s_waitcnt vmcnt(2)\n\ts_barrier" ::: "memory");
  else if constexpr (PENDING == 4) asm volatile("s_waitcnt vmcnt(4)\n\ts_barrier" ::: "memory");
  else if constexpr (PENDING == 6) asm volatile("s_waitcnt vmcnt(6)\n\ts_barrier" ::: "memory");
  else if constexpr (PENDING == 8) asm volatile("s_waitcnt vmcnt(8)\n\ts_barrier" ::: "memory");
  else if constexpr (PENDING == 12) asm volatile("s_waitcnt vmcnt(12)\n\ts_barrier" ::: "memory");
  else if constexpr (PENDING == 16) asm volatile("s_waitcnt vmcnt(16)\n\ts_barrier" ::: "memory");
  else if constexpr (PENDING == 24) asm volatile("s_waitcnt vmcnt(24)\n\ts_barrier" ::: "memory");
  else if constexpr (PENDING == 32) asm volatile("s_waitcnt vmcnt(32)\n\ts_barrier" ::: "memory");
  else static_assert(PENDING == 0, "unsupported in-flight count");
}

template <int PENDING>
__device__ inline void ring_sync() {
  __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0), vmcnt/expcnt untouched
  ring_sync_dma<PENDING>();
}

// Wait for all but `stages` of this wave's stages in flight, then barrier.
// (MAXS: the most stages a caller can leave in flight; larger counts are not
// instantiated, since vmcnt holds at most 63.)
template <int PS, int MAXS>
__device__ inline void ring_wait(int stages) {
  static_assert(MAXS * PS <= 63, "in-flight count beyond vmcnt");
  __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0), vmcnt/expcnt untouched
  if constexpr (MAXS >= 3) {
    if (stages >= 3) { ring_sync_dma<3 * PS>(); return; }
  }
  if constexpr (MAXS >= 2) {
    if (stages == 2) { ring_sync_dma<2 * PS>(); return; }
  }
  if constexpr (MAXS >= 1) {
    if (stages == 1) { ring_sync_dma<PS>(); return; }
  }
  ring_sync_dma<0>();
}

// DMA-only wait (no barrier): at most PENDING DMA instructions of this wave
// still in flight.
template <int PENDING>
__device__ inline void dma_wait() {
  if constexpr (PENDING == 0) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  else if constexpr (PENDING == 2) asm volatile("s_waitcnt vmcnt(2)" ::: "memory");
  else if constexpr (PENDING == 4) asm volatile("s_waitcnt vmcnt(4)" ::: "memory");
  else if constexpr (PENDING == 6) asm volatile("s_waitcnt vmcnt(6)" ::: "memory");
  else if constexpr (PENDING == 8) asm volatile("s_waitcnt vmcnt(8)" ::: "memory");
  else if constexpr (PENDING == 12) asm volatile("s_waitcnt vmcnt(12)" ::: "memory");
  else if constexpr (PENDING == 16) asm volatile("s_waitcnt vmcnt(16)" ::: "memory");
  else if constexpr (PENDING == 24) asm volatile("s_waitcnt vmcnt(24)" ::: "memory");
  else static_assert(PENDING == 0, "unsupported in-flight count");
}

// DMA-only wait for all but `stages` stages of PS instructions (stages <= MAXS).
template <int PS, int MAXS>
__device__ inline void dma_wait_upto(int stages) {
  static_assert(MAXS * PS <= 63, "in-flight count beyond vmcnt");
  if constexpr (MAXS >= 2) {
    if (stages >= 2) { dma_wait<2 * PS>(); return; }
  }
  if constexpr (MAXS >= 1) {
    if (stages == 1) { dma_wait<PS>(); return; }
  }
  dma_wait<0>();
}

__device__ inline void barrier_pinned() {
  __builtin_amdgcn_sched_barrier(0);
  asm volatile("s_barrier" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
}

// ---------------------------------------------------------------- DMA issue
// The per-lane offset of a DMA is 32 bits: the base address of every call
// starts at the instruction's first row, so an offset spans the rows of one
// wave's instructions (at most 256) of a row of at most 65536 + 7 elements.
//
// K-contiguous operand: T rows x BK bf16 in the swizzled row layout of Ring.
// One instruction fills 1 KB = 64 / CPR rows; lane i writes chunk i % CPR of
// its row, i.e. it loads logical chunk (i % CPR) ^ swizzle.  Split over NI
// issuing waves (w = 0 .. NI - 1): instruction q of wave w fills 1 KB block
// w + NI q of the operand stage.  The rows of that block's first row and the
// K offset go into the (uniform) base address, so the per-lane offset only
// holds the lane's row within the instructions of wave w and its swizzled
// chunk, which the compiler can keep in one or two registers.
template <int T, int BK, int NI>
__device__ inline void dma_kc_w(const uint16_t* src, int64_t ld, int k0, uint32_t lds, int q, int w) {
  using R = Ring<T, BK>;
  constexpr int RPI = 64 / R::CPR;
  const int lane = threadIdx.x & 63;
  const int j = w + NI * q;
  const int rq = NI * q * RPI;                  // uniform row offset of the instruction
  const int rl = w * RPI + lane / R::CPR;       // row within it
  const int r = rq + rl;
  const int c = (lane % R::CPR) ^ ((r / R::RPB) % R::CPR);
  const uint16_t* base = src + int64_t(rq) * ld + k0;
  const uint32_t voff = uint32_t((int64_t(rl) * ld + c * 8) * 2);
  dma16(base, voff, __builtin_amdgcn_readfirstlane(lds + uint32_t(j) * 1024u));
}

// All NW compute waves issuing: instruction q of wave w fills block w + NW q.
template <int T, int BK>
__device__ inline void dma_kc(const uint16_t* src, int64_t ld, int k0, uint32_t lds, int q) {
  dma_kc_w<T, BK, Tile<T>::NW>(src, ld, k0, lds, q, int(threadIdx.x >> 6));
}

template <int T, int BK>
__device__ inline void issue_kc(const uint16_t* src, int64_t ld, int k0, uint32_t lds) {
#pragma unroll
  for (int q = 0; q < Ring<T, BK>::DMA_OP; ++q) dma_kc<T, BK>(src, ld, k0, lds, q);
}

// The transposing reads of a 16 x 32 (K) operand block touch, per half wave,
// 8 rows (bits 0, 1 and 3 of the row vary) at one logical chunk: the swizzle
// sends them to 8 different 32-byte bank groups (with 4 chunks per row, the
// 64 tile, row parity supplies the third bit).
template <int T>
__device__ inline int swz_y(int r) {
  return T >= 128 ? ((r & 3) | (((r >> 3) & 1) << 2)) : (((r >> 1) & 1) | (((r >> 3) & 1) << 1));
}

// Row-major operand (the update's Y): BK rows (K) x T columns, row = 2T bytes,
// 32-byte chunks swizzled per row.  Split over NI issuing waves as dma_kc_w;
// the instruction's first row (K offset k0 + its rows) goes into the 64-bit
// base address, so the 32-bit per-lane offset spans a few rows only,
// whatever the matrix size.
template <int T, int BK, int NI>
__device__ inline void dma_rm_w(const uint16_t* src, int64_t ld, int k0, uint32_t lds, int q, int w) {
  constexpr int ROWB = 2 * T;
  constexpr int LPR = ROWB / 16;          // lanes per row
  constexpr int RPI = 1024 / ROWB;        // rows per instruction
  const int lane = threadIdx.x & 63;
  const int j = w + NI * q;
  const int rq = NI * q * RPI;
  const int rl = w * RPI + lane / LPR;
  const int p16 = lane % LPR;
  const int c = (p16 >> 1) ^ swz_y<T>(rq + rl);
  const uint16_t* base = src + int64_t(k0 + rq) * ld;
  const uint32_t voff = uint32_t((int64_t(rl) * ld + c * 16 + (p16 & 1) * 8) * 2);
  dma16(base, voff, __builtin_amdgcn_readfirstlane(lds + uint32_t(j) * 1024u));
}

template <int T, int BK>
__device__ inline void dma_rm(const uint16_t* src, int64_t ld, int k0, uint32_t lds, int q) {
  dma_rm_w<T, BK, Tile<T>::NW>(src, ld, k0, lds, q, int(threadIdx.x >> 6));
}

// ---------------------------------------------------------------- compute
template <int T>
struct Frags {
  uint4 a[Tile<T>::FM], b[Tile<T>::FN];
};

template <int T>
__device__ inline void zero_acc(AccT<T>& acc) {
#pragma unroll
  for (int fm = 0; fm < Tile<T>::FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < Tile<T>::FN; ++fn) acc[fm][fn] = f32x4_t{0.f, 0.f, 0.f, 0.f};
}

// MFMA operands of the 32-wide K slice s of one stage.  K-contiguous operand,
// block of 16 rows: lane L loads the 16 bytes (8 K values) at K offset 32 s +
// 8 (L / 16) of row L % 16; the rows of a wave's blocks are 16 apart, which
// keeps the chunk swizzle, so one address serves all of them.  Row-major
// operand (the update's Y, RM): lane L needs the 8 K values 32 s + 8 (L / 16)
// .. + 7 of column L % 16 of the block, gathered by two transposing reads of
// four rows each: lane q of a 16-lane group addresses row kb + q / 4, columns
// 4 (q % 4) .. + 3 of the block, and receives rows kb .. kb + 3 of column q.
template <int T, int BK>
__device__ inline void load_frags_a(Frags<T>& fr, const char* sa, int s, int wm) {
  using R = Ring<T, BK>;
  const int lane = threadIdx.x & 63;
  const int lr = lane & 15, g = lane >> 4;
  const int c = 4 * s + g;
  const int r0 = wm * Tile<T>::TWM + lr;
  const char* p = sa + r0 * R::RB + 16 * (c ^ ((r0 / R::RPB) % R::CPR));
#pragma unroll
  for (int f = 0; f < Tile<T>::FM; ++f) fr.a[f] = *reinterpret_cast<const uint4*>(p + f * 16 * R::RB);
}

template <int T, bool RM, int BK>
__device__ inline void load_frags_b(Frags<T>& fr, const char* sb, int s, int wn) {
  constexpr int FN = Tile<T>::FN;
  using R = Ring<T, BK>;
  const int lane = threadIdx.x & 63;
  const int lr = lane & 15, g = lane >> 4;
  const int c = 4 * s + g;
  if constexpr (!RM) {
    const int r0 = wn * Tile<T>::TWN + lr;
    const char* p = sb + r0 * R::RB + 16 * (c ^ ((r0 / R::RPB) % R::CPR));
#pragma unroll
    for (int f = 0; f < FN; ++f) fr.b[f] = *reinterpret_cast<const uint4*>(p + f * 16 * R::RB);
  } else {
    // Column block f of wave wn is block f WGN + wn of the tile (the waves'
    // blocks interleave), i.e. 32-byte chunk f WGN + wn of a stage row.  Row of
    // the first read within the slice; the second read's row (+ 4) and every
    // slice share its swizzle (bits 0, 1 and 3 of the row).  chunk ^ sw =
    // (f ^ hi) WGN + (wn ^ lo) with hi = sw / WGN, lo = sw % WGN.
    constexpr int WGN = Tile<T>::WGN;
    const int rl = 8 * g + (lr >> 2);
    const int sw = swz_y<T>(rl);
    const int hi = sw / WGN;
    const char* base = sb + (32 * s + rl) * (2 * T) + 8 * (lr & 3) + 32 * (wn ^ (sw % WGN));
    // when hi is 0 or 1 (sw < 2 WGN), f ^ hi = f + hi for even f and f - hi for
    // odd f: two addresses and immediate offsets serve every block
    constexpr bool two = (T >= 128 ? 8 : 4) <= 2 * WGN;   // largest sw + 1 <= 2 WGN
    const char* pe = base + 32 * WGN * hi;
    const char* po = base - 32 * WGN * hi;
#pragma unroll
    for (int f = 0; f < FN; ++f) {
      const char* p = two ? ((f & 1) ? po : pe) + 32 * WGN * f : base + 32 * WGN * (f ^ hi);
      s16x4_t v[2];
#pragma unroll
      for (int h = 0; h < 2; ++h)
        v[h] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (__attribute__((address_space(3))) s16x4_t*)(lds_addr(p + h * 4 * (2 * T))));
      fr.b[f] = __builtin_bit_cast(uint4, v);
    }
  }
}

template <int T, bool RM, int BK>
__device__ inline void load_frags(Frags<T>& fr, const char* sa, const char* sb, int s, int wm,
                                  int wn) {
  load_frags_a<T, BK>(fr, sa, s, wm);
  load_frags_b<T, RM, BK>(fr, sb, s, wn);
}

// SWAP = false: acc[fm][fn] = a-rows x b-rows^T (the MFMA layout of AccT).
// SWAP = true feeds the operands the other way round, so acc[fm][fn] holds
// the transposed block: each lane then owns 4 consecutive columns of one row.
template <int T, bool SWAP>
__device__ inline void mma(AccT<T>& acc, const Frags<T>& fr) {
#pragma unroll
  for (int fm = 0; fm < Tile<T>::FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < Tile<T>::FN; ++fn) {
      if constexpr (SWAP)
        acc[fm][fn] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
            __builtin_bit_cast(bf16x8_t, fr.b[fn]), __builtin_bit_cast(bf16x8_t, fr.a[fm]),
            acc[fm][fn], 0, 0, 0);
      else
        acc[fm][fn] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
            __builtin_bit_cast(bf16x8_t, fr.a[fm]), __builtin_bit_cast(bf16x8_t, fr.b[fn]),
            acc[fm][fn], 0, 0, 0);
    }
}

// Runs slice(kt, s, cur, nxt) over every 32-wide slice s of every stage kt in
// increasing K order; cur holds the slice's operands, nxt receives the next
// one's.  With an even number of slices per stage the two operand buffers
// alternate within a stage; with one slice per stage, across stages.
template <int NS, class Fr, class Slice>
__device__ inline void for_each_slice(int nk, Fr& f0, Fr& f1, Slice slice) {
  if constexpr (NS % 2 == 0) {
    for (int kt = 0; kt < nk; ++kt)
#pragma unroll
      for (int s = 0; s < NS; s += 2) {
        slice(kt, s, f0, f1);
        slice(kt, s + 1, f1, f0);
      }
  } else {
    static_assert(NS == 1, "one or an even number of slices per stage");
    int kt = 0;
    for (; kt + 1 < nk; kt += 2) {
      slice(kt, 0, f0, f1);
      slice(kt + 1, 0, f1, f0);
    }
    if (kt < nk) slice(kt, 0, f0, f1);
  }
}

// 4-wave main loop of the update's 128 and 64 tiles.  acc = A (T x K,
// K-contiguous rows of a) * B^T where B's rows are the K-contiguous rows of b
// (RM = false) or B = the K x T row-major block of b (RM = true); K is a
// multiple of BK and every tile is full.  The operands of each 32-wide K
// slice are read from LDS while the previous slice's MFMAs run.  The DMA is
// spread over the K slices: while stage kt is read and multiplied, each wave
// issues its share of stage kt + NSTAGE - 1, PS / NS instructions per slice,
// into the buffer of stage kt - 1 (every wave finished reading it before the
// barrier that opened stage kt).  The global -> LDS path (about 64 bytes per
// clock and compute unit) is then fed evenly instead of in one burst per stage
// that stalls every wave.  Slices are consumed in increasing order whatever BK
// is, so every output element accumulates the same products in the same order.
template <int T, bool RM, bool SWAP, int BK>
__device__ inline void mainloop(AccT<T>& acc, char* smem, const uint16_t* a, int64_t lda,
                                const uint16_t* b, int64_t ldb, int K) {
  using R = Ring<T, BK>;
  constexpr int PS = R::PER_STAGE, NS = BK / 32, NST = R::NSTAGE, DO = R::DMA_OP;
  constexpr int PPS = PS / NS;
  static_assert(PPS * NS == PS && PPS >= 1, "whole DMA instructions per slice");
  const int wave = threadIdx.x >> 6;
  const int wm = wave / Tile<T>::WGN, wn = wave % Tile<T>::WGN;
  zero_acc<T>(acc);

  const uint32_t lds0 = lds_addr(smem);
  const int nk = K / BK;
  auto stage_lds = [&](int kt) { return lds0 + uint32_t((kt % NST) * R::STAGE); };
  // DMA instruction i (0 .. PS - 1) of stage kt: operand a first, then b
  auto dma_one = [&](int kt, int i) {
    if (i < DO) {
      dma_kc<T, BK>(a, lda, kt * BK, stage_lds(kt), i);
    } else {
      if constexpr (RM) dma_rm<T, BK>(b, ldb, kt * BK, stage_lds(kt) + R::A_BYTES, i - DO);
      else dma_kc<T, BK>(b, ldb, kt * BK, stage_lds(kt) + R::A_BYTES, i - DO);
    }
  };
  auto stage_ptr = [&](int kt) { return smem + (kt % NST) * R::STAGE; };
#pragma unroll
  for (int s = 0; s + 1 < NST; ++s)
    if (s < nk)
      for (int i = 0; i < PS; ++i) dma_one(s, i);
  ring_wait<PS, NST - 2>(min(nk - 1, NST - 2));

  Frags<T> f0, f1;
  load_frags<T, RM, BK>(f0, stage_ptr(0), stage_ptr(0) + R::A_BYTES, 0, wm, wn);
  for_each_slice<NS>(nk, f0, f1, [&](int kt, int s, Frags<T>& cur, Frags<T>& nxt) {
    const char* st = stage_ptr(kt);
    const int nx = kt + NST - 1;   // stage refilled during this one
    const bool fill = nx < nk;
    if (s + 1 < NS) {
      load_frags<T, RM, BK>(nxt, st, st + R::A_BYTES, s + 1, wm, wn);
      if (fill)
#pragma unroll
        for (int i = 0; i < PPS; ++i) dma_one(nx, s * PPS + i);
      mma<T, SWAP>(acc, cur);
    } else {
      if (fill)
#pragma unroll
        for (int i = 0; i < PPS; ++i) dma_one(nx, s * PPS + i);
      __builtin_amdgcn_sched_barrier(0);
      if (kt + 1 < nk) {
        ring_wait<PS, NST - 2>(min(nk - 1, kt + NST - 1) - (kt + 1));
        const char* nxp = stage_ptr(kt + 1);
        load_frags<T, RM, BK>(nxt, nxp, nxp + R::A_BYTES, 0, wm, wn);
      }
      __builtin_amdgcn_sched_barrier(0);
      mma<T, SWAP>(acc, cur);
    }
  });
  ring_sync<0>();   // the ring is free for the epilogue
}

// Producer/consumer main loop of the smaller tiles' Gram and polynomial
// (both operands K-contiguous).  With one compute wave
// per SIMD, the stall of a DMA issue (the wave waits while the compute
// unit's global -> LDS queue drains) left the SIMD's matrix core idle, so
// NP extra waves issue the whole ring's DMA while the NW compute waves only
// read LDS and multiply.  Per stage kt, between two workgroup barriers: the
// producers issue stage kt + NST - 1 into the buffer of stage kt - 1 (read
// before the last barrier) and wait for their DMA of stage kt + 1; the
// compute waves multiply stage kt, loading the operands of each 32-wide
// slice while the previous slice's MFMAs run, and finish their LDS reads
// before the barrier.  Slices are consumed in increasing K order, so every
// output element accumulates the same products in the same order as in the
// other loops.  The producer waves return afterwards; a barrier then waits
// only for the waves still running.
template <int T, bool SWAP, int BK>
__device__ inline bool mainloop_pc(AccT<T>& acc, char* smem, const uint16_t* a, int64_t lda,
                                   const uint16_t* b, int64_t ldb, int K) {
  using R = Ring<T, BK>;
  constexpr int NW = Tile<T>::NW, NP = Tile<T>::NP, NS = BK / 32, NST = R::NSTAGE;
  constexpr int DOP = T * BK / 512 / NP;     // 1 KB DMAs per producer and operand stage
  constexpr int PSP = 2 * DOP;
  static_assert(NP >= 1 && DOP * NP * 512 == T * BK, "whole DMA instructions per producer");
  const int wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x >> 6));
  const bool prod = wave >= NW;
  const uint32_t lds0 = lds_addr(smem);
  const int nk = K / BK;
  auto stage_ptr = [&](int kt) { return smem + (kt % NST) * R::STAGE; };
  if (prod) {
    const int pw = wave - NW;
    auto issue = [&](int kt) {
      const uint32_t st = lds0 + uint32_t((kt % NST) * R::STAGE);
#pragma unroll
      for (int q = 0; q < DOP; ++q) dma_kc_w<T, BK, NP>(a, lda, kt * BK, st, q, pw);
#pragma unroll
      for (int q = 0; q < DOP; ++q) dma_kc_w<T, BK, NP>(b, ldb, kt * BK, st + R::A_BYTES, q, pw);
    };
    for (int s = 0; s + 1 < NST && s < nk; ++s) issue(s);
    dma_wait_upto<PSP, NST - 2>(min(nk - 1, NST - 2));
    barrier_pinned();
    for (int kt = 0; kt < nk; ++kt) {
      if (kt + NST - 1 < nk) issue(kt + NST - 1);
      dma_wait_upto<PSP, NST - 2>(min(nk - 1, kt + NST - 1) - (kt + 1));
      barrier_pinned();
    }
    dma_wait<0>();
    return false;
  }
  const int wm = wave / Tile<T>::WGN, wn = wave % Tile<T>::WGN;
  zero_acc<T>(acc);
  barrier_pinned();   // stage 0 has landed
  Frags<T> f0, f1;
  load_frags<T, false, BK>(f0, stage_ptr(0), stage_ptr(0) + R::A_BYTES, 0, wm, wn);
  for_each_slice<NS>(nk, f0, f1, [&](int kt, int s, Frags<T>& cur, Frags<T>& nxt) {
    const char* st = stage_ptr(kt);
    if (s + 1 < NS) {
      load_frags<T, false, BK>(nxt, st, st + R::A_BYTES, s + 1, wm, wn);
      mma<T, SWAP>(acc, cur);
    } else {
      __builtin_amdgcn_sched_barrier(0);
      __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0): stage kt is read
      barrier_pinned();                     // and stage kt + 1 has landed
      if (kt + 1 < nk) {
        const char* nxp = stage_ptr(kt + 1);
        load_frags<T, false, BK>(nxt, nxp, nxp + R::A_BYTES, 0, wm, wn);
      }
      __builtin_amdgcn_sched_barrier(0);
      mma<T, SWAP>(acc, cur);
    }
  });
  return true;
}

// Ping-pong schedule of the 8-wave tile (mainloop_pp below).  Waves 0-3
// (group 0) and 4-7 (group 1) occupy one slot per SIMD each; group 1 runs
// one phase behind, so that while one wave of a SIMD issues the MFMAs of a
// whole 64-wide K stage from registers, the other reads its operands of the
// next stage from LDS and issues its group's DMA.  Every phase ends with a
// workgroup barrier:
//   group 0: [MEM(j) | COMP(j)] for each stage j, then one idle phase;
//   group 1: one idle phase, then [MEM(j) | COMP(j)].
// A COMP phase is 2 slices x FM x FN = 64 v_mfma_f32_16x16x32_bf16 per wave
// (96 operand registers next to the 128 accumulators), so a stage costs two
// barriers.  K-contiguous rows of a stage are one full 128-byte line, which
// the global -> LDS path moves at twice the rate of 64-byte half lines.
//
// The LDS holds five operand slots of one operand stage (32 KB) each, the
// whole 160 KB, filled in the order a(0), b(0), a(1), b(1), ...: operand stage
// i goes into slot i % 5.  In MEM(j), group 0 issues b(j + 1) into the slot of
// a(j - 1) and group 1 (one phase later) issues a(j + 2) into the slot of
// b(j - 1); both slots were read by both groups in MEM(j - 1).  Five operand
// stages are live at most (a(j), b(j) being read, a(j + 1), b(j + 1),
// a(j + 2)).  Before the barrier that ends its COMP(j), group 0 waits for its
// b(j + 1); before the barrier that ends its MEM(j), group 1 waits for its
// a(j + 1), leaving a(j + 2) in flight: the barrier that opens group 0's
// MEM(j + 1) comes after both.
template <int T, bool RM, bool SWAP, int BK>
__device__ inline void mainloop_pp(AccT<T>& acc, char* smem, const uint16_t* a, int64_t lda,
                                   const uint16_t* b, int64_t ldb, int K) {
  static_assert(Tile<T>::NW == 8, "ping-pong needs two waves per SIMD");
  static_assert(BK == 64, "two 32-wide slices per stage");
  using R = Ring<T, BK>;
  constexpr int SLOTS = 5;
  constexpr int QG = T * BK / 512 / 4;    // 1 KB DMAs per wave of a group and operand stage
  static_assert(SLOTS * R::A_BYTES <= R::LDS, "five operand slots");
  const int wave = threadIdx.x >> 6;
  const int wm = wave / 4, wn = wave % 4;
  const int w4 = wave & 3;
  const bool g1 = __builtin_amdgcn_readfirstlane(wave) >= 4;
  zero_acc<T>(acc);

  const uint32_t lds0 = lds_addr(smem);
  const int nk = K / BK;
  auto slot_lds = [&](int i) { return lds0 + uint32_t((i % SLOTS) * R::A_BYTES); };
  auto slot_ptr = [&](int i) { return smem + (i % SLOTS) * R::A_BYTES; };
  // instructions q0 .. q1 - 1 of this wave's share of operand stage a(kt) / b(kt)
  auto issue_a = [&](int kt, int q0, int q1) {
#pragma unroll
    for (int q = q0; q < q1; ++q) dma_kc_w<T, BK, 4>(a, lda, kt * BK, slot_lds(2 * kt), q, w4);
  };
  auto issue_b = [&](int kt, int q0, int q1) {
#pragma unroll
    for (int q = q0; q < q1; ++q) {
      if constexpr (RM) dma_rm_w<T, BK, 4>(b, ldb, kt * BK, slot_lds(2 * kt + 1), q, w4);
      else dma_kc_w<T, BK, 4>(b, ldb, kt * BK, slot_lds(2 * kt + 1), q, w4);
    }
  };

  if (!g1) {
    issue_b(0, 0, QG);
  } else {
    issue_a(0, 0, QG);
    if (nk > 1) issue_a(1, 0, QG);
  }
  __builtin_amdgcn_s_waitcnt(0xC07F);
  ring_sync_dma<0>();
  if (g1) barrier_pinned();

  Frags<T> f0, f1;
  for (int j = 0; j < nk; ++j) {
    const char* sa = slot_ptr(2 * j);
    const char* sb = slot_ptr(2 * j + 1);
    // MEM: the group's DMA first, then the LDS reads of both slices.  The
    // two share the LDS (the DMA writes its data there), so they take about
    // the sum of their times in either order; issued first, the DMA lands
    // a whole memory phase earlier, which removes most of group 0's wait
    // for b(j + 1) at the end of its COMP(j).
    if (!g1) {
      if (j + 1 < nk) issue_b(j + 1, 0, QG);
    } else {
      if (j + 2 < nk) issue_a(j + 2, 0, QG);
    }
    __builtin_amdgcn_sched_barrier(0);
    load_frags<T, RM, BK>(f0, sa, sb, 0, wm, wn);
    load_frags<T, RM, BK>(f1, sa, sb, 1, wm, wn);
    __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0)
    if (g1) {
      if (j + 2 < nk) dma_wait<QG>();
      else dma_wait<0>();
    }
    barrier_pinned();
    // COMP
    mma<T, SWAP>(acc, f0);
    mma<T, SWAP>(acc, f1);
    if (!g1) dma_wait<0>();
    barrier_pinned();
  }
  if (!g1) barrier_pinned();
  __builtin_amdgcn_s_waitcnt(0xC07F);
  dma_wait<0>();
}

template <int T, bool RM, bool SWAP, int BK>
// Returns false in the producer waves, which then leave the kernel.
__device__ inline bool run_mainloop(AccT<T>& acc, char* smem, const uint16_t* a, int64_t lda,
                                    const uint16_t* b, int64_t ldb, int K) {
  if constexpr (Tile<T>::NW == 8) {
    mainloop_pp<T, RM, SWAP, BK>(acc, smem, a, lda, b, ldb, K);
    return true;
  } else if constexpr (RM) {   // the update's smaller tiles: compute waves issue the DMA
    mainloop<T, RM, SWAP, BK>(acc, smem, a, lda, b, ldb, K);
    return true;
  } else {
    return mainloop_pc<T, SWAP, BK>(acc, smem, a, lda, b, ldb, K);
  }
}

// ---------------------------------------------------------------- mapping
// Workgroup p runs on XCD p % 8 (round-robin dispatch).  Logical tiles are
// dealt to the XCDs in chunks of 32 consecutive tiles: XCD x's j-th group of
// 32 workgroups takes chunk 8 (j / 32) + x.  Neighbouring tiles (which share
// operand rows) then run together on one XCD and hit its L2, while the eight
// XCDs work on adjacent chunks of the same matrices, so operand panels that
// leave one L2 are still in the memory-side cache when the next XCD asks for
// them.  The workgroups past the last full round of 8 chunks (all of them in
// a launch of fewer than 256 tiles) split the remaining n tiles the same way:
// XCD x takes a contiguous run of n / 8 of them, one more for x < n % 8 (XCD
// x has exactly that many of those workgroups), so the tiles of one matrix
// still share an L2.
__device__ inline int xcd_remap(int p, int total) {
  constexpr int C = 32;
  const int full = total / (8 * C) * (8 * C);
  if (p < full) {
    const int x = p & 7, j = p >> 3;
    return ((j / C) * 8 + x) * C + (j % C);
  }
  const int n = total - full, q = p - full;
  const int x = q & 7, j = q >> 3;
  return full + x * (n >> 3) + min(x, n & 7) + j;
}

struct Loc {
  int ent, mat, tile;
};

__device__ inline Loc locate(const Phase& P, int lid) {
  // last entry whose first block is <= lid (entries without blocks share the
  // start of the next entry and are never the last such entry)
  int e = 0, hi = P.nent - 1;
  while (e < hi) {
    const int mid = (e + hi + 1) >> 1;
    if (lid >= int(P.e[mid].tile_start)) e = mid;
    else hi = mid - 1;
  }
  const int r = lid - int(P.e[e].tile_start);
  const int per = int(P.e[e].tiles_per);
  Loc L;
  L.ent = e;
  L.mat = r / per;
  L.tile = r - L.mat * per;
  return L;
}

// kByMatrix: workgroup p runs on XCD p % 8 (round-robin dispatch), and XCD x's
// workgroups take, in launch order, the tiles of the launch's matrices whose
// index is x mod 8: each XCD gets an eighth of every kind of matrix (balanced
// when tile costs differ between entries) and a matrix's tiles share one L2.
// False for the workgroups past the end of their XCD's list.
__device__ inline bool locate_by_matrix(const Phase& P, int p, Loc& L) {
  const int x = p & 7;
  int j = p >> 3, g0 = 0;
  for (int e = 0; e < P.nent; ++e) {
    const int c = int(P.e[e].count), tp = int(P.e[e].tiles_per);
    const int i0 = (x - (g0 & 7) + 8) & 7;        // first matrix of the entry on XCD x
    const int nt = (i0 < c ? (c - 1 - i0) / 8 + 1 : 0) * tp;
    if (j < nt) {
      L.ent = e;
      L.mat = i0 + 8 * (j / tp);
      L.tile = j - (j / tp) * tp;
      return true;
    }
    j -= nt;
    g0 += c;
  }
  return false;
}

__device__ inline char* ws_of(const Phase& P, const Entry& E, int mat) {
  return P.ws + (uint64_t(E.ws256) << 8) + uint64_t(mat) * ws_layout(E.kp, E.Np, 2).total;
}

__device__ inline uint16_t* user_of(const Phase& P, const Entry& E, int mat) {
  char* x = (E.flags & kPtrTab) ? P.xp[E.xbase + mat] : E.x + uint64_t(mat) * E.k * E.N * 2u;
  return reinterpret_cast<uint16_t*>(x);
}

// Y buffer of a slot (kp x Np, ld ldy): the first slot is W1 (or, for a
// kDirect entry, the caller's matrix, which then has exactly that layout),
// then W2, W1, ... (the final slot is the caller's matrix, handled by the
// update).
__device__ inline uint16_t* wbuf(const Phase& P, const Entry& E, int mat, int slot) {
  if (slot == kSlotFirst && (E.flags & kDirect)) return user_of(P, E, mat);
  const WsLayout L = ws_layout(E.kp, E.Np, 2);
  const bool w1 = slot == kSlotFirst || slot == kSlotAlt2;
  return reinterpret_cast<uint16_t*>(ws_of(P, E, mat) + (w1 ? L.w1 : L.w2));
}

__device__ inline void tri_tile(int t, int nb, int& I, int& J) {
  I = 0;
  while (t >= nb - I) {
    t -= nb - I;
    ++I;
  }
  J = I + t;
}

// Upper tile (I, J) of a symmetric product for this block.  Normally block
// -> logical tile through the XCD mapping.  Under kTail the launch covers the
// logical tiles (of size 2T) from P.tail_base on, four blocks per tile, one
// per T x T sub-tile; the sub-tile below the diagonal of a diagonal tile has
// no work (false).
template <int T>
__device__ inline bool sym_tile(const Phase& P, Loc& L, int& I, int& J) {
  if (P.flags & kTail) {
    const int sub = int(blockIdx.x) & 3;
    L = locate(P, P.tail_base + int(blockIdx.x >> 2));
    int I2, J2;
    tri_tile(L.tile, int(P.e[L.ent].kp) / (2 * T), I2, J2);
    if (I2 == J2 && sub == 2) return false;
    I = 2 * I2 + (sub >> 1);
    J = 2 * J2 + (sub & 1);
    return true;
  }
  if (P.flags & kByMatrix) {
    if (!locate_by_matrix(P, int(blockIdx.x), L)) return false;
  } else {
    L = locate(P, xcd_remap(blockIdx.x, P.total));
  }
  tri_tile(L.tile, int(P.e[L.ent].kp) / T, I, J);
  return true;
}

// First of the 4 consecutive rows, and the column, of this lane's elements of
// accumulator block (fm, fn) (operands not swapped).
template <int T>
__device__ inline int acc_row(int wm, int fm) {
  return wm * Tile<T>::TWM + fm * 16 + 4 * ((threadIdx.x & 63) >> 4);
}
template <int T>
__device__ inline int acc_col(int wn, int fn) {
  return wn * Tile<T>::TWN + fn * 16 + (threadIdx.x & 15);
}
__device__ inline int wave_m(int wgn) { return int(threadIdx.x >> 6) / wgn; }
__device__ inline int wave_n(int wgn) { return int(threadIdx.x >> 6) % wgn; }

// ---------------------------------------------------------------- epilogues
// Output tiles are staged through LDS (the ring is free after the main loop)
// as T x T bf16 with rows padded to T + 8 elements, so that global stores are
// full 16-byte vectors along contiguous rows.
template <int T>
struct Stage {
  static constexpr int RS = (T + 8) * 2;            // padded row stride in bytes
  static constexpr int BYTES = T * RS;
  static constexpr int CPR = T / 8;                 // 16-byte chunks per row
  static constexpr int PER_THREAD = T * CPR / Tile<T>::NT;  // chunks per thread
};

template <int T, int BK>
constexpr int smem_bytes() {
  return Ring<T, BK>::LDS > Stage<T>::BYTES ? Ring<T, BK>::LDS : Stage<T>::BYTES;
}

// LDS row r of the stage -> dst row row0 + r, columns col0.. (whole tile).
template <int T>
__device__ inline void store_rows(const char* st, uint16_t* dst, int64_t ld, int64_t row0,
                                  int64_t col0) {
#pragma unroll 4
  for (int it = 0; it < Stage<T>::PER_THREAD; ++it) {
    const int q = it * Tile<T>::NT + int(threadIdx.x);
    const int r = q / Stage<T>::CPR, c8 = q % Stage<T>::CPR;
    const uint4 v = *reinterpret_cast<const uint4*>(st + r * Stage<T>::RS + c8 * 16);
    *reinterpret_cast<uint4*>(dst + (row0 + r) * ld + col0 + c8 * 8) = v;
  }
}

// Transposed: stage element (r, c) -> dst row row0 + c, column col0 + r.
// Each 16-lane group moves an 8-row x 16-column block of the stage with two
// ds_read_b64_tr_b16 (lane q addresses row 4h + q/4, columns 4(q%4).. of the
// block and receives rows 4h..4h+3 of column q), then stores the 8 values of
// its column as one 16-byte vector.  The four groups of a wave take adjacent
// row blocks, so each destination row gets 64 contiguous bytes.
template <int T>
__device__ inline void store_cols(const char* st, uint16_t* dst, int64_t ld, int64_t row0,
                                  int64_t col0) {
  constexpr int RB = T / 8;                      // 8-row blocks
  constexpr int GROUPS = (T / 16) * RB;
  constexpr int NG = Tile<T>::NT / 16;
  static_assert(GROUPS % NG == 0, "whole passes");
  const int q = threadIdx.x & 15;
#pragma unroll 2
  for (int g = int(threadIdx.x) >> 4; g < GROUPS; g += NG) {
    const int r8 = g % RB, cb = g / RB;
    s16x4_t v[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const char* p = st + (r8 * 8 + 4 * h + (q >> 2)) * Stage<T>::RS + (cb * 16 + 4 * (q & 3)) * 2;
      v[h] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
          (__attribute__((address_space(3))) s16x4_t*)(lds_addr(p)));
    }
    *reinterpret_cast<uint4*>(dst + (row0 + cb * 16 + q) * ld + col0 + r8 * 8) =
        __builtin_bit_cast(uint4, v);
  }
}

// Caller's wide matrix (rows < k, columns < N, ld = N).
template <int T>
__device__ inline void store_rows_user(const char* st, uint16_t* dst, int k, int N, int row0,
                                       int col0) {
  const bool vec = (N % 8) == 0 && (reinterpret_cast<uintptr_t>(dst) & 15u) == 0u;
#pragma unroll 2
  for (int it = 0; it < Stage<T>::PER_THREAD; ++it) {
    const int q = it * Tile<T>::NT + int(threadIdx.x);
    const int r = q / Stage<T>::CPR, c8 = q % Stage<T>::CPR;
    const int i = row0 + r, l = col0 + c8 * 8;
    if (i >= k || l >= N) continue;
    const uint4 v = *reinterpret_cast<const uint4*>(st + r * Stage<T>::RS + c8 * 16);
    uint16_t* p = dst + int64_t(i) * N + l;
    if (vec && l + 8 <= N) {
      *reinterpret_cast<uint4*>(p) = v;
    } else {
      const uint16_t* e = reinterpret_cast<const uint16_t*>(&v);
      for (int u = 0; u < 8 && l + u < N; ++u) p[u] = e[u];
    }
  }
}

// Caller's tall matrix: stage element (i, l) of the wide view -> dst[l * k + i].
template <int T>
__device__ inline void store_cols_user(const char* st, uint16_t* dst, int k, int N, int row0,
                                       int col0) {
  const bool vec = (k % 8) == 0 && (reinterpret_cast<uintptr_t>(dst) & 15u) == 0u;
#pragma unroll 2
  for (int it = 0; it < Stage<T>::PER_THREAD; ++it) {
    const int q = it * Tile<T>::NT + int(threadIdx.x);
    const int c = q / Stage<T>::CPR, r8 = q % Stage<T>::CPR;
    const int l = col0 + c, i = row0 + r8 * 8;
    if (l >= N || i >= k) continue;
    uint16_t v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e)
      v[e] = *reinterpret_cast<const uint16_t*>(st + (r8 * 8 + e) * Stage<T>::RS + c * 2);
    uint16_t* p = dst + int64_t(l) * k + i;
    if (vec && i + 8 <= k) {
      *reinterpret_cast<uint4*>(p) = *reinterpret_cast<const uint4*>(v);
    } else {
      for (int u = 0; u < 8 && i + u < k; ++u) p[u] = v[u];
    }
  }
}

// Global rows row0.. (T x T bf16 block at col0, ld) -> stage rows.
template <int T>
__device__ inline void load_rows(char* st, const uint16_t* src, int64_t ld, int64_t row0,
                                 int64_t col0) {
#pragma unroll 4
  for (int it = 0; it < Stage<T>::PER_THREAD; ++it) {
    const int q = it * Tile<T>::NT + int(threadIdx.x);
    const int r = q / Stage<T>::CPR, c8 = q % Stage<T>::CPR;
    *reinterpret_cast<uint4*>(st + r * Stage<T>::RS + c8 * 16) =
        *reinterpret_cast<const uint4*>(src + (row0 + r) * ld + col0 + c8 * 8);
  }
}

// Symmetric-product epilogue (Gram, polynomial): value f(i_local, j_local, x,
// staged) of C element (i, j) is written transposed into the stage as
// (j, i); the stage then holds tile (J, I), stored as rows of block J and,
// off the diagonal, transposed as tile (I, J).  `staged` is the stage's
// previous bf16 at that position (the polynomial preloads A's tile (J, I)).
// Each lane's 4 elements of a block are consecutive rows of one column: one
// 8-byte stage row piece.
template <int T, class Fv>
__device__ inline void epilogue_sym(const AccT<T>& acc, char* st, uint16_t* D, int64_t ld, int I,
                                    int J, Fv f) {
  const int wm = wave_m(Tile<T>::WGN), wn = wave_n(Tile<T>::WGN);
#pragma unroll
  for (int fm = 0; fm < Tile<T>::FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < Tile<T>::FN; ++fn) {
      const int c = acc_col<T>(wn, fn);
      const int r0 = acc_row<T>(wm, fm);
      char* p = st + c * Stage<T>::RS + r0 * 2;
      const uint2 old = *reinterpret_cast<const uint2*>(p);
      const uint16_t* o = reinterpret_cast<const uint16_t*>(&old);
      uint16_t out[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) out[u] = f2bf(f(r0 + u, c, acc[fm][fn][u], o[u]));
      *reinterpret_cast<uint2*>(p) = *reinterpret_cast<const uint2*>(out);
    }
  __syncthreads();
  store_rows<T>(st, D, ld, int64_t(J) * T, int64_t(I) * T);
  if (I != J) store_cols<T>(st, D, ld, int64_t(I) * T, int64_t(J) * T);
}

// First polynomial after a scaling pre-conditioner: C = B~ diag(s), so that
// the first update reads X0 itself (B~ X1 = B~ diag(s) X0).  C is not
// symmetric: the mirror C[j][i] = B~_ij s_i and the tile C[i][j] = B~_ij s_j
// of the upper tile (I, J) differ.  Both are rounded once from the fp32 B~_ij;
// the first goes through the stage while the second waits in registers as
// packed bf16, then takes the stage in a second pass.
template <int T, class Fv>
__device__ inline void epilogue_sym_scaled(const AccT<T>& acc, char* st, uint16_t* D, int64_t ld,
                                           int I, int J, Fv f, const float* __restrict__ s) {
  constexpr int FM = Tile<T>::FM, FN = Tile<T>::FN;
  const int wm = wave_m(Tile<T>::WGN), wn = wave_n(Tile<T>::WGN);
  uint2 keep[FM][FN];
#pragma unroll
  for (int fm = 0; fm < FM; ++fm) {
    const int r0 = acc_row<T>(wm, fm);
    const float4 si = *reinterpret_cast<const float4*>(s + I * T + r0);   // s of the 4 rows
    const float sv[4] = {si.x, si.y, si.z, si.w};
#pragma unroll
    for (int fn = 0; fn < FN; ++fn) {
      const int c = acc_col<T>(wn, fn);
      const float sj = s[J * T + c];
      char* p = st + c * Stage<T>::RS + r0 * 2;
      const uint2 old = *reinterpret_cast<const uint2*>(p);
      const uint16_t* o = reinterpret_cast<const uint16_t*>(&old);
      uint16_t out[4], out2[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const float x = f(r0 + u, c, acc[fm][fn][u], o[u]);
        out[u] = f2bf(x * sv[u]);
        out2[u] = f2bf(x * sj);
      }
      *reinterpret_cast<uint2*>(p) = *reinterpret_cast<const uint2*>(out);
      keep[fm][fn] = *reinterpret_cast<const uint2*>(out2);
    }
    __builtin_amdgcn_sched_barrier(0);   // keeps the loads of the next block here
  }
  __syncthreads();
  store_rows<T>(st, D, ld, int64_t(J) * T, int64_t(I) * T);   // C[j][i], j in J, i in I
  if (I == J) return;
  __syncthreads();
#pragma unroll
  for (int fm = 0; fm < FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < FN; ++fn)
      *reinterpret_cast<uint2*>(st + acc_col<T>(wn, fn) * Stage<T>::RS + acc_row<T>(wm, fm) * 2) =
          keep[fm][fn];
  __syncthreads();
  store_cols<T>(st, D, ld, int64_t(I) * T, int64_t(J) * T);   // C[i][j]
}

// fp32 store of an upper tile straight from the registers (first Gram only;
// k_apply_s reads the upper tiles and writes both halves of A1).
template <int T>
__device__ inline void store_sym_f32(const AccT<T>& acc, float* D, int64_t ld, int I, int J) {
  const int wm = wave_m(Tile<T>::WGN), wn = wave_n(Tile<T>::WGN);
#pragma unroll
  for (int fm = 0; fm < Tile<T>::FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < Tile<T>::FN; ++fn) {
      const int j = J * T + acc_col<T>(wn, fn);
      const int ib = I * T + acc_row<T>(wm, fm);
#pragma unroll
      for (int u = 0; u < 4; ++u) D[int64_t(ib + u) * ld + j] = acc[fm][fn][u];
    }
}

// ---------------------------------------------------------------- kernels
template <int T, int BK>
__global__ __launch_bounds__(Tile<T>::NTT) void k_gram_fast(const Phase P) {
  __shared__ __attribute__((aligned(1024))) char smem[smem_bytes<T, BK>()];
  constexpr int FM = Tile<T>::FM, FN = Tile<T>::FN;
  Loc L;
  int I, J;
  if (!sym_tile<T>(P, L, I, J)) return;
  const Entry& E = P.e[L.ent];
  const int kp = int(E.kp), Np = int(E.Np);
  const uint16_t* Y = wbuf(P, E, L.mat, P.src);
  char* w = ws_of(P, E, L.mat);
  const WsLayout WL = ws_layout(E.kp, E.Np, 2);
  const int64_t ldy = WL.ldy;
  AccT<T> acc;
  if (!run_mainloop<T, false, false, BK>(acc, smem, Y + int64_t(I) * T * ldy, ldy, Y + int64_t(J) * T * ldy, ldy, Np)) return;

  if (P.flags & kA32) {
    store_sym_f32<T>(acc, reinterpret_cast<float*>(w + WL.a32), kp, I, J);
  } else {
    auto f = [](int, int, float x, uint16_t) { return x; };
    epilogue_sym<T>(acc, smem, reinterpret_cast<uint16_t*>(w + WL.a), WL.ldg, I, J, f);
  }

  // The host never asks a 32 tile for row sums (their partials cover 64 columns).
  if (T >= kMinTile && (P.flags & kRowSum)) {
    // part[b][i] = sum over the 64 columns of block b of |A0_ij| (with kRowSq:
    // A0_ij^2, whose total is ||A0||_F^2 for the Schatten-4 scale), from the fp32
    // accumulators.  The reduction tree is fixed for every tile size: each
    // 16 x 16 MFMA block is reduced first, pairing column (row) index bits 0,
    // 1, 2, 3 in that order for the row (column) sums, then the four 16-blocks
    // of a 64-column block are added as (b0 + b1) + (b2 + b3).  Off-diagonal
    // tiles also emit the partials of the mirrored tile (column sums, bit for
    // bit the row sums of the transposed block, which a smaller tile size may
    // compute as row sums), so every row of A0 gets kp / 64 partials,
    // identical whichever tile size produced them.
    __syncthreads();
    float* part = reinterpret_cast<float*>(w + WL.part);
    const bool sq = (P.flags & kRowSq) != 0u;   // Schatten-4: sums of A0_ij^2
    auto mag = [sq](float x) { return sq ? x * x : fabsf(x); };
    constexpr int NB = T / 16;
    float* rs = reinterpret_cast<float*>(smem);       // [NB][T] row sums over 16-column blocks
    float* cs = rs + NB * T;                          // [NB][T] column sums over 16-row blocks
    const int lane = threadIdx.x & 63;
    const int wm = wave_m(Tile<T>::WGN), wn = wave_n(Tile<T>::WGN);
#pragma unroll
    for (int fm = 0; fm < FM; ++fm)
#pragma unroll
      for (int fn = 0; fn < FN; ++fn) {
        // row sums: lanes 16 g .. 16 g + 15 hold the 16 columns of rows
        // 4 g + v; butterfly over lane bits 0..3
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          float x = mag(acc[fm][fn][v]);
#pragma unroll
          for (int off = 1; off <= 8; off <<= 1) x += __shfl_xor(x, off, 64);
          if ((lane & 15) == 0) rs[((wn * Tile<T>::TWN) / 16 + fn) * T + acc_row<T>(wm, fm) + v] = x;
        }
        // column sums: row bits 0, 1 are v's, bits 2, 3 the lane's bits 4, 5
        const float y = (mag(acc[fm][fn][0]) + mag(acc[fm][fn][1])) +
                        (mag(acc[fm][fn][2]) + mag(acc[fm][fn][3]));
        float col = y + __shfl_xor(y, 16, 64);
        col += __shfl_xor(col, 32, 64);
        if (lane < 16) cs[((wm * Tile<T>::TWM) / 16 + fm) * T + acc_col<T>(wn, fn)] = col;
      }
    __syncthreads();
    constexpr int NB64 = T / 64;
    for (int q = threadIdx.x; q < NB64 * T; q += Tile<T>::NT) {
      const int b = q / T, r = q - b * T;
      const float* x = rs + (4 * b) * T + r;
      part[int64_t(J * NB64 + b) * kp + I * T + r] = (x[0] + x[T]) + (x[2 * T] + x[3 * T]);
      if (I != J) {
        const float* y = cs + (4 * b) * T + r;
        part[int64_t(I * NB64 + b) * kp + J * T + r] = (y[0] + y[T]) + (y[2 * T] + y[3 * T]);
      }
    }
  }
}

// B~ = b A + c A A + a I (upper tiles, mirrored).  The stage is preloaded with
// A's tile (J, I), whose element (j, i) equals A_ij.
template <int T, int BK, bool SCALED>
__global__ __launch_bounds__(Tile<T>::NTT) void k_poly_fast(const Phase P) {
  __shared__ __attribute__((aligned(1024))) char smem[smem_bytes<T, BK>()];
  constexpr int FM = Tile<T>::FM, FN = Tile<T>::FN;
  Loc L;
  int I, J;
  if (!sym_tile<T>(P, L, I, J)) return;
  const Entry& E = P.e[L.ent];
  const int kp = int(E.kp);
  char* w = ws_of(P, E, L.mat);
  const WsLayout WL = ws_layout(E.kp, E.Np, 2);
  const uint16_t* A = reinterpret_cast<const uint16_t*>(w + WL.a);
  uint16_t* B = reinterpret_cast<uint16_t*>(w + WL.b);
  const int64_t ldg = WL.ldg;
  AccT<T> acc;
  if (!run_mainloop<T, false, false, BK>(acc, smem, A + int64_t(I) * T * ldg, ldg, A + int64_t(J) * T * ldg, ldg, kp)) return;
  load_rows<T>(smem, A, ldg, int64_t(J) * T, int64_t(I) * T);
  __syncthreads();
  const float a = P.a, b = P.b, c = P.c;
  const bool diag = I == J;
  auto f = [=](int i, int j, float x, uint16_t aij) {
    return b * bf2f(aij) + c * x + ((diag && i == j) ? a : 0.f);
  };
  if constexpr (SCALED)   // kScale: a separate kernel, so that neither epilogue spills
    epilogue_sym_scaled<T>(acc, smem, B, ldg, I, J, f, reinterpret_cast<const float*>(w + WL.s));
  else
    epilogue_sym<T>(acc, smem, B, ldg, I, J, f);
}

// Y' = B~ Y.  The operands are fed transposed so that each lane holds 4
// consecutive columns of an output row; the tile goes out through the stage.
// dst = kSlotFinal writes the caller's matrix (tall: transposed), otherwise
// the workspace slot.
template <int T, int BK>
__global__ __launch_bounds__(Tile<T>::NT) void k_update_fast(const Phase P) {
  __shared__ __attribute__((aligned(1024))) char smem[smem_bytes<T, BK>()];
  constexpr int FM = Tile<T>::FM, FN = Tile<T>::FN;
  // Logical tile -> (block row, block column) in groups of 4 block rows, so
  // that concurrently running tiles share rows of B~.  Under kTail the launch
  // covers the logical tiles (of size F T) from P.tail_base on as F x F
  // sub-tiles, one per block (F = 2, or 4 with kTail4).
  const bool tail = (P.flags & kTail) != 0u;
  const int F = !tail ? 1 : ((P.flags & kTail4) ? 4 : 2);
  const int FF = F * F;
  Loc L;
  if (tail) L = locate(P, P.tail_base + int(blockIdx.x) / FF);
  else if (!(P.flags & kByMatrix)) L = locate(P, xcd_remap(blockIdx.x, P.total));
  else if (!locate_by_matrix(P, int(blockIdx.x), L)) return;
  const Entry& E = P.e[L.ent];
  const int kp = int(E.kp), Np = int(E.Np), k = int(E.k), N = int(E.N);
  const int TL = F * T;
  const int nI = kp / TL, nL = Np / TL;
  constexpr int GM = 4;
  const int grp = L.tile / (GM * nL);
  const int first = grp * GM;
  const int gsz = min(nI - first, GM);
  const int rem = L.tile - grp * GM * nL;
  const int sub = tail ? int(blockIdx.x) % FF : 0;
  const int I = F * (first + rem % gsz) + sub / F;
  const int Lb = F * (rem / gsz) + sub % F;

  char* w = ws_of(P, E, L.mat);
  const WsLayout WL = ws_layout(E.kp, E.Np, 2);
  const uint16_t* B = reinterpret_cast<const uint16_t*>(w + WL.b);
  const uint16_t* Y = wbuf(P, E, L.mat, P.src);
  const int64_t ldg = WL.ldg, ldy = WL.ldy;
  AccT<T> acc;
  run_mainloop<T, true, true, BK>(acc, smem, B + int64_t(I) * T * ldg, ldg, Y + int64_t(Lb) * T, ldy, kp);

  // acc[fm][fn] element u: output row i = wm*TWM + fm*16 + lane%16, column
  // l0 + u with l0 = 16 (fn WGN + wn) + 4(lane/16) (the waves' column blocks
  // interleave, as the operand reads of the row-major Y stage assign them)
  const int lane = threadIdx.x & 63;
  const int wm = wave_m(Tile<T>::WGN), wn = wave_n(Tile<T>::WGN);
#pragma unroll
  for (int fm = 0; fm < FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < FN; ++fn) {
      const int i = wm * Tile<T>::TWM + fm * 16 + (lane & 15);
      const int l0 = 16 * (fn * Tile<T>::WGN + wn) + 4 * (lane >> 4);
      uint16_t out[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) out[u] = f2bf(acc[fm][fn][u]);
      *reinterpret_cast<uint2*>(smem + i * Stage<T>::RS + l0 * 2) = *reinterpret_cast<const uint2*>(out);
    }
  __syncthreads();
  if (P.dst != kSlotFinal)
    store_rows<T>(smem, wbuf(P, E, L.mat, P.dst), ldy, int64_t(I) * T, int64_t(Lb) * T);
  else if ((E.flags & kTall) == 0u)
    store_rows_user<T>(smem, user_of(P, E, L.mat), k, N, I * T, Lb * T);
  else
    store_cols_user<T>(smem, user_of(P, E, L.mat), k, N, I * T, Lb * T);
}

// W1 = X (wide) or X^T (tall) in the padded layout, zeros outside the matrix.
// One block per 64 x 64 tile of W1; each thread moves 8 consecutive elements
// of two rows, with 16-byte loads where the row allows them and 16-byte
// stores.  Tall: X is N x k row-major and W1's row i is X's column i; the
// tile goes through LDS, whose rows of 66 elements (33 words, an odd count)
// spread the column reads over the banks.
__global__ __launch_bounds__(256) void k_load_in(const Phase P) {
  __shared__ __attribute__((aligned(16))) uint16_t tile[kTransposeTile][kTransposeTile + 2];
  const Loc L = locate(P, blockIdx.x);
  const Entry& E = P.e[L.ent];
  const int k = int(E.k), N = int(E.N);
  const int64_t ldy = ws_layout(E.kp, E.Np, 2).ldy;
  const int nI = int(E.kp) / kTransposeTile;
  const int ti = L.tile % nI, tl = L.tile / nI;
  const uint16_t* X = user_of(P, E, L.mat);
  uint16_t* W = wbuf(P, E, L.mat, kSlotFirst);
  const bool tall = (E.flags & kTall) != 0u;
  if (tall) {
    const int c8 = threadIdx.x & 7, r0 = threadIdx.x >> 3;
    const int i0 = ti * kTransposeTile + c8 * 8;
    const bool vec = (k % 8) == 0 && (reinterpret_cast<uintptr_t>(X) & 15u) == 0u;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int r = r0 + 32 * h, l = tl * kTransposeTile + r;   // tile row r = X row l
      uint4 v = make_uint4(0u, 0u, 0u, 0u);
      if (l < N && vec && i0 + 8 <= k) {
        v = *reinterpret_cast<const uint4*>(X + int64_t(l) * k + i0);
      } else if (l < N) {
        uint16_t* e = reinterpret_cast<uint16_t*>(&v);
        for (int u = 0; u < 8; ++u) e[u] = i0 + u < k ? X[int64_t(l) * k + i0 + u] : uint16_t(0);
      }
      uint32_t* d = reinterpret_cast<uint32_t*>(&tile[r][c8 * 8]);   // 4-byte aligned
      d[0] = v.x;
      d[1] = v.y;
      d[2] = v.z;
      d[3] = v.w;
    }
    __syncthreads();
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int rr = r0 + 32 * h, i = ti * kTransposeTile + rr;   // tile column rr = W1 row i
      uint4 v;
      uint16_t* e = reinterpret_cast<uint16_t*>(&v);
#pragma unroll
      for (int u = 0; u < 8; ++u) e[u] = tile[c8 * 8 + u][rr];
      *reinterpret_cast<uint4*>(W + int64_t(i) * ldy + tl * kTransposeTile + c8 * 8) = v;
    }
  } else {
    const bool vec = (N % 8) == 0 && (reinterpret_cast<uintptr_t>(X) & 15u) == 0u;
    const int c8 = threadIdx.x & 7, r0 = threadIdx.x >> 3;
    const int l = tl * kTransposeTile + c8 * 8;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int i = ti * kTransposeTile + r0 + 32 * h;
      uint4 v = make_uint4(0u, 0u, 0u, 0u);
      if (i < k && vec && l + 8 <= N) {
        v = *reinterpret_cast<const uint4*>(X + int64_t(i) * N + l);
      } else if (i < k) {
        uint16_t* e = reinterpret_cast<uint16_t*>(&v);
        for (int u = 0; u < 8; ++u) e[u] = l + u < N ? X[int64_t(i) * N + l + u] : uint16_t(0);
      }
      *reinterpret_cast<uint4*>(W + int64_t(i) * ldy + l) = v;
    }
  }
}

// First iteration after the scaling: A1 = bf16(s_i A0_ij s_j).  The Gram
// stored A0 (fp32) as its upper tiles only, which contain every upper 64 x 64
// tile whatever its tile size; one block per upper 64 x 64 tile (I <= J)
// reads it once and writes A1's tile (I, J) and, off the diagonal, its
// transpose (J, I) through LDS (s_i s_j = s_j s_i, so the mirror holds the
// same values).  Thread: row tid / 4 of the tile, 16 columns.  Under kFuseS
// the block first forms s for its 64 rows and 64 columns from the Gram's row
// partials, and the diagonal blocks store s for the first polynomial.
__global__ __launch_bounds__(256) void k_apply_s(const Phase P) {
  __shared__ uint16_t tt[64][64 + 2];
  __shared__ float sv[128];   // s of the tile's 64 rows, then of its 64 columns
  const Loc L = locate(P, blockIdx.x);
  const Entry& E = P.e[L.ent];
  const int kp = int(E.kp);
  char* w = ws_of(P, E, L.mat);
  const WsLayout WL = ws_layout(E.kp, E.Np, 2);
  float* s = reinterpret_cast<float*>(w + WL.s);
  const float* A0 = reinterpret_cast<const float*>(w + WL.a32);
  uint16_t* A = reinterpret_cast<uint16_t*>(w + WL.a);
  int I, J;
  tri_tile(L.tile, kp / 64, I, J);
  if (threadIdx.x < 128) {
    const int q = int(threadIdx.x);
    const int x = (q < 64 ? I : J) * 64 + (q & 63);
    float v;
    if (P.flags & kFuseS) {
      // s_x = 1 / sqrt(sum of |A0_xj|), the row partials added in column-block
      // order exactly as the separate AOL-vector kernel adds them
      const float* part = reinterpret_cast<const float*>(w + WL.part);
      const int nb = int(cdiv(E.kp, uint32_t(P.aux)));
      float rs = 0.f;
      if (x < int(E.k))
        for (int b = 0; b < nb; ++b) rs += part[int64_t(b) * kp + x];
      v = rs >= 1.17549435e-38f ? 1.0f / sqrtf(rs) : 0.f;   // padding rows: 0
      if (I == J && q < 64) s[x] = v;   // for the first polynomial
    } else {
      v = s[x];
    }
    sv[q] = v;
  }
  __syncthreads();
  const int r = int(threadIdx.x) >> 2, c0 = (int(threadIdx.x) & 3) * 16;
  const int i = I * 64 + r, j0 = J * 64 + c0;
  const float si = sv[r];
  const float* src = A0 + int64_t(i) * kp + j0;
  uint16_t o[16];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const float4 v = *reinterpret_cast<const float4*>(src + 4 * q);
    o[4 * q + 0] = f2bf(v.x * (si * sv[64 + c0 + 4 * q + 0]));
    o[4 * q + 1] = f2bf(v.y * (si * sv[64 + c0 + 4 * q + 1]));
    o[4 * q + 2] = f2bf(v.z * (si * sv[64 + c0 + 4 * q + 2]));
    o[4 * q + 3] = f2bf(v.w * (si * sv[64 + c0 + 4 * q + 3]));
  }
  uint16_t* dst = A + int64_t(i) * WL.ldg + j0;
  reinterpret_cast<uint4*>(dst)[0] = reinterpret_cast<const uint4*>(o)[0];
  reinterpret_cast<uint4*>(dst)[1] = reinterpret_cast<const uint4*>(o)[1];
  if (I == J) return;   // uniform per block
#pragma unroll
  for (int e = 0; e < 16; ++e) tt[r][c0 + e] = o[e];
  __syncthreads();
  // mirror row J*64 + r, columns I*64 + c0 .. + 15 = tile column r
  uint16_t m[16];
#pragma unroll
  for (int e = 0; e < 16; ++e) m[e] = tt[c0 + e][r];
  uint16_t* d2 = A + int64_t(J * 64 + r) * WL.ldg + I * 64 + c0;
  reinterpret_cast<uint4*>(d2)[0] = reinterpret_cast<const uint4*>(m)[0];
  reinterpret_cast<uint4*>(d2)[1] = reinterpret_cast<const uint4*>(m)[1];
}

#define TM_LAUNCH(kern) \
  do { hipLaunchKernelGGL(kern, dim3(P.total), dim3(Tile<T>::NTT), 0, st, P); return hipGetLastError(); } while (0)

template <int T, int BK>
static hipError_t launch_t(int kind, const Phase& P, hipStream_t st) {
  switch (kind) {
    case kKindGram: TM_LAUNCH((k_gram_fast<T, BK>));
    case kKindPoly:
      if (P.flags & kScale) TM_LAUNCH((k_poly_fast<T, BK, true>));
      TM_LAUNCH((k_poly_fast<T, BK, false>));
    case kKindUpdate:
      if constexpr (T >= 64) {   // layout tiles only; no producer waves
        hipLaunchKernelGGL((k_update_fast<T, BK>), dim3(P.total), dim3(Tile<T>::NT), 0, st, P);
        return hipGetLastError();
      }
      break;
  }
  return hipErrorInvalidValue;
}

}  // namespace fast

hipError_t launch_fast_bf16(int kind, int cfg, int step, const Phase& P, hipStream_t st) {
  if (P.total <= 0) return hipSuccess;
  if (kind == kKindLoadIn) {
    hipLaunchKernelGGL(fast::k_load_in, dim3(P.total), dim3(256), 0, st, P);
    return hipGetLastError();
  }
  if (kind == kKindScaleA) {
    hipLaunchKernelGGL(fast::k_apply_s, dim3(P.total), dim3(256), 0, st, P);
    return hipGetLastError();
  }
  switch (cfg_tile(cfg)) {
    case 256: return fast::launch_t<256, fast::kPingPongBK>(kind, P, st);
    case 128:
      return step == 64 ? fast::launch_t<128, 64>(kind, P, st) : fast::launch_t<128, 32>(kind, P, st);
    case 64:
      return step == 128 ? fast::launch_t<64, 128>(kind, P, st)
             : step == 64 ? fast::launch_t<64, 64>(kind, P, st)
                          : fast::launch_t<64, 32>(kind, P, st);
    case 32:
      if (kind == kKindUpdate || (kind == kKindGram && (P.flags & kRowSum))) break;
      return step == 128 ? fast::launch_t<32, 128>(kind, P, st) : fast::launch_t<32, 32>(kind, P, st);
  }
  return hipErrorInvalidValue;
}

}  // namespace tmk
