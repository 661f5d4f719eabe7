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
// accumulates 32 x 32 v_mfma_f32_32x32x16_bf16 blocks.  Operands reach LDS
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
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef short s16x4_t __attribute__((ext_vector_type(4)));

// Tile T x T computed by NW wave64s in a WGM x WGN grid (2 x 4, 2 x 2, or a
// single wave for the 32 tile); each wave owns TWM x TWN of the output as
// 32 x 32 MFMA blocks.
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
  static constexpr int FM = TWM / 32, FN = TWN / 32;
};

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
// starts at the tile's first row (kc) or the stage's first row (rm), so an
// offset spans at most 256 rows of a row of at most 65536 + 7 elements.
//
// K-contiguous operand: T rows x BK bf16 in the swizzled row layout of Ring.
// One instruction fills 1 KB = 64 / CPR rows; lane i writes chunk i % CPR of
// its row, i.e. it loads logical chunk (i % CPR) ^ swizzle.
template <int T, int BK>
__device__ inline void dma_kc(const uint16_t* src, int64_t ld, int k0, uint32_t lds, int q) {
  using R = Ring<T, BK>;
  constexpr int RPI = 64 / R::CPR;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int j = wave + Tile<T>::NW * q;
  const int r = j * RPI + lane / R::CPR;
  const int c = (lane % R::CPR) ^ ((r / R::RPB) % R::CPR);
  const uint32_t voff = uint32_t((int64_t(r) * ld + k0 + c * 8) * 2);
  dma16(src, voff, __builtin_amdgcn_readfirstlane(lds + uint32_t(j) * 1024u));
}

// The same 1 KB instructions split over NI issuing waves (w = 0 .. NI - 1):
// instruction q of wave w fills 1 KB block w + NI q of the operand stage.
template <int T, int BK, int NI>
__device__ inline void dma_kc_w(const uint16_t* src, int64_t ld, int k0, uint32_t lds, int q, int w) {
  using R = Ring<T, BK>;
  constexpr int RPI = 64 / R::CPR;
  const int lane = threadIdx.x & 63;
  const int j = w + NI * q;
  const int r = j * RPI + lane / R::CPR;
  const int c = (lane % R::CPR) ^ ((r / R::RPB) % R::CPR);
  const uint32_t voff = uint32_t((int64_t(r) * ld + k0 + c * 8) * 2);
  dma16(src, voff, __builtin_amdgcn_readfirstlane(lds + uint32_t(j) * 1024u));
}

template <int T, int BK>
__device__ inline void issue_kc(const uint16_t* src, int64_t ld, int k0, uint32_t lds) {
#pragma unroll
  for (int q = 0; q < Ring<T, BK>::DMA_OP; ++q) dma_kc<T, BK>(src, ld, k0, lds, q);
}

// 32-byte chunk swizzle of the row-major Y stage (row = 2T bytes).
template <int T>
__device__ inline int swz_y(int r) {
  return T >= 128 ? 2 * (r & 3) : 2 * ((r >> 1) & 1);
}

// Row-major operand (the update's Y): BK rows (K) x T columns, row = 2T bytes.
// The stage's first row goes into the 64-bit base address, so the 32-bit
// per-lane offset spans BK rows only, whatever the matrix size.
template <int T, int BK>
__device__ inline void dma_rm(const uint16_t* src, int64_t ld, int k0, uint32_t lds, int q) {
  constexpr int ROWB = 2 * T;
  constexpr int LPR = ROWB / 16;          // lanes per row
  constexpr int RPI = 1024 / ROWB;        // rows per instruction
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint16_t* base = src + int64_t(k0) * ld;
  const int j = wave + Tile<T>::NW * q;
  const int r = j * RPI + lane / LPR;
  const int p16 = lane % LPR;
  const int c = (p16 >> 1) ^ swz_y<T>(r);
  const uint32_t voff = uint32_t((int64_t(r) * ld + c * 16 + (p16 & 1) * 8) * 2);
  dma16(base, voff, __builtin_amdgcn_readfirstlane(lds + uint32_t(j) * 1024u));
}

// ---------------------------------------------------------------- compute
template <int T>
struct Frags {
  uint4 a[Tile<T>::FM], b[Tile<T>::FN];
};

// MFMA operands of K slice kk (16 wide) of one stage.
template <int T, bool RM, int BK>
__device__ inline void load_frags(Frags<T>& fr, const char* sa, const char* sb, int kk, int wm,
                                  int wn) {
  constexpr int FM = Tile<T>::FM, FN = Tile<T>::FN;
  using R = Ring<T, BK>;
  const int lane = threadIdx.x & 63;
  const int lr = lane & 31, lh = lane >> 5;
  const int c = 2 * kk + lh;
#pragma unroll
  for (int f = 0; f < FM; ++f) {
    const int r = wm * Tile<T>::TWM + f * 32 + lr;
    fr.a[f] = *reinterpret_cast<const uint4*>(sa + r * R::RB + 16 * (c ^ ((r / R::RPB) % R::CPR)));
  }
  if constexpr (!RM) {
#pragma unroll
    for (int f = 0; f < FN; ++f) {
      const int r = wn * Tile<T>::TWN + f * 32 + lr;
      fr.b[f] = *reinterpret_cast<const uint4*>(sb + r * R::RB + 16 * (c ^ ((r / R::RPB) % R::CPR)));
    }
  } else {
    // Lane q of 16-lane group g addresses row kb + q/4, columns n + 4(q%4);
    // the transposed read returns rows kb..kb+3 of column n + q.
    const int g = lane >> 4, q = lane & 15;
    const int kb = 16 * kk + 8 * (g >> 1) + (q >> 2);
#pragma unroll
    for (int f = 0; f < FN; ++f) {
      const int chunk = (wn * Tile<T>::TWN + f * 32) / 16 + (g & 1);
      s16x4_t v[2];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int row = kb + 4 * h;
        const char* p = sb + row * (2 * T) + 32 * (chunk ^ swz_y<T>(row)) + 8 * (q & 3);
        v[h] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (__attribute__((address_space(3))) s16x4_t*)(lds_addr(p)));
      }
      fr.b[f] = __builtin_bit_cast(uint4, v);
    }
  }
}

// SWAP = false: acc[fm][fn] holds C block (fm, fn) in the MFMA layout (lane
// L, element v: row 8(v/4) + 4(L/32) + v%4, column L%32).  SWAP = true feeds
// the operands the other way round, so acc[fm][fn] holds the transposed block:
// each lane then owns 4 consecutive columns of one C row.
template <int T, bool SWAP>
__device__ inline void mma(f32x16_t (&acc)[Tile<T>::FM][Tile<T>::FN], const Frags<T>& fr) {
#pragma unroll
  for (int fm = 0; fm < Tile<T>::FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < Tile<T>::FN; ++fn) {
      if constexpr (SWAP)
        acc[fm][fn] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            __builtin_bit_cast(bf16x8_t, fr.b[fn]), __builtin_bit_cast(bf16x8_t, fr.a[fm]),
            acc[fm][fn], 0, 0, 0);
      else
        acc[fm][fn] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            __builtin_bit_cast(bf16x8_t, fr.a[fm]), __builtin_bit_cast(bf16x8_t, fr.b[fn]),
            acc[fm][fn], 0, 0, 0);
    }
}

// 4-wave main loop of the update's 128 and 64 tiles.  acc = A (T x K,
// K-contiguous rows of a) * B^T where B's rows are the K-contiguous rows of b
// (RM = false) or B = the K x T row-major block of b (RM = true); K is a
// multiple of BK and every tile is full.  The
// operands of each 16-wide K slice are read from LDS while the previous
// slice's MFMAs run.  The DMA is spread over the K slices: while stage kt is
// read and multiplied, each wave issues its share of stage kt + NSTAGE - 1,
// PS / NS instructions per slice, into the buffer of stage kt - 1 (every wave
// finished reading it before the barrier that opened stage kt).  The
// global -> LDS path (about 64 bytes per clock and compute unit) is then fed
// evenly instead of in one burst per stage that stalls every wave.  Slices
// are consumed in increasing order whatever BK is, so every output element
// accumulates the same products in the same order.
template <int T, bool RM, bool SWAP, int BK>
__device__ inline void mainloop(f32x16_t (&acc)[Tile<T>::FM][Tile<T>::FN], char* smem,
                                const uint16_t* a, int64_t lda, const uint16_t* b,
                                int64_t ldb, int K) {
  using R = Ring<T, BK>;
  constexpr int PS = R::PER_STAGE, NS = BK / 16, NST = R::NSTAGE, DO = R::DMA_OP;
  constexpr int PPS = PS / NS;
  static_assert(PPS * NS == PS && PPS >= 1, "whole DMA instructions per slice");
  const int wave = threadIdx.x >> 6;
  const int wm = wave / Tile<T>::WGN, wn = wave % Tile<T>::WGN;
#pragma unroll
  for (int fm = 0; fm < Tile<T>::FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < Tile<T>::FN; ++fn)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[fm][fn][v] = 0.f;

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
  for (int kt = 0; kt < nk; ++kt) {
    const char* st = stage_ptr(kt);
    const int nx = kt + NST - 1;   // stage refilled during this one
    const bool fill = nx < nk;
#pragma unroll
    for (int s = 0; s < NS; s += 2) {
      load_frags<T, RM, BK>(f1, st, st + R::A_BYTES, s + 1, wm, wn);
      if (fill)
#pragma unroll
        for (int i = 0; i < PPS; ++i) dma_one(nx, s * PPS + i);
      mma<T, SWAP>(acc, f0);
      if (s + 2 < NS) {
        load_frags<T, RM, BK>(f0, st, st + R::A_BYTES, s + 2, wm, wn);
        if (fill)
#pragma unroll
          for (int i = 0; i < PPS; ++i) dma_one(nx, (s + 1) * PPS + i);
        mma<T, SWAP>(acc, f1);
      } else {
        if (fill)
#pragma unroll
          for (int i = 0; i < PPS; ++i) dma_one(nx, (s + 1) * PPS + i);
        __builtin_amdgcn_sched_barrier(0);
        if (kt + 1 < nk) {
          ring_wait<PS, NST - 2>(min(nk - 1, kt + NST - 1) - (kt + 1));
          const char* nxp = stage_ptr(kt + 1);
          load_frags<T, RM, BK>(f0, nxp, nxp + R::A_BYTES, 0, wm, wn);
        }
        __builtin_amdgcn_sched_barrier(0);
        mma<T, SWAP>(acc, f1);
      }
    }
  }
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
// compute waves multiply stage kt, loading the operands of each 16-wide
// slice while the previous slice's MFMAs run, and finish their LDS reads
// before the barrier.  Slices are consumed in increasing K order, so every
// output element accumulates the same products in the same order as in the
// other loops.  The producer waves return afterwards; a barrier then waits
// only for the waves still running.
template <int T, bool SWAP, int BK>
__device__ inline bool mainloop_pc(f32x16_t (&acc)[Tile<T>::FM][Tile<T>::FN], char* smem,
                                   const uint16_t* a, int64_t lda, const uint16_t* b,
                                   int64_t ldb, int K) {
  using R = Ring<T, BK>;
  constexpr int NW = Tile<T>::NW, NP = Tile<T>::NP, NS = BK / 16, NST = R::NSTAGE;
  constexpr int DOP = T * BK / 512 / NP;     // 1 KB DMAs per producer and operand stage
  constexpr int PSP = 2 * DOP;
  static_assert(NP >= 1 && DOP * NP * 512 == T * BK, "whole DMA instructions per producer");
  static_assert(NS % 2 == 0, "slices in pairs");
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
#pragma unroll
  for (int fm = 0; fm < Tile<T>::FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < Tile<T>::FN; ++fn)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[fm][fn][v] = 0.f;
  barrier_pinned();   // stage 0 has landed
  Frags<T> f0, f1;
  load_frags<T, false, BK>(f0, stage_ptr(0), stage_ptr(0) + R::A_BYTES, 0, wm, wn);
  for (int kt = 0; kt < nk; ++kt) {
    const char* st = stage_ptr(kt);
#pragma unroll
    for (int s = 0; s < NS; s += 2) {
      load_frags<T, false, BK>(f1, st, st + R::A_BYTES, s + 1, wm, wn);
      mma<T, SWAP>(acc, f0);
      if (s + 2 < NS) {
        load_frags<T, false, BK>(f0, st, st + R::A_BYTES, s + 2, wm, wn);
        mma<T, SWAP>(acc, f1);
      } else {
        __builtin_amdgcn_sched_barrier(0);
        __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0): stage kt is read
        barrier_pinned();                     // and stage kt + 1 has landed
        if (kt + 1 < nk) {
          const char* nxp = stage_ptr(kt + 1);
          load_frags<T, false, BK>(f0, nxp, nxp + R::A_BYTES, 0, wm, wn);
        }
        __builtin_amdgcn_sched_barrier(0);
        mma<T, SWAP>(acc, f1);
      }
    }
  }
  return true;
}

// Ping-pong schedule of the 8-wave tile (mainloop_pp_kc5 below).  Waves 0-3
// (group 0) and 4-7 (group 1) occupy one slot per SIMD each; group 1 runs
// one phase behind, so that while one wave of a SIMD issues the 16 MFMAs of
// a 32-wide K step from registers, the other issues its DMA and reads its
// operands of the next step from LDS.  Every phase ends
// with a workgroup barrier:
//   group 0: [MEM(h) | COMP(h)] for each 32-wide step h, then one idle phase;
//   group 1: one idle phase, then [MEM(h) | COMP(h)].
// Stages are 64 K elements wide (two steps), so a K-contiguous row of a
// stage is one full 128-byte line, which the global -> LDS path moves at
// twice the rate of 64-byte half lines.  That path takes about 64 bytes per
// clock and compute unit, so the loop issues one operand stage (32 KB per
// workgroup) per step rather than a whole stage every other step.  The data
// a step reads must be in LDS before group 0's MEM of that step: at the end
// of the step before, group 0 waits for its own DMAs at the end of its COMP,
// group 1 at the end of its MEM (together with its LDS reads), both before
// the same barrier.  A buffer is refilled only after the barrier that ends
// its last reader's MEM phase.  A MEM phase issues its LDS reads before its
// DMA: issuing a DMA stalls the wave while the compute unit's queue drains,
// and that stall then overlaps the reads' completion instead of delaying
// their start.

// Ping-pong loop of the 8-wave tile: operand a K-contiguous rows (of Y for
// the Gram, of A for the polynomial, of B~ for the update), operand b
// K-contiguous rows too (RM = false) or the update's K x T row-major block of
// Y (RM = true).  A stage of K-contiguous rows cannot be split along K
// without halving its 128-byte row pieces, so instead of two stages the ring
// holds five operand slots of one operand stage each (the whole 160 KB),
// filled in the order a(0), b(0), a(1), b(1), ...: operand stage i goes into
// slot i % 5.  The slot of a(j + 2) is that of b(j - 1) and the slot of
// b(j + 1) that of a(j - 1), both free once stage j - 1 has been read, so the
// first step of stage j issues b(j + 1) and the second a(j + 2): one operand
// stage per step.  At the end of stage j's second step every wave waits for
// a(j + 1) and b(j + 1), leaving a(j + 2) in flight; five consecutive operand
// stages are live at most (a(j), b(j) read, a(j + 1), b(j + 1), a(j + 2)).
template <int T, bool RM, bool SWAP, int BK>
__device__ inline void mainloop_pp_kc5(f32x16_t (&acc)[Tile<T>::FM][Tile<T>::FN], char* smem,
                                       const uint16_t* a, int64_t lda, const uint16_t* b,
                                       int64_t ldb, int K) {
  static_assert(Tile<T>::NW == 8, "ping-pong needs two waves per SIMD");
  using R = Ring<T, BK>;
  constexpr int DO = R::DMA_OP, SLOTS = 5;
  static_assert(BK == 64, "two 32-wide steps per stage");
  static_assert(SLOTS * R::A_BYTES <= R::LDS, "five operand slots");
  const int wave = threadIdx.x >> 6;
  const int wm = wave / 4, wn = wave % 4;
  const bool g1 = __builtin_amdgcn_readfirstlane(wave) >= 4;
#pragma unroll
  for (int fm = 0; fm < Tile<T>::FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < Tile<T>::FN; ++fn)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[fm][fn][v] = 0.f;

  const uint32_t lds0 = lds_addr(smem);
  const int nk = K / BK;
  auto slot_lds = [&](int i) { return lds0 + uint32_t((i % SLOTS) * R::A_BYTES); };
  auto slot_ptr = [&](int i) { return smem + (i % SLOTS) * R::A_BYTES; };
  auto issue_a = [&](int kt) { issue_kc<T, BK>(a, lda, kt * BK, slot_lds(2 * kt)); };
  auto issue_b = [&](int kt) {
    if constexpr (RM) {
#pragma unroll
      for (int q = 0; q < DO; ++q) dma_rm<T, BK>(b, ldb, kt * BK, slot_lds(2 * kt + 1), q);
    } else {
      issue_kc<T, BK>(b, ldb, kt * BK, slot_lds(2 * kt + 1));
    }
  };

  issue_a(0);
  issue_b(0);
  if (nk > 1) {
    issue_a(1);
    __builtin_amdgcn_s_waitcnt(0xC07F);
    ring_sync_dma<DO>();
  } else {
    __builtin_amdgcn_s_waitcnt(0xC07F);
    ring_sync_dma<0>();
  }
  if (g1) barrier_pinned();

  Frags<T> f0, f1;
  for (int j = 0; j < nk; ++j) {
    const char* sa = slot_ptr(2 * j);
    const char* sb = slot_ptr(2 * j + 1);
#pragma unroll
    for (int hs = 0; hs < 2; ++hs) {
      // MEM
      load_frags<T, RM, BK>(f0, sa, sb, 2 * hs, wm, wn);
      load_frags<T, RM, BK>(f1, sa, sb, 2 * hs + 1, wm, wn);
      if (hs == 0) {
        if (j + 1 < nk) issue_b(j + 1);
      } else {
        if (j + 2 < nk) issue_a(j + 2);
      }
      if (g1) {
        __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0)
        if (hs == 1) {
          if (j + 2 < nk) dma_wait<DO>();
          else dma_wait<0>();
        }
      }
      barrier_pinned();
      // COMP
      mma<T, SWAP>(acc, f0);
      mma<T, SWAP>(acc, f1);
      if (!g1 && hs == 1) {
        if (j + 2 < nk) dma_wait<DO>();
        else dma_wait<0>();
      }
      barrier_pinned();
    }
  }
  if (!g1) barrier_pinned();
  __builtin_amdgcn_s_waitcnt(0xC07F);
  dma_wait<0>();
}

template <int T, bool RM, bool SWAP, int BK>
// Returns false in the producer waves, which then leave the kernel.
__device__ inline bool run_mainloop(f32x16_t (&acc)[Tile<T>::FM][Tile<T>::FN], char* smem,
                                    const uint16_t* a, int64_t lda, const uint16_t* b,
                                    int64_t ldb, int K) {
  if constexpr (Tile<T>::NW == 8) {
    mainloop_pp_kc5<T, RM, SWAP, BK>(acc, smem, a, lda, b, ldb, K);
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
  L = locate(P, xcd_remap(blockIdx.x, P.total));
  tri_tile(L.tile, int(P.e[L.ent].kp) / T, I, J);
  return true;
}

template <int T>
__device__ inline int acc_row(int wm, int fm, int v) {
  return wm * Tile<T>::TWM + fm * 32 + 8 * (v >> 2) + 4 * ((threadIdx.x & 63) >> 5) + (v & 3);
}
template <int T>
__device__ inline int acc_col(int wn, int fn) {
  return wn * Tile<T>::TWN + fn * 32 + (threadIdx.x & 31);
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
template <int T, class Fv>
__device__ inline void epilogue_sym(const f32x16_t (&acc)[Tile<T>::FM][Tile<T>::FN], char* st,
                                    uint16_t* D, int64_t ld, int I, int J, Fv f) {
  const int wm = wave_m(Tile<T>::WGN), wn = wave_n(Tile<T>::WGN);
#pragma unroll
  for (int fm = 0; fm < Tile<T>::FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < Tile<T>::FN; ++fn) {
      const int c = acc_col<T>(wn, fn);
#pragma unroll
      for (int v4 = 0; v4 < 4; ++v4) {
        const int r0 = acc_row<T>(wm, fm, 4 * v4);
        char* p = st + c * Stage<T>::RS + r0 * 2;
        const uint2 old = *reinterpret_cast<const uint2*>(p);
        const uint16_t* o = reinterpret_cast<const uint16_t*>(&old);
        uint16_t out[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) out[u] = f2bf(f(r0 + u, c, acc[fm][fn][4 * v4 + u], o[u]));
        *reinterpret_cast<uint2*>(p) = *reinterpret_cast<const uint2*>(out);
      }
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
__device__ inline void epilogue_sym_scaled(const f32x16_t (&acc)[Tile<T>::FM][Tile<T>::FN],
                                           char* st, uint16_t* D, int64_t ld, int I, int J, Fv f,
                                           const float* __restrict__ s) {
  constexpr int FM = Tile<T>::FM, FN = Tile<T>::FN;
  const int wm = wave_m(Tile<T>::WGN), wn = wave_n(Tile<T>::WGN);
  uint2 keep[FM][FN][4];
#pragma unroll
  for (int fm = 0; fm < FM; ++fm) {
    // s of this lane's 16 rows of the 32-row block fm (4 runs of 4 rows)
    float4 si[4];
#pragma unroll
    for (int v4 = 0; v4 < 4; ++v4)
      si[v4] = *reinterpret_cast<const float4*>(s + I * T + acc_row<T>(wm, fm, 4 * v4));
#pragma unroll
    for (int fn = 0; fn < FN; ++fn) {
      const int c = acc_col<T>(wn, fn);
      const float sj = s[J * T + c];
#pragma unroll
      for (int v4 = 0; v4 < 4; ++v4) {
        const int r0 = acc_row<T>(wm, fm, 4 * v4);
        char* p = st + c * Stage<T>::RS + r0 * 2;
        const uint2 old = *reinterpret_cast<const uint2*>(p);
        const uint16_t* o = reinterpret_cast<const uint16_t*>(&old);
        const float sv[4] = {si[v4].x, si[v4].y, si[v4].z, si[v4].w};
        uint16_t out[4], out2[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const float x = f(r0 + u, c, acc[fm][fn][4 * v4 + u], o[u]);
          out[u] = f2bf(x * sv[u]);
          out2[u] = f2bf(x * sj);
        }
        *reinterpret_cast<uint2*>(p) = *reinterpret_cast<const uint2*>(out);
        keep[fm][fn][v4] = *reinterpret_cast<const uint2*>(out2);
      }
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
    for (int fn = 0; fn < FN; ++fn) {
      const int c = acc_col<T>(wn, fn);
#pragma unroll
      for (int v4 = 0; v4 < 4; ++v4)
        *reinterpret_cast<uint2*>(st + c * Stage<T>::RS + acc_row<T>(wm, fm, 4 * v4) * 2) =
            keep[fm][fn][v4];
    }
  __syncthreads();
  store_cols<T>(st, D, ld, int64_t(I) * T, int64_t(J) * T);   // C[i][j]
}

// fp32 store of an upper tile straight from the registers (first Gram only;
// k_apply_s reads the upper tiles and writes both halves of A1).
template <int T>
__device__ inline void store_sym_f32(const f32x16_t (&acc)[Tile<T>::FM][Tile<T>::FN], float* D,
                                     int64_t ld, int I, int J) {
  const int wm = wave_m(Tile<T>::WGN), wn = wave_n(Tile<T>::WGN);
#pragma unroll
  for (int fm = 0; fm < Tile<T>::FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < Tile<T>::FN; ++fn) {
      const int j = J * T + acc_col<T>(wn, fn);
#pragma unroll
      for (int v4 = 0; v4 < 4; ++v4) {
        const int ib = I * T + acc_row<T>(wm, fm, 4 * v4);
        float m[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          m[u] = acc[fm][fn][4 * v4 + u];
          D[int64_t(ib + u) * ld + j] = m[u];
        }
      }
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
  f32x16_t acc[FM][FN];
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
    // 32 x 32 MFMA block is reduced first (a butterfly over its 32 columns for
    // the row sums, the same pairing over its 32 rows for the column sums),
    // then two adjacent 32-blocks are added.  Off-diagonal tiles also emit the
    // partials of the mirrored tile (column sums), so every row of A0 gets
    // kp / 64 partials, identical whichever tile size produced them.
    __syncthreads();
    float* part = reinterpret_cast<float*>(w + WL.part);
    const bool sq = (P.flags & kRowSq) != 0u;   // Schatten-4: sums of A0_ij^2
    auto mag = [sq](float x) { return sq ? x * x : fabsf(x); };
    constexpr int NB = T / 32;
    float* rs = reinterpret_cast<float*>(smem);       // [NB][T] row sums over 32-column blocks
    float* cs = rs + NB * T;                          // [NB][T] column sums over 32-row blocks
    const int lane = threadIdx.x & 63;
    const int wm = wave_m(Tile<T>::WGN), wn = wave_n(Tile<T>::WGN);
#pragma unroll
    for (int fm = 0; fm < FM; ++fm)
#pragma unroll
      for (int fn = 0; fn < FN; ++fn) {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          float x = mag(acc[fm][fn][v]);
#pragma unroll
          for (int off = 16; off >= 1; off >>= 1) x += __shfl_xor(x, off, 64);
          if ((lane & 31) == 0) rs[((wn * Tile<T>::TWN) / 32 + fn) * T + acc_row<T>(wm, fm, v)] = x;
        }
        // Column sums with the pairing of the row butterfly above, applied to
        // the row index 8 (v / 4) + 4 (lane / 32) + v % 4: bit 4 (v ^ 8),
        // bit 3 (v ^ 4), bit 2 (the other lane half), bit 1, bit 0.  A column
        // sum is then bit for bit the row sum of the transposed block, which
        // the mirrored tile of a smaller tile size computes as a row sum.
        float y[8];
#pragma unroll
        for (int v = 0; v < 8; ++v) y[v] = mag(acc[fm][fn][v]) + mag(acc[fm][fn][v + 8]);
#pragma unroll
        for (int v = 0; v < 4; ++v) y[v] += y[v + 4];
#pragma unroll
        for (int v = 0; v < 4; ++v) y[v] += __shfl_xor(y[v], 32, 64);
        const float col = (y[0] + y[2]) + (y[1] + y[3]);
        if (lane < 32) cs[((wm * Tile<T>::TWM) / 32 + fm) * T + acc_col<T>(wn, fn)] = col;
      }
    __syncthreads();
    constexpr int NB64 = T / 64;
    for (int q = threadIdx.x; q < NB64 * T; q += Tile<T>::NT) {
      const int b = q / T, r = q - b * T;
      part[int64_t(J * NB64 + b) * kp + I * T + r] = rs[(2 * b) * T + r] + rs[(2 * b + 1) * T + r];
      if (I != J)
        part[int64_t(I * NB64 + b) * kp + J * T + r] = cs[(2 * b) * T + r] + cs[(2 * b + 1) * T + r];
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
  f32x16_t acc[FM][FN];
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
  const Loc L = tail ? locate(P, P.tail_base + int(blockIdx.x) / FF)
                     : locate(P, xcd_remap(blockIdx.x, P.total));
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
  f32x16_t acc[FM][FN];
  run_mainloop<T, true, true, BK>(acc, smem, B + int64_t(I) * T * ldg, ldg, Y + int64_t(Lb) * T, ldy, kp);

  // acc[fm][fn] element v: output row i = wm*TWM + fm*32 + lane%32, columns
  // l0..l0+3 with l0 = wn*TWN + fn*32 + 8(v/4) + 4(lane/32)
  const int lane = threadIdx.x & 63;
  const int wm = wave_m(Tile<T>::WGN), wn = wave_n(Tile<T>::WGN);
#pragma unroll
  for (int fm = 0; fm < FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < FN; ++fn) {
      const int i = wm * Tile<T>::TWM + fm * 32 + (lane & 31);
#pragma unroll
      for (int v4 = 0; v4 < 4; ++v4) {
        const int l0 = wn * Tile<T>::TWN + fn * 32 + 8 * v4 + 4 * (lane >> 5);
        uint16_t out[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) out[u] = f2bf(acc[fm][fn][4 * v4 + u]);
        *reinterpret_cast<uint2*>(smem + i * Stage<T>::RS + l0 * 2) = *reinterpret_cast<const uint2*>(out);
      }
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
