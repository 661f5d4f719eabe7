// Shared between the host planner (tm_api.cpp) and the gfx950 kernels
// (tm_kernels.hip): launch descriptors and the per-matrix workspace layout.
#pragma once

#include <stdint.h>

#ifndef __HIPCC__
#define TM_HD inline
#else
#define TM_HD __host__ __device__ inline
#endif

namespace tmk {

TM_HD uint64_t align256(uint64_t v) { return (v + 255u) & ~uint64_t(255u); }
TM_HD uint32_t cdiv(uint32_t a, uint32_t b) { return (a + b - 1u) / b; }
TM_HD uint32_t kpad(uint32_t k) { return (k + 7u) & ~7u; }   // ld of A and B

// Matrices of one launch are described by up to kMaxEntries entries; an entry
// covers `count` matrices of one shape, stored back to back (a batched call)
// or, with kPtrTab, wherever the launch's pointer table puts them (matrices of
// one shape that follow each other in a grouped call; their workspace regions
// are consecutive).  Groups that need more entries or pointers are split into
// several launches per phase.  The descriptor stays within about 3 KB of
// kernel arguments.
constexpr int kMaxEntries = 48;
constexpr int kMaxPtrs = 96;

// Y slots named by the phase descriptors.  A slot resolves per matrix:
//   slot   wide (m <= n)          tall (m > n)
//   0      user matrix (X1)       W1 (X^T copied in)
//   1      W1                     W2
//   2      W2                     W1
//   3      user matrix            user matrix, stored transposed (N x k, ld = k)
// (fp32 path; the bf16 path pads every matrix into W1 = slot 0 first, W2 and
// W1 being slots 1 and 2, unless the entry is kDirect: then slot 0 is the
// user matrix itself.)
// Iteration 1 reads slot 0, iterations write 1, 2, 1, 2, ... and the last
// one writes slot 3, so no update ever reads the buffer it writes.
constexpr int kSlotFirst = 0;
constexpr int kSlotAlt1 = 1;
constexpr int kSlotAlt2 = 2;
constexpr int kSlotFinal = 3;

// Phase flags.
constexpr uint32_t kScale = 1u;   // first iteration after AOL / Frobenius: apply s (bf16
                                  // polynomial: store B~ diag(s))
constexpr uint32_t kRowSum = 2u;  // Gram epilogue emits AOL row-sum partials
constexpr uint32_t kFrob = 4u;    // AOL-vector kernel: uniform s from the Frobenius partials
constexpr uint32_t kA32 = 8u;     // Gram stores A0 in fp32 (first iteration, before scaling)
constexpr uint32_t kRowSq = 16u;  // with kRowSum: partials of A0_ij^2 instead of |A0_ij|
constexpr uint32_t kS4 = 32u;     // with kFrob: s = (sum of the partials)^(-1/4) (Schatten-4)
constexpr uint32_t kFromPart = 64u;  // Frobenius-partial kernel sums the Gram's row partials
constexpr uint32_t kTail = 128u;  // matrix-core kernels: blocks are 2 x 2 sub-tiles of the
                                  // tiles of twice their size from tail_base on
constexpr uint32_t kTail4 = 512u; // with kTail (update only): 4 x 4 sub-tiles of a quarter size
constexpr uint32_t kByMatrix = 1024u; // matrix-core kernels: XCD x runs every tile of the launch's
                                      // matrices x, x + 8, ... (blocks p with p % 8 == x)
constexpr uint32_t kFuseS = 256u; // bf16 rescale of A0: the AOL vector is summed in the same
                                  // kernel from the Gram's row partials (aux columns each)

// Entry flags.
constexpr uint32_t kTall = 1u;    // the user matrix is N x k (m > n); work on its transpose
constexpr uint32_t kDirect = 2u;  // bf16: the user matrix already has the padded layout (wide,
                                  // dims multiples of the tile, 16-byte aligned); iteration 1
                                  // reads it in place of the W1 copy
constexpr uint32_t kPtrTab = 4u;  // matrix j's user pointer is xp[xbase + j] of the launch

constexpr int kFrobBlocks = 32;   // partial sums of squares per matrix
constexpr int kMinTile = 64;      // smallest Gram tile: bounds the row-sum partial count

struct Entry {
  char* x;             // user matrix of element 0 (without kPtrTab)
  uint32_t ws256;      // byte offset of element 0's workspace region / 256
  uint32_t k, N;       // wide view: k = min(m, n) rows, N = max(m, n) columns
  uint32_t kp, Np;     // padded workspace dims: rows of Y, A, B and ld of A, B (kp); ld of Y (Np)
  uint32_t count;      // matrices in this entry
  uint32_t flags;      // kTall, kDirect, kPtrTab
  uint32_t tile_start; // first logical block of this entry in the launch
  uint32_t tiles_per;  // blocks per matrix in the launch
  uint32_t xbase;      // with kPtrTab: first pointer of this entry in xp
};

struct Phase {
  Entry e[kMaxEntries];
  char* ws;            // workspace base
  int32_t nent;
  int32_t total;       // logical blocks in the launch
  int32_t src, dst;    // Y slots
  float a, b, c;       // coefficients of this iteration
  uint32_t flags;
  int32_t aux;         // AOL-vector / partial kernels: columns per row partial of the Gram
  int32_t tail_base;   // with kTail: first logical tile (of size 2T) covered by the launch
  char* xp[kMaxPtrs];  // user matrices of the kPtrTab entries
};
static_assert(sizeof(Entry) == 48 && sizeof(Phase) <= 3200, "kernel arguments of one launch");

// Fused small-matrix path (bf16, every matrix of the call with k <= 128 and
// its zero-padded Y, A and B within the LDS): one workgroup per matrix runs
// every iteration in one launch.  Entries as in Phase (tiles_per = 1); the
// per-iteration coefficients travel with the launch.
constexpr int kMaxSmallEntries = 32;
constexpr int kMaxSmallPtrs = 64;
constexpr int kMaxIters = 64;           // TM_MAX_ITERS
constexpr int kSmallMaxK = 128;

struct SmallPhase {
  Entry e[kMaxSmallEntries];
  char* xp[kMaxSmallPtrs];
  float coef[kMaxIters][3];
  int32_t nent;
  int32_t total;       // workgroups (matrices) in the launch
  int32_t iters;
  int32_t precond;     // TM_PRECOND_*
};
static_assert(sizeof(SmallPhase) <= 3200, "kernel arguments of one launch");

// LDS bytes of the fused path for one matrix: Y (kp x Np), A and B (kp x kp),
// bf16 rows padded by 16 bytes, plus the row-sum scratch (kp / 16 x kp fp32),
// the scale vector and the reduction scratch (32 x 4 fp32).
TM_HD uint32_t small_kp(uint32_t k) { return (k + 31u) / 32u * 32u; }
TM_HD uint32_t small_np(uint32_t N) { return (N + 31u) / 32u * 32u; }
TM_HD uint64_t small_lds_bytes(uint32_t k, uint32_t N) {
  const uint64_t kp = small_kp(k), Np = small_np(N);
  return kp * (2 * Np + 16) + 2 * kp * (2 * kp + 16) + (kp / 16) * kp * 4 + kp * 4 + 512;
}

// Optimizer step (fp32 parameters): elementwise launches over the elements of
// up to kMaxOptEntries matrices, blocks of kOptBlock elements.
constexpr int kMaxOptEntries = 32;
constexpr int kOptBlock = 2048;

struct OptEntry {
  float* w;            // parameter, rows x cols fp32
  const float* g;      // gradient
  float* m;            // momentum buffer
  uint16_t* u;         // bf16 U, then the orthogonalized update O (library workspace)
  uint64_t size;       // rows * cols
  uint32_t block_start;  // first block of this matrix in the launch
  uint32_t vec;        // w, g, m 16-byte aligned: 4-element vectors
  float scale;         // shape factor of the update
  uint32_t pad;
};

struct OptPhase {
  OptEntry e[kMaxOptEntries];
  int32_t nent;
  int32_t nesterov;
  uint32_t total;      // blocks in the launch (each within one matrix)
  float lr, mu, wd;
};

// Tile configurations of the matrix-core kernels (square tiles, 256 threads).
constexpr int kNumCfg = 3;
// bf16 Gram (without row sums) and polynomial only: 32 x 32 tiles, one wave
// each, for phases with too few 64 x 64 tiles to fill the chip.
constexpr int kCfgSym32 = 3;
TM_HD int cfg_tile(int cfg) { return cfg == 0 ? 256 : (cfg == 1 ? 128 : (cfg == 2 ? 64 : 32)); }


// Logical blocks per matrix of each kernel.
// The numbering matches the TM_PHASE_* timing phases of turbomuon.h.
enum Kind { kKindTransposeIn, kKindFrob, kKindGram, kKindAolVector, kKindPoly,
            kKindUpdate, kKindApplyScale, kKindCopyOut, kKindLoadIn, kKindScaleA,
            kKindOptMomentum, kKindOptApply, kKindSmall, kNumKinds };
constexpr int kTransposeTile = 64;
constexpr int kElemBlock = 2048;     // elements per block of the elementwise kernels

TM_HD uint32_t tri(uint32_t nb) { return nb * (nb + 1u) / 2u; }

// k, N: wide-view dims; kp, Np: padded workspace dims.
TM_HD uint32_t blocks_per_matrix(int kind, int cfg, uint32_t k, uint32_t N, uint32_t kp,
                                 uint32_t Np) {
  const uint32_t T = uint32_t(cfg_tile(cfg));
  switch (kind) {
    case kKindTransposeIn: return cdiv(k, kTransposeTile) * cdiv(N, kTransposeTile);
    case kKindLoadIn: return cdiv(kp, kTransposeTile) * cdiv(Np, kTransposeTile);
    case kKindFrob: return uint32_t(kFrobBlocks);
    case kKindGram:
    case kKindPoly: return tri(cdiv(kp, T));
    case kKindAolVector: return cdiv(kp, 256u);
    case kKindUpdate: return cdiv(kp, T) * cdiv(Np, T);
    case kKindApplyScale:
    case kKindCopyOut: return uint32_t((uint64_t(k) * N + kElemBlock - 1) / kElemBlock);
    case kKindScaleA: return tri(kp / 64u);   // upper 64 x 64 tiles (kp % 64 == 0)
  }
  return 0;
}

struct WsLayout {
  uint64_t w1, w2, a, b, a32, s, part, fpart, total;
  uint32_t ldy, ldg;   // row strides (elements) of the Y buffers and of A, B
};

// Byte offsets of the sub-buffers of one matrix's workspace region, for
// padded dims kp x Np: Y buffers kp x Np (ld ldy = Np), A, B kp x kp (ld
// ldg = kp), the fp32 first Gram kp x kp (ld kp), s (kp floats), row-sum
// partials [ceil(kp / 64)][kp] and the Frobenius partials.
TM_HD WsLayout ws_layout(uint32_t kp, uint32_t Np, uint32_t esz) {
  WsLayout L;
  L.ldy = Np;
  L.ldg = kp;
  const uint64_t y = align256(uint64_t(kp) * L.ldy * esz);
  const uint64_t g = align256(uint64_t(kp) * L.ldg * esz);
  L.w1 = 0;
  L.w2 = L.w1 + y;
  L.a = L.w2 + y;
  L.b = L.a + g;
  L.a32 = L.b + g;
  L.s = L.a32 + align256(uint64_t(kp) * kp * 4u);
  L.part = L.s + align256(uint64_t(kp) * 4u);
  L.fpart = L.part + align256(uint64_t(cdiv(kp, kMinTile)) * kp * 4u);
  L.total = L.fpart + align256(uint64_t(kFrobBlocks) * 4u);
  return L;
}

// Padded dims of the generic (fp32) path: A and B rows padded to 8 for
// 16-byte row alignment, Y unpadded.
TM_HD void generic_dims(uint32_t k, uint32_t N, uint32_t* kp, uint32_t* Np) {
  *kp = kpad(k);
  *Np = N;
}

// Padded dims of the bf16 matrix-core path with square tiles of size T:
// every tile is full and the padding is kept at zero.
TM_HD void tiled_dims(uint32_t k, uint32_t N, uint32_t T, uint32_t* kp, uint32_t* Np) {
  *kp = cdiv(k, T) * T;
  *Np = cdiv(N, T) * T;
}

}  // namespace tmk
