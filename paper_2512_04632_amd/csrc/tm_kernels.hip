// gfx950 (MI355X, CDNA4) kernels of the Turbo-Muon orthogonalizer.
//
// Every phase of Algorithm 2 is one launch over the tiles of all matrices of
// a call (see tm_internal.h for the descriptors):
//   k_transpose_in   tall inputs: W1 = X^T, so the Gram is always min(m, n) square
//   k_frob_partial   Algorithm 1, first line: deterministic partial sums of squares
//   k_gram           A = Y Y^T on the matrix cores, upper tiles only, mirrored
//                    store; at iteration 1 the epilogue emits the AOL row sums
//                    sum_j |A_ij| from the fp32 accumulators (eq. (aol))
//   k_aol_vector     s_i = 1/sqrt(row sum) (Algorithm 2, second line), or the
//                    uniform 1/||X||_F of Algorithm 1
//   k_poly           B = b A + c A A, upper tiles, mirrored store; at iteration 1
//                    the operands are rescaled on load (A1 = diag(s) A0 diag(s))
//   k_update         Y' = a Y + B Y with the axpy fused in the epilogue; at
//                    iteration 1 the rescaled X1 = diag(s) X0 is folded in
//   k_apply_scale    iters = 0: X1 = diag(s) X0 in place
//
// These are the fp32 path's kernels; a bf16 call runs only the elementwise
// ones from here (Frobenius partials, AOL vector, iters = 0 rescale) and its
// matrix-core phases in tm_fast.hip.
//
// Matrix-core tiles: 256 threads = 4 wave64s in a 2 x 2 grid; each wave owns
// (BM/2) x (BN/2) of the output as 32 x 32 MFMA blocks (v_mfma_f32_32x32x2_f32).
// K advances by 128 bytes per step through double-buffered LDS; global loads
// of step k+1 are issued before the MFMAs of step k.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "tm_internal.h"

namespace tmk {

typedef float f32x16_t __attribute__((ext_vector_type(16)));

// ---------------------------------------------------------------- elements
template <typename T> struct Elem;
template <> struct Elem<uint16_t> {            // bf16 stored as its bit pattern
  static constexpr int VE = 8;                 // elements per 16-byte vector
  __device__ static float to_f(uint16_t v) { return __uint_as_float(uint32_t(v) << 16); }
  __device__ static uint16_t from_f(float f) {  // v_cvt_pk_bf16_f32: nearest even
    __bf16 h = static_cast<__bf16>(f);
    return __builtin_bit_cast(uint16_t, h);
  }
};
template <> struct Elem<float> {
  static constexpr int VE = 4;
  __device__ static float to_f(float v) { return v; }
  __device__ static float from_f(float f) { return f; }
};

constexpr int kRowBytes = 128;                 // K bytes per LDS row and per K step
constexpr int kLdsStride = kRowBytes + 16;     // padded LDS row stride (bytes)

template <int BM_, int BN_>
struct Cfg {
  static constexpr int BM = BM_, BN = BN_;
  static constexpr int TM = BM / 2, TN = BN / 2;       // wave tile
  static constexpr int FM = TM / 32, FN = TN / 32;     // 32x32 MFMA blocks per wave
  static constexpr int STAGE = (BM + BN) * kLdsStride;
  static constexpr int LDS = 2 * STAGE;
};
using Cfg256 = Cfg<256, 256>;
using Cfg128 = Cfg<128, 128>;
using Cfg64 = Cfg<64, 64>;

// ---------------------------------------------------------------- launch mapping
// Workgroups are dealt to the 8 XCDs round robin; renumber them so that each
// XCD (with its own L2) runs a contiguous range of logical tiles.
__device__ inline int xcd_remap(int p, int total) {
  const int q = total >> 3, r = total & 7;
  const int x = p & 7, j = p >> 3;
  return x * q + min(x, r) + j;
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

template <typename T>
__device__ inline char* ws_of(const Phase& P, const Entry& E, int mat) {
  const WsLayout L = ws_layout(E.kp, E.Np, sizeof(T));
  return P.ws + (uint64_t(E.ws256) << 8) + uint64_t(mat) * L.total;
}

template <typename T>
__device__ inline T* user_of(const Phase& P, const Entry& E, int mat) {
  char* x = (E.flags & kPtrTab) ? P.xp[E.xbase + mat] : E.x + uint64_t(mat) * E.k * E.N * sizeof(T);
  return reinterpret_cast<T*>(x);
}

// Wide-view Y buffer of a slot (ld = N), see tm_internal.h.
template <typename T>
__device__ inline T* slot_ptr(const Phase& P, const Entry& E, int mat, int slot) {
  const bool tall = (E.flags & kTall) != 0u;
  if (!tall && (slot == kSlotFirst || slot == kSlotFinal)) return user_of<T>(P, E, mat);
  if (tall && slot == kSlotFinal) return user_of<T>(P, E, mat);
  const WsLayout L = ws_layout(E.kp, E.Np, sizeof(T));
  char* w = ws_of<T>(P, E, mat);
  const bool w1 = tall ? (slot == kSlotFirst || slot == kSlotAlt2) : (slot == kSlotAlt1);
  return reinterpret_cast<T*>(w + (w1 ? L.w1 : L.w2));
}

__device__ inline bool aligned16(const void* p) {
  return (reinterpret_cast<uintptr_t>(p) & 15u) == 0u;
}

// ---------------------------------------------------------------- tile loaders
// K-contiguous operand: R rows of a row-major source, K along the row.
// Thread t handles the 16-byte LDS chunk (t % 8) of rows t/8 + 32 i.  TS is
// the source element type and TD the LDS (MFMA operand) type: an fp32 source
// feeding bf16 MFMAs is scaled and rounded once on its way to LDS.
template <typename TS, typename TD, int R>
struct KLoad {
  static constexpr int VE = Elem<TD>::VE;                  // elements per LDS chunk
  static constexpr int NV = R * 8 / 256;
  static constexpr int NL = int(sizeof(TS) / sizeof(TD));  // 16-byte source loads per chunk
  uint4 raw[NV][NL];

  __device__ void load(const TS* __restrict__ src, int64_t ld, int rows, int K, int k0,
                       bool vec) {
    const int ch = threadIdx.x & 7;
    const int kk = k0 + ch * VE;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int r = (threadIdx.x >> 3) + 32 * i;
      const TS* p = src + int64_t(r) * ld + kk;
      if (vec && r < rows && kk + VE <= K) {
#pragma unroll
        for (int q = 0; q < NL; ++q) raw[i][q] = reinterpret_cast<const uint4*>(p)[q];
      } else {
        TS tmp[VE];
#pragma unroll
        for (int e = 0; e < VE; ++e) tmp[e] = (r < rows && kk + e < K) ? p[e] : TS(0);
#pragma unroll
        for (int q = 0; q < NL; ++q) raw[i][q] = reinterpret_cast<const uint4*>(tmp)[q];
      }
    }
  }

  // Unscaled store (TS == TD).
  __device__ void store(char* lds) const {
    static_assert(sizeof(TS) == sizeof(TD), "conversion needs store_scaled");
    const int ch = threadIdx.x & 7;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int r = (threadIdx.x >> 3) + 32 * i;
      *reinterpret_cast<uint4*>(lds + r * kLdsStride + ch * 16) = raw[i][0];
    }
  }

  // Store element (r, kk + e) times srow[r] * scol[kk + e], rounded once to TD.
  __device__ void store_scaled(char* lds, const float* __restrict__ srow,
                               const float* __restrict__ scol, int rows, int K, int k0) const {
    const int ch = threadIdx.x & 7;
    const int kk = k0 + ch * VE;
    float sc[VE];
#pragma unroll
    for (int e = 0; e < VE; ++e) sc[e] = (kk + e < K) ? scol[kk + e] : 0.f;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int r = (threadIdx.x >> 3) + 32 * i;
      const float sr = r < rows ? srow[r] : 0.f;
      TS in[VE];
#pragma unroll
      for (int q = 0; q < NL; ++q) reinterpret_cast<uint4*>(in)[q] = raw[i][q];
      TD out[VE];
#pragma unroll
      for (int e = 0; e < VE; ++e) out[e] = Elem<TD>::from_f(Elem<TS>::to_f(in[e]) * (sr * sc[e]));
      *reinterpret_cast<uint4*>(lds + r * kLdsStride + ch * 16) = *reinterpret_cast<const uint4*>(out);
    }
  }
};

// MN-contiguous operand (the Y factor of the update): the source is row-major
// with K along its rows (index j) and the C output columns along a row (index
// l).  Each thread loads a VE x VE block (VE rows of one 16-byte column chunk),
// transposes it in registers and writes VE K-contiguous 16-byte LDS rows, so
// the MFMA reads are the same as for K-contiguous operands.
// Block q: kb = q % 8 (K chunk), cb = q / 8 (column chunk): the 8 lanes of a
// quarter-wave read 8 rows of the same 128-byte column span.
template <typename T, int C>
struct TLoad {
  static constexpr int VE = Elem<T>::VE;
  static constexpr int NCB = C / VE;
  static constexpr int NBLK = 8 * NCB;
  static constexpr int NB = (NBLK + 255) / 256;
  uint4 v[NB][VE];

  __device__ void load(const T* __restrict__ src, int64_t ld, int ncols, int K, int k0,
                       bool vec) {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const int q = threadIdx.x + 256 * nb;
      if (NBLK % 256 != 0 && q >= NBLK) break;
      const int kb = q & 7, cb = q >> 3;
      const int l = cb * VE;
#pragma unroll
      for (int r = 0; r < VE; ++r) {
        const int j = k0 + kb * VE + r;
        const T* p = src + int64_t(j) * ld + l;
        if (vec && j < K && l + VE <= ncols) {
          v[nb][r] = *reinterpret_cast<const uint4*>(p);
        } else {
          T tmp[VE];
#pragma unroll
          for (int e = 0; e < VE; ++e) tmp[e] = (j < K && l + e < ncols) ? p[e] : T(0);
          v[nb][r] = __builtin_bit_cast(uint4, tmp);
        }
      }
    }
  }

  __device__ void store(char* lds) const {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const int q = threadIdx.x + 256 * nb;
      if (NBLK % 256 != 0 && q >= NBLK) break;
      const int kb = q & 7, cb = q >> 3;
      T in[VE][VE];
#pragma unroll
      for (int r = 0; r < VE; ++r) *reinterpret_cast<uint4*>(in[r]) = v[nb][r];
#pragma unroll
      for (int c = 0; c < VE; ++c) {
        T out[VE];
#pragma unroll
        for (int r = 0; r < VE; ++r) out[r] = in[r][c];
        *reinterpret_cast<uint4*>(lds + (cb * VE + c) * kLdsStride + kb * 16) =
            *reinterpret_cast<const uint4*>(out);
      }
    }
  }
};

// ---------------------------------------------------------------- MFMA stage
template <typename T, class C>
__device__ inline void mma_stage(f32x16_t (&acc)[C::FM][C::FN], const char* ldsA,
                                 const char* ldsB, int wm, int wn) {
  static_assert(sizeof(T) == 4, "bf16 products run in tm_fast.hip");
  const int lane = threadIdx.x & 63;
  const int lr = lane & 31, lh = lane >> 5;
#pragma unroll
  for (int kk = 0; kk < kRowBytes / 32; ++kk) {
    uint4 a[C::FM], b[C::FN];
#pragma unroll
    for (int fm = 0; fm < C::FM; ++fm)
      a[fm] = *reinterpret_cast<const uint4*>(ldsA + (wm * C::TM + fm * 32 + lr) * kLdsStride +
                                              kk * 32 + lh * 16);
#pragma unroll
    for (int fn = 0; fn < C::FN; ++fn)
      b[fn] = *reinterpret_cast<const uint4*>(ldsB + (wn * C::TN + fn * 32 + lr) * kLdsStride +
                                              kk * 32 + lh * 16);
#pragma unroll
    for (int fm = 0; fm < C::FM; ++fm)
#pragma unroll
      for (int fn = 0; fn < C::FN; ++fn) {
        // Lanes 0-31 hold k = 0..3 and lanes 32-63 k = 4..7 of the 8-wide K
        // chunk; both operands share the assignment, so the 4 rank-2 MFMAs
        // sum the chunk exactly once.
        const float* af = reinterpret_cast<const float*>(&a[fm]);
        const float* bf = reinterpret_cast<const float*>(&b[fn]);
#pragma unroll
        for (int q = 0; q < 4; ++q)
          acc[fm][fn] = __builtin_amdgcn_mfma_f32_32x32x2f32(af[q], bf[q], acc[fm][fn], 0, 0, 0);
      }
  }
}

// C tile (BM x BN) += A (BM x K) * B^T where A's rows come from a K-contiguous
// source and B's from a K-contiguous source (TRANSB = false) or an
// MN-contiguous one (TRANSB = true).  SCALE (K-contiguous B only) rescales both
// operands on load: element (r, l) of A by sA[r] sK[l], of B by sB[r] sK[l];
// the sources then have element type TA and are rounded once to T.
template <typename T, class C, bool TRANSB, bool SCALE, typename TA = T>
__device__ inline void gemm_tile(f32x16_t (&acc)[C::FM][C::FN], char* smem,
                                 const TA* __restrict__ Asrc, int64_t lda, int arows, bool avec,
                                 const void* Bsrc_, int64_t ldb, int bext, bool bvec,
                                 int K, const float* sA, const float* sB, const float* sK) {
  static_assert(!(SCALE && TRANSB), "scaling is for the symmetric products");
  using TB = typename std::conditional<TRANSB, T, TA>::type;
  const TB* __restrict__ Bsrc = static_cast<const TB*>(Bsrc_);
  constexpr int BK = kRowBytes / int(sizeof(T));
  const int wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1;
#pragma unroll
  for (int fm = 0; fm < C::FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < C::FN; ++fn)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[fm][fn][v] = 0.f;

  KLoad<TA, T, C::BM> la;
  typename std::conditional<TRANSB, TLoad<T, C::BN>, KLoad<TA, T, C::BN>>::type lb;
  const int nk = int(cdiv(uint32_t(K), uint32_t(BK)));

  auto stage_store = [&](char* dst, int k0) {
    if constexpr (SCALE) {
      la.store_scaled(dst, sA, sK, arows, K, k0);
      lb.store_scaled(dst + C::BM * kLdsStride, sB, sK, bext, K, k0);
    } else {
      la.store(dst);
      lb.store(dst + C::BM * kLdsStride);
    }
  };

  la.load(Asrc, lda, arows, K, 0, avec);
  lb.load(Bsrc, ldb, bext, K, 0, bvec);
  stage_store(smem, 0);
  __syncthreads();

  for (int kt = 0; kt < nk; ++kt) {
    char* cur = smem + (kt & 1) * C::STAGE;
    char* nxt = smem + ((kt + 1) & 1) * C::STAGE;
    const bool more = kt + 1 < nk;
    if (more) {
      la.load(Asrc, lda, arows, K, (kt + 1) * BK, avec);
      lb.load(Bsrc, ldb, bext, K, (kt + 1) * BK, bvec);
    }
    mma_stage<T, C>(acc, cur, cur + C::BM * kLdsStride, wm, wn);
    if (more) stage_store(nxt, (kt + 1) * BK);
    __syncthreads();
  }
}

// Position of accumulator element v of block (fm, fn) inside the C tile.
template <class C>
__device__ inline int acc_row(int wm, int fm, int v) {
  const int lane = threadIdx.x & 63;
  return wm * C::TM + fm * 32 + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
}
template <class C>
__device__ inline int acc_col(int wn, int fn) {
  return wn * C::TN + fn * 32 + (threadIdx.x & 31);
}

// Upper-triangle tile t of an nb x nb tile grid, row-major over the triangle.
__device__ inline void tri_tile(int t, int nb, int& I, int& J) {
  I = 0;
  while (t >= nb - I) {
    t -= nb - I;
    ++I;
  }
  J = I + t;
}

// Store a symmetric-product tile (rows I, cols J of a k x k matrix, ld) and,
// off the diagonal, its transpose at (J, I).  f(i, j, x) gives the value stored
// at (i, j); g(i, j, x) the value stored at the mirrored (j, i).
template <typename T, class C, class F, class G>
__device__ inline void store_sym(const f32x16_t (&acc)[C::FM][C::FN], T* __restrict__ D, int64_t ld,
                                 int k, int I, int J, F f, G g) {
  const int wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int i0 = I * C::BM, j0 = J * C::BN;
#pragma unroll
  for (int fm = 0; fm < C::FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < C::FN; ++fn) {
      const int j = j0 + acc_col<C>(wn, fn);
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int i = i0 + acc_row<C>(wm, fm, v);
        if (i < k && j < k) D[int64_t(i) * ld + j] = Elem<T>::from_f(f(i, j, acc[fm][fn][v]));
      }
      if (I != J && j < k) {
#pragma unroll
        for (int v4 = 0; v4 < 4; ++v4) {
          const int ib = i0 + acc_row<C>(wm, fm, 4 * v4);   // 4 consecutive rows
          T out[4];
#pragma unroll
          for (int u = 0; u < 4; ++u) out[u] = Elem<T>::from_f(g(ib + u, j, acc[fm][fn][4 * v4 + u]));
          T* p = D + int64_t(j) * ld + ib;
          if (ib + 3 < k) {
            *reinterpret_cast<uint4*>(p) = *reinterpret_cast<uint4*>(out);
          } else {
            for (int u = 0; u < 4; ++u)
              if (ib + u < k) p[u] = out[u];
          }
        }
      }
    }
}

// ---------------------------------------------------------------- kernels
// A = Y Y^T (upper tiles).  With kRowSum: part[Jb][i] = sum_{j in block Jb} |A_ij|
// (A_ij^2 with kRowSq) for every row i < k and column block Jb, each written
// exactly once.
template <typename T, class C>
__global__ __launch_bounds__(256) void k_gram(const Phase P) {
  __shared__ __attribute__((aligned(16))) char smem[C::LDS];
  static_assert(C::BM == C::BN, "square tiles");
  const Loc L = locate(P, xcd_remap(blockIdx.x, P.total));
  const Entry& E = P.e[L.ent];
  const int k = int(E.k), N = int(E.N);
  int I, J;
  tri_tile(L.tile, int(cdiv(E.k, C::BM)), I, J);
  const T* Y = slot_ptr<T>(P, E, L.mat, P.src);
  const bool vec = (N % Elem<T>::VE) == 0 && aligned16(Y);
  f32x16_t acc[C::FM][C::FN];
  gemm_tile<T, C, false, false>(acc, smem, Y + int64_t(I) * C::BM * N, N, min(C::BM, k - I * C::BM),
                                vec, Y + int64_t(J) * C::BN * N, N, min(C::BN, k - J * C::BN), vec,
                                N, nullptr, nullptr, nullptr);
  char* w = ws_of<T>(P, E, L.mat);
  const WsLayout WL = ws_layout(E.kp, E.Np, sizeof(T));
  auto ident = [](int, int, float x) { return x; };
  if (P.flags & kA32)   // first iteration: keep A0 unrounded until it is rescaled
    store_sym<float, C>(acc, reinterpret_cast<float*>(w + WL.a32), E.kp, k, I, J, ident, ident);
  else
    store_sym<T, C>(acc, reinterpret_cast<T*>(w + WL.a), E.kp, k, I, J, ident, ident);

  if (P.flags & kRowSum) {
    float* part = reinterpret_cast<float*>(w + WL.part);
    const bool sq = (P.flags & kRowSq) != 0u;   // Schatten-4: sums of A0_ij^2
    auto mag = [sq](float x) { return sq ? x * x : fabsf(x); };
    float* rs = reinterpret_cast<float*>(smem);            // [2][BM] row sums per wn
    float* cs = rs + 2 * C::BM;                            // [2][BN] column sums per wm
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int wm = wave >> 1, wn = wave & 1;
    // smem was last read by the final MFMA stage; gemm_tile ends with a barrier.
#pragma unroll
    for (int fm = 0; fm < C::FM; ++fm)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        float x = 0.f;
#pragma unroll
        for (int fn = 0; fn < C::FN; ++fn) x += mag(acc[fm][fn][v]);
#pragma unroll
        for (int off = 16; off >= 1; off >>= 1) x += __shfl_xor(x, off, 64);
        if ((lane & 31) == 0) rs[wn * C::BM + acc_row<C>(wm, fm, v)] = x;
      }
#pragma unroll
    for (int fn = 0; fn < C::FN; ++fn) {
      float x = 0.f;
#pragma unroll
      for (int fm = 0; fm < C::FM; ++fm)
#pragma unroll
        for (int v = 0; v < 16; ++v) x += mag(acc[fm][fn][v]);
      x += __shfl_xor(x, 32, 64);
      if (lane < 32) cs[wm * C::BN + acc_col<C>(wn, fn)] = x;
    }
    __syncthreads();
    for (int r = threadIdx.x; r < C::BM; r += 256) {
      const int i = I * C::BM + r;
      if (i < k) part[int64_t(J) * E.kp + i] = rs[r] + rs[C::BM + r];
      const int j = J * C::BN + r;
      if (I != J && j < k) part[int64_t(I) * E.kp + j] = cs[r] + cs[C::BN + r];
    }
  }
}

// B = b A1 + c A1 A1 with A1 = A, or under kScale A1 = diag(s) A0 diag(s)
// from the fp32 A0 of the first Gram, rounded once on its way to the matrix
// cores.  Under kScale the stored matrix is B1 diag(s) (tile (i, j) times s_j,
// the mirror times s_i) so that the update applies X1 = diag(s) X0 for free.
template <typename T, class C, bool SCALE>
__global__ __launch_bounds__(256) void k_poly(const Phase P) {
  __shared__ __attribute__((aligned(16))) char smem[C::LDS];
  const Loc L = locate(P, xcd_remap(blockIdx.x, P.total));
  const Entry& E = P.e[L.ent];
  const int k = int(E.k);
  int I, J;
  tri_tile(L.tile, int(cdiv(E.k, C::BM)), I, J);
  char* w = ws_of<T>(P, E, L.mat);
  const WsLayout WL = ws_layout(E.kp, E.Np, sizeof(T));
  T* B = reinterpret_cast<T*>(w + WL.b);
  const float* s = reinterpret_cast<const float*>(w + WL.s);
  const int64_t ld = E.kp;
  const float b = P.b, c = P.c;
  f32x16_t acc[C::FM][C::FN];
  if constexpr (SCALE) {
    const float* A0 = reinterpret_cast<const float*>(w + WL.a32);
    gemm_tile<T, C, false, true, float>(acc, smem, A0 + int64_t(I) * C::BM * ld, ld,
                                        min(C::BM, k - I * C::BM), true,
                                        A0 + int64_t(J) * C::BN * ld, ld, min(C::BN, k - J * C::BN),
                                        true, k, s + I * C::BM, s + J * C::BN, s);
    auto f = [=](int i, int j, float x) {
      const float a1 = A0[int64_t(i) * ld + j] * (s[i] * s[j]);
      return (b * a1 + c * x) * s[j];
    };
    auto g = [=](int i, int j, float x) {
      const float a1 = A0[int64_t(i) * ld + j] * (s[i] * s[j]);
      return (b * a1 + c * x) * s[i];
    };
    store_sym<T, C>(acc, B, ld, k, I, J, f, g);
  } else {
    const T* A = reinterpret_cast<const T*>(w + WL.a);
    gemm_tile<T, C, false, false>(acc, smem, A + int64_t(I) * C::BM * ld, ld,
                                  min(C::BM, k - I * C::BM), true, A + int64_t(J) * C::BN * ld, ld,
                                  min(C::BN, k - J * C::BN), true, k, nullptr, nullptr, nullptr);
    auto f = [=](int i, int j, float x) { return b * Elem<T>::to_f(A[int64_t(i) * ld + j]) + c * x; };
    store_sym<T, C>(acc, B, ld, k, I, J, f, f);
  }
}

// Y' = a Y + B Y (Y = slot src, Y' = slot dst).  Under kScale, Y is X0 and
// B holds B1 diag(s): Y' = a diag(s) X0 + B1 diag(s) X0.
template <typename T, class C, bool SCALE>
__global__ __launch_bounds__(256) void k_update(const Phase P) {
  __shared__ __attribute__((aligned(16))) char smem[C::LDS];
  const Loc L = locate(P, xcd_remap(blockIdx.x, P.total));
  const Entry& E = P.e[L.ent];
  const int k = int(E.k), N = int(E.N);
  // Tiles ordered in groups of 4 block rows so concurrent tiles share B rows.
  const int nI = int(cdiv(E.k, C::BM)), nL = int(cdiv(E.N, C::BN));
  constexpr int GM = 4;
  const int grp = L.tile / (GM * nL);
  const int first = grp * GM;
  const int gsz = min(nI - first, GM);
  const int rem = L.tile - grp * GM * nL;
  const int I = first + rem % gsz;
  const int Lb = rem / gsz;

  char* w = ws_of<T>(P, E, L.mat);
  const WsLayout WL = ws_layout(E.kp, E.Np, sizeof(T));
  const T* B = reinterpret_cast<const T*>(w + WL.b);
  const float* s = reinterpret_cast<const float*>(w + WL.s);
  const T* Y = slot_ptr<T>(P, E, L.mat, P.src);
  T* D = slot_ptr<T>(P, E, L.mat, P.dst);
  const bool vec = (N % Elem<T>::VE) == 0 && aligned16(Y);
  const int64_t ldb = E.kp;
  f32x16_t acc[C::FM][C::FN];
  gemm_tile<T, C, true, false>(acc, smem, B + int64_t(I) * C::BM * ldb, ldb,
                               min(C::BM, k - I * C::BM), true, Y + int64_t(Lb) * C::BN, N,
                               N - Lb * C::BN, vec, k, nullptr, nullptr, nullptr);
  const float a = P.a;
  const bool trans = (E.flags & kTall) != 0u && P.dst == kSlotFinal;
  const int wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1;
#pragma unroll
  for (int fm = 0; fm < C::FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < C::FN; ++fn) {
      const int l = Lb * C::BN + acc_col<C>(wn, fn);
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int i = I * C::BM + acc_row<C>(wm, fm, v);
        if (i < k && l < N) {
          float y = Elem<T>::to_f(Y[int64_t(i) * N + l]);
          if constexpr (SCALE) y *= s[i];
          const T o = Elem<T>::from_f(a * y + acc[fm][fn][v]);
          if (trans) D[int64_t(l) * k + i] = o;
          else D[int64_t(i) * N + l] = o;
        }
      }
    }
}

// W1 = X^T for tall inputs (X is N x k row-major): 64 x 64 tiles through LDS.
template <typename T>
__global__ __launch_bounds__(256) void k_transpose_in(const Phase P) {
  __shared__ T tile[kTransposeTile][kTransposeTile + 1];
  const Loc L = locate(P, blockIdx.x);
  const Entry& E = P.e[L.ent];
  const int k = int(E.k), N = int(E.N);
  const int nI = int(cdiv(E.k, kTransposeTile));
  const int ti = L.tile % nI, tl = L.tile / nI;
  const T* X = user_of<T>(P, E, L.mat);
  T* W = slot_ptr<T>(P, E, L.mat, kSlotFirst);
  const int c = threadIdx.x & 63, r0 = threadIdx.x >> 6;
  for (int r = r0; r < kTransposeTile; r += 4) {
    const int l = tl * kTransposeTile + r, i = ti * kTransposeTile + c;
    tile[r][c] = (l < N && i < k) ? X[int64_t(l) * k + i] : T(0);
  }
  __syncthreads();
  for (int r = r0; r < kTransposeTile; r += 4) {
    const int i = ti * kTransposeTile + r, l = tl * kTransposeTile + c;
    if (i < k && l < N) W[int64_t(i) * N + l] = tile[c][r];
  }
}

__device__ inline float block_sum_256(float x, float* red) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) x += __shfl_xor(x, off, 64);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = x;
  __syncthreads();
  return red[0] + red[1] + red[2] + red[3];
}

// Partial sums of squares of each user matrix (any orientation: ||X||_F = ||X^T||_F).
// With kFromPart: partial sums of the first Gram's row partials part[b][i]
// (i < k, P.aux columns per block b), i.e. of ||A0||_F^2 for Schatten-4.
template <typename T>
__global__ __launch_bounds__(256) void k_frob_partial(const Phase P) {
  __shared__ float red[4];
  const Loc L = locate(P, blockIdx.x);
  const Entry& E = P.e[L.ent];
  const bool from_part = (P.flags & kFromPart) != 0u;
  // partials past column k are zero: their count follows k, not the padding,
  // so the chunks (and the sum) do not depend on the tile size
  const int64_t nb = int64_t(cdiv(E.k, uint32_t(max(P.aux, 1))));
  const int64_t total = from_part ? nb * E.k : int64_t(E.k) * E.N;
  const int64_t chunk = (total + kFrobBlocks - 1) / kFrobBlocks;
  const int64_t lo = chunk * L.tile, hi = min(total, lo + chunk);
  const T* X = user_of<T>(P, E, L.mat);
  const float* part = reinterpret_cast<const float*>(ws_of<T>(P, E, L.mat) +
                                                     ws_layout(E.kp, E.Np, sizeof(T)).part);
  float x = 0.f;
  if (from_part) {
    for (int64_t q = lo + threadIdx.x; q < hi; q += 256) {
      const int64_t b = q / E.k, i = q - b * E.k;
      x += part[b * E.kp + i];
    }
  } else {
    for (int64_t i = lo + threadIdx.x; i < hi; i += 256) {
      const float v = Elem<T>::to_f(X[i]);
      x += v * v;
    }
  }
  x = block_sum_256(x, red);
  if (threadIdx.x == 0) {
    float* fp = reinterpret_cast<float*>(ws_of<T>(P, E, L.mat) + ws_layout(E.kp, E.Np, sizeof(T)).fpart);
    fp[L.tile] = x;
  }
}

// s_i = 1/sqrt(sum_Jb part[Jb][i]) (0 for a zero sum), or with kFrob the
// uniform 1/sqrt(sum of the Frobenius partials), with kFrob | kS4 the uniform
// (sum of the partials)^(-1/4).  Fixed summation order.
template <typename T>
__global__ __launch_bounds__(256) void k_aol_vector(const Phase P) {
  const Loc L = locate(P, blockIdx.x);
  const Entry& E = P.e[L.ent];
  const int k = int(E.k), kp = int(E.kp);
  const int i = L.tile * 256 + int(threadIdx.x);
  if (i >= kp) return;
  char* w = ws_of<T>(P, E, L.mat);
  const WsLayout WL = ws_layout(E.kp, E.Np, sizeof(T));
  float* s = reinterpret_cast<float*>(w + WL.s);
  float r = 0.f;
  if (i < k) {
    if (P.flags & kFrob) {
      const float* fp = reinterpret_cast<const float*>(w + WL.fpart);
#pragma unroll 8
      for (int b = 0; b < kFrobBlocks; ++b) r += fp[b];
    } else {
      // unrolled so that the loads are in flight together; the sum keeps its order
      const float* part = reinterpret_cast<const float*>(w + WL.part);
      const int nb = int(cdiv(E.kp, uint32_t(P.aux)));
#pragma unroll 8
      for (int b = 0; b < nb; ++b) r += part[int64_t(b) * kp + i];
    }
  }
  const float q = (P.flags & kS4) ? sqrtf(r) : r;         // Schatten-4: ||A0||_F
  s[i] = r >= 1.17549435e-38f ? 1.0f / sqrtf(q) : 0.f;   // padding rows: 0
}

// X1 = diag(s) X0 in place on the user matrix (rows of the wide view).
template <typename T>
__global__ __launch_bounds__(256) void k_apply_scale(const Phase P) {
  const Loc L = locate(P, blockIdx.x);
  const Entry& E = P.e[L.ent];
  const int64_t total = int64_t(E.k) * E.N;
  T* X = user_of<T>(P, E, L.mat);
  const float* s = reinterpret_cast<const float*>(ws_of<T>(P, E, L.mat) +
                                                  ws_layout(E.kp, E.Np, sizeof(T)).s);
  const bool tall = (E.flags & kTall) != 0u;
  const int64_t lo = int64_t(L.tile) * kElemBlock;
  for (int64_t idx = lo + threadIdx.x; idx < min(total, lo + kElemBlock); idx += 256) {
    const int64_t i = tall ? idx % E.k : idx / E.N;
    X[idx] = Elem<T>::from_f(Elem<T>::to_f(X[idx]) * s[i]);
  }
}

// Final slot <- slot src, for a single iteration (whose update cannot write the
// buffer it reads): wide matrices copy, tall ones store transposed.
template <typename T>
__global__ __launch_bounds__(256) void k_copy_out(const Phase P) {
  const Loc L = locate(P, blockIdx.x);
  const Entry& E = P.e[L.ent];
  const int64_t total = int64_t(E.k) * E.N;
  const T* S = slot_ptr<T>(P, E, L.mat, P.src);
  T* D = user_of<T>(P, E, L.mat);
  const bool tall = (E.flags & kTall) != 0u;
  const int64_t lo = int64_t(L.tile) * kElemBlock;
  for (int64_t idx = lo + threadIdx.x; idx < min(total, lo + kElemBlock); idx += 256) {
    const int64_t i = idx / E.N, l = idx - i * E.N;
    D[tall ? l * E.k + i : idx] = S[idx];
  }
}

// ---------------------------------------------------------------- host launchers
#define TM_LAUNCH(kern) \
  do { hipLaunchKernelGGL(kern, dim3(P.total), dim3(256), 0, st, P); return hipGetLastError(); } while (0)

template <typename T>
static hipError_t gram_t(int cfg, const Phase& P, hipStream_t st) {
  if (cfg == 0) TM_LAUNCH((k_gram<T, Cfg256>));
  if (cfg == 1) TM_LAUNCH((k_gram<T, Cfg128>));
  TM_LAUNCH((k_gram<T, Cfg64>));
}
template <typename T, bool S>
static hipError_t poly_t(int cfg, const Phase& P, hipStream_t st) {
  if (cfg == 0) TM_LAUNCH((k_poly<T, Cfg256, S>));
  if (cfg == 1) TM_LAUNCH((k_poly<T, Cfg128, S>));
  TM_LAUNCH((k_poly<T, Cfg64, S>));
}
template <typename T, bool S>
static hipError_t update_t(int cfg, const Phase& P, hipStream_t st) {
  if (cfg == 0) TM_LAUNCH((k_update<T, Cfg256, S>));
  if (cfg == 1) TM_LAUNCH((k_update<T, Cfg128, S>));
  TM_LAUNCH((k_update<T, Cfg64, S>));
}

#ifndef TM_ELEM_BYTES
#define TM_ELEM_BYTES 4
#endif

#if TM_ELEM_BYTES == 2
// bf16: the elementwise phases; the matrix-core phases live in tm_fast.hip.
hipError_t launch_elementwise_bf16(int kind, const Phase& P, hipStream_t st) {
  using T = uint16_t;
  if (P.total <= 0) return hipSuccess;
  switch (kind) {
    case kKindFrob: TM_LAUNCH(k_frob_partial<T>);
    case kKindAolVector: TM_LAUNCH(k_aol_vector<T>);
    case kKindApplyScale: TM_LAUNCH(k_apply_scale<T>);
  }
  return hipErrorInvalidValue;
}
#else
hipError_t launch_phase_f32(int kind, int cfg, const Phase& P, hipStream_t st) {
  using T = float;
  if (P.total <= 0) return hipSuccess;
  const bool scale = (P.flags & kScale) != 0u;
  switch (kind) {
    case kKindTransposeIn: TM_LAUNCH(k_transpose_in<T>);
    case kKindFrob: TM_LAUNCH(k_frob_partial<T>);
    case kKindGram: return gram_t<T>(cfg, P, st);
    case kKindAolVector: TM_LAUNCH(k_aol_vector<T>);
    case kKindPoly: return scale ? poly_t<T, true>(cfg, P, st) : poly_t<T, false>(cfg, P, st);
    case kKindUpdate: return scale ? update_t<T, true>(cfg, P, st) : update_t<T, false>(cfg, P, st);
    case kKindApplyScale: TM_LAUNCH(k_apply_scale<T>);
    case kKindCopyOut: TM_LAUNCH(k_copy_out<T>);
  }
  return hipErrorInvalidValue;
}
#endif

}  // namespace tmk
