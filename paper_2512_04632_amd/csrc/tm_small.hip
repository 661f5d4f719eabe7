// Fused Newton-Schulz for small matrices (bf16, k = min(m, n) <= 128): one
// workgroup of 4 wave64s per matrix keeps the matrix Y (k x N, the wide
// view), its Gram A and the polynomial B in LDS and runs every iteration of
// Algorithm 2 (or 1) in a single launch: pre-conditioning, then per
// iteration Gram, polynomial and update, with barriers between the phases
// instead of kernel boundaries.  For calls made only of small matrices the
// tiled path's dozen launches per call, each a few microseconds of latency
// for a handful of tiny tiles, become one.
//
// The arithmetic is that of the tiled kernels step for step, so a matrix
// comes out bit for bit as it does from them:
//   * every product is v_mfma_f32_16x16x32_bf16 over 32-wide K slices in
//     increasing order (the padded K range adds exact zeros);
//   * Gram and polynomial accumulators are symmetric bit for bit (the same
//     products in the same order), so both are formed in full and A, B are
//     written through their transposes where that gives contiguous stores;
//   * AOL row sums: 16-column blocks reduced with the butterfly pairing of
//     index bits 0..3, four of them added as (b0 + b1) + (b2 + b3) into the
//     64-column partials, the partials added in order; s = 1 / sqrt(sum);
//   * Frobenius: 32 chunks of the stored matrix, each summed by 256 threads
//     strided by 256 and reduced across lanes and waves, then added in order;
//     Schatten-4: the same chunking over the 64-column partials of A0^2;
//   * A1 = bf16(A0_ij (s_i s_j)), the first polynomial stores
//     C = bf16(B~_ij s_j) and the first update computes C X0; every other
//     stored A, B~ and Y is rounded once to bf16.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "tm_internal.h"
#include "turbomuon.h"

namespace tmk {
namespace small {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef short s16x4_t __attribute__((ext_vector_type(4)));

constexpr int NR = 256;   // threads of the reduction and product structure: 4 waves in a 2 x 2 grid
constexpr float kTiny = 1.17549435e-38f;     // FLT_MIN: smaller sums give a zero scale

__device__ inline float bf2f(uint16_t v) { return __uint_as_float(uint32_t(v) << 16); }
__device__ inline uint16_t f2bf(float f) {
  __bf16 h = static_cast<__bf16>(f);
  return __builtin_bit_cast(uint16_t, h);
}
__device__ inline uint32_t lds_addr(const void* p) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>(p));
}
__device__ inline f32x4_t mfma(uint4 a, uint4 b, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                 __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
}

// Matrix of this workgroup.
__device__ inline int locate(const SmallPhase& P, int b, int& mat) {
  int e = 0, hi = P.nent - 1;
  while (e < hi) {
    const int mid = (e + hi + 1) >> 1;
    if (b >= int(P.e[mid].tile_start)) e = mid;
    else hi = mid - 1;
  }
  mat = b - int(P.e[e].tile_start);
  return e;
}

__device__ inline uint16_t* user_of(const SmallPhase& P, const Entry& E, int mat) {
  char* x = (E.flags & kPtrTab) ? P.xp[E.xbase + mat] : E.x + uint64_t(mat) * E.k * E.N * 2u;
  return reinterpret_cast<uint16_t*>(x);
}

// q / d for q d <= 2^32 (every index here): multiply by ceil(2^32 / d).
struct Div {
  uint64_t m;
  __device__ explicit Div(uint32_t d) : m(((uint64_t(1) << 32) + d - 1u) / d) {}
  __device__ uint32_t operator()(uint32_t q) const { return uint32_t((uint64_t(q) * m) >> 32); }
};

// LDS carve-up of one matrix: Y kp x Np bf16 (row stride ry), A and B kp x kp
// bf16 (row stride ra), the 16-column row sums [kp / 16][kp], s[kp] and the
// reduction scratch [32][4].  Rows are padded by 16 bytes: a row stride of 4
// (mod 8) 16-byte chunks sends the 16 rows of a fragment read to 16
// different bank groups.
struct Geo {
  int k, N, kp, Np, ry, ra;
  char *y, *a, *b;
  float *rs, *s, *red;
};

__device__ inline Geo geometry(char* smem, int k, int N) {
  Geo G;
  G.k = k;
  G.N = N;
  G.kp = int(small_kp(uint32_t(k)));
  G.Np = int(small_np(uint32_t(N)));
  G.ry = 2 * G.Np + 16;
  G.ra = 2 * G.kp + 16;
  G.y = smem;
  G.a = G.y + G.kp * G.ry;
  G.b = G.a + G.kp * G.ra;
  G.rs = reinterpret_cast<float*>(G.b + G.kp * G.ra);
  G.s = G.rs + (G.kp / 16) * G.kp;
  G.red = G.s + G.kp;
  return G;
}

constexpr int LB = 8;   // global accesses in flight per thread

// 16-bit element t of a 16-byte piece, and a piece from four words.
__device__ inline uint16_t half_of(const uint4& v, int t) {
  const uint32_t w = (t >> 1) == 0 ? v.x : ((t >> 1) == 1 ? v.y : ((t >> 1) == 2 ? v.z : v.w));
  return uint16_t(w >> (16 * (t & 1)));
}

__device__ inline uint32_t word_of(const uint4& v, int d) {
  return d == 0 ? v.x : (d == 1 ? v.y : (d == 2 ? v.z : v.w));
}

// 8 x 8 block of 16-bit elements, rows in[r] (element c = half c % 2 of word
// c / 2): out[c] = column c, its element r from in[r].
__device__ inline void transpose8(const uint4 (&in)[8], uint4 (&out)[8]) {
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    const uint32_t sel = (c & 1) ? 0x07060302u : 0x05040100u;
    uint32_t w[4];
#pragma unroll
    for (int d = 0; d < 4; ++d)
      w[d] = __builtin_amdgcn_perm(word_of(in[2 * d + 1], c >> 1), word_of(in[2 * d], c >> 1), sel);
    out[c] = make_uint4(w[0], w[1], w[2], w[3]);
  }
}

// Y = the wide view of X (X itself, or X^T for a tall matrix), zero padded.
// Each thread issues LB loads before it stores any of them; a load outside
// the matrix reads X's first element instead and its value is replaced by
// zero, so that no load sits behind a branch (which would make each wait for
// the previous one).
template <int NT>
__device__ inline void load_y(const Geo& G, const uint16_t* X, bool tall) {
  const int tid = threadIdx.x;
  const bool vec = (reinterpret_cast<uintptr_t>(X) & 15u) == 0u;
  const uint4 z = make_uint4(0u, 0u, 0u, 0u);
  if (!tall) {
    const int cpr = G.Np / 8;                        // 16-byte chunks per padded row
    const int total = G.kp * cpr;
    const Div dv{uint32_t(cpr)};
    if (vec && (G.N % 8) == 0) {                     // whole 16-byte pieces of X rows
      for (int q0 = tid; q0 < total; q0 += LB * NT) {
        uint4 v[LB];
#pragma unroll
        for (int u = 0; u < LB; ++u) {
          const int q = q0 + u * NT;
          const int i = int(dv(uint32_t(q))), l = (q - i * cpr) * 8;
          const bool ok = q < total && i < G.k && l < G.N;
          const uint4 x = *reinterpret_cast<const uint4*>(X + (ok ? int64_t(i) * G.N + l : 0));
          const uint32_t m = ok ? ~0u : 0u;   // per word: a select of whole vectors goes through memory
          v[u] = make_uint4(x.x & m, x.y & m, x.z & m, x.w & m);
        }
#pragma unroll
        for (int u = 0; u < LB; ++u) {
          const int q = q0 + u * NT;
          const int i = int(dv(uint32_t(q))), l = (q - i * cpr) * 8;
          if (q < total) *reinterpret_cast<uint4*>(G.y + i * G.ry + l * 2) = v[u];
        }
      }
    } else {                                         // element by element
      for (int q0 = tid; q0 < total; q0 += LB * NT) {
        uint32_t v[LB][4];
#pragma unroll
        for (int u = 0; u < LB; ++u) {
          const int q = q0 + u * NT;
          const int i = int(dv(uint32_t(q))), l = (q - i * cpr) * 8;
#pragma unroll
          for (int t = 0; t < 8; ++t) {
            const bool ok = q < total && i < G.k && l + t < G.N;
            const uint32_t x = X[ok ? int64_t(i) * G.N + l + t : 0];
            const uint32_t h = ok ? x << (16 * (t & 1)) : 0u;
            v[u][t >> 1] = (t & 1) ? (v[u][t >> 1] | h) : h;
          }
        }
#pragma unroll
        for (int u = 0; u < LB; ++u) {
          const int q = q0 + u * NT;
          const int i = int(dv(uint32_t(q))), l = (q - i * cpr) * 8;
          if (q < total)
            *reinterpret_cast<uint4*>(G.y + i * G.ry + l * 2) = make_uint4(v[u][0], v[u][1], v[u][2], v[u][3]);
        }
      }
    }
  } else if (vec && (G.k % 8) == 0) {
    // 8 x 8 blocks of the padded Y: 8 rows of X (8 elements each) are loaded,
    // transposed in registers and written as 8 16-byte row pieces of Y
    const int nbi = G.kp / 8;
    const int total = (G.Np / 8) * nbi;
    const Div dv{uint32_t(nbi)};
    for (int q = tid; q < total; q += NT) {
      const int lb = int(dv(uint32_t(q))), i0 = (q - lb * nbi) * 8, l0 = lb * 8;
      uint4 v[8];
#pragma unroll
      for (int r = 0; r < 8; ++r) {
        const bool ok = l0 + r < G.N && i0 < G.k;
        const uint4 x = *reinterpret_cast<const uint4*>(X + (ok ? int64_t(l0 + r) * G.k + i0 : 0));
        const uint32_t m = ok ? ~0u : 0u;
        v[r] = make_uint4(x.x & m, x.y & m, x.z & m, x.w & m);
      }
      uint4 o[8];
      transpose8(v, o);
#pragma unroll
      for (int c = 0; c < 8; ++c) *reinterpret_cast<uint4*>(G.y + (i0 + c) * G.ry + l0 * 2) = o[c];
    }
  } else {
    const int cpr = G.Np / 8;
    for (int q = tid; q < G.kp * cpr; q += NT) {   // zero fill, then scatter the columns
      const int i = q / cpr, l = (q - i * cpr) * 8;
      *reinterpret_cast<uint4*>(G.y + i * G.ry + l * 2) = z;
    }
    __syncthreads();
    const int ck = (G.k + 7) / 8;                  // 8-element pieces of an X row
    const int total = G.N * ck;
    const Div dv{uint32_t(ck)};
    constexpr int LE = LB / 2;   // pieces in flight: 8 element loads each
    for (int q0 = tid; q0 < total; q0 += LE * NT) {
      uint4 v[LE];
#pragma unroll
      for (int u = 0; u < LE; ++u) {
        const int q = q0 + u * NT;
        const int l = int(dv(uint32_t(q))), i0 = (q - l * ck) * 8;
        uint32_t h[4];
#pragma unroll
        for (int t = 0; t < 8; ++t) {
          const bool ok = q < total && i0 + t < G.k;
          const uint32_t x = uint32_t(X[ok ? int64_t(l) * G.k + i0 + t : 0]) << (16 * (t & 1));
          h[t >> 1] = (t & 1) ? (h[t >> 1] | x) : x;
        }
        v[u] = make_uint4(h[0], h[1], h[2], h[3]);
      }
#pragma unroll
      for (int u = 0; u < LE; ++u) {
        const int q = q0 + u * NT;
        const int l = int(dv(uint32_t(q))), i0 = (q - l * ck) * 8;
        if (q < total) {
#pragma unroll
          for (int t = 0; t < 8; ++t)
            if (i0 + t < G.k) *reinterpret_cast<uint16_t*>(G.y + (i0 + t) * G.ry + l * 2) = half_of(v[u], t);
        }
      }
    }
  }
}

// X = Y (wide) or Y^T (tall), the unpadded part; LB pieces read from LDS per
// thread before they are stored.
template <int NT>
__device__ inline void store_y(const Geo& G, uint16_t* X, bool tall) {
  const int tid = threadIdx.x;
  const bool vec = (reinterpret_cast<uintptr_t>(X) & 15u) == 0u;
  if (!tall) {
    const int cpr = (G.N + 7) / 8;
    const int total = G.k * cpr;
    const Div dv{uint32_t(cpr)};
    const bool rowvec = vec && (G.N % 8) == 0;
    for (int q0 = tid; q0 < total; q0 += LB * NT) {
      uint4 v[LB];
#pragma unroll
      for (int u = 0; u < LB; ++u) {
        const int q = min(q0 + u * NT, total - 1);
        const int i = int(dv(uint32_t(q))), l = (q - i * cpr) * 8;
        v[u] = *reinterpret_cast<const uint4*>(G.y + i * G.ry + l * 2);
      }
#pragma unroll
      for (int u = 0; u < LB; ++u) {
        const int q = q0 + u * NT;
        const int i = int(dv(uint32_t(q))), l = (q - i * cpr) * 8;
        if (q >= total) continue;
        uint16_t* dst = X + int64_t(i) * G.N + l;
        if (rowvec) {
          *reinterpret_cast<uint4*>(dst) = v[u];
        } else {
#pragma unroll
          for (int t = 0; t < 8; ++t)
            if (l + t < G.N) dst[t] = half_of(v[u], t);
        }
      }
    }
  } else if (vec && (G.k % 8) == 0) {
    // 8 x 8 blocks: 8 16-byte row pieces of Y read, transposed in registers,
    // stored as 8 rows of X
    const int nbi = G.k / 8;
    const int total = ((G.N + 7) / 8) * nbi;
    const Div dv{uint32_t(nbi)};
    for (int q = tid; q < total; q += NT) {
      const int lb = int(dv(uint32_t(q))), i0 = (q - lb * nbi) * 8, l0 = lb * 8;
      uint4 v[8];
#pragma unroll
      for (int c = 0; c < 8; ++c) v[c] = *reinterpret_cast<const uint4*>(G.y + (i0 + c) * G.ry + l0 * 2);
      uint4 o[8];
      transpose8(v, o);
#pragma unroll
      for (int r = 0; r < 8; ++r)
        if (l0 + r < G.N) *reinterpret_cast<uint4*>(X + int64_t(l0 + r) * G.k + i0) = o[r];
    }
  } else {
    const int ck = (G.k + 7) / 8;
    const int total = G.N * ck;
    const Div dv{uint32_t(ck)};
    for (int q0 = tid; q0 < total; q0 += LB * NT) {
      uint4 e[LB];
#pragma unroll
      for (int u = 0; u < LB; ++u) {
        const int q = min(q0 + u * NT, total - 1);
        const int l = int(dv(uint32_t(q))), i0 = (q - l * ck) * 8;
        uint32_t h[4];
#pragma unroll
        for (int t = 0; t < 8; ++t) {
          const uint32_t x = uint32_t(*reinterpret_cast<const uint16_t*>(G.y + (i0 + t) * G.ry + l * 2))
                             << (16 * (t & 1));
          h[t >> 1] = (t & 1) ? (h[t >> 1] | x) : x;
        }
        e[u] = make_uint4(h[0], h[1], h[2], h[3]);
      }
#pragma unroll
      for (int u = 0; u < LB; ++u) {
        const int q = q0 + u * NT;
        const int l = int(dv(uint32_t(q))), i0 = (q - l * ck) * 8;
        if (q >= total) continue;
        uint16_t* dst = X + int64_t(l) * G.k + i0;
#pragma unroll
        for (int t = 0; t < 8; ++t)
          if (i0 + t < G.k) dst[t] = half_of(e[u], t);
      }
    }
  }
}

// acc = R R^T over K (16-byte rows of R at row stride rb, K a multiple of 32):
// wave (wm, wn) owns the F x F blocks of 16 x 16 at rows wm 16 F + 16 fm,
// columns wn 16 F + 16 fn.  Element v of block (fm, fn) is row 4 (L / 16) + v,
// column L % 16 of the block.  The fragments of the K slice two ahead (one
// ahead for F = 1) are read while the current one multiplies; the reads past
// the last slice land in the next row or the next region of the LDS (at most
// 128 bytes past a row's data) and are discarded.
template <int F>
__device__ inline void sym_product(f32x4_t (&acc)[F][F], const char* R, int rb, int K) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int wm = w >> 1, wn = w & 1;
  const int lr = lane & 15, g = lane >> 4;
#pragma unroll
  for (int fm = 0; fm < F; ++fm)
#pragma unroll
    for (int fn = 0; fn < F; ++fn) acc[fm][fn] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  const char* pa = R + (wm * 16 * F + lr) * rb + 16 * g;
  const char* pb = R + (wn * 16 * F + lr) * rb + 16 * g;
  auto fetch = [&](uint4 (&fa)[F], uint4 (&fb)[F], int k0) {
#pragma unroll
    for (int f = 0; f < F; ++f) {
      fa[f] = *reinterpret_cast<const uint4*>(pa + f * 16 * rb + k0 * 2);
      fb[f] = *reinterpret_cast<const uint4*>(pb + f * 16 * rb + k0 * 2);
    }
  };
  auto mult = [&](const uint4 (&fa)[F], const uint4 (&fb)[F]) {
#pragma unroll
    for (int fm = 0; fm < F; ++fm)
#pragma unroll
      for (int fn = 0; fn < F; ++fn) acc[fm][fn] = mfma(fa[fm], fb[fn], acc[fm][fn]);
  };
  uint4 a0[F], b0[F], a1[F], b1[F];
  fetch(a0, b0, 0);
  int k0 = 0;
  if constexpr (F == 1) {   // one slice ahead: a third set would halve the blocks per compute unit
    for (; k0 + 64 <= K; k0 += 64) {
      fetch(a1, b1, k0 + 32);
      mult(a0, b0);
      fetch(a0, b0, k0 + 64);
      mult(a1, b1);
    }
    if (k0 < K) mult(a0, b0);
  } else {
    uint4 a2[F], b2[F];
    fetch(a1, b1, 32);
    for (; k0 + 96 <= K; k0 += 96) {
      fetch(a2, b2, k0 + 64);
      mult(a0, b0);
      fetch(a0, b0, k0 + 96);
      mult(a1, b1);
      fetch(a1, b1, k0 + 128);
      mult(a2, b2);
    }
    if (k0 < K) mult(a0, b0);
    if (k0 + 32 < K) mult(a1, b1);
  }
}

template <int F>
__device__ inline int row0(int fm) {   // first of the lane's 4 rows of block fm
  return (threadIdx.x >> 7) * 16 * F + 16 * fm + 4 * ((threadIdx.x & 63) >> 4);
}
template <int F>
__device__ inline int col0(int fn) {
  return ((threadIdx.x >> 6) & 1) * 16 * F + 16 * fn + (threadIdx.x & 15);
}

// Value of another lane of the same row of 16 lanes (DPP).
template <int CTRL>
__device__ inline float dpp(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), CTRL, 0xF, 0xF, false));
}

// Sum over each row of 16 lanes with the butterfly that pairs lane bits 0, 1,
// 2, 3 in that order.  After the first two steps all four lanes of a quad
// hold the same value, so the lane that the half-row mirror (and then the row
// mirror) supplies holds what the lane with bit 2 (bit 3) flipped holds: the
// sums are those of the xor butterfly, bit for bit.
__device__ inline float sum16(float x) {
  x += dpp<0xB1>(x);    // quad_perm [1, 0, 3, 2]: lane ^ 1
  x += dpp<0x4E>(x);    // quad_perm [2, 3, 0, 1]: lane ^ 2
  x += dpp<0x141>(x);   // row_half_mirror: the other quad of the half-row
  x += dpp<0x140>(x);   // row_mirror: the other half of the row
  return x;
}

// 16-column row sums of |A0_ij| (or A0_ij^2) of the fp32 Gram: rs[cb][i].
template <int F>
__device__ inline void row_sums16(const Geo& G, const f32x4_t (&acc)[F][F], bool sq) {
  const int lane = threadIdx.x & 63;
  const int cb0 = ((threadIdx.x >> 6) & 1) * F;
  float x[F][F][4];
#pragma unroll
  for (int fm = 0; fm < F; ++fm)
#pragma unroll
    for (int fn = 0; fn < F; ++fn)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const float y = acc[fm][fn][v];
        x[fm][fn][v] = sum16(sq ? y * y : fabsf(y));
      }
  if ((lane & 15) == 0) {
#pragma unroll
    for (int fm = 0; fm < F; ++fm)
#pragma unroll
      for (int fn = 0; fn < F; ++fn)
#pragma unroll
        for (int v = 0; v < 4; ++v) G.rs[(cb0 + fn) * G.kp + row0<F>(fm) + v] = x[fm][fn][v];
  }
}

// 64-column partial b of row i: its four 16-column sums as (b0 + b1) + (b2 + b3)
// (blocks past the padded width are the tiled path's zero columns).
__device__ inline float part64(const Geo& G, int b, int i) {
  const int nb16 = G.kp / 16;
  float x[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) x[q] = 4 * b + q < nb16 ? G.rs[(4 * b + q) * G.kp + i] : 0.f;
  return (x[0] + x[1]) + (x[2] + x[3]);
}

// Sum of `total` terms in 32 chunks, as the tiled path's partial kernels form
// it: within a chunk thread t adds terms lo + t, lo + t + 256, ... in order
// (x += v * v with SQ, else x += v), the 64 lanes of a wave are reduced by the
// xor butterfly over offsets 32, 16, ..., 1 and the four wave sums added in
// order; the chunk sums are then added in order.  Every thread forms its sums
// of CG chunks (LB terms read before they are added), then their CG
// butterflies run side by side.  Only the first 256 threads take part.
template <bool SQ, class V>
__device__ inline float chunked_sum(const Geo& G, uint32_t total, V term) {
  constexpr int CG = 8;                          // chunks reduced side by side
  const uint32_t chunk = (total + kFrobBlocks - 1) / kFrobBlocks;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  for (int c0 = 0; c0 < kFrobBlocks; c0 += CG) {
    float x[CG];
#pragma unroll
    for (int j = 0; j < CG; ++j) {
      const uint32_t lo = chunk * uint32_t(c0 + j), hi = threadIdx.x < NR ? min(total, lo + chunk) : 0u;
      x[j] = 0.f;
      for (uint32_t q = lo + threadIdx.x; q < hi; q += LB * NR) {
        float e[LB];
#pragma unroll
        for (int u = 0; u < LB; ++u) {
          const uint32_t qq = q + uint32_t(u * NR);
          e[u] = term(qq < hi ? qq : lo);
          e[u] = qq < hi ? e[u] : 0.f;
        }
#pragma unroll
        for (int u = 0; u < LB; ++u) {
          if constexpr (SQ) x[j] += e[u] * e[u];   // +0 for the terms past the chunk
          else x[j] += e[u];
        }
      }
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1)
#pragma unroll
      for (int j = 0; j < CG; ++j) x[j] += __shfl_xor(x[j], off, 64);
    if (lane == 0 && w < 4) {
#pragma unroll
      for (int j = 0; j < CG; ++j) G.red[4 * (c0 + j) + w] = x[j];
    }
  }
  __syncthreads();
  float r = 0.f;
  for (int c = 0; c < kFrobBlocks; ++c)
    r += ((G.red[4 * c] + G.red[4 * c + 1]) + G.red[4 * c + 2]) + G.red[4 * c + 3];
  return r;
}

// One matrix per workgroup, every iteration in LDS.  F = kp / 32; NW waves:
// the first four form the 2 x 2 grid of the Gram and polynomial products and
// the reductions, all NW share the loads, the stores and the update (8 for
// F <= 2: two waves per SIMD hide each other's LDS and matrix-core
// latencies; the register footprint of F = 3, 4 allows one).
template <int F, int LDSB, int NW>
__global__ __launch_bounds__(64 * NW) void k_small_ns(const SmallPhase P) {
  constexpr int NT = 64 * NW;
  __shared__ __attribute__((aligned(16))) char smem[LDSB];
  int mat;
  const Entry& E = P.e[locate(P, int(blockIdx.x), mat)];
  uint16_t* X = user_of(P, E, mat);
  const bool tall = (E.flags & kTall) != 0u;
  const Geo G = geometry(smem, int(E.k), int(E.N));
  const int precond = P.precond;
  const bool scaled = precond != TM_PRECOND_NONE;
  const bool from_gram = precond == TM_PRECOND_AOL || precond == TM_PRECOND_SCHATTEN4;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int lr = lane & 15, g = lane >> 4;
  const bool prod = w < 4;   // a wave of the product grid

  load_y<NT>(G, X, tall);
  __syncthreads();

  // Frobenius scale (Algorithm 1), over the elements of X in its storage order
  float s_uniform = 0.f;
  if (precond == TM_PRECOND_FROBENIUS) {
    const int d = tall ? G.k : G.N;
    const Div dv{uint32_t(d)};
    const float r = chunked_sum<true>(G, uint32_t(G.k * G.N), [&](uint32_t q) {
      const int r0 = int(dv(q)), c0 = int(q) - r0 * d;   // X[r0][c0]
      const int i = tall ? c0 : r0, l = tall ? r0 : c0;
      return bf2f(*reinterpret_cast<const uint16_t*>(G.y + i * G.ry + l * 2));
    });
    s_uniform = r >= kTiny ? 1.0f / sqrtf(r) : 0.f;
  }

  f32x4_t acc[F][F];
  for (int it = 0; it < P.iters; ++it) {
    const float ca = P.coef[it][0], cb = P.coef[it][1], cc = P.coef[it][2];
    const bool first = it == 0;
    // ---- Gram A = Y Y^T (fp32 accumulators)
    if (prod) {
      sym_product<F>(acc, G.y, G.ry, G.Np);
      if (first && from_gram) row_sums16<F>(G, acc, precond == TM_PRECOND_SCHATTEN4);
    }
    if (first && scaled) {
      if (from_gram) {
        __syncthreads();
        const int nb = (G.k + 63) / 64;   // 64-column partials per row
        if (precond == TM_PRECOND_AOL) {
          for (int i = threadIdx.x; i < G.kp; i += NT) {   // eq. (aol)
            float r = 0.f;
            if (i < G.k)
              for (int b = 0; b < nb; ++b) r += part64(G, b, i);
            G.s[i] = r >= kTiny ? 1.0f / sqrtf(r) : 0.f;
          }
        } else {   // ||X||_S4 = ||A0||_F^(1/2) from the partials of A0_ij^2
          const Div dk{uint32_t(G.k)};
          const float r = chunked_sum<false>(G, uint32_t(nb * G.k), [&](uint32_t q) {
            const int b = int(dk(q)), i = int(q) - b * G.k;
            return part64(G, b, i);
          });
          const float q = sqrtf(r);
          s_uniform = r >= kTiny ? 1.0f / sqrtf(q) : 0.f;
        }
      }
      if (precond != TM_PRECOND_AOL)
        for (int i = threadIdx.x; i < G.kp; i += NT) G.s[i] = i < G.k ? s_uniform : 0.f;
      __syncthreads();
    }
    // A (bf16), written through its transpose: 4 consecutive rows of one
    // column of the lane's block become 4 consecutive elements of a row
    if (prod) {
#pragma unroll
      for (int fm = 0; fm < F; ++fm)
#pragma unroll
        for (int fn = 0; fn < F; ++fn) {
          const int i0 = row0<F>(fm), j = col0<F>(fn);
          uint16_t o[4];
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const float x = acc[fm][fn][u];
            o[u] = f2bf(first && scaled ? x * (G.s[i0 + u] * G.s[j]) : x);
          }
          *reinterpret_cast<uint2*>(G.a + j * G.ra + i0 * 2) = *reinterpret_cast<const uint2*>(o);
        }
    }
    __syncthreads();
    // ---- polynomial B~ = b A + c A A + a I (C = B~ diag(s) after a scaling)
    if (prod) {
      sym_product<F>(acc, G.a, G.ra, G.kp);
#pragma unroll
      for (int fm = 0; fm < F; ++fm)
#pragma unroll
        for (int fn = 0; fn < F; ++fn) {
          const int i0 = row0<F>(fm), j = col0<F>(fn);
          const uint2 araw = *reinterpret_cast<const uint2*>(G.a + j * G.ra + i0 * 2);
          const uint16_t* av = reinterpret_cast<const uint16_t*>(&araw);
          uint16_t o[4];
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const float x = cb * bf2f(av[u]) + cc * acc[fm][fn][u] + (i0 + u == j ? ca : 0.f);
            // stored at (j, i0 + u): B~ is symmetric; C[j][i] = B~_ij s_i
            o[u] = f2bf(first && scaled ? x * G.s[i0 + u] : x);
          }
          *reinterpret_cast<uint2*>(G.b + j * G.ra + i0 * 2) = *reinterpret_cast<const uint2*>(o);
        }
    }
    __syncthreads();
    // ---- update Y' = B~ Y (C X0 at the first iteration), in place.  Every
    // wave holds all of B~'s fragments in registers; wave w owns the
    // 16-column blocks w, w + NW, ... of Y, reads all their rows and writes
    // them back.
    {
      constexpr int FR = 2 * F;                   // 16-row blocks of kp
      uint4 bq[F][FR];                            // [K slice][row block]
#pragma unroll
      for (int s = 0; s < F; ++s)
#pragma unroll
        for (int f = 0; f < FR; ++f)
          bq[s][f] = *reinterpret_cast<const uint4*>(G.b + (16 * f + lr) * G.ra + (32 * s + 8 * g) * 2);
      // Y fragment of slice s: rows 32 s + 8 g + 4 h + lr / 4, columns
      // 16 cblk + 4 (lr % 4), transposed by the read
      auto yfrag = [&](uint4 (&yf)[F], int cblk) {
#pragma unroll
        for (int s = 0; s < F; ++s) {
          s16x4_t yv[2];
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const char* p = G.y + (32 * s + 8 * g + 4 * h + (lr >> 2)) * G.ry + (16 * cblk + 4 * (lr & 3)) * 2;
            yv[h] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                (__attribute__((address_space(3))) s16x4_t*)(lds_addr(p)));
          }
          yf[s] = __builtin_bit_cast(uint4, yv);
        }
      };
      const int nblk = G.Np / 16;
      auto mult = [&](f32x4_t (&u)[FR], const uint4 (&yf)[F]) {
#pragma unroll
        for (int f = 0; f < FR; ++f) u[f] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < F; ++s)
#pragma unroll
          for (int f = 0; f < FR; ++f) u[f] = mfma(yf[s], bq[s][f], u[f]);
      };
      // element q of u[f]: row 16 f + lr, column 16 cblk + 4 g + q
      auto put = [&](const f32x4_t (&u)[FR], int cblk) {
#pragma unroll
        for (int f = 0; f < FR; ++f) {
          uint16_t o[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) o[q] = f2bf(u[f][q]);
          *reinterpret_cast<uint2*>(G.y + (16 * f + lr) * G.ry + (16 * cblk + 4 * g) * 2) =
              *reinterpret_cast<const uint2*>(o);
        }
      };
      // Two blocks (c, c + NW) per step: the fragments of the wave's next
      // block are read while the current one multiplies, and the first
      // block's results are converted and stored while the second one's
      // products run.  Reads past the last block land in the row padding or
      // the next LDS region and are discarded.
      uint4 ya[F], yb[F];
      f32x4_t ua[FR], ub[FR];
      yfrag(ya, w);
      for (int c = w; c < nblk; c += 2 * NW) {
        yfrag(yb, c + NW);
        mult(ua, ya);
        yfrag(ya, c + 2 * NW);
        mult(ub, yb);
        put(ua, c);
        if (c + NW < nblk) put(ub, c + NW);
      }
    }
    __syncthreads();
  }
  store_y<NT>(G, X, tall);
}

template <int F>
static hipError_t launch_f(int big, const SmallPhase& P, hipStream_t st) {
  constexpr int NW = F <= 2 ? 8 : 4;
  if (big) hipLaunchKernelGGL((k_small_ns<F, 160 * 1024, NW>), dim3(P.total), dim3(64 * NW), 0, st, P);
  else hipLaunchKernelGGL((k_small_ns<F, 64 * 1024, NW>), dim3(P.total), dim3(64 * NW), 0, st, P);
  return hipGetLastError();
}

}  // namespace small

// F = kp / 32 (1..4); big: the 160 KB LDS variant (else 64 KB, two
// workgroups per compute unit).
hipError_t launch_small_bf16(int F, int big, const SmallPhase& P, hipStream_t st) {
  if (P.total <= 0) return hipSuccess;
  switch (F) {
    case 1: return small::launch_f<1>(big, P, st);
    case 2: return small::launch_f<2>(big, P, st);
    case 3: return small::launch_f<3>(big, P, st);
    case 4: return small::launch_f<4>(big, P, st);
  }
  return hipErrorInvalidValue;
}

}  // namespace tmk
