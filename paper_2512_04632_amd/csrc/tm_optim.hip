// Elementwise kernels of the optimizer step around the orthogonalization
// (Muon's step with the orthogonalization done by this library):
//   k_opt_momentum  M <- mu M + G;  U = G + mu M (Nesterov) or M, stored as bf16
//   k_opt_apply     W <- W (1 - lr wd) - lr scale O   (O: the orthogonalized U)
// One launch covers all matrices of a call; each block takes kOptBlock
// consecutive elements of one matrix (the matrix comes from a binary search
// over the blocks' starts, once per block), each thread 2 x 4 of them with
// 16-byte accesses where the matrix's pointers allow.  Both kernels are
// HBM-bound: 14 and 10 bytes per element.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "tm_internal.h"

namespace tmk {
namespace opt {

__device__ inline uint16_t f2bf(float f) {     // round to nearest even
  __bf16 h = static_cast<__bf16>(f);
  return __builtin_bit_cast(uint16_t, h);
}
__device__ inline float bf2f(uint16_t v) { return __uint_as_float(uint32_t(v) << 16); }

// Matrix of this block: the last entry whose first block is <= blockIdx.x.
__device__ inline const OptEntry& block_entry(const OptPhase& P) {
  const uint32_t b = blockIdx.x;
  int e = 0, hi = P.nent - 1;
  while (e < hi) {
    const int mid = (e + hi + 1) >> 1;
    if (b >= P.e[mid].block_start) e = mid;
    else hi = mid - 1;
  }
  return P.e[e];
}

constexpr int kHalf = kOptBlock / 2;   // elements per pass of the 256 threads (4 each)

__global__ __launch_bounds__(256) void k_opt_momentum(const OptPhase P) {
  const OptEntry& E = block_entry(P);
  const uint64_t base = uint64_t(blockIdx.x - E.block_start) * kOptBlock;
  const float mu = P.mu;
  const bool nest = P.nesterov != 0;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const uint64_t i0 = base + uint64_t(h) * kHalf + uint64_t(threadIdx.x) * 4;
    if (E.vec && i0 + 4 <= E.size) {
      const float4 g = *reinterpret_cast<const float4*>(E.g + i0);
      float4 m = *reinterpret_cast<const float4*>(E.m + i0);
      m.x = mu * m.x + g.x;
      m.y = mu * m.y + g.y;
      m.z = mu * m.z + g.z;
      m.w = mu * m.w + g.w;
      *reinterpret_cast<float4*>(E.m + i0) = m;
      uint16_t u[4];
      u[0] = f2bf(nest ? g.x + mu * m.x : m.x);
      u[1] = f2bf(nest ? g.y + mu * m.y : m.y);
      u[2] = f2bf(nest ? g.z + mu * m.z : m.z);
      u[3] = f2bf(nest ? g.w + mu * m.w : m.w);
      *reinterpret_cast<uint2*>(E.u + i0) = *reinterpret_cast<const uint2*>(u);
    } else {
      for (int j = 0; j < 4; ++j) {
        const uint64_t i = i0 + j;
        if (i >= E.size) break;
        const float g = E.g[i];
        const float m = mu * E.m[i] + g;
        E.m[i] = m;
        E.u[i] = f2bf(nest ? g + mu * m : m);
      }
    }
  }
}

__global__ __launch_bounds__(256) void k_opt_apply(const OptPhase P) {
  const OptEntry& E = block_entry(P);
  const uint64_t base = uint64_t(blockIdx.x - E.block_start) * kOptBlock;
  const float decay = 1.0f - P.lr * P.wd;
  const float step = P.lr * E.scale;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const uint64_t i0 = base + uint64_t(h) * kHalf + uint64_t(threadIdx.x) * 4;
    if (E.vec && i0 + 4 <= E.size) {
      float4 w = *reinterpret_cast<const float4*>(E.w + i0);
      const uint2 ou = *reinterpret_cast<const uint2*>(E.u + i0);
      const uint16_t* o = reinterpret_cast<const uint16_t*>(&ou);
      w.x = w.x * decay - step * bf2f(o[0]);
      w.y = w.y * decay - step * bf2f(o[1]);
      w.z = w.z * decay - step * bf2f(o[2]);
      w.w = w.w * decay - step * bf2f(o[3]);
      *reinterpret_cast<float4*>(E.w + i0) = w;
    } else {
      for (int j = 0; j < 4; ++j) {
        const uint64_t i = i0 + j;
        if (i >= E.size) break;
        E.w[i] = E.w[i] * decay - step * bf2f(E.u[i]);
      }
    }
  }
}

}  // namespace opt

hipError_t launch_opt(int apply, const OptPhase& P, hipStream_t st) {
  if (P.total == 0) return hipSuccess;
  if (apply) hipLaunchKernelGGL(opt::k_opt_apply, dim3(P.total), dim3(256), 0, st, P);
  else hipLaunchKernelGGL(opt::k_opt_momentum, dim3(P.total), dim3(256), 0, st, P);
  return hipGetLastError();
}

}  // namespace tmk
