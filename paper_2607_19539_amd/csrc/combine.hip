// combine.hip -- gfx950 kernel of the weighted combine on a source rank (paper Section 2.1,
// step 5): each token's k returned expert rows, weighted by the router's gate values, summed
// in fp32 and rounded to bf16.  HBM-bound gather: every row is read once with 16-byte
// vector loads and the output row is written once.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

#include "kernels.hpp"

namespace moe {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(1))) u32x4 g_u32x4;
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// Two floats -> two bf16, round to nearest even (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t to_bf16x2(float lo, float hi) {
  const f32x2_t v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}

// out[t] = bf16(sum_j gate[t, j] * recv[slot[t, j]]).
// A workgroup covers kVec * 256 16-byte vectors of one token's row; each thread keeps
// kVec * 8 fp32 sums.  The k choices are taken four at a time: the rows of a batch are
// loaded together, then added in choice order as separately rounded products and sums
// (contraction off), so the result does not depend on the batching.  Out-of-range
// slots are skipped and counted.
template <int kVec>
__global__ __launch_bounds__(256) void combine_kernel(CombineArgs a) {
#pragma clang fp contract(off)
  const int64_t nvec = a.H / 8;
  const int64_t spans = (nvec + 256 * kVec - 1) / (256 * kVec);
  const int64_t work = a.tokens * spans;
  for (int64_t w = blockIdx.x; w < work; w += gridDim.x) {
    const int64_t t = w / spans;
    const int64_t span = w - t * spans;
    const int64_t v0 = span * (256 * kVec) + threadIdx.x;
    float acc[kVec][8];
#pragma unroll
    for (int u = 0; u < kVec; ++u)
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[u][e] = 0.0f;
    for (int j0 = 0; j0 < a.k; j0 += 4) {
      u32x4 v[4][kVec];
      float g[4];
      bool ok[4];
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        const int j = j0 + jj;
        const int32_t s = j < a.k ? a.slot[t * a.k + j] : -1;
        ok[jj] = s >= 0 && (int64_t)s < a.recv_rows;
        if (j < a.k && !ok[jj] && span == 0 && threadIdx.x == 0 && a.bad_slots)
          atomicAdd(a.bad_slots, 1u);
        g[jj] = ok[jj] ? a.gate[t * a.k + j] : 0.0f;
        const u32x4* row = (const u32x4*)(a.recv + (int64_t)(ok[jj] ? s : 0) * a.H);
#pragma unroll
        for (int u = 0; u < kVec; ++u) {
          const int64_t i = v0 + u * 256;
          v[jj][u] = (ok[jj] && i < nvec) ? row[i] : u32x4{0u, 0u, 0u, 0u};
        }
      }
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        if (!ok[jj]) continue;
#pragma unroll
        for (int u = 0; u < kVec; ++u)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const uint32_t word = v[jj][u][q];
            const float lo = __uint_as_float(word << 16), hi = __uint_as_float(word & 0xFFFF0000u);
            acc[u][2 * q] = acc[u][2 * q] + g[jj] * lo;
            acc[u][2 * q + 1] = acc[u][2 * q + 1] + g[jj] * hi;
          }
      }
    }
    g_u32x4* dst = (g_u32x4*)(a.out + t * a.H);
#pragma unroll
    for (int u = 0; u < kVec; ++u) {
      const int64_t i = v0 + u * 256;
      if (i < nvec) {
        u32x4 o;
#pragma unroll
        for (int q = 0; q < 4; ++q) o[q] = to_bf16x2(acc[u][2 * q], acc[u][2 * q + 1]);
        dst[i] = o;
      }
    }
  }
}

hipError_t launch_combine(const CombineArgs& a, hipStream_t s) {
  if (a.tokens <= 0) return hipSuccess;
  const int64_t nvec = a.H / 8;
  const int vec = nvec <= 256 ? 1 : nvec <= 512 ? 2 : 4;
  const int64_t spans = (nvec + 256 * vec - 1) / (256 * vec);
  const int grid = (int)std::min<int64_t>(a.tokens * spans, 65536);
  if (vec == 1)
    hipLaunchKernelGGL(combine_kernel<1>, dim3(grid), dim3(256), 0, s, a);
  else if (vec == 2)
    hipLaunchKernelGGL(combine_kernel<2>, dim3(grid), dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(combine_kernel<4>, dim3(grid), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace moe
