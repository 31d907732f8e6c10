// Redundancy-aware initialisation of the schedule search (Sec. 3.3): the
// dissimilarity score of Eq. 6 from activations recorded by the uncached
// policy.  For every query r and unit b a workgroup forms the step x step
// Gram matrix of that unit's activation vectors on fp32 MFMA and reduces it
// to the mean cosine dissimilarity of each step against the other steps;
// a second kernel averages the queries in order (deterministic).
#include <hip/hip_runtime.h>

#include "evo_kernels.hpp"

namespace evo {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kNW = 4;            // waves per workgroup
constexpr int kKC = 64;           // activation elements per LDS chunk
constexpr int kMT = kGramMaxSteps / 16;          // step tiles (max)
constexpr int kIT = (kMT + kNW - 1) / kNW;       // step tiles per wave (max)
constexpr int kLD = kKC + 4;      // LDS row stride (floats)

__device__ __forceinline__ f32x4 mfma4(float a, float b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float row16_sum(float v) {
  v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0xB1, 0xF, 0xF, true));
  v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x4E, 0xF, 0xF, true));
  v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x141, 0xF, 0xF, true));
  v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x140, 0xF, 0xF, true));
  return v;
}

// part[r][b][t] = 1/(T-1) sum_{t' != t} (1 - cos(a_{r,b,t}, a_{r,b,t'})),
// a zero vector's cosine taken as 0.  Grid: R * U workgroups of kNW waves.
__global__ void __launch_bounds__(kNW * 64) gram_kernel(const float* __restrict__ acts, int U, int T, long long V,
                                                        float* __restrict__ part) {
  __shared__ __attribute__((aligned(16))) float tile[kGramMaxSteps * kLD];
  __shared__ float nrm[kGramMaxSteps];
  const int rb = blockIdx.x;  // r * U + b
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, lc = lane & 15, lq = lane >> 4;
  const int MT = (T + 15) / 16;
  const float* A = acts + (size_t)rb * T * V;
  // G tiles owned by this wave: rows of step tile i = w + kNW * ii, columns of every step tile
  f32x4 g[kIT][kMT];
#pragma unroll
  for (int ii = 0; ii < kIT; ++ii)
#pragma unroll
    for (int j = 0; j < kMT; ++j) g[ii][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (long long k0 = 0; k0 < V; k0 += kKC) {
    __syncthreads();
    // stage steps x kKC elements; rows >= T and elements >= V are zero
    for (int it = tid; it < MT * 16 * (kKC / 4); it += kNW * 64) {
      const int row = it / (kKC / 4), c4 = it % (kKC / 4);
      const long long k = k0 + 4 * c4;
      f32x4 v = f32x4{0.f, 0.f, 0.f, 0.f};
      if (row < T) {
        const float* src = A + (size_t)row * V + k;
        if (k + 4 <= V && (V & 3) == 0) {
          v = *reinterpret_cast<const f32x4*>(src);
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = (k + e < V) ? src[e] : 0.f;
        }
      }
      *reinterpret_cast<f32x4*>(tile + row * kLD + 4 * c4) = v;
    }
    __syncthreads();
    // the chunk's contribution: lane (row lc, group lq) takes k = 16 lq + s at
    // step s (a permutation of k shared by both operands)
#pragma unroll
    for (int ii = 0; ii < kIT; ++ii) {
      const int i = w + kNW * ii;
      if (i >= MT) break;
      f32x4 a[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) a[q] = *reinterpret_cast<const f32x4*>(tile + (i * 16 + lc) * kLD + 16 * lq + 4 * q);
#pragma unroll
      for (int j = 0; j < kMT; ++j) {
        if (j >= MT) break;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const f32x4 bq = *reinterpret_cast<const f32x4*>(tile + (j * 16 + lc) * kLD + 16 * lq + 4 * q);
#pragma unroll
          for (int e = 0; e < 4; ++e) g[ii][j] = mfma4(a[q][e], bq[e], g[ii][j]);
        }
      }
    }
  }
  // squared norms from the diagonal tiles (D layout: lane holds column lc,
  // rows 4 lq + e of the tile)
  __syncthreads();
#pragma unroll
  for (int ii = 0; ii < kIT; ++ii) {
    const int i = w + kNW * ii;
    if (i >= MT) break;
#pragma unroll
    for (int j = 0; j < kMT; ++j)
      if (j == i) {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (4 * lq + e == lc) nrm[i * 16 + lc] = g[ii][j][e];
      }
  }
  __syncthreads();
#pragma unroll
  for (int ii = 0; ii < kIT; ++ii) {
    const int i = w + kNW * ii;
    if (i >= MT) break;
    float sum[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < kMT; ++j) {
      if (j >= MT) break;
      const int tc = j * 16 + lc;  // column step t'
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int tr = i * 16 + 4 * lq + e;  // row step t
        float dis = 0.f;
        if (tc < T && tr < T && tc != tr) {
          const float n2 = nrm[tr] * nrm[tc];
          const float cs = n2 > 0.f ? g[ii][j][e] / sqrtf(n2) : 0.f;
          dis = 1.f - cs;
        }
        sum[e] += dis;
      }
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float tot = row16_sum(sum[e]);
      const int tr = i * 16 + 4 * lq + e;
      if (lc == 0 && tr < T) part[(size_t)rb * T + tr] = tot / (float)(T - 1);
    }
  }
}

__global__ void mean_kernel(const float* __restrict__ part, int R, int n, float* __restrict__ d) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  float s = 0.f;
  for (int r = 0; r < R; ++r) s += part[(size_t)r * n + i];
  d[i] = s / (float)R;
}

}  // namespace

hipError_t launch_redundancy(const float* acts, int R, int U, int T, long long V, float* part, float* d,
                             hipStream_t stream) {
  if (R < 1 || U < 1 || T < 2 || T > kGramMaxSteps || V < 1) return hipErrorInvalidValue;
  hipLaunchKernelGGL(gram_kernel, dim3(R * U), dim3(kNW * 64), 0, stream, acts, U, T, V, part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int n = U * T;
  hipLaunchKernelGGL(mean_kernel, dim3((n + 255) / 256), dim3(256), 0, stream, part, R, n, d);
  return hipGetLastError();
}

}  // namespace evo
