// Observation encoder on the GPU: a ResNet-18-topology image network with
// GroupNorm and global average pooling (the pretrained policy's encoder,
// which the method leaves unchanged, Sec. 3.1 and Sec. 3.4).
//
// Activations are NHWC fp32 in HBM.  Convolutions are implicit GEMMs on
// MFMA: M = output pixels, N = output channels, K = kh * kw * Cin in
// (kh, kw, Cin) order, which is the packed weight layout [Cout][K] (padded
// to the K step).  The A tile is gathered from the input with the
// convolution's padding on the fly (no im2col buffer) and converted to the
// operand type in LDS.  GroupNorm is a statistics pass (per image and group,
// fp32 partial sums reduced in fp64) and an elementwise pass that applies
// the affine, the optional residual and ReLU.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <vector>

#include "evo_host.hpp"
#include "evo_kernels.hpp"

using namespace evo;

namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));

constexpr int kBM = 64, kBN = 64, kThreads = 256;

template <class AT> struct ConvOp;
template <> struct ConvOp<__bf16> {
  static constexpr int KS = 32;  // K per step: one 16x16x32 MFMA per tile
};
template <> struct ConvOp<float> {
  static constexpr int KS = 16;  // K per step: four 16x16x4 MFMAs per tile
};

__device__ __forceinline__ void put(__bf16* p, float v) { *p = (__bf16)v; }
__device__ __forceinline__ void put(float* p, float v) { *p = v; }

struct ConvArgs {
  const float* x;   // [N][H][W][Cin]
  const void* w;    // [Cout][Kp] operand type
  float* y;         // [N][Ho][Wo][Cout]
  int N, H, W, Cin, Ho, Wo, Cout, kh, kw, stride, pad, K, Kp;
};

// One 64 x 64 output tile per workgroup; wave (wm, wn) owns a 32 x 32 quarter
// as 2 x 2 MFMA tiles.  Thread t stages A row t / 4 (one output pixel) and B
// row t / 4 (one output channel), 8 consecutive K elements each.
template <class AT>
__global__ void __launch_bounds__(kThreads) conv_kernel(const ConvArgs a) {
  constexpr int KS = ConvOp<AT>::KS, LDK = KS + 8;
  __shared__ __attribute__((aligned(16))) AT As[kBM * LDK];
  __shared__ __attribute__((aligned(16))) AT Bs[kBN * LDK];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int wm = w >> 1, wn = w & 1;
  const int M = a.N * a.Ho * a.Wo;
  const int m0 = blockIdx.x * kBM, n0 = blockIdx.y * kBN;
  // the staged A row: output pixel (n, oh, ow)
  const int ar = tid >> 2, aseg = (tid & 3) * (KS / 4);
  const int pm = m0 + ar;
  const bool prow = pm < M;
  int pn = 0, poh = 0, pow_ = 0;
  if (prow) {
    pn = pm / (a.Ho * a.Wo);
    const int r = pm - pn * a.Ho * a.Wo;
    poh = r / a.Wo;
    pow_ = r - poh * a.Wo;
  }
  const int ih0 = poh * a.stride - a.pad, iw0 = pow_ * a.stride - a.pad;
  const float* xn = a.x + (size_t)pn * a.H * a.W * a.Cin;
  // the staged B row: output channel n0 + ar
  const int bc = n0 + ar;
  const AT* wrow = reinterpret_cast<const AT*>(a.w) + (size_t)(bc < a.Cout ? bc : 0) * a.Kp;
  const bool vec = (a.Cin % (KS / 4)) == 0;  // the thread's K run stays inside one input pixel

  f32x4 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int k0 = 0; k0 < a.Kp; k0 += KS) {
    // ---- stage A: KS / 4 consecutive K of this pixel
    {
      AT* dst = As + ar * LDK + aseg;
      const int kk = k0 + aseg;
      if (vec) {
        float v[KS / 4];
#pragma unroll
        for (int q = 0; q < KS / 4; ++q) v[q] = 0.f;
        if (prow && kk < a.K) {
          const int c = kk % a.Cin, ab = kk / a.Cin;
          const int kb = ab % a.kw, ka = ab / a.kw;
          const int ih = ih0 + ka, iw = iw0 + kb;
          if (ih >= 0 && ih < a.H && iw >= 0 && iw < a.W) {
            const f32x4* src = reinterpret_cast<const f32x4*>(xn + ((size_t)ih * a.W + iw) * a.Cin + c);
#pragma unroll
            for (int q = 0; q < KS / 16; ++q) {
              const f32x4 t = src[q];
              v[4 * q] = t[0];
              v[4 * q + 1] = t[1];
              v[4 * q + 2] = t[2];
              v[4 * q + 3] = t[3];
            }
          }
        }
#pragma unroll
        for (int q = 0; q < KS / 4; ++q) put(dst + q, v[q]);
      } else {
#pragma unroll
        for (int q = 0; q < KS / 4; ++q) {
          const int k = kk + q;
          float v = 0.f;
          if (prow && k < a.K) {
            const int c = k % a.Cin, ab = k / a.Cin;
            const int kb = ab % a.kw, ka = ab / a.kw;
            const int ih = ih0 + ka, iw = iw0 + kb;
            if (ih >= 0 && ih < a.H && iw >= 0 && iw < a.W) v = xn[((size_t)ih * a.W + iw) * a.Cin + c];
          }
          put(dst + q, v);
        }
      }
    }
    // ---- stage B: KS / 4 consecutive K of this output channel (zero padded in memory)
    {
      AT* dst = Bs + ar * LDK + aseg;
      if (bc < a.Cout) {
        const AT* src = wrow + k0 + aseg;
#pragma unroll
        for (int q = 0; q < KS / 4; ++q) dst[q] = src[q];
      } else {
#pragma unroll
        for (int q = 0; q < KS / 4; ++q) put(dst + q, 0.f);
      }
    }
    __syncthreads();
    const int lr = lane & 15, lq = lane >> 4;
    if constexpr (sizeof(AT) == 2) {
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const uint4 av = *reinterpret_cast<const uint4*>(As + (wm * 32 + i * 16 + lr) * LDK + lq * 8);
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const uint4 bv = *reinterpret_cast<const uint4*>(Bs + (wn * 32 + j * 16 + lr) * LDK + lq * 8);
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, av),
                                                              __builtin_bit_cast(bf16x8_t, bv), acc[i][j], 0, 0, 0);
        }
      }
    } else {
#pragma unroll
      for (int s4 = 0; s4 < 4; ++s4)
#pragma unroll
        for (int i = 0; i < 2; ++i) {
          const float av = As[(wm * 32 + i * 16 + lr) * LDK + s4 * 4 + lq];
#pragma unroll
          for (int j = 0; j < 2; ++j) {
            const float bv = Bs[(wn * 32 + j * 16 + lr) * LDK + s4 * 4 + lq];
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(av, bv, acc[i][j], 0, 0, 0);
          }
        }
    }
    __syncthreads();
  }
  // ---- D: lane holds rows 4 * (lane / 16) + r of column lane % 16 of each tile
  const int lr = lane & 15, lq = lane >> 4;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int col = n0 + wn * 32 + j * 16 + lr;
      if (col >= a.Cout) continue;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = m0 + wm * 32 + i * 16 + lq * 4 + r;
        if (row < M) a.y[(size_t)row * a.Cout + col] = acc[i][j][r];
      }
    }
}

// GroupNorm statistics: one workgroup per (image, group); mean and 1/sqrt(var + eps)
__global__ void __launch_bounds__(256) gn_stats_kernel(const float* __restrict__ x, int HW, int C, int G,
                                                       float eps, float2* __restrict__ stats) {
  const int ng = blockIdx.x, groups = C / G;
  const int n = ng / groups, g = ng % groups;
  const float* base = x + (size_t)n * HW * C + (size_t)g * G;
  // sums of (x - x0) with x0 the group's first element, so that a mean far
  // from zero does not cancel the variance
  const float x0 = base[0];
  float s = 0.f, q = 0.f;
  for (int e = threadIdx.x; e < HW * G; e += 256) {
    const int p = e / G, c = e - p * G;
    const float v = base[(size_t)p * C + c] - x0;
    s += v;
    q += v * v;
  }
  __shared__ double rs[256], rq[256];
  rs[threadIdx.x] = s;
  rq[threadIdx.x] = q;
  __syncthreads();
  for (int h = 128; h > 0; h >>= 1) {
    if (threadIdx.x < h) {
      rs[threadIdx.x] += rs[threadIdx.x + h];
      rq[threadIdx.x] += rq[threadIdx.x + h];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const double cnt = (double)HW * G;
    const double m = rs[0] / cnt;
    const double var = std::max(rq[0] / cnt - m * m, 0.0);
    stats[ng] = make_float2((float)((double)x0 + m), (float)(1.0 / std::sqrt(var + (double)eps)));
  }
}

// y = [relu]((x - mean) rstd gamma + beta [+ res]); element i of [N][HW][C]
// (x and y may be the same buffer: every element is read and written by one thread)
__global__ void __launch_bounds__(256) gn_apply_kernel(const float* x, const float2* __restrict__ stats,
                                                       const float* __restrict__ gamma, const float* __restrict__ beta,
                                                       const float* res, int relu, long long total, int HW, int C,
                                                       int G, float* y) {
  const int groups = C / G;
  for (long long i = (long long)blockIdx.x * 256 + threadIdx.x; i < total; i += (long long)gridDim.x * 256) {
    const int c = (int)(i % C);
    const long long n = i / ((long long)HW * C);
    const float2 st = stats[n * groups + c / G];
    float v = (x[i] - st.x) * st.y * gamma[c] + beta[c];
    if (res) v += res[i];
    y[i] = relu ? fmaxf(v, 0.f) : v;
  }
}

// 3x3 stride-2 max pooling, padding 1 (padding excluded)
__global__ void __launch_bounds__(256) max_pool_kernel(const float* __restrict__ x, int N, int H, int W, int C,
                                                       int Ho, int Wo, float* __restrict__ y) {
  const long long total = (long long)N * Ho * Wo * C;
  for (long long i = (long long)blockIdx.x * 256 + threadIdx.x; i < total; i += (long long)gridDim.x * 256) {
    const int c = (int)(i % C);
    long long r = i / C;
    const int ow = (int)(r % Wo);
    r /= Wo;
    const int oh = (int)(r % Ho);
    const int n = (int)(r / Ho);
    float m = -INFINITY;
    for (int a = 0; a < 3; ++a) {
      const int ih = oh * 2 - 1 + a;
      if (ih < 0 || ih >= H) continue;
      for (int b = 0; b < 3; ++b) {
        const int iw = ow * 2 - 1 + b;
        if (iw < 0 || iw >= W) continue;
        m = fmaxf(m, x[(((size_t)n * H + ih) * W + iw) * C + c]);
      }
    }
    y[i] = m;
  }
}

// global average pooling: out[n * stride + c] = mean over pixels
__global__ void __launch_bounds__(256) avg_pool_kernel(const float* __restrict__ x, int N, int HW, int C,
                                                       float* __restrict__ out, int stride) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= N * C) return;
  const int n = i / C, c = i % C;
  float s = 0.f;
  for (int p = 0; p < HW; ++p) s += x[((size_t)n * HW + p) * C + c];
  out[(size_t)n * stride + c] = s / (float)HW;
}

// weights [Cout][K] fp32 -> [Cout][Kp] operand type, zero padded
__global__ void pack_conv_kernel(const float* __restrict__ w, int Cout, int K, int Kp, int bf, void* dst) {
  const long long total = (long long)Cout * Kp;
  for (long long i = (long long)blockIdx.x * 256 + threadIdx.x; i < total; i += (long long)gridDim.x * 256) {
    const int k = (int)(i % Kp), o = (int)(i / Kp);
    const float v = k < K ? w[(size_t)o * K + k] : 0.f;
    if (bf) reinterpret_cast<__bf16*>(dst)[i] = (__bf16)v;
    else reinterpret_cast<float*>(dst)[i] = v;
  }
}

unsigned grid_for(long long total) {
  return (unsigned)std::min<long long>((total + 255) / 256, 16384);
}

struct ConvLayer {
  int cin, cout, k, stride, pad, K, Kp;
  void* w = nullptr;            // packed operand weights
  const float* gamma = nullptr;  // GroupNorm affine (device, inside the raw copy)
  const float* beta = nullptr;
};

}  // namespace

struct evo_encoder {
  evo_encoder_desc desc{};
  int device = 0;
  int bf = 1;
  float* d_raw = nullptr;             // fp32 parameter copy (GroupNorm affine, packing source)
  std::vector<ConvLayer> convs;       // stem, then per block a, b[, d]
  float* buf[4] = {nullptr, nullptr, nullptr, nullptr};
  size_t buf_floats = 0;
  float2* d_stats = nullptr;
  uint64_t flops_per_image = 0;
};

namespace {

int enc_check(const evo_encoder_desc* d) {
  if (!d) return fail(EVO_E_INVALID, "desc is NULL");
  if (d->height < 8 || d->width < 8 || d->height > 4096 || d->width > 4096)
    return fail(EVO_E_INVALID, "image size %d x %d outside [8, 4096]", d->height, d->width);
  if (d->in_ch < 1 || d->in_ch > 64) return fail(EVO_E_INVALID, "in_ch %d outside [1, 64]", d->in_ch);
  if (d->n_stages < 1 || d->n_stages > 4) return fail(EVO_E_INVALID, "n_stages %d outside [1, 4]", d->n_stages);
  if (d->gn_group < 1 || d->stem_ch < 1 || d->stem_ch % d->gn_group)
    return fail(EVO_E_INVALID, "stem_ch %d must be a positive multiple of gn_group %d", d->stem_ch, d->gn_group);
  if (d->stem_ch % 8) return fail(EVO_E_UNSUPPORTED, "stem_ch must be a multiple of 8");
  for (int s = 0; s < d->n_stages; ++s) {
    if (d->widths[s] < 8 || d->widths[s] % 8 || d->widths[s] % d->gn_group || d->widths[s] > 4096)
      return fail(EVO_E_INVALID, "width %d of stage %d must be a multiple of 8 and of gn_group, at most 4096",
                  d->widths[s], s);
    if (d->blocks[s] < 1 || d->blocks[s] > 16) return fail(EVO_E_INVALID, "blocks[%d] = %d", s, d->blocks[s]);
  }
  if (d->dtype != EVO_FP32 && d->dtype != EVO_BF16) return fail(EVO_E_INVALID, "bad dtype");
  if (d->max_batch < 1 || d->max_batch > (1 << 16)) return fail(EVO_E_INVALID, "max_batch %d", d->max_batch);
  // pixel indices of a batch (stem output and below) are 32-bit
  if ((int64_t)d->max_batch * d->height * d->width >= (int64_t(1) << 31))
    return fail(EVO_E_UNSUPPORTED, "max_batch * height * width must stay below 2^31");
  return EVO_OK;
}

// every convolution of the network in execution order (stem; per block a, b, [d])
std::vector<ConvLayer> enc_layers(const evo_encoder_desc* d) {
  std::vector<ConvLayer> v;
  v.push_back({d->in_ch, d->stem_ch, 7, 2, 3, 0, 0});
  int cin = d->stem_ch;
  for (int s = 0; s < d->n_stages; ++s)
    for (int b = 0; b < d->blocks[s]; ++b) {
      const int c = d->widths[s], stride = (s > 0 && b == 0) ? 2 : 1;
      v.push_back({cin, c, 3, stride, 1, 0, 0});
      v.push_back({c, c, 3, 1, 1, 0, 0});
      if (stride != 1 || cin != c) v.push_back({cin, c, 1, stride, 0, 0, 0});
      cin = c;
    }
  return v;
}

inline int out_size(int h, int k, int s, int p) { return (h + 2 * p - k) / s + 1; }

hipError_t launch_conv(const evo_encoder* e, const ConvLayer& L, const float* x, int N, int H, int W, float* y,
                       int* Ho, int* Wo, hipStream_t st) {
  ConvArgs a;
  a.x = x;
  a.w = L.w;
  a.y = y;
  a.N = N;
  a.H = H;
  a.W = W;
  a.Cin = L.cin;
  a.Ho = *Ho = out_size(H, L.k, L.stride, L.pad);
  a.Wo = *Wo = out_size(W, L.k, L.stride, L.pad);
  a.Cout = L.cout;
  a.kh = a.kw = L.k;
  a.stride = L.stride;
  a.pad = L.pad;
  a.K = L.K;
  a.Kp = L.Kp;
  const long long M = (long long)N * a.Ho * a.Wo;
  dim3 grid((unsigned)((M + kBM - 1) / kBM), (unsigned)((L.cout + kBN - 1) / kBN));
  if (e->bf) hipLaunchKernelGGL(conv_kernel<__bf16>, grid, dim3(kThreads), 0, st, a);
  else hipLaunchKernelGGL(conv_kernel<float>, grid, dim3(kThreads), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_gn(const evo_encoder* e, const ConvLayer& L, const float* x, int N, int HW, const float* res,
                     int relu, float* y, hipStream_t st) {
  const int C = L.cout, G = e->desc.gn_group;
  hipLaunchKernelGGL(gn_stats_kernel, dim3((unsigned)(N * (C / G))), dim3(256), 0, st, x, HW, C, G, 1e-5f,
                     e->d_stats);
  const long long total = (long long)N * HW * C;
  hipLaunchKernelGGL(gn_apply_kernel, dim3(grid_for(total)), dim3(256), 0, st, x, e->d_stats, L.gamma, L.beta, res,
                     relu, total, HW, C, G, y);
  return hipGetLastError();
}

}  // namespace

extern "C" {

int64_t evo_encoder_weight_count(const evo_encoder_desc* desc) {
  clear_error();
  int rc = enc_check(desc);
  if (rc) return rc;
  int64_t n = 0;
  for (const ConvLayer& L : enc_layers(desc)) n += (int64_t)L.cout * L.k * L.k * L.cin + 2 * L.cout;
  return n;
}

int evo_create_encoder(const evo_encoder_desc* desc, const float* host_weights, size_t n_floats,
                       evo_encoder** out) {
  clear_error();
  int rc = enc_check(desc);
  if (rc) return rc;
  if (!host_weights || !out) return fail(EVO_E_INVALID, "NULL pointer");
  const int64_t need = evo_encoder_weight_count(desc);
  if ((int64_t)n_floats != need) return fail(EVO_E_INVALID, "n_floats is %zu, this encoder needs %lld", n_floats,
                                             (long long)need);
  evo_encoder* e = new (std::nothrow) evo_encoder();
  if (!e) return fail(EVO_E_NOMEM, "host allocation failed");
  const auto body = [&]() -> int {
    e->desc = *desc;
    e->bf = desc->dtype == EVO_BF16;
    if (hipGetDevice(&e->device) != hipSuccess) return fail(EVO_E_HIP, "no current HIP device");
#define ENC_TRY(expr)                                                                              \
    do {                                                                                           \
      hipError_t e_ = (expr);                                                                      \
      if (e_ != hipSuccess)                                                                        \
        return fail(e_ == hipErrorOutOfMemory ? EVO_E_NOMEM : EVO_E_HIP, "%s failed: %s", #expr,   \
                    hipGetErrorString(e_));                                                        \
    } while (0)
    ENC_TRY(hipMalloc(&e->d_raw, n_floats * sizeof(float)));
    ENC_TRY(hipMemcpy(e->d_raw, host_weights, n_floats * sizeof(float), hipMemcpyHostToDevice));
    e->convs = enc_layers(desc);
    const int KS = e->bf ? 32 : 16;
    size_t off = 0;
    int H = desc->height, W = desc->width, maxg = 0;
    size_t maxact = 0;
    uint64_t flops = 0;
    for (ConvLayer& L : e->convs) {
      L.K = L.k * L.k * L.cin;
      L.Kp = (L.K + KS - 1) / KS * KS;
      ENC_TRY(hipMalloc(&L.w, (size_t)L.cout * L.Kp * (e->bf ? 2 : 4)));
      hipLaunchKernelGGL(pack_conv_kernel, dim3(grid_for((long long)L.cout * L.Kp)), dim3(256), 0, 0,
                         e->d_raw + off, L.cout, L.K, L.Kp, e->bf, L.w);
      ENC_TRY(hipGetLastError());
      off += (size_t)L.cout * L.K;
      L.gamma = e->d_raw + off;
      L.beta = e->d_raw + off + L.cout;
      off += 2 * (size_t)L.cout;
      maxg = std::max(maxg, L.cout / desc->gn_group);
    }
    // activation sizes: walk the network once
    {
      int h = out_size(H, 7, 2, 3), w = out_size(W, 7, 2, 3);
      maxact = std::max(maxact, (size_t)h * w * desc->stem_ch);
      flops += 2ull * h * w * desc->stem_ch * 49 * desc->in_ch;
      h = out_size(h, 3, 2, 1);
      w = out_size(w, 3, 2, 1);
      int cin = desc->stem_ch;
      for (int s = 0; s < desc->n_stages; ++s)
        for (int b = 0; b < desc->blocks[s]; ++b) {
          const int c = desc->widths[s], stride = (s > 0 && b == 0) ? 2 : 1;
          const int ho = out_size(h, 3, stride, 1), wo = out_size(w, 3, stride, 1);
          if (ho < 1 || wo < 1) return fail(EVO_E_INVALID, "the image is too small for the network");
          maxact = std::max(maxact, (size_t)ho * wo * c);
          flops += 2ull * ho * wo * c * 9 * cin + 2ull * ho * wo * c * 9 * c;
          if (stride != 1 || cin != c) flops += 2ull * ho * wo * c * cin;
          h = ho;
          w = wo;
          cin = c;
        }
    }
    e->flops_per_image = flops;
    e->buf_floats = maxact * desc->max_batch;
    for (int i = 0; i < 4; ++i) ENC_TRY(hipMalloc(&e->buf[i], e->buf_floats * sizeof(float)));
    ENC_TRY(hipMalloc(&e->d_stats, (size_t)desc->max_batch * maxg * sizeof(float2)));
    ENC_TRY(hipDeviceSynchronize());
#undef ENC_TRY
    *out = e;
    return (int)EVO_OK;
  };
  rc = guarded(body);
  if (rc) evo_destroy_encoder(e);
  return rc;
}

int evo_encode(evo_encoder* e, int32_t batch, const float* images, float* features_out, int32_t out_stride,
               void* hip_stream) {
  clear_error();
  if (!e) return fail(EVO_E_INVALID, "encoder is NULL");
  const evo_encoder_desc& d = e->desc;
  if (batch < 1 || batch > d.max_batch) return fail(EVO_E_INVALID, "batch %d outside [1, %d]", batch, d.max_batch);
  if (!images || !features_out) return fail(EVO_E_INVALID, "NULL device pointer");
  const int C_out = d.widths[d.n_stages - 1];
  if (out_stride < C_out) return fail(EVO_E_INVALID, "out_stride %d < feature size %d", out_stride, C_out);
  DeviceGuard guard(e->device);
  hipStream_t st = (hipStream_t)hip_stream;
  float *X = e->buf[0], *Y = e->buf[1], *Z = e->buf[2], *R = e->buf[3];
  int H = d.height, W = d.width, Ho, Wo;
  size_t li = 0;
#define ENC_HIP(expr)                                                                               \
  do {                                                                                              \
    hipError_t e_ = (expr);                                                                         \
    if (e_ != hipSuccess) return fail(EVO_E_HIP, "%s failed: %s", #expr, hipGetErrorString(e_));    \
  } while (0)
  // stem: conv 7x7/2, GN, ReLU, max pool 3x3/2
  {
    const ConvLayer& L = e->convs[li++];
    ENC_HIP(launch_conv(e, L, images, batch, H, W, Y, &Ho, &Wo, st));
    ENC_HIP(launch_gn(e, L, Y, batch, Ho * Wo, nullptr, 1, Y, st));
    const int Hp = out_size(Ho, 3, 2, 1), Wp = out_size(Wo, 3, 2, 1);
    const long long total = (long long)batch * Hp * Wp * L.cout;
    hipLaunchKernelGGL(max_pool_kernel, dim3(grid_for(total)), dim3(256), 0, st, Y, batch, Ho, Wo, L.cout, Hp, Wp, X);
    ENC_HIP(hipGetLastError());
    H = Hp;
    W = Wp;
  }
  int cin = d.stem_ch;
  for (int s = 0; s < d.n_stages; ++s)
    for (int b = 0; b < d.blocks[s]; ++b) {
      const int c = d.widths[s];
      const ConvLayer& La = e->convs[li++];
      const ConvLayer& Lb = e->convs[li++];
      const bool proj = La.stride != 1 || cin != c;
      int H2, W2, H3, W3;
      ENC_HIP(launch_conv(e, La, X, batch, H, W, Y, &H2, &W2, st));
      ENC_HIP(launch_gn(e, La, Y, batch, H2 * W2, nullptr, 1, Y, st));
      ENC_HIP(launch_conv(e, Lb, Y, batch, H2, W2, Z, &H3, &W3, st));
      const float* shortcut = X;
      if (proj) {
        const ConvLayer& Ld = e->convs[li++];
        int Hd, Wd;
        ENC_HIP(launch_conv(e, Ld, X, batch, H, W, R, &Hd, &Wd, st));
        ENC_HIP(launch_gn(e, Ld, R, batch, Hd * Wd, nullptr, 0, R, st));
        shortcut = R;
      }
      // block output = ReLU(GN(conv b) + shortcut), written over the block input
      ENC_HIP(launch_gn(e, Lb, Z, batch, H3 * W3, shortcut, 1, Y, st));
      std::swap(X, Y);
      H = H3;
      W = W3;
      cin = c;
    }
  hipLaunchKernelGGL(avg_pool_kernel, dim3((unsigned)((batch * C_out + 255) / 256)), dim3(256), 0, st, X, batch,
                     H * W, C_out, features_out, out_stride);
  ENC_HIP(hipGetLastError());
#undef ENC_HIP
  return EVO_OK;
}

int evo_encoder_flops(const evo_encoder* e, int32_t batch, uint64_t* flops_out) {
  clear_error();
  if (!e || !flops_out) return fail(EVO_E_INVALID, "NULL pointer");
  *flops_out = e->flops_per_image * (uint64_t)std::max(batch, 0);
  return EVO_OK;
}

void evo_destroy_encoder(evo_encoder* e) {
  if (!e) return;
  DeviceGuard guard(e->device);
  (void)hipDeviceSynchronize();
  for (ConvLayer& L : e->convs) (void)hipFree(L.w);
  for (int i = 0; i < 4; ++i) (void)hipFree(e->buf[i]);
  (void)hipFree(e->d_stats);
  (void)hipFree(e->d_raw);
  delete e;
}

}  // extern "C"
