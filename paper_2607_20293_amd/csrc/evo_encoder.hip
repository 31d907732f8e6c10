// Observation encoder on the GPU: a ResNet-18-topology image network with
// GroupNorm and global average pooling (the pretrained policy's encoder,
// which the method leaves unchanged, Sec. 3.1 and Sec. 3.4).
//
// Activations are NHWC fp32 in HBM.  Convolutions are implicit GEMMs on
// MFMA: M = output pixels, N = output channels, K = kh * kw * Cin in
// (kh, kw, Cin) order, which is the packed weight layout [Cout][Kp] (K
// padded to the K step).  The A tile is gathered from the input with the
// convolution's padding on the fly (no im2col buffer), converted to the
// operand type and double-buffered in LDS with the next step's global loads
// in flight during the current step's MFMAs, in 64 x 64 output tiles.  The
// gather keeps its K position (kernel tap and channel) from step to step
// instead of dividing, and every lane loads: positions outside the input
// (padding, rows beyond the output, K beyond the kernel) read a small block
// of zero bytes, so no branch surrounds the loads.
// Layers with few output tiles (small batches, late stages) split K over
// workgroups into partial outputs that the GroupNorm statistics pass sums
// in a fixed order.
//
// GroupNorm statistics are shifted sums (x - x0, x0 the group's first
// element), fp32 per thread and fp64 across threads.  Where there are many
// (image, channel chunk) workgroups or the map is small, one kernel per
// GroupNorm takes an image's groups whole (statistics, then apply);
// otherwise two passes: partial statistics over pixel chunks, then apply.
// The apply adds the residual and ReLU and, where the network pools next,
// does the pooling itself: 3x3/2 max pooling after the stem, global average
// pooling after the last block (the last block's output is never stored).
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

constexpr int kThreads = 256;
constexpr int kTargetWG = 512;      // split K below this many output tiles
constexpr int kMaxSplit = 16;
constexpr long long kWsFloats = 1024ll * 4096;  // split-K partials (>= splits * tiles * 64 * 64)
// GroupNorm workgroups aimed at when chunking an image's pixels (statistics
// and apply passes).  The K splits of the convolutions and the pixel chunks
// of the GroupNorm statistics are planned for the encoder's max_batch, not
// for the batch of a call: every call then sums an image's products and
// statistics in the same groupings, so an image's features do not depend on
// the batch size or on the other images.  A smaller batch runs the same
// per-image plan on fewer workgroups (an encoder meant for small batches is
// created with a small max_batch).  The apply pass is elementwise, so its
// chunking follows the call's batch.  (Fixed chunks of 64 or 128 pixels
// measured 3-8% slower.)
constexpr int kGnTarget = 1024;
// One GroupNorm kernel instead of two for maps of at most kFusedPixels
// pixels, and for maps of at most kFusedPixelsWide pixels where the
// max_batch plan has at least kFusedWG (image, channel chunk) workgroups;
// with fewer workgroups than kFusedWG it takes one group per workgroup.
// (Measured on 84x84 frames: 2 frames 0.290 -> 0.279 ms; one kernel for
// every map at 2 frames 0.50 ms; at 512 frames the stem's 1764-pixel maps
// took 165 us in one kernel against 126 us in two, the 441-pixel maps 10%
// less in one.)
constexpr int kFusedWG = 256;
constexpr int kFusedPixels = 128;
constexpr int kFusedPixelsWide = 1024;

template <class AT> struct ConvStep;
template <> struct ConvStep<__bf16> {
  static constexpr int KS = 64;  // K per stage: two 16x16x32 MFMAs per tile
};
template <> struct ConvStep<float> {
  static constexpr int KS = 32;  // K per stage: eight 16x16x4 MFMAs per tile
};

struct ConvArgs {
  const float* x;    // [N][H][W][Cin]
  const void* w;     // [Cout][Kp] operand type
  float* y;          // [N][Ho][Wo][Cout], or split z at y + z * split_stride
  const float* zeros;  // 64 zero bytes (16-byte aligned): the source of loads outside the input
  int H, W, Cin, Ho, Wo, Cout, kw, stride, pad, K, Kp;
  int M, mt, nt, splits, spp;  // pixels, tile counts, K splits, K steps per split
  long long split_stride;
};

// Maps a workgroup to a logical tile so that the workgroups of one XCD
// (blockIdx % 8) take a contiguous range of logical ids: neighbouring tiles
// that share input pixels or weights then meet in the same L2.
__device__ __forceinline__ int xcd_linear(int b, int total) {
  const int per = total >> 3, rem = total & 7, xcd = b & 7, slot = b >> 3;
  return xcd < rem ? xcd * (per + 1) + slot : rem * (per + 1) + (xcd - rem) * per + slot;
}

// Block tile BM x BN, 4 waves as 2 x 2, wave tile (BM/2) x (BN/2) of 16x16
// MFMA tiles.  Thread t stages chunk t % 4 (SEG = KS / 4 consecutive K) of
// rows t / 4 + p * 64 of the A (pixels) and B (output channels) tiles.
template <class AT, int BM, int BN>
__global__ void __launch_bounds__(kThreads) conv_kernel(const ConvArgs a) {
  constexpr int KS = ConvStep<AT>::KS, LDK = KS + 8, SEG = KS / 4, CPR = 4, RPP = kThreads / CPR;
  constexpr int PA = BM / RPP, PB = BN / RPP, MI = BM / 32, NJ = BN / 32;
  constexpr int BV = SEG * (int)sizeof(AT) / 16;  // 16-byte loads per B chunk
  static_assert(BM % RPP == 0 && BN % RPP == 0, "tile rows must be a multiple of the staging rows");
  __shared__ __attribute__((aligned(16))) AT As[2][BM * LDK];
  __shared__ __attribute__((aligned(16))) AT Bs[2][BN * LDK];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, wm = wv >> 1, wn = wv & 1;
  const int lr = lane & 15, lq = lane >> 4;

  const int id = xcd_linear(blockIdx.x, a.mt * a.nt * a.splits);
  const int nti = id % a.nt, rest = id / a.nt, mti = rest % a.mt, z = rest / a.mt;
  const int m0 = mti * BM, n0 = nti * BN;
  const int steps = a.Kp / KS;
  const int s_begin = z * a.spp, s_end = min(steps, s_begin + a.spp);

  const int chunk = tid % CPR, row0 = tid / CPR;
  // the A rows this thread stages: output pixel -> image base and window origin
  // (rlo, rhi: the part of a kernel row of kw * Cin contiguous K elements
  // that falls inside the image horizontally)
  // (wo0: element offset of the window origin within the image, negative
  // where the window starts in the padding; an image has fewer than 2^31
  // elements, checked at creation)
  const float* xb[PA];
  int ih0[PA], iw0[PA], wo0[PA], rlo[PA], rhi[PA];
  bool pv[PA];
#pragma unroll
  for (int p = 0; p < PA; ++p) {
    const int pm = m0 + row0 + p * RPP;
    pv[p] = pm < a.M;
    const int hw = a.Ho * a.Wo;
    const int pn = pv[p] ? pm / hw : 0;
    const int r = pv[p] ? pm - pn * hw : 0;
    const int oh = r / a.Wo, ow = r - oh * a.Wo;
    xb[p] = a.x + (size_t)pn * a.H * a.W * a.Cin;
    ih0[p] = oh * a.stride - a.pad;
    iw0[p] = ow * a.stride - a.pad;
    wo0[p] = (ih0[p] * a.W + iw0[p]) * a.Cin;
    rlo[p] = max(0, -iw0[p]) * a.Cin;
    rhi[p] = min(a.kw, a.W - iw0[p]) * a.Cin;
  }
  // weight rows beyond Cout read the zero bytes (their B step is SEG
  // operands, at most 64 bytes)
  const AT* wb[PB];
  bool bv[PB];
#pragma unroll
  for (int p = 0; p < PB; ++p) {
    const int c = n0 + row0 + p * RPP;
    bv[p] = c < a.Cout;
    wb[p] = reinterpret_cast<const AT*>(a.w) + (size_t)(bv[p] ? c : 0) * a.Kp + chunk * SEG;
  }
  const bool vec = (a.Cin % SEG) == 0;  // a chunk then lies inside one input pixel

  // one K step of staged operands
  struct Regs {
    float a[PA][SEG];
    uint4 b[PB][BV];
  };

  // the K position of this thread's chunk, advanced by KS per step (loads
  // are requested for consecutive steps): vec: tap (ka, kb) and channel c;
  // otherwise kernel row ka0 and offset r0 within it
  int kc = 0, kka = 0, kkb = 0;
  const int rowlen = a.kw * a.Cin;
  {
    const int kk0 = s_begin * KS + chunk * SEG;
    if (vec) {
      const int pix = kk0 / a.Cin;
      kc = kk0 - pix * a.Cin;
      kka = pix / a.kw;
      kkb = pix - kka * a.kw;
    } else {
      kka = kk0 / rowlen;
      kc = kk0 - kka * rowlen;
    }
  }
  const auto advance = [&]() {
    kc += KS;
    if (vec) {
      while (kc >= a.Cin) {
        kc -= a.Cin;
        if (++kkb == a.kw) {
          kkb = 0;
          ++kka;
        }
      }
    } else {
      while (kc >= rowlen) {
        kc -= rowlen;
        ++kka;
      }
    }
  };
  auto load = [&](Regs& rg, int s) {
    const int kk = s * KS + chunk * SEG;
    if (vec) {
      // every lane loads: from the input inside the image, from the zero
      // bytes outside it (no branch around the loads; the tests are combined
      // with & so that they compile to compares and selects)
      const int ka = kka, kb = kkb, toff = (ka * a.W + kb) * a.Cin + kc;
#pragma unroll
      for (int p = 0; p < PA; ++p) {
        const int ih = ih0[p] + ka, iw = iw0[p] + kb;
        const bool in = pv[p] & (kk < a.K) & (ih >= 0) & (ih < a.H) & (iw >= 0) & (iw < a.W);
        const f32x4* src = reinterpret_cast<const f32x4*>(in ? xb[p] + (wo0[p] + toff) : a.zeros);
#pragma unroll
        for (int q = 0; q < SEG / 4; ++q) {
          const f32x4 t = src[q];
          rg.a[p][4 * q] = t[0];
          rg.a[p][4 * q + 1] = t[1];
          rg.a[p][4 * q + 2] = t[2];
          rg.a[p][4 * q + 3] = t[3];
        }
      }
    } else {
      // walk the chunk along kernel rows: K element (ka, r) sits at input
      // row ih0 + ka, offset iw0 * Cin + r of that row
      const int ka0 = kka, r0 = kc;
#pragma unroll
      for (int p = 0; p < PA; ++p) {
        int ka = ka0, r = r0;
#pragma unroll
        for (int q = 0; q < SEG; ++q) {
          const int ih = ih0[p] + ka;
          const bool in = pv[p] & (kk + q < a.K) & (ih >= 0) & (ih < a.H) & (r >= rlo[p]) & (r < rhi[p]);
          rg.a[p][q] = *(in ? xb[p] + ((ih * a.W + iw0[p]) * a.Cin + r) : a.zeros);
          if (++r == rowlen) {
            r = 0;
            ++ka;
          }
        }
      }
    }
#pragma unroll
    for (int p = 0; p < PB; ++p) {
      const uint4* src = bv[p] ? reinterpret_cast<const uint4*>(wb[p] + (size_t)s * KS)
                               : reinterpret_cast<const uint4*>(a.zeros);
#pragma unroll
      for (int q = 0; q < BV; ++q) rg.b[p][q] = src[q];
    }
    advance();
  };
  auto store = [&](const Regs& rg, int buf) {
#pragma unroll
    for (int p = 0; p < PA; ++p) {
      AT* dst = As[buf] + (row0 + p * RPP) * LDK + chunk * SEG;
      if constexpr (sizeof(AT) == 2) {
#pragma unroll
        for (int h = 0; h < SEG / 8; ++h) {
          bf16x8_t t;
#pragma unroll
          for (int q = 0; q < 8; ++q) t[q] = (__bf16)rg.a[p][8 * h + q];
          *reinterpret_cast<bf16x8_t*>(dst + 8 * h) = t;
        }
      } else {
#pragma unroll
        for (int h = 0; h < SEG / 4; ++h)
          *reinterpret_cast<f32x4*>(dst + 4 * h) =
              f32x4{rg.a[p][4 * h], rg.a[p][4 * h + 1], rg.a[p][4 * h + 2], rg.a[p][4 * h + 3]};
      }
    }
#pragma unroll
    for (int p = 0; p < PB; ++p) {
      uint4* dst = reinterpret_cast<uint4*>(Bs[buf] + (row0 + p * RPP) * LDK + chunk * SEG);
#pragma unroll
      for (int q = 0; q < BV; ++q) dst[q] = rg.b[p][q];
    }
  };

  f32x4 acc[MI][NJ];
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < NJ; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto compute = [&](int buf) {
    const AT* A = As[buf] + (wm * (BM / 2) + lr) * LDK;
    const AT* B = Bs[buf] + (wn * (BN / 2) + lr) * LDK;
    if constexpr (sizeof(AT) == 2) {
#pragma unroll
      for (int kk = 0; kk < KS / 32; ++kk) {
        bf16x8_t af[MI], bf[NJ];
#pragma unroll
        for (int i = 0; i < MI; ++i) af[i] = *reinterpret_cast<const bf16x8_t*>(A + i * 16 * LDK + kk * 32 + lq * 8);
#pragma unroll
        for (int j = 0; j < NJ; ++j) bf[j] = *reinterpret_cast<const bf16x8_t*>(B + j * 16 * LDK + kk * 32 + lq * 8);
#pragma unroll
        for (int i = 0; i < MI; ++i)
#pragma unroll
          for (int j = 0; j < NJ; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bf[j], acc[i][j], 0, 0, 0);
      }
    } else {
#pragma unroll
      for (int k4 = 0; k4 < KS / 4; ++k4) {
        float af[MI], bf[NJ];
#pragma unroll
        for (int i = 0; i < MI; ++i) af[i] = A[i * 16 * LDK + k4 * 4 + lq];
#pragma unroll
        for (int j = 0; j < NJ; ++j) bf[j] = B[j * 16 * LDK + k4 * 4 + lq];
#pragma unroll
        for (int i = 0; i < MI; ++i)
#pragma unroll
          for (int j = 0; j < NJ; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(af[i], bf[j], acc[i][j], 0, 0, 0);
      }
    }
  };

  // Step i computes from LDS buffer i % 2 while the loads of step i + 1 are
  // in flight; they go to the other buffer, which step i - 1 read before the
  // barrier that ended it.  (A second register set for two steps of slack
  // costs occupancy and measured slower.)
  const int n = s_end - s_begin;
  Regs r;
  if (n > 0) {
    load(r, s_begin);
    store(r, 0);
  }
  __syncthreads();
  for (int i = 0; i < n; ++i) {
    const bool more = i + 1 < n;
    if (more) load(r, s_begin + i + 1);
    compute(i & 1);
    if (more) store(r, (i & 1) ^ 1);
    __syncthreads();
  }
  // D: lane holds rows 4 * (lane / 16) + r of column lane % 16 of each tile
  float* y = a.y + (long long)z * a.split_stride;
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int col = n0 + wn * (BN / 2) + j * 16 + lr;
      if (col >= a.Cout) continue;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = m0 + wm * (BM / 2) + i * 16 + lq * 4 + r;
        if (row < a.M) y[(size_t)row * a.Cout + col] = acc[i][j][r];
      }
    }
}

enum { GN_PLAIN = 0, GN_MAXPOOL = 1, GN_AVGPOOL = 2 };

struct GnArgs {
  const float* ws;   // split-K partials (splits > 1): x = sum over z of ws[z * split_stride + i]
  int splits;
  long long split_stride;
  float* x;          // conv output [N][HW][C] (written by the statistics pass when splits > 1)
  const float* gamma;
  const float* beta;
  const float* res;  // residual [N][HW][C] or NULL
  float* y;          // PLAIN: [N][HW][C] (may be x); MAXPOOL: [N][Hp][Wp][C]; AVGPOOL: out + n * out_stride
  double2* part;     // [N][groups][ps_stats] shifted (sum, sum of squares)
  float* shift;      // [N][groups] the shift x0 (read before the apply pass may overwrite x in place)
  int relu, mode, H, W, C, G, gpw, ps_stats, ps_apply, Hp, Wp, out_stride;
  float eps;
};

// Statistics pass: workgroup (image n, channel chunk of gpw groups, pixel
// chunk); thread t reads float4 column t % Q of pixel rows t / Q + i * RP.
// Sums are of (x - x0), x0 the group's first element, so that a mean far
// from zero does not cancel the variance.
__global__ void __launch_bounds__(kThreads) gn_stats_kernel(const GnArgs a) {
  const int HW = a.H * a.W, CW = a.G * a.gpw, Q = CW >> 2, RP = kThreads / Q;
  const int chunks = a.C / CW, groups = a.C / a.G;
  const int pi = blockIdx.x % a.ps_stats, rest = blockIdx.x / a.ps_stats;
  const int ch = rest % chunks, n = rest / chunks;
  const int tid = threadIdx.x, col = tid % Q, prow = tid / Q;
  const int c = ch * CW + col * 4, j = (col * 4) / a.G;
  const size_t base = (size_t)n * HW * a.C;
  const int pc = (HW + a.ps_stats - 1) / a.ps_stats, p0 = pi * pc, p1 = min(HW, p0 + pc);
  const bool split = a.splits > 1;

  float x0;
  {
    const size_t i0 = base + ch * CW + j * a.G;
    if (!split) {
      x0 = a.x[i0];
    } else {  // all partials requested before the first is added (same order of additions)
      float t[kMaxSplit];
#pragma unroll
      for (int z = 0; z < kMaxSplit; ++z) t[z] = z < a.splits ? a.ws[(long long)z * a.split_stride + i0] : 0.f;
      x0 = t[0];
#pragma unroll
      for (int z = 1; z < kMaxSplit; ++z)
        if (z < a.splits) x0 += t[z];
    }
  }
  float s = 0.f, q = 0.f;
  for (int p = p0 + prow; p < p1; p += RP) {
    const size_t i = base + (size_t)p * a.C + c;
    f32x4 v;
    if (!split) {
      v = *reinterpret_cast<const f32x4*>(a.x + i);
    } else {
      f32x4 t[kMaxSplit];
#pragma unroll
      for (int z = 0; z < kMaxSplit; ++z)
        t[z] = z < a.splits ? *reinterpret_cast<const f32x4*>(a.ws + (long long)z * a.split_stride + i)
                            : f32x4{0.f, 0.f, 0.f, 0.f};
      v = t[0];
#pragma unroll
      for (int z = 1; z < kMaxSplit; ++z)
        if (z < a.splits) v += t[z];
      *reinterpret_cast<f32x4*>(a.x + i) = v;
    }
    const f32x4 d = v - x0;
    s += (d[0] + d[1]) + (d[2] + d[3]);
    q += (d[0] * d[0] + d[1] * d[1]) + (d[2] * d[2] + d[3] * d[3]);
  }
  __shared__ double sd[kThreads], qd[kThreads];
  sd[tid] = s;
  qd[tid] = q;
  __syncthreads();
  for (int h = RP >> 1; h > 0; h >>= 1) {
    if (prow < h) {
      sd[tid] += sd[tid + h * Q];
      qd[tid] += qd[tid + h * Q];
    }
    __syncthreads();
  }
  if (tid < a.gpw) {
    const int cols = a.G >> 2;
    double S = 0.0, Qs = 0.0;
    for (int k = 0; k < cols; ++k) {
      S += sd[tid * cols + k];
      Qs += qd[tid * cols + k];
    }
    a.part[((size_t)n * groups + ch * a.gpw + tid) * a.ps_stats + pi] = make_double2(S, Qs);
  }
  if (pi == 0 && col * 4 % a.G == 0 && prow == 0) a.shift[(size_t)n * groups + ch * a.gpw + j] = x0;
}

// Apply pass: mean and 1/sqrt(var + eps) from the partials, then
// f(v) = [relu]((v - mean) rstd gamma + beta [+ res]) per mode.
__global__ void __launch_bounds__(kThreads) gn_apply_kernel(const GnArgs a) {
  const int HW = a.H * a.W, CW = a.G * a.gpw, Q = CW >> 2, RP = kThreads / Q;
  const int chunks = a.C / CW, groups = a.C / a.G;
  const int pi = blockIdx.x % a.ps_apply, rest = blockIdx.x / a.ps_apply;
  const int ch = rest % chunks, n = rest / chunks;
  const int tid = threadIdx.x, col = tid % Q, prow = tid / Q;
  const int c = ch * CW + col * 4, j = (col * 4) / a.G;
  const size_t base = (size_t)n * HW * a.C;
  // merge the partials of each of the gpw groups (a fixed order per chunk
  // count): one thread per group when there are few, else L = kThreads / gpw
  // threads per group, thread l summing partials l, l + L, ..., then a tree
  // over l
  __shared__ float2 st[16];
  __shared__ double2 mrg[kThreads];
  const auto finish = [&](int jg, double S, double Qs) {
    const int g = ch * a.gpw + jg;
    const double cnt = (double)HW * a.G, m = S / cnt;
    const double var = std::max(Qs / cnt - m * m, 0.0);
    const float x0 = a.shift[(size_t)n * groups + g];
    st[jg] = make_float2((float)((double)x0 + m), (float)(1.0 / std::sqrt(var + (double)a.eps)));
  };
  if (a.ps_stats <= 8) {
    if (tid < a.gpw) {
      const double2* pp = a.part + ((size_t)n * groups + ch * a.gpw + tid) * a.ps_stats;
      double S = 0.0, Qs = 0.0;
      for (int k = 0; k < a.ps_stats; ++k) {
        S += pp[k].x;
        Qs += pp[k].y;
      }
      finish(tid, S, Qs);
    }
  } else {
    const int L = kThreads / a.gpw, jg = tid / L, l = tid - jg * L;
    const double2* pp = a.part + ((size_t)n * groups + ch * a.gpw + jg) * a.ps_stats;
    double S = 0.0, Qs = 0.0;
    for (int k = l; k < a.ps_stats; k += L) {
      S += pp[k].x;
      Qs += pp[k].y;
    }
    mrg[tid] = make_double2(S, Qs);
    __syncthreads();
    for (int h = L >> 1; h > 0; h >>= 1) {
      if (l < h) {
        mrg[tid].x += mrg[tid + h].x;
        mrg[tid].y += mrg[tid + h].y;
      }
      __syncthreads();
    }
    if (l == 0) finish(jg, mrg[tid].x, mrg[tid].y);
  }
  __syncthreads();
  const float2 ms = st[j];
  const f32x4 gm = *reinterpret_cast<const f32x4*>(a.gamma + c);
  const f32x4 bt = *reinterpret_cast<const f32x4*>(a.beta + c);
  auto f = [&](f32x4 v, size_t i) -> f32x4 {
    f32x4 r;
#pragma unroll
    for (int k = 0; k < 4; ++k) r[k] = (v[k] - ms.x) * ms.y * gm[k] + bt[k];
    if (a.res) r += *reinterpret_cast<const f32x4*>(a.res + i);
    if (a.relu) {
#pragma unroll
      for (int k = 0; k < 4; ++k) r[k] = fmaxf(r[k], 0.f);
    }
    return r;
  };
  if (a.mode == GN_PLAIN) {
    const int pc = (HW + a.ps_apply - 1) / a.ps_apply, p0 = pi * pc, p1 = min(HW, p0 + pc);
    for (int p = p0 + prow; p < p1; p += RP) {
      const size_t i = base + (size_t)p * a.C + c;
      *reinterpret_cast<f32x4*>(a.y + i) = f(*reinterpret_cast<const f32x4*>(a.x + i), i);
    }
  } else if (a.mode == GN_MAXPOOL) {
    const int HWp = a.Hp * a.Wp, pc = (HWp + a.ps_apply - 1) / a.ps_apply, p0 = pi * pc, p1 = min(HWp, p0 + pc);
    for (int p = p0 + prow; p < p1; p += RP) {
      const int oh = p / a.Wp, ow = p - oh * a.Wp;
      f32x4 m = {-INFINITY, -INFINITY, -INFINITY, -INFINITY};
      for (int u = 0; u < 3; ++u) {
        const int ih = oh * 2 - 1 + u;
        if (ih < 0 || ih >= a.H) continue;
        for (int v = 0; v < 3; ++v) {
          const int iw = ow * 2 - 1 + v;
          if (iw < 0 || iw >= a.W) continue;
          const size_t i = base + ((size_t)ih * a.W + iw) * a.C + c;
          const f32x4 r = f(*reinterpret_cast<const f32x4*>(a.x + i), i);
#pragma unroll
          for (int k = 0; k < 4; ++k) m[k] = fmaxf(m[k], r[k]);
        }
      }
      *reinterpret_cast<f32x4*>(a.y + (size_t)n * HWp * a.C + (size_t)p * a.C + c) = m;
    }
  } else {
    // global average pooling (one pixel chunk): column sums over the rows
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int p = prow; p < HW; p += RP) {
      const size_t i = base + (size_t)p * a.C + c;
      acc += f(*reinterpret_cast<const f32x4*>(a.x + i), i);
    }
    __shared__ f32x4 red[kThreads];
    red[tid] = acc;
    __syncthreads();
    for (int h = RP >> 1; h > 0; h >>= 1) {
      if (prow < h) red[tid] += red[tid + h * Q];
      __syncthreads();
    }
    if (prow == 0) {
      const f32x4 m = red[tid] / (float)HW;
      float* o = a.y + (size_t)n * a.out_stride + c;
      o[0] = m[0];
      o[1] = m[1];
      o[2] = m[2];
      o[3] = m[3];
    }
  }
}

// One kernel per GroupNorm: workgroup (image n, channel chunk of gpw
// groups) computes the statistics of its groups over the whole image, then
// applies them (the apply reads what the first sweep just touched, mostly
// from L2).  Thread t reads float4 column t % Q of pixel rows t / Q + i *
// RP, as the two-pass kernels do.
__global__ void __launch_bounds__(kThreads) gn_fused_kernel(const GnArgs a) {
  const int HW = a.H * a.W, CW = a.G * a.gpw, Q = CW >> 2, RP = kThreads / Q;
  const int chunks = a.C / CW;
  const int ch = blockIdx.x % chunks, n = blockIdx.x / chunks;
  const int tid = threadIdx.x, col = tid % Q, prow = tid / Q;
  const int c = ch * CW + col * 4, j = (col * 4) / a.G;
  const size_t base = (size_t)n * HW * a.C;
  const bool split = a.splits > 1;
  __shared__ float sx0[16];
  __shared__ float2 st[16];
  __shared__ double sd[kThreads], qd[kThreads];
  // the conv output at i: the sum of the split partials in split order (all
  // requested before the first is added), or x itself
  const auto value = [&](size_t i) -> f32x4 {
    if (!split) return *reinterpret_cast<const f32x4*>(a.x + i);
    f32x4 t[kMaxSplit];
#pragma unroll
    for (int z = 0; z < kMaxSplit; ++z)
      t[z] = z < a.splits ? *reinterpret_cast<const f32x4*>(a.ws + (long long)z * a.split_stride + i)
                          : f32x4{0.f, 0.f, 0.f, 0.f};
    f32x4 v = t[0];
#pragma unroll
    for (int z = 1; z < kMaxSplit; ++z)
      if (z < a.splits) v += t[z];
    return v;
  };
  // shift: the group's first element (pixel 0, first channel of the group;
  // a multiple of four channels, so the float4 load is aligned)
  const float x0 = value(base + ch * CW + j * a.G)[0];
  float s = 0.f, q = 0.f;
  const auto add = [&](f32x4 v, size_t i) {
    if (split) *reinterpret_cast<f32x4*>(a.x + i) = v;
    const f32x4 d = v - x0;
    s += (d[0] + d[1]) + (d[2] + d[3]);
    q += (d[0] * d[0] + d[1] * d[1]) + (d[2] * d[2] + d[3] * d[3]);
  };
  {
    constexpr int U = 4;  // pixel rows requested together
    int p = prow;
    for (; p + (U - 1) * RP < HW; p += U * RP) {
      f32x4 v[U];
#pragma unroll
      for (int u = 0; u < U; ++u) v[u] = value(base + (size_t)(p + u * RP) * a.C + c);
#pragma unroll
      for (int u = 0; u < U; ++u) add(v[u], base + (size_t)(p + u * RP) * a.C + c);
    }
    for (; p < HW; p += RP) add(value(base + (size_t)p * a.C + c), base + (size_t)p * a.C + c);
  }
  sd[tid] = s;
  qd[tid] = q;
  if (prow == 0 && col * 4 % a.G == 0) sx0[j] = x0;
  __syncthreads();
  for (int h = RP >> 1; h > 0; h >>= 1) {
    if (prow < h) {
      sd[tid] += sd[tid + h * Q];
      qd[tid] += qd[tid + h * Q];
    }
    __syncthreads();
  }
  if (tid < a.gpw) {
    const int cols = a.G >> 2;
    double S = 0.0, Qs = 0.0;
    for (int k = 0; k < cols; ++k) {
      S += sd[tid * cols + k];
      Qs += qd[tid * cols + k];
    }
    const double cnt = (double)HW * a.G, m = S / cnt;
    const double var = std::max(Qs / cnt - m * m, 0.0);
    st[tid] = make_float2((float)((double)sx0[tid] + m), (float)(1.0 / std::sqrt(var + (double)a.eps)));
  }
  __syncthreads();  // also orders the split sums stored above before the reads below
  const float2 ms = st[j];
  const f32x4 gm = *reinterpret_cast<const f32x4*>(a.gamma + c);
  const f32x4 bt = *reinterpret_cast<const f32x4*>(a.beta + c);
  auto f = [&](f32x4 v, size_t i) -> f32x4 {
    f32x4 r;
#pragma unroll
    for (int k = 0; k < 4; ++k) r[k] = (v[k] - ms.x) * ms.y * gm[k] + bt[k];
    if (a.res) r += *reinterpret_cast<const f32x4*>(a.res + i);
    if (a.relu) {
#pragma unroll
      for (int k = 0; k < 4; ++k) r[k] = fmaxf(r[k], 0.f);
    }
    return r;
  };
  if (a.mode == GN_PLAIN) {
    for (int p = prow; p < HW; p += RP) {
      const size_t i = base + (size_t)p * a.C + c;
      *reinterpret_cast<f32x4*>(a.y + i) = f(*reinterpret_cast<const f32x4*>(a.x + i), i);
    }
  } else if (a.mode == GN_MAXPOOL) {
    const int HWp = a.Hp * a.Wp;
    for (int p = prow; p < HWp; p += RP) {
      const int oh = p / a.Wp, ow = p - oh * a.Wp;
      f32x4 m = {-INFINITY, -INFINITY, -INFINITY, -INFINITY};
      for (int u = 0; u < 3; ++u) {
        const int ih = oh * 2 - 1 + u;
        if (ih < 0 || ih >= a.H) continue;
        for (int v = 0; v < 3; ++v) {
          const int iw = ow * 2 - 1 + v;
          if (iw < 0 || iw >= a.W) continue;
          const size_t i = base + ((size_t)ih * a.W + iw) * a.C + c;
          const f32x4 r = f(*reinterpret_cast<const f32x4*>(a.x + i), i);
#pragma unroll
          for (int k = 0; k < 4; ++k) m[k] = fmaxf(m[k], r[k]);
        }
      }
      *reinterpret_cast<f32x4*>(a.y + (size_t)n * HWp * a.C + (size_t)p * a.C + c) = m;
    }
  } else {
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int p = prow; p < HW; p += RP) {
      const size_t i = base + (size_t)p * a.C + c;
      acc += f(*reinterpret_cast<const f32x4*>(a.x + i), i);
    }
    __shared__ f32x4 red[kThreads];
    red[tid] = acc;
    __syncthreads();
    for (int h = RP >> 1; h > 0; h >>= 1) {
      if (prow < h) red[tid] += red[tid + h * Q];
      __syncthreads();
    }
    if (prow == 0) {
      const f32x4 m = red[tid] / (float)HW;
      float* o = a.y + (size_t)n * a.out_stride + c;
      o[0] = m[0];
      o[1] = m[1];
      o[2] = m[2];
      o[3] = m[3];
    }
  }
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

unsigned grid_for(long long total) { return (unsigned)std::min<long long>((total + 255) / 256, 16384); }

struct ConvLayer {
  int cin, cout, k, stride, pad, K, Kp;
  void* w = nullptr;             // packed operand weights
  const float* gamma = nullptr;  // GroupNorm affine (device, inside the raw copy)
  const float* beta = nullptr;
};

}  // namespace

struct evo_encoder {
  evo_encoder_desc desc{};
  int device = 0;
  int bf = 1;
  float* d_raw = nullptr;        // fp32 parameter copy (GroupNorm affine, packing source)
  std::vector<ConvLayer> convs;  // stem, then per block a, b[, d]
  float* buf[4] = {nullptr, nullptr, nullptr, nullptr};
  size_t buf_floats = 0;
  float* zeros = nullptr;        // 256 zero bytes: the convolutions' loads outside their inputs
  float* ws = nullptr;           // split-K partials, kWsFloats
  double2* part = nullptr;       // GroupNorm partial statistics
  size_t part_cap = 0;
  float* shift = nullptr;        // GroupNorm shifts [image][group]
  size_t shift_cap = 0;
  uint64_t flops_per_image = 0;
  hipEvent_t ev_done = nullptr;  // recorded after the last encode's launches
  bool launched = false;
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
  if (d->gn_group != 4 && d->gn_group != 8 && d->gn_group != 16 && d->gn_group != 32 && d->gn_group != 64)
    return fail(EVO_E_UNSUPPORTED, "gn_group must be 4, 8, 16, 32 or 64");
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
inline int cdiv(long long a, long long b) { return (int)((a + b - 1) / b); }

// Launch shape of one convolution: 64 x 64 tiles (four workgroups fit a CU;
// 128 x 128 and 128 x 64 tiles, two per CU, measured 8% slower over the
// 512-frame encode), K split where there are few tiles.
constexpr int kBM = 64, kBN = 64;
struct ConvPlan {
  int mt, nt, splits, spp;
};

ConvPlan plan_conv(int M, int Cout, int steps) {
  ConvPlan pl{};
  pl.mt = cdiv(M, kBM);
  pl.nt = cdiv(Cout, kBN);
  const int tiles = pl.mt * pl.nt;
  int splits = 1;
  if (tiles < kTargetWG) splits = std::min({cdiv(kTargetWG, tiles), std::max(1, steps / 2), kMaxSplit});
  pl.spp = cdiv(steps, splits);
  pl.splits = cdiv(steps, pl.spp);  // every split has at least one step
  return pl;
}

// The conv result lands in `y` (one split) or as partials in the encoder's
// workspace; `*gn` gets the source fields of the GroupNorm that follows.
hipError_t launch_conv(const evo_encoder* e, const ConvLayer& L, const float* x, int N, int H, int W, float* y,
                       int* Ho, int* Wo, GnArgs* gn, hipStream_t st) {
  ConvArgs a;
  a.x = x;
  a.w = L.w;
  a.H = H;
  a.W = W;
  a.Cin = L.cin;
  a.Ho = *Ho = out_size(H, L.k, L.stride, L.pad);
  a.Wo = *Wo = out_size(W, L.k, L.stride, L.pad);
  a.Cout = L.cout;
  a.kw = L.k;
  a.stride = L.stride;
  a.pad = L.pad;
  a.K = L.K;
  a.Kp = L.Kp;
  a.M = N * a.Ho * a.Wo;
  const int KS = e->bf ? ConvStep<__bf16>::KS : ConvStep<float>::KS;
  // K splits of the max_batch plan; tiles for this call's pixels
  ConvPlan pl = plan_conv(e->desc.max_batch * a.Ho * a.Wo, L.cout, L.Kp / KS);
  pl.mt = cdiv(a.M, kBM);
  a.mt = pl.mt;
  a.nt = pl.nt;
  a.splits = pl.splits;
  a.spp = pl.spp;
  a.split_stride = (long long)a.M * L.cout;
  // splits * tiles * 64 * 64 bounds the partials, below the workspace by construction
  if (pl.splits > 1 && (long long)pl.splits * a.split_stride > kWsFloats) return hipErrorInvalidValue;
  a.y = pl.splits > 1 ? e->ws : y;
  a.zeros = e->zeros;
  gn->ws = e->ws;
  gn->splits = pl.splits;
  gn->split_stride = a.split_stride;
  gn->x = y;
  const unsigned grid = (unsigned)((long long)pl.mt * pl.nt * pl.splits);
  if (e->bf) hipLaunchKernelGGL((conv_kernel<__bf16, kBM, kBN>), dim3(grid), dim3(kThreads), 0, st, a);
  else hipLaunchKernelGGL((conv_kernel<float, kBM, kBN>), dim3(grid), dim3(kThreads), 0, st, a);
  return hipGetLastError();
}

// One GroupNorm pass (gn_fused_kernel) or two (statistics over pixel
// chunks, then apply).  Chosen from the encoder's max_batch and the map
// size, never from a call's batch, so an image's statistics are summed in
// the same order at every batch size.
bool fused_gn(const evo_encoder* e, int HW, int chunks) {
  return HW <= kFusedPixels || ((long long)e->desc.max_batch * chunks >= kFusedWG && HW <= kFusedPixelsWide);
}

// GroupNorm of layer L's conv output (g.ws / splits / x set by launch_conv).
hipError_t launch_gn(const evo_encoder* e, const ConvLayer& L, GnArgs g, int N, int H, int W, const float* res,
                     int relu, int mode, float* y, int out_stride, hipStream_t st) {
  const int C = L.cout, G = e->desc.gn_group, groups = C / G;
  int gpw = 1;  // groups per workgroup: up to 64 channels, a power of two dividing the group count
  while (gpw * 2 * G <= 64 && groups % (gpw * 2) == 0) gpw *= 2;
  int chunks = groups / gpw;
  const int HW = H * W;
  const bool fused = fused_gn(e, HW, chunks);
  if (fused && (long long)e->desc.max_batch * chunks < kFusedWG) {
    gpw = 1;  // few images: one group per workgroup, for more workgroups
    chunks = groups;
  }
  const int base = N * chunks;
  // statistics chunks of the max_batch plan (see kGnTarget)
  const int ps = std::max(1, std::min(cdiv(kGnTarget, e->desc.max_batch * chunks), cdiv(HW, 16)));
  if ((size_t)N * groups * ps > e->part_cap) return hipErrorInvalidValue;  // sized at creation
  g.gamma = L.gamma;
  g.beta = L.beta;
  g.res = res;
  g.y = y;
  g.part = e->part;
  g.shift = e->shift;
  g.relu = relu;
  g.mode = mode;
  g.H = H;
  g.W = W;
  g.C = C;
  g.G = G;
  g.gpw = gpw;
  g.ps_stats = ps;
  g.Hp = mode == GN_MAXPOOL ? out_size(H, 3, 2, 1) : 0;
  g.Wp = mode == GN_MAXPOOL ? out_size(W, 3, 2, 1) : 0;
  g.out_stride = out_stride;
  g.eps = 1e-5f;
  const int out_px = mode == GN_MAXPOOL ? g.Hp * g.Wp : HW;
  g.ps_apply = mode == GN_AVGPOOL ? 1 : std::max(1, std::min(cdiv(kGnTarget, base), cdiv(out_px, 16)));
  if (fused) {
    hipLaunchKernelGGL(gn_fused_kernel, dim3((unsigned)base), dim3(kThreads), 0, st, g);
  } else {
    hipLaunchKernelGGL(gn_stats_kernel, dim3((unsigned)(base * ps)), dim3(kThreads), 0, st, g);
    hipLaunchKernelGGL(gn_apply_kernel, dim3((unsigned)(base * g.ps_apply)), dim3(kThreads), 0, st, g);
  }
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
  if ((int64_t)n_floats != need)
    return fail(EVO_E_INVALID, "n_floats is %zu, this encoder needs %lld", n_floats, (long long)need);
  evo_encoder* e = new (std::nothrow) evo_encoder();
  if (!e) return fail(EVO_E_NOMEM, "host allocation failed");
  const auto body = [&]() -> int {
    e->desc = *desc;
    e->bf = desc->dtype == EVO_BF16;
    if (hipGetDevice(&e->device) != hipSuccess) return fail(EVO_E_HIP, "no current HIP device");
#define ENC_TRY(expr)                                                                          \
  do {                                                                                         \
    hipError_t e_ = (expr);                                                                    \
    if (e_ != hipSuccess)                                                                      \
      return fail(e_ == hipErrorOutOfMemory ? EVO_E_NOMEM : EVO_E_HIP, "%s failed: %s", #expr, \
                  hipGetErrorString(e_));                                                      \
  } while (0)
    // activation sizes and FLOPs: walk the network once
    size_t maxact = 0, maxpart = 0;  // per image: activation floats, GroupNorm partials
    int maxgroups = 0;
    uint64_t flops = 0;
    {
      int h = out_size(desc->height, 7, 2, 3), w = out_size(desc->width, 7, 2, 3);
      maxact = std::max(maxact, (size_t)h * w * desc->stem_ch);
      maxgroups = desc->stem_ch / desc->gn_group;
      maxpart = (size_t)maxgroups * cdiv((long long)h * w, 16);
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
          maxgroups = std::max(maxgroups, c / desc->gn_group);
          maxpart = std::max(maxpart, (size_t)(c / desc->gn_group) * cdiv((long long)ho * wo, 16));
          flops += 2ull * ho * wo * c * 9 * cin + 2ull * ho * wo * c * 9 * c;
          if (stride != 1 || cin != c) flops += 2ull * ho * wo * c * cin;
          h = ho;
          w = wo;
          cin = c;
        }
    }
    if (maxact * desc->max_batch >= (size_t(1) << 31))
      return fail(EVO_E_UNSUPPORTED, "activations of max_batch images exceed 2^31 floats");
    e->flops_per_image = flops;
    e->buf_floats = maxact * desc->max_batch;
    e->part_cap = (size_t)desc->max_batch * maxpart;
    e->shift_cap = (size_t)desc->max_batch * maxgroups;
    ENC_TRY(hipMalloc(&e->d_raw, n_floats * sizeof(float)));
    ENC_TRY(hipMemcpy(e->d_raw, host_weights, n_floats * sizeof(float), hipMemcpyHostToDevice));
    e->convs = enc_layers(desc);
    const int KS = e->bf ? ConvStep<__bf16>::KS : ConvStep<float>::KS;
    size_t off = 0;
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
    }
    for (int i = 0; i < 4; ++i) ENC_TRY(hipMalloc(&e->buf[i], e->buf_floats * sizeof(float)));
    ENC_TRY(hipMalloc(&e->ws, (size_t)kWsFloats * sizeof(float)));
    ENC_TRY(hipMalloc(&e->zeros, 256));
    ENC_TRY(hipMemset(e->zeros, 0, 256));
    ENC_TRY(hipMalloc(&e->part, e->part_cap * sizeof(double2)));
    ENC_TRY(hipMalloc(&e->shift, e->shift_cap * sizeof(float)));
    ENC_TRY(hipEventCreateWithFlags(&e->ev_done, hipEventDisableTiming));
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
  // the convolutions read whole input pixels with 16-byte loads where the channel count allows
  if (reinterpret_cast<uintptr_t>(images) % 16)
    return fail(EVO_E_INVALID, "images must be 16-byte aligned");
  const int C_out = d.widths[d.n_stages - 1];
  if (out_stride < C_out) return fail(EVO_E_INVALID, "out_stride %d < feature size %d", out_stride, C_out);
  DeviceGuard guard(e->device);
  hipStream_t st = (hipStream_t)hip_stream;
  float *X = e->buf[0], *Y = e->buf[1], *Z = e->buf[2], *R = e->buf[3];
  int H = d.height, W = d.width, Ho, Wo;
  size_t li = 0;
  GnArgs g{};
#define ENC_HIP(expr)                                                                            \
  do {                                                                                           \
    hipError_t e_ = (expr);                                                                      \
    if (e_ != hipSuccess) return fail(EVO_E_HIP, "%s failed: %s", #expr, hipGetErrorString(e_)); \
  } while (0)
  // stem: conv 7x7/2, then GroupNorm + ReLU + max pool 3x3/2 in one apply pass
  {
    const ConvLayer& L = e->convs[li++];
    ENC_HIP(launch_conv(e, L, images, batch, H, W, Y, &Ho, &Wo, &g, st));
    ENC_HIP(launch_gn(e, L, g, batch, Ho, Wo, nullptr, 1, GN_MAXPOOL, X, 0, st));
    H = out_size(Ho, 3, 2, 1);
    W = out_size(Wo, 3, 2, 1);
  }
  int cin = d.stem_ch;
  for (int s = 0; s < d.n_stages; ++s)
    for (int b = 0; b < d.blocks[s]; ++b) {
      const int c = d.widths[s];
      const bool last = s == d.n_stages - 1 && b == d.blocks[s] - 1;
      const ConvLayer& La = e->convs[li++];
      const ConvLayer& Lb = e->convs[li++];
      const bool proj = La.stride != 1 || cin != c;
      int H2, W2, H3, W3;
      ENC_HIP(launch_conv(e, La, X, batch, H, W, Y, &H2, &W2, &g, st));
      ENC_HIP(launch_gn(e, La, g, batch, H2, W2, nullptr, 1, GN_PLAIN, Y, 0, st));
      const float* shortcut = X;
      if (proj) {  // before conv b: each conv's partials are consumed before the next conv runs
        const ConvLayer& Ld = e->convs[li++];
        int Hd, Wd;
        ENC_HIP(launch_conv(e, Ld, X, batch, H, W, R, &Hd, &Wd, &g, st));
        ENC_HIP(launch_gn(e, Ld, g, batch, Hd, Wd, nullptr, 0, GN_PLAIN, R, 0, st));
        shortcut = R;
      }
      ENC_HIP(launch_conv(e, Lb, Y, batch, H2, W2, Z, &H3, &W3, &g, st));
      // block output = ReLU(GN(conv b) + shortcut): into Y, or averaged into the features
      if (last) ENC_HIP(launch_gn(e, Lb, g, batch, H3, W3, shortcut, 1, GN_AVGPOOL, features_out, out_stride, st));
      else ENC_HIP(launch_gn(e, Lb, g, batch, H3, W3, shortcut, 1, GN_PLAIN, Y, 0, st));
      std::swap(X, Y);
      H = H3;
      W = W3;
      cin = c;
    }
  ENC_HIP(hipEventRecord(e->ev_done, st));
  e->launched = true;
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
  // the encoder's own launches end before its buffers are freed (no
  // device-wide wait: other work on the device is not this encoder's)
  if (e->launched && e->ev_done) (void)hipEventSynchronize(e->ev_done);
  for (ConvLayer& L : e->convs) (void)hipFree(L.w);
  for (int i = 0; i < 4; ++i) (void)hipFree(e->buf[i]);
  (void)hipFree(e->ws);
  (void)hipFree(e->zeros);
  (void)hipFree(e->part);
  (void)hipFree(e->shift);
  (void)hipFree(e->d_raw);
  if (e->ev_done) (void)hipEventDestroy(e->ev_done);
  delete e;
}

}  // extern "C"
