// HIP kernels (gfx950) of the schedule-driven cached denoising loop.
//
// Design: one workgroup owns a tile of whole samples (rows = samples x
// horizon tokens) for the entire T-step reverse process.  Samples never
// interact, so a tile needs no communication with other workgroups: the
// whole query is one launch with no grid-wide synchronisation.
//
//  * The residual stream h of the tile lives in registers, laid out as the
//    accumulator fragments of the 16x16 MFMA tiles (each wave owns a fixed
//    set of 16-column blocks of d).
//  * Cacheable units (Sec. 3.1: SA, CA, FFN residual branches) are evaluated
//    only where the schedule says so (Eq. 1); their residual is then
//    stored in a per-tile cache in HBM only if a later step reuses it.
//    Elsewhere the unit adds the cached residual of its most recent refresh.
//  * Every unit is "LayerNorm -> chunked stage-1 product -> per-chunk
//    transform (attention per head group, or GELU) -> stage-2 product
//    accumulated into the unit's residual".  Activations stay in LDS;
//    projection weights are streamed from L2/HBM as pre-packed 1 KiB MFMA
//    fragments (16 output columns x 32 bf16 / 16 fp32 of K, 16 bytes per
//    lane), so every weight load is one coalesced 16-byte load per lane.
//  * The head (final LayerNorm + linear) and the DDPM update are fused at
//    the end of every step.
#include "evo_kernels.hpp"

#include <cmath>
#include <type_traits>

namespace evo {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

enum : uint8_t { C_EVAL = 1, C_STORE = 2, C_REUSE = 4, C_MERGED = 8 };

// float -> bfloat16 bits, round to nearest even (finite inputs)
__device__ __forceinline__ uint32_t bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}

// Operand traits of the two matmul precisions.  A fragment is 16 bytes per
// lane: 8 bf16 (K = 32 per fragment, one 16x16x32 MFMA) or 4 fp32 (K = 16
// per fragment, four 16x16x4 MFMAs).
template <class AT> struct Op;

template <> struct Op<__bf16> {
  static constexpr int KF = 32, VE = 8, PAD = 8;
  __device__ static __forceinline__ void store(__bf16* buf, int ld, int row, int k, float v) {
    reinterpret_cast<uint16_t*>(buf)[row * ld + k] = (uint16_t)bf16_rne(v);
  }
  __device__ static __forceinline__ void mma(f32x4& acc, uint4 a, uint4 b) {
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                  __builtin_bit_cast(bf16x8_t, b), acc, 0, 0, 0);
  }
};

template <> struct Op<float> {
  static constexpr int KF = 16, VE = 4, PAD = 4;
  // Within each 16-wide k block, element k is stored at 4*(k%4) + (k/4)%4 so
  // that the four values one lane feeds to four 16x16x4 MFMAs are adjacent.
  __device__ static __forceinline__ int pcol(int k) { return (k & ~15) | ((k & 3) << 2) | ((k >> 2) & 3); }
  __device__ static __forceinline__ void store(float* buf, int ld, int row, int k, float v) {
    buf[row * ld + pcol(k)] = v;
  }
  __device__ static __forceinline__ void mma(f32x4& acc, uint4 a, uint4 b) {
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), acc, 0, 0, 0);
  }
};

// acc[m][rb] += A[rb*16 .. +16][k-range] x W[col block gcb(m)][k-range]^T
// A: LDS operand, row stride lda elements, already offset to the k-range
// start.  W: packed fragments of a matrix with KBT fragments per column
// block; kf0 is the first fragment of the k-range, NKF its length.  The
// next k step's weight fragments are loaded before the current MFMAs.
template <class AT, int RBk, int MPW, int NKF, class GCB>
__device__ __forceinline__ void gemm_acc(f32x4 (&acc)[MPW][RBk], const AT* A, int lda, const uint4* W,
                                         int KBT, int kf0, GCB gcb, int lane) {
  using O = Op<AT>;
  const int lc = lane & 15, lq = lane >> 4;
  const uint4* wp[MPW];
#pragma unroll
  for (int m = 0; m < MPW; ++m) wp[m] = W + ((size_t)gcb(m) * KBT + kf0) * 64 + lane;
  uint4 bc[MPW], bn[MPW];
#pragma unroll
  for (int m = 0; m < MPW; ++m) bc[m] = wp[m][0];
#pragma unroll
  for (int kf = 0; kf < NKF; ++kf) {
    if (kf + 1 < NKF) {
#pragma unroll
      for (int m = 0; m < MPW; ++m) bn[m] = wp[m][(kf + 1) * 64];
    }
    uint4 a[RBk];
#pragma unroll
    for (int rb = 0; rb < RBk; ++rb)
      a[rb] = *reinterpret_cast<const uint4*>(A + (rb * 16 + lc) * lda + kf * O::KF + lq * O::VE);
#pragma unroll
    for (int m = 0; m < MPW; ++m)
#pragma unroll
      for (int rb = 0; rb < RBk; ++rb) O::mma(acc[m][rb], a[rb], bc[m]);
    if (kf + 1 < NKF) {
#pragma unroll
      for (int m = 0; m < MPW; ++m) bc[m] = bn[m];
    }
  }
}

__device__ __forceinline__ float gelu_erf(float v) { return 0.5f * v * (1.0f + erff(v * 0.70710678118654752f)); }

template <int D, int DH, int HZ, int SPT, int DFF, int NW, int HG, int FC, int SMAX>
struct Cfg {
  static constexpr int NWV = NW;
  static constexpr int NT = NW * 64;
  static constexpr int R = SPT * HZ;
  static constexpr int RB = R / 16;
  static constexpr int NH = D / DH;
  static constexpr int CB = D / 16;
  static constexpr int CBW = CB / NW;
  static constexpr int GW = HG * DH;
  static constexpr int LDY = 3 * GW + 4;
  static constexpr int ZW = GW > FC ? GW : FC;
  static constexpr int AMAX = 16;
  static constexpr int KOBS = 64;
  static constexpr int PW = HZ > SMAX ? HZ : SMAX;
};

// Per-lane rows of the fragment layout: row = rb*16 + lq*4 + i.
// LayerNorm statistics of the tile rows from the register-resident stream.
template <class C>
__device__ __forceinline__ void row_stats(const f32x4 (&h)[C::CBW][C::RB], float (*red)[C::NWV][C::R],
                                          float (&mu)[C::RB][4], float (&rs)[C::RB][4], int w, int lc,
                                          int lq) {
  constexpr int D = C::CB * 16;
  float s[C::RB][4];
#pragma unroll
  for (int rb = 0; rb < C::RB; ++rb)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float v = 0.f;
#pragma unroll
      for (int c = 0; c < C::CBW; ++c) v += h[c][rb][i];
#pragma unroll
      for (int off = 1; off < 16; off <<= 1) v += __shfl_xor(v, off);
      s[rb][i] = v;
    }
  if (lc == 0) {
#pragma unroll
    for (int rb = 0; rb < C::RB; ++rb)
#pragma unroll
      for (int i = 0; i < 4; ++i) red[0][w][rb * 16 + lq * 4 + i] = s[rb][i];
  }
  __syncthreads();
#pragma unroll
  for (int rb = 0; rb < C::RB; ++rb)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float v = 0.f;
#pragma unroll
      for (int ww = 0; ww < C::NWV; ++ww) v += red[0][ww][rb * 16 + lq * 4 + i];
      mu[rb][i] = v * (1.0f / D);
      float q = 0.f;
#pragma unroll
      for (int c = 0; c < C::CBW; ++c) {
        const float e = h[c][rb][i] - mu[rb][i];
        q += e * e;
      }
#pragma unroll
      for (int off = 1; off < 16; off <<= 1) q += __shfl_xor(q, off);
      s[rb][i] = q;
    }
  if (lc == 0) {
#pragma unroll
    for (int rb = 0; rb < C::RB; ++rb)
#pragma unroll
      for (int i = 0; i < 4; ++i) red[1][w][rb * 16 + lq * 4 + i] = s[rb][i];
  }
  __syncthreads();
#pragma unroll
  for (int rb = 0; rb < C::RB; ++rb)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float v = 0.f;
#pragma unroll
      for (int ww = 0; ww < C::NWV; ++ww) v += red[1][ww][rb * 16 + lq * 4 + i];
      rs[rb][i] = 1.0f / sqrtf(v * (1.0f / D) + 1e-5f);
    }
}

template <class AT, int D, int DH, int HZ, int SPT, int DFF, int NW, int HG, int FC, int SMAX>
__global__ void __launch_bounds__(NW * 64) denoise_kernel(const KParams p) {
  using O = Op<AT>;
  using C = Cfg<D, DH, HZ, SPT, DFF, NW, HG, FC, SMAX>;
  constexpr int NT = C::NT, R = C::R, RB = C::RB, NH = C::NH, CB = C::CB, CBW = C::CBW, GW = C::GW;
  constexpr int LDA = D + O::PAD, LDY = C::LDY, LDZ = C::ZW + O::PAD, AMAX = C::AMAX;
  constexpr int KOBS = C::KOBS, LDO = KOBS + O::PAD;
  static_assert(R % 16 == 0 && CB % NW == 0 && NH % HG == 0 && DFF % FC == 0, "tile shape");
  static_assert((3 * GW / 16) % NW == 0 && (GW / 16) % NW == 0 && (FC / 16) % NW == 0, "block split");
  static_assert(HZ % 4 == 0 && (HZ & (HZ - 1)) == 0 && HZ <= 64, "horizon must be a power of two in [4, 64]");
  static_assert(NW * R * AMAX <= R * LDY, "head partials must fit the stage-1 buffer");
  static_assert(16 * LDO * (int)sizeof(AT) <= R * LDY * 4, "observation operand must fit");

  __shared__ __attribute__((aligned(16))) AT xa[R * LDA];
  __shared__ __attribute__((aligned(16))) float ybuf[R * LDY];
  __shared__ __attribute__((aligned(16))) AT zbuf[R * LDZ];
  __shared__ float pbuf[SPT * HG * HZ * C::PW];
  __shared__ __attribute__((aligned(16))) float kvbuf[SPT * SMAX * 2 * GW];
  __shared__ float red[2][NW][R];
  __shared__ float xs[R * AMAX];
  __shared__ int smp[SPT], slt[SPT];

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, lc = lane & 15, lq = lane >> 4;
  const int tile = blockIdx.x;
  const int L = p.L, A = p.A, T = p.T, U = 3 * L, nobs = p.n_obs, S = 1 + nobs;
  const float* raw = p.raw;
  constexpr float kScale = (DH == 64) ? 0.125f : (DH == 32 ? 0.17677669529663688f : 0.0f);
  static_assert(DH == 64 || DH == 32, "head dim");

  if (tid < SPT) {
    smp[tid] = p.tile_sample[tile * SPT + tid];
    slt[tid] = p.tile_slot[tile * SPT + tid];
  }
  __syncthreads();

  // initial sample x_T
  for (int it = tid; it < R * A; it += NT) {
    const int row = it / A, a = it % A, j = row / HZ, s = smp[j];
    xs[row * AMAX + a] = s >= 0 ? p.noise[((size_t)s * HZ + (row % HZ)) * A + a] : 0.f;
  }

  // ---- per query: observation tokens and their keys/values in every layer
  {
    constexpr int MPWO = CB / NW;
    f32x4 acc[MPWO][1];
#pragma unroll
    for (int m = 0; m < MPWO; ++m) acc[m][0] = f32x4{0.f, 0.f, 0.f, 0.f};
    AT* ob = reinterpret_cast<AT*>(ybuf);
    const int nch = p.obs_pad / KOBS;
    for (int c = 0; c < nch; ++c) {
      __syncthreads();
      for (int it = tid; it < 16 * KOBS; it += NT) {
        const int row = it / KOBS, k = it % KOBS, kk = c * KOBS + k;
        float v = 0.f;
        if (row < SPT * nobs) {
          const int j = row / nobs, o = row % nobs;
          if (smp[j] >= 0 && kk < p.obs_dim) v = p.obs[((size_t)smp[j] * nobs + o) * p.obs_dim + kk];
        }
        O::store(ob, LDO, row, k, v);
      }
      __syncthreads();
      gemm_acc<AT, 1, MPWO, KOBS / O::KF>(acc, ob, LDO, p.pk + p.pk_obs, p.obs_pad / O::KF,
                                           c * (KOBS / O::KF), [&](int m) { return w + NW * m; }, lane);
    }
    // memory-token operand rows (row = slot*n_obs + token) in xa
#pragma unroll
    for (int m = 0; m < MPWO; ++m) {
      const int gcol = (w + NW * m) * 16 + lc;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = lq * 4 + i;
        float v = 0.f;
        if (row < SPT * nobs) {
          const int j = row / nobs, o = row % nobs;
          if (smp[j] >= 0) v = acc[m][0][i] + raw[p.b_obs + gcol] + raw[p.P_mem + (size_t)(1 + o) * D + gcol];
        }
        O::store(xa, LDA, row, gcol, v);
      }
    }
    __syncthreads();
    constexpr int MPWK = 2 * CB / NW;
    for (int l = 0; l < L; ++l) {
      f32x4 kv[MPWK][1];
#pragma unroll
      for (int m = 0; m < MPWK; ++m) kv[m][0] = f32x4{0.f, 0.f, 0.f, 0.f};
      gemm_acc<AT, 1, MPWK, D / O::KF>(kv, xa, LDA, p.pk + p.poff[l].kv, D / O::KF, 0,
                                        [&](int m) { return w + NW * m; }, lane);
      const uint32_t bkv = p.loff[l].b_kv;
#pragma unroll
      for (int m = 0; m < MPWK; ++m) {
        const int gcol = (w + NW * m) * 16 + lc;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int row = lq * 4 + i;
          if (row < SPT * nobs) {
            const int j = row / nobs, o = row % nobs;
            if (smp[j] >= 0)
              p.okv[(((size_t)smp[j] * L + l) * nobs + o) * (2 * D) + gcol] = kv[m][0][i] + raw[bkv + gcol];
          }
        }
      }
    }
    __syncthreads();
  }

  const uint8_t* codes[SPT];
#pragma unroll
  for (int j = 0; j < SPT; ++j) codes[j] = p.codes + (size_t)slt[j] * U * T;
  float* cbase = p.cache + (size_t)tile * U * (R * D);

  f32x4 h[CBW][RB], mac[CBW][RB];
#pragma unroll
  for (int c = 0; c < CBW; ++c)
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) mac[c][rb] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int t = 0; t < T; ++t) {
    const int k = T - 1 - t;
    // noise added by this step's update (prefetched)
    constexpr int ZPT = (R * AMAX + NT - 1) / NT;
    float zpre[ZPT];
#pragma unroll
    for (int q = 0; q < ZPT; ++q) {
      const int it = tid + q * NT;
      zpre[q] = 0.f;
      if (k > 0 && it < R * A) {
        const int row = it / A, a = it % A, s = smp[row / HZ];
        if (s >= 0) zpre[q] = p.noise[(((size_t)(t + 1) * p.batch + s) * HZ + (row % HZ)) * A + a];
      }
    }
    // embedding of the current sample: h = x W_in^T + b_in + P_act
#pragma unroll
    for (int c = 0; c < CBW; ++c) {
      const int col = (w * CBW + c) * 16 + lc;
      const float bi = raw[p.b_in + col];
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int row = rb * 16 + lq * 4 + i;
          float v = 0.f;
          for (int a = 0; a < A; ++a) v += xs[row * AMAX + a] * raw[p.W_in + (size_t)col * A + a];
          h[c][rb][i] = v + bi + raw[p.P_act + (size_t)(row % HZ) * D + col];
        }
    }

    for (int b = 0; b < U; ++b) {
      const int l = b / 3, u = b - 3 * (b / 3);
      uint8_t code[SPT];
      bool ev = false;
#pragma unroll
      for (int j = 0; j < SPT; ++j) {
        code[j] = smp[j] >= 0 ? codes[j][(size_t)b * T + t] : (uint8_t)0;
        ev |= (code[j] & C_EVAL) != 0;
      }
      f32x4 r[CBW][RB];
      if (ev) {
        const LayerOff lo = p.loff[l];
        const PackOff po = p.poff[l];
        float mu[RB][4], rs[RB][4];
        row_stats<C>(h, red, mu, rs, w, lc, lq);
        const uint32_t gofs = u == 0 ? lo.ln1_g : (u == 1 ? lo.ln2_g : lo.ln3_g);
        const uint32_t bofs = u == 0 ? lo.ln1_b : (u == 1 ? lo.ln2_b : lo.ln3_b);
#pragma unroll
        for (int c = 0; c < CBW; ++c) {
          const int col = (w * CBW + c) * 16 + lc;
          const float g = raw[gofs + col], bb = raw[bofs + col];
#pragma unroll
          for (int rb = 0; rb < RB; ++rb)
#pragma unroll
            for (int i = 0; i < 4; ++i)
              O::store(xa, LDA, rb * 16 + lq * 4 + i, col, (h[c][rb][i] - mu[rb][i]) * rs[rb][i] * g + bb);
        }
#pragma unroll
        for (int c = 0; c < CBW; ++c)
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) r[c][rb] = f32x4{0.f, 0.f, 0.f, 0.f};
        __syncthreads();
        const auto own = [&](int m) { return w * CBW + m; };

        if (u == 0) {
          // ---------------- self-attention unit (causal over the action tokens)
          for (int g = 0; g < NH / HG; ++g) {
            constexpr int MPW1 = (3 * GW / 16) / NW;
            const auto gcb = [&](int m) {
              const int iloc = w + NW * m, part = iloc / (GW / 16), within = iloc % (GW / 16);
              return part * CB + g * (GW / 16) + within;
            };
            f32x4 y[MPW1][RB];
#pragma unroll
            for (int m = 0; m < MPW1; ++m)
#pragma unroll
              for (int rb = 0; rb < RB; ++rb) y[m][rb] = f32x4{0.f, 0.f, 0.f, 0.f};
            gemm_acc<AT, RB, MPW1, D / O::KF>(y, xa, LDA, p.pk + po.qkv, D / O::KF, 0, gcb, lane);
#pragma unroll
            for (int m = 0; m < MPW1; ++m) {
              const int loc = (w + NW * m) * 16 + lc, gcol = gcb(m) * 16 + lc;
              const float bq = raw[lo.b_qkv + gcol];
#pragma unroll
              for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                for (int i = 0; i < 4; ++i) ybuf[(rb * 16 + lq * 4 + i) * LDY + loc] = y[m][rb][i] + bq;
            }
            __syncthreads();
            // scores and softmax: one lane per (sample, head, query, key)
            constexpr int NIT = SPT * HG * HZ * HZ;
            for (int base = 0; base < NIT; base += NT) {
              const int it = base + tid;
              const bool valid = it < NIT;
              const int kk = it % HZ, qi = (it / HZ) % HZ, hh = (it / (HZ * HZ)) % HG, j = it / (HZ * HZ * HG);
              const bool live = valid && kk <= qi;
              float s = -INFINITY;
              if (live) {
                const float* qp = ybuf + (j * HZ + qi) * LDY + hh * DH;
                const float* kp = ybuf + (j * HZ + kk) * LDY + GW + hh * DH;
                float acc = 0.f;
#pragma unroll
                for (int cc = 0; cc < DH; cc += 4) {
                  const float4 a4 = *reinterpret_cast<const float4*>(qp + cc);
                  const float4 b4 = *reinterpret_cast<const float4*>(kp + cc);
                  acc += a4.x * b4.x + a4.y * b4.y + a4.z * b4.z + a4.w * b4.w;
                }
                s = acc * kScale;
              }
              float mx = s;
#pragma unroll
              for (int off = HZ / 2; off >= 1; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
              const float e = live ? expf(s - mx) : 0.f;
              float sum = e;
#pragma unroll
              for (int off = HZ / 2; off >= 1; off >>= 1) sum += __shfl_xor(sum, off);
              if (valid) pbuf[it] = e / sum;
            }
            __syncthreads();
            constexpr int NIT2 = SPT * HG * HZ * DH;
            for (int it = tid; it < NIT2; it += NT) {
              const int cc = it % DH, qi = (it / DH) % HZ, hh = (it / (DH * HZ)) % HG, j = it / (DH * HZ * HG);
              const float* pr = pbuf + ((j * HG + hh) * HZ + qi) * HZ;
              const float* vp = ybuf + (j * HZ) * LDY + 2 * GW + hh * DH + cc;
              float o = 0.f;
              for (int kk = 0; kk <= qi; ++kk) o += pr[kk] * vp[kk * LDY];
              O::store(zbuf, LDZ, j * HZ + qi, hh * DH + cc, o);
            }
            __syncthreads();
            gemm_acc<AT, RB, CBW, GW / O::KF>(r, zbuf, LDZ, p.pk + po.o, D / O::KF, g * (GW / O::KF), own, lane);
          }
#pragma unroll
          for (int c = 0; c < CBW; ++c) {
            const float bo = raw[lo.b_o + (w * CBW + c) * 16 + lc];
#pragma unroll
            for (int rb = 0; rb < RB; ++rb) r[c][rb] += bo;
          }
        } else if (u == 1) {
          // ---------------- cross-attention unit (time token + observation tokens)
          for (int g = 0; g < NH / HG; ++g) {
            for (int it = tid; it < SPT * S * 2 * GW; it += NT) {
              const int col = it % (2 * GW), sm = (it / (2 * GW)) % S, j = it / (2 * GW * S);
              const int gcol = col < GW ? g * GW + col : D + g * GW + (col - GW);
              float v = 0.f;
              if (smp[j] >= 0)
                v = sm == 0 ? p.tkv[((size_t)k * L + l) * (2 * D) + gcol]
                            : p.okv[(((size_t)smp[j] * L + l) * nobs + (sm - 1)) * (2 * D) + gcol];
              kvbuf[(j * SMAX + sm) * (2 * GW) + col] = v;
            }
            constexpr int MPW1 = (GW / 16) / NW;
            const auto gcb = [&](int m) { return g * (GW / 16) + w + NW * m; };
            f32x4 y[MPW1][RB];
#pragma unroll
            for (int m = 0; m < MPW1; ++m)
#pragma unroll
              for (int rb = 0; rb < RB; ++rb) y[m][rb] = f32x4{0.f, 0.f, 0.f, 0.f};
            gemm_acc<AT, RB, MPW1, D / O::KF>(y, xa, LDA, p.pk + po.q, D / O::KF, 0, gcb, lane);
#pragma unroll
            for (int m = 0; m < MPW1; ++m) {
              const int loc = (w + NW * m) * 16 + lc, gcol = gcb(m) * 16 + lc;
              const float bq = raw[lo.b_q + gcol];
#pragma unroll
              for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                for (int i = 0; i < 4; ++i) ybuf[(rb * 16 + lq * 4 + i) * LDY + loc] = y[m][rb][i] + bq;
            }
            __syncthreads();
            for (int it = tid; it < SPT * HG * HZ; it += NT) {
              const int qi = it % HZ, hh = (it / HZ) % HG, j = it / (HZ * HG);
              const float* qp = ybuf + (j * HZ + qi) * LDY + hh * DH;
              float sc[SMAX];
              float mx = -INFINITY;
#pragma unroll
              for (int sm = 0; sm < SMAX; ++sm) {
                sc[sm] = -INFINITY;
                if (sm < S) {
                  const float* kp = kvbuf + (j * SMAX + sm) * (2 * GW) + hh * DH;
                  float acc = 0.f;
#pragma unroll
                  for (int cc = 0; cc < DH; cc += 4) {
                    const float4 a4 = *reinterpret_cast<const float4*>(qp + cc);
                    const float4 b4 = *reinterpret_cast<const float4*>(kp + cc);
                    acc += a4.x * b4.x + a4.y * b4.y + a4.z * b4.z + a4.w * b4.w;
                  }
                  sc[sm] = acc * kScale;
                  mx = fmaxf(mx, sc[sm]);
                }
              }
              float sum = 0.f;
#pragma unroll
              for (int sm = 0; sm < SMAX; ++sm) {
                const float e = sm < S ? expf(sc[sm] - mx) : 0.f;
                sc[sm] = e;
                sum += e;
              }
#pragma unroll
              for (int sm = 0; sm < SMAX; ++sm) pbuf[it * SMAX + sm] = sc[sm] / sum;
            }
            __syncthreads();
            constexpr int NIT2 = SPT * HG * HZ * DH;
            for (int it = tid; it < NIT2; it += NT) {
              const int cc = it % DH, qi = (it / DH) % HZ, hh = (it / (DH * HZ)) % HG, j = it / (DH * HZ * HG);
              const float* pr = pbuf + ((j * HG + hh) * HZ + qi) * SMAX;
              float o = 0.f;
              for (int sm = 0; sm < S; ++sm) o += pr[sm] * kvbuf[(j * SMAX + sm) * (2 * GW) + GW + hh * DH + cc];
              O::store(zbuf, LDZ, j * HZ + qi, hh * DH + cc, o);
            }
            __syncthreads();
            gemm_acc<AT, RB, CBW, GW / O::KF>(r, zbuf, LDZ, p.pk + po.o2, D / O::KF, g * (GW / O::KF), own, lane);
          }
#pragma unroll
          for (int c = 0; c < CBW; ++c) {
            const float bo = raw[lo.b_o2 + (w * CBW + c) * 16 + lc];
#pragma unroll
            for (int rb = 0; rb < RB; ++rb) r[c][rb] += bo;
          }
        } else {
          // ---------------- feed-forward unit, d_ff streamed in chunks of FC
          for (int ch = 0; ch < DFF / FC; ++ch) {
            constexpr int MPW1 = (FC / 16) / NW;
            const auto gcb = [&](int m) { return ch * (FC / 16) + w + NW * m; };
            f32x4 y[MPW1][RB];
#pragma unroll
            for (int m = 0; m < MPW1; ++m)
#pragma unroll
              for (int rb = 0; rb < RB; ++rb) y[m][rb] = f32x4{0.f, 0.f, 0.f, 0.f};
            gemm_acc<AT, RB, MPW1, D / O::KF>(y, xa, LDA, p.pk + po.w1, D / O::KF, 0, gcb, lane);
#pragma unroll
            for (int m = 0; m < MPW1; ++m) {
              const int loc = (w + NW * m) * 16 + lc;
              const float b1 = raw[lo.b_1 + ch * FC + loc];
#pragma unroll
              for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                for (int i = 0; i < 4; ++i)
                  O::store(zbuf, LDZ, rb * 16 + lq * 4 + i, loc, gelu_erf(y[m][rb][i] + b1));
            }
            __syncthreads();
            gemm_acc<AT, RB, CBW, FC / O::KF>(r, zbuf, LDZ, p.pk + po.w2, DFF / O::KF, ch * (FC / O::KF), own, lane);
            __syncthreads();
          }
#pragma unroll
          for (int c = 0; c < CBW; ++c) {
            const float b2 = raw[lo.b_2 + (w * CBW + c) * 16 + lc];
#pragma unroll
            for (int rb = 0; rb < RB; ++rb) r[c][rb] += b2;
          }
        }
      }
      // Eq. 1 per sample: evaluated residual (and cache refresh) or the
      // residual cached at the unit's most recent refresh.
      float* cunit = cbase + (size_t)b * (R * D);
#pragma unroll
      for (int c = 0; c < CBW; ++c)
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
          const int j = (rb * 16 + lq * 4) / HZ;
          uint8_t cd = code[0];
#pragma unroll
          for (int jj = 1; jj < SPT; ++jj)
            if (j == jj) cd = code[jj];
          f32x4* cp = reinterpret_cast<f32x4*>(cunit + ((size_t)((w * RB + rb) * CBW + c) * 64 + lane) * 4);
          if (cd & C_EVAL) {
            const f32x4 v = r[c][rb];
            if (cd & C_MERGED) mac[c][rb] = (u == 0) ? v : mac[c][rb] + v;
            if (cd & C_STORE) *cp = (cd & C_MERGED) ? mac[c][rb] : v;
            h[c][rb] += v;
          } else if (cd & C_REUSE) {
            h[c][rb] += *cp;
          }
        }
    }

    // ---- head (final LayerNorm + linear, predicts epsilon) and DDPM update
    {
      float mu[RB][4], rs[RB][4];
      row_stats<C>(h, red, mu, rs, w, lc, lq);
      f32x4 nrm[CBW][RB];
#pragma unroll
      for (int c = 0; c < CBW; ++c) {
        const int col = (w * CBW + c) * 16 + lc;
        const float g = raw[p.lnf_g + col], bb = raw[p.lnf_b + col];
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
#pragma unroll
          for (int i = 0; i < 4; ++i) nrm[c][rb][i] = (h[c][rb][i] - mu[rb][i]) * rs[rb][i] * g + bb;
      }
      float* epsp = ybuf;  // [NW][R][AMAX] partial dot products
      for (int a = 0; a < A; ++a) {
        float wo[CBW];
#pragma unroll
        for (int c = 0; c < CBW; ++c) wo[c] = raw[p.W_out + (size_t)a * D + (w * CBW + c) * 16 + lc];
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            float v = 0.f;
#pragma unroll
            for (int c = 0; c < CBW; ++c) v += nrm[c][rb][i] * wo[c];
#pragma unroll
            for (int off = 1; off < 16; off <<= 1) v += __shfl_xor(v, off);
            if (lc == 0) epsp[(w * R + rb * 16 + lq * 4 + i) * AMAX + a] = v;
          }
      }
      __syncthreads();
      const float* dd = p.ddpm + (size_t)k * 8;
      const float s1 = dd[0], sa = dd[1], c0 = dd[2], ct = dd[3], sg = dd[4];
#pragma unroll
      for (int q = 0; q < ZPT; ++q) {
        const int it = tid + q * NT;
        if (it < R * A) {
          const int row = it / A, a = it % A;
          float e = raw[p.b_out + a];
          float part = 0.f;
#pragma unroll
          for (int ww = 0; ww < NW; ++ww) part += epsp[(ww * R + row) * AMAX + a];
          e += part;
          const float x = xs[row * AMAX + a];
          float x0 = (x - s1 * e) / sa;
          if (p.clip) x0 = fminf(fmaxf(x0, -1.f), 1.f);
          float xn = c0 * x0 + ct * x;
          if (k > 0) xn += sg * zpre[q];
          xs[row * AMAX + a] = xn;
          if (t == T - 1) {
            const int s = smp[row / HZ];
            if (s >= 0) p.out[((size_t)s * HZ + (row % HZ)) * A + a] = xn;
          }
        }
      }
      __syncthreads();
    }
  }
}

// ---------------------------------------------------------------- creation
__global__ void pack_kernel(const float* __restrict__ raw, size_t off, int N, int K, int Kpad, int bf,
                            uint4* __restrict__ dst) {
  const int KF = bf ? 32 : 16;
  const int KBT = Kpad / KF;
  const size_t gid = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const size_t nfrag = (size_t)(N / 16) * KBT;
  if (gid >= nfrag * 64) return;
  const int lane = (int)(gid % 64);
  const size_t fr = gid / 64;
  const int kb = (int)(fr % KBT), nb = (int)(fr / KBT);
  const int n = nb * 16 + (lane & 15), q = lane >> 4;
  const float* W = raw + off + (size_t)n * K;
  uint32_t e[4];
  if (bf) {
    for (int i = 0; i < 4; ++i) {
      const int k0 = kb * 32 + q * 8 + 2 * i;
      const uint32_t lo = k0 < K ? bf16_rne(W[k0]) : 0u;
      const uint32_t hi = k0 + 1 < K ? bf16_rne(W[k0 + 1]) : 0u;
      e[i] = lo | (hi << 16);
    }
  } else {
    for (int j = 0; j < 4; ++j) {
      const int kk = kb * 16 + 4 * j + q;
      e[j] = kk < K ? __float_as_uint(W[kk]) : 0u;
    }
  }
  dst[gid] = make_uint4(e[0], e[1], e[2], e[3]);
}

// memory row 0 of every timestep: sinusoid(k) + P_mem[0], fp64 -> fp32
__global__ void time_row_kernel(const float* __restrict__ raw, uint32_t pmem0, int T, int D,
                                float* __restrict__ rows) {
  const int gid = blockIdx.x * blockDim.x + threadIdx.x;
  if (gid >= T * D) return;
  const int k = gid / D, j = gid % D, half = D / 2;
  const int jj = j < half ? j : j - half;
  const double om = exp(-log(10000.0) * (double)jj / (double)(half - 1));
  const double a = (double)k * om;
  const double v = (j < half ? sin(a) : cos(a)) + (double)raw[pmem0 + j];
  rows[gid] = (float)v;
}

// keys/values of the time token for every (timestep, layer)
__global__ void time_kv_kernel(const float* __restrict__ raw, const float* __restrict__ rows,
                               const uint32_t* __restrict__ wkv, const uint32_t* __restrict__ bkv, int T,
                               int L, int D, int bf, float* __restrict__ tkv) {
  const size_t gid = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (gid >= (size_t)T * L * 2 * D) return;
  const int col = (int)(gid % (2 * D));
  const int l = (int)((gid / (2 * D)) % L);
  const int k = (int)(gid / ((size_t)2 * D * L));
  const float* W = raw + wkv[l] + (size_t)col * D;
  const float* m = rows + (size_t)k * D;
  float acc = 0.f;
  for (int j = 0; j < D; ++j) {
    const float wv = bf ? __uint_as_float(bf16_rne(W[j]) << 16) : W[j];
    acc = fmaf(m[j], wv, acc);
  }
  tkv[gid] = acc + raw[bkv[l] + col];
}

// DDPM constants (squared-cosine betas, fixed-small variance), fp64 -> fp32:
// per timestep i: sqrt(1-abar), sqrt(abar), c0, ct, sigma.
__global__ void ddpm_kernel(int T, float* tab) {
  if (blockIdx.x != 0 || threadIdx.x != 0) return;
  const double s = 0.008, half_pi = 1.5707963267948966;
  double abar = 1.0;
  for (int i = 0; i < T; ++i) {
    double f0 = cos(((double)i / T + s) / (1.0 + s) * half_pi);
    double f1 = cos(((double)(i + 1) / T + s) / (1.0 + s) * half_pi);
    f0 *= f0;
    f1 *= f1;
    const double beta = fmin(1.0 - f1 / f0, 0.999);
    const double alpha = 1.0 - beta;
    const double abar_prev = abar;
    abar *= alpha;
    const double c0 = sqrt(abar_prev) * beta / (1.0 - abar);
    const double ct = sqrt(alpha) * (1.0 - abar_prev) / (1.0 - abar);
    const double var = fmax((1.0 - abar_prev) / (1.0 - abar) * beta, 1e-20);
    float* r = tab + (size_t)i * 8;
    r[0] = (float)sqrt(1.0 - abar);
    r[1] = (float)sqrt(abar);
    r[2] = (float)c0;
    r[3] = (float)ct;
    r[4] = (float)sqrt(var);
    r[5] = r[6] = r[7] = 0.f;
  }
}

hipError_t launch_pack(const float* raw, size_t off, int N, int K, int Kpad, int dtype, uint4* dst,
                       hipStream_t stream) {
  const int KF = dtype == 1 ? 32 : 16;
  const size_t n = (size_t)(N / 16) * (Kpad / KF) * 64;
  const int bs = 256;
  hipLaunchKernelGGL(pack_kernel, dim3((unsigned)((n + bs - 1) / bs)), dim3(bs), 0, stream, raw, off, N, K,
                     Kpad, dtype == 1 ? 1 : 0, dst);
  return hipGetLastError();
}

hipError_t launch_time_kv(const float* raw, uint32_t pmem0, const uint32_t* wkv, const uint32_t* bkv,
                          int T, int L, int D, int dtype, float* rows_scratch, float* tkv,
                          hipStream_t stream) {
  const int bs = 256;
  hipLaunchKernelGGL(time_row_kernel, dim3((T * D + bs - 1) / bs), dim3(bs), 0, stream, raw, pmem0, T, D,
                     rows_scratch);
  const size_t n = (size_t)T * L * 2 * D;
  hipLaunchKernelGGL(time_kv_kernel, dim3((unsigned)((n + bs - 1) / bs)), dim3(bs), 0, stream, raw,
                     rows_scratch, wkv, bkv, T, L, D, dtype == 1 ? 1 : 0, tkv);
  return hipGetLastError();
}

hipError_t launch_ddpm_table(int T, float* table, hipStream_t stream) {
  hipLaunchKernelGGL(ddpm_kernel, dim3(1), dim3(1), 0, stream, T, table);
  return hipGetLastError();
}

// ---------------------------------------------------------------- dispatch
#define EVO_SHAPES(X)                                  \
  X(float, 64, 32, 8, 2, 256, 4, 2, 256, 8)            \
  X(__bf16, 64, 32, 8, 2, 256, 4, 2, 256, 8)           \
  X(float, 256, 64, 16, 1, 1024, 8, 4, 256, 8)         \
  X(float, 256, 64, 16, 2, 1024, 8, 2, 256, 8)         \
  X(__bf16, 256, 64, 16, 1, 1024, 8, 4, 512, 8)        \
  X(__bf16, 256, 64, 16, 2, 1024, 8, 2, 256, 8)        \
  X(__bf16, 768, 64, 32, 1, 3072, 8, 2, 256, 5)

template <class AT> constexpr int dtype_of() { return std::is_same<AT, float>::value ? 0 : 1; }

bool kernel_available(const KernelKey& key, int* threads) {
#define X(AT, D, DH, HZ, SPT, DFF, NW, HG, FC, SMAX)                                                     \
  if (key.d == D && key.dh == DH && key.horizon == HZ && key.d_ff == DFF && key.dtype == dtype_of<AT>() && \
      key.spt == SPT) {                                                                                  \
    if (threads) *threads = NW * 64;                                                                     \
    return true;                                                                                         \
  }
  EVO_SHAPES(X)
#undef X
  return false;
}

int kernel_max_obs_tokens_for(const KernelKey& key) {
#define X(AT, D, DH, HZ, SPT, DFF, NW, HG, FC, SMAX)                                                     \
  if (key.d == D && key.dh == DH && key.horizon == HZ && key.d_ff == DFF && key.dtype == dtype_of<AT>() && \
      key.spt == SPT)                                                                                    \
    return (SMAX - 1) < 16 / SPT ? (SMAX - 1) : 16 / SPT;
  EVO_SHAPES(X)
#undef X
  return 0;
}

int kernel_max_action_dim() { return 16; }

hipError_t launch_denoise(const KernelKey& key, const KParams& p, hipStream_t stream) {
#define X(AT, D, DH, HZ, SPT, DFF, NW, HG, FC, SMAX)                                                     \
  if (key.d == D && key.dh == DH && key.horizon == HZ && key.d_ff == DFF && key.dtype == dtype_of<AT>() && \
      key.spt == SPT) {                                                                                  \
    hipLaunchKernelGGL((denoise_kernel<AT, D, DH, HZ, SPT, DFF, NW, HG, FC, SMAX>), dim3(p.n_tiles),      \
                       dim3(NW * 64), 0, stream, p);                                                     \
    return hipGetLastError();                                                                            \
  }
  EVO_SHAPES(X)
#undef X
  return hipErrorInvalidValue;
}

}  // namespace evo
