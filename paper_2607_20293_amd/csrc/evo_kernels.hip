// HIP kernels (gfx950) of the schedule-driven cached denoising loop.
//
// Design: one workgroup owns a tile of whole samples (rows = samples x
// horizon tokens) for the entire T-step reverse process.  Samples never
// interact, so a tile needs no communication with other workgroups: the
// whole query is one launch with no grid-wide synchronisation.
//
//  * The residual stream h of the tile lives in registers, laid out as the
//    accumulator fragments of 16x16 MFMA tiles (each wave owns a fixed set
//    of 16-column blocks of d).
//  * The schedule arrives as per-step unit bitmasks {evaluate, reuse,
//    store}.  Cacheable units (Sec. 3.1: SA, CA, FFN residual branches) are
//    evaluated only where the schedule says so (Eq. 1); a refreshed residual
//    is stored in the tile's cache in HBM only if a later step reuses it.
//    Between two evaluated units the reused residuals of the skipped units
//    are added in order, their cache loads issued in batches.
//  * Every unit is "LayerNorm -> chunked stage-1 product -> per-chunk
//    transform (attention per head group, or GELU) -> stage-2 product
//    accumulated into the unit's residual".  Activations stay in LDS;
//    projection weights are streamed from L2/HBM as pre-packed 1 KiB MFMA
//    fragments (16 output columns x 32 bf16 / 16 fp32 of K, 16 bytes per
//    lane), so every weight load is one coalesced 16-byte load per lane, and
//    the first fragments of each product are requested before the phase
//    that precedes it.
//  * Attention, the action embedding and the head use fp32 16x16x4 MFMA
//    tiles; the DDPM update is fused at the end of every step.
#include "evo_kernels.hpp"

#include <algorithm>
#include <cmath>
#include <type_traits>

namespace evo {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x2 __attribute__((ext_vector_type(2)));

constexpr uint64_t kMergedBit = 1ull << 63;
constexpr int kMaskEntries = 341;  // (T x samples per tile) entries of 3 x u64 in LDS (8 KiB)
constexpr int kMaxLayers = 21;     // 3L <= 63 units (one 64-bit mask per step)

// float -> bfloat16 bits, round to nearest even: gfx950's conversion
// instruction (v_cvt_pk_bf16_f32), two values at a time where possible
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t bf16_rne(float f) {
  return __builtin_bit_cast(uint16_t, (__bf16)f);
}
// (bf16(lo) | bf16(hi) << 16)
__device__ __forceinline__ uint32_t bf16x2_rne(float lo, float hi) {
  const bf16x2_t v = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, v);
}

// fp16 pair: each value clamped to the finite fp16 range, then rounded to
// nearest even (a residual beyond +-65504 is stored as +-65504)
typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t f16x2_sat(float lo, float hi) {
  const f16x2_t v = {(_Float16)__builtin_amdgcn_fmed3f(lo, -65504.f, 65504.f),
                     (_Float16)__builtin_amdgcn_fmed3f(hi, -65504.f, 65504.f)};
  return __builtin_bit_cast(uint32_t, v);
}
__device__ __forceinline__ f32x4 f16x4_to_f32(uint32_t x0, uint32_t x1) {
  const f16x2_t a = __builtin_bit_cast(f16x2_t, x0), b = __builtin_bit_cast(f16x2_t, x1);
  return f32x4{(float)a[0], (float)a[1], (float)b[0], (float)b[1]};
}

__device__ __forceinline__ f32x4 mfma4(float a, float b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// 16x16 tile of q · kᵀ over a DH-long dot product on fp32 MFMA.  The K order
// is permuted (any bijection of k works when both operands use it): lane
// group lq takes k = 16·lq + j at step j, so each lane reads 16 contiguous
// floats of its row (four 16-byte LDS reads) instead of 16 strided ones, and
// four independent accumulators shorten the dependent MFMA chain.
template <int DH>
__device__ __forceinline__ f32x4 qk_tile(const float* qrow, const float* krow, bool kvalid, int lq) {
  static_assert(DH % 64 == 0 || DH == 32, "head size");
  f32x4 acc[4] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
  constexpr int KPL = DH / 4;  // k per lane group
#pragma unroll
  for (int j4 = 0; j4 < KPL / 4; ++j4) {
    const f32x4 qv = *reinterpret_cast<const f32x4*>(qrow + lq * KPL + 4 * j4);
    f32x4 kv = *reinterpret_cast<const f32x4*>(krow + lq * KPL + 4 * j4);
    if (!kvalid) kv = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int e = 0; e < 4; ++e) acc[e] = mfma4(qv[e], kv[e], acc[e]);
  }
  return (acc[0] + acc[1]) + (acc[2] + acc[3]);
}

// waves sharing one (head, 16-query block) of attention: each repeats the
// scores and computes its share of the DH / 16 value column blocks
constexpr int attn_waves_per_pair(int nw, int npair, int ncb) {
  int wpp = 1;
  while (wpp * 2 <= nw / (npair > 0 ? npair : 1) && ncb % (wpp * 2) == 0) wpp *= 2;
  return wpp;
}

// Cross-lane moves within a row of 16 lanes (DPP): swap neighbours, swap
// pairs, mirror within 8, mirror within 16.  Each pairs every lane with a
// lane of the other half of its group, so four steps combine all 16 lanes
// and every lane ends with the same value.
template <int CTRL>
__device__ __forceinline__ float dpp_mov(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xF, 0xF, true));
}
__device__ __forceinline__ float row16_sum(float v) {
  v += dpp_mov<0xB1>(v);
  v += dpp_mov<0x4E>(v);
  v += dpp_mov<0x141>(v);
  v += dpp_mov<0x140>(v);
  return v;
}
__device__ __forceinline__ float row16_max(float v) {
  v = fmaxf(v, dpp_mov<0xB1>(v));
  v = fmaxf(v, dpp_mov<0x4E>(v));
  v = fmaxf(v, dpp_mov<0x141>(v));
  v = fmaxf(v, dpp_mov<0x140>(v));
  return v;
}

// Orders a wave's own LDS writes before its following LDS reads (other
// lanes' data) without a workgroup barrier.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
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
    acc = mfma4(__uint_as_float(a.x), __uint_as_float(b.x), acc);
    acc = mfma4(__uint_as_float(a.y), __uint_as_float(b.y), acc);
    acc = mfma4(__uint_as_float(a.z), __uint_as_float(b.z), acc);
    acc = mfma4(__uint_as_float(a.w), __uint_as_float(b.w), acc);
  }
};

// k-steps a product keeps in flight: about INFL 1 KiB fragments per wave
template <int MPW, int NKF, int INFL>
constexpr int pd_of() {
  constexpr int pd0 = INFL / MPW > 0 ? INFL / MPW : 1;
  return pd0 < NKF ? pd0 : (NKF > 1 ? NKF - 1 : 1);
}
// k-steps requested ahead of a product (before the phase that precedes it):
// about PF fragments per wave, at least one k-step, at most the in-flight depth
template <int MPW, int NKF, int INFL, int PF>
constexpr int np_of() {
  constexpr int n = PF / MPW > 0 ? PF / MPW : 1;
  constexpr int pd = pd_of<MPW, NKF, INFL>();
  return n < pd ? n : pd;
}

// First NP k-steps of weight fragments of a product (issued ahead of it).
template <int NP, int MPW, class GCB>
__device__ __forceinline__ void gemm_pref(uint4 (&bc)[NP][MPW], const uint4* W, int KBT, int kf0, GCB gcb,
                                          int lane) {
#pragma unroll
  for (int d = 0; d < NP; ++d)
#pragma unroll
    for (int m = 0; m < MPW; ++m) bc[d][m] = W[((size_t)gcb(m) * KBT + kf0 + d) * 64 + lane];
}

// acc[m][rb] += A[rb*16 .. +16][k-range] x W[col block gcb(m)][k-range]^T
// A: LDS operand, row stride lda elements, offset to the k-range start.
// W: packed fragments of a matrix with KBT fragments per column block; kf0
// is the first fragment of the k-range, NKF its length; bc holds the
// fragments of the first NP k-steps (gemm_pref).  Weight fragments are
// requested PD k-steps ahead of their MFMAs (about INFL 1 KiB fragments in
// flight per wave); a scheduling fence per step keeps the compiler from
// hoisting further loads.
template <class AT, int RBk, int MPW, int NKF, int INFL, int NP, class GCB>
__device__ __forceinline__ void gemm_run(f32x4 (&acc)[MPW][RBk], const AT* A, int lda, const uint4* W, int KBT,
                                         int kf0, GCB gcb, int lane, uint4 (&bc)[NP][MPW]) {
  using O = Op<AT>;
  constexpr int PD = pd_of<MPW, NKF, INFL>();
  static_assert(NP >= 1 && NP <= PD, "prefetched k-steps");
  const int lc = lane & 15, lq = lane >> 4;
  const uint4* wp[MPW];
#pragma unroll
  for (int m = 0; m < MPW; ++m) wp[m] = W + ((size_t)gcb(m) * KBT + kf0) * 64 + lane;
  uint4 buf[PD + 1][MPW];
#pragma unroll
  for (int d = 0; d < NP; ++d)
#pragma unroll
    for (int m = 0; m < MPW; ++m) buf[d][m] = bc[d][m];
#pragma unroll
  for (int d = NP; d < PD; ++d)
#pragma unroll
    for (int m = 0; m < MPW; ++m)
      if (d < NKF) buf[d][m] = wp[m][d * 64];
#pragma unroll
  for (int kf = 0; kf < NKF; ++kf) {
    if (kf + PD < NKF) {
#pragma unroll
      for (int m = 0; m < MPW; ++m) buf[(kf + PD) % (PD + 1)][m] = wp[m][(kf + PD) * 64];
    }
    uint4 a[RBk];
#pragma unroll
    for (int rb = 0; rb < RBk; ++rb)
      a[rb] = *reinterpret_cast<const uint4*>(A + (rb * 16 + lc) * lda + kf * O::KF + lq * O::VE);
#pragma unroll
    for (int m = 0; m < MPW; ++m)
#pragma unroll
      for (int rb = 0; rb < RBk; ++rb) O::mma(acc[m][rb], a[rb], buf[kf % (PD + 1)][m]);
    __builtin_amdgcn_sched_barrier(0);
  }
}

template <class AT, int RBk, int MPW, int NKF, class GCB>
__device__ __forceinline__ void gemm_acc(f32x4 (&acc)[MPW][RBk], const AT* A, int lda, const uint4* W, int KBT,
                                         int kf0, GCB gcb, int lane) {
  uint4 bc[1][MPW];
  gemm_pref<1, MPW>(bc, W, KBT, kf0, gcb, lane);
  gemm_run<AT, RBk, MPW, NKF, 6, 1>(acc, A, lda, W, KBT, kf0, gcb, lane, bc);
}

// Hardware transcendental approximations (v_rsq_f32, v_exp_f32, v_rcp_f32;
// about 1 ulp).  The phases around the matrix products run at one or two
// waves per SIMD, where every dependent instruction is exposed latency; the
// correctly rounded library sequences cost tens of instructions each.
__device__ __forceinline__ float fast_rsqrt(float x) { return __builtin_amdgcn_rsqf(x); }
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float fast_rcp(float x) { return __builtin_amdgcn_rcpf(x); }
constexpr float kLog2e = 1.4426950408889634f;

// GELU with the error function (0.5 v (1 + erf(v / sqrt 2))).  erfc(x) for
// x >= 0 uses the rational-exponential approximation of Abramowitz and
// Stegun, Handbook of Mathematical Functions, formula 7.1.26 (absolute error
// below 1.5e-7); 1 + erf(v/sqrt2) is then erfc(|x|) for v < 0 and
// 2 - erfc(|x|) for v >= 0, which avoids cancellation on the negative side.
__device__ __forceinline__ float gelu_erf(float v) {
  const float x = fabsf(v) * 0.70710678118654752f;
  const float t = fast_rcp(1.0f + 0.3275911f * x);
  const float poly =
      t * (0.254829592f + t * (-0.284496736f + t * (1.421413741f + t * (-1.453152027f + t * 1.061405429f))));
  const float q = poly * fast_exp2(-x * x * kLog2e);  // erfc(x)
  return 0.5f * v * (v >= 0.f ? 2.0f - q : q);
}

template <int D, int DH, int HZ, int SPT, int DFF, int NW, int HG, int FC, int SMAX, int TEAM>
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
  static constexpr int KOBS = 64;
  static constexpr int NJB = HZ >= 16 ? HZ / 16 : 1;   // key blocks per query block (self-attention)
  static constexpr int SPB = HZ >= 16 ? 1 : 16 / HZ;   // samples per 16-row block
  static constexpr int SLOTS = 16 / SPB;               // memory columns per sample in a 16-wide tile
  static constexpr int PS = 17;                        // stride of a 16x16 fp32 scratch tile
  static constexpr int PWN = (NJB > RB ? NJB : RB) * 16 * PS;
  static constexpr int NB = (8 / (CBW * RB)) > 0 ? (8 / (CBW * RB)) : 1;  // reuse loads per batch
  // cross-attention folded into per-token fold records (width 256; one
  // sample per 16-row block); used when n_heads x memory tokens <= 16
  static constexpr bool FOLD = D == 256 && HZ >= 16;
  static constexpr int REC = 2 * NH * D + 16;                              // floats per fold record
  static constexpr int FOLD_LDS = FOLD ? NW * RB * 256 + 16 * R + RB * 16 * D : 0;
};

// Cross-attention with few memory tokens, folded.  With q = x W_q^T + b_q
// (x the LayerNorm output of a row), the score of head h against memory
// token j is q_h . k_jh = x . u_jh + c_jh with u_jh = W_q,h^T k_jh (W_q,h the
// head's DH rows of W_q) and c_jh = b_q,h . k_jh, and the unit's output
// sum_h sum_j p_jh v_jh W_o2,h^T + b_o2 = sum_h sum_j p_jh w_jh + b_o2 with
// w_jh = W_o2,h v_jh (W_o2,h the head's DH columns of W_o2).  Projecting the
// S tokens once per (token, layer) replaces the two d x d products of every
// evaluation by two products with S x n_heads columns.
//
// A fold record holds u [NH][D] (for fp32 operands in the fragment column
// order of the LDS operand, Op<float>::pcol), w [NH][D] and c [NH].  The
// workgroup folds `nrows` <= MR key/value rows (kv: [row][2D] keys then
// values, row stride ldkv, in LDS) with the layer's W_q (rows), the
// transposed W_o2 (row e = column e of W_o2) and b_q; dst(row) is the record
// of a row or null.  Weights are rounded to bf16 first when BF, as the packed matrices.
template <int D, int DH, int NT, int MR, bool BF, class DST>
__device__ void fold_rows(const float* __restrict__ raw, uint32_t wq, uint32_t wo2t,
                                                    uint32_t bq, const float* kv, int ldkv, int nrows, DST dst,
                                                    int tid) {
  constexpr int NH = D / DH, C4 = D / 4, EB = 32;  // EB weight rows requested at once
  static_assert(DH % EB == 0, "fold batches");
  // work item = (u or w, head, 4 columns): the head's DH weight rows are
  // read 16 bytes per lane, EB rows in flight
  for (int it = tid; it < 2 * NH * C4; it += NT) {
    const int isw = it / (NH * C4), hd = (it / C4) % NH, c0 = (it % C4) * 4;
    const float* W = raw + (isw ? wo2t : wq) + (size_t)hd * DH * D + c0;
    const float* kr = kv + (isw ? D : 0) + hd * DH;
    f32x4 acc[MR];
#pragma unroll
    for (int r = 0; r < MR; ++r) acc[r] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int e0 = 0; e0 < DH; e0 += EB) {
      f32x4 wv[EB];
#pragma unroll
      for (int e = 0; e < EB; ++e) wv[e] = *reinterpret_cast<const f32x4*>(W + (size_t)(e0 + e) * D);
      if (BF) {
#pragma unroll
        for (int e = 0; e < EB; ++e)
#pragma unroll
          for (int q = 0; q < 4; ++q) wv[e][q] = __uint_as_float(bf16_rne(wv[e][q]) << 16);
      }
#pragma unroll
      for (int r = 0; r < MR; ++r)
        if (r < nrows) {
#pragma unroll
          for (int e4 = 0; e4 < EB / 4; ++e4) {
            const f32x4 kk = *reinterpret_cast<const f32x4*>(kr + r * ldkv + e0 + 4 * e4);
#pragma unroll
            for (int q = 0; q < 4; ++q)
#pragma unroll
              for (int t = 0; t < 4; ++t) acc[r][t] = fmaf(wv[4 * e4 + q][t], kk[q], acc[r][t]);
          }
        }
    }
#pragma unroll
    for (int r = 0; r < MR; ++r)
      if (r < nrows) {
        float* q = dst(r);
        if (!q) continue;
        if (isw) {
          *reinterpret_cast<f32x4*>(q + NH * D + hd * D + c0) = acc[r];
        } else {
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            const int c = c0 + t;
            q[hd * D + (BF ? c : ((c & ~15) | ((c & 3) << 2) | ((c >> 2) & 3)))] = acc[r][t];
          }
        }
      }
  }
  for (int it = tid; it < nrows * NH; it += NT) {
    const int r = it / NH, hd = it % NH;
    float a = 0.f;
    for (int e = 0; e < DH; ++e) a = fmaf(raw[bq + hd * DH + e], kv[r * ldkv + hd * DH + e], a);
    float* q = dst(r);
    if (q) q[2 * NH * D + hd] = a;
  }
}

// LayerNorm statistics of the tile rows from the register-resident stream:
// per-lane (mean, M2) over its columns, merged across the 16 lanes of a row
// group with shuffles; the waves' partials meet in LDS (one barrier) and
// every wave merges them for all rows in a fixed tree (pairwise, equal
// counts), so all waves hold the same bits.
template <class C>
__device__ __forceinline__ void ln_stats(const f32x4 (&h)[C::CBW][C::RB], float (*red)[C::R][2],
                                         float (&mu)[C::RB][4], float (&rs)[C::RB][4], int w, int lc, int lq) {
  constexpr int D = C::CB * 16;
  constexpr float nw = 16.0f * C::CBW;
#pragma unroll
  for (int rb = 0; rb < C::RB; ++rb)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float m = 0.f;
#pragma unroll
      for (int c = 0; c < C::CBW; ++c) m += h[c][rb][i];
      m *= (1.0f / C::CBW);
      float q = 0.f;
#pragma unroll
      for (int c = 0; c < C::CBW; ++c) {
        const float e = h[c][rb][i] - m;
        q += e * e;
      }
      // merge equal-count groups pairwise: mean of the two means, M2 sum
      // plus the spread term (symmetric, so both partners agree bitwise)
      float n = (float)C::CBW;
      const auto merge = [&](float mo, float qo) {
        const float d = mo - m;
        m = 0.5f * (m + mo);
        q = q + qo + d * d * (0.5f * n);
        n *= 2.f;
      };
      merge(dpp_mov<0xB1>(m), dpp_mov<0xB1>(q));
      merge(dpp_mov<0x4E>(m), dpp_mov<0x4E>(q));
      merge(dpp_mov<0x141>(m), dpp_mov<0x141>(q));
      merge(dpp_mov<0x140>(m), dpp_mov<0x140>(q));
      if (lc == 0) {
        red[w][rb * 16 + lq * 4 + i][0] = m;
        red[w][rb * 16 + lq * 4 + i][1] = q;
      }
    }
  __syncthreads();
  // every wave merges the wave partials itself (no second barrier): the
  // four lanes of a quad take one row, each its share of the waves, then
  // two symmetric quad merges give all four the same bits; lane l then
  // holds the statistics of row l / 4 of the row block
  static_assert(C::NWV % 4 == 0, "waves per quad lane");
  constexpr int WPL = C::NWV / 4;
  const int lane = lc + 16 * lq, qrow = lane >> 2, qp = lane & 3;
#pragma unroll
  for (int rb = 0; rb < C::RB; ++rb) {
    const int row = rb * 16 + qrow;
    float m = red[qp * WPL][row][0], q = red[qp * WPL][row][1], n = nw;
    const auto merge = [&](float mo, float qo) {
      const float d = mo - m;
      m = 0.5f * (m + mo);
      q = q + qo + d * d * (0.5f * n);
      n *= 2.f;
    };
#pragma unroll
    for (int x = 1; x < WPL; ++x) merge(red[qp * WPL + x][row][0], red[qp * WPL + x][row][1]);
    merge(dpp_mov<0xB1>(m), dpp_mov<0xB1>(q));
    merge(dpp_mov<0x4E>(m), dpp_mov<0x4E>(q));
    const float r_ = fast_rsqrt(q * (1.0f / D) + 1e-5f);
    // rows lq * 4 + i sit in lanes 16 lq + 4 i: a swizzle inside each
    // 32-lane half keeps lane bit 4 and sets bits 2..3 to i
#define EVO_LN_PICK(i)                                                                              \
    mu[rb][i] = __int_as_float(__builtin_amdgcn_ds_swizzle(__float_as_int(m), 0x10 | ((4 * (i)) << 5))); \
    rs[rb][i] = __int_as_float(__builtin_amdgcn_ds_swizzle(__float_as_int(r_), 0x10 | ((4 * (i)) << 5)));
    EVO_LN_PICK(0)
    EVO_LN_PICK(1)
    EVO_LN_PICK(2)
    EVO_LN_PICK(3)
#undef EVO_LN_PICK
  }
}

template <class AT, int D, int DH, int HZ, int SPT, int DFF, int NW, int HG, int FC, int SMAX, int TEAM>
__global__ void __launch_bounds__(NW * 64) denoise_kernel(const KParams p) {
  using O = Op<AT>;
  using OF = Op<float>;
  using C = Cfg<D, DH, HZ, SPT, DFF, NW, HG, FC, SMAX, TEAM>;
  constexpr int NT = C::NT, R = C::R, RB = C::RB, NH = C::NH, CB = C::CB, CBW = C::CBW, GW = C::GW;
  constexpr int LDA = D + O::PAD, LDY = C::LDY, LDZ = C::ZW + O::PAD;
  constexpr int KOBS = C::KOBS, LDO = KOBS + O::PAD;
  constexpr int NJB = C::NJB, SLOTS = C::SLOTS, PS = C::PS, PWN = C::PWN, NB = C::NB;
  static_assert(R % 16 == 0 && CB % NW == 0 && NH % HG == 0 && DFF % FC == 0, "tile shape");
  static_assert((3 * GW / 16) % NW == 0 && (GW / 16) % NW == 0 && (FC / 16) % NW == 0, "block split");
  static_assert((NH / HG) % TEAM == 0 && (DFF / FC) % TEAM == 0, "team members split head groups and chunks");
  static_assert(HZ % 4 == 0 && (HZ & (HZ - 1)) == 0 && HZ <= 64, "horizon must be a power of two in [4, 64]");
  static_assert(NW * R * 16 <= R * LDY, "head partials must fit the stage-1 buffer");
  static_assert(16 * LDO * (int)sizeof(AT) <= R * LDY * 4, "observation operand must fit");
  static_assert(SMAX <= SLOTS, "memory tokens per sample must fit a 16-column tile");
  static_assert(DH % 16 == 0, "head dim");
  // embedding / head constants of the lane's columns, kept across steps in
  // LDS (EMB_LDS, where it fits) or in registers (KEEP_EMB), else re-read
  constexpr bool EMB_LDS = RB == 1 && CBW <= 4 && (sizeof(AT) == 2 || TEAM > 1 || D <= 64);
  constexpr bool KEEP_EMB = RB == 1 && CBW <= 4 && !EMB_LDS;
  constexpr bool PB_LDS = EMB_LDS && (TEAM > 1 || D <= 64);  // else the row biases stay in registers
  // layer-merged residual sum accumulated in registers, else in its cache slot
  constexpr bool MAC_REG = CBW * RB <= 4;
  static_assert(MAC_REG || SPT == 1 || sizeof(AT) == 4, "bf16 layer sums in memory need one sample per tile");
  // weight fragments in flight per wave in the unit products (at width 768
  // and in two-sample bf16 tiles the residual stream and the unit output
  // leave room for 8)
  constexpr int INFL = D > 256 ? 8
                       : (TEAM > 1 && RB == 1) ? 16
                       : (RB == 1 && CBW <= 2) ? 12
                       : sizeof(AT) == 2 ? 8 : 6;
  constexpr float kScale = (DH == 64) ? 0.125f : (DH == 32 ? 0.17677669529663688f : 0.0f);
  static_assert(DH == 64 || DH == 32, "head dim");

  __shared__ __attribute__((aligned(16))) AT xa[R * LDA];
  __shared__ __attribute__((aligned(16))) float ybuf[R * LDY > C::FOLD_LDS ? R * LDY : C::FOLD_LDS];
  // the feed-forward chunks alternate between two operand buffers, so a
  // chunk's GELU outputs never overwrite the previous chunk's while a wave
  // may still read them, and no barrier ends a chunk (where LDS allows)
  constexpr bool ZB2 = D <= 256 && !(sizeof(AT) == 4 && SPT > 1);
  __shared__ __attribute__((aligned(16))) AT zbuf[(ZB2 ? 2 : 1) * R * LDZ];
  __shared__ __attribute__((aligned(16))) float pw[NW * PWN];
  __shared__ __attribute__((aligned(16))) float kvbuf[SPT * SMAX * 2 * GW];
  __shared__ float red[NW][R][2];
  __shared__ __attribute__((aligned(16))) float xs[R * 16];
  __shared__ uint64_t msk[kMaskEntries * 3];
  __shared__ LayerOff s_loff[kMaxLayers];
  __shared__ PackOff s_poff[kMaxLayers];
  __shared__ int smp[SPT];

  const int tid = threadIdx.x, w = tid >> 6;
  // lane indices are made opaque to the optimiser (an empty asm) once per
  // step, unit, head group and d_ff chunk, so that the address arithmetic
  // derived from them is recomputed inside the loops instead of being
  // hoisted into registers held for the whole kernel (which spilled)
  int lane = tid & 63, lc = lane & 15, lq = lane >> 4;
  // a team of TEAM workgroups shares a tile: each member evaluates its share
  // of every unit's head groups / d_ff chunks and the partial residuals are
  // summed through HBM; everything else is replicated in every member
  const int member = blockIdx.x % TEAM;
  const int tile = blockIdx.x / TEAM;
  __shared__ int s_abort;
  const int L = p.L, A = p.A, T = p.T, U = 3 * L, nobs = p.n_obs, S = 1 + nobs;
  const float* raw = p.raw;
  // folded cross-attention (n_heads x S <= 16, checked by the host): okv
  // then holds fold records [batch][L][n_obs][REC] instead of keys/values
  const bool fold = C::FOLD && p.fold != 0;
  constexpr int REC = C::REC;

  if (tid < SPT) smp[tid] = p.tile_sample[tile * SPT + tid];
  if (tid == 0) s_abort = 0;
  float* const okv = p.okv + (size_t)member * p.okv_member_stride;
  for (int it = tid; it < L * (int)(sizeof(LayerOff) / 4); it += NT)
    reinterpret_cast<uint32_t*>(s_loff)[it] = reinterpret_cast<const uint32_t*>(p.loff)[it];
  for (int it = tid; it < L * (int)(sizeof(PackOff) / 8); it += NT)
    reinterpret_cast<uint64_t*>(s_poff)[it] = reinterpret_cast<const uint64_t*>(p.poff)[it];
  for (int it = tid; it < SPT * T * 3; it += NT) {
    const int j = it / (T * 3), r = it % (T * 3);
    msk[it] = p.masks[(size_t)p.tile_slot[tile * SPT + j] * T * 3 + r];
  }
  __syncthreads();

  // initial sample x_T, stored [row][pcol(a)] (zero-padded to 16 columns)
  for (int it = tid; it < R * 16; it += NT) {
    const int row = it / 16, a = it % 16, s = smp[row / HZ];
    xs[row * 16 + OF::pcol(a)] = (s >= 0 && a < A) ? p.noise[((size_t)s * HZ + (row % HZ)) * A + a] : 0.f;
  }

  // ---- per query: observation tokens and their keys/values in every layer
  // (folded: their fold records come from the observation pre-pass)
  if (!fold) {
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
      gemm_acc<AT, 1, MPWO, KOBS / O::KF>(acc, ob, LDO, p.pk + p.pk_obs, p.obs_pad / O::KF, c * (KOBS / O::KF),
                                           [&](int m) { return w + NW * m; }, lane);
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
      gemm_acc<AT, 1, MPWK, D / O::KF>(kv, xa, LDA, p.pk + s_poff[l].kv, D / O::KF, 0,
                                        [&](int m) { return w + NW * m; }, lane);
      const uint32_t bkv = s_loff[l].b_kv;
#pragma unroll
      for (int m = 0; m < MPWK; ++m) {
        const int gcol = (w + NW * m) * 16 + lc;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int row = lq * 4 + i;
          if (row < SPT * nobs) {
            const int j = row / nobs, o = row % nobs;
            if (smp[j] >= 0)
              okv[(((size_t)smp[j] * L + l) * nobs + o) * (2 * D) + gcol] = kv[m][0][i] + raw[bkv + gcol];
          }
        }
      }
    }
    __syncthreads();
  }

  // sample slot of each of this lane's fragment row groups (4 rows, one sample)
  int jrow[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) jrow[rb] = (rb * 16 + lq * 4) / HZ;
  // residual caches of this workgroup: [3L][R*D] values in fragment order.
  // fp16 with bf16 operands (rounded once per stored residual, clamped to
  // the finite fp16 range; the stream and the layer sums stay fp32): half
  // the bytes of the reuse loads, which every tile of a shared schedule
  // issues at the same time.  fp16 rather than bf16: bf16 caches took the
  // 512-sample population's worst sample past the bf16 error bar
  // (3.04e-2).  fp32 with fp32 operands.  One format for every tile size,
  // so that a sample's result does not depend on the batch.
  constexpr int CE = (sizeof(AT) == 2) ? 2 : 4;
  unsigned char* const cbase = reinterpret_cast<unsigned char*>(p.cache) + (size_t)(tile * TEAM + member) * U * (R * D) * CE;
  // Team exchange slots: [tile][3][TEAM][R*D] floats, slot n % 3 carries
  // the partials of the n-th evaluated unit.  A slot word that still holds
  // the sentinel has not been written yet; every member resets its own slot
  // of unit n-1 once it holds all partials of unit n (then every member has
  // finished reading unit n-1), which is the slot's next use at unit n+2.
  // SC1 cache-policy bit: device-coherent access; at width 768 also the
  // non-temporal bit, so that the exchange traffic (three 96 KiB slots per
  // member and unit) does not displace the weights from the L2
  constexpr int kCoherent = D > 256 ? (16 | 2) : 16;
  constexpr unsigned kEmpty = 0xFFFFFFFFu;  // never produced by arithmetic (canonical NaN differs)
  int nbar = 0;                             // evaluated units exchanged so far
  float* const xb = TEAM > 1 ? p.xchg + (size_t)tile * (3 * TEAM) * (R * D) : nullptr;
  const auto xr = __builtin_amdgcn_make_buffer_rsrc(xb, (short)0, TEAM > 1 ? 3 * TEAM * R * D * 4 : 0, 0x00020000);
  // byte offset of this lane's fragment (c, rb) in a member's slot, split
  // into a per-lane part (VGPR) and a constant part (SGPR), so that a wide
  // tile does not hold one offset register per fragment
  const auto xoff = [&](int slot, int m) { return ((slot * TEAM + m) * (R * D) + (w * RB * CBW * 64 + lane) * 4) * 4; };
  const auto xcst = [](int c, int rb) { return (rb * CBW + c) * 1024; };
  if constexpr (TEAM > 1) {
    // all three slots of this member start empty; one counter barrier makes
    // sure no member reads a slot before its owner has emptied it
    const u32x4 empty = {kEmpty, kEmpty, kEmpty, kEmpty};
#pragma unroll
    for (int sl = 0; sl < 3; ++sl)
#pragma unroll
      for (int c = 0; c < CBW; ++c)
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
          __builtin_amdgcn_raw_buffer_store_b128(empty, xr, xoff(sl, member), xcst(c, rb), kCoherent);
    __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
    __syncthreads();
    if (tid == 0) {
      unsigned* ctr = p.tctr + (size_t)tile * 16;
      __hip_atomic_fetch_add(ctr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      unsigned spins = 0;
      while (__hip_atomic_load(ctr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < (unsigned)TEAM) {
        if (__hip_atomic_load(p.derr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0u || ++spins > 4u * p.spin_limit) {
          __hip_atomic_store(p.derr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          s_abort = 1;
          break;
        }
        __builtin_amdgcn_s_sleep(1);
      }
    }
    __syncthreads();
    if (s_abort) return;
  }
  // element index of this lane's fragment (c, rb) in a unit's cache slot
  const auto cidx = [&](int unit, int c, int rb) {
    return (size_t)unit * (R * D) + ((size_t)((w * RB + rb) * CBW + c) * 64 + lane) * 4;
  };
  // Cache-policy bits of the residual-cache accesses (and of the layer
  // sums kept in cache slots and the memory tokens' keys and values).  At
  // width 768 a unit's weights exceed an XCD's L2 and a cached residual is
  // 48 KiB, so these reads and writes are non-temporal (evicted first) and
  // leave the L2 to the weights; at width 256 the default policy measured
  // faster.
  constexpr int CPOL = D > 256 ? 2 : 0;
  const auto cload = [&](int unit, int c, int rb) -> f32x4 {
    if constexpr (CE == 2) {
      const u32x2* q = reinterpret_cast<const u32x2*>(cbase + cidx(unit, c, rb) * 2);
      const u32x2 x = CPOL ? __builtin_nontemporal_load(q) : *q;
      return f16x4_to_f32(x[0], x[1]);
    } else {
      const f32x4* q = reinterpret_cast<const f32x4*>(cbase + cidx(unit, c, rb) * 4);
      return CPOL ? __builtin_nontemporal_load(q) : *q;
    }
  };
  const auto cstore = [&](int unit, int c, int rb, f32x4 v) {
    if constexpr (CE == 2) {
      u32x2* q = reinterpret_cast<u32x2*>(cbase + cidx(unit, c, rb) * 2);
      const u32x2 x = {f16x2_sat(v[0], v[1]), f16x2_sat(v[2], v[3])};
      if (CPOL) __builtin_nontemporal_store(x, q);
      else *q = x;
    } else {
      f32x4* q = reinterpret_cast<f32x4*>(cbase + cidx(unit, c, rb) * 4);
      if (CPOL) __builtin_nontemporal_store(v, q);
      else *q = v;
    }
  };
  const uint4* pk = p.pk;

  // embedding / head constants of this lane's columns (each lane writes and
  // later reads only its own LDS entries, so no barrier is needed)
  __shared__ uint4 s_win[EMB_LDS ? CB * 64 : 1], s_wout[EMB_LDS ? CB * 64 : 1];
  __shared__ f32x4 s_pb[PB_LDS ? CB * 64 : 1];
  __shared__ float s_lf[EMB_LDS ? 2 * D : 1];
  constexpr int KE = KEEP_EMB ? CBW : 1, KP = (KEEP_EMB || (EMB_LDS && !PB_LDS)) ? CBW : 1;
  uint4 win[KE], wout[KE];
  f32x4 pb[KP][KP > 1 ? RB : 1];
  float lfg[KE], lfb[KE];
  if constexpr (KEEP_EMB || EMB_LDS) {
#pragma unroll
    for (int c = 0; c < CBW; ++c) {
      const int col = (w * CBW + c) * 16 + lc, fi = (w * CBW + c) * 64 + lane;
      const uint4 wi = pk[p.pk_win + (size_t)fi], wo = pk[p.pk_wout + (size_t)fi];
      const float bi = raw[p.b_in + col];
      f32x4 pv[RB];
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int i = 0; i < 4; ++i) pv[rb][i] = bi + raw[p.P_act + (size_t)((rb * 16 + lq * 4 + i) % HZ) * D + col];
      const float g_ = raw[p.lnf_g + col], b_ = raw[p.lnf_b + col];
      if constexpr (EMB_LDS) {
        s_win[fi] = wi;
        s_wout[fi] = wo;
        if constexpr (PB_LDS) s_pb[fi] = pv[0];
        else pb[c][0] = pv[0];
        s_lf[col] = g_;
        s_lf[D + col] = b_;
      } else {
        win[c] = wi;
        wout[c] = wo;
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) pb[c][rb] = pv[rb];
        lfg[c] = g_;
        lfb[c] = b_;
      }
    }
  }

  f32x4 h[CBW][RB], mac[MAC_REG ? CBW : 1][MAC_REG ? RB : 1];
#pragma unroll
  for (int c = 0; c < (MAC_REG ? CBW : 1); ++c)
#pragma unroll
    for (int rb = 0; rb < (MAC_REG ? RB : 1); ++rb) mac[c][rb] = f32x4{0.f, 0.f, 0.f, 0.f};

  // LayerNorm gain/shift and output bias of the next unit to evaluate, for
  // this lane's columns (loaded one unit ahead)
  float nlg[CBW], nlb[CBW], nrb[CBW];
  // Width 256: every prefetch below is issued unconditionally (a merge of
  // an in-flight load with an older register value costs a wait for the
  // load at the merge).  Width 768 keeps the conditional form, which its
  // register allocation favours.
  constexpr bool UNCOND = D <= 256;
  int loaded_t = -1, loaded_u = -1;  // (step, unit) the prefetched parameters belong to
  const auto load_unit_params = [&](int tt, int unit) {
    loaded_t = tt;
    loaded_u = unit;
    const int ul = unit / 3, uu = unit - 3 * ul;
    const LayerOff& q = s_loff[ul];
    const uint32_t go = uu == 0 ? q.ln1_g : (uu == 1 ? q.ln2_g : q.ln3_g);
    const uint32_t bo = uu == 0 ? q.ln1_b : (uu == 1 ? q.ln2_b : q.ln3_b);
    const uint32_t ro = uu == 0 ? q.b_o : (uu == 1 ? q.b_o2 : q.b_2);
#pragma unroll
    for (int c = 0; c < CBW; ++c) {
      const int col = (w * CBW + c) * 16 + lc;
      nlg[c] = raw[go + col];
      nlb[c] = raw[bo + col];
      nrb[c] = raw[ro + col];
    }
  };
  // first unit any sample of the tile evaluates at step tt (U if none)
  const auto first_eval = [&](int tt) {
    uint64_t m = 0;
#pragma unroll
    for (int j = 0; j < SPT; ++j)
      if (smp[j] >= 0) m |= msk[(j * T + tt) * 3 + 0] & ~kMergedBit;
    return m ? __builtin_ctzll(m) : U;
  };

  // reuse-cache loads: a batch takes the NB lowest units of a mask
  const auto seg_mask = [](int lo, int hi) {
    const uint64_t lo_m = (lo >= 64) ? ~0ull : ((1ull << lo) - 1);
    const uint64_t hi_m = (hi >= 64) ? ~0ull : ((1ull << hi) - 1);
    return hi_m & ~lo_m;
  };
  uint64_t mru_cur[SPT];
  // The loads of a batch are issued unconditionally (an entry that is not
  // needed reads past the end of a buffer resource, which returns zeros
  // without a memory access), so that they are all in flight before the
  // first is consumed.
  const auto crs = __builtin_amdgcn_make_buffer_rsrc(cbase, (short)0, U * (R * D) * CE, 0x00020000);
  const auto issue_batch = [&](uint64_t& um, auto& ub, auto& v) {
#pragma unroll
    for (int q = 0; q < NB; ++q) {
      ub[q] = um ? __builtin_ctzll(um) : -1;
      um = um ? (um & (um - 1)) : 0ull;
    }
#pragma unroll
    for (int q = 0; q < NB; ++q)
#pragma unroll
      for (int c = 0; c < CBW; ++c)
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
          uint64_t mj = mru_cur[0];
#pragma unroll
          for (int jj = 1; jj < SPT; ++jj)
            if (jrow[rb] == jj) mj = mru_cur[jj];
          const bool use = ub[q] >= 0 && ((mj >> ub[q]) & 1ull);
          const int off = use ? (ub[q] * (R * D) + (w * RB * CBW * 64 + lane) * 4) * CE : 0x7FFFFFF0;
          const int cst = (rb * CBW + c) * 256 * CE;
          if constexpr (CE == 2) {
            const auto x = __builtin_amdgcn_raw_buffer_load_b64(crs, off, cst, CPOL);
            v[q][c][rb] = f16x4_to_f32(x[0], x[1]);
          } else {
            v[q][c][rb] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(crs, off, cst, CPOL));
          }
        }
  };

  constexpr int ZPT = (R * 16 + NT - 1) / NT;
  constexpr int MPWQ = (3 * GW / 16) / NW, MPWC = (GW / 16) / NW, MPWF = (FC / 16) / NW;
  constexpr int WPP = attn_waves_per_pair(NW, HG * RB, DH / 16);
  // fragments per wave requested ahead of each product (where registers allow)
  constexpr int PF = ((sizeof(AT) == 4 && RB > 1) || D > 256) ? 1 : 8;
  constexpr int NPQ = np_of<MPWQ, D / O::KF, INFL, PF>();
  constexpr int NPC = np_of<MPWC, D / O::KF, INFL, PF>();
  constexpr int NPF = np_of<MPWF, D / O::KF, INFL, PF>();
  constexpr int NP2A = np_of<CBW, GW / O::KF, INFL, PF>();
  constexpr int NP2F = np_of<CBW, FC / O::KF, INFL, PF>();

  for (int t = 0; t < T; ++t) {
    asm volatile("" : "+v"(lane), "+v"(lc), "+v"(lq));
    const int k = T - 1 - t;
    // schedule of this step for every sample slot
    uint64_t mev[SPT], mru[SPT], mst[SPT];
    bool mmg[SPT];
    uint64_t evT = 0, ruT = 0;
#pragma unroll
    for (int j = 0; j < SPT; ++j) {
      const bool live = smp[j] >= 0;
      const uint64_t e0 = live ? msk[(j * T + t) * 3 + 0] : 0ull;
      mmg[j] = (e0 & kMergedBit) != 0;
      mev[j] = e0 & ~kMergedBit;
      mru[j] = live ? msk[(j * T + t) * 3 + 1] : 0ull;
      mst[j] = live ? msk[(j * T + t) * 3 + 2] : 0ull;
      evT |= mev[j];
      ruT |= mru[j];
      mru_cur[j] = mru[j];
    }

    const auto pick = [&](const uint64_t (&m)[SPT], int j) {
      uint64_t v = m[0];
#pragma unroll
      for (int jj = 1; jj < SPT; ++jj)
        if (j == jj) v = m[jj];
      return v;
    };
    // noise added by this step's update (prefetched)
    // (unconditional form: always loaded from an existing slice; the last
    // step adds none, and a dead slot's rows, which read sample 0's noise,
    // are never output)
    float zpre[ZPT];
#pragma unroll
    for (int q = 0; q < ZPT; ++q) {
      const int it = tid + q * NT;
      if constexpr (UNCOND) {
        const int itc = it < R * A ? it : 0;
        const int row = itc / A, a = itc % A, s = smp[row / HZ];
        const int tn = t + 1 < T ? t + 1 : T - 1;
        zpre[q] = p.noise[(((size_t)tn * p.batch + (s >= 0 ? s : 0)) * HZ + (row % HZ)) * A + a];
      } else {
        zpre[q] = 0.f;
        if (k > 0 && it < R * A) {
          const int row = it / A, a = it % A, s = smp[row / HZ];
          if (s >= 0) zpre[q] = p.noise[(((size_t)(t + 1) * p.batch + s) * HZ + (row % HZ)) * A + a];
        }
      }
    }
    // parameters of this step's first evaluated unit (unconditional form:
    // always, unit 0 if none; else unless the previous step requested them)
    if constexpr (UNCOND) {
      load_unit_params(t, evT ? __builtin_ctzll(evT) : 0);
    } else {
      const int f = evT ? __builtin_ctzll(evT) : U;
      if (f < U && !(loaded_t == t && loaded_u == f)) load_unit_params(t, f);
    }
    // sampler constants and head bias of this step's update (prefetched)
    // (a lane-indexed vector load: a uniform scalar load would be waited for
    // by the next LDS access)
    const float ddl = UNCOND ? p.ddpm[(size_t)k * 8 + (lane & 7)] : (lane < 5 ? p.ddpm[(size_t)k * 8 + lane] : 0.f);
    float bout[ZPT];
#pragma unroll
    for (int q = 0; q < ZPT; ++q) {
      const int it = tid + q * NT;
      bout[q] = UNCOND ? raw[p.b_out + it % A] : (it < R * A ? raw[p.b_out + it % A] : 0.f);
    }
    // ---- embedding of the current sample on fp32 MFMA: h = (b_in + P_act) + x W_in^T
    {
      uint4 xf[RB];
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) xf[rb] = *reinterpret_cast<const uint4*>(xs + (rb * 16 + lc) * 16 + lq * 4);
#pragma unroll
      for (int c = 0; c < CBW; ++c) {
        uint4 wv;
        if constexpr (EMB_LDS) wv = s_win[(w * CBW + c) * 64 + lane];
        else if constexpr (KEEP_EMB) wv = win[c];
        else wv = pk[p.pk_win + (size_t)(w * CBW + c) * 64 + lane];
        const int col = (w * CBW + c) * 16 + lc;
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
          f32x4 acc;
          if constexpr (PB_LDS) {
            acc = s_pb[(w * CBW + c) * 64 + lane];
          } else if constexpr (KEEP_EMB || EMB_LDS) {
            acc = pb[c][rb];
          } else {
            const float bi = raw[p.b_in + col];
#pragma unroll
            for (int i = 0; i < 4; ++i) acc[i] = bi + raw[p.P_act + (size_t)((rb * 16 + lq * 4 + i) % HZ) * D + col];
          }
          OF::mma(acc, xf[rb], wv);
          h[c][rb] = acc;
        }
      }
    }

    // ---- the cacheable units (Eq. 1)
    int b = 0;
    while (true) {
      const uint64_t rest = evT >> b;
      const int e = rest ? b + __builtin_ctzll(rest) : U;
      // reused residuals of the units in [b, e), in unit order, loaded in
      // batches of NB units
      {
        uint64_t um = ruT & seg_mask(b, e);
        while (um) {
          int ub[NB];
          f32x4 v[NB][CBW][RB];
          issue_batch(um, ub, v);
#pragma unroll
          for (int q = 0; q < NB; ++q)
#pragma unroll
            for (int c = 0; c < CBW; ++c)
#pragma unroll
              for (int rb = 0; rb < RB; ++rb) h[c][rb] += v[q][c][rb];
        }
      }
      if (e >= U) break;

      // ---- evaluate unit e for the tile
      asm volatile("" : "+v"(lane), "+v"(lc), "+v"(lq));
      const int l = e / 3, u = e - 3 * l;
      const LayerOff lo = s_loff[l];
      const PackOff po = s_poff[l];
      float lg[CBW], lb[CBW], rbias[CBW];
#pragma unroll
      for (int c = 0; c < CBW; ++c) {
        lg[c] = nlg[c];
        lb[c] = nlb[c];
        rbias[c] = nrb[c];
      }
      // request the parameters of the next evaluated unit (this step or the
      // next) now, so that they have the whole unit to arrive
      const auto request_next_params = [&]() {
        const uint64_t later = (e + 1 < 64) ? (evT >> (e + 1)) : 0ull;
        if constexpr (UNCOND) {
          // this unit's own parameters again when no later unit of the
          // step is evaluated (the next step loads its first)
          load_unit_params(t, later ? e + 1 + __builtin_ctzll(later) : e);
        } else if (later) load_unit_params(t, e + 1 + __builtin_ctzll(later));
        else if (t + 1 < T) {
          const int f = first_eval(t + 1);
          if (f < U) load_unit_params(t + 1, f);
        }
      };
      request_next_params();
      const auto gcb_sa = [&](int g) {
        return [=](int m) {
          const int iloc = w + NW * m, part = iloc / (GW / 16), within = iloc % (GW / 16);
          return part * CB + g * (GW / 16) + within;
        };
      };
      const auto gcb_ca = [&](int g) { return [=](int m) { return g * (GW / 16) + w + NW * m; }; };
      const auto gcb_ff = [&](int ch) { return [=](int m) { return ch * (FC / 16) + w + NW * m; }; };
      const auto own = [&](int m) { return w * CBW + m; };
      f32x4 r[CBW][RB];
#pragma unroll
      for (int c = 0; c < CBW; ++c)
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) r[c][rb] = f32x4{0.f, 0.f, 0.f, 0.f};
      // LayerNorm of the unit's input into the stage-1 operand buffer
      const auto layer_norm_to_xa = [&]() {
        float mu[RB][4], rs[RB][4];
        ln_stats<C>(h, red, mu, rs, w, lc, lq);
#pragma unroll
        for (int c = 0; c < CBW; ++c) {
          const int col = (w * CBW + c) * 16 + lc;
#pragma unroll
          for (int rb = 0; rb < RB; ++rb)
#pragma unroll
            for (int i = 0; i < 4; ++i)
              O::store(xa, LDA, rb * 16 + lq * 4 + i, col, (h[c][rb][i] - mu[rb][i]) * rs[rb][i] * lg[c] + lb[c]);
        }
        __syncthreads();
      };

      if (u == 0) {
        // ---------------- self-attention unit (causal over the action tokens)
        uint4 b1q[NPQ][MPWQ];  // stage-1 weights of the first chunk, requested before the LayerNorm
        gemm_pref<NPQ, MPWQ>(b1q, pk + po.qkv, D / O::KF, 0, gcb_sa(member), lane);
        layer_norm_to_xa();
        for (int g = member; g < NH / HG; g += TEAM) {
          asm volatile("" : "+v"(lane), "+v"(lc), "+v"(lq));
          f32x4 y[MPWQ][RB];
#pragma unroll
          for (int m = 0; m < MPWQ; ++m)
#pragma unroll
            for (int rb = 0; rb < RB; ++rb) y[m][rb] = f32x4{0.f, 0.f, 0.f, 0.f};
          float bq[MPWQ];  // stage-1 biases, requested before the GEMM so their latency is hidden
#pragma unroll
          for (int m = 0; m < MPWQ; ++m) bq[m] = raw[lo.b_qkv + gcb_sa(g)(m) * 16 + lc];
          gemm_run<AT, RB, MPWQ, D / O::KF, INFL, NPQ>(y, xa, LDA, pk + po.qkv, D / O::KF, 0, gcb_sa(g), lane, b1q);
          uint4 b2[NP2A][CBW];
          gemm_pref<NP2A, CBW>(b2, pk + po.o, D / O::KF, g * (GW / O::KF), own, lane);
#pragma unroll
          for (int m = 0; m < MPWQ; ++m) {
            const int loc = (w + NW * m) * 16 + lc;
#pragma unroll
            for (int rb = 0; rb < RB; ++rb)
#pragma unroll
              for (int i = 0; i < 4; ++i) ybuf[(rb * 16 + lq * 4 + i) * LDY + loc] = y[m][rb][i] + bq[m];
          }
          __syncthreads();
          // scores, softmax and values on fp32 MFMA tiles: WPP waves per
          // (head, query block), each with DH / 16 / WPP value column blocks
          for (int it = w; it < HG * RB * WPP; it += NW) {
            const int pr = it / WPP, part = it % WPP;
            const int hh = pr % HG, ib = pr / HG;
            const int jb0 = (HZ >= 16) ? ((ib * 16) / HZ) * (HZ / 16) : ib;
            f32x4 s[NJB];
#pragma unroll
            for (int jj = 0; jj < NJB; ++jj) {
              s[jj] = f32x4{0.f, 0.f, 0.f, 0.f};
              const int jb = jb0 + jj;
              if (jb <= ib)
                s[jj] = qk_tile<DH>(ybuf + (ib * 16 + lc) * LDY + hh * DH, ybuf + (jb * 16 + lc) * LDY + GW + hh * DH,
                                    true, lq);
            }
            float sm[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int gi = ib * 16 + lq * 4 + i;
              float m = -INFINITY;
#pragma unroll
              for (int jj = 0; jj < NJB; ++jj) {
                const int gj = (jb0 + jj) * 16 + lc;
                const bool ok = (gj <= gi) && (gj / HZ == gi / HZ);
                s[jj][i] = ok ? s[jj][i] * (kScale * kLog2e) : -INFINITY;
                m = fmaxf(m, s[jj][i]);
              }
              m = row16_max(m);
              float su = 0.f;
#pragma unroll
              for (int jj = 0; jj < NJB; ++jj) {
                const float ev = (s[jj][i] == -INFINITY) ? 0.f : fast_exp2(s[jj][i] - m);
                s[jj][i] = ev;
                su += ev;
              }
              sm[i] = row16_sum(su);
            }
            float* sc = pw + w * PWN;
#pragma unroll
            for (int jj = 0; jj < NJB; ++jj)
#pragma unroll
              for (int i = 0; i < 4; ++i) sc[(jj * 16 + lq * 4 + i) * PS + lc] = s[jj][i] * fast_rcp(sm[i]);
            wave_lds_sync();
#pragma unroll
            for (int cbi = 0; cbi < DH / 16 / WPP; ++cbi) {
              const int cb = part * (DH / 16 / WPP) + cbi;
              f32x4 o = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
              for (int jj = 0; jj < NJB; ++jj) {
                const int jb = jb0 + jj;
                if (jb <= ib) {
#pragma unroll
                  for (int kk = 0; kk < 4; ++kk) {
                    const float a = sc[(jj * 16 + lc) * PS + 4 * kk + lq];
                    const float v = ybuf[(jb * 16 + 4 * kk + lq) * LDY + 2 * GW + hh * DH + cb * 16 + lc];
                    o = mfma4(a, v, o);
                  }
                }
              }
#pragma unroll
              for (int i = 0; i < 4; ++i) O::store(zbuf, LDZ, ib * 16 + lq * 4 + i, hh * DH + cb * 16 + lc, o[i]);
            }
            wave_lds_sync();
          }
          // the next head group's first stage-1 k-steps stream in during this output product
          if (g + TEAM < NH / HG) gemm_pref<NPQ, MPWQ>(b1q, pk + po.qkv, D / O::KF, 0, gcb_sa(g + TEAM), lane);
          __syncthreads();
          gemm_run<AT, RB, CBW, GW / O::KF, INFL, NP2A>(r, zbuf, LDZ, pk + po.o, D / O::KF, g * (GW / O::KF), own, lane,
                                                       b2);
        }
      } else if (C::FOLD && fold && u == 1) {
        if constexpr (C::FOLD) {
          // ---------------- cross-attention unit, folded (time token + observation tokens)
          // Score columns n = j * NH + h (memory token j, head h) of the row
          // block's sample, padded to 16 with zero columns.  Every team
          // member evaluates the whole unit (no partials to exchange).
          constexpr int KPW = (D / O::KF) / NW, VQ = O::VE / 4, SJ = 16 / NH;
          static_assert(KPW * NW == D / O::KF && SJ * NH == 16, "folded cross-attention split");
          const float* trec = p.tfold + ((size_t)k * L + l) * REC;
          // record of memory token j of the sample in row block rb, and
          // whether it exists (else the time-token record stands in and the
          // loaded values are replaced by zeros)
          const auto rec = [&](int rb, int j, bool& ok) -> const float* {
            const int s_ = smp[(rb * 16) / HZ];
            ok = s_ >= 0 && j < S;
            return (ok && j > 0) ? okv + (((size_t)s_ * L + l) * nobs + (j - 1)) * REC : trec;
          };
          const f32x4 zero4 = {0.f, 0.f, 0.f, 0.f};
          // u columns of this wave's k-range (the B operand of the scores)
          // (loaded values are zeroed where they do not exist only at their
          // use, after the LayerNorm, so that no wait for them sits before
          // its barriers)
          f32x4 ub[RB][KPW][VQ];
          bool ubok[RB];
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) {
            const float* q = rec(rb, lc / NH, ubok[rb]) + (lc % NH) * D + w * KPW * O::KF + lq * O::VE;
#pragma unroll
            for (int kf = 0; kf < KPW; ++kf)
#pragma unroll
              for (int v = 0; v < VQ; ++v) ub[rb][kf][v] = *reinterpret_cast<const f32x4*>(q + kf * O::KF + 4 * v);
          }
          // w vectors of the row blocks' samples, staged through LDS
          constexpr int WQN = RB * 16 * D / 4, WQ = (WQN + NT - 1) / NT;
          f32x4 wv[WQ];
          bool wvok[WQ];
#pragma unroll
          for (int q = 0; q < WQ; ++q) {
            const int it = tid + q * NT;
            const int f = it * 4, rb = f / (16 * D), n = (f / D) % 16, c = f % D;
            bool ok = false;
            const float* src = it < WQN ? rec(rb, n / NH, ok) : trec;
            wv[q] = *reinterpret_cast<const f32x4*>(src + NH * D + (n % NH) * D + c);
            wvok[q] = it < WQN && ok;
          }
          // c terms of the softmax thread's (row, head)
          float cqv[SJ];
          bool cqok[SJ];
          {
            const int r = tid / NH, hd = tid % NH;
#pragma unroll
            for (int j = 0; j < SJ; ++j) {
              bool ok = false;
              const float* src = tid < R * NH ? rec(r >> 4, j, ok) : trec;
              cqv[j] = src[2 * NH * D + hd];
              cqok[j] = tid < R * NH && ok;
            }
          }
          layer_norm_to_xa();
          // partial scores over this wave's k-range on MFMA
          float* const sb = ybuf;                    // [NW][RB][64 lanes][4]
          float* const pb = ybuf + NW * RB * 256;    // [16][R] probabilities (column n, row)
          float* const wst = pb + 16 * R;            // [RB][16][D] w vectors
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) {
            f32x4 acc = zero4;
#pragma unroll
            for (int kf = 0; kf < KPW; ++kf) {
              const uint4 a =
                  *reinterpret_cast<const uint4*>(xa + (rb * 16 + lc) * LDA + (w * KPW + kf) * O::KF + lq * O::VE);
              uint4 bq;
              if constexpr (sizeof(AT) == 2) {
                const f32x4 x0 = ubok[rb] ? ub[rb][kf][0] : zero4, x1 = ubok[rb] ? ub[rb][kf][1] : zero4;
                bq.x = bf16x2_rne(x0[0], x0[1]);
                bq.y = bf16x2_rne(x0[2], x0[3]);
                bq.z = bf16x2_rne(x1[0], x1[1]);
                bq.w = bf16x2_rne(x1[2], x1[3]);
              } else {
                bq = __builtin_bit_cast(uint4, ubok[rb] ? ub[rb][kf][0] : zero4);
              }
              O::mma(acc, a, bq);
            }
            *reinterpret_cast<f32x4*>(sb + ((w * RB + rb) * 64 + lane) * 4) = acc;
          }
#pragma unroll
          for (int q = 0; q < WQ; ++q)
            if (tid + q * NT < WQN) *reinterpret_cast<f32x4*>(wst + (tid + q * NT) * 4) = wvok[q] ? wv[q] : zero4;
          __syncthreads();
          // softmax over the memory tokens of each (row, head)
          if (tid < R * NH) {
            const int r = tid / NH, hd = tid % NH, rb = r >> 4, rr = r & 15;
            float sc[SJ], mx = -INFINITY;
#pragma unroll
            for (int j = 0; j < SJ; ++j) {
              const int n = j * NH + hd;
              float a = 0.f;
#pragma unroll
              for (int ww = 0; ww < NW; ++ww) a += sb[((ww * RB + rb) * 64 + (rr >> 2) * 16 + n) * 4 + (rr & 3)];
              sc[j] = j < S ? (a + (cqok[j] ? cqv[j] : 0.f)) * (kScale * kLog2e) : -INFINITY;
              mx = fmaxf(mx, sc[j]);
            }
            float den = 0.f;
#pragma unroll
            for (int j = 0; j < SJ; ++j) {
              sc[j] = j < S ? fast_exp2(sc[j] - mx) : 0.f;
              den += sc[j];
            }
            const float inv = fast_rcp(den);
#pragma unroll
            for (int j = 0; j < SJ; ++j) pb[(j * NH + hd) * R + r] = sc[j] * inv;
          }
          __syncthreads();
          // output: r = P W over the 16 columns (padding columns are zero),
          // four k-steps of fp32 MFMA per column block
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) {
            float pa[4];
#pragma unroll
            for (int kk = 0; kk < 4; ++kk) pa[kk] = pb[(4 * kk + lq) * R + rb * 16 + lc];
#pragma unroll
            for (int c = 0; c < CBW; ++c)
#pragma unroll
              for (int kk = 0; kk < 4; ++kk)
                r[c][rb] = mfma4(pa[kk], wst[(rb * 16 + 4 * kk + lq) * D + (w * CBW + c) * 16 + lc], r[c][rb]);
          }
        }
      } else if (u == 1) {
        // ---------------- cross-attention unit (time token + observation tokens)
        uint4 b1c[NPC][MPWC];
        gemm_pref<NPC, MPWC>(b1c, pk + po.q, D / O::KF, 0, gcb_ca(member), lane);
        // memory keys/values of a head group: time token + observation tokens
        constexpr int KVN = SPT * SMAX * 2 * GW, KVQ = (KVN + NT - 1) / NT;
        float kvv[KVQ];
        bool kvok[KVQ];
        // branch-free: every lane loads (entries outside the memory tokens
        // read the time-token row and are zeroed), so the loads issue back
        // to back instead of one guarded branch each
        const auto load_kv = [&](int g) {
          const float* trow = p.tkv + ((size_t)k * L + l) * (2 * D);
#pragma unroll
          for (int q = 0; q < KVQ; ++q) {
            const int it = tid + q * NT;
            const int col = it % (2 * GW), sm_ = (it / (2 * GW)) % SMAX, j = it / (2 * GW * SMAX);
            const int gcol = col < GW ? g * GW + col : D + g * GW + (col - GW);
            const int s_ = smp[j < SPT ? j : 0];
            const bool ok = it < KVN && sm_ < S && s_ >= 0;
            const bool obs_tok = ok && sm_ > 0;
            // 32-bit offsets: the observation K/V of a member is below 2^31 floats
            const int off = obs_tok ? ((s_ * L + l) * nobs + (sm_ - 1)) * (2 * D) + gcol : gcol;
            const float* src = &(obs_tok ? okv : trow)[off];
            kvv[q] = CPOL ? __builtin_nontemporal_load(src) : *src;  // read once per evaluation
            kvok[q] = ok;
          }
        };
        load_kv(member);
        layer_norm_to_xa();
        for (int g = member; g < NH / HG; g += TEAM) {
          asm volatile("" : "+v"(lane), "+v"(lc), "+v"(lq));
          if (g != member) load_kv(g);
          f32x4 y[MPWC][RB];
#pragma unroll
          for (int m = 0; m < MPWC; ++m)
#pragma unroll
            for (int rb = 0; rb < RB; ++rb) y[m][rb] = f32x4{0.f, 0.f, 0.f, 0.f};
          float bq[MPWC];
#pragma unroll
          for (int m = 0; m < MPWC; ++m) bq[m] = raw[lo.b_q + gcb_ca(g)(m) * 16 + lc];
          gemm_run<AT, RB, MPWC, D / O::KF, INFL, NPC>(y, xa, LDA, pk + po.q, D / O::KF, 0, gcb_ca(g), lane, b1c);
          uint4 b2[NP2A][CBW];
          gemm_pref<NP2A, CBW>(b2, pk + po.o2, D / O::KF, g * (GW / O::KF), own, lane);
#pragma unroll
          for (int m = 0; m < MPWC; ++m) {
            const int loc = (w + NW * m) * 16 + lc;
#pragma unroll
            for (int rb = 0; rb < RB; ++rb)
#pragma unroll
              for (int i = 0; i < 4; ++i) ybuf[(rb * 16 + lq * 4 + i) * LDY + loc] = y[m][rb][i] + bq[m];
          }
#pragma unroll
          for (int q = 0; q < KVQ; ++q)
            if (tid + q * NT < KVN) kvbuf[tid + q * NT] = kvok[q] ? kvv[q] : 0.f;
          __syncthreads();
          // Each row attends to the S = 1 + n_obs memory tokens of its own
          // sample: few keys, so the products run on the vector ALUs (fp32
          // MFMA tiles would be mostly padding).  Lane = (row, quarter of the
          // head's dims); a row's four lanes are adjacent, so the score
          // reduction is two quad shuffles.  WPP waves per (head, row block)
          // each produce DH / WPP output dims.
          for (int it = w; it < HG * RB * WPP; it += NW) {
            const int pr = it / WPP, part = it % WPP;
            const int hh = pr % HG, ib = pr / HG;
            const int qr = lane >> 2, qg = lane & 3;  // row in the block, dim quarter
            const int row = ib * 16 + qr, js = row / HZ;
            constexpr int DQ = DH / 4, OD = DH / 4 / WPP;
            const float* qrow = ybuf + row * LDY + hh * DH + qg * DQ;
            const int c0 = hh * DH + part * (DH / WPP) + qg * OD;  // first output column of this lane
            // one pass over the keys with a running maximum (online softmax)
            float mx = -INFINITY, den = 0.f, o[OD];
#pragma unroll
            for (int d = 0; d < OD; ++d) o[d] = 0.f;
#pragma unroll 1
            for (int j = 0; j < S; ++j) {
              const float* kr = kvbuf + (js * SMAX + j) * (2 * GW) + hh * DH + qg * DQ;
              float a = 0.f;
#pragma unroll
              for (int d4 = 0; d4 < DQ / 4; ++d4) {
                const f32x4 kv = *reinterpret_cast<const f32x4*>(kr + 4 * d4);
                const f32x4 qv = *reinterpret_cast<const f32x4*>(qrow + 4 * d4);
                a += qv[0] * kv[0] + qv[1] * kv[1] + qv[2] * kv[2] + qv[3] * kv[3];
              }
              a += dpp_mov<0xB1>(a);  // sum over the row's four lanes
              a += dpp_mov<0x4E>(a);
              a *= kScale * kLog2e;
              const float mn = fmaxf(mx, a);
              const float sc = fast_exp2(mx - mn), pj = fast_exp2(a - mn);
              den = den * sc + pj;
              mx = mn;
              const float* vr = kvbuf + (js * SMAX + j) * (2 * GW) + GW + c0;
#pragma unroll
              for (int d4 = 0; d4 < OD / 4; ++d4) {
                const f32x4 vv = *reinterpret_cast<const f32x4*>(vr + 4 * d4);
#pragma unroll
                for (int e = 0; e < 4; ++e) o[4 * d4 + e] = o[4 * d4 + e] * sc + pj * vv[e];
              }
            }
            const float inv = fast_rcp(den);
#pragma unroll
            for (int d = 0; d < OD; ++d) O::store(zbuf, LDZ, row, c0 + d, o[d] * inv);
          }
          if (g + TEAM < NH / HG) gemm_pref<NPC, MPWC>(b1c, pk + po.q, D / O::KF, 0, gcb_ca(g + TEAM), lane);
          __syncthreads();
          gemm_run<AT, RB, CBW, GW / O::KF, INFL, NP2A>(r, zbuf, LDZ, pk + po.o2, D / O::KF, g * (GW / O::KF), own,
                                                       lane, b2);
        }
      } else {
        // ---------------- feed-forward unit, d_ff streamed in chunks of FC
        uint4 b1f[NPF][MPWF];
        gemm_pref<NPF, MPWF>(b1f, pk + po.w1, D / O::KF, 0, gcb_ff(member), lane);
        layer_norm_to_xa();
        for (int ch = member; ch < DFF / FC; ch += TEAM) {
          asm volatile("" : "+v"(lane), "+v"(lc), "+v"(lq));
          AT* const zb = zbuf + (ZB2 ? (((ch - member) / TEAM) & 1) * (R * LDZ) : 0);
          f32x4 y[MPWF][RB];
#pragma unroll
          for (int m = 0; m < MPWF; ++m)
#pragma unroll
            for (int rb = 0; rb < RB; ++rb) y[m][rb] = f32x4{0.f, 0.f, 0.f, 0.f};
          float b1v[MPWF];
#pragma unroll
          for (int m = 0; m < MPWF; ++m) b1v[m] = raw[lo.b_1 + ch * FC + (w + NW * m) * 16 + lc];
          gemm_run<AT, RB, MPWF, D / O::KF, INFL, NPF>(y, xa, LDA, pk + po.w1, D / O::KF, 0, gcb_ff(ch), lane, b1f);
          uint4 b2[NP2F][CBW];
          gemm_pref<NP2F, CBW>(b2, pk + po.w2, DFF / O::KF, ch * (FC / O::KF), own, lane);
#pragma unroll
          for (int m = 0; m < MPWF; ++m) {
            const int loc = (w + NW * m) * 16 + lc;
#pragma unroll
            for (int rb = 0; rb < RB; ++rb)
#pragma unroll
              for (int i = 0; i < 4; ++i)
                O::store(zb, LDZ, rb * 16 + lq * 4 + i, loc, gelu_erf(y[m][rb][i] + b1v[m]));
          }
          // the next chunk's first stage-1 k-steps stream in during this chunk's second product
          if (ch + TEAM < DFF / FC) gemm_pref<NPF, MPWF>(b1f, pk + po.w1, D / O::KF, 0, gcb_ff(ch + TEAM), lane);
          __syncthreads();
          gemm_run<AT, RB, CBW, FC / O::KF, INFL, NP2F>(r, zb, LDZ, pk + po.w2, DFF / O::KF, ch * (FC / O::KF), own,
                                                        lane, b2);
          // (with one buffer, the next chunk's GELU outputs wait for every
          // wave's reads of this one)
          if constexpr (!ZB2) __syncthreads();
        }
      }
      if constexpr (TEAM > 1) if (!(fold && u == 1)) {
        // Sum the members' partial residuals in member order, so that every
        // member obtains the same bits.  The partials travel through memory
        // with device-coherent (SC1) buffer stores and loads, which leave no
        // stale or dirty lines in the per-XCD caches (the weight stream stays
        // in L2).  Each thread waits only for the words it sums: a word is
        // ready once it no longer holds the sentinel.  Waits are bounded;
        // on a timeout the device error flag is set and every later wait
        // ends at once, so the kernel always finishes.
        const int cur = nbar % 3, prev = (nbar + 2) % 3;
        __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): the reset of this slot (one unit ago) has landed
#pragma unroll
        for (int c = 0; c < CBW; ++c)
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) {
            u32x4 v = __builtin_bit_cast(u32x4, r[c][rb]);
#pragma unroll
            for (int q = 0; q < 4; ++q) v[q] = v[q] == kEmpty ? 0x7FC00000u : v[q];
            if (!(p.withhold && member == 0))
              __builtin_amdgcn_raw_buffer_store_b128(v, xr, xoff(cur, member), xcst(c, rb), kCoherent);
          }
        // bounded wait for every word of `v` (loaded by `load`) to be written;
        // polls back to back (each is a memory round trip), the error flag
        // and the limit are checked every 32 polls
        const auto poll = [&](auto& v, auto load, auto ready) {
          unsigned spins = 0;
          while (true) {
            load(v);
            if (ready(v)) break;
            if ((++spins & 31u) == 0u &&
                (__hip_atomic_load(p.derr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0u || spins > p.spin_limit)) {
              __hip_atomic_store(p.derr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
              break;
            }
          }
        };
        const auto full = [&](const u32x4& x) {
          return x[0] != kEmpty && x[1] != kEmpty && x[2] != kEmpty && x[3] != kEmpty;
        };
        if constexpr (TEAM == 2) {
          // two operands: r + other is the same sum on both members
          // (commutative), so only the other member's partial is held, a few
          // column blocks at a time
          constexpr int XC = (CBW * RB > 4) ? (4 / RB > 0 ? 4 / RB : 1) : CBW;
          static_assert(CBW % XC == 0, "exchange chunks");
          const int other = 1 - member;
#pragma unroll
          for (int c0 = 0; c0 < CBW; c0 += XC) {
            u32x4 part[XC][RB];
            poll(part,
                 [&](u32x4 (&v)[XC][RB]) {
#pragma unroll
                   for (int c = 0; c < XC; ++c)
#pragma unroll
                     for (int rb = 0; rb < RB; ++rb)
                       v[c][rb] = __builtin_amdgcn_raw_buffer_load_b128(xr, xoff(cur, other), xcst(c0 + c, rb), kCoherent);
                 },
                 [&](const u32x4 (&v)[XC][RB]) {
                   bool ok = true;
#pragma unroll
                   for (int c = 0; c < XC; ++c)
#pragma unroll
                     for (int rb = 0; rb < RB; ++rb) ok = ok && full(v[c][rb]);
                   return ok;
                 });
#pragma unroll
            for (int c = 0; c < XC; ++c)
#pragma unroll
              for (int rb = 0; rb < RB; ++rb) r[c0 + c][rb] += __builtin_bit_cast(f32x4, part[c][rb]);
          }
        } else {
          // more operands: every member sums the partials in member order
          u32x4 part[TEAM][CBW][RB];
          unsigned pending = ((1u << TEAM) - 1u) & ~(1u << member);
          poll(part,
               [&](u32x4 (&v)[TEAM][CBW][RB]) {
#pragma unroll
                 for (int m = 0; m < TEAM; ++m)
                   if (pending >> m & 1u) {
#pragma unroll
                     for (int c = 0; c < CBW; ++c)
#pragma unroll
                       for (int rb = 0; rb < RB; ++rb)
                         v[m][c][rb] = __builtin_amdgcn_raw_buffer_load_b128(xr, xoff(cur, m), xcst(c, rb), kCoherent);
                   }
               },
               [&](const u32x4 (&v)[TEAM][CBW][RB]) {
#pragma unroll
                 for (int m = 0; m < TEAM; ++m)
                   if (pending >> m & 1u) {
                     bool ok = true;
#pragma unroll
                     for (int c = 0; c < CBW; ++c)
#pragma unroll
                       for (int rb = 0; rb < RB; ++rb) ok = ok && full(v[m][c][rb]);
                     if (ok) pending &= ~(1u << m);
                   }
                 return pending == 0u;
               });
#pragma unroll
          for (int c = 0; c < CBW; ++c)
#pragma unroll
            for (int rb = 0; rb < RB; ++rb) {
              f32x4 acc = member == 0 ? r[c][rb] : __builtin_bit_cast(f32x4, part[0][c][rb]);
#pragma unroll
              for (int m = 1; m < TEAM; ++m)
                acc += member == m ? r[c][rb] : __builtin_bit_cast(f32x4, part[m][c][rb]);
              r[c][rb] = acc;
            }
        }
        // every member has read the partials of the previous unit: empty
        // this member's slot of it for its next use
        const u32x4 empty = {kEmpty, kEmpty, kEmpty, kEmpty};
#pragma unroll
        for (int c = 0; c < CBW; ++c)
#pragma unroll
          for (int rb = 0; rb < RB; ++rb)
            __builtin_amdgcn_raw_buffer_store_b128(empty, xr, xoff(prev, member), xcst(c, rb), kCoherent);
        ++nbar;
      }
#pragma unroll
      for (int c = 0; c < CBW; ++c)
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) r[c][rb] += rbias[c];

      // Layer sums kept in memory (tiles too wide for registers): the
      // unit's partial layer sums are read in one batch through the cache's
      // buffer resource before any is written (element by element, every
      // load would wait for the store before it); an entry that is not
      // needed reads past the end of the resource (zeros, no memory access)
      const int lacc_base = CE == 4 ? (int)(cidx(3 * l + 2, 0, 0) * 4) : (int)((size_t)(3 * l) * (R * D) * 2 + cidx(0, 0, 0) * 4);
      const auto lacc_cst = [](int c, int rb) { return (rb * CBW + c) * 1024; };
      f32x4 lsum[MAC_REG ? 1 : CBW][MAC_REG ? 1 : RB];
      if constexpr (!MAC_REG) {
#pragma unroll
        for (int c = 0; c < CBW; ++c)
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) {
            const int j = jrow[rb];
            bool mg = mmg[0];
#pragma unroll
            for (int jj = 1; jj < SPT; ++jj)
              if (j == jj) mg = mmg[jj];
            const bool need = u > 0 && mg && ((pick(mev, j) >> e) & 1ull);
            lsum[c][rb] = __builtin_bit_cast(
                f32x4, __builtin_amdgcn_raw_buffer_load_b128(crs, need ? lacc_base : 0x7FFFFFF0, lacc_cst(c, rb), CPOL));
          }
      }
      // Eq. 1 per sample at unit e: evaluated residual (and cache refresh) or
      // the residual cached at the unit's most recent refresh.
#pragma unroll
      for (int c = 0; c < CBW; ++c)
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
          const int j = jrow[rb];
          const uint64_t bit = 1ull << e;
          bool mg = mmg[0];
#pragma unroll
          for (int jj = 1; jj < SPT; ++jj)
            if (j == jj) mg = mmg[jj];
          if (pick(mev, j) & bit) {
            const f32x4 v = r[c][rb];
            if constexpr (MAC_REG) {
              if (mg) mac[c][rb] = (u == 0) ? v : mac[c][rb] + v;
              if (pick(mst, j) & bit) cstore(e, c, rb, mg ? mac[c][rb] : v);
            } else if (mg) {
              // layer sum accumulated in memory, in fp32: in the FFN
              // position's slot (fp32 caches) or across the SA and CA slots,
              // which a merged layer leaves unused (fp16 caches; one sample
              // per tile, so no other sample's rows share them); the sum of
              // the three residuals is stored at the FFN position
              const f32x4 sum = (u == 0) ? v : lsum[c][rb] + v;
              if (CE == 4 || u < 2) {
                __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, sum), crs, lacc_base, lacc_cst(c, rb), CPOL);
              } else if (pick(mst, j) & bit) {
                if constexpr (CE == 2)
                  __builtin_amdgcn_raw_buffer_store_b64(u32x2{f16x2_sat(sum[0], sum[1]), f16x2_sat(sum[2], sum[3])}, crs,
                                                        (int)(cidx(e, 0, 0) * 2), (rb * CBW + c) * 512, CPOL);
                else
                  cstore(e, c, rb, sum);
              }
            } else if (pick(mst, j) & bit) {
              cstore(e, c, rb, v);
            }
            h[c][rb] += v;
            if (p.acts != nullptr && member == 0) {
              // activation record of the uncached policy (Sec. 3.3): a[sample][unit][step][H][d]
              float* ap = p.acts + (((size_t)smp[j] * U + e) * T + t) * (HZ * D) + (w * CBW + c) * 16 + lc;
#pragma unroll
              for (int i = 0; i < 4; ++i) ap[(size_t)((rb * 16 + lq * 4 + i) % HZ) * D] = v[i];
            }
          } else if (pick(mru, j) & bit) {
            h[c][rb] += cload(e, c, rb);
          }
        }
      b = e + 1;
    }

    // ---- head (final LayerNorm + linear on fp32 MFMA) and DDPM update
    {
      float mu[RB][4], rs[RB][4];
      ln_stats<C>(h, red, mu, rs, w, lc, lq);
      f32x4 eacc[RB];
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) eacc[rb] = f32x4{0.f, 0.f, 0.f, 0.f};
      float* sc = pw + w * PWN;
#pragma unroll
      for (int c = 0; c < CBW; ++c) {
        float g_, b_;
        if constexpr (EMB_LDS) {
          g_ = s_lf[(w * CBW + c) * 16 + lc];
          b_ = s_lf[D + (w * CBW + c) * 16 + lc];
        } else if constexpr (KEEP_EMB) {
          g_ = lfg[c];
          b_ = lfb[c];
        } else {
          const int col = (w * CBW + c) * 16 + lc;
          g_ = raw[p.lnf_g + col];
          b_ = raw[p.lnf_b + col];
        }
        uint4 wo;
        if constexpr (EMB_LDS) wo = s_wout[(w * CBW + c) * 64 + lane];
        else if constexpr (KEEP_EMB) wo = wout[c];
        else wo = pk[p.pk_wout + (size_t)(w * CBW + c) * 64 + lane];
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
#pragma unroll
          for (int i = 0; i < 4; ++i)
            sc[(rb * 16 + lq * 4 + i) * PS + lc] = (h[c][rb][i] - mu[rb][i]) * rs[rb][i] * g_ + b_;
        wave_lds_sync();
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
          const float* ar = sc + (rb * 16 + lc) * PS + lq;
          eacc[rb] = mfma4(ar[0], __uint_as_float(wo.x), eacc[rb]);
          eacc[rb] = mfma4(ar[4], __uint_as_float(wo.y), eacc[rb]);
          eacc[rb] = mfma4(ar[8], __uint_as_float(wo.z), eacc[rb]);
          eacc[rb] = mfma4(ar[12], __uint_as_float(wo.w), eacc[rb]);
        }
        wave_lds_sync();
      }
      float* epsp = ybuf;  // [NW][R][16] partial products of this wave's columns
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int i = 0; i < 4; ++i) epsp[(w * R + rb * 16 + lq * 4 + i) * 16 + lc] = eacc[rb][i];
      __syncthreads();
#pragma unroll
      for (int q = 0; q < ZPT; ++q) {
        const int it = tid + q * NT;
        if (it < R * A) {
          const int row = it / A, a = it % A;
          float part = 0.f;
#pragma unroll
          for (int ww = 0; ww < NW; ++ww) part += epsp[(ww * R + row) * 16 + a];
          const float e = bout[q] + part;
          const auto dd = [&](int i) { return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(ddl), i)); };
          const float s1 = dd(0), rsa = dd(1), c0 = dd(2), ct = dd(3), sg = dd(4);
          float* xp = xs + row * 16 + OF::pcol(a);
          const float x = *xp;
          float x0 = (x - s1 * e) * rsa;
          if (p.clip) x0 = fminf(fmaxf(x0, -1.f), 1.f);
          float xn = c0 * x0 + ct * x;
          if (k > 0) xn += sg * zpre[q];
          *xp = xn;
          if (t == T - 1) {
            const int s = smp[row / HZ];
            if (s >= 0 && member == 0) p.out[((size_t)s * HZ + (row % HZ)) * A + a] = xn;
          }
        }
      }
      __syncthreads();
    }
  }
}

// ---------------------------------------------------------------- observation pre-pass
// Folded cross-attention: observation tokens, their keys/values and fold
// records, computed once per query before the denoising launch.  Workgroup
// (g, l) takes the 16 (sample, token) rows g*16 .. g*16+15 of the flattened
// [batch][n_obs] tokens and layer l; the tokens' embedding (a product with
// the observation matrix) is repeated by every layer's workgroup.
template <class AT>
__global__ void __launch_bounds__(512) obs_fold_kernel(const KParams p) {
  using O = Op<AT>;
  constexpr int D = 256, DH = 64, NW = 8, NT = NW * 64, CB = D / 16, REC = 2 * (D / DH) * D + 16;
  constexpr int KOBS = 64, LDO = KOBS + O::PAD, LDA = D + O::PAD;
  __shared__ __attribute__((aligned(16))) AT ob[16 * LDO];
  __shared__ __attribute__((aligned(16))) AT xa[16 * LDA];
  __shared__ __attribute__((aligned(16))) float kvr[16 * 2 * D];
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, lc = lane & 15, lq = lane >> 4;
  const int nobs = p.n_obs, L = p.L, l = blockIdx.y;
  const int row0 = blockIdx.x * 16, nrows = min(16, p.batch * nobs - row0);
  const float* raw = p.raw;
  constexpr int MPWO = CB / NW;
  f32x4 acc[MPWO][1];
#pragma unroll
  for (int m = 0; m < MPWO; ++m) acc[m][0] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int nch = p.obs_pad / KOBS;
  for (int c = 0; c < nch; ++c) {
    __syncthreads();
    for (int it = tid; it < 16 * KOBS; it += NT) {
      const int row = it / KOBS, k = it % KOBS, kk = c * KOBS + k;
      const float v = (row < nrows && kk < p.obs_dim) ? p.obs[(size_t)(row0 + row) * p.obs_dim + kk] : 0.f;
      O::store(ob, LDO, row, k, v);
    }
    __syncthreads();
    gemm_acc<AT, 1, MPWO, KOBS / O::KF>(acc, ob, LDO, p.pk + p.pk_obs, p.obs_pad / O::KF, c * (KOBS / O::KF),
                                         [&](int m) { return w + NW * m; }, lane);
  }
#pragma unroll
  for (int m = 0; m < MPWO; ++m) {
    const int gcol = (w + NW * m) * 16 + lc;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = lq * 4 + i, o = (row0 + row) % nobs;
      const float v = row < nrows ? acc[m][0][i] + raw[p.b_obs + gcol] + raw[p.P_mem + (size_t)(1 + o) * D + gcol] : 0.f;
      O::store(xa, LDA, row, gcol, v);
    }
  }
  __syncthreads();
  const LayerOff lo = p.loff[l];
  constexpr int MPWK = 2 * CB / NW;
  f32x4 kv[MPWK][1];
#pragma unroll
  for (int m = 0; m < MPWK; ++m) kv[m][0] = f32x4{0.f, 0.f, 0.f, 0.f};
  gemm_acc<AT, 1, MPWK, D / O::KF>(kv, xa, LDA, p.pk + p.poff[l].kv, D / O::KF, 0,
                                    [&](int m) { return w + NW * m; }, lane);
#pragma unroll
  for (int m = 0; m < MPWK; ++m) {
    const int gcol = (w + NW * m) * 16 + lc;
#pragma unroll
    for (int i = 0; i < 4; ++i) kvr[(lq * 4 + i) * (2 * D) + gcol] = kv[m][0][i] + raw[lo.b_kv + gcol];
  }
  __syncthreads();
  fold_rows<D, DH, NT, 16, sizeof(AT) == 2>(
      raw, lo.w_q, lo.w_o2t, lo.b_q, kvr, 2 * D, nrows,
      [&](int row) -> float* {
        const int tok = row0 + row, s = tok / nobs, o = tok % nobs;
        return p.okv + (((size_t)s * L + l) * nobs + o) * REC;
      },
      tid);
}

hipError_t launch_obs_fold(const KParams& p, int dtype, hipStream_t stream) {
  const int rows = p.batch * p.n_obs;
  if (rows <= 0) return hipSuccess;
  const dim3 grid((unsigned)((rows + 15) / 16), (unsigned)p.L);
  if (dtype == 1) hipLaunchKernelGGL(obs_fold_kernel<__bf16>, grid, dim3(512), 0, stream, p);
  else hipLaunchKernelGGL(obs_fold_kernel<float>, grid, dim3(512), 0, stream, p);
  return hipGetLastError();
}
// ---------------------------------------------------------------- creation
__global__ void pack_kernel(const float* __restrict__ raw, size_t off, int N, int Nvalid, int K, int Kpad, int bf,
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
  uint32_t e[4] = {0u, 0u, 0u, 0u};
  if (n < Nvalid) {
    const float* W = raw + off + (size_t)n * K;
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
    r[1] = (float)(1.0 / sqrt(abar));  // stored as a reciprocal: the update multiplies
    r[2] = (float)c0;
    r[3] = (float)ct;
    r[4] = (float)sqrt(var);
    r[5] = r[6] = r[7] = 0.f;
  }
}

// fold records of the time token: one workgroup per (timestep, layer)
template <bool BF>
__global__ void __launch_bounds__(512) time_fold_kernel(const float* __restrict__ raw, const LayerOff* __restrict__ loff,
                                                        const float* __restrict__ tkv, int L, float* __restrict__ tfold) {
  constexpr int D = 256, DH = 64, REC = 2 * (D / DH) * D + 16;
  __shared__ __attribute__((aligned(16))) float kv[2 * D];
  const int kl = blockIdx.x, l = kl % L;
  for (int i = threadIdx.x; i < 2 * D; i += 512) kv[i] = tkv[(size_t)kl * 2 * D + i];
  __syncthreads();
  const LayerOff q = loff[l];
  fold_rows<D, DH, 512, 1, BF>(raw, q.w_q, q.w_o2t, q.b_q, kv, 2 * D, 1,
                            [&](int) -> float* { return tfold + (size_t)kl * REC; }, (int)threadIdx.x);
}

hipError_t launch_time_fold(const float* raw, const LayerOff* loff, const float* tkv, int T, int L, int d, int dh,
                            int dtype, float* tfold, hipStream_t stream) {
  if (d != 256 || dh != 64) return hipErrorInvalidValue;
  if (dtype == 1)
    hipLaunchKernelGGL(time_fold_kernel<true>, dim3(T * L), dim3(512), 0, stream, raw, loff, tkv, L, tfold);
  else
    hipLaunchKernelGGL(time_fold_kernel<false>, dim3(T * L), dim3(512), 0, stream, raw, loff, tkv, L, tfold);
  return hipGetLastError();
}

hipError_t launch_pack(const float* raw, size_t off, int N, int Nvalid, int K, int Kpad, int dtype, uint4* dst,
                       hipStream_t stream) {
  const int KF = dtype == 1 ? 32 : 16;
  const size_t n = (size_t)(N / 16) * (Kpad / KF) * 64;
  const int bs = 256;
  hipLaunchKernelGGL(pack_kernel, dim3((unsigned)((n + bs - 1) / bs)), dim3(bs), 0, stream, raw, off, N, Nvalid,
                     K, Kpad, dtype == 1 ? 1 : 0, dst);
  return hipGetLastError();
}

hipError_t launch_time_kv(const float* raw, uint32_t pmem0, const uint32_t* wkv, const uint32_t* bkv, int T, int L,
                          int D, int dtype, float* rows_scratch, float* tkv, hipStream_t stream) {
  const int bs = 256;
  hipLaunchKernelGGL(time_row_kernel, dim3((T * D + bs - 1) / bs), dim3(bs), 0, stream, raw, pmem0, T, D,
                     rows_scratch);
  const size_t n = (size_t)T * L * 2 * D;
  hipLaunchKernelGGL(time_kv_kernel, dim3((unsigned)((n + bs - 1) / bs)), dim3(bs), 0, stream, raw,
                     rows_scratch, wkv, bkv, T, L, D, dtype == 1 ? 1 : 0, tkv);
  return hipGetLastError();
}

__global__ void zero_u32_kernel(unsigned* dst, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) dst[i] = 0u;
}

hipError_t launch_zero_u32(unsigned* dst, int n, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(zero_u32_kernel, dim3((n + 255) / 256), dim3(256), 0, stream, dst, n);
  return hipGetLastError();
}

hipError_t launch_ddpm_table(int T, float* table, hipStream_t stream) {
  hipLaunchKernelGGL(ddpm_kernel, dim3(1), dim3(1), 0, stream, T, table);
  return hipGetLastError();
}

// ---------------------------------------------------------------- dispatch
#define EVO_SHAPES(X)                                     \
  X(float, 64, 32, 8, 2, 256, 4, 2, 256, 8, 1)            \
  X(__bf16, 64, 32, 8, 2, 256, 4, 2, 256, 8, 1)           \
  X(float, 256, 64, 16, 1, 1024, 8, 4, 256, 8, 1)         \
  X(float, 256, 64, 16, 2, 1024, 8, 2, 128, 8, 1)         \
  X(__bf16, 256, 64, 16, 1, 1024, 8, 4, 256, 8, 1)        \
  X(__bf16, 256, 64, 16, 2, 1024, 8, 2, 256, 8, 1)        \
  X(__bf16, 768, 64, 32, 1, 3072, 8, 2, 256, 5, 1)        \
  X(float, 256, 64, 16, 1, 1024, 4, 1, 256, 8, 4)         \
  X(__bf16, 256, 64, 16, 1, 1024, 4, 1, 256, 8, 4)        \
  X(float, 256, 64, 16, 1, 1024, 8, 2, 256, 8, 2)         \
  X(__bf16, 256, 64, 16, 1, 1024, 8, 2, 256, 8, 2)        \
  X(__bf16, 768, 64, 32, 1, 3072, 8, 2, 256, 5, 2)

template <class AT> constexpr int dtype_of() { return std::is_same<AT, float>::value ? 0 : 1; }

#define EVO_MATCH(AT, D, DH, HZ, SPT, DFF, TEAM)                                                          \
  (key.d == D && key.dh == DH && key.horizon == HZ && key.d_ff == DFF && key.dtype == dtype_of<AT>() && \
   key.spt == SPT && key.team == TEAM)

bool kernel_available(const KernelKey& key, int* threads) {
#define X(AT, D, DH, HZ, SPT, DFF, NW, HG, FC, SMAX, TEAM) \
  if (EVO_MATCH(AT, D, DH, HZ, SPT, DFF, TEAM)) {          \
    if (threads) *threads = NW * 64;                       \
    return true;                                           \
  }
  EVO_SHAPES(X)
#undef X
  return false;
}

int kernel_max_obs_tokens_for(const KernelKey& key) {
#define X(AT, D, DH, HZ, SPT, DFF, NW, HG, FC, SMAX, TEAM) \
  if (EVO_MATCH(AT, D, DH, HZ, SPT, DFF, TEAM)) return (SMAX - 1) < 16 / SPT ? (SMAX - 1) : 16 / SPT;
  EVO_SHAPES(X)
#undef X
  return 0;
}

int kernel_max_action_dim() { return 16; }

int kernel_team_sizes(const KernelKey& key, int out[4]) {
  int n = 0;
#define X(AT, D, DH, HZ, SPT, DFF, NW, HG, FC, SMAX, TEAM) \
  if (TEAM > 1 && n < 4 && key.d == D && key.dh == DH && key.horizon == HZ && key.d_ff == DFF &&      \
      key.dtype == dtype_of<AT>() && key.spt == SPT)                                                   \
    out[n++] = TEAM;
  EVO_SHAPES(X)
#undef X
  std::sort(out, out + n, [](int a, int b) { return a > b; });
  return n;
}

int kernel_max_steps_x_spt() { return kMaskEntries; }

hipError_t launch_denoise(const KernelKey& key, const KParams& p, hipStream_t stream) {
#define X(AT, D, DH, HZ, SPT, DFF, NW, HG, FC, SMAX, TEAM)                                                   \
  if (EVO_MATCH(AT, D, DH, HZ, SPT, DFF, TEAM)) {                                                          \
    const void* fn = reinterpret_cast<const void*>(&denoise_kernel<AT, D, DH, HZ, SPT, DFF, NW, HG, FC, SMAX, TEAM>); \
    if (TEAM == 1) {                                                                                       \
      hipLaunchKernelGGL((denoise_kernel<AT, D, DH, HZ, SPT, DFF, NW, HG, FC, SMAX, TEAM>), dim3(p.n_tiles), \
                         dim3(NW * 64), 0, stream, p);                                                     \
      return hipGetLastError();                                                                            \
    }                                                                                                      \
    /* team members wait for each other: all workgroups must be resident */                                \
    KParams pc = p;                                                                                        \
    void* args[] = {&pc};                                                                                  \
    return hipLaunchCooperativeKernel(fn, dim3(p.n_tiles * TEAM), dim3(NW * 64), args, 0, stream);         \
  }
  EVO_SHAPES(X)
#undef X
  return hipErrorInvalidValue;
}

}  // namespace evo
