// Fused diagonal-covariance GMM EM iteration for AMD Instinct MI355X (gfx950).
//
// One EM iteration (Flash-GMM paper, Sec. 3.1 and Algorithm 1, with the
// diagonal model) is computed without ever storing the n x k responsibility
// matrix:
//
//   prep        per component: the expanded-form operands
//                 W_kd = mu_kd / var_kd,  P_kd = -1/2 / var_kd,
//                 c_k  = log pi_k - 1/2 sum_d (mu_kd^2 / var_kd + log(2 pi var_kd))
//               (computed in fp64, all pre-scaled by log2(e) so the kernels
//               work in base 2), packed in the register order of the MFMA B
//               operands: bf16 hi and lo parts for the split-bf16 screening,
//               fp32 for the fp32 screening and the statistics.
//   logz        Step 1 of Algorithm 1: log-densities l = [x | x^2] . [W | P]^T + c
//               on MFMA (three bf16 products per fp32 product, or fp32), an
//               online log-sum-exp over all components, the pairs that carry
//               a point's mass recomputed in the direct form in fp64, one fp64
//               log-normaliser per point and per-workgroup log-likelihood
//               partials.
//   stats       Step 2 of Algorithm 1: the same log-densities recomputed on
//               fp32 MFMA for the (point, 64-component block) pairs that can
//               hold a responsibility above 2^-64, r = 2^(l - log2 Z) kept in
//               registers, and the statistic contraction r^T [x | x^2] on fp32
//               MFMA whose accumulators are added into fp64 partials every 4096
//               queued points; the few pairs that carry most of a point's
//               mass are summed exactly in fp64 on the vector ALU (fp32
//               products are exact in fp64).
//   reduce      fixed-order fp64 sums of the partials (instead of the paper's
//               atomics), added into the caller's accumulators.
//   mstep       closed-form M-step (Eqs. Nk, muk, sig per dimension) in fp64.
//
// Conditioning.  The expanded form sums terms of size about mu^2/var that
// cancel; its fp32 rounding error grows like u * sum_d (mu_kd^2 + var_kd)/var_kd.
// Components that have shrunk onto a few points (tiny variances) make this
// sum reach 1e5..1e9, where fp32 logits are meaningless.  Such components are
// routed to the direct form (x - mu)^2 / var on the vector ALU, whose fp32
// error is relative to the result.  Routing depends only on the parameters.
// The statistics are fp64 for every component: the M-step forms the variance
// as q/n - mu^2, which cancels by a factor mu^2/var that reaches 1e7 for a
// component collapsing onto one point, beyond any fp32 accumulation.
//
// Results are bitwise reproducible run to run: every sum runs in a fixed
// order.  The only atomics are LDS integer counters: the exact pairs' counts
// per bucket (sums of ones, the same in any order) and the counters with
// which the assignment kernels append candidates to per-point lists; a list
// is sorted before its terms are summed, and the fallback's list of points
// only decides which points a workgroup visits, each point's result being
// its own.

#include <hip/hip_runtime.h>

#include <math.h>
#include <stdint.h>
#include <string.h>

#include <mutex>
#include <thread>
#include <vector>
#include <type_traits>

#include "flashgmm.h"

namespace {

constexpr int kBK = 32;                 // components per MFMA block of the screening pass
constexpr int kWB = 64;                 // components per workgroup of k_stats_well
constexpr double kLog2e = 1.4426950408889634073599246810019;
constexpr double kLn2 = 0.69314718055994530941723212145818;
constexpr double kLog2Pi = 1.8378770664093454835606594728112;  // log(2 pi)
// routing threshold (see header comment) on sum_d (mu^2 + var) / var: below it
// the fp32 expanded form is good to ~1e-2 in log2 units, plenty for screening
constexpr double kIllSum = 2.0e5;
constexpr int kT = 4;                   // exact responsibilities stored per point
constexpr int kFlush = 128;             // k_stats_well: fp32 -> fp64 every 128 iterations
constexpr int kStatsWin = 4096;         // k_stats_well: points scanned per queue window
// Refined lists store component slots as 16-bit values; kNoSlot marks an
// empty entry (slots are < k <= GMM_MAX_K = 65535).
constexpr unsigned short kNoSlot = 0xFFFF;
// Refinement rule of k_logz.  A screened term r (relative to the screening
// normaliser) is recomputed exactly when r > 2^-window, with window = 40 for
// components whose fp32 expanded-form error bound (about 4 u log2(e) (e + d),
// e = sum mu^2 / var) exceeds 2^-12 log2 units, and window = 10 for the others,
// whose screened terms are already good to that bound; and, within 2^-40,
// whenever its lane state is among the point's four largest.  The exact
// top-kT list then holds a point's largest pairs even when they are tiny:
// those pairs carry the variance of a component that sits on a few points.
constexpr double kWideWindow = 40.0;
// a lane state whose components other than its arg-max carry a screened mass
// whose error bound exceeds this share of the point's total is refined in full
constexpr float kFullErr = 0x1p-20f;
// refinement list entries held in LDS at a time by k_logz
constexpr int kRefCap = 1024;
// lanes that share one direct-form sum of the k_logz refinement (bf16 path)
constexpr int kRefLanes = 4;
constexpr double kNarrowWindow = 10.0;
constexpr double kLooseBound = -12.0;
// Dense statistics are formed only for the (point, 64-component block) pairs
// that can hold a responsibility above 2^-kDenseWindow that is not among the
// point's stored exact pairs: a lane state within kDenseWindow of the
// screening log2 Z marks its arg-max component's block (unless that component
// is stored), and all of its blocks when the screened mass of its other
// components exceeds kDenseMass of the point's total.  Every pair left out
// has r < 2^-kDenseWindow up to the screening error (a few log2 units at
// most), so a component's N_k moves by less than N 2^-58.
constexpr float kDenseWindow = 64.0f;
constexpr float kDenseMass = 0x1p-64f;

typedef float f16v __attribute__((ext_vector_type(16)));

__device__ __forceinline__ f16v mfma32(float a, float b, f16v c) {
  return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float exp2_fast(float v) { return __builtin_amdgcn_exp2f(v); }

// bf16 MFMA (32x32x16): lane l holds A[l % 32][8 (l / 32) + e] and B[8 (l / 32) + e][l % 32],
// e = 0..7; the accumulator has the layout of the fp32 32x32 MFMAs.  An fp32 value v is
// carried as hi + lo, hi = bf16(v), lo = bf16(v - hi) (16 of its 24 bits), and a product
// as hi.hi + hi.lo + lo.hi; the dropped lo.lo and the representation error leave a
// relative error of about 2^-16 per product.
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
__device__ __forceinline__ f16v mfma32b(bf16x8 a, bf16x8 b, f16v c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// ---------------------------------------------------------------- online LSE (base 2)
// State (m, s) represents log2 sum_j 2^(l_j) = m + log2 s, with m = -inf, s = 0
// for the empty set.
__device__ __forceinline__ void lse_add(float& m, float& s, float l) {
  const float dl = l - m;                      // NaN only when both are -inf
  const float e = exp2_fast(-fabsf(dl));
  const bool gt = l > m;
  const float s_gt = __fmaf_rn(s, e, 1.0f);
  const float s_le = s + e;
  s = gt ? s_gt : ((l > -INFINITY) ? s_le : s);
  m = gt ? l : m;
}

__device__ __forceinline__ void lse_merge(float& m, float& s, float m2, float s2) {
  const float mm = fmaxf(m, m2);
  if (mm == -INFINITY) { m = -INFINITY; s = 0.0f; return; }
  s = s * exp2_fast(m - mm) + s2 * exp2_fast(m2 - mm);
  m = mm;
}

// Lane-state update of k_logz: the state starts at m = kEmpty (finite, below any
// log-density), s = 0, a = -1, so l = -inf (a dead or padded component) adds
// exactly 0 and no NaN can arise.  a tracks the arg-max slot.
constexpr float kEmpty = -3.0e38f;
__device__ __forceinline__ void lse_add_arg(float& m, float& s, int& a, float l, int slot) {
  const float dl = l - m;
  const float e = exp2_fast(-fabsf(dl));
  const bool gt = dl > 0.0f;
  s = gt ? __fmaf_rn(s, e, 1.0f) : s + e;
  m = gt ? l : m;
  a = gt ? slot : a;
}

// Inserts (l, slot) into the descending list tl/tsl of length kT; an entry
// equal to an existing one goes after it.  Static indexing only.
__device__ __forceinline__ void topk_insert(float* tl, int* tsl, float l, int slot) {
#pragma unroll
  for (int j = kT - 1; j > 0; --j) {
    if (l > tl[j - 1]) {
      tl[j] = tl[j - 1];
      tsl[j] = tsl[j - 1];
    } else if (l > tl[j]) {
      tl[j] = l;
      tsl[j] = slot;
    }
  }
  if (l > tl[0]) {
    tl[0] = l;
    tsl[0] = slot;
  }
}

// Lane-state update without arg-max (same kEmpty convention).
__device__ __forceinline__ void lse_add_e(float& m, float& s, float l) {
  const float dl = l - m;
  const float e = exp2_fast(-fabsf(dl));
  const bool gt = dl > 0.0f;
  s = gt ? __fmaf_rn(s, e, 1.0f) : s + e;
  m = gt ? l : m;
}

// ---------------------------------------------------------------- tiles
// rows x D64 fp32 tile of x (rows [r0, r0+rows)) into LDS with row pitch D64+4;
// rows >= nend and columns >= d are zero.
template <int D64>
__device__ __forceinline__ void load_tile(const float* __restrict__ x, int64_t nend, int d,
                                          int64_t r0, int rows, float* xs, bool vec4) {
  constexpr int P = D64 + 4;
  if (vec4) {
    constexpr int Q4 = D64 / 4;
    for (int idx = threadIdx.x; idx < rows * Q4; idx += blockDim.x) {
      const int r = idx / Q4, c = (idx % Q4) * 4;
      const int64_t nn = r0 + r;
      float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
      if (nn < nend && c < d) v = *reinterpret_cast<const float4*>(x + nn * d + c);
      *reinterpret_cast<float4*>(xs + r * P + c) = v;
    }
  } else {
    for (int idx = threadIdx.x; idx < rows * D64; idx += blockDim.x) {
      const int r = idx / D64, c = idx % D64;
      const int64_t nn = r0 + r;
      xs[r * P + c] = (nn < nend && c < d) ? x[nn * d + c] : 0.0f;
    }
  }
}

// ---------------------------------------------------------------- expanded-form logits (MFMA)
// Step s of a contraction over the x (or x^2) part feeds lane half h the
// dimension 8*(s/4) + 4*h + s%4.  Accumulator layout (32x32): register v of
// lane l holds point row0 + 8*(v/4) + 4*(l/32) + v%4 and component slot l%32
// of the block.  k_logz and k_stats_well form the same log-densities with
// different summation orders; they agree to fp32 rounding, far inside the
// screening error that both passes tolerate.

// ---------------------------------------------------------------- direct-form logits (VALU)
// l2 = c - sum_d (x_d - mu_d)^2 hh_d in log2 units, hh = log2(e) / (2 var) and c
// in fp64, summed in fp64 in dimension order; padded dimensions have
// x = mu = hh = 0.  fp64 because with small variances or many dimensions the
// constant and the sum reach 1e3 log2 units and more, where fp32 rounding alone
// (of the sum, of c and of hh) would exceed the responsibility tolerances.
template <int D64>
__device__ __forceinline__ double ill_logit(const float* xrow, const float* __restrict__ mu,
                                            const double* __restrict__ hh, double c) {
  double acc = 0.0;
#pragma unroll 4
  for (int j = 0; j < D64; j += 4) {
    const float4 xv = *reinterpret_cast<const float4*>(xrow + j);
    const float4 m = *reinterpret_cast<const float4*>(mu + j);
    const double2 g0 = *reinterpret_cast<const double2*>(hh + j);
    const double2 g1 = *reinterpret_cast<const double2*>(hh + j + 2);
    double t;
    t = (double)xv.x - (double)m.x; acc = fma(t * t, g0.x, acc);
    t = (double)xv.y - (double)m.y; acc = fma(t * t, g0.y, acc);
    t = (double)xv.z - (double)m.z; acc = fma(t * t, g1.x, acc);
    t = (double)xv.w - (double)m.w; acc = fma(t * t, g1.y, acc);
  }
  return c - acc;
}

// Same sum with a per-lane bound: the terms are >= 0, so once the partial sum
// of a lane exceeds `bound` its log-density is below c - bound, where the
// callers treat it as exactly nothing; such a lane returns -inf.  Every 16
// dimensions the wave stops when all of its lanes are past their bound
// (collapsed components are far from almost every point), so the result of a
// lane never depends on the other lanes.
template <int D64>
__device__ __forceinline__ double ill_logit_bounded(const float* xrow,
                                                    const float* __restrict__ mu,
                                                    const double* __restrict__ hh, double c,
                                                    double bound) {
  double acc = 0.0;
  for (int j0 = 0; j0 < D64; j0 += 16) {
#pragma unroll
    for (int j = j0; j < j0 + 16; j += 4) {
      const float4 xv = *reinterpret_cast<const float4*>(xrow + j);
      const float4 m = *reinterpret_cast<const float4*>(mu + j);
      const double2 g0 = *reinterpret_cast<const double2*>(hh + j);
      const double2 g1 = *reinterpret_cast<const double2*>(hh + j + 2);
      double t;
      t = (double)xv.x - (double)m.x; acc = fma(t * t, g0.x, acc);
      t = (double)xv.y - (double)m.y; acc = fma(t * t, g0.y, acc);
      t = (double)xv.z - (double)m.z; acc = fma(t * t, g1.x, acc);
      t = (double)xv.w - (double)m.w; acc = fma(t * t, g1.y, acc);
    }
    if (__ballot(!(acc > bound)) == 0ull) break;
  }
  return acc > bound ? -INFINITY : c - acc;
}

// The same two sums over a row of x in global memory (d values, no padding):
// the terms are taken in the same order, and the padded dimensions of the
// tile forms add exact zeros, so the results are bit-identical to theirs.
__device__ __forceinline__ double ill_logit_gr(const float* __restrict__ xrow, int d, int vec4,
                                               const float* __restrict__ mu,
                                               const double* __restrict__ hh, double c) {
  double acc = 0.0;
  int j = 0;
  if (vec4) {
    for (; j + 4 <= d; j += 4) {
      const float4 xv = *reinterpret_cast<const float4*>(xrow + j);
      const float4 m = *reinterpret_cast<const float4*>(mu + j);
      const double2 g0 = *reinterpret_cast<const double2*>(hh + j);
      const double2 g1 = *reinterpret_cast<const double2*>(hh + j + 2);
      double t;
      t = (double)xv.x - (double)m.x; acc = fma(t * t, g0.x, acc);
      t = (double)xv.y - (double)m.y; acc = fma(t * t, g0.y, acc);
      t = (double)xv.z - (double)m.z; acc = fma(t * t, g1.x, acc);
      t = (double)xv.w - (double)m.w; acc = fma(t * t, g1.y, acc);
    }
  }
  for (; j < d; ++j) {
    const double t = (double)xrow[j] - (double)mu[j];
    acc = fma(t * t, hh[j], acc);
  }
  return c - acc;
}

// acc0 carries the sum of dimensions 0 .. j_start-1 (j_start a multiple of 4).
__device__ __forceinline__ double ill_logit_bounded_gr(const float* __restrict__ xrow, int d,
                                                       int vec4, const float* __restrict__ mu,
                                                       const double* __restrict__ hh, double c,
                                                       double bound, double acc0 = 0.0,
                                                       int j_start = 0) {
  double acc = acc0;
  for (int j0 = j_start; j0 < d; j0 += 16) {
    const int j1 = j0 + 16 < d ? j0 + 16 : d;
    int j = j0;
    if (vec4) {
      for (; j + 4 <= j1; j += 4) {
        const float4 xv = *reinterpret_cast<const float4*>(xrow + j);
        const float4 m = *reinterpret_cast<const float4*>(mu + j);
        const double2 g0 = *reinterpret_cast<const double2*>(hh + j);
        const double2 g1 = *reinterpret_cast<const double2*>(hh + j + 2);
        double t;
        t = (double)xv.x - (double)m.x; acc = fma(t * t, g0.x, acc);
        t = (double)xv.y - (double)m.y; acc = fma(t * t, g0.y, acc);
        t = (double)xv.z - (double)m.z; acc = fma(t * t, g1.x, acc);
        t = (double)xv.w - (double)m.w; acc = fma(t * t, g1.y, acc);
      }
    }
    for (; j < j1; ++j) {
      const double t = (double)xrow[j] - (double)mu[j];
      acc = fma(t * t, hh[j], acc);
    }
    if (__ballot(!(acc > bound)) == 0ull) break;
  }
  return acc > bound ? -INFINITY : c - acc;
}

// ---------------------------------------------------------------- prep
// Workspace counters: [0] well components, [1] ill-conditioned components,
// [2] well 32-blocks, [3] ill 32-blocks.

__global__ __launch_bounds__(64) void k_prep_class(const float* __restrict__ w,
                                                   const float* __restrict__ mu,
                                                   const float* __restrict__ var, int d,
                                                   int* __restrict__ cls,
                                                   double* __restrict__ cwell,
                                                   double* __restrict__ cdir,
                                                   float2* __restrict__ cthr) {
  const int comp = blockIdx.x, lane = threadIdx.x;
  double e = 0.0, lg = 0.0;
  for (int j = lane; j < d; j += 64) {
    const double m = mu[(int64_t)comp * d + j], v = var[(int64_t)comp * d + j];
    e += m * m / v;
    lg += kLog2Pi + log(v);
  }
  for (int off = 32; off > 0; off >>= 1) {
    e += __shfl_xor(e, off);
    lg += __shfl_xor(lg, off);
  }
  if (lane == 0) {
    const double wk = w[comp];
    int c;
    if (!(wk > 0.0)) c = 2;
    else if (e + d > kIllSum || !(e == e)) c = 1;
    else c = 0;
    cls[comp] = c;
    const double lw = wk > 0.0 ? log(wk) : -INFINITY;
    cwell[comp] = kLog2e * (lw - 0.5 * (e + lg));
    cdir[comp] = kLog2e * (lw - 0.5 * lg);
    // screening error bound: about u * sum of |terms|, the terms of size
    // log2(e) * (mu^2 + x^2) / var for x near mu; taken as 4 u log2(e) (e + d)
    const double ldelta = -22.0 + log2(kLog2e * (e + d));
    // relative error bound of a screened responsibility: 4 u per step of the
    // running sum, over sqrt(2 d) steps of a random walk, the running sum of the
    // size of the constant plus the terms, in log2 units, times ln 2
    const double mag = fabs(kLog2e * (lw - 0.5 * (e + lg))) + kLog2e * (e + d);
    const double feb = kLn2 * 0x1p-22 * sqrt(2.0 * d) * mag;
    cthr[comp] = make_float2((float)(ldelta > kLooseBound ? -kWideWindow : -kNarrowWindow),
                             wk > 0.0 ? (float)feb : 0.0f);
  }
}

__global__ __launch_bounds__(256) void k_prep_scan(const int* __restrict__ cls, int k,
                                                   int* __restrict__ well_idx,
                                                   int* __restrict__ ill_idx,
                                                   int* __restrict__ counts) {
  __shared__ int cw[256], ci[256];
  const int t = threadIdx.x;
  const int b = (int)((int64_t)k * t / 256), e = (int)((int64_t)k * (t + 1) / 256);
  int nw = 0, ni = 0;
  for (int c = b; c < e; ++c) { nw += cls[c] == 0; ni += cls[c] == 1; }
  cw[t] = nw;
  ci[t] = ni;
  __syncthreads();
  if (t == 0) {
    int aw = 0, ai = 0;
    for (int i = 0; i < 256; ++i) {
      const int x = cw[i], y = ci[i];
      cw[i] = aw; ci[i] = ai;
      aw += x; ai += y;
    }
    counts[0] = aw;
    counts[1] = ai;
    counts[2] = (aw + kBK - 1) / kBK;
    counts[3] = (ai + kBK - 1) / kBK;
  }
  __syncthreads();
  int pw = cw[t], pi = ci[t];
  for (int c = b; c < e; ++c) {
    if (cls[c] == 0) well_idx[pw++] = c;
    else if (cls[c] == 1) ill_idx[pi++] = c;
  }
}

// Packed expanded-form operand: wp[(kb*(D64/4) + q)*64 + lane] is the float4 of
// MFMA steps 4q..4q+3 for lane `lane` of component block kb.
template <int D64>
__global__ __launch_bounds__(256) void k_prep_pack_well(
    const float* __restrict__ mu, const float* __restrict__ var, int d, int kpad,
    const double* __restrict__ cwell, const float2* __restrict__ cthr,
    const int* __restrict__ counts, const int* __restrict__ well_idx, float4* __restrict__ wp,
    float* __restrict__ cw, float2* __restrict__ thr) {
  constexpr int QQ = D64 / 4, QH = D64 / 8;
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= (int64_t)kpad * QQ * 2) return;   // kpad/32 blocks * QQ * 64 lanes
  const int lane = (int)(t & 63);
  const int q = (int)((t >> 6) % QQ);
  const int kb = (int)((t >> 6) / QQ);
  const int slot = kb * kBK + (lane & 31), h = lane >> 5;
  const int nw = counts[0];
  const int comp = slot < nw ? well_idx[slot] : -1;
  const bool xpart = q < QH;
  const int qq = xpart ? q : q - QH;
  float vals[4];
  for (int i = 0; i < 4; ++i) {
    const int j = 8 * qq + 4 * h + i;
    float v = 0.0f;
    if (comp >= 0 && j < d) {
      const double m = mu[(int64_t)comp * d + j], s2 = var[(int64_t)comp * d + j];
      v = xpart ? (float)(kLog2e * m / s2) : (float)(-0.5 * kLog2e / s2);
    }
    vals[i] = v;
  }
  wp[t] = make_float4(vals[0], vals[1], vals[2], vals[3]);
  if (q == 0 && h == 0) {
    cw[slot] = comp >= 0 ? (float)cwell[comp] : -INFINITY;
    thr[slot] = comp >= 0 ? cthr[comp] : make_float2(0.0f, 0.0f);
  }
}

// Steps (16 k each) of the split-bf16 screening: [x | x^2], or for tied
// variances [x | ||x||^2] (the x part, then one step for ||x||^2).
template <int D64, bool ISO>
__host__ __device__ constexpr int screen_steps() {
  return ISO ? D64 / 16 + 1 : D64 / 8;
}

// bf16 screening operand: for 32-component block kb and 16-k step s (k over
// [x | x^2], k < D64 the x part), wpb[((kb * NS16 + s) * 64 + l) * 2 + {0, 1}] holds the
// hi and lo parts of B[k = 16 s + 8 (l / 32) + e][slot 32 kb + l % 32], e = 0..7, where
// B is log2(e) mu/var (x part) or -log2(e) / (2 var) (x^2 part), split from fp64.
// ISO (tied variances, var[comp * d] the component's one variance): the x
// part as above, then one step whose lane half 0 holds -1/2 log2(e) / var in
// its first three places (they meet the three bf16 pieces of ||x||^2 in the
// split tile) and zeros elsewhere.

template <int D64, bool ISO>
__global__ __launch_bounds__(256) void k_prep_pack_b16(
    const float* __restrict__ mu, const float* __restrict__ var, int d, int kpad,
    const int* __restrict__ counts, const int* __restrict__ well_idx, bf16x8* __restrict__ wpb) {
  constexpr int NS16 = screen_steps<D64, ISO>();
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= (int64_t)(kpad / kBK) * NS16 * 64) return;
  const int lane = (int)(t & 63);
  const int s = (int)((t >> 6) % NS16);
  const int kb = (int)((t >> 6) / NS16);
  const int slot = kb * kBK + (lane & 31), h = lane >> 5;
  const int comp = slot < counts[0] ? well_idx[slot] : -1;
  bf16x8 hi, lo;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int k = 16 * s + 8 * h + e;
    const bool xpart = k < D64;
    const int j = xpart ? k : k - D64;
    double v = 0.0;
    if (ISO && !xpart) {
      // the ||x||^2 step, lane half 0: p = -1/2 log2(e) / var in three bf16
      // pieces, (hi, lo) in places 0..2 and (rest, 0) in places 3..5, each
      // group meeting the three pieces of ||x||^2 (one variance for all the
      // dimensions: this product's rounding does not average out over them)
      hi[e] = lo[e] = (__bf16)0.0f;
      if (comp >= 0 && j < 6) {
        const double pv = -0.5 * kLog2e / (double)var[(int64_t)comp * d];
        const __bf16 ph = (__bf16)(float)pv;
        const double r1 = pv - (double)(float)ph;
        const __bf16 pl = (__bf16)(float)r1;
        const __bf16 pr = (__bf16)(float)(r1 - (double)(float)pl);
        hi[e] = j < 3 ? ph : pr;
        lo[e] = j < 3 ? pl : (__bf16)0.0f;
      }
      continue;
    }
    if (comp >= 0 && j < d) {
      const double m = mu[(int64_t)comp * d + j], s2 = var[(int64_t)comp * d + j];
      v = xpart ? kLog2e * m / s2 : -0.5 * kLog2e / s2;
    }
    const __bf16 vh = (__bf16)(float)v;
    hi[e] = vh;
    lo[e] = (__bf16)(float)(v - (double)(float)vh);
  }
  wpb[2 * t] = hi;
  wpb[2 * t + 1] = lo;
}

// Packed 16x16x4 operand of k_stats_well: wq[(g * WQS + s) * 64 + lane] is,
// for 16-component group g and lane l, component slot 16g + l%16 at step s:
// W of dimension 16(s/4) + 4(l/16) + s%4 for s < D64/4, P of that dimension
// (s - D64/4 in place of s) for s < D64/2 (same fp64 -> fp32 values as wp),
// then for each 32-dimension group b the bias step s = D64/2 + b: 1 in lane
// groups l/16 = 0 and 2, the group's share of the log-density constant,
// log2(e) (log pi / NGB - 1/2 sum over its dimensions of (mu^2/var + log 2 pi var)),
// in lane group 1 (-inf for a dead or padded slot), and 0 in group 3.
constexpr int wq_steps(int D64) { return D64 / 2 + D64 / 32; }
// Tied variances (ISO): the x steps, then per 32-dimension group one norm step
// (-1/2 log2(e) / var in every lane group: it meets each lane's sum of squares
// over its 8 dimensions of the group), then the bias steps.
constexpr int wq_steps_iso(int D64) { return D64 / 4 + D64 / 16; }

template <int D64, bool ISO>
__global__ __launch_bounds__(256) void k_prep_pack_w16(
    const float* __restrict__ w, const float* __restrict__ mu, const float* __restrict__ var,
    int d, int kpad, const int* __restrict__ counts, const int* __restrict__ well_idx,
    float* __restrict__ wq) {
  constexpr int NS = D64 / 4, NGB = D64 / 32, WQS = ISO ? wq_steps_iso(D64) : wq_steps(D64);
  // first bias step
  constexpr int SB = ISO ? NS + NGB : 2 * NS;
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= (int64_t)(kpad / 16) * WQS * 64) return;
  const int lane = (int)(t & 63);
  const int s = (int)((t >> 6) % WQS);
  const int g = (int)((t >> 6) / WQS);
  const int slot = g * 16 + (lane & 15);
  const int comp = slot < counts[0] ? well_idx[slot] : -1;
  float v = 0.0f;
  if (ISO && s >= NS && s < SB) {
    if (comp >= 0) v = (float)(-0.5 * kLog2e / (double)var[(int64_t)comp * d]);
  } else if (s < SB) {
    const bool xpart = s < NS;
    const int ss = xpart ? s : s - NS;
    const int j = 16 * (ss / 4) + 4 * (lane >> 4) + ss % 4;
    if (comp >= 0 && j < d) {
      const double m = mu[(int64_t)comp * d + j], s2 = var[(int64_t)comp * d + j];
      v = xpart ? (float)(kLog2e * m / s2) : (float)(-0.5 * kLog2e / s2);
    }
  } else {
    const int b = s - SB, lg = lane >> 4;
    if (lg == 0) {
      v = 1.0f;
    } else if (lg == 1) {
      const double wk = comp >= 0 ? (double)w[comp] : 0.0;
      if (!(wk > 0.0)) {
        v = -INFINITY;
      } else {
        double e = 0.0;
        for (int j = 32 * b; j < 32 * b + 32 && j < d; ++j) {
          const double m = mu[(int64_t)comp * d + j], s2 = var[(int64_t)comp * d + j];
          e += m * m / s2 + kLog2Pi + log(s2);
        }
        v = (float)(kLog2e * (log(wk) / NGB - 0.5 * e));
      }
    } else if (lg == 2) {
      v = 1.0f;
    }
  }
  wq[t] = v;
}

// Direct-form parameters of every component (indexed by component):
// dmu = mu (fp32), dh = log2(e) / (2 var) (fp64), zero-padded to D64
// dimensions; the constant is cdir (fp64, from k_prep_class).
template <int D64>
__global__ __launch_bounds__(256) void k_prep_pack_direct(
    const float* __restrict__ mu, const float* __restrict__ var, int d, int k,
    float* __restrict__ dmu, double* __restrict__ dh) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= (int64_t)k * D64) return;
  const int comp = (int)(t / D64), j = (int)(t % D64);
  float m = 0.0f;
  double g = 0.0;
  if (j < d) {
    m = mu[(int64_t)comp * d + j];
    g = 0.5 * kLog2e / (double)var[(int64_t)comp * d + j];
  }
  dmu[t] = m;
  dh[t] = g;
}

// ---------------------------------------------------------------- Step 1: log-normalisers
// Points per screening workgroup: two 32-point MFMA tiles while a 64-point X
// tile fits in LDS next to the per-point state (D64 <= 256), one tile above.
__host__ __device__ constexpr int logz_tiles(int D64) { return D64 <= 256 ? 2 : 1; }
// The screening contraction runs on split bf16 MFMA from a split X tile in LDS
// while 64 points of it fit beside the post-screening state (D64 <= 128).  Its
// error, typically about 2^-16.5 of a product over D64/8 accumulation steps, is of
// the order of the fp32 chain's (2^-24 per step of a running sum of some hundred
// log2 units over D64 steps), so the refinement rules are the same for both.
__host__ __device__ constexpr bool screen_b16(int D64) { return D64 <= 128; }
// D64 > 256 (32-point tiles): split-bf16 screening too, the operands of the
// points split on the fly from the fp32 tile (logz_group16)
__host__ __device__ constexpr bool screen_x16(int D64) { return D64 > 256; }
__host__ __device__ constexpr bool screen_split(int D64) { return screen_b16(D64) || screen_x16(D64); }

// One software-pipelined step of a screening pass for one wave: when MF, the
// log-densities of the NT 32-point tiles against component block wpb are
// formed on MFMA into n0 (and n1), one chain per tile: bias first, then for
// every group of 8 dimensions the four x steps and the four x^2 steps.  When
// EPI, epi(v, c0[v], c1[v]) takes in the previous block's log-densities
// (c1 = c0 when NT == 1), spread over the contraction so that the vector ALU
// work overlaps the matrix work.
template <int D64, bool MF, bool EPI, int NT, class Epi>
__device__ __forceinline__ void logz_step(const float* xs, const float4* __restrict__ wpb,
                                          float cb, f16v& n0, f16v& n1, const f16v& c0,
                                          const f16v& c1, Epi&& epi) {
  constexpr int P = D64 + 4, QH = D64 / 8;
  const int lane = threadIdx.x & 63, h = lane >> 5, col = lane & 31;
  const float* xr0 = xs + col * P + 4 * h;
  const float* xr1 = xs + ((NT == 2 ? 32 : 0) + col) * P + 4 * h;
  float4 bw[3], bp[3];
  if (MF) {
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      n0[v] = cb;
      if constexpr (NT == 2) n1[v] = cb;
    }
    bw[0] = wpb[lane];
    bp[0] = wpb[QH * 64 + lane];
    bw[1] = wpb[64 + lane];
    bp[1] = wpb[(QH + 1) * 64 + lane];
  }
#pragma unroll
  for (int q = 0; q < QH; ++q) {
    if (MF) {
      if (q + 2 < QH) {
        bw[(q + 2) % 3] = wpb[(q + 2) * 64 + lane];
        bp[(q + 2) % 3] = wpb[(QH + q + 2) * 64 + lane];
      }
      const float4 a = *reinterpret_cast<const float4*>(xr0 + 8 * q);
      const float4 w = bw[q % 3], pp = bp[q % 3];
      if constexpr (NT == 2) {
        const float4 c = *reinterpret_cast<const float4*>(xr1 + 8 * q);
        n0 = mfma32(a.x, w.x, n0);
        n1 = mfma32(c.x, w.x, n1);
        n0 = mfma32(a.y, w.y, n0);
        n1 = mfma32(c.y, w.y, n1);
        n0 = mfma32(a.z, w.z, n0);
        n1 = mfma32(c.z, w.z, n1);
        n0 = mfma32(a.w, w.w, n0);
        n1 = mfma32(c.w, w.w, n1);
        n0 = mfma32(a.x * a.x, pp.x, n0);
        n1 = mfma32(c.x * c.x, pp.x, n1);
        n0 = mfma32(a.y * a.y, pp.y, n0);
        n1 = mfma32(c.y * c.y, pp.y, n1);
        n0 = mfma32(a.z * a.z, pp.z, n0);
        n1 = mfma32(c.z * c.z, pp.z, n1);
        n0 = mfma32(a.w * a.w, pp.w, n0);
        n1 = mfma32(c.w * c.w, pp.w, n1);
      } else {
        n0 = mfma32(a.x, w.x, n0);
        n0 = mfma32(a.y, w.y, n0);
        n0 = mfma32(a.z, w.z, n0);
        n0 = mfma32(a.w, w.w, n0);
        n0 = mfma32(a.x * a.x, pp.x, n0);
        n0 = mfma32(a.y * a.y, pp.y, n0);
        n0 = mfma32(a.z * a.z, pp.z, n0);
        n0 = mfma32(a.w * a.w, pp.w, n0);
      }
    }
    if (EPI) {
#pragma unroll
      for (int v = q * 16 / QH; v < (q + 1) * 16 / QH; ++v) {
        if constexpr (NT == 2) epi(v, c0[v], c1[v]);
        else epi(v, c0[v], c0[v]);
      }
    }
    // keep each step's loads in their step (unbounded hoisting exhausts registers)
    __builtin_amdgcn_sched_barrier(0);
  }
}

// The same step on bf16 MFMA (32x32x16, hi/lo split): the X tile is held in
// LDS as split 8-value chunks xa[p * (D64/2 + 1) + 2 c + {hi, lo}], chunk c
// covering k = 8c .. 8c+7 of [x | x^2]; step s consumes chunks 2s (lane half 0)
// and 2s + 1 (lane half 1); wpb is the block's packed split operand.
template <int NS, int RPV, bool MF, bool EPI, int NT, class Epi>
__device__ __forceinline__ void logz_step16(const bf16x8* xa, const bf16x8* __restrict__ wpb,
                                            float cb, f16v& n0, f16v& n1, const f16v& c0,
                                            const f16v& c1, Epi&& epi) {
  const int lane = threadIdx.x & 63, h = lane >> 5, col = lane & 31;
  const bf16x8* xr0 = xa + col * RPV + 2 * h;
  const bf16x8* xr1 = xa + ((NT == 2 ? 32 : 0) + col) * RPV + 2 * h;
  bf16x8 bh[3], bl[3];
  if (MF) {
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      n0[v] = cb;
      if constexpr (NT == 2) n1[v] = cb;
    }
    bh[0] = wpb[2 * lane];
    bl[0] = wpb[2 * lane + 1];
    bh[1] = wpb[2 * (64 + lane)];
    bl[1] = wpb[2 * (64 + lane) + 1];
  }
#pragma unroll
  for (int q = 0; q < NS; ++q) {
    if (MF) {
      if (q + 2 < NS) {
        bh[(q + 2) % 3] = wpb[2 * ((q + 2) * 64 + lane)];
        bl[(q + 2) % 3] = wpb[2 * ((q + 2) * 64 + lane) + 1];
      }
      const bf16x8 wh = bh[q % 3], wl = bl[q % 3];
      const bf16x8 ah = xr0[4 * q], al = xr0[4 * q + 1];
      if constexpr (NT == 2) {
        const bf16x8 ch = xr1[4 * q], cl = xr1[4 * q + 1];
        n0 = mfma32b(ah, wh, n0);
        n1 = mfma32b(ch, wh, n1);
        n0 = mfma32b(ah, wl, n0);
        n1 = mfma32b(ch, wl, n1);
        n0 = mfma32b(al, wh, n0);
        n1 = mfma32b(cl, wh, n1);
      } else {
        n0 = mfma32b(ah, wh, n0);
        n0 = mfma32b(ah, wl, n0);
        n0 = mfma32b(al, wh, n0);
      }
    }
    if (EPI) {
#pragma unroll
      for (int v = q * 16 / NS; v < (q + 1) * 16 / NS; ++v) {
        if constexpr (NT == 2) epi(v, c0[v], c1[v]);
        else epi(v, c0[v], c0[v]);
      }
    }
    if (MF && EPI && NT == 2) {
      // the step's LDS and global loads first, then six rounds of one MFMA and
      // three VALU instructions of the previous block's epilogue (2 % faster
      // than the compiler's own order at N = 1e8)
      __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
      __builtin_amdgcn_sched_group_barrier(0x020, 2, 0);
#pragma unroll
      for (int r = 0; r < 6; ++r) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, 3, 0);
      }
    }
    __builtin_amdgcn_sched_barrier(0);
  }
}

// Split-bf16 screening straight from the fp32 tile (D64 > 256, 32-point
// tiles), GB component blocks at a time.  Pair-step q covers dimensions
// 16 q .. 16 q + 15 of both parts of [x | x^2]: each lane reads its eight
// values of x once from the tile (lane half h: dimensions 16 q + 8 h + e),
// splits x and x^2 into hi and lo bf16 parts, and multiplies them with the
// packed operands of steps q (x part) and q + D64/16 (x^2 part) of every
// block kb[j], three products per fp32 product, into accumulator n[j] (chains
// interleaved over the blocks).  The B operands of pair-step q + 1 are loaded
// during pair-step q.  EPI: the previous group's log-densities c[j] (blocks
// j < nvp) are taken in by epi(j, v, value) during the first eight pair-steps,
// eight values each (fixed register indices).
// ISO (tied variances): the x part only, then one step for ||x||^2: each lane
// sums the squares of its values (eight a pair-step, then over the
// pair-steps), the two lane halves' sums are added, and lane half 0 meets
// -1/2 log2(e) / var in three bf16 pieces with the three bf16 pieces of the
// norm (the operand layout of k_prep_pack_b16<D64, true>).
template <int D64, int GB, bool MF, bool EPI, bool ISO, class Epi>
__device__ __forceinline__ void logz_group16(const float* xs, const bf16x8* __restrict__ wpb,
                                             const int (&kb)[GB], const float (&cb)[GB],
                                             f16v (&n)[GB], const f16v (&c)[GB], int nvp,
                                             Epi&& epi) {
  constexpr int P = D64 + 4, NQ = D64 / 16;
  constexpr size_t BS = (size_t)screen_steps<D64, ISO>() * 64 * 2;
  constexpr int NB = ISO ? 2 : 4;                 // B operands a block and pair-step
  static_assert(NQ % 8 == 0 && 16 * GB == 64, "eight pair-steps of eight epilogue values");
  const int lane = threadIdx.x & 63, h = lane >> 5, col = lane & 31;
  const float* xr = xs + col * P + 8 * h;
  bf16x8 bw[2][GB][NB];                           // ring of two pair-steps of B operands
  float ssq = 0.0f;                               // ISO: this lane's sum of squares
  auto load_b = [&](auto slot, int q) {
    constexpr int sl = decltype(slot)::value;
#pragma unroll
    for (int j = 0; j < GB; ++j) {
      const bf16x8* w = wpb + (size_t)kb[j] * BS;
      bw[sl][j][0] = w[2 * (q * 64 + lane)];
      bw[sl][j][1] = w[2 * (q * 64 + lane) + 1];
      if constexpr (!ISO) {
        bw[sl][j][2] = w[2 * ((q + NQ) * 64 + lane)];
        bw[sl][j][3] = w[2 * ((q + NQ) * 64 + lane) + 1];
      }
    }
  };
  if (MF) {
#pragma unroll
    for (int j = 0; j < GB; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) n[j][v] = cb[j];
    load_b(std::integral_constant<int, 0>{}, 0);
  }
  auto step = [&](auto slot, auto tc, int q, bool first) {
    constexpr int sl = decltype(slot)::value, t8 = decltype(tc)::value;
    if (MF) {
      if (q + 1 < NQ) load_b(std::integral_constant<int, 1 - sl>{}, q + 1);
      const float4 u0 = *reinterpret_cast<const float4*>(xr + 16 * q);
      const float4 u1 = *reinterpret_cast<const float4*>(xr + 16 * q + 4);
      const float v8[8] = {u0.x, u0.y, u0.z, u0.w, u1.x, u1.y, u1.z, u1.w};
      bf16x8 xh, xl, qh, ql;
      float sq8 = 0.0f;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const __bf16 vh = (__bf16)v8[e];
        xh[e] = vh;
        xl[e] = (__bf16)(v8[e] - (float)vh);
        const float sq = v8[e] * v8[e];
        if constexpr (ISO) {
          sq8 += sq;
        } else {
          const __bf16 sh = (__bf16)sq;
          qh[e] = sh;
          ql[e] = (__bf16)(sq - (float)sh);
        }
      }
      if constexpr (ISO) ssq += sq8;
#pragma unroll
      for (int j = 0; j < GB; ++j) n[j] = mfma32b(xh, bw[sl][j][0], n[j]);
#pragma unroll
      for (int j = 0; j < GB; ++j) n[j] = mfma32b(xh, bw[sl][j][1], n[j]);
#pragma unroll
      for (int j = 0; j < GB; ++j) n[j] = mfma32b(xl, bw[sl][j][0], n[j]);
      if constexpr (!ISO) {
#pragma unroll
        for (int j = 0; j < GB; ++j) n[j] = mfma32b(qh, bw[sl][j][2], n[j]);
#pragma unroll
        for (int j = 0; j < GB; ++j) n[j] = mfma32b(qh, bw[sl][j][3], n[j]);
#pragma unroll
        for (int j = 0; j < GB; ++j) n[j] = mfma32b(ql, bw[sl][j][2], n[j]);
      }
    }
    if (EPI && first) {
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        constexpr int e0 = 8 * t8;
        const int e = e0 + i, j = e >> 4, v = e & 15;
        if (j < nvp) epi(j, v, c[j][v]);
      }
    }
    __builtin_amdgcn_sched_barrier(0);
  };
  for (int q0 = 0; q0 < NQ; q0 += 8) {
    const bool first = q0 == 0;
    step(std::integral_constant<int, 0>{}, std::integral_constant<int, 0>{}, q0, first);
    step(std::integral_constant<int, 1>{}, std::integral_constant<int, 1>{}, q0 + 1, first);
    step(std::integral_constant<int, 0>{}, std::integral_constant<int, 2>{}, q0 + 2, first);
    step(std::integral_constant<int, 1>{}, std::integral_constant<int, 3>{}, q0 + 3, first);
    step(std::integral_constant<int, 0>{}, std::integral_constant<int, 4>{}, q0 + 4, first);
    step(std::integral_constant<int, 1>{}, std::integral_constant<int, 5>{}, q0 + 5, first);
    step(std::integral_constant<int, 0>{}, std::integral_constant<int, 6>{}, q0 + 6, first);
    step(std::integral_constant<int, 1>{}, std::integral_constant<int, 7>{}, q0 + 7, first);
  }
  if constexpr (ISO) {
    if (MF) {
      // the norm step: ||x||^2 of point col in three bf16 pieces, in places
      // 0..2 and 3..5 of lane half 0, against the step's (hi, lo) operands
      const float nrm = ssq + __shfl_xor(ssq, 32);
      const __bf16 p0 = (__bf16)nrm;
      const float r1 = nrm - (float)p0;
      const __bf16 p1 = (__bf16)r1;
      const __bf16 p2 = (__bf16)(r1 - (float)p1);
      bf16x8 a;
#pragma unroll
      for (int e = 0; e < 8; ++e) a[e] = (__bf16)0.0f;
      if (h == 0) {
        a[0] = a[3] = p0;
        a[1] = a[4] = p1;
        a[2] = a[5] = p2;
      }
#pragma unroll
      for (int j = 0; j < GB; ++j) {
        const bf16x8* w = wpb + (size_t)kb[j] * BS;
        n[j] = mfma32b(a, w[2 * (NQ * 64 + lane)], n[j]);
        n[j] = mfma32b(a, w[2 * (NQ * 64 + lane) + 1], n[j]);
      }
    }
  }
}

// Transposing reduction over the 32 lanes of a lane half.  Every lane holds NV
// (16 or 32) values, value i of lane col belonging to the same point in every
// lane of the half; comb(j, half, off, up) merges value j (up: value j + half)
// of this lane with the other of the pair j, j + half of lane col ^ off (the
// partner sends the value this lane does not keep) into value j.  Each level
// halves the values, the last ones pair lanes with a plain butterfly, so after
// the five levels value 0 of lane col holds the reduction of value index col
// (NV = 32) or col / 2 (NV = 16): 31 merges per lane instead of 5 NV.
// j and half reach comb as std::integral_constant, so that the register
// arrays it indexes stay in registers.
template <int J, int HALF, int OFF, class Comb>
__device__ __forceinline__ void xpose_pairs(Comb& comb, bool up) {
  if constexpr (J < HALF) {
    comb(std::integral_constant<int, J>{}, std::integral_constant<int, HALF>{},
         std::integral_constant<int, OFF>{}, up);
    xpose_pairs<J + 1, HALF, OFF>(comb, up);
  }
}

template <int NV, int LVL = 0, class Comb>
__device__ __forceinline__ void xpose_levels(int col, Comb&& comb) {
  if constexpr (LVL < 5) {
    constexpr int off = 16 >> LVL, cnt = NV >> LVL;
    if constexpr (cnt > 1)
      xpose_pairs<0, cnt / 2, off>(comb, (col & off) != 0);
    else
      comb(std::integral_constant<int, 0>{}, std::integral_constant<int, 0>{},
           std::integral_constant<int, off>{}, false);
    xpose_levels<NV, LVL + 1>(col, comb);
  }
}

// v of lane (lane ^ OFF), OFF a constant: a DPP quad permutation for 1 and 2
// (no data-share instruction), a swizzle within 32 lanes for 4, 8 and 16 (no
// lane-index operand), a permute for 32.
template <int OFF>
__device__ __forceinline__ int xshfl_i(int v) {
  if constexpr (OFF == 1) return __builtin_amdgcn_mov_dpp(v, 0xB1, 0xF, 0xF, false);
  else if constexpr (OFF == 2) return __builtin_amdgcn_mov_dpp(v, 0x4E, 0xF, 0xF, false);
  else if constexpr (OFF == 4 || OFF == 8 || OFF == 16)
    return __builtin_amdgcn_ds_swizzle(v, 0x1F | (OFF << 10));
  else return __shfl_xor(v, OFF);
}
template <int OFF>
__device__ __forceinline__ float xshfl(float v) {
  return __int_as_float(xshfl_i<OFF>(__float_as_int(v)));
}
template <int OFF>
__device__ __forceinline__ double xshfl(double v) {
  const long long b = __double_as_longlong(v);
  const int lo = xshfl_i<OFF>((int)(b & 0xFFFFFFFFll)), hi = xshfl_i<OFF>((int)(b >> 32));
  return __longlong_as_double(((long long)hi << 32) | (unsigned)lo);
}

// The point whose reduction xpose_levels leaves in lane (h, col): value index
// i = col (NT = 2) or col / 2 (NT = 1) is block i / 16, register i % 16.
template <int NT>
__device__ __forceinline__ int xpose_point(int col, int h) {
  const int i = NT == 2 ? col : (col >> 1);
  const int v = i & 15;
  return 32 * (i >> 4) + 8 * (v >> 2) + 4 * h + (v & 3);
}

// One workgroup = PTS = 32 NT points (64 for D64 <= 256, else 32), 4 waves;
// wave w takes well component blocks w, w+4, ... and ill-conditioned
// components w, w+4, ...
//
//   1. screen: expanded-form log-densities on MFMA with a per-lane online LSE
//      that also remembers the arg-max; a "lane state" (wave, lane column,
//      point) covers every 32nd component of the wave's blocks.
//   2. the lane states are merged (within the wave by butterflies, then across
//      waves in a fixed order) into a screening log2 Z per point.
//   3. refinement: a lane state whose maximum, relative to that log2 Z, passes
//      its arg-max component's threshold (kWideWindow / kNarrowWindow) marks that
//      component as a candidate; the candidates' log-densities are recomputed
//      in the direct form (fp32 error relative to the result), thread (wave w,
//      point p) taking the candidates of wave w's lane states; their screened
//      terms are taken out of the sum and the exact ones put in, merged over
//      waves in a fixed order.  The result is the log2 Z written for the point,
//      and the kT largest exact responsibilities are stored for the statistics
//      pass.
// A significant component is missed only if a larger one of the same point
// shares its lane state; its responsibility then keeps the screening error.
// Chunk c of point p of the split tile of k_logz: v holds x of dims
// 8c .. 8c+7, each value stored as bf16 hi + lo; its square likewise in chunk
// c + D64/8 ([x | x^2] tile), or, ISO, the chunk's sum of squares is
// returned instead (fp32, in dimension order) for the ||x||^2 chunk.
template <int D64, bool ISO>
__device__ __forceinline__ float split_store(bf16x8* xa, int p, int c, const float (&v)[8]) {
  constexpr int NC8 = D64 / 8, RPV = 4 * screen_steps<D64, ISO>() + 1;
  bf16x8 hi, lo, hq, lq;
  float ssq = 0.0f;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const __bf16 vh = (__bf16)v[e];
    hi[e] = vh;
    lo[e] = (__bf16)(v[e] - (float)vh);
    const float q = v[e] * v[e];
    if (ISO) {
      ssq += q;
    } else {
      const __bf16 qh = (__bf16)q;
      hq[e] = qh;
      lq[e] = (__bf16)(q - (float)qh);
    }
  }
  xa[p * RPV + 2 * c] = hi;
  xa[p * RPV + 2 * c + 1] = lo;
  if (!ISO) {
    xa[p * RPV + 2 * (c + NC8)] = hq;
    xa[p * RPV + 2 * (c + NC8) + 1] = lq;
  }
  return ssq;
}

// ISO: the ||x||^2 chunk of point p from its chunks' sums of squares (summed
// in chunk order), split into three bf16 pieces (together exact to about
// 2^-24), in places 0..2 and again in 3..5 (they meet the pieces of the
// operand -1/2 log2(e) / var), followed by the zero chunk of the last step's
// lane half 1.
template <int D64>
__device__ __forceinline__ void split_store_norm(bf16x8* xa, int p, const float* csq) {
  constexpr int NC8 = D64 / 8, RPV = 4 * screen_steps<D64, true>() + 1;
  float nrm = 0.0f;
  for (int c = 0; c < NC8; ++c) nrm += csq[c];
  bf16x8 hi, z;
#pragma unroll
  for (int e = 0; e < 8; ++e) hi[e] = z[e] = (__bf16)0.0f;
  const __bf16 n0 = (__bf16)nrm;
  const float r1 = nrm - (float)n0;
  const __bf16 n1 = (__bf16)r1;
  hi[0] = hi[3] = n0;
  hi[1] = hi[4] = n1;
  hi[2] = hi[5] = (__bf16)(r1 - (float)n1);
  xa[p * RPV + 2 * NC8] = hi;
  xa[p * RPV + 2 * NC8 + 1] = z;
  xa[p * RPV + 2 * NC8 + 2] = z;
  xa[p * RPV + 2 * NC8 + 3] = z;
}

// First-chunk operands (dimensions 0..7) of a batch of ill-conditioned
// components, staged in LDS by k_logz.
constexpr int kIllStage = 128;
// Well slots whose refinement thresholds k_logz copies to LDS (bf16 screening).
constexpr int kThrStage = 1024;
struct IllStage {
  float mu[kIllStage][8];
  double h[kIllStage][8];
  double c[kIllStage];
  int comp[kIllStage];
};

// LDS state of k_logz after the screening pass, per workgroup of PTS points.
template <int PTS>
struct LogzPost {
  float2 stw[4][PTS];         // per wave: merged well state (M_w, S_w) per point
  float2 sti[4][PTS];         // per wave: ill state per point (maximum rounded to fp32)
  double stim[4][PTS];        // per wave: the ill state's maximum in fp64
  float cms[4][PTS];          // per wave: candidate mass relative to M_w
  float lzm[PTS];             // screening log2 Z
  float2 top2[4][PTS];        // per wave: the two largest lane-state maxima per point
  float s4m[PTS];             // lower bound of the 4th largest lane-state maximum
  unsigned cmask[PTS][4];     // candidate lane columns per (point, wave)
  unsigned fmask[PTS][4];     // of those, the lane states refined in full
  unsigned smask[PTS][4];     // lane states within kDenseWindow of the screening log2 Z
  unsigned omask[PTS][4];     // of those, the ones whose other components carry mass
  unsigned short cidx[PTS][128];  // arg-max well slot per (point, lane state)
  float2 rmc[4][PTS];         // per (wave, point): exact candidate LSE state
  int rcnt[256];              // refinement list: entries per (point, wave), then offsets
  int rwsum[8];
  int rlist[kRefCap];         // (point << 16) | slot
  float rres[kRefCap];        // exact log-density relative to the screening log2 Z
  int rts[4][kT][PTS];        // per (wave, point): largest exact candidates
  float rtl[4][kT][PTS];
};

// REFINE = false (the screened E-step): the candidates keep their screened
// log-densities instead of the direct-form ones; everything else is the same.
template <int D64, bool REFINE, bool ISO>
__global__ __launch_bounds__(256, screen_b16(D64) ? 2 : 1) void k_logz(
    const float* __restrict__ x, int64_t n, int d, int vec4, const float4* __restrict__ wp,
    const bf16x8* __restrict__ wpb,
    const float* __restrict__ cw, const float2* __restrict__ thr,
    const int* __restrict__ well_idx, const int* __restrict__ ill_idx,
    const float* __restrict__ dmu, const double* __restrict__ dh, const double* __restrict__ cdir,
    const int* __restrict__ counts, double* __restrict__ logz2,
    unsigned short* __restrict__ cslot, float* __restrict__ cr, double* __restrict__ ll_part,
    unsigned long long* __restrict__ bmask, unsigned char* __restrict__ iflag,
    unsigned char* __restrict__ lflag) {
  constexpr int P = D64 + 4, NT = logz_tiles(D64), PTS = 32 * NT;
  constexpr bool B16 = screen_b16(D64);
  static_assert(!ISO || screen_split(D64), "the isotropic screening is a split-bf16 one");
  // split tile row: [x | x^2] chunks (hi, lo), or for ISO the x chunks, one
  // ||x||^2 chunk and one zero chunk; one padding entry
  constexpr int NSTEP = screen_steps<D64, ISO>();
  constexpr int RPV = 4 * NSTEP + 1;
  // bf16 screening: the split [x | x^2] tile, whose space the post-screening
  // state takes over (direct-form sums then read x from global memory), so
  // that two workgroups fit a compute unit.  fp32 screening: the fp32 tile,
  // which the direct-form sums also read, and the state after it.
  constexpr size_t XS_BYTES = B16 ? 0 : (size_t)PTS * P * sizeof(float);
  constexpr size_t XA_BYTES = B16 ? (size_t)PTS * RPV * sizeof(bf16x8) : 0;
  constexpr size_t PS_BYTES = sizeof(LogzPost<PTS>);
  // bf16 screening: the ill components' staged operands follow the state
  constexpr size_t IST_OFF = (PS_BYTES + 15) / 16 * 16;
  constexpr size_t IST_END = B16 ? IST_OFF + sizeof(IllStage) : PS_BYTES;
  // bf16 screening: then the refinement thresholds and the components of up to
  // kThrStage well slots
  constexpr size_t THR_END =
      B16 ? IST_END + kThrStage * (sizeof(float2) + sizeof(int)) : PS_BYTES;
  constexpr size_t CSQ_END = XA_BYTES + (ISO ? (size_t)PTS * (D64 / 8) * sizeof(float) : 0);
  constexpr size_t SM_BYTES =
      B16 ? (CSQ_END > THR_END ? CSQ_END : THR_END) : XS_BYTES + PS_BYTES;
  static_assert(!B16 || SM_BYTES <= 80 * 1024, "two workgroups per compute unit");
  __shared__ __align__(16) unsigned char smem[SM_BYTES];
  float* const xs = reinterpret_cast<float*>(smem);
  bf16x8* const xa = reinterpret_cast<bf16x8*>(smem);
  // ISO: per-chunk sums of squares, after the tile (only used while building it)
  float* const csq = reinterpret_cast<float*>(smem + XA_BYTES);
  LogzPost<PTS>& post = *reinterpret_cast<LogzPost<PTS>*>(smem + XS_BYTES);
  auto& stw = post.stw;
  auto& sti = post.sti;
  auto& stim = post.stim;
  auto& cms = post.cms;
  auto& lzm = post.lzm;
  auto& top2 = post.top2;
  auto& s4m = post.s4m;
  auto& cmask = post.cmask;
  auto& fmask = post.fmask;
  auto& smask = post.smask;
  auto& omask = post.omask;
  auto& cidx = post.cidx;
  auto& rmc = post.rmc;
  auto& rcnt = post.rcnt;
  auto& rwsum = post.rwsum;
  auto& rlist = post.rlist;
  auto& rres = post.rres;
  auto& rts = post.rts;
  auto& rtl = post.rtl;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, h = lane >> 5, col = lane & 31;
  const int64_t n0 = (int64_t)blockIdx.x * PTS;
  if constexpr (B16) {
    // split tile: chunk c < D64/8 holds x of dims 8c .. 8c+7, chunk c + D64/8
    // x^2 of the same dims; rows >= n and dims >= d are zero
    constexpr int NC8 = D64 / 8, NIT = (PTS * NC8 + 255) / 256;
    if (vec4) {
      // every load of the thread issued before the first conversion (one
      // memory round trip per workgroup); out-of-range chunks load row 0,
      // dims 0..3 (always present: d is a multiple of 4 here) and are zeroed
      // after the load
      float4 ld[NIT][2];
      bool ok[NIT][2];
#pragma unroll
      for (int it = 0; it < NIT; ++it) {
        const int t = tid + 256 * it, p = t / NC8, c = t % NC8;
        const int64_t row = n0 + p;
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
          const int j = 8 * c + 4 * hf;
          ok[it][hf] = t < PTS * NC8 && row < n && j < d;
          ld[it][hf] = *reinterpret_cast<const float4*>(x + (ok[it][hf] ? row * d + j : 0));
        }
      }
      // the loaded registers are made opaque, so that the zeroing below stays a
      // register select and no load is moved under a branch
#pragma unroll
      for (int it = 0; it < NIT; ++it)
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
          asm volatile("" : "+v"(ld[it][hf].x), "+v"(ld[it][hf].y), "+v"(ld[it][hf].z),
                       "+v"(ld[it][hf].w));
          if (!ok[it][hf]) ld[it][hf] = make_float4(0.f, 0.f, 0.f, 0.f);
        }
#pragma unroll
      for (int it = 0; it < NIT; ++it) {
        const int t = tid + 256 * it;
        if (t < PTS * NC8) {
          const float v[8] = {ld[it][0].x, ld[it][0].y, ld[it][0].z, ld[it][0].w,
                              ld[it][1].x, ld[it][1].y, ld[it][1].z, ld[it][1].w};
          const float ssq = split_store<D64, ISO>(xa, t / NC8, t % NC8, v);
          if constexpr (ISO) csq[t] = ssq;
        }
      }
    } else {
      for (int t = tid; t < PTS * NC8; t += 256) {
        const int p = t / NC8, c = t % NC8;
        const int64_t row = n0 + p;
        float v[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int j = 8 * c + e;
          v[e] = (row < n && j < d) ? x[row * d + j] : 0.0f;
        }
        const float ssq = split_store<D64, ISO>(xa, p, c, v);
        if constexpr (ISO) csq[t] = ssq;
      }
    }
    if constexpr (ISO) {
      __syncthreads();
      if (tid < PTS) split_store_norm<D64>(xa, tid, csq + tid * NC8);
    }
  } else {
    load_tile<D64>(x, n, d, n0, PTS, xs, vec4 != 0);
  }
  __syncthreads();
  const int n_wkb = counts[2], n_ill = counts[1], n_well = counts[0];

  float m0[16], s0[16], m1[16], s1[16];
  int a0[16], a1[16];
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    m0[v] = m1[v] = kEmpty;
    s0[v] = s1[v] = 0.0f;
    a0[v] = a1[v] = -1;
  }
  {
    // wave w takes blocks w, w+4, ...: the MFMAs of block i+1 run while the
    // lane states take in block i
    const int nb = n_wkb > wave ? (n_wkb - wave + 3) / 4 : 0;
    constexpr size_t BS = (size_t)(D64 / 4) * 64;
    f16v c0, c1, x0, x1;
    int slot = 0;
    auto epi = [&](int v, float l0, float l1) {
      lse_add_arg(m0[v], s0[v], a0[v], l0, slot);
      if constexpr (NT == 2) lse_add_arg(m1[v], s1[v], a1[v], l1, slot);
    };
    constexpr size_t BS16 = (size_t)NSTEP * 64 * 2;
    if constexpr (screen_x16(D64)) {
      // GB blocks of this wave at a time: blocks wave + 4 i, i = GB g + j; a
      // group's missing blocks repeat its last one and are not taken in
      constexpr int GB = 4;
      const int ng = (nb + GB - 1) / GB;
      int kbc[GB], kbp[GB];
      float cbc[GB];
      f16v na[GB], nc[GB];
      int nvp = 0;
      auto epi16 = [&](int j, int v, float l) {
        lse_add_arg(m0[v], s0[v], a0[v], l, kbp[j] * kBK + col);
      };
      for (int g = 0; g <= ng; ++g) {
        if (g < ng) {
#pragma unroll
          for (int j = 0; j < GB; ++j) {
            const int i = GB * g + j < nb ? GB * g + j : nb - 1;
            kbc[j] = wave + 4 * i;
            cbc[j] = cw[kbc[j] * kBK + col];
          }
          if (g == 0)
            logz_group16<D64, GB, true, false, ISO>(xs, wpb, kbc, cbc, na, nc, 0, epi16);
          else
            logz_group16<D64, GB, true, true, ISO>(xs, wpb, kbc, cbc, na, nc, nvp, epi16);
        } else if (ng > 0) {
          logz_group16<D64, GB, false, true, ISO>(xs, wpb, kbc, cbc, na, nc, nvp, epi16);
        }
        // this group's log-densities become the previous group's
#pragma unroll
        for (int j = 0; j < GB; ++j) {
          nc[j] = na[j];
          kbp[j] = kbc[j];
        }
        nvp = nb - GB * g < GB ? nb - GB * g : GB;
      }
    } else if (nb > 0) {
      if constexpr (B16)
        logz_step16<NSTEP, RPV, true, false, NT>(xa, wpb + (size_t)wave * BS16, cw[wave * kBK + col], c0,
                                          c1, x0, x1, epi);
      else
        logz_step<D64, true, false, NT>(xs, wp + (size_t)wave * BS, cw[wave * kBK + col], c0, c1,
                                        x0, x1, epi);
      float cbn = nb > 1 ? cw[(wave + 4) * kBK + col] : 0.0f;
      for (int i = 0; i + 1 < nb; ++i) {
        const int kb = wave + 4 * i;
        const float cb = cbn;
        if (i + 2 < nb) cbn = cw[(kb + 8) * kBK + col];
        slot = kb * kBK + col;
        if constexpr (B16)
          logz_step16<NSTEP, RPV, true, true, NT>(xa, wpb + (size_t)(kb + 4) * BS16, cb, x0, x1, c0, c1,
                                           epi);
        else
          logz_step<D64, true, true, NT>(xs, wp + (size_t)(kb + 4) * BS, cb, x0, x1, c0, c1, epi);
        c0 = x0;
        c1 = x1;
      }
      slot = (wave + 4 * (nb - 1)) * kBK + col;
      if constexpr (B16)
        logz_step16<NSTEP, RPV, false, true, NT>(xa, wpb, 0.0f, x0, x1, c0, c1, epi);
      else
        logz_step<D64, false, true, NT>(xs, wp, 0.0f, x0, x1, c0, c1, epi);
    }
  }
  // the state below takes over the split tile's space
  if constexpr (B16) __syncthreads();
  // arg-max of every lane state, and the per-wave merged state of every point:
  // the LSE states and the two largest lane-state maxima (A >= B) of the 32
  // lanes of a lane half are merged by a transposing reduction (xpose_levels)
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const int p = 8 * (v >> 2) + 4 * h + (v & 3);
    cidx[p][wave * 32 + col] = (unsigned short)a0[v];
    if constexpr (NT == 2) cidx[32 + p][wave * 32 + col] = (unsigned short)a1[v];
  }
  {
    constexpr int NV = 16 * NT;
    float XM[NV], XS[NV], XA[NV], XB[NV];
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      XM[v] = m0[v];
      XS[v] = s0[v];
      XA[v] = m0[v];
      XB[v] = kEmpty;
      if constexpr (NT == 2) {
        XM[16 + v] = m1[v];
        XS[16 + v] = s1[v];
        XA[16 + v] = m1[v];
        XB[16 + v] = kEmpty;
      }
    }
    xpose_levels<NV>(col, [&](auto jc, auto hc, auto oc, bool up) {
      constexpr int j = decltype(jc)::value, half = decltype(hc)::value;
      constexpr int off = decltype(oc)::value;
      const float km = up ? XM[j + half] : XM[j], sm = up ? XM[j] : XM[j + half];
      const float ks = up ? XS[j + half] : XS[j], ss = up ? XS[j] : XS[j + half];
      const float ka = up ? XA[j + half] : XA[j], sa = up ? XA[j] : XA[j + half];
      const float kb = up ? XB[j + half] : XB[j], sb = up ? XB[j] : XB[j + half];
      const float rm = xshfl<off>(sm), rs = xshfl<off>(ss);
      const float ra = xshfl<off>(sa), rb = xshfl<off>(sb);
      float M = km, S = ks;
      lse_merge(M, S, rm, rs);
      XM[j] = M;
      XS[j] = S;
      XB[j] = fmaxf(fminf(ka, ra), fmaxf(kb, rb));
      XA[j] = fmaxf(ka, ra);
    });
    const int p = xpose_point<NT>(col, h);
    if (NT == 2 || (col & 1) == 0) {
      stw[wave][p] = make_float2(XM[0], XS[0]);
      top2[wave][p] = make_float2(XA[0], XB[0]);
    }
  }
  // the refinement thresholds, read by every lane state below, and the
  // components of the well slots, read by every refined pair: loaded now,
  // stored to LDS after the ill-conditioned components (bf16 screening, at
  // most kThrStage slots; else read from global memory)
  const int kpad_w = (n_well + kWB - 1) / kWB * kWB;
  const bool thr_lds = B16 && kpad_w <= kThrStage;
  float2* const thr_s = reinterpret_cast<float2*>(smem + IST_END);
  int* const wid_s = reinterpret_cast<int*>(smem + IST_END + kThrStage * sizeof(float2));
  constexpr int NTHR = kThrStage / 256;
  float2 thr_r[NTHR];
  int wid_r[NTHR];
  if (thr_lds) {
#pragma unroll
    for (int i = 0; i < NTHR; ++i) {
      const int e = tid + 256 * i;
      thr_r[i] = e < kpad_w ? thr[e] : make_float2(0.0f, 0.0f);
      wid_r[i] = e < n_well ? well_idx[e] : 0;
    }
  }
  // ill-conditioned components, direct form, lane = point; a term 2^-60 below
  // the point's largest well lane state is nothing in the sum and is not
  // finished (a routed component that is the point's largest is finished)
  __syncthreads();
  if (lane < PTS) {
    float mw = kEmpty;
    for (int w2 = 0; w2 < 4; ++w2) mw = fmaxf(mw, stw[w2][lane].x);
    // maximum kept in fp64: routed components can have log-densities of 1e4
    // log2 units, where an fp32 value is off by up to 5e-4
    double mi = -INFINITY;
    float si = 0.0f;
    // rows >= n (zero rows of the fp32 tile) are skipped with the split tile
    const int64_t row = n0 + lane;
    auto take = [&](double l) {
      if (l > mi) {
        si = __fmaf_rn(si, exp2_fast((float)(mi - l)), 1.0f);
        mi = l;
      } else if (l > -INFINITY) {
        si += exp2_fast((float)(l - mi));
      }
    };
    if constexpr (B16) {
      // The first 8 dimensions of the point's row are read once for all of the
      // wave's ill components (lane = point, so these reads are not
      // coalesced); the first chunk dismisses almost every component.  The
      // first-chunk operands of up to kIllStage components at a time are
      // staged in LDS by the whole workgroup (one memory round trip per batch
      // instead of one per component).  Same sums, in the same order, as the
      // plain bounded form; the partial sums only grow, so an earlier
      // dismissal gives the same -inf.
      constexpr int H = 8;
      static_assert(PTS == 64, "every thread of the workgroup stages operands");
      IllStage& ist = *reinterpret_cast<IllStage*>(smem + IST_OFF);
      const bool live = row < n;
      float xh[H];
#pragma unroll
      for (int q4 = 0; q4 < H / 4; ++q4) {
        const int j = 4 * q4;
        float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
        if (live && vec4) {
          if (j < d) v = *reinterpret_cast<const float4*>(x + row * d + j);
        } else if (live) {
          v.x = j < d ? x[row * d + j] : 0.0f;
          v.y = j + 1 < d ? x[row * d + j + 1] : 0.0f;
          v.z = j + 2 < d ? x[row * d + j + 2] : 0.0f;
          v.w = j + 3 < d ? x[row * d + j + 3] : 0.0f;
        }
        xh[j] = v.x;
        xh[j + 1] = v.y;
        xh[j + 2] = v.z;
        xh[j + 3] = v.w;
      }
      for (int base = 0; base < n_ill; base += kIllStage) {
        const int cnt = n_ill - base < kIllStage ? n_ill - base : kIllStage;
        // thread t: half t % 2 (dimensions 4 (t % 2) .. + 3) of component t / 2
        if (tid < 2 * cnt) {
          const int i = tid >> 1, hf = tid & 1;
          const int cp = ill_idx[base + i];
          const float4 mv = *reinterpret_cast<const float4*>(dmu + (size_t)cp * D64 + 4 * hf);
          const double2 h0 = *reinterpret_cast<const double2*>(dh + (size_t)cp * D64 + 4 * hf);
          const double2 h1 = *reinterpret_cast<const double2*>(dh + (size_t)cp * D64 + 4 * hf + 2);
          *reinterpret_cast<float4*>(&ist.mu[i][4 * hf]) = mv;
          *reinterpret_cast<double2*>(&ist.h[i][4 * hf]) = h0;
          *reinterpret_cast<double2*>(&ist.h[i][4 * hf + 2]) = h1;
          if (hf == 0) {
            ist.c[i] = cdir[cp];
            ist.comp[i] = cp;
          }
        }
        __syncthreads();
        // components base + kl, kl = wave, wave + 4, ...: the order of the
        // unbatched loop, as kIllStage is a multiple of 4
        if (live) {
          for (int kl = wave; kl < cnt; kl += 4) {
            const double c = ist.c[kl];
            const double bnd = c - ((double)mw - 60.0);
            double acc = 0.0;
#pragma unroll
            for (int j = 0; j < H; ++j) {
              if (j < d) {
                const double t = (double)xh[j] - (double)ist.mu[kl][j];
                acc = fma(t * t, ist.h[kl][j], acc);
              }
            }
            double l = -INFINITY;
            if (__ballot(!(acc > bnd)) != 0ull) {
              const int cp = ist.comp[kl];
              l = ill_logit_bounded_gr(x + row * d, d, vec4, dmu + (size_t)cp * D64,
                                       dh + (size_t)cp * D64, c, bnd, acc, H);
            }
            take(l);
          }
        }
        __syncthreads();                        // the next batch reuses the staging
      }
    } else {
      for (int ki = wave; ki < n_ill; ki += 4) {
        const int comp = ill_idx[ki];
        const double c = cdir[comp];
        const double bnd = c - ((double)mw - 60.0);
        take(ill_logit_bounded<D64>(xs + lane * P, dmu + (size_t)comp * D64,
                                    dh + (size_t)comp * D64, c, bnd));
      }
    }
    sti[wave][lane] = make_float2((float)mi, si);
    stim[wave][lane] = mi;
  }
  if (thr_lds) {
#pragma unroll
    for (int i = 0; i < NTHR; ++i) {
      const int e = tid + 256 * i;
      if (e < kpad_w) {
        thr_s[e] = thr_r[i];
        wid_s[e] = wid_r[i];
      }
    }
  }
  __syncthreads();
  if (tid < PTS) {
    float mm = -INFINITY, ss = 0.0f;
    for (int w2 = 0; w2 < 4; ++w2) {
      lse_merge(mm, ss, stw[w2][tid].x, stw[w2][tid].y);
      lse_merge(mm, ss, sti[w2][tid].x, sti[w2][tid].y);
    }
    lzm[tid] = mm + __log2f(ss);
    // a lower bound of the 4th largest lane-state maximum: the 4th largest of
    // the waves' two largest (eight distinct lane states)
    float t4[4] = {kEmpty, kEmpty, kEmpty, kEmpty};
    for (int w2 = 0; w2 < 4; ++w2) {
      const float vv[2] = {top2[w2][tid].x, top2[w2][tid].y};
      for (int u = 0; u < 2; ++u) {
        const float v = vv[u];
#pragma unroll
        for (int j = 3; j > 0; --j) {
          if (v > t4[j - 1]) t4[j] = t4[j - 1];
          else if (v > t4[j]) t4[j] = v;
        }
        if (v > t4[0]) t4[0] = v;
      }
    }
    s4m[tid] = t4[3];
  }
  __syncthreads();
  // candidates: lane states whose maximum is within the window of the screening log2 Z
  float XT[16 * NT];                 // candidate mass per lane state, summed below
  unsigned cbits = 0u;               // this lane's candidate lane states, bit 16 blk + v
  // every operand read and every exp2 taken without branches; the pass is
  // compiled once per place of the thresholds (LDS or global memory), so that
  // each read is a plain LDS or global load
  auto cand_pass = [&](const float2* __restrict__ tsrc) {
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int p = 8 * (v >> 2) + 4 * h + (v & 3);
#pragma unroll
      for (int blk = 0; blk < NT; ++blk) {
        const int pp = blk * 32 + p;
        const float mv = blk ? m1[v] : m0[v];
        const float sv = blk ? s1[v] : s0[v];
        const int av = blk ? a1[v] : a0[v];
        const bool valid = av >= 0;
        // refined: within the component's window, or among the point's four
        // largest lane states (those fill the exact top-kT list); refined in
        // full (every component of the lane state) when the screening error of
        // its other components' mass (bound: that mass times the arg-max
        // component's relative error bound) could exceed kFullErr of the
        // point's total
        const float rel = mv - lzm[pp];
        const float s4 = s4m[pp], swx = stw[wave][pp].x;
        const float2 tr = tsrc[valid ? av : 0];
        const float2 tf = valid ? tr : make_float2(0.0f, 0.0f);
        const float er = exp2_fast(rel), ex = exp2_fast(mv - swx);
        const bool full = REFINE & valid & ((sv - 1.0f) * er * tf.y > kFullErr);
        const bool cand =
            valid & (full | (rel > tf.x) | ((mv >= s4) & (rel > -(float)kWideWindow)));
        if (cand) cbits |= 1u << (16 * blk + v);
        XT[16 * blk + v] = cand ? (full ? sv : 1.0f) * ex : 0.0f;
        const bool sig = (bmask != nullptr) & valid & (rel > -kDenseWindow);
        const bool oth = sig & ((sv - 1.0f) * er > kDenseMass);
        if constexpr (B16) {
          // one flag byte per lane state (IllStage's space is free now); the
          // (point, wave) masks are assembled from them below
          unsigned char* fl = smem + IST_OFF;
          fl[pp * 128 + wave * 32 + col] =
              (unsigned char)((cand ? 1 : 0) | (full ? 2 : 0) | (sig ? 4 : 0) | (oth ? 8 : 0));
        } else {
          const unsigned long long bal = __ballot(cand);
          const unsigned long long balf = __ballot(full);
          if (col == 0) {
            cmask[pp][wave] = (unsigned)(bal >> (32 * h));
            fmask[pp][wave] = (unsigned)(balf >> (32 * h));
          }
          if (bmask != nullptr) {
            const unsigned long long bals = __ballot(sig);
            const unsigned long long balo = __ballot(oth);
            if (col == 0) {
              smask[pp][wave] = (unsigned)(bals >> (32 * h));
              omask[pp][wave] = (unsigned)(balo >> (32 * h));
            }
          }
        }
      }
    }
  };
  if (thr_lds) cand_pass(thr_s);
  else cand_pass(thr);
  xpose_levels<16 * NT>(col, [&](auto jc, auto hc, auto oc, bool up) {
    constexpr int j = decltype(jc)::value, half = decltype(hc)::value;
    constexpr int off = decltype(oc)::value;
    const float kt = up ? XT[j + half] : XT[j], st = up ? XT[j] : XT[j + half];
    XT[j] = kt + xshfl<off>(st);
  });
  if (NT == 2 || (col & 1) == 0) cms[wave][xpose_point<NT>(col, h)] = XT[0];
  __syncthreads();
  if constexpr (B16) {
    // thread (point tid / 4, wave tid % 4): its four 32-bit lane-column masks
    // from the 32 flag bytes (bit b of byte c goes to bit c of mask b: four
    // bytes at a time, (w & 0x01010101) * 0x01020408 gathers their bit 0 in
    // bits 24..27 without carries)
    static_assert(4 * PTS == 256, "one thread per (point, wave)");
    const unsigned char* fl = smem + IST_OFF;
    const int p = tid >> 2, w2 = tid & 3;
    const uint4 f0 = *reinterpret_cast<const uint4*>(fl + p * 128 + w2 * 32);
    const uint4 f1 = *reinterpret_cast<const uint4*>(fl + p * 128 + w2 * 32 + 16);
    const unsigned wd[8] = {f0.x, f0.y, f0.z, f0.w, f1.x, f1.y, f1.z, f1.w};
    unsigned mk[4] = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int b = 0; b < 4; ++b)
        mk[b] |= ((((wd[i] >> b) & 0x01010101u) * 0x01020408u) >> 24) << (4 * i);
    cmask[p][w2] = mk[0];
    fmask[p][w2] = mk[1];
    smask[p][w2] = mk[2];
    omask[p][w2] = mk[3];
    __syncthreads();
  }
  // Refinement, spread over the workgroup: the candidates of (point p, wave
  // w2) are listed in (point, wave, lane column, block) order, every thread
  // computes exact log-densities of list entries (relative to the point's
  // screening log2 Z, fp64 sums), and the owner thread of (w2, p) then takes
  // its entries in list order, so the result does not depend on the split.
  {
    const int p = lane, w2 = wave;
    const bool owner = lane < PTS && n0 + lane < n;
    unsigned cm = 0u, fm = 0u;
    int my_c = 0;
    // components of lane state (w2, b): slots 32 kb + b, kb = w2, w2 + 4, ... < n_wkb
    const int nkb_w = n_wkb > w2 ? (n_wkb - w2 + 3) / 4 : 0;
    const int kb_last = w2 + 4 * (nkb_w - 1);
    if (owner) {
      cm = cmask[p][w2];
      fm = fmask[p][w2];
      my_c = __popc(cm & ~fm);
      unsigned f = fm;
      while (f) {
        const int b = __ffs(f) - 1;
        f &= f - 1;
        my_c += nkb_w - (kb_last * kBK + b >= n_well ? 1 : 0);
      }
    }
    rcnt[p * 4 + w2] = owner ? my_c : 0;
    __syncthreads();
    // exclusive scan of rcnt in (point, wave) order, entry t by thread t
    {
      const int v = rcnt[tid];
      int inc = v;
      for (int o = 1; o < 64; o <<= 1) {
        const int t2 = __shfl_up(inc, o);
        if (lane >= o) inc += t2;
      }
      if (lane == 63) rwsum[wave] = inc;
      __syncthreads();
      int before = 0, all = 0;
      for (int q = 0; q < 4; ++q) {
        if (q < wave) before += rwsum[q];
        all += rwsum[q];
      }
      __syncthreads();                          // every thread has read rcnt[tid]
      rcnt[tid] = before + inc - v;
      if (tid == 0) rwsum[4] = all;
    }
    __syncthreads();
    const int total = rwsum[4];
    const int my_base = owner ? rcnt[p * 4 + w2] : 0;
    float mc = -INFINITY, sc = 0.0f;
    int tsl[kT];
    float tl[kT];
#pragma unroll
    for (int j = 0; j < kT; ++j) { tsl[j] = -1; tl[j] = -INFINITY; }
    for (int lo = 0; lo < total; lo += kRefCap) {
      const int hi = total < lo + kRefCap ? total : lo + kRefCap;
      if constexpr (REFINE) {
        if (owner && my_base < hi && my_base + my_c > lo) {
          int j = my_base;
          unsigned msk = cm;
          while (msk && j < hi) {
            const int b = __ffs(msk) - 1;
            msk &= msk - 1;
            if ((fm >> b) & 1u) {
              for (int kb = w2; kb < n_wkb && j < hi; kb += 4) {
                const int slot = kb * kBK + b;
                if (slot >= n_well) break;
                if (j >= lo) rlist[j - lo] = (p << 16) | slot;
                ++j;
              }
            } else {
              if (j >= lo) rlist[j - lo] = (p << 16) | cidx[p][w2 * 32 + b];
              ++j;
            }
          }
        }
        __syncthreads();
        if (B16 && vec4) {
          // kRefLanes lanes per entry: lane g of a group sums, in fp64, the float4
          // chunks g, g + kRefLanes, ... of the row (coalesced over the group),
          // and the group adds its partial sums in a fixed butterfly order.
          // Compiled once per place of the slots' components (LDS or global
          // memory), so that each lookup is a plain LDS or global load.
          constexpr int G = kRefLanes, NCK = D64 / 4 / G;
          const int g = tid & (G - 1);
          auto refine_entries = [&](const int* __restrict__ widx) {
          for (int j = lo + tid / G; j < hi; j += 256 / G) {
            const int e = rlist[j - lo], pp = e >> 16;
            const int comp = widx[e & 0xFFFF];
            const float* xr = x + (n0 + pp) * d;
            const float* mu = dmu + (size_t)comp * D64;
            const double* hh = dh + (size_t)comp * D64;
            const double cd = cdir[comp];
            // every chunk loaded before the arithmetic (no branch between the
            // loads): chunks past d read dimensions 0..3 of the row, and their
            // direct-form weights are the zero padding, so they add exact zeros
            float4 xv[NCK], mv[NCK];
            double2 g0[NCK], g1[NCK];
  #pragma unroll
            for (int t = 0; t < NCK; ++t) {
              const int c4 = 4 * (g + G * t);
              xv[t] = *reinterpret_cast<const float4*>(xr + (c4 < d ? c4 : 0));
              mv[t] = *reinterpret_cast<const float4*>(mu + c4);
              g0[t] = *reinterpret_cast<const double2*>(hh + c4);
              g1[t] = *reinterpret_cast<const double2*>(hh + c4 + 2);
            }
            double acc = 0.0;
  #pragma unroll
            for (int t = 0; t < NCK; ++t) {
              double u;
              u = (double)xv[t].x - (double)mv[t].x; acc = fma(u * u, g0[t].x, acc);
              u = (double)xv[t].y - (double)mv[t].y; acc = fma(u * u, g0[t].y, acc);
              u = (double)xv[t].z - (double)mv[t].z; acc = fma(u * u, g1[t].x, acc);
              u = (double)xv[t].w - (double)mv[t].w; acc = fma(u * u, g1[t].y, acc);
            }
            static_assert(G == 4, "the butterfly below takes four lanes");
            acc += xshfl<1>(acc);
            acc += xshfl<2>(acc);
            if (g == 0) {
              const double ref = lzm[pp] > -INFINITY ? (double)lzm[pp] : 0.0;
              rres[j - lo] = (float)((cd - acc) - ref);
            }
          }
          };
          if (thr_lds) refine_entries(wid_s);
          else refine_entries(well_idx);
        } else {
          for (int j = lo + tid; j < hi; j += 256) {
            const int e = rlist[j - lo], pp = e >> 16;
            int comp;
            if (thr_lds) comp = wid_s[e & 0xFFFF];
            else comp = well_idx[e & 0xFFFF];
            const double ref = lzm[pp] > -INFINITY ? (double)lzm[pp] : 0.0;
            const double l =
                B16 ? ill_logit_gr(x + (n0 + pp) * d, d, vec4, dmu + (size_t)comp * D64,
                                   dh + (size_t)comp * D64, cdir[comp])
                    : ill_logit<D64>(xs + pp * P, dmu + (size_t)comp * D64,
                                     dh + (size_t)comp * D64, cdir[comp]);
            rres[j - lo] = (float)(l - ref);
          }
        }
      } else {
        // screened E-step: every candidate lane state puts its own entry, with
        // its screened log-density, where the owner would have listed it
#pragma unroll
        for (int v = 0; v < 16; ++v) {
#pragma unroll
          for (int blk = 0; blk < NT; ++blk) {
            const int pp = blk * 32 + 8 * (v >> 2) + 4 * h + (v & 3);
            if (((cbits >> (16 * blk + v)) & 1u) && n0 + pp < n) {
              const int pos = rcnt[pp * 4 + wave] + __popc(cmask[pp][wave] & ((1u << col) - 1u));
              if (pos >= lo && pos < hi) {
                const float mv = blk ? m1[v] : m0[v];
                const int av = blk ? a1[v] : a0[v];
                const double ref = lzm[pp] > -INFINITY ? (double)lzm[pp] : 0.0;
                rlist[pos - lo] = (pp << 16) | av;
                rres[pos - lo] = (float)((double)mv - ref);
              }
            }
          }
        }
      }
      __syncthreads();
      if (owner) {
        const int j1 = my_base + my_c < hi ? my_base + my_c : hi;
        for (int j = my_base > lo ? my_base : lo; j < j1; ++j) {
          const float l = rres[j - lo];
          lse_add(mc, sc, l);
          topk_insert(tl, tsl, l, rlist[j - lo] & 0xFFFF);
        }
      }
      __syncthreads();                          // the next pass reuses rlist / rres
    }
    if (owner) {
      rmc[w2][p] = make_float2(mc, sc);
#pragma unroll
      for (int j = 0; j < kT; ++j) {
        rts[w2][j][p] = tsl[j];
        rtl[w2][j][p] = tl[j];
      }
    }
  }
  __syncthreads();
  if (tid < 64) {
    const int p = tid;
    double contrib = 0.0;
    if (p < PTS) {
      const float ref = lzm[p] > -INFINITY ? lzm[p] : 0.0f;
      // screened mass of everything that is not a candidate (ill states are exact)
      float mm = -INFINITY;
      for (int w2 = 0; w2 < 4; ++w2) mm = fmaxf(mm, fmaxf(stw[w2][p].x, sti[w2][p].x));
      float snc = 0.0f;
      if (mm > -INFINITY) {
        for (int w2 = 0; w2 < 4; ++w2) {
          const float2 a = stw[w2][p], b = sti[w2][p];
          if (a.x > -INFINITY) snc += fmaxf(a.y - cms[w2][p], 0.0f) * exp2_fast(a.x - mm);
          if (b.x > -INFINITY) snc += b.y * exp2_fast((float)(stim[w2][p] - (double)mm));
        }
      }
      // merge the per-wave exact candidates (relative to ref) in wave order
      float mc = -INFINITY, sc = 0.0f;
      int tsl[kT];
      float tl[kT];
#pragma unroll
      for (int j = 0; j < kT; ++j) { tsl[j] = -1; tl[j] = -INFINITY; }
      for (int w2 = 0; w2 < 4; ++w2) {
        const float2 st2 = rmc[w2][p];
        lse_merge(mc, sc, st2.x, st2.y);
        for (int j2 = 0; j2 < kT; ++j2) {
          const int sl2 = rts[w2][j2][p];
          const float l = rtl[w2][j2][p];
          if (sl2 >= 0) topk_insert(tl, tsl, l, sl2);
        }
      }
      const float mmr = mm - ref;
      float mt = fmaxf(mmr, mc), stot = 0.0f;
      if (mt > -INFINITY) {
        if (mmr > -INFINITY) stot += snc * exp2_fast(mmr - mt);
        if (mc > -INFINITY) stot += sc * exp2_fast(mc - mt);
      }
      const float lzr = mt + __log2f(stot);   // log2 Z - ref
      const int64_t nn = n0 + p;
      if (nn < n) {
        contrib = (double)ref + (double)lzr;
        logz2[nn] = contrib;
#pragma unroll
        for (int j = 0; j < kT; ++j) {
          cslot[nn * kT + j] = tsl[j] >= 0 ? (unsigned short)tsl[j] : kNoSlot;
          cr[nn * kT + j] = tsl[j] >= 0 ? exp2_fast(tl[j] - lzr) : 0.0f;
        }
        // routed components: the ill sums above are -inf for every component more
        // than 2^-60 below the point's largest well lane state, so a finite
        // maximum marks the points k_stats_ill has to take
        {
          double mi_all = -INFINITY;
          for (int w2 = 0; w2 < 4; ++w2) mi_all = fmax(mi_all, stim[w2][p]);
          iflag[nn] = mi_all > -INFINITY ? 1 : 0;
          // cleared here, set by the dense statistics pass where a light
          // component holds more than about 2^-72 of the point
          lflag[nn] = 0;
        }
        if (bmask != nullptr) {
          // 64-component blocks the dense statistics pass takes for this point
          unsigned long long bm = 0ull;
          for (int w2 = 0; w2 < 4; ++w2) {
            if (omask[p][w2] != 0u)
              for (int kb = w2; kb < n_wkb; kb += 4) bm |= 1ull << (kb >> 1);
            unsigned sm = smask[p][w2];
            while (sm) {
              const int b = __ffs(sm) - 1;
              sm &= sm - 1;
              const int slot = cidx[p][w2 * 32 + b];
              bool stored = false;
#pragma unroll
              for (int j = 0; j < kT; ++j) stored = stored || tsl[j] == slot;
              if (!stored) bm |= 1ull << (slot >> 6);
            }
          }
          bmask[nn] = bm;
        }
      }
    }
    for (int off = 32; off > 0; off >>= 1) contrib += __shfl_xor(contrib, off);
    if (lane == 0) ll_part[blockIdx.x] = contrib;
  }
}

// ---------------------------------------------------------------- Step 2: statistics, well set
// Grid: (64-component block, point chunk), 16x16x4 fp32 MFMA.  Wave w owns the
// 16 components 16w .. 16w+15 of the block and works on its own: its
// log-density operand (W and P of its components, 2 * D64 values per lane in
// the MFMA B-operand order of the packed array wq) stays in registers for the
// whole chunk; for every 16-point tile it forms the log-densities of its
// components, takes r = 2^(l - log2 Z) with the refined pairs set to 0
// (k_stats_sparse sums those exactly), and
// contracts r^T [x | x^2] into fp32 accumulators (its 16 components x 2 D64
// columns) that are folded into the workgroup's fp64 partial every kFlush
// iterations; N_k is summed on the vector ALU.  The log-density accumulator
// layout (point 4(l/16)+v, component l%16) is the B-operand layout of the
// statistic MFMA, so r stays in registers.  The waves share only the X tile:
// 32 points per iteration, double-buffered in LDS and loaded one iteration
// ahead, one barrier per iteration.
//
// The log-density chain yields l - log2 Z directly: for every group of 32
// dimensions its x steps, its x^2 steps, then one step that adds the group's
// share of the constant and -log2 Z / NGB (operands from the packed bias
// steps and the point's log2 Z).  The running sum then stays near the result
// instead of passing through values of the size of sum mu^2/var, which keeps
// the fp32 rounding of far-from-centre pairs about ten times smaller (their
// share of a variance can be large when a component sits on one point).
// Orders.  Log-density step s (< D64/4) of lane l uses dimension
// 16(s/4) + 4(l/16) + s%4, so a lane reads 4 dimensions with one float4.
// Statistic column block c = 4g + e (x part; the x^2 part likewise) row i is
// dimension 64g + 4i + e, so a lane reads the 4 blocks of a group with one
// float4 too.
typedef float f4v __attribute__((ext_vector_type(4)));
__device__ __forceinline__ f4v mfma16(float a, float b, f4v c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// ISO (tied variances): per 32-dimension group the x steps, one norm step
// (each lane's sum of squares over its 8 dimensions of the group against
// -1/2 log2(e) / var, the MFMA summing the four lane groups) and the bias
// step; the statistics contract r^T x on MFMA and add r ||x||^2 on the vector
// ALU, written into dimension 0 of Q (the isotropic Q is the sum over the
// dimensions).
template <int D64, bool ISO>
__global__ __launch_bounds__(256, D64 <= 128 ? 2 : 1) void k_stats_well(
    const float* __restrict__ x, int64_t n, int d, int vec4, const float* __restrict__ wq,
    const float* __restrict__ cw, const int* __restrict__ counts,
    const double* __restrict__ logz2, const unsigned short* __restrict__ cslot,
    const unsigned long long* __restrict__ bmask, int nch, int64_t chunk_pts,
    const unsigned char* __restrict__ sflag, unsigned char* __restrict__ lflag,
    double* __restrict__ part) {
  constexpr int P = D64 + 4;
  constexpr int NS = D64 / 4;                   // MFMA steps per chain
  constexpr int NG = D64 / 64;                  // float4 column groups per part
  constexpr int NB = D64 / 16;                  // 16-column blocks per part
  constexpr int NGB = D64 / 32;                 // 32-dimension groups (bias steps)
  constexpr int WQS = ISO ? wq_steps_iso(D64) : wq_steps(D64);
  constexpr int SB = ISO ? NS + NGB : 2 * NS;   // first bias step
  constexpr int NACC = ISO ? NB : 2 * NB;       // accumulator blocks
  constexpr int PTS = 32;                       // points per iteration (two tiles)
  constexpr int Q4 = D64 / 4;
  constexpr int LD = PTS * Q4 / 256;            // float4 per thread per X tile
  constexpr int STRIDE = 1 + 2 * D64;
  static_assert(kT == 4, "refined lists are loaded as int4");
  static_assert(LD >= 1 && PTS * Q4 % 256 == 0, "tile split");
  __shared__ __align__(16) float xs[2][PTS * P];
  __shared__ float2 lzb[2][PTS];                // -log2 Z / NGB as a (hi, lo) pair
  __shared__ unsigned long long rbb[2][PTS];
  __shared__ unsigned pqo[2][PTS];              // the tile's points (offsets from p0, ~0u: none)
  __shared__ unsigned long long lbits;          // light slots of this block
  __shared__ unsigned qpt[kStatsWin + PTS];     // queued points (offsets from the chunk start)
  static_assert(kStatsWin == 16 * 256, "a window is 16 points per thread");
  __shared__ int qsum[4];
  const int kb = blockIdx.x / nch, chunk = blockIdx.x % nch;
  if (2 * kb >= counts[2]) return;              // counts[2]: well blocks of 32
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int i16 = lane & 15, k4 = lane >> 4;
  const int64_t p0 = (int64_t)chunk * chunk_pts;
  const int64_t p1 = p0 + chunk_pts < n ? p0 + chunk_pts : n;
  double* pw = part + (size_t)blockIdx.x * kWB * STRIDE;
  if (p0 >= p1) {
    for (int i = tid; i < kWB * STRIDE; i += 256) pw[i] = 0.0;
    return;
  }
  const int grp = kb * 4 + wave;                // 16-component group
  if (wave == 0) {
    const int sl = kb * kWB + lane;
    const unsigned long long lb =
        __ballot(sflag != nullptr && sl < counts[0] && sflag[sl] != 0);
    if (lane == 0) lbits = lb;
  }
  float wb[WQS];
#pragma unroll
  for (int s2 = 0; s2 < WQS; ++s2) wb[s2] = wq[((size_t)grp * WQS + s2) * 64 + lane];

  // ---- X tile: global -> registers -> LDS
  float4 px[LD];
  float2 plz = make_float2(-INFINITY, 0.0f);
  unsigned long long prb = 0ull;
  unsigned ppo = ~0u;
  // tile i holds queue entries PTS i .. PTS i + PTS - 1 (rows past qn are zero)
  int qn = 0;                                   // queued points (uniform)
  auto load_regs = [&](int i) {
#pragma unroll
    for (int j = 0; j < LD; ++j) {
      const int idx = tid + 256 * j, r = idx / Q4, c = (idx % Q4) * 4;
      const int e = PTS * i + r;
      const int64_t nn = e < qn ? p0 + qpt[e] : p1;
      float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
      if (vec4) {
        if (nn < p1 && c < d) v = *reinterpret_cast<const float4*>(x + nn * d + c);
      } else if (nn < p1) {
        const float* xr = x + nn * d;
        v.x = c < d ? xr[c] : 0.f;
        v.y = c + 1 < d ? xr[c + 1] : 0.f;
        v.z = c + 2 < d ? xr[c + 2] : 0.f;
        v.w = c + 3 < d ? xr[c + 3] : 0.f;
      }
      px[j] = v;
    }
    if (tid < PTS) {
      const int e = PTS * i + tid;
      const int64_t nn = e < qn ? p0 + qpt[e] : p1;
      plz = make_float2(-INFINITY, 0.0f);
      prb = 0ull;
      ppo = nn < p1 ? (unsigned)(nn - p0) : ~0u;
      if (nn < p1) {
        const double b64 = -logz2[nn] / NGB;
        const float bh = (float)b64;
        plz = make_float2(bh, (float)(b64 - (double)bh));
        const ushort4 sl = *reinterpret_cast<const ushort4*>(cslot + nn * kT);
        const int v4[4] = {sl.x, sl.y, sl.z, sl.w};
#pragma unroll
        for (int j = 0; j < kT; ++j)
          if (v4[j] != kNoSlot && v4[j] / kWB == kb) prb |= 1ull << (v4[j] % kWB);
      }
    }
  };
  auto store_regs = [&](int buf) {
#pragma unroll
    for (int j = 0; j < LD; ++j) {
      const int idx = tid + 256 * j, r = idx / Q4, c = (idx % Q4) * 4;
      *reinterpret_cast<float4*>(&xs[buf][r * P + c]) = px[j];
    }
    if (tid < PTS) {
      lzb[buf][tid] = plz;
      rbb[buf][tid] = prb;
      pqo[buf][tid] = ppo;
    }
  };

  f4v acc[NACC];
#pragma unroll
  for (int c = 0; c < NACC; ++c) acc[c] = f4v{0.f, 0.f, 0.f, 0.f};
  float nkacc = 0.0f;
  float qacc = 0.0f;                            // ISO: sum of r ||x||^2
  bool first = true;
  const int myc = wave * 16 + i16;              // this lane's component in the block
  __syncthreads();                              // lbits
  // a light component is left out here and recomputed exactly; the points
  // where it comes within 2^-72 of log2 Z are flagged for that
  const bool mylight = ((lbits >> myc) & 1ull) != 0ull;

  // fp32 accumulators -> fp64 partial.  Register v of block c at lane l is
  // column 4(l/16) + v of the block: dimension 64 (c/4 % NG) + 4 (4 k4 + v) + c % 4.
  auto flush = [&]() {
    float nk2 = nkacc + __shfl_xor(nkacc, 16);
    nk2 += __shfl_xor(nk2, 32);
    float q2 = 0.0f;
    if constexpr (ISO) {
      q2 = qacc + __shfl_xor(qacc, 16);
      q2 += __shfl_xor(q2, 32);
    }
    double* row = pw + (size_t)myc * STRIDE;
    if (k4 == 0) row[0] = first ? (double)nk2 : row[0] + (double)nk2;
#pragma unroll
    for (int part2 = 0; part2 < 2; ++part2) {
#pragma unroll
      for (int g = 0; g < NG; ++g) {
        double o[16];
#pragma unroll
        for (int e = 0; e < 4; ++e)
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const int dim = 64 * g + 4 * (4 * k4 + v) + e;
            o[4 * e + v] = first ? 0.0 : row[1 + part2 * D64 + dim];
          }
#pragma unroll
        for (int e = 0; e < 4; ++e)
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const int dim = 64 * g + 4 * (4 * k4 + v) + e;
            if (ISO && part2 == 1) {
              // dimension 0 (lane group 0) carries the whole isotropic Q
              row[1 + D64 + dim] = o[4 * e + v] + (dim == 0 ? (double)q2 : 0.0);
            } else {
              const int c = part2 * NB + 4 * g + e;
              row[1 + part2 * D64 + dim] = o[4 * e + v] + (double)acc[c][v];
              acc[c][v] = 0.0f;
            }
          }
      }
    }
    nkacc = 0.0f;
    qacc = 0.0f;
    first = false;
  };

  // The chunk is taken in windows of kStatsWin points: the points of a window
  // that need this block (every point when bmask is null) are appended to the
  // queue in point order, the full tiles of the queue are processed (at the
  // chunk's end also the partial one) and the rest moves to the queue's front.
  const unsigned long long kbit = 1ull << (kb & 63);
  int tiles = 0;                                // tiles processed (flush schedule)
  for (int64_t wb0 = p0; wb0 < p1; wb0 += kStatsWin) {
    const int64_t we = wb0 + kStatsWin < p1 ? wb0 + kStatsWin : p1;
    {
      // thread t takes points wb0 + 16 t .. wb0 + 16 t + 15
      const int64_t a = wb0 + 16 * tid;
      unsigned sel = 0u;
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int64_t pt = a + e;
        if (pt < we && (bmask == nullptr || (bmask[pt] & kbit) != 0ull)) sel |= 1u << e;
      }
      const int c = __popc(sel);
      int inc = c;
      for (int o = 1; o < 64; o <<= 1) {
        const int t2 = __shfl_up(inc, o);
        if (lane >= o) inc += t2;
      }
      if (lane == 63) qsum[wave] = inc;
      __syncthreads();
      int pos = qn + inc - c, all = 0;
#pragma unroll
      for (int w2 = 0; w2 < 4; ++w2) {
        if (w2 < wave) pos += qsum[w2];
        all += qsum[w2];
      }
      while (sel) {
        const int e = __ffs(sel) - 1;
        sel &= sel - 1;
        qpt[pos++] = (unsigned)(a + e - p0);
      }
      qn += all;
      __syncthreads();                          // queue complete, qsum free
    }
    const int nt = we >= p1 ? (qn + PTS - 1) / PTS : qn / PTS;
    if (nt > 0) {
  load_regs(0);
  store_regs(0);
  for (int i = 0; i < nt; ++i) {
    const int cur = i & 1;
    __syncthreads();                            // tile i in xs[cur]; xs[cur ^ 1] free
    if (i + 1 < nt) load_regs(i + 1);
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      // log-densities of points t*16 .. t*16+15 against this wave's components
      f4v la = {0.f, 0.f, 0.f, 0.f};
      const float* xr = &xs[cur][(t * 16 + i16) * P + 4 * k4];
      // A operand of the bias steps: -log2 Z / NGB of row point i16 as a
      // (hi, lo) pair in lane groups 0 and 2, 1 in lane group 1, 0 in group 3
      const float2 bz = lzb[cur][t * 16 + i16];
      const float ab = k4 == 0 ? bz.x : (k4 == 1 ? 1.0f : (k4 == 2 ? bz.y : 0.0f));
      // wide D: keep each group's operand loads in their group (hoisting all
      // of them exhausts the registers)
      constexpr bool kPin = D64 > 128;
      float nrm = 0.0f;                         // ISO: this lane's sum of squares
#pragma unroll
      for (int b = 0; b < NGB; ++b) {
        const float4 u0 = *reinterpret_cast<const float4*>(xr + 32 * b);
        const float4 u1 = *reinterpret_cast<const float4*>(xr + 32 * b + 16);
        const int j0 = 8 * b;                   // steps of dims 32b .. 32b+31
        la = mfma16(u0.x, wb[j0], la);
        la = mfma16(u0.y, wb[j0 + 1], la);
        la = mfma16(u0.z, wb[j0 + 2], la);
        la = mfma16(u0.w, wb[j0 + 3], la);
        la = mfma16(u1.x, wb[j0 + 4], la);
        la = mfma16(u1.y, wb[j0 + 5], la);
        la = mfma16(u1.z, wb[j0 + 6], la);
        la = mfma16(u1.w, wb[j0 + 7], la);
        if constexpr (ISO) {
          const float sq = ((u0.x * u0.x + u0.y * u0.y) + (u0.z * u0.z + u0.w * u0.w)) +
                           ((u1.x * u1.x + u1.y * u1.y) + (u1.z * u1.z + u1.w * u1.w));
          nrm += sq;
          la = mfma16(sq, wb[NS + b], la);
        } else {
          la = mfma16(u0.x * u0.x, wb[NS + j0], la);
          la = mfma16(u0.y * u0.y, wb[NS + j0 + 1], la);
          la = mfma16(u0.z * u0.z, wb[NS + j0 + 2], la);
          la = mfma16(u0.w * u0.w, wb[NS + j0 + 3], la);
          la = mfma16(u1.x * u1.x, wb[NS + j0 + 4], la);
          la = mfma16(u1.y * u1.y, wb[NS + j0 + 5], la);
          la = mfma16(u1.z * u1.z, wb[NS + j0 + 6], la);
          la = mfma16(u1.w * u1.w, wb[NS + j0 + 7], la);
        }
        la = mfma16(ab, wb[SB + b], la);
        if constexpr (kPin) __builtin_amdgcn_sched_barrier(0);
      }
      // ISO: ||x||^2 of row point i16 (the four lane groups' sums, in a fixed
      // order; every lane of the point gets the same value)
      float nfull = 0.0f;
      if constexpr (ISO) {
        nfull = nrm + __shfl_xor(nrm, 16);
        nfull += __shfl_xor(nfull, 32);
      }
      float r[4];
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int pt = t * 16 + 4 * k4 + v;
        const float e = exp2_fast(la[v]);
        r[v] = (((rbb[cur][pt] >> myc) & 1ull) || mylight) ? 0.0f : e;
        if (mylight && e > 0x1p-72f) {
          const unsigned po = pqo[cur][pt];
          if (po != ~0u) lflag[p0 + po] = 1;
        }
        nkacc += r[v];
        if constexpr (ISO) qacc += r[v] * __shfl(nfull, 4 * k4 + v);
      }
      // statistics: step v contracts points t*16 + 4k + v (k = 0..3)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const float* yr = &xs[cur][(t * 16 + 4 * k4 + v) * P + 4 * i16];
#pragma unroll
        for (int g = 0; g < NG; ++g) {
          const float4 y = *reinterpret_cast<const float4*>(yr + 64 * g);
          acc[4 * g + 0] = mfma16(y.x, r[v], acc[4 * g + 0]);
          acc[4 * g + 1] = mfma16(y.y, r[v], acc[4 * g + 1]);
          acc[4 * g + 2] = mfma16(y.z, r[v], acc[4 * g + 2]);
          acc[4 * g + 3] = mfma16(y.w, r[v], acc[4 * g + 3]);
          if constexpr (!ISO) {
            acc[NB + 4 * g + 0] = mfma16(y.x * y.x, r[v], acc[NB + 4 * g + 0]);
            acc[NB + 4 * g + 1] = mfma16(y.y * y.y, r[v], acc[NB + 4 * g + 1]);
            acc[NB + 4 * g + 2] = mfma16(y.z * y.z, r[v], acc[NB + 4 * g + 2]);
            acc[NB + 4 * g + 3] = mfma16(y.w * y.w, r[v], acc[NB + 4 * g + 3]);
          }
          if constexpr (kPin) __builtin_amdgcn_sched_barrier(0);
        }
      }
    }
    if (i + 1 < nt) store_regs(cur ^ 1);
    if ((tiles % kFlush) == kFlush - 1) flush();
    ++tiles;
  }
    }
    // the entries not taken move to the front of the queue
    const int used = PTS * nt < qn ? PTS * nt : qn;
    const int left = qn - used;
    __syncthreads();                            // every read of the queue and the tiles done
    const unsigned keep = tid < left ? qpt[used + tid] : 0u;
    __syncthreads();
    if (tid < left) qpt[tid] = keep;
    qn = left;
  }
  // the last partial sums (zeros when no point of the chunk needs this block)
  if (first || (tiles % kFlush) != 0) flush();
}

// ---------------------------------------------------------------- Step 2: statistics, wide D
// Well set for DW >= 256 (DW a multiple of 128).  A workgroup owns one
// 16-component group and a chunk of points; its NW = DW / 128 waves split the
// dimensions, wave w owning [128 w, 128 w + 128): the W and P steps of those
// dimensions (from the packed operand wq) stay in registers, and its 16-point
// X tiles pass through its own LDS region.  Per tile every wave forms the
// x . W + x^2 . P part of the log-densities over its dimensions in 16-dimension
// subgroups, each summed from zero on fp32 MFMA (x and x^2 steps of the same
// four dimensions in turn, so the running sum stays small) and folded into
// fp64; the waves' fp64 partials are exchanged through LDS and summed in wave
// order, identically in every wave, and the constant and -log2 Z are added in
// fp64.  With hundreds of dimensions the terms reach 1e3 log2 units in total,
// and a single fp32 chain would leave errors of 1e-4 on log2 r, too much for a
// pair that carries the variance of a component sitting on one point.  Then
// r = 2^(sum) (refined pairs set to 0) and each wave contracts r^T [x | x^2]
// over its own dimensions into fp32 accumulators, folded into the
// workgroup's fp64 partial every kFlushWide tiles.  N_k is summed by wave 0.
// ISO (tied variances, every P of a component equal): per lane and pair of its
// four dimensions one step with the pair's sum of squares in place of the two
// x^2 steps, and for the statistics r^T x on MFMA while r ||x||^2 (each wave
// over its dimensions) is summed on the vector ALU into the first Q entry of
// the wave's dimensions; the isotropic Q is the sum of Q over the dimensions.
constexpr int kFlushWide = 256;

template <int DW, bool ISO>
__global__ __launch_bounds__(64 * (DW / 128)) void k_stats_wide(
    const float* __restrict__ x, int64_t n, int d, int vec4, const float* __restrict__ wq,
    const double* __restrict__ cwell, const int* __restrict__ well_idx,
    const int* __restrict__ counts, const double* __restrict__ logz2,
    const unsigned short* __restrict__ cslot, const unsigned long long* __restrict__ bmask,
    int nch, int64_t chunk_pts, const unsigned char* __restrict__ sflag,
    unsigned char* __restrict__ lflag, double* __restrict__ part) {
  constexpr int NW = DW / 128, DQ = 128, P = DQ + 4;
  constexpr int NS = DW / 4, WQS = wq_steps(DW);
  constexpr int SW = DQ / 4, NBQ = DQ / 16, NG = DQ / 64;
  constexpr int STRIDE = 1 + 2 * DW;
  constexpr int LD = 16 * DQ / 4 / 64;          // float4 per lane per X tile
  static_assert(kT == 4, "refined lists are loaded as ushort4");
  __shared__ __align__(16) float xs[NW][16 * P];
  __shared__ double lpart[NW][4][64];
  constexpr int WPT = 8, WIN = WPT * 64 * NW;   // points per thread and per queue window
  __shared__ unsigned qpt[WIN + 16];            // queued points (offsets from the chunk start)
  __shared__ int qsum[NW];
  const int g = blockIdx.x / nch, chunk = blockIdx.x % nch;
  const int n_well = counts[0];
  if (16 * g >= n_well) return;                // no well component in this group
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int i16 = lane & 15, k4 = lane >> 4;
  const int64_t p0 = (int64_t)chunk * chunk_pts;
  const int64_t p1 = p0 + chunk_pts < n ? p0 + chunk_pts : n;
  double* pw = part + (size_t)blockIdx.x * 16 * STRIDE;
  if (p0 >= p1) {
    for (int i = tid; i < 16 * STRIDE; i += 64 * NW) pw[i] = 0.0;
    return;
  }
  const int dq0 = DQ * wave;                    // this wave's first dimension
  // this lane's component (B-operand column i16): its expanded-form constant
  const int myslot = 16 * g + i16;
  const double cst = myslot < n_well ? cwell[well_idx[myslot]] : -INFINITY;
  // a light component is left out here and recomputed exactly; the points
  // where it comes within 2^-72 of log2 Z are flagged for that
  const bool mylight = sflag != nullptr && myslot < n_well && sflag[myslot] != 0;
  float wb[2 * SW];
#pragma unroll
  for (int s2 = 0; s2 < SW; ++s2) {
    wb[s2] = wq[((size_t)g * WQS + SW * wave + s2) * 64 + lane];
    wb[SW + s2] = wq[((size_t)g * WQS + NS + SW * wave + s2) * 64 + lane];
  }

  // this wave's 16 x 128 block of the next tile, in registers; lanes 0..15
  // also hold the tile's log2 Z and refined-slot mask (bits of this group)
  float4 px[LD];
  double plz = INFINITY;
  unsigned prb = 0u;
  unsigned ppo = ~0u;
  // tile i holds queue entries 16 i .. 16 i + 15 (rows past qn are zero)
  int qn = 0;                                   // queued points (uniform)
  auto load_regs = [&](int i) {
#pragma unroll
    for (int j = 0; j < LD; ++j) {
      const int idx = lane + 64 * j, r = idx / (DQ / 4), c = dq0 + (idx % (DQ / 4)) * 4;
      const int e = 16 * i + r;
      const int64_t nn = e < qn ? p0 + qpt[e] : p1;
      float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
      if (vec4) {
        if (nn < p1 && c < d) v = *reinterpret_cast<const float4*>(x + nn * d + c);
      } else if (nn < p1) {
        const float* xr = x + nn * d;
        v.x = c < d ? xr[c] : 0.f;
        v.y = c + 1 < d ? xr[c + 1] : 0.f;
        v.z = c + 2 < d ? xr[c + 2] : 0.f;
        v.w = c + 3 < d ? xr[c + 3] : 0.f;
      }
      px[j] = v;
    }
    if (lane < 16) {
      const int e = 16 * i + lane;
      const int64_t nn = e < qn ? p0 + qpt[e] : p1;
      plz = INFINITY;
      prb = 0u;
      ppo = nn < p1 ? (unsigned)(nn - p0) : ~0u;
      if (nn < p1) {
        plz = logz2[nn];
        const ushort4 sl = *reinterpret_cast<const ushort4*>(cslot + nn * kT);
        const int v4[4] = {sl.x, sl.y, sl.z, sl.w};
#pragma unroll
        for (int j = 0; j < kT; ++j)
          if (v4[j] != kNoSlot && (v4[j] >> 4) == g) prb |= 1u << (v4[j] & 15);
      }
    }
  };
  auto store_regs = [&]() {
#pragma unroll
    for (int j = 0; j < LD; ++j) {
      const int idx = lane + 64 * j, r = idx / (DQ / 4), c = (idx % (DQ / 4)) * 4;
      *reinterpret_cast<float4*>(&xs[wave][r * P + c]) = px[j];
    }
  };

  constexpr int NACC = ISO ? NBQ : 2 * NBQ;
  f4v acc[NACC];
#pragma unroll
  for (int c = 0; c < NACC; ++c) acc[c] = f4v{0.f, 0.f, 0.f, 0.f};
  float nkacc = 0.0f;
  float qacc = 0.0f;                            // ISO: sum of r ||x||^2 over this wave's dims
  bool first = true;
  // fp32 accumulators -> fp64 partial.  Register v of block c at lane l is
  // column 4(l/16) + v of the block: local dimension 64 (c/4 % NG) + 4 (4 k4 + v) + c % 4.
  auto flush = [&]() {
    double* row = pw + (size_t)i16 * STRIDE;
    if (wave == 0) {
      float nk2 = nkacc + __shfl_xor(nkacc, 16);
      nk2 += __shfl_xor(nk2, 32);
      if (k4 == 0) row[0] = first ? (double)nk2 : row[0] + (double)nk2;
    }
#pragma unroll
    for (int c = 0; c < 2 * NBQ; ++c) {
      const int part2 = c / NBQ, gg = (c % NBQ) / 4, e = c % 4;
      double* dst = row + 1 + part2 * DW + dq0 + 64 * gg + 16 * k4 + e;
      double o[4];
#pragma unroll
      for (int v = 0; v < 4; ++v) o[v] = first ? 0.0 : dst[4 * v];
      if constexpr (ISO) {
        if (c >= NBQ) {
          // the wave's r ||x||^2 in its first dimension's entry, zeros elsewhere
          float q2 = qacc + __shfl_xor(qacc, 16);
          q2 += __shfl_xor(q2, 32);
#pragma unroll
          for (int v = 0; v < 4; ++v)
            dst[4 * v] = o[v] + (c == NBQ && k4 == 0 && v == 0 ? (double)q2 : 0.0);
          continue;
        }
      }
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        dst[4 * v] = o[v] + (double)acc[c % NACC][v];
        acc[c % NACC][v] = 0.0f;
      }
    }
    nkacc = 0.0f;
    qacc = 0.0f;
    first = false;
  };

  // Windows of WIN points: the points that need this group's 64-component
  // block (every point when bmask is null) are queued in point order, the
  // full 16-point tiles of the queue are processed (at the chunk's end also
  // the partial one) and the rest moves to the queue's front.
  const unsigned long long kbit = 1ull << ((g >> 2) & 63);
  int tiles = 0;                                // tiles processed (flush schedule)
  for (int64_t wb0 = p0; wb0 < p1; wb0 += WIN) {
    const int64_t we = wb0 + WIN < p1 ? wb0 + WIN : p1;
    {
      const int64_t a = wb0 + WPT * tid;
      unsigned sel = 0u;
#pragma unroll
      for (int e = 0; e < WPT; ++e) {
        const int64_t pt = a + e;
        if (pt < we && (bmask == nullptr || (bmask[pt] & kbit) != 0ull)) sel |= 1u << e;
      }
      const int c = __popc(sel);
      int inc = c;
      for (int o = 1; o < 64; o <<= 1) {
        const int t2 = __shfl_up(inc, o);
        if (lane >= o) inc += t2;
      }
      if (lane == 63) qsum[wave] = inc;
      __syncthreads();
      int pos = qn + inc - c, all = 0;
#pragma unroll
      for (int w2 = 0; w2 < NW; ++w2) {
        if (w2 < wave) pos += qsum[w2];
        all += qsum[w2];
      }
      while (sel) {
        const int e = __ffs(sel) - 1;
        sel &= sel - 1;
        qpt[pos++] = (unsigned)(a + e - p0);
      }
      qn += all;
      __syncthreads();                          // queue complete, qsum free
    }
    const int nt = we >= p1 ? (qn + 15) / 16 : qn / 16;
    if (nt > 0) {
  load_regs(0);
  for (int i = 0; i < nt; ++i) {
    store_regs();
    unsigned rbv[4], pov[4];
    double lzv[4];
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      rbv[v] = __shfl(prb, 4 * k4 + v);
      lzv[v] = __shfl(plz, 4 * k4 + v);
      pov[v] = __shfl(ppo, 4 * k4 + v);
    }
    __builtin_amdgcn_wave_barrier();
    if (i + 1 < nt) load_regs(i + 1);
    // x . W + x^2 . P of the tile's 16 points against the group's 16
    // components over this wave's dimensions, 16 dimensions per fp32 sum
    double t64[4] = {0.0, 0.0, 0.0, 0.0};
    const float* xr = &xs[wave][i16 * P + 4 * k4];
    float ssl = 0.0f;                           // ISO: point i16's squares over this lane's dims
#pragma unroll
    for (int q = 0; q < DQ / 16; ++q) {
      const float4 u = *reinterpret_cast<const float4*>(xr + 16 * q);
      f4v la = {0.f, 0.f, 0.f, 0.f};
      if constexpr (ISO) {
        // P of the lane's first dimension: equal for its four (zero x past d)
        const float sxy = u.x * u.x + u.y * u.y, szw = u.z * u.z + u.w * u.w;
        ssl += sxy + szw;
        la = mfma16(u.x, wb[4 * q], la);
        la = mfma16(u.y, wb[4 * q + 1], la);
        la = mfma16(sxy, wb[SW + 4 * q], la);
        la = mfma16(u.z, wb[4 * q + 2], la);
        la = mfma16(u.w, wb[4 * q + 3], la);
        la = mfma16(szw, wb[SW + 4 * q], la);
      } else {
        la = mfma16(u.x, wb[4 * q], la);
        la = mfma16(u.x * u.x, wb[SW + 4 * q], la);
        la = mfma16(u.y, wb[4 * q + 1], la);
        la = mfma16(u.y * u.y, wb[SW + 4 * q + 1], la);
        la = mfma16(u.z, wb[4 * q + 2], la);
        la = mfma16(u.z * u.z, wb[SW + 4 * q + 2], la);
        la = mfma16(u.w, wb[4 * q + 3], la);
        la = mfma16(u.w * u.w, wb[SW + 4 * q + 3], la);
      }
#pragma unroll
      for (int v = 0; v < 4; ++v) t64[v] += (double)la[v];
    }
    // ISO: point i16's ||x||^2 over this wave's dimensions (the four lane groups)
    float ssw = 0.0f;
    if constexpr (ISO) {
      ssw = ssl + __shfl_xor(ssl, 16);
      ssw += __shfl_xor(ssw, 32);
    }
#pragma unroll
    for (int v = 0; v < 4; ++v) lpart[wave][v][lane] = t64[v];
    __syncthreads();
    float r[4];
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      double tot = lpart[0][v][lane];
#pragma unroll
      for (int w2 = 1; w2 < NW; ++w2) tot += lpart[w2][v][lane];
      tot += cst - lzv[v];
      const float e = exp2_fast((float)tot);
      r[v] = (((rbv[v] >> i16) & 1u) || mylight) ? 0.0f : e;
      if (mylight && wave == 0 && e > 0x1p-72f && pov[v] != ~0u) lflag[p0 + pov[v]] = 1;
      nkacc += r[v];
    }
    // statistics over this wave's dimensions: step v contracts points 4k + v
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const float* yr = &xs[wave][(4 * k4 + v) * P + 4 * i16];
      if constexpr (ISO) qacc += r[v] * __shfl(ssw, 4 * k4 + v);
#pragma unroll
      for (int gg = 0; gg < NG; ++gg) {
        const float4 y = *reinterpret_cast<const float4*>(yr + 64 * gg);
        acc[4 * gg + 0] = mfma16(y.x, r[v], acc[4 * gg + 0]);
        acc[4 * gg + 1] = mfma16(y.y, r[v], acc[4 * gg + 1]);
        acc[4 * gg + 2] = mfma16(y.z, r[v], acc[4 * gg + 2]);
        acc[4 * gg + 3] = mfma16(y.w, r[v], acc[4 * gg + 3]);
        if constexpr (!ISO) {
          acc[NBQ + 4 * gg + 0] = mfma16(y.x * y.x, r[v], acc[NBQ + 4 * gg + 0]);
          acc[NBQ + 4 * gg + 1] = mfma16(y.y * y.y, r[v], acc[NBQ + 4 * gg + 1]);
          acc[NBQ + 4 * gg + 2] = mfma16(y.z * y.z, r[v], acc[NBQ + 4 * gg + 2]);
          acc[NBQ + 4 * gg + 3] = mfma16(y.w * y.w, r[v], acc[NBQ + 4 * gg + 3]);
        }
      }
    }
    if ((tiles % kFlushWide) == kFlushWide - 1) flush();
    ++tiles;
    __syncthreads();                            // this tile's LDS reads before the next writes
  }
    }
    // the entries not taken move to the front of the queue
    const int used = 16 * nt < qn ? 16 * nt : qn;
    const int left = qn - used;
    __syncthreads();
    const unsigned keep = tid < left ? qpt[used + tid] : 0u;
    __syncthreads();
    if (tid < left) qpt[tid] = keep;
    qn = left;
  }
  // the last partial sums (zeros when no point of the chunk needs this group)
  if (first || (tiles % kFlushWide) != 0) flush();
}

// ---------------------------------------------------------------- Step 2: refined pairs
// The stored refined pairs (at most kT per point, the pairs that carry a
// component's mass) are summed exactly in fp64, grouped by bucket: a bucket is
// sparse_cb(D64) consecutive well slots.  Three light passes put the pairs of
// every bucket into one contiguous list, in a fixed order:
//   k_sparse_count    per unit (a contiguous range of points): pairs per bucket
//   k_sparse_scan     exclusive prefix over (bucket, unit), bucket-major
//   k_sparse_scatter  per unit: every pair to its bucket's segment, the unit's
//                     points taken 64 at a time, slot rank j outer, lanes inner
// and k_stats_sparse sums each bucket's list, split into parts, in list order.
// Integer counts make the lists, and so the sums, independent of scheduling.
struct SPair {
  int64_t pt;   // point index
  float r;      // exact responsibility
  int c;        // component slot within the bucket
};

__host__ __device__ constexpr int sparse_cb(int D64) {
  return D64 <= 128 ? 32 : (D64 <= 256 ? 16 : (D64 <= 512 ? 8 : 4));
}
// k_stats_sparse waves per workgroup: eight, so that several waves share each
// SIMD and hide one another's LDS and fp64 latencies.  Each wave owns C/8
// slots of the bucket, or, for buckets of four slots (the widest rows), one
// slot and half of the dimensions.
constexpr int kSparseWaves = 8;
__host__ __device__ constexpr int sparse_lcb(int D64) {
  return D64 <= 128 ? 5 : (D64 <= 256 ? 4 : (D64 <= 512 ? 3 : 2));
}
constexpr int kSparseTab = 1 << 18;     // (bucket, unit) table entries at most
// k_stats_sparse: batches of rows in flight into registers while one is summed
constexpr int kSparseDepth = 3;
static_assert(kSparseDepth <= 3, "records are stored four batches ahead");

__global__ __launch_bounds__(64) void k_sparse_count(const unsigned short* __restrict__ cslot,
                                                     int64_t n, int64_t upts, int nb, int lcb,
                                                     int nunit, int* __restrict__ gcnt) {
  extern __shared__ int lc[];
  const int u = blockIdx.x, lane = threadIdx.x;
  for (int b = lane; b < nb; b += 64) lc[b] = 0;
  __syncthreads();
  const int64_t p0 = (int64_t)u * upts;
  const int64_t p1 = p0 + upts < n ? p0 + upts : n;
  for (int64_t p = p0 + lane; p < p1; p += 64) {
    const ushort4 s4 = *reinterpret_cast<const ushort4*>(cslot + p * kT);
    if (s4.x != kNoSlot) atomicAdd(&lc[s4.x >> lcb], 1);
    if (s4.y != kNoSlot) atomicAdd(&lc[s4.y >> lcb], 1);
    if (s4.z != kNoSlot) atomicAdd(&lc[s4.z >> lcb], 1);
    if (s4.w != kNoSlot) atomicAdd(&lc[s4.w >> lcb], 1);
  }
  __syncthreads();
  for (int b = lane; b < nb; b += 64) gcnt[(size_t)b * nunit + u] = lc[b];
}

// Exclusive prefix of cnt[0 .. tot) into off[0 .. tot] (64-bit), off[tot] =
// total.  One workgroup of 1024 threads, 4096 entries per round.
__global__ __launch_bounds__(1024) void k_sparse_scan(const int* __restrict__ cnt, int tot,
                                                      int64_t* __restrict__ off) {
  __shared__ int64_t wsum[16];
  __shared__ int64_t carry_s;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (tid == 0) carry_s = 0;
  __syncthreads();
  for (int base = 0; base < tot; base += 4096) {
    int64_t v[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int i = base + 4 * tid + j;
      v[j] = i < tot ? (int64_t)(unsigned)cnt[i] : 0;
    }
    const int64_t own = v[0] + v[1] + v[2] + v[3];
    int64_t inc = own;
    for (int o = 1; o < 64; o <<= 1) {
      const int64_t t = __shfl_up(inc, o);
      if (lane >= o) inc += t;
    }
    if (lane == 63) wsum[wave] = inc;
    __syncthreads();
    int64_t before = carry_s, all = 0;
    for (int w = 0; w < 16; ++w) {
      if (w < wave) before += wsum[w];
      all += wsum[w];
    }
    int64_t run = before + inc - own;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int i = base + 4 * tid + j;
      if (i < tot) off[i] = run;
      run += v[j];
    }
    __syncthreads();                            // wsum and carry_s read by all
    if (tid == 0) carry_s += all;
    __syncthreads();
  }
  if (tid == 0) off[tot] = carry_s;
}

// Buckets up to which k_sparse_scatter keeps its unit's list positions in LDS
// (8 bytes each); above, it reads each segment start with a scalar load.
constexpr int kScatterCache = 4096;

__host__ __device__ inline size_t scatter_lds(int nb) {
  return (size_t)nb * (nb <= kScatterCache ? sizeof(int64_t) : sizeof(int));
}

// No memory load waits inside the per-bucket loop: on this GPU a wait for a
// vector load also waits for every store before it, so a load there would
// serialise the scattered stores.
__global__ __launch_bounds__(64) void k_sparse_scatter(
    const unsigned short* __restrict__ cslot, const float* __restrict__ cr, int64_t n,
    int64_t upts, int nb, int lcb, int nunit, const int64_t* __restrict__ goff,
    SPair* __restrict__ list) {
  extern __shared__ int64_t cur[];           // cached: next list position per bucket
  int* const pos = reinterpret_cast<int*>(cur);  // else: pairs placed so far per bucket
  const bool cached = nb <= kScatterCache;
  const int u = blockIdx.x, lane = threadIdx.x;
  for (int b = lane; b < nb; b += 64) {
    if (cached) cur[b] = goff[(size_t)b * nunit + u];
    else pos[b] = 0;
  }
  __syncthreads();
  const int64_t p0 = (int64_t)u * upts;
  const int64_t p1 = p0 + upts < n ? p0 + upts : n;
  const unsigned long long below = (1ull << lane) - 1ull;
  int nbits = 0;                             // bits of the largest bucket index
  while ((nb - 1) >> nbits) ++nbits;
  for (int64_t pb = p0; pb < p1; pb += 64) {
    const int64_t p = pb + lane;
    int sl[kT] = {-1, -1, -1, -1};
    float4 r4 = make_float4(0.f, 0.f, 0.f, 0.f);
    if (p < p1) {
      const ushort4 s4 = *reinterpret_cast<const ushort4*>(cslot + p * kT);
      sl[0] = s4.x == kNoSlot ? -1 : s4.x;
      sl[1] = s4.y == kNoSlot ? -1 : s4.y;
      sl[2] = s4.z == kNoSlot ? -1 : s4.z;
      sl[3] = s4.w == kNoSlot ? -1 : s4.w;
      if (sl[0] >= 0 || sl[1] >= 0 || sl[2] >= 0 || sl[3] >= 0)
        r4 = *reinterpret_cast<const float4*>(cr + p * kT);
    }
    const float rr[kT] = {r4.x, r4.y, r4.z, r4.w};
#pragma unroll
    for (int j = 0; j < kT; ++j) {
      const bool valid = sl[j] >= 0;
      const int bk = valid ? (sl[j] >> lcb) : -1;
      if (cached) {
        // the lanes of each bucket found with one ballot per bit of the bucket
        // index; a lane's place is its rank among them (lane order), as in
        // the loop over buckets below
        unsigned long long same = __ballot(valid);
        for (int bb = 0; bb < nbits; ++bb) {
          const bool bit = ((bk >> bb) & 1) != 0;
          const unsigned long long m = __ballot(bit);
          same &= bit ? m : ~m;
        }
        int64_t base = 0;
        if (valid) {
          base = cur[bk];
          SPair e;
          e.pt = p;
          e.r = rr[j];
          e.c = sl[j] & ((1 << lcb) - 1);
          list[base + __popcll(same & below)] = e;
        }
        __builtin_amdgcn_wave_barrier();
        if (valid && (same & below) == 0ull) cur[bk] = base + __popcll(same);
        __builtin_amdgcn_wave_barrier();
        continue;
      }
      unsigned long long act = __ballot(valid);
      while (act) {
        const int leader = __ffsll(act) - 1;
        const int bl = __builtin_amdgcn_readfirstlane(__shfl(bk, leader));
        const unsigned long long same = __ballot(bk == bl);
        const int64_t base =
            cached ? cur[bl] : goff[(size_t)bl * nunit + u] + (int64_t)pos[bl];
        if (bk == bl) {
          SPair e;
          e.pt = p;
          e.r = rr[j];
          e.c = sl[j] & ((1 << lcb) - 1);
          list[base + __popcll(same & below)] = e;
        }
        __builtin_amdgcn_wave_barrier();
        if (lane == leader) {
          if (cached) cur[bl] = base + __popcll(same);
          else pos[bl] += __popcll(same);
        }
        __builtin_amdgcn_wave_barrier();
        act &= ~same;
      }
    }
  }
}

// Sums of one part of one bucket's list.  Batches of NB pairs: while batch t
// is consumed from LDS, the rows of batches t+1 .. t+kSparseDepth are in
// flight into registers, and the records of batch t+4 (stored to LDS at the
// end of batch t), so that no memory round trip is waited for within a
// batch.  Each of the NWV waves owns CW slots of the bucket and one of DS
// parts of the dimensions (DS = 2 for buckets of four slots, else 1) and
// takes its slots' pairs of a batch in order, up to four at a time; lane l owns the
// part's dimensions l, l + 64, ... and adds r x and r x^2 of them in fp64
// (r x is exact), and r itself (N_k, every lane the same sum; lane 0 of the
// first part writes it).
template <int D64>
__global__ __launch_bounds__(64 * kSparseWaves) void k_stats_sparse(
    const float* __restrict__ x, int64_t n, int d, const SPair* __restrict__ list,
    const int64_t* __restrict__ goff, int nunit, int nparts, double* __restrict__ part) {
  constexpr int NWV = kSparseWaves, T = 64 * NWV;
  constexpr int C = sparse_cb(D64);
  constexpr int DS = NWV > C ? NWV / C : 1;      // dimension parts per slot
  constexpr int CW = C * DS / NWV;               // slots per wave
  constexpr int DP = D64 / DS;                   // dimensions per part
  static_assert(CW >= 1 && CW * NWV == C * DS && DP % 64 == 0, "slots and dimensions split evenly");
  constexpr int STRIDE = 1 + 2 * D64;
  // pairs per batch: as many as a wave has lanes up to 128 dimensions (one
  // record per lane), 16 from 512 dimensions (two batches of rows then take
  // 64 to 128 KB of LDS: one workgroup per compute unit, more rows in flight)
  constexpr int NB = D64 <= 128 ? 64 : (D64 <= 256 ? 4096 / D64 : 16);
  static_assert(NB <= 64, "a batch's records are held one per lane");
  constexpr int CPR = D64 / 4;                   // float4 chunks per row
  constexpr int GQ = (NB * CPR + T - 1) / T;     // float4 gathered per thread and batch
  __shared__ __align__(16) float xb[2][NB * D64];
  __shared__ int2 rb[8][NB];                     // (slot in bucket, r bits) per pair
  __shared__ int64_t pb[8][NB];                  // point per pair
  const int bucket = blockIdx.x / nparts, prt = blockIdx.x % nparts;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int64_t lo = goff[(size_t)bucket * nunit], hi = goff[(size_t)(bucket + 1) * nunit];
  const int64_t cnt = hi - lo;
  const int64_t a0 = lo + cnt * prt / nparts, a1 = lo + cnt * (prt + 1) / nparts;
  const int nbatch = (int)((a1 - a0 + NB - 1) / NB);
  const bool vec4 = (d & 3) == 0 && (reinterpret_cast<uintptr_t>(x) & 15) == 0;
  constexpr int NX = DP / 64;                    // dimensions per lane
  // this wave: slots sb .. sb + CW - 1, dimensions dh DP .. dh DP + DP - 1
  const int sb = (wave % (NWV / DS)) * CW, dh = wave / (NWV / DS);
  double accs[CW][NX], accq[CW][NX], accn[CW];
#pragma unroll
  for (int j = 0; j < CW; ++j) {
    accn[j] = 0.0;
#pragma unroll
    for (int u = 0; u < NX; ++u) accs[j][u] = accq[j][u] = 0.0;
  }
  auto batch_len = [&](int t) {
    const int64_t left = a1 - a0 - (int64_t)t * NB;
    return (int)(left < NB ? left : NB);
  };
  auto load_rec = [&](int t) {
    if (tid < NB) {
      const int64_t e = a0 + (int64_t)t * NB + tid;
      if (e < a1) {
        const SPair q = list[e];
        rb[t & 7][tid] = make_int2(q.c, __float_as_int(q.r));
        pb[t & 7][tid] = q.pt;
      }
    }
  };
  // flat float4 index f = tid + T i of a batch: row f / CPR, chunk f % CPR;
  // chunks past the batch load row 0, dims 0..3 (always present) and are
  // zeroed afterwards
  float4 g[kSparseDepth][GQ];
  auto gather = [&](int t, float4 (&g)[GQ]) {
    const int nbt = batch_len(t);
    int64_t pt[GQ];
    bool ok[GQ];
#pragma unroll
    for (int i = 0; i < GQ; ++i) {
      const int f = tid + T * i, e = f / CPR, c4 = 4 * (f % CPR);
      ok[i] = f < NB * CPR && e < nbt && c4 < d;
      pt[i] = ok[i] ? pb[t & 7][e] : 0;
    }
    if (vec4) {
#pragma unroll
      for (int i = 0; i < GQ; ++i) {
        const int c4 = 4 * ((tid + T * i) % CPR);
        g[i] = *reinterpret_cast<const float4*>(x + (ok[i] ? pt[i] * d + c4 : 0));
      }
#pragma unroll
      for (int i = 0; i < GQ; ++i) {
        asm volatile("" : "+v"(g[i].x), "+v"(g[i].y), "+v"(g[i].z), "+v"(g[i].w));
        if (!ok[i]) g[i] = make_float4(0.f, 0.f, 0.f, 0.f);
      }
    } else {
#pragma unroll
      for (int i = 0; i < GQ; ++i) {
        const int c4 = 4 * ((tid + T * i) % CPR);
        float v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e)
          v[e] = ok[i] && c4 + e < d ? x[pt[i] * d + c4 + e] : 0.0f;
        g[i] = make_float4(v[0], v[1], v[2], v[3]);
      }
    }
  };
  auto consume = [&](int t, const float4 (&g)[GQ]) {
    const int xbuf = t & 1;
    float4* const xw = reinterpret_cast<float4*>(xb[xbuf]);
#pragma unroll
    for (int i = 0; i < GQ; ++i)
      if (tid + T * i < NB * CPR) xw[tid + T * i] = g[i];
    __syncthreads();            // rows of batch t, records of batches t .. t+3 in LDS
    // records of batch t+4: loaded now, stored at the end of this batch
    SPair qn = SPair{-1, 0.0f, 0};
    if (t + 4 < nbatch && tid < NB) {
      const int64_t e = a0 + (int64_t)(t + 4) * NB + tid;
      if (e < a1) qn = list[e];
    }
    return qn;
  };
  auto accumulate = [&](int t) {
    const int xbuf = t & 1;
    const int nbt = batch_len(t);
    int2 en = make_int2(0, 0);
    if (lane < nbt) en = rb[t & 7][lane];
    const int cl = en.x - sb;
    // slot by slot (each slot's pairs in list order), up to four pairs at a
    // time (their rows read before the sums)
#pragma unroll
    for (int j = 0; j < CW; ++j) {
      unsigned long long own = __ballot(lane < nbt && cl == j);
      while (own) {
        int e[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          e[i] = own ? __ffsll(own) - 1 : -1;
          if (e[i] >= 0) own &= own - 1;
        }
        double xv[4][NX];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float* xr = xb[xbuf] + (e[i] >= 0 ? e[i] : e[0]) * D64 + dh * DP + lane;
#pragma unroll
          for (int u = 0; u < NX; ++u) xv[i][u] = (double)xr[64 * u];
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          if (e[i] < 0) break;
          const double r = (double)__int_as_float(__builtin_amdgcn_readlane(en.y, e[i]));
          accn[j] += r;
#pragma unroll
          for (int u = 0; u < NX; ++u) {
            accs[j][u] = fma(r, xv[i][u], accs[j][u]);
            accq[j][u] = fma(r, xv[i][u] * xv[i][u], accq[j][u]);
          }
        }
      }
    }
  };
  // at the end of batch t: the records of batch t+4 (loaded after the barrier
  // of batch t) go to the buffer of batch t-4, whose rows and records every
  // wave has finished with (the barrier of batch t); batch t+4's rows are
  // gathered after the barrier of batch t+1
  auto store_rec = [&](int t, const SPair& q) {
    if (q.pt >= 0) {
      rb[(t + 4) & 7][tid] = make_int2(q.c, __float_as_int(q.r));
      pb[(t + 4) & 7][tid] = q.pt;
    }
  };
  if (nbatch > 0) {
#pragma unroll
    for (int t = 0; t < 4; ++t)
      if (t < nbatch) load_rec(t);
    __syncthreads();
#pragma unroll
    for (int s = 0; s < kSparseDepth; ++s)
      if (s < nbatch) gather(s, g[s]);
  }
  // kSparseDepth batches per trip, so that the register sets g[s] are named
  // statically
  for (int t = 0; t < nbatch; t += kSparseDepth) {
#pragma unroll
    for (int s = 0; s < kSparseDepth; ++s) {
      const int u = t + s;
      if (u < nbatch) {
        const SPair q = consume(u, g[s]);
        if (u + kSparseDepth < nbatch) gather(u + kSparseDepth, g[s]);
        accumulate(u);
        store_rec(u, q);
      }
    }
  }
#pragma unroll
  for (int j = 0; j < CW; ++j) {
    double* out = part + ((size_t)blockIdx.x * C + sb + j) * STRIDE;
    if (lane == 0 && dh == 0) out[0] = accn[j];
#pragma unroll
    for (int u = 0; u < NX; ++u) {
      out[1 + dh * DP + lane + 64 * u] = accs[j][u];
      out[1 + D64 + dh * DP + lane + 64 * u] = accq[j][u];
    }
  }
}

// ---------------------------------------------------------------- Step 2: statistics, ill set
// Ill-conditioned components (few).  Grid of fixed size; each of the
// cdiv(n_ill, ICB) blocks of ICB = 4 CW such components gets grid/blocks point
// chunks.  Per PT-point iteration wave w forms r for components CW w ..
// CW w + CW - 1 of the block with the direct form (lane = point), then
// accumulates the statistics of those components in fp64 (lane = column).
__host__ __device__ constexpr int ill_pt(int D64) { return D64 <= 256 ? 64 : (D64 <= 512 ? 32 : 16); }
__host__ __device__ constexpr int ill_cw(int D64) { return D64 <= 256 ? 8 : (D64 <= 512 ? 4 : 2); }

__host__ __device__ inline int ill_chunks(int grid, int n_ikb, int64_t n, int pt) {
  int c = grid / (n_ikb > 0 ? n_ikb : 1);
  const int64_t cap = (n + pt - 1) / pt;
  if (c > cap) c = (int)cap;
  return c < 1 ? 1 : c;
}

template <int D64>
__global__ __launch_bounds__(256) void k_stats_ill(
    const float* __restrict__ x, int64_t n, int d, int vec4, const int* __restrict__ ill_idx,
    const float* __restrict__ dmu, const double* __restrict__ dh,
    const double* __restrict__ cdir, const int* __restrict__ counts,
    const double* __restrict__ logz2, const unsigned char* __restrict__ iflag,
    const unsigned char* __restrict__ lflag, const unsigned short* __restrict__ cslot,
    const int* __restrict__ small_pos, double* __restrict__ part) {
  constexpr int P = D64 + 4, NJ = D64 / 64, STRIDE = 1 + 2 * D64;
  constexpr int PT = ill_pt(D64), CW = ill_cw(D64), ICB = 4 * CW;
  constexpr int WIN = 16 * 256;                 // points scanned per queue window
  __shared__ __align__(16) float xs[PT * P];
  __shared__ float rs[ICB * PT];
  __shared__ double lzs[PT];
  __shared__ int lsx[PT][kT];                   // light: list index of each stored pair, or -1
  __shared__ unsigned qpt[WIN + PT];            // queued points (offsets from the chunk start)
  __shared__ int qsum[4];
  const int n_ill = counts[1];
  const int n_ikb = (n_ill + ICB - 1) / ICB;
  if (n_ikb == 0) return;
  const int nchk = ill_chunks(gridDim.x, n_ikb, n, PT);
  const int kb = blockIdx.x / nchk, chunk = blockIdx.x % nchk;
  if (kb >= n_ikb) return;
  const int64_t chunk_pts = (n + nchk - 1) / nchk;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int64_t p0 = (int64_t)chunk * chunk_pts;
  const int64_t p1 = p0 + chunk_pts < n ? p0 + chunk_pts : n;
  double S[CW][NJ], Q[CW][NJ], NK[CW];
#pragma unroll
  for (int c = 0; c < CW; ++c) {
    NK[c] = 0.0;
#pragma unroll
    for (int j = 0; j < NJ; ++j) S[c][j] = Q[c][j] = 0.0;
  }
  // Only the points whose flag says a routed component holds more than 2^-60
  // of them (every point when iflag is null) are taken: windows of WIN points
  // are scanned, flagged points queued in order, and tiles of PT queued points
  // gathered (the queue's rest moves to its front).  For the light components
  // (small_pos given: each well slot's index in their list, or -1) a point is
  // taken when the dense pass flagged it (lflag: a light component's dense
  // log-density there came within 2^-72 of log2 Z), and the point's stored
  // exact pairs are left out there: the exact-pair pass has summed them.  At
  // every other point each light component is either stored or has
  // r < 2^-64.
  int qn = 0;
  for (int64_t wb0 = p0; wb0 < p1; wb0 += WIN) {
    const int64_t we = wb0 + WIN < p1 ? wb0 + WIN : p1;
    {
      const int64_t a = wb0 + 16 * tid;
      unsigned sel = 0u;
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int64_t pt = a + e;
        bool take = pt < we;
        if (take && iflag != nullptr) take = iflag[pt] != 0;
        if (take && small_pos != nullptr) take = lflag[pt] != 0;
        if (take) sel |= 1u << e;
      }
      const int cnt = __popc(sel);
      int inc = cnt;
      for (int o = 1; o < 64; o <<= 1) {
        const int t2 = __shfl_up(inc, o);
        if (lane >= o) inc += t2;
      }
      if (lane == 63) qsum[wave] = inc;
      __syncthreads();
      int pos = qn + inc - cnt, all = 0;
#pragma unroll
      for (int w2 = 0; w2 < 4; ++w2) {
        if (w2 < wave) pos += qsum[w2];
        all += qsum[w2];
      }
      while (sel) {
        const int e = __ffs(sel) - 1;
        sel &= sel - 1;
        qpt[pos++] = (unsigned)(a + e - p0);
      }
      qn += all;
      __syncthreads();                          // queue complete, qsum free
    }
    const int nt = we >= p1 ? (qn + PT - 1) / PT : qn / PT;
  for (int ti = 0; ti < nt; ++ti) {
    __syncthreads();                            // the previous tile's reads are done
    {
      // gathered tile: queue entries PT ti .. PT ti + PT - 1 (rows past qn are zero)
      constexpr int Q4 = D64 / 4;
      for (int idx = tid; idx < PT * Q4; idx += 256) {
        const int r = idx / Q4, c = (idx % Q4) * 4;
        const int e = PT * ti + r;
        float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
        if (e < qn && c < d) {
          const float* xr = x + (p0 + qpt[e]) * d;
          if (vec4) {
            v = *reinterpret_cast<const float4*>(xr + c);
          } else {
            v.x = xr[c];
            v.y = c + 1 < d ? xr[c + 1] : 0.f;
            v.z = c + 2 < d ? xr[c + 2] : 0.f;
            v.w = c + 3 < d ? xr[c + 3] : 0.f;
          }
        }
        *reinterpret_cast<float4*>(xs + r * P + c) = v;
      }
      if (tid < PT) {
        const int e = PT * ti + tid;
        lzs[tid] = e < qn ? logz2[p0 + qpt[e]] : INFINITY;
        if (small_pos != nullptr) {
          int v4[kT] = {kNoSlot, kNoSlot, kNoSlot, kNoSlot};
          if (e < qn) {
            const ushort4 sl = *reinterpret_cast<const ushort4*>(cslot + (p0 + qpt[e]) * kT);
            v4[0] = sl.x; v4[1] = sl.y; v4[2] = sl.z; v4[3] = sl.w;
          }
#pragma unroll
          for (int j = 0; j < kT; ++j) lsx[tid][j] = v4[j] != kNoSlot ? small_pos[v4[j]] : -1;
        }
      }
    }
    __syncthreads();
    // nz[c]: the points of this tile with r > 0 for component c (wave-uniform)
    unsigned long long nz[CW];
#pragma unroll
    for (int c = 0; c < CW; ++c) {
      const int ki = kb * ICB + wave * CW + c;
      float r = 0.0f;
      bool stored = false;
      if (small_pos != nullptr && lane < PT) {
#pragma unroll
        for (int j = 0; j < kT; ++j) stored = stored || lsx[lane][j] == ki;
      }
      if (ki < n_ill && lane < PT && !stored) {
        const int comp = ill_idx[ki];
        const double c0 = cdir[comp];
        // r < 2^-150 is 0 in fp32: such pairs are not finished
        const double l = ill_logit_bounded<D64>(xs + lane * P, dmu + (size_t)comp * D64,
                                                dh + (size_t)comp * D64, c0,
                                                c0 - (lzs[lane] - 150.0));
        r = exp2_fast((float)(l - lzs[lane]));
      }
      if (lane < PT) rs[(wave * CW + c) * PT + lane] = r;
      nz[c] = __ballot(r > 0.0f);
    }
    __syncthreads();
    // pairs with r == 0 add exactly nothing and are skipped; per component the
    // points are still taken in increasing order
#pragma unroll
    for (int c = 0; c < CW; ++c) {
      unsigned long long msk = nz[c];
      while (msk) {
        const int p = __ffsll(msk) - 1;
        msk &= msk - 1;
        const double r = (double)rs[(wave * CW + c) * PT + p];
        NK[c] += r;
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
          const double xv = (double)xs[p * P + lane + 64 * j];
          const double rx = r * xv;
          S[c][j] += rx;
          Q[c][j] = fma(rx, xv, Q[c][j]);
        }
      }
    }
  }
    // the entries not taken move to the front of the queue
    const int used = PT * nt < qn ? PT * nt : qn;
    const int left = qn - used;
    __syncthreads();
    const unsigned keep = tid < left ? qpt[used + tid] : 0u;
    __syncthreads();
    if (tid < left) qpt[tid] = keep;
    qn = left;
  }
#pragma unroll
  for (int c = 0; c < CW; ++c) {
    double* base = part + ((size_t)blockIdx.x * ICB + wave * CW + c) * STRIDE;
    if (lane == 0) base[0] = NK[c];
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      base[1 + lane + 64 * j] = S[c][j];
      base[1 + D64 + lane + 64 * j] = Q[c][j];
    }
  }
}

// ---------------------------------------------------------------- assignment (Sec. 4.2, 4.3)
// Top-m multi-assignment at the given parameters, exact in the component order:
//   1. k_assign_theta: the screened log-densities of every point (the MFMA
//      pass of k_logz) give the T-th largest of its 128 lane-state maxima,
//      S_T (T = m + 2), and from it the thresholds below which no component
//      among the point's T largest can have its screened log-density.
//   2. k_assign_collect: a second screening pass keeps every component at or
//      above its threshold as a candidate (at most kACap per point) and sums
//      all others in a log-sum-exp; the candidates' log-densities are
//      recomputed in fp64 (direct form), ranked (ties to the lower index), and
//      normalised with log Z = log(sum over candidates of exp(exact) + the
//      screened sum of the others).  Rank 1 is always assigned, rank j > 1
//      only if its responsibility is > tau.
//   3. k_assign_fallback: points with more than kACap candidates are done
//      exactly over all components in fp64.
// Thresholds, fp32 screening (128 < D64 <= 256): S_T - 2 kScreenSlack for
// every component, kScreenSlack >= the screening error of the well-conditioned
// ones.  Split-bf16 screening (the other widths), from an error bound of each
// component: a screened log-density (log2 units) is the bias plus the products
// of [x | x^2] with [W | P]; three split products per fp32 product leave out at
// most 3 2^-16 of the product and the fp32 accumulation adds (3 D64 / 8 + 8)
// roundings of 2^-24 of the running sums, so its error is at most eps =
// split_eps(D64) (twice that) times the sum of the magnitudes of the bias and
// the products.  With |x mu| <= (x^2 +
// mu^2) / 2 and x^2 <= 2 (x - mu)^2 + 2 mu^2, that sum is at most
// 4 (cdir_k - l_k) + A_k, l_k the exact log-density, cdir_k its value at the
// mean and A_k = 5 (cdir_k - cwell_k) + |cwell_k|.  The arg-max components of
// the T largest lane states have exact log-densities of at least
// theta0 = S_T - max_i eps (4 (cdir_i - S_T) + A_i) / (1 - 4 eps), and so has
// the T-th largest component; a component j with l_j >= theta0 has a screened
// value >= theta0 - eps (4 (cdir_j - theta0) + A_j) = theta0 (1 + 4 eps) - b_j,
// b_j = eps (4 cdir_j + A_j), its candidate threshold.  Routed components,
// whose fp64 log-densities are rounded to fp32, take theta0 less that rounding.
constexpr int kACap = 32;
constexpr float kScreenSlack = 1.0f;
constexpr int kTMax = GMM_MAX_M + 2;
// eps of the split-bf16 screening error bound: twice the three left-out
// split terms (3 2^-16 of a product) plus the roundings of the accumulation
// chain (3 D64 / 8 MFMAs of up to five roundings each, and the bias and x^2
// in fp32), each 2^-24 of a running sum
__host__ __device__ constexpr float split_eps(int D64) {
  return 2.0f * (3.0f * 0x1p-16f + (3.0f * D64 / 8.0f + 8.0f) * 0x1p-24f);
}

// fp64 direct-form log-density (natural log) of component comp at point xr
// (fp32 row, LDS or global memory), from the caller's fp32 parameters and the
// fp64 constant cdir (log2 units).
__device__ __forceinline__ double ell64(const float* xr, const float* __restrict__ mu,
                                        const float* __restrict__ var, double cdir_k, int d) {
  double acc = 0.0;
  for (int j = 0; j < d; ++j) {
    const double t = (double)xr[j] - (double)mu[j];
    acc += t * t / (double)var[j];
  }
  return cdir_k * kLn2 - 0.5 * acc;
}

// Per well slot, the terms of its error bound: (cdir_j, A_j) in log2 units;
// (-inf, 0) for the padding slots.
__global__ __launch_bounds__(256) void k_assign_slots(const double* __restrict__ cwell,
                                                      const double* __restrict__ cdir,
                                                      const int* __restrict__ counts,
                                                      const int* __restrict__ well_idx, int kpad,
                                                      float2* __restrict__ ca) {
  const int slot = blockIdx.x * blockDim.x + threadIdx.x;
  if (slot >= kpad) return;
  float2 r = make_float2(-INFINITY, 0.0f);
  if (slot < counts[0]) {
    const int comp = well_idx[slot];
    const double c = cdir[comp], cw = cwell[comp];
    // rounded up to fp32: the bound only grows
    r = make_float2(__double2float_ru(c), __double2float_ru(5.0 * (c - cw) + fabs(cw)));
  }
  ca[slot] = r;
}

// Split X tile of the bf16 screening (the [x | x^2] layout of k_logz) from
// rows n0 .. n0 + 63; rows >= n and dimensions >= d are zero.  The whole
// chunks of every thread are loaded first (one memory round trip), the
// partial ones value by value.
template <int D64>
__device__ __forceinline__ void split_tile(const float* __restrict__ x, int64_t n, int d,
                                           int vec4, int64_t n0, bf16x8* xa) {
  constexpr int NC8 = D64 / 8, PTS = 64, NIT = (PTS * NC8 + 255) / 256;
  const int tid = threadIdx.x;
  float4 ld[NIT][2];
  bool whole[NIT];
#pragma unroll
  for (int it = 0; it < NIT; ++it) {
    const int t = tid + 256 * it, p = t / NC8, c = t % NC8;
    const int64_t row = n0 + p;
    whole[it] = vec4 && t < PTS * NC8 && row < n && 8 * c + 8 <= d;
    if (whole[it]) {
      ld[it][0] = *reinterpret_cast<const float4*>(x + row * d + 8 * c);
      ld[it][1] = *reinterpret_cast<const float4*>(x + row * d + 8 * c + 4);
    }
  }
#pragma unroll
  for (int it = 0; it < NIT; ++it) {
    const int t = tid + 256 * it, p = t / NC8, c = t % NC8;
    if (t >= PTS * NC8) continue;
    const int64_t row = n0 + p;
    float v[8];
    if (whole[it]) {
      v[0] = ld[it][0].x; v[1] = ld[it][0].y; v[2] = ld[it][0].z; v[3] = ld[it][0].w;
      v[4] = ld[it][1].x; v[5] = ld[it][1].y; v[6] = ld[it][1].z; v[7] = ld[it][1].w;
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int j = 8 * c + e;
        v[e] = (row < n && j < d) ? x[row * d + j] : 0.0f;
      }
    }
    split_store<D64, false>(xa, p, c, v);
  }
}

// Screening pass shared by the two assignment kernels: wave w takes the well
// blocks w, w + 4, ...; epi(v, l0, l1, slot, b) receives the log-densities of
// lane element v of the two point tiles for component slot `slot`, and b =
// pre(slot), which is called one block ahead (its loads then have a block's
// MFMA work to arrive).
template <int D64, class Pre, class Epi>
__device__ __forceinline__ void assign_screen(const float* xs, const bf16x8* xa,
                                              const float4* __restrict__ wp,
                                              const bf16x8* __restrict__ wpb,
                                              const float* __restrict__ cw, int n_wkb,
                                              Pre&& pre, Epi&& epi) {
  constexpr int NT = logz_tiles(D64);
  constexpr bool SPL = screen_b16(D64);
  constexpr int NSTEP = screen_steps<D64, false>(), RPV = 4 * NSTEP + 1;
  constexpr size_t BS = (size_t)(D64 / 4) * 64, BS16 = (size_t)NSTEP * 64 * 2;
  const int tid = threadIdx.x, wave = tid >> 6, col = tid & 31;
  const int nb = n_wkb > wave ? (n_wkb - wave + 3) / 4 : 0;
  if (nb == 0) return;
  if constexpr (screen_x16(D64)) {
    // GB blocks at a time from the fp32 tile, as in k_logz: blocks wave + 4 i,
    // i = GB g + j; a group's missing blocks repeat its last one and are not
    // taken in
    constexpr int GB = 4;
    const int ng = (nb + GB - 1) / GB;
    int kbc[GB], kbp[GB];
    float cbc[GB], bc[GB], bp[GB];
    f16v na[GB], nc[GB];
    int nvp = 0;
    auto epi16 = [&](int j, int v, float l) { epi(v, l, l, kbp[j] * kBK + col, bp[j]); };
    for (int g = 0; g <= ng; ++g) {
      if (g < ng) {
#pragma unroll
        for (int j = 0; j < GB; ++j) {
          const int i = GB * g + j < nb ? GB * g + j : nb - 1;
          kbc[j] = wave + 4 * i;
          cbc[j] = cw[kbc[j] * kBK + col];
          bc[j] = pre(kbc[j] * kBK + col);
        }
        if (g == 0)
          logz_group16<D64, GB, true, false, false>(xs, wpb, kbc, cbc, na, nc, 0, epi16);
        else
          logz_group16<D64, GB, true, true, false>(xs, wpb, kbc, cbc, na, nc, nvp, epi16);
      } else if (ng > 0) {
        logz_group16<D64, GB, false, true, false>(xs, wpb, kbc, cbc, na, nc, nvp, epi16);
      }
#pragma unroll
      for (int j = 0; j < GB; ++j) {
        nc[j] = na[j];
        kbp[j] = kbc[j];
        bp[j] = bc[j];
      }
      nvp = nb - GB * g < GB ? nb - GB * g : GB;
    }
    return;
  }
  f16v c0, c1, x0, x1;
  int slot = 0;
  float bv = 0.0f, bn = pre(wave * kBK + col);
  auto e2 = [&](int v, float l0, float l1) { epi(v, l0, l1, slot, bv); };
  if constexpr (SPL)
    logz_step16<NSTEP, RPV, true, false, NT>(xa, wpb + (size_t)wave * BS16,
                                             cw[wave * kBK + col], c0, c1, x0, x1, e2);
  else
    logz_step<D64, true, false, NT>(xs, wp + (size_t)wave * BS, cw[wave * kBK + col], c0, c1,
                                    x0, x1, e2);
  for (int i = 0; i + 1 < nb; ++i) {
    const int kb = wave + 4 * i;
    slot = kb * kBK + col;
    bv = bn;
    bn = pre((kb + 4) * kBK + col);
    if constexpr (SPL)
      logz_step16<NSTEP, RPV, true, true, NT>(xa, wpb + (size_t)(kb + 4) * BS16,
                                              cw[(kb + 4) * kBK + col], x0, x1, c0, c1, e2);
    else
      logz_step<D64, true, true, NT>(xs, wp + (size_t)(kb + 4) * BS, cw[(kb + 4) * kBK + col],
                                     x0, x1, c0, c1, e2);
    c0 = x0;
    c1 = x1;
  }
  slot = (wave + 4 * (nb - 1)) * kBK + col;
  bv = bn;
  if constexpr (SPL)
    logz_step16<NSTEP, RPV, false, true, NT>(xa, wpb, 0.0f, x0, x1, c0, c1, e2);
  else
    logz_step<D64, false, true, NT>(xs, wp, 0.0f, x0, x1, c0, c1, e2);
}

// Thresholds of each point: theta[p] = (well-component base, routed-component
// threshold); a well slot j is a candidate when its screened log-density is
// >= theta[p].x - b_j (b_j = 0 for the fp32 screening).
// TL: length of the per-point list of the largest lane states (>= tsel):
// 4 for m <= 2, kTMax otherwise.
template <int D64, int TL>
__global__ __launch_bounds__(256, screen_b16(D64) ? 2 : 1) void k_assign_theta(
    const float* __restrict__ x, int64_t n, int d, int vec4, const float4* __restrict__ wp,
    const bf16x8* __restrict__ wpb, const float* __restrict__ cw,
    const float2* __restrict__ ca, const int* __restrict__ counts, int tsel,
    float2* __restrict__ theta) {
  constexpr int P = D64 + 4, NT = logz_tiles(D64), PTS = 32 * NT;
  // SPL: split tile in LDS; SPB: split-bf16 screening (from the split tile or,
  // D64 > 256, from the fp32 tile), whose thresholds need the arg-max slots
  constexpr bool SPL = screen_b16(D64), SPB = screen_split(D64);
  constexpr int RPV = 4 * screen_steps<D64, false>() + 1;
  constexpr float kEps = split_eps(D64);
  // SPB: the X tile (split or fp32), whose space the lane-state maxima and their
  // arg-max slots take over after the screening; else the fp32 tile and the
  // maxima
  constexpr size_t XB = SPL ? (size_t)PTS * RPV * sizeof(bf16x8) : (size_t)PTS * P * sizeof(float);
  constexpr size_t LB = (size_t)PTS * 129 * (SPB ? sizeof(float2) : sizeof(float));
  constexpr size_t SB = SPB ? (XB > LB ? XB : LB) : XB + LB;
  __shared__ __align__(16) unsigned char smem[SB];
  float* const xs = reinterpret_cast<float*>(smem);
  bf16x8* const xa = reinterpret_cast<bf16x8*>(smem);
  float* const lmx = reinterpret_cast<float*>(smem + XB);                  // [PTS][129]
  float2* const lma = reinterpret_cast<float2*>(smem);                     // [PTS][129]
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, h = lane >> 5, col = lane & 31;
  const int64_t n0 = (int64_t)blockIdx.x * PTS;
  if constexpr (SPL) split_tile<D64>(x, n, d, vec4, n0, xa);
  else load_tile<D64>(x, n, d, n0, PTS, xs, vec4 != 0);
  __syncthreads();
  float m0[16], m1[16];
  int a0[16], a1[16];
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    m0[v] = m1[v] = kEmpty;
    a0[v] = a1[v] = -1;
  }
  assign_screen<D64>(xs, xa, wp, wpb, cw, counts[2], [](int) { return 0.0f; },
                     [&](int v, float l0, float l1, int slot, float) {
    if constexpr (SPB) {
      a0[v] = l0 > m0[v] ? slot : a0[v];
      if constexpr (NT == 2) a1[v] = l1 > m1[v] ? slot : a1[v];
    }
    m0[v] = fmaxf(m0[v], l0);
    if constexpr (NT == 2) m1[v] = fmaxf(m1[v], l1);
  });
  if constexpr (SPB) __syncthreads();        // the maxima take over the tile
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const int p = 8 * (v >> 2) + 4 * h + (v & 3);
    if constexpr (SPB) {
      lma[p * 129 + wave * 32 + col] = make_float2(m0[v], __int_as_float(a0[v]));
      if constexpr (NT == 2) lma[(32 + p) * 129 + wave * 32 + col] = make_float2(m1[v], __int_as_float(a1[v]));
    } else {
      lmx[p * 129 + wave * 32 + col] = m0[v];
      if constexpr (NT == 2) lmx[(32 + p) * 129 + wave * 32 + col] = m1[v];
    }
  }
  __syncthreads();
  {
    // G threads per point, each over 128 / G lane states, then their lists
    // merged across the group (disjoint lane states: no entry twice)
    constexpr int G = 256 / PTS, LPT = 128 / G;
    const int p = tid / G, r = tid % G;
    float tl[TL];
    int ta[TL];
#pragma unroll
    for (int j = 0; j < TL; ++j) {
      tl[j] = -INFINITY;
      ta[j] = -1;
    }
    auto insert = [&](float v, int a) {
#pragma unroll
      for (int j = TL - 1; j > 0; --j) {
        if (v > tl[j - 1]) { tl[j] = tl[j - 1]; ta[j] = ta[j - 1]; }
        else if (v > tl[j]) { tl[j] = v; ta[j] = a; }
      }
      if (v > tl[0]) { tl[0] = v; ta[0] = a; }
    };
    for (int c = LPT * r; c < LPT * r + LPT; ++c) {
      float v;
      int a = -1;
      if constexpr (SPB) {
        const float2 e = lma[p * 129 + c];
        v = e.x;
        a = __float_as_int(e.y);
      } else {
        v = lmx[p * 129 + c];
      }
      // empty lane states (kEmpty) and those below the list are skipped
      if (v > 0.5f * kEmpty && v > tl[TL - 1]) insert(v, a);
    }
#pragma unroll
    for (int off = 1; off < G; off <<= 1) {
      float ol[TL];
      int oa[TL];
#pragma unroll
      for (int j = 0; j < TL; ++j) {
        ol[j] = __shfl_xor(tl[j], off);
        oa[j] = __shfl_xor(ta[j], off);
      }
#pragma unroll
      for (int j = 0; j < TL; ++j)
        if (ol[j] > tl[TL - 1]) insert(ol[j], oa[j]);
    }
    if (r != 0 || n0 + p >= n) return;
    float st = -INFINITY;
#pragma unroll
    for (int j = 0; j < TL; ++j)
      if (j == tsel - 1) st = tl[j];
    float2 out;
    if constexpr (SPB) {
      float dm = 0.0f;
#pragma unroll
      for (int j = 0; j < TL; ++j) {
        if (j < tsel && ta[j] >= 0) {
          const float2 e = ca[ta[j]];
          dm = fmaxf(dm, kEps * (4.0f * fmaxf(e.x - st, 0.0f) + e.y));
        }
      }
      const float th0 = st - dm / (1.0f - 4.0f * kEps);
      // fp32 rounding of these few operations: 2^-20 of the magnitude
      const float mg = 0x1p-20f * (fabsf(th0) + 1.0f);
      out = make_float2(th0 * (1.0f + 4.0f * kEps) - mg, th0 - 0x1p-22f * (fabsf(th0) + 1.0f) - mg);
    } else {
      out = make_float2(st - 2.0f * kScreenSlack, st - 2.0f * kScreenSlack);
    }
    theta[n0 + p] = out;
  }
}

template <int D64>
__global__ __launch_bounds__(256, screen_b16(D64) ? 2 : 1) void k_assign_collect(
    const float* __restrict__ x, int64_t n, int d, int vec4, const float4* __restrict__ wp,
    const bf16x8* __restrict__ wpb, const float* __restrict__ cw,
    const float2* __restrict__ ca, const int* __restrict__ well_idx,
    const int* __restrict__ ill_idx, const float* __restrict__ dmu,
    const double* __restrict__ dh, const int* __restrict__ counts,
    const float2* __restrict__ theta, const float* __restrict__ mu,
    const float* __restrict__ var, const double* __restrict__ cdir, int m, float tau,
    int* __restrict__ idx, float* __restrict__ resp, int* __restrict__ ovf) {
  constexpr int P = D64 + 4, NT = logz_tiles(D64), PTS = 32 * NT;
  constexpr bool SPL = screen_b16(D64);
  constexpr int RPV = 4 * screen_steps<D64, false>() + 1;
  // the X tile (SPL: split, its space then taken over by the exact log-densities)
  constexpr size_t XB = SPL ? (size_t)PTS * RPV * sizeof(bf16x8) : (size_t)PTS * P * sizeof(float);
  constexpr size_t CB = (size_t)PTS * kACap * sizeof(double);
  static_assert(!SPL || CB <= XB, "the exact log-densities fit the split tile's space");
  constexpr size_t SB = SPL ? XB : XB + CB;
  __shared__ __align__(16) unsigned char smem[SB];
  __shared__ int ccnt[PTS];
  __shared__ int eoff[PTS + 1];            // first entry of each point's candidates
  __shared__ int cand[PTS][kACap];         // well slot s >= 0, or -(ill component + 1)
  __shared__ float2 stw[4][PTS];
  __shared__ float2 sti[4][PTS];
  float* const xs = reinterpret_cast<float*>(smem);
  bf16x8* const xa = reinterpret_cast<bf16x8*>(smem);
  double* const cl = reinterpret_cast<double*>(smem + (SPL ? 0 : XB));    // [PTS][kACap]
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, h = lane >> 5, col = lane & 31;
  const int64_t n0 = (int64_t)blockIdx.x * PTS;
  if constexpr (SPL) split_tile<D64>(x, n, d, vec4, n0, xa);
  else load_tile<D64>(x, n, d, n0, PTS, xs, vec4 != 0);
  if (tid < PTS) ccnt[tid] = 0;
  __syncthreads();
  const int n_wkb = counts[2], n_ill = counts[1];
  float th0[16], th1[16], m0[16], s0[16], m1[16], s1[16];
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const int p = 8 * (v >> 2) + 4 * h + (v & 3);
    th0[v] = n0 + p < n ? theta[n0 + p].x : INFINITY;
    th1[v] = (NT == 2 && n0 + 32 + p < n) ? theta[n0 + 32 + p].x : INFINITY;
    m0[v] = m1[v] = kEmpty;
    s0[v] = s1[v] = 0.0f;
  }
  {
    // the slot's share b_j of its candidate threshold (0 for the fp32 screening)
    auto pre = [&](int slot) {
      if constexpr (screen_split(D64)) {
        const float2 e = ca[slot];
        return split_eps(D64) * (4.0f * e.x + e.y);
      } else {
        return 0.0f;
      }
    };
    // the sums take every value, a candidate's as -inf (which adds nothing);
    // the rare candidates are pushed under a wave-uniform test, so that the
    // common path has no branch between the MFMAs
    assign_screen<D64>(xs, xa, wp, wpb, cw, n_wkb, pre,
                       [&](int v, float l0, float l1, int slot, float bj) {
      const int p = 8 * (v >> 2) + 4 * h + (v & 3);
      const bool c0 = (l0 >= th0[v] - bj) & (l0 > -INFINITY);
      lse_add_e(m0[v], s0[v], c0 ? -INFINITY : l0);
      bool c1 = false;
      if constexpr (NT == 2) {
        c1 = (l1 >= th1[v] - bj) & (l1 > -INFINITY);
        lse_add_e(m1[v], s1[v], c1 ? -INFINITY : l1);
      }
      if (__ballot(c0 | c1) != 0ull) {
        if (c0) {
          const int pos = atomicAdd(&ccnt[p], 1);
          if (pos < kACap) cand[p][pos] = slot;
        }
        if (c1) {
          const int pos = atomicAdd(&ccnt[32 + p], 1);
          if (pos < kACap) cand[32 + p][pos] = slot;
        }
      }
    });
  }
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const int p = 8 * (v >> 2) + 4 * h + (v & 3);
    float M0 = m0[v], S0 = s0[v], M1 = m1[v], S1 = s1[v];
    auto merge = [&](auto oc) {
      constexpr int off = decltype(oc)::value;
      lse_merge(M0, S0, xshfl<off>(M0), xshfl<off>(S0));
      if constexpr (NT == 2) lse_merge(M1, S1, xshfl<off>(M1), xshfl<off>(S1));
    };
    merge(std::integral_constant<int, 16>{});
    merge(std::integral_constant<int, 8>{});
    merge(std::integral_constant<int, 4>{});
    merge(std::integral_constant<int, 2>{});
    merge(std::integral_constant<int, 1>{});
    if (col == 0) {
      stw[wave][p] = make_float2(M0, S0);
      if constexpr (NT == 2) stw[wave][32 + p] = make_float2(M1, S1);
    }
  }
  if (lane < PTS) {
    // ill-conditioned components, direct form, lane = point.  A component more
    // than 64 log2 units below the point's threshold (so below 2^-62 of its
    // mass) is left out of the normaliser: its sum stops early (most of them
    // after 16 dimensions), as in k_logz.
    const int64_t row = n0 + lane;
    const float thl = row < n ? theta[row].y : INFINITY;
    const float* xr = SPL ? x + (row < n ? row : 0) * d : xs + lane * P;
    float mi = kEmpty, si = 0.0f;
    for (int ki = wave; ki < n_ill; ki += 4) {
      const int comp = ill_idx[ki];
      const double c = cdir[comp];
      const double bnd = c - ((double)thl - 64.0);
      float l;
      if constexpr (SPL)
        l = (float)ill_logit_bounded_gr(xr, d, vec4, dmu + (size_t)comp * D64,
                                        dh + (size_t)comp * D64, c, bnd);
      else
        l = (float)ill_logit_bounded<D64>(xr, dmu + (size_t)comp * D64,
                                          dh + (size_t)comp * D64, c, bnd);
      if (l >= thl && l > -INFINITY) {
        const int pos = atomicAdd(&ccnt[lane], 1);
        if (pos < kACap) cand[lane][pos] = -(comp + 1);
      } else {
        lse_add_e(mi, si, l);
      }
    }
    sti[wave][lane] = make_float2(mi, si);
  }
  __syncthreads();
  // The waves appended the candidates in the order they found them; each
  // point's list is put in ascending code order, so that the fp64 normaliser
  // below adds the same terms in the same order on every run.
  if (tid < PTS) {
    const int cnt = ccnt[tid];
    if (cnt <= kACap) {
      for (int i = 1; i < cnt; ++i) {
        const int v = cand[tid][i];
        int j = i - 1;
        while (j >= 0 && cand[tid][j] > v) {
          cand[tid][j + 1] = cand[tid][j];
          --j;
        }
        cand[tid][j + 1] = v;
      }
    }
  }
  if (tid == 0) {
    // the (point, candidate) entries in point order: each point's first entry
    // (points past n and overflowing lists have none)
    int acc = 0;
    for (int p = 0; p < PTS; ++p) {
      eoff[p] = acc;
      const int c = ccnt[p];
      acc += (c <= kACap && n0 + p < n) ? c : 0;
    }
    eoff[PTS] = acc;
  }
  __syncthreads();
  {
    // exact fp64 log-densities of the candidates: kRefLanes lanes per entry,
    // lane g summing the direct form over the float4 chunks g, g + kRefLanes,
    // ... of the row (coalesced over the group; global rows when SPL), the
    // group's partial sums added in a fixed butterfly order; log2 units, then
    // natural log
    constexpr int G = kRefLanes;
    const int g = tid & (G - 1);
    const int total = eoff[PTS];
    for (int e = tid / G; e < total; e += 256 / G) {
      // the entry's point: the last one whose first entry is <= e
      int p = 0;
      for (int s = PTS / 2; s > 0; s >>= 1)
        if (p + s < PTS && eoff[p + s] <= e) p += s;
      const int j = e - eoff[p];
      const int code = cand[p][j];
      const int comp = code >= 0 ? well_idx[code] : -code - 1;
      const float* xr = SPL ? x + (n0 + p) * d : xs + p * P;
      const float* mu = dmu + (size_t)comp * D64;
      const double* hh = dh + (size_t)comp * D64;
      const bool v4 = !SPL || vec4;
      double acc = 0.0;
      for (int c4 = 4 * g; c4 < d; c4 += 4 * G) {
        float xv[4];
        if (v4 && c4 + 4 <= d) {
          const float4 t4 = *reinterpret_cast<const float4*>(xr + c4);
          xv[0] = t4.x; xv[1] = t4.y; xv[2] = t4.z; xv[3] = t4.w;
        } else {
#pragma unroll
          for (int u = 0; u < 4; ++u) xv[u] = c4 + u < d ? xr[c4 + u] : 0.0f;
        }
        const float4 m4 = *reinterpret_cast<const float4*>(mu + c4);
        const double2 h0 = *reinterpret_cast<const double2*>(hh + c4);
        const double2 h1 = *reinterpret_cast<const double2*>(hh + c4 + 2);
        double t;
        t = (double)xv[0] - (double)m4.x; acc = fma(t * t, h0.x, acc);
        t = (double)xv[1] - (double)m4.y; acc = fma(t * t, h0.y, acc);
        t = (double)xv[2] - (double)m4.z; acc = fma(t * t, h1.x, acc);
        t = (double)xv[3] - (double)m4.w; acc = fma(t * t, h1.y, acc);
      }
#pragma unroll
      for (int o = 1; o < G; o <<= 1) acc += __shfl_xor(acc, o);
      if (g == 0) cl[p * kACap + j] = kLn2 * (cdir[comp] - acc);
    }
  }
  __syncthreads();
  if (tid < PTS && n0 + tid < n) {
    const int p = tid;
    const int64_t nn = n0 + p;
    const int cnt = ccnt[p];
    if (cnt > kACap) {
      ovf[nn] = 1;
      return;
    }
    ovf[nn] = 0;
    // screened sum of the non-candidates (log2 units) -> natural log, fp64
    float mm = kEmpty;
    for (int w2 = 0; w2 < 4; ++w2) mm = fmaxf(mm, fmaxf(stw[w2][p].x, sti[w2][p].x));
    double snc = 0.0;
    for (int w2 = 0; w2 < 4; ++w2) {
      snc += (double)stw[w2][p].y * exp2((double)stw[w2][p].x - (double)mm);
      snc += (double)sti[w2][p].y * exp2((double)sti[w2][p].x - (double)mm);
    }
    const double lnc = snc > 0.0 ? (double)mm * kLn2 + log(snc) : -INFINITY;
    // rank the candidates: exact log-density descending, ties to the lower index
    double tl[GMM_MAX_M];
    int ti[GMM_MAX_M];
#pragma unroll
    for (int j = 0; j < GMM_MAX_M; ++j) { tl[j] = -INFINITY; ti[j] = -1; }
    double lmx = lnc;
    for (int j = 0; j < cnt; ++j) {
      const int code = cand[p][j];
      const int comp = code >= 0 ? well_idx[code] : -code - 1;
      const double l = cl[p * kACap + j];
      lmx = fmax(lmx, l);
#pragma unroll
      for (int q = GMM_MAX_M - 1; q >= 0; --q) {
        const bool above = l > tl[q] || (l == tl[q] && ti[q] >= 0 && comp < ti[q]) || ti[q] < 0;
        const bool above_prev =
            q > 0 && (l > tl[q - 1] || (l == tl[q - 1] && ti[q - 1] >= 0 && comp < ti[q - 1]) ||
                      ti[q - 1] < 0);
        if (above_prev) { tl[q] = tl[q - 1]; ti[q] = ti[q - 1]; }
        else if (above) { tl[q] = l; ti[q] = comp; }
      }
    }
    double z = lnc > -INFINITY ? exp(lnc - lmx) : 0.0;
    for (int j = 0; j < cnt; ++j) z += exp(cl[p * kACap + j] - lmx);
    const double lz = lmx + log(z);
#pragma unroll
    for (int j = 0; j < GMM_MAX_M; ++j) {
      if (j >= m) break;
      int oi = -1;
      float orr = 0.0f;
      if (ti[j] >= 0) {
        const double r = exp(tl[j] - lz);
        if (j == 0 || r > (double)tau) { oi = ti[j]; orr = (float)r; }
      }
      idx[nn * m + j] = oi;
      resp[nn * m + j] = orr;
    }
  }
}

// Points whose candidate list overflowed: every component's log-density in
// fp64, thread t taking components t, t + 256, ...; per-thread top-m lists and
// log-sum-exp states merged by one thread in thread order.
__global__ __launch_bounds__(256) void k_assign_fallback(
    const float* __restrict__ x, int64_t n, int d, int k, const float* __restrict__ mu,
    const float* __restrict__ var, const double* __restrict__ cdir, int m, float tau,
    const int* __restrict__ ovf, int* __restrict__ idx, float* __restrict__ resp) {
  __shared__ float xr[GMM_MAX_D];
  __shared__ int plist[1024];
  __shared__ int pcnt;
  __shared__ double lm[256], ls[256];
  __shared__ double ltl[256][GMM_MAX_M];
  __shared__ int lti[256][GMM_MAX_M];
  const int tid = threadIdx.x;
  const int64_t b0 = (int64_t)blockIdx.x * 1024;
  if (tid == 0) pcnt = 0;
  __syncthreads();
  // the order of the list does not matter: every point's result is its own
  for (int i = tid; i < 1024; i += 256)
    if (b0 + i < n && ovf[b0 + i]) plist[atomicAdd(&pcnt, 1)] = i;
  __syncthreads();
  const int np = pcnt;
  for (int ip = 0; ip < np; ++ip) {
    const int64_t nn = b0 + plist[ip];
    for (int j = tid; j < d; j += 256) xr[j] = x[nn * d + j];
    __syncthreads();
    double tl[GMM_MAX_M];
    int ti[GMM_MAX_M];
#pragma unroll
    for (int j = 0; j < GMM_MAX_M; ++j) { tl[j] = -INFINITY; ti[j] = -1; }
    double mx = -INFINITY, sm = 0.0;
    for (int comp = tid; comp < k; comp += 256) {
      const double l = ell64(xr, mu + (size_t)comp * d, var + (size_t)comp * d, cdir[comp], d);
      if (!(l > -INFINITY)) continue;
      if (l > mx) { sm = sm * exp(mx - l) + 1.0; mx = l; }
      else sm += exp(l - mx);
#pragma unroll
      for (int q = GMM_MAX_M - 1; q >= 0; --q) {
        // components arrive in increasing index order: ties keep the earlier
        const bool above = ti[q] < 0 || l > tl[q];
        const bool above_prev = q > 0 && (ti[q - 1] < 0 || l > tl[q - 1]);
        if (above_prev) { tl[q] = tl[q - 1]; ti[q] = ti[q - 1]; }
        else if (above) { tl[q] = l; ti[q] = comp; }
      }
    }
    lm[tid] = mx;
    ls[tid] = sm;
#pragma unroll
    for (int j = 0; j < GMM_MAX_M; ++j) { ltl[tid][j] = tl[j]; lti[tid][j] = ti[j]; }
    __syncthreads();
    if (tid == 0) {
      double M = -INFINITY;
      for (int t = 0; t < 256; ++t) M = fmax(M, lm[t]);
      double z = 0.0;
      for (int t = 0; t < 256; ++t)
        if (lm[t] > -INFINITY) z += ls[t] * exp(lm[t] - M);
      const double lz = M + log(z);
      double bl[GMM_MAX_M];
      int bi[GMM_MAX_M];
      for (int j = 0; j < GMM_MAX_M; ++j) { bl[j] = -INFINITY; bi[j] = -1; }
      for (int t = 0; t < 256; ++t)
        for (int j2 = 0; j2 < GMM_MAX_M; ++j2) {
          const int c = lti[t][j2];
          if (c < 0) break;
          const double l = ltl[t][j2];
          for (int q = GMM_MAX_M - 1; q >= 0; --q) {
            const bool above = bi[q] < 0 || l > bl[q] || (l == bl[q] && c < bi[q]);
            const bool above_prev =
                q > 0 && (bi[q - 1] < 0 || l > bl[q - 1] || (l == bl[q - 1] && c < bi[q - 1]));
            if (above_prev) { bl[q] = bl[q - 1]; bi[q] = bi[q - 1]; }
            else if (above) { bl[q] = l; bi[q] = c; }
          }
        }
      for (int j = 0; j < m; ++j) {
        int oi = -1;
        float orr = 0.0f;
        if (bi[j] >= 0) {
          const double r = exp(bl[j] - lz);
          if (j == 0 || r > (double)tau) { oi = bi[j]; orr = (float)r; }
        }
        idx[nn * m + j] = oi;
        resp[nn * m + j] = orr;
      }
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------- fixed-order reductions
// Partial layouts (rows of 1 + 2 D64 fp64: N, then S over D64, then Q):
//   well    ((slot / wbk) * nch + chunk) * wbk + slot % wbk
//   sparse  ((slot / sbk) * nparts + part) * sbk + slot % sbk
//   ill     ((islot / ibk) * nchk + chunk) * ibk + islot % ibk
// summed here in chunk (part) order.
// acc + p[0] + p[step] + ... + p[(cnt - 1) step], added in that order, with
// 8 loads in flight at a time.
__device__ __forceinline__ double sum_strided(const double* __restrict__ p, int cnt, size_t step,
                                              double acc) {
  int ch = 0;
  for (; ch + 8 <= cnt; ch += 8) {
    double v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = p[(size_t)(ch + j) * step];
#pragma unroll
    for (int j = 0; j < 8; ++j) acc += v[j];
  }
  for (; ch < cnt; ++ch) acc += p[(size_t)ch * step];
  return acc;
}

// ---------------------------------------------------------------- light components
// A component that holds little mass in a call can have its variance carried
// by a few pairs outside the point's stored exact ones: a component sitting on
// one point gets its variance from the tails of other points' responsibilities.
// The dense pass forms those pairs' log-densities in fp32 with an error of up
// to about 2^-16 (S + d) log2 units (the expanded form's terms cancel), far
// too coarse when one pair makes the whole variance (or the whole of a small
// N_k).  Every well-conditioned component whose stored exact pairs hold less
// than kSmallMass is therefore light: the dense pass leaves it out and flags
// the points where its fp32 log-density comes within 2^-72 of log2 Z (eight
// log2 units of slack over the 2^-64 cut for the dense pass's error); its
// pairs at those points, except the stored ones, are computed in the direct
// form with fp64 sums (k_stats_ill), and its stored pairs come from the
// exact-pair pass as for every component.  A component with more
// mass spreads its variance over enough pairs that their independent
// rounding errors stay well inside the variance tolerance.
constexpr double kSmallMass = 64.0;

// flag[slot] = 1 for the live well slots whose stored exact pairs hold less
// than kSmallMass (every component with N_k < kSmallMass is among them, since
// the stored pairs are part of its mass; a dead one has log pi = -inf).
__global__ __launch_bounds__(256) void k_small_mass(
    const double* __restrict__ part_s, const int* __restrict__ counts,
    const int* __restrict__ well_idx, const double* __restrict__ cdir, int nparts, int sbk,
    int D64, unsigned char* __restrict__ flag) {
  const int slot = blockIdx.x * blockDim.x + threadIdx.x;
  if (slot >= counts[0]) return;
  const size_t stride = 1 + 2 * (size_t)D64;
  const double* ps = part_s + ((size_t)(slot / sbk) * nparts * sbk + (slot % sbk)) * stride;
  const double m = sum_strided(ps, nparts, (size_t)sbk * stride, 0.0);
  const bool live = cdir[well_idx[slot]] > -INFINITY;
  flag[slot] = (live && m < kSmallMass) ? 1 : 0;
}

// The flagged slots in slot order: pos[slot] = index in the list or -1,
// idx[i] = the component, cnt[1] = the list's length (cnt[0] = 0), so that
// (idx, cnt) take the place of (ill_idx, counts) for k_stats_ill.
__global__ __launch_bounds__(1024) void k_small_list(const unsigned char* __restrict__ flag,
                                                     const int* __restrict__ counts,
                                                     const int* __restrict__ well_idx,
                                                     int* __restrict__ pos, int* __restrict__ idx,
                                                     int* __restrict__ cnt) {
  __shared__ int wsum[16];
  const int nw = counts[0];
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int per = (nw + 1023) / 1024;
  const int a = t * per < nw ? t * per : nw;
  const int b = a + per < nw ? a + per : nw;
  int c = 0;
  for (int sl = a; sl < b; ++sl) c += flag[sl];
  int inc = c;
  for (int o = 1; o < 64; o <<= 1) {
    const int v = __shfl_up(inc, o);
    if (lane >= o) inc += v;
  }
  if (lane == 63) wsum[wave] = inc;
  __syncthreads();
  int before = 0, total = 0;
  for (int w = 0; w < 16; ++w) {
    if (w < wave) before += wsum[w];
    total += wsum[w];
  }
  int p = before + inc - c;
  for (int sl = a; sl < b; ++sl) {
    if (flag[sl]) {
      pos[sl] = p;
      idx[p] = well_idx[sl];
      ++p;
    } else {
      pos[sl] = -1;
    }
  }
  if (t == 0) {
    cnt[0] = 0;
    cnt[1] = total;
  }
}

__global__ __launch_bounds__(256) void k_reduce_stats(
    const double* __restrict__ part_w, const double* __restrict__ part_s,
    const double* __restrict__ part_i,
    const int* __restrict__ counts, const int* __restrict__ well_idx,
    const int* __restrict__ ill_idx, int nch, int wbk, int nparts, int sbk, int grid_i, int ibk,
    int ipt, int64_t n, int k, int d, int D64, const int* __restrict__ small_pos,
    const double* __restrict__ part_x, const int* __restrict__ small_cnt,
    double* __restrict__ nk, double* __restrict__ s, double* __restrict__ q) {
  const int64_t width = 1 + 2 * (int64_t)d;
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= 2 * (int64_t)k * width) return;
  const int which = (int)(t / ((int64_t)k * width));
  const int64_t rem = t % ((int64_t)k * width);
  const int slot = (int)(rem / width), c = (int)(rem % width);
  const int64_t stride = 1 + 2 * (int64_t)D64;
  const int64_t off = c == 0 ? 0 : (c <= d ? 1 + (c - 1) : 1 + D64 + (c - 1 - d));
  double acc = 0.0;
  int comp;
  if (which == 0) {
    if (slot >= counts[0]) return;
    comp = well_idx[slot];
    const int xp = small_pos != nullptr ? small_pos[slot] : -1;
    if (xp >= 0) {
      // a light component: its exact recomputation at the flagged points
      // replaces the dense pass; its stored pairs come from the exact-pair pass
      const int n_xkb = (small_cnt[1] + ibk - 1) / ibk;
      const int nchk = ill_chunks(grid_i, n_xkb, n, ipt);
      const double* p = part_x + ((size_t)(xp / ibk) * nchk * ibk + (xp % ibk)) * stride + off;
      acc = sum_strided(p, nchk, (size_t)ibk * stride, acc);
      const double* ps =
          part_s + ((size_t)(slot / sbk) * nparts * sbk + (slot % sbk)) * stride + off;
      acc = sum_strided(ps, nparts, (size_t)sbk * stride, acc);
    } else {
      const double* p = part_w + ((size_t)(slot / wbk) * nch * wbk + (slot % wbk)) * stride + off;
      acc = sum_strided(p, nch, (size_t)wbk * stride, acc);
      const double* ps =
          part_s + ((size_t)(slot / sbk) * nparts * sbk + (slot % sbk)) * stride + off;
      acc = sum_strided(ps, nparts, (size_t)sbk * stride, acc);
    }
  } else {
    if (slot >= counts[1]) return;
    comp = ill_idx[slot];
    const int n_ikb = (counts[1] + ibk - 1) / ibk;
    const int nchk = ill_chunks(grid_i, n_ikb, n, ipt);
    const double* p = part_i + ((size_t)(slot / ibk) * nchk * ibk + (slot % ibk)) * stride + off;
    acc = sum_strided(p, nchk, (size_t)ibk * stride, acc);
  }
  if (c == 0) nk[comp] += acc;
  else if (c <= d) s[(int64_t)comp * d + (c - 1)] += acc;
  else q[(int64_t)comp * d + (c - 1 - d)] += acc;
}

__global__ __launch_bounds__(1024) void k_reduce_ll(const double* __restrict__ ll_part,
                                                    int64_t cnt, double* __restrict__ out,
                                                    int accumulate) {
  __shared__ double sh[1024];
  const int t = threadIdx.x;
  double a = 0.0;
  // entries t, t + 1024, ... added in that order; 16 loads in flight at a time
  int64_t i = t;
  for (; i + 15 * 1024 < cnt; i += 16 * 1024) {
    double v[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) v[j] = ll_part[i + 1024 * j];
#pragma unroll
    for (int j = 0; j < 16; ++j) a += v[j];
  }
  for (; i < cnt; i += 1024) a += ll_part[i];
  sh[t] = a;
  __syncthreads();
  for (int w = 512; w > 0; w >>= 1) {
    if (t < w) sh[t] += sh[t + w];
    __syncthreads();
  }
  if (t == 0) {
    const double v = sh[0] * kLn2;
    *out = accumulate ? *out + v : v;
  }
}

__global__ __launch_bounds__(256) void k_mstep(const double* __restrict__ nk,
                                               const double* __restrict__ s,
                                               const double* __restrict__ q, double n_total,
                                               int d, int k, double var_floor,
                                               float* __restrict__ w, float* __restrict__ mu,
                                               float* __restrict__ var) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= (int64_t)k * d) return;
  const int comp = (int)(t / d), j = (int)(t % d);
  const double nn = nk[comp];
  if (nn == 0.0) {  // dead component: keep mean and variances, weight 0
    if (j == 0) w[comp] = 0.0f;
    return;
  }
  const double m = s[t] / nn;
  double v = q[t] / nn - m * m;
  if (!(v > var_floor)) v = var_floor;
  mu[t] = (float)m;
  var[t] = (float)v;
  if (j == 0) w[comp] = (float)(nn / n_total);
}

// ---------------------------------------------------------------- isotropic model
// The paper's own model (Sec. 2): one variance per component, N(mu_k, var_k I).
// Its E-step is the diagonal one with var_kd = var_k for every d, so the
// isotropic calls expand the variances and run the diagonal kernels; the
// isotropic second moment is Q_k = sum_d Q_kd = sum_i r_ik ||x_i||^2.
__global__ __launch_bounds__(256) void k_iso_expand(const float* __restrict__ var_iso, int d,
                                                    int k, float* __restrict__ var) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= (int64_t)k * d) return;
  var[t] = var_iso[t / d];
}

// q[c] += sum_d qd[c d + j], dimensions in order, fp64.
__global__ __launch_bounds__(256) void k_iso_qsum(const double* __restrict__ qd, int d, int k,
                                                  double* __restrict__ q) {
  const int c = blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= k) return;
  double acc = 0.0;
  for (int j = 0; j < d; ++j) acc += qd[(int64_t)c * d + j];
  q[c] += acc;
}

// Isotropic M-step (Eqs. Nk, muk, sig): pi = N / n, mu = S / N and
// var = max(floor, (Q / N - ||mu||^2) / D), which is sum_i r ||x_i - mu||^2 / (D N)
// for the new mean; N == 0 exactly keeps mu and var and sets pi = 0.
__global__ __launch_bounds__(256) void k_mstep_iso(const double* __restrict__ nk,
                                                   const double* __restrict__ s,
                                                   const double* __restrict__ q, double n_total,
                                                   int d, int k, double var_floor,
                                                   float* __restrict__ w, float* __restrict__ mu,
                                                   float* __restrict__ var) {
  const int c = blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= k) return;
  const double nn = nk[c];
  if (nn == 0.0) {
    w[c] = 0.0f;
    return;
  }
  double mm = 0.0;
  for (int j = 0; j < d; ++j) {
    const double m = s[(int64_t)c * d + j] / nn;
    mm += m * m;
    mu[(int64_t)c * d + j] = (float)m;
  }
  double v = (q[c] / nn - mm) / (double)d;
  if (!(v > var_floor)) v = var_floor;
  var[c] = (float)v;
  w[c] = (float)(nn / n_total);
}

// ---------------------------------------------------------------- k-means++ seeding
// D^2 sampling (Arthur and Vassilvitskii 2007) with the caller's uniforms:
// centre 0 is row floor(u_0 n); centre t is the first row whose running sum
// of D^2 (squared distance to the nearest chosen centre) exceeds u_t times
// the total.  Every sum has a fixed order, so each choice is a pure function
// of the data and u: D^2 of a row is 16 fp64 partial sums (partial l takes
// the dimensions 4 (l + 16 j) + e, e = 0..3, j = 0, 1, ..., in that order,
// fma(t, t, acc), t = x - c) combined pairwise by xor 8, 4, 2, 1 (16 lanes per
// row, float4 loads where the rows allow them, the same order otherwise); a
// block of kKppBlock rows is kKppRuns runs of kKppRun consecutive rows; a run
// adds its rows in order, a block its runs; the total is the sum, in order,
// of 256 consecutive stretches of blocks, each summed in order, and the
// search walks stretches, blocks, runs and rows in that order.
constexpr int kKppRun = 16;
constexpr int kKppRuns = 64;
constexpr int kKppBlock = kKppRun * kKppRuns;

__device__ __forceinline__ int64_t kpp_first(double u, int64_t n) {
  int64_t i = (int64_t)(u * (double)n);
  return i < 0 ? 0 : (i >= n ? n - 1 : i);
}

// One workgroup per block: folds centre idx[t-1] into D^2 (first: D^2 is
// that centre's distance) and writes the block's sum.  Wave w of the 4 takes
// runs w, w + 4, ...; a run's 16 rows go 4 at a time, lane group g (16
// lanes) forming the D^2 of row 4 s + g, and lane 0 adds the rows in order.
__global__ __launch_bounds__(256) void k_kpp_update(const float* __restrict__ x, int64_t n, int d,
                                                   int vec4, const int64_t* __restrict__ idx,
                                                   int t, int first, double* __restrict__ dist,
                                                   double* __restrict__ bsum) {
  __shared__ double rsum[kKppRuns];
  __shared__ __align__(16) float cs[GMM_MAX_D];
  const int64_t b = blockIdx.x;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, g = lane >> 4, l16 = lane & 15;
  const float* c = x + idx[t - 1] * (int64_t)d;
  for (int e = tid; e < d; e += 256) cs[e] = c[e];
  __syncthreads();
  const int nc4 = (d + 3) / 4;                  // chunks of four dimensions
  for (int q = wave; q < kKppRuns; q += 4) {
    const int64_t r0 = b * kKppBlock + (int64_t)kKppRun * q;
    double rs = 0.0;
    for (int sub = 0; sub < kKppRun / 4; ++sub) {
      const int64_t i = r0 + 4 * sub + g;
      double v = 0.0;
      if (i < n) {
        const float* xr = x + i * (int64_t)d;
        double acc = 0.0;
        for (int c4 = l16; c4 < nc4; c4 += 16) {
          float xv[4];
          if (vec4) {
            const float4 f = *reinterpret_cast<const float4*>(xr + 4 * c4);
            xv[0] = f.x; xv[1] = f.y; xv[2] = f.z; xv[3] = f.w;
          } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) xv[e] = 4 * c4 + e < d ? xr[4 * c4 + e] : 0.0f;
          }
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            if (4 * c4 + e < d) {
              const double u = (double)xv[e] - (double)cs[4 * c4 + e];
              acc = fma(u, u, acc);
            }
          }
        }
        acc += __shfl_xor(acc, 8);
        acc += __shfl_xor(acc, 4);
        acc += __shfl_xor(acc, 2);
        acc += __shfl_xor(acc, 1);
        v = acc;
        if (l16 == 0) {
          const double old = dist[i];
          if (!first && !(acc < old)) v = old;
          dist[i] = v;
        }
      }
      // the run's rows in order (rows past n add 0)
#pragma unroll
      for (int gg = 0; gg < 4; ++gg) rs += __shfl(v, 16 * gg);
    }
    if (lane == 0) rsum[q] = rs;
  }
  __syncthreads();
  if (tid == 0) {
    double sb = 0.0;
    for (int q = 0; q < kKppRuns; ++q) sb += rsum[q];
    bsum[b] = sb;
  }
}

// One workgroup: centre t (t = 0: floor(u_0 n)) into idx[t] and its row into
// centres.  The blocks are taken in 256 consecutive stretches, thread j
// summing stretch j in order.
__global__ __launch_bounds__(256) void k_kpp_select(const float* __restrict__ x, int64_t n, int d,
                                                   const double* __restrict__ uu, int t,
                                                   const double* __restrict__ dist,
                                                   const double* __restrict__ bsum,
                                                   int64_t nblk, int64_t* __restrict__ idx,
                                                   float* __restrict__ centres) {
  __shared__ double ssum[256];
  __shared__ double rsum[kKppRuns];
  __shared__ double sh[2];      // run (sum of the blocks before), target
  __shared__ int64_t sb[2];     // block, pick
  const int j = threadIdx.x;
  const int64_t per = (nblk + 255) / 256;
  if (t > 0) {
    const int64_t s0 = per * j, s1 = s0 + per < nblk ? s0 + per : nblk;
    double ss = 0.0;
    for (int64_t b = s0; b < s1; ++b) ss += bsum[b];
    ssum[j] = ss;
  }
  __syncthreads();
  if (j == 0) {
    int64_t pick = -1, blk = -1;
    const double u = uu[t];
    if (t > 0) {
      double total = 0.0;
      for (int q = 0; q < 256; ++q) total += ssum[q];
      if (total > 0.0) {
        const double target = u * total;
        double run = 0.0;
        int q = 0;
        while (q + 1 < 256 && !(run + ssum[q] > target)) run += ssum[q++];
        int64_t b = per * q;
        const int64_t b1 = b + per < nblk ? b + per : nblk;
        while (b + 1 < b1 && !(run + bsum[b] > target)) run += bsum[b++];
        blk = b < nblk ? b : nblk - 1;
        sh[0] = run;
        sh[1] = target;
      }
    }
    if (blk < 0) pick = kpp_first(u, n);
    sb[0] = blk;
    sb[1] = pick;
  }
  __syncthreads();
  const int64_t blk = sb[0];
  if (blk >= 0) {
    // run sums of the block, as k_kpp_update formed them
    if (j < kKppRuns) {
      const int64_t r0 = blk * kKppBlock + (int64_t)kKppRun * j;
      double rs = 0.0;
      for (int64_t i = r0; i < r0 + kKppRun && i < n; ++i) rs += dist[i];
      rsum[j] = rs;
    }
    __syncthreads();
    if (j == 0) {
      const double run = sh[0], target = sh[1];
      double bs = 0.0;
      int64_t pick = -1;
      for (int q = 0; q < kKppRuns && pick < 0; ++q) {
        const int64_t q0 = blk * kKppBlock + (int64_t)kKppRun * q;
        if (q0 >= n) break;
        if (!(run + (bs + rsum[q]) > target)) {
          bs += rsum[q];
          continue;
        }
        double ps = 0.0;
        for (int64_t i = q0; i < q0 + kKppRun && i < n; ++i) {
          ps += dist[i];
          if (run + (bs + ps) > target) {
            pick = i;
            break;
          }
        }
      }
      sb[1] = pick >= 0 ? pick : kpp_first(uu[t], n);   // not reached for finite data
    }
  }
  __syncthreads();
  const int64_t pick = sb[1];
  if (j == 0) idx[t] = pick;
  for (int e = j; e < d; e += 256) centres[(int64_t)t * d + e] = x[pick * (int64_t)d + e];
}

// ---------------------------------------------------------------- k-means warm start
// Lloyd iterations with the pieces of the EM path: the nearest centre is the
// top-1 of the exact assignment with equal weights and unit variances (its
// ranking is the fp64 direct form, ties to the lower index), a row and its
// centre form one stored pair with r = 1, and the exact-pair pipeline sums
// them per centre in a fixed order (N_k, sum x, sum x^2, fp64).
__global__ __launch_bounds__(256) void k_km_fill(float* __restrict__ w, int k, float wv,
                                                 float* __restrict__ ones, int64_t kd) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t < k) w[t] = wv;
  if (t < kd) ones[t] = 1.0f;
}

__global__ __launch_bounds__(256) void k_km_pairs(const int* __restrict__ assign, int64_t n,
                                                  unsigned short* __restrict__ cslot,
                                                  float* __restrict__ cr) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int a = assign[i];
  *reinterpret_cast<ushort4*>(cslot + i * kT) =
      make_ushort4(a >= 0 ? (unsigned short)a : kNoSlot, kNoSlot, kNoSlot, kNoSlot);
  *reinterpret_cast<float4*>(cr + i * kT) = make_float4(a >= 0 ? 1.0f : 0.0f, 0.f, 0.f, 0.f);
}

// nk, s, q of every centre (slot = centre) from the exact-pair partials, parts in order.
__global__ __launch_bounds__(256) void k_km_reduce(const double* __restrict__ part_s,
                                                   int nparts, int sbk, int k, int d, int D64,
                                                   double* __restrict__ nk,
                                                   double* __restrict__ s,
                                                   double* __restrict__ q) {
  const int64_t width = 1 + 2 * (int64_t)d;
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= (int64_t)k * width) return;
  const int slot = (int)(t / width), c = (int)(t % width);
  const int64_t stride = 1 + 2 * (int64_t)D64;
  const int64_t off = c == 0 ? 0 : (c <= d ? 1 + (c - 1) : 1 + D64 + (c - 1 - d));
  const double* ps = part_s + ((size_t)(slot / sbk) * nparts * sbk + (slot % sbk)) * stride + off;
  const double acc = sum_strided(ps, nparts, (size_t)sbk * stride, 0.0);
  if (c == 0) nk[slot] = acc;
  else if (c <= d) s[(int64_t)slot * d + (c - 1)] = acc;
  else q[(int64_t)slot * d + (c - 1 - d)] = acc;
}

// centre = mean of its rows (fp64, stored fp32); a centre without rows stays.
__global__ __launch_bounds__(256) void k_km_move(const double* __restrict__ nk,
                                                 const double* __restrict__ s, int d, int k,
                                                 float* __restrict__ centres) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= (int64_t)k * d) return;
  const double nn = nk[t / d];
  if (nn > 0.0) centres[t] = (float)(s[t] / nn);
}

__global__ __launch_bounds__(256) void k_zero(double* __restrict__ p, int64_t cnt) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t < cnt) p[t] = 0.0;
}

// ---------------------------------------------------------------- host side
inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

struct Layout {
  int64_t n;
  int d, k, kpad, D64, m;
  bool wide;                // D64 > 256: 32-point screening tiles
  int wbk, nch;             // well statistics: components per workgroup (64 for
                            // k_stats_well, 16 for k_stats_wide at D64 >= 256), chunks
  int64_t chunk;
  int ibk, ipt, grid_i;     // ill set: components per block, points per tile, grid
  int sbk, lsbk, nb;        // refined pairs: bucket size (log2), buckets
  int nunit, nparts;        // refined pairs: units, parts per bucket
  int64_t upts;
  int pts_logz;
  int64_t n_wg_logz;
  bool bmask_on;            // per-point dense-block masks (at most 64 blocks of 64 components)
  bool refine = true;       // false: the screened E-step (no direct-form refinement)
  bool iso = false;         // tied variances: [x | ||x||^2] screening (split-bf16 path)
  size_t off_counts, off_cls, off_cwell, off_cdir, off_cthr, off_thr, off_well_idx, off_ill_idx,
      off_cw, off_wp, off_wq, off_wpb, off_dmu, off_dh, off_logz2, off_cslot, off_cr, off_llpart,
      off_part_w, off_part_s, off_part_i, off_scnt, off_soff, off_slist, off_bmask, off_fit_nk,
      off_fit_s, off_fit_q, off_iso_var, off_iso_q, off_iflag, off_sflag, off_spos, off_sidx,
      off_scnt2, off_part_x, off_lflag, total;
};

// Process-wide cap on the number of point chunks of the dense statistics pass
// (0: the automatic count).  Set by gmm_set_stats_chunk_limit.
int g_stats_chunk_cap = 0;

// Padded dimension count of the kernels: a multiple of 64 up to 256, of 128 above.
inline int padded_d(int d) { return d <= 256 ? (int)cdiv(d, 64) * 64 : (int)cdiv(d, 128) * 128; }

void layout_offsets(Layout* L);

// budget > 0: shrink the split counts until the workspace fits in `budget`
// bytes (false if it cannot).
bool make_layout(int64_t n, int d, int k, int m, Layout* L, size_t budget = 0) {
  if (n < 1 || d < 1 || k < 1 || d > GMM_MAX_D || k > GMM_MAX_K || m < 0 || m > GMM_MAX_M)
    return false;
  L->n = n; L->d = d; L->k = k; L->m = m;
  L->kpad = (int)cdiv(k, kWB) * kWB;
  L->D64 = padded_d(d);
  L->wide = L->D64 > 256;
  const int stride = 1 + 2 * L->D64;
  // chunking depends only on (n, d, k), never on the device
  L->wbk = L->D64 >= 256 ? 16 : kWB;
  const int nwb = L->kpad / L->wbk;
  if (L->D64 < 256) {
    // about 2048 workgroups (four rounds at two per CU) for k_stats_well, and
    // up to 8192 while the chunks keep 65536 points or more: the blocks'
    // shares of the points differ, and many short rounds let the workgroups
    // of the busy blocks spread over the chip and leave no long tail, while
    // a workgroup's fixed cost (its operands, its partial sums) stays small
    int maxc = 2048 / nwb;
    {
      const int64_t more = cdiv(n, 65536) < 8192 / nwb ? cdiv(n, 65536) : 8192 / nwb;
      if (more > maxc) maxc = (int)more;
    }
    if (maxc < 8) maxc = 8;
    int64_t c = cdiv(n, 1024);
    if (c > maxc) c = maxc;
    if (c >= 8) c = c / 8 * 8;
    L->nch = (int)(c < 1 ? 1 : c);
  } else {
    int maxc = 2048 / nwb;
    {
      const int64_t more = cdiv(n, 65536) < 8192 / nwb ? cdiv(n, 65536) : 8192 / nwb;
      if (more > maxc) maxc = (int)more;
    }
    if (maxc < 1) maxc = 1;
    int64_t c = cdiv(n, 1024);
    if (c > maxc) c = maxc;
    L->nch = (int)(c < 1 ? 1 : c);
  }
  {
    // the caller's cap on the chunk count (gmm_set_stats_chunk_limit); fewer,
    // longer chunks never need more workspace
    const int cap = g_stats_chunk_cap;
    if (cap > 0 && L->nch > cap) L->nch = cap;
  }
  L->chunk = cdiv(n, L->nch);
  L->sbk = L->wide ? (L->D64 <= 512 ? 8 : 4) : (L->D64 <= 128 ? 32 : 16);
  L->lsbk = L->sbk == 32 ? 5 : (L->sbk == 16 ? 4 : (L->sbk == 8 ? 3 : 2));
  L->nb = L->kpad / L->sbk;
  {
    int64_t u = cdiv(n, 256);
    const int64_t cap = kSparseTab / L->nb;
    if (u > cap) u = cap;
    L->nunit = (int)(u < 1 ? 1 : u);
    L->upts = cdiv(n, L->nunit);
    // about 8192 workgroups for the exact pairs (16384 for rows of more than
    // 512 dimensions, one workgroup per compute unit), so that the parts of
    // the buckets of popular components, whose lists are the longest, leave
    // no long tail; but the parts' partial sums (kpad pp rows of 1 + 2 D64
    // doubles) no larger than a quarter of X, which they would outweigh at
    // small n, unless that leaves fewer than about 1024 workgroups
    int64_t pp = (L->D64 > 512 ? 16384 : 8192) / L->nb;
    int64_t by_bytes = n * (int64_t)d / (8 * (int64_t)L->kpad * stride);
    if (by_bytes < 1024 / L->nb) by_bytes = 1024 / L->nb;
    if (pp > by_bytes) pp = by_bytes;
    L->nparts = (int)(pp < 1 ? 1 : pp);
  }
  L->ipt = L->D64 <= 256 ? 64 : (L->D64 <= 512 ? 32 : 16);
  L->ibk = 4 * (L->D64 <= 256 ? 8 : (L->D64 <= 512 ? 4 : 2));
  {
    // at least one workgroup per block of routed components; about 512 in all,
    // but no more chunks than tiles of points
    const int64_t nib = cdiv(k, L->ibk);
    int64_t g = nib * cdiv(n, L->ipt);
    if (g > 512) g = 512;
    L->grid_i = (int)(g > nib ? g : nib);
  }
  L->pts_logz = L->D64 <= 256 ? 64 : 32;
  L->n_wg_logz = cdiv(n, L->pts_logz);
  L->bmask_on = L->kpad / kWB <= 64;
  layout_offsets(L);
  if (budget > 0) {
    // fewer chunks of the dense statistics, fewer parts of the exact pairs and
    // fewer chunks of the routed components (each a change of summation
    // splits only) until the workspace fits the budget
    const int nib = (int)cdiv(k, L->ibk);
    while (L->total > budget) {
      if (L->nch > 1) {
        L->nch = (L->nch + 1) / 2;
        L->chunk = cdiv(n, L->nch);
      } else if (L->nparts > 1) {
        L->nparts = (L->nparts + 1) / 2;
      } else if (L->grid_i > nib) {
        L->grid_i = (L->grid_i + 1) / 2 > nib ? (L->grid_i + 1) / 2 : nib;
      } else {
        return false;
      }
      layout_offsets(L);
    }
  }
  return true;
}

// Byte offsets of the workspace regions for the layout's sizes.
void layout_offsets(Layout* L) {
  const int64_t n = L->n;
  const int d = L->d, k = L->k;
  const int stride = 1 + 2 * L->D64;
  const int nwb = L->kpad / L->wbk;
  size_t o = 0;
  auto take = [&](size_t bytes) { const size_t r = o; o = align256(o + bytes); return r; };
  L->off_counts = take(16 * sizeof(int));
  L->off_cls = take((size_t)k * sizeof(int));
  L->off_cwell = take((size_t)k * sizeof(double));
  L->off_cdir = take((size_t)k * sizeof(double));
  L->off_well_idx = take((size_t)k * sizeof(int));
  L->off_ill_idx = take((size_t)k * sizeof(int));
  L->off_cw = take((size_t)L->kpad * sizeof(float));
  L->off_cthr = take((size_t)k * sizeof(float2));
  L->off_thr = take((size_t)L->kpad * sizeof(float2));
  L->off_wp = take((size_t)L->kpad * 2 * L->D64 * sizeof(float));
  L->off_wq = take((size_t)(L->kpad / 16) * (L->D64 / 2 + L->D64 / 32) * 64 * sizeof(float));
  L->off_wpb = take(screen_split(L->D64) ? (size_t)L->kpad * L->D64 * 8 : 16);
  L->off_dmu = take((size_t)k * L->D64 * sizeof(float));
  L->off_dh = take((size_t)k * L->D64 * sizeof(double));
  L->off_logz2 = take((size_t)n * sizeof(double));
  // refined slots (16-bit); gmm_assign_topk reuses the region for n int flags
  L->off_cslot = take((size_t)n * kT * sizeof(unsigned short));
  L->off_cr = take((size_t)n * kT * sizeof(float));
  L->off_llpart = take((size_t)L->n_wg_logz * sizeof(double));
  L->off_part_w = take((size_t)nwb * L->nch * L->wbk * stride * sizeof(double));
  L->off_part_s = take((size_t)L->nb * L->nparts * L->sbk * stride * sizeof(double));
  L->off_part_i = take((size_t)L->grid_i * L->ibk * stride * sizeof(double));
  L->off_scnt = take((size_t)L->nb * L->nunit * sizeof(int));
  L->off_soff = take(((size_t)L->nb * L->nunit + 1) * sizeof(int64_t));
  L->off_slist = take((size_t)n * kT * sizeof(SPair));
  L->off_bmask = take(L->bmask_on ? (size_t)n * sizeof(unsigned long long) : 16);
  // per point: a light component holds more than about 2^-72 of it
  L->off_lflag = take((size_t)n);
  L->off_iflag = take((size_t)n);                // points with a routed component's mass
  // light components recomputed exactly: flags, list positions, the list, its
  // length and the partials of its k_stats_ill pass
  L->off_sflag = take((size_t)k);
  L->off_spos = take((size_t)k * sizeof(int));
  L->off_sidx = take((size_t)k * sizeof(int));
  L->off_scnt2 = take(16 * sizeof(int));
  L->off_part_x = take((size_t)L->grid_i * L->ibk * stride * sizeof(double));
  L->off_fit_nk = take((size_t)k * sizeof(double) + sizeof(double));  // + loglik slot
  L->off_fit_s = take((size_t)k * d * sizeof(double));
  L->off_fit_q = take((size_t)k * d * sizeof(double));
  // isotropic calls: the expanded variances and the isotropic Q of gmm_fit_iso
  L->off_iso_var = take((size_t)k * d * sizeof(float));
  L->off_iso_q = take((size_t)k * sizeof(double));
  L->total = o;
}

template <typename T>
T* at(void* ws, size_t off) { return reinterpret_cast<T*>(static_cast<char*>(ws) + off); }

int launch_status() {
  const hipError_t e = hipGetLastError();
  return e == hipSuccess ? GMM_OK : GMM_ERR_DEVICE;
}

// ---------------------------------------------------------------- phase timing
// Measurement aid: while enabled, every E-step records HIP events on its
// stream between its phases, waits for the last one and adds the phase
// durations up.  Process-wide state for one device; not for concurrent calls.
struct PhaseTimer {
  bool on = false;
  bool made = false;
  hipEvent_t ev[GMM_TIMING_PHASES + 1];
  double ms[GMM_TIMING_PHASES] = {};
  int64_t calls = 0;
};
PhaseTimer g_timer;

inline bool phase_mark(int i, hipStream_t st) {
  return !g_timer.on || hipEventRecord(g_timer.ev[i], st) == hipSuccess;
}

inline bool phase_collect() {
  if (!g_timer.on) return true;
  if (hipEventSynchronize(g_timer.ev[GMM_TIMING_PHASES]) != hipSuccess) return false;
  for (int i = 0; i < GMM_TIMING_PHASES; ++i) {
    float t = 0.0f;
    if (hipEventElapsedTime(&t, g_timer.ev[i], g_timer.ev[i + 1]) != hipSuccess) return false;
    g_timer.ms[i] += t;
  }
  ++g_timer.calls;
  return true;
}

template <int D64>
int estep_impl(const Layout& L, const float* x, const float* w, const float* mu,
               const float* var, double* nk, double* s, double* q, double* loglik,
               int ll_accumulate, void* ws, hipStream_t st) {
  const int64_t n = L.n;
  const int d = L.d, k = L.k, kpad = L.kpad;
  int* counts = at<int>(ws, L.off_counts);
  int* cls = at<int>(ws, L.off_cls);
  double* cwell = at<double>(ws, L.off_cwell);
  double* cdir = at<double>(ws, L.off_cdir);
  int* well_idx = at<int>(ws, L.off_well_idx);
  int* ill_idx = at<int>(ws, L.off_ill_idx);
  float* cw = at<float>(ws, L.off_cw);
  float2* cthr = at<float2>(ws, L.off_cthr);
  float2* thr = at<float2>(ws, L.off_thr);
  float4* wp = at<float4>(ws, L.off_wp);
  float* wq = at<float>(ws, L.off_wq);
  float* dmu = at<float>(ws, L.off_dmu);
  double* dh = at<double>(ws, L.off_dh);
  unsigned short* cslot = at<unsigned short>(ws, L.off_cslot);
  float* cr = at<float>(ws, L.off_cr);
  double* logz2 = at<double>(ws, L.off_logz2);
  double* llpart = at<double>(ws, L.off_llpart);
  double* part_w = at<double>(ws, L.off_part_w);
  double* part_s = at<double>(ws, L.off_part_s);
  double* part_i = at<double>(ws, L.off_part_i);
  const int vec4 = ((d & 3) == 0 && (reinterpret_cast<uintptr_t>(x) & 15) == 0) ? 1 : 0;
  bf16x8* wpb = at<bf16x8>(ws, L.off_wpb);
  unsigned long long* bmask = L.bmask_on ? at<unsigned long long>(ws, L.off_bmask) : nullptr;
  unsigned char* lflag = at<unsigned char>(ws, L.off_lflag);
  unsigned char* iflag = at<unsigned char>(ws, L.off_iflag);

  bool tm = phase_mark(0, st);
  hipLaunchKernelGGL(k_prep_class, dim3(k), dim3(64), 0, st, w, mu, var, d, cls, cwell, cdir,
                     cthr);
  hipLaunchKernelGGL(k_prep_scan, dim3(1), dim3(256), 0, st, cls, k, well_idx, ill_idx, counts);
  {
    const int64_t tot = (int64_t)kpad * (D64 / 4) * 2;
    hipLaunchKernelGGL(k_prep_pack_well<D64>, dim3((unsigned)cdiv(tot, 256)), dim3(256), 0, st,
                       mu, var, d, kpad, cwell, cthr, counts, well_idx, wp, cw, thr);
    if constexpr (screen_x16(D64)) {
      if (L.iso && L.refine) {
        const int64_t tb = (int64_t)(kpad / kBK) * screen_steps<D64, true>() * 64;
        hipLaunchKernelGGL((k_prep_pack_b16<D64, true>), dim3((unsigned)cdiv(tb, 256)), dim3(256),
                           0, st, mu, var, d, kpad, counts, well_idx, wpb);
      } else {
        const int64_t tb = (int64_t)(kpad / kBK) * screen_steps<D64, false>() * 64;
        hipLaunchKernelGGL((k_prep_pack_b16<D64, false>), dim3((unsigned)cdiv(tb, 256)),
                           dim3(256), 0, st, mu, var, d, kpad, counts, well_idx, wpb);
      }
    }
    if constexpr (screen_b16(D64)) {
      if (L.iso) {
        const int64_t tb = (int64_t)(kpad / kBK) * screen_steps<D64, true>() * 64;
        hipLaunchKernelGGL((k_prep_pack_b16<D64, true>), dim3((unsigned)cdiv(tb, 256)), dim3(256),
                           0, st, mu, var, d, kpad, counts, well_idx, wpb);
      } else {
        const int64_t tb = (int64_t)(kpad / kBK) * screen_steps<D64, false>() * 64;
        hipLaunchKernelGGL((k_prep_pack_b16<D64, false>), dim3((unsigned)cdiv(tb, 256)),
                           dim3(256), 0, st, mu, var, d, kpad, counts, well_idx, wpb);
      }
    }
    if (D64 < 256 && L.iso)
      hipLaunchKernelGGL((k_prep_pack_w16<D64, true>),
                         dim3((unsigned)cdiv((int64_t)(kpad / 16) * wq_steps_iso(D64) * 64, 256)),
                         dim3(256), 0, st, w, mu, var, d, kpad, counts, well_idx, wq);
    else
      hipLaunchKernelGGL((k_prep_pack_w16<D64, false>),
                         dim3((unsigned)cdiv((int64_t)(kpad / 16) * wq_steps(D64) * 64, 256)),
                         dim3(256), 0, st, w, mu, var, d, kpad, counts, well_idx, wq);
    const int64_t toti = (int64_t)k * D64;
    hipLaunchKernelGGL(k_prep_pack_direct<D64>, dim3((unsigned)cdiv(toti, 256)), dim3(256), 0,
                       st, mu, var, d, k, dmu, dh);
  }
  tm = phase_mark(1, st) && tm;
  bool launched = false;
  if constexpr (screen_split(D64)) {
    if (L.iso && L.refine) {
      hipLaunchKernelGGL((k_logz<D64, true, true>), dim3((unsigned)L.n_wg_logz), dim3(256), 0, st,
                         x, n, d, vec4, wp, wpb, cw, thr, well_idx, ill_idx, dmu, dh, cdir, counts,
                         logz2, cslot, cr, llpart, bmask, iflag, lflag);
      launched = true;
    }
  }
  if (!launched) {
    if (L.refine)
      hipLaunchKernelGGL((k_logz<D64, true, false>), dim3((unsigned)L.n_wg_logz), dim3(256), 0, st,
                         x, n, d, vec4, wp, wpb, cw, thr, well_idx, ill_idx, dmu, dh, cdir, counts,
                         logz2, cslot, cr, llpart, bmask, iflag, lflag);
    else
      hipLaunchKernelGGL((k_logz<D64, false, false>), dim3((unsigned)L.n_wg_logz), dim3(256), 0,
                         st, x, n, d, vec4, wp, wpb, cw, thr, well_idx, ill_idx, dmu, dh, cdir,
                         counts, logz2, cslot, cr, llpart, bmask, iflag, lflag);
  }
  tm = phase_mark(2, st) && tm;
  {
    // the stored exact pairs, in fp64
    int* scnt = at<int>(ws, L.off_scnt);
    int64_t* soff = at<int64_t>(ws, L.off_soff);
    SPair* slist = at<SPair>(ws, L.off_slist);
    const size_t lds = (size_t)L.nb * sizeof(int);
    hipLaunchKernelGGL(k_sparse_count, dim3((unsigned)L.nunit), dim3(64), lds, st, cslot, n,
                       L.upts, L.nb, L.lsbk, L.nunit, scnt);
    hipLaunchKernelGGL(k_sparse_scan, dim3(1), dim3(1024), 0, st, scnt, L.nb * L.nunit, soff);
    hipLaunchKernelGGL(k_sparse_scatter, dim3((unsigned)L.nunit), dim3(64), scatter_lds(L.nb), st,
                       cslot, cr, n, L.upts, L.nb, L.lsbk, L.nunit, soff, slist);
    hipLaunchKernelGGL(k_stats_sparse<D64>, dim3((unsigned)(L.nb * L.nparts)),
                       dim3(64 * kSparseWaves), 0, st,
                       x, n, d, slist, soff, L.nunit, L.nparts, part_s);
  }
  tm = phase_mark(3, st) && tm;
  // light components (exact path only): their stored pairs' mass is below
  // kSmallMass; the dense pass leaves them out and flags their points
  int* spos = nullptr;
  double* part_x = at<double>(ws, L.off_part_x);
  int* scnt2 = at<int>(ws, L.off_scnt2);
  unsigned char* sflag = nullptr;
  int* sidx = at<int>(ws, L.off_sidx);
  if (L.refine) {
    sflag = at<unsigned char>(ws, L.off_sflag);
    spos = at<int>(ws, L.off_spos);
    hipLaunchKernelGGL(k_small_mass, dim3((unsigned)cdiv(k, 256)), dim3(256), 0, st, part_s,
                       counts, well_idx, cdir, L.nparts, L.sbk, D64, sflag);
    hipLaunchKernelGGL(k_small_list, dim3(1), dim3(1024), 0, st, sflag, counts, well_idx, spos,
                       sidx, scnt2);
  }
  if constexpr (D64 < 256) {
    if (L.iso)
      hipLaunchKernelGGL((k_stats_well<D64, true>), dim3((unsigned)((kpad / kWB) * L.nch)),
                         dim3(256), 0, st, x, n, d, vec4, wq, cw, counts, logz2, cslot, bmask,
                         L.nch, L.chunk, sflag, lflag, part_w);
    else
      hipLaunchKernelGGL((k_stats_well<D64, false>), dim3((unsigned)((kpad / kWB) * L.nch)),
                         dim3(256), 0, st, x, n, d, vec4, wq, cw, counts, logz2, cslot, bmask,
                         L.nch, L.chunk, sflag, lflag, part_w);
  } else {
    if (L.iso)
      hipLaunchKernelGGL((k_stats_wide<D64, true>), dim3((unsigned)((kpad / 16) * L.nch)),
                         dim3(64 * (D64 / 128)), 0, st, x, n, d, vec4, wq, cwell, well_idx,
                         counts, logz2, cslot, bmask, L.nch, L.chunk, sflag, lflag, part_w);
    else
      hipLaunchKernelGGL((k_stats_wide<D64, false>), dim3((unsigned)((kpad / 16) * L.nch)),
                         dim3(64 * (D64 / 128)), 0, st, x, n, d, vec4, wq, cwell, well_idx,
                         counts, logz2, cslot, bmask, L.nch, L.chunk, sflag, lflag, part_w);
  }
  tm = phase_mark(4, st) && tm;
  hipLaunchKernelGGL(k_stats_ill<D64>, dim3((unsigned)L.grid_i), dim3(256), 0, st, x, n, d, vec4,
                     ill_idx, dmu, dh, cdir, counts, logz2, iflag, nullptr, nullptr, nullptr,
                     part_i);
  if (L.refine)
    hipLaunchKernelGGL(k_stats_ill<D64>, dim3((unsigned)L.grid_i), dim3(256), 0, st, x, n, d,
                       vec4, sidx, dmu, dh, cdir, scnt2, logz2, nullptr, lflag, cslot, spos,
                       part_x);
  {
    const int64_t tot = 2 * (int64_t)k * (1 + 2 * (int64_t)d);
    hipLaunchKernelGGL(k_reduce_stats, dim3((unsigned)cdiv(tot, 256)), dim3(256), 0, st, part_w,
                       part_s, part_i, counts, well_idx, ill_idx, L.nch, L.wbk, L.nparts, L.sbk,
                       L.grid_i, L.ibk, L.ipt, n, k, d, D64, spos, part_x, scnt2, nk, s, q);
  }
  hipLaunchKernelGGL(k_reduce_ll, dim3(1), dim3(1024), 0, st, llpart, L.n_wg_logz, loglik,
                     ll_accumulate);
  const int rc = launch_status();
  if (rc != GMM_OK) return rc;
  tm = phase_mark(GMM_TIMING_PHASES, st) && tm;
  return tm && phase_collect() ? GMM_OK : GMM_ERR_DEVICE;
}

template <int D64>
int assign_impl(const Layout& L, const float* x, const float* w, const float* mu,
                const float* var, int m, float tau, int* idx, float* resp, void* ws,
                hipStream_t st) {
  const int64_t n = L.n;
  const int d = L.d, k = L.k, kpad = L.kpad;
  int* counts = at<int>(ws, L.off_counts);
  int* cls = at<int>(ws, L.off_cls);
  double* cwell = at<double>(ws, L.off_cwell);
  double* cdir = at<double>(ws, L.off_cdir);
  float2* cthr = at<float2>(ws, L.off_cthr);
  float2* thr = at<float2>(ws, L.off_thr);
  int* well_idx = at<int>(ws, L.off_well_idx);
  int* ill_idx = at<int>(ws, L.off_ill_idx);
  float* cw = at<float>(ws, L.off_cw);
  float4* wp = at<float4>(ws, L.off_wp);
  float* dmu = at<float>(ws, L.off_dmu);
  double* dh = at<double>(ws, L.off_dh);
  float2* theta = at<float2>(ws, L.off_logz2);    // n float pairs, free during assignment
  int* ovf = at<int>(ws, L.off_cslot);            // n ints, likewise
  float2* ca = thr;                               // kpad pairs, likewise
  bf16x8* wpb = at<bf16x8>(ws, L.off_wpb);
  const int vec4 = ((d & 3) == 0 && (reinterpret_cast<uintptr_t>(x) & 15) == 0) ? 1 : 0;
  hipLaunchKernelGGL(k_prep_class, dim3(k), dim3(64), 0, st, w, mu, var, d, cls, cwell, cdir,
                     cthr);
  hipLaunchKernelGGL(k_prep_scan, dim3(1), dim3(256), 0, st, cls, k, well_idx, ill_idx, counts);
  {
    const int64_t tot = (int64_t)kpad * (D64 / 4) * 2;
    hipLaunchKernelGGL(k_prep_pack_well<D64>, dim3((unsigned)cdiv(tot, 256)), dim3(256), 0, st,
                       mu, var, d, kpad, cwell, cthr, counts, well_idx, wp, cw, thr);
    const int64_t toti = (int64_t)k * D64;
    hipLaunchKernelGGL(k_prep_pack_direct<D64>, dim3((unsigned)cdiv(toti, 256)), dim3(256), 0,
                       st, mu, var, d, k, dmu, dh);
    if constexpr (screen_split(D64)) {
      const int64_t tb = (int64_t)(kpad / kBK) * screen_steps<D64, false>() * 64;
      hipLaunchKernelGGL((k_prep_pack_b16<D64, false>), dim3((unsigned)cdiv(tb, 256)), dim3(256),
                         0, st, mu, var, d, kpad, counts, well_idx, wpb);
      hipLaunchKernelGGL(k_assign_slots, dim3((unsigned)cdiv(kpad, 256)), dim3(256), 0, st,
                         cwell, cdir, counts, well_idx, kpad, ca);
    }
  }
  if (m + 2 <= 4)
    hipLaunchKernelGGL((k_assign_theta<D64, 4>), dim3((unsigned)L.n_wg_logz), dim3(256), 0, st, x,
                       n, d, vec4, wp, wpb, cw, ca, counts, m + 2, theta);
  else
    hipLaunchKernelGGL((k_assign_theta<D64, kTMax>), dim3((unsigned)L.n_wg_logz), dim3(256), 0, st,
                       x, n, d, vec4, wp, wpb, cw, ca, counts, m + 2, theta);
  hipLaunchKernelGGL(k_assign_collect<D64>, dim3((unsigned)L.n_wg_logz), dim3(256), 0, st, x, n,
                     d, vec4, wp, wpb, cw, ca, well_idx, ill_idx, dmu, dh, counts, theta, mu, var,
                     cdir, m, tau, idx, resp, ovf);
  hipLaunchKernelGGL(k_assign_fallback, dim3((unsigned)cdiv(n, 1024)), dim3(256), 0, st, x, n, d,
                     k, mu, var, cdir, m, tau, ovf, idx, resp);
  return launch_status();
}

#define GMM_FOR_EACH_D64(X) \
  X(64) X(128) X(192) X(256) X(384) X(512) X(640) X(768) X(896) X(1024)

// n_iters Lloyd iterations on `means` (the centres), a last assignment, and
// the hard-assignment mixture by the M-step (k_mstep with r in {0, 1}).
template <int D64>
int kmeans_impl(const Layout& L, const float* x, int n_iters, float var_floor, float* weights,
                float* means, float* vars, int* assign, void* ws, hipStream_t st) {
  const int64_t n = L.n;
  const int d = L.d, k = L.k;
  const int64_t kd = (int64_t)k * d;
  float* weq = at<float>(ws, L.off_iso_q);       // k floats: equal weights
  float* ones = at<float>(ws, L.off_iso_var);    // k*d unit variances
  unsigned short* cslot = at<unsigned short>(ws, L.off_cslot);
  float* cr = at<float>(ws, L.off_cr);
  double* fnk = at<double>(ws, L.off_fit_nk);
  double* fs = at<double>(ws, L.off_fit_s);
  double* fq = at<double>(ws, L.off_fit_q);
  double* part_s = at<double>(ws, L.off_part_s);
  int* scnt = at<int>(ws, L.off_scnt);
  int64_t* soff = at<int64_t>(ws, L.off_soff);
  SPair* slist = at<SPair>(ws, L.off_slist);
  hipLaunchKernelGGL(k_km_fill, dim3((unsigned)cdiv(kd > k ? kd : k, 256)), dim3(256), 0, st, weq,
                     k, 1.0f / (float)k, ones, kd);
  for (int it = 0; it <= n_iters; ++it) {
    // nearest centre; the top-1 responsibility goes to the cr region, which the
    // pairs overwrite below
    int rc = assign_impl<D64>(L, x, weq, means, ones, 1, 0.0f, assign, cr, ws, st);
    if (rc != GMM_OK) return rc;
    hipLaunchKernelGGL(k_km_pairs, dim3((unsigned)cdiv(n, 256)), dim3(256), 0, st, assign, n,
                       cslot, cr);
    const size_t lds = (size_t)L.nb * sizeof(int);
    hipLaunchKernelGGL(k_sparse_count, dim3((unsigned)L.nunit), dim3(64), lds, st, cslot, n,
                       L.upts, L.nb, L.lsbk, L.nunit, scnt);
    hipLaunchKernelGGL(k_sparse_scan, dim3(1), dim3(1024), 0, st, scnt, L.nb * L.nunit, soff);
    hipLaunchKernelGGL(k_sparse_scatter, dim3((unsigned)L.nunit), dim3(64), scatter_lds(L.nb), st,
                       cslot, cr, n, L.upts, L.nb, L.lsbk, L.nunit, soff, slist);
    hipLaunchKernelGGL(k_stats_sparse<D64>, dim3((unsigned)(L.nb * L.nparts)),
                       dim3(64 * kSparseWaves), 0, st,
                       x, n, d, slist, soff, L.nunit, L.nparts, part_s);
    hipLaunchKernelGGL(k_km_reduce, dim3((unsigned)cdiv((int64_t)k * (1 + 2 * (int64_t)d), 256)),
                       dim3(256), 0, st, part_s, L.nparts, L.sbk, k, d, D64, fnk, fs, fq);
    if (it < n_iters)
      hipLaunchKernelGGL(k_km_move, dim3((unsigned)cdiv(kd, 256)), dim3(256), 0, st, fnk, fs, d,
                         k, means);
  }
  hipLaunchKernelGGL(k_mstep, dim3((unsigned)cdiv(kd, 256)), dim3(256), 0, st, fnk, fs, fq,
                     (double)n, d, k, (double)var_floor, weights, means, vars);
  return launch_status();
}

int estep_dispatch(const Layout& L, const float* x, const float* w, const float* mu,
                   const float* var, double* nk, double* s, double* q, double* loglik,
                   int ll_accumulate, void* ws, hipStream_t st) {
  switch (L.D64) {
#define GMM_CASE(D) \
  case D: return estep_impl<D>(L, x, w, mu, var, nk, s, q, loglik, ll_accumulate, ws, st);
    GMM_FOR_EACH_D64(GMM_CASE)
#undef GMM_CASE
    default: return GMM_ERR_UNSUPPORTED;
  }
}

int check_ws(const Layout& L, void* ws, size_t ws_bytes) {
  if (ws == nullptr || (reinterpret_cast<uintptr_t>(ws) & 255) != 0 || ws_bytes < L.total)
    return GMM_ERR_WORKSPACE;
  return GMM_OK;
}

int check_shape(int64_t n, int32_t d, int32_t k) {
  if (n < 1 || d < 1 || k < 1) return GMM_ERR_INVALID_ARG;
  if (d > GMM_MAX_D || k > GMM_MAX_K) return GMM_ERR_UNSUPPORTED;
  return GMM_OK;
}

// Events of one streamed E-step call: start (the compute stream's work before
// the call), and per staging buffer b: up[b] (its chunk uploaded) and done[b]
// (the E-step that read it finished).  Each call makes its own and releases
// them once everything is enqueued (HIP frees an event only after its
// pending records and waits), so concurrent calls never share one.
struct StreamEvents {
  hipEvent_t ev[5] = {nullptr, nullptr, nullptr, nullptr, nullptr};
  hipEvent_t& start() { return ev[0]; }
  hipEvent_t& up(int b) { return ev[1 + b]; }
  hipEvent_t& done(int b) { return ev[3 + b]; }
  bool make() {
    for (hipEvent_t& e : ev)
      if (hipEventCreateWithFlags(&e, hipEventDisableTiming) != hipSuccess) return false;
    return true;
  }
  ~StreamEvents() {
    for (hipEvent_t e : ev)
      if (e) (void)hipEventDestroy(e);
  }
};

// ---------------------------------------------------------------- allocation-free E-step
// The workspace of gmm_estep_accumulate_static: an array of the library's
// code object, one per GPU, which that GPU holds until the process ends.  Host
// code never uses the array's name as an address: its device address on each
// GPU comes from hipGetSymbolAddress, taken once per device with the device
// current.  Every call on a GPU uses the same array, so calls that overlap on
// one GPU race; nothing in it needs to start at zero (every region is written
// before it is read within a call).
constexpr size_t kStaticScratchBytes = (size_t)64 << 20;
constexpr int kStaticMaxDevices = 64;
__device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

struct StaticScratch {
  std::mutex mu;
  void* ptr[kStaticMaxDevices] = {};
};
StaticScratch g_static;

// The device address of `scratch` on the current device (looked up on the
// device's first call, then reused).
int static_scratch(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kStaticMaxDevices)
    return GMM_ERR_DEVICE;
  std::lock_guard<std::mutex> lock(g_static.mu);
  if (g_static.ptr[dev] == nullptr) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr)
      return GMM_ERR_DEVICE;
    g_static.ptr[dev] = p;
  }
  *out = g_static.ptr[dev];
  return GMM_OK;
}

}  // namespace

extern "C" {

int gmm_estep_accumulate_static(const float* x, int64_t n, int32_t d, int32_t k,
                                const float* weights, const float* means, const float* vars,
                                double* nk, double* s, double* q, double* loglik,
                                hipStream_t stream) {
  int rc = check_shape(n, d, k);
  if (rc != GMM_OK) return rc;
  if (!x || !weights || !means || !vars || !nk || !s || !q || !loglik) return GMM_ERR_INVALID_ARG;
  Layout L;
  // the split counts shrink until the workspace fits the static array; a
  // shape whose per-point buffers alone exceed it is refused
  if (!make_layout(n, d, k, 0, &L, kStaticScratchBytes)) return GMM_ERR_WORKSPACE;
  void* ws = nullptr;
  rc = static_scratch(&ws);
  if (rc != GMM_OK) return rc;
  return estep_dispatch(L, x, weights, means, vars, nk, s, q, loglik, 1, ws, stream);
}

int gmm_timing_enable(int on) {
  if (on && !g_timer.made) {
    for (int i = 0; i <= GMM_TIMING_PHASES; ++i)
      if (hipEventCreate(&g_timer.ev[i]) != hipSuccess) return GMM_ERR_DEVICE;
    g_timer.made = true;
  }
  g_timer.on = on != 0;
  for (int i = 0; i < GMM_TIMING_PHASES; ++i) g_timer.ms[i] = 0.0;
  g_timer.calls = 0;
  return GMM_OK;
}

int gmm_timing_read(double* ms, int32_t n_phases, int64_t* calls) {
  if (!ms || !calls || n_phases < 0) return GMM_ERR_INVALID_ARG;
  for (int i = 0; i < n_phases; ++i) ms[i] = i < GMM_TIMING_PHASES ? g_timer.ms[i] : 0.0;
  *calls = g_timer.calls;
  return GMM_OK;
}

int gmm_set_stats_chunk_limit(int32_t max_chunks) {
  if (max_chunks < 0) return GMM_ERR_INVALID_ARG;
  g_stats_chunk_cap = max_chunks;
  return GMM_OK;
}

const char* gmm_status_string(int status) {
  switch (status) {
    case GMM_OK: return "GMM_OK";
    case GMM_ERR_INVALID_ARG: return "GMM_ERR_INVALID_ARG";
    case GMM_ERR_UNSUPPORTED: return "GMM_ERR_UNSUPPORTED";
    case GMM_ERR_WORKSPACE: return "GMM_ERR_WORKSPACE";
    case GMM_ERR_DEVICE: return "GMM_ERR_DEVICE";
    case GMM_ERR_FILL: return "GMM_ERR_FILL";
    default: return "GMM_UNKNOWN_STATUS";
  }
}

size_t gmm_workspace_bytes(int64_t n, int32_t d, int32_t k, int32_t m) {
  Layout L;
  if (!make_layout(n, d, k, m, &L)) return 0;
  return L.total;
}

static int estep_entry(const float* x, int64_t n, int32_t d, int32_t k, const float* weights,
                       const float* means, const float* vars, double* nk, double* s, double* q,
                       double* loglik, void* ws, size_t ws_bytes, hipStream_t stream,
                       bool refine) {
  int rc = check_shape(n, d, k);
  if (rc != GMM_OK) return rc;
  if (!x || !weights || !means || !vars || !nk || !s || !q || !loglik) return GMM_ERR_INVALID_ARG;
  Layout L;
  if (!make_layout(n, d, k, 0, &L)) return GMM_ERR_UNSUPPORTED;
  L.refine = refine;
  rc = check_ws(L, ws, ws_bytes);
  if (rc != GMM_OK) return rc;
  return estep_dispatch(L, x, weights, means, vars, nk, s, q, loglik, 1, ws, stream);
}

int gmm_estep_accumulate(const float* x, int64_t n, int32_t d, int32_t k, const float* weights,
                         const float* means, const float* vars, double* nk, double* s, double* q,
                         double* loglik, void* ws, size_t ws_bytes, hipStream_t stream) {
  return estep_entry(x, n, d, k, weights, means, vars, nk, s, q, loglik, ws, ws_bytes, stream,
                     true);
}

int gmm_estep_accumulate_screened(const float* x, int64_t n, int32_t d, int32_t k,
                                  const float* weights, const float* means, const float* vars,
                                  double* nk, double* s, double* q, double* loglik, void* ws,
                                  size_t ws_bytes, hipStream_t stream) {
  return estep_entry(x, n, d, k, weights, means, vars, nk, s, q, loglik, ws, ws_bytes, stream,
                     false);
}

int gmm_mstep(const double* nk, const double* s, const double* q, double n_total, int32_t d,
              int32_t k, float var_floor, float* weights, float* means, float* vars,
              hipStream_t stream) {
  if (d < 1 || k < 1) return GMM_ERR_INVALID_ARG;
  if (d > GMM_MAX_D || k > GMM_MAX_K) return GMM_ERR_UNSUPPORTED;
  if (!nk || !s || !q || !weights || !means || !vars) return GMM_ERR_INVALID_ARG;
  if (!(n_total > 0.0) || !(var_floor >= 0.0f)) return GMM_ERR_INVALID_ARG;
  const int64_t tot = (int64_t)k * d;
  hipLaunchKernelGGL(k_mstep, dim3((unsigned)cdiv(tot, 256)), dim3(256), 0, stream, nk, s, q,
                     n_total, d, k, (double)var_floor, weights, means, vars);
  return launch_status();
}

static int fit_entry(const float* x, int64_t n, int32_t d, int32_t k, int32_t n_iters,
                     float var_floor, float* weights, float* means, float* vars,
                     double* loglik_hist, void* ws, size_t ws_bytes, hipStream_t stream,
                     bool refine) {
  int rc = check_shape(n, d, k);
  if (rc != GMM_OK) return rc;
  if (n_iters < 0 || !x || !weights || !means || !vars || (n_iters > 0 && !loglik_hist))
    return GMM_ERR_INVALID_ARG;
  if (!(var_floor >= 0.0f)) return GMM_ERR_INVALID_ARG;
  Layout L;
  if (!make_layout(n, d, k, 0, &L)) return GMM_ERR_UNSUPPORTED;
  L.refine = refine;
  rc = check_ws(L, ws, ws_bytes);
  if (rc != GMM_OK) return rc;
  double* fnk = at<double>(ws, L.off_fit_nk);
  double* fs = at<double>(ws, L.off_fit_s);
  double* fq = at<double>(ws, L.off_fit_q);
  const int64_t kd = (int64_t)k * d;
  for (int t = 0; t < n_iters; ++t) {
    hipLaunchKernelGGL(k_zero, dim3((unsigned)cdiv(k, 256)), dim3(256), 0, stream, fnk,
                       (int64_t)k);
    hipLaunchKernelGGL(k_zero, dim3((unsigned)cdiv(kd, 256)), dim3(256), 0, stream, fs, kd);
    hipLaunchKernelGGL(k_zero, dim3((unsigned)cdiv(kd, 256)), dim3(256), 0, stream, fq, kd);
    rc = estep_dispatch(L, x, weights, means, vars, fnk, fs, fq, loglik_hist + t, 0, ws, stream);
    if (rc != GMM_OK) return rc;
    hipLaunchKernelGGL(k_mstep, dim3((unsigned)cdiv(kd, 256)), dim3(256), 0, stream, fnk, fs, fq,
                       (double)n, d, k, (double)var_floor, weights, means, vars);
    rc = launch_status();
    if (rc != GMM_OK) return rc;
  }
  return GMM_OK;
}

int gmm_fit(const float* x, int64_t n, int32_t d, int32_t k, int32_t n_iters, float var_floor,
            float* weights, float* means, float* vars, double* loglik_hist, void* ws,
            size_t ws_bytes, hipStream_t stream) {
  return fit_entry(x, n, d, k, n_iters, var_floor, weights, means, vars, loglik_hist, ws,
                   ws_bytes, stream, true);
}

int gmm_fit_screened(const float* x, int64_t n, int32_t d, int32_t k, int32_t n_iters,
                     float var_floor, float* weights, float* means, float* vars,
                     double* loglik_hist, void* ws, size_t ws_bytes, hipStream_t stream) {
  return fit_entry(x, n, d, k, n_iters, var_floor, weights, means, vars, loglik_hist, ws,
                   ws_bytes, stream, false);
}

int gmm_estep_accumulate_iso(const float* x, int64_t n, int32_t d, int32_t k,
                             const float* weights, const float* means, const float* vars,
                             double* nk, double* s, double* q, double* loglik, void* ws,
                             size_t ws_bytes, hipStream_t stream) {
  int rc = check_shape(n, d, k);
  if (rc != GMM_OK) return rc;
  if (!x || !weights || !means || !vars || !nk || !s || !q || !loglik) return GMM_ERR_INVALID_ARG;
  Layout L;
  if (!make_layout(n, d, k, 0, &L)) return GMM_ERR_UNSUPPORTED;
  L.iso = true;
  rc = check_ws(L, ws, ws_bytes);
  if (rc != GMM_OK) return rc;
  float* vfull = at<float>(ws, L.off_iso_var);
  double* qd = at<double>(ws, L.off_fit_q);
  const int64_t kd = (int64_t)k * d;
  hipLaunchKernelGGL(k_iso_expand, dim3((unsigned)cdiv(kd, 256)), dim3(256), 0, stream, vars, d,
                     k, vfull);
  hipLaunchKernelGGL(k_zero, dim3((unsigned)cdiv(kd, 256)), dim3(256), 0, stream, qd, kd);
  rc = estep_dispatch(L, x, weights, means, vfull, nk, s, qd, loglik, 1, ws, stream);
  if (rc != GMM_OK) return rc;
  hipLaunchKernelGGL(k_iso_qsum, dim3((unsigned)cdiv(k, 256)), dim3(256), 0, stream, qd, d, k, q);
  return launch_status();
}

int gmm_mstep_iso(const double* nk, const double* s, const double* q, double n_total, int32_t d,
                  int32_t k, float var_floor, float* weights, float* means, float* vars,
                  hipStream_t stream) {
  if (d < 1 || k < 1) return GMM_ERR_INVALID_ARG;
  if (d > GMM_MAX_D || k > GMM_MAX_K) return GMM_ERR_UNSUPPORTED;
  if (!nk || !s || !q || !weights || !means || !vars) return GMM_ERR_INVALID_ARG;
  if (!(n_total > 0.0) || !(var_floor >= 0.0f)) return GMM_ERR_INVALID_ARG;
  hipLaunchKernelGGL(k_mstep_iso, dim3((unsigned)cdiv(k, 256)), dim3(256), 0, stream, nk, s, q,
                     n_total, d, k, (double)var_floor, weights, means, vars);
  return launch_status();
}

int gmm_fit_iso(const float* x, int64_t n, int32_t d, int32_t k, int32_t n_iters, float var_floor,
                float* weights, float* means, float* vars, double* loglik_hist, void* ws,
                size_t ws_bytes, hipStream_t stream) {
  int rc = check_shape(n, d, k);
  if (rc != GMM_OK) return rc;
  if (n_iters < 0 || !x || !weights || !means || !vars || (n_iters > 0 && !loglik_hist))
    return GMM_ERR_INVALID_ARG;
  if (!(var_floor >= 0.0f)) return GMM_ERR_INVALID_ARG;
  Layout L;
  if (!make_layout(n, d, k, 0, &L)) return GMM_ERR_UNSUPPORTED;
  L.iso = true;
  rc = check_ws(L, ws, ws_bytes);
  if (rc != GMM_OK) return rc;
  double* fnk = at<double>(ws, L.off_fit_nk);
  double* fs = at<double>(ws, L.off_fit_s);
  double* fqd = at<double>(ws, L.off_fit_q);
  double* fq = at<double>(ws, L.off_iso_q);
  float* vfull = at<float>(ws, L.off_iso_var);
  const int64_t kd = (int64_t)k * d;
  for (int t = 0; t < n_iters; ++t) {
    hipLaunchKernelGGL(k_zero, dim3((unsigned)cdiv(k, 256)), dim3(256), 0, stream, fnk,
                       (int64_t)k);
    hipLaunchKernelGGL(k_zero, dim3((unsigned)cdiv(k, 256)), dim3(256), 0, stream, fq,
                       (int64_t)k);
    hipLaunchKernelGGL(k_zero, dim3((unsigned)cdiv(kd, 256)), dim3(256), 0, stream, fs, kd);
    hipLaunchKernelGGL(k_zero, dim3((unsigned)cdiv(kd, 256)), dim3(256), 0, stream, fqd, kd);
    hipLaunchKernelGGL(k_iso_expand, dim3((unsigned)cdiv(kd, 256)), dim3(256), 0, stream, vars,
                       d, k, vfull);
    rc = estep_dispatch(L, x, weights, means, vfull, fnk, fs, fqd, loglik_hist + t, 0, ws,
                        stream);
    if (rc != GMM_OK) return rc;
    hipLaunchKernelGGL(k_iso_qsum, dim3((unsigned)cdiv(k, 256)), dim3(256), 0, stream, fqd, d, k,
                       fq);
    hipLaunchKernelGGL(k_mstep_iso, dim3((unsigned)cdiv(k, 256)), dim3(256), 0, stream, fnk, fs,
                       fq, (double)n, d, k, (double)var_floor, weights, means, vars);
    rc = launch_status();
    if (rc != GMM_OK) return rc;
  }
  return GMM_OK;
}

int gmm_estep_accumulate_streamed(const float* x_host, int64_t n, int32_t d, int32_t k,
                                  const float* weights, const float* means, const float* vars,
                                  double* nk, double* s, double* q, double* loglik,
                                  int64_t chunk_rows, float* staging, void* ws, size_t ws_bytes,
                                  hipStream_t stream, hipStream_t copy_stream) {
  int rc = check_shape(n, d, k);
  if (rc != GMM_OK) return rc;
  if (!x_host || !weights || !means || !vars || !nk || !s || !q || !loglik || !staging ||
      chunk_rows < 1)
    return GMM_ERR_INVALID_ARG;
  const int64_t rows = chunk_rows < n ? chunk_rows : n;
  Layout L;
  if (!make_layout(rows, d, k, 0, &L)) return GMM_ERR_UNSUPPORTED;
  rc = check_ws(L, ws, ws_bytes);
  if (rc != GMM_OK) return rc;
  StreamEvents sev;
  if (!sev.make()) return GMM_ERR_DEVICE;
  // the staging buffers may still be read by work enqueued on `stream` before
  // this call: the first uploads wait for it
  if (hipEventRecord(sev.start(), stream) != hipSuccess ||
      hipStreamWaitEvent(copy_stream, sev.start(), 0) != hipSuccess)
    return GMM_ERR_DEVICE;
  const int64_t nchunks = (n + rows - 1) / rows;
  for (int64_t c = 0; c < nchunks; ++c) {
    const int b = (int)(c & 1);
    const int64_t r0 = c * rows, nr = n - r0 < rows ? n - r0 : rows;
    float* buf = staging + (size_t)b * rows * d;
    // upload chunk c once the E-step of chunk c - 2 has read this buffer
    if (c >= 2 && hipStreamWaitEvent(copy_stream, sev.done(b), 0) != hipSuccess)
      return GMM_ERR_DEVICE;
    if (hipMemcpyAsync(buf, x_host + r0 * d, (size_t)nr * d * sizeof(float),
                       hipMemcpyHostToDevice, copy_stream) != hipSuccess ||
        hipEventRecord(sev.up(b), copy_stream) != hipSuccess ||
        hipStreamWaitEvent(stream, sev.up(b), 0) != hipSuccess)
      return GMM_ERR_DEVICE;
    Layout Lc;
    if (!make_layout(nr, d, k, 0, &Lc)) return GMM_ERR_UNSUPPORTED;
    rc = estep_dispatch(Lc, buf, weights, means, vars, nk, s, q, loglik, 1, ws, stream);
    if (rc != GMM_OK) return rc;
    if (hipEventRecord(sev.done(b), stream) != hipSuccess) return GMM_ERR_DEVICE;
  }
  return GMM_OK;
}

// ---------------------------------------------------------------- out-of-core ring
int gmm_fill_pageable(void* user, int64_t row0, int64_t rows, int32_t d, float* dst) {
  if (!user || !dst || rows < 0 || row0 < 0 || d < 1) return 1;
  const char* src = reinterpret_cast<const char*>(user) + (size_t)row0 * d * sizeof(float);
  char* out = reinterpret_cast<char*>(dst);
  const size_t bytes = (size_t)rows * d * sizeof(float);
  // one memcpy per thread over disjoint byte ranges; a single thread below 64 MiB
  constexpr size_t kPiece = (size_t)64 << 20;
  const size_t nt = bytes / kPiece < 8 ? (bytes / kPiece > 1 ? bytes / kPiece : 1) : 8;
  if (nt == 1) {
    memcpy(out, src, bytes);
    return 0;
  }
  const size_t per = (bytes + nt - 1) / nt;
  auto piece = [=](size_t t) {
    const size_t b0 = t * per, b1 = b0 + per < bytes ? b0 + per : bytes;
    if (b0 < b1) memcpy(out + b0, src + b0, b1 - b0);
  };
  std::vector<std::thread> th;
  size_t t = 1;
  for (; t < nt; ++t) {
    try {
      th.emplace_back(piece, t);
    } catch (...) {
      break;                    // no more threads: the calling thread copies the rest
    }
  }
  for (; t < nt; ++t) piece(t);
  piece(0);
  for (std::thread& w : th) w.join();
  return 0;
}

int gmm_estep_accumulate_ring(gmm_fill_fn fill, void* user, int64_t n, int32_t d, int32_t k,
                              const float* weights, const float* means, const float* vars,
                              double* nk, double* s, double* q, double* loglik,
                              int64_t chunk_rows, float* ring, int32_t ring_slots,
                              float* staging, void* ws, size_t ws_bytes, hipStream_t stream,
                              hipStream_t copy_stream) {
  int rc = check_shape(n, d, k);
  if (rc != GMM_OK) return rc;
  if (!fill || !weights || !means || !vars || !nk || !s || !q || !loglik || !ring || !staging ||
      chunk_rows < 1 || ring_slots < 2)
    return GMM_ERR_INVALID_ARG;
  const int64_t rows = chunk_rows < n ? chunk_rows : n;
  Layout L;
  if (!make_layout(rows, d, k, 0, &L)) return GMM_ERR_UNSUPPORTED;
  rc = check_ws(L, ws, ws_bytes);
  if (rc != GMM_OK) return rc;
  StreamEvents sev;
  if (!sev.make()) return GMM_ERR_DEVICE;
  // one event per ring slot: recorded after the slot's upload, waited for on
  // the host before the slot is filled again
  struct SlotEvents {
    std::vector<hipEvent_t> ev;
    ~SlotEvents() {
      for (hipEvent_t e : ev)
        if (e) (void)hipEventDestroy(e);
    }
  } slot;
  slot.ev.assign((size_t)ring_slots, nullptr);
  for (hipEvent_t& e : slot.ev)
    if (hipEventCreateWithFlags(&e, hipEventDisableTiming) != hipSuccess) return GMM_ERR_DEVICE;
  // earlier uploads on copy_stream may still read the ring (the host waits for
  // them), and earlier work on `stream` the staging buffer (the uploads wait)
  if (hipEventRecord(slot.ev[0], copy_stream) != hipSuccess ||
      hipEventSynchronize(slot.ev[0]) != hipSuccess ||
      hipEventRecord(sev.start(), stream) != hipSuccess ||
      hipStreamWaitEvent(copy_stream, sev.start(), 0) != hipSuccess)
    return GMM_ERR_DEVICE;
  const int64_t nchunks = (n + rows - 1) / rows;
  const size_t slot_elems = (size_t)rows * d;
  for (int64_t c = 0; c < nchunks; ++c) {
    const int b = (int)(c & 1);
    const int sl = (int)(c % ring_slots);
    const int64_t r0 = c * rows, nr = n - r0 < rows ? n - r0 : rows;
    float* src = ring + (size_t)sl * slot_elems;
    float* buf = staging + (size_t)b * slot_elems;
    if (c >= ring_slots && hipEventSynchronize(slot.ev[sl]) != hipSuccess) return GMM_ERR_DEVICE;
    if (fill(user, r0, nr, d, src) != 0) return GMM_ERR_FILL;
    // upload chunk c once the E-step of chunk c - 2 has read this half of staging
    if (c >= 2 && hipStreamWaitEvent(copy_stream, sev.done(b), 0) != hipSuccess)
      return GMM_ERR_DEVICE;
    if (hipMemcpyAsync(buf, src, (size_t)nr * d * sizeof(float), hipMemcpyHostToDevice,
                       copy_stream) != hipSuccess ||
        hipEventRecord(slot.ev[sl], copy_stream) != hipSuccess ||
        hipEventRecord(sev.up(b), copy_stream) != hipSuccess ||
        hipStreamWaitEvent(stream, sev.up(b), 0) != hipSuccess)
      return GMM_ERR_DEVICE;
    Layout Lc;
    if (!make_layout(nr, d, k, 0, &Lc)) return GMM_ERR_UNSUPPORTED;
    rc = estep_dispatch(Lc, buf, weights, means, vars, nk, s, q, loglik, 1, ws, stream);
    if (rc != GMM_OK) return rc;
    if (hipEventRecord(sev.done(b), stream) != hipSuccess) return GMM_ERR_DEVICE;
  }
  return GMM_OK;
}

int gmm_kmeans(const float* x, int64_t n, int32_t d, int32_t k, int32_t n_iters, float var_floor,
               float* weights, float* means, float* vars, int32_t* assign, void* ws,
               size_t ws_bytes, hipStream_t stream) {
  int rc = check_shape(n, d, k);
  if (rc != GMM_OK) return rc;
  if (n_iters < 0 || !x || !weights || !means || !vars || !assign || !(var_floor >= 0.0f))
    return GMM_ERR_INVALID_ARG;
  Layout L;
  if (!make_layout(n, d, k, 1, &L)) return GMM_ERR_UNSUPPORTED;
  rc = check_ws(L, ws, ws_bytes);
  if (rc != GMM_OK) return rc;
  switch (L.D64) {
#define GMM_CASE(D) \
  case D: return kmeans_impl<D>(L, x, n_iters, var_floor, weights, means, vars, assign, ws, stream);
    GMM_FOR_EACH_D64(GMM_CASE)
#undef GMM_CASE
    default: return GMM_ERR_UNSUPPORTED;
  }
}

size_t gmm_kmeanspp_workspace_bytes(int64_t n) {
  if (n < 1) return 0;
  const int64_t nblk = cdiv(n, kKppBlock);
  return align256((size_t)n * sizeof(double)) + align256((size_t)nblk * sizeof(double));
}

int gmm_kmeanspp(const float* x, int64_t n, int32_t d, int32_t k, const double* u, int64_t* idx,
                 float* centers, void* ws, size_t ws_bytes, hipStream_t stream) {
  int rc = check_shape(n, d, k);
  if (rc != GMM_OK) return rc;
  if (!x || !u || !idx || !centers) return GMM_ERR_INVALID_ARG;
  if (ws == nullptr || (reinterpret_cast<uintptr_t>(ws) & 255) != 0 ||
      ws_bytes < gmm_kmeanspp_workspace_bytes(n))
    return GMM_ERR_WORKSPACE;
  const int64_t nblk = cdiv(n, kKppBlock);
  const int vec4 = (d & 3) == 0 && (reinterpret_cast<uintptr_t>(x) & 15) == 0;
  double* dist = static_cast<double*>(ws);
  double* bsum = at<double>(ws, align256((size_t)n * sizeof(double)));
  hipLaunchKernelGGL(k_kpp_select, dim3(1), dim3(256), 0, stream, x, n, d, u, 0, dist, bsum,
                     nblk, idx, centers);
  for (int t = 1; t < k; ++t) {
    hipLaunchKernelGGL(k_kpp_update, dim3((unsigned)nblk), dim3(256), 0, stream, x, n, d, vec4,
                       idx, t, t == 1 ? 1 : 0, dist, bsum);
    hipLaunchKernelGGL(k_kpp_select, dim3(1), dim3(256), 0, stream, x, n, d, u, t, dist, bsum,
                       nblk, idx, centers);
  }
  return launch_status();
}

int gmm_assign_topk(const float* x, int64_t n, int32_t d, int32_t k, const float* weights,
                    const float* means, const float* vars, int32_t m, float tau, int32_t* idx,
                    float* resp, void* ws, size_t ws_bytes, hipStream_t stream) {
  int rc = check_shape(n, d, k);
  if (rc != GMM_OK) return rc;
  if (m > GMM_MAX_M) return GMM_ERR_UNSUPPORTED;
  if (!x || !weights || !means || !vars || !idx || !resp) return GMM_ERR_INVALID_ARG;
  if (m < 1 || m > k || !(tau >= 0.0f && tau < 1.0f)) return GMM_ERR_INVALID_ARG;
  Layout L;
  if (!make_layout(n, d, k, m, &L)) return GMM_ERR_UNSUPPORTED;
  rc = check_ws(L, ws, ws_bytes);
  if (rc != GMM_OK) return rc;
  switch (L.D64) {
#define GMM_CASE(D) \
  case D: return assign_impl<D>(L, x, weights, means, vars, m, tau, idx, resp, ws, stream);
    GMM_FOR_EACH_D64(GMM_CASE)
#undef GMM_CASE
    default: return GMM_ERR_UNSUPPORTED;
  }
}

}  // extern "C"
