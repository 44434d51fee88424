// Device helpers shared by the LapSum kernels (gfx950, wave64).
//
// Notation follows the paper: scores r, temperature t = -alpha > 0, threshold
// b with LapSum(b) = sum_i sigma((r_i - b)/t) = k (Eq. (1), Suppl. A).  After
// a descending sort s_1 >= ... >= s_n the node curve
//     N_i = LapSum(s_i) = i - P_i / 2 + E_i / 2,
//     P_i = sum_{j <= i} e^{-(s_j - s_i)/t},   E_i = sum_{j > i} e^{-(s_i - s_j)/t}
// is non-decreasing in i (the three-group split of Suppl. A), and inside the
// interval [s_{m+1}, s_m] holding b the budget equation has two exponentials
// and a closed-form root.
//
// Both sums are scanned in "shift-carrying" form: a group of sorted scores is
// summarised by (anchor, sum) where every term is an exponential of a
// non-positive exponent relative to the anchor, so nothing overflows and no
// sum is ever formed by subtracting two large numbers.
//   Pre (anchor u = the group's smallest score):  S = sum e^{-(r - u)/t}
//   Suf (anchor v = the group's largest score):   T = sum e^{-(v - r)/t}
// Combining an earlier (larger) group A with a later group B:
//   Pre(A then B) = (u_B, S_B + e^{-(u_A - u_B)/t} S_A)
//   Suf(A then B) = (v_A, T_A + e^{-(v_A - v_B)/t} T_B)
// This is the associative form of the affine recurrence x_i = w_i x_{i-1} + 1
// of Suppl. A (the 2x2 matrix [[w,1],[0,1]]), with each weight formed from
// the anchors directly rather than as a product of per-step weights.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lapsum {

constexpr int kWave = 64;
constexpr double kLog2e = 1.4426950408889634074;

// ---------------------------------------------------------------- keys ----
// uint32 key whose ascending order is the descending order of the float.
// Ascending map: non-negative floats get the sign bit set, negative floats
// are inverted; the descending key is the complement of that.
__device__ __forceinline__ uint32_t desc_key(float f) {
  uint32_t u = __float_as_uint(f);
  uint32_t asc = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return ~asc;
}

__device__ __forceinline__ float key_float(uint32_t dk) {
  uint32_t asc = ~dk;
  uint32_t u = (asc & 0x80000000u) ? (asc & 0x7fffffffu) : ~asc;
  return __uint_as_float(u);
}

// ----------------------------------------------------------- exponentials --
// 2^x on the hardware transcendental unit (results below the normal range
// flush to zero, which only drops terms under 1e-38).
__device__ __forceinline__ float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

// Streams touched once per call (the scores in the partition, p and grad_r
// written by the band passes) use non-temporal accesses, so that they
// neither evict nor leave behind dirty lines that the next pass would have
// to write back.
typedef float stream_v4f __attribute__((ext_vector_type(4)));
__device__ __forceinline__ float4 load_stream4(const float* p) {
  const stream_v4f v = __builtin_nontemporal_load(reinterpret_cast<const stream_v4f*>(p));
  return make_float4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ void store_stream4(float* p, float4 x) {
  const stream_v4f v = {x.x, x.y, x.z, x.w};
  __builtin_nontemporal_store(v, reinterpret_cast<stream_v4f*>(p));
}

// e^{-d/t} for d >= 0 with the exponent formed in float64 (d may be the
// difference of two float32 scores of very different size) and the
// exponential in float32; c2 = log2(e)/t.  For per-score terms summed in
// float64: each term carries one float32 rounding, never a product of them.
__device__ __forceinline__ double wexp_f32(double d, double c2) {
  return static_cast<double>(exp2_fast(static_cast<float>(-d * c2)));
}

// Laplace(0, t) draw number s of the bracket's default kernel noise (the
// sample takes it when the caller passes no table).  A counter-based
// generator, so the same (seed, s) always gives the same draw and no state
// is kept: z is the (s+1)-th output of SplitMix64 started at `seed` (Steele,
// Lea and Flood, "Fast splittable pseudorandom number generators", 2014),
// its top 52 bits m give u = (2m + 1) 2^-53, strictly inside (0, 1) and
// never 1/2 (1 - u is exact), and the Laplace inverse CDF gives
// t ln(2u) for u < 1/2 and -t ln(2(1 - u)) above, in float64, rounded to
// float32.
__device__ __forceinline__ float counter_laplace(uint64_t seed, int64_t s, double t) {
  uint64_t z = seed + static_cast<uint64_t>(s + 1) * 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  z ^= z >> 31;
  const uint64_t m = z >> 12;
  const double u = static_cast<double>(2 * m + 1) * 0x1p-53;
  const double e = u < 0.5 ? t * log(2.0 * u) : -t * log(2.0 * (1.0 - u));
  return static_cast<float>(e);
}

// e^{-d/t} in float64, for scan combines and the root.
__device__ __forceinline__ double wexp_f64(double d, double inv_t) { return exp(-d * inv_t); }

// ----------------------------------------------------------- pair algebra --
struct Pre {   // sum_j e^{-(r_j - u)/t}; S == 0 means "no scores"
  float u;
  double S;
};
struct Suf {   // sum_j e^{-(v - r_j)/t}; T == 0 means "no scores"
  float v;
  double T;
};

__device__ __forceinline__ Pre pre_empty() { return Pre{0.0f, 0.0}; }
__device__ __forceinline__ Suf suf_empty() { return Suf{0.0f, 0.0}; }

// a is the earlier group (larger scores), b the later one.
__device__ __forceinline__ Pre pre_combine(Pre a, Pre b, double inv_t) {
  if (a.S == 0.0) return b;
  if (b.S == 0.0) return a;
  double w = wexp_f64(static_cast<double>(a.u) - static_cast<double>(b.u), inv_t);
  return Pre{b.u, b.S + w * a.S};
}

__device__ __forceinline__ Suf suf_combine(Suf a, Suf b, double inv_t) {
  if (a.T == 0.0) return b;
  if (b.T == 0.0) return a;
  double w = wexp_f64(static_cast<double>(a.v) - static_cast<double>(b.v), inv_t);
  return Suf{a.v, a.T + w * b.T};
}

// ------------------------------------------------------------ wave scans ---
__device__ __forceinline__ int lane_id() { return threadIdx.x & (kWave - 1); }

// Cross-lane moves within rows of 16 lanes (DPP): lane l takes the value of
// the lane the control names in its row; a lane whose source lies outside
// the row keeps `id`.  Controls used: row_shr:d = 0x110 + d (source l - d),
// row_shl:d = 0x100 + d (source l + d).  No LDS traffic, unlike a shuffle.
// Every helper below needs the whole wave active.
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t x, uint32_t id) {
  return static_cast<uint32_t>(
      __builtin_amdgcn_update_dpp(static_cast<int>(id), static_cast<int>(x), CTRL, 0xf, 0xf, false));
}
template <int CTRL, typename T>
__device__ __forceinline__ T dpp_move(T x, T id) {
  static_assert(sizeof(T) == 4 || sizeof(T) == 8, "32- or 64-bit values");
  if constexpr (sizeof(T) == 4) {
    return __builtin_bit_cast(T, dpp_u32<CTRL>(__builtin_bit_cast(uint32_t, x),
                                               __builtin_bit_cast(uint32_t, id)));
  } else {
    const uint64_t xb = __builtin_bit_cast(uint64_t, x);
    const uint64_t ib = __builtin_bit_cast(uint64_t, id);
    const uint32_t lo = dpp_u32<CTRL>(static_cast<uint32_t>(xb), static_cast<uint32_t>(ib));
    const uint32_t hi = dpp_u32<CTRL>(static_cast<uint32_t>(xb >> 32), static_cast<uint32_t>(ib >> 32));
    return __builtin_bit_cast(T, (static_cast<uint64_t>(hi) << 32) | lo);
  }
}
template <typename T>
__device__ __forceinline__ T readlane_as(T x, int l) {
  static_assert(sizeof(T) == 4 || sizeof(T) == 8, "32- or 64-bit values");
  if constexpr (sizeof(T) == 4) {
    return __builtin_bit_cast(
        T, static_cast<uint32_t>(__builtin_amdgcn_readlane(__builtin_bit_cast(int, x), l)));
  } else {
    const uint64_t xb = __builtin_bit_cast(uint64_t, x);
    const uint32_t lo = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(xb), l));
    const uint32_t hi = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(xb >> 32), l));
    return __builtin_bit_cast(T, (static_cast<uint64_t>(hi) << 32) | lo);
  }
}

// Reduction over the wave in a fixed order, the result in every lane:
// partial results inside each row of 16 lanes, then the four rows as
// (r0 op r1) op (r2 op r3).
template <typename T, typename Op>
__device__ __forceinline__ T wave_reduce(T v, T id, Op op) {
  v = op(v, dpp_move<0x111>(v, id));
  v = op(v, dpp_move<0x112>(v, id));
  v = op(v, dpp_move<0x114>(v, id));
  v = op(v, dpp_move<0x118>(v, id));
  return op(op(readlane_as(v, 15), readlane_as(v, 31)), op(readlane_as(v, 47), readlane_as(v, 63)));
}
template <typename T>
__device__ __forceinline__ T wave_sum(T v) {
  return wave_reduce(v, T(0), [](T a, T b) { return a + b; });
}
template <typename T>
__device__ __forceinline__ T wave_max(T v, T id) {
  return wave_reduce(v, id, [](T a, T b) { return a > b ? a : b; });
}
template <typename T>
__device__ __forceinline__ T wave_min(T v, T id) {
  return wave_reduce(v, id, [](T a, T b) { return a < b ? a : b; });
}
template <typename T>
__device__ __forceinline__ T wave_or(T v) {
  return wave_reduce(v, T(0), [](T a, T b) { return a | b; });
}
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t x) { return wave_max(x, 0u); }
__device__ __forceinline__ uint32_t wave_min_u32(uint32_t x) { return wave_min(x, 0xffffffffu); }

// Inclusive sum over lanes 0 .. l.
template <typename T>
__device__ __forceinline__ T wave_incl_add(T x) {
  x += dpp_move<0x111>(x, T(0));
  x += dpp_move<0x112>(x, T(0));
  x += dpp_move<0x114>(x, T(0));
  x += dpp_move<0x118>(x, T(0));
  const T r0 = readlane_as(x, 15), r1 = readlane_as(x, 31), r2 = readlane_as(x, 47);
  const int row = lane_id() >> 4;
  return x + (row == 0 ? T(0) : (row == 1 ? r0 : (row == 2 ? r0 + r1 : r0 + r1 + r2)));
}

// Affine maps x -> A x + B composed along the wave.  Left to right, lane l
// ends with x_l o ... o x_0 (apply lane 0's map first); right to left, with
// x_l o ... o x_63.  Hillis-Steele inside each row of 16, then every row
// takes the composition of the rows before (after) it from lanes read out
// as scalars.
#define LAPSUM_AFFINE_STEP(C)                                                  \
  {                                                                            \
    const double eA = dpp_move<C>(A, 1.0), eB = dpp_move<C>(B, 0.0);           \
    B = fma(A, eB, B);                                                         \
    A *= eA;                                                                   \
  }
__device__ __forceinline__ void wave_affine_up(double& A, double& B) {
  LAPSUM_AFFINE_STEP(0x111)
  LAPSUM_AFFINE_STEP(0x112)
  LAPSUM_AFFINE_STEP(0x114)
  LAPSUM_AFFINE_STEP(0x118)
  const double a0 = readlane_as(A, 15), b0 = readlane_as(B, 15);
  const double a1 = readlane_as(A, 31), b1 = readlane_as(B, 31);
  const double a2 = readlane_as(A, 47), b2 = readlane_as(B, 47);
  const double e2A = a1 * a0, e2B = fma(a1, b0, b1);
  const double e3A = a2 * e2A, e3B = fma(a2, e2B, b2);
  const int row = lane_id() >> 4;
  const double eA = row == 0 ? 1.0 : (row == 1 ? a0 : (row == 2 ? e2A : e3A));
  const double eB = row == 0 ? 0.0 : (row == 1 ? b0 : (row == 2 ? e2B : e3B));
  B = fma(A, eB, B);
  A *= eA;
}
__device__ __forceinline__ void wave_affine_down(double& A, double& B) {
  LAPSUM_AFFINE_STEP(0x101)
  LAPSUM_AFFINE_STEP(0x102)
  LAPSUM_AFFINE_STEP(0x104)
  LAPSUM_AFFINE_STEP(0x108)
  const double a1 = readlane_as(A, 16), b1 = readlane_as(B, 16);
  const double a2 = readlane_as(A, 32), b2 = readlane_as(B, 32);
  const double a3 = readlane_as(A, 48), b3 = readlane_as(B, 48);
  const double e1A = a2 * a3, e1B = fma(a2, b3, b2);
  const double e0A = a1 * e1A, e0B = fma(a1, e1B, b1);
  const int row = lane_id() >> 4;
  const double eA = row == 3 ? 1.0 : (row == 2 ? a3 : (row == 1 ? e1A : e0A));
  const double eB = row == 3 ? 0.0 : (row == 2 ? b3 : (row == 1 ? e1B : e0B));
  B = fma(A, eB, B);
  A *= eA;
}
#undef LAPSUM_AFFINE_STEP

// Scratch for the block-level scans and the crossing search.
template <int WAVES>
struct ScanSmem {
  double A[WAVES], B[WAVES];   // per-wave affine maps
  float au[WAVES];             // per-wave anchor of the last (first) non-empty group
  int ah[WAVES];
  double A2[WAVES], B2[WAVES];   // the suffix scan's, when both run together
  float au2[WAVES];
  int ah2[WAVES];
  int cnt[WAVES];
  double b;
  double P[64];   // crossing refinement (at most 64 items per thread)
  double Q[64];
  float sv[64];
  Pre pre_c;
  Suf suf_c;
  int cnt_c;
};

// Block scans of the pairs.  The combine of two prefix pairs is the affine
// map P -> w P + S with w = e^{-(u_earlier - u_later)/t}, and likewise for
// suffix pairs, so a scan over the threads' groups is an affine scan once
// every group knows the anchor of the nearest non-empty group before it
// (after it, for suffixes): each thread forms its one exponential, and the
// scan itself multiplies and adds.  Weights never exceed 1 (anchors are
// non-increasing along the order), so products only underflow, when the
// carried terms are negligible.

// Exclusive block scans of the prefix pairs xp in thread order, seeded
// with pc (the groups before the block), and of the suffix pairs xs from
// the right, seeded with sc (the groups after it), run together on three
// barriers.  *pre_in / *suf_in get this thread's exclusive prefix / suffix,
// *pre_total = pc (+) all and *suf_total = all (+) sc.  Empty groups (S == 0,
// T == 0) are skipped.  The two exponentials and the two wave scans of a
// thread are independent of each other.
template <int WAVES>
__device__ void block_excl_pre_suf(Pre xp, Pre pc, Suf xs, Suf sc, double inv_t,
                                   ScanSmem<WAVES>& sm, Pre* pre_in, Pre* pre_total, Suf* suf_in,
                                   Suf* suf_total) {
  const int lane = lane_id();
  const int wid = threadIdx.x / kWave;
  const bool phas = xp.S != 0.0, shas = xs.T != 0.0;
  const bool pchas = pc.S != 0.0, schas = sc.T != 0.0;
  // 1. anchors of the nearest non-empty groups before (prefix) and after
  //    (suffix) each thread
  const uint64_t phm = __ballot(phas);
  const uint64_t shm = __ballot(shas);
  const float lu = __shfl(xp.u, phm != 0ull ? 63 - __clzll(phm) : 0, kWave);
  const float fv = __shfl(xs.v, shm != 0ull ? __ffsll(static_cast<long long>(shm)) - 1 : 0, kWave);
  if (lane == 0) {
    sm.ah[wid] = phm != 0ull ? 1 : 0;
    sm.au[wid] = lu;
    sm.ah2[wid] = shm != 0ull ? 1 : 0;
    sm.au2[wid] = fv;
  }
  const uint64_t before = phm & ((1ull << lane) - 1ull);
  const float bu = __shfl(xp.u, before ? 63 - __clzll(before) : 0, kWave);
  const uint64_t after = lane == kWave - 1 ? 0ull : shm & (~0ull << (lane + 1));
  const float av = __shfl(xs.v, after ? __ffsll(static_cast<long long>(after)) - 1 : 0, kWave);
  __syncthreads();
  int eh = pchas ? 1 : 0;
  float eu = pc.u;
#pragma unroll
  for (int w = 0; w < WAVES; ++w) {
    const int h = sm.ah[w];
    const float a = sm.au[w];
    if (w < wid && h) {
      eh = 1;
      eu = a;
    }
  }
  int fh = schas ? 1 : 0;
  float fv2 = sc.v;
#pragma unroll
  for (int w = WAVES - 1; w >= 0; --w) {
    const int h = sm.ah2[w];
    const float a = sm.au2[w];
    if (w > wid && h) {
      fh = 1;
      fv2 = a;
    }
  }
  const int ph = before != 0ull ? 1 : eh;
  const float pu = before != 0ull ? bu : eu;
  const int nh = after != 0ull ? 1 : fh;
  const float nv = after != 0ull ? av : fv2;
  // 2. P_i = A_i P_{i-1} + B_i and T_i = B_i + A_i T_{i+1}
  double Ap = phas ? (ph ? wexp_f64(static_cast<double>(pu) - static_cast<double>(xp.u), inv_t) : 0.0) : 1.0;
  double Bp = phas ? xp.S : 0.0;
  double As = shas ? (nh ? wexp_f64(static_cast<double>(xs.v) - static_cast<double>(nv), inv_t) : 0.0) : 1.0;
  double Bs = shas ? xs.T : 0.0;
  wave_affine_up(Ap, Bp);
  wave_affine_down(As, Bs);
  if (lane == kWave - 1) {
    sm.A[wid] = Ap;
    sm.B[wid] = Bp;
  }
  if (lane == 0) {
    sm.A2[wid] = As;
    sm.B2[wid] = Bs;
  }
  __syncthreads();
  const double P_in = pchas ? pc.S : 0.0;
  double P0 = P_in;   // P entering this wave
  double Pt = P_in;
  int pth = pchas ? 1 : 0;
  float ptu = pc.u;
#pragma unroll
  for (int w = 0; w < WAVES; ++w) {
    const double Aw = sm.A[w], Bw = sm.B[w];
    if (w < wid) P0 = fma(Aw, P0, Bw);
    Pt = fma(Aw, Pt, Bw);
    if (sm.ah[w]) {
      pth = 1;
      ptu = sm.au[w];
    }
  }
  const double T_in = schas ? sc.T : 0.0;
  double T0 = T_in;   // T following this wave
  double Tt = T_in;
  int sth = schas ? 1 : 0;
  float stv = sc.v;
#pragma unroll
  for (int w = WAVES - 1; w >= 0; --w) {
    const double Aw = sm.A2[w], Bw = sm.B2[w];
    if (w > wid) T0 = fma(Aw, T0, Bw);
    Tt = fma(Aw, Tt, Bw);
    if (sm.ah2[w]) {
      sth = 1;
      stv = sm.au2[w];
    }
  }
  const double Pi = fma(Ap, P0, Bp);
  double Pe = __shfl_up(Pi, 1, kWave);
  if (lane == 0) Pe = P0;
  const double Ti = fma(As, T0, Bs);
  double Te = __shfl_down(Ti, 1, kWave);
  if (lane == kWave - 1) Te = T0;
  *pre_total = pth ? Pre{ptu, Pt} : pre_empty();
  *suf_total = sth ? Suf{stv, Tt} : suf_empty();
  *pre_in = ph ? Pre{pu, Pe} : pre_empty();
  *suf_in = nh ? Suf{nv, Te} : suf_empty();
  __syncthreads();
}

// Number of threads in the block with flag set.
template <int WAVES>
__device__ int block_count(bool flag, ScanSmem<WAVES>& sm) {
  const int wid = threadIdx.x / kWave;
  uint64_t m = __ballot(flag);
  if (lane_id() == 0) sm.cnt[wid] = __popcll(m);
  __syncthreads();
  int c = 0;
#pragma unroll
  for (int w = 0; w < WAVES; ++w) c += sm.cnt[w];
  __syncthreads();
  return c;
}

// ------------------------------------------------------------- the root ----
// For v <= b <= u let the c_up scores above the interval be summarised at u
// (A = sum e^{-(r-u)/t}) and the scores below at v (B = sum e^{-(v-r)/t}).
// Then LapSum(b) = c_up - (A/2) e^{-(u-b)/t} + (B/2) e^{-(b-v)/t}, and with
// y = e^{(u-b)/t}, E = B e^{-(u-v)/t}, c = k - c_up the budget equation is the
// quadratic E y^2 - 2 c y - A = 0 whose positive root is
//     y = (c + D) / E = A / (D - c),   D = sqrt(c^2 + A E).
// The form without cancellation is used for each sign of c, in logarithms
// because E underflows when the interval is many temperatures wide.  A group
// whose sum is zero (no scores, or all saturated) drops out: then
// b = v + t ln(B / (2(k - c_up))) or b = u - t ln(A / (2(c_up - k))).
__device__ inline double gap_root(double k, double t, double c_up, bool has_up, double u,
                                  double lnA, bool has_dn, double v, double lnB) {
  if (!has_up) return v + t * (lnB - log(2.0 * (k - c_up)));
  if (!has_dn) return u - t * (lnA - log(2.0 * (c_up - k)));
  const double g = (u - v) / t;
  const double lnE = lnB - g;
  const double c = k - c_up;
  double lny;
  if (c == 0.0) {
    lny = 0.5 * (lnA - lnE);
  } else {
    const double D = sqrt(c * c + exp(lnA + lnE));   // A E <= n^2, never overflows
    lny = (c > 0.0) ? log(c + D) - lnE : lnA - log(D - c);
  }
  lny = fmin(fmax(lny, 0.0), g);
  return u - t * lny;
}

// ------------------------------------------------------ block-level solve ---
// A block holds a run of sorted scores, thread tid owning the consecutive
// positions tid*ITEMS .. tid*ITEMS+cnt-1 (blocked arrangement, descending).
// ext_pre summarises every score ranked before the block (rank0 of them,
// rank0 counted from 0), ext_suf every score ranked after it.  The block is
// known to hold the crossing, or b lies between the block's first score and
// whatever precedes it.  Returns b (the same value in every thread) and the
// block totals ext_pre (+) block, block (+) ext_suf.
template <int BLOCK, int ITEMS>
__device__ double block_solve(const float (&s)[ITEMS], int cnt, double rank0, Pre ext_pre,
                              Suf ext_suf, double k, double t, ScanSmem<BLOCK / kWave>& sm,
                              Pre* pre_total, Suf* suf_total) {
  static_assert(ITEMS <= 64, "crossing refinement scratch");
  constexpr int WAVES = BLOCK / kWave;
  const int tid = threadIdx.x;
  const double inv_t = 1.0 / t;
  const double c2 = kLog2e / t;

  // 1. this thread's group summaries (direct terms relative to the anchors)
  Pre mine_pre = pre_empty();
  Suf mine_suf = suf_empty();
  double suf_x = 0.0;   // sum over positions after the first
  float lastf = s[0];
#pragma unroll
  for (int i = 0; i < ITEMS; ++i)
    if (i == cnt - 1) lastf = s[i];
  if (cnt > 0) {
    const double last = lastf;
    const double first = s[0];
    double sp = 0.0;
#pragma unroll
    for (int i = 0; i < ITEMS; ++i) {
      if (i < cnt) {
        sp += wexp_f32(static_cast<double>(s[i]) - last, c2);
        if (i > 0) suf_x += wexp_f32(first - static_cast<double>(s[i]), c2);
      }
    }
    mine_pre = Pre{lastf, sp};
    mine_suf = Suf{s[0], 1.0 + suf_x};
  }

  // 2. carries into this thread from both sides
  Pre pre_in;
  Suf suf_in;
  block_excl_pre_suf<WAVES>(mine_pre, ext_pre, mine_suf, ext_suf, inv_t, sm, &pre_in, pre_total,
                            &suf_in, suf_total);

  // 3. node value at this thread's first position
  bool below_k = false;
  if (cnt > 0) {
    const double first = s[0];
    double P0 = 1.0;
    if (pre_in.S != 0.0) P0 += wexp_f64(static_cast<double>(pre_in.u) - first, inv_t) * pre_in.S;
    double E0 = suf_x;
    if (suf_in.T != 0.0) E0 += wexp_f64(first - static_cast<double>(suf_in.v), inv_t) * suf_in.T;
    const double N0 = rank0 + static_cast<double>(tid) * ITEMS + 1.0 - 0.5 * P0 + 0.5 * E0;
    below_k = (N0 <= k);
  }
  const int nthr = block_count<WAVES>(below_k, sm);

  // 4. the run holding the crossing is refined position by position: its
  //    owner publishes the scores and carries, then one thread per position
  //    forms P_i and E_i directly (independent terms, no serial chain)
  if (nthr == 0) {
    if (tid == 0) {
      // b lies above every score of the block
      Suf all = *suf_total;
      sm.b = gap_root(k, t, rank0, ext_pre.S != 0.0, ext_pre.u, log(ext_pre.S > 0 ? ext_pre.S : 1.0),
                      true, all.v, log(all.T));
    }
    __syncthreads();
  } else {
    const int owner = nthr - 1;
    if (tid == owner) {
#pragma unroll
      for (int i = 0; i < ITEMS; ++i)
        if (i < cnt) sm.sv[i] = s[i];
      sm.pre_c = pre_in;
      sm.suf_c = suf_in;
      sm.cnt_c = cnt;
    }
    __syncthreads();
    const int oc = sm.cnt_c;
    const Pre pc = sm.pre_c;
    const Suf sc = sm.suf_c;
    const double base = rank0 + static_cast<double>(owner) * ITEMS;
    bool le = false;
    if (tid < oc) {
      const double si = sm.sv[tid];
      double P = 1.0, E = 0.0;
      if (pc.S != 0.0) P += wexp_f64(static_cast<double>(pc.u) - si, inv_t) * pc.S;
      if (sc.T != 0.0) E += wexp_f64(si - static_cast<double>(sc.v), inv_t) * sc.T;
      // the run's own terms are per-score terms like those of the group
      // summaries (float32 exponentials of float64 differences), unrolled
      // over the run's capacity so that they are all independent (runs of
      // 32 keep the loop: their kernels are short of registers already)
      double Pt = 0.0, Et = 0.0;
      if constexpr (ITEMS <= 16) {
#pragma unroll
        for (int j = 0; j < ITEMS; ++j) {
          if (j < oc) {
            const double sj = sm.sv[j];
            if (j < tid) Pt += wexp_f32(sj - si, c2);
            else if (j > tid) Et += wexp_f32(si - sj, c2);
          }
        }
      } else {
        for (int j = 0; j < oc; ++j) {
          const double sj = sm.sv[j];
          if (j < tid) Pt += wexp_f32(sj - si, c2);
          else if (j > tid) Et += wexp_f32(si - sj, c2);
        }
      }
      P += Pt;
      E += Et;
      sm.P[tid] = P;
      sm.Q[tid] = 1.0 + E;
      le = (base + static_cast<double>(tid) + 1.0 - 0.5 * P + 0.5 * E) <= k;
    }
    int m = block_count<WAVES>(le, sm);   // node values are non-decreasing
    if (m == 0) m = 1;                    // the first position was found at or below k
    if (tid < 2) {
      // the logarithms of the gap's two sums side by side (lanes 0 and 1);
      // without a lower side gap_root does not use the second
      const bool has_dn = m < oc || sc.T != 0.0;
      const double arg = tid == 0 ? sm.P[m - 1] : (m < oc ? sm.Q[m] : (has_dn ? sc.T : 1.0));
      const double lg = log(arg);
      const double lnB = __shfl(lg, 1, kWave);
      if (tid == 0) {
        const double c_up = base + m;
        const double u = sm.sv[m - 1];
        sm.b = (m < oc) ? gap_root(k, t, c_up, true, u, lg, true, sm.sv[m], lnB)
                        : gap_root(k, t, c_up, true, u, lg, has_dn, sc.v, lnB);
      }
    }
    __syncthreads();
  }
  const double b = sm.b;
  __syncthreads();
  return b;
}

// ---------------------------------------------------------------- emit -----
// p = sigma((r - b)/t) with the difference taken in float64 (b is float64)
// and the exponential in float32.
__device__ __forceinline__ float laplace_p(float r, double b, double inv_t) {
  const float u = static_cast<float>((static_cast<double>(r) - b) * inv_t);
  // beyond these the float32 result is exactly 0 or 1 anyway; stating it
  // makes the band bounds of a bracket exact by construction
  if (u < -104.0f) return 0.0f;
  if (u > 17.0f) return 1.0f;
  const float e = exp2_fast(-fabsf(u) * static_cast<float>(kLog2e));
  return (u <= 0.0f) ? 0.5f * e : 1.0f - 0.5f * e;
}

// u = (r - b)/t recovered from p = sigma(u) by inverting Eq. (3): with
// s = min(p, 1 - p) = e^{-|u|}/2, |u| = -ln(2s), and u <= 0 exactly where
// p <= 1/2.  Called only where s > 0.
__device__ __forceinline__ float laplace_u_from_p(float p, float s) {
  const float a = logf(2.0f * s);
  return p > 0.5f ? -a : a;
}

}  // namespace lapsum
