// Threshold solve on the middle set M of a bracket without sorting all of
// M (the scan, lookup and closed-form root of Suppl. A / Suppl. B, applied
// where the root is).
//
// M is cut into 2048 buckets of consecutive order-preserving keys (bucket
// d = (key - key(max M)) >> shift, so bucket 0 holds the largest scores).
// Bucket d covers the score interval [u_d, v_d] (its lowest and highest
// possible float, clamped to the range of M) and is summarised by its count
// and the two sums
//     D_d = sum_{r in d} e^{-(r - u_d)/t}    (a prefix pair anchored at u_d)
//     U_d = sum_{r in d} e^{-(v_d - r)/t}    (a suffix pair anchored at v_d).
// The shift-carrying scans over the buckets, seeded with the bracket tails,
// give LapSum at every bucket's upper edge,
//     LapSum(v_d) = n_above - (1/2) e^{-(u - v_d)/t} S_above
//                   + (1/2) (U_d + e^{-(v_d - v')/t} T_below),
// which is non-decreasing in d; the root lies in the last bucket d* with
// LapSum(v_d*) <= k (or above every bucket).  Only bucket d* is then sorted
// (on chip) and solved by block_solve with the scans as carries; the scan
// totals give the certificate LapSum(a_R) <= k <= LapSum(a_L) as before.
//
// The bucket sums are accumulated in 64-bit fixed point (2^F per unit,
// F = 62 - bits(|M|), so no sum can overflow): integer additions commute,
// which keeps the result independent of the order in which the atomics land.
// A term below 2^-F is dropped, an absolute error of at most |M| 2^-F in a
// sum that enters LapSum with weight 1/2.
//
// Two launches: bucket_count (one block per 4096 keys of M) and
// bucket_solve (one workgroup).  Both read |M| and its range from the
// partition totals on the device, so the host need not wait for them.  When
// bucket d* holds more keys than the workgroup can sort (kBucketSortCap) the
// record reports side = 2, and when |M| exceeds what the launch covers (or M
// was not gathered) side = 3; the caller then solves M by the full sort.
#include <math.h>

#include "block_sort.hpp"
#include "kernels.hpp"
#include "solve_common.hpp"

namespace lapsum {

namespace {

constexpr int kBuckets = kBucketCount;
constexpr int CT = 256;             // bucket_count threads
constexpr int CI = 16;              // keys per thread
constexpr int ST = 256;             // bucket_solve threads
constexpr int SW = ST / kWave;      // 4 waves
constexpr int BPT = kBuckets / ST;  // buckets per thread
constexpr int SI = kBucketSortCap / ST;   // keys per thread in the largest on-chip sort

struct BucketGeom {
  uint32_t kmin, kmax;   // keys of max M and min M
  int shift;
  float mmin, mmax;
};

__device__ __forceinline__ float bucket_hi(const BucketGeom& g, int d) {
  // highest score bucket d can hold (its smallest key); buckets past the
  // range of M are empty and anchored at min M, so that anchors never
  // increase along the bucket order
  const uint64_t first = static_cast<uint64_t>(g.kmin) + (static_cast<uint64_t>(d) << g.shift);
  if (first > g.kmax) return g.mmin;
  return fminf(key_float(static_cast<uint32_t>(first)), g.mmax);
}
__device__ __forceinline__ float bucket_lo(const BucketGeom& g, int d) {
  // lowest score bucket d can hold (its largest key, at most key(min M))
  const uint64_t last = static_cast<uint64_t>(g.kmin) + ((static_cast<uint64_t>(d) + 1) << g.shift) - 1;
  const uint32_t key = last < g.kmax ? static_cast<uint32_t>(last) : g.kmax;
  return fmaxf(key_float(key), g.mmin);
}

// Bucket geometry from the range of M, the same in every block.
__device__ __forceinline__ BucketGeom geom_of(const PartTotals& T) {
  BucketGeom g;
  g.mmin = T.mmin;
  g.mmax = T.mmax;
  g.kmin = desc_key(T.mmax);
  g.kmax = desc_key(T.mmin);
  const uint32_t span = g.kmax - g.kmin;
  const int bits = span ? 32 - __clz(static_cast<int>(span)) : 0;
  g.shift = bits > 11 ? bits - 11 : 0;
  return g;
}

// |M| terms of at most 2^F each fit in 62 bits.
__device__ __forceinline__ int fixed_bits(int64_t m) {
  const int mbits = m > 0 ? 64 - __clzll(static_cast<long long>(m)) : 0;
  return 62 - mbits;
}

}  // namespace

// acc: [kBuckets] u32 counts, then [kBuckets] u64 U, then [kBuckets] u64 D;
// zero on entry (bucket_solve clears it again).  |M| and its range come from
// the partition totals; nothing is counted when |M| exceeds m_cap (M was not
// gathered) or the keys this grid covers.
__global__ __launch_bounds__(CT) void bucket_count_kernel(const uint32_t* __restrict__ keys,
                                                          const PartTotals* __restrict__ tot,
                                                          int64_t m_cap, double c2,
                                                          uint32_t* __restrict__ acc_n,
                                                          unsigned long long* __restrict__ acc_u,
                                                          unsigned long long* __restrict__ acc_d,
                                                          uint32_t* __restrict__ bkeys,
                                                          uint32_t* __restrict__ boff) {
  __shared__ uint32_t cn[kBuckets];
  __shared__ unsigned long long cu[kBuckets];
  __shared__ unsigned long long cd[kBuckets];
  __shared__ uint32_t cur[kBuckets];
  __shared__ uint32_t wtot[CT / kWave];
  const int tid = threadIdx.x;
  const PartTotals T = *tot;
  const int64_t m = T.nM;
  if (m < 1 || m > m_cap || m > static_cast<int64_t>(gridDim.x) * CT * CI) return;
  const int64_t base = static_cast<int64_t>(blockIdx.x) * CT * CI;
  if (base >= m) return;   // the launch is sized for the largest expected |M|
  const BucketGeom g = geom_of(T);
  const double fscale = ldexp(1.0, fixed_bits(m));
  for (int e = tid; e < kBuckets; e += CT) {
    cn[e] = 0u;
    cu[e] = 0ull;
    cd[e] = 0ull;
  }
  __syncthreads();
  uint32_t kv[CI];
#pragma unroll
  for (int i = 0; i < CI; ++i) {
    const int64_t pos = base + i * CT + tid;
    kv[i] = pos < m ? keys[pos] : 0u;
  }
#pragma unroll
  for (int i = 0; i < CI; ++i) {
    const int64_t pos = base + i * CT + tid;
    if (pos < m) {
      const uint32_t key = kv[i];
      const int d = static_cast<int>((key - g.kmin) >> g.shift);
      const double r = key_float(key);
      const double up = wexp_f32(static_cast<double>(bucket_hi(g, d)) - r, c2);   // e^{-(v_d - r)/t}
      const double dn = wexp_f32(r - static_cast<double>(bucket_lo(g, d)), c2);   // e^{-(r - u_d)/t}
      atomicAdd(&cn[d], 1u);
      atomicAdd(&cu[d], static_cast<unsigned long long>(__double2ull_rn(up * fscale)));
      atomicAdd(&cd[d], static_cast<unsigned long long>(__double2ull_rn(dn * fscale)));
    }
  }
  __syncthreads();
  // this block's keys in bucket order (any order inside a bucket), with the
  // bucket offsets, so that the solve reads only the bucket it needs
  {
    constexpr int PER = kBuckets / CT;
    const int b0 = PER * tid;
    uint32_t loc = 0;
#pragma unroll
    for (int q = 0; q < PER; ++q) loc += cn[b0 + q];
    uint32_t incl = loc;
    const int lane = lane_id();
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
      const uint32_t y = __shfl_up(incl, o, kWave);
      if (lane >= o) incl += y;
    }
    const int wid = tid / kWave;
    if (lane == kWave - 1) wtot[wid] = incl;
    __syncthreads();
    uint32_t run = incl - loc;
#pragma unroll
    for (int w = 0; w < CT / kWave; ++w)
      if (w < wid) run += wtot[w];
    uint32_t* bo = boff + static_cast<int64_t>(blockIdx.x) * (kBuckets + 1);
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      cur[b0 + q] = run;
      bo[b0 + q] = run;
      run += cn[b0 + q];
    }
    if (tid == CT - 1) bo[kBuckets] = run;
  }
  __syncthreads();
  uint32_t* bk = bkeys + static_cast<int64_t>(blockIdx.x) * CT * CI;
#pragma unroll
  for (int i = 0; i < CI; ++i) {
    const int64_t pos = base + i * CT + tid;
    if (pos < m) {
      const int d = static_cast<int>((kv[i] - g.kmin) >> g.shift);
      bk[atomicAdd(&cur[d], 1u)] = kv[i];
    }
  }
  for (int e = tid; e < kBuckets; e += CT) {
    if (cn[e]) {
      atomicAdd(&acc_n[e], cn[e]);
      atomicAdd(&acc_u[e], cu[e]);
      atomicAdd(&acc_d[e], cd[e]);
    }
  }
}

namespace {
// Sort c relative keys held in buf (any order) on chip and solve on them.
template <int ITEMS>
__device__ double sort_and_solve(uint32_t* buf, int c, const BucketGeom& g, double rank0,
                                 Pre ext_pre, Suf ext_suf, double k, double t, SortSmem<ST>& ssm,
                                 ScanSmem<SW>& csm) {
  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wid = tid / kWave;
  uint32_t key[ITEMS];
  int32_t val[ITEMS];
#pragma unroll
  for (int i = 0; i < ITEMS; ++i) {
    const int pos = wid * (kWave * ITEMS) + i * kWave + lane;
    key[i] = pos < c ? buf[buf_at(pos)] : 0xffffffffu;
    val[i] = 0;
  }
  __syncthreads();
  // relative keys of one bucket differ only in their low `shift` bits; the
  // padding (all ones) stays behind every member in each pass
  const int passes = g.shift <= 8 ? 1 : (g.shift + 7) / 8;
  for (int pidx = 0; pidx < passes; ++pidx)
    block_sort_pass<ST, ITEMS, false>(key, val, 8 * pidx, buf, ssm, pidx == passes - 1);
  float s[ITEMS];
#pragma unroll
  for (int i = 0; i < ITEMS; ++i) s[i] = key_float(key[i] + g.kmin);
  int cnt = c - tid * ITEMS;
  cnt = cnt < 0 ? 0 : (cnt > ITEMS ? ITEMS : cnt);
  Pre pt;
  Suf st;
  return block_solve<ST, ITEMS>(s, cnt, rank0, ext_pre, ext_suf, k, t, csm, &pt, &st);
}
}  // namespace

// One workgroup.  Thread tid owns buckets BPT tid .. BPT tid + BPT - 1.
// Inside a thread the pairs chain through every bucket's own anchors (empty
// buckets carry their geometric anchors and a zero sum), so the in-thread
// folds need one exponential per bucket and no search for the previous
// non-empty bucket; the block scans then join the threads.
__global__ __launch_bounds__(ST) void bucket_solve_kernel(const uint32_t* __restrict__ bkeys,
                                                          const uint32_t* __restrict__ boff,
                                                          int64_t m_cap, int64_t m_grid,
                                                          uint32_t* __restrict__ acc_n,
                                                          unsigned long long* __restrict__ acc_u,
                                                          unsigned long long* __restrict__ acc_d,
                                                          const PartTotals* __restrict__ tot,
                                                          double k, double t, int64_t n_total,
                                                          SolveRec* __restrict__ out) {
  __shared__ uint32_t buf[sort_buf_words<ST, SI>()];
  __shared__ SortSmem<ST> ssm;
  __shared__ ScanSmem<SW> csm;
  __shared__ int64_t cw[SW];
  __shared__ int64_t red_i[SW];
  __shared__ Pre cpre_s;
  __shared__ Suf csuf_s;
  __shared__ int64_t cabove_s;
  __shared__ uint32_t ccount_s;
  __shared__ uint32_t gathered_s;
  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wid = tid / kWave;
  const double inv_t = 1.0 / t;
  const Tails x = load_tails(tot);
  const int d0 = BPT * tid;
  const int64_t m = tot->nM;
  if (m > m_cap || m > m_grid) {
    // M was not gathered, or not counted: the caller solves with |M| known
    if (tid == 0) {
      SolveRec rec;
      rec.b = 0.0;
      rec.lap_aL = NAN;
      rec.lap_aR = NAN;
      rec.ok = 0;
      rec.side = 3;
      *out = rec;
    }
    return;
  }
  if (m == 0) {
    // every score is in a tail
    if (tid == 0) {
      SolveRec rec;
      rec.ok = 1;
      rec.side = 0;
      certify(x, 0.0, static_cast<double>(n_total), k, t, x.pre, x.suf, rec);
      rec.b = root_above(x, x.suf, k, t);
      *out = rec;
    }
    return;
  }
  const BucketGeom g = geom_of(*tot);
  const double inv_fscale = ldexp(1.0, -fixed_bits(m));

  // 1. this thread's buckets, cleared behind us for the next attempt
  uint32_t cnt[BPT];
  double U[BPT], D[BPT];
  float v[BPT], u[BPT];
#pragma unroll
  for (int q = 0; q < BPT; ++q) {
    cnt[q] = acc_n[d0 + q];
    U[q] = static_cast<double>(acc_u[d0 + q]) * inv_fscale;
    D[q] = static_cast<double>(acc_d[d0 + q]) * inv_fscale;
    v[q] = bucket_hi(g, d0 + q);
    u[q] = bucket_lo(g, d0 + q);
  }
#pragma unroll
  for (int q = 0; q < BPT; ++q) {
    acc_n[d0 + q] = 0u;
    acc_u[d0 + q] = 0ull;
    acc_d[d0 + q] = 0ull;
  }
  // links between consecutive anchors of this thread (all independent)
  double wu[BPT], wv[BPT];   // wu[q] = e^{-(u_{q-1} - u_q)/t}, wv[q] = e^{-(v_q - v_{q+1})/t}
#pragma unroll
  for (int q = 0; q < BPT; ++q) {
    wu[q] = q > 0 ? wexp_f64(static_cast<double>(u[q - 1]) - u[q], inv_t) : 0.0;
    wv[q] = q + 1 < BPT ? wexp_f64(static_cast<double>(v[q]) - v[q + 1], inv_t) : 0.0;
  }
  // The prefix pair may sit at any anchor at or above the root, so it
  // chains through the geometric anchors of empty buckets.  A suffix pair
  // is anchored at the upper edge of a non-empty bucket: the root lies above
  // the upper edge of the first non-empty bucket after the crossing, but can
  // lie below the edge of an empty bucket in between.
  double Pm = 0.0;   // prefix pair of the thread, anchored at u[BPT-1]
  int64_t mine = 0;
#pragma unroll
  for (int q = 0; q < BPT; ++q) {
    Pm = fma(wu[q], Pm, D[q]);
    mine += cnt[q];
  }
  double Tl[BPT];    // suffix within the thread from bucket q, anchored at v[q]
#pragma unroll
  for (int q = BPT - 1; q >= 0; --q) Tl[q] = fma(wv[q], q + 1 < BPT ? Tl[q + 1] : 0.0, U[q]);
  Suf mys = suf_empty();   // anchored at the first non-empty bucket of the thread
#pragma unroll
  for (int q = BPT - 1; q >= 0; --q)
    if (cnt[q] && Tl[q] != 0.0) mys = Suf{v[q], Tl[q]};

  // 2. block scans, seeded with the tails
  Pre pre_all;
  Suf suf_all;
  const Pre pre_in = block_excl_pre<SW>(Pre{u[BPT - 1], Pm}, x.pre, inv_t, csm, &pre_all);
  const Suf suf_in = block_excl_suf<SW>(mys, x.suf, inv_t, csm, &suf_all);
  int64_t incl = mine;
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const int64_t y = __shfl_up(incl, o, kWave);
    if (lane >= o) incl += y;
  }
  if (lane == kWave - 1) cw[wid] = incl;
  __syncthreads();
  int64_t above = incl - mine;
#pragma unroll
  for (int w = 0; w < SW; ++w)
    if (w < wid) above += cw[w];

  // 3. suffix sums from each bucket on (anchored at its v), right to left,
  //    then LapSum at each non-empty bucket's upper edge, left to right:
  //    LapSum(v_q) = n_R + above_q - (1/2) e^{-(u_prev - v_q)/t} P_before + (1/2) T_q
  double T[BPT];
  {
    double tn = suf_in.T;
    float vn = suf_in.v;
#pragma unroll
    for (int q = BPT - 1; q >= 0; --q) {
      const double w = (q + 1 < BPT) ? wv[q]
                       : (tn != 0.0 ? wexp_f64(static_cast<double>(v[q]) - vn, inv_t) : 0.0);
      T[q] = fma(w, (q + 1 < BPT) ? T[q + 1] : tn, U[q]);
    }
  }
  int64_t below = 0;   // 1 + the last bucket with LapSum(v_d) <= k
  {
    double P = pre_in.S;   // prefix before bucket q, anchored at pu
    float pu = pre_in.u;
    int64_t ab = above;
#pragma unroll
    for (int q = 0; q < BPT; ++q) {
      if (cnt[q]) {
        double lap = x.nR + static_cast<double>(ab) + 0.5 * T[q];
        if (P != 0.0) lap -= 0.5 * wexp_f64(static_cast<double>(pu) - v[q], inv_t) * P;
        if (lap <= k) below = d0 + q + 1;
      }
      const double w = (P != 0.0) ? wexp_f64(static_cast<double>(pu) - u[q], inv_t) : 0.0;
      P = fma(w, P, D[q]);
      pu = u[q];
      ab += cnt[q];
    }
  }
#pragma unroll
  for (int o = kWave / 2; o >= 1; o >>= 1) {
    const int64_t y = __shfl_xor(below, o, kWave);
    below = y > below ? y : below;
  }
  if (lane == 0) red_i[wid] = below;
  if (tid == 0) gathered_s = 0u;
  __syncthreads();
  below = 0;
#pragma unroll
  for (int w = 0; w < SW; ++w) below = red_i[w] > below ? red_i[w] : below;
  const int dstar = static_cast<int>(below) - 1;
  if (dstar >= d0 && dstar < d0 + BPT) {
    // carries around bucket d*: the prefix of everything before it and the
    // suffix of everything after it
    double P = pre_in.S;
    float pu = pre_in.u;
    int64_t ab = above;
#pragma unroll
    for (int q = 0; q < BPT; ++q) {
      if (d0 + q == dstar) {
        cpre_s = (P != 0.0) ? Pre{pu, P} : pre_empty();
        Suf after = suf_in;   // from the next non-empty bucket on
#pragma unroll
        for (int q2 = BPT - 1; q2 > q; --q2)
          if (cnt[q2] && T[q2] != 0.0) after = Suf{v[q2], T[q2]};
        csuf_s = after;
        cabove_s = ab;
        ccount_s = cnt[q];
      }
      const double w = (P != 0.0) ? wexp_f64(static_cast<double>(pu) - u[q], inv_t) : 0.0;
      P = fma(w, P, D[q]);
      pu = u[q];
      ab += cnt[q];
    }
  }
  __syncthreads();

  SolveRec rec;
  rec.ok = 1;
  rec.side = 0;
  rec.lap_aL = 0.0;
  rec.lap_aR = 0.0;
  certify(x, static_cast<double>(m), static_cast<double>(n_total), k, t, pre_all, suf_all, rec);
  double b = 0.0;
  if (dstar < 0) {
    b = root_above(x, suf_all, k, t);
  } else if (ccount_s > static_cast<uint32_t>(kBucketSortCap)) {
    rec.ok = 0;
    rec.side = 2;   // the bucket is too large to sort here: solve M by the full sort
  } else {
    // 4. gather bucket d* from each count block's bucket-ordered keys, as
    //    keys relative to key(max M), whose low `shift` bits order the
    //    bucket (the order in LDS is irrelevant: it is sorted next)
    const int nbl = static_cast<int>((m + CT * CI - 1) / (CT * CI));
    for (int b0 = 0; b0 < nbl; b0 += ST) {
      const int bl = b0 + tid;
      uint32_t from = 0, cnt_b = 0;
      if (bl < nbl) {
        const uint32_t* bo = boff + static_cast<int64_t>(bl) * (kBuckets + 1);
        from = bo[dstar];
        cnt_b = bo[dstar + 1] - from;
      }
      const uint32_t* bk = bkeys + static_cast<int64_t>(bl) * CT * CI + from;
      for (uint32_t j = 0; j < cnt_b; ++j) {
        const uint32_t at = atomicAdd(&gathered_s, 1u);
        if (at < static_cast<uint32_t>(kBucketSortCap)) buf[buf_at(static_cast<int>(at))] = bk[j] - g.kmin;
      }
    }
    __syncthreads();
    const int c = static_cast<int>(ccount_s);
    const double rank0 = x.nR + static_cast<double>(cabove_s);
    if (c <= ST)
      b = sort_and_solve<1>(buf, c, g, rank0, cpre_s, csuf_s, k, t, ssm, csm);
    else if (c <= 4 * ST)
      b = sort_and_solve<4>(buf, c, g, rank0, cpre_s, csuf_s, k, t, ssm, csm);
    else
      b = sort_and_solve<SI>(buf, c, g, rank0, cpre_s, csuf_s, k, t, ssm, csm);
  }
  if (tid == 0) {
    rec.b = b;
    *out = rec;
  }
}

hipError_t launch_bucket_solve(const uint32_t* m_keys, int64_t m_cap, int64_t m_grid, BucketAcc acc,
                               const PartTotals* tot, double k, double t, int64_t n_total,
                               SolveRec* out, hipStream_t s) {
  if (m_grid < 1) m_grid = 1;
  if (m_grid > kBucketMaxM) m_grid = kBucketMaxM;
  const int64_t blocks = (m_grid + CT * CI - 1) / (CT * CI);
  const int64_t covered = blocks * CT * CI;
  { ProfScope ps_("bucket_count", s);
  hipLaunchKernelGGL(bucket_count_kernel, dim3(static_cast<unsigned>(blocks)), dim3(CT), 0, s,
                     m_keys, tot, m_cap, kLog2e / t, acc.n, acc.u, acc.d, acc.keys, acc.offs); }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  { ProfScope ps_("bucket_solve", s);
  hipLaunchKernelGGL(bucket_solve_kernel, dim3(1), dim3(ST), 0, s, acc.keys, acc.offs, m_cap,
                     covered, acc.n, acc.u, acc.d, tot, k, t, n_total, out); }
  return hipGetLastError();
}

size_t bucket_keys_words() { return static_cast<size_t>(kBucketMaxM); }
size_t bucket_offs_words() {
  return static_cast<size_t>((kBucketMaxM + CT * CI - 1) / (CT * CI)) * (kBuckets + 1);
}

}  // namespace lapsum
