// Threshold solve on the middle set M of a bracket without sorting all of
// M (the scan, lookup and closed-form root of Suppl. A / Suppl. B, applied
// where the root is).
//
// M is cut into 2048 buckets of consecutive order-preserving keys (bucket
// d = (key - key(max M)) >> shift, so bucket 0 holds the largest scores).
// Bucket d covers the scores up to v_d, the highest float it can hold
// (clamped to the range of M); v_{d+1}, the highest the next bucket can
// hold, lies below every score of bucket d.  Bucket d is summarised by its
// count and the two sums
//     U_d = sum_{r in d} e^{-(v_d - r)/t}       (a suffix pair anchored at v_d)
//     D_d = sum_{r in d} e^{-(r - v_{d+1})/t}   (a prefix pair anchored at v_{d+1}),
// so the prefix and the suffix chains move between the same anchors by the
// same links e^{-(v_d - v_{d+1})/t}, one exponential per bucket.  The
// shift-carrying scans over the buckets, seeded with the bracket tails, give
// LapSum at every bucket's upper edge,
//     LapSum(v_d) = n_above - (1/2) S_above + (1/2) (U_d + e^{-(v_d - v')/t} T_below),
// with S_above (the buckets before d and the upper tail) anchored at v_d,
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
// Two launches, straight from the partition's per-block staging (the
// order of M within a bucket does not matter): bucket_count (one block per
// group of 8 to kBucketGroup partition blocks, at most 32 groups) and
// bucket_solve (one workgroup).  Every
// count block derives |M| and the range of M from the block records itself
// (integer min / max of keys, so all agree exactly) and folds its group's
// tails in a fixed order; bucket_solve folds those partials, so the host
// need not wait for anything.  When bucket d* holds more keys than the
// workgroup can sort (kBucketSortCap) the record reports side = 2, and when
// a block's staging overflowed or |M| exceeds the capacity side = 3; the
// caller then gathers M in index order and solves it by the full sort.
#include <math.h>

#include "block_sort.hpp"
#include "kernels.hpp"
#include "solve_common.hpp"

namespace lapsum {

namespace {

constexpr int kBuckets = kBucketCount;
constexpr int CT = 256;             // bucket_count threads
constexpr int CG = kBucketGroup;    // most partition blocks per count block
constexpr int CU = 8;               // keys per thread per batch
constexpr int ST = 512;             // bucket_solve threads: two waves per SIMD hide
                                    // the latency of each other's float64 chains
constexpr int SW = ST / kWave;      // 8 waves
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
// Bucket geometry from the keys of max M and min M, the same in every
// block.
__device__ __forceinline__ BucketGeom geom_of(uint32_t kmin, uint32_t kmax) {
  BucketGeom g;
  g.kmin = kmin;
  g.kmax = kmax;
  g.mmin = key_float(kmax);
  g.mmax = key_float(kmin);
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
// zero on entry (bucket_solve clears it again).  Count block c writes its
// partial of the totals to parts[c] whatever happens; it counts nothing when
// a block's staging overflowed or |M| exceeds m_cap (the solve then reports
// side 3).
template <int cg>
__global__ __launch_bounds__(CT) void bucket_count_kernel(const PartBlock* __restrict__ blk,
                                                          int nblocks,
                                                          const float* __restrict__ stage_v,
                                                          int64_t m_cap, double c2,
                                                          uint32_t* __restrict__ acc_n,
                                                          unsigned long long* __restrict__ acc_u,
                                                          unsigned long long* __restrict__ acc_d,
                                                          uint32_t* __restrict__ bkeys,
                                                          uint32_t* __restrict__ boff,
                                                          CountPart* __restrict__ parts) {
  __shared__ uint32_t cn[kBuckets];
  __shared__ unsigned long long cu[kBuckets];
  __shared__ unsigned long long cd[kBuckets];
  __shared__ uint32_t cur[kBuckets];
  __shared__ uint32_t wtot[CT / kWave];
  __shared__ int32_t goff[CG + 1];   // start of each group block's staged M
  __shared__ uint32_t rk[2][CT / kWave];
  __shared__ unsigned long long rm[CT / kWave];
  __shared__ uint32_t rov[CT / kWave];
  __shared__ int32_t ro[CT / kWave];
  __shared__ int32_t rdn[CT / kWave];
  __shared__ double rd[2][CT / kWave];
  __shared__ int64_t ri[3][CT / kWave];
  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wid = tid / kWave;
  const int g0 = static_cast<int>(blockIdx.x) * cg;
  constexpr int gw = (cg + kWave - 1) / kWave;   // waves holding the group's records
  static_assert(cg >= 1 && cg <= CG && (cg & (cg - 1)) == 0, "a power of two up to CG");
  // this thread's record of the group, loaded with the heads below
  const bool own = tid < cg && g0 + tid < nblocks;
  const PartBlock rec = blk[own ? g0 + tid : 0];

  // 1. |M|, the range of M and any overflow over every block (the first 16
  //    bytes of each record, all loads in flight together)
  {
    constexpr int Q = kPartMaxBlocks / CT;
    uint4 hd[Q];
#pragma unroll
    for (int q = 0; q < Q; ++q) {
      const int b = tid + CT * q;
      hd[q] = *reinterpret_cast<const uint4*>(&blk[b < nblocks ? b : nblocks - 1]);
    }
    uint32_t kmin = 0xffffffffu, kmax = 0u, ov = 0u;
    unsigned long long m = 0ull;
#pragma unroll
    for (int q = 0; q < Q; ++q) {
      if (tid + CT * q < nblocks) {
        const uint32_t nm = hd[q].z;
        if (nm > 0) {
          kmin = min(kmin, desc_key(__uint_as_float(hd[q].y)));   // key of the block's max
          kmax = max(kmax, desc_key(__uint_as_float(hd[q].x)));   // key of the block's min
        }
        m += nm;
        ov |= hd[q].w;
      }
    }
    kmin = wave_min(kmin, 0xffffffffu);
    kmax = wave_max(kmax, 0u);
    ov = wave_or(ov);
    m = wave_sum(m);
    if (lane == 0) {
      rk[0][wid] = kmin;
      rk[1][wid] = kmax;
      rm[wid] = m;
      rov[wid] = ov;
    }
  }
  // 2. this group's records: tails folded in a fixed order, and the start of
  //    each block's staged M within the group
  {
    double TL = 0.0, TR = 0.0;
    int64_t nL = 0, nR = 0, nM = 0;
    int32_t nm = 0, ov = 0, nd = 0;
    if (own) {
      TL = rec.TL;
      TR = rec.TR;
      nL = rec.nL;
      nR = rec.nR;
      nm = rec.nM;
      ov = rec.overflow;
      nd = static_cast<int32_t>(rec.band_dense);
    }
    nM = nm;
    const int32_t incl = wave_incl_add(nm);
    TL = wave_sum(TL);
    TR = wave_sum(TR);
    nL = wave_sum(nL);
    nR = wave_sum(nR);
    nM = wave_sum(nM);
    ov = wave_or(ov);
    nd = wave_sum(nd);
    if (lane == kWave - 1) wtot[wid] = static_cast<uint32_t>(incl);
    if (lane == 0) {
      rdn[wid] = nd;
      rd[0][wid] = TL;
      rd[1][wid] = TR;
      ri[0][wid] = nL;
      ri[1][wid] = nR;
      ri[2][wid] = nM;
      ro[wid] = ov;
    }
    __syncthreads();
    if (tid < cg) {
      int32_t base = 0;
#pragma unroll
      for (int w = 0; w < CG / kWave; ++w)
        if (w < wid) base += static_cast<int32_t>(wtot[w]);
      goff[tid] = base + incl - nm;
      if (tid == cg - 1) goff[cg] = base + incl;
    }
    __syncthreads();
  }
  uint32_t kmin = 0xffffffffu, kmax = 0u, aov = 0u;
  int64_t m = 0;
#pragma unroll
  for (int w = 0; w < CT / kWave; ++w) {
    kmin = min(kmin, rk[0][w]);
    kmax = max(kmax, rk[1][w]);
    m += static_cast<int64_t>(rm[w]);
    aov |= rov[w];
  }
  const int32_t any_ov = aov != 0u ? 1 : 0;
  int32_t grp_ov = 0;
#pragma unroll
  for (int w = 0; w < CG / kWave; ++w)
    if (w < gw) grp_ov |= ro[w];
  if (tid == 0) {
    CountPart cp;
    cp.TL = 0.0;
    cp.TR = 0.0;
    cp.nL = cp.nR = cp.nM = 0;
#pragma unroll
    for (int w = 0; w < CG / kWave; ++w) {
      if (w < gw) {
        cp.TL += rd[0][w];
        cp.TR += rd[1][w];
        cp.nL += ri[0][w];
        cp.nR += ri[1][w];
        cp.nM += ri[2][w];
      }
    }
    cp.overflow = grp_ov;
    cp.ndense = 0;
#pragma unroll
    for (int w = 0; w < CG / kWave; ++w)
      if (w < gw) cp.ndense += rdn[w];
    cp.pad = 0;
    cp.kmin = kmin;
    cp.kmax = kmax;
    cp.any_overflow = any_ov;
    cp.m_all = m;
    parts[blockIdx.x] = cp;
  }
  if (any_ov != 0 || m < 1 || m > m_cap) return;
  const int cb = goff[cg];   // this group's members of M (no staging overflowed)
  if (cb == 0) return;       // the solve skips a group with no members

  // 3. bucket sums of the group's members, CU keys per thread at a time;
  //    member j of the group is found by a search over goff
  const BucketGeom g = geom_of(kmin, kmax);
  const double fscale = ldexp(1.0, fixed_bits(m));
  for (int e = tid; e < kBuckets; e += CT) {
    cn[e] = 0u;
    cu[e] = 0ull;
    cd[e] = 0ull;
  }
  __syncthreads();
  auto member_key = [&](int j) -> uint32_t {
    int lo = 0, hi = cg;   // goff[lo] <= j < goff[hi]
#pragma unroll
    for (int w = cg; w > 1; w >>= 1) {
      const int mid = (lo + hi) >> 1;
      if (goff[mid] <= j) lo = mid; else hi = mid;
    }
    return desc_key(stage_v[static_cast<int64_t>(g0 + lo) * kPartStageCap + (j - goff[lo])]);
  };
  // the first batch stays in registers for the scatter below
  uint32_t kv0[CU];
  for (int j0 = 0; j0 < cb; j0 += CT * CU) {
    uint32_t kv[CU];
#pragma unroll
    for (int u = 0; u < CU; ++u) {
      const int j = j0 + u * CT + tid;
      kv[u] = member_key(j < cb ? j : cb - 1);
    }
    if (j0 == 0) {
#pragma unroll
      for (int u = 0; u < CU; ++u) kv0[u] = kv[u];
    }
#pragma unroll
    for (int u = 0; u < CU; ++u) {
      if (j0 + u * CT + tid < cb) {
        const uint32_t key = kv[u];
        const int d = static_cast<int>((key - g.kmin) >> g.shift);
        const double r = key_float(key);
        // e^{-(v_d - r)/t}, and e^{-(r - v_{d+1})/t} anchored at the next
        // bucket's upper edge (the highest score below bucket d)
        const double up = wexp_f32(static_cast<double>(bucket_hi(g, d)) - r, c2);
        const double dn = wexp_f32(r - static_cast<double>(bucket_hi(g, d + 1)), c2);
        atomicAdd(&cn[d], 1u);
        atomicAdd(&cu[d], static_cast<unsigned long long>(__double2ull_rn(up * fscale)));
        atomicAdd(&cd[d], static_cast<unsigned long long>(__double2ull_rn(dn * fscale)));
      }
    }
  }
  __syncthreads();
  // 4. the group's keys in bucket order (any order inside a bucket), with
  //    the bucket offsets, so that the solve reads only the bucket it needs
  {
    constexpr int PER = kBuckets / CT;
    const int b0 = PER * tid;
    uint32_t loc = 0;
#pragma unroll
    for (int q = 0; q < PER; ++q) loc += cn[b0 + q];
    uint32_t incl = wave_incl_add<uint32_t>(loc);
    if (lane == kWave - 1) wtot[wid] = incl;   // (its last readers passed two barriers ago)
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
  uint32_t* bk = bkeys + static_cast<int64_t>(blockIdx.x) * (static_cast<int64_t>(cg) * kPartStageCap);
  for (int j0 = 0; j0 < cb; j0 += CT * CU) {
    uint32_t kv[CU];
#pragma unroll
    for (int u = 0; u < CU; ++u) {
      const int j = j0 + u * CT + tid;
      kv[u] = j0 == 0 ? kv0[u] : member_key(j < cb ? j : cb - 1);
    }
#pragma unroll
    for (int u = 0; u < CU; ++u) {
      if (j0 + u * CT + tid < cb) {
        const int d = static_cast<int>((kv[u] - g.kmin) >> g.shift);
        bk[atomicAdd(&cur[d], 1u)] = kv[u];
      }
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

// A small bucket (c <= kDirectMax keys) is solved without sorting it:
// LapSum at each of its scores is formed term by term,
//     N(s_i) = rank0 + #{s_j > s_i} + #{s_j = s_i}/2
//              - (1/2) (sum_{s_j > s_i} e^{-(s_j - s_i)/t} + pre carry)
//              + (1/2) (sum_{s_j < s_i} e^{-(s_i - s_j)/t} + suf carry),
// which is what the scan gives at that score's positions; each key gets TPK
// threads, each summing a fixed slice of the bucket in order.  The root is
// then in the gap between u, the lowest score with N <= k, and v, the
// highest with N > k (or a carry's anchor when either side is empty), as in
// the sorted block solve.
constexpr int kDirectMax = 256;
constexpr int kDirectTpk = 16;          // at most this many threads per key
constexpr int kGatherLanes = ST / 32;   // threads per count group in the gather (<= 32 groups)
constexpr int kGatherBatch = 4;         // keys a gather thread loads at a time
struct DirectSmem {
  float4 sv4[(kDirectMax + 4 * kDirectTpk) / 4];   // the keys' scores, NaN past the end
  uint32_t ukey, vkey, has_u, has_v;
  double uA, uc, vB;
};

__device__ double direct_solve(const uint32_t* buf, int c, const BucketGeom& g, double rank0,
                               Pre ext_pre, Suf ext_suf, double k, double t, DirectSmem& ds) {
  const int tid = threadIdx.x;
  const double inv_t = 1.0 / t;
  const double c2 = kLog2e / t;
  float* sv = reinterpret_cast<float*>(ds.sv4);
  // threads per key (adjacent lanes, as many as the block holds, at most
  // kDirectTpk) and the slice of keys each sums, a multiple of 4 so that it
  // is read as float4; the slices cover tpk * slice < c + 4 tpk entries,
  // NaN past c (a NaN difference counts nowhere)
  int tpk = kDirectTpk;
  while (tpk > 1 && c * tpk > ST) tpk >>= 1;
  const int slice = ((c + tpk - 1) / tpk + 3) & ~3;
  if (tid < c) sv[tid] = key_float(buf[buf_at(tid)] + g.kmin);
  for (int e = c + tid; e < tpk * slice; e += ST) sv[e] = __int_as_float(0x7fc00000);
  if (tid == 0) {
    ds.ukey = 0u;
    ds.vkey = 0xffffffffu;
    ds.has_u = 0u;
    ds.has_v = 0u;
  }
  __syncthreads();
  const int i = tid / tpk;
  const int q = tid - i * tpk;
  const bool active = i < c;
  const float si = sv[active ? i : 0];
  const double sd = si;
  // four independent chains (one per lane of a float4), joined in order
  double Pg[4] = {0.0, 0.0, 0.0, 0.0}, El[4] = {0.0, 0.0, 0.0, 0.0};
  int gt = 0, eq = 0;
  for (int j = q * slice; j < (q + 1) * slice; j += 4) {
    const float4 v = ds.sv4[j >> 2];
    const float vv[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const double d = static_cast<double>(vv[e]) - sd;
      const double w = wexp_f32(fabs(d), c2);
      Pg[e] += d > 0.0 ? w : 0.0;
      El[e] += d < 0.0 ? w : 0.0;
      gt += d > 0.0 ? 1 : 0;
      eq += d == 0.0 ? 1 : 0;
    }
  }
  double Pgs = (Pg[0] + Pg[1]) + (Pg[2] + Pg[3]);
  double Els = (El[0] + El[1]) + (El[2] + El[3]);
  // the key's threads are adjacent lanes: join their slices
  for (int o = 1; o < tpk; o <<= 1) {
    Pgs += __shfl_xor(Pgs, o, kWave);
    Els += __shfl_xor(Els, o, kWave);
    gt += __shfl_xor(gt, o, kWave);
    eq += __shfl_xor(eq, o, kWave);
  }
  const double Pc = ext_pre.S != 0.0 ? ext_pre.S * wexp_f64(static_cast<double>(ext_pre.u) - sd, inv_t) : 0.0;
  const double Ec = ext_suf.T != 0.0 ? ext_suf.T * wexp_f64(sd - static_cast<double>(ext_suf.v), inv_t) : 0.0;
  const double N = rank0 + gt + 0.5 * eq - 0.5 * (Pgs + Pc) + 0.5 * (Els + Ec);
  const bool le = N <= k;
  const uint32_t key = desc_key(si);
  const bool lead = active && q == 0;
  {
    // the lowest score at or below k (largest key) and the highest above k
    // (smallest key): reduced in the wave, then one atomic per wave
    const uint32_t uk = wave_max_u32((lead && le) ? key : 0u);
    const uint32_t vk = wave_min_u32((lead && !le) ? key : 0xffffffffu);
    const bool hu = __ballot(lead && le) != 0ull, hv = __ballot(lead && !le) != 0ull;
    if (lane_id() == 0) {
      if (hu) {
        atomicMax(&ds.ukey, uk);
        atomicOr(&ds.has_u, 1u);
      }
      if (hv) {
        atomicMin(&ds.vkey, vk);
        atomicOr(&ds.has_v, 1u);
      }
    }
  }
  __syncthreads();
  // equal scores give equal sums, so any holder of u (or v) may publish
  if (lead && le && key == ds.ukey) {
    ds.uA = Pgs + eq + Pc;
    ds.uc = gt + eq;
  }
  if (lead && !le && key == ds.vkey) ds.vB = Els + eq + Ec;
  __syncthreads();
  double b = 0.0;
  if (tid < 2) {
    // the two logarithms of the gap's sums side by side (lanes 0 and 1)
    const bool has_u = ds.has_u != 0u, has_v = ds.has_v != 0u;
    const bool has_dn = ext_suf.T != 0.0;
    double arg;
    if (tid == 0)
      arg = has_u ? ds.uA : (ext_pre.S > 0 ? ext_pre.S : 1.0);
    else
      arg = has_v ? ds.vB : (has_dn ? ext_suf.T : 1.0);
    const double lg = log(arg);
    const double lnB = __shfl(lg, 1, kWave);
    if (tid == 0) {
      const double lnA = lg;
      const double v = key_float(ds.vkey);
      if (!has_u) {
        // b lies above every score of the bucket
        b = gap_root(k, t, rank0, ext_pre.S != 0.0, ext_pre.u, lnA, true, v, lnB);
      } else {
        const double u = key_float(ds.ukey);
        if (has_v)
          b = gap_root(k, t, rank0 + ds.uc, true, u, lnA, true, v, lnB);
        else
          b = gap_root(k, t, rank0 + ds.uc, true, u, lnA, has_dn, ext_suf.v, lnB);
      }
    }
  }
  return b;   // thread 0's value
}

// Shared memory of the bucketed solve (one workgroup of ST threads).
struct BucketSolveSmem {
  uint32_t buf[sort_buf_words<ST, SI>()];
  SortSmem<ST> ssm;
  ScanSmem<SW> csm;
  int64_t cw[SW];
  int64_t red_i[SW];
  Pre cpre_s;
  Suf csuf_s;
  int64_t cabove_s;
  uint32_t ccount_s;
  uint32_t gathered_s;
  DirectSmem dsm;
};

// The scans over the buckets, the lookup of the bucket holding the root, the
// certificate and the root, by one workgroup of ST threads.  Thread tid owns
// buckets BPT tid .. BPT tid + BPT - 1 with their counts and the two sums
// (U anchored at the bucket's upper edge, D at the next bucket's upper
// edge).  Inside a thread the pairs chain through every bucket's own anchors
// (empty buckets carry their geometric anchors and a zero sum), so the
// in-thread folds need one exponential per bucket and no search for the
// previous non-empty bucket; the block scans then join the threads.
// gather(dstar, S) appends the keys of bucket dstar, relative to g.kmin, to
// S.buf (buf_at order, one atomicAdd on S.gathered_s per key, at most
// kBucketSortCap kept); every thread calls it.  Returns b (valid in thread
// 0) and fills rec (ok = 0, side = 2 when the root's bucket exceeds
// kBucketSortCap keys).
template <class Gather>
__device__ double bucket_core(const uint32_t (&cnt)[BPT], const double (&U)[BPT],
                              const double (&D)[BPT], const BucketGeom& g, int64_t m,
                              const Tails& x, double k, double t, int64_t n_total,
                              BucketSolveSmem& S, SolveRec& rec, Gather&& gather) {
  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wid = tid / kWave;
  const double inv_t = 1.0 / t;
  const int d0 = BPT * tid;
  // 1. the links between consecutive anchors: the suffix sum of bucket q is
  //    anchored at its upper edge v_q and the prefix sum at v_{q+1}, the
  //    upper edge of the bucket after it, so both chains move between
  //    anchors by the same links wv[q] = e^{-(v_q - v_{q+1})/t}, one
  //    exponential per bucket (all independent)
  float v[BPT + 1];   // v[BPT]: the upper edge of the next thread's first bucket
#pragma unroll
  for (int q = 0; q <= BPT; ++q) v[q] = bucket_hi(g, d0 + q);
  double wv[BPT];
#pragma unroll
  for (int q = 0; q < BPT; ++q) wv[q] = wexp_f64(static_cast<double>(v[q]) - v[q + 1], inv_t);
  // The prefix pair may sit at any anchor at or above the root, so it
  // chains through the geometric anchors of empty buckets.  A suffix pair
  // is anchored at the upper edge of a non-empty bucket: the root lies above
  // the upper edge of the first non-empty bucket after the crossing, but can
  // lie below the edge of an empty bucket in between.
  double Pm = 0.0;   // prefix pair of the thread, anchored at v[BPT]
  int64_t mine = 0;
#pragma unroll
  for (int q = 0; q < BPT; ++q) {
    Pm = fma(wv[q], Pm, D[q]);
    mine += cnt[q];
  }
  double Tl[BPT];    // suffix within the thread from bucket q, anchored at v[q]
#pragma unroll
  for (int q = BPT - 1; q >= 0; --q) Tl[q] = q + 1 < BPT ? fma(wv[q], Tl[q + 1], U[q]) : U[q];
  Suf mys = suf_empty();   // anchored at the first non-empty bucket of the thread
#pragma unroll
  for (int q = BPT - 1; q >= 0; --q)
    if (cnt[q] && Tl[q] != 0.0) mys = Suf{v[q], Tl[q]};

  // 2. block scans, seeded with the tails
  Pre pre_all;
  Suf suf_all;
  Pre pre_in;
  Suf suf_in;
  block_excl_pre_suf<SW>(Pre{v[BPT], Pm}, x.pre, mys, x.suf, inv_t, S.csm, &pre_in, &pre_all, &suf_in,
                         &suf_all);
  // the counts scan in 32 bits (fewer than 2^31 keys)
  const int64_t incl = static_cast<int64_t>(wave_incl_add(static_cast<uint32_t>(mine)));
  if (lane == kWave - 1) S.cw[wid] = incl;
  __syncthreads();
  int64_t above = incl - mine;
#pragma unroll
  for (int w = 0; w < SW; ++w)
    if (w < wid) above += S.cw[w];

  // 3. suffix sums from each bucket on (anchored at its v), right to left,
  //    then LapSum at each non-empty bucket's upper edge, left to right:
  //    LapSum(v_q) = n_R + above_q - (1/2) e^{-(a - v_q)/t} P_before + (1/2) T_q
  //    with P_before anchored at a, which is v_q itself (weight 1) unless
  //    the prefix still sits on the seed's anchor.  Moving P past bucket q
  //    takes the link wv[q] in the same case.
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
      const bool at_v = pu == v[q];
      if (cnt[q]) {
        double lap = x.nR + static_cast<double>(ab) + 0.5 * T[q];
        if (P != 0.0) lap -= 0.5 * (at_v ? P : wexp_f64(static_cast<double>(pu) - v[q], inv_t) * P);
        if (lap <= k) below = d0 + q + 1;
      }
      const double w = (P != 0.0) ? (at_v ? wv[q] : wexp_f64(static_cast<double>(pu) - v[q + 1], inv_t))
                                  : 0.0;
      P = fma(w, P, D[q]);
      pu = v[q + 1];
      ab += cnt[q];
    }
  }
  below = static_cast<int64_t>(wave_max_u32(static_cast<uint32_t>(below)));
  if (lane == 0) S.red_i[wid] = below;
  if (tid == 0) S.gathered_s = 0u;
  __syncthreads();
  below = 0;
#pragma unroll
  for (int w = 0; w < SW; ++w) below = S.red_i[w] > below ? S.red_i[w] : below;
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
        S.cpre_s = (P != 0.0) ? Pre{pu, P} : pre_empty();
        Suf after = suf_in;   // from the next non-empty bucket on
#pragma unroll
        for (int q2 = BPT - 1; q2 > q; --q2)
          if (cnt[q2] && T[q2] != 0.0) after = Suf{v[q2], T[q2]};
        S.csuf_s = after;
        S.cabove_s = ab;
        S.ccount_s = cnt[q];
      }
      const double w = (P != 0.0) ? (pu == v[q] ? wv[q]
                                                : wexp_f64(static_cast<double>(pu) - v[q + 1], inv_t))
                                  : 0.0;
      P = fma(w, P, D[q]);
      pu = v[q + 1];
      ab += cnt[q];
    }
  }
  __syncthreads();

  rec.ok = 1;
  rec.side = 0;
  rec.lap_aL = 0.0;
  rec.lap_aR = 0.0;
  certify(x, static_cast<double>(m), static_cast<double>(n_total), k, t, pre_all, suf_all, rec);
  double b = 0.0;
  if (dstar < 0) {
    b = root_above(x, suf_all, k, t);
  } else if (S.ccount_s > static_cast<uint32_t>(kBucketSortCap)) {
    rec.ok = 0;
    rec.side = 2;   // the bucket is too large to sort here
  } else {
    // 4. bucket d*'s keys relative to g.kmin, whose low `shift` bits order
    //    the bucket (the order in LDS is irrelevant: it is sorted next)
    gather(dstar, S);
    __syncthreads();
    const int c = static_cast<int>(S.ccount_s);
    const double rank0 = x.nR + static_cast<double>(S.cabove_s);
    if (c <= kDirectMax)
      b = direct_solve(S.buf, c, g, rank0, S.cpre_s, S.csuf_s, k, t, S.dsm);
    else if (c <= 2 * ST)
      b = sort_and_solve<2>(S.buf, c, g, rank0, S.cpre_s, S.csuf_s, k, t, S.ssm, S.csm);
    else
      b = sort_and_solve<SI>(S.buf, c, g, rank0, S.cpre_s, S.csuf_s, k, t, S.ssm, S.csm);
  }
  return b;
}
}  // namespace

// One workgroup: the middle set's buckets from the count blocks, then
// bucket_core.
__global__ __launch_bounds__(ST) void bucket_solve_kernel(const uint32_t* __restrict__ bkeys,
                                                          const uint32_t* __restrict__ boff,
                                                          const CountPart* __restrict__ parts,
                                                          int ngroups, int64_t gstride,
                                                          int64_t m_cap,
                                                          const SelectRec* __restrict__ sel,
                                                          int use_sel, float aL_arg, float aR_arg,
                                                          uint32_t* __restrict__ acc_n,
                                                          unsigned long long* __restrict__ acc_u,
                                                          unsigned long long* __restrict__ acc_d,
                                                          PartTotals* __restrict__ tot,
                                                          double k, double t, int64_t n_total,
                                                          SolveRec* __restrict__ out,
                                                          AttemptRec* __restrict__ host,
                                                          uint32_t* __restrict__ host_seq,
                                                          uint32_t seq) {
  __shared__ BucketSolveSmem S;
  __shared__ PartTotals tot_s;
  __shared__ int64_t gcount_s[kPartMaxBlocks / CG];
  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wid = tid / kWave;
  const int d0 = BPT * tid;
  // this thread's buckets, loaded with the partials below (they are zero
  // when nothing was counted), and cleared behind us for the next attempt
  uint32_t cnt[BPT];
  unsigned long long Ur[BPT], Dr[BPT];
#pragma unroll
  for (int q = 0; q < BPT; ++q) {
    cnt[q] = acc_n[d0 + q];
    Ur[q] = acc_u[d0 + q];
    Dr[q] = acc_d[d0 + q];
  }
  // 0. the partition totals from the count blocks' partials (wave 0, in a
  //    fixed order), for this solve, the host and the emit
  if (wid == 0) {
    const CountPart cp = parts[lane < ngroups ? lane : 0];
    const bool on = lane < ngroups;
    const double TL = wave_sum(on ? cp.TL : 0.0);
    const double TR = wave_sum(on ? cp.TR : 0.0);
    const int64_t nL = wave_sum(on ? cp.nL : int64_t(0));
    const int64_t nR = wave_sum(on ? cp.nR : int64_t(0));
    const int32_t nd = wave_sum(on ? cp.ndense : 0);
    if (on) gcount_s[lane] = cp.nM;
    if (lane == 0) {
      // |M|, its range and the overflow flag are the same in every partial
      PartTotals T;
      T.TL = TL;
      T.TR = TR;
      T.nL = nL;
      T.nR = nR;
      T.nM = cp.m_all;
      T.aL = use_sel ? sel->aL : aL_arg;
      T.aR = use_sel ? sel->aR : aR_arg;
      T.mmin = cp.m_all > 0 ? key_float(cp.kmax) : INFINITY;
      T.mmax = cp.m_all > 0 ? key_float(cp.kmin) : -INFINITY;
      T.any_block_overflow = cp.any_overflow;
      T.dense_blocks = nd;
      tot_s = T;
      *tot = T;
    }
  }
#pragma unroll
  for (int q = 0; q < BPT; ++q) {
    acc_n[d0 + q] = 0u;
    acc_u[d0 + q] = 0ull;
    acc_d[d0 + q] = 0ull;
  }
  __syncthreads();
  // thread 0: the record, for the emit, and with the totals for the host
  auto publish = [&](const SolveRec& rec) {
    *out = rec;
    if (host) {
      host->tot = tot_s;
      host->rec = rec;
      __threadfence_system();   // the record lands before the sequence number
      *reinterpret_cast<volatile uint32_t*>(host_seq) = seq;
    }
  };
  const Tails x = load_tails(&tot_s);
  const int64_t m = tot_s.nM;
  if (m > m_cap || tot_s.any_block_overflow != 0) {
    // M was not counted: the caller gathers it and solves with |M| known
    if (tid == 0) {
      SolveRec rec;
      rec.b = 0.0;
      rec.lap_aL = NAN;
      rec.lap_aR = NAN;
      rec.ok = 0;
      rec.side = 3;
      publish(rec);
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
      publish(rec);
    }
    return;
  }
  const BucketGeom g = geom_of(parts[0].kmin, parts[0].kmax);
  const double inv_fscale = ldexp(1.0, -fixed_bits(m));
  double U[BPT], D[BPT];
#pragma unroll
  for (int q = 0; q < BPT; ++q) {
    U[q] = static_cast<double>(Ur[q]) * inv_fscale;
    D[q] = static_cast<double>(Dr[q]) * inv_fscale;
  }
  // bucket d* from each count block's bucket-ordered keys (a group with no
  // members wrote no offsets); kGatherLanes threads per group, each loading
  // its keys before placing any
  auto gather = [&](int dstar, BucketSolveSmem& Sm) {
    const int grp = tid / kGatherLanes;
    const int sub = tid % kGatherLanes;
    if (grp < ngroups && gcount_s[grp] > 0) {
      const uint32_t* bo = boff + static_cast<int64_t>(grp) * (kBuckets + 1);
      const uint32_t from = bo[dstar];
      const uint32_t cnt_b = bo[dstar + 1] - from;
      const uint32_t* bk = bkeys + static_cast<int64_t>(grp) * gstride + from;
      for (uint32_t j0 = 0; j0 < cnt_b; j0 += kGatherLanes * kGatherBatch) {
        uint32_t kv[kGatherBatch];
#pragma unroll
        for (int u = 0; u < kGatherBatch; ++u) {
          const uint32_t j = j0 + static_cast<uint32_t>(u * kGatherLanes + sub);
          kv[u] = bk[j < cnt_b ? j : 0];
        }
#pragma unroll
        for (int u = 0; u < kGatherBatch; ++u) {
          if (j0 + static_cast<uint32_t>(u * kGatherLanes + sub) < cnt_b) {
            const uint32_t at = atomicAdd(&Sm.gathered_s, 1u);
            if (at < static_cast<uint32_t>(kBucketSortCap)) Sm.buf[buf_at(static_cast<int>(at))] = kv[u] - g.kmin;
          }
        }
      }
    }
  };
  SolveRec rec;
  const double b = bucket_core(cnt, U, D, g, m, x, k, t, n_total, S, rec, gather);
  if (tid == 0) {
    rec.b = b;
    publish(rec);
  }
}

// ------------------------------------------------------------ bucketed rows --
// The full-sort forward's threshold for a row of n <= kRowOnChipMax scores
// without sorting the row (used when no permutation is asked for): one
// workgroup per row holds the row in registers, cuts it into kBuckets
// buckets of consecutive keys over the row's own range, sums each bucket
// as the middle-set solve does (count, and the two exponential sums in
// 64-bit fixed point, by LDS atomics), and runs bucket_core without tails:
// the scans give LapSum at every bucket edge, and only the bucket holding
// the root is sorted (or solved term by term).  The same equation is solved
// in the same interval as by the sort, so b agrees to rounding.  p is then
// written from the registers: the row is read once and p written once.
// A row whose root bucket holds more than kBucketSortCap scores (many equal
// or near-equal scores; only a row longer than that can) gets b = NaN and no
// p; row_forward_kernel, launched behind this kernel in its gated form for
// such row lengths, then solves those rows by the full sort.
//
// Item i of thread tid is score 4 (tid + ST (i/4)) + i%4 with float4 loads
// (VEC, n a multiple of 4), else tid + ST i.
template <int ITEMS, bool VEC>
__device__ __forceinline__ int row_item_index(int tid, int i) {
  return VEC ? 4 * (tid + ST * (i / 4)) + (i % 4) : tid + ST * i;
}

template <int ITEMS, bool VEC>
__global__ __launch_bounds__(ST) void row_bucket_forward_kernel(const float* __restrict__ scores,
                                                                int n, double k, double t,
                                                                float* __restrict__ p,
                                                                double* __restrict__ b_out) {
  static_assert(!VEC || ITEMS % 4 == 0, "float4 items");
  __shared__ BucketSolveSmem S;
  __shared__ uint32_t cn[kBuckets];
  __shared__ unsigned long long cu[kBuckets];
  __shared__ unsigned long long cd[kBuckets];
  __shared__ uint32_t rk[2][SW];
  __shared__ double b_s;
  __shared__ float edge[kBuckets + 1];   // bucket_hi of every bucket edge, read twice per score
  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wid = tid / kWave;
  const int64_t row = blockIdx.x;
  const float* r = scores + row * static_cast<int64_t>(n);

  // 1. the row, all loads in flight together
  float x[ITEMS];
  if constexpr (VEC) {
    const float4* r4 = reinterpret_cast<const float4*>(r);
    const int n4 = n / 4;
#pragma unroll
    for (int j = 0; j < ITEMS / 4; ++j) {
      const int q = tid + ST * j;
      const float4 v = r4[q < n4 ? q : 0];
      x[4 * j] = v.x;
      x[4 * j + 1] = v.y;
      x[4 * j + 2] = v.z;
      x[4 * j + 3] = v.w;
    }
  } else {
#pragma unroll
    for (int i = 0; i < ITEMS; ++i) {
      const int e = tid + ST * i;
      x[i] = r[e < n ? e : 0];
    }
  }
  // 2. the range of the row's keys (the bucket geometry) and clear the
  //    bucket sums
  uint32_t kmin = 0xffffffffu, kmax = 0u;
#pragma unroll
  for (int i = 0; i < ITEMS; ++i) {
    if (row_item_index<ITEMS, VEC>(tid, i) < n) {
      const uint32_t key = desc_key(x[i]);
      kmin = min(kmin, key);
      kmax = max(kmax, key);
    }
  }
  kmin = wave_min(kmin, 0xffffffffu);
  kmax = wave_max(kmax, 0u);
  if (lane == 0) {
    rk[0][wid] = kmin;
    rk[1][wid] = kmax;
  }
  for (int e = tid; e < kBuckets; e += ST) {
    cn[e] = 0u;
    cu[e] = 0ull;
    cd[e] = 0ull;
  }
  __syncthreads();
#pragma unroll
  for (int w = 0; w < SW; ++w) {
    kmin = min(kmin, rk[0][w]);
    kmax = max(kmax, rk[1][w]);
  }
  const BucketGeom g = geom_of(kmin, kmax);
  const double fscale = ldexp(1.0, fixed_bits(n));
  const double c2 = kLog2e / t;
  for (int e = tid; e <= kBuckets; e += ST) edge[e] = bucket_hi(g, e);
  __syncthreads();

  // 3. bucket counts and sums: e^{-(v_d - r)/t} anchored at the bucket's
  //    upper edge and e^{-(r - v_{d+1})/t} at the next bucket's
#pragma unroll
  for (int i = 0; i < ITEMS; ++i) {
    if (row_item_index<ITEMS, VEC>(tid, i) < n) {
      const uint32_t key = desc_key(x[i]);
      const int d = static_cast<int>((key - g.kmin) >> g.shift);
      const double rv = x[i];
      const double up = wexp_f32(static_cast<double>(edge[d]) - rv, c2);
      const double dn = wexp_f32(rv - static_cast<double>(edge[d + 1]), c2);
      atomicAdd(&cn[d], 1u);
      atomicAdd(&cu[d], static_cast<unsigned long long>(__double2ull_rn(up * fscale)));
      atomicAdd(&cd[d], static_cast<unsigned long long>(__double2ull_rn(dn * fscale)));
    }
  }
  __syncthreads();
  const int d0 = BPT * tid;
  const double inv_fscale = ldexp(1.0, -fixed_bits(n));
  uint32_t cnt[BPT];
  double U[BPT], D[BPT];
#pragma unroll
  for (int q = 0; q < BPT; ++q) {
    cnt[q] = cn[d0 + q];
    U[q] = static_cast<double>(cu[d0 + q]) * inv_fscale;
    D[q] = static_cast<double>(cd[d0 + q]) * inv_fscale;
  }
  // 4. scans, lookup and root; the root's bucket gathered from registers
  auto gather = [&](int dstar, BucketSolveSmem& Sm) {
#pragma unroll
    for (int i = 0; i < ITEMS; ++i) {
      if (row_item_index<ITEMS, VEC>(tid, i) < n) {
        const uint32_t rel = desc_key(x[i]) - g.kmin;
        if (static_cast<int>(rel >> g.shift) == dstar) {
          const uint32_t at = atomicAdd(&Sm.gathered_s, 1u);
          if (at < static_cast<uint32_t>(kBucketSortCap)) Sm.buf[buf_at(static_cast<int>(at))] = rel;
        }
      }
    }
  };
  const Tails tails = load_tails(nullptr);
  SolveRec rec;
  const double b = bucket_core(cnt, U, D, g, static_cast<int64_t>(n), tails, k, t,
                               static_cast<int64_t>(n), S, rec, gather);
  if (tid == 0) {
    b_s = rec.ok ? b : NAN;
    b_out[row] = b_s;
  }
  __syncthreads();
  const double bb = b_s;
  if (!(bb == bb)) return;   // the gated full-sort kernel solves this row
  // 5. p from the registers
  const double inv_t = 1.0 / t;
  float* pr = p + row * static_cast<int64_t>(n);
  if constexpr (VEC) {
    float4* p4 = reinterpret_cast<float4*>(pr);
    const int n4 = n / 4;
#pragma unroll
    for (int j = 0; j < ITEMS / 4; ++j) {
      const int q = tid + ST * j;
      if (q < n4) {
        float4 o;
        o.x = laplace_p(x[4 * j], bb, inv_t);
        o.y = laplace_p(x[4 * j + 1], bb, inv_t);
        o.z = laplace_p(x[4 * j + 2], bb, inv_t);
        o.w = laplace_p(x[4 * j + 3], bb, inv_t);
        p4[q] = o;
      }
    }
  } else {
#pragma unroll
    for (int i = 0; i < ITEMS; ++i) {
      const int e = tid + ST * i;
      if (e < n) pr[e] = laplace_p(x[i], bb, inv_t);
    }
  }
}

hipError_t launch_row_bucket_forward(const float* scores, int64_t batch, int64_t n, double k,
                                     double t, float* p, double* b, hipStream_t s) {
  if (n < 1 || n > kRowOnChipMax || batch < 1) return hipErrorInvalidValue;
  const dim3 grid(static_cast<unsigned>(batch)), block(ST);
  const int ni = static_cast<int>(n);
  const bool vec = (n % 4) == 0;
  { ProfScope ps_("row_bucket_forward", s);
#define LAPSUM_ROWB(IT)                                                                          \
  if (vec)                                                                                       \
    hipLaunchKernelGGL((row_bucket_forward_kernel<IT, true>), grid, block, 0, s, scores, ni, k,  \
                       t, p, b);                                                                 \
  else                                                                                           \
    hipLaunchKernelGGL((row_bucket_forward_kernel<IT, false>), grid, block, 0, s, scores, ni, k, \
                       t, p, b)
  if (n <= ST * 4) {
    LAPSUM_ROWB(4);
  } else if (n <= ST * 8) {
    LAPSUM_ROWB(8);
  } else if (n <= ST * 16) {
    LAPSUM_ROWB(16);
  } else if (n <= ST * 32) {
    LAPSUM_ROWB(32);
  } else {
    LAPSUM_ROWB(64);
  }
#undef LAPSUM_ROWB
  }
  return hipGetLastError();
}

// Partition blocks per count block: the smallest power of two from 8 to CG
// that keeps the groups within 32 (one lane each in the solve), so that a
// short row with a wide middle set still spreads its counting over up to 32
// blocks (a row of 2^20 scores with |M| = 1e5 gave its two count blocks of
// 128 partition blocks 38.7 us).
int bucket_group_size(int nblocks) {
  int cg = CG;
  while (cg > 8 && (nblocks + cg / 2 - 1) / (cg / 2) <= 32) cg /= 2;
  return cg;
}
int bucket_groups(int nblocks) {
  const int cg = bucket_group_size(nblocks);
  return (nblocks + cg - 1) / cg;
}
size_t bucket_keys_words(int nblocks) {
  return static_cast<size_t>(bucket_groups(nblocks)) * static_cast<size_t>(bucket_group_size(nblocks)) *
         static_cast<size_t>(kPartStageCap);
}
size_t bucket_offs_words(int nblocks) {
  return static_cast<size_t>(bucket_groups(nblocks)) * (kBuckets + 1);
}

hipError_t launch_bucket_solve(const PartSource& ps, int64_t m_cap, BucketAcc acc, PartTotals* tot,
                               double k, double t, int64_t n_total, SolveRec* out,
                               AttemptRec* host, uint32_t* host_seq, uint32_t seq, hipStream_t s) {
  if (ps.nblocks < 1 || ps.nblocks > kPartMaxBlocks) return hipErrorInvalidValue;
  const int groups = bucket_groups(ps.nblocks);   // <= 32: one lane each in the solve
  const int cg = bucket_group_size(ps.nblocks);
  { ProfScope ps_("bucket_count", s);
#define LAPSUM_COUNT(G)                                                                          \
  hipLaunchKernelGGL(bucket_count_kernel<G>, dim3(static_cast<unsigned>(groups)), dim3(CT), 0, s, \
                     ps.blk, ps.nblocks, ps.stage_v, m_cap, kLog2e / t, acc.n, acc.u, acc.d,      \
                     acc.keys, acc.offs, acc.parts)
  switch (cg) {
    case 8: LAPSUM_COUNT(8); break;
    case 16: LAPSUM_COUNT(16); break;
    case 32: LAPSUM_COUNT(32); break;
    case 64: LAPSUM_COUNT(64); break;
    default: LAPSUM_COUNT(CG); break;
  }
#undef LAPSUM_COUNT
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  { ProfScope ps_("bucket_solve", s);
  hipLaunchKernelGGL(bucket_solve_kernel, dim3(1), dim3(ST), 0, s, acc.keys, acc.offs, acc.parts,
                     groups, static_cast<int64_t>(cg) * kPartStageCap, m_cap, ps.sel, ps.use_sel,
                     ps.aL, ps.aR, acc.n, acc.u, acc.d, tot, k, t, n_total, out, host, host_seq,
                     seq); }
  return hipGetLastError();
}

}  // namespace lapsum
