// The probabilistic bracket (§4, Suppl. B, Suppl. C, Algorithm 1):
//   sample            y_s = fl32(r[s * floor(n/K)] + eps_s) (the systematic
//                     sampler: strided view + cached kernel noise), stored as
//                     ascending uint32 keys grouped per block by their top
//                     11 bits, with the bin offsets
//   select            the j-th and l-th smallest y (Eq. (8)) by an 11/11/10
//                     bit radix select in one workgroup (only the keys of the
//                     target's top-11-bit bin are fetched)
//   partition         the single streaming pass: L = {r < a_L},
//                     M = {a_L <= r < a_R}, R = {r >= a_R}, the tail sums of
//                     Eq. (7) and counts, M compacted in index order into the
//                     block's staging area          (4 bytes read per score)
//   partition_totals  fixed-order totals and each block's M offset
//   gather            M to one contiguous array of (key, index)
#include <math.h>

#include <type_traits>

#include "block_sort.hpp"
#include "kernels.hpp"

namespace lapsum {

namespace {

__device__ __forceinline__ uint32_t asc_key(float f) { return ~desc_key(f); }
__device__ __forceinline__ float asc_key_float(uint32_t k) { return key_float(~k); }

constexpr int kSampleThreads = 256;
// 1024 draws per block: twice the blocks of 2048 took the sample from 11.0 to
// 8.6 us at K = 1e5 and cost the select 1.1 us more of level-1 counts
constexpr int kSampleItems = 4;
constexpr int64_t kSampleBlock = static_cast<int64_t>(kSampleThreads) * kSampleItems;   // 1024
constexpr int kSelThreads = 1024;
constexpr int PT = kPartThreads;               // 256
constexpr int PW = PT / kWave;                 // 4 waves

}  // namespace

// ----------------------------------------------------------------- sample --
// Block b draws samples [b SB, b SB + SB) (kSampleItems per thread, all loads
// in flight together; sample s reads r[s floor(n/K)], or r[idx[s]] when the
// caller gives i.i.d. indices) and writes their keys grouped by the top 11 bits
// (kSelectBins bins, any order inside a bin) into its own region of ykeys,
// with the exclusive bin offsets soffs[b (kSelectBins + 1) + bin], the bin
// counts packed two to a word (16 bits each) in scnt[b kSampleCntWords + i]
// and after them the counts of the kSelectGroups groups of consecutive bins;
// nothing needs to be zero beforehand.  The blocks also clear `zero`
// (zero_words u32), which later passes accumulate into.
__global__ __launch_bounds__(kSampleThreads) void sample_kernel(const float* __restrict__ r,
                                                                int64_t n,
                                                                const float* __restrict__ noise,
                                                                uint64_t seed, double t,
                                                                const int32_t* __restrict__ idx,
                                                                int64_t K, uint32_t* __restrict__ ykeys,
                                                                uint32_t* __restrict__ soffs,
                                                                uint32_t* __restrict__ scnt,
                                                                uint32_t* __restrict__ zero,
                                                                int64_t zero_words) {
  __shared__ uint32_t h[kSelectBins];
  __shared__ uint32_t wsum[kSampleThreads / kWave];
  const int tid = threadIdx.x;
  for (int e = tid; e < kSelectBins; e += kSampleThreads) h[e] = 0u;
  for (int64_t w = static_cast<int64_t>(blockIdx.x) * kSampleThreads + tid; w < zero_words;
       w += static_cast<int64_t>(gridDim.x) * kSampleThreads)
    zero[w] = 0u;
  const int64_t stride = n / K;
  const int64_t base = static_cast<int64_t>(blockIdx.x) * kSampleBlock;
  float rv[kSampleItems], ev[kSampleItems];
#pragma unroll
  for (int i = 0; i < kSampleItems; ++i) {
    const int64_t s = base + static_cast<int64_t>(i) * kSampleThreads + tid;
    const int64_t sc = s < K ? s : K - 1;
    int64_t at = sc * stride;
    if (idx) {   // i.i.d. sampler: the caller's indices, clamped to the row
      const int32_t q = idx[sc];
      at = q < 0 ? 0 : (q >= n ? n - 1 : q);
    }
    rv[i] = r[at];
    ev[i] = noise ? noise[sc] : counter_laplace(seed, sc, t);
  }
  __syncthreads();
  uint32_t key[kSampleItems], slot[kSampleItems];
#pragma unroll
  for (int i = 0; i < kSampleItems; ++i) {
    const int64_t s = base + static_cast<int64_t>(i) * kSampleThreads + tid;
    key[i] = asc_key(rv[i] + ev[i]);   // float32 addition
    slot[i] = s < K ? atomicAdd(&h[key[i] >> 21], 1u) : 0u;
  }
  __syncthreads();
  // exclusive offsets of the bins, PER consecutive bins per thread
  constexpr int PER = kSelectBins / kSampleThreads;
  uint32_t c[PER];
  uint32_t loc = 0u;
#pragma unroll
  for (int e = 0; e < PER; ++e) {
    c[e] = h[PER * tid + e];
    loc += c[e];
  }
  uint32_t incl = wave_incl_add<uint32_t>(loc);
  const int lane = lane_id();
  const int wid = tid / kWave;
  if (lane == kWave - 1) wsum[wid] = incl;
  __syncthreads();
  uint32_t run = incl - loc;
#pragma unroll
  for (int w = 0; w < kSampleThreads / kWave; ++w) {
    const uint32_t x = wsum[w];
    run += w < wid ? x : 0u;
  }
  uint32_t* so = soffs + static_cast<int64_t>(blockIdx.x) * (kSelectBins + 1);
  uint32_t* sc = scnt + static_cast<int64_t>(blockIdx.x) * kSampleCntWords;
  {
    // the count of each group of kSelectBins / kSelectGroups bins (the
    // bins of TPG adjacent threads)
    constexpr int TPG = kSelectBins / kSelectGroups / PER;
    static_assert(TPG >= 1 && TPG <= 4 && (TPG & (TPG - 1)) == 0, "a group is 1, 2 or 4 threads' bins");
    uint32_t gsum = loc;
    if (TPG >= 2) gsum += __shfl_xor(gsum, 1, kWave);
    if (TPG >= 4) gsum += __shfl_xor(gsum, 2, kWave);
    if (tid % TPG == 0) sc[kSelectBins / 2 + tid / TPG] = gsum;
  }
#pragma unroll
  for (int e = 0; e < PER; ++e) {
    h[PER * tid + e] = run;
    so[PER * tid + e] = run;
    run += c[e];
  }
#pragma unroll
  for (int e = 0; e < PER / 2; ++e) sc[PER / 2 * tid + e] = c[2 * e] | (c[2 * e + 1] << 16);
  if (tid == kSampleThreads - 1) so[kSelectBins] = run;
  __syncthreads();
  uint32_t* yk = ykeys + base;
#pragma unroll
  for (int i = 0; i < kSampleItems; ++i) {
    const int64_t s = base + static_cast<int64_t>(i) * kSampleThreads + tid;
    if (s < K) yk[h[key[i] >> 21] + slot[i]] = key[i];
  }
}

int sample_blocks(int64_t K) { return static_cast<int>((K + kSampleBlock - 1) / kSampleBlock); }

hipError_t launch_sample(const float* r, int64_t n, NoiseSrc noise, double t, const int32_t* idx,
                         int64_t K, uint32_t* ykeys, uint32_t* soffs, uint32_t* scnt, uint32_t* zero,
                         int64_t zero_words, hipStream_t s) {
  { ProfScope ps_("sample", s);
  hipLaunchKernelGGL(sample_kernel, dim3(static_cast<unsigned>(sample_blocks(K))),
                     dim3(kSampleThreads), 0, s, r, n, noise.table, noise.seed, t, idx, K, ykeys,
                     soffs, scnt, zero, zero_words); }
  return hipGetLastError();
}

// The draws the sample takes when it is given no table.
__global__ __launch_bounds__(256) void noise_table_kernel(uint64_t seed, int64_t K, double t,
                                                          float* __restrict__ out) {
  const int64_t s = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (s < K) out[s] = counter_laplace(seed, s, t);
}

hipError_t launch_noise_table(uint64_t seed, int64_t K, double t, float* out, hipStream_t s) {
  { ProfScope ps_("noise_table", s);
  hipLaunchKernelGGL(noise_table_kernel, dim3(static_cast<unsigned>((K + 255) / 256)), dim3(256),
                     0, s, seed, K, t, out); }
  return hipGetLastError();
}

// ----------------------------------------------------------------- select --
namespace {

// 1-based rank `rank` in the histogram h (nb bins in LDS, nb / kSelThreads
// consecutive bins per thread): writes (bin, rank inside the bin).  Ends
// with a barrier.
__device__ void find_bin(const uint32_t* h, int nb, uint32_t rank, uint32_t* wsum, int* bin_out,
                         uint32_t* rank_out) {
  const int tid = threadIdx.x;
  const int per = nb / kSelThreads;
  uint32_t loc = 0;
  for (int q = 0; q < per; ++q) loc += h[tid * per + q];
  uint32_t incl = wave_incl_add<uint32_t>(loc);
  const int lane = lane_id();
  const int wid = tid / kWave;
  if (lane == kWave - 1) wsum[wid] = incl;
  __syncthreads();
  uint32_t base = 0;
#pragma unroll
  for (int w = 0; w < kSelThreads / kWave; ++w) {
    const uint32_t x = wsum[w];
    base += w < wid ? x : 0u;
  }
  uint32_t c = base + incl - loc;   // exclusive count before my first bin
  for (int q = 0; q < per; ++q) {
    const uint32_t v = h[tid * per + q];
    if (c < rank && rank <= c + v) {
      *bin_out = tid * per + q;
      *rank_out = rank - c;
    }
    c += v;
  }
  __syncthreads();
}

constexpr int kCand = 16384;   // candidates per target kept in LDS (64 KB)
constexpr int kFewCand = 256;   // a bin this small is ranked directly

// Histogram (into h, nb bins) of (key >> lo) & mask over the keys whose
// bits above `hi` equal `prefix`.
__device__ void prefix_hist(const uint32_t* keys, int64_t count, int hi, uint32_t prefix, int lo,
                            uint32_t mask, int nb, uint32_t* h) {
  for (int e = threadIdx.x; e < nb; e += kSelThreads) h[e] = 0u;
  __syncthreads();
  for (int64_t i = threadIdx.x; i < count; i += kSelThreads) {
    const uint32_t key = keys[i];
    if ((key >> hi) == prefix) atomicAdd(&h[(key >> lo) & mask], 1u);
  }
  __syncthreads();
}
}  // namespace

// One workgroup.  Targets are 1-based ranks among the K sample keys; a rank
// outside 1..K gives -inf (below) or +inf (above).  Level 1 (top 11 bits)
// locates each target's group of bins from the sample blocks' group counts,
// then its bin from the bin counts of that group only.  A bin of at most
// kFewCand keys is gathered into LDS in any order and its key of the target
// rank found by counting; otherwise the bin's keys are fetched from every block's region
// (only that bin) into LDS, where bits 10..20 and 0..9 are resolved, and a
// bin too large for LDS is resolved by passes over all keys in memory.
__global__ __launch_bounds__(kSelThreads) void select_kernel(const uint32_t* __restrict__ ykeys,
                                                             int64_t K,
                                                             const uint32_t* __restrict__ soffs,
                                                             const uint32_t* __restrict__ scnt,
                                                             int nsb, int64_t j, int64_t l,
                                                             SelectRec* __restrict__ out) {
  __shared__ uint32_t hc[kSelectGroups];   // group counts over all blocks
  __shared__ uint32_t hf[2][kSelectBins / kSelectGroups];   // bin counts of each target's group
  __shared__ int grp_s[2], pre_s[2];
  __shared__ uint32_t grank_s[2], rk_s[2], tot_s[2];
  __shared__ uint32_t h[kSelectBins];
  __shared__ uint32_t h2[kSelectBins];   // the level-2 histogram, kept for the other target
  __shared__ uint32_t wsum[kSelThreads / kWave];
  __shared__ int bin_s;
  __shared__ uint32_t rank_s;
  __shared__ uint32_t ncand_s;
  __shared__ uint32_t key_s;
  __shared__ __align__(16) uint32_t cand[kCand];
  __shared__ uint32_t bst[kSelThreads];    // per sample block: start of the bin in its region
  __shared__ uint32_t bpre[kSelThreads + 1];   // exclusive prefix of the bin's counts over blocks
  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wid = tid / kWave;
  const int64_t tgt[2] = {j, l};
  bool live[2];
  uint32_t key_out[2] = {0u, 0u};
  for (int q = 0; q < 2; ++q) live[q] = (tgt[q] >= 1 && tgt[q] <= K);

  // 1. each live target's bin and its rank inside the bin: the group counts
  //    summed over the sample blocks locate the group, then the bin counts
  //    of that group only
  {
    constexpr int GB = kSelectBins / kSelectGroups;   // bins per group
    static_assert(kSelectGroups == kWave && GB <= kWave && GB % 2 == 0, "one lane per group or bin");
    if (tid < kSelectGroups) hc[tid] = 0u;
    if (tid < 2 * GB) hf[tid / GB][tid % GB] = 0u;
    __syncthreads();
    {
      // eight blocks' counts per thread in flight at a time
      constexpr int BS = kSelThreads / kSelectGroups;   // blocks per sweep
      const int gi = tid % kSelectGroups;
      uint32_t sum = 0u;
      for (int b0 = tid / kSelectGroups; b0 < nsb; b0 += 8 * BS) {
        uint32_t v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int b = b0 + u * BS;
          v[u] = b < nsb ? scnt[static_cast<int64_t>(b) * kSampleCntWords + kSelectBins / 2 + gi] : 0u;
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) sum += v[u];
      }
      if (sum) atomicAdd(&hc[gi], sum);
    }
    __syncthreads();
    if (wid == 0) {
      const uint32_t v = hc[lane];
      const uint32_t incl = wave_incl_add<uint32_t>(v);
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        const uint32_t t = static_cast<uint32_t>(live[q] ? tgt[q] : 1);
        if (incl - v < t && t <= incl) {
          grp_s[q] = lane;
          grank_s[q] = t - (incl - v);
        }
      }
    }
    __syncthreads();
    {
      // GB / 2 packed words of the group per block, both targets at once
      constexpr int WPG = GB / 2;
      constexpr int BS = kSelThreads / WPG;   // blocks per sweep
      const int wi = tid % WPG;
      uint32_t lo[2] = {0u, 0u}, hi[2] = {0u, 0u};
      for (int b0 = tid / WPG; b0 < nsb; b0 += 4 * BS) {
        uint32_t wv[4][2];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int b = b0 + u * BS;
          const uint32_t* sc = scnt + static_cast<int64_t>(b < nsb ? b : 0) * kSampleCntWords;
#pragma unroll
          for (int q = 0; q < 2; ++q) wv[u][q] = (b < nsb && live[q]) ? sc[grp_s[q] * WPG + wi] : 0u;
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
#pragma unroll
          for (int q = 0; q < 2; ++q) {
            lo[q] += wv[u][q] & 0xffffu;
            hi[q] += wv[u][q] >> 16;
          }
        }
      }
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        if (lo[q]) atomicAdd(&hf[q][2 * wi], lo[q]);
        if (hi[q]) atomicAdd(&hf[q][2 * wi + 1], hi[q]);
      }
    }
    __syncthreads();
    if (wid == 0) {
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        if (!live[q]) continue;
        const uint32_t v = lane < GB ? hf[q][lane] : 0u;
        const uint32_t incl = wave_incl_add<uint32_t>(v);
        const uint32_t t = grank_s[q];
        if (lane < GB && incl - v < t && t <= incl) {
          pre_s[q] = grp_s[q] * GB + lane;
          rk_s[q] = t - (incl - v);
          tot_s[q] = v;
        }
      }
    }
    __syncthreads();
  }

  // The two targets often share their level-1 bin (and sometimes their
  // level-2 bin): the bin's keys in LDS and the histograms of the first
  // target are kept for the second (which ones: uniform across threads).
  // In the paper's setting at n = 1e8 (bins of thousands of sample keys)
  // this took the select from 25.4 to 20.5 us.
  int64_t cand_pre = -1, h2_pre = -1, h3_pre = -1;
  for (int q = 0; q < 2; ++q) {
    if (!live[q]) continue;   // the same in every thread
    const uint32_t pre = static_cast<uint32_t>(pre_s[q]);
    const uint32_t rk = rk_s[q];
    const uint32_t total = tot_s[q];
    const uint32_t* src = ykeys;
    int64_t count = K;
    if (total <= static_cast<uint32_t>(kFewCand)) {
      cand_pre = -1;   // cand is overwritten below
      // 2'. a small bin: its keys from every block's region in any order,
      //     then the key of rank rk among them by counting (ties share a
      //     value, so any holder of the rank may write it)
      if (tid == 0) ncand_s = 0u;
      // tpb threads per sample block (a power of two), each taking every
      // tpb-th key of the block's part of the bin
      int tpb = kSelThreads;
      while (tpb > 1 && tpb * nsb > kSelThreads) tpb >>= 1;
      __syncthreads();
      for (int b = tid / tpb; b < nsb; b += kSelThreads / tpb) {
        const uint32_t* so = soffs + static_cast<int64_t>(b) * (kSelectBins + 1);
        const uint32_t st = so[pre];
        const uint32_t cnt = so[pre + 1] - st;
        const uint32_t* yk = ykeys + static_cast<int64_t>(b) * kSampleBlock + st;
        for (uint32_t e = static_cast<uint32_t>(tid % tpb); e < cnt; e += static_cast<uint32_t>(tpb)) {
          const uint32_t key = yk[e];
          const uint32_t at = atomicAdd(&ncand_s, 1u);
          if (at < static_cast<uint32_t>(kFewCand)) cand[at] = key;
        }
      }
      __syncthreads();
      {
        // tpc adjacent threads per candidate, each counting a slice of the
        // candidates (a multiple of 4, read four at a time; slots past
        // `total` never count), joined across the candidate's threads
        int tpc = kWave / 4;
        while (tpc > 1 && tpc * static_cast<int>(total) > kSelThreads) tpc >>= 1;
        const int slice = ((static_cast<int>(total) + tpc - 1) / tpc + 3) & ~3;
        const int ci = tid / tpc;
        const int part = tid % tpc;
        const uint32_t x = cand[ci < static_cast<int>(total) ? ci : 0];
        uint32_t below = 0u, same = 0u;
        for (int e0 = part * slice; e0 < (part + 1) * slice; e0 += 4) {
          const uint4 y4 = *reinterpret_cast<const uint4*>(&cand[e0]);
          const uint32_t y[4] = {y4.x, y4.y, y4.z, y4.w};
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const bool in = e0 + u < static_cast<int>(total);
            below += (in && y[u] < x) ? 1u : 0u;
            same += (in && y[u] == x) ? 1u : 0u;
          }
        }
        for (int o = 1; o < tpc; o <<= 1) {
          below += __shfl_xor(below, o, kWave);
          same += __shfl_xor(same, o, kWave);
        }
        if (ci < static_cast<int>(total) && part == 0 && below < rk && rk <= below + same) key_s = x;
      }
      __syncthreads();
      key_out[q] = key_s;
      __syncthreads();
      continue;
    }
    if (total <= static_cast<uint32_t>(kCand) && cand_pre != static_cast<int64_t>(pre)) {
      // 2. the bin's keys from every block's region, in block order
      cand_pre = pre;
      uint32_t run = 0u;   // keys fetched so far (same in every thread)
      for (int b0 = 0; b0 < nsb; b0 += kSelThreads) {
        const int b = b0 + tid;
        uint32_t st = 0u, cnt = 0u;
        if (b < nsb) {
          const uint32_t* so = soffs + static_cast<int64_t>(b) * (kSelectBins + 1);
          st = so[pre];
          cnt = so[pre + 1] - st;
        }
        uint32_t incl = wave_incl_add<uint32_t>(cnt);
        if (lane == kWave - 1) wsum[wid] = incl;
        __syncthreads();
        uint32_t wb = 0u, all = 0u;
        for (int w = 0; w < kSelThreads / kWave; ++w) {
          if (w < wid) wb += wsum[w];
          all += wsum[w];
        }
        bst[tid] = st;
        bpre[tid] = wb + incl - cnt;
        if (tid == 0) bpre[kSelThreads] = all;
        __syncthreads();
        const int nb = nsb - b0 < kSelThreads ? nsb - b0 : kSelThreads;
        for (uint32_t e = tid; e < all; e += kSelThreads) {
          int lo = 0, hi = nb;   // bpre[lo] <= e < bpre[hi]
          while (hi - lo > 1) {
            const int mid = (lo + hi) >> 1;
            if (bpre[mid] <= e) lo = mid; else hi = mid;
          }
          cand[run + e] = ykeys[static_cast<int64_t>(b0 + lo) * kSampleBlock + bst[lo] + (e - bpre[lo])];
        }
        run += all;
        __syncthreads();
      }
    }
    if (total <= static_cast<uint32_t>(kCand)) {
      src = cand;
      count = total;
    }
    // 3. bits 10..20, then 0..9, of the bin's keys
    if (h2_pre != static_cast<int64_t>(pre)) {
      prefix_hist(src, count, 21, pre, 10, 2047u, 2048, h2);
      h2_pre = pre;
    }
    find_bin(h2, 2048, rk, wsum, &bin_s, &rank_s);
    const uint32_t pre2 = (pre << 11) | static_cast<uint32_t>(bin_s);
    const uint32_t rk2 = rank_s;
    __syncthreads();
    if (h3_pre != static_cast<int64_t>(pre2)) {
      prefix_hist(src, count, 10, pre2, 0, 1023u, 1024, h);
      h3_pre = pre2;
    }
    find_bin(h, 1024, rk2, wsum, &bin_s, &rank_s);
    key_out[q] = (pre2 << 10) | static_cast<uint32_t>(bin_s);
    __syncthreads();
  }
  if (tid == 0) {
    SelectRec rec;
    rec.keyL = key_out[0];
    rec.keyR = key_out[1];
    rec.aL = live[0] ? asc_key_float(key_out[0]) : (tgt[0] < 1 ? -INFINITY : INFINITY);
    rec.aR = live[1] ? asc_key_float(key_out[1]) : (tgt[1] < 1 ? -INFINITY : INFINITY);
    *out = rec;
  }
}

hipError_t launch_select(const uint32_t* ykeys, int64_t K, const uint32_t* soffs,
                         const uint32_t* scnt, int64_t j, int64_t l, SelectRec* out,
                         hipStream_t s) {
  { ProfScope ps_("select", s);
  hipLaunchKernelGGL(select_kernel, dim3(1), dim3(kSelThreads), 0, s, ykeys, K, soffs, scnt,
                     sample_blocks(K), j, l, out); }
  return hipGetLastError();
}

// -------------------------------------------------------------- partition --
int partition_blocks(int64_t n, int64_t* chunk) {
  // up to 4096 blocks; a block's chunk is a multiple of four writer tiles so
  // that each wave owns a contiguous quarter of it made of whole tiles
  constexpr int64_t q = PW * kBandTile;
  int64_t c = (n + kPartMaxBlocks - 1) / kPartMaxBlocks;
  c = (c + q - 1) / q * q;
  if (c < q) c = q;
  *chunk = c;
  return static_cast<int>((n + c - 1) / c);
}

namespace {

struct PartState {
  double TL, TR;
  int64_t nL, nR;
  int32_t nM;   // M count of this wave (uniform across the wave)
  float mmin, mmax;
  int32_t nB;   // band members of this wave (uniform across the wave)
};

// Where a wave stages its band members and its bits of r >= hi.  Both go
// to LDS while the wave streams (a global store inside the loop would make
// every wait for the next loads also wait for the store) and are copied out
// once at the end.
constexpr int kOnesWaveWords = static_cast<int>(kBandMaxChunk / 4 / 32);   // 512

struct BandWave {
  BandEntry* sbuf;   // LDS, cap entries
  uint32_t* sones;   // LDS, kOnesWaveWords words: bit i of the wave's range
  int cap;
  bool stage;        // false when the block's range is too long for the band passes
  float lo, hi;      // band: lo <= r < hi
  int64_t w0;        // first score of the wave's range (a multiple of 256)
};

// Classify 4 consecutive scores of one lane (the slow path of the gather);
// M members are reported in index order within the wave (lane-major, then
// element).
template <typename Emit>
__device__ __forceinline__ void classify4(const float (&v)[4], const bool (&ok)[4], int64_t i0,
                                          float aL, float aR, PartState& st, Emit&& emit) {
  bool inM[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) inM[e] = ok[e] && !(v[e] < aL) && !(v[e] >= aR);
  uint32_t before = 0;
  uint32_t total = 0;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const uint64_t bal = __ballot(inM[e]);
    before += lanes_below(bal);
    total += static_cast<uint32_t>(__popcll(bal));
  }
  uint32_t idx = before;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    if (inM[e]) {
      emit(st.nM + idx, v[e], i0 + e);
      ++idx;
    }
  }
  st.nM += total;
}

constexpr int kWaveStage = kPartStageCap / PW;   // M entries staged per wave

// Per-wave pass over [w0, w1): tails in float32 over one float4 and float64
// across, R counted only when a_R is finite (HAS_R), band members and M
// members (a subset of the band) staged in index order, and with a finite
// a_R one bit per score for r >= hi.  L is not counted:
// n_L = scores - n_M - n_R.
// With STAGE the L tail is summed once at the end from the wave's staged
// band (its members below a_L are the only nonzero terms).  Once the list
// could not take another step's members (a band as wide as the scores, when
// t is large against their spread) the wave stops staging the band and
// forms each later member's term as it is met; its block then takes the
// dense passes.  Without STAGE (a range too long to stage) every term is
// formed as it is met.
// tb: lane q ends with the band members met before tile q of the range (the
// range starts on a tile boundary; tiles are kBandTile scores).
template <bool HAS_R, bool STAGE>
__device__ __forceinline__ void partition_range(const float* __restrict__ r, int64_t w0, int64_t w1,
                                                bool vec, float aL, float aR, float c2f,
                                                float* sv, int32_t* si, const BandWave& bw,
                                                PartState& st, int32_t& tb) {
  const int lane = lane_id();
  auto tile_start = [&](int64_t at) {
    if (lane == static_cast<int>((at - w0) / kBandTile)) tb = static_cast<int32_t>(st.nB);
  };
  // staging stopped (uniform across the wave); the list then holds the
  // members met before, `listed` of them
  bool spill = !STAGE;
  int32_t listed = 0;
  // the lower tail's terms of a step's band members, formed directly:
  // below the band's lower edge (a_L - 105 t) a term e^{(r - a_L)/t} is
  // exactly 0 in float32
  auto direct_tl = [&](const float (&v)[4], const bool (&ok)[4]) {
    float tl = 0.0f;
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (ok[e] && !(v[e] < bw.lo) && v[e] < aL) tl += exp2_fast((v[e] - aL) * c2f);
    st.TL += static_cast<double>(tl);
  };
  // it: first score of this wave's 256-score step (a multiple of 256).
  // DIRECT: the band is not staged, each member's lower-tail term is formed
  // as it is met.  The wave's list is then incomplete and its block takes
  // the dense passes, which read neither the band count nor the bits of
  // r >= hi: DIRECT leaves nB as it was when staging stopped (above the
  // list's capacity) and forms no bits.
  auto one = [&](auto direct, const float (&v)[4], const bool (&ok)[4], int64_t it) {
    constexpr bool DIRECT = decltype(direct)::value;
    const int64_t i0 = it + 4 * lane;
    // membership as lane masks: a comparison is its own ballot
    bool inB[4], inM[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      if constexpr (HAS_R) {
        inB[e] = ok[e] && !(v[e] < bw.lo) && !(v[e] >= bw.hi);
        inM[e] = ok[e] && !(v[e] < aL) && !(v[e] >= aR);
      } else {
        inB[e] = ok[e] && !(v[e] < bw.lo);
        inM[e] = ok[e] && !(v[e] < aL);
      }
    }
    // M members of the step: staged in index order, with the range of M
    auto stage_m = [&](float x, int64_t i, uint32_t at) {
      st.mmin = fminf(st.mmin, x);
      st.mmax = fmaxf(st.mmax, x);
      if (at < static_cast<uint32_t>(kWaveStage)) {
        sv[at] = x;
        si[at] = static_cast<int32_t>(i);
      }
    };
    auto stage_all_m = [&]() {
      if (__ballot(inM[0] || inM[1] || inM[2] || inM[3])) {
        uint32_t before = 0, total = 0;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const uint64_t bal = __ballot(inM[e]);
          before += lanes_below(bal);
          total += static_cast<uint32_t>(__popcll(bal));
        }
        uint32_t at = static_cast<uint32_t>(st.nM) + before;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          if (inM[e]) {
            stage_m(v[e], i0 + e, at);
            ++at;
          }
        }
        st.nM += total;
      }
    };
    // formed directly with both tails: a score lies in at most one of them,
    // so one exponential per score serves both (the lower tail's below)
    float ex[4];
    if constexpr (DIRECT && HAS_R) {
#pragma unroll
      for (int e = 0; e < 4; ++e) ex[e] = exp2_fast((v[e] < aL ? v[e] - aL : aR - v[e]) * c2f);
    }
    if constexpr (HAS_R) {
      float tr = 0.0f;
      uint32_t ob = 0;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const bool R = v[e] >= aR;
        if constexpr (DIRECT)
          tr += (ok[e] && R) ? ex[e] : 0.0f;
        else
          tr += (ok[e] && R) ? exp2_fast((aR - v[e]) * c2f) : 0.0f;
        st.nR += (ok[e] && R) ? 1 : 0;
        if constexpr (!DIRECT)
          if (ok[e] && v[e] >= bw.hi) ob |= 1u << e;
      }
      st.TR += static_cast<double>(tr);
      if constexpr (!DIRECT) {
        // 8 lanes hold the 32 bits of one word
        uint32_t x = ob << (4 * (lane & 7));
        x |= __shfl_xor(x, 1, kWave);
        x |= __shfl_xor(x, 2, kWave);
        x |= __shfl_xor(x, 4, kWave);
        if (bw.stage && (lane & 7) == 0) bw.sones[((it - bw.w0) >> 5) + (lane >> 3)] = x;
      }
    }
    if constexpr (DIRECT) {
      // a lower-tail term lies in the band (lo <= r < a_L <= hi)
      if constexpr (HAS_R) {
        float tl = 0.0f;
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (ok[e] && !(v[e] < bw.lo) && v[e] < aL) tl += ex[e];
        st.TL += static_cast<double>(tl);
      } else {
        direct_tl(v, ok);
      }
      stage_all_m();
      return;
    }
    // band members take slots in index order from the masks and the wave's
    // running count.  M lies inside the band (lo <= a_L, hi >= a_R, both
    // rounded outwards), so a step without band members has no M members
    // either, and a lane's one band member is its only possible M member.
    uint64_t bm[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) bm[e] = __ballot(inB[e]);
    const uint64_t any = bm[0] | bm[1] | bm[2] | bm[3];
    if (any) {
      const uint32_t nb0 = static_cast<uint32_t>(st.nB);   // uniform across the wave
      const uint32_t cap = static_cast<uint32_t>(bw.cap);
      const uint64_t two = (bm[0] & (bm[1] | bm[2] | bm[3])) | (bm[1] & (bm[2] | bm[3])) |
                           (bm[2] & bm[3]);   // lanes with two or more members
      if (two == 0ull) {
        // each lane holds at most one member: its slot is its rank among
        // the lanes that hold one (scalar mask work, a few vector ops)
        const bool mine = inB[0] || inB[1] || inB[2] || inB[3];
        const int e0 = inB[0] ? 0 : (inB[1] ? 1 : (inB[2] ? 2 : 3));
        const float x0 = inB[0] ? v[0] : (inB[1] ? v[1] : (inB[2] ? v[2] : v[3]));
        if (mine) {
          const uint32_t slot = nb0 + lanes_below(any);
          if (slot < cap) {
            BandEntry en;
            en.idx = static_cast<int32_t>(i0 + e0);
            en.bits = __float_as_uint(x0);
            bw.sbuf[slot] = en;
          }
        }
        st.nB = nb0 + static_cast<uint32_t>(__popcll(any));
        bool m0 = mine && !(x0 < aL);
        if constexpr (HAS_R) m0 = m0 && !(x0 >= aR);
        const uint64_t mm = __ballot(m0);
        if (mm) {   // rare: some lane holds an M member
          if (m0) stage_m(x0, i0 + e0, static_cast<uint32_t>(st.nM) + lanes_below(mm));
          st.nM += static_cast<uint32_t>(__popcll(mm));
        }
      } else {
        // a lane's members follow those of the lanes below it
        uint32_t slot = nb0, tot = 0;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          slot += lanes_below(bm[e]);
          tot += static_cast<uint32_t>(__popcll(bm[e]));
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          if (inB[e]) {
            if (slot < cap) {
              BandEntry en;
              en.idx = static_cast<int32_t>(i0 + e);
              en.bits = __float_as_uint(v[e]);
              bw.sbuf[slot] = en;
            }
            ++slot;
          }
        }
        st.nB = nb0 + tot;
        stage_all_m();
      }
    }
  };
  constexpr int U = 4;   // float4 loads per lane per batch, two batches in flight
  static_assert(U * 256 == kBandTile, "a batch of the vector loop is one tile");
  int64_t it = w0;
  if (vec && it + U * 256 <= w1) {
    // two buffers taking turns, so that no registers are copied per batch.
    // The loads are unconditional (past the last batch every lane reads the
    // range's first float4 again, one line per wave): a conditional load
    // would make the compiler merge the old and new values with copies that
    // wait for the load right away.
    auto load = [&](float4 (&q)[U], int64_t at, bool real) {
#pragma unroll
      for (int u = 0; u < U; ++u)
        q[u] = load_stream4(real ? r + at + u * 256 + 4 * lane : r + w0);
    };
    // one batch (tile).  A staged batch that overflows the list keeps its M
    // and has its lower-tail terms formed again directly; the wave then
    // stops staging (returns true)
    auto run = [&](auto direct, const float4 (&q)[U], int64_t at) -> bool {
      constexpr bool DIRECT = decltype(direct)::value;
      const bool ok[4] = {true, true, true, true};
      const int32_t nb_start = st.nB;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const float v[4] = {q[u].x, q[u].y, q[u].z, q[u].w};
        one(direct, v, ok, at + u * 256);
      }
      if constexpr (!DIRECT) {
        if (st.nB > bw.cap) {
          spill = true;
          listed = nb_start;
#pragma unroll
          for (int u = 0; u < U; ++u) {
            const float v[4] = {q[u].x, q[u].y, q[u].z, q[u].w};
            direct_tl(v, ok);
          }
          return true;
        }
      }
      return false;
    };
    // the batches from `from` on, two buffers taking turns so that no
    // registers are copied per batch; returns where it stopped (after the
    // last whole batch, or after the batch where staging stopped).  The
    // staged and the direct passes are separate loops, so that neither
    // carries the other's registers
    // the start of the wave's first batch says its list will overflow: the
    // band members among the batch's first 256 scores, times U, exceed the
    // list, or, counted over all the wave's batches at that rate, twice the
    // list.  A wrong guess (a row whose band members bunch at the start of
    // a wave) only costs speed: the block takes the dense passes, which are
    // exact for every score.
    auto crowded = [&](const float4 (&q)[U]) -> bool {
      const float v[4] = {q[0].x, q[0].y, q[0].z, q[0].w};
      uint32_t c = 0;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        bool in = !(v[e] < bw.lo);
        if constexpr (HAS_R) in = in && !(v[e] >= bw.hi);
        c += static_cast<uint32_t>(__popcll(__ballot(in)));
      }
      c *= U;
      const int64_t nb = (w1 - w0) / (U * 256);
      const int64_t cap = bw.cap;
      return c > cap || static_cast<int64_t>(c) * nb > 2 * cap;
    };
    auto stream = [&](auto direct, int64_t from) -> int64_t {
      constexpr bool DIRECT = decltype(direct)::value;
      int64_t at = from;
      if (at + U * 256 > w1) return at;
      float4 qa[U], qb[U];
      load(qa, at, true);
      if constexpr (!DIRECT) {
        if (at == w0 && crowded(qa)) {
          // no list: every batch, this one included (read again, from
          // the L2 as a rule), is formed by the direct loop
          spill = true;
          listed = 0;
          return at;
        }
      }
      while (true) {
        const int64_t ca = at;
        at += U * 256;
        const bool more_a = at + U * 256 <= w1;
        load(qb, at, more_a);
        tile_start(ca);
        if (run(direct, qa, ca) || !more_a) return at;
        const int64_t cb = at;
        at += U * 256;
        const bool more_b = at + U * 256 <= w1;
        load(qa, at, more_b);
        tile_start(cb);
        if (run(direct, qb, cb) || !more_b) return at;
      }
    };
    if (!spill) it = stream(std::false_type{}, it);
    if (spill) it = stream(std::true_type{}, it);
  }
  for (; it < w1; it += 256) {
    if (((it - w0) & (kBandTile - 1)) == 0) tile_start(it);
    const int64_t i0 = it + 4 * lane;
    float v[4];
    bool ok[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      ok[e] = (i0 + e) < w1;
      v[e] = ok[e] ? r[i0 + e] : 0.0f;
    }
    if (spill) {
      one(std::true_type{}, v, ok, it);
    } else {
      const int32_t nb_start = st.nB;
      one(std::false_type{}, v, ok, it);
      if (st.nB > bw.cap) {
        spill = true;
        listed = nb_start;
        direct_tl(v, ok);
      }
    }
  }
  if constexpr (STAGE) {
    // the L tail of the listed members: e^{(r - a_L)/t} over the band
    // members below a_L, each term in float32 and summed per lane in float64
    const int nl = static_cast<int>(spill ? listed : st.nB);   // <= bw.cap
    double tl = 0.0;
    for (int q = lane; q < nl; q += kWave) {
      const float x = __uint_as_float(bw.sbuf[q].bits);
      if (x < aL) tl += static_cast<double>(exp2_fast((x - aL) * c2f));
    }
    st.TL += tl;
    // an incomplete list reports more members than it can hold, so that
    // the block takes the dense passes
    if (spill && st.nB <= bw.cap) st.nB = bw.cap + 1;
  }
}

}  // namespace

// Totals over the partition blocks in a fixed order and the exclusive
// prefix of their M counts (each block's offset into M), TOT_T threads.
// Records are read coalesced (all loads of a thread independent), the M
// counts go through LDS (`nm`, kPartMaxBlocks words) for the prefix.
constexpr int TOT_T = 1024;   // threads of the totals kernel
constexpr int TOT_W = TOT_T / kWave;

__device__ void partition_totals_block(const PartBlock* __restrict__ blk, int nblocks, float aL,
                                       float aR, int64_t* __restrict__ offsets,
                                       PartTotals* __restrict__ tot, int32_t* nm) {
  constexpr int Q = kPartMaxBlocks / TOT_T;
  constexpr int PT = TOT_T;
  constexpr int PW = TOT_W;
  __shared__ double rd[2][PW];
  __shared__ int64_t ri[5][PW];
  __shared__ float rf[2][PW];
  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wid = tid / kWave;
  double TL = 0.0, TR = 0.0;
  int64_t nL = 0, nR = 0, ov = 0, nd = 0;
  float mn = INFINITY, mx = -INFINITY;
#pragma unroll
  for (int q = 0; q < Q; ++q) {
    const int b = tid + PT * q;
    if (b < nblocks) {
      const PartBlock rec = blk[b];
      TL += rec.TL;
      TR += rec.TR;
      nL += rec.nL;
      nR += rec.nR;
      ov += rec.overflow;
      nd += rec.band_dense;
      mn = fminf(mn, rec.mmin);
      mx = fmaxf(mx, rec.mmax);
      nm[b] = static_cast<int32_t>(rec.nM);
    }
  }
  __syncthreads();
  // prefix of the M counts: thread tid owns blocks [Q tid, Q tid + Q)
  int64_t loc = 0;
#pragma unroll
  for (int q = 0; q < Q; ++q) {
    const int b = Q * tid + q;
    loc += (b < nblocks) ? nm[b] : 0;
  }
  int64_t incl = wave_incl_add<int64_t>(loc);
  TL = wave_sum(TL);
  TR = wave_sum(TR);
  const int64_t sL = wave_sum(nL), sR = wave_sum(nR), sO = wave_sum(ov), sD = wave_sum(nd);
mn = wave_min(mn, INFINITY);
mx = wave_max(mx, -INFINITY);
  if (lane == kWave - 1) ri[3][wid] = incl;
  if (lane == 0) {
    rd[0][wid] = TL;
    rd[1][wid] = TR;
    ri[0][wid] = sL;
    ri[1][wid] = sR;
    ri[2][wid] = sO;
    ri[4][wid] = sD;
    rf[0][wid] = mn;
    rf[1][wid] = mx;
  }
  __syncthreads();
  int64_t base = 0, allm = 0;
#pragma unroll
  for (int w = 0; w < PW; ++w) {
    if (w < wid) base += ri[3][w];
    allm += ri[3][w];
  }
  int64_t off = base + incl - loc;
#pragma unroll
  for (int q = 0; q < Q; ++q) {
    const int b = Q * tid + q;
    if (b < nblocks) {
      offsets[b] = off;
      off += nm[b];
    }
  }
  if (tid == 0) {
    PartTotals x;
    double tl = 0.0, tr = 0.0;
    int64_t cl = 0, cr = 0, co = 0, cd = 0;
    float fmn = INFINITY, fmx = -INFINITY;
#pragma unroll
    for (int w = 0; w < PW; ++w) {
      tl += rd[0][w];
      tr += rd[1][w];
      cl += ri[0][w];
      cr += ri[1][w];
      co += ri[2][w];
      cd += ri[4][w];
      fmn = fminf(fmn, rf[0][w]);
      fmx = fmaxf(fmx, rf[1][w]);
    }
    x.TL = tl;
    x.TR = tr;
    x.nL = cl;
    x.nR = cr;
    x.nM = allm;
    x.aL = aL;
    x.aR = aR;
    x.mmin = fmn;
    x.mmax = fmx;
    x.any_block_overflow = co > 0 ? 1 : 0;
    x.dense_blocks = static_cast<int32_t>(cd);
    *tot = x;
  }
}

// One workgroup: the totals of one partition pass.  (A separate launch
// rather than the last block of the pass: making the records of every block
// visible to that block would take a device-scope release per block, which
// writes back the L2 of its XCD.)
__global__ __launch_bounds__(TOT_T) void partition_totals_kernel(const PartBlock* __restrict__ blk,
                                                              int nblocks,
                                                              const SelectRec* __restrict__ sel,
                                                              int use_sel, float aL_arg,
                                                              float aR_arg,
                                                              int64_t* __restrict__ offsets,
                                                              PartTotals* __restrict__ tot) {
  __shared__ int32_t nm[kPartMaxBlocks];
  const float aL = use_sel ? sel->aL : aL_arg;
  const float aR = use_sel ? sel->aR : aR_arg;
  partition_totals_block(blk, nblocks, aL, aR, offsets, tot, nm);
}

// Block b owns [b*chunk, (b+1)*chunk) and wave w the w-th contiguous
// quarter of it, so each wave sees its scores in index order and stages its
// M members in LDS with a wave-private counter; the block then writes them
// to its slot of the global staging area (wave 0's first) and one record of
// tails and counts.
// HAS_R: a_R is finite (the host knows: for the first bracket from the rank
// l <= K, afterwards from the endpoints it passes).  One instance per case
// keeps the common one (a_R infinite) in fewer registers.
template <bool HAS_R>
__global__ __launch_bounds__(PT) void partition_kernel(const float* __restrict__ r, int64_t n,
                                                       const SelectRec* __restrict__ sel,
                                                       int use_sel, float aL_arg, float aR_arg,
                                                       float c2f, int64_t chunk,
                                                       float* __restrict__ stage_v,
                                                       int32_t* __restrict__ stage_i,
                                                       PartBlock* __restrict__ blk, double t,
                                                       BandEntry* __restrict__ bent,
                                                       BandBlock* __restrict__ bblk,
                                                       BandTile* __restrict__ btile, int bcap,
                                                       uint32_t* __restrict__ ones) {
  __shared__ float sv[PW][kWaveStage];
  __shared__ int32_t si[PW][kWaveStage];
  __shared__ BandEntry sband[PW][kBandWaveCapMax];
  __shared__ uint32_t sones[PW][kOnesWaveWords];
  __shared__ double red_d[2][PW];
  __shared__ int64_t red_i[2][PW];
  __shared__ float red_f[2][PW];
  __shared__ int64_t red_b[PW];
  const float aL = use_sel ? sel->aL : aL_arg;
  const float aR = use_sel ? sel->aR : aR_arg;
  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wid = tid / kWave;
  const int64_t b0 = static_cast<int64_t>(blockIdx.x) * chunk;
  const int64_t wq = chunk / PW;
  const int64_t w0 = b0 + wid * wq < n ? b0 + wid * wq : n;
  const int64_t w1 = w0 + wq < n ? w0 + wq : n;
  const bool vec = (reinterpret_cast<uintptr_t>(r) & 15) == 0;
  BandWave bw;
  bw.sbuf = sband[wid];
  bw.sones = sones[wid];
  bw.stage = chunk <= kBandMaxChunk;
  bw.cap = bw.stage ? (bcap < kBandWaveCapMax ? bcap : kBandWaveCapMax) : 0;
  // rounded outwards so that the float comparisons imply the float64 bounds
  bw.lo = __double2float_rd(static_cast<double>(aL) - kBandLowT * t);
  bw.hi = __double2float_ru(static_cast<double>(aR) + kBandHighT * t);
  bw.w0 = w0;
  PartState st{0.0, 0.0, 0, 0, 0, INFINITY, -INFINITY, 0};
  int32_t tb = 0;
  const bool has_r = HAS_R;
  if (bw.stage)
    partition_range<HAS_R, true>(r, w0, w1, vec, aL, aR, c2f, sv[wid], si[wid], bw, st, tb);
  else
    partition_range<HAS_R, false>(r, w0, w1, vec, aL, aR, c2f, sv[wid], si[wid], bw, st, tb);
  // this wave's bits and band list out of LDS
  if (bw.stage) {
    // a wave whose list is incomplete formed no bits once staging stopped;
    // its block takes the dense passes, which do not read them
    if (has_r && st.nB <= bw.cap) {
      const int nw = static_cast<int>((w1 - w0 + 31) / 32);   // <= kOnesWaveWords
      for (int q = lane; q < nw; q += kWave) ones[(w0 >> 5) + q] = bw.sones[q];
    }
    if (st.nB <= bw.cap) {
      BandEntry* out = bent + (static_cast<int64_t>(blockIdx.x) * PW + wid) * bcap;
      for (int q = lane; q < static_cast<int>(st.nB); q += kWave) out[q] = bw.sbuf[q];
    }
  }
  if (lane == 0) {
    bblk[blockIdx.x].cnt[wid] = static_cast<int32_t>(st.nB);
    red_b[wid] = st.nB;
  }

  const double TL = wave_sum(st.TL);
  const double TR = wave_sum(st.TR);
  const int64_t nR = wave_sum(st.nR);
  float mn = st.mmin, mx = st.mmax;
mn = wave_min(mn, INFINITY);
mx = wave_max(mx, -INFINITY);
  if (lane == 0) {
    red_d[0][wid] = TL;
    red_d[1][wid] = TR;
    red_i[0][wid] = nR;
    red_i[1][wid] = st.nM;
    red_f[0][wid] = mn;
    red_f[1][wid] = mx;
  }
  __syncthreads();
  // per tile of this wave's range: its members' place in the lists, or -1
  // when the block's lists are incomplete
  {
    bool bdense = !bw.stage;
#pragma unroll
    for (int w = 0; w < PW; ++w) bdense |= red_b[w] > bcap;
    const int ntw = static_cast<int>((w1 - w0 + kBandTile - 1) / kBandTile);
    const int32_t nb = static_cast<int32_t>(st.nB);
    const int32_t next = __shfl_down(tb, 1, kWave);   // tile q + 1's start
    const int32_t seg = (static_cast<int32_t>(blockIdx.x) * PW + wid) * bcap;
    for (int q = lane; q < ntw; q += kWave) {
      BandTile tr;
      if (bdense) {
        tr.first = 0;
        tr.count = -1;
      } else {
        tr.first = seg + tb;
        tr.count = (q + 1 < ntw ? next : nb) - tb;
      }
      btile[w0 / kBandTile + q] = tr;
    }
  }
  int64_t off = 0, mtot = 0;
  bool over = false;
#pragma unroll
  for (int w = 0; w < PW; ++w) {
    if (w < wid) off += red_i[1][w];
    mtot += red_i[1][w];
    over |= red_i[1][w] > kWaveStage;
  }
  if (!over && st.nM > 0) {
    float* ov = stage_v + static_cast<int64_t>(blockIdx.x) * kPartStageCap;
    int32_t* oi = stage_i + static_cast<int64_t>(blockIdx.x) * kPartStageCap;
    for (int64_t q = lane; q < st.nM; q += kWave) {
      ov[off + q] = sv[wid][q];
      oi[off + q] = si[wid][q];
    }
  }
  if (tid == 0) {
    PartBlock rec;
    double tl = 0.0, tr = 0.0;
    int64_t nr = 0;
#pragma unroll
    for (int w = 0; w < PW; ++w) {
      tl += red_d[0][w];
      tr += red_d[1][w];
      nr += red_i[0][w];
    }
    const int64_t b1 = b0 + chunk < n ? b0 + chunk : n;
    rec.TL = tl;
    rec.TR = tr;
    rec.nR = nr;
    rec.nM = static_cast<int32_t>(mtot);
    rec.nL = (b1 - b0) - mtot - nr;
    float mn2 = INFINITY, mx2 = -INFINITY;
#pragma unroll
    for (int w = 0; w < PW; ++w) {
      mn2 = fminf(mn2, red_f[0][w]);
      mx2 = fmaxf(mx2, red_f[1][w]);
    }
    rec.mmin = mn2;
    rec.mmax = mx2;
    rec.overflow = over ? 1 : 0;
    bool bover = chunk > kBandMaxChunk;
#pragma unroll
    for (int w = 0; w < PW; ++w) bover |= red_b[w] > bcap;
    rec.band_dense = bover ? 1 : 0;
    rec.pad = 0;
    blk[blockIdx.x] = rec;
    bblk[blockIdx.x].dense = bover ? 1 : 0;
  }
}

hipError_t launch_partition(const float* r, int64_t n, const SelectRec* sel, int use_sel, float aL,
                            float aR, bool has_r, double t, int nblocks, int64_t chunk,
                            float* stage_v, int32_t* stage_i, PartBlock* blk, const BandCtx& band,
                            uint32_t* ones, hipStream_t s) {
  if (band.nblocks != nblocks || band.chunk != chunk || nblocks > kPartMaxBlocks)
    return hipErrorInvalidValue;
  const float c2f = static_cast<float>(kLog2e / t);
  { ProfScope ps_("partition", s);
  if (has_r)
    hipLaunchKernelGGL(partition_kernel<true>, dim3(nblocks), dim3(PT), 0, s, r, n, sel, use_sel,
                       aL, aR, c2f, chunk, stage_v, stage_i, blk, t, band.ent, band.blk,
                       band.tiles, band.cap, ones);
  else
    hipLaunchKernelGGL(partition_kernel<false>, dim3(nblocks), dim3(PT), 0, s, r, n, sel, use_sel,
                       aL, aR, c2f, chunk, stage_v, stage_i, blk, t, band.ent, band.blk,
                       band.tiles, band.cap, ones); }
  return hipGetLastError();
}

hipError_t launch_partition_totals(const PartBlock* blk, int nblocks, const SelectRec* sel,
                                   int use_sel, float aL, float aR, int64_t* offsets,
                                   PartTotals* tot, hipStream_t s) {
  { ProfScope ps_("partition_totals", s);
  hipLaunchKernelGGL(partition_totals_kernel, dim3(1), dim3(TOT_T), 0, s, blk, nblocks, sel, use_sel,
                     aL, aR, offsets, tot); }
  return hipGetLastError();
}

int band_wave_cap(int64_t chunk) {
  const int64_t q = chunk / PW;
  return static_cast<int>(q < kBandWaveCapMax ? q : kBandWaveCapMax);
}

namespace {
// Layout of one row's context: header, block records, entries.
struct CtxLayout {
  int nblocks;
  int64_t chunk;
  int cap;
  size_t blk_off, tile_off, ent_off, bytes;
};
CtxLayout ctx_layout(int64_t n) {
  CtxLayout L{};
  L.nblocks = partition_blocks(n, &L.chunk);
  L.cap = band_wave_cap(L.chunk);
  const size_t ntiles = static_cast<size_t>((n + kBandTile - 1) / kBandTile);
  L.blk_off = 256;
  L.tile_off = L.blk_off + (static_cast<size_t>(L.nblocks) * sizeof(BandBlock) + 255) / 256 * 256;
  L.ent_off = L.tile_off + (ntiles * sizeof(BandTile) + 255) / 256 * 256;
  L.bytes = (L.ent_off + static_cast<size_t>(L.nblocks) * PW * L.cap * sizeof(BandEntry) + 255) /
            256 * 256;
  return L;
}
}  // namespace

size_t band_ctx_bytes(int64_t n) { return ctx_layout(n).bytes; }

BandCtx band_ctx_view(void* base, int64_t n) {
  const CtxLayout L = ctx_layout(n);
  BandCtx v{};
  v.nblocks = L.nblocks;
  v.chunk = L.chunk;
  v.cap = L.cap;
  char* b = static_cast<char*>(base);
  v.hdr = reinterpret_cast<CtxHeader*>(b);
  v.blk = b ? reinterpret_cast<BandBlock*>(b + L.blk_off) : nullptr;
  v.tiles = b ? reinterpret_cast<BandTile*>(b + L.tile_off) : nullptr;
  v.ent = b ? reinterpret_cast<BandEntry*>(b + L.ent_off) : nullptr;
  return v;
}

// Copy each block's staged M to M[offset..]; a block whose staging
// overflowed re-reads its chunk (one wave, in index order).  Nothing is
// written when M exceeds the capacity (the host then falls back).
__global__ __launch_bounds__(PT) void gather_kernel(const float* __restrict__ r, int64_t n,
                                                    const PartTotals* __restrict__ tot,
                                                    const PartBlock* __restrict__ blk,
                                                    const int64_t* __restrict__ offsets,
                                                    int64_t chunk, const float* __restrict__ stage_v,
                                                    const int32_t* __restrict__ stage_i,
                                                    int64_t m_capacity, uint32_t* __restrict__ m_keys,
                                                    int32_t* __restrict__ m_idx) {
  if (tot->nM > m_capacity) return;
  const int b = blockIdx.x;
  const int64_t cnt = blk[b].nM;
  if (cnt == 0) return;
  const int64_t off = offsets[b];
  const int tid = threadIdx.x;
  if (!blk[b].overflow) {
    const float* sv = stage_v + static_cast<int64_t>(b) * kPartStageCap;
    const int32_t* si = stage_i + static_cast<int64_t>(b) * kPartStageCap;
    for (int64_t q = tid; q < cnt; q += PT) {
      m_keys[off + q] = desc_key(sv[q]);
      m_idx[off + q] = si[q];
    }
    return;
  }
  if (tid >= kWave) return;
  const float aL = tot->aL;
  const float aR = tot->aR;
  const int lane = lane_id();
  const int64_t b0 = static_cast<int64_t>(b) * chunk;
  int64_t b1 = b0 + chunk;
  if (b1 > n) b1 = n;
  PartState st{0.0, 0.0, 0, 0, 0, INFINITY, -INFINITY, 0};
  auto put = [&](int64_t slot, float v, int64_t gi) {
    m_keys[off + slot] = desc_key(v);
    m_idx[off + slot] = static_cast<int32_t>(gi);
  };
  // walk the chunk in index order with one wave, 256 scores at a time
  for (int64_t it = b0; it < b1; it += 256) {
    const int64_t i0 = it + 4 * lane;
    float v[4];
    bool ok[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      ok[e] = (i0 + e) < b1;
      v[e] = ok[e] ? r[i0 + e] : 0.0f;
    }
    classify4(v, ok, i0, aL, aR, st, put);
  }
}

hipError_t launch_gather(const float* r, int64_t n, const PartTotals* tot, const PartBlock* blk,
                         const int64_t* offsets, int nblocks, int64_t chunk, const float* stage_v,
                         const int32_t* stage_i, int64_t m_capacity, uint32_t* m_keys,
                         int32_t* m_idx, hipStream_t s) {
  { ProfScope ps_("gather", s);
  hipLaunchKernelGGL(gather_kernel, dim3(nblocks), dim3(PT), 0, s, r, n, tot, blk, offsets, chunk,
                     stage_v, stage_i, m_capacity, m_keys, m_idx); }
  return hipGetLastError();
}

}  // namespace lapsum
