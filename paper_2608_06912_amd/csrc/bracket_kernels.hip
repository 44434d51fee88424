// The probabilistic bracket (§4, Suppl. B, Suppl. C, Algorithm 1):
//   sample            y_s = fl32(r[s * floor(n/K)] + eps_s) (the systematic
//                     sampler: strided view + cached kernel noise), stored as
//                     ascending uint32 keys, plus a histogram of their top
//                     11 bits
//   select            the j-th and l-th smallest y (Eq. (8)) by an 11/11/10
//                     bit radix select in one workgroup
//   partition         the single streaming pass: L = {r < a_L},
//                     M = {a_L <= r < a_R}, R = {r >= a_R}, the tail sums of
//                     Eq. (7) and counts, M compacted in index order into the
//                     block's staging area          (4 bytes read per score)
//   partition_totals  fixed-order totals and each block's M offset
//   gather            M to one contiguous array of (key, index)
#include <math.h>

#include "block_sort.hpp"
#include "kernels.hpp"

namespace lapsum {

namespace {

__device__ __forceinline__ uint32_t asc_key(float f) { return ~desc_key(f); }
__device__ __forceinline__ float asc_key_float(uint32_t k) { return key_float(~k); }

constexpr int kSampleThreads = 256;
constexpr int kSelThreads = 1024;
constexpr int PT = kPartThreads;               // 256
constexpr int PW = PT / kWave;                 // 4 waves
constexpr int kWaveStage = kPartStageCap / PW; // 512 M entries staged per wave

}  // namespace

// ----------------------------------------------------------------- sample --
__global__ __launch_bounds__(kSampleThreads) void sample_kernel(const float* __restrict__ r,
                                                                int64_t n,
                                                                const float* __restrict__ noise,
                                                                int64_t K, uint32_t* __restrict__ ykeys,
                                                                uint32_t* __restrict__ hist) {
  __shared__ uint32_t h[kSelectBins];
  for (int e = threadIdx.x; e < kSelectBins; e += kSampleThreads) h[e] = 0u;
  __syncthreads();
  const int64_t s = static_cast<int64_t>(blockIdx.x) * kSampleThreads + threadIdx.x;
  const int64_t stride = n / K;
  if (s < K) {
    const float y = r[s * stride] + noise[s];   // float32 addition
    const uint32_t key = asc_key(y);
    ykeys[s] = key;
    atomicAdd(&h[key >> 21], 1u);
  }
  __syncthreads();
  for (int e = threadIdx.x; e < kSelectBins; e += kSampleThreads)
    if (h[e]) atomicAdd(&hist[e], h[e]);
}

hipError_t launch_sample(const float* r, int64_t n, const float* noise, int64_t K,
                         uint32_t* ykeys, uint32_t* hist, hipStream_t s) {
  const int64_t blocks = (K + kSampleThreads - 1) / kSampleThreads;
  { ProfScope ps_("sample", s);
  hipLaunchKernelGGL(sample_kernel, dim3(static_cast<unsigned>(blocks)), dim3(kSampleThreads), 0,
                     s, r, n, noise, K, ykeys, hist); }
  return hipGetLastError();
}

// ----------------------------------------------------------------- select --
namespace {

// Find the bin of a histogram (nb bins in LDS) holding 1-based rank `rank`;
// writes (bin, rank inside the bin) to *bin_out, *rank_out.
__device__ void find_bin(const uint32_t* h, int nb, uint32_t rank, uint32_t* wsum, int* bin_out,
                         uint32_t* rank_out) {
  // each thread owns nb / kSelThreads consecutive bins (nb = 1024 or 2048)
  const int tid = threadIdx.x;
  const int per = nb / kSelThreads;
  uint32_t loc = 0;
  for (int q = 0; q < per; ++q) loc += h[tid * per + q];
  uint32_t incl = loc;
  const int lane = lane_id();
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const uint32_t x = __shfl_up(incl, o, kWave);
    if (lane >= o) incl += x;
  }
  const int wid = tid / kWave;
  if (lane == kWave - 1) wsum[wid] = incl;
  __syncthreads();
  uint32_t base = 0;
  for (int w = 0; w < wid; ++w) base += wsum[w];
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

}  // namespace

// One workgroup.  Targets are 1-based ranks among the K sample keys; a rank
// outside 1..K gives -inf (below) or +inf (above).
__global__ __launch_bounds__(kSelThreads) void select_kernel(const uint32_t* __restrict__ ykeys,
                                                             int64_t K,
                                                             const uint32_t* __restrict__ hist,
                                                             int64_t j, int64_t l,
                                                             SelectRec* __restrict__ out) {
  __shared__ uint32_t h[2][kSelectBins];
  __shared__ uint32_t wsum[kSelThreads / kWave];
  __shared__ int bin_s[2];
  __shared__ uint32_t rank_s[2];
  const int tid = threadIdx.x;
  const int64_t tgt[2] = {j, l};
  bool live[2];
  uint32_t prefix[2] = {0u, 0u};
  for (int q = 0; q < 2; ++q) live[q] = (tgt[q] >= 1 && tgt[q] <= K);

  // pass 0: top 11 bits, histogram built by the sample kernel
  for (int q = 0; q < 2; ++q) {
    if (!live[q]) continue;
    for (int e = tid; e < kSelectBins; e += kSelThreads) h[0][e] = hist[e];
    __syncthreads();
    find_bin(h[0], kSelectBins, static_cast<uint32_t>(tgt[q]), wsum, &bin_s[q], &rank_s[q]);
    __syncthreads();
  }
  for (int q = 0; q < 2; ++q) prefix[q] = static_cast<uint32_t>(bin_s[q]);
  // passes 1 and 2: bits 10..20 (11 bits), then bits 0..9 (10 bits)
  for (int pass = 1; pass <= 2; ++pass) {
    const int hi_shift = (pass == 1) ? 21 : 10;   // bits already fixed
    const int lo_shift = (pass == 1) ? 10 : 0;
    const uint32_t mask = (pass == 1) ? 2047u : 1023u;
    const int nb = (pass == 1) ? 2048 : 1024;
    for (int e = tid; e < 2 * kSelectBins; e += kSelThreads) (&h[0][0])[e] = 0u;
    __syncthreads();
    for (int64_t i = tid; i < K; i += kSelThreads) {
      const uint32_t key = ykeys[i];
      for (int q = 0; q < 2; ++q)
        if (live[q] && (key >> hi_shift) == prefix[q]) atomicAdd(&h[q][(key >> lo_shift) & mask], 1u);
    }
    __syncthreads();
    for (int q = 0; q < 2; ++q) {
      if (!live[q]) continue;
      find_bin(h[q], nb, rank_s[q], wsum, &bin_s[q], &rank_s[q]);
      __syncthreads();
      prefix[q] = (prefix[q] << (pass == 1 ? 11 : 10)) | static_cast<uint32_t>(bin_s[q]);
    }
  }
  if (tid == 0) {
    SelectRec rec;
    rec.keyL = live[0] ? prefix[0] : 0u;
    rec.keyR = live[1] ? prefix[1] : 0u;
    rec.aL = live[0] ? asc_key_float(prefix[0]) : -INFINITY;
    rec.aR = live[1] ? asc_key_float(prefix[1]) : (tgt[1] < 1 ? -INFINITY : INFINITY);
    if (!live[0] && tgt[0] > K) rec.aL = INFINITY;
    *out = rec;
  }
}

hipError_t launch_select(const uint32_t* ykeys, int64_t K, const uint32_t* hist, int64_t j,
                         int64_t l, SelectRec* out, hipStream_t s) {
  { ProfScope ps_("select", s);
  hipLaunchKernelGGL(select_kernel, dim3(1), dim3(kSelThreads), 0, s, ykeys, K, hist, j, l, out); }
  return hipGetLastError();
}

// -------------------------------------------------------------- partition --
int partition_blocks(int64_t n, int64_t* chunk) {
  // ~2048 blocks; each block's chunk is a multiple of 1024 scores so that
  // every wave owns a contiguous, float4-aligned quarter of it
  int64_t c = (n + 2047) / 2048;
  c = (c + 1023) / 1024 * 1024;
  if (c < 1024) c = 1024;
  *chunk = c;
  return static_cast<int>((n + c - 1) / c);
}

namespace {

struct PartState {
  double TL, TR;
  int64_t nL, nR;
  int64_t nM;   // M count of this wave (uniform across the wave)
};

// Classify 4 consecutive scores of one lane; tails accumulate in float32
// over the four and in float64 across calls.  M members are reported by
// the callback in index order within the wave (lane-major, then element).
template <typename Emit>
__device__ __forceinline__ void classify4(const float (&v)[4], const bool (&ok)[4], int64_t i0,
                                          float aL, float aR, float c2f, PartState& st,
                                          Emit&& emit) {
  float tl = 0.0f, tr = 0.0f;
  int cl = 0, cr = 0;
  bool inM[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const bool L = ok[e] && v[e] < aL;
    const bool R = ok[e] && v[e] >= aR;
    inM[e] = ok[e] && !L && !R;
    // e^{-(a_L - r)/t} for L, e^{-(r - a_R)/t} for R (exponent <= 0)
    const float x = L ? (v[e] - aL) : (aR - v[e]);
    const float term = exp2_fast(x * c2f);
    tl += L ? term : 0.0f;
    tr += R ? term : 0.0f;
    cl += L;
    cr += R;
  }
  st.TL += static_cast<double>(tl);
  st.TR += static_cast<double>(tr);
  st.nL += cl;
  st.nR += cr;
  uint64_t bal[4];
  uint32_t before = 0;
  uint32_t total = 0;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    bal[e] = __ballot(inM[e]);
    before += lanes_below(bal[e]);
    total += static_cast<uint32_t>(__popcll(bal[e]));
  }
  if (total) {
    uint32_t idx = before;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      if (inM[e]) {
        emit(st.nM + idx, v[e], i0 + e);
        ++idx;
      }
    }
  }
  st.nM += total;
}

}  // namespace

// Each block owns [b*chunk, (b+1)*chunk); wave w the w-th contiguous quarter
// of it, walked 256 scores (one float4 per lane) at a time, so the wave sees
// its scores in index order.  M members are staged per wave in LDS, then
// written to the block's slot of the global staging area in index order.
__global__ __launch_bounds__(PT) void partition_kernel(const float* __restrict__ r, int64_t n,
                                                       const SelectRec* __restrict__ sel,
                                                       int use_sel, float aL_arg, float aR_arg,
                                                       float c2f, int64_t chunk,
                                                       float* __restrict__ stage_v,
                                                       int32_t* __restrict__ stage_i,
                                                       PartBlock* __restrict__ blk) {
  __shared__ float sv[PW][kWaveStage];
  __shared__ int32_t si[PW][kWaveStage];
  __shared__ double red_d[2][PW];
  __shared__ int64_t red_i[3][PW];
  const float aL = use_sel ? sel->aL : aL_arg;
  const float aR = use_sel ? sel->aR : aR_arg;
  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wid = tid / kWave;
  const int64_t b0 = static_cast<int64_t>(blockIdx.x) * chunk;
  const int64_t wq = chunk / PW;
  const int64_t w0 = b0 + wid * wq;
  int64_t w1 = w0 + wq;
  if (w1 > n) w1 = n;
  PartState st{0.0, 0.0, 0, 0, 0};
  auto stage = [&](int64_t slot, float v, int64_t gi) {
    if (slot < kWaveStage) {
      sv[wid][slot] = v;
      si[wid][slot] = static_cast<int32_t>(gi);
    }
  };
  constexpr int U = 4;   // float4 loads in flight per lane
  const bool vec = (reinterpret_cast<uintptr_t>(r) & 15) == 0;
  int64_t it = w0;
  for (; vec && it + U * 256 <= w1; it += U * 256) {
    float4 q[U];
#pragma unroll
    for (int u = 0; u < U; ++u) q[u] = *reinterpret_cast<const float4*>(r + it + u * 256 + 4 * lane);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const float v[4] = {q[u].x, q[u].y, q[u].z, q[u].w};
      const bool ok[4] = {true, true, true, true};
      classify4(v, ok, it + u * 256 + 4 * lane, aL, aR, c2f, st, stage);
    }
  }
  for (; it < w1; it += 256) {
    const int64_t i0 = it + 4 * lane;
    float v[4];
    bool ok[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      ok[e] = (i0 + e) < w1;
      v[e] = ok[e] ? r[i0 + e] : 0.0f;
    }
    classify4(v, ok, i0, aL, aR, c2f, st, stage);
  }
  // block totals in a fixed order
  const double TL = wave_sum(st.TL);
  const double TR = wave_sum(st.TR);
  const int64_t nL = wave_sum(st.nL);
  const int64_t nR = wave_sum(st.nR);
  if (lane == 0) {
    red_d[0][wid] = TL;
    red_d[1][wid] = TR;
    red_i[0][wid] = nL;
    red_i[1][wid] = nR;
    red_i[2][wid] = st.nM;
  }
  __syncthreads();
  int64_t off = 0, mtot = 0;
  bool over = false;
#pragma unroll
  for (int w = 0; w < PW; ++w) {
    if (w < wid) off += red_i[2][w];
    mtot += red_i[2][w];
    over |= red_i[2][w] > kWaveStage;
  }
  if (!over) {
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
    int64_t cl = 0, cr = 0;
#pragma unroll
    for (int w = 0; w < PW; ++w) {
      tl += red_d[0][w];
      tr += red_d[1][w];
      cl += red_i[0][w];
      cr += red_i[1][w];
    }
    rec.TL = tl;
    rec.TR = tr;
    rec.nL = cl;
    rec.nR = cr;
    rec.nM = mtot;
    rec.overflow = over ? 1 : 0;
    rec.pad = 0;
    blk[blockIdx.x] = rec;
  }
}

hipError_t launch_partition(const float* r, int64_t n, const SelectRec* sel, int use_sel, float aL,
                            float aR, double t, int nblocks, int64_t chunk, float* stage_v,
                            int32_t* stage_i, PartBlock* blk, hipStream_t s) {
  const float c2f = static_cast<float>(kLog2e / t);
  { ProfScope ps_("partition", s);
  hipLaunchKernelGGL(partition_kernel, dim3(nblocks), dim3(PT), 0, s, r, n, sel, use_sel, aL, aR,
                     c2f, chunk, stage_v, stage_i, blk); }
  return hipGetLastError();
}

// One workgroup: totals over the partition blocks in a fixed order, and the
// exclusive prefix of their M counts (each block's offset into M).
__global__ __launch_bounds__(1024) void partition_totals_kernel(const PartBlock* __restrict__ blk,
                                                                int nblocks,
                                                                const SelectRec* __restrict__ sel,
                                                                int use_sel, float aL_arg,
                                                                float aR_arg,
                                                                int64_t* __restrict__ offsets,
                                                                PartTotals* __restrict__ tot) {
  constexpr int T = 1024;
  constexpr int W = T / kWave;
  __shared__ double rd[2][W];
  __shared__ int64_t ri[4][W];
  __shared__ int64_t carry_s;
  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wid = tid / kWave;
  double TL = 0.0, TR = 0.0;
  int64_t nL = 0, nR = 0, ov = 0;
  for (int b = tid; b < nblocks; b += T) {
    TL += blk[b].TL;
    TR += blk[b].TR;
    nL += blk[b].nL;
    nR += blk[b].nR;
    ov += blk[b].overflow;
  }
  TL = wave_sum(TL);
  TR = wave_sum(TR);
  nL = wave_sum(nL);
  nR = wave_sum(nR);
  ov = wave_sum(ov);
  if (lane == 0) {
    rd[0][wid] = TL;
    rd[1][wid] = TR;
    ri[0][wid] = nL;
    ri[1][wid] = nR;
    ri[2][wid] = ov;
  }
  if (tid == 0) carry_s = 0;
  __syncthreads();
  // exclusive scan of nM over blocks, T at a time
  for (int c0 = 0; c0 < nblocks; c0 += T) {
    const int b = c0 + tid;
    const int64_t v = (b < nblocks) ? blk[b].nM : 0;
    int64_t incl = v;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
      const int64_t x = __shfl_up(incl, o, kWave);
      if (lane >= o) incl += x;
    }
    if (lane == kWave - 1) ri[3][wid] = incl;
    __syncthreads();
    int64_t base = carry_s, all = 0;
#pragma unroll
    for (int w = 0; w < W; ++w) {
      if (w < wid) base += ri[3][w];
      all += ri[3][w];
    }
    if (b < nblocks) offsets[b] = base + incl - v;
    __syncthreads();
    if (tid == 0) carry_s += all;
    __syncthreads();
  }
  if (tid == 0) {
    PartTotals x;
    double tl = 0.0, tr = 0.0;
    int64_t cl = 0, cr = 0, co = 0;
#pragma unroll
    for (int w = 0; w < W; ++w) {
      tl += rd[0][w];
      tr += rd[1][w];
      cl += ri[0][w];
      cr += ri[1][w];
      co += ri[2][w];
    }
    x.TL = tl;
    x.TR = tr;
    x.nL = cl;
    x.nR = cr;
    x.nM = carry_s;
    x.aL = use_sel ? sel->aL : aL_arg;
    x.aR = use_sel ? sel->aR : aR_arg;
    x.any_block_overflow = co > 0 ? 1 : 0;
    x.pad = 0;
    *tot = x;
  }
}

hipError_t launch_partition_totals(const PartBlock* blk, int nblocks, const SelectRec* sel,
                                   int use_sel, float aL, float aR, int64_t* offsets,
                                   PartTotals* tot, hipStream_t s) {
  { ProfScope ps_("partition_totals", s);
  hipLaunchKernelGGL(partition_totals_kernel, dim3(1), dim3(1024), 0, s, blk, nblocks, sel, use_sel,
                     aL, aR, offsets, tot); }
  return hipGetLastError();
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
  PartState st{0.0, 0.0, 0, 0, 0};
  auto put = [&](int64_t slot, float v, int64_t gi) {
    m_keys[off + slot] = desc_key(v);
    m_idx[off + slot] = static_cast<int32_t>(gi);
  };
  for (int64_t it = b0; it < b1; it += 256) {
    const int64_t i0 = it + 4 * lane;
    float v[4];
    bool ok[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      ok[e] = (i0 + e) < b1;
      v[e] = ok[e] ? r[i0 + e] : 0.0f;
    }
    classify4(v, ok, i0, aL, aR, 0.0f, st, put);
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
