// Passes over the band a bracket's partition staged (the scores whose p is
// strictly between 0 and 1 can only lie there; see BandEntry):
//   band_emit      p for one partition block's range: band members from
//                  their staged score and b, every other score 0 or 1 from
//                  the side it lies on (one bit per score when a_R is
//                  finite).  Writes p densely without reading r: 4 B/score
//                  plus 8 B per band member.  The entries then hold p, the
//                  forward's context for the backward.
//   band_vjp       Eq. (5) from the context: sums of f = min(p, 1 - p) and
//                  f g over the band (g read only where f != 0), then
//                  grad_r written densely (zero outside the band), each emit
//                  block summing the partials in a fixed order: 4 B/score
//                  plus the band.
// A block whose lists overflowed (or whose range is too long for the LDS
// map) takes the dense form of each pass over its own range.
#include "common.hpp"
#include "kernels.hpp"

namespace lapsum {

namespace {

constexpr int BT = 256;
constexpr int BW = BT / kWave;   // one list segment per wave of the partition
static_assert(BW == 4, "the partition stages one list per wave of four");
constexpr int kMaxWords = static_cast<int>(kBandMaxChunk / 32);
constexpr int kMaxEnt = 4 * kBandWaveCapMax;
constexpr int kWordsPerThread = kMaxWords / BT;

// LDS map from a block-local offset to the rank of its band member, sized
// for the row's chunk and list capacity (dynamic LDS: a block of a shorter
// chunk needs less, so that more blocks share a CU).
struct BandLds {
  uint32_t* bits;   // [words] one bit per score of the chunk
  uint32_t* pre;    // [words] members in the words before
  float* vals;      // [4 cap] value of the member of each rank
  uint32_t* wtot;   // [BW]
};

__host__ __device__ inline int band_lds_words(int64_t chunk) {
  const int64_t c = chunk < kBandMaxChunk ? chunk : kBandMaxChunk;
  return static_cast<int>((c + 31) / 32);
}
__host__ __device__ inline size_t band_lds_bytes(int64_t chunk, int cap) {
  const int e = 4 * (cap < kBandWaveCapMax ? cap : kBandWaveCapMax);
  return static_cast<size_t>(2 * band_lds_words(chunk) + e + BW) * 4;
}
__device__ inline BandLds band_lds(uint32_t* base, int64_t chunk, int cap) {
  const int w = band_lds_words(chunk);
  const int e = 4 * (cap < kBandWaveCapMax ? cap : kBandWaveCapMax);
  BandLds L;
  L.bits = base;
  L.pre = base + w;
  L.vals = reinterpret_cast<float*>(base + 2 * w);
  L.wtot = base + 2 * w + e;
  return L;
}

struct BlockRange {
  int64_t b0, b1;
};

__device__ __forceinline__ BlockRange block_range(int64_t n, int64_t chunk) {
  BlockRange br;
  br.b0 = static_cast<int64_t>(blockIdx.x) * chunk;
  br.b1 = br.b0 + chunk < n ? br.b0 + chunk : n;
  return br;
}

__device__ __forceinline__ BlockRange range_of(int64_t n, int64_t chunk, int pb) {
  BlockRange br;
  br.b0 = static_cast<int64_t>(pb) * chunk;
  br.b1 = br.b0 + chunk < n ? br.b0 + chunk : n;
  return br;
}

// The lists of partition block pb are complete and consistent with the layout.
__device__ __forceinline__ bool lists_usable(const BandCtx& c, int pb) {
  const BandBlock& bb = c.blk[pb];
  bool ok = bb.dense == 0 && c.chunk <= kBandMaxChunk && c.cap <= kBandWaveCapMax;
#pragma unroll
  for (int w = 0; w < BW; ++w) ok = ok && bb.cnt[w] >= 0 && bb.cnt[w] <= c.cap;
  return ok;
}

// Backward: the saved header must describe this row (a band saved for
// another length, or a forward that fell back to the full sort, makes every
// pass dense).
__device__ __forceinline__ bool block_dense(const BandCtx& c, int64_t n, int pb) {
  const CtxHeader h = *c.hdr;
  if (h.mode != 0 || h.n != n || h.nblocks != c.nblocks || h.chunk != c.chunk || h.cap != c.cap)
    return true;
  return !lists_usable(c, pb);
}

// Build the map of this block's band.  Entries come either as the
// partition left them (four wave segments, each in the order its members
// were met; `from_segments`) or as the emit leaves them (one list in index
// order at the start of the block's region).  value(entry, rank) gives the
// float stored for each member; with `writeback` the members are written
// back as one list in index order, each carrying its value.  `aux` (or
// null) is a float per slot of the block's region, loaded with the entries
// and handed to value(entry, rank, aux of its slot).  Ends with a barrier.
template <typename Value>
__device__ void build_map(const BandCtx& c, int64_t b0, int64_t len, const BandLds& L,
                          bool from_segments, bool writeback, const float* aux, Value&& value) {
  constexpr int EPT = kMaxEnt / BT;   // entries per thread
  const int tid = threadIdx.x;
  // every thread reads the four segment counts (one broadcast load)
  int seg[BW + 1];
  {
    const int4 cnt = *reinterpret_cast<const int4*>(c.blk[blockIdx.x].cnt);
    seg[0] = 0;
    seg[1] = cnt.x;
    seg[2] = cnt.x + cnt.y;
    seg[3] = cnt.x + cnt.y + cnt.z;
    seg[4] = cnt.x + cnt.y + cnt.z + cnt.w;
  }
  const int total = seg[BW];
  BandEntry* base = c.ent + static_cast<int64_t>(blockIdx.x) * BW * c.cap;
  const float* abase = aux ? aux + static_cast<int64_t>(blockIdx.x) * BW * c.cap : nullptr;
  BandEntry en[EPT];
  float av[EPT];
  int off[EPT];
  // all loads first (slot 0 of the region stands in past the end); the
  // bits are cleared while they are in flight
#pragma unroll
  for (int q = 0; q < EPT; ++q) {
    const int e = tid + q * BT;
    int j = 0;
    if (e < total) {
      j = e;
      if (from_segments) {
        int w = 0;
#pragma unroll
        for (int x = 1; x < BW; ++x) w += (e >= seg[x]) ? 1 : 0;
        j = w * c.cap + (e - seg[w]);
      }
    }
    en[q] = base[j];
    av[q] = abase ? abase[j] : 0.0f;
  }
  const int nwords = static_cast<int>((len + 31) / 32);
  for (int w = tid; w < nwords; w += BT) L.bits[w] = 0u;
  __syncthreads();
#pragma unroll
  for (int q = 0; q < EPT; ++q) {
    const int e = tid + q * BT;
    off[q] = -1;
    if (e < total) {
      const int64_t o = static_cast<int64_t>(en[q].idx) - b0;
      if (o >= 0 && o < len) {
        off[q] = static_cast<int>(o);
        atomicOr(&L.bits[o >> 5], 1u << (o & 31));
      }
    }
  }
  __syncthreads();
  // exclusive prefix of the members per word: each thread owns a run of words
  const int w0 = tid * kWordsPerThread;
  uint32_t loc = 0;
#pragma unroll
  for (int q = 0; q < kWordsPerThread; ++q)
    loc += (w0 + q < nwords) ? static_cast<uint32_t>(__popc(L.bits[w0 + q])) : 0u;
  uint32_t incl = loc;
  const int lane = lane_id();
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const uint32_t x = __shfl_up(incl, o, kWave);
    if (lane >= o) incl += x;
  }
  const int wid = tid / kWave;
  if (lane == kWave - 1) L.wtot[wid] = incl;
  __syncthreads();
  uint32_t run = incl - loc;
#pragma unroll
  for (int w = 0; w < BW; ++w)
    if (w < wid) run += L.wtot[w];
#pragma unroll
  for (int q = 0; q < kWordsPerThread; ++q) {
    if (w0 + q < nwords) {
      L.pre[w0 + q] = run;
      run += static_cast<uint32_t>(__popc(L.bits[w0 + q]));
    }
  }
  __syncthreads();
  // each member's rank in index order
#pragma unroll
  for (int q = 0; q < EPT; ++q) {
    if (off[q] >= 0) {
      const int o = off[q];
      const uint32_t word = L.bits[o >> 5];
      const int rank = static_cast<int>(L.pre[o >> 5] + __popc(word & ((1u << (o & 31)) - 1u)));
      const float val = value(en[q], rank, av[q]);
      L.vals[rank] = val;
      if (writeback) {
        BandEntry w;
        w.idx = en[q].idx;
        w.bits = __float_as_uint(val);
        base[rank] = w;
      }
    }
  }
  __syncthreads();
}

// Write out[b0 .. b1) from the map: members take their value, other scores
// 0, or 1 where their bit in `ones` is set (ones may be null).
__device__ void write_dense(int64_t b0, int64_t b1, const BandLds& L, const uint32_t* ones,
                            float* __restrict__ out) {
  const int tid = threadIdx.x;
  const int64_t len = b1 - b0;
  auto value = [&](int64_t o) -> float {   // o: block-local offset
    const uint32_t word = L.bits[o >> 5];
    const uint32_t bit = 1u << (o & 31);
    if (word & bit) return L.vals[L.pre[o >> 5] + __popc(word & (bit - 1u))];
    return (ones && ((ones[(b0 + o) >> 5] >> ((b0 + o) & 31)) & 1u)) ? 1.0f : 0.0f;
  };
  if ((reinterpret_cast<uintptr_t>(out + b0) & 15) == 0) {
    const int64_t n4 = len / 4;
    // float4 q takes nibble q & 7 of word q >> 3; WB float4 per thread at
    // a time, their words (and bits of `ones`) read before any store
    auto one4 = [&](int64_t q, uint32_t word, uint32_t oword) {
      const int sh = static_cast<int>(q & 7) * 4;
      const uint32_t nib = (word >> sh) & 15u;
      const uint32_t onib = (oword >> sh) & 15u;
      float v[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = ((onib >> e) & 1u) ? 1.0f : 0.0f;
      if (nib) {
        uint32_t rk = L.pre[q >> 3] + static_cast<uint32_t>(__popc(word & ((1u << sh) - 1u)));
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if ((nib >> e) & 1u) v[e] = L.vals[rk++];
      }
      store_stream4(out + b0 + 4 * q, make_float4(v[0], v[1], v[2], v[3]));
    };
    constexpr int WB = 8;
    int64_t q0 = 0;
    for (; q0 + WB * BT <= n4; q0 += WB * BT) {
      uint32_t wd[WB], ow[WB];
#pragma unroll
      for (int k = 0; k < WB; ++k) {
        const int64_t q = q0 + k * BT + tid;
        wd[k] = L.bits[q >> 3];
        ow[k] = ones ? ones[(b0 >> 5) + (q >> 3)] : 0u;
      }
#pragma unroll
      for (int k = 0; k < WB; ++k) one4(q0 + k * BT + tid, wd[k], ow[k]);
    }
    for (int64_t q = q0 + tid; q < n4; q += BT)
      one4(q, L.bits[q >> 3], ones ? ones[(b0 >> 5) + (q >> 3)] : 0u);
    for (int64_t o = n4 * 4 + tid; o < len; o += BT) out[b0 + o] = value(o);
  } else {
    for (int64_t o = tid; o < len; o += BT) out[b0 + o] = value(o);
  }
}

// Dense emit of one block's range.
__device__ void dense_emit(const float* __restrict__ r, int64_t b0, int64_t b1, double b,
                           double inv_t, float* __restrict__ p) {
  const int tid = threadIdx.x;
  const bool vec = ((reinterpret_cast<uintptr_t>(r + b0) | reinterpret_cast<uintptr_t>(p + b0)) & 15) == 0;
  int64_t i = b0 + tid;
  if (vec) {
    const int64_t n4 = (b1 - b0) / 4;
    for (int64_t q = tid; q < n4; q += BT) {
      const float4 v = load_stream4(r + b0 + 4 * q);
      store_stream4(p + b0 + 4 * q, make_float4(laplace_p(v.x, b, inv_t), laplace_p(v.y, b, inv_t),
                                                laplace_p(v.z, b, inv_t), laplace_p(v.w, b, inv_t)));
    }
    i = b0 + n4 * 4 + tid;
  }
  for (; i < b1; i += BT) p[i] = laplace_p(r[i], b, inv_t);
}

}  // namespace

__global__ __launch_bounds__(BT) void band_emit_kernel(const float* __restrict__ r, int64_t n,
                                                       const SolveRec* __restrict__ rec,
                                                       double inv_t, BandCtx c,
                                                       const uint32_t* __restrict__ ones_all,
                                                       const PartTotals* __restrict__ tot,
                                                       float* __restrict__ p,
                                                       double* __restrict__ b_out) {
  extern __shared__ uint32_t band_lds_mem[];
  const BandLds L = band_lds(band_lds_mem, c.chunk, c.cap);
  if (!rec->ok) return;
  const uint32_t* ones = tot->aR < INFINITY ? ones_all : nullptr;
  const double b = rec->b;
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    b_out[0] = b;
    CtxHeader h;
    h.mode = 0;
    h.nblocks = c.nblocks;
    h.chunk = c.chunk;
    h.cap = c.cap;
    h.pad = 0;
    h.n = n;
    *c.hdr = h;
  }
  const BlockRange br = block_range(n, c.chunk);
  if (!lists_usable(c, static_cast<int>(blockIdx.x))) {
    dense_emit(r, br.b0, br.b1, b, inv_t, p);
    return;
  }
  build_map(c, br.b0, br.b1 - br.b0, L, true, true, nullptr, [&](const BandEntry& en, int, float) {
    return laplace_p(__uint_as_float(en.bits), b, inv_t);
  });
  write_dense(br.b0, br.b1, L, ones, p);
}

hipError_t launch_band_emit(const float* r, int64_t n, const SolveRec* rec, double t,
                            const BandCtx& band, const uint32_t* ones, const PartTotals* tot,
                            float* p, double* b_out, hipStream_t s) {
  { ProfScope ps_("band_emit", s);
  hipLaunchKernelGGL(band_emit_kernel, dim3(band.nblocks), dim3(BT),
                     static_cast<unsigned>(band_lds_bytes(band.chunk, band.cap)), s, r, n, rec, 1.0 / t, band,
                     ones, tot, p, b_out); }
  return hipGetLastError();
}

__global__ void ctx_dense_kernel(BandCtx c, int64_t n) {
  CtxHeader h;
  h.mode = 1;
  h.nblocks = c.nblocks;
  h.chunk = c.chunk;
  h.cap = c.cap;
  h.pad = 0;
  h.n = n;
  *c.hdr = h;
}

hipError_t launch_ctx_dense(const BandCtx& band, int64_t n, hipStream_t s) {
  { ProfScope ps_("ctx_dense", s);
  hipLaunchKernelGGL(ctx_dense_kernel, dim3(1), dim3(1), 0, s, band, n); }
  return hipGetLastError();
}

// ---------------------------------------------------------------- backward --
// One wave of a reduce block per partition block; the emit blocks sum the
// reduce partials themselves (fixed order), so no launch sits between.
constexpr int kVjpWaveBlocks = BW;             // partition blocks per reduce block
constexpr int kVjpMaxParts = 4 * BT;           // partials an emit block sums

__global__ __launch_bounds__(BT) void band_vjp_reduce_kernel(const float* __restrict__ g,
                                                             const float* __restrict__ p,
                                                             int64_t n, BandCtx c,
                                                             float* __restrict__ gstash,
                                                             double* __restrict__ partials) {
  __shared__ double red[2][BW];
  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wid = tid / kWave;
  const int pb = static_cast<int>(blockIdx.x) * kVjpWaveBlocks + wid;
  double F = 0.0, G = 0.0;
  if (pb < c.nblocks) {
    const BlockRange br = range_of(n, c.chunk, pb);
    if (block_dense(c, n, pb)) {
      for (int64_t i = br.b0 + lane; i < br.b1; i += kWave) {
        const float pv = p[i];
        const float f = fminf(pv, 1.0f - pv);
        if (f != 0.0f) {
          F += static_cast<double>(f);
          G += static_cast<double>(f) * static_cast<double>(g[i]);
        }
      }
    } else {
      // after the emit the block's members form one list in index order;
      // VB entries per lane at a time, all their loads (then all the loads
      // of g they select) in flight together; each lane still adds its
      // entries in list order
      const BandBlock& bb = c.blk[pb];
      const int total = bb.cnt[0] + bb.cnt[1] + bb.cnt[2] + bb.cnt[3];
      const int64_t base = static_cast<int64_t>(pb) * BW * c.cap;
      constexpr int VB = 8;
      for (int e0 = 0; e0 < total; e0 += VB * kWave) {
        BandEntry en[VB];
#pragma unroll
        for (int u = 0; u < VB; ++u) {
          const int e = e0 + u * kWave + lane;
          en[u] = c.ent[base + (e < total ? e : 0)];
        }
        float fv[VB], gv[VB];
        bool use[VB];
#pragma unroll
        for (int u = 0; u < VB; ++u) {
          const int e = e0 + u * kWave + lane;
          const float pv = __uint_as_float(en[u].bits);
          fv[u] = fminf(pv, 1.0f - pv);
          use[u] = e < total && fv[u] != 0.0f && en[u].idx >= br.b0 && en[u].idx < br.b1;
          gv[u] = g[use[u] ? en[u].idx : br.b0];   // an index of this block either way
        }
#pragma unroll
        for (int u = 0; u < VB; ++u) {
          if (use[u]) {
            gstash[base + e0 + u * kWave + lane] = gv[u];
            F += static_cast<double>(fv[u]);
            G += static_cast<double>(fv[u]) * static_cast<double>(gv[u]);
          }
        }
      }
    }
  }
  F = wave_sum(F);
  G = wave_sum(G);
  if (lane == 0) {
    red[0][wid] = F;
    red[1][wid] = G;
  }
  __syncthreads();
  if (tid == 0) {
    double fs = 0.0, gs = 0.0;
#pragma unroll
    for (int w = 0; w < BW; ++w) {
      fs += red[0][w];
      gs += red[1][w];
    }
    partials[2 * blockIdx.x] = fs;
    partials[2 * blockIdx.x + 1] = gs;
  }
}

// grad_r = (f/t)(g - <g,q>); <g,q> = sum f g / sum f from the partials, 0
// (and grad_r = 0) when sum f == 0.
__global__ __launch_bounds__(BT) void band_vjp_emit_kernel(const float* __restrict__ g,
                                                           const float* __restrict__ p,
                                                           int64_t n, BandCtx c,
                                                           const float* __restrict__ gstash,
                                                           const double* __restrict__ partials,
                                                           int nparts, double inv_t,
                                                           float* __restrict__ grad) {
  extern __shared__ uint32_t band_lds_mem[];
  const BandLds L = band_lds(band_lds_mem, c.chunk, c.cap);
  __shared__ double red[2][BW];
  const int tid = threadIdx.x;
  double F = 0.0, G = 0.0;
  {
    // every load issued before the first add (nparts >= 1)
    double2 pr[kVjpMaxParts / BT];
#pragma unroll
    for (int q = 0; q < kVjpMaxParts / BT; ++q) {
      const int i = q * BT + tid;
      pr[q] = reinterpret_cast<const double2*>(partials)[i < nparts ? i : 0];
    }
#pragma unroll
    for (int q = 0; q < kVjpMaxParts / BT; ++q) {
      if (q * BT + tid < nparts) {
        F += pr[q].x;
        G += pr[q].y;
      }
    }
  }
  F = wave_sum(F);
  G = wave_sum(G);
  if (lane_id() == 0) {
    red[0][tid / kWave] = F;
    red[1][tid / kWave] = G;
  }
  __syncthreads();
  double fs = 0.0, gsum = 0.0;
#pragma unroll
  for (int w = 0; w < BW; ++w) {
    fs += red[0][w];
    gsum += red[1][w];
  }
  const float coef = static_cast<float>(fs > 0.0 ? gsum / fs : 0.0);
  const float scale = static_cast<float>(fs > 0.0 ? inv_t : 0.0);
  const BlockRange br = block_range(n, c.chunk);
  if (block_dense(c, n, static_cast<int>(blockIdx.x))) {
    for (int64_t i = br.b0 + tid; i < br.b1; i += BT) {
      const float pv = p[i];
      const float f = fminf(pv, 1.0f - pv);
      grad[i] = (f != 0.0f) ? f * scale * (g[i] - coef) : 0.0f;
    }
    return;
  }
  // g of each member was stashed at its slot by the reduce (where f != 0)
  build_map(c, br.b0, br.b1 - br.b0, L, false, false, gstash,
            [&](const BandEntry& en, int, float gv) {
              const float pv = __uint_as_float(en.bits);
              const float f = fminf(pv, 1.0f - pv);
              return (f != 0.0f) ? f * scale * (gv - coef) : 0.0f;
            });
  write_dense(br.b0, br.b1, L, nullptr, grad);
}

int band_vjp_parts(int nblocks) { return (nblocks + kVjpWaveBlocks - 1) / kVjpWaveBlocks; }

hipError_t launch_band_vjp(const float* g, const float* p, int64_t n, const BandCtx& band,
                           float* gstash, double* partials, double t, float* grad,
                           hipStream_t s) {
  const int parts = band_vjp_parts(band.nblocks);
  { ProfScope ps_("band_vjp_reduce", s);
  hipLaunchKernelGGL(band_vjp_reduce_kernel, dim3(parts), dim3(BT), 0, s, g, p, n, band, gstash,
                     partials); }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  { ProfScope ps_("band_vjp_emit", s);
  hipLaunchKernelGGL(band_vjp_emit_kernel, dim3(band.nblocks), dim3(BT),
                     static_cast<unsigned>(band_lds_bytes(band.chunk, band.cap)), s, g, p, n, band,
                     gstash, partials, parts, 1.0 / t, grad); }
  return hipGetLastError();
}

}  // namespace lapsum
