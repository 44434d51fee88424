// Passes over the band a bracket's partition staged (the scores whose p is
// strictly between 0 and 1 can only lie there; see BandEntry):
//   band_emit        p for every score: band members from their staged score
//                    and b, every other score 0 or 1 from the side it lies
//                    on (one bit per score when a_R is finite).  Writes p
//                    without reading r: 4 B/score plus 8 B per band member.
//   band_vjp_reduce  Eq. (5)'s sums of f = min(p, 1 - p) and f g over the
//                    band, p recomputed from the staged score and the b the
//                    emit saved, g read only where f != 0 (and stashed at the
//                    member's list slot).
//   band_vjp_write   grad_r for every score, zero outside the band, each
//                    writer block summing the reduce partials in a fixed
//                    order: 4 B/score plus 12 B per band member.
// Both dense outputs are written by one persistent scheme (band_write): one
// workgroup per CU, four waves that only store and one wave that only loads.
// The row is cut into tiles of kBandTile scores and workgroup w writes tiles
// w, w + G, w + 2G, ... (G workgroups), kRound of them per round: at any time
// the device writes one contiguous window of G tiles, one tile per CU, which
// is the write pattern the memory system takes at its full rate.  The
// loading wave prefetches the tile records, member lists and ones bits of
// the next round and lays the round's member values into an LDS tile; the
// storing waves read LDS and store.  No wave both loads from and stores to
// memory in the stream, so no wait for a load is also a wait for earlier
// stores (one counter tracks both on this architecture).
// A tile whose block's lists are incomplete takes the dense form: its
// storing threads read r (forward) or p and g (backward) themselves.
#include "common.hpp"
#include "kernels.hpp"

namespace lapsum {

namespace {

constexpr int BT = 256;
constexpr int BW = BT / kWave;   // one list segment per wave of the partition
static_assert(BW == 4, "the partition stages one list per wave of four");

__device__ __forceinline__ int64_t clamp_end(int64_t a, int64_t n) { return a < n ? a : n; }

struct BlockRange {
  int64_t b0, b1;
};

__device__ __forceinline__ BlockRange range_of(int64_t n, int64_t chunk, int pb) {
  BlockRange br;
  br.b0 = static_cast<int64_t>(pb) * chunk;
  br.b1 = clamp_end(br.b0 + chunk, n);
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
__device__ __forceinline__ bool header_dense(const CtxHeader& h, const BandCtx& c, int64_t n) {
  return h.mode != 0 || h.n != n || h.nblocks != c.nblocks || h.chunk != c.chunk || h.cap != c.cap;
}

// ------------------------------------------------------------ tile writer --
constexpr int kRound = 8;          // tiles per round of a writer workgroup
constexpr int kSlots = 3;          // member slots per loading lane and round
constexpr int kStoreWaves = 4;
constexpr int WT = (kStoreWaves + 1) * kWave;   // 320 threads
constexpr int kTileF4 = static_cast<int>(kBandTile / 4);
constexpr int kTileWords = static_cast<int>(kBandTile / 32);
constexpr int kLanesPerTile = kWave / kRound;              // loading lanes per tile's ones words
constexpr int kWriterBlocks = 256;                         // one per CU
static_assert(kTileF4 == kStoreWaves * kWave, "one float4 of a tile per storing thread");
static_assert(kTileWords == 4 * kLanesPerTile, "a tile's ones words are one uint4 per lane");

struct WriterLds {
  float4 tile[2][kRound][kTileF4];      // member values of a round (0 elsewhere)
  uint32_t ow[2][kRound][kTileWords];   // ones bits of a round's tiles
  uint32_t dense[2];                    // bit i: tile i of the round is dense
  double red[4][kStoreWaves];
};

// Forward: p.
struct EmitPass {
  static constexpr bool kOnes = true;
  static constexpr int kInputs = 1;   // arrays a dense score reads
  const float* r;
  const uint32_t* ones;   // null when a_R is infinite
  double b, inv_t;
  __device__ float member(const BandEntry& e, float) const {
    return laplace_p(__uint_as_float(e.bits), b, inv_t);
  }
  __device__ float dense(float x, float) const { return laplace_p(x, b, inv_t); }
  __device__ const float* in0() const { return r; }
  __device__ const float* in1() const { return nullptr; }
  __device__ const float* stash() const { return nullptr; }
};

// Backward: grad_r = (f/t)(g - <g,q>), f = min(p, 1 - p).
struct VjpPass {
  static constexpr bool kOnes = false;
  static constexpr int kInputs = 2;
  const float* p;
  const float* g;
  const float* gstash;
  double b, inv_t;
  float coef, scale;
  __device__ float member(const BandEntry& e, float gs) const {
    const float pv = laplace_p(__uint_as_float(e.bits), b, inv_t);
    const float f = fminf(pv, 1.0f - pv);
    return (f != 0.0f) ? f * scale * (gs - coef) : 0.0f;
  }
  __device__ float dense(float pv, float gv) const {
    const float f = fminf(pv, 1.0f - pv);
    return (f != 0.0f) ? f * scale * (gv - coef) : 0.0f;
  }
  __device__ const float* in0() const { return p; }
  __device__ const float* in1() const { return g; }
  __device__ const float* stash() const { return gstash; }
};

__device__ __forceinline__ float4 load4_at(const float* x, int64_t o, int64_t n, bool vec) {
  if (vec && o + 3 < n) return load_stream4(x + o);
  float4 v;
  v.x = o < n ? x[o] : 0.0f;
  v.y = o + 1 < n ? x[o + 1] : 0.0f;
  v.z = o + 2 < n ? x[o + 2] : 0.0f;
  v.w = o + 3 < n ? x[o + 3] : 0.0f;
  return v;
}

// Storing waves: one float4 of each tile per thread and round.
template <class Pass>
__device__ void writer_store(const Pass& P, WriterLds& S, float* __restrict__ out, int64_t n,
                             int64_t nt, int64_t nr, bool vec_out, bool vec_in) {
  const int tid = threadIdx.x;
  const int64_t G = gridDim.x;
  for (int64_t k = 0; k < nr; ++k) {
    __syncthreads();
    const int buf = static_cast<int>(k & 1);
    const uint32_t dm = S.dense[buf];
    float4 v[kRound];
    uint32_t w[kRound];
#pragma unroll
    for (int i = 0; i < kRound; ++i) {
      v[i] = S.tile[buf][i][tid];
      if constexpr (Pass::kOnes) w[i] = S.ow[buf][i][tid >> 3];
      else w[i] = 0u;
    }
    if (dm) {
      // dense tiles (rare): every load of the round first, then the values
      float4 a[kRound], c[kRound];
#pragma unroll
      for (int i = 0; i < kRound; ++i) {
        if ((dm >> i) & 1u) {
          const int64_t o = ((blockIdx.x + (k * kRound + i) * G) * kTileF4 + tid) * 4;
          a[i] = load4_at(P.in0(), o, n, vec_in);
          if (P.in1()) c[i] = load4_at(P.in1(), o, n, vec_in);
          else c[i] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
        }
      }
#pragma unroll
      for (int i = 0; i < kRound; ++i) {
        if ((dm >> i) & 1u) {
          v[i] = make_float4(P.dense(a[i].x, c[i].x), P.dense(a[i].y, c[i].y),
                             P.dense(a[i].z, c[i].z), P.dense(a[i].w, c[i].w));
          w[i] = 0u;
        }
      }
    }
#pragma unroll
    for (int i = 0; i < kRound; ++i) {
      const int64_t t = k * kRound + i;
      if (t < nt) {
        const uint32_t nib = (w[i] >> ((tid & 7) * 4)) & 15u;
        float4 x;
        x.x = (nib & 1u) ? 1.0f : v[i].x;
        x.y = (nib & 2u) ? 1.0f : v[i].y;
        x.z = (nib & 4u) ? 1.0f : v[i].z;
        x.w = (nib & 8u) ? 1.0f : v[i].w;
        const int64_t o = ((blockIdx.x + t * G) * kTileF4 + tid) * 4;
        if (vec_out && o + 3 < n) {
          store_stream4(out + o, x);
        } else {
          if (o < n) out[o] = x.x;
          if (o + 1 < n) out[o + 1] = x.y;
          if (o + 2 < n) out[o + 2] = x.z;
          if (o + 3 < n) out[o + 3] = x.w;
        }
      }
    }
#pragma unroll
    for (int i = 0; i < kRound; ++i) S.tile[buf][i][tid] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
  }
}

// The loading wave.  Round k's tile records are loaded two rounds ahead and
// its lists and ones bits one round ahead; member slot s of a round (lane +
// 64 q) takes the s-th member of the round's tiles taken in order.  A round's
// bookkeeping stays in registers, lane i < kRound holding tile i (record and
// count), and per-slot choices are made from scalars read out of those
// lanes: no private array, so nothing of the loop goes through scratch
// memory (whose loads would join the wait for the prefetched data).
template <class Pass>
__device__ void writer_load(const Pass& P, WriterLds& S, const BandTile* __restrict__ tiles,
                            const BandEntry* __restrict__ ent, int64_t nt, int64_t nr,
                            bool all_dense) {
  const int lane = lane_id();
  const int64_t G = gridDim.x;
  // tile t of this workgroup (tile 0 stands in past the end)
  auto tile_at = [&](int64_t t) -> int64_t { return t < nt ? blockIdx.x + t * G : 0; };
  // lane i < kRound: the record of tile i of round k
  auto ld_rec = [&](int64_t k) -> int2 {
    const int64_t j = tile_at(k * kRound + (lane < kRound ? lane : 0));
    return reinterpret_cast<const int2*>(tiles)[j];
  };
  struct RoundInfo {
    int32_t first;   // lane i < kRound: tile i's first list slot
    int32_t cnt;     // lane i < kRound: its members in the lists (0 if dense or past the end)
    int32_t total;   // members of the round
    uint32_t dense;  // bit i: tile i is dense
  };
  auto info_of = [&](int64_t k, int2 rec) -> RoundInfo {
    RoundInfo ri;
    const bool valid = lane < kRound && k * kRound + lane < nt;
    const bool dn = valid && (all_dense || rec.y < 0);
    ri.first = rec.x;
    ri.cnt = (valid && !dn) ? rec.y : 0;
    ri.total = 0;
#pragma unroll
    for (int x = 0; x < kRound; ++x) ri.total += __builtin_amdgcn_readlane(ri.cnt, x);
    ri.dense = static_cast<uint32_t>(__ballot(dn));
    return ri;
  };
  struct Data {
    uint4 ov;
    BandEntry e[kSlots];
    float gs[kSlots];
    int ti[kSlots];
  };
  auto ld_data = [&](int64_t k, const RoundInfo& ri, Data& d) {
    if constexpr (Pass::kOnes) {
      if (P.ones) {
        const int64_t j = tile_at(k * kRound + lane / kLanesPerTile);
        d.ov = reinterpret_cast<const uint4*>(P.ones)[j * (kTileWords / 4) + lane % kLanesPerTile];
      } else {
        d.ov = make_uint4(0u, 0u, 0u, 0u);
      }
    }
#pragma unroll
    for (int q = 0; q < kSlots; ++q) {
      const int32_t s = lane + kWave * q;
      // tile of slot s: the last tile whose members start at or before s
      int i = 0;
      int32_t f = __builtin_amdgcn_readlane(ri.first, 0), p0 = 0;
      int32_t run = __builtin_amdgcn_readlane(ri.cnt, 0);   // members of tiles 0 .. x-1
#pragma unroll
      for (int x = 1; x < kRound; ++x) {
        const int32_t fx = __builtin_amdgcn_readlane(ri.first, x);
        const bool at_or_past = s >= run;
        i = at_or_past ? x : i;
        f = at_or_past ? fx : f;
        p0 = at_or_past ? run : p0;
        run += __builtin_amdgcn_readlane(ri.cnt, x);
      }
      const bool valid = s < ri.total;
      const int32_t at = valid ? f + (s - p0) : 0;
      d.ti[q] = valid ? i : -1;
      d.e[q] = ent[at];
      d.gs[q] = P.stash() ? P.stash()[at] : 0.0f;
    }
  };
  auto place = [&](int buf, int i, const BandEntry& e, float gs) {
    float* tl = reinterpret_cast<float*>(S.tile[buf][i]);
    tl[e.idx & static_cast<int32_t>(kBandTile - 1)] = P.member(e, gs);
  };
  int2 rec1 = ld_rec(1), rec2;
  RoundInfo ri0 = info_of(0, ld_rec(0));
  Data cur, nxt;
  ld_data(0, ri0, cur);
  // round 0's data in hand before the loop (an empty asm that reads it): the
  // loop's own loads are then only waited for at its end (the copies into
  // `cur`), never while the round's members are placed
#pragma unroll
  for (int q = 0; q < kSlots; ++q)
    asm volatile("" ::"v"(cur.e[q].idx), "v"(cur.e[q].bits), "v"(cur.gs[q]), "v"(cur.ti[q]));
  if constexpr (Pass::kOnes)
    asm volatile("" ::"v"(cur.ov.x), "v"(cur.ov.y), "v"(cur.ov.z), "v"(cur.ov.w));
  for (int64_t k = 0; k < nr; ++k) {
    rec2 = ld_rec(k + 2);
    const RoundInfo ri1 = info_of(k + 1, rec1);
    ld_data(k + 1, ri1, nxt);
    const int buf = static_cast<int>(k & 1);
    if constexpr (Pass::kOnes)
      reinterpret_cast<uint4*>(S.ow[buf][lane / kLanesPerTile])[lane % kLanesPerTile] = cur.ov;
    if (lane == 0) S.dense[buf] = ri0.dense;
#pragma unroll
    for (int q = 0; q < kSlots; ++q)
      if (cur.ti[q] >= 0) place(buf, cur.ti[q], cur.e[q], cur.gs[q]);
    if (ri0.total > kWave * kSlots) {
      // members past the slots (dense bands): read here, one at a time
      int32_t pi = 0;   // members of the tiles before tile i
      for (int i = 0; i < kRound; ++i) {
        const int32_t fi = __builtin_amdgcn_readlane(ri0.first, i);
        const int32_t ci = __builtin_amdgcn_readlane(ri0.cnt, i);
        for (int32_t e = lane; e < ci; e += kWave) {
          if (pi + e >= kWave * kSlots) {
            const int32_t at = fi + e;
            place(buf, i, ent[at], P.stash() ? P.stash()[at] : 0.0f);
          }
        }
        pi += ci;
      }
    }
    __syncthreads();
    rec1 = rec2;
    ri0 = ri1;
    cur = nxt;
  }
}

// A row without usable lists, streamed: out[i] = P.dense(in0[i], in1[i])
// for every score, by the first kStoreWaves waves of each workgroup, float4
// grid-strided so that the workgroups write neighbouring 4 KB pieces of one
// 1 MB window at a time (the pattern that reaches the full write rate).
template <class Pass>
__device__ void stream_row(const Pass& P, int64_t n, float* __restrict__ out) {
  constexpr int T = kStoreWaves * kWave;
  if (threadIdx.x >= T) return;
  const float* a = P.in0();
  const float* g = P.in1();
  const bool vec = ((reinterpret_cast<uintptr_t>(a) | reinterpret_cast<uintptr_t>(g) |
                     reinterpret_cast<uintptr_t>(out)) & 15) == 0;
  const int64_t n4 = vec ? n / 4 : 0;
  const int64_t G = static_cast<int64_t>(gridDim.x) * T;
  int64_t i = static_cast<int64_t>(blockIdx.x) * T + threadIdx.x;
  auto apply = [&](const float4& x, const float4& y) {
    float4 o;
    o.x = P.dense(x.x, y.x);
    o.y = P.dense(x.y, y.y);
    o.z = P.dense(x.z, y.z);
    o.w = P.dense(x.w, y.w);
    return o;
  };
  // eight float4 in flight per lane for one input stream, four for two
  // (measured: the emit's single stream gains, the backward's two do not)
  constexpr int U = Pass::kInputs == 1 ? 8 : 4;
  for (; i + (U - 1) * G < n4; i += U * G) {
    float4 x[U], y[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      x[u] = load_stream4(a + 4 * (i + u * G));
      y[u] = g ? load_stream4(g + 4 * (i + u * G)) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) store_stream4(out + 4 * (i + u * G), apply(x[u], y[u]));
  }
  for (; i < n4; i += G) {
    const float4 y = g ? load_stream4(g + 4 * i) : make_float4(0.f, 0.f, 0.f, 0.f);
    store_stream4(out + 4 * i, apply(load_stream4(a + 4 * i), y));
  }
  for (int64_t j = n4 * 4 + static_cast<int64_t>(blockIdx.x) * T + threadIdx.x; j < n; j += G)
    out[j] = P.dense(a[j], g ? g[j] : 0.0f);
}

template <class Pass>
__device__ void band_write(const Pass& P, WriterLds& S, const BandCtx& c, int64_t n,
                           float* __restrict__ out, bool all_dense) {
  const int64_t ntiles = (n + kBandTile - 1) / kBandTile;
  const int64_t nt = static_cast<int64_t>(blockIdx.x) < ntiles
                         ? (ntiles - 1 - static_cast<int64_t>(blockIdx.x)) / gridDim.x + 1
                         : 0;
  const int64_t nr = (nt + kRound - 1) / kRound;
  const bool vec_out = (reinterpret_cast<uintptr_t>(out) & 15) == 0;
  const bool vec_in = ((reinterpret_cast<uintptr_t>(P.in0()) |
                        reinterpret_cast<uintptr_t>(P.in1())) & 15) == 0;
  if (threadIdx.x < kStoreWaves * kWave) {
#pragma unroll
    for (int i = 0; i < kRound; ++i) {
      S.tile[0][i][threadIdx.x] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
      S.tile[1][i][threadIdx.x] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    }
    __syncthreads();
    writer_store(P, S, out, n, nt, nr, vec_out, vec_in);
  } else {
    __syncthreads();
    writer_load(P, S, c.tiles, c.ent, nt, nr, all_dense);
  }
}

int writer_blocks(int64_t n) {
  const int64_t ntiles = (n + kBandTile - 1) / kBandTile;
  return static_cast<int>(ntiles < kWriterBlocks ? ntiles : kWriterBlocks);
}

}  // namespace

__global__ __launch_bounds__(WT) void band_emit_kernel(const float* __restrict__ r, int64_t n,
                                                       const SolveRec* __restrict__ rec,
                                                       double inv_t, BandCtx c,
                                                       const uint32_t* __restrict__ ones_all,
                                                       const PartTotals* __restrict__ tot,
                                                       float* __restrict__ p,
                                                       double* __restrict__ b_out) {
  __shared__ WriterLds S;
  if (!rec->ok) return;
  const double b = rec->b;
  // a band as wide as the scores (t large against their spread) leaves most
  // blocks without lists: the whole row is then streamed, here and in the
  // backward (the dense form gives the same values everywhere)
  const bool dense_row = 4 * static_cast<int64_t>(tot->dense_blocks) >= c.nblocks;
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    b_out[0] = b;
    CtxHeader h;
    h.mode = dense_row ? 1 : 0;
    h.nblocks = c.nblocks;
    h.chunk = c.chunk;
    h.cap = c.cap;
    h.pad = 0;
    h.n = n;
    h.b = b;
    *c.hdr = h;
  }
  EmitPass P;
  P.r = r;
  P.ones = tot->aR < INFINITY ? ones_all : nullptr;
  P.b = b;
  P.inv_t = inv_t;
  if (dense_row)
    stream_row(P, n, p);
  else
    band_write(P, S, c, n, p, false);
}

hipError_t launch_band_emit(const float* r, int64_t n, const SolveRec* rec, double t,
                            const BandCtx& band, const uint32_t* ones, const PartTotals* tot,
                            float* p, double* b_out, hipStream_t s) {
  { ProfScope ps_("band_emit", s);
  hipLaunchKernelGGL(band_emit_kernel, dim3(writer_blocks(n)), dim3(WT), 0, s, r, n, rec, 1.0 / t,
                     band, ones, tot, p, b_out); }
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
  h.b = 0.0;
  *c.hdr = h;
}

hipError_t launch_ctx_dense(const BandCtx& band, int64_t n, hipStream_t s) {
  { ProfScope ps_("ctx_dense", s);
  hipLaunchKernelGGL(ctx_dense_kernel, dim3(1), dim3(1), 0, s, band, n); }
  return hipGetLastError();
}

// ---------------------------------------------------------------- backward --
// One wave of a reduce block per partition block; the writer blocks sum the
// reduce partials themselves (fixed order), so no launch sits between.
constexpr int kVjpWaveBlocks = BW;             // partition blocks per reduce block
constexpr int kVjpMaxParts = 4 * BT;           // partials a writer block sums

// With PARAMS each part also carries sum s u and sum s g u (u = (r - b)/t:
// from the score for list members, recovered from p for dense blocks), for
// the budget and temperature gradients.
template <bool PARAMS>
__global__ __launch_bounds__(BT) void band_vjp_reduce_kernel(const float* __restrict__ g,
                                                             const float* __restrict__ p,
                                                             int64_t n, BandCtx c, double inv_t,
                                                             float* __restrict__ gstash,
                                                             double* __restrict__ partials) {
  constexpr int NS = PARAMS ? 4 : 2;
  __shared__ double red[NS][BW];
  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wid = tid / kWave;
  const int pb = static_cast<int>(blockIdx.x) * kVjpWaveBlocks + wid;
  const CtxHeader h = *c.hdr;
  double F = 0.0, G = 0.0, U = 0.0, H = 0.0;
  if (pb < c.nblocks) {
    const BlockRange br = range_of(n, c.chunk, pb);
    if (header_dense(h, c, n) || !lists_usable(c, pb)) {
      // the block's range from p (float4 loads, four per lane in flight; g
      // only where some f != 0); a block starts on a multiple of 4096 scores
      auto add = [&](float pv, float gv) {
        const float f = fminf(pv, 1.0f - pv);
        if (f != 0.0f) {
          const double fg = static_cast<double>(f) * static_cast<double>(gv);
          F += static_cast<double>(f);
          G += fg;
          if constexpr (PARAMS) {
            const double u = static_cast<double>(laplace_u_from_p(pv, f));
            U += static_cast<double>(f) * u;
            H += fg * u;
          }
        }
      };
      const bool vec = ((reinterpret_cast<uintptr_t>(p) | reinterpret_cast<uintptr_t>(g)) & 15) == 0;
      int64_t i = br.b0 + 4 * lane;
      if (vec) {
        constexpr int VU = 4;
        for (; i + 4 * kWave * (VU - 1) + 3 < br.b1; i += 4 * kWave * VU) {
          float4 pv[VU];
#pragma unroll
          for (int u = 0; u < VU; ++u) pv[u] = load_stream4(p + i + 4 * kWave * u);
          // every g load of the batch is issued before any is used: a lane
          // that needs none reads the block's first float4 instead (one
          // line for all such lanes), so that no load sits in a branch that
          // the compiler would fill with its use (a load followed by its use
          // made the next load wait for it)
          float4 gv[VU];
          bool need[VU];
#pragma unroll
          for (int u = 0; u < VU; ++u) {
            const float4 q = pv[u];
            need[u] = (fminf(q.x, 1.0f - q.x) + fminf(q.y, 1.0f - q.y)) +
                          (fminf(q.z, 1.0f - q.z) + fminf(q.w, 1.0f - q.w)) != 0.0f;
            gv[u] = load_stream4(need[u] ? g + i + 4 * kWave * u : g + br.b0);
          }
#pragma unroll
          for (int u = 0; u < VU; ++u) {
            if (need[u]) {
              add(pv[u].x, gv[u].x);
              add(pv[u].y, gv[u].y);
              add(pv[u].z, gv[u].z);
              add(pv[u].w, gv[u].w);
            }
          }
        }
        for (; i + 3 < br.b1; i += 4 * kWave) {
          const float4 q = load_stream4(p + i);
          const float4 gv = load_stream4(g + i);
          add(q.x, gv.x);
          add(q.y, gv.y);
          add(q.z, gv.z);
          add(q.w, gv.w);
        }
        for (int e = 0; e < 4; ++e)
          if (i + e < br.b1) add(p[i + e], g[i + e]);
      } else {
        for (int64_t j = br.b0 + lane; j < br.b1; j += kWave) add(p[j], g[j]);
      }
    } else {
      // the block's members in index order are the four wave segments one
      // after the other; VB members per lane at a time, all their loads
      // (then all the loads of g they select) in flight together; each lane
      // still adds its members in list order
      const int4 cnt = *reinterpret_cast<const int4*>(c.blk[pb].cnt);
      const int s1 = cnt.x, s2 = cnt.x + cnt.y, s3 = cnt.x + cnt.y + cnt.z;
      const int total = s3 + cnt.w;
      const int64_t base = static_cast<int64_t>(pb) * BW * c.cap;
      auto slot_of = [&](int e) -> int64_t {
        const int w = (e >= s1 ? 1 : 0) + (e >= s2 ? 1 : 0) + (e >= s3 ? 1 : 0);
        const int sb = w == 0 ? 0 : (w == 1 ? s1 : (w == 2 ? s2 : s3));
        return base + static_cast<int64_t>(w) * c.cap + (e - sb);
      };
      constexpr int VB = 8;
      for (int e0 = 0; e0 < total; e0 += VB * kWave) {
        BandEntry en[VB];
        int64_t at[VB];
#pragma unroll
        for (int u = 0; u < VB; ++u) {
          const int e = e0 + u * kWave + lane;
          at[u] = slot_of(e < total ? e : 0);
          en[u] = c.ent[at[u]];
        }
        float fv[VB], gv[VB];
        bool use[VB];
#pragma unroll
        for (int u = 0; u < VB; ++u) {
          const int e = e0 + u * kWave + lane;
          const float pv = laplace_p(__uint_as_float(en[u].bits), h.b, inv_t);
          fv[u] = fminf(pv, 1.0f - pv);
          use[u] = e < total && fv[u] != 0.0f && en[u].idx >= br.b0 && en[u].idx < br.b1;
          gv[u] = g[use[u] ? en[u].idx : br.b0];   // an index of this block either way
        }
#pragma unroll
        for (int u = 0; u < VB; ++u) {
          if (use[u]) {
            gstash[at[u]] = gv[u];
            const double fg = static_cast<double>(fv[u]) * static_cast<double>(gv[u]);
            F += static_cast<double>(fv[u]);
            G += fg;
            if constexpr (PARAMS) {
              const double uu =
                  (static_cast<double>(__uint_as_float(en[u].bits)) - h.b) * inv_t;
              U += static_cast<double>(fv[u]) * uu;
              H += fg * uu;
            }
          }
        }
      }
    }
  }
  F = wave_sum(F);
  G = wave_sum(G);
  if constexpr (PARAMS) {
    U = wave_sum(U);
    H = wave_sum(H);
  }
  if (lane == 0) {
    red[0][wid] = F;
    red[1][wid] = G;
    if constexpr (PARAMS) {
      red[2][wid] = U;
      red[3][wid] = H;
    }
  }
  __syncthreads();
  if (tid < NS) {
    double acc = 0.0;
#pragma unroll
    for (int w = 0; w < BW; ++w) acc += red[tid][w];
    partials[NS * blockIdx.x + tid] = acc;
  }
}

// grad_r = (f/t)(g - <g,q>); <g,q> = sum f g / sum f from the partials, 0
// (and grad_r = 0) when sum f == 0.  With PARAMS block 0 also stores
// dL/dk = <g,q> and dL/dalpha = (H - (U/F) G)/t (0 when F == 0).
template <bool PARAMS>
__global__ __launch_bounds__(WT) void band_vjp_write_kernel(const float* __restrict__ g,
                                                            const float* __restrict__ p,
                                                            int64_t n, BandCtx c,
                                                            const float* __restrict__ gstash,
                                                            const double* __restrict__ partials,
                                                            int nparts, double inv_t,
                                                            float* __restrict__ grad,
                                                            double* __restrict__ grad_k,
                                                            double* __restrict__ grad_alpha) {
  constexpr int NS = PARAMS ? 4 : 2;
  __shared__ WriterLds S;
  const int tid = threadIdx.x;
  const CtxHeader h = *c.hdr;
  if (tid < BT) {
    // the partials in a fixed order: thread tid adds parts tid, tid + BT, ...
    double acc[NS];
#pragma unroll
    for (int q = 0; q < NS; ++q) acc[q] = 0.0;
    double2 pr[kVjpMaxParts / BT][NS / 2];
#pragma unroll
    for (int q = 0; q < kVjpMaxParts / BT; ++q) {
      const int i = q * BT + tid;
#pragma unroll
      for (int h2 = 0; h2 < NS / 2; ++h2)
        pr[q][h2] = reinterpret_cast<const double2*>(partials)[(i < nparts ? i : 0) * (NS / 2) + h2];
    }
#pragma unroll
    for (int q = 0; q < kVjpMaxParts / BT; ++q) {
      if (q * BT + tid < nparts) {
#pragma unroll
        for (int h2 = 0; h2 < NS / 2; ++h2) {
          acc[2 * h2] += pr[q][h2].x;
          acc[2 * h2 + 1] += pr[q][h2].y;
        }
      }
    }
#pragma unroll
    for (int q = 0; q < NS; ++q) acc[q] = wave_sum(acc[q]);
    if (lane_id() == 0) {
#pragma unroll
      for (int q = 0; q < NS; ++q) S.red[q][tid / kWave] = acc[q];
    }
  }
  __syncthreads();
  double tot[NS];
#pragma unroll
  for (int q = 0; q < NS; ++q) {
    tot[q] = 0.0;
#pragma unroll
    for (int w = 0; w < BW; ++w) tot[q] += S.red[q][w];
  }
  const double fs = tot[0], gsum = tot[1];
  if constexpr (PARAMS) {
    if (blockIdx.x == 0 && tid == 0) {
      if (grad_k) *grad_k = fs > 0.0 ? gsum / fs : 0.0;
      if (grad_alpha) *grad_alpha = fs > 0.0 ? (tot[3] - (tot[2] / fs) * gsum) * inv_t : 0.0;
    }
  }
  VjpPass P;
  P.p = p;
  P.g = g;
  P.gstash = gstash;
  P.b = h.b;
  P.inv_t = inv_t;
  P.coef = static_cast<float>(fs > 0.0 ? gsum / fs : 0.0);
  P.scale = static_cast<float>(fs > 0.0 ? inv_t : 0.0);
  if (header_dense(h, c, n))
    stream_row(P, n, grad);
  else
    band_write(P, S, c, n, grad, false);
}

int band_vjp_parts(int nblocks) { return (nblocks + kVjpWaveBlocks - 1) / kVjpWaveBlocks; }

hipError_t launch_band_vjp(const float* g, const float* p, int64_t n, const BandCtx& band,
                           float* gstash, double* partials, double t, float* grad,
                           double* grad_k, double* grad_alpha, hipStream_t s) {
  const int parts = band_vjp_parts(band.nblocks);
  if (parts > kVjpMaxParts) return hipErrorInvalidValue;
  const bool params = grad_k || grad_alpha;
  { ProfScope ps_("band_vjp_reduce", s);
  if (params)
    hipLaunchKernelGGL(band_vjp_reduce_kernel<true>, dim3(parts), dim3(BT), 0, s, g, p, n, band,
                       1.0 / t, gstash, partials);
  else
    hipLaunchKernelGGL(band_vjp_reduce_kernel<false>, dim3(parts), dim3(BT), 0, s, g, p, n, band,
                       1.0 / t, gstash, partials); }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  { ProfScope ps_("band_vjp_emit", s);
  if (params)
    hipLaunchKernelGGL(band_vjp_write_kernel<true>, dim3(writer_blocks(n)), dim3(WT), 0, s, g, p,
                       n, band, gstash, partials, parts, 1.0 / t, grad, grad_k, grad_alpha);
  else
    hipLaunchKernelGGL(band_vjp_write_kernel<false>, dim3(writer_blocks(n)), dim3(WT), 0, s, g, p,
                       n, band, gstash, partials, parts, 1.0 / t, grad, grad_k, grad_alpha); }
  return hipGetLastError();
}

}  // namespace lapsum
