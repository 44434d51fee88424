// Device-wide stable LSD radix sort of one array into descending float order
// (the sort step of the full-sort solver, §1/§3, and of the middle band M,
// Suppl. B).  Up to four passes of 8-bit digits; each pass is
//   upsweep    per-tile digit counts                               read keys
//   scan       per digit, exclusive prefix of the counts over tiles (folded
//              into the downsweep when there are at most 64 tiles)
//   downsweep  stable rank inside the tile (ballot digit matching),
//              staged through LDS so that each digit run leaves the tile as
//              a contiguous burst                                  read + write
// Tiles hold 1024 keys for inputs up to 393216 keys (shorter serial ranking
// per block), 2048 up to 2^20 keys and 4096 above.  Passes whose digit is
// the same for every key are skipped (the caller knows the leading bytes all
// keys share).  Ties keep their input order (tile order, then position
// inside the tile), which for the first pass is the original index: the
// sort is stable.
#include "block_sort.hpp"
#include "kernels.hpp"

namespace lapsum {

namespace {

constexpr int TT = kTileThreads;           // 256
constexpr int TW = TT / kWave;             // 4 waves
constexpr int kFusedScanTiles = 64;

struct PassArgs {
  const float* src_f;      // pass 0 from floats, else null
  const uint32_t* src_k;
  const int32_t* src_v;    // null => values are source positions (mode 1)
  uint32_t* dst_k;
  int32_t* dst_v;          // null => keys only
  int64_t len;
  const int64_t* len_dev;
  uint32_t* hist;          // [256][max_tiles]
  uint32_t* totals;        // [256]
  int64_t max_tiles;
  int shift;
};

__device__ __forceinline__ int64_t eff_len(const PassArgs& a) {
  if (a.len_dev == nullptr) return a.len;
  const int64_t d = *a.len_dev;
  return d < a.len ? (d < 0 ? 0 : d) : a.len;
}

__device__ __forceinline__ uint32_t load_key(const PassArgs& a, int64_t i) {
  return a.src_f ? desc_key(a.src_f[i]) : a.src_k[i];
}

// position of item i of this thread inside the tile (wave-striped)
template <int TI>
__device__ __forceinline__ int tile_pos(int i) {
  return (threadIdx.x / kWave) * (kWave * TI) + i * kWave + lane_id();
}

}  // namespace

// Per-tile digit counts (the order is the downsweep's): one LDS atomic per
// key on counters of its own wave, cheaper than matching the digit across
// the wave (36 -> 22 us per pass over 1e7 keys).  Counting does not depend on
// which thread holds which key, so the keys are read four at a time (16-byte
// loads: 17 -> 12 us per pass over 1e7 keys in a probe).
//   TPB  tiles per block, one group of TT threads each.  With four, each
//        digit's four counts leave as one 16-byte store: the histogram is
//        digit-major, so one count per tile is a scattered 4-byte store
//        (12.1 -> 11.4 us per pass over 1e7 spread digits; 60 -> 45 MB of
//        HBM traffic).
//   QS   counter sets per wave.  The leading digit of float keys takes few
//        values, and lanes adding to one LDS address are served one after
//        another; with a set per quarter wave a hot digit spreads over four
//        addresses (22.9 -> 17.2 us on the leading digit of 1e7 |Laplace|
//        keys; on spread digits it costs 0.6 us, so only that pass uses it).
template <int TI, int TPB, int QS>
__global__ __launch_bounds__(TT * TPB) void sort_upsweep_kernel(PassArgs a) {
  constexpr int64_t TILE = static_cast<int64_t>(TT) * TI;
  constexpr int SETS = TW * QS;
  const int64_t len = eff_len(a);
  const int64_t ntiles = (len + TILE - 1) / TILE;
  const int64_t tile0 = static_cast<int64_t>(blockIdx.x) * TPB;
  if (tile0 >= ntiles) return;
  __shared__ uint32_t cnt[TPB][cnt_words<SETS>()];
  const int tid = threadIdx.x;
  const int grp = tid / TT;
  const int gt = tid % TT;
  const int lane = lane_id();
  const int set = (gt / kWave) * QS + lane / (kWave / QS);
  for (int e = tid; e < TPB * cnt_words<SETS>(); e += TT * TPB) (&cnt[0][0])[e] = 0u;
  __syncthreads();
  const int64_t tile = tile0 + grp;
  const int64_t base = tile * TILE;
  const void* src = a.src_f ? static_cast<const void*>(a.src_f) : static_cast<const void*>(a.src_k);
  uint32_t* c = cnt[grp];
  auto count = [&](uint32_t key) { atomicAdd(&c[cnt_at<SETS>((key >> a.shift) & 255u, set)], 1u); };
  if (tile < ntiles) {
    const bool vec = (reinterpret_cast<uintptr_t>(src) & 15) == 0;
    if (vec) {
      constexpr int V = TI / 4;
      static_assert(TI % 4 == 0, "four keys per load");
      uint4 q[V];
#pragma unroll
      for (int j = 0; j < V; ++j) {
        const int64_t at = base + 4 * (static_cast<int64_t>(j) * TT + gt);
        q[j] = at + 3 < len ? *reinterpret_cast<const uint4*>(static_cast<const uint32_t*>(src) + at)
                            : make_uint4(0u, 0u, 0u, 0u);
      }
#pragma unroll
      for (int j = 0; j < V; ++j) {
        const int64_t at = base + 4 * (static_cast<int64_t>(j) * TT + gt);
        if (at + 3 < len) {
          const uint32_t w[4] = {q[j].x, q[j].y, q[j].z, q[j].w};
#pragma unroll
          for (int e = 0; e < 4; ++e) count(a.src_f ? desc_key(__uint_as_float(w[e])) : w[e]);
        } else {
          for (int e = 0; e < 4; ++e)
            if (at + e < len) count(load_key(a, at + e));
        }
      }
    } else {
      // a source not 16-byte aligned (a row of a batch whose length is not
      // a multiple of 4): one word per load, all issued before any key is
      // formed
      const uint32_t* sw = static_cast<const uint32_t*>(src);
      uint32_t w[TI];
#pragma unroll
      for (int i = 0; i < TI; ++i) {
        const int64_t pos = base + i * TT + gt;
        w[i] = sw[pos < len ? pos : base];
      }
#pragma unroll
      for (int i = 0; i < TI; ++i) {
        if (base + i * TT + gt < len) count(a.src_f ? desc_key(__uint_as_float(w[i])) : w[i]);
      }
    }
  }
  __syncthreads();
  if (tid < 256) {
    uint32_t sum[TPB];
#pragma unroll
    for (int g = 0; g < TPB; ++g) {
      sum[g] = 0u;
#pragma unroll
      for (int w = 0; w < SETS; ++w) sum[g] += cnt[g][cnt_at<SETS>(tid, w)];
    }
    uint32_t* h = a.hist + static_cast<int64_t>(tid) * a.max_tiles + tile0;
    if constexpr (TPB == 4)
      *reinterpret_cast<uint4*>(h) = make_uint4(sum[0], sum[1], sum[2], sum[3]);   // max_tiles % 4 == 0
    else
      h[0] = sum[0];
  }
}

// One block per digit: exclusive prefix of hist[d][0..ntiles) in place.
template <int TI>
__global__ __launch_bounds__(TT) void sort_scan_kernel(PassArgs a) {
  constexpr int64_t TILE = static_cast<int64_t>(TT) * TI;
  const int64_t len = eff_len(a);
  const int64_t ntiles = (len + TILE - 1) / TILE;
  const int d = blockIdx.x;
  __shared__ uint32_t wtot[TW];
  uint32_t* h = a.hist + static_cast<int64_t>(d) * a.max_tiles;
  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wid = tid / kWave;
  uint32_t carry = 0;
  for (int64_t c0 = 0; c0 < ntiles; c0 += 4 * TT) {
    uint32_t v[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int64_t idx = c0 + 4 * tid + q;
      v[q] = idx < ntiles ? h[idx] : 0u;
    }
    const uint32_t sum = v[0] + v[1] + v[2] + v[3];
    uint32_t incl = sum;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
      const uint32_t x = __shfl_up(incl, o, kWave);
      if (lane >= o) incl += x;
    }
    if (lane == kWave - 1) wtot[wid] = incl;
    __syncthreads();
    uint32_t wbase = 0, all = 0;
#pragma unroll
    for (int w = 0; w < TW; ++w) {
      if (w < wid) wbase += wtot[w];
      all += wtot[w];
    }
    uint32_t ex = carry + wbase + incl - sum;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int64_t idx = c0 + 4 * tid + q;
      if (idx < ntiles) h[idx] = ex;
      ex += v[q];
    }
    carry += all;
    __syncthreads();
  }
  if (tid == 0) a.totals[d] = carry;
}

// The same scan in one round for rows of at most C * TT tiles: thread tid
// holds tiles C tid .. C tid + C - 1, read and written as 16-byte groups
// (histogram rows are 16-byte aligned and padded to a multiple of 4 tiles;
// entries past ntiles are read as zero and written with values nobody
// reads), instead of rounds of 1024 tiles that each wait for their loads:
// 4.9 against 5.0 us per pass at 2442 tiles, 2.6 against 3.0 at 489.
template <int TI, int C>
__global__ __launch_bounds__(TT) void sort_scan1_kernel(PassArgs a) {
  static_assert(C % 4 == 0, "16-byte groups");
  constexpr int64_t TILE = static_cast<int64_t>(TT) * TI;
  const int64_t len = eff_len(a);
  const int64_t ntiles = (len + TILE - 1) / TILE;
  const int d = blockIdx.x;
  __shared__ uint32_t wtot[TW];
  uint4* h = reinterpret_cast<uint4*>(a.hist + static_cast<int64_t>(d) * a.max_tiles);
  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wid = tid / kWave;
  const int64_t t0 = static_cast<int64_t>(tid) * C;
  uint32_t v[C];
#pragma unroll
  for (int j = 0; j < C / 4; ++j) {
    const int64_t at = t0 + 4 * j;
    const uint4 q = at < ntiles ? h[at / 4] : make_uint4(0u, 0u, 0u, 0u);
    v[4 * j] = q.x;
    v[4 * j + 1] = at + 1 < ntiles ? q.y : 0u;
    v[4 * j + 2] = at + 2 < ntiles ? q.z : 0u;
    v[4 * j + 3] = at + 3 < ntiles ? q.w : 0u;
  }
  uint32_t sum = 0;
#pragma unroll
  for (int j = 0; j < C; ++j) sum += v[j];
  uint32_t incl = sum;
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const uint32_t x = __shfl_up(incl, o, kWave);
    if (lane >= o) incl += x;
  }
  if (lane == kWave - 1) wtot[wid] = incl;
  __syncthreads();
  uint32_t ex = incl - sum, all = 0;
#pragma unroll
  for (int w = 0; w < TW; ++w) {
    if (w < wid) ex += wtot[w];
    all += wtot[w];
  }
#pragma unroll
  for (int j = 0; j < C / 4; ++j) {
    const int64_t at = t0 + 4 * j;
    uint4 q;
    q.x = ex;
    ex += v[4 * j];
    q.y = ex;
    ex += v[4 * j + 1];
    q.z = ex;
    ex += v[4 * j + 2];
    q.w = ex;
    ex += v[4 * j + 3];
    if (at < ntiles) h[at / 4] = q;
  }
  if (tid == 0) a.totals[d] = all;
}

// Stable ranks of one tile's keys and their scatter: keys (and values) in
// registers, wave-striped; `off` holds each digit's first output position
// for this tile on entry and becomes the offset from a tile-local position
// to its output position (unsigned arithmetic, so the difference may wrap).
// FULL tiles (every position valid) skip the validity masks.
template <int TI, bool PAIRS, bool FULL>
__device__ __forceinline__ void downsweep_tile(const PassArgs& a, int64_t base, int64_t len,
                                               uint32_t (&key)[TI], int32_t (&val)[TI],
                                               uint32_t* cnt, uint32_t* wave_tot, uint32_t* off,
                                               uint32_t* buf, uint8_t* dg) {
  constexpr int64_t TILE = static_cast<int64_t>(TT) * TI;
  const int tid = threadIdx.x;
  const int wid = tid / kWave;
  const int lane = lane_id();
  uint32_t pos[TI];
  uint64_t validm[TI];
#pragma unroll
  for (int i = 0; i < TI; ++i) validm[i] = FULL ? ~0ull : __ballot(base + tile_pos<TI>(i) < len);
#pragma unroll
  for (int i = 0; i < TI; ++i) {
    const uint32_t d = (key[i] >> a.shift) & 255u;
    const uint64_t peers = FULL ? match_digit8(d) : (match_digit8(d) & validm[i]);
    const uint32_t below = lanes_below(peers);
    uint32_t* slot = &cnt[cnt_at<TW>(d, wid)];
    const uint32_t c = *slot;
    pos[i] = c + below;
    const bool valid = FULL || ((validm[i] >> lane) & 1ull);
    if (valid && below == 0u) *slot = c + static_cast<uint32_t>(__popcll(peers));
  }
  __syncthreads();
  block_excl_scan_u32x4<TT>(cnt, wave_tot);
  // output position of tile-local position q with digit d: off[d] + q
  off[tid] -= cnt[cnt_at<TW>(tid, 0)];
#pragma unroll
  for (int i = 0; i < TI; ++i) {
    pos[i] += cnt[cnt_at<TW>((key[i] >> a.shift) & 255u, wid)];
    if (FULL || ((validm[i] >> lane) & 1ull)) buf[pos[i]] = key[i];
  }
  __syncthreads();
  const int nvalid = FULL ? static_cast<int>(TILE) : static_cast<int>(len - base);
  for (int q = tid; q < nvalid; q += TT) {
    const uint32_t k = buf[q];
    const uint32_t d = (k >> a.shift) & 255u;
    a.dst_k[off[d] + static_cast<uint32_t>(q)] = k;
    if constexpr (PAIRS) dg[q] = static_cast<uint8_t>(d);
  }
  if constexpr (PAIRS) {
    __syncthreads();
#pragma unroll
    for (int i = 0; i < TI; ++i)
      if (FULL || ((validm[i] >> lane) & 1ull)) buf[pos[i]] = static_cast<uint32_t>(val[i]);
    __syncthreads();
    for (int q = tid; q < nvalid; q += TT)
      a.dst_v[off[dg[q]] + static_cast<uint32_t>(q)] = static_cast<int32_t>(buf[q]);
  }
}

template <int TI, bool PAIRS, bool FUSED>
__global__ __launch_bounds__(TT) void sort_downsweep_kernel(PassArgs a) {
  constexpr int64_t TILE = static_cast<int64_t>(TT) * TI;
  const int64_t len = eff_len(a);
  const int64_t ntiles = (len + TILE - 1) / TILE;
  const int64_t tile = blockIdx.x;
  if (tile >= ntiles) return;
  __shared__ uint32_t cnt[cnt_words<TW>()];
  __shared__ uint32_t wave_tot[TW];
  __shared__ uint32_t off[256];      // first output position of each digit for this tile
  __shared__ uint32_t buf[TILE];
  __shared__ uint8_t dg[PAIRS ? TILE : 1];   // digit of each tile-local position
  const int tid = threadIdx.x;
  const int wid = tid / kWave;
  const int lane = lane_id();
  const int64_t base = tile * TILE;
  const bool full = base + TILE <= len;

  // the tile's raw words first, so that their latency overlaps the digit
  // bases; keys are formed from them (floats, and the sentinel past the end)
  // only after that.  Forming each key right after its own load made every
  // load wait for the previous one in the pass from floats.  Full tiles need
  // no bounds.
  const bool from_f = a.src_f != nullptr;
  uint32_t key[TI];
  int32_t val[TI];
  {
    const uint32_t* src = from_f ? reinterpret_cast<const uint32_t*>(a.src_f) : a.src_k;
    if (full) {
      const uint32_t* ts = src + base;
#pragma unroll
      for (int i = 0; i < TI; ++i) key[i] = ts[tile_pos<TI>(i)];
    } else {
#pragma unroll
      for (int i = 0; i < TI; ++i) {
        const int64_t gp = base + tile_pos<TI>(i);
        key[i] = gp < len ? src[gp] : 0u;
      }
    }
    if constexpr (PAIRS) {
#pragma unroll
      for (int i = 0; i < TI; ++i) {
        const int64_t gp = base + tile_pos<TI>(i);
        val[i] = gp < len ? (a.src_v ? a.src_v[gp] : static_cast<int32_t>(gp)) : -1;
      }
    }
  }

  // digit base over the whole array: exclusive prefix of totals over digits
  {
    uint32_t tot, before_tile;
    if constexpr (FUSED) {
      // few tiles: this digit's total and its count in earlier tiles
      const uint32_t* h = a.hist + static_cast<int64_t>(tid) * a.max_tiles;
      tot = 0;
      before_tile = 0;
      for (int64_t q0 = 0; q0 < ntiles; q0 += 8) {   // eight independent loads in flight
        uint32_t c[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) c[u] = (q0 + u < ntiles) ? h[q0 + u] : 0u;
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          if (q0 + u < tile) before_tile += c[u];
          tot += c[u];
        }
      }
    } else {
      tot = a.totals[tid];
      before_tile = a.hist[static_cast<int64_t>(tid) * a.max_tiles + tile];
    }
    uint32_t incl = tot;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
      const uint32_t x = __shfl_up(incl, o, kWave);
      if (lane >= o) incl += x;
    }
    if (lane == kWave - 1) wave_tot[wid] = incl;
    __syncthreads();
    uint32_t wbase = 0;
#pragma unroll
    for (int w = 0; w < TW; ++w)
      if (w < wid) wbase += wave_tot[w];
    off[tid] = wbase + incl - tot + before_tile;
  }
  for (int e = tid; e < cnt_words<TW>(); e += TT) cnt[e] = 0u;
  if (full) {
    if (from_f) {
#pragma unroll
      for (int i = 0; i < TI; ++i) key[i] = desc_key(__uint_as_float(key[i]));
    }
  } else {
#pragma unroll
    for (int i = 0; i < TI; ++i) {
      const bool valid = base + tile_pos<TI>(i) < len;
      key[i] = !valid ? 0xffffffffu : (from_f ? desc_key(__uint_as_float(key[i])) : key[i]);
    }
  }
  __syncthreads();
  if (full)
    downsweep_tile<TI, PAIRS, true>(a, base, len, key, val, cnt, wave_tot, off, buf, dg);
  else
    downsweep_tile<TI, PAIRS, false>(a, base, len, key, val, cnt, wave_tot, off, buf, dg);
}

int64_t sort_max_tiles(int64_t len) {
  // sized for the smallest tile, a multiple of 4 so that every histogram row
  // is 16-byte aligned for the four-tile counting blocks
  const int64_t tiles = (len + 1023) / 1024;
  return ((tiles < 1 ? 1 : tiles) + 3) / 4 * 4;
}

size_t sort_hist_words(int64_t len) {
  return static_cast<size_t>(256) * static_cast<size_t>(sort_max_tiles(len));
}

namespace {
template <int TI>
hipError_t sort_passes(const float* src_f, const uint32_t* src_k, const int32_t* src_v,
                       bool with_vals, int64_t len, const int64_t* len_dev, SortBuffers& sb,
                       unsigned pass_mask, const uint32_t** keys_out, const int32_t** vals_out,
                       hipStream_t s) {
  constexpr int64_t TILE = static_cast<int64_t>(TT) * TI;
  const int64_t tiles = (len + TILE - 1) / TILE;
  if (tiles > sb.max_tiles) return hipErrorInvalidValue;
  const unsigned grid = static_cast<unsigned>(tiles < 1 ? 1 : tiles);
  const bool fused = tiles <= kFusedScanTiles && len_dev == nullptr;
  const uint32_t* cur_k = src_k;
  const int32_t* cur_v = src_v;
  const float* cur_f = src_f;
  int nxt = 0;
  // the leading digit that varies: the one whose values crowd onto a few
  // counters (the sign and exponent bits of float keys)
  int lead = 0;
  for (int pass = 1; pass < 4; ++pass)
    if (pass_mask & (1u << pass)) lead = pass;
  for (int pass = 0; pass < 4; ++pass) {
    if (!(pass_mask & (1u << pass)) && cur_f == nullptr) continue;   // digit shared by all keys
    PassArgs a{};
    a.len = len;
    a.len_dev = len_dev;
    a.hist = sb.hist;
    a.totals = sb.totals;
    a.max_tiles = sb.max_tiles;
    a.shift = 8 * pass;
    a.src_f = cur_f;
    a.src_k = cur_k;
    a.src_v = cur_v;
    a.dst_k = sb.keys[nxt];
    a.dst_v = with_vals ? sb.vals[nxt] : nullptr;
    {
      ProfScope ps_("sort_upsweep", s);
      bool four = false;   // four tiles per block: only with enough blocks to fill the device
      if constexpr (TI == 16) four = pass != lead && tiles >= 1024;
      if (pass == lead)
        hipLaunchKernelGGL((sort_upsweep_kernel<TI, 1, 4>), dim3(grid), dim3(TT), 0, s, a);
      else if (four) {
        if constexpr (TI == 16)
          hipLaunchKernelGGL((sort_upsweep_kernel<TI, 4, 1>), dim3(static_cast<unsigned>((tiles + 3) / 4)),
                             dim3(4 * TT), 0, s, a);
      } else
        hipLaunchKernelGGL((sort_upsweep_kernel<TI, 1, 1>), dim3(grid), dim3(TT), 0, s, a);
    }
    if (!fused) {
      ProfScope ps_("sort_scan", s);
      const int64_t per = (tiles + TT - 1) / TT;   // tiles per scan thread
      if (per <= 4)
        hipLaunchKernelGGL((sort_scan1_kernel<TI, 4>), dim3(256), dim3(TT), 0, s, a);
      else if (per <= 8)
        hipLaunchKernelGGL((sort_scan1_kernel<TI, 8>), dim3(256), dim3(TT), 0, s, a);
      else if (per <= 16)
        hipLaunchKernelGGL((sort_scan1_kernel<TI, 16>), dim3(256), dim3(TT), 0, s, a);
      else
        hipLaunchKernelGGL((sort_scan_kernel<TI>), dim3(256), dim3(TT), 0, s, a);
    }
    {
      ProfScope ps_("sort_downsweep", s);
      if (with_vals) {
        if (fused) hipLaunchKernelGGL((sort_downsweep_kernel<TI, true, true>), dim3(grid), dim3(TT), 0, s, a);
        else hipLaunchKernelGGL((sort_downsweep_kernel<TI, true, false>), dim3(grid), dim3(TT), 0, s, a);
      } else {
        if (fused) hipLaunchKernelGGL((sort_downsweep_kernel<TI, false, true>), dim3(grid), dim3(TT), 0, s, a);
        else hipLaunchKernelGGL((sort_downsweep_kernel<TI, false, false>), dim3(grid), dim3(TT), 0, s, a);
      }
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    cur_f = nullptr;
    cur_k = sb.keys[nxt];
    cur_v = with_vals ? sb.vals[nxt] : nullptr;
    nxt ^= 1;
  }
  *keys_out = cur_k;
  if (vals_out) *vals_out = cur_v;
  return hipSuccess;
}
}  // namespace

hipError_t launch_sort(const float* src_f, const uint32_t* src_k, const int32_t* src_v,
                       bool with_vals, int64_t len, const int64_t* len_dev, SortBuffers& sb,
                       unsigned pass_mask, const uint32_t** keys_out, const int32_t** vals_out,
                       hipStream_t s) {
  // tile size by row length (forward + backward of one Gaussian row, 1024
  // against 2048 keys per tile: 72.8 / 74.9 us at 262145 keys, 80.0 / 81.3
  // at 4e5, 91.7 / 97.5 at 2^20)
  if (len <= int64_t(384) * 1024)
    return sort_passes<4>(src_f, src_k, src_v, with_vals, len, len_dev, sb, pass_mask, keys_out,
                          vals_out, s);
  if (len <= (int64_t(1) << 20))
    return sort_passes<8>(src_f, src_k, src_v, with_vals, len, len_dev, sb, pass_mask, keys_out,
                          vals_out, s);
  return sort_passes<16>(src_f, src_k, src_v, with_vals, len, len_dev, sb, pass_mask, keys_out,
                         vals_out, s);
}

}  // namespace lapsum
