// Threshold solve on a sorted array (descending keys), device-wide.
//
// The node curve N_i = LapSum(s_i) is non-decreasing, so the interval that
// holds b lies in exactly one tile: only that tile needs per-position node
// values.  Two kernels:
//   solve_tiles     one block per 4096-key tile: the tile's summaries
//                   Pre = (last, sum e^{-(s-last)/t}) and
//                   Suf = (first, 1 + sum_{after first} e^{-(first-s)/t}),
//                   every term relative to the tile's own anchor
//   solve_finalize  one block: shift-carrying scans over the tile summaries
//                   from both ends (seeded with the bracket tails), the node
//                   value at each tile's first score, the crossing tile, and
//                   block_solve on that tile; for a bracket also the
//                   certificate LapSum(a_R) <= k <= LapSum(a_L) from the totals
//                   (Suppl. B / Suppl. C)
// Reads the sorted keys once plus one tile: 4 bytes per score.
//
// For |M| <= 32768 one workgroup sorts M on chip and solves it in a single
// launch (small_m_solve).
#include <math.h>

#include "block_sort.hpp"
#include "kernels.hpp"
#include "solve_common.hpp"

namespace lapsum {

namespace {
constexpr int TT = kTileThreads;
constexpr int TI = kTileItems;
constexpr int64_t TILE = kTile;
// The tile records are stored field by field (kTileRec arrays of max_tiles
// doubles), so that the lanes of a wave reading the records of neighbouring
// tiles read neighbouring words: S, X, first, last, then e^{-(first - last)/t}
// (the wide finalize) or the suffix after (v, T) and the prefix before (u, S)
// (the finalize of longer rows).
constexpr int kTileRec = 8;
static_assert(kTileRec == kSolveTileDoubles, "the caller's tile buffer holds kTileRec arrays");
enum TileField { kFS = 0, kFX, kFFirst, kFLast, kFSpan, kFAfterV = 4, kFAfterT, kFBeforeU, kFBeforeS };

__device__ __forceinline__ int64_t eff_len(int64_t len, const int64_t* len_dev) {
  if (len_dev == nullptr) return len;
  const int64_t d = *len_dev;
  return d < len ? (d < 0 ? 0 : d) : len;
}

template <int WAVES>
__device__ int64_t block_max_i64(int64_t v, int64_t* scratch) {
#pragma unroll
  for (int o = kWave / 2; o >= 1; o >>= 1) {
    const int64_t w = __shfl_xor(v, o, kWave);
    v = w > v ? w : v;
  }
  if (lane_id() == 0) scratch[threadIdx.x / kWave] = v;
  __syncthreads();
  v = 0;
#pragma unroll
  for (int w = 0; w < WAVES; ++w) v = scratch[w] > v ? scratch[w] : v;
  __syncthreads();
  return v;
}

}  // namespace

__global__ __launch_bounds__(TT) void solve_tiles_kernel(const uint32_t* __restrict__ keys,
                                                         int64_t len, const int64_t* len_dev,
                                                         double t, double* __restrict__ tiles,
                                                         int64_t mt) {
  const int64_t m = eff_len(len, len_dev);
  const int64_t ntiles = (m + TILE - 1) / TILE;
  const int64_t tile = blockIdx.x;
  if (tile >= ntiles) return;
  __shared__ double red[2][TT / kWave];
  const int tid = threadIdx.x;
  const int64_t base = tile * TILE;
  const int64_t nv = (m - base) < TILE ? (m - base) : TILE;
  const double first = key_float(keys[base]);
  const double last = key_float(keys[base + nv - 1]);
  const double c2 = kLog2e / t;
  double S = 0.0, X = 0.0;
  const int64_t p0 = base + static_cast<int64_t>(tid) * TI;
  uint32_t kv[TI];
  if (nv == TILE && ((reinterpret_cast<uintptr_t>(keys) & 15) == 0)) {
    const uint4* k4 = reinterpret_cast<const uint4*>(keys + p0);
#pragma unroll
    for (int q = 0; q < TI / 4; ++q) {
      const uint4 v = k4[q];
      kv[4 * q + 0] = v.x;
      kv[4 * q + 1] = v.y;
      kv[4 * q + 2] = v.z;
      kv[4 * q + 3] = v.w;
    }
  } else {
#pragma unroll
    for (int i = 0; i < TI; ++i)
      kv[i] = (static_cast<int64_t>(tid) * TI + i < nv) ? keys[p0 + i] : 0u;
  }
#pragma unroll
  for (int i = 0; i < TI; ++i) {
    if (static_cast<int64_t>(tid) * TI + i < nv) {
      const double s = key_float(kv[i]);
      S += wexp_f32(s - last, c2);
      if (tid * TI + i > 0) X += wexp_f32(first - s, c2);
    }
  }
  S = wave_sum(S);
  X = wave_sum(X);
  const int wid = tid / kWave;
  if (lane_id() == 0) {
    red[0][wid] = S;
    red[1][wid] = X;
  }
  __syncthreads();
  if (tid == 0) {
    double s = 0.0, x = 0.0;
#pragma unroll
    for (int w = 0; w < TT / kWave; ++w) {
      s += red[0][w];
      x += red[1][w];
    }
    tiles[kFS * mt + tile] = s;
    tiles[kFX * mt + tile] = x;
    tiles[kFFirst * mt + tile] = first;
    tiles[kFLast * mt + tile] = last;
    tiles[kFSpan * mt + tile] = wexp_f64(first - last, 1.0 / t);   // the link across the tile
  }
}

__global__ __launch_bounds__(TT) void solve_finalize_kernel(SolveArgs a, double* b_out) {
  constexpr int WAVES = TT / kWave;
  __shared__ ScanSmem<WAVES> sm;
  __shared__ int64_t cnt_s[WAVES];
  __shared__ Pre tile_pre_s;
  __shared__ Suf tile_suf_s;
  const int tid = threadIdx.x;
  const double t = a.t;
  const double inv_t = 1.0 / t;
  const double k = a.k;
  const int64_t m = eff_len(a.len, a.len_dev);
  const int64_t ntiles = (m + TILE - 1) / TILE;
  const Tails x = load_tails(a.tails);
  double* tb = a.tile_buf;
  const int64_t mt = a.max_tiles;
  auto F = [&](int f, int64_t q) -> double& { return tb[f * mt + q]; };

  Pre pre_all;
  Suf suf_all;
  int64_t below = 0;
  if (ntiles <= TT) {
    // at most one tile per thread: its record stays in registers
    const bool has = tid < ntiles;
    double S = 0.0, X = 0.0, first = 0.0, last = 0.0;
    if (has) {
      S = F(kFS, tid);
      X = F(kFX, tid);
      first = F(kFFirst, tid);
      last = F(kFLast, tid);
    }
    const Pre mp = has ? Pre{static_cast<float>(last), S} : pre_empty();
    const Suf ms = has ? Suf{static_cast<float>(first), 1.0 + X} : suf_empty();
    Pre pre_in;
    Suf suf_in;
    block_excl_pre_suf<WAVES>(mp, x.pre, ms, x.suf, inv_t, sm, &pre_in, &pre_all, &suf_in, &suf_all);
    if (has) {
      double P = 1.0;
      if (pre_in.S != 0.0) P += wexp_f64(static_cast<double>(pre_in.u) - first, inv_t) * pre_in.S;
      double E = X;
      if (suf_in.T != 0.0) E += wexp_f64(first - static_cast<double>(suf_in.v), inv_t) * suf_in.T;
      const double N = x.nR + static_cast<double>(tid) * TILE + 1.0 - 0.5 * P + 0.5 * E;
      if (N <= k) below = tid + 1;
    }
    below = block_max_i64<WAVES>(below, cnt_s);
    if (below > 0 && tid == below - 1) {
      tile_pre_s = pre_in;
      tile_suf_s = suf_in;
    }
    __syncthreads();
  } else {
    // 1. this thread's run of tiles
    const int64_t per = (ntiles + TT - 1) / TT;
    const int64_t t0 = static_cast<int64_t>(tid) * per;
    const int64_t t1 = (t0 + per < ntiles) ? t0 + per : ntiles;
    Pre mp = pre_empty();
    Suf ms = suf_empty();
    for (int64_t q = t0; q < t1; ++q) {
      mp = pre_combine(mp, Pre{static_cast<float>(F(kFLast, q)), F(kFS, q)}, inv_t);
    }
    for (int64_t q = t1 - 1; q >= t0; --q) {
      ms = suf_combine(Suf{static_cast<float>(F(kFFirst, q)), 1.0 + F(kFX, q)}, ms, inv_t);
    }
    Pre pre_in;
    Suf suf_in;
    block_excl_pre_suf<WAVES>(mp, x.pre, ms, x.suf, inv_t, sm, &pre_in, &pre_all, &suf_in, &suf_all);

    // 2. suffix carried into each tile from the right (stored), then the
    //    node value at each tile's first score walking left to right
    {
      Suf after = suf_in;
      for (int64_t q = t1 - 1; q >= t0; --q) {
        F(kFAfterV, q) = after.v;
        F(kFAfterT, q) = after.T;
        after = suf_combine(Suf{static_cast<float>(F(kFFirst, q)), 1.0 + F(kFX, q)}, after, inv_t);
      }
    }
    {
      Pre before = pre_in;
      for (int64_t q = t0; q < t1; ++q) {
        F(kFBeforeU, q) = before.u;
        F(kFBeforeS, q) = before.S;
        const double first = F(kFFirst, q);
        double P = 1.0;
        if (before.S != 0.0) P += wexp_f64(static_cast<double>(before.u) - first, inv_t) * before.S;
        double E = F(kFX, q);
        if (F(kFAfterT, q) != 0.0) E += wexp_f64(first - F(kFAfterV, q), inv_t) * F(kFAfterT, q);
        const double N = x.nR + static_cast<double>(q * TILE) + 1.0 - 0.5 * P + 0.5 * E;
        if (N <= k) below = q + 1;   // non-decreasing: the last such tile
        before = pre_combine(before, Pre{static_cast<float>(F(kFLast, q)), F(kFS, q)}, inv_t);
      }
    }
    below = block_max_i64<WAVES>(below, cnt_s);
    if (below > 0 && tid == 0) {
      tile_pre_s = Pre{static_cast<float>(F(kFBeforeU, below - 1)), F(kFBeforeS, below - 1)};
      tile_suf_s = Suf{static_cast<float>(F(kFAfterV, below - 1)), F(kFAfterT, below - 1)};
    }
    __syncthreads();
  }

  SolveRec rec;
  rec.ok = 1;
  rec.side = 0;
  rec.lap_aL = 0.0;
  rec.lap_aR = 0.0;
  if (x.bracketed) {
    // pre_all / suf_all already include the tails
    certify(x, static_cast<double>(m), static_cast<double>(a.n_total), k, t, pre_all, suf_all, rec);
  }

  double b;
  if (m == 0 || below == 0) {
    b = root_above(x, suf_all, k, t);
  } else {
    const int64_t ct = below - 1;
    __syncthreads();
    const Pre tp = tile_pre_s;
    const Suf ts = tile_suf_s;
    const int64_t base = ct * TILE;
    const int64_t nv = (m - base) < TILE ? (m - base) : TILE;
    float s[TI];
    int cnt = static_cast<int>(nv - static_cast<int64_t>(tid) * TI);
    cnt = cnt < 0 ? 0 : (cnt > TI ? TI : cnt);
#pragma unroll
    for (int i = 0; i < TI; ++i)
      s[i] = (i < cnt) ? key_float(a.keys[base + static_cast<int64_t>(tid) * TI + i]) : 0.0f;
    Pre pt;
    Suf st;
    b = block_solve<TT, TI>(s, cnt, x.nR + static_cast<double>(base), tp, ts, k, t, sm, &pt, &st);
  }
  if (tid == 0) {
    rec.b = b;
    *a.out = rec;
    if (b_out) *b_out = b;
  }
}

// The same as solve_finalize_kernel for up to kFinPer * FT tiles, by FT =
// 512 threads with each thread's run of at most kFinPer tiles in registers:
// all tile records are loaded at once, every exponential (the links between
// the run's anchors and the node terms) is formed independently, and the
// chains along a run are fused multiply-adds only.  The crossing tile is
// solved by block_solve with 512 threads of 8 keys.
constexpr int FT = 512;
constexpr int FW = FT / kWave;
constexpr int kFinPer = 8;
constexpr int FTI = static_cast<int>(TILE / FT);   // 8 keys per thread in the crossing tile

__global__ __launch_bounds__(FT) void solve_finalize_wide_kernel(SolveArgs a, double* b_out) {
  __shared__ ScanSmem<FW> sm;
  __shared__ int64_t cnt_s[FW];
  __shared__ Pre tile_pre_s;
  __shared__ Suf tile_suf_s;
  const int tid = threadIdx.x;
  const double t = a.t;
  const double inv_t = 1.0 / t;
  const double k = a.k;
  const int64_t m = eff_len(a.len, a.len_dev);
  const int64_t ntiles = (m + TILE - 1) / TILE;
  const Tails x = load_tails(a.tails);
  const double* tb = a.tile_buf;
  const int64_t mt = a.max_tiles;

  // 1. this thread's run of tiles [t0, t0 + nr)
  const int64_t per = (ntiles + FT - 1) / FT;   // <= kFinPer (checked by the launcher)
  const int64_t t0 = static_cast<int64_t>(tid) * per;
  int nr = static_cast<int>(ntiles - t0 < per ? ntiles - t0 : per);
  nr = nr < 0 ? 0 : nr;
  double S[kFinPer], X[kFinPer], span[kFinPer];
  float fst[kFinPer], lst[kFinPer];
#pragma unroll
  for (int q = 0; q < kFinPer; ++q) {
    const bool on = q < nr;
    const int64_t at = on ? t0 + q : 0;   // always a record of the buffer
    S[q] = on ? tb[kFS * mt + at] : 0.0;
    X[q] = on ? tb[kFX * mt + at] : 0.0;
    fst[q] = on ? static_cast<float>(tb[kFFirst * mt + at]) : 0.0f;
    lst[q] = on ? static_cast<float>(tb[kFLast * mt + at]) : 0.0f;
    span[q] = on ? tb[kFSpan * mt + at] : 0.0;
  }
  // links between the run's anchors.  With span_q = e^{-(first_q - last_q)/t}
  // from the tile pass and the gaps L_q = e^{-(last_{q-1} - first_q)/t}
  // between tiles (one exponential per tile, all independent), the prefix
  // pairs move from last_{q-1} to last_q by wp = L_q span_q and the suffix
  // pairs from first_{q+1} to first_q by ws = span_q L_{q+1}; L_q itself
  // moves a prefix pair to the tile's first score
  double L[kFinPer];
#pragma unroll
  for (int q = 0; q < kFinPer; ++q)
    L[q] = (q >= 1 && q < nr) ? wexp_f64(static_cast<double>(lst[q - 1]) - fst[q], inv_t) : 0.0;
  double wp[kFinPer], ws[kFinPer];
#pragma unroll
  for (int q = 0; q < kFinPer; ++q) {
    wp[q] = (q >= 1 && q < nr) ? L[q] * span[q] : 0.0;
    ws[q] = (q + 1 < nr) ? span[q] * L[q + 1] : 0.0;
  }
  // a tile's prefix sum anchored at its last score is S (>= 1), its suffix
  // sum anchored at its first score 1 + X: no tile is empty
  double Pm = 0.0, Tm = 0.0;
#pragma unroll
  for (int q = 0; q < kFinPer; ++q)
    if (q < nr) Pm = fma(wp[q], Pm, S[q]);
#pragma unroll
  for (int q = kFinPer - 1; q >= 0; --q)
    if (q < nr) Tm = fma(ws[q], Tm, 1.0 + X[q]);
  const Pre mp = nr > 0 ? Pre{lst[nr - 1 < 0 ? 0 : nr - 1], Pm} : pre_empty();
  const Suf ms = nr > 0 ? Suf{fst[0], Tm} : suf_empty();
  Pre pre_all;
  Suf suf_all;
  Pre pre_in;
  Suf suf_in;
  block_excl_pre_suf<FW>(mp, x.pre, ms, x.suf, inv_t, sm, &pre_in, &pre_all, &suf_in, &suf_all);

  // 2. the prefix before each tile (anchored at the previous tile's last
  //    score, or the carry's anchor) and the suffix after it (anchored at
  //    the next tile's first score, or the carry's), then the node value at
  //    each tile's first score: the carry into the run is moved to the first
  //    tile's first score (pin0) and on to its last (pin_w = pin0 span_0)
  const double pin0 = (nr > 0 && pre_in.S != 0.0)
                          ? wexp_f64(static_cast<double>(pre_in.u) - fst[0], inv_t) * pre_in.S : 0.0;
  const double pin_w = pin0 * span[0];
  double sin_w = 0.0;   // suffix after the run moved to the run's last tile's first score
#pragma unroll
  for (int q = 0; q < kFinPer; ++q)
    if (q == nr - 1 && suf_in.T != 0.0)
      sin_w = wexp_f64(static_cast<double>(fst[q]) - suf_in.v, inv_t) * suf_in.T;
  Pre bef[kFinPer];
  Suf aft[kFinPer];
  double Pin[kFinPer];   // the prefix before tile q moved to its first score
  {
    Pre cur = pre_in;
    double run = 0.0;   // prefix through tile q, anchored at lst[q]
#pragma unroll
    for (int q = 0; q < kFinPer; ++q) {
      if (q < nr) {
        bef[q] = cur;
        Pin[q] = (q == 0) ? pin0 : L[q] * run;
        run = (q == 0) ? S[0] + pin_w : fma(wp[q], run, S[q]);
        cur = Pre{lst[q], run};
      }
    }
  }
  double Ein[kFinPer];   // the suffix after tile q moved to its first score
  {
    Suf cur = suf_in;
    double run = 0.0;   // suffix from tile q on, anchored at fst[q]
#pragma unroll
    for (int q = kFinPer - 1; q >= 0; --q) {
      if (q < nr) {
        aft[q] = cur;
        Ein[q] = (q == nr - 1) ? sin_w : ws[q] * run;
        run = (q == nr - 1) ? (1.0 + X[q]) + sin_w : fma(ws[q], run, 1.0 + X[q]);
        cur = Suf{fst[q], run};
      }
    }
  }
  int64_t below = 0;
#pragma unroll
  for (int q = 0; q < kFinPer; ++q) {
    if (q < nr) {
      const double P = 1.0 + Pin[q];
      const double E = X[q] + Ein[q];
      const double N = x.nR + static_cast<double>((t0 + q) * TILE) + 1.0 - 0.5 * P + 0.5 * E;
      if (N <= k) below = t0 + q + 1;   // non-decreasing: the last such tile
    }
  }
  below = block_max_i64<FW>(below, cnt_s);
  if (below > 0 && below - 1 >= t0 && below - 1 < t0 + nr) {
#pragma unroll
    for (int q = 0; q < kFinPer; ++q) {
      if (t0 + q == below - 1) {
        tile_pre_s = bef[q];
        tile_suf_s = aft[q];
      }
    }
  }
  __syncthreads();

  SolveRec rec;
  rec.ok = 1;
  rec.side = 0;
  rec.lap_aL = 0.0;
  rec.lap_aR = 0.0;
  if (x.bracketed)
    certify(x, static_cast<double>(m), static_cast<double>(a.n_total), k, t, pre_all, suf_all, rec);

  double b;
  if (m == 0 || below == 0) {
    b = root_above(x, suf_all, k, t);
  } else {
    const int64_t ct = below - 1;
    const Pre tp = tile_pre_s;
    const Suf ts = tile_suf_s;
    const int64_t base = ct * TILE;
    const int64_t nv = (m - base) < TILE ? (m - base) : TILE;
    float sv[FTI];
    int cnt = static_cast<int>(nv - static_cast<int64_t>(tid) * FTI);
    cnt = cnt < 0 ? 0 : (cnt > FTI ? FTI : cnt);
#pragma unroll
    for (int i = 0; i < FTI; ++i)
      sv[i] = (i < cnt) ? key_float(a.keys[base + static_cast<int64_t>(tid) * FTI + i]) : 0.0f;
    Pre pt;
    Suf st;
    b = block_solve<FT, FTI>(sv, cnt, x.nR + static_cast<double>(base), tp, ts, k, t, sm, &pt, &st);
  }
  if (tid == 0) {
    rec.b = b;
    *a.out = rec;
    if (b_out) *b_out = b;
  }
}

hipError_t launch_sorted_solve(const SolveArgs& a, hipStream_t s) {
  const int64_t tiles = (a.len + TILE - 1) / TILE;
  if (tiles > a.max_tiles) return hipErrorInvalidValue;
  if (tiles > 0)
    { ProfScope ps_("solve_tiles", s);
    hipLaunchKernelGGL(solve_tiles_kernel, dim3(static_cast<unsigned>(tiles)), dim3(TT), 0, s,
                       a.keys, a.len, a.len_dev, a.t, a.tile_buf, a.max_tiles); }
  if (tiles > TT && tiles <= static_cast<int64_t>(kFinPer) * FT) {
    { ProfScope ps_("solve_finalize", s);
    hipLaunchKernelGGL(solve_finalize_wide_kernel, dim3(1), dim3(FT), 0, s, a, a.b_out); }
  } else {
    { ProfScope ps_("solve_finalize", s);
    hipLaunchKernelGGL(solve_finalize_kernel, dim3(1), dim3(TT), 0, s, a, a.b_out); }
  }
  return hipGetLastError();
}

// ---------------------------------------------------- small middle set ----
template <int BLOCK, int ITEMS, bool PAIRS>
__global__ __launch_bounds__(BLOCK) void small_m_solve_kernel(const uint32_t* __restrict__ m_keys,
                                                              const int32_t* __restrict__ m_idx,
                                                              const PartTotals* __restrict__ tot,
                                                              double k, double t, int64_t n_total,
                                                              SolveRec* __restrict__ out,
                                                              int32_t* __restrict__ idx_sorted) {
  constexpr int WAVES = BLOCK / kWave;
  __shared__ uint32_t buf[sort_buf_words<BLOCK, ITEMS>()];
  __shared__ SortSmem<BLOCK> ssm;
  __shared__ ScanSmem<WAVES> csm;
  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wid = tid / kWave;
  const Tails x = load_tails(tot);
  const int m = static_cast<int>(tot->nM);

  uint32_t key[ITEMS];
  int32_t val[ITEMS];
#pragma unroll
  for (int i = 0; i < ITEMS; ++i) {
    const int pos = wid * (kWave * ITEMS) + i * kWave + lane;
    key[i] = (pos < m) ? m_keys[pos] : 0xffffffffu;
    val[i] = (pos < m) ? m_idx[pos] : -1;
  }
  if (m > 0) block_sort_u32<BLOCK, ITEMS, PAIRS>(key, val, buf, ssm);
  float s[ITEMS];
#pragma unroll
  for (int i = 0; i < ITEMS; ++i) s[i] = key_float(key[i]);
  int cnt = m - tid * ITEMS;
  cnt = cnt < 0 ? 0 : (cnt > ITEMS ? ITEMS : cnt);

  SolveRec rec;
  rec.ok = 1;
  rec.side = 0;
  double b;
  if (m == 0) {
    certify(x, 0.0, static_cast<double>(n_total), k, t, x.pre, x.suf, rec);
    b = root_above(x, x.suf, k, t);
  } else {
    Pre pt;
    Suf st;
    b = block_solve<BLOCK, ITEMS>(s, cnt, x.nR, x.pre, x.suf, k, t, csm, &pt, &st);
    certify(x, static_cast<double>(m), static_cast<double>(n_total), k, t, pt, st, rec);
  }
  if constexpr (PAIRS) {
#pragma unroll
    for (int i = 0; i < ITEMS; ++i)
      if (i < cnt) idx_sorted[tid * ITEMS + i] = val[i];
  }
  if (tid == 0) {
    rec.b = b;
    *out = rec;
  }
}

namespace {
template <int BLOCK, int ITEMS>
hipError_t small_m_items(const uint32_t* m_keys, const int32_t* m_idx, bool with_idx,
                         const PartTotals* tot, double k, double t, int64_t n_total, SolveRec* out,
                         int32_t* m_idx_sorted, hipStream_t s) {
  ProfScope ps_("small_m_solve", s);
  if (with_idx)
    hipLaunchKernelGGL((small_m_solve_kernel<BLOCK, ITEMS, true>), dim3(1), dim3(BLOCK), 0, s,
                       m_keys, m_idx, tot, k, t, n_total, out, m_idx_sorted);
  else
    hipLaunchKernelGGL((small_m_solve_kernel<BLOCK, ITEMS, false>), dim3(1), dim3(BLOCK), 0, s,
                       m_keys, m_idx, tot, k, t, n_total, out, m_idx_sorted);
  return hipGetLastError();
}
}  // namespace

hipError_t launch_small_m_solve(const uint32_t* m_keys, const int32_t* m_idx, int64_t m_len,
                                bool with_idx, const PartTotals* tot, double k, double t,
                                int64_t n_total, SolveRec* out, int32_t* m_idx_sorted,
                                hipStream_t s) {
  // the on-chip capacity follows |M| (known to the host after the partition)
  if (m_len <= 1024) return small_m_items<256, 4>(m_keys, m_idx, with_idx, tot, k, t, n_total, out, m_idx_sorted, s);
  if (m_len <= 4096) return small_m_items<256, 16>(m_keys, m_idx, with_idx, tot, k, t, n_total, out, m_idx_sorted, s);
  if (m_len <= 8192) return small_m_items<1024, 8>(m_keys, m_idx, with_idx, tot, k, t, n_total, out, m_idx_sorted, s);
  if (m_len <= 16384) return small_m_items<1024, 16>(m_keys, m_idx, with_idx, tot, k, t, n_total, out, m_idx_sorted, s);
  if (m_len <= kRowOnChipMax) return small_m_items<1024, 32>(m_keys, m_idx, with_idx, tot, k, t, n_total, out, m_idx_sorted, s);
  return hipErrorInvalidValue;
}

__global__ void write_m_idx_kernel(const int32_t* __restrict__ src, int64_t m, int64_t cap,
                                   int32_t* __restrict__ out) {
  int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
  for (; i < cap; i += stride) out[i] = (i < m) ? src[i] : -1;
}

hipError_t launch_write_m_idx(const int32_t* sorted_idx, int64_t m_len, int64_t m_capacity,
                              int32_t* out, hipStream_t s) {
  int64_t blocks = (m_capacity + 255) / 256;
  if (blocks > 2048) blocks = 2048;
  if (blocks < 1) blocks = 1;
  { ProfScope ps_("write_m_idx", s);
  hipLaunchKernelGGL(write_m_idx_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, s,
                     sorted_idx, m_len, m_capacity, out); }
  return hipGetLastError();
}

}  // namespace lapsum
