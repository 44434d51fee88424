// Streaming passes over one long row: the Laplace-CDF emit (the fused CDF
// evaluation of Suppl. D) and the two passes of the Eq. (5) backward.
//
// All three are HBM-bound.  Algorithmic bytes per score:
//   emit        read r, write p                          8 B
//   vjp reduce  read p, read g where f != 0              4 B + 4 B x (active share)
//   vjp emit    read p, read g where f != 0, write grad  8 B + 4 B x (active share)
// f = min(p, 1 - p) is exactly zero for scores whose p rounded to 0 or 1 in
// float32; their g is never read.
#include "common.hpp"
#include "kernels.hpp"

namespace lapsum {

namespace {
constexpr int kStreamThreads = 256;
constexpr int kStreamVec = 4;   // float4 per thread per block
constexpr int64_t kStreamTile = static_cast<int64_t>(kStreamThreads) * kStreamVec * 4;   // scores
}  // namespace

__global__ void fill_u32_kernel(uint32_t* __restrict__ dst, int64_t count, uint32_t value) {
  int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
  for (; i < count; i += stride) dst[i] = value;
}

hipError_t launch_fill_u32(uint32_t* dst, int64_t count, uint32_t value, hipStream_t s) {
  if (count <= 0) return hipSuccess;
  int64_t blocks = (count + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  { ProfScope ps_("fill_u32", s);
  hipLaunchKernelGGL(fill_u32_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, s, dst,
                     count, value); }
  return hipGetLastError();
}

// ------------------------------------------------------------ top-k mask ---
// mask[row][perm[row][j]] = (j < k ? 1 : 0): one thread per position j of the
// descending order; an index outside [0, n) is skipped.
__global__ __launch_bounds__(256) void topk_mask_kernel(const int32_t* __restrict__ perm,
                                                        int64_t n, int64_t k, int64_t total,
                                                        float* __restrict__ mask) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * 256;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; i < total; i += stride) {
    const int64_t row = i / n;
    const int64_t j = i - row * n;
    const int32_t at = perm[i];
    if (at >= 0 && at < n) mask[row * n + at] = j < k ? 1.0f : 0.0f;
  }
}

hipError_t launch_topk_mask(const int32_t* perm, int64_t batch, int64_t n, int64_t k, float* mask,
                            hipStream_t s) {
  const int64_t total = batch * n;
  int64_t blocks = (total + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  { ProfScope ps_("topk_mask", s);
  hipLaunchKernelGGL(topk_mask_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, s, perm,
                     n, k, total, mask); }
  return hipGetLastError();
}

// ------------------------------------------------------------------ emit ---
__global__ __launch_bounds__(kStreamThreads) void emit_kernel(const float* __restrict__ r,
                                                              int64_t n,
                                                              const double* __restrict__ b_dev,
                                                              double inv_t,
                                                              float* __restrict__ p) {
  const double b = *b_dev;
  const int64_t base = static_cast<int64_t>(blockIdx.x) * kStreamTile;
  const int tid = threadIdx.x;
  const bool vec = ((reinterpret_cast<uintptr_t>(r) | reinterpret_cast<uintptr_t>(p)) & 15) == 0;
  if (vec && base + kStreamTile <= n) {
    const float4* r4 = reinterpret_cast<const float4*>(r + base);
    float4* p4 = reinterpret_cast<float4*>(p + base);
    float4 v[kStreamVec];
#pragma unroll
    for (int j = 0; j < kStreamVec; ++j) v[j] = r4[j * kStreamThreads + tid];
#pragma unroll
    for (int j = 0; j < kStreamVec; ++j) {
      float4 o;
      o.x = laplace_p(v[j].x, b, inv_t);
      o.y = laplace_p(v[j].y, b, inv_t);
      o.z = laplace_p(v[j].z, b, inv_t);
      o.w = laplace_p(v[j].w, b, inv_t);
      p4[j * kStreamThreads + tid] = o;
    }
  } else {
    for (int64_t i = base + tid; i < n && i < base + kStreamTile; i += kStreamThreads)
      p[i] = laplace_p(r[i], b, inv_t);
  }
}

hipError_t launch_emit(const float* r, int64_t n, const double* b_dev, double t, float* p,
                       hipStream_t s) {
  const int64_t blocks = (n + kStreamTile - 1) / kStreamTile;
  { ProfScope ps_("emit", s);
  hipLaunchKernelGGL(emit_kernel, dim3(static_cast<unsigned>(blocks)), dim3(kStreamThreads), 0, s,
                     r, n, b_dev, 1.0 / t, p); }
  return hipGetLastError();
}

// ------------------------------------------------------------ vjp reduce ---
// Wave tiles of 256 float4 (1024 scores); wave w of the grid's G waves takes
// tiles w, w + G, w + 2G, ..., so that the waves of the chip read
// neighbouring tiles at any time, and the grid is at most kVjpBlocks
// workgroups (about one round of resident ones) so that each wave streams
// many tiles.  (Each workgroup streaming its own contiguous range read the
// 400 MB of p at n = 1e8 at 3.6 TB/s.)
// Rows up to 2^24 scores take one tile per wave (all of a wave's loads in
// flight at once, up to 4096 workgroups): there the row sits in the
// last-level cache and a short pipeline only adds steps.
constexpr int kVjpBlocks = 1280;
constexpr int kVjpOneTileBlocks = 4096;

int vjp_reduce_blocks(int64_t n) {
  const int64_t tiles = n / 1024;   // whole wave tiles
  const int64_t b = (tiles + 3) / 4;
  const int64_t cap = b <= kVjpOneTileBlocks ? kVjpOneTileBlocks : kVjpBlocks;
  return static_cast<int>(b < 1 ? 1 : (b > cap ? cap : b));
}

// Sums of f = min(p, 1-p) and f g over the row, g read only for float4s with
// some f != 0: float32 within a float4, float64 across, then a fixed-order
// block reduction (DPP within a wave, waves in order) to partials[block].
// With PARAMS also sum s u and sum s g u, u recovered from p.
//
// Software pipeline per wave, one tile per step: step s issues the p loads
// of tile s + 2 into the buffer tile s - 1 freed, then the g loads tile s
// needs, then adds tile s; so the next two p tiles are in flight while a
// tile's g is read, and no loaded register is copied (three p buffers rotate
// through an unrolled period of three).  Loads past a wave's last tile read
// one line of its first tile instead; only lanes that need g load it.  The
// float4s past the whole tiles and the scalar tail go to the last workgroup.
template <bool PARAMS>
__global__ __launch_bounds__(kStreamThreads, 4) void vjp_reduce_kernel(const float* __restrict__ g,
                                                                    const float* __restrict__ p,
                                                                    int64_t n,
                                                                    double* __restrict__ partials) {
  constexpr int NS = PARAMS ? 4 : 2;
  constexpr int W = kStreamThreads / kWave;
  __shared__ double red[NS][W];
  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wid = tid / kWave;
  const bool vec = ((reinterpret_cast<uintptr_t>(g) | reinterpret_cast<uintptr_t>(p)) & 15) == 0;
  const float4* p4 = reinterpret_cast<const float4*>(p);
  const float4* g4 = reinterpret_cast<const float4*>(g);
  double F = 0.0, G = 0.0, Us = 0.0, H = 0.0;
  // one float4 of p with its g (g meaningful only where some f != 0).  No
  // contraction into fused multiply-adds, so that both instances (with and
  // without the parameter sums) round the same sums the same way.
  auto add4 = [&](const float4& pv, const float4& gv) {
#pragma clang fp contract(off)
    const float f[4] = {fminf(pv.x, 1.0f - pv.x), fminf(pv.y, 1.0f - pv.y),
                        fminf(pv.z, 1.0f - pv.z), fminf(pv.w, 1.0f - pv.w)};
    const float fs = (f[0] + f[1]) + (f[2] + f[3]);
    if (fs != 0.0f) {
      F += static_cast<double>(fs);
      G += static_cast<double>((f[0] * gv.x + f[1] * gv.y) + (f[2] * gv.z + f[3] * gv.w));
      if constexpr (PARAMS) {
        const float pw[4] = {pv.x, pv.y, pv.z, pv.w};
        const float gw[4] = {gv.x, gv.y, gv.z, gv.w};
        float a = 0.0f, c = 0.0f;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const float fu = f[q] != 0.0f ? f[q] * laplace_u_from_p(pw[q], f[q]) : 0.0f;
          a += fu;
          c += fu * gw[q];
        }
        Us += static_cast<double>(a);
        H += static_cast<double>(c);
      }
    }
  };
  auto add1 = [&](float pp, float gg) {
#pragma clang fp contract(off)
    const float f1 = fminf(pp, 1.0f - pp);
    if (f1 != 0.0f) {
      const double gj = static_cast<double>(gg);
      F += static_cast<double>(f1);
      G += static_cast<double>(f1) * gj;
      if constexpr (PARAMS) {
        const double fu = static_cast<double>(f1) * static_cast<double>(laplace_u_from_p(pp, f1));
        Us += fu;
        H += fu * gj;
      }
    }
  };

  if (vec) {
    const int64_t n4 = n / 4;
    const int64_t nt = n / 1024;   // whole wave tiles
    const int64_t GW = static_cast<int64_t>(gridDim.x) * W;
    const int64_t w0 = static_cast<int64_t>(blockIdx.x) * W + wid;
    const int cnt = w0 < nt ? static_cast<int>((nt - w0 + GW - 1) / GW) : 0;
    if (cnt > 0) {
      const float4* pd = p4 + w0 * 256;   // the line loads past the end read
      auto base_of = [&](int j) { return (w0 + static_cast<int64_t>(j) * GW) * 256 + lane; };
      auto load_p = [&](float4 (&q)[4], int j) {
        const bool real = j < cnt;
        const int64_t b = base_of(j);
#pragma unroll
        for (int u = 0; u < 4; ++u) q[u] = load_stream4(reinterpret_cast<const float*>(real ? p4 + b + 64 * u : pd));
      };
      // tile s: its p loaded, the p of tiles s + 1 and s + 2 issued, then
      // its g (issued after them, so waiting for g waits for tile s + 1's p
      // as well, which the next step needs anyway; tile s + 2 stays in
      // flight), then the sums
      auto step = [&](const float4 (&pc)[4], float4 (&pn2)[4], int st) {
        load_p(pn2, st + 2);
        const int64_t b = base_of(st);
        float4 gq[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const bool need = (fminf(pc[u].x, 1.0f - pc[u].x) + fminf(pc[u].y, 1.0f - pc[u].y)) +
                                (fminf(pc[u].z, 1.0f - pc[u].z) + fminf(pc[u].w, 1.0f - pc[u].w)) != 0.0f;
          // only lanes that need g load it (a lane that needs none issues no
          // request); g is used within this step, so no register is copied
          gq[u] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
          if (need) gq[u] = g4[b + 64 * u];
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) add4(pc[u], gq[u]);
      };
      float4 P0[4], P1[4], P2[4];   // tile s sits in P[s % 3]
      load_p(P0, 0);
      load_p(P1, 1);
      for (int s0 = 0;; s0 += 3) {
        step(P0, P2, s0);
        if (s0 + 1 >= cnt) break;
        step(P1, P0, s0 + 1);
        if (s0 + 2 >= cnt) break;
        step(P2, P1, s0 + 2);
        if (s0 + 3 >= cnt) break;
      }
    }
    if (blockIdx.x == gridDim.x - 1) {
      // the float4s past the whole tiles, then the scalars past them
      for (int64_t i = nt * 256 + tid; i < n4; i += kStreamThreads) {
        const float4 pv = p4[i];
        add4(pv, g4[i]);
      }
      for (int64_t j = n4 * 4 + tid; j < n; j += kStreamThreads) add1(p[j], g[j]);
    }
  } else {
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kStreamThreads;
    for (int64_t j = static_cast<int64_t>(blockIdx.x) * kStreamThreads + tid; j < n; j += stride)
      add1(p[j], g[j]);
  }
  F = wave_sum(F);
  G = wave_sum(G);
  if constexpr (PARAMS) {
    Us = wave_sum(Us);
    H = wave_sum(H);
  }
  if (lane == 0) {
    red[0][wid] = F;
    red[1][wid] = G;
    if constexpr (PARAMS) {
      red[2][wid] = Us;
      red[3][wid] = H;
    }
  }
  __syncthreads();
  if (tid < NS) {
    double acc = 0.0;
#pragma unroll
    for (int w = 0; w < W; ++w) acc += red[tid][w];
    partials[NS * blockIdx.x + tid] = acc;
  }
}

// The partials summed in a fixed order by one block of T threads (thread
// tid takes partials tid, tid + T, ..., then the waves in order); thread 0
// returns the totals.
template <int NS, int T>
__device__ void vjp_totals(const double* __restrict__ partials, int nparts,
                           double (&red)[NS][T / kWave], double (&tot)[NS]) {
  const int tid = threadIdx.x;
  double acc[NS];
#pragma unroll
  for (int q = 0; q < NS; ++q) acc[q] = 0.0;
  for (int j = tid; j < nparts; j += T) {
#pragma unroll
    for (int q = 0; q < NS; ++q) acc[q] += partials[NS * j + q];
  }
#pragma unroll
  for (int q = 0; q < NS; ++q) acc[q] = wave_sum(acc[q]);
  const int wid = tid / kWave;
  if (lane_id() == 0) {
#pragma unroll
    for (int q = 0; q < NS; ++q) red[q][wid] = acc[q];
  }
  __syncthreads();
#pragma unroll
  for (int q = 0; q < NS; ++q) {
    tot[q] = 0.0;
#pragma unroll
    for (int w = 0; w < T / kWave; ++w) tot[q] += red[q][w];
  }
}

// From the totals: coef = <g, q> = sum f g / sum f and scale = 1/t (both 0
// when sum f == 0); with PARAMS also dL/dk = <g, q> and
// dL/dalpha = (H - (U/F) G)/t (either output may be null).
template <bool PARAMS, int NS>
__device__ void vjp_coefs(const double (&tot)[NS], double inv_t, double* coef, double* grad_k,
                          double* grad_alpha) {
  const double f = tot[0], gg = tot[1];
  coef[0] = (f > 0.0) ? gg / f : 0.0;
  coef[1] = (f > 0.0) ? inv_t : 0.0;
  if constexpr (PARAMS) {
    if (grad_k) *grad_k = coef[0];
    if (grad_alpha) *grad_alpha = (f > 0.0) ? (tot[3] - (tot[2] / f) * gg) * inv_t : 0.0;
  }
}

// One block: the coefficients of the emit from the partials of a long row.
template <bool PARAMS>
__global__ __launch_bounds__(1024) void vjp_finalize_kernel(const double* __restrict__ partials,
                                                            int nparts, double inv_t,
                                                            double* __restrict__ coef,
                                                            double* __restrict__ grad_k,
                                                            double* __restrict__ grad_alpha) {
  constexpr int T = 1024;
  constexpr int NS = PARAMS ? 4 : 2;
  __shared__ double red[NS][T / kWave];
  double tot[NS];
  vjp_totals<NS, T>(partials, nparts, red, tot);
  if (threadIdx.x == 0) vjp_coefs<PARAMS, NS>(tot, inv_t, coef, grad_k, grad_alpha);
}

// Rows whose reduce leaves at most this many partials skip the finalize:
// every emit block sums them itself (at most 4 KB each).
constexpr int kFoldParts = 256;

hipError_t launch_vjp_reduce(const float* g, const float* p, int64_t n, double* partials,
                             int nblocks, double t, double* coef, double* grad_k,
                             double* grad_alpha, hipStream_t s) {
  const bool params = grad_k || grad_alpha;
  { ProfScope ps_("vjp_reduce", s);
  if (params)
    hipLaunchKernelGGL(vjp_reduce_kernel<true>, dim3(nblocks), dim3(kStreamThreads), 0, s, g, p,
                       n, partials);
  else
    hipLaunchKernelGGL(vjp_reduce_kernel<false>, dim3(nblocks), dim3(kStreamThreads), 0, s, g, p,
                       n, partials); }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (nblocks <= kFoldParts) return hipSuccess;   // the emit combines the partials
  { ProfScope ps_("vjp_finalize", s);
  if (params)
    hipLaunchKernelGGL(vjp_finalize_kernel<true>, dim3(1), dim3(1024), 0, s, partials, nblocks,
                       1.0 / t, coef, grad_k, grad_alpha);
  else
    hipLaunchKernelGGL(vjp_finalize_kernel<false>, dim3(1), dim3(1024), 0, s, partials, nblocks,
                       1.0 / t, coef, grad_k, grad_alpha); }
  return hipGetLastError();
}

// -------------------------------------------------------------- vjp emit ---
// grad_r = (f/t)(g - <g,q>), q = f / sum f; zero where f == 0.  NT: grad_r
// is stored non-temporally (rows of kNtStoreMin scores and more): with
// ordinary stores the dirty lines of such a row are written back while the
// next pass reads, while a shorter row's stay in the last-level cache.
constexpr int64_t kNtStoreMin = int64_t(1) << 24;

// FOLD: coef comes from the reduce partials, summed by every block in the
// same order (block 0 also stores the parameter gradients); otherwise from
// the finalize.
template <bool NT, bool FOLD, bool PARAMS>
__global__ __launch_bounds__(kStreamThreads) void vjp_emit_kernel(const float* __restrict__ g,
                                                                  const float* __restrict__ p,
                                                                  int64_t n,
                                                                  const double* __restrict__ coef2,
                                                                  const double* __restrict__ partials,
                                                                  int nparts, double inv_t,
                                                                  double* __restrict__ grad_k,
                                                                  double* __restrict__ grad_alpha,
                                                                  float* __restrict__ grad) {
  float coef, scale;
  if constexpr (FOLD) {
    constexpr int NS = PARAMS ? 4 : 2;
    __shared__ double red[NS][kStreamThreads / kWave];
    double tot[NS];
    vjp_totals<NS, kStreamThreads>(partials, nparts, red, tot);
    double c[2];
    vjp_coefs<PARAMS, NS>(tot, inv_t, c, blockIdx.x == 0 && threadIdx.x == 0 ? grad_k : nullptr,
                          blockIdx.x == 0 && threadIdx.x == 0 ? grad_alpha : nullptr);
    coef = static_cast<float>(c[0]);
    scale = static_cast<float>(c[1]);
  } else {
    coef = static_cast<float>(coef2[0]);
    scale = static_cast<float>(coef2[1]);
  }
  const int tid = threadIdx.x;
  const int64_t base = static_cast<int64_t>(blockIdx.x) * kStreamTile;
  const bool vec =
      ((reinterpret_cast<uintptr_t>(g) | reinterpret_cast<uintptr_t>(p) | reinterpret_cast<uintptr_t>(grad)) & 15) == 0;
  if (vec && base + kStreamTile <= n) {
    const float4* p4 = reinterpret_cast<const float4*>(p + base);
    const float4* g4 = reinterpret_cast<const float4*>(g + base);
    float4* o4 = reinterpret_cast<float4*>(grad + base);
    float4 pv[kStreamVec];
#pragma unroll
    for (int j = 0; j < kStreamVec; ++j) pv[j] = p4[j * kStreamThreads + tid];
#pragma unroll
    for (int j = 0; j < kStreamVec; ++j) {
      const float fx = fminf(pv[j].x, 1.0f - pv[j].x), fy = fminf(pv[j].y, 1.0f - pv[j].y);
      const float fz = fminf(pv[j].z, 1.0f - pv[j].z), fw = fminf(pv[j].w, 1.0f - pv[j].w);
      float4 o = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
      if ((fx + fy) + (fz + fw) != 0.0f) {
        const float4 gv = g4[j * kStreamThreads + tid];
        o.x = fx * scale * (gv.x - coef);
        o.y = fy * scale * (gv.y - coef);
        o.z = fz * scale * (gv.z - coef);
        o.w = fw * scale * (gv.w - coef);
      }
      if constexpr (NT)
        store_stream4(reinterpret_cast<float*>(o4 + j * kStreamThreads + tid), o);
      else
        o4[j * kStreamThreads + tid] = o;
    }
  } else {
    for (int64_t i = base + tid; i < n && i < base + kStreamTile; i += kStreamThreads) {
      const float pp = p[i];
      const float f = fminf(pp, 1.0f - pp);
      grad[i] = (f != 0.0f) ? f * scale * (g[i] - coef) : 0.0f;
    }
  }
}

hipError_t launch_vjp_emit(const float* g, const float* p, int64_t n, const double* coef,
                           const double* partials, int nparts, double t, double* grad_k,
                           double* grad_alpha, float* grad, hipStream_t s) {
  const int64_t blocks = (n + kStreamTile - 1) / kStreamTile;
  const dim3 grid(static_cast<unsigned>(blocks)), block(kStreamThreads);
  const double inv_t = 1.0 / t;
  const bool params = grad_k || grad_alpha;
  { ProfScope ps_("vjp_emit", s);
  if (nparts > kFoldParts) {
    if (n >= kNtStoreMin)
      hipLaunchKernelGGL((vjp_emit_kernel<true, false, false>), grid, block, 0, s, g, p, n, coef,
                         partials, nparts, inv_t, grad_k, grad_alpha, grad);
    else
      hipLaunchKernelGGL((vjp_emit_kernel<false, false, false>), grid, block, 0, s, g, p, n, coef,
                         partials, nparts, inv_t, grad_k, grad_alpha, grad);
  } else if (params) {
    hipLaunchKernelGGL((vjp_emit_kernel<false, true, true>), grid, block, 0, s, g, p, n, coef,
                       partials, nparts, inv_t, grad_k, grad_alpha, grad);
  } else {
    hipLaunchKernelGGL((vjp_emit_kernel<false, true, false>), grid, block, 0, s, g, p, n, coef,
                       partials, nparts, inv_t, grad_k, grad_alpha, grad);
  } }
  return hipGetLastError();
}

}  // namespace lapsum
