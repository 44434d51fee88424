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
int vjp_reduce_blocks(int64_t n) {
  const int64_t b = (n + kStreamTile - 1) / kStreamTile;
  return static_cast<int>(b < 1 ? 1 : (b > 4096 ? 4096 : b));
}

// Block b sums f = min(p, 1-p) and f g over a contiguous range of float4s,
// four per lane in flight; g is read only for float4s with some f != 0.
// float32 within a float4, float64 across, then a fixed-order block
// reduction (DPP within a wave, waves in order).  With PARAMS also sum s u
// and sum s g u, u recovered from p.
template <bool PARAMS>
__global__ __launch_bounds__(kStreamThreads) void vjp_reduce_kernel(const float* __restrict__ g,
                                                                    const float* __restrict__ p,
                                                                    int64_t n,
                                                                    double* __restrict__ partials) {
  constexpr int NS = PARAMS ? 4 : 2;
  __shared__ double red[NS][kStreamThreads / kWave];
  const int tid = threadIdx.x;
  const bool vec = ((reinterpret_cast<uintptr_t>(g) | reinterpret_cast<uintptr_t>(p)) & 15) == 0;
  const int64_t n4 = vec ? n / 4 : 0;
  const int64_t per = (n4 + gridDim.x - 1) / gridDim.x;
  const int64_t lo = static_cast<int64_t>(blockIdx.x) * per;
  const int64_t hi = (lo + per < n4) ? lo + per : n4;
  const float4* p4 = reinterpret_cast<const float4*>(p);
  const float4* g4 = reinterpret_cast<const float4*>(g);
  double F = 0.0, G = 0.0, Us = 0.0, H = 0.0;
  // sum s u and sum s g u of four scores (float32; s == 0 terms skipped)
  auto su4 = [&](const float4& pv, const float (&f)[4], const float4& gv) {
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
  };
  constexpr int U = 4;   // float4 of p per lane per batch, two batches in flight
  int64_t i = lo + tid;
  auto batch = [&](const float4 (&pv)[U], int64_t at) {
    float f[U][4];
    bool need[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      f[u][0] = fminf(pv[u].x, 1.0f - pv[u].x);
      f[u][1] = fminf(pv[u].y, 1.0f - pv[u].y);
      f[u][2] = fminf(pv[u].z, 1.0f - pv[u].z);
      f[u][3] = fminf(pv[u].w, 1.0f - pv[u].w);
      need[u] = ((f[u][0] + f[u][1]) + (f[u][2] + f[u][3])) != 0.0f;
    }
    float4 gv[U];
#pragma unroll
    for (int u = 0; u < U; ++u)
      gv[u] = need[u] ? g4[at + u * kStreamThreads] : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (need[u]) {
        F += static_cast<double>((f[u][0] + f[u][1]) + (f[u][2] + f[u][3]));
        G += static_cast<double>((f[u][0] * gv[u].x + f[u][1] * gv[u].y) +
                                 (f[u][2] * gv[u].z + f[u][3] * gv[u].w));
        if constexpr (PARAMS) su4(pv[u], f[u], gv[u]);
      }
    }
  };
  if (i + (U - 1) * kStreamThreads < hi) {
    float4 pv[U];
#pragma unroll
    for (int u = 0; u < U; ++u) pv[u] = p4[i + u * kStreamThreads];
    while (true) {
      const int64_t cur = i;
      i += U * kStreamThreads;
      const bool more = i + (U - 1) * kStreamThreads < hi;
      float4 pn[U];
      if (more) {
#pragma unroll
        for (int u = 0; u < U; ++u) pn[u] = p4[i + u * kStreamThreads];
      }
      batch(pv, cur);
      if (!more) break;
#pragma unroll
      for (int u = 0; u < U; ++u) pv[u] = pn[u];
    }
  }
  for (; i < hi; i += kStreamThreads) {
    const float4 pv = p4[i];
    const float f[4] = {fminf(pv.x, 1.0f - pv.x), fminf(pv.y, 1.0f - pv.y),
                        fminf(pv.z, 1.0f - pv.z), fminf(pv.w, 1.0f - pv.w)};
    const float fs = (f[0] + f[1]) + (f[2] + f[3]);
    if (fs != 0.0f) {
      const float4 gq = g4[i];
      F += static_cast<double>(fs);
      G += static_cast<double>((f[0] * gq.x + f[1] * gq.y) + (f[2] * gq.z + f[3] * gq.w));
      if constexpr (PARAMS) su4(pv, f, gq);
    }
  }
  if (blockIdx.x == gridDim.x - 1) {   // scalar tail (all of it when unaligned)
    for (int64_t j = n4 * 4 + tid; j < n; j += kStreamThreads) {
      const float pp = p[j];
      const float f1 = fminf(pp, 1.0f - pp);
      if (f1 != 0.0f) {
        const double gj = static_cast<double>(g[j]);
        F += static_cast<double>(f1);
        G += static_cast<double>(f1) * gj;
        if constexpr (PARAMS) {
          const double fu = static_cast<double>(f1) * static_cast<double>(laplace_u_from_p(pp, f1));
          Us += fu;
          H += fu * gj;
        }
      }
    }
  }
  F = wave_sum(F);
  G = wave_sum(G);
  if constexpr (PARAMS) {
    Us = wave_sum(Us);
    H = wave_sum(H);
  }
  const int wid = tid / kWave;
  if (lane_id() == 0) {
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
    for (int w = 0; w < kStreamThreads / kWave; ++w) acc += red[tid][w];
    partials[NS * blockIdx.x + tid] = acc;
  }
}

// One block: sum the partials in a fixed order and store
// coef = <g, q> = sum f g / sum f and scale = 1/t (both 0 when sum f == 0);
// with PARAMS also dL/dk = <g, q> and dL/dalpha = (H - (U/F) G)/t.
template <bool PARAMS>
__global__ __launch_bounds__(1024) void vjp_finalize_kernel(const double* __restrict__ partials,
                                                            int nparts, double inv_t,
                                                            double* __restrict__ coef,
                                                            double* __restrict__ grad_k,
                                                            double* __restrict__ grad_alpha) {
  constexpr int T = 1024;
  constexpr int NS = PARAMS ? 4 : 2;
  __shared__ double red[NS][T / kWave];
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
  if (tid == 0) {
    double tot[NS];
#pragma unroll
    for (int q = 0; q < NS; ++q) {
      tot[q] = 0.0;
#pragma unroll
      for (int w = 0; w < T / kWave; ++w) tot[q] += red[q][w];
    }
    const double f = tot[0], gg = tot[1];
    coef[0] = (f > 0.0) ? gg / f : 0.0;
    coef[1] = (f > 0.0) ? inv_t : 0.0;
    if constexpr (PARAMS) {
      if (grad_k) *grad_k = coef[0];
      if (grad_alpha) *grad_alpha = (f > 0.0) ? (tot[3] - (tot[2] / f) * gg) * inv_t : 0.0;
    }
  }
}

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
// grad_r = (f/t)(g - <g,q>), q = f / sum f; zero where f == 0
__global__ __launch_bounds__(kStreamThreads) void vjp_emit_kernel(const float* __restrict__ g,
                                                                  const float* __restrict__ p,
                                                                  int64_t n,
                                                                  const double* __restrict__ coef2,
                                                                  float* __restrict__ grad) {
  const float coef = static_cast<float>(coef2[0]);
  const float scale = static_cast<float>(coef2[1]);
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
                           float* grad, hipStream_t s) {
  const int64_t blocks = (n + kStreamTile - 1) / kStreamTile;
  { ProfScope ps_("vjp_emit", s);
  hipLaunchKernelGGL(vjp_emit_kernel, dim3(static_cast<unsigned>(blocks)), dim3(kStreamThreads), 0,
                     s, g, p, n, coef, grad); }
  return hipGetLastError();
}

}  // namespace lapsum
