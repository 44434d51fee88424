// Comparators the paper measures Fast LapSum against, built so that its
// speed and budget claims can be reproduced on this device:
//
//   bisect   the per-query bisection baseline of §5 "Speed": one thread per
//            row runs a fixed number of bisection steps on LapSum(b) = k,
//            each re-summing all n terms, in float32 throughout;
//   dftopk   DFTopK (§2, Suppl. "Comparison with DFTopK"): a threshold fixed
//            at the midpoint c of the k-th and (k+1)-th largest scores and a
//            logistic step around it, p = 1 / (1 + e^{-(r - c)/t}), with its
//            vector-Jacobian product.
//
// Neither is on the library's own path; they are written plainly.
#include <cmath>

#include "common.hpp"
#include "kernels.hpp"

namespace lapsum {

namespace {

constexpr int kCmpThreads = 256;

// Laplace CDF of Eq. (3) in float32 for the baseline.
__device__ __forceinline__ float sigma32(float u) {
  const float e = expf(-fabsf(u));
  return u <= 0.0f ? 0.5f * e : 1.0f - 0.5f * e;
}

}  // namespace

// ---------------------------------------------------------------- bisect ---
// Thread `row`: the initial bracket from the row's extremes (lo below every
// score by t (ln(n / (2 (n - k)))^+ + 1), hi above by t (ln(n / (2k)))^+ + 1,
// so LapSum(lo) > k > LapSum(hi)), `steps` halvings keeping the root inside,
// b = the last midpoint, then p for the row.
__global__ __launch_bounds__(kWave) void bisect_kernel(const float* __restrict__ r, int64_t batch,
                                                       int64_t n, float k, float t, float lo_pad,
                                                       float hi_pad, int steps,
                                                       float* __restrict__ p,
                                                       double* __restrict__ b_out) {
  const int64_t row = static_cast<int64_t>(blockIdx.x) * kWave + threadIdx.x;
  if (row >= batch) return;
  const float* x = r + row * n;
  float mn = x[0], mx = x[0];
  for (int64_t i = 1; i < n; ++i) {
    mn = fminf(mn, x[i]);
    mx = fmaxf(mx, x[i]);
  }
  float lo = mn - lo_pad, hi = mx + hi_pad;
  const float inv_t = 1.0f / t;
  for (int s = 0; s < steps; ++s) {
    const float mid = 0.5f * (lo + hi);
    float sum = 0.0f;
    for (int64_t i = 0; i < n; ++i) sum += sigma32((x[i] - mid) * inv_t);
    if (sum > k)
      lo = mid;
    else
      hi = mid;
  }
  const float b = 0.5f * (lo + hi);
  b_out[row] = static_cast<double>(b);
  float* pr = p + row * n;
  for (int64_t i = 0; i < n; ++i) pr[i] = sigma32((x[i] - b) * inv_t);
}

hipError_t launch_bisect(const float* r, int64_t batch, int64_t n, double k, double t, int steps,
                         float* p, double* b, hipStream_t s) {
  const double lo_pad = t * (std::fmax(0.0, std::log(static_cast<double>(n) / (2.0 * (n - k)))) + 1.0);
  const double hi_pad = t * (std::fmax(0.0, std::log(static_cast<double>(n) / (2.0 * k))) + 1.0);
  const int64_t blocks = (batch + kWave - 1) / kWave;
  { ProfScope ps_("bisect", s);
  hipLaunchKernelGGL(bisect_kernel, dim3(static_cast<unsigned>(blocks)), dim3(kWave), 0, s, r,
                     batch, n, static_cast<float>(k), static_cast<float>(t),
                     static_cast<float>(lo_pad), static_cast<float>(hi_pad), steps, p, b); }
  return hipGetLastError();
}

// ---------------------------------------------------------------- dftopk ---
// The k-th and (k+1)-th largest scores from the descending sort: c in
// float64 from the two float32 values, and their original indices.
__global__ void dftopk_pick_kernel(const uint32_t* __restrict__ keys,
                                   const int32_t* __restrict__ vals, int64_t k,
                                   double* __restrict__ c, int32_t* __restrict__ pair) {
  if (threadIdx.x != 0) return;
  const float a = key_float(keys[k - 1]);
  const float b = key_float(keys[k]);
  *c = 0.5 * (static_cast<double>(a) + static_cast<double>(b));
  pair[0] = vals[k - 1];
  pair[1] = vals[k];
}

// p = 1 / (1 + e^{-(r - c)/t}): the difference in float64, the step in
// float32.
__global__ __launch_bounds__(kCmpThreads) void dftopk_emit_kernel(const float* __restrict__ r,
                                                                  int64_t n,
                                                                  const double* __restrict__ c_dev,
                                                                  double inv_t,
                                                                  float* __restrict__ p) {
  const double c = *c_dev;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kCmpThreads;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * kCmpThreads + threadIdx.x; i < n;
       i += stride) {
    const float u = static_cast<float>((static_cast<double>(r[i]) - c) * inv_t);
    p[i] = 1.0f / (1.0f + expf(-u));
  }
}

// Partial sums of g s, s = p (1 - p), one per block (float64, fixed order).
__global__ __launch_bounds__(kCmpThreads) void dftopk_reduce_kernel(const float* __restrict__ g,
                                                                    const float* __restrict__ p,
                                                                    int64_t n,
                                                                    double* __restrict__ partials) {
  __shared__ double red[kCmpThreads / kWave];
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kCmpThreads;
  double acc = 0.0;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * kCmpThreads + threadIdx.x; i < n;
       i += stride) {
    const float pv = p[i];
    acc += static_cast<double>(g[i]) * static_cast<double>(pv * (1.0f - pv));
  }
  acc = wave_sum(acc);
  if (lane_id() == 0) red[threadIdx.x / kWave] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    double s = 0.0;
#pragma unroll
    for (int w = 0; w < kCmpThreads / kWave; ++w) s += red[w];
    partials[blockIdx.x] = s;
  }
}

// grad_i = g_i s_i / t, minus (1/(2t)) sum_j g_j s_j at the two boundary
// scores (the threshold moves with them by 1/2 each).  Every block sums the
// partials itself, in the same order.
__global__ __launch_bounds__(kCmpThreads) void dftopk_grad_kernel(
    const float* __restrict__ g, const float* __restrict__ p, int64_t n,
    const double* __restrict__ partials, int nparts, const int32_t* __restrict__ pair, double inv_t,
    float* __restrict__ grad) {
  __shared__ double red[kCmpThreads / kWave];
  double acc = 0.0;
  for (int j = threadIdx.x; j < nparts; j += kCmpThreads) acc += partials[j];
  acc = wave_sum(acc);
  if (lane_id() == 0) red[threadIdx.x / kWave] = acc;
  __syncthreads();
  double tot = 0.0;
#pragma unroll
  for (int w = 0; w < kCmpThreads / kWave; ++w) tot += red[w];
  const float corr = static_cast<float>(0.5 * tot * inv_t);
  const int32_t i0 = pair[0], i1 = pair[1];
  const float it = static_cast<float>(inv_t);
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kCmpThreads;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * kCmpThreads + threadIdx.x; i < n;
       i += stride) {
    const float pv = p[i];
    float v = g[i] * (pv * (1.0f - pv)) * it;
    if (i == i0 || i == i1) v -= corr;
    grad[i] = v;
  }
}

int dftopk_blocks(int64_t n) {
  const int64_t b = (n + 4 * kCmpThreads - 1) / (4 * kCmpThreads);
  return static_cast<int>(b < 1 ? 1 : (b > 1024 ? 1024 : b));
}

hipError_t launch_dftopk_pick(const uint32_t* keys, const int32_t* vals, int64_t k, double* c,
                              int32_t* pair, hipStream_t s) {
  { ProfScope ps_("dftopk_pick", s);
  hipLaunchKernelGGL(dftopk_pick_kernel, dim3(1), dim3(kWave), 0, s, keys, vals, k, c, pair); }
  return hipGetLastError();
}

hipError_t launch_dftopk_emit(const float* r, int64_t n, const double* c, double t, float* p,
                              hipStream_t s) {
  { ProfScope ps_("dftopk_emit", s);
  hipLaunchKernelGGL(dftopk_emit_kernel, dim3(dftopk_blocks(n)), dim3(kCmpThreads), 0, s, r, n,
                     c, 1.0 / t, p); }
  return hipGetLastError();
}

hipError_t launch_dftopk_backward(const float* g, const float* p, int64_t n, const int32_t* pair,
                                  double t, double* partials, float* grad, hipStream_t s) {
  const int nb = dftopk_blocks(n);
  { ProfScope ps_("dftopk_reduce", s);
  hipLaunchKernelGGL(dftopk_reduce_kernel, dim3(nb), dim3(kCmpThreads), 0, s, g, p, n, partials); }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  { ProfScope ps_("dftopk_grad", s);
  hipLaunchKernelGGL(dftopk_grad_kernel, dim3(nb), dim3(kCmpThreads), 0, s, g, p, n, partials, nb,
                     pair, 1.0 / t, grad); }
  return hipGetLastError();
}

}  // namespace lapsum
