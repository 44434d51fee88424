// One workgroup per row, the whole row on chip (n <= 32768): the full-sort
// forward of §1/§3/Suppl. A and the VJP of Eq. (5).
//
// Forward: the row's keys are sorted in LDS (block_sort.hpp), the sorted run
// is solved by block_solve (scan, lookup, closed-form root, common.hpp), and
// p is written in the original order.  HBM traffic: read r, write p (the
// second read of r for the emit hits L2).  Backward: p and g stay in
// registers between the reduction and the emit, so read g, p and write
// grad_r once each.
#include "block_sort.hpp"
#include "kernels.hpp"

namespace lapsum {

template <int BLOCK, int ITEMS, bool PAIRS>
__global__ __launch_bounds__(BLOCK) void row_forward_kernel(const float* __restrict__ scores,
                                                            int n, double k, double t,
                                                            float* __restrict__ p,
                                                            double* __restrict__ b_out,
                                                            int32_t* __restrict__ perm,
                                                            int gated) {
  constexpr int WAVES = BLOCK / kWave;
  __shared__ uint32_t buf[sort_buf_words<BLOCK, ITEMS>()];
  __shared__ SortSmem<BLOCK> ssm;
  __shared__ ScanSmem<WAVES> csm;

  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wid = tid / kWave;
  const int64_t row = blockIdx.x;
  const float* r = scores + row * n;
  // gated: only the rows the bucketed forward left unsolved (b = NaN)
  if (gated) {
    const double b0 = b_out[row];
    if (b0 == b0) return;
  }

  uint32_t key[ITEMS];
  int32_t val[ITEMS];
#pragma unroll
  for (int i = 0; i < ITEMS; ++i) {
    const int pos = wid * (kWave * ITEMS) + i * kWave + lane;
    if (pos < n) {
      key[i] = desc_key(r[pos]);
      val[i] = pos;
    } else {
      key[i] = 0xffffffffu;   // after every finite score
      val[i] = -1;
    }
  }
  block_sort_u32<BLOCK, ITEMS, PAIRS>(key, val, buf, ssm);

  float s[ITEMS];
#pragma unroll
  for (int i = 0; i < ITEMS; ++i) s[i] = key_float(key[i]);
  int cnt = n - tid * ITEMS;
  cnt = cnt < 0 ? 0 : (cnt > ITEMS ? ITEMS : cnt);
  Pre pt;
  Suf st;
  const double b = block_solve<BLOCK, ITEMS>(s, cnt, 0.0, pre_empty(), suf_empty(), k, t, csm, &pt, &st);
  if (tid == 0) b_out[row] = b;

  if constexpr (PAIRS) {
    int32_t* pr = perm + row * n;
#pragma unroll
    for (int i = 0; i < ITEMS; ++i)
      if (i < cnt) pr[tid * ITEMS + i] = val[i];
  }

  const double inv_t = 1.0 / t;
  float* pr = p + row * n;
  if ((n & 3) == 0) {
    const float4* r4 = reinterpret_cast<const float4*>(r);
    float4* p4 = reinterpret_cast<float4*>(pr);
    for (int j = tid; j < n / 4; j += BLOCK) {
      const float4 v = r4[j];
      float4 o;
      o.x = laplace_p(v.x, b, inv_t);
      o.y = laplace_p(v.y, b, inv_t);
      o.z = laplace_p(v.z, b, inv_t);
      o.w = laplace_p(v.w, b, inv_t);
      p4[j] = o;
    }
  } else {
    for (int j = tid; j < n; j += BLOCK) pr[j] = laplace_p(r[j], b, inv_t);
  }
}

// Eq. (5) for one row; with PARAMS also the budget and temperature gradients
// dL/dk = G/F and dL/dalpha = (H - (U/F) G)/t, from F = sum s, G = sum s g,
// U = sum s u, H = sum s g u over s = min(p, 1 - p), u = (r - b)/t (implicit
// differentiation of Eq. (1)); both 0 when F == 0.  p and g stay in
// registers between the reduction and the write, so each is read once
// (float4 accesses when n is a multiple of 4: item i of thread tid is
// element 4 (tid + BLOCK (i/4)) + i%4, else tid + BLOCK i).
template <int BLOCK, int ITEMS, bool PARAMS, bool VEC>
__global__ __launch_bounds__(BLOCK) void row_backward_kernel(const float* __restrict__ g,
                                                             const float* __restrict__ p, int n,
                                                             double t, float* __restrict__ grad,
                                                             double* __restrict__ grad_k,
                                                             double* __restrict__ grad_alpha) {
  static_assert(!VEC || ITEMS % 4 == 0, "float4 items");
  constexpr int WAVES = BLOCK / kWave;
  constexpr int NS = PARAMS ? 4 : 2;
  __shared__ double red[NS * WAVES];
  const int tid = threadIdx.x;
  const int64_t row = blockIdx.x;
  const float* pr = p + row * n;
  const float* gr = g + row * n;
  auto index = [&](int i) { return VEC ? 4 * (tid + BLOCK * (i / 4)) + (i % 4) : tid + BLOCK * i; };
  float pv[ITEMS], gv[ITEMS];
  if constexpr (VEC) {
    const float4* p4 = reinterpret_cast<const float4*>(pr);
    const float4* g4 = reinterpret_cast<const float4*>(gr);
    const int n4 = n / 4;
#pragma unroll
    for (int j = 0; j < ITEMS / 4; ++j) {
      const int q = tid + BLOCK * j;
      const bool in = q < n4;
      const float4 a = in ? p4[q] : make_float4(0.f, 0.f, 0.f, 0.f);
      const float4 c = in ? g4[q] : make_float4(0.f, 0.f, 0.f, 0.f);
      pv[4 * j] = a.x; pv[4 * j + 1] = a.y; pv[4 * j + 2] = a.z; pv[4 * j + 3] = a.w;
      gv[4 * j] = c.x; gv[4 * j + 1] = c.y; gv[4 * j + 2] = c.z; gv[4 * j + 3] = c.w;
    }
  } else {
#pragma unroll
    for (int i = 0; i < ITEMS; ++i) {
      const int j = index(i);
      pv[i] = j < n ? pr[j] : 0.0f;
      gv[i] = j < n ? gr[j] : 0.0f;
    }
  }
  double F = 0.0, G = 0.0, U = 0.0, H = 0.0;
#pragma unroll
  for (int i = 0; i < ITEMS; ++i) {
    const float pp = pv[i];
    const float f = fminf(pp, 1.0f - pp);   // e^{-|b-r|/t} / 2, exact from p (0 past n)
    F += static_cast<double>(f);
    // g is not used where f == 0 (p exactly 0 or 1)
    const double fg = f != 0.0f ? static_cast<double>(f) * static_cast<double>(gv[i]) : 0.0;
    G += fg;
    if constexpr (PARAMS) {
      if (f != 0.0f) {
        const double u = static_cast<double>(laplace_u_from_p(pp, f));
        U += static_cast<double>(f) * u;
        H += fg * u;
      }
    }
  }
  F = wave_sum(F);
  G = wave_sum(G);
  if constexpr (PARAMS) {
    U = wave_sum(U);
    H = wave_sum(H);
  }
  const int wid = tid / kWave;
  if (lane_id() == 0) {
    red[wid] = F;
    red[WAVES + wid] = G;
    if constexpr (PARAMS) {
      red[2 * WAVES + wid] = U;
      red[3 * WAVES + wid] = H;
    }
  }
  __syncthreads();
  F = 0.0;
  G = 0.0;
#pragma unroll
  for (int w = 0; w < WAVES; ++w) {
    F += red[w];
    G += red[WAVES + w];
  }
  // grad_r = (f/t) (g - <g, q>), q = f / sum f; zero when sum f == 0
  const double coef = (F > 0.0) ? G / F : 0.0;
  const double scale = (F > 0.0) ? 1.0 / t : 0.0;
  if constexpr (PARAMS) {
    if (tid == 0) {
      U = 0.0;
      H = 0.0;
#pragma unroll
      for (int w = 0; w < WAVES; ++w) {
        U += red[2 * WAVES + w];
        H += red[3 * WAVES + w];
      }
      if (grad_k) grad_k[row] = coef;
      if (grad_alpha) grad_alpha[row] = (F > 0.0) ? (H - (U / F) * G) / t : 0.0;
    }
  }
  // the write in float32 (the sums above are float64): each output carries
  // a few float32 roundings, far below the VJP's tolerance
  const float coef32 = static_cast<float>(coef);
  const float scale32 = static_cast<float>(scale);
  auto one = [&](int i) -> float {
    const float f = fminf(pv[i], 1.0f - pv[i]);
    return (f != 0.0f) ? (f * scale32) * (gv[i] - coef32) : 0.0f;
  };
  float* out = grad + row * n;
  if constexpr (VEC) {
    float4* o4 = reinterpret_cast<float4*>(out);
    const int n4 = n / 4;
#pragma unroll
    for (int j = 0; j < ITEMS / 4; ++j) {
      const int q = tid + BLOCK * j;
      if (q < n4) o4[q] = make_float4(one(4 * j), one(4 * j + 1), one(4 * j + 2), one(4 * j + 3));
    }
  } else {
#pragma unroll
    for (int i = 0; i < ITEMS; ++i) {
      const int j = index(i);
      if (j < n) out[j] = one(i);
    }
  }
}

namespace {

template <int BLOCK, int ITEMS>
hipError_t fwd_items(const float* scores, int64_t batch, int64_t n, double k, double t, float* p,
                     double* b, int32_t* perm, bool gated, hipStream_t s) {
  const char* name = gated ? "row_forward_gated" : "row_forward";
  if (perm)
    { ProfScope ps_(name, s);
    hipLaunchKernelGGL((row_forward_kernel<BLOCK, ITEMS, true>), dim3(batch), dim3(BLOCK), 0, s,
                       scores, static_cast<int>(n), k, t, p, b, perm, gated ? 1 : 0); }
  else
    { ProfScope ps_(name, s);
    hipLaunchKernelGGL((row_forward_kernel<BLOCK, ITEMS, false>), dim3(batch), dim3(BLOCK), 0, s,
                       scores, static_cast<int>(n), k, t, p, b, perm, gated ? 1 : 0); }
  return hipGetLastError();
}

template <int BLOCK, int ITEMS>
hipError_t bwd_items(const float* g, const float* p, int64_t batch, int64_t n, double t,
                     float* grad, double* grad_k, double* grad_alpha, hipStream_t s) {
  const bool vec = (n % 4) == 0 && ITEMS % 4 == 0;
  { ProfScope ps_("row_backward", s);
#define LAPSUM_ROWBWD(P, V)                                                                      \
  hipLaunchKernelGGL((row_backward_kernel<BLOCK, ITEMS, P, V>), dim3(batch), dim3(BLOCK), 0, s, g, \
                     p, static_cast<int>(n), t, grad, grad_k, grad_alpha)
  if (grad_k || grad_alpha) {
    if (vec) LAPSUM_ROWBWD(true, ITEMS % 4 == 0); else LAPSUM_ROWBWD(true, false);
  } else {
    if (vec) LAPSUM_ROWBWD(false, ITEMS % 4 == 0); else LAPSUM_ROWBWD(false, false);
  }
#undef LAPSUM_ROWBWD
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_row_forward(const float* scores, int64_t batch, int64_t n, double k, double t,
                              float* p, double* b, int32_t* perm, bool gated, hipStream_t s) {
  if (n <= 256) return fwd_items<256, 1>(scores, batch, n, k, t, p, b, perm, gated, s);
  if (n <= 512) return fwd_items<256, 2>(scores, batch, n, k, t, p, b, perm, gated, s);
  if (n <= 1024) return fwd_items<256, 4>(scores, batch, n, k, t, p, b, perm, gated, s);
  if (n <= 2048) return fwd_items<256, 8>(scores, batch, n, k, t, p, b, perm, gated, s);
  if (n <= 4096) return fwd_items<1024, 4>(scores, batch, n, k, t, p, b, perm, gated, s);
  if (n <= 8192) return fwd_items<1024, 8>(scores, batch, n, k, t, p, b, perm, gated, s);
  if (n <= 16384) return fwd_items<1024, 16>(scores, batch, n, k, t, p, b, perm, gated, s);
  if (n <= kRowOnChipMax) return fwd_items<1024, 32>(scores, batch, n, k, t, p, b, perm, gated, s);
  return hipErrorInvalidValue;
}

hipError_t launch_row_backward(const float* grad_p, const float* p, int64_t batch, int64_t n,
                               double t, float* grad_r, double* grad_k, double* grad_alpha,
                               hipStream_t s) {
  if (n <= 1024) return bwd_items<256, 4>(grad_p, p, batch, n, t, grad_r, grad_k, grad_alpha, s);
  if (n <= 4096) return bwd_items<1024, 4>(grad_p, p, batch, n, t, grad_r, grad_k, grad_alpha, s);
  if (n <= 8192) return bwd_items<1024, 8>(grad_p, p, batch, n, t, grad_r, grad_k, grad_alpha, s);
  if (n <= 16384) return bwd_items<1024, 16>(grad_p, p, batch, n, t, grad_r, grad_k, grad_alpha, s);
  if (n <= kRowOnChipMax)
    return bwd_items<1024, 32>(grad_p, p, batch, n, t, grad_r, grad_k, grad_alpha, s);
  return hipErrorInvalidValue;
}

}  // namespace lapsum
