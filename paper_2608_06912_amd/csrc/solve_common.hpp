// Pieces shared by the sorted-array solve and the bucketed middle-set solve:
// the bracket tails as scan carries, the certificate of Suppl. B / Suppl. C
// from the scan totals, and the root above every score of the array.
#pragma once

#include <math.h>

#include "common.hpp"
#include "kernels.hpp"

namespace lapsum {
namespace {

struct Tails {
  double nR, nL;
  float aR, aL;
  Pre pre;   // R tail at a_R
  Suf suf;   // L tail at a_L
  bool bracketed;
};

__device__ Tails load_tails(const PartTotals* tot) {
  Tails x;
  if (tot == nullptr) {
    x.nR = x.nL = 0.0;
    x.aR = INFINITY;
    x.aL = -INFINITY;
    x.pre = pre_empty();
    x.suf = suf_empty();
    x.bracketed = false;
    return x;
  }
  x.nR = static_cast<double>(tot->nR);
  x.nL = static_cast<double>(tot->nL);
  x.aR = tot->aR;
  x.aL = tot->aL;
  x.pre = (tot->nR > 0 && tot->TR > 0.0) ? Pre{tot->aR, tot->TR} : pre_empty();
  x.suf = (tot->nL > 0 && tot->TL > 0.0) ? Suf{tot->aL, tot->TL} : suf_empty();
  x.bracketed = true;
  return x;
}

// Certificate values from the scan totals.  pre_all = R tail (+) M (anchor:
// last of M, or a_R when M is empty); suf_all = M (+) L tail.
__device__ void certify(const Tails& x, double m_len, double n_total, double k, double t,
                        Pre pre_all, Suf suf_all, SolveRec& rec) {
  const double inv_t = 1.0 / t;
  double lap_aR = 0.0, lap_aL = n_total;
  if (isfinite(x.aR)) {
    // scores >= a_R contribute 1 - e^{-(r-a_R)/t}/2, the others e^{-(a_R-r)/t}/2
    const double TR = x.pre.S;
    lap_aR = x.nR - 0.5 * TR;
    if (suf_all.T != 0.0)
      lap_aR += 0.5 * wexp_f64(static_cast<double>(x.aR) - static_cast<double>(suf_all.v), inv_t) * suf_all.T;
  }
  if (isfinite(x.aL)) {
    lap_aL = x.nR + m_len + 0.5 * x.suf.T;
    if (pre_all.S != 0.0)
      lap_aL -= 0.5 * wexp_f64(static_cast<double>(pre_all.u) - static_cast<double>(x.aL), inv_t) * pre_all.S;
  }
  rec.lap_aL = lap_aL;
  rec.lap_aR = lap_aR;
  const bool okR = lap_aR <= k;
  const bool okL = k <= lap_aL;
  rec.ok = (okR && okL) ? 1 : 0;
  rec.side = okR ? (okL ? 0 : -1) : 1;
}

// b when the array is empty, or when b lies above its first score:
// the c_up = n_R scores above are the R tail, the rest summarised by `below`.
__device__ double root_above(const Tails& x, Suf below, double k, double t) {
  const bool has_up = x.pre.S != 0.0;
  const bool has_dn = below.T != 0.0;
  return gap_root(k, t, x.nR, has_up, x.pre.u, has_up ? log(x.pre.S) : 0.0, has_dn, below.v,
                  has_dn ? log(below.T) : 0.0);
}

}  // namespace
}  // namespace lapsum
