// Adaptive segmented lookup tables (ROSETTA Sec. 3.1) on the host: segment
// boundaries, per-interval linear coefficients, the protocol polynomials of
// Sec. 3.2, fixed-point encoding into Z_p, and a cleartext simulator of the
// three-step lookup that reports precision in bits (-log2 RMSE, Sec. 5.1).
// The simulator can shift each input's interval index by a given offset,
// which models the selection error of the encrypted lookup (the modulus
// switch of the blind rotation moves the selected coefficient by a few
// positions).
//
// The domain [lo, hi] is cut into nseg segments (uniform or geometric
// boundaries); segment s holds nbr equal intervals, interval i carrying the
// line through f at the interval's two Chebyshev nodes c -+ r cos(pi/4)
// (c the midpoint, r the half-width) -- the paper prints the coefficients
// of its running example but not the fitting rule; this rule reproduces all
// of them -- or, for the single-LUT baseline, the constant f(c).
#include <cmath>
#include <cstdint>
#include <vector>

#include "gl.hpp"
#include "internal.hpp"
#include "rosetta.h"

using namespace rosetta;

namespace {

bool eval_fn(int fn, double x, double *y) {
  switch (fn) {
    case ROSETTA_FN_INV: *y = 1.0 / x; return true;
    case ROSETTA_FN_INV_SQRT: *y = 1.0 / std::sqrt(x); return true;
    case ROSETTA_FN_SILU: *y = x / (1.0 + std::exp(-x)); return true;
    case ROSETTA_FN_GELU: *y = 0.5 * x * (1.0 + std::erf(x / std::sqrt(2.0))); return true;
    case ROSETTA_FN_EXP: *y = std::exp(x); return true;
    default: return false;
  }
}

rosetta_status err(rosetta_status st, const char *msg) {
  set_last_error(msg);
  return st;
}

bool increasing(const double *tau, uint32_t nseg) {
  for (uint32_t s = 0; s < nseg; ++s)
    if (!(tau[s] < tau[s + 1])) return false;
  return true;
}

// Segment index S = #{j in 1..nseg-1 : x >= tau_j}, then the local interval
// floor((x - tau_S) / (tau_{S+1} - tau_S) * nbr) clamped to [0, nbr).
void locate(const double *tau, uint32_t nseg, uint32_t nbr, double x, uint32_t *S, uint32_t *I) {
  uint32_t s = 0;
  for (uint32_t j = 1; j < nseg; ++j) s += x >= tau[j] ? 1u : 0u;
  double t = std::floor((x - tau[s]) / (tau[s + 1] - tau[s]) * nbr);
  if (t < 0) t = 0;
  if (t > nbr - 1) t = nbr - 1;
  *S = s;
  *I = (uint32_t)t;
}

}  // namespace

extern "C" {

rosetta_status rosetta_seglut_boundaries(double lo, double hi, uint32_t nseg, int spacing,
                                         double *tau) {
  if (!tau) return err(ROSETTA_ERR_NULL, "tau is NULL");
  if (nseg < 1 || !(lo < hi)) return err(ROSETTA_ERR_PARAMS, "need nseg >= 1 and lo < hi");
  if (spacing == ROSETTA_SPACING_LOG && !(lo > 0))
    return err(ROSETTA_ERR_PARAMS, "log spacing needs lo > 0");
  if (spacing != ROSETTA_SPACING_UNIFORM && spacing != ROSETTA_SPACING_LOG)
    return err(ROSETTA_ERR_PARAMS, "unknown spacing");
  for (uint32_t j = 0; j <= nseg; ++j) {
    const double f = (double)j / nseg;
    tau[j] = spacing == ROSETTA_SPACING_LOG ? lo * std::pow(hi / lo, f) : lo + (hi - lo) * f;
  }
  tau[0] = lo;
  tau[nseg] = hi;
  return ROSETTA_OK;
}

rosetta_status rosetta_seglut_build(int function, const double *tau, uint32_t nseg, uint32_t nbr,
                                    int fit, double *a, double *b) {
  if (!tau || !a || !b) return err(ROSETTA_ERR_NULL, "NULL pointer argument");
  if (nseg < 1 || nbr < 1) return err(ROSETTA_ERR_PARAMS, "need nseg, nbr >= 1");
  if (!increasing(tau, nseg)) return err(ROSETTA_ERR_PARAMS, "boundaries must increase");
  if (fit != ROSETTA_FIT_LINEAR && fit != ROSETTA_FIT_CONSTANT)
    return err(ROSETTA_ERR_PARAMS, "unknown fit");
  double probe;
  if (!eval_fn(function, 1.0, &probe)) return err(ROSETTA_ERR_PARAMS, "unknown function");
  const double cq = std::cos(M_PI / 4);
  for (uint32_t s = 0; s < nseg; ++s) {
    const double w = (tau[s + 1] - tau[s]) / nbr;
    for (uint32_t i = 0; i < nbr; ++i) {
      const double lo = tau[s] + i * w, hi = tau[s] + (i + 1) * w;
      const double c = (lo + hi) / 2, r = (hi - lo) / 2;
      double *as = a + (size_t)s * nbr + i, *bs = b + (size_t)s * nbr + i;
      if (fit == ROSETTA_FIT_CONSTANT) {
        *as = 0.0;
        eval_fn(function, c, bs);
      } else {
        const double x1 = c - r * cq, x2 = c + r * cq;
        double y1, y2;
        eval_fn(function, x1, &y1);
        eval_fn(function, x2, &y2);
        const double slope = (y2 - y1) / (x2 - x1);
        *as = slope;
        *bs = y1 - slope * x1;
      }
    }
  }
  return ROSETTA_OK;
}

rosetta_status rosetta_seglut_protocol_polys(const double *tau, uint32_t nseg, uint32_t nbr,
                                             double *p, double *q) {
  if (!tau || !p || !q) return err(ROSETTA_ERR_NULL, "NULL pointer argument");
  if (nseg < 1 || nbr < 1) return err(ROSETTA_ERR_PARAMS, "need nseg, nbr >= 1");
  if (!increasing(tau, nseg)) return err(ROSETTA_ERR_PARAMS, "boundaries must increase");
  for (uint32_t s = 0; s < nseg; ++s) {
    const double w = tau[s + 1] - tau[s];
    p[s] = nbr / w;
    q[s] = -tau[s] * nbr / w;
  }
  return ROSETTA_OK;
}

rosetta_status rosetta_seglut_eval(const double *tau, uint32_t nseg, uint32_t nbr,
                                   const double *a, const double *b, const double *x,
                                   const int32_t *index_offset, size_t count, double *y) {
  if (!tau || !a || !b || (count && (!x || !y))) return err(ROSETTA_ERR_NULL, "NULL pointer");
  if (nseg < 1 || nbr < 1) return err(ROSETTA_ERR_PARAMS, "need nseg, nbr >= 1");
  if (!increasing(tau, nseg)) return err(ROSETTA_ERR_PARAMS, "boundaries must increase");
  for (size_t k = 0; k < count; ++k) {
    uint32_t S, I;
    locate(tau, nseg, nbr, x[k], &S, &I);
    if (index_offset) {
      const int64_t J = (int64_t)I + index_offset[k];
      I = (uint32_t)(J < 0 ? 0 : (J > (int64_t)nbr - 1 ? (int64_t)nbr - 1 : J));
    }
    y[k] = a[(size_t)S * nbr + I] * x[k] + b[(size_t)S * nbr + I];
  }
  return ROSETTA_OK;
}

rosetta_status rosetta_seglut_precision(int function, const double *tau, uint32_t nseg,
                                        uint32_t nbr, const double *a, const double *b,
                                        const double *x, const int32_t *index_offset,
                                        size_t count, double *bits) {
  if (!bits) return err(ROSETTA_ERR_NULL, "bits is NULL");
  if (count == 0) return err(ROSETTA_ERR_PARAMS, "need count >= 1");
  std::vector<double> y(count);
  rosetta_status st =
      rosetta_seglut_eval(tau, nseg, nbr, a, b, x, index_offset, count, y.data());
  if (st) return st;
  double se = 0;
  for (size_t k = 0; k < count; ++k) {
    double f;
    if (!eval_fn(function, x[k], &f)) return err(ROSETTA_ERR_PARAMS, "unknown function");
    se += (y[k] - f) * (y[k] - f);
  }
  *bits = -std::log2(std::sqrt(se / count));
  return ROSETTA_OK;
}

rosetta_status rosetta_encode_fixed(const double *v, size_t count, int scale_log,
                                    uint64_t *out) {
  if (count && (!v || !out)) return err(ROSETTA_ERR_NULL, "NULL pointer argument");
  if (scale_log < 0 || scale_log > 62) return err(ROSETTA_ERR_PARAMS, "need 0 <= scale_log <= 62");
  for (size_t k = 0; k < count; ++k) {
    const double r = std::nearbyint(std::ldexp(v[k], scale_log));
    if (!(std::fabs(r) < 0x1p62)) return err(ROSETTA_ERR_PARAMS, "value out of range for the scale");
    out[k] = gl_from_i64((int64_t)r);
  }
  return ROSETTA_OK;
}

}  // extern "C"
