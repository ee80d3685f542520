// SLO-constrained EC-aware chunk scheduling (SPEAR §4.3): iteration latency
// from per-module latency tables, and the largest prefill chunk that keeps an
// iteration within the latency target. Host code only; the ABI and the
// readings taken where the paper is silent are documented in spear_sched.h.
#include "spear_sched.h"

#include <cmath>
#include <cstddef>
#include <vector>

namespace {

constexpr int32_t kMaxTable = 1 << 16;
constexpr int64_t kMaxCalls = 1 << 20;

bool table_ok(const spear_lut_t* t) {
  if (!t || t->n < 1 || t->n > kMaxTable || !t->M || !t->lat_w4 || !t->lat_ec) return false;
  for (int32_t i = 0; i < t->n; ++i) {
    if (t->M[i] < 1 || (i > 0 && t->M[i] <= t->M[i - 1])) return false;
    const double a = t->lat_w4[i], b = t->lat_ec[i];
    if (!std::isfinite(a) || !std::isfinite(b) || a < 0.0 || b < 0.0) return false;
  }
  return true;
}

spear_status_t model_ok(const spear_model_lat_t* m) {
  if (!m || !m->luts || !m->selection) return SPEAR_E_NULL;
  if (m->layers < 1 || m->modules < 1 || (int64_t)m->layers * m->modules > kMaxCalls)
    return SPEAR_E_SHAPE;
  for (int32_t j = 0; j < m->modules; ++j)
    if (!table_ok(&m->luts[j])) return SPEAR_E_SHAPE;
  if (m->extra && !table_ok(m->extra)) return SPEAR_E_SHAPE;
  return SPEAR_OK;
}

// One column of a table at token count x, read as its running maximum over
// M: floor below the first entry, linear between entries, linear
// extrapolation along the last segment above the last.
double lookup(const int64_t* M, const double* lat, int32_t n, int64_t x) {
  if (x <= 0) return 0.0;
  double prev = lat[0];  // running maximum up to entry i
  if (x <= M[0]) return prev;
  for (int32_t i = 1; i < n; ++i) {
    const double cur = lat[i] > prev ? lat[i] : prev;
    if (x <= M[i] || i == n - 1) {
      const double slope = (cur - prev) / (double)(M[i] - M[i - 1]);
      return prev + slope * (double)(x - M[i - 1]);
    }
    prev = cur;
  }
  return prev;  // n == 1 and x > M[0]
}

struct Counts {
  std::vector<int64_t> ec, w4;  // per module: layers with / without the EC
};

Counts count(const spear_model_lat_t* m) {
  Counts c;
  c.ec.assign(m->modules, 0);
  c.w4.assign(m->modules, 0);
  for (int32_t l = 0; l < m->layers; ++l)
    for (int32_t j = 0; j < m->modules; ++j) {
      if (m->selection[(size_t)l * m->modules + j]) ++c.ec[j];
      else ++c.w4[j];
    }
  return c;
}

// T_S(x) = sum over modules j of ec_j * l_EC,j(x) + w4_j * l_W4,j(x), in
// module order, plus layers * extra(x).
double iteration_us(const spear_model_lat_t* m, const Counts& c, int64_t x) {
  double t = 0.0;
  for (int32_t j = 0; j < m->modules; ++j) {
    const spear_lut_t& L = m->luts[j];
    if (c.ec[j]) t += (double)c.ec[j] * lookup(L.M, L.lat_ec, L.n, x);
    if (c.w4[j]) t += (double)c.w4[j] * lookup(L.M, L.lat_w4, L.n, x);
  }
  if (m->extra) t += (double)m->layers * lookup(m->extra->M, m->extra->lat_w4, m->extra->n, x);
  return t;
}

}  // namespace

extern "C" {

spear_status_t spear_sched_latency(const spear_model_lat_t* model, int64_t m, double* out_us) {
  if (!out_us) return SPEAR_E_NULL;
  const spear_status_t st = model_ok(model);
  if (st != SPEAR_OK) return st;
  *out_us = iteration_us(model, count(model), m);
  return SPEAR_OK;
}

spear_status_t spear_sched_chunk(const spear_model_lat_t* model, int64_t d, double t_slo_us,
                                 int64_t c_min, int64_t c_max, int64_t* out_c) {
  if (!out_c) return SPEAR_E_NULL;
  const spear_status_t st = model_ok(model);
  if (st != SPEAR_OK) return st;
  if (d < 0 || c_min < 1 || c_max < c_min || !std::isfinite(t_slo_us)) return SPEAR_E_SHAPE;
  const Counts c = count(model);
  const double td = iteration_us(model, c, d);
  auto fits = [&](int64_t x) { return td + iteration_us(model, c, x) <= t_slo_us; };
  if (!fits(c_min)) {
    *out_c = 0;
    return SPEAR_OK;
  }
  // T_S is nondecreasing: the chunks that fit form a prefix of [c_min, c_max]
  int64_t lo = c_min, hi = c_max;  // fits(lo) holds
  while (lo < hi) {
    const int64_t mid = lo + (hi - lo + 1) / 2;
    if (fits(mid)) lo = mid;
    else hi = mid - 1;
  }
  *out_c = lo;
  return SPEAR_OK;
}

}  // extern "C"
