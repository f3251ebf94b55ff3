// Layer allocator of section IV-D: Algorithm 1 (coarse allocation by
// memory) and Algorithm 2 (workload fine-tuning) over a partition index
// pi[0..D], device i holding layers pi[i] .. pi[i+1]-1.  Host code only.
#include <cmath>
#include <vector>

#include "../../include/alloc.h"

namespace {

bool finite_nonneg(const double* v, int n) {
  for (int k = 0; k < n; ++k)
    if (!std::isfinite(v[k]) || v[k] < 0.0) return false;
  return true;
}

bool valid_pi(int L, int D, const int* pi) {
  if (pi[0] != 0 || pi[D] != L) return false;
  for (int i = 0; i < D; ++i)
    if (pi[i + 1] <= pi[i]) return false;
  return true;
}

int layers_of(const std::vector<int>& pi, int i) { return pi[i + 1] - pi[i]; }

// Memory allocated to device i (sum of lm over its block).
double mem_of(const std::vector<int>& pi, const double* lm, int i) {
  double s = 0.0;
  for (int j = pi[i]; j < pi[i + 1]; ++j) s += lm[j];
  return s;
}

// Section IV-D workload: sum over the block of dt[i] * lf[j] + ct[i].
double work_of(const std::vector<int>& pi, const double* dt, const double* ct, const double* lf,
               int i) {
  double s = 0.0;
  for (int j = pi[i]; j < pi[i + 1]; ++j) s += dt[i] * lf[j] + ct[i];
  return s;
}

}  // namespace

extern "C" {

alloc_status alloc_coarse(int L, int D, const double* lm, const double* dm, int* pi_out,
                          int* sweeps) {
  if (sweeps) *sweeps = 0;
  if (D < 1 || L < D || !lm || !dm || !pi_out) return ALLOC_EINVAL;
  if (!finite_nonneg(lm, L) || !finite_nonneg(dm, D)) return ALLOC_EINVAL;
  // Equal split: device i starts at floor(i L / D).
  std::vector<int> pi(D + 1);
  for (int i = 0; i <= D; ++i) pi[i] = (int)((long long)i * L / D);
  std::vector<double> am(D);
  auto fits = [&]() {
    for (int i = 0; i < D; ++i)
      if (am[i] > dm[i]) return false;
    return true;
  };
  for (int i = 0; i < D; ++i) am[i] = mem_of(pi, lm, i);
  alloc_status st = ALLOC_ENOFIT;
  int n = 0;  // sweeps run
  // Each sweep either changes pi or ends the search; L * D sweeps bound a
  // search that keeps moving layers without meeting the limits.  Allocated
  // memory is re-summed over the block after every move (no drift).
  for (;;) {
    if (fits()) {
      st = ALLOC_OK;
      break;
    }
    if (n > L * D) break;
    const std::vector<int> before = pi;
    for (int i = 0; i + 1 < D; ++i) {
      // over the limit: hand the last layer to device i+1
      while (am[i] > dm[i] && layers_of(pi, i) > 1) {
        pi[i + 1] -= 1;
        am[i] = mem_of(pi, lm, i);
        am[i + 1] = mem_of(pi, lm, i + 1);
      }
      // room for device i+1's first layer: take it
      while (dm[i] > am[i] + lm[pi[i + 1]] && layers_of(pi, i + 1) > 1) {
        pi[i + 1] += 1;
        am[i] = mem_of(pi, lm, i);
        am[i + 1] = mem_of(pi, lm, i + 1);
      }
    }
    ++n;
    if (pi == before) break;
  }
  if (sweeps) *sweeps = n;
  for (int i = 0; i <= D; ++i) pi_out[i] = pi[i];
  return st;
}

alloc_status alloc_fine(int L, int D, const double* dt, const double* dm, const double* ct,
                        const double* lf, const double* lm, int max_iter, int* pi_io,
                        int* rounds) {
  if (rounds) *rounds = 0;
  if (D < 1 || L < D || !dt || !dm || !ct || !lf || !lm || !pi_io || max_iter < 0)
    return ALLOC_EINVAL;
  if (!finite_nonneg(dt, D) || !finite_nonneg(dm, D) || !finite_nonneg(ct, D) ||
      !finite_nonneg(lf, L) || !finite_nonneg(lm, L) || !valid_pi(L, D, pi_io))
    return ALLOC_EINVAL;
  std::vector<int> pi(pi_io, pi_io + D + 1);
  int counter = 0;
  while (counter < max_iter) {
    // target: mean workload of the partition at the start of the round
    double target = 0.0;
    for (int i = 0; i < D; ++i) target += work_of(pi, dt, ct, lf, i);
    target /= D;
    const std::vector<int> before = pi;
    for (int i = 0; i + 1 < D; ++i) {
      const double w_this = work_of(pi, dt, ct, lf, i);
      const int first_next = pi[i + 1];  // device i+1's first layer
      if (w_this < target && layers_of(pi, i + 1) > 1 &&
          mem_of(pi, lm, i) + lm[first_next] <= dm[i]) {
        pi[i + 1] += 1;
      } else {
        const double w_next = work_of(pi, dt, ct, lf, i + 1);
        const int last_this = pi[i + 1] - 1;  // device i's last layer
        const double w_last = dt[i] * lf[last_this] + ct[i];
        if (w_next < target && w_this - w_last > target && layers_of(pi, i) > 1 &&
            mem_of(pi, lm, i + 1) + lm[last_this] <= dm[i + 1]) {
          pi[i + 1] -= 1;
        }
      }
    }
    ++counter;
    if (pi == before) break;
  }
  if (rounds) *rounds = counter;
  for (int i = 0; i <= D; ++i) pi_io[i] = pi[i];
  return ALLOC_OK;
}

alloc_status alloc_workloads(int L, int D, const double* dt, const double* ct, const double* lf,
                             const int* pi, alloc_ct_mode mode, double* w_out) {
  if (D < 1 || L < D || !dt || !ct || !lf || !pi || !w_out) return ALLOC_EINVAL;
  if (mode != ALLOC_CT_PER_LAYER && mode != ALLOC_CT_PER_DEVICE) return ALLOC_EINVAL;
  if (!finite_nonneg(dt, D) || !finite_nonneg(ct, D) || !finite_nonneg(lf, L) ||
      !valid_pi(L, D, pi))
    return ALLOC_EINVAL;
  std::vector<int> p(pi, pi + D + 1);
  for (int i = 0; i < D; ++i) {
    if (mode == ALLOC_CT_PER_DEVICE) {
      double f = 0.0;
      for (int j = pi[i]; j < pi[i + 1]; ++j) f += lf[j];
      w_out[i] = dt[i] * f + ct[i];
    } else {
      w_out[i] = work_of(p, dt, ct, lf, i);
    }
  }
  return ALLOC_OK;
}

}  // extern "C"
