// Host eigensolver for the principal Query subspace (Eq. 15): symmetric
// threshold Jacobi in fp64 (Rutishauser's rotation form with accumulated
// diagonal updates). d <= 128, once per head at calibration time.
#include <algorithm>
#include <cmath>
#include <numeric>
#include <vector>

namespace qwm {

void host_eigh(const double* a_in, int n, double* lam, double* vecs_t) {
  std::vector<double> a(a_in, a_in + size_t(n) * n), v(size_t(n) * n, 0.0);
  std::vector<double> diag(n), acc(n, 0.0);
  for (int i = 0; i < n; ++i) {
    v[size_t(i) * n + i] = 1.0;
    diag[i] = a[size_t(i) * n + i];
  }
  auto at = [&](int i, int j) -> double& { return a[size_t(i) * n + j]; };
  for (int sweep = 0; sweep < 60; ++sweep) {
    double off = 0.0, scale = 0.0;
    for (int i = 0; i < n; ++i) {
      scale += diag[i] * diag[i];
      for (int j = i + 1; j < n; ++j) off += at(i, j) * at(i, j);
    }
    if (off == 0.0 || off <= 1e-30 * (scale + off)) break;
    const double thresh = sweep < 3 ? 0.2 * std::sqrt(off) / (double(n) * n) : 0.0;
    for (int p = 0; p < n - 1; ++p) {
      for (int q = p + 1; q < n; ++q) {
        const double apq = at(p, q);
        if (std::fabs(apq) <= thresh || apq == 0.0) continue;
        const double diff = diag[q] - diag[p];
        const double theta = 0.5 * diff / apq;
        double t = 1.0 / (std::fabs(theta) + std::sqrt(1.0 + theta * theta));
        if (theta < 0.0) t = -t;
        const double c = 1.0 / std::sqrt(1.0 + t * t), s = t * c, tau = s / (1.0 + c);
        const double h = t * apq;
        acc[p] -= h; acc[q] += h;
        diag[p] -= h; diag[q] += h;
        at(p, q) = 0.0;
        for (int k = 0; k < p; ++k) {
          const double g = at(k, p), hh = at(k, q);
          at(k, p) = g - s * (hh + g * tau);
          at(k, q) = hh + s * (g - hh * tau);
        }
        for (int k = p + 1; k < q; ++k) {
          const double g = at(p, k), hh = at(k, q);
          at(p, k) = g - s * (hh + g * tau);
          at(k, q) = hh + s * (g - hh * tau);
        }
        for (int k = q + 1; k < n; ++k) {
          const double g = at(p, k), hh = at(q, k);
          at(p, k) = g - s * (hh + g * tau);
          at(q, k) = hh + s * (g - hh * tau);
        }
        for (int k = 0; k < n; ++k) {
          const double g = v[size_t(k) * n + p], hh = v[size_t(k) * n + q];
          v[size_t(k) * n + p] = g - s * (hh + g * tau);
          v[size_t(k) * n + q] = hh + s * (g - hh * tau);
        }
      }
    }
    // refresh the diagonal: original entry plus the sum of its rotation updates
    for (int i = 0; i < n; ++i) diag[i] = at(i, i) + acc[i];
  }
  // descending eigenvalues, equal values keep their index; largest-magnitude
  // entry of each eigenvector positive (lowest index on ties)
  std::vector<int> order(n);
  std::iota(order.begin(), order.end(), 0);
  std::stable_sort(order.begin(), order.end(), [&](int x, int y) { return diag[x] > diag[y]; });
  for (int i = 0; i < n; ++i) {
    const int o = order[i];
    lam[i] = diag[o];
    int arg = 0;
    for (int k = 1; k < n; ++k)
      if (std::fabs(v[size_t(k) * n + o]) > std::fabs(v[size_t(arg) * n + o])) arg = k;
    const double sg = v[size_t(arg) * n + o] < 0.0 ? -1.0 : 1.0;
    for (int k = 0; k < n; ++k) vecs_t[size_t(i) * n + k] = sg * v[size_t(k) * n + o];
  }
}

}  // namespace qwm
