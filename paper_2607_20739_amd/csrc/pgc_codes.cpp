// Host-side tables of pipelined gradient coding (see pgc_codes.h).
#include "pgc_codes.h"

#include <algorithm>
#include <cmath>
#include <numeric>

namespace pgc {

int held_partition(int scheme, int n, int c, int i, int l) {
  if (scheme == kFR) return (i / c) * c + l;
  return (i + l) % n;
}

uint64_t splitmix64(uint64_t seed, uint64_t index) {
  // Golden-ratio increment and the variant-13 output mix of SplitMix64.
  uint64_t z = seed + (index + 1) * 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

namespace {

// Uniform double in [0, 1) from the top 53 bits (exact).
double uniform01(uint64_t z) { return static_cast<double>(z >> 11) * 0x1.0p-53; }

// Integer in [0, r) by Lemire's multiply-shift on the top 32 bits (r < 2^32).
uint64_t bounded(uint64_t z, uint64_t r) { return ((z >> 32) * r) >> 32; }

// Keep k items chosen by a partial Fisher-Yates shuffle that consumes draws
// first_draw, first_draw + 1, ... of step t.
void partial_shuffle(uint64_t seed, int64_t t, uint64_t first_draw,
                     std::vector<int>* items, int k) {
  const int len = static_cast<int>(items->size());
  for (int i = 0; i < k; ++i) {
    const int r = static_cast<int>(bounded(step_draw(seed, t, first_draw + i),
                                           static_cast<uint64_t>(len - i)));
    std::swap((*items)[i], (*items)[i + r]);
  }
  items->resize(k);
}

}  // namespace

bool make_mask(uint64_t seed, int64_t t, int policy, int n, int cap, double p,
               uint8_t* out) {
  if (n <= 0 || cap < 0 || t < 0 || out == nullptr) return false;
  std::vector<int> chosen;
  if (policy == 0) {
    chosen.resize(n);
    std::iota(chosen.begin(), chosen.end(), 0);
    partial_shuffle(seed, t, 0, &chosen, std::min(cap, n));
  } else if (policy == 1) {
    const int count = static_cast<int>(bounded(step_draw(seed, t, 0), static_cast<uint64_t>(cap) + 1));
    chosen.resize(n);
    std::iota(chosen.begin(), chosen.end(), 0);
    partial_shuffle(seed, t, 1, &chosen, std::min(count, n));
  } else if (policy == 2) {
    if (!(p >= 0.0 && p <= 1.0)) return false;
    for (int i = 0; i < n; ++i)
      if (uniform01(step_draw(seed, t, static_cast<uint64_t>(i))) < p) chosen.push_back(i);
    if (static_cast<int>(chosen.size()) > cap)
      partial_shuffle(seed, t, static_cast<uint64_t>(n), &chosen, cap);
  } else if (policy == 3) {
    // The cap workers with the largest delay draws (lower index first on ties).
    std::vector<double> u(n);
    for (int i = 0; i < n; ++i) u[i] = uniform01(step_draw(seed, t, static_cast<uint64_t>(i)));
    chosen.resize(n);
    std::iota(chosen.begin(), chosen.end(), 0);
    std::stable_sort(chosen.begin(), chosen.end(), [&](int a, int b) { return u[a] > u[b]; });
    chosen.resize(std::min(cap, n));
  } else {
    return false;
  }
  std::fill(out, out + n, uint8_t{0});
  for (int i : chosen) out[i] = 1;
  return true;
}

bool delay_step(uint64_t seed, int64_t t, int n, int s, double mean_delay, double compute_seconds,
                uint8_t* mask, double* delays, double* step_seconds) {
  if (n <= 0 || s < 0 || s >= n || t < 0 || mask == nullptr || step_seconds == nullptr) return false;
  if (!(mean_delay >= 0.0 && std::isfinite(mean_delay))) return false;
  if (!(compute_seconds >= 0.0 && std::isfinite(compute_seconds))) return false;
  // Inverse-CDF exponential delays; the same uniforms rank the workers for the
  // mask, so the stragglers are exactly the s largest delays.
  std::vector<double> delay(n);
  for (int i = 0; i < n; ++i)
    delay[i] = -mean_delay * std::log1p(-uniform01(step_draw(seed, t, static_cast<uint64_t>(i))));
  if (!make_mask(seed, t, 3, n, s, 0.0, mask)) return false;
  std::vector<double> sorted(delay);
  std::sort(sorted.begin(), sorted.end());
  *step_seconds = compute_seconds + sorted[n - s - 1];
  if (delays != nullptr) std::copy(delay.begin(), delay.end(), delays);
  return true;
}

std::vector<double> null_space_generator(uint64_t seed, int s, int n) {
  std::vector<double> H(static_cast<size_t>(s) * n, 0.0);
  for (int a = 0; a < s; ++a) {
    double acc = 0.0;
    for (int k = 0; k < n - 1; ++k) {
      const double v = 2.0 * uniform01(step_draw(seed, 0, static_cast<uint64_t>(a) * n + k)) - 1.0;
      H[static_cast<size_t>(a) * n + k] = v;
      acc += v;
    }
    H[static_cast<size_t>(a) * n + (n - 1)] = -acc;
  }
  return H;
}

namespace {

// Solve the dense s x s system M x = r (row-major M) by Gaussian elimination
// with partial pivoting.  Returns false when a pivot vanishes.
bool solve_dense(int s, std::vector<double> M, std::vector<double> r, std::vector<double>* x) {
  double scale = 0.0;
  for (double v : M) scale = std::max(scale, std::fabs(v));
  if (scale == 0.0) return false;
  for (int k = 0; k < s; ++k) {
    int piv = k;
    for (int i = k + 1; i < s; ++i)
      if (std::fabs(M[i * s + k]) > std::fabs(M[piv * s + k])) piv = i;
    if (std::fabs(M[piv * s + k]) <= 1e-13 * scale) return false;
    if (piv != k) {
      for (int j = 0; j < s; ++j) std::swap(M[k * s + j], M[piv * s + j]);
      std::swap(r[k], r[piv]);
    }
    for (int i = k + 1; i < s; ++i) {
      const double f = M[i * s + k] / M[k * s + k];
      if (f == 0.0) continue;
      for (int j = k; j < s; ++j) M[i * s + j] -= f * M[k * s + j];
      r[i] -= f * r[k];
    }
  }
  x->assign(s, 0.0);
  for (int i = s - 1; i >= 0; --i) {
    double acc = r[i];
    for (int j = i + 1; j < s; ++j) acc -= M[i * s + j] * (*x)[j];
    (*x)[i] = acc / M[i * s + i];
  }
  return true;
}

// Householder reflector H = I - tau v v^T with v[0] = 1 mapping x to beta e_1.
// x (length len, stride 1) is overwritten: x[0] = beta, x[1..] = v[1..].
double householder(double* x, int len) {
  double tail = 0.0;
  for (int i = 1; i < len; ++i) tail += x[i] * x[i];
  if (tail == 0.0) return 0.0;
  const double alpha = x[0];
  const double beta = (alpha >= 0.0 ? -1.0 : 1.0) * std::sqrt(alpha * alpha + tail);
  const double tau = (beta - alpha) / beta;
  const double inv = 1.0 / (alpha - beta);
  for (int i = 1; i < len; ++i) x[i] *= inv;
  x[0] = beta;
  return tau;
}

// y <- H y for the reflector stored in v (v[0] implicitly 1), length len.
void apply_reflector(const double* v, double tau, double* y, int len) {
  if (tau == 0.0) return;
  double w = y[0];
  for (int i = 1; i < len; ++i) w += v[i] * y[i];
  w *= tau;
  y[0] -= w;
  for (int i = 1; i < len; ++i) y[i] -= w * v[i];
}

}  // namespace

int min_norm_solve(int rows, int cols, const std::vector<double>& A_colmajor,
                   const std::vector<double>& b, std::vector<double>* x) {
  std::vector<double> A = A_colmajor;
  std::vector<int> perm(cols);
  std::iota(perm.begin(), perm.end(), 0);
  const int kmax = std::min(rows, cols);
  std::vector<double> tau(kmax, 0.0);
  auto at = [&](int i, int j) -> double& { return A[static_cast<size_t>(j) * rows + i]; };

  // QR with column pivoting: A P = Q R.
  for (int k = 0; k < kmax; ++k) {
    int piv = k;
    double best = -1.0;
    for (int j = k; j < cols; ++j) {
      double nrm = 0.0;
      for (int i = k; i < rows; ++i) nrm += at(i, j) * at(i, j);
      if (nrm > best) { best = nrm; piv = j; }
    }
    if (piv != k) {
      for (int i = 0; i < rows; ++i) std::swap(at(i, k), at(i, piv));
      std::swap(perm[k], perm[piv]);
    }
    tau[k] = householder(&at(k, k), rows - k);
    for (int j = k + 1; j < cols; ++j) {
      // Apply the reflector to column j below row k.
      double w = at(k, j);
      for (int i = k + 1; i < rows; ++i) w += at(i, k) * at(i, j);
      w *= tau[k];
      at(k, j) -= w;
      for (int i = k + 1; i < rows; ++i) at(i, j) -= w * at(i, k);
    }
  }
  // c = Q^T b.
  std::vector<double> qb = b;
  std::vector<double> col(rows);
  for (int k = 0; k < kmax; ++k) {
    for (int i = k; i < rows; ++i) col[i] = at(i, k);
    col[k] = 1.0;
    apply_reflector(&col[k], tau[k], &qb[k], rows - k);
  }
  // Numerical rank from the pivoted diagonal.
  int rank = 0;
  const double r00 = kmax > 0 ? std::fabs(at(0, 0)) : 0.0;
  while (rank < kmax && std::fabs(at(rank, rank)) > 1e-11 * r00) ++rank;

  x->assign(cols, 0.0);
  if (rank == 0) return 0;
  // The leading rank x cols block R1 is upper trapezoidal.  QR of R1^T
  // (cols x rank): R1^T = Z T, so R1 = T^T Z^T and the minimum-norm solution
  // of R1 x' = c is x' = Z [T^{-T} c; 0].
  std::vector<double> M(static_cast<size_t>(cols) * rank, 0.0);   // R1^T, column-major cols x rank
  auto m_at = [&](int i, int j) -> double& { return M[static_cast<size_t>(j) * cols + i]; };
  for (int i = 0; i < rank; ++i)
    for (int j = i; j < cols; ++j) m_at(j, i) = at(i, j);
  std::vector<double> ztau(rank, 0.0);
  for (int k = 0; k < rank; ++k) {
    ztau[k] = householder(&m_at(k, k), cols - k);
    for (int j = k + 1; j < rank; ++j) {
      double w = m_at(k, j);
      for (int i = k + 1; i < cols; ++i) w += m_at(i, k) * m_at(i, j);
      w *= ztau[k];
      m_at(k, j) -= w;
      for (int i = k + 1; i < cols; ++i) m_at(i, j) -= w * m_at(i, k);
    }
  }
  // Forward substitution T^T u = c (T upper triangular, rank x rank).
  std::vector<double> xp(cols, 0.0);
  for (int i = 0; i < rank; ++i) {
    double acc = qb[i];
    for (int j = 0; j < i; ++j) acc -= m_at(j, i) * xp[j];
    xp[i] = acc / m_at(i, i);
  }
  // x' = Z [u; 0], applying the reflectors in reverse order.
  std::vector<double> v(cols);
  for (int k = rank - 1; k >= 0; --k) {
    for (int i = k; i < cols; ++i) v[i] = m_at(i, k);
    v[k] = 1.0;
    apply_reflector(&v[k], ztau[k], &xp[k], cols - k);
  }
  for (int i = 0; i < cols; ++i) (*x)[perm[i]] = xp[i];
  return rank;
}

bool cyclic_encoding_matrix(int n, int c, const std::vector<double>& H,
                            std::vector<double>* B, std::string* err) {
  const int s = c - 1;
  B->assign(static_cast<size_t>(n) * n, 0.0);
  for (int j = 0; j < n; ++j) {
    (*B)[static_cast<size_t>(j) * n + j] = 1.0;
    if (s == 0) continue;
    std::vector<double> M(static_cast<size_t>(s) * s), r(s), x;
    for (int a = 0; a < s; ++a) {
      for (int l = 1; l < c; ++l)
        M[static_cast<size_t>(a) * s + (l - 1)] = H[static_cast<size_t>(a) * n + (j + l) % n];
      r[a] = -H[static_cast<size_t>(a) * n + j];
    }
    if (!solve_dense(s, M, r, &x)) {
      if (err) *err = "encoding matrix: singular system for row " + std::to_string(j);
      return false;
    }
    for (int l = 1; l < c; ++l) (*B)[static_cast<size_t>(j) * n + (j + l) % n] = x[l - 1];
  }
  return true;
}

DecodeStatus decode_coefficients(int scheme, int n, int c, const std::vector<double>& B,
                                 const uint8_t* mask, Decode* out, std::string* err) {
  out->survivors.clear();
  for (int i = 0; i < n; ++i)
    if (mask[i] == 0) out->survivors.push_back(i);
  const int nj = static_cast<int>(out->survivors.size());
  if (scheme == kISSGD) {
    // Ignore-straggler SGD: the master averages whatever arrived (Sec. VI-A).
    if (nj < 1) {
      if (err) *err = "every worker straggles";
      return kDecodeStragglers;
    }
    out->d.assign(nj, 1.0);
    out->scale = 1.0 / nj;
    return kDecodeOk;
  }
  const int s = c - 1;
  if (nj < n - s) {
    if (err) *err = std::to_string(n - nj) + " stragglers exceed s = " + std::to_string(s);
    return kDecodeStragglers;
  }
  out->d.assign(nj, 0.0);
  if (scheme == kFR) {
    std::vector<int> seen(n / c, 0);
    for (int m = 0; m < nj; ++m) {
      const int g = out->survivors[m] / c;
      if (!seen[g]) { seen[g] = 1; out->d[m] = 1.0; }
    }
    for (int g = 0; g < n / c; ++g)
      if (!seen[g]) {
        if (err) *err = "FR group " + std::to_string(g) + " has no survivor";
        return kDecodeStragglers;
      }
    out->scale = 1.0 / n;
    return kDecodeOk;
  }
  if (scheme == kCR) {
    std::fill(out->d.begin(), out->d.end(), 1.0);
    out->scale = 1.0 / (static_cast<double>(nj) * c);
    return kDecodeOk;
  }
  // Real-valued code: A = B_J^T (n x |J|, column m = row J[m] of B).
  std::vector<double> A(static_cast<size_t>(n) * nj);
  for (int m = 0; m < nj; ++m)
    for (int k = 0; k < n; ++k)
      A[static_cast<size_t>(m) * n + k] = B[static_cast<size_t>(out->survivors[m]) * n + k];
  std::vector<double> ones(n, 1.0);
  min_norm_solve(n, nj, A, ones, &out->d);
  double resid = 0.0;
  for (int k = 0; k < n; ++k) {
    double acc = 0.0;
    for (int m = 0; m < nj; ++m) acc += A[static_cast<size_t>(m) * n + k] * out->d[m];
    resid = std::max(resid, std::fabs(acc - 1.0));
  }
  if (!(resid <= 1e-9)) {
    if (err) *err = "real-valued code cannot decode this straggler set (residual " +
                    std::to_string(resid) + ")";
    return kDecodeSingular;
  }
  out->scale = 1.0 / n;
  return kDecodeOk;
}

}  // namespace pgc
