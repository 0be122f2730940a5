// Exercises the library's host tables (placement, straggler masks, the delay
// model, the real-valued cyclic code, decode coefficients and the minimum-norm
// solver) under AddressSanitizer and UndefinedBehaviorSanitizer.  Built and run
// by tests/test_host_sanitize.py with g++; exits 0 when every check holds and
// the sanitizers report nothing.
#include <cmath>
#include <cstdio>
#include <cstdint>
#include <string>
#include <vector>

#include "pgc_codes.h"

namespace {

int failures = 0;

void check(bool ok, const std::string& what) {
  if (!ok) {
    ++failures;
    if (failures <= 20) std::fprintf(stderr, "FAILED: %s\n", what.c_str());
  }
}

// Small deterministic generator for test data (not the library's SplitMix64).
struct Lcg {
  uint64_t s;
  double uniform() {
    s = s * 6364136223846793005ull + 1442695040888963407ull;
    return static_cast<double>(s >> 11) * 0x1.0p-53;
  }
};

void placements() {
  const int shapes[][2] = {{1, 1}, {4, 2}, {6, 3}, {6, 6}, {12, 4}, {256, 8}, {7, 7}, {9, 2}};
  for (auto& nc : shapes) {
    const int n = nc[0], c = nc[1];
    for (int scheme : {pgc::kFR, pgc::kCR}) {
      if (scheme == pgc::kFR && n % c != 0) continue;
      std::vector<int> held(n, 0);
      for (int i = 0; i < n; ++i) {
        std::vector<int> mine;
        for (int l = 0; l < c; ++l) {
          const int k = pgc::held_partition(scheme, n, c, i, l);
          check(k >= 0 && k < n, "partition in range");
          if (k < 0 || k >= n) continue;
          ++held[k];
          for (int o : mine) check(o != k, "a worker's slots hold distinct partitions");
          mine.push_back(k);
        }
      }
      for (int k = 0; k < n; ++k) check(held[k] == c, "every partition held c times");
    }
  }
}

void masks() {
  std::vector<uint8_t> m(256);
  for (int policy = 0; policy < 4; ++policy)
    for (int n : {1, 2, 7, 64, 256})
      for (int cap : {0, 1, n / 2, n})
        for (double p : {0.0, 0.3, 1.0})
          for (int64_t t = 0; t < 12; ++t) {
            const bool ok = pgc::make_mask(99, t, policy, n, cap, p, m.data());
            check(ok, "make_mask accepts a valid request");
            int count = 0;
            for (int i = 0; i < n; ++i) {
              check(m[i] == 0 || m[i] == 1, "mask entries are 0 or 1");
              count += m[i];
            }
            const int top = cap < n ? cap : n;
            if (policy == 0 || policy == 3) check(count == top, "exact and slowest draw cap stragglers");
            else check(count <= top, "uniform-count and Bernoulli stay within cap");
            if (policy == 2 && p == 0.0) check(count == 0, "Bernoulli(0) draws no straggler");
          }
  check(!pgc::make_mask(1, 0, 0, 0, 0, 0.0, m.data()), "n = 0 rejected");
  check(!pgc::make_mask(1, 0, 0, 4, -1, 0.0, m.data()), "cap < 0 rejected");
  check(!pgc::make_mask(1, -1, 0, 4, 1, 0.0, m.data()), "t < 0 rejected");
  check(!pgc::make_mask(1, 0, 4, 4, 1, 0.0, m.data()), "unknown policy rejected");
  check(!pgc::make_mask(1, 0, 2, 4, 1, 1.5, m.data()), "p > 1 rejected");
  check(!pgc::make_mask(1, 0, 2, 4, 1, std::nan(""), m.data()), "p = NaN rejected");
  check(!pgc::make_mask(1, 0, 0, 4, 1, 0.0, nullptr), "null output rejected");
}

void delays() {
  std::vector<uint8_t> m(256);
  std::vector<double> d(256);
  for (int n : {1, 5, 256})
    for (int s : {0, n / 2, n - 1})
      for (int64_t t = 0; t < 6; ++t) {
        double seconds = -1.0;
        const bool ok = pgc::delay_step(7, t, n, s, 1.5, 0.25, m.data(), d.data(), &seconds);
        check(ok, "delay_step accepts a valid request");
        int count = 0;
        double slowest_waited = 0.0;
        for (int i = 0; i < n; ++i) {
          count += m[i];
          check(d[i] >= 0.0 && std::isfinite(d[i]), "delays are finite and non-negative");
          if (!m[i] && d[i] > slowest_waited) slowest_waited = d[i];
        }
        check(count == s, "the master skips exactly s workers");
        check(seconds == 0.25 + slowest_waited, "step time is compute plus the last waited delay");
        for (int i = 0; i < n; ++i)
          if (m[i]) check(d[i] >= slowest_waited, "skipped workers are the slowest");
      }
  double sec;
  check(!pgc::delay_step(7, 0, 4, 4, 1.0, 0.0, m.data(), nullptr, &sec), "s = n rejected");
  check(!pgc::delay_step(7, 0, 4, 1, std::nan(""), 0.0, m.data(), nullptr, &sec), "NaN mean rejected");
  check(!pgc::delay_step(7, 0, 4, 1, 1.0, -1.0, m.data(), nullptr, &sec), "negative compute rejected");
  check(!pgc::delay_step(7, 0, 4, 1, 1.0, 0.0, m.data(), nullptr, nullptr), "null step time rejected");
}

// Solves the r x r system M y = b by Gaussian elimination with partial pivoting.
std::vector<double> dense_solve(std::vector<double> M, std::vector<double> b, int r) {
  for (int col = 0; col < r; ++col) {
    int piv = col;
    for (int i = col + 1; i < r; ++i)
      if (std::fabs(M[i * r + col]) > std::fabs(M[piv * r + col])) piv = i;
    for (int j = 0; j < r; ++j) std::swap(M[col * r + j], M[piv * r + j]);
    std::swap(b[col], b[piv]);
    for (int i = col + 1; i < r; ++i) {
      const double f = M[i * r + col] / M[col * r + col];
      for (int j = col; j < r; ++j) M[i * r + j] -= f * M[col * r + j];
      b[i] -= f * b[col];
    }
  }
  std::vector<double> y(r);
  for (int i = r - 1; i >= 0; --i) {
    double acc = b[i];
    for (int j = i + 1; j < r; ++j) acc -= M[i * r + j] * y[j];
    y[i] = acc / M[i * r + i];
  }
  return y;
}

void solver() {
  Lcg g{12345};
  for (int trial = 0; trial < 200; ++trial) {
    const int rows = 1 + trial % 9, cols = rows + trial % 5;   // wide, full row rank
    std::vector<double> A(static_cast<size_t>(rows) * cols), b(rows);
    for (double& a : A) a = 2.0 * g.uniform() - 1.0;
    for (double& v : b) v = 2.0 * g.uniform() - 1.0;
    std::vector<double> x;
    const int rank = pgc::min_norm_solve(rows, cols, A, b, &x);
    check(rank == rows, "full row rank detected");
    // Reference: x = A^T (A A^T)^{-1} b.
    std::vector<double> AAt(static_cast<size_t>(rows) * rows, 0.0);
    for (int i = 0; i < rows; ++i)
      for (int j = 0; j < rows; ++j)
        for (int k = 0; k < cols; ++k) AAt[i * rows + j] += A[k * rows + i] * A[k * rows + j];
    const std::vector<double> y = dense_solve(AAt, b, rows);
    double err = 0.0, scale = 0.0;
    for (int k = 0; k < cols; ++k) {
      double ref = 0.0;
      for (int i = 0; i < rows; ++i) ref += A[k * rows + i] * y[i];
      err = std::fmax(err, std::fabs(x[k] - ref));
      scale = std::fmax(scale, std::fabs(ref));
    }
    check(err <= 1e-9 * (1.0 + scale), "minimum-norm solution matches A^T (A A^T)^-1 b");
  }
  // Rank-deficient but consistent: b in the span of two repeated columns.
  std::vector<double> A = {1, 2, 3, 1, 2, 3, 0, 1, 0};   // 3 x 3 column-major, rank 2
  std::vector<double> b = {1, 3, 3}, x;
  const int rank = pgc::min_norm_solve(3, 3, A, b, &x);
  check(rank == 2, "rank 2 detected");
  for (int i = 0; i < 3; ++i) {
    double acc = 0.0;
    for (int k = 0; k < 3; ++k) acc += A[k * 3 + i] * x[k];
    check(std::fabs(acc - b[i]) <= 1e-12, "rank-deficient system solved");
  }
  check(std::fabs(x[0] - x[1]) <= 1e-12, "minimum norm splits the repeated column evenly");
}

void codes_and_decode() {
  const int shapes[][2] = {{4, 2}, {8, 3}, {12, 6}, {16, 4}, {64, 4}, {5, 1}};
  for (auto& nc : shapes) {
    const int n = nc[0], c = nc[1], s = c - 1;
    std::vector<double> B;
    std::string err;
    const std::vector<double> H = pgc::null_space_generator(3, s, n);
    check(H.size() == static_cast<size_t>(s) * n, "H is s x n");
    check(pgc::cyclic_encoding_matrix(n, c, H, &B, &err), "cyclic code builds: " + err);
    if (B.size() != static_cast<size_t>(n) * n) continue;
    for (int j = 0; j < n; ++j) {
      check(B[j * n + j] == 1.0, "B[j][j] = 1");
      for (int k = 0; k < n; ++k) {
        const bool in_support = ((k - j) % n + n) % n < c;
        if (!in_support) check(B[j * n + k] == 0.0, "row support is {j..j+c-1} mod n");
      }
      for (int r = 0; r < s; ++r) {
        double acc = 0.0;
        for (int k = 0; k < n; ++k) acc += H[r * n + k] * B[j * n + k];
        check(std::fabs(acc) <= 1e-9, "rows of B lie in the null space of H");
      }
    }
    Lcg g{static_cast<uint64_t>(n * 131 + c)};
    std::vector<uint8_t> mask(n);
    for (int trial = 0; trial < 50; ++trial) {
      std::fill(mask.begin(), mask.end(), uint8_t{0});
      const int count = static_cast<int>(g.uniform() * (s + 1));
      for (int x = 0; x < count; ++x) mask[static_cast<int>(g.uniform() * n)] = 1;
      for (int scheme : {pgc::kFR, pgc::kCR, pgc::kCRReal}) {
        if (scheme == pgc::kFR && n % c != 0) continue;
        pgc::Decode dec;
        const pgc::DecodeStatus st = pgc::decode_coefficients(scheme, n, c, B, mask.data(), &dec, &err);
        if (scheme == pgc::kFR) {
          // A group may lose every member only if c <= count; then the decode must say so.
          std::vector<int> alive(n / c, 0);
          for (int i = 0; i < n; ++i) alive[i / c] += !mask[i];
          bool all_groups = true;
          for (int a : alive) all_groups = all_groups && a > 0;
          check((st == pgc::kDecodeOk) == all_groups, "FR decodes exactly when every group survives");
          if (st != pgc::kDecodeOk) continue;
          std::vector<int> ones(n / c, 0);
          for (size_t m = 0; m < dec.survivors.size(); ++m) ones[dec.survivors[m] / c] += dec.d[m] == 1.0;
          for (int o : ones) check(o == 1, "one representative per FR group");
          continue;
        }
        check(st == pgc::kDecodeOk, "at most s stragglers decode");
        if (st != pgc::kDecodeOk) continue;
        if (scheme == pgc::kCR) {
          check(dec.scale == 1.0 / (static_cast<double>(dec.survivors.size()) * c), "CR scale 1/(|J| c)");
          continue;
        }
        for (int k = 0; k < n; ++k) {
          double acc = 0.0;
          for (size_t m = 0; m < dec.survivors.size(); ++m) acc += dec.d[m] * B[dec.survivors[m] * n + k];
          check(std::fabs(acc - 1.0) <= 1e-9, "real code recovers the sum of every partition");
        }
      }
    }
    // More than s stragglers.
    std::fill(mask.begin(), mask.end(), uint8_t{0});
    for (int i = 0; i <= s && i < n; ++i) mask[i] = 1;
    pgc::Decode dec;
    if (s + 1 < n || c == 1)
      check(pgc::decode_coefficients(pgc::kCR, n, c, B, mask.data(), &dec, &err) == pgc::kDecodeStragglers,
            "more than s stragglers rejected");
  }
  // A real-valued code that cannot decode: an all-zero matrix.
  const int n = 6, c = 3;
  std::vector<double> zero(static_cast<size_t>(n) * n, 0.0);
  std::vector<uint8_t> none(n, 0);
  pgc::Decode dec;
  std::string err;
  check(pgc::decode_coefficients(pgc::kCRReal, n, c, zero, none.data(), &dec, &err) == pgc::kDecodeSingular,
        "an undecodable real code is reported as singular");
  // IS-SGD: any number of stragglers below n; all of them is an error.
  std::vector<uint8_t> most(n, 1);
  most[4] = 0;
  check(pgc::decode_coefficients(pgc::kISSGD, n, 1, zero, most.data(), &dec, &err) == pgc::kDecodeOk &&
            dec.scale == 1.0,
        "IS-SGD averages the one survivor");
  std::vector<uint8_t> all(n, 1);
  check(pgc::decode_coefficients(pgc::kISSGD, n, 1, zero, all.data(), &dec, &err) == pgc::kDecodeStragglers,
        "IS-SGD with no survivor rejected");
}

}  // namespace

int main() {
  placements();
  masks();
  delays();
  solver();
  codes_and_decode();
  if (failures) {
    std::fprintf(stderr, "%d checks failed\n", failures);
    return 1;
  }
  std::printf("host tables: all checks passed\n");
  return 0;
}
