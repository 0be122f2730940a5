// Host-side tables of pipelined gradient coding: placement, schedule,
// straggler draws, the real-valued cyclic code and decode coefficients.
// Pure C++ (no HIP), so it runs and is tested on any host.
#pragma once

#include <cstdint>
#include <string>
#include <vector>

namespace pgc {

enum Scheme { kFR = 0, kCR = 1, kCRReal = 2, kISSGD = 3 };

// Partition held by worker i in slot l (Sec. III).
//   FR: (i / c) * c + l          CR (and IS-SGD, c = 1): (i + l) mod n
int held_partition(int scheme, int n, int c, int i, int l);

// Slot every worker evaluates at pipelined step t >= 1 (Sec. IV-A, Sec. V-B).
inline int evaluated_slot(int64_t t, int c) { return static_cast<int>((t - 1) % c); }

// SplitMix64 (Steele, Lea and Flood, OOPSLA 2014), counter form: output
// `index` of the stream seeded with `seed` is mix64(seed + (index + 1) * gamma).
uint64_t splitmix64(uint64_t seed, uint64_t index);

// j-th draw of step t: stream output t * 2^32 + j.
inline uint64_t step_draw(uint64_t seed, int64_t t, uint64_t j) {
  return splitmix64(seed, (static_cast<uint64_t>(t) << 32) + j);
}

// Straggler mask of step t (1 = straggles).  Policies: exactly `cap`;
// a count uniform in {0..cap}; independent Bernoulli(p) per worker keeping at
// most `cap` (partial Fisher-Yates over the straggler list); the `cap` workers
// with the largest uniform delay draws (the slowest under i.i.d. exponential
// delays, lower index first on ties).
bool make_mask(uint64_t seed, int64_t t, int policy, int n, int cap, double p,
               uint8_t* out);

// One step of the simulated cluster of Sec. VI-B: worker i finishes after
// compute_seconds + delay_i, delay_i = -mean_delay * ln(1 - u_i) with u_i the
// draw i of step t; the master proceeds at the (n - s)-th finish.  Writes the
// mask of the s workers it did not wait for (as the slowest-draws policy), the
// delays (optional) and the step's duration.
bool delay_step(uint64_t seed, int64_t t, int n, int s, double mean_delay, double compute_seconds,
                uint8_t* mask, double* delays, double* step_seconds);

// The s x n matrix H (row-major) whose null space holds the real-valued code:
// uniform entries in [-1, 1) for columns < n-1, last column = minus the row
// sum accumulated left to right, so H * 1 = 0.
std::vector<double> null_space_generator(uint64_t seed, int s, int n);

// Real-valued cyclic-repetition matrix B (n x n, row-major): row j supported on
// {j..j+c-1} mod n, B[j][j] = 1, and H B[j]^T = 0.  Any n - s rows then span a
// space that contains the all-ones vector (the decodability of Sec. V-A).
// Returns false if a row's s x s system is singular.
bool cyclic_encoding_matrix(int n, int c, const std::vector<double>& H,
                            std::vector<double>* B, std::string* err);

struct Decode {
  std::vector<int32_t> survivors;  // J, ascending
  std::vector<double> d;           // unscaled weight per survivor (same order)
  double scale = 0.0;
};

enum DecodeStatus { kDecodeOk = 0, kDecodeStragglers = 1, kDecodeSingular = 2 };

// Decode coefficients for a straggler mask (Sec. IV-A, Sec. V-A, Sec. V-B,
// Sec. VI-A):
//   FR:      1 for the lowest-index survivor of each group; scale 1/n.
//   CR:      1 for every survivor; scale 1/(|J| c).
//   CR_REAL: minimum-norm d with B_J^T d = 1, residual <= 1e-9; scale 1/n.
//   IS_SGD:  1 for every survivor (any number of stragglers below n); scale 1/|J|.
DecodeStatus decode_coefficients(int scheme, int n, int c, const std::vector<double>& B,
                                 const uint8_t* mask, Decode* out, std::string* err);

// Minimum-norm solution of the consistent system A x = b (A: rows x cols,
// column-major) by Householder QR with column pivoting followed by an
// orthogonal reduction of the leading rank rows (a complete orthogonal
// decomposition).  Returns the numerical rank.
int min_norm_solve(int rows, int cols, const std::vector<double>& A_colmajor,
                   const std::vector<double>& b, std::vector<double>* x);

}  // namespace pgc
