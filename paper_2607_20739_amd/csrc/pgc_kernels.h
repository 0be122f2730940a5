// Launchers of the PGC step's device kernels (gfx950).  Internal to the library.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "pgc.h"

namespace pgc {

// Per-partition gradient of a linear model (Sec. III with a mean over each
// partition's rows): for each evaluated partition k = e * part_stride +
// part_offset, e < n_eval, block b of that partition sums
//   slope(x_r . w, y_r) * x_r
// over its rows r and writes the fp32 sum to partials[(e * blocks_per_part + b) * d].
struct LinearGradArgs {
  const float* X;          // N x d row-major
  const float* y;          // N
  const float* w;          // d
  float* partials;         // n_eval * blocks_per_part * d
  int64_t m;               // rows per partition
  int64_t rows_per_block;  // contiguous rows handled by one block
  int32_t d;
  int32_t blocks_per_part;
  int32_t n_eval;
  int32_t part_stride;
  int32_t part_offset;
  int32_t model;           // PGC_LOGISTIC or PGC_LSQ
};

// Launch shape the gradient kernel uses for d (the caller sizes partials with it).
struct LinearGradShape {
  int threads;       // threads per block
  int vec_width;     // 4 (float4 loads) or 1
  bool supported;
};
LinearGradShape linear_grad_shape(int d, bool aligned16);

hipError_t launch_linear_gradient(const LinearGradArgs& a, bool aligned16, hipStream_t s);

// ring[(plane_first + p) * n + k][:] = (sum_b partials[e][b][:]) / m for each
// evaluated e (partition k = e * part_stride + part_offset) and p < plane_count.
// Sums run in fp64 in block order.
struct ReduceArgs {
  const float* partials;
  float* ring;             // planes x n x q
  int64_t q;
  double inv_m;
  int32_t n;
  int32_t n_eval;
  int32_t blocks_per_part;
  int32_t part_stride;
  int32_t part_offset;
  int32_t plane_first;
  int32_t plane_count;
};
hipError_t launch_reduce(const ReduceArgs& a, hipStream_t s);

// Encode, masked decode and update, column by column:
//   coded_j = sum_o coef(j, o) * ring[slot(j, o)]          (Sec. IV-A, V-A, V-B)
//   ghat    = sum_j a_j * coded_j  over j with a_j != 0    (stragglers skipped)
//   w      <- w - lr * ghat
// FR (fr = 1): j is a group, slot(j, o) = plane 0, partition j*c + o.
// CR: j is a worker, slot(j, o) = plane o, partition (j + o) mod n.
// coef == nullptr means unit coefficients; else coef[j * c + o] (fp64).
struct CodeArgs {
  const float* ring;
  float* coded;            // n_coded x q
  float* decoded;          // q
  float* w;                // q
  const double* coef;      // n_coded x c, or nullptr
  int64_t q;
  double lr;
  int32_t n;
  int32_t c;
  int32_t n_coded;
  int32_t fr;
  double a[PGC_MAX_N];     // decode weight per coded index (already scaled)
};
hipError_t launch_code(const CodeArgs& a, hipStream_t s);

}  // namespace pgc
