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
// Blocks per launch the gradient grid aims for (depends on d only, so the grid,
// and with it every result, is independent of pointer alignment and device).
int linear_grad_target_blocks(int d);

hipError_t launch_linear_gradient(const LinearGradArgs& a, bool aligned16, hipStream_t s);

// Encode, masked decode and update, column by column:
//   coded_j = sum_o coef(j, o) * ring[slot(j, o)]          (Sec. IV-A, V-A, V-B)
//   ghat    = sum_j a_j * coded_j  over j with a_j != 0    (stragglers skipped)
//   w      <- w - lr * ghat
// FR (fr = 1): j is a group, slot(j, o) = plane 0, partition j*c + o.
// CR: j is a worker, slot(j, o) = plane o, partition (j + o) mod n.
// coef == nullptr means unit coefficients; else coef[j * c + o] (fp64).
struct CodeArgs {
  const float* ring;       // planes x n x ld  (ld >= q, a multiple of 256)
  float* coded;            // n_coded x ld
  float* decoded;          // q
  float* w;                // q
  const double* coef;      // n_coded x c, or nullptr
  int64_t q;
  int64_t ld;
  double lr;
  int32_t n;
  int32_t c;
  int32_t n_coded;
  int32_t fr;
  double a[PGC_MAX_N];     // decode weight per coded index (already scaled)
};
hipError_t launch_code(const CodeArgs& a, hipStream_t s);

// The linear models' block partials folded into the ring, then the code step,
// in one launch: for each evaluated e (partition k = e * part_stride +
// part_offset) and p < plane_count,
//   ring[(plane_first + p) * n + k][:] = inv_m * sum_b partials[e][b][:]
// (fp64, block order), then encode / decode / update of the same columns.
struct ReduceCodeArgs {
  CodeArgs code;
  float* ring;             // the ring code.ring reads, written here first
  const float* partials;   // n_eval x blocks_per_part x q
  double inv_m;
  int32_t n_eval;
  int32_t blocks_per_part;
  int32_t part_stride;
  int32_t part_offset;
  int32_t plane_first;
  int32_t plane_count;
};
hipError_t launch_reduce_code(const ReduceCodeArgs& a, hipStream_t s);

// ---------------------------------------------------------------------------
// Two-layer MLP (d_in -> hidden, ReLU -> classes, softmax cross-entropy), bf16
// operands with fp32 accumulation on MFMA.  Parameters w (fp32) are laid out
// W1[d_in][hidden], b1[hidden], W2[hidden][classes], b2[classes].
// Shape limits: d_in % 8 == 0, hidden % 256 == 0 and <= 1024, classes <= 16.
// ---------------------------------------------------------------------------

constexpr int kMlpMaxClasses = 16;
constexpr int kMlpMaxHidden = 1024;

// bf16 copies of the weights for the GEMMs: W1T[hidden][kpad] (kpad a multiple
// of 64; zero past d_in),
// W2T[16][hidden] and W2p[hidden][16] (zero past `classes`).
struct MlpCastArgs {
  const float* w;
  __bf16* W1T;
  __bf16* W2T;
  __bf16* W2p;
  int32_t d_in, kpad, hidden, classes;
};
hipError_t launch_mlp_cast(const MlpCastArgs& a, hipStream_t s);

// H layout, blocked by 16 rows x 128 hidden units in the order of the head's
// MFMA fragments: element (r, h) of evaluated partition e, with r = 16 rb + i
// and h = 128 hb + 32 s + 8 g + j, at
//   H[((((e * m_pad / 16 + rb) * hidden / 128 + hb) * 4 + s) * 64 + 16 g + i) * 8 + j].
// A (16-row, 128-unit) block is 4 KiB of contiguous memory, and for each s the
// 64 lanes of a head wave read 1 KiB of it in lane order.

// H(e; r, h) = bf16(relu(X[k*m + r] . W1[:, h] + b1[h])) for each evaluated
// partition k = e * part_stride + part_offset, e < n_eval, r < m, in the
// blocked layout above; rows m .. m_pad - 1 are written as zeros.
struct MlpForwardArgs {
  const __bf16* X;
  const __bf16* W1T;
  const float* b1;
  __bf16* H;
  int64_t m, m_pad;
  int32_t d_in, kpad, hidden, n_eval, part_stride, part_offset;
};
hipError_t launch_mlp_forward(const MlpForwardArgs& a, hipStream_t s);

// dZ1 layout, blocked by 16 rows: element (r, h) of evaluated partition e at
// dZ1[((e * m_pad / 16 + r / 16) * hidden + h) * 16 + r % 16], r < m_pad (a
// multiple of 64; zero for r >= m).  A 16-row tile is one contiguous run, and
// 8 consecutive rows of one hidden unit are 16 contiguous bytes.
__host__ __device__ inline int64_t mlp_dz1_index(int64_t m_pad, int32_t hidden, int32_t e, int64_t r, int32_t h) {
  return ((static_cast<int64_t>(e) * (m_pad / 16) + r / 16) * hidden + h) * 16 + r % 16;
}

// Per 16-row tile: logits, softmax, dZ2 = (p - onehot(y)) / m, dZ1 = (dZ2 W2^T)
// masked by H > 0, written to dZ1 in the blocked layout above.  Each block writes partial sums of dW2^T[16][hidden], db1[hidden]
// and db2[16] to partials[(e * blocks_per_part + b) * pstride].
struct MlpHeadArgs {
  const __bf16* H;
  const int32_t* y;
  const __bf16* W2T;
  const __bf16* W2p;
  const float* b2;
  __bf16* dZ1;
  float* partials;
  int64_t m, m_pad, rows_per_block;
  float inv_m;
  int32_t hidden, classes, blocks_per_part, n_eval, part_stride, part_offset, pstride;
};
int mlp_head_threads(int hidden);
hipError_t launch_mlp_head(const MlpHeadArgs& a, hipStream_t s);

// dW1[i][h] = sum_r X[k*m + r][i] dZ1(e; r, h), written into the ring slot of
// partition k: ring[((plane * n + k) * ld) + i * hidden + h].
struct MlpWgradArgs {
  const __bf16* X;
  const __bf16* dZ1;
  float* ring;
  int64_t m, m_pad, ld;
  int32_t d_in, hidden, n, plane, n_eval, part_stride, part_offset;
};
hipError_t launch_mlp_wgrad(const MlpWgradArgs& a, hipStream_t s);

// Fold the head partials of each evaluated partition (fp64, block order) into
// the b1, W2 and b2 parts of its ring slot.
struct MlpReduceArgs {
  const float* partials;
  float* ring;
  int64_t ld;
  int32_t d_in, hidden, classes, n, plane, n_eval, blocks_per_part, part_stride, part_offset,
      pstride;
};
hipError_t launch_mlp_reduce(const MlpReduceArgs& a, hipStream_t s);

// Header of a saved pipeline state: the first kStateHeaderBytes bytes of the
// caller's buffer (the rest of the struct's space is zero), followed by the
// ring.  Every field but t must match the loading context.
struct StateHeader {
  uint64_t magic;     // kStateMagic
  uint64_t version;   // kStateVersion
  int64_t t, N, q, ld;
  uint64_t code_seed;
  int32_t scheme, n, c, model, d_in, hidden, classes, planes;
};
constexpr uint64_t kStateMagic = 0x4554415453434750ull;   // the bytes "PGCSTATE"
constexpr uint64_t kStateVersion = 1;
constexpr size_t kStateHeaderBytes = 256;
static_assert(sizeof(StateHeader) <= kStateHeaderBytes && sizeof(StateHeader) % 8 == 0, "state header");
// Writes h (zero-padded to kStateHeaderBytes) to out, which is 8-byte aligned.
hipError_t launch_write_state_header(const StateHeader& h, void* out, hipStream_t s);

}  // namespace pgc
