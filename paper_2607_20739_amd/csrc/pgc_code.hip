// Post-gradient kernels of the PGC step for gfx950: the linear models' fused
// partial reduction + ring write + encode + masked decode + update, and the
// encode + masked decode + update alone (used after the MLP gradient).
// Sec. IV-A (FR encode / decode), Sec. V-A (real coefficients), Sec. V-B (CR).
#include <hip/hip_runtime.h>

#include "pgc_kernels.h"

namespace pgc {
namespace {

// Encode, masked decode and update of 256 columns by a 256-thread block: a
// thread owns 4 consecutive columns (16-byte ring loads; slots are padded to
// ld, a multiple of 256, so a block never leaves its slot), the four waves split
// the coded words (j = wave, wave + 4, ...), each word is summed in fp64, and
// the waves' decode partials are added in wave order.
constexpr int kCodeCols = 256;
typedef float f4v __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256)
void code_kernel(CodeArgs a) {
  __shared__ double part[4][kCodeCols];
  const int lane = threadIdx.x % 64, sub = threadIdx.x / 64;
  const int64_t col = static_cast<int64_t>(blockIdx.x) * kCodeCols + 4 * lane;
  double ghat[4] = {0.0, 0.0, 0.0, 0.0};
  for (int j = sub; j < a.n_coded; j += 4) {
    double word[4] = {0.0, 0.0, 0.0, 0.0};
    for (int o = 0; o < a.c; ++o) {
      const int64_t slot = a.fr ? static_cast<int64_t>(j) * a.c + o
                                : static_cast<int64_t>(o) * a.n + (j + o) % a.n;
      const f4v v = *reinterpret_cast<const f4v*>(a.ring + slot * a.ld + col);
      const double cf = a.coef ? a.coef[j * a.c + o] : 1.0;
#pragma unroll
      for (int i = 0; i < 4; ++i) word[i] += cf * static_cast<double>(v[i]);
    }
    f4v out;
#pragma unroll
    for (int i = 0; i < 4; ++i) out[i] = static_cast<float>(word[i]);
    *reinterpret_cast<f4v*>(a.coded + static_cast<int64_t>(j) * a.ld + col) = out;
    if (a.a[j] != 0.0) {
#pragma unroll
      for (int i = 0; i < 4; ++i) ghat[i] += a.a[j] * word[i];
    }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) part[sub][4 * lane + i] = ghat[i];
  __syncthreads();
  const int c = threadIdx.x;   // one column per thread for the result
  const int64_t gc = static_cast<int64_t>(blockIdx.x) * kCodeCols + c;
  if (gc < a.q) {
    const double g = ((part[0][c] + part[1][c]) + part[2][c]) + part[3][c];
    a.decoded[gc] = static_cast<float>(g);
    a.w[gc] = static_cast<float>(static_cast<double>(a.w[gc]) - a.lr * g);
  }
}

// Block b owns columns [16 b, 16 b + 16).  It first folds every evaluated
// partition's block partials for those columns into the ring (fp64, block
// order, one (partition, column) pair per thread), then -- after a barrier, so
// the fresh slots written by its own threads are visible -- encodes, decodes
// and updates the same columns with the 16 lanes of each column splitting the
// coded words.  No block depends on another.
constexpr int kFusedCols = 16;
constexpr int kFusedSubs = 256 / kFusedCols;

__global__ __launch_bounds__(256)
void reduce_code_kernel(ReduceCodeArgs a) {
  __shared__ double part[kFusedSubs][kFusedCols];
  const CodeArgs& ca = a.code;
  const int64_t col0 = static_cast<int64_t>(blockIdx.x) * kFusedCols;
  for (int pair = threadIdx.x; pair < a.n_eval * kFusedCols; pair += 256) {
    const int e = pair / kFusedCols;
    const int64_t col = col0 + pair % kFusedCols;
    if (col >= ca.q) continue;
    const float* p = a.partials + static_cast<int64_t>(e) * a.blocks_per_part * ca.q + col;
    // Loads go out 32 at a time (one memory latency per 32 partials); the
    // fp64 sum still runs in block order.
    double s = 0.0;
    int b = 0;
    for (; b + 32 <= a.blocks_per_part; b += 32) {
      float t[32];
#pragma unroll
      for (int i = 0; i < 32; ++i) t[i] = p[static_cast<int64_t>(b + i) * ca.q];
#pragma unroll
      for (int i = 0; i < 32; ++i) s += static_cast<double>(t[i]);
    }
    for (; b + 8 <= a.blocks_per_part; b += 8) {
      float t[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) t[i] = p[static_cast<int64_t>(b + i) * ca.q];
#pragma unroll
      for (int i = 0; i < 8; ++i) s += static_cast<double>(t[i]);
    }
    for (; b < a.blocks_per_part; ++b) s += static_cast<double>(p[static_cast<int64_t>(b) * ca.q]);
    const float g = static_cast<float>(s * a.inv_m);
    const int64_t k = static_cast<int64_t>(e) * a.part_stride + a.part_offset;
    for (int pl = 0; pl < a.plane_count; ++pl)
      a.ring[((a.plane_first + pl) * static_cast<int64_t>(ca.n) + k) * ca.ld + col] = g;
  }
  __syncthreads();

  const int lane = threadIdx.x % kFusedCols, sub = threadIdx.x / kFusedCols;
  const int64_t col = col0 + lane;
  const bool live = col < ca.q;
  double ghat = 0.0;
  if (live) {
    for (int j = sub; j < ca.n_coded; j += kFusedSubs) {
      double word = 0.0;
      for (int o = 0; o < ca.c; ++o) {
        const int64_t slot = ca.fr ? static_cast<int64_t>(j) * ca.c + o
                                   : static_cast<int64_t>(o) * ca.n + (j + o) % ca.n;
        const double v = static_cast<double>(a.ring[slot * ca.ld + col]);
        word += ca.coef ? ca.coef[j * ca.c + o] * v : v;
      }
      ca.coded[static_cast<int64_t>(j) * ca.ld + col] = static_cast<float>(word);
      if (ca.a[j] != 0.0) ghat += ca.a[j] * word;
    }
  }
  part[sub][lane] = ghat;
  __syncthreads();
  if (sub == 0 && live) {
    double g = part[0][lane];
#pragma unroll
    for (int i = 1; i < kFusedSubs; ++i) g += part[i][lane];
    ca.decoded[col] = static_cast<float>(g);
    ca.w[col] = static_cast<float>(static_cast<double>(ca.w[col]) - ca.lr * g);
  }
}

}  // namespace

hipError_t launch_reduce_code(const ReduceCodeArgs& a, hipStream_t stream) {
  dim3 grid(static_cast<unsigned>((a.code.q + kFusedCols - 1) / kFusedCols));
  hipLaunchKernelGGL(reduce_code_kernel, grid, dim3(256), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_code(const CodeArgs& a, hipStream_t stream) {
  dim3 grid(static_cast<unsigned>((a.q + kCodeCols - 1) / kCodeCols));
  hipLaunchKernelGGL(code_kernel, grid, dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace pgc
