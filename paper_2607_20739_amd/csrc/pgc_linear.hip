// Device kernels of the PGC step for gfx950 (CDNA4, wave64).
//
// Gradient of the linear models (Sec. III; per-partition mean, Sec. IV-A /
// V-B evaluate one partition per worker per step).  Every evaluated row is
// read from HBM exactly once:
//   * the lanes of a "row group" (WAVES waves) own fixed column chunks of
//     VW floats (float4 when d % 4 == 0), VEC chunks per lane, so w and the
//     gradient accumulators stay in registers for the whole block;
//   * ROWS rows are loaded per iteration (all loads issued before use),
//     their dot products reduced by a wave butterfly and, when a row spans
//     several waves, through a double-buffered LDS exchange (one barrier per
//     ROWS rows);
//   * the loss slope scales the row still held in registers (axpy);
//   * GROUPS row groups share a block and fold their accumulators through
//     LDS in a fixed order, so one fp32 partial per block leaves the kernel.
// All reductions have a fixed order: results are bitwise reproducible.
#include <hip/hip_runtime.h>

#include "pgc_kernels.h"

namespace pgc {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));

template <int VW> struct VecOf;
template <> struct VecOf<4> { using T = f4; };
template <> struct VecOf<1> { using T = float; };

__device__ __forceinline__ float hsum(f4 v) { return (v.x + v.y) + (v.z + v.w); }
__device__ __forceinline__ float hsum(float v) { return v; }

template <int VW>
__device__ __forceinline__ typename VecOf<VW>::T stream_load(const float* p) {
  // X is streamed once per step: non-temporal loads keep it from evicting
  // the small, reused vectors (w, partials) from the caches.
  return __builtin_nontemporal_load(reinterpret_cast<const typename VecOf<VW>::T*>(p));
}

template <int VW>
__device__ __forceinline__ typename VecOf<VW>::T plain_load(const float* p) {
  return *reinterpret_cast<const typename VecOf<VW>::T*>(p);
}

template <int VW>
__device__ __forceinline__ void plain_store(float* p, typename VecOf<VW>::T v) {
  *reinterpret_cast<typename VecOf<VW>::T*>(p) = v;
}

// Butterfly sum over the 64 lanes of a wave.  Partners add the same two
// values (commuted), so every lane ends with bitwise the same total.
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

template <int MODEL>
__device__ __forceinline__ float loss_slope(float z, float y) {
  if constexpr (MODEL == PGC_LOGISTIC) {
    return 1.0f / (1.0f + expf(-z)) - y;   // d/dz [log(1 + e^z) - y z]
  } else {
    return z - y;                          // d/dz [(z - y)^2 / 2]
  }
}

template <int MODEL, int VW, int WAVES, int VEC, int GROUPS, int ROWS>
__global__ __launch_bounds__(64 * WAVES * GROUPS)
void linear_gradient_kernel(LinearGradArgs a) {
  using V = typename VecOf<VW>::T;
  constexpr int kRowLanes = 64 * WAVES;
  constexpr int kSpan = kRowLanes * VEC * VW;   // columns a row group covers
  const int lane = threadIdx.x % kRowLanes;
  const int group = threadIdx.x / kRowLanes;
  const int wave = lane / 64;

  const int e = blockIdx.y;
  const int64_t k = static_cast<int64_t>(e) * a.part_stride + a.part_offset;
  const int64_t part_end = (k + 1) * a.m;
  const int64_t row_begin = k * a.m + static_cast<int64_t>(blockIdx.x) * a.rows_per_block;
  const int64_t row_end = min(row_begin + a.rows_per_block, part_end);
  const int d = a.d;

  V wv[VEC], acc[VEC];
  bool own[VEC];
#pragma unroll
  for (int v = 0; v < VEC; ++v) {
    const int col = (v * kRowLanes + lane) * VW;
    own[v] = col < d;
    wv[v] = own[v] ? plain_load<VW>(a.w + col) : V{};
    acc[v] = V{};
  }

  __shared__ float dots[2][GROUPS][ROWS][WAVES];
  int buf = 0;
  for (int64_t base = row_begin; base < row_end; base += GROUPS * ROWS) {
    const int64_t r0 = base + group * ROWS;
    V x[ROWS][VEC];
#pragma unroll
    for (int r = 0; r < ROWS; ++r) {
      const bool in = r0 + r < row_end;
      const float* row = a.X + (r0 + r) * d;
#pragma unroll
      for (int v = 0; v < VEC; ++v)
        x[r][v] = (in && own[v]) ? stream_load<VW>(row + (v * kRowLanes + lane) * VW) : V{};
    }
    float dot[ROWS];
#pragma unroll
    for (int r = 0; r < ROWS; ++r) {
      V p = x[r][0] * wv[0];
#pragma unroll
      for (int v = 1; v < VEC; ++v) p += x[r][v] * wv[v];
      dot[r] = wave_sum(hsum(p));
    }
    if constexpr (WAVES > 1) {
      if (lane % 64 == 0) {
#pragma unroll
        for (int r = 0; r < ROWS; ++r) dots[buf][group][r][wave] = dot[r];
      }
      __syncthreads();
#pragma unroll
      for (int r = 0; r < ROWS; ++r) {
        float s = dots[buf][group][r][0];
#pragma unroll
        for (int q = 1; q < WAVES; ++q) s += dots[buf][group][r][q];
        dot[r] = s;
      }
      buf ^= 1;
    }
#pragma unroll
    for (int r = 0; r < ROWS; ++r) {
      const int64_t row = r0 + r;
      const float slope = row < row_end ? loss_slope<MODEL>(dot[r], a.y[row]) : 0.0f;
#pragma unroll
      for (int v = 0; v < VEC; ++v) acc[v] += slope * x[r][v];
    }
  }

  float* out = a.partials +
               (static_cast<int64_t>(e) * a.blocks_per_part + blockIdx.x) * static_cast<int64_t>(d);
  if constexpr (GROUPS > 1) {
    __shared__ V fold[GROUPS - 1][VEC][kRowLanes];
    if (group > 0) {
#pragma unroll
      for (int v = 0; v < VEC; ++v) fold[group - 1][v][lane] = acc[v];
    }
    __syncthreads();
    if (group == 0) {
#pragma unroll
      for (int v = 0; v < VEC; ++v) {
        V s = acc[v];
#pragma unroll
        for (int g = 0; g < GROUPS - 1; ++g) s += fold[g][v][lane];
        if (own[v]) plain_store<VW>(out + (v * kRowLanes + lane) * VW, s);
      }
    }
  } else {
#pragma unroll
    for (int v = 0; v < VEC; ++v)
      if (own[v]) plain_store<VW>(out + (v * kRowLanes + lane) * VW, acc[v]);
  }
  static_assert(kSpan > 0, "empty row span");
}

// Launch shapes: row-group waves, chunks per lane, row groups per block and
// rows per iteration, chosen from the number of column chunks.  Each entry
// keeps the x tile at <= 64 VGPRs per lane; 16-wave blocks are limited to
// 128 VGPRs per lane and take fewer rows per iteration.
struct Shape { int max_chunks, waves, vec, groups, rows; };
constexpr Shape kShapes4[] = {
    {64, 1, 1, 4, 8},  {128, 1, 2, 4, 8}, {256, 1, 4, 4, 4},  {512, 2, 4, 2, 4},
    {1024, 2, 8, 2, 2}, {2048, 8, 4, 1, 4}, {4096, 8, 8, 1, 2}, {8192, 16, 8, 1, 1}};
constexpr Shape kShapes1[] = {
    {64, 1, 1, 4, 8},  {128, 1, 2, 4, 8}, {256, 1, 4, 4, 8},  {512, 2, 4, 2, 8},
    {1024, 4, 4, 1, 8}, {2048, 4, 8, 1, 4}, {4096, 8, 8, 1, 4}, {8192, 16, 8, 1, 1}};
constexpr int kNumShapes = 8;
// Blocks per launch that the grid aims for, by the same feature-count classes
// as the shapes (d <= 256, 512, 1024, 2048, 4096, 8192, 16384, 32768).  The
// float4 shapes and these targets were chosen by timing on MI355X (d = 1024,
// 4096 and 8192 reach 84-91% of the 8 TB/s HBM peak).
constexpr int kTargetBlocks[kNumShapes] = {1024, 1024, 512, 1024, 512, 1024, 1024, 1024};

using GradKernel = void (*)(LinearGradArgs);

template <int MODEL, int VW, int I>
constexpr GradKernel pick() {
  constexpr Shape s = VW == 4 ? kShapes4[I] : kShapes1[I];
  return linear_gradient_kernel<MODEL, VW, s.waves, s.vec, s.groups, s.rows>;
}

template <int MODEL, int VW>
GradKernel kernel_for(int index) {
  switch (index) {
    case 0: return pick<MODEL, VW, 0>();
    case 1: return pick<MODEL, VW, 1>();
    case 2: return pick<MODEL, VW, 2>();
    case 3: return pick<MODEL, VW, 3>();
    case 4: return pick<MODEL, VW, 4>();
    case 5: return pick<MODEL, VW, 5>();
    case 6: return pick<MODEL, VW, 6>();
    case 7: return pick<MODEL, VW, 7>();
  }
  return nullptr;
}

int shape_index(int d, int vw) {
  const Shape* table = vw == 4 ? kShapes4 : kShapes1;
  const int chunks = d / vw;
  for (int i = 0; i < kNumShapes; ++i)
    if (chunks <= table[i].max_chunks) return i;
  return -1;
}

}  // namespace

int linear_grad_target_blocks(int d) {
  const int i = shape_index(d % 4 == 0 ? d : (d + 3) / 4 * 4, 4);
  return kTargetBlocks[i < 0 ? kNumShapes - 1 : i];
}

LinearGradShape linear_grad_shape(int d, bool aligned16) {
  const int vw = (aligned16 && d % 4 == 0) ? 4 : 1;
  const int i = shape_index(d, vw);
  if (i < 0) return {0, vw, false};
  const Shape& s = vw == 4 ? kShapes4[i] : kShapes1[i];
  return {64 * s.waves * s.groups, vw, true};
}

hipError_t launch_linear_gradient(const LinearGradArgs& a, bool aligned16, hipStream_t stream) {
  const LinearGradShape shape = linear_grad_shape(a.d, aligned16);
  if (!shape.supported) return hipErrorInvalidValue;
  const int i = shape_index(a.d, shape.vec_width);
  GradKernel k = nullptr;
  if (a.model == PGC_LOGISTIC)
    k = shape.vec_width == 4 ? kernel_for<PGC_LOGISTIC, 4>(i) : kernel_for<PGC_LOGISTIC, 1>(i);
  else if (a.model == PGC_LSQ)
    k = shape.vec_width == 4 ? kernel_for<PGC_LSQ, 4>(i) : kernel_for<PGC_LSQ, 1>(i);
  if (k == nullptr) return hipErrorInvalidValue;
  dim3 grid(a.blocks_per_part, a.n_eval);
  hipLaunchKernelGGL(k, grid, dim3(shape.threads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace pgc
