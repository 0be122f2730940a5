// Reductions over the 16-lane rows of a gfx950 wave64, built from DPP lane
// moves, which go register to register (no LDS permute round trip).  Every
// reduction has a fixed order, so results are bitwise reproducible.
#pragma once
#include <hip/hip_runtime.h>

namespace pgc {

// v from the lane that DPP control `ctrl` selects (all rows and banks on).
template <int ctrl>
__device__ __forceinline__ float dpp_move(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), ctrl, 0xF, 0xF, true));
}

// DPP controls of the 16-lane row reductions: swap neighbours, swap pairs,
// mirror each half row, mirror the row.  After the two quad steps each lane
// holds its quad's result; each mirror step combines a lane with one holding
// the other half's result, so every lane of the row ends with the same value.
constexpr int kDppSwap1 = 0xB1, kDppSwap2 = 0x4E, kDppHalfMirror = 0x141, kDppMirror = 0x140;

__device__ __forceinline__ float row16_max(float v) {
  v = fmaxf(v, dpp_move<kDppSwap1>(v));
  v = fmaxf(v, dpp_move<kDppSwap2>(v));
  v = fmaxf(v, dpp_move<kDppHalfMirror>(v));
  return fmaxf(v, dpp_move<kDppMirror>(v));
}

__device__ __forceinline__ float row16_sum(float v) {
  v += dpp_move<kDppSwap1>(v);
  v += dpp_move<kDppSwap2>(v);
  v += dpp_move<kDppHalfMirror>(v);
  return v + dpp_move<kDppMirror>(v);
}

}  // namespace pgc
