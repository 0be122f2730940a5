// Two-layer MLP gradient of the PGC step on gfx950: bf16 MFMA with fp32
// accumulation (the per-partition gradient of Sec. III for a network model;
// every worker evaluates one partition per step, Sec. IV-A / V-B).
//
// Per step, for the evaluated partitions:
//   cast     w (fp32) -> W1T, W2T, W2p (bf16 copies laid out for the MFMAs)
//   forward  H = relu(X W1 + b1)                       MFMA 16x16x32, tiles loaded
//            straight into swizzled LDS, XCD-aware tile order
//   head     logits = H W2 + b2, softmax, dZ2 = (p - onehot) / m,
//            dZ1 = (dZ2 W2^T) * [H > 0] (16-row blocked), and block
//            partials of dW2 = H^T dZ2, db1, db2         MFMA 16x16x32 / 16x16x16
//   wgrad    dW1 = X^T dZ1 straight into the ring slot  MFMA 16x16x32, both tiles
//            loaded straight into LDS, X fragments by transposing LDS reads
//   reduce   head partials -> b1, W2, b2 parts of the ring slot (fp64, fixed order)
//
// MFMA lane layouts (gfx950, wave64; l = lane, lr = l % 16, lg = l / 16):
//   16x16x32 bf16: A[lr][8 lg + j], B[8 lg + j][lr], j < 8;  D[4 lg + i][lr]
//   16x16x16 bf16: A[lr][4 lg + j], B[4 lg + j][lr], j < 4;  D[4 lg + i][lr]
#include <hip/hip_runtime.h>

#include <cmath>
#include <type_traits>

#include "pgc_kernels.h"
#include "pgc_lanes.h"

namespace pgc {
namespace {

typedef __bf16 bf16;
typedef bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f32x4 mfma_k32(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mfma_k16(bf16x4 a, bf16x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, b, c, 0, 0, 0);
}

template <class T>
__device__ __forceinline__ T load_vec(const bf16* p) { return *reinterpret_cast<const T*>(p); }

// ---------------------------------------------------------------------------
// cast
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(256)
void mlp_cast_w1_kernel(MlpCastArgs a) {
  __shared__ float tile[32][33];
  const int i0 = blockIdx.x * 32, h0 = blockIdx.y * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
  for (int j = ty; j < 32; j += 8) {
    const int i = i0 + j;
    tile[j][tx] = i < a.d_in ? a.w[static_cast<int64_t>(i) * a.hidden + h0 + tx] : 0.0f;
  }
  __syncthreads();
  for (int j = ty; j < 32; j += 8)
    a.W1T[static_cast<int64_t>(h0 + j) * a.kpad + i0 + tx] = static_cast<bf16>(tile[tx][j]);
}

__global__ __launch_bounds__(256)
void mlp_cast_w2_kernel(MlpCastArgs a) {
  const int idx = blockIdx.x * 256 + threadIdx.x;
  if (idx >= a.hidden * kMlpMaxClasses) return;
  const int h = idx / kMlpMaxClasses, c = idx % kMlpMaxClasses;
  const int64_t w2 = static_cast<int64_t>(a.d_in) * a.hidden + a.hidden;
  const float v = c < a.classes ? a.w[w2 + static_cast<int64_t>(h) * a.classes + c] : 0.0f;
  a.W2T[static_cast<int64_t>(c) * a.hidden + h] = static_cast<bf16>(v);
  a.W2p[idx] = static_cast<bf16>(v);
}

// ---------------------------------------------------------------------------
// forward: H = relu(X W1 + b1).  Block tile BM samples x 256 hidden, K step
// 64, 8 waves as WH (hidden) x WS (samples), one block per CU.  With BM = 384
// the waves are 2 x 4 of 128 hidden x 96 samples (192 fp32 accumulators per
// lane) and a K step's two tiles fill the 160 KiB of LDS in two buffers: per
// MFMA FLOP a quarter fewer fragment reads and a sixth fewer tile bytes than a
// 256 x 256 tile, and a third fewer blocks to start and drain.  Tiles travel
// from global memory straight into LDS (16 bytes per lane, no register
// staging), loaded one K step ahead: one barrier per K step.  In a tile row of
// 64 bf16 (eight 16-byte chunks) chunk ch of row r sits at slot
// ch ^ (r & 7) ^ ((r >> 3) & 1), so the 16 rows of a fragment read spread over
// the slots.  The MFMAs produce H^T (A = W1^T rows, B = X rows), which leaves four
// consecutive hidden units of one sample in each lane.  Block ids are mapped
// so that all hidden tiles of a row tile run on the same XCD (workgroups are
// dealt to the 8 XCDs round-robin) and share its L2.
// ---------------------------------------------------------------------------

constexpr int kFwBN = 256, kFwBK = 64, kFwStages = 2;
constexpr int kFwThreads = 512;
constexpr int kFwCpr = kFwBK / 8;                   // 16-byte chunks per tile row
constexpr int kFwLdsBytes = 160 * 1024;
constexpr int kXcds = 8;

// Wave grid (hidden x samples) and epilogue passes per block tile height.
// 256 x 256 tiles (4 x 2 waves of 64 x 128, one epilogue pass) measured 7%
// slower than 384 x 256 on the 784 -> 1024 workload, with bitwise the same H.
template <int BM> struct FwShape;
template <> struct FwShape<384> { static constexpr int WH = 2, WS = 4, PASSES = 2; };
constexpr int kFwBM = 384;   // samples per block tile

typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(1))) void global_void;

// 16 bytes from global memory to LDS: lane l of the wave writes lds_wave_base + 16 l.
__device__ __forceinline__ void load_lds16(const void* src, void* lds_wave_base) {
  __builtin_amdgcn_global_load_lds((global_void*)src, (lds_void*)lds_wave_base, 16, 0, 0);
}

// Swizzle of a tile row's 16-byte chunks: chunk ch of row r sits at slot
// ch ^ fw_swizzle(r).  It depends only on the row within its 16-row group, so a
// lane's fragment reads for successive 16-row groups are a constant stride
// apart, and rows r and r + 8 of a group land in different slots.
__device__ __forceinline__ int fw_swizzle(int row) { return (row & 7) ^ ((row >> 3) & 1); }

// 16 bytes from a wave-uniform base plus a per-lane byte offset to LDS.
__device__ __forceinline__ void load_lds16_at(const bf16* base, uint32_t offset_bytes, void* lds_wave_base) {
  load_lds16(reinterpret_cast<const char*>(base) + offset_bytes, lds_wave_base);
}

// Workgroup barrier that orders LDS only: the wave's own LDS reads and writes
// complete (lgkmcnt 0) before it, but outstanding global loads and stores do
// not have to, unlike the release fence of __syncthreads(), which would drain
// every prefetch.  Callers wait for the global loads they need with
// wait_vmcnt.  The empty asm statements keep the compiler from moving memory
// accesses across it.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xC07F);   // vmcnt 63 (no wait), expcnt 7, lgkmcnt 0
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// s_waitcnt with vmcnt = n (n < 16) and the other counters left alone.
template <int n>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(n >= 0 && n < 16, "vmcnt field");
  __builtin_amdgcn_s_waitcnt(0x0F70 | n);
}

template <int BM>
__global__ __launch_bounds__(kFwThreads, 1)
void mlp_forward_kernel(MlpForwardArgs a) {
  using S = FwShape<BM>;
  constexpr int kTH = kFwBN / S::WH, kTS = BM / S::WS;   // wave tile: hidden x samples
  constexpr int kNT = kTH / 16, kMT = kTS / 16;
  constexpr int kXTile = BM * kFwBK, kWTile = kFwBN * kFwBK;   // bf16 per operand tile
  constexpr int kStage = kXTile + kWTile;
  constexpr int kXRounds = kXTile / 8 / kFwThreads, kWRounds = kWTile / 8 / kFwThreads;
  constexpr int kPassRows = BM / S::PASSES;   // output rows staged through LDS at a time
  static_assert(S::WH * S::WS * 64 == kFwThreads && kTH % 16 == 0 && kTS % 16 == 0, "wave grid");
  static_assert(kFwStages == 2, "one K step in flight: every load is waited for at the next barrier");
  static_assert(kFwStages * kStage * 2 <= kFwLdsBytes, "LDS");
  static_assert(kPassRows * kFwBN * 2 <= kFwStages * kStage * 2 && kPassRows % 16 == 0, "output staging");
  static_assert(S::WS % S::PASSES == 0, "each pass stages whole sample groups");
  __shared__ __attribute__((aligned(16))) bf16 smem[kFwStages * kStage];   // per buffer: X tile, W1^T tile
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int wh = wave % S::WH, ws = wave / S::WH;

  const int htiles = a.hidden / kFwBN;
  const int64_t tiles_per_part = (a.m + BM - 1) / BM;
  const int64_t rtiles = tiles_per_part * a.n_eval;
  const int64_t id = blockIdx.x;
  const int64_t rest = id / kXcds;
  const int ht = static_cast<int>(rest % htiles);
  const int64_t rt = (rest / htiles) * kXcds + id % kXcds;
  if (rt >= rtiles) return;
  const int e = static_cast<int>(rt / tiles_per_part);
  const int64_t r0 = (rt % tiles_per_part) * BM;
  const int h0 = ht * kFwBN;
  const int64_t part = static_cast<int64_t>(e) * a.part_stride + a.part_offset;
  const bf16* Xp = a.X + part * a.m * a.d_in;
  const int ksteps = a.kpad / kFwBK;
  const int dchunks = a.d_in / 8;

  // Chunk c = u * 512 + tid of a tile is row c / 8 = u * 64 + tid / 8 at slot
  // c % 8 = tid % 8, which holds logical chunk (tid % 8) ^ swizzle(row); the
  // swizzle does not change when 64 is added to the row, so the chunk is the
  // same in every round.  Addresses are 32-bit byte offsets from the tile's
  // first row (wave-uniform bases).  Rows past the partition read its last
  // row, chunks past d_in read the row's first chunk: both are finite values
  // that meet zero weights or land in rows that are never stored.
  const int chunk = (tid & 7) ^ fw_swizzle(tid >> 3);
  const bf16* Xt = Xp + r0 * a.d_in;
  const int last_row = static_cast<int>(min<int64_t>(BM, a.m - r0)) - 1;
  uint32_t xrow[kXRounds];
#pragma unroll
  for (int u = 0; u < kXRounds; ++u)
    xrow[u] = static_cast<uint32_t>(min(u * 64 + (tid >> 3), last_row)) * static_cast<uint32_t>(a.d_in) * 2u;
  const bf16* Wt = a.W1T + static_cast<int64_t>(h0) * a.kpad;
  const uint32_t wrow = static_cast<uint32_t>(tid >> 3) * static_cast<uint32_t>(a.kpad) * 2u;
  // The last K step covers columns kpad - 64 .. kpad - 1.  When its second
  // half lies wholly past d_in (784 features: 800 .. 831), that half is
  // neither loaded nor multiplied: its products with the zero W1^T columns
  // are exact zeros.
  const bool half_last = a.kpad - 32 >= a.d_in;
  auto issue = [&](int ks, int buf, bool skip_upper) {
    const int kc = ks * kFwCpr + chunk;
    if (skip_upper && chunk >= kFwCpr / 2) return;
    const uint32_t xk = static_cast<uint32_t>(kc < dchunks ? kc : 0) * 16u;
#pragma unroll
    for (int u = 0; u < kXRounds; ++u)
      load_lds16_at(Xt, xrow[u] + xk, &smem[buf * kStage + (u * kFwThreads + wave * 64) * 8]);
#pragma unroll
    for (int u = 0; u < kWRounds; ++u)
      load_lds16_at(Wt + static_cast<int64_t>(u * 64) * a.kpad, wrow + static_cast<uint32_t>(kc) * 16u,
                    &smem[buf * kStage + kXTile + (u * kFwThreads + wave * 64) * 8]);
  };

  f32x4 acc[kNT][kMT];   // [hidden tile][sample tile], D = H^T
#pragma unroll
  for (int nt = 0; nt < kNT; ++nt)
#pragma unroll
    for (int mt = 0; mt < kMT; ++mt) acc[nt][mt] = f32x4{};
  // A lane reads rows ws * kTS + mt * 16 + lr of the X tile and
  // wh * kTH + nt * 16 + lr of the W1^T tile, chunk kk * 4 + lg of each.
  const int lane_swz = fw_swizzle(lr);
  // MFMAs over 32-column halves [K0, K1) of the K step held in buffer buf.
  auto compute = [&](int buf, auto k0, auto k1) {
    const bf16* Xs = smem + buf * kStage + (ws * kTS + lr) * kFwBK;
    const bf16* Ws = smem + buf * kStage + kXTile + (wh * kTH + lr) * kFwBK;
#pragma unroll
    for (int kk = decltype(k0)::value; kk < decltype(k1)::value; ++kk) {
      const int slot = ((kk * 4 + lg) ^ lane_swz) << 3;
      bf16x8 xf[kMT];
#pragma unroll
      for (int mt = 0; mt < kMT; ++mt) xf[mt] = *reinterpret_cast<const bf16x8*>(Xs + mt * 16 * kFwBK + slot);
#pragma unroll
      for (int nt = 0; nt < kNT; ++nt) {
        const bf16x8 wf = *reinterpret_cast<const bf16x8*>(Ws + nt * 16 * kFwBK + slot);
#pragma unroll
        for (int mt = 0; mt < kMT; ++mt) acc[nt][mt] = mfma_k32(wf, xf[mt], acc[nt][mt]);
      }
    }
  };

  using H0 = std::integral_constant<int, 0>;
  using H1 = std::integral_constant<int, 1>;
  using H2 = std::integral_constant<int, 2>;
  static_assert(kFwBK == 64, "two 32-column halves per K step");
  issue(0, 0, ksteps == 1 && half_last);
  for (int ks = 0; ks + 1 < ksteps; ++ks) {
    // This wave's loads of step ks have landed; after the barrier every
    // wave's have, and every wave is done reading buffer (ks + 1) % 2, which
    // the loads of step ks + 1 then overwrite.
    wait_vmcnt<0>();
    lds_barrier();
    issue(ks + 1, (ks + 1) % kFwStages, ks + 2 == ksteps && half_last);
    compute(ks % kFwStages, H0{}, H2{});
  }
  wait_vmcnt<0>();
  lds_barrier();
  compute((ksteps - 1) % kFwStages, H0{}, H1{});
  if (!half_last) compute((ksteps - 1) % kFwStages, H1{}, H2{});

  // Epilogue: bias and ReLU, then the tile goes through LDS, kPassRows rows at
  // a time (row r's 16-byte chunk cc at slot cc ^ (r & 31)), so that H leaves
  // in its blocked layout, 1 KiB of contiguous memory per store instruction.
  lds_barrier();   // every wave is done reading the operand buffers
  bf16* out = smem;
  const int64_t hblocks = a.hidden / 128;
  bf16* Hb = a.H + ((static_cast<int64_t>(e) * (a.m_pad / 16) + r0 / 16) * hblocks + h0 / 128) * 2048;
  constexpr int kGroupsPerPass = S::WS / S::PASSES;
#pragma unroll
  for (int p = 0; p < S::PASSES; ++p) {
    if (ws / kGroupsPerPass == p) {
#pragma unroll
      for (int nt = 0; nt < kNT; ++nt) {
        const int hl = wh * kTH + nt * 16 + lg * 4;   // hidden column within the tile
        float bias[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) bias[i] = a.b1[h0 + hl + i];
#pragma unroll
        for (int mt = 0; mt < kMT; ++mt) {
          const int r = (ws % kGroupsPerPass) * kTS + mt * 16 + lr;   // row within the pass
          bf16x4 v;
#pragma unroll
          for (int i = 0; i < 4; ++i) v[i] = static_cast<bf16>(fmaxf(acc[nt][mt][i] + bias[i], 0.0f));
          *reinterpret_cast<bf16x4*>(&out[r * kFwBN + (((hl >> 3) ^ (r & 31)) << 3) + (hl & 4)]) = v;
        }
      }
    }
    lds_barrier();
    // The pass is kPassRows / 16 row blocks x 2 hidden blocks of 4 KiB; chunk
    // q of a block is fragment slice q / 64, lane q % 64 (row q % 16, 8-unit
    // group (q / 16) % 4).
#pragma unroll 4
    for (int it = 0; it < kPassRows * kFwBN / 8 / kFwThreads; ++it) {
      const int q = it * kFwThreads + tid;
      const int blk = q >> 8, rbl = blk >> 1, hbl = blk & 1, within = q & 255;
      const int r = rbl * 16 + (within & 15);
      const int cc = hbl * 16 + (within >> 6) * 4 + ((within >> 4) & 3);
      const int64_t row = r0 + p * kPassRows + r;
      if (row < a.m_pad) {
        const bf16x8 v = row < a.m ? *reinterpret_cast<const bf16x8*>(&out[r * kFwBN + ((cc ^ (r & 31)) << 3)])
                                   : bf16x8{};
        // H (2 GB per step) cannot stay in the caches until the head reads it:
        // streaming stores keep it from evicting the reused X and W1^T tiles.
        __builtin_nontemporal_store(
            v, reinterpret_cast<bf16x8*>(Hb + ((p * kPassRows / 16 + rbl) * hblocks + hbl) * 2048 + within * 8));
      }
    }
    if (p + 1 < S::PASSES) lds_barrier();   // the next pass overwrites the staging area
  }
}

// ---------------------------------------------------------------------------
// head: one wave per 128 hidden columns, 16-row tiles.  The wave's partial
// logits are summed across waves through LDS in wave order (one barrier per
// tile).  Each wave stages its 16 x 128 tile of H through its own LDS area,
// from which each lane reads the four rows of one hidden unit that
// serve as the ReLU mask and the dW2 operand.  dH comes out of the MFMA as
// four consecutive rows of one hidden unit per lane, which is dZ1's 16-row
// blocked layout: the tile's dZ1 leaves straight from registers, a contiguous
// 512-byte run per store.
// ---------------------------------------------------------------------------

constexpr int kHeadCols = 128;
constexpr int kHeadMaxWaves = kMlpMaxHidden / kHeadCols;
constexpr int kHtLd = kHeadCols + 16;  // H tile row stride (bf16): 288 bytes, so the four
                                       // 32-byte row pieces of a transposing read hit
                                       // distinct banks

typedef bf16 bf16x4t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) bf16x4t lds_bf16x4t;

__global__ __launch_bounds__(64 * kHeadMaxWaves)
void mlp_head_kernel(MlpHeadArgs a) {
  __shared__ float zpart[2][kHeadMaxWaves][16][16];
  __shared__ float dzt[kHeadMaxWaves][16][17];
  __shared__ bf16 Ht[kHeadMaxWaves][16][kHtLd];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int waves = a.hidden / kHeadCols;
  const int e = blockIdx.y;
  const int64_t part = static_cast<int64_t>(e) * a.part_stride + a.part_offset;
  const int hw0 = wave * kHeadCols;
  const int64_t hidden = a.hidden;
  // This wave's 4 KiB block of H for row block rb starts at Hw + rb * hblocks * 2048.
  const int64_t hblocks = hidden / 128;
  const bf16* Hw = a.H + (static_cast<int64_t>(e) * (a.m_pad / 16) * hblocks + wave) * 2048;
  const int32_t* yp = a.y + part * a.m;
  bf16* dz1 = a.dZ1 + mlp_dz1_index(a.m_pad, a.hidden, e, 0, 0);
  const int64_t rbeg = static_cast<int64_t>(blockIdx.x) * a.rows_per_block;
  const int64_t rend = min(rbeg + a.rows_per_block, a.m_pad);

  bf16x8 w2t[4];
#pragma unroll
  for (int ks = 0; ks < 4; ++ks) w2t[ks] = load_vec<bf16x8>(a.W2T + lr * hidden + hw0 + ks * 32 + lg * 8);
  bf16x4 w2p[8];
#pragma unroll
  for (int ht = 0; ht < 8; ++ht) w2p[ht] = load_vec<bf16x4>(a.W2p + (hw0 + ht * 16 + lr) * 16 + lg * 4);
  const float b2 = lr < a.classes ? a.b2[lr] : 0.0f;

  f32x4 dw2[8];
  float db1[8];   // this lane's rows' share of db1[hw0 + 16 ht + lr]
#pragma unroll
  for (int ht = 0; ht < 8; ++ht) {
    dw2[ht] = f32x4{};
    db1[ht] = 0.0f;
  }
  float db2 = 0.0f;
  int buf = 0;
  // H fragments of the logits GEMM (row r0 + lr, columns hw0 + 32 ks + 8 lg ..)
  // and the labels of rows r0 + 4 lg + i, fetched two tiles ahead into two
  // alternating register sets (labels loaded later would make every wait for
  // them wait for the prefetched tiles too: loads complete in order).
  bf16x8 ha[4], hb[4];
  int la[4], lb[4];
  // Every fetch issues the same loads on every path (H rows m .. m_pad - 1 are
  // zeros; labels past the partition read its last row), and the values are
  // only masked where a tile uses them, so the compiler's waits for a register
  // set count exactly the loads issued after it.  Slice ks of the block is
  // 1 KiB in lane order: row r0 + lr, columns hw0 + 32 ks + 8 lg .. + 7.
  auto fetch_h = [&](int64_t r0, bf16x8* dst, int* lab) {
    const bf16* blk = Hw + (r0 / 16) * hblocks * 2048;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) dst[ks] = load_vec<bf16x8>(blk + ks * 512 + lane * 8);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t lrow = r0 + lg * 4 + i;
      lab[i] = yp[lrow < a.m ? lrow : a.m - 1];
    }
  };
  auto tile = [&](int64_t r0, bf16x8* hcur, int* lcur) {
    f32x4 z = f32x4{};
    const bool hrow = r0 + lr < a.m;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const bf16x8 hv = hrow ? hcur[ks] : bf16x8{};
      z = mfma_k32(hv, w2t[ks], z);
      *reinterpret_cast<bf16x8*>(&Ht[wave][lr][ks * 32 + lg * 8]) = hv;
    }
    int label[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) label[i] = r0 + lg * 4 + i < a.m ? lcur[i] : -1;
    // The last two tiles of the block refetch themselves; the values go unused.
    fetch_h(r0 + 32 < rend ? r0 + 32 : r0, hcur, lcur);
#pragma unroll
    for (int i = 0; i < 4; ++i) zpart[buf][wave][lg * 4 + i][lr] = z[i];
    // LDS-only barrier: the H prefetch and the dZ1 stores stay in flight.
    lds_barrier();
    // Softmax over the classes of rows r0 + 4 lg + i (class lr on this lane).
    float dz2[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float s = 0.0f;
      for (int w = 0; w < waves; ++w) s += zpart[buf][w][lg * 4 + i][lr];
      const int64_t row = r0 + lg * 4 + i;
      const bool live = lr < a.classes;
      const float v = live ? s + b2 : -INFINITY;
      const float mx = row16_max(v);
      const float ex = live ? expf(v - mx) : 0.0f;
      const float sum = row16_sum(ex);
      dz2[i] = (row < a.m && live) ? (ex / sum - (lr == label[i] ? 1.0f : 0.0f)) * a.inv_m : 0.0f;
      db2 += dz2[i];
    }
    buf ^= 1;
    // The transposes below go through this wave's private LDS areas; a wave's
    // LDS operations complete in order, so they need no barrier.
#pragma unroll
    for (int i = 0; i < 4; ++i) dzt[wave][lg * 4 + i][lr] = dz2[i];
    bf16x4 dz_b, dz_a;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      dz_b[j] = static_cast<bf16>(dzt[wave][lr][lg * 4 + j]);   // dZ2[r0 + lr][4 lg + j]
      dz_a[j] = static_cast<bf16>(dz2[j]);                     // dZ2[r0 + 4 lg + j][lr]
    }
#pragma unroll
    for (int ht = 0; ht < 8; ++ht) {
      const int h = ht * 16;   // within the wave's columns
      // H[r0 + 4 lg + j][hw0 + h + lr]: the ReLU mask of dH below and the B
      // operand of dW2.
      // One transposing read: within each 16-lane group, lane i receives
      // element i % 4 of the 4-element row pieces addressed by lanes 4 j + i / 4,
      // so lane q addresses row 4 lg + q / 4, columns h + 4 (q % 4) .. + 3.
      const bf16x4t ht4 = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
          (lds_bf16x4t*)&Ht[wave][lg * 4 + (lr >> 2)][h + 4 * (lr & 3)]);
      const bf16x4 hcol = {ht4[0], ht4[1], ht4[2], ht4[3]};
      // dH[r0 + 4 lg + i][hw0 + h + lr] = sum_c dZ2[r0 + 4 lg + i][c] W2[hw0 + h + lr][c]
      // (A = dZ2 rows, B = W2^T columns: the lane's four values are four
      // consecutive rows of one hidden unit, 8 contiguous bytes of dZ1's
      // 16-row blocked layout).
      const f32x4 dh = mfma_k16(dz_b, w2p[ht], f32x4{});
      bf16x4 g4;
      float gsum = 0.0f;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float g = static_cast<float>(hcol[i]) > 0.0f ? dh[i] : 0.0f;
        gsum += g;
        g4[i] = static_cast<bf16>(g);
      }
      db1[ht] += gsum;
      // The 64 lanes write one contiguous 512-byte run of the dZ1 block.
      *reinterpret_cast<bf16x4*>(dz1 + ((r0 / 16) * hidden + hw0 + h + lr) * 16 + lg * 4) = g4;
      // dW2^T[4 lg + i][h + lr] += sum_r dZ2[r][4 lg + i] H[r][h + lr]
      dw2[ht] = mfma_k16(dz_a, hcol, dw2[ht]);
    }
  };
  // A block covers a multiple of 64 rows (head grid), so tiles come in pairs.
  if (rbeg < rend) {
    fetch_h(rbeg, ha, la);
    fetch_h(rbeg + 16, hb, lb);
  }
  for (int64_t r0 = rbeg; r0 < rend; r0 += 32) {
    tile(r0, ha, la);
    tile(r0 + 16, hb, lb);
  }

  float* out = a.partials + (static_cast<int64_t>(e) * a.blocks_per_part + blockIdx.x) * a.pstride;
#pragma unroll
  for (int ht = 0; ht < 8; ++ht) {
    const int h = hw0 + ht * 16;
#pragma unroll
    for (int i = 0; i < 4; ++i) out[(lg * 4 + i) * hidden + h + lr] = dw2[ht][i];
    float s = db1[ht];
    s += __shfl_xor(s, 16, 64);
    s += __shfl_xor(s, 32, 64);
    if (lg == 0) out[kMlpMaxClasses * hidden + h + lr] = s;
  }
  if (wave == 0) {
    float s = db2;
    s += __shfl_xor(s, 16, 64);
    s += __shfl_xor(s, 32, 64);
    if (lane < 16) out[(kMlpMaxClasses + 1) * hidden + lane] = s;
  }
}

// ---------------------------------------------------------------------------
// wgrad: dW1^T = dZ1^T X per partition, block tile 256 hidden x 224 features,
// K = rows in steps of 64.  8 waves: wave (wh, wf) owns hidden rows
// 64 wh .. 64 wh + 63 and features 112 wf .. 112 wf + 111 of the tile (a wave
// whose features all lie past d_in skips its MFMAs).  Both operands travel
// from global memory straight into LDS, one K step ahead, through two buffers
// (every load in the loop is such a load, so they complete in order and the
// per-step waits count them exactly):
//   A (dZ1, 16-row blocked): [4 row blocks][256 hidden][2 halves of 8 rows],
//     half s of hidden h stored at s ^ (((h >> 2) ^ (h >> 3)) & 1); the
//     fragments are plain 16-byte reads.
//   B (X rows): [64 rows][32 chunks of 16 bytes], the tile's 28 feature
//     chunks plus 4 spare, chunk j of row r at slot j ^ g(r) with g(r) even
//     and distinct over rows {0..3, 8..11}, so that the 32-byte row pieces a
//     transposing read gathers spread over the banks.  The fragments (8 rows
//     of one feature per lane) come from two transposing 8-byte reads: within
//     each 16-lane group, lane i receives element i % 4 of the 4-element row
//     pieces addressed by lanes 4 j + i / 4, j = 0..3.
// ---------------------------------------------------------------------------

constexpr int kWgBM = 256, kWgBN = 224, kWgBK = 64, kWgStages = 2;
constexpr int kWgThreads = 512;
constexpr int kWgAChunks = kWgBM * kWgBK / 8;          // 16-byte chunks of an A stage (2048)
constexpr int kWgBRowChunks = kWgBN / 8;               // 28 per X row ...
constexpr int kWgBRowSlots = 32;                       // ... in 32 slots
constexpr int kWgBChunks = kWgBK * kWgBRowSlots;       // 2048
constexpr int kWgStageBytes = (kWgAChunks + kWgBChunks) * 16;
constexpr int kWgALoads = kWgAChunks / kWgThreads, kWgBLoads = kWgBChunks / kWgThreads;
static_assert(kWgALoads * kWgThreads == kWgAChunks && kWgBLoads * kWgThreads == kWgBChunks, "load rounds");
static_assert(kWgStages * kWgStageBytes <= 160 * 1024, "LDS");

typedef bf16 bf16x4v __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) bf16x4v lds_bf16x4;

__device__ __forceinline__ int wg_half_swizzle(int h) { return ((h >> 2) ^ (h >> 3)) & 1; }
__device__ __forceinline__ int wg_row_swizzle(int r) { return 2 * ((r & 3) | (((r >> 3) & 1) << 2)); }

// Transposing 8-byte LDS read, issued as inline assembly: for the builtin the
// compiler waits for every outstanding direct-to-LDS load first (it cannot
// tell the buffers apart), which would drain the prefetch.  The kernel's own
// waits and barrier order the loads; the caller waits for lgkmcnt before use.
__device__ __forceinline__ bf16x4v ds_read_tr16(const bf16* p) {
  bf16x4v v;
  const uint32_t addr = static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_bf16x4*)p));
  asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(v) : "v"(addr));
  return v;
}

__global__ __launch_bounds__(kWgThreads, 1)
void mlp_wgrad_kernel(MlpWgradArgs a) {
  __shared__ __attribute__((aligned(16))) unsigned char smem[kWgStages * kWgStageBytes];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int wh = wave & 3, wf = wave >> 2;
  // With at least 8 evaluated partitions, every tile of a partition goes to
  // the same XCD (workgroups are dealt to the 8 XCDs round-robin), so its L2
  // serves the dZ1 rows to all feature tiles and the X rows to all hidden
  // tiles; otherwise the tiles are spread over the chip.
  const int htiles = a.hidden / kWgBM, ftiles = (a.d_in + kWgBN - 1) / kWgBN;
  const int tiles = htiles * ftiles;
  int e, tile;
  if (a.n_eval >= kXcds) {
    const int local = static_cast<int>(blockIdx.x) / kXcds;
    e = (local / tiles) * kXcds + static_cast<int>(blockIdx.x) % kXcds;
    tile = local % tiles;
    if (e >= a.n_eval) return;
  } else {
    e = static_cast<int>(blockIdx.x) / tiles;
    tile = static_cast<int>(blockIdx.x) % tiles;
  }
  const int64_t part = static_cast<int64_t>(e) * a.part_stride + a.part_offset;
  const int hb0 = (tile % htiles) * kWgBM;
  const int i0 = (tile / htiles) * kWgBN;
  const bool active = i0 + wf * (kWgBN / 2) < a.d_in;   // uniform per wave
  const bf16* Xp = a.X + part * a.m * a.d_in;
  const bf16* dz = a.dZ1 + mlp_dz1_index(a.m_pad, a.hidden, e, 0, 0);
  const int ksteps = static_cast<int>(a.m_pad / kWgBK);

  // A chunk c = u * 512 + tid: row block c / 512, hidden (c % 512) / 2, slot
  // c % 2 holding half (c % 2) ^ swizzle; its source is that half of the row
  // block of dZ1 (a run of 8 KiB per row block in global memory).
  int32_t aoff[kWgALoads];
#pragma unroll
  for (int u = 0; u < kWgALoads; ++u) {
    const int c = u * kWgThreads + tid, rb = c >> 9, h = (c & 511) >> 1;
    aoff[u] = (rb * a.hidden + hb0 + h) * 16 + ((c & 1) ^ wg_half_swizzle(h)) * 8;
  }
  // B chunk c: row c / 32 at slot c % 32, holding feature chunk
  // j = (c % 32) ^ g(row).  Spare chunks (j >= 28) and chunks past d_in read
  // the tile's first chunk of the row; a row past the partition reads its last
  // row: all meet zeros or land in columns that are never used or stored.
  int32_t brow[kWgBLoads], bcol[kWgBLoads];
#pragma unroll
  for (int u = 0; u < kWgBLoads; ++u) {
    const int c = u * kWgThreads + tid, row = c / kWgBRowSlots;
    const int j = (c % kWgBRowSlots) ^ wg_row_swizzle(row);
    const int col = i0 + j * 8;
    brow[u] = row;
    bcol[u] = (j < kWgBRowChunks && col < a.d_in) ? col : i0;
  }
  auto stage_a = [&](int buf) { return reinterpret_cast<bf16*>(smem + buf * kWgStageBytes); };
  auto stage_b = [&](int buf) { return reinterpret_cast<bf16*>(smem + buf * kWgStageBytes + kWgAChunks * 16); };
  auto issue = [&](int ks, int buf) {
    const bf16* dzk = dz + static_cast<int64_t>(ks) * (kWgBK / 16) * a.hidden * 16;
#pragma unroll
    for (int u = 0; u < kWgALoads; ++u)
      load_lds16(dzk + aoff[u], stage_a(buf) + (u * kWgThreads + wave * 64) * 8);
#pragma unroll
    for (int u = 0; u < kWgBLoads; ++u) {
      const int64_t r = static_cast<int64_t>(ks) * kWgBK + brow[u];
      load_lds16(Xp + (r < a.m ? r : a.m - 1) * a.d_in + bcol[u], stage_b(buf) + (u * kWgThreads + wave * 64) * 8);
    }
  };

  f32x4 acc[4][7];
#pragma unroll
  for (int mt = 0; mt < 4; ++mt)
#pragma unroll
    for (int nt = 0; nt < 7; ++nt) acc[mt][nt] = f32x4{};
  auto compute = [&](int buf) {
    const bf16* As = stage_a(buf);
    const bf16* Bs = stage_b(buf);
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      const int row = kk * 32 + lg * 8 + (lr >> 2);
      // Feature 112 wf + 16 nt + 4 (lr & 3) .. + 3 of the tile sits in chunk
      // 14 wf + 2 nt + ((lr & 3) >> 1), half (lr & 1).
      auto bpos = [&](int r, int nt) {
        return (r * kWgBRowSlots + ((14 * wf + 2 * nt + ((lr & 3) >> 1)) ^ wg_row_swizzle(r))) * 8 + (lr & 1) * 4;
      };
      bf16x4v lo[7], hi[7];
#pragma unroll
      for (int nt = 0; nt < 7; ++nt) {
        lo[nt] = ds_read_tr16(&Bs[bpos(row, nt)]);
        hi[nt] = ds_read_tr16(&Bs[bpos(row + 4, nt)]);
      }
      const int rb = kk * 2 + (lg >> 1), half = lg & 1;
      bf16x8 af[4];
#pragma unroll
      for (int mt = 0; mt < 4; ++mt) {
        const int h = wh * 64 + mt * 16 + lr;
        af[mt] = *reinterpret_cast<const bf16x8*>(&As[((rb * kWgBM + h) * 2 + (half ^ wg_half_swizzle(h))) * 8]);
      }
      // The transposing reads are invisible to the compiler's wait insertion:
      // wait here, with every result tied to the wait so no use moves above it.
      asm volatile("s_waitcnt lgkmcnt(0)"
                   : "+v"(lo[0]), "+v"(lo[1]), "+v"(lo[2]), "+v"(lo[3]), "+v"(lo[4]), "+v"(lo[5]), "+v"(lo[6]),
                     "+v"(hi[0]), "+v"(hi[1]), "+v"(hi[2]), "+v"(hi[3]), "+v"(hi[4]), "+v"(hi[5]), "+v"(hi[6]));
#pragma unroll
      for (int nt = 0; nt < 7; ++nt) {
        const bf16x8 bv = {lo[nt][0], lo[nt][1], lo[nt][2], lo[nt][3], hi[nt][0], hi[nt][1], hi[nt][2], hi[nt][3]};
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) acc[mt][nt] = mfma_k32(af[mt], bv, acc[mt][nt]);
      }
    }
  };

  issue(0, 0);
  for (int ks = 0; ks < ksteps; ++ks) {
    // This wave's loads of step ks have landed; after the barrier every
    // wave's have, and every wave is done reading the other buffer.
    wait_vmcnt<0>();
    lds_barrier();
    if (ks + 1 < ksteps) issue(ks + 1, (ks + 1) % kWgStages);
    if (active) compute(ks % kWgStages);
  }

  if (!active) return;
  float* slot = a.ring + (static_cast<int64_t>(a.plane) * a.n + part) * a.ld;
#pragma unroll
  for (int nt = 0; nt < 7; ++nt) {
    const int feat = i0 + wf * (kWgBN / 2) + nt * 16 + lr;
    if (feat >= a.d_in) continue;
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
      *reinterpret_cast<f32x4*>(slot + static_cast<int64_t>(feat) * a.hidden + hb0 + wh * 64 + mt * 16 + lg * 4) =
          acc[mt][nt];
  }
}

// ---------------------------------------------------------------------------
// reduce: head partials -> ring (b1, W2 in [hidden][classes] order, b2)
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(256)
void mlp_reduce_kernel(MlpReduceArgs a) {
  const int j = blockIdx.x * 256 + threadIdx.x;
  if (j >= a.pstride) return;
  const int e = blockIdx.y;
  const int64_t part = static_cast<int64_t>(e) * a.part_stride + a.part_offset;
  const float* p = a.partials + static_cast<int64_t>(e) * a.blocks_per_part * a.pstride + j;
  double s = 0.0;
  for (int b = 0; b < a.blocks_per_part; ++b) s += static_cast<double>(p[static_cast<int64_t>(b) * a.pstride]);
  float* slot = a.ring + (static_cast<int64_t>(a.plane) * a.n + part) * a.ld;
  const int64_t w1 = static_cast<int64_t>(a.d_in) * a.hidden;
  const int hw = kMlpMaxClasses * a.hidden;
  if (j < hw) {
    const int c = j / a.hidden, h = j % a.hidden;
    if (c < a.classes) slot[w1 + a.hidden + static_cast<int64_t>(h) * a.classes + c] = static_cast<float>(s);
  } else if (j < hw + a.hidden) {
    slot[w1 + (j - hw)] = static_cast<float>(s);
  } else {
    const int c = j - hw - a.hidden;
    if (c < a.classes)
      slot[w1 + a.hidden + static_cast<int64_t>(a.hidden) * a.classes + c] = static_cast<float>(s);
  }
}

}  // namespace

hipError_t launch_mlp_cast(const MlpCastArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(mlp_cast_w1_kernel, dim3(a.kpad / 32, a.hidden / 32), dim3(256), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(mlp_cast_w2_kernel, dim3((a.hidden * kMlpMaxClasses + 255) / 256), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_mlp_forward(const MlpForwardArgs& a, hipStream_t s) {
  const int64_t rtiles = (a.m + kFwBM - 1) / kFwBM * a.n_eval;
  dim3 grid(static_cast<unsigned>((rtiles + kXcds - 1) / kXcds * kXcds * (a.hidden / kFwBN)));
  hipLaunchKernelGGL(mlp_forward_kernel<kFwBM>, grid, dim3(kFwThreads), 0, s, a);
  return hipGetLastError();
}

int mlp_head_threads(int hidden) { return 64 * (hidden / kHeadCols); }

hipError_t launch_mlp_head(const MlpHeadArgs& a, hipStream_t s) {
  dim3 grid(a.blocks_per_part, a.n_eval);
  hipLaunchKernelGGL(mlp_head_kernel, grid, dim3(mlp_head_threads(a.hidden)), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_mlp_wgrad(const MlpWgradArgs& a, hipStream_t s) {
  const int tiles = (a.hidden / kWgBM) * ((a.d_in + kWgBN - 1) / kWgBN);
  const int parts = a.n_eval >= kXcds ? (a.n_eval + kXcds - 1) / kXcds * kXcds : a.n_eval;
  dim3 grid(static_cast<unsigned>(tiles * parts));
  hipLaunchKernelGGL(mlp_wgrad_kernel, grid, dim3(kWgThreads), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_mlp_reduce(const MlpReduceArgs& a, hipStream_t s) {
  dim3 grid((a.pstride + 255) / 256, a.n_eval);
  hipLaunchKernelGGL(mlp_reduce_kernel, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace pgc
