// C ABI of the PGC step (include/pgc.h): context, validation, workspace
// layout and the per-step launch sequence.
#include <hip/hip_runtime_api.h>
#include <rocprofiler-sdk-roctx/roctx.h>

#include <algorithm>
#include <cstring>
#include <cmath>
#include <string>
#include <vector>

#include "pgc.h"
#include "pgc_codes.h"
#include "pgc_kernels.h"
#include "pgc_step.h"

namespace {

constexpr size_t kAlign = 256;
// Gradient grid: about pgc::linear_grad_target_blocks(d) blocks per launch,
// never fewer than kMinRowsPerBlock rows per block.  The grid depends only on
// the problem shape, so results do not depend on the device.
constexpr int64_t kMinRowsPerBlock = 16;
// MLP head: about this many blocks per launch, rows per block a multiple of 64.
constexpr int64_t kHeadTargetBlocks = 1024;
// Ring slots and coded words are padded to a multiple of this many floats:
// every slot starts 1 KiB aligned, and the code kernel's 256-column blocks
// cover a slot exactly (never spilling into the next one).
constexpr int64_t kSlotAlign = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }
int64_t round_up(int64_t x, int64_t a) { return (x + a - 1) / a * a; }

struct Grid {
  int32_t n_eval = 0;
  int32_t blocks_per_part = 0;
  int64_t rows_per_block = 0;
};

Grid make_grid(int64_t m, int32_t n_eval, int64_t target_blocks) {
  Grid g;
  g.n_eval = n_eval;
  int64_t b = (target_blocks + n_eval - 1) / n_eval;
  b = std::max<int64_t>(1, std::min<int64_t>(b, (m + kMinRowsPerBlock - 1) / kMinRowsPerBlock));
  g.rows_per_block = (m + b - 1) / b;
  g.blocks_per_part = static_cast<int32_t>((m + g.rows_per_block - 1) / g.rows_per_block);
  return g;
}

// Head grid of the MLP: blocks of a multiple of 64 rows over the m_pad rows.
Grid make_head_grid(int64_t m_pad, int32_t n_eval) {
  Grid g;
  g.n_eval = n_eval;
  int64_t b = (kHeadTargetBlocks + n_eval - 1) / n_eval;
  b = std::max<int64_t>(1, std::min<int64_t>(b, m_pad / 64));
  g.rows_per_block = round_up((m_pad + b - 1) / b, 64);
  g.blocks_per_part = static_cast<int32_t>((m_pad + g.rows_per_block - 1) / g.rows_per_block);
  return g;
}

struct Timed {
  hipEvent_t start = nullptr, stop = nullptr;
  int kernel = 0;
};

}  // namespace

struct pgc_ctx {
  int scheme = 0, n = 0, c = 0;
  int64_t d = 0;
  bool configured = false;
  pgc_config cfg{};
  int64_t m = 0;
  std::vector<double> B;      // n x n encoding matrix (row-major)
  std::vector<double> coef;   // n_coded x c slot coefficients (real-valued code only)
  // Workspace layout (byte offsets).
  int planes = 0, n_coded = 0;
  int64_t ld = 0;             // floats between ring slots / coded words
  Grid warm, pipe;            // linear gradient grids
  Grid head_warm, head_pipe;  // MLP head grids
  int64_t kpad = 0, m_pad = 0, pstride = 0;
  size_t off_ring = 0, off_coded = 0, off_decoded = 0, off_partials = 0, off_coef = 0, ws_need = 0;
  size_t off_w1t = 0, off_w2t = 0, off_w2p = 0, off_h = 0, off_dz1 = 0;
  size_t partials_bytes = 0;  // linear models: block partial sums of the larger gradient grid
  char* ws = nullptr;
  size_t ws_bytes = 0;
  hipStream_t stream = nullptr;
  int64_t t = 0;
  bool pipelined = true;      // false: gradient coding (every slot evaluated each step)
  std::string err;
  unsigned timing = 0;        // bit k: time kernel k
  int64_t timing_period = 1;  // time one launch in this many of each selected kernel
  int64_t seen[PGC_KERNEL_COUNT] = {};   // launches of each kernel since timing was set
  std::vector<Timed> pending;
  std::vector<Timed> spare;
  double total_ms[PGC_KERNEL_COUNT] = {};
  int64_t launches[PGC_KERNEL_COUNT] = {};
};

namespace {

int fail(pgc_ctx* ctx, int status, const std::string& msg) {
  if (ctx) ctx->err = msg;
  return status;
}
int fail(const pgc_ctx* ctx, int status, const std::string& msg) {
  return fail(const_cast<pgc_ctx*>(ctx), status, msg);
}

int device_fail(pgc_ctx* ctx, hipError_t e, const char* what) {
  return fail(ctx, PGC_EDEVICE, std::string(what) + ": " + hipGetErrorString(e));
}

bool is_linear(int model) { return model == PGC_LOGISTIC || model == PGC_LSQ; }

void compute_layout(pgc_ctx* ctx) {
  const int64_t q = ctx->d;
  const int n = ctx->n;
  const int32_t n_pipe = ctx->scheme == PGC_FR ? n / ctx->c : n;
  ctx->planes = ctx->scheme == PGC_FR ? 1 : ctx->c;
  ctx->n_coded = ctx->scheme == PGC_FR ? n / ctx->c : n;
  ctx->ld = round_up(q, kSlotAlign);
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off = align_up(off + bytes);
    return at;
  };
  ctx->off_ring = take(sizeof(float) * static_cast<size_t>(ctx->planes) * n * ctx->ld);
  ctx->off_coded = take(sizeof(float) * static_cast<size_t>(ctx->n_coded) * ctx->ld);
  ctx->off_decoded = take(sizeof(float) * static_cast<size_t>(q));
  ctx->off_coef = take(sizeof(double) * ctx->coef.size());
  if (ctx->cfg.model == PGC_MLP) {
    const int64_t hidden = ctx->cfg.hidden;
    ctx->kpad = round_up(ctx->cfg.d_in, 64);   // the forward GEMM's K step
    ctx->m_pad = round_up(ctx->m, 64);   // the weight-gradient GEMM's K step
    ctx->pstride = (pgc::kMlpMaxClasses + 1) * hidden + pgc::kMlpMaxClasses;
    ctx->head_warm = make_head_grid(ctx->m_pad, n);
    ctx->head_pipe = make_head_grid(ctx->m_pad, n_pipe);
    const int64_t head_blocks =
        std::max<int64_t>(static_cast<int64_t>(ctx->head_warm.n_eval) * ctx->head_warm.blocks_per_part,
                          static_cast<int64_t>(ctx->head_pipe.n_eval) * ctx->head_pipe.blocks_per_part);
    ctx->off_w1t = take(2 * static_cast<size_t>(hidden * ctx->kpad));
    ctx->off_w2t = take(2 * static_cast<size_t>(pgc::kMlpMaxClasses * hidden));
    ctx->off_w2p = take(2 * static_cast<size_t>(hidden * pgc::kMlpMaxClasses));
    ctx->off_h = take(2 * static_cast<size_t>(n) * ctx->m_pad * hidden);
    ctx->off_dz1 = take(2 * static_cast<size_t>(n) * hidden * ctx->m_pad);
    ctx->off_partials = take(sizeof(float) * static_cast<size_t>(head_blocks * ctx->pstride));
  } else {
    const int64_t target = pgc::linear_grad_target_blocks(static_cast<int>(q));
    ctx->warm = make_grid(ctx->m, n, target);
    ctx->pipe = make_grid(ctx->m, n_pipe, target);
    const int64_t max_blocks =
        std::max<int64_t>(static_cast<int64_t>(ctx->warm.n_eval) * ctx->warm.blocks_per_part,
                          static_cast<int64_t>(ctx->pipe.n_eval) * ctx->pipe.blocks_per_part);
    ctx->partials_bytes = sizeof(float) * static_cast<size_t>(max_blocks) * q;
    ctx->off_partials = take(ctx->partials_bytes);
  }
  ctx->ws_need = off;
}

template <class T>
T* ws_ptr(const pgc_ctx* ctx, size_t off) {
  return reinterpret_cast<T*>(ctx->ws + off);
}

// Resolve recorded kernel events whose work has completed, or all of them.
int resolve_timing(pgc_ctx* ctx, bool wait) {
  size_t done = 0;
  int status = PGC_OK;
  for (; done < ctx->pending.size(); ++done) {
    Timed& tm = ctx->pending[done];
    if (wait) {
      hipError_t e = hipEventSynchronize(tm.stop);
      if (e != hipSuccess) {
        status = device_fail(ctx, e, "hipEventSynchronize");
        break;
      }
    } else {
      const hipError_t q = hipEventQuery(tm.stop);
      if (q == hipErrorNotReady) break;
      if (q != hipSuccess) {
        status = device_fail(ctx, q, "hipEventQuery");
        break;
      }
    }
    float ms = 0.f;
    hipError_t e = hipEventElapsedTime(&ms, tm.start, tm.stop);
    if (e != hipSuccess) {
      status = device_fail(ctx, e, "hipEventElapsedTime");
      break;
    }
    ctx->total_ms[tm.kernel] += ms;
    ctx->launches[tm.kernel] += 1;
    ctx->spare.push_back(tm);
  }
  // Pairs already counted leave the pending list even when a later one fails,
  // so no launch is counted twice and no pair is both pending and spare.
  ctx->pending.erase(ctx->pending.begin(), ctx->pending.begin() + done);
  return status;
}

// Launch `fn` on the context stream, bracketed by events when timing is on.
template <class Fn>
int timed_launch(pgc_ctx* ctx, int kernel, const char* what, Fn fn) {
  Timed tm;
  const bool timed = ((ctx->timing >> kernel) & 1u) && ctx->seen[kernel]++ % ctx->timing_period == 0;
  if (timed) {
    if (ctx->pending.size() >= 4096) {
      int st = resolve_timing(ctx, false);
      if (st != PGC_OK) return st;
    }
    if (!ctx->spare.empty()) {
      tm = ctx->spare.back();
      ctx->spare.pop_back();
    } else {
      hipError_t e = hipEventCreate(&tm.start);
      if (e == hipSuccess) {
        e = hipEventCreate(&tm.stop);
        if (e != hipSuccess) (void)hipEventDestroy(tm.start);
      }
      if (e != hipSuccess) return device_fail(ctx, e, "hipEventCreate");
    }
    tm.kernel = kernel;
    hipError_t e = hipEventRecord(tm.start, ctx->stream);
    if (e != hipSuccess) {
      ctx->spare.push_back(tm);
      return device_fail(ctx, e, "hipEventRecord");
    }
  }
  hipError_t e = fn();
  if (e != hipSuccess) {
    if (timed) ctx->spare.push_back(tm);   // the pair is reused; its start is simply re-recorded
    return device_fail(ctx, e, what);
  }
  if (timed) {
    e = hipEventRecord(tm.stop, ctx->stream);
    if (e != hipSuccess) {
      ctx->spare.push_back(tm);
      return device_fail(ctx, e, "hipEventRecord");
    }
    ctx->pending.push_back(tm);
  }
  return PGC_OK;
}

void release_events(pgc_ctx* ctx) {
  for (auto* list : {&ctx->pending, &ctx->spare})
    for (Timed& tm : *list) {
      if (tm.start) (void)hipEventDestroy(tm.start);
      if (tm.stop) (void)hipEventDestroy(tm.stop);
    }
  ctx->pending.clear();
  ctx->spare.clear();
}

}  // namespace

extern "C" {

const char* pgc_strerror(int status) {
  switch (status) {
    case PGC_OK: return "ok";
    case PGC_EINVAL: return "invalid argument";
    case PGC_ESTRAGGLERS: return "too many stragglers for the scheme";
    case PGC_ESINGULAR: return "the real-valued code cannot decode this straggler set";
    case PGC_EDEVICE: return "HIP runtime error";
    case PGC_ESTATE: return "call out of order";
  }
  return "unknown status";
}

const char* pgc_last_error(const pgc_ctx* ctx) {
  return ctx ? ctx->err.c_str() : "null context";
}

int pgc_init(pgc_ctx** out, int scheme, int n, int c, int64_t d) {
  if (out == nullptr) return PGC_EINVAL;
  *out = nullptr;
  if (scheme != PGC_FR && scheme != PGC_CR && scheme != PGC_CR_REAL && scheme != PGC_IS_SGD)
    return PGC_EINVAL;
  if (n < 1 || n > PGC_MAX_N || c < 1 || c > n || d < 1) return PGC_EINVAL;
  if (scheme == PGC_FR && n % c != 0) return PGC_EINVAL;
  if (scheme == PGC_IS_SGD && c != 1) return PGC_EINVAL;
  pgc_ctx* ctx = new (std::nothrow) pgc_ctx;
  if (ctx == nullptr) return PGC_EINVAL;
  ctx->scheme = scheme;
  ctx->n = n;
  ctx->c = c;
  ctx->d = d;
  *out = ctx;
  return PGC_OK;
}

int pgc_destroy(pgc_ctx* ctx) {
  if (ctx == nullptr) return PGC_OK;
  release_events(ctx);
  delete ctx;
  return PGC_OK;
}

int pgc_configure(pgc_ctx* ctx, const pgc_config* cfg) {
  if (ctx == nullptr) return PGC_EINVAL;
  if (cfg == nullptr) return fail(ctx, PGC_EINVAL, "null config");
  ctx->configured = false;
  ctx->ws = nullptr;
  ctx->ws_bytes = 0;
  ctx->t = 0;
  if (cfg->N <= 0 || cfg->N % ctx->n != 0)
    return fail(ctx, PGC_EINVAL, "N must be a positive multiple of n");
  if (is_linear(cfg->model)) {
    if (cfg->d_in != ctx->d) return fail(ctx, PGC_EINVAL, "d_in must equal d for linear models");
    if (ctx->d > PGC_MAX_LINEAR_D)
      return fail(ctx, PGC_EINVAL, "d exceeds PGC_MAX_LINEAR_D");
  } else if (cfg->model == PGC_MLP) {
    const int64_t d_in = cfg->d_in, hidden = cfg->hidden, classes = cfg->classes;
    if (d_in < 8 || d_in % 8 != 0) return fail(ctx, PGC_EINVAL, "MLP d_in must be a positive multiple of 8");
    // The forward GEMM addresses a row tile of X with 32-bit byte offsets.
    if (d_in > PGC_MLP_MAX_D_IN) return fail(ctx, PGC_EINVAL, "MLP d_in exceeds PGC_MLP_MAX_D_IN");
    if (hidden < 256 || hidden % 256 != 0 || hidden > PGC_MLP_MAX_HIDDEN)
      return fail(ctx, PGC_EINVAL, "MLP hidden must be a multiple of 256 up to PGC_MLP_MAX_HIDDEN");
    if (classes < 1 || classes > PGC_MLP_MAX_CLASSES)
      return fail(ctx, PGC_EINVAL, "MLP classes must be in 1..PGC_MLP_MAX_CLASSES");
    if (ctx->d != d_in * hidden + hidden + hidden * classes + classes)
      return fail(ctx, PGC_EINVAL, "d must equal d_in*hidden + hidden + hidden*classes + classes");
  } else {
    return fail(ctx, PGC_EINVAL, "unknown model");
  }
  ctx->cfg = *cfg;
  ctx->m = cfg->N / ctx->n;
  const int n = ctx->n, c = ctx->c;
  ctx->B.assign(static_cast<size_t>(n) * n, 0.0);
  ctx->coef.clear();
  if (ctx->scheme == PGC_CR_REAL) {
    std::string err;
    const std::vector<double> H = pgc::null_space_generator(cfg->code_seed, c - 1, n);
    if (!pgc::cyclic_encoding_matrix(n, c, H, &ctx->B, &err)) return fail(ctx, PGC_ESINGULAR, err);
    ctx->coef.resize(static_cast<size_t>(n) * c);
    for (int j = 0; j < n; ++j)
      for (int o = 0; o < c; ++o)
        ctx->coef[static_cast<size_t>(j) * c + o] = ctx->B[static_cast<size_t>(j) * n + (j + o) % n];
  } else {
    for (int j = 0; j < n; ++j)
      for (int o = 0; o < c; ++o)
        ctx->B[static_cast<size_t>(j) * n + pgc::held_partition(ctx->scheme, n, c, j, o)] = 1.0;
  }
  compute_layout(ctx);
  ctx->configured = true;
  return PGC_OK;
}

int pgc_set_pipelining(pgc_ctx* ctx, int enabled) {
  if (ctx == nullptr) return PGC_EINVAL;
  ctx->pipelined = enabled != 0;
  return PGC_OK;
}

int pgc_set_stream(pgc_ctx* ctx, void* hip_stream) {
  if (ctx == nullptr) return PGC_EINVAL;
  hipStream_t next = static_cast<hipStream_t>(hip_stream);
  if (next != ctx->stream) {
    // Later steps read the ring, partials and w that steps enqueued on the old
    // stream write: wait for them, unless either stream is being captured
    // into a graph (a synchronisation there would end the capture; the
    // caller orders the streams around a capture).
    hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
    hipError_t e = hipStreamIsCapturing(next, &cap);
    if (e != hipSuccess) return device_fail(ctx, e, "hipStreamIsCapturing (new stream)");
    if (cap == hipStreamCaptureStatusNone) {
      e = hipStreamIsCapturing(ctx->stream, &cap);
      if (e != hipSuccess) return device_fail(ctx, e, "hipStreamIsCapturing (old stream)");
      if (cap == hipStreamCaptureStatusNone) {
        e = hipStreamSynchronize(ctx->stream);
        if (e != hipSuccess) return device_fail(ctx, e, "hipStreamSynchronize (old stream)");
      }
    }
  }
  ctx->stream = next;
  return PGC_OK;
}

int pgc_workspace_bytes(const pgc_ctx* ctx, size_t* bytes) {
  if (ctx == nullptr || bytes == nullptr) return PGC_EINVAL;
  if (!ctx->configured) return fail(ctx, PGC_ESTATE, "pgc_configure first");
  *bytes = ctx->ws_need;
  return PGC_OK;
}

int pgc_bind_workspace(pgc_ctx* ctx, void* dev_workspace, size_t bytes) {
  if (ctx == nullptr) return PGC_EINVAL;
  if (!ctx->configured) return fail(ctx, PGC_ESTATE, "pgc_configure first");
  if (dev_workspace == nullptr) return fail(ctx, PGC_EINVAL, "null workspace");
  if (reinterpret_cast<uintptr_t>(dev_workspace) % kAlign != 0)
    return fail(ctx, PGC_EINVAL, "workspace must be 256-byte aligned");
  if (bytes < ctx->ws_need)
    return fail(ctx, PGC_EINVAL, "workspace too small: need " + std::to_string(ctx->ws_need) + " bytes");
  // Work already enqueued on the context stream may still read the old
  // workspace (a rebind of the same memory rewrites the code table below).
  hipError_t e = hipStreamSynchronize(ctx->stream);
  if (e != hipSuccess) return device_fail(ctx, e, "hipStreamSynchronize");
  ctx->ws = static_cast<char*>(dev_workspace);
  ctx->ws_bytes = bytes;
  ctx->t = 0;
  if (!ctx->coef.empty()) {
    e = hipMemcpy(ctx->ws + ctx->off_coef, ctx->coef.data(), sizeof(double) * ctx->coef.size(),
                  hipMemcpyHostToDevice);
    if (e != hipSuccess) {
      ctx->ws = nullptr;
      return device_fail(ctx, e, "uploading the encoding table");
    }
  }
  return PGC_OK;
}

int pgc_decode_coeffs(const pgc_ctx* ctx, const uint8_t* straggler_mask, double* d_out,
                      double* scale_out, int32_t* survivors_out, int32_t* n_survivors_out) {
  if (ctx == nullptr) return PGC_EINVAL;
  if (!ctx->configured) return fail(ctx, PGC_ESTATE, "pgc_configure first");
  if (!straggler_mask || !d_out || !scale_out || !survivors_out || !n_survivors_out)
    return fail(ctx, PGC_EINVAL, "null pointer");
  pgc::Decode dec;
  std::string err;
  switch (pgc::decode_coefficients(ctx->scheme, ctx->n, ctx->c, ctx->B, straggler_mask, &dec, &err)) {
    case pgc::kDecodeStragglers: return fail(ctx, PGC_ESTRAGGLERS, err);
    case pgc::kDecodeSingular: return fail(ctx, PGC_ESINGULAR, err);
    default: break;
  }
  const int nj = static_cast<int>(dec.survivors.size());
  for (int i = 0; i < nj; ++i) {
    survivors_out[i] = dec.survivors[i];
    d_out[i] = dec.d[i];
  }
  for (int i = nj; i < ctx->n; ++i) {
    survivors_out[i] = -1;
    d_out[i] = 0.0;
  }
  *scale_out = dec.scale;
  *n_survivors_out = nj;
  return PGC_OK;
}

int pgc_placement(const pgc_ctx* ctx, int32_t* out) {
  if (ctx == nullptr || out == nullptr) return PGC_EINVAL;
  for (int i = 0; i < ctx->n; ++i)
    for (int l = 0; l < ctx->c; ++l)
      out[i * ctx->c + l] = pgc::held_partition(ctx->scheme, ctx->n, ctx->c, i, l);
  return PGC_OK;
}

int pgc_schedule(const pgc_ctx* ctx, int64_t t, int32_t* out) {
  if (ctx == nullptr || out == nullptr) return PGC_EINVAL;
  if (t < 1) return fail(ctx, PGC_EINVAL, "step 0 evaluates every held partition (see pgc_placement)");
  const int o = pgc::evaluated_slot(t, ctx->c);
  for (int i = 0; i < ctx->n; ++i) out[i] = pgc::held_partition(ctx->scheme, ctx->n, ctx->c, i, o);
  return PGC_OK;
}

int pgc_encoding_matrix(const pgc_ctx* ctx, double* out) {
  if (ctx == nullptr || out == nullptr) return PGC_EINVAL;
  if (!ctx->configured) return fail(ctx, PGC_ESTATE, "pgc_configure first");
  std::copy(ctx->B.begin(), ctx->B.end(), out);
  return PGC_OK;
}

int pgc_num_coded(const pgc_ctx* ctx, int32_t* out) {
  if (ctx == nullptr || out == nullptr) return PGC_EINVAL;
  *out = ctx->scheme == PGC_FR ? ctx->n / ctx->c : ctx->n;
  return PGC_OK;
}

int pgc_make_mask(uint64_t seed, int64_t t, int policy, int n, int cap, double p, uint8_t* out) {
  if (n < 1 || n > PGC_MAX_N) return PGC_EINVAL;
  return pgc::make_mask(seed, t, policy, n, cap, p, out) ? PGC_OK : PGC_EINVAL;
}

int pgc_delay_step(uint64_t seed, int64_t t, int n, int s, double mean_delay, double compute_seconds,
                   uint8_t* mask, double* delays, double* step_seconds) {
  if (n < 1 || n > PGC_MAX_N) return PGC_EINVAL;
  return pgc::delay_step(seed, t, n, s, mean_delay, compute_seconds, mask, delays, step_seconds)
             ? PGC_OK : PGC_EINVAL;
}

int pgc_splitmix64(uint64_t seed, uint64_t index, uint64_t* out) {
  if (out == nullptr) return PGC_EINVAL;
  *out = pgc::splitmix64(seed, index);
  return PGC_OK;
}

int pgc_get_step(const pgc_ctx* ctx, int64_t* t) {
  if (ctx == nullptr || t == nullptr) return PGC_EINVAL;
  *t = ctx->t;
  return PGC_OK;
}

}  // extern "C"

namespace {

// Arguments of the encode + masked decode + update (a6-a8).
pgc::CodeArgs code_args(pgc_ctx* ctx, const pgc::Decode& dec, float* w, float lr) {
  const int c = ctx->c;
  const bool fr = ctx->scheme == PGC_FR;
  pgc::CodeArgs ca{};
  ca.ring = ws_ptr<float>(ctx, ctx->off_ring);
  ca.coded = ws_ptr<float>(ctx, ctx->off_coded);
  ca.decoded = ws_ptr<float>(ctx, ctx->off_decoded);
  ca.w = w;
  ca.coef = ctx->coef.empty() ? nullptr : ws_ptr<double>(ctx, ctx->off_coef);
  ca.q = ctx->d;
  ca.ld = ctx->ld;
  ca.lr = static_cast<double>(lr);
  ca.n = ctx->n;
  ca.c = c;
  ca.n_coded = ctx->n_coded;
  ca.fr = fr ? 1 : 0;
  // FR's coded words are per group (its members' words are identical); CR's per worker.
  for (size_t m = 0; m < dec.survivors.size(); ++m) {
    if (dec.d[m] == 0.0) continue;
    const int j = fr ? dec.survivors[m] / c : dec.survivors[m];
    ca.a[j] = dec.scale * dec.d[m];
  }
  return ca;
}

// The linear models' step: the gradient kernel (a4), then one launch that
// folds its partials into the ring (a5) and runs encode, decode and update (a6-a8).
int linear_step(pgc_ctx* ctx, const void* X, const void* y, float* w, const pgc::Decode& dec, float lr,
                bool warm, int32_t part_stride, int32_t part_offset, int plane_first, int plane_count,
                float* partials) {
  const Grid& grid = warm ? ctx->warm : ctx->pipe;
  pgc::LinearGradArgs ga{};
  ga.X = static_cast<const float*>(X);
  ga.y = static_cast<const float*>(y);
  ga.w = w;
  ga.partials = partials;
  ga.m = ctx->m;
  ga.rows_per_block = grid.rows_per_block;
  ga.d = static_cast<int32_t>(ctx->d);
  ga.blocks_per_part = grid.blocks_per_part;
  ga.n_eval = grid.n_eval;
  ga.part_stride = part_stride;
  ga.part_offset = part_offset;
  ga.model = ctx->cfg.model;
  const bool aligned16 = reinterpret_cast<uintptr_t>(X) % 16 == 0 &&
                         reinterpret_cast<uintptr_t>(w) % 16 == 0;

  pgc::ReduceCodeArgs ra{};
  ra.code = code_args(ctx, dec, w, lr);
  ra.ring = ws_ptr<float>(ctx, ctx->off_ring);
  ra.partials = ga.partials;
  ra.inv_m = 1.0 / static_cast<double>(ctx->m);
  ra.n_eval = grid.n_eval;
  ra.blocks_per_part = grid.blocks_per_part;
  ra.part_stride = part_stride;
  ra.part_offset = part_offset;
  ra.plane_first = plane_first;
  ra.plane_count = plane_count;

  int st = timed_launch(ctx, PGC_KERNEL_GRADIENT, "gradient kernel",
                        [&] { return pgc::launch_linear_gradient(ga, aligned16, ctx->stream); });
  if (st != PGC_OK) return st;
  return timed_launch(ctx, PGC_KERNEL_CODE, "reduce/code kernel",
                      [&] { return pgc::launch_reduce_code(ra, ctx->stream); });
}

// a4-a5 for the MLP: cast, forward, head, weight gradient, small-part reduce,
// then copies of the slot into the other planes at the CR warm-up.
int mlp_step(pgc_ctx* ctx, const void* X, const void* y, float* w, const pgc::Decode& dec, float lr,
             bool warm, int32_t part_stride, int32_t part_offset, int plane_first, int plane_count) {
  const Grid& hg = warm ? ctx->head_warm : ctx->head_pipe;
  const int32_t d_in = ctx->cfg.d_in, hidden = ctx->cfg.hidden, classes = ctx->cfg.classes;
  const int64_t w1 = static_cast<int64_t>(d_in) * hidden;
  __bf16* W1T = ws_ptr<__bf16>(ctx, ctx->off_w1t);
  __bf16* W2T = ws_ptr<__bf16>(ctx, ctx->off_w2t);
  __bf16* W2p = ws_ptr<__bf16>(ctx, ctx->off_w2p);
  __bf16* H = ws_ptr<__bf16>(ctx, ctx->off_h);
  __bf16* dZ1 = ws_ptr<__bf16>(ctx, ctx->off_dz1);
  float* ring = ws_ptr<float>(ctx, ctx->off_ring);
  float* partials = ws_ptr<float>(ctx, ctx->off_partials);

  pgc::MlpCastArgs cast{w, W1T, W2T, W2p, d_in, static_cast<int32_t>(ctx->kpad), hidden, classes};
  pgc::MlpForwardArgs fw{};
  fw.X = static_cast<const __bf16*>(X);
  fw.W1T = W1T;
  fw.b1 = w + w1;
  fw.H = H;
  fw.m = ctx->m;
  fw.m_pad = ctx->m_pad;
  fw.d_in = d_in;
  fw.kpad = static_cast<int32_t>(ctx->kpad);
  fw.hidden = hidden;
  fw.n_eval = hg.n_eval;
  fw.part_stride = part_stride;
  fw.part_offset = part_offset;
  pgc::MlpHeadArgs hd{};
  hd.H = H;
  hd.y = static_cast<const int32_t*>(y);
  hd.W2T = W2T;
  hd.W2p = W2p;
  hd.b2 = w + w1 + hidden + static_cast<int64_t>(hidden) * classes;
  hd.dZ1 = dZ1;
  hd.partials = partials;
  hd.m = ctx->m;
  hd.m_pad = ctx->m_pad;
  hd.rows_per_block = hg.rows_per_block;
  hd.inv_m = static_cast<float>(1.0 / static_cast<double>(ctx->m));
  hd.hidden = hidden;
  hd.classes = classes;
  hd.blocks_per_part = hg.blocks_per_part;
  hd.n_eval = hg.n_eval;
  hd.part_stride = part_stride;
  hd.part_offset = part_offset;
  hd.pstride = static_cast<int32_t>(ctx->pstride);
  pgc::MlpWgradArgs wg{};
  wg.X = fw.X;
  wg.dZ1 = dZ1;
  wg.ring = ring;
  wg.m = ctx->m;
  wg.m_pad = ctx->m_pad;
  wg.ld = ctx->ld;
  wg.d_in = d_in;
  wg.hidden = hidden;
  wg.n = ctx->n;
  wg.plane = plane_first;
  wg.n_eval = hg.n_eval;
  wg.part_stride = part_stride;
  wg.part_offset = part_offset;
  pgc::MlpReduceArgs rd{};
  rd.partials = partials;
  rd.ring = ring;
  rd.ld = ctx->ld;
  rd.d_in = d_in;
  rd.hidden = hidden;
  rd.classes = classes;
  rd.n = ctx->n;
  rd.plane = plane_first;
  rd.n_eval = hg.n_eval;
  rd.blocks_per_part = hg.blocks_per_part;
  rd.part_stride = part_stride;
  rd.part_offset = part_offset;
  rd.pstride = static_cast<int32_t>(ctx->pstride);

  int st = timed_launch(ctx, PGC_KERNEL_MLP_CAST, "MLP cast kernels",
                        [&] { return pgc::launch_mlp_cast(cast, ctx->stream); });
  if (st == PGC_OK)
    st = timed_launch(ctx, PGC_KERNEL_MLP_FORWARD, "MLP forward kernel",
                      [&] { return pgc::launch_mlp_forward(fw, ctx->stream); });
  if (st == PGC_OK)
    st = timed_launch(ctx, PGC_KERNEL_MLP_HEAD, "MLP head kernel",
                      [&] { return pgc::launch_mlp_head(hd, ctx->stream); });
  if (st == PGC_OK)
    st = timed_launch(ctx, PGC_KERNEL_MLP_WGRAD, "MLP weight-gradient kernel",
                      [&] { return pgc::launch_mlp_wgrad(wg, ctx->stream); });
  if (st == PGC_OK)
    st = timed_launch(ctx, PGC_KERNEL_REDUCE, "MLP reduce kernel", [&] {
      hipError_t e = pgc::launch_mlp_reduce(rd, ctx->stream);
      // CR warm-up: every plane holds the step-0 gradient of each partition.
      const size_t plane_bytes = sizeof(float) * static_cast<size_t>(ctx->n) * ctx->ld;
      for (int p = 1; p < plane_count && e == hipSuccess; ++p)
        e = hipMemcpyAsync(reinterpret_cast<char*>(ring) + (plane_first + p) * plane_bytes,
                           reinterpret_cast<char*>(ring) + plane_first * plane_bytes, plane_bytes,
                           hipMemcpyDeviceToDevice, ctx->stream);
      return e;
    });
  if (st == PGC_OK) {
    const pgc::CodeArgs ca = code_args(ctx, dec, w, lr);
    st = timed_launch(ctx, PGC_KERNEL_CODE, "code kernel", [&] { return pgc::launch_code(ca, ctx->stream); });
  }
  return st;
}

}  // namespace

namespace pgc {

size_t linear_partials_bytes(const pgc_ctx* ctx) { return ctx->partials_bytes; }

bool context_is_linear(const pgc_ctx* ctx) { return ctx->configured && is_linear(ctx->cfg.model); }

bool context_is_configured(const pgc_ctx* ctx) { return ctx->configured; }

bool context_has_workspace(const pgc_ctx* ctx) { return ctx->ws != nullptr; }

int set_error(pgc_ctx* ctx, int status, const char* msg) { return fail(ctx, status, msg); }

int step_impl(pgc_ctx* ctx, const void* X, const void* y, float* w, const uint8_t* straggler_mask,
              float lr, float* partials) {
  if (ctx == nullptr) return PGC_EINVAL;
  if (!ctx->configured) return fail(ctx, PGC_ESTATE, "pgc_configure first");
  if (ctx->ws == nullptr) return fail(ctx, PGC_ESTATE, "pgc_bind_workspace first");
  if (!X || !y || !w || !straggler_mask) return fail(ctx, PGC_EINVAL, "null pointer");
  if (!std::isfinite(lr)) return fail(ctx, PGC_EINVAL, "learning rate must be finite");
  pgc::Decode dec;
  std::string err;
  switch (pgc::decode_coefficients(ctx->scheme, ctx->n, ctx->c, ctx->B, straggler_mask, &dec, &err)) {
    case pgc::kDecodeStragglers: return fail(ctx, PGC_ESTRAGGLERS, err);
    case pgc::kDecodeSingular: return fail(ctx, PGC_ESINGULAR, err);
    default: break;
  }
  const int c = ctx->c;
  const bool fr = ctx->scheme == PGC_FR;
  // The warm-up step, and every step of gradient coding, evaluates all slots.
  const bool warm = ctx->t == 0 || !ctx->pipelined;
  const int o = warm ? 0 : pgc::evaluated_slot(ctx->t, c);
  // Evaluated partitions: all at the warm-up; one per FR group (jc + o) or
  // every partition for CR at t >= 1.
  const int32_t part_stride = (fr && !warm) ? c : 1;
  const int32_t part_offset = (fr && !warm) ? o : 0;
  // Ring slot written: FR keeps one slot per partition; CR writes plane o
  // (worker (k - o) mod n holds partition k in slot o), all planes at t = 0.
  const int plane_first = fr ? 0 : o;
  const int plane_count = (!fr && warm) ? c : 1;

  bool aligned16 = false;
  if (ctx->cfg.model == PGC_MLP) {
    if (reinterpret_cast<uintptr_t>(X) % 16 != 0 || reinterpret_cast<uintptr_t>(y) % 4 != 0 ||
        reinterpret_cast<uintptr_t>(w) % 4 != 0)
      return fail(ctx, PGC_EINVAL, "MLP: X must be 16-byte aligned, y and w 4-byte aligned");
  } else {
    aligned16 = reinterpret_cast<uintptr_t>(X) % 16 == 0 && reinterpret_cast<uintptr_t>(w) % 16 == 0;
    if (!pgc::linear_grad_shape(static_cast<int>(ctx->d), aligned16).supported)
      return fail(ctx, PGC_EINVAL, "d = " + std::to_string(ctx->d) +
                                       " needs d % 4 == 0 and 16-byte aligned X and w");
  }
  // A host-side range per step, for profilers that record roctx markers.
  roctxRangePushA(warm ? "pgc_step (warm-up)" : "pgc_step");
  const int st = ctx->cfg.model == PGC_MLP
                     ? mlp_step(ctx, X, y, w, dec, lr, warm, part_stride, part_offset, plane_first, plane_count)
                     : linear_step(ctx, X, y, w, dec, lr, warm, part_stride, part_offset, plane_first, plane_count,
                                   partials ? partials : ws_ptr<float>(ctx, ctx->off_partials));
  roctxRangePop();
  if (st != PGC_OK) return st;
  ctx->t += 1;
  return PGC_OK;
}

}  // namespace pgc

extern "C" {

int pgc_step(pgc_ctx* ctx, const void* X, const void* y, float* w,
             const uint8_t* straggler_mask, float lr) {
  return pgc::step_impl(ctx, X, y, w, straggler_mask, lr, nullptr);
}

namespace {

size_t ring_bytes(const pgc_ctx* ctx) {
  return sizeof(float) * static_cast<size_t>(ctx->planes) * ctx->n * ctx->ld;
}

pgc::StateHeader state_header(const pgc_ctx* ctx) {
  pgc::StateHeader h{};
  h.magic = pgc::kStateMagic;
  h.version = pgc::kStateVersion;
  h.t = ctx->t;
  h.N = ctx->cfg.N;
  h.q = ctx->d;
  h.ld = ctx->ld;
  h.code_seed = ctx->scheme == PGC_CR_REAL ? ctx->cfg.code_seed : 0;
  h.scheme = ctx->scheme;
  h.n = ctx->n;
  h.c = ctx->c;
  h.model = ctx->cfg.model;
  h.d_in = ctx->cfg.d_in;
  h.hidden = ctx->cfg.hidden;
  h.classes = ctx->cfg.classes;
  h.planes = ctx->planes;
  return h;
}

// Checks shared by save and load; the state holds the ring, so a workspace
// must be bound.
int state_args(const pgc_ctx* ctx, const void* dev, size_t bytes) {
  if (ctx == nullptr) return PGC_EINVAL;
  if (!ctx->configured) return fail(ctx, PGC_ESTATE, "pgc_configure first");
  if (ctx->ws == nullptr) return fail(ctx, PGC_ESTATE, "pgc_bind_workspace first");
  if (dev == nullptr) return fail(ctx, PGC_EINVAL, "null state buffer");
  if (reinterpret_cast<uintptr_t>(dev) % 16 != 0) return fail(ctx, PGC_EINVAL, "state buffer must be 16-byte aligned");
  const size_t need = pgc::kStateHeaderBytes + ring_bytes(ctx);
  if (bytes < need) return fail(ctx, PGC_EINVAL, "state buffer too small: need " + std::to_string(need) + " bytes");
  return PGC_OK;
}

}  // namespace

int pgc_state_bytes(const pgc_ctx* ctx, size_t* bytes) {
  if (ctx == nullptr || bytes == nullptr) return PGC_EINVAL;
  if (!ctx->configured) return fail(ctx, PGC_ESTATE, "pgc_configure first");
  *bytes = pgc::kStateHeaderBytes + ring_bytes(ctx);
  return PGC_OK;
}

int pgc_save_state(const pgc_ctx* ctx, void* dev_out, size_t bytes) {
  const int st = state_args(ctx, dev_out, bytes);
  if (st != PGC_OK) return st;
  pgc_ctx* mctx = const_cast<pgc_ctx*>(ctx);
  hipError_t e = pgc::launch_write_state_header(state_header(ctx), dev_out, ctx->stream);
  if (e != hipSuccess) return device_fail(mctx, e, "writing the state header");
  e = hipMemcpyAsync(static_cast<char*>(dev_out) + pgc::kStateHeaderBytes, ctx->ws + ctx->off_ring, ring_bytes(ctx),
                     hipMemcpyDeviceToDevice, ctx->stream);
  return e == hipSuccess ? PGC_OK : device_fail(mctx, e, "copying the ring");
}

int pgc_load_state(pgc_ctx* ctx, const void* dev_in, size_t bytes) {
  const int st = state_args(ctx, dev_in, bytes);
  if (st != PGC_OK) return st;
  pgc::StateHeader h{};
  hipError_t e = hipMemcpyAsync(&h, dev_in, sizeof(h), hipMemcpyDeviceToHost, ctx->stream);
  if (e == hipSuccess) e = hipStreamSynchronize(ctx->stream);
  if (e != hipSuccess) return device_fail(ctx, e, "reading the state header");
  if (h.magic != pgc::kStateMagic || h.version != pgc::kStateVersion)
    return fail(ctx, PGC_EINVAL, "not a saved PGC state (magic or version)");
  pgc::StateHeader mine = state_header(ctx);
  mine.t = h.t;
  if (std::memcmp(&h, &mine, sizeof(h)) != 0)
    return fail(ctx, PGC_EINVAL, "saved state belongs to a different scheme, code or shape");
  if (h.t < 0) return fail(ctx, PGC_EINVAL, "saved state has a negative step counter");
  e = hipMemcpyAsync(ctx->ws + ctx->off_ring, static_cast<const char*>(dev_in) + pgc::kStateHeaderBytes,
                     ring_bytes(ctx), hipMemcpyDeviceToDevice, ctx->stream);
  if (e != hipSuccess) return device_fail(ctx, e, "restoring the ring");
  ctx->t = h.t;
  return PGC_OK;
}

int pgc_read_ring(const pgc_ctx* ctx, int worker, int slot, float* dev_out) {
  if (ctx == nullptr || dev_out == nullptr) return PGC_EINVAL;
  if (ctx->ws == nullptr) return fail(ctx, PGC_ESTATE, "no workspace bound");
  if (worker < 0 || worker >= ctx->n || slot < 0 || slot >= ctx->c)
    return fail(ctx, PGC_EINVAL, "worker or slot out of range");
  const int k = pgc::held_partition(ctx->scheme, ctx->n, ctx->c, worker, slot);
  const int plane = ctx->scheme == PGC_FR ? 0 : slot;
  const float* src = ws_ptr<float>(ctx, ctx->off_ring) + (static_cast<int64_t>(plane) * ctx->n + k) * ctx->ld;
  hipError_t e = hipMemcpyAsync(dev_out, src, sizeof(float) * ctx->d, hipMemcpyDeviceToDevice, ctx->stream);
  return e == hipSuccess ? PGC_OK : device_fail(const_cast<pgc_ctx*>(ctx), e, "hipMemcpyAsync");
}

int pgc_read_coded(const pgc_ctx* ctx, int index, float* dev_out) {
  if (ctx == nullptr || dev_out == nullptr) return PGC_EINVAL;
  if (ctx->ws == nullptr) return fail(ctx, PGC_ESTATE, "no workspace bound");
  if (index < 0 || index >= ctx->n_coded) return fail(ctx, PGC_EINVAL, "coded index out of range");
  const float* src = ws_ptr<float>(ctx, ctx->off_coded) + static_cast<int64_t>(index) * ctx->ld;
  hipError_t e = hipMemcpyAsync(dev_out, src, sizeof(float) * ctx->d, hipMemcpyDeviceToDevice, ctx->stream);
  return e == hipSuccess ? PGC_OK : device_fail(const_cast<pgc_ctx*>(ctx), e, "hipMemcpyAsync");
}

int pgc_read_decoded(const pgc_ctx* ctx, float* dev_out) {
  if (ctx == nullptr || dev_out == nullptr) return PGC_EINVAL;
  if (ctx->ws == nullptr) return fail(ctx, PGC_ESTATE, "no workspace bound");
  hipError_t e = hipMemcpyAsync(dev_out, ws_ptr<float>(ctx, ctx->off_decoded), sizeof(float) * ctx->d,
                                hipMemcpyDeviceToDevice, ctx->stream);
  return e == hipSuccess ? PGC_OK : device_fail(const_cast<pgc_ctx*>(ctx), e, "hipMemcpyAsync");
}

int pgc_set_timing(pgc_ctx* ctx, int kernel_mask) {
  if (ctx == nullptr) return PGC_EINVAL;
  int st = resolve_timing(ctx, true);
  if (st != PGC_OK) return st;
  ctx->timing = static_cast<unsigned>(kernel_mask) & ((1u << PGC_KERNEL_COUNT) - 1u);
  std::fill(ctx->total_ms, ctx->total_ms + PGC_KERNEL_COUNT, 0.0);
  std::fill(ctx->launches, ctx->launches + PGC_KERNEL_COUNT, int64_t{0});
  std::fill(ctx->seen, ctx->seen + PGC_KERNEL_COUNT, int64_t{0});
  return PGC_OK;
}

int pgc_set_timing_period(pgc_ctx* ctx, int64_t period) {
  if (ctx == nullptr) return PGC_EINVAL;
  if (period < 1) return fail(ctx, PGC_EINVAL, "timing period must be >= 1");
  ctx->timing_period = period;
  std::fill(ctx->seen, ctx->seen + PGC_KERNEL_COUNT, int64_t{0});
  return PGC_OK;
}

int pgc_kernel_time(pgc_ctx* ctx, int kernel, double* total_ms, int64_t* launches) {
  if (ctx == nullptr || total_ms == nullptr || launches == nullptr) return PGC_EINVAL;
  if (kernel < 0 || kernel >= PGC_KERNEL_COUNT) return fail(ctx, PGC_EINVAL, "unknown kernel");
  int st = resolve_timing(ctx, true);
  if (st != PGC_OK) return st;
  *total_ms = ctx->total_ms[kernel];
  *launches = ctx->launches[kernel];
  return PGC_OK;
}

}  // extern "C"
