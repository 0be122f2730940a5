// C ABI of the PGC step (include/pgc.h): context, validation, workspace
// layout and the per-step launch sequence.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cstring>
#include <string>
#include <vector>

#include "pgc.h"
#include "pgc_codes.h"
#include "pgc_kernels.h"

namespace {

constexpr size_t kAlign = 256;
// Gradient grid: about this many blocks per launch (>= 4 per CU on 256 CUs),
// never fewer than kMinRowsPerBlock rows per block.  The grid depends only on
// the problem shape, so results do not depend on the device.
constexpr int64_t kTargetBlocks = 1024;
constexpr int64_t kMinRowsPerBlock = 16;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

struct Grid {
  int32_t n_eval = 0;
  int32_t blocks_per_part = 0;
  int64_t rows_per_block = 0;
};

Grid make_grid(int64_t m, int32_t n_eval) {
  Grid g;
  g.n_eval = n_eval;
  int64_t b = (kTargetBlocks + n_eval - 1) / n_eval;
  b = std::max<int64_t>(1, std::min<int64_t>(b, (m + kMinRowsPerBlock - 1) / kMinRowsPerBlock));
  g.rows_per_block = (m + b - 1) / b;
  g.blocks_per_part = static_cast<int32_t>((m + g.rows_per_block - 1) / g.rows_per_block);
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
  Grid warm, pipe;
  size_t off_ring = 0, off_coded = 0, off_decoded = 0, off_partials = 0, off_coef = 0, ws_need = 0;
  char* ws = nullptr;
  size_t ws_bytes = 0;
  hipStream_t stream = nullptr;
  int64_t t = 0;
  std::string err;
  bool timing = false;
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
  ctx->planes = ctx->scheme == PGC_FR ? 1 : ctx->c;
  ctx->n_coded = ctx->scheme == PGC_FR ? ctx->n / ctx->c : ctx->n;
  ctx->warm = make_grid(ctx->m, ctx->n);
  ctx->pipe = make_grid(ctx->m, ctx->scheme == PGC_FR ? ctx->n / ctx->c : ctx->n);
  const int64_t max_blocks =
      std::max<int64_t>(static_cast<int64_t>(ctx->warm.n_eval) * ctx->warm.blocks_per_part,
                        static_cast<int64_t>(ctx->pipe.n_eval) * ctx->pipe.blocks_per_part);
  size_t off = 0;
  ctx->off_ring = off;
  off = align_up(off + sizeof(float) * static_cast<size_t>(ctx->planes) * ctx->n * q);
  ctx->off_coded = off;
  off = align_up(off + sizeof(float) * static_cast<size_t>(ctx->n_coded) * q);
  ctx->off_decoded = off;
  off = align_up(off + sizeof(float) * static_cast<size_t>(q));
  ctx->off_partials = off;
  off = align_up(off + sizeof(float) * static_cast<size_t>(max_blocks) * q);
  ctx->off_coef = off;
  off = align_up(off + sizeof(double) * ctx->coef.size());
  ctx->ws_need = off;
}

template <class T>
T* ws_ptr(const pgc_ctx* ctx, size_t off) {
  return reinterpret_cast<T*>(ctx->ws + off);
}

// Resolve recorded kernel events whose work has completed, or all of them.
int resolve_timing(pgc_ctx* ctx, bool wait) {
  size_t done = 0;
  for (; done < ctx->pending.size(); ++done) {
    Timed& tm = ctx->pending[done];
    if (wait) {
      hipError_t e = hipEventSynchronize(tm.stop);
      if (e != hipSuccess) return device_fail(ctx, e, "hipEventSynchronize");
    } else if (hipEventQuery(tm.stop) != hipSuccess) {
      break;
    }
    float ms = 0.f;
    hipError_t e = hipEventElapsedTime(&ms, tm.start, tm.stop);
    if (e != hipSuccess) return device_fail(ctx, e, "hipEventElapsedTime");
    ctx->total_ms[tm.kernel] += ms;
    ctx->launches[tm.kernel] += 1;
    ctx->spare.push_back(tm);
  }
  ctx->pending.erase(ctx->pending.begin(), ctx->pending.begin() + done);
  return PGC_OK;
}

// Launch `fn` on the context stream, bracketed by events when timing is on.
template <class Fn>
int timed_launch(pgc_ctx* ctx, int kernel, const char* what, Fn fn) {
  Timed tm;
  if (ctx->timing) {
    if (ctx->pending.size() >= 4096) {
      int st = resolve_timing(ctx, false);
      if (st != PGC_OK) return st;
    }
    if (!ctx->spare.empty()) {
      tm = ctx->spare.back();
      ctx->spare.pop_back();
    } else {
      hipError_t e = hipEventCreate(&tm.start);
      if (e == hipSuccess) e = hipEventCreate(&tm.stop);
      if (e != hipSuccess) return device_fail(ctx, e, "hipEventCreate");
    }
    tm.kernel = kernel;
    hipError_t e = hipEventRecord(tm.start, ctx->stream);
    if (e != hipSuccess) return device_fail(ctx, e, "hipEventRecord");
  }
  hipError_t e = fn();
  if (e != hipSuccess) return device_fail(ctx, e, what);
  if (ctx->timing) {
    e = hipEventRecord(tm.stop, ctx->stream);
    if (e != hipSuccess) return device_fail(ctx, e, "hipEventRecord");
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
  if (scheme != PGC_FR && scheme != PGC_CR && scheme != PGC_CR_REAL) return PGC_EINVAL;
  if (n < 1 || n > PGC_MAX_N || c < 1 || c > n || d < 1) return PGC_EINVAL;
  if (scheme == PGC_FR && n % c != 0) return PGC_EINVAL;
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
    return fail(ctx, PGC_EINVAL, "the MLP model is not available in this build");
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

int pgc_set_stream(pgc_ctx* ctx, void* hip_stream) {
  if (ctx == nullptr) return PGC_EINVAL;
  ctx->stream = static_cast<hipStream_t>(hip_stream);
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
  ctx->ws = static_cast<char*>(dev_workspace);
  ctx->ws_bytes = bytes;
  ctx->t = 0;
  if (!ctx->coef.empty()) {
    hipError_t e = hipMemcpy(ctx->ws + ctx->off_coef, ctx->coef.data(),
                             sizeof(double) * ctx->coef.size(), hipMemcpyHostToDevice);
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

int pgc_step(pgc_ctx* ctx, const void* X, const void* y, float* w,
             const uint8_t* straggler_mask, float lr) {
  if (ctx == nullptr) return PGC_EINVAL;
  if (!ctx->configured) return fail(ctx, PGC_ESTATE, "pgc_configure first");
  if (ctx->ws == nullptr) return fail(ctx, PGC_ESTATE, "pgc_bind_workspace first");
  if (!X || !y || !w || !straggler_mask) return fail(ctx, PGC_EINVAL, "null pointer");
  pgc::Decode dec;
  std::string err;
  switch (pgc::decode_coefficients(ctx->scheme, ctx->n, ctx->c, ctx->B, straggler_mask, &dec, &err)) {
    case pgc::kDecodeStragglers: return fail(ctx, PGC_ESTRAGGLERS, err);
    case pgc::kDecodeSingular: return fail(ctx, PGC_ESINGULAR, err);
    default: break;
  }
  const int n = ctx->n, c = ctx->c;
  const int64_t q = ctx->d;
  const bool fr = ctx->scheme == PGC_FR;
  const bool warm = ctx->t == 0;
  const Grid& grid = warm ? ctx->warm : ctx->pipe;
  const int o = warm ? 0 : pgc::evaluated_slot(ctx->t, c);

  // a4: per-partition gradients of the evaluated partitions.
  pgc::LinearGradArgs ga{};
  ga.X = static_cast<const float*>(X);
  ga.y = static_cast<const float*>(y);
  ga.w = w;
  ga.partials = ws_ptr<float>(ctx, ctx->off_partials);
  ga.m = ctx->m;
  ga.rows_per_block = grid.rows_per_block;
  ga.d = static_cast<int32_t>(q);
  ga.blocks_per_part = grid.blocks_per_part;
  ga.n_eval = grid.n_eval;
  ga.part_stride = (fr && !warm) ? c : 1;     // FR evaluates one partition per group
  ga.part_offset = (fr && !warm) ? o : 0;
  ga.model = ctx->cfg.model;
  const bool aligned16 = reinterpret_cast<uintptr_t>(X) % 16 == 0 &&
                         reinterpret_cast<uintptr_t>(w) % 16 == 0;
  const pgc::LinearGradShape shape = pgc::linear_grad_shape(ga.d, aligned16);
  if (!shape.supported)
    return fail(ctx, PGC_EINVAL, "d = " + std::to_string(q) + " needs d % 4 == 0 and 16-byte aligned X and w");

  // a5: ring write.  FR keeps one slot per partition; CR keeps plane o of
  // partition k as the copy held by worker (k - o) mod n in slot o.
  pgc::ReduceArgs ra{};
  ra.partials = ga.partials;
  ra.ring = ws_ptr<float>(ctx, ctx->off_ring);
  ra.q = q;
  ra.inv_m = 1.0 / static_cast<double>(ctx->m);
  ra.n = n;
  ra.n_eval = grid.n_eval;
  ra.blocks_per_part = grid.blocks_per_part;
  ra.part_stride = ga.part_stride;
  ra.part_offset = ga.part_offset;
  ra.plane_first = fr ? 0 : o;
  ra.plane_count = (!fr && warm) ? c : 1;

  // a6-a8: encode, masked decode, update.
  pgc::CodeArgs ca{};
  ca.ring = ra.ring;
  ca.coded = ws_ptr<float>(ctx, ctx->off_coded);
  ca.decoded = ws_ptr<float>(ctx, ctx->off_decoded);
  ca.w = w;
  ca.coef = ctx->coef.empty() ? nullptr : ws_ptr<double>(ctx, ctx->off_coef);
  ca.q = q;
  ca.lr = static_cast<double>(lr);
  ca.n = n;
  ca.c = c;
  ca.n_coded = ctx->n_coded;
  ca.fr = fr ? 1 : 0;
  for (size_t m = 0; m < dec.survivors.size(); ++m) {
    if (dec.d[m] == 0.0) continue;
    const int j = fr ? dec.survivors[m] / c : dec.survivors[m];
    ca.a[j] = dec.scale * dec.d[m];
  }

  int st = timed_launch(ctx, PGC_KERNEL_GRADIENT, "gradient kernel",
                        [&] { return pgc::launch_linear_gradient(ga, aligned16, ctx->stream); });
  if (st != PGC_OK) return st;
  st = timed_launch(ctx, PGC_KERNEL_REDUCE, "reduce kernel",
                    [&] { return pgc::launch_reduce(ra, ctx->stream); });
  if (st != PGC_OK) return st;
  st = timed_launch(ctx, PGC_KERNEL_CODE, "code kernel",
                    [&] { return pgc::launch_code(ca, ctx->stream); });
  if (st != PGC_OK) return st;
  ctx->t += 1;
  return PGC_OK;
}

int pgc_read_ring(const pgc_ctx* ctx, int worker, int slot, float* dev_out) {
  if (ctx == nullptr || dev_out == nullptr) return PGC_EINVAL;
  if (ctx->ws == nullptr) return fail(ctx, PGC_ESTATE, "no workspace bound");
  if (worker < 0 || worker >= ctx->n || slot < 0 || slot >= ctx->c)
    return fail(ctx, PGC_EINVAL, "worker or slot out of range");
  const int k = pgc::held_partition(ctx->scheme, ctx->n, ctx->c, worker, slot);
  const int plane = ctx->scheme == PGC_FR ? 0 : slot;
  const float* src = ws_ptr<float>(ctx, ctx->off_ring) + (static_cast<int64_t>(plane) * ctx->n + k) * ctx->d;
  hipError_t e = hipMemcpyAsync(dev_out, src, sizeof(float) * ctx->d, hipMemcpyDeviceToDevice, ctx->stream);
  return e == hipSuccess ? PGC_OK : device_fail(const_cast<pgc_ctx*>(ctx), e, "hipMemcpyAsync");
}

int pgc_read_coded(const pgc_ctx* ctx, int index, float* dev_out) {
  if (ctx == nullptr || dev_out == nullptr) return PGC_EINVAL;
  if (ctx->ws == nullptr) return fail(ctx, PGC_ESTATE, "no workspace bound");
  if (index < 0 || index >= ctx->n_coded) return fail(ctx, PGC_EINVAL, "coded index out of range");
  const float* src = ws_ptr<float>(ctx, ctx->off_coded) + static_cast<int64_t>(index) * ctx->d;
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

int pgc_set_timing(pgc_ctx* ctx, int enable) {
  if (ctx == nullptr) return PGC_EINVAL;
  int st = resolve_timing(ctx, true);
  if (st != PGC_OK) return st;
  ctx->timing = enable != 0;
  std::fill(ctx->total_ms, ctx->total_ms + PGC_KERNEL_COUNT, 0.0);
  std::fill(ctx->launches, ctx->launches + PGC_KERNEL_COUNT, int64_t{0});
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
