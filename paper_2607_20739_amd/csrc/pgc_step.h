// The step of include/pgc.h with the gradient kernel's block partial sums at a
// caller-chosen device address.  Internal to the library.
#pragma once

#include <cstddef>
#include <cstdint>

#include "pgc.h"

namespace pgc {

// pgc_step with the linear models' block partials at `partials` (device; at
// least linear_partials_bytes(ctx) bytes), or in the bound workspace when
// `partials` is null.  Same checks, errors and effects as pgc_step.
int step_impl(pgc_ctx* ctx, const void* X, const void* y, float* w, const uint8_t* straggler_mask,
              float lr, float* partials);

// Bytes of block partial sums a linear-model step of the configured context
// writes at most (the larger of the warm-up and pipelined gradient grids).
size_t linear_partials_bytes(const pgc_ctx* ctx);

bool context_is_configured(const pgc_ctx* ctx);
bool context_has_workspace(const pgc_ctx* ctx);
bool context_is_linear(const pgc_ctx* ctx);

// Records `msg` as the context's last error and returns `status`.
int set_error(pgc_ctx* ctx, int status, const char* msg);

}  // namespace pgc
