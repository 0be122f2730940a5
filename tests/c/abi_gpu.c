/* A plain C caller of the PGC step on the GPU: device memory from the HIP C
 * runtime API, no Python and no torch.
 *   abi_gpu SCHEME MODEL n c d N steps lr  in.bin masks.bin  out.bin
 * in.bin: X (N*d fp32), y (N fp32), w0 (d fp32); masks.bin: steps*n bytes.
 * out.bin: per step the decoded gradient then w (2*d fp32 each). */
#include <hip/hip_runtime_api.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include "pgc.h"

#define HIP_OK(call) do { hipError_t e_ = (call); if (e_ != hipSuccess) { \
  fprintf(stderr, "%s: %s\n", #call, hipGetErrorString(e_)); return 2; } } while (0)
#define PGC_OK_OR_FAIL(ctx, call) do { int s_ = (call); if (s_ != PGC_OK) { \
  fprintf(stderr, "%s: %d %s\n", #call, s_, pgc_last_error(ctx)); return 3; } } while (0)

static void* read_all(const char* path, size_t bytes) {
  FILE* f = fopen(path, "rb");
  if (!f) return NULL;
  void* buf = malloc(bytes);
  if (buf && fread(buf, 1, bytes, f) != bytes) { free(buf); buf = NULL; }
  fclose(f);
  return buf;
}

int main(int argc, char** argv) {
  if (argc != 12) { fprintf(stderr, "usage: see the header\n"); return 1; }
  const int scheme = atoi(argv[1]), model = atoi(argv[2]), n = atoi(argv[3]), c = atoi(argv[4]);
  const int d = atoi(argv[5]);
  const long long N = atoll(argv[6]);
  const int steps = atoi(argv[7]);
  const float lr = (float)atof(argv[8]);
  const size_t xb = sizeof(float) * (size_t)N * d, yb = sizeof(float) * (size_t)N, wb = sizeof(float) * d;
  float* in = (float*)read_all(argv[9], xb + yb + wb);
  uint8_t* masks = (uint8_t*)read_all(argv[10], (size_t)steps * n);
  float* out = (float*)malloc(2 * wb * steps);
  if (!in || !masks || !out) { fprintf(stderr, "reading inputs\n"); return 1; }

  void *X, *y, *w, *ghat, *ws;
  HIP_OK(hipMalloc(&X, xb));
  HIP_OK(hipMalloc(&y, yb));
  HIP_OK(hipMalloc(&w, wb));
  HIP_OK(hipMalloc(&ghat, wb));
  HIP_OK(hipMemcpy(X, in, xb, hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(y, (char*)in + xb, yb, hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(w, (char*)in + xb + yb, wb, hipMemcpyHostToDevice));

  pgc_ctx* ctx = NULL;
  if (pgc_init(&ctx, scheme, n, c, d) != PGC_OK) { fprintf(stderr, "pgc_init\n"); return 3; }
  pgc_config cfg = {model, d, N, 0, 0, 0};
  PGC_OK_OR_FAIL(ctx, pgc_configure(ctx, &cfg));
  size_t bytes = 0;
  PGC_OK_OR_FAIL(ctx, pgc_workspace_bytes(ctx, &bytes));
  HIP_OK(hipMalloc(&ws, bytes));
  PGC_OK_OR_FAIL(ctx, pgc_bind_workspace(ctx, ws, bytes));
  for (int t = 0; t < steps; ++t) {
    PGC_OK_OR_FAIL(ctx, pgc_step(ctx, X, y, (float*)w, masks + (size_t)t * n, lr));
    PGC_OK_OR_FAIL(ctx, pgc_read_decoded(ctx, (float*)ghat));
    HIP_OK(hipDeviceSynchronize());
    HIP_OK(hipMemcpy(out + (size_t)2 * d * t, ghat, wb, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(out + (size_t)2 * d * t + d, w, wb, hipMemcpyDeviceToHost));
  }
  pgc_destroy(ctx);
  FILE* f = fopen(argv[11], "wb");
  if (!f || fwrite(out, 1, 2 * wb * steps, f) != 2 * wb * steps) { fprintf(stderr, "writing\n"); return 1; }
  fclose(f);
  HIP_OK(hipFree(X));
  HIP_OK(hipFree(y));
  HIP_OK(hipFree(w));
  HIP_OK(hipFree(ghat));
  HIP_OK(hipFree(ws));
  free(in);
  free(masks);
  free(out);
  printf("ok %d steps\n", steps);
  return 0;
}
