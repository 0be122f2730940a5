/* A plain C99 caller of the PGC C ABI (include/pgc.h): host-only entry points,
 * no GPU work.  Prints one line per result for tests/test_c_abi.py to check. */
#include <stdint.h>
#include <stdio.h>

#include "pgc.h"

static int check(int st, const char* what) {
  if (st != PGC_OK) printf("status %s %d\n", what, st);
  return st;
}

static void print_ints(const char* tag, const int32_t* v, int count) {
  printf("%s", tag);
  for (int i = 0; i < count; ++i) printf(" %d", (int)v[i]);
  printf("\n");
}

int main(void) {
  pgc_ctx* ctx = NULL;
  int32_t ints[64];
  double d[8], scale = 0.0;
  int32_t surv[8], n_surv = 0;
  uint8_t mask[8] = {0};
  size_t bytes = 0;
  uint64_t r = 0;

  /* FR, n = 4, c = 2: placement and schedule (Sec. III, Sec. IV-A). */
  if (check(pgc_init(&ctx, PGC_FR, 4, 2, 16), "init_fr")) return 1;
  pgc_config cfg = {PGC_LOGISTIC, 16, 64, 0, 0, 0};
  if (check(pgc_configure(ctx, &cfg), "configure_fr")) return 1;
  check(pgc_placement(ctx, ints), "placement_fr");
  print_ints("placement_fr", ints, 8);
  check(pgc_schedule(ctx, 2, ints), "schedule_fr");
  print_ints("schedule_fr_t2", ints, 4);
  mask[0] = 1;
  check(pgc_decode_coeffs(ctx, mask, d, &scale, surv, &n_surv), "decode_fr");
  print_ints("survivors_fr", surv, n_surv);
  printf("decode_fr %g %g %g scale %.17g\n", d[0], d[1], d[2], scale);
  check(pgc_workspace_bytes(ctx, &bytes), "workspace_fr");
  printf("workspace_fr %zu\n", bytes);
  /* No workspace bound yet: the step is refused before any device work. */
  const int st_step = pgc_step(ctx, (const void*)16, (const void*)16, (float*)16, mask, 0.1f);
  printf("step_unbound %d %s\n", st_step, pgc_last_error(ctx));
  pgc_destroy(ctx);

  /* CR, n = 5, c = 3, two stragglers: unit weights, scale 1/(|J| c) (Sec. V-B). */
  if (check(pgc_init(&ctx, PGC_CR, 5, 3, 8), "init_cr")) return 1;
  pgc_config cfg_cr = {PGC_LSQ, 8, 40, 0, 0, 0};
  if (check(pgc_configure(ctx, &cfg_cr), "configure_cr")) return 1;
  check(pgc_placement(ctx, ints), "placement_cr");
  print_ints("placement_cr", ints, 15);
  uint8_t mask_cr[5] = {0, 1, 0, 1, 0};
  check(pgc_decode_coeffs(ctx, mask_cr, d, &scale, surv, &n_surv), "decode_cr");
  print_ints("survivors_cr", surv, n_surv);
  printf("decode_cr %g %g %g scale %.17g\n", d[0], d[1], d[2], scale);
  uint8_t mask_bad[5] = {1, 1, 1, 0, 0};
  const int st_bad = pgc_decode_coeffs(ctx, mask_bad, d, &scale, surv, &n_surv);
  printf("too_many %d %s\n", st_bad, pgc_strerror(st_bad));
  pgc_destroy(ctx);

  /* Context-free calls. */
  check(pgc_splitmix64(0, 0, &r), "splitmix");
  printf("splitmix64_0_0 %llu\n", (unsigned long long)r);
  uint8_t m8[8];
  check(pgc_make_mask((5ull << 32) | 1, 3, PGC_POLICY_EXACT, 8, 2, 0.0, m8), "mask");
  for (int i = 0; i < 8; ++i) ints[i] = m8[i];
  print_ints("mask_exact_8_2_t3", ints, 8);
  printf("init_bad %d\n", pgc_init(&ctx, PGC_FR, 6, 4, 8));
  printf("done\n");
  return 0;
}
