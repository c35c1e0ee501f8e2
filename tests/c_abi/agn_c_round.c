/* A plain C99 user of libagn (test fixture).
 *
 *   agn_c_round validate            argument validation only (no device needed)
 *   agn_c_round run IN OUT          run a workload on the GPU through the C ABI
 *
 * IN (little-endian): int32 L, int32 dims[L+1], int32 m, int32 n,
 * int32 lambda, float32 eta, uint64 seed, int64 N, int32 rounds,
 * float32 X[N][dims[0]], int32 y[N], int32 orders[rounds][n].
 * OUT: per round, float32 central[P] then float32 loss[n].
 *
 * Every call goes through agn.h as a C program sees it: plain pointers and
 * sizes, device buffers from the HIP runtime's C API. */
#include <hip/hip_runtime_api.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "agn.h"

static int failures = 0;
#define CHECK(cond)                                                  \
  do {                                                               \
    if (!(cond)) {                                                   \
      fprintf(stderr, "FAIL %s:%d: %s\n", __FILE__, __LINE__, #cond); \
      ++failures;                                                    \
    }                                                                \
  } while (0)

static void rejected(int rc, agn_ctx* c) {
  const char* msg = agn_last_error(NULL);
  CHECK(rc == AGN_EINVAL);
  CHECK(c == NULL);
  CHECK(msg != NULL && strlen(msg) > 0);
}

static int validate(void) {
  const int32_t dims[3] = {8, 4, 3};
  agn_shapes s;
  agn_ctx* c = NULL;
  double te = 0.0;
  const double t[3] = {0.0, 1.0, 2.0}, f[3] = {1.0, 0.5, 0.25};
  s.num_layers = 2;
  s.dims = dims;
  s.batch = 4;
  s.dtype = AGN_FP32;
  rejected(agn_create(NULL, 2, 2, 0.1f, 1, &c), c);
  s.num_layers = 0;
  rejected(agn_create(&s, 2, 2, 0.1f, 1, &c), c);
  s.num_layers = AGN_MAX_LAYERS + 1;
  rejected(agn_create(&s, 2, 2, 0.1f, 1, &c), c);
  s.num_layers = 2;
  rejected(agn_create(&s, 0, 2, 0.1f, 1, &c), c);
  rejected(agn_create(&s, AGN_MAX_WORKERS + 1, 2, 0.1f, 1, &c), c);
  rejected(agn_create(&s, 2, 0, 0.1f, 1, &c), c);
  s.dtype = 7;
  rejected(agn_create(&s, 2, 2, 0.1f, 1, &c), c);
  CHECK(agn_create(NULL, 2, 2, 0.1f, 1, NULL) == AGN_EINVAL);
  CHECK(agn_num_params(NULL) == -1);
  CHECK(agn_round(NULL, NULL, NULL) == AGN_EINVAL);
  CHECK(agn_central(NULL, NULL) == AGN_EINVAL);
  CHECK(agn_loss(NULL, NULL) == AGN_EINVAL);
  agn_destroy(NULL);
  /* Eq. 4 of two identical curves */
  CHECK(agn_temporal_efficiency(t, f, 3, t, f, 3, &te) == AGN_OK);
  CHECK(te == 1.0);
  printf("%d failure(s)\n", failures);
  return failures ? 1 : 0;
}

static int read_exact(FILE* fp, void* p, size_t bytes) { return fread(p, 1, bytes, fp) == bytes; }

static int run(const char* in_path, const char* out_path) {
  FILE* fp = fopen(in_path, "rb");
  FILE* out = NULL;
  int32_t L = 0, dims[AGN_MAX_LAYERS + 1], m = 0, n = 0, lam = 0, rounds = 0, r;
  float eta = 0.f;
  uint64_t seed = 0;
  int64_t N = 0, P = 0;
  float *x = NULL, *central = NULL, *loss = NULL;
  int32_t *y = NULL, *orders = NULL;
  void *dx = NULL, *dy = NULL, *dc = NULL, *dl = NULL;
  agn_ctx* ctx = NULL;
  agn_shapes s;
  agn_data d;
  int rc = 1;
  if (!fp) return 2;
  if (!read_exact(fp, &L, 4) || L < 1 || L > AGN_MAX_LAYERS || !read_exact(fp, dims, 4 * (size_t)(L + 1)) ||
      !read_exact(fp, &m, 4) || !read_exact(fp, &n, 4) || !read_exact(fp, &lam, 4) || !read_exact(fp, &eta, 4) ||
      !read_exact(fp, &seed, 8) || !read_exact(fp, &N, 8) || !read_exact(fp, &rounds, 4))
    goto done;
  x = (float*)malloc(sizeof(float) * (size_t)N * (size_t)dims[0]);
  y = (int32_t*)malloc(sizeof(int32_t) * (size_t)N);
  orders = (int32_t*)malloc(sizeof(int32_t) * (size_t)rounds * (size_t)n);
  if (!x || !y || !orders) goto done;
  if (!read_exact(fp, x, sizeof(float) * (size_t)N * (size_t)dims[0]) || !read_exact(fp, y, 4 * (size_t)N) ||
      !read_exact(fp, orders, 4 * (size_t)rounds * (size_t)n))
    goto done;
  if (hipMalloc(&dx, sizeof(float) * (size_t)N * (size_t)dims[0]) != hipSuccess ||
      hipMalloc(&dy, 4 * (size_t)N) != hipSuccess)
    goto done;
  if (hipMemcpy(dx, x, sizeof(float) * (size_t)N * (size_t)dims[0], hipMemcpyHostToDevice) != hipSuccess ||
      hipMemcpy(dy, y, 4 * (size_t)N, hipMemcpyHostToDevice) != hipSuccess)
    goto done;
  s.num_layers = L;
  s.dims = dims;
  s.batch = m;
  s.dtype = AGN_FP32;
  if (agn_create(&s, n, lam, eta, seed, &ctx) != AGN_OK) {
    fprintf(stderr, "agn_create: %s\n", agn_last_error(NULL));
    goto done;
  }
  P = agn_num_params(ctx);
  central = (float*)malloc(sizeof(float) * (size_t)P);
  loss = (float*)malloc(sizeof(float) * (size_t)n);
  out = fopen(out_path, "wb");
  if (P <= 0 || !central || !loss || !out) goto done;
  if (hipMalloc(&dc, sizeof(float) * (size_t)P) != hipSuccess || hipMalloc(&dl, sizeof(float) * (size_t)n) != hipSuccess)
    goto done;
  d.x = dx;
  d.y = (const int32_t*)dy;
  d.num_samples = N;
  d.x_dtype = 0;
  for (r = 0; r < rounds; ++r) {
    /* the commit order is a HOST array; agn_central and agn_loss fill
       DEVICE buffers and wait for the context's stream */
    if (agn_round(ctx, &d, orders + (size_t)r * (size_t)n) != AGN_OK || agn_central(ctx, (float*)dc) != AGN_OK ||
        agn_loss(ctx, (float*)dl) != AGN_OK) {
      fprintf(stderr, "round %d: %s\n", (int)r, agn_last_error(ctx));
      goto done;
    }
    if (hipMemcpy(central, dc, sizeof(float) * (size_t)P, hipMemcpyDeviceToHost) != hipSuccess ||
        hipMemcpy(loss, dl, sizeof(float) * (size_t)n, hipMemcpyDeviceToHost) != hipSuccess)
      goto done;
    if (fwrite(central, sizeof(float), (size_t)P, out) != (size_t)P || fwrite(loss, sizeof(float), (size_t)n, out) != (size_t)n)
      goto done;
  }
  rc = 0;
done:
  if (out) fclose(out);
  agn_destroy(ctx);
  if (dx) (void)hipFree(dx);
  if (dy) (void)hipFree(dy);
  if (dc) (void)hipFree(dc);
  if (dl) (void)hipFree(dl);
  free(x);
  free(y);
  free(orders);
  free(central);
  free(loss);
  fclose(fp);
  return rc;
}

int main(int argc, char** argv) {
  if (argc == 2 && strcmp(argv[1], "validate") == 0) return validate();
  if (argc == 4 && strcmp(argv[1], "run") == 0) return run(argv[2], argv[3]);
  fprintf(stderr, "usage: agn_c_round validate | run IN OUT\n");
  return 2;
}
