// Host-side checks of the C ABI under AddressSanitizer / UndefinedBehavior-
// Sanitizer: argument validation (every rejected call returns AGN_EINVAL and
// hands back no context), the error path of a context that cannot reach a
// device (everything allocated on the host is freed), calls on a NULL
// context, and the temporal efficiency of Eq. 4 (host arithmetic) on curves
// with closed-form areas and on malformed curves.  Built against a
// host-only build of the library; no kernel is launched.
#include <cmath>
#include <cstdio>
#include <cstring>
#include <vector>

#include "agn.h"

static int failures = 0;
#define CHECK(cond)                                                          \
  do {                                                                       \
    if (!(cond)) {                                                           \
      std::fprintf(stderr, "FAIL %s:%d: %s\n", __FILE__, __LINE__, #cond); \
      ++failures;                                                            \
    }                                                                        \
  } while (0)

static int create(int L, const int32_t* dims, int batch, int dtype, int n, int lam, float eta, agn_ctx** out) {
  agn_shapes s{L, dims, batch, dtype};
  return agn_create(&s, n, lam, eta, 7, out);
}

static void rejected(int rc, agn_ctx* c) {
  CHECK(rc == AGN_EINVAL);
  CHECK(c == nullptr);
  const char* msg = agn_last_error(nullptr);
  CHECK(msg != nullptr && std::strlen(msg) > 0);
}

static void check_create() {
  const int32_t dims[3] = {8, 4, 3};
  agn_ctx* c = reinterpret_cast<agn_ctx*>(1);
  agn_shapes s{2, dims, 4, AGN_FP32};
  CHECK(agn_create(&s, 2, 2, 0.1f, 1, nullptr) == AGN_EINVAL);
  c = reinterpret_cast<agn_ctx*>(1);
  rejected(agn_create(nullptr, 2, 2, 0.1f, 1, &c), c);
  c = reinterpret_cast<agn_ctx*>(1);
  rejected(create(0, dims, 4, AGN_FP32, 2, 2, 0.1f, &c), c);
  c = reinterpret_cast<agn_ctx*>(1);
  rejected(create(AGN_MAX_LAYERS + 1, dims, 4, AGN_FP32, 2, 2, 0.1f, &c), c);
  c = reinterpret_cast<agn_ctx*>(1);
  rejected(create(2, nullptr, 4, AGN_FP32, 2, 2, 0.1f, &c), c);
  const int32_t zero_width[3] = {8, 0, 3}, one_class[3] = {8, 4, 1}, huge[3] = {8, (1 << 20) + 1, 3};
  c = reinterpret_cast<agn_ctx*>(1);
  rejected(create(2, zero_width, 4, AGN_FP32, 2, 2, 0.1f, &c), c);
  c = reinterpret_cast<agn_ctx*>(1);
  rejected(create(2, one_class, 4, AGN_FP32, 2, 2, 0.1f, &c), c);
  c = reinterpret_cast<agn_ctx*>(1);
  rejected(create(2, huge, 4, AGN_FP32, 2, 2, 0.1f, &c), c);
  c = reinterpret_cast<agn_ctx*>(1);
  rejected(create(2, dims, 0, AGN_FP32, 2, 2, 0.1f, &c), c);
  c = reinterpret_cast<agn_ctx*>(1);
  rejected(create(2, dims, 4, 2, 2, 2, 0.1f, &c), c);
  c = reinterpret_cast<agn_ctx*>(1);
  rejected(create(2, dims, 4, AGN_FP32, 0, 2, 0.1f, &c), c);
  c = reinterpret_cast<agn_ctx*>(1);
  rejected(create(2, dims, 4, AGN_FP32, AGN_MAX_WORKERS + 1, 2, 0.1f, &c), c);
  c = reinterpret_cast<agn_ctx*>(1);
  rejected(create(2, dims, 4, AGN_FP32, 2, 0, 0.1f, &c), c);
  c = reinterpret_cast<agn_ctx*>(1);
  rejected(create(2, dims, 4, AGN_FP32, 2, 2, std::nanf(""), &c), c);
  c = reinterpret_cast<agn_ctx*>(1);
  rejected(create(2, dims, 4, AGN_FP32, 2, 2, INFINITY, &c), c);

  // valid arguments: a context on a device, or (no device here) AGN_EHIP
  // after the host state is built and freed again
  c = reinterpret_cast<agn_ctx*>(1);
  const int rc = create(2, dims, 4, AGN_FP32, 2, 2, 0.1f, &c);
  if (rc == AGN_OK) {
    CHECK(c != nullptr);
    CHECK(agn_num_params(c) == 8 * 4 + 4 + 4 * 3 + 3);
    agn_destroy(c);
  } else {
    CHECK(rc == AGN_EHIP || rc == AGN_ENOMEM);
    CHECK(c == nullptr);
  }
}

static void check_null_context() {
  float f[4] = {};
  int64_t i64[4] = {};
  CHECK(agn_num_params(nullptr) == -1);
  CHECK(agn_last_error(nullptr) != nullptr);
  CHECK(agn_set_stream(nullptr, nullptr) != AGN_OK);
  CHECK(agn_set_normalization(nullptr, 1) != AGN_OK);
  CHECK(agn_set_staleness_scaling(nullptr, 1) != AGN_OK);
  CHECK(agn_staleness(nullptr, i64) != AGN_OK);
  CHECK(agn_set_optimizer(nullptr, 0, 0.9f, 0.999f, 1e-8f) != AGN_OK);
  CHECK(agn_round(nullptr, nullptr, nullptr) != AGN_OK);
  CHECK(agn_central(nullptr, f) != AGN_OK);
  CHECK(agn_loss(nullptr, f) != AGN_OK);
  CHECK(agn_set_central(nullptr, f) != AGN_OK);
  CHECK(agn_worker_params(nullptr, 0, f) != AGN_OK);
  CHECK(agn_debug_delta(nullptr, 0, f) != AGN_OK);
  CHECK(agn_debug_batch_indices(nullptr, 0, 0, 8, i64) != AGN_OK);
  agn_destroy(nullptr);
}

static void check_temporal_efficiency() {
  double e = 0.0;
  // the same curve: 1
  const double t[4] = {0.0, 1.0, 2.5, 4.0}, f[4] = {0.1, 0.5, 0.7, 0.8};
  CHECK(agn_temporal_efficiency(t, f, 4, t, f, 4, &e) == AGN_OK && e == 1.0);
  // twice the curve: 2
  const double f2[4] = {0.2, 1.0, 1.4, 1.6};
  CHECK(agn_temporal_efficiency(t, f2, 4, t, f, 4, &e) == AGN_OK && std::fabs(e - 2.0) < 1e-15);
  // a = 1 on [0, 2]; b = t on [0, 1], then 1 up to 3: cut at tm = 2,
  // areas 2 and 0.5 + 1 = 1.5
  const double ta[2] = {0.0, 2.0}, fa[2] = {1.0, 1.0}, tb[3] = {0.0, 1.0, 3.0}, fb[3] = {0.0, 1.0, 1.0};
  CHECK(agn_temporal_efficiency(ta, fa, 2, tb, fb, 3, &e) == AGN_OK && std::fabs(e - 4.0 / 3.0) < 1e-15);
  // b cut inside a segment: a = 1 on [0, 1]; b = t on [0, 4]: tm = 1,
  // areas 1 and 1/2
  const double ta2[2] = {0.0, 1.0}, tb2[2] = {0.0, 4.0}, fb2[2] = {0.0, 4.0};
  CHECK(agn_temporal_efficiency(ta2, fa, 2, tb2, fb2, 2, &e) == AGN_OK && std::fabs(e - 2.0) < 1e-15);
  // long curves (the trapezoid rule is exact on lines): a = 3t, b = t
  std::vector<double> tl(10001), fl3(10001), fl1(10001);
  for (int k = 0; k <= 10000; ++k) {
    tl[k] = k * 1e-3;
    fl3[k] = 3.0 * tl[k];
    fl1[k] = tl[k];
  }
  CHECK(agn_temporal_efficiency(tl.data(), fl3.data(), 10001, tl.data(), fl1.data(), 10001, &e) == AGN_OK &&
        std::fabs(e - 3.0) < 1e-12);
  // malformed curves and a zero area of b
  const double t_bad0[2] = {0.5, 1.0}, t_dec[3] = {0.0, 2.0, 1.0}, f_nan[2] = {0.0, NAN}, f0[2] = {0.0, 0.0};
  CHECK(agn_temporal_efficiency(t, f, 1, t, f, 4, &e) == AGN_EINVAL);
  CHECK(agn_temporal_efficiency(t_bad0, fa, 2, t, f, 4, &e) == AGN_EINVAL);
  CHECK(agn_temporal_efficiency(t_dec, fb, 3, t, f, 4, &e) == AGN_EINVAL);
  CHECK(agn_temporal_efficiency(ta, f_nan, 2, t, f, 4, &e) == AGN_EINVAL);
  CHECK(agn_temporal_efficiency(ta, fa, 2, ta, f0, 2, &e) == AGN_EINVAL);
  CHECK(agn_temporal_efficiency(nullptr, fa, 2, ta, fa, 2, &e) == AGN_EINVAL);
  CHECK(agn_temporal_efficiency(ta, fa, 2, ta, fa, 2, nullptr) == AGN_EINVAL);
}

int main() {
  check_create();
  check_null_context();
  check_temporal_efficiency();
  std::printf("host ABI checks: %d failure(s)\n", failures);
  return failures ? 1 : 0;
}
