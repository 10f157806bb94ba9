// Host-side driver of the tkef C ABI for AddressSanitizer / UndefinedBehavior-
// Sanitizer builds of the library's host code (built with the sanitizers on
// the host side only; the GPU code is not instrumented and never launched).
// Every call here either fails its argument checks before any HIP call or,
// on a machine without a GPU, reaches the HIP runtime, which reports that no
// device is present (TKEF_EHIP), so the error paths that release host memory
// run too. The calls of the second kind pass made-up device addresses, so
// they are made only when the runtime sees no device. Exit status: the
// number of failed checks.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <limits>
#include <vector>

#include "tkef.h"

static int g_fail = 0;
static bool g_no_gpu = false;  // calls that pass every check are made only then

#define CHECK(expr)                                                     \
  do {                                                                  \
    if (!(expr)) {                                                      \
      std::fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #expr); \
      ++g_fail;                                                         \
    }                                                                   \
  } while (0)

static void helpers() {
  CHECK(tkef_version() == TKEF_VERSION);
  for (int c = -8; c <= 1; ++c) CHECK(tkef_strerror(c) != nullptr);
  CHECK(tkef_k_from_rho(1 << 20, 0.001) == 1049);
  CHECK(tkef_k_from_rho(0, 0.5) == 0);
  CHECK(tkef_k_from_rho(3, 1e-9) == 1);
  CHECK(tkef_k_from_rho(10, 0.0) == TKEF_ERANGE);
  CHECK(tkef_k_from_rho(10, std::nan("")) == TKEF_ERANGE);
  CHECK(tkef_k_from_rho(10, std::numeric_limits<double>::infinity()) == TKEF_ERANGE);
  CHECK(tkef_k_from_rho(-1, 0.5) < 0);
  CHECK(tkef_k_from_rho(INT64_MAX, 0.5) == (int64_t)1 << 62);
  CHECK(tkef_k_from_rho(INT64_MAX, 1.0) == INT64_MAX);  // rho * d rounds to 2^63
  CHECK(tkef_k_from_rho(INT64_MAX, 1.0 - 1e-16) == INT64_MAX - 1023);  // (1 - 2^-53) 2^63
}

static void sparsify_plans() {
  struct Case {
    std::vector<int64_t> n;
    int32_t mode;
    double rho;
    int64_t k;
    int expect;
  };
  std::vector<int64_t> many(5000, 37);
  many[17] = 0;
  std::vector<int64_t> tiles(1 << 17, 4096);
  tiles.resize(1 << 18, 1);  // exactly 2^18 tiles
  std::vector<int64_t> over = tiles;
  over.push_back(1);         // one tile too many
  const std::vector<Case> cases = {
      {{10, 20}, TKEF_GLOBAL, 0.01, 0, TKEF_OK},
      {{10, 20}, TKEF_PER_TENSOR, 0.01, 0, TKEF_OK},
      {{10, 20}, TKEF_APPROX, 0.01, 0, TKEF_OK},
      {{2147483647}, TKEF_GLOBAL, 0.001, 0, TKEF_OK},
      {{2147483647}, TKEF_PER_TENSOR, 0.01, 0, TKEF_OK},
      {{2147483648LL}, TKEF_GLOBAL, 0.01, 0, TKEF_ERANGE},
      {{1LL << 30, 1LL << 30}, TKEF_GLOBAL, 0.01, 0, TKEF_ERANGE},
      {{0, 0}, TKEF_GLOBAL, 0.01, 0, TKEF_ERANGE},
      {{10, -1}, TKEF_GLOBAL, 0.01, 0, TKEF_EINVAL},
      {{10}, 7, 0.01, 0, TKEF_EINVAL},
      {{10}, TKEF_GLOBAL, 0.0, 0, TKEF_ERANGE},
      {{10}, TKEF_GLOBAL, 1.5, 0, TKEF_ERANGE},
      {{10}, TKEF_GLOBAL, 0.0, 10, TKEF_OK},
      {{10}, TKEF_GLOBAL, 0.0, 11, TKEF_ERANGE},
      {{10}, TKEF_GLOBAL, 0.5, -1, TKEF_ERANGE},
      {{10}, TKEF_PER_TENSOR, 0.0, 3, TKEF_EINVAL},
      {many, TKEF_PER_TENSOR, 0.01, 0, TKEF_OK},
      {many, TKEF_GLOBAL, 0.01, 0, TKEF_OK},
      {tiles, TKEF_GLOBAL, 0.001, 0, TKEF_OK},
      {tiles, TKEF_APPROX, 0.001, 0, TKEF_OK},
      {over, TKEF_GLOBAL, 0.001, 0, TKEF_ERANGE},
      {over, TKEF_PER_TENSOR, 0.001, 0, TKEF_ERANGE},
  };
  for (const Case& c : cases) {
    tkef_sparsify_plan p = nullptr;
    const int rc = tkef_sparsify_plan_create(c.n.data(), (int32_t)c.n.size(), c.mode, c.rho, c.k,
                                             &p);
    if (rc != c.expect) {
      std::fprintf(stderr, "create: %zu tensors mode %d rho %g k %lld -> %d, expected %d\n",
                   c.n.size(), c.mode, c.rho, (long long)c.k, rc, c.expect);
      ++g_fail;
    }
    size_t ws = 0, ws2 = 0;
    int64_t kt = 0, kt2 = 0;
    const int wrc = tkef_sparsify_workspace(c.n.data(), (int32_t)c.n.size(), c.mode, c.rho, c.k,
                                            &ws2, &kt2);
    CHECK(wrc == c.expect);
    if (rc != TKEF_OK) continue;
    int64_t d = 0;
    int32_t ng = 0, nl = 0;
    CHECK(tkef_sparsify_plan_info(p, &ws, &kt, &d, &ng, &nl) == TKEF_OK);
    CHECK(ws == ws2 && kt == kt2 && ws > 0 && kt > 0 && nl > 0);
    CHECK(ng == (c.mode == TKEF_PER_TENSOR ? (int32_t)c.n.size() : 1));
    std::vector<int64_t> gk(ng > 0 ? ng : 1);
    CHECK(tkef_sparsify_plan_group_k(p, gk.data(), ng) == TKEF_OK);
    int64_t sum = 0;
    for (int32_t i = 0; i < ng; ++i) sum += gk[i];
    CHECK(sum == kt);
    CHECK(tkef_sparsify_plan_group_k(p, gk.data(), ng - 1) != TKEF_OK || ng == 0);
    for (int32_t i = -1; i <= nl; ++i) {
      const char* name = tkef_sparsify_plan_launch_name(p, i);
      CHECK((name != nullptr) == (i >= 0 && i < nl));
    }
    CHECK(tkef_sparsify_plan_set_value_format(p, TKEF_VAL_F16) == TKEF_OK);
    CHECK(tkef_sparsify_plan_set_value_format(p, 5) == TKEF_EINVAL);
    CHECK(tkef_sparsify_plan_set_approx(p, 30, 12345) ==
          (c.mode == TKEF_APPROX ? TKEF_OK : TKEF_EINVAL));
    CHECK(tkef_sparsify_plan_set_approx(p, 0, 0) == TKEF_EINVAL);
    CHECK(tkef_sparsify_plan_set_approx(p, 49, 0) == TKEF_EINVAL);
    CHECK(tkef_sparsify_plan_set_events(p, nullptr, 0) == TKEF_OK);
    // bind / execute argument checks (no GPU work is reached)
    CHECK(tkef_sparsify_plan_bind(p, nullptr, nullptr, nullptr, 0, nullptr) != TKEF_OK);
    CHECK(tkef_sparsify_execute(p, nullptr, 0, nullptr, nullptr, nullptr, nullptr) != TKEF_OK);
    CHECK(tkef_sparsify_execute(p, reinterpret_cast<void*>(0x10000), ws, nullptr, nullptr,
                                nullptr, nullptr) != TKEF_OK);
    CHECK(tkef_sparsify_plan_destroy(p) == TKEF_OK);
  }
  CHECK(tkef_sparsify_plan_create(nullptr, 2, TKEF_GLOBAL, 0.1, 0, nullptr) == TKEF_EINVAL);
}

static void sparsify_oneshots() {
  const int64_t n[2] = {1000, 24};
  float* fake = reinterpret_cast<float*>(0x100000);
  const float* g[2] = {fake, fake + 2000};
  float* r[2] = {fake + 4000, fake + 6000};
  int64_t counts[2] = {-7, -7};
  // a null workspace is rejected after the counts are written
  CHECK(tkef_sparsify(g, r, n, 2, TKEF_PER_TENSOR, 0.01, 0, TKEF_VAL_F32,
                      reinterpret_cast<int32_t*>(fake + 8000), fake + 9000, counts, nullptr, 0,
                      nullptr, nullptr) == TKEF_EWORKSPACE);
  CHECK(counts[0] == 10 && counts[1] == 1);
  CHECK(tkef_sparsify(nullptr, r, n, 2, TKEF_GLOBAL, 0.01, 0, TKEF_VAL_F32, nullptr, nullptr,
                      nullptr, nullptr, 0, nullptr, nullptr) == TKEF_EINVAL);
  CHECK(tkef_sparsify(g, r, n, 2, TKEF_GLOBAL, 0.01, 0, 9, reinterpret_cast<int32_t*>(fake),
                      fake, nullptr, reinterpret_cast<void*>(0x200000), 1 << 30, nullptr,
                      nullptr) == TKEF_EINVAL);
  // overlapping g and r
  const float* g_ov[1] = {fake};
  float* r_ov[1] = {fake + 10};
  const int64_t n1[1] = {100};
  CHECK(tkef_sparsify(g_ov, r_ov, n1, 1, TKEF_GLOBAL, 0.1, 0, TKEF_VAL_F32,
                      reinterpret_cast<int32_t*>(fake + 5000), fake + 6000, nullptr,
                      reinterpret_cast<void*>(0x200000), 1 << 30, nullptr,
                      nullptr) == TKEF_EINVAL);
  CHECK(tkef_sparsify1(fake, fake + 100, 100, 0, reinterpret_cast<int32_t*>(fake + 300),
                       fake + 400, reinterpret_cast<void*>(0x200000), 1 << 30, nullptr,
                       nullptr) == TKEF_ERANGE);
  CHECK(tkef_sparsify1(fake, fake + 100, 100, 101, reinterpret_cast<int32_t*>(fake + 300),
                       fake + 400, reinterpret_cast<void*>(0x200000), 1 << 30, nullptr,
                       nullptr) == TKEF_ERANGE);
  CHECK(tkef_sparsify1(fake, fake + 100, 0, 1, nullptr, nullptr, nullptr, 0, nullptr,
                       nullptr) == TKEF_ERANGE);
  CHECK(tkef_sparsify1_static(fake, fake + 100, TKEF_STATIC_MAX_D + 1, 5,
                              reinterpret_cast<int32_t*>(fake), fake, nullptr,
                              nullptr) == TKEF_ERANGE);
  CHECK(tkef_sparsify1_static(fake, fake + 100, 1000, TKEF_STATIC_MAX_K + 1,
                              reinterpret_cast<int32_t*>(fake), fake, nullptr,
                              nullptr) == TKEF_ERANGE);
  CHECK(tkef_sparsify1_static(fake, fake + 100, 100, 0, reinterpret_cast<int32_t*>(fake), fake,
                              nullptr, nullptr) == TKEF_ERANGE);
  CHECK(tkef_sparsify1_static(nullptr, fake + 100, 100, 5, reinterpret_cast<int32_t*>(fake),
                              fake, nullptr, nullptr) == TKEF_EINVAL);
  // a valid call on a machine without a GPU: the HIP runtime reports it
  if (g_no_gpu)
    CHECK(tkef_sparsify1_static(fake, fake + 1000, 100, 5,
                                reinterpret_cast<int32_t*>(fake + 2000), fake + 3000, nullptr,
                                nullptr) == TKEF_EHIP);
}

static void update_plans() {
  const int64_t n[3] = {10, 0, 20};
  tkef_update_plan p = nullptr;
  CHECK(tkef_update_plan_create(n, 3, 4, 5, &p) == TKEF_OK);
  size_t ws = 0, ws2 = 0;
  int64_t d = 0;
  int32_t nl = 0;
  CHECK(tkef_update_plan_info(p, &ws, &d, &nl) == TKEF_OK);
  CHECK(d == 30 && ws > 0 && nl == 2);
  CHECK(tkef_update_workspace(n, 3, 4, 5, &ws2) == TKEF_OK && ws2 == ws);
  for (int32_t i = -1; i <= nl; ++i)
    CHECK((tkef_update_plan_launch_name(p, i) != nullptr) == (i >= 0 && i < nl));
  for (int32_t i = -1; i <= 4; ++i) {
    CHECK((tkef_lars_launch_name(0, i) != nullptr) == (i >= 0 && i < 4));
    CHECK((tkef_lars_launch_name(1, i) != nullptr) == (i >= 0 && i < 2));
  }
  CHECK(tkef_lars_launch_name(2, 0) == nullptr);
  CHECK(tkef_update_plan_set_value_format(p, TKEF_VAL_F16) == TKEF_OK);
  CHECK(tkef_update_plan_set_value_format(p, 3) == TKEF_EINVAL);
  CHECK(tkef_update_plan_set_deterministic(p, 1) == TKEF_OK);
  CHECK(tkef_update_plan_set_deterministic(p, -1) == TKEF_EINVAL);
  CHECK(tkef_update_plan_set_events(p, nullptr, 0) == TKEF_OK);
  float* fake = reinterpret_cast<float*>(0x100000);
  float* w[3] = {fake, nullptr, fake + 100};
  float* b_ov[3] = {fake + 4, nullptr, fake + 300};
  float* b[3] = {fake + 200, nullptr, fake + 300};
  void* wsp = reinterpret_cast<void*>(0x400000);
  CHECK(tkef_update_plan_bind(p, w, b_ov, wsp, ws, nullptr) == TKEF_EINVAL);   // w, b overlap
  CHECK(tkef_update_plan_bind(p, nullptr, b, wsp, ws, nullptr) == TKEF_EINVAL);
  CHECK(tkef_update_plan_bind(p, w, b, reinterpret_cast<void*>(0x400010), ws, nullptr) ==
        TKEF_EWORKSPACE);                                                       // misaligned
  CHECK(tkef_update_plan_bind(p, w, b, wsp, ws - 1, nullptr) == TKEF_EWORKSPACE);
  const int32_t* idx = reinterpret_cast<const int32_t*>(0x500000);
  CHECK(tkef_update_execute(p, idx, fake, nullptr, 0.1f, 0.0f, 0.0f, wsp, ws, nullptr,
                            nullptr) == TKEF_ESTATE);                           // not bound
  CHECK(tkef_update_execute(p, idx, fake, nullptr, std::nanf(""), 0.0f, 0.0f, wsp, ws, nullptr,
                            nullptr) == TKEF_ERANGE);
  CHECK(tkef_lars_update_execute(p, idx, fake, nullptr, 0.001, 0.1, -1.0, 0.0f, nullptr, wsp, ws,
                                 nullptr, nullptr) == TKEF_ERANGE);
  CHECK(tkef_lars_update_execute(p, idx, fake, nullptr, INFINITY, 0.1, 0.0, 0.0f, nullptr, wsp,
                                 ws, nullptr, nullptr) == TKEF_ERANGE);
  CHECK(tkef_lars_rates_execute(p, 0.001, 0.1, 1e-4, reinterpret_cast<double*>(fake), wsp, ws,
                                nullptr) != TKEF_OK);
  // a bind that passes every check reaches the HIP runtime (no GPU here)
  if (g_no_gpu) CHECK(tkef_update_plan_bind(p, w, b, wsp, ws, nullptr) == TKEF_EHIP);
  CHECK(tkef_update_plan_destroy(p) == TKEF_OK);

  CHECK(tkef_update_plan_create(n, 3, 0, 5, &p) == TKEF_EINVAL);
  CHECK(tkef_update_plan_create(n, 3, 65536, 5, &p) == TKEF_EINVAL);
  CHECK(tkef_update_plan_create(n, 3, 4, -1, &p) == TKEF_ERANGE);
  CHECK(tkef_update_plan_create(n, 3, 65535, 2147483647LL, &p) == TKEF_ERANGE);
  CHECK(tkef_update_plan_create(n, 3, 512, 2147483647LL, &p) == TKEF_OK);
  CHECK(tkef_update_plan_destroy(p) == TKEF_OK);
  const int64_t big[1] = {2147483647LL};
  CHECK(tkef_update_plan_create(big, 1, 128, 25600, &p) == TKEF_OK);
  CHECK(tkef_update_plan_info(p, &ws, &d, &nl) == TKEF_OK && d == 2147483647LL);
  CHECK(tkef_update_plan_destroy(p) == TKEF_OK);
  CHECK(tkef_update_plan_create(nullptr, 3, 4, 5, &p) == TKEF_EINVAL);
}

static void aggregate_oneshots() {
  const int64_t n[2] = {100, 50};
  size_t ws = 0;
  CHECK(tkef_aggregate_workspace(n, 2, 3, &ws) == TKEF_OK && ws > 0);
  CHECK(tkef_aggregate_workspace(n, 2, 0, &ws) == TKEF_EINVAL);
  CHECK(tkef_aggregate_workspace(nullptr, 2, 3, &ws) == TKEF_EINVAL);
  float* fake = reinterpret_cast<float*>(0x100000);
  float* w[2] = {fake, fake + 1000};
  const int32_t* idx[3] = {reinterpret_cast<const int32_t*>(0x300000), nullptr,
                           reinterpret_cast<const int32_t*>(0x310000)};
  const float* val[3] = {fake + 5000, nullptr, fake + 6000};
  int64_t nnz[3] = {10, 0, 5};
  void* wsp = reinterpret_cast<void*>(0x400000);
  nnz[2] = -1;
  CHECK(tkef_aggregate_update(w, nullptr, n, 2, idx, val, nnz, 3, 0.1f, 0.0f, 0.0f, wsp, ws,
                              nullptr, nullptr) == TKEF_EINVAL);
  nnz[2] = 5;
  nnz[1] = 3;  // a non-empty list with null pointers
  CHECK(tkef_aggregate_update(w, nullptr, n, 2, idx, val, nnz, 3, 0.1f, 0.0f, 0.0f, wsp, ws,
                              nullptr, nullptr) == TKEF_EINVAL);
  nnz[1] = 0;
  CHECK(tkef_aggregate_update(w, nullptr, n, 2, idx, val, nnz, 3, 0.1f, 0.9f, 0.0f, wsp, ws,
                              nullptr, nullptr) == TKEF_EINVAL);  // momentum needed
  CHECK(tkef_aggregate_update(w, nullptr, n, 2, idx, val, nnz, 3, 0.1f, 0.0f, 0.0f, wsp, ws - 1,
                              nullptr, nullptr) == TKEF_EWORKSPACE);
  if (g_no_gpu)
    CHECK(tkef_aggregate_update(w, nullptr, n, 2, idx, val, nnz, 3, 0.1f, 0.0f, 0.0f, wsp, ws,
                                nullptr, nullptr) == TKEF_EHIP);  // no GPU here
  const int32_t* gidx = reinterpret_cast<const int32_t*>(0x300000);
  size_t uws = 0;
  CHECK(tkef_update_workspace(n, 2, 3, 10, &uws) == TKEF_OK);
  CHECK(tkef_sparse_aggregate_update(w, nullptr, n, 2, gidx, fake + 5000, 3, 10, nullptr, 0.1f,
                                     0.0f, 0.0f, nullptr, 0, nullptr,
                                     nullptr) == TKEF_EWORKSPACE);
  CHECK(tkef_sparse_aggregate(w, n, 2, gidx, fake + 5000, 7, 3, 10, nullptr, wsp, uws, nullptr,
                              nullptr) == TKEF_EINVAL);            // value format
}

int main() {
  int ndev = 0;
  g_no_gpu = hipGetDeviceCount(&ndev) != hipSuccess || ndev == 0;
  std::printf("host ABI driver: %s\n", g_no_gpu ? "no GPU: the HIP error paths run too"
                                                 : "a GPU is present: argument checks only");
  helpers();
  sparsify_plans();
  sparsify_oneshots();
  update_plans();
  aggregate_oneshots();
  std::printf("host ABI driver: %d failed checks\n", g_fail);
  return g_fail;
}
