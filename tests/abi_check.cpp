// Host-only exercise of the C ABI under AddressSanitizer and UBSan: the
// ranking call on random and tied scores, and every entry point's argument
// validation (NULL handles and pointers, bad sizes, bad descriptors, bad
// alignment).  Every call made here returns before any device work, so no
// GPU is needed.  Exit status 0 and the line "ABI CHECK OK" on success.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <random>
#include <vector>

#include "cs.h"

#define EXPECT(c)                                                             \
  do {                                                                        \
    if (!(c)) {                                                               \
      std::fprintf(stderr, "FAIL %s:%d: %s (last error: %s)\n", __FILE__,     \
                   __LINE__, #c, cs_last_error());                            \
      return 1;                                                               \
    }                                                                         \
  } while (0)

static bool is_permutation_desc(const std::vector<int32_t>& o, const std::vector<double>& s) {
  const int n = (int)o.size();
  std::vector<int> seen(n, 0);
  for (int i = 0; i < n; ++i) {
    if (o[i] < 0 || o[i] >= n || seen[o[i]]++) return false;
    if (i > 0) {
      const double a = s[o[i - 1]], b = s[o[i]];
      if (a < b || (a == b && o[i - 1] > o[i])) return false;   // descending, ties by index
    }
  }
  return true;
}

static int check_rank() {
  std::mt19937_64 g(12345);
  std::normal_distribution<double> nd;
  for (int it = 0; it < 3000; ++it) {
    const int n = 2 + (int)(g() % 63);
    std::vector<double> a(n), b(n);
    const bool ties = it % 2 == 0;
    for (int i = 0; i < n; ++i) {
      a[i] = ties ? (double)(g() % 4) : nd(g);
      b[i] = ties ? (double)(g() % 3) : nd(g);
    }
    std::vector<int32_t> oc(n), of(n);
    double rho = 0.0;
    int32_t top1 = -1;
    EXPECT(cs_rank(a.data(), b.data(), n, oc.data(), of.data(), &rho, &top1) == CS_OK);
    EXPECT(is_permutation_desc(oc, a) && is_permutation_desc(of, b));
    EXPECT(std::isnan(rho) || (rho >= -1.0 - 1e-12 && rho <= 1.0 + 1e-12));
    EXPECT(top1 == (oc[0] == of[0] ? 1 : 0));
    double rho_same = 0.0;
    EXPECT(cs_rank(a.data(), a.data(), n, nullptr, nullptr, &rho_same, nullptr) == CS_OK);
    bool constant = true;
    for (int i = 1; i < n; ++i) constant &= a[i] == a[0];
    EXPECT(constant ? std::isnan(rho_same) : std::fabs(rho_same - 1.0) < 1e-12);
    EXPECT(cs_rank(a.data(), b.data(), n, nullptr, nullptr, nullptr, nullptr) == CS_OK);
    std::vector<int32_t> oo(n);
    EXPECT(cs_rank(a.data(), nullptr, n, oo.data(), nullptr, nullptr, nullptr) == CS_OK);
    EXPECT(oo == oc);
  }
  double one = 1.5, nan2[2] = {1.0, NAN}, two[2] = {1.0, 2.0};
  int32_t o1 = -1, o2[2];
  double rho;
  EXPECT(cs_rank(&one, nullptr, 1, &o1, nullptr, nullptr, nullptr) == CS_OK && o1 == 0);
  EXPECT(cs_rank(&one, &one, 1, &o1, &o1, &rho, nullptr) == CS_E_INVAL);
  EXPECT(cs_rank(two, nullptr, 0, o2, nullptr, nullptr, nullptr) == CS_E_INVAL);
  EXPECT(cs_rank(nan2, two, 2, o2, o2, &rho, nullptr) == CS_E_INVAL);
  EXPECT(cs_rank(two, nan2, 2, o2, o2, &rho, nullptr) == CS_E_INVAL);
  EXPECT(cs_rank(nullptr, two, 2, o2, o2, &rho, nullptr) == CS_E_INVAL);
  EXPECT(cs_rank(two, nullptr, 2, o2, o2, nullptr, nullptr) == CS_E_INVAL);
  return 0;
}

static int check_model_desc() {
  const cs_model_desc tiny = {2, 128, 4, 32, 512, 128, 32, 256, 16, 4, 16, 16, 1, 2, 2, CS_BF16};
  const cs_model_desc wan = {30, 1536, 12, 128, 8960, 4096, 512, 256, 16, 21, 60, 104, 1, 2, 2, CS_BF16};
  size_t n = 0;
  EXPECT(cs_model_weight_count(&tiny, &n) == CS_OK && n > 0);
  EXPECT(cs_model_weight_count(&wan, &n) == CS_OK && n > 1000000000u);
  EXPECT(cs_model_weight_count(nullptr, &n) == CS_E_INVAL);
  EXPECT(cs_model_weight_count(&tiny, nullptr) == CS_E_INVAL);
  struct Bad { int field; int value; int expect; };
  const Bad bad[] = {{1, 100, CS_E_INVAL},  {3, 16, CS_E_INVAL},    {0, 0, CS_E_INVAL},
                     {7, 128, CS_E_UNSUPPORTED}, {11, 15, CS_E_INVAL}, {12, 2, CS_E_UNSUPPORTED},
                     {15, 7, CS_E_INVAL},   {8, 8, CS_E_UNSUPPORTED}, {9, 1 << 20, CS_E_UNSUPPORTED}};
  for (const Bad& b : bad) {
    cs_model_desc d = tiny;
    reinterpret_cast<int32_t*>(&d)[b.field] = b.value;
    const int s = cs_model_weight_count(&d, &n);
    if (s != b.expect) std::fprintf(stderr, "field %d = %d: status %d (%s)\n", b.field, b.value, s, cs_last_error());
    EXPECT(s == b.expect);
    EXPECT(std::strlen(cs_last_error()) > 0);
  }
  cs_model* m = reinterpret_cast<cs_model*>(0x1);
  EXPECT(cs_model_init(&tiny, nullptr, n, nullptr, &m) == CS_E_INVAL);
  size_t nt = 0;
  EXPECT(cs_model_weight_count(&tiny, &nt) == CS_OK);
  float dummy[4] = {0, 0, 0, 0};
  EXPECT(cs_model_init(&tiny, dummy, nt - 1, nullptr, &m) == CS_E_INVAL);
  EXPECT(cs_model_init(&tiny, dummy, nt, nullptr, nullptr) == CS_E_INVAL);
  return 0;
}

static int check_null_handles() {
  float f[4] = {0, 0, 0, 0};
  double d[4];
  uint8_t u[4];
  size_t bytes = 0;
  cs_rollout* r = nullptr;
  cs_rollout_stats_t st;
  EXPECT(cs_velocity(nullptr, f, 1, 0.5f, f, f + 1) == CS_E_INVAL);
  EXPECT(cs_rollout_init(nullptr, nullptr, f, f, nullptr, &r) == CS_E_INVAL);
  EXPECT(cs_cache_decide(nullptr, 1, u, u, d) == CS_E_INVAL);
  EXPECT(cs_denoise_step(nullptr, 1) == CS_E_INVAL);
  EXPECT(cs_score(nullptr, f, d) == CS_E_INVAL);
  EXPECT(cs_preview_score(nullptr, f, d) == CS_E_INVAL);
  EXPECT(cs_rollout_enable_preview(nullptr, 1) == CS_E_INVAL);
  int32_t keep[1] = {0};
  EXPECT(cs_rollout_retain(nullptr, keep, 1) == CS_E_INVAL);
  EXPECT(cs_rollout_latents(nullptr, f) == CS_E_INVAL);
  EXPECT(cs_rollout_stats(nullptr, &st) == CS_E_INVAL);
  EXPECT(cs_rollout_export(nullptr, nullptr, &bytes) == CS_E_INVAL);
  EXPECT(cs_rollout_import(nullptr, f, sizeof f) == CS_E_INVAL);
  EXPECT(cs_profile_enable(nullptr, 1) == CS_E_INVAL);
  EXPECT(cs_profile_reset(nullptr) == CS_E_INVAL);
  EXPECT(cs_profile_read(nullptr, 0, d, nullptr) == CS_E_INVAL);
  cs_rollout_free(nullptr);
  cs_model_free(nullptr);
  return 0;
}

static int check_score_noalloc() {
  alignas(16) float x[8] = {0};
  alignas(8) double s[2];
  EXPECT(cs_score_noalloc(nullptr, x, 1, 8, s, nullptr) == CS_E_INVAL);
  EXPECT(cs_score_noalloc(x, nullptr, 1, 8, s, nullptr) == CS_E_INVAL);
  EXPECT(cs_score_noalloc(x, x, 1, 8, nullptr, nullptr) == CS_E_INVAL);
  EXPECT(cs_score_noalloc(x, x, 0, 8, s, nullptr) == CS_E_INVAL);
  EXPECT(cs_score_noalloc(x, x, 70000, 8, s, nullptr) == CS_E_INVAL);
  EXPECT(cs_score_noalloc(x, x, 1, 6, s, nullptr) == CS_E_INVAL);
  EXPECT(cs_score_noalloc(x, x, 1, 0, s, nullptr) == CS_E_INVAL);
  EXPECT(cs_score_noalloc(x + 1, x, 1, 4, s, nullptr) == CS_E_INVAL);
  EXPECT(cs_score_noalloc(x, x, 65535, (int64_t)8192 * 9, s, nullptr) == CS_E_INVAL);
  EXPECT(std::strstr(cs_last_error(), "scratch capacity") != nullptr);
  return 0;
}

int main() {
  if (check_rank() || check_model_desc() || check_null_handles() || check_score_noalloc()) return 1;
  std::printf("ABI CHECK OK\n");
  return 0;
}
