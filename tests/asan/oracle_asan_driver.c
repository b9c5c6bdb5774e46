/* Calls every entry point of the oracle's C library on edge-case sizes, each
 * buffer allocated at exactly the size the entry point's contract names, so
 * that an AddressSanitizer / UndefinedBehaviorSanitizer build reports any
 * access outside it (test infrastructure; built and run by
 * tests/test_oracle_asan.py). */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

int lethe_oracle_attend(int64_t n, int D, int G, const float* q, const float* K, const float* V, double scale,
                        double gamma, const double* s_in, double* s_out, double* out);
double lethe_oracle_hoyer(int64_t n, const double* a);
double lethe_oracle_layer_sparsity(int64_t n, int H, const double* s);
int lethe_oracle_budget(int L, const int32_t* n, const float* S, int32_t recent, int32_t sink, int64_t G_b,
                        int32_t* budget);
int lethe_oracle_select(int64_t n, const float* s, int64_t k, int32_t recent, int32_t sink, uint8_t* keep);
void lethe_oracle_head_sum_f32(int64_t n, int H, const float* s, float* a);
int64_t lethe_oracle_shrink(int64_t n, const float* a, int32_t D, float tau, int32_t recent, int32_t sink,
                            int32_t* L_evict, uint8_t* keep);
int lethe_oracle_prefill(int64_t n, int64_t qlen, int D, int G, const float* q, const float* K, const float* V,
                         double scale, const double* s_in, double* s_out, double* out);

static uint32_t rng_state = 12345u;
static float frand(void) {
  rng_state = rng_state * 1664525u + 1013904223u;
  return (float)((rng_state >> 8) & 0xffff) / 65536.0f * 2.0f - 1.0f;
}
static float* fbuf(int64_t n) {
  float* p = (float*)malloc((size_t)n * sizeof(float));
  for (int64_t i = 0; i < n; ++i) p[i] = frand();
  return p;
}
static double* dbuf(int64_t n) {
  double* p = (double*)malloc((size_t)n * sizeof(double));
  for (int64_t i = 0; i < n; ++i) p[i] = fabs((double)frand()) * 3.0;
  return p;
}

static int fails = 0;
#define CHECK(c)                                                        \
  do {                                                                  \
    if (!(c)) {                                                         \
      fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #c); \
      ++fails;                                                          \
    }                                                                   \
  } while (0)

static void attend_cases(void) {
  const int64_t ns[] = {0, 1, 2, 37};
  const int Ds[] = {1, 64};
  const int Gs[] = {1, 8};
  for (int a = 0; a < 4; ++a)
    for (int b = 0; b < 2; ++b)
      for (int c = 0; c < 2; ++c)
        for (int with_s = 0; with_s < 2; ++with_s) {
          const int64_t n = ns[a];
          const int D = Ds[b], G = Gs[c];
          float* q = fbuf((int64_t)G * D);
          float* K = fbuf(n * D);
          float* V = fbuf(n * D);
          double* s_in = with_s ? dbuf(n) : NULL;
          double* s_out = dbuf(n);
          double* out = dbuf((int64_t)G * D);
          CHECK(lethe_oracle_attend(n, D, G, q, K, V, 0.125, 0.99, s_in, s_out, out) == 0);
          free(q), free(K), free(V), free(s_in), free(s_out), free(out);
        }
}

static void prefill_cases(void) {
  const int64_t ns[] = {0, 1, 20};
  for (int a = 0; a < 3; ++a) {
    const int64_t n = ns[a];
    const int64_t qls[] = {0, 1, n, n + 1};
    for (int b = 0; b < 4; ++b) {
      const int64_t ql = qls[b];
      const int D = 16, G = 3;
      float* q = fbuf(ql * G * D);
      float* K = fbuf(n * D);
      float* V = fbuf(n * D);
      double* s_in = dbuf(n);
      double* s_out = dbuf(n);
      double* out = dbuf(ql * G * D);
      const int rc = lethe_oracle_prefill(n, ql, D, G, q, K, V, 0.25, s_in, s_out, out);
      CHECK(ql > n ? rc == -1 : rc == 0);
      free(q), free(K), free(V), free(s_in), free(s_out), free(out);
    }
  }
}

static void sparsity_cases(void) {
  const int64_t ns[] = {0, 1, 5, 9};
  for (int a = 0; a < 4; ++a) {
    const int64_t n = ns[a];
    double* x = dbuf(n);
    const double h = lethe_oracle_hoyer(n, x);
    CHECK(h >= 0.0 && h <= 1.0 + 1e-12);
    free(x);
    for (int H = 1; H <= 4; H += 3) {
      double* s = dbuf(n * H);
      const double S = lethe_oracle_layer_sparsity(n, H, s);
      CHECK(S >= 0.0 && S <= 1.0 + 1e-12);
      float* sf = fbuf(n * H);
      float* hs = (float*)malloc((size_t)n * sizeof(float));
      lethe_oracle_head_sum_f32(n, H, sf, hs);
      free(s), free(sf), free(hs);
    }
  }
}

static void budget_cases(void) {
  const int Ls[] = {1, 7, 256, 257};
  for (int a = 0; a < 4; ++a) {
    const int L = Ls[a];
    int32_t* n = (int32_t*)malloc((size_t)L * sizeof(int32_t));
    float* S = (float*)malloc((size_t)L * sizeof(float));
    int32_t* b = (int32_t*)malloc((size_t)L * sizeof(int32_t));
    int64_t total = 0;
    for (int l = 0; l < L; ++l) {
      n[l] = (l * 37) % 1000;
      S[l] = (l % 5 == 0) ? NAN : (float)(l % 11) / 10.0f;
      total += n[l];
    }
    const int64_t Gs[] = {0, total / 3, total, total + 5};
    for (int g = 0; g < 4; ++g) {
      const int rc = lethe_oracle_budget(L, n, S, 16, 4, Gs[g], b);
      CHECK(L > 256 ? rc < 0 : (rc == 0 || rc == 1));
    }
    free(n), free(S), free(b);
  }
}

static void select_cases(void) {
  const int64_t ns[] = {0, 1, 50};
  const int64_t ks[] = {-1, 0, 10, 50, 60};
  const int32_t rs[] = {0, 5, 100};
  const int32_t sks[] = {0, 3, 100};
  for (int a = 0; a < 3; ++a)
    for (int b = 0; b < 5; ++b)
      for (int c = 0; c < 3; ++c)
        for (int d = 0; d < 3; ++d) {
          const int64_t n = ns[a];
          float* s = fbuf(n);
          if (n > 3) s[3] = NAN;
          uint8_t* keep = (uint8_t*)malloc((size_t)n);
          CHECK(lethe_oracle_select(n, s, ks[b], rs[c], sks[d], keep) == 0);
          int64_t kept = 0;
          for (int64_t j = 0; j < n; ++j) kept += keep[j];
          const int64_t want = ks[b] < 0 ? 0 : (ks[b] < n ? ks[b] : n);
          CHECK(kept == want);
          free(s), free(keep);
        }
}

static void shrink_cases(void) {
  const int64_t ns[] = {0, 1, 100, 1000};
  const int32_t Ds[] = {1, 10};
  const int32_t levs[] = {0, 50, 2147483647};
  for (int a = 0; a < 4; ++a)
    for (int b = 0; b < 2; ++b)
      for (int c = 0; c < 3; ++c) {
        const int64_t n = ns[a];
        float* s = fbuf(n);
        for (int64_t j = 0; j < n; ++j) s[j] = fabsf(s[j]) * (float)(1 + (j % 7));
        uint8_t* keep = (uint8_t*)malloc((size_t)n);
        int32_t lev = levs[c];
        const int64_t bp = lethe_oracle_shrink(n, s, Ds[b], 400.0f, 8, 2, &lev, keep);
        CHECK(bp >= -2 && bp < (n > 0 ? n : 1));
        free(s), free(keep);
      }
}

int main(void) {
  attend_cases();
  prefill_cases();
  sparsity_cases();
  budget_cases();
  select_cases();
  shrink_cases();
  if (fails) {
    fprintf(stderr, "%d checks failed\n", fails);
    return 1;
  }
  printf("ok\n");
  return 0;
}
