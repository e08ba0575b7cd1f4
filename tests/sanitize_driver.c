/* Test driver for a sanitizer build of the oracle (AddressSanitizer and
 * UndefinedBehaviorSanitizer, host code only): runs every oracle entry point on
 * seeded random instances (every policy and flag, releases, KV budgets, B from
 * 1 to unlimited, alpha from 0 to infinity, invalid tables) and checks the
 * cost identity and the re-scorer's agreement, so that any out-of-bounds
 * access, leak or undefined operation on these paths stops the run. */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
  int64_t T, O, Q, E, C, W, sc, sl, sext, busy, peak, unfair;
  int32_t maxext, maxact;
} m_t;

int oracle_simulate(int32_t, const int32_t*, const int32_t*, const int32_t*, int32_t, int32_t,
                    int64_t, int32_t, uint32_t, int64_t, int64_t, m_t*, int32_t*, int32_t*);
int oracle_simulate_robust(int32_t, const int32_t*, const int32_t*, const int32_t*,
                           const int32_t*, int32_t, int32_t, int64_t, int32_t, uint32_t,
                           int64_t, int64_t, m_t*, int32_t*, int32_t*);
int oracle_decompose(int32_t, const int32_t*, const int32_t*, const int32_t*, int32_t, int32_t,
                     int64_t, int64_t, int64_t, const int32_t*, m_t*, uint32_t*);
int oracle_opt(int32_t, const int32_t*, const int32_t*, const int32_t*, int32_t, int32_t,
               int64_t, int64_t*, int32_t*);

static uint64_t rs = 0x9E3779B97F4A7C15ull;
static uint32_t rnd(uint32_t m) { /* xorshift64*, uniform enough for test inputs */
  rs ^= rs >> 12;
  rs ^= rs << 25;
  rs ^= rs >> 27;
  return (uint32_t)((rs * 0x2545F4914F6CDD1Dull) >> 33) % m;
}

#define CHECK(c)                                                   \
  do {                                                             \
    if (!(c)) {                                                    \
      fprintf(stderr, "check failed line %d: %s\n", __LINE__, #c); \
      return 1;                                                    \
    }                                                              \
  } while (0)

int main(int argc, char** argv) {
  int trials = argc > 1 ? atoi(argv[1]) : 300;
  const uint32_t flag_sets[] = {0u, 8u, 16u, 32u, 8u | 16u};
  for (int t = 0; t < trials; ++t) {
    int32_t n = 1 + (int32_t)rnd(t % 10 == 0 ? 300 : 24);
    int32_t* a = malloc(sizeof(int32_t) * n);
    int32_t* p = malloc(sizeof(int32_t) * n);
    int32_t* o = malloc(sizeof(int32_t) * n);
    int32_t* u = malloc(sizeof(int32_t) * n);
    int32_t* st = malloc(sizeof(int32_t) * n);
    int32_t* fi = malloc(sizeof(int32_t) * n);
    int32_t* st2 = malloc(sizeof(int32_t) * n);
    const int rel = rnd(3);
    int32_t acc = 0;
    for (int i = 0; i < n; ++i) {
      if (rel == 1) acc += (int32_t)rnd(4);
      a[i] = rel == 0 ? 0 : (rel == 1 ? acc : (int32_t)rnd(40));
      p[i] = (int32_t)rnd(6);
      o[i] = 1 + (int32_t)rnd(30);
      u[i] = o[i] + (int32_t)rnd(8);
    }
    const int32_t B = (int32_t)rnd(6);              /* 0 = unlimited */
    const int32_t alphas[] = {0, 1, 2, 3, 7, 15, 2147483647};
    const int32_t alpha = alphas[rnd(7)];
    const int64_t M = rnd(3) == 0 ? 0 : 30 + rnd(60); /* 0 = no KV budget */
    const int64_t c = rnd(5), tau = 1 + rnd(3);
    for (int pol = 0; pol < 4; ++pol) {
      for (unsigned f = 0; f < sizeof(flag_sets) / sizeof(flag_sets[0]); ++f) {
        m_t m, d;
        uint32_t v = 99;
        memset(&m, 0, sizeof(m));
        int rc = oracle_simulate(n, a, p, o, B, alpha, M, pol, flag_sets[f], c, tau, &m, st, fi);
        CHECK(rc == 0);
        CHECK(m.T >= 0 && m.busy <= m.T);
        if (!(flag_sets[f] & 32u)) {
          CHECK(m.C == c * m.T + tau * (m.Q + m.E));
          rc = oracle_decompose(n, a, p, o, B, alpha, M, c, tau, st, &d, &v);
          CHECK(rc == 0 && d.T == m.T && d.E == m.E && d.C == m.C);
          CHECK((v & ~8u) == 0); /* only FCFS / SJF may break fairness */
          if (pol == 1 || pol == 2) CHECK(v == 0);
        }
        if (pol == 2) {
          rc = oracle_simulate_robust(n, a, p, o, u, B, alpha, M, pol, flag_sets[f], c, tau, &m,
                                      st2, NULL);
          CHECK(rc == 0 && m.unfair == 0);
        }
      }
    }
    if (n <= 6) {
      int64_t T = 0;
      int rc = oracle_opt(n, a, p, o, B == 0 ? 2 : B, alpha, M, &T, st2);
      CHECK(rc == 0 && T > 0);
    }
    /* invalid tables are refused, not read out of range */
    o[n - 1] = 0;
    m_t m;
    CHECK(oracle_simulate(n, a, p, o, B, alpha, M, 2, 0, c, tau, &m, NULL, NULL) != 0);
    free(a);
    free(p);
    free(o);
    free(u);
    free(st);
    free(fi);
    free(st2);
  }
  printf("sanitized oracle: %d trials ok\n", trials);
  return 0;
}
