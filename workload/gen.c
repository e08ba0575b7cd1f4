/*
 * Seeded synthetic job tables for the batched scheduling evaluator.
 *
 * This file only draws random numbers and turns them into integer job tables
 * (arrival step, prompt tokens, output tokens).  It contains none of the
 * scheduling method's arithmetic; both the oracle and the GPU library read the
 * bytes it writes.
 *
 * Randomness: SplitMix64 (Steele, Lea & Flood, "Fast splittable pseudorandom
 * number generators", OOPSLA 2014).  Each instance owns one stream whose seed is
 * the SplitMix64 finaliser applied to (config tag, seed, instance index), so an
 * instance's jobs do not depend on how many threads generate the table or on
 * which other instances are generated.
 *
 * Per job, draws are taken in this order: arrival gap (Poisson arrivals only),
 * prompt, output.
 *   u in [0,1)         : (x >> 11) * 2^-53
 *   U{a..b}            : a + floor(u * (b - a + 1))
 *   N(0,1)             : Box-Muller, sqrt(-2 ln(1-u1)) * cos(2 pi u2)
 *   LN(median m, s)    : llround(m * exp(s * z)), clipped to [lo, hi]
 *   Pareto(a, xmin)    : floor(xmin * (1-u)^(-1/a)), capped at hi
 *   two-part uniform   : with probability p U{a1..b1}, else U{a2..b2}
 *   Poisson arrivals   : S_j = S_{j-1} - ln(1-u)/rate, arrival_j = floor(S_j)
 *                        (rate 0 means every job arrives at step 0)
 */
#include <math.h>
#include <stdint.h>

enum { DIST_UNIFORM = 0, DIST_LOGNORMAL = 1, DIST_PARETO = 2, DIST_TWO_UNIFORM = 3 };

typedef struct {
  int32_t kind;
  int32_t pad;
  double p0, p1;      /* lognormal: median, sigma; pareto: shape, xmin; two-part: probability */
  int64_t a1, b1;     /* uniform / first uniform part bounds                                   */
  int64_t a2, b2;     /* second uniform part bounds                                            */
  int64_t lo, hi;     /* clip range (lognormal) / cap (pareto uses hi)                          */
} gen_dist;

typedef struct {
  uint64_t cfg_tag;
  uint64_t seed;
  double rate;        /* Poisson arrival rate per step; 0 => all arrive at step 0 */
  gen_dist prompt;
  gen_dist output;
} gen_recipe;

static uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

typedef struct { uint64_t s; } sm64;

static uint64_t sm_next(sm64* g) {
  g->s += 0x9E3779B97F4A7C15ULL;
  return mix64(g->s);
}

static double sm_u01(sm64* g) { return (double)(sm_next(g) >> 11) * 0x1.0p-53; }

static int64_t uniform_int(sm64* g, int64_t a, int64_t b) {
  double u = sm_u01(g);
  int64_t v = a + (int64_t)floor(u * (double)(b - a + 1));
  if (v > b) v = b; /* u < 1 makes this unreachable; kept as a guard */
  return v;
}

static int64_t draw(sm64* g, const gen_dist* d) {
  switch (d->kind) {
    case DIST_UNIFORM:
      return uniform_int(g, d->a1, d->b1);
    case DIST_LOGNORMAL: {
      double u1 = sm_u01(g), u2 = sm_u01(g);
      double z = sqrt(-2.0 * log(1.0 - u1)) * cos(6.283185307179586 * u2);
      double x = d->p0 * exp(d->p1 * z);
      int64_t v;
      if (x >= 9.0e18) v = d->hi;
      else v = llround(x);
      if (v < d->lo) v = d->lo;
      if (v > d->hi) v = d->hi;
      return v;
    }
    case DIST_PARETO: {
      double u = sm_u01(g);
      double x = d->p1 * pow(1.0 - u, -1.0 / d->p0);
      int64_t v;
      if (x >= (double)d->hi) v = d->hi;
      else v = (int64_t)floor(x);
      return v;
    }
    case DIST_TWO_UNIFORM: {
      double u = sm_u01(g);
      if (u < d->p0) return uniform_int(g, d->a1, d->b1);
      return uniform_int(g, d->a2, d->b2);
    }
    default:
      return -1;
  }
}

/* Fill rows [0, n_inst) of three [n_inst][n_jobs] int32 tables for the instances
 * inst_begin .. inst_begin + n_inst - 1.  Returns 0, or -1 on a bad recipe. */
int gen_jobs(const gen_recipe* r, int64_t inst_begin, int64_t n_inst, int32_t n_jobs,
             int32_t* arrival, int32_t* prompt, int32_t* output) {
  if (!r || n_inst < 0 || n_jobs < 1 || !arrival || !prompt || !output) return -1;
  if (r->prompt.kind < 0 || r->prompt.kind > 3 || r->output.kind < 0 || r->output.kind > 3) return -1;
  int bad = 0;
#pragma omp parallel for schedule(static) reduction(| : bad)
  for (int64_t k = 0; k < n_inst; ++k) {
    uint64_t key = mix64(r->cfg_tag + 0x9E3779B97F4A7C15ULL);
    key = mix64(key ^ r->seed);
    key = mix64(key ^ (uint64_t)(inst_begin + k));
    sm64 g = {key};
    double S = 0.0;
    int32_t* ar = arrival + k * (int64_t)n_jobs;
    int32_t* pr = prompt + k * (int64_t)n_jobs;
    int32_t* ou = output + k * (int64_t)n_jobs;
    for (int32_t j = 0; j < n_jobs; ++j) {
      if (r->rate > 0.0) {
        S += -log(1.0 - sm_u01(&g)) / r->rate;
        double f = floor(S);
        ar[j] = f > 2.0e9 ? 2000000000 : (int32_t)f;
      } else {
        ar[j] = 0;
      }
      int64_t p = draw(&g, &r->prompt);
      int64_t o = draw(&g, &r->output);
      if (p < 0 || o < 0 || p > INT32_MAX || o > INT32_MAX) bad = 1;
      pr[j] = (int32_t)p;
      ou[j] = (int32_t)o;
    }
  }
  return bad ? -1 : 0;
}

int gen_abi_version(void) { return 1; }
