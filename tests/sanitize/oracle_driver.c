/* Sanitizer driver for the CPU oracle (test infrastructure): random instances
 * through orc_simulate with every policy, with and without arrivals, tie keys,
 * priorities, event logs (also too small ones) and statistics.  Built with
 * -fsanitize=address,undefined by tests/test_sanitizers_cpu.py; any report
 * fails the test.  Exit status 0 when every call returned a valid status. */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include "sched_oracle.h"

static uint64_t rng_state = 0x9E3779B97F4A7C15ull;
static uint32_t next_u32(void) { /* xorshift64* */
  rng_state ^= rng_state >> 12;
  rng_state ^= rng_state << 25;
  rng_state ^= rng_state >> 27;
  return (uint32_t)((rng_state * 0x2545F4914F6CDD1Dull) >> 32);
}
static int32_t uni(int32_t lo, int32_t hi) { return lo + (int32_t)(next_u32() % (uint32_t)(hi - lo + 1)); }

int main(int argc, char** argv) {
  const int reps = argc > 1 ? atoi(argv[1]) : 2000;
  int bad = 0;
  for (int rep = 0; rep < reps; ++rep) {
    const int32_t n = uni(0, 40);
    const int64_t M = uni(1, 60);
    int32_t *a = malloc(sizeof(int32_t) * (n + 1)), *s = malloc(sizeof(int32_t) * (n + 1));
    int32_t *o = malloc(sizeof(int32_t) * (n + 1)), *l = malloc(sizeof(int32_t) * (n + 1));
    int32_t *u = malloc(sizeof(int32_t) * (n + 1)), *pr = malloc(sizeof(int32_t) * (n + 1));
    int32_t *tk = malloc(sizeof(int32_t) * (n + 1)), *comp = malloc(sizeof(int32_t) * (n + 1));
    int32_t *ev = malloc(sizeof(int32_t) * (n + 1));
    int32_t t0 = 0;
    for (int32_t i = 0; i < n; ++i) {
      t0 += rep % 3 == 0 ? uni(0, 3) : 0;
      a[i] = (rep % 17 == 5 && i == n / 2) ? -1 : t0; /* now and then an invalid arrival */
      s[i] = uni(rep % 13 == 0 ? -1 : 0, 8);
      o[i] = uni(rep % 11 == 0 ? 0 : 1, 12);
      l[i] = o[i] > 0 ? uni(rep % 7 == 0 ? 0 : 1, o[i]) : 1;
      u[i] = o[i] + uni(rep % 9 == 0 ? -1 : 0, 6);
      pr[i] = uni(0, n);
      tk[i] = (int32_t)next_u32();
    }
    for (int32_t algo = 0; algo <= 5; ++algo) {
      int64_t tel, mk, rs, te, nev, stats[ORC_STAT_COUNT];
      orc_event_t evs[8];
      const int st = orc_simulate(n, rep % 2 ? a : NULL, s, o, l, u, pr, rep % 4 < 2 ? tk : NULL, algo, M,
                                  rep % 5 == 0 ? uni(1, 20) : 0, comp, ev, &tel, &mk, &rs, &te, stats,
                                  evs, rep % 6 == 0 ? 0 : 8, &nev);
      if (st > 0 || st < -7) bad++;
    }
    free(a); free(s); free(o); free(l); free(u); free(pr); free(tk); free(comp); free(ev);
  }
  printf("oracle driver: %d repetitions, %d unexpected statuses\n", reps, bad);
  return bad != 0;
}
