/* Sanitizer driver for the library's host-side argument checks (test
 * infrastructure): every call below is rejected before any HIP call, so it
 * runs without a GPU.  Built with host AddressSanitizer and
 * UndefinedBehaviorSanitizer by tests/test_sanitizers_cpu.py. */
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "schedsim.h"

static int expect(const char* what, int got, int want) {
  if (got != want) {
    printf("%s: got %d, want %d\n", what, got, want);
    return 1;
  }
  return 0;
}

int main(void) {
  int fails = 0;
  int64_t offs[2] = {0, 4};
  int32_t f[4] = {1, 1, 1, 1}, st[1];
  int64_t tel[1];
  sched_instances_t in;
  memset(&in, 0, sizeof(in));
  in.num_instances = 1; in.max_requests = 4; in.total_requests = 4; in.offsets = offs;
  in.prompt = f; in.output = f; in.lower = f; in.upper = f; in.priority = f;
  sched_results_t out;
  memset(&out, 0, sizeof(out));
  out.completion = f; out.total_latency = tel; out.status = st;
  sched_options_t o;
  memset(&o, 0, sizeof(o));
  fails += expect("null instances", sched_simulate(NULL, SCHED_AMIN, 16, &out, NULL), SCHED_E_INVAL);
  fails += expect("null results", sched_simulate(&in, SCHED_AMIN, 16, NULL, NULL), SCHED_E_INVAL);
  fails += expect("M = 0", sched_simulate(&in, SCHED_AMIN, 0, &out, NULL), SCHED_E_INVAL);
  fails += expect("M = 2^30", sched_simulate(&in, SCHED_AMIN, (int64_t)1 << 30, &out, NULL), SCHED_E_INVAL);
  fails += expect("algo", sched_simulate(&in, (sched_algo_t)9, 16, &out, NULL), SCHED_E_INVAL);
  o.step_cap = (int64_t)1 << 31;
  fails += expect("step cap", sched_simulate_opts(&in, SCHED_AMIN, 16, &out, NULL, &o), SCHED_E_INVAL);
  o.step_cap = 0; o.running_capacity = 4096;
  fails += expect("running capacity", sched_simulate_opts(&in, SCHED_AMIN, 16, &out, NULL, &o), SCHED_E_UNSUPPORTED);
  fails += expect("running capacity (no alloc)", sched_simulate_noalloc(&in, SCHED_AMIN, 16, &out, NULL, &o),
                  SCHED_E_UNSUPPORTED);
  o.running_capacity = 0; o.evicted_lds_limit = -3;
  fails += expect("lds limit", sched_simulate_opts(&in, SCHED_AMIN, 16, &out, NULL, &o), SCHED_E_INVAL);
  in.max_requests = 1 << 17;
  fails += expect("n_max", sched_simulate(&in, SCHED_AMIN, 16, &out, NULL), SCHED_E_UNSUPPORTED);
  fails += expect("validate n_max", sched_validate(&in, SCHED_AMIN, 16, st, NULL), SCHED_E_UNSUPPORTED);
  in.max_requests = 4; in.lower = NULL;
  fails += expect("no lower", sched_simulate(&in, SCHED_AMIN, 16, &out, NULL), SCHED_E_INVAL);
  fails += expect("validate no lower", sched_validate(&in, SCHED_ADAPTIVE, 16, st, NULL), SCHED_E_INVAL);
  in.lower = f; in.num_instances = 0;
  fails += expect("empty batch", sched_simulate(&in, SCHED_AMIN, 16, &out, NULL), SCHED_OK);
  in.num_instances = 1;
  fails += expect("validate null status", sched_validate(&in, SCHED_AMIN, 16, NULL, NULL), SCHED_E_INVAL);
  for (int c = -9; c <= 1; ++c)
    if (!sched_strerror(c) || !sched_strerror(c)[0]) fails++;
  fails += expect("version", sched_version() >= 130, 1);
  printf("abi driver: %d failures\n", fails);
  return fails != 0;
}
