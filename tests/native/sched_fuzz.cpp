// Drives the scheduler's C ABI through every policy / chunking / APC
// combination on a random request stream, for a build with AddressSanitizer
// and UndefinedBehaviorSanitizer (tests/test_native_sanitizers.py).  Exits
// non-zero if a call fails or a request never finishes.
#include <cstdio>
#include <random>
#include <vector>

#include "cp_sched.h"
int main() {
  std::mt19937 g(1);
  for (int policy = 0; policy < 2; ++policy)
    for (int chunking = 0; chunking < 2; ++chunking)
      for (int apc = 0; apc < 2; ++apc) {
        cps_config c{};
        c.policy = policy; c.alpha = 1e-3; c.beta = -1.0; c.max_tokens = 256; c.max_seqs = 8;
        c.max_seq_len = 2048; c.chunking = chunking; c.target_us = 50; c.delta = 16;
        c.lambda_u = 1; c.lambda_o = 4; c.apc = apc; c.max_active = 2; c.min_chunk = 16;
        int err = 0;
        cps_sched* s = cps_create(&c, &err);
        if (!s) { printf("create failed %d\n", err); return 1; }
        if (chunking) {
          int32_t dims[3] = {16, 8, 1};
          std::vector<double> w(16 * 8 + 8), b(9), mean(16, 0.0), sd(16, 1.0);
          for (auto& x : w) x = std::uniform_real_distribution<double>(-0.1, 0.1)(g);
          for (auto& x : b) x = 0.5;
          if (cps_set_predictor(s, 2, dims, w.data(), b.data(), mean.data(), sd.data(), 10.0)) return 2;
        }
        for (int i = 0; i < 40; ++i)
          cps_add_request(s, i, i * 3.0, 1 + (int)(g() % 300), 1 + (int)(g() % 20));
        std::vector<cp_row_meta> rows(64);
        std::vector<int64_t> ids(64);
        double now = 0;
        for (int round = 0; round < 2000 && cps_pending(s) > 0; ++round) {
          int32_t n = 0, nd = 0;
          int rc = cps_schedule(s, now, rows.data(), ids.data(), 64, &n, &nd);
          if (rc) { printf("schedule rc %d\n", rc); return 3; }
          now += 10.0;
          if (cps_complete(s, now)) return 4;
        }
        cps_stats st;
        cps_get_stats(s, &st);
        printf("policy %d chunking %d apc %d: rounds %lld finished %lld pending %lld\n", policy, chunking, apc,
               (long long)st.rounds, (long long)st.finished, (long long)cps_pending(s));
        if (cps_pending(s) != 0) return 5;
        cps_destroy(s);
      }
  return 0;
}
