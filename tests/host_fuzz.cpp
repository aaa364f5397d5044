// Randomised run of libhsap's host entry points (planner, run grouping, load matrix, balance,
// instruction emitter), built with AddressSanitizer and UndefinedBehaviorSanitizer by
// tests/test_host_sanitizers.py: any out-of-bounds access, leak, signed overflow or other
// undefined behaviour aborts the run.  Inputs: random document lengths (zero-length and
// one-token documents included), batch 1-3, every layout, P in {1,2,3,4,8,16}, tile sizes
// 16-128, and now and then an invalid shard, length or cu_seqlens order, which must be
// rejected with an error.  Structural checks: the two-call (count, then fill) patterns agree and
// every run lies inside the tile list, the runs covering it exactly once in total.
#include <cstdio>
#include <cstdlib>
#include <random>
#include <vector>
#include <algorithm>
#include "../include/hsap.h"
static std::mt19937_64 rng(getenv("SEED") ? atoll(getenv("SEED")) : 12345);
static int64_t U(int64_t lo, int64_t hi) { return std::uniform_int_distribution<int64_t>(lo, hi)(rng); }
int main(int argc, char** argv) {
  const int iters = argc > 1 ? atoi(argv[1]) : 2000;
  int64_t ok = 0, errs = 0;
  for (int it = 0; it < iters; ++it) {
    const int P = std::vector<int>{1, 2, 3, 4, 8, 16}[U(0, 5)];
    const int layout = (int)U(0, 1);
    const int bm = std::vector<int>{16, 32, 64, 128}[U(0, 3)], bn = std::vector<int>{16, 32, 64, 128}[U(0, 3)];
    const int B = (int)U(1, 3);
    int64_t unit = (int64_t)std::max(bm, bn) * (layout ? 2 * P : P);
    int64_t N = unit * U(1, 8);
    if (U(0, 9) == 0) N += U(-3, 3);  // sometimes invalid
    if (N <= 0) N = unit;
    // documents over B sequences (a boundary at every b*N)
    std::vector<int32_t> cu{0};
    for (int b = 0; b < B; ++b) {
      int64_t pos = 0;
      while (pos < N) {
        int64_t len = U(0, 4) == 0 ? 0 : (U(0, 3) == 0 ? 1 : U(1, N));
        len = std::min(len, N - pos);
        pos += len;
        cu.push_back((int32_t)(b * N + pos));
      }
    }
    if (U(0, 19) == 0 && cu.size() > 2) std::swap(cu[1], cu[2]);  // sometimes non-monotone
    const int nd = (int)cu.size() - 1;
    hsap_shard_desc sd{N, P, layout, (int32_t)U(0, P - 1), bm, bn, B};
    if (U(0, 29) == 0) sd.shard_id = P;  // invalid
    int64_t nt = 0;
    std::vector<int64_t> off(P + 1), pairs(P);
    hsap_status st = hsap_plan(cu.data(), nd, &sd, nullptr, 0, &nt, off.data(), pairs.data());
    if (st != HSAP_ERR_CAPACITY && st != HSAP_OK) { ++errs; continue; }
    std::vector<hsap_tile> tiles(nt + 1);
    st = hsap_plan(cu.data(), nd, &sd, tiles.data(), nt, &nt, off.data(), pairs.data());
    if (st != HSAP_OK) { printf("plan second call failed %d\n", st); return 1; }
    for (int major = 0; major < 3; ++major) {
      const int mrt = (int)U(-1, 8);
      int64_t nr = 0;
      int32_t slots = 0;
      std::vector<hsap_tile> sorted(nt + 1);
      st = hsap_plan_runs(&sd, tiles.data(), nt, major, mrt, sorted.data(), nullptr, 0, &nr, &slots);
      if (st != HSAP_ERR_CAPACITY && st != HSAP_OK) { printf("runs count failed %d: %s\n", st, hsap_last_error()); return 1; }
      std::vector<hsap_run> runs(nr + 1);
      st = hsap_plan_runs(&sd, tiles.data(), nt, major, mrt, sorted.data(), runs.data(), nr, &nr, &slots);
      if (st != HSAP_OK) { printf("runs failed %d: %s\n", st, hsap_last_error()); return 1; }
      int64_t covered = 0;
      for (int64_t i = 0; i < nr; ++i) {
        if (runs[i].first < 0 || runs[i].count < 0 || runs[i].first + runs[i].count > nt) { printf("bad run\n"); return 1; }
        covered += runs[i].count;
      }
      if (covered != nt) { printf("runs cover %lld of %lld (major %d)\n", (long long)covered, (long long)nt, major); return 1; }
    }
    (void)hsap_split_length(&sd, nt, (int32_t)U(1, 64), (int32_t)U(1, 1024));
    std::vector<int64_t> lt((size_t)P * P), lp((size_t)P * P);
    st = hsap_load_matrix(cu.data(), nd, &sd, lt.data(), lp.data());
    if (st != HSAP_OK) { printf("load matrix failed: %s\n", hsap_last_error()); return 1; }
    std::vector<int32_t> ex((size_t)P * P);
    std::vector<int64_t> load(P);
    st = hsap_balance(P, lt.data(), ex.data(), load.data());
    if (st != HSAP_OK) { printf("balance failed: %s\n", hsap_last_error()); return 1; }
    std::vector<int64_t> ro(P + 1);
    int32_t ns = 0;
    st = hsap_emit_forward(P, lt.data(), ex.data(), nullptr, 0, ro.data(), &ns);
    if (st != HSAP_ERR_CAPACITY && st != HSAP_OK) { printf("emit count failed: %s\n", hsap_last_error()); return 1; }
    std::vector<hsap_op> ops(ro[P] + 1);
    st = hsap_emit_forward(P, lt.data(), ex.data(), ops.data(), ro[P], ro.data(), &ns);
    if (st != HSAP_OK) { printf("emit failed: %s\n", hsap_last_error()); return 1; }
    ++ok;
  }
  printf("ok %lld, rejected %lld\n", (long long)ok, (long long)errs);
  return 0;
}
