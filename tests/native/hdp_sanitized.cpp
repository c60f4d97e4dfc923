// Exercises libbs_hdp's C ABI on seeded random batches and on its error paths; built with the
// address and undefined-behaviour sanitizers by tests/test_hdp_sanitized.py.  Checks that a
// successful plan places every sequence exactly once on valid ranks, and that every error
// status leaves the outputs untouched.  Prints "ok <plans>" and exits 0 when all checks pass.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <vector>

#include "../../include/bs_hdp.h"

static uint64_t g_state = 0x9E3779B97F4A7C15ull;
static uint64_t next_u64() {  // xorshift64*
  g_state ^= g_state >> 12;
  g_state ^= g_state << 25;
  g_state ^= g_state >> 27;
  return g_state * 0x2545F4914F6CDD1Dull;
}
static double uniform() { return (next_u64() >> 11) * (1.0 / 9007199254740992.0); }
static int64_t irange(int64_t lo, int64_t hi) { return lo + (int64_t)(next_u64() % (uint64_t)(hi - lo + 1)); }

#define CHECK(cond, ...)                                      \
  do {                                                        \
    if (!(cond)) {                                            \
      std::fprintf(stderr, "check failed: " #cond " -- ");    \
      std::fprintf(stderr, __VA_ARGS__);                      \
      std::fprintf(stderr, "\n");                             \
      std::exit(1);                                           \
    }                                                         \
  } while (0)

int main() {
  int plans = 0;
  for (int iter = 0; iter < 2000; ++iter) {
    bs_hdp_cost cost;
    cost.alpha1 = uniform() * 1e-10;
    cost.beta1 = uniform() * 1e-7;
    cost.gamma = uniform() * 1e-4;
    cost.alpha2 = 1.0 + uniform() * 1e6;
    cost.beta2 = uniform() * 1e6;
    cost.layers = (int32_t)irange(3, 96);
    cost.bw_d2h = uniform() * 1e11;
    cost.bw_h2d = uniform() * 1e11;
    const int32_t n = (int32_t)irange(1, 300);
    const int64_t capacity = irange(256, 32768);
    const int32_t d_hdp = (int32_t)irange(1, 64);
    std::vector<int64_t> lengths(n);
    for (auto& l : lengths) l = 1 + (int64_t)std::exp(uniform() * std::log(4.0 * capacity));
    const int algorithm = (int)irange(0, 2);
    const double delta = uniform() < 0.2 ? 0.0 : uniform() * 1e-3;
    const int32_t n_buckets = (int32_t)irange(1, 16);

    for (int i = 0; i < n; i += 17) {
      double r = -1.0;
      int32_t ranks = -1;
      const int st = bs_hdp_offload_ratio(&cost, lengths[i], capacity, &r, &ranks);
      CHECK(st == BS_HDP_OK, "offload_ratio status %d: %s", st, bs_hdp_last_error());
      CHECK(r >= 0.0 && r <= 1.0 && ranks >= 1, "r %g ranks %d", r, ranks);
      if (lengths[i] <= capacity) CHECK(r == 0.0 && ranks == 1, "short sequence r %g D %d", r, ranks);
    }

    const int32_t max_mbs = n;
    const int64_t max_ranks = (int64_t)n * d_hdp;
    std::vector<bs_hdp_microbatch> mbs(max_mbs);
    std::vector<int32_t> seqs(n, -7), ranks(max_ranks, -7);
    std::vector<double> rank_time(d_hdp, -7.0);
    int32_t n_mbs = -7;
    const int st = bs_hdp_plan(algorithm, &cost, lengths.data(), n, capacity, d_hdp, delta, n_buckets,
                               mbs.data(), max_mbs, seqs.data(), ranks.data(), max_ranks, &n_mbs,
                               rank_time.data());
    if (st == BS_HDP_ERR_INFEASIBLE) {
      CHECK(n_mbs == -7 && seqs[0] == -7 && rank_time[0] == -7.0, "outputs written on error");
      continue;
    }
    CHECK(st == BS_HDP_OK, "plan status %d: %s", st, bs_hdp_last_error());
    ++plans;
    CHECK(n_mbs >= 1 && n_mbs <= max_mbs, "n_mbs %d", n_mbs);
    std::vector<int> seen(n, 0);
    int64_t next_seq = 0, next_rank = 0;
    for (int32_t m = 0; m < n_mbs; ++m) {
      const bs_hdp_microbatch& mb = mbs[m];
      CHECK(mb.seq_offset == next_seq && mb.n_seqs >= 1, "mb %d seq range", m);
      CHECK(mb.rank_offset == next_rank && mb.n_ranks >= 1 && mb.n_ranks <= d_hdp, "mb %d ranks", m);
      CHECK(mb.offload_ratio >= 0.0 && mb.offload_ratio <= 1.0 && mb.time >= 0.0, "mb %d r/time", m);
      int64_t tokens = 0;
      for (int32_t j = 0; j < mb.n_seqs; ++j) {
        const int32_t s = seqs[mb.seq_offset + j];
        CHECK(s >= 0 && s < n, "sequence index %d", s);
        ++seen[s];
        tokens += lengths[s];
      }
      if (mb.n_ranks == 1 && mb.n_seqs > 1) CHECK(tokens <= capacity, "packed mb %d over capacity", m);
      for (int32_t j = 0; j < mb.n_ranks; ++j) {
        const int32_t g = ranks[mb.rank_offset + j];
        CHECK(g >= 0 && g < d_hdp, "rank %d", g);
      }
      next_seq += mb.n_seqs;
      next_rank += mb.n_ranks;
    }
    CHECK(next_seq == n, "placed %lld of %d sequences", (long long)next_seq, n);
    for (int32_t s = 0; s < n; ++s) CHECK(seen[s] == 1, "sequence %d placed %d times", s, seen[s]);
    for (int32_t g = 0; g < d_hdp; ++g) CHECK(rank_time[g] >= 0.0 && std::isfinite(rank_time[g]), "rank time");

    // too small an output: BS_HDP_ERR_CAPACITY, outputs untouched
    if (n_mbs > 1) {
      std::vector<bs_hdp_microbatch> small(n_mbs - 1);
      std::vector<int32_t> s2(n, -7), r2(max_ranks, -7);
      std::vector<double> t2(d_hdp, -7.0);
      int32_t k2 = -7;
      const int st2 = bs_hdp_plan(algorithm, &cost, lengths.data(), n, capacity, d_hdp, delta,
                                  n_buckets, small.data(), n_mbs - 1, s2.data(), r2.data(), max_ranks,
                                  &k2, t2.data());
      CHECK(st2 == BS_HDP_ERR_CAPACITY, "small max_mbs status %d", st2);
      CHECK(k2 == -7 && s2[0] == -7 && t2[0] == -7.0, "outputs written on capacity error");
    }
  }
  // invalid arguments
  bs_hdp_cost cost = {1e-11, 1e-8, 1e-5, 1.0, 0.0, 8, 1e10, 1e10};
  int64_t len1 = 100;
  int32_t k = -7, seq = -7, rank = -7;
  double rt = -7.0, r = -7.0;
  bs_hdp_microbatch mb;
  CHECK(bs_hdp_plan(0, nullptr, &len1, 1, 128, 1, 0.0, 1, &mb, 1, &seq, &rank, 1, &k, &rt) ==
            BS_HDP_ERR_INVALID_ARG, "null cost");
  CHECK(bs_hdp_plan(0, &cost, nullptr, 1, 128, 1, 0.0, 1, &mb, 1, &seq, &rank, 1, &k, &rt) ==
            BS_HDP_ERR_INVALID_ARG, "null lengths");
  CHECK(bs_hdp_plan(7, &cost, &len1, 1, 128, 1, 0.0, 1, &mb, 1, &seq, &rank, 1, &k, &rt) ==
            BS_HDP_ERR_INVALID_ARG, "bad algorithm");
  CHECK(bs_hdp_plan(1, &cost, &len1, 1, 128, 1, -1.0, 1, &mb, 1, &seq, &rank, 1, &k, &rt) ==
            BS_HDP_ERR_INVALID_ARG, "negative delta");
  int64_t zero = 0;
  CHECK(bs_hdp_plan(0, &cost, &zero, 1, 128, 1, 0.0, 1, &mb, 1, &seq, &rank, 1, &k, &rt) ==
            BS_HDP_ERR_INVALID_ARG, "zero-length sequence");
  bs_hdp_cost neg = cost;
  neg.alpha1 = -1.0;
  CHECK(bs_hdp_offload_ratio(&neg, 100, 128, &r, &k) == BS_HDP_ERR_INVALID_ARG, "negative cost");
  neg = cost;
  neg.gamma = NAN;
  CHECK(bs_hdp_offload_ratio(&neg, 100, 128, &r, &k) == BS_HDP_ERR_INVALID_ARG, "NaN cost");
  CHECK(k == -7 && seq == -7 && rank == -7 && rt == -7.0 && r == -7.0, "outputs written on error");
  std::printf("ok %d\n", plans);
  return 0;
}
