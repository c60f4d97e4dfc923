// Host-side HDP planners (Sec. 5.2 Eq. 3, Alg. 1, Sec. 6 Alg. 2): the C ABI of bs_hdp.h.
//
// The decisions are those the header states; this file makes them in O(n log n):
// best fit keeps the open micro-batches in an ordered set by (room left, index); rank choices
// keep the ranks ordered by (micro-batch count, rank) or (finish time, rank); a bucket keeps its
// remaining positions in an ordered set, and since a bucket's lengths do not increase along it,
// the first remaining sequence that fits a given room is found by a binary search for the first
// position whose length fits, then the next remaining position at or after it.
//
// Every double is formed by the same operations in the same order as the statement of the
// rule (left to right), and the build turns contraction into fused multiply-adds off
// (-ffp-contract=off), so the plans are reproducible bit for bit by any implementation of the
// same rules.

#include <algorithm>
#include <climits>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <set>
#include <utility>
#include <vector>

#include "../../include/bs_hdp.h"

namespace {

thread_local char g_err[256] = "";

int fail(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return code;
}

int ok() {
  g_err[0] = '\0';
  return BS_HDP_OK;
}

struct Cost {
  double a1, b1, g, a2, b2;
  int l;
  double bw_d2h, bw_h2d;
  double T(int64_t len) const {
    const double s = (double)len;
    return a1 * s * s + b1 * s + g;
  }
  double act(int64_t len) const { return a2 * (double)len + b2; }
};

bool finite_nonneg(double x) { return std::isfinite(x) && x >= 0.0; }

int check_cost(const bs_hdp_cost* c, Cost* out) {
  if (c == nullptr) return fail(BS_HDP_ERR_INVALID_ARG, "cost is NULL");
  if (!finite_nonneg(c->alpha1) || !finite_nonneg(c->beta1) || !finite_nonneg(c->gamma))
    return fail(BS_HDP_ERR_INVALID_ARG, "alpha1, beta1, gamma must be finite and >= 0");
  if (!std::isfinite(c->alpha2) || !std::isfinite(c->beta2) || !(c->alpha2 + c->beta2 > 0.0) ||
      c->alpha2 < 0.0)
    return fail(BS_HDP_ERR_INVALID_ARG, "Act(s) = alpha2 s + beta2 must be finite and > 0");
  if (c->layers < 3) return fail(BS_HDP_ERR_INVALID_ARG, "layers = %d must be >= 3", c->layers);
  if (!finite_nonneg(c->bw_d2h) || !finite_nonneg(c->bw_h2d))
    return fail(BS_HDP_ERR_INVALID_ARG, "bandwidths must be finite and >= 0");
  *out = Cost{c->alpha1, c->beta1, c->gamma, c->alpha2, c->beta2, c->layers, c->bw_d2h, c->bw_h2d};
  return BS_HDP_OK;
}

// Eq. 3.  Returns false if D does not fit an int32.
bool offload(int64_t s, int64_t C, const Cost& c, double* r_out, int64_t* d_out) {
  if (s <= C) {
    *r_out = 0.0;
    *d_out = 1;
    return true;
  }
  const double a_s = c.act(s), a_c = c.act(C);
  const double l = (double)c.l, l2 = (double)(c.l - 2);
  const double r_lo = std::min(1.0, (l * a_c) / (l2 * a_s));
  const double bw = std::min(c.bw_d2h, c.bw_h2d);
  const double r_hi = std::min(1.0, c.T(s) * bw / a_s);
  const double r = r_hi >= r_lo ? r_hi : 0.0;
  const double D = std::ceil((2.0 * a_s + (1.0 - r) * l2 * a_s) / (l * a_c));
  if (!(D <= 2147483647.0)) return false;
  *r_out = r;
  *d_out = (int64_t)D;
  return true;
}

struct Unit {
  std::vector<int32_t> seqs;
  std::vector<int32_t> ranks;
  double r, start, t;
};

// Ranks ordered by (key, rank) with O(log d) updates.
template <typename K>
struct RankOrder {
  std::set<std::pair<K, int32_t>> s;
  std::vector<K> key;
  explicit RankOrder(int32_t d, K init) : key(d, init) {
    for (int32_t g = 0; g < d; ++g) s.insert({init, g});
  }
  void set(int32_t g, K k) {
    s.erase({key[g], g});
    key[g] = k;
    s.insert({k, g});
  }
};

// The ranks start together when the last of them is free; each finishes at start + t.
double place(RankOrder<double>& fin, const std::vector<int32_t>& ranks, double t) {
  double start = fin.key[ranks[0]];
  for (int32_t g : ranks) start = std::max(start, fin.key[g]);
  for (int32_t g : ranks) fin.set(g, start + t);
  return start;
}

int naive(const int64_t* len, int32_t n, int64_t C, int32_t d, const Cost& c,
          std::vector<Unit>* units, std::vector<double>* fin_out) {
  std::vector<int32_t> pack;
  for (int32_t i = 0; i < n; ++i) {
    double r;
    int64_t D;
    if (!offload(len[i], C, c, &r, &D) || (len[i] > C && D > d))
      return fail(BS_HDP_ERR_INFEASIBLE, "sequence %d needs more than d_hdp = %d ranks", i, d);
    if (len[i] <= C) {
      pack.push_back(i);
    } else {
      units->push_back(Unit{{i}, {}, r, 0.0, c.T(len[i]) / (double)D});
      units->back().ranks.resize((size_t)D);
    }
  }
  // best fit, largest first
  std::stable_sort(pack.begin(), pack.end(), [&](int32_t a, int32_t b) {
    return len[a] != len[b] ? len[a] > len[b] : a < b;
  });
  std::set<std::pair<int64_t, int32_t>> open;  // (room left, micro-batch index)
  std::vector<std::vector<int32_t>> bins;
  std::vector<int64_t> room;
  for (int32_t i : pack) {
    auto it = open.lower_bound({len[i], INT32_MIN});
    if (it == open.end()) {
      bins.push_back({i});
      room.push_back(C - len[i]);
      open.insert({room.back(), (int32_t)bins.size() - 1});
    } else {
      const int32_t b = it->second;
      open.erase(it);
      bins[b].push_back(i);
      room[b] -= len[i];
      open.insert({room[b], b});
    }
  }
  for (auto& b : bins) {
    double t = 0.0;
    for (int32_t i : b) t += c.T(len[i]);
    Unit u{b, {0}, 0.0, 0.0, t};
    units->push_back(std::move(u));
  }
  // deal by count
  RankOrder<int64_t> count(d, 0);
  RankOrder<double> fin(d, 0.0);
  for (Unit& u : *units) {
    auto it = count.s.begin();
    for (size_t k = 0; k < u.ranks.size(); ++k, ++it) u.ranks[k] = it->second;
    u.start = place(fin, u.ranks, u.t);
    for (int32_t g : u.ranks) count.set(g, count.key[g] + 1);
  }
  *fin_out = fin.key;
  return BS_HDP_OK;
}

// A bucket: sequence ids in order of decreasing length and the positions still present.
struct Bucket {
  std::vector<int32_t> ids;
  std::set<int32_t> live;
};

int balance(const int64_t* len, int32_t n, int64_t C, int32_t d, const Cost& c, double delta,
            int strategy, int32_t nb, std::vector<Unit>* units, std::vector<double>* fin_out) {
  for (int32_t i = 0; i < n; ++i) {
    double r;
    int64_t D;
    if (!offload(len[i], C, c, &r, &D) || (len[i] > C && D > d))
      return fail(BS_HDP_ERR_INFEASIBLE, "sequence %d needs more than d_hdp = %d ranks", i, d);
  }
  std::vector<int32_t> order(n);
  for (int32_t i = 0; i < n; ++i) order[i] = i;
  std::stable_sort(order.begin(), order.end(), [&](int32_t a, int32_t b) {
    return len[a] != len[b] ? len[a] > len[b] : a < b;
  });
  std::vector<double> cost(n);
  double total = 0.0;
  for (int32_t k = 0; k < n; ++k) {
    cost[k] = c.T(len[order[k]]);
    total += cost[k];
  }
  std::vector<Bucket> all(nb);
  double cum = 0.0;
  for (int32_t k = 0; k < n; ++k) {
    int64_t b = 0;
    if (total > 0.0) b = std::min<int64_t>(nb - 1, (int64_t)(cum * (double)nb / total));
    all[b].ids.push_back(order[k]);
    cum += cost[k];
  }
  std::vector<Bucket> buckets;
  for (Bucket& b : all) {
    if (b.ids.empty()) continue;
    for (int32_t p = 0; p < (int32_t)b.ids.size(); ++p) b.live.insert(p);
    buckets.push_back(std::move(b));
  }
  RankOrder<double> fin(d, 0.0);

  auto take = [&](Bucket& b, std::vector<int32_t>* seqs) {
    const int32_t head = *b.live.begin();
    if (len[b.ids[head]] > C) {
      seqs->push_back(b.ids[head]);
      b.live.erase(b.live.begin());
      return;
    }
    int64_t room = C;
    while (!b.live.empty()) {
      // first position whose length fits the room (lengths do not increase along the bucket)
      const auto first_fit = std::partition_point(b.ids.begin(), b.ids.end(),
                                                  [&](int32_t i) { return len[i] > room; });
      auto it = b.live.lower_bound((int32_t)(first_fit - b.ids.begin()));
      if (it == b.live.end()) break;
      const int32_t i = b.ids[*it];
      seqs->push_back(i);
      room -= len[i];
      b.live.erase(it);
    }
  };

  auto give = [&](int32_t g) {
    const size_t bi = strategy == BS_HDP_DP_BALANCE ? 0 : (size_t)g % buckets.size();
    Unit u{{}, {}, 0.0, 0.0, 0.0};
    take(buckets[bi], &u.seqs);
    if (buckets[bi].live.empty()) buckets.erase(buckets.begin() + (std::ptrdiff_t)bi);
    if (u.seqs.size() == 1 && len[u.seqs[0]] > C) {
      int64_t D;
      offload(len[u.seqs[0]], C, c, &u.r, &D);
      auto it = fin.s.begin();
      for (int64_t k = 0; k < D; ++k, ++it) u.ranks.push_back(it->second);
      u.t = c.T(len[u.seqs[0]]) / (double)D;
    } else {
      u.ranks.push_back(g);
      double t = 0.0;
      for (int32_t i : u.seqs) t += c.T(len[i]);
      u.t = t;
    }
    u.start = place(fin, u.ranks, u.t);
    units->push_back(std::move(u));
  };

  while (!buckets.empty()) {
    const double max_t = fin.s.rbegin()->first;
    auto lagging = [&]() {
      const auto& first = *fin.s.begin();
      return max_t - first.first > delta ? first.second : -1;
    };
    int32_t g = lagging();
    if (g < 0) {
      give(fin.s.begin()->second);
      continue;
    }
    while (g >= 0 && !buckets.empty()) {
      give(g);
      g = lagging();
    }
  }
  *fin_out = fin.key;
  return BS_HDP_OK;
}

}  // namespace

extern "C" {

int bs_hdp_offload_ratio(const bs_hdp_cost* cost, int64_t s, int64_t capacity, double* ratio,
                         int32_t* ranks) {
  Cost c;
  int rc = check_cost(cost, &c);
  if (rc != BS_HDP_OK) return rc;
  if (s < 1 || capacity < 1) return fail(BS_HDP_ERR_INVALID_ARG, "s and capacity must be >= 1");
  if (ratio == nullptr || ranks == nullptr) return fail(BS_HDP_ERR_INVALID_ARG, "output is NULL");
  double r;
  int64_t D;
  if (!offload(s, capacity, c, &r, &D)) return fail(BS_HDP_ERR_INFEASIBLE, "D(s) overflows");
  *ratio = r;
  *ranks = (int32_t)D;
  return ok();
}

int bs_hdp_plan(int algorithm, const bs_hdp_cost* cost, const int64_t* lengths, int32_t n,
                int64_t capacity, int32_t d_hdp, double delta, int32_t n_buckets,
                bs_hdp_microbatch* mbs, int32_t max_mbs, int32_t* seqs, int32_t* ranks,
                int64_t max_ranks, int32_t* n_mbs, double* rank_time) {
  Cost c;
  int rc = check_cost(cost, &c);
  if (rc != BS_HDP_OK) return rc;
  if (algorithm < BS_HDP_NAIVE || algorithm > BS_HDP_PP_BALANCE)
    return fail(BS_HDP_ERR_INVALID_ARG, "unknown algorithm %d", algorithm);
  if (n < 0 || capacity < 1 || d_hdp < 1)
    return fail(BS_HDP_ERR_INVALID_ARG, "n >= 0, capacity >= 1 and d_hdp >= 1 are required");
  if (algorithm != BS_HDP_NAIVE && (!finite_nonneg(delta) || n_buckets < 1 || n_buckets > (1 << 20)))
    return fail(BS_HDP_ERR_INVALID_ARG, "delta must be finite and >= 0, n_buckets in [1, 2^20]");
  if ((n > 0 && (lengths == nullptr || mbs == nullptr || seqs == nullptr || ranks == nullptr)) ||
      n_mbs == nullptr || rank_time == nullptr)
    return fail(BS_HDP_ERR_INVALID_ARG, "an array is NULL");
  for (int32_t i = 0; i < n; ++i)
    if (lengths[i] < 1) return fail(BS_HDP_ERR_INVALID_ARG, "lengths[%d] = %lld < 1", i,
                                    (long long)lengths[i]);
  std::vector<Unit> units;
  std::vector<double> fin(d_hdp, 0.0);
  rc = algorithm == BS_HDP_NAIVE
           ? naive(lengths, n, capacity, d_hdp, c, &units, &fin)
           : balance(lengths, n, capacity, d_hdp, c, delta, algorithm, n_buckets, &units, &fin);
  if (rc != BS_HDP_OK) return rc;
  int64_t nr = 0;
  for (const Unit& u : units) nr += (int64_t)u.ranks.size();
  if ((int64_t)units.size() > max_mbs || nr > max_ranks)
    return fail(BS_HDP_ERR_CAPACITY, "the plan has %zu micro-batches and %lld rank entries",
                units.size(), (long long)nr);
  int32_t so = 0;
  int64_t ro = 0;
  for (size_t k = 0; k < units.size(); ++k) {
    const Unit& u = units[k];
    mbs[k] = bs_hdp_microbatch{so, (int32_t)u.seqs.size(), (int32_t)ro, (int32_t)u.ranks.size(),
                               u.r, u.start, u.t};
    for (int32_t i : u.seqs) seqs[so++] = i;
    for (int32_t g : u.ranks) ranks[ro++] = g;
  }
  *n_mbs = (int32_t)units.size();
  for (int32_t g = 0; g < d_hdp; ++g) rank_time[g] = fin[g];
  return ok();
}

const char* bs_hdp_last_error(void) { return g_err; }

}  // extern "C"
