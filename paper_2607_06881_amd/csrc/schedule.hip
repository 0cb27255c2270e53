// Product schedules of the level GEMMs: which FP64 GEMMs produce the levels
// G_t = sum over p + q = t of DA_p DB_q, t <= T (section 2, equation (3)).
// Host code only; declarations and the table format are in schedule.h.
//
// The Karatsuba schedule treats the digits of an element as the coefficients
// of a polynomial in x = 2^-w and forms the low part (degrees 0..T) of the
// product of two such polynomials recursively.  For A = A0 + x^k A1 and
// B = B0 + x^k B1 (A0, B0 the first k coefficients):
//   schoolbook:  A B = A0 B0 + x^k (A0 B1 + A1 B0) + x^2k A1 B1
//   Karatsuba:   A B = A0 B0 + x^k [(A0 + A1)(B0 + B1) - A0 B0 - A1 B1] + x^2k A1 B1
// each truncated at degree T, so that the sub-products only need their own
// low parts.  Unbalanced splits are allowed (a short product of 8 digits is
// cheapest as a 6 + 2 split: 24 products instead of 36).  A "term" is one
// product of two combinations (a coefficient of a sub-polynomial is a sum of
// original digits); terms with the same (combination a, combination b) are
// merged, and terms with the same level coefficients share a GEMM job whose
// output plane enters those levels.
#include "schedule.h"

#include <algorithm>
#include <map>
#include <set>
#include <tuple>
#include <utility>

namespace mdg {
namespace {

struct Term {
  uint64_t ma, mb;                      // digit sets of the two combinations
  std::vector<std::pair<int, int>> v;   // (level, coefficient), increasing level
};
using Terms = std::vector<Term>;

inline int popcount64(uint64_t x) { return __builtin_popcountll(x); }
inline int64_t weight(const Term& t) { return static_cast<int64_t>(popcount64(t.ma)) * popcount64(t.mb); }

// Terms with equal combination pairs added, levels above T and zero
// coefficients dropped; deterministic order (by combination pair).
Terms merged(const Terms& in, int T) {
  struct Item {
    uint64_t ma, mb;
    int level, coef;
  };
  std::vector<Item> items;
  for (const Term& t : in)
    for (const auto& lc : t.v)
      if (lc.first <= T) items.push_back({t.ma, t.mb, lc.first, lc.second});
  std::sort(items.begin(), items.end(), [](const Item& x, const Item& y) {
    return std::tie(x.ma, x.mb, x.level) < std::tie(y.ma, y.mb, y.level);
  });
  Terms out;
  for (size_t i = 0; i < items.size();) {
    Term t{items[i].ma, items[i].mb, {}};
    while (i < items.size() && items[i].ma == t.ma && items[i].mb == t.mb) {
      const int level = items[i].level;
      int c = 0;
      for (; i < items.size() && items[i].ma == t.ma && items[i].mb == t.mb && items[i].level == level; ++i)
        c += items[i].coef;
      if (c != 0) t.v.push_back({level, c});
    }
    if (!t.v.empty()) out.push_back(std::move(t));
  }
  return out;
}

void append_shifted(Terms& out, const Terms& in, int shift, int sign, int sa, int sb, int max_level) {
  for (const Term& t : in) {
    Term u{t.ma << sa, t.mb << sb, {}};
    for (const auto& lc : t.v)
      if (lc.first <= max_level) u.v.push_back({lc.first + shift, sign * lc.second});
    if (!u.v.empty()) out.push_back(std::move(u));
  }
}

// Position i of (A0 + A1) is position i of A (if i < n0) plus position i + k (if i < n1).
uint64_t spread(uint64_t m, int k, int n0, int n1) {
  uint64_t out = 0;
  for (int i = 0; m; ++i, m >>= 1)
    if (m & 1u) {
      if (i < n0) out |= 1ull << i;
      if (i < n1) out |= 1ull << (i + k);
    }
  return out;
}

constexpr int kShortSplit = 16;

class Planner {
 public:
  Planner(int64_t budget, const ScheduleCosts& costs) : budget_(budget), costs_(costs) {}

  // Terms for the coefficients 0..T of the product of an na-coefficient and an
  // nb-coefficient polynomial whose coefficients are single positions.
  const Terms& build(int na, int nb, int T) {
    if (na <= 0 || nb <= 0 || T < 0) return empty_;
    T = std::min(T, na + nb - 2);
    const auto key = std::make_tuple(na, nb, T);
    auto it = memo_.find(key);
    if (it != memo_.end()) return it->second;

    Terms best;
    for (int i = 0; i < na; ++i)
      for (int j = 0; j < nb && i + j <= T; ++j) best.push_back(Term{1ull << i, 1ull << j, {{i + j, 1}}});
    double best_cost = cost(best);

    const int n = std::max(na, nb);
    // split points: halves, and for short polynomials the unbalanced splits too
    std::set<int> ks = {n / 2, (n + 1) / 2, (3 * n) / 4};
    if (n <= kShortSplit) ks.insert({(2 * n) / 3, (3 * n + 3) / 4, n - 1, n - 2});
    for (int k : ks) {
      if (k < 1 || k >= n) continue;
      const int a0 = std::min(k, na), a1 = std::max(0, na - k);
      const int b0 = std::min(k, nb), b1 = std::max(0, nb - k);
      // schoolbook split
      {
        Terms c = build(a0, b0, T);
        append_shifted(c, build(a0, b1, T - k), k, 1, 0, k, T);
        append_shifted(c, build(a1, b0, T - k), k, 1, k, 0, T);
        append_shifted(c, build(a1, b1, T - 2 * k), 2 * k, 1, k, k, T);
        consider(merged(c, T), best, best_cost);
      }
      // Karatsuba split
      if (a1 > 0 && b1 > 0 && T >= k) {
        const int la = std::max(a0, a1), lb = std::max(b0, b1);
        const Terms t00 = build(a0, b0, T);
        const Terms t11 = build(a1, b1, T - k);
        Terms tm = build(la, lb, T - k);
        for (Term& t : tm) {
          t.ma = spread(t.ma, k, a0, a1);
          t.mb = spread(t.mb, k, b0, b1);
        }
        Terms c = t00;
        append_shifted(c, t00, k, -1, 0, 0, T - k);
        append_shifted(c, t11, 2 * k, 1, k, k, T);
        append_shifted(c, t11, k, -1, k, k, T - k);
        append_shifted(c, tm, k, 1, 0, 0, T);
        consider(merged(c, T), best, best_cost);
      }
    }
    return memo_.emplace(key, std::move(best)).first->second;
  }

 private:
  // terms + planes (distinct level vectors) + entries + multi-digit combinations
  double cost(const Terms& t) const {
    std::vector<const std::vector<std::pair<int, int>>*> v;
    std::vector<uint64_t> ma, mb;
    for (const Term& x : t) {
      v.push_back(&x.v);
      if (popcount64(x.ma) > 1) ma.push_back(x.ma);
      if (popcount64(x.mb) > 1) mb.push_back(x.mb);
    }
    std::sort(v.begin(), v.end(), [](auto* x, auto* y) { return *x < *y; });
    v.erase(std::unique(v.begin(), v.end(), [](auto* x, auto* y) { return *x == *y; }), v.end());
    size_t entries = 0;
    for (auto* x : v) entries += x->size();
    std::sort(ma.begin(), ma.end());
    std::sort(mb.begin(), mb.end());
    const size_t ca = std::unique(ma.begin(), ma.end()) - ma.begin();
    const size_t cb = std::unique(mb.begin(), mb.end()) - mb.begin();
    return static_cast<double>(t.size()) + costs_.plane * static_cast<double>(v.size()) +
           costs_.entry * static_cast<double>(entries) + costs_.combo_a * static_cast<double>(ca) +
           costs_.combo_b * static_cast<double>(cb);
  }
  void consider(Terms&& c, Terms& best, double& best_cost) const {
    for (const Term& t : c)
      if (weight(t) > budget_) return;
    const double cc = cost(c);
    if (cc < best_cost) {
      best_cost = cc;
      best = std::move(c);
    }
  }

  int64_t budget_;
  ScheduleCosts costs_;
  std::map<std::tuple<int, int, int>, Terms> memo_;
  const Terms empty_;
};

// Combinations of one operand: digits 0..S-1, then every needed digit set as a
// sum of two disjoint sets already present (the largest available subset whose
// complement is present, else the complement is built first).
struct Combos {
  std::vector<uint64_t> mask;
  std::vector<int> p1, p2, depth;
  std::map<uint64_t, int> index;

  explicit Combos(int S) {
    for (int s = 0; s < S; ++s) add(1ull << s, -1, -1);
  }
  int add(uint64_t m, int a, int b) {
    const int id = static_cast<int>(mask.size());
    mask.push_back(m);
    p1.push_back(a);
    p2.push_back(b);
    depth.push_back(a < 0 ? 0 : 1 + std::max(depth[a], depth[b]));
    index[m] = id;
    return id;
  }
  int make(uint64_t m) {
    auto it = index.find(m);
    if (it != index.end()) return it->second;
    // largest present proper subset whose complement is present
    int best = -1, best_pc = 0, fallback = -1, fallback_pc = 0;
    for (const auto& e : index) {
      const uint64_t x = e.first;
      if ((x & ~m) != 0 || x == m) continue;
      const int pc = popcount64(x);
      if (index.count(m & ~x) && pc > best_pc) {
        best = e.second;
        best_pc = pc;
      }
      if (pc > fallback_pc) {
        fallback = e.second;
        fallback_pc = pc;
      }
    }
    if (best >= 0) {
      const uint64_t x = mask[best];
      return add(m, best, index.at(m & ~x));
    }
    const uint64_t x = mask[fallback];
    const int rest = make(m & ~x);
    return add(m, fallback, rest);
  }
};

}  // namespace

Schedule pair_schedule(int S, int T) {
  Schedule s;
  s.S = S;
  s.T = T;
  s.direct_levels = true;
  for (int c = 0; c < S; ++c) {
    // digit sets are read only for combinations, which take digits 0..63
    s.mask_a.push_back(c < kMaxComboDigits ? 1ull << c : 0ull);
    s.mask_b.push_back(c < kMaxComboDigits ? 1ull << c : 0ull);
    s.par1_a.push_back(-1);
    s.par2_a.push_back(-1);
    s.par1_b.push_back(-1);
    s.par2_b.push_back(-1);
    s.depth_a.push_back(0);
    s.depth_b.push_back(0);
  }
  std::vector<int> order;
  auto lo = [S](int t) { return std::max(0, t - (S - 1)); };
  auto hi = [S](int t) { return std::min(t, S - 1); };
  for (int t = 0; t <= T; ++t) order.push_back(t);
  std::stable_sort(order.begin(), order.end(),
                   [&](int x, int y) { return hi(x) - lo(x) > hi(y) - lo(y); });
  for (int t : order) {
    s.job_first.push_back(static_cast<int>(s.pair_a.size()));
    s.job_count.push_back(hi(t) - lo(t) + 1);
    s.job_out.push_back(t);
    for (int p = lo(t); p <= hi(t); ++p) {
      s.pair_a.push_back(p);
      s.pair_b.push_back(t - p);
    }
    s.max_job_weight = std::max<int64_t>(s.max_job_weight, hi(t) - lo(t) + 1);
  }
  s.terms = static_cast<int>(s.pair_a.size());
  s.planes = T + 1;
  for (int t = 0; t <= T; ++t) {
    s.plane_first.push_back(t);
    s.entry_level.push_back(t);
    s.entry_coef.push_back(1);
  }
  s.plane_first.push_back(T + 1);
  return s;
}

Schedule group_schedule(int S, int T, int Ge, bool sign) {
  const int G = (sign ? 2 : 1) * Ge;
  auto off = [Ge](int g) { return g % Ge; };  // exponent class of group g, in digits
  const int Tg = T + 2 * (Ge - 1);
  Schedule s;
  s.S = G * S;
  s.T = Tg;
  s.direct_levels = true;
  for (int c = 0; c < G * S; ++c) {
    s.mask_a.push_back(0ull);  // no combinations: digit sets are never read
    s.mask_b.push_back(0ull);
    s.par1_a.push_back(-1);
    s.par2_a.push_back(-1);
    s.par1_b.push_back(-1);
    s.par2_b.push_back(-1);
    s.depth_a.push_back(0);
    s.depth_b.push_back(0);
  }
  std::vector<std::vector<std::pair<int, int>>> lv(Tg + 1);
  for (int g = 0; g < G; ++g)
    for (int h = 0; h < G; ++h)
      for (int p = 0; p < S; ++p)
        for (int q = 0; q < S && p + q <= T; ++q) lv[p + q + off(g) + off(h)].push_back({g * S + p, h * S + q});
  std::vector<int> order;
  for (int t = 0; t <= Tg; ++t) order.push_back(t);
  std::stable_sort(order.begin(), order.end(), [&](int x, int y) { return lv[x].size() > lv[y].size(); });
  for (int t : order) {
    if (lv[t].empty()) continue;  // (cannot happen: level t always has the pair (0, t) of some class pair)
    s.job_first.push_back(static_cast<int>(s.pair_a.size()));
    s.job_count.push_back(static_cast<int>(lv[t].size()));
    s.job_out.push_back(t);
    for (const auto& pq : lv[t]) {
      s.pair_a.push_back(pq.first);
      s.pair_b.push_back(pq.second);
    }
    s.max_job_weight = std::max<int64_t>(s.max_job_weight, static_cast<int64_t>(lv[t].size()));
  }
  s.terms = static_cast<int>(s.pair_a.size());
  s.planes = Tg + 1;
  for (int t = 0; t <= Tg; ++t) {
    s.plane_first.push_back(t);
    s.entry_level.push_back(t);
    s.entry_coef.push_back(1);
  }
  s.plane_first.push_back(Tg + 1);
  return s;
}

Schedule per_pair_schedule(int S, int T) {
  Schedule s = pair_schedule(S, T);
  s.job_first.clear();
  s.job_count.clear();
  s.job_out.clear();
  s.pair_a.clear();
  s.pair_b.clear();
  s.plane_first.clear();
  s.entry_level.clear();
  s.entry_coef.clear();
  s.planes = S * S;
  for (int p = 0; p < S; ++p)
    for (int q = 0; q < S; ++q) {
      s.plane_first.push_back(static_cast<int>(s.entry_level.size()));
      if (p + q > T) continue;
      s.job_first.push_back(static_cast<int>(s.pair_a.size()));
      s.job_count.push_back(1);
      s.job_out.push_back(p * S + q);
      s.pair_a.push_back(p);
      s.pair_b.push_back(q);
      s.entry_level.push_back(p + q);
      s.entry_coef.push_back(1);
    }
  s.plane_first.push_back(static_cast<int>(s.entry_level.size()));
  s.terms = static_cast<int>(s.pair_a.size());
  s.max_job_weight = 1;
  return s;
}

double schedule_cost(const Schedule& s, const ScheduleCosts& costs) {
  return static_cast<double>(s.terms) + costs.plane * s.planes +
         costs.entry * static_cast<double>(s.entry_level.size()) +
         costs.combo_a * static_cast<double>(s.mask_a.size() - s.S) +
         costs.combo_b * static_cast<double>(s.mask_b.size() - s.S);
}

Schedule karatsuba_schedule(int S, int T, int64_t budget, const ScheduleCosts& costs, bool fallback) {
  // combinations carry their digit sets in 64-bit masks: more digits keep the pair schedule
  if (S > kMaxComboDigits) return pair_schedule(S, T);
  Planner planner(budget, costs);
  const Terms terms = planner.build(S, S, T);
  Schedule pairs = pair_schedule(S, T);
  if (terms.empty() || static_cast<int>(terms.size()) >= pairs.terms) return pairs;

  Schedule s;
  s.S = S;
  s.T = T;
  s.direct_levels = false;
  s.terms = static_cast<int>(terms.size());
  Combos ca(S), cb(S);
  // combinations in increasing digit count, so that small sums exist first
  std::vector<uint64_t> need_a, need_b;
  for (const Term& t : terms) {
    need_a.push_back(t.ma);
    need_b.push_back(t.mb);
  }
  auto by_count = [](uint64_t x, uint64_t y) {
    return popcount64(x) != popcount64(y) ? popcount64(x) < popcount64(y) : x < y;
  };
  std::sort(need_a.begin(), need_a.end(), by_count);
  std::sort(need_b.begin(), need_b.end(), by_count);
  for (uint64_t m : need_a) ca.make(m);
  for (uint64_t m : need_b) cb.make(m);
  s.mask_a = ca.mask;
  s.par1_a = ca.p1;
  s.par2_a = ca.p2;
  s.depth_a = ca.depth;
  s.mask_b = cb.mask;
  s.par1_b = cb.p1;
  s.par2_b = cb.p2;
  s.depth_b = cb.depth;

  // group by level coefficients; pack each group into jobs within the budget
  std::map<std::vector<std::pair<int, int>>, std::vector<const Term*>> groups;
  for (const Term& t : terms) groups[t.v].push_back(&t);
  struct Job {
    std::vector<const Term*> t;
    int64_t w = 0;
    const std::vector<std::pair<int, int>>* v = nullptr;
  };
  std::vector<Job> jobs;
  for (auto& g : groups) {
    std::vector<const Term*> ts = g.second;
    std::stable_sort(ts.begin(), ts.end(), [](const Term* x, const Term* y) { return weight(*x) > weight(*y); });
    const size_t first = jobs.size();
    for (const Term* t : ts) {
      size_t j = first;
      while (j < jobs.size() && jobs[j].w + weight(*t) > budget) ++j;
      if (j == jobs.size()) {
        jobs.emplace_back();
        jobs.back().v = &g.first;
      }
      jobs[j].t.push_back(t);
      jobs[j].w += weight(*t);
    }
  }
  std::stable_sort(jobs.begin(), jobs.end(), [](const Job& x, const Job& y) { return x.t.size() > y.t.size(); });
  s.planes = static_cast<int>(jobs.size());
  for (size_t j = 0; j < jobs.size(); ++j) {
    s.job_first.push_back(static_cast<int>(s.pair_a.size()));
    s.job_count.push_back(static_cast<int>(jobs[j].t.size()));
    s.job_out.push_back(static_cast<int>(j));
    for (const Term* t : jobs[j].t) {
      s.pair_a.push_back(ca.index.at(t->ma));
      s.pair_b.push_back(cb.index.at(t->mb));
    }
    s.max_job_weight = std::max(s.max_job_weight, jobs[j].w);
    s.plane_first.push_back(static_cast<int>(s.entry_level.size()));
    for (const auto& lc : *jobs[j].v) {
      s.entry_level.push_back(lc.first);
      s.entry_coef.push_back(lc.second);
    }
  }
  s.plane_first.push_back(static_cast<int>(s.entry_level.size()));
  if (fallback && schedule_cost(s, costs) >= schedule_cost(pairs, costs)) return pairs;
  return s;
}

Schedule split_k(const Schedule& s, int sigma) {
  if (sigma <= 1) return s;
  Schedule r = s;
  r.direct_levels = false;
  r.ksplit = sigma;
  r.job_first.clear();
  r.job_count.clear();
  r.job_out.clear();
  r.job_chunk.clear();
  r.plane_first.clear();
  r.entry_level.clear();
  r.entry_coef.clear();
  int plane = 0;
  for (size_t j = 0; j < s.job_first.size(); ++j) {
    std::vector<std::pair<int, int>> ent;  // the level entries of job j's plane
    if (s.direct_levels) {
      ent.push_back({s.job_out[j], 1});
    } else {
      const int pl = s.job_out[j];
      for (int e = s.plane_first[pl]; e < s.plane_first[pl + 1]; ++e)
        ent.push_back({s.entry_level[e], s.entry_coef[e]});
    }
    for (int c = 0; c < sigma; ++c) {
      r.job_first.push_back(s.job_first[j]);
      r.job_count.push_back(s.job_count[j]);
      r.job_out.push_back(plane++);
      r.job_chunk.push_back(c);
      r.plane_first.push_back(static_cast<int>(r.entry_level.size()));
      for (const auto& lc : ent) {
        r.entry_level.push_back(lc.first);
        r.entry_coef.push_back(lc.second);
      }
    }
  }
  r.plane_first.push_back(static_cast<int>(r.entry_level.size()));
  r.planes = plane;
  return r;
}

ScheduleTable schedule_table(const Schedule& s) {
  ScheduleTable t;
  const size_t J = s.job_first.size();
  t.jobs_off = 0;
  for (size_t j = 0; j < J; ++j) {
    t.words.push_back(static_cast<uint32_t>(s.job_first[j]) | (static_cast<uint32_t>(s.job_count[j]) << 16));
    t.words.push_back(static_cast<uint32_t>(s.job_out[j]));
    const uint32_t chunk = s.job_chunk.empty() ? 0u : static_cast<uint32_t>(s.job_chunk[j]);
    t.words.push_back(chunk | (static_cast<uint32_t>(s.ksplit) << 16));
  }
  t.pairs_off = static_cast<int64_t>(t.words.size());
  for (size_t i = 0; i < s.pair_a.size(); ++i)
    t.words.push_back(static_cast<uint32_t>(s.pair_a[i]) | (static_cast<uint32_t>(s.pair_b[i]) << 16));
  // accumulation chunks: four 16-bit entries per chunk, planes padded to whole chunks
  std::vector<uint32_t> chunk_first, chunks;
  const uint32_t trash = static_cast<uint32_t>(s.T + 1);
  for (int j = 0; j < s.planes; ++j) {
    chunk_first.push_back(static_cast<uint32_t>(chunks.size() / 2));
    std::vector<uint32_t> e;
    for (int i = s.plane_first[j]; i < s.plane_first[j + 1]; ++i)
      e.push_back(static_cast<uint32_t>(s.entry_level[i]) |
                  (static_cast<uint32_t>(static_cast<uint8_t>(static_cast<int8_t>(s.entry_coef[i]))) << 8));
    while (e.size() % 4) e.push_back(trash);
    for (size_t i = 0; i < e.size(); i += 2) chunks.push_back(e[i] | (e[i + 1] << 16));
  }
  chunk_first.push_back(static_cast<uint32_t>(chunks.size() / 2));
  t.chunk_first_off = static_cast<int64_t>(t.words.size());
  t.words.insert(t.words.end(), chunk_first.begin(), chunk_first.end());
  // chunks start on an even word: one 8-byte load each
  if (t.words.size() % 2) t.words.push_back(0);
  t.chunks_off = static_cast<int64_t>(t.words.size());
  t.words.insert(t.words.end(), chunks.begin(), chunks.end());
  // combination digit sets (the split writes the combinations beside the digits)
  t.masks_a_off = static_cast<int64_t>(t.words.size());
  for (uint64_t m : s.mask_a) {
    t.words.push_back(static_cast<uint32_t>(m));
    t.words.push_back(static_cast<uint32_t>(m >> 32));
  }
  t.masks_b_off = static_cast<int64_t>(t.words.size());
  for (uint64_t m : s.mask_b) {
    t.words.push_back(static_cast<uint32_t>(m));
    t.words.push_back(static_cast<uint32_t>(m >> 32));
  }
  return t;
}

}  // namespace mdg
