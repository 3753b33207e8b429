// Exact per-projection bit allocation (host).
//
// The paper's ILP (Sec. 3.3, Eq. ilp_piecewise_projection; App. B.4, Eq.
// ilp_piecewise_eps) picks one width per spectral unit to minimize the summed
// loss under a total-bit budget: a multiple-choice knapsack.  It is solved
// exactly here, without an external MILP solver:
//
//  1. Costs are mapped to int64, rint(L * 2^K / max|L|) with
//     K = 62 - ceil(log2(units + 1)), so every sum below is exact.
//  2. Small instances: a dynamic program over the extra bits above the
//     narrowest width, with a forward pass that keeps the smallest width that
//     still attains the optimum (the lexicographically smallest optimal width
//     vector).
//  3. Large instances: the LP relaxation is solved by the greedy over the
//     upper convex hulls of every unit's (extra bits, saving) points, giving a
//     multiplier lambda = p/q and a feasible integer solution of value LB.
//     With UB = sum_u max_j (s_uj - lambda w_j) + lambda * cap, every optimum
//     y satisfies sum_u rc_u(y_u) + lambda * slack(y) <= UB - LB, where
//     rc_u(j) = max_k (s_uk - lambda w_k) - (s_uj - lambda w_j) >= 0.  So a
//     width with rc > UB - LB is used by no optimum: units left with a single
//     admissible width are fixed, and the dynamic program of step 2 runs on
//     the remaining ("core") units with their admissible widths only.  All
//     comparisons are exact integer arithmetic (lambda kept as p/q, products
//     in 128 bits).
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <string>
#include <vector>

#include "bitsmoe.h"
#include "internal.hpp"

using namespace bitsmoe;

namespace {

using i128 = __int128;

constexpr int64_t kDefaultFullDp = int64_t(1) << 26;
constexpr int64_t kMaxDpEntries = int64_t(1) << 30;  // 8 GiB of int64 tables

int bit_length(uint64_t v) { return v == 0 ? 0 : 64 - __builtin_clzll(v); }

// Exact DP over `units` (indices into the problem) with admissible-width masks.
// Minimizes sum Li[u][j] subject to sum ex[j] <= cap over those units; writes
// the lexicographically smallest optimal choice into choice[u].
struct CoreDp {
  const int64_t* Li;
  int nb;
  const int* ex;
  const std::vector<int64_t>& units;
  const std::vector<uint32_t>& mask;  // per listed unit: admissible widths
  int64_t cap;

  bitsmoe_status run(std::vector<int>* choice) const {
    const int64_t n = static_cast<int64_t>(units.size());
    if (n == 0) return BITSMOE_OK;
    // Shift every unit by its narrowest admissible width.
    std::vector<int> wmin(n), wmax(n);
    int64_t base = 0, span = 0;
    for (int64_t i = 0; i < n; ++i) {
      int lo = 1 << 30, hi = -1;
      for (int j = 0; j < nb; ++j)
        if (mask[i] >> j & 1u) {
          lo = std::min(lo, ex[j]);
          hi = std::max(hi, ex[j]);
        }
      wmin[i] = lo;
      wmax[i] = hi;
      base += lo;
      span += hi - lo;
    }
    const int64_t capc = std::min(cap - base, span);
    if (capc < 0) return fail(BITSMOE_ERR_INFEASIBLE, "allocate: core capacity negative");
    const int64_t S = capc + 1;
    int64_t block = 256;
    const bool full = n * S <= (int64_t(1) << 26);
    if (!full) {
      if ((n / block + 2 + block) * S > kMaxDpEntries)
        return fail(BITSMOE_ERR_NOMEM, "allocate: exact search too large (" + std::to_string(n) +
                                           " units x " + std::to_string(S) + " states)");
    }
    auto step = [&](const int64_t* gnext, int64_t i, int64_t* g) {
      const int64_t u = units[i];
      const int64_t* row = Li + u * nb;
      for (int64_t c = 0; c < S; ++c) g[c] = INT64_MAX;
      for (int j = 0; j < nb; ++j) {
        if (!(mask[i] >> j & 1u)) continue;
        const int e = ex[j] - wmin[i];
        if (e >= S) continue;
        const int64_t cost = row[j];
        for (int64_t c = e; c < S; ++c) {
          const int64_t v = gnext[c - e] + cost;
          if (v < g[c]) g[c] = v;
        }
      }
    };
    auto pick = [&](int64_t i, const int64_t* gi, const int64_t* gn, int64_t* c) -> bool {
      const int64_t u = units[i];
      const int64_t* row = Li + u * nb;
      for (int j = 0; j < nb; ++j) {
        if (!(mask[i] >> j & 1u)) continue;
        const int e = ex[j] - wmin[i];
        if (e > *c) continue;
        if (gn[*c - e] + row[j] == gi[*c]) {
          (*choice)[u] = j;
          *c -= e;
          return true;
        }
      }
      return false;
    };
    std::vector<int64_t> zero(S, 0);
    if (full) {
      std::vector<int64_t> T(static_cast<size_t>(n + 1) * S);
      std::memcpy(&T[static_cast<size_t>(n) * S], zero.data(), S * sizeof(int64_t));
      for (int64_t i = n - 1; i >= 0; --i) step(&T[(i + 1) * S], i, &T[i * S]);
      int64_t c = capc;
      for (int64_t i = 0; i < n; ++i)
        if (!pick(i, &T[i * S], &T[(i + 1) * S], &c))
          return fail(BITSMOE_ERR_NUMERIC, "allocate: reconstruction failed");
      return BITSMOE_OK;
    }
    // Checkpointed: keep g_i for i % block == 0 and g_n; recompute blocks.
    const int64_t nck = n / block + 1;
    std::vector<int64_t> ck(static_cast<size_t>(nck + 1) * S);
    std::vector<int64_t> cur(zero), nxt(S);
    std::memcpy(&ck[static_cast<size_t>(nck) * S], zero.data(), S * sizeof(int64_t));  // g_n
    for (int64_t i = n - 1; i >= 0; --i) {
      step(cur.data(), i, nxt.data());
      std::swap(cur, nxt);
      if (i % block == 0) std::memcpy(&ck[(i / block) * S], cur.data(), S * sizeof(int64_t));
    }
    std::vector<int64_t> T(static_cast<size_t>(block + 1) * S);
    int64_t c = capc;
    for (int64_t i0 = 0; i0 < n; i0 += block) {
      const int64_t i1 = std::min(i0 + block, n);
      const int64_t len = i1 - i0;
      const int64_t* top = (i1 == n) ? &ck[static_cast<size_t>(nck) * S] : &ck[(i1 / block) * S];
      std::memcpy(&T[len * S], top, S * sizeof(int64_t));
      for (int64_t t = len - 1; t >= 1; --t) step(&T[(t + 1) * S], i0 + t, &T[t * S]);
      std::memcpy(&T[0], &ck[(i0 / block) * S], S * sizeof(int64_t));
      for (int64_t i = i0; i < i1; ++i)
        if (!pick(i, &T[(i - i0) * S], &T[(i - i0 + 1) * S], &c))
          return fail(BITSMOE_ERR_NUMERIC, "allocate: reconstruction failed");
    }
    return BITSMOE_OK;
  }
};

struct Segment {
  int64_t u;
  int from, to;
  int64_t dw, ds;  // dw > 0, ds > 0
};

}  // namespace

extern "C" bitsmoe_status bitsmoe_allocate_ex(const float* L_host, int64_t units,
                                              const int* bits_host, int nbits, int64_t budget_bits,
                                              uint8_t* bits_out_host, double* objective_out,
                                              int64_t full_dp_limit, int64_t* core_units_out) {
  if (!L_host || !bits_host || !bits_out_host) return fail(BITSMOE_ERR_ARG, "allocate: null pointer");
  if (units <= 0) return fail(BITSMOE_ERR_ARG, "allocate: units must be positive");
  if (nbits < 1 || nbits > BITSMOE_MAX_NBITS) return fail(BITSMOE_ERR_ARG, "allocate: nbits outside 1..8");
  for (int j = 0; j < nbits; ++j) {
    if (bits_host[j] < 0 || bits_host[j] > BITSMOE_ALLOC_MAX_BITS)
      return fail(BITSMOE_ERR_ARG, "allocate: width outside 0..16");
    if (j > 0 && bits_host[j] <= bits_host[j - 1])
      return fail(BITSMOE_ERR_ARG, "allocate: widths must be strictly ascending");
  }
  if (full_dp_limit < 0) full_dp_limit = kDefaultFullDp;
  const int nb = nbits;
  if (budget_bits < static_cast<int64_t>(bits_host[0]) * units)
    return fail(BITSMOE_ERR_INFEASIBLE, "allocate: budget below min(bits) * units");

  // 1. integerize
  double maxabs = 0.0;
  const size_t total = static_cast<size_t>(units) * nb;
  for (size_t i = 0; i < total; ++i) {
    const double v = static_cast<double>(L_host[i]);
    if (!std::isfinite(v)) return fail(BITSMOE_ERR_NUMERIC, "allocate: non-finite cost");
    maxabs = std::max(maxabs, std::fabs(v));
  }
  std::vector<int64_t> Li;
  try {
    Li.assign(total, 0);
  } catch (...) {
    return fail(BITSMOE_ERR_NOMEM, "allocate: host allocation failed");
  }
  if (maxabs > 0.0) {
    const int K = 62 - bit_length(static_cast<uint64_t>(units));
    const double scale = std::ldexp(1.0, K) / maxabs;
    for (size_t i = 0; i < total; ++i) Li[i] = std::llrint(static_cast<double>(L_host[i]) * scale);
  }
  int ex[BITSMOE_MAX_NBITS];
  for (int j = 0; j < nb; ++j) ex[j] = bits_host[j] - bits_host[0];
  int64_t cap = budget_bits - static_cast<int64_t>(bits_host[0]) * units;
  cap = std::min<int64_t>(cap, units * static_cast<int64_t>(ex[nb - 1]));

  std::vector<int> choice(static_cast<size_t>(units), 0);
  std::vector<int64_t> core;
  std::vector<uint32_t> mask;
  const uint32_t all = (nb >= 32) ? 0xffffffffu : ((1u << nb) - 1u);

  if (units * (cap + 1) <= full_dp_limit || nb == 1) {
    core.resize(static_cast<size_t>(units));
    for (int64_t u = 0; u < units; ++u) core[u] = u;
    mask.assign(static_cast<size_t>(units), all);
    CoreDp dp{Li.data(), nb, ex, core, mask, cap};
    bitsmoe_status st = dp.run(&choice);
    if (st != BITSMOE_OK) return st;
  } else {
    // 3a. upper hulls of (extra bits, saving) per unit, positive slopes only
    std::vector<Segment> segs;
    segs.reserve(static_cast<size_t>(units) * (nb - 1));
    std::vector<int> hull(nb);
    for (int64_t u = 0; u < units; ++u) {
      const int64_t* row = &Li[u * nb];
      auto sav = [&](int j) { return row[0] - row[j]; };
      int h = 0;
      hull[h++] = 0;
      for (int j = 1; j < nb; ++j) {
        while (h >= 2) {
          const int a = hull[h - 2], b = hull[h - 1];
          const i128 lhs = static_cast<i128>(sav(b) - sav(a)) * (ex[j] - ex[b]);
          const i128 rhs = static_cast<i128>(sav(j) - sav(b)) * (ex[b] - ex[a]);
          if (lhs <= rhs) --h; else break;
        }
        hull[h++] = j;
      }
      for (int t = 1; t < h; ++t) {
        const int64_t ds = sav(hull[t]) - sav(hull[t - 1]);
        if (ds <= 0) break;
        segs.push_back({u, hull[t - 1], hull[t], ex[hull[t]] - ex[hull[t - 1]], ds});
      }
    }
    std::sort(segs.begin(), segs.end(), [](const Segment& a, const Segment& b) {
      const i128 l = static_cast<i128>(a.ds) * b.dw, r = static_cast<i128>(b.ds) * a.dw;
      if (l != r) return l > r;
      if (a.u != b.u) return a.u < b.u;
      return a.from < b.from;
    });
    // 3b. greedy (LP order); the first segment that does not fit is critical
    std::vector<int> pos(static_cast<size_t>(units), 0);
    int64_t rem = cap;
    int64_t p = 0, q = 1;
    bool have_crit = false;
    for (const Segment& s : segs) {
      if (pos[s.u] != s.from) continue;
      if (s.dw <= rem) {
        pos[s.u] = s.to;
        rem -= s.dw;
      } else if (!have_crit) {
        have_crit = true;
        p = s.ds;
        q = s.dw;
      }
    }
    // 3c. bounds and reduced-cost fixing
    i128 LB = 0, UBq = static_cast<i128>(p) * cap;
    std::vector<i128> best(static_cast<size_t>(units));
    for (int64_t u = 0; u < units; ++u) {
      const int64_t* row = &Li[u * nb];
      LB += row[0] - row[pos[u]];
      i128 m = 0;
      for (int j = 0; j < nb; ++j) {
        const i128 v = static_cast<i128>(q) * (row[0] - row[j]) - static_cast<i128>(p) * ex[j];
        if (j == 0 || v > m) m = v;
      }
      best[u] = m;
      UBq += m;
    }
    const i128 gapq = UBq - static_cast<i128>(q) * LB;
    if (gapq < 0) return fail(BITSMOE_ERR_NUMERIC, "allocate: negative LP gap");
    int64_t capc = cap;
    for (int64_t u = 0; u < units; ++u) {
      const int64_t* row = &Li[u * nb];
      uint32_t mk = 0;
      int cnt = 0, only = 0;
      for (int j = 0; j < nb; ++j) {
        const i128 v = static_cast<i128>(q) * (row[0] - row[j]) - static_cast<i128>(p) * ex[j];
        if (best[u] - v <= gapq) {
          mk |= 1u << j;
          ++cnt;
          only = j;
        }
      }
      if (cnt == 1) {
        choice[u] = only;
        capc -= ex[only];
      } else {
        core.push_back(u);
        mask.push_back(mk);
      }
    }
    CoreDp dp{Li.data(), nb, ex, core, mask, capc};
    bitsmoe_status st = dp.run(&choice);
    if (st != BITSMOE_OK) return st;
  }
  double obj = 0.0;
  int64_t used = 0;
  for (int64_t u = 0; u < units; ++u) {
    bits_out_host[u] = static_cast<uint8_t>(bits_host[choice[u]]);
    obj += static_cast<double>(L_host[u * nb + choice[u]]);
    used += bits_host[choice[u]];
  }
  if (used > budget_bits) return fail(BITSMOE_ERR_NUMERIC, "allocate: internal budget violation");
  if (objective_out) *objective_out = obj;
  if (core_units_out) *core_units_out = static_cast<int64_t>(core.size());
  return ok();
}

extern "C" bitsmoe_status bitsmoe_allocate(const float* L_host, int64_t units, const int* bits_host,
                                           int nbits, int64_t budget_bits, uint8_t* bits_out_host,
                                           double* objective_out) {
  return bitsmoe_allocate_ex(L_host, units, bits_host, nbits, budget_bits, bits_out_host,
                             objective_out, -1, nullptr);
}
