// Host planner: which chain boundaries to keep, and the exact bytes of the
// executor's static layout for a plan.  Integer arithmetic only, no HIP calls.
//
// Modes (Chen et al., section 4):
//   SQRT       section 4.3, Eq. 1: cost = max segment + O(k); k = sqrt(n)
//              equal segments balance the two.  Stride s = ceil(sqrt n) unless
//              given; cut targets s-1, 2s-1, ... below n-1; a target that is not
//              a candidate moves forward to the next candidate.
//   GREEDY     Alg. 3: running total of per-unit bytes; cut at a candidate
//              whose running total exceeds the budget B (strict), then restart
//              the total.  x, y reported as Alg. 3 computes them.
//   RECURSIVE  section 4.4 (Eq. 2-3, g(n) = k + g(n/(k+1)) = k log_{k+1} n):
//              split every range of length L > 1 into at most k + 1 parts at
//              floor(j L / (k+1)), keep the split boundaries while the parts
//              are handled last to first, dropping each after its part.
//   USER       caller's cut list (the user-settable mirror attribute, 4.5).
//   NONE       one segment with the first forward's activations kept.
#include <algorithm>
#include <cstring>

#include "common.h"

namespace ckpt {

static uint64_t ceil_isqrt(uint64_t n) {
  uint64_t r = 0;
  // largest r with r*r <= n, by bisection on exact integers
  uint64_t lo = 0, hi = 1;
  while (hi * hi <= n) hi <<= 1;
  lo = hi >> 1;
  while (lo + 1 < hi) {
    uint64_t mid = (lo + hi) / 2;
    if (mid * mid <= n) lo = mid; else hi = mid;
  }
  r = lo;
  return r * r == n ? r : r + 1;
}

std::vector<int32_t> rec_splits(int32_t lo, int32_t hi, int32_t k) {
  std::vector<int32_t> s;
  const int64_t L = int64_t(hi) - lo;
  // k >= L - 1 gives every point lo+1 .. hi-1, exactly as k = L - 1 does
  // (steps of L/(k+1) <= 1 reach each integer), so cap the loop there
  const int64_t kk = std::min<int64_t>(k, L - 1);
  for (int64_t j = 1; j <= kk; ++j) {
    const int64_t m = lo + j * L / (kk + 1);
    if (m > lo && m < hi && (s.empty() || m > s.back())) s.push_back(int32_t(m));
  }
  return s;
}

// unit forwards re-run for [a, b): the sweep up to the last split, then the
// parts (a single unit: one re-forward)
static uint64_t rec_range(int32_t a, int32_t b, int32_t k) {
  if (b - a == 1) return 1;
  const std::vector<int32_t> s = rec_splits(a, b, k);
  uint64_t t = uint64_t(s.back() - a);
  int32_t lo = a;
  for (int32_t m : s) {
    t += rec_range(lo, m, k);
    lo = m;
  }
  return t + rec_range(lo, b, k);
}

uint64_t recursive_extra(int32_t n, int32_t k) {
  if (n == 1) return rec_range(0, 1, k);
  const std::vector<int32_t> s = rec_splits(0, n, k);
  uint64_t t = 0;
  int32_t lo = 0;
  for (int32_t m : s) {
    t += rec_range(lo, m, k);
    lo = m;
  }
  return t + rec_range(lo, n, k);
}

static void xy_of_cuts(const uint64_t *lb, const uint64_t *cb, const std::vector<int32_t> &cuts,
                       uint64_t &x, uint64_t &y) {
  x = 0;
  y = 0;
  int32_t lo = 0;
  for (int32_t c : cuts) {
    x += cb[c];
    uint64_t s = 0;
    for (int32_t i = lo; i <= c; ++i) s += lb[i];
    y = std::max(y, s);
    lo = c + 1;
  }
}

Plan make_plan(int32_t n, const uint64_t *lb, const uint64_t *cb, uint64_t budget, int32_t mode,
               const int32_t *user_cuts, int32_t n_user_cuts, int32_t flags) {
  if (n <= 0) fail(CKPT_E_INVALID, "plan_checkpoints: n_layers must be positive");
  if (!lb || !cb) fail(CKPT_E_INVALID, "plan_checkpoints: null size array");
  if (cb[n - 1] != 0) fail(CKPT_E_INVALID, "plan_checkpoints: the last unit cannot be a cut");
  if (flags & ~CKPT_FLAG_KEEP_LAST) fail(CKPT_E_INVALID, "plan_checkpoints: unknown flag bits");
  Plan p;
  p.mode = mode;
  p.n = n;
  p.keep_last = (flags & CKPT_FLAG_KEEP_LAST) != 0;
  switch (mode) {
    case CKPT_NONE:
      p.keep_last = true;
      return p;
    case CKPT_SQRT: {
      uint64_t s = budget > 0 ? budget : ceil_isqrt(uint64_t(n));
      for (uint64_t j = 1;; ++j) {
        uint64_t t = j * s - 1;
        if (t >= uint64_t(n - 1)) break;
        int64_t c = int64_t(t);
        while (c < n - 1 && cb[c] == 0) ++c;
        if (c < n - 1 && (p.cuts.empty() || c > p.cuts.back())) p.cuts.push_back(int32_t(c));
      }
      break;
    }
    case CKPT_GREEDY: {
      // Alg. 3 step by step: temp grows by each unit's bytes; a candidate whose
      // running total exceeds B becomes a cut, adds its kept bytes to x and its
      // segment total to y, and restarts the total.
      uint64_t temp = 0;
      for (int32_t i = 0; i < n; ++i) {
        temp += lb[i];
        if (cb[i] > 0 && temp > budget) {
          p.x += cb[i];
          p.y = std::max(p.y, temp);
          p.cuts.push_back(i);
          temp = 0;
        }
      }
      p.extra = p.keep_last ? (p.cuts.empty() ? 0 : uint64_t(p.cuts.back()) + 1) : uint64_t(n);
      return p;
    }
    case CKPT_USER: {
      if (n_user_cuts < 0 || (n_user_cuts > 0 && !user_cuts))
        fail(CKPT_E_INVALID, "plan_checkpoints: bad user cut list");
      for (int32_t k = 0; k < n_user_cuts; ++k) {
        int32_t c = user_cuts[k];
        if (c < 0 || c >= n - 1 || cb[c] == 0 || (k > 0 && c <= user_cuts[k - 1]))
          fail(CKPT_E_INVALID,
               "plan_checkpoints: user cuts must be strictly ascending candidates below n-1");
        p.cuts.push_back(c);
      }
      break;
    }
    case CKPT_RECURSIVE:
      for (int32_t i = 0; i + 1 < n; ++i)
        if (cb[i] == 0)
          fail(CKPT_E_UNSUPPORTED,
               "plan_checkpoints: the recursive schedule needs every boundary to be a candidate");
      if (budget >= (uint64_t(1) << 31))
        fail(CKPT_E_INVALID, "plan_checkpoints: the recursion fan-out must fit in 31 bits");
      p.keep_last = false;
      p.fanout = budget > 0 ? int32_t(budget) : 1;
      p.extra = recursive_extra(n, p.fanout);
      return p;
    default:
      fail(CKPT_E_INVALID, "plan_checkpoints: unknown mode");
  }
  xy_of_cuts(lb, cb, p.cuts, p.x, p.y);
  if (p.keep_last)
    p.extra = p.cuts.empty() ? 0 : uint64_t(p.cuts.back()) + 1;
  else
    p.extra = uint64_t(n);
  return p;
}

static void put32(std::vector<uint8_t> &v, uint32_t x) {
  for (int i = 0; i < 4; ++i) v.push_back(uint8_t(x >> (8 * i)));
}
static void put64(std::vector<uint8_t> &v, uint64_t x) {
  for (int i = 0; i < 8; ++i) v.push_back(uint8_t(x >> (8 * i)));
}

std::vector<uint8_t> serialize(const Plan &p) {
  std::vector<uint8_t> v = {'C', 'K', 'P', 'L'};
  put32(v, 2);
  put32(v, uint32_t(p.mode));
  put32(v, p.keep_last ? 1u : 0u);
  put32(v, uint32_t(p.fanout));
  put32(v, uint32_t(p.n));
  put32(v, uint32_t(p.cuts.size()));
  for (int32_t c : p.cuts) put32(v, uint32_t(c));
  put64(v, p.x);
  put64(v, p.y);
  put64(v, p.extra);
  return v;
}

// Arena need of a forward sweep over [lo, hi) whose first input lives outside
// the arena; `stored(i)` says unit i's output goes outside the arena.
template <class Stored>
static uint64_t sweep_need(const std::vector<uint64_t> &b, const std::vector<uint64_t> &a,
                           int32_t lo, int32_t hi, Stored stored) {
  uint64_t need = 0;
  for (int32_t i = lo; i < hi; ++i) {
    bool in_arena = i > lo && !stored(i - 1);
    bool out_arena = !stored(i);
    need = std::max(need, (in_arena ? b[i] : 0) + a[i] + (out_arena ? b[i + 1] : 0));
  }
  return need;
}

struct RecState {
  const std::vector<uint64_t> &b, &a;
  int32_t k;
  uint64_t arena = 0, stack = 0, stack_max = 0;
};

static void rec_account(RecState &st, int32_t lo, int32_t hi);

// A forward sweep over [lo, last split) keeps every split boundary; the parts
// are then handled last to first, each split boundary dropped after its part.
static void rec_sweep_and_parts(RecState &st, int32_t lo, int32_t hi, int32_t sweep_hi) {
  const std::vector<int32_t> s = rec_splits(lo, hi, st.k);
  auto is_split_out = [&s](int32_t i) { return std::binary_search(s.begin(), s.end(), i + 1); };
  st.arena = std::max(st.arena, sweep_need(st.b, st.a, lo, sweep_hi, is_split_out));
  for (int32_t m : s) st.stack += st.b[size_t(m)];
  st.stack_max = std::max(st.stack_max, st.stack);
  for (size_t t = s.size() + 1; t-- > 0;) {
    const int32_t p_lo = t == 0 ? lo : s[t - 1], p_hi = t == s.size() ? hi : s[t];
    rec_account(st, p_lo, p_hi);
    if (t > 0) st.stack -= st.b[size_t(s[t - 1])];
  }
}

static void rec_account(RecState &st, int32_t lo, int32_t hi) {
  if (hi - lo == 1) {
    st.arena = std::max(st.arena, st.a[size_t(lo)] + st.b[size_t(lo) + 1]);
    return;
  }
  rec_sweep_and_parts(st, lo, hi, rec_splits(lo, hi, st.k).back());
}

Accounting account(const Plan &p, const std::vector<uint64_t> &b, const std::vector<uint64_t> &a,
                   const std::vector<uint64_t> &q, uint64_t slot, uint64_t extra) {
  const int32_t n = p.n;
  Accounting acc;
  uint64_t maxb = 0, maxq = 0;
  for (int32_t i = 1; i <= n; ++i) maxb = std::max(maxb, b[i]);
  for (int32_t i = 0; i < n; ++i) maxq = std::max(maxq, q[i]);
  acc.grad = 2 * (slot ? slot : maxb) + maxq + extra;
  if (p.mode == CKPT_RECURSIVE) {
    RecState st{b, a, p.fanout};
    if (n == 1) {
      st.arena = sweep_need(b, a, 0, 1, [](int32_t) { return false; });
      rec_account(st, 0, 1);
    } else {
      rec_sweep_and_parts(st, 0, n, n);  // the first forward runs the whole chain
    }
    acc.ckpt = st.stack_max;
    acc.arena = st.arena;
    return acc;
  }
  std::vector<char> is_cut(size_t(n), 0);
  for (int32_t c : p.cuts) {
    is_cut[size_t(c)] = 1;
    acc.ckpt += b[size_t(c) + 1];
  }
  auto segs = p.segments();
  int32_t fwd_hi = p.keep_last ? segs.back().first : n;
  if (fwd_hi > 0)
    acc.arena = sweep_need(b, a, 0, fwd_hi, [&](int32_t i) { return is_cut[size_t(i)] != 0; });
  for (auto &s : segs) {
    uint64_t t = 0;
    for (int32_t i = s.first; i < s.second; ++i) t += a[size_t(i)] + b[size_t(i) + 1];
    acc.arena = std::max(acc.arena, t);
  }
  return acc;
}

// ---------------------------------------------------- budget search --
// Appendix A: Alg. 3 with B = 0 gives x and y; B0 = floor(sqrt(x y)); the
// candidates are B0 and six evenly spaced budgets from floor(B0 / sqrt 2) to
// floor(sqrt(2) B0), all from exact integer square roots.
static uint64_t isqrt128(unsigned __int128 v) {
  uint64_t lo = 0, hi = ~uint64_t(0);
  while (lo < hi) {  // largest r with r*r <= v
    const uint64_t mid = lo + (hi - lo) / 2 + 1;
    if ((unsigned __int128)mid * mid <= v) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

std::vector<uint64_t> search_candidates(int32_t n, const uint64_t *lb, const uint64_t *cb) {
  const Plan z = make_plan(n, lb, cb, 0, CKPT_GREEDY, nullptr, 0, 0);
  const uint64_t b0 = isqrt128((unsigned __int128)z.x * z.y);
  const unsigned __int128 sq = (unsigned __int128)b0 * b0;
  const uint64_t lo = isqrt128(sq / 2), hi = isqrt128(sq * 2);
  std::vector<uint64_t> c{b0};
  for (uint64_t j = 0; j < 6; ++j) c.push_back(lo + uint64_t((unsigned __int128)(hi - lo) * j / 5));
  std::sort(c.begin(), c.end());
  c.erase(std::unique(c.begin(), c.end()), c.end());
  return c;
}

Plan search_plan(int32_t n, const uint64_t *lb, const uint64_t *cb, const std::vector<uint64_t> &b,
                 const std::vector<uint64_t> &a, const std::vector<uint64_t> &q, uint64_t slot,
                 uint64_t extra, int32_t flags, uint64_t *budget, uint64_t *peak) {
  bool have = false;
  Plan best;
  uint64_t best_b = 0, best_pk = 0;
  for (uint64_t B : search_candidates(n, lb, cb)) {
    Plan p = make_plan(n, lb, cb, B, CKPT_GREEDY, nullptr, 0, flags);
    const uint64_t pk = account(p, b, a, q, slot, extra).peak();
    if (!have || pk < best_pk) {  // candidates ascend: ties keep the smaller budget
      have = true;
      best = std::move(p);
      best_b = B;
      best_pk = pk;
    }
  }
  if (budget) *budget = best_b;
  if (peak) *peak = best_pk;
  return best;
}

}  // namespace ckpt

