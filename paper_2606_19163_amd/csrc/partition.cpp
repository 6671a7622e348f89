// Skip-aware balanced partitioning (host code): the bidirectional dynamic
// program of Sec. IV-B over (prefix end i, suffix start j), one collocated
// stage pair per level, outermost pair first.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <limits>
#include <vector>

#include "error.hpp"
#include "pulse_plan.h"

namespace {

constexpr double kInf = std::numeric_limits<double>::infinity();
constexpr int kMaxOps = 512;
constexpr int kMaxStages = 128;

pulse_status bad(const char* msg) { return pulse::set_last_error(PULSE_E_INVALID_ARG, msg); }

bool finite_nonneg(double v) { return std::isfinite(v) && v >= 0.0; }

pulse_status check_problem(const pulse_part_problem* pb, int32_t p) {
  if (!pb) return bad("problem is NULL");
  if (pb->n_ops < 1 || pb->n_ops > kMaxOps) return bad("n_ops must be in [1, 512]");
  if (!pb->t_f || !pb->m_a) return bad("t_f or m_a is NULL");
  if (pb->n_skips < 0 || (pb->n_skips > 0 && !pb->skips)) return bad("bad skip list");
  if (p < 2 || p % 2 != 0 || p > pb->n_ops || p > kMaxStages)
    return bad("p must be even, >= 2, <= n_ops and <= 128");
  for (int l = 0; l < pb->n_ops; ++l)
    if (!finite_nonneg(pb->t_f[l]) || !finite_nonneg(pb->m_a[l]))
      return bad("t_f and m_a must be finite and >= 0");
  for (int k = 0; k < 2 * pb->n_skips; ++k)
    if (pb->skips[k] < 0 || pb->skips[k] >= pb->n_ops) return bad("skip index out of range");
  if (!finite_nonneg(pb->lambda) || !finite_nonneg(pb->t_lat))
    return bad("lambda and t_lat must be finite and >= 0");
  if (!(std::isfinite(pb->b_inter) && pb->b_inter > 0.0)) return bad("b_inter must be > 0");
  return PULSE_OK;
}

// Skip pairs that constrain placement (ends more than one op apart), as
// c1 < c2, folded per start op: lo[c1] / hi[c1] = smallest / largest c2.
struct Skips {
  std::vector<int> lo, hi;
  std::vector<int> pre_lo;   // pre_lo[i] = min lo[c] over c <= i
  std::vector<int> suf_hi;   // suf_hi[i] = max hi[c] over c > i  (index i = -1 .. n-1)
};

Skips fold_skips(const pulse_part_problem* pb) {
  const int n = pb->n_ops;
  Skips s;
  s.lo.assign(n, n + 1);
  s.hi.assign(n, -1);
  for (int k = 0; k < pb->n_skips; ++k) {
    int a = pb->skips[2 * k], b = pb->skips[2 * k + 1];
    if (a > b) std::swap(a, b);
    if (b - a <= 1) continue;
    s.lo[a] = std::min(s.lo[a], b);
    s.hi[a] = std::max(s.hi[a], b);
  }
  s.pre_lo.assign(n, n + 1);
  for (int i = 0; i < n; ++i) s.pre_lo[i] = std::min(i ? s.pre_lo[i - 1] : n + 1, s.lo[i]);
  s.suf_hi.assign(n + 1, -1);  // suf_hi[i + 1] holds the value for i
  for (int i = n - 2; i >= -1; --i) s.suf_hi[i + 1] = std::max(s.suf_hi[i + 2], s.hi[i + 1]);
  return s;
}

struct Costs {
  int n;
  std::vector<double> pre;  // pre[l] = sum of t_f over ops < l
  std::vector<double> comm; // lambda * (t_lat + m_a[l] / b_inter)
  // left stage (i0, i]: ops i0+1 .. i, pays the output of op i
  double left(int i0, int i) const { return pre[i + 1] - pre[i0 + 1] + comm[i]; }
  // right stage [j, j1): ops j .. j1-1, pays the output of op j-1
  double right(int j, int j1) const { return pre[j1] - pre[j] + comm[j - 1]; }
};

Costs make_costs(const pulse_part_problem* pb) {
  Costs c;
  c.n = pb->n_ops;
  c.pre.assign(c.n + 1, 0.0);
  c.comm.assign(c.n, 0.0);
  for (int l = 0; l < c.n; ++l) {
    c.pre[l + 1] = c.pre[l] + pb->t_f[l];
    c.comm[l] = pb->lambda * (pb->t_lat + pb->m_a[l] / pb->b_inter);
  }
  return c;
}

}  // namespace

extern "C" {

pulse_status pulse_partition(const pulse_part_problem* pb, int32_t p, int32_t* cuts,
                             double* cost) {
  if (pulse_status st = check_problem(pb, p)) return st;
  if (!cuts || !cost) return bad("cuts or cost is NULL");
  const int n = pb->n_ops, H = p / 2;
  const Skips sk = fold_skips(pb);
  const Costs cs = make_costs(pb);
  // State (i, j), i < j: the pairs placed so far cover ops 0..i and j..n-1;
  // its value is their largest stage cost.  Level h adds stage h-1 (ops
  // i0+1..i) and stage p-h (ops j..j1-1) inside the state (i0, j1) of level
  // h-1.  A skip (c1, c2) is consistent with the new pair when
  //   (1) c1 <= i0       implies c2 >= j1,
  //   (2) i0 < c1 <= i   implies j <= c2 < j1,
  //   (3) c1 > i         implies c2 < j,
  // which is the penalty term of the recurrence.
  const int W = n + 1;
  auto at = [W](int i, int j) { return (size_t)i * W + j; };
  std::vector<double> prev((size_t)n * W, kInf), cur((size_t)n * W, kInf);
  std::vector<std::vector<int32_t>> from(H, std::vector<int32_t>((size_t)n * W, -1));
  for (int h = 1; h <= H; ++h) {
    std::fill(cur.begin(), cur.end(), kInf);
    std::vector<int32_t>& arg_h = from[h - 1];
    for (int i = h - 1; i < n; ++i) {
      for (int j = i + 1; j <= n - h; ++j) {
        if (sk.suf_hi[i + 1] >= j) continue;  // (3)
        if (h == 1) {
          // the outermost pair: stage 0 = ops 0..i, stage p-1 = ops j..n-1
          if (sk.pre_lo[i] < j) continue;     // (2)
          cur[at(i, j)] = std::max(cs.left(-1, i), cs.right(j, n));
          arg_h[at(i, j)] = n;                // (i0, j1) = (-1, n)
          continue;
        }
        double best = kInf;
        int32_t arg = -1;
        int lo_run = n + 1, hi_run = -1;      // skips starting in (i0, i]
        for (int i0 = i - 1; i0 >= h - 2; --i0) {
          lo_run = std::min(lo_run, sk.lo[i0 + 1]);
          hi_run = std::max(hi_run, sk.hi[i0 + 1]);
          if (lo_run < j) break;              // (2), and for every smaller i0
          const double L = cs.left(i0, i);
          if (L >= best) break;               // L grows as i0 falls
          const int j1_lo = std::max(j + 1, hi_run + 1);        // (2)
          const int j1_hi = std::min(n - h + 1, sk.pre_lo[i0]); // (1), room outside
          for (int j1 = j1_lo; j1 <= j1_hi; ++j1) {
            const double R = cs.right(j, j1);
            if (R >= best) break;             // R grows with j1
            const double outer = prev[at(i0, j1)];
            const double v = std::max(std::max(L, R), outer);
            if (v < best) {
              best = v;
              arg = (int32_t)(i0 + 1) * W + j1;
            }
          }
        }
        cur[at(i, j)] = best;
        arg_h[at(i, j)] = arg;
      }
    }
    prev.swap(cur);
  }
  // the halves meet: the innermost pair is stage H-1 = ..i and stage H = i+1..
  double best = kInf;
  int bi = -1;
  for (int i = H - 1; i + 1 <= n - H; ++i) {
    const double v = prev[at(i, i + 1)];
    if (v < best) {
      best = v;
      bi = i;
    }
  }
  *cost = best;
  for (int k = 0; k < p - 1; ++k) cuts[k] = -1;
  if (bi < 0) return PULSE_OK;
  // walk back outward: level h fixes the last op of stage h-1 (i) and of
  // stage p-h-1 (j-1, the op before stage p-h)
  int i = bi, j = bi + 1;
  for (int h = H; h >= 1; --h) {
    cuts[h - 1] = i;
    cuts[p - 1 - h] = j - 1;
    const int32_t a = from[h - 1][at(i, j)];
    i = a / W - 1;
    j = a % W;
  }
  return PULSE_OK;
}

pulse_status pulse_partition_cost(const pulse_part_problem* pb, int32_t p, const int32_t* cuts,
                                  double* cost, int32_t* valid, double* stage_costs) {
  if (pulse_status st = check_problem(pb, p)) return st;
  if (!cuts || !cost || !valid) return bad("cuts, cost or valid is NULL");
  const int n = pb->n_ops;
  for (int k = 0; k < p - 1; ++k)
    if (cuts[k] < 0 || cuts[k] >= n - 1 || (k && cuts[k] <= cuts[k - 1]))
      return bad("cuts must increase strictly and lie in [0, n_ops - 2]");
  std::vector<int> part(n);
  for (int q = 0, l = 0; q < p; ++q) {
    const int last = q < p - 1 ? cuts[q] : n - 1;
    for (; l <= last; ++l) part[l] = q;
  }
  bool ok = true;
  for (int k = 0; k < pb->n_skips; ++k) {
    int a = pb->skips[2 * k], b = pb->skips[2 * k + 1];
    if (a > b) std::swap(a, b);
    if (b - a > 1 && part[b] != p - 1 - part[a]) ok = false;
  }
  const Costs cs = make_costs(pb);
  double worst = 0.0;
  for (int q = 0; q < p; ++q) {
    const int first = q ? cuts[q - 1] + 1 : 0, last = q < p - 1 ? cuts[q] : n - 1;
    const double c = q < p / 2 ? cs.left(first - 1, last) : cs.right(first, last + 1);
    if (stage_costs) stage_costs[q] = c;
    worst = std::max(worst, c);
  }
  *valid = ok ? 1 : 0;
  *cost = ok ? worst : kInf;
  return PULSE_OK;
}

}  // extern "C"
