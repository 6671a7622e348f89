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

// The dynamic program; arguments already checked.
void partition_dp(const pulse_part_problem* pb, int32_t p, int32_t* cuts, double* cost) {
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
  if (bi < 0) return;
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
}

}  // namespace

extern "C" {

pulse_status pulse_partition(const pulse_part_problem* pb, int32_t p, int32_t* cuts,
                             double* cost) {
  if (pulse_status st = check_problem(pb, p)) return st;
  if (!cuts || !cost) return bad("cuts or cost is NULL");
  partition_dp(pb, p, cuts, cost);
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

pulse_status pulse_comm_volume(const pulse_part_problem* pb, int32_t n_stages,
                               const int32_t* cuts, int32_t collocated, double* bytes) {
  if (pulse_status st = check_problem(pb, 2)) return st;
  if (!cuts || !bytes) return bad("cuts or bytes is NULL");
  const int n = pb->n_ops;
  if (n_stages < 1 || n_stages > n || (collocated && n_stages % 2))
    return bad("n_stages must be in [1, n_ops], and even when collocated");
  for (int k = 0; k < n_stages - 1; ++k)
    if (cuts[k] < 0 || cuts[k] >= n - 1 || (k && cuts[k] <= cuts[k - 1]))
      return bad("cuts must increase strictly and lie in [0, n_ops - 2]");
  std::vector<int> dev(n);
  auto dev_of_stage = [&](int st) {
    return collocated ? std::min(st, n_stages - 1 - st) : st;
  };
  for (int st = 0, l = 0; st < n_stages; ++st) {
    const int last = st < n_stages - 1 ? cuts[st] : n - 1;
    for (; l <= last; ++l) dev[l] = dev_of_stage(st);
  }
  double v = 0.0;
  for (int st = 0; st + 1 < n_stages; ++st)
    if (dev_of_stage(st) != dev_of_stage(st + 1)) v += pb->m_a[cuts[st]];
  for (int k = 0; k < pb->n_skips; ++k) {
    int a = pb->skips[2 * k], b = pb->skips[2 * k + 1];
    if (a > b) std::swap(a, b);
    if (dev[a] == dev[b]) continue;
    if (collocated && b - a > 1)
      return bad("a skip crosses devices: the cuts violate the collocation rule");
    v += pb->m_a[a] * std::abs(dev[b] - dev[a]);
  }
  *bytes = v;
  return PULSE_OK;
}

}  // extern "C"

// ---- hybrid data/pipeline parallelism (Sec. VI) ---------------------------

namespace {

pulse_status check_tune(const pulse_tune_problem* tp) {
  if (!tp) return bad("problem is NULL");
  if (tp->n_ops < 2 || tp->n_ops > kMaxOps) return bad("n_ops must be in [2, 512]");
  if (tp->n_b < 1 || tp->n_b > 32 || !tp->b) return bad("n_b must be in [1, 32] and b set");
  for (int k = 0; k < tp->n_b; ++k)
    if (tp->b[k] < 1 || (k && tp->b[k] <= tp->b[k - 1]))
      return bad("b must be strictly increasing and >= 1");
  if (!tp->t_f || !tp->m_theta || !tp->m_a || !tp->m_o) return bad("a per-op array is NULL");
  for (long k = 0; k < (long)tp->n_b * tp->n_ops; ++k)
    if (!finite_nonneg(tp->t_f[k])) return bad("t_f must be finite and >= 0");
  for (int l = 0; l < tp->n_ops; ++l)
    if (!finite_nonneg(tp->m_theta[l]) || !finite_nonneg(tp->m_a[l]) ||
        !finite_nonneg(tp->m_o[l]))
      return bad("memory sizes must be finite and >= 0");
  if (!(std::isfinite(tp->b_intra) && tp->b_intra > 0.0)) return bad("b_intra must be > 0");
  if (!(tp->m_limit > 0.0)) return bad("m_limit must be > 0");
  return PULSE_OK;
}

// The partition problem of candidate k: op times at b[k], boundary bytes
// b[k] * m_o.
struct PartAtB {
  std::vector<double> ma;
  pulse_part_problem pp;
};

PartAtB part_at_b(const pulse_tune_problem* tp, int k) {
  PartAtB r;
  r.ma.resize(tp->n_ops);
  for (int l = 0; l < tp->n_ops; ++l) r.ma[l] = tp->b[k] * tp->m_o[l];
  r.pp.n_ops = tp->n_ops;
  r.pp.t_f = tp->t_f + (long)k * tp->n_ops;
  r.pp.m_a = r.ma.data();
  r.pp.n_skips = tp->n_skips;
  r.pp.skips = tp->skips;
  r.pp.lambda = tp->lambda;
  r.pp.t_lat = tp->t_lat;
  r.pp.b_inter = tp->b_inter;
  return r;
}

// The models of Sec. VI for one configuration (stages from `cuts`).
pulse_tune_row eval_config(const pulse_tune_problem* tp, int P, int G, int k,
                           const int32_t* cuts) {
  const int n = tp->n_ops, S = 2 * P;
  const double* tf = tp->t_f + (long)k * n;
  const double b = tp->b[k];
  std::vector<double> Tf(S, 0.0), Mth(S, 0.0), Ma(S, 0.0), Mo(S, 0.0);
  for (int s = 0, l = 0; s < S; ++s) {
    const int last = s < S - 1 ? cuts[s] : n - 1;
    for (; l <= last; ++l) {
      Tf[s] += tf[l];
      Mth[s] += tp->m_theta[l];
      Ma[s] += tp->m_a[l];
    }
    Mo[s] = tp->m_o[last];
  }
  // stage s of the formulas (1-based) is index s-1
  double m_peak = 7.0 * (Mth[P - 1] + Mth[P]) + P * (Ma[P - 1] + Ma[P]) * b;
  if (P >= 2) m_peak += P * Mo[P - 2];
  const double mth_max = *std::max_element(Mth.begin(), Mth.end());
  const double t_ar = tp->t_lat + 2.0 * (G - 1) * mth_max / (G * tp->b_intra);
  const double tf_max = *std::max_element(Tf.begin(), Tf.end());
  const double mo_max = *std::max_element(Mo.begin(), Mo.end());
  const double steps = std::max(0, 10 * P - 12);
  const double t_sched = (10.0 * P - 4.0) * tf_max +
                         steps * (tp->t_lat + b * mo_max / tp->b_inter) + t_ar;
  pulse_tune_row r;
  r.P = P;
  r.G = G;
  r.b = tp->b[k];
  r.feasible = m_peak < tp->m_limit ? 1 : 0;
  r.t_sample = t_sched / (b * P * G);
  r.t_sched = t_sched;
  r.m_peak = m_peak;
  r.t_ar = t_ar;
  return r;
}

}  // namespace

extern "C" {

pulse_status pulse_tune(const pulse_tune_problem* tp, int32_t n_devices, pulse_tune_row* best,
                        int32_t* found, pulse_tune_row* rows, int32_t cap, int32_t* n_rows) {
  if (pulse_status st = check_tune(tp)) return st;
  if (n_devices < 1 || n_devices > 1 << 20) return bad("n_devices must be in [1, 2^20]");
  if (!best || !found || !n_rows || (cap > 0 && !rows) || cap < 0)
    return bad("best, found or n_rows is NULL, or rows missing for cap > 0");
  {
    // the problem's partition fields must hold for every candidate b
    PartAtB pa = part_at_b(tp, 0);
    if (pulse_status st = check_problem(&pa.pp, 2)) return st;
  }
  *found = 0;
  int count = 0;
  for (int P = 1; P <= n_devices && 2 * P <= tp->n_ops; ++P) {
    if (n_devices % P) continue;
    if (2 * P > kMaxStages) break;
    const int G = n_devices / P;
    pulse_tune_row chosen{};
    bool have = false;
    std::vector<int32_t> cuts(2 * P - 1);
    for (int k = 0; k < tp->n_b; ++k) {
      PartAtB pa = part_at_b(tp, k);
      double cost;
      partition_dp(&pa.pp, 2 * P, cuts.data(), &cost);
      if (!std::isfinite(cost)) continue;
      const pulse_tune_row r = eval_config(tp, P, G, k, cuts.data());
      if (count < cap) rows[count] = r;
      ++count;
      if (r.feasible) {
        chosen = r;  // candidates ascend: the last feasible one has the largest b
        have = true;
      }
    }
    if (have && (!*found || chosen.t_sample < best->t_sample)) {
      *best = chosen;
      *found = 1;
    }
  }
  *n_rows = count;
  return PULSE_OK;
}

pulse_status pulse_tune_eval(const pulse_tune_problem* tp, int32_t P, int32_t G, int32_t b_index,
                             const int32_t* cuts, pulse_tune_row* row) {
  if (pulse_status st = check_tune(tp)) return st;
  if (!cuts || !row) return bad("cuts or row is NULL");
  if (P < 1 || 2 * P > tp->n_ops || G < 1) return bad("P or G out of range");
  if (b_index < 0 || b_index >= tp->n_b) return bad("b_index out of range");
  for (int s = 0; s < 2 * P - 1; ++s)
    if (cuts[s] < 0 || cuts[s] >= tp->n_ops - 1 || (s && cuts[s] <= cuts[s - 1]))
      return bad("cuts must increase strictly and lie in [0, n_ops - 2]");
  *row = eval_config(tp, P, G, b_index, cuts);
  return PULSE_OK;
}

}  // extern "C"
