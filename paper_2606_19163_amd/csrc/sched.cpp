// Collocated pipeline schedule (host code): the wave order of a model cut
// into P = 2D partitions on D devices, where partition p and its skip partner
// P-1-p share a device (Sec. IV-B) and one device holds one skip-collocated
// stage (encoder stage q, decoder stage 2D-1-q, Sec. V-B); the constraints of
// the scheduling formulation (Sec. V-A) as a checker; and the executor that
// drives one device's stage through its share of the schedule.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <cstring>
#include <string>
#include <unordered_map>
#include <vector>

#include "error.hpp"
#include "pulse_stage.h"
#include "pulse_tstage.h"

namespace {

// Stage s of one microbatch's chain: the forward of partition s for s < P,
// then the backward of partition 2P-1-s.
int partition_of(int D, int s) {
  const int P = 2 * D;
  return s < P ? s : 2 * P - 1 - s;
}

// collocated pair (and, under the symmetric placement, device) of partition p
int pair_of(int D, int p) { return std::min(p, 2 * D - 1 - p); }

bool args_ok(int32_t D, int32_t M) { return D >= 1 && D <= 64 && M >= 1 && M <= 4096; }

pulse_status bad_arg(const char* msg) { return pulse::set_last_error(PULSE_E_INVALID_ARG, msg); }

constexpr const char* kDM = "D must be in [1, 64] and M in [1, 4096]";

// Exact minimum-makespan schedule under the symmetric placement, by
// breadth-first search over progress vectors k[s] (microbatches finished by
// stage s): with each stage taking microbatches in order, stage s can run
// microbatch k[s] when k[s-1] > k[s], and a step advances at most one
// runnable stage per device.  Returns false when the state space exceeds
// `max_states` (the caller then uses the list schedule).
bool exact_schedule(int D, int M, size_t max_states, std::vector<std::vector<int>>& rows) {
  const int S = 4 * D;
  std::vector<int> dev(S);
  for (int s = 0; s < S; ++s) dev[s] = pair_of(D, partition_of(D, s));
  using Key = std::string;
  struct Node {
    Key parent;
    uint64_t move;  // bit s: stage s advanced on the step into this state
  };
  std::unordered_map<Key, Node> seen;
  Key start(S, '\0'), goal(S, (char)M);
  seen.emplace(start, Node{Key(), 0});
  std::vector<Key> frontier{start}, next;
  bool found = start == goal;
  while (!found && !frontier.empty()) {
    next.clear();
    for (const Key& k : frontier) {
      // runnable stages per device, in stage order
      std::vector<std::vector<int>> run(D);
      for (int s = 0; s < S; ++s)
        if ((int)(unsigned char)k[s] < M &&
            (s == 0 || (unsigned char)k[s - 1] > (unsigned char)k[s]))
          run[dev[s]].push_back(s);
      // every combination of one runnable stage (or none) per device
      std::vector<int> pick(D, -1);
      for (;;) {
        uint64_t mv = 0;
        for (int d = 0; d < D; ++d)
          if (pick[d] >= 0) mv |= 1ull << run[d][pick[d]];
        if (mv) {
          Key nk = k;
          for (int s = 0; s < S; ++s)
            if (mv >> s & 1) nk[s] = (char)((unsigned char)nk[s] + 1);
          if (seen.find(nk) == seen.end()) {
            seen.emplace(nk, Node{k, mv});
            if (seen.size() > max_states) return false;
            if (nk == goal) found = true;
            next.push_back(nk);
          }
        }
        int d = 0;
        while (d < D && ++pick[d] >= (int)run[d].size()) pick[d++] = -1;
        if (d == D) break;
      }
      if (found) break;
    }
    frontier.swap(next);
  }
  if (!found) return false;
  // walk back from the goal: each step's move runs microbatch k_before[s]
  std::vector<std::pair<Key, uint64_t>> path;
  for (Key k = goal; k != start;) {
    const Node& n = seen.at(k);
    path.emplace_back(n.parent, n.move);
    k = n.parent;
  }
  std::reverse(path.begin(), path.end());
  const int T = (int)path.size();
  rows.assign(D, std::vector<int>(T, -1));
  for (int t = 0; t < T; ++t)
    for (int s = 0; s < S; ++s)
      if (path[t].second >> s & 1)
        rows[dev[s]][t] = s * M + (int)(unsigned char)path[t].first[s];
  return true;
}

// List schedules: at every step each device runs one of its runnable stages,
// the lowest microbatch of that stage first.  BWD_FIRST takes the stage with
// the largest s (backward before forward, deeper before shallower): it keeps
// at most 2D-1-d microbatches in flight on device d and reaches the
// minimum when D divides M.  FWD_FIRST takes forwards before backwards, each
// deepest first: every microbatch's forward finishes early, which reaches
// the minimum for every (D, M) tried, with all M microbatches in flight.
enum Rule { BWD_FIRST, FWD_FIRST };

void list_schedule(int D, int M, Rule rule, std::vector<std::vector<int>>& rows) {
  const int S = 4 * D, P = 2 * D;
  std::vector<int> dev(S), k(S, 0);
  for (int s = 0; s < S; ++s) dev[s] = pair_of(D, partition_of(D, s));
  std::vector<std::vector<int>> done_at(S, std::vector<int>(M, -1));
  rows.assign(D, {});
  auto rank = [&](int s) { return rule == FWD_FIRST && s < P ? s + S : s; };
  for (int t = 0;; ++t) {
    bool left = false;
    for (int s = 0; s < S; ++s) left |= k[s] < M;
    if (!left) break;
    std::vector<int> pick(D, -1);
    for (int s = 0; s < S; ++s) {
      if (k[s] >= M) continue;
      const int m = k[s];
      if (s > 0 && !(k[s - 1] > m && done_at[s - 1][m] <= t - 1)) continue;
      int& p = pick[dev[s]];
      if (p < 0 || rank(s) > rank(p)) p = s;
    }
    for (int d = 0; d < D; ++d) {
      const int s = pick[d];
      if (s >= 0) {
        rows[d].push_back(s * M + k[s]);
        done_at[s][k[s]] = t;
      } else {
        rows[d].push_back(-1);
      }
    }
    for (int d = 0; d < D; ++d)
      if (pick[d] >= 0) ++k[pick[d]];
  }
}

// Largest number of microbatches device d holds between its encoder forward
// (stage d) and its encoder backward (stage 4D-1-d), over a table[d * T + t].
int peak_inflight(int D, int M, const int32_t* table, int T, int d) {
  int cur = 0, peak = 0;
  for (int t = 0; t < T; ++t) {
    const int v = table[(long)d * T + t];
    if (v < 0) continue;
    const int s = v / M;
    if (s == d) peak = std::max(peak, ++cur);
    if (s == 4 * D - 1 - d) --cur;
  }
  return peak;
}

int max_inflight_of(int D, int M, const std::vector<std::vector<int>>& rows) {
  const int T = (int)rows[0].size();
  std::vector<int32_t> flat((size_t)D * T);
  for (int d = 0; d < D; ++d) std::copy(rows[d].begin(), rows[d].end(), flat.begin() + (long)d * T);
  int worst = 0;
  for (int d = 0; d < D; ++d) worst = std::max(worst, peak_inflight(D, M, flat.data(), T, d));
  return worst;
}

// The four stages a device runs: the forward and backward of its encoder
// partition d and of its decoder partition 2D - 1 - d.
enum Cell { F_ENC, F_DEC, B_DEC, B_ENC };

// Steps [t0, t1) of device d's row, each cell handed to call(cell, m) in
// step order; every cell of the range is checked first, so that nothing
// runs when one is not this device's.
template <class Call>
pulse_status run_row(int32_t D, int32_t d, int32_t M, const int32_t* table, int32_t T,
                     int32_t t0, int32_t t1, Call call) {
  if (!args_ok(D, M)) return bad_arg(kDM);
  if (!table) return bad_arg("table is NULL");
  if (d < 0 || d >= D) return bad_arg("device index out of range");
  if (t0 < 0 || t0 > t1 || t1 > T) return bad_arg("step range outside [0, T]");
  const int P = 2 * D;
  const int f_enc = d, f_dec = P - 1 - d;                          // forward stages
  const int b_dec = 2 * P - 1 - f_dec, b_enc = 2 * P - 1 - f_enc;  // their backwards
  for (int t = t0; t < t1; ++t) {
    const int v = table[(long)d * T + t];
    if (v < 0) continue;
    const int s = v / M;
    if (v >= 4 * D * M || (s != f_enc && s != f_dec && s != b_dec && s != b_enc))
      return bad_arg("a cell of the row is not one of this device's stages");
  }
  for (int t = t0; t < t1; ++t) {
    const int v = table[(long)d * T + t];
    if (v < 0) continue;
    const int s = v / M, m = v - s * M;
    const Cell c = s == f_enc ? F_ENC : s == f_dec ? F_DEC : s == b_dec ? B_DEC : B_ENC;
    const pulse_status ps = call(c, m);
    if (ps != PULSE_OK) return ps;
  }
  return PULSE_OK;
}

}  // namespace

extern "C" {

pulse_status pulse_sched_build(int32_t D, int32_t M, int32_t* table, int32_t cap, int32_t* T,
                               int32_t* exact) {
  if (!args_ok(D, M)) return bad_arg(kDM);
  if (!T) return bad_arg("T is NULL");
  // candidates: both list schedules, and the exact search when its state
  // space is small (the progress vectors are non-increasing sequences of
  // S = 4D values in [0, M]: C(M + S, S) of them).  The fewest steps win;
  // among equals, the fewest microbatches in flight on any device.
  std::vector<std::vector<int>> rows, cand;
  int best_t = 0, best_mem = 0;
  auto consider = [&](std::vector<std::vector<int>>& c) {
    const int t = (int)c[0].size(), mem = max_inflight_of(D, M, c);
    if (rows.empty() || t < best_t || (t == best_t && mem < best_mem)) {
      rows.swap(c);
      best_t = t;
      best_mem = mem;
    }
  };
  list_schedule(D, M, BWD_FIRST, cand);
  consider(cand);
  list_schedule(D, M, FWD_FIRST, cand);
  consider(cand);
  double states = 1.0;
  for (int i = 1; i <= 4 * D; ++i) states = states * (M + i) / i;
  bool ex = false;
  if (D <= 4 && M <= 200 && states <= 2e5 && exact_schedule(D, M, 200000, cand)) {
    ex = true;  // best_t can only tie or lose to the exact minimum
    consider(cand);
  }
  const int t = (int)rows[0].size();
  *T = t;
  if (exact) *exact = ex ? 1 : 0;
  if (!table) return PULSE_OK;  // size query
  if (cap < t) return pulse::set_last_error(PULSE_E_SHAPE, "cap is below the schedule length");
  for (int d = 0; d < D; ++d)
    for (int i = 0; i < t; ++i) table[(long)d * t + i] = rows[d][i];
  return PULSE_OK;
}

pulse_status pulse_sched_check(int32_t D, int32_t M, const int32_t* table, int32_t T,
                               int32_t* violated) {
  if (!args_ok(D, M)) return bad_arg(kDM);
  if (!table || !violated || T < 0) return bad_arg("table or violated is NULL, or T < 0");
  const int S = 4 * D;
  int32_t bad = 0;
  std::vector<int> dev_of(S, -1), time_of((size_t)S * M, -1);
  std::vector<int> count((size_t)S * M, 0);
  for (int d = 0; d < D; ++d)
    for (int t = 0; t < T; ++t) {
      const int v = table[(long)d * T + t];
      if (v < 0) continue;
      if (v >= S * M) {
        bad |= 1 << 1;
        continue;
      }
      const int s = v / M;
      ++count[v];
      time_of[v] = t;
      if (dev_of[s] < 0)
        dev_of[s] = d;
      else if (dev_of[s] != d)
        bad |= 1 << 3;  // (3) fixed device mapping
    }
  for (int v = 0; v < S * M; ++v)
    if (count[v] != 1) bad |= 1 << 1;  // (1) unique assignment
  // (2) one cell per (device, step): holds by the table's shape
  if (!(bad & (1 << 3))) {
    for (int s = 0; s < S; ++s)
      for (int s2 = 0; s2 < S; ++s2)
        if (dev_of[s] >= 0 && dev_of[s2] >= 0 &&
            pair_of(D, partition_of(D, s)) == pair_of(D, partition_of(D, s2)) &&
            dev_of[s] != dev_of[s2])
          bad |= 1 << 4;  // (4) collocation
    if (dev_of[0] > 0) bad |= 1;  // anchor: the first stage on device 0
  }
  for (int m = 0; m < M; ++m)
    for (int s = 0; s + 1 < S; ++s) {
      const int a = time_of[s * M + m], b = time_of[(s + 1) * M + m];
      if (a >= 0 && b >= 0 && b < a + 1) bad |= 1 << 5;  // (5) sequential execution
    }
  for (int s = 0; s < S; ++s)
    for (int m = 0; m + 1 < M; ++m) {
      const int a = time_of[s * M + m], b = time_of[s * M + m + 1];
      if (a >= 0 && b >= 0 && b < a) bad |= 1 << 6;  // (6) monotonic microbatch order
    }
  *violated = bad;
  return PULSE_OK;
}

pulse_status pulse_sched_inflight(int32_t D, int32_t M, const int32_t* table, int32_t T,
                                  int32_t* peak) {
  if (!args_ok(D, M)) return bad_arg(kDM);
  if (!table || !peak || T < 0) return bad_arg("table or peak is NULL, or T < 0");
  for (int d = 0; d < D; ++d) peak[d] = peak_inflight(D, M, table, T, d);
  return PULSE_OK;
}

pulse_status pulse_sched_run_device(pulse_stage* st, int32_t D, int32_t d, int32_t M,
                                    const int32_t* table, int32_t T, int32_t t0, int32_t t1,
                                    const pulse_mb_io* io, void* stream) {
  if (!st || !io) return bad_arg("stage or io is NULL");
  return run_row(D, d, M, table, T, t0, t1, [&](Cell c, int m) {
    const pulse_mb_io& b = io[m];
    switch (c) {
      case F_ENC: return pulse_stage_forward(st, PULSE_ENC, m, b.x, b.temb, b.y_enc, stream);
      case F_DEC: return pulse_stage_forward(st, PULSE_DEC, m, b.u, b.temb, b.y_dec, stream);
      case B_DEC: return pulse_stage_backward(st, PULSE_DEC, m, b.g_dec, b.du, b.dtemb, stream);
      default: return pulse_stage_backward(st, PULSE_ENC, m, b.g_enc, b.dx, b.dtemb, stream);
    }
  });
}

pulse_status pulse_tsched_run_device(pulse_tstage* st, int32_t D, int32_t d, int32_t M,
                                     const int32_t* table, int32_t T, int32_t t0, int32_t t1,
                                     const pulse_mb_io* io, void* stream) {
  if (!st || !io) return bad_arg("stage or io is NULL");
  return run_row(D, d, M, table, T, t0, t1, [&](Cell c, int m) {
    const pulse_mb_io& b = io[m];
    switch (c) {
      case F_ENC: return pulse_tstage_forward(st, PULSE_ENC, m, b.x, b.y_enc, stream);
      case F_DEC: return pulse_tstage_forward(st, PULSE_DEC, m, b.u, b.y_dec, stream);
      case B_DEC: return pulse_tstage_backward(st, PULSE_DEC, m, b.g_dec, b.du, stream);
      default: return pulse_tstage_backward(st, PULSE_ENC, m, b.g_enc, b.dx, stream);
    }
  });
}

}  // extern "C"
