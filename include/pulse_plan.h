/*
 * pulse_plan.h -- host-side planning of a skip-collocated pipeline (part of
 * the same library as pulse_stage.h; plain C ABI, host memory only, no GPU
 * work).
 *
 * Skip-aware balanced partitioning (Sec. IV-B).  A model is an ordered
 * sequence of n operations (op 0 .. n-1) with forward times t_f[l] and
 * output activation sizes m_a[l] (bytes of the tensor op l passes to op
 * l+1), and skip connections (c1, c2) between operation indices.  A
 * partition cuts the sequence into p contiguous, non-empty stages (p even);
 * stage q (0-based) is collocated with stage p-1-q.  It is valid when every
 * skip pair more than one op apart has its two ends in collocated stages
 * (the symmetric placement rule of Sec. IV-B).  Stage cost:
 *
 *   sum of t_f over the stage + lambda * (t_lat + a / b_inter)
 *
 * where a is the boundary tensor the stage pays for: the output of its last
 * op for stages 0 .. p/2-1, the output of the op before its first op for
 * stages p/2 .. p-1 (the L and R terms of the recurrence of Sec. IV-B).
 * The partition sought minimises the largest stage cost.
 *
 * Conventions: every pointer is caller-owned host memory; calls validate
 * before they compute and report errors through the status and
 * pulse_last_error(); they are thread-safe (no shared state).
 */
#ifndef PULSE_PLAN_H
#define PULSE_PLAN_H

#include <stdint.h>

#include "pulse_stage.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
  int32_t n_ops;          /* 1 .. 512 */
  const double* t_f;      /* [n_ops] forward time of each op (>= 0, any unit) */
  const double* m_a;      /* [n_ops] bytes of each op's output (>= 0) */
  int32_t n_skips;        /* >= 0 */
  const int32_t* skips;   /* [n_skips][2] op indices of each skip pair, any order */
  double lambda;          /* weight of the communication term (>= 0) */
  double t_lat;           /* static latency of a transfer, in t_f's unit (>= 0) */
  double b_inter;         /* bytes per t_f unit of the inter-device link (> 0) */
} pulse_part_problem;

/* Skip-aware balanced partition into p stages (p even, 2 <= p <= n_ops, and
 * p <= 128) by the bidirectional dynamic program of Sec. IV-B: dp over
 * (prefix end, suffix start) grows one collocated stage pair per level,
 * from the outermost pair inward, and the two halves meet in the middle.
 * cuts (p - 1 entries, caller-owned) receives the last op of stages
 * 0 .. p-2; *cost the largest stage cost.  When no partition is valid the
 * call succeeds with *cost = +infinity and every cut = -1.
 * PULSE_E_INVALID_ARG for a NULL pointer, a bad p, an op index out of range,
 * or a negative or non-finite time, size or weight. */
pulse_status pulse_partition(const pulse_part_problem* pb, int32_t p, int32_t* cuts,
                             double* cost);

/* Cost of a given partition (cuts: p - 1 strictly increasing last-op
 * indices, each below n_ops - 1): *valid = 1 and *cost = its largest stage
 * cost when it satisfies the skip constraints, else *valid = 0 and
 * *cost = +infinity.  stage_costs (p entries, may be NULL) receives every
 * stage's cost. */
pulse_status pulse_partition_cost(const pulse_part_problem* pb, int32_t p, const int32_t* cuts,
                                  double* cost, int32_t* valid, double* stage_costs);

/* Forward point-to-point bytes of one sample through a cut model
 * (Sec. II-C, Sec. V-B).  Stage s of n_stages holds ops cuts[s-1]+1 ..
 * cuts[s].  With collocated = 0 stage s runs on device s, as a sequential
 * pipeline places it: every stage boundary is one transfer of the boundary
 * op's output, and a skip (c1, c2) crossing devices is passed on from
 * stage to stage, one transfer of c1's output per device it crosses.  With
 * collocated = 1, n_stages is even and stage s runs on device
 * min(s, n_stages-1-s): boundaries between stages on different devices
 * are transferred once, and skips between non-adjacent ops, which a valid
 * partition keeps on one device, cost nothing (PULSE_E_INVALID_ARG if one
 * would cross).  A skip between adjacent ops is charged like any other
 * when it crosses devices (the traffic model of Sec. II-C counts it apart
 * from the boundary).  Backward passes send the same volume of gradients
 * again. */
pulse_status pulse_comm_volume(const pulse_part_problem* pb, int32_t n_stages,
                               const int32_t* cuts, int32_t collocated, double* bytes);

/* Hybrid data/pipeline parallelism (Sec. VI).  N devices run G replicas of
 * a P-device pipeline (N = P G) of 2P collocated stages, on microbatches of
 * b samples.  Per stage s (1-based), summed over the ops the skip-aware
 * partition puts in it: T_f^s(b) forward time at b, M_theta^s parameter
 * bytes, M_a^s activation bytes kept per sample; M_o^s the output bytes per
 * sample of its last op.  The models of Sec. VI:
 *
 *   M_peak  = 7 (M_theta^P + M_theta^(P+1)) + P (M_a^P + M_a^(P+1)) b
 *             + P M_o^(P-1)                       (no last term for P = 1)
 *   T_sched = (10P - 4) max_s T_f^s(b)
 *             + max(0, 10P - 12) (t_lat + b max_s M_o^s / b_inter) + T_AR
 *   T_AR    = t_lat + 2 (G - 1) max_s M_theta^s / (G b_intra)
 *   T_sample = T_sched / (b P G)
 *
 * The partition for (P, b) is pulse_partition of the op forward times at b
 * into 2P stages, with boundary bytes b * m_o and the problem's lambda,
 * t_lat and b_inter. */
typedef struct {
  int32_t n_ops;          /* 2 .. 512 */
  int32_t n_b;            /* 1 .. 32 candidate microbatch sizes */
  const int32_t* b;       /* [n_b] strictly increasing, >= 1 */
  const double* t_f;      /* [n_b][n_ops] forward time of each op at each b (seconds) */
  const double* m_theta;  /* [n_ops] parameter bytes */
  const double* m_a;      /* [n_ops] activation bytes kept per sample */
  const double* m_o;      /* [n_ops] output bytes per sample */
  int32_t n_skips;
  const int32_t* skips;   /* [n_skips][2] op index pairs */
  double lambda;          /* partition communication weight (>= 0) */
  double t_lat;           /* seconds per transfer (>= 0) */
  double b_inter;         /* bytes/s of the pipeline link (> 0) */
  double b_intra;         /* bytes/s of the all-reduce (> 0) */
  double m_limit;         /* bytes of memory per device (> 0, may be +infinity) */
} pulse_tune_problem;

typedef struct {
  int32_t P, G, b;
  int32_t feasible;       /* M_peak < m_limit */
  double t_sample, t_sched, m_peak, t_ar;
} pulse_tune_row;

/* Enumerate every factorisation N = P G with 2P <= n_ops; for each, keep
 * the largest candidate b whose partition exists and fits in memory, and
 * return the configuration with the smallest T_sample in *best (*found = 0
 * when nothing fits; ties go to the smaller P).  rows (cap entries, may be
 * NULL) receives one row per (P, b) evaluated, P ascending then b
 * ascending; *n_rows their count (all of them, even beyond cap).
 * PULSE_E_INVALID_ARG for a NULL pointer, N < 1 or a bad problem. */
pulse_status pulse_tune(const pulse_tune_problem* pb, int32_t n_devices, pulse_tune_row* best,
                        int32_t* found, pulse_tune_row* rows, int32_t cap, int32_t* n_rows);

/* The models above for one configuration whose 2P stages are given by cuts
 * (2P - 1 entries, as pulse_partition returns them), at candidate b_index. */
pulse_status pulse_tune_eval(const pulse_tune_problem* pb, int32_t P, int32_t G, int32_t b_index,
                             const int32_t* cuts, pulse_tune_row* row);

#ifdef __cplusplus
}
#endif
#endif /* PULSE_PLAN_H */
