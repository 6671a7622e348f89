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

#ifdef __cplusplus
}
#endif
#endif /* PULSE_PLAN_H */
