/*
 * synerdiff_sched.h - the inter-concurrency scheduler's sequence planner
 * (Sec. III-D).  Host only; no GPU work.
 *
 * A workload of M UNet tasks, N VAE tasks and at most K Skip-CFG-eligible
 * UNet tasks (those past the quality threshold's minimum step) runs as a
 * sequence of concurrent stages (m_t, n_t, k_t).  The offline profiler's
 * lookup table (Sec. III-C) gives each stage configuration's concurrent round
 * latency tau(m, n, k) and VAE decoding latency delta(m, n, k).  Problem P
 * (Eq. (3a)-(3f)) minimises the VAE tasks' completion times
 *   sum_t n_t V(t),  V(t) = (sum of tau over the stages before t) + delta(stage t),
 * subject to completing every task, 0 <= n_t, k_t <= m_t, sum k_t <= K and a
 * total latency of at most T_lim (the throughput cap (1 + alpha) tau(M, N, K)).
 * Readings: a stage runs 1 <= m_t <= bmax UNet tasks; the U_i and A_i terms
 * of (3a) are constants of the placement and drop out.
 */
#ifndef SYNERDIFF_SCHED_H
#define SYNERDIFF_SCHED_H

#include "synerdiff.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Plan the stage sequence.
 *   tau, delta: lookup tables of (bmax + 1)^3 doubles, entry [m][n][k] at
 *     (m (bmax + 1) + n) (bmax + 1) + k, read for 1 <= m <= bmax, n, k <= m;
 *     finite, tau >= 0.
 *   mode 0: Alg. 1 as printed: one <cost, time> label per state (i, j, u),
 *     states in lexicographic order, actions (m, n, k) in lexicographic
 *     order, a label replaced only by a strictly smaller cost, transitions
 *     whose time exceeds T_lim dropped, the answer the first u with the
 *     smallest cost at (M, N, u).
 *   mode 1: every non-dominated <cost, time> label per state kept, which
 *     makes the result the optimum of Problem P (mode 0 keeps one label, so
 *     a cheaper label that arrives later can hide a cheaper completion).
 *   seq receives n_stages triples (m_t, n_t, k_t) (room for max_stages);
 *   cost = sum_t n_t V(t), time = total latency of the sequence.
 * Returns SD_ERR_UNSUPPORTED (n_stages = 0, cost = time = inf) when no
 * sequence meets T_lim, SD_ERR_CAPACITY when the sequence has more than
 * max_stages stages (n_stages is set), SD_ERR_INVALID_ARG on bad input.
 * M = 0 and N = 0 gives an empty sequence. */
sd_status synerdiff_plan_sequence(int32_t M, int32_t N, int32_t K, int32_t bmax, const double* tau,
                                  const double* delta, double T_lim, int32_t mode, int32_t max_stages, int32_t* seq,
                                  int32_t* n_stages, double* cost, double* time);

#ifdef __cplusplus
}
#endif
#endif /* SYNERDIFF_SCHED_H */
