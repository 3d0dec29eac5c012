/*
 * nightjar_planner.h -- the speculative-length planner of Nightjar (arXiv
 * 2512.22420, Sec. 5): a contextual bandit that picks, at every decoding step,
 * the speculative length gamma in {0..Gamma_max} for the current batch size B
 * (gamma = 0: plain decoding, Sec. 4).  Host code only (no device work); part
 * of libnightjar.so.
 *
 * Algorithm 1 (Sec. 5.2), per batch size B an independent timeline of blocks
 * j_B of length H_B = 2^(j_B - 1), each split into bins of up to sqrt(H_B)
 * rounds (decoding steps with that B):
 *   - at a bin start (tau_B = 1) the bin explores with probability 1/b_B (gamma
 *     uniform over the allowed arms) and otherwise exploits: gamma minimises
 *     Eq. (exploitation_min)
 *         l~_{B,gamma} + I(gamma_{t-1} = 0 and gamma > 0) * C_switch / gamma,
 *     l~ the empirical mean latency per committed token of arm gamma at B and
 *     C_switch the draft model's KV-reconstruction cost (Sec. 5.2, Table
 *     "ttft_diff"), looked up by the effective skip length delta_max and B;
 *   - the chosen gamma stays locked for the rest of the bin;
 *   - after the step, tau_B += 1; tau_B > sqrt(H_B) ends the bin (b_B += 1);
 *     b_B > sqrt(H_B) ends the block (j_B += 1, H_B = 2^(j_B - 1), b_B = 1).
 *
 * Readings where the paper leaves a choice open (chosen by the config):
 *   - gamma_{t-1}: the arm played at the previous decoding step of the whole
 *     system (the draft model's cache goes stale whenever any step ran with
 *     gamma = 0), or, with prev_per_batch = 1, the previous arm at the same B.
 *     Before the first step gamma_{t-1} counts as speculating (no penalty).
 *   - an arm never played at B has l~ = unplayed_latency (0: optimistic, so
 *     exploitation tries it; a large value: exploitation never does).
 *   - ties in the argmin go to the smallest gamma.
 *   - C_switch between profiled points: bilinear interpolation, linear in the
 *     skip length and in log2 of the batch size (the profile uses
 *     geometrically growing batch sizes), clamped to the profiled range.
 *   - latency per token: step latency / committed tokens of the step (the
 *     inverse of the step's goodput, Sec. 5.1).
 * Units: seconds for latencies and C_switch.
 *
 * Every function returns NJ_OK (0) or NJ_EINVAL (-1) with the message in
 * nightjar_last_error(); a planner is not thread-safe (one decision loop).
 */
#ifndef NIGHTJAR_PLANNER_H
#define NIGHTJAR_PLANNER_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct nj_planner nj_planner;

typedef struct nj_planner_config {
  int32_t max_batch;       /* B_max >= 1: batch sizes 1..B_max                         */
  int32_t max_gamma;       /* Gamma_max in [0, 15]: arms 0..Gamma_max                   */
  uint64_t seed;           /* the planner's own random stream (exploration draws)       */
  int32_t prev_per_batch;  /* 0: gamma_{t-1} of the whole system; 1: of the same B      */
  double unplayed_latency; /* l~ of an arm not yet played at B (seconds per token)      */
} nj_planner_config;

/* Per-batch-size state of Algorithm 1 (for inspection and tests). */
typedef struct nj_planner_bstate {
  int32_t block;         /* j_B                                   */
  int64_t block_len;     /* H_B = 2^(j_B - 1)                     */
  int64_t bin;           /* b_B                                   */
  int64_t round;         /* tau_B (1 = the next step starts a bin) */
  int32_t gamma;         /* the arm locked for the current bin    */
  int64_t steps;         /* steps played at B                     */
  int64_t bins;          /* bins started at B                     */
  int64_t explore_bins;  /* of which exploration bins             */
} nj_planner_bstate;

/* NULL on a bad config (message in nightjar_last_error()). */
nj_planner* nightjar_planner_create(const nj_planner_config* cfg);
void nightjar_planner_destroy(nj_planner* p);

/*
 * The C_switch table: seconds[i * n_batches + j] is the cost at skip length
 * lengths[i] and batch size batches[j] (both strictly increasing, batches >= 1).
 * Without a table C_switch is 0 (the original ADA-BINGREEDY loss).
 */
int nightjar_planner_set_switch_cost(nj_planner* p, const int32_t* lengths, int32_t n_lengths,
                                     const int32_t* batches, int32_t n_batches, const double* seconds);
/* C_switch(delta_max, B) from the table (interpolated), 0 without one; < 0 on bad arguments. */
double nightjar_planner_switch_cost(const nj_planner* p, int32_t delta_max, int32_t B);

/*
 * The arm for the next decoding step at batch size B (1..B_max).  delta_max:
 * the effective skip length (largest number of tokens a request's draft cache
 * is behind), used for C_switch; gamma_limit: the largest arm allowed now
 * (0 when the draft model is offloaded; arms above it are neither explored nor
 * exploited, and a locked arm above it plays as gamma_limit).  Counts the step
 * on B's timeline.
 */
int nightjar_planner_select(nj_planner* p, int32_t B, int32_t delta_max, int32_t gamma_limit, int32_t* gamma);

/*
 * Feedback of a step played with `gamma` at B: its latency and the tokens it
 * committed (accepted drafts plus one per sequence), giving latency per token
 * step_seconds / committed_tokens for l~_{B,gamma}.
 */
int nightjar_planner_observe(nj_planner* p, int32_t B, int32_t gamma, double step_seconds, int32_t committed_tokens);

int nightjar_planner_bstate(const nj_planner* p, int32_t B, nj_planner_bstate* out);
/* l~_{B,gamma} and its sample count (mean = unplayed_latency when count == 0). */
int nightjar_planner_arm(const nj_planner* p, int32_t B, int32_t gamma, double* mean, int64_t* count);

#ifdef __cplusplus
}
#endif

#endif /* NIGHTJAR_PLANNER_H */
