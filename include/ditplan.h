/* Exploration planner and seed bank: host-side C ABI of libditstep.so.
 *
 * The planner picks, once per training iteration, the exploration configuration
 * a = (d, s) that runs on the spare GPUs while the model trains (the bandit-based
 * hyper-parameter adaptation of section 4.3):
 *   * action space: d sequences per prompt x s effective denoising steps, from the
 *     caller's lists of values (section 4.3.1);
 *   * eligibility: T_plan(a) = d * C * s * t_step <= W = T_train * N_spot for C prompts
 *     (section 4.3.1);
 *   * feedback after an iteration: r = sigma_all / sigma_unc, the mean per-group reward
 *     std over all prompt groups divided by the mean over the unexplored groups
 *     (section 4.3.2); sigma_g is the std that group_reward_stats returns;
 *   * selection: UCB(a_i) = mu_i + beta sqrt(ln(N + 1) / n_i), mu_i the mean of the
 *     window_b most recent feedbacks of a_i, n_i = min(N_i, window_b), N = sum N_i;
 *     UCB = +inf while n_i = 0; the argmax over the eligible set, ties to lower planned
 *     cost, then fewer steps s, then fewer sequences d (section 4.3.3).
 *   When no action fits the window, the planner returns the cheapest action overall
 *   (same tie order) with *fits = 0: the exploration that overflows the window then
 *   continues after the model update (section 4.3.4).
 * The seed bank keeps, per prompt, the top ceil(k/2) and bottom floor(k/2) seeds by
 * exploration reward (descending reward, ties by ascending position), the seeds the
 * next iteration's rollout uses (section 5, dynamic exploration).
 *
 * All pointers are host pointers owned by the caller. Handles are not thread-safe:
 * one thread (or a caller-held lock) per handle. Errors return a dit_status with the
 * detail in dit_last_error_message() (declared in ditstep.h). */
#ifndef DITPLAN_H
#define DITPLAN_H

#include <stdint.h>

#include "ditstep.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct dit_planner dit_planner;
typedef struct dit_seed_bank dit_seed_bank;

/* Action grid d_values[n_d] x s_values[n_s] (positive, distinct within each list); action
 * index = i_d * n_s + i_s. beta >= 0 (the paper uses 0.5), window >= 1, prompts = C >= 1.
 * *out receives a new handle (free with dit_planner_destroy). DIT_ERR_INVALID_ARG on bad
 * parameters; *out is then NULL. */
dit_status dit_planner_create(const int32_t* d_values, int32_t n_d, const int32_t* s_values,
                              int32_t n_s, double beta, int32_t window, int32_t prompts,
                              dit_planner** out);
void dit_planner_destroy(dit_planner* p);
int32_t dit_planner_num_actions(const dit_planner* p);
/* d and s of action `index`. */
dit_status dit_planner_action(const dit_planner* p, int32_t index, int32_t* d, int32_t* s);

/* eligible[num_actions] = 1 if T_plan <= T_train * N_spot, else 0; *count = number of 1s.
 * t_train >= 0, n_spot >= 0, t_step > 0 (else DIT_ERR_DOMAIN). */
dit_status dit_planner_eligible(const dit_planner* p, double t_train, int32_t n_spot, double t_step,
                                int32_t* eligible, int32_t* count);

/* The next action (see above); *fits = 1 if it is eligible. ucb may be NULL, else it
 * receives the chosen action's UCB (+inf for an unobserved action). */
dit_status dit_planner_select(const dit_planner* p, double t_train, int32_t n_spot, double t_step,
                              int32_t* index, int32_t* fits, double* ucb);

/* Record the feedback r (finite) of one iteration that ran action `index`. */
dit_status dit_planner_update(dit_planner* p, int32_t index, double r);

/* Current state of action `index`: N_i, n_i, window mean (0 when n_i = 0) and UCB. */
dit_status dit_planner_stats(const dit_planner* p, int32_t index, int32_t* total, int32_t* in_window,
                             double* mean, double* ucb);

/* r = mean(sigma[g] over all g) / mean(sigma[g] over g with explored[g] == 0), sigma [groups]
 * fp32 per-group reward std, explored [groups] 0/1. DIT_ERR_DOMAIN without an unexplored
 * group or when their mean std is 0; DIT_ERR_NAN for a non-finite sigma. */
dit_status dit_planner_feedback(const float* sigma, const int32_t* explored, int32_t groups, double* r);

/* Seed bank keeping k seeds per prompt (k >= 0). */
dit_status dit_seed_bank_create(int32_t k, dit_seed_bank** out);
void dit_seed_bank_destroy(dit_seed_bank* b);
/* Stores, for prompt_id, the kept seeds of seeds[d] given their exploration rewards[d]
 * (min(k, d) seeds: top ceil/bottom floor halves as above); replaces an earlier entry.
 * DIT_ERR_NAN for a non-finite reward. */
dit_status dit_seed_bank_put(dit_seed_bank* b, int64_t prompt_id, const int64_t* seeds,
                             const float* rewards, int32_t d);
/* Same from group_reward_stats' `selected` output copied to the host: for each of `groups`
 * prompts, seeds[g][d] and selected[g][k] (positions into that prompt's seeds). */
dit_status dit_seed_bank_put_selected(dit_seed_bank* b, const int64_t* prompt_ids, int32_t groups,
                                      const int64_t* seeds, int32_t d, const int32_t* selected,
                                      int32_t k);
/* Copies the kept seeds of prompt_id (at most `capacity`) into out; *count = how many are
 * stored (0 if the prompt has no entry: the caller then draws fresh seeds). */
dit_status dit_seed_bank_get(const dit_seed_bank* b, int64_t prompt_id, int64_t* out, int32_t capacity,
                             int32_t* count);
/* Number of prompts with an entry. */
int32_t dit_seed_bank_size(const dit_seed_bank* b);

#ifdef __cplusplus
}
#endif

#endif /* DITPLAN_H */
