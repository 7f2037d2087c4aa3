// Exploration planner (bandit over (sequences, effective steps), section 4.3) and seed bank
// (top / bottom seeds per prompt, section 5): host code behind include/ditplan.h.
#include <cmath>
#include <cstdint>
#include <deque>
#include <limits>
#include <new>
#include <unordered_map>
#include <vector>

#include "../../include/ditplan.h"
#include "status.h"

using dit::set_error;

struct dit_planner {
  struct Action {
    int32_t d, s;
    int64_t total = 0;          // N_i
    std::deque<double> recent;  // the last `window` feedbacks, oldest first
  };
  std::vector<Action> actions;
  double beta;
  int32_t window, prompts;
  int64_t updates = 0;          // N

  double planned_time(const Action& a, double t_step) const {
    return (double)((int64_t)a.d * prompts * a.s) * t_step;
  }
  double ucb(const Action& a) const {
    const size_t n = a.recent.size();
    if (n == 0) return std::numeric_limits<double>::infinity();
    double sum = 0.0;
    for (double r : a.recent) sum += r;
    return sum / (double)n + beta * std::sqrt(std::log((double)(updates + 1)) / (double)n);
  }
  // planned cost is proportional to d * s; ties go to fewer steps, then fewer sequences
  bool cheaper(const Action& a, const Action& b) const {
    const int64_t ca = (int64_t)a.d * a.s, cb = (int64_t)b.d * b.s;
    if (ca != cb) return ca < cb;
    if (a.s != b.s) return a.s < b.s;
    return a.d < b.d;
  }
};

struct dit_seed_bank {
  int32_t k;
  std::unordered_map<int64_t, std::vector<int64_t>> kept;
};

namespace {

dit_status check_budget(double t_train, int32_t n_spot, double t_step) {
  if (!(t_train >= 0.0) || !std::isfinite(t_train) || n_spot < 0 || !(t_step > 0.0) || !std::isfinite(t_step))
    return set_error(DIT_ERR_DOMAIN, "need t_train >= 0, n_spot >= 0, t_step > 0 (got %g, %d, %g)", t_train, n_spot,
                     t_step);
  return DIT_OK;
}

// positions 0..d-1 ranked by descending reward, ties by ascending position; keeps the first
// ceil(k/2) and the last floor(k/2)
std::vector<int32_t> keep_positions(const float* rewards, int32_t d, int32_t k) {
  std::vector<int32_t> order(d);
  for (int32_t j = 0; j < d; j++) order[j] = j;
  // insertion sort: stable, and d is a seed count (tens)
  for (int32_t i = 1; i < d; i++) {
    const int32_t cur = order[i];
    int32_t j = i - 1;
    while (j >= 0 && rewards[order[j]] < rewards[cur]) {
      order[j + 1] = order[j];
      j--;
    }
    order[j + 1] = cur;
  }
  std::vector<int32_t> keep;
  const int32_t top = (k + 1) / 2, bottom = k / 2;
  for (int32_t j = 0; j < top; j++) keep.push_back(order[j]);
  for (int32_t j = d - bottom; j < d; j++) keep.push_back(order[j]);
  return keep;
}

}  // namespace

extern "C" {

dit_status dit_planner_create(const int32_t* d_values, int32_t n_d, const int32_t* s_values, int32_t n_s,
                              double beta, int32_t window, int32_t prompts, dit_planner** out) {
  if (!out) return set_error(DIT_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  if (!d_values || !s_values || n_d < 1 || n_s < 1) return set_error(DIT_ERR_INVALID_ARG, "empty action grid");
  if (!(beta >= 0.0) || !std::isfinite(beta)) return set_error(DIT_ERR_INVALID_ARG, "beta %g must be >= 0", beta);
  if (window < 1 || prompts < 1) return set_error(DIT_ERR_INVALID_ARG, "window %d / prompts %d must be >= 1", window, prompts);
  for (int32_t i = 0; i < n_d; i++) {
    if (d_values[i] < 1) return set_error(DIT_ERR_INVALID_ARG, "d_values[%d] = %d < 1", i, d_values[i]);
    for (int32_t j = 0; j < i; j++)
      if (d_values[j] == d_values[i]) return set_error(DIT_ERR_INVALID_ARG, "d value %d repeated", d_values[i]);
  }
  for (int32_t i = 0; i < n_s; i++) {
    if (s_values[i] < 1) return set_error(DIT_ERR_INVALID_ARG, "s_values[%d] = %d < 1", i, s_values[i]);
    for (int32_t j = 0; j < i; j++)
      if (s_values[j] == s_values[i]) return set_error(DIT_ERR_INVALID_ARG, "s value %d repeated", s_values[i]);
  }
  dit_planner* p = new (std::nothrow) dit_planner();
  if (!p) return set_error(DIT_ERR_INVALID_ARG, "out of host memory");
  for (int32_t i = 0; i < n_d; i++)
    for (int32_t j = 0; j < n_s; j++) {
      dit_planner::Action a;
      a.d = d_values[i];
      a.s = s_values[j];
      p->actions.push_back(a);
    }
  p->beta = beta;
  p->window = window;
  p->prompts = prompts;
  *out = p;
  return DIT_OK;
}

void dit_planner_destroy(dit_planner* p) { delete p; }

int32_t dit_planner_num_actions(const dit_planner* p) { return p ? (int32_t)p->actions.size() : 0; }

dit_status dit_planner_action(const dit_planner* p, int32_t index, int32_t* d, int32_t* s) {
  if (!p) return set_error(DIT_ERR_INVALID_ARG, "planner is NULL");
  if (index < 0 || index >= (int32_t)p->actions.size()) return set_error(DIT_ERR_INVALID_ARG, "action %d out of range", index);
  if (d) *d = p->actions[index].d;
  if (s) *s = p->actions[index].s;
  return DIT_OK;
}

dit_status dit_planner_eligible(const dit_planner* p, double t_train, int32_t n_spot, double t_step, int32_t* eligible,
                                int32_t* count) {
  if (!p) return set_error(DIT_ERR_INVALID_ARG, "planner is NULL");
  if (dit_status st = check_budget(t_train, n_spot, t_step)) return st;
  const double w = t_train * (double)n_spot;
  int32_t c = 0;
  for (size_t i = 0; i < p->actions.size(); i++) {
    const int32_t e = p->planned_time(p->actions[i], t_step) <= w;
    if (eligible) eligible[i] = e;
    c += e;
  }
  if (count) *count = c;
  return DIT_OK;
}

dit_status dit_planner_select(const dit_planner* p, double t_train, int32_t n_spot, double t_step, int32_t* index,
                              int32_t* fits, double* ucb) {
  if (!p || !index) return set_error(DIT_ERR_INVALID_ARG, "planner / index is NULL");
  if (dit_status st = check_budget(t_train, n_spot, t_step)) return st;
  const double w = t_train * (double)n_spot;
  int32_t best = -1;
  double best_u = 0.0;
  for (int32_t i = 0; i < (int32_t)p->actions.size(); i++) {
    const auto& a = p->actions[i];
    if (!(p->planned_time(a, t_step) <= w)) continue;
    const double u = p->ucb(a);
    if (best < 0 || u > best_u || (u == best_u && p->cheaper(a, p->actions[best]))) {
      best = i;
      best_u = u;
    }
  }
  int32_t f = 1;
  if (best < 0) {   // nothing fits the window: the cheapest action overall
    f = 0;
    best = 0;
    for (int32_t i = 1; i < (int32_t)p->actions.size(); i++)
      if (p->cheaper(p->actions[i], p->actions[best])) best = i;
    best_u = p->ucb(p->actions[best]);
  }
  *index = best;
  if (fits) *fits = f;
  if (ucb) *ucb = best_u;
  return DIT_OK;
}

dit_status dit_planner_update(dit_planner* p, int32_t index, double r) {
  if (!p) return set_error(DIT_ERR_INVALID_ARG, "planner is NULL");
  if (index < 0 || index >= (int32_t)p->actions.size()) return set_error(DIT_ERR_INVALID_ARG, "action %d out of range", index);
  if (!std::isfinite(r)) return set_error(DIT_ERR_NAN, "feedback %g is not finite", r);
  auto& a = p->actions[index];
  a.recent.push_back(r);
  if ((int32_t)a.recent.size() > p->window) a.recent.pop_front();
  a.total++;
  p->updates++;
  return DIT_OK;
}

dit_status dit_planner_stats(const dit_planner* p, int32_t index, int32_t* total, int32_t* in_window, double* mean,
                             double* ucb) {
  if (!p) return set_error(DIT_ERR_INVALID_ARG, "planner is NULL");
  if (index < 0 || index >= (int32_t)p->actions.size()) return set_error(DIT_ERR_INVALID_ARG, "action %d out of range", index);
  const auto& a = p->actions[index];
  double sum = 0.0;
  for (double r : a.recent) sum += r;
  if (total) *total = (int32_t)a.total;
  if (in_window) *in_window = (int32_t)a.recent.size();
  if (mean) *mean = a.recent.empty() ? 0.0 : sum / (double)a.recent.size();
  if (ucb) *ucb = p->ucb(a);
  return DIT_OK;
}

dit_status dit_planner_feedback(const float* sigma, const int32_t* explored, int32_t groups, double* r) {
  if (!sigma || !explored || !r || groups < 1) return set_error(DIT_ERR_INVALID_ARG, "sigma / explored / r NULL or groups < 1");
  double all = 0.0, unc = 0.0;
  int32_t n_unc = 0;
  for (int32_t g = 0; g < groups; g++) {
    if (!std::isfinite(sigma[g])) return set_error(DIT_ERR_NAN, "sigma[%d] is not finite", g);
    all += (double)sigma[g];
    if (!explored[g]) {
      unc += (double)sigma[g];
      n_unc++;
    }
  }
  if (n_unc == 0) return set_error(DIT_ERR_DOMAIN, "feedback needs at least one unexplored group");
  const double s_unc = unc / n_unc;
  if (s_unc == 0.0) return set_error(DIT_ERR_DOMAIN, "unexplored groups have zero reward std");
  *r = (all / groups) / s_unc;
  return DIT_OK;
}

dit_status dit_seed_bank_create(int32_t k, dit_seed_bank** out) {
  if (!out) return set_error(DIT_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  if (k < 0) return set_error(DIT_ERR_INVALID_ARG, "k %d < 0", k);
  dit_seed_bank* b = new (std::nothrow) dit_seed_bank();
  if (!b) return set_error(DIT_ERR_INVALID_ARG, "out of host memory");
  b->k = k;
  *out = b;
  return DIT_OK;
}

void dit_seed_bank_destroy(dit_seed_bank* b) { delete b; }

dit_status dit_seed_bank_put(dit_seed_bank* b, int64_t prompt_id, const int64_t* seeds, const float* rewards, int32_t d) {
  if (!b) return set_error(DIT_ERR_INVALID_ARG, "seed bank is NULL");
  if (d < 0 || (d > 0 && (!seeds || !rewards))) return set_error(DIT_ERR_INVALID_ARG, "seeds / rewards NULL or d < 0");
  for (int32_t j = 0; j < d; j++)
    if (!std::isfinite(rewards[j])) return set_error(DIT_ERR_NAN, "rewards[%d] is not finite", j);
  const int32_t k = b->k < d ? b->k : d;
  std::vector<int64_t> kept;
  for (int32_t j : keep_positions(rewards, d, k)) kept.push_back(seeds[j]);
  b->kept[prompt_id] = std::move(kept);
  return DIT_OK;
}

dit_status dit_seed_bank_put_selected(dit_seed_bank* b, const int64_t* prompt_ids, int32_t groups, const int64_t* seeds,
                                      int32_t d, const int32_t* selected, int32_t k) {
  if (!b) return set_error(DIT_ERR_INVALID_ARG, "seed bank is NULL");
  if (groups < 0 || d < 0 || k < 0 || k > d) return set_error(DIT_ERR_INVALID_ARG, "need groups, d >= 0 and 0 <= k <= d");
  if (groups > 0 && (!prompt_ids || (d > 0 && !seeds) || (k > 0 && !selected)))
    return set_error(DIT_ERR_INVALID_ARG, "prompt_ids / seeds / selected NULL");
  for (int64_t i = 0; i < (int64_t)groups * k; i++)
    if (selected[i] < 0 || selected[i] >= d) return set_error(DIT_ERR_INVALID_ARG, "selected[%lld] = %d outside [0, %d)", (long long)i, selected[i], d);
  for (int32_t g = 0; g < groups; g++) {
    std::vector<int64_t> kept;
    for (int32_t j = 0; j < k; j++) kept.push_back(seeds[(int64_t)g * d + selected[(int64_t)g * k + j]]);
    b->kept[prompt_ids[g]] = std::move(kept);
  }
  return DIT_OK;
}

dit_status dit_seed_bank_get(const dit_seed_bank* b, int64_t prompt_id, int64_t* out, int32_t capacity, int32_t* count) {
  if (!b || !count) return set_error(DIT_ERR_INVALID_ARG, "seed bank / count is NULL");
  if (capacity < 0 || (capacity > 0 && !out)) return set_error(DIT_ERR_INVALID_ARG, "out NULL or capacity < 0");
  auto it = b->kept.find(prompt_id);
  if (it == b->kept.end()) {
    *count = 0;
    return DIT_OK;
  }
  const auto& v = it->second;
  for (int32_t j = 0; j < capacity && j < (int32_t)v.size(); j++) out[j] = v[j];
  *count = (int32_t)v.size();
  return DIT_OK;
}

int32_t dit_seed_bank_size(const dit_seed_bank* b) { return b ? (int32_t)b->kept.size() : 0; }

}  // extern "C"
