// One rollout round and its training under Slime, CGP or CGP+FGD scheduling
// (Sections 3.2-3.3, Eq. 2-6, Algorithm 1), as a discrete-event simulation on
// the host.
//
// Rollout node: between two events (a request finishing) the running set is
// fixed, so the simulation jumps from one finishing step to the next instead
// of visiting every request at every step: a min-heap holds each running
// request's finishing step, the context sum grows by n tokens per step, and
// only the per-step time is accumulated step by step (in the documented
// order, so the result is bitwise reproducible). Admission happens at the
// scheduling cycle before each step: the FGD frontier is refilled in group
// order while it holds fewer than F_w groups (cgp_fgd), then admitted requests
// move first come first served into the running set while it holds fewer
// than max_running, the first request of a group bringing the group's
// prompt prefill into that step.
//
// Control node: a serving-complete group is trainable after its
// materialisation delay and joins the FIFO (by time, ties by group order).
// Training node: update k takes FIFO entries kU..kU+U-1 once the trainer is
// free and they are all trainable (CGP), or once every group is (Slime).
//
// Built without floating-point contraction: each time is the same IEEE
// expression, evaluated in the same order, as the definition in rp.h.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <deque>
#include <queue>
#include <vector>

#include "rp.h"
#include "rp_host.h"

namespace {

struct Finish {
  int64_t step;  // the request finishes at the end of this step (1-based)
  int32_t req;
  bool operator>(const Finish& o) const { return step != o.step ? step > o.step : req > o.req; }
};

bool finite_nonneg(double x) { return std::isfinite(x) && x >= 0.0; }

}  // namespace

extern "C" rp_status rp_sched_simulate(const rp_sched_config* cfg, const int32_t* prompt_lens,
                                       const int32_t* resp_lens, rp_sched_summary* summary, double* serve_done,
                                       double* frontier_enter, double* trainable, int32_t* fifo,
                                       double* update_start, double* update_end) {
  rp::clear_error();
  if (cfg == nullptr || prompt_lens == nullptr || resp_lens == nullptr || summary == nullptr)
    return rp::set_error(RP_ERR_INVALID_ARG, "config, prompt_lens, resp_lens and summary must be non-NULL");
  const int R = cfg->num_groups, K = cfg->group_size, U = cfg->update_groups;
  const int mode = rp::enum_bits(cfg->mode);
  const bool fgd = mode == RP_SCHED_CGP_FGD, slime = mode == RP_SCHED_SLIME;
  if (mode != RP_SCHED_SLIME && mode != RP_SCHED_CGP && !fgd)
    return rp::set_error(RP_ERR_INVALID_ARG, "unknown scheduling mode");
  if (R < 1 || K < 1 || U < 1 || R % U != 0 || cfg->max_running < 1 || (int64_t)R * K > INT32_MAX)
    return rp::set_error(RP_ERR_INVALID_ARG,
                         "need num_groups, group_size, update_groups, max_running >= 1 and update_groups | num_groups");
  if (fgd && cfg->frontier_width < 1) return rp::set_error(RP_ERR_INVALID_ARG, "frontier_width must be >= 1");
  const double costs[] = {cfg->step_base, cfg->step_per_seq, cfg->step_per_ctx_token, cfg->prefill_per_token,
                          cfg->mat_base, cfg->mat_per_token, cfg->train_base, cfg->train_per_token, cfg->opt_step};
  for (double c : costs)
    if (!finite_nonneg(c)) return rp::set_error(RP_ERR_INVALID_ARG, "cost parameters must be finite and >= 0");
  const int N = R * K;
  for (int g = 0; g < R; ++g)
    if (prompt_lens[g] < 0) return rp::set_error(RP_ERR_INVALID_ARG, "prompt lengths must be >= 0");
  for (int q = 0; q < N; ++q)
    if (resp_lens[q] < 1) return rp::set_error(RP_ERR_INVALID_ARG, "response lengths must be >= 1");

  // ---- rollout node ---------------------------------------------------------
  std::deque<int32_t> admitted;
  if (!fgd)
    for (int q = 0; q < N; ++q) admitted.push_back(q);
  int next_deferred = 0, frontier = 0;
  std::vector<double> done(R, 0.0), enter(R, 0.0);
  std::vector<int> left(R, K);
  std::vector<char> started(R, 0);
  std::priority_queue<Finish, std::vector<Finish>, std::greater<Finish>> running;
  int64_t n = 0, ctx = 0, steps = 0;
  double t = 0.0;
  const double per_step = cfg->step_base, per_seq = cfg->step_per_seq, per_ctx = cfg->step_per_ctx_token;
  for (;;) {
    if (fgd) {
      while (frontier < cfg->frontier_width && next_deferred < R) {
        const int g = next_deferred++;
        ++frontier;
        enter[g] = t;
        for (int i = 0; i < K; ++i) admitted.push_back(g * K + i);
      }
    }
    double prefill = 0.0;
    while (n < cfg->max_running && !admitted.empty()) {
      const int q = admitted.front();
      admitted.pop_front();
      const int g = q / K;
      running.push({steps + resp_lens[q], q});
      ++n;
      ctx += prompt_lens[g];
      if (!started[g]) {
        started[g] = 1;
        prefill += cfg->prefill_per_token * (double)prompt_lens[g];
      }
    }
    if (n == 0) break;
    // Steps up to and including the next one in which a request finishes.
    const int64_t k = running.top().step - steps;
    for (int64_t j = 0; j < k; ++j) {
      double d = per_step + per_seq * (double)n;
      d = d + per_ctx * (double)(ctx + j * n);
      d = d + (j == 0 ? prefill : 0.0);
      t = t + d;
    }
    steps += k;
    ctx += k * n;
    while (!running.empty() && running.top().step == steps) {
      const int q = running.top().req;
      running.pop();
      const int g = q / K;
      --n;
      ctx -= prompt_lens[g] + resp_lens[q];
      if (--left[g] == 0) {
        done[g] = t;
        if (fgd) --frontier;
      }
    }
  }

  // ---- control node ---------------------------------------------------------
  std::vector<int64_t> resp_tok(R, 0);
  for (int q = 0; q < N; ++q) resp_tok[q / K] += resp_lens[q];
  std::vector<double> ready(R);
  for (int g = 0; g < R; ++g) ready[g] = done[g] + (cfg->mat_base + cfg->mat_per_token * (double)resp_tok[g]);
  std::vector<int32_t> order(R);
  for (int g = 0; g < R; ++g) order[g] = g;
  std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return ready[a] < ready[b]; });

  // ---- training node --------------------------------------------------------
  double t_complete = ready[0];
  for (int g = 1; g < R; ++g) t_complete = std::max(t_complete, ready[g]);
  std::vector<double> comp(R);
  for (int g = 0; g < R; ++g)
    comp[g] = cfg->train_base + cfg->train_per_token * (double)((int64_t)K * prompt_lens[g] + resp_tok[g]);
  double free_at = 0.0, compute = 0.0, first_start = 0.0;
  for (int k = 0; k < R / U; ++k) {
    const double avail = slime ? t_complete : ready[order[(k + 1) * U - 1]];
    const double start = std::max(free_at, avail);
    double dur = 0.0;
    for (int u = 0; u < U; ++u) dur = dur + comp[order[k * U + u]];
    dur = dur + cfg->opt_step;
    free_at = start + dur;
    compute = compute + dur;
    if (k == 0) first_start = start;
    if (update_start != nullptr) update_start[k] = start;
    if (update_end != nullptr) update_end[k] = free_at;
  }

  summary->t_first_u = ready[order[U - 1]];
  summary->t_complete = t_complete;
  summary->t_start = first_start;
  summary->delta_cgp = t_complete - summary->t_first_u;
  summary->t_train_end = free_at;
  summary->compute = compute;
  summary->wait = free_at - compute;
  summary->w_train = free_at > 0.0 ? first_start / free_at : 0.0;
  summary->wait_ratio = free_at > 0.0 ? summary->wait / free_at : 0.0;
  summary->steps = steps;
  for (int g = 0; g < R; ++g) {
    if (serve_done != nullptr) serve_done[g] = done[g];
    if (frontier_enter != nullptr) frontier_enter[g] = enter[g];
    if (trainable != nullptr) trainable[g] = ready[g];
    if (fifo != nullptr) fifo[g] = order[g];
  }
  return RP_OK;
}
