// Hysteresis-guided reconfiguration (Sec. 3.4): decides when to move between
// pre-specified Train:Rollout configurations so that only sustained
// directional imbalance triggers a resize.  A small host-side state machine,
// fed one (rollout time, training time) pair per step:
//
//   imbalance r = (tr - tt) / max(tr, tt)
//   signal: off -> +1 above +enter, -1 below -enter; +1 holds while r > exit
//           (flips to -1 below -enter, else turns off); -1 symmetric
//   run: consecutive steps with the same nonzero signal
//   resize toward the signal when run >= consecutive, no cooldown is pending,
//   the configuration has been held for `dwell` steps, the next configuration
//   exists, and the resize pays off: the stages' work over the last
//   `consecutive` steps (mean time x GPUs of the current split) predicts the
//   step time in the target split, and the predicted gain per step must be
//   positive and, times the horizon, cover the switch cost (Exp#3: a resize
//   must amortize; the paper's figures give 187 s / (39.84 s - 23.93 s),
//   about 11.75 steps).
#include <cmath>
#include <new>
#include <vector>

#include "dr_internal.h"

struct dr_hyst {
  dr_hyst_params p{};
  std::vector<int32_t> train_gpus, rollout_gpus;  // per configuration
  int32_t config = 0;
  int32_t signal = 0;
  int32_t run = 0;
  int64_t in_config = 0;
  int32_t cooldown_left = 0;
  std::vector<double> win_tr, win_tt;  // the last `consecutive` stage times, oldest first
  int64_t steps = 0;
};

namespace {

// Longest signal run the controller may require; its window holds that many steps.
constexpr int32_t kHystMaxConsecutive = 1 << 20;

// Step time saved per step by moving from split cur to split tgt, predicted
// from the window's work (GPU-seconds = mean stage time x GPUs of the split).
double predicted_gain(const dr_hyst* h, int32_t cur, int32_t tgt) {
  const size_t n = h->win_tr.size();
  double s_tr = 0.0, s_tt = 0.0, s_step = 0.0;
  for (size_t i = 0; i < n; ++i) {
    s_tr += h->win_tr[i];
    s_tt += h->win_tt[i];
    s_step += h->win_tr[i] > h->win_tt[i] ? h->win_tr[i] : h->win_tt[i];
  }
  const double mean_tr = s_tr / (double)n, mean_tt = s_tt / (double)n, mean_step = s_step / (double)n;
  const double work_r = mean_tr * (double)h->rollout_gpus[cur];
  const double work_t = mean_tt * (double)h->train_gpus[cur];
  const double tr2 = work_r / (double)h->rollout_gpus[tgt], tt2 = work_t / (double)h->train_gpus[tgt];
  return mean_step - (tr2 > tt2 ? tr2 : tt2);
}

}  // namespace

using namespace dr;

extern "C" double dr_break_even_steps(double switch_cost_s, double step_before_s, double step_after_s) {
  return switch_cost_s / (step_before_s - step_after_s);
}

extern "C" int dr_hyst_create(const dr_hyst_params* p, dr_hyst** out) {
  clear_error();
  if (!p || !out) return fail(DR_EINVAL, "dr_hyst_create: null argument");
  *out = nullptr;
  if (p->num_configs < 1) return fail(DR_EINVAL, "dr_hyst_create: num_configs must be >= 1");
  if (!p->train_gpus || !p->rollout_gpus) return fail(DR_EINVAL, "dr_hyst_create: null GPU split arrays");
  for (int32_t i = 0; i < p->num_configs; ++i) {
    if (p->train_gpus[i] < 1 || p->rollout_gpus[i] < 1)
      return fail(DR_EINVAL, "dr_hyst_create: configuration %d needs >= 1 GPU in each role", i);
    if (i > 0 && (p->train_gpus[i] >= p->train_gpus[i - 1] || p->rollout_gpus[i] <= p->rollout_gpus[i - 1]))
      return fail(DR_EINVAL, "dr_hyst_create: configurations must go from most training to most rollout GPUs");
  }
  if (p->initial < 0 || p->initial >= p->num_configs) return fail(DR_EINVAL, "dr_hyst_create: initial out of range");
  if (!(p->exit >= 0.0 && p->exit <= p->enter && p->enter < 1.0))
    return fail(DR_EINVAL, "dr_hyst_create: need 0 <= exit <= enter < 1");
  if (p->consecutive < 1 || p->consecutive > kHystMaxConsecutive)
    return fail(DR_EINVAL, "dr_hyst_create: consecutive must be in [1, %d]", kHystMaxConsecutive);
  if (p->dwell < 0 || p->cooldown < 0) return fail(DR_EINVAL, "dr_hyst_create: dwell and cooldown must be >= 0");
  if (!(p->switch_cost_s >= 0.0) || !std::isfinite(p->switch_cost_s))
    return fail(DR_EINVAL, "dr_hyst_create: switch_cost_s must be finite and >= 0");
  if (p->horizon_steps < 0 || (p->switch_cost_s > 0.0 && p->horizon_steps < 1))
    return fail(DR_EINVAL, "dr_hyst_create: horizon_steps must be >= 1 when switch_cost_s > 0");
  dr_hyst* h = nullptr;
  try {
    h = new dr_hyst();
    h->p = *p;
    h->train_gpus.assign(p->train_gpus, p->train_gpus + p->num_configs);
    h->rollout_gpus.assign(p->rollout_gpus, p->rollout_gpus + p->num_configs);
    // the window never grows past `consecutive`, so dr_hyst_step never allocates
    h->win_tr.reserve((size_t)p->consecutive);
    h->win_tt.reserve((size_t)p->consecutive);
  } catch (...) {
    delete h;
    return fail(DR_ENOMEM, "dr_hyst_create: out of memory");
  }
  h->p.train_gpus = h->train_gpus.data();
  h->p.rollout_gpus = h->rollout_gpus.data();
  h->config = p->initial;
  *out = h;
  return DR_OK;
}

extern "C" void dr_hyst_destroy(dr_hyst* h) { delete h; }

extern "C" int dr_hyst_step(dr_hyst* h, double tr, double tt, dr_hyst_decision* out) {
  clear_error();
  if (!h || !out) return fail(DR_EINVAL, "dr_hyst_step: null argument");
  if (!(tr >= 0.0) || !(tt >= 0.0) || !std::isfinite(tr) || !std::isfinite(tt))
    return fail(DR_EINVAL, "dr_hyst_step: stage times must be finite and >= 0");
  const dr_hyst_params& p = h->p;
  h->steps += 1;
  h->in_config += 1;
  const bool blocked = h->cooldown_left > 0;
  if (blocked) h->cooldown_left -= 1;
  const double m = tr > tt ? tr : tt;
  const double r = m == 0.0 ? 0.0 : (tr - tt) / m;
  int32_t sig;
  if (h->signal == 0)
    sig = r > p.enter ? 1 : (r < -p.enter ? -1 : 0);
  else if (h->signal == 1)
    sig = r > p.exit ? 1 : (r < -p.enter ? -1 : 0);
  else
    sig = r < -p.exit ? -1 : (r > p.enter ? 1 : 0);
  h->run = (sig != 0 && sig == h->signal) ? h->run + 1 : (sig != 0 ? 1 : 0);
  h->signal = sig;
  if ((int32_t)h->win_tr.size() == p.consecutive) {
    h->win_tr.erase(h->win_tr.begin());
    h->win_tt.erase(h->win_tt.begin());
  }
  h->win_tr.push_back(tr);
  h->win_tt.push_back(tt);

  int32_t reason;
  double gain = 0.0;
  if (sig == 0)
    reason = DR_HYST_BALANCED;
  else if (h->run < p.consecutive)
    reason = DR_HYST_PERSISTENCE;
  else if (blocked)
    reason = DR_HYST_COOLDOWN;
  else if (h->in_config < p.dwell)
    reason = DR_HYST_DWELL;
  else if (h->config + sig < 0 || h->config + sig >= p.num_configs)
    reason = DR_HYST_EDGE;
  else if (!((gain = predicted_gain(h, h->config, h->config + sig)) > 0.0) ||
           (p.switch_cost_s > 0.0 && gain * (double)p.horizon_steps < p.switch_cost_s))
    reason = DR_HYST_AMORTIZE;
  else
    reason = DR_HYST_RESIZE;
  out->action = 0;
  out->run = h->run;
  out->imbalance = r;
  out->predicted_gain_s = gain;
  if (reason == DR_HYST_RESIZE) {
    out->action = sig;
    h->config += sig;
    h->signal = 0;
    h->run = 0;
    h->in_config = 0;
    h->cooldown_left = p.cooldown;
  }
  out->config = h->config;
  out->reason = reason;
  return DR_OK;
}
