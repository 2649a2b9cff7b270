// nf_control.cpp - the controller-input layer on the host: Supervisor
// recovery (CUSUM over a smoothed loss, cooldown, guarded readmission,
// noise-aware short recovery), Commander's admission point, the route-use
// budget guard, route accounting (L/F/P, MGTR) and the endpoint-capacity
// guard's cost model.  Its outputs are the admitted / veto / guard_ok inputs
// of nf_route_policy.  Pure host code: no device calls.
//
// Readings (the paper describes these mechanisms without formulas; §4.3,
// §4.4, §6.4 and the appendix's controller table name their inputs):
//   R22 Health signal: s_0 = loss_0, s_t = s_{t-1} + alpha (loss_t - s_{t-1}).
//   R23 Detector (Page's one-sided CUSUM on the per-step increase of s, §4.1's
//       slack and threshold): x_t = s_t - s_{t-1};
//       S_t = max(0, S_{t-1} + x_t - slack), accumulated only on steps run
//       with low-bit admitted and not vetoed; alarm when S_t > threshold
//       (threshold * guard_scale while the readmission guard is active).
//   R24 Recovery: an alarm starts an FP32 cooldown (veto) of cooldown_steps
//       steps and resets S; a near-threshold alarm (S_t <= threshold_eff *
//       (1 + near_band)) with a small loss movement (|loss_t - loss_{t-1}| <=
//       small_move) uses short_cooldown_steps instead when that is > 0.
//   R25 Readmission: after the cooldown, low-bit is readmitted under a guard
//       of guard_steps steps with the stricter threshold; an alarm in the
//       guard starts a new cooldown; guard_steps = 0 readmits directly.
//   R26 Commander: low-bit is admitted from step admit_step on (before it the
//       route is plain FP32, NOT_ADMITTED).
//   R27 Route-use budget: the realized low-bit share L / (L + F + P) over the
//       route events recorded so far; when it exceeds target_share +
//       share_margin the next step's eligible buckets are vetoed.
//   R28 Endpoint-capacity guard, per bucket of n elements (n_E eligible) on
//       N nodes x P GPUs (W = N P), b payload bits per eligible element:
//         T_fp32 = lat_fp32 + 2 (W - 1) / W * 4 n / B_net  (ring all-reduce)
//         T_low  = lat_low + b n_E / 8 / B_net             (payload to the node endpoint)
//                + P b n_E / 8 / R_ep                      (node-local counting)
//                + 2 (N - 1) / N * n_E / B_net             (uint8 partial-count exchange)
//                + n_E / B_net                             (aggregate return)
//                + 2 (W - 1) / W * 4 (n - n_E) / B_net     (routed part, FP32)
//       guard_ok = T_low < T_fp32.
#include <math.h>
#include <string.h>

#include "nf_internal.h"

namespace {

bool is_finite(double x) { return x - x == 0.0; }

nf_status bad(const char* what) { return nf::set_error(NF_ERR_INVALID_ARG, what); }

}  // namespace

extern "C" {

nf_status nf_supervisor_init(const nf_supervisor_profile* p, nf_supervisor_state* s) {
  if (!p || !s) return bad("NULL profile or state");
  if (!(p->ema_alpha > 0.0 && p->ema_alpha <= 1.0)) return bad("ema_alpha outside (0, 1]");
  if (!is_finite(p->slack) || !(p->threshold > 0.0) || !is_finite(p->threshold)) return bad("slack must be finite, threshold finite and > 0");
  if (p->admit_step < 0 || p->cooldown_steps < 0 || p->guard_steps < 0 || p->short_cooldown_steps < 0)
    return bad("negative step count");
  if (!(p->guard_scale > 0.0 && p->guard_scale <= 1.0)) return bad("guard_scale outside (0, 1]");
  if (!(p->near_band >= 0.0) || !(p->small_move >= 0.0) || !is_finite(p->near_band) || !is_finite(p->small_move))
    return bad("near_band and small_move must be finite and >= 0");
  if (!(p->share_margin >= 0.0) || p->target_share != p->target_share) return bad("share_margin must be >= 0, target_share a number");
  memset(s, 0, sizeof *s);
  s->state = p->admit_step > 0 ? NF_SUP_WARMUP : NF_SUP_LOWBIT;
  return nf::set_error(NF_OK, "");
}

nf_status nf_supervisor_policy(const nf_supervisor_profile* p, const nf_supervisor_state* s,
                               nf_route_policy* pol) {
  if (!p || !s || !pol) return bad("NULL profile, state or policy");
  pol->admitted = s->state != NF_SUP_WARMUP;
  const int64_t events = s->events_l + s->events_f + s->events_p;
  const bool over_budget =
      events > 0 && (double)s->events_l / (double)events > p->target_share + p->share_margin;
  pol->veto = s->state == NF_SUP_COOLDOWN || over_budget;
  return nf::set_error(NF_OK, "");
}

nf_status nf_supervisor_update(const nf_supervisor_profile* p, nf_supervisor_state* s,
                               const nf_route_decision* decisions_host, int64_t nb, double loss) {
  if (!p || !s || nb < 0 || (nb > 0 && !decisions_host) || !is_finite(loss))
    return bad("NULL profile/state/decisions, nb < 0 or a non-finite loss");
  // the step's route events and modeled bytes (§3.2)
  nf_route_policy pol;
  nf_supervisor_policy(p, s, &pol);
  for (int64_t b = 0; b < nb; ++b) {
    const nf_route_decision& d = decisions_host[b];
    if (d.route == NF_ROUTE_LOWBIT) ++s->events_l;
    else if (d.route == NF_ROUTE_FALLBACK) ++s->events_f;
    else ++s->events_p;
    s->bytes_route += d.bytes_route;
    s->bytes_fp32 += d.bytes_fp32;
  }
  if (pol.veto && s->state != NF_SUP_COOLDOWN) ++s->budget_vetoes;
  // health signal and detector (R22, R23)
  const bool first = !s->has_prev;
  const double prev_s = first ? loss : s->smoothed;
  const double cur_s = first ? loss : s->smoothed + p->ema_alpha * (loss - s->smoothed);
  const double x = cur_s - prev_s;
  const double move = first ? 0.0 : fabs(loss - s->prev_loss);
  s->smoothed = cur_s;
  s->prev_loss = loss;
  s->has_prev = 1;
  const bool watching = (s->state == NF_SUP_LOWBIT || s->state == NF_SUP_GUARD) && !pol.veto;
  bool alarm = false;
  double thr = p->threshold;
  if (watching) {
    if (s->state == NF_SUP_GUARD) thr = p->threshold * p->guard_scale;
    const double v = s->cusum + x - p->slack;
    s->cusum = v > 0.0 ? v : 0.0;
    alarm = s->cusum > thr;
  }
  // state machine (R24-R26)
  const int64_t next = s->step + 1;
  switch (s->state) {
    case NF_SUP_WARMUP:
      if (next >= p->admit_step) s->state = NF_SUP_LOWBIT;
      break;
    case NF_SUP_LOWBIT:
    case NF_SUP_GUARD:
      if (alarm) {
        ++s->alarms;
        const bool near = s->cusum <= thr * (1.0 + p->near_band) && move <= p->small_move;
        int32_t len = p->cooldown_steps;
        if (near && p->short_cooldown_steps > 0) {
          len = p->short_cooldown_steps;
          ++s->short_recoveries;
        }
        s->cusum = 0.0;
        if (len > 0) {
          s->state = NF_SUP_COOLDOWN;
          s->cooldown_left = len;
        } else if (p->guard_steps > 0) {
          s->state = NF_SUP_GUARD;
          s->guard_left = p->guard_steps;
          ++s->readmissions;
        } else {
          s->state = NF_SUP_LOWBIT;
          ++s->readmissions;
        }
      } else if (s->state == NF_SUP_GUARD && !pol.veto) {
        if (--s->guard_left <= 0) s->state = NF_SUP_LOWBIT;
      }
      break;
    case NF_SUP_COOLDOWN:
      if (--s->cooldown_left <= 0) {
        ++s->readmissions;
        s->cusum = 0.0;
        if (p->guard_steps > 0) {
          s->state = NF_SUP_GUARD;
          s->guard_left = p->guard_steps;
        } else {
          s->state = NF_SUP_LOWBIT;
        }
      }
      break;
    default:
      return bad("state holds an unknown Supervisor state");
  }
  s->step = next;
  return nf::set_error(NF_OK, "");
}

nf_status nf_endpoint_guard(const nf_endpoint_model* m, int64_t n, int64_t n_eligible,
                            double* t_fp32, double* t_lowbit, int32_t* guard_ok) {
  if (!m || !t_fp32 || !t_lowbit || !guard_ok) return bad("NULL model or output");
  if (m->nodes < 1 || m->gpus_per_node < 1 || (m->bits_per_element != 1 && m->bits_per_element != 2))
    return bad("nodes and gpus_per_node >= 1, bits_per_element 1 or 2");
  if (!(m->net_bytes_per_s > 0.0) || !(m->endpoint_bytes_per_s > 0.0) || !(m->latency_fp32_s >= 0.0) ||
      !(m->latency_lowbit_s >= 0.0))
    return bad("rates must be > 0 and latencies >= 0");
  if (n < 0 || n_eligible < 0 || n_eligible > n) return bad("need 0 <= n_eligible <= n");
  const double N = m->nodes, P = m->gpus_per_node, W = N * P, B = m->net_bytes_per_s;
  const double b = m->bits_per_element, nE = (double)n_eligible, nF = (double)(n - n_eligible);
  const double ring = 2.0 * (W - 1.0) / W;
  const double tf = m->latency_fp32_s + ring * 4.0 * (double)n / B;
  const double payload = b * nE / 8.0;
  const double tl = m->latency_lowbit_s + payload / B + P * payload / m->endpoint_bytes_per_s +
                    2.0 * (N - 1.0) / N * nE / B + nE / B + ring * 4.0 * nF / B;
  *t_fp32 = tf;
  *t_lowbit = tl;
  *guard_ok = tl < tf;
  return nf::set_error(NF_OK, "");
}

}  // extern "C"
