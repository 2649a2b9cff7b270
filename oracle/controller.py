"""Reference controller: Supervisor recovery, Commander admission, the
route-use budget guard, route accounting and the endpoint-capacity guard.

TEST INFRASTRUCTURE ONLY (like the rest of oracle/): plain Python written
from the paper's description of the controller, used to check the library's
host controller.  It shares no code with the library.

The paper gives these mechanisms without formulas (§4.1 defines slack and
threshold of the CUSUM detector; §4.3 fallback, cooldown and guarded
readmission; §4.4 and the appendix's controller table the route-use budget
with a guard band and the noise-aware short recovery; §6.4 the endpoint
guard's comparison and its inputs).  The readings it follows:
  R22 smoothed health signal: s_0 = loss_0, s_t = s_{t-1} + alpha (loss_t - s_{t-1})
  R23 Page's one-sided CUSUM on the increase x_t = s_t - s_{t-1}:
      S_t = max(0, S_{t-1} + x_t - slack), only on steps run in low-bit
      (admitted, not vetoed); alarm when S_t exceeds the threshold (times
      guard_scale during the readmission guard)
  R24 an alarm starts an FP32 cooldown of cooldown_steps and resets S; a
      near-threshold alarm (S_t <= thr (1 + near_band)) with a small loss move
      (|loss_t - loss_{t-1}| <= small_move) gets short_cooldown_steps if > 0
  R25 after the cooldown, a guard of guard_steps low-bit steps with the
      stricter threshold; an alarm there restarts the cooldown
  R26 Commander admits low-bit from step admit_step on
  R27 the next step is vetoed when L / (L + F + P) over the events so far
      exceeds target_share + share_margin
  R28 endpoint guard: ring FP32 time against the hierarchical low-bit time
      (payload to the node, node-local counting at the endpoint rate,
      partial-count exchange between nodes, aggregate return, routed part
      in FP32); low-bit is admitted when it is strictly faster.
"""
WARMUP, LOWBIT, COOLDOWN, GUARD = 0, 1, 2, 3
ROUTE_L, ROUTE_F, ROUTE_P = 0, 1, 2


class Supervisor:
    """One run of the controller; `profile` is a dict with the fields of
    nf_supervisor_profile."""

    def __init__(self, profile):
        self.p = dict(profile)
        self.step = 0
        self.state = WARMUP if self.p["admit_step"] > 0 else LOWBIT
        self.smoothed = None
        self.prev_loss = None
        self.cusum = 0.0
        self.cooldown_left = 0
        self.guard_left = 0
        self.alarms = 0
        self.short_recoveries = 0
        self.readmissions = 0
        self.budget_vetoes = 0
        self.events = {ROUTE_L: 0, ROUTE_F: 0, ROUTE_P: 0}
        self.bytes_route = 0.0
        self.bytes_fp32 = 0.0

    # -- inputs of the next step's route policy
    def over_budget(self):
        total = self.events[ROUTE_L] + self.events[ROUTE_F] + self.events[ROUTE_P]
        if total == 0:
            return False
        share = self.events[ROUTE_L] / total
        return share > self.p["target_share"] + self.p["share_margin"]

    def policy(self):
        """(admitted, veto) for the next step."""
        admitted = self.state != WARMUP
        veto = self.state == COOLDOWN or self.over_budget()
        return admitted, veto

    def mgtr(self):
        return self.bytes_route / self.bytes_fp32 if self.bytes_fp32 else None

    # -- after the step
    def update(self, decisions, loss):
        """decisions: (route, bytes_route, bytes_fp32) per bucket of the step."""
        admitted, veto = self.policy()
        for route, b_route, b_fp32 in decisions:
            self.events[route] += 1
            self.bytes_route += b_route
            self.bytes_fp32 += b_fp32
        if veto and self.state != COOLDOWN:
            self.budget_vetoes += 1

        if self.smoothed is None:
            x, move = 0.0, 0.0
            self.smoothed = loss
        else:
            before = self.smoothed
            self.smoothed = before + self.p["ema_alpha"] * (loss - before)
            x = self.smoothed - before
            move = abs(loss - self.prev_loss)
        self.prev_loss = loss

        thr = self.p["threshold"]
        alarm = False
        if self.state in (LOWBIT, GUARD) and not veto:
            if self.state == GUARD:
                thr = self.p["threshold"] * self.p["guard_scale"]
            self.cusum = max(0.0, self.cusum + x - self.p["slack"])
            alarm = self.cusum > thr

        if self.state == WARMUP:
            if self.step + 1 >= self.p["admit_step"]:
                self.state = LOWBIT
        elif self.state in (LOWBIT, GUARD):
            if alarm:
                self.alarms += 1
                near = self.cusum <= thr * (1.0 + self.p["near_band"]) and move <= self.p["small_move"]
                length = self.p["cooldown_steps"]
                if near and self.p["short_cooldown_steps"] > 0:
                    length = self.p["short_cooldown_steps"]
                    self.short_recoveries += 1
                self.cusum = 0.0
                if length > 0:
                    self.state, self.cooldown_left = COOLDOWN, length
                else:
                    self.readmissions += 1
                    self._readmit()
            elif self.state == GUARD and not veto:
                self.guard_left -= 1
                if self.guard_left <= 0:
                    self.state = LOWBIT
        elif self.state == COOLDOWN:
            self.cooldown_left -= 1
            if self.cooldown_left <= 0:
                self.readmissions += 1
                self.cusum = 0.0
                self._readmit()
        self.step += 1

    def _readmit(self):
        if self.p["guard_steps"] > 0:
            self.state, self.guard_left = GUARD, self.p["guard_steps"]
        else:
            self.state = LOWBIT


def endpoint_times(nodes, gpus_per_node, bits_per_element, net_bytes_per_s, endpoint_bytes_per_s,
                   latency_fp32_s, latency_lowbit_s, n, n_eligible):
    """(t_fp32, t_lowbit, guard_ok) of one bucket (R28)."""
    workers = nodes * gpus_per_node
    ring = 2.0 * (workers - 1) / workers            # ring all-reduce: each byte crosses 2 (W-1)/W links
    t_fp32 = latency_fp32_s + ring * 4.0 * n / net_bytes_per_s
    payload = bits_per_element * n_eligible / 8.0   # one worker's low-bit payload, bytes
    t_send = payload / net_bytes_per_s              # worker -> node endpoint
    t_count = gpus_per_node * payload / endpoint_bytes_per_s   # the endpoint counts P streams
    t_exchange = 2.0 * (nodes - 1) / nodes * n_eligible / net_bytes_per_s  # uint8 partial counts
    t_return = n_eligible / net_bytes_per_s         # aggregate back to the workers
    t_routed = ring * 4.0 * (n - n_eligible) / net_bytes_per_s
    t_low = latency_lowbit_s + t_send + t_count + t_exchange + t_return + t_routed
    return t_fp32, t_low, t_low < t_fp32
