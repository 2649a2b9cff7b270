"""Planted mistakes in copies of the reference controller (oracle/controller.py)
must each fail at least one pin of tests/test_controller.py.  The real
module is never modified: each mutant is loaded from a temporary copy."""
import importlib.util
import os
import tempfile

import pytest

from oracle import controller
from tests import test_controller as tc

SRC = controller.__file__

MUTANTS = [
    ("ema_no_smoothing", "self.smoothed = before + self.p[\"ema_alpha\"] * (loss - before)", "self.smoothed = loss"),
    ("increase_from_raw_loss", "x = self.smoothed - before", "x = loss - self.prev_loss"),
    ("cusum_without_slack", "self.cusum + x - self.p[\"slack\"]", "self.cusum + x"),
    ("cusum_two_sided", "self.cusum = max(0.0, self.cusum + x - self.p[\"slack\"])",
     "self.cusum = max(0.0, self.cusum + abs(x) - self.p[\"slack\"])"),
    ("alarm_ge", "alarm = self.cusum > thr", "alarm = self.cusum >= thr"),
    ("guard_threshold_ignored", "thr = self.p[\"threshold\"] * self.p[\"guard_scale\"]", "thr = self.p[\"threshold\"]"),
    ("watch_during_warmup", "if self.state in (LOWBIT, GUARD) and not veto:", "if not veto:"),
    ("cusum_not_reset_on_alarm", "                self.cusum = 0.0\n                if length > 0:",
     "                if length > 0:"),
    ("cooldown_one_short", "self.state, self.cooldown_left = COOLDOWN, length",
     "self.state, self.cooldown_left = COOLDOWN, length - 1"),
    ("short_recovery_ignores_move", " and move <= self.p[\"small_move\"]", ""),
    ("admission_one_late", "if self.step + 1 >= self.p[\"admit_step\"]:", "if self.step + 1 > self.p[\"admit_step\"]:"),
    ("budget_without_margin", "return share > self.p[\"target_share\"] + self.p[\"share_margin\"]",
     "return share > self.p[\"target_share\"]"),
    ("budget_ge", "return share > self.p[\"target_share\"] + self.p[\"share_margin\"]",
     "return share >= self.p[\"target_share\"] + self.p[\"share_margin\"]"),
    ("mgtr_inverted", "return self.bytes_route / self.bytes_fp32", "return self.bytes_fp32 / self.bytes_route"),
    ("ring_factor_one", "ring = 2.0 * (workers - 1) / workers", "ring = (workers - 1) / workers"),
    ("fp32_bytes_not_four", "t_fp32 = latency_fp32_s + ring * 4.0 * n / net_bytes_per_s",
     "t_fp32 = latency_fp32_s + ring * n / net_bytes_per_s"),
    ("count_not_times_fanin", "t_count = gpus_per_node * payload / endpoint_bytes_per_s",
     "t_count = payload / endpoint_bytes_per_s"),
    ("exchange_over_workers", "t_exchange = 2.0 * (nodes - 1) / nodes * n_eligible / net_bytes_per_s",
     "t_exchange = 2.0 * (workers - 1) / workers * n_eligible / net_bytes_per_s"),
    ("routed_part_dropped", "t_routed = ring * 4.0 * (n - n_eligible) / net_bytes_per_s", "t_routed = 0.0"),
    ("payload_bits_as_bytes", "payload = bits_per_element * n_eligible / 8.0", "payload = bits_per_element * n_eligible"),
]


def load_mutant(old, new):
    src = open(SRC).read()
    assert src.count(old) == 1, old
    d = tempfile.mkdtemp()
    path = os.path.join(d, "controller_mutant.py")
    open(path, "w").write(src.replace(old, new))
    spec = importlib.util.spec_from_file_location("controller_mutant", path)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_fails_a_pin(name, old, new):
    mod = load_mutant(old, new)
    failed = []
    for pin in tc.PINS:
        try:
            pin(mod)
        except (AssertionError, ZeroDivisionError, TypeError, KeyError):
            failed.append(pin.__name__)
    assert failed, f"mutant {name} passes every pin"
