"""Meta-test: the schedule oracle's pins are discriminating.  Each case plants one
plausible mistake in a copy of oracle/schedule.py (an off-by-one gate of Lemma 1, a
swapped row of Table 2, a wrong warmup count, a dropped edge, a simulator that ignores
dependencies, a cost without the slab share, ...) and runs the pin suite against it:
at least one pin must fail."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "schedule.py")

MUTATIONS = {
    "send_gate_inclusive": ("sends = [any(trainable[i] for i in range(j)) for j in range(k)]",
                            "sends = [any(trainable[i] for i in range(j + 1)) for j in range(k)]"),
    "receive_gate_strict": ("receives = [any(trainable[i] for i in range(j + 1)) for j in range(k)]",
                            "receives = [any(trainable[i] for i in range(max(j, 1))) for j in range(k)]"),
    "seam_rows_swapped": ('("Sharded", "Replicated"): ("Scatter", "Gather"),',
                          '("Sharded", "Replicated"): ("Gather", "Scatter"),'),
    "reduce_group_swapped": ('"ReplicaGroup" if lay[j] == "Replicated" else "DataGroup"',
                             '"DataGroup" if lay[j] == "Replicated" else "ReplicaGroup"'),
    "warmup_off_by_one": ("warm = min(P - 1 - r, M)", "warm = min(P - r, M)"),
    "interleaved_warmup_halved": ("min(2 * (P - 1 - r) + (S - 1) * P, total)",
                                  "min((P - 1 - r) + (S - 1) * P, total)"),
    "no_stored_activation_edge": ('edges.append((("Fwd", j, r, m), e, "Activation"))\n', ""),
    "turnaround_as_gradient": ('prev, kind = ("Loss", m), "Turnaround"',
                               'prev, kind = ("Loss", m), "Gradient"'),
    "simulator_ignores_edges": ("ready = all(p in done for p in preds[e])", "ready = True"),
    "slab_share_dropped": ("c = c * (hi - lo) / (bounds[j + 1] - bounds[j])", "c = c"),
    "frozen_activation_kept": ('if ("Bwd",) + e[1:] not in bwds:\n                    live -= act_bytes[e]',
                               'if False:\n                    live -= act_bytes[e]'),
    "encoder_backward_first": ('        if lay[0] == "Replicated" and receives[k - 1]:\n            for m in mine:\n                bwd(0, m)\n',
                               ""),
    "validity_allows_adjacent_transposes": ('return not any(layout(schedule[i]) == "Replicated" == layout(schedule[i + 1])',
                                            'return True or not any(layout(schedule[i]) == "Replicated" == layout(schedule[i + 1])'),
}


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_planted_mistake_is_caught(name, tmp_path):
    a, b = MUTATIONS[name]
    src = open(SRC).read()
    assert a in src, f"mutation anchor for {name} no longer present in the oracle source"
    mut = tmp_path / "schedule_mut.py"
    mut.write_text(src.replace(a, b, 1))
    env = dict(os.environ, MPIPE_SCHEDULE_ORACLE=str(mut))
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_oracle_schedule_pins.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode != 0, f"no pin caught the planted mistake '{name}'"
    assert "failed" in r.stdout or "error" in r.stdout.lower()
