"""Plants one plausible mistake at a time in a copy of the oracle's discovery
procedure (oracle/discover.py, on the CPU) and checks that the procedure
pins catch each one."""
import importlib.util
import os

import pytest

import tests.test_oracle_discover as P

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "discover.py")

MUTATIONS = {
    "necessity_ge": ("necessary.append(1 if d > eps else 0)", "necessary.append(1 if d >= eps else 0)"),
    "greedy_picks_largest": ("if best_d is None or dc < best_d:", "if best_d is None or dc > best_d:"),
    "ties_to_highest_index": ("if best_d is None or dc < best_d:", "if best_d is None or dc <= best_d:"),
    "greedy_stops_after_one": ("while d > eps and sum(pcs) < k:", "if d > eps and sum(pcs) < k:"),
    "control_inverted": ("control_ok = 1 if d_control > eps else 0", "control_ok = 1 if d_control <= eps else 0"),
    "sufficiency_skipped": ("    d_necessary = run(pcs)\n", "    d_necessary = 0.0\n"),
}

PINS = [P.test_procedure_necessity_and_sufficiency, P.test_procedure_redundant_pair_tie_goes_to_lowest_index,
        P.test_procedure_multi_step_greedy, P.test_procedure_tolerance_and_no_convergence]


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_planted_mistake_is_caught(tmp_path, name, monkeypatch):
    old, new = MUTATIONS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, name
    path = tmp_path / "discover_mut.py"
    path.write_text(src.replace(old, new))
    spec = importlib.util.spec_from_file_location("oracle.discover_mut", str(path))
    mod = importlib.util.module_from_spec(spec)
    mod.__package__ = "oracle"
    spec.loader.exec_module(mod)
    monkeypatch.setattr(P, "D", mod)
    caught = 0
    for pin in PINS:
        try:
            pin()
        except AssertionError:
            caught += 1
    assert caught > 0, name
