"""Pins the oracle's discovery procedure (Sec. 4, procedure FINGERPRINT),
the Philox4x32-10 generator of its mock world model, and the model itself.

The procedure is checked on synthetic probes whose distance is a closed-form
function of the snapshot mask, so every branch (necessity, sufficiency,
ties, a multi-step greedy fallback, no convergence, a failed control) has a
hand-derived answer.  Philox is checked against its published known-answer
values.  The mock model is checked for the properties it is built to have,
and its two implementations (the oracle's numpy one, and the torch one the
GPU side runs, here on the CPU device) are checked against each other.
"""
import os

import numpy as np
import pytest

import oracle
from oracle import discover as D
from oracle.mock_world import MockWorld, T, T_inv, rotl
from workloads.mock_world import MockSpec, fresh_state, initial_state, trajectory

KAT = os.path.join(os.path.dirname(__file__), "golden", "philox4x32_10_kat.txt")


def test_philox_known_answers():
    n = 0
    for line in open(KAT):
        line = line.split("#")[0].strip()
        if not line:
            continue
        ctr, key, out = [[int(w, 16) for w in part.split()] for part in line.split("|")]
        assert oracle.philox4x32_10(ctr, key).tolist() == out
        n += 1
    assert n == 3


def table_probe(fn):
    """A synthetic probe: D is fn(mask), the control corrupts nothing the
    probe reads unless fn says so."""
    def probe(mask, corrupt=-1):
        return fn(mask, corrupt)
    return probe


def test_procedure_necessity_and_sufficiency():
    # D = 0.5 if component 0 is missing, + 0.3 if component 2 is missing.
    f = lambda m, c: 0.5 * (1 - m[0]) + 0.3 * (1 - m[2]) + (0.25 if c == 0 else 0.0)
    r = D.discover(table_probe(f), 4, 0.0, control=0)
    assert r["necessary"] == [1, 0, 1, 0] and r["pcs"] == [1, 0, 1, 0] and r["added"] == []
    assert r["d_without"] == [0.5, 0.0, 0.3, 0.0] and r["d_necessary"] == 0.0 and r["converged"] == 1
    assert r["probes"] == 4 + 1 + 1 and r["d_control"] == 0.25 and r["control_ok"] == 1


def test_procedure_redundant_pair_tie_goes_to_lowest_index():
    # Components 3 and 4 each stand in for the other; 0 is necessary.
    f = lambda m, c: 0.6 * (1 - m[0]) + 0.2 * (1 - max(m[3], m[4]))
    r = D.discover(table_probe(f), 5, 0.0)
    assert r["necessary"] == [1, 0, 0, 0, 0] and r["d_necessary"] == 0.2
    assert r["added"] == [3] and r["pcs"] == [1, 0, 0, 1, 0] and r["d_final"] == 0.0
    assert r["probes"] == 5 + 1 + 4 and r["control_ok"] == -1 and r["d_control"] == -1.0


def test_procedure_multi_step_greedy():
    # Any two of {1, 2, 3} suffice; one of them halves the distance.
    def f(m, c):
        have = m[1] + m[2] + m[3]
        return 0.0 if have >= 2 else (0.5 if have == 1 else 1.0)
    r = D.discover(table_probe(f), 4, 0.0)
    assert r["necessary"] == [0, 0, 0, 0] and r["d_necessary"] == 1.0
    assert r["added"] == [1, 2] and r["pcs"] == [0, 1, 1, 0] and r["d_final"] == 0.0
    assert r["probes"] == 4 + 1 + 4 + 3


def test_procedure_tolerance_and_no_convergence():
    f = lambda m, c: 0.01 * (4 - sum(m)) + 0.5   # never below 0.5: the probe is not reproducible
    r = D.discover(table_probe(f), 4, 0.1, control=2)
    assert r["necessary"] == [1, 1, 1, 1] and r["converged"] == 0 and r["d_final"] == 0.5
    assert r["control_ok"] == 1
    g = lambda m, c: 0.05 * (1 - m[1])           # within tolerance: nothing is necessary
    r = D.discover(table_probe(g), 3, 0.1, control=1)
    assert r["necessary"] == [0, 0, 0] and r["pcs"] == [0, 0, 0] and r["converged"] == 1
    assert r["control_ok"] == 0                   # the control catches a probe that ignores the state
    r = D.discover(table_probe(lambda m, c: 0.0), 0, 0.0)
    assert r["pcs"] == [] and r["probes"] == 1 and r["converged"] == 1


def test_mock_model_pieces():
    x = (np.arange(1000, dtype=np.uint64) * 0x9E3779B97F4A7C15) & 0xFFFFFFFF
    assert np.array_equal(T_inv(T(x)), x)
    assert int(rotl(0x80000001, 1)) == 3 and int(rotl(7, 32)) == 7
    spec = MockSpec(height=16, width=16, bank_cap=8, entry_words=16, kv_words=32)
    a = MockWorld(spec, initial_state(spec, 2))
    b = MockWorld(spec, initial_state(spec, 2))
    wa, pa = trajectory(2, 5, 3)
    assert np.array_equal(a.run(wa), b.run(wa))                     # deterministic
    parts = a.parts()
    # Either half of the context pair rebuilds the other: a session missing one
    # half continues exactly like the full one.
    for drop in (6, 7):
        p2 = [x.copy() for x in parts]
        p2[drop][:] = 0
        assert np.array_equal(MockWorld(spec, p2).run(pa), MockWorld(spec, parts).run(pa))
    p3 = [x.copy() for x in parts]
    p3[6][:] = 0
    p3[7][:] = 0
    assert not np.array_equal(MockWorld(spec, p3).run(pa), MockWorld(spec, parts).run(pa))
    # Derivable components: overwriting them changes nothing.
    p4 = [x.copy() for x in parts]
    p4[4][:] = 0x5A
    p4[5][:] = 0xC3
    assert np.array_equal(MockWorld(spec, p4).run(pa), MockWorld(spec, parts).run(pa))
    assert len(fresh_state(spec)) == 8


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_procedure_on_the_mock_model(seed):
    spec = MockSpec()
    w = MockWorld(spec, initial_state(spec, seed))
    wa, pa = trajectory(seed, 24, 8)
    w.run(wa)
    anchor = w.parts()
    ref_h = oracle.fingerprint([MockWorld(spec, anchor).run(pa)])[0]
    r = D.discover(D.mock_probe(spec, anchor, pa, ref_h), 8, 0.0, control=1)
    # obs, rng, bank, pose necessary; feat, scratch derivable; kv_a (the lower
    # index of the interchangeable pair) added by the fallback.
    assert r["necessary"] == [1, 1, 1, 1, 0, 0, 0, 0]
    assert r["pcs"] == [1, 1, 1, 1, 0, 0, 1, 0] and r["added"] == [6]
    assert r["d_necessary"] > 0 and r["d_final"] == 0 and r["control_ok"] == 1 and r["probes"] == 14


def test_torch_model_matches_oracle_model_on_cpu():
    torch = pytest.importorskip("torch")
    from workloads.mock_world_gpu import MockWorldGPU
    spec = MockSpec(height=32, width=32, bank_cap=16, entry_words=64, kv_words=128)
    init = initial_state(spec, 5)
    wa, pa = trajectory(5, 12, 4)
    o = MockWorld(spec, init)
    g = MockWorldGPU.from_host(spec, init, device="cpu")
    assert np.array_equal(np.concatenate([o.run(wa), o.run(pa)]), torch.cat([g.run(wa), g.run(pa)]).numpy())
    assert all(np.array_equal(a, b.numpy()) for a, b in zip(o.parts(), g.parts))
