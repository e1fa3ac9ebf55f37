"""Verification cost profile R(K) and the offline budget choice: the oracle
against closed forms and limiting cases, the library's replay (its own
cursor) against the oracle's.  No GPU."""
import random

import pytest

from oracle import budget as ob
from workload import gen


def test_cost_reduction_closed_forms():
    flat = {K: 2.0 for K in range(1, 17)}               # a call costs the same at any width
    assert ob.cost_reduction(flat) == pytest.approx({K: 100.0 * (1 - 1 / K) for K in range(1, 17)})
    linear = {K: 2.0 * K for K in range(1, 17)}         # no batching benefit
    assert ob.cost_reduction(linear) == pytest.approx({K: 0.0 for K in range(1, 17)})
    assert ob.cost_reduction({1: 3.0, 4: 6.0})[4] == pytest.approx(50.0)


def test_replay_counts_every_token_once():
    rng = random.Random(1)
    for _ in range(100):
        target = [rng.randrange(5) for _ in range(rng.randrange(3, 60))]
        n = len(target) - 1
        draft = gen.edited_stream(target, 5, 0.2, 0.1, 0.1, seed=rng.randrange(1000))
        calls = ob.replay_calls(draft, target, rng.randrange(0, 10), n)
        assert sum(a + 1 for _, a in calls) == n
        assert all(0 <= a <= k for k, a in calls)


def test_budget_choice_limits():
    target = list(range(1, 200))
    exact = [(target, target, 160)]                    # the draft is the target's own text
    flat = {K: 1.0 for K in range(1, 17)}
    b, thr = ob.select_budget(flat, exact, range(0, 16))
    assert b == 15                                     # free width and perfect drafts: the widest
    assert thr[15] == pytest.approx(160 / 10) and thr[14] == pytest.approx(160 / 11)
    linear = {K: float(K) for K in range(1, 17)}
    b, thr = ob.select_budget(linear, exact, range(0, 16))
    assert b == 0 and all(v == pytest.approx(1.0) for v in thr.values())   # every budget ties at 1
    noise = [([999] * 300, target, 160)]                # never accepted
    b, _ = ob.select_budget(flat, noise, range(0, 16))
    assert b == 0


@pytest.fixture(scope="module")
def budget_mod():
    from tests.harness import ensure_built
    ensure_built()
    from paper_2609_37617_amd import budget
    return budget


def test_library_replay_matches_oracle(budget_mod):
    rng = random.Random(7)
    for trial in range(200):
        alpha = rng.choice([4, 30])
        target = [rng.randrange(alpha) for _ in range(rng.randrange(3, 80))]
        n = len(target) - 1
        draft = gen.edited_stream(target, alpha, rng.random() * 0.4, rng.random() * 0.2, rng.random() * 0.2, seed=trial)
        b = rng.randrange(0, 16)
        assert budget_mod.replay_calls(draft, target, b, n) == ob.replay_calls(draft, target, b, n), trial
    vbar = {K: 3.0 + 0.05 * K * K for K in range(1, 17)}
    traces = [(gen.edited_stream(list(range(300)), 300, 0.2, 0.05, 0.05, seed=s), list(range(300)), 250) for s in range(3)]
    assert budget_mod.select_budget(vbar, traces, range(0, 16))[0] == ob.select_budget(vbar, traces, range(0, 16))[0]
    assert budget_mod.cost_reduction(vbar) == pytest.approx(ob.cost_reduction(vbar))
