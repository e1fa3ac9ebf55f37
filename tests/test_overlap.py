"""Run time accounting (D, V, O, H): the library's interval arithmetic
against the oracle's point-counting definition, the accounting identity,
the overlap bounds and the break-even equivalence.  No GPU."""
import random

from oracle import overlap as oo
from paper_2609_37617_amd import overlap as po


def random_log(rng, total, serial=False):
    log, t = [], 0
    if serial:
        while t < total - 2:
            s = t + rng.randrange(0, 3)
            e = min(total, s + rng.randrange(1, 9))
            log.append((s, e, rng.randrange(2), rng.randrange(1, 5)))
            t = e
        return log
    for _ in range(rng.randrange(0, 40)):
        s = rng.randrange(0, total)
        e = min(total, s + rng.randrange(0, 15))
        log.append((s, e, rng.randrange(2), rng.randrange(1, 5)))
    return log


def test_accounting_matches_point_count():
    rng = random.Random(2)
    for trial in range(400):
        total = rng.randrange(1, 120)
        log = random_log(rng, total, serial=trial % 4 == 0)
        a, o = po.accounting(log, total), oo.accounting(log, total)
        assert a == o, (trial, log)
        assert a["T"] == a["D"] + a["V"] - a["O"] + a["H"]
        assert 0 <= a["O"] <= min(a["D"], a["V"])
        if trial % 4 == 0:
            assert a["O"] == 0                          # stages that never run at once


def test_break_even_equivalence_and_bound():
    rng = random.Random(4)
    for _ in range(300):
        ts, ta = rng.randrange(20, 120), rng.randrange(20, 120)
        s = po.accounting(random_log(rng, ts, serial=True), ts)
        a = po.accounting(random_log(rng, ta), ta)
        c = po.compare(s, a)
        assert s["O"] == 0
        assert c["saving"] == c["O_a"] - c["added"]         # T_s - T_a = O_a - dD - dV - dH
        assert c["break_even_holds"]
        assert c["speedup"] <= c["bound"] + 1e-12
