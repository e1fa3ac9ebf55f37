"""Plain Python oracle of the run time accounting.

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

Appendix D.2, "Overlap, added work, and performance limits": D, V, O and H
are measures of the producer's and verifier's service sets and of the
remainder of [0, T] (Eq. performance-intervals), written here as a count
of the integer time points each set covers (intervals [s, e) on an
integer clock), which is the definition for integer end points.
"""


def covered(intervals):
    pts = set()
    for s, e in intervals:
        pts.update(range(s, e))
    return pts


def accounting(intervals, total):
    P = covered([(s, e) for s, e, k, _ in intervals if k == 0])
    V = covered([(s, e) for s, e, k, _ in intervals if k == 1])
    T = set(range(total))
    return dict(T=total, D=len(P), V=len(V), O=len(P & V), H=len(T - (P | V)),
                R=sum(1 for *_, k, _ in intervals if k == 1), N=sum(t for *_, k, t in intervals if k == 1))
