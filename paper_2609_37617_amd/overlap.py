"""Time accounting of a decoding run (Appendix D.2, "Overlap, added work,
and performance limits").

With P and V the unions of the producer's and the verifier's service
intervals within [0, T]:
    D = |P|,  V = |V|,  O = |P n V|,  H = |[0, T] \\ (P u V)|,
and T = D + V - O + H (inclusion-exclusion).  Between a serial run s
(O_s = 0) and an asynchronous run a committing the same tokens,
T_s - T_a = O_a - dD - dV - dH, so a strict gain happens exactly when
O_a > dD + dV + dH; and T_a >= max(D_a, V_a) + H_a bounds the speedup.
Per-round progress: V / N = v / m with the round means v = V / R and
m = N / R.
"""
from typing import Dict, List, Sequence, Tuple


def merge(iv: Sequence[Tuple[int, int]]) -> List[Tuple[int, int]]:
    """Union of closed intervals as sorted disjoint intervals."""
    out = []
    for s, e in sorted(iv):
        if out and s <= out[-1][1]:
            out[-1] = (out[-1][0], max(out[-1][1], e))
        else:
            out.append((s, e))
    return out


def length(u: Sequence[Tuple[int, int]]) -> int:
    return sum(e - s for s, e in u)


def intersect(a: Sequence[Tuple[int, int]], b: Sequence[Tuple[int, int]]) -> List[Tuple[int, int]]:
    """Intersection of two sorted disjoint interval lists."""
    out, i, j = [], 0, 0
    while i < len(a) and j < len(b):
        s, e = max(a[i][0], b[j][0]), min(a[i][1], b[j][1])
        if s < e:
            out.append((s, e))
        if a[i][1] < b[j][1]:
            i += 1
        else:
            j += 1
    return out


def accounting(intervals: Sequence[Tuple[int, int, int, int]], total: int) -> Dict[str, float]:
    """D, V, O, H, T (same unit as the intervals), rounds R and tokens N of
    one run from its stage log (kind 0 producer, 1 verifier)."""
    P = merge([(s, e) for s, e, k, _ in intervals if k == 0])
    Vu = merge([(s, e) for s, e, k, _ in intervals if k == 1])
    D, V = length(P), length(Vu)
    O = length(intersect(P, Vu))
    H = total - length(merge(P + Vu))
    R = sum(1 for *_, k, _ in intervals if k == 1)
    N = sum(t for *_, k, t in intervals if k == 1)
    return dict(T=total, D=D, V=V, O=O, H=H, R=R, N=N)


def compare(serial: Dict[str, float], asyn: Dict[str, float]) -> Dict[str, float]:
    """The speedup and the terms of the break-even condition and bound."""
    dD, dV, dH = asyn["D"] - serial["D"], asyn["V"] - serial["V"], asyn["H"] - serial["H"]
    return dict(speedup=serial["T"] / asyn["T"], saving=serial["T"] - asyn["T"], O_a=asyn["O"],
                added=dD + dV + dH, dD=dD, dV=dV, dH=dH,
                break_even_holds=(asyn["O"] > dD + dV + dH) == (asyn["T"] < serial["T"]),
                bound=serial["T"] / (max(asyn["D"], asyn["V"]) + asyn["H"]))
