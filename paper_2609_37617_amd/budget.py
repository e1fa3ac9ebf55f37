"""Device cost profile and offline budget selection (host side).

Verification width profile (Section 4.3, "Device cost profiling"; Appendix
B.2, Eq. R(K)): V(K) is the mean time of a verification call of physical
width K (the root plus K - 1 candidates, all of them the target's own
continuation), and

    R(K) = 100 (1 - V(K) / (K V(1)))  percent

is the saving per verified position against K single-position calls.

Offline budget selection (Section 4.3, "Offline budget selection";
Appendix D.2, "Fixed configurations and development splits"): a fixed
proposal budget b (at most b candidates per call, physical width at most
b + 1) is chosen before deployment by comparing pooled throughput on
development traces.  Here a trace is a draft and the target stream it is
verified against; the decoding loop (proposals from the read cursor,
greedy verification, alignment) is replayed exactly with the library's
own cursor, and its calls are priced with the measured V(K), so the
estimate needs no GPU once V is known.
"""
from typing import Dict, List, Sequence, Tuple

from . import as2d


def cost_reduction(vbar: Dict[int, float]) -> Dict[int, float]:
    """R(K) in percent for every measured width K (vbar must hold K = 1)."""
    v1 = vbar[1]
    return {K: 100.0 * (1.0 - v / (K * v1)) for K, v in sorted(vbar.items())}


def replay_calls(draft: Sequence[int], target: Sequence[int], budget: int, n_tokens: int,
                 radius: int = 8) -> List[Tuple[int, int]]:
    """(k, accepted) of every call when `n_tokens` tokens after the root are
    decoded from `draft` (all of it published before the first call) by a
    target whose greedy continuation is `target`."""
    if len(target) < n_tokens + 1:
        raise ValueError("the target stream must cover n_tokens + 1 tokens")
    buf = as2d.CandidateBuffer(max(len(draft), 1))
    for i in range(0, len(draft), 8):
        buf.publish(draft[i:i + 8])
    cur = as2d.ReadCursor(radius)
    n = buf.snapshot()
    pos, calls = 0, []
    while pos < n_tokens:
        cands = cur.propose(buf, n, min(budget, n_tokens - pos - 1))
        a = 0
        while a < len(cands) and cands[a] == target[pos + a]:
            a += 1
        calls.append((len(cands), a))
        cur.update(buf, n, len(cands), a, int(target[pos + a]))
        pos += a + 1
    buf.close()
    return calls


def estimated_time(calls: Sequence[Tuple[int, int]], vbar: Dict[int, float]) -> float:
    """Sum of V(k + 1) over the calls."""
    return sum(vbar[k + 1] for k, _ in calls)


def select_budget(vbar: Dict[int, float], traces: Sequence[Tuple[Sequence[int], Sequence[int], int]],
                  budgets: Sequence[int], radius: int = 8) -> Tuple[int, Dict[int, float]]:
    """The budget with the highest pooled estimated throughput (tokens per
    unit of V) over the traces (draft, target stream, tokens); budgets whose
    width has no measured cost are skipped.  Returns (budget, throughput by
    budget); ties go to the smaller budget."""
    thr = {}
    for b in budgets:
        if b + 1 not in vbar:
            continue
        tokens = sum(n for _, _, n in traces)
        t = sum(estimated_time(replay_calls(d, y, b, n, radius), vbar) for d, y, n in traces)
        thr[b] = tokens / t
    best = max(sorted(thr), key=lambda b: thr[b])
    return best, thr
