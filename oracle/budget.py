"""Plain Python oracle of the verification cost profile and the offline
budget choice.

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

  * R(K) = 100 (1 - V(K) / (K V(1))) percent: the per-position saving of a
    width-K verification call against K width-1 calls (Appendix B.2,
    Eq. R(K)).
  * A fixed budget is chosen offline by pooled throughput over development
    traces (Section 4.3, "Offline budget selection"; Appendix D.2); a trace
    is replayed through the decoding loop (oracle.align.ReadCursor, greedy
    verification against the trace's target stream) and each call of k
    candidates is priced at V(k + 1).
"""
from .align import CandidateBuffer, ReadCursor
from .model import verify_block


def cost_reduction(vbar):
    return {K: 100.0 * (1.0 - vbar[K] / (K * vbar[1])) for K in sorted(vbar)}


def replay_calls(draft, target, budget, n_tokens, radius=8):
    buf = CandidateBuffer()
    for i in range(0, len(draft), 8):
        buf.publish(draft[i:i + 8])
    cur = ReadCursor(radius)
    n = buf.snapshot()
    pos, calls = 0, []
    while pos < n_tokens:
        cands = cur.propose(buf.tokens, n, min(budget, n_tokens - pos - 1))
        k = len(cands)
        a, y = verify_block(list(target[pos:pos + k + 1]), cands, k)
        calls.append((k, a))
        cur.update(buf.tokens, n, k, a, y)
        pos += a + 1
    return calls


def pooled_throughput(vbar, traces, budget, radius=8):
    tokens = sum(n for _, _, n in traces)
    time = sum(sum(vbar[k + 1] for k, _ in replay_calls(d, y, budget, n, radius)) for d, y, n in traces)
    return tokens / time


def select_budget(vbar, traces, budgets, radius=8):
    thr = {b: pooled_throughput(vbar, traces, b, radius) for b in budgets if b + 1 in vbar}
    best = None
    for b in sorted(thr):
        if best is None or thr[b] > thr[best]:
            best = b
    return best, thr
