"""Plain Python oracle of the candidate buffer, the read cursor and candidate
alignment.

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

What it follows (paper: AS2D, arXiv 2609.37617):
  * Ordered publication (Section 4.1, "Ordered publication and buffering";
    Appendix C.1): the producer appends immutable batches of up to eight
    tokens, each with its source ID, producer ID, token offset, publication
    time and confidence; the buffer exposes only published tokens, in
    order, and a verification reads a snapshot (the published length at
    that moment) while later batches are appended.
  * A read cursor that moves independently of publication; verification
    takes the ready candidates from the cursor (Section 4.1; Figure 4(a)),
    at most the budget b, at most what the remaining reply allows, and a
    K1 step (no candidates) when none is ready (Appendix C.2).
  * Candidate alignment (Section 4.2, "Candidate alignment"; Appendix C.3;
    Figure 4(c)): full acceptance advances the cursor; after a rejection
    the cursor is realigned by a bounded local search for the target's
    token; unmatched positions are retired.  Alignment never changes the
    buffer, and every reused candidate is verified again.

The alignment rule, as read here (the paper states it in words only).
The runtime carries the target's correction (or bonus) token y into the
next call as its root, so the target token that follows y is known only
after that call.  After a call that proposed buffer positions
[c, c + k) and committed a of them plus y, with m = c + a the position y
stands for:
  1. positions c .. m-1 were accepted: the floor f (lowest eligible
     position) becomes m;
  2. if the buffer holds y at m (full acceptance whose bonus equals the
     next published candidate), that candidate is consumed: c = f = m + 1;
  3. else search for y at distance d = 1 .. R from m, forward (m + d, a
     published position) before backward (m - d, not below f); a match at
     j consumes it: c = f = j + 1 (positions before j are retired).  A
     forward match is a target deletion of draft tokens; a backward match
     recovers a target insertion (the candidate the target had not yet
     reached stays eligible, as the paper requires);
  4. else the substitution reading: c = m + 1 with f unchanged, so
     position m stays eligible for a later backward match.
R = 8, one publication batch.  Whatever the rule picks, verification
decides what is committed, so the output is the target-only output for
any buffer content (Appendix C.4, Proposition); the rule only changes how
many tokens each call commits.
"""
import math

BATCH = 8          # tokens per publication batch (Appendix C.1)
RADIUS = 8         # bounded local search radius, in buffer positions


class CandidateBuffer:
    """Ordered, append-only buffer of published candidate tokens."""

    def __init__(self):
        self.tokens = []
        self.records = []      # (first position, count, source, producer, offset, time, confidence)

    def publish(self, tokens, source_id=0, producer_id=0, offset=None, publish_time=0, confidence=math.nan):
        """Append one immutable batch (1..BATCH tokens); returns the new
        published length."""
        tokens = [int(t) for t in tokens]
        if not 1 <= len(tokens) <= BATCH:
            raise ValueError("a batch holds 1..8 tokens")
        if offset is None:
            offset = len(self.tokens)
        self.records.append((len(self.tokens), len(tokens), int(source_id), int(producer_id), int(offset),
                             int(publish_time), float(confidence)))
        self.tokens.extend(tokens)
        return len(self.tokens)

    def snapshot(self):
        """The published length: the tokens a verification may read."""
        return len(self.tokens)


class ReadCursor:
    """Read cursor c and floor f over a CandidateBuffer."""

    def __init__(self, radius=RADIUS):
        self.c = 0
        self.f = 0
        self.radius = radius

    def propose(self, tokens, n, k_max):
        """Ready candidates at the cursor: at most k_max of the first n
        (snapshot) tokens."""
        if k_max <= 0 or self.c >= n:
            return []
        return list(tokens[self.c:min(n, self.c + k_max)])

    def update(self, tokens, n, k, a, y):
        """Realign after a call that proposed k candidates from the cursor,
        accepted a of them and committed the target token y (steps 1-4 of
        the module docstring).  `tokens[:n]` is the snapshot the next
        proposal will read."""
        if not 0 <= a <= k:
            raise ValueError("accepted length outside [0, k]")
        m = self.c + a
        if a > 0:
            self.f = m
        if m < n and tokens[m] == y:
            self.c = self.f = m + 1
            return
        for d in range(1, self.radius + 1):
            j = m + d
            if j < n and tokens[j] == y:
                self.c = self.f = j + 1
                return
            j = m - d
            if j >= self.f and j < n and tokens[j] == y:
                self.c = self.f = j + 1
                return
        self.c = m + 1


def decode_with_buffer(model, publish_schedule, budget, reply_len, radius=RADIUS, cursor=None):
    """Greedy decoding of `reply_len` tokens after a prefilled model state,
    proposing candidates from a CandidateBuffer through a ReadCursor.

    model: an OracleModel (or anything with .root and .verify(cands, k)).
    publish_schedule(step, buffer): called before each verification call;
    publishes whatever batches are ready at that step.
    cursor: the ReadCursor to use (default: a fresh one of `radius`), so a
    schedule can look at it.
    Returns (committed tokens, per-call (k, a) list).  The first committed
    token of each call is the previous root's successor, so the returned
    stream starts after the root that was current on entry."""
    buf = CandidateBuffer()
    cur = ReadCursor(radius) if cursor is None else cursor
    out, calls = [], []
    step = 0
    while len(out) < reply_len:
        publish_schedule(step, buf)
        n = buf.snapshot()
        k_max = min(budget, reply_len - len(out) - 1)
        cands = cur.propose(buf.tokens, n, k_max)
        r = model.verify(cands, len(cands))
        a, y = r["accepted_len"], r["correction_token"]
        out.extend(list(cands[:a]) + [y])
        calls.append((len(cands), a))
        cur.update(buf.tokens, buf.snapshot(), len(cands), a, y)
        step += 1
    return out[:reply_len], calls
