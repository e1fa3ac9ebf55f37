"""Candidate buffer, read cursor and alignment: the oracle against the
paper's Figure 4 example and the alignment cases its text names, the
library's C++ implementation against the oracle (bit-exact), and the
buffer's publication semantics.  No GPU."""
import json
import os
import random
import threading

import numpy as np
import pytest

from oracle import CandidateBuffer, ReadCursor, decode_with_buffer, verify_block
from oracle.align import RADIUS
from workload import TINY, gen

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


class ScriptedTarget:
    """Greedy verification (oracle.verify_block) against a target whose
    greedy continuation is a fixed token stream."""

    def __init__(self, stream):
        self.y = list(stream)
        self.pos = 0

    def verify(self, cands, k):
        t = [self.y[self.pos + i] for i in range(k + 1)]
        a, corr = verify_block(t, cands, k)
        self.pos += a + 1
        return dict(accepted_len=a, correction_token=corr)


def run_oracle(draft, target, budget, batches_per_step=None, radius=RADIUS, steps=None):
    """Decode len(target) - 1 tokens with the oracle aligner; returns the
    committed stream and the per-call proposals."""
    buf, cur = CandidateBuffer(), ReadCursor(radius)
    tgt = ScriptedTarget(target)
    pub = [draft[i:i + 8] for i in range(0, len(draft), 8)]
    out, props = [], []
    step = 0
    while len(out) < len(target) - 1:
        n_ready = len(pub) if batches_per_step is None else min(len(pub), 1 + step * batches_per_step)
        while len(buf.records) < n_ready:
            buf.publish(pub[len(buf.records)])
        n = buf.snapshot()
        cands = cur.propose(buf.tokens, n, min(budget, len(target) - 1 - len(out) - 1))
        r = tgt.verify(cands, len(cands))
        out += cands[:r["accepted_len"]] + [r["correction_token"]]
        props.append((list(cands), r["accepted_len"], cur.c, cur.f))
        cur.update(buf.tokens, buf.snapshot(), len(cands), r["accepted_len"], r["correction_token"])
        props[-1] = props[-1] + (cur.c, cur.f)
        step += 1
    return out, props


# -- oracle pins -----------------------------------------------------------------

def test_figure4_alignment():
    """Figure 4: A B C D published, A B accepted, X committed; D E F are
    verified next and the committed text is the target's."""
    fx = json.load(open(os.path.join(ROOT, "tests", "golden", "fig4_alignment.json")))
    sym = fx["symbols"]
    enc = lambda xs: [sym[x] for x in xs]
    buf, cur = CandidateBuffer(), ReadCursor()
    tgt = ScriptedTarget(enc(fx["target_stream"]))
    buf.publish(enc(fx["published_first"]))
    c1 = cur.propose(buf.tokens, buf.snapshot(), 4)
    assert c1 == enc(fx["first_call"]["candidates"])
    r1 = tgt.verify(c1, len(c1))
    assert r1["accepted_len"] == fx["first_call"]["accepted"]
    committed = c1[:r1["accepted_len"]] + [r1["correction_token"]]
    assert committed == enc(fx["first_call"]["committed"])
    buf.publish(enc(fx["published_after_first_call"]))
    cur.update(buf.tokens, buf.snapshot(), len(c1), r1["accepted_len"], r1["correction_token"])
    c2 = cur.propose(buf.tokens, buf.snapshot(), 4)
    assert c2 == enc(fx["second_call_verifies"])
    r2 = tgt.verify(c2, len(c2))
    committed += c2[:r2["accepted_len"]] + [r2["correction_token"]]
    assert committed == enc(fx["committed_after_two_calls"])
    assert buf.tokens == enc(fx["published_first"] + fx["published_after_first_call"])   # never changed


def test_full_acceptance_advances_the_cursor():
    """Full acceptance advances the cursor; a bonus equal to the next
    candidate consumes it."""
    buf, cur = CandidateBuffer(), ReadCursor()
    buf.publish([1, 2, 3, 4, 5])
    assert cur.propose(buf.tokens, 5, 2) == [1, 2]
    cur.update(buf.tokens, 5, 2, 2, 3)
    assert (cur.c, cur.f) == (3, 3)
    assert cur.propose(buf.tokens, 5, 8) == [4, 5]


def test_insertion_keeps_the_mismatch_position_eligible():
    """The target inserts Y before C: the candidate at the mismatch position
    stays usable and the suffix after it is not discarded."""
    draft = [1, 2, 3, 4, 5, 6, 7, 8]
    target = [1, 2, 9, 3, 4, 5, 6, 7, 8, 10, 11, 12]
    out, props = run_oracle(draft, target, budget=4)
    assert out == target[:-1]
    # call 1: A B accepted, Y committed; call 2 (root Y) proposes D.. and the
    # target's C is found one position back; call 3 proposes D.. again
    assert [p[0] for p in props][:3] == [[1, 2, 3, 4], [4, 5, 6, 7], [4, 5, 6, 7]]
    assert props[1][1] == 0 and props[2][1] == 4


def test_deletion_skips_draft_tokens():
    """The target leaves out C: D is found one position ahead."""
    out, props = run_oracle([1, 2, 3, 4, 5, 6], [1, 2, 4, 5, 6, 7], budget=4)
    assert out == [1, 2, 4, 5, 6]
    assert props[0][0] == [1, 2, 3, 4] and props[0][1] == 2
    assert props[0][4:] == (4, 4)            # cursor and floor after the match at position 3


def test_substitution_keeps_the_suffix():
    target = [1, 2, 9, 4, 5, 6, 7, 8, 10, 11]
    out, props = run_oracle([1, 2, 3, 4, 5, 6, 7, 8], target, budget=4)
    assert out == target[:-1]
    assert props[1][0] == [4, 5, 6, 7] and props[1][1] == 4


def test_search_is_bounded_and_respects_the_floor():
    buf, cur = CandidateBuffer(), ReadCursor(radius=2)
    toks = [1, 2, 3, 4, 5, 6, 7, 8]
    buf.publish(toks)
    cur.update(buf.tokens, 8, 4, 1, 6)     # m = 1: 6 sits at distance 4 > radius
    assert (cur.c, cur.f) == (2, 1)
    cur2 = ReadCursor(radius=8)
    cur2.c, cur2.f = 4, 4
    cur2.update(buf.tokens, 8, 2, 0, 2)     # 2 sits at position 1, below the floor
    assert (cur2.c, cur2.f) == (5, 4)


def test_nearest_match_forward_first():
    """Equal distances: the forward match (a deletion) is taken before the
    backward one; a nearer match wins over a farther one."""
    toks = [5, 9, 3, 9, 5, 5, 9]
    cur = ReadCursor(8)
    cur.c, cur.f = 2, 0
    cur.update(toks, 7, 3, 0, 9)             # m = 2: 9 at 3 (d = 1 forward) and at 1 (d = 1 backward)
    assert (cur.c, cur.f) == (4, 4)
    cur = ReadCursor(8)
    cur.c, cur.f = 2, 0
    cur.update(toks, 7, 3, 0, 5)             # m = 2: 5 at 0 (d = 2 backward) before 4 (d = 2 forward)? forward first
    assert (cur.c, cur.f) == (5, 5)
    cur = ReadCursor(8)
    cur.c, cur.f = 3, 0
    cur.update(toks, 7, 3, 0, 3)             # m = 3: 3 at 2 (d = 1 backward), nearer than anything forward
    assert (cur.c, cur.f) == (3, 3)


def test_nothing_ready_is_a_target_only_step():
    out, props = run_oracle([], [5, 6, 7, 8], budget=4)
    assert out == [5, 6, 7]
    assert all(p[0] == [] for p in props)


def test_any_buffer_gives_the_target_stream():
    """Appendix C.4, Proposition, with the loop around the aligner: random
    drafts (edits of the target text, or noise) never change the output."""
    rng = random.Random(5)
    for trial in range(200):
        target = [rng.randrange(6) for _ in range(rng.randrange(2, 40))]
        kind = trial % 3
        if kind == 0:
            draft = [rng.randrange(6) for _ in range(rng.randrange(0, 50))]
        else:
            draft = gen.edited_stream(target, 6, 0.2, 0.15, 0.15, seed=trial)
        out, _ = run_oracle(draft, target, budget=rng.randrange(0, 9), batches_per_step=rng.choice([None, 1, 2]),
                            radius=rng.randrange(0, 9))
        assert out == target[:len(target) - 1]


def test_oracle_model_loop_matches_target_only():
    """The same with the float64 model: decode_with_buffer over an edited
    draft commits the target-only stream."""
    from oracle import OracleModel
    w = gen.weights_dict(TINY, gen.make_weights(TINY, 0))
    om = OracleModel(TINY, w, capacity=128)
    audio = gen.audio_embeddings(TINY, 16, 0, fmt="oracle")
    instr = gen.instruction_tokens(TINY, 4, 0)
    f, L = om.prefill(audio, instr)
    ref = om.target_only(24)
    om.rollback(L, f)
    draft = gen.edited_stream(ref[1:], TINY.vocab, 0.15, 0.1, 0.1, seed=3)
    sched = lambda step, buf: [buf.publish(draft[i:i + 8]) for i in range(8 * len(buf.records), min(len(draft), 8 * (step + 1)), 8)]
    out, calls = decode_with_buffer(om, sched, budget=4, reply_len=24)
    assert out == ref[1:25]
    assert sum(a for _, a in calls) > 0


# -- the library's implementation against the oracle ----------------------------

@pytest.fixture(scope="module")
def lib():
    from tests.harness import ensure_built
    ensure_built()
    from paper_2609_37617_amd import as2d
    as2d.load_library()
    return as2d


def test_library_alignment_matches_oracle(lib):
    rng = random.Random(11)
    for trial in range(300):
        alpha = rng.choice([3, 6, 50])
        target = [rng.randrange(alpha) for _ in range(rng.randrange(2, 60))]
        draft = (gen.edited_stream(target, alpha, rng.random() * 0.4, rng.random() * 0.3, rng.random() * 0.3, seed=trial)
                 if trial % 4 else [rng.randrange(alpha) for _ in range(rng.randrange(0, 70))])
        budget = rng.randrange(0, 12)
        radius = rng.randrange(0, 12)
        per_step = rng.choice([None, 1, 2])
        _, props = run_oracle(draft, target, budget, per_step, radius)
        # the library, driven by the same scripted target and schedule
        buf = lib.CandidateBuffer(max(len(draft), 1))
        cur = lib.ReadCursor(radius)
        tgt = ScriptedTarget(target)
        pub = [draft[i:i + 8] for i in range(0, len(draft), 8)]
        n_pub = 0
        out = []
        for step, (o_cands, o_a, o_c, o_f, o_c2, o_f2) in enumerate(props):
            n_ready = len(pub) if per_step is None else min(len(pub), 1 + step * per_step)
            while n_pub < n_ready:
                buf.publish(pub[n_pub])
                n_pub += 1
            assert (cur.cursor, cur.floor) == (o_c, o_f)
            n = buf.snapshot()
            cands = cur.propose(buf, n, min(budget, len(target) - 1 - len(out) - 1))
            assert cands == o_cands, (trial, step)
            r = tgt.verify(cands, len(cands))
            assert r["accepted_len"] == o_a
            out += cands[:r["accepted_len"]] + [r["correction_token"]]
            cur.update(buf, buf.snapshot(), len(cands), r["accepted_len"], r["correction_token"])
            assert (cur.cursor, cur.floor) == (o_c2, o_f2), (trial, step)
        buf.close()


def test_library_update_matches_oracle_on_random_states(lib):
    """Single updates from arbitrary (cursor, floor) states with repeated tokens."""
    rng = random.Random(3)
    toks = [rng.randrange(4) for _ in range(64)]
    buf = lib.CandidateBuffer(64)
    for i in range(0, 64, 8):
        buf.publish(toks[i:i + 8])
    for _ in range(3000):
        f = rng.randrange(0, 60)
        c = rng.randrange(f, 62)
        k = rng.randrange(0, 9)
        a = rng.randrange(0, k + 1)
        y = rng.randrange(5)
        n = rng.randrange(c, 65)
        radius = rng.randrange(0, 10)
        o = ReadCursor(radius)
        o.c, o.f = c, f
        o.update(toks, n, k, a, y)
        cur = lib.ReadCursor(radius)
        cur.c.cursor, cur.c.floor = c, f
        cur.update(buf, n, k, a, y)
        assert (cur.cursor, cur.floor) == (o.c, o.f), (c, f, k, a, y, n, radius)


# -- publication semantics ---------------------------------------------------------

def test_buffer_batches_records_and_errors(lib):
    from paper_2609_37617_amd import as2d
    buf = lib.CandidateBuffer(20)
    assert buf.publish([1, 2, 3], source_id=7, producer_id=2, offset=0, publish_ns=100, confidence=0.5) == 3
    assert buf.publish(list(range(10, 18)), source_id=7, producer_id=2, offset=3, publish_ns=250) == 11
    assert buf.snapshot() == 11
    assert buf.read(0, 11) == [1, 2, 3] + list(range(10, 18))
    recs = buf.records()
    assert [(r["first"], r["count"], r["source_id"], r["producer_id"], r["offset"], r["publish_ns"]) for r in recs] == \
        [(0, 3, 7, 2, 0, 100), (3, 8, 7, 2, 3, 250)]
    assert recs[0]["confidence"] == pytest.approx(0.5) and np.isnan(recs[1]["confidence"])
    for bad in ([], list(range(9))):
        with pytest.raises(as2d.As2dError):
            buf.publish(bad)
    with pytest.raises(as2d.As2dError):
        buf.read(5, 7)                       # past the published length
    assert buf.read(40, 0) == []             # an empty read is valid anywhere
    buf.publish(list(range(8)))
    with pytest.raises(as2d.As2dError) as e:
        buf.publish([1, 2])                  # 19 + 2 > 20
    assert e.value.code == as2d.ECAPACITY
    cur = lib.ReadCursor(8)
    with pytest.raises(as2d.As2dError):
        cur.propose(buf, buf.snapshot() + 1, 4)
    with pytest.raises(as2d.As2dError):
        cur.update(buf, 4, 2, 3, 1)          # accepted > k
    with pytest.raises(as2d.As2dError):
        lib.ReadCursor(65)


def test_snapshots_are_immutable_under_concurrent_publication(lib):
    """A reader's snapshot never changes while a producer thread appends."""
    total = 4096
    stream = [(i * 7919) % 1000 for i in range(total)]
    buf = lib.CandidateBuffer(total)
    done = threading.Event()

    def producer():
        for i in range(0, total, 8):
            buf.publish(stream[i:i + 8], offset=i, publish_ns=i)
        done.set()

    th = threading.Thread(target=producer)
    th.start()
    seen = 0
    while not done.is_set() or seen < total:
        n = buf.snapshot()
        assert n % 8 == 0 and n >= seen
        if n > seen:
            assert buf.read(seen, n - seen) == stream[seen:n]
            seen = n
    th.join()
    assert buf.read(0, total) == stream
