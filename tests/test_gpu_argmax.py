"""The LM head's arg-max on the GPU at exact ties, and non-finite logits
in one request of a fused pass.

Ties are planted by copying one LM-head row over another: the two token
ids then get bit-identical logits (the same weights times the same
activations), and the greedy token must be the lower id (the
deterministic tie-break of Appendix C.4, Eq. reference-transition, read
as the lowest token id) wherever the two sit: in one 32-column tile pair,
in two pairs of one workgroup, or in two workgroups.  Both orders are
planted (the copy above and below the original id), so a scan that kept
the first or the last maximum it met would fail one of them.  The device's
top-2 margin of the tied row must be exactly 0.

The vocabulary is widened to 16,384 (512 tile pairs) so that the LM head's
balanced plan gives each of its 256 workgroups two pairs (2 b, 2 b + 1)."""
import dataclasses

import numpy as np
import pytest

from tests.harness import ensure_built, prefix
from workload import TINY_BF16, gen

pytestmark = pytest.mark.gpu

SHAPE = dataclasses.replace(TINY_BF16, name="tiny-bf16-v16k", vocab=16384)
BF16_INF = 0x7F80


def load(tensors, max_requests=1):
    from paper_2609_37617_amd import as2d
    ensure_built()
    m = as2d.Model(SHAPE, tensors, max_requests=max_requests, max_kv_len=256, max_k=8)
    m.set_keep_logits(True)
    return m


def lm_index():
    return [i for i, e in enumerate(gen.weight_spec(SHAPE)) if e[0] == "lm_head"][0]


@pytest.fixture(scope="module")
def base():
    w = gen.make_weights(SHAPE, seed=0, fmt="device")
    _, a_dev, instr = prefix(SHAPE, 40, 6, seed=0)
    m = load(w)
    first, _ = m.prefill(0, a_dev, instr)
    lg = m.logits(0)[0]
    margin = float(m.row_margins(0)[0])
    m.close()
    assert int(np.argmax(lg)) == first
    top = np.sort(lg)
    assert margin == top[-1] - top[-2] and margin > 0
    return w, (a_dev, instr), first


def partner(t, where, below):
    """A token id tied with t: in t's pair, in the other pair of t's LM-head
    workgroup, or in another workgroup; below: a lower id than t."""
    pair, col = divmod(t, 32)
    if where == "pair":
        c = [x for x in range(32) if (x < col) == below and x != col]
        return pair * 32 + (c[len(c) // 2] if c else (col + 1) % 32)
    if where == "workgroup":
        other = pair ^ 1
    else:
        other = (pair + 128) % (SHAPE.vocab // 32) if not below else (pair - 128) % (SHAPE.vocab // 32)
    return other * 32 + col


@pytest.mark.parametrize("where", ["pair", "workgroup", "grid"])
@pytest.mark.parametrize("below", [True, False], ids=["copy-below", "copy-above"])
def test_exact_tie_goes_to_the_lowest_id(base, where, below):
    w, (a_dev, instr), t = base
    t2 = partner(t, where, below)
    if (t2 < t) != below or t2 == t:
        pytest.skip(f"no {where} partner {'below' if below else 'above'} token {t}")
    tied = list(w)
    lm = tied[lm_index()].copy()
    lm[t2] = lm[t]
    tied[lm_index()] = lm
    m = load(tied)
    first, _ = m.prefill(0, a_dev, instr)
    lg = m.logits(0)[0]
    mg = float(m.row_margins(0)[0])
    m.close()
    assert lg[t] == lg[t2] and lg[t] == lg.max()
    assert first == min(t, t2), (where, t, t2, first)
    assert mg == 0.0


def test_non_finite_logits_fail_only_their_request():
    """A token whose embedding row is +inf makes every logit of its row
    NaN.  In a fused pass, the request that proposes it gets AS2D_ENUMERIC
    and keeps its state; the other request is committed exactly as when
    verified alone."""
    from paper_2609_37617_amd import as2d
    w = gen.make_weights(SHAPE, seed=1, fmt="device")
    bad_tok = 777
    emb = w[0].copy()
    emb[bad_tok] = BF16_INF
    w[0] = emb
    m = load(w, max_requests=2)
    states = {}
    for req in (0, 1):
        _, a_dev, instr = prefix(SHAPE, 30, 4, seed=2, req=req)
        states[req] = m.prefill(req, a_dev, instr)[::-1]
    good = [5, 6, 7]
    single = m.verify(0, good)
    single_logits = m.logits(0)
    m.rollback(0, *states[0])
    rc, outs = m.verify_batch_status([0, 1], [good, [bad_tok, 9]])
    assert rc == as2d.ENUMERIC
    assert outs[0] == single
    assert np.array_equal(m.logits(0), single_logits)
    assert outs[1]["accepted_len"] == -1 and outs[1]["correction_token"] == -1
    assert m.state(1)[:2] == states[1]
    assert not np.all(np.isfinite(m.logits(1)))
    # the request goes on once the offending candidate is gone
    r = m.verify(1, [9])
    assert r["kv_len"] == states[1][0] + r["accepted_len"] + 1
    m.close()
