"""Oracle parity of the full-depth 7B shape (28 layers, hidden 3584, 28/4
heads, FFN 18944, vocabulary 152064, bf16 weights): every verification
decision, logit and the first and last layers' KV cache of the HIP path
against the float64 oracle on the same seeded inputs, for

* the ASR-like workload (750 audio + 32 instruction rows) at k in
  {0, 1, 2, 4, 8, 16} and p in {0.1, 0.3, 0.6};
* the long-audio workload (7,500 + 64 prefix rows, k = 8, p = 0.4);
* the mixed batch: all sixteen requests verified in fused passes (68 rows,
  the staged GEMM path), two of them against the oracle;

plus the bitwise properties of the full-depth GPU model itself: batched
verification equals sequential decoding (Appendix C.4, requirement 1), a
fused pass equals each request alone, and corrupted proposals commit the
target-only stream (Proposition).

The bar: logits within 3e-2, KV within 2e-3, decisions identical unless
the first differing row's oracle top-2 margin is at most 0.05 (then the
oracle follows the GPU's commit; tests/harness.py).  One model and one
oracle (float64 weights, about 61 GB of host memory) serve the module."""
import copy

import numpy as np
import pytest

from tests.harness import (Stats, check_round, compare_kv, full_pair, log, oracle_prefill, parity_round, prefix,
                           restore, snapshot)
from workload import QWEN7B, workload
from workload.gen import CandidateSource

pytestmark = pytest.mark.gpu

TOL = 3e-2
KV_TOL = 2e-3
MAX_KV = 7680          # the long-audio prefix (7,564 rows) and its rounds
LAST = QWEN7B.n_layers - 1


@pytest.fixture(scope="module")
def m7():
    om, gpu = full_pair(QWEN7B, seed=0, max_requests=16, max_kv_len=MAX_KV, max_k=16)
    gpu.set_keep_logits(True)
    yield om, gpu
    gpu.close()


def prefill_both(om, gpu, req, n_audio, n_instr, seed=0):
    """Prefill slot `req` and the oracle (in causal row chunks); the first
    token follows the near-tie protocol.  Returns (kv_len, first root)."""
    a_or, a_dev, instr = prefix(QWEN7B, n_audio, n_instr, seed, req)
    f_o, L_o = oracle_prefill(om, a_or, instr)
    f_g, L_g = gpu.prefill(req, a_dev, instr)
    assert L_o == L_g == n_audio + n_instr
    err = float(np.max(np.abs(gpu.logits(req)[0] - om.last_logits[0])))
    assert err <= TOL, err
    if f_g != f_o:
        top = np.sort(om.last_logits[0])
        assert top[-1] - top[-2] <= 0.05, "first token differs outside a near tie"
        om.root = f_g
    log(f"  prefill of {L_g} rows (slot {req}): first token {f_g}, logit error {err:.3g}")
    return L_g, om.root


def rounds(om, gpu, req, src, k, n_rounds, st):
    n = 0
    for _ in range(n_rounds):
        r = parity_round(om, gpu, req, src.block(n, k), k, TOL, st)
        n += r["accepted_len"] + 1
    return n


# ---------------------------------------------------------------------------
# the ASR-like workload: k and p sweep from one prefill

@pytest.fixture(scope="module")
def asr(m7):
    om, gpu = m7
    rq = workload(2).requests[0]
    log("[7B ASR] prefill")
    L, root = prefill_both(om, gpu, 0, rq.n_audio, rq.n_instr)
    snap = snapshot(om)
    y = om.target_only(36)        # y_0 (the root) .. y_36: covers every sweep case below
    restore(om, snap)
    log(f"[7B ASR] oracle reference stream of {len(y) - 1} tokens")
    return (L, root), snap, y


@pytest.mark.parametrize("k,p,n_rounds", [(8, 0.3, 4), (16, 0.1, 1), (8, 0.6, 3), (4, 0.6, 3), (2, 0.3, 3),
                                          (1, 0.1, 3), (0, 0.3, 2)])
def test_qwen7b_asr_rounds(m7, asr, k, p, n_rounds):
    om, gpu = m7
    state, snap, y = asr
    restore(om, snap)
    gpu.rollback(0, *state)
    src = CandidateSource(y, QWEN7B.vocab, p, seed=0)
    st = Stats()
    n = rounds(om, gpu, 0, src, k, n_rounds, st)
    assert gpu.state(0) == (om.kv_len, om.root, om.kv_len - state[0])
    ek, ev = compare_kv(om, gpu, 0, 0, om.kv_len, KV_TOL)
    ek2, ev2 = compare_kv(om, gpu, 0, LAST, om.kv_len, KV_TOL)
    log(f"[7B ASR k={k} p={p}] rounds={st.rounds} committed={n} near_ties={st.near_ties} "
        f"max_logit_err={st.max_err:.3g} kv_err first={max(ek, ev):.3g} last={max(ek2, ev2):.3g}")


# ---------------------------------------------------------------------------
# bitwise properties of the full-depth GPU model

def target_only(gpu, req, state, n):
    gpu.rollback(req, *state)
    toks, logits = [], []
    for _ in range(n):
        toks.append(gpu.decode_one(req)["correction_token"])
        logits.append(gpu.logits(req)[0].copy())
    gpu.rollback(req, *state)
    return toks, logits


@pytest.fixture(scope="module")
def two_requests(m7):
    _, gpu = m7
    states = {}
    for req, (n_audio, n_instr) in ((1, (750, 32)), (2, (300, 32))):
        _, a_dev, instr = prefix(QWEN7B, n_audio, n_instr, 0, req)
        states[req] = gpu.prefill(req, a_dev, instr)[::-1]       # (kv_len, first root)
    return states


@pytest.mark.parametrize("k", [8, 16])
def test_verify_equals_sequential_decoding(m7, two_requests, k):
    _, gpu = m7
    s = two_requests[1]
    ref, ref_logits = target_only(gpu, 1, s, k + 1)
    r = gpu.verify(1, ref[:k])
    assert r["accepted_len"] == k and r["correction_token"] == ref[k]
    lg = gpu.logits(1)
    for i in range(k + 1):
        assert np.array_equal(lg[i], ref_logits[i]), i
    gpu.rollback(1, *s)


def test_batch_equals_single(m7, two_requests):
    _, gpu = m7
    states = two_requests
    ref1, _ = target_only(gpu, 1, states[1], 9)
    ref2, _ = target_only(gpu, 2, states[2], 5)
    c1, c2 = ref1[:8], [ref2[0], ref2[1], (ref2[2] + 1) % QWEN7B.vocab, ref2[3]]
    outs = gpu.verify_batch([1, 2], [c1, c2])
    lg1, lg2 = gpu.logits(1), gpu.logits(2)
    singles = []
    for req, c in ((1, c1), (2, c2)):
        gpu.rollback(req, *states[req])
        singles.append((gpu.verify(req, c), gpu.logits(req)))
    assert outs[0] == singles[0][0] and outs[1] == singles[1][0]
    assert np.array_equal(lg1, singles[0][1]) and np.array_equal(lg2, singles[1][1])
    assert outs[0]["accepted_len"] == 8 and outs[1]["accepted_len"] == 2
    for req in (1, 2):
        gpu.rollback(req, *states[req])


def test_corrupted_proposals_commit_the_target_stream(m7, two_requests):
    _, gpu = m7
    s = two_requests[1]
    n = 48
    ref, _ = target_only(gpu, 1, s, n + 1)
    src = CandidateSource([s[1]] + ref, QWEN7B.vocab, 0.4, seed=3)
    gpu.set_keep_logits(False)
    out = []
    while len(out) < n:
        k = min(8, n - len(out) - 1)
        r = gpu.verify(1, src.block(len(out), k))
        out += src.block(len(out), k)[:r["accepted_len"]] + [r["correction_token"]]
    gpu.set_keep_logits(True)
    assert out == ref[:n]
    gpu.rollback(1, *s)


# ---------------------------------------------------------------------------
# the mixed batch: sixteen requests in fused passes, two against the oracle

def test_qwen7b_mixed_batch(m7):
    om0, gpu = m7
    wl = workload(4)
    reqs = wl.requests
    sample = (3, 10)               # k = 8 (699 prefix rows) and k = 4 (1,074 rows)
    n_rounds = 2
    oms, srcs = {}, {}
    log("[7B mixed batch] prefill")
    for i, r in enumerate(reqs):
        if i in sample:
            om = copy.copy(om0)    # same weights, a state of its own
            om.reset()
            prefill_both(om, gpu, i, r.n_audio, r.n_instr, seed=wl.seed)
            snap = snapshot(om)
            y = om.target_only(n_rounds * (r.k + 1) + 1)
            restore(om, snap)
            oms[i] = om
            srcs[i] = CandidateSource(y, QWEN7B.vocab, r.p, seed=wl.seed, req=i)
        else:
            _, a_dev, instr = prefix(QWEN7B, r.n_audio, r.n_instr, wl.seed, i)
            gpu.prefill(i, a_dev, instr)
    rng = np.random.default_rng(4)
    done = {i: 0 for i in range(len(reqs))}
    st = Stats()
    ids = list(range(len(reqs)))
    for rnd in range(n_rounds):
        cands = [srcs[i].block(done[i], reqs[i].k) if i in srcs else
                 [int(t) for t in rng.integers(0, QWEN7B.vocab, reqs[i].k)] for i in ids]
        rows = sum(len(c) + 1 for c in cands)
        before = {i: gpu.state(i) for i in ids}
        snaps = {i: snapshot(oms[i]) for i in oms}
        outs = gpu.verify_batch(ids, cands)
        lgs = {i: gpu.logits(i) for i in ids}
        toks = {i: gpu.row_tokens(i) for i in ids}
        for i in oms:
            k = len(cands[i])
            ro = oms[i].verify(cands[i], k)
            check_round(oms[i], snaps[i], ro, outs[i], toks[i], lgs[i], cands[i], k, TOL, st)
        after = {i: gpu.state(i) for i in ids}
        for i in ids:             # each request alone: the same bits (direct path)
            gpu.rollback(i, before[i][0], before[i][1])
            assert gpu.verify(i, cands[i]) == outs[i], i
            assert np.array_equal(gpu.logits(i), lgs[i]), i
            assert gpu.state(i) == after[i]
        for i in ids:
            done[i] += outs[i]["accepted_len"] + 1
        log(f"[7B mixed batch] round {rnd}: {rows} rows in the fused pass")
    assert rows > 32               # the staged GEMM path
    for i in oms:
        compare_kv(oms[i], gpu, i, 0, oms[i].kv_len, KV_TOL)
        compare_kv(oms[i], gpu, i, LAST, oms[i].kv_len, KV_TOL)
    log(f"[7B mixed batch] rounds={st.rounds} committed={st.committed} near_ties={st.near_ties} "
        f"max_logit_err={st.max_err:.3g}")


# ---------------------------------------------------------------------------
# the long-audio workload

def test_qwen7b_long_audio(m7):
    om, gpu = m7
    rq = workload(3).requests[0]
    n_rounds = 2
    log("[7B long audio] prefill (the oracle takes about two minutes)")
    om.reset()
    L, root = prefill_both(om, gpu, 0, rq.n_audio, rq.n_instr)
    snap = snapshot(om)
    y = om.target_only(n_rounds * (rq.k + 1) + 1)
    restore(om, snap)
    src = CandidateSource(y, QWEN7B.vocab, rq.p, seed=0)
    st = Stats()
    n = rounds(om, gpu, 0, src, rq.k, n_rounds, st)
    assert gpu.state(0)[0] == om.kv_len
    ek, ev = compare_kv(om, gpu, 0, 0, om.kv_len, KV_TOL)
    ek2, ev2 = compare_kv(om, gpu, 0, LAST, om.kv_len, KV_TOL)
    log(f"[7B long audio] rounds={st.rounds} committed={n} near_ties={st.near_ties} max_logit_err={st.max_err:.3g} "
        f"kv_err first={max(ek, ev):.3g} last={max(ek2, ev2):.3g}")
