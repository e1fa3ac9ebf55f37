"""GPU parity on the long-audio and mixed-batch workloads at the 7B widths
(one decoder layer, full hidden size, heads, FFN and vocabulary), with the
workloads' real prefix lengths and request mix:

* long audio: a 7,500-row audio prefix plus 64 instruction tokens, k = 8
  and p = 0.4; the attention spans 237 key chunks;
* mixed batch: the sixteen requests of the batch workload (ragged
  prefixes of 282..3032 rows, k in {0, 4, 8}) verified in fused passes of
  up to 144 rows (the staged GEMM path); a sample of the requests is
  checked against the oracle, and every request's result in the fused pass
  must equal, bit for bit, the same request verified alone (the direct
  GEMM path), which is the batch-invariance property at full width."""
import copy

import numpy as np
import pytest

from tests.harness import (Stats, check_round, compare_kv, logit_tol, make_pair, oracle_prefill, parity_round, prefix,
                           restore, snapshot)
from workload import QWEN7B, workload
from workload.gen import CandidateSource

pytestmark = pytest.mark.gpu


def _prefill_both(om, gpu, req, shape, n_audio, n_instr, seed=0):
    a_or, a_dev, instr = prefix(shape, n_audio, n_instr, seed, req)
    f_o, L_o = oracle_prefill(om, a_or, instr)
    f_g, L_g = gpu.prefill(req, a_dev, instr)
    assert L_o == L_g == n_audio + n_instr
    err = float(np.max(np.abs(gpu.logits(req)[0] - om.last_logits[0])))
    assert err <= logit_tol(shape), err
    if f_g != f_o:   # a near tie on the first token: follow the GPU
        assert om.last_logits[0].max() - np.sort(om.last_logits[0])[-2] <= 0.05
        om.root = f_g
    return err


def test_qwen7b_long_audio_width():
    """Workload 3 (7,500 audio + 64 instruction rows, k = 8, p = 0.4) at the
    7B widths, one layer: prefill, verification rounds against the oracle,
    and the whole KV cache afterwards."""
    rq = workload(3).requests[0]
    shape = QWEN7B.with_layers(1)
    rounds, reply = 4, 40
    max_kv = (rq.n_audio + rq.n_instr + reply + 16 + 63) // 64 * 64
    om, gpu = make_pair(shape, seed=0, max_requests=1, max_kv_len=max_kv, max_k=rq.k)
    gpu.set_keep_logits(True)
    perr = _prefill_both(om, gpu, 0, shape, rq.n_audio, rq.n_instr)
    snap = snapshot(om)
    y = om.target_only(reply)
    restore(om, snap)
    src = CandidateSource(y, shape.vocab, rq.p, seed=0)
    st = Stats()
    n = 0
    for _ in range(rounds):
        k = max(0, min(rq.k, reply - n - 1))
        r = parity_round(om, gpu, 0, src.block(n, k), k, logit_tol(shape), st)
        n += r["accepted_len"] + 1
    compare_kv(om, gpu, 0, 0, om.kv_len, 2e-3)
    print(f"long audio: rounds={st.rounds} committed={st.committed} near_ties={st.near_ties} "
          f"max_logit_err={st.max_err:.3g} prefill_err={perr:.3g}")
    gpu.close()


def test_qwen7b_mixed_batch_width():
    """Workload 4 (16 requests) at the 7B widths, one layer."""
    wl = workload(4)
    reqs = wl.requests
    shape = QWEN7B.with_layers(1)
    rounds = 3
    sample = [3, 8, 10, 15]     # k = 8, 0, 4, 8; prefixes of 699 .. 2481 rows
    max_kv = (max(r.n_audio + r.n_instr for r in reqs) + rounds * 9 + 16 + 63) // 64 * 64
    om0, gpu = make_pair(shape, seed=0, max_requests=len(reqs), max_kv_len=max_kv, max_k=8)
    gpu.set_keep_logits(True)
    oms = {}
    for i in sample:            # one oracle state per sampled request, sharing the weights
        oms[i] = copy.copy(om0)
        oms[i].reset()
    srcs = {}
    for i, r in enumerate(reqs):
        if i in oms:
            _prefill_both(oms[i], gpu, i, shape, r.n_audio, r.n_instr, seed=wl.seed)
            snap = snapshot(oms[i])
            y = oms[i].target_only(rounds * 9 + 2)
            restore(oms[i], snap)
            srcs[i] = CandidateSource(y, shape.vocab, r.p, seed=wl.seed, req=i)
        else:
            _, a_dev, instr = prefix(shape, r.n_audio, r.n_instr, wl.seed, i)
            gpu.prefill(i, a_dev, instr)
    rng = np.random.default_rng(4)
    done = {i: 0 for i in range(len(reqs))}
    st = Stats()
    rows_max = 0
    for _ in range(rounds):
        ids = list(range(len(reqs)))
        cands = []
        for i in ids:
            k = reqs[i].k
            cands.append(srcs[i].block(done[i], k) if i in srcs else [int(t) for t in rng.integers(0, shape.vocab, k)])
        rows_max = max(rows_max, sum(len(c) + 1 for c in cands))
        before = {i: gpu.state(i) for i in ids}
        snaps = {i: snapshot(oms[i]) for i in oms}
        outs = gpu.verify_batch(ids, cands)
        lgs = {i: gpu.logits(i) for i in ids}
        toks = {i: gpu.row_tokens(i) for i in ids}
        # the oracle, for the sampled requests
        for i in oms:
            k = len(cands[i])
            ro = oms[i].verify(cands[i], k)
            check_round(oms[i], snaps[i], ro, outs[i], toks[i], lgs[i], cands[i], k, logit_tol(shape), st)
        # each request alone gives the same bits (direct path, M = k + 1)
        after = {i: gpu.state(i) for i in ids}
        for i in ids:
            gpu.rollback(i, before[i][0], before[i][1])
            single = gpu.verify(i, cands[i])
            assert single == outs[i], (i, single, outs[i])
            assert np.array_equal(gpu.logits(i), lgs[i]), i
            assert gpu.state(i) == after[i]
        for i in ids:
            done[i] += outs[i]["accepted_len"] + 1
    assert rows_max > 32, rows_max    # the fused passes took the staged path
    for i in oms:
        compare_kv(oms[i], gpu, i, 0, oms[i].kv_len, 2e-3)
    print(f"mixed batch: rounds={st.rounds} committed={st.committed} near_ties={st.near_ties} "
          f"max_logit_err={st.max_err:.3g} max_rows={rows_max}")
    gpu.close()
