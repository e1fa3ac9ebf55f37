"""Oracle parity of the full-depth 3B shape (36 layers, hidden 2048, 16/2
heads, FFN 11008, vocabulary 151936, bf16 weights) on the ASR-like
workload: 750 audio + 32 instruction rows, verification rounds at k = 4
(p = 0.3, the workload's setting) and k = 8 (p = 0.1); logits within 3e-2,
decisions under the near-tie protocol, the first and last layers' KV within
2e-3 (tests/harness.py)."""
import numpy as np
import pytest

from tests.harness import Stats, compare_kv, full_pair, log, parity_round, prefix, restore, snapshot
from workload import QWEN3B, workload
from workload.gen import CandidateSource

pytestmark = pytest.mark.gpu


def test_qwen3b_full_depth():
    rq = workload(1).requests[0]
    om, gpu = full_pair(QWEN3B, seed=0, max_requests=1, max_kv_len=1024, max_k=8)
    gpu.set_keep_logits(True)
    a_or, a_dev, instr = prefix(QWEN3B, rq.n_audio, rq.n_instr)
    f_o, L_o = om.prefill(a_or, instr)
    f_g, L_g = gpu.prefill(0, a_dev, instr)
    assert L_o == L_g
    err = float(np.max(np.abs(gpu.logits(0)[0] - om.last_logits[0])))
    assert err <= 3e-2, err
    if f_g != f_o:
        top = np.sort(om.last_logits[0])
        assert top[-1] - top[-2] <= 0.05
        om.root = f_g
    state = (L_g, om.root)
    snap = snapshot(om)
    y = om.target_only(30)
    restore(om, snap)
    log(f"[3B] prefill {L_g} rows, logit error {err:.3g}; oracle reference stream of 30 tokens")
    for k, p, n_rounds in ((rq.k, rq.p, 6), (8, 0.1, 2)):
        restore(om, snap)
        gpu.rollback(0, *state)
        src = CandidateSource(y, QWEN3B.vocab, p, seed=0)
        st = Stats()
        n = 0
        for _ in range(n_rounds):
            r = parity_round(om, gpu, 0, src.block(n, k), k, 3e-2, st)
            n += r["accepted_len"] + 1
        assert gpu.state(0)[0] == om.kv_len
        kv = [max(compare_kv(om, gpu, 0, l, om.kv_len, 2e-3)) for l in (0, QWEN3B.n_layers - 1)]
        log(f"[3B k={k} p={p}] rounds={st.rounds} committed={n} near_ties={st.near_ties} "
            f"max_logit_err={st.max_err:.3g} kv_err first={kv[0]:.3g} last={kv[1]:.3g}")
    gpu.close()
