"""GPU parity at the real widths of the 3B and 7B shapes, with the same
kernels and launch configurations the benchmark times (the k-split plan
and tile grids depend only on the matrix shapes, which are unchanged):
one or two decoder layers, full hidden size, heads, FFN and vocabulary,
and the workloads' prefix lengths."""
import numpy as np
import pytest

from tests.harness import Stats, compare_kv, logit_tol, make_pair, parity_round, prefix, restore, snapshot
from workload import QWEN3B, QWEN7B, workload
from workload.gen import CandidateSource

pytestmark = pytest.mark.gpu


def run_rounds(shape, n_audio, n_instr, k, p, rounds, reply, max_kv):
    om, gpu = make_pair(shape, seed=0, max_requests=1, max_kv_len=max_kv, max_k=max(k, 1))
    gpu.set_keep_logits(True)
    a_or, a_dev, instr = prefix(shape, n_audio, n_instr)
    f_o, L_o = om.prefill(a_or, instr)
    f_g, L_g = gpu.prefill(0, a_dev, instr)
    assert L_o == L_g
    err = float(np.max(np.abs(gpu.logits(0)[0] - om.last_logits[0])))
    assert err <= logit_tol(shape)
    if f_g != f_o:
        assert om.last_logits[0].max() - np.sort(om.last_logits[0])[-2] <= 0.05
        om.root = f_g
    snap = snapshot(om)
    y = om.target_only(reply)
    restore(om, snap)
    src = CandidateSource(y, shape.vocab, p, seed=0)
    st = Stats()
    n = 0
    for _ in range(rounds):
        kk = min(k, reply - n - 1)
        if kk < 0:
            break
        r = parity_round(om, gpu, 0, src.block(n, kk), kk, logit_tol(shape), st)
        n += r["accepted_len"] + 1
    for l in range(shape.n_layers):
        compare_kv(om, gpu, 0, l, om.kv_len, 2e-3)
    print(f"{shape.name} k={k}: rounds={st.rounds} committed={st.committed} near_ties={st.near_ties} "
          f"max_logit_err={st.max_err:.3g} prefill_err={err:.3g}")
    gpu.close()
    return st


def test_qwen7b_width_k8():
    """7B widths, 750 audio + 32 instruction rows, k = 8, p = 0.3."""
    rq = workload(2).requests[0]
    run_rounds(QWEN7B.with_layers(1), rq.n_audio, rq.n_instr, 8, 0.3, rounds=6, reply=30, max_kv=1152)


def test_qwen7b_width_k16_two_layers():
    """k = 16 (two M-tiles of rows) through two layers."""
    rq = workload(2).requests[0]
    run_rounds(QWEN7B.with_layers(2), rq.n_audio, rq.n_instr, 16, 0.1, rounds=3, reply=40, max_kv=1152)


def test_qwen3b_width_k4():
    rq = workload(1).requests[0]
    run_rounds(QWEN3B.with_layers(1), rq.n_audio, rq.n_instr, 4, 0.3, rounds=6, reply=20, max_kv=1024)
