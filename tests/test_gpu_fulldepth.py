"""Exact properties of the full-depth 7B-shaped model (28 layers; too slow
for the float64 oracle, which covers the same widths with one or two
layers): batched verification equals sequential target-only decoding bit
for bit (Appendix C.4, requirement 1) at widths 9 and 17 (both direct row
tiles), a fused pass of two requests equals each request alone, and a
corrupted proposal stream commits the target-only stream (Proposition)."""
import numpy as np
import pytest

from tests.harness import make_pair, prefix
from workload import QWEN7B, gen
from workload.gen import CandidateSource

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def model():
    _, gpu = make_pair(QWEN7B, seed=0, max_requests=2, max_kv_len=896, max_k=16, oracle=False)
    gpu.set_keep_logits(True)
    states = {}
    for req, (n_audio, n_instr) in enumerate(((750, 32), (300, 32))):
        _, a_dev, instr = prefix(QWEN7B, n_audio, n_instr, 0, req)
        states[req] = gpu.prefill(req, a_dev, instr)[::-1]       # (kv_len, first root)
    yield gpu, states
    gpu.close()


def target_only(gpu, req, state, n):
    gpu.rollback(req, *state)
    toks, logits = [], []
    for _ in range(n):
        toks.append(gpu.decode_one(req)["correction_token"])
        logits.append(gpu.logits(req)[0].copy())
    gpu.rollback(req, *state)
    return toks, logits


@pytest.mark.parametrize("k", [8, 16])
def test_verify_equals_sequential_decoding(model, k):
    gpu, states = model
    ref, ref_logits = target_only(gpu, 0, states[0], k + 1)
    r = gpu.verify(0, ref[:k])
    assert r["accepted_len"] == k and r["correction_token"] == ref[k]
    lg = gpu.logits(0)
    for i in range(k + 1):
        assert np.array_equal(lg[i], ref_logits[i]), i
    gpu.rollback(0, *states[0])


def test_batch_equals_single(model):
    gpu, states = model
    ref0, _ = target_only(gpu, 0, states[0], 9)
    ref1, _ = target_only(gpu, 1, states[1], 5)
    c0, c1 = ref0[:8], [ref1[0], ref1[1], (ref1[2] + 1) % QWEN7B.vocab, ref1[3]]
    outs = gpu.verify_batch([0, 1], [c0, c1])
    lg0, lg1 = gpu.logits(0), gpu.logits(1)
    singles = []
    for req, c in ((0, c0), (1, c1)):
        gpu.rollback(req, *states[req])
        singles.append((gpu.verify(req, c), gpu.logits(req)))
    assert outs[0] == singles[0][0] and outs[1] == singles[1][0]
    assert np.array_equal(lg0, singles[0][1]) and np.array_equal(lg1, singles[1][1])
    assert outs[0]["accepted_len"] == 8 and outs[1]["accepted_len"] == 2
    for req in (0, 1):
        gpu.rollback(req, *states[req])


def test_corrupted_proposals_commit_the_target_stream(model):
    gpu, states = model
    n = 48
    ref, _ = target_only(gpu, 0, states[0], n + 1)
    src = CandidateSource([states[0][1]] + ref, QWEN7B.vocab, 0.4, seed=3)
    gpu.set_keep_logits(False)
    out = []
    while len(out) < n:
        k = min(8, n - len(out) - 1)
        r = gpu.verify(0, src.block(len(out), k))
        out += src.block(len(out), k)[:r["accepted_len"]] + [r["correction_token"]]
    gpu.set_keep_logits(True)
    assert out == ref[:n]
    gpu.rollback(0, *states[0])
