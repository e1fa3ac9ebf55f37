"""The persistent step kernel on the 7B shape (four layers): a verification
pass through one persistent launch (every phase on the balanced GEMM
units, grid-wide waits between phases) gives the per-operation graph's
result bit for bit -- logits, outcome and appended KV -- for one request
at widths 1, 9 and 21 (one and two row tiles) and for a fused pass of
three requests, replay after replay."""
import numpy as np
import pytest

from tests.harness import make_pair, prefix
from workload import QWEN7B

pytestmark = pytest.mark.gpu

SHAPE = QWEN7B.with_layers(4)


@pytest.fixture(scope="module")
def model():
    from paper_2609_37617_amd import as2d
    _, gpu = make_pair(SHAPE, seed=3, max_requests=3, max_kv_len=1024, max_k=24, oracle=False)
    gpu.set_keep_logits(True)
    states = {}
    for req, (n_audio, n_instr) in enumerate(((750, 32), (300, 16), (90, 8))):
        _, a_dev, instr = prefix(SHAPE, n_audio, n_instr, 3, req)
        states[req] = gpu.prefill(req, a_dev, instr)[::-1]       # (kv_len, first root)
    mode, grid = gpu.exec_info()
    assert grid >= 1
    yield as2d, gpu, states
    gpu.set_exec_mode(as2d.EXEC_GRAPH)
    gpu.close()


def run(gpu, reqs, cands, states):
    outs = gpu.verify_batch(reqs, cands) if len(reqs) > 1 else [gpu.verify(reqs[0], cands[0])]
    res = []
    for req, c, o in zip(reqs, cands, outs):
        L = states[req][0]
        res.append((o, gpu.logits(req).copy(), gpu.read_kv(req, SHAPE.n_layers - 1, L + len(c) + 1)))
        gpu.rollback(req, *states[req])
    return res


@pytest.mark.parametrize("ks", [(0,), (8,), (20,), (8, 4, 6)], ids=["w1", "w9", "w21", "batch3"])
def test_persistent_equals_graph(model, ks):
    as2d, gpu, states = model
    rng = np.random.default_rng(sum(ks) + len(ks))
    reqs = list(range(len(ks)))
    cands = [[int(t) for t in rng.integers(0, SHAPE.vocab, k)] for k in ks]
    print(f"persistent vs graph: ks={ks}", flush=True)
    gpu.set_exec_mode(as2d.EXEC_GRAPH)
    ref = run(gpu, reqs, cands, states)
    for rep in range(3):
        gpu.set_exec_mode(as2d.EXEC_PERSISTENT)
        got = run(gpu, reqs, cands, states)
        for (o, lg, kv), (ro, rlg, rkv) in zip(got, ref):
            assert o == ro, rep
            assert np.array_equal(lg, rlg), rep
            assert np.array_equal(kv[0], rkv[0]) and np.array_equal(kv[1], rkv[1]), rep
        gpu.set_exec_mode(as2d.EXEC_GRAPH)
        gpu.decode_one(0)                     # other work between replays
        gpu.rollback(0, *states[0])
