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


def test_persistent_after_cu_budget_equals_graph(model):
    """A compute-unit budget rebuilds the persistent kernel's grid and its
    per-layer argument arrays.  On 224 CUs the persistent pass runs on 224
    workgroups; on 128 the LM head's 4,752 tile pairs need 198 workgroups of
    24 units, more than the budget, so persistent mode runs the graph path
    (reported grid 0).  Either way, and after the budget is lifted again,
    the result is the whole-device graph's bit for bit."""
    as2d, gpu, states = model
    rng = np.random.default_rng(11)
    reqs = [0, 1]
    cands = [[int(t) for t in rng.integers(0, SHAPE.vocab, k)] for k in (8, 5)]
    gpu.set_exec_mode(as2d.EXEC_GRAPH)
    ref = run(gpu, reqs, cands, states)
    try:
        for cus, grid in ((224, 224), (128, 0), (0, None)):
            gpu.set_cu_budget(cus)
            print(f"persistent after cu budget {cus}", flush=True)
            if grid is not None:
                assert gpu.exec_info()[1] == grid
            for mode in (as2d.EXEC_PERSISTENT, as2d.EXEC_EAGER):
                gpu.set_exec_mode(mode)
                got = run(gpu, reqs, cands, states)
                for (o, lg, kv), (ro, rlg, rkv) in zip(got, ref):
                    assert o == ro, (cus, mode)
                    assert np.array_equal(lg, rlg), (cus, mode)
                    assert np.array_equal(kv[0], rkv[0]) and np.array_equal(kv[1], rkv[1]), (cus, mode)
    finally:
        gpu.set_cu_budget(0)
        gpu.set_exec_mode(as2d.EXEC_GRAPH)
