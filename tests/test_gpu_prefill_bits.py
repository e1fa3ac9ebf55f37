"""A prefilled cache equals the incrementally built one bit for bit at the 7B
widths, with prefixes of several spans.

Commit-and-repair (Appendix C.4): after verification rounds with rejections,
a fresh prefill of the committed prefix must reproduce the retained cache.
Prefill attention runs its spans two at a time (two groups of four waves, the
second handing its span state to the first) while verification stores every
span's state and merges them in order; both must reach the same bits. The
second layer's keys and values depend on the first layer's attention output,
so they compare the two attention paths. Prefixes of 256 and 300 rows (two
and three spans) are extended by the verification rounds and prefilled again
in two passes of at most 144 rows, so the row tiles see even and odd span
counts, and one whose last span is the group-1 span run again.
"""
import numpy as np
import pytest

from tests.harness import make_pair, prefix
from workload import QWEN7B

pytestmark = pytest.mark.gpu

SHAPE = QWEN7B.with_layers(2)


@pytest.mark.parametrize("n_audio,n_instr", [(240, 16), (284, 16)])
def test_prefill_equals_incremental_several_spans(n_audio, n_instr):
    print(f"7B shape, 2 layers, prefix {n_audio} + {n_instr}", flush=True)
    _, gpu = make_pair(SHAPE, seed=11, max_requests=2, max_kv_len=1024, max_k=8, oracle=False)
    try:
        _, a_dev, instr = prefix(SHAPE, n_audio, n_instr, 11, 0)
        first, L = gpu.prefill(0, a_dev, instr)
        rng = np.random.default_rng(11)
        committed = [first]
        for _ in range(10):
            c = [int(t) for t in rng.integers(0, SHAPE.vocab, 3)]
            r = gpu.verify(0, c)
            committed += c[:r["accepted_len"]] + [r["correction_token"]]
        kv, root, _ = gpu.state(0)
        assert kv > L
        processed = np.array(list(instr) + committed[:-1], dtype=np.int32)
        first2, kv2 = gpu.prefill(1, a_dev, processed)
        assert kv2 == kv and first2 == root
        for layer in range(SHAPE.n_layers):
            k1, v1 = gpu.read_kv(0, layer, kv)
            k2, v2 = gpu.read_kv(1, layer, kv)
            assert np.array_equal(k1, k2) and np.array_equal(v1, v2), f"layer {layer}"
    finally:
        gpu.close()
