"""as2d_verify_static (the pass's buffers in the library's static scratch
array, no allocation) against as2d_verify through the C ABI: two calls in a
row, the second with fewer candidates (it finds the first call's contents
in the array), give the same outcome, state, row tokens, margins and
logits bit for bit; a pass too large for the array is refused with
AS2D_ECAPACITY and leaves the request untouched."""
import numpy as np
import pytest

from tests.harness import make_pair, prefix
from workload import QWEN7B, TINY, TINY_BF16

pytestmark = pytest.mark.gpu


def run(gpu, req, calls, static):
    out = []
    for c in calls:
        r = gpu.verify_static(req, c) if static else gpu.verify(req, c)
        out.append((r, gpu.state(req), gpu.row_tokens(req), gpu.row_margins(req), gpu.logits(req)))
    return out


@pytest.mark.parametrize("shape", [TINY, TINY_BF16, QWEN7B.with_layers(2)], ids=lambda s: s.name)
def test_static_verify_equals_verify(shape):
    _, gpu = make_pair(shape, seed=0, max_requests=2, max_kv_len=1152, max_k=16, oracle=False)
    gpu.set_keep_logits(True)
    n_audio = 750 if shape.n_layers == 2 else 96
    _, a_dev, instr = prefix(shape, n_audio, 32, seed=1)
    first, L = gpu.prefill(0, a_dev, instr)
    ref = [gpu.decode_one(0)["correction_token"] for _ in range(12)]
    gpu.rollback(0, L, first)
    calls = [ref[:6] + [(ref[6] + 1) % shape.vocab, ref[7]], ref[7:10]]   # k = 8, then k = 3
    a = run(gpu, 0, calls, static=False)
    gpu.rollback(0, L, first)
    b = run(gpu, 0, calls, static=True)
    for (ra, sa, ta, ma, la), (rb, sb, tb, mb, lb) in zip(a, b):
        assert ra == rb and sa == sb and ta == tb
        assert np.array_equal(ma, mb) and np.array_equal(la, lb)
    assert a[0][0]["accepted_len"] == 6
    gpu.close()


def test_static_verify_refuses_a_pass_beyond_the_array():
    from paper_2609_37617_amd import as2d
    shape = QWEN7B.with_layers(1)
    _, gpu = make_pair(shape, seed=0, max_requests=1, max_kv_len=16064, max_k=8, oracle=False)
    _, a_dev, instr = prefix(shape, 16000, 32, seed=2)     # 126 spans of 128 keys: about 36 MiB in all
    first, L = gpu.prefill(0, a_dev, instr)
    with pytest.raises(as2d.As2dError) as e:
        gpu.verify_static(0, [1, 2, 3])
    assert e.value.code == as2d.ECAPACITY and "static scratch" in str(e.value)
    assert gpu.state(0) == (L, first, 0)
    r = gpu.verify(0, [1, 2, 3])           # the regular call still runs
    assert r["kv_len"] == L + r["accepted_len"] + 1
    gpu.close()
