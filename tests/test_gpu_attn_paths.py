"""Every attention path of the verification step gives the same bits.

A slot capacity of at most 16 spans (2,048 keys) has the span kernel's last
item of each row block merge that block's span states; a larger capacity
merges them in the wave-per-row merge kernel.  The span kernel takes blocks
of one or two row tiles (chosen per launch, or fixed at context creation by
AS2D_ATTN_RT), and runs of several spans per workgroup once the items
outnumber its grid.  Every combination must reach the result of the others
bit for bit (logits, outcome and the appended KV): 7B shape, two layers, one
request verifying k = 8 after a prefix of 900 tokens (8 spans of one-tile
blocks, one workgroup each: in a 1,024-key slot merged by the last item, in
an 8,192-key slot by the merge kernel) and of 4,500 tokens (36 spans: runs
of two spans with two-tile blocks, of three with one-tile blocks).
"""
import os

import numpy as np
import pytest

from tests.harness import make_pair, prefix
from workload import QWEN7B

pytestmark = pytest.mark.gpu

SHAPE = QWEN7B.with_layers(2)
K = 8


def run_once(max_kv_len, n_audio, rt=None, seed=5):
    """Prefill, one verification of K random candidates; (outcome, logits,
    last layer's K and V over the prefix and the appended rows)."""
    old = os.environ.pop("AS2D_ATTN_RT", None)
    if rt is not None:
        os.environ["AS2D_ATTN_RT"] = str(rt)
    try:
        _, gpu = make_pair(SHAPE, seed=seed, max_kv_len=max_kv_len, max_k=K, oracle=False)
    finally:
        os.environ.pop("AS2D_ATTN_RT", None)
        if old is not None:
            os.environ["AS2D_ATTN_RT"] = old
    try:
        gpu.set_keep_logits(True)
        _, a_dev, instr = prefix(SHAPE, n_audio, 16, seed, 0)
        gpu.prefill(0, a_dev, instr)
        L = n_audio + 16
        cands = [int(t) for t in np.random.default_rng(seed).integers(0, SHAPE.vocab, K)]
        out = gpu.verify(0, cands)
        return out, gpu.logits(0).copy(), gpu.read_kv(0, SHAPE.n_layers - 1, L + K + 1)
    finally:
        gpu.close()


def same(a, b, what):
    (oa, la, ka), (ob, lb, kb) = a, b
    assert oa == ob, what
    assert np.array_equal(la, lb), what
    assert np.array_equal(ka[0], kb[0]) and np.array_equal(ka[1], kb[1]), what


def test_merge_in_span_kernel_equals_merge_kernel():
    print("900-token prefix: slot of 1,024 keys vs 8,192 keys", flush=True)
    same(run_once(1024, 884), run_once(8192, 884), "merge paths")


def test_block_sizes_and_runs_agree():
    print("4,500-token prefix: blocks chosen per launch, one tile, two tiles", flush=True)
    ref = run_once(4608, 4484)
    for rt in (1, 2):
        same(run_once(4608, 4484, rt=rt), ref, f"AS2D_ATTN_RT={rt}")
