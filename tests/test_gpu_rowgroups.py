"""Prefill through the staged GEMMs gives the same bits whatever the row
grouping: groups of 3 row tiles with two tile pairs per wave on every
matrix, a mix of 3 tiles for gate/up, 2 for QKV and 1 for O and down, the
default (3 tiles for gate/up, 1 elsewhere), and single-tile groups
everywhere.  Row grouping only changes which
workgroup computes which rows, never the order of a sum.  7B shape, two
layers (the second layer's KV depends on every GEMM of the first), the
782-row prefix (passes of 144 rows and one of 62); compares both layers'
KV, the first token and the logits of one decode step after the prefill."""
import numpy as np
import pytest

from tests.harness import ensure_built, prefix
from workload import QWEN7B, gen

pytestmark = pytest.mark.gpu

SHAPE = QWEN7B.with_layers(2)
# least grid for row groups of 2-3 tiles: 0 -> always 3 tiles; 448 -> groups
# of 2 for QKV; 700 -> the library's default; 1e5 -> always 1 tile
SETTINGS = (0, 448, 700, 100000)


@pytest.fixture(scope="module")
def weights():
    ensure_built()
    return gen.make_weights(SHAPE, 0, fmt="device")


def run(weights, rg_grid, monkeypatch):
    from paper_2609_37617_amd import as2d
    monkeypatch.setenv("AS2D_RG_GRID", str(rg_grid))   # read when the model is created
    m = as2d.Model(SHAPE, weights, max_requests=1, max_kv_len=1024, max_k=8)
    try:
        _, a_dev, instr = prefix(SHAPE, 750, 32)
        first, L = m.prefill(0, a_dev, instr)
        kv = [m.read_kv(0, layer, L) for layer in range(SHAPE.n_layers)]
        m.set_keep_logits(True)
        out = m.decode_one(0)
        lg = m.logits(0, 1).copy()
    finally:
        m.close()
    return first, L, kv, out, lg


def test_prefill_bits_independent_of_row_groups(weights, monkeypatch):
    ref = None
    for g in SETTINGS:
        print(f"row-group grid threshold {g}", flush=True)
        got = run(weights, g, monkeypatch)
        if ref is None:
            ref = got
            continue
        first, L, kv, out, lg = got
        assert (first, L) == ref[:2], g
        for layer in range(SHAPE.n_layers):
            assert np.array_equal(kv[layer][0], ref[2][layer][0]), (g, layer)
            assert np.array_equal(kv[layer][1], ref[2][layer][1]), (g, layer)
        assert out == ref[3], g
        assert np.array_equal(lg, ref[4]), g
