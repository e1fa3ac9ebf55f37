"""Shared helpers of the parity tests: build the oracle and the GPU model
on the same seeded inputs and drive both through verification rounds.

The near-tie protocol: logits are compared within a tolerance; accepted
lengths and committed tokens must match exactly unless the first row whose
greedy decision differs has an oracle top-2 margin <= 0.05, in which case
the oracle is teacher-forced onto the GPU's commit (the paper records such
near-tied top-1 differences rather than hiding them, Appendix F.6).
"""
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from oracle import OracleModel, greedy          # noqa: E402
from workload import gen                        # noqa: E402
from workload.configs import BF16               # noqa: E402

NEAR_TIE_MARGIN = 0.05


def logit_tol(shape):
    return 3e-2 if shape.dtype == BF16 else 1e-4


def ensure_built():
    from paper_2609_37617_amd import as2d
    if not os.path.exists(as2d.LIB_PATH):
        from paper_2609_37617_amd import build
        build.build()
    if not os.path.exists(gen._LIB_PATH):
        gen.build()


def make_pair(shape, seed=0, max_requests=1, max_kv_len=512, max_k=8, oracle=True):
    """(oracle or None, GPU model) with identical weights."""
    from paper_2609_37617_amd import as2d
    ensure_built()
    dev = gen.make_weights(shape, seed, fmt="device")
    gpu = as2d.Model(shape, dev, max_requests=max_requests, max_kv_len=max_kv_len, max_k=max_k)
    del dev
    om = None
    if oracle:
        om = OracleModel(shape, gen.weights_dict(shape, gen.make_weights(shape, seed)), capacity=max_kv_len)
    return om, gpu


class DeviceValues:
    """Read-only mapping {(name, layer): float64 tensor} over the canonical
    tensors in the C ABI's format (workload.gen.make_weights(fmt="device")):
    bf16 bit patterns become their exact float64 values when read, so the
    oracle and the GPU are built from the very same arrays."""

    def __init__(self, shape, tensors):
        self.w = gen.weights_dict(shape, tensors)

    def __getitem__(self, key):
        t = self.w[key]
        return gen.bf16_bits_to_f64(t) if t.dtype == np.uint16 else np.asarray(t, dtype=np.float64)


def full_pair(shape, seed=0, max_requests=1, max_kv_len=1024, max_k=8):
    """(oracle, GPU model) of a full-size shape from one set of generated
    weights: the GPU model is loaded first, then the oracle converts the
    same arrays to float64 one tensor at a time."""
    import time
    from paper_2609_37617_amd import as2d
    ensure_built()
    t0 = time.time()
    dev = gen.make_weights(shape, seed, fmt="device")
    gpu = as2d.Model(shape, dev, max_requests=max_requests, max_kv_len=max_kv_len, max_k=max_k)
    om = OracleModel(shape, DeviceValues(shape, dev), capacity=max_kv_len)
    del dev
    log(f"[{shape.name}] weights generated, loaded on the GPU and held by the oracle in {time.time() - t0:.1f}s")
    return om, gpu


def log(msg):
    """Progress line (long full-depth tests print one per stage)."""
    print(msg, flush=True)


def prefix(shape, n_audio, n_instr, seed=0, req=0):
    return (gen.audio_embeddings(shape, n_audio, seed, req, fmt="oracle"),
            gen.audio_embeddings(shape, n_audio, seed, req, fmt="device"),
            gen.instruction_tokens(shape, n_instr, seed, req))


def oracle_prefill(om, audio, instr, chunk=2048):
    """The oracle's prefill taken through its forward in causal row chunks:
    row t attends to positions <= t either way, so this is the same
    arithmetic as one forward over the whole prefix, with temporaries of
    chunk x prefix rows instead of prefix x prefix (long prefixes)."""
    om.reset()
    x = np.concatenate([np.asarray(audio, dtype=np.float64).reshape(-1, om.s.hidden),
                        om.embed_tokens(instr)], axis=0)
    T = x.shape[0]
    om._check_capacity(T)
    for c0 in range(0, T, chunk):
        c1 = min(T, c0 + chunk)
        rows = np.array([c1 - c0 - 1]) if c1 == T else np.array([], dtype=np.int64)
        logits = om.forward(x[c0:c1], c0, logit_rows=rows)
        if T > chunk:
            log(f"  oracle prefill: rows {c0}..{c1 - 1} of {T}")
    om.last_logits = logits
    om.root = greedy(logits[0])
    om.kv_len = om.prefix_len = T
    return om.root, om.kv_len


def snapshot(om):
    """The oracle's decoding state.  Shallow: the oracle never writes into a
    cache array (appending and truncating both make new arrays or views),
    so holding the per-layer arrays keeps their contents."""
    return (list(om.k_cache), list(om.v_cache), om.kv_len, om.root)


def restore(om, snap):
    om.k_cache, om.v_cache, om.kv_len, om.root = list(snap[0]), list(snap[1]), snap[2], snap[3]


def teacher_force(om, snap, cands, a, corr):
    """Put the oracle in the state of committing cands[:a] + [corr] from snap."""
    restore(om, snap)
    L0 = om.kv_len
    om.forward(om.embed_tokens([om.root] + list(cands[:a])), L0, logit_rows=np.array([0]))
    om.kv_len = L0 + a + 1
    for l in range(om.s.n_layers):
        om.k_cache[l] = om.k_cache[l][:, :om.kv_len]
        om.v_cache[l] = om.v_cache[l][:, :om.kv_len]
    om.root = int(corr)


class Stats:
    def __init__(self):
        self.rounds = 0
        self.near_ties = 0
        self.max_err = 0.0
        self.committed = 0


def parity_round(om, gpu, req, cands, k, tol, stats, check_logits=True):
    """One verify call on both sides; asserts the protocol; returns the
    GPU result (the oracle follows the GPU's commit)."""
    snap = snapshot(om)
    ro = om.verify(cands, k)
    rg = gpu.verify(req, cands[:k], k)
    check_round(om, snap, ro, rg, gpu.row_tokens(req), gpu.logits(req) if check_logits else None,
                cands, k, tol, stats, gpu.row_margins(req))
    return rg


def check_round(om, snap, ro, rg, toks, lg, cands, k, tol, stats, margins=None):
    """The near-tie protocol for one request's verify result rg (GPU row
    tokens toks, logits lg or None, device top-2 margins or None) against
    the oracle's ro from state snap."""
    if lg is not None:
        assert lg.shape == ro["logits"].shape
        err = float(np.max(np.abs(lg.astype(np.float64) - ro["logits"])))
        stats.max_err = max(stats.max_err, err)
        assert err <= tol, f"logit error {err} > {tol}"
        # the GPU's greedy tokens are the arg-max of its own logits (same precision)
        assert toks == [int(np.argmax(r)) for r in lg]
        if margins is not None:
            # the device's top-2 margin is that of its own logits, exactly
            top = np.sort(lg, axis=1)
            assert np.array_equal(margins, top[:, -1] - top[:, -2])
    stats.rounds += 1
    if (rg["accepted_len"], rg["correction_token"]) != (ro["accepted_len"], ro["correction_token"]):
        i = next(j for j in range(k + 1) if toks[j] != ro["tokens"][j])
        assert i <= min(ro["accepted_len"], rg["accepted_len"]), "divergence after the decision row"
        m = ro["margins"][i]
        assert m <= NEAR_TIE_MARGIN, f"decision differs at row {i} with oracle margin {m}"
        stats.near_ties += 1
        teacher_force(om, snap, cands, rg["accepted_len"], rg["correction_token"])
    else:
        assert toks[:rg["accepted_len"] + 1] == ro["tokens"][:ro["accepted_len"] + 1]
    assert rg["kv_len"] == om.kv_len
    stats.committed += rg["accepted_len"] + 1


def compare_kv(om, gpu, req, layer, n_tok, tol):
    k_g, v_g = gpu.read_kv(req, layer, n_tok)
    k_o, v_o = om.kv(layer)
    ek = float(np.max(np.abs(k_g - k_o[:, :n_tok])))
    ev = float(np.max(np.abs(v_g - v_o[:, :n_tok])))
    assert ek <= tol and ev <= tol, (ek, ev)
    return ek, ev
