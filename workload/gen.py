"""Seeded synthetic inputs for both the oracle and the GPU path.

Nothing here computes any part of the decoding method.  Weights, audio
embeddings, instruction tokens and candidate corruption are pure functions
of (seed, stream name, index), drawn by the counter-based generator in
synth.c, so any subset (e.g. the first layers of a model) is identical to
the corresponding part of the full set.
"""
import ctypes
import os
import subprocess
from typing import Dict, List, Optional, Sequence

import numpy as np

from .configs import BF16, F32, ModelShape

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libsynth.so")
_lib = None
_MASK = (1 << 64) - 1


def build(force: bool = True) -> str:
    """Compile synth.c into libsynth.so (plain gcc, no GPU code)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-ffp-contract=off", "-fPIC", "-shared",
                               os.path.join(_HERE, "synth.c"), "-o", tmp, "-lm", "-lpthread"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build(force=True)
        lib = ctypes.CDLL(_LIB_PATH)
        lib.synth_normal.argtypes = [ctypes.c_uint64, ctypes.c_double, ctypes.c_int, ctypes.c_void_p,
                                     ctypes.c_int64, ctypes.c_int]
        lib.synth_uniform_int.argtypes = [ctypes.c_uint64, ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64]
        lib.synth_uniform_f64.argtypes = [ctypes.c_uint64, ctypes.c_void_p, ctypes.c_int64]
        _lib = lib
    return _lib


def _threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def stream_key(seed: int, name: str, index: int = 0) -> int:
    """64-bit stream key from (seed, name, index): FNV-1a of the name mixed
    with the seed and index."""
    h = 0xCBF29CE484222325
    for b in name.encode():
        h = ((h ^ b) * 0x100000001B3) & _MASK
    h ^= (seed * 0x9E3779B97F4A7C15) & _MASK
    h = (h * 0xD6E8FEB86659FD93) & _MASK
    h ^= (index + 1) * 0xC2B2AE3D27D4EB4F & _MASK
    return h & _MASK


def normal(key: int, shape, std: float, fmt: str = "f32") -> np.ndarray:
    """N(0, std^2) array.  fmt: 'f32' plain float32, 'bf16r' float32 holding
    bf16-rounded values, 'bf16' uint16 bf16 bit patterns (same values as
    'bf16r')."""
    mode = {"f32": 0, "bf16r": 1, "bf16": 2}[fmt]
    out = np.empty(shape, dtype=np.uint16 if mode == 2 else np.float32)
    _load().synth_normal(key, std, mode, out.ctypes.data, out.size, _threads())
    return out


def uniform_int(key: int, hi: int, n: int) -> np.ndarray:
    out = np.empty(n, dtype=np.int32)
    _load().synth_uniform_int(key, hi, out.ctypes.data, n)
    return out


def uniform_f64(key: int, n: int) -> np.ndarray:
    out = np.empty(n, dtype=np.float64)
    _load().synth_uniform_f64(key, out.ctypes.data, n)
    return out


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (b.astype(np.uint32) << 16).view(np.float32)


def bf16_bits_to_f64(b: np.ndarray) -> np.ndarray:
    """float64 array holding the values of bf16 bit patterns (exact), in row
    blocks on several threads (the 7B-shaped matrices are large)."""
    from concurrent.futures import ThreadPoolExecutor
    b = np.ascontiguousarray(b, dtype=np.uint16)
    out = np.empty(b.shape, dtype=np.float64)
    flat_in, flat_out = b.reshape(-1), out.reshape(-1)
    n = _threads()
    edges = np.linspace(0, flat_in.size, n + 1).astype(np.int64)

    def conv(i):
        lo, hi = edges[i], edges[i + 1]
        flat_out[lo:hi] = (flat_in[lo:hi].astype(np.uint32) << 16).view(np.float32)
    with ThreadPoolExecutor(n) as ex:
        list(ex.map(conv, range(n)))
    return out


def f32_to_bf16_bits(f: np.ndarray) -> np.ndarray:
    """Exact for float32 arrays whose values are bf16-representable."""
    u = np.ascontiguousarray(f, dtype=np.float32).view(np.uint32)
    return (u >> 16).astype(np.uint16)


# ---------------------------------------------------------------------------
# Weights in the canonical tensor order of the C ABI (include/as2d.h).

def weight_spec(shape: ModelShape) -> List[tuple]:
    """[(name, layer, dims, kind)] in canonical order.  kind: 'mat' (matrix
    or embedding, model dtype), 'gain' (RMSNorm gain, float32, ones), 'bias'
    (QKV bias, float32 holding values of the model dtype)."""
    H, F, V, d = shape.hidden, shape.ffn, shape.vocab, shape.head_dim
    nq, nkv = shape.n_q_heads, shape.n_kv_heads
    spec = [("embed", -1, (V, H), "mat")]
    for l in range(shape.n_layers):
        spec += [("attn_norm", l, (H,), "gain"),
                 ("wq", l, (nq * d, H), "mat"),
                 ("wk", l, (nkv * d, H), "mat"),
                 ("wv", l, (nkv * d, H), "mat")]
        if shape.qkv_bias:
            spec += [("bq", l, (nq * d,), "bias"), ("bk", l, (nkv * d,), "bias"),
                     ("bv", l, (nkv * d,), "bias")]
        spec += [("wo", l, (H, nq * d), "mat"),
                 ("mlp_norm", l, (H,), "gain"),
                 ("w_gate", l, (F, H), "mat"),
                 ("w_up", l, (F, H), "mat"),
                 ("w_down", l, (H, F), "mat")]
    spec += [("final_norm", -1, (H,), "gain"), ("lm_head", -1, (V, H), "mat")]
    return spec


def make_tensor(shape: ModelShape, entry, seed: int = 0, fmt: str = "oracle") -> np.ndarray:
    """One weight tensor.  fmt 'oracle': float32 values (bf16-representable
    for bf16 models).  fmt 'device': what the C ABI takes, i.e. uint16 bf16
    bits for matrices of bf16 models, float32 otherwise.  Both carry the
    same values."""
    name, layer, dims, kind = entry
    if kind == "gain":
        return np.ones(dims, dtype=np.float32)
    key = stream_key(seed, name, layer)
    if shape.dtype == F32:
        return normal(key, dims, shape.weight_std, "f32")
    if kind == "mat" and fmt == "device":
        return normal(key, dims, shape.weight_std, "bf16")
    return normal(key, dims, shape.weight_std, "bf16r")


def make_weights(shape: ModelShape, seed: int = 0, fmt: str = "oracle") -> List[np.ndarray]:
    return [make_tensor(shape, e, seed, fmt) for e in weight_spec(shape)]


def weights_dict(shape: ModelShape, tensors: Sequence[np.ndarray]) -> Dict[tuple, np.ndarray]:
    return {(e[0], e[1]): t for e, t in zip(weight_spec(shape), tensors)}


# ---------------------------------------------------------------------------
# Request inputs.

def audio_embeddings(shape: ModelShape, n_audio: int, seed: int = 0, req: int = 0,
                     fmt: str = "oracle") -> np.ndarray:
    """[n_audio, hidden] N(0,1) rows standing in for encoder output.  bf16
    models get bf16-representable values ('device' fmt: uint16 bits)."""
    key = stream_key(seed, "audio", req)
    if shape.dtype == F32:
        return normal(key, (n_audio, shape.hidden), 1.0, "f32")
    return normal(key, (n_audio, shape.hidden), 1.0, "bf16" if fmt == "device" else "bf16r")


def instruction_tokens(shape: ModelShape, n_instr: int, seed: int = 0, req: int = 0) -> np.ndarray:
    return uniform_int(stream_key(seed, "instr", req), shape.vocab, n_instr)


class CandidateSource:
    """Proposals built from a greedy reference stream y_0, y_1, ... (y_0 is
    the token chosen at the end of prefill): the candidate for stream
    position j is y_j, replaced with probability p by a uniform random token.
    The replacement at j is a fixed function of (seed, req, j)."""

    def __init__(self, reference: Sequence[int], vocab: int, p: float, seed: int = 0, req: int = 0,
                 max_len: Optional[int] = None):
        self.ref = np.asarray(reference, dtype=np.int64)
        n = len(self.ref) if max_len is None else max_len
        self.u = uniform_f64(stream_key(seed, "corrupt-u", req), n)
        self.tok = uniform_int(stream_key(seed, "corrupt-tok", req), vocab, n)
        self.p = p

    def candidate(self, j: int) -> int:
        if j < len(self.u) and self.u[j] < self.p:
            return int(self.tok[j])
        return int(self.ref[j])

    def block(self, n_committed: int, k: int) -> List[int]:
        """Candidates after the root y_n: positions n+1 .. n+k."""
        return [self.candidate(j) for j in range(n_committed + 1, n_committed + 1 + k)]


def edited_stream(reference: Sequence[int], vocab: int, p_sub: float, p_ins: float, p_del: float,
                  seed: int = 0, req: int = 0) -> List[int]:
    """A synthetic draft of a reference token stream (the producer's text is
    the target's text with local edits): walking the reference, each token
    is dropped with probability p_del, else replaced by a uniform random
    token with probability p_sub, else kept; after it, a uniform random
    token is inserted with probability p_ins.  Draws are a fixed function
    of (seed, req, position)."""
    n = len(reference)
    u = uniform_f64(stream_key(seed, "edit-u", req), 2 * n)
    tok = uniform_int(stream_key(seed, "edit-tok", req), vocab, 2 * n)
    out = []
    for i, t in enumerate(reference):
        r = u[2 * i]
        if r < p_del:
            pass
        elif r < p_del + p_sub:
            out.append(int(tok[2 * i]))
        else:
            out.append(int(t))
        if u[2 * i + 1] < p_ins:
            out.append(int(tok[2 * i + 1]))
    return out
