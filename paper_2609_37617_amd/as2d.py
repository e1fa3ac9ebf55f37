"""ctypes binding of libas2d.so (include/as2d.h).

Argument marshalling only: every step of the verification path runs in the
library's HIP kernels.  Importing this module does not touch the GPU;
loading the library fails loudly if it has not been built.
"""
import ctypes
import os
from typing import List, Optional, Sequence

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libas2d.so")

OK, EINVAL, ECAPACITY, ESTATE, EHIP, ENUMERIC, ENOMEM = 0, -1, -2, -3, -4, -5, -6
EXEC_EAGER, EXEC_GRAPH, EXEC_PERSISTENT = 0, 1, 2
F32, BF16 = 0, 1

# Every symbol include/as2d.h declares.
EXPORTS = ["as2d_load_weights", "as2d_prefill_kv", "as2d_verify", "as2d_decode_one",
           "as2d_verify_batch", "as2d_set_keep_logits", "as2d_get_logits", "as2d_get_row_tokens",
           "as2d_get_row_margins",
           "as2d_rollback", "as2d_get_state", "as2d_read_kv", "as2d_release_request",
           "as2d_set_exec_mode", "as2d_get_exec_info", "as2d_set_step_trace", "as2d_step_trace_read",
           "as2d_set_timing", "as2d_timing_read", "as2d_timing_reset", "as2d_time_gemm",
           "as2d_stream_bandwidth", "as2d_step_bytes", "as2d_free", "as2d_last_error",
           "as2d_cbuf_create", "as2d_cbuf_free", "as2d_cbuf_publish", "as2d_cbuf_snapshot",
           "as2d_cbuf_read", "as2d_cbuf_n_records", "as2d_cbuf_get_record", "as2d_cursor_init",
           "as2d_cursor_propose", "as2d_cursor_update", "as2d_verify_from_buffer", "as2d_run_decoupled",
           "as2d_set_stream", "as2d_set_cu_budget", "as2d_verify_static"]


class Config(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("hidden", ctypes.c_int32),
                ("n_q_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("ffn", ctypes.c_int32), ("vocab", ctypes.c_int32),
                ("rope_theta", ctypes.c_float), ("rms_eps", ctypes.c_float),
                ("dtype", ctypes.c_int32), ("qkv_bias", ctypes.c_int32),
                ("max_requests", ctypes.c_int32), ("max_kv_len", ctypes.c_int32),
                ("max_k", ctypes.c_int32)]


class VerifyOut(ctypes.Structure):
    _fields_ = [("accepted_len", ctypes.c_int32), ("correction_token", ctypes.c_int32),
                ("kv_len", ctypes.c_int32), ("committed", ctypes.c_int32)]

    def as_dict(self):
        return dict(accepted_len=self.accepted_len, correction_token=self.correction_token,
                    kv_len=self.kv_len, committed=self.committed)


class CbufRecord(ctypes.Structure):
    _fields_ = [("first", ctypes.c_int64), ("count", ctypes.c_int32), ("source_id", ctypes.c_int32),
                ("producer_id", ctypes.c_int32), ("pad", ctypes.c_int32), ("offset", ctypes.c_int64),
                ("publish_ns", ctypes.c_int64), ("confidence", ctypes.c_float), ("pad2", ctypes.c_int32)]


class ReadCursorC(ctypes.Structure):
    _fields_ = [("cursor", ctypes.c_int64), ("floor", ctypes.c_int64), ("radius", ctypes.c_int32),
                ("pad", ctypes.c_int32)]


class Interval(ctypes.Structure):
    _fields_ = [("start_ns", ctypes.c_int64), ("end_ns", ctypes.c_int64), ("kind", ctypes.c_int32),
                ("tokens", ctypes.c_int32)]


class As2dError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"as2d error {code}: {msg}")
        self.code = code


_lib = None
_P = ctypes.c_void_p
_I = ctypes.c_int32


def load_library(path: str = LIB_PATH):
    """Load libas2d.so; raises if it is missing (no fallback path exists)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise FileNotFoundError(f"{path} is not built; run __graft_entry__.build() "
                                f"or python paper_2609_37617_amd/build.py")
    lib = ctypes.CDLL(path)
    lib.as2d_load_weights.argtypes = [ctypes.POINTER(Config), ctypes.POINTER(_P), _I, _P,
                                      ctypes.POINTER(_P)]
    lib.as2d_prefill_kv.argtypes = [_P, _I, _P, _I, _P, _I, ctypes.POINTER(_I), ctypes.POINTER(_I)]
    lib.as2d_verify.argtypes = [_P, _I, _P, _I, ctypes.POINTER(VerifyOut)]
    lib.as2d_verify_static.argtypes = [_P, _I, _P, _I, ctypes.POINTER(VerifyOut)]
    lib.as2d_decode_one.argtypes = [_P, _I, ctypes.POINTER(VerifyOut)]
    lib.as2d_verify_batch.argtypes = [_P, _I, _P, _P, _P, _P]
    lib.as2d_set_keep_logits.argtypes = [_P, _I]
    lib.as2d_get_logits.argtypes = [_P, _I, _P, _I, ctypes.POINTER(_I)]
    lib.as2d_get_row_tokens.argtypes = [_P, _I, _P, _I, ctypes.POINTER(_I)]
    lib.as2d_get_row_margins.argtypes = [_P, _I, _P, _I, ctypes.POINTER(_I)]
    lib.as2d_rollback.argtypes = [_P, _I, _I, _I]
    lib.as2d_get_state.argtypes = [_P, _I, ctypes.POINTER(_I), ctypes.POINTER(_I), ctypes.POINTER(_I)]
    lib.as2d_read_kv.argtypes = [_P, _I, _I, _P, _P, _I]
    lib.as2d_release_request.argtypes = [_P, _I]
    lib.as2d_set_exec_mode.argtypes = [_P, _I]
    lib.as2d_set_step_trace.argtypes = [_P, _I]
    lib.as2d_step_trace_read.argtypes = [_P, _P, ctypes.c_int64, ctypes.POINTER(_I), ctypes.POINTER(_I)]
    lib.as2d_get_exec_info.argtypes = [_P, ctypes.POINTER(_I), ctypes.POINTER(_I)]
    lib.as2d_set_timing.argtypes = [_P, _I]
    lib.as2d_timing_read.argtypes = [_P, _P, _P, _P, _I]
    lib.as2d_timing_reset.argtypes = [_P]
    lib.as2d_time_gemm.argtypes = [_P, _I, _I, _I, ctypes.POINTER(ctypes.c_double)]
    lib.as2d_stream_bandwidth.argtypes = [_P, ctypes.c_int64, _I, ctypes.POINTER(ctypes.c_double)]
    lib.as2d_step_bytes.argtypes = [_P, _I, ctypes.c_int64]
    lib.as2d_step_bytes.restype = ctypes.c_int64
    _L = ctypes.c_int64
    lib.as2d_cbuf_create.argtypes = [_L, ctypes.POINTER(_P)]
    lib.as2d_cbuf_free.argtypes = [_P]
    lib.as2d_cbuf_publish.argtypes = [_P, _P, _I, _I, _I, _L, _L, ctypes.c_float, ctypes.POINTER(_L)]
    lib.as2d_cbuf_snapshot.argtypes = [_P, ctypes.POINTER(_L)]
    lib.as2d_cbuf_read.argtypes = [_P, _L, _I, _P]
    lib.as2d_cbuf_n_records.argtypes = [_P, ctypes.POINTER(_L)]
    lib.as2d_cbuf_get_record.argtypes = [_P, _L, ctypes.POINTER(CbufRecord)]
    lib.as2d_cursor_init.argtypes = [ctypes.POINTER(ReadCursorC), _I]
    lib.as2d_cursor_propose.argtypes = [_P, ctypes.POINTER(ReadCursorC), _L, _I, _P, ctypes.POINTER(_I)]
    lib.as2d_cursor_update.argtypes = [_P, ctypes.POINTER(ReadCursorC), _L, _I, _I, _I]
    lib.as2d_verify_from_buffer.argtypes = [_P, _I, _P, ctypes.POINTER(ReadCursorC), _I, _I,
                                            ctypes.POINTER(VerifyOut), ctypes.POINTER(_I)]
    lib.as2d_run_decoupled.argtypes = [_P, _I, _P, _I, _P, _I, _I, _I, _I, _P, ctypes.POINTER(ReadCursorC), _P,
                                       _P, _I, ctypes.POINTER(_I), ctypes.POINTER(_L), ctypes.POINTER(_I)]
    lib.as2d_set_stream.argtypes = [_P, _P]
    lib.as2d_set_cu_budget.argtypes = [_P, _I]
    lib.as2d_free.argtypes = [_P]
    lib.as2d_free.restype = None
    lib.as2d_last_error.argtypes = [_P]
    lib.as2d_last_error.restype = ctypes.c_char_p
    for name in EXPORTS:
        if name not in ("as2d_free", "as2d_last_error", "as2d_step_bytes"):
            getattr(lib, name).restype = ctypes.c_int
    _lib = lib
    return lib


def _ptr(a: np.ndarray) -> int:
    return a.ctypes.data


class Model:
    """One library context: a loaded target model with its KV slots."""

    def __init__(self, shape, tensors: Sequence[np.ndarray], max_requests: int = 1,
                 max_kv_len: int = 1024, max_k: int = 8, stream: Optional[int] = None):
        """shape: workload.configs.ModelShape; tensors: the canonical list
        in the 'device' format of workload.gen.make_weights."""
        self.lib = load_library()
        self.shape = shape
        cfg = Config(shape.n_layers, shape.hidden, shape.n_q_heads, shape.n_kv_heads, shape.head_dim,
                     shape.ffn, shape.vocab, shape.rope_theta, shape.rms_eps, shape.dtype,
                     int(shape.qkv_bias), max_requests, max_kv_len, max_k)
        self.cfg = cfg
        self._keep = [np.ascontiguousarray(t) for t in tensors]
        arr = (_P * len(self._keep))(*[_ptr(t) for t in self._keep])
        ctx = _P()
        rc = self.lib.as2d_load_weights(ctypes.byref(cfg), arr, len(self._keep), stream, ctypes.byref(ctx))
        self._keep = None
        if rc != OK:
            raise As2dError(rc, self.lib.as2d_last_error(None).decode())
        self.ctx = ctx

    def close(self):
        if getattr(self, "ctx", None):
            self.lib.as2d_free(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def _check(self, rc):
        if rc != OK:
            raise As2dError(rc, self.lib.as2d_last_error(self.ctx).decode())

    def call(self, name, *args):
        """Raw call returning the status code (for error-path tests)."""
        return getattr(self.lib, name)(self.ctx, *args)

    def prefill(self, req: int, audio: np.ndarray, instr: Sequence[int]):
        audio = np.ascontiguousarray(audio)
        instr = np.ascontiguousarray(instr, dtype=np.int32)
        first, kv = _I(), _I()
        n_audio = audio.shape[0] if audio.size else 0
        self._check(self.lib.as2d_prefill_kv(self.ctx, req, _ptr(audio) if n_audio else None, n_audio,
                                             _ptr(instr) if len(instr) else None, len(instr),
                                             ctypes.byref(first), ctypes.byref(kv)))
        return first.value, kv.value

    def verify(self, req: int, cands: Sequence[int], k: Optional[int] = None) -> dict:
        c = np.ascontiguousarray(cands, dtype=np.int32)
        k = len(c) if k is None else k
        out = VerifyOut()
        self._check(self.lib.as2d_verify(self.ctx, req, _ptr(c) if c.size else None, k, ctypes.byref(out)))
        return out.as_dict()

    def verify_static(self, req: int, cands: Sequence[int]) -> dict:
        """as2d_verify_static: the same call with the pass's buffers in the
        library's static scratch array (allocates nothing)."""
        c = np.ascontiguousarray(cands, dtype=np.int32)
        out = VerifyOut()
        self._check(self.lib.as2d_verify_static(self.ctx, req, _ptr(c) if c.size else None, len(c),
                                                ctypes.byref(out)))
        return out.as_dict()

    def decode_one(self, req: int) -> dict:
        out = VerifyOut()
        self._check(self.lib.as2d_decode_one(self.ctx, req, ctypes.byref(out)))
        return out.as_dict()

    def verify_batch(self, reqs: Sequence[int], cands: Sequence[Sequence[int]]) -> List[dict]:
        n = len(reqs)
        r = np.ascontiguousarray(reqs, dtype=np.int32)
        ks = np.array([len(c) for c in cands], dtype=np.int32)
        flat = np.ascontiguousarray(np.concatenate([np.asarray(c, dtype=np.int32) for c in cands])
                                    if ks.sum() else np.zeros(1, np.int32), dtype=np.int32)
        outs = (VerifyOut * n)()
        self._check(self.lib.as2d_verify_batch(self.ctx, n, _ptr(r), _ptr(flat), _ptr(ks), outs))
        return [o.as_dict() for o in outs]

    def verify_batch_status(self, reqs: Sequence[int], cands: Sequence[Sequence[int]]):
        """as2d_verify_batch returning (status, per-request results) without
        raising: with AS2D_ENUMERIC the requests whose logits are finite are
        committed and the others report accepted_len -1."""
        n = len(reqs)
        r = np.ascontiguousarray(reqs, dtype=np.int32)
        ks = np.array([len(c) for c in cands], dtype=np.int32)
        flat = np.ascontiguousarray(np.concatenate([np.asarray(c, dtype=np.int32) for c in cands])
                                    if ks.sum() else np.zeros(1, np.int32), dtype=np.int32)
        outs = (VerifyOut * n)()
        rc = self.lib.as2d_verify_batch(self.ctx, n, _ptr(r), _ptr(flat), _ptr(ks), outs)
        return rc, [o.as_dict() for o in outs]

    def set_keep_logits(self, on: bool):
        self._check(self.lib.as2d_set_keep_logits(self.ctx, int(on)))

    def logits(self, req: int, max_rows: int = 32) -> np.ndarray:
        buf = np.empty((max_rows, self.shape.vocab), dtype=np.float32)
        n = _I()
        self._check(self.lib.as2d_get_logits(self.ctx, req, _ptr(buf), max_rows, ctypes.byref(n)))
        return buf[:n.value].copy()

    def row_tokens(self, req: int, max_rows: int = 32) -> List[int]:
        buf = np.empty(max_rows, dtype=np.int32)
        n = _I()
        self._check(self.lib.as2d_get_row_tokens(self.ctx, req, _ptr(buf), max_rows, ctypes.byref(n)))
        return [int(t) for t in buf[:n.value]]

    def row_margins(self, req: int, max_rows: int = 32) -> np.ndarray:
        """Top-2 logit margin of every row of the last call (device-side)."""
        buf = np.empty(max_rows, dtype=np.float32)
        n = _I()
        self._check(self.lib.as2d_get_row_margins(self.ctx, req, _ptr(buf), max_rows, ctypes.byref(n)))
        return buf[:n.value].copy()

    def rollback(self, req: int, kv_len: int, root: int):
        self._check(self.lib.as2d_rollback(self.ctx, req, kv_len, root))

    def state(self, req: int):
        kv, root, com = _I(), _I(), _I()
        self._check(self.lib.as2d_get_state(self.ctx, req, ctypes.byref(kv), ctypes.byref(root),
                                            ctypes.byref(com)))
        return kv.value, root.value, com.value

    def read_kv(self, req: int, layer: int, n_tok: int):
        s = self.shape
        k = np.empty((s.n_kv_heads, n_tok, s.head_dim), dtype=np.float32)
        v = np.empty_like(k)
        self._check(self.lib.as2d_read_kv(self.ctx, req, layer, _ptr(k), _ptr(v), n_tok))
        return k, v

    def release(self, req: int):
        self._check(self.lib.as2d_release_request(self.ctx, req))

    def set_exec_mode(self, mode: int):
        """EXEC_EAGER, EXEC_GRAPH or EXEC_PERSISTENT (include/as2d.h)."""
        self._check(self.lib.as2d_set_exec_mode(self.ctx, mode))

    def exec_info(self):
        mode, grid = _I(), _I()
        self._check(self.lib.as2d_get_exec_info(self.ctx, ctypes.byref(mode), ctypes.byref(grid)))
        return mode.value, grid.value

    def set_step_trace(self, on: bool):
        self._check(self.lib.as2d_set_step_trace(self.ctx, int(on)))

    def step_trace(self) -> np.ndarray:
        """[grid, n_phase, 3] wall-clock stamps of the last persistent pass."""
        n = 1 << 22
        buf = np.zeros(n, dtype=np.int64)
        g, ph = _I(), _I()
        self._check(self.lib.as2d_step_trace_read(self.ctx, _ptr(buf), n, ctypes.byref(g), ctypes.byref(ph)))
        return buf[:g.value * ph.value * 3].reshape(g.value, ph.value, 3)

    def set_timing(self, on: bool):
        self._check(self.lib.as2d_set_timing(self.ctx, int(on)))

    def timing_reset(self):
        self._check(self.lib.as2d_timing_reset(self.ctx))

    def timing(self) -> dict:
        names = ctypes.create_string_buffer(32 * 16)
        ms = (ctypes.c_double * 16)()
        cnt = (ctypes.c_int64 * 16)()
        n = self.lib.as2d_timing_read(self.ctx, names, ms, cnt, 16)
        out = {}
        for i in range(n):
            nm = names.raw[32 * i:32 * i + 32].split(b"\0")[0].decode()
            out[nm] = (ms[i], cnt[i])
        return out

    def time_gemm(self, which: int, rows: int, reps: int) -> float:
        """Average microseconds of one GEMM launch (0 QKV, 1 O, 2 gate/up,
        3 down, 4 LM head); measurement only, clobbers activations."""
        us = ctypes.c_double()
        self._check(self.lib.as2d_time_gemm(self.ctx, which, rows, reps, ctypes.byref(us)))
        return us.value

    def stream_bandwidth(self, nbytes: int = 1 << 30, reps: int = 10) -> float:
        """Achievable read bandwidth (GB/s) of a plain streaming kernel."""
        gbps = ctypes.c_double()
        self._check(self.lib.as2d_stream_bandwidth(self.ctx, nbytes, reps, ctypes.byref(gbps)))
        return gbps.value

    def set_stream(self, stream: Optional[int]):
        """Rebind to a HIP stream handle (None: a stream of its own)."""
        self._check(self.lib.as2d_set_stream(self.ctx, stream))

    def set_cu_budget(self, cus: int):
        """Size the balanced GEMM grids for `cus` compute units (0: all the
        stream's)."""
        self._check(self.lib.as2d_set_cu_budget(self.ctx, cus))

    def step_bytes(self, rows: int, kv_keys: int) -> int:
        return int(self.lib.as2d_step_bytes(self.ctx, rows, kv_keys))


def _rc(rc, what):
    if rc != OK:
        raise As2dError(rc, what)


class CandidateBuffer:
    """The library's candidate buffer (one producer, any readers)."""

    def __init__(self, capacity: int):
        self.lib = load_library()
        self.h = _P()
        _rc(self.lib.as2d_cbuf_create(capacity, ctypes.byref(self.h)), "as2d_cbuf_create")

    def close(self):
        if getattr(self, "h", None):
            self.lib.as2d_cbuf_free(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def publish(self, tokens, source_id=0, producer_id=0, offset=-1, publish_ns=0, confidence=float("nan")) -> int:
        t = np.ascontiguousarray(tokens, dtype=np.int32)
        n = ctypes.c_int64()
        _rc(self.lib.as2d_cbuf_publish(self.h, _ptr(t) if t.size else None, len(t), source_id, producer_id, offset,
                                       publish_ns, confidence, ctypes.byref(n)), "as2d_cbuf_publish")
        return n.value

    def snapshot(self) -> int:
        n = ctypes.c_int64()
        _rc(self.lib.as2d_cbuf_snapshot(self.h, ctypes.byref(n)), "as2d_cbuf_snapshot")
        return n.value

    def read(self, start: int, n: int) -> List[int]:
        out = np.empty(max(n, 1), dtype=np.int32)
        _rc(self.lib.as2d_cbuf_read(self.h, start, n, _ptr(out)), "as2d_cbuf_read")
        return [int(v) for v in out[:n]]

    def records(self) -> List[dict]:
        n = ctypes.c_int64()
        _rc(self.lib.as2d_cbuf_n_records(self.h, ctypes.byref(n)), "as2d_cbuf_n_records")
        out = []
        for i in range(n.value):
            r = CbufRecord()
            _rc(self.lib.as2d_cbuf_get_record(self.h, i, ctypes.byref(r)), "as2d_cbuf_get_record")
            out.append(dict(first=r.first, count=r.count, source_id=r.source_id, producer_id=r.producer_id,
                            offset=r.offset, publish_ns=r.publish_ns, confidence=r.confidence))
        return out


class ReadCursor:
    """A read cursor over a CandidateBuffer (the library's alignment rule)."""

    def __init__(self, radius: int = 8):
        self.lib = load_library()
        self.c = ReadCursorC()
        _rc(self.lib.as2d_cursor_init(ctypes.byref(self.c), radius), "as2d_cursor_init")

    @property
    def cursor(self) -> int:
        return self.c.cursor

    @property
    def floor(self) -> int:
        return self.c.floor

    def propose(self, buf: CandidateBuffer, snapshot: int, k_max: int) -> List[int]:
        out = np.empty(max(k_max, 1), dtype=np.int32)
        k = _I()
        _rc(self.lib.as2d_cursor_propose(buf.h, ctypes.byref(self.c), snapshot, k_max, _ptr(out), ctypes.byref(k)),
            "as2d_cursor_propose")
        return [int(v) for v in out[:k.value]]

    def update(self, buf: CandidateBuffer, snapshot: int, k: int, accepted: int, token: int):
        _rc(self.lib.as2d_cursor_update(buf.h, ctypes.byref(self.c), snapshot, k, accepted, token),
            "as2d_cursor_update")

    def verify_from_buffer(self, model: "Model", req: int, buf: CandidateBuffer, budget: int, max_commit: int):
        """One decoding step of `model`'s request `req` from the buffer;
        returns (verify result dict, candidates verified)."""
        out = VerifyOut()
        k = _I()
        model._check(self.lib.as2d_verify_from_buffer(model.ctx, req, buf.h, ctypes.byref(self.c), budget,
                                                      max_commit, ctypes.byref(out), ctypes.byref(k)))
        return out.as_dict(), k.value


def run_decoupled(target: Model, treq: int, drafter: Model, dreq: int, draft: Sequence[int], budget: int,
                  n_commit: int, concurrent: bool, radius: int = 8, log_cap: int = 1 << 16) -> dict:
    """as2d_run_decoupled on a fresh buffer and cursor.  Returns the
    committed tokens, the stage intervals [(start_ns, end_ns, kind,
    tokens)] (kind 0 producer step, 1 verifier call), the run's total ns
    and the producer's status."""
    lib = load_library()
    d = np.ascontiguousarray(draft, dtype=np.int32)
    buf = CandidateBuffer(max(len(d), 1))
    cur = ReadCursor(radius)
    out = np.empty(n_commit, dtype=np.int32)
    log = (Interval * log_cap)()
    n_log, total, prc = _I(), ctypes.c_int64(), _I()
    rc = lib.as2d_run_decoupled(target.ctx, treq, drafter.ctx, dreq, _ptr(d) if d.size else None, len(d), budget,
                                n_commit, int(concurrent), buf.h, ctypes.byref(cur.c), _ptr(out), log, log_cap,
                                ctypes.byref(n_log), ctypes.byref(total), ctypes.byref(prc))
    target._check(rc)
    iv = [(log[i].start_ns, log[i].end_ns, log[i].kind, log[i].tokens) for i in range(n_log.value)]
    res = dict(committed=[int(t) for t in out], intervals=iv, total_ns=total.value, producer_rc=prc.value,
               published=buf.snapshot(), records=len(buf.records()))
    buf.close()
    return res

