"""Plain float64 CPU oracle of the target model and its greedy verification.

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).  Slow and obvious on
purpose: every step is the textbook definition, in float64, with no blocking
or fusion.

What it computes (paper: AS2D, arXiv 2609.37617):
  * The greedy target reference: y_{n+1} = g(kappa_n), kappa_{n+1} =
    F(kappa_n, y_{n+1}), with deterministic tie-breaking (Appendix C.4,
    Eq. reference-transition; Appendix A.1, Eq. exact-output).  g is the
    arg-max of the target's logits, ties to the lowest token id.
  * A verification call: one known target root followed by up to b
    candidates, processed at consecutive positions under the committed
    prefix; only the longest prefix of candidates equal to the target's
    greedy tokens is committed, followed by the target's own correction,
    and rejected cache entries are removed (Section 4.2 "Target
    verification"; Appendix C.2 "Verification and state repair"; Appendix
    C.4 requirements 1-2).
  * The known-root convention: the correction (or bonus token after full
    acceptance) is not processed at once; it becomes the root of the next
    call (Appendix C.2; Appendix D.1.1 "Runtime state and timing").
  * A K1 (target-only) step is a verification call with no candidates
    (Appendix C.2).
  * Prefill: audio rows and instruction tokens processed causally into the
    KV cache; the last row's greedy token is the first root (Appendix A.1;
    Appendix C.2).

The target architecture is a decoder-only transformer of the Qwen2 family
(the paper's targets are Qwen3-ASR and Qwen2.5-Omni language models,
Section 5.1): pre-RMSNorm, grouped-query attention with rotary position
embedding (rotate-half convention), SwiGLU MLP, untied LM head.  The paper
does not spell these layers out; they are the standard definitions.
"""
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

F64 = np.float64


def to_f64(a):
    """float64 copy of an array (a plain cast, done in row blocks on
    several threads because the matrices are large)."""
    a = np.asarray(a)
    if a.dtype == F64:
        return a
    out = np.empty(a.shape, dtype=F64)
    if a.ndim == 0 or a.shape[0] < 64:
        out[...] = a
        return out
    n = min(16, os.cpu_count() or 1)
    edges = np.linspace(0, a.shape[0], n + 1).astype(int)
    with ThreadPoolExecutor(n) as ex:
        list(ex.map(lambda i: np.copyto(out[edges[i]:edges[i + 1]], a[edges[i]:edges[i + 1]]), range(n)))
    return out


def rms_norm(x, gain, eps):
    """x / sqrt(mean(x^2) + eps) * gain, per row."""
    x = np.asarray(x, dtype=F64)
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * np.asarray(gain, dtype=F64)


def rope(x, pos, theta):
    """Rotary embedding, rotate-half convention.  x: [T, heads, d]; pos: [T].
    Dimension pairs (i, i + d/2) rotate by angle pos * theta^(-2i/d)."""
    x = np.asarray(x, dtype=F64)
    d = x.shape[-1]
    half = d // 2
    inv_freq = np.power(F64(theta), -2.0 * np.arange(half, dtype=F64) / d)
    ang = np.asarray(pos, dtype=F64)[:, None] * inv_freq[None, :]
    cos = np.cos(ang)[:, None, :]
    sin = np.sin(ang)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * cos - x2 * sin, x2 * cos + x1 * sin], axis=-1)


def silu(x):
    return x / (1.0 + np.exp(-x))


def softmax(s):
    s = s - np.max(s, axis=-1, keepdims=True)
    e = np.exp(s)
    return e / np.sum(e, axis=-1, keepdims=True)


def attention(q, k_cache, v_cache, q_pos):
    """Causal grouped-query attention.
    q: [T, n_q, d] queries at positions q_pos [T];
    k_cache, v_cache: [n_kv, S, d], the entry at index j holds position j.
    Query head h reads KV head floor(h * n_kv / n_q); row t sees keys
    j <= q_pos[t].  Returns [T, n_q, d].

    The heads are independent; for large score matrices they are computed
    on several threads (each head's arithmetic is the same either way, and
    each writes only its own slice of the output)."""
    T, n_q, d = q.shape
    n_kv = k_cache.shape[0]
    out = np.zeros((T, n_q, d), dtype=F64)
    j = np.arange(k_cache.shape[1])

    def head(h):
        g = h * n_kv // n_q
        s = (q[:, h, :] @ k_cache[g].T) / np.sqrt(F64(d))            # [T, S]
        s = np.where(j[None, :] <= np.asarray(q_pos)[:, None], s, -np.inf)
        out[:, h, :] = softmax(s) @ v_cache[g]

    if T * k_cache.shape[1] < (1 << 20):
        for h in range(n_q):
            head(h)
    else:
        with ThreadPoolExecutor(min(n_q, os.cpu_count() or 1, 16)) as ex:
            list(ex.map(head, range(n_q)))
    return out


def greedy(logits_row):
    """The target's greedy token: arg-max, lowest token id on ties.
    A non-finite logit row is an error."""
    row = np.asarray(logits_row)
    if not np.all(np.isfinite(row)):
        raise FloatingPointError("non-finite logits")
    return int(np.argmax(row))  # numpy returns the first maximal index


def top2_margin(logits_row):
    """Gap between the largest and second-largest logit."""
    row = np.asarray(logits_row, dtype=F64)
    if row.size < 2:
        return np.inf
    top = np.partition(row, -2)[-2:]
    return float(top[1] - top[0])


def verify_block(target_tokens, cands, k):
    """Greedy verification of one block (Section 4.2; Appendix C.2):
    target_tokens[i] is the target's greedy token after the root and the
    first i candidates (i = 0..k).  Returns (accepted_len, correction):
    accepted_len a is the first i < k with cands[i] != target_tokens[i]
    (k when all match) and the correction is target_tokens[a]."""
    a = 0
    while a < k and int(cands[a]) == int(target_tokens[a]):
        a += 1
    return a, int(target_tokens[a])


class OracleModel:
    """Target model state machine mirroring the C ABI calls.

    weights: mapping {(name, layer): array} with the tensors of
    workload.gen.weight_spec (float32 or float64 arrays; bf16 models hold
    bf16-representable values).  Each is read once, when the model is
    built, and held in float64 (a mapping that produces tensors on demand
    keeps only one extra tensor alive at a time).  All arithmetic is
    float64.
    """

    def __init__(self, shape, weights, capacity=None):
        self.s = shape
        self.cap = capacity
        w = weights
        L = shape.n_layers
        self.embed = w[("embed", -1)]                    # gathered rows are upcast on use
        self.lm_head = to_f64(w[("lm_head", -1)])
        self.final_norm = to_f64(w[("final_norm", -1)])
        self.layers = []
        for l in range(L):
            lw = {}
            for name in ("attn_norm", "wq", "wk", "wv", "wo", "mlp_norm", "w_gate", "w_up", "w_down"):
                lw[name] = to_f64(w[(name, l)])
            for name in ("bq", "bk", "bv"):
                lw[name] = to_f64(w[(name, l)]) if shape.qkv_bias else None
            self.layers.append(lw)
        self.reset()

    # -- state -------------------------------------------------------------
    def reset(self):
        s = self.s
        self.k_cache = [np.zeros((s.n_kv_heads, 0, s.head_dim)) for _ in range(s.n_layers)]
        self.v_cache = [np.zeros((s.n_kv_heads, 0, s.head_dim)) for _ in range(s.n_layers)]
        self.kv_len = 0
        self.prefix_len = 0
        self.root = None
        self.last_logits = None

    @property
    def committed(self):
        """Tokens committed by verify calls since prefill (the first root,
        chosen at prefill, excluded).  Every call commits a+1 tokens and
        grows the cache by a+1 (root + accepted), so this is kv_len minus
        the prefix length."""
        return self.kv_len - self.prefix_len

    def _write_kv(self, l, pos0, k, v):
        """Place k, v ([n_kv, T, d]) at cache positions pos0..pos0+T-1,
        dropping whatever was stored at or beyond pos0."""
        self.k_cache[l] = np.concatenate([self.k_cache[l][:, :pos0], k], axis=1)
        self.v_cache[l] = np.concatenate([self.v_cache[l][:, :pos0], v], axis=1)

    # -- one forward over a block of rows --------------------------------------
    def forward(self, x, pos0, logit_rows=None):
        """Process rows x [T, hidden] at positions pos0..pos0+T-1 against the
        cache holding positions 0..pos0-1; appends their K/V.  Returns the
        logits [len(logit_rows), vocab] (all rows by default)."""
        s = self.s
        x = np.array(x, dtype=F64)
        T = x.shape[0]
        pos = pos0 + np.arange(T)
        for l, lw in enumerate(self.layers):
            xn = rms_norm(x, lw["attn_norm"], s.rms_eps)
            q = xn @ lw["wq"].T
            k = xn @ lw["wk"].T
            v = xn @ lw["wv"].T
            if s.qkv_bias:
                q, k, v = q + lw["bq"], k + lw["bk"], v + lw["bv"]
            q = rope(q.reshape(T, s.n_q_heads, s.head_dim), pos, s.rope_theta)
            k = rope(k.reshape(T, s.n_kv_heads, s.head_dim), pos, s.rope_theta)
            v = v.reshape(T, s.n_kv_heads, s.head_dim)
            self._write_kv(l, pos0, k.transpose(1, 0, 2), v.transpose(1, 0, 2))
            o = attention(q, self.k_cache[l], self.v_cache[l], pos)
            x = x + o.reshape(T, -1) @ lw["wo"].T
            xn = rms_norm(x, lw["mlp_norm"], s.rms_eps)
            x = x + (silu(xn @ lw["w_gate"].T) * (xn @ lw["w_up"].T)) @ lw["w_down"].T
        if logit_rows is None:
            logit_rows = np.arange(T)
        xf = rms_norm(x[logit_rows], self.final_norm, s.rms_eps)
        return xf @ self.lm_head.T

    def embed_tokens(self, tokens):
        return np.asarray(self.embed[np.asarray(tokens, dtype=np.int64)], dtype=F64)

    # -- C ABI mirror ------------------------------------------------------
    def prefill(self, audio, instr):
        """Audio rows (used directly as hidden states) then instruction
        tokens, at positions 0..; returns (first_token, kv_len)."""
        self.reset()
        rows = [np.asarray(audio, dtype=F64).reshape(-1, self.s.hidden)]
        if len(instr):
            rows.append(self.embed_tokens(instr))
        x = np.concatenate(rows, axis=0)
        if x.shape[0] == 0:
            raise ValueError("empty prefix")
        self._check_capacity(x.shape[0])
        logits = self.forward(x, 0, logit_rows=np.array([x.shape[0] - 1]))
        self.last_logits = logits
        self.root = greedy(logits[0])
        self.kv_len = self.prefix_len = x.shape[0]
        return self.root, self.kv_len

    def _check_capacity(self, end):
        if self.cap is not None and end > self.cap:
            raise OverflowError("KV capacity exceeded")

    def verify(self, cands, k):
        """One verification call of the root plus cands[:k].  Returns a dict
        with accepted_len, correction_token, kv_len, committed, the greedy
        tokens and top-2 margins of every row, and the logits."""
        if self.root is None:
            raise RuntimeError("verify before prefill")
        cands = [int(c) for c in cands[:k]]
        L0 = self.kv_len
        self._check_capacity(L0 + k + 1)
        x = self.embed_tokens([self.root] + cands)
        logits = self.forward(x, L0)
        t = [greedy(r) for r in logits]
        a, corr = verify_block(t, cands, k)
        # Retained state = committed prefix: root and a accepted candidates.
        self.kv_len = L0 + a + 1
        for l in range(self.s.n_layers):
            self.k_cache[l] = self.k_cache[l][:, :self.kv_len]
            self.v_cache[l] = self.v_cache[l][:, :self.kv_len]
        self.root = corr
        self.last_logits = logits
        return dict(accepted_len=a, correction_token=corr, kv_len=self.kv_len,
                    committed=self.committed, tokens=t,
                    margins=[top2_margin(r) for r in logits], logits=logits)

    def decode_one(self):
        return self.verify([], 0)

    def rollback(self, kv_len, root):
        if not (self.prefix_len <= kv_len <= self.kv_len):
            raise ValueError("rollback beyond kv_len")
        self.kv_len = kv_len
        for l in range(self.s.n_layers):
            self.k_cache[l] = self.k_cache[l][:, :kv_len]
            self.v_cache[l] = self.v_cache[l][:, :kv_len]
        self.root = int(root)

    def kv(self, layer):
        """(K, V) of a layer, [n_kv, kv_len, d] each (K after rotation)."""
        return self.k_cache[layer][:, :self.kv_len], self.v_cache[layer][:, :self.kv_len]

    def target_only(self, n_tokens):
        """The greedy reference stream: n_tokens K1 steps from the current
        state; returns [root, y_1, ..., y_n] (the root first)."""
        out = [self.root]
        for _ in range(n_tokens):
            r = self.decode_one()
            out.append(r["correction_token"])
        return out
