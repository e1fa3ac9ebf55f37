"""Model shapes and synthetic workloads.

The five workloads are synthetic stand-ins for the paper's on-demand audio
decoding (Section 5.1 and Appendix D.1.2: ASR windows, speech translation and
spoken QA): a prefix of audio embeddings and instruction tokens is prefilled
into the target KV cache, then the reply is decoded by verify calls of a
known root plus k candidates (Appendix C.2).  The model shapes are the
public Qwen2.5-3B / Qwen2-7B decoder shapes with random weights; the paper's
datasets and trained models are not used.
"""
from dataclasses import dataclass, field, replace
from typing import List, Optional, Tuple

F32, BF16 = 0, 1


@dataclass(frozen=True)
class ModelShape:
    name: str
    n_layers: int
    hidden: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    ffn: int
    vocab: int
    rope_theta: float
    rms_eps: float = 1e-6
    dtype: int = BF16          # F32 or BF16: weights, GEMM operands, KV cache
    qkv_bias: bool = True
    weight_std: float = 0.02

    @property
    def qkv_out(self) -> int:
        return (self.n_q_heads + 2 * self.n_kv_heads) * self.head_dim

    def with_layers(self, n: int) -> "ModelShape":
        return replace(self, name=f"{self.name}-L{n}", n_layers=n)

    def param_count(self) -> int:
        H, F, V = self.hidden, self.ffn, self.vocab
        per_layer = H * self.qkv_out + self.n_q_heads * self.head_dim * H + 3 * H * F
        return self.n_layers * per_layer + 2 * V * H

    def weight_bytes_per_step(self) -> int:
        """Bytes a verify step must stream from HBM for weights: every layer
        matrix and the LM head once, plus the gathered embedding rows (not
        counted here; they are W rows, see `step_bytes`)."""
        es = 4 if self.dtype == F32 else 2
        H, F, V = self.hidden, self.ffn, self.vocab
        per_layer = H * self.qkv_out + self.n_q_heads * self.head_dim * H + 3 * H * F
        return es * (self.n_layers * per_layer + V * H)

    def kv_bytes_per_token(self) -> int:
        es = 4 if self.dtype == F32 else 2
        return es * 2 * self.n_layers * self.n_kv_heads * self.head_dim


TINY = ModelShape("tiny", 2, 256, 4, 2, 64, 1024, 4096, 1e4, dtype=F32, qkv_bias=False)
# Same shape in bf16 with QKV bias: exercises the bf16 kernels at oracle-cheap sizes.
TINY_BF16 = replace(TINY, name="tiny-bf16", dtype=BF16, qkv_bias=True)
QWEN3B = ModelShape("qwen2.5-3b-shape", 36, 2048, 16, 2, 128, 11008, 151936, 1e6)
QWEN7B = ModelShape("qwen2-7b-shape", 28, 3584, 28, 4, 128, 18944, 152064, 1e6)
# Drafter-sized decoder (Qwen2.5-0.5B dimensions, untied head): the producer
# of the concurrent-drafting measurement, next to the 3B shape.
QWEN05B = ModelShape("qwen2.5-0.5b-shape", 24, 896, 14, 2, 64, 4864, 151936, 1e6)


@dataclass
class Request:
    """One decoding request: prefix sizes, reply length N, proposal cap k and
    candidate corruption probability p."""
    n_audio: int
    n_instr: int
    reply_len: int
    k: int
    p: float
    max_rounds: Optional[int] = None   # stop after this many verify calls


@dataclass
class Workload:
    name: str
    shape: ModelShape
    requests: List[Request]
    seed: int = 0
    k_sweep: Tuple[int, ...] = ()
    p_sweep: Tuple[float, ...] = ()


def workload(i: int) -> Workload:
    """The five synthetic workloads (index 0..4)."""
    if i == 0:
        return Workload("tiny-fp32", TINY, [Request(128, 16, 32 * 5, 4, 0.3, max_rounds=32)])
    if i == 1:
        return Workload("qwen3b-asr", QWEN3B, [Request(750, 32, 128, 4, 0.3)])
    if i == 2:
        return Workload("qwen7b-asr", QWEN7B, [Request(750, 32, 256, 8, 0.3)],
                        k_sweep=(0, 1, 2, 3, 4, 7, 8, 15, 16), p_sweep=(0.1, 0.3, 0.6))
    if i == 3:
        return Workload("qwen7b-long-audio", QWEN7B, [Request(7500, 64, 512, 8, 0.4)])
    if i == 4:
        return Workload("qwen7b-mixed-batch", QWEN7B, mixed_batch_requests(16, seed=0))
    raise IndexError(i)


def mixed_batch_requests(n: int, seed: int = 0) -> List[Request]:
    """Config of the mixed batch: prefixes U{250..3000} audio rows + 32
    instruction tokens, replies U{32..512}, k from {0,4,8}, p ~ U[0.1,0.7]."""
    from . import gen
    u = gen.uniform_f64(gen.stream_key(seed, "batch", 0), 4 * n)
    reqs = []
    for r in range(n):
        n_audio = 250 + int(u[4 * r] * 2751)
        reply = 32 + int(u[4 * r + 1] * 481)
        k = (0, 4, 8)[int(u[4 * r + 2] * 3)]
        p = 0.1 + 0.6 * float(u[4 * r + 3])
        reqs.append(Request(n_audio, 32, reply, k, p))
    return reqs
