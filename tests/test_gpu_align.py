"""Decoding from the candidate buffer on the GPU (as2d_verify_from_buffer):
for drafts with substitutions, insertions and deletions, published ahead of
time, one batch per step, or by a concurrent producer thread, the
committed stream is the GPU's own target-only stream bit for bit
(Appendix C.4, Proposition), and alignment lets calls commit more than one
token."""
import threading
import time

import pytest

from tests.harness import make_pair, prefix
from workload import QWEN7B, TINY, TINY_BF16, gen

pytestmark = pytest.mark.gpu


def setup(shape, n_audio, n_instr, reply, budget):
    """GPU model prefilled on request 0, its target-only stream of `reply`
    tokens after the first root, and the post-prefill state (kv_len, root)."""
    from paper_2609_37617_amd import as2d
    max_kv = (n_audio + n_instr + reply + budget + 2 + 63) // 64 * 64
    _, gpu = make_pair(shape, seed=0, max_requests=1, max_kv_len=max_kv, max_k=budget, oracle=False)
    _, a_dev, instr = prefix(shape, n_audio, n_instr, 0, 0)
    first, L = gpu.prefill(0, a_dev, instr)
    ref = [gpu.decode_one(0)["correction_token"] for _ in range(reply)]
    gpu.rollback(0, L, first)
    return as2d, gpu, ref, (L, first)


def decode_from_buffer(as2d, gpu, buf, reply, budget, publish=None):
    """The decoding loop; publish(step) runs before each call.  Returns the
    committed tokens, the number of calls and the accepted candidates."""
    cur = as2d.ReadCursor(8)
    committed, calls, accepted = [], 0, 0
    while len(committed) < reply:
        if publish:
            publish(calls)
        c0 = cur.cursor
        r, k = cur.verify_from_buffer(gpu, 0, buf, budget, reply - len(committed))
        assert k >= r["accepted_len"]
        committed += buf.read(c0, r["accepted_len"]) + [r["correction_token"]]
        calls += 1
        accepted += r["accepted_len"]
    return committed, calls, accepted


@pytest.mark.parametrize("shape,edits", [(TINY, (0.15, 0.1, 0.1)), (TINY_BF16, (0.15, 0.1, 0.1)),
                                         (TINY_BF16, (0.0, 0.0, 0.0)), (QWEN7B.with_layers(1), (0.2, 0.05, 0.05))],
                         ids=["tiny-f32", "tiny-bf16", "tiny-bf16-exact-draft", "qwen7b-width-1l"])
def test_buffer_decoding_commits_the_target_stream(shape, edits):
    budget, reply = 8, 64
    as2d, gpu, ref, state0 = setup(shape, 48, 8, reply, budget)
    draft = gen.edited_stream(ref, shape.vocab, *edits, seed=1)
    batches = [draft[i:i + 8] for i in range(0, len(draft), 8)]
    for schedule in ("ahead", "per-step"):
        print(f"{shape.name} edits={edits} schedule={schedule}", flush=True)
        gpu.rollback(0, *state0)
        buf = as2d.CandidateBuffer(max(len(draft), 1))
        if schedule == "ahead":
            for b in batches:
                buf.publish(b)
            publish = None
        else:
            publish = lambda step: step < len(batches) and buf.publish(batches[step])
        committed, calls, accepted = decode_from_buffer(as2d, gpu, buf, reply, budget, publish)
        assert committed == ref, (schedule, calls)
        assert gpu.state(0)[0] == state0[0] + reply
        assert accepted > 0 and calls < reply
        if edits == (0.0, 0.0, 0.0) and schedule == "ahead":
            assert calls == -(-reply // (budget + 1))        # an exact draft is accepted in full
        buf.close()
    gpu.close()


def test_concurrent_producer_thread():
    """A producer thread publishes while the target verifies: whatever is
    ready at each snapshot, the output is the target-only stream."""
    shape = TINY_BF16
    budget, reply = 8, 96
    as2d, gpu, ref, _ = setup(shape, 48, 8, reply, budget)
    draft = gen.edited_stream(ref, shape.vocab, 0.1, 0.05, 0.05, seed=2)
    buf = as2d.CandidateBuffer(len(draft))

    def producer():
        for i in range(0, len(draft), 8):
            buf.publish(draft[i:i + 8], offset=i, publish_ns=time.monotonic_ns())
            time.sleep(0.0005)

    th = threading.Thread(target=producer)
    th.start()
    committed, calls, accepted = decode_from_buffer(as2d, gpu, buf, reply, budget)
    th.join()
    assert committed == ref
    assert [r["offset"] for r in buf.records()] == list(range(0, len(draft), 8))
    buf.close()
    gpu.close()
