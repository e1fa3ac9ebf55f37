"""Target-decoupled decoding with a drafter on the same GPU
(as2d_run_decoupled): serial and concurrent runs both commit the target's
own stream bit for bit (Appendix C.4, Proposition); the serial run never
overlaps its stages; the stage log satisfies the accounting identity
(Appendix D.2)."""
import pytest

from paper_2609_37617_amd import overlap as po
from tests.harness import make_pair, prefix
from workload import QWEN05B, QWEN3B, QWEN7B, TINY, TINY_BF16, gen

pytestmark = pytest.mark.gpu


def models(tshape, dshape, n_audio, n_instr, reply, budget):
    from paper_2609_37617_amd import as2d
    max_kv = (n_audio + n_instr + 2 * reply + budget + 2 + 63) // 64 * 64
    _, tgt = make_pair(tshape, seed=0, max_requests=1, max_kv_len=max_kv, max_k=budget, oracle=False)
    _, drf = make_pair(dshape, seed=5, max_requests=1, max_kv_len=max_kv, max_k=1, oracle=False)
    _, a_dev, instr = prefix(tshape, n_audio, n_instr, 0, 0)
    first, L = tgt.prefill(0, a_dev, instr)
    ref = [tgt.decode_one(0)["correction_token"] for _ in range(reply)]
    tgt.rollback(0, L, first)
    _, d_dev, d_instr = prefix(dshape, n_audio, n_instr, 7, 0)
    d_first, d_L = drf.prefill(0, d_dev, d_instr)
    return as2d, tgt, drf, ref, (L, first), (d_L, d_first)


@pytest.mark.parametrize("tshape,dshape", [(TINY_BF16, TINY), (QWEN7B.with_layers(1), QWEN3B.with_layers(2)),
                                           (QWEN7B.with_layers(1), QWEN05B.with_layers(2))],
                         ids=["tiny", "7b-3b-width", "7b-0.5b-width"])
def test_serial_and_concurrent_runs_commit_the_target_stream(tshape, dshape):
    budget, reply = 7, 96
    as2d, tgt, drf, ref, t0, d0 = models(tshape, dshape, 40, 8, reply, budget)
    draft = gen.edited_stream(ref, tshape.vocab, 0.2, 0.05, 0.05, seed=9)
    res = {}
    for concurrent in (False, True):      # the serial run captures the graphs first
        print(f"{tshape.name} + {dshape.name} concurrent={concurrent}", flush=True)
        tgt.rollback(0, *t0)
        drf.rollback(0, *d0)
        r = as2d.run_decoupled(tgt, 0, drf, 0, draft, budget, reply, concurrent)
        assert r["committed"] == ref
        assert r["producer_rc"] == 0
        acc = po.accounting(r["intervals"], r["total_ns"])
        assert acc["T"] == acc["D"] + acc["V"] - acc["O"] + acc["H"]
        assert acc["N"] == reply and acc["H"] >= 0
        assert all(0 <= s <= e <= r["total_ns"] for s, e, _, _ in r["intervals"])
        if not concurrent:
            assert acc["O"] == 0
            assert r["published"] % 8 == 0 or r["published"] == len(draft)
        assert tgt.state(0)[0] == t0[0] + reply
        res[concurrent] = acc
    c = po.compare(res[False], res[True])
    assert c["break_even_holds"]
    print(f"serial {res[False]}\nconcurrent {res[True]}\ncompare {c}")
    tgt.close()
    drf.close()


def test_cu_budget_runs_and_keeps_results():
    """With CU budgets (target and drafter GEMMs on complementary numbers of
    workgroups) the concurrent run still commits the target stream, and a
    budget never changes a logit: split counts are unchanged."""
    budget, reply = 7, 64
    as2d, tgt, drf, ref, t0, d0 = models(QWEN7B.with_layers(1), QWEN05B.with_layers(2), 40, 8, reply, budget)
    tgt.set_keep_logits(True)
    tgt.rollback(0, *t0)
    tgt.verify(0, ref[:5])
    full = tgt.logits(0)
    tgt.set_cu_budget(192)
    drf.set_cu_budget(64)
    tgt.rollback(0, *t0)
    tgt.verify(0, ref[:5])
    assert (tgt.logits(0) == full).all()
    tgt.set_keep_logits(False)
    for k in range(budget + 1):               # capture the graphs one thread at a time
        tgt.rollback(0, *t0)
        tgt.verify(0, ref[:k])
    drf.rollback(0, *d0)
    drf.decode_one(0)
    tgt.rollback(0, *t0)
    drf.rollback(0, *d0)
    draft = gen.edited_stream(ref, QWEN7B.vocab, 0.2, 0.05, 0.05, seed=9)
    r = as2d.run_decoupled(tgt, 0, drf, 0, draft, budget, reply, True)
    assert r["committed"] == ref and r["producer_rc"] == 0
    with pytest.raises(as2d.As2dError):
        tgt.set_cu_budget(100000)
    tgt.set_cu_budget(0)
    tgt.close()
    drf.close()
