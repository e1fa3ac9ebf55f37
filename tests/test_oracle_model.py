"""Pins of the oracle's full model and of its verification state machine
(CPU only).

* The forward pass is checked against an independent implementation of the
  same architecture (transformers' Qwen2 model, float64, eager attention).
* Verification is checked against what the paper's exactness conditions fix
  (Appendix C.4): batched verification equals sequential greedy decoding,
  a chain equal to the target's own greedy output is fully accepted with
  the correction taken at k, a wrong first candidate gives accepted_len 0,
  arbitrary proposals reproduce the target-only output (the Proposition),
  and the retained KV equals a fresh prefill of the committed prefix.
"""
import numpy as np
import pytest
import torch

from oracle import OracleModel
from workload import TINY, TINY_BF16, gen
from workload.configs import ModelShape


def small_shape(**kw):
    base = dict(name="micro", n_layers=2, hidden=64, n_q_heads=4, n_kv_heads=2, head_dim=16,
                ffn=128, vocab=97, rope_theta=1e4, dtype=0, qkv_bias=True, weight_std=0.2)
    base.update(kw)
    return ModelShape(**base)


def build(shape, seed=0):
    w = gen.weights_dict(shape, gen.make_weights(shape, seed))
    return OracleModel(shape, w), w


def prefix(shape, n_audio, n_instr, seed=0):
    return (gen.audio_embeddings(shape, n_audio, seed), gen.instruction_tokens(shape, n_instr, seed))


def hf_model(shape, w):
    from transformers import Qwen2Config, Qwen2ForCausalLM
    cfg = Qwen2Config(vocab_size=shape.vocab, hidden_size=shape.hidden, intermediate_size=shape.ffn,
                      num_hidden_layers=shape.n_layers, num_attention_heads=shape.n_q_heads,
                      num_key_value_heads=shape.n_kv_heads, head_dim=shape.head_dim,
                      rope_theta=shape.rope_theta, rms_norm_eps=shape.rms_eps,
                      tie_word_embeddings=False, attn_implementation="eager",
                      max_position_embeddings=4096)
    m = Qwen2ForCausalLM(cfg).double().eval()
    sd = {"model.embed_tokens.weight": w[("embed", -1)], "model.norm.weight": w[("final_norm", -1)],
          "lm_head.weight": w[("lm_head", -1)]}
    names = {"attn_norm": "input_layernorm.weight", "wq": "self_attn.q_proj.weight",
             "wk": "self_attn.k_proj.weight", "wv": "self_attn.v_proj.weight",
             "bq": "self_attn.q_proj.bias", "bk": "self_attn.k_proj.bias", "bv": "self_attn.v_proj.bias",
             "wo": "self_attn.o_proj.weight", "mlp_norm": "post_attention_layernorm.weight",
             "w_gate": "mlp.gate_proj.weight", "w_up": "mlp.up_proj.weight", "w_down": "mlp.down_proj.weight"}
    for l in range(shape.n_layers):
        for ours, theirs in names.items():
            key = f"model.layers.{l}.{theirs}"
            if (ours, l) in w:
                sd[key] = w[(ours, l)]
            else:  # no QKV bias in this shape: Qwen2 always has one, set it to zero
                sd[key] = np.zeros(m.state_dict()[key].shape)
    m.load_state_dict({k: torch.tensor(np.asarray(v, dtype=np.float64)) for k, v in sd.items()})
    return m


@pytest.mark.parametrize("shape", [TINY, TINY_BF16], ids=lambda s: s.name)
def test_forward_matches_transformers_qwen2(shape):
    om, w = build(shape)
    audio, instr = prefix(shape, 40, 8)
    x = np.concatenate([audio.astype(np.float64), np.asarray(w[("embed", -1)], np.float64)[instr]])
    ours = om.forward(x, 0)
    with torch.no_grad():
        ref = hf_model(shape, w)(inputs_embeds=torch.tensor(x)[None]).logits[0].numpy()
    # transformers evaluates the rotary angles in float32; everything else is float64
    assert np.max(np.abs(ours - ref)) < 2e-5 * np.max(np.abs(ref))
    assert np.array_equal(ours.argmax(-1), ref.argmax(-1))


def test_batched_verify_equals_sequential_decodes():
    """Pathwise equivalence (Appendix C.4, requirement 1)."""
    shape = small_shape()
    om, _ = build(shape)
    audio, instr = prefix(shape, 12, 3)
    om.prefill(audio, instr)
    state = (om.kv_len, om.root)
    ref = om.target_only(6)                       # root, y1..y6 by K1 steps
    seq_logits = []
    om.rollback(*state)
    for i in range(6):
        seq_logits.append(om.decode_one()["logits"][0])
    om.rollback(*state)
    r = om.verify(ref[1:6], 5)                     # root + y1..y5 in one call
    assert r["tokens"] == ref[1:7]
    assert r["accepted_len"] == 5 and r["correction_token"] == ref[6]
    assert np.allclose(r["logits"], np.array(seq_logits), atol=1e-10)


def test_full_acceptance_and_wrong_first_candidate():
    shape = small_shape()
    om, _ = build(shape, seed=1)
    audio, instr = prefix(shape, 10, 2, seed=1)
    om.prefill(audio, instr)
    st = (om.kv_len, om.root)
    y = om.target_only(5)
    om.rollback(*st)
    r = om.verify(y[1:5], 4)
    assert (r["accepted_len"], r["correction_token"]) == (4, y[5])
    assert r["kv_len"] == st[0] + 5 and r["committed"] == 5
    om.rollback(*st)
    wrong = [(y[1] + 1) % shape.vocab] + y[2:5]
    r = om.verify(wrong, 4)
    assert (r["accepted_len"], r["correction_token"]) == (0, y[1])
    assert r["kv_len"] == st[0] + 1


@pytest.mark.parametrize("mode", ["random", "corrupted", "all-wrong", "mixed-k"])
def test_proposal_independent_exactness(mode):
    """Proposition (Appendix C.4): any proposal stream commits Y_T."""
    shape = small_shape(n_layers=1)
    om, _ = build(shape, seed=2)
    audio, instr = prefix(shape, 9, 2, seed=2)
    first, _ = om.prefill(audio, instr)
    st = (om.kv_len, om.root)
    n = 24
    y = om.target_only(n)
    om.rollback(*st)
    rng = np.random.default_rng(hash(mode) % 2**32)
    out = [first]
    while len(out) <= n:
        n_done = len(out) - 1
        k = min(int(rng.integers(0, 6)) if mode == "mixed-k" else 4, n - n_done - 1) if n - n_done - 1 > 0 else 0
        true = y[n_done + 1:n_done + 1 + k]
        if mode == "random":
            cands = list(rng.integers(0, shape.vocab, k))
        elif mode == "all-wrong":
            cands = [(t + 1) % shape.vocab for t in true]
        else:
            cands = [t if rng.random() > 0.4 else int(rng.integers(0, shape.vocab)) for t in true]
        r = om.verify(cands, k)
        out += cands[:r["accepted_len"]] + [r["correction_token"]]
    assert out[:n + 1] == y


def test_retained_kv_equals_fresh_prefill_of_committed_prefix():
    """Commit-and-repair (Appendix C.4, requirement 2): after verify rounds
    with rejections, the cache equals the one built from scratch."""
    shape = small_shape()
    om, _ = build(shape, seed=3)
    audio, instr = prefix(shape, 11, 3, seed=3)
    first, _ = om.prefill(audio, instr)
    rng = np.random.default_rng(3)
    committed = [first]
    for _ in range(6):
        cands = list(rng.integers(0, shape.vocab, 3))
        r = om.verify(cands, 3)
        committed += [int(c) for c in cands[:r["accepted_len"]]] + [r["correction_token"]]
    # processed tokens: everything committed except the pending root
    fresh, _ = build(shape, seed=3)
    fresh.prefill(audio, np.concatenate([instr, committed[:-1]]).astype(np.int32))
    assert fresh.kv_len == om.kv_len
    for l in range(shape.n_layers):
        k1, v1 = om.kv(l)
        k2, v2 = fresh.kv(l)
        assert np.allclose(k1, k2, atol=1e-11) and np.allclose(v1, v2, atol=1e-11)
    assert fresh.root == om.root


def test_state_errors():
    shape = small_shape(n_layers=1)
    w = gen.weights_dict(shape, gen.make_weights(shape, 0))
    om = OracleModel(shape, w, capacity=16)
    with pytest.raises(RuntimeError):
        om.verify([1], 1)
    audio, instr = prefix(shape, 10, 2)
    om.prefill(audio, instr)
    with pytest.raises(OverflowError):
        om.verify([1, 2, 3, 4], 4)      # 12 + 5 > 16
    with pytest.raises(ValueError):
        om.rollback(13, 0)
