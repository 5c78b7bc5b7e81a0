"""Pins for the oracle's fresh-query scoring and repair metrics (no GPU).

Section 3, "What counts as repaired": the appended query/answer tokens read the
cache; m_x is a difference of length-averaged teacher-forced log-probabilities;
MR (Eq. 2) and the flip rate (Eq. 3) are built from it.  The scoring forward is
pinned to a third-party causal language model (transformers Llama in float64:
full forward over context + appended tokens, log-softmax of its logits, and its
greedy generation), the metrics to their closed forms.
"""
import numpy as np
import pytest
import torch

import synth
from oracle import decoder as od
from oracle import scoring as osc
from tests.test_oracle import SMALL, dense, relmax


def _causal_lm(shape, W, lm_head):
    import transformers as tf
    cfg = tf.LlamaConfig(vocab_size=shape.vocab, hidden_size=shape.d_model, intermediate_size=shape.d_ffn,
                         num_hidden_layers=shape.n_layers, num_attention_heads=shape.n_heads,
                         num_key_value_heads=shape.n_kv_heads, head_dim=shape.head_dim, rms_norm_eps=shape.rms_eps,
                         max_position_embeddings=4096, tie_word_embeddings=False,
                         rope_parameters={"rope_type": "default", "rope_theta": shape.rope_theta},
                         attention_bias=False, mlp_bias=False)
    cfg._attn_implementation = "eager"
    model = tf.LlamaForCausalLM(cfg).double().eval()
    sd = {"model.embed_tokens.weight": W.embed, "model.norm.weight": W.final_norm, "lm_head.weight": lm_head}
    names = {"wq": "self_attn.q_proj", "wk": "self_attn.k_proj", "wv": "self_attn.v_proj", "wo": "self_attn.o_proj",
             "w_gate": "mlp.gate_proj", "w_up": "mlp.up_proj", "w_down": "mlp.down_proj"}
    for l, lw in enumerate(W.layers):
        p = f"model.layers.{l}."
        sd[p + "input_layernorm.weight"] = lw["attn_norm"]
        sd[p + "post_attention_layernorm.weight"] = lw["mlp_norm"]
        for a, b in names.items():
            sd[p + b + ".weight"] = lw[a]
    missing, unexpected = model.load_state_dict({k: torch.from_numpy(np.array(v)) for k, v in sd.items()},
                                                strict=False)
    assert not unexpected and all("rotary" in m for m in missing), (missing, unexpected)
    return model


def _setup(n, m, seed=21):
    shape = SMALL
    W, _ = dense(shape, seed=seed, std=0.1)
    lm = synth.make_lm_head(shape, dtype=torch.float32, seed=seed, std=0.1).to(torch.float64).numpy()
    toks = synth.make_tokens(n + m, shape.vocab, seed=seed + 1).numpy().astype(np.int64)
    return shape, W, lm, toks


def test_score_matches_causal_lm():
    """Teacher-forced log-probabilities and argmax of the appended block equal
    those of one full causal-LM forward over context + appended tokens."""
    n, m = 30, 10
    shape, W, lm, toks = _setup(n, m)
    cache, _ = od.prefill(shape, W, toks[:n], n_cap=n + m)
    lp, am = osc.score(shape, W, lm, cache, toks, n, m)
    model = _causal_lm(shape, W, lm)
    with torch.no_grad():
        logits = model(input_ids=torch.from_numpy(toks)[None]).logits[0].numpy()
    lsm = osc.log_softmax(logits)
    ref = np.array([lsm[n + j, toks[n + j + 1]] for j in range(m - 1)])
    assert relmax(lp, ref) < 1e-5
    top2 = np.sort(logits[n:n + m], axis=-1)[:, -2:]
    clear = (top2[:, 1] - top2[:, 0]) > 1e-6
    assert np.array_equal(am[clear], np.argmax(logits[n:n + m], axis=-1)[clear])
    # the appended keys/values equal the causal LM's cache rows at those positions
    full, _ = od.prefill(shape, W, toks)
    assert relmax(cache[:, :, :, n:n + m], full[:, :, :, n:n + m]) < 1e-12


def test_generate_matches_causal_lm_greedy():
    n, q, new = 24, 6, 8
    shape, W, lm, toks = _setup(n, q, seed=23)
    cache, _ = od.prefill(shape, W, toks[:n], n_cap=n + q + new)
    out = osc.generate(shape, W, lm, cache, toks, n, q, new)
    model = _causal_lm(shape, W, lm)
    with torch.no_grad():
        g = model.generate(torch.from_numpy(toks[:n + q])[None], max_new_tokens=new, do_sample=False,
                           pad_token_id=0)[0, n + q:].tolist()
    assert out == g


def test_score_after_full_repair_equals_score_after_prefill():
    """Eq. 1 through the scoring forward: repairing every position of the
    stale cache and then scoring equals scoring over K(C')."""
    n, m = 20, 5
    shape, W, lm, toks = _setup(n, m, seed=25)
    new = synth.apply_edit(torch.from_numpy(toks[:n].astype(np.int32)), 5, 3, shape.vocab, seed=4).numpy()
    full = np.concatenate([new.astype(np.int64), toks[n:]])
    stale, _ = od.prefill(shape, W, toks[:n], n_cap=n + m)
    od.repair(shape, W, stale, full, 0, n, [])
    ref_cache, _ = od.prefill(shape, W, new, n_cap=n + m)
    lp_a, am_a = osc.score(shape, W, lm, stale, full, n, m)
    lp_b, am_b = osc.score(shape, W, lm, ref_cache, full, n, m)
    assert relmax(lp_a, lp_b) < 1e-12 and np.array_equal(am_a, am_b)


def test_log_softmax_closed_forms():
    z = np.zeros((2, 7))
    assert np.allclose(osc.log_softmax(z), -np.log(7), atol=0, rtol=1e-15)
    r = np.random.default_rng(0).normal(size=(3, 50)) * 5
    assert np.allclose(np.exp(osc.log_softmax(r)).sum(-1), 1.0, rtol=1e-13)
    assert np.allclose(osc.log_softmax(r + 123.0), osc.log_softmax(r), atol=1e-12)


def test_margin_recovery_and_flip_closed_forms():
    assert osc.margin(-1.0, -3.0) == 2.0
    assert osc.margin_recovery(5.0, 1.0, 5.0) == 1.0
    assert osc.margin_recovery(1.0, 1.0, 5.0) == 0.0
    assert osc.margin_recovery(3.0, 1.0, 5.0) == 0.5
    assert osc.margin_recovery(-1.0, 1.0, 5.0) == -0.5  # unclipped
    assert osc.margin_recovery(2.0, 1.0, 1.0) is None   # zero gap: excluded
    assert osc.mean_answer_logprob(np.array([-9.0, -1.0, -2.0, -3.0, -7.0]), q=2, k=3) == -2.0
    assert osc.flip([5, 6, 7, 8], [6, 7], [9]) is True
    assert osc.flip([5, 6, 7, 8], [6, 7], [8]) is False
    assert osc.flip([5, 6, 7, 8], [7, 6], [9]) is False
    assert osc.flip_rate([([1, 2], [2], [3]), ([1, 2], [3], [1])]) == 0.5
