"""Pins for the fp64 CPU oracle (no GPU).

Each test ties the oracle to something other than itself:
* a third-party implementation of the same decoder family (Hugging Face
  ``transformers`` Llama / Qwen2 / Mistral, run in float64) for prefill;
* a brute-force scalar incremental decoder (tests/brute.py) for the repair of
  scattered and contiguous position sets;
* the paper's invariants (Section 3): the full-position endpoint (Eq. 1),
  upstream positions unaffected by the edit, untouched slots outside P,
  transplant equal to recompute for a suffix set;
* closed forms of the building blocks (rotary relative-position property,
  RMSNorm scale invariance, attention over identical keys).
"""
import numpy as np
import pytest
import torch

import synth
from oracle import decoder as od
from tests import brute

MICRO = synth.ModelShape("micro", 2, 16, 4, 2, 4, 24, 32, 1e-5, 10000.0)
MICRO_BIAS = synth.scaled_shape(MICRO, name="micro-bias", qkv_bias=True)
SMALL = synth.ModelShape("small", 2, 64, 4, 2, 16, 96, 128, 1e-5, 10000.0)


def to_np(t):
    return None if t is None else t.to(torch.float64).numpy()


def dense(shape, seed=0, std=0.02):
    w = synth.make_weights(shape, dtype=torch.float32, seed=seed, std=std)
    return od.DenseWeights(to_np(w["embed"]), [{k: to_np(v) for k, v in lw.items()} for lw in w["layers"]],
                           to_np(w["final_norm"])), w


def as_lists(W):
    def conv(a):
        return None if a is None else a.tolist()
    return {"embed": W.embed.tolist(), "final_norm": W.final_norm.tolist(),
            "layers": [{k: conv(v) for k, v in lw.items()} for lw in W.layers]}


def relmax(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return float(np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300))


# ---------------------------------------------------------------- transformers pin

def _hf_model(kind, shape, W):
    import transformers as tf
    common = dict(vocab_size=shape.vocab, hidden_size=shape.d_model, intermediate_size=shape.d_ffn,
                  num_hidden_layers=shape.n_layers, num_attention_heads=shape.n_heads,
                  num_key_value_heads=shape.n_kv_heads, head_dim=shape.head_dim,
                  rms_norm_eps=shape.rms_eps, max_position_embeddings=4096)
    rope = {"rope_parameters": {"rope_type": "default", "rope_theta": shape.rope_theta}}
    if kind == "llama":
        cfg = tf.LlamaConfig(**common, **rope, attention_bias=False, mlp_bias=False)
        model = tf.LlamaModel(cfg)
    elif kind == "qwen2":
        cfg = tf.Qwen2Config(**common, **rope, use_sliding_window=False)
        model = tf.Qwen2Model(cfg)
    else:
        cfg = tf.MistralConfig(**common, **rope, sliding_window=None)
        model = tf.MistralModel(cfg)
    cfg._attn_implementation = "eager"
    model = model.double().eval()
    sd = {"embed_tokens.weight": W.embed, "norm.weight": W.final_norm}
    for l, lw in enumerate(W.layers):
        p = f"layers.{l}."
        sd[p + "input_layernorm.weight"] = lw["attn_norm"]
        sd[p + "post_attention_layernorm.weight"] = lw["mlp_norm"]
        for a, b in (("wq", "q_proj"), ("wk", "k_proj"), ("wv", "v_proj"), ("wo", "o_proj")):
            sd[p + f"self_attn.{b}.weight"] = lw[a]
        if kind == "qwen2":
            for a, b in (("bq", "q_proj"), ("bk", "k_proj"), ("bv", "v_proj")):
                sd[p + f"self_attn.{b}.bias"] = lw[a]
        for a, b in (("w_gate", "gate_proj"), ("w_up", "up_proj"), ("w_down", "down_proj")):
            sd[p + f"mlp.{b}.weight"] = lw[a]
    missing, unexpected = model.load_state_dict({k: torch.from_numpy(np.array(v)) for k, v in sd.items()},
                                                strict=False)
    assert not unexpected, unexpected
    assert all("rotary" in m for m in missing), missing
    return model


@pytest.mark.parametrize("kind,shape", [("llama", SMALL), ("qwen2", synth.scaled_shape(SMALL, qkv_bias=True)),
                                        ("mistral", synth.scaled_shape(SMALL, rope_theta=1e6))])
def test_prefill_matches_transformers(kind, shape):
    """The oracle's decoder equals a third-party float64 implementation of the
    same family (Section 4, "Models and decoding").  transformers computes rotary
    angles in float32, hence the 1e-5 tolerance."""
    W, _ = dense(shape, seed=11, std=0.1)
    toks = synth.make_tokens(40, shape.vocab, seed=5).numpy()
    cache, y = od.prefill(shape, W, toks)
    model = _hf_model(kind, shape, W)
    with torch.no_grad():
        out = model(input_ids=torch.from_numpy(toks.astype(np.int64))[None], use_cache=True)
    assert relmax(y, out.last_hidden_state[0].numpy()) < 1e-5
    for l in range(shape.n_layers):
        lay = out.past_key_values.layers[l]
        assert relmax(cache[l, 0], lay.keys[0].numpy()) < 1e-5
        assert relmax(cache[l, 1], lay.values[0].numpy()) < 1e-5


# ---------------------------------------------------------------- brute force pin

@pytest.mark.parametrize("shape", [MICRO, MICRO_BIAS])
def test_prefill_matches_brute_force(shape):
    W, _ = dense(shape, seed=3, std=0.3)
    toks = synth.make_tokens(10, shape.vocab, seed=9).numpy()
    cache, y = od.prefill(shape, W, toks)
    bc, by = brute.prefill(shape, as_lists(W), toks)
    assert relmax(y, by) < 1e-12
    assert relmax(cache, np.array(bc, dtype=np.float64)) < 1e-12


@pytest.mark.parametrize("P_kind", ["scattered", "window", "upstream+scattered"])
def test_repair_matches_brute_force(P_kind):
    shape = MICRO_BIAS
    n = 12
    W, _ = dense(shape, seed=4, std=0.3)
    toks = synth.make_tokens(n, shape.vocab, seed=1).numpy()
    new = synth.apply_edit(torch.from_numpy(toks), 3, 2, shape.vocab, seed=2).numpy()
    stale, _ = od.prefill(shape, W, toks)
    A = {"scattered": [6, 9], "window": [5, 6, 7], "upstream+scattered": [1, 7, 10]}[P_kind]
    cache = stale.copy()
    y = od.repair(shape, W, cache, new, 3, 5, A)
    bcache = [[[[list(stale[l, kv, g, t]) for t in range(n)] for g in range(shape.n_kv_heads)]
                for kv in range(2)] for l in range(shape.n_layers)]
    by = brute.repair(shape, as_lists(W), bcache, new, sorted(set(range(3, 5)) | set(A)))
    assert relmax(y, by) < 1e-12
    assert relmax(cache, np.array(bcache, dtype=np.float64)) < 1e-12


# ---------------------------------------------------------------- paper invariants

@pytest.fixture(scope="module")
def small_case():
    shape = synth.scaled_shape(SMALL, qkv_bias=True, n_layers=3)
    W, _ = dense(shape, seed=21, std=0.08)
    n = 48
    toks = synth.make_tokens(n, shape.vocab, seed=8).numpy()
    new = synth.apply_edit(torch.from_numpy(toks), 17, 4, shape.vocab, seed=6).numpy()
    assert (new != toks).any()
    stale, _ = od.prefill(shape, W, toks)
    oracle_cache, oracle_y = od.prefill(shape, W, new)
    return shape, W, n, toks, new, stale, oracle_cache, oracle_y


def test_endpoint_identity(small_case):
    """Eq. 1: recomputing every position reproduces the full prefill of C'."""
    shape, W, n, toks, new, stale, oc, oy = small_case
    cache = stale.copy()
    y = od.repair(shape, W, cache, new, 17, 21, [p for p in range(n) if not 17 <= p < 21])
    assert relmax(cache, oc) < 1e-12
    assert relmax(y, oy) < 1e-12


def test_suffix_set_equals_prefill(small_case):
    """Positions before the span cannot depend on the edit, so P = [s_start, n)
    also reproduces K(C') (Section 3, upstream exclusion)."""
    shape, W, n, toks, new, stale, oc, oy = small_case
    cache = stale.copy()
    y = od.repair(shape, W, cache, new, 17, 21, list(range(21, n)))
    assert relmax(cache, oc) < 1e-12
    assert relmax(y, oy[17:]) < 1e-12


def test_upstream_rows_unaffected(small_case):
    shape, W, n, toks, new, stale, oc, oy = small_case
    assert np.array_equal(stale[:, :, :, :17], oc[:, :, :, :17])
    assert not np.allclose(stale[:, :, :, 17:], oc[:, :, :, 17:])


def test_empty_edit_is_noop(small_case):
    shape, W, n, toks, new, stale, oc, oy = small_case
    cache = stale.copy()
    y = od.repair(shape, W, cache, new, 30, 30, [])
    assert y.shape == (0, shape.d_model)
    assert np.array_equal(cache, stale)


def test_null_edit_is_fixed_point(small_case):
    """With C' = C a consistent cache is unchanged by any repair set (the paper's
    null-content control, Section 5 "Sanity checks")."""
    shape, W, n, toks, new, stale, oc, oy = small_case
    cache = stale.copy()
    od.repair(shape, W, cache, toks, 17, 21, [25, 33, 40])
    assert relmax(cache, stale) < 1e-12


def test_untouched_slots_and_idempotence(small_case):
    shape, W, n, toks, new, stale, oc, oy = small_case
    A = [22, 29, 35, 46]
    cache = stale.copy()
    y1 = od.repair(shape, W, cache, new, 17, 21, A)
    P = od.repaired_set(17, 21, A)
    others = np.setdiff1d(np.arange(n), P)
    assert np.array_equal(cache[:, :, :, others], stale[:, :, :, others])
    once = cache.copy()
    y2 = od.repair(shape, W, cache, new, 17, 21, A)
    assert relmax(cache, once) < 1e-13 and relmax(y2, y1) < 1e-13


def test_transplant_vs_recompute(small_case):
    """Section 3 "Transplant is not recomputation": on a suffix set the two
    operators agree; on a scattered set recompute reads stale neighbours and
    differs from the transplanted oracle states."""
    shape, W, n, toks, new, stale, oc, oy = small_case
    P_suffix = list(range(17, n))
    rec = stale.copy()
    od.repair(shape, W, rec, new, 17, 21, list(range(21, n)))
    tr = stale.copy()
    od.transplant(tr, oc, P_suffix)
    assert relmax(rec, tr) < 1e-12
    A = [30, 40]
    rec = stale.copy()
    od.repair(shape, W, rec, new, 17, 21, A)
    tr = stale.copy()
    od.transplant(tr, oc, od.repaired_set(17, 21, A))
    assert relmax(rec[:, :, :, 17:21], tr[:, :, :, 17:21]) < 1e-12  # span: same inputs
    # layer-0/1 states outside the span depend only on unchanged tokens; from layer 2
    # on, a recomputed row reads stale neighbours that the oracle cache has refreshed
    assert relmax(rec[:2, :, :, [30, 40]], tr[:2, :, :, [30, 40]]) < 1e-12
    assert relmax(rec[2, :, :, [30, 40]], tr[2, :, :, [30, 40]]) > 1e-6


# ---------------------------------------------------------------- building blocks

def test_rope_relative_position():
    rng = np.random.default_rng(0)
    q = rng.standard_normal((1, 1, 16))
    k = rng.standard_normal((1, 1, 16))
    dots = []
    for m, nn in ((5, 2), (103, 100), (7003, 7000)):
        qm = od.rope(q, np.array([m]), 10000.0)
        kn = od.rope(k, np.array([nn]), 10000.0)
        dots.append(float(np.sum(qm * kn)))
    assert abs(dots[0] - dots[1]) < 1e-10 and abs(dots[0] - dots[2]) < 1e-9
    assert np.allclose(od.rope(q, np.array([0]), 10000.0), q)
    # norm preserved, and the pairing is (i, i + hd/2)
    r = od.rope(q, np.array([3]), 10000.0)
    assert abs(np.linalg.norm(r) - np.linalg.norm(q)) < 1e-12
    e0 = np.zeros((1, 1, 16))
    e0[0, 0, 0] = 1.0
    r = od.rope(e0, np.array([1]), 10000.0)
    assert abs(r[0, 0, 0] - np.cos(1.0)) < 1e-15 and abs(r[0, 0, 8] - np.sin(1.0)) < 1e-15


def test_rmsnorm_closed_form():
    x = np.array([[3.0, 4.0]])
    y = od.rms_norm(x, np.array([1.0, 2.0]), 0.0)
    rms = np.sqrt(12.5)
    assert np.allclose(y, [[3 / rms, 8 / rms]], rtol=0, atol=1e-15)
    rng = np.random.default_rng(1)
    x = rng.standard_normal((3, 32))
    assert relmax(od.rms_norm(7.5 * x, np.ones(32), 0.0), od.rms_norm(x, np.ones(32), 0.0)) < 1e-14


def test_attention_special_cases():
    rng = np.random.default_rng(2)
    # identical keys -> uniform weights -> mean of the values
    K = np.tile(rng.standard_normal((1, 1, 8)), (2, 6, 1))
    V = rng.standard_normal((2, 6, 8))
    q = rng.standard_normal((1, 4, 8))
    o = od.attend(q, np.array([5]), K, V)
    assert np.allclose(o[0, 0], V[0].mean(0)) and np.allclose(o[0, 3], V[1].mean(0))
    # a query at position 0 returns the value of slot 0
    o = od.attend(q, np.array([0]), rng.standard_normal((2, 6, 8)), V)
    assert np.allclose(o[0, 1], V[0, 0]) and np.allclose(o[0, 2], V[1, 0])
    # GQA with H_kv = H_q is MHA: compare with torch's scaled_dot_product_attention
    Kf = rng.standard_normal((4, 6, 8))
    Vf = rng.standard_normal((4, 6, 8))
    qs = rng.standard_normal((6, 4, 8))
    o = od.attend(qs, np.arange(6), Kf, Vf)
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(qs.transpose(1, 0, 2)), torch.from_numpy(Kf), torch.from_numpy(Vf), is_causal=True)
    assert relmax(o, ref.numpy().transpose(1, 0, 2)) < 1e-13
