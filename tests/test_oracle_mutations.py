"""Plant plausible mistakes in the oracle (CPU only) and check that a pin fails.

Each mutant replaces one oracle building block for the duration of a test; the
pins of test_oracle.py (transformers decoder, brute-force decode) must reject it.
"""
import numpy as np
import pytest
import torch

import synth
from oracle import decoder as od
from tests import brute
from tests.test_oracle import SMALL, MICRO_BIAS, _hf_model, as_lists, dense, relmax


def _rope_interleaved(x, positions, theta):
    hd = x.shape[-1]
    i = np.arange(hd // 2, dtype=np.float64)
    ang = np.asarray(positions, dtype=np.float64)[:, None] * theta ** (-2.0 * i / hd)[None, :]
    c, s = np.cos(ang)[:, None, :], np.sin(ang)[:, None, :]
    x1, x2 = x[..., 0::2], x[..., 1::2]
    out = np.empty_like(x)
    out[..., 0::2] = x1 * c - x2 * s
    out[..., 1::2] = x2 * c + x1 * s
    return out


_ORIG_ROPE = od.rope


def _rope_sign(x, positions, theta):
    return _ORIG_ROPE(x, -np.asarray(positions), theta)


def _attend_gqa_modulo(q, positions, k_cache, v_cache):
    Hq, Hkv = q.shape[1], k_cache.shape[0]
    perm = [j % Hkv * (Hq // Hkv) + j // Hkv for j in range(Hq)]
    out = od._orig_attend(q[:, perm], positions, k_cache, v_cache)
    inv = np.argsort(perm)
    return out[:, inv]


def _attend_no_self(q, positions, k_cache, v_cache):
    out = np.zeros_like(q)
    for r, p in enumerate(positions):
        if p > 0:
            out[r:r + 1] = od._orig_attend(q[r:r + 1], np.array([p - 1]), k_cache, v_cache)
    return out


def _rms_no_eps_mean(h, gain, eps):
    return h / np.sqrt(np.sum(h * h, axis=-1, keepdims=True) + eps) * gain


def _silu_wrong(z):
    return z / (1.0 + np.exp(z))


MUTANTS = {
    "rope_interleaved": ("rope", _rope_interleaved),
    "rope_sign": ("rope", _rope_sign),
    "gqa_modulo": ("attend", _attend_gqa_modulo),
    "attend_no_self": ("attend", _attend_no_self),
    "rms_sum": ("rms_norm", _rms_no_eps_mean),
    "silu_sign": ("silu", _silu_wrong),
}


def _hf_pin_passes(shape):
    W, _ = dense(shape, seed=11, std=0.1)
    toks = synth.make_tokens(24, shape.vocab, seed=5).numpy()
    cache, y = od.prefill(shape, W, toks)
    model = _hf_model("qwen2" if shape.qkv_bias else "llama", shape, W)
    with torch.no_grad():
        out = model(input_ids=torch.from_numpy(toks.astype(np.int64))[None], use_cache=True)
    ok = relmax(y, out.last_hidden_state[0].numpy()) < 1e-5
    for l in range(shape.n_layers):
        ok &= relmax(cache[l, 0], out.past_key_values.layers[l].keys[0].numpy()) < 1e-5
    return ok


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_rejected_by_transformers_pin(monkeypatch, name):
    attr, fn = MUTANTS[name]
    monkeypatch.setattr(od, "_orig_attend", od.attend, raising=False)
    assert _hf_pin_passes(SMALL)
    monkeypatch.setattr(od, attr, fn)
    assert not _hf_pin_passes(SMALL)


def _brute_repair_pin_passes():
    shape = MICRO_BIAS
    n = 12
    W, _ = dense(shape, seed=4, std=0.3)
    toks = synth.make_tokens(n, shape.vocab, seed=1).numpy()
    new = synth.apply_edit(torch.from_numpy(toks), 3, 2, shape.vocab, seed=2).numpy()
    stale, _ = od.prefill(shape, W, toks)
    A = [6, 9]
    cache = stale.copy()
    y = od.repair(shape, W, cache, new, 3, 5, A)
    bcache = [[[[list(stale[l, kv, g, t]) for t in range(n)] for g in range(shape.n_kv_heads)]
                for kv in range(2)] for l in range(shape.n_layers)]
    by = brute.repair(shape, as_lists(W), bcache, new, [3, 4, 6, 9])
    return relmax(y, by) < 1e-12 and relmax(cache, np.array(bcache, dtype=np.float64)) < 1e-12


def test_attend_before_scatter_rejected(monkeypatch):
    """Attending before the fresh K/V of P are written breaks the repair pin."""
    assert _brute_repair_pin_passes()

    def layer_stale(shape, w, h, positions, k_cache, v_cache):
        R = h.shape[0]
        Hq, Hkv, hd = shape.n_heads, shape.n_kv_heads, shape.head_dim
        x = od.rms_norm(h, w["attn_norm"], shape.rms_eps)
        q = x @ w["wq"].T + (w["bq"] if w.get("bq") is not None else 0)
        k = x @ w["wk"].T + (w["bk"] if w.get("bk") is not None else 0)
        v = x @ w["wv"].T + (w["bv"] if w.get("bv") is not None else 0)
        q = od.rope(q.reshape(R, Hq, hd), positions, shape.rope_theta)
        k = od.rope(k.reshape(R, Hkv, hd), positions, shape.rope_theta)
        o = od.attend(q, positions, k_cache, v_cache).reshape(R, Hq * hd)
        k_cache[:, positions, :] = k.transpose(1, 0, 2)
        v_cache[:, positions, :] = v.reshape(R, Hkv, hd).transpose(1, 0, 2)
        h = h + o @ w["wo"].T
        x = od.rms_norm(h, w["mlp_norm"], shape.rms_eps)
        return h + (od.silu(x @ w["w_gate"].T) * (x @ w["w_up"].T)) @ w["w_down"].T

    monkeypatch.setattr(od, "layer_forward", layer_stale)
    assert not _brute_repair_pin_passes()
