"""C-ABI checks that need no GPU: the library loads, exports every symbol the
header declares, host-side selection equals the oracle bit for bit, and
argument validation rejects bad input before touching a device."""
import ctypes
import os
import random
import re

import pytest

import paper_2609_17983_amd as kvr
from oracle import select as osel

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    with open(os.path.join(ROOT, "include", "kvr.h")) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(kvr_[a-z_]+)\s*\(", text)))


def test_exports_every_declared_symbol():
    lib = kvr.load()
    names = _declared()
    assert set(names) == set(kvr.EXPORTED)
    for n in names:
        assert hasattr(lib, n), n
        assert ctypes.cast(getattr(lib, n), ctypes.c_void_p).value


def test_select_edit_local_matches_oracle():
    rnd = random.Random(0)
    for _ in range(300):
        n = rnd.randint(1, 9000)
        s0 = rnd.randint(0, n)
        s1 = rnd.randint(s0, min(n, s0 + 64))
        K = rnd.randint(0, 600)
        assert kvr.kvr_select(kvr.KVR_EDIT_LOCAL, n, s0, s1, K) == osel.select_edit_local(n, s0, s1, K)


def test_select_random_matches_oracle():
    rnd = random.Random(1)
    for i in range(200):
        n = rnd.randint(1, 9000)
        s0 = rnd.randint(0, n)
        s1 = rnd.randint(s0, min(n, s0 + 64))
        K = rnd.choice([0, 1, 8, 32, 128, 512, n])
        seed = rnd.getrandbits(64)
        assert kvr.kvr_select(kvr.KVR_RANDOM, n, s0, s1, K, seed) == osel.select_random(n, s0, s1, K, seed)


@pytest.mark.parametrize("seed", range(5))
def test_select_random_paper_seeds(seed):
    """The five seeds of the Random control (Table 1) on the 5000-token shape."""
    a = kvr.kvr_select(kvr.KVR_RANDOM, 5000, 2000, 2016, 32, seed)
    assert a == osel.select_random(5000, 2000, 2016, 32, seed)
    assert len(a) == 32 and all(2016 <= p < 4999 for p in a)


def test_select_errors():
    with pytest.raises(kvr.KvrError) as e:
        kvr.kvr_select(kvr.KVR_EDIT_LOCAL, 10, 5, 4, 2)
    assert e.value.status == kvr.KVR_E_RANGE
    with pytest.raises(kvr.KvrError) as e:
        kvr.kvr_select(kvr.KVR_EDIT_LOCAL, 0, 0, 0, 2)
    assert e.value.status == kvr.KVR_E_RANGE
    with pytest.raises(kvr.KvrError) as e:
        kvr.kvr_select(kvr.KVR_RANDOM, 10, 2, 3, -1)
    assert e.value.status == kvr.KVR_E_ARG
    with pytest.raises(kvr.KvrError) as e:
        kvr.kvr_select(7, 10, 2, 3, 1)
    assert e.value.status == kvr.KVR_E_ARG
    lib = kvr.load()
    assert lib.kvr_select(0, 10, 2, 3, 1, 0, None, None) == kvr.KVR_E_ARG
    assert "kvr_select" in kvr.kvr_last_error(None)


def _dims(**kw):
    base = dict(n_layers=2, d_model=256, n_heads=4, n_kv_heads=4, head_dim=64, d_ffn=688, vocab=1024, qkv_bias=0,
                rms_eps=1e-5, rope_theta=10000.0, max_ctx=512, max_rows=64, dtype=kvr.KVR_F32)
    base.update(kw)
    return kvr.kvr_dims(**base)


def test_cache_bytes():
    assert kvr.kvr_cache_bytes(_dims(), 512) == 2 * 2 * 4 * 512 * 64 * 4
    assert kvr.kvr_cache_bytes(_dims(dtype=kvr.KVR_BF16, n_kv_heads=2), 100) == 2 * 2 * 2 * 100 * 64 * 2
    assert kvr.kvr_cache_bytes(_dims(n_heads=3, n_kv_heads=2), 10) == 0
    # shapes the row kernels cannot take are rejected when the dims are
    # checked, before any launch: d_model not a multiple of 4 or above 16384,
    # fused Q|K|V width (3 + 2) * 6 = 30 not a multiple of 4
    assert kvr.kvr_cache_bytes(_dims(d_model=250), 10) == 0
    assert kvr.kvr_cache_bytes(_dims(d_model=16388), 10) == 0
    assert kvr.kvr_cache_bytes(_dims(d_model=24, n_heads=3, n_kv_heads=1, head_dim=6), 10) == 0
    assert kvr.kvr_cache_bytes(_dims(d_model=24, n_heads=4, n_kv_heads=2, head_dim=6), 10) == 2 * 2 * 2 * 10 * 6 * 4


@pytest.mark.parametrize("bad,status", [
    (dict(n_heads=6, n_kv_heads=4), kvr.KVR_E_ARG),
    (dict(head_dim=65), kvr.KVR_E_ARG),
    (dict(head_dim=256), kvr.KVR_E_UNSUPPORTED),
    (dict(max_rows=0), kvr.KVR_E_ARG),
    (dict(dtype=5), kvr.KVR_E_ARG),
    (dict(n_layers=0), kvr.KVR_E_ARG),
])
def test_create_rejects_bad_dims(bad, status):
    lib = kvr.load()
    d = _dims(**bad)
    w = kvr.kvr_weights(16, 16, None)
    out = ctypes.c_void_p(1)
    assert lib.kvr_create(ctypes.byref(d), ctypes.byref(w), ctypes.byref(out)) == status
    assert out.value is None
    assert kvr.kvr_last_error(None)


def test_create_rejects_missing_or_misaligned_weights():
    lib = kvr.load()
    d = _dims()
    out = ctypes.c_void_p()
    layers = (kvr.kvr_layer_weights * 2)()
    for lw in layers:
        for f, _ in kvr.kvr_layer_weights._fields_:
            setattr(lw, f, 4096)
        lw.bq = lw.bk = lw.bv = None
    w = kvr.kvr_weights(4096, 4096, ctypes.cast(layers, ctypes.POINTER(kvr.kvr_layer_weights)))
    layers[1].w_up = None
    assert lib.kvr_create(ctypes.byref(d), ctypes.byref(w), ctypes.byref(out)) == kvr.KVR_E_ARG
    layers[1].w_up = 4096 + 8
    assert lib.kvr_create(ctypes.byref(d), ctypes.byref(w), ctypes.byref(out)) == kvr.KVR_E_ARG
    layers[1].w_up = 4096
    layers[0].bq = 4096  # a bias without qkv_bias
    assert lib.kvr_create(ctypes.byref(d), ctypes.byref(w), ctypes.byref(out)) == kvr.KVR_E_ARG
    assert lib.kvr_create(None, ctypes.byref(w), ctypes.byref(out)) == kvr.KVR_E_ARG
    assert lib.kvr_create(ctypes.byref(d), None, ctypes.byref(out)) == kvr.KVR_E_ARG


def test_null_context_calls():
    lib = kvr.load()
    assert lib.kvr_prefill(None, None, 1, 1, None, None, None) == kvr.KVR_E_ARG
    assert lib.kvr_repair(None, None, 0, None) == kvr.KVR_E_ARG
    assert lib.kvr_workspace_bytes(None) == 0
    lib.kvr_destroy(None)


def test_select_to_boundary_matches_oracle():
    rnd = random.Random(2)
    for _ in range(300):
        n = rnd.randint(1, 9000)
        s0 = rnd.randint(0, n)
        s1 = rnd.randint(s0, min(n, s0 + 64))
        b = s1 + rnd.randint(0, 80)
        assert kvr.kvr_select_to_boundary(n, s0, s1, b) == osel.select_to_boundary(n, s0, s1, b)


def test_select_to_boundary_errors():
    with pytest.raises(kvr.KvrError) as e:
        kvr.kvr_select_to_boundary(100, 10, 14, 13)
    assert e.value.status == kvr.KVR_E_RANGE
    with pytest.raises(kvr.KvrError) as e:
        kvr.kvr_select_to_boundary(100, 10, 14, 40, capacity=8)  # 26 positions
    assert e.value.status == kvr.KVR_E_RANGE
    assert kvr.kvr_select_to_boundary(100, 10, 14, 40, capacity=26) == list(range(14, 40))
    lib = kvr.load()
    assert lib.kvr_select_to_boundary(100, 10, 14, 40, 4, None, None) == kvr.KVR_E_ARG
    assert lib.kvr_transplant(None, None, 0, None, 0, None, 0, None) == kvr.KVR_E_ARG


def test_metrics_closed_forms():
    """Eq. 2 / Eq. 3 helpers of the library: closed-form cases, then random
    cases against the oracle's own formulas (oracle/scoring.py)."""
    from oracle import scoring as osc
    assert kvr.kvr_answer_logprob([-9.0, -1.0, -2.0, -3.0, -7.0], 2, 3) == -2.0
    assert kvr.kvr_margin_recovery(3.0, 1.0, 5.0) == 0.5
    assert kvr.kvr_margin_recovery(-1.0, 1.0, 5.0) == -0.5
    assert kvr.kvr_margin_recovery(2.0, 1.0, 1.0) is None
    assert kvr.kvr_flipped([5, 6, 7, 8], [6, 7], [9]) and not kvr.kvr_flipped([5, 6, 7, 8], [6, 7], [8])
    assert kvr.kvr_flipped([1, 2], [], [3]) and not kvr.kvr_flipped([1, 2], [2], [])
    with pytest.raises(kvr.KvrError) as e:
        kvr.kvr_answer_logprob([-1.0, -2.0], 2, 2)  # the answer runs past the block
    assert e.value.status == kvr.KVR_E_RANGE
    lib = kvr.load()
    assert lib.kvr_flipped(None, 3, None, 0, None, 0, None) == kvr.KVR_E_ARG
    assert lib.kvr_margin_recovery(1.0, 0.0, 2.0, None, None) == kvr.KVR_E_ARG
    rnd = random.Random(3)
    for _ in range(200):
        lp = [rnd.uniform(-12.0, 0.0) for _ in range(rnd.randint(2, 30))]
        q = rnd.randint(1, len(lp))
        k = rnd.randint(1, len(lp) - q + 1)
        # the C side sums float32 inputs in double, in order
        import numpy as np
        lp32 = np.asarray(lp, dtype=np.float32).astype(np.float64)
        assert abs(kvr.kvr_answer_logprob(lp, q, k) - osc.mean_answer_logprob(lp32, q, k)) < 1e-12
        m = [rnd.choice([rnd.uniform(-5, 5), 1.0]) for _ in range(3)]
        ref = osc.margin_recovery(*m)
        got = kvr.kvr_margin_recovery(*m)
        assert (got is None and ref is None) or abs(got - ref) < 1e-12
        y = [rnd.randint(0, 5) for _ in range(rnd.randint(0, 16))]
        a = [rnd.randint(0, 5) for _ in range(rnd.randint(0, 3))]
        b = [rnd.randint(0, 5) for _ in range(rnd.randint(0, 3))]
        assert kvr.kvr_flipped(y, a, b) == osc.flip(y, a, b)
