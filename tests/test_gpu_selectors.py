"""GPU parity of the CacheBlend selector (kvr_select_cacheblend) against the
fp64 oracle (oracle/selectors.py), Table 1.

Deviations: max |gpu - oracle| / max |oracle| within 1e-5 (fp32) / 2e-2
(bf16).  The selection is an integer decided by floating point: where the
oracle's K-th and (K+1)-th largest deviations are separated by more than the
tolerance, the sets must be equal; otherwise the GPU set must be the top-K of
the GPU's own deviations and agree with the oracle's above the ambiguous band.
The stale cache is only read.
"""
import numpy as np
import pytest
import torch

import paper_2609_17983_amd as kvr
import synth
from oracle import decoder as od
from oracle import selectors as osl
from tests.gpu_util import TOL, Engine, OracleWeights, relmax, say, to_device_weights

pytestmark = pytest.mark.gpu

MID = synth.ModelShape("mid-bf16", 2, 512, 8, 2, 128, 1024, 2048, 1e-5, 500000.0)


def _run(shape, dtype, n, s0, span, K, layer, seed=0):
    tdt = torch.bfloat16 if dtype == kvr.KVR_BF16 else torch.float32
    w = synth.make_weights(shape, dtype=tdt, seed=seed)
    eng = Engine(shape, to_device_weights(w), dtype, max_ctx=n, max_rows=64)
    try:
        ow = OracleWeights(w, cache=True)
        toks = synth.make_tokens(n, shape.vocab, seed=seed + 1)
        new = synth.apply_edit(toks, s0, span, shape.vocab)
        cache = eng.new_cache(n)
        eng.prefill(toks.cuda(), cache)
        torch.cuda.synchronize()
        before = cache.clone()
        m = n - 1 - (s0 + span)
        out = torch.full((K,), -1, dtype=torch.int32, device="cuda")
        dev = torch.empty(m, dtype=torch.float32, device="cuda")
        say(f"cacheblend {shape.name} n={n} edit [{s0},{s0 + span}) K={K} layer={layer}")
        cnt = kvr.kvr_select_cacheblend(eng.ctx, cache.data_ptr(), n, n, new.cuda().data_ptr(), s0, s0 + span, K,
                                        layer, out.data_ptr(), dev.data_ptr(), torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
        assert torch.equal(cache, before)
        cache_np = cache.to(torch.float64).cpu().numpy()
        ref_dev = osl.cacheblend_deviation(shape, ow, cache_np, new.numpy(), s0, s0 + span, layer)
        got_dev = dev.cpu().numpy()
        e = relmax(got_dev, ref_dev)
        say(f"  deviation err {e:.3e}")
        assert e <= TOL[dtype]
        got = out.cpu().numpy()[:cnt].tolist()
        assert cnt == min(K, m)
        assert got == osl.top_k_positions(got_dev, s0 + span, K)  # the GPU's own top-K, ascending
        ref = osl.top_k_positions(ref_dev, s0 + span, K)
        srt = np.sort(ref_dev)[::-1]
        band = 2 * TOL[dtype] * np.max(np.abs(ref_dev))
        if K < m and srt[K - 1] - srt[K] > band:
            assert got == ref
        else:
            sure = {s0 + span + i for i in range(m) if ref_dev[i] > srt[min(K, m) - 1] + band}
            assert sure <= set(got)
        return got
    finally:
        eng.close()


def test_cacheblend_tiny_fp32():
    _run(synth.TINY, kvr.KVR_F32, 512, 128, 8, 32, 1)


def test_cacheblend_mid_bf16():
    _run(MID, kvr.KVR_BF16, 700, 300, 16, 48, 1)


def test_cacheblend_first_layer_sees_no_deviation():
    """At layer 0 a pool position's keys/values depend only on its own token
    and position, which an in-place edit leaves unchanged: the deviation is
    exactly zero (same kernels, row-independent), so the rule degenerates to
    the lowest positions (EditLocal's window)."""
    shape, n, s0, span, K = MID, 700, 300, 16, 48
    w = synth.make_weights(shape, dtype=torch.bfloat16)
    eng = Engine(shape, to_device_weights(w), kvr.KVR_BF16, max_ctx=n, max_rows=64)
    try:
        toks = synth.make_tokens(n, shape.vocab, seed=1)
        new = synth.apply_edit(toks, s0, span, shape.vocab)
        cache = eng.new_cache(n)
        eng.prefill(toks.cuda(), cache)
        out = torch.empty(K, dtype=torch.int32, device="cuda")
        dev = torch.full((n - 1 - s0 - span,), -1.0, device="cuda")
        kvr.kvr_select_cacheblend(eng.ctx, cache.data_ptr(), n, n, new.cuda().data_ptr(), s0, s0 + span, K, 0,
                                  out.data_ptr(), dev.data_ptr(), torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
        assert torch.count_nonzero(dev).item() == 0
        assert out.cpu().tolist() == list(range(s0 + span, s0 + span + K))
    finally:
        eng.close()


def test_cacheblend_edge_cases():
    shape = synth.TINY
    w = synth.make_weights(shape, dtype=torch.float32)
    eng = Engine(shape, to_device_weights(w), kvr.KVR_F32, max_ctx=64, max_rows=64)
    try:
        toks = synth.make_tokens(64, shape.vocab, seed=1).cuda()
        cache = eng.new_cache(64)
        eng.prefill(toks, cache)
        out = torch.empty(64, dtype=torch.int32, device="cuda")
        s = torch.cuda.current_stream().cuda_stream
        # pool smaller than K, edit at the very start, empty pool
        assert kvr.kvr_select_cacheblend(eng.ctx, cache.data_ptr(), 64, 64, toks.data_ptr(), 0, 4, 100, 1,
                                         out.data_ptr(), None, s) == 59
        torch.cuda.synchronize()
        assert out[:59].cpu().tolist() == list(range(4, 63))
        assert kvr.kvr_select_cacheblend(eng.ctx, cache.data_ptr(), 64, 64, toks.data_ptr(), 60, 63, 8, 1,
                                         out.data_ptr(), None, s) == 0
        for args, status in (((64, 64, 5, 4, 8, 1), kvr.KVR_E_RANGE), ((64, 64, 5, 8, 8, 2), kvr.KVR_E_RANGE),
                             ((64, 64, 5, 8, -1, 1), kvr.KVR_E_ARG)):
            n, ncap, a, b, K, layer = args
            with pytest.raises(kvr.KvrError) as e:
                kvr.kvr_select_cacheblend(eng.ctx, cache.data_ptr(), n, ncap, toks.data_ptr(), a, b, K, layer,
                                          out.data_ptr(), None, s)
            assert e.value.status == status
    finally:
        eng.close()


# ---- Attention selector (kvr_select_attention): parity of the per-position
# attention mass with the oracle (same tolerance), the selection as above, and
# the stale rows [0, n) left untouched (the query's own keys/values go to the
# scratch slots [n, n + q)).

QWEN_LIKE = synth.ModelShape("qwen-like-bf16", 2, 1792, 14, 2, 128, 1024, 2048, 1e-6, 1000000.0, qkv_bias=True)


def _run_attention(shape, dtype, n, q, s0, span, K, max_rows=64, seed=0):
    tdt = torch.bfloat16 if dtype == kvr.KVR_BF16 else torch.float32
    w = synth.make_weights(shape, dtype=tdt, seed=seed)
    eng = Engine(shape, to_device_weights(w), dtype, max_ctx=n + q, max_rows=max_rows)
    try:
        ow = OracleWeights(w, cache=True)
        toks = synth.make_tokens(n + q, shape.vocab, seed=seed + 1)
        cache = eng.new_cache(n + q)
        eng.prefill(toks[:n].cuda(), cache, n=n)
        torch.cuda.synchronize()
        before = cache[:, :, :, :n].clone()
        m = n - 1 - (s0 + span)
        out = torch.full((max(K, 1),), -1, dtype=torch.int32, device="cuda")
        mass = torch.full((n,), float("nan"), dtype=torch.float32, device="cuda")
        cache_np = cache.to(torch.float64).cpu().numpy()
        say(f"attention selector {shape.name} n={n} q={q} edit [{s0},{s0 + span}) K={K}")
        cnt = kvr.kvr_select_attention(eng.ctx, cache.data_ptr(), n, n + q, toks.cuda().data_ptr(), q, s0, s0 + span,
                                       K, out.data_ptr(), mass.data_ptr(), torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
        assert torch.equal(cache[:, :, :, :n], before)
        ref = osl.attention_mass(shape, ow, cache_np, toks.numpy(), n, q)
        got = mass.cpu().numpy().astype(np.float64)
        e = relmax(got, ref)
        say(f"  mass err {e:.3e} (sum {got.sum():.4f} of at most {shape.n_layers * shape.n_heads * q})")
        assert e <= TOL[dtype]
        assert np.all(got >= 0) and got.sum() <= shape.n_layers * shape.n_heads * q * (1 + 1e-5)
        assert cnt == min(K, m)
        sel = out.cpu().numpy()[:cnt].tolist()
        D0 = s0 + span
        assert sel == osl.top_k_positions(got[D0:n - 1], D0, K)
        ref_d, srt = ref[D0:n - 1], np.sort(ref[D0:n - 1])[::-1]
        band = 2 * TOL[dtype] * np.max(np.abs(ref))
        if K < m and srt[K - 1] - srt[K] > band:
            assert sel == osl.top_k_positions(ref_d, D0, K)
        else:
            sure = {D0 + i for i in range(m) if ref_d[i] > srt[min(K, m) - 1] + band}
            assert sure <= set(sel)
        return sel
    finally:
        eng.close()


def test_attention_tiny_fp32():
    _run_attention(synth.TINY, kvr.KVR_F32, 300, 12, 128, 8, 32)


def test_attention_tiny_bf16_head_dim_64():
    _run_attention(synth.TINY, kvr.KVR_BF16, 300, 12, 128, 8, 32)


def test_attention_mid_bf16_ragged():
    # n not a multiple of the 64-key tile, q spanning two 16-row tiles
    _run_attention(MID, kvr.KVR_BF16, 701, 20, 300, 16, 48)


def test_attention_mid_bf16_long_query():
    # 100 query rows: several (head, row tile) pairs per wavefront, tiled projections
    _run_attention(MID, kvr.KVR_BF16, 450, 100, 100, 16, 32, max_rows=128)


def test_attention_group_of_seven_bf16():
    _run_attention(QWEN_LIKE, kvr.KVR_BF16, 333, 9, 50, 6, 17)


def test_attention_edge_cases():
    shape = synth.TINY
    w = synth.make_weights(shape, dtype=torch.float32)
    eng = Engine(shape, to_device_weights(w), kvr.KVR_F32, max_ctx=80, max_rows=16)
    try:
        toks = synth.make_tokens(80, shape.vocab, seed=1).cuda()
        cache = eng.new_cache(80)
        eng.prefill(toks[:64], cache)
        out = torch.empty(64, dtype=torch.int32, device="cuda")
        mass = torch.empty(64, device="cuda")
        s = torch.cuda.current_stream().cuda_stream
        # K beyond the pool: the whole pool, ascending
        assert kvr.kvr_select_attention(eng.ctx, cache.data_ptr(), 64, 80, toks.data_ptr(), 4, 0, 4, 100,
                                        out.data_ptr(), None, s) == 59
        torch.cuda.synchronize()
        assert out[:59].cpu().tolist() == list(range(4, 63))
        # empty pool: nothing selected, the mass is still written when asked for
        assert kvr.kvr_select_attention(eng.ctx, cache.data_ptr(), 64, 80, toks.data_ptr(), 4, 60, 63, 8,
                                        out.data_ptr(), mass.data_ptr(), s) == 0
        torch.cuda.synchronize()
        assert torch.isfinite(mass).all() and (mass >= 0).all()
        for args, status in (((64, 80, 0, 4, 8), kvr.KVR_E_RANGE),     # q = 0
                             ((64, 66, 4, 4, 8), kvr.KVR_E_RANGE),     # n + q > n_cap
                             ((64, 80, 17, 4, 8), kvr.KVR_E_RANGE),    # q above the rows per pass
                             ((64, 80, 4, 8, -1), kvr.KVR_E_ARG)):
            n, ncap, q, b, K = args
            with pytest.raises(kvr.KvrError) as e:
                kvr.kvr_select_attention(eng.ctx, cache.data_ptr(), n, ncap, toks.data_ptr(), q, 0, b, K,
                                         out.data_ptr(), None, s)
            assert e.value.status == status
    finally:
        eng.close()
