"""GPU parity of kvr_prefill / kvr_repair against the fp64 oracle, at sizes the
oracle finishes in seconds (several tiles, ragged tails).

* The tiny fp32 Llama-style decoder of the workload list (2 layers, d_model 256,
  4 heads x 64, FFN 688, vocab 1024, 512-token context, 8-token edit at 128,
  EditLocal K=32): tolerance 1e-5.
* A bf16 decoder with head_dim 128 and 4-way grouped-query attention that
  exercises every MFMA kernel (weight-streaming GEMM for <= 64 rows, tiled GEMM
  above, split and unsplit attention): tolerance 2e-2.

Tolerance = max |gpu - oracle| / max |oracle| per tensor group (each layer's
repaired K rows, V rows, and the final hidden rows); slots outside P are
compared bitwise.  The stale cache given to both sides is the oracle's own
prefill of the original context, rounded to the model dtype.
"""
import numpy as np
import pytest
import torch

import paper_2609_17983_amd as kvr
import synth
from oracle import decoder as od
from oracle import select as osel
from tests.gpu_util import TOL, Engine, OracleWeights, compare_repair, relmax, say, to_device_weights

pytestmark = pytest.mark.gpu

MID = synth.ModelShape("mid-bf16", 2, 512, 8, 2, 128, 1024, 2048, 1e-5, 500000.0)
MID_BIAS = synth.scaled_shape(MID, name="mid-bf16-bias", n_heads=14, n_kv_heads=2, d_model=448, qkv_bias=True,
                              rope_theta=1e6, rms_eps=1e-6)


def _setup(shape, dtype, n, max_rows, seed=0, std=0.02):
    tdt = torch.bfloat16 if dtype == kvr.KVR_BF16 else torch.float32
    w = synth.make_weights(shape, dtype=tdt, seed=seed, std=std)
    wd = to_device_weights(w)
    eng = Engine(shape, wd, dtype, max_ctx=n + 64, max_rows=max_rows)
    ow = OracleWeights(w, cache=True)
    toks = synth.make_tokens(n, shape.vocab, seed=seed + 1)
    return eng, ow, toks


@pytest.fixture(scope="module")
def tiny():
    shape = synth.TINY
    eng, ow, toks = _setup(shape, kvr.KVR_F32, 512, 512)
    new = synth.apply_edit(toks, 128, 8, shape.vocab)
    stale_np, y_c = od.prefill(shape, ow, toks.numpy())
    yield shape, eng, ow, toks, new, stale_np, y_c
    eng.close()


@pytest.fixture(scope="module")
def mid():
    shape = MID
    n = 700
    eng, ow, toks = _setup(shape, kvr.KVR_BF16, n, 700)
    new = synth.apply_edit(toks, 300, 16, shape.vocab)
    stale_np, _ = od.prefill(shape, ow, toks.numpy())
    yield shape, eng, ow, toks, new, stale_np
    eng.close()


def _repair_case(shape, eng, ow, stale_np, new, s0, s1, positions, tag, n_cap=None):
    tdt = eng.tdtype
    n = new.numel()
    n_cap = n_cap or stale_np.shape[3]
    stale_dev = torch.zeros((shape.n_layers, 2, shape.n_kv_heads, n_cap, shape.head_dim), dtype=tdt, device="cuda")
    stale_dev[:, :, :, :stale_np.shape[3]] = torch.from_numpy(stale_np).to(tdt).cuda()
    ref_in = stale_dev.to(torch.float64).cpu().numpy()  # the exact values the GPU starts from
    cache = stale_dev.clone()
    P = od.repaired_set(s0, s1, positions)
    hidden = torch.full((len(P), shape.d_model), float("nan"), device="cuda")
    eng.repair([dict(cache=cache, tokens=new.cuda(), n=n, edit_start=s0, edit_end=s1, positions=positions,
                     hidden=hidden)])
    torch.cuda.synchronize()
    oc = ref_in.copy()
    y = od.repair(shape, ow, oc, new.numpy(), s0, s1, positions)
    return compare_repair(shape, None, stale_dev, cache, hidden, oc, y, P, n, TOL[eng.dtype], tag)


# ------------------------------------------------------------------------- tiny fp32

def test_tiny_prefill(tiny):
    shape, eng, ow, toks, new, stale_np, y_c = tiny
    say("case: tiny fp32 prefill n=512")
    cache = eng.new_cache(512)
    hidden = torch.empty((512, shape.d_model), device="cuda")
    eng.prefill(toks.cuda(), cache, hidden)
    torch.cuda.synchronize()
    got = cache.to(torch.float64).cpu().numpy()
    for l in range(shape.n_layers):
        for kv in range(2):
            assert relmax(got[l, kv], stale_np[l, kv]) <= TOL[kvr.KVR_F32], (l, kv)
    assert relmax(hidden.cpu().numpy(), y_c) <= TOL[kvr.KVR_F32]


def test_tiny_repair_edit_local(tiny):
    shape, eng, ow, toks, new, stale_np, _ = tiny
    A = osel.select_edit_local(512, 128, 136, 32)
    assert A == list(range(136, 168))
    _repair_case(shape, eng, ow, stale_np, new, 128, 136, A, "tiny EditLocal K=32")


@pytest.mark.parametrize("seed", range(5))
def test_tiny_repair_random(tiny, seed):
    shape, eng, ow, toks, new, stale_np, _ = tiny
    A = osel.select_random(512, 128, 136, 32, seed)
    _repair_case(shape, eng, ow, stale_np, new, 128, 136, A, f"tiny Random K=32 seed={seed}")


def test_tiny_endpoint_identity(tiny):
    """Eq. 1: recomputing all positions gives the oracle's prefill of C'."""
    shape, eng, ow, toks, new, stale_np, _ = tiny
    A = [p for p in range(512) if not 128 <= p < 136]
    errs = _repair_case(shape, eng, ow, stale_np, new, 128, 136, A, "tiny endpoint")
    oc, oy = od.prefill(shape, ow, new.numpy())
    cache = torch.from_numpy(stale_np).float().cuda()
    hidden = torch.empty((512, shape.d_model), device="cuda")
    eng.repair([dict(cache=cache, tokens=new.cuda(), edit_start=128, edit_end=136, positions=A, hidden=hidden)])
    torch.cuda.synchronize()
    assert relmax(cache.double().cpu().numpy(), oc) <= TOL[kvr.KVR_F32]
    assert relmax(hidden.cpu().numpy(), oy) <= TOL[kvr.KVR_F32]
    assert errs


def test_tiny_upstream_and_suffix(tiny):
    """P = [s_start, n) reproduces K(C') (upstream rows cannot depend on the edit)."""
    shape, eng, ow, toks, new, stale_np, _ = tiny
    oc, oy = od.prefill(shape, ow, new.numpy())
    cache = torch.from_numpy(stale_np).float().cuda()
    hidden = torch.empty((512 - 128, shape.d_model), device="cuda")
    eng.repair([dict(cache=cache, tokens=new.cuda(), edit_start=128, edit_end=136, positions=list(range(136, 512)),
                     hidden=hidden)])
    torch.cuda.synchronize()
    assert relmax(cache.double().cpu().numpy(), oc) <= TOL[kvr.KVR_F32]
    assert relmax(hidden.cpu().numpy(), oy[128:]) <= TOL[kvr.KVR_F32]


def test_transplant_matches_oracle(tiny):
    """Transplant (Section 3, "Transplant is not recomputation"): the rows of
    the given positions come from K(C') bit for bit, every layer and kv head;
    all other rows stay the stale cache's.  The source cache has a larger
    capacity than the destination."""
    shape, eng, ow, toks, new, stale_np, _ = tiny
    oracle_np, _ = od.prefill(shape, ow, new.numpy())
    n = stale_np.shape[3]
    pos = [0, 1, 2, 127, 128, 129, 130, 200, 301, 302, n - 1]
    stream = torch.cuda.current_stream().cuda_stream
    dst = torch.from_numpy(stale_np).float().cuda()
    src = torch.zeros((shape.n_layers, 2, shape.n_kv_heads, n + 40, shape.head_dim), dtype=torch.float32,
                      device="cuda")
    src[:, :, :, :n] = torch.from_numpy(oracle_np).float().cuda()
    kvr.kvr_transplant(eng.ctx, src.data_ptr(), n + 40, dst.data_ptr(), n, pos, stream)
    ref = stale_np.astype(np.float32)
    od.transplant(ref, oracle_np.astype(np.float32), pos)
    torch.cuda.synchronize()
    assert np.array_equal(dst.cpu().numpy(), ref)
    # every position: the destination becomes K(C')
    full = torch.from_numpy(stale_np).float().cuda()
    kvr.kvr_transplant(eng.ctx, src.data_ptr(), n + 40, full.data_ptr(), n, list(range(n)), stream)
    torch.cuda.synchronize()
    assert np.array_equal(full.cpu().numpy(), oracle_np.astype(np.float32))
    # rejected calls leave the destination untouched
    before = dst.clone()
    for bad, status in (([n], kvr.KVR_E_RANGE), ([5, 4], kvr.KVR_E_ARG), ([-1], kvr.KVR_E_RANGE)):
        with pytest.raises(kvr.KvrError) as e:
            kvr.kvr_transplant(eng.ctx, src.data_ptr(), n + 40, dst.data_ptr(), n, bad, stream)
        assert e.value.status == status
    kvr.kvr_transplant(eng.ctx, src.data_ptr(), n + 40, dst.data_ptr(), n, [], stream)
    torch.cuda.synchronize()
    assert torch.equal(dst, before)


def test_transplant_bf16(mid):
    shape, eng, ow, toks, new, stale_np = mid
    n = stale_np.shape[3]
    rng = np.random.default_rng(3)
    pos = sorted(rng.choice(n, size=57, replace=False).tolist())
    src = torch.randn((shape.n_layers, 2, shape.n_kv_heads, n, shape.head_dim), device="cuda").to(torch.bfloat16)
    dst = torch.from_numpy(stale_np).to(torch.bfloat16).cuda()
    ref = dst.clone()
    ref[:, :, :, pos] = src[:, :, :, pos]
    kvr.kvr_transplant(eng.ctx, src.data_ptr(), n, dst.data_ptr(), n, pos, torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    assert torch.equal(dst, ref)


def test_tiny_empty_edit_is_noop(tiny):
    shape, eng, ow, toks, new, stale_np, _ = tiny
    cache = torch.from_numpy(stale_np).float().cuda()
    before = cache.clone()
    eng.repair([dict(cache=cache, tokens=new.cuda(), edit_start=200, edit_end=200, positions=[])])
    eng.repair([])
    torch.cuda.synchronize()
    assert torch.equal(cache, before)


def test_tiny_errors_leave_cache_untouched(tiny):
    shape, eng, ow, toks, new, stale_np, _ = tiny
    cache = torch.from_numpy(stale_np).float().cuda()
    before = cache.clone()
    t = new.cuda()
    bad = [
        (dict(edit_start=130, edit_end=128, positions=[]), kvr.KVR_E_RANGE),
        (dict(edit_start=128, edit_end=136, positions=[140, 139]), kvr.KVR_E_ARG),
        (dict(edit_start=128, edit_end=136, positions=[140, 140]), kvr.KVR_E_ARG),
        (dict(edit_start=128, edit_end=136, positions=[130]), kvr.KVR_E_ARG),
        (dict(edit_start=128, edit_end=136, positions=[512]), kvr.KVR_E_RANGE),
        (dict(edit_start=128, edit_end=136, positions=[-1]), kvr.KVR_E_RANGE),
    ]
    for kw, status in bad:
        with pytest.raises(kvr.KvrError) as e:
            eng.repair([dict(cache=cache, tokens=t, **kw)])
        assert e.value.status == status, kw
    # |P| above max_rows
    with pytest.raises(kvr.KvrError) as e:
        eng.repair([dict(cache=cache, tokens=t, edit_start=0, edit_end=300, positions=list(range(300, 511))),
                    dict(cache=cache, tokens=t, edit_start=0, edit_end=2, positions=[])])
    assert e.value.status == kvr.KVR_E_RANGE
    # n above n_cap / max_ctx
    with pytest.raises(kvr.KvrError) as e:
        eng.repair([dict(cache=cache, tokens=t, n=513, edit_start=0, edit_end=1, positions=[])])
    assert e.value.status == kvr.KVR_E_RANGE
    with pytest.raises(kvr.KvrError):
        kvr.kvr_prefill(eng.ctx, t.data_ptr(), 0, 512, cache.data_ptr(), None, None)
    # two documents over one cache (or overlapping parts of one allocation):
    # one pass would let each read the other's fresh rows, so it is refused
    flat = torch.zeros(2 * cache.numel(), dtype=cache.dtype, device="cuda")
    inner = flat[1024:1024 + cache.numel()].view(cache.shape)
    for pair in ((cache, cache), (flat[:cache.numel()].view(cache.shape), inner)):
        with pytest.raises(kvr.KvrError) as e:
            eng.repair([dict(cache=pair[0], tokens=t, edit_start=128, edit_end=136, positions=[]),
                        dict(cache=pair[1], tokens=t, edit_start=200, edit_end=201, positions=[])])
        assert e.value.status == kvr.KVR_E_ARG
        assert "share cache memory" in kvr.kvr_last_error(eng.ctx)
    # a document with nothing to repair may name any cache
    eng.repair([dict(cache=flat[:cache.numel()].view(cache.shape), tokens=t, edit_start=128, edit_end=128,
                     positions=[]),
                dict(cache=inner, tokens=t, edit_start=128, edit_end=128, positions=[])])
    torch.cuda.synchronize()
    assert torch.equal(cache, before)
    assert not flat.any()


# ------------------------------------------------------------------------- mid bf16

def test_mid_prefill(mid):
    shape, eng, ow, toks, new, stale_np = mid
    say("case: mid bf16 prefill n=700")
    n = 700
    cache = eng.new_cache(704)
    hidden = torch.empty((n, shape.d_model), device="cuda")
    eng.prefill(toks.cuda(), cache, hidden)
    torch.cuda.synchronize()
    got = cache.to(torch.float64).cpu().numpy()
    errs = {}
    for l in range(shape.n_layers):
        for kv in range(2):
            errs[(l, kv)] = relmax(got[l, kv, :, :n], stale_np[l, kv])
    errs["hidden"] = relmax(hidden.cpu().numpy(), od.prefill(shape, ow, toks.numpy())[1])
    say(f"mid prefill errors {errs}")
    assert max(errs.values()) <= TOL[kvr.KVR_BF16]
    assert torch.count_nonzero(cache[:, :, :, n:]) == 0


@pytest.mark.parametrize("policy,K", [("edit_local", 32), ("edit_local", 0), ("random", 8), ("random", 128),
                                      ("edit_local", 48)])
def test_mid_repair(mid, policy, K):
    shape, eng, ow, toks, new, stale_np = mid
    A = (osel.select_edit_local(700, 300, 316, K) if policy == "edit_local"
         else osel.select_random(700, 300, 316, K, 3))
    _repair_case(shape, eng, ow, stale_np, new, 300, 316, A, f"mid {policy} K={K}", n_cap=704)


# Seeded sweep over edit placements, span lengths, budgets and both policies,
# so that one run covers every projection kernel (skinny up to 64 rows, tall to
# 192, tiled above), split and unsplit attention items, and the pool's edges:
# an edit at position 0, an edit that ends at the last position (empty pool),
# a budget larger than the pool.
def _sweep_cases():
    rng = np.random.default_rng(2609)
    cases = [(0, 8, 32, "edit_local", 0), (690, 9, 0, "edit_local", 0), (640, 4, 500, "random", 11),
             (100, 16, 250, "random", 5), (50, 24, 400, "edit_local", 0)]
    for i in range(9):
        span = int(rng.integers(1, 25))
        s0 = int(rng.integers(0, 700 - span))
        K = int(rng.choice([1, 5, 17, 40, 63, 100, 150, 250]))
        policy = "edit_local" if i % 2 == 0 else "random"
        cases.append((s0, span, K, policy, int(rng.integers(0, 1 << 30))))
    return cases


SWEEP = _sweep_cases()


@pytest.mark.parametrize("s0,span,K,policy,seed", SWEEP,
                         ids=[f"{p}-e{s}+{n}-K{k}" for s, n, k, p, _ in SWEEP])
def test_mid_repair_sweep(mid, s0, span, K, policy, seed):
    shape, eng, ow, toks, _, stale_np = mid
    n, s1 = 700, s0 + span
    new_i = synth.apply_edit(toks, s0, span, shape.vocab, label=seed & 0xffff)
    A = (osel.select_edit_local(n, s0, s1, K) if policy == "edit_local"
         else osel.select_random(n, s0, s1, K, seed))
    _repair_case(shape, eng, ow, stale_np, new_i, s0, s1, A,
                 f"mid sweep {policy} edit [{s0},{s1}) K={K} ({span + len(A)} rows)", n_cap=704)


def test_mid_repair_is_idempotent_and_deterministic(mid):
    shape, eng, ow, toks, new, stale_np = mid
    cache = torch.from_numpy(stale_np).to(torch.bfloat16).cuda()
    A = osel.select_random(700, 300, 316, 32, 1)
    h1 = torch.empty((48, shape.d_model), device="cuda")
    h2 = torch.empty_like(h1)
    doc = dict(cache=cache, tokens=new.cuda(), edit_start=300, edit_end=316, positions=A)
    eng.repair([dict(doc, hidden=h1)])
    once = cache.clone()
    eng.repair([dict(doc, hidden=h2)])
    torch.cuda.synchronize()
    assert torch.equal(cache, once) and torch.equal(h1, h2)


def test_mid_batched_documents(mid):
    """Several documents with their own caches, lengths and edits in one call."""
    shape, eng, ow, toks, new, stale_np = mid
    specs = [(700, 300, 316, osel.select_edit_local(700, 300, 316, 32)),
             (700, 650, 651, osel.select_edit_local(700, 650, 651, 32)),
             (700, 5, 9, osel.select_random(700, 5, 9, 40, 7))]
    docs, refs = [], []
    for i, (n, s0, s1, A) in enumerate(specs):
        t_new = synth.apply_edit(toks, s0, s1 - s0, shape.vocab, label=i)
        cache = torch.from_numpy(stale_np).to(torch.bfloat16).cuda()
        ref_in = cache.to(torch.float64).cpu().numpy()
        P = od.repaired_set(s0, s1, A)
        hidden = torch.empty((len(P), shape.d_model), device="cuda")
        docs.append(dict(cache=cache, tokens=t_new.cuda(), edit_start=s0, edit_end=s1, positions=A, hidden=hidden))
        refs.append((ref_in, t_new, s0, s1, A, P, cache.clone()))
    eng.repair(docs)
    torch.cuda.synchronize()
    for d, (ref_in, t_new, s0, s1, A, P, stale_dev) in zip(docs, refs):
        oc = ref_in.copy()
        y = od.repair(shape, ow, oc, t_new.numpy(), s0, s1, A)
        compare_repair(shape, None, stale_dev, d["cache"], d["hidden"], oc, y, P, 700, TOL[kvr.KVR_BF16],
                       f"mid batched span=[{s0},{s1})")


@pytest.fixture(scope="module")
def mid_bias():
    shape = MID_BIAS
    n = 333
    eng, ow, toks = _setup(shape, kvr.KVR_BF16, n, 400, seed=5)
    new = synth.apply_edit(toks, 100, 16, shape.vocab)
    stale_np, _ = od.prefill(shape, ow, toks.numpy())
    yield shape, eng, ow, toks, new, stale_np
    eng.close()


@pytest.mark.parametrize("K", [32, 200])
def test_mid_bias_gqa7_repair(mid_bias, K):
    """QKV bias and 7 query heads per kv head (the Qwen2.5 arrangement)."""
    shape, eng, ow, toks, new, stale_np = mid_bias
    A = osel.select_edit_local(333, 100, 116, K)
    _repair_case(shape, eng, ow, stale_np, new, 100, 116, A, f"mid-bias K={K}")


# A wide feed-forward (8192 features: 1024 gate/up weight tiles) and 1100 rows
# give the gate/up projection 9 x 64 = 576 blocks of 128 rows, enough for the
# tiled kernel's 128-row shape (two blocks per compute unit); the other
# projections of the same pass take the 64-row shape.  The last 128-row block
# holds 5 of its 8 row tiles.
WIDE = synth.ModelShape("wide-ffn-bf16", 1, 512, 8, 2, 128, 8192, 2048, 1e-5, 500000.0)


def test_wide_prefill_both_tile_shapes():
    shape, n = WIDE, 1100
    w = synth.make_weights(shape, dtype=torch.bfloat16, seed=5)
    eng = Engine(shape, to_device_weights(w), kvr.KVR_BF16, max_ctx=n, max_rows=64)
    try:
        toks = synth.make_tokens(n, shape.vocab, seed=6)
        cache = eng.new_cache(n)
        hidden = torch.empty((n, shape.d_model), device="cuda")
        say(f"case: {shape.name} prefill n={n}")
        eng.prefill(toks.cuda(), cache, hidden)
        torch.cuda.synchronize()
        oc, oy = od.prefill(shape, OracleWeights(w), toks.numpy())
        got = cache.to(torch.float64).cpu().numpy()
        errs = {(l, kv): relmax(got[l, kv], oc[l, kv]) for l in range(shape.n_layers) for kv in range(2)}
        errs["hidden"] = relmax(hidden.cpu().numpy(), oy)
        say(f"  {errs}")
        assert max(errs.values()) <= TOL[kvr.KVR_BF16]
    finally:
        eng.close()


def test_wide_repair_split_tiled_projections():
    """166 repaired rows (above the skinny kernel's 64) of the wide shape: the
    tiled projections with K split into slices (down over 8192 features,
    output over 1024), their partial tiles summed by the next row kernel."""
    shape, n = WIDE, 900
    w = synth.make_weights(shape, dtype=torch.bfloat16, seed=7)
    eng = Engine(shape, to_device_weights(w), kvr.KVR_BF16, max_ctx=n, max_rows=256)
    try:
        ow = OracleWeights(w, cache=True)
        stale = synth.make_stale_cache(shape, n, label=7).to(torch.float64).numpy()
        toks = synth.make_tokens(n, shape.vocab, seed=8)
        new = synth.apply_edit(toks, 200, 16, shape.vocab)
        A = osel.select_edit_local(n, 200, 216, 150)
        _repair_case(shape, eng, ow, stale, new, 200, 216, A, f"{shape.name} EditLocal K=150 (166 rows)")
    finally:
        eng.close()


# 4160 features: 520 gate/up weight tiles, which the engine packs in groups of
# three (the skinny plan's tiles per block for up to 64 rows), so the last
# group holds a single tile.  Prefill reads the grouped weights through the
# tiled kernel, the 48-row repair through the skinny kernel.
RAGGED = synth.ModelShape("ragged-groups-bf16", 1, 512, 8, 2, 128, 4160, 2048, 1e-5, 500000.0)


def test_ragged_gateup_groups_prefill_and_repair():
    shape, n = RAGGED, 700
    w = synth.make_weights(shape, dtype=torch.bfloat16, seed=9)
    eng = Engine(shape, to_device_weights(w), kvr.KVR_BF16, max_ctx=n, max_rows=64)
    try:
        toks = synth.make_tokens(n, shape.vocab, seed=10)
        cache = eng.new_cache(n)
        hidden = torch.empty((n, shape.d_model), device="cuda")
        say(f"case: {shape.name} prefill n={n}")
        eng.prefill(toks.cuda(), cache, hidden)
        torch.cuda.synchronize()
        oc, oy = od.prefill(shape, OracleWeights(w), toks.numpy())
        got = cache.to(torch.float64).cpu().numpy()
        errs = {(l, kv): relmax(got[l, kv], oc[l, kv]) for l in range(shape.n_layers) for kv in range(2)}
        errs["hidden"] = relmax(hidden.cpu().numpy(), oy)
        say(f"  {errs}")
        assert max(errs.values()) <= TOL[kvr.KVR_BF16]

        ow = OracleWeights(w, cache=True)
        stale = synth.make_stale_cache(shape, n, label=9).to(torch.float64).numpy()
        new = synth.apply_edit(toks, 300, 16, shape.vocab)
        A = osel.select_edit_local(n, 300, 316, 32)
        _repair_case(shape, eng, ow, stale, new, 300, 316, A, f"{shape.name} EditLocal K=32 (48 rows)")
    finally:
        eng.close()


# Skinny-GEMM plans forced through the planner's overrides (read on every
# pass), so that every tile count per block (1-8), cross-block splits up to 8
# and gate/up blocks whose tiles straddle the packing groups are checked
# against the oracle, not only the plans the cost model picks.
PLAN_OVERRIDES = [
    {"KVR_NT_QKV": "1", "KVR_SPLIT_QKV": "1", "KVR_NT_O": "2", "KVR_SPLIT_O": "8", "KVR_NT_GATEUP": "1",
     "KVR_NT_DOWN": "3", "KVR_SPLIT_DOWN": "2"},
    {"KVR_NT_QKV": "5", "KVR_SPLIT_QKV": "2", "KVR_NT_O": "6", "KVR_SPLIT_O": "1", "KVR_NT_GATEUP": "4",
     "KVR_NT_DOWN": "7", "KVR_SPLIT_DOWN": "4"},
    {"KVR_NT_QKV": "8", "KVR_SPLIT_QKV": "4", "KVR_NT_O": "8", "KVR_SPLIT_O": "2", "KVR_NT_GATEUP": "6",
     "KVR_NT_DOWN": "8", "KVR_SPLIT_DOWN": "8"},
    # blocks of nine and ten tiles (passes of at most 48 rows), ragged last blocks
    {"KVR_NT_QKV": "9", "KVR_SPLIT_QKV": "2", "KVR_NT_O": "10", "KVR_SPLIT_O": "4", "KVR_NT_GATEUP": "10",
     "KVR_NT_DOWN": "9", "KVR_SPLIT_DOWN": "3"},
]


@pytest.mark.parametrize("env", PLAN_OVERRIDES, ids=["nt1-2-3", "nt4-5-6-7", "nt6-8", "nt9-10"])
def test_mid_skinny_plan_overrides(mid, monkeypatch, env):
    shape, eng, ow, toks, new, stale_np = mid
    for k, v in env.items():
        monkeypatch.setenv(k, v)
    A = osel.select_edit_local(700, 300, 316, 32)
    _repair_case(shape, eng, ow, stale_np, new, 300, 316, A, f"mid EditLocal K=32, skinny plans {env}")


# Attention plans forced through the planner's overrides: items of two or
# three row tiles when keys are split (the combine then merges multi-tile
# items), one-tile key ranges, and a target so low that no key range is split.
ATT_OVERRIDES = [{"KVR_ATT_MT": "2"}, {"KVR_ATT_MT": "3"}, {"KVR_ATT_MINKS": "64", "KVR_ATT_TARGET": "1024"},
                 {"KVR_ATT_TARGET": "1"}]


@pytest.mark.parametrize("env", ATT_OVERRIDES, ids=["mt2", "mt3", "one-tile-items", "unsplit"])
def test_mid_attention_plan_overrides(mid, monkeypatch, env):
    shape, eng, ow, toks, new, stale_np = mid
    for k, v in env.items():
        monkeypatch.setenv(k, v)
    A = osel.select_edit_local(700, 300, 316, 32)
    _repair_case(shape, eng, ow, stale_np, new, 300, 316, A, f"mid EditLocal K=32, attention plan {env}")


# Passes of 65-192 rows run the tall kernel (a block holds every row): one
# repair per row-tile count 5-12, with the plans the planner picks.
TALL_ROWS = [(66, "edit_local"), (95, "random"), (100, "edit_local"), (128, "random"), (129, "edit_local"),
             (150, "random"), (170, "edit_local"), (192, "random")]


@pytest.mark.parametrize("rows,policy", TALL_ROWS, ids=[f"{r}-{p}" for r, p in TALL_ROWS])
def test_mid_tall_rows(mid, rows, policy):
    shape, eng, ow, toks, new, stale_np = mid
    K = rows - 16
    A = (osel.select_edit_local(700, 300, 316, K) if policy == "edit_local"
         else osel.select_random(700, 300, 316, K, rows))
    _repair_case(shape, eng, ow, stale_np, new, 300, 316, A, f"mid {policy} K={K} ({rows} rows, tall kernel)",
                 n_cap=704)


# Tall plans forced through the overrides: tiles per block that leave some
# wavefronts with fewer tiles (or none), K splits of every STORE projection
# that do not divide its k-steps, blocks of more than 12 tiles (five per
# wavefront), the gate/up projection fused with its SwiGLU or split in two
# (partials finished by the SwiGLU pass; the default plan at these sizes),
# the tiled kernel for the same rows, and the per-row RMSNorm kernel in place
# of the residual step by column blocks with the RMS scale applied by the
# projections.
TALL_OVERRIDES = [{"KVR_TALL_TPB": "5", "KVR_TALL_SPLIT": "3"}, {"KVR_TALL_TPB": "1", "KVR_TALL_SPLIT": "7"},
                  {"KVR_TALL_TPB": "12", "KVR_TALL_SPLIT": "1", "KVR_TALL_GU_SPLIT": "1"},
                  {"KVR_TALL_TPB": "17", "KVR_TALL_SPLIT": "2"},
                  {"KVR_TALL_TPB": "20", "KVR_TALL_SPLIT": "1", "KVR_TALL_GU_SPLIT": "2"},
                  {"KVR_TALL_GU_SPLIT": "1"}, {"KVR_TALL": "0"}, {"KVR_TALL_ROWSCALE": "0"}]


@pytest.mark.parametrize("env", TALL_OVERRIDES, ids=["tpb5-split3", "tpb1-split7", "tpb12-unsplit", "tpb17-split2",
                                                     "tpb20-gu-split2", "fused-swiglu", "tiled", "per-row-norm"])
def test_mid_tall_plan_overrides(mid, monkeypatch, env):
    shape, eng, ow, toks, new, stale_np = mid
    for k, v in env.items():
        monkeypatch.setenv(k, v)
    A = osel.select_random(700, 300, 316, 128, 5)
    _repair_case(shape, eng, ow, stale_np, new, 300, 316, A, f"mid Random K=128, tall plan {env}", n_cap=704)


def test_mid_short_prefill_tall():
    """A 150-token prefill: every projection of the pass on the tall kernel."""
    shape, n = MID, 150
    eng, ow, toks = _setup(shape, kvr.KVR_BF16, n, n, seed=21)
    try:
        say(f"case: {shape.name} prefill n={n} (tall kernel)")
        cache = eng.new_cache(n)
        hidden = torch.empty((n, shape.d_model), device="cuda")
        eng.prefill(toks.cuda(), cache, hidden)
        torch.cuda.synchronize()
        oc, oy = od.prefill(shape, ow, toks.numpy())
        got = cache.to(torch.float64).cpu().numpy()
        errs = {(l, kv): relmax(got[l, kv], oc[l, kv]) for l in range(shape.n_layers) for kv in range(2)}
        errs["hidden"] = relmax(hidden.cpu().numpy(), oy)
        say(f"  {errs}")
        assert max(errs.values()) <= TOL[kvr.KVR_BF16]
    finally:
        eng.close()


@pytest.mark.parametrize("nt", ["2", "5"])
def test_ragged_gateup_blocks_across_groups(monkeypatch, nt):
    """Gate/up packed in groups of three tiles, read by blocks of two or five
    tiles: every block's tiles start inside a group or straddle two."""
    monkeypatch.setenv("KVR_NT_GATEUP", nt)
    shape, n = RAGGED, 700
    w = synth.make_weights(shape, dtype=torch.bfloat16, seed=9)
    eng = Engine(shape, to_device_weights(w), kvr.KVR_BF16, max_ctx=n, max_rows=64)
    try:
        toks = synth.make_tokens(n, shape.vocab, seed=10)
        ow = OracleWeights(w, cache=True)
        stale = synth.make_stale_cache(shape, n, label=9).to(torch.float64).numpy()
        new = synth.apply_edit(toks, 300, 16, shape.vocab)
        A = osel.select_edit_local(n, 300, 316, 32)
        _repair_case(shape, eng, ow, stale, new, 300, 316, A, f"{shape.name} gate/up blocks of {nt} tiles")
    finally:
        eng.close()


# head_dim 12 (even, not a multiple of 8) and d_model 48: RoPE and the cache
# scatter take the row kernel that stages the fused Q|K|V row in LDS, and the
# projections and attention the generic kernels (the MFMA paths need 64-wide
# shapes and head_dim 128).
ODD_HD = synth.ModelShape("odd-head-dim", 2, 48, 4, 2, 12, 80, 256, 1e-5, 10000.0)


def _prefill_then_repair(shape, dtype, n, seed, edit, tag):
    tdt = torch.bfloat16 if dtype == kvr.KVR_BF16 else torch.float32
    w = synth.make_weights(shape, dtype=tdt, seed=seed)
    eng = Engine(shape, to_device_weights(w), dtype, max_ctx=n, max_rows=64)
    try:
        toks = synth.make_tokens(n, shape.vocab, seed=seed + 1)
        cache = eng.new_cache(n)
        hidden = torch.empty((n, shape.d_model), device="cuda")
        say(f"case: {tag} prefill n={n}")
        eng.prefill(toks.cuda(), cache, hidden)
        torch.cuda.synchronize()
        ow = OracleWeights(w, cache=True)
        oc, oy = od.prefill(shape, ow, toks.numpy())
        got = cache.to(torch.float64).cpu().numpy()
        errs = {(l, kv): relmax(got[l, kv], oc[l, kv]) for l in range(shape.n_layers) for kv in range(2)}
        errs["hidden"] = relmax(hidden.cpu().numpy(), oy)
        say(f"  {errs}")
        assert max(errs.values()) <= TOL[dtype]
        s0, s1 = edit
        new = synth.apply_edit(toks, s0, s1 - s0, shape.vocab)
        A = osel.select_edit_local(n, s0, s1, 32)
        _repair_case(shape, eng, ow, oc, new, s0, s1, A, f"{tag} EditLocal K=32")
    finally:
        eng.close()


@pytest.mark.parametrize("dtype", [kvr.KVR_F32, kvr.KVR_BF16], ids=["f32", "bf16"])
def test_odd_head_dim_prefill_and_repair(dtype):
    _prefill_then_repair(ODD_HD, dtype, 200, 13, (60, 68), f"{ODD_HD.name} {'bf16' if dtype else 'f32'}")


def test_bf16_generic_kernels_forced(monkeypatch):
    """KVR_SIMPLE=1 at context creation switches a bf16 model that the MFMA
    kernels would take to the generic projection and attention kernels (the
    reference path for debugging); it must meet the same bound."""
    monkeypatch.setenv("KVR_SIMPLE", "1")
    _prefill_then_repair(MID, kvr.KVR_BF16, 300, 15, (100, 116), "mid-bf16 generic kernels")


@pytest.mark.parametrize("rt", ["16", "8", "4"])
def test_wide_prefill_forced_row_blocks(monkeypatch, rt):
    """Each of the tiled kernel's row-block shapes forced on the 1100-row
    prefill (69 row tiles of 16): 256 rows (eight wavefronts, three LDS
    stages; the launcher picks it only for grids of eight rounds or more),
    128 rows (two stages, two blocks per compute unit) and 64 rows; the last
    row block is partial in each."""
    monkeypatch.setenv("KVR_TILED_RT", rt)
    shape, n = WIDE, 1100
    w = synth.make_weights(shape, dtype=torch.bfloat16, seed=11)
    eng = Engine(shape, to_device_weights(w), kvr.KVR_BF16, max_ctx=n, max_rows=64)
    try:
        toks = synth.make_tokens(n, shape.vocab, seed=12)
        cache = eng.new_cache(n)
        hidden = torch.empty((n, shape.d_model), device="cuda")
        say(f"case: {shape.name} prefill n={n}, {16 * int(rt)}-row blocks")
        eng.prefill(toks.cuda(), cache, hidden)
        torch.cuda.synchronize()
        oc, oy = od.prefill(shape, OracleWeights(w), toks.numpy())
        got = cache.to(torch.float64).cpu().numpy()
        errs = {(l, kv): relmax(got[l, kv], oc[l, kv]) for l in range(shape.n_layers) for kv in range(2)}
        errs["hidden"] = relmax(hidden.cpu().numpy(), oy)
        say(f"  {errs}")
        assert max(errs.values()) <= TOL[kvr.KVR_BF16]
    finally:
        eng.close()
