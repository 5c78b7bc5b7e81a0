"""GPU parity at the workloads' full sizes, in the launch configuration the
benchmark times (one kvr_repair call over the whole position set).

* Llama-3-8B shape (32 layers, d 4096, 32/8 heads x 128, FFN 14336, vocab
  128256), 5000-token context, 16-token edit at a seeded position in
  [1000, 4000], EditLocal K=32 (48 rows): every repaired output is compared
  with the oracle; and 128 rows at 4850-4977 with unsplit attention items
  (the prefill's variant) over ~4900 keys.  Prefill at n=5000 is checked on its first 32 rows (which
  depend only on the first 32 tokens) and, at any size, by the endpoint
  property (repairing every position equals prefill).
* Qwen2.5-7B shape (QKV bias, 28/4 heads): K in {8, 32, 128, 512} for both
  EditLocal and Random (seed 0), and Random K=32 at seeds 1-4.
* Mistral-7B shape: edit near the end (4900) and near the start (200).
* Batched repair, Llama-3-8B shape: 64 documents of 2000-8000 tokens, each with
  its own 16-token edit and EditLocal K=32, in one call (3072 rows); two
  documents are compared with the oracle in full, all of them for untouched
  slots.

The stale caches are synthetic (synth.make_stale_cache): repair is defined for
any stale cache, and the oracle repairs from exactly the same values.
Tolerance: 2e-2, max |gpu - oracle| / max |oracle| per tensor group.
"""
import numpy as np
import pytest
import torch

import paper_2609_17983_amd as kvr
import synth
from oracle import decoder as od
from oracle import select as osel
from oracle import selectors as osl
from tests.gpu_util import TOL, Engine, OracleWeights, compare_repair, relmax, say

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(900)]

N = 5000
SPAN = 16


def _engine(shape, max_rows=3072, max_ctx=8192):
    say(f"generating {shape.name} weights on the GPU")
    w = synth.make_weights(shape, dtype=torch.bfloat16, device="cuda")
    torch.cuda.synchronize()
    return Engine(shape, w, kvr.KVR_BF16, max_ctx=max_ctx, max_rows=max_rows)


def _release(eng):
    eng.close()
    eng.weights = None
    torch.cuda.empty_cache()


def _full_repair(eng, n, s0, s1, A, label=0, tag=""):
    shape = eng.shape
    toks = synth.make_tokens(n, shape.vocab)
    new = synth.apply_edit(toks, s0, s1 - s0, shape.vocab, label=label)
    stale = synth.make_stale_cache(shape, n, device="cuda", label=label)
    ref_in = stale.to(torch.float64).cpu().numpy()
    cache = stale.clone()
    P = od.repaired_set(s0, s1, A)
    hidden = torch.full((len(P), shape.d_model), float("nan"), device="cuda")
    say(f"{tag}: GPU repair of {len(P)} rows")
    eng.repair([dict(cache=cache, tokens=new.cuda(), edit_start=s0, edit_end=s1, positions=A, hidden=hidden)])
    torch.cuda.synchronize()
    say(f"{tag}: oracle repair")
    oc = ref_in
    y = od.repair(shape, OracleWeights(eng.weights), oc, new.numpy(), s0, s1, A)
    return compare_repair(shape, None, stale, cache, hidden, oc, y, P, n, TOL[kvr.KVR_BF16], tag)


@pytest.fixture(scope="module")
def llama():
    eng = _engine(synth.LLAMA3_8B)
    yield eng
    _release(eng)


def test_llama8b_repair_edit_local(llama):
    e = synth.edit_position(1000, 4000)
    A = osel.select_edit_local(N, e, e + SPAN, 32)
    _full_repair(llama, N, e, e + SPAN, A, tag=f"llama8b n=5000 edit@{e} EditLocal K=32")


def test_llama8b_long_key_unsplit_attention(llama, monkeypatch):
    """The prefill's attention variant (64-row items, one key group, every
    key of the row block in one item) over ~4900 keys at full size: 128 rows
    at the end of a 5000-token context, with the attention planner's target
    forced so low that no key range is split."""
    monkeypatch.setenv("KVR_ATT_TARGET", "1")
    e = 4850
    A = osel.select_edit_local(N, e, e + SPAN, 112)
    _full_repair(llama, N, e, e + SPAN, A, tag=f"llama8b n=5000 edit@{e} EditLocal K=112, unsplit attention")


def test_llama8b_prefill_prefix(llama):
    shape = llama.shape
    toks = synth.make_tokens(N, shape.vocab)
    cache = llama.new_cache(N)
    hidden = torch.empty((N, shape.d_model), device="cuda")
    say("llama8b prefill n=5000")
    llama.prefill(toks.cuda(), cache, hidden)
    torch.cuda.synchronize()
    m = 32
    say("llama8b oracle prefill of the first 32 tokens")
    oc, oy = od.prefill(shape, OracleWeights(llama.weights), toks[:m].numpy())
    got = cache[:, :, :, :m].to(torch.float64).cpu().numpy()
    errs = {f"{'KV'[kv]}{l}": relmax(got[l, kv], oc[l, kv]) for l in range(shape.n_layers) for kv in range(2)}
    errs["hidden"] = relmax(hidden[:m].cpu().numpy(), oy)
    worst = max(errs, key=errs.get)
    say(f"llama8b prefill prefix worst {worst}={errs[worst]:.3e}")
    assert errs[worst] <= TOL[kvr.KVR_BF16]
    assert torch.isfinite(hidden).all()


def test_llama8b_endpoint_property(llama):
    """Eq. 1 at full size: repairing every position of a stale cache equals
    the prefill of C' (GPU against GPU: a property that holds at any size)."""
    shape = llama.shape
    n = 3072
    toks = synth.make_tokens(n, shape.vocab, seed=9)
    pre = llama.new_cache(n)
    h_pre = torch.empty((n, shape.d_model), device="cuda")
    llama.prefill(toks.cuda(), pre, h_pre)
    stale = synth.make_stale_cache(shape, n, device="cuda", label=3)
    h_rep = torch.empty_like(h_pre)
    llama.repair([dict(cache=stale, tokens=toks.cuda(), edit_start=0, edit_end=16, positions=list(range(16, n)),
                       hidden=h_rep)])
    torch.cuda.synchronize()
    e_cache = relmax(stale.to(torch.float64).cpu().numpy(), pre.to(torch.float64).cpu().numpy())
    e_h = relmax(h_rep.cpu().numpy(), h_pre.cpu().numpy())
    say(f"llama8b endpoint: cache {e_cache:.3e} hidden {e_h:.3e}")
    assert e_cache <= TOL[kvr.KVR_BF16] and e_h <= TOL[kvr.KVR_BF16]


def test_llama8b_attention_selector(llama):
    """Attention selector at full size: a 16-token query over a 5000-position
    synthetic stale cache; the per-position mass is compared with the oracle
    in full, the selection where it is decided by a clear gap."""
    shape = llama.shape
    q, K = 16, 32
    e = synth.edit_position(1000, 4000, label=5)
    toks = synth.make_tokens(N + q, shape.vocab, seed=21)
    cache = synth.make_stale_cache(shape, N + q, device="cuda", label=21)
    ref_in = cache.to(torch.float64).cpu().numpy()
    out = torch.full((K,), -1, dtype=torch.int32, device="cuda")
    mass = torch.empty(N, device="cuda")
    say(f"llama8b attention selector n={N} q={q} edit@{e}")
    cnt = kvr.kvr_select_attention(llama.ctx, cache.data_ptr(), N, N + q, toks.cuda().data_ptr(), q, e, e + SPAN, K,
                                   out.data_ptr(), mass.data_ptr(), torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    assert cnt == K
    say("llama8b attention selector: oracle mass")
    ref = osl.attention_mass(shape, OracleWeights(llama.weights), ref_in, toks.numpy(), N, q)
    got = mass.cpu().numpy().astype(np.float64)
    err = relmax(got, ref)
    say(f"llama8b attention selector: mass err {err:.3e}")
    assert err <= TOL[kvr.KVR_BF16]
    sel = out.cpu().tolist()
    D0 = e + SPAN
    assert sel == osl.top_k_positions(got[D0:N - 1], D0, K)
    srt = np.sort(ref[D0:N - 1])[::-1]
    band = 2 * TOL[kvr.KVR_BF16] * np.max(ref)
    sure = {D0 + i for i in range(N - 1 - D0) if ref[D0 + i] > srt[K - 1] + band}
    assert sure <= set(sel)


def test_llama8b_score(llama):
    """Fresh-query scoring at full size: 24 tokens appended after a 5000-position
    synthetic cache, LM head tied to the 128256-entry embedding; teacher-forced
    log-probabilities against the oracle, argmax where the top-two gap is clear."""
    from oracle import scoring as osc
    shape = llama.shape
    m = 24
    toks = synth.make_tokens(N + m, shape.vocab, seed=31)
    cache = synth.make_stale_cache(shape, N + m, device="cuda", label=31)
    ref_in = cache.to(torch.float64).cpu().numpy()
    lp = torch.empty(m - 1, device="cuda")
    am = torch.empty(m, dtype=torch.int32, device="cuda")
    say(f"llama8b score n={N} m={m}")
    kvr.kvr_score(llama.ctx, cache.data_ptr(), N, N + m, toks.cuda().data_ptr(), m, lp.data_ptr(), am.data_ptr(),
                  torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    say("llama8b score: oracle")
    ow = OracleWeights(llama.weights)
    lm = llama.weights["embed"].to(torch.float64).cpu().numpy()
    ref_lp, ref_am = osc.score(shape, ow, lm, ref_in.copy(), toks.numpy(), N, m)
    err = relmax(lp.cpu().numpy(), ref_lp)
    say(f"llama8b score: logprob err {err:.3e}")
    assert err <= TOL[kvr.KVR_BF16]
    y = od.repair(shape, ow, ref_in.copy(), toks.numpy(), N, N + m, [])
    logits = y @ lm.T
    top2 = np.sort(logits, axis=-1)[:, -2:]
    clear = (top2[:, 1] - top2[:, 0]) > 2e-3 * np.max(np.abs(logits))
    say(f"llama8b score: {int(clear.sum())} of {m} argmax decisions clear")
    assert np.array_equal(am.cpu().numpy()[clear], ref_am[clear])


def test_llama8b_batched_64_docs(llama):
    shape = llama.shape
    lens = synth.doc_lengths(64, 2000, 8000)
    docs, keep = [], {}
    check = {0, 37}
    for i, L in enumerate(lens):
        e = synth.edit_position(int(0.2 * L), int(0.8 * L) - SPAN, label=i)
        A = osel.select_edit_local(L, e, e + SPAN, 32)
        toks = synth.make_tokens(L, shape.vocab, seed=100 + i)
        new = synth.apply_edit(toks, e, SPAN, shape.vocab, label=i)
        stale = synth.make_stale_cache(shape, L, device="cuda", label=100 + i)
        P = od.repaired_set(e, e + SPAN, A)
        hidden = torch.full((len(P), shape.d_model), float("nan"), device="cuda")
        ref_in = stale.to(torch.float64).cpu().numpy() if i in check else None
        keep[i] = (stale.clone(), ref_in, new, e, A, P)
        docs.append(dict(cache=stale, tokens=new.cuda(), edit_start=e, edit_end=e + SPAN, positions=A, hidden=hidden))
    assert sum(len(k[5]) for k in keep.values()) == 3072
    say("batched: GPU repair of 64 documents (3072 rows)")
    llama.repair(docs)
    torch.cuda.synchronize()
    for i, d in enumerate(docs):
        stale0, ref_in, new, e, A, P = keep[i]
        assert torch.isfinite(d["hidden"]).all()
        if ref_in is None:
            mask = torch.ones(lens[i], dtype=torch.bool, device="cuda")
            mask[torch.as_tensor(P, device="cuda")] = False
            assert torch.equal(d["cache"][:, :, :, mask], stale0[:, :, :, mask])
            continue
        say(f"batched: oracle repair of document {i} (n={lens[i]}, edit@{e})")
        oc = ref_in
        y = od.repair(shape, OracleWeights(llama.weights), oc, new.numpy(), e, e + SPAN, A)
        compare_repair(shape, None, stale0, d["cache"], d["hidden"], oc, y, P, lens[i], TOL[kvr.KVR_BF16],
                       f"batched doc {i}")


@pytest.fixture(scope="module")
def qwen():
    eng = _engine(synth.QWEN25_7B, max_rows=1024)
    yield eng
    _release(eng)


# The Qwen2.5-7B sweep: K in {8, 32, 128, 512} for the EditLocal window and
# for the Random policy (seed 0), and the Random policy's other four seeds at
# K = 32 (Table 1 runs it over five seeds).  Random sets scatter 8-512 rows
# over [edit_end, n - 1): attention row blocks then span thousands of
# positions and most key tiles take the masked path.
QWEN_SWEEP = ([(p, K, 0) for p in ("edit_local", "random") for K in (8, 32, 128, 512)] +
              [("random", 32, seed) for seed in (1, 2, 3, 4)])


@pytest.mark.parametrize("policy,K,seed", QWEN_SWEEP, ids=[f"{p}-K{K}-seed{s}" for p, K, s in QWEN_SWEEP])
def test_qwen7b_repair(qwen, policy, K, seed):
    e = synth.edit_position(1000, 4000)
    A = (osel.select_edit_local(N, e, e + SPAN, K) if policy == "edit_local"
         else osel.select_random(N, e, e + SPAN, K, seed))
    assert len(A) == K
    _full_repair(qwen, N, e, e + SPAN, A, tag=f"qwen7b edit@{e} {policy} K={K} seed={seed}")


@pytest.fixture(scope="module")
def mistral():
    eng = _engine(synth.MISTRAL_7B, max_rows=1024)
    yield eng
    _release(eng)


@pytest.mark.parametrize("e", [4900, 200])
def test_mistral7b_repair(mistral, e):
    A = osel.select_edit_local(N, e, e + SPAN, 32)
    _full_repair(mistral, N, e, e + SPAN, A, tag=f"mistral7b edit@{e} EditLocal K=32")
