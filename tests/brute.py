"""Brute-force scalar reference for tiny models (pure Python, no numpy).

Textbook incremental KV-cache decoding: a token at position p runs through
all layers alone, writes its key/value slot at every layer and attends over
slots 0..p of that layer.  Repairing a position set P over a stale cache is
the same as decoding the positions of P one at a time in ascending order over
that cache (each p depends only on slots t <= p, which are already fresh for
t in P and stale otherwise), so this loop pins the oracle's layer-by-layer
repair for scattered P as well as its full prefill.

Written independently of ``oracle/`` with scalar loops only; used on models
with a few dozen hidden units.
"""
import math


def _rmsnorm(x, g, eps):
    ms = sum(v * v for v in x) / len(x)
    r = 1.0 / math.sqrt(ms + eps)
    return [v * r * gi for v, gi in zip(x, g)]


def _matvec(w, x, b=None):
    out = []
    for i, row in enumerate(w):
        s = 0.0
        for a, c in zip(row, x):
            s += a * c
        out.append(s + (b[i] if b is not None else 0.0))
    return out


def _rotate(vec, pos, theta):
    hd = len(vec)
    half = hd // 2
    out = [0.0] * hd
    for i in range(half):
        ang = pos * theta ** (-2.0 * i / hd)
        c, s = math.cos(ang), math.sin(ang)
        a, b = vec[i], vec[i + half]
        out[i] = a * c - b * s
        out[i + half] = b * c + a * s
    return out


def decode_one(shape, W, cache, token, pos):
    """Run one token at position ``pos`` through every layer.

    W: dict with 'embed' (list of rows), 'final_norm', 'layers' (list of dicts of
    nested lists; matrices [out][in]).  cache[l][0|1][g][t] is a list of head_dim
    floats (mutable).  Returns the final-normed hidden vector.
    """
    Hq, Hkv, hd = shape.n_heads, shape.n_kv_heads, shape.head_dim
    G = Hq // Hkv
    h = list(W["embed"][token])
    for l, lw in enumerate(W["layers"]):
        x = _rmsnorm(h, lw["attn_norm"], shape.rms_eps)
        q = _matvec(lw["wq"], x, lw.get("bq"))
        k = _matvec(lw["wk"], x, lw.get("bk"))
        v = _matvec(lw["wv"], x, lw.get("bv"))
        for g in range(Hkv):
            cache[l][0][g][pos] = _rotate(k[g * hd:(g + 1) * hd], pos, shape.rope_theta)
            cache[l][1][g][pos] = list(v[g * hd:(g + 1) * hd])
        o = []
        for j in range(Hq):
            g = j // G
            qj = _rotate(q[j * hd:(j + 1) * hd], pos, shape.rope_theta)
            scores = []
            for t in range(pos + 1):
                kt = cache[l][0][g][t]
                scores.append(sum(a * b for a, b in zip(qj, kt)) / math.sqrt(hd))
            m = max(scores)
            e = [math.exp(s - m) for s in scores]
            z = sum(e)
            acc = [0.0] * hd
            for t in range(pos + 1):
                vt = cache[l][1][g][t]
                wt = e[t] / z
                for i in range(hd):
                    acc[i] += wt * vt[i]
            o.extend(acc)
        att = _matvec(lw["wo"], o)
        h = [a + b for a, b in zip(h, att)]
        x = _rmsnorm(h, lw["mlp_norm"], shape.rms_eps)
        gt = _matvec(lw["w_gate"], x)
        up = _matvec(lw["w_up"], x)
        a = [(gv / (1.0 + math.exp(-gv))) * uv for gv, uv in zip(gt, up)]
        mlp = _matvec(lw["w_down"], a)
        h = [p + r for p, r in zip(h, mlp)]
    return _rmsnorm(h, W["final_norm"], shape.rms_eps)


def empty_cache(shape, n):
    return [[[[None] * n for _ in range(shape.n_kv_heads)] for _ in range(2)]
            for _ in range(shape.n_layers)]


def prefill(shape, W, tokens):
    cache = empty_cache(shape, len(tokens))
    ys = [decode_one(shape, W, cache, int(t), p) for p, t in enumerate(tokens)]
    return cache, ys


def repair(shape, W, cache, tokens_new, P):
    """Decode the positions of P (ascending) over ``cache`` in place."""
    return [decode_one(shape, W, cache, int(tokens_new[p]), p) for p in sorted(P)]
