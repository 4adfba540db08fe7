"""Checks that pin the fp64 reference to facts other than itself.

Each ``pin_*`` takes the reference module and raises ``AssertionError`` when
the module disagrees with a closed form, an invariant, a special case that
reduces to a simpler formula, or a brute-force evaluation on a tiny input.
``test_oracle_pins.py`` runs them on the real module; ``test_oracle_mutations.py``
runs them on copies with planted mistakes and requires each mistake to be caught.
"""
from __future__ import annotations

import math

import numpy as np

from paper_2508_10259_amd.workload import random_gaussian


def _rand(shape, *key, std=1.0):
    return random_gaussian(shape, 11, *key, std=std).astype(np.float64)


def tiny_params(D, key=0, n_layers=2, d=8, H=2, F=12, V=20, n_bins=6, std=0.4,
                eps=1e-5, theta=10000.0, gains=True):
    """Random small decoder with non-unit gains (so gain handling is exercised)."""
    dh = d // H
    cfg = D.Config(n_layers, d, H, dh, F, V, n_bins, eps, theta)
    r = lambda *s, k: _rand(s, key, k, std=std)
    g = (lambda *s, k: 1.0 + 0.3 * _rand(s, key, k)) if gains else (lambda *s, k: np.ones(s))
    embed = _rand((V, d), key, 90)
    head = _rand((V, d), key, 91, std=std)
    return D.Params(
        cfg,
        w_q=r(n_layers, d, d, k=1), w_k=r(n_layers, d, d, k=2), w_v=r(n_layers, d, d, k=3),
        w_o=r(n_layers, d, d, k=4), w_gate=r(n_layers, F, d, k=5), w_up=r(n_layers, F, d, k=6),
        w_down=r(n_layers, d, F, k=7), g_attn=g(n_layers, d, k=8), g_ffn=g(n_layers, d, k=9),
        g_final=g(d, k=10), embed=embed, head_bins=head[V - n_bins:],
    )


def _close(a, b, tol=1e-12, what=""):
    a, b = np.asarray(a, dtype=np.float64), np.asarray(b, dtype=np.float64)
    assert a.shape == b.shape, (what, a.shape, b.shape)
    err = float(np.max(np.abs(a - b))) if a.size else 0.0
    assert err <= tol, f"{what}: max abs err {err:.3e} > {tol:.1e}"


# ----------------------------------------------------------------------------
# building blocks


def pin_linear_bruteforce(D):
    """y[t][o] = sum_i W[o][i] x[t][i], evaluated with scalar loops."""
    w = _rand((3, 5), 1)
    x = _rand((4, 5), 2)
    y = D.linear(w, x)
    ref = [[sum(float(w[o, i]) * float(x[t, i]) for i in range(5)) for o in range(3)] for t in range(4)]
    _close(y, ref, 1e-13, "linear")


def pin_rms_closed_forms(D):
    """Constant vector: c / sqrt(c^2 + eps) * g.  Mean square of the output: m / (m + eps)."""
    d, eps = 6, 1e-3
    g = np.array([1.0, 2.0, 0.5, -1.0, 3.0, 1.0])
    c = -1.7
    out = D.rms_norm(np.full((1, d), c), g, eps)
    _close(out, (c / math.sqrt(c * c + eps)) * g[None], 1e-14, "rms const")
    x = _rand((3, 16), 3)
    m = np.mean(x * x, axis=-1)
    out = D.rms_norm(x, np.ones(16), eps)
    _close(np.mean(out * out, axis=-1), m / (m + eps), 1e-13, "rms mean square")
    # scale invariance with eps = 0
    _close(D.rms_norm(x * 7.5, np.ones(16), 0.0), D.rms_norm(x, np.ones(16), 0.0), 1e-13, "rms scale")


def pin_silu(D):
    """silu(0) = 0; silu(z) - silu(-z) = z; silu(1) = 1 / (1 + e^-1)."""
    z = np.linspace(-6, 6, 25)
    _close(D.silu(np.zeros(3)), np.zeros(3), 0.0, "silu(0)")
    _close(D.silu(z) - D.silu(-z), z, 1e-13, "silu odd part")
    _close(D.silu(np.array([1.0])), [1.0 / (1.0 + math.exp(-1.0))], 1e-15, "silu(1)")
    _close(D.silu(np.array([-2.0])), [-2.0 / (1.0 + math.exp(2.0))], 1e-15, "silu(-2)")


def pin_rope_dh2_is_rotation(D):
    """head_dim 2: theta_0 = 1, so position t rotates the pair by angle t."""
    x = np.array([[[0.3, -1.2]], [[2.0, 0.5]], [[-0.7, 0.9]]])  # [T=3, H=1, 2]
    pos = np.array([0, 1, 5])
    out = D.apply_rope(x, pos, 10000.0)
    for t in range(3):
        a, b = x[t, 0]
        c, s = math.cos(pos[t]), math.sin(pos[t])
        _close(out[t, 0], [a * c - b * s, a * s + b * c], 1e-15, f"rope dh2 t={pos[t]}")


def pin_rope_dh4_pairing(D):
    """head_dim 4, base 100: pair (0,2) turns by t, pair (1,3) by t/10."""
    x = np.array([[[1.0, 2.0, 3.0, 4.0]]])
    t = 3
    out = D.apply_rope(x, np.array([t]), 100.0)[0, 0]
    a0, a1, a2, a3 = 1.0, 2.0, 3.0, 4.0
    c0, s0 = math.cos(t), math.sin(t)
    c1, s1 = math.cos(t / 10.0), math.sin(t / 10.0)
    ref = [a0 * c0 - a2 * s0, a1 * c1 - a3 * s1, a0 * s0 + a2 * c0, a1 * s1 + a3 * c1]
    _close(out, ref, 1e-14, "rope dh4")


def pin_rope_invariants(D):
    """Identity at t=0, norm preserving, and q.k depends only on the position difference."""
    x = _rand((5, 3, 8), 4)
    _close(D.apply_rope(x, np.zeros(5, int), 10000.0), x, 0.0, "rope t=0")
    pos = np.array([0, 3, 17, 100, 1023])
    y = D.apply_rope(x, pos, 10000.0)
    _close(np.linalg.norm(y, axis=-1), np.linalg.norm(x, axis=-1), 1e-12, "rope norm")
    q, k = _rand((1, 1, 16), 5), _rand((1, 1, 16), 6)
    for (t, tau, c) in [(7, 2, 13), (40, 40, 300), (5, 0, 1000)]:
        s0 = np.sum(D.apply_rope(q, np.array([t]), 10000.0) * D.apply_rope(k, np.array([tau]), 10000.0))
        s1 = np.sum(D.apply_rope(q, np.array([t + c]), 10000.0) * D.apply_rope(k, np.array([tau + c]), 10000.0))
        _close(s0, s1, 1e-11, "rope relative")


def pin_softmax(D):
    """Rows sum to 1; shift invariant; [0, ln 3] -> [1/4, 3/4]; -inf -> 0."""
    s = _rand((4, 9), 7) * 5
    p = D.softmax(s)
    _close(np.sum(p, axis=-1), np.ones(4), 1e-14, "softmax sum")
    _close(D.softmax(s + 123.0), p, 1e-14, "softmax shift")
    _close(D.softmax(np.array([0.0, math.log(3.0)])), [0.25, 0.75], 1e-15, "softmax closed form")
    _close(D.softmax(np.array([1.0, -np.inf, 1.0])), [0.5, 0.0, 0.5], 0.0, "softmax -inf")


def pin_attention_t1_t2(D):
    """T=1: o = v0.  T=2 brute force: o1 = (e^s0 v0 + e^s1 v1) / (e^s0 + e^s1), s = q1.k / sqrt(dh)."""
    q, k, v = _rand((2, 1, 4), 8), _rand((2, 1, 4), 9), _rand((2, 1, 4), 10)
    pos = np.array([0, 1])
    o = D.causal_attention(q, k, v, pos, pos)
    _close(o[0, 0], v[0, 0], 1e-15, "attn t=0")
    s0 = float(np.dot(q[1, 0], k[0, 0])) / 2.0
    s1 = float(np.dot(q[1, 0], k[1, 0])) / 2.0
    e0, e1 = math.exp(s0), math.exp(s1)
    _close(o[1, 0], (e0 * v[0, 0] + e1 * v[1, 0]) / (e0 + e1), 1e-14, "attn t=1 brute force")
    # explicit scores: q=(2,0,0,0), keys (1,0,0,0) and 0 -> s = (1, 0)
    q = np.zeros((1, 1, 4)); q[0, 0, 0] = 2.0
    k = np.zeros((2, 1, 4)); k[0, 0, 0] = 1.0
    v = np.array([[[1.0, 0, 0, 0]], [[0, 1.0, 0, 0]]])
    o = D.causal_attention(q, k, v, np.array([1]), np.array([0, 1]))
    e = math.e
    _close(o[0, 0], [e / (e + 1), 1 / (e + 1), 0, 0], 1e-15, "attn scale")


def pin_attention_uniform_causal(D):
    """q = 0 gives uniform weights over the visible keys: o_t = mean(v_0..v_t)."""
    T = 6
    v = _rand((T, 2, 4), 11)
    k = _rand((T, 2, 4), 12)
    pos = np.arange(T)
    o = D.causal_attention(np.zeros((T, 2, 4)), k, v, pos, pos)
    for t in range(T):
        _close(o[t], np.mean(v[: t + 1], axis=0), 1e-14, f"attn uniform t={t}")


def pin_attention_heads_independent(D):
    """Head 1's output does not depend on head 0's inputs."""
    q, k, v = _rand((4, 2, 4), 13), _rand((4, 2, 4), 14), _rand((4, 2, 4), 15)
    pos = np.arange(4)
    o = D.causal_attention(q, k, v, pos, pos)
    q2, k2, v2 = q.copy(), k.copy(), v.copy()
    q2[:, 0] += 1.0; k2[:, 0] -= 2.0; v2[:, 0] *= 3.0
    o2 = D.causal_attention(q2, k2, v2, pos, pos)
    _close(o2[:, 1], o[:, 1], 1e-15, "attn head isolation")
    o1 = D.causal_attention(q[:, 1:], k[:, 1:], v[:, 1:], pos, pos)
    _close(o[:, 1:], o1, 1e-15, "attn single head")


def pin_argmax_lowest_tie(D):
    assert D.greedy(np.array([1.0, 3.0, 3.0, 2.0])) == 1
    assert D.greedy(np.array([5.0, 5.0])) == 0
    assert D.greedy(np.array([-1.0, -3.0, 0.5])) == 2


def pin_bin_embedding_row(D):
    """Bin b feeds back vocabulary id V - n_bins + b."""
    p = tiny_params(D, key=1, V=20, n_bins=6)
    for b in range(6):
        _close(D.bin_embedding(p, b), p.get("embed")[14 + b], 0.0, f"bin {b}")


def pin_embed_ids_rows(D):
    """Instruction ids look up rows of the embedding table directly: id i gives row i,
    including the first id, the last non-bin id and the last id; no ids give [0, d]."""
    p = tiny_params(D, key=1, V=20, n_bins=6)
    table = p.get("embed")
    ids = [0, 13, 7, 0, 19, 1]  # 13 = V - n_bins - 1, 19 = V - 1
    out = D.embed_ids(p, ids)
    assert out.shape == (len(ids), 8)
    for r, i in enumerate(ids):
        _close(out[r], table[i], 0.0, f"embed id {i}")
    assert D.embed_ids(p, []).shape == (0, 8)


# ----------------------------------------------------------------------------
# whole-decoder special cases


def pin_ffn_scalar_layer(D):
    """1 layer, d=2 (one head of 2), F=1, attention output projection zero.

    With W_o = 0 the layer is h = x + W_down (silu(W_gate u) * (W_up u)),
    u = rms(x) * g_ffn; with single-entry matrices that is scalar arithmetic.
    """
    a, b, c = 1.3, -0.6, 0.9
    gffn = np.array([[1.5, 1.0]])
    cfg = D.Config(1, 2, 1, 2, 1, 4, 2, 1e-5, 10000.0)
    z2 = np.zeros((1, 2, 2))
    p = D.Params(cfg, w_q=_rand((1, 2, 2), 20), w_k=_rand((1, 2, 2), 21), w_v=_rand((1, 2, 2), 22),
                 w_o=z2, w_gate=np.array([[[a, 0.0]]]), w_up=np.array([[[b, 0.0]]]),
                 w_down=np.array([[[c], [0.0]]]), g_attn=np.ones((1, 2)), g_ffn=gffn,
                 g_final=np.ones(2), embed=np.zeros((4, 2)), head_bins=np.zeros((2, 2)))
    x = np.array([[0.8, -2.1], [1.1, 0.4]])
    h, _ = D.forward(p, x)
    for t in range(2):
        x0, x1 = x[t]
        r = 1.0 / math.sqrt((x0 * x0 + x1 * x1) / 2 + 1e-5)
        u0 = x0 * r * 1.5
        gte, up = a * u0, b * u0
        y0 = c * (gte / (1 + math.exp(-gte))) * up
        _close(h[t], [x0 + y0, x1], 1e-14, f"ffn scalar t={t}")


def pin_zero_blocks_logits(D):
    """With W_o = W_down = 0 the hidden state is the input and logits = head_bins @ rms(x)*g."""
    p = tiny_params(D, key=2, n_layers=3)
    p.arrays["w_o"] = np.zeros_like(p.arrays["w_o"])
    p.arrays["w_down"] = np.zeros_like(p.arrays["w_down"])
    x = _rand((5, 8), 30)
    h, _ = D.forward(p, x)
    _close(h, x, 0.0, "identity layers")
    xl = x[-1]
    r = 1.0 / math.sqrt(sum(float(t) * float(t) for t in xl) / 8 + 1e-5)
    g = p.get("g_final"); hb = p.get("head_bins")
    ref = [sum(float(hb[i, k]) * float(xl[k]) * r * float(g[k]) for k in range(8)) for i in range(6)]
    _close(D.bin_logits(p, xl), ref, 1e-13, "zero-block logits")


def pin_uniform_attention_layer(D):
    """W_q = 0 makes attention uniform: with W_down = 0 and unit gains,
    h_t = x_t + W_o W_v mean_{tau<=t} rms(x_tau)."""
    p = tiny_params(D, key=3, n_layers=1, gains=False)
    p.arrays["w_q"] = np.zeros_like(p.arrays["w_q"])
    p.arrays["w_down"] = np.zeros_like(p.arrays["w_down"])
    x = _rand((5, 8), 31)
    h, _ = D.forward(p, x)
    u = x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + 1e-5)
    wv, wo = p.layer("w_v", 0), p.layer("w_o", 0)
    for t in range(5):
        _close(h[t], x[t] + wo @ (wv @ np.mean(u[: t + 1], axis=0)), 1e-13, f"uniform layer t={t}")


def pin_causality(D):
    """Changing token t+1 leaves outputs 0..t unchanged; changing token t changes output t."""
    p = tiny_params(D, key=4)
    x = _rand((6, 8), 32)
    h, _ = D.forward(p, x)
    y = x.copy(); y[4] += 1.0
    h2, _ = D.forward(p, y)
    _close(h2[:4], h[:4], 0.0, "causal prefix")
    assert np.max(np.abs(h2[4] - h[4])) > 1e-3


def pin_head_permutation(D):
    """Relabelling heads (row blocks of W_q/W_k/W_v, column blocks of W_o) changes nothing."""
    p = tiny_params(D, key=5, d=12, H=3)
    dh = 4
    perm = [2, 0, 1]
    idx = np.concatenate([np.arange(h * dh, (h + 1) * dh) for h in perm])
    q = D.Params(p.cfg, **dict(p.arrays))
    for n in ("w_q", "w_k", "w_v"):
        q.arrays[n] = p.arrays[n][:, idx, :]
    q.arrays["w_o"] = p.arrays["w_o"][:, :, idx]
    x = _rand((7, 12), 33)
    _close(D.forward(q, x)[0], D.forward(p, x)[0], 1e-12, "head permutation")


def _bf_layer(p, l, xs):
    """Scalar-loop evaluation of one pre-norm layer over tokens xs (lists), positions 0..T-1."""
    cfg = p.cfg
    d, H, dh, F = cfg.d_model, cfg.n_heads, cfg.head_dim, cfg.d_ffn
    W = {n: p.layer(n, l).tolist() for n in ("w_q", "w_k", "w_v", "w_o", "w_gate", "w_up", "w_down")}
    ga, gf = p.layer("g_attn", l).tolist(), p.layer("g_ffn", l).tolist()

    def norm(x, g):
        r = 1.0 / math.sqrt(sum(t * t for t in x) / len(x) + cfg.rms_eps)
        return [x[i] * r * g[i] for i in range(len(x))]

    def mv(m, x):
        return [sum(m[o][i] * x[i] for i in range(len(x))) for o in range(len(m))]

    def rot(vec, t):
        out = list(vec)
        for hh in range(H):
            for i in range(dh // 2):
                ang = t * cfg.rope_theta ** (-2.0 * i / dh)
                a, b = vec[hh * dh + i], vec[hh * dh + i + dh // 2]
                out[hh * dh + i] = a * math.cos(ang) - b * math.sin(ang)
                out[hh * dh + i + dh // 2] = a * math.sin(ang) + b * math.cos(ang)
        return out

    us = [norm(x, ga) for x in xs]
    qs = [rot(mv(W["w_q"], u), t) for t, u in enumerate(us)]
    ks = [rot(mv(W["w_k"], u), t) for t, u in enumerate(us)]
    vs = [mv(W["w_v"], u) for u in us]
    out = []
    for t, x in enumerate(xs):
        o = [0.0] * d
        for hh in range(H):
            sl = range(hh * dh, (hh + 1) * dh)
            s = [sum(qs[t][i] * ks[tau][i] for i in sl) / math.sqrt(dh) for tau in range(t + 1)]
            mx = max(s)
            e = [math.exp(si - mx) for si in s]
            z = sum(e)
            for i in sl:
                o[i] = sum(e[tau] * vs[tau][i] for tau in range(t + 1)) / z
        h = [x[i] + a for i, a in enumerate(mv(W["w_o"], o))]
        u = norm(h, gf)
        g, up = mv(W["w_gate"], u), mv(W["w_up"], u)
        a = [g[j] / (1.0 + math.exp(-g[j])) * up[j] for j in range(F)]
        out.append([h[i] + y for i, y in enumerate(mv(W["w_down"], a))])
    return out


def pin_layer_bruteforce(D):
    """Two layers, d=4 (2 heads of 2), F=3, 3 tokens: against scalar loops written from the definition."""
    p = tiny_params(D, key=9, n_layers=2, d=4, H=2, F=3, V=5, n_bins=3, theta=7.0)
    x = _rand((3, 4), 34)
    xs = x.tolist()
    for l in range(2):
        xs = _bf_layer(p, l, xs)
    h, _ = D.forward(p, x)
    _close(h, xs, 1e-13, "layer brute force")


# ----------------------------------------------------------------------------
# the action context against the definition


def _ctx_vs_full(D, p, prefixes, news, n_actions, forced=None, tol=1e-12):
    ctx = D.ActionContext(p, len(prefixes))
    ctx.build(prefixes)
    seqs = [np.asarray(x) for x in prefixes]
    for s, new in enumerate(news):
        f = None if forced is None else forced[s]
        t1, z1 = ctx.step(new, n_actions, f)
        t0, z0, seqs = D.full_step(p, seqs, new, n_actions, f)
        _close(z1, z0, tol, f"cached vs full logits step {s}")
        assert np.array_equal(t1, t0), f"cached vs full tokens step {s}"
        assert list(ctx.lengths()) == [len(x) for x in seqs]
    return ctx, seqs


def pin_cached_equals_full(D):
    """Reusing the context gives the full-recomputation result (to 1e-12), K/V included."""
    p = tiny_params(D, key=6, n_layers=2)
    prefixes = [_rand((5, 8), 40), _rand((3, 8), 41), _rand((8, 8), 42)]
    news = [None, [_rand((2, 8), 43), None, _rand((1, 8), 44)], [None, _rand((3, 8), 45), None]]
    ctx, seqs = _ctx_vs_full(D, p, prefixes, news, n_actions=4)
    for b in range(3):
        _, kv_full = D.forward(p, seqs[b])
        for l in range(2):
            _close(ctx.kv[b][l][0], kv_full[l][0], 1e-12, f"K row {b} layer {l}")
            _close(ctx.kv[b][l][1], kv_full[l][1], 1e-12, f"V row {b} layer {l}")
    forced = [np.array([[1, 2, 3], [0, 0, 0], [5, 4, 3]])]
    _ctx_vs_full(D, p, prefixes, [None], n_actions=4, forced=forced)


def pin_forced_decoding(D):
    """Teacher forcing: the logits of action j are those of a plain forward pass over the
    committed sequence followed by the embeddings (table rows V - n_bins + f) of the forced
    bins f_0..f_{j-1}, in both the full-recomputation and the cached path; the reported
    tokens stay the argmax of those logits."""
    p = tiny_params(D, key=10, V=20, n_bins=6)
    table = p.get("embed")
    seq = _rand((5, 8), 70)
    forced = [4, 1, 5]
    direct = []
    for j in range(4):
        x = np.concatenate([seq] + [table[14 + f][None] for f in forced[:j]], axis=0)
        h, _ = D.forward(p, x)
        direct.append(D.bin_logits(p, h[-1]))
    direct = np.stack(direct)
    t_full, z_full = D.full_decode(p, seq, 4, forced)
    _close(z_full, direct, 1e-12, "forced full_decode")
    assert list(t_full) == [int(np.argmax(z)) for z in direct]
    ctx = D.ActionContext(p, 1)
    ctx.build([seq])
    t_c, z_c = ctx.step(None, 4, np.array([forced]))
    _close(z_c[0], direct, 1e-12, "forced cached step")
    assert list(t_c[0]) == list(t_full)
    # the forced bins differ from the free-running choices, so forcing is observable
    t_free, _ = D.full_decode(p, seq, 4)
    assert list(t_free[:3]) != forced


def pin_rows_independent(D):
    """Row b of a ragged batch equals a solo run of row b, bit for bit."""
    p = tiny_params(D, key=7)
    prefixes = [_rand((4, 8), 50), _rand((9, 8), 51)]
    new = [_rand((2, 8), 52), None]
    ctx = D.ActionContext(p, 2); ctx.build(prefixes)
    t, z = ctx.step(new, 3)
    for b in range(2):
        solo = D.ActionContext(p, 1); solo.build([prefixes[b]])
        ts, zs = solo.step([new[b]], 3)
        assert np.array_equal(ts[0], t[b]) and np.array_equal(zs[0], z[b])


def pin_lifecycle(D):
    """invalidate + build(P) == fresh build(P); step(N), step() == build(P||N), step();
    stepping an invalidated context is an error."""
    p = tiny_params(D, key=8)
    P, N = _rand((6, 8), 60), _rand((3, 8), 61)
    a = D.ActionContext(p, 1); a.build([P])
    a.step([N], 3)
    ta, za = a.step(None, 3)
    b = D.ActionContext(p, 1); b.build([np.concatenate([P, N])])
    tb, zb = b.step(None, 3)
    _close(za, zb, 1e-12, "commit semantics")
    a.invalidate()
    try:
        a.step(None, 3)
        raise AssertionError("step after invalidate must fail")
    except RuntimeError:
        pass
    a.build([P])
    c = D.ActionContext(p, 1); c.build([P])
    _close(a.step(None, 3)[1], c.step(None, 3)[1], 0.0, "rebuild == fresh")


def pin_row_lifecycle(D):
    """One row of a batch invalidated and rebuilt from a new prefix: that row then equals a fresh
    context built from the new prefix, the other rows equal a batch that never saw the row
    operations (bit for bit: rows are independent); while the row is invalid the batch cannot
    step.  append(N) then step() equals step(N)."""
    p = tiny_params(D, key=12)
    P = [_rand((4 + 2 * b, 8), 80, b) for b in range(3)]
    P1 = _rand((7, 8), 81)
    N = [_rand((2, 8), 82, b) for b in range(3)]
    a = D.ActionContext(p, 3); a.build(P)
    ref = D.ActionContext(p, 3); ref.build(P)
    a.step(N, 3); ref.step(N, 3)
    a.invalidate_rows([1])
    assert list(a.lengths()) == [len(P[0]) + 2, 0, len(P[2]) + 2]
    try:
        a.step(None, 3)
        raise AssertionError("step with an invalidated row must fail")
    except RuntimeError:
        pass
    a.build_rows([1], [P1])
    ta, za = a.step(None, 3)
    tr, zr = ref.step(None, 3)
    for b in (0, 2):
        assert np.array_equal(ta[b], tr[b]) and np.array_equal(za[b], zr[b]), f"row {b} disturbed"
    fresh = D.ActionContext(p, 1); fresh.build([P1])
    tf, zf = fresh.step(None, 3)
    assert np.array_equal(ta[1], tf[0]) and np.array_equal(za[1], zf[0]), "rebuilt row != fresh build"
    # append-only commit
    c = D.ActionContext(p, 3); c.build(P)
    d_ = D.ActionContext(p, 3); d_.build(P)
    c.append(N)
    tc, zc = c.step(None, 3)
    td, zd = d_.step(N, 3)
    assert np.array_equal(tc, td) and np.array_equal(zc, zd), "append + step != step with new tokens"
    assert list(c.lengths()) == list(d_.lengths())


ALL_PINS = [v for k, v in sorted(globals().items()) if k.startswith("pin_")]
