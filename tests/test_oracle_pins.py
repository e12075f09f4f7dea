"""Pins of the fp64 oracle against what the paper and the mathematics fix.

No test here retypes an oracle formula to compare with itself.  Each check is
one of: a closed form, an invariant the paper states or implies, a special case
that reduces to a textbook routine, or brute force with pure-Python loops on
tiny inputs.  tests/test_oracle_mutations.py plants plausible mistakes in the
oracle and shows that each one makes at least one of these checks fail.
"""
import math

import numpy as np
import pytest

from oracle import dflare_oracle as orc
from paper_2606_02091_amd import synth

MICRO = synth.ModelConfig("micro", hidden=32, n_q_heads=4, n_kv_heads=2, head_dim=8, ffn=48,
                          vocab=64, n_draft_layers=2, n_target_layers=3, block_size=4,
                          context=6, random_block=True)


def micro_weights(cfg=MICRO, seed=0):
    w = synth.make_weights(cfg, seed=seed, threads=1)
    logits = w.pop("fusion_logits")
    return w, logits


def rel(a, b):
    return float(np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300))


def build(cfg, w, logits, L, seed=1):
    o = orc.DraftOracle(cfg, w, logits)
    if L:
        o.append(synth.hidden_rows(cfg, 0, L, seed=seed))
    return o


def f64(u):
    return orc.bf16_to_f64(u)


def bf16(x):
    return synth.round_bf16(np.asarray(x, np.float32))


# --------------------------------------------------------------------------------------
# fusion weights (Sec. 4.1, Eq. 3 first line; cached at inference)
# --------------------------------------------------------------------------------------

def check_alpha_sums_to_one():
    rng = np.random.default_rng(5)
    lg = rng.standard_normal((7, 9)) * 3
    a = orc.fusion_weights(lg)
    assert a.shape == (7, 9)
    assert np.all(np.abs(a.sum(axis=1) - 1.0) <= 9 * 2.0 ** -52)
    assert np.all(a > 0)


def check_alpha_two_layer_logistic():
    # softmax of two logits is the logistic function of their difference
    for l0, l1 in [(0.3, -1.2), (2.0, 2.0), (-4.0, 1.5)]:
        a = orc.fusion_weights(np.array([[l0, l1]]))
        assert abs(a[0, 0] - 1.0 / (1.0 + math.exp(l1 - l0))) < 1e-15
        assert abs(a[0, 1] - 1.0 / (1.0 + math.exp(l0 - l1))) < 1e-15


def check_alpha_extremes():
    a = orc.fusion_weights(np.zeros((2, 5)))
    assert np.all(a == 0.2)
    # a logit 1e4 below the others gives an exact zero weight (e^-1e4 underflows)
    a = orc.fusion_weights(np.array([[0.0, -1e4, 0.0]]))
    assert a[0, 1] == 0.0 and a[0, 0] == 0.5
    # large logits must not overflow: softmax is shift invariant
    a = orc.fusion_weights(np.array([[1000.0, 1001.0, 999.0]]))
    b = np.exp([0.0, 1.0, -1.0]) / np.exp([0.0, 1.0, -1.0]).sum()
    assert np.allclose(a[0], b, rtol=1e-14, atol=0)


def test_alpha_sums_to_one():
    check_alpha_sums_to_one()


def test_alpha_two_layer_logistic():
    check_alpha_two_layer_logistic()


def test_alpha_extremes_and_errors():
    check_alpha_extremes()
    with pytest.raises(ValueError):
        orc.fusion_weights(np.array([[0.0, np.nan]]))
    with pytest.raises(ValueError):
        orc.fusion_weights(np.array([[-np.inf, -np.inf]]))
    with pytest.raises(ValueError):
        orc.fusion_weights(np.array([[0.0, np.inf]]))


def test_fusion_parameter_count():
    # Sec. 4.1: the fusion adds D x T scalars, 63 for D = 7, T = 9 (tests/golden/paper_values.json)
    import json
    import os
    with open(os.path.join(os.path.dirname(__file__), "golden", "paper_values.json")) as fh:
        g = json.load(fh)["fusion_parameter_count"]
    assert orc.fusion_weights(np.zeros((g["D"], g["T"]))).size == g["count"]


# --------------------------------------------------------------------------------------
# RMSNorm and RoPE building blocks
# --------------------------------------------------------------------------------------

def check_rmsnorm_closed_form():
    eps = 1e-6
    x = np.array([[3.0, 4.0]])
    r = math.sqrt((9.0 + 16.0) / 2.0 + eps)
    g = np.array([2.0, -0.5])
    y = orc.rms_norm(x, g, eps)
    assert abs(y[0, 0] - 2.0 * 3.0 / r) < 1e-15 and abs(y[0, 1] + 0.5 * 4.0 / r) < 1e-15
    c = -7.0
    y = orc.rms_norm(np.full((1, 16), c), None, eps)
    assert np.allclose(y, c / math.sqrt(c * c + eps), rtol=1e-15, atol=0)


def check_rope_unit_vectors():
    hd, base = 8, 1.0e6
    for m in range(hd):
        x = np.zeros((1, 1, hd))
        x[0, 0, m] = 1.0
        p = 37.0
        j = m % (hd // 2)
        theta = p / (base ** (2.0 * j / hd))
        y = orc.rope(x, [p], base)[0, 0]
        e = np.zeros(hd)
        if m < hd // 2:   # first half rotates into its partner m + hd/2
            e[m], e[m + hd // 2] = math.cos(theta), math.sin(theta)
        else:             # second half rotates into m - hd/2 with the opposite sign
            e[m], e[m - hd // 2] = math.cos(theta), -math.sin(theta)
        assert np.allclose(y, e, rtol=0, atol=1e-15), (m, y, e)
    # position 0 is the identity
    x = np.random.default_rng(1).standard_normal((3, 2, hd))
    assert np.array_equal(orc.rope(x, [0, 0, 0], base), x)


def check_rope_relative():
    rng = np.random.default_rng(2)
    q = rng.standard_normal((1, 1, 16))
    k = rng.standard_normal((1, 1, 16))
    d0 = float(np.sum(orc.rope(q, [11.0], 1e4) * orc.rope(k, [4.0], 1e4)))
    d1 = float(np.sum(orc.rope(q, [111.0], 1e4) * orc.rope(k, [104.0], 1e4)))
    assert abs(d0 - d1) < 1e-12
    n0 = np.linalg.norm(q)
    assert abs(np.linalg.norm(orc.rope(q, [123.0], 1e4)) - n0) < 1e-13


def test_rmsnorm_closed_form():
    check_rmsnorm_closed_form()


def test_rope_unit_vectors():
    check_rope_unit_vectors()


def test_rope_relative_and_isometric():
    check_rope_relative()


# --------------------------------------------------------------------------------------
# layer fusion (Sec. 4.1, Eq. 3) and context K/V (Sec. 4.2, Eq. 4)
# --------------------------------------------------------------------------------------

def check_one_hot_fusion():
    """One-hot fusion logits reproduce conditioning on a single target layer exactly."""
    cfg = MICRO
    w, _ = micro_weights(cfg)
    hid = synth.hidden_rows(cfg, 0, 5)
    D, S = cfg.n_draft_layers, cfg.n_target_layers
    for pick in ([0, 2], [2, 1], [1, 0]):
        lg = np.full((D, S), -1e4)
        for i, j in enumerate(pick):
            lg[i, j] = 0.0
        o = orc.DraftOracle(cfg, w, lg)
        f = o.append(hid)
        for i, j in enumerate(pick):
            # single-layer model: S = 1, fed only target layer j
            c1 = cfg.replace(n_target_layers=1)
            w1 = dict(w)
            w1["fuse_norm"] = w["fuse_norm"][i:i + 1]
            w1["wk_t"], w1["wv_t"] = w["wk_t"][i:i + 1], w["wv_t"][i:i + 1]
            o1 = orc.DraftOracle(c1.replace(n_draft_layers=1), w1, np.zeros((1, 1)))
            f1 = o1.append(hid[j:j + 1])
            assert np.array_equal(f[i], f1[0])
            assert np.array_equal(o.k_cache[i], o1.k_cache[0])
            assert np.array_equal(o.v_cache[i], o1.v_cache[0])
            # and the fused row is the RMS-normalised hidden row times the gain
            h = f64(hid[j])
            r = np.sqrt(np.mean(h * h, axis=1, keepdims=True) + cfg.rms_eps)
            assert rel(f[i], h / r * f64(w["fuse_norm"][i])) < 1e-15


def check_identical_rows_alpha_free():
    cfg = MICRO
    w, _ = micro_weights(cfg)
    one = synth.hidden_rows(cfg, 0, 3)[:1]
    hid = np.repeat(one, cfg.n_target_layers, axis=0)
    ref = None
    for seed in range(3):
        lg = np.random.default_rng(seed).standard_normal((cfg.n_draft_layers, cfg.n_target_layers)) * 4
        f = orc.DraftOracle(cfg, w, lg).append(hid)
        if ref is None:
            ref = f
        assert rel(f, ref) < 1e-14


def check_context_kv_bruteforce():
    """K/V of appended rows by explicit loops: K[r,g,d] = RoPE(sum_k f[r,k] Wk[g*hd+d, k])."""
    cfg = MICRO
    w, lg = micro_weights(cfg)
    hid = synth.hidden_rows(cfg, 0, 3)
    o = orc.DraftOracle(cfg, w, lg)
    f = o.append(hid)
    H, nkv, hd = cfg.hidden, cfg.n_kv_heads, cfg.head_dim
    for i in range(cfg.n_draft_layers):
        wk, wv = f64(w["wk_t"][i]), f64(w["wv_t"][i])
        for r in range(3):
            for g in range(nkv):
                kr = [sum(f[i, r, k] * wk[g * hd + d, k] for k in range(H)) for d in range(hd)]
                vr = [sum(f[i, r, k] * wv[g * hd + d, k] for k in range(H)) for d in range(hd)]
                rot = []
                for d in range(hd):
                    m = d % (hd // 2)
                    th = r / (cfg.rope_base ** (2.0 * m / hd))
                    if d < hd // 2:
                        rot.append(kr[d] * math.cos(th) - kr[d + hd // 2] * math.sin(th))
                    else:
                        rot.append(kr[d] * math.cos(th) + kr[d - hd // 2] * math.sin(th))
                assert np.allclose(o.k_cache[i][r, g], rot, rtol=1e-12, atol=1e-13)
                assert np.allclose(o.v_cache[i][r, g], vr, rtol=1e-12, atol=1e-13)


def check_incremental_equals_bulk():
    cfg = MICRO.replace(hidden=64)
    w, lg = micro_weights(cfg)
    n = 64
    hid = synth.hidden_rows(cfg, 0, n)
    bulk = orc.DraftOracle(cfg, w, lg)
    fb = bulk.append(hid)
    for sizes in ([8] * 8, list(synth.append_sizes(40, seed=9))):
        inc = orc.DraftOracle(cfg, w, lg)
        fs, s = [], 0
        for c in sizes:
            c = min(c, n - s)
            if c <= 0:
                break
            fs.append(inc.append(hid[:, s:s + c]))
            s += c
        assert s == n
        assert np.array_equal(np.concatenate(fs, axis=1), fb)          # fused rows: bitwise
        for i in range(cfg.n_draft_layers):
            assert rel(inc.k_cache[i], bulk.k_cache[i]) <= 1e-14
            assert rel(inc.v_cache[i], bulk.v_cache[i]) <= 1e-14


def test_one_hot_fusion_is_single_layer_conditioning():
    check_one_hot_fusion()


def test_identical_target_rows_make_alpha_irrelevant():
    check_identical_rows_alpha_free()


def test_context_kv_bruteforce():
    check_context_kv_bruteforce()


def test_incremental_append_equals_bulk():
    check_incremental_equals_bulk()


# --------------------------------------------------------------------------------------
# block attention (Sec. 3.2 drafting phase, Sec. 4.2)
# --------------------------------------------------------------------------------------

def brute_attention(q, kc, vc, kb, vb):
    """Pure-Python loops: softmax over all context and block keys of the KV head."""
    B, nq, hd = q.shape
    nkv = kb.shape[1]
    keys = [kc[j] for j in range(kc.shape[0])] + [kb[j] for j in range(B)]
    vals = [vc[j] for j in range(vc.shape[0])] + [vb[j] for j in range(B)]
    out = np.zeros((B, nq, hd))
    for b in range(B):
        for h in range(nq):
            g = (h * nkv) // nq
            s = [sum(q[b, h, d] * k[g, d] for d in range(hd)) / math.sqrt(hd) for k in keys]
            mx = max(s)
            e = [math.exp(x - mx) for x in s]
            z = sum(e)
            for d in range(hd):
                out[b, h, d] = sum(e[j] * vals[j][g, d] for j in range(len(keys))) / z
    return out


def check_attention_bruteforce():
    rng = np.random.default_rng(11)
    for (B, nq, nkv, hd, L) in [(4, 4, 2, 8, 6), (3, 6, 3, 4, 0), (2, 2, 1, 8, 5), (1, 4, 1, 4, 1)]:
        q = rng.standard_normal((B, nq, hd)) * 2
        kc, vc = rng.standard_normal((L, nkv, hd)), rng.standard_normal((L, nkv, hd))
        kb, vb = rng.standard_normal((B, nkv, hd)), rng.standard_normal((B, nkv, hd))
        assert rel(orc.block_attention(q, kc, vc, kb, vb), brute_attention(q, kc, vc, kb, vb)) < 1e-12


def check_uniform_attention():
    # zero queries: every score is 0, so the output is the plain mean of all values
    rng = np.random.default_rng(3)
    L, B, nq, nkv, hd = 5, 4, 4, 2, 8
    vc, vb = rng.standard_normal((L, nkv, hd)), rng.standard_normal((B, nkv, hd))
    o = orc.block_attention(np.zeros((B, nq, hd)), rng.standard_normal((L, nkv, hd)), vc,
                            rng.standard_normal((B, nkv, hd)), vb)
    mean = np.concatenate([vc, vb]).mean(axis=0)
    for h in range(nq):
        assert np.allclose(o[:, h], mean[h // 2][None, :], rtol=1e-14, atol=1e-15)


def check_single_key():
    # empty context and a one-position block: the only key is the row itself
    rng = np.random.default_rng(4)
    vb = rng.standard_normal((1, 2, 8))
    o = orc.block_attention(rng.standard_normal((1, 4, 8)), np.zeros((0, 2, 8)), np.zeros((0, 2, 8)),
                            rng.standard_normal((1, 2, 8)), vb)
    for h in range(4):
        assert np.array_equal(o[0, h], vb[0, h // 2])


def test_attention_bruteforce():
    check_attention_bruteforce()


def test_uniform_attention_closed_form():
    check_uniform_attention()


def test_single_key_attention():
    check_single_key()


# --------------------------------------------------------------------------------------
# whole block pass
# --------------------------------------------------------------------------------------

def brute_layer(X, lw, kc, vc, pos, cfg):
    """One draft layer with explicit loops (tiny shapes only)."""
    B, H = X.shape
    nq, nkv, hd, F = cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, cfg.ffn
    eps = cfg.rms_eps

    def norm(row, g):
        r = math.sqrt(sum(v * v for v in row) / len(row) + eps)
        return [row[k] / r * g[k] for k in range(len(row))]

    def lin(row, W):
        return [sum(row[k] * W[o, k] for k in range(len(row))) for o in range(W.shape[0])]

    def rot(vec, p):
        out = list(vec)
        for m in range(hd // 2):
            th = p / (cfg.rope_base ** (2.0 * m / hd))
            a, b = vec[m], vec[m + hd // 2]
            out[m] = a * math.cos(th) - b * math.sin(th)
            out[m + hd // 2] = b * math.cos(th) + a * math.sin(th)
        return out

    A = [norm(list(X[b]), lw["attn_norm"]) for b in range(B)]
    Q = np.array([[rot(lin(A[b], lw["wq"])[h * hd:(h + 1) * hd], pos[b]) for h in range(nq)] for b in range(B)])
    Kb = np.array([[rot(lin(A[b], lw["wk_d"])[g * hd:(g + 1) * hd], pos[b]) for g in range(nkv)] for b in range(B)])
    Vb = np.array([[lin(A[b], lw["wv_d"])[g * hd:(g + 1) * hd] for g in range(nkv)] for b in range(B)])
    O = brute_attention(Q, kc, vc, Kb, Vb).reshape(B, nq * hd)
    X1 = [[X[b, c] + v for c, v in enumerate(lin(list(O[b]), lw["wo"]))] for b in range(B)]
    out = []
    for b in range(B):
        M = norm(X1[b], lw["mlp_norm"])
        gt, up = lin(M, lw["w_gate"]), lin(M, lw["w_up"])
        hmid = [gt[f] / (1.0 + math.exp(-gt[f])) * up[f] for f in range(F)]
        out.append([X1[b][c] + v for c, v in enumerate(lin(hmid, lw["w_down"]))])
    return np.array(out)


def check_block_pass_bruteforce():
    cfg = MICRO
    w, lg = micro_weights(cfg, seed=4)
    o = build(cfg, w, lg, L=5)
    ids = np.array([3, 63, 63, 17])
    res = o.draft_block(ids)
    X = f64(w["embed"][ids])
    pos = [5, 6, 7, 8]
    for i in range(cfg.n_draft_layers):
        X = brute_layer(X, o.layer_weights(i), o.k_cache[i], o.v_cache[i], pos, cfg)
        assert rel(res["hidden"][i], X) < 1e-12
    gf, wl = f64(w["final_norm"]), f64(w["lm_head"])
    for b in range(len(ids)):
        r = math.sqrt(sum(v * v for v in X[b]) / cfg.hidden + cfg.rms_eps)
        xn = [X[b, k] / r * gf[k] for k in range(cfg.hidden)]
        z = [sum(xn[k] * wl[v, k] for k in range(cfg.hidden)) for v in range(cfg.vocab)]
        assert np.allclose(res["logits"][b], z, rtol=1e-11, atol=1e-12)
        best = max(range(cfg.vocab), key=lambda v: (z[v], -v))
        assert res["tokens"][b] == best


def check_joint_permutation():
    """Permuting block ids together with their positions permutes every output."""
    cfg = MICRO
    w, lg = micro_weights(cfg, seed=6)
    o = build(cfg, w, lg, L=6)
    ids = np.array([5, 9, 63, 40])
    pos = np.array([6, 7, 8, 9])
    base = o.draft_block(ids, positions=pos)
    for perm in ([1, 0, 2, 3], [3, 2, 1, 0], [2, 3, 0, 1]):
        p = np.array(perm)
        r = o.draft_block(ids[p], positions=pos[p])
        assert rel(r["hidden"], base["hidden"][:, p]) < 1e-12
        assert rel(r["logits"], base["logits"][p]) < 1e-12
        assert np.array_equal(r["tokens"], base["tokens"][p])


def check_gqa_equals_duplicated_mha():
    cfg = MICRO
    w, lg = micro_weights(cfg, seed=7)
    G = cfg.n_q_heads // cfg.n_kv_heads
    hd = cfg.head_dim
    cm = cfg.replace(n_kv_heads=cfg.n_q_heads)
    wm = dict(w)
    for k in ("wk_d", "wv_d", "wk_t", "wv_t"):
        a = w[k].reshape(cfg.n_draft_layers, cfg.n_kv_heads, hd, cfg.hidden)
        wm[k] = np.repeat(a, G, axis=1).reshape(cfg.n_draft_layers, cfg.n_q_heads * hd, cfg.hidden)
    ids = np.array([1, 2, 63, 63])
    a = build(cfg, w, lg, L=6).draft_block(ids)
    b = build(cm, wm, lg, L=6).draft_block(ids)
    assert rel(a["logits"], b["logits"]) < 1e-12
    assert np.array_equal(a["tokens"], b["tokens"])


def check_position_shift_invariance():
    cfg = MICRO
    w, lg = micro_weights(cfg, seed=8)
    hid = synth.hidden_rows(cfg, 0, 6)
    ids = np.array([7, 63, 63, 63])
    outs = []
    for shift in (0, 1000):
        o = orc.DraftOracle(cfg, w, lg)
        o.append(hid, positions=np.arange(6) + shift)
        outs.append(o.draft_block(ids, positions=np.arange(6, 10) + shift))
    assert rel(outs[1]["hidden"], outs[0]["hidden"]) < 1e-10
    assert rel(outs[1]["logits"], outs[0]["logits"]) < 1e-10


def check_zero_branches():
    """W_O = 0 and W_down = 0: the block rows stay the embeddings, logits reduce to
    RMSNorm(E[ids]) W_lm^T, evaluated here with explicit loops."""
    cfg = MICRO
    w, lg = micro_weights(cfg, seed=9)
    w = dict(w)
    w["wo"] = np.zeros_like(w["wo"])
    w["w_down"] = np.zeros_like(w["w_down"])
    ids = np.array([0, 31, 63, 31])
    r = build(cfg, w, lg, L=4).draft_block(ids)
    E, gf, wl = f64(w["embed"]), f64(w["final_norm"]), f64(w["lm_head"])
    for i in range(cfg.n_draft_layers):
        assert np.array_equal(r["hidden"][i], E[ids])
    for b, t in enumerate(ids):
        rr = math.sqrt(sum(E[t, k] ** 2 for k in range(cfg.hidden)) / cfg.hidden + cfg.rms_eps)
        for v in range(cfg.vocab):
            z = sum(E[t, k] / rr * gf[k] * wl[v, k] for k in range(cfg.hidden))
            assert abs(r["logits"][b, v] - z) < 1e-12 * max(1.0, abs(z))
    assert r["tokens"][1] == r["tokens"][3]


def check_mlp_closed_form():
    """Attention branch off, MLP wired so that only feature 0 is live:
    gate_0 = c m_0, up_0 = m_0, and W_down sends it to column 1 with weight w.
    Then X_1 = X_0 + w * silu(c m_0) * m_0 at column 1 and X_0 elsewhere."""
    cfg = MICRO.replace(n_draft_layers=1)
    w, _ = micro_weights(cfg, seed=10)
    w = dict(w)
    D, H, F = 1, cfg.hidden, cfg.ffn
    c, wd = 1.5, -0.75
    w["wo"] = np.zeros_like(w["wo"])
    g = np.zeros((D, F, H), np.float32); g[0, 0, 0] = c
    u = np.zeros((D, F, H), np.float32); u[0, 0, 0] = 1.0
    dn = np.zeros((D, H, F), np.float32); dn[0, 1, 0] = wd
    w["w_gate"], w["w_up"], w["w_down"] = bf16(g), bf16(u), bf16(dn)
    ids = np.array([4, 8, 15, 16])
    r = orc.DraftOracle(cfg, w, np.zeros((1, cfg.n_target_layers))).draft_block(ids)
    E, gm = f64(w["embed"]), f64(w["mlp_norm"][0])
    for b, t in enumerate(ids):
        x = E[t]
        m0 = x[0] / math.sqrt(float(np.sum(x * x)) / H + cfg.rms_eps) * gm[0]
        z = c * m0
        expect = x.copy()
        expect[1] += wd * (z / (1.0 + math.exp(-z))) * m0
        assert np.allclose(r["hidden"][0, b], expect, rtol=1e-14, atol=1e-15)


def check_argmax_ties():
    z = np.array([[0.0, 3.0, 1.0, 3.0], [2.0, 2.0, 2.0, 2.0], [-1.0, -5.0, -1.0, -2.0]])
    assert list(orc.argmax_lowest(z)) == [1, 0, 0]
    # duplicated LM-head rows: the lower id wins
    cfg = MICRO
    w, lg = micro_weights(cfg, seed=12)
    o = build(cfg, w, lg, L=3)
    ids = np.array([1, 2, 3, 4])
    t = o.draft_block(ids)["tokens"]
    w2 = dict(w)
    lm = w["lm_head"].copy()
    lo = int(t[0]) // 2
    lm[lo] = lm[t[0]]
    w2["lm_head"] = lm
    t2 = build(cfg, w2, lg, L=3).draft_block(ids)["tokens"]
    assert t2[0] == min(lo, int(t[0]))


def check_empty_context():
    cfg = MICRO
    w, lg = micro_weights(cfg, seed=13)
    o = orc.DraftOracle(cfg, w, lg)
    r = o.draft_block(np.array([1, 2, 3, 4]))
    assert r["tokens"].shape == (4,)
    assert np.isfinite(r["logits"]).all()


def test_block_pass_bruteforce():
    check_block_pass_bruteforce()


def test_joint_permutation_of_block():
    check_joint_permutation()


def test_gqa_equals_duplicated_mha():
    check_gqa_equals_duplicated_mha()


def test_position_shift_invariance():
    check_position_shift_invariance()


def test_zero_branches_reduce_to_lm_head():
    check_zero_branches()


def test_mlp_closed_form():
    check_mlp_closed_form()


def test_argmax_ties_lowest_index():
    check_argmax_ties()


def test_empty_context_block():
    check_empty_context()


def test_truncate_and_context_full():
    cfg = MICRO
    w, lg = micro_weights(cfg)
    o = orc.DraftOracle(cfg, w, lg, max_context=8)
    o.append(synth.hidden_rows(cfg, 0, 6))
    with pytest.raises(ValueError):
        o.append(synth.hidden_rows(cfg, 6, 3))
    assert o.L == 6
    k2 = o.k_cache[1][:4].copy()
    o.truncate(4)
    assert o.L == 4 and np.array_equal(o.k_cache[1], k2)
    with pytest.raises(ValueError):
        o.truncate(5)


# ---- temperature sampling: Philox4x64-10 uniforms and Gumbel-max draws ----

def check_philox_matches_numpy():
    # numpy's Philox bit generator is the same Philox4x64-10; it advances its 256-bit counter
    # before each block, so its block after counter c - 1 is the function's block at c
    cases = [((1, 0, 0, 0), (0, 0)), ((0x243F6A8885A308D3, 0x13198A2E03707344, 7, 0xFFFFFFFFFFFFFFFF),
                                     (0xA4093822299F31D0, 0x082EFA98EC4E6C89)),
             ((123456789, 42, 3, 1), (2026, 0))]
    for ctr, key in cases:
        bg = np.random.Philox(key=np.array(key, dtype=np.uint64),
                              counter=np.array((ctr[0] - 1,) + ctr[1:], dtype=np.uint64))
        ref = [int(x) for x in bg.random_raw(4)]
        got = [int(x) for x in orc.philox4x64_10(tuple(np.uint64(c) for c in ctr), key)]
        assert got == ref, (ctr, key, [hex(x) for x in got], [hex(x) for x in ref])


def check_sampling_uniforms():
    u = orc.sampling_uniforms(seed=5, draw=0, slot=0, n_pos=64, vocab=2048)
    assert u.shape == (64, 2048) and u.min() > 0.0 and u.max() < 1.0
    assert abs(u.mean() - 0.5) < 5e-3 and abs(u.var() - 1.0 / 12.0) < 2e-3
    # single precision holds every uniform exactly, the extremes included: the largest is
    # 1 - 2^-24, below 1 in fp32 as well, so fp32 noise -log(-log U) stays finite
    assert np.array_equal(u.astype(np.float32).astype(np.float64), u)
    for k in (0, (1 << 23) - 1):
        top = (float(k) + 0.5) / float(1 << 23)
        assert np.float32(top) == top and np.float32(top) < np.float32(1.0)
        assert np.isfinite(np.float32(-np.log(-np.log(np.float32(top)))))
    # the four positions served by one generator call take different output words
    for b in range(1, 4):
        assert np.mean(u[0] == u[b]) < 1e-3 and np.mean(u[4 + b] == u[4]) < 1e-3
    # one generator call per four positions: positions 4 q + j, word j of counter (v, q, ...)
    c = orc.philox4x64_10((np.arange(2048, dtype=np.uint64), np.uint64(3), np.uint64(0), np.uint64(0)),
                          (np.uint64(5), np.uint64(0)))
    for j in range(4):
        assert np.array_equal(u[12 + j], ((c[j] >> np.uint64(41)).astype(np.float64) + 0.5) / 2.0 ** 23)
    # every counter word matters: another draw, slot or seed gives other numbers
    for kw in ({"draw": 1}, {"slot": 1}, {"seed": 6}):
        args = {"seed": 5, "draw": 0, "slot": 0}
        args.update(kw)
        v = orc.sampling_uniforms(n_pos=64, vocab=2048, **args)
        assert np.mean(v == u) < 1e-3


def _chi2(counts, probs):
    n = counts.sum()
    return float(np.sum((counts - n * probs) ** 2 / (n * probs)))


def check_gumbel_max_draws_follow_softmax():
    # 20000 independent draws (one per block position) from a 6-token distribution; chi-square
    # against softmax(z / T) with 5 degrees of freedom: 25.7 is its 1e-4 upper quantile
    z = np.array([0.3, -1.0, 1.2, 0.0, 2.0, -0.5])
    n = 20000
    for temperature in (1.0, 2.0, 0.5):
        tok, _ = orc.sample_tokens(np.tile(z, (n, 1)), temperature, seed=11, draw=3, slot=2)
        counts = np.bincount(tok, minlength=z.size).astype(np.float64)
        p = np.exp(z / temperature - (z / temperature).max())
        p /= p.sum()
        assert _chi2(counts, p) < 25.7, (temperature, counts, n * p)


def check_sampling_limits_and_replay():
    rng = np.random.default_rng(9)
    z = rng.standard_normal((8, 300))
    assert np.array_equal(orc.sample_tokens(z, 0.0, 1, 0)[0], orc.argmax_lowest(z))
    # vanishing temperature: the noise is negligible against z / T
    assert np.array_equal(orc.sample_tokens(z, 1e-9, 1, 0)[0], orc.argmax_lowest(z))
    a = orc.sample_tokens(z, 1.0, seed=3, draw=4, slot=1)[0]
    assert np.array_equal(a, orc.sample_tokens(z, 1.0, seed=3, draw=4, slot=1)[0])
    # a flat distribution: other draws give other tokens at almost every position
    flat = np.zeros((64, 1000))
    t0 = orc.sample_tokens(flat, 1.0, seed=3, draw=0)[0]
    t1 = orc.sample_tokens(flat, 1.0, seed=3, draw=1)[0]
    assert np.mean(t0 == t1) < 0.05


def test_philox_matches_numpy():
    check_philox_matches_numpy()


def test_sampling_uniforms():
    check_sampling_uniforms()


def test_gumbel_max_draws_follow_softmax():
    check_gumbel_max_draws_follow_softmax()


def test_sampling_limits_and_replay():
    check_sampling_limits_and_replay()


# --------------------------------------------------------------------------------------
# model variants: the ablations of Sec. 6.3 (Table 2) and the DFlash baseline (Eq. 1-2)
# --------------------------------------------------------------------------------------

VAR = orc.VARIANT_NO_SOFTMAX, orc.VARIANT_SHARED_KV, orc.VARIANT_POST_FC, orc.VARIANT_DFLASH


def variant_weights(cfg=MICRO, seed=0):
    w = synth.make_weights(cfg, seed=seed, threads=1, kinds=synth.WEIGHT_KINDS)
    logits = w.pop("fusion_logits")
    return w, logits


def loops_kv(f_rows, wk, wv, positions, cfg):
    """K (rotated) and V of fused rows by explicit loops, as in check_context_kv_bruteforce."""
    H, nkv, hd = cfg.hidden, cfg.n_kv_heads, cfg.head_dim
    K, V = [], []
    for r, p in zip(range(len(f_rows)), positions):
        kr_all, vr_all = [], []
        for g in range(nkv):
            kr = [sum(f_rows[r][k] * wk[g * hd + d, k] for k in range(H)) for d in range(hd)]
            vr = [sum(f_rows[r][k] * wv[g * hd + d, k] for k in range(H)) for d in range(hd)]
            rot = []
            for d in range(hd):
                m = d % (hd // 2)
                th = p / (cfg.rope_base ** (2.0 * m / hd))
                if d < hd // 2:
                    rot.append(kr[d] * math.cos(th) - kr[d + hd // 2] * math.sin(th))
                else:
                    rot.append(kr[d] * math.cos(th) + kr[d - hd // 2] * math.sin(th))
            kr_all.append(rot)
            vr_all.append(vr)
        K.append(kr_all)
        V.append(vr_all)
    return np.array(K), np.array(V)


def check_no_softmax_scale_invariance():
    """-Softmax: alpha is W^fuse as given.  RMSNorm ignores a common positive scale of the
    fused sum (up to eps), so raw weights c * softmax(x) reproduce the model with logits x;
    a softmax left in place would turn c * softmax(x) into other weights."""
    cfg = MICRO
    w, lg = micro_weights(cfg)
    hid = synth.hidden_rows(cfg, 0, 5)
    ref = orc.DraftOracle(cfg, w, lg)
    ref.append(hid)
    a = orc.fusion_weights(lg)
    for c in (0.37, 5.0):
        raw = c * a
        assert np.array_equal(orc.fusion_weights(raw, normalize=False), raw)
        o = orc.DraftOracle(cfg, w, raw, variant=orc.VARIANT_NO_SOFTMAX)
        o.append(hid)
        # the eps term: RMSNorm(c u) / RMSNorm(u) = sqrt((m + eps) / (m + eps / c^2)), within
        # eps (1 / c^2 - 1) / (2 m) ~ 2e-5 of 1 for rows with mean square m ~ 0.4
        for i in range(cfg.n_draft_layers):
            assert rel(o.k_cache[i], ref.k_cache[i]) < 1e-4 and rel(o.v_cache[i], ref.v_cache[i]) < 1e-4
    # a raw weight vector that is not a scaled softmax gives another model
    skew = a.copy()
    skew[:, 0] *= 3.0
    o = orc.DraftOracle(cfg, w, skew, variant=orc.VARIANT_NO_SOFTMAX)
    o.append(hid)
    assert rel(o.k_cache[0], ref.k_cache[0]) > 1e-3
    for bad in (np.nan, np.inf, -np.inf):
        x = a.copy()
        x[0, 1] = bad
        with pytest.raises(ValueError):
            orc.fusion_weights(x, normalize=False)


def check_shared_kv_bruteforce():
    """-KVProj: the context K/V of layer i come from its own W_K^d, W_V^d (loops)."""
    cfg = MICRO
    w, lg = micro_weights(cfg)
    hid = synth.hidden_rows(cfg, 0, 2)
    o = orc.DraftOracle(cfg, w, lg, variant=orc.VARIANT_SHARED_KV)
    f = o.append(hid)
    for i in range(cfg.n_draft_layers):
        K, V = loops_kv(f[i], f64(w["wk_d"][i]), f64(w["wv_d"][i]), [0, 1], cfg)
        assert np.allclose(o.k_cache[i], K, rtol=1e-12, atol=1e-13)
        assert np.allclose(o.v_cache[i], V, rtol=1e-12, atol=1e-13)


def check_post_fc():
    """+FC: f' = f W^T + b on the fused rows.  Identity layer without bias: the plain model,
    bit for bit.  Zero weights: every row becomes b, so V = W_V^t b for all rows.  A random
    layer against loops."""
    cfg = MICRO
    H, D = cfg.hidden, cfg.n_draft_layers
    w, lg = variant_weights(cfg)
    hid = synth.hidden_rows(cfg, 0, 3)
    plain = orc.DraftOracle(cfg, w, lg)
    plain.append(hid)
    eye = dict(w, post_fc=np.broadcast_to(bf16(np.eye(H)), (D, H, H)).copy(), post_fc_bias=None)
    o = orc.DraftOracle(cfg, eye, lg, variant=orc.VARIANT_POST_FC)
    o.append(hid)
    for i in range(D):
        assert np.array_equal(o.k_cache[i], plain.k_cache[i]) and np.array_equal(o.v_cache[i], plain.v_cache[i])
    zero = dict(w, post_fc=np.zeros((D, H, H), np.uint16))
    o = orc.DraftOracle(cfg, zero, lg, variant=orc.VARIANT_POST_FC)
    o.append(hid)
    for i in range(D):
        b = f64(w["post_fc_bias"][i])
        wv = f64(w["wv_t"][i])
        vb = [[sum(wv[g * cfg.head_dim + d, k] * b[k] for k in range(H)) for d in range(cfg.head_dim)]
              for g in range(cfg.n_kv_heads)]
        for r in range(3):
            assert np.allclose(o.v_cache[i][r], vb, rtol=1e-12, atol=1e-13)
    o = orc.DraftOracle(cfg, w, lg, variant=orc.VARIANT_POST_FC)
    fp = o.append(hid)
    f = orc.fuse_rows(orc.fusion_weights(lg), f64(hid), f64(w["fuse_norm"]), cfg.rms_eps)
    for i in range(D):
        W, b = f64(w["post_fc"][i]), f64(w["post_fc_bias"][i])
        for r in range(3):
            want = [sum(W[oo, k] * f[i, r, k] for k in range(H)) + b[oo] for oo in range(H)]
            assert np.allclose(fp[i, r], want, rtol=1e-12, atol=1e-13)
        K, V = loops_kv(fp[i], f64(w["wk_t"][i]), f64(w["wv_t"][i]), [0, 1, 2], cfg)
        assert np.allclose(o.k_cache[i], K, rtol=1e-12, atol=1e-13)
        assert np.allclose(o.v_cache[i], V, rtol=1e-12, atol=1e-13)


def check_dflash_context():
    """DFlash (Eq. 1-2): c_t = W_fc [h^(1); ...; h^(S)] + b_fc by loops, the same context for
    every layer, projected by each layer's W_K^d, W_V^d; a W_fc that selects target layer j
    (identity in block j, no bias) makes C the rows of layer j."""
    cfg = MICRO
    H, S, D = cfg.hidden, cfg.n_target_layers, cfg.n_draft_layers
    w, _ = variant_weights(cfg)
    hid = synth.hidden_rows(cfg, 0, 2)
    h = f64(hid)
    o = orc.DraftOracle(cfg, w, None, variant=orc.VARIANT_DFLASH)
    c = o.append(hid)
    W, b = f64(w["fc"]), f64(w["fc_bias"])
    for t in range(2):
        want = [sum(W[oo, j * H + k] * h[j, t, k] for j in range(S) for k in range(H)) + b[oo] for oo in range(H)]
        assert np.allclose(c[0, t], want, rtol=1e-12, atol=1e-13)
    for i in range(D):
        assert np.array_equal(c[i], c[0])
        K, V = loops_kv(c[i], f64(w["wk_d"][i]), f64(w["wv_d"][i]), [0, 1], cfg)
        assert np.allclose(o.k_cache[i], K, rtol=1e-12, atol=1e-13)
        assert np.allclose(o.v_cache[i], V, rtol=1e-12, atol=1e-13)
    sel = np.zeros((H, S * H), np.float32)
    sel[:, H:2 * H] = np.eye(H)
    o = orc.DraftOracle(cfg, dict(w, fc=bf16(sel), fc_bias=None), None, variant=orc.VARIANT_DFLASH)
    assert np.array_equal(o.append(hid)[0], h[1])
    with pytest.raises(ValueError):
        orc.DraftOracle(cfg, w, None, variant=orc.VARIANT_DFLASH | orc.VARIANT_POST_FC)


def test_no_softmax_scale_invariance():
    check_no_softmax_scale_invariance()


def test_shared_kv_bruteforce():
    check_shared_kv_bruteforce()


def test_post_fc():
    check_post_fc()


def test_dflash_context():
    check_dflash_context()


# --------------------------------------------------------------------------------------
# verification (Sec. 3.2, verification phase)
# --------------------------------------------------------------------------------------

def check_accept_block_exhaustive():
    """Every (candidates, target predictions) over a 3-token alphabet with B = 4: k is the
    number of leading positions where candidate j equals the target's prediction after
    position j - 1; the emitted tokens are exactly the target's own predictions 0..k (the
    loop emits what the target alone would have emitted greedily); the bonus is the last."""
    import itertools
    B = 4
    for d_tail in itertools.product(range(3), repeat=B - 1):
        d = (7,) + d_tail
        for t in itertools.product(range(3), repeat=B):
            k, bonus, emitted = orc.accept_block(d, t)
            lead = 0
            for j in range(1, B):
                if d[j] != t[j - 1]:
                    break
                lead += 1
            assert k == lead
            assert emitted == list(t[:k + 1]) and bonus == t[k]
    assert orc.accept_block([3], [5]) == (0, 5, [5])


def check_accept_appends_verified_rows():
    """accept appends the target rows of positions 0..k only: L grows by k + 1 and the
    cache equals that of appending those rows directly."""
    cfg = MICRO
    w, lg = micro_weights(cfg)
    B = cfg.block_size
    hid = synth.hidden_rows(cfg, 0, 4)
    blk = synth.hidden_rows(cfg, 4, B, seed=3)
    for k_want in range(B):
        d = [9] + list(range(1, B))
        t = list(range(1, B)) + [0]
        if k_want < B - 1:
            t[k_want] = 63  # first disagreement after k_want accepted candidates
        a = build(cfg, w, lg, 0)
        a.append(hid)
        k, bonus, _ = a.accept(d, t, blk)
        assert k == k_want and a.L == 4 + k + 1 and bonus == t[k]
        b = build(cfg, w, lg, 0)
        b.append(hid)
        b.append(blk[:, :k + 1])
        for i in range(cfg.n_draft_layers):
            assert np.array_equal(a.k_cache[i], b.k_cache[i])


def test_accept_block_exhaustive():
    check_accept_block_exhaustive()


def test_accept_appends_verified_rows():
    check_accept_appends_verified_rows()


ALL_CHECKS = [v for k, v in sorted(globals().items()) if k.startswith("check_")]
