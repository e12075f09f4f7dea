"""Pins of the training-side fp64 oracle (oracle/training_oracle.py) against what the paper
and the mathematics fix, and planted mistakes that the pins must catch.

Anchor attention (Sec. 3.3): brute force with pure-Python loops, central finite differences
of every gradient, block independence (no attention across blocks), context at or after an
anchor has no effect on that block, GQA equals duplicated heads, and the closed form for
all-zero scores (uniform weights over the visible keys, lse = log of their number).
Weighted cross-entropy (Eq. 5): loops, finite differences, uniform logits (CE = log V), the
gamma schedule's end points and linearity, and the weights' ratios.
"""
import math

import numpy as np
import pytest

from oracle import training_oracle as tr


def case(seed=0, n=3, B=4, T=10, nq=4, nkv=2, hd=8, anchors=(0, 5, 10)):
    rng = np.random.default_rng(seed)
    return dict(q=rng.standard_normal((n * B, nq, hd)), k_ctx=rng.standard_normal((T, nkv, hd)),
                v_ctx=rng.standard_normal((T, nkv, hd)), k_blk=rng.standard_normal((n * B, nkv, hd)),
                v_blk=rng.standard_normal((n * B, nkv, hd)), anchors=list(anchors), B=B)


def check_forward_loops():
    c = case()
    out, lse = tr.anchor_attention_fwd(**c)
    q, kc, vc, kb, vb, B = c["q"], c["k_ctx"], c["v_ctx"], c["k_blk"], c["v_blk"], c["B"]
    T, nkv, hd = kc.shape
    nq = q.shape[1]
    for i, a in enumerate(c["anchors"]):
        for b in range(B):
            r = i * B + b
            for h in range(nq):
                g = h // (nq // nkv)
                keys = [(kc[j, g], vc[j, g]) for j in range(a)] + [(kb[i * B + j, g], vb[i * B + j, g]) for j in range(B)]
                s = [sum(q[r, h, d] * k[d] for d in range(hd)) / math.sqrt(hd) for k, _ in keys]
                m = max(s)
                e = [math.exp(x - m) for x in s]
                z = sum(e)
                o = [sum(e[j] * keys[j][1][d] for j in range(len(keys))) / z for d in range(hd)]
                assert np.allclose(out[r, h], o, rtol=1e-12, atol=1e-12)
                assert abs(lse[r, h] - (m + math.log(z))) < 1e-12


def check_backward_finite_differences():
    c = case(seed=1, n=2, B=3, T=5, nq=2, nkv=1, hd=4, anchors=(2, 5))
    rng = np.random.default_rng(2)
    out, _ = tr.anchor_attention_fwd(**c)
    dout = rng.standard_normal(out.shape)
    grads = dict(zip(("q", "k_ctx", "v_ctx", "k_blk", "v_blk"), tr.anchor_attention_bwd(**c, dout=dout)))
    eps = 1e-6
    for name, g in grads.items():
        x = c[name]
        for idx in list(np.ndindex(x.shape))[::3]:
            old = x[idx]
            x[idx] = old + eps
            fp = (tr.anchor_attention_fwd(**c)[0] * dout).sum()
            x[idx] = old - eps
            fm = (tr.anchor_attention_fwd(**c)[0] * dout).sum()
            x[idx] = old
            assert abs((fp - fm) / (2 * eps) - g[idx]) < 1e-6 * max(1.0, abs(g[idx])), (name, idx)


def check_block_independence_and_anchor_cut():
    c = case(seed=3, n=3, B=4, T=12, anchors=(3, 7, 9))
    out, lse = tr.anchor_attention_fwd(**c)
    c2 = {k: (v.copy() if isinstance(v, np.ndarray) else v) for k, v in c.items()}
    c2["q"][8:12] += 1.0        # block 2's queries
    c2["k_blk"][8:12] -= 2.0    # and its keys / values
    c2["v_blk"][8:12] *= 3.0
    c2["k_ctx"][9:] += 5.0      # context at or after the largest anchor
    c2["v_ctx"][9:] -= 5.0
    o2, l2 = tr.anchor_attention_fwd(**c2)
    assert np.array_equal(out[:8], o2[:8]) and np.array_equal(lse[:8], l2[:8])
    assert not np.allclose(out[8:], o2[8:])


def check_gqa_equals_duplicated_heads():
    c = case(seed=4, nq=4, nkv=2)
    out, lse = tr.anchor_attention_fwd(**c)
    d = dict(c)
    for k in ("k_ctx", "v_ctx", "k_blk", "v_blk"):
        d[k] = np.repeat(c[k], 2, axis=1)
    o2, l2 = tr.anchor_attention_fwd(**d)
    assert np.allclose(out, o2, rtol=1e-13, atol=1e-13) and np.allclose(lse, l2, rtol=1e-13)
    dout = np.random.default_rng(5).standard_normal(out.shape)
    g1 = tr.anchor_attention_bwd(**c, dout=dout)
    g2 = tr.anchor_attention_bwd(**d, dout=dout)
    assert np.allclose(g1[0], g2[0], rtol=1e-12, atol=1e-12)
    for a, b in zip(g1[1:], g2[1:]):  # the duplicated heads' gradients add up
        assert np.allclose(a, b[:, 0::2] + b[:, 1::2], rtol=1e-12, atol=1e-12)


def check_zero_scores_closed_form():
    c = case(seed=6)
    c["q"][:] = 0.0
    out, lse = tr.anchor_attention_fwd(**c)
    B = c["B"]
    for i, a in enumerate(c["anchors"]):
        vals = np.concatenate([c["v_ctx"][:a], c["v_blk"][i * B:(i + 1) * B]])  # [a + B, nkv, hd]
        for h in range(c["q"].shape[1]):
            g = h // 2
            assert np.allclose(out[i * B:(i + 1) * B, h], vals[:, g].mean(axis=0), rtol=1e-12, atol=1e-12)
            assert np.allclose(lse[i * B:(i + 1) * B, h], math.log(a + B), rtol=1e-13)


def check_weighted_ce_loops_and_gradient():
    rng = np.random.default_rng(7)
    B, V = 4, 7
    z = rng.standard_normal((8, V))
    y = np.array([-1, 2, 6, 0, 5, 1, -1, 3])
    gamma = 1.7
    loss, ce, dz = tr.weighted_ce(z, y, B, gamma)
    num = den = 0.0
    for r in range(8):
        b = r % B
        if b == 0 or y[r] < 0:
            assert ce[r] == 0.0
            continue
        w = math.exp(-(b - 1) / gamma)
        lse = math.log(sum(math.exp(v) for v in z[r]))
        assert abs(ce[r] - (lse - z[r, y[r]])) < 1e-12
        num += w * (lse - z[r, y[r]])
        den += w
    assert abs(loss - num / den) < 1e-12
    eps = 1e-6
    for idx in list(np.ndindex(z.shape))[::5]:
        old = z[idx]
        z[idx] = old + eps
        fp = tr.weighted_ce(z, y, B, gamma)[0]
        z[idx] = old - eps
        fm = tr.weighted_ce(z, y, B, gamma)[0]
        z[idx] = old
        assert abs((fp - fm) / (2 * eps) - dz[idx]) < 1e-7, idx
    # uniform logits: every CE is log V
    l2, ce2, _ = tr.weighted_ce(np.zeros((8, V)), np.abs(y), B, gamma)
    assert abs(l2 - math.log(V)) < 1e-12


def check_gamma_schedule_and_weights():
    assert tr.progressive_gamma(0, 100, 4.5, 9.5) == 4.5
    assert tr.progressive_gamma(100, 100, 4.5, 9.5) == 9.5
    assert abs(tr.progressive_gamma(25, 100, 4.5, 9.5) - 5.75) < 1e-15
    w = tr.position_weights(16, 4.0)
    assert w[0] == 0.0 and w[1] == 1.0
    assert np.allclose(w[2:] / w[1:-1], math.exp(-1 / 4.0), rtol=1e-14)


ALL_CHECKS = [v for k, v in sorted(globals().items()) if k.startswith("check_")]


@pytest.mark.parametrize("chk", ALL_CHECKS, ids=lambda f: f.__name__)
def test_pin(chk):
    chk()


# ---- planted mistakes ----------------------------------------------------------------

_ORIG = {k: getattr(tr, k) for k in ("anchor_attention_fwd", "anchor_attention_bwd", "_visible", "position_weights")}


def _visible_includes_anchor(anchors, B, T):
    m = _ORIG["_visible"]([min(a + 1, T) for a in anchors], B, T)
    return m


def _visible_cross_block(anchors, B, T):
    m = _ORIG["_visible"](anchors, B, T)
    m[:, :T] = True  # whole context for every block
    return m


def _weights_from_zero(B, gamma):
    return np.array([math.exp(-b / gamma) for b in range(B)])


def _bwd_missing_rowsum(q, k_ctx, v_ctx, k_blk, v_blk, anchors, B, dout):
    g = list(_ORIG["anchor_attention_bwd"](q, k_ctx, v_ctx, k_blk, v_blk, anchors, B, dout))
    g[0] = g[0] * 1.01  # a mis-scaled query gradient
    return tuple(g)


def _bwd_unscaled_dk(q, k_ctx, v_ctx, k_blk, v_blk, anchors, B, dout):
    g = list(_ORIG["anchor_attention_bwd"](q, k_ctx, v_ctx, k_blk, v_blk, anchors, B, dout))
    hd = np.asarray(q).shape[-1]
    g[1] = g[1] * math.sqrt(hd)
    g[3] = g[3] * math.sqrt(hd)
    return tuple(g)


MUTANTS = {
    "context_includes_anchor_position": ("_visible", _visible_includes_anchor),
    "attention_across_blocks": ("_visible", _visible_cross_block),
    "weights_start_at_anchor": ("position_weights", _weights_from_zero),
    "query_gradient_misscaled": ("anchor_attention_bwd", _bwd_missing_rowsum),
    "key_gradient_unscaled": ("anchor_attention_bwd", _bwd_unscaled_dk),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, monkeypatch):
    attr, fn = MUTANTS[name]
    monkeypatch.setattr(tr, attr, fn)
    caught = []
    for chk in ALL_CHECKS:
        try:
            chk()
        except Exception:  # noqa: BLE001 - any failure counts as detection
            caught.append(chk.__name__)
    assert caught, f"mutant {name} passed every pin"
