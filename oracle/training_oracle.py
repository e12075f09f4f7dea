"""Plain fp64 CPU oracle of the training-side operations of DFlare (arXiv 2606.02091).

TEST INFRASTRUCTURE ONLY.  Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline
leg may import this module.  The HIP library and its Python binding never import, call or
link it, and it imports nothing from them.

* anchor attention (Sec. 3.3, training of the block diffusion draft model): the sampled
  blocks of one sequence are processed together; a row of block i (anchored at sequence
  position a_i, its B positions a_i .. a_i + B - 1) attends to the target context features
  of the positions before its anchor (context keys 0 .. a_i - 1) and bidirectionally to
  the B positions of its own block, never to another block.  Scale 1/sqrt(hd); query head
  h reads KV head floor(h / (n_q / n_kv)).  Forward: outputs and log-sum-exp per row and
  head; backward: gradients of q, context k/v and block k/v for a given output gradient.
* progressive position-weighted cross-entropy (Sec. 4.3, Eq. 5): gamma(s) =
  gamma_0 + (s / S)(gamma_max - gamma_0), w_k = exp(-(k - 1) / gamma) for the k-th masked
  position of a block (block position b = k, b >= 1); the anchor position is not predicted.

Readings (the paper does not fix them): "the corresponding target context features" of a
block are those of the positions before its anchor (the same context the block sees at
inference, Sec. 3.2); the loss is the weighted mean sum_k w_k CE_k / sum_k w_k over the
predicted positions of all blocks; a label < 0 marks a position without a target.

Pins: tests/test_training_pins.py (brute-force loops, finite differences, invariants,
closed forms).
"""
from __future__ import annotations

import math

import numpy as np

__all__ = ["anchor_attention_fwd", "anchor_attention_bwd", "progressive_gamma", "position_weights",
           "weighted_ce"]


def _visible(anchors, B, T):
    """mask [n_blocks, T + B]: context keys before the anchor, then the block's own keys."""
    n = len(anchors)
    m = np.zeros((n, T + B), dtype=bool)
    for i, a in enumerate(anchors):
        m[i, :a] = True
        m[i, T:] = True
    return m


def anchor_attention_fwd(q, k_ctx, v_ctx, k_blk, v_blk, anchors, B):
    """q [n*B, n_q, hd]; k_ctx, v_ctx [T, n_kv, hd]; k_blk, v_blk [n*B, n_kv, hd];
    anchors [n] in [0, T].  Returns out [n*B, n_q, hd] and lse [n*B, n_q] (natural log)."""
    q, k_ctx, v_ctx, k_blk, v_blk = (np.asarray(x, np.float64) for x in (q, k_ctx, v_ctx, k_blk, v_blk))
    M, nq, hd = q.shape
    T, nkv, _ = k_ctx.shape
    n = M // B
    G = nq // nkv
    scale = 1.0 / math.sqrt(hd)
    vis = _visible(anchors, B, T)
    out = np.zeros((M, nq, hd))
    lse = np.zeros((M, nq))
    for i in range(n):
        rows = slice(i * B, (i + 1) * B)
        for h in range(nq):
            g = h // G
            keys = np.concatenate([k_ctx[:, g], k_blk[rows, g]])      # [T + B, hd]
            vals = np.concatenate([v_ctx[:, g], v_blk[rows, g]])
            s = q[rows, h] @ keys.T * scale                           # [B, T + B]
            s[:, ~vis[i]] = -np.inf
            mx = s.max(axis=1, keepdims=True)
            p = np.exp(s - mx)
            z = p.sum(axis=1, keepdims=True)
            out[rows, h] = (p / z) @ vals
            lse[rows, h] = (mx + np.log(z))[:, 0]
    return out, lse


def anchor_attention_bwd(q, k_ctx, v_ctx, k_blk, v_blk, anchors, B, dout):
    """Gradients for a given dout [n*B, n_q, hd]: (dq, dk_ctx, dv_ctx, dk_blk, dv_blk), from
    the probabilities P = softmax(S) of the forward pass: dV = P^T dO, dP = dO V^T,
    dS = P (dP - rowsum(dP P)), dQ = scale dS K, dK = scale dS^T Q."""
    q, k_ctx, v_ctx, k_blk, v_blk, dout = (np.asarray(x, np.float64)
                                           for x in (q, k_ctx, v_ctx, k_blk, v_blk, dout))
    M, nq, hd = q.shape
    T, nkv, _ = k_ctx.shape
    n = M // B
    G = nq // nkv
    scale = 1.0 / math.sqrt(hd)
    vis = _visible(anchors, B, T)
    dq = np.zeros_like(q)
    dkc, dvc = np.zeros_like(k_ctx), np.zeros_like(v_ctx)
    dkb, dvb = np.zeros_like(k_blk), np.zeros_like(v_blk)
    for i in range(n):
        rows = slice(i * B, (i + 1) * B)
        for h in range(nq):
            g = h // G
            keys = np.concatenate([k_ctx[:, g], k_blk[rows, g]])
            vals = np.concatenate([v_ctx[:, g], v_blk[rows, g]])
            s = q[rows, h] @ keys.T * scale
            s[:, ~vis[i]] = -np.inf
            p = np.exp(s - s.max(axis=1, keepdims=True))
            p /= p.sum(axis=1, keepdims=True)
            do = dout[rows, h]
            dv = p.T @ do                                             # [T + B, hd]
            dp = do @ vals.T                                          # [B, T + B]
            ds = p * (dp - (dp * p).sum(axis=1, keepdims=True))
            dq[rows, h] = scale * ds @ keys
            dk = scale * ds.T @ q[rows, h]
            dkc[:, g] += dk[:T]
            dvc[:, g] += dv[:T]
            dkb[rows, g] += dk[T:]
            dvb[rows, g] += dv[T:]
    return dq, dkc, dvc, dkb, dvb


def progressive_gamma(step: int, total: int, gamma0: float, gamma_max: float) -> float:
    """gamma(s) = gamma_0 + (s / S)(gamma_max - gamma_0)  (Eq. 5, first line)."""
    return gamma0 + (step / total) * (gamma_max - gamma0)


def position_weights(B: int, gamma: float) -> np.ndarray:
    """w over block positions b = 0 .. B-1: 0 for the anchor, exp(-(b - 1) / gamma) for the
    masked positions b = k >= 1  (Eq. 5, second line)."""
    w = np.zeros(B)
    for b in range(1, B):
        w[b] = math.exp(-(b - 1) / gamma)
    return w


def weighted_ce(logits, labels, B: int, gamma: float):
    """Weighted mean cross-entropy over the predicted positions of all blocks and its gradient.

    logits [n*B, V]; labels [n*B] (< 0: no target).  Returns (loss, per-row CE [n*B] (0 where
    not predicted), dlogits [n*B, V])."""
    z = np.asarray(logits, np.float64)
    y = np.asarray(labels)
    M, V = z.shape
    w = np.tile(position_weights(B, gamma), M // B)
    w[y < 0] = 0.0
    wsum = w.sum()
    mx = z.max(axis=1, keepdims=True)
    lse = (mx + np.log(np.exp(z - mx).sum(axis=1, keepdims=True)))[:, 0]
    ce = np.zeros(M)
    ok = w > 0
    ce[ok] = lse[ok] - z[ok, y[ok]]
    loss = float((w * ce).sum() / wsum) if wsum > 0 else 0.0
    p = np.exp(z - lse[:, None])
    onehot = np.zeros_like(z)
    onehot[ok, y[ok]] = 1.0
    dz = (w / wsum if wsum > 0 else w)[:, None] * (p - onehot)
    return loss, ce, dz
