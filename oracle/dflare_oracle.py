"""Plain fp64 CPU oracle of the DFlare draft step (arXiv 2606.02091).

TEST INFRASTRUCTURE ONLY.  Only tests/, __graft_entry__.smoke() and bench.py's
cpu_baseline leg may import this module.  The HIP library and its Python binding
never import, call or link it, and it imports nothing from them.

What is computed (all floating point in fp64; inputs are bfloat16 bit patterns
(uint16) up-cast exactly):

* fusion weights  alpha^(i) = softmax(W^fuse_{i,:})        -- Sec. 4.1, Eq. 3, first line;
                                                              cached once (Sec. 4.1, text after Eq. 3)
* fused rows      f_t^(i) = RMSNorm(sum_j alpha_j^(i) h_t^(j)) -- Sec. 4.1, Eq. 3, second line
* context K/V     K = F^(i) W_K^t,  V = F^(i) W_V^t           -- Sec. 4.2, Eq. 4, first block
* block K/V/Q     x W_K^d, x W_V^d, x W_Q for the B block rows -- Sec. 4.2, Eq. 4, other blocks
* attention       bidirectional inside the block and over the full context;
                  only the B block rows go on to the next layer, the context is
                  fixed across layers                           -- Sec. 3.2 (drafting phase)
* MLP sub-layer, final LM head, one token per block position    -- Sec. 3.2 (drafting phase)

Readings where the paper is silent:
  pre-norm block with residuals around attention and MLP, SwiGLU MLP, no biases,
  final RMSNorm before the LM head; RMSNorm(x; g) = x / sqrt(mean(x^2) + eps) * g;
  rotary position embedding in the rotate-half convention on Q and K (context K
  rotated at its own position when appended, V never rotated); context row r sits
  at position r and block row b at position L + b; scale 1/sqrt(head_dim); query
  head h reads KV head floor(h / (n_q / n_kv)); the block's own K/V are not kept
  in the cache; greedy argmax with ties going to the lowest token id.

Weights use the [out, in] row-major convention: y = x @ W.T (the paper writes x W
with W in R^{d x d_kv}; it is the same map).

Temperature sampling (Sec. 5, Table 1 lower half): Gumbel-max draws with uniforms from
Philox4x64-10; see sample_tokens.

Verification (Sec. 3.2, verification phase), given the target's outputs: accept_block takes
the longest prefix of candidates that the target agrees with and the bonus token;
DraftOracle.accept appends the target rows of the verified positions.

Variants (DraftOracle's `variant` bit field; 0 is the method as described):
* VARIANT_NO_SOFTMAX  -Softmax of Sec. 6.3 (Table 2): alpha = W^fuse as given
* VARIANT_SHARED_KV   -KVProj of Sec. 6.3: the context goes through the draft layer's own
                      W_K^d, W_V^d (as in Eq. 2) instead of W_K^t, W_V^t
* VARIANT_POST_FC     +FC of Sec. 6.3: f' = f W_pfc^T + b_pfc per draft layer, between the
                      fusion (Eq. 3) and the context projection (Eq. 4)
* VARIANT_DFLASH      the DFlash baseline of Sec. 3.1-3.2: c_t = W_fc [h^(1); ...; h^(S)] + b_fc
                      (Eq. 1), one context shared by every draft layer, projected by each
                      layer's W_K^d, W_V^d (Eq. 2); no fusion weights, no fusion norm

Parity pins: see tests/test_oracle_pins.py (closed forms, invariants, brute force,
library routines).  Parity unpinned: the readings above that the paper leaves
open (layer internals, rotary convention, positions) -- any consistent reading
satisfies the paper's equations, so nothing in the paper can fix them.
"""
from __future__ import annotations

import math

import numpy as np

__all__ = [
    "bf16_to_f64", "fusion_weights", "rms_norm", "rope", "silu", "fuse_rows",
    "context_kv", "block_attention", "draft_layer", "lm_head_logits", "argmax_lowest",
    "philox4x64_10", "sampling_uniforms", "sample_tokens", "post_fc", "dflash_context", "accept_block",
    "DraftOracle",
    "VARIANT_NO_SOFTMAX", "VARIANT_SHARED_KV", "VARIANT_POST_FC", "VARIANT_DFLASH",
]

VARIANT_NO_SOFTMAX, VARIANT_SHARED_KV, VARIANT_POST_FC, VARIANT_DFLASH = 1, 2, 4, 8


def bf16_to_f64(u16) -> np.ndarray:
    """bfloat16 bit patterns -> float64 (exact: bf16 is a prefix of fp32)."""
    u = np.asarray(u16, dtype=np.uint16)
    return (u.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def fusion_weights(fusion_logits, normalize: bool = True) -> np.ndarray:
    """alpha^(i) = softmax over target layers of row i of W^fuse  (Sec. 4.1, Eq. 3).

    fusion_logits: [D, S] real.  Returns [D, S] fp64 with rows summing to 1.
    The maximum of each row is subtracted first so that large logits do not
    overflow; this does not change the softmax.  Raises ValueError for a row with
    a NaN, +inf, or no finite entry.  normalize=False is the -Softmax ablation
    (Sec. 6.3): W^fuse itself, every entry finite.
    """
    lg = np.asarray(fusion_logits, dtype=np.float64)
    if lg.ndim != 2:
        raise ValueError("fusion logits must be [D, S]")
    if not normalize:
        if not np.isfinite(lg).all():
            raise ValueError("unnormalised fusion weights must be finite")
        return lg.copy()
    if np.isnan(lg).any() or np.isposinf(lg).any():
        raise ValueError("fusion logits must not contain NaN or +inf")
    if not np.isfinite(lg).any(axis=1).all():
        raise ValueError("each fusion-logit row needs a finite entry")
    m = lg.max(axis=1, keepdims=True)
    e = np.exp(lg - m)
    return e / e.sum(axis=1, keepdims=True)


def rms_norm(x: np.ndarray, gain, eps: float) -> np.ndarray:
    """RMSNorm over the last axis: x / sqrt(mean(x^2) + eps), times gain if given."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    y = x / np.sqrt(ms + eps)
    return y if gain is None else y * gain


def rope(x: np.ndarray, positions, base: float) -> np.ndarray:
    """Rotary embedding, rotate-half convention.

    x: [n, heads, hd]; positions: [n].  For m < hd/2, theta = p * base^(-2m/hd) and
    (x_m, x_{m+hd/2}) -> (x_m cos - x_{m+hd/2} sin, x_{m+hd/2} cos + x_m sin).
    """
    hd = x.shape[-1]
    half = hd // 2
    inv_freq = base ** (-(2.0 * np.arange(half, dtype=np.float64)) / hd)
    theta = np.asarray(positions, dtype=np.float64)[:, None] * inv_freq[None, :]
    c = np.cos(theta)[:, None, :]
    s = np.sin(theta)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def silu(z: np.ndarray) -> np.ndarray:
    return z / (1.0 + np.exp(-z))


def fuse_rows(alpha: np.ndarray, hidden: np.ndarray, gains, eps: float) -> np.ndarray:
    """Layer-specific fused rows f^(i)  (Sec. 4.1, Eq. 3).

    alpha: [D, S]; hidden: [S, n, H] fp64; gains: [D, H] or None.
    u^(i) = sum_j alpha[i, j] h^(j) is accumulated in j order, one row at a time,
    so a row's value does not depend on which other rows are fused with it.
    Returns [D, n, H].
    """
    D, S = alpha.shape
    out = np.empty((D,) + hidden.shape[1:], dtype=np.float64)
    for i in range(D):
        u = np.zeros(hidden.shape[1:], dtype=np.float64)
        for j in range(S):
            u += alpha[i, j] * hidden[j]
        out[i] = rms_norm(u, None if gains is None else gains[i], eps)
    return out


def context_kv(f_i: np.ndarray, wk_t: np.ndarray, wv_t: np.ndarray, positions,
               n_kv: int, hd: int, base: float):
    """Context keys/values of one draft layer  (Sec. 4.2, Eq. 4, first block).

    f_i: [n, H] fused rows; wk_t, wv_t: [n_kv*hd, H].  K is rotated at the rows'
    own positions; V is not rotated.  Returns K, V as [n, n_kv, hd].
    """
    n = f_i.shape[0]
    k = (f_i @ wk_t.T).reshape(n, n_kv, hd)
    v = (f_i @ wv_t.T).reshape(n, n_kv, hd)
    return rope(k, positions, base), v


def post_fc(f_i: np.ndarray, w: np.ndarray, b) -> np.ndarray:
    """+FC ablation (Sec. 6.3): one more fully connected layer on a draft layer's fused
    rows before they are projected into its cache, f' = f W^T + b.  f_i: [n, H];
    w: [H, H] ([out, in]); b: [H] or None."""
    out = f_i @ w.T
    return out if b is None else out + b


def dflash_context(hidden: np.ndarray, w_fc: np.ndarray, b_fc) -> np.ndarray:
    """DFlash context features (Sec. 3.1, Eq. 1): c_t = W_fc [h_t^(1); ...; h_t^(S)] + b_fc.

    hidden: [S, n, H] (target layer major); w_fc: [H, S*H] ([out, in], the input being
    the S rows of a position concatenated in layer order); b_fc: [H] or None.
    Returns C: [n, H], one row per position, shared by every draft layer.
    """
    S, n, H = hidden.shape
    concat = np.transpose(hidden, (1, 0, 2)).reshape(n, S * H)
    out = concat @ w_fc.T
    return out if b_fc is None else out + b_fc


def block_attention(q, k_ctx, v_ctx, k_blk, v_blk) -> np.ndarray:
    """Block attention without any mask  (Sec. 3.2, drafting phase; Sec. 4.2).

    q: [B, n_q, hd]; k_ctx/v_ctx: [L, n_kv, hd]; k_blk/v_blk: [B, n_kv, hd].
    Every block row attends to all L context keys and all B block keys (itself
    included).  Query head h uses KV head h // (n_q / n_kv).  Returns [B, n_q, hd].
    """
    B, nq, hd = q.shape
    nkv = k_blk.shape[1]
    group = nq // nkv
    keys = np.concatenate([k_ctx, k_blk], axis=0)
    vals = np.concatenate([v_ctx, v_blk], axis=0)
    out = np.empty_like(q)
    for h in range(nq):
        g = h // group
        s = (q[:, h, :] @ keys[:, g, :].T) / math.sqrt(hd)
        s = s - s.max(axis=1, keepdims=True)
        p = np.exp(s)
        p = p / p.sum(axis=1, keepdims=True)
        out[:, h, :] = p @ vals[:, g, :]
    return out


def draft_layer(X, lw: dict, k_ctx, v_ctx, positions, cfg) -> np.ndarray:
    """One draft Transformer layer over the B block rows.

    lw holds this layer's fp64 weights: attn_norm, mlp_norm [H]; wq, wk_d, wv_d,
    wo, w_gate, w_up, w_down as [out, in].  Queries and block keys/values come from
    the block rows through W_Q, W_K^d, W_V^d (Eq. 4); the context K/V come from the
    cache.  Returns the new block rows [B, H].
    """
    B = X.shape[0]
    nq, nkv, hd = cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim
    a = rms_norm(X, lw["attn_norm"], cfg.rms_eps)
    q = rope((a @ lw["wq"].T).reshape(B, nq, hd), positions, cfg.rope_base)
    kb = rope((a @ lw["wk_d"].T).reshape(B, nkv, hd), positions, cfg.rope_base)
    vb = (a @ lw["wv_d"].T).reshape(B, nkv, hd)
    o = block_attention(q, k_ctx, v_ctx, kb, vb).reshape(B, nq * hd)
    X = X + o @ lw["wo"].T
    m = rms_norm(X, lw["mlp_norm"], cfg.rms_eps)
    return X + (silu(m @ lw["w_gate"].T) * (m @ lw["w_up"].T)) @ lw["w_down"].T


def lm_head_logits(X, final_norm, lm_head_bf16, eps: float, chunk: int = 16384) -> np.ndarray:
    """Logits z = RMSNorm(X; g_final) W_lm^T over the full vocabulary (Sec. 3.2).

    lm_head_bf16: [V, H] bf16 bits, converted in vocabulary chunks.
    """
    xn = rms_norm(X, final_norm, eps)
    V = lm_head_bf16.shape[0]
    z = np.empty((X.shape[0], V), dtype=np.float64)
    for v0 in range(0, V, chunk):
        z[:, v0:v0 + chunk] = xn @ bf16_to_f64(lm_head_bf16[v0:v0 + chunk]).T
    return z


def argmax_lowest(z: np.ndarray) -> np.ndarray:
    """Greedy token per row: the lowest index among the maxima."""
    return np.argmax(z, axis=-1).astype(np.int32)


# ---- temperature sampling (the paper's temperature-1 decoding, Sec. 5, Table 1 lower half) ----
# A candidate is drawn from softmax(z / T) by the Gumbel-max rule: argmax_v (z_v / T + G_v) with
# G_v = -log(-log(U_v)) and U_v independent uniforms on (0, 1).  The uniforms come from the
# counter-based generator Philox4x64-10 (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as
# easy as 1, 2, 3", SC 2011) keyed by (seed, 0): U of vocabulary id v at block position b in draw
# `draw` of sequence slot `slot` is made from output word b mod 4 at counter (v, b div 4, draw,
# slot), so one generator call serves four consecutive positions; U = (top 23 bits of the word +
# 1/2) / 2^23, a value that single precision holds exactly and that stays below 1 there too, so a
# kernel computing the noise in fp32 never meets log(1).  These generator details are this
# library's convention (the paper fixes none of them).

_PHILOX_M0 = np.uint64(0xD2E7470EE14C6C93)
_PHILOX_M1 = np.uint64(0xCA5A826395121157)
_PHILOX_W0 = np.uint64(0x9E3779B97F4A7C15)
_PHILOX_W1 = np.uint64(0xBB67AE8584CAA73B)


def _mulhilo64(a: np.ndarray, m: np.uint64):
    """(high, low) 64-bit halves of the 128-bit products a * m, from 32-bit partial products."""
    m32 = np.uint64(0xFFFFFFFF)
    s32 = np.uint64(32)
    a_lo, a_hi = a & m32, a >> s32
    m_lo, m_hi = m & m32, m >> s32
    ll, lh, hl, hh = a_lo * m_lo, a_lo * m_hi, a_hi * m_lo, a_hi * m_hi
    mid = (ll >> s32) + (lh & m32) + (hl & m32)
    lo = (ll & m32) | ((mid & m32) << s32)
    hi = hh + (lh >> s32) + (hl >> s32) + (mid >> s32)
    return hi, lo


def philox4x64_10(counter, key):
    """Philox4x64 with 10 rounds (Salmon et al. 2011): counter = 4 uint64 arrays (broadcast),
    key = 2 uint64 values.  Each round multiplies words 0 and 2 by the two round constants,
    mixes the high halves with words 1, 3 and the key, and bumps the key by the Weyl constants."""
    c0, c1, c2, c3 = (np.asarray(x, dtype=np.uint64) for x in counter)
    c0, c1, c2, c3 = np.broadcast_arrays(c0, c1, c2, c3)
    k0, k1 = np.uint64(key[0]), np.uint64(key[1])
    with np.errstate(over="ignore"):
        for _ in range(10):
            hi0, lo0 = _mulhilo64(c0, _PHILOX_M0)
            hi1, lo1 = _mulhilo64(c2, _PHILOX_M1)
            c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
            k0 = np.uint64((int(k0) + int(_PHILOX_W0)) & 0xFFFFFFFFFFFFFFFF)
            k1 = np.uint64((int(k1) + int(_PHILOX_W1)) & 0xFFFFFFFFFFFFFFFF)
    return c0, c1, c2, c3


def sampling_uniforms(seed: int, draw: int, slot: int, n_pos: int, vocab: int) -> np.ndarray:
    """U[b, v] in (0, 1) for block positions b < n_pos and vocabulary ids v < vocab."""
    v = np.arange(vocab, dtype=np.uint64)[None, :]
    b = np.arange(n_pos, dtype=np.uint64)[:, None]
    words = np.stack(philox4x64_10((v, b >> np.uint64(2), np.uint64(draw), np.uint64(slot)),
                                   (np.uint64(seed), np.uint64(0))))  # [4, n_pos, vocab]
    w = words[(np.arange(n_pos) % 4)[:, None], np.arange(n_pos)[:, None], np.arange(vocab)[None, :]]
    return ((w >> np.uint64(41)).astype(np.float64) + 0.5) / float(1 << 23)


def sample_tokens(z: np.ndarray, temperature: float, seed: int, draw: int, slot: int = 0):
    """Candidates from logits z [B, V]: greedy argmax for temperature <= 0, else the
    Gumbel-max draw from softmax(z / temperature).  Returns (tokens, perturbed scores)."""
    if temperature <= 0:
        return argmax_lowest(z), z
    u = sampling_uniforms(seed, draw, slot, z.shape[0], z.shape[1])
    y = z / temperature - np.log(-np.log(u))
    return argmax_lowest(y), y


def accept_block(draft_tokens, target_tokens):
    """One verification (Sec. 3.2, verification phase).  The block is x_t followed by the
    candidates draft_tokens[1..B-1]; target_tokens[b] is the target's own next token after
    block position b.  The longest prefix of candidates equal to the target's predictions is
    accepted (k of them, 0 <= k <= B-1), and the target's prediction after the last accepted
    position is the bonus token.  Returns (k, bonus, emitted) with emitted = the k accepted
    candidates followed by the bonus token (k + 1 tokens)."""
    d = [int(x) for x in draft_tokens]
    t = [int(x) for x in target_tokens]
    B = len(d)
    k = 0
    while k + 1 < B and d[k + 1] == t[k]:
        k += 1
    return k, t[k], d[1:k + 1] + [t[k]]


_LAYER_KINDS = ("attn_norm", "mlp_norm", "wq", "wk_d", "wv_d", "wo", "w_gate", "w_up", "w_down")


class DraftOracle:
    """Stateful fp64 draft model: a context cache per draft layer plus block passes.

    cfg: any object with the attributes hidden, n_q_heads, n_kv_heads, head_dim,
    ffn, vocab, n_draft_layers, n_target_layers, block_size, rope_base, rms_eps.
    weights: dict of bf16 bit arrays as laid out by the input generator
    (embed, lm_head [V, H]; final_norm [H]; fuse/attn/mlp_norm [D, H]; linear
    weights [D, out, in]); a norm entry may be None for unit gains.
    fusion_logits: [D, S].
    """

    def __init__(self, cfg, weights: dict, fusion_logits, max_context: int = 1 << 16,
                 cache_weights: bool = False, variant: int = 0):
        self.cfg = cfg
        self.w = weights
        self.variant = variant
        D = cfg.n_draft_layers
        if variant & ~15 or (variant & VARIANT_DFLASH and variant != VARIANT_DFLASH):
            raise ValueError("unknown variant, or DFlash combined with another variant")
        if variant & VARIANT_DFLASH:
            self.alpha = None
        else:
            self.alpha = fusion_weights(fusion_logits, normalize=not variant & VARIANT_NO_SOFTMAX)
            if self.alpha.shape != (D, cfg.n_target_layers):
                raise ValueError("fusion logits must be [D, S]")
        self.max_context = max_context
        self.L = 0
        # context keys/values per draft layer, grown by doubling; rows [0, L) are live
        self._k = [np.zeros((0, cfg.n_kv_heads, cfg.head_dim)) for _ in range(D)]
        self._v = [np.zeros((0, cfg.n_kv_heads, cfg.head_dim)) for _ in range(D)]
        self._cache_weights = cache_weights
        self._lw: dict[int, dict] = {}
        self.last_fused = None

    @property
    def k_cache(self):
        """Context keys per draft layer, each [L, n_kv, hd] (after RoPE)."""
        return [k[:self.L] for k in self._k]

    @property
    def v_cache(self):
        """Context values per draft layer, each [L, n_kv, hd]."""
        return [v[:self.L] for v in self._v]

    def _reserve(self, n: int) -> None:
        cap = self._k[0].shape[0]
        if n <= cap:
            return
        cap = max(n, 2 * cap)
        for lst in (self._k, self._v):
            for i, a in enumerate(lst):
                b = np.zeros((cap,) + a.shape[1:])
                b[:self.L] = a[:self.L]
                lst[i] = b

    # -- weights -------------------------------------------------------------
    def _gain(self, kind, i=None):
        g = self.w.get(kind)
        if g is None:
            return None
        return bf16_to_f64(g if i is None else g[i])

    def layer_weights(self, i: int) -> dict:
        if i in self._lw:
            return self._lw[i]
        lw = {k: (self._gain(k, i) if k.endswith("norm") else bf16_to_f64(self.w[k][i]))
              for k in _LAYER_KINDS}
        if self._cache_weights:
            self._lw[i] = lw
        return lw

    # -- context -------------------------------------------------------------
    def append(self, hidden_bf16, positions=None) -> np.ndarray:
        """Fuse n new target rows [S, n, H] and append their K/V to every layer.

        Returns the fused rows [D, n, H] (Eq. 3; with +FC after the extra layer; with DFlash
        the shared context C of Eq. 1 for every layer).  Positions default to L..L+n-1.
        """
        cfg = self.cfg
        h = bf16_to_f64(hidden_bf16)
        S, n, H = h.shape
        if S != cfg.n_target_layers or H != cfg.hidden:
            raise ValueError("target hidden rows must be [S, n, H]")
        if self.L + n > self.max_context:
            raise ValueError("context full")
        pos = np.arange(self.L, self.L + n) if positions is None else np.asarray(positions)
        D = cfg.n_draft_layers
        if self.variant & VARIANT_DFLASH:
            b = self.w.get("fc_bias")
            c = dflash_context(h, bf16_to_f64(self.w["fc"]), None if b is None else bf16_to_f64(b))
            f = np.broadcast_to(c, (D,) + c.shape)
        else:
            fuse_g = self.w.get("fuse_norm")
            gains = None if fuse_g is None else bf16_to_f64(fuse_g)
            f = fuse_rows(self.alpha, h, gains, cfg.rms_eps)
            if self.variant & VARIANT_POST_FC:
                bias = self.w.get("post_fc_bias")
                f = np.stack([post_fc(f[i], bf16_to_f64(self.w["post_fc"][i]),
                                      None if bias is None else bf16_to_f64(bias[i])) for i in range(D)])
        shared = self.variant & (VARIANT_SHARED_KV | VARIANT_DFLASH)
        wk, wv = ("wk_d", "wv_d") if shared else ("wk_t", "wv_t")
        self._reserve(self.L + n)
        for i in range(D):
            k, v = context_kv(f[i], bf16_to_f64(self.w[wk][i]), bf16_to_f64(self.w[wv][i]),
                              pos, cfg.n_kv_heads, cfg.head_dim, cfg.rope_base)
            self._k[i][self.L:self.L + n] = k
            self._v[i][self.L:self.L + n] = v
        self.L += n
        self.last_fused = f
        return f

    def accept(self, draft_tokens, target_tokens, target_hidden_bf16):
        """Verify a drafted block against the target's outputs and append the target rows of
        the verified positions: target_hidden [S, B, H] holds the target's hidden rows at the
        B block positions; rows 0..k (x_t and the k accepted candidates) become context rows
        L .. L + k.  Returns (k, bonus, emitted) as accept_block; the bonus token is the x_t of
        the next block."""
        k, bonus, emitted = accept_block(draft_tokens, target_tokens)
        self.append(np.asarray(target_hidden_bf16)[:, :k + 1])
        return k, bonus, emitted

    def truncate(self, new_len: int) -> None:
        if not 0 <= new_len <= self.L:
            raise ValueError("truncate length out of range")
        self.L = new_len

    # -- block pass ----------------------------------------------------------
    def draft_block(self, ids, positions=None, keep_logits: bool = True, temperature: float = 0.0,
                    seed: int = 0, draw: int = 0, slot: int = 0) -> dict:
        """One drafting forward pass over the block ids [B]  (Sec. 3.2).

        Returns dict(tokens [B] int32, logits [B, V] (if keep_logits),
        hidden [D, B, H] = block rows after each layer).  With temperature > 0 the
        tokens are Gumbel-max draws (see sample_tokens) and "scores" holds the
        perturbed scores z / T + G they maximise.
        """
        cfg = self.cfg
        ids = np.asarray(ids, dtype=np.int64)
        B = ids.shape[0]
        pos = np.arange(self.L, self.L + B) if positions is None else np.asarray(positions)
        X = bf16_to_f64(self.w["embed"][ids])
        hs = []
        for i in range(cfg.n_draft_layers):
            X = draft_layer(X, self.layer_weights(i), self._k[i][:self.L], self._v[i][:self.L], pos, cfg)
            hs.append(X)
        z = lm_head_logits(X, self._gain("final_norm"), self.w["lm_head"], cfg.rms_eps)
        tokens, scores = sample_tokens(z, temperature, seed, draw, slot)
        out = {"tokens": tokens, "hidden": np.stack(hs)}
        if keep_logits:
            out["logits"] = z
            out["scores"] = scores
        return out
