"""Planted mistakes in the oracle (on the CPU): each must trip at least one pin.

Every mutant below is a plausible slip -- a dropped term, a wrong sign, a wrong
index or axis, a transposed operand -- patched into the oracle module for the
duration of one test.  The test passes when at least one check of
tests/test_oracle_pins.py fails under the mutant, i.e. the pins are strong
enough to notice it.
"""
import math

import numpy as np
import pytest

from oracle import dflare_oracle as orc
import test_oracle_pins as pins


def _softmax_wrong_axis(lg, normalize=True):
    lg = np.asarray(lg, np.float64)
    e = np.exp(lg - lg.max(axis=0, keepdims=True))
    return e / e.sum(axis=0, keepdims=True)


def _softmax_unnormalised(lg, normalize=True):
    return np.exp(np.asarray(lg, np.float64))


def _fuse_drop_last(alpha, hidden, gains, eps):
    D, S = alpha.shape
    out = np.empty((D,) + hidden.shape[1:])
    for i in range(D):
        u = sum(alpha[i, j] * hidden[j] for j in range(S - 1))
        out[i] = orc.rms_norm(u, None if gains is None else gains[i], eps)
    return out


def _fuse_reversed_layers(alpha, hidden, gains, eps):
    return _ORIG["fuse_rows"](alpha[:, ::-1], hidden, gains, eps)


def _fuse_no_norm(alpha, hidden, gains, eps):
    D, S = alpha.shape
    return np.stack([sum(alpha[i, j] * hidden[j] for j in range(S)) for i in range(D)])


def _rms_eps_outside(x, gain, eps):
    y = x / (np.sqrt(np.mean(x * x, axis=-1, keepdims=True)) + eps)
    return y if gain is None else y * gain


def _rms_sum(x, gain, eps):
    y = x / np.sqrt(np.sum(x * x, axis=-1, keepdims=True) + eps)
    return y if gain is None else y * gain


def _rope_sign(x, positions, base):
    y = _ORIG["rope"](x, -np.asarray(positions, np.float64), base)
    return y


def _rope_interleaved(x, positions, base):
    hd = x.shape[-1]
    inv = base ** (-(2.0 * np.arange(hd // 2)) / hd)
    th = np.asarray(positions, np.float64)[:, None] * inv[None, :]
    c, s = np.cos(th)[:, None, :], np.sin(th)[:, None, :]
    x1, x2 = x[..., 0::2], x[..., 1::2]
    out = np.empty_like(x)
    out[..., 0::2] = x1 * c - x2 * s
    out[..., 1::2] = x2 * c + x1 * s
    return out


def _rope_wrong_freq(x, positions, base):
    hd = x.shape[-1]
    half = hd // 2
    inv = base ** (-(np.arange(half, dtype=np.float64)) / hd)
    th = np.asarray(positions, np.float64)[:, None] * inv[None, :]
    c, s = np.cos(th)[:, None, :], np.sin(th)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def _kv_no_rope(f_i, wk_t, wv_t, positions, n_kv, hd, base):
    n = f_i.shape[0]
    return (f_i @ wk_t.T).reshape(n, n_kv, hd), (f_i @ wv_t.T).reshape(n, n_kv, hd)


def _kv_rope_on_v(f_i, wk_t, wv_t, positions, n_kv, hd, base):
    k, v = _ORIG["context_kv"](f_i, wk_t, wv_t, positions, n_kv, hd, base)
    return k, orc.rope(v, positions, base)


def _kv_swapped(f_i, wk_t, wv_t, positions, n_kv, hd, base):
    return _ORIG["context_kv"](f_i, wv_t, wk_t, positions, n_kv, hd, base)


def _attn_variant(gqa_mod=False, no_scale=False, causal=False, drop_block=False, drop_ctx=False):
    def attn(q, k_ctx, v_ctx, k_blk, v_blk):
        B, nq, hd = q.shape
        nkv = k_blk.shape[1]
        L = k_ctx.shape[0]
        if drop_ctx:
            k_ctx, v_ctx, L = k_ctx[:0], v_ctx[:0], 0
        keys = k_ctx if drop_block else np.concatenate([k_ctx, k_blk])
        vals = v_ctx if drop_block else np.concatenate([v_ctx, v_blk])
        out = np.empty_like(q)
        for h in range(nq):
            g = h % nkv if gqa_mod else h // (nq // nkv)
            s = q[:, h] @ keys[:, g].T
            if not no_scale:
                s = s / math.sqrt(hd)
            if causal:
                for b in range(B):
                    s[b, L + b + 1:] = -np.inf
            s = s - s.max(axis=1, keepdims=True)
            p = np.exp(s)
            out[:, h] = (p / p.sum(axis=1, keepdims=True)) @ vals[:, g]
        return out
    return attn


def _layer_variant(no_attn_residual=False, bad_silu=False, swap_gate_up=False, kb_no_rope=False,
                   wo_transposed=False, no_mlp_norm=False):
    def layer(X, lw, k_ctx, v_ctx, positions, cfg):
        B = X.shape[0]
        nq, nkv, hd = cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim
        a = orc.rms_norm(X, lw["attn_norm"], cfg.rms_eps)
        q = orc.rope((a @ lw["wq"].T).reshape(B, nq, hd), positions, cfg.rope_base)
        kb = (a @ lw["wk_d"].T).reshape(B, nkv, hd)
        if not kb_no_rope:
            kb = orc.rope(kb, positions, cfg.rope_base)
        vb = (a @ lw["wv_d"].T).reshape(B, nkv, hd)
        o = orc.block_attention(q, k_ctx, v_ctx, kb, vb).reshape(B, nq * hd)
        proj = o @ (lw["wo"] if wo_transposed else lw["wo"].T)
        X = proj if no_attn_residual else X + proj
        m = X if no_mlp_norm else orc.rms_norm(X, lw["mlp_norm"], cfg.rms_eps)
        g, u = m @ lw["w_gate"].T, m @ lw["w_up"].T
        if swap_gate_up:
            g, u = u, g
        act = g / (1.0 + np.exp(g)) if bad_silu else orc.silu(g)
        return X + (act * u) @ lw["w_down"].T
    return layer


def _lm_no_norm(X, final_norm, lm_head_bf16, eps, chunk=16384):
    return X @ orc.bf16_to_f64(lm_head_bf16).T


def _argmax_highest(z):
    return (z.shape[-1] - 1 - np.argmax(z[..., ::-1], axis=-1)).astype(np.int32)


def _sample_exponential_noise(z, temperature, seed, draw, slot=0):
    if temperature <= 0:
        return orc.argmax_lowest(z), z
    u = orc.sampling_uniforms(seed, draw, slot, z.shape[0], z.shape[1])
    y = z / temperature - np.log(u)  # exponential, not Gumbel, noise
    return orc.argmax_lowest(y), y


def _sample_temperature_multiplies(z, temperature, seed, draw, slot=0):
    if temperature <= 0:
        return orc.argmax_lowest(z), z
    u = orc.sampling_uniforms(seed, draw, slot, z.shape[0], z.shape[1])
    y = z * temperature - np.log(-np.log(u))
    return orc.argmax_lowest(y), y


def _philox_no_key_schedule(counter, key):
    c0, c1, c2, c3 = np.broadcast_arrays(*(np.asarray(x, dtype=np.uint64) for x in counter))
    k0, k1 = np.uint64(key[0]), np.uint64(key[1])
    for _ in range(10):
        hi0, lo0 = orc._mulhilo64(c0, orc._PHILOX_M0)
        hi1, lo1 = orc._mulhilo64(c2, orc._PHILOX_M1)
        c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
    return c0, c1, c2, c3


def _philox_swapped_multipliers(counter, key):
    c0, c1, c2, c3 = np.broadcast_arrays(*(np.asarray(x, dtype=np.uint64) for x in counter))
    k0, k1 = int(key[0]), int(key[1])
    for _ in range(10):
        hi0, lo0 = orc._mulhilo64(c0, orc._PHILOX_M1)
        hi1, lo1 = orc._mulhilo64(c2, orc._PHILOX_M0)
        c0, c1, c2, c3 = hi1 ^ c1 ^ np.uint64(k0), lo1, hi0 ^ c3 ^ np.uint64(k1), lo0
        k0 = (k0 + int(orc._PHILOX_W0)) & 0xFFFFFFFFFFFFFFFF
        k1 = (k1 + int(orc._PHILOX_W1)) & 0xFFFFFFFFFFFFFFFF
    return c0, c1, c2, c3


def _uniform_words(seed, draw, slot, n_pos, vocab):
    v = np.arange(vocab, dtype=np.uint64)[None, :]
    b = np.arange(n_pos, dtype=np.uint64)[:, None]
    words = np.stack(orc.philox4x64_10((v, b >> np.uint64(2), np.uint64(draw), np.uint64(slot)),
                                       (np.uint64(seed), np.uint64(0))))
    return words[(np.arange(n_pos) % 4)[:, None], np.arange(n_pos)[:, None], np.arange(vocab)[None, :]]


def _uniforms_24_bits(seed, draw, slot, n_pos, vocab):
    w = _uniform_words(seed, draw, slot, n_pos, vocab)
    return ((w >> np.uint64(40)).astype(np.float64) + 0.5) / float(1 << 24)  # not exact in fp32


def _uniforms_word0_only(seed, draw, slot, n_pos, vocab):
    v = np.arange(vocab, dtype=np.uint64)[None, :]
    b = np.arange(n_pos, dtype=np.uint64)[:, None]
    w = orc.philox4x64_10((v, b >> np.uint64(2), np.uint64(draw), np.uint64(slot)),
                          (np.uint64(seed), np.uint64(0)))[0]  # four positions share one number
    return ((w >> np.uint64(41)).astype(np.float64) + 0.5) / float(1 << 23)


def _no_softmax_still_normalises(lg, normalize=True):
    return _ORIG["fusion_weights"](lg)


def _post_fc_transposed(f_i, w, b):
    out = f_i @ w
    return out if b is None else out + b


def _post_fc_drops_bias(f_i, w, b):
    return f_i @ w.T


def _dflash_concat_wrong_order(hidden, w_fc, b_fc):
    S, n, H = hidden.shape
    concat = hidden.reshape(S * H, n).T  # not the S rows of one position side by side
    out = concat @ w_fc.T
    return out if b_fc is None else out + b_fc


def _dflash_drops_bias(hidden, w_fc, b_fc):
    return _ORIG["dflash_context"](hidden, w_fc, None)


def _accept_bonus_off_by_one(draft_tokens, target_tokens):
    d, t = list(draft_tokens), list(target_tokens)
    k = 0
    while k + 1 < len(d) and d[k + 1] == t[k]:
        k += 1
    b = t[min(k + 1, len(t) - 1)]
    return k, b, d[1:k + 1] + [b]


def _accept_compares_same_position(draft_tokens, target_tokens):
    d, t = list(draft_tokens), list(target_tokens)
    k = 0
    while k + 1 < len(d) and d[k + 1] == t[k + 1]:
        k += 1
    return k, t[k], d[1:k + 1] + [t[k]]


_ORIG = {k: getattr(orc, k) for k in ("fuse_rows", "rope", "context_kv", "fusion_weights", "dflash_context")}

MUTANTS = {
    "softmax_wrong_axis": ("fusion_weights", _softmax_wrong_axis),
    "softmax_unnormalised": ("fusion_weights", _softmax_unnormalised),
    "fuse_drops_last_layer": ("fuse_rows", _fuse_drop_last),
    "fuse_reversed_layers": ("fuse_rows", _fuse_reversed_layers),
    "fuse_without_rmsnorm": ("fuse_rows", _fuse_no_norm),
    "rmsnorm_eps_outside_sqrt": ("rms_norm", _rms_eps_outside),
    "rmsnorm_sum_not_mean": ("rms_norm", _rms_sum),
    "rope_wrong_sign": ("rope", _rope_sign),
    "rope_interleaved_pairs": ("rope", _rope_interleaved),
    "rope_wrong_frequency": ("rope", _rope_wrong_freq),
    "context_k_not_rotated": ("context_kv", _kv_no_rope),
    "context_v_rotated": ("context_kv", _kv_rope_on_v),
    "context_k_v_swapped": ("context_kv", _kv_swapped),
    "gqa_head_modulo": ("block_attention", _attn_variant(gqa_mod=True)),
    "attention_unscaled": ("block_attention", _attn_variant(no_scale=True)),
    "attention_causal_in_block": ("block_attention", _attn_variant(causal=True)),
    "attention_drops_block_keys": ("block_attention", _attn_variant(drop_block=True)),
    "attention_drops_context": ("block_attention", _attn_variant(drop_ctx=True)),
    "layer_no_attention_residual": ("draft_layer", _layer_variant(no_attn_residual=True)),
    "layer_silu_sign": ("draft_layer", _layer_variant(bad_silu=True)),
    "layer_gate_up_swapped": ("draft_layer", _layer_variant(swap_gate_up=True)),
    "layer_block_k_not_rotated": ("draft_layer", _layer_variant(kb_no_rope=True)),
    "layer_wo_transposed": ("draft_layer", _layer_variant(wo_transposed=True)),
    "layer_no_mlp_norm": ("draft_layer", _layer_variant(no_mlp_norm=True)),
    "lm_head_without_final_norm": ("lm_head_logits", _lm_no_norm),
    "argmax_ties_to_highest": ("argmax_lowest", _argmax_highest),
    "sampling_exponential_noise": ("sample_tokens", _sample_exponential_noise),
    "sampling_temperature_multiplies": ("sample_tokens", _sample_temperature_multiplies),
    "philox_without_key_schedule": ("philox4x64_10", _philox_no_key_schedule),
    "philox_multipliers_swapped": ("philox4x64_10", _philox_swapped_multipliers),
    "uniforms_not_exact_in_fp32": ("sampling_uniforms", _uniforms_24_bits),
    "uniforms_same_word_for_four_positions": ("sampling_uniforms", _uniforms_word0_only),
    "no_softmax_still_normalises": ("fusion_weights", _no_softmax_still_normalises),
    "post_fc_transposed": ("post_fc", _post_fc_transposed),
    "post_fc_drops_bias": ("post_fc", _post_fc_drops_bias),
    "dflash_concat_wrong_order": ("dflash_context", _dflash_concat_wrong_order),
    "dflash_drops_bias": ("dflash_context", _dflash_drops_bias),
    "accept_bonus_off_by_one": ("accept_block", _accept_bonus_off_by_one),
    "accept_compares_same_position": ("accept_block", _accept_compares_same_position),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, monkeypatch):
    attr, fn = MUTANTS[name]
    monkeypatch.setattr(orc, attr, fn)
    caught = []
    for chk in pins.ALL_CHECKS:
        try:
            chk()
        except Exception:  # noqa: BLE001 - any failure counts as detection
            caught.append(chk.__name__)
    assert caught, f"mutant {name} passed every pin"


def test_unmutated_oracle_passes_every_pin():
    for chk in pins.ALL_CHECKS:
        chk()
