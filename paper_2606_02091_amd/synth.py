"""Seeded synthetic inputs for the DFlare draft step.

This module only draws random numbers and rounds them to bfloat16 storage.  It
holds none of the method's arithmetic, so both the fp64 oracle (tests) and the
HIP path (library, bench) can consume exactly the same bits.

Workloads (model shapes follow the draft models the paper pairs with its target
models, Sec. 5.1; value distributions are synthetic stand-ins because no trained
weights or benchmark data are used):

  tiny         H=256,  4q/2kv x 64,  F=768,   V=1024,   D=2, S=6,  L=64,   B=8
  qwen3_4b     H=2560, 32q/8kv x 128, F=9728, V=151936, D=8, S=18, L=2048, B=16
  qwen3_8b     H=4096, 32q/8kv x 128, F=12288,V=151936, D=8, S=36, L=4096, B=16
  gpt_oss_20b  H=2880, 64q/8kv x 64,  F=2880, V=201088, D=8, S=24, L=8192, B=16

Distributions: projection weights, embedding and LM head N(0, 0.02); RMSNorm
gains 1 + N(0, 0.02); fusion logits N(0, 1); target hidden rows N(0, 1) with
target layer s (0-based) scaled by (1 + 0.2 s).  Every float tensor is rounded
to bfloat16 (round to nearest even) before either side sees it.

Seeds: weights 0, hidden stream 1, append sizes 2, block ids 3.
"""
from __future__ import annotations

import dataclasses
from concurrent.futures import ThreadPoolExecutor

import numpy as np

__all__ = [
    "ModelConfig", "CONFIGS", "round_bf16", "bf16_to_f32", "make_weights",
    "hidden_rows", "append_sizes", "block_ids", "WEIGHT_KINDS", "BATCHED", "batched_lengths",
]


@dataclasses.dataclass(frozen=True)
class ModelConfig:
    name: str
    hidden: int          # H (the paper's d)
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    ffn: int
    vocab: int
    n_draft_layers: int  # D
    n_target_layers: int  # S (the paper's T)
    block_size: int      # B
    context: int         # L used by the workload
    rope_base: float = 1.0e6
    rms_eps: float = 1.0e-6
    append_chunk: int = 8  # chunk size of the context prefill in the workload
    random_block: bool = False  # tiny: B random ids; others: [id, mask x (B-1)]

    @property
    def q_dim(self) -> int:
        return self.n_q_heads * self.head_dim

    @property
    def kv_dim(self) -> int:
        return self.n_kv_heads * self.head_dim

    def replace(self, **kw) -> "ModelConfig":
        return dataclasses.replace(self, **kw)

    # algorithmic HBM bytes of one draft block and of one append (bf16 storage)
    def block_bytes(self, L: int | None = None) -> int:
        L = self.context if L is None else L
        H, F, V, D = self.hidden, self.ffn, self.vocab, self.n_draft_layers
        q, kv = self.q_dim, self.kv_dim
        weights = D * (H * q + 2 * H * kv + q * H + 3 * H * F) + V * H
        return weights * 2 + D * 2 * L * kv * 2 + self.block_size * H * 2

    def append_bytes(self, n_new: float) -> float:
        H, D, S, kv = self.hidden, self.n_draft_layers, self.n_target_layers, self.kv_dim
        return D * 2 * H * kv * 2 + S * n_new * H * 2 + D * 2 * n_new * kv * 2


CONFIGS: dict[str, ModelConfig] = {
    "tiny": ModelConfig("tiny", 256, 4, 2, 64, 768, 1024, 2, 6, 8, 64,
                        append_chunk=8, random_block=True),
    "qwen3_4b": ModelConfig("qwen3_4b", 2560, 32, 8, 128, 9728, 151936, 8, 18, 16, 2048,
                            append_chunk=512),
    "qwen3_8b": ModelConfig("qwen3_8b", 4096, 32, 8, 128, 12288, 151936, 8, 36, 16, 4096,
                            append_chunk=512),
    "gpt_oss_20b": ModelConfig("gpt_oss_20b", 2880, 64, 8, 64, 2880, 201088, 8, 24, 16, 8192,
                               append_chunk=512),
}

# Order in which weight tensors are drawn; each gets its own child seed so that
# they can be drawn in parallel and a single tensor can be regenerated alone.
BASE_KINDS = (
    "embed", "lm_head", "final_norm", "fusion_logits",
    "fuse_norm", "attn_norm", "mlp_norm",
    "wq", "wk_d", "wv_d", "wk_t", "wv_t", "wo", "w_gate", "w_up", "w_down",
)
# weights of the model variants only: the +FC layer after the fusion and the DFlash FC
# fusion (Eq. 1); drawn only when asked for
VARIANT_KINDS = ("post_fc", "post_fc_bias", "fc", "fc_bias")
WEIGHT_KINDS = BASE_KINDS + VARIANT_KINDS


def round_bf16(x: np.ndarray, out: np.ndarray | None = None) -> np.ndarray:
    """float32 -> bfloat16 bit patterns (uint16), round to nearest even.

    NaN maps to the quiet NaN 0x7FC0.  `out` (uint16, same size) may be given.
    """
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    r = (u >> np.uint32(16)) & np.uint32(1)
    r += np.uint32(0x7FFF)
    r += u
    r >>= np.uint32(16)
    if out is None:
        out = np.empty(x.shape, np.uint16)
    np.copyto(out, r, casting="unsafe")
    nan = np.isnan(x)
    if nan.any():
        out[nan] = 0x7FC0
    return out


def bf16_to_f32(u: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns (uint16) -> float32 (exact)."""
    return (np.asarray(u, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def _shape(cfg: ModelConfig, kind: str) -> tuple[int, ...]:
    H, D, S = cfg.hidden, cfg.n_draft_layers, cfg.n_target_layers
    q, kv, F, V = cfg.q_dim, cfg.kv_dim, cfg.ffn, cfg.vocab
    return {
        "embed": (V, H), "lm_head": (V, H), "final_norm": (H,), "fusion_logits": (D, S),
        "fuse_norm": (D, H), "attn_norm": (D, H), "mlp_norm": (D, H),
        "wq": (D, q, H), "wk_d": (D, kv, H), "wv_d": (D, kv, H),
        "wk_t": (D, kv, H), "wv_t": (D, kv, H), "wo": (D, H, q),
        "w_gate": (D, F, H), "w_up": (D, F, H), "w_down": (D, H, F),
        "post_fc": (D, H, H), "post_fc_bias": (D, H), "fc": (H, S * H), "fc_bias": (H,),
    }[kind]


_CHUNK = 1 << 22  # values per independently seeded chunk


def _draw_chunk(kind: str, idx: int, seed: int, c: int, flat_out: np.ndarray) -> None:
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, idx, c])))
    n = flat_out.size
    z = rng.standard_normal(size=n, dtype=np.float32)
    z *= np.float32(0.02)
    if kind.endswith("norm"):
        z += np.float32(1.0)                 # gains 1 + N(0, 0.02)
    round_bf16(z, out=flat_out)


def make_weights(cfg: ModelConfig, seed: int = 0, kinds=BASE_KINDS,
                 threads: int = 8) -> dict[str, np.ndarray]:
    """All draft weights as bf16 bit arrays (uint16); fusion logits as float32.

    Linear weights use the [out, in] row-major convention, stacked over the D
    draft layers: y = x @ W.T.  Each tensor is drawn in chunks of 2^22 values,
    chunk c of tensor kind k seeded by (seed, k, c), so the result does not
    depend on the thread count.
    """
    out: dict[str, np.ndarray] = {}
    jobs = []
    for kind in kinds:
        idx = WEIGHT_KINDS.index(kind)
        shape = _shape(cfg, kind)
        if kind == "fusion_logits":           # host fp32 logits, N(0, 1)
            rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, idx])))
            out[kind] = rng.standard_normal(size=shape, dtype=np.float32)
            continue
        arr = np.empty(shape, np.uint16)
        flat = arr.reshape(-1)
        for c, lo in enumerate(range(0, flat.size, _CHUNK)):
            jobs.append((kind, idx, c, flat[lo:lo + _CHUNK]))
        out[kind] = arr
    if threads <= 1:
        for kind, idx, c, view in jobs:
            _draw_chunk(kind, idx, seed, c, view)
    else:
        with ThreadPoolExecutor(max_workers=threads) as ex:
            list(ex.map(lambda j: _draw_chunk(j[0], j[1], seed, j[2], j[3]), jobs))
    return {k: out[k] for k in kinds}


_ROW_BLOCK = 64


def _hidden_block(cfg: ModelConfig, blk: int, seed: int) -> np.ndarray:
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 7919, blk])))
    z = rng.standard_normal(size=(cfg.n_target_layers, _ROW_BLOCK, cfg.hidden), dtype=np.float32)
    scale = (1.0 + 0.2 * np.arange(cfg.n_target_layers, dtype=np.float32))[:, None, None]
    return round_bf16(z * scale)


def hidden_rows(cfg: ModelConfig, start: int, n: int, seed: int = 1) -> np.ndarray:
    """Target hidden rows for absolute context positions [start, start+n).

    Returns bf16 bits [S, n, H].  Row r's values depend only on (seed, r), so any
    chunking of the stream yields the same rows.
    """
    if n <= 0:
        return np.zeros((cfg.n_target_layers, 0, cfg.hidden), np.uint16)
    b0, b1 = start // _ROW_BLOCK, (start + n - 1) // _ROW_BLOCK
    with ThreadPoolExecutor(max_workers=8) as ex:
        blocks = list(ex.map(lambda b: _hidden_block(cfg, b, seed), range(b0, b1 + 1)))
    cat = np.concatenate(blocks, axis=1)
    off = start - b0 * _ROW_BLOCK
    return np.ascontiguousarray(cat[:, off:off + n])


def append_sizes(count: int, seed: int = 2, lo: int = 1, hi: int = 16) -> np.ndarray:
    """Per-step accepted-token append sizes, uniform on {lo..hi}."""
    rng = np.random.Generator(np.random.PCG64(seed))
    return rng.integers(lo, hi + 1, size=count).astype(np.int32)


def block_ids(cfg: ModelConfig, step: int = 0, seed: int = 3) -> np.ndarray:
    """Block token ids [B] int32: x_t then the mask id (V-1) at B-1 positions.

    The tiny workload draws all B ids uniformly instead.
    """
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, step])))
    if cfg.random_block:
        return rng.integers(0, cfg.vocab, size=cfg.block_size).astype(np.int32)
    ids = np.full(cfg.block_size, cfg.vocab - 1, np.int32)
    ids[0] = rng.integers(0, cfg.vocab - 1)
    return ids


# Batched serving workload: n_seq sequences of the Qwen3-8B-shaped draft drafted together,
# ragged context lengths, each sequence appending U{1..16} accepted rows per step.
BATCHED = {"model": "qwen3_8b", "n_seq": 32, "lo": 512, "hi": 4096}


def batched_lengths(n_seq: int = 32, lo: int = 512, hi: int = 4096, seed: int = 4) -> np.ndarray:
    """Context length of each sequence of the batched workload, uniform on {lo..hi}."""
    rng = np.random.Generator(np.random.PCG64(seed))
    return rng.integers(lo, hi + 1, size=n_seq).astype(np.int32)
