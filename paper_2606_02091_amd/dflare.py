"""ctypes binding of libdflare.so (include/dflare.h).

Argument marshalling only: every step of the draft path runs in the library's HIP
kernels.  Tensors are PyTorch device tensors (PyTorch supplies device memory and
the current stream); bf16 data may be given as torch.bfloat16 or as 16-bit
integer tensors holding the bit patterns.  Loading fails loudly when the library
has not been built -- there is no fallback.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np
import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "_lib", "libdflare.so")

OK, ERR_INVALID_ARG, ERR_OUT_OF_MEMORY, ERR_CONTEXT_FULL, ERR_HIP, ERR_UNSUPPORTED = 0, -1, -2, -3, -4, -5
DBG_FUSED, DBG_KCACHE, DBG_VCACHE, DBG_HIDDEN, DBG_LOGITS, DBG_ALPHA, DBG_TRACE, DBG_BLOGITS = range(8)
OPT_PERSISTENT, OPT_TRACE, OPT_CAPTURE_PERSISTENT, OPT_COOPERATIVE, OPT_GENERIC_KERNEL = 1, 2, 3, 4, 5

EXPORTED = (
    "dflare_init", "dflare_fuse_append", "dflare_draft_block", "dflare_draft_block_pos",
    "dflare_truncate", "dflare_context_len", "dflare_set_stream", "dflare_destroy",
    "dflare_status_str", "dflare_last_error", "dflare_debug_capture", "dflare_debug_read",
    "dflare_kernel_stats", "dflare_profile_begin", "dflare_profile_end", "dflare_set_option",
    "dflare_fuse_append_batched", "dflare_draft_block_batched", "dflare_truncate_seq",
    "dflare_context_len_seq", "dflare_debug_read_seq", "dflare_set_sampling", "dflare_accept", "dflare_accept_async",
    "dflare_anchor_attention_workspace", "dflare_anchor_attention_fwd", "dflare_anchor_attention_bwd",
    "dflare_weighted_ce_workspace", "dflare_weighted_ce", "dflare_weighted_ce_noalloc", "dflare_read_probe",
)
K_QKV, K_ATTN, K_O, K_GATE_UP, K_DOWN, K_LM_HEAD, K_FUSE, K_KV_T, K_DRAFT = range(1, 10)
(K_B_QKV, K_B_ATTN, K_B_O, K_B_GATE_UP, K_B_DOWN, K_B_LM_HEAD, K_B_KV_T, K_B_EPI, K_B_FUSE, K_B_DRAFT,
 K_B_APPEND) = range(10, 21)


class DFlareError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{msg} (status {status})")
        self.status = status


class dflare_config(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "hidden", "n_q_heads", "n_kv_heads", "head_dim", "ffn", "vocab", "n_draft_layers",
        "n_target_layers", "block_size", "max_context", "max_new")] + [
        ("rope_base", ctypes.c_float), ("rms_eps", ctypes.c_float), ("max_batch", ctypes.c_int32),
        ("variant", ctypes.c_int32)]


# model variants (dflare_config.variant), as in include/dflare.h
VARIANT_NO_SOFTMAX, VARIANT_SHARED_KV, VARIANT_POST_FC, VARIANT_DFLASH = 1, 2, 4, 8


WEIGHT_FIELDS = ("embed", "lm_head", "final_norm", "fuse_norm", "attn_norm", "mlp_norm", "wq", "wk_d",
                 "wv_d", "wk_t", "wv_t", "wo", "w_gate", "w_up", "w_down", "post_fc", "post_fc_bias", "fc",
                 "fc_bias")


class dflare_weights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in WEIGHT_FIELDS]


_lib = None


def lib() -> ctypes.CDLL:
    """Load libdflare.so once; raise if it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built; run __graft_entry__.build() first")
    L = ctypes.CDLL(LIB_PATH)
    vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    sig = {
        "dflare_init": ([ctypes.POINTER(dflare_config), ctypes.POINTER(dflare_weights),
                         ctypes.POINTER(ctypes.c_float), vp, ctypes.POINTER(vp)], ctypes.c_int),
        "dflare_fuse_append": ([vp, vp, i32], ctypes.c_int),
        "dflare_draft_block": ([vp, vp, vp], ctypes.c_int),
        "dflare_draft_block_pos": ([vp, vp, ctypes.POINTER(i32), vp], ctypes.c_int),
        "dflare_truncate": ([vp, i32], ctypes.c_int),
        "dflare_context_len": ([vp, ctypes.POINTER(i32)], ctypes.c_int),
        "dflare_set_stream": ([vp, vp], ctypes.c_int),
        "dflare_destroy": ([vp], ctypes.c_int),
        "dflare_status_str": ([ctypes.c_int], ctypes.c_char_p),
        "dflare_last_error": ([vp], ctypes.c_char_p),
        "dflare_debug_capture": ([vp, ctypes.c_int], ctypes.c_int),
        "dflare_debug_read": ([vp, ctypes.c_int, ctypes.c_int, ctypes.POINTER(ctypes.c_float), i64],
                              ctypes.c_int),
        "dflare_kernel_stats": ([vp, ctypes.POINTER(i32), i32], ctypes.c_int),
        "dflare_profile_begin": ([vp, ctypes.c_int], ctypes.c_int),
        "dflare_profile_end": ([vp, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(i32)], ctypes.c_int),
        "dflare_set_option": ([vp, ctypes.c_int, ctypes.c_int], ctypes.c_int),
        "dflare_fuse_append_batched": ([vp, i32, ctypes.POINTER(i32), ctypes.POINTER(i32), vp], ctypes.c_int),
        "dflare_draft_block_batched": ([vp, i32, ctypes.POINTER(i32), vp, vp], ctypes.c_int),
        "dflare_truncate_seq": ([vp, i32, i32], ctypes.c_int),
        "dflare_set_sampling": ([vp, ctypes.c_float, ctypes.c_uint64], ctypes.c_int),
        "dflare_accept": ([vp, vp, vp, vp, vp, vp, vp, ctypes.POINTER(ctypes.c_int32)], ctypes.c_int),
        "dflare_accept_async": ([vp, vp, vp, vp, vp, vp, vp, vp], ctypes.c_int),
        "dflare_anchor_attention_workspace": ([ctypes.c_int32] * 6, ctypes.c_size_t),
        "dflare_anchor_attention_fwd": ([vp] * 6 + [ctypes.c_int32] * 6 + [vp, vp, vp, ctypes.c_size_t, vp],
                                        ctypes.c_int),
        "dflare_anchor_attention_bwd": ([vp] * 6 + [ctypes.c_int32] * 6 + [vp] * 9 + [ctypes.c_size_t, vp],
                                        ctypes.c_int),
        "dflare_weighted_ce_workspace": ([ctypes.c_int32], ctypes.c_size_t),
        "dflare_weighted_ce": ([vp, vp, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_float, vp, vp, vp,
                                vp, ctypes.c_size_t, vp], ctypes.c_int),
        "dflare_weighted_ce_noalloc": ([vp, vp, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_float, vp,
                                        vp, vp, vp], ctypes.c_int),
        "dflare_read_probe": ([vp, i64, vp, vp], ctypes.c_int),
        "dflare_context_len_seq": ([vp, i32, ctypes.POINTER(i32)], ctypes.c_int),
        "dflare_debug_read_seq": ([vp, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.POINTER(ctypes.c_float),
                                   i64], ctypes.c_int),
    }
    for name, (args, res) in sig.items():
        fn = getattr(L, name)
        fn.argtypes = args
        fn.restype = res
    _lib = L
    return L


def _check(rc: int, h=None):
    if rc != OK:
        msg = lib().dflare_last_error(h).decode() or lib().dflare_status_str(rc).decode()
        raise DFlareError(rc, msg)


def _ptr(t) -> int | None:
    if t is None:
        return None
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError("expected a device tensor")
    if not t.is_contiguous():
        raise ValueError("tensor must be contiguous")
    return t.data_ptr()


def _stream(stream) -> int:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def make_config(cfg, max_context: int, max_new: int = 16, max_batch: int = 1, variant: int = 0) -> dflare_config:
    """dflare_config from any object with the model attributes (hidden, n_q_heads, ...)."""
    return dflare_config(cfg.hidden, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, cfg.ffn, cfg.vocab,
                         cfg.n_draft_layers, cfg.n_target_layers, cfg.block_size, max_context, max_new,
                         cfg.rope_base, cfg.rms_eps, max_batch, variant)


def dflare_init(config: dflare_config, weights: dict, fusion_logits, stream=None) -> int:
    """Create a handle; weights maps field name -> device tensor (None for unit norm gains)."""
    w = dflare_weights(**{k: _ptr(weights.get(k)) for k in WEIGHT_FIELDS})
    lg_ptr = None
    if fusion_logits is not None:  # may be None for the DFlash variant
        lg = np.ascontiguousarray(np.asarray(fusion_logits, dtype=np.float32))
        lg_ptr = lg.ctypes.data_as(ctypes.POINTER(ctypes.c_float))
    h = ctypes.c_void_p()
    rc = lib().dflare_init(ctypes.byref(config), ctypes.byref(w), lg_ptr, _stream(stream), ctypes.byref(h))
    _check(rc, None)
    return h.value


def dflare_fuse_append(h: int, target_hidden: torch.Tensor, n_new: int | None = None) -> None:
    if n_new is None:
        n_new = target_hidden.shape[1]
    _check(lib().dflare_fuse_append(h, _ptr(target_hidden), int(n_new)), h)


def dflare_draft_block(h: int, block_ids: torch.Tensor, draft_tokens: torch.Tensor) -> None:
    _check(lib().dflare_draft_block(h, _ptr(block_ids), _ptr(draft_tokens)), h)


def dflare_draft_block_pos(h: int, block_ids: torch.Tensor, positions, draft_tokens: torch.Tensor) -> None:
    pos = np.ascontiguousarray(np.asarray(positions, dtype=np.int32))
    _check(lib().dflare_draft_block_pos(h, _ptr(block_ids), pos.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                                        _ptr(draft_tokens)), h)


def _i32_array(values) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(values, dtype=np.int32).reshape(-1))


def _i32p(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))


def dflare_fuse_append_batched(h: int, seq, n_new, target_hidden: torch.Tensor) -> None:
    """Append n_new[i] rows to slot seq[i]; target_hidden is [S, sum(n_new), H], sequence-major rows."""
    sq, nn = _i32_array(seq), _i32_array(n_new)
    if sq.size != nn.size:
        raise ValueError("seq and n_new differ in length")
    _check(lib().dflare_fuse_append_batched(h, sq.size, _i32p(sq), _i32p(nn), _ptr(target_hidden)), h)


def dflare_draft_block_batched(h: int, seq, block_ids: torch.Tensor, draft_tokens: torch.Tensor) -> None:
    """block_ids / draft_tokens: device int32 [n_seq, B]; row i belongs to slot seq[i]."""
    sq = _i32_array(seq)
    _check(lib().dflare_draft_block_batched(h, sq.size, _i32p(sq), _ptr(block_ids), _ptr(draft_tokens)), h)


def dflare_accept(h: int, block_ids: torch.Tensor, draft_tokens: torch.Tensor, target_tokens: torch.Tensor,
                  target_hidden: torch.Tensor, next_ids: torch.Tensor, emitted: torch.Tensor) -> int:
    """Verify a drafted block against the target's outputs; returns k (see include/dflare.h)."""
    k = ctypes.c_int32(-1)
    _check(lib().dflare_accept(h, _ptr(block_ids), _ptr(draft_tokens), _ptr(target_tokens), _ptr(target_hidden),
                               _ptr(next_ids), _ptr(emitted), ctypes.byref(k)), h)
    return k.value


def dflare_accept_async(h: int, block_ids: torch.Tensor, draft_tokens: torch.Tensor, target_tokens: torch.Tensor,
                        target_hidden: torch.Tensor, next_ids: torch.Tensor, emitted: torch.Tensor,
                        accepted: torch.Tensor | None = None) -> None:
    """As dflare_accept without the host wait: k goes to the device int32 `accepted` (if
    given) and the context length stays on the device (see include/dflare.h)."""
    _check(lib().dflare_accept_async(h, _ptr(block_ids), _ptr(draft_tokens), _ptr(target_tokens),
                                     _ptr(target_hidden), _ptr(next_ids), _ptr(emitted),
                                     _ptr(accepted) if accepted is not None else None), h)


# ---- training-side kernels (no handle) ----

def _train_check(rc: int, what: str) -> None:
    if rc != 0:
        raise DFlareError(rc, what)


def anchor_attention_fwd(q, k_ctx, v_ctx, k_blk, v_blk, anchors, B: int, stream=None):
    """Anchor attention forward (include/dflare.h).  q [n*B, n_q, hd], k/v_ctx [T, n_kv, hd],
    k/v_blk [n*B, n_kv, hd] as bf16-bit int16/uint16 device tensors, anchors int32 [n].
    Returns (out fp32 [n*B, n_q, hd], lse fp32 [n*B, n_q])."""
    M, n_q, hd = q.shape
    T, n_kv = k_ctx.shape[0], k_blk.shape[1]
    n = M // B
    ws_bytes = lib().dflare_anchor_attention_workspace(n, B, T, n_q, n_kv, hd)
    if ws_bytes == 0:
        raise DFlareError(-5, "unsupported anchor attention shape")
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=q.device)
    out = torch.empty((M, n_q, hd), dtype=torch.float32, device=q.device)
    lse = torch.empty((M, n_q), dtype=torch.float32, device=q.device)
    _train_check(lib().dflare_anchor_attention_fwd(
        _ptr(q), _ptr(k_ctx) if T else None, _ptr(v_ctx) if T else None, _ptr(k_blk), _ptr(v_blk), _ptr(anchors),
        n, B, T, n_q, n_kv, hd, _ptr(out), _ptr(lse), _ptr(ws), ws_bytes, _stream(stream)), "anchor attention fwd")
    return out, lse


def anchor_attention_bwd(q, k_ctx, v_ctx, k_blk, v_blk, anchors, B: int, out, lse, dout, stream=None):
    """Anchor attention backward: returns (dq, dk_ctx, dv_ctx, dk_blk, dv_blk), fp32."""
    M, n_q, hd = q.shape
    T, n_kv = k_ctx.shape[0], k_blk.shape[1]
    n = M // B
    ws_bytes = lib().dflare_anchor_attention_workspace(n, B, T, n_q, n_kv, hd)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=q.device)
    f = dict(dtype=torch.float32, device=q.device)
    dq = torch.empty((M, n_q, hd), **f)
    dkc, dvc = torch.empty((T, n_kv, hd), **f), torch.empty((T, n_kv, hd), **f)
    dkb, dvb = torch.empty((M, n_kv, hd), **f), torch.empty((M, n_kv, hd), **f)
    _train_check(lib().dflare_anchor_attention_bwd(
        _ptr(q), _ptr(k_ctx) if T else None, _ptr(v_ctx) if T else None, _ptr(k_blk), _ptr(v_blk), _ptr(anchors),
        n, B, T, n_q, n_kv, hd, _ptr(out), _ptr(lse), _ptr(dout), _ptr(dq), _ptr(dkc) if T else None,
        _ptr(dvc) if T else None, _ptr(dkb), _ptr(dvb), _ptr(ws), ws_bytes, _stream(stream)), "anchor attention bwd")
    return dq, dkc, dvc, dkb, dvb


def weighted_ce(logits, labels, B: int, gamma: float, stream=None):
    """Position-weighted cross-entropy: returns (loss fp32 [1], row_ce fp32 [rows], dlogits fp32 [rows, V])."""
    rows, V = logits.shape
    ws_bytes = lib().dflare_weighted_ce_workspace(rows)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=logits.device)
    loss = torch.empty(1, dtype=torch.float32, device=logits.device)
    ce = torch.empty(rows, dtype=torch.float32, device=logits.device)
    dz = torch.empty_like(logits)
    _train_check(lib().dflare_weighted_ce(_ptr(logits), _ptr(labels), rows, V, B, float(gamma), _ptr(loss), _ptr(ce),
                                          _ptr(dz), _ptr(ws), ws_bytes, _stream(stream)), "weighted ce")
    return loss, ce, dz


def read_probe(buf: torch.Tensor, sink: torch.Tensor, stream=None) -> None:
    """Measurement: one streaming read of the device tensor buf (the HBM read ceiling)."""
    _train_check(lib().dflare_read_probe(_ptr(buf), buf.numel() * buf.element_size(), _ptr(sink), _stream(stream)),
                 "read probe")


WEIGHTED_CE_NOALLOC_MAX_ROWS = 65536  # DFLARE_WEIGHTED_CE_NOALLOC_MAX_ROWS


def weighted_ce_noalloc(logits, labels, B: int, gamma: float, loss, row_ce, dlogits, stream=None):
    """The weighted CE through the allocation-free entry point: writes the caller's loss
    [1], row_ce [rows] and dlogits [rows, V] (fp32 device tensors); the library allocates
    nothing (its scratch is a fixed device array)."""
    rows, V = logits.shape
    _train_check(lib().dflare_weighted_ce_noalloc(_ptr(logits), _ptr(labels), rows, V, B, float(gamma), _ptr(loss),
                                                  _ptr(row_ce), _ptr(dlogits), _stream(stream)),
                 "weighted ce (no allocation)")


def dflare_set_sampling(h: int, temperature: float, seed: int = 0) -> None:
    """temperature 0: greedy argmax; > 0: Gumbel-max draws from softmax(z / temperature)."""
    _check(lib().dflare_set_sampling(h, float(temperature), int(seed) & 0xFFFFFFFFFFFFFFFF), h)


def dflare_truncate_seq(h: int, seq: int, new_len: int) -> None:
    _check(lib().dflare_truncate_seq(h, int(seq), int(new_len)), h)


def dflare_context_len_seq(h: int, seq: int) -> int:
    out = ctypes.c_int32()
    _check(lib().dflare_context_len_seq(h, int(seq), ctypes.byref(out)), h)
    return out.value


def dflare_debug_read_seq(h: int, what: int, seq: int, layer: int, shape) -> np.ndarray:
    out = np.empty(int(np.prod(shape)), dtype=np.float32)
    _check(lib().dflare_debug_read_seq(h, what, int(seq), layer,
                                       out.ctypes.data_as(ctypes.POINTER(ctypes.c_float)), out.size), h)
    return out.reshape(shape)


def dflare_truncate(h: int, new_len: int) -> None:
    _check(lib().dflare_truncate(h, int(new_len)), h)


def dflare_context_len(h: int) -> int:
    out = ctypes.c_int32()
    _check(lib().dflare_context_len(h, ctypes.byref(out)), h)
    return out.value


def dflare_set_stream(h: int, stream) -> None:
    _check(lib().dflare_set_stream(h, _stream(stream)), h)


def dflare_destroy(h: int) -> None:
    _check(lib().dflare_destroy(h), None)


def dflare_debug_capture(h: int, on: bool) -> None:
    _check(lib().dflare_debug_capture(h, int(bool(on))), h)


def dflare_debug_read(h: int, what: int, layer: int, shape) -> np.ndarray:
    out = np.empty(int(np.prod(shape)), dtype=np.float32)
    _check(lib().dflare_debug_read(h, what, layer, out.ctypes.data_as(ctypes.POINTER(ctypes.c_float)),
                                   out.size), h)
    return out.reshape(shape)


def dflare_kernel_stats(h: int) -> tuple[int, ...]:
    """(kernels per draft_block, kernels per fuse_append, work-groups, phases, grid barriers,
    plan signature of the draft-block kernel, 0 for the generic one)."""
    out = (ctypes.c_int32 * 6)()
    _check(lib().dflare_kernel_stats(h, out, 6), h)
    return tuple(out)


def dflare_set_option(h: int, option: int, value: int) -> None:
    _check(lib().dflare_set_option(h, int(option), int(value)), h)


def dflare_profile_begin(h: int, kind: int) -> None:
    _check(lib().dflare_profile_begin(h, int(kind)), h)


def dflare_profile_end(h: int) -> tuple[float, int]:
    """(summed kernel milliseconds, launches) since dflare_profile_begin."""
    ms, n = ctypes.c_double(), ctypes.c_int32()
    _check(lib().dflare_profile_end(h, ctypes.byref(ms), ctypes.byref(n)), h)
    return ms.value, n.value


def bf16_tensor(bits: np.ndarray, device="cuda") -> torch.Tensor:
    """bf16 bit patterns (uint16 numpy) -> torch.bfloat16 device tensor (same bits)."""
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16))
    return t.view(torch.bfloat16).to(device)


class DraftModel:
    """Owner of one handle: the three calls of the draft step plus helpers."""

    def __init__(self, cfg, weights_bits: dict, fusion_logits, max_context: int, max_new: int = 16,
                 device="cuda", stream=None, max_batch: int = 1, variant: int = 0):
        self.cfg = cfg
        self.config = make_config(cfg, max_context, max_new, max_batch, variant)
        dev = {k: (None if weights_bits.get(k) is None else bf16_tensor(weights_bits[k], device))
               for k in WEIGHT_FIELDS}
        self.h = dflare_init(self.config, dev, fusion_logits, stream)
        del dev  # the library keeps packed copies
        self.device = device

    def fuse_append(self, target_hidden: torch.Tensor) -> None:
        dflare_fuse_append(self.h, target_hidden)

    def draft_block(self, block_ids: torch.Tensor, out: torch.Tensor | None = None) -> torch.Tensor:
        if out is None:
            out = torch.empty(self.cfg.block_size, dtype=torch.int32, device=self.device)
        dflare_draft_block(self.h, block_ids, out)
        return out

    def truncate(self, n: int) -> None:
        dflare_truncate(self.h, n)

    def fuse_append_batched(self, seq, n_new, target_hidden: torch.Tensor) -> None:
        dflare_fuse_append_batched(self.h, seq, n_new, target_hidden)

    def draft_block_batched(self, seq, block_ids: torch.Tensor, out: torch.Tensor | None = None) -> torch.Tensor:
        if out is None:
            out = torch.empty(block_ids.shape, dtype=torch.int32, device=self.device)
        dflare_draft_block_batched(self.h, seq, block_ids, out)
        return out

    @property
    def context_len(self) -> int:
        return dflare_context_len(self.h)

    def close(self) -> None:
        if self.h:
            dflare_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:  # noqa: BLE001 - interpreter shutdown
            pass
