"""The C-ABI library loads, exports every symbol its header declares, and rejects
bad arguments before touching the GPU (these paths make no HIP call)."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2606_02091_amd import dflare as dfl
from paper_2606_02091_amd import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dflare.h")


def header_symbols():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(dflare_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(dfl.LIB_PATH):
        pytest.fail("libdflare.so is not built (run __graft_entry__.build())")
    return dfl.lib()


def test_header_declares_the_binding_names():
    assert header_symbols() == sorted(dfl.EXPORTED)


def test_library_exports_every_declared_symbol(L):
    for name in header_symbols():
        assert hasattr(L, name), name


def test_status_strings(L):
    for code in (0, -1, -2, -3, -4, -5):
        assert L.dflare_status_str(code)
    assert L.dflare_status_str(-99) == b"unknown status"


def _cfg(**kw):
    c = dfl.make_config(synth.CONFIGS["tiny"], max_context=64, max_new=16)
    for k, v in kw.items():
        setattr(c, k, v)
    return c


def _init(cfg, logits=None, weights=True, drop=()):
    w = dfl.dflare_weights(**{k: (0x1000 if weights and k not in drop else None) for k in dfl.WEIGHT_FIELDS})
    lg = np.zeros((cfg.n_draft_layers, cfg.n_target_layers), np.float32) if logits is None else logits
    lg = np.ascontiguousarray(lg, np.float32)
    h = ctypes.c_void_p()
    rc = dfl.lib().dflare_init(ctypes.byref(cfg), ctypes.byref(w),
                               lg.ctypes.data_as(ctypes.POINTER(ctypes.c_float)), None, ctypes.byref(h))
    return rc, h.value


@pytest.mark.parametrize("field,value,code", [
    ("hidden", 0, dfl.ERR_INVALID_ARG),
    ("n_kv_heads", 3, dfl.ERR_INVALID_ARG),
    ("block_size", 17, dfl.ERR_UNSUPPORTED),
    ("head_dim", 96, dfl.ERR_UNSUPPORTED),
    ("hidden", 264, dfl.ERR_UNSUPPORTED),
    ("max_new", 0, dfl.ERR_INVALID_ARG),
    ("rope_base", 0.0, dfl.ERR_INVALID_ARG),
    ("max_batch", 65, dfl.ERR_UNSUPPORTED),
    ("max_batch", -1, dfl.ERR_UNSUPPORTED),
])
def test_init_rejects_bad_config(L, field, value, code):
    rc, h = _init(_cfg(**{field: value}))
    assert rc == code and not h
    assert L.dflare_last_error(None)


def test_init_rejects_bad_fusion_logits(L):
    cfg = _cfg()
    for bad in (np.nan, np.inf):
        lg = np.zeros((cfg.n_draft_layers, cfg.n_target_layers), np.float32)
        lg[1, 2] = bad
        rc, h = _init(cfg, lg)
        assert rc == dfl.ERR_INVALID_ARG and not h
    lg = np.full((cfg.n_draft_layers, cfg.n_target_layers), -np.inf, np.float32)
    assert _init(cfg, lg)[0] == dfl.ERR_INVALID_ARG


@pytest.mark.parametrize("variant", [16, dfl.VARIANT_DFLASH | dfl.VARIANT_NO_SOFTMAX,
                                     dfl.VARIANT_DFLASH | dfl.VARIANT_SHARED_KV, -1])
def test_init_rejects_bad_variant(L, variant):
    rc, h = _init(_cfg(variant=variant))
    assert rc == dfl.ERR_INVALID_ARG and not h


def test_init_rejects_variants_without_their_weights(L):
    # +FC needs post_fc, DFlash needs fc (checked before any device work)
    for variant, field in ((dfl.VARIANT_POST_FC, "post_fc"), (dfl.VARIANT_DFLASH, "fc")):
        rc, h = _init(_cfg(variant=variant), drop=(field,))
        assert rc == dfl.ERR_INVALID_ARG and not h
        assert b"needs" in L.dflare_last_error(None)
    # -Softmax takes W^fuse as the weights: every entry must be finite
    cfg = _cfg(variant=dfl.VARIANT_NO_SOFTMAX)
    for bad in (np.nan, np.inf, -np.inf):
        lg = np.zeros((cfg.n_draft_layers, cfg.n_target_layers), np.float32)
        lg[0, 1] = bad
        rc, h = _init(cfg, lg)
        assert rc == dfl.ERR_INVALID_ARG and not h


def test_init_rejects_missing_weights(L):
    rc, h = _init(_cfg(), weights=False)
    assert rc == dfl.ERR_INVALID_ARG and not h


def test_calls_on_invalid_handles(L):
    out = ctypes.c_int32()
    assert L.dflare_context_len(None, ctypes.byref(out)) == dfl.ERR_INVALID_ARG
    assert L.dflare_destroy(None) == dfl.ERR_INVALID_ARG
    assert L.dflare_truncate(0x1234, 0) == dfl.ERR_INVALID_ARG
    assert L.dflare_fuse_append(0x1234, 0x1000, 1) == dfl.ERR_INVALID_ARG
    assert L.dflare_draft_block(None, 0x1000, 0x1000) == dfl.ERR_INVALID_ARG
    seq = (ctypes.c_int32 * 1)(0)
    assert L.dflare_fuse_append_batched(0x1234, 1, seq, seq, 0x1000) == dfl.ERR_INVALID_ARG
    assert L.dflare_draft_block_batched(None, 1, seq, 0x1000, 0x1000) == dfl.ERR_INVALID_ARG
    assert L.dflare_truncate_seq(0x1234, 0, 0) == dfl.ERR_INVALID_ARG
    assert L.dflare_accept(None, 0x1000, 0x1000, 0x1000, 0x1000, 0x1000, 0x1000, None) == dfl.ERR_INVALID_ARG
    assert L.dflare_context_len_seq(None, 0, ctypes.byref(out)) == dfl.ERR_INVALID_ARG
    buf = (ctypes.c_float * 4)()
    assert L.dflare_debug_read_seq(None, dfl.DBG_KCACHE, 0, 0, buf, 4) == dfl.ERR_INVALID_ARG


# ---- training-side entry points: shape and argument checks (no HIP call is made) ----

def test_anchor_attention_workspace_sizes(L):
    ws = L.dflare_anchor_attention_workspace
    ok = ws(4, 16, 100, 8, 2, 128)
    assert ok > 0
    assert ws(4, 16, 200, 8, 2, 128) > ok          # more context keys, more workspace
    assert ws(4, 16, 0, 8, 2, 128) > 0             # no context at all is a valid call
    for bad in [(0, 16, 100, 8, 2, 128),            # no block
                (4, 17, 100, 8, 2, 128),            # B above 16
                (4, 0, 100, 8, 2, 128),
                (4, 16, -1, 8, 2, 128),
                (4, 16, 100, 9, 2, 128),            # query heads not a multiple of KV heads
                (4, 16, 100, 8, 2, 96),             # head size other than 64 or 128
                (4, 16, 100, 18, 2, 128)]:          # 9 query heads per group x 16 rows > 128
        assert ws(*bad) == 0, bad


def test_anchor_attention_rejects_bad_arguments(L):
    p = ctypes.c_void_p(0x1000)  # never dereferenced: every case fails its checks first
    f = ctypes.cast(0x1000, ctypes.POINTER(ctypes.c_float))
    i32 = ctypes.cast(0x1000, ctypes.POINTER(ctypes.c_int32))
    need = L.dflare_anchor_attention_workspace(4, 16, 100, 8, 2, 128)
    fwd = L.dflare_anchor_attention_fwd
    assert fwd(p, p, p, p, p, i32, 4, 16, 100, 8, 2, 96, f, f, p, need, None) == dfl.ERR_UNSUPPORTED
    assert fwd(p, p, p, p, p, i32, 4, 17, 100, 8, 2, 128, f, f, p, need, None) == dfl.ERR_INVALID_ARG
    assert fwd(None, p, p, p, p, i32, 4, 16, 100, 8, 2, 128, f, f, p, need, None) == dfl.ERR_INVALID_ARG
    assert fwd(p, None, p, p, p, i32, 4, 16, 100, 8, 2, 128, f, f, p, need, None) == dfl.ERR_INVALID_ARG
    assert fwd(p, p, p, p, p, i32, 4, 16, 100, 8, 2, 128, f, f, p, need - 1, None) == dfl.ERR_INVALID_ARG
    bwd = L.dflare_anchor_attention_bwd
    assert bwd(p, p, p, p, p, i32, 4, 16, 100, 8, 2, 128, f, f, None, f, f, f, f, f, p, need, None) \
        == dfl.ERR_INVALID_ARG                    # no output gradient
    assert bwd(p, p, p, p, p, i32, 4, 16, 100, 8, 2, 128, f, f, f, f, f, f, f, f, p, need - 1, None) \
        == dfl.ERR_INVALID_ARG
    assert bwd(p, p, p, p, p, i32, 4, 16, 100, 8, 2, 64, f, f, f, f, None, f, f, f, p, need, None) \
        == dfl.ERR_INVALID_ARG                    # context keys (T > 0) without their gradient


def test_weighted_ce_rejects_bad_arguments(L):
    p = ctypes.c_void_p(0x1000)
    f = ctypes.cast(0x1000, ctypes.POINTER(ctypes.c_float))
    i32 = ctypes.cast(0x1000, ctypes.POINTER(ctypes.c_int32))
    need = L.dflare_weighted_ce_workspace(64)
    assert need >= 3 * 64 * 4
    ce = L.dflare_weighted_ce
    assert ce(f, i32, 64, 1000, 16, 4.5, f, f, f, p, need - 1, None) == dfl.ERR_INVALID_ARG
    assert ce(f, i32, 60, 1000, 16, 4.5, f, f, f, p, need, None) == dfl.ERR_INVALID_ARG  # rows % B
    for gamma in (0.0, -1.0, float("nan"), float("inf")):
        assert ce(f, i32, 64, 1000, 16, gamma, f, f, f, p, need, None) == dfl.ERR_INVALID_ARG
    assert ce(None, i32, 64, 1000, 16, 4.5, f, f, f, p, need, None) == dfl.ERR_INVALID_ARG
    assert ce(f, i32, 64, 0, 16, 4.5, f, f, f, p, need, None) == dfl.ERR_INVALID_ARG


def test_weighted_ce_noalloc_rejects_bad_arguments(L):
    """Argument checks of the allocation-free CE come before any HIP call."""
    f = ctypes.cast(0x1000, ctypes.POINTER(ctypes.c_float))
    i32 = ctypes.cast(0x1000, ctypes.POINTER(ctypes.c_int32))
    ce = L.dflare_weighted_ce_noalloc
    big = dfl.WEIGHTED_CE_NOALLOC_MAX_ROWS + 16
    assert ce(f, i32, big, 1000, 16, 4.5, f, f, f, None) == dfl.ERR_INVALID_ARG  # beyond the scratch
    assert ce(f, i32, 60, 1000, 16, 4.5, f, f, f, None) == dfl.ERR_INVALID_ARG   # rows % B
    for gamma in (0.0, -1.0, float("nan"), float("inf")):
        assert ce(f, i32, 64, 1000, 16, gamma, f, f, f, None) == dfl.ERR_INVALID_ARG
    assert ce(None, i32, 64, 1000, 16, 4.5, f, f, f, None) == dfl.ERR_INVALID_ARG
    assert ce(f, i32, 64, 1000, 16, 4.5, f, f, None, None) == dfl.ERR_INVALID_ARG
