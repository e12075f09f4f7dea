"""GPU parity: the HIP draft step against the fp64 oracle on the same seeded inputs.

Sizes here finish in seconds on the oracle yet span several MFMA tiles, several
attention chunks and ragged tails (vocab not a multiple of 16, block sizes below
16, context lengths off the chunk grid, appends of 1..16 rows and of several
16-row tiles).  Every call goes through the C ABI.
"""
import numpy as np
import pytest
import torch

from paper_2606_02091_amd import dflare as dfl
from paper_2606_02091_amd import synth
import parity as P

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover - CPU container
    pytest.skip("needs a GPU", allow_module_level=True)

CASES = {
    # name: (config, context length, append sizes: 'chunk' uses cfg.append_chunk)
    "tiny": (synth.CONFIGS["tiny"], 64, "chunk"),
    "ragged": (synth.ModelConfig("ragged", hidden=96, n_q_heads=6, n_kv_heads=2, head_dim=64, ffn=160,
                                 vocab=1000, n_draft_layers=3, n_target_layers=5, block_size=5, context=77,
                                 random_block=True), 77, "random"),
    "gqa8_hd64": (synth.ModelConfig("gqa8", hidden=128, n_q_heads=16, n_kv_heads=2, head_dim=64, ffn=128,
                                    vocab=2048, n_draft_layers=2, n_target_layers=4, block_size=16,
                                    context=300), 300, "random"),
    "hd128": (synth.ModelConfig("hd128", hidden=256, n_q_heads=4, n_kv_heads=1, head_dim=128, ffn=512,
                                vocab=4096, n_draft_layers=2, n_target_layers=8, block_size=16,
                                context=520), 520, "random"),
}


def dev(bits):
    return dfl.bf16_tensor(bits)


def ids_tensor(ids):
    return torch.from_numpy(np.asarray(ids, np.int32)).cuda()


def append_plan(cfg, L, mode, seed=2):
    if mode == "chunk":
        return [cfg.append_chunk] * (L // cfg.append_chunk) + ([L % cfg.append_chunk] if L % cfg.append_chunk else [])
    sizes, s = [], 0
    for n in synth.append_sizes(L, seed=seed):
        n = int(min(n, L - s))
        if n <= 0:
            break
        sizes.append(n)
        s += n
    return sizes


def build_pair(cfg, L, mode, max_new=16, debug=True):
    w, lg = P.weights_for(cfg)
    model = dfl.DraftModel(cfg, w, lg, max_context=L + 64, max_new=max_new)
    if debug:
        dfl.dflare_debug_capture(model.h, True)
    orc = P.oracle_for(cfg, w, lg, L + 64)
    s = 0
    for n in append_plan(cfg, L, mode):
        rows = synth.hidden_rows(cfg, s, n)
        model.fuse_append(dev(rows))
        orc.append(rows)
        s += n
    torch.cuda.synchronize()
    return model, orc, w, lg


def compare_step(model, orc, cfg, ids, tag=""):
    out = model.draft_block(ids_tensor(ids))
    torch.cuda.synchronize()
    ref = orc.draft_block(ids)
    H, B, V = cfg.hidden, cfg.block_size, cfg.vocab
    errs = {}
    for i in range(cfg.n_draft_layers):
        g = dfl.dflare_debug_read(model.h, dfl.DBG_HIDDEN, i, (B, H))
        errs[f"hidden{i}"] = P.relinf(g, ref["hidden"][i])
    lg = dfl.dflare_debug_read(model.h, dfl.DBG_LOGITS, 0, (B, V))
    errs["logits"] = P.relinf(lg, ref["logits"])
    for k, e in errs.items():
        assert e <= P.REL_TOL, f"{tag} {k}: rel err {e:.3g}"
    P.check_tokens(out.cpu().numpy(), ref["logits"])
    return errs, out.cpu().numpy(), ref


@pytest.mark.parametrize("case", sorted(CASES))
def test_parity_append_and_block(case):
    cfg, L, mode = CASES[case]
    print(f"[parity] case={case} L={L}", flush=True)
    model, orc, w, lg = build_pair(cfg, L, mode)
    # cached fusion weights
    a = dfl.dflare_debug_read(model.h, dfl.DBG_ALPHA, 0, (cfg.n_draft_layers, cfg.n_target_layers))
    assert np.all(np.abs(a.sum(axis=1) - 1.0) <= cfg.n_target_layers * 2.0 ** -23)
    assert P.relinf(a, orc.alpha) <= 1e-6
    # fused rows of the last append and the whole context cache
    n_last = orc.last_fused.shape[1]
    for i in range(cfg.n_draft_layers):
        f = dfl.dflare_debug_read(model.h, dfl.DBG_FUSED, i, (n_last, cfg.hidden))
        assert P.relinf(f, orc.last_fused[i]) <= P.REL_TOL
        k = dfl.dflare_debug_read(model.h, dfl.DBG_KCACHE, i, (L, cfg.n_kv_heads, cfg.head_dim))
        v = dfl.dflare_debug_read(model.h, dfl.DBG_VCACHE, i, (L, cfg.n_kv_heads, cfg.head_dim))
        ek, ev = P.relinf(k, orc.k_cache[i]), P.relinf(v, orc.v_cache[i])
        assert ek <= P.REL_TOL and ev <= P.REL_TOL, (i, ek, ev)
    # two draft steps with an append in between
    errs, _, _ = compare_step(model, orc, cfg, synth.block_ids(cfg, step=0), case)
    print(f"[parity] {case} step0 max rel err {max(errs.values()):.3g}", flush=True)
    n = 7
    rows = synth.hidden_rows(cfg, L, n)
    model.fuse_append(dev(rows))
    orc.append(rows)
    errs, _, _ = compare_step(model, orc, cfg, synth.block_ids(cfg, step=1), case)
    assert model.context_len == L + n
    model.close()


def test_empty_context():
    cfg = CASES["ragged"][0]
    w, lg = P.weights_for(cfg)
    model = dfl.DraftModel(cfg, w, lg, max_context=32)
    dfl.dflare_debug_capture(model.h, True)
    orc = P.oracle_for(cfg, w, lg, 32)
    compare_step(model, orc, cfg, synth.block_ids(cfg, step=5), "empty")
    model.close()


def test_multi_tile_append_and_truncate():
    cfg = CASES["gqa8_hd64"][0]
    w, lg = P.weights_for(cfg)
    model = dfl.DraftModel(cfg, w, lg, max_context=256, max_new=64)
    dfl.dflare_debug_capture(model.h, True)
    orc = P.oracle_for(cfg, w, lg, 256)
    rows = synth.hidden_rows(cfg, 0, 50)        # 4 row tiles, the last one ragged
    model.fuse_append(dev(rows))
    orc.append(rows)
    model.truncate(41)
    orc.truncate(41)
    rows = synth.hidden_rows(cfg, 1000, 13, seed=5)
    model.fuse_append(dev(rows))
    orc.append(rows)
    for i in range(cfg.n_draft_layers):
        k = dfl.dflare_debug_read(model.h, dfl.DBG_KCACHE, i, (54, cfg.n_kv_heads, cfg.head_dim))
        assert P.relinf(k, orc.k_cache[i]) <= P.REL_TOL
    compare_step(model, orc, cfg, synth.block_ids(cfg, step=2), "truncate")
    model.close()


def test_incremental_append_is_bitwise_bulk():
    cfg = CASES["hd128"][0]
    w, lg = P.weights_for(cfg)
    rows = synth.hidden_rows(cfg, 0, 64)
    bulk = dfl.DraftModel(cfg, w, lg, max_context=128, max_new=64)
    inc = dfl.DraftModel(cfg, w, lg, max_context=128, max_new=64)
    for m in (bulk, inc):
        dfl.dflare_debug_capture(m.h, True)
    bulk.fuse_append(dev(rows))
    s = 0
    for n in [8] * 4 + list(synth.append_sizes(10, seed=11)):
        n = min(int(n), 64 - s)
        if n <= 0:
            break
        inc.fuse_append(dev(np.ascontiguousarray(rows[:, s:s + n])))
        s += n
    assert s == 64
    for i in range(cfg.n_draft_layers):
        for what in (dfl.DBG_KCACHE, dfl.DBG_VCACHE):
            a = dfl.dflare_debug_read(bulk.h, what, i, (64, cfg.n_kv_heads, cfg.head_dim))
            b = dfl.dflare_debug_read(inc.h, what, i, (64, cfg.n_kv_heads, cfg.head_dim))
            assert np.array_equal(a, b)
    ids = ids_tensor(synth.block_ids(cfg))
    ta, tb = bulk.draft_block(ids), inc.draft_block(ids)
    la = dfl.dflare_debug_read(bulk.h, dfl.DBG_LOGITS, 0, (cfg.block_size, cfg.vocab))
    lb = dfl.dflare_debug_read(inc.h, dfl.DBG_LOGITS, 0, (cfg.block_size, cfg.vocab))
    assert np.array_equal(la, lb) and torch.equal(ta, tb)
    bulk.close()
    inc.close()


def test_repeat_is_deterministic_and_cache_untouched():
    cfg = CASES["gqa8_hd64"][0]
    model, orc, _, _ = build_pair(cfg, 300, "random")
    ids = ids_tensor(synth.block_ids(cfg, step=3))
    k0 = dfl.dflare_debug_read(model.h, dfl.DBG_KCACHE, 1, (300, cfg.n_kv_heads, cfg.head_dim))
    outs, logits = [], []
    for _ in range(3):
        outs.append(model.draft_block(ids).cpu())
        logits.append(dfl.dflare_debug_read(model.h, dfl.DBG_LOGITS, 0, (cfg.block_size, cfg.vocab)))
    assert all(torch.equal(outs[0], o) for o in outs[1:])
    assert all(np.array_equal(logits[0], l) for l in logits[1:])
    k1 = dfl.dflare_debug_read(model.h, dfl.DBG_KCACHE, 1, (300, cfg.n_kv_heads, cfg.head_dim))
    assert np.array_equal(k0, k1)
    assert model.context_len == 300
    model.close()


def test_joint_permutation_with_explicit_positions():
    cfg = CASES["gqa8_hd64"][0]
    model, orc, _, _ = build_pair(cfg, 300, "random")
    B, V = cfg.block_size, cfg.vocab
    ids = np.random.default_rng(4).integers(0, V, size=B).astype(np.int32)
    pos = np.arange(300, 300 + B, dtype=np.int32)
    out = torch.empty(B, dtype=torch.int32, device="cuda")
    dfl.dflare_draft_block_pos(model.h, ids_tensor(ids), pos, out)
    base_logits = dfl.dflare_debug_read(model.h, dfl.DBG_LOGITS, 0, (B, V))
    base_tok = out.cpu().numpy()
    ref = orc.draft_block(ids, positions=pos)
    assert P.relinf(base_logits, ref["logits"]) <= P.REL_TOL
    perm = np.random.default_rng(5).permutation(B)
    dfl.dflare_draft_block_pos(model.h, ids_tensor(ids[perm]), pos[perm], out)
    lg = dfl.dflare_debug_read(model.h, dfl.DBG_LOGITS, 0, (B, V))
    assert P.relinf(lg, base_logits[perm]) <= 1e-4
    P.check_tokens(out.cpu().numpy(), ref["logits"][perm])
    # the permuted call's tokens are the base call's, permuted, wherever the oracle's top-1
    # to top-2 margin leaves no near tie
    zp = ref["logits"][perm]
    top2 = np.sort(zp, axis=1)[:, -2:]
    clear = (top2[:, 1] - top2[:, 0]) > P.MARGIN
    assert clear.any()
    assert np.array_equal(out.cpu().numpy()[clear], base_tok[perm][clear])
    model.close()


def test_one_hot_fusion_matches_single_layer_model():
    cfg = CASES["ragged"][0]
    w, _ = P.weights_for(cfg)
    D, S = cfg.n_draft_layers, cfg.n_target_layers
    pick = [4, 0, 2]
    lg = np.full((D, S), -1e4, np.float32)
    for i, j in enumerate(pick):
        lg[i, j] = 0.0
    model = dfl.DraftModel(cfg, w, lg, max_context=64)
    dfl.dflare_debug_capture(model.h, True)
    rows = synth.hidden_rows(cfg, 0, 12)
    model.fuse_append(dev(rows))
    a = dfl.dflare_debug_read(model.h, dfl.DBG_ALPHA, 0, (D, S))
    assert np.array_equal(a, (lg == 0).astype(np.float32))
    for i, j in enumerate(pick):
        c1 = cfg.replace(n_draft_layers=1, n_target_layers=1)
        w1 = {k: (v[i:i + 1] if k in ("fuse_norm", "attn_norm", "mlp_norm", "wq", "wk_d", "wv_d", "wk_t",
                                      "wv_t", "wo", "w_gate", "w_up", "w_down") else v) for k, v in w.items()}
        single = dfl.DraftModel(c1, w1, np.zeros((1, 1), np.float32), max_context=64)
        single.fuse_append(dev(np.ascontiguousarray(rows[j:j + 1])))
        for what in (dfl.DBG_KCACHE, dfl.DBG_VCACHE):
            x = dfl.dflare_debug_read(model.h, what, i, (12, cfg.n_kv_heads, cfg.head_dim))
            y = dfl.dflare_debug_read(single.h, what, 0, (12, cfg.n_kv_heads, cfg.head_dim))
            assert np.array_equal(x, y), (i, what)
        single.close()
    model.close()


def test_context_full_and_bad_sizes_leave_state():
    cfg = CASES["tiny"][0]
    w, lg = P.weights_for(cfg)
    model = dfl.DraftModel(cfg, w, lg, max_context=20, max_new=16)
    dfl.dflare_debug_capture(model.h, True)
    rows = synth.hidden_rows(cfg, 0, 16)
    model.fuse_append(dev(rows))
    k0 = dfl.dflare_debug_read(model.h, dfl.DBG_KCACHE, 0, (16, cfg.n_kv_heads, cfg.head_dim))
    with pytest.raises(dfl.DFlareError) as ei:
        model.fuse_append(dev(synth.hidden_rows(cfg, 16, 5)))
    assert ei.value.status == dfl.ERR_CONTEXT_FULL
    with pytest.raises(dfl.DFlareError) as ei:
        dfl.dflare_fuse_append(model.h, dev(synth.hidden_rows(cfg, 16, 2)), 17)
    assert ei.value.status == dfl.ERR_INVALID_ARG
    with pytest.raises(dfl.DFlareError):
        dfl.dflare_truncate(model.h, 17)
    assert model.context_len == 16
    k1 = dfl.dflare_debug_read(model.h, dfl.DBG_KCACHE, 0, (16, cfg.n_kv_heads, cfg.head_dim))
    assert np.array_equal(k0, k1)
    model.close()


@pytest.mark.parametrize("case", sorted(CASES))
def test_persistent_matches_per_phase(case):
    """The persistent launch (phases separated by grid barriers, non-default stream) gives
    the very tokens of one launch per phase, bitwise, step after step, with eager work
    (appends, truncation, synchronisation) between the calls; both agree with the oracle."""
    cfg, L, mode = CASES[case]
    print(f"[persistent] case={case}", flush=True)
    w, lg = P.weights_for(cfg)
    side = torch.cuda.Stream()
    with torch.cuda.stream(side):
        model = dfl.DraftModel(cfg, w, lg, max_context=L + 64, max_new=16)
        n_blocks = dfl.dflare_kernel_stats(model.h)[2]
        orc = P.oracle_for(cfg, w, lg, L + 64)
        s = 0
        for n in append_plan(cfg, L, mode):
            rows = synth.hidden_rows(cfg, s, n)
            model.fuse_append(dev(rows))
            orc.append(rows)
            s += n
        out = torch.empty(cfg.block_size, dtype=torch.int32, device="cuda")
        for k in range(3):
            ids_np = synth.block_ids(cfg, step=k)
            ids = ids_tensor(ids_np)
            dfl.dflare_set_option(model.h, dfl.OPT_PERSISTENT, 1)
            assert dfl.dflare_kernel_stats(model.h)[0] == 1
            model.draft_block(ids, out)
            model.draft_block(ids, out)  # repeated: the block slots are rewritten, the context is not
            side.synchronize()
            persistent = out.cpu().numpy().copy()
            # the same kernel through the cooperative launch
            dfl.dflare_set_option(model.h, dfl.OPT_COOPERATIVE, 1)
            model.draft_block(ids, out)
            side.synchronize()
            dfl.dflare_set_option(model.h, dfl.OPT_COOPERATIVE, 0)
            assert np.array_equal(out.cpu().numpy(), persistent), (case, k)
            # the persistent launch again, writing its own logits and block rows
            dfl.dflare_debug_capture(model.h, True)
            dfl.dflare_set_option(model.h, dfl.OPT_CAPTURE_PERSISTENT, 1)
            cap = model.draft_block(ids).cpu().numpy()
            assert dfl.dflare_kernel_stats(model.h)[0] == 1
            p_logits = dfl.dflare_debug_read(model.h, dfl.DBG_LOGITS, 0, (cfg.block_size, cfg.vocab))
            p_hidden = [dfl.dflare_debug_read(model.h, dfl.DBG_HIDDEN, i, (cfg.block_size, cfg.hidden))
                        for i in range(cfg.n_draft_layers)]
            dfl.dflare_set_option(model.h, dfl.OPT_CAPTURE_PERSISTENT, 0)
            dfl.dflare_set_option(model.h, dfl.OPT_PERSISTENT, 0)
            per_phase = model.draft_block(ids).cpu().numpy()
            side.synchronize()
            s_logits = dfl.dflare_debug_read(model.h, dfl.DBG_LOGITS, 0, (cfg.block_size, cfg.vocab))
            dfl.dflare_debug_capture(model.h, False)
            assert np.array_equal(persistent, per_phase), (case, k, persistent, per_phase)
            assert np.array_equal(cap, persistent), (case, k)
            assert np.array_equal(p_logits, s_logits), (case, k)
            ref = orc.draft_block(ids_np)
            P.check_tokens(persistent, ref["logits"])
            assert P.relinf(p_logits, ref["logits"]) <= P.REL_TOL, (case, k)
            for i in range(cfg.n_draft_layers):
                assert P.relinf(p_hidden[i], ref["hidden"][i]) <= P.REL_TOL, (case, k, i)
            extra = synth.hidden_rows(cfg, s, 3, seed=9 + k)  # eager work between the calls
            model.fuse_append(dev(extra))
            orc.append(extra)
            s += 3
    assert n_blocks >= 16
    model.close()


SPLIT_CFG = synth.ModelConfig("splits", hidden=256, n_q_heads=4, n_kv_heads=2, head_dim=128, ffn=640,
                              vocab=8000, n_draft_layers=2, n_target_layers=6, block_size=16, context=300,
                              random_block=True)


# GEMM plans (chunk width tn, K split kg) per phase kind for SPLIT_CFG on 16 work-groups:
# QKV 64 x 8 tiles, O 16 x 16, gate/up 80 x 8, down 16 x 20, LM head 500 x 8 (n x k).
PLANS = {
    "chunks2": {"QKV": "2,1", "O": "2,1", "GU": "2,1", "DOWN": "2,1"},   # several chunks per work-group
    "chunks8": {"QKV": "8,1", "O": "8,1", "GU": "8,1", "DOWN": "8,1"},   # padding tiles in every chunk
    "split": {"QKV": "8,2", "O": "8,8", "GU": "6,1", "DOWN": "4,4"},     # K split over 2, 8, 4 work-groups
    "split_thin": {"QKV": "4,1", "O": "4,4", "GU": "4,1", "DOWN": "8,8"},  # K parts of 2-3 tiles: idle waves
}


@pytest.mark.parametrize("plan", sorted(PLANS))
def test_gemm_plans(plan, monkeypatch):
    """Every way a GEMM phase can lay out its work: 16 work-groups, so each owns many output
    tiles; chunks of 2 to 8 tiles with padding; K split over 2 to 8 work-groups, including
    parts so thin that some waves hold no k-tile; the LM head in many chunks.  Per-phase
    launches match the oracle; the persistent launch matches them bitwise."""
    cfg = SPLIT_CFG
    print(f"[plans] {plan}", flush=True)
    monkeypatch.setenv("DFLARE_BLOCKS", "16")
    for name, v in PLANS[plan].items():
        monkeypatch.setenv(f"DFLARE_PLAN_{name}", v)
    model, orc, w, lg = build_pair(cfg, cfg.context, "random")
    assert dfl.dflare_kernel_stats(model.h)[2] == 16
    for k in range(2):
        ids = synth.block_ids(cfg, step=k)
        _, per_phase, _ = compare_step(model, orc, cfg, ids, tag=f"plan={plan} step={k}")
        dfl.dflare_debug_capture(model.h, False)
        persistent = model.draft_block(ids_tensor(ids)).cpu().numpy()
        torch.cuda.synchronize()
        dfl.dflare_debug_capture(model.h, True)
        assert np.array_equal(persistent, per_phase), (plan, k)
    model.close()


def test_many_attention_items_per_work_group(monkeypatch):
    """16 work-groups and a 3,000-row context: 24 chunks x 2 KV heads = 48 attention items,
    three per work-group (only the first is staged ahead; the others load everything after
    the barrier), and the merge of 24 chunks by 8 work-groups per KV head.  Per-phase
    launches match the oracle; the persistent launch matches them bitwise."""
    cfg = SPLIT_CFG.replace(context=3000)
    monkeypatch.setenv("DFLARE_BLOCKS", "16")
    model, orc, w, lg = build_pair(cfg, cfg.context, "random", max_new=16)
    for k in range(2):
        ids = synth.block_ids(cfg, step=k)
        _, per_phase, _ = compare_step(model, orc, cfg, ids, tag=f"items step={k}")
        dfl.dflare_debug_capture(model.h, False)
        persistent = model.draft_block(ids_tensor(ids)).cpu().numpy()
        torch.cuda.synchronize()
        dfl.dflare_debug_capture(model.h, True)
        assert np.array_equal(persistent, per_phase), k
    model.close()


def test_large_magnitude_cache():
    """The fp16 context cache at large magnitudes: fusion-norm gains scaled by 2000 give
    context keys and values in the thousands (fp16 keeps its relative precision there); the
    cache, the block rows and the logits stay within the bar of the fp64 oracle, and the
    timed (persistent) launch gives the same tokens.  Values beyond +-65504 would saturate
    (the cache format's range; not reached here)."""
    cfg = CASES["hd128"][0]
    L = 200
    w, lg = P.weights_for(cfg)
    g = synth.bf16_to_f32(w["fuse_norm"]) * 2000.0
    w["fuse_norm"] = synth.round_bf16(g)
    model = dfl.DraftModel(cfg, w, lg, max_context=L + 64, max_new=16)
    dfl.dflare_debug_capture(model.h, True)
    orc = P.oracle_for(cfg, w, lg, L + 64)
    s = 0
    for n in append_plan(cfg, L, "random"):
        rows = synth.hidden_rows(cfg, s, n)
        model.fuse_append(dev(rows))
        orc.append(rows)
        s += n
    kmax = 0.0
    for i in range(cfg.n_draft_layers):
        k = dfl.dflare_debug_read(model.h, dfl.DBG_KCACHE, i, (L, cfg.n_kv_heads, cfg.head_dim))
        v = dfl.dflare_debug_read(model.h, dfl.DBG_VCACHE, i, (L, cfg.n_kv_heads, cfg.head_dim))
        assert P.relinf(k, orc.k_cache[i]) <= P.REL_TOL and P.relinf(v, orc.v_cache[i]) <= P.REL_TOL, i
        kmax = max(kmax, float(np.abs(orc.k_cache[i]).max()), float(np.abs(orc.v_cache[i]).max()))
    assert 1000.0 < kmax < 65504.0, kmax
    ids = synth.block_ids(cfg, step=0)
    _, per_phase, _ = compare_step(model, orc, cfg, ids, tag="large")
    dfl.dflare_debug_capture(model.h, False)
    persistent = model.draft_block(ids_tensor(ids)).cpu().numpy()
    torch.cuda.synchronize()
    assert np.array_equal(persistent, per_phase)
    model.close()
