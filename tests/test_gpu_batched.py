"""GPU parity of the batched draft step: several sequences, each with its own context
cache and length, appended to and drafted together through the batched C-ABI calls,
against one fp64 oracle per sequence on the same seeded inputs (the bar of
tests/parity.py).

Sizes finish in seconds on the oracle yet span several 128-row GEMM groups, ragged
row counts (B = 5 gives sequences that straddle 16-row tiles), empty and one-row
contexts, contexts on and off the 64-key block and 512-key range grids of the
attention, 64 and 128 query rows per KV head, vocabularies that are not a multiple of
16, slots listed out of order and calls on subsets of the slots.

Besides the oracle bar, two batched results are compared directly: the same sequence
drafted by batched calls of other shapes (other rows, other K splits), and by the
batch-1 path.  The batched GEMMs take fp16 operands, rounded to 2^-11 relative; which
way each rounding falls depends on the order of the fp32 sums before it (the K split),
and the draft layers carry such differences forward, so a batched result sits about
2.5e-3 of the logit range from the exact one at full size (1e-3 on the small cases
here) and any two of them, or one and the batch-1 path's, agree within AGREE_TOL =
5e-3, a quarter of the oracle bar.
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

AGREE_TOL = 5e-3

CASES = {
    # name: (config, context length per listed slot, slots, max_batch)
    "hd128_b16": (synth.ModelConfig("bhd128", hidden=256, n_q_heads=4, n_kv_heads=1, head_dim=128, ffn=512,
                                    vocab=4001, n_draft_layers=2, n_target_layers=8, block_size=16, context=300),
                  [0, 1, 40, 128, 129, 200, 300, 77, 255], [3, 0, 7, 1, 9, 4, 11, 2, 5], 12),
    "hd64_gqa_b5": (synth.ModelConfig("bhd64", hidden=96, n_q_heads=6, n_kv_heads=2, head_dim=64, ffn=160,
                                      vocab=1000, n_draft_layers=3, n_target_layers=5, block_size=5, context=130,
                                      random_block=True),
                    [33, 0, 130, 7, 64], [1, 4, 0, 2, 3], 5),
    # 8 query heads per KV head (128 query rows per work item) and contexts spanning
    # several 512-key attention ranges, one of them ending a single key into a range
    "hd128_gqa8_long": (synth.ModelConfig("bgqa8", hidden=128, n_q_heads=8, n_kv_heads=1, head_dim=128,
                                          ffn=256, vocab=700, n_draft_layers=2, n_target_layers=3,
                                          block_size=16, context=1030),
                        [497, 1030, 0, 700, 511], [2, 0, 4, 1, 3], 5),
    "hd64_gqa8_long": (synth.ModelConfig("bgqa8h64", hidden=128, n_q_heads=16, n_kv_heads=2, head_dim=64,
                                         ffn=256, vocab=900, n_draft_layers=2, n_target_layers=3,
                                         block_size=16, context=1100),
                       [1100, 496, 40], [1, 0, 2], 3),
}


def dev(bits):
    return dfl.bf16_tensor(bits)


def ids_tensor(ids):
    return torch.from_numpy(np.ascontiguousarray(np.asarray(ids, np.int32))).cuda()


def slot_rows(cfg, slot, start, n):
    return synth.hidden_rows(cfg, start, n, seed=100 + slot)


def slot_ids(cfg, slot, step=0):
    return synth.block_ids(cfg, step=step, seed=200 + slot)


def build_batched(cfg, lengths, slots, max_batch, seed=5):
    """Fill every slot's context with batched appends of 1..16 rows per listed sequence,
    in rounds where the order of the sequences changes and some sequences sit out."""
    w, lg = P.weights_for(cfg)
    maxc = max(lengths) + 64
    model = dfl.DraftModel(cfg, w, lg, max_context=maxc, max_new=16 * max_batch, max_batch=max_batch)
    dfl.dflare_debug_capture(model.h, True)
    orcs = {s: P.oracle_for(cfg, w, lg, maxc) for s in slots}
    target = dict(zip(slots, lengths))
    filled = {s: 0 for s in slots}
    rng = np.random.default_rng(seed)
    last = None
    while any(filled[s] < target[s] for s in slots):
        seq, nn, parts, fused = [], [], [], []
        for s in rng.permutation(slots):
            s = int(s)
            left = target[s] - filled[s]
            if left <= 0 or rng.random() < 0.3:
                continue
            n = int(min(left, rng.integers(1, 17)))
            rows = slot_rows(cfg, s, filled[s], n)
            seq.append(s)
            nn.append(n)
            parts.append(rows)
            fused.append(orcs[s].append(rows))
            filled[s] += n
        if seq:
            model.fuse_append_batched(seq, nn, dev(np.concatenate(parts, axis=1)))
            last = np.concatenate(fused, axis=1)
    torch.cuda.synchronize()
    return model, orcs, last


def compare_draft(model, orcs, cfg, seq, step=0):
    B, V = cfg.block_size, cfg.vocab
    ids = np.stack([slot_ids(cfg, s, step) for s in seq])
    out = model.draft_block_batched(seq, ids_tensor(ids))
    torch.cuda.synchronize()
    tokens = out.cpu().numpy()
    logits = dfl.dflare_debug_read(model.h, dfl.DBG_BLOGITS, 0, (len(seq), B, V))
    worst = 0.0
    for i, s in enumerate(seq):
        ref = orcs[s].draft_block(ids[i])
        e = P.relinf(logits[i], ref["logits"])
        assert e <= P.REL_TOL, (s, e)
        P.check_tokens(tokens[i], ref["logits"])
        worst = max(worst, e)
    return tokens, logits, worst


@pytest.mark.parametrize("name", list(CASES))
def test_batched_matches_oracles(name):
    cfg, lengths, slots, max_batch = CASES[name]
    print(f"[batched] {name}: slots {slots} lengths {lengths}", flush=True)
    model, orcs, last_fused = build_batched(cfg, lengths, slots, max_batch)
    for s, L in zip(slots, lengths):
        assert dfl.dflare_context_len_seq(model.h, s) == L
    # fused rows of the last batched append (all of its rows, in call order)
    for i in range(cfg.n_draft_layers):
        got = dfl.dflare_debug_read(model.h, dfl.DBG_FUSED, i, (last_fused.shape[1], cfg.hidden))
        assert P.relinf(got, last_fused[i]) <= P.REL_TOL
    # every slot's cache
    for s, L in zip(slots, lengths):
        for i in range(cfg.n_draft_layers):
            for what, ref in ((dfl.DBG_KCACHE, orcs[s].k_cache[i]), (dfl.DBG_VCACHE, orcs[s].v_cache[i])):
                got = dfl.dflare_debug_read_seq(model.h, what, s, i, (L, cfg.n_kv_heads, cfg.head_dim))
                assert P.relinf(got, ref) <= P.REL_TOL, (s, i, what)
    # all slots, in the listed order
    tokens, logits, worst = compare_draft(model, orcs, cfg, slots)
    print(f"[batched] {name}: {len(slots)} sequences, logits rel err {worst:.2e}", flush=True)
    # a subset in another order gives the same rows
    sub = slots[::-2]
    t2, l2, _ = compare_draft(model, orcs, cfg, sub)
    for j, s in enumerate(sub):
        i = slots.index(s)
        assert P.relinf(l2[j], logits[i]) <= AGREE_TOL
    model.close()


def test_batched_single_equals_batch1():
    """Slot 0 through the batch-1 calls, slot 1 through the batched calls, same rows."""
    cfg = CASES["hd128_b16"][0]
    w, lg = P.weights_for(cfg)
    L = 190
    model = dfl.DraftModel(cfg, w, lg, max_context=L + 64, max_new=16, max_batch=2)
    dfl.dflare_debug_capture(model.h, True)
    orc = P.oracle_for(cfg, w, lg, L + 64)
    s = 0
    for n in synth.append_sizes(40, seed=6):
        n = int(min(n, L - s))
        if n <= 0:
            break
        rows = slot_rows(cfg, 0, s, n)
        model.fuse_append(dev(rows))
        model.fuse_append_batched([1], [n], dev(rows))
        orc.append(rows)
        s += n
    torch.cuda.synchronize()
    assert model.context_len == L and dfl.dflare_context_len_seq(model.h, 1) == L
    for i in range(cfg.n_draft_layers):
        for what in (dfl.DBG_KCACHE, dfl.DBG_VCACHE):
            a = dfl.dflare_debug_read_seq(model.h, what, 0, i, (L, cfg.n_kv_heads, cfg.head_dim))
            b = dfl.dflare_debug_read_seq(model.h, what, 1, i, (L, cfg.n_kv_heads, cfg.head_dim))
            assert P.relinf(b, a) <= AGREE_TOL, (i, what)
    for step in range(2):
        ids = slot_ids(cfg, 0, step)
        t1 = model.draft_block(ids_tensor(ids)).cpu().numpy()
        z1 = dfl.dflare_debug_read(model.h, dfl.DBG_LOGITS, 0, (cfg.block_size, cfg.vocab))
        tb = model.draft_block_batched([1], ids_tensor(ids[None])).cpu().numpy()[0]
        zb = dfl.dflare_debug_read(model.h, dfl.DBG_BLOGITS, 0, (1, cfg.block_size, cfg.vocab))[0]
        ref = orc.draft_block(ids)
        assert P.relinf(zb, ref["logits"]) <= P.REL_TOL
        assert P.relinf(zb, z1) <= AGREE_TOL
        P.check_tokens(t1, ref["logits"])
        P.check_tokens(tb, ref["logits"])
        # the batched call on slot 0 reads the batch-1 context
        t0 = model.draft_block_batched([0], ids_tensor(ids[None])).cpu().numpy()[0]
        z0 = dfl.dflare_debug_read(model.h, dfl.DBG_BLOGITS, 0, (1, cfg.block_size, cfg.vocab))[0]
        assert P.relinf(z0, z1) <= AGREE_TOL
        assert P.relinf(z0, zb) <= AGREE_TOL
        P.check_tokens(t0, ref["logits"])
    model.close()


def test_batched_truncate_and_validation():
    cfg = CASES["hd64_gqa_b5"][0]
    w, lg = P.weights_for(cfg)
    model = dfl.DraftModel(cfg, w, lg, max_context=24, max_new=20, max_batch=3)
    dfl.dflare_debug_capture(model.h, True)
    orcs = {s: P.oracle_for(cfg, w, lg, 24) for s in range(3)}
    rows = {s: slot_rows(cfg, s, 0, 30) for s in range(3)}
    model.fuse_append_batched([2, 0], [10, 6], dev(np.concatenate([rows[2][:, :10], rows[0][:, :6]], axis=1)))
    orcs[2].append(rows[2][:, :10])
    orcs[0].append(rows[0][:, :6])
    h = model.h

    def err(fn, *a):
        with pytest.raises(dfl.DFlareError) as e:
            fn(*a)
        return e.value.status

    x = dev(rows[1][:, :4])
    assert err(dfl.dflare_fuse_append_batched, h, [1, 1], [2, 2], x) == dfl.ERR_INVALID_ARG   # repeated slot
    assert err(dfl.dflare_fuse_append_batched, h, [3], [4], x) == dfl.ERR_INVALID_ARG         # slot out of range
    assert err(dfl.dflare_fuse_append_batched, h, [1], [0], x) == dfl.ERR_INVALID_ARG         # empty append
    big = dev(np.concatenate([rows[1][:, :15], rows[0][:, :6]], axis=1))
    assert err(dfl.dflare_fuse_append_batched, h, [1, 0], [15, 6], big) == dfl.ERR_INVALID_ARG  # sum > max_new
    full = dev(np.concatenate([rows[1][:, :4], rows[2][:, :16]], axis=1))
    assert err(dfl.dflare_fuse_append_batched, h, [1, 2], [4, 16], full) == dfl.ERR_CONTEXT_FULL
    ids = ids_tensor(np.zeros((2, cfg.block_size)))
    assert err(dfl.dflare_draft_block_batched, h, [0, 0], ids, ids) == dfl.ERR_INVALID_ARG
    assert err(dfl.dflare_truncate_seq, h, 2, 11) == dfl.ERR_INVALID_ARG
    # failed calls changed nothing
    assert [dfl.dflare_context_len_seq(h, s) for s in range(3)] == [6, 0, 10]
    # truncate one slot, append to it again, draft all three (slot 1 empty)
    dfl.dflare_truncate_seq(h, 2, 7)
    orcs[2].truncate(7)
    model.fuse_append_batched([2], [3], dev(rows[1][:, 20:23]))
    orcs[2].append(rows[1][:, 20:23])
    assert [dfl.dflare_context_len_seq(h, s) for s in range(3)] == [6, 0, 10]
    assert model.context_len == 6
    compare_draft(model, orcs, cfg, [1, 2, 0])
    model.close()
