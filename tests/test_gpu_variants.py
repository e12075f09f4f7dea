"""GPU parity of the model variants: the ablations of Sec. 6.3 (Table 2: -Softmax, -KVProj,
+FC) and the DFlash baseline of Sec. 3.1-3.2 (Eq. 1-2), each against the fp64 oracle of
the same variant on the same seeded inputs, to the bar of tests/parity.py.

Checked after appends of 1..16 rows (batch-1 calls) and after batched appends of several
sequences: every layer's context K/V cache, the fused rows (the shared context rows for
DFlash; for +FC the rows before the folded layer), the logits and the draft tokens of a
draft step.  +FC runs with the layer folded into the context projection at init
(W' = W W_pfc rounded to bf16, b' = W b_pfc in fp32); DFlash runs its append on fp16
matrix-core operands, as the batched path does.
"""
import numpy as np
import pytest
import torch

from oracle import dflare_oracle as orc
from paper_2606_02091_amd import dflare as dfl
from paper_2606_02091_amd import synth
import parity as P
import test_gpu_batched as TB
import test_gpu_parity as TP

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover - CPU container
    pytest.skip("needs a GPU", allow_module_level=True)

VARIANTS = {
    "no_softmax": dfl.VARIANT_NO_SOFTMAX,
    "shared_kv": dfl.VARIANT_SHARED_KV,
    "post_fc": dfl.VARIANT_POST_FC,
    "post_fc_shared_kv": dfl.VARIANT_POST_FC | dfl.VARIANT_SHARED_KV,
    "dflash": dfl.VARIANT_DFLASH,
}
CFGS = {
    "hd128": (TP.CASES["hd128"][0], 300),
    "gqa_hd64": (synth.ModelConfig("vgqa", hidden=192, n_q_heads=6, n_kv_heads=2, head_dim=64, ffn=256,
                                   vocab=1500, n_draft_layers=3, n_target_layers=5, block_size=7,
                                   context=150, random_block=True), 150),
}


def weights(cfg):
    w = synth.make_weights(cfg, kinds=synth.WEIGHT_KINDS)
    return w, w.pop("fusion_logits")


def check_fused(model, cfg, variant, ref_fused, n, seq=None):
    layers = 1 if variant & dfl.VARIANT_DFLASH else cfg.n_draft_layers
    for i in range(layers):
        got = dfl.dflare_debug_read(model.h, dfl.DBG_FUSED, i, (n, cfg.hidden))
        assert P.relinf(got, ref_fused[i]) <= P.REL_TOL, ("fused", i)


def pre_fc_rows(orc_model, w, hid_bits, cfg):
    """fused rows before the +FC layer (what the library's debug capture holds)"""
    return orc.fuse_rows(orc_model.alpha, orc.bf16_to_f64(hid_bits), orc.bf16_to_f64(w["fuse_norm"]), cfg.rms_eps)


@pytest.mark.parametrize("cfg_name", sorted(CFGS))
@pytest.mark.parametrize("vname", list(VARIANTS))
def test_variant_batch1(vname, cfg_name):
    variant = VARIANTS[vname]
    cfg, L = CFGS[cfg_name]
    print(f"[variant] {vname} {cfg_name} batch-1", flush=True)
    w, lg = weights(cfg)
    if variant & dfl.VARIANT_NO_SOFTMAX:
        lg = (0.5 * lg).astype(np.float32)  # raw weights of either sign
    dl = None if variant & dfl.VARIANT_DFLASH else lg
    model = dfl.DraftModel(cfg, w, dl, max_context=L + 64, max_new=16, variant=variant)
    dfl.dflare_debug_capture(model.h, True)
    o = orc.DraftOracle(cfg, w, dl, max_context=L + 64, variant=variant)
    s = 0
    for n in TP.append_plan(cfg, L, "random"):
        rows = synth.hidden_rows(cfg, s, n)
        model.fuse_append(dfl.bf16_tensor(rows))
        f = o.append(rows)
        s += n
    torch.cuda.synchronize()
    ref = pre_fc_rows(o, w, rows, cfg) if variant & dfl.VARIANT_POST_FC else f
    check_fused(model, cfg, variant, ref, rows.shape[1])
    for i in range(cfg.n_draft_layers):
        for what, r in ((dfl.DBG_KCACHE, o.k_cache[i]), (dfl.DBG_VCACHE, o.v_cache[i])):
            got = dfl.dflare_debug_read(model.h, what, i, (L, cfg.n_kv_heads, cfg.head_dim))
            e = P.relinf(got, r)
            assert e <= P.REL_TOL, (vname, i, what, e)
    errs, _, _ = TP.compare_step(model, o, cfg, synth.block_ids(cfg, step=0), vname)
    print(f"[variant] {vname} {cfg_name}: max rel err {max(errs.values()):.2e}", flush=True)
    model.close()


@pytest.mark.parametrize("vname", ["no_softmax", "post_fc_shared_kv", "dflash"])
def test_variant_batched(vname):
    variant = VARIANTS[vname]
    cfg, lengths, slots, max_batch = TB.CASES["hd64_gqa_b5"]
    print(f"[variant] {vname} batched", flush=True)
    w, lg = weights(cfg)
    dl = None if variant & dfl.VARIANT_DFLASH else lg
    maxc = max(lengths) + 64
    model = dfl.DraftModel(cfg, w, dl, max_context=maxc, max_new=16 * max_batch, max_batch=max_batch,
                           variant=variant)
    dfl.dflare_debug_capture(model.h, True)
    orcs = {s: orc.DraftOracle(cfg, w, dl, max_context=maxc, variant=variant) for s in slots}
    target = dict(zip(slots, lengths))
    filled = {s: 0 for s in slots}
    rng = np.random.default_rng(3)
    while any(filled[s] < target[s] for s in slots):
        seq, nn, parts = [], [], []
        for s in rng.permutation(slots):
            s = int(s)
            n = int(min(target[s] - filled[s], rng.integers(1, 17)))
            if n <= 0:
                continue
            rows = TB.slot_rows(cfg, s, filled[s], n)
            seq.append(s)
            nn.append(n)
            parts.append(rows)
            orcs[s].append(rows)
            filled[s] += n
        model.fuse_append_batched(seq, nn, dfl.bf16_tensor(np.concatenate(parts, axis=1)))
    torch.cuda.synchronize()
    for s, L in zip(slots, lengths):
        for i in range(cfg.n_draft_layers):
            for what, r in ((dfl.DBG_KCACHE, orcs[s].k_cache[i]), (dfl.DBG_VCACHE, orcs[s].v_cache[i])):
                got = dfl.dflare_debug_read_seq(model.h, what, s, i, (L, cfg.n_kv_heads, cfg.head_dim))
                assert P.relinf(got, r) <= P.REL_TOL, (vname, s, i, what)
    _, _, worst = TB.compare_draft(model, orcs, cfg, slots)
    print(f"[variant] {vname} batched: logits rel err {worst:.2e}", flush=True)
    model.close()
