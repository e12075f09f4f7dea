"""GPU parity at the workloads' full sizes, in the launch configuration bench.py times.

For each model shape (Qwen3-8B, Qwen3-4B and GPT-OSS-20B shaped drafts at their full
context lengths) the library and the fp64 oracle prefill the same seeded context in
512-row appends, then run draft steps.  Checked against the oracle: the whole
context K/V cache of every draft layer, the block rows after every layer, the logits
and the draft tokens (the bar of tests/parity.py).  The bench's configuration -- a
non-default stream, the draft block as one persistent launch whose phases wait at grid
barriers -- must produce the very same tokens, bitwise, as the debug run with one
launch per phase, and the kernel built for the shape's GEMM plans the very same logits
and rows as the generic kernel.
"""
import os

import numpy as np
import pytest
import torch

from paper_2606_02091_amd import dflare as dfl
from paper_2606_02091_amd import synth
import parity as P

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover - CPU container
    pytest.skip("needs a GPU", allow_module_level=True)

NAMES = os.environ.get("DFLARE_FULLSIZE", "qwen3_8b,qwen3_4b,gpt_oss_20b").split(",")


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", NAMES)
def test_fullsize_parity(name):
    cfg = synth.CONFIGS[name]
    L = cfg.context
    print(f"[fullsize] {name}: generating weights", flush=True)
    w, lg = P.weights_for(cfg)
    side = torch.cuda.Stream()
    with torch.cuda.stream(side):
        model = dfl.DraftModel(cfg, w, lg, max_context=L + 64, max_new=512)
        orc = P.oracle_for(cfg, w, lg, L + 64)
        for s in range(0, L, 512):
            n = min(512, L - s)
            rows = synth.hidden_rows(cfg, s, n)
            model.fuse_append(dfl.bf16_tensor(rows))
            orc.append(rows)
        print(f"[fullsize] {name}: context {L} appended", flush=True)
        side.synchronize()
        for i in range(cfg.n_draft_layers):
            for what, ref in ((dfl.DBG_KCACHE, orc.k_cache[i]), (dfl.DBG_VCACHE, orc.v_cache[i])):
                got = dfl.dflare_debug_read(model.h, what, i, (L, cfg.n_kv_heads, cfg.head_dim))
                e = P.relinf(got, ref)
                assert e <= P.REL_TOL, (name, i, what, e)
        ids = synth.block_ids(cfg, step=0)
        ids_t = torch.from_numpy(ids).cuda()
        out = torch.empty(cfg.block_size, dtype=torch.int32, device="cuda")
        for step in range(2):
            # bench configuration first: persistent launch on the side stream, no debug capture
            model.draft_block(ids_t, out)
            model.draft_block(ids_t, out)
            side.synchronize()
            assert dfl.dflare_kernel_stats(model.h)[0] == 1
            persistent_tokens = out.cpu().numpy().copy()
            dfl.dflare_debug_capture(model.h, True)
            # the timed launch configuration writing its own logits and block rows
            dfl.dflare_set_option(model.h, dfl.OPT_CAPTURE_PERSISTENT, 1)
            model.draft_block(ids_t, out)
            side.synchronize()
            assert dfl.dflare_kernel_stats(model.h)[0] == 1
            assert np.array_equal(out.cpu().numpy(), persistent_tokens)
            p_logits = dfl.dflare_debug_read(model.h, dfl.DBG_LOGITS, 0, (cfg.block_size, cfg.vocab))
            p_hidden = [dfl.dflare_debug_read(model.h, dfl.DBG_HIDDEN, i, (cfg.block_size, cfg.hidden))
                        for i in range(cfg.n_draft_layers)]
            # these shapes' plans on 256 CUs have a kernel built for them; the generic kernel
            # (plans read at run time) gives the same logits and rows bitwise
            stats = dfl.dflare_kernel_stats(model.h)
            if stats[2] == 256:
                assert stats[5] != 0, (name, stats)
            dfl.dflare_set_option(model.h, dfl.OPT_GENERIC_KERNEL, 1)
            assert dfl.dflare_kernel_stats(model.h)[5] == 0
            model.draft_block(ids_t, out)
            side.synchronize()
            dfl.dflare_set_option(model.h, dfl.OPT_GENERIC_KERNEL, 0)
            assert np.array_equal(out.cpu().numpy(), persistent_tokens), (name, step, "generic kernel")
            assert np.array_equal(p_logits, dfl.dflare_debug_read(model.h, dfl.DBG_LOGITS, 0,
                                                                  (cfg.block_size, cfg.vocab))), (name, step)
            for i in range(cfg.n_draft_layers):
                g = dfl.dflare_debug_read(model.h, dfl.DBG_HIDDEN, i, (cfg.block_size, cfg.hidden))
                assert np.array_equal(p_hidden[i], g), (name, step, "generic kernel", i)
            dfl.dflare_set_option(model.h, dfl.OPT_CAPTURE_PERSISTENT, 0)
            eager = model.draft_block(ids_t).cpu().numpy()
            side.synchronize()
            dfl.dflare_debug_capture(model.h, False)
            assert np.array_equal(persistent_tokens, eager)
            ref = orc.draft_block(ids)
            print(f"[fullsize] {name}: step {step} oracle done", flush=True)
            e = P.relinf(p_logits, ref["logits"])
            assert e <= P.REL_TOL, (name, step, "persistent logits", e)
            for i in range(cfg.n_draft_layers):
                assert P.relinf(p_hidden[i], ref["hidden"][i]) <= P.REL_TOL, (name, step, "persistent", i)
            # the per-phase launches of the debug run give the same numbers bitwise
            assert np.array_equal(p_logits, dfl.dflare_debug_read(model.h, dfl.DBG_LOGITS, 0,
                                                                  (cfg.block_size, cfg.vocab)))
            for i in range(cfg.n_draft_layers):
                g = dfl.dflare_debug_read(model.h, dfl.DBG_HIDDEN, i, (cfg.block_size, cfg.hidden))
                e = P.relinf(g, ref["hidden"][i])
                assert e <= P.REL_TOL, (name, step, i, e)
            zl = dfl.dflare_debug_read(model.h, dfl.DBG_LOGITS, 0, (cfg.block_size, cfg.vocab))
            e = P.relinf(zl, ref["logits"])
            assert e <= P.REL_TOL, (name, step, "logits", e)
            stats = P.check_tokens(eager, ref["logits"])
            print(f"[fullsize] {name}: step {step} logits rel err {e:.2e} tokens {stats}", flush=True)
            # next step: append accepted rows, as in the bench's draft loop
            n = int(synth.append_sizes(1, seed=10 + step)[0])
            rows = synth.hidden_rows(cfg, L + 100 * step, n, seed=4)
            model.fuse_append(dfl.bf16_tensor(rows))
            orc.append(rows)
            ids = synth.block_ids(cfg, step=step + 1)
            ids_t = torch.from_numpy(ids).cuda()
        model.close()


@pytest.mark.timeout(900)
def test_fullsize_batched():
    """The batched workload at full size: 32 Qwen3-8B-shaped sequences with ragged contexts
    (L ~ U{512..4096}), prefilled and drafted as bench.py --config batched does.  The oracle
    checks the shortest sequence (its whole cache, logits and tokens); every sequence is
    checked against drafting it alone (n_seq = 1), to the agreement bound of the batched
    parity tests; debug capture must not change any token."""
    spec = synth.BATCHED
    cfg = synth.CONFIGS[spec["model"]]
    n_seq = spec["n_seq"]
    lengths = [int(x) for x in synth.batched_lengths(n_seq, spec["lo"], spec["hi"])]
    B, V = cfg.block_size, cfg.vocab
    print(f"[fullsize] batched: generating weights", flush=True)
    w, lg = P.weights_for(cfg)
    side = torch.cuda.Stream()
    with torch.cuda.stream(side):
        model = dfl.DraftModel(cfg, w, lg, max_context=max(lengths) + 16, max_new=16 * n_seq, max_batch=n_seq)
        base = [16 * i for i in range(n_seq)]
        rows_dev = dfl.bf16_tensor(synth.hidden_rows(cfg, 0, max(b + L for b, L in zip(base, lengths))))
        for i, L in enumerate(lengths):
            for s0 in range(0, L, 512):
                n = min(512, L - s0)
                model.fuse_append_batched([i], [n], rows_dev[:, base[i] + s0:base[i] + s0 + n].contiguous())
        side.synchronize()
        print(f"[fullsize] batched: {n_seq} contexts appended", flush=True)
        seqs = list(range(n_seq))
        ids = np.stack([synth.block_ids(cfg, step=0, seed=200 + i) for i in seqs])
        ids_t = torch.from_numpy(ids).cuda()
        out = model.draft_block_batched(seqs, ids_t)
        side.synchronize()
        plain = out.cpu().numpy().copy()
        dfl.dflare_debug_capture(model.h, True)
        dbg = model.draft_block_batched(seqs, ids_t).cpu().numpy()
        side.synchronize()
        assert np.array_equal(plain, dbg)
        logits = dfl.dflare_debug_read(model.h, dfl.DBG_BLOGITS, 0, (n_seq, B, V))
        for i in seqs:
            one = model.draft_block_batched([i], ids_t[i:i + 1]).cpu().numpy()[0]
            z = dfl.dflare_debug_read(model.h, dfl.DBG_BLOGITS, 0, (1, B, V))[0]
            assert P.relinf(z, logits[i]) <= 5e-3, i
            P.check_tokens(one, logits[i])
        print(f"[fullsize] batched: every sequence agrees with drafting it alone", flush=True)
        j = int(np.argmin(lengths))
        orc = P.oracle_for(cfg, w, lg, lengths[j] + 64)
        orc.append(synth.hidden_rows(cfg, base[j], lengths[j]))
        for i in range(cfg.n_draft_layers):
            for what, ref in ((dfl.DBG_KCACHE, orc.k_cache[i]), (dfl.DBG_VCACHE, orc.v_cache[i])):
                got = dfl.dflare_debug_read_seq(model.h, what, j, i, (lengths[j], cfg.n_kv_heads, cfg.head_dim))
                assert P.relinf(got, ref) <= P.REL_TOL, (i, what)
        ref = orc.draft_block(ids[j])
        e = P.relinf(logits[j], ref["logits"])
        assert e <= P.REL_TOL, e
        stats = P.check_tokens(dbg[j], ref["logits"])
        print(f"[fullsize] batched: sequence {j} (L {lengths[j]}) logits rel err {e:.2e} tokens {stats}",
              flush=True)
        model.close()
