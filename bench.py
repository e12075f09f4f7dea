#!/usr/bin/env python3
"""Benchmark of the DFlare draft step on one MI355X.

One step = dflare_fuse_append(n_new ~ U{1..16} accepted target rows) followed by
dflare_draft_block(B = 16) at a fixed context length L: before each step the
context is truncated by n_new so that every step sees exactly L context rows.
Default workload: Qwen3-8B-shaped draft (H 4096, 32 q / 8 kv heads x 128,
SwiGLU 12288, vocab 151936, D = 8 draft layers fusing S = 36 target layers),
L = 4096, batch 1.  Weights and inputs are seeded synthetic data (no trained
weights exist here); all inputs are resident in HBM before the timed region.

The draft block runs as one persistent launch (its phases wait at grid barriers),
fuse_append as two kernels.  Prints one JSON line.  Per-kernel durations come from
hipEvents placed by the library around the launches of one kernel kind at a time (a
separate pass after the timed region, so the headline number carries no event
overhead); per-phase times come from the kernel's own wall-clock trace.
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "draft blocks/sec (B=16, Qwen3-8B shape, batch 1) + % HBM roofline"
SHAPE_NAMES = {"qwen3_8b": "Qwen3-8B", "qwen3_4b": "Qwen3-4B", "gpt_oss_20b": "GPT-OSS-20B"}


def shape_name(cfg):
    return SHAPE_NAMES.get(cfg.name, cfg.name)
HBM_PEAK_GBS = 8000.0


# --variant -> (library flags, extra weight kinds)
VARIANTS = {
    "dflare": (0, ()),
    "no_softmax": (1, ()),
    "shared_kv": (2, ()),
    "post_fc": (4, ("post_fc", "post_fc_bias")),
    "dflash": (8, ("fc", "fc_bias")),
}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--config", default="qwen3_8b",
                    help="qwen3_8b (default), qwen3_4b, gpt_oss_20b, or batched (32 ragged sequences)")
    ap.add_argument("--variant", default="dflare", choices=sorted(VARIANTS),
                    help="model variant: the method (dflare), the Sec. 6.3 ablations (no_softmax, "
                         "shared_kv, post_fc) or the DFlash FC fusion baseline (dflash)")
    ap.add_argument("--target-layers", type=int, default=0,
                    help="number S of fused target layers (default: the model's)")
    ap.add_argument("--temperature", type=float, default=0.0,
                    help="0 (default): greedy drafts; > 0: Gumbel-max draws from softmax(z / T)")
    ap.add_argument("--loop-sync", action="store_true",
                    help="with --loop: verify with dflare_accept, which waits for k every iteration")
    ap.add_argument("--loop", action="store_true",
                    help="time the draft-then-verify loop (draft_block, a synthetic target, accept) instead")
    ap.add_argument("--training", action="store_true",
                    help="time the training-side kernels (anchor attention fwd/bwd, weighted CE) instead")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-context", type=int, default=0,
                    help="context rows of the oracle's timed sample (default: the workload's own)")
    ap.add_argument("--profile-steps", type=int, default=20)
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a plain 1 GiB device copy (reference for HBM byte counters)")
    ap.add_argument("--summarize-counters", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="write profiles/hbm_counters_<config>.json from two rocprofv3 --pmc output folders")
    ap.add_argument("--counter-scale", default="2.0,1.0",
                    help="bytes per counted FETCH_SIZE and WRITE_SIZE byte (from --calibrate-copy)")
    args = ap.parse_args()
    if args.profile_steps < 1:
        ap.error("--profile-steps must be at least 1: the per-kernel table and the roofline are timed over them")
    return args


def calibrate_copy():
    """A plain device-to-device copy of known size: the byte counters of the profiler
    read against it give the scale from counter units to bytes."""
    import torch
    n = 1 << 30
    src = torch.empty(n, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    src.fill_(1)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"calibration": "device copy", "bytes_read": n, "bytes_written": n, "launches": 3}), flush=True)


def kernel_bytes(cfg, L, n_mean, variant="dflare"):
    """Algorithmic HBM bytes per launch of each kernel kind (bf16 storage; the DFlash
    append's "fuse" is the concatenation and the FC layer of Eq. 1, whose fp16 W_fc is read
    once per append)."""
    H, F, V, D, S = cfg.hidden, cfg.ffn, cfg.vocab, cfg.n_draft_layers, cfg.n_target_layers
    q, kv = cfg.q_dim, cfg.kv_dim
    fc = H * S * H * 2 if variant == "dflash" else 0
    return {
        "draft_block": cfg.block_bytes(L),    # every draft-layer weight, LM head, context K/V
        "qkv": (q + 2 * kv) * H * 2,          # W_Q, W_K^d, W_V^d of one layer
        "attn": 2 * L * kv * 2,               # context K and V of one layer
        "o": H * q * 2,
        "gate_up": 2 * F * H * 2,
        "down": H * F * 2,
        "lm_head": V * H * 2,
        "fuse": S * n_mean * H * 2 + fc,      # the target rows, read once (+ W_fc)
        "kv_t": D * 2 * kv * H * 2,           # W_K^t, W_V^t of all layers (one launch)
    }


# device sources of the kernels a workload's counter record covers: the batch-1 step runs the
# draft-block, fusion and context K/V kernels; the batched step the batched kernels
KERNEL_SOURCES = {"batch1": ("kernels.hip", "device_common.h", "dflare_impl.h"),
                  "batched": ("batched.hip", "batched.h", "device_common.h", "dflare_impl.h")}


def source_sha(workload: str = "qwen3_8b") -> str:
    """sha256 prefix of the device sources the recorded counter values of `workload` belong to."""
    import hashlib
    h = hashlib.sha256()
    for name in KERNEL_SOURCES["batched" if workload == "batched" else "batch1"]:
        with open(os.path.join(ROOT, "paper_2606_02091_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def counter_record_path(workload: str) -> str:
    return os.path.join(ROOT, "profiles", f"hbm_counters_{workload}.json")


def counter_traffic(kernel: str, workload: str, context: int):
    """HBM bytes per launch of `kernel` measured with rocprofv3 byte counters on this very
    workload (config name and context length), if the recorded measurement belongs to the
    device sources of this build; else None."""
    try:
        rec = json.load(open(counter_record_path(workload)))
        sha = source_sha(workload)
    except (OSError, ValueError):
        return None
    k = rec.get("kernels", {}).get(kernel)
    if (rec.get("sources_sha256_16") != sha or k is None or rec.get("workload") != workload
            or rec.get("context") != context):
        return None
    return int(k["fetch_kib"] * 1024 * rec["fetch_scale"] + k["write_kib"] * 1024 * rec["write_scale"])


# rocprofv3 kernel-name fragments of the kernels whose counters are recorded
COUNTER_KERNELS = {"draft_block": "k_draft", "kv_t": "k_kvt", "fuse": "k_fuse", "qkv": "BEPI_QKV",
                   "gate_up": "BEPI_SWIGLU", "attn": "k_battn"}


def summarize_counters(fetch_dir: str, write_dir: str, workload: str, context: int, scale: dict):
    """Write profiles/hbm_counters_<workload>.json from two rocprofv3 --pmc runs of this script
    (FETCH_SIZE, then WRITE_SIZE): per kernel the median KiB per dispatch over the step's
    launches.  Whole draft blocks are told from the single-phase launches of the per-phase
    pass by their fetch (over 0.8 of the largest; the LM head alone reads up to
    0.55 of a block); the step's appends and fusions from the
    untimed prefill's by their grid (at most 16 times the smallest); both runs launch the
    same sequence, so the write counters are taken at the same positions."""
    import csv
    import glob
    import statistics

    def load(d, counter):
        rows = []
        for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
            for r in csv.DictReader(open(f)):
                if r["Counter_Name"] == counter:
                    rows.append((int(r["Dispatch_Id"]), r["Kernel_Name"], int(r["Grid_Size"]),
                                 float(r["Counter_Value"])))
        rows.sort()
        return rows

    fetch_rows, write_rows = load(fetch_dir, "FETCH_SIZE"), load(write_dir, "WRITE_SIZE")
    out = {"kernels": {}}
    if workload == "batched":
        # the batched GEMMs by epilogue template (k_bgemm<epilogue, tile width>) and grid: Q/K/V
        # is the most frequent grid of k_bgemm<0, ...> (8 per step; the append's context K/V GEMM
        # runs once); the residual GEMMs k_bgemm<1, ...> alternate, output projection then down
        # projection, in every layer, so they are told apart by their order of dispatch
        def grids(frag):
            from collections import Counter
            return Counter(g for _, n, g, _ in fetch_rows if frag in n)
        g0 = grids("k_bgemm<0,")
        sel = {"gate_up": ("k_bgemm<2,", None, None), "lm_head": ("k_bgemm<3,", None, None),
               "attn": ("k_battn", None, None), "o": ("k_bgemm<1,", None, 0), "down": ("k_bgemm<1,", None, 1)}
        if g0:
            sel["qkv"] = ("k_bgemm<0,", g0.most_common(1)[0][0], None)

        def pick(rows_, frag, grid, parity):
            r = sorted((d, v) for d, n, g, v in rows_ if frag in n and (grid is None or g == grid))
            return [v for i, (_, v) in enumerate(r) if parity is None or i % 2 == parity]
        for kname, (frag, grid, parity) in sel.items():
            fr = pick(fetch_rows, frag, grid, parity)
            wr = pick(write_rows, frag, grid, parity)
            if fr and len(fr) == len(wr):
                out["kernels"][kname] = {"fetch_kib": int(statistics.median(fr)), "write_kib": int(statistics.median(wr)),
                                         "dispatches": len(fr)}
    for kname, frag in ({} if workload == "batched" else COUNTER_KERNELS).items():
        # the kernel's dispatches in launch order; both runs launch the same sequence
        fr = [(g, v) for _, n, g, v in fetch_rows if frag in n]
        wr = [(g, v) for _, n, g, v in write_rows if frag in n]
        if not fr or len(fr) != len(wr):
            continue
        if kname == "draft_block":
            top = max(v for _, v in fr)
            pick = [i for i, (_, v) in enumerate(fr) if v > 0.8 * top]
        else:  # the step's appends (1 to 16 rows), not the prefill's 512-row ones
            gmin = min(g for g, _ in fr)
            pick = [i for i, (g, _) in enumerate(fr) if g <= 16 * gmin]
        out["kernels"][kname] = {"fetch_kib": int(statistics.median(fr[i][1] for i in pick)),
                                 "write_kib": int(statistics.median(wr[i][1] for i in pick)),
                                 "dispatches": len(pick)}
    out.update({"workload": workload, "context": context, "sources_sha256_16": source_sha(workload),
                "fetch_scale": scale["fetch"], "write_scale": scale["write"],
                "_comment": "HBM KiB per dispatch from rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE runs of bench.py on "
                            "this workload, scaled to bytes by a plain 1 GiB device copy read with the same counters; "
                            "valid only for the device sources with this sha256 prefix"})
    with open(counter_record_path(workload), "w") as f:
        json.dump(out, f, indent=1)
    print(json.dumps(out))


def main():
    args = parse()
    if args.calibrate_copy:
        calibrate_copy()
        return
    if args.summarize_counters:
        from paper_2606_02091_amd import synth
        fs, ws = (float(x) for x in args.counter_scale.split(","))
        ctx = synth.CONFIGS[synth.BATCHED["model"]].context if args.config == "batched" else \
            synth.CONFIGS[args.config].context
        summarize_counters(*args.summarize_counters, args.config, ctx, {"fetch": fs, "write": ws})
        return
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(json.dumps({"error": "this build runs the draft step on one GPU only; "
                                   "bench.py --gpus N with N > 1 is not supported"}), flush=True)
        sys.exit(2)

    if args.config == "batched":
        bench_batched(args)
        return
    if args.loop:
        bench_loop(args)
        return
    if args.training:
        bench_training(args)
        return

    import numpy as np
    import torch

    from paper_2606_02091_amd import dflare as dfl
    from paper_2606_02091_amd import synth

    cfg = synth.CONFIGS[args.config]
    if args.target_layers:
        cfg = cfg.replace(n_target_layers=args.target_layers)
    L, B, S, H = cfg.context, cfg.block_size, cfg.n_target_layers, cfg.hidden
    variant, extra = VARIANTS[args.variant]
    dflash = args.variant == "dflash"
    torch.cuda.set_device(0)
    # a non-default stream of default priority, as a serving loop would use
    side = torch.cuda.Stream()
    torch.cuda.set_stream(side)
    t0 = time.time()
    w = synth.make_weights(cfg, kinds=synth.BASE_KINDS + extra)
    fusion_logits = w.pop("fusion_logits")
    print(f"[bench] weights generated in {time.time() - t0:.1f}s", file=sys.stderr, flush=True)
    model = dfl.DraftModel(cfg, w, None if dflash else fusion_logits, max_context=L + 16, max_new=512,
                           variant=variant)
    h = model.h
    dfl.dflare_set_sampling(h, args.temperature, 1)
    chunk = 512
    for s in range(0, L, chunk):
        n = min(chunk, L - s)
        model.fuse_append(dfl.bf16_tensor(synth.hidden_rows(cfg, s, n)))
    torch.cuda.synchronize()
    print(f"[bench] context prefilled to {model.context_len} rows", file=sys.stderr, flush=True)

    total = args.warmup + args.steps
    sizes = [int(x) for x in synth.append_sizes(total)]
    hid = {n: dfl.bf16_tensor(synth.hidden_rows(cfg, L - n, n)) for n in range(1, 17)}
    ids = torch.from_numpy(synth.block_ids(cfg)).cuda()
    out = torch.empty(B, dtype=torch.int32, device="cuda")

    def step(k):
        n = sizes[k % len(sizes)]
        dfl.dflare_truncate(h, L - n)
        dfl.dflare_fuse_append(h, hid[n], n)
        dfl.dflare_draft_block(h, ids, out)

    for k in range(args.warmup):
        step(k)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for k in range(args.warmup, total):
        step(k)
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    n_mean = float(np.mean(sizes[args.warmup:total]))
    print(f"[bench] timed {args.steps} steps: {ms:.4f} ms/step", file=sys.stderr, flush=True)

    # draft_block alone
    for _ in range(5):
        dfl.dflare_draft_block(h, ids, out)
    e0.record(stream)
    for _ in range(args.steps):
        dfl.dflare_draft_block(h, ids, out)
    e1.record(stream)
    torch.cuda.synchronize()
    block_ms = e0.elapsed_time(e1) / args.steps

    # per-kernel durations (hipEvents in the library, one kind per pass).  The kernels of a
    # step: the persistent draft-block kernel, fusion and context K/V projection.
    kb = kernel_bytes(cfg, L, n_mean, args.variant)

    def profile(kinds):
        res = {}
        for name, kind in kinds.items():
            dfl.dflare_profile_begin(h, kind)
            for k in range(args.profile_steps):
                step(k)
            tot, launches = dfl.dflare_profile_end(h)
            avg_us = 1000.0 * tot / max(launches, 1)
            per_step_us = 1000.0 * tot / args.profile_steps
            gbs = kb[name] / (avg_us * 1e-6) / 1e9 if avg_us > 0 else 0.0
            res[name] = {"avg_us": round(avg_us, 3), "launches_per_step": launches / args.profile_steps,
                         "us_per_step": round(per_step_us, 2), "bytes_per_launch": int(kb[name]),
                         "achieved_GBs": round(gbs, 1)}
        return res

    # the DFlash append runs on the batched GEMM kernels (slot 0)
    kern = profile({"draft_block": dfl.K_DRAFT, "fuse": dfl.K_B_FUSE if dflash else dfl.K_FUSE,
                    "kv_t": dfl.K_B_KV_T if dflash else dfl.K_KV_T})
    dom = max(kern, key=lambda k: kern[k]["us_per_step"])
    d = kern[dom]
    # the same phases launched one kernel each (what the persistent launch saves)
    per_phase = profile({"qkv": dfl.K_QKV, "attn": dfl.K_ATTN, "o": dfl.K_O, "gate_up": dfl.K_GATE_UP,
                         "down": dfl.K_DOWN, "lm_head": dfl.K_LM_HEAD})
    phases = phase_trace(dfl, h, step, cfg, kb, args.profile_steps)

    step_bytes = cfg.block_bytes(L) + cfg.append_bytes(n_mean) + (H * S * H * 2 if dflash else 0)
    step_gbs = step_bytes / (ms * 1e-3) / 1e9
    result = {
        "metric": METRIC.replace("Qwen3-8B", shape_name(cfg)),
        "value": round(1000.0 / ms, 2),
        "unit": "blocks/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{cfg.name}-shaped draft step: H={H}, {cfg.n_q_heads}q/{cfg.n_kv_heads}kv x "
                               f"{cfg.head_dim}, F={cfg.ffn}, V={cfg.vocab}, D={cfg.n_draft_layers}, S={S}, "
                               f"L={L}, B={B}, batch 1, n_new~U{{1..16}}"
                               + (f", sampled at T={args.temperature}" if args.temperature > 0 else ", greedy")
                               + (f", variant {args.variant}" if args.variant != "dflare" else ""),
                   "global_batch": 1, "seq_len": L, "parallelism": "single GPU"},
        "roofline": {"bound": "hbm", "achieved": round(d["achieved_GBs"], 1), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(d["achieved_GBs"] / HBM_PEAK_GBS, 4),
                     "traffic": counter_traffic(dom, args.config, L),
                     "kernel": dom, "bytes_per_launch": d["bytes_per_launch"], "avg_us": d["avg_us"]},
        "step_roofline": {"bytes_per_step": int(step_bytes), "achieved_GBs": round(step_gbs, 1),
                          "frac": round(step_gbs / HBM_PEAK_GBS, 4)},
        "draft_block_ms": round(block_ms, 5),
        "kernels": kern,
        "phases": phases,
        "per_phase_launches": per_phase,
    }

    probe = read_probe_gbs(dfl)
    result["roofline"]["probe_GBs"] = round(probe, 1)
    result["roofline"]["frac_of_probe"] = round(d["achieved_GBs"] / probe, 4)
    result["step_roofline"]["frac_of_probe"] = round(step_gbs / probe, 4)
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(cfg, w, fusion_logits, args.cpu_context or L, variant)
    print(json.dumps(result), flush=True)
    model.close()


def bench_loop(args):
    """The draft-then-verify loop at batch 1: per iteration draft_block, a synthetic target
    (its predictions agree with the first k candidates, k drawn ~ U{0..B-1} from a seeded
    generator and applied on the device; its hidden rows are a fixed seeded block), then
    dflare_accept_async, which appends the verified rows with the context length kept on
    the device, so the host enqueues iteration after iteration without waiting (with
    --loop-sync: dflare_accept, which waits once per iteration for k).  The target model's
    own forward pass is not part of the loop (no target weights exist here)."""
    import numpy as np
    import torch

    from paper_2606_02091_amd import dflare as dfl
    from paper_2606_02091_amd import synth

    cfg = synth.CONFIGS[args.config]
    L, B, V = cfg.context, cfg.block_size, cfg.vocab
    torch.cuda.set_device(0)
    side = torch.cuda.Stream()
    torch.cuda.set_stream(side)
    w = synth.make_weights(cfg)
    lg = w.pop("fusion_logits")
    total = args.warmup + args.steps
    model = dfl.DraftModel(cfg, w, lg, max_context=L + (total + 1) * B, max_new=512)
    h = model.h
    for s0 in range(0, L, 512):
        model.fuse_append(dfl.bf16_tensor(synth.hidden_rows(cfg, s0, min(512, L - s0))))
    hid = dfl.bf16_tensor(synth.hidden_rows(cfg, L, B, seed=11))
    ks = torch.from_numpy(np.random.default_rng(5).integers(0, B, size=total).astype(np.int64)).cuda()
    pos = torch.arange(B, device="cuda")
    # the target's disagreement pattern of every iteration, made before the timed region: XOR 1
    # at positions >= k changes a token and keeps it in the vocabulary (V is even)
    assert V % 2 == 0
    flip = (pos[None, :] >= ks[:, None]).to(torch.int32)
    ids = torch.from_numpy(synth.block_ids(cfg)).cuda()
    draft = torch.empty(B, dtype=torch.int32, device="cuda")
    tgt = torch.empty(B, dtype=torch.int32, device="cuda")
    em = torch.empty(B, dtype=torch.int32, device="cuda")
    k_dev = torch.zeros(total, dtype=torch.int32, device="cuda")

    def it(i):
        dfl.dflare_draft_block(h, ids, draft)
        # synthetic target: agrees with candidates 1..k, then predicts another token
        torch.bitwise_xor(torch.roll(draft, -1), flip[i], out=tgt)
        # the next block's ids are written over this block's (each position is read first)
        if args.loop_sync:
            k_dev[i] = dfl.dflare_accept(h, ids, draft, tgt, hid, ids, em)
        else:
            dfl.dflare_accept_async(h, ids, draft, tgt, hid, ids, em, k_dev[i:i + 1])

    for i in range(args.warmup):
        it(i)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.warmup, total):
        it(i)
    torch.cuda.synchronize()
    sec = time.perf_counter() - t0
    accepted = [int(x) for x in k_dev[args.warmup:].cpu()]
    assert accepted == [int(x) for x in ks[args.warmup:].cpu()], "the loop accepted other lengths than the target's"
    assert dfl.dflare_context_len(h) == L + sum(int(x) + 1 for x in ks.cpu())
    ms = 1000.0 * sec / args.steps
    tokens = sum(k + 1 for k in accepted)
    print(f"[bench] loop: {args.steps} iterations, {ms:.4f} ms each, {tokens / sec:.0f} tokens/s",
          file=sys.stderr, flush=True)
    print(json.dumps({
        "metric": f"draft-then-verify iterations/sec (draft side; B=16, {shape_name(cfg)} shape, batch 1)",
        "value": round(1000.0 / ms, 2), "unit": "iterations/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 5), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"{cfg.name}-shaped draft-then-verify loop from context {L}: draft_block, "
                               f"a synthetic target accepting k ~ U{{0..{B - 1}}} candidates, "
                               + ("dflare_accept (k + 1 rows appended, one host wait per iteration)" if args.loop_sync
                                  else "dflare_accept_async (k + 1 rows appended, length kept on the device, "
                                       "no host wait)"),
                   "global_batch": 1, "seq_len": L, "parallelism": "single GPU"},
        "tokens_per_s": round(tokens / sec, 1), "mean_accepted": round(float(np.mean(accepted)), 3),
        "timing": "host wall clock over the enqueued iterations, synchronized at both ends"
                  + (" (the loop waits for k every iteration)" if args.loop_sync else ""),
    }), flush=True)


def bench_training(args):
    """Training-side kernels at the paper's training shape (a 3,072-token sequence, 512
    anchors of 16-position blocks, Qwen3-8B heads: 32 query / 8 KV heads of 128): one draft
    layer's anchor attention forward and backward, and the position-weighted cross-entropy
    over the 151,936-token vocabulary (logits of the 8,192 block positions).  Inputs are seeded
    synthetic tensors; anchors ~ U{0..T-B}."""
    import numpy as np
    import torch

    from paper_2606_02091_amd import dflare as dfl

    T, n, B, nq, nkv, hd, V = 3072, 512, 16, 32, 8, 128, 151936
    torch.cuda.set_device(0)
    side = torch.cuda.Stream()
    torch.cuda.set_stream(side)
    g = torch.Generator(device="cuda").manual_seed(0)

    def bf(*shape):
        return torch.randn(*shape, device="cuda", generator=g).to(torch.bfloat16).view(torch.int16)

    q, kc, vc = bf(n * B, nq, hd), bf(T, nkv, hd), bf(T, nkv, hd)
    kb, vb = bf(n * B, nkv, hd), bf(n * B, nkv, hd)
    anchors_np = np.random.default_rng(1).integers(0, T - B + 1, size=n).astype(np.int32)
    anchors = torch.from_numpy(anchors_np).cuda()
    dout = torch.randn(n * B, nq, hd, device="cuda", generator=g)
    logits = 3.0 * torch.randn(n * B, V, device="cuda", generator=g)
    labels = torch.randint(0, V, (n * B,), device="cuda", generator=g, dtype=torch.int32)
    stream = torch.cuda.current_stream()

    def timed(fn, reps):
        for _ in range(2):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    out, lse = dfl.anchor_attention_fwd(q, kc, vc, kb, vb, anchors, B)
    reps = max(args.steps // 20, 3)
    fwd_ms = timed(lambda: dfl.anchor_attention_fwd(q, kc, vc, kb, vb, anchors, B), reps)
    bwd_ms = timed(lambda: dfl.anchor_attention_bwd(q, kc, vc, kb, vb, anchors, B, out, lse, dout), reps)
    ce_ms = timed(lambda: dfl.weighted_ce(logits, labels, B, 4.5), reps)
    # algorithmic work: per (block, query head) the two products over its a_i + B keys; the
    # backward counts the usual five (scores recomputed, dP, dV, dQ, dK)
    keys = (anchors_np.astype(np.float64) + B).sum()
    fwd_flop = 4.0 * B * hd * nq * keys
    bwd_flop = 2.5 * fwd_flop
    ce_bytes = 2.0 * n * B * V * 4  # logits read once, their gradient written once
    total_ms = fwd_ms + bwd_ms + ce_ms
    print(json.dumps({
        "metric": "training-side kernels (anchor attention fwd+bwd, weighted CE), one draft layer",
        "value": round((fwd_flop + bwd_flop) / ((fwd_ms + bwd_ms) * 1e-3) / 1e12, 2), "unit": "TFLOP/s",
        "n_gpus": 1, "steps": reps, "warmup": 2, "ms_per_step": round(total_ms, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"anchor attention of one draft layer: T={T}, {n} anchors ~ U{{0..{T - B}}}, "
                               f"B={B}, {nq}q/{nkv}kv x {hd}; weighted CE over V={V} for {n * B} rows",
                   "global_batch": n, "seq_len": T, "parallelism": "single GPU"},
        "kernels": {
            "attn_fwd": {"ms": round(fwd_ms, 4), "TFLOPs": round(fwd_flop / (fwd_ms * 1e-3) / 1e12, 1),
                         "flop": fwd_flop},
            "attn_bwd": {"ms": round(bwd_ms, 4), "TFLOPs": round(bwd_flop / (bwd_ms * 1e-3) / 1e12, 1),
                         "flop": bwd_flop},
            "weighted_ce": {"ms": round(ce_ms, 4), "GBs": round(ce_bytes / (ce_ms * 1e-3) / 1e9, 1),
                            "bytes": ce_bytes},
        },
        "roofline": {"bound": "mfma", "achieved": round((fwd_flop + bwd_flop) / ((fwd_ms + bwd_ms) * 1e-3) / 1e12, 1),
                     "peak": MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": round((fwd_flop + bwd_flop) / ((fwd_ms + bwd_ms) * 1e-3) / 1e12 / MFMA_PEAK_TFLOPS, 4),
                     "traffic": None, "kernel": "anchor attention fwd+bwd"},
        "ce_roofline": {"bound": "hbm", "achieved": round(ce_bytes / (ce_ms * 1e-3) / 1e9, 1), "peak": HBM_PEAK_GBS,
                        "unit": "GB/s", "frac": round(ce_bytes / (ce_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)},
    }), flush=True)


MFMA_PEAK_TFLOPS = 2500.0  # dense bf16 / fp16


def bench_batched(args):
    """Batched serving workload: 32 Qwen3-8B-shaped sequences with ragged contexts
    (L ~ U{512..4096}) drafted together.  One step = per sequence, truncate by its n_new and
    append n_new ~ U{1..16} rows (one batched fuse_append), then one batched draft_block:
    32 draft blocks per step."""
    import numpy as np
    import torch

    from paper_2606_02091_amd import dflare as dfl
    from paper_2606_02091_amd import synth

    spec = synth.BATCHED
    cfg = synth.CONFIGS[spec["model"]]
    n_seq = spec["n_seq"]
    lengths = [int(x) for x in synth.batched_lengths(n_seq, spec["lo"], spec["hi"])]
    B, S, H, V = cfg.block_size, cfg.n_target_layers, cfg.hidden, cfg.vocab
    q, kv, F, D = cfg.q_dim, cfg.kv_dim, cfg.ffn, cfg.n_draft_layers
    torch.cuda.set_device(0)
    side = torch.cuda.Stream()
    torch.cuda.set_stream(side)
    t0 = time.time()
    w = synth.make_weights(cfg)
    fusion_logits = w.pop("fusion_logits")
    print(f"[bench] weights generated in {time.time() - t0:.1f}s", file=sys.stderr, flush=True)
    model = dfl.DraftModel(cfg, w, fusion_logits, max_context=max(lengths) + 16, max_new=16 * n_seq,
                           max_batch=n_seq)
    h = model.h
    dfl.dflare_set_sampling(h, args.temperature, 1)
    # one shared stream of target rows on the device; sequence i reads rows 16 i + (0 .. L_i)
    base = [16 * i for i in range(n_seq)]
    R = max(b + L for b, L in zip(base, lengths))
    rows_dev = dfl.bf16_tensor(synth.hidden_rows(cfg, 0, R))
    for i, L in enumerate(lengths):
        for s0 in range(0, L, 512):
            n = min(512, L - s0)
            model.fuse_append_batched([i], [n], rows_dev[:, base[i] + s0:base[i] + s0 + n].contiguous())
    torch.cuda.synchronize()
    print(f"[bench] {n_seq} contexts prefilled, mean L {np.mean(lengths):.0f}", file=sys.stderr, flush=True)

    seqs = list(range(n_seq))
    total = args.warmup + args.steps
    pool = 8
    sizes = synth.append_sizes(pool * n_seq).reshape(pool, n_seq)
    inputs = []
    for k in range(pool):
        parts = [rows_dev[:, base[i] + lengths[i] - int(sizes[k, i]):base[i] + lengths[i]] for i in seqs]
        inputs.append(torch.cat(parts, dim=1).contiguous())
    ids = torch.from_numpy(np.stack([synth.block_ids(cfg, step=0, seed=200 + i) for i in seqs])).cuda()
    out = torch.empty((n_seq, B), dtype=torch.int32, device="cuda")

    def step(k):
        nk = sizes[k % pool]
        for i in seqs:
            dfl.dflare_truncate_seq(h, i, lengths[i] - int(nk[i]))
        dfl.dflare_fuse_append_batched(h, seqs, nk, inputs[k % pool])
        dfl.dflare_draft_block_batched(h, seqs, ids, out)

    for k in range(args.warmup):
        step(k)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for k in range(args.warmup, total):
        step(k)
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    print(f"[bench] timed {args.steps} batched steps: {ms:.4f} ms/step", file=sys.stderr, flush=True)

    # per-kind durations (library hipEvents, one kind per pass)
    M = n_seq * B
    n_mean = float(sizes.mean()) * n_seq
    kv_bytes = sum(2 * L * kv * 2 for L in lengths)          # context K and V of one layer, all sequences
    work = {  # algorithmic (FLOPs, HBM bytes) per launch
        "qkv": (2 * M * (q + 2 * kv) * H, (q + 2 * kv) * H * 2),
        "attn": (sum(4 * q * B * (L + B) for L in lengths), kv_bytes),
        "o": (2 * M * H * q, H * q * 2),
        "gate_up": (2 * M * 2 * F * H, 2 * F * H * 2),
        "down": (2 * M * H * F, H * F * 2),
        "lm_head": (2 * M * V * H, V * H * 2),
        "kv_t": (D * 2 * n_mean * 2 * kv * H, D * 2 * kv * H * 2),  # one launch for every layer
        "epilogues": (0, 0),
        "fuse": (0, S * n_mean * H * 2),
        "draft": (0, 0),
        "append": (0, 0),
    }
    kinds = {"qkv": dfl.K_B_QKV, "attn": dfl.K_B_ATTN, "o": dfl.K_B_O, "gate_up": dfl.K_B_GATE_UP,
             "down": dfl.K_B_DOWN, "lm_head": dfl.K_B_LM_HEAD, "kv_t": dfl.K_B_KV_T, "epilogues": dfl.K_B_EPI,
             "fuse": dfl.K_B_FUSE, "draft": dfl.K_B_DRAFT, "append": dfl.K_B_APPEND}
    kern = {}
    for name, kind in kinds.items():
        dfl.dflare_profile_begin(h, kind)
        for k in range(args.profile_steps):
            step(k)
        tot, launches = dfl.dflare_profile_end(h)
        avg_us = 1000.0 * tot / max(launches, 1)
        fl, by = work[name]
        kern[name] = {"avg_us": round(avg_us, 3), "launches_per_step": launches / args.profile_steps,
                      "us_per_step": round(1000.0 * tot / args.profile_steps, 2)}
        if fl:
            kern[name]["TFLOPs"] = round(fl / (avg_us * 1e-6) / 1e12, 1)
            kern[name]["flops_per_launch"] = int(fl)
        if by:
            kern[name]["GBs"] = round(by / (avg_us * 1e-6) / 1e9, 1)
            kern[name]["bytes_per_launch"] = int(by)
    gemms = ("qkv", "o", "gate_up", "down", "lm_head")
    dom = max(gemms, key=lambda k: kern[k]["us_per_step"])
    d = kern[dom]
    # whole step: every GEMM and the attention, against both roofs
    step_flops = sum(work[k][0] * kern[k]["launches_per_step"] for k in ("qkv", "attn", "o", "gate_up", "down",
                                                                          "lm_head", "kv_t"))
    step_bytes = cfg.block_bytes(0) - B * H * 2 + D * kv_bytes + M * H * 2 + cfg.append_bytes(n_mean)
    result = {
        "metric": "draft blocks/sec (B=16, Qwen3-8B shape, batch 32, ragged contexts)",
        "value": round(1000.0 * n_seq / ms, 1),
        "unit": "blocks/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{cfg.name}-shaped draft step for {n_seq} sequences at once: L ~ U{{"
                               f"{spec['lo']}..{spec['hi']}}} per sequence (mean {np.mean(lengths):.0f}), "
                               f"n_new ~ U{{1..16}} per sequence per step, B={B}"
                               + (f", sampled at T={args.temperature}" if args.temperature > 0 else ", greedy"),
                   "global_batch": n_seq, "seq_len": int(max(lengths)), "parallelism": "single GPU"},
        "roofline": {"bound": "mfma", "achieved": d["TFLOPs"], "peak": MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(d["TFLOPs"] / MFMA_PEAK_TFLOPS, 4),
                     "traffic": counter_traffic(dom, "batched", cfg.context), "kernel": dom,
                     "flops_per_launch": d["flops_per_launch"], "avg_us": d["avg_us"]},
        "step_roofline": {"flops_per_step": int(step_flops), "bytes_per_step": int(step_bytes),
                          "mfma_frac": round(step_flops / (ms * 1e-3) / 1e12 / MFMA_PEAK_TFLOPS, 4),
                          "hbm_frac": round(step_bytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)},
        "kernels": kern,
    }
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(cfg, w, fusion_logits, args.cpu_context or cfg.context)
    print(json.dumps(result), flush=True)
    model.close()


def phase_trace(dfl, h, step, cfg, kb, steps):
    """Per-phase time inside the persistent draft-block kernel, from its wall-clock trace
    (100 MHz, four marks per phase).  For each phase kind, microseconds per step (summed
    over layers), medians over work-groups: "us" from the moment the work-groups pass the
    grid barrier into the phase to the moment they pass into the next one; "body" until the
    work-group's stores are complete, "body_max" for the slowest work-group; "wait" at the
    next barrier.  "seg" splits the body at the phase's inner marks (GEMM: main loop, chunk
    epilogues, split-K combine and final epilogue; attention: key staging, scores and
    values, merge and stores).  "GBs" relates "us" to the phase's algorithmic bytes."""
    import numpy as np
    n_launch, _, blocks, n_phase = dfl.dflare_kernel_stats(h)[:4]
    if n_launch != 1:
        return None
    dfl.dflare_set_option(h, dfl.OPT_TRACE, 1)
    names = ["embed"] + ["qkv", "attn", "comb", "o", "gate_up", "down"] * cfg.n_draft_layers + ["lm_head"]
    acc = {}
    for k in range(steps):
        step(k)
        t = dfl.dflare_debug_read(h, dfl.DBG_TRACE, 0, (blocks, n_phase, 4)).astype(np.float64)
        start, end = t[:, :, 0], t[:, :, 3]
        nxt = np.concatenate([start[:, 1:], end[:, -1:]], axis=1)
        for p, name in enumerate(names):
            a = acc.setdefault(name, np.zeros(7))
            m1, m2 = t[:, p, 1], t[:, p, 2]
            seg = [np.nan, np.nan, np.nan]
            ok1, ok2 = m1 >= 0, m2 >= 0
            if ok1.any() and ok2.any():
                seg = [np.median((m1 - start[:, p])[ok1]), np.median((m2 - m1)[ok1 & ok2]),
                       np.median((end[:, p] - m2)[ok2])]
            a += [np.median(nxt[:, p] - start[:, p]), np.median(end[:, p] - start[:, p]),
                  np.max(end[:, p] - start[:, p]), np.median(nxt[:, p] - end[:, p])] + seg
    dfl.dflare_set_option(h, dfl.OPT_TRACE, 0)
    layer_bytes = {"qkv": kb["qkv"], "attn": kb["attn"], "o": kb["o"], "gate_up": kb["gate_up"],
                   "down": kb["down"]}
    out = {}
    for name, a in acc.items():
        us, body, body_max, wait, s1, s2, s3 = (a / steps).tolist()
        reps = cfg.n_draft_layers if name in layer_bytes else 1
        nbytes = layer_bytes.get(name, kb["lm_head"] if name == "lm_head" else 0) * reps
        out[name] = {"us": round(us, 2), "body": round(body, 2), "body_max": round(body_max, 2),
                     "wait": round(wait, 2),
                     "GBs": round(nbytes / (us * 1e-6) / 1e9, 1) if nbytes and us > 0 else None}
        if not np.isnan(s1):
            out[name]["seg"] = [round(s1, 2), round(s2, 2), round(s3, 2)]
    return out


def cpu_baseline(cfg, w, fusion_logits, ctx, variant=0):
    """The fp64 oracle, as it stands, timed on this host: whole draft steps (truncate back,
    append 8 rows, draft a block) at context ctx after an untimed prefill, first with every
    core this process may run on, then one step on one thread."""
    import numpy as np
    from threadpoolctl import threadpool_info, threadpool_limits

    from oracle import dflare_oracle as orc
    from paper_2606_02091_amd import synth

    cores = len(os.sched_getaffinity(0))
    o = orc.DraftOracle(cfg, w, None if variant & 8 else fusion_logits, max_context=ctx + 64, variant=variant)
    with threadpool_limits(cores):
        t = time.perf_counter()
        for s0 in range(0, ctx, 512):
            o.append(synth.hidden_rows(cfg, s0, min(512, ctx - s0)))
        prefill_s = time.perf_counter() - t
        used = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    rows = synth.hidden_rows(cfg, ctx, 8)
    ids = synth.block_ids(cfg)

    def timed(threads, min_seconds, max_steps):
        with threadpool_limits(threads):
            steps, t = 0, time.perf_counter()
            while steps == 0 or (time.perf_counter() - t < min_seconds and steps < max_steps):
                o.truncate(ctx)
                o.append(rows)
                o.draft_block(ids, keep_logits=False)
                steps += 1
            return (time.perf_counter() - t) / steps, steps

    sec, steps = timed(cores, 10.0, 100)
    sec1, steps1 = timed(1, 0.0, 1)
    cpu = "unknown"
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    cpu = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"value": round(1.0 / sec, 5), "unit": "blocks/s", "cores": int(used), "kind": "oracle",
            "sample": f"{steps} steps (fuse_append of 8 rows + draft_block each) of the same model at context {ctx} "
                      f"after an untimed {prefill_s:.0f} s prefill, {sec:.2f} s per step on {used} threads "
                      f"({cores} cores in the affinity mask); then {steps1} step on 1 thread, {sec1:.2f} s; "
                      f"{cpu} ({platform.machine()})",
            "seconds": round(sec, 3), "affinity_cores": cores,
            "value_1thread": round(1.0 / sec1, 5), "seconds_1thread": round(sec1, 3)}


def read_probe_gbs(dfl, nbytes=2 << 30, reps=6):
    """The best rate of a plain streaming read of nbytes of device memory (the library's
    read probe), GB/s: the HBM read ceiling of this machine."""
    import torch
    buf = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    buf.fill_(1)
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    st = torch.cuda.current_stream()
    best = 1e30
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(st)
        dfl.read_probe(buf, sink)
        e1.record(st)
        torch.cuda.synchronize()
        best = min(best, e0.elapsed_time(e1) * 1e-3)
    del buf
    return nbytes / best / 1e9


if __name__ == "__main__":
    main()
