"""GPU parity of temperature sampling (the paper's temperature-1 decoding, Sec. 5, Table 1):
the library's Gumbel-max draws against the oracle's, which use the same Philox4x64-10
uniforms (word b mod 4 at counter: token id, block position b div 4, draw, sequence slot).  A sampled token must
equal the oracle's wherever the oracle's perturbed-score margin (top-1 minus top-2 of
z / T + G) exceeds the bar of tests/parity.py, and otherwise score within it of the maximum.
Also: draws replay after dflare_set_sampling, temperature 0 is greedy, the persistent and
the per-phase launches draw the same tokens, and batched calls draw per sequence slot."""
import numpy as np
import pytest
import torch

from paper_2606_02091_amd import dflare as dfl
from paper_2606_02091_amd import synth
import parity as P
import test_gpu_batched as TB
import test_gpu_parity as TP

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover - CPU container
    pytest.skip("needs a GPU", allow_module_level=True)

SEED = 20260601


@pytest.mark.parametrize("name,temperature", [("tiny", 1.0), ("hd128", 1.0), ("gqa8_hd64", 0.5),
                                              ("ragged", 2.0)])
def test_sampled_tokens_match_oracle(name, temperature):
    cfg, L, mode = TP.CASES[name]
    model, orc, _, _ = TP.build_pair(cfg, L, mode, debug=False)
    dfl.dflare_set_sampling(model.h, temperature, SEED)
    ids = synth.block_ids(cfg, step=0)
    stats = {"strict": 0, "near_ties": 0}
    first = None
    for draw in range(3):
        out = model.draft_block(TP.ids_tensor(ids)).cpu().numpy()
        ref = orc.draft_block(ids, temperature=temperature, seed=SEED, draw=draw)
        s = P.check_tokens(out, ref["scores"])
        stats = {k: stats[k] + s[k] for k in stats}
        if draw == 0:
            first = out.copy()
    print(f"[sampling] {name} T={temperature}: {stats}", flush=True)
    # the draw counter restarts with the seed: the first draw replays bit for bit
    dfl.dflare_set_sampling(model.h, temperature, SEED)
    assert np.array_equal(model.draft_block(TP.ids_tensor(ids)).cpu().numpy(), first)
    # temperature 0 is the greedy argmax again
    dfl.dflare_set_sampling(model.h, 0.0, SEED)
    greedy = model.draft_block(TP.ids_tensor(ids)).cpu().numpy()
    P.check_tokens(greedy, orc.draft_block(ids)["logits"])
    model.close()


def test_sampling_same_in_persistent_and_per_phase_launches():
    cfg, L, mode = TP.CASES["hd128"]
    side = torch.cuda.Stream()
    with torch.cuda.stream(side):
        model, orc, _, _ = TP.build_pair(cfg, L, mode, debug=False)
        ids_np = synth.block_ids(cfg, step=1)
        ids = TP.ids_tensor(ids_np)
        out = torch.empty(cfg.block_size, dtype=torch.int32, device="cuda")
        for draw in range(2):
            dfl.dflare_set_sampling(model.h, 1.0, SEED)
            for _ in range(draw):
                model.draft_block(ids, out)
            dfl.dflare_set_option(model.h, dfl.OPT_PERSISTENT, 1)
            assert dfl.dflare_kernel_stats(model.h)[0] == 1
            model.draft_block(ids, out)
            side.synchronize()
            persistent = out.cpu().numpy().copy()
            dfl.dflare_set_sampling(model.h, 1.0, SEED)
            for _ in range(draw):
                model.draft_block(ids, out)
            dfl.dflare_set_option(model.h, dfl.OPT_PERSISTENT, 0)
            per_phase = model.draft_block(ids).cpu().numpy()
            side.synchronize()
            assert np.array_equal(persistent, per_phase), (draw, persistent, per_phase)
            P.check_tokens(persistent, orc.draft_block(ids_np, temperature=1.0, seed=SEED, draw=draw)["scores"])
        for bad in (-1.0, float("nan"), float("inf")):
            with pytest.raises(dfl.DFlareError):
                dfl.dflare_set_sampling(model.h, bad, SEED)
        model.close()


def test_batched_sampling_matches_oracles():
    cfg, lengths, slots, max_batch = TB.CASES["hd128_b16"]
    model, orcs, _ = TB.build_batched(cfg, lengths, slots, max_batch)
    dfl.dflare_set_sampling(model.h, 1.0, SEED)
    for draw in range(2):
        ids = np.stack([TB.slot_ids(cfg, s, draw) for s in slots])
        out = model.draft_block_batched(slots, TB.ids_tensor(ids)).cpu().numpy()
        for i, s in enumerate(slots):
            ref = orcs[s].draft_block(ids[i], temperature=1.0, seed=SEED, draw=draw, slot=s)
            P.check_tokens(out[i], ref["scores"])
    # a batch-1 call on slot 0 and a batched call on slot 0 with the same draw use the same noise
    ids0 = TB.slot_ids(cfg, 0, 5)
    dfl.dflare_set_sampling(model.h, 1.0, SEED)
    one = model.draft_block(TB.ids_tensor(ids0)).cpu().numpy()
    dfl.dflare_set_sampling(model.h, 1.0, SEED)
    bat = model.draft_block_batched([0], TB.ids_tensor(ids0[None])).cpu().numpy()[0]
    ref = orcs[0].draft_block(ids0, temperature=1.0, seed=SEED, draw=0, slot=0)
    P.check_tokens(one, ref["scores"])
    P.check_tokens(bat, ref["scores"])
    model.close()
