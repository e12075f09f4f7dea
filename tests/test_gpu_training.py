"""GPU parity of the training-side kernels against the fp64 oracle (oracle/training_oracle.py)
on the same seeded bf16 inputs: anchor attention (Sec. 3.3) forward and backward, and the
progressive position-weighted cross-entropy (Eq. 5).

Shapes span several 32-key tiles with ragged tails, block sizes 16 and 5, GQA groups of 4 and
3, more blocks than one 64-block gradient chunk, anchors 0 (no context) and T (all of it), and
T = 0.  The attention's products run on bf16 matrix cores with probabilities and gradients
rounded to bf16 as operands; the bar is the per-tensor relative error of tests/parity.py
(2e-2 of the tensor's largest magnitude).  Gradients must repeat bit for bit.
"""
import numpy as np
import pytest
import torch

from oracle import training_oracle as tr
from paper_2606_02091_amd import dflare as dfl
from paper_2606_02091_amd import synth
import parity as P

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover - CPU container
    pytest.skip("needs a GPU", allow_module_level=True)

CASES = {
    # name: (n_blocks, B, T, n_q, n_kv, hd)
    "b16_hd128": (5, 16, 200, 8, 2, 128),
    "b5_hd64_gqa3": (7, 5, 77, 6, 2, 64),
    "chunks_hd64": (150, 4, 300, 4, 1, 64),
    "no_context": (3, 8, 0, 4, 2, 128),
}


def inputs(n, B, T, nq, nkv, hd, seed=0):
    rng = np.random.default_rng(seed)

    def bf(shape):
        return synth.round_bf16(rng.standard_normal(shape).astype(np.float32))

    x = dict(q=bf((n * B, nq, hd)), k_ctx=bf((T, nkv, hd)), v_ctx=bf((T, nkv, hd)),
             k_blk=bf((n * B, nkv, hd)), v_blk=bf((n * B, nkv, hd)))
    anchors = rng.integers(0, T + 1, size=n).astype(np.int32)
    if n >= 2:
        anchors[0], anchors[1] = 0, T
    dout = rng.standard_normal((n * B, nq, hd))
    return x, anchors, dout


def dev(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda()


@pytest.mark.parametrize("name", list(CASES))
def test_anchor_attention_matches_oracle(name):
    n, B, T, nq, nkv, hd = CASES[name]
    print(f"[training] attention {name}", flush=True)
    x, anchors, dout = inputs(n, B, T, nq, nkv, hd)
    f64 = {k: synth.bf16_to_f32(v).astype(np.float64) for k, v in x.items()}
    d = {k: dev(v) for k, v in x.items()}
    a = torch.from_numpy(anchors).cuda()
    out, lse = dfl.anchor_attention_fwd(d["q"], d["k_ctx"], d["v_ctx"], d["k_blk"], d["v_blk"], a, B)
    ro, rl = tr.anchor_attention_fwd(**f64, anchors=list(anchors), B=B)
    e_out, e_lse = P.relinf(out.cpu().numpy(), ro), P.relinf(lse.cpu().numpy(), rl)
    assert e_out <= P.REL_TOL and e_lse <= P.REL_TOL, (e_out, e_lse)
    do = torch.from_numpy(dout.astype(np.float32)).cuda()
    g = dfl.anchor_attention_bwd(d["q"], d["k_ctx"], d["v_ctx"], d["k_blk"], d["v_blk"], a, B, out, lse, do)
    ref = tr.anchor_attention_bwd(**f64, anchors=list(anchors), B=B, dout=dout)
    errs = {}
    for nm, got, want in zip(("dq", "dk_ctx", "dv_ctx", "dk_blk", "dv_blk"), g, ref):
        if want.size == 0:
            continue
        errs[nm] = P.relinf(got.cpu().numpy(), want)
        assert errs[nm] <= P.REL_TOL, (nm, errs[nm])
    g2 = dfl.anchor_attention_bwd(d["q"], d["k_ctx"], d["v_ctx"], d["k_blk"], d["v_blk"], a, B, out, lse, do)
    for u, v in zip(g, g2):
        assert torch.equal(u, v)
    print(f"[training] {name}: out {e_out:.2e} lse {e_lse:.2e} "
          + " ".join(f"{k} {v:.2e}" for k, v in errs.items()), flush=True)


# (V, blocks): rows streamed twice (V = 1000, 1003), and rows held on chip (V a multiple of 4 in
# 111,616 .. 152,512): none in LDS, the Qwen3 vocabulary, LDS full; 17 blocks = 272 rows give
# work-groups a second row
@pytest.mark.parametrize("V,n", [(1000, 6), (1003, 6), (111616, 17), (151936, 2), (152512, 2)])
def test_weighted_ce_matches_oracle(V, n):
    B = 16
    rng = np.random.default_rng(3)
    z = (3.0 * rng.standard_normal((n * B, V))).astype(np.float32)
    y = rng.integers(0, V, size=n * B).astype(np.int32)
    y[rng.random(n * B) < 0.1] = -1
    y[1], y[2], y[3] = V - 1, 0, min(V - 1, 111616)  # last value, first value, first value past the registers
    gamma = 4.5
    loss, ce, dz = dfl.weighted_ce(torch.from_numpy(z).cuda(), torch.from_numpy(y).cuda(), B, gamma)
    rloss, rce, rdz = tr.weighted_ce(z.astype(np.float64), y, B, gamma)
    assert abs(float(loss.cpu()[0]) - rloss) <= 1e-5 * max(1.0, abs(rloss))
    assert P.relinf(ce.cpu().numpy(), rce) <= 1e-5
    assert P.relinf(dz.cpu().numpy(), rdz) <= 1e-5
    with pytest.raises(dfl.DFlareError):
        dfl.weighted_ce(torch.from_numpy(z[:17]).cuda(), torch.from_numpy(y[:17]).cuda(), B, gamma)


def test_anchor_attention_full_training_shape_sampled():
    """The training shape the benchmark times (T = 3,072, 512 blocks of B = 16, 32 query / 8 KV
    heads x 128): every kernel runs on the whole problem in its benchmark launch configuration
    (8 gradient chunks, XCD-grouped work order), and sampled blocks are checked against the
    oracle run on that block alone — its outputs, lse, dQ and block-key gradients depend on
    nothing else.  Anchors lie in 0 .. 2,900 except one block's, T - B: the context keys from
    2,901 up to it are seen by that block only, so their gradients are that block's too, and
    keys at or past T - B are seen by no block (zero gradients)."""
    n, B, T, nq, nkv, hd = 512, 16, 3072, 32, 8, 128
    print("[training] full shape sampled", flush=True)
    rng = np.random.default_rng(11)

    def bf(shape):
        return synth.round_bf16(rng.standard_normal(shape).astype(np.float32))

    x = dict(q=bf((n * B, nq, hd)), k_ctx=bf((T, nkv, hd)), v_ctx=bf((T, nkv, hd)),
             k_blk=bf((n * B, nkv, hd)), v_blk=bf((n * B, nkv, hd)))
    anchors = rng.integers(0, 2901, size=n).astype(np.int32)
    top = 7
    anchors[0], anchors[top] = 0, T - B
    dout = rng.standard_normal((n * B, nq, hd)).astype(np.float32)
    d = {k: dev(v) for k, v in x.items()}
    a = torch.from_numpy(anchors).cuda()
    out, lse = dfl.anchor_attention_fwd(d["q"], d["k_ctx"], d["v_ctx"], d["k_blk"], d["v_blk"], a, B)
    g = dfl.anchor_attention_bwd(d["q"], d["k_ctx"], d["v_ctx"], d["k_blk"], d["v_blk"], a, B, out, lse,
                                 torch.from_numpy(dout).cuda())
    out, lse = out.cpu().numpy(), lse.cpu().numpy()
    dq, dkc, dvc, dkb, dvb = (t.cpu().numpy() for t in g)
    assert not dkc[T - B:].any() and not dvc[T - B:].any()
    kc64 = synth.bf16_to_f32(x["k_ctx"]).astype(np.float64)
    vc64 = synth.bf16_to_f32(x["v_ctx"]).astype(np.float64)
    for i in (0, top, 200, n - 1):
        rows = slice(i * B, (i + 1) * B)
        blk = {k: synth.bf16_to_f32(x[k][rows]).astype(np.float64) for k in ("q", "k_blk", "v_blk")}
        ro, rl = tr.anchor_attention_fwd(blk["q"], kc64, vc64, blk["k_blk"], blk["v_blk"], [int(anchors[i])], B)
        rdq, rdkc, rdvc, rdkb, rdvb = tr.anchor_attention_bwd(blk["q"], kc64, vc64, blk["k_blk"], blk["v_blk"],
                                                               [int(anchors[i])], B, dout[rows].astype(np.float64))
        errs = {"out": P.relinf(out[rows], ro), "lse": P.relinf(lse[rows], rl), "dq": P.relinf(dq[rows], rdq),
                "dk_blk": P.relinf(dkb[rows], rdkb), "dv_blk": P.relinf(dvb[rows], rdvb)}
        if i == top:
            only = slice(2901, T - B)
            errs["dk_ctx_own"] = P.relinf(dkc[only], rdkc[only])
            errs["dv_ctx_own"] = P.relinf(dvc[only], rdvc[only])
        print(f"[training] full shape block {i} (anchor {anchors[i]}): "
              + " ".join(f"{k} {v:.2e}" for k, v in errs.items()), flush=True)
        for k, v in errs.items():
            assert v <= P.REL_TOL, (i, k, v)
