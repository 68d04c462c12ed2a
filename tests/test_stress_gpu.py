"""Stress cases of the HIP path against the float64 oracle, through the C ABI:

* peaked rows: logits with a standard deviation of 12-15 (the spread of a
  trained model's logits) instead of the workloads' 2, so that a few entries
  carry most of each row's probability, with old log-probs perturbed so that
  about a fifth of the tokens clip; through the fused step (its fp16 logit
  chunk), the separate calls (the recomputing backward) and the loss-only call;
* a NaN in a valid row: that row's log-prob and the loss are NaN, every other
  row is unchanged, and the calls return;
* a mid-size fused step with row chunks of 16384 rows (three chunks, the last
  ragged) and a vocabulary above 8192, so that every GEMM of the step runs its
  full super-group tile order, compared with the oracle on the whole dH and dW.
"""
import math
import zlib

import numpy as np
import pytest
import torch

import paper_2505_17826_amd as R
from gen import synth
from oracle import rft_oracle as O
from tests.gpu_cases import (TOL_GRAD_FRO, TOL_LOGP, TOL_LOSS_ABS, TOL_LOSS_REL, compare_stats,
                             compare_step, cpu, gpu_fused_step, gpu_step, oracle_eps,
                             oracle_step, params_of, perturbed_logprobs, rel_fro, requires_gpu,
                             tokens_of)

pytestmark = [pytest.mark.gpu, requires_gpu]
DEV = torch.device("cuda")


def _batch(cid, name, over):
    cfg = synth.config(cid, **over)
    return synth.make_batch(cfg, "cpu", seed_key=(cid, zlib.crc32(("stress" + name).encode()) % 100003))


# ------------------------------------------------------------ peaked rows ----
PEAKED = [
    ("d128-V4099-std12", dict(n_prompts=2, group=8, len_lo=20, len_hi=150, pad_to=150, d=128,
                              V=4099, dtype="bf16", logit_std=12.0, reward="normal")),
    ("d256-V9000-std15", dict(n_prompts=1, group=8, len_lo=100, len_hi=300, pad_to=300, d=256,
                              V=9000, dtype="bf16", logit_std=15.0, reward="normal")),
]


@pytest.mark.parametrize("name,over", PEAKED, ids=[c[0] for c in PEAKED])
def test_peaked_logits_fused_step_and_separate_calls(name, over):
    b = _batch(1, name, over)
    lp, ent, _ = O.token_logprobs(b.H, b.W, b.ids, b.mask)
    m = b.mask.numpy() != 0
    old, ref = perturbed_logprobs(lp, b)
    o = oracle_step(b, old, ref)
    of = o["fwd"]
    clipfrac = of["clipfrac"]
    print(f"[stress peaked] {name}: mean entropy {ent[m].mean():.3f} nats, mean logp "
          f"{lp[m].mean():.3f}, clipfrac {clipfrac:.3f}", flush=True)
    # the rows are peaked and the clip branch is exercised
    assert ent[m].mean() < 0.5 * math.log(b.cfg.V)
    assert 0.1 <= clipfrac <= 0.3
    gf = gpu_fused_step(b, old, ref)        # fp16 logit chunk, dZ from it
    compare_step(gf, o, b)
    gs = gpu_step(b, old, ref)              # recomputing backward
    compare_step(gs, o, b)
    print(f"[stress peaked] {name}: fused dH {rel_fro(gf['dH'], o['dH']):.2e} dW "
          f"{rel_fro(gf['dW'], o['dW']):.2e}; separate dH {rel_fro(gs['dH'], o['dH']):.2e} "
          f"dW {rel_fro(gs['dW'], o['dW']):.2e}", flush=True)


@pytest.mark.parametrize("V,std", [(8192, 15.0), (152004, 12.0)])
def test_peaked_logits_loss_only(V, std):
    n_prompts = 8 if V < 100000 else 2
    cfg = synth.config(4, n_prompts=n_prompts, group=8, V=V, logit_std=std)
    b = synth.make_batch(cfg, "cpu", seed_key=(4, 1000 + V))
    lp, ent, lse = O.token_logprobs_from_logits(b.logits, b.ids, b.mask)
    old, ref = perturbed_logprobs(lp, b)
    el, eh, be = oracle_eps(cfg)
    o = O.loss_only_step(b.logits, b.ids, b.mask, b.seq_start, b.rewards, cfg.group,
                         old.astype(np.float64), ref.astype(np.float64), el, eh, be, cfg.agg)
    m = b.mask.numpy() != 0
    print(f"[stress peaked loss-only] V={V}: mean entropy {ent[m].mean():.3f}, clipfrac "
          f"{o['fwd']['clipfrac']:.3f}", flush=True)
    assert ent[m].mean() < 0.5 * math.log(V)
    tok = tokens_of(b)
    t = lambda x: torch.from_numpy(x).to(DEV)
    adv = R.rft_group_advantages(b.rewards.to(DEV), cfg.group)
    glp = torch.empty(b.T, device=DEV); gent = torch.empty_like(glp); glse = torch.empty_like(glp)
    ggrad = torch.empty_like(glp)
    _, dl, st = R.rft_ppo_clip_fused_logits(tok, b.logits.to(DEV), t(old), t(ref), adv,
                                            params_of(cfg), logp=glp, entropy=gent, lse=glse,
                                            grad_logp=ggrad)
    torch.cuda.synchronize()
    for k, g in (("logp", glp), ("entropy", gent), ("lse", glse)):
        gg = cpu(g)
        assert np.all(gg[~m] == 0)
        err = np.abs(gg[m] - o[k][m]).max()
        assert err <= TOL_LOGP, (k, err)
    keep = o["fwd"]["margin"] >= 1e-4
    compare_stats(R.stats_to_dict(st), o["fwd"], n_near=int((~keep).sum()))
    rows = o["fwd"]["weights_rows"][keep]
    go, gg = o["fwd"]["grad_logp"][rows], cpu(ggrad)[rows]
    np.testing.assert_allclose(gg, go, rtol=1e-3, atol=1e-7 * np.abs(go).max())
    dl_o = np.zeros(b.logits.shape)
    for r_, v in o["dlogits"].items():
        dl_o[r_] = v
    e = rel_fro(cpu(dl), dl_o)
    print(f"[stress peaked loss-only] V={V}: dlogits rel {e:.2e}", flush=True)
    assert e <= TOL_GRAD_FRO


# ------------------------------------------------------- NaN in a valid row ----
def test_nan_in_a_valid_hidden_row():
    """A NaN in one valid row of the hidden states: that row's log-prob, entropy
    and lse are NaN, the loss is NaN, the other rows' outputs are bit-identical
    to the run without the NaN, and every call returns (separate calls and the
    fused step)."""
    over = dict(n_prompts=2, group=8, len_lo=20, len_hi=90, pad_to=96, d=128, V=3000, dtype="bf16")
    b = _batch(1, "nan", over)
    lp, _, _ = O.token_logprobs(b.H, b.W, b.ids, b.mask)
    old, ref = perturbed_logprobs(lp, b)
    valid = np.nonzero(b.mask.numpy())[0]
    r_nan = int(valid[len(valid) // 3])
    H1 = b.H.clone()
    H1[r_nan, 17] = float("nan")
    runs = {}
    for name, H in (("clean", b.H), ("nan", H1)):
        bb = synth.Batch(**{**b.__dict__, "H": H})
        print(f"[stress nan] {name}: separate calls", flush=True)
        gs = gpu_step(bb, old, ref)
        print(f"[stress nan] {name}: fused step", flush=True)
        gf = gpu_fused_step(bb, old, ref)
        runs[name] = (gs, gf)
    others = np.ones(b.T, dtype=bool)
    others[r_nan] = False
    for i, path in enumerate(("separate", "fused")):
        g0, g1 = runs["clean"][i], runs["nan"][i]
        for k in ("logp", "entropy", "lse"):
            assert math.isnan(g1[k][r_nan]), (path, k)
            assert np.array_equal(g0[k][others], g1[k][others]), (path, k)
        assert math.isnan(g1["stats"]["loss"]), path
        assert np.isnan(g1["dH"][r_nan]).any(), path
        # d_hidden is row-local: the other rows are unchanged too
        assert np.array_equal(g0["dH"][others], g1["dH"][others]), path
        # rows other than the NaN row keep their log-probs; their per-token
        # gradient depends only on their own row
        assert np.array_equal(g0["grad_logp"][others], g1["grad_logp"][others]), path


def test_nan_in_a_valid_logits_row():
    cfg = synth.config(4, n_prompts=4, group=8, V=5000)
    b = synth.make_batch(cfg, "cpu", seed_key=(4, 555))
    lp, _, _ = O.token_logprobs_from_logits(b.logits, b.ids, b.mask)
    old, ref = perturbed_logprobs(lp, b)
    valid = np.nonzero(b.mask.numpy())[0]
    r_nan = int(valid[7])
    L1 = b.logits.clone()
    L1[r_nan, 1234] = float("nan")
    tok = tokens_of(b)
    t = lambda x: torch.from_numpy(x).to(DEV)
    adv = R.rft_group_advantages(b.rewards.to(DEV), cfg.group)
    outs = []
    for L in (b.logits, L1):
        lpg, dl, st = R.rft_ppo_clip_fused_logits(tok, L.to(DEV), t(old), t(ref), adv,
                                                  params_of(cfg))
        torch.cuda.synchronize()
        outs.append((cpu(lpg), cpu(dl), R.stats_to_dict(st)))
    others = np.ones(b.T, dtype=bool)
    others[r_nan] = False
    assert math.isnan(outs[1][0][r_nan]) and math.isnan(outs[1][2]["loss"])
    assert np.array_equal(outs[0][0][others], outs[1][0][others])
    assert np.array_equal(outs[0][1][others], outs[1][1][others])


# ---------------------------------------------- mid-size multi-chunk step ----
def _ws_for_chunk(tok, d, V, rows):
    """Smallest workspace whose row chunk for the fused step is >= rows."""
    lo = R.workspace_bytes(R.RFT_OP_PPO_STEP, tok, d, V, R.RFT_BF16, minimum=True)
    hi = R.workspace_bytes(R.RFT_OP_PPO_STEP, tok, d, V, R.RFT_BF16)
    assert R.chunk_rows(R.RFT_OP_PPO_STEP, tok, d, V, R.RFT_BF16, hi) >= rows
    while hi - lo > 256:
        mid = (lo + hi) // 2 // 256 * 256
        if R.chunk_rows(R.RFT_OP_PPO_STEP, tok, d, V, R.RFT_BF16, mid) >= rows:
            hi = mid
        else:
            lo = mid
    return hi


MIDSIZE_CASES = [
    # d = 72: the forward on 256 x 256 tiles (a K tail), chunks of 16384 rows
    # (64 M-tiles: the full super-group of 8 x 8 tiles per XCD); d_hidden and
    # d_weight on 384 x 256 tiles (43 M-tiles of d_hidden: a full super-group
    # of 4 x 8 and a remainder)
    ("d72", dict(d=72, n_prompts=5, chunk=16384, store_tile="384")),
    # d = 128: the forward on 384 x 256 tiles, chunks of 24576 rows (64 M-tiles
    # of 384: its full super-group), 384-row tiles that start half way into a
    # 256-row panel and chunk ends inside a tile; d_hidden and d_weight on
    # 256 x 256 tiles (96 and 33 M-tiles)
    ("d128", dict(d=128, n_prompts=7, chunk=24576, store_tile="256")),
]


@pytest.mark.parametrize("name,case", MIDSIZE_CASES, ids=[c[0] for c in MIDSIZE_CASES])
def test_midsize_fused_step_full_tile_order(name, case, monkeypatch):
    """Row chunks that fill the forward's full super-group of tiles, V = 8292;
    three chunks, the last ragged; the backward GEMMs on the tile size the
    case names (RFT_GEMM_STORE_TILE).  Whole dH and dW against the oracle."""
    monkeypatch.setenv("RFT_GEMM_STORE_TILE", case["store_tile"])
    d, V, rows = case["d"], 8292, case["chunk"]
    over = dict(n_prompts=case["n_prompts"], group=8, len_lo=900, len_hi=1100, pad_to=1100, d=d,
                V=V, dtype="bf16")
    b = _batch(2, "midsize" if d == 72 else "midsize" + name, over)
    tok = tokens_of(b)
    N = int(b.mask.sum())
    ws = _ws_for_chunk(tok, d, V, rows)
    Tc = R.chunk_rows(R.RFT_OP_PPO_STEP, tok, d, V, R.RFT_BF16, ws)
    print(f"[stress midsize {name}] N={N} T={b.T} chunk={Tc} chunks={-(-N // Tc)}", flush=True)
    assert Tc == rows and N > 2 * Tc and N % Tc != 0     # three chunks, the last ragged
    lp, _, _ = O.token_logprobs(b.H, b.W, b.ids, b.mask)
    old, ref = perturbed_logprobs(lp, b)
    gf = gpu_fused_step(b, old, ref, ws_bytes=ws)
    print(f"[stress midsize {name}] oracle step", flush=True)
    o = oracle_step(b, old, ref)
    compare_step(gf, o, b)
    print(f"[stress midsize {name}] dH rel {rel_fro(gf['dH'], o['dH']):.2e} dW rel "
          f"{rel_fro(gf['dW'], o['dW']):.2e}", flush=True)
