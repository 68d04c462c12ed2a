"""GPU parity of the advantage variants over explicit, variable-size groups
(failed, skipped or lagged rollouts leave groups smaller) against the float64
oracle, and of micro-batch gradient accumulation through denom_override
(two calls on halves of a batch, the weight gradient accumulated, equal the
whole batch)."""
import zlib

import numpy as np
import pytest
import torch

import paper_2505_17826_amd as R
from gen import synth
from oracle import rft_oracle as O
from tests.gpu_cases import (TOL_ADV, TOL_GRAD_FRO, TOL_LOSS_ABS, TOL_LOSS_REL, cpu, f32,
                             oracle_eps, params_of, perturbed_logprobs, rel_fro, requires_gpu)

pytestmark = [pytest.mark.gpu, requires_gpu]
DEV = torch.device("cuda")


def _t(x):
    return torch.from_numpy(np.ascontiguousarray(x)).to(DEV)


@pytest.mark.parametrize("mode", [R.RFT_ADV_GRPO, R.RFT_ADV_MEAN_CENTER, R.RFT_ADV_LEAVE_ONE_OUT])
@pytest.mark.parametrize("n,n_groups", [(1000, 97), (65536, 8192), (5, 1)])
def test_advantages_ids(mode, n, n_groups):
    rng = np.random.default_rng(n + mode)
    r = rng.random(n).astype(np.float32)
    r[rng.random(n) < 0.3] = 1.0                       # ties, and some all-equal groups
    gid = rng.integers(-1, n_groups + 2, size=n).astype(np.int32)   # some left out
    print(f"[adv ids] mode={mode} n={n} groups={n_groups}", flush=True)
    a = R.rft_group_advantages_ids(_t(r), _t(gid), n_groups, mode, eps=1e-6)
    o = O.group_advantages_ids(r, gid, mode, f32(1e-6), n_groups=n_groups)
    np.testing.assert_allclose(cpu(a), o, atol=TOL_ADV, rtol=0)
    if mode == R.RFT_ADV_GRPO:
        a0 = R.rft_group_advantages_ids(_t(r), _t(gid), n_groups, mode, eps=1e-6, unbiased=False)
        o0 = O.group_advantages_ids(r, gid, mode, f32(1e-6), n_groups=n_groups, unbiased=False)
        np.testing.assert_allclose(cpu(a0), o0, atol=TOL_ADV, rtol=0)
    ga = cpu(a)
    out = (gid < 0) | (gid >= n_groups)
    assert np.all(ga[out] == 0.0)


def test_advantages_ids_contiguous_matches_fixed_groups():
    rng = np.random.default_rng(5)
    G, ng = 8, 256
    r = (rng.random(G * ng) < 0.4).astype(np.float32)
    gid = np.repeat(np.arange(ng, dtype=np.int32), G)
    a = R.rft_group_advantages_ids(_t(r), _t(gid), ng, R.RFT_ADV_GRPO)
    b = R.rft_group_advantages(_t(r), G)
    np.testing.assert_allclose(cpu(a), cpu(b), atol=2e-7, rtol=0)
    z = torch.zeros(0, device=DEV)
    R.rft_group_advantages_ids(z, torch.zeros(0, dtype=torch.int32, device=DEV), 0)


def _slice_batch(b, lo, hi):
    """Rollouts [lo, hi) of a batch as a batch of their own."""
    ss = b.seq_start.numpy()
    r0, r1 = int(ss[lo]), int(ss[hi])
    cut = lambda x: None if x is None else x[r0:r1]
    nb = synth.Batch(cfg=b.cfg, seq_start=torch.from_numpy((ss[lo:hi + 1] - r0).astype(np.int32)),
                     mask=cut(b.mask), lengths=b.lengths[lo:hi], ids=cut(b.ids),
                     rewards=b.rewards[lo:hi], old_noise=cut(b.old_noise),
                     ref_noise=cut(b.ref_noise), H=cut(b.H), W=b.W)
    return nb, r0, r1


@pytest.mark.parametrize("agg", [0, 1])
def test_microbatch_accumulation_with_denom_override(agg):
    """Whole GRPO groups split over two calls of the fused step: with the
    global S (or N) passed as denom_override and dW accumulated, the two
    halves give the whole batch's loss, dH and dW."""
    over = dict(n_prompts=4, group=8, len_lo=1, len_hi=200, pad_to=200, d=128, V=3001,
                dtype="bf16", agg=agg)
    cfg = synth.config(1, **over)
    b = synth.make_batch(cfg, "cpu", seed_key=(1, zlib.crc32(b"micro") % 100003 + agg))
    lp, _, _ = O.token_logprobs(b.H, b.W, b.ids, b.mask)
    old, ref = perturbed_logprobs(lp, b)
    el, eh, be = oracle_eps(cfg)
    o = O.trainer_step(b.H, b.W, b.ids, b.mask, b.seq_start, b.rewards, cfg.group,
                       old.astype(np.float64), ref.astype(np.float64), el, eh, be, agg)
    cnt = O.token_counts(b.mask, b.seq_start)
    denom = float(cnt["S"] if agg == 0 else cnt["N"])
    adv = R.rft_group_advantages(b.rewards.to(DEV), cfg.group)   # on the whole batch
    W = b.W.to(DEV).contiguous()
    dW = torch.empty(W.shape, dtype=torch.float32, device=DEV)
    dH = np.zeros(o["dH"].shape)
    loss = 0.0
    half = cfg.n_seq // 2                                           # a group boundary
    for k, (lo, hi) in enumerate(((0, half), (half, cfg.n_seq))):
        mb, r0, r1 = _slice_batch(b, lo, hi)
        tok = R.Tokens(mb.seq_start.to(DEV), mb.mask.to(DEV).contiguous(),
                       mb.ids.to(DEV).contiguous())
        out = R.rft_ppo_clip_step(tok, mb.H.to(DEV).contiguous(), W, _t(old[r0:r1]),
                                  _t(ref[r0:r1]), adv[lo:hi].contiguous(),
                                  params_of(cfg, denom=denom, agg=agg), d_weight=dW,
                                  accumulate_dw=k > 0)
        torch.cuda.synchronize()
        dH[r0:r1] = cpu(out[4])
        loss += R.stats_to_dict(out[6])["loss"]
    assert abs(loss - o["fwd"]["loss"]) <= TOL_LOSS_REL * abs(o["fwd"]["loss"]) + TOL_LOSS_ABS
    assert rel_fro(dH, o["dH"]) <= TOL_GRAD_FRO
    assert rel_fro(cpu(dW), o["dW"]) <= TOL_GRAD_FRO


def test_advantages_ids_million_rollouts_linear_and_deterministic():
    """1e6 rollouts in 117,501 groups of 8, 300 and 20000 members, shuffled,
    5% left out: the sort-by-group path (both per-group sort sizes and the
    scan for a group beyond the sort) against the oracle, the same bits on a
    second run, and a run time of milliseconds (work linear in n)."""
    rng = np.random.default_rng(1234)
    n = 1_000_000
    sizes = [20000] + [300] * 100 + [8] * 117400
    gid = np.repeat(np.arange(len(sizes), dtype=np.int32), sizes)
    assert gid.size == 20000 + 30000 + 939200
    gid = np.concatenate([gid, np.full(n - gid.size, -1, np.int32)])   # left out
    gid = gid[rng.permutation(n)]
    n_groups = len(sizes)
    r = rng.random(n).astype(np.float32)
    r[rng.random(n) < 0.2] = 0.5
    rt, gt = _t(r), _t(gid)
    ws = torch.empty(int(R.lib().rft_group_advantages_ids_workspace_bytes(n, n_groups)),
                     dtype=torch.uint8, device=DEV)
    a1 = R.rft_group_advantages_ids(rt, gt, n_groups, R.RFT_ADV_GRPO, ws=ws)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    a2 = R.rft_group_advantages_ids(rt, gt, n_groups, R.RFT_ADV_GRPO, ws=ws)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1)
    print(f"[adv ids] n={n} groups={n_groups}: {ms:.3f} ms", flush=True)
    assert torch.equal(a1, a2)
    assert ms < 20.0
    o = O.group_advantages_ids(r, gid, R.RFT_ADV_GRPO, f32(1e-6), n_groups=n_groups)
    np.testing.assert_allclose(cpu(a1), o, atol=TOL_ADV, rtol=0)
    for mode in (R.RFT_ADV_MEAN_CENTER, R.RFT_ADV_LEAVE_ONE_OUT):
        a = R.rft_group_advantages_ids(rt, gt, n_groups, mode, ws=ws)
        o = O.group_advantages_ids(r, gid, mode, f32(1e-6), n_groups=n_groups)
        np.testing.assert_allclose(cpu(a), o, atol=TOL_ADV, rtol=0)
