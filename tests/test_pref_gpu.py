"""GPU parity of the train-only losses (SFT and DPO) against the float64
oracle: the loss kernels on synthetic log-probs (counts bit-exact, the fp64
pair sums to rounding), and the whole chain log-probs -> loss -> backward to
the hidden states and weight (bf16 MFMA path) or to given logits."""
import zlib

import numpy as np
import pytest
import torch

import paper_2505_17826_amd as R
from gen import synth
from oracle import rft_oracle as O
from tests.gpu_cases import (TOL_GRAD_FRO, TOL_LOGP, TOL_LOSS_ABS, TOL_LOSS_REL, cpu, f32,
                             rel_fro, requires_gpu, tokens_of)

pytestmark = [pytest.mark.gpu, requires_gpu]
DEV = torch.device("cuda")


def _t(x):
    return torch.from_numpy(np.ascontiguousarray(x)).to(DEV)


def _layout_case(seed, n_prompts=6, group=8, pad=160):
    cfg = synth.config(1, n_prompts=n_prompts, group=group, len_lo=0, len_hi=pad, pad_to=pad,
                       d=8, V=1000)
    b = synth.make_batch(cfg, "cpu", seed_key=(31, seed), layout_only=True)
    ss = b.seq_start.numpy()
    b.mask[int(ss[3]):int(ss[4])] = 0          # pair 1 has an empty rejected rollout
    rng = np.random.default_rng(seed)
    mk = b.mask.numpy() != 0
    T = b.T
    logp = np.where(mk, -rng.random(T) * 6, 0).astype(np.float32)
    ref = np.where(mk, logp + rng.standard_normal(T) * 0.3, 0).astype(np.float32)
    ids = b.ids.numpy().copy()
    bad = np.nonzero(mk)[0][[7, 400]]
    ids[bad[0]] = cfg.V
    ids[bad[1]] = -3
    b.ids = torch.from_numpy(ids)
    return cfg, b, logp, ref


@pytest.mark.parametrize("agg,denom", [(1, 0.0), (0, 0.0), (1, 5000.0)])
def test_sft_loss_kernel(agg, denom):
    cfg, b, logp, _ = _layout_case(41 + agg)
    tok = tokens_of(b)
    grad, st = R.rft_sft_loss_fwd(tok, cfg.V, _t(logp), agg=agg, denom_override=denom)
    torch.cuda.synchronize()
    s = R.stats_to_dict(st)
    o = O.sft_loss_fwd(logp, b.mask, b.seq_start, b.ids, cfg.V, agg=agg, denom_override=denom)
    for k in ("n_valid", "n_seq_valid", "n_bad_ids"):
        assert s[k] == o[k], (k, s[k], o[k])
    assert o["n_bad_ids"] == 2
    assert s["loss"] == pytest.approx(o["loss"], rel=1e-9)
    assert s["sft_loss"] == s["loss"]
    assert s["pg_loss"] == 0.0 and s["n_clipped"] == 0
    np.testing.assert_allclose(cpu(grad), o["grad_logp"], rtol=1e-6, atol=0)


@pytest.mark.parametrize("ls", [0.0, 0.1])
def test_dpo_loss_kernel(ls):
    """Pairs of unequal lengths, empty rollouts (pairs that do not count) and
    two bad ids."""
    cfg, b, logp, ref = _layout_case(43)
    n_i = np.array([int(b.mask[b.seq_start[i]:b.seq_start[i + 1]].sum())
                    for i in range(cfg.n_seq)])
    assert (n_i == 0).any(), "the layout should hold an empty rollout"
    tok = tokens_of(b)
    beta = 0.1
    grad, seq_lp, st = R.rft_dpo_loss_fwd(tok, cfg.V, _t(logp), _t(ref), beta=beta,
                                          label_smoothing=ls)
    torch.cuda.synchronize()
    s = R.stats_to_dict(st, R.rft_dpo_stats)
    o = O.dpo_loss_fwd(logp, ref, b.mask, b.seq_start, b.ids, cfg.V, beta=f32(beta),
                       label_smoothing=f32(ls))
    for k in ("n_pairs", "n_valid", "n_bad_ids"):
        assert s[k] == o[k], (k, s[k], o[k])
    assert o["n_pairs"] < cfg.n_seq // 2
    for k in ("loss", "chosen_reward", "rejected_reward", "margin_mean", "reward_acc"):
        assert s[k] == pytest.approx(o[k], rel=1e-9, abs=1e-12), (k, s[k], o[k])
    np.testing.assert_allclose(cpu(grad), o["grad_logp"], rtol=1e-6, atol=0)
    np.testing.assert_allclose(cpu(seq_lp), o["seq_logp"], rtol=1e-6, atol=1e-6)


def test_dpo_no_counted_pair_and_empty():
    """Every pair has an empty rollout: loss 0, every gradient 0; and a batch
    with no rows at all."""
    ss = torch.tensor([0, 3, 3, 3, 5], dtype=torch.int32)
    mask = torch.ones(5, dtype=torch.uint8)
    ids = torch.zeros(5, dtype=torch.int32)
    tok = R.Tokens(ss.to(DEV), mask.to(DEV), ids.to(DEV))
    lp = torch.full((5,), -1.0, device=DEV)
    grad, _, st = R.rft_dpo_loss_fwd(tok, 10, lp, lp * 0.5)
    s = R.stats_to_dict(st, R.rft_dpo_stats)
    assert s["n_pairs"] == 0 and s["loss"] == 0.0 and s["n_valid"] == 5
    assert torch.count_nonzero(grad).item() == 0
    e = torch.zeros(0, device=DEV)
    tok0 = R.Tokens(torch.zeros(3, dtype=torch.int32, device=DEV),
                    torch.zeros(0, dtype=torch.uint8, device=DEV),
                    torch.zeros(0, dtype=torch.int32, device=DEV))
    _, sl, st0 = R.rft_dpo_loss_fwd(tok0, 10, e, e)
    s0 = R.stats_to_dict(st0, R.rft_dpo_stats)
    assert s0["n_pairs"] == 0 and s0["loss"] == 0.0 and s0["n_valid"] == 0
    assert torch.all(sl == 0)


BF16_PREF = ("pref-3x8-d200-V4099", dict(n_prompts=3, group=8, len_lo=1, len_hi=300, pad_to=300,
                                         d=200, V=4099, dtype="bf16"))


def test_dpo_and_sft_chain_bf16():
    """log-probs (MFMA) -> DPO / SFT loss -> backward to hidden and weight."""
    name, over = BF16_PREF
    cfg = synth.config(1, **over)
    b = synth.make_batch(cfg, "cpu", seed_key=(1, zlib.crc32(name.encode()) % 100003))
    tok = tokens_of(b)
    H, W = b.H.to(DEV).contiguous(), b.W.to(DEV).contiguous()
    logp, ent, lse = R.rft_token_logprobs(tok, H, W)
    lp_o, _, lse_o = O.token_logprobs(b.H, b.W, b.ids, b.mask)
    m = b.mask.numpy() != 0
    assert np.abs(cpu(logp)[m] - lp_o[m]).max() <= TOL_LOGP
    ref = np.where(m, lp_o + b.ref_noise.numpy(), 0).astype(np.float32)
    beta = 0.2
    grad, _, st = R.rft_dpo_loss_fwd(tok, cfg.V, logp, _t(ref), beta=beta)
    dH, dW = R.rft_ppo_clip_loss_bwd(tok, H, W, lse, grad)
    torch.cuda.synchronize()
    s = R.stats_to_dict(st, R.rft_dpo_stats)
    o = O.dpo_loss_fwd(lp_o, ref, b.mask, b.seq_start, b.ids, cfg.V, beta=f32(beta))
    assert s["n_pairs"] == o["n_pairs"] and s["n_valid"] == o["n_valid"]
    assert abs(s["loss"] - o["loss"]) <= TOL_LOSS_REL * abs(o["loss"]) + TOL_LOSS_ABS
    dH_o, dW_o = O.ppo_clip_loss_bwd(b.H, b.W, lse_o, o["grad_logp"], b.ids, b.mask)
    assert rel_fro(cpu(dH), dH_o) <= TOL_GRAD_FRO
    assert rel_fro(cpu(dW), dW_o) <= TOL_GRAD_FRO
    # SFT through the same chain
    g2, st2 = R.rft_sft_loss_fwd(tok, cfg.V, logp, agg=R.RFT_AGG_SEQ_MEAN_TOKEN_MEAN)
    dH2, dW2 = R.rft_ppo_clip_loss_bwd(tok, H, W, lse, g2)
    torch.cuda.synchronize()
    o2 = O.sft_loss_fwd(lp_o, b.mask, b.seq_start, b.ids, cfg.V, agg=O.AGG_SEQ_MEAN_TOKEN_MEAN)
    s2 = R.stats_to_dict(st2)
    assert abs(s2["loss"] - o2["loss"]) <= TOL_LOSS_REL * abs(o2["loss"]) + TOL_LOSS_ABS
    dH2_o, dW2_o = O.ppo_clip_loss_bwd(b.H, b.W, lse_o, o2["grad_logp"], b.ids, b.mask)
    assert rel_fro(cpu(dH2), dH2_o) <= TOL_GRAD_FRO
    assert rel_fro(cpu(dW2), dW2_o) <= TOL_GRAD_FRO


def test_dpo_loss_only_logits():
    """From given fp32 logits: statistics -> DPO loss -> d_logits."""
    cfg = synth.config(4, n_prompts=4, group=8, V=8192)
    b = synth.make_batch(cfg, "cpu", seed_key=(4, 55))
    tok = tokens_of(b)
    logits = b.logits.to(DEV)
    lp, _, lse, _ = R.rft_token_logprobs_from_logits(tok, logits)
    lp_o, _, lse_o = O.token_logprobs_from_logits(b.logits, b.ids, b.mask)
    m = b.mask.numpy() != 0
    ref = np.where(m, lp_o + b.ref_noise.numpy(), 0).astype(np.float32)
    grad, _, st = R.rft_dpo_loss_fwd(tok, cfg.V, lp, _t(ref), beta=0.5, label_smoothing=0.05)
    dl = R.rft_ppo_clip_loss_bwd_logits(tok, logits, lse, grad)
    torch.cuda.synchronize()
    o = O.dpo_loss_fwd(lp_o, ref, b.mask, b.seq_start, b.ids, cfg.V, beta=0.5,
                       label_smoothing=f32(0.05))
    s = R.stats_to_dict(st, R.rft_dpo_stats)
    assert abs(s["loss"] - o["loss"]) <= TOL_LOSS_REL * abs(o["loss"]) + TOL_LOSS_ABS
    dl_o = np.zeros(b.logits.shape)
    for r_, v in O.bwd_logits(b.logits, lse_o, o["grad_logp"], b.ids, b.mask).items():
        dl_o[r_] = v
    assert rel_fro(cpu(dl), dl_o) <= TOL_GRAD_FRO
