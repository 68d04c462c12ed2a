"""GPU parity of the entropy bonus (loss - c_H sum_t w_t H_t, with its
gradient through the entropy into the logits) against the float64 oracle:
the loss kernel, the separate calls (bf16 and fp32), the fused step, the
loss-only paths, and cases where the bonus is the only term, so that the
backward's entropy part is checked on its own."""
import zlib

import numpy as np
import pytest
import torch

import paper_2505_17826_amd as R
from gen import synth
from oracle import rft_oracle as O
from tests.gpu_cases import (TOL_GRAD_FRO, TOL_LOSS_ABS, TOL_LOSS_REL, compare_step, cpu, f32,
                             gpu_fused_step, gpu_step, oracle_eps, oracle_step, params_of,
                             perturbed_logprobs, rel_fro, requires_gpu, tokens_of)

pytestmark = [pytest.mark.gpu, requires_gpu]
DEV = torch.device("cuda")


def _t(x):
    return torch.from_numpy(np.ascontiguousarray(x)).to(DEV)


@pytest.mark.parametrize("agg,mix", [(0, False), (1, False), (0, True)])
def test_entropy_loss_kernel(agg, mix):
    """The loss kernel on synthetic fp32 log-probs and entropies: loss,
    entropy_loss and both per-token gradients against the oracle."""
    cfg = synth.config(1, n_prompts=8, group=8, len_lo=1, len_hi=200, pad_to=200, d=8, V=1000,
                       agg=agg)
    b = synth.make_batch(cfg, "cpu", seed_key=(12, agg, int(mix)), layout_only=True)
    rng = np.random.default_rng(8)
    T = b.T
    mk = b.mask.numpy() != 0
    logp = np.where(mk, -rng.random(T) * 9, 0).astype(np.float32)
    old = np.where(mk, logp + rng.standard_normal(T) * 0.3, 0).astype(np.float32)
    ref = np.where(mk, logp + rng.standard_normal(T) * 0.2, 0).astype(np.float32)
    ent = np.where(mk, rng.random(T) * 5, 0).astype(np.float32)
    ex = (np.arange(cfg.n_seq) % 3 == 1).astype(np.uint8) if mix else None
    mu, coef = (0.2 if mix else 0.0), 0.03
    advd = O.group_advantages(b.rewards.numpy(), cfg.group).astype(np.float32)
    tok = tokens_of(b, ex)
    eg = torch.empty(T, dtype=torch.float32, device=DEV)
    grad, st = R.rft_ppo_clip_loss_fwd(tok, cfg.V, _t(logp), _t(old), _t(ref), _t(advd),
                                       params_of(cfg, mix_mu=mu, ent=coef), entropy=_t(ent),
                                       grad_entropy=eg)
    torch.cuda.synchronize()
    s = R.stats_to_dict(st)
    el, eh, be = oracle_eps(cfg)
    o = O.ppo_clip_loss_fwd(logp, old, ref, advd, b.mask, b.seq_start, b.ids, cfg.V, el, eh, be,
                            agg, entropy=ent, is_expert=ex, mix_mu=f32(mu),
                            entropy_coef=f32(coef))
    for k in ("n_valid", "n_clipped", "n_expert", "n_bad_ids"):
        assert s[k] == o[k], (k, s[k], o[k])
    for k in ("loss", "entropy_loss", "pg_loss", "sft_loss"):
        assert abs(s[k] - o[k]) <= TOL_LOSS_REL * abs(o[k]) + TOL_LOSS_ABS, (k, s[k], o[k])
    np.testing.assert_allclose(cpu(eg), o["grad_entropy"], rtol=1e-6, atol=0)
    np.testing.assert_allclose(cpu(grad), o["grad_logp"], rtol=1e-4,
                               atol=1e-7 * np.abs(o["grad_logp"]).max())
    # entropy_coef = 0: entropy_loss is still reported, the loss carries no
    # bonus (which enters the MIX loss scaled by 1 - mu)
    grad0, st0 = R.rft_ppo_clip_loss_fwd(tok, cfg.V, _t(logp), _t(old), _t(ref), _t(advd),
                                         params_of(cfg, mix_mu=mu), entropy=_t(ent))
    s0 = R.stats_to_dict(st0)
    assert s0["entropy_loss"] == s["entropy_loss"]
    bonus = (1.0 - f32(mu)) * f32(coef) * s["entropy_loss"]
    assert s0["loss"] == pytest.approx(s["loss"] + bonus, rel=1e-9, abs=1e-12)
    assert torch.equal(grad0, grad)


BF16_ENT = ("ent-2x8-d200-V4099", dict(n_prompts=2, group=8, len_lo=1, len_hi=300, pad_to=300,
                                       d=200, V=4099, dtype="bf16"))
F32_ENT = ("ent-f32-3x8-d72-V1000", dict(n_prompts=3, group=8, len_lo=1, len_hi=90, pad_to=90,
                                         d=72, V=1000, dtype="f32"))


def _batch(name, over, **cfg_over):
    cfg = synth.config(1, **over, **cfg_over)
    return synth.make_batch(cfg, "cpu", seed_key=(1, zlib.crc32(name.encode()) % 100003))


@pytest.mark.parametrize("case", [BF16_ENT, F32_ENT], ids=["bf16", "f32"])
@pytest.mark.parametrize("mix", [False, True])
def test_entropy_step_separate_and_fused(case, mix):
    name, over = case
    b = _batch(name, over)
    print(f"[entropy step] {name} mix={mix}", flush=True)
    lp, _, _ = O.token_logprobs(b.H, b.W, b.ids, b.mask)
    old, ref = perturbed_logprobs(lp, b)
    ex = (np.arange(b.cfg.n_seq) % 4 == 1).astype(np.uint8) if mix else None
    kw = dict(is_expert=ex, mu=0.1 if mix else 0.0, ent_coef=0.05)
    o = oracle_step(b, old, ref, **kw)
    gs = gpu_step(b, old, ref, **kw)
    compare_step(gs, o, b)
    gf = gpu_fused_step(b, old, ref, **kw)
    compare_step(gf, o, b)
    for k in ("logp", "entropy", "grad_logp"):
        assert np.array_equal(gf[k], gs[k], equal_nan=True), k
    for k in ("loss", "entropy_loss"):
        assert gf["stats"][k] == gs["stats"][k], k


@pytest.mark.parametrize("case", [BF16_ENT, F32_ENT], ids=["bf16", "f32"])
def test_entropy_only_backward(case):
    """Equal rewards in every group (advantages 0) and no KL: the entropy bonus
    is the whole gradient, so dH and dW check its backward alone."""
    name, over = case
    b = _batch(name + "-only", over, beta=0.0)
    b.rewards = torch.ones_like(b.rewards)
    lp, _, _ = O.token_logprobs(b.H, b.W, b.ids, b.mask)
    old, ref = perturbed_logprobs(lp, b)
    o = oracle_step(b, old, ref, ent_coef=1.0)
    assert np.all(o["fwd"]["grad_logp"] == 0) and np.linalg.norm(o["dW"]) > 0
    for g in (gpu_step(b, old, ref, ent_coef=1.0), gpu_fused_step(b, old, ref, ent_coef=1.0)):
        assert np.all(g["grad_logp"] == 0)
        compare_step(g, o, b)


def test_entropy_loss_only_paths():
    """Loss-only from fp32 logits: the fused one-pass kernel, and the separate
    statistics / loss / d_logits calls, with the bonus as the dominant term."""
    cfg = synth.config(4, n_prompts=4, group=8, V=8192)
    b = synth.make_batch(cfg, "cpu", seed_key=(4, 77))
    lp, _, _ = O.token_logprobs_from_logits(b.logits, b.ids, b.mask)
    old, ref = perturbed_logprobs(lp, b)
    el, eh, be = oracle_eps(cfg)
    coef = 0.5
    o = O.loss_only_step(b.logits, b.ids, b.mask, b.seq_start, b.rewards, cfg.group,
                         old.astype(np.float64), ref.astype(np.float64), el, eh, be, cfg.agg,
                         entropy_coef=f32(coef))
    dl_o = np.zeros(b.logits.shape)
    for r_, v in o["dlogits"].items():
        dl_o[r_] = v
    tok = tokens_of(b)
    adv = R.rft_group_advantages(b.rewards.to(DEV), cfg.group)
    logits = b.logits.to(DEV)
    p = params_of(cfg, ent=coef)
    lpg, dl, st = R.rft_ppo_clip_fused_logits(tok, logits, _t(old), _t(ref), adv, p)
    torch.cuda.synchronize()
    s = R.stats_to_dict(st)
    for k in ("loss", "entropy_loss"):
        assert abs(s[k] - o["fwd"][k]) <= TOL_LOSS_REL * abs(o["fwd"][k]) + TOL_LOSS_ABS, k
    assert rel_fro(cpu(dl), dl_o) <= TOL_GRAD_FRO
    # separate calls
    lp2, ent2, lse2, _ = R.rft_token_logprobs_from_logits(tok, logits)
    eg = torch.empty_like(lp2)
    grad, st2 = R.rft_ppo_clip_loss_fwd(tok, cfg.V, lp2, _t(old), _t(ref), adv, p, entropy=ent2,
                                        grad_entropy=eg)
    dl2 = R.rft_ppo_clip_loss_bwd_logits(tok, logits, lse2, grad, grad_entropy=eg, entropy=ent2)
    torch.cuda.synchronize()
    assert rel_fro(cpu(dl2), dl_o) <= TOL_GRAD_FRO
    np.testing.assert_allclose(cpu(eg), o["fwd"]["grad_entropy"], rtol=1e-6, atol=0)
    s2 = R.stats_to_dict(st2)
    assert abs(s2["loss"] - o["fwd"]["loss"]) <= TOL_LOSS_REL * abs(o["fwd"]["loss"]) + TOL_LOSS_ABS
    # the two paths agree far inside the tolerance
    assert rel_fro(cpu(dl), cpu(dl2)) <= 1e-5


def _mask_vocab(logits, ids, mask, seed):
    """Set vocabulary entries to -inf (masked), never the sampled id: row
    kinds by index mod 3: 30% of the entries at random; all but a window of
    64 entries (most threads then see only -inf); none."""
    z = logits.numpy().copy()
    rng = np.random.default_rng(seed)
    T, V = z.shape
    for t in range(T):
        if t % 3 == 0:
            z[t, rng.random(V) < 0.3] = -np.inf
        elif t % 3 == 1:
            w0 = int(rng.integers(0, V - 64))
            keep = z[t, w0:w0 + 64].copy()
            z[t, :] = -np.inf
            z[t, w0:w0 + 64] = keep
        y = int(ids[t])
        if mask[t] and 0 <= y < V:
            z[t, y] = float(logits[t, y])
    return torch.from_numpy(z)


@pytest.mark.parametrize("V,group", [(8192, 8), (8190, 8), (160000, 2)])
def test_masked_vocabulary_logits(V, group):
    """Loss-only paths on logits with -inf entries (reading R15): fused and
    separate calls against the oracle, no NaN anywhere, and d_logits exactly
    0 in the masked columns.  V = 8190 takes the scalar path, V = 160000
    exceeds the on-chip row cache."""
    cfg = synth.config(4, n_prompts=1, group=group, V=V)
    b = synth.make_batch(cfg, "cpu", seed_key=(4, 151, V))
    zm = _mask_vocab(b.logits, b.ids.numpy(), b.mask.numpy(), V)
    lp, _, _ = O.token_logprobs_from_logits(zm, b.ids, b.mask)
    old, ref = perturbed_logprobs(lp, b)
    el, eh, be = oracle_eps(cfg)
    coef = 0.5
    print(f"[masked vocab] V={V} T={b.T}", flush=True)
    o = O.loss_only_step(zm, b.ids, b.mask, b.seq_start, b.rewards, cfg.group,
                         old.astype(np.float64), ref.astype(np.float64), el, eh, be, cfg.agg,
                         entropy_coef=f32(coef))
    dl_o = np.zeros(zm.shape)
    for r_, v in o["dlogits"].items():
        dl_o[r_] = v
    masked = ~np.isfinite(zm.numpy())
    assert masked.any() and np.all(dl_o[masked] == 0)
    tok = tokens_of(b)
    adv = R.rft_group_advantages(b.rewards.to(DEV), cfg.group)
    logits = zm.to(DEV)
    p = params_of(cfg, ent=coef)
    ent_f = torch.empty(b.T, device=DEV)
    lpg, dl, st = R.rft_ppo_clip_fused_logits(tok, logits, _t(old), _t(ref), adv, p,
                                              entropy=ent_f)
    lp2, ent2, lse2, _ = R.rft_token_logprobs_from_logits(tok, logits)
    eg = torch.empty_like(lp2)
    grad, st2 = R.rft_ppo_clip_loss_fwd(tok, cfg.V, lp2, _t(old), _t(ref), adv, p, entropy=ent2,
                                        grad_entropy=eg)
    dl2 = R.rft_ppo_clip_loss_bwd_logits(tok, logits, lse2, grad, grad_entropy=eg, entropy=ent2)
    torch.cuda.synchronize()
    mk = b.mask.numpy() != 0
    lp_o, ent_o, lse_o = O.token_logprobs_from_logits(zm, b.ids, b.mask)
    for name, g in (("fused", dl), ("separate", dl2)):
        gd = cpu(g)
        assert np.all(np.isfinite(gd)), name
        assert np.all(gd[masked] == 0.0), name
        assert rel_fro(gd, dl_o) <= TOL_GRAD_FRO, name
    for x, ref_ in ((lpg, lp_o), (lp2, lp_o), (ent_f, ent_o), (ent2, ent_o), (lse2, lse_o)):
        xv = cpu(x)
        assert np.all(np.isfinite(xv[mk]))
        np.testing.assert_allclose(xv[mk], ref_[mk], rtol=0, atol=2e-3)
    for s in (R.stats_to_dict(st), R.stats_to_dict(st2)):
        for k in ("loss", "entropy_loss"):
            assert abs(s[k] - o["fwd"][k]) <= TOL_LOSS_REL * abs(o["fwd"][k]) + TOL_LOSS_ABS, k
