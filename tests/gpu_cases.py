"""Shared helpers of the GPU parity tests: run the HIP path through the C ABI
binding and the float64 oracle on the same seeded inputs."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import paper_2505_17826_amd as R
from gen import synth
from oracle import rft_oracle as O

requires_gpu = pytest.mark.skipif(not torch.cuda.is_available(), reason="needs an MI355X")

# tolerances (the required bars, plus the derived ones)
TOL_LOGP = 2e-3          # absolute, log-probs (also entropy and lse)
TOL_LOSS_REL = 1e-3      # relative, loss ...
TOL_LOSS_ABS = 1e-6      # ... with an absolute floor (zero-mean advantages cancel)
TOL_GRAD_FRO = 2e-2      # relative Frobenius, dH / dW / dlogits
TOL_ADV = 1e-5           # absolute, advantages


def f32(x):
    return float(np.float32(x))


def rel_fro(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    nb = np.linalg.norm(b)
    return np.linalg.norm(a - b) / (nb if nb > 0 else 1.0)


def cpu(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def tokens_of(b: synth.Batch, is_expert=None) -> R.Tokens:
    dev = torch.device("cuda")
    ex = None if is_expert is None else torch.from_numpy(np.asarray(is_expert, np.uint8)).to(dev)
    return R.Tokens(b.seq_start.to(dev).contiguous(), b.mask.to(dev).contiguous(),
                    b.ids.to(dev).contiguous(), ex)


def params_of(cfg: synth.Config, denom=0.0, agg=None, mix_mu=0.0, ent=0.0) -> R.rft_ppo_params:
    return R.ppo_params(cfg.eps_low, cfg.eps_high, cfg.beta, cfg.agg if agg is None else agg, denom,
                        mix_mu, ent)


def oracle_eps(cfg):
    """The float32 values the library receives, as the oracle's fp64 inputs."""
    return f32(cfg.eps_low), f32(cfg.eps_high), f32(cfg.beta)


def near_bound(logp, old, eps_low, eps_high):
    """Relative distance of rho = exp(logp - old) (fp64) from the nearer clip
    bound 1 - eps_low or 1 + eps_high (inf where a bound cannot be reached)."""
    rho = np.exp(np.asarray(logp, np.float64) - np.asarray(old, np.float64))
    hi, lo = 1.0 + eps_high, 1.0 - eps_low
    d_hi = np.abs(rho / hi - 1.0) if np.isfinite(hi) else np.full(rho.shape, np.inf)
    d_lo = np.abs(rho / lo - 1.0) if lo > 0 else np.full(rho.shape, np.inf)
    return np.minimum(d_hi, d_lo)


def perturbed_logprobs(logp_fp64, batch: synth.Batch):
    """Old / reference log-probs = given log-probs + the batch's noise, as fp32."""
    m = batch.mask.cpu().numpy() != 0
    old = np.where(m, logp_fp64 + batch.old_noise.cpu().numpy(), 0.0).astype(np.float32)
    ref = np.where(m, logp_fp64 + batch.ref_noise.cpu().numpy(), 0.0).astype(np.float32)
    return old, ref


def gpu_step(b: synth.Batch, old32, ref32, denom=0.0, ws_bwd_bytes=None, is_expert=None, mu=0.0,
             ent_coef=0.0):
    """adv -> log-probs -> loss -> backward through the binding; CPU results."""
    dev = torch.device("cuda")
    cfg = b.cfg
    tok = tokens_of(b, is_expert)
    H, W = b.H.to(dev).contiguous(), b.W.to(dev).contiguous()
    adv = R.rft_group_advantages(b.rewards.to(dev), cfg.group)
    logp, ent, lse = R.rft_token_logprobs(tok, H, W)
    old = torch.from_numpy(old32).to(dev)
    ref = torch.from_numpy(ref32).to(dev)
    egrad = torch.empty_like(logp) if ent_coef > 0 else None
    grad, st = R.rft_ppo_clip_loss_fwd(tok, cfg.V, logp, old, ref, adv,
                                       params_of(cfg, denom, mix_mu=mu, ent=ent_coef), entropy=ent,
                                       grad_entropy=egrad)
    ws = None
    if ws_bwd_bytes is not None:
        ws = torch.empty(ws_bwd_bytes, dtype=torch.uint8, device=dev)
    dH, dW = R.rft_ppo_clip_loss_bwd(tok, H, W, lse, grad, ws=ws, grad_entropy=egrad,
                                     entropy=ent if egrad is not None else None)
    torch.cuda.synchronize()
    out = {"adv": cpu(adv), "logp": cpu(logp), "entropy": cpu(ent), "lse": cpu(lse),
           "grad_logp": cpu(grad), "stats": R.stats_to_dict(st), "dH": cpu(dH), "dW": cpu(dW)}
    if egrad is not None:
        out["grad_entropy"] = cpu(egrad)
    return out


def gpu_fused_step(b: synth.Batch, old32, ref32, denom=0.0, ws_bytes=None, dW_init=None,
                   is_expert=None, mu=0.0, ent_coef=0.0):
    """adv -> rft_ppo_clip_step (the whole step in one call); CPU results."""
    dev = torch.device("cuda")
    cfg = b.cfg
    tok = tokens_of(b, is_expert)
    H, W = b.H.to(dev).contiguous(), b.W.to(dev).contiguous()
    adv = R.rft_group_advantages(b.rewards.to(dev), cfg.group)
    old = torch.from_numpy(old32).to(dev)
    ref = torch.from_numpy(ref32).to(dev)
    ws = None
    if ws_bytes is not None:
        ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    dW = None if dW_init is None else torch.from_numpy(dW_init).to(dev)
    logp, ent, lse, grad, dH, dW, st = R.rft_ppo_clip_step(
        tok, H, W, old, ref, adv, params_of(cfg, denom, mix_mu=mu, ent=ent_coef), d_weight=dW,
        accumulate_dw=dW_init is not None, ws=ws)
    torch.cuda.synchronize()
    return {"adv": cpu(adv), "logp": cpu(logp), "entropy": cpu(ent), "lse": cpu(lse),
            "grad_logp": cpu(grad), "stats": R.stats_to_dict(st), "dH": cpu(dH), "dW": cpu(dW)}


def oracle_step(b: synth.Batch, old32, ref32, denom=0.0, is_expert=None, mu=0.0, ent_coef=0.0):
    cfg = b.cfg
    el, eh, be = oracle_eps(cfg)
    return O.trainer_step(b.H, b.W, b.ids, b.mask, b.seq_start, b.rewards, cfg.group,
                          old32.astype(np.float64), ref32.astype(np.float64), el, eh, be, cfg.agg,
                          denom, is_expert=is_expert, mix_mu=f32(mu), entropy_coef=f32(ent_coef))


def compare_stats(st, of, n_near=0):
    """Every loss statistic of the library against the oracle's.  The
    per-token log-probs may differ by TOL_LOGP, so the means over tokens of
    kl, ratio and entropy are held to that (absolute; relative for the
    ratio); the weighted sums like the loss; the clip fraction may differ by
    the tokens near a bound (n_near)."""
    assert st["n_bad_ids"] == of["n_bad_ids"], (st["n_bad_ids"], of["n_bad_ids"])
    assert st["n_valid"] == of["n_valid"] and st["n_seq_valid"] == of["n_seq_valid"]
    for k in ("loss", "pg_loss", "kl_loss", "entropy_loss", "sft_loss"):
        assert abs(st[k] - of[k]) <= TOL_LOSS_REL * abs(of[k]) + TOL_LOSS_ABS, (k, st[k], of[k])
    for k in ("kl_mean", "entropy_mean"):
        assert abs(st[k] - of[k]) <= TOL_LOGP, (k, st[k], of[k])
    assert abs(st["ratio_mean"] - of["ratio_mean"]) <= TOL_LOGP * max(abs(of["ratio_mean"]), 1e-30) \
        + 1e-12, (st["ratio_mean"], of["ratio_mean"])
    assert abs(st["n_clipped"] - of["n_clipped"]) <= n_near, (st["n_clipped"], of["n_clipped"])
    n_pol = of["n_valid"] - of.get("n_expert", 0)
    if n_pol > 0:
        assert abs(st["clipfrac"] - of["clipfrac"]) <= n_near / n_pol + 1e-12, \
            (st["clipfrac"], of["clipfrac"])


def compare_step(g, o, b: synth.Batch, check_bwd=True):
    m = b.mask.cpu().numpy() != 0
    np.testing.assert_allclose(g["adv"], o["adv"], atol=TOL_ADV, rtol=0)
    for k in ("logp", "entropy", "lse"):
        assert np.all(g[k][~m] == 0.0), f"{k}: masked rows must be exactly 0"
        # a valid row with an out-of-range id has a NaN log-prob on both sides
        gn, on = np.isnan(g[k][m]), np.isnan(o[k][m])
        assert np.array_equal(gn, on), f"{k}: NaN rows differ"
        err = np.abs(g[k][m][~on] - o[k][m][~on]).max() if (~on).any() else 0.0
        assert err <= TOL_LOGP, f"{k}: max abs err {err}"
    st, of = g["stats"], o["fwd"]
    assert st["n_valid"] == of["n_valid"] and st["n_seq_valid"] == of["n_seq_valid"]
    assert abs(st["loss"] - of["loss"]) <= TOL_LOSS_REL * abs(of["loss"]) + TOL_LOSS_ABS, \
        (st["loss"], of["loss"])
    assert np.all(g["grad_logp"][~m] == 0.0)
    # per-token gradient, leaving out tokens within 1e-4 of a clip bound
    # (there the two sides may take different, equally valid branches)
    rows = of["weights_rows"]
    keep = of["margin"] >= 1e-4
    gr, orr = g["grad_logp"][rows][keep], of["grad_logp"][rows][keep]
    scale = np.abs(orr).max() if orr.size else 0.0
    bad = np.abs(gr - orr) > 1e-3 * np.abs(orr) + 1e-7 * scale
    assert not bad.any(), f"grad_logp: {bad.sum()} tokens off"
    assert abs(st["n_clipped"] - of["n_clipped"]) <= int((~keep).sum())
    compare_stats(st, of, n_near=int((~keep).sum()))
    assert st["n_expert"] == of["n_expert"]
    assert abs(st["sft_loss"] - of["sft_loss"]) <= TOL_LOSS_REL * abs(of["sft_loss"]) + TOL_LOSS_ABS
    ent_l = of.get("entropy_loss", 0.0)
    assert abs(st["entropy_loss"] - ent_l) <= TOL_LOSS_REL * abs(ent_l) + TOL_LOSS_ABS, \
        (st["entropy_loss"], ent_l)
    if "grad_entropy" in g:
        np.testing.assert_allclose(g["grad_entropy"], of["grad_entropy"], rtol=1e-6, atol=0)
    er = of.get("expert_rows")
    if er is not None and er.size:
        np.testing.assert_allclose(g["grad_logp"][er], of["grad_logp"][er], rtol=1e-6)
    if check_bwd:
        assert np.all(g["dH"][~m] == 0.0), "dH masked rows must be exactly 0"
        assert rel_fro(g["dH"], o["dH"]) <= TOL_GRAD_FRO, rel_fro(g["dH"], o["dH"])
        assert rel_fro(g["dW"], o["dW"]) <= TOL_GRAD_FRO, rel_fro(g["dW"], o["dW"])
