"""Parity at the workloads' full sizes, in the launch configuration the
benchmark times: outputs the oracle can compute one by one are sampled (rows of
log-probs / entropy / lse, rows of dH and dW), the loss kernel is checked on
every token with synthetic inputs, and the weight gradient is checked against
a property that holds at any size (the columns of dW sum to zero)."""
import concurrent.futures as cf
import math

import numpy as np
import pytest
import torch

import paper_2505_17826_amd as R
from gen import synth
from oracle import rft_oracle as O
from tests.gpu_cases import (TOL_GRAD_FRO, TOL_LOGP, TOL_LOSS_ABS, TOL_LOSS_REL, cpu, f32, near_bound,
                             oracle_eps, params_of, rel_fro, requires_gpu)

pytestmark = [pytest.mark.gpu, requires_gpu]
DEV = torch.device("cuda")


def _sample_rows(mask, k, seed):
    v = np.nonzero(mask.cpu().numpy())[0]
    rng = np.random.default_rng(seed)
    return np.sort(rng.choice(v, size=min(k, v.size), replace=False))


def _ws(op, tok, d, V, dt):
    n = R.workspace_bytes(op, tok, d, V, dt)
    return torch.empty(max(n, 1), dtype=torch.uint8, device=DEV)


@pytest.mark.parametrize("cid", [1, 2, 3])
def test_fullsize_bf16(cid):
    cfg = synth.config(cid)
    print(f"[fullsize] {cfg.name}", flush=True)
    b = synth.make_batch(cfg, DEV)
    tok = R.Tokens(b.seq_start, b.mask, b.ids)
    T, d, V = b.T, cfg.d, cfg.V
    m = b.mask.bool()
    dt = R.RFT_BF16
    # ---- forward in the benchmark's configuration
    adv = R.rft_group_advantages(b.rewards, cfg.group)
    logp, ent, lse = R.rft_token_logprobs(tok, b.H, b.W, ws=_ws(R.RFT_OP_TOKEN_LOGPROBS, tok, d, V, dt))
    old = torch.where(m, logp + b.old_noise, torch.zeros_like(logp))
    ref = torch.where(m, logp + b.ref_noise, torch.zeros_like(logp))
    grad, st = R.rft_ppo_clip_loss_fwd(tok, V, logp, old, ref, adv, params_of(cfg), entropy=ent,
                                       ws=_ws(R.RFT_OP_PPO_FWD, tok, d, V, dt))
    dH, dW = R.rft_ppo_clip_loss_bwd(tok, b.H, b.W, lse, grad, ws=_ws(R.RFT_OP_PPO_BWD, tok, d, V, dt))
    torch.cuda.synchronize()
    s = R.stats_to_dict(st)
    assert s["n_valid"] == int(m.sum()) and s["n_bad_ids"] == 0
    assert math.isfinite(s["loss"]) and 0.05 < s["clipfrac"] < 0.4
    # sampled rows of the forward, one by one in the oracle
    rows = _sample_rows(b.mask, 24, cid)
    olp, oent, olse = O.token_logprobs(b.H, b.W, b.ids, b.mask, rows=rows)
    for name, g, o in (("logp", logp, olp), ("entropy", ent, oent), ("lse", lse, olse)):
        err = np.abs(cpu(g)[rows] - o[rows]).max()
        assert err <= TOL_LOGP, (name, err)
    # property at full size: columns of dW sum to zero (rows of dZ sum to zero)
    dWn = dW.double()
    colsum = dWn.sum(dim=0).norm().item()
    assert colsum <= 2e-2 * dWn.norm().item(), (colsum, dWn.norm().item())
    assert torch.all(dH[~m] == 0)
    del dWn

    # ---- the backward alone on synthetic lse / grad_logp, sampled rows of dH and dW
    lse_s = torch.where(m, math.log(V) + 2.0 + synth.extra_normal(T, (cid, 1), DEV, std=0.05),
                        torch.zeros(T, device=DEV))
    c_s = torch.where(m, synth.extra_normal(T, (cid, 2), DEV, std=1.0 / max(1, int(m.sum()))),
                      torch.zeros(T, device=DEV))
    dH2, dW2 = R.rft_ppo_clip_loss_bwd(tok, b.H, b.W, lse_s, c_s,
                                       ws=_ws(R.RFT_OP_PPO_BWD, tok, d, V, dt))
    torch.cuda.synchronize()
    hrows = _sample_rows(b.mask, 12, cid + 10)
    wrows = np.sort(np.random.default_rng(cid).choice(V, size=6, replace=False))
    wrows[0] = int(b.ids[int(hrows[0])].item())          # a row that receives a one-hot term
    wrows = np.unique(wrows)
    odH, odW = O.ppo_clip_loss_bwd(b.H, b.W, lse_s, c_s, b.ids, b.mask, rows=hrows, dw_rows=wrows)
    e1 = rel_fro(cpu(dH2)[hrows], odH[hrows])
    e2 = rel_fro(cpu(dW2[torch.as_tensor(wrows, device=DEV)]), odW)
    print(f"[fullsize] {cfg.name}: dH sampled rel {e1:.2e}, dW sampled rel {e2:.2e}", flush=True)
    assert e1 <= TOL_GRAD_FRO and e2 <= TOL_GRAD_FRO


@pytest.mark.parametrize("cid", [1, 2, 3])
def test_fullsize_loss_all_tokens(cid):
    """The loss kernel on every token of the workload's layout, synthetic fp32
    log-probs: clip decisions and counts bit-exact, loss and per-token gradient
    within tolerance."""
    cfg = synth.config(cid)
    b = synth.make_batch(cfg, "cpu", layout_only=True)   # layout, ids, rewards only
    rng = np.random.default_rng(cid)
    T = b.T
    mk = b.mask.numpy() != 0
    logp = np.where(mk, -rng.random(T) * 14, 0).astype(np.float32)
    old = np.where(mk, logp + rng.standard_normal(T) * math.sqrt(cfg.old_var), 0).astype(np.float32)
    ref = np.where(mk, logp + rng.standard_normal(T) * math.sqrt(cfg.ref_var), 0).astype(np.float32)
    advd = O.group_advantages(b.rewards.numpy(), cfg.group)
    adv = advd.astype(np.float32)
    t = lambda x: torch.from_numpy(x).to(DEV)
    tok = R.Tokens(t(b.seq_start.numpy()), t(b.mask.numpy()), t(b.ids.numpy()))
    gadv = R.rft_group_advantages(t(b.rewards.numpy()), cfg.group)
    grad, st = R.rft_ppo_clip_loss_fwd(tok, cfg.V, t(logp), t(old), t(ref), t(adv), params_of(cfg))
    torch.cuda.synchronize()
    assert np.abs(cpu(gadv) - advd).max() <= 1e-5
    s = R.stats_to_dict(st)
    el, eh, be = oracle_eps(cfg)
    o = O.ppo_clip_loss_fwd(logp, old, ref, adv, b.mask, b.seq_start, b.ids, cfg.V, el, eh, be,
                            cfg.agg)
    assert s["n_clipped"] == o["n_clipped"] and s["n_valid"] == o["n_valid"]
    assert s["n_seq_valid"] == o["n_seq_valid"]
    assert abs(s["loss"] - o["loss"]) <= TOL_LOSS_REL * abs(o["loss"]) + TOL_LOSS_ABS
    g = cpu(grad)
    np.testing.assert_allclose(g, o["grad_logp"], rtol=1e-4, atol=1e-7 * np.abs(o["grad_logp"]).max())


def test_fullsize_loss_only():
    """The loss-only workload at full size (fp32 logits 32768 x 151936): the
    oracle computes every row's log-probs (in row blocks, several threads), the
    loss over all tokens and sampled rows of d_logits."""
    cfg = synth.config(4)
    b = synth.make_batch(cfg, DEV)
    T, V = b.T, cfg.V
    mk = b.mask.cpu().numpy() != 0
    blocks = [np.arange(i, min(T, i + 1024)) for i in range(0, T, 1024)]

    def part(rr):
        return O.token_logprobs_from_logits(b.logits, b.ids, b.mask, rows=rr)
    olp = np.zeros(T); oent = np.zeros(T); olse = np.zeros(T)
    with cf.ThreadPoolExecutor(8) as ex:
        for rr, (a, e, l_) in zip(blocks, ex.map(part, blocks)):
            olp[rr], oent[rr], olse[rr] = a[rr], e[rr], l_[rr]
    old = np.where(mk, olp + b.old_noise.cpu().numpy(), 0).astype(np.float32)
    ref = np.where(mk, olp + b.ref_noise.cpu().numpy(), 0).astype(np.float32)
    t = lambda x: torch.from_numpy(x).to(DEV)
    tok = R.Tokens(b.seq_start, b.mask, b.ids)
    adv = R.rft_group_advantages(b.rewards, cfg.group)
    lp = torch.empty(T, device=DEV); ent = torch.empty(T, device=DEV)
    lse = torch.empty(T, device=DEV); grad = torch.empty(T, device=DEV)
    _, dl, st = R.rft_ppo_clip_fused_logits(tok, b.logits, t(old), t(ref), adv, params_of(cfg),
                                            logp=lp, entropy=ent, lse=lse, grad_logp=grad)
    torch.cuda.synchronize()
    for name, g, o in (("logp", lp, olp), ("entropy", ent, oent), ("lse", lse, olse)):
        gg = cpu(g)
        assert np.all(gg[~mk] == 0)
        err = np.abs(gg[mk] - o[mk]).max()
        assert err <= TOL_LOGP, (name, err)
    el, eh, be = oracle_eps(cfg)
    advo = O.group_advantages(b.rewards.cpu().numpy(), cfg.group)
    o = O.ppo_clip_loss_fwd(olp, old, ref, advo, b.mask, b.seq_start, b.ids, V, el, eh, be, cfg.agg)
    s = R.stats_to_dict(st)
    assert s["n_valid"] == o["n_valid"]
    assert abs(s["loss"] - o["loss"]) <= TOL_LOSS_REL * abs(o["loss"]) + TOL_LOSS_ABS, (s["loss"], o["loss"])
    keep = o["margin"] >= 1e-4
    assert abs(s["n_clipped"] - o["n_clipped"]) <= int((~keep).sum())
    rows = _sample_rows(b.mask, 32, 4)
    odl = O.bwd_logits(b.logits, olse, o["grad_logp"], b.ids, b.mask, rows=rows)
    gdl = cpu(dl[torch.as_tensor(rows, device=DEV)])
    e = rel_fro(gdl, np.stack([odl[int(r)] for r in rows]))
    assert e <= TOL_GRAD_FRO, e
    masked = np.nonzero(~mk)[0][:16]
    assert torch.all(dl[torch.as_tensor(masked, device=DEV)] == 0)


@pytest.mark.parametrize("cid", [1, 2, 3])
def test_fullsize_step(cid):
    """The fused step at full size in the benchmark's configuration.  old / ref
    log-probs are synthetic (independent of the HIP path); the oracle computes
    sampled rows of logp / entropy / lse, their per-token gradient and their
    rows of dH on its own; dW is checked by its zero column sums and against
    the separate backward call of the library on the step's own lse and
    gradient (a consistency check between the two formulations)."""
    cfg = synth.config(cid)
    print(f"[fullsize-step] {cfg.name}", flush=True)
    b = synth.make_batch(cfg, DEV)
    tok = R.Tokens(b.seq_start, b.mask, b.ids)
    T, d, V = b.T, cfg.d, cfg.V
    m = b.mask.bool()
    lp0 = -math.log(V)
    old = torch.where(m, lp0 + synth.extra_normal(T, (cid, 3), DEV, std=1.0), torch.zeros(T, device=DEV))
    ref = torch.where(m, old + synth.extra_normal(T, (cid, 4), DEV, std=0.1), torch.zeros(T, device=DEV))
    adv = R.rft_group_advantages(b.rewards, cfg.group)
    ws = _ws(R.RFT_OP_PPO_STEP, tok, d, V, R.RFT_BF16)
    logp, ent, lse, grad, dH, dW, st = R.rft_ppo_clip_step(tok, b.H, b.W, old, ref, adv,
                                                           params_of(cfg), ws=ws)
    torch.cuda.synchronize()
    s = R.stats_to_dict(st)
    cnt = O.token_counts(b.mask, b.seq_start)
    assert s["n_valid"] == cnt["N"] and s["n_seq_valid"] == cnt["S"] and s["n_bad_ids"] == 0
    assert math.isfinite(s["loss"])
    assert torch.all(logp[~m] == 0) and torch.all(grad[~m] == 0) and torch.all(dH[~m] == 0)
    rows = _sample_rows(b.mask, 24, cid + 20)
    olp, oent, olse = O.token_logprobs(b.H, b.W, b.ids, b.mask, rows=rows)
    for name, g, o in (("logp", logp, olp), ("entropy", ent, oent), ("lse", lse, olse)):
        err = np.abs(cpu(g)[rows] - o[rows]).max()
        assert err <= TOL_LOGP, (name, err)
    el, eh, be = oracle_eps(cfg)
    advo = O.group_advantages(b.rewards.cpu().numpy(), cfg.group)
    of = O.ppo_clip_loss_fwd(olp, cpu(old), cpu(ref), advo, b.mask, b.seq_start, b.ids, V, el, eh,
                             be, cfg.agg)
    pos = np.searchsorted(of["weights_rows"], rows)
    keep = of["margin"][pos] >= 1e-4
    go, gg = of["grad_logp"][rows][keep], cpu(grad)[rows][keep]
    np.testing.assert_allclose(gg, go, rtol=1e-3, atol=1e-7 * np.abs(go).max())
    hrows = rows[keep][:12]
    odH, _ = O.ppo_clip_loss_bwd(b.H, b.W, olse, of["grad_logp"], b.ids, b.mask, rows=hrows,
                                 want_dw=False)
    e1 = rel_fro(cpu(dH)[hrows], odH[hrows])
    dWn = dW.double()
    colsum = dWn.sum(dim=0).norm().item()
    assert colsum <= 2e-2 * dWn.norm().item(), (colsum, dWn.norm().item())
    del dWn
    dH2, dW2 = R.rft_ppo_clip_loss_bwd(tok, b.H, b.W, lse, grad,
                                       ws=_ws(R.RFT_OP_PPO_BWD, tok, d, V, R.RFT_BF16))
    torch.cuda.synchronize()
    e2 = (torch.linalg.norm(dW - dW2) / torch.linalg.norm(dW2)).item()
    e3 = (torch.linalg.norm(dH - dH2) / torch.linalg.norm(dH2)).item()
    print(f"[fullsize-step] {cfg.name}: dH sampled rel {e1:.2e}; step vs separate backward "
          f"dW {e2:.2e} dH {e3:.2e}", flush=True)
    assert e1 <= TOL_GRAD_FRO and e2 <= 5e-3 and e3 <= 5e-3


def test_fullsize_step_mix_entropy():
    """The fused step at the 7B shape with expert rollouts (MIX, mu = 0.1) and an
    entropy bonus: sampled rows of the per-token gradients and of dH against the
    oracle, the expert count, and the zero column sums of dW (the bonus term
    p (z - mu) sums to zero over the vocabulary like onehot - p)."""
    cid = 2
    cfg = synth.config(cid)
    print(f"[fullsize-step-mix-entropy] {cfg.name}", flush=True)
    b = synth.make_batch(cfg, DEV)
    ex = (np.arange(cfg.n_seq) % 4 == 1).astype(np.uint8)
    tok = R.Tokens(b.seq_start, b.mask, b.ids, torch.from_numpy(ex).to(DEV))
    T, d, V = b.T, cfg.d, cfg.V
    m = b.mask.bool()
    lp0 = -math.log(V)
    old = torch.where(m, lp0 + synth.extra_normal(T, (cid, 5), DEV, std=1.0), torch.zeros(T, device=DEV))
    ref = torch.where(m, old + synth.extra_normal(T, (cid, 6), DEV, std=0.1), torch.zeros(T, device=DEV))
    adv = R.rft_group_advantages(b.rewards, cfg.group)
    mu, coef = 0.1, 0.01
    ws = _ws(R.RFT_OP_PPO_STEP, tok, d, V, R.RFT_BF16)
    logp, ent, lse, grad, dH, dW, st = R.rft_ppo_clip_step(
        tok, b.H, b.W, old, ref, adv, params_of(cfg, mix_mu=mu, ent=coef), ws=ws)
    torch.cuda.synchronize()
    s = R.stats_to_dict(st)
    cnt = O.token_counts(b.mask, b.seq_start)
    n_exp = int(sum(cnt["n"][i] for i in range(cfg.n_seq) if ex[i]))
    assert s["n_valid"] == cnt["N"] and s["n_expert"] == n_exp and n_exp > 0
    assert math.isfinite(s["loss"]) and s["entropy_loss"] > 0
    rows = _sample_rows(b.mask, 24, 41)
    olp, oent, olse = O.token_logprobs(b.H, b.W, b.ids, b.mask, rows=rows)
    for name, g, o in (("logp", logp, olp), ("entropy", ent, oent), ("lse", lse, olse)):
        err = np.abs(cpu(g)[rows] - o[rows]).max()
        assert err <= TOL_LOGP, (name, err)
    el, eh, be = oracle_eps(cfg)
    advo = O.group_advantages(b.rewards.cpu().numpy(), cfg.group)
    of = O.ppo_clip_loss_fwd(olp, cpu(old), cpu(ref), advo, b.mask, b.seq_start, b.ids, V, el, eh,
                             be, cfg.agg, entropy=oent, is_expert=ex, mix_mu=f32(mu),
                             entropy_coef=f32(coef))
    # tokens near a clip bound are left out (either branch is valid there)
    g_o = of["grad_logp"][rows]
    near = near_bound(olp[rows], cpu(old)[rows], el, eh) < 1e-4
    gg = cpu(grad)[rows]
    np.testing.assert_allclose(gg[~near], g_o[~near], rtol=1e-3, atol=1e-7 * np.abs(g_o).max())
    hrows = rows[~near][:12]
    odH, _ = O.ppo_clip_loss_bwd(b.H, b.W, olse, of["grad_logp"], b.ids, b.mask, rows=hrows,
                                 want_dw=False, grad_entropy=of["grad_entropy"], entropy=oent)
    e1 = rel_fro(cpu(dH)[hrows], odH[hrows])
    dWn = dW.double()
    colsum = dWn.sum(dim=0).norm().item()
    assert colsum <= 2e-2 * dWn.norm().item(), (colsum, dWn.norm().item())
    print(f"[fullsize-step-mix-entropy] dH sampled rel {e1:.2e}", flush=True)
    assert e1 <= TOL_GRAD_FRO
