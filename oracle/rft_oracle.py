"""Float64 CPU oracle for the GRPO/PPO trainer-step core.

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the CPU-baseline
leg of the benchmark import this module; the library's product path never
calls it and shares no code with it.

It is the plain definition of what the trainer step computes, written out in
numpy float64, row block by row block, with no online log-sum-exp, no fusion
and no reordering beyond what the definitions state:

* Log-probabilities of the sampled response tokens under the policy (Sec. 3.1.1,
  the ``Experience`` carries the rollout model's log-probs of the response
  tokens because PPO and GRPO need them; Sec. 2.1.2, the trainer computes the
  policy's).  The policy head is ``z = W h`` over the whole vocabulary,
  ``log p = z - logsumexp(z)``.
* Entropy of the policy per token (Sec. 3.4.2, the "actor entropy" plotted as
  an exploration signal): ``H = -sum_j p_j log p_j``.
* GRPO group-relative advantages (Sec. 3.2, Listing 4, ``advantage_fn:
  "grpo"`` with ``repeat_times: 8``; Sec. 3.3.1, 8 rollouts per task): every
  reward is normalised by the mean and standard deviation of its group.
* The clipped PPO surrogate (Sec. 3.3.2: the clipping range of the probability
  ratio defaults to 1 +/- 0.2) and a KL term toward the reference model
  (Sec. 3.3.2, "KL penalty or loss"; Sec. 3.2, Listing 4, ``use_reference``),
  over the tokens the action mask marks (Sec. 2.2 and Sec. 3.1.2: multi-turn
  rollouts are concatenated and masked; Listing 4: the loss takes
  ``logprob, old_logprob, action_mask, advantages``).
* The gradient of that loss with respect to the log-probs, the logits, the
  hidden states and the lm_head weight (the trainer's backward through the
  policy head).

Readings where the paper is silent (it prints no formula):
  R1 KL estimator: k3 = exp(d) - d - 1 with d = ref - logp, added to the loss
     with coefficient beta.
  R2 Aggregation: mode 0 = mean over rollouts of the per-rollout token mean
     (weight 1/(S n_i)); mode 1 = mean over all valid tokens (weight 1/N).
     ``denom_override > 0`` replaces S (mode 0) or N (mode 1).
  R3 Group std: sample std (divisor G-1) by default, the population std
     (divisor G) on request; eps = 1e-6 added to the std; a group whose rewards
     are all equal (or G = 1) gets advantage exactly 0.
  R4 Clip decision: by the definition, in fp64: a token is clipped when
     A > 0 and rho > 1 + eps_high, or A < 0 and rho < 1 - eps_low, with
     strict inequalities (at a bound both branches have the same value and the
     gradient is the interior one, -A rho), rho = exp(logp - old) in fp64.
     The value and the gradient take the same decision.
  R5 Masked rows give 0 in every per-row output; out-of-range token ids in a
     valid row give NaN log-prob, are counted in ``n_bad_ids`` and contribute
     nothing to the loss, its metrics or its gradient (they still count in N
     and n_i).
  R6 N = 0 gives loss 0 and zero gradients.
  R10 MIX (the paper's example of a new algorithm, Sec. 4, combining online
     GRPO with SFT on expert trajectories, mu = 0.1 by default): with
     per-rollout expert flags the loss is (1 - mu) * (the GRPO loss of the
     non-expert rollouts, computed on that sub-batch with its own counts) +
     mu * (the SFT loss of the expert rollouts: the mean of -logp over their
     valid tokens).  The GRPO metrics come from the sub-batch; the entropy
     mean, N, S and the bad-id count cover every valid token.
  R11 Entropy bonus (the paper logs the actor's entropy as the signal of
     exploration that diversity shaping keeps high, Sec. 3.4.2, and prints no
     formula for a bonus): with coefficient c_H >= 0 the loss gains
     -c_H * sum_t w_t H_t over the tokens of the PPO term, with that term's
     aggregation weights w_t (under MIX: the non-expert sub-batch, scaled by
     1 - mu like the rest of the GRPO part); ``entropy_loss`` reports
     sum_t w_t H_t.  Its gradient reaches the logits through
     dH/dz_j = -p_j (z_j - sum_k p_k z_k).
  R12 SFT loss (the train-only mode treats SFT as a special case, Sec. 2.1.1):
     sum_t w_t (-logp_t) over the valid tokens with the weights of R2 (token
     mean by default, which is the SFT term of R10); d loss / d logp_t = -w_t.
  R13 DPO loss (the same mode names DPO on preference pairs, Sec. 2.1.1 and
     Sec. 2.3.1's preference-pair data model; the paper cites DPO and prints no
     formula, so the published sigmoid form is used): rollouts 2k and 2k+1 are
     the chosen and the rejected response of pair k; pi_s and rho_s are the sums
     of the policy and reference log-probs over rollout s's valid tokens (bad
     ids left out); u_k = beta ((pi_c - rho_c) - (pi_r - rho_r)); a pair counts
     when both rollouts have a valid token; the loss is the mean over the P
     counted pairs of -(1 - ls) log sigmoid(u_k) - ls log sigmoid(-u_k) (ls the
     label smoothing of conservative DPO, 0 by default).
  R14 Advantage variants over explicit groups (rollouts that failed, were
     skipped or whose reward has not arrived leave their group smaller,
     Sec. 2.2): rollout i belongs to group id_i (an id outside [0, number of
     groups) leaves it out: advantage 0); a group's size G is the number of
     its rollouts.  Modes: GRPO (R3 on
     the group); mean-centred r_i - mean; leave-one-out r_i - (mean of the
     other G - 1 rewards).  Groups of one rollout give 0 in every mode.
  R15 Masked vocabulary entries: a given logit of -inf (an entry the caller
     excludes) has p = 0, and the products p log p in the entropy and
     p (z - mu) in its gradient are taken as their limit 0 (the convention
     0 log 0 = 0 of the entropy's definition), so masking entries by -inf gives
     the statistics and gradient of the vocabulary without them (and 0 at
     their columns).  A row needs one finite logit.
"""
from __future__ import annotations

import math

import numpy as np

AGG_SEQ_MEAN_TOKEN_MEAN = 0
AGG_TOKEN_MEAN = 1


def _f64(x):
    if hasattr(x, "detach"):
        x = x.detach().cpu()
        if str(x.dtype) == "torch.bfloat16":
            x = x.float()
        x = x.numpy()
    return np.asarray(x, dtype=np.float64)


def _take(X, rr):
    """Rows ``rr`` of a numpy array or a (possibly device) torch tensor, as fp64."""
    if hasattr(X, "detach"):
        import torch
        return _f64(X[torch.as_tensor(rr, dtype=torch.long, device=X.device)])
    return _f64(X[rr])


def _int(x, dtype=np.int64):
    if hasattr(x, "detach"):
        x = x.detach().cpu().numpy()
    return np.asarray(x).astype(dtype)


# ---------------------------------------------------------------- counts ----
def token_counts(mask, seq_start):
    """Valid-token bookkeeping (Sec. 2.2 / Sec. 3.1.2 masking; Listing 4
    ``action_mask``).

    Returns a dict with ``rows`` (indices of valid rows, ascending), ``seq``
    (rollout of each valid row), ``n`` (valid tokens per rollout), ``N`` and
    ``S`` (rollouts with at least one valid token).
    """
    m = _int(mask) != 0
    ss = _int(seq_start)
    n_seq = len(ss) - 1
    n = np.zeros(n_seq, dtype=np.int64)
    for i in range(n_seq):
        n[i] = int(np.count_nonzero(m[ss[i]:ss[i + 1]]))
    rows = np.nonzero(m)[0].astype(np.int64)
    seq = np.searchsorted(ss, rows, side="right") - 1
    return {"rows": rows, "seq": seq.astype(np.int64), "n": n,
            "N": int(n.sum()), "S": int(np.count_nonzero(n))}


# ------------------------------------------------------------ advantages ----
def group_advantages(rewards, group_size, eps=1e-6, unbiased=True):
    """GRPO advantages (Sec. 3.2 Listing 4 ``advantage_fn: "grpo"``; reading R3).

    Rewards of consecutive rollouts ``[g*G, (g+1)*G)`` form one group:
    ``A_i = (r_i - mean) / (std + eps)`` with the sample standard deviation
    (divisor G - 1), or the population one (divisor G) when not ``unbiased``.
    """
    r = _f64(rewards)
    G = int(group_size)
    assert r.size % G == 0
    out = np.zeros_like(r)
    for g0 in range(0, r.size, G):
        grp = r[g0:g0 + G]
        if G < 2 or np.all(grp == grp[0]):
            continue                      # degenerate group: advantage 0
        mu = grp.sum() / G
        sd = math.sqrt(((grp - mu) ** 2).sum() / (G - 1 if unbiased else G))
        out[g0:g0 + G] = (grp - mu) / (sd + eps)
    return out


ADV_GRPO, ADV_MEAN_CENTER, ADV_LEAVE_ONE_OUT = 0, 1, 2


def group_advantages_ids(rewards, group_id, mode=ADV_GRPO, eps=1e-6, n_groups=None,
                         unbiased=True):
    """Advantages over explicit, variable-size groups (reading R14); with
    ``n_groups`` given, ids at or above it also leave their rollout out."""
    r = _f64(rewards)
    gid = _int(group_id)
    out = np.zeros_like(r)
    groups = {}
    for i in range(r.size):
        g = int(gid[i])
        if g >= 0 and (n_groups is None or g < n_groups):
            groups.setdefault(g, []).append(i)
    for g, members in groups.items():
        G = len(members)
        if G < 2:
            continue
        vals = [r[i] for i in members]
        total = sum(vals)
        mu = total / G
        sd = math.sqrt(sum((v - mu) ** 2 for v in vals) / (G - 1 if unbiased else G))
        tied = all(v == vals[0] for v in vals)
        for i in members:
            if mode == ADV_GRPO:
                out[i] = 0.0 if tied else (r[i] - mu) / (sd + eps)
            elif mode == ADV_MEAN_CENTER:
                out[i] = r[i] - mu
            elif mode == ADV_LEAVE_ONE_OUT:
                out[i] = r[i] - (total - r[i]) / (G - 1)
            else:
                raise ValueError(mode)
    return out


# ------------------------------------------------------------- log-probs ----
def _plogp(p, x):
    """p * x with 0 where p == 0 (x may then be -inf: reading R15)."""
    return np.where(p > 0, p * np.where(p > 0, x, 0.0), 0.0)


def _row_stats(z, y, V):
    """Plain two-pass log-softmax statistics of one block of logit rows."""
    M = z.max(axis=1, keepdims=True)
    lse = (M + np.log(np.exp(z - M).sum(axis=1, keepdims=True)))[:, 0]
    logp_all = z - lse[:, None]
    p = np.exp(logp_all)
    ent = -_plogp(p, logp_all).sum(axis=1)
    ok = (y >= 0) & (y < V)
    logp = np.full(z.shape[0], np.nan)
    idx = np.nonzero(ok)[0]
    logp[idx] = logp_all[idx, y[idx]]
    return logp, ent, lse


def token_logprobs(H, W, ids, mask, rows=None, block=256):
    """Per-token log-prob of the sampled id, entropy and log-sum-exp of the
    policy head ``z = W h`` (Sec. 3.1.1 log-probs of response tokens; Sec. 3.4.2
    actor entropy).  Masked rows are 0.

    ``rows`` restricts the computation to those row indices (all rows of the
    returned arrays outside it stay 0); it is how full-size workloads are
    sampled one row at a time.
    """
    Wd = _f64(W)
    V = Wd.shape[0]
    m = _int(mask) != 0
    y = _int(ids)
    T = m.size
    logp = np.zeros(T)
    ent = np.zeros(T)
    lse = np.zeros(T)
    want = np.nonzero(m)[0] if rows is None else np.asarray([r for r in _int(rows) if m[r]],
                                                            dtype=np.int64)
    for b0 in range(0, want.size, block):
        rr = want[b0:b0 + block]
        h = _take(H, rr)
        z = h @ Wd.T
        lp, en, ls = _row_stats(z, y[rr], V)
        logp[rr], ent[rr], lse[rr] = lp, en, ls
    return logp, ent, lse


def token_logprobs_from_logits(logits, ids, mask, rows=None, block=256):
    """Same statistics from given logits ``[T, V]`` (the loss-only path)."""
    m = _int(mask) != 0
    y = _int(ids)
    T = m.size
    V = logits.shape[1]
    logp = np.zeros(T)
    ent = np.zeros(T)
    lse = np.zeros(T)
    want = np.nonzero(m)[0] if rows is None else np.asarray([r for r in _int(rows) if m[r]],
                                                            dtype=np.int64)
    for b0 in range(0, want.size, block):
        rr = want[b0:b0 + block]
        z = _take(logits, rr)
        lp, en, ls = _row_stats(z, y[rr], V)
        logp[rr], ent[rr], lse[rr] = lp, en, ls
    return logp, ent, lse


# ------------------------------------------------------------------ loss ----
def ppo_clip_loss_fwd(logp, old_logp, ref_logp, adv_seq, mask, seq_start, ids=None, V=None,
                      eps_low=0.2, eps_high=0.2, beta=0.0, agg=AGG_SEQ_MEAN_TOKEN_MEAN,
                      denom_override=0.0, entropy=None, is_expert=None, mix_mu=0.0,
                      entropy_coef=0.0):
    if entropy_coef > 0 and entropy is None:
        raise ValueError("the entropy bonus needs the entropies")
    if is_expert is not None:
        return _mix_loss_fwd(logp, old_logp, ref_logp, adv_seq, mask, seq_start, ids, V, eps_low,
                             eps_high, beta, agg, denom_override, entropy, is_expert, mix_mu,
                             entropy_coef)
    return _grpo_loss_fwd(logp, old_logp, ref_logp, adv_seq, mask, seq_start, ids, V, eps_low,
                          eps_high, beta, agg, denom_override, entropy, entropy_coef)


def _mix_loss_fwd(logp, old_logp, ref_logp, adv_seq, mask, seq_start, ids, V, eps_low, eps_high,
                  beta, agg, denom_override, entropy, is_expert, mu, entropy_coef=0.0):
    """MIX loss (reading R10): the GRPO loss of the non-expert rollouts and the
    SFT loss of the expert rollouts, weighted 1 - mu and mu."""
    m = _int(mask) != 0
    ss = _int(seq_start)
    ex = _int(is_expert) != 0
    T = m.size
    row_expert = np.zeros(T, dtype=bool)
    for i in range(ex.size):
        a, b = max(0, min(ss[i], T)), max(0, min(ss[i + 1], T))
        row_expert[a:b] = ex[i]
    # GRPO on the sub-batch of non-expert rollouts (expert rows masked out)
    g = _grpo_loss_fwd(logp, old_logp, ref_logp, adv_seq, m & ~row_expert, seq_start, ids, V,
                       eps_low, eps_high, beta, agg, denom_override, entropy, entropy_coef)
    # SFT on the expert rollouts: mean of -logp over their valid tokens
    lp = _f64(logp)
    er = np.nonzero(m & row_expert)[0]
    good_e = np.ones(er.size, dtype=bool)
    if ids is not None and V is not None:
        yy = _int(ids)[er]
        good_e = (yy >= 0) & (yy < V)
    Ne = er.size
    sft = float(-lp[er][good_e].sum() / Ne) if Ne else 0.0
    grad = (1.0 - mu) * g["grad_logp"]
    if Ne:
        grad[er[good_e]] = -mu / Ne
    cnt = token_counts(m, seq_start)
    N = cnt["N"]
    out = dict(g)
    out.update({
        "loss": (1.0 - mu) * g["loss"] + mu * sft,
        "sft_loss": sft, "n_expert": Ne, "n_valid": N, "n_seq_valid": cnt["S"],
        "n_bad_ids": g["n_bad_ids"] + int((~good_e).sum()),
        "grad_logp": grad, "expert_rows": er[good_e],
        "grad_entropy": (1.0 - mu) * g["grad_entropy"],
    })
    if entropy is not None:
        rows = cnt["rows"]
        good = np.ones(rows.size, dtype=bool)
        if ids is not None and V is not None:
            yy = _int(ids)[rows]
            good = (yy >= 0) & (yy < V)
        out["entropy_mean"] = float(_f64(entropy)[rows][good].sum() / N) if N else 0.0
    else:
        out["entropy_mean"] = 0.0
    return out


def _grpo_loss_fwd(logp, old_logp, ref_logp, adv_seq, mask, seq_start, ids, V, eps_low,
                   eps_high, beta, agg, denom_override, entropy, entropy_coef=0.0):
    """Clipped PPO surrogate with a k3 KL term toward the reference policy,
    aggregated over the masked tokens (Sec. 3.3.2 clip 1 +/- 0.2 and KL; Sec. 3.2
    Listing 4 loss-function call shape returning the loss and its metrics;
    readings R1, R2, R4, R5, R6).

    Returns a dict with the loss, its parts, the statistics, ``grad_logp``
    (d loss / d logp per row, 0 on masked rows) and ``grad_entropy`` (minus
    d loss / d H per row: the entropy-bonus coefficient, reading R11).
    """
    cnt = token_counts(mask, seq_start)
    rows, seq, n, N, S = cnt["rows"], cnt["seq"], cnt["n"], cnt["N"], cnt["S"]
    lp_all = _f64(logp)
    T = lp_all.size
    lp = lp_all[rows]
    old = _f64(old_logp)[rows]
    # without a reference policy there is no KL term: ref = logp, kl = 0
    ref = _f64(ref_logp)[rows] if ref_logp is not None else lp.copy()
    A = _f64(adv_seq)[seq]
    good = np.ones(rows.size, dtype=bool)
    if ids is not None and V is not None:
        yy = _int(ids)[rows]
        good = (yy >= 0) & (yy < V)
    n_bad = int((~good).sum())

    if agg == AGG_SEQ_MEAN_TOKEN_MEAN:
        Sd = denom_override if denom_override > 0 else S
        w = np.zeros(rows.size) if Sd == 0 else 1.0 / (Sd * n[seq].astype(np.float64))
    elif agg == AGG_TOKEN_MEAN:
        Nd = denom_override if denom_override > 0 else N
        w = np.zeros(rows.size) if Nd == 0 else np.full(rows.size, 1.0 / Nd)
    else:
        raise ValueError(agg)

    # ratio, clipped surrogate and the clip decision by the definition (R4)
    rho = np.exp(lp - old)
    lo, hi = 1.0 - eps_low, 1.0 + eps_high
    rho_bar = np.clip(rho, lo, hi)
    pg = np.maximum(-A * rho, -A * rho_bar)
    clipped = ((A > 0) & (rho > hi)) | ((A < 0) & (rho < lo))
    dk = ref - lp
    kl = np.exp(dk) - dk - 1.0
    # beta = 0 switches the KL term off (kl is still reported as a metric)
    bkl = beta * kl if beta > 0 else np.zeros_like(kl)
    ell = pg + bkl
    g = np.where(clipped, 0.0, -A * rho) + (beta * (1.0 - np.exp(dk)) if beta > 0 else 0.0)
    c = w * g
    # bad ids contribute nothing
    pg = np.where(good, pg, 0.0)
    kl = np.where(good, kl, 0.0)
    bkl = np.where(good, bkl, 0.0)
    ell = np.where(good, ell, 0.0)
    c = np.where(good, c, 0.0)
    clipped = clipped & good
    rho_s = np.where(good, rho, 0.0)

    grad = np.zeros(T)
    grad[rows] = c
    # entropy bonus (R11): -c_H sum_t w_t H_t over the rows with a valid id
    ent_rows = np.where(good, _f64(entropy)[rows], 0.0) if entropy is not None else None
    ent_w = float((w * ent_rows).sum()) if entropy is not None else 0.0
    grad_ent = np.zeros(T)
    if entropy_coef > 0:
        grad_ent[rows] = np.where(good, entropy_coef * w, 0.0)
    out = {
        "loss": float((w * ell).sum()) - entropy_coef * ent_w,
        "entropy_loss": ent_w, "grad_entropy": grad_ent,
        "pg_loss": float((w * pg).sum()),
        "kl_loss": float((w * bkl).sum()),
        "kl_mean": float(kl.sum() / N) if N else 0.0,
        "ratio_mean": float(rho_s.sum() / N) if N else 0.0,
        "clipfrac": float(clipped.sum() / N) if N else 0.0,
        "n_valid": N, "n_seq_valid": S, "n_clipped": int(clipped.sum()), "n_bad_ids": n_bad,
        "sft_loss": 0.0, "n_expert": 0,
        "grad_logp": grad, "weights_rows": rows, "weights": w,
        "clipped_rows": rows[clipped],
        # relative distance of rho from the nearer clip bound (an infinite
        # bound, or a lower bound of 0, is never near)
        "margin": np.minimum(np.abs(rho / hi - 1.0) if math.isfinite(hi) else np.inf,
                             np.abs(rho / lo - 1.0) if lo > 0 else np.inf),
    }
    if entropy is not None:
        ent = np.where(good, _f64(entropy)[rows], 0.0)
        out["entropy_mean"] = float(ent.sum() / N) if N else 0.0
    else:
        out["entropy_mean"] = 0.0
    return out


# ---------------------------------------------------- train-only losses ----
def _weights(cnt, agg, denom_override):
    """Aggregation weights w_t of the valid rows (reading R2)."""
    rows, seq, n, N, S = cnt["rows"], cnt["seq"], cnt["n"], cnt["N"], cnt["S"]
    if agg == AGG_SEQ_MEAN_TOKEN_MEAN:
        Sd = denom_override if denom_override > 0 else S
        return np.zeros(rows.size) if Sd == 0 else 1.0 / (Sd * n[seq].astype(np.float64))
    if agg == AGG_TOKEN_MEAN:
        Nd = denom_override if denom_override > 0 else N
        return np.zeros(rows.size) if Nd == 0 else np.full(rows.size, 1.0 / Nd)
    raise ValueError(agg)


def _good_rows(rows, ids, V):
    if ids is None or V is None:
        return np.ones(rows.size, dtype=bool)
    yy = _int(ids)[rows]
    return (yy >= 0) & (yy < V)


def sft_loss_fwd(logp, mask, seq_start, ids=None, V=None, agg=AGG_TOKEN_MEAN,
                 denom_override=0.0):
    """SFT loss of the train-only mode (Sec. 2.1.1; reading R12): the
    aggregated negative log-likelihood of the valid tokens."""
    cnt = token_counts(mask, seq_start)
    rows = cnt["rows"]
    w = _weights(cnt, agg, denom_override)
    good = _good_rows(rows, ids, V)
    lp = _f64(logp)
    nll = np.where(good, -lp[rows], 0.0)
    grad = np.zeros(lp.size)
    grad[rows] = np.where(good, -w, 0.0)
    return {"loss": float((w * nll).sum()), "grad_logp": grad, "n_valid": cnt["N"],
            "n_seq_valid": cnt["S"], "n_bad_ids": int((~good).sum())}


def _log_sigmoid(x):
    """log(1 / (1 + exp(-x))) without overflow."""
    return -(np.maximum(-x, 0.0) + np.log1p(np.exp(-np.abs(x))))


def _sigmoid(x):
    return np.exp(_log_sigmoid(x))


def dpo_loss_fwd(logp, ref_logp, mask, seq_start, ids=None, V=None, beta=0.1,
                 label_smoothing=0.0):
    """DPO loss over preference pairs (Sec. 2.1.1 train-only mode, Sec. 2.3.1
    preference pairs; reading R13).  Returns the loss, the per-token gradient,
    the per-rollout policy sums and the pair statistics."""
    m = _int(mask) != 0
    ss = _int(seq_start)
    n_seq = len(ss) - 1
    if n_seq % 2:
        raise ValueError("DPO needs an even number of rollouts")
    T = m.size
    lp, rf = _f64(logp), _f64(ref_logp)
    cnt = token_counts(mask, seq_start)
    rows = cnt["rows"]
    good = _good_rows(rows, ids, V)
    good_row = np.zeros(T, dtype=bool)
    good_row[rows[good]] = True
    pi = np.zeros(n_seq)
    rho = np.zeros(n_seq)
    for s_ in range(n_seq):
        rr = [t for t in range(ss[s_], ss[s_ + 1]) if good_row[t]]
        pi[s_] = float(sum(lp[t] for t in rr))
        rho[s_] = float(sum(rf[t] for t in rr))
    n = cnt["n"]
    c_, r_ = np.arange(0, n_seq, 2), np.arange(1, n_seq, 2)
    counted = (n[c_] > 0) & (n[r_] > 0)
    P = int(counted.sum())
    rc = beta * (pi[c_] - rho[c_])
    rj = beta * (pi[r_] - rho[r_])
    u = rc - rj
    ls = label_smoothing
    loss_k = -(1.0 - ls) * _log_sigmoid(u) - ls * _log_sigmoid(-u)
    dldu = -(1.0 - ls) * _sigmoid(-u) + ls * _sigmoid(u)     # d loss_k / d u
    coef = np.zeros(n_seq)                                   # d loss / d pi_s
    if P:
        coef[c_] = np.where(counted, beta * dldu / P, 0.0)
        coef[r_] = np.where(counted, -beta * dldu / P, 0.0)
    grad = np.zeros(T)
    seq_of = np.searchsorted(ss, np.arange(T), side="right") - 1
    grad[good_row] = coef[seq_of[good_row]]
    mean = (lambda x: float(x[counted].sum() / P)) if P else (lambda x: 0.0)
    return {"loss": mean(loss_k), "chosen_reward": mean(rc), "rejected_reward": mean(rj),
            "reward_acc": float((u[counted] > 0).sum() / P) if P else 0.0,
            "margin_mean": mean(u), "n_pairs": P, "n_valid": cnt["N"],
            "n_bad_ids": int((~good).sum()), "grad_logp": grad, "seq_logp": pi,
            "pair_counted": counted, "margins": u}


# -------------------------------------------------------------- backward ----
def logit_grad_rows(z, y, lse, c, e=None, ent=None):
    """d loss / d z for a block of rows: ``c (onehot(y) - p)`` with
    ``p = exp(z - lse)``, plus, with the entropy bonus (R11), ``e`` times
    ``-dH/dz = p (z - mu)``, ``mu = lse - H`` the softmax mean of z."""
    p = np.exp(z - lse[:, None])
    dz = -p
    ok = np.nonzero((y >= 0) & (y < z.shape[1]))[0]
    dz[ok, y[ok]] += 1.0
    out = c[:, None] * dz
    if e is not None:
        mu = lse - ent
        out += e[:, None] * _plogp(p, z - mu[:, None])
    return out


def ppo_clip_loss_bwd(H, W, lse, grad_logp, ids, mask, rows=None, dw_rows=None, block=256,
                      want_dw=True, grad_entropy=None, entropy=None):
    """Backward through the policy head: ``dZ = c (onehot(y) - softmax(z))``
    (plus the entropy-bonus term when ``grad_entropy`` and ``entropy`` are
    given), ``dH = dZ W`` and ``dW = dZ^T H`` over the valid rows.

    ``rows`` restricts which rows of dH are returned (others 0).  ``dw_rows``
    returns only those rows of dW, each summed over every valid token, so a
    full-size weight gradient can be sampled without forming all of it.
    """
    Wd = _f64(W)
    V, d = Wd.shape
    m = _int(mask) != 0
    y = _int(ids)
    L = _f64(lse)
    C = _f64(grad_logp)
    E = _f64(grad_entropy) if grad_entropy is not None else None
    Hn = _f64(entropy) if grad_entropy is not None else None
    T = m.size

    def eh(rr):
        return (None, None) if E is None else (E[rr], Hn[rr])

    valid = np.nonzero(m)[0]
    dH = np.zeros((T, d))
    want = valid if rows is None else np.asarray([r for r in _int(rows) if m[r]], dtype=np.int64)
    for b0 in range(0, want.size, block):
        rr = want[b0:b0 + block]
        h = _take(H, rr)
        dz = logit_grad_rows(h @ Wd.T, y[rr], L[rr], C[rr], *eh(rr))
        dH[rr] = dz @ Wd
    dW = None
    if want_dw and dw_rows is None:
        dW = np.zeros((V, d))
        for b0 in range(0, valid.size, block):
            rr = valid[b0:b0 + block]
            h = _take(H, rr)
            dz = logit_grad_rows(h @ Wd.T, y[rr], L[rr], C[rr], *eh(rr))
            dW += dz.T @ h
    elif want_dw:
        js = _int(dw_rows)
        dW = np.zeros((js.size, d))
        Wj = Wd[js]
        for b0 in range(0, valid.size, 4096):
            rr = valid[b0:b0 + 4096]
            h = _take(H, rr)
            zj = h @ Wj.T                                  # [B, J]
            p = np.exp(zj - L[rr][:, None])
            dz = (y[rr][:, None] == js[None, :]) - p
            dz *= C[rr][:, None]
            if E is not None:
                mu = L[rr] - Hn[rr]
                dz += E[rr][:, None] * p * (zj - mu[:, None])
            dW += dz.T @ h
    return dH, dW


def bwd_logits(logits, lse, grad_logp, ids, mask, rows=None, block=256, grad_entropy=None,
               entropy=None):
    """``dlogits = c (onehot(y) - exp(z - lse))`` (plus the entropy-bonus term
    when ``grad_entropy`` and ``entropy`` are given) on valid rows."""
    m = _int(mask) != 0
    y = _int(ids)
    L = _f64(lse)
    C = _f64(grad_logp)
    E = _f64(grad_entropy) if grad_entropy is not None else None
    Hn = _f64(entropy) if grad_entropy is not None else None
    T, V = logits.shape
    want = np.nonzero(m)[0] if rows is None else np.asarray([r for r in _int(rows) if m[r]],
                                                            dtype=np.int64)
    out = {}
    for b0 in range(0, want.size, block):
        rr = want[b0:b0 + block]
        z = _take(logits, rr)
        dz = logit_grad_rows(z, y[rr], L[rr], C[rr], *((None, None) if E is None
                                                       else (E[rr], Hn[rr])))
        for k, r in enumerate(rr):
            out[int(r)] = dz[k]
    return out


# ------------------------------------------------------------ whole step ----
def trainer_step(H, W, ids, mask, seq_start, rewards, group_size, old_logp, ref_logp,
                 eps_low, eps_high, beta, agg, denom_override=0.0, adv_eps=1e-6, want_dw=True,
                 is_expert=None, mix_mu=0.0, entropy_coef=0.0):
    """One pass of the whole path: advantages, log-probs/entropy, loss and the
    gradients to H and W."""
    adv = group_advantages(rewards, group_size, adv_eps)
    logp, ent, lse = token_logprobs(H, W, ids, mask)
    V = _f64(W).shape[0]
    fw = ppo_clip_loss_fwd(logp, old_logp, ref_logp, adv, mask, seq_start, ids, V,
                           eps_low, eps_high, beta, agg, denom_override, entropy=ent,
                           is_expert=is_expert, mix_mu=mix_mu, entropy_coef=entropy_coef)
    eg = (fw["grad_entropy"], ent) if entropy_coef > 0 else (None, None)
    dH, dW = ppo_clip_loss_bwd(H, W, lse, fw["grad_logp"], ids, mask, want_dw=want_dw,
                               grad_entropy=eg[0], entropy=eg[1])
    return {"adv": adv, "logp": logp, "entropy": ent, "lse": lse, "fwd": fw, "dH": dH, "dW": dW}


def loss_only_step(logits, ids, mask, seq_start, rewards, group_size, old_logp, ref_logp,
                   eps_low, eps_high, beta, agg, denom_override=0.0, adv_eps=1e-6, rows=None,
                   is_expert=None, mix_mu=0.0, entropy_coef=0.0):
    """The loss-only path from given logits: log-probs, entropy, loss, dlogits.
    ``rows`` samples the dlogits rows returned; the loss always uses every row."""
    adv = group_advantages(rewards, group_size, adv_eps)
    logp, ent, lse = token_logprobs_from_logits(logits, ids, mask)
    V = logits.shape[1]
    fw = ppo_clip_loss_fwd(logp, old_logp, ref_logp, adv, mask, seq_start, ids, V,
                           eps_low, eps_high, beta, agg, denom_override, entropy=ent,
                           is_expert=is_expert, mix_mu=mix_mu, entropy_coef=entropy_coef)
    eg = (fw["grad_entropy"], ent) if entropy_coef > 0 else (None, None)
    dl = bwd_logits(logits, lse, fw["grad_logp"], ids, mask, rows=rows, grad_entropy=eg[0],
                    entropy=eg[1])
    return {"adv": adv, "logp": logp, "entropy": ent, "lse": lse, "fwd": fw, "dlogits": dl}
