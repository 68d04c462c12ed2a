"""Pins of the float64 oracle against what the objective fixes (CPU only).

Each test checks the oracle against something other than itself: closed
forms, invariants, library routines, brute force or finite differences, so
that a dropped term, a wrong sign or index, or a transposed operand fails at
least one of them.
"""
import json
import math
import os

import mpmath
import numpy as np
import pytest
import scipy.special
import scipy.stats
import torch

from oracle import rft_oracle as O

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "closed_forms.json")))
rng0 = np.random.default_rng(12345)


def _layout(lengths, pad):
    n_seq = len(lengths)
    ss = np.arange(n_seq + 1, dtype=np.int32) * pad
    mask = np.zeros(n_seq * pad, dtype=np.uint8)
    for i, L in enumerate(lengths):
        mask[i * pad:i * pad + L] = 1
    return ss, mask


# ------------------------------------------------------------------ counts --
def test_counts_brute_force():
    rng = np.random.default_rng(1)
    for _ in range(20):
        n_seq = int(rng.integers(1, 9))
        lens = rng.integers(0, 7, size=n_seq)
        ss = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
        T = int(ss[-1])
        mask = (rng.random(T) < 0.6).astype(np.uint8)
        c = O.token_counts(mask, ss)
        # pure-Python loops
        rows, seq, n = [], [], [0] * n_seq
        for i in range(n_seq):
            for t in range(int(ss[i]), int(ss[i + 1])):
                if mask[t]:
                    rows.append(t)
                    seq.append(i)
                    n[i] += 1
        assert c["rows"].tolist() == rows
        assert c["seq"].tolist() == seq
        assert c["n"].tolist() == n
        assert c["N"] == sum(n)
        assert c["S"] == sum(1 for x in n if x > 0)


# -------------------------------------------------------------- log-probs --
def _one_layer(T=6, d=5, V=11, scale=1.0, seed=0):
    rng = np.random.default_rng(seed)
    H = rng.standard_normal((T, d))
    W = rng.standard_normal((V, d)) * scale
    ids = rng.integers(0, V, size=T)
    return H, W, ids


def test_logprobs_normalise_over_vocab():
    H, W, _ = _one_layer(T=4, d=6, V=37, scale=1.5)
    mask = np.ones(4, dtype=np.uint8)
    tot = np.zeros(4)
    for j in range(37):
        lp, _, _ = O.token_logprobs(H, W, np.full(4, j), mask)
        tot += np.exp(lp)
    np.testing.assert_allclose(tot, 1.0, rtol=0, atol=1e-13)


def test_logprobs_zero_weight_is_uniform():
    V = 512
    H = rng0.standard_normal((5, 8))
    W = np.zeros((V, 8))
    lp, ent, lse = O.token_logprobs(H, W, np.arange(5), np.ones(5, np.uint8))
    assert np.all(lp == -math.log(V)) or np.allclose(lp, -math.log(V), atol=1e-15)
    np.testing.assert_allclose(ent, math.log(V), atol=1e-13)
    np.testing.assert_allclose(lse, math.log(V), atol=1e-13)


def test_logprobs_dominant_logit():
    V = 64
    logits = rng0.standard_normal((3, V))
    logits[:, 5] += 1000.0
    lp, ent, lse = O.token_logprobs_from_logits(logits, np.full(3, 5), np.ones(3, np.uint8))
    np.testing.assert_allclose(lp, 0.0, atol=1e-300)
    np.testing.assert_allclose(ent, 0.0, atol=1e-300)
    np.testing.assert_allclose(lse, logits[:, 5], rtol=1e-15)


def test_logprobs_row_shift_invariance_and_library():
    V = 300
    logits = rng0.standard_normal((7, V)) * 3
    ids = rng0.integers(0, V, size=7)
    m = np.ones(7, np.uint8)
    lp, ent, lse = O.token_logprobs_from_logits(logits, ids, m)
    shift = rng0.standard_normal(7) * 50
    lp2, ent2, lse2 = O.token_logprobs_from_logits(logits + shift[:, None], ids, m)
    np.testing.assert_allclose(lp2, lp, atol=1e-12)
    np.testing.assert_allclose(ent2, ent, atol=1e-11)
    np.testing.assert_allclose(lse2, lse + shift, atol=1e-12)
    # library routines: scipy logsumexp, scipy entropy
    np.testing.assert_allclose(lse, scipy.special.logsumexp(logits, axis=1), rtol=1e-14)
    p = scipy.special.softmax(logits, axis=1)
    np.testing.assert_allclose(ent, scipy.stats.entropy(p, axis=1), rtol=1e-12)
    np.testing.assert_allclose(lp, np.log(p[np.arange(7), ids]), rtol=1e-12)


def test_logprobs_mpmath_brute_force():
    H, W, ids = _one_layer(T=3, d=4, V=9, scale=2.0, seed=3)
    lp, ent, lse = O.token_logprobs(H, W, ids, np.ones(3, np.uint8))
    mpmath.mp.dps = 40
    for t in range(3):
        z = [mpmath.fsum(mpmath.mpf(float(W[j, k])) * mpmath.mpf(float(H[t, k])) for k in range(4))
             for j in range(9)]
        s = mpmath.fsum(mpmath.e ** zj for zj in z)
        L = mpmath.log(s)
        assert abs(float(L) - lse[t]) < 1e-14
        assert abs(float(z[ids[t]] - L) - lp[t]) < 1e-14
        Hent = -mpmath.fsum((mpmath.e ** (zj - L)) * (zj - L) for zj in z)
        assert abs(float(Hent) - ent[t]) < 1e-14


def test_golden_two_logit():
    g = GOLD["two_logit_softmax"]
    logits = np.array([g["logits"], g["logits"]])
    lp, ent, lse = O.token_logprobs_from_logits(logits, np.array([1, 0]), np.ones(2, np.uint8))
    assert lse[0] == pytest.approx(g["lse"], abs=1e-15)
    assert lp[0] == pytest.approx(g["logp_id1"], abs=1e-15)
    assert lp[1] == pytest.approx(g["logp_id0"], abs=1e-15)
    assert ent[0] == pytest.approx(g["entropy"], abs=1e-15)


def test_two_logit_entropy_closed_form():
    for a in [-30.0, -2.0, 0.0, 0.3, 5.0, 40.0]:
        logits = np.array([[0.0, a]])
        _, ent, _ = O.token_logprobs_from_logits(logits, np.array([0]), np.ones(1, np.uint8))
        s = 1.0 / (1.0 + math.exp(-a))              # p of the second logit
        expect = math.log1p(math.exp(a)) - a * s if a < 30 else (1 + a) * math.exp(-a)
        assert ent[0] == pytest.approx(expect, rel=1e-9, abs=1e-12)
        assert ent[0] >= 0


def test_gaussian_logits_statistics():
    # logits ~ N(0, 2^2), V = 151936: lse ~ ln V + 2, entropy ~ ln V - 2
    rng = np.random.default_rng(7)
    V = 151936
    logits = rng.standard_normal((4, V)) * 2.0
    _, ent, lse = O.token_logprobs_from_logits(logits, np.zeros(4, np.int64), np.ones(4, np.uint8))
    assert np.all(np.abs(lse - (math.log(V) + 2)) < 0.1)
    assert np.all(np.abs(ent - (math.log(V) - 2)) < 0.2)


def test_masked_rows_and_compaction():
    H, W, ids = _one_layer(T=10, d=4, V=13, seed=5)
    mask = np.array([1, 0, 1, 1, 0, 0, 1, 0, 1, 1], np.uint8)
    lp, ent, lse = O.token_logprobs(H, W, ids, mask)
    v = np.nonzero(mask)[0]
    lp2, ent2, lse2 = O.token_logprobs(H[v], W, ids[v], np.ones(v.size, np.uint8))
    assert np.all(lp[mask == 0] == 0) and np.all(ent[mask == 0] == 0) and np.all(lse[mask == 0] == 0)
    np.testing.assert_array_equal(lp[v], lp2)
    np.testing.assert_array_equal(ent[v], ent2)


def test_bad_ids_give_nan_logp():
    H, W, ids = _one_layer(T=4, d=3, V=5)
    ids = np.array([0, 5, -1, 4])
    lp, ent, _ = O.token_logprobs(H, W, ids, np.ones(4, np.uint8))
    assert np.isfinite(lp[0]) and np.isfinite(lp[3])
    assert np.isnan(lp[1]) and np.isnan(lp[2])
    assert np.all(np.isfinite(ent))


# ------------------------------------------------------------- advantages --
def test_advantages_moments_and_degenerate():
    rng = np.random.default_rng(11)
    for G in [2, 3, 8, 16, 33]:
        r = rng.standard_normal(G * 5)
        r[:G] = 0.7                                   # degenerate group
        a = O.group_advantages(r, G)
        assert np.all(a[:G] == 0.0)
        for g in range(1, 5):
            grp = a[g * G:(g + 1) * G]
            raw = r[g * G:(g + 1) * G]
            assert abs(grp.mean()) < 1e-12
            sd = np.std(raw, ddof=1)                  # library sample std
            assert abs(np.std(grp, ddof=1) - sd / (sd + 1e-6)) < 1e-12
            assert abs(np.std(grp, ddof=1) - 1.0) <= 1e-5


def test_advantages_group_of_two_golden():
    g = GOLD["grpo_group_of_two"]
    a = O.group_advantages(np.array(g["rewards"]), 2)
    np.testing.assert_allclose(a, g["adv"], rtol=1e-14)
    np.testing.assert_allclose(np.abs(a), 1 / math.sqrt(2), rtol=2e-6)


def test_advantages_affine_and_permutation():
    rng = np.random.default_rng(2)
    r = rng.random(32)
    a = O.group_advantages(r, 8)
    a2 = O.group_advantages(3.5 * r - 7.0, 8)
    np.testing.assert_allclose(a2, a, atol=1e-5)      # eps breaks exact scale invariance
    perm = np.concatenate([g * 8 + rng.permutation(8) for g in range(4)])
    np.testing.assert_allclose(O.group_advantages(r[perm], 8), a[perm], atol=1e-14)
    assert np.all(O.group_advantages(np.ones(8), 1) == 0)


def test_advantages_binary_rewards():
    # k successes out of G with 0/1 rewards: A = (r - k/G) / (sqrt(k(G-k)/(G(G-1))) + eps)
    G = 8
    for k in range(1, G):
        r = np.array([1.0] * k + [0.0] * (G - k))
        sd = math.sqrt(k * (G - k) / (G * (G - 1)))
        np.testing.assert_allclose(O.group_advantages(r, G), (r - k / G) / (sd + 1e-6), rtol=1e-14)


# ------------------------------------------------------------------- loss --
def _loss_case(seed=0, n_seq=6, pad=7, V=50):
    rng = np.random.default_rng(seed)
    lens = rng.integers(0, pad + 1, size=n_seq)
    lens[0] = pad
    ss, mask = _layout(lens, pad)
    T = n_seq * pad
    logp = -rng.random(T) * 5
    old = logp + rng.standard_normal(T) * 0.3
    ref = logp + rng.standard_normal(T) * 0.3
    adv = rng.standard_normal(n_seq)
    ids = rng.integers(0, V, size=T)
    return ss, mask, logp, old, ref, adv, ids, V


def test_ratio_one_gives_minus_mean_advantage():
    ss, mask, logp, _, ref, adv, ids, V = _loss_case(seed=4)
    c = O.token_counts(mask, ss)
    for agg in (0, 1):
        out = O.ppo_clip_loss_fwd(logp, logp, ref, adv, mask, ss, ids, V, 0.2, 0.2, 0.0, agg)
        # pure-Python expectation
        if agg == 0:
            S = sum(1 for x in c["n"] if x > 0)
            exp = -sum(adv[i] for i in range(len(adv)) if c["n"][i] > 0) / S
        else:
            tot = 0.0
            for t in range(mask.size):
                if mask[t]:
                    i = int(np.searchsorted(ss, t, side="right") - 1)
                    tot += adv[i]
            exp = -tot / c["N"]
        assert out["loss"] == pytest.approx(exp, rel=1e-13, abs=1e-15)
        assert out["clipfrac"] == 0.0 and out["kl_loss"] == 0.0
        assert out["ratio_mean"] == pytest.approx(1.0, abs=1e-15)


def test_zero_advantage():
    ss, mask, logp, old, ref, adv, ids, V = _loss_case(seed=5)
    out = O.ppo_clip_loss_fwd(logp, old, ref, np.zeros_like(adv), mask, ss, ids, V, 0.2, 0.2, 0.0, 0)
    assert out["pg_loss"] == 0.0 and np.all(out["grad_logp"] == 0.0)
    out = O.ppo_clip_loss_fwd(logp, old, ref, np.zeros_like(adv), mask, ss, ids, V, 0.2, 0.2, 0.3, 0)
    w = dict(zip(out["weights_rows"].tolist(), out["weights"].tolist()))
    for t in range(mask.size):
        if mask[t]:
            assert out["grad_logp"][t] == pytest.approx(w[t] * 0.3 * (1 - math.exp(ref[t] - logp[t])),
                                                        rel=1e-13)


@pytest.mark.parametrize("eps_low,eps_high", [(0.2, 0.2), (0.2, 0.28), (0.1, 0.5)])
def test_clip_branches_single_token(eps_low, eps_high):
    ss = np.array([0, 1], np.int32)
    mask = np.ones(1, np.uint8)
    cases = [  # (A, rho, clipped, pg)
        (1.0, 1.6, 1.6 > 1 + eps_high, -min(1.6, 1 + eps_high)),
        (1.0, 0.5, False, -0.5),
        (-1.0, 0.5, 0.5 < 1 - eps_low, max(0.5, 1 - eps_low)),
        (-1.0, 1.6, False, 1.6),
        (2.0, 1.1, False, -2.2),
    ]
    for A, rho, clipped, pg in cases:
        lp = np.array([-1.0])
        old = lp - math.log(rho)
        out = O.ppo_clip_loss_fwd(lp, old, None, np.array([A]), mask, ss, None, None,
                                  eps_low, eps_high, 0.0, 0)
        assert out["pg_loss"] == pytest.approx(pg, rel=1e-12)
        assert out["n_clipped"] == int(clipped)
        g = 0.0 if clipped else -A * rho
        assert out["grad_logp"][0] == pytest.approx(g, rel=1e-12, abs=1e-300)


def test_golden_ppo_tokens():
    for key in ("ppo_single_token_clipped", "ppo_single_token_unclipped_negative_adv"):
        g = GOLD[key]
        out = O.ppo_clip_loss_fwd(np.array([g["logp"]]), np.array([g["old_logp"]]),
                                  np.array([g["ref_logp"]]), np.array([g["adv"]]),
                                  np.ones(1, np.uint8), np.array([0, 1]), None, None,
                                  g["eps"], g["eps"], g["beta"], 0)
        assert out["pg_loss"] == pytest.approx(g["pg_loss"], rel=1e-12)
        assert out["loss"] == pytest.approx(g["loss"], rel=1e-12)
        assert out["grad_logp"][0] == pytest.approx(g["grad_logp"], rel=1e-12)


def test_unbounded_clip_is_plain_importance_gradient():
    ss, mask, logp, old, ref, adv, ids, V = _loss_case(seed=6)
    out = O.ppo_clip_loss_fwd(logp, old, ref, adv, mask, ss, ids, V, 1.0, math.inf, 0.0, 0)
    c = O.token_counts(mask, ss)
    A = adv[c["seq"]]
    rho = np.exp(logp[c["rows"]] - old[c["rows"]])
    np.testing.assert_allclose(out["grad_logp"][c["rows"]], out["weights"] * (-A * rho), rtol=1e-13)
    assert out["n_clipped"] == 0


def test_kl_properties():
    ss, mask, logp, old, ref, adv, ids, V = _loss_case(seed=7)
    out0 = O.ppo_clip_loss_fwd(logp, old, logp, adv, mask, ss, ids, V, 0.2, 0.2, 0.7, 0)
    assert out0["kl_loss"] == 0.0 and out0["kl_mean"] == 0.0
    small = logp + 1e-3 * np.random.default_rng(0).standard_normal(logp.size)
    out = O.ppo_clip_loss_fwd(logp, old, small, adv, mask, ss, ids, V, 0.2, 0.2, 1.0, 1)
    c = O.token_counts(mask, ss)
    dlt = (small - logp)[c["rows"]]
    assert out["kl_mean"] == pytest.approx(float((dlt ** 2 / 2).mean()), rel=2e-3)
    out = O.ppo_clip_loss_fwd(logp, old, ref, adv, mask, ss, ids, V, 0.2, 0.2, 1.0, 0)
    assert out["kl_mean"] > 0
    # kl of one token against the closed form
    g = GOLD["ppo_single_token_clipped"]
    o1 = O.ppo_clip_loss_fwd(np.array([g["logp"]]), np.array([g["logp"]]), np.array([g["ref_logp"]]),
                             np.array([0.0]), np.ones(1, np.uint8), np.array([0, 1]), None, None,
                             0.2, 0.2, 1.0, 0)
    assert o1["kl_mean"] == pytest.approx(g["kl"], rel=1e-13)


def test_kl_off_at_zero_coefficient():
    """beta = 0 switches the KL term off: the loss and gradient equal those
    without a reference, even where the reference makes kl overflow to inf
    (ref - logp = 1000); kl_mean still reports the KL to the given reference,
    and no reference means no KL (kl_mean 0)."""
    ss, mask, logp, old, ref, adv, ids, V = _loss_case(seed=31)
    none = O.ppo_clip_loss_fwd(logp, old, None, adv, mask, ss, ids, V, 0.2, 0.2, 0.0, 0)
    far = O.ppo_clip_loss_fwd(logp, old, logp + 1000.0, adv, mask, ss, ids, V, 0.2, 0.2, 0.0, 0)
    assert none["kl_mean"] == 0.0 and none["kl_loss"] == 0.0
    assert far["loss"] == none["loss"] and far["kl_loss"] == 0.0
    np.testing.assert_array_equal(far["grad_logp"], none["grad_logp"])
    assert far["kl_mean"] == math.inf
    near = O.ppo_clip_loss_fwd(logp, old, ref, adv, mask, ss, ids, V, 0.2, 0.2, 0.0, 0)
    c = O.token_counts(mask, ss)
    d = (ref - logp)[c["rows"]]
    assert near["kl_mean"] == pytest.approx(float((np.exp(d) - d - 1).mean()), rel=1e-12)
    assert near["loss"] == none["loss"]


def test_aggregations_coincide_on_equal_lengths():
    rng = np.random.default_rng(9)
    ss = np.arange(5, dtype=np.int32) * 6
    mask = np.ones(24, np.uint8)
    logp = -rng.random(24)
    old = logp + 0.2 * rng.standard_normal(24)
    adv = rng.standard_normal(4)
    a = O.ppo_clip_loss_fwd(logp, old, logp, adv, mask, ss, None, None, 0.2, 0.2, 0.0, 0)
    b = O.ppo_clip_loss_fwd(logp, old, logp, adv, mask, ss, None, None, 0.2, 0.2, 0.0, 1)
    assert a["loss"] == pytest.approx(b["loss"], rel=1e-14)
    np.testing.assert_allclose(a["grad_logp"], b["grad_logp"], rtol=1e-14)


def test_denominator_override_scales():
    ss, mask, logp, old, ref, adv, ids, V = _loss_case(seed=10)
    for agg in (0, 1):
        a = O.ppo_clip_loss_fwd(logp, old, ref, adv, mask, ss, ids, V, 0.2, 0.2, 0.1, agg)
        base = a["n_seq_valid"] if agg == 0 else a["n_valid"]
        b = O.ppo_clip_loss_fwd(logp, old, ref, adv, mask, ss, ids, V, 0.2, 0.2, 0.1, agg,
                                denom_override=4.0 * base)
        assert b["loss"] == pytest.approx(a["loss"] / 4.0, rel=1e-13)


def test_empty_batch():
    ss = np.array([0, 3, 6], np.int32)
    mask = np.zeros(6, np.uint8)
    out = O.ppo_clip_loss_fwd(np.zeros(6), np.zeros(6), np.zeros(6), np.ones(2), mask, ss,
                              None, None, 0.2, 0.2, 0.1, 0)
    assert out["loss"] == 0.0 and out["n_valid"] == 0 and np.all(out["grad_logp"] == 0)


def test_bad_ids_in_loss():
    ss, mask, logp, old, ref, adv, ids, V = _loss_case(seed=12)
    v = np.nonzero(mask)[0]
    ids = ids.copy()
    ids[v[0]] = V
    ids[v[3]] = -2
    out = O.ppo_clip_loss_fwd(logp, old, ref, adv, mask, ss, ids, V, 0.2, 0.2, 0.1, 0)
    assert out["n_bad_ids"] == 2
    assert out["grad_logp"][v[0]] == 0.0 and out["grad_logp"][v[3]] == 0.0
    assert out["n_valid"] == v.size


def test_golden_bad_id_every_metric():
    """Hand-derived fixture: a valid row with an out-of-range id (holding
    finite values that would clip, add KL and entropy if counted) changes no
    returned metric, gradient or entropy-bonus coefficient, and still counts
    in N and n_i (reading R5)."""
    g = GOLD["ppo_bad_id_all_metrics"]
    ss = np.array([0, 3], np.int32)
    mask = np.ones(3, np.uint8)
    out = O.ppo_clip_loss_fwd(np.array(g["logp"]), np.array(g["old_logp"]), np.array(g["ref_logp"]),
                              np.array([g["adv"]]), mask, ss, np.array(g["ids"]), g["V"],
                              g["eps"], g["eps"], g["beta"], O.AGG_SEQ_MEAN_TOKEN_MEAN,
                              entropy=np.array(g["entropy"]), entropy_coef=g["entropy_coef"])
    for k in ("loss", "pg_loss", "kl_loss", "kl_mean", "ratio_mean", "clipfrac", "entropy_mean",
              "entropy_loss"):
        assert out[k] == pytest.approx(g[k], rel=1e-12, abs=1e-15), k
    for k in ("n_clipped", "n_bad_ids", "n_valid", "n_seq_valid"):
        assert out[k] == g[k], k
    np.testing.assert_allclose(out["grad_logp"], g["grad_logp"], rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(out["grad_entropy"], g["grad_entropy"], rtol=1e-12, atol=1e-15)


@pytest.mark.parametrize("A", [2.0, -3.0])
def test_clip_exactly_on_the_bound_takes_the_interior_gradient(A):
    """rho exactly on a bound (reading R4: strict inequalities): with eps = 0
    and logp = old, rho = 1 is both bounds and the gradient is -A rho; with
    eps_high = 1 and logp - old = ln 2 (rho = 2 exactly in fp64), likewise."""
    ss = np.array([0, 1], np.int32)
    mask = np.ones(1, np.uint8)
    lp = np.array([-0.75])
    out = O.ppo_clip_loss_fwd(lp, lp.copy(), None, np.array([A]), mask, ss, None, None,
                              0.0, 0.0, 0.0, 0)
    assert out["n_clipped"] == 0 and out["clipfrac"] == 0.0
    assert out["grad_logp"][0] == -A
    assert out["pg_loss"] == -A
    old = lp - math.log(2.0)
    assert math.exp(lp[0] - old[0]) == 2.0
    out = O.ppo_clip_loss_fwd(lp, old, None, np.array([abs(A)]), mask, ss, None, None,
                              0.0, 1.0, 0.0, 0)
    assert out["n_clipped"] == 0 and out["grad_logp"][0] == -abs(A) * 2.0
    # just past the bound: clipped, gradient 0, value at the bound
    out = O.ppo_clip_loss_fwd(lp, old - 1e-9, None, np.array([abs(A)]), mask, ss, None, None,
                              0.0, 1.0, 0.0, 0)
    assert out["n_clipped"] == 1 and out["grad_logp"][0] == 0.0
    assert out["pg_loss"] == -abs(A) * 2.0


def test_clip_value_and_gradient_agree_near_a_bound():
    """On tokens a hair inside and outside each bound the gradient is the
    slope of the value: central differences of pg with a step far smaller
    than the distance to the bound."""
    ss = np.array([0, 1], np.int32)
    mask = np.ones(1, np.uint8)
    for A, rho in ((1.0, 1.2 * (1 - 1e-7)), (1.0, 1.2 * (1 + 1e-7)), (-1.0, 0.8 * (1 - 1e-7)),
                   (-1.0, 0.8 * (1 + 1e-7))):
        lp = np.array([-1.0])
        old = lp - math.log(rho)
        out = O.ppo_clip_loss_fwd(lp, old, None, np.array([A]), mask, ss, None, None,
                                  0.2, 0.2, 0.0, 0)
        h = 1e-11
        f = lambda x: O.ppo_clip_loss_fwd(np.array([x]), old, None, np.array([A]), mask, ss,
                                          None, None, 0.2, 0.2, 0.0, 0)["pg_loss"]
        fd = (f(lp[0] + h) - f(lp[0] - h)) / (2 * h)
        assert fd == pytest.approx(out["grad_logp"][0], rel=1e-3, abs=1e-6), (A, rho)


def test_golden_mix_entropy_mean_over_every_valid_token():
    """Under MIX the entropy mean covers every valid token, expert ones
    included, while the GRPO metrics cover the non-expert rollouts
    (hand-derived fixture, reading R10)."""
    g = GOLD["mix_entropy_mean_scope"]
    lp = np.array(g["logp"])
    out = O.ppo_clip_loss_fwd(lp, lp.copy(), lp.copy(), np.array(g["adv"]), np.ones(3, np.uint8),
                              np.array(g["seq_start"], np.int32), np.array(g["ids"]), g["V"],
                              0.2, 0.2, 0.0, O.AGG_SEQ_MEAN_TOKEN_MEAN,
                              entropy=np.array(g["entropy"]),
                              is_expert=np.array(g["is_expert"], np.uint8), mix_mu=g["mu"])
    for k in ("loss", "pg_loss", "sft_loss", "entropy_mean", "entropy_loss", "ratio_mean",
              "clipfrac"):
        assert out[k] == pytest.approx(g[k], rel=1e-13, abs=1e-15), k
    assert out["n_expert"] == g["n_expert"] and out["n_valid"] == g["n_valid"]
    np.testing.assert_allclose(out["grad_logp"], g["grad_logp"], rtol=1e-13)


# --------------------------------------------------------------- gradients --
def _loss_of(H, W, ids, mask, ss, old, ref, adv, eps_l, eps_h, beta, agg):
    lp, _, _ = O.token_logprobs(H, W, ids, mask)
    return O.ppo_clip_loss_fwd(lp, old, ref, adv, mask, ss, ids, W.shape[0], eps_l, eps_h,
                               beta, agg)


def _grad_case(seed):
    rng = np.random.default_rng(seed)
    lens = [5, 3, 0, 4]
    ss, mask = _layout(lens, 5)
    T, d, V = 20, 6, 9
    H = rng.standard_normal((T, d))
    W = rng.standard_normal((V, d)) * 0.8
    ids = rng.integers(0, V, size=T)
    lp, _, _ = O.token_logprobs(H, W, ids, mask)
    old = lp + rng.standard_normal(T) * 0.25
    ref = lp + rng.standard_normal(T) * 0.3
    adv = rng.standard_normal(4)
    return H, W, ids, mask, ss, old, ref, adv


@pytest.mark.parametrize("agg", [0, 1])
def test_finite_difference_gradients(agg):
    # first seed whose tokens all lie more than 1e-3 from a clip bound
    for seed in range(21 + 100 * agg, 121 + 100 * agg):
        H, W, ids, mask, ss, old, ref, adv = _grad_case(seed)
        args = (ids, mask, ss, old, ref, adv, 0.2, 0.28, 0.05, agg)
        base = _loss_of(H, W, *args)
        if base["margin"].min() > 1e-3:
            break
    assert base["margin"].min() > 1e-3
    assert base["n_clipped"] > 0          # the clipped branch is exercised
    _, _, lse = O.token_logprobs(H, W, ids, mask)
    dH, dW = O.ppo_clip_loss_bwd(H, W, lse, base["grad_logp"], ids, mask)
    h = 1e-6
    for X, G in ((H, dH), (W, dW)):
        for idx in np.ndindex(X.shape):
            if X is H and not mask[idx[0]]:
                assert G[idx] == 0.0
                continue
            Xp = X.copy(); Xp[idx] += h
            Xm = X.copy(); Xm[idx] -= h
            Hp, Wp = (Xp, W) if X is H else (H, Xp)
            Hm, Wm = (Xm, W) if X is H else (H, Xm)
            fd = (_loss_of(Hp, Wp, *args)["loss"] - _loss_of(Hm, Wm, *args)["loss"]) / (2 * h)
            assert abs(fd - G[idx]) <= 1e-6 * max(1.0, abs(G).max()), (X is H, idx, fd, G[idx])


def test_finite_difference_logits():
    rng = np.random.default_rng(5)
    ss = np.array([0, 4, 8], np.int32)
    mask = np.array([1, 1, 0, 1, 1, 1, 1, 0], np.uint8)
    T, V = 8, 7
    logits = rng.standard_normal((T, V)) * 2
    ids = rng.integers(0, V, size=T)
    lp, _, lse = O.token_logprobs_from_logits(logits, ids, mask)
    old = lp + 0.2 * rng.standard_normal(T)
    ref = lp + 0.2 * rng.standard_normal(T)
    adv = np.array([0.8, -1.1])

    def L(z):
        l2, _, _ = O.token_logprobs_from_logits(z, ids, mask)
        return O.ppo_clip_loss_fwd(l2, old, ref, adv, mask, ss, ids, V, 0.2, 0.2, 0.1, 0)

    base = L(logits)
    dl = O.bwd_logits(logits, lse, base["grad_logp"], ids, mask)
    h = 1e-6
    for t in range(T):
        for j in range(V):
            zp = logits.copy(); zp[t, j] += h
            zm = logits.copy(); zm[t, j] -= h
            fd = (L(zp)["loss"] - L(zm)["loss"]) / (2 * h)
            g = dl[t][j] if t in dl else 0.0
            assert abs(fd - g) < 1e-8, (t, j, fd, g)


def test_torch_autograd_third_implementation():
    """torch float64 autograd of the naive loss expression on tiny inputs."""
    H, W, ids, mask, ss, old, ref, adv = _grad_case(31)
    eps_l, eps_h, beta = 0.2, 0.28, 0.05
    base = _loss_of(H, W, ids, mask, ss, old, ref, adv, eps_l, eps_h, beta, 0)
    _, _, lse = O.token_logprobs(H, W, ids, mask)
    dH, dW = O.ppo_clip_loss_bwd(H, W, lse, base["grad_logp"], ids, mask)

    Ht = torch.tensor(H, requires_grad=True)
    Wt = torch.tensor(W, requires_grad=True)
    logits = Ht @ Wt.T
    logprob = torch.log_softmax(logits, dim=-1).gather(1, torch.tensor(ids)[:, None])[:, 0]
    m = torch.tensor(mask, dtype=torch.float64)
    T = mask.size
    seq = torch.tensor(np.searchsorted(ss, np.arange(T), side="right") - 1)
    A = torch.tensor(adv)[seq]
    ratio = torch.exp(logprob - torch.tensor(old))
    surr = torch.maximum(-A * ratio, -A * torch.clamp(ratio, 1 - eps_l, 1 + eps_h))
    dk = torch.tensor(ref) - logprob
    per_tok = surr + beta * (torch.exp(dk) - dk - 1)
    n_i = torch.zeros(len(ss) - 1, dtype=torch.float64).index_add_(0, seq, m)
    S = (n_i > 0).sum()
    loss = ((per_tok * m) / n_i[seq].clamp(min=1)).sum() / S
    loss.backward()
    assert loss.item() == pytest.approx(base["loss"], rel=1e-12)
    np.testing.assert_allclose(dH, Ht.grad.numpy(), rtol=1e-10, atol=1e-14)
    np.testing.assert_allclose(dW, Wt.grad.numpy(), rtol=1e-10, atol=1e-14)


def test_weight_gradient_invariants():
    H, W, ids, mask, ss, old, ref, adv = _grad_case(41)
    base = _loss_of(H, W, ids, mask, ss, old, ref, adv, 0.2, 0.2, 0.01, 0)
    _, _, lse = O.token_logprobs(H, W, ids, mask)
    dH, dW = O.ppo_clip_loss_bwd(H, W, lse, base["grad_logp"], ids, mask)
    # rows of dZ sum to zero, hence the columns of dW sum to zero
    np.testing.assert_allclose(dW.sum(axis=0), 0.0, atol=1e-13)
    # adding a common vector to every row of W leaves log-probs and dH unchanged
    u = np.random.default_rng(0).standard_normal(W.shape[1])
    W2 = W + u[None, :]
    lp2, _, lse2 = O.token_logprobs(H, W2, ids, mask)
    lp1, _, _ = O.token_logprobs(H, W, ids, mask)
    np.testing.assert_allclose(lp2, lp1, atol=1e-12)
    dH2, _ = O.ppo_clip_loss_bwd(H, W2, lse2, base["grad_logp"], ids, mask)
    np.testing.assert_allclose(dH2, dH, atol=1e-12)
    # sampled dW rows agree with the full dW
    _, dWs = O.ppo_clip_loss_bwd(H, W, lse, base["grad_logp"], ids, mask, dw_rows=[0, 3, 8])
    np.testing.assert_allclose(dWs, dW[[0, 3, 8]], rtol=1e-12, atol=1e-15)


def test_whole_step_composition():
    rng = np.random.default_rng(3)
    ss, mask = _layout([4, 4, 2, 3], 4)
    T, d, V = 16, 5, 11
    H = rng.standard_normal((T, d))
    W = rng.standard_normal((V, d))
    ids = rng.integers(0, V, size=T)
    r = np.array([1.0, 0.0, 1.0, 1.0])
    lp, _, _ = O.token_logprobs(H, W, ids, mask)
    out = O.trainer_step(H, W, ids, mask, ss, r, 2, lp, lp, 0.2, 0.2, 0.0, 0)
    # ratio 1, no KL: loss = -mean advantage over rollouts with tokens
    a = O.group_advantages(r, 2)
    assert out["fwd"]["loss"] == pytest.approx(-a.mean(), abs=1e-14)


# ------------------------------------------------------------ MIX (R10) ----
def test_mix_without_experts_scales_grpo():
    """No expert rollout: the MIX loss is (1 - mu) times the GRPO loss, its
    gradient likewise, and the GRPO metrics are the plain ones."""
    ss, mask, logp, old, ref, adv, ids, V = _loss_case(seed=21)
    mu = 0.3
    plain = O.ppo_clip_loss_fwd(logp, old, ref, adv, mask, ss, ids, V, 0.2, 0.28, 0.05, 0)
    mix = O.ppo_clip_loss_fwd(logp, old, ref, adv, mask, ss, ids, V, 0.2, 0.28, 0.05, 0,
                              is_expert=np.zeros(adv.size, np.uint8), mix_mu=mu)
    assert mix["loss"] == pytest.approx((1 - mu) * plain["loss"], rel=1e-13)
    np.testing.assert_allclose(mix["grad_logp"], (1 - mu) * plain["grad_logp"], rtol=1e-13)
    for k in ("pg_loss", "kl_loss", "kl_mean", "ratio_mean", "clipfrac", "n_clipped"):
        assert mix[k] == plain[k], k
    assert mix["sft_loss"] == 0.0 and mix["n_expert"] == 0


def test_mix_all_experts_is_sft():
    """Every rollout is an expert one and mu = 1: the loss is the mean of -logp
    over the valid tokens (pure-Python sum) and every valid token's gradient
    is -1/N."""
    ss, mask, logp, old, ref, adv, ids, V = _loss_case(seed=22)
    out = O.ppo_clip_loss_fwd(logp, old, ref, adv, mask, ss, ids, V, 0.2, 0.2, 0.1, 0,
                              is_expert=np.ones(adv.size, np.uint8), mix_mu=1.0)
    vals = [-float(logp[t]) for t in range(mask.size) if mask[t]]
    assert out["loss"] == pytest.approx(sum(vals) / len(vals), rel=1e-13)
    assert out["sft_loss"] == pytest.approx(sum(vals) / len(vals), rel=1e-13)
    g = out["grad_logp"]
    assert np.all(g[mask == 0] == 0)
    np.testing.assert_allclose(g[mask != 0], -1.0 / len(vals), rtol=1e-15)
    assert out["n_expert"] == len(vals) and out["n_clipped"] == 0


def test_mix_equals_two_separate_batches():
    """A mixed batch gives (1 - mu) * the GRPO loss of its non-expert rollouts,
    computed as a separate batch with its own counts, + mu * the mean -logp of
    its expert rollouts, also taken apart; likewise the per-token gradient."""
    rng = np.random.default_rng(23)
    pad, V, mu = 9, 40, 0.1
    lens = np.array([9, 4, 0, 7, 9, 2, 5, 8])
    ex = np.array([0, 1, 0, 0, 1, 0, 1, 0], np.uint8)
    ss, mask = _layout(lens, pad)
    T = mask.size
    logp = -rng.random(T) * 4
    old = logp + rng.standard_normal(T) * 0.4
    ref = logp + rng.standard_normal(T) * 0.2
    adv = rng.standard_normal(lens.size)
    ids = rng.integers(0, V, size=T)
    for agg in (0, 1):
        out = O.ppo_clip_loss_fwd(logp, old, ref, adv, mask, ss, ids, V, 0.2, 0.2, 0.02, agg,
                                  is_expert=ex, mix_mu=mu)
        keep = np.nonzero(ex == 0)[0]
        rows_g = np.concatenate([np.arange(i * pad, (i + 1) * pad) for i in keep])
        ss_g, mask_g = _layout(lens[keep], pad)
        sub = O.ppo_clip_loss_fwd(logp[rows_g], old[rows_g], ref[rows_g], adv[keep], mask_g, ss_g,
                                  ids[rows_g], V, 0.2, 0.2, 0.02, agg)
        rows_e = [t for i in np.nonzero(ex)[0] for t in range(i * pad, i * pad + lens[i])]
        sft = -sum(float(logp[t]) for t in rows_e) / len(rows_e)
        assert out["loss"] == pytest.approx((1 - mu) * sub["loss"] + mu * sft, rel=1e-12)
        assert out["pg_loss"] == pytest.approx(sub["pg_loss"], rel=1e-12)
        np.testing.assert_allclose(out["grad_logp"][rows_g], (1 - mu) * sub["grad_logp"],
                                   rtol=1e-12, atol=1e-300)
        np.testing.assert_allclose(out["grad_logp"][rows_e], -mu / len(rows_e), rtol=1e-14)
        assert out["n_valid"] == int(lens.sum()) and out["n_expert"] == len(rows_e)


def test_mix_finite_difference():
    """Central differences of the MIX loss with respect to each valid logp
    (tokens near a clip bound skipped)."""
    ss, mask, logp, old, ref, adv, ids, V = _loss_case(seed=24)
    ex = (np.arange(adv.size) % 3 == 1).astype(np.uint8)
    args = (old, ref, adv, mask, ss, ids, V, 0.2, 0.2, 0.03, 0)
    kw = dict(is_expert=ex, mix_mu=0.25)
    out = O.ppo_clip_loss_fwd(logp, *args, **kw)
    h = 1e-6
    checked = 0
    for t in np.nonzero(mask)[0]:
        d = logp[t] - old[t]
        if min(abs(d - math.log(1.2)), abs(d - math.log(0.8))) < 1e-3:
            continue
        lp1, lp2 = logp.copy(), logp.copy()
        lp1[t] += h
        lp2[t] -= h
        fd = (O.ppo_clip_loss_fwd(lp1, *args, **kw)["loss"] -
              O.ppo_clip_loss_fwd(lp2, *args, **kw)["loss"]) / (2 * h)
        assert fd == pytest.approx(out["grad_logp"][t], rel=1e-6, abs=1e-9), t
        checked += 1
    assert checked > 10


# ---------------------------------------------------- entropy bonus (R11) ----
def _ent_loss_of_logits(z, ids, mask, ss, old, ref, adv, agg, coef, **kw):
    lp, ent, _ = O.token_logprobs_from_logits(z, ids, mask)
    return O.ppo_clip_loss_fwd(lp, old, ref, adv, mask, ss, ids, z.shape[1], 0.2, 0.2, 0.05, agg,
                               entropy=ent, entropy_coef=coef, **kw)


@pytest.mark.parametrize("mix", [False, True])
def test_entropy_bonus_finite_difference_logits(mix):
    """Central differences of the loss with the entropy bonus (entropy taken
    from the logits by its definition) against the oracle's d loss / d z."""
    rng = np.random.default_rng(61)
    ss = np.array([0, 4, 8, 12], np.int32)
    mask = np.array([1, 1, 0, 1, 1, 1, 1, 0, 1, 1, 1, 0], np.uint8)
    T, V = 12, 7
    z = rng.standard_normal((T, V)) * 1.5
    ids = rng.integers(0, V, size=T)
    lp, ent, lse = O.token_logprobs_from_logits(z, ids, mask)
    old = lp + 0.1 * rng.standard_normal(T)
    ref = lp + 0.2 * rng.standard_normal(T)
    adv = np.array([0.8, -1.1, 0.4])
    kw = dict(is_expert=np.array([0, 1, 0], np.uint8), mix_mu=0.3) if mix else {}
    args = (ids, mask, ss, old, ref, adv, 0, 0.07)
    base = _ent_loss_of_logits(z, *args, **kw)
    assert base["margin"].min() > 1e-3
    assert base["grad_entropy"].max() > 0
    dl = O.bwd_logits(z, lse, base["grad_logp"], ids, mask, grad_entropy=base["grad_entropy"],
                      entropy=ent)
    h = 1e-6
    for t in range(T):
        for j in range(V):
            zp = z.copy(); zp[t, j] += h
            zm = z.copy(); zm[t, j] -= h
            fd = (_ent_loss_of_logits(zp, *args, **kw)["loss"] -
                  _ent_loss_of_logits(zm, *args, **kw)["loss"]) / (2 * h)
            g = dl[t][j] if t in dl else 0.0
            assert abs(fd - g) < 1e-8, (t, j, fd, g)


def test_entropy_bonus_uniform_rows():
    """Rows of equal logits: H = log V, the bonus moves the loss by exactly
    -c_H log V (the weights of the sequence-mean token-mean sum to 1) and
    leaves d loss / d z unchanged (dH/dz = 0 at the uniform distribution)."""
    ss, mask = _layout([3, 5, 2], 5)
    T, V, coef = 15, 13, 0.3
    z = np.repeat(np.linspace(-1, 1, T)[:, None], V, axis=1)
    rng = np.random.default_rng(62)
    ids = rng.integers(0, V, size=T)
    lp, ent, lse = O.token_logprobs_from_logits(z, ids, mask)
    np.testing.assert_allclose(ent[mask != 0], math.log(V), rtol=1e-14)
    old = lp + 0.05 * rng.standard_normal(T)
    adv = np.array([1.0, -0.5, 0.25])
    a0 = O.ppo_clip_loss_fwd(lp, old, lp, adv, mask, ss, ids, V, 0.2, 0.2, 0.0, 0, entropy=ent)
    a1 = O.ppo_clip_loss_fwd(lp, old, lp, adv, mask, ss, ids, V, 0.2, 0.2, 0.0, 0, entropy=ent,
                             entropy_coef=coef)
    assert a1["loss"] - a0["loss"] == pytest.approx(-coef * math.log(V), rel=1e-12)
    assert a1["entropy_loss"] == pytest.approx(math.log(V), rel=1e-13)
    d0 = O.bwd_logits(z, lse, a0["grad_logp"], ids, mask)
    d1 = O.bwd_logits(z, lse, a1["grad_logp"], ids, mask, grad_entropy=a1["grad_entropy"],
                      entropy=ent)
    for t in d0:
        np.testing.assert_allclose(d1[t], d0[t], atol=1e-15)


def test_entropy_loss_token_mean_equals_entropy_mean():
    """With token-mean weights 1/N the weighted entropy sum is the entropy
    mean, which the oracle aggregates separately."""
    ss, mask, logp, old, ref, adv, ids, V = _loss_case(seed=63)
    ent = np.random.default_rng(63).random(mask.size) * 3
    out = O.ppo_clip_loss_fwd(logp, old, ref, adv, mask, ss, ids, V, 0.2, 0.2, 0.0, 1,
                              entropy=ent, entropy_coef=0.01)
    assert out["n_bad_ids"] == 0
    assert out["entropy_loss"] == pytest.approx(out["entropy_mean"], rel=1e-13)
    np.testing.assert_allclose(out["grad_entropy"][mask != 0], 0.01 / out["n_valid"], rtol=1e-15)
    assert np.all(out["grad_entropy"][mask == 0] == 0)


def test_entropy_bonus_torch_autograd():
    """torch float64 autograd of the naive expression with the entropy taken
    as -sum p log p, through H and W (a third implementation)."""
    H, W, ids, mask, ss, old, ref, adv = _grad_case(33)
    eps_l, eps_h, beta, coef = 0.2, 0.28, 0.05, 0.02
    lp, ent, lse = O.token_logprobs(H, W, ids, mask)
    base = O.ppo_clip_loss_fwd(lp, old, ref, adv, mask, ss, ids, W.shape[0], eps_l, eps_h, beta,
                               0, entropy=ent, entropy_coef=coef)
    dH, dW = O.ppo_clip_loss_bwd(H, W, lse, base["grad_logp"], ids, mask,
                                 grad_entropy=base["grad_entropy"], entropy=ent)
    _, dWs = O.ppo_clip_loss_bwd(H, W, lse, base["grad_logp"], ids, mask, dw_rows=[1, 4],
                                 grad_entropy=base["grad_entropy"], entropy=ent)

    Ht = torch.tensor(H, requires_grad=True)
    Wt = torch.tensor(W, requires_grad=True)
    logits = Ht @ Wt.T
    logsm = torch.log_softmax(logits, dim=-1)
    logprob = logsm.gather(1, torch.tensor(ids)[:, None])[:, 0]
    entropy = -(logsm.exp() * logsm).sum(-1)
    m = torch.tensor(mask, dtype=torch.float64)
    T = mask.size
    seq = torch.tensor(np.searchsorted(ss, np.arange(T), side="right") - 1)
    A = torch.tensor(adv)[seq]
    ratio = torch.exp(logprob - torch.tensor(old))
    surr = torch.maximum(-A * ratio, -A * torch.clamp(ratio, 1 - eps_l, 1 + eps_h))
    dk = torch.tensor(ref) - logprob
    per_tok = surr + beta * (torch.exp(dk) - dk - 1) - coef * entropy
    n_i = torch.zeros(len(ss) - 1, dtype=torch.float64).index_add_(0, seq, m)
    S = (n_i > 0).sum()
    loss = ((per_tok * m) / n_i[seq].clamp(min=1)).sum() / S
    loss.backward()
    assert loss.item() == pytest.approx(base["loss"], rel=1e-12)
    np.testing.assert_allclose(dH, Ht.grad.numpy(), rtol=1e-10, atol=1e-14)
    np.testing.assert_allclose(dW, Wt.grad.numpy(), rtol=1e-10, atol=1e-14)
    np.testing.assert_allclose(dWs, dW[[1, 4]], rtol=1e-12, atol=1e-15)


# ------------------------------------------------------ SFT (R12) -----------
def test_golden_sft_two_rollouts():
    g = GOLD["sft_two_rollouts"]
    lens = [len(x) for x in g["logp"]]
    ss, mask = _layout(lens, 3)
    logp = np.zeros(6)
    for i, x in enumerate(g["logp"]):
        logp[i * 3:i * 3 + len(x)] = x
    tm = O.sft_loss_fwd(logp, mask, ss, agg=O.AGG_TOKEN_MEAN)
    assert tm["loss"] == pytest.approx(g["loss_token_mean"], rel=1e-15)
    np.testing.assert_allclose(tm["grad_logp"][mask != 0], g["grad_token_mean"], rtol=1e-15)
    sm = O.sft_loss_fwd(logp, mask, ss, agg=O.AGG_SEQ_MEAN_TOKEN_MEAN)
    assert sm["loss"] == pytest.approx(g["loss_seq_mean"], rel=1e-15)
    assert sm["grad_logp"][0] == pytest.approx(g["grad_seq_mean"][0], rel=1e-15)
    np.testing.assert_allclose(sm["grad_logp"][3:6], g["grad_seq_mean"][1], rtol=1e-15)
    assert np.all(sm["grad_logp"][mask == 0] == 0)


def test_sft_matches_mix_all_expert_and_finite_differences():
    """Token-mean SFT is the MIX loss with every rollout an expert one and
    mu = 1 (a separate code path); bad ids are left out of both; central
    differences of the loss in each logp give the gradient."""
    ss, mask, logp, old, ref, adv, ids, V = _loss_case(seed=71)
    ids = ids.copy()
    ids[np.nonzero(mask)[0][3]] = V + 2           # one bad id
    sft = O.sft_loss_fwd(logp, mask, ss, ids, V, agg=O.AGG_TOKEN_MEAN)
    mix = O.ppo_clip_loss_fwd(logp, old, ref, adv, mask, ss, ids, V, 0.2, 0.2, 0.0, 0,
                              is_expert=np.ones(adv.size, np.uint8), mix_mu=1.0)
    assert sft["n_bad_ids"] == 1 == mix["n_bad_ids"]
    assert sft["loss"] == pytest.approx(mix["loss"], rel=1e-13)
    np.testing.assert_allclose(sft["grad_logp"], mix["grad_logp"], rtol=1e-13, atol=0)
    for agg in (0, 1):
        base = O.sft_loss_fwd(logp, mask, ss, ids, V, agg=agg, denom_override=3.5 * agg)
        for t in np.nonzero(mask)[0][:12]:
            lp1, lp2 = logp.copy(), logp.copy()
            lp1[t] += 1e-6
            lp2[t] -= 1e-6
            fd = (O.sft_loss_fwd(lp1, mask, ss, ids, V, agg=agg, denom_override=3.5 * agg)["loss"]
                  - O.sft_loss_fwd(lp2, mask, ss, ids, V, agg=agg,
                                   denom_override=3.5 * agg)["loss"]) / 2e-6
            assert fd == pytest.approx(base["grad_logp"][t], rel=1e-7, abs=1e-10)


# ------------------------------------------------------ DPO (R13) -----------
def _dpo_golden_layout():
    g = GOLD["dpo_single_pair"]
    ss = np.array([0, 2, 3], np.int32)
    mask = np.ones(3, np.uint8)
    logp = np.array(g["logp_chosen"] + g["logp_rejected"])
    ref = np.array(g["ref_chosen"] + g["ref_rejected"])
    return g, ss, mask, logp, ref


def test_golden_dpo_single_pair():
    g, ss, mask, logp, ref = _dpo_golden_layout()
    out = O.dpo_loss_fwd(logp, ref, mask, ss, beta=g["beta"])
    assert out["loss"] == pytest.approx(g["loss"], rel=1e-15)
    np.testing.assert_allclose(out["grad_logp"], [g["grad_chosen"]] * 2 + [g["grad_rejected"]],
                               rtol=1e-15)
    assert out["chosen_reward"] == pytest.approx(g["chosen_reward"], rel=1e-15)
    assert out["rejected_reward"] == pytest.approx(g["rejected_reward"], rel=1e-15)
    assert out["margin_mean"] == pytest.approx(g["margin"], rel=1e-15)
    assert out["reward_acc"] == 1.0 and out["n_pairs"] == 1
    ls = O.dpo_loss_fwd(logp, ref, mask, ss, beta=g["beta"], label_smoothing=0.1)
    assert ls["loss"] == pytest.approx(g["loss_label_smoothing_0.1"], rel=1e-15)


def _dpo_case(seed, n_pairs=5, pad=6, V=30):
    rng = np.random.default_rng(seed)
    lens = rng.integers(1, pad + 1, size=2 * n_pairs)
    lens[3] = 0                                    # pair 1 has an empty rejected rollout
    ss, mask = _layout(lens, pad)
    T = mask.size
    logp = -rng.random(T) * 3
    ref = logp + rng.standard_normal(T) * 0.5
    ids = rng.integers(0, V, size=T)
    return ss, mask, logp, ref, ids, V


def test_dpo_policy_equals_reference():
    """pi = rho: every margin is 0, the loss is ln 2 whatever the smoothing,
    and each token's gradient is +-beta (2 ls - 1) / (2 P)."""
    ss, mask, logp, _, ids, V = _dpo_case(72)
    for ls in (0.0, 0.2):
        out = O.dpo_loss_fwd(logp, logp, mask, ss, ids, V, beta=0.3, label_smoothing=ls)
        P = out["n_pairs"]
        assert P == 4
        assert out["loss"] == pytest.approx(math.log(2.0), rel=1e-15)
        g = 0.3 * (2 * ls - 1) / (2 * P)
        for s_ in range(len(ss) - 1):
            k, role = divmod(s_, 2)
            want = 0.0 if k == 1 else (g if role == 0 else -g)
            rr = [t for t in range(ss[s_], ss[s_ + 1]) if mask[t]]
            np.testing.assert_allclose(out["grad_logp"][rr], want, rtol=1e-14, atol=0)


def test_dpo_swap_identity():
    """Swapping chosen and rejected turns each -log sigmoid(u) into
    -log sigmoid(-u) = -log sigmoid(u) + u: the mean loss grows by the mean
    margin, and the tokens of the new chosen rollout get -beta sigmoid(u) / P,
    those of the new rejected one +beta sigmoid(u) / P."""
    ss, mask, logp, ref, ids, V = _dpo_case(73)
    beta = 0.2
    out = O.dpo_loss_fwd(logp, ref, mask, ss, ids, V, beta=beta)
    n_seq = len(ss) - 1
    lens = np.diff(ss)
    perm = np.arange(n_seq).reshape(-1, 2)[:, ::-1].ravel()
    rows = np.concatenate([np.arange(ss[i], ss[i + 1]) for i in perm])
    ss2 = np.concatenate([[0], np.cumsum(lens[perm])]).astype(np.int32)
    sw = O.dpo_loss_fwd(logp[rows], ref[rows], mask[rows], ss2, ids[rows], V, beta=beta)
    assert sw["loss"] == pytest.approx(out["loss"] + out["margin_mean"], rel=1e-13)
    assert sw["margin_mean"] == pytest.approx(-out["margin_mean"], rel=1e-13)
    P = out["n_pairs"]
    seq2 = np.searchsorted(ss2, np.arange(rows.size), side="right") - 1
    for t in np.nonzero(mask[rows])[0]:
        pair, role = divmod(int(seq2[t]), 2)
        if not out["pair_counted"][pair]:
            assert sw["grad_logp"][t] == 0.0
            continue
        sg = 1.0 / (1.0 + math.exp(-out["margins"][pair]))
        want = -beta * sg / P if role == 0 else beta * sg / P
        assert sw["grad_logp"][t] == pytest.approx(want, rel=1e-12)


def test_dpo_torch_autograd_and_bad_ids():
    """torch float64 autograd of the naive pairwise expression (segment sums
    by index_add, F.logsigmoid) as a third implementation; a bad id is left out
    of the sums and gets no gradient."""
    ss, mask, logp, ref, ids, V = _dpo_case(74)
    ids = ids.copy()
    bad_t = int(np.nonzero(mask)[0][5])
    ids[bad_t] = -1
    beta, ls = 0.15, 0.05
    out = O.dpo_loss_fwd(logp, ref, mask, ss, ids, V, beta=beta, label_smoothing=ls)
    assert out["n_bad_ids"] == 1 and out["grad_logp"][bad_t] == 0.0
    T = mask.size
    keep = torch.tensor((mask != 0) & (ids >= 0) & (ids < V), dtype=torch.float64)
    seq = torch.tensor(np.searchsorted(ss, np.arange(T), side="right") - 1)
    lp = torch.tensor(logp, requires_grad=True)
    n_seq = len(ss) - 1
    pi = torch.zeros(n_seq, dtype=torch.float64).index_add(0, seq, lp * keep)
    rho = torch.zeros(n_seq, dtype=torch.float64).index_add(0, seq, torch.tensor(ref) * keep)
    n_i = torch.zeros(n_seq, dtype=torch.float64).index_add(0, seq,
                                                              torch.tensor(mask, dtype=torch.float64))
    u = beta * ((pi[0::2] - rho[0::2]) - (pi[1::2] - rho[1::2]))
    ok = (n_i[0::2] > 0) & (n_i[1::2] > 0)
    lk = -(1 - ls) * torch.nn.functional.logsigmoid(u) - ls * torch.nn.functional.logsigmoid(-u)
    loss = lk[ok].sum() / ok.sum()
    loss.backward()
    assert loss.item() == pytest.approx(out["loss"], rel=1e-13)
    np.testing.assert_allclose(out["grad_logp"], lp.grad.numpy(), rtol=1e-12, atol=1e-16)
    assert out["reward_acc"] == pytest.approx(float((u[ok] > 0).double().mean()), rel=1e-15)


# ------------------------------------------------- advantage variants (R14) --
def test_golden_advantages_variable_groups():
    g = GOLD["advantages_variable_groups"]
    r, gid = np.array(g["rewards"]), np.array(g["group_id"])
    np.testing.assert_allclose(O.group_advantages_ids(r, gid, O.ADV_MEAN_CENTER),
                               g["mean_center"], rtol=1e-15, atol=1e-15)
    np.testing.assert_allclose(O.group_advantages_ids(r, gid, O.ADV_LEAVE_ONE_OUT),
                               g["leave_one_out"], rtol=1e-15, atol=1e-15)
    np.testing.assert_allclose(O.group_advantages_ids(r, gid, O.ADV_GRPO, eps=0.0),
                               g["grpo_eps0"], rtol=1e-14, atol=1e-15)


def test_advantages_ids_contiguous_equals_grpo_and_identities():
    """Contiguous ids reproduce the fixed-size GRPO advantages (a separate
    implementation); mean-centred values sum to 0 per group; leave-one-out is
    G / (G - 1) times mean-centred; a permutation of the rollouts permutes the
    advantages; leaving rollouts out equals computing on the rest alone."""
    rng = np.random.default_rng(81)
    G, ng = 8, 12
    r = rng.random(G * ng)
    r[16:24] = 0.5                                  # a degenerate group
    gid = np.repeat(np.arange(ng), G)
    np.testing.assert_allclose(O.group_advantages_ids(r, gid, O.ADV_GRPO, 1e-6),
                               O.group_advantages(r, G, 1e-6), rtol=1e-13, atol=1e-15)
    gid2 = rng.integers(-1, 9, size=r.size)
    mc = O.group_advantages_ids(r, gid2, O.ADV_MEAN_CENTER)
    lo = O.group_advantages_ids(r, gid2, O.ADV_LEAVE_ONE_OUT)
    for g in range(9):
        idx = np.nonzero(gid2 == g)[0]
        if idx.size >= 2:
            assert abs(mc[idx].sum()) < 1e-12
            np.testing.assert_allclose(lo[idx], idx.size / (idx.size - 1) * mc[idx], rtol=1e-12,
                                       atol=1e-15)
        else:
            assert np.all(mc[idx] == 0) and np.all(lo[idx] == 0)
    assert np.all(mc[gid2 < 0] == 0)
    perm = rng.permutation(r.size)
    for mode in (O.ADV_GRPO, O.ADV_MEAN_CENTER, O.ADV_LEAVE_ONE_OUT):
        a = O.group_advantages_ids(r, gid2, mode)
        np.testing.assert_allclose(O.group_advantages_ids(r[perm], gid2[perm], mode), a[perm],
                                   rtol=1e-13, atol=1e-15)
        keep = gid2 >= 0
        np.testing.assert_allclose(O.group_advantages_ids(r[keep], gid2[keep], mode), a[keep],
                                   rtol=1e-13, atol=1e-15)
        # ids at or above the group count leave their rollouts out as well
        a7 = O.group_advantages_ids(r, gid2, mode, n_groups=7)
        k7 = gid2 < 7
        np.testing.assert_allclose(a7[k7], O.group_advantages_ids(r[k7], gid2[k7], mode),
                                   rtol=1e-13, atol=1e-15)
        assert np.all(a7[~k7] == 0)


def test_advantages_population_std():
    """Population std (divisor G): numpy's std with ddof=0 (library routine),
    the G = 2 closed form (std 1/2), and A_pop = A_sample sqrt(G / (G - 1))
    at eps = 0."""
    rng = np.random.default_rng(91)
    G = 8
    r = rng.random(G * 5)
    a = O.group_advantages(r, G, 0.0, unbiased=False)
    for g0 in range(0, r.size, G):
        grp = r[g0:g0 + G]
        np.testing.assert_allclose(a[g0:g0 + G], (grp - grp.mean()) / np.std(grp, ddof=0),
                                   rtol=1e-12)
    np.testing.assert_allclose(a, O.group_advantages(r, G, 0.0) * math.sqrt(G / (G - 1)),
                               rtol=1e-12)
    two = O.group_advantages(np.array([0.0, 1.0]), 2, 1e-6, unbiased=False)
    np.testing.assert_allclose(two, [-0.5 / (0.5 + 1e-6), 0.5 / (0.5 + 1e-6)], rtol=1e-15)
    gid = np.repeat(np.arange(5), G)
    np.testing.assert_allclose(O.group_advantages_ids(r, gid, O.ADV_GRPO, 0.0, unbiased=False),
                               a, rtol=1e-12)


def test_masked_vocabulary_equals_removed_entries():
    """Reading R15: logits of -inf act as entries removed from the vocabulary.
    Log-prob, entropy and lse equal those of the reduced rows; the logit
    gradient with the entropy bonus is the reduced rows' gradient, with 0 at
    the masked columns; the entropy equals scipy's entr (0 log 0 = 0) summed
    over the softmax."""
    rng = np.random.default_rng(15)
    T, V = 9, 40
    z = rng.standard_normal((T, V)) * 2
    ids = rng.integers(0, V, size=T)
    keep = np.ones((T, V), bool)
    for t in range(T):                                   # row 0 stays unmasked
        others = np.setdiff1d(np.arange(V), [ids[t]])
        keep[t, rng.choice(others, size=4 * t, replace=False)] = False
    zm = np.where(keep, z, -np.inf)
    mask = np.ones(T, np.uint8)
    lp, en, ls = O.token_logprobs_from_logits(zm, ids, mask)
    assert np.all(np.isfinite(lp)) and np.all(np.isfinite(en)) and np.all(np.isfinite(ls))
    np.testing.assert_allclose(en, scipy.special.entr(scipy.special.softmax(zm, axis=1)).sum(1),
                               rtol=1e-12)
    np.testing.assert_allclose(ls, scipy.special.logsumexp(zm, axis=1), rtol=1e-13)
    c = rng.standard_normal(T)
    e = rng.random(T)
    g = O.bwd_logits(zm, ls, c, ids, mask, grad_entropy=e, entropy=en)
    for t in range(T):
        zr = z[t, keep[t]][None, :]
        yr = np.array([np.count_nonzero(keep[t, :ids[t]])])
        one = np.ones(1, np.uint8)
        lp_r, en_r, ls_r = O.token_logprobs_from_logits(zr, yr, one)
        assert lp[t] == pytest.approx(lp_r[0], abs=1e-12)
        assert en[t] == pytest.approx(en_r[0], abs=1e-12)
        assert ls[t] == pytest.approx(ls_r[0], abs=1e-12)
        g_r = O.bwd_logits(zr, ls_r, c[t:t + 1], yr, one, grad_entropy=e[t:t + 1],
                           entropy=en_r)[0]
        np.testing.assert_allclose(g[t][keep[t]], g_r, rtol=0, atol=1e-13)
        assert np.all(g[t][~keep[t]] == 0.0)
