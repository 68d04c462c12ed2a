"""GPU parity of the HIP path against the float64 oracle, through the C ABI,
at sizes the oracle finishes in seconds (several tiles plus ragged tails)."""
import math
import zlib

import numpy as np
import pytest
import torch

import paper_2505_17826_amd as R
from gen import synth
from oracle import rft_oracle as O
from tests.gpu_cases import (TOL_ADV, TOL_GRAD_FRO, TOL_LOGP, TOL_LOSS_ABS, TOL_LOSS_REL,
                             compare_step, cpu, f32, gpu_step, oracle_eps, oracle_step,
                             params_of, perturbed_logprobs, rel_fro, requires_gpu, tokens_of)

pytestmark = [pytest.mark.gpu, requires_gpu]
DEV = torch.device("cuda")

# reduced bf16 shapes: (name, overrides) - ragged lengths, vocab and hidden sizes
# that are not multiples of the 256x256 tile or the K step of 64
BF16_CASES = [
    ("ragged-2x8-d200-V4099", dict(n_prompts=2, group=8, len_lo=1, len_hi=300, pad_to=300, d=200,
                                   V=4099, dtype="bf16")),
    ("1x4-d8-V7", dict(n_prompts=1, group=4, len_lo=1, len_hi=40, pad_to=40, d=8, V=7,
                       dtype="bf16")),
    ("2x8-d72-V513", dict(n_prompts=2, group=8, len_lo=20, len_hi=90, pad_to=96, d=72, V=513,
                          dtype="bf16")),
    ("1x8-d256-V1", dict(n_prompts=1, group=8, len_lo=3, len_hi=9, pad_to=9, d=256, V=1,
                         dtype="bf16")),
    ("4x16-d128-V2048-tokmean", dict(n_prompts=4, group=16, len_lo=30, len_hi=130, pad_to=130,
                                     d=128, V=2048, dtype="bf16")),
]


def _batch(cid, name, over, poison=False):
    cfg = synth.config(cid, **over)
    return synth.make_batch(cfg, "cpu", poison=poison, seed_key=(cid, zlib.crc32(name.encode()) % 100003))


# --------------------------------------------------------------- advantages --
@pytest.mark.parametrize("G", [1, 2, 8, 16, 33, 100])
def test_group_advantages(G):
    rng = np.random.default_rng(G)
    n_groups = 37
    r = rng.standard_normal(n_groups * G).astype(np.float32)
    r[:G] = 0.25                                   # degenerate group
    if G >= 4:
        r[G:2 * G] = (rng.random(G) < 0.5).astype(np.float32)   # binary rewards
    for unbiased in (True, False):
        a = R.rft_group_advantages(torch.from_numpy(r).to(DEV), G, unbiased=unbiased)
        torch.cuda.synchronize()
        got = cpu(a)
        exp = O.group_advantages(r.astype(np.float64), G, f32(1e-6), unbiased=unbiased)
        assert np.all(got[:G] == 0.0)
        np.testing.assert_allclose(got, exp, atol=TOL_ADV, rtol=0)


# -------------------------------------------------------------- whole step --
def test_whole_step_tiny_fp32():
    """The tiny fp32 workload (4 prompts x 8 rollouts x 8 tokens, d=64, V=512)."""
    b = synth.make_batch(synth.config(0), "cpu")
    lp, _, _ = O.token_logprobs(b.H, b.W, b.ids, b.mask)
    old, ref = perturbed_logprobs(lp, b)
    g = gpu_step(b, old, ref)
    o = oracle_step(b, old, ref)
    compare_step(g, o, b)
    # fp32 arithmetic: much tighter than the bar
    assert np.abs(g["logp"] - o["logp"]).max() < 1e-4
    assert rel_fro(g["dW"], o["dW"]) < 1e-4


@pytest.mark.parametrize("name,over", BF16_CASES, ids=[c[0] for c in BF16_CASES])
def test_whole_step_bf16(name, over):
    cid = 3 if "tokmean" in name else 1
    b = _batch(cid, name, over)
    lp, _, _ = O.token_logprobs(b.H, b.W, b.ids, b.mask)
    old, ref = perturbed_logprobs(lp, b)
    g = gpu_step(b, old, ref)
    o = oracle_step(b, old, ref)
    compare_step(g, o, b)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_backward_small_workspace_chunks(dtype):
    """A workspace that only fits one row chunk at a time: several chunks, the
    last one ragged, dW accumulated across chunks."""
    over = dict(n_prompts=3, group=8, len_lo=10, len_hi=120, pad_to=120, d=96, V=1000, dtype=dtype)
    b = _batch(2, "chunks" + dtype, over)
    lp, _, _ = O.token_logprobs(b.H, b.W, b.ids, b.mask)
    old, ref = perturbed_logprobs(lp, b)
    tok = tokens_of(b)
    dt = R.RFT_BF16 if dtype == "bf16" else R.RFT_F32
    mn = R.workspace_bytes(R.RFT_OP_PPO_BWD, tok, 96, 1000, dt, minimum=True)
    g = gpu_step(b, old, ref, ws_bwd_bytes=mn)
    o = oracle_step(b, old, ref)
    compare_step(g, o, b)


def test_accumulate_dw():
    over = dict(n_prompts=1, group=8, len_lo=10, len_hi=60, pad_to=64, d=64, V=700, dtype="bf16")
    b = _batch(1, "acc", over)
    lp, _, lse = O.token_logprobs(b.H, b.W, b.ids, b.mask)
    tok = tokens_of(b)
    H, W = b.H.to(DEV), b.W.to(DEV)
    c = synth.extra_normal(b.T, (91,), "cpu", std=1e-3)
    c[b.mask == 0] = 0
    prior = synth.extra_normal((700, 64), (92,), "cpu")
    dW = prior.to(DEV).clone()
    R.rft_ppo_clip_loss_bwd(tok, H, W, torch.from_numpy(lse.astype(np.float32)).to(DEV),
                            c.to(DEV), d_weight=dW, accumulate_dw=True)
    torch.cuda.synchronize()
    _, odW = O.ppo_clip_loss_bwd(b.H, b.W, lse, c, b.ids, b.mask)
    assert rel_fro(cpu(dW) - prior.double().numpy(), odW) <= TOL_GRAD_FRO


# ----------------------------------------------------------- loss alone ----
@pytest.mark.parametrize("agg,eps_hi,denom", [(0, 0.2, 0.0), (1, 0.28, 0.0), (0, 0.2, 5.0),
                                              (1, math.inf, 100.0)])
def test_loss_fwd_bit_exact_decisions(agg, eps_hi, denom):
    """Same fp32 inputs on both sides: clip decisions and counts agree exactly."""
    cfg = synth.config(1, n_prompts=8, group=8, len_lo=1, len_hi=200, pad_to=200, d=8, V=1000,
                       eps_high=eps_hi, agg=agg, beta=0.05)
    b = synth.make_batch(cfg, "cpu", seed_key=(77, agg))
    rng = np.random.default_rng(5)
    T = b.T
    m = b.mask.numpy() != 0
    logp = np.where(m, -rng.random(T) * 12, 0).astype(np.float32)
    old = np.where(m, logp + rng.standard_normal(T) * 0.3, 0).astype(np.float32)
    ref = np.where(m, logp + rng.standard_normal(T) * 0.3, 0).astype(np.float32)
    adv = O.group_advantages(b.rewards.numpy(), cfg.group).astype(np.float32)
    ent = np.where(m, rng.random(T) * 10, 0).astype(np.float32)
    tok = tokens_of(b)
    t = lambda x: torch.from_numpy(x).to(DEV)
    grad, st = R.rft_ppo_clip_loss_fwd(tok, cfg.V, t(logp), t(old), t(ref), t(adv),
                                       params_of(cfg, denom), entropy=t(ent))
    torch.cuda.synchronize()
    s = R.stats_to_dict(st)
    el, eh, be = oracle_eps(cfg)
    o = O.ppo_clip_loss_fwd(logp, old, ref, adv, b.mask, b.seq_start, b.ids, cfg.V, el, eh, be,
                            agg, denom, entropy=ent)
    # The kernel decides in fp32 on logp - old, the oracle by the definition
    # in fp64: they may differ only for a token within 1e-6 of a bound.
    near = o["margin"] < 1e-6
    n_near = int(near.sum())
    print(f"[loss-fwd agg={agg} eps_hi={eps_hi}] clipped {o['n_clipped']}, "
          f"{n_near} tokens within 1e-6 of a bound", flush=True)
    assert abs(s["n_clipped"] - o["n_clipped"]) <= n_near and o["n_clipped"] > 0
    assert s["n_valid"] == o["n_valid"] and s["n_seq_valid"] == o["n_seq_valid"]
    assert s["n_bad_ids"] == 0
    for k in ("loss", "pg_loss", "kl_loss", "entropy_loss"):
        assert abs(s[k] - o[k]) <= TOL_LOSS_REL * abs(o[k]) + TOL_LOSS_ABS, (k, s[k], o[k])
    for k in ("kl_mean", "ratio_mean", "entropy_mean"):
        assert abs(s[k] - o[k]) <= 1e-5 * max(1.0, abs(o[k])), (k, s[k], o[k])
    assert abs(s["clipfrac"] - o["clipfrac"]) <= n_near / o["n_valid"] + 1e-12
    g = cpu(grad)
    assert np.all(g[~m] == 0)
    rows = o["weights_rows"][~near]
    np.testing.assert_allclose(g[rows], o["grad_logp"][rows], rtol=1e-4,
                               atol=1e-7 * np.abs(o["grad_logp"]).max())


def test_loss_ratio_one_is_minus_mean_advantage():
    cfg = synth.config(1, n_prompts=4, group=8, len_lo=5, len_hi=50, pad_to=50, d=8, V=100,
                       beta=0.0)
    b = synth.make_batch(cfg, "cpu", seed_key=(78,))
    m = b.mask.numpy() != 0
    logp = np.where(m, -1.5, 0).astype(np.float32)
    adv = np.random.default_rng(0).standard_normal(cfg.n_seq).astype(np.float32)
    tok = tokens_of(b)
    t = lambda x: torch.from_numpy(x).to(DEV)
    _, st = R.rft_ppo_clip_loss_fwd(tok, cfg.V, t(logp), t(logp), None, t(adv), params_of(cfg))
    torch.cuda.synchronize()
    s = R.stats_to_dict(st)
    n = np.array([m[b.seq_start[i]:b.seq_start[i + 1]].sum() for i in range(cfg.n_seq)])
    expect = -adv[n > 0].astype(np.float64).mean()
    assert abs(s["loss"] - expect) <= 1e-6 * max(1, abs(expect))
    assert s["clipfrac"] == 0.0 and s["ratio_mean"] == pytest.approx(1.0, abs=1e-7)


# ---------------------------------------------------------- logits paths ----
# V = 8192: every thread's row chunks fit in registers (ragged across threads);
# 134692: the part kept in LDS ends mid-way; 152004: the LDS part ends just
# before its capacity (rows up to 153600 stay on chip); 160004: a ragged
# remainder past registers and LDS is read twice; 4099 and 1: scalar path.
@pytest.mark.parametrize("V,n_prompts", [(8192, 16), (4099, 16), (1, 16), (134692, 2),
                                         (152004, 2), (160004, 2)])
def test_logits_paths(V, n_prompts):
    cfg = synth.config(4, n_prompts=n_prompts, group=8, V=V)  # 8 seqs per prompt x 16 tokens
    b = synth.make_batch(cfg, "cpu", seed_key=(4, V))
    lp, ent, lse = O.token_logprobs_from_logits(b.logits, b.ids, b.mask)
    old, ref = perturbed_logprobs(lp, b)
    el, eh, be = oracle_eps(cfg)
    o = O.loss_only_step(b.logits, b.ids, b.mask, b.seq_start, b.rewards, cfg.group,
                         old.astype(np.float64), ref.astype(np.float64), el, eh, be, cfg.agg)
    tok = tokens_of(b)
    L = b.logits.to(DEV)
    t = lambda x: torch.from_numpy(x).to(DEV)
    adv = R.rft_group_advantages(b.rewards.to(DEV), cfg.group)
    # statistics only
    glp, gent, glse, gath = R.rft_token_logprobs_from_logits(tok, L, want_gathered=True)
    # fused
    flp = torch.empty_like(glp); fent = torch.empty_like(glp); flse = torch.empty_like(glp)
    fgrad = torch.empty_like(glp)
    _, fdl, fst = R.rft_ppo_clip_fused_logits(tok, L, t(old), t(ref), adv, params_of(cfg),
                                              logp=flp, entropy=fent, lse=flse, grad_logp=fgrad)
    # unfused composition
    ugrad, ust = R.rft_ppo_clip_loss_fwd(tok, V, glp, t(old), t(ref), adv, params_of(cfg),
                                         entropy=gent)
    udl = R.rft_ppo_clip_loss_bwd_logits(tok, L, glse, ugrad)
    torch.cuda.synchronize()
    m = b.mask.numpy() != 0
    ids = b.ids.numpy()
    # gathered logit is a bit-exact copy
    gg = gath.cpu().numpy()
    rr = np.nonzero(m)[0]
    assert np.array_equal(gg[rr], b.logits.numpy()[rr, ids[rr]])
    assert np.all(gg[~m] == 0)
    for got in (cpu(glp), cpu(flp)):
        assert np.all(got[~m] == 0)
        assert np.abs(got[m] - o["logp"][m]).max() <= TOL_LOGP
    for got in (cpu(gent), cpu(fent)):
        assert np.abs(got[m] - o["entropy"][m]).max() <= TOL_LOGP
    for got in (cpu(glse), cpu(flse)):
        assert np.abs(got[m] - o["lse"][m]).max() <= TOL_LOGP
    for st in (R.stats_to_dict(fst), R.stats_to_dict(ust)):
        assert st["n_valid"] == o["fwd"]["n_valid"]
        assert abs(st["loss"] - o["fwd"]["loss"]) <= TOL_LOSS_REL * abs(o["fwd"]["loss"]) + TOL_LOSS_ABS
    # fused and unfused paths give the same numbers (same kernels' arithmetic)
    assert torch.equal(flp, glp) and torch.equal(flse, glse)
    assert torch.equal(fgrad, ugrad)
    # d logits
    dl_o = np.zeros(b.logits.shape)
    for r_, v in o["dlogits"].items():
        dl_o[r_] = v
    for dl in (cpu(fdl), cpu(udl)):
        assert np.all(dl[~m] == 0)
        assert rel_fro(dl, dl_o) <= TOL_GRAD_FRO, rel_fro(dl, dl_o)
    assert torch.equal(fdl, udl)


# --------------------------------------------------------------- edge cases --
@pytest.mark.parametrize("d,V,n_prompts", [(128, 2048, 4), (192, 5003, 6), (64, 300, 1)])
def test_token_logprobs_blocked_equals_row_major(d, V, n_prompts):
    """rft_token_logprobs with the recommended workspace (tile-blocked copies,
    384 x 256 GEMM tiles) and with the minimum workspace (row-major operands,
    256 x 256 tiles): the same numbers bit for bit, and the oracle's."""
    over = dict(n_prompts=n_prompts, group=8, len_lo=1, len_hi=200, pad_to=200, d=d, V=V,
                dtype="bf16")
    b = _batch(1, f"blk{d}-{V}", over)
    print(f"[fwd blocked] d={d} V={V} T={b.T} N={int(b.mask.sum())}", flush=True)
    tok = tokens_of(b)
    H, W = b.H.to(DEV).contiguous(), b.W.to(DEV).contiguous()
    big = R.workspace_bytes(R.RFT_OP_TOKEN_LOGPROBS, tok, d, V, R.RFT_BF16)
    small = R.workspace_bytes(R.RFT_OP_TOKEN_LOGPROBS, tok, d, V, R.RFT_BF16, minimum=True)
    assert big > small
    outs = []
    for nb in (big, small):
        ws = torch.empty(nb, dtype=torch.uint8, device=DEV)
        outs.append([cpu(x) for x in R.rft_token_logprobs(tok, H, W, ws=ws)])
    torch.cuda.synchronize()
    for a_, b_, k in zip(outs[0], outs[1], ("logp", "entropy", "lse")):
        assert np.array_equal(a_, b_), (k, np.nanmax(np.abs(a_ - b_)))
    m = b.mask.numpy() != 0
    for got, want, k in zip(outs[0], O.token_logprobs(b.H, b.W, b.ids, b.mask),
                            ("logp", "entropy", "lse")):
        assert np.abs(got[m] - np.asarray(want)[m]).max() <= TOL_LOGP, k


def test_all_masked_batch():
    cfg = synth.config(1, n_prompts=1, group=8, len_lo=0, len_hi=0, pad_to=16, d=64, V=300)
    b = synth.make_batch(cfg, "cpu", seed_key=(3,))
    assert int(b.mask.sum()) == 0
    z = np.zeros(b.T, np.float32)
    g = gpu_step(b, z, z)
    assert g["stats"]["loss"] == 0.0 and g["stats"]["n_valid"] == 0
    assert np.all(g["logp"] == 0) and np.all(g["grad_logp"] == 0)
    assert np.all(g["dH"] == 0) and np.all(g["dW"] == 0)


def test_empty_batch():
    tok = R.Tokens(torch.zeros(1, dtype=torch.int32, device=DEV),
                   torch.zeros(0, dtype=torch.uint8, device=DEV),
                   torch.zeros(0, dtype=torch.int32, device=DEV))
    H = torch.zeros((0, 64), dtype=torch.bfloat16, device=DEV)
    W = torch.randn((50, 64), device=DEV).to(torch.bfloat16)
    logp, ent, lse = R.rft_token_logprobs(tok, H, W)
    e = torch.zeros(0, device=DEV)
    grad, st = R.rft_ppo_clip_loss_fwd(tok, 50, e, e, e, e, R.ppo_params(kl_coef=0.1))
    dW = torch.full((50, 64), 7.0, device=DEV)
    R.rft_ppo_clip_loss_bwd(tok, H, W, e, e, d_hidden=torch.zeros((0, 64), device=DEV), d_weight=dW)
    torch.cuda.synchronize()
    assert R.stats_to_dict(st)["loss"] == 0.0
    assert torch.all(dW == 0)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_nan_poisoned_padding_is_never_read(dtype):
    over = dict(n_prompts=2, group=4, len_lo=5, len_hi=70, pad_to=80, d=64, V=600, dtype=dtype)
    b0 = _batch(1, "poison", over, poison=False)
    b1 = _batch(1, "poison", over, poison=True)
    m = b0.mask.numpy() != 0
    assert np.isnan(b1.H.float().numpy()[~m]).all() and (b1.ids.numpy()[~m] == 600 + 7).all()
    lp, _, _ = O.token_logprobs(b0.H, b0.W, b0.ids, b0.mask)
    old, ref = perturbed_logprobs(lp, b0)
    g0 = gpu_step(b0, old, ref)
    g1 = gpu_step(b1, old, ref)
    for k in ("logp", "entropy", "lse", "grad_logp", "dH", "dW"):
        assert np.array_equal(g0[k], g1[k]), k
    assert g0["stats"] == g1["stats"]


def test_poisoned_logits_rows():
    cfg = synth.config(4, n_prompts=4, group=8, V=1024)
    b0 = synth.make_batch(cfg, "cpu", seed_key=(9,))
    b1 = synth.make_batch(cfg, "cpu", seed_key=(9,), poison=True)
    tok0, tok1 = tokens_of(b0), tokens_of(b1)
    z = torch.zeros(b0.T, device=DEV)
    adv = torch.zeros(cfg.n_seq, device=DEV)
    outs = []
    for tok, b in ((tok0, b0), (tok1, b1)):
        lp, dl, st = R.rft_ppo_clip_fused_logits(tok, b.logits.to(DEV), z, z, adv, params_of(cfg))
        torch.cuda.synchronize()
        outs.append((cpu(lp), cpu(dl), R.stats_to_dict(st)))
    assert np.array_equal(outs[0][0], outs[1][0]) and np.array_equal(outs[0][1], outs[1][1])
    assert outs[0][2] == outs[1][2]


def test_out_of_range_ids():
    over = dict(n_prompts=1, group=8, len_lo=10, len_hi=30, pad_to=32, d=64, V=400, dtype="bf16")
    b = _batch(1, "badids", over)
    ids = b.ids.clone()
    valid = np.nonzero(b.mask.numpy())[0]
    ids[valid[0]] = 400
    ids[valid[5]] = -3
    b.ids = ids
    lp, _, _ = O.token_logprobs(b.H, b.W, b.ids, b.mask)
    lp_filled = np.nan_to_num(lp, nan=-5.0)
    old, ref = perturbed_logprobs(lp_filled, b)
    g = gpu_step(b, old, ref)
    assert np.isnan(g["logp"][valid[0]]) and np.isnan(g["logp"][valid[5]])
    assert g["stats"]["n_bad_ids"] == 2
    assert g["grad_logp"][valid[0]] == 0 and g["grad_logp"][valid[5]] == 0
    assert np.all(g["dH"][valid[0]] == 0) and np.all(g["dH"][valid[5]] == 0)
    o = oracle_step(b, old, ref)
    assert o["fwd"]["n_bad_ids"] == 2
    # every statistic, the per-token gradients and both weight gradients
    compare_step(g, o, b)


def test_run_to_run_determinism():
    over = dict(n_prompts=2, group=8, len_lo=50, len_hi=200, pad_to=200, d=128, V=3000, dtype="bf16")
    b = _batch(1, "det", over)
    lp, _, _ = O.token_logprobs(b.H, b.W, b.ids, b.mask)
    old, ref = perturbed_logprobs(lp, b)
    g1 = gpu_step(b, old, ref)
    g2 = gpu_step(b, old, ref)
    for k in ("adv", "logp", "entropy", "lse", "grad_logp", "dH", "dW"):
        assert np.array_equal(g1[k], g2[k]), k
    assert g1["stats"] == g2["stats"]


def test_counts_bit_exact():
    """Valid-token counts and the compaction agree with brute force bit-exactly
    (through the loss statistics, which report N and S)."""
    rng = np.random.default_rng(1)
    n_seq = 300
    lens = rng.integers(0, 50, size=n_seq)
    ss = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    T = int(ss[-1])
    mask = (rng.random(T) < 0.7).astype(np.uint8)
    tok = R.Tokens(torch.from_numpy(ss).to(DEV), torch.from_numpy(mask).to(DEV),
                   torch.zeros(T, dtype=torch.int32, device=DEV))
    z = torch.zeros(T, device=DEV)
    _, st = R.rft_ppo_clip_loss_fwd(tok, 10, z, z, None, torch.zeros(n_seq, device=DEV),
                                    R.ppo_params())
    torch.cuda.synchronize()
    s = R.stats_to_dict(st)
    c = O.token_counts(mask, ss)
    assert s["n_valid"] == c["N"] and s["n_seq_valid"] == c["S"]
