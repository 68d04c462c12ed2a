"""GPU parity of the fused trainer step (rft_ppo_clip_step) against the float64
oracle and against the separate calls it replaces: log-probs, entropy, lse,
per-token gradients and the loss statistics are the same numbers bit for bit
(same kernels' arithmetic and reduction order), the weight and hidden
gradients agree with the oracle to the gradient tolerance (dZ is formed from
the fp16-stored logits instead of a recomputation)."""
import zlib

import numpy as np
import pytest
import torch

import paper_2505_17826_amd as R
from gen import synth
from oracle import rft_oracle as O
from tests.gpu_cases import (TOL_GRAD_FRO, compare_step, gpu_fused_step, gpu_step, oracle_step,
                             perturbed_logprobs, rel_fro, requires_gpu, tokens_of)
from tests.test_parity_gpu import BF16_CASES

pytestmark = [pytest.mark.gpu, requires_gpu]


def _batch(cid, name, over):
    cfg = synth.config(cid, **over)
    return synth.make_batch(cfg, "cpu", seed_key=(cid, zlib.crc32(("step" + name).encode()) % 100003))


def _same_fwd(gf, gs):
    for k in ("logp", "entropy", "lse", "grad_logp"):
        a, b = gf[k], gs[k]
        assert np.array_equal(a, b, equal_nan=True), (k, np.nanmax(np.abs(a - b)))
    for k in ("loss", "pg_loss", "kl_loss", "kl_mean", "entropy_mean", "ratio_mean", "clipfrac",
              "n_valid", "n_seq_valid", "n_clipped", "n_bad_ids"):
        assert gf["stats"][k] == gs["stats"][k], k


@pytest.mark.parametrize("name,over", BF16_CASES, ids=[c[0] for c in BF16_CASES])
def test_step_bf16(name, over):
    cid = 3 if "tokmean" in name else 1
    b = _batch(cid, name, over)
    print(f"[step] {name}", flush=True)
    lp, _, _ = O.token_logprobs(b.H, b.W, b.ids, b.mask)
    old, ref = perturbed_logprobs(lp, b)
    gf = gpu_fused_step(b, old, ref)
    o = oracle_step(b, old, ref)
    compare_step(gf, o, b)
    gs = gpu_step(b, old, ref)
    _same_fwd(gf, gs)
    # the two backward formulations agree far inside the oracle tolerance
    # (scaled by the oracle's gradient, which is exactly 0 when V = 1)
    for k in ("dW", "dH"):
        diff = np.linalg.norm(gf[k] - gs[k])
        assert diff <= 5e-3 * np.linalg.norm(o[k]) + 1e-6, (k, diff, np.linalg.norm(o[k]))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_step_small_workspace_chunks(dtype):
    """Minimum workspace: 256-row chunks, the last ragged, dW accumulated over
    the chunks inside the call."""
    over = dict(n_prompts=3, group=8, len_lo=10, len_hi=120, pad_to=120, d=96, V=1000, dtype=dtype)
    b = _batch(2, "chunks" + dtype, over)
    lp, _, _ = O.token_logprobs(b.H, b.W, b.ids, b.mask)
    old, ref = perturbed_logprobs(lp, b)
    dt = R.RFT_BF16 if dtype == "bf16" else R.RFT_F32
    mn = R.workspace_bytes(R.RFT_OP_PPO_STEP, tokens_of(b), 96, 1000, dt, minimum=True)
    assert mn < R.workspace_bytes(R.RFT_OP_PPO_STEP, tokens_of(b), 96, 1000, dt)
    gf = gpu_fused_step(b, old, ref, ws_bytes=mn)
    o = oracle_step(b, old, ref)
    compare_step(gf, o, b)
    _same_fwd(gf, gpu_step(b, old, ref))


def test_step_tiny_fp32():
    b = synth.make_batch(synth.config(0), "cpu", seed_key=(0, 77))
    lp, _, _ = O.token_logprobs(b.H, b.W, b.ids, b.mask)
    old, ref = perturbed_logprobs(lp, b)
    gf = gpu_fused_step(b, old, ref)
    o = oracle_step(b, old, ref)
    compare_step(gf, o, b)
    assert rel_fro(gf["dW"], o["dW"]) < 1e-4


def test_step_accumulate_dw():
    over = dict(n_prompts=1, group=8, len_lo=10, len_hi=60, pad_to=64, d=64, V=700, dtype="bf16")
    b = _batch(1, "acc", over)
    lp, _, _ = O.token_logprobs(b.H, b.W, b.ids, b.mask)
    old, ref = perturbed_logprobs(lp, b)
    o = oracle_step(b, old, ref)
    # a prior ten times the gradient's rms, so fp32 rounding of the sum stays small
    scale = 10.0 * float(np.sqrt(np.mean(o["dW"] ** 2)))
    x = (scale * np.random.default_rng(5).standard_normal((700, 64))).astype(np.float32)
    gf = gpu_fused_step(b, old, ref, dW_init=x)
    assert rel_fro(gf["dW"] - x, o["dW"]) <= TOL_GRAD_FRO


def test_step_all_masked_and_empty():
    cfg = synth.config(1, n_prompts=1, group=8, len_lo=0, len_hi=0, pad_to=16, d=64, V=300)
    b = synth.make_batch(cfg, "cpu", seed_key=(3, 9))
    assert int(b.mask.sum()) == 0
    z = np.zeros(b.T, np.float32)
    gf = gpu_fused_step(b, z, z)
    assert gf["stats"]["loss"] == 0.0 and gf["stats"]["n_valid"] == 0
    for k in ("logp", "entropy", "lse", "grad_logp", "dH", "dW"):
        assert np.all(gf[k] == 0), k
    # T = 0: no rows at all
    dev = torch.device("cuda")
    tok = R.Tokens(torch.zeros(2, dtype=torch.int32, device=dev),
                   torch.zeros(0, dtype=torch.uint8, device=dev),
                   torch.zeros(0, dtype=torch.int32, device=dev))
    W = torch.randn(300, 64, device=dev).to(torch.bfloat16)
    H = torch.zeros(0, 64, device=dev, dtype=torch.bfloat16)
    e = torch.zeros(0, device=dev)
    adv = torch.zeros(1, device=dev)
    out = R.rft_ppo_clip_step(tok, H, W, e, e, adv, R.ppo_params(0.2, 0.2, 0.01, 0))
    torch.cuda.synchronize()
    assert torch.all(out[5] == 0) and R.stats_to_dict(out[6])["n_valid"] == 0


def test_store_tile_choice_bit_identical(monkeypatch):
    """d_hidden and d_weight on 256 x 256 or 384 x 256 tiles (RFT_GEMM_STORE_TILE
    fixes the choice; unset, the round model picks one per call and, for
    d_hidden whose rows are counted on the device, on the device): the same
    numbers bit for bit, in the fused step (two row chunks) and in the
    separate backward."""
    over = dict(n_prompts=4, group=8, len_lo=100, len_hi=400, pad_to=400, d=128, V=3000,
                dtype="bf16")
    b = _batch(1, "storetile", over)
    lp, _, _ = O.token_logprobs(b.H, b.W, b.ids, b.mask)
    old, ref = perturbed_logprobs(lp, b)
    tok = tokens_of(b)
    N = int(b.mask.sum())
    ws = R.workspace_bytes_rows(R.RFT_OP_PPO_STEP, tok, 128, 3000, R.RFT_BF16, (N // 2 + 255) // 256 * 256)
    outs = {}
    for tile in ("256", "384", None):
        if tile is None:
            monkeypatch.delenv("RFT_GEMM_STORE_TILE", raising=False)
        else:
            monkeypatch.setenv("RFT_GEMM_STORE_TILE", tile)
        print(f"[store tile] {tile}", flush=True)
        outs[tile] = (gpu_fused_step(b, old, ref, ws_bytes=ws), gpu_step(b, old, ref))
    for tile in ("384", None):
        for i in range(2):
            for k in ("dH", "dW"):
                assert np.array_equal(outs[tile][i][k], outs["256"][i][k]), (tile, i, k)
    compare_step(outs["384"][0], oracle_step(b, old, ref), b)
