"""The entry point that allocates nothing (rft_ppo_clip_fused_logits_noalloc)
against the loss-only call with a workspace (rft_ppo_clip_fused_logits): the
same kernels on the same inputs, so every output must be bit-identical.  Two
calls in a row, the second with a smaller layout (the library's scratch keeps
the first call's contents), then one at the largest supported row count."""
import numpy as np
import pytest
import torch

import paper_2505_17826_amd as R
from gen import synth
from tests.gpu_cases import params_of, requires_gpu, tokens_of

pytestmark = [pytest.mark.gpu, requires_gpu]
DEV = torch.device("cuda")


def _inputs(n_prompts, V, key):
    cfg = synth.config(4, n_prompts=n_prompts, group=8, V=V)
    b = synth.make_batch(cfg, DEV, seed_key=(4, key))
    m = b.mask.bool()
    # old / ref: a plain offset from -ln V plus the batch's noise (inputs only)
    base = torch.full((b.T,), -float(np.log(V)), device=DEV)
    old = torch.where(m, base + b.old_noise, torch.zeros_like(base))
    ref = torch.where(m, base + b.ref_noise, torch.zeros_like(base))
    adv = R.rft_group_advantages(b.rewards, cfg.group)
    return cfg, b, tokens_of(b), old, ref, adv


def _outputs(T, V):
    f = lambda: torch.full((T,), 7.0, device=DEV)
    return (f(), f(), f(), f(), torch.full((T, V), 7.0, device=DEV),
            torch.full((R.STATS_BYTES,), 255, dtype=torch.uint8, device=DEV))


def _both(n_prompts, V, key):
    cfg, b, tok, old, ref, adv = _inputs(n_prompts, V, key)
    p = params_of(cfg)
    a = _outputs(b.T, V)
    R.rft_ppo_clip_fused_logits(tok, b.logits, old, ref, adv, p, logp=a[0], entropy=a[1],
                                lse=a[2], grad_logp=a[3], d_logits=a[4], stats=a[5])
    z = _outputs(b.T, V)
    R.rft_ppo_clip_fused_logits_noalloc(tok, b.logits, old, ref, adv, p, logp=z[0], d_logits=z[4],
                                        stats=z[5], entropy=z[1], lse=z[2], grad_logp=z[3])
    torch.cuda.synchronize()
    for name, x, y in zip(("logp", "entropy", "lse", "grad_logp", "d_logits"), a[:5], z[:5]):
        assert torch.equal(x, y), name
    sa, sz = R.stats_to_dict(a[5]), R.stats_to_dict(z[5])
    assert sa == sz
    assert sa["n_valid"] == int(b.mask.sum())
    return sa


def test_noalloc_matches_workspace_call_twice_then_smaller():
    print("[noalloc] call 1: T=2048 V=8192", flush=True)
    s1 = _both(16, 8192, 11)
    print("[noalloc] call 2: T=512 V=5000 (smaller)", flush=True)
    s2 = _both(4, 5000, 12)
    assert s1["n_valid"] > s2["n_valid"] > 0


def test_noalloc_largest_layout_and_rejection():
    # 131072 rows (1024 prompts x 8 rollouts x 16 tokens): the documented limit
    print("[noalloc] T=131072 V=512", flush=True)
    _both(1024, 512, 13)
    print("[noalloc] T=512 after the largest", flush=True)
    _both(4, 700, 14)
    # a layout whose scratch does not fit is refused before anything runs
    T = 200000
    tok = R.Tokens(torch.zeros(2, dtype=torch.int32, device=DEV).index_fill_(0, torch.tensor([1], device=DEV), T),
                   torch.ones(T, dtype=torch.uint8, device=DEV),
                   torch.zeros(T, dtype=torch.int32, device=DEV))
    z = torch.zeros(T, device=DEV)
    with pytest.raises(R.RftError) as ei:
        R.rft_ppo_clip_fused_logits_noalloc(tok, torch.zeros((T, 4), device=DEV), z, z,
                                            torch.zeros(1, device=DEV), R.ppo_params(), logp=z,
                                            d_logits=torch.zeros((T, 4), device=DEV),
                                            stats=torch.zeros(R.STATS_BYTES, dtype=torch.uint8,
                                                              device=DEV))
    assert ei.value.status == R.RFT_E_WORKSPACE
