"""Seeded synthetic trainer batches.

Recipe (the same on every machine, up to the RNG of the device used for the
large arrays):

* Layout.  ``n_prompts * group`` rollouts.  Response lengths are integers
  drawn uniformly from the inclusive range ``[len_lo, len_hi]``; each rollout
  occupies ``pad_to`` rows of a padded ``[n_seq, pad_to]`` layout, the first
  ``L_i`` rows are response tokens (mask 1), the rest padding (mask 0).  With
  ``mask_frac > 0`` exactly ``round(mask_frac * T)`` rows, chosen without
  replacement, are masked instead (the loss-only workload).
* Hidden states ``H[T, d]`` ~ N(0, 1); lm_head weight ``W[V, d]`` =
  2 * N(0, 1) / sqrt(d) (logit variance 4 for unit-variance h), rounded to the
  input dtype with round-to-nearest-even.  Masked rows of ``H`` are zero, or
  NaN when ``poison=True``.
* Loss-only workload: ``logits[T, V]`` ~ N(0, 2^2) in fp32.
* ``logit_std`` (2 by default, the value above) scales W or the given logits;
  the stress tests raise it to 10-20, the spread of a trained model's logits,
  so that rows are peaked (a few entries carry most of the probability).
* Token ids are drawn from softmax of the rollout logits ``h . W^T`` (or of
  ``logits``) by the Gumbel-max rule ``argmax_j (z_j - log(-log u_j))``.
  This stands in for the rollout model of the explorer, not for the trainer;
  logits are formed in fp32 from the already-rounded inputs.
* Old / reference log-prob perturbations: N(0, 0.05) and N(0, 0.1), the
  second argument read as a variance.  The caller adds them to the current
  log-probs it has at hand (the oracle's, or the GPU's for timing only).
* Rewards: Bernoulli(0.5) per rollout, or Bernoulli(p_prompt) with
  p_prompt ~ U(0, 1) per prompt, or N(0, 1) per rollout.

Streams: numpy ``SeedSequence([2505, 17826, cfg, stream])`` for each stream in
the fixed order lengths, H, W, sampling, old-noise, ref-noise, rewards, mask,
logits.  Small arrays (layout, rewards, mask) come from numpy PCG64; the large
ones from a ``torch.Generator`` on the target device seeded from the same
stream, so full-size batches are generated on the GPU in seconds.
"""
from __future__ import annotations

import dataclasses
import math
from dataclasses import dataclass
from typing import Optional

import numpy as np
import torch

AGG_SEQ_MEAN_TOKEN_MEAN = 0
AGG_TOKEN_MEAN = 1

_STREAMS = ("lengths", "H", "W", "sampling", "old", "ref", "rewards", "mask",
            "logits", "extra")


@dataclass(frozen=True)
class Config:
    cid: int
    name: str
    n_prompts: int
    group: int
    len_lo: int
    len_hi: int
    pad_to: int
    d: int
    V: int
    dtype: str                 # "f32" | "bf16" | "logits"
    eps_low: float
    eps_high: float
    beta: float
    agg: int
    reward: str                # "bern05" | "bern_prompt" | "normal"
    mask_frac: float = 0.0
    old_var: float = 0.05
    ref_var: float = 0.1
    logit_std: float = 2.0     # std of the logits: W = logit_std N(0,1)/sqrt(d), or given logits

    @property
    def n_seq(self) -> int:
        return self.n_prompts * self.group

    @property
    def T(self) -> int:
        return self.n_seq * self.pad_to

    def replace(self, **kw) -> "Config":
        return dataclasses.replace(self, **kw)


CONFIGS = {
    0: Config(0, "tiny-fp32 T=256 d=64 V=512 G=8", 4, 8, 8, 8, 8, 64, 512, "f32",
              0.2, 0.2, 0.01, AGG_SEQ_MEAN_TOKEN_MEAN, "bern05"),
    1: Config(1, "1.5B-shape bf16 d=1536 V=151936 32x8 L=U[256,1024]", 32, 8, 256, 1024,
              1024, 1536, 151936, "bf16", 0.2, 0.2, 0.001, AGG_SEQ_MEAN_TOKEN_MEAN,
              "bern_prompt"),
    2: Config(2, "7B-shape bf16 d=3584 V=152064 16x8 L=U[512,2048]", 16, 8, 512, 2048,
              2048, 3584, 152064, "bf16", 0.2, 0.2, 0.001, AGG_SEQ_MEAN_TOKEN_MEAN,
              "bern_prompt"),
    3: Config(3, "long-CoT bf16 d=3584 V=152064 4x16 L=U[1024,8192]", 4, 16, 1024, 8192,
              8192, 3584, 152064, "bf16", 0.2, 0.28, 0.001, AGG_TOKEN_MEAN, "normal"),
    4: Config(4, "loss-only fp32 logits T=32768 V=151936 10% masked", 256, 8, 16, 16, 16,
              0, 151936, "logits", 0.2, 0.2, 0.01, AGG_SEQ_MEAN_TOKEN_MEAN, "bern05",
              mask_frac=0.1),
}


def config(cid: int, **overrides) -> Config:
    """Return config ``cid``, optionally with some fields replaced (reduced sizes)."""
    c = CONFIGS[cid]
    return c.replace(**overrides) if overrides else c


def _seed(cfg_key, stream: str) -> int:
    ss = np.random.SeedSequence([2505, 17826, *cfg_key, _STREAMS.index(stream)])
    return int(ss.generate_state(1, np.uint64)[0] & ((1 << 63) - 1))


def _np_rng(cfg_key, stream):
    return np.random.Generator(np.random.PCG64(_seed(cfg_key, stream)))


def _torch_gen(cfg_key, stream, device):
    g = torch.Generator(device=device)
    g.manual_seed(_seed(cfg_key, stream))
    return g


@dataclass
class Batch:
    cfg: Config
    seq_start: torch.Tensor     # int32 [n_seq+1]
    mask: torch.Tensor          # uint8 [T]
    lengths: np.ndarray         # int64 [n_seq] response lengths (before random masking)
    ids: torch.Tensor           # int32 [T]
    rewards: torch.Tensor       # f32 [n_seq]
    old_noise: torch.Tensor     # f32 [T]
    ref_noise: torch.Tensor     # f32 [T]
    H: Optional[torch.Tensor] = None       # [T, d] f32/bf16
    W: Optional[torch.Tensor] = None       # [V, d] f32/bf16
    logits: Optional[torch.Tensor] = None  # [T, V] f32

    @property
    def T(self):
        return int(self.mask.numel())


def _layout(cfg: Config, key):
    rng = _np_rng(key, "lengths")
    lengths = rng.integers(cfg.len_lo, cfg.len_hi + 1, size=cfg.n_seq, dtype=np.int64)
    seq_start = (np.arange(cfg.n_seq + 1, dtype=np.int64) * cfg.pad_to).astype(np.int32)
    pos = np.arange(cfg.pad_to, dtype=np.int64)[None, :]
    mask = (pos < lengths[:, None]).reshape(-1).astype(np.uint8)
    if cfg.mask_frac > 0:
        mrng = _np_rng(key, "mask")
        n_mask = int(round(cfg.mask_frac * cfg.T))
        drop = mrng.choice(cfg.T, size=n_mask, replace=False)
        mask[drop] = 0
    return seq_start, mask, lengths


def _rewards(cfg: Config, key):
    rng = _np_rng(key, "rewards")
    if cfg.reward == "bern05":
        r = (rng.random(cfg.n_seq) < 0.5).astype(np.float32)
    elif cfg.reward == "bern_prompt":
        p = rng.random(cfg.n_prompts)
        u = rng.random(cfg.n_seq)
        r = (u < np.repeat(p, cfg.group)).astype(np.float32)
    elif cfg.reward == "normal":
        r = rng.standard_normal(cfg.n_seq).astype(np.float32)
    else:
        raise ValueError(cfg.reward)
    return r


def _gumbel_argmax(z: torch.Tensor, g: torch.Generator) -> torch.Tensor:
    u = torch.rand(z.shape, generator=g, device=z.device, dtype=torch.float32)
    u.clamp_(min=1e-30)
    return torch.argmax(z - torch.log(-torch.log(u)), dim=1)


def make_batch(cfg: Config, device="cpu", poison: bool = False, seed_key=None,
               chunk_rows: int = 4096, layout_only: bool = False) -> Batch:
    """Build the synthetic batch of ``cfg`` on ``device``.

    ``seed_key`` (a tuple of ints) selects the random streams; it defaults to
    ``(cfg.cid,)`` so each named workload has one fixed batch.  With
    ``poison=True`` masked rows of H / logits are NaN and their token ids are
    out of range, which a correct consumer never reads.  ``layout_only=True``
    skips H, W and logits and draws the token ids uniformly (for kernels that
    only need the layout, ids, rewards and noise).
    """
    key = tuple(seed_key) if seed_key is not None else (cfg.cid,)
    dev = torch.device(device)
    seq_start, mask_np, lengths = _layout(cfg, key)
    T = cfg.T
    valid_np = mask_np.astype(bool)
    valid = torch.from_numpy(valid_np).to(dev)

    H = W = logits = None
    ids = torch.zeros(T, dtype=torch.int64, device=dev)
    g_samp = _torch_gen(key, "sampling", dev)
    valid_rows = torch.from_numpy(np.nonzero(valid_np)[0]).to(dev)
    if layout_only:
        u = _np_rng(key, "sampling").integers(0, cfg.V, size=T)
        ids = torch.from_numpy(u).to(dev)
        ids[~valid] = 0
    elif cfg.dtype in ("f32", "bf16"):
        tdt = torch.float32 if cfg.dtype == "f32" else torch.bfloat16
        gH = _torch_gen(key, "H", dev)
        H = torch.empty((T, cfg.d), dtype=tdt, device=dev)
        for r0 in range(0, T, chunk_rows):
            r1 = min(T, r0 + chunk_rows)
            H[r0:r1] = torch.randn((r1 - r0, cfg.d), generator=gH, device=dev).to(tdt)
        gW = _torch_gen(key, "W", dev)
        W = torch.empty((cfg.V, cfg.d), dtype=tdt, device=dev)
        scale = cfg.logit_std / math.sqrt(cfg.d)
        for r0 in range(0, cfg.V, chunk_rows):
            r1 = min(cfg.V, r0 + chunk_rows)
            W[r0:r1] = (torch.randn((r1 - r0, cfg.d), generator=gW, device=dev) * scale).to(tdt)
        Wf = W.float()
        for c0 in range(0, valid_rows.numel(), chunk_rows):
            rr = valid_rows[c0:c0 + chunk_rows]
            z = H[rr].float() @ Wf.t()
            ids[rr] = _gumbel_argmax(z, g_samp)
        del Wf
        H[~valid] = float("nan") if poison else 0.0
    elif cfg.dtype == "logits":
        gL = _torch_gen(key, "logits", dev)
        logits = torch.empty((T, cfg.V), dtype=torch.float32, device=dev)
        for r0 in range(0, T, chunk_rows):
            r1 = min(T, r0 + chunk_rows)
            logits[r0:r1] = torch.randn((r1 - r0, cfg.V), generator=gL, device=dev) * cfg.logit_std
        for c0 in range(0, valid_rows.numel(), chunk_rows):
            rr = valid_rows[c0:c0 + chunk_rows]
            ids[rr] = _gumbel_argmax(logits[rr], g_samp)
        if poison:
            logits[~valid] = float("nan")
    else:
        raise ValueError(cfg.dtype)

    if poison:
        ids[~valid] = cfg.V + 7
    ids = ids.to(torch.int32)

    g_old = _torch_gen(key, "old", dev)
    g_ref = _torch_gen(key, "ref", dev)
    old_noise = torch.randn(T, generator=g_old, device=dev) * math.sqrt(cfg.old_var)
    ref_noise = torch.randn(T, generator=g_ref, device=dev) * math.sqrt(cfg.ref_var)
    old_noise[~valid] = 0.0
    ref_noise[~valid] = 0.0

    return Batch(cfg=cfg,
                 seq_start=torch.from_numpy(seq_start).to(dev),
                 mask=torch.from_numpy(mask_np).to(dev),
                 lengths=lengths,
                 ids=ids,
                 rewards=torch.from_numpy(_rewards(cfg, key)).to(dev),
                 old_noise=old_noise, ref_noise=ref_noise,
                 H=H, W=W, logits=logits)


def extra_normal(shape, key, device="cpu", std=1.0, dtype=torch.float32):
    """Extra seeded N(0, std^2) values for stand-alone kernel tests (e.g. a
    synthetic per-token gradient or a log-sum-exp offset)."""
    g = _torch_gen(tuple(key), "extra", torch.device(device))
    return (torch.randn(shape, generator=g, device=device) * std).to(dtype)
