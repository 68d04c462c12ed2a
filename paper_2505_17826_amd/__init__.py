"""MI355X (gfx950) core of a GRPO/PPO reinforcement fine-tuning trainer step.

A thin ctypes binding of ``librft.so``; every function keeps the name of the
C entry point it marshals (``include/rft.h``).  torch supplies device memory
and the current HIP stream; every step of the computation runs in the
library's HIP kernels.  There is no CPU fallback: if the library is missing
or no GPU is present the calls raise.
"""
from __future__ import annotations

import ctypes
import math
import os
from dataclasses import dataclass

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "librft.so")

RFT_OK, RFT_E_NULL, RFT_E_SHAPE, RFT_E_DTYPE, RFT_E_PARAM, RFT_E_WORKSPACE, \
    RFT_E_UNSUPPORTED, RFT_E_HIP = range(8)
RFT_F32, RFT_BF16 = 0, 1
RFT_AGG_SEQ_MEAN_TOKEN_MEAN, RFT_AGG_TOKEN_MEAN = 0, 1
RFT_ADV_GRPO, RFT_ADV_MEAN_CENTER, RFT_ADV_LEAVE_ONE_OUT = 0, 1, 2
(RFT_OP_TOKEN_LOGPROBS, RFT_OP_TOKEN_LOGPROBS_FROM_LOGITS, RFT_OP_PPO_FWD, RFT_OP_PPO_BWD,
 RFT_OP_PPO_BWD_LOGITS, RFT_OP_PPO_FUSED_LOGITS, RFT_OP_PPO_STEP, RFT_OP_SFT_FWD,
 RFT_OP_DPO_FWD) = range(9)

_p = ctypes.c_void_p
_i64 = ctypes.c_int64


class rft_tokens(ctypes.Structure):
    _fields_ = [("T", ctypes.c_int64), ("n_seq", ctypes.c_int64), ("seq_start", _p),
                ("mask", _p), ("token_ids", _p), ("is_expert", _p)]


class rft_ppo_params(ctypes.Structure):
    _fields_ = [("eps_low", ctypes.c_float), ("eps_high", ctypes.c_float),
                ("kl_coef", ctypes.c_float), ("agg", ctypes.c_int32),
                ("denom_override", ctypes.c_double), ("mix_mu", ctypes.c_float),
                ("entropy_coef", ctypes.c_float)]


class rft_ppo_stats(ctypes.Structure):
    _fields_ = [("loss", ctypes.c_double), ("pg_loss", ctypes.c_double),
                ("kl_loss", ctypes.c_double), ("kl_mean", ctypes.c_double),
                ("entropy_mean", ctypes.c_double), ("ratio_mean", ctypes.c_double),
                ("clipfrac", ctypes.c_double), ("n_valid", ctypes.c_int64),
                ("n_seq_valid", ctypes.c_int64), ("n_clipped", ctypes.c_int64),
                ("n_bad_ids", ctypes.c_int64), ("sft_loss", ctypes.c_double),
                ("n_expert", ctypes.c_int64), ("entropy_loss", ctypes.c_double)]


class rft_dpo_stats(ctypes.Structure):
    _fields_ = [("loss", ctypes.c_double), ("chosen_reward", ctypes.c_double),
                ("rejected_reward", ctypes.c_double), ("reward_acc", ctypes.c_double),
                ("margin_mean", ctypes.c_double), ("n_pairs", ctypes.c_int64),
                ("n_valid", ctypes.c_int64), ("n_bad_ids", ctypes.c_int64)]


STATS_BYTES = ctypes.sizeof(rft_ppo_stats)
DPO_STATS_BYTES = ctypes.sizeof(rft_dpo_stats)

_SIGS = {
    "rft_abi_version": (ctypes.c_int, []),
    "rft_status_str": (ctypes.c_char_p, [ctypes.c_int]),
    "rft_last_error": (ctypes.c_char_p, []),
    "rft_workspace_bytes": (ctypes.c_size_t, [ctypes.c_int, ctypes.POINTER(rft_tokens), _i64, _i64,
                                              ctypes.c_int]),
    "rft_workspace_min_bytes": (ctypes.c_size_t, [ctypes.c_int, ctypes.POINTER(rft_tokens), _i64,
                                                  _i64, ctypes.c_int]),
    "rft_noalloc_scratch_bytes": (ctypes.c_size_t, []),
    "rft_ppo_clip_fused_logits_noalloc": (ctypes.c_int, [ctypes.POINTER(rft_tokens), _p, _i64, _p,
                                                         _p, _p, ctypes.POINTER(rft_ppo_params),
                                                         _p, _p, _p, _p, _p, _p, _p]),
    "rft_workspace_bytes_rows": (ctypes.c_size_t, [ctypes.c_int, ctypes.POINTER(rft_tokens), _i64,
                                                   _i64, ctypes.c_int, _i64]),
    "rft_chunk_rows": (_i64, [ctypes.c_int, ctypes.POINTER(rft_tokens), _i64, _i64, ctypes.c_int,
                              ctypes.c_size_t]),
    "rft_group_advantages": (ctypes.c_int, [_p, _i64, ctypes.c_int32, ctypes.c_float, ctypes.c_int32,
                                            _p, _p]),
    "rft_group_advantages_ids_workspace_bytes": (ctypes.c_size_t, [_i64, _i64]),
    "rft_group_advantages_ids": (ctypes.c_int, [_p, _p, _i64, _i64, ctypes.c_int32, ctypes.c_float,
                                                ctypes.c_int32, _p, _p, ctypes.c_size_t, _p]),
    "rft_token_logprobs": (ctypes.c_int, [ctypes.POINTER(rft_tokens), _p, _p, ctypes.c_int, _i64,
                                          _i64, _p, _p, _p, _p, ctypes.c_size_t, _p]),
    "rft_token_logprobs_from_logits": (ctypes.c_int, [ctypes.POINTER(rft_tokens), _p, _i64, _p,
                                                      _p, _p, _p, _p, ctypes.c_size_t, _p]),
    "rft_ppo_clip_loss_fwd": (ctypes.c_int, [ctypes.POINTER(rft_tokens), _i64, _p, _p, _p, _p, _p,
                                             ctypes.POINTER(rft_ppo_params), _p, _p, _p, _p,
                                             ctypes.c_size_t, _p]),
    "rft_ppo_clip_loss_bwd": (ctypes.c_int, [ctypes.POINTER(rft_tokens), _p, _p, ctypes.c_int, _i64,
                                             _i64, _p, _p, _p, _p, _p, _p, ctypes.c_int32, _p,
                                             ctypes.c_size_t, _p]),
    "rft_ppo_clip_loss_bwd_logits": (ctypes.c_int, [ctypes.POINTER(rft_tokens), _p, _i64, _p, _p,
                                                    _p, _p, _p, _p, ctypes.c_size_t, _p]),
    "rft_ppo_clip_fused_logits": (ctypes.c_int, [ctypes.POINTER(rft_tokens), _p, _i64, _p, _p, _p,
                                                 ctypes.POINTER(rft_ppo_params), _p, _p, _p, _p,
                                                 _p, _p, _p, ctypes.c_size_t, _p]),
    "rft_ppo_clip_step": (ctypes.c_int, [ctypes.POINTER(rft_tokens), _p, _p, ctypes.c_int, _i64,
                                         _i64, _p, _p, _p, ctypes.POINTER(rft_ppo_params), _p, _p,
                                         _p, _p, _p, _p, ctypes.c_int32, _p, _p, ctypes.c_size_t,
                                         _p]),
    "rft_sft_loss_fwd": (ctypes.c_int, [ctypes.POINTER(rft_tokens), _i64, _p, ctypes.c_int32,
                                        ctypes.c_double, _p, _p, _p, ctypes.c_size_t, _p]),
    "rft_dpo_loss_fwd": (ctypes.c_int, [ctypes.POINTER(rft_tokens), _i64, _p, _p, ctypes.c_float,
                                        ctypes.c_float, _p, _p, _p, _p, ctypes.c_size_t, _p]),
}

_LIB = None


def lib() -> ctypes.CDLL:
    """Load librft.so (built in-tree by ``build_lib``); raise if it is missing."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run python -m paper_2505_17826_amd.build_lib")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _LIB = L
    return _LIB


class RftError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"{msg} (status {status})")
        self.status = status


def _check(st):
    if st != RFT_OK:
        L = lib()
        raise RftError(st, L.rft_last_error().decode())


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _need_gpu(*ts):
    for t in ts:
        if t is not None and t.device.type != "cuda":
            raise RuntimeError("librft works on device tensors only (no CPU fallback)")


def _dtype_code(t):
    if t.dtype == torch.bfloat16:
        return RFT_BF16
    if t.dtype == torch.float32:
        return RFT_F32
    raise TypeError(f"unsupported dtype {t.dtype}")


@dataclass
class Tokens:
    """Token layout of one batch: rollout row offsets, action mask, sampled ids,
    and optionally per-rollout expert flags (MIX)."""
    seq_start: torch.Tensor   # int32 [n_seq + 1]
    mask: torch.Tensor        # uint8 [T]
    token_ids: torch.Tensor   # int32 [T]
    is_expert: torch.Tensor = None  # uint8 [n_seq] or None

    @property
    def T(self):
        return int(self.mask.numel())

    @property
    def n_seq(self):
        return int(self.seq_start.numel()) - 1

    def c(self) -> rft_tokens:
        for t, dt in ((self.seq_start, torch.int32), (self.mask, torch.uint8),
                      (self.token_ids, torch.int32)):
            if t.dtype != dt or not t.is_contiguous():
                raise TypeError("tokens: seq_start int32, mask uint8, token_ids int32, contiguous")
        ex = None
        if self.is_expert is not None:
            if (self.is_expert.dtype != torch.uint8 or not self.is_expert.is_contiguous()
                    or self.is_expert.numel() != self.n_seq):
                raise TypeError("tokens: is_expert must be contiguous uint8 [n_seq]")
            ex = self.is_expert.data_ptr()
        return rft_tokens(self.T, self.n_seq, self.seq_start.data_ptr(), self.mask.data_ptr(),
                          self.token_ids.data_ptr(), ex)


def ppo_params(eps_low=0.2, eps_high=0.2, kl_coef=0.0, agg=RFT_AGG_SEQ_MEAN_TOKEN_MEAN,
               denom_override=0.0, mix_mu=0.0, entropy_coef=0.0) -> rft_ppo_params:
    return rft_ppo_params(eps_low, eps_high, kl_coef, agg, denom_override, mix_mu, entropy_coef)


def stats_to_dict(buf: torch.Tensor, kind=None) -> dict:
    """Decode an rft_ppo_stats (or, with kind=rft_dpo_stats, an rft_dpo_stats)
    device buffer (synchronises on the copy)."""
    kind = rft_ppo_stats if kind is None else kind
    raw = bytes(buf.detach().cpu().numpy().tobytes())
    s = kind.from_buffer_copy(raw[:ctypes.sizeof(kind)])
    return {k: getattr(s, k) for k, _ in kind._fields_}


def workspace_bytes(op, tokens: Tokens, d=0, V=1, dtype=RFT_F32, minimum=False) -> int:
    L = lib()
    tk = tokens.c()
    f = L.rft_workspace_min_bytes if minimum else L.rft_workspace_bytes
    return int(f(op, ctypes.byref(tk), d, V, dtype))


def workspace_bytes_rows(op, tokens: Tokens, d, V, dtype, rows) -> int:
    """Workspace with which RFT_OP_PPO_BWD / RFT_OP_PPO_STEP runs row chunks of `rows` rows."""
    tk = tokens.c()
    return int(lib().rft_workspace_bytes_rows(op, ctypes.byref(tk), d, V, dtype, rows))


def chunk_rows(op, tokens: Tokens, d, V, dtype, ws_bytes) -> int:
    tk = tokens.c()
    return int(lib().rft_chunk_rows(op, ctypes.byref(tk), d, V, dtype, ws_bytes))


def _workspace(nbytes, device, ws=None):
    if nbytes == 0:
        return None, 0
    if ws is not None:
        return ws, ws.numel() * ws.element_size()
    return torch.empty(nbytes, dtype=torch.uint8, device=device), nbytes


# ------------------------------------------------------------ entry points --
def rft_group_advantages(rewards, group_size, eps=1e-6, out=None, stream=None, unbiased=True):
    _need_gpu(rewards)
    out = torch.empty_like(rewards) if out is None else out
    n_groups = rewards.numel() // group_size if group_size > 0 else 0
    _check(lib().rft_group_advantages(_ptr(rewards), n_groups, group_size, eps,
                                      1 if unbiased else 0, _ptr(out), _stream(stream)))
    return out


def rft_group_advantages_ids(rewards, group_id, n_groups, mode=RFT_ADV_GRPO, eps=1e-6, out=None,
                             stream=None, unbiased=True, ws=None):
    _need_gpu(rewards, group_id)
    out = torch.empty_like(rewards) if out is None else out
    need = int(lib().rft_group_advantages_ids_workspace_bytes(rewards.numel(), n_groups))
    ws, nb = _workspace(need, rewards.device, ws)
    _check(lib().rft_group_advantages_ids(_ptr(rewards), _ptr(group_id), rewards.numel(), n_groups,
                                          mode, eps, 1 if unbiased else 0, _ptr(out), _ptr(ws), nb,
                                          _stream(stream)))
    return out


def rft_token_logprobs(tokens: Tokens, hidden, weight, logp=None, entropy=None, lse=None, ws=None,
                       stream=None, want_entropy=True):
    _need_gpu(hidden, weight)
    T, dev = tokens.T, hidden.device
    d, V = hidden.shape[1], weight.shape[0]
    dt = _dtype_code(hidden)
    logp = torch.empty(T, dtype=torch.float32, device=dev) if logp is None else logp
    lse = torch.empty(T, dtype=torch.float32, device=dev) if lse is None else lse
    if entropy is None and want_entropy:
        entropy = torch.empty(T, dtype=torch.float32, device=dev)
    need = workspace_bytes(RFT_OP_TOKEN_LOGPROBS, tokens, d, V, dt)
    ws, nb = _workspace(need, dev, ws)
    tk = tokens.c()
    _check(lib().rft_token_logprobs(ctypes.byref(tk), _ptr(hidden), _ptr(weight), dt, d, V,
                                    _ptr(logp), _ptr(entropy), _ptr(lse), _ptr(ws), nb,
                                    _stream(stream)))
    return logp, entropy, lse


def rft_token_logprobs_from_logits(tokens: Tokens, logits, logp=None, entropy=None, lse=None,
                                   gathered=None, want_gathered=False, stream=None):
    _need_gpu(logits)
    T, dev, V = tokens.T, logits.device, logits.shape[1]
    logp = torch.empty(T, dtype=torch.float32, device=dev) if logp is None else logp
    lse = torch.empty(T, dtype=torch.float32, device=dev) if lse is None else lse
    entropy = torch.empty(T, dtype=torch.float32, device=dev) if entropy is None else entropy
    if gathered is None and want_gathered:
        gathered = torch.empty(T, dtype=torch.float32, device=dev)
    tk = tokens.c()
    _check(lib().rft_token_logprobs_from_logits(ctypes.byref(tk), _ptr(logits), V, _ptr(logp),
                                                _ptr(entropy), _ptr(lse), _ptr(gathered), None, 0,
                                                _stream(stream)))
    return logp, entropy, lse, gathered


def rft_ppo_clip_loss_fwd(tokens: Tokens, V, logp, old_logp, ref_logp, adv, params, entropy=None,
                          grad_logp=None, stats=None, ws=None, stream=None, grad_entropy=None):
    """Returns (grad_logp, stats); grad_entropy, when given, receives e_t."""
    _need_gpu(logp, old_logp, adv)
    dev = logp.device
    grad_logp = torch.empty_like(logp) if grad_logp is None else grad_logp
    stats = torch.zeros(STATS_BYTES, dtype=torch.uint8, device=dev) if stats is None else stats
    need = workspace_bytes(RFT_OP_PPO_FWD, tokens, 0, V)
    ws, nb = _workspace(need, dev, ws)
    tk = tokens.c()
    _check(lib().rft_ppo_clip_loss_fwd(ctypes.byref(tk), V, _ptr(logp), _ptr(old_logp),
                                       _ptr(ref_logp), _ptr(adv), _ptr(entropy),
                                       ctypes.byref(params), _ptr(grad_logp), _ptr(grad_entropy),
                                       _ptr(stats), _ptr(ws), nb, _stream(stream)))
    return grad_logp, stats


def rft_ppo_clip_loss_bwd(tokens: Tokens, hidden, weight, lse, grad_logp, d_hidden=None,
                          d_weight=None, accumulate_dw=False, ws=None, stream=None,
                          grad_entropy=None, entropy=None):
    _need_gpu(hidden, weight, lse, grad_logp)
    dev = hidden.device
    T, d, V = tokens.T, hidden.shape[1], weight.shape[0]
    dt = _dtype_code(hidden)
    d_hidden = torch.empty((T, d), dtype=torch.float32, device=dev) if d_hidden is None else d_hidden
    d_weight = torch.empty((V, d), dtype=torch.float32, device=dev) if d_weight is None else d_weight
    need = workspace_bytes(RFT_OP_PPO_BWD, tokens, d, V, dt)
    ws, nb = _workspace(need, dev, ws)
    tk = tokens.c()
    _check(lib().rft_ppo_clip_loss_bwd(ctypes.byref(tk), _ptr(hidden), _ptr(weight), dt, d, V,
                                       _ptr(lse), _ptr(grad_logp), _ptr(grad_entropy),
                                       _ptr(entropy), _ptr(d_hidden), _ptr(d_weight),
                                       1 if accumulate_dw else 0, _ptr(ws), nb, _stream(stream)))
    return d_hidden, d_weight


def rft_ppo_clip_loss_bwd_logits(tokens: Tokens, logits, lse, grad_logp, d_logits=None,
                                 stream=None, grad_entropy=None, entropy=None):
    _need_gpu(logits, lse, grad_logp)
    d_logits = torch.empty_like(logits) if d_logits is None else d_logits
    tk = tokens.c()
    _check(lib().rft_ppo_clip_loss_bwd_logits(ctypes.byref(tk), _ptr(logits), logits.shape[1],
                                              _ptr(lse), _ptr(grad_logp), _ptr(grad_entropy),
                                              _ptr(entropy), _ptr(d_logits), None, 0,
                                              _stream(stream)))
    return d_logits


def rft_ppo_clip_fused_logits(tokens: Tokens, logits, old_logp, ref_logp, adv, params, logp=None,
                              entropy=None, lse=None, grad_logp=None, d_logits=None, stats=None,
                              ws=None, stream=None):
    _need_gpu(logits, old_logp, adv)
    T, dev, V = tokens.T, logits.device, logits.shape[1]
    logp = torch.empty(T, dtype=torch.float32, device=dev) if logp is None else logp
    d_logits = torch.empty_like(logits) if d_logits is None else d_logits
    stats = torch.zeros(STATS_BYTES, dtype=torch.uint8, device=dev) if stats is None else stats
    need = workspace_bytes(RFT_OP_PPO_FUSED_LOGITS, tokens, 0, V)
    ws, nb = _workspace(need, dev, ws)
    tk = tokens.c()
    _check(lib().rft_ppo_clip_fused_logits(ctypes.byref(tk), _ptr(logits), V, _ptr(old_logp),
                                           _ptr(ref_logp), _ptr(adv), ctypes.byref(params),
                                           _ptr(logp), _ptr(entropy), _ptr(lse), _ptr(grad_logp),
                                           _ptr(d_logits), _ptr(stats), _ptr(ws), nb,
                                           _stream(stream)))
    return logp, d_logits, stats


def rft_ppo_clip_fused_logits_noalloc(tokens: Tokens, logits, old_logp, ref_logp, adv, params,
                                      logp, d_logits, stats, entropy=None, lse=None,
                                      grad_logp=None, stream=None):
    """rft_ppo_clip_fused_logits without a workspace: the library's own scratch
    array is used and nothing is allocated, so every output must be given."""
    _need_gpu(logits, old_logp, adv, logp, d_logits, stats)
    tk = tokens.c()
    _check(lib().rft_ppo_clip_fused_logits_noalloc(
        ctypes.byref(tk), _ptr(logits), logits.shape[1], _ptr(old_logp), _ptr(ref_logp),
        _ptr(adv), ctypes.byref(params), _ptr(logp), _ptr(entropy), _ptr(lse), _ptr(grad_logp),
        _ptr(d_logits), _ptr(stats), _stream(stream)))
    return logp, d_logits, stats


def rft_ppo_clip_step(tokens: Tokens, hidden, weight, old_logp, ref_logp, adv, params,
                      logp=None, entropy=None, lse=None, grad_logp=None, d_hidden=None,
                      d_weight=None, accumulate_dw=False, stats=None, ws=None, stream=None):
    """Returns (logp, entropy, lse, grad_logp, d_hidden, d_weight, stats)."""
    _need_gpu(hidden, weight, old_logp, adv)
    dev = hidden.device
    T, d, V = tokens.T, hidden.shape[1], weight.shape[0]
    dt = _dtype_code(hidden)
    f32 = dict(dtype=torch.float32, device=dev)
    logp = torch.empty(T, **f32) if logp is None else logp
    entropy = torch.empty(T, **f32) if entropy is None else entropy
    lse = torch.empty(T, **f32) if lse is None else lse
    grad_logp = torch.empty(T, **f32) if grad_logp is None else grad_logp
    d_hidden = torch.empty((T, d), **f32) if d_hidden is None else d_hidden
    d_weight = torch.empty((V, d), **f32) if d_weight is None else d_weight
    stats = torch.zeros(STATS_BYTES, dtype=torch.uint8, device=dev) if stats is None else stats
    need = workspace_bytes(RFT_OP_PPO_STEP, tokens, d, V, dt)
    ws, nb = _workspace(need, dev, ws)
    tk = tokens.c()
    _check(lib().rft_ppo_clip_step(ctypes.byref(tk), _ptr(hidden), _ptr(weight), dt, d, V,
                                   _ptr(old_logp), _ptr(ref_logp), _ptr(adv), ctypes.byref(params),
                                   _ptr(logp), _ptr(entropy), _ptr(lse), _ptr(grad_logp),
                                   _ptr(d_hidden), _ptr(d_weight), 1 if accumulate_dw else 0,
                                   _ptr(stats), _ptr(ws), nb, _stream(stream)))
    return logp, entropy, lse, grad_logp, d_hidden, d_weight, stats


def rft_sft_loss_fwd(tokens: Tokens, V, logp, agg=RFT_AGG_TOKEN_MEAN, denom_override=0.0,
                     grad_logp=None, stats=None, ws=None, stream=None):
    """Returns (grad_logp, stats)."""
    _need_gpu(logp)
    dev = logp.device
    grad_logp = torch.empty_like(logp) if grad_logp is None else grad_logp
    stats = torch.zeros(STATS_BYTES, dtype=torch.uint8, device=dev) if stats is None else stats
    ws, nb = _workspace(workspace_bytes(RFT_OP_SFT_FWD, tokens, 0, V), dev, ws)
    tk = tokens.c()
    _check(lib().rft_sft_loss_fwd(ctypes.byref(tk), V, _ptr(logp), agg, denom_override,
                                  _ptr(grad_logp), _ptr(stats), _ptr(ws), nb, _stream(stream)))
    return grad_logp, stats


def rft_dpo_loss_fwd(tokens: Tokens, V, logp, ref_logp, beta=0.1, label_smoothing=0.0,
                     grad_logp=None, seq_logp=None, want_seq_logp=True, stats=None, ws=None,
                     stream=None):
    """Returns (grad_logp, seq_logp, stats); decode stats with
    stats_to_dict(stats, rft_dpo_stats)."""
    _need_gpu(logp, ref_logp)
    dev = logp.device
    grad_logp = torch.empty_like(logp) if grad_logp is None else grad_logp
    if seq_logp is None and want_seq_logp:
        seq_logp = torch.empty(tokens.n_seq, dtype=torch.float32, device=dev)
    stats = torch.zeros(DPO_STATS_BYTES, dtype=torch.uint8, device=dev) if stats is None else stats
    ws, nb = _workspace(workspace_bytes(RFT_OP_DPO_FWD, tokens, 0, V), dev, ws)
    tk = tokens.c()
    _check(lib().rft_dpo_loss_fwd(ctypes.byref(tk), V, _ptr(logp), _ptr(ref_logp), beta,
                                  label_smoothing, _ptr(grad_logp), _ptr(seq_logp), _ptr(stats),
                                  _ptr(ws), nb, _stream(stream)))
    return grad_logp, seq_logp, stats


def loaded_library_path() -> str:
    return LIB_PATH if _LIB is not None else ""
