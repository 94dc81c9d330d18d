"""Shared set-up of the GPU parity tests: seeded inputs, oracle results, tolerances.

Inputs come from the seeded generators; expected values come from the oracle
only.  The rollout log-probs fed to both sides are the oracle's own log-probs
plus noise, nudged away from the clip boundaries r = 1 +- eps by a margin, so
that the clip decision (a discontinuity) is the same on both sides whatever
their rounding.
"""
import dataclasses

import numpy as np
import torch

from oracle import merge as om
from oracle import model as M
from workloads import get_config, make_timelines, make_weights_numpy
from workloads.configs import ModelConfig


def bf16_case_model(hd=64, d=256, hq=4, hkv=2, ff=512, vocab=2000, chunk=768):
    return ModelConfig(d_model=d, n_q_heads=hq, n_kv_heads=hkv, head_dim=hd, d_ff=ff,
                       vocab=vocab, dtype="bf16", vocab_chunk=chunk)


def workload(model, n_traj=8, seed=0, **kw):
    """The small trajectory recipe (8 x 4 calls, one rewrite each) on `model`;
    keyword arguments override fields of the recipe."""
    return dataclasses.replace(get_config(0), model=model, n_traj=n_traj, seed=seed, **kw)


def episodes(tl, old):
    return om.episodes_from_flat(tl.traj_tl_off, tl.tl_tok_off, tl.tok, tl.flags, old, tl.adv,
                                 tl.blk_text)


def nudge_old(cur, noise, llm, eps, margin):
    """old = cur + noise on llm tokens, kept `margin` (in log space) off the clip kinks."""
    old = np.where(llm, cur + noise, 0.0)
    for kink in (np.log(1 + eps), np.log(1 - eps)):
        d = (cur - old) - kink                     # log r - log(1 +- eps)
        close = llm & (np.abs(d) < margin)
        old = np.where(close, old - np.sign(d + 1e-30) * 2 * margin, old)
    return old.astype(np.float32)


class Case:
    """One seeded actor-update case with the oracle's merged/unmerged results."""

    def __init__(self, cfg, noise_std=0.05, margin=0.0, gain_std=0.1, wseed=1000, think_p=None,
                 text=False, lora=None, lora_scale=1.0):
        """think_p: draw text keys and strip thinking (see make_timelines);
        text: the merged layout uses text-level Match; lora: LoRA matrices (then
        only they train, scaled by lora_scale)."""
        m = cfg.model
        self.cfg, self.m, self.text = cfg, m, text
        self.lora, self.lora_scale = lora, lora_scale
        self.tl = tl = make_timelines(cfg, think_p=think_p)
        self.W = make_weights_numpy(m, seed=wseed, gain_std=gain_std)
        if m.dtype == "bf16":
            from workloads import bf16_round
            self.W = {k: bf16_round(v) for k, v in self.W.items()}
        zero = np.zeros(tl.n_tok, np.float32)
        un = om.unmerged_batch(episodes(tl, zero))
        W_used = self.W if lora is None else M.lora_effective(self.W, lora, lora_scale, m)
        cur = M.current_logprob(un, W_used, m)
        if text:
            # under text-level Match a response can be scored in another
            # context than it was sampled in: keep the clip margin around the
            # log-probs of the text-merged layout, traced back to input tokens
            tr, _ = om.merge_batch(episodes(tl, np.arange(tl.n_tok, dtype=np.float64)),
                                   om.match_text)
            cur_m = M.current_logprob(tr, W_used, m)
            sel = tr.mask == 1
            cur = np.full(tl.n_tok, np.nan)
            cur[tr.old_logprob[sel].astype(np.int64)] = cur_m[sel]
        llm = (tl.flags & 3) == 2
        rng = np.random.default_rng(cfg.seed + 77)
        noise = tl.lp_noise if noise_std == 0.05 else rng.normal(0, noise_std, tl.n_tok)
        self.old = nudge_old(np.nan_to_num(cur), noise, llm, m.clip_eps, margin)
        eps_ = episodes(tl, self.old)
        self.merged, self.absorbers = om.merge_batch(eps_, om.match_text if text else om.match_token)
        self.unmerged = om.unmerged_batch(eps_)
        self._ref = {}

    def oracle(self, merged=True):
        if merged not in self._ref:
            p = self.merged if merged else self.unmerged
            if self.lora is None:
                self._ref[merged] = M.actor_update(p, self.W, self.m)
            else:
                self._ref[merged] = M.lora_actor_update(p, self.W, self.lora, self.lora_scale,
                                                        self.m)
        return self._ref[merged]

    def device_weights(self, device="cuda", which=None):
        dt = torch.bfloat16 if self.m.dtype == "bf16" else torch.float32
        src = self.W if which is None else which
        return {k: torch.from_numpy(v).to(device=device, dtype=dt) for k, v in src.items()}


def rel_l2(a, b):
    a, b = np.asarray(a, np.float64).ravel(), np.asarray(b, np.float64).ravel()
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def cosine(a, b):
    a, b = np.asarray(a, np.float64).ravel(), np.asarray(b, np.float64).ravel()
    return float(a @ b / max(np.linalg.norm(a) * np.linalg.norm(b), 1e-300))


def loss_rel_err(got, ref, terms):
    """|dL| / max(|L|, mean |term|): the token mean of -A r can sit near 0."""
    return abs(got - ref) / max(abs(ref), float(np.mean(np.abs(terms))))
