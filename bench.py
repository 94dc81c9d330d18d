#!/usr/bin/env python
"""Merged actor-update benchmark on one MI355X.

A step is one whole actor update over one batch of synthetic trajectories:
timeline merging -> (per pack of <= 131072 tokens) embedding, decoder-block
forward, fused LM-head / clipped policy-gradient loss forward and backward,
block backward, embedding backward.  Inputs sit in HBM before timing starts.
The same batch is also run unmerged (every LLM call its own sample) for the
merged-vs-unmerged speedup.

The headline is the largest workload, long32b-8x60 (the 32B-class block over
8 episodes of 60 calls); the 1.5B-class, agent-shaped 7B-class and
multi-agent 7B-class workloads follow as sub-records, merged and unmerged.
Prints one JSON line on stdout; progress goes to stderr.
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
PEAK_F32_TFLOPS = 157.3        # MI355X fp32 vector
PEAK_HBM_GBS = 8000.0


HEADLINE = "4"                 # long32b-8x60, the largest single-GPU workload
SUB_RECORDS = "1,2,3"          # block1.5b-64x8, agent7b-32x10..30, multiagent7b-16x4x12


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", default=HEADLINE, help="headline workload index (0..4) or name")
    ap.add_argument("--unmerged-steps", type=int, default=2,
                    help="timed unmerged steps of the headline workload (no extra warm-up: the "
                         "merged run has loaded every kernel)")
    ap.add_argument("--sub", default=SUB_RECORDS,
                    help="comma-separated workloads measured as sub-records ('' for none)")
    ap.add_argument("--sub-steps", type=int, default=2)
    ap.add_argument("--sub-warmup", type=int, default=1)
    ap.add_argument("--no-unmerged", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample-tokens", type=int, default=0)
    ap.add_argument("--no-extras", action="store_true",
                    help="skip the KL / GRPO selection / AdamW / text-merge / full-model / "
                         "scaled-merge measurements")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                    help="only run a plain device copy of BYTES three times and exit: the "
                         "reference for scaling the HBM byte counters")
    ap.add_argument("--merge-scaled-only", action="store_true",
                    help="only run the scaled merge (the agent-shaped workload's 32 episodes "
                         "repeated to 1024) and print that record")
    return ap.parse_args()


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


# HBM bytes per launch of the dominant kernel class, from two rocprofv3 --pmc
# passes (FETCH_SIZE, WRITE_SIZE) over the same bench command, each scaled by
# the counter's reading for a plain copy of known size.  Keyed by (kernel
# class, workload); an entry holds while the GEMM sources hash to `sources`
# and a step launches the class `launches` times (the same mix of products),
# otherwise the line reports null.
TRAFFIC = {
    ("gemm4_tn", "block1.5b-64x8"): {"bytes_per_launch": 4840.4e6, "launches": 27,
                                     "sources": "c74b4918568820ba"},
    ("gemm4_tn", "long32b-8x60"): {"bytes_per_launch": 17968.3e6, "launches": 56,
                                   "sources": "c74b4918568820ba"},
    ("gemm4_nn", "long32b-8x60"): {"bytes_per_launch": 23618.3e6, "launches": 68,
                                   "sources": "c74b4918568820ba"},
}


def source_hash(files):
    import hashlib
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, "paper_2606_04484_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


GEMM_SOURCES = ("gemm_core.h", "gemm.hip")


def copy_calibration(nbytes):
    """A plain elementwise copy (one read and one write of nbytes each) for
    calibrating FETCH_SIZE / WRITE_SIZE against known traffic."""
    import torch
    n = nbytes // 4
    src = torch.ones(n, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        torch.mul(src, 1.0, out=dst)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": 4 * n, "dispatches": 3}), flush=True)


def attention_flops(cu, m):
    """Causal attention, fwd + bwd (bwd = 2.5 x fwd; recompute not credited)."""
    L = np.diff(np.asarray(cu, np.float64))
    fwd = 2.0 * m.head_dim * m.n_q_heads * np.sum(L * (L + 1))
    return 3.5 * fwd, fwd


def step_flops(L, m):
    blk = 6.0 * m.block_params() * L.n_tok
    lm = 6.0 * m.d_model * m.vocab * L.n_mask
    att, att_fwd = attention_flops(L.cu_host, m)
    return blk, lm, att, att_fwd


def timed(A, merger, merged, steps, warmup, torch, capi, record=False):
    L = None
    for _ in range(warmup):
        A.zero_grads()
        merger.launch(merged)
        L = merger.layout(A.m.pack_tokens)
        A.step(L)
    torch.cuda.synchronize()
    if record:
        capi.aj_timing_enable(True)
    t0 = time.perf_counter()
    for _ in range(steps):
        A.zero_grads()
        merger.launch(merged)
        L = merger.layout(A.m.pack_tokens)
        A.step(L)
    torch.cuda.synchronize()
    dt = (time.perf_counter() - t0) / steps
    rec = None
    if record:
        rec = capi.aj_timing_read()
        capi.aj_timing_enable(False)
    return L, dt, rec


def extras(A, merger, cfg, tl, dev, torch, capi, actor, steps):
    """The steps around the update, measured on the same workload:
    the update with the KL penalty (a reference forward of a frozen copy of
    the policy, then the step with the penalty), GRPO advantages + the
    non-dummy episode selection, one AdamW step over every parameter, and
    text-level Match on a stripped-thinking draw of the workload."""
    m = cfg.model
    from workloads import make_rewards
    out = {}
    # KL: reference log-probs (forward only) + the step with the penalty
    Wref = {k: v.clone() for k, v in A.W.items()}
    R = actor.ActorUpdate(m, Wref)
    merger.launch(True)
    L = merger.layout(m.pack_tokens)
    R.prepare(L)
    A.prepare(L)
    for i in range(steps + 1):
        if i == 1:
            torch.cuda.synchronize()
            t0 = time.perf_counter()
        A.zero_grads()
        merger.launch(True)
        L = merger.layout(m.pack_tokens)
        ref = R.forward_logprob(L)
        A.step(L, ref_logprob=ref, kl_coef=2e-3)
    torch.cuda.synchronize()
    out["kl_step"] = {"ms_per_step": round((time.perf_counter() - t0) / steps * 1e3, 3),
                      "kl_coef": 2e-3, "includes": "reference forward + step with the KL term"}
    del R, Wref
    # GRPO advantages + selection (groups of 8 episodes)
    off, rew = make_rewards(tl.n_traj, 8, seed=1)
    goff, grew = torch.from_numpy(off).cuda(), torch.from_numpy(rew).cuda()
    adv = torch.empty(tl.n_traj, dtype=torch.float32, device="cuda")
    keep = torch.empty(tl.n_traj, dtype=torch.uint8, device="cuda")
    so = {"traj_tl_off": torch.empty(tl.n_traj + 1, dtype=torch.int32, device="cuda"),
          "tl_tok_off": torch.empty(tl.n_tl + 1, dtype=torch.int64, device="cuda"),
          "tok": torch.empty(tl.n_tok, dtype=torch.int32, device="cuda"),
          "flags": torch.empty(tl.n_tok, dtype=torch.uint8, device="cuda"),
          "old_logprob": torch.empty(tl.n_tok, dtype=torch.float32, device="cuda"),
          "adv": torch.empty(tl.n_tok, dtype=torch.float32, device="cuda"),
          "counts": torch.zeros(3, dtype=torch.int64, device="cuda")}
    ws = torch.empty(capi.aj_select_workspace_bytes(tl.n_traj, tl.n_tl), dtype=torch.uint8,
                     device="cuda")
    for i in range(3):
        if i == 2:
            capi.aj_timing_enable(True)
        capi.aj_grpo_advantages(goff, grew, 1e-6, adv, keep)
        capi.aj_select_episodes(dev, keep, adv, so, ws)
    rec = capi.aj_timing_read()
    capi.aj_timing_enable(False)
    kept = so["counts"].cpu().numpy()
    ms = rec["select"][0]
    # bytes: every input token's flags + the kept ones' id, flags, log-prob read and
    # id, flags, log-prob, advantage written; offsets are negligible
    nb = tl.n_tok * 1 + int(kept[2]) * (4 + 1 + 4 + 4 + 1 + 4 + 4)
    out["grpo_select"] = {"ms": round(ms, 4), "launches": rec["select"][1],
                          "episodes_kept": int(kept[0]), "tokens_kept": int(kept[2]),
                          "tokens_in": int(tl.n_tok), "GB/s": round(nb / (ms * 1e-3) / 1e9, 1),
                          "hbm_frac": round(nb / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)}
    # AdamW over every parameter: float32 master copy, moments, bfloat16 copy out
    n = sum(v.numel() for v in A.W.values())
    P = torch.cat([v.float().flatten() for v in A.W.values()])
    G = torch.cat([v.flatten() for v in A.G.values()])
    M1, M2 = torch.zeros_like(P), torch.zeros_like(P)
    Pc = torch.empty(n, dtype=A.W["emb"].dtype, device="cuda")
    for i in range(4):
        if i == 1:
            capi.aj_timing_enable(True)
        capi.aj_adamw_step(P, G, M1, M2, 1e-6, 0.9, 0.999, 1e-8, 0.01, i + 1, param_copy=Pc)
    rec = capi.aj_timing_read()
    capi.aj_timing_enable(False)
    ms = rec["adamw"][0] / rec["adamw"][1]
    nb = n * (4 * 4 + 3 * 4 + Pc.element_size())
    out["adamw"] = {"params": n, "ms": round(ms, 4), "bytes_per_param": nb // n,
                    "GB/s": round(nb / (ms * 1e-3) / 1e9, 1),
                    "hbm_frac": round(nb / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)}
    del P, G, M1, M2, Pc
    out["text_merge"] = text_merge(A, cfg, torch, capi, actor, steps)
    out["full_model"] = full_model(merger, cfg, torch, capi, actor)
    return out


FULL_LAYERS = 28        # decoder blocks of a 1.5B-class model at this block shape


def merge_scaled(merger, tl, torch, capi, actor, R=32):
    """The merge on R copies of the workload's timelines side by side (the
    episodes are independent, so every count is R times the workload's): at
    a workload's own size the merge is a chain of short launches whose
    latency hides its bandwidth; here its bytes dominate.  With the
    agent-shaped 7B-class workload (32 episodes) and R = 32 this is the
    1024-episode instance of that workload's recipe."""
    d0 = merger.tl
    n_tok, n_tl, n_traj = tl.n_tok, tl.n_tl, tl.n_traj
    rep = torch.arange(R, device="cuda", dtype=torch.int64)
    dev = {
        "traj_tl_off": torch.cat([d0["traj_tl_off"][:1],
                                  (d0["traj_tl_off"][1:].long()[None, :] + n_tl * rep[:, None])
                                  .flatten().int()]),
        "tl_tok_off": torch.cat([d0["tl_tok_off"][:1],
                                 (d0["tl_tok_off"][1:][None, :] + n_tok * rep[:, None]).flatten()]),
        "tok": d0["tok"].repeat(R), "flags": d0["flags"].repeat(R),
        "old_logprob": d0["old_logprob"].repeat(R), "adv": d0["adv"].repeat(R),
    }
    big = actor.Merger(dev)
    for i in range(4):
        if i == 1:
            capi.aj_timing_enable(True)
        big.launch(True)
    rec = capi.aj_timing_read()
    capi.aj_timing_enable(False)
    counts = big.out["counts"].cpu().numpy()
    base = merger.out["counts"].cpu().numpy()
    ms = rec["merge"][0] / rec["merge"][1]
    n_llm = R * int(np.count_nonzero((tl.flags & 3) == 2))
    mb = 5 * R * n_tok + 8 * n_llm + 17 * int(counts[1]) + 4 * int(counts[2])
    res = {"copies": R, "episodes": R * n_traj, "unmerged_tokens": R * n_tok,
           "merged_tokens": int(counts[1]),
           "counts_match": bool(np.array_equal(counts[:3], R * base[:3])),
           "ms": round(ms, 4), "launches_per_merge": rec["merge"][1] // 3,
           "algorithmic_MB": round(mb / 1e6, 1),
           "GB/s": round(mb / (ms * 1e-3) / 1e9, 1),
           "hbm_frac": round(mb / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)}
    del big, dev
    torch.cuda.empty_cache()
    return res


def full_model(merger, cfg, torch, capi, actor):
    """The whole actor update of a FULL_LAYERS-block policy on the same merged
    batch: activation checkpointing (layer inputs kept, every block but the
    last recomputed in the backward).  Flops count the model once (the
    recompute is not credited)."""
    import dataclasses
    from workloads import make_weights_torch
    m = dataclasses.replace(cfg.model, n_layers=FULL_LAYERS)
    W = make_weights_torch(m, seed=1000, device="cuda")
    A = actor.ActorUpdate(m, W)
    merger.launch(True)
    L = merger.layout(m.pack_tokens)
    A.prepare(L)
    L, t, _ = timed(A, merger, True, 1, 1, torch, capi)
    blk, lm, att, _ = step_flops(L, m)
    total = FULL_LAYERS * (blk + att) + lm
    peak = PEAK_BF16_TFLOPS if m.dtype == "bf16" else PEAK_F32_TFLOPS
    ckpt = capi.aj_stack_ckpt_bytes(A.bcfg, FULL_LAYERS, max(p["t1"] - p["t0"] for p in L.packs))
    res = {"n_layers": FULL_LAYERS, "params": sum(v.numel() for v in W.values()),
           "merged_tokens": L.n_tok, "ms_per_step": round(t * 1e3, 1),
           "tokens_per_s": round(L.n_tok / t, 1),
           "algorithmic_tflop_per_step": round(total / 1e12, 2),
           "mfma_util": round(total / t / 1e12 / peak, 4),
           "checkpoint_GB_per_pack": round(ckpt / 1e9, 2)}
    del A
    # the same model trained through LoRA adapters (rank 32, alpha 64) on all
    # four projections of every block: base weights, embedding and LM head frozen
    from workloads import make_lora_numpy
    rank = 32
    lora = {k: torch.from_numpy(v).to(device="cuda", dtype=W["emb"].dtype)
            for k, v in make_lora_numpy(m, rank, seed=2000, b_std=1e-3).items()}
    A = actor.ActorUpdate(m, W, lora=lora, lora_rank=rank, lora_scale=64.0 / rank)
    A.prepare(L)
    L, t, _ = timed(A, merger, True, 1, 1, torch, capi)
    res["lora"] = {"rank": rank, "alpha": 64, "trainable_params": sum(v.numel() for v in lora.values()),
                   "ms_per_step": round(t * 1e3, 1), "tokens_per_s": round(L.n_tok / t, 1)}
    del A, W, lora
    torch.cuda.empty_cache()
    return res


def text_merge(A, cfg, torch, capi, actor, steps):
    """Text- vs token-level Match on the same workload drawn with every
    response's thinking section stripped from later calls' contexts: merge
    time and sizes, the TI report, and the update step on either layout."""
    from workloads import make_timelines
    m = A.m
    tl = make_timelines(cfg, think_p=1.0)
    llm = (tl.flags & 3) == 2
    old = np.where(llm, -np.log(m.vocab) + tl.lp_noise, 0.0).astype(np.float32)
    dev = actor.upload_timelines(tl, old)
    res = {"think_p": 1.0, "unmerged_tokens": int(tl.n_tok), "blocks": int(tl.n_blk)}
    for name, text in (("text", True), ("token", False)):
        mg = actor.Merger(dev, text=text)
        for i in range(4):
            if i == 1:
                capi.aj_timing_enable(True)
            mg.launch(True)
        rec = capi.aj_timing_read()
        capi.aj_timing_enable(False)
        L = mg.layout(m.pack_tokens)
        A.prepare(L)
        L, t, _ = timed(A, mg, True, steps, 1, torch, capi)
        r = {"merged_tokens": L.n_tok, "segments": L.n_seg, "loss_tokens": L.n_mask,
             "merge_ms": round(rec["merge"][0] / rec["merge"][1], 4),
             "step_ms": round(t * 1e3, 3), "tokens_per_s": round(L.n_tok / t, 1)}
        if text:
            ti = mg.ti.cpu().tolist()
            r["ti_drift_blocks"], r["ti_drift_tokens"] = int(ti[0]), int(ti[1])
        res[name] = r
    res["step_speedup_text_vs_token"] = round(res["token"]["step_ms"] / res["text"]["step_ms"], 3)
    return res


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(cfg, tl, old, W_dev, sample_tokens, all_tl):
    """The oracle, as is, on a bounded sample of the headline workload: its
    first episode merged by the oracle, then the float64 actor update on the
    first `sample_tokens` merged tokens (whole segments, the last one cut);
    plus the oracle's merge (Algorithm 1, pure Python) timed on every full
    workload measured in this run."""
    from threadpoolctl import threadpool_info
    from oracle import merge as om
    from oracle import model as M
    sub = tl.subset([0])
    n0 = sub.n_tok
    eps = om.episodes_from_flat(sub.traj_tl_off, sub.tl_tok_off, sub.tok, sub.flags, old[:n0],
                                sub.adv)
    packed, _ = om.merge_batch(eps)
    L = min(sample_tokens, packed.n_tok)
    cu = [int(c) for c in packed.cu_seqlens if c < L] + [L]
    cut = om.Packed(cu, packed.tok[:L], packed.mask[:L], packed.old_logprob[:L],
                    packed.adv[:L], packed.pos[:L])
    W = {k: v.float().cpu().numpy() for k, v in W_dev.items()}
    t0 = time.perf_counter()
    M.actor_update(cut, W, cfg.model)
    t_model = time.perf_counter() - t0
    del W
    merges = {}
    for name, t in all_tl.items():
        e = om.episodes_from_flat(t.traj_tl_off, t.tl_tok_off, t.tok, t.flags, t.lp_noise, t.adv)
        t0 = time.perf_counter()
        p, _ = om.merge_batch(e)
        dt = time.perf_counter() - t0
        merges[name] = {"unmerged_tokens": int(t.n_tok), "merged_tokens": int(p.n_tok),
                        "s": round(dt, 3), "unmerged_tokens_per_s": round(t.n_tok / dt, 1)}
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    return {"value": round(L / t_model, 3), "unit": "tokens/s",
            "cores": int(threads), "kind": "oracle",
            "sample": f"{cfg.name}: episode 0 merged by the oracle ({n0} unmerged -> "
                      f"{packed.n_tok} merged tokens), then the float64 actor update (forward "
                      f"+ backward, every gradient) on its first {L} merged tokens "
                      f"({len(cu) - 1} segments, {t_model:.1f} s)",
            "cpu_model": cpu_model(), "host_cpus": os.cpu_count(),
            "merge_oracle": merges}


def rollout_logprobs(A, tl, torch, actor):
    """Rollout log-probs: the policy's own log-probs (an untimed forward of
    this path) plus the generator's N(0, 0.05) noise.  The forward runs on the
    merged layout, whose log-prob of every response token is the unmerged
    one's; merging with the token index as the log-prob payload carries each
    target back to its unmerged token."""
    m = A.m
    if tl.n_tok < (1 << 24):
        dev = actor.upload_timelines(tl, np.arange(tl.n_tok, dtype=np.float32))
        L = actor.merge(dev, merged=True, pack_tokens=m.pack_tokens)
    else:
        dev = actor.upload_timelines(tl, np.zeros(tl.n_tok, np.float32))
        L = actor.merge(dev, merged=False, pack_tokens=m.pack_tokens)
    cur = A.forward_logprob(L).float().cpu().numpy()
    tg = L.targets[:L.n_mask].cpu().numpy()
    src = L.old_logprob[L.targets[:L.n_mask].long()].long().cpu().numpy() \
        if tl.n_tok < (1 << 24) else tg
    old = np.zeros(tl.n_tok, np.float32)
    old[src] = cur + tl.lp_noise[src]
    return old


def measure(cfg, steps, warmup, u_steps, u_warmup, torch, capi, actor, record=False,
            keep=False):
    """One workload: merged steps (timed), one recorded step (per-class kernel
    times), unmerged steps.  Returns the record (and, with keep, the live
    objects for the extras)."""
    from workloads import make_timelines, make_weights_torch
    m = cfg.model
    tl = make_timelines(cfg)
    W = make_weights_torch(m, seed=1000, device="cuda")
    A = actor.ActorUpdate(m, W)
    old = rollout_logprobs(A, tl, torch, actor)
    dev = actor.upload_timelines(tl, old)
    merger = actor.Merger(dev)
    merger.launch(True)
    Lm = merger.layout(m.pack_tokens)
    A.prepare(Lm)
    log(f"{cfg.name}: {tl.n_tok} -> {Lm.n_tok} tokens, {len(Lm.packs)} packs; "
        f"{warmup} + {steps} merged steps")
    Lm, t_m, _ = timed(A, merger, True, steps, warmup, torch, capi)
    rec = None
    if record:
        _, _, rec = timed(A, merger, True, 1, 0, torch, capi, record=True)
    stats = A.stats.cpu().numpy()
    blk, lm, att, att_fwd = step_flops(Lm, m)
    peak = PEAK_BF16_TFLOPS if m.dtype == "bf16" else PEAK_F32_TFLOPS
    r = {"workload": cfg.name, "merged_tokens": Lm.n_tok, "unmerged_tokens": int(tl.n_tok),
         "loss_tokens": Lm.n_mask, "segments": Lm.n_seg, "packs": len(Lm.packs),
         "steps": steps, "warmup": warmup, "ms_per_step": round(t_m * 1e3, 3),
         "tokens_per_s": round(Lm.n_tok / t_m, 1),
         "effective_tokens_per_s": round(tl.n_tok / t_m, 1),
         "loss_tokens_per_s": round(Lm.n_mask / t_m, 1),
         "mfma_util": round((blk + lm + att) / t_m / 1e12 / peak, 4),
         "algorithmic_tflop_per_step": {"block": round(blk / 1e12, 3),
                                        "lm_head": round(lm / 1e12, 3),
                                        "attention": round(att / 1e12, 3)},
         "loss": float(stats[0])}
    if u_steps > 0:
        mu = actor.Merger(dev)
        mu.launch(False)
        Lu = mu.layout(m.pack_tokens)
        A.prepare(Lu)
        log(f"{cfg.name}: unmerged {Lu.n_tok} tokens, {len(Lu.packs)} packs; "
            f"{u_warmup} + {u_steps} steps")
        Lu, t_u, _ = timed(A, mu, False, u_steps, u_warmup, torch, capi)
        r["unmerged"] = {"steps": u_steps, "warmup": u_warmup,
                         "ms_per_step": round(t_u * 1e3, 3), "tokens": Lu.n_tok,
                         "tokens_per_s": round(Lu.n_tok / t_u, 1), "packs": len(Lu.packs)}
        r["speedup_vs_unmerged"] = round(t_u / t_m, 3)
        del mu, Lu
    log(f"{cfg.name}: merged {t_m * 1e3:.1f} ms/step"
        + (f", unmerged {r['unmerged']['ms_per_step']:.1f}" if u_steps > 0 else ""))
    live = dict(tl=tl, W=W, A=A, old=old, dev=dev, merger=merger, Lm=Lm, t_m=t_m, rec=rec,
                flops=(blk, lm, att, att_fwd), peak=peak)
    if not keep:
        for k in ("A", "W", "dev", "merger", "Lm"):
            live.pop(k)
        del A, W, dev, merger, Lm
        torch.cuda.empty_cache()
    return r, live


KERNEL_NAMES = {"gemm_nt": "gemm_mfma_kernel<true, true>",
                "gemm_nn": "gemm_mfma_kernel<true, false>",
                "gemm_tn": "gemm_mfma_kernel<false, false>",
                "gemm4_nt": "gemm_mfma4s_kernel<true, true>",
                "gemm4_nn": "gemm_mfma4s_kernel<true, false>",
                "gemm4_tn": "gemm_mfma4s_kernel<false, false>", "attn_fwd": "attn_fwd_mfma_kernel",
                "lm_fwd": "lm_fwd_fused_kernel", "lm_dz": "lm_dz_fused_kernel"}


def roofline(rec, flops, peak, workload):
    """Per-class kernel times of one step and the dominant kernel against its
    roofline (HIP events on the launch stream)."""
    blk, lm, att, att_fwd = flops
    classes = {}
    for k, (ms, n, fl) in rec.items():
        if k == "attn_fwd":
            fl = att_fwd
        elif k == "attn_bwd":
            fl = att - att_fwd
        classes[k] = dict(ms=ms, launches=n, tflops=(fl / (ms * 1e-3) / 1e12) if ms > 0 else 0.0)
    # the roofline names one kernel with algorithmic flops: not the multi-kernel
    # attention backward, not the logits recompute of the LM-head backward
    dom = max((k for k in classes
               if k not in ("merge", "attn_bwd", "lm_dz") and not k.startswith("stage_")),
              key=lambda k: classes[k]["ms"])
    d = classes[dom]
    fl_dom = {"attn_fwd": att_fwd}.get(dom, rec[dom][2])
    roof = {"kernel": KERNEL_NAMES.get(dom, dom), "bound": "mfma",
            "achieved": round(fl_dom / (d["ms"] * 1e-3) / 1e12, 2), "peak": peak,
            "unit": "TFLOP/s", "frac": round(fl_dom / (d["ms"] * 1e-3) / 1e12 / peak, 4),
            "traffic": None, "launches": d["launches"],
            "avg_launch_ms": round(d["ms"] / max(d["launches"], 1), 4)}
    tr = TRAFFIC.get((dom, workload))
    if (tr and dom.startswith("gemm") and tr["launches"] == d["launches"]
            and tr["sources"] == source_hash(GEMM_SOURCES)):
        roof["traffic"] = tr["bytes_per_launch"]
        roof["traffic_unit"] = "bytes"
    kc = {k: {kk: round(vv, 4) if isinstance(vv, float) else vv for kk, vv in v.items()}
          for k, v in classes.items()}
    return roof, kc


def ceilings(torch, capi):
    """What this chip sustains, measured on it (the roofline lines keep the
    published peaks): the bf16 MFMA rate from registers with random and with
    constant operands, no memory traffic (the random-operand rate is the
    ceiling for products of random or trained weights: the matrix cores draw
    more power when their inputs toggle), and the HBM rates of a streaming
    copy and a read-only stream."""
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    scratch = torch.empty(2 * cus * 256, dtype=torch.float32, device="cuda")
    rnd = capi.aj_ceiling_mfma_bf16(True, scratch)
    const = capi.aj_ceiling_mfma_bf16(False, scratch)
    buf = torch.empty(2 << 30, dtype=torch.uint8, device="cuda")
    copy, read = capi.aj_ceiling_copy(buf)
    del scratch, buf
    torch.cuda.empty_cache()
    return {"mfma_bf16_random_tflops": round(rnd, 1), "mfma_bf16_constant_tflops": round(const, 1),
            "hbm_copy_gbps": round(copy, 1), "hbm_read_gbps": round(read, 1), "cus": cus}


def stage_records(rec, flops, peak, n_tok, n_mask, n_packs, m):
    """The decoder-block and LM-head/loss stages of one step (whole library
    calls, HIP events on the launch stream) against the MFMA roofline, and
    the loss stage's algorithmic HBM traffic for completeness: the hidden
    states of the scored rows read by the forward and the backward, d hidden
    written in float32 for every token, the vocab matrix read by both, and
    its float32 gradient read and written once per pack."""
    blk, lm, att, _ = flops
    out = {}
    ms, n, _ = rec.get("stage_block", (0.0, 0, 0.0))
    if n:
        tf = (blk + att) / (ms * 1e-3) / 1e12
        out["block"] = {"ms": round(ms, 3), "calls": n, "tflops": round(tf, 1),
                        "mfma_frac": round(tf / peak, 4)}
    ms, n, _ = rec.get("stage_loss", (0.0, 0, 0.0))
    if n:
        es = 2 if m.dtype == "bf16" else 4
        d, V = m.d_model, m.vocab
        nb = 2 * n_mask * d * es + n_tok * d * 4 + n_packs * (2 * V * d * es + 8 * V * d)
        tf = lm / (ms * 1e-3) / 1e12
        out["loss"] = {"ms": round(ms, 3), "calls": n, "tflops": round(tf, 1),
                       "mfma_frac": round(tf / peak, 4), "algorithmic_GB": round(nb / 1e9, 2),
                       "GB/s": round(nb / (ms * 1e-3) / 1e9, 1),
                       "hbm_frac": round(nb / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)}
    return out


def merge_record(rec, tl, Lm):
    """The merge against HBM: algorithmic bytes = every unmerged token's id and
    flags, the llm tokens' log-prob and advantage read once; every merged
    token's id, position, mask, log-prob and advantage and every target written."""
    if "merge" not in rec or not rec["merge"][1]:
        return None
    mms = rec["merge"][0] / rec["merge"][1]
    n_llm = int(np.count_nonzero((tl.flags & 3) == 2))
    mb = 5 * tl.n_tok + 8 * n_llm + 17 * Lm.n_tok + 4 * Lm.n_mask
    return {"ms": round(mms, 4), "algorithmic_MB": round(mb / 1e6, 2),
            "GB/s": round(mb / (mms * 1e-3) / 1e9, 1),
            "hbm_frac": round(mb / (mms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)}


def main():
    args = parse()
    if args.copy_calibration:
        copy_calibration(args.copy_calibration)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print(json.dumps({"error": "the actor update runs on one GPU only; --gpus must be 1 "
                          "(sharding over GPUs is designed, not implemented)"}))
        sys.exit(2)
    import torch
    from paper_2606_04484_amd import actor, capi
    if not os.path.exists(capi.LIB_PATH):
        from paper_2606_04484_amd.build import build
        build()
    from workloads import get_config, make_timelines

    key = lambda c: int(c) if c.isdigit() else c
    cfg = get_config(key(args.config))
    torch.cuda.set_device(0)
    if args.merge_scaled_only:
        c = get_config(key(args.config)) if args.config != HEADLINE else get_config(2)
        tl = make_timelines(c)
        dev = actor.upload_timelines(tl, tl.lp_noise)
        merger = actor.Merger(dev)
        merger.launch(True)
        merger.layout(c.model.pack_tokens)
        ms = merge_scaled(merger, tl, torch, capi, actor)
        ceil = ceilings(torch, capi)
        ms["frac_of_copy"] = round(ms["GB/s"] / ceil["hbm_copy_gbps"], 4)
        print(json.dumps({"workload": c.name, "merge_scaled": ms, "ceilings": ceil}))
        return

    m = cfg.model
    head, live = measure(cfg, args.steps, args.warmup,
                         0 if args.no_unmerged else args.unmerged_steps, 0, torch, capi, actor,
                         record=True, keep=True)
    roof, kc = roofline(live["rec"], live["flops"], live["peak"], cfg.name)
    all_tl = {cfg.name: live["tl"]}
    out = {
        "metric": "merged actor-update tokens/sec/GPU",
        "value": head["tokens_per_s"],
        "unit": "tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": m.dtype, "data": "synthetic",
        "config": {"workload": cfg.name, "merged_tokens": head["merged_tokens"],
                   "unmerged_tokens": head["unmerged_tokens"],
                   "loss_tokens": head["loss_tokens"], "segments": head["segments"],
                   "packs": head["packs"], "pack_tokens": m.pack_tokens, "d_model": m.d_model,
                   "heads": [m.n_q_heads, m.n_kv_heads], "head_dim": m.head_dim,
                   "d_ff": m.d_ff, "vocab": m.vocab, "vocab_chunk": m.vocab_chunk},
        "effective_tokens_per_s": head["effective_tokens_per_s"],
        "loss_tokens_per_s": head["loss_tokens_per_s"],
        "mfma_util": head["mfma_util"],
        "algorithmic_tflop_per_step": head["algorithmic_tflop_per_step"],
        "kernel_classes": kc,
        "roofline": roof,
        "loss": head["loss"],
    }
    mr = merge_record(live["rec"], live["tl"], live["Lm"])
    out["stages"] = stage_records(live["rec"], live["flops"], live["peak"], head["merged_tokens"],
                                  head["loss_tokens"], head["packs"], m)
    if mr:
        out["stages"]["merge"] = mr
    if not args.no_extras:
        # The LM-head backward reading the forward's kept float32 logits instead
        # of recomputing the vocab projection (bitwise the same step): an
        # option that trades ~4 bytes of HBM per logit of a pack for the
        # second projection; the headline keeps the streaming design, which
        # never materialises the logits.
        log("kept-logits variant on " + cfg.name)
        A = live["A"]
        A.set_keep_logits(True)
        A.prepare(live["Lm"])
        _, t_k, _ = timed(A, live["merger"], True, 2, 1, torch, capi)
        out["kept_logits"] = {"steps": 2, "warmup": 1, "ms_per_step": round(t_k * 1e3, 3),
                              "tokens_per_s": round(live["Lm"].n_tok / t_k, 1),
                              "vs_streaming": round(head["ms_per_step"] / (t_k * 1e3), 3)}
        A.set_keep_logits(False)
        del A
    if "unmerged" in head:
        out["unmerged"] = head["unmerged"]
        out["speedup_vs_unmerged"] = head["speedup_vs_unmerged"]
    head_old, head_tl = live["old"], live["tl"]
    W_head = None if args.no_cpu_baseline else {k: v.cpu() for k, v in live["W"].items()}
    del live
    torch.cuda.empty_cache()
    ceil = ceilings(torch, capi)
    if roof and roof.get("unit") == "TFLOP/s":
        ceil["roofline_frac_of_random_mfma"] = round(roof["achieved"] / ceil["mfma_bf16_random_tflops"], 4)
    out["ceilings"] = ceil

    subs = {}
    for k in [x for x in args.sub.split(",") if x.strip()]:
        c = get_config(key(k.strip()))
        if c.name == cfg.name:
            continue
        is_b15 = c.name == "block1.5b-64x8"
        want_extras = not args.no_extras and (is_b15 or c.name == "agent7b-32x10..30")
        r, lv = measure(c, args.sub_steps, args.sub_warmup,
                        0 if args.no_unmerged else (2 if is_b15 else 1), 0, torch, capi, actor,
                        record=True, keep=want_extras)
        r["roofline"], r["kernel_classes"] = roofline(lv["rec"], lv["flops"], lv["peak"], c.name)
        r["stages"] = stage_records(lv["rec"], lv["flops"], lv["peak"], r["merged_tokens"],
                                    r["loss_tokens"], r["packs"], c.model)
        if not args.no_extras and is_b15:
            log("extras on " + c.name)
            r["extras"] = extras(lv["A"], lv["merger"], c, lv["tl"], lv["dev"], torch, capi,
                                 actor, 2)
        if not args.no_extras and c.name == "agent7b-32x10..30":
            log("scaled merge on " + c.name)
            r["merge_scaled"] = merge_scaled(lv["merger"], lv["tl"], torch, capi, actor)
        all_tl[c.name] = lv["tl"]
        subs[c.name] = r
        del lv
        torch.cuda.empty_cache()
    if subs:
        out["sub_records"] = subs
        scaled = subs.get("agent7b-32x10..30", {}).get("merge_scaled")
        if scaled:
            scaled["frac_of_copy"] = round(scaled["GB/s"] / ceil["hbm_copy_gbps"], 4)
    if mr:
        out["merge"] = mr
    if not args.no_cpu_baseline:
        log("cpu baseline (oracle)")
        st = args.cpu_sample_tokens or (head["merged_tokens"] if cfg.name.startswith("tiny")
                                        else 1024)
        out["cpu_baseline"] = cpu_baseline(cfg, head_tl, head_old, W_head, st, all_tl)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
