#!/usr/bin/env python
"""Merged actor-update benchmark on one MI355X.

A step is one whole actor update over one batch of synthetic trajectories:
timeline merging -> (per pack of <= 131072 tokens) embedding, decoder-block
forward, fused LM-head / clipped policy-gradient loss forward and backward,
block backward, embedding backward.  Inputs sit in HBM before timing starts.
The same batch is also run unmerged (every LLM call its own sample) for the
merged-vs-unmerged speedup.  Prints one JSON line.
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


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", default="1", help="workload index (0..4) or name")
    ap.add_argument("--no-unmerged", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample-tokens", type=int, default=0)
    ap.add_argument("--no-extras", action="store_true",
                    help="skip the KL / GRPO selection / AdamW measurements")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                    help="only run a plain device copy of BYTES three times and exit: the "
                         "reference for scaling the HBM byte counters")
    ap.add_argument("--merge-scaled-only", action="store_true",
                    help="only merge the workload and 64 side-by-side copies of it (the "
                         "merge_scaled extra) and print that record")
    return ap.parse_args()


# HBM bytes per launch of the dominant kernel (the TN and NN long-reduction
# GEMMs take nearly the same time per step here, so both are listed), from two rocprofv3 --pmc passes
# (FETCH_SIZE, WRITE_SIZE) over the same bench command, each scaled by the
# counter's reading for a plain copy of known size.  Keyed by (kernel class,
# workload); `sources` are hashed so that a changed kernel reports null.
TRAFFIC = {
    ("gemm4_tn", "block1.5b-64x8"): {"bytes_per_launch": 4840.7e6, "sources": "7e2861621a20400e"},
    ("gemm4_nn", "block1.5b-64x8"): {"bytes_per_launch": 5465.2e6, "sources": "7e2861621a20400e"},
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
    out["merge_scaled"] = merge_scaled(merger, tl, torch, capi, actor)
    out["text_merge"] = text_merge(A, cfg, torch, capi, actor, steps)
    out["full_model"] = full_model(merger, cfg, torch, capi, actor)
    return out


FULL_LAYERS = 28        # decoder blocks of a 1.5B-class model at this block shape


def merge_scaled(merger, tl, torch, capi, actor, R=64):
    """The merge on R copies of the workload's timelines side by side (the
    episodes are independent, so every count is R times the workload's): at
    the workload's own size the merge is a chain of short launches whose
    latency hides its bandwidth; here its bytes dominate."""
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
    res = {"copies": R, "unmerged_tokens": R * n_tok, "merged_tokens": int(counts[1]),
           "counts_match": bool(np.array_equal(counts[:3], R * base[:3])),
           "ms": round(ms, 4), "algorithmic_MB": round(mb / 1e6, 1),
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


def cpu_baseline(cfg, tl, old, W_dev, sample_tokens):
    """The oracle, as is, on a bounded sample of the same workload: the first
    episode, merged by the oracle, its first `sample_tokens` merged tokens
    (whole segments, the last one cut)."""
    from threadpoolctl import threadpool_info
    from oracle import merge as om
    from oracle import model as M
    sub = tl.subset([0])
    n0 = sub.n_tok
    eps = om.episodes_from_flat(sub.traj_tl_off, sub.tl_tok_off, sub.tok, sub.flags, old[:n0],
                                sub.adv)
    t0 = time.perf_counter()
    packed, _ = om.merge_batch(eps)
    t_merge = time.perf_counter() - t0
    L = min(sample_tokens, packed.n_tok)
    cu = [int(c) for c in packed.cu_seqlens if c < L] + [L]
    cut = om.Packed(cu, packed.tok[:L], packed.mask[:L], packed.old_logprob[:L],
                    packed.adv[:L], packed.pos[:L])
    W = {k: v.float().cpu().numpy() for k, v in W_dev.items()}
    t0 = time.perf_counter()
    M.actor_update(cut, W, cfg.model)
    t_model = time.perf_counter() - t0
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    return {"value": L / (t_model + t_merge * L / max(n0, 1)), "unit": "tokens/s",
            "cores": int(threads), "kind": "oracle",
            "sample": f"episode 0 of the same batch merged by the oracle ({n0} unmerged -> "
                      f"{packed.n_tok} merged tokens, {t_merge:.2f} s), then the float64 actor "
                      f"update on its first {L} merged tokens ({len(cu) - 1} segments, "
                      f"{t_model:.1f} s); merge time pro-rated to {L} tokens",
            "host_cpus": os.cpu_count()}


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
    from workloads import get_config, make_timelines, make_weights_torch

    key = int(args.config) if args.config.isdigit() else args.config
    cfg = get_config(key)
    m = cfg.model
    torch.cuda.set_device(0)
    tl = make_timelines(cfg)
    if args.merge_scaled_only:
        dev = actor.upload_timelines(tl, tl.lp_noise)
        merger = actor.Merger(dev)
        merger.launch(True)
        merger.layout(m.pack_tokens)
        print(json.dumps({"workload": cfg.name, "merge_scaled": merge_scaled(merger, tl, torch, capi, actor)}))
        return
    W = make_weights_torch(m, seed=1000, device="cuda")
    # rollout log-probs: the policy's own log-probs (untimed forward of this
    # path on the unmerged layout) plus the generator's N(0, 0.05) noise
    dev = actor.upload_timelines(tl, np.zeros(tl.n_tok, np.float32))
    A = actor.ActorUpdate(m, W)
    Lu = actor.merge(dev, merged=False, pack_tokens=m.pack_tokens)
    cur = A.forward_logprob(Lu).float().cpu().numpy()
    tg = Lu.targets[:Lu.n_mask].cpu().numpy()
    old = np.zeros(tl.n_tok, np.float32)
    old[tg] = cur + tl.lp_noise[tg]
    dev["old_logprob"] = torch.from_numpy(old).cuda()
    del Lu

    merger = actor.Merger(dev)
    merger.launch(True)
    Lm = merger.layout(m.pack_tokens)
    A.prepare(Lm)
    Lm, t_m, rec = timed(A, merger, True, args.steps, args.warmup, torch, capi, record=False)
    _, _, rec = timed(A, merger, True, 1, 0, torch, capi, record=True)
    stats = A.stats.cpu().numpy()
    res_u = None
    if not args.no_unmerged:
        mu = actor.Merger(dev)
        mu.launch(False)
        Lu = mu.layout(m.pack_tokens)
        A.prepare(Lu)
        Lu, t_u, _ = timed(A, mu, False, max(1, args.steps // 2), 1, torch, capi)
        res_u = dict(ms_per_step=t_u * 1e3, tokens=Lu.n_tok, tokens_per_s=Lu.n_tok / t_u,
                     packs=len(Lu.packs))

    blk, lm, att, att_fwd = step_flops(Lm, m)
    total = blk + lm + att
    peak = PEAK_BF16_TFLOPS if m.dtype == "bf16" else PEAK_F32_TFLOPS
    # per-class kernel times of one timed step (HIP events on the launch stream)
    classes = {}
    for k, (ms, n, fl) in rec.items():
        if k == "attn_fwd":
            fl = att_fwd
        elif k == "attn_bwd":
            fl = att - att_fwd
        classes[k] = dict(ms=ms, launches=n, tflops=(fl / (ms * 1e-3) / 1e12) if ms > 0 else 0.0)
    # the roofline names one kernel with algorithmic flops: not the multi-kernel
    # attention backward, not the logits recompute of the LM-head backward
    dom = max((k for k in classes if k not in ("merge", "attn_bwd", "lm_dz")),
              key=lambda k: classes[k]["ms"])
    d = classes[dom]
    kernel_names = {"gemm_nt": "gemm_mfma_kernel<true, true>", "gemm_nn": "gemm_mfma_kernel<true, false>",
                    "gemm_tn": "gemm_mfma_kernel<false, false>",
                    "gemm4_nt": "gemm_mfma4s_kernel<true, true>", "gemm4_nn": "gemm_mfma4s_kernel<true, false>",
                    "gemm4_tn": "gemm_mfma4s_kernel<false, false>", "attn_fwd": "attn_fwd_mfma_kernel",
                    "lm_fwd": "lm_fwd_fused_kernel", "lm_dz": "lm_dz_fused_kernel"}
    fl_dom = {"attn_fwd": att_fwd}.get(dom, rec[dom][2])
    roof = {"kernel": kernel_names.get(dom, dom), "bound": "mfma", "achieved": round(fl_dom / (d["ms"] * 1e-3) / 1e12, 2),
            "peak": peak, "unit": "TFLOP/s",
            "frac": round(fl_dom / (d["ms"] * 1e-3) / 1e12 / peak, 4), "traffic": None,
            "launches": d["launches"], "avg_launch_ms": round(d["ms"] / max(d["launches"], 1), 4)}

    tr = TRAFFIC.get((dom, cfg.name))
    if tr and dom.startswith("gemm") and tr["sources"] == source_hash(GEMM_SOURCES):
        roof["traffic"] = tr["bytes_per_launch"]
        roof["traffic_unit"] = "bytes"

    out = {
        "metric": "merged actor-update tokens/sec/GPU",
        "value": round(Lm.n_tok / t_m, 1),
        "unit": "tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(t_m * 1e3, 3),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": m.dtype, "data": "synthetic",
        "config": {"workload": cfg.name, "merged_tokens": Lm.n_tok, "unmerged_tokens": tl.n_tok,
                   "loss_tokens": Lm.n_mask, "segments": Lm.n_seg, "packs": len(Lm.packs),
                   "pack_tokens": m.pack_tokens, "d_model": m.d_model, "heads": [m.n_q_heads, m.n_kv_heads],
                   "head_dim": m.head_dim, "d_ff": m.d_ff, "vocab": m.vocab},
        "effective_tokens_per_s": round(tl.n_tok / t_m, 1),
        "loss_tokens_per_s": round(Lm.n_mask / t_m, 1),
        "mfma_util": round(total / t_m / 1e12 / peak, 4),
        "algorithmic_tflop_per_step": {"block": round(blk / 1e12, 3), "lm_head": round(lm / 1e12, 3),
                                       "attention": round(att / 1e12, 3)},
        "kernel_classes": {k: {kk: round(vv, 4) if isinstance(vv, float) else vv
                               for kk, vv in v.items()} for k, v in classes.items()},
        "roofline": roof,
        "loss": float(stats[0]),
    }
    # the merge against HBM: algorithmic bytes = every unmerged token's id and
    # flags, the llm tokens' log-prob and advantage read once; every merged
    # token's id, position, mask, log-prob and advantage and every target written
    if "merge" in rec and rec["merge"][1]:
        mms = rec["merge"][0] / rec["merge"][1]
        n_llm = int(np.count_nonzero((tl.flags & 3) == 2))
        mb = 5 * tl.n_tok + 8 * n_llm + 17 * Lm.n_tok + 4 * Lm.n_mask
        out["merge"] = {"ms": round(mms, 4), "algorithmic_MB": round(mb / 1e6, 2),
                        "GB/s": round(mb / (mms * 1e-3) / 1e9, 1),
                        "hbm_frac": round(mb / (mms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)}
    if res_u:
        out["unmerged"] = {k: round(v, 3) if isinstance(v, float) else v for k, v in res_u.items()}
        out["speedup_vs_unmerged"] = round(res_u["ms_per_step"] / (t_m * 1e3), 3)
    if not args.no_extras:
        out["extras"] = extras(A, merger, cfg, tl, dev, torch, capi, actor, max(1, args.steps // 2))
    if not args.no_cpu_baseline:
        st = args.cpu_sample_tokens or (Lm.n_tok if cfg.name.startswith("tiny") else 4096)
        out["cpu_baseline"] = cpu_baseline(cfg, tl, old, W, st)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
