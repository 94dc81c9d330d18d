"""The actor update at the benchmark's full size and launch configuration:
block1.5b-64x8 (64 episodes x 8 LLM calls, one 1.5B-class decoder block,
the full 151936-word LM head, bfloat16, packs of <= 131072 tokens), checked
where the float64 oracle can follow it one output at a time, and through
properties that hold at any size.

* Sampled log-probs: for the two shortest and the two longest merged
  segments that carry loss tokens (~1.1k to ~4.9k tokens), up to 8 target
  positions each, spread to the segment's last target; the oracle computes the block
  output at just the rows that predict them (keys and values over the whole
  prefix of the segment) and the LM head at those rows.  Tolerance: the
  bfloat16 log-prob bound, 2e-2 absolute.
* The loss: the GPU's own per-token log-probs, put through the oracle's
  clipped policy-gradient terms in float64, give the loss the GPU reports
  (relative 1e-3: only the order of a float32 sum differs).
* Gradients: the merged update equals the unmerged one (the paper's
  premise: merging changes cost, not results), relative L2 <= 1e-2 per
  weight gradient.

Inputs are the seeded workload and weights; rollout log-probs are -ln(V) plus the
generator's N(0, 0.05) noise, close to what the random-init policy assigns.
"""
import numpy as np
import pytest
import torch

from oracle import merge as om
from oracle import model as M
from workloads import get_config, make_timelines, make_weights_torch
from tests.gpu_cases import rel_l2

pytestmark = pytest.mark.gpu

GRADS = ("emb", "attn_norm", "w_qkv", "w_o", "mlp_norm", "w_gate_up", "w_down", "final_norm",
         "w_vocab")


@pytest.fixture(scope="module")
def full():
    cfg = get_config(1)
    m = cfg.model
    tl = make_timelines(cfg)
    llm = (tl.flags & 3) == 2
    old = np.where(llm, -np.log(m.vocab) + tl.lp_noise, 0.0).astype(np.float32)
    # the seeded generator's full-size recipe (drawn on the device, bfloat16);
    # the oracle reads the same values on the host
    Wd = make_weights_torch(m, seed=1000, device="cuda", gain_std=0.1)
    W = {k: v.float().cpu().numpy() for k, v in Wd.items()}
    del Wd
    print(f"full size: {tl.n_tok} unmerged tokens, {tl.n_tl} timelines", flush=True)
    return cfg, m, tl, old, W


def run_step(m, tl, old, W, merged):
    from paper_2606_04484_amd import actor
    dev = actor.upload_timelines(tl, old)
    L = actor.merge(dev, merged=merged, pack_tokens=m.pack_tokens)
    Wd = {k: torch.from_numpy(v).to(device="cuda", dtype=torch.bfloat16) for k, v in W.items()}
    A = actor.ActorUpdate(m, Wd)
    A.zero_grads()
    A.step(L)
    torch.cuda.synchronize()
    out = dict(lp=A.logprob[:L.n_mask].cpu().numpy().astype(np.float64),
               targets=L.targets[:L.n_mask].cpu().numpy(),
               stats=A.stats.cpu().numpy(), err=int(A.err.cpu()[0]), n_tok=L.n_tok,
               n_mask=L.n_mask, packs=len(L.packs))
    out["grads"] = {k: v.cpu().numpy() for k, v in A.G.items()}
    del A, Wd
    torch.cuda.empty_cache()
    return out


@pytest.fixture(scope="module")
def merged_run(full):
    cfg, m, tl, old, W = full
    return run_step(m, tl, old, W, True)


def test_fullsize_sampled_logprobs(full, merged_run):
    cfg, m, tl, old, W = full
    got = merged_run
    assert got["err"] == 0 and got["packs"] >= 2
    eps = om.episodes_from_flat(tl.traj_tl_off, tl.tl_tok_off, tl.tok, tl.flags, old, tl.adv)
    ref, _ = om.merge_batch(eps)
    # the GPU's loss targets, in merged positions, are the oracle's
    tgt = M.target_positions(ref.cu_seqlens, ref.n_tok)
    tgt = tgt[ref.mask[tgt] == 1]
    np.testing.assert_array_equal(got["targets"], tgt)
    W64 = M.f64_weights(W)
    lens = np.diff(ref.cu_seqlens)
    with_t = [s for s in np.argsort(lens, kind="stable")
              if np.any((tgt > ref.cu_seqlens[s]) & (tgt < ref.cu_seqlens[s + 1]))]
    # the two shortest and the two longest segments with targets: 8 targets
    # spread over each, the last of them near the segment's end
    cand = list(dict.fromkeys(with_t[:2] + with_t[-2:]))
    worst = 0.0
    for s in cand:
        a, b = int(ref.cu_seqlens[s]), int(ref.cu_seqlens[s + 1])
        seg_t = tgt[(tgt > a) & (tgt < b)]
        pick = seg_t[np.unique(np.linspace(0, len(seg_t) - 1, min(8, len(seg_t))).astype(int))]
        x_seg = W64["emb"][ref.tok[a:b]]
        y = M.block_forward_rows(x_seg, ref.pos[a:b], pick - 1 - a, W64, m)
        tok_l = np.concatenate([[0], ref.tok[pick]])
        _, _, lp, _ = M.lm_head_forward(y, W64, tok_l, np.arange(1, len(pick) + 1), m)
        gpu = got["lp"][np.searchsorted(tgt, pick)]
        err = float(np.max(np.abs(gpu - lp)))
        worst = max(worst, err)
        print(f"segment {s}: {b - a} tokens, {len(pick)} sampled targets, max |dlogprob| {err:.3g}",
              flush=True)
    assert worst <= 2e-2


def test_fullsize_loss_matches_logprobs(full, merged_run):
    cfg, m, tl, old, W = full
    got = merged_run
    eps = om.episodes_from_flat(tl.traj_tl_off, tl.tl_tok_off, tl.tok, tl.flags, old, tl.adv)
    ref, _ = om.merge_batch(eps)
    t = got["targets"]
    term, _, _ = M.pg_terms(got["lp"], ref.old_logprob[t], ref.adv[t], m.clip_eps)
    loss = float(np.sum(term) / len(t))
    assert got["stats"][3] == len(t)
    assert abs(got["stats"][0] - loss) <= 1e-3 * max(abs(loss), float(np.mean(np.abs(term))))


def test_fullsize_merged_equals_unmerged(full, merged_run):
    cfg, m, tl, old, W = full
    a = merged_run
    b = run_step(m, tl, old, W, False)
    assert b["err"] == 0 and b["n_mask"] == a["n_mask"] and b["n_tok"] > 2 * a["n_tok"]
    assert abs(a["stats"][0] - b["stats"][0]) <= 1e-2 * max(abs(b["stats"][0]), 1e-3)
    for k in GRADS:
        r = rel_l2(a["grads"][k], b["grads"][k])
        print(f"{k}: rel_l2 merged vs unmerged {r:.3g}", flush=True)
        assert r <= 1e-2, k
