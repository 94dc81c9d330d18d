"""Pins for the merge oracle (Section 4.4.2, Algorithm 1), CPU only.

* golden cases worked out by hand from Algorithm 1;
* a closed form of Algorithm 1's result, checked on random episodes
  (hypothesis): timeline j is absorbed iff some later timeline has it as a
  block-aligned prefix, its absorber is the largest such timeline, and an
  absorbed llm block's payload comes from the largest absorbed j carrying one;
* invariants on the seeded workloads: merged never has more tokens than
  unmerged, every response token is trained exactly once in both layouts,
  and merged token ids equal the survivor's own ids.
"""
import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle import merge as om
from workloads import get_config, make_timelines
from tests.cases import golden_merge_cases, case_to_flat


def _episodes(tl, lp):
    return om.episodes_from_flat(tl.traj_tl_off, tl.tl_tok_off, tl.tok, tl.flags, lp, tl.adv)


@pytest.mark.parametrize("case", golden_merge_cases(), ids=lambda c: c["name"])
def test_golden_cases(case):
    tl, lp = case_to_flat(case)
    eps = _episodes(tl, lp)
    packed, absorbers = om.merge_batch(eps)
    assert absorbers == case["expect"]["absorber"]
    segs = case["expect"]["segments"]
    assert packed.n_seg == len(segs)
    for s, exp in enumerate(segs):
        lo, hi = packed.cu_seqlens[s], packed.cu_seqlens[s + 1]
        np.testing.assert_array_equal(packed.tok[lo:hi], exp["tokens"])
        np.testing.assert_array_equal(packed.mask[lo:hi], exp["mask"])
        np.testing.assert_allclose(packed.old_logprob[lo:hi], np.float32(exp["logprob"]), rtol=0, atol=0)
        np.testing.assert_allclose(packed.adv[lo:hi], np.float32(exp["adv"]), rtol=0, atol=0)
        np.testing.assert_array_equal(packed.pos[lo:hi], np.arange(hi - lo))


# ------------------------------------------------------------------ closed form

def _is_prefix(tj, ti):
    """Brute force: every block of tj equals the aligned block of ti (token ids)."""
    if len(ti) < len(tj):
        return False
    return all(list(a.tokens) == list(b.tokens) for a, b in zip(tj, ti))


@st.composite
def random_episode(draw):
    """Episodes over a 3-letter alphabet so that accidental matches are common."""
    n = draw(st.integers(1, 7))
    blk = st.lists(st.integers(0, 2), min_size=1, max_size=3)
    tls = []
    for _ in range(n):
        kind = draw(st.sampled_from(["fresh", "extend", "copy_prefix", "duplicate"]))
        if kind == "fresh" or not tls:
            base = [(draw(blk), draw(st.sampled_from([0, 1, 2])))]
        else:
            src = tls[draw(st.integers(0, len(tls) - 1))]
            if kind == "duplicate":
                base = [(list(t), a) for t, a in src]
            elif kind == "copy_prefix":
                base = [(list(t), a) for t, a in src[:draw(st.integers(1, len(src)))]]
            else:
                base = [(list(t), draw(st.sampled_from([0, 1]))) for t, _ in src] + [(draw(blk), 1)]
        if kind != "duplicate":
            base = base + [(draw(blk), 2)] * draw(st.integers(0, 1))
        tls.append(base)
    out = []
    for i, tl in enumerate(tls):
        blocks = []
        for k, (t, a) in enumerate(tl):
            lp = [-(i + 1) - 0.01 * (k + 1)] * len(t)   # identifies (timeline, block)
            blocks.append(om.Block(t, a, lp, [float(i)] * len(t)))
        out.append(blocks)
    return out


@settings(max_examples=400, deadline=None)
@given(random_episode())
def test_closed_form_of_algorithm_1(tls):
    surv, absorber = om.merge_episode(tls)
    n = len(tls)
    for j in range(n):
        later = [i for i in range(j + 1, n) if _is_prefix(tls[j], tls[i])]
        if later:
            assert absorber[j] == max(later)
        else:
            assert absorber[j] == -1
    # absorbed timelines never absorb
    for j in range(n):
        if absorber[j] >= 0:
            assert absorber[absorber[j]] == -1
    # payload of every survivor block: own llm block, else the largest absorbed j with llm there
    survivors = [i for i in range(n) if absorber[i] == -1]
    assert len(surv) == len(survivors)
    for s, i in zip(surv, survivors):
        assert [list(b.tokens) for b in s] == [list(b.tokens) for b in tls[i]]
        for k, b in enumerate(s):
            if tls[i][k].author == om.LLM:
                src = i
            else:
                cands = [j for j in range(n) if absorber[j] == i and k < len(tls[j])
                         and tls[j][k].author == om.LLM]
                src = max(cands) if cands else None
            if src is None:
                assert b.author == tls[i][k].author
                np.testing.assert_array_equal(b.logprob, tls[i][k].logprob)
            else:
                assert b.author == om.LLM
                np.testing.assert_array_equal(b.logprob, tls[src][k].logprob)
                np.testing.assert_array_equal(b.adv, tls[src][k].adv)


# ------------------------------------------------------------------ workload invariants

@pytest.mark.parametrize("cfg_id,n_traj", [(0, None), (1, 6), (2, 2), (3, 2), (4, 1)])
def test_workload_invariants(cfg_id, n_traj):
    cfg = get_config(cfg_id)
    tl = make_timelines(cfg, n_traj=n_traj)
    lp = tl.lp_noise.copy()          # unique per response token: a tracer
    eps = _episodes(tl, lp)
    merged, absorbers = om.merge_batch(eps)
    unmerged = om.unmerged_batch(eps)
    assert merged.n_tok <= unmerged.n_tok
    assert unmerged.n_tok == tl.n_tok
    # every response token is trained exactly once in both layouts
    llm = (tl.flags & 3) == 2
    assert int(unmerged.mask.sum()) == int(llm.sum()) == int(merged.mask.sum())
    np.testing.assert_array_equal(np.sort(merged.old_logprob[merged.mask == 1]),
                                  np.sort(tl.lp_noise[llm].astype(np.float64)))
    np.testing.assert_array_equal(np.sort(merged.adv[merged.mask == 1]),
                                  np.sort(tl.adv[llm].astype(np.float64)))
    # merged token ids are each survivor's own ids
    s = 0
    for e, absb in enumerate(absorbers):
        base = int(tl.traj_tl_off[e])
        for i, a in enumerate(absb):
            if a == -1:
                lo, hi = tl.tl_tok_off[base + i], tl.tl_tok_off[base + i + 1]
                np.testing.assert_array_equal(
                    merged.tok[merged.cu_seqlens[s]:merged.cu_seqlens[s + 1]], tl.tok[lo:hi])
                s += 1
    assert s == merged.n_seg


def test_pure_chain_collapses_to_last_call():
    cfg = get_config(4)          # 0% rewrites: one survivor per trajectory
    tl = make_timelines(cfg, n_traj=1)
    eps = _episodes(tl, tl.lp_noise)
    merged, absorbers = om.merge_batch(eps)
    assert merged.n_seg == 1 and absorbers[0][-1] == -1
    assert all(a == len(absorbers[0]) - 1 for a in absorbers[0][:-1])
    assert merged.n_tok == int(tl.tl_tok_off[-1] - tl.tl_tok_off[-2])


def test_all_rewritten_is_identity():
    """Timelines with pairwise different first blocks: nothing merges."""
    tls = [[om.Block([i, i], 0, [0, 0], [0, 0]), om.Block([9], 2, [-1.0], [1.0])] for i in range(5)]
    surv, absorber = om.merge_episode(tls)
    assert absorber == [-1] * 5 and len(surv) == 5
