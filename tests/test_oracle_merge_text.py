"""Pins for the merge oracle under text-level Match (Section 4.4.2, Relaxed
Matching Strategies), CPU only.

* golden cases worked out by hand (the paper's stripped-thinking figure case,
  a re-encoded observation, a re-layout where blocks grow and shrink, the
  first transfer winning, episodes kept apart): absorbers under both Match
  strategies, the merged segments and the TI-consistency report;
* the token-level golden cases again, with text keys that follow the token
  ids: text-level Match must then give the token-level result;
* a closed form of Algorithm 1 under text-level Match on random episodes
  whose messages have several renderings (hypothesis);
* TI report: zero under token-level Match, always;
* on the seeded workloads with stripped thinking, text-level Match finds
  exactly the absorbers token-level Match finds on the same draw without the
  stripping, and trains every response token once.
"""
import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle import merge as om
from workloads import get_config, make_timelines
from tests.cases import golden_merge_cases, golden_text_cases, case_to_flat


def _episodes(tl, lp):
    return om.episodes_from_flat(tl.traj_tl_off, tl.tl_tok_off, tl.tok, tl.flags, lp, tl.adv,
                                 tl.blk_text)


def _check_segments(packed, segs):
    assert packed.n_seg == len(segs)
    for s, exp in enumerate(segs):
        lo, hi = packed.cu_seqlens[s], packed.cu_seqlens[s + 1]
        np.testing.assert_array_equal(packed.tok[lo:hi], exp["tokens"])
        np.testing.assert_array_equal(packed.mask[lo:hi], exp["mask"])
        np.testing.assert_array_equal(packed.old_logprob[lo:hi], np.float32(exp["logprob"]))
        np.testing.assert_array_equal(packed.adv[lo:hi], np.float32(exp["adv"]))
        np.testing.assert_array_equal(packed.pos[lo:hi], np.arange(hi - lo))


@pytest.mark.parametrize("case", golden_text_cases(), ids=lambda c: c["name"])
def test_golden_text_cases(case):
    tl, lp = case_to_flat(case)
    eps = _episodes(tl, lp)
    packed, absorbers = om.merge_batch(eps, om.match_text)
    assert absorbers == case["expect"]["absorber"]
    _check_segments(packed, case["expect"]["segments"])
    assert list(om.ti_report(eps, om.match_text)) == case["expect"]["ti"]
    _, tok_absorbers = om.merge_batch(eps, om.match_token)
    assert tok_absorbers == case["expect"]["token_absorber"]
    assert om.ti_report(eps, om.match_token) == (0, 0)


def _keys_from_tokens(tl):
    """Text keys that follow the token ids: equal tokens <=> equal key."""
    starts = np.flatnonzero(tl.flags & 4).tolist() + [tl.n_tok]
    interned = {}
    return np.array([interned.setdefault(tuple(tl.tok[a:b].tolist()), len(interned) + 1)
                     for a, b in zip(starts[:-1], starts[1:])], np.uint64)


@pytest.mark.parametrize("case", golden_merge_cases(), ids=lambda c: c["name"])
def test_token_golden_cases_under_text_match(case):
    tl, lp = case_to_flat(case)
    tl.blk_text = _keys_from_tokens(tl)
    eps = _episodes(tl, lp)
    packed, absorbers = om.merge_batch(eps, om.match_text)
    assert absorbers == case["expect"]["absorber"]
    _check_segments(packed, case["expect"]["segments"])
    assert om.ti_report(eps, om.match_text) == (0, 0)


def test_text_match_needs_texts():
    b = om.Block([1], 0, [0.0], [0.0])
    with pytest.raises(ValueError):
        om.match_text(b, b)


# ------------------------------------------------------------------ closed form

@st.composite
def text_episode(draw):
    """Timelines over 4 messages, each with 1-2 renderings (token arrays), so
    that text matches without token matches are common."""
    rend = {m: [draw(st.lists(st.integers(0, 3), min_size=1, max_size=3))
                for _ in range(draw(st.integers(1, 2)))] for m in range(4)}
    n = draw(st.integers(1, 6))
    tls = []
    for i in range(n):
        if tls and draw(st.booleans()):
            _, src = tls[draw(st.integers(0, len(tls) - 1))]
            msgs = src[:draw(st.integers(1, len(src)))]
        else:
            msgs = []
        msgs = msgs + draw(st.lists(st.integers(0, 3), min_size=0 if msgs else 1, max_size=2))
        blocks = []
        for k, m in enumerate(msgs):
            toks = rend[m][draw(st.integers(0, len(rend[m]) - 1))]
            a = draw(st.sampled_from([0, 1, 2]))
            lp = [-(i + 1) - 0.01 * (k + 1)] * len(toks)      # identifies (timeline, block)
            blocks.append(om.Block(toks, a, lp, [float(i)] * len(toks), text=m))
        tls.append((blocks, msgs))
    return [b for b, _ in tls]


def _text_prefix(tj, ti):
    return len(ti) >= len(tj) and all(a.text == b.text for a, b in zip(tj, ti))


@settings(max_examples=400, deadline=None)
@given(text_episode())
def test_closed_form_under_text_match(tls):
    surv, absorber = om.merge_episode(tls, om.match_text)
    n = len(tls)
    for j in range(n):
        later = [i for i in range(j + 1, n) if _text_prefix(tls[j], tls[i])]
        assert absorber[j] == (max(later) if later else -1)
    survivors = [i for i in range(n) if absorber[i] == -1]
    assert len(surv) == len(survivors)
    for s, i in zip(surv, survivors):
        assert [b.text for b in s] == [b.text for b in tls[i]]
        for k, b in enumerate(s):
            if tls[i][k].author == om.LLM:
                src = i
            else:
                cands = [j for j in range(n) if absorber[j] == i and k < len(tls[j])
                         and tls[j][k].author == om.LLM]
                src = max(cands) if cands else None
            if src is None:
                assert b.author == tls[i][k].author
                np.testing.assert_array_equal(b.tokens, tls[i][k].tokens)
            else:
                assert b.author == om.LLM and b.src == (src, k)
                np.testing.assert_array_equal(b.tokens, tls[src][k].tokens)
                np.testing.assert_array_equal(b.logprob, tls[src][k].logprob)
    # flattening lays every survivor out with its (possibly new) block lengths
    packed = om.flatten(surv)
    for s, tl in enumerate(surv):
        n_s = sum(len(b.tokens) for b in tl)
        assert packed.cu_seqlens[s + 1] - packed.cu_seqlens[s] == n_s


@settings(max_examples=200, deadline=None)
@given(text_episode())
def test_token_match_is_always_ti_consistent(tls):
    assert om.ti_report([tls], om.match_token) == (0, 0)


# ------------------------------------------------------------------ workloads

@pytest.mark.parametrize("cfg_id,n_traj", [(0, None), (1, 4), (2, 2), (3, 2)])
def test_stripped_thinking_workload(cfg_id, n_traj):
    cfg = get_config(cfg_id)
    plain = make_timelines(cfg, n_traj=n_traj)
    drift = make_timelines(cfg, n_traj=n_traj, think_p=1.0)
    e_plain = _episodes(plain, plain.lp_noise)
    e_drift = _episodes(drift, drift.lp_noise)
    _, ab_token_plain = om.merge_batch(e_plain, om.match_token)
    text_packed, ab_text = om.merge_batch(e_drift, om.match_text)
    tok_packed, ab_token = om.merge_batch(e_drift, om.match_token)
    # texts and block structure are those of the plain draw: same absorbers
    assert ab_text == ab_token_plain
    assert text_packed.n_seg < tok_packed.n_seg
    # every response token trained exactly once, with its own log-prob and advantage
    llm = (drift.flags & 3) == 2
    assert int(text_packed.mask.sum()) == int(llm.sum())
    np.testing.assert_array_equal(np.sort(text_packed.old_logprob[text_packed.mask == 1]),
                                  np.sort(drift.lp_noise[llm].astype(np.float64)))
    assert text_packed.n_tok <= drift.n_tok
    n_blk, n_tok = om.ti_report(e_drift, om.match_text)
    assert n_blk > 0 and n_tok > 0
    assert om.ti_report(e_drift, om.match_token) == (0, 0)


def test_no_stripping_text_equals_token():
    cfg = get_config(1)
    tl = make_timelines(cfg, n_traj=4, think_p=0.0)
    eps = _episodes(tl, tl.lp_noise)
    a, ab_a = om.merge_batch(eps, om.match_text)
    b, ab_b = om.merge_batch(eps, om.match_token)
    assert ab_a == ab_b
    for k in ("cu_seqlens", "tok", "mask", "old_logprob", "adv", "pos"):
        np.testing.assert_array_equal(getattr(a, k), getattr(b, k))
    assert om.ti_report(eps, om.match_text) == (0, 0)
