"""Test inputs: golden merge fixtures as flat arrays, and small seeded workloads."""
import json
import os

import numpy as np

from workloads import AUTHOR_LLM, FLAG_BLOCK_START, Timelines

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
AUTHORS = {"user": 0, "env": 1, "llm": AUTHOR_LLM}


def golden_merge_cases(name="merge_cases.json"):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)["cases"]


def golden_text_cases():
    return golden_merge_cases("merge_text_cases.json")


def case_to_flat(case):
    """Golden fixture episodes -> (Timelines, old_logprob float32[n_tok]).

    Blocks that carry a message text get text keys: the texts interned in
    order of first appearance (keys from 1), so equal text <=> equal key."""
    traj = [0]
    tl_off = [0]
    tok, flags, lp, adv = [], [], [], []
    keys, interned = [], {}
    for ep in case["episodes"]:
        for tl in ep:
            n = 0
            for tokens, author, logprob, a, *text in tl:
                if text:
                    keys.append(interned.setdefault(text[0], len(interned) + 1))
                m = len(tokens)
                f = np.full(m, AUTHORS[author], np.uint8)
                f[0] |= FLAG_BLOCK_START
                tok.extend(tokens)
                flags.append(f)
                lp.extend(logprob)
                adv.extend([a] * m)
                n += m
            tl_off.append(tl_off[-1] + n)
        traj.append(traj[-1] + len(ep))
    t = Timelines(np.asarray(traj, np.int32), np.asarray(tl_off, np.int64),
                  np.asarray(tok, np.int32), np.concatenate(flags),
                  np.asarray(adv, np.float32), np.zeros(len(tok), np.float32),
                  np.asarray(keys, np.uint64) if keys else None)
    return t, np.asarray(lp, np.float32)
