"""Around the actor update: GRPO advantages, the non-dummy batch filter and
the AdamW step, float64, plain loops -- test infrastructure only.

* GRPO advantages.  Section 3 trains with GRPO-style policy-gradient updates,
  and the training recipes draw groups of rollouts per task (group size 8 in
  the multi-task study of Section 5.3).  GRPO normalises each episode's reward inside its
  group: adv = (r - mean) / (std + eps).  The paper gives no formula; this
  reading takes the sample standard deviation (Bessel's correction) and
  eps = 1e-6, and gives every LLM token of an episode the episode's
  advantage (outcome supervision; other tokens carry 0).
* The non-dummy filter.  Section 4.3's collection strategy C3 counts a task
  only if its episodes do not all share one reward (there are j != k with
  r_j != r_k); such groups carry no policy-gradient signal.  Here the
  episodes of a group with a single distinct reward (including a group of
  one) are dropped from the batch before merging, and get advantage 0.
* AdamW.  Step (4) of Section 4.2 (the Weight_Syncing phase) runs optimizer
  steps after the loss; the optimizer is not named, so this is a reading: Adam with decoupled weight
  decay (Loshchilov and Hutter), bias-corrected moments, on float32 master
  parameters.
"""
import numpy as np


def grpo_advantages(group_off, reward, eps=1e-6):
    """Per-episode advantage and keep flag (group has two different rewards)."""
    reward = np.asarray(reward, np.float64)
    adv = np.zeros(len(reward))
    keep = np.zeros(len(reward), np.uint8)
    for g in range(len(group_off) - 1):
        a, b = int(group_off[g]), int(group_off[g + 1])
        r = reward[a:b]
        n = b - a
        if n < 2 or np.all(r == r[0]):
            continue
        mu = sum(r) / n
        sd = np.sqrt(sum((x - mu) ** 2 for x in r) / (n - 1))
        adv[a:b] = (r - mu) / (sd + eps)
        keep[a:b] = 1
    return adv, keep


def select_episodes(traj_tl_off, tl_tok_off, tok, flags, old_logprob, keep, ep_adv):
    """The kept episodes in order, with every llm token's advantage set to its
    episode's (0 on the other tokens, as in the input layout).
    Returns (traj_tl_off, tl_tok_off, tok, flags, old_logprob, adv)."""
    t_off, k_off = [0], [0]
    toks, fl, olp, adv = [], [], [], []
    for e in range(len(traj_tl_off) - 1):
        if not keep[e]:
            continue
        for i in range(int(traj_tl_off[e]), int(traj_tl_off[e + 1])):
            a, b = int(tl_tok_off[i]), int(tl_tok_off[i + 1])
            toks.append(tok[a:b])
            fl.append(flags[a:b])
            olp.append(old_logprob[a:b])
            adv.append(np.where((flags[a:b] & 3) == 2, ep_adv[e], 0.0))
            k_off.append(k_off[-1] + (b - a))
        t_off.append(t_off[-1] + int(traj_tl_off[e + 1]) - int(traj_tl_off[e]))
    cat = lambda xs, dt: np.concatenate(xs).astype(dt) if xs else np.zeros(0, dt)
    return (np.array(t_off, np.int32), np.array(k_off, np.int64), cat(toks, np.int32),
            cat(fl, np.uint8), cat(olp, np.float64), cat(adv, np.float64))


def adamw_step(p, g, m, v, lr, beta1, beta2, eps, weight_decay, step, grad_scale=1.0):
    """One AdamW step; returns the new (p, m, v)."""
    p = np.asarray(p, np.float64)
    g = np.asarray(g, np.float64) * grad_scale
    m = beta1 * np.asarray(m, np.float64) + (1 - beta1) * g
    v = beta2 * np.asarray(v, np.float64) + (1 - beta2) * g * g
    m_hat = m / (1 - beta1 ** step)
    v_hat = v / (1 - beta2 ** step)
    p = p - lr * weight_decay * p - lr * m_hat / (np.sqrt(v_hat) + eps)
    return p, m, v
