"""Timeline merging, token-level Match (Section 4.4.2, Algorithm 1).

Data model (Section 4.4.2, the block tuple equation): a timeline is an ordered
list of message blocks; each block has token ids, an author in
{user, env, llm}, a per-token log-prob and a loss mask that is 1 exactly on
llm-authored tokens.  The per-token advantage rides along with the log-prob
(the reading that per-turn advantages travel with the tokens they score).

Readings taken where the paper is silent:
  * |T| counts blocks and Match compares aligned blocks (the pairwise
    mergeability definition above Algorithm 1);
  * Match is token-id equality of the block's tokens; authors are not compared;
  * merging stays inside one episode.
"""
import numpy as np

USER, ENV, LLM = 0, 1, 2
BLOCK_START = 4


class Block:
    __slots__ = ("tokens", "author", "logprob", "adv")

    def __init__(self, tokens, author, logprob, adv):
        self.tokens = np.asarray(tokens, dtype=np.int64)
        self.author = int(author)
        self.logprob = np.asarray(logprob, dtype=np.float64)
        self.adv = np.asarray(adv, dtype=np.float64)

    def copy(self):
        return Block(self.tokens.copy(), self.author, self.logprob.copy(), self.adv.copy())


def split_blocks(tok, flags, logprob, adv):
    """Cut one timeline's flat token arrays into blocks at the block-start bits."""
    starts = np.flatnonzero(np.asarray(flags) & BLOCK_START).tolist()
    if not starts or starts[0] != 0:
        raise ValueError("a timeline must start a block at its first token")
    ends = starts[1:] + [len(tok)]
    return [Block(tok[s:e], int(flags[s]) & 3, logprob[s:e], adv[s:e])
            for s, e in zip(starts, ends)]


def episodes_from_flat(traj_tl_off, tl_tok_off, tok, flags, logprob, adv):
    """Flat compressed-row timelines -> [episode][timeline][block]."""
    eps = []
    for e in range(len(traj_tl_off) - 1):
        tls = []
        for i in range(int(traj_tl_off[e]), int(traj_tl_off[e + 1])):
            s, t = int(tl_tok_off[i]), int(tl_tok_off[i + 1])
            tls.append(split_blocks(tok[s:t], flags[s:t], logprob[s:t], adv[s:t]))
        eps.append(tls)
    return eps


def match_token(a: Block, b: Block) -> bool:
    """Token-level Match: identical token-id arrays."""
    return a.tokens.shape == b.tokens.shape and bool(np.array_equal(a.tokens, b.tokens))


def merge_episode(timelines, match=match_token):
    """Algorithm 1 on one episode's timelines (collection order).

    Later, not-yet-absorbed timelines are visited from the last one down; each
    absorbs every earlier not-yet-absorbed timeline whose blocks it matches
    one by one, taking over llm authorship (author, tokens, log-prob -- and the
    advantage) on the aligned blocks where its own block is not llm.

    Returns (survivors, absorber): the surviving timelines in original order
    (deep copies, with transfers applied) and, per input timeline, the index of
    the timeline that absorbed it or -1.
    """
    T = [[b.copy() for b in tl] for tl in timelines]
    n = len(T)
    absorbed = set()
    absorber = [-1] * n
    for i in range(n - 1, 0, -1):
        if i in absorbed:
            continue
        for j in range(i - 1, -1, -1):
            if j in absorbed:
                continue
            if len(T[i]) >= len(T[j]) and all(match(T[i][k], T[j][k]) for k in range(len(T[j]))):
                for k in range(len(T[j])):
                    if T[j][k].author == LLM and T[i][k].author != LLM:
                        T[i][k].author = LLM
                        T[i][k].tokens = T[j][k].tokens.copy()
                        T[i][k].logprob = T[j][k].logprob.copy()
                        T[i][k].adv = T[j][k].adv.copy()
                absorbed.add(j)
                absorber[j] = i
    survivors = [T[i] for i in range(n) if i not in absorbed]
    return survivors, absorber


class Packed:
    """Segments laid end to end: the layout the model consumes."""

    def __init__(self, cu_seqlens, tok, mask, logprob, adv, pos):
        self.cu_seqlens = np.asarray(cu_seqlens, np.int64)
        self.tok = np.asarray(tok, np.int64)
        self.mask = np.asarray(mask, np.uint8)
        self.old_logprob = np.asarray(logprob, np.float64)
        self.adv = np.asarray(adv, np.float64)
        self.pos = np.asarray(pos, np.int64)

    @property
    def n_seg(self):
        return len(self.cu_seqlens) - 1

    @property
    def n_tok(self):
        return int(self.cu_seqlens[-1])


def flatten(segments):
    """Concatenate timelines (lists of blocks) into one packed batch.

    mask is 1 on llm-authored tokens; pos restarts at 0 in every segment.
    """
    cu = [0]
    tok, mask, lp, adv, pos = [], [], [], [], []
    for tl in segments:
        L = 0
        for b in tl:
            m = len(b.tokens)
            tok.append(b.tokens)
            mask.append(np.full(m, 1 if b.author == LLM else 0, np.uint8))
            lp.append(b.logprob)
            adv.append(b.adv)
            L += m
        pos.append(np.arange(L, dtype=np.int64))
        cu.append(cu[-1] + L)
    cat = lambda xs, dt: np.concatenate(xs).astype(dt) if xs else np.zeros(0, dt)
    return Packed(cu, cat(tok, np.int64), cat(mask, np.uint8), cat(lp, np.float64),
                  cat(adv, np.float64), cat(pos, np.int64))


def merge_batch(episodes, match=match_token):
    """Merge every episode; survivors flattened in (episode, original index) order.

    Returns (packed, absorbers) with absorbers[e][i] indexing within episode e.
    """
    segs, absorbers = [], []
    for tls in episodes:
        surv, absb = merge_episode(tls, match)
        segs.extend(surv)
        absorbers.append(absb)
    return flatten(segs), absorbers


def unmerged_batch(episodes):
    """Every timeline as its own segment, in collection order."""
    return flatten([tl for tls in episodes for tl in tls])
