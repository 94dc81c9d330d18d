"""Timeline merging (Section 4.4.2, Algorithm 1) with either Match strategy
of its Relaxed Matching paragraph -- test infrastructure only.

Data model (Section 4.4.2, the block tuple equation): a timeline is an ordered
list of message blocks; each block has its message text, token ids, an author
in {user, env, llm}, a per-token log-prob and a loss mask that is 1 exactly on
llm-authored tokens.  The per-token advantage rides along with the log-prob
(the reading that per-turn advantages travel with the tokens they score).

Readings taken where the paper is silent:
  * |T| counts blocks and Match compares aligned blocks (the pairwise
    mergeability definition above Algorithm 1);
  * token-level Match is token-id equality of the two blocks; text-level Match
    is equality of the two blocks' message texts.  A block's text is held as
    a key with equal text <=> equal key (an interned id; the oracle compares
    the keys as the texts themselves).  Authors are not compared;
  * merging stays inside one episode;
  * a block's author is the author bits of its first token.

Under text-level Match a transfer replaces the survivor's block by the
absorbed block's tokens, so the block -- and the timeline -- can change
length (Figure: text- vs token-level matching, where a stripped thinking
section makes the two renderings of one message differ in token ids).

Train-inference (TI) consistency report (a reading of the trade-off the
Relaxed Matching paragraph names): an llm block of a merged segment is
consistent when the tokens before it in the segment equal the tokens before it
in the timeline that generated it, i.e. its log-probs are scored in the
context they were sampled in.  Token-level Match never breaks this; text-level
Match breaks it exactly where a re-rendering changed token ids.
"""
import numpy as np

USER, ENV, LLM = 0, 1, 2
BLOCK_START = 4


class Block:
    """One message block.  `src` = (timeline, block) within the episode of the
    block whose tokens this is: itself, or the absorbed block a transfer
    copied (the provenance the TI report needs)."""
    __slots__ = ("tokens", "author", "logprob", "adv", "text", "src")

    def __init__(self, tokens, author, logprob, adv, text=None, src=None):
        self.tokens = np.asarray(tokens, dtype=np.int64)
        self.author = int(author)
        self.logprob = np.asarray(logprob, dtype=np.float64)
        self.adv = np.asarray(adv, dtype=np.float64)
        self.text = text
        self.src = src

    def copy(self):
        return Block(self.tokens.copy(), self.author, self.logprob.copy(), self.adv.copy(),
                     self.text, self.src)


def split_blocks(tok, flags, logprob, adv, text=None, tl_index=None):
    """Cut one timeline's flat token arrays into blocks at the block-start bits.
    `text`: the blocks' text keys in order (or None)."""
    starts = np.flatnonzero(np.asarray(flags) & BLOCK_START).tolist()
    if not starts or starts[0] != 0:
        raise ValueError("a timeline must start a block at its first token")
    if text is not None and len(text) != len(starts):
        raise ValueError("one text key per block")
    ends = starts[1:] + [len(tok)]
    return [Block(tok[s:e], int(flags[s]) & 3, logprob[s:e], adv[s:e],
                  None if text is None else text[k], None if tl_index is None else (tl_index, k))
            for k, (s, e) in enumerate(zip(starts, ends))]


def episodes_from_flat(traj_tl_off, tl_tok_off, tok, flags, logprob, adv, blk_text=None):
    """Flat compressed-row timelines -> [episode][timeline][block].

    blk_text: optional text key of every block, blocks in token order."""
    starts = np.flatnonzero(np.asarray(flags) & BLOCK_START)
    if blk_text is not None and len(blk_text) != len(starts):
        raise ValueError("blk_text needs one key per block start")
    eps = []
    for e in range(len(traj_tl_off) - 1):
        tls = []
        e0 = int(traj_tl_off[e])
        for i in range(e0, int(traj_tl_off[e + 1])):
            s, t = int(tl_tok_off[i]), int(tl_tok_off[i + 1])
            text = None
            if blk_text is not None:
                b0, b1 = np.searchsorted(starts, [s, t])
                text = [int(k) for k in blk_text[b0:b1]]
            tls.append(split_blocks(tok[s:t], flags[s:t], logprob[s:t], adv[s:t], text, i - e0))
        eps.append(tls)
    return eps


def match_token(a: Block, b: Block) -> bool:
    """Token-level Match: identical token-id arrays."""
    return a.tokens.shape == b.tokens.shape and bool(np.array_equal(a.tokens, b.tokens))


def match_text(a: Block, b: Block) -> bool:
    """Text-level Match: identical message texts (the blocks' text keys)."""
    if a.text is None or b.text is None:
        raise ValueError("text-level Match needs the blocks' texts")
    return a.text == b.text


def mergeable(longer, shorter, match):
    """The pairwise mergeability of Section 4.4.2: a timeline S can absorb a
    timeline T when S has at least as many blocks as T and every block of T
    matches the block of S at the same index."""
    return len(longer) >= len(shorter) and all(match(s, t) for s, t in zip(longer, shorter))


def take_over_llm_blocks(survivor, absorbed):
    """The transfer of one absorption (Section 4.4.2): wherever the absorbed
    timeline's block is llm-authored and the survivor's aligned block is not,
    the survivor's block takes the absorbed one's author, tokens, log-probs
    and, here, advantages (and its provenance for the TI report); the block
    keeps its own text."""
    for k, blk in enumerate(absorbed):
        if blk.author == LLM and survivor[k].author != LLM:
            new = blk.copy()
            new.text = survivor[k].text
            survivor[k] = new


def merge_episode(timelines, match=match_token):
    """Timeline merging (Algorithm 1) on one episode's timelines (collection
    order), organised as a worklist of undecided timelines.

    The latest undecided timeline can no longer be absorbed (only later
    timelines absorb, and every later one is decided), so it survives; it
    then absorbs each undecided earlier timeline it can, the nearest first,
    taking over their llm blocks as it goes; those leave the worklist, and
    the next latest undecided timeline is taken.  This is the paper's
    reverse-order sweep: the last timeline absorbs what it can, then the
    latest one not yet absorbed, and so on.

    Returns (survivors, absorber): the surviving timelines in original order
    (deep copies, with transfers applied) and, per input timeline, the index of
    the timeline that absorbed it or -1.
    """
    T = [[b.copy() for b in tl] for tl in timelines]
    for i, tl in enumerate(T):
        for k, b in enumerate(tl):
            if b.src is None:
                b.src = (i, k)
    absorber = [-1] * len(T)
    undecided = list(range(len(T)))
    kept = []
    while undecided:
        s = undecided.pop()
        kept.append(s)
        for j in reversed(undecided):
            if mergeable(T[s], T[j], match):
                take_over_llm_blocks(T[s], T[j])
                absorber[j] = s
        undecided = [j for j in undecided if absorber[j] < 0]
    return [T[s] for s in sorted(kept)], absorber


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


def ti_report(episodes, match=match_token):
    """TI consistency of the merged batch: (llm blocks, llm tokens) whose
    context in their merged segment differs from the context they were
    generated in (the tokens before them in their own original timeline)."""
    n_blk = n_tok = 0
    for tls in episodes:
        surv, _ = merge_episode(tls, match)
        for tl in surv:
            for k, b in enumerate(tl):
                if b.author != LLM:
                    continue
                i, kk = b.src
                trained = np.concatenate([blk.tokens for blk in tl[:k]] + [np.zeros(0, np.int64)])
                sampled = np.concatenate([blk.tokens for blk in tls[i][:kk]] +
                                         [np.zeros(0, np.int64)])
                if not np.array_equal(trained, sampled):
                    n_blk += 1
                    n_tok += len(b.tokens)
    return n_blk, n_tok


def unmerged_batch(episodes):
    """Every timeline as its own segment, in collection order."""
    return flatten([tl for tls in episodes for tl in tls])
