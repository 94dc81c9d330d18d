"""Seeded generators: multi-turn trajectories as per-call timelines, and weights.

Layout of a batch of unmerged timelines (compressed rows, collection order):
  traj_tl_off int32[n_traj+1]  timelines of episode e are [traj_tl_off[e], traj_tl_off[e+1])
  tl_tok_off  int64[n_tl+1]    tokens of timeline i are [tl_tok_off[i], tl_tok_off[i+1])
  tok         int32[n_tok]     token ids
  flags       uint8[n_tok]     author in bits 0..1 (user 0, env 1, llm 2) | 4 on a block's first token
  adv         float32[n_tok]   the call's advantage on its own response tokens, else 0
  lp_noise    float32[n_tok]   N(0, 0.05) on the call's own response tokens, else 0;
                               the rollout log-prob of a response token is the policy's
                               log-prob plus this noise.

Each timeline is one intercepted LLM call: its prompt (the context so far, as
user/env blocks) followed by its own response as the single llm block.
"""
import dataclasses
from dataclasses import dataclass

import numpy as np

AUTHOR_USER = 0
AUTHOR_ENV = 1
AUTHOR_LLM = 2
AUTHOR_MASK = 3
FLAG_BLOCK_START = 4


@dataclass
class Timelines:
    traj_tl_off: np.ndarray
    tl_tok_off: np.ndarray
    tok: np.ndarray
    flags: np.ndarray
    adv: np.ndarray
    lp_noise: np.ndarray
    blk_text: np.ndarray = None      # uint64 text key per block (token order), when drawn

    @property
    def n_blk(self) -> int:
        return int(np.count_nonzero(self.flags & FLAG_BLOCK_START))

    @property
    def n_traj(self) -> int:
        return len(self.traj_tl_off) - 1

    @property
    def n_tl(self) -> int:
        return len(self.tl_tok_off) - 1

    @property
    def n_tok(self) -> int:
        return int(self.tl_tok_off[-1])

    def subset(self, episodes) -> "Timelines":
        """The timelines of the given episodes (ascending indices), re-based."""
        tl_off, tok_off = [0], [0]
        parts = []
        for e in episodes:
            a, b = int(self.traj_tl_off[e]), int(self.traj_tl_off[e + 1])
            s, t = int(self.tl_tok_off[a]), int(self.tl_tok_off[b])
            parts.append((s, t))
            tl_off.append(tl_off[-1] + (b - a))
            base = tok_off[-1] - s
            tok_off.extend((self.tl_tok_off[a + 1:b + 1] + base).tolist())
        take = np.concatenate([np.arange(s, t) for s, t in parts]) if parts else np.zeros(0, np.int64)
        text = None
        if self.blk_text is not None:
            starts = np.flatnonzero(self.flags & FLAG_BLOCK_START)
            keep = [np.arange(*np.searchsorted(starts, [s, t])) for s, t in parts]
            text = self.blk_text[np.concatenate(keep)] if keep else np.zeros(0, np.uint64)
        return Timelines(np.asarray(tl_off, np.int32), np.asarray(tok_off, np.int64),
                         self.tok[take], self.flags[take], self.adv[take], self.lp_noise[take],
                         text)


class _Ids:
    def __init__(self, rng, vocab, zipf_s):
        self.rng, self.vocab = rng, vocab
        self.cdf = None
        if zipf_s > 0:
            w = np.arange(1, vocab + 1, dtype=np.float64) ** (-zipf_s)
            self.cdf = np.cumsum(w / w.sum())

    def __call__(self, n):
        if self.cdf is None:
            return self.rng.integers(0, self.vocab, size=n, dtype=np.int64).astype(np.int32)
        u = self.rng.random(n)
        return np.minimum(np.searchsorted(self.cdf, u, side="right"), self.vocab - 1).astype(np.int32)


def _u(rng, lohi):
    return int(rng.integers(lohi[0], lohi[1] + 1))


def make_timelines(cfg, seed=None, n_traj=None, think_p=None) -> Timelines:
    """Draw a batch of unmerged timelines for workload `cfg`.

    Draw order (numpy default_rng(seed)), per episode: number of calls n; the
    rewrite call t* (one-rewrite workloads); per role its prompt length and
    tokens; then per round t = 1..n, per role in a freshly permuted order
    (single-role workloads skip the permutation): the rewrite coin (t >= 2) and
    fresh context tokens when it lands; the response length, tokens, advantage
    and log-prob noise; and, unless t == n, the observation length and tokens.

    think_p: None draws no texts.  A number also gives every message block a
    text key (a fresh key per message; a message keeps its key wherever it is
    re-rendered) and, from a second stream default_rng([seed, 1]), gives each
    response with probability think_p a thinking section of U{1..na//2}
    leading tokens that later calls' contexts leave out (a chat template that
    strips earlier thinking): the same text, other token ids.  The first
    stream's draws do not depend on think_p (rewrites and the length cap count
    unstripped lengths), so every timeline's blocks are those of think_p=None
    except for the stripped re-renderings.
    """
    seed = cfg.seed if seed is None else seed
    n_traj = cfg.n_traj if n_traj is None else n_traj
    rng = np.random.default_rng(seed)
    ids = _Ids(rng, cfg.model.vocab, cfg.zipf_s)
    texts = think_p is not None
    rng2 = np.random.default_rng([seed, 1]) if texts else None
    keys = []
    next_key = [1]

    def new_key():
        next_key[0] += 1
        return next_key[0] - 1

    traj_tl_off = [0]
    tl_lens = []
    toks, flags, advs, noises = [], [], [], []

    def block_flags(n, author):
        f = np.full(n, author, np.uint8)
        if n:
            f[0] |= FLAG_BLOCK_START
        return f

    for _ in range(n_traj):
        n = _u(rng, cfg.turns)
        t_star = int(rng.integers(2, n + 1)) if cfg.one_rewrite else -1
        # per role: list of (tokens, author, text key, length before any stripping)
        ctx = []
        alive = []
        for _r in range(cfg.roles):
            plen = _u(rng, cfg.prompt)
            ctx.append([(ids(plen), AUTHOR_USER, new_key(), plen)])
            alive.append(True)
        n_here = 0
        for t in range(1, n + 1):
            order = rng.permutation(cfg.roles) if cfg.roles > 1 else (0,)
            for r in order:
                if not alive[r]:
                    continue
                c = ctx[r]
                if t >= 2:
                    coin = rng.random()
                    rewrite = (t == t_star) if cfg.one_rewrite else (coin < cfg.rewrite_p)
                    if rewrite:
                        clen = sum(b[3] for b in c)
                        c = [(ids(clen), AUTHOR_USER, new_key(), clen)]
                na = _u(rng, cfg.resp)
                a = ids(na)
                adv = np.float32(rng.standard_normal())
                noise = rng.normal(0.0, 0.05, na).astype(np.float32)
                clen = sum(b[3] for b in c)
                if clen + na > cfg.max_tokens:
                    alive[r] = False
                    continue
                a_key = new_key()
                for btok, auth, key, _ in c:
                    toks.append(btok)
                    flags.append(block_flags(len(btok), auth))
                    advs.append(np.zeros(len(btok), np.float32))
                    noises.append(np.zeros(len(btok), np.float32))
                    keys.append(key)
                toks.append(a)
                flags.append(block_flags(na, AUTHOR_LLM))
                advs.append(np.full(na, adv, np.float32))
                noises.append(noise)
                keys.append(a_key)
                tl_lens.append(sum(len(b[0]) for b in c) + na)
                n_here += 1
                if t < n:
                    no = _u(rng, cfg.obs)
                    o = ids(no)
                    shown = a
                    if texts and na >= 2 and rng2.random() < think_p:
                        shown = a[int(rng2.integers(1, na // 2 + 1)):]
                    c = c + [(shown, AUTHOR_USER, a_key, na), (o, AUTHOR_ENV, new_key(), no)]
                ctx[r] = c
        traj_tl_off.append(traj_tl_off[-1] + n_here)

    tl_tok_off = np.zeros(len(tl_lens) + 1, np.int64)
    tl_tok_off[1:] = np.cumsum(np.asarray(tl_lens, np.int64))
    cat = lambda xs, dt: np.concatenate(xs).astype(dt) if xs else np.zeros(0, dt)
    return Timelines(np.asarray(traj_tl_off, np.int32), tl_tok_off,
                     cat(toks, np.int32), cat(flags, np.uint8),
                     cat(advs, np.float32), cat(noises, np.float32),
                     np.asarray(keys, np.uint64) if texts else None)


def bf16_round(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even); returns float32."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32)


WEIGHT_NAMES = ("emb", "attn_norm", "w_qkv", "w_o", "mlp_norm", "w_gate_up", "w_down",
                "final_norm", "w_vocab")
BLOCK_WEIGHTS = ("attn_norm", "w_qkv", "w_o", "mlp_norm", "w_gate_up", "w_down")


def layer_key(name, layer):
    """Key of a block weight in the weight dict: layer 0 under its plain name,
    layer l >= 1 under "name.l"."""
    return name if layer == 0 else f"{name}.{layer}"


def weight_shapes(m):
    """Shapes by key: the one-block names first (drawn first), then the block
    weights of layers 1 .. n_layers-1."""
    d = m.d_model
    shapes = {
        "emb": (m.vocab, d), "attn_norm": (d,), "w_qkv": (m.qkv_dim, d),
        "w_o": (d, m.n_q_heads * m.head_dim), "mlp_norm": (d,),
        "w_gate_up": (2 * m.d_ff, d), "w_down": (d, m.d_ff), "final_norm": (d,),
        "w_vocab": (m.vocab, d),
    }
    for layer in range(1, m.n_layers):
        for name in BLOCK_WEIGHTS:
            shapes[layer_key(name, layer)] = shapes[name]
    return shapes


def make_weights_numpy(m, seed=1000, gain_std=0.0, scale=None):
    """float32 arrays (bf16-representable when m.dtype == 'bf16').

    Matrices are N(0, init_std^2); norm gains are 1 (+ N(0, gain_std^2) when
    gain_std > 0, which tests use so that a dropped gain shows).  Row-major
    [out, in]; w_gate_up stacks the gate rows (first d_ff) over the up rows.
    `scale` optionally overrides init_std per weight name.
    """
    rng = np.random.default_rng(seed)
    out = {}
    for name, shape in weight_shapes(m).items():
        base = name.split(".")[0]
        if base.endswith("norm"):
            w = np.ones(shape, np.float32)
            if gain_std:
                w += rng.normal(0.0, gain_std, shape).astype(np.float32)
        else:
            std = m.init_std if scale is None else scale.get(base, m.init_std)
            w = (rng.standard_normal(shape, dtype=np.float32) * np.float32(std))
        out[name] = bf16_round(w) if m.dtype == "bf16" else w.astype(np.float32)
    return out


LORA_PROJ = ("w_qkv", "w_o", "w_gate_up", "w_down")


def lora_key(kind, proj, layer):
    """Key of a LoRA matrix: kind "a" ([rank, in]) or "b" ([out, rank]) of the
    block projection `proj` in `layer`, e.g. "lora_a.w_qkv", "lora_b.w_o.2"."""
    return layer_key(f"lora_{kind}.{proj}", layer)


def lora_shapes(m, rank):
    shapes = weight_shapes(dataclasses.replace(m, n_layers=1))
    out = {}
    for layer in range(m.n_layers):
        for proj in LORA_PROJ:
            n_out, n_in = shapes[proj]
            out[lora_key("a", proj, layer)] = (rank, n_in)
            out[lora_key("b", proj, layer)] = (n_out, rank)
    return out


def make_lora_numpy(m, rank, seed=2000, a_std=None, b_std=0.0):
    """float32 LoRA matrices (bf16-representable when m.dtype == 'bf16'):
    A ~ N(0, a_std^2) (default 1/sqrt(in)), B ~ N(0, b_std^2) -- b_std = 0 is
    the usual zero start; tests draw B too so that the adapters act."""
    rng = np.random.default_rng(seed)
    out = {}
    for name, shape in lora_shapes(m, rank).items():
        if name.startswith("lora_a"):
            std = a_std if a_std is not None else 1.0 / np.sqrt(shape[1])
        else:
            std = b_std
        w = (rng.standard_normal(shape, dtype=np.float32) * np.float32(std)) if std else \
            np.zeros(shape, np.float32)
        out[name] = bf16_round(w) if m.dtype == "bf16" else w
    return out


def make_weights_torch(m, seed=1000, device="cuda", gain_std=0.0):
    """Same recipe drawn with torch's seeded generator on `device` (for full-size shapes).

    Values differ from make_weights_numpy; returns torch tensors in the
    storage dtype (bfloat16 or float32).
    """
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    dt = torch.bfloat16 if m.dtype == "bf16" else torch.float32
    out = {}
    for name, shape in weight_shapes(m).items():
        if name.split(".")[0].endswith("norm"):
            w = torch.ones(shape, device=device, dtype=torch.float32)
            if gain_std:
                w += torch.randn(shape, generator=g, device=device) * gain_std
        else:
            w = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
            w.mul_(m.init_std)
        out[name] = w.to(dt)
    return out


def make_rewards(n_traj, group_size=8, seed=0, p_one=0.5, p_flat=0.25):
    """Outcome rewards for consecutive groups of `group_size` episodes (the last
    group may be shorter): group_off int32[n_groups+1], reward float32[n_traj].

    A group is flat (every episode 0, or every episode 1) with probability
    p_flat; otherwise each episode draws Bernoulli(p_one), which can also
    come out flat.  Draw order: per group, the flat flag, then the rewards.
    """
    rng = np.random.default_rng(seed)
    off = list(range(0, n_traj, group_size)) + [n_traj]
    reward = np.zeros(n_traj, np.float32)
    for a, b in zip(off[:-1], off[1:]):
        if rng.random() < p_flat:
            reward[a:b] = float(rng.integers(0, 2))
        else:
            reward[a:b] = (rng.random(b - a) < p_one).astype(np.float32)
    return np.array(off, np.int32), reward
