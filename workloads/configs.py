"""The five workloads: trajectory shape plus the one-block policy it trains.

Each workload pairs a multi-turn trajectory recipe (how many LLM calls per
episode, prompt and per-turn append lengths, how often a call rewrites its
context, how token ids are distributed) with the shapes of one pre-norm
decoder block, its LM head and the clipped policy-gradient loss.

Readings of the workload text that the recipe fixes (see the design notes):
  * an "append" of X..Y tokens is a response of U{X/2..Y/2} llm tokens
    followed by an observation of U{X/2..Y/2} env tokens;
  * a rewriting call replaces its whole context by fresh random tokens of
    the same length, as one user block;
  * every later call's prompt holds the earlier responses as non-llm blocks.
"""
from dataclasses import dataclass, field


@dataclass(frozen=True)
class ModelConfig:
    d_model: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    d_ff: int
    vocab: int
    dtype: str = "bf16"          # "f32" or "bf16": storage type of weights/activations
    rms_eps: float = 1e-6
    rope_theta: float = 1e6
    init_std: float = 0.02
    clip_eps: float = 0.2
    vocab_chunk: int = 32768
    pack_tokens: int = 131072
    n_layers: int = 1            # decoder blocks between the embedding and the final norm

    @property
    def qkv_dim(self) -> int:
        return (self.n_q_heads + 2 * self.n_kv_heads) * self.head_dim

    def block_params(self) -> int:
        d, hd = self.d_model, self.head_dim
        return (d * (self.n_q_heads + 2 * self.n_kv_heads) * hd
                + self.n_q_heads * hd * d + 3 * d * self.d_ff)


@dataclass(frozen=True)
class WorkloadConfig:
    name: str
    n_traj: int                      # episodes
    turns: tuple                     # (lo, hi) LLM calls per role per episode, inclusive
    prompt: tuple                    # (lo, hi) turn-1 prompt length per role
    resp: tuple                      # (lo, hi) response (llm) tokens per call
    obs: tuple                       # (lo, hi) observation (env) tokens after a call
    rewrite_p: float = 0.0           # chance that a call t>=2 rewrites its context
    one_rewrite: bool = False        # exactly one rewrite per trajectory at t ~ U{2..n}
    roles: int = 1                   # agent roles per episode, interleaved per round
    zipf_s: float = 0.0              # 0: uniform ids; >0: finite-support Zipf exponent
    max_tokens: int = 1 << 30        # a trajectory stops before a timeline would exceed this
    seed: int = 0
    model: ModelConfig = field(default=None)


TINY = WorkloadConfig(
    name="tiny-8x4-d128", n_traj=8, turns=(4, 4), prompt=(64, 64), resp=(16, 48),
    obs=(16, 32), one_rewrite=True, seed=0,
    model=ModelConfig(d_model=128, n_q_heads=4, n_kv_heads=4, head_dim=32, d_ff=512,
                      vocab=1024, dtype="f32", vocab_chunk=1024))

B1P5 = WorkloadConfig(
    name="block1.5b-64x8", n_traj=64, turns=(8, 8), prompt=(1024, 1024), resp=(64, 256),
    obs=(64, 256), rewrite_p=0.10,
    model=ModelConfig(d_model=1536, n_q_heads=12, n_kv_heads=2, head_dim=128, d_ff=8960,
                      vocab=151936))

AGENT7B = WorkloadConfig(
    name="agent7b-32x10..30", n_traj=32, turns=(10, 30), prompt=(4096, 4096),
    resp=(100, 400), obs=(100, 400), rewrite_p=0.15, max_tokens=32768,
    model=ModelConfig(d_model=3584, n_q_heads=28, n_kv_heads=4, head_dim=128, d_ff=18944,
                      vocab=152064))

MULTI7B = WorkloadConfig(
    name="multiagent7b-16x4x12", n_traj=16, turns=(12, 12), prompt=(512, 2048),
    resp=(100, 400), obs=(100, 400), rewrite_p=0.25, roles=4, zipf_s=1.1,
    model=ModelConfig(d_model=3584, n_q_heads=28, n_kv_heads=4, head_dim=128, d_ff=18944,
                      vocab=152064))

LONG32B = WorkloadConfig(
    name="long32b-8x60", n_traj=8, turns=(60, 60), prompt=(8192, 8192), resp=(128, 512),
    obs=(128, 512), rewrite_p=0.0,
    model=ModelConfig(d_model=5120, n_q_heads=40, n_kv_heads=8, head_dim=128, d_ff=27648,
                      vocab=152064, vocab_chunk=8192))

CONFIGS = {c.name: c for c in (TINY, B1P5, AGENT7B, MULTI7B, LONG32B)}
ORDER = [TINY.name, B1P5.name, AGENT7B.name, MULTI7B.name, LONG32B.name]


def get_config(key) -> WorkloadConfig:
    """Look a workload up by name or by its position (0..4) in ORDER."""
    if isinstance(key, int):
        return CONFIGS[ORDER[key]]
    return CONFIGS[key]
