"""Seeded synthetic inputs for the merged actor update.

This package only draws random numbers and lays them out: trajectories of
per-call timelines (token ids, author flags, per-turn advantages, the noise
added to the rollout log-probs), per-episode outcome rewards in groups, and
model weights.  It holds none of the
method's arithmetic, so both the CPU oracle and the GPU path may consume it.
"""
from .configs import CONFIGS, WorkloadConfig, ModelConfig, get_config
from .gen import (Timelines, make_timelines, make_weights_numpy, make_weights_torch,
                  AUTHOR_USER, AUTHOR_ENV, AUTHOR_LLM, AUTHOR_MASK, FLAG_BLOCK_START,
                  bf16_round, make_rewards, layer_key, BLOCK_WEIGHTS, LORA_PROJ, lora_key,
                  lora_shapes, make_lora_numpy)

__all__ = ["CONFIGS", "WorkloadConfig", "ModelConfig", "get_config", "Timelines",
           "make_timelines", "make_weights_numpy", "make_weights_torch",
           "AUTHOR_USER", "AUTHOR_ENV", "AUTHOR_LLM", "AUTHOR_MASK", "FLAG_BLOCK_START",
           "bf16_round", "make_rewards", "layer_key", "BLOCK_WEIGHTS", "LORA_PROJ", "lora_key",
           "lora_shapes", "make_lora_numpy"]
