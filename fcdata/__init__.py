"""Seeded synthetic inputs shared by the oracle tests, the GPU tests and the benchmark.

This package only draws random numbers and lays them out (frames, camera
trajectories, decoder-layer weights and hidden states).  It holds none of the
FreqCache arithmetic: no transform, similarity, threshold, selection or layer
math lives here, so the CPU oracle and the HIP path stay independent.
"""
from .frames import (canvas, tiny_pair, sel_pairs, episode_frames, TINY, SEL,
                     EPISODE, BATCH)
from .layer import (LayerShape, TINY_LAYER, QWEN_LAYER, bf16_round, bf16_to_f32,
                    layer_weights, layer_state, random_reuse_ids, text_kv, token_embeddings,
                    VitShape, QWEN_VIT, TINY_VIT, vit_weights, MergerShape, QWEN_MERGER,
                    TINY_MERGER, merger_weights)

__all__ = [
    "canvas", "tiny_pair", "sel_pairs", "episode_frames", "TINY", "SEL", "EPISODE",
    "BATCH", "LayerShape", "TINY_LAYER", "QWEN_LAYER", "bf16_round", "bf16_to_f32",
    "layer_weights", "layer_state", "random_reuse_ids", "text_kv", "token_embeddings",
    "VitShape", "QWEN_VIT", "TINY_VIT", "vit_weights", "MergerShape", "QWEN_MERGER",
    "TINY_MERGER", "merger_weights",
]
