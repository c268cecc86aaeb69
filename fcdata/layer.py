"""Seeded decoder-layer inputs: bf16 weights, hidden states, cache contents, masks.

bf16 values are carried as raw uint16 bit patterns so both sides see exactly the
same numbers (the oracle upcasts them to float32 exactly).  The weight layout is
row-major [out, in], like torch.nn.Linear.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np


@dataclass(frozen=True)
class LayerShape:
    d: int          # hidden size
    n_heads: int    # query heads
    n_kv: int       # key/value heads
    hd: int         # head dim
    ffn: int        # SwiGLU intermediate size
    eps: float = 1e-6
    theta: float = 1e6

    @property
    def qkv(self) -> int:
        return (self.n_heads + 2 * self.n_kv) * self.hd


# Toy block (4 heads x 64, MHA) and the Qwen2.5-VL-7B LLM block shape.
TINY_LAYER = LayerShape(d=256, n_heads=4, n_kv=4, hd=64, ffn=1024)
QWEN_LAYER = LayerShape(d=3584, n_heads=28, n_kv=4, hd=128, ffn=18944)


def bf16_round(a: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns (uint16), round to nearest even."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    r = ((u >> 16) & 1) + np.uint32(0x7FFF)
    return ((u + r) >> 16).astype(np.uint16)


def bf16_to_f32(u: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) -> float32 (exact)."""
    return (np.asarray(u, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def _normal_bf16(rng: np.random.Generator, shape, std: float) -> np.ndarray:
    return bf16_round(rng.standard_normal(shape, dtype=np.float32) * np.float32(std))


def layer_weights(seed: int, shape: LayerShape, std: float = 0.02) -> dict:
    """Random-init weights of one pre-norm SwiGLU decoder block, bf16 bit patterns.

    Linear weights and the q/k/v biases are N(0, std); RMSNorm gains are 1.
    Keys: w_qkv [qkv, d] (rows q | k | v), b_qkv [qkv], w_o [d, n_heads*hd],
    w_gate [ffn, d], w_up [ffn, d], w_down [d, ffn], g_attn [d], g_mlp [d].
    """
    rng = np.random.default_rng(seed)
    one = bf16_round(np.ones(shape.d, np.float32))
    return dict(
        w_qkv=_normal_bf16(rng, (shape.qkv, shape.d), std),
        b_qkv=_normal_bf16(rng, (shape.qkv,), std),
        w_o=_normal_bf16(rng, (shape.d, shape.n_heads * shape.hd), std),
        w_gate=_normal_bf16(rng, (shape.ffn, shape.d), std),
        w_up=_normal_bf16(rng, (shape.ffn, shape.d), std),
        w_down=_normal_bf16(rng, (shape.d, shape.ffn), std),
        g_attn=one.copy(),
        g_mlp=one.copy(),
    )


def layer_state(seed: int, shape: LayerShape, n_prefix: int, n_frame: int,
                delta: float = 0.1) -> dict:
    """Hidden states for one layer call: prefix rows (text + history frames) and the
    current frame at the previous step, both N(0, 1); the current frame now is
    x_prev + delta * N(0, 1).  All bf16 bit patterns, [rows, d].
    """
    rng = np.random.default_rng(seed)
    prefix = rng.standard_normal((n_prefix, shape.d), dtype=np.float32)
    x_prev = rng.standard_normal((n_frame, shape.d), dtype=np.float32)
    x_cur = x_prev + np.float32(delta) * rng.standard_normal((n_frame, shape.d), dtype=np.float32)
    return dict(prefix=bf16_round(prefix), x_prev=bf16_round(x_prev), x_cur=bf16_round(x_cur))


def text_kv(seed: int, shape: LayerShape, rows: int, std: float = 1.0):
    """Seeded K/V cache contents (bf16 bit patterns, [rows, n_kv, hd] each), used as
    the prompt/pre-history state of an episode's caches."""
    rng = np.random.default_rng(seed)
    k = _normal_bf16(rng, (rows, shape.n_kv, shape.hd), std)
    v = _normal_bf16(rng, (rows, shape.n_kv, shape.hd), std)
    return k, v


def random_reuse_ids(seed: int, n_tokens: int, reuse_percent: int) -> np.ndarray:
    """Recompute ids (int32, ascending) for a random mask that reuses
    floor(reuse_percent * n_tokens / 100) tokens drawn from a seeded permutation."""
    rng = np.random.default_rng(seed)
    k = (reuse_percent * n_tokens) // 100
    perm = rng.permutation(n_tokens)
    reused = np.zeros(n_tokens, bool)
    reused[perm[:k]] = True
    return np.flatnonzero(~reused).astype(np.int32)


def token_embeddings(frames: np.ndarray, d: int, token_px: int, seed: int,
                     std: float = 0.02) -> np.ndarray:
    """Stand-in for the vision tower (out of scope): a fixed seeded linear map of each
    token's token_px x token_px x 3 pixels to d.  frames [F, 3, H, W] float32 ->
    bf16 bit patterns [F, N, d], tokens row-major on the token grid."""
    rng = np.random.default_rng(seed)
    nf, _, h, w = frames.shape
    gh, gw = h // token_px, w // token_px
    proj = rng.standard_normal((3 * token_px * token_px, d), dtype=np.float32) * np.float32(std)
    px = np.asarray(frames, np.float32).reshape(nf, 3, gh, token_px, gw, token_px)
    px = px.transpose(0, 2, 4, 1, 3, 5).reshape(nf, gh * gw, 3 * token_px * token_px)
    return bf16_round(px @ proj)


@dataclass(frozen=True)
class VitShape:
    """A vision-encoder block: hidden size, heads x head dim, MLP size."""
    d: int
    heads: int
    hd: int
    ffn: int
    eps: float = 1e-6
    theta: float = 10000.0


QWEN_VIT = VitShape(d=1280, heads=16, hd=80, ffn=3420)     # Qwen2.5-VL vision block
TINY_VIT = VitShape(d=160, heads=2, hd=80, ffn=192)


def vit_weights(seed: int, shape: VitShape, std: float = 0.02) -> dict:
    """Random-init weights of one vision block, bf16 bit patterns: linear weights and
    biases N(0, std), RMSNorm gains 1 + N(0, 0.1).  Keys: w_qkv [3d, d] (rows q | k | v,
    each head's dims contiguous), b_qkv [3d], w_o [d, d], b_o [d], w_gate / w_up [ffn, d],
    b_gate / b_up [ffn], w_down [d, ffn], b_down [d], g1 [d], g2 [d]."""
    rng = np.random.default_rng(seed)
    d, f = shape.d, shape.ffn

    def gain():
        return bf16_round(1.0 + 0.1 * rng.standard_normal(d, dtype=np.float32))
    return dict(
        w_qkv=_normal_bf16(rng, (3 * d, d), std), b_qkv=_normal_bf16(rng, (3 * d,), std),
        w_o=_normal_bf16(rng, (d, d), std), b_o=_normal_bf16(rng, (d,), std),
        w_gate=_normal_bf16(rng, (f, d), std), b_gate=_normal_bf16(rng, (f,), std),
        w_up=_normal_bf16(rng, (f, d), std), b_up=_normal_bf16(rng, (f,), std),
        w_down=_normal_bf16(rng, (d, f), std), b_down=_normal_bf16(rng, (d,), std),
        g1=gain(), g2=gain())


@dataclass(frozen=True)
class MergerShape:
    """The patch merger: per-patch hidden size d, merge side m, output size d_out."""
    d: int
    m: int
    d_out: int
    eps: float = 1e-6

    @property
    def hidden(self) -> int:
        return self.m * self.m * self.d


QWEN_MERGER = MergerShape(d=1280, m=2, d_out=3584)         # Qwen2.5-VL merger
TINY_MERGER = MergerShape(d=160, m=2, d_out=256)


def merger_weights(seed: int, shape: MergerShape, std: float = 0.02) -> dict:
    """Random-init merger weights, bf16 bit patterns: g [d] = 1 + N(0, 0.1); w1 [hidden,
    hidden], b1 [hidden], w2 [d_out, hidden], b2 [d_out] ~ N(0, std)."""
    rng = np.random.default_rng(seed)
    h = shape.hidden
    return dict(g=bf16_round(1.0 + 0.1 * rng.standard_normal(shape.d, dtype=np.float32)),
                w1=_normal_bf16(rng, (h, h), std), b1=_normal_bf16(rng, (h,), std),
                w2=_normal_bf16(rng, (shape.d_out, h), std),
                b2=_normal_bf16(rng, (shape.d_out,), std))
