"""Visual-encoder side partial recompute -- CPU oracle, float32.

TEST INFRASTRUCTURE ONLY.  The plain reference for the cached vision block that the
HIP path is checked against.  Only tests/, __graft_entry__.smoke() and the
cpu_baseline leg of bench.py may import it.  It shares no code with the HIP sources.
bf16 inputs arrive as uint16 bit patterns and are upcast exactly; all arithmetic is
float32 (rotary angles formed in float64 and rounded).

The paper flushes the cache by recomputing every token in the visual encoder
(Sec. 4.1) and reuses the cached results of the other tokens; the encoder of the
deployed model is the Qwen2.5-VL vision transformer (Sec. 2.1, Sec. 6.1).  The block
is read as that encoder's block: pre-norm RMSNorm, q/k/v with bias, 2-D rotary
positions, bidirectional attention inside windows of window_tokens x window_tokens
merged tokens (or over the whole frame in the full-attention blocks), an output
projection with bias, and a SiLU-gated MLP with biases.

Patches are stored token-major: the m x m patches of merged token t = (I, J) are rows
t m^2 + a m + c, the patch at pixel-grid position (I m + a, J m + c).  A patch is
recomputed exactly when its token is (the selection decides per token).  Partial
recompute (the same reading as the decoder layer's): recomputed patches get new q, k,
v from their input rows and attend, per block, to the keys of their window, the
reused patches' keys and values coming from the cache (raw keys, rotated at their
position in the current frame); their outputs replace the cached ones, and reused
patches keep their cached outputs.

The encoder ends in the 2 x 2 patch merger (Sec. 2.1: the visual tokens handed to the
language model are merged patches): each patch row RMS-normalised, the m^2 rows of a
merged token concatenated, then a two-layer MLP with biases and the exact (erf) GELU.
It acts on each merged token alone, so only the recomputed tokens go through it.
"""
from __future__ import annotations

from dataclasses import dataclass

import math

import numpy as np

from oracle.layer import f32, rmsnorm, silu


@dataclass(frozen=True)
class VitShape:
    d: int = 1280          # hidden size
    heads: int = 16
    hd: int = 80           # head dim
    ffn: int = 3420        # MLP intermediate size
    eps: float = 1e-6
    theta: float = 10000.0


def patch_positions(gh: int, gw: int, m: int) -> np.ndarray:
    """(row, column) on the patch grid of every patch row, token-major order."""
    t = np.arange(gh * gw)
    I, J = t // gw, t % gw
    a = np.arange(m * m)
    pr = (I[:, None] * m + a[None, :] // m).ravel()
    pc = (J[:, None] * m + a[None, :] % m).ravel()
    return np.stack([pr, pc], axis=1)


def vision_rope(pos: np.ndarray, hd: int, theta: float):
    """cos, sin [n, hd] of the 2-D rotary embedding: the hd/4 frequencies
    theta^(-2i / (hd/2)) times the patch row fill the first hd/4 angles, times the
    patch column the next hd/4; the angle list is repeated for the two halves rotated
    together (rotate-half pairing of dims j and j + hd/2)."""
    half = hd // 2
    inv = 1.0 / theta ** (np.arange(0, half, 2, dtype=np.float64) / half)
    ang = np.concatenate([pos[:, 0:1] * inv[None, :], pos[:, 1:2] * inv[None, :]], axis=1)
    ang = np.concatenate([ang, ang], axis=1)
    return np.cos(ang).astype(np.float32), np.sin(ang).astype(np.float32)


def rotate(x: np.ndarray, cos: np.ndarray, sin: np.ndarray) -> np.ndarray:
    """x [n, heads, hd] rotated: x cos + rotate_half(x) sin, rotate_half(u, v) = (-v, u)."""
    h = x.shape[-1] // 2
    rh = np.concatenate([-x[..., h:], x[..., :h]], axis=-1)
    return x * cos[:, None, :] + rh * sin[:, None, :]


def window_ids(gh: int, gw: int, m: int, window_tokens: int) -> np.ndarray:
    """Window of every patch row: merged token (I, J) lies in window
    (I // wt) * ceil(gw / wt) + J // wt; window_tokens = 0: one window (full attention)."""
    t = np.arange(gh * gw)
    if window_tokens <= 0:
        win = np.zeros_like(t)
    else:
        per_row = -(-gw // window_tokens)
        win = (t // gw) // window_tokens * per_row + (t % gw) // window_tokens
    return np.repeat(win, m * m)


def _lin(x, w, b):
    return x @ w.T + b


def vit_attention(q, k, v, win_q, win_k):
    """Bidirectional softmax attention of queries q [nq, heads, hd] over keys k, v
    [nk, heads, hd] of the same window, scale 1/sqrt(hd)."""
    hd = q.shape[-1]
    s = np.einsum("qhd,khd->hqk", q, k) / np.float32(np.sqrt(hd))
    s = np.where((win_q[:, None] == win_k[None, :])[None], s, -np.inf)
    s = s - s.max(axis=-1, keepdims=True)
    p = np.exp(s)
    p = p / p.sum(axis=-1, keepdims=True)
    return np.einsum("hqk,khd->qhd", p, v).astype(np.float32)


def block_rows(x_rows, rows, k_all, v_all, win, cos, sin, wt, shape):
    """The block for the patch rows `rows` (inputs x_rows, float32) given the raw keys
    and values of every patch (k_all, v_all [Np, heads, hd], the rows' own entries
    already the new ones).  Returns the outputs of those rows."""
    H, hd = shape.heads, shape.hd
    xn = rmsnorm(x_rows, wt["g1"], shape.eps)
    qkv = _lin(xn, wt["w_qkv"], wt["b_qkv"]).reshape(len(rows), 3, H, hd)
    q = rotate(qkv[:, 0], cos[rows], sin[rows])
    kr = rotate(k_all, cos, sin)
    a = vit_attention(q, kr, v_all, win[rows], win).reshape(len(rows), H * hd)
    h1 = x_rows + _lin(a, wt["w_o"], wt["b_o"])
    hn = rmsnorm(h1, wt["g2"], shape.eps)
    act = silu(_lin(hn, wt["w_gate"], wt["b_gate"])) * _lin(hn, wt["w_up"], wt["b_up"])
    return (h1 + _lin(act, wt["w_down"], wt["b_down"])).astype(np.float32)


def new_kv(x_rows, wt, shape):
    """Raw keys and values [n, heads, hd] of the given input rows."""
    xn = rmsnorm(x_rows, wt["g1"], shape.eps)
    qkv = _lin(xn, wt["w_qkv"], wt["b_qkv"]).reshape(len(x_rows), 3, shape.heads, shape.hd)
    return qkv[:, 1], qkv[:, 2]


def vit_block_full(x_u16, wt_u16, shape, gh, gw, m, window_tokens):
    """The whole block on every patch of a frame: outputs y [Np, d] and raw k, v."""
    wt = {k: f32(v) for k, v in wt_u16.items()}
    x = f32(x_u16)
    cos, sin = vision_rope(patch_positions(gh, gw, m), shape.hd, shape.theta)
    win = window_ids(gh, gw, m, window_tokens)
    k, v = new_kv(x, wt, shape)
    rows = np.arange(x.shape[0])
    return block_rows(x, rows, k, v, win, cos, sin, wt, shape), k, v


def vit_block_partial(x_u16, rec_tokens, k_cache_u16, v_cache_u16, y_cache_u16, wt_u16, shape,
                      gh, gw, m, window_tokens):
    """Partial recompute: the patches of the merged tokens rec_tokens get new k, v
    (written into copies of the caches) and new outputs; the other rows keep the
    cache's.  Caches [Np, heads, hd], y_cache [Np, d].  Returns (y, k, v) float32."""
    wt = {k: f32(v) for k, v in wt_u16.items()}
    x = f32(x_u16)
    kc = f32(k_cache_u16).copy()
    vc = f32(v_cache_u16).copy()
    y = f32(y_cache_u16).copy()
    mm = m * m
    rows = (np.asarray(rec_tokens, np.int64)[:, None] * mm + np.arange(mm)[None, :]).ravel()
    if rows.size == 0:
        return y, kc, vc
    kn, vn = new_kv(x[rows], wt, shape)
    kc[rows], vc[rows] = kn, vn
    cos, sin = vision_rope(patch_positions(gh, gw, m), shape.hd, shape.theta)
    win = window_ids(gh, gw, m, window_tokens)
    y[rows] = block_rows(x[rows], rows, kc, vc, win, cos, sin, wt, shape)
    return y, kc, vc


def vit_cache_update(k_cache, v_cache, y_prev, y_cur, shift, reuse_mask, gw: int, m: int):
    """Cache preparation of the encoder for a new frame (one frame slot): every reused
    merged token (I, J) takes the m x m patch rows of K, V (from the caches, which hold
    the previous frame) and of the outputs (from y_prev) of its source token
    (I + di, J + dj).  Other rows are left as they are; copies are returned."""
    kc, vc, yc = k_cache.copy(), v_cache.copy(), y_cur.copy()
    di, dj = shift
    mm = m * m
    for t in np.flatnonzero(np.asarray(reuse_mask) != 0):
        s = (t // gw + di) * gw + (t % gw + dj)
        kc[t * mm:(t + 1) * mm] = k_cache[s * mm:(s + 1) * mm]
        vc[t * mm:(t + 1) * mm] = v_cache[s * mm:(s + 1) * mm]
        yc[t * mm:(t + 1) * mm] = y_prev[s * mm:(s + 1) * mm]
    return kc, vc, yc


@dataclass(frozen=True)
class MergerShape:
    d: int = 1280          # vision hidden size (per patch)
    m: int = 2             # merge side: m^2 patches per token
    d_out: int = 3584      # language-model hidden size
    eps: float = 1e-6

    @property
    def hidden(self) -> int:
        return self.m * self.m * self.d


def gelu(x: np.ndarray) -> np.ndarray:
    """Exact GELU: x Phi(x) = x (1 + erf(x / sqrt 2)) / 2, erf in float64."""
    xd = np.asarray(x, np.float64)
    erf = np.vectorize(math.erf, otypes=[np.float64])
    return (0.5 * xd * (1.0 + erf(xd / math.sqrt(2.0)))).astype(np.float32)


def merger_rows(y_u16, tokens, wt_u16, shape: MergerShape) -> np.ndarray:
    """The merger for the merged tokens `tokens` of one frame: y [Np, d] (the last
    block's outputs, token-major patch rows); weights g [d] (per-patch RMSNorm gain),
    w1 [hidden, hidden], b1 [hidden], w2 [d_out, hidden], b2 [d_out].  Returns
    [len(tokens), d_out] float32."""
    wt = {k: f32(v) for k, v in wt_u16.items()}
    y = f32(y_u16)
    mm = shape.m * shape.m
    t = np.asarray(tokens, np.int64)
    rows = (t[:, None] * mm + np.arange(mm)[None, :]).ravel()
    xn = rmsnorm(y[rows], wt["g"], shape.eps).reshape(len(t), shape.hidden)
    h = gelu(_lin(xn, wt["w1"], wt["b1"]))
    return _lin(h, wt["w2"], wt["b2"]).astype(np.float32)
