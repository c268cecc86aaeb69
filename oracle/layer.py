"""Partial-recompute decoder layer and token-cache update -- CPU oracle, float32.

TEST INFRASTRUCTURE ONLY.  The plain reference for the cached decoder layer
that the HIP path is checked against.  Only tests/, __graft_entry__.smoke() and
the cpu_baseline leg of bench.py may import it.  It shares no code with the
HIP sources.  bf16 inputs (weights, hidden states, cached K/V) arrive as uint16
bit patterns and are upcast exactly; all arithmetic is float32 (RoPE angles are
formed in float64 and rounded).

The paper fixes only what the layer is for: reused tokens keep their cached
results, the rest are recomputed by the model and written back (Sec. 1 and
2.2, Sec. 4.1 on the flush, Sec. 5.2 on the cache the model consumes).  The
block itself is read as a Qwen2-style pre-norm block (RMSNorm, q/k/v bias,
rotate-half RoPE, GQA, SwiGLU), which is the LLM block of the model the paper
deploys (Sec. 6.1).

Sequence layout (the same for every step): [T text tokens][W frame slots of N
tokens].  The frame slots form a ring: physical slot p holds the frame whose
logical index is (p - head) mod W (0 = oldest, W-1 = current).  A key or query
sits at position T + logical * N + token for frames and at its index for text,
so positions are those of the current step's prompt and the K cache holds raw
(pre-RoPE) keys, rotated when used.  With the multimodal RoPE of Qwen2.5-VL (a
reading: the paper deploys that model but does not describe its RoPE) the
rotation angles come from each token's (t, h, w) position instead, while
causality stays by prompt index.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np


def f32(u16: np.ndarray) -> np.ndarray:
    """bf16 bit patterns -> float32 (exact).  float32 arrays pass through unchanged, so
    a caller may carry float32 state (an episode's caches between steps) or hand in
    weights upcast once."""
    if isinstance(u16, np.ndarray) and u16.dtype == np.float32:
        return u16
    return (np.asarray(u16, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


@dataclass(frozen=True)
class Layout:
    T: int      # text tokens
    N: int      # tokens per frame
    W: int      # frames in the window (including the current one)
    head: int   # physical slot of the oldest frame
    gw: int = 0                 # token-grid width of a frame (multimodal RoPE)
    mrope: tuple = (0, 0, 0)    # rotary pairs per (t, h, w) section; zeros = 1-D RoPE
    U: int = 0                  # text tokens after the frames

    @property
    def S(self) -> int:
        return self.T + self.W * self.N + self.U

    def trail_rows(self) -> np.ndarray:
        """Rows (= prompt indices) of the text after the frames."""
        return self.T + self.W * self.N + np.arange(self.U)

    def cur_slot(self) -> int:
        return (self.head + self.W - 1) % self.W

    def prev_slot(self) -> int:
        """Slot of the previous frame (the current slot itself when W == 1)."""
        return (self.head + self.W - 2) % self.W if self.W > 1 else self.cur_slot()

    def row_positions(self) -> np.ndarray:
        """Position of every physical cache row."""
        pos = np.empty(self.S, np.int64)
        pos[:self.T] = np.arange(self.T)
        pos[self.T + self.W * self.N:] = self.trail_rows()
        for p in range(self.W):
            logical = (p - self.head) % self.W
            pos[self.T + p * self.N:self.T + (p + 1) * self.N] = \
                self.T + logical * self.N + np.arange(self.N)
        return pos

    def cur_rows(self, tok: np.ndarray) -> np.ndarray:
        return self.T + self.cur_slot() * self.N + np.asarray(tok)

    def cur_positions(self, tok: np.ndarray) -> np.ndarray:
        return self.T + (self.W - 1) * self.N + np.asarray(tok)

    def rope_positions(self, seqpos: np.ndarray) -> np.ndarray:
        """Multimodal RoPE positions [n, 3] = (t, h, w) of the tokens at prompt indices
        `seqpos` (Qwen2.5-VL): a text token p has (p, p, p); token (I, J) of the frame
        with logical index l has (st, st + I, st + J), st = T + l max(N / gw, gw) -- each
        frame takes as many positions as its longer grid side, after the previous one;
        text after the frames continues at T + W max(N / gw, gw)."""
        pos = np.asarray(seqpos, dtype=np.int64)
        out = np.repeat(pos[:, None], 3, axis=1)
        span = max(self.N // self.gw, self.gw)
        end = self.T + self.W * self.N
        after = pos >= end                 # text after the frames continues after the spans
        out[after] = (pos[after] - end + self.T + self.W * span)[:, None]
        vis = (pos >= self.T) & ~after
        r = pos[vis] - self.T
        l, tok = r // self.N, r % self.N
        st = self.T + l * span
        out[vis, 0] = st
        out[vis, 1] = st + tok // self.gw
        out[vis, 2] = st + tok % self.gw
        return out


def rmsnorm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * g, per row."""
    x = x.astype(np.float32)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return (x / np.sqrt(ms + np.float32(eps))) * g.astype(np.float32)


def rope_cos_sin(pos: np.ndarray, hd: int, theta: float):
    """Rotate-half RoPE angles phi = pos * theta^(-2i/hd), i < hd/2 (float64 -> float32)."""
    inv = theta ** (-(2.0 * np.arange(hd // 2)) / hd)
    ang = np.asarray(pos, dtype=np.float64)[:, None] * inv[None, :]
    return np.cos(ang).astype(np.float32), np.sin(ang).astype(np.float32)


def mrope_cos_sin(pos3: np.ndarray, sections, hd: int, theta: float):
    """Multimodal RoPE angles: rotary pair i of the first sections[0] pairs turns by the
    temporal position, of the next sections[1] by the row position and of the last
    sections[2] by the column position, phi_i = pos_c(i) theta^(-2i/hd)
    (float64 -> float32)."""
    inv = theta ** (-(2.0 * np.arange(hd // 2)) / hd)
    comp = np.repeat(np.arange(3), sections)                      # component of each pair
    assert comp.size == hd // 2
    ang = np.asarray(pos3, dtype=np.float64)[:, comp] * inv[None, :]
    return np.cos(ang).astype(np.float32), np.sin(ang).astype(np.float32)


def layout_rope(lay, seqpos: np.ndarray, hd: int, theta: float):
    """(cos, sin) of the tokens at prompt indices seqpos under the layout's RoPE."""
    if sum(lay.mrope) == 0:
        return rope_cos_sin(seqpos, hd, theta)
    return mrope_cos_sin(lay.rope_positions(seqpos), lay.mrope, hd, theta)


def rope(x: np.ndarray, cos: np.ndarray, sin: np.ndarray) -> np.ndarray:
    """Apply rotate-half RoPE to x [rows, heads, hd] with per-row cos/sin [rows, hd/2]."""
    h = x.shape[-1] // 2
    x1, x2 = x[..., :h], x[..., h:]
    c, s = cos[:, None, :], sin[:, None, :]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def silu(z: np.ndarray) -> np.ndarray:
    return z / (np.float32(1.0) + np.exp(-z))


def attention(q: np.ndarray, qpos: np.ndarray, k: np.ndarray, v: np.ndarray,
              kpos: np.ndarray) -> np.ndarray:
    """Causal softmax attention by position: query r sees keys with kpos <= qpos[r].
    q [n, H, hd] (already rotated), k, v [S, Hkv, hd] (k already rotated); GQA maps
    query head h to kv head h // (H / Hkv).  Returns [n, H, hd]."""
    n, nh, hd = q.shape
    nkv = k.shape[1]
    grp = nh // nkv
    scale = np.float32(1.0 / np.sqrt(hd))
    out = np.empty_like(q)
    visible = kpos[None, :] <= np.asarray(qpos)[:, None]          # [n, S]
    for h in range(nh):
        g = h // grp
        s = (q[:, h, :] @ k[:, g, :].T) * scale                   # [n, S]
        s = np.where(visible, s, -np.inf)
        s = s - s.max(axis=1, keepdims=True)
        p = np.exp(s)
        p = p / p.sum(axis=1, keepdims=True)
        out[:, h, :] = p @ v[:, g, :]
    return out


def _proj(x, w):
    return x @ f32(w).T


def block_rows(x: np.ndarray, qpos: np.ndarray, kc: np.ndarray, vc: np.ndarray,
               kpos: np.ndarray, rows: np.ndarray, wt: dict, shape, lay=None):
    """One decoder block for the rows `x` [n, d] whose K/V go to physical cache rows
    `rows`.  kc/vc [S, Hkv, hd] float32 (raw keys).  qpos/kpos are prompt indices
    (causality); the RoPE angles follow the layout `lay` (1-D by prompt index when
    None).  Returns (y [n, d], kc', vc').

    QKV for every listed row is computed and written first; attention then runs
    over the whole cache, so the rows see each other's new keys and values."""
    nh, nkv, hd = shape.n_heads, shape.n_kv, shape.hd
    n = x.shape[0]
    hn = rmsnorm(x, f32(wt["g_attn"]), shape.eps)
    qkv = _proj(hn, wt["w_qkv"]) + f32(wt["b_qkv"])
    q = qkv[:, :nh * hd].reshape(n, nh, hd)
    k_raw = qkv[:, nh * hd:(nh + nkv) * hd].reshape(n, nkv, hd)
    v_new = qkv[:, (nh + nkv) * hd:].reshape(n, nkv, hd)
    kc = kc.copy()
    vc = vc.copy()
    kc[rows] = k_raw
    vc[rows] = v_new
    if lay is None:
        cq, sq = rope_cos_sin(qpos, hd, shape.theta)
        ck, sk = rope_cos_sin(kpos, hd, shape.theta)
    else:
        cq, sq = layout_rope(lay, qpos, hd, shape.theta)
        ck, sk = layout_rope(lay, kpos, hd, shape.theta)
    o = attention(rope(q, cq, sq), qpos, rope(kc, ck, sk), vc, kpos)
    h1 = x + _proj(o.reshape(n, nh * hd), wt["w_o"])
    h2 = rmsnorm(h1, f32(wt["g_mlp"]), shape.eps)
    act = silu(_proj(h2, wt["w_gate"])) * _proj(h2, wt["w_up"])
    y = h1 + _proj(act, wt["w_down"])
    return y, kc, vc


def layer_full(x_seq_u16: np.ndarray, wt: dict, shape):
    """Full causal forward of an S-row sequence (positions 0..S-1).
    Returns float32 (y [S, d], k_raw [S, Hkv, hd], v [S, Hkv, hd])."""
    x = f32(x_seq_u16)
    s = x.shape[0]
    pos = np.arange(s)
    kc = np.zeros((s, shape.n_kv, shape.hd), np.float32)
    vc = np.zeros_like(kc)
    return block_rows(x, pos, kc, vc, pos, np.arange(s), wt, shape)


def layer_partial(x_cur_u16: np.ndarray, recompute_idx: np.ndarray, k_cache_u16: np.ndarray,
                  v_cache_u16: np.ndarray, y_cur_u16: np.ndarray, lay: Layout, wt: dict, shape):
    """The partial-recompute layer call for one batch item.

    x_cur [N, d]: layer input of the current frame (only recompute_idx rows are
    used); k/v cache [S, Hkv, hd]; y_cur [N, d] output cache of the current
    frame.  Recomputed tokens get new K/V rows in the current slot and new
    output rows; every other row is returned unchanged.  Returns float32
    (y_cur', k_cache', v_cache')."""
    idx = np.asarray(recompute_idx, dtype=np.int64)
    kc, vc = f32(k_cache_u16), f32(v_cache_u16)
    y = f32(y_cur_u16).copy()
    if idx.size == 0:
        return y, kc, vc
    x = f32(x_cur_u16)[idx]
    yr, kc, vc = block_rows(x, lay.cur_positions(idx), kc, vc, lay.row_positions(),
                            lay.cur_rows(idx), wt, shape, lay)
    y[idx] = yr
    return y, kc, vc


def layer_partial_sampled(x_cur_u16: np.ndarray, recompute_idx: np.ndarray,
                          sample_idx: np.ndarray, k_cache_u16: np.ndarray,
                          v_cache_u16: np.ndarray, lay: Layout, wt: dict, shape):
    """The partial-recompute layer call for one batch item, with the block's output
    computed only for `sample_idx` (a subset of recompute_idx): the K/V rows of every
    recomputed token are still computed and written first, since every sampled query
    attends to them.  For large shapes, where computing every output row is too slow.
    Returns float32 (y rows [len(sample_idx), d], k_cache', v_cache')."""
    idx = np.asarray(recompute_idx, dtype=np.int64)
    smp = np.asarray(sample_idx, dtype=np.int64)
    assert np.isin(smp, idx).all(), "samples must be recomputed tokens"
    nh, nkv, hd = shape.n_heads, shape.n_kv, shape.hd
    kc, vc = f32(k_cache_u16).copy(), f32(v_cache_u16).copy()
    x = f32(x_cur_u16)
    hn = rmsnorm(x[idx], f32(wt["g_attn"]), shape.eps)
    kv_rows = slice(nh * hd, (nh + 2 * nkv) * hd)
    kv = _proj(hn, wt["w_qkv"][kv_rows]) + f32(wt["b_qkv"])[kv_rows]
    rows = lay.cur_rows(idx)
    kc[rows] = kv[:, :nkv * hd].reshape(-1, nkv, hd)
    vc[rows] = kv[:, nkv * hd:].reshape(-1, nkv, hd)
    y, kc, vc = block_rows(x[smp], lay.cur_positions(smp), kc, vc, lay.row_positions(),
                           lay.cur_rows(smp), wt, shape, lay)
    return y, kc, vc


def layer_trail(x_trail_u16: np.ndarray, k_cache_u16: np.ndarray, v_cache_u16: np.ndarray,
                lay: Layout, wt: dict, shape):
    """The text after the frames through the block for one batch item: all U rows are
    recomputed (they follow the current frame), their K/V go to rows T + W N + u, and
    they attend causally to the whole cache.  Returns float32 (y [U, d], k', v')."""
    kc, vc = f32(k_cache_u16), f32(v_cache_u16)
    rows = lay.trail_rows()
    return block_rows(f32(x_trail_u16), rows, kc, vc, lay.row_positions(), rows, wt, shape, lay)


def cache_update(k_cache: np.ndarray, v_cache: np.ndarray, y_prev: np.ndarray,
                 y_cur: np.ndarray, shift, reuse_mask: np.ndarray, gw: int, lay: Layout):
    """Token-cache preparation for a new step (window already advanced in `lay`).

    Each reused current-frame token (I, J) takes the cached K/V rows and output
    row of its source token (I + di, J + dj) of the previous frame (Sec. 4.1:
    aligned tokens have a counterpart in the history frame).  Other rows are left
    as they are.  Arrays may be any dtype; copies are returned."""
    kc, vc, yc = k_cache.copy(), v_cache.copy(), y_cur.copy()
    di, dj = shift
    t_ids = np.flatnonzero(np.asarray(reuse_mask) != 0)
    src = (t_ids // gw + di) * gw + (t_ids % gw + dj)
    prev_rows = lay.T + lay.prev_slot() * lay.N + src
    cur_rows = lay.cur_rows(t_ids)
    kc[cur_rows] = k_cache[prev_rows]
    vc[cur_rows] = v_cache[prev_rows]
    yc[t_ids] = y_prev[src]
    return kc, vc, yc
