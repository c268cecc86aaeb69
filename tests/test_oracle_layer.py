"""Pins of the layer / cache oracle against things other than itself.

Library special cases (torch modules and scaled_dot_product_attention on the
CPU in float64), closed forms (RMSNorm of a constant row, RoPE identities) and
the invariants a partial-recompute cache must satisfy: 0 % reuse equals the full
forward, 100 % reuse returns the cache unchanged, and a cache built from the
same inputs makes every mask reproduce the full forward.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import fcdata
from oracle import layer as ol

SMALL = fcdata.LayerShape(d=64, n_heads=4, n_kv=2, hd=16, ffn=96)


def _rel_l2(a, b):
    return float(np.linalg.norm(a - b) / np.linalg.norm(b))


# ------------------------------------------------------------------ PIN-18 RMSNorm
def test_rmsnorm_constant_row():
    """PIN-18: RMSNorm of c * 1 is c / sqrt(c^2 + eps) in every element."""
    for c in (0.5, -3.0, 1e-3):
        x = np.full((2, 64), c, np.float32)
        y = ol.rmsnorm(x, np.ones(64, np.float32), 1e-6)
        np.testing.assert_allclose(y, c / np.sqrt(c * c + 1e-6), rtol=1e-6)


def test_rmsnorm_matches_torch_module():
    x = np.random.default_rng(0).standard_normal((5, 64)).astype(np.float32)
    g = np.random.default_rng(1).uniform(0.5, 1.5, 64).astype(np.float32)
    m = torch.nn.RMSNorm(64, eps=1e-6, dtype=torch.float64)
    m.weight.data = torch.tensor(g, dtype=torch.float64)
    ref = m(torch.tensor(x, dtype=torch.float64)).detach().numpy()
    np.testing.assert_allclose(ol.rmsnorm(x, g, 1e-6), ref, rtol=2e-6, atol=1e-6)


# ------------------------------------------------------------------ PIN-17 RoPE
def test_rope_identities():
    """PIN-17: position 0 is the identity; rotation preserves norms; the score of a
    rotated query/key pair depends only on the position difference."""
    rng = np.random.default_rng(2)
    q = rng.standard_normal((1, 3, 32)).astype(np.float32)
    k = rng.standard_normal((1, 3, 32)).astype(np.float32)
    c0, s0 = ol.rope_cos_sin(np.array([0]), 32, 1e6)
    np.testing.assert_array_equal(ol.rope(q, c0, s0), q)
    c, s = ol.rope_cos_sin(np.array([1234]), 32, 1e6)
    np.testing.assert_allclose(np.linalg.norm(ol.rope(q, c, s), axis=-1),
                               np.linalg.norm(q, axis=-1), rtol=1e-5)

    def score(pq, pk):
        cq, sq = ol.rope_cos_sin(np.array([pq]), 32, 1e4)
        ck, sk = ol.rope_cos_sin(np.array([pk]), 32, 1e4)
        return np.sum(ol.rope(q, cq, sq) * ol.rope(k, ck, sk), axis=-1)
    np.testing.assert_allclose(score(17, 5), score(17 + 300, 5 + 300), rtol=2e-4, atol=2e-4)
    # rotate-half pairs dimension i with i + hd/2 (not adjacent pairs)
    e = np.zeros((1, 1, 32), np.float32)
    e[0, 0, 0] = 1.0
    c1, s1 = ol.rope_cos_sin(np.array([1]), 32, 1e6)
    r = ol.rope(e, c1, s1)
    assert r[0, 0, 16] == pytest.approx(np.sin(1.0), rel=1e-6) and r[0, 0, 1] == 0.0


# ------------------------------------------------------------------ PIN-16 attention
def test_attention_matches_torch_sdpa_gqa():
    """PIN-16: explicit causal softmax attention by position equals torch's
    scaled_dot_product_attention (float64, CPU) with an explicit boolean mask and
    GQA; n_kv = n_heads reduces to MHA."""
    rng = np.random.default_rng(3)
    for nh, nkv in [(4, 2), (6, 6), (7, 1)]:
        n, s, hd = 5, 19, 16
        q = rng.standard_normal((n, nh, hd)).astype(np.float32)
        k = rng.standard_normal((s, nkv, hd)).astype(np.float32)
        v = rng.standard_normal((s, nkv, hd)).astype(np.float32)
        kpos = rng.permutation(s)
        qpos = np.array([3, 18, 7, 0, 12])
        out = ol.attention(q, qpos, k, v, kpos)
        mask = torch.tensor(kpos[None, :] <= qpos[:, None])
        ref = F.scaled_dot_product_attention(
            torch.tensor(q, dtype=torch.float64).transpose(0, 1),
            torch.tensor(k, dtype=torch.float64).transpose(0, 1),
            torch.tensor(v, dtype=torch.float64).transpose(0, 1),
            attn_mask=mask, enable_gqa=True).transpose(0, 1).numpy()
        np.testing.assert_allclose(out, ref, rtol=1e-5, atol=1e-5)


# ------------------------------------------------------------------ block vs library modules
def test_full_block_matches_torch_module_composition():
    """The whole block equals a composition of torch library modules in float64
    (RMSNorm, Linear with bias, SDPA with a causal mask and GQA, SiLU)."""
    sh = SMALL
    wt = fcdata.layer_weights(5, sh, std=0.2)
    x = fcdata.bf16_round(np.random.default_rng(6).standard_normal((11, sh.d)).astype(np.float32))
    y, k_raw, v = ol.layer_full(x, wt, sh)

    t = lambda a: torch.tensor(fcdata.bf16_to_f32(a), dtype=torch.float64)  # noqa: E731
    xt = t(x)
    nrm = torch.nn.RMSNorm(sh.d, eps=sh.eps, dtype=torch.float64)
    hn = nrm(xt)
    qkv = F.linear(hn, t(wt["w_qkv"]), t(wt["b_qkv"]))
    nh, nkv, hd = sh.n_heads, sh.n_kv, sh.hd
    q = qkv[:, :nh * hd].reshape(-1, nh, hd)
    k = qkv[:, nh * hd:(nh + nkv) * hd].reshape(-1, nkv, hd)
    vv = qkv[:, (nh + nkv) * hd:].reshape(-1, nkv, hd)
    pos = torch.arange(11, dtype=torch.float64)
    inv = sh.theta ** (-(torch.arange(hd // 2, dtype=torch.float64) * 2) / hd)
    ang = pos[:, None] * inv[None]
    cos, sin = torch.cos(ang)[:, None, :], torch.sin(ang)[:, None, :]

    def rot(z):
        z1, z2 = z[..., :hd // 2], z[..., hd // 2:]
        return torch.cat([z1 * cos - z2 * sin, z2 * cos + z1 * sin], -1)
    o = F.scaled_dot_product_attention(rot(q).transpose(0, 1), rot(k).transpose(0, 1),
                                       vv.transpose(0, 1), is_causal=True, enable_gqa=True)
    h1 = xt + F.linear(o.transpose(0, 1).reshape(11, -1), t(wt["w_o"]))
    h2 = nrm(h1)
    yr = h1 + F.linear(F.silu(F.linear(h2, t(wt["w_gate"]))) * F.linear(h2, t(wt["w_up"])),
                       t(wt["w_down"]))
    np.testing.assert_allclose(y, yr.detach().numpy(), rtol=2e-4, atol=2e-4)
    np.testing.assert_allclose(k_raw, k.detach().numpy(), rtol=2e-4, atol=2e-4)
    np.testing.assert_allclose(v, vv.detach().numpy(), rtol=2e-4, atol=2e-4)


# ------------------------------------------------------------------ layout
def test_layout_positions_form_the_current_prompt():
    """Physical rows map one-to-one onto prompt positions; the current frame takes the
    last N positions, history frames keep oldest -> newest order whatever the head."""
    for head in range(4):
        lay = ol.Layout(T=3, N=5, W=4, head=head)
        pos = lay.row_positions()
        assert sorted(pos.tolist()) == list(range(lay.S))
        cur = lay.cur_rows(np.arange(5))
        assert pos[cur].tolist() == list(range(lay.S - 5, lay.S))
        assert lay.cur_positions(np.arange(5)).tolist() == list(range(lay.S - 5, lay.S))
        prev = lay.T + lay.prev_slot() * lay.N + np.arange(5)
        assert pos[prev].tolist() == list(range(lay.S - 10, lay.S - 5))


# ------------------------------------------------------------------ PIN-13/14/15 invariants
def _setup(seed=7, T=6, N=8, W=3, head=1, sh=SMALL):
    lay = ol.Layout(T=T, N=N, W=W, head=head)
    wt = fcdata.layer_weights(seed, sh, std=0.1)
    st = fcdata.layer_state(seed + 1, sh, n_prefix=T + (W - 1) * N, n_frame=N)
    # full sequence in position order, then scattered to physical rows
    pos = lay.row_positions()
    seq = np.concatenate([st["prefix"], st["x_prev"]])             # position order
    y, k, v = ol.layer_full(seq, wt, sh)
    kc = fcdata.bf16_round(k[pos])
    vc = fcdata.bf16_round(v[pos])
    y_prev = fcdata.bf16_round(y[-N:])
    return lay, wt, st, kc, vc, y_prev, (y, k, v, pos)


def test_zero_reuse_equals_full_recompute():
    """PIN-13: with every current-frame token recomputed, the layer call reproduces the
    full forward of [prefix; x_cur] on the current rows (K/V of the prefix taken
    from the cache, which holds the full forward's values)."""
    sh = SMALL
    lay, wt, st, kc, vc, y_prev, (_, _, _, pos) = _setup(sh=sh)
    seq_cur = np.concatenate([st["prefix"], st["x_cur"]])
    yf, kf, vf = ol.layer_full(seq_cur, wt, sh)
    # the cache holds bf16 K/V; build the comparison from the same bf16 prefix values
    y, k, v = ol.layer_partial(st["x_cur"], np.arange(lay.N), kc, vc, y_prev, lay, wt, sh)
    assert _rel_l2(y, yf[-lay.N:]) < 1e-2
    np.testing.assert_allclose(k[lay.cur_rows(np.arange(lay.N))], kf[-lay.N:], rtol=1e-5, atol=1e-5)
    # exact version: a cache that stores the full forward's float32 K/V
    kc32 = fcdata.bf16_round(kf[pos])
    y2, _, _ = ol.layer_partial(st["x_cur"], np.arange(lay.N), kc32, fcdata.bf16_round(vf[pos]),
                                y_prev, lay, wt, sh)
    assert _rel_l2(y2, yf[-lay.N:]) < 5e-3


def test_full_reuse_returns_cache_unchanged():
    """PIN-14: with nothing recomputed, K/V and the output cache come back identical."""
    lay, wt, st, kc, vc, y_prev, _ = _setup()
    y, k, v = ol.layer_partial(st["x_cur"], np.array([], np.int32), kc, vc, y_prev, lay, wt, SMALL)
    np.testing.assert_array_equal(fcdata.bf16_round(y), y_prev)
    np.testing.assert_array_equal(fcdata.bf16_round(k), kc)
    np.testing.assert_array_equal(fcdata.bf16_round(v), vc)


def test_cache_from_same_input_makes_every_mask_exact():
    """PIN-15: when the cache was built from the same current-frame input, any subset
    of recomputed tokens reproduces the full forward (to rounding), and untouched
    rows keep their cached values."""
    sh = SMALL
    T, N, W = 6, 8, 3
    lay = ol.Layout(T=T, N=N, W=W, head=2)
    wt = fcdata.layer_weights(11, sh, std=0.1)
    st = fcdata.layer_state(12, sh, n_prefix=T + (W - 1) * N, n_frame=N)
    seq = np.concatenate([st["prefix"], st["x_cur"]])
    yf, kf, vf = ol.layer_full(seq, wt, sh)
    pos = lay.row_positions()
    kc32 = fcdata.bf16_to_f32(fcdata.bf16_round(kf))[pos]
    vc32 = fcdata.bf16_to_f32(fcdata.bf16_round(vf))[pos]
    y_prev = fcdata.bf16_round(yf[-N:])
    for ids in ([0, 3, 7], [5], list(range(N))):
        ids = np.array(ids)
        y, k, _ = ol.layer_partial(st["x_cur"], ids, fcdata.bf16_round(kc32),
                                   fcdata.bf16_round(vc32), y_prev, lay, wt, sh)
        assert _rel_l2(y[ids], yf[-N:][ids]) < 5e-3
        keep = np.setdiff1d(np.arange(N), ids)
        np.testing.assert_array_equal(fcdata.bf16_round(y[keep]), y_prev[keep])


def test_recomputed_rows_see_each_others_new_keys():
    """All recomputed rows' K/V are written before attention: changing the input of one
    recomputed token changes another recomputed token's output only if that token is
    later in the frame (causal), never an earlier one."""
    sh = SMALL
    lay, wt, st, kc, vc, y_prev, _ = _setup(sh=sh)
    ids = np.array([1, 4, 6])
    y0, _, _ = ol.layer_partial(st["x_cur"], ids, kc, vc, y_prev, lay, wt, sh)
    x2 = st["x_cur"].copy()
    x2[4] = fcdata.bf16_round(np.random.default_rng(9).standard_normal(sh.d).astype(np.float32))
    y1, _, _ = ol.layer_partial(x2, ids, kc, vc, y_prev, lay, wt, sh)
    np.testing.assert_array_equal(y0[1], y1[1])
    assert np.abs(y0[6] - y1[6]).max() > 1e-4


# ------------------------------------------------------------------ cache update
def test_cache_update_copies_source_rows():
    """The reused token (I, J) takes the previous frame's token (I+di, J+dj) rows; other
    rows are untouched; W = 1 reads the pre-update copy of the same slot."""
    T, N, gw = 2, 12, 4
    for W, head in [(3, 0), (3, 2), (1, 0)]:
        lay = ol.Layout(T=T, N=N, W=W, head=head)
        rng = np.random.default_rng(W * 10 + head)
        k = rng.standard_normal((lay.S, 2, 4))
        v = rng.standard_normal((lay.S, 2, 4))
        y_prev = rng.standard_normal((N, 5))
        y_cur = rng.standard_normal((N, 5))
        mask = np.zeros(N, np.uint8)
        mask[[0, 5, 6]] = 1            # tokens (0,0), (1,1), (1,2) on a 3x4 grid
        k2, v2, y2 = ol.cache_update(k, v, y_prev, y_cur, (1, 1), mask, gw, lay)
        src = {0: 5, 5: 10, 6: 11}
        for t, s in src.items():
            np.testing.assert_array_equal(k2[lay.cur_rows(t)], k[T + lay.prev_slot() * N + s])
            np.testing.assert_array_equal(v2[lay.cur_rows(t)], v[T + lay.prev_slot() * N + s])
            np.testing.assert_array_equal(y2[t], y_prev[s])
        other = np.setdiff1d(np.arange(N), list(src))
        np.testing.assert_array_equal(y2[other], y_cur[other])
        untouched = np.setdiff1d(np.arange(lay.S), lay.cur_rows(np.array(list(src))))
        np.testing.assert_array_equal(k2[untouched], k[untouched])


def test_sampled_rows_equal_the_full_partial_call():
    """The sampled-output form (every recomputed token's K/V, outputs for a subset)
    gives the same K/V cache and, on the sampled rows, the same outputs as the full
    partial call; it is what the full-size GPU check uses."""
    sh = SMALL
    lay, wt, st, kc, vc, y_prev, _ = _setup(sh=sh)
    ids = fcdata.random_reuse_ids(17, lay.N, 40)
    y, k, v = ol.layer_partial(st["x_cur"], ids, kc, vc, y_prev, lay, wt, sh)
    smp = ids[[0, len(ids) // 2, len(ids) - 1]]
    ys, ks, vs = ol.layer_partial_sampled(st["x_cur"], ids, smp, kc, vc, lay, wt, sh)
    np.testing.assert_allclose(ks, k, rtol=1e-5, atol=1e-6)
    np.testing.assert_allclose(vs, v, rtol=1e-5, atol=1e-6)
    np.testing.assert_allclose(ys, y[smp], rtol=1e-4, atol=1e-5)


# ------------------------------------------------------------------ multimodal RoPE
def test_mrope_positions_hand_layout():
    """Multimodal RoPE positions of a small prompt (2 text tokens, two frames of a 2 x 2
    token grid, ring head 1): text p -> (p, p, p); frame l, token (I, J) ->
    (st, st + I, st + J) with st = T + l max(grid rows, grid cols) = 2 + 2 l."""
    lay = ol.Layout(T=2, N=4, W=2, head=1, gw=2, mrope=(16, 24, 24))
    want = [[0, 0, 0], [1, 1, 1], [2, 2, 2], [2, 2, 3], [2, 3, 2], [2, 3, 3],
            [4, 4, 4], [4, 4, 5], [4, 5, 4], [4, 5, 5]]
    np.testing.assert_array_equal(lay.rope_positions(np.arange(lay.S)), want)
    # a 3-wide, 2-high grid: each frame takes max(2, 3) = 3 positions
    lay = ol.Layout(T=1, N=6, W=2, head=0, gw=3, mrope=(16, 24, 24))
    np.testing.assert_array_equal(lay.rope_positions(np.array([1, 6, 7, 12])),
                                  [[1, 1, 1], [1, 2, 3], [4, 4, 4], [4, 5, 6]])


def test_mrope_matches_transformers_qwen2_vl():
    """The rotation equals transformers' apply_multimodal_rotary_pos_emb of Qwen2-VL (an
    independent implementation: per-component cos/sin over the full head dim, spliced
    by section) for random queries at random (t, h, w) positions."""
    import torch
    from transformers.models.qwen2_vl.modeling_qwen2_vl import apply_multimodal_rotary_pos_emb
    rng = np.random.default_rng(5)
    hd, theta, sec = 128, 1e6, (16, 24, 24)
    n = 40
    pos3 = rng.integers(0, 3000, size=(n, 3))
    x = rng.standard_normal((n, 2, hd)).astype(np.float32)
    c, s = ol.mrope_cos_sin(pos3, sec, hd, theta)
    got = ol.rope(x, c, s)
    inv = theta ** (-(torch.arange(0, hd, 2, dtype=torch.float64) / hd))
    ang = torch.from_numpy(pos3.T.astype(np.float64))[:, None, :, None] * inv       # [3,1,n,64]
    emb = torch.cat([ang, ang], dim=-1)
    xt = torch.from_numpy(x.astype(np.float64)).permute(1, 0, 2)[None]             # [1,2,n,hd]
    q, _ = apply_multimodal_rotary_pos_emb(xt, xt, emb.cos(), emb.sin(), list(sec))
    want = q[0].permute(1, 0, 2).numpy()
    np.testing.assert_allclose(got, want, rtol=2e-5, atol=2e-5)


def test_mrope_reduces_to_rope_and_keeps_relative_positions():
    """Equal components (a text token) rotate exactly as 1-D RoPE; each section turns
    only with its own component; and a common shift of all three components leaves
    every query-key product unchanged (relative positions per component)."""
    rng = np.random.default_rng(6)
    hd, theta, sec = 128, 1e6, (16, 24, 24)
    p = rng.integers(0, 2000, size=9)
    c1, s1 = ol.rope_cos_sin(p, hd, theta)
    c3, s3 = ol.mrope_cos_sin(np.stack([p, p, p], 1), sec, hd, theta)
    np.testing.assert_array_equal(c1, c3)
    np.testing.assert_array_equal(s1, s3)
    base = np.array([[100, 200, 300]])
    for comp, (lo, hi) in enumerate([(0, 16), (16, 40), (40, 64)]):
        moved = base.copy()
        moved[0, comp] += 37
        ca, _ = ol.mrope_cos_sin(base, sec, hd, theta)
        cb, _ = ol.mrope_cos_sin(moved, sec, hd, theta)
        changed = np.flatnonzero(ca[0] != cb[0])
        assert changed.min() >= lo and changed.max() < hi
    q = rng.standard_normal((1, 1, hd)).astype(np.float32)
    k = rng.standard_normal((1, 1, hd)).astype(np.float32)
    pq, pk = np.array([[50, 60, 70]]), np.array([[10, 90, 30]])
    dots = []
    for d in (0, 123):
        cq, sq = ol.mrope_cos_sin(pq + d, sec, hd, theta)
        ck, sk = ol.mrope_cos_sin(pk + d, sec, hd, theta)
        dots.append(float((ol.rope(q, cq, sq) * ol.rope(k, ck, sk)).sum()))
    assert dots[0] == pytest.approx(dots[1], rel=1e-4)


# ------------------------------------------------------------------ text after the frames
def test_trailing_text_positions():
    """Text after the frames sits at its prompt index (1-D) and, with multimodal RoPE,
    continues after the last frame's span: T + W max(grid rows, cols) + u."""
    lay = ol.Layout(T=2, N=4, W=2, head=1, gw=2, mrope=(16, 24, 24), U=3)
    np.testing.assert_array_equal(lay.trail_rows(), [10, 11, 12])
    np.testing.assert_array_equal(lay.row_positions()[10:], [10, 11, 12])
    np.testing.assert_array_equal(lay.rope_positions(np.array([10, 12])), [[6, 6, 6], [8, 8, 8]])


def test_trailing_text_equals_full_causal_forward():
    """With the ring head at 0 (physical = prompt order), recomputing the text after the
    frames over the cache of everything before it gives exactly the rows a full causal
    forward of the whole prompt gives (1-D positions = indices)."""
    shape = fcdata.TINY_LAYER
    wt = fcdata.layer_weights(12, shape)
    lay = ol.Layout(T=8, N=16, W=2, head=0, U=5)
    rng = np.random.default_rng(4)
    x = fcdata.bf16_round(rng.standard_normal((lay.S, shape.d), dtype=np.float32))
    y_full, k_full, v_full = ol.layer_full(x, wt, shape)
    pre = lay.T + lay.W * lay.N
    kc = k_full.copy()
    vc = v_full.copy()
    kc[pre:] = rng.standard_normal(kc[pre:].shape)        # stale trailing rows are rewritten
    vc[pre:] = rng.standard_normal(vc[pre:].shape)
    y, k2, v2 = ol.layer_trail(x[pre:], kc, vc, lay, wt, shape)
    np.testing.assert_allclose(y, y_full[pre:], rtol=2e-5, atol=2e-5)
    np.testing.assert_allclose(k2, k_full, rtol=2e-5, atol=2e-5)
    np.testing.assert_allclose(v2, v_full, rtol=2e-5, atol=2e-5)


def test_frame_tokens_do_not_see_trailing_text():
    """Causality: the current frame's recomputed rows are the same whether or not text
    rows follow the frames (whatever those rows hold)."""
    shape = fcdata.TINY_LAYER
    wt = fcdata.layer_weights(13, shape)
    rng = np.random.default_rng(5)
    base = ol.Layout(T=8, N=16, W=2, head=1)
    with_text = ol.Layout(T=8, N=16, W=2, head=1, U=6)
    k = fcdata.bf16_round(rng.standard_normal((with_text.S, shape.n_kv, shape.hd), dtype=np.float32))
    v = fcdata.bf16_round(rng.standard_normal((with_text.S, shape.n_kv, shape.hd), dtype=np.float32))
    x = fcdata.bf16_round(rng.standard_normal((16, shape.d), dtype=np.float32))
    y0 = fcdata.bf16_round(rng.standard_normal((16, shape.d), dtype=np.float32))
    ids = np.array([1, 4, 9, 15])
    ya, ka, va = ol.layer_partial(x, ids, k[:base.S], v[:base.S], y0, base, wt, shape)
    yb, kb, vb = ol.layer_partial(x, ids, k, v, y0, with_text, wt, shape)
    np.testing.assert_array_equal(ya, yb)
    np.testing.assert_array_equal(ka, kb[:base.S])
