"""GPU parity of fc_layer_forward against the float32 oracle (through the C ABI).

Recomputed output rows and the K/V rows they write must be within 2e-2 relative
L2 of the oracle (also for y - x, which removes the exact residual); every other
row of the output cache and of K/V must come back byte-identical.
"""
import numpy as np
import pytest
import torch

import fcdata
from oracle import layer as ol
from tests import fcutil

pytestmark = pytest.mark.gpu

GQA_SMALL = fcdata.LayerShape(d=512, n_heads=7, n_kv=1, hd=128, ffn=1024)


@pytest.fixture(scope="module")
def fc():
    import paper_2604_24391_amd as fc
    return fc


@pytest.fixture(scope="module")
def ctx(fc):
    c = fc.Context(fc.Caps(max_batch=2, max_height=224, max_width=224, max_tokens=256,
                           max_seq=2176, max_d_model=3584, max_ffn=18944, max_qkv=4608))
    yield c
    c.close()


class Case:
    """Seeded inputs for one layer call, the oracle's cache from a full forward of
    [prefix; x_prev], and the GPU tensors."""

    def __init__(self, shape, T, N, W, head, B, seed, wt=None, gw=0, mrope=(0, 0, 0),
                 slot_seed=None):
        self.shape, self.B = shape, B
        self.lay = ol.Layout(T=T, N=N, W=W, head=head, gw=gw, mrope=tuple(mrope))
        self.wt = wt if wt is not None else fcdata.layer_weights(seed, shape)
        pos = self.lay.row_positions()
        S = self.lay.S
        self.x_cur = np.empty((B, N, shape.d), np.uint16)
        self.k = np.empty((B, S, shape.n_kv, shape.hd), np.uint16)
        self.v = np.empty_like(self.k)
        self.y_prev = np.empty((B, N, shape.d), np.uint16)
        for b in range(B):
            st = fcdata.layer_state(seed + 101 + b, shape, n_prefix=T + (W - 1) * N, n_frame=N)
            y, k, v = ol.layer_full(np.concatenate([st["prefix"], st["x_prev"]]), self.wt, shape)
            self.k[b] = fcdata.bf16_round(k[pos])
            self.v[b] = fcdata.bf16_round(v[pos])
            self.y_prev[b] = fcdata.bf16_round(y[-N:])
            self.x_cur[b] = st["x_cur"]
        self.wgpu = fcutil.weights_gpu(self.wt)
        # slot-mapped cache: each item's frame rows at a seeded permutation of the frame
        # pool rows (text rows in place); the physical arrays hold row r at map[r]
        self.smap = None
        if slot_seed is not None:
            rng = np.random.default_rng(slot_seed)
            self.smap = np.tile(np.arange(S, dtype=np.int32), (B, 1))
            for b in range(B):
                self.smap[b, T:T + W * N] = T + rng.permutation(W * N).astype(np.int32)

    def run(self, fc, ctx, ids_per_item):
        B, N = self.B, self.lay.N
        idx = np.full((B, N), -1, np.int32)
        nrec = np.zeros(B, np.int32)
        for b, ids in enumerate(ids_per_item):
            idx[b, :len(ids)] = ids
            nrec[b] = len(ids)
        S = self.lay.S
        kp, vp, state = self.k, self.v, None
        if self.smap is not None:
            kp, vp = np.empty_like(self.k), np.empty_like(self.v)
            for b in range(B):
                kp[b][self.smap[b]] = self.k[b]
                vp[b][self.smap[b]] = self.v[b]
            state = fc.slot_state_alloc(B, S)
            state[:B * S] = torch.from_numpy(self.smap.ravel()).cuda()
        kc, vc = fcutil.bf16_gpu(kp), fcutil.bf16_gpu(vp)
        y = fcutil.bf16_gpu(self.y_prev)
        kv = fc.KVCache(kc, vc, self.lay.T, N, self.lay.W, self.lay.head, grid_w=self.lay.gw,
                        mrope=self.lay.mrope, slot_map=state)
        fc.fc_layer_forward(ctx, fcutil.layer_desc(self.shape, self.wgpu), kv,
                            fcutil.bf16_gpu(self.x_cur), torch.from_numpy(idx).cuda(),
                            torch.from_numpy(nrec).cuda(), y)
        torch.cuda.synchronize()
        k, v = fcutil.bf16_np(kc), fcutil.bf16_np(vc)
        if self.smap is not None:
            k = np.stack([k[b][self.smap[b]] for b in range(B)])
            v = np.stack([v[b][self.smap[b]] for b in range(B)])
        return fcutil.bf16_np(y), k, v

    def check(self, fc, ctx, ids_per_item):
        y, k, v = self.run(fc, ctx, ids_per_item)
        worst = 0.0
        for b, ids in enumerate(ids_per_item):
            ids = np.asarray(ids, np.int64)
            yo, ko, vo = ol.layer_partial(self.x_cur[b], ids, self.k[b], self.v[b],
                                          self.y_prev[b], self.lay, self.wt, self.shape)
            keep = np.setdiff1d(np.arange(self.lay.N), ids)
            np.testing.assert_array_equal(y[b][keep], self.y_prev[b][keep])
            rows = self.lay.cur_rows(ids)
            other = np.setdiff1d(np.arange(self.lay.S), rows)
            np.testing.assert_array_equal(k[b][other], self.k[b][other])
            np.testing.assert_array_equal(v[b][other], self.v[b][other])
            if ids.size == 0:
                continue
            yg = fcdata.bf16_to_f32(y[b][ids])
            x = fcdata.bf16_to_f32(self.x_cur[b][ids])
            e1 = fcutil.rel_l2(yg, yo[ids])
            e2 = fcutil.rel_l2(yg - x, yo[ids] - x)
            e3 = fcutil.rel_l2(fcdata.bf16_to_f32(k[b][rows]), ko[rows])
            e4 = fcutil.rel_l2(fcdata.bf16_to_f32(v[b][rows]), vo[rows])
            print(f"item {b} n={ids.size}: y {e1:.2e}  y-x {e2:.2e}  k {e3:.2e}  v {e4:.2e}")
            for e in (e1, e3, e4):
                assert e <= fcutil.LAYER_RTOL
            # y - x removes the exact residual; the bf16 rounding of the stored output
            # is part of the error budget, on top of 2e-2 of the layer's own update.
            yo_r = yo[ids]
            rnd = np.linalg.norm(fcdata.bf16_to_f32(fcdata.bf16_round(yo_r)) - yo_r)
            assert np.linalg.norm(yg - yo_r) <= fcutil.LAYER_RTOL * np.linalg.norm(yo_r - x) + 2 * rnd
            worst = max(worst, e1, e3, e4)
        return worst


def test_tiny_layer_half_reuse(fc, ctx):
    """Toy block (d 256, 4 heads x 64, SwiGLU 1024), 32 text + 256 visual tokens, the
    cache from a full forward of the previous frame, a random 50 % reuse mask."""
    c = Case(fcdata.TINY_LAYER, T=32, N=256, W=1, head=0, B=1, seed=10)
    c.check(fc, ctx, [fcdata.random_reuse_ids(3, 256, 50)])


@pytest.mark.parametrize("ids", [np.arange(11), np.arange(245, 256), np.array([3, 40, 130])])
def test_key_blocks_after_the_last_query(fc, ctx, ids):
    """Only a few early tokens recomputed: the current frame's key blocks after the
    tile's last query are skipped, which here leaves two of the four key splits with
    no block at all (their partials must drop out of the merge); late tokens skip
    nothing."""
    c = Case(GQA_SMALL, T=32, N=256, W=2, head=0, B=1, seed=25)
    c.check(fc, ctx, [ids])


@pytest.mark.parametrize("head", [0, 2])
def test_gqa_ring_layout_two_items(fc, ctx, head):
    """GQA 7:1 with head_dim 128, a 3-frame ring at two head positions, two batch
    items with different recompute counts (one ragged 32-row tile)."""
    c = Case(GQA_SMALL, T=16, N=64, W=3, head=head, B=2, seed=20 + head)
    c.check(fc, ctx, [fcdata.random_reuse_ids(5, 64, 25), fcdata.random_reuse_ids(6, 64, 75)])


@pytest.mark.parametrize("head", [0, 2])
def test_slot_mapped_gqa_ring_two_items(fc, ctx, head):
    """The same on slot-mapped caches: every frame row at a seeded permutation of the
    pool rows, so attention, the K/V scatter and the untouched rows all go through the
    map (compared in row order)."""
    c = Case(GQA_SMALL, T=16, N=64, W=3, head=head, B=2, seed=20 + head, slot_seed=90 + head)
    c.check(fc, ctx, [fcdata.random_reuse_ids(5, 64, 25), fcdata.random_reuse_ids(6, 64, 75)])


def test_slot_mapped_qwen_layer(fc, ctx):
    """The Qwen2.5-VL-7B-shaped layer (2176 cached rows, multimodal RoPE) on a
    slot-mapped cache at 50 % reuse."""
    c = Case(fcdata.QWEN_LAYER, T=128, N=256, W=8, head=3, B=1, seed=41, gw=16,
             mrope=QWEN_MROPE, slot_seed=95)
    c.check(fc, ctx, [fcdata.random_reuse_ids(150, 256, 50)])


def test_full_reuse_leaves_cache_untouched(fc, ctx):
    """100 % reuse (n_recompute = 0): K/V and the output cache come back unchanged."""
    c = Case(fcdata.TINY_LAYER, T=32, N=256, W=1, head=0, B=1, seed=11)
    y, k, v = c.run(fc, ctx, [np.array([], np.int32)])
    np.testing.assert_array_equal(y, c.y_prev)
    np.testing.assert_array_equal(k, c.k)
    np.testing.assert_array_equal(v, c.v)


def test_deterministic(fc, ctx):
    c = Case(GQA_SMALL, T=16, N=64, W=2, head=1, B=1, seed=30)
    ids = [fcdata.random_reuse_ids(1, 64, 50)]
    a = c.run(fc, ctx, ids)
    b = c.run(fc, ctx, ids)
    for x, y in zip(a, b):
        np.testing.assert_array_equal(x, y)


@pytest.fixture(scope="module")
def qwen_case():
    """One Qwen2.5-VL-7B-shaped layer: 128 text + 8 frames x 256 tokens = 2176."""
    return Case(fcdata.QWEN_LAYER, T=128, N=256, W=8, head=3, B=1, seed=40)


@pytest.mark.parametrize("reuse", [0, 25, 50, 75, 90])
def test_qwen_layer_reuse_ratios(fc, ctx, qwen_case, reuse):
    """Full-size layer at reuse 0/25/50/75/90 % with random masks (0 % = full
    recompute of the current frame), in the launch configuration the benchmark uses."""
    qwen_case.check(fc, ctx, [fcdata.random_reuse_ids(100 + reuse, 256, reuse)])


@pytest.mark.parametrize("W,head,B", [(1, 0, 1), (3, 2, 2), (8, 5, 1)])
def test_cache_update_matches_oracle(fc, ctx, W, head, B):
    """fc_cache_update against the oracle's remap (Sec. 4.1 alignment, Eq. 4-2): each
    reused token takes the K/V rows of its aligned source token in the previous frame's
    slot and its output row; every other byte of K, V and the output cache stays as it
    was.  W = 1 is the in-place window (the previous frame's rows are the current
    slot's), W > 1 a ring at a nonzero head; per-item shifts differ in sign."""
    shape = GQA_SMALL
    N, gw, T = 64, 8, 16
    lay = ol.Layout(T=T, N=N, W=W, head=head)
    rng = np.random.default_rng(100 + 10 * W + B)
    kvw = shape.n_kv * shape.hd
    k = rng.integers(0, 1 << 16, size=(B, lay.S, shape.n_kv, shape.hd), dtype=np.uint16)
    v = rng.integers(0, 1 << 16, size=k.shape, dtype=np.uint16)
    y_prev = rng.integers(0, 1 << 16, size=(B, N, shape.d), dtype=np.uint16)
    y_cur = rng.integers(0, 1 << 16, size=(B, N, shape.d), dtype=np.uint16)
    shifts = np.array([[1, -2], [-3, 1]][:B], np.int32)
    mask = np.zeros((B, N), np.uint8)
    for b in range(B):
        I, J = np.divmod(np.arange(N), gw)
        si, sj = I + shifts[b, 0], J + shifts[b, 1]
        aligned = (si >= 0) & (si < N // gw) & (sj >= 0) & (sj < gw)
        mask[b] = aligned & (rng.random(N) < 0.6)
    kc, vc = fcutil.bf16_gpu(k), fcutil.bf16_gpu(v)
    yp, yc = fcutil.bf16_gpu(y_prev), fcutil.bf16_gpu(y_cur)
    wg = fcutil.weights_gpu(fcdata.layer_weights(0, shape))
    desc = fcutil.layer_desc(shape, wg)
    kv = fc.KVCache(kc, vc, T, N, W, head)
    fc.fc_cache_update(ctx, desc, kv, yp, yc, torch.from_numpy(shifts).cuda(),
                       torch.from_numpy(mask).cuda(), gw)
    torch.cuda.synchronize()
    kg, vg, yg = fcutil.bf16_np(kc), fcutil.bf16_np(vc), fcutil.bf16_np(yc)
    for b in range(B):
        ko, vo, yo = ol.cache_update(k[b].reshape(lay.S, kvw), v[b].reshape(lay.S, kvw),
                                     y_prev[b], y_cur[b], tuple(shifts[b]), mask[b], gw, lay)
        np.testing.assert_array_equal(kg[b].reshape(lay.S, kvw), ko)
        np.testing.assert_array_equal(vg[b].reshape(lay.S, kvw), vo)
        np.testing.assert_array_equal(yg[b], yo)
        assert mask[b].sum() > 0


@pytest.mark.parametrize("W,head", [(1, 0), (3, 2)])
def test_cache_step_advances_and_remaps(fc, ctx, W, head):
    """fc_cache_step(FC_ADVANCE_WINDOW | FC_REMAP) = the head advanced by one slot, then
    fc_cache_update: the descriptor's head and every byte of K, V and the output cache
    equal the oracle's remap on the advanced layout."""
    shape = GQA_SMALL
    N, gw, T, B = 64, 8, 16, 2
    rng = np.random.default_rng(7100 + W)
    kvw = shape.n_kv * shape.hd
    nxt = (head + 1) % W
    lay = ol.Layout(T=T, N=N, W=W, head=nxt)
    k = rng.integers(0, 1 << 16, size=(B, lay.S, shape.n_kv, shape.hd), dtype=np.uint16)
    v = rng.integers(0, 1 << 16, size=k.shape, dtype=np.uint16)
    y_prev = rng.integers(0, 1 << 16, size=(B, N, shape.d), dtype=np.uint16)
    y_cur = rng.integers(0, 1 << 16, size=(B, N, shape.d), dtype=np.uint16)
    shifts = np.array([[1, -2], [-3, 1]], np.int32)
    mask = np.zeros((B, N), np.uint8)
    for b in range(B):
        I, J = np.divmod(np.arange(N), gw)
        si, sj = I + shifts[b, 0], J + shifts[b, 1]
        mask[b] = (si >= 0) & (si < N // gw) & (sj >= 0) & (sj < gw) & (rng.random(N) < 0.6)
    kc, vc = fcutil.bf16_gpu(k), fcutil.bf16_gpu(v)
    yp, yc = fcutil.bf16_gpu(y_prev), fcutil.bf16_gpu(y_cur)
    desc = fcutil.layer_desc(shape, fcutil.weights_gpu(fcdata.layer_weights(0, shape)))
    kv = fc.KVCache(kc, vc, T, N, W, head)
    fc.fc_cache_step(ctx, desc, kv, yp, yc, torch.from_numpy(shifts).cuda(),
                     torch.from_numpy(mask).cuda(), gw, fc.FC_ADVANCE_WINDOW | fc.FC_REMAP, B)
    torch.cuda.synchronize()
    assert kv.head == nxt
    kg, vg, yg = fcutil.bf16_np(kc), fcutil.bf16_np(vc), fcutil.bf16_np(yc)
    for b in range(B):
        ko, vo, yo = ol.cache_update(k[b].reshape(lay.S, kvw), v[b].reshape(lay.S, kvw),
                                     y_prev[b], y_cur[b], tuple(shifts[b]), mask[b], gw, lay)
        np.testing.assert_array_equal(kg[b].reshape(lay.S, kvw), ko)
        np.testing.assert_array_equal(vg[b].reshape(lay.S, kvw), vo)
        np.testing.assert_array_equal(yg[b], yo)
    # the advance alone moves no byte
    before = [fcutil.bf16_np(t) for t in (kc, vc, yc)]
    fc.fc_cache_step(ctx, desc, kv, None, None, None, None, gw, fc.FC_ADVANCE_WINDOW, B)
    torch.cuda.synchronize()
    assert kv.head == (nxt + 1) % W
    for a, t in zip(before, (kc, vc, yc)):
        np.testing.assert_array_equal(fcutil.bf16_np(t), a)


@pytest.mark.parametrize("W,head,n_layers", [(1, 0, 3), (3, 2, 4), (2, 1, 35)])
def test_cache_update_layers_matches_oracle(fc, ctx, W, head, n_layers):
    """fc_cache_update_layers (one launch for many layers' caches) against the oracle's
    remap of each layer (Sec. 4.1 alignment, Eq. 4-2): every layer's cache and output
    buffer holds different bytes, so a layer reading another's rows fails.  35 layers
    take two launches of at most 32; W = 1 takes the in-place per-layer path."""
    shape = GQA_SMALL
    N, gw, T, B = 64, 8, 16, 2
    lay = ol.Layout(T=T, N=N, W=W, head=head)
    rng = np.random.default_rng(7000 + 10 * W + n_layers)
    kvw = shape.n_kv * shape.hd
    shifts = np.array([[1, -2], [-3, 1]], np.int32)
    mask = np.zeros((B, N), np.uint8)
    for b in range(B):
        I, J = np.divmod(np.arange(N), gw)
        si, sj = I + shifts[b, 0], J + shifts[b, 1]
        aligned = (si >= 0) & (si < N // gw) & (sj >= 0) & (sj < gw)
        mask[b] = aligned & (rng.random(N) < 0.6)
    host, kvs, yps, ycs = [], [], [], []
    for _ in range(n_layers):
        k = rng.integers(0, 1 << 16, size=(B, lay.S, shape.n_kv, shape.hd), dtype=np.uint16)
        v = rng.integers(0, 1 << 16, size=k.shape, dtype=np.uint16)
        y_prev = rng.integers(0, 1 << 16, size=(B, N, shape.d), dtype=np.uint16)
        y_cur = rng.integers(0, 1 << 16, size=(B, N, shape.d), dtype=np.uint16)
        host.append((k, v, y_prev, y_cur))
        kvs.append(fc.KVCache(fcutil.bf16_gpu(k), fcutil.bf16_gpu(v), T, N, W, head))
        yps.append(fcutil.bf16_gpu(y_prev))
        ycs.append(fcutil.bf16_gpu(y_cur))
    wg = fcutil.weights_gpu(fcdata.layer_weights(0, shape))
    desc = fcutil.layer_desc(shape, wg)
    fc.fc_cache_update_layers(ctx, desc, kvs, yps, ycs, torch.from_numpy(shifts).cuda(),
                              torch.from_numpy(mask).cuda(), gw)
    torch.cuda.synchronize()
    for (k, v, y_prev, y_cur), kv, yc in zip(host, kvs, ycs):
        kg, vg, yg = fcutil.bf16_np(kv.k), fcutil.bf16_np(kv.v), fcutil.bf16_np(yc)
        for b in range(B):
            ko, vo, yo = ol.cache_update(k[b].reshape(lay.S, kvw), v[b].reshape(lay.S, kvw),
                                         y_prev[b], y_cur[b], tuple(shifts[b]), mask[b], gw, lay)
            np.testing.assert_array_equal(kg[b].reshape(lay.S, kvw), ko)
            np.testing.assert_array_equal(vg[b].reshape(lay.S, kvw), vo)
            np.testing.assert_array_equal(yg[b], yo)
    assert mask.sum() > 0


def test_cache_update_layers_rejects_mixed_heads(fc, ctx):
    """Caches advanced to different steps cannot share one remap."""
    shape = GQA_SMALL
    N, T, W, B = 64, 16, 3, 1
    S = T + W * N
    mk = lambda: torch.zeros(B, S, shape.n_kv, shape.hd, dtype=torch.bfloat16, device="cuda")
    kvs = [fc.KVCache(mk(), mk(), T, N, W, 0), fc.KVCache(mk(), mk(), T, N, W, 1)]
    ys = [torch.zeros(B, N, shape.d, dtype=torch.bfloat16, device="cuda") for _ in range(4)]
    desc = fcutil.layer_desc(shape, fcutil.weights_gpu(fcdata.layer_weights(0, shape)))
    with pytest.raises(fc.FcError, match="head differs"):
        fc.fc_cache_update_layers(ctx, desc, kvs, ys[:2], ys[2:],
                                  torch.zeros(B, 2, dtype=torch.int32, device="cuda"),
                                  torch.zeros(B, N, dtype=torch.uint8, device="cuda"), 8)


# ----------------------------------------------------------------- multimodal RoPE
QWEN_MROPE = (16, 24, 24)      # Qwen2.5-VL's rotary pairs per (t, h, w), head_dim 128


def test_mrope_qwen_layer(fc, ctx, qwen_case):
    """The Qwen2.5-VL-7B-shaped layer with multimodal RoPE (t, h, w sections 16/24/24 of
    the 64 rotary pairs, 16 x 16 token grid) at 25 % reuse, against the oracle."""
    c = Case(fcdata.QWEN_LAYER, T=128, N=256, W=8, head=3, B=1, seed=40, wt=qwen_case.wt,
             gw=16, mrope=QWEN_MROPE)
    c.check(fc, ctx, [fcdata.random_reuse_ids(125, 256, 25)])


@pytest.mark.parametrize("head", [0, 2])
def test_mrope_gqa_ring_two_items(fc, ctx, head):
    """Multimodal RoPE on a 3-frame ring (8 x 8 token grid: each frame spans 8 positions)
    at two head positions, two items; and with head_dim 64 (sections 8/8/16) on the toy
    block."""
    c = Case(GQA_SMALL, T=16, N=64, W=3, head=head, B=2, seed=50 + head, gw=8, mrope=QWEN_MROPE)
    c.check(fc, ctx, [fcdata.random_reuse_ids(7, 64, 25), fcdata.random_reuse_ids(8, 64, 60)])
    c = Case(fcdata.TINY_LAYER, T=32, N=256, W=2, head=head % 2, B=1, seed=55, gw=16,
             mrope=(8, 8, 16))
    c.check(fc, ctx, [fcdata.random_reuse_ids(9, 256, 50)])


def test_mrope_rejects_bad_sections(fc, ctx):
    c = Case(fcdata.TINY_LAYER, T=32, N=256, W=1, head=0, B=1, seed=56, gw=16, mrope=(8, 8, 8))
    with pytest.raises(fc.FcError, match="M-RoPE"):
        c.run(fc, ctx, [np.arange(4)])


# ----------------------------------------------------------------- text after the frames
@pytest.mark.parametrize("mrope", [(0, 0, 0), QWEN_MROPE])
def test_trailing_text_rows(fc, ctx, mrope):
    """A prompt with 40 text tokens after a 3-frame ring: fc_layer_forward on the current
    frame's recomputed tokens (which must not see the trailing text), then
    fc_layer_forward_trail on all 40 trailing rows (which see everything before them,
    the new frame rows included); both against the oracle's two calls in the same
    order, with 1-D and multimodal RoPE."""
    shape = GQA_SMALL
    T, N, W, U, head = 16, 64, 3, 40, 2
    lay = ol.Layout(T=T, N=N, W=W, head=head, gw=8 if sum(mrope) else 0, mrope=tuple(mrope), U=U)
    wt = fcdata.layer_weights(57, shape)
    rng = np.random.default_rng(58)

    def rnd(*shp):
        return fcdata.bf16_round(rng.standard_normal(shp, dtype=np.float32))
    k, v = rnd(1, lay.S, shape.n_kv, shape.hd), rnd(1, lay.S, shape.n_kv, shape.hd)
    x, y_prev, xt = rnd(1, N, shape.d), rnd(1, N, shape.d), rnd(1, U, shape.d)
    ids = fcdata.random_reuse_ids(59, N, 50)
    idx = np.full((1, N), -1, np.int32)
    idx[0, :len(ids)] = ids
    kc, vc, y, yt = fcutil.bf16_gpu(k), fcutil.bf16_gpu(v), fcutil.bf16_gpu(y_prev), fcutil.bf16_gpu(rnd(1, U, shape.d))
    kv = fc.KVCache(kc, vc, T, N, W, head, grid_w=lay.gw, mrope=lay.mrope, trail_tokens=U)
    desc = fcutil.layer_desc(shape, fcutil.weights_gpu(wt))
    fc.fc_layer_forward(ctx, desc, kv, fcutil.bf16_gpu(x), torch.from_numpy(idx).cuda(),
                        torch.tensor([len(ids)], dtype=torch.int32, device="cuda"), y)
    fc.fc_layer_forward_trail(ctx, desc, kv, fcutil.bf16_gpu(xt), yt)
    torch.cuda.synchronize()
    yo, ko, vo = ol.layer_partial(x[0], ids, k[0], v[0], y_prev[0], lay, wt, shape)
    yto, kto, vto = ol.layer_trail(xt[0], ko, vo, lay, wt, shape)
    yg, ytg = fcutil.bf16_np(y)[0], fcutil.bf16_np(yt)[0]
    kg, vg = fcutil.bf16_np(kc)[0], fcutil.bf16_np(vc)[0]
    written = np.concatenate([lay.cur_rows(ids), lay.trail_rows()])
    other = np.setdiff1d(np.arange(lay.S), written)
    np.testing.assert_array_equal(kg[other], k[0][other])
    np.testing.assert_array_equal(vg[other], v[0][other])
    np.testing.assert_array_equal(yg[np.setdiff1d(np.arange(N), ids)],
                                  y_prev[0][np.setdiff1d(np.arange(N), ids)])
    errs = dict(y=fcutil.rel_l2(fcdata.bf16_to_f32(yg[ids]), yo[ids]),
                y_trail=fcutil.rel_l2(fcdata.bf16_to_f32(ytg), yto),
                k=fcutil.rel_l2(fcdata.bf16_to_f32(kg[written]), kto[written]),
                v=fcutil.rel_l2(fcdata.bf16_to_f32(vg[written]), vto[written]))
    print(errs)
    for name, e in errs.items():
        assert e <= fcutil.LAYER_RTOL, name
    # y - x without the exact residual: 2e-2 of the layer's own update, plus the bf16
    # rounding of the stored output (as for the frame rows)
    yt32, xt32 = fcdata.bf16_to_f32(ytg), fcdata.bf16_to_f32(xt[0])
    rnd = np.linalg.norm(fcdata.bf16_to_f32(fcdata.bf16_round(yto)) - yto)
    assert np.linalg.norm(yt32 - yto) <= fcutil.LAYER_RTOL * np.linalg.norm(yto - xt32) + 2 * rnd


# ----------------------------------------------------------------- many gathered rows
# With B * N >= 2048 token slots the projections run as square MFMA tiles with fused
# epilogues (the batched-episode regime); these cases take that path.

@pytest.fixture(scope="module")
def ctx_big(fc):
    c = fc.Context(fc.Caps(max_batch=3, max_height=896, max_width=896, max_tokens=1024,
                           max_seq=4224, max_d_model=3584, max_ffn=18944, max_qkv=4608))
    yield c
    c.close()


def test_batch_path_gqa_ragged(fc, ctx_big):
    """GQA 7:1, head_dim 128, 1024 tokens per frame, three items: a ragged third
    256-row tile (n = 646), a single partial tile (n = 103) and nothing recomputed."""
    c = Case(GQA_SMALL, T=128, N=1024, W=2, head=1, B=3, seed=60)
    worst = c.check(fc, ctx_big, [fcdata.random_reuse_ids(61, 1024, 37),
                                  fcdata.random_reuse_ids(62, 1024, 90),
                                  np.array([], np.int32)])
    print(f"worst rel-L2 {worst:.2e}")


def test_batch_path_mha64_full_recompute(fc, ctx_big):
    """MHA with head_dim 64 (two heads per 128-column wave span), 0 % and 50 % reuse."""
    c = Case(fcdata.TINY_LAYER, T=32, N=1024, W=1, head=0, B=2, seed=70)
    c.check(fc, ctx_big, [fcdata.random_reuse_ids(71, 1024, 0), fcdata.random_reuse_ids(72, 1024, 50)])


def test_batch_path_mrope(fc, ctx_big):
    """The large-M path (keys rotated once per call, fused QKV epilogue) with
    multimodal RoPE on a 32 x 32 token grid, two items."""
    c = Case(GQA_SMALL, T=64, N=1024, W=2, head=1, B=2, seed=75, gw=32, mrope=QWEN_MROPE)
    worst = c.check(fc, ctx_big, [fcdata.random_reuse_ids(76, 1024, 40),
                                  fcdata.random_reuse_ids(77, 1024, 70)])
    print(f"worst rel-L2 {worst:.2e}")


def test_batch_path_slot_map(fc, ctx_big):
    """The large-M path on slot-mapped caches (frame rows at seeded permutations of the
    pool rows): keys rotated and values gathered through the map, the fused QKV
    epilogue scattering into the mapped rows; two ragged items, multimodal RoPE."""
    c = Case(GQA_SMALL, T=64, N=1024, W=2, head=1, B=2, seed=78, gw=32, mrope=QWEN_MROPE,
             slot_seed=79)
    worst = c.check(fc, ctx_big, [fcdata.random_reuse_ids(80, 1024, 40),
                                  fcdata.random_reuse_ids(81, 1024, 85)])
    print(f"worst rel-L2 {worst:.2e}")


@pytest.fixture(scope="module")
def ctx_episodes(fc):
    c = fc.Context(fc.Caps(max_batch=16, max_height=896, max_width=896, max_tokens=1024,
                           max_seq=4224, max_d_model=3584, max_ffn=18944, max_qkv=4608))
    yield c
    c.close()


def test_batched_episode_qwen_layer_sampled(fc, ctx_episodes):
    """The batched-episode launch at full size: the Qwen2.5-VL-7B-shaped layer over 16
    items x 1024 tokens, 128 text + 4 frames = 4224 cached positions, about 35 % reuse
    per item, so the packed 256-row tiles straddle items.  For items 0, 7 and 15 the
    K/V rows of every recomputed token and the outputs of six sampled tokens are
    checked against the oracle; every row that must not change, byte for byte."""
    sh = fcdata.QWEN_LAYER
    B, N = 16, 1024
    lay = ol.Layout(T=128, N=N, W=4, head=1)
    S = lay.S
    wt = fcdata.layer_weights(80, sh)
    rng = np.random.default_rng(81)
    x = fcdata.bf16_round(rng.standard_normal((B, N, sh.d), dtype=np.float32))
    k = fcdata.bf16_round(rng.standard_normal((B, S, sh.n_kv, sh.hd), dtype=np.float32))
    v = fcdata.bf16_round(rng.standard_normal((B, S, sh.n_kv, sh.hd), dtype=np.float32))
    y_prev = fcdata.bf16_round(rng.standard_normal((B, N, sh.d), dtype=np.float32))
    ids = [fcdata.random_reuse_ids(90 + b, N, 35) for b in range(B)]
    idx = np.full((B, N), -1, np.int32)
    nrec = np.array([len(i) for i in ids], np.int32)
    for b in range(B):
        idx[b, :nrec[b]] = ids[b]
    kc, vc, y = fcutil.bf16_gpu(k), fcutil.bf16_gpu(v), fcutil.bf16_gpu(y_prev)
    kv = fc.KVCache(kc, vc, lay.T, N, lay.W, lay.head)
    fc.fc_layer_forward(ctx_episodes, fcutil.layer_desc(sh, fcutil.weights_gpu(wt)), kv,
                        fcutil.bf16_gpu(x), torch.from_numpy(idx).cuda(),
                        torch.from_numpy(nrec).cuda(), y)
    torch.cuda.synchronize()
    yg, kg, vg = fcutil.bf16_np(y), fcutil.bf16_np(kc), fcutil.bf16_np(vc)
    for b in (0, 7, 15):
        n = len(ids[b])
        pick = np.unique(np.concatenate([[0, n - 1], rng.choice(n, 4, replace=False)]))
        smp = ids[b][pick]
        yo, ko, vo = ol.layer_partial_sampled(x[b], ids[b], smp, k[b], v[b], lay, wt, sh)
        rows = lay.cur_rows(ids[b])
        other = np.setdiff1d(np.arange(S), rows)
        np.testing.assert_array_equal(kg[b][other], k[b][other])
        np.testing.assert_array_equal(vg[b][other], v[b][other])
        keep = np.setdiff1d(np.arange(N), ids[b])
        np.testing.assert_array_equal(yg[b][keep], y_prev[b][keep])
        ek = fcutil.rel_l2(fcdata.bf16_to_f32(kg[b][rows]), ko[rows])
        ev = fcutil.rel_l2(fcdata.bf16_to_f32(vg[b][rows]), vo[rows])
        ys = fcdata.bf16_to_f32(yg[b][smp])
        xs = fcdata.bf16_to_f32(x[b][smp])
        ey = fcutil.rel_l2(ys, yo)
        rnd = np.linalg.norm(fcdata.bf16_to_f32(fcdata.bf16_round(yo)) - yo)
        print(f"item {b} n={n}: y {ey:.2e}  y-x {fcutil.rel_l2(ys - xs, yo - xs):.2e}  "
              f"k {ek:.2e}  v {ev:.2e}")
        for e in (ey, ek, ev):
            assert e <= fcutil.LAYER_RTOL
        assert np.linalg.norm(ys - yo) <= fcutil.LAYER_RTOL * np.linalg.norm(yo - xs) + 2 * rnd


# The remaining head groupings the attention kernels are built for: MHA at head_dim 128,
# two query heads per kv head at head_dim 64, four per kv head at head_dim 128.
GROUPINGS = {
    "mha_hd128": fcdata.LayerShape(d=512, n_heads=4, n_kv=4, hd=128, ffn=1024),
    "gqa2_hd64": fcdata.LayerShape(d=512, n_heads=8, n_kv=4, hd=64, ffn=1024),
    "gqa4_hd128": fcdata.LayerShape(d=512, n_heads=8, n_kv=2, hd=128, ffn=1024),
}


@pytest.mark.parametrize("name", sorted(GROUPINGS))
def test_other_head_groupings(fc, ctx, name):
    """Few-row path: two ragged items (30 % and 75 % reuse) on a ring of two frames."""
    c = Case(GROUPINGS[name], T=64, N=256, W=2, head=1, B=2, seed=80)
    worst = c.check(fc, ctx, [fcdata.random_reuse_ids(81, 256, 30),
                              fcdata.random_reuse_ids(82, 256, 75)])
    print(f"{name}: worst rel-L2 {worst:.2e}")


@pytest.mark.parametrize("name", sorted(GROUPINGS))
def test_batch_path_other_head_groupings(fc, ctx_big, name):
    """Large-M path (2 x 1024 token slots): two ragged items at 20 % and 60 % reuse."""
    c = Case(GROUPINGS[name], T=64, N=1024, W=1, head=0, B=2, seed=85)
    worst = c.check(fc, ctx_big, [fcdata.random_reuse_ids(86, 1024, 20),
                                  fcdata.random_reuse_ids(87, 1024, 60)])
    print(f"{name}: worst rel-L2 {worst:.2e}")


@pytest.mark.parametrize("slots", [False, True])
def test_long_cache_few_rows(fc, ctx_big, slots):
    """The few-row path (one item, 1024 tokens per frame) over a window of 4 frames plus
    128 text rows, 4224 cached positions: twice the key blocks per split of the
    benchmark's cache; on copied rows and on a slot-mapped cache."""
    c = Case(GQA_SMALL, T=128, N=1024, W=4, head=2, B=1, seed=90,
             slot_seed=91 if slots else None)
    worst = c.check(fc, ctx_big, [fcdata.random_reuse_ids(92, 1024, 84)])
    print(f"worst rel-L2 {worst:.2e}")
