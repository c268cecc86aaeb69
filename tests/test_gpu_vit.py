"""Vision-encoder partial recompute (fc_vit_block_forward, fc_vit_cache_update) through
the C ABI against the oracle (oracle/vit.py): recomputed patch rows and the K/V rows
they write within 2e-2 relative L2 of the float32 oracle, every other row byte-identical,
the cache update byte-exact, and a two-step chain driven by the selection."""
import numpy as np
import pytest
import torch

import fcdata
from oracle import select as osel
from oracle import vit as ov
from tests import fcutil

pytestmark = pytest.mark.gpu

SMALL = fcdata.VitShape(d=320, heads=4, hd=80, ffn=448)
SMALL_MERGER = fcdata.MergerShape(d=320, m=2, d_out=256)


@pytest.fixture(scope="module")
def fc():
    import paper_2604_24391_amd as fc
    fc.lib()
    return fc


@pytest.fixture(scope="module")
def ctx(fc):
    c = fc.Context(fc.Caps(max_batch=3, max_height=448, max_width=448, max_tokens=1024,
                           max_seq=64, max_d_model=3584, max_ffn=18944, max_qkv=4608))
    yield c
    c.close()


def oshape(sh):
    return ov.VitShape(d=sh.d, heads=sh.heads, hd=sh.hd, ffn=sh.ffn)


def gpu_desc(fc, wt, sh):
    """Device weights; the MLP padded to a multiple of 64 with zeros (exact)."""
    f = sh.ffn
    fp = (f + 63) // 64 * 64

    def rows(a, n):
        out = np.zeros((n,) + a.shape[1:], np.uint16)
        out[:a.shape[0]] = a
        return out
    wd = np.zeros((sh.d, fp), np.uint16)
    wd[:, :f] = wt["w_down"]
    w = dict(w_qkv=wt["w_qkv"], b_qkv=wt["b_qkv"], w_o=wt["w_o"], b_o=wt["b_o"],
             w_gate_up=np.concatenate([rows(wt["w_gate"], fp), rows(wt["w_up"], fp)]),
             b_gate_up=np.concatenate([rows(wt["b_gate"], fp), rows(wt["b_up"], fp)]),
             w_down=wd, b_down=wt["b_down"], g1=wt["g1"], g2=wt["g2"])
    return fc.VitDesc(sh.d, sh.heads, sh.hd, fp, {k: fcutil.bf16_gpu(v) for k, v in w.items()})


class VitCase:
    """Previous-frame caches from the oracle's whole block on x_prev; x_cur = x_prev + 0.1 noise."""

    def __init__(self, sh, gh, gw, m, window, B, seed):
        self.sh, self.gh, self.gw, self.m, self.win, self.B = sh, gh, gw, m, window, B
        self.wt = fcdata.vit_weights(seed, sh)
        np_ = gh * gw * m * m
        rng = np.random.default_rng(seed + 1)
        self.x = np.empty((B, np_, sh.d), np.uint16)
        self.k = np.empty((B, np_, sh.heads, sh.hd), np.uint16)
        self.v = np.empty_like(self.k)
        self.y = np.empty((B, np_, sh.d), np.uint16)
        for b in range(B):
            xp = rng.standard_normal((np_, sh.d), dtype=np.float32)
            xc = xp + np.float32(0.1) * rng.standard_normal((np_, sh.d), dtype=np.float32)
            y, k, v = ov.vit_block_full(fcdata.bf16_round(xp), self.wt, oshape(sh), gh, gw, m, window)
            self.k[b], self.v[b], self.y[b] = (fcdata.bf16_round(a) for a in (k, v, y))
            self.x[b] = fcdata.bf16_round(xc)

    def run(self, fc, ctx, ids_per_item):
        B, N = self.B, self.gh * self.gw
        idx = np.full((B, N), -1, np.int32)
        nrec = np.zeros(B, np.int32)
        for b, ids in enumerate(ids_per_item):
            idx[b, :len(ids)] = ids
            nrec[b] = len(ids)
        kc, vc, y = fcutil.bf16_gpu(self.k), fcutil.bf16_gpu(self.v), fcutil.bf16_gpu(self.y)
        cache = fc.VitCache(kc, vc, self.gh, self.gw, self.m, self.win)
        fc.fc_vit_block_forward(ctx, gpu_desc(fc, self.wt, self.sh), cache, fcutil.bf16_gpu(self.x),
                                torch.from_numpy(idx).cuda(), torch.from_numpy(nrec).cuda(), y)
        torch.cuda.synchronize()
        return fcutil.bf16_np(y), fcutil.bf16_np(kc), fcutil.bf16_np(vc)

    def check(self, fc, ctx, ids_per_item):
        y, k, v = self.run(fc, ctx, ids_per_item)
        mm = self.m * self.m
        worst = 0.0
        for b, ids in enumerate(ids_per_item):
            ids = np.asarray(ids, np.int64)
            yo, ko, vo = ov.vit_block_partial(self.x[b], ids, self.k[b], self.v[b], self.y[b],
                                              self.wt, oshape(self.sh), self.gh, self.gw, self.m,
                                              self.win)
            rows = (ids[:, None] * mm + np.arange(mm)[None, :]).ravel()
            keep = np.setdiff1d(np.arange(y.shape[1]), rows)
            np.testing.assert_array_equal(y[b][keep], self.y[b][keep])
            np.testing.assert_array_equal(k[b][keep], self.k[b][keep])
            np.testing.assert_array_equal(v[b][keep], self.v[b][keep])
            if rows.size == 0:
                continue
            errs = [fcutil.rel_l2(fcdata.bf16_to_f32(y[b][rows]), yo[rows]),
                    fcutil.rel_l2(fcdata.bf16_to_f32(k[b][rows]), ko[rows]),
                    fcutil.rel_l2(fcdata.bf16_to_f32(v[b][rows]), vo[rows])]
            x = fcdata.bf16_to_f32(self.x[b][rows])
            yg = fcdata.bf16_to_f32(y[b][rows])
            rnd = np.linalg.norm(fcdata.bf16_to_f32(fcdata.bf16_round(yo[rows])) - yo[rows])
            assert np.linalg.norm(yg - yo[rows]) <= fcutil.LAYER_RTOL * np.linalg.norm(yo[rows] - x) + 2 * rnd
            print(f"item {b} tokens {ids.size}: y {errs[0]:.2e} k {errs[1]:.2e} v {errs[2]:.2e}")
            assert max(errs) <= fcutil.LAYER_RTOL
            worst = max(worst, *errs)
        return worst


@pytest.mark.parametrize("window", [4, 0, 3])
def test_small_block_two_ragged_items(fc, ctx, window):
    """d 320 (4 heads x 80), 8 x 8 merged tokens with the 2 x 2 merge (256 patches), two
    items recomputing 30 % and 70 % of their tokens; windows of 4 tokens, full attention,
    and windows of 3 (ragged last window row and column)."""
    c = VitCase(SMALL, 8, 8, 2, window, 2, seed=300 + window)
    c.check(fc, ctx, [np.sort(fcdata.random_reuse_ids(301, 64, 70)),
                      np.sort(fcdata.random_reuse_ids(302, 64, 30))])


def test_small_block_edges(fc, ctx):
    """Nothing recomputed (everything untouched) and everything recomputed (the whole
    block), in one call."""
    c = VitCase(SMALL, 6, 10, 2, 4, 2, seed=310)
    c.check(fc, ctx, [np.array([], np.int32), np.arange(60, dtype=np.int32)])


def test_qwen_vit_block(fc, ctx):
    """The Qwen2.5-VL vision block shape (1280 = 16 x 80, MLP 3420 padded to 3456) on a
    448 x 448 frame (16 x 16 merged tokens, 1024 patches), windows of 4 tokens, half of
    the tokens recomputed."""
    c = VitCase(fcdata.QWEN_VIT, 16, 16, 2, 4, 1, seed=320)
    worst = c.check(fc, ctx, [np.sort(fcdata.random_reuse_ids(321, 256, 50))])
    print(f"worst rel-L2 {worst:.2e}")


@pytest.mark.parametrize("mode", ["in_place", "separate", "separate_no_y"])
def test_vit_cache_update_matches_oracle(fc, ctx, mode):
    """in_place: the cache holds the previous frame and is remapped in place; separate:
    the reused rows are copied from a previous-frame cache into a distinct one, whose
    other rows stay as they were; separate_no_y: the same without the output rows."""
    sh = SMALL
    gh, gw, m, B = 8, 8, 2, 2
    rng = np.random.default_rng(330)
    np_ = gh * gw * m * m
    k = fcdata.bf16_round(rng.standard_normal((B, np_, sh.heads, sh.hd), dtype=np.float32))
    v = fcdata.bf16_round(rng.standard_normal((B, np_, sh.heads, sh.hd), dtype=np.float32))
    yp = fcdata.bf16_round(rng.standard_normal((B, np_, sh.d), dtype=np.float32))
    yc = fcdata.bf16_round(rng.standard_normal((B, np_, sh.d), dtype=np.float32))
    shifts = np.array([[1, -2], [0, 0]], np.int32)
    reuse = np.zeros((B, gh * gw), np.uint8)
    for b in range(B):
        al = osel.align_mask(gh, gw, *shifts[b]).ravel()
        reuse[b] = al & (rng.random(gh * gw) < 0.6)
    wt = fcdata.vit_weights(331, sh)
    # the destination of the separate modes: stale rows from an older frame
    k_old = fcdata.bf16_round(rng.standard_normal(k.shape, dtype=np.float32))
    v_old = fcdata.bf16_round(rng.standard_normal(v.shape, dtype=np.float32))
    if mode == "in_place":
        kg, vg = fcutil.bf16_gpu(k), fcutil.bf16_gpu(v)
        cache = fc.VitCache(kg, vg, gh, gw, m, 4)
    else:
        kg, vg = fcutil.bf16_gpu(k_old), fcutil.bf16_gpu(v_old)
        cache = fc.VitCache(kg, vg, gh, gw, m, 4, k_prev=fcutil.bf16_gpu(k), v_prev=fcutil.bf16_gpu(v))
    ypg, ycg = fcutil.bf16_gpu(yp), fcutil.bf16_gpu(yc)
    no_y = mode == "separate_no_y"
    fc.fc_vit_cache_update(ctx, gpu_desc(fc, wt, sh), cache, None if no_y else ypg,
                           None if no_y else ycg, torch.from_numpy(shifts).cuda(),
                           torch.from_numpy(reuse).cuda())
    torch.cuda.synchronize()
    mm = m * m
    for b in range(B):
        ko, vo, yo = ov.vit_cache_update(k[b], v[b], yp[b], yc[b], tuple(shifts[b]), reuse[b], gw, m)
        if mode != "in_place":
            moved = np.repeat(reuse[b] != 0, mm)
            ko = np.where(moved[:, None, None], ko, k_old[b])
            vo = np.where(moved[:, None, None], vo, v_old[b])
        np.testing.assert_array_equal(fcutil.bf16_np(kg)[b], ko)
        np.testing.assert_array_equal(fcutil.bf16_np(vg)[b], vo)
        np.testing.assert_array_equal(fcutil.bf16_np(ycg)[b], yc[b] if no_y else yo)


@pytest.mark.parametrize("two_caches", [False, True])
def test_encoder_chain_driven_by_selection(fc, ctx, two_caches):
    """Four frames of a camera trajectory (224 x 224, 2 x 2 merge, 64 tokens; steps up to
    30 px, so the shifts found are (-1, 0), (1, 0) and (4, 2) tokens): each step
    selects on the GPU, remaps the encoder cache, runs one vision block on the recomputed
    tokens and the patch merger on their outputs; the oracle runs the same chain from
    the same start.  The
    selection must match bit for bit and the block's rows as in the single-call tests.
    two_caches: the encoder cache alternates between two buffers (the remap copies the
    reused rows from the previous one, no staging) and no output rows are remapped (a
    block reads only the recomputed rows of its input), so y is compared on those rows."""
    sh = SMALL
    frames = fcdata.episode_frames(43, size=224, n_frames=4, max_step=30)
    m, gh, gw = 2, 8, 8
    mm = m * m
    np_ = gh * gw * mm
    prm = fc.SelectParams(merge=m)
    op = fcutil.oracle_select_params(prm)
    wt = fcdata.vit_weights(340, sh)
    desc = gpu_desc(fc, wt, sh)
    rng = np.random.default_rng(341)
    k0 = fcdata.bf16_round(rng.standard_normal((np_, sh.heads, sh.hd), dtype=np.float32))
    y0 = fcdata.bf16_round(rng.standard_normal((np_, sh.d), dtype=np.float32))
    kvs = [(fcutil.bf16_gpu(k0[None]), fcutil.bf16_gpu(k0[None])),
           (fcutil.bf16_gpu(k0[None]), fcutil.bf16_gpu(k0[None]))]
    ys = [fcutil.bf16_gpu(y0[None]), fcutil.bf16_gpu(y0[None])]
    ko, vo, yo = ov.f32(k0), ov.f32(k0), [ov.f32(y0), ov.f32(y0)]
    sel = fc.SelectOut.alloc(1, gh * gw)
    fr = torch.from_numpy(frames).cuda()
    mwt = fcdata.merger_weights(342, SMALL_MERGER)
    mdesc = merger_desc(fc, mwt, SMALL_MERGER)
    xo_g = torch.zeros(1, gh * gw, SMALL_MERGER.d_out, dtype=torch.bfloat16, device="cuda")
    cur = 0
    for s in range(4):
        x = fcdata.bf16_round(rng.standard_normal((np_, sh.d), dtype=np.float32))
        nxt = 1 - cur
        fc.fc_select(ctx, prm, None if s == 0 else fr[s - 1:s], fr[s:s + 1], sel)
        if two_caches:
            kg, vg = kvs[nxt]
            cache = fc.VitCache(kg, vg, gh, gw, m, 4, k_prev=kvs[cur][0], v_prev=kvs[cur][1])
            fc.fc_vit_cache_update(ctx, desc, cache, None, None, sel.shift, sel.reuse_mask)
        else:
            kg, vg = kvs[0]
            cache = fc.VitCache(kg, vg, gh, gw, m, 4)
            fc.fc_vit_cache_update(ctx, desc, cache, ys[cur], ys[nxt], sel.shift, sel.reuse_mask)
        fc.fc_vit_block_forward(ctx, desc, cache, fcutil.bf16_gpu(x[None]), sel.recompute_idx,
                                sel.n_recompute, ys[nxt])
        torch.cuda.synchronize()
        res = osel.select_item(None if s == 0 else frames[s - 1], frames[s], op)
        mg, esc = fcutil.check_select(fcutil.select_out_np(sel), res, op, 0)
        assert not esc
        kc, vc, yc = ov.vit_cache_update(ko, vo, yo[cur], yo[nxt], res.shift, res.reuse_mask, gw, m)
        y, ko, vo = ov.vit_block_partial(x, res.recompute_idx, kc, vc, yc, wt, oshape(sh), gh, gw,
                                         m, 4)
        yo[nxt] = y
        rows = (res.recompute_idx[:, None].astype(np.int64) * mm + np.arange(mm)).ravel()
        yg = ov.f32(fcutil.bf16_np(ys[nxt])[0])
        kgn = ov.f32(fcutil.bf16_np(kg)[0])
        if not two_caches:
            assert fcutil.rel_l2(yg, y) <= fcutil.LAYER_RTOL, s
        assert fcutil.rel_l2(kgn, ko) <= fcutil.LAYER_RTOL, s
        assert fcutil.rel_l2(ov.f32(fcutil.bf16_np(vg)[0]), vo) <= fcutil.LAYER_RTOL, s
        if rows.size:
            assert fcutil.rel_l2(yg[rows], y[rows]) <= fcutil.LAYER_RTOL, s
        # the merger on the block's outputs: the decoder's input rows of the recomputed tokens
        fc.fc_vit_merger_forward(ctx, mdesc, ys[nxt], sel.recompute_idx, sel.n_recompute, xo_g)
        torch.cuda.synchronize()
        if res.n_recompute:
            want = ov.merger_rows(y, res.recompute_idx, mwt, omerger(SMALL_MERGER))
            got = fcdata.bf16_to_f32(fcutil.bf16_np(xo_g)[0][res.recompute_idx])
            assert fcutil.rel_l2(got, want) <= fcutil.LAYER_RTOL, s
        print(f"step {s}: recomputed {res.n_recompute} tokens, shift {res.shift}")
        cur = nxt


def merger_desc(fc, wt, sh):
    return fc.MergerDesc(sh.d, sh.m, sh.d_out, {k: fcutil.bf16_gpu(v) for k, v in wt.items()})


def omerger(sh):
    return ov.MergerShape(d=sh.d, m=sh.m, d_out=sh.d_out)


def check_merger(fc, ctx, sh, n_tokens, ids_per_item, seed):
    B = len(ids_per_item)
    mm = sh.m * sh.m
    wt = fcdata.merger_weights(seed, sh)
    rng = np.random.default_rng(seed + 1)
    y = fcdata.bf16_round(rng.standard_normal((B, n_tokens * mm, sh.d), dtype=np.float32))
    x0 = fcdata.bf16_round(rng.standard_normal((B, n_tokens, sh.d_out), dtype=np.float32))
    idx = np.full((B, n_tokens), -1, np.int32)
    nrec = np.zeros(B, np.int32)
    for b, ids in enumerate(ids_per_item):
        idx[b, :len(ids)] = ids
        nrec[b] = len(ids)
    xg = fcutil.bf16_gpu(x0)
    fc.fc_vit_merger_forward(ctx, merger_desc(fc, wt, sh), fcutil.bf16_gpu(y),
                             torch.from_numpy(idx).cuda(), torch.from_numpy(nrec).cuda(), xg)
    torch.cuda.synchronize()
    x = fcutil.bf16_np(xg)
    worst = 0.0
    for b, ids in enumerate(ids_per_item):
        keep = np.setdiff1d(np.arange(n_tokens), ids)
        np.testing.assert_array_equal(x[b][keep], x0[b][keep])
        if len(ids) == 0:
            continue
        want = ov.merger_rows(y[b], ids, wt, omerger(sh))
        err = fcutil.rel_l2(fcdata.bf16_to_f32(x[b][ids]), want)
        print(f"merger item {b}: {len(ids)} tokens, rel-L2 {err:.2e}")
        assert err <= fcutil.LAYER_RTOL
        worst = max(worst, err)
    return worst


def test_merger_small_ragged_and_edges(fc, ctx):
    """d 320, 2 x 2 merge (hidden 1280) -> 256, 64 tokens: items recomputing 30 %, none,
    and all of their tokens."""
    check_merger(fc, ctx, SMALL_MERGER, 64,
                 [np.sort(fcdata.random_reuse_ids(350, 64, 70)), np.array([], np.int32)], 351)
    check_merger(fc, ctx, SMALL_MERGER, 64, [np.arange(64, dtype=np.int32)], 352)


@pytest.mark.parametrize("m", [1, 3, 4])
def test_merger_other_merge_factors(fc, ctx, m):
    """d 320 with 1 x 1, 3 x 3 and 4 x 4 merges (hidden 320, 2880, 5120) -> 256, 36
    tokens: one item recomputing 60 % of them, one all of them."""
    sh = fcdata.MergerShape(d=320, m=m, d_out=256)
    check_merger(fc, ctx, sh, 36, [np.sort(fcdata.random_reuse_ids(370 + m, 36, 40)),
                                   np.arange(36, dtype=np.int32)], 375 + m)


def test_merger_qwen_shape(fc, ctx):
    """The Qwen2.5-VL merger (1280 x 4 = 5120 -> 5120 -> 3584) on a 448 x 448 frame's 256
    tokens, half of them recomputed."""
    check_merger(fc, ctx, fcdata.QWEN_MERGER, 256,
                 [np.sort(fcdata.random_reuse_ids(360, 256, 50))], 361)


def test_block_and_merger_replay_from_graph(fc, ctx):
    """The vision block and the merger captured in a HIP graph (they launch kernels only:
    no allocation, memset or host synchronisation); every replay reproduces the eager
    bytes, with eager calls in between."""
    c = VitCase(SMALL, 8, 8, 2, 4, 1, seed=370)
    ids = np.sort(fcdata.random_reuse_ids(371, 64, 50))
    idx = torch.full((1, 64), -1, dtype=torch.int32)
    idx[0, :len(ids)] = torch.from_numpy(ids)
    idx, nrec = idx.cuda(), torch.tensor([len(ids)], dtype=torch.int32, device="cuda")
    desc = gpu_desc(fc, c.wt, SMALL)
    mwt = fcdata.merger_weights(372, SMALL_MERGER)
    mdesc = merger_desc(fc, mwt, SMALL_MERGER)
    k0, v0, y0 = fcutil.bf16_gpu(c.k), fcutil.bf16_gpu(c.v), fcutil.bf16_gpu(c.y)
    kc, vc, y = k0.clone(), v0.clone(), y0.clone()
    x = fcutil.bf16_gpu(c.x)
    xo = torch.zeros(1, 64, SMALL_MERGER.d_out, dtype=torch.bfloat16, device="cuda")
    cache = fc.VitCache(kc, vc, 8, 8, 2, 4)

    def restore():
        kc.copy_(k0)
        vc.copy_(v0)
        y.copy_(y0)
        xo.zero_()

    def call():
        fc.fc_vit_block_forward(ctx, desc, cache, x, idx, nrec, y)
        fc.fc_vit_merger_forward(ctx, mdesc, y, idx, nrec, xo)

    def snap():
        torch.cuda.synchronize()
        return [fcutil.bf16_np(t) for t in (kc, vc, y, xo)]

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        restore()
        call()
    torch.cuda.current_stream().wait_stream(side)
    want = snap()
    graph = torch.cuda.CUDAGraph()
    restore()
    torch.cuda.synchronize()
    with torch.cuda.graph(graph):
        call()
    for rep in range(3):
        restore()
        graph.replay()
        for a, b in zip(snap(), want):
            np.testing.assert_array_equal(a, b, err_msg=f"replay {rep}")
        restore()
        call()
        for a, b in zip(snap(), want):
            np.testing.assert_array_equal(a, b, err_msg=f"eager call after replay {rep}")


@pytest.mark.parametrize("d,heads,hd,ffn,gh,gw,m,window,B", [
    (256, 4, 64, 512, 8, 8, 2, 8, 3),     # head dim 64; one window of 256 keys (4 key blocks);
                                          # 768 slots: the large-tile GEMM over 3 packed items
    (256, 2, 128, 320, 16, 16, 1, 4, 2),  # head dim 128, merge 1 (a patch per token)
    (384, 6, 64, 448, 6, 9, 2, 0, 1),     # full attention over 216 patches (ragged key block)
    (320, 4, 80, 448, 5, 6, 3, 2, 2),     # merge 3: windows of 2 x 2 tokens (36 keys), ragged
                                          # last window row; 540 slots on the large tiles
    (256, 4, 64, 512, 4, 4, 4, 0, 1),     # merge 4: full attention over 16 x 16 patches
])
def test_block_variants(fc, ctx, d, heads, hd, ffn, gh, gw, m, window, B):
    """Shapes beyond the Qwen block: other head dims (attention instantiations), windows
    of several key blocks, merge 1, and items packed across tile borders; ragged
    recompute sets per item (one of them empty when B = 3)."""
    sh = fcdata.VitShape(d=d, heads=heads, hd=hd, ffn=ffn)
    c = VitCase(sh, gh, gw, m, window, B, seed=400 + d + gh + window)
    n = gh * gw
    pct = [60, 15, 100][:B]
    ids = [np.sort(fcdata.random_reuse_ids(401 + b, n, p)) for b, p in enumerate(pct)]
    c.check(fc, ctx, ids)
