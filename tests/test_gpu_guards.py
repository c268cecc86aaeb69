"""Canary guards: every output buffer of the ABI calls is a view into a larger allocation
whose bytes before and after it hold a fixed pattern; after the call (selection, the
pixel-resolution estimates, the decoder layer and its cache remap, the vision block,
its cache remap and the merger) the guard bytes must be unchanged, so a write just past
either end of a buffer is caught."""
import numpy as np
import pytest
import torch

import fcdata
from tests import fcutil

pytestmark = pytest.mark.gpu

GUARD = 4096          # elements on each side (a multiple of 16 bytes for every dtype)


@pytest.fixture(scope="module")
def fc():
    import paper_2604_24391_amd as fc
    fc.lib()
    return fc


class Guarded:
    """Views into guarded allocations; check() compares every guard with its pattern."""

    def __init__(self):
        self.bufs = []

    def new(self, shape, dtype, fill=None):
        n = int(np.prod(shape))
        full = torch.empty(n + 2 * GUARD, dtype=dtype, device="cuda")
        raw = full.view(torch.uint8)
        raw.copy_(torch.arange(raw.numel(), device="cuda", dtype=torch.int32).remainder(251)
                  .to(torch.uint8))
        view = full[GUARD:GUARD + n].view(*shape)
        if fill is not None:
            view.copy_(fill)
        self.bufs.append((full, n, full.view(torch.uint8).clone()))
        return view

    def check(self):
        torch.cuda.synchronize()
        for i, (full, n, ref) in enumerate(self.bufs):
            b = full.view(torch.uint8)
            es = full.element_size()
            head, tail = GUARD * es, (GUARD + n) * es
            assert torch.equal(b[:head], ref[:head]), f"buffer {i}: bytes before it written"
            assert torch.equal(b[tail:], ref[tail:]), f"buffer {i}: bytes after it written"


def test_selection_outputs(fc):
    """fc_select (token grid, pixel and rotation alignment) and fc_select_carry."""
    prev, cur, _ = fcdata.sel_pairs(1, batch=3, size=224)
    B, N = 3, 64
    ctx = fc.Context(fc.Caps(max_batch=B, max_height=224, max_width=224, max_tokens=256,
                             max_seq=64, max_d_model=64, max_ffn=64, max_qkv=64))
    try:
        g = Guarded()
        out = fc.SelectOut(
            sim=g.new((B, N), torch.float32), energy=g.new((B, N), torch.float64),
            reuse_mask=g.new((B, N), torch.uint8), recompute_idx=g.new((B, N), torch.int32),
            n_recompute=g.new((B,), torch.int32), shift=g.new((B, 2), torch.int32),
            scalars=g.new((B, fc.freqcache.NSCALARS), torch.float64),
            counts=g.new((B, fc.freqcache.NCOUNTS), torch.int32),
            flags=g.new((B, N), torch.uint8))
        fp, fcur = torch.from_numpy(prev).cuda(), torch.from_numpy(cur).cuda()
        for prm in (fc.SelectParams(merge=2), fc.SelectParams(merge=2, align_pixel=True),
                    fc.SelectParams(merge=2, align_pixel=True, align_rotation=True)):
            fc.fc_select(ctx, prm, fp, fcur, out)
            g.check()
        nb = fc.select_state_bytes(B, 224, 224)
        st0 = g.new((nb,), torch.uint8)
        st1 = g.new((nb,), torch.uint8)
        fc.fc_select_carry(ctx, fc.SelectParams(merge=2), None, fp, st0, out)
        fc.fc_select_carry(ctx, fc.SelectParams(merge=2), st0, fcur, st1, out)
        g.check()
        sp = g.new((B, 2), torch.float64)
        pk = g.new((B, 2), torch.int32)
        resp = g.new((B, 224, 224), torch.float64)
        ang = g.new((B,), torch.float64)
        fc.fc_phase_correlate(ctx, fp, fcur, sp, pk, resp)
        fc.fc_phase_correlate_rotation(ctx, fp, fcur, sp, ang)
        g.check()
    finally:
        ctx.close()


def test_layer_and_remap_outputs(fc):
    """fc_cache_update (in place, W = 1, and a ring, W = 2) and fc_layer_forward."""
    shape = fcdata.LayerShape(d=512, n_heads=7, n_kv=1, hd=128, ffn=1024)
    T, N, gw, B = 16, 64, 8, 2
    ctx = fc.Context(fc.Caps(max_batch=B, max_height=224, max_width=224, max_tokens=N,
                             max_seq=T + 2 * N, max_d_model=shape.d, max_ffn=shape.ffn,
                             max_qkv=shape.qkv))
    try:
        rng = np.random.default_rng(5)
        desc = fcutil.layer_desc(shape, fcutil.weights_gpu(fcdata.layer_weights(1, shape)))
        for W in (1, 2):
            S = T + W * N
            g = Guarded()

            def rnd(*shp):
                return fcutil.bf16_gpu(fcdata.bf16_round(rng.standard_normal(shp, dtype=np.float32)))
            k = g.new((B, S, shape.n_kv, shape.hd), torch.bfloat16, rnd(B, S, shape.n_kv, shape.hd))
            v = g.new((B, S, shape.n_kv, shape.hd), torch.bfloat16, rnd(B, S, shape.n_kv, shape.hd))
            yp = g.new((B, N, shape.d), torch.bfloat16, rnd(B, N, shape.d))
            yc = g.new((B, N, shape.d), torch.bfloat16, rnd(B, N, shape.d))
            kv = fc.KVCache(k, v, T, N, W, head=W - 1)
            shift = torch.tensor([[1, 0], [0, -1]], dtype=torch.int32, device="cuda")
            reuse = torch.zeros(B, N, dtype=torch.uint8)
            reuse[0, :56] = 1
            reuse[1, 1::2] = 1
            fc.fc_cache_update(ctx, desc, kv, yp, yc, shift, reuse.cuda(), gw)
            g.check()
            ids = np.sort(fcdata.random_reuse_ids(6, N, 50))
            idx = torch.full((B, N), -1, dtype=torch.int32)
            idx[:, :len(ids)] = torch.from_numpy(ids)
            nrec = torch.tensor([len(ids), len(ids) // 2], dtype=torch.int32, device="cuda")
            fc.fc_layer_forward(ctx, desc, kv, rnd(B, N, shape.d), idx.cuda(), nrec, yc)
            g.check()
    finally:
        ctx.close()


def test_vision_outputs(fc):
    """fc_vit_cache_update (in place and from a separate cache), fc_vit_block_forward on
    both GEMM paths (few and many rows) and fc_vit_merger_forward."""
    sh = fcdata.VitShape(d=320, heads=4, hd=80, ffn=448)
    msh = fcdata.MergerShape(d=320, m=2, d_out=256)
    ctx = fc.Context(fc.Caps(max_batch=2, max_height=448, max_width=448, max_tokens=256,
                             max_seq=64, max_d_model=3584, max_ffn=18944, max_qkv=4608))
    try:
        rng = np.random.default_rng(9)
        wt = fcdata.vit_weights(3, sh)
        f = (sh.ffn + 63) // 64 * 64

        def rows(a, n):
            o = np.zeros((n,) + a.shape[1:], np.uint16)
            o[:a.shape[0]] = a
            return o
        wd = np.zeros((sh.d, f), np.uint16)
        wd[:, :sh.ffn] = wt["w_down"]
        w = dict(w_qkv=wt["w_qkv"], b_qkv=wt["b_qkv"], w_o=wt["w_o"], b_o=wt["b_o"],
                 w_gate_up=np.concatenate([rows(wt["w_gate"], f), rows(wt["w_up"], f)]),
                 b_gate_up=np.concatenate([rows(wt["b_gate"], f), rows(wt["b_up"], f)]),
                 w_down=wd, b_down=wt["b_down"], g1=wt["g1"], g2=wt["g2"])
        desc = fc.VitDesc(sh.d, sh.heads, sh.hd, f, {k: fcutil.bf16_gpu(v) for k, v in w.items()})
        mw = fcdata.merger_weights(4, msh)
        mdesc = fc.MergerDesc(msh.d, msh.m, msh.d_out, {k: fcutil.bf16_gpu(v) for k, v in mw.items()})

        def rnd(*shp):
            return fcutil.bf16_gpu(fcdata.bf16_round(rng.standard_normal(shp, dtype=np.float32)))
        for gh, gw, B in ((6, 10, 2), (8, 8, 2)):       # 480 and 512 patch rows in all
            N = gh * gw
            np_ = N * 4
            g = Guarded()
            k = g.new((B, np_, sh.heads, sh.hd), torch.bfloat16, rnd(B, np_, sh.heads, sh.hd))
            v = g.new((B, np_, sh.heads, sh.hd), torch.bfloat16, rnd(B, np_, sh.heads, sh.hd))
            kp = g.new((B, np_, sh.heads, sh.hd), torch.bfloat16, rnd(B, np_, sh.heads, sh.hd))
            vp = g.new((B, np_, sh.heads, sh.hd), torch.bfloat16, rnd(B, np_, sh.heads, sh.hd))
            yp = g.new((B, np_, sh.d), torch.bfloat16, rnd(B, np_, sh.d))
            yc = g.new((B, np_, sh.d), torch.bfloat16, rnd(B, np_, sh.d))
            xo = g.new((B, N, msh.d_out), torch.bfloat16, rnd(B, N, msh.d_out))
            shift = torch.tensor([[1, -1], [0, 2]], dtype=torch.int32, device="cuda")
            reuse = torch.zeros(B, N, dtype=torch.uint8)
            reuse[0, :gw * (gh - 1)] = 1
            reuse[1, ::3] = 1
            reuse = reuse.cuda()
            fc.fc_vit_cache_update(ctx, desc, fc.VitCache(k, v, gh, gw, 2, 4), yp, yc, shift, reuse)
            fc.fc_vit_cache_update(ctx, desc, fc.VitCache(k, v, gh, gw, 2, 4, k_prev=kp, v_prev=vp),
                                   None, None, shift, reuse)
            g.check()
            idx = torch.full((B, N), -1, dtype=torch.int32)
            ids = [np.sort(fcdata.random_reuse_ids(7, N, 30)), np.arange(N, dtype=np.int32)]
            for b in range(B):
                idx[b, :len(ids[b])] = torch.from_numpy(ids[b])
            nrec = torch.tensor([len(i) for i in ids], dtype=torch.int32, device="cuda")
            for win in (4, 0):
                fc.fc_vit_block_forward(ctx, desc, fc.VitCache(k, v, gh, gw, 2, win), rnd(B, np_, sh.d),
                                        idx.cuda(), nrec, yc)
                g.check()
            fc.fc_vit_merger_forward(ctx, mdesc, yc, idx.cuda(), nrec, xo)
            g.check()
    finally:
        ctx.close()


def test_layers_remap_trail_slot_map_and_noalloc_outputs(fc):
    """fc_cache_update_layers over three layers (with and without output rows),
    fc_layer_forward_trail, fc_slot_map_init and the slot-mapped per-step update, and
    fc_select_noalloc."""
    shape = fcdata.LayerShape(d=512, n_heads=7, n_kv=1, hd=128, ffn=1024)
    T, N, W, U, gw, B = 16, 64, 2, 24, 8, 2
    S = T + W * N + U
    ctx = fc.Context(fc.Caps(max_batch=B, max_height=224, max_width=224, max_tokens=N,
                             max_seq=S, max_d_model=shape.d, max_ffn=shape.ffn,
                             max_qkv=shape.qkv))
    try:
        rng = np.random.default_rng(12)
        desc = fcutil.layer_desc(shape, fcutil.weights_gpu(fcdata.layer_weights(2, shape)))

        def rnd(*shp):
            return fcutil.bf16_gpu(fcdata.bf16_round(rng.standard_normal(shp, dtype=np.float32)))
        g = Guarded()
        shift = torch.tensor([[1, 0], [0, -1]], dtype=torch.int32, device="cuda")
        reuse = torch.zeros(B, N, dtype=torch.uint8)
        reuse[0, :40] = 1
        reuse[1, 1::2] = 1
        reuse = reuse.cuda()
        kvs, yps, ycs = [], [], []
        for _ in range(3):
            k = g.new((B, S, shape.n_kv, shape.hd), torch.bfloat16, rnd(B, S, shape.n_kv, shape.hd))
            v = g.new((B, S, shape.n_kv, shape.hd), torch.bfloat16, rnd(B, S, shape.n_kv, shape.hd))
            kvs.append(fc.KVCache(k, v, T, N, W, head=1, trail_tokens=U))
            yps.append(g.new((B, N, shape.d), torch.bfloat16, rnd(B, N, shape.d)))
            ycs.append(g.new((B, N, shape.d), torch.bfloat16, rnd(B, N, shape.d)))
        fc.fc_cache_update_layers(ctx, desc, kvs, yps, ycs, shift, reuse, gw)
        fc.fc_cache_update_layers(ctx, desc, kvs, None, None, shift, reuse, gw)
        g.check()
        ids = np.sort(fcdata.random_reuse_ids(13, N, 40))
        idx = torch.full((B, N), -1, dtype=torch.int32)
        idx[:, :len(ids)] = torch.from_numpy(ids)
        nrec = torch.tensor([len(ids), 5], dtype=torch.int32, device="cuda")
        yt = g.new((B, U, shape.d), torch.bfloat16, rnd(B, U, shape.d))
        fc.fc_layer_forward(ctx, desc, kvs[0], rnd(B, N, shape.d), idx.cuda(), nrec, ycs[0])
        fc.fc_layer_forward_trail(ctx, desc, kvs[0], rnd(B, U, shape.d), yt)
        g.check()
        state = g.new((fc.slot_state_bytes(B, S) // 4,), torch.int32)
        kvm = [fc.KVCache(kvs[i].k, kvs[i].v, T, N, W, head=1, trail_tokens=U, slot_map=state)
               for i in range(2)]
        fc.fc_slot_map_init(ctx, desc, kvm[0], B)
        fc.fc_cache_update_layers(ctx, desc, kvm, None, None, shift, reuse, gw)
        g.check()
    finally:
        ctx.close()
    prev, cur, _ = fcdata.sel_pairs(3, batch=2, size=224)
    g = Guarded()
    B, N = 2, 64
    out = fc.SelectOut(
        sim=g.new((B, N), torch.float32), energy=g.new((B, N), torch.float64),
        reuse_mask=g.new((B, N), torch.uint8), recompute_idx=g.new((B, N), torch.int32),
        n_recompute=g.new((B,), torch.int32), shift=g.new((B, 2), torch.int32),
        scalars=g.new((B, fc.freqcache.NSCALARS), torch.float64),
        counts=g.new((B, fc.freqcache.NCOUNTS), torch.int32),
        flags=g.new((B, N), torch.uint8))
    fc.fc_select_noalloc(fc.SelectParams(merge=2), torch.from_numpy(prev).cuda(),
                         torch.from_numpy(cur).cuda(), out)
    g.check()
