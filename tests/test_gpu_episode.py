"""The per-step chain of an episode against an oracle chain (through the C ABI).

A step is: fc_select_carry on the current frame (the previous frame's spectra carried
from the previous step), the window advance of
every layer's cache, one fc_cache_update_layers call for all layers (each reused
token takes its aligned source token's cached rows, Sec. 4.1 / Eq. 4-2), then
fc_layer_forward layer by layer on the tokens the selection left for recompute
(Algorithm 1 feeding the cache reuse).  The GPU runs it exactly as the benchmark
does: the remap of every layer is launched before the first layer runs.

The oracle runs its own chain from the same seeded start: oracle selection, then
for each layer in order its cache remap and its float32 layer, carrying float32
state from step to step.  Nothing computed on the GPU enters the oracle.  At every
step the selection must match bit for bit (no tolerated mismatch), and every
layer's output rows and K/V rows must be within 2e-2 relative L2 of the oracle's;
cache rows that neither side has written must still hold their initial bytes.
"""
import numpy as np
import pytest
import torch

import fcdata
from oracle import layer as ol
from oracle import select as osel
from tests import fcutil

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def fc():
    import paper_2604_24391_amd as fc
    fc.lib()
    return fc


def check_slot_state(state, S, T, WN):
    """Invariants of a slot state after a step: text and trailing rows in place, frame
    rows on frame pool rows, every reference counted, the free list exactly the frame
    pool rows nobody maps to."""
    st = state.cpu().numpy()
    mp, ref, fre, top = st[:S], st[S:2 * S], st[2 * S:3 * S], int(st[3 * S])
    rows = np.arange(S)
    frame = (rows >= T) & (rows < T + WN)
    np.testing.assert_array_equal(mp[~frame], rows[~frame])
    assert ((mp[frame] >= T) & (mp[frame] < T + WN)).all()
    cnt = np.bincount(mp[frame], minlength=S)
    np.testing.assert_array_equal(ref[T:T + WN], cnt[T:T + WN])
    free = np.sort(fre[:top])
    np.testing.assert_array_equal(free, np.flatnonzero(cnt[T:T + WN] == 0) + T)


def run_chain(fc, ctx, shape, frames, prm, L, T, W, steps, seed, check_every=1, log=print,
              mrope=(0, 0, 0), U=0, slot=False, no_y=False):
    """Run `steps` episode steps on both sides and compare after every checked step.
    slot: the GPU caches are slot-mapped (one state for all layers); no_y: the GPU
    remap moves no output rows (only the recomputed rows of y are compared).
    Returns the per-step recompute counts."""
    F, _, H, Wpx = frames.shape
    m = prm.merge
    gh, gw = H // (14 * m), Wpx // (14 * m)
    N = gh * gw
    S = T + W * N + U
    op = fcutil.oracle_select_params(prm)
    # text after the frames: seeded embeddings (the layer-0 input at every step)
    x_text = fcdata.bf16_round(np.random.default_rng(seed + 2).standard_normal((U, shape.d),
                                                                               dtype=np.float32))
    x_text_gpu = fcutil.bf16_gpu(x_text[None]) if U else None
    emb = fcdata.token_embeddings(frames, shape.d, 14 * m, seed + 1)        # [F, N, d] bf16
    emb_gpu = fcutil.bf16_gpu(emb)
    frames_gpu = torch.from_numpy(np.ascontiguousarray(frames)).cuda()
    sel = fc.SelectOut.alloc(1, N)
    states = [fc.select_state_alloc(1, H, Wpx), fc.select_state_alloc(1, H, Wpx)]
    slot_state = fc.slot_state_alloc(1, S) if slot else None

    # seeded start: random caches and output buffers per layer, identical on both sides
    gpu, ora = [], []
    rng = np.random.default_rng(seed)
    for li in range(L):
        log(f"[episode] generating layer {li} of {L} (d {shape.d})")
        wt = fcdata.layer_weights(seed + 100 + li, shape)
        k0, v0 = fcdata.text_kv(seed + 200 + li, shape, S)
        y0 = fcdata.bf16_round(rng.standard_normal((2, N, shape.d), dtype=np.float32))
        kv = fc.KVCache(fcutil.bf16_gpu(k0[None]), fcutil.bf16_gpu(v0[None]), T, N, W, head=0,
                        grid_w=gw, mrope=tuple(mrope), trail_tokens=U, slot_map=slot_state)
        gpu.append(dict(desc=fcutil.layer_desc(shape, fcutil.weights_gpu(wt)), kv=kv,
                        y=[fcutil.bf16_gpu(y0[0][None]), fcutil.bf16_gpu(y0[1][None])],
                        yt=torch.empty((1, U, shape.d), dtype=torch.bfloat16, device="cuda")
                        if U else None))
        ora.append(dict(wt={k: ol.f32(v).copy() for k, v in wt.items()}, k=ol.f32(k0).copy(),
                        v=ol.f32(v0).copy(), y=[ol.f32(y0[0]).copy(), ol.f32(y0[1]).copy()],
                        k0=k0, v0=v0, written=np.zeros(S, bool)))
    if slot:
        fc.fc_slot_map_init(ctx, gpu[0]["desc"], gpu[0]["kv"], 1)
    head, cur = 0, 0
    counts = []
    for s in range(steps):
        fi = s % F
        prev = None if fi == 0 else frames[fi - 1]
        nxt = 1 - cur
        # ---- GPU: the benchmark's step
        fc.fc_select_carry(ctx, prm, None if fi == 0 else states[(s - 1) % 2],
                           frames_gpu[fi:fi + 1], states[s % 2], sel)
        for g in gpu:
            g["kv"].advance()
        fc.fc_cache_update_layers(ctx, gpu[0]["desc"], [g["kv"] for g in gpu],
                                  None if no_y else [g["y"][cur] for g in gpu],
                                  None if no_y else [g["y"][nxt] for g in gpu],
                                  sel.shift, sel.reuse_mask, gw)
        x = emb_gpu[fi:fi + 1]
        xt = x_text_gpu
        for g in gpu:
            fc.fc_layer_forward(ctx, g["desc"], g["kv"], x, sel.recompute_idx, sel.n_recompute,
                                g["y"][nxt])
            x = g["y"][nxt]
            if U:
                fc.fc_layer_forward_trail(ctx, g["desc"], g["kv"], xt, g["yt"])
                xt = g["yt"]
        # ---- oracle: its own chain
        res = osel.select_item(prev, frames[fi], op)
        head = (head + 1) % W
        lay = ol.Layout(T=T, N=N, W=W, head=head, gw=gw, mrope=tuple(mrope), U=U)
        xo = ol.f32(emb[fi])
        xto = ol.f32(x_text) if U else None
        xs = []
        for o in ora:
            kc, vc, yc = ol.cache_update(o["k"], o["v"], o["y"][cur], o["y"][nxt], res.shift,
                                         res.reuse_mask, gw, lay)
            y, kc, vc = ol.layer_partial(xo, res.recompute_idx, kc, vc, yc, lay, o["wt"], shape)
            o["k"], o["v"], o["y"][nxt] = kc, vc, y
            o["written"][lay.cur_rows(np.arange(N))[res.reuse_mask != 0]] = True
            o["written"][lay.cur_rows(res.recompute_idx)] = True
            xs.append(xo)
            xo = y
            if U:
                yt, o["k"], o["v"] = ol.layer_trail(xto, o["k"], o["v"], lay, o["wt"], shape)
                o["written"][lay.trail_rows()] = True
                o["yt"] = yt
                xto = yt
        cur = nxt
        counts.append(res.n_recompute)
        if s % check_every and s != steps - 1:
            continue
        # ---- compare
        torch.cuda.synchronize()
        o_sel = fcutil.select_out_np(sel)
        mg, esc = fcutil.check_select(o_sel, res, op, 0)
        assert not esc, f"step {s}: {esc}"
        idx = res.recompute_idx
        worst = 0.0
        if slot:
            check_slot_state(slot_state, S, T, W * N)
        for li, (g, o) in enumerate(zip(gpu, ora)):
            yg = ol.f32(fcutil.bf16_np(g["y"][cur])[0])
            kl = g["kv"].logical(g["kv"].k, 1)
            vl = g["kv"].logical(g["kv"].v, 1)
            kg = ol.f32(fcutil.bf16_np(kl)[0])
            vg = ol.f32(fcutil.bf16_np(vl)[0])
            xg = ol.f32(fcutil.bf16_np(emb_gpu[fi:fi + 1] if li == 0 else gpu[li - 1]["y"][cur])[0])
            e_y = fcutil.rel_l2(yg, o["y"][cur]) if not no_y else 0.0
            e_rec = fcutil.rel_l2(yg[idx], o["y"][cur][idx]) if idx.size else 0.0
            e_res = fcutil.rel_l2((yg - xg)[idx], (o["y"][cur] - xs[li])[idx]) if idx.size else 0.0
            w = o["written"]
            e_k = fcutil.rel_l2(kg[w], o["k"][w]) if w.any() else 0.0
            e_v = fcutil.rel_l2(vg[w], o["v"][w]) if w.any() else 0.0
            e_t = fcutil.rel_l2(ol.f32(fcutil.bf16_np(g["yt"])[0]), o["yt"]) if U else 0.0
            for name, e in (("y", e_y), ("y rec", e_rec), ("y-x rec", e_res), ("K", e_k), ("V", e_v),
                            ("y trail", e_t)):
                assert e <= fcutil.LAYER_RTOL, f"step {s} layer {li}: {name} rel-L2 {e:.3e}"
                worst = max(worst, e)
            # rows nobody has written still hold their initial bytes
            np.testing.assert_array_equal(fcutil.bf16_np(kl)[0][~w], o["k0"][~w],
                                          err_msg=f"step {s} layer {li}: unwritten K rows")
            np.testing.assert_array_equal(fcutil.bf16_np(vl)[0][~w], o["v0"][~w],
                                          err_msg=f"step {s} layer {li}: unwritten V rows")
        log(f"[episode] step {s}: n_recompute {res.n_recompute}, shift {res.shift}, "
            f"worst rel-L2 {worst:.2e}")
    return counts


def test_two_toy_layers_ring_of_two(fc):
    """Two toy layers (d 256, 4 heads x 64, SwiGLU 1024), 32 text tokens, a ring of two
    frame slots and 24 text tokens after the frames (recomputed every step, after
    each layer's frame tokens), over six steps of a 448x448 camera trajectory with the
    2x2 merge (256 tokens): the first step is flushed (no previous frame), the rest
    reuse part of the cache."""
    shape = fcdata.TINY_LAYER
    frames = fcdata.episode_frames(31, n_frames=6)
    T, W, N = 32, 2, 256
    ctx = fc.Context(fc.Caps(max_batch=1, max_height=448, max_width=448, max_tokens=N,
                             max_seq=T + W * N + 24, max_d_model=shape.d, max_ffn=shape.ffn,
                             max_qkv=shape.qkv))
    try:
        counts = run_chain(fc, ctx, shape, frames, fc.SelectParams(merge=2), L=2, T=T, W=W,
                           steps=6, seed=500, U=24)
    finally:
        ctx.close()
    assert counts[0] == N and min(counts[1:]) < N


def test_qwen_episode_two_layers(fc):
    """The benchmark's episode workload (seed-2024 trajectory of 448x448 frames, 2x2
    merge, 256 tokens, 128 text tokens, 8-frame window: 2176 cached positions) on
    two Qwen2.5-VL-7B-shaped layers with its multimodal RoPE (t, h, w sections
    16/24/24), in the benchmark's launch configuration (the same context capacities),
    over its 7 warm-up and first 9 measured steps, every step compared."""
    shape = fcdata.QWEN_LAYER
    frames = fcdata.episode_frames(2024, size=448, n_frames=16)
    T, W, N = 128, 8, 256
    ctx = fc.Context(fc.Caps(max_batch=64, max_height=448, max_width=448, max_tokens=1024,
                             max_seq=T + W * N, max_d_model=shape.d, max_ffn=shape.ffn,
                             max_qkv=shape.qkv))
    try:
        counts = run_chain(fc, ctx, shape, frames, fc.SelectParams(merge=2), L=2, T=T, W=W,
                           steps=16, seed=900, mrope=(16, 24, 24))
    finally:
        ctx.close()
    assert counts[0] == N and min(counts[1:]) < N


def test_episode_selection_every_step(fc):
    """Selection of the benchmark's whole trajectory (7 warm-up + 32 measured steps),
    every pair bit-exact against the oracle in one batched call."""
    frames = fcdata.episode_frames(2024, size=448)
    prm = fc.SelectParams(merge=2)
    op = fcutil.oracle_select_params(prm)
    ctx = fc.Context(fc.Caps(max_batch=64, max_height=448, max_width=448, max_tokens=1024,
                             max_seq=64, max_d_model=64, max_ffn=64, max_qkv=64))
    try:
        fr = torch.from_numpy(frames).cuda()
        out = fc.SelectOut.alloc(frames.shape[0] - 1, 256)
        fc.fc_select(ctx, prm, fr[:-1], fr[1:], out)
        torch.cuda.synchronize()
        o = fcutil.select_out_np(out)
        for b in range(frames.shape[0] - 1):
            res = osel.select_item(frames[b], frames[b + 1], op)
            mg, esc = fcutil.check_select(o, res, op, b)
            assert not esc
    finally:
        ctx.close()


def test_toy_chain_in_debug_mode(fc):
    """The toy chain (three steps) with the debug mode on: every launch waits for its
    stream and checks for errors; the results still match the oracle chain."""
    shape = fcdata.TINY_LAYER
    frames = fcdata.episode_frames(31, n_frames=3)
    T, W, N = 32, 2, 256
    before = fc.fc_debug(True)
    ctx = fc.Context(fc.Caps(max_batch=1, max_height=448, max_width=448, max_tokens=N,
                             max_seq=T + W * N + 24, max_d_model=shape.d, max_ffn=shape.ffn,
                             max_qkv=shape.qkv))
    try:
        assert fc.fc_debug() is True
        counts = run_chain(fc, ctx, shape, frames, fc.SelectParams(merge=2), L=2, T=T, W=W,
                           steps=3, seed=501, U=24)
    finally:
        ctx.close()
        fc.fc_debug(before)
    assert counts[0] == N


@pytest.mark.parametrize("W,no_y", [(2, False), (1, False), (3, True)])
def test_slot_mapped_toy_chain(fc, W, no_y):
    """The toy chain on slot-mapped caches (one state for both layers): the remap moves
    no K/V row, reused tokens share their source's pool row, and every step's caches in
    row order match the oracle chain; the slot state stays consistent (references
    counted, free list exact).  W = 1 reuses rows of the frame being replaced; no_y
    leaves the output rows of reused tokens unmoved."""
    shape = fcdata.TINY_LAYER
    frames = fcdata.episode_frames(33, n_frames=7)
    T, N = 32, 256
    ctx = fc.Context(fc.Caps(max_batch=1, max_height=448, max_width=448, max_tokens=N,
                             max_seq=T + W * N + 24, max_d_model=shape.d, max_ffn=shape.ffn,
                             max_qkv=shape.qkv))
    try:
        counts = run_chain(fc, ctx, shape, frames, fc.SelectParams(merge=2), L=2, T=T, W=W,
                           steps=7, seed=510 + W, U=24, slot=True, no_y=no_y)
    finally:
        ctx.close()
    assert counts[0] == N and min(counts[1:]) < N


def test_slot_mapped_qwen_episode(fc):
    """The benchmark's episode workload (two Qwen2.5-VL-7B-shaped layers, multimodal RoPE,
    8-frame window) on slot-mapped caches, 12 steps, every step compared."""
    shape = fcdata.QWEN_LAYER
    frames = fcdata.episode_frames(2024, size=448, n_frames=12)
    T, W, N = 128, 8, 256
    ctx = fc.Context(fc.Caps(max_batch=64, max_height=448, max_width=448, max_tokens=1024,
                             max_seq=T + W * N, max_d_model=shape.d, max_ffn=shape.ffn,
                             max_qkv=shape.qkv))
    try:
        counts = run_chain(fc, ctx, shape, frames, fc.SelectParams(merge=2), L=2, T=T, W=W,
                           steps=12, seed=910, mrope=(16, 24, 24), slot=True)
    finally:
        ctx.close()
    assert counts[0] == N and min(counts[1:]) < N
