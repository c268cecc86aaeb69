"""The per-step path under HIP-graph capture: fc_select, the one-launch cache remap
and two decoder layers captured once, replayed with eager steps in between; every
replay must reproduce the eager step byte for byte (the path launches kernels only:
no allocation, no memset and no host synchronisation inside a step)."""
import numpy as np
import pytest
import torch

import fcdata
from tests import fcutil

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def fc():
    import paper_2604_24391_amd as fc
    fc.lib()
    return fc


def test_captured_step_replays_match_eager(fc):
    shape = fcdata.TINY_LAYER
    T, N, W, gw, L = 32, 256, 2, 16, 2
    S = T + W * N
    ctx = fc.Context(fc.Caps(max_batch=1, max_height=224, max_width=224, max_tokens=N,
                             max_seq=S, max_d_model=shape.d, max_ffn=shape.ffn,
                             max_qkv=shape.qkv))
    prev, cur, _ = fcdata.tiny_pair(0)
    fp, fcur = torch.from_numpy(prev).cuda(), torch.from_numpy(cur).cuda()
    prm = fc.SelectParams(adaptive=False, alpha_fixed=0.5)
    sel = fc.SelectOut.alloc(1, N)
    rng = np.random.default_rng(41)
    init, layers = [], []
    for li in range(L):
        wg = fcutil.weights_gpu(fcdata.layer_weights(20 + li, shape))
        desc = fcutil.layer_desc(shape, wg)
        st = {n: fcutil.bf16_gpu(fcdata.bf16_round(rng.standard_normal(sz).astype(np.float32)))
              for n, sz in (("k", (1, S, shape.n_kv, shape.hd)), ("v", (1, S, shape.n_kv, shape.hd)),
                            ("y0", (1, N, shape.d)), ("y1", (1, N, shape.d)))}
        init.append({n: t.clone() for n, t in st.items()})
        layers.append(dict(desc=desc, st=st, kv=fc.KVCache(st["k"], st["v"], T, N, W, head=1)))
    x = fcutil.bf16_gpu(fcdata.bf16_round(rng.standard_normal((1, N, shape.d)).astype(np.float32)))

    def restore():
        for lay, s0 in zip(layers, init):
            for n, t in lay["st"].items():
                t.copy_(s0[n])

    def step():
        fc.fc_select(ctx, prm, fp, fcur, sel)
        fc.fc_cache_update_layers(ctx, layers[0]["desc"], [l["kv"] for l in layers],
                                  [l["st"]["y0"] for l in layers], [l["st"]["y1"] for l in layers],
                                  sel.shift, sel.reuse_mask, gw)
        h = x
        for l in layers:
            fc.fc_layer_forward(ctx, l["desc"], l["kv"], h, sel.recompute_idx, sel.n_recompute,
                                l["st"]["y1"])
            h = l["st"]["y1"]

    def snapshot():
        torch.cuda.synchronize()
        out = [fcutil.bf16_np(l["st"][n]) for l in layers for n in ("k", "v", "y1")]
        return out + [sel.reuse_mask.cpu().numpy(), sel.recompute_idx.cpu().numpy()]

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        restore()
        step()
    torch.cuda.current_stream().wait_stream(side)
    want = snapshot()
    assert 0 < int(sel.n_recompute[0]) < N
    graph = torch.cuda.CUDAGraph()
    restore()
    torch.cuda.synchronize()
    with torch.cuda.graph(graph):
        step()
    for rep in range(3):
        restore()
        graph.replay()
        got = snapshot()
        for a, b in zip(got, want):
            np.testing.assert_array_equal(a, b, err_msg=f"replay {rep}")
        restore()
        step()                                    # eager work between the replays
        for a, b in zip(snapshot(), want):
            np.testing.assert_array_equal(a, b, err_msg=f"eager step after replay {rep}")
    ctx.close()


def test_captured_batch_selection_replays_match_eager(fc):
    """fc_select on 64 pairs (the batch the selection benchmark times) captured into a
    graph: every replay, after eager calls on other frames have overwritten the
    outputs, must give the eager result byte for byte."""
    B = 64
    ctx = fc.Context(fc.Caps(max_batch=B, max_height=448, max_width=448, max_tokens=1024,
                             max_seq=64, max_d_model=64, max_ffn=64, max_qkv=64))
    try:
        prev, cur, _ = fcdata.sel_pairs(1)
        prev2, cur2, _ = fcdata.sel_pairs(2)
        fp, fcur = torch.from_numpy(prev).cuda(), torch.from_numpy(cur).cuda()
        gp, gcur = torch.from_numpy(prev2).cuda(), torch.from_numpy(cur2).cuda()
        prm = fc.SelectParams()
        out = fc.SelectOut.alloc(B, 1024)
        keys = ("sim", "energy", "reuse_mask", "recompute_idx", "n_recompute", "shift", "scalars",
                "counts", "flags")

        def snap():
            torch.cuda.synchronize()
            return {k: getattr(out, k).cpu().numpy().copy() for k in keys}

        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            fc.fc_select(ctx, prm, fp, fcur, out)
        torch.cuda.current_stream().wait_stream(side)
        want = snap()
        with torch.cuda.stream(side):
            fc.fc_select(ctx, prm, gp, gcur, out)
        torch.cuda.current_stream().wait_stream(side)
        other = snap()
        assert not np.array_equal(other["reuse_mask"], want["reuse_mask"])
        graph = torch.cuda.CUDAGraph()
        torch.cuda.synchronize()
        with torch.cuda.graph(graph):
            fc.fc_select(ctx, prm, fp, fcur, out)
        for rep in range(3):
            fc.fc_select(ctx, prm, gp, gcur, out)            # eager, other frames
            got = snap()
            for k in keys:
                np.testing.assert_array_equal(got[k], other[k], err_msg=f"eager {k}, round {rep}")
            graph.replay()
            got = snap()
            for k in keys:
                np.testing.assert_array_equal(got[k], want[k], err_msg=f"replay {k}, round {rep}")
    finally:
        ctx.close()
