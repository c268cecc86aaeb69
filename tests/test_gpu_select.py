"""GPU parity of fc_select against the float64 oracle (called through the C ABI).

Masks, ids, shifts and counts must match bit for bit (an exception is allowed
only where the oracle's own decision margin is below 1e-5, and the GPU result
must then still be a valid selection); similarities, energies and scalars
within 1e-5 relative.
"""
import numpy as np
import pytest
import torch

import fcdata
from oracle import select as osel
from tests import fcutil

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def fc():
    import paper_2604_24391_amd as fc
    return fc


@pytest.fixture(scope="module")
def ctx(fc):
    c = fc.Context(fc.Caps(max_batch=64, max_height=448, max_width=448, max_tokens=1024,
                           max_seq=64, max_d_model=64, max_ffn=64, max_qkv=64))
    yield c
    c.close()


def run_select(fc, ctx, prm, prev, cur):
    B, _, H, W = cur.shape
    gh, gw = fc.token_grid(H, W, prm)
    out = fc.SelectOut.alloc(B, gh * gw)
    p = None if prev is None else torch.from_numpy(np.ascontiguousarray(prev)).cuda()
    c = torch.from_numpy(np.ascontiguousarray(cur)).cuda()
    fc.fc_select(ctx, prm, p, c, out)
    torch.cuda.synchronize()
    return fcutil.select_out_np(out)


def compare(fc, ctx, prm, prev, cur, items=None):
    o = run_select(fc, ctx, prm, prev, cur)
    op = fcutil.oracle_select_params(prm)
    items = range(cur.shape[0]) if items is None else items
    margins = []
    for b in items:
        res = osel.select_item(None if prev is None else prev[b], cur[b], op)
        mg, esc = fcutil.check_select(o, res, op, b)
        assert not esc
        margins.append(mg)
    return o, margins


def test_tiny_pair_fixed_budget(fc, ctx):
    """224x224 pair, 256 patches, fixed 50 % budget (K_reuse = 128)."""
    prev, cur, _ = fcdata.tiny_pair(0)
    prm = fc.SelectParams(adaptive=False, alpha_fixed=0.5)
    o, _ = compare(fc, ctx, prm, prev, cur)
    assert int(o["counts"][0][0]) == 128


def test_tiny_pair_adaptive(fc, ctx):
    prev, cur, _ = fcdata.tiny_pair(3)
    compare(fc, ctx, fc.SelectParams(), prev, cur)


def test_selection_at_scale_all_pairs(fc, ctx):
    """64 pairs at 448x448 (1024 patches each), adaptive budget: the launch the
    benchmark times; every pair is checked against the oracle, with no tolerated
    mismatch."""
    prev, cur, _ = fcdata.sel_pairs(1)
    o, margins = compare(fc, ctx, fc.SelectParams(), prev, cur)
    print("min top-K margin", min(m["topk"] for m in margins),
          "min shift margin", min(m["shift"] for m in margins))


def test_odd_batch_with_and_without_previous_frames(fc, ctx):
    """19 pairs at 448x448 (an odd batch, not a power of two), every pair against the
    oracle; then the same current frames with the previous frames missing (all-zero)."""
    prev, cur, _ = fcdata.sel_pairs(17, batch=19)
    compare(fc, ctx, fc.SelectParams(), prev, cur)
    compare(fc, ctx, fc.SelectParams(), None, cur)


def test_budget_clamped_to_candidates(fc, ctx):
    """Algorithm 1 takes K_final = min(K_reuse, |C|): with a 100 % budget on a pair
    rolled by one token (one row and one column unaligned, edge tokens refreshed)
    the budget exceeds the candidates, so every candidate is reused and nothing
    else."""
    rng = np.random.default_rng(21)
    base = fcdata.canvas(rng, 224, 224)[None].astype(np.float32)
    rolled = np.roll(base, (14, 0), (2, 3))
    o, _ = compare(fc, ctx, fc.SelectParams(adaptive=False, alpha_fixed=1.0), base, rolled)
    k_reuse, k_cand, k_final, flushed = (int(x) for x in o["counts"][0])
    assert k_reuse == 256 and k_cand < 256 and k_final == k_cand and not flushed
    flags = o["flags"][0]
    np.testing.assert_array_equal(o["reuse_mask"][0].astype(bool), (flags & 4) != 0)


def test_flush_without_previous_frame(fc, ctx):
    """No previous frame: flushed, K_final = 0, every token recomputed (Sec. 4.1)."""
    _, cur, _ = fcdata.tiny_pair(5)
    o, _ = compare(fc, ctx, fc.SelectParams(), None, cur)
    assert int(o["counts"][0][3]) == 1 and int(o["n_recompute"][0]) == 256
    np.testing.assert_array_equal(o["recompute_idx"][0], np.arange(256))


def test_zero_previous_frame_flushes(fc, ctx):
    prev, cur, _ = fcdata.tiny_pair(6)
    o, _ = compare(fc, ctx, fc.SelectParams(), np.zeros_like(prev), cur)
    assert int(o["counts"][0][3]) == 1


def test_identical_and_rolled_frames(fc, ctx):
    """Identical frames: Delta = 0, all aligned, similarity 1.  Frames rolled by one
    token: Delta = -1 on both axes, first row and column unaligned."""
    rng = np.random.default_rng(7)
    fr = rng.uniform(size=(1, 3, 224, 224)).astype(np.float32)
    o, _ = compare(fc, ctx, fc.SelectParams(), fr, fr)
    assert tuple(o["shift"][0]) == (0, 0)
    np.testing.assert_allclose(o["sim"][0], 1.0, atol=1e-6)
    rolled = np.roll(fr, (14, 14), (2, 3))
    o, _ = compare(fc, ctx, fc.SelectParams(), fr, rolled)
    assert tuple(o["shift"][0]) == (-1, -1)


def test_flat_frames_tie_to_lowest_ids(fc, ctx):
    """Flat content has energy exactly 0 on both sides, so the ascending top-K takes
    the lowest token ids (ties broken by id)."""
    fr = np.full((1, 3, 224, 224), 0.4, np.float32)
    fr[:, :, 100:, 150:] = 0.9
    o, _ = compare(fc, ctx, fc.SelectParams(adaptive=False, alpha_fixed=0.25), fr, fr)
    assert int(o["counts"][0][2]) == 64


def test_merge2_episode_frames(fc, ctx):
    """448x448 camera frames with 2x2 token merge (256 tokens), consecutive steps."""
    fr = fcdata.episode_frames(11, n_frames=4)
    prm = fc.SelectParams(merge=2)
    compare(fc, ctx, prm, fr[:3], fr[1:4])


@pytest.mark.parametrize("ablation", [dict(align=False), dict(refresh=False),
                                      dict(align=False, refresh=False, tau_sim=0.9),
                                      dict(adaptive=False, alpha_fixed=0.3)])
def test_module_ablations(fc, ctx, ablation):
    """The module ablations of Table 3 (Sec. 6.3) on camera frames (2x2 merge) and on
    a rolled pair: without alignment the shift is (0, 0) and every token aligned;
    without refresh no token is fresh; the fixed 30 % budget."""
    fr = fcdata.episode_frames(12, n_frames=3)
    prm = fc.SelectParams(merge=2, **ablation)
    o, _ = compare(fc, ctx, prm, fr[:2], fr[1:3])
    rng = np.random.default_rng(13)
    base = rng.uniform(size=(1, 3, 224, 224)).astype(np.float32)
    o2, _ = compare(fc, ctx, fc.SelectParams(**ablation), base, np.roll(base, (14, 28), (2, 3)))
    if not ablation.get("align", True):
        assert (o["shift"] == 0).all() and (o2["shift"] == 0).all()
    else:
        assert tuple(o2["shift"][0]) == (-1, -2)


@pytest.mark.parametrize("hw", [(154, 154), (168, 252), (196, 112), (42, 70)])
def test_ragged_frame_sizes(fc, ctx, hw):
    """Patch rows that do not fill a 16-patch workgroup and widths that are not a
    multiple of 4 floats (scalar load path)."""
    h, w = hw
    rng = np.random.default_rng(h * 1000 + w)
    cv = fcdata.canvas(rng, h + 16, w + 16)
    prev = cv[None, :, 8:8 + h, 8:8 + w].astype(np.float32)
    cur = np.clip(cv[None, :, 5:5 + h, 10:10 + w] + rng.normal(0, 0.01, (1, 3, h, w)), 0, 1)
    compare(fc, ctx, fc.SelectParams(), prev, cur.astype(np.float32))


def test_batch_items_are_independent(fc, ctx):
    """Item b of a batch equals the same pair run alone."""
    prev, cur, _ = fcdata.sel_pairs(9, batch=3, size=224)
    prm = fc.SelectParams()
    ob = run_select(fc, ctx, prm, prev, cur)
    for b in range(3):
        o1 = run_select(fc, ctx, prm, prev[b:b + 1], cur[b:b + 1])
        for k in ("sim", "energy", "reuse_mask", "recompute_idx", "shift", "scalars", "counts"):
            np.testing.assert_array_equal(ob[k][b], o1[k][0], err_msg=k)


def test_two_contexts_on_two_streams(fc, ctx):
    """Independent batches on two streams, each with its own context, overlapping in
    time: both give exactly the single-stream outputs."""
    prev, cur, _ = fcdata.sel_pairs(1)
    p, c = torch.from_numpy(prev).cuda(), torch.from_numpy(cur).cuda()
    prm = fc.SelectParams()
    ref = fc.SelectOut.alloc(64, 1024)
    fc.fc_select(ctx, prm, p, c, ref)
    torch.cuda.synchronize()
    ref_np = fcutil.select_out_np(ref)
    ctx2 = fc.Context(fc.Caps(max_batch=64, max_height=448, max_width=448, max_tokens=1024,
                              max_seq=64, max_d_model=64, max_ffn=64, max_qkv=64))
    outs = [fc.SelectOut.alloc(64, 1024), fc.SelectOut.alloc(64, 1024)]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    for s_ in streams:
        s_.wait_stream(torch.cuda.current_stream())
    for i in range(6):
        fc.fc_select((ctx, ctx2)[i % 2], prm, p, c, outs[i % 2], stream=streams[i % 2])
    torch.cuda.synchronize()
    ctx2.close()
    for o in outs:
        on = fcutil.select_out_np(o)
        for k, v in ref_np.items():
            if v is not None:
                np.testing.assert_array_equal(on[k], v, err_msg=k)


def test_deterministic(fc, ctx):
    """Two runs on the same inputs are byte-identical."""
    prev, cur, _ = fcdata.sel_pairs(4, batch=8)
    prm = fc.SelectParams()
    a = run_select(fc, ctx, prm, prev, cur)
    b = run_select(fc, ctx, prm, prev, cur)
    for k, v in a.items():
        np.testing.assert_array_equal(v, b[k], err_msg=k)


def test_boundary_errors(fc, ctx):
    """Shape and capacity errors come back as status codes and launch nothing."""
    prm = fc.SelectParams()
    out = fc.SelectOut.alloc(1, 256)
    bad = torch.zeros(1, 3, 100, 224, device="cuda")
    with pytest.raises(fc.FcError) as e:
        fc.fc_select(ctx, prm, None, bad, out)
    assert e.value.status == 2
    big = torch.zeros(1, 3, 896, 896, device="cuda")
    with pytest.raises(fc.FcError) as e:
        fc.fc_select(ctx, prm, None, big, fc.SelectOut.alloc(1, 4096))
    assert e.value.status in (3, 6)
    with pytest.raises(fc.FcError) as e:
        fc.fc_select(ctx, fc.SelectParams(patch=16), None, torch.zeros(1, 3, 224, 224, device="cuda"), out)
    assert e.value.status == 6


def test_batched_episode_frames_896(fc):
    """The batched-episode shape: 896x896 frames, 4096 patches, 2x2 merge -> 1024 tokens
    on a 32x32 grid, two independent trajectories (each over its own texture) in one
    call, consecutive steps."""
    c = fc.Context(fc.Caps(max_batch=2, max_height=896, max_width=896, max_tokens=1024,
                           max_seq=64, max_d_model=64, max_ffn=64, max_qkv=64))
    try:
        eps = [fcdata.episode_frames(5000 + e, size=896, n_frames=2) for e in range(2)]
        prev = np.stack([e[0] for e in eps])
        cur = np.stack([e[1] for e in eps])
        o, margins = compare(fc, c, fc.SelectParams(merge=2), prev, cur)
        assert o["n_recompute"].shape == (2,)
        print(f"n_recompute {o['n_recompute'].tolist()}, min top-K margin "
              f"{min(m['topk'] for m in margins):.2e}")
    finally:
        c.close()


@pytest.mark.parametrize("case", ["episode_merge2", "pairs_448"])
def test_naive_selector(fc, ctx, case):
    """The naive frequency baseline of Sec. 6.1 (position-wise amplitude similarity,
    static reuse at a fixed threshold), run as fc_select with alignment, refresh, the
    adaptive budget and the gate switched off, against the oracle's direct
    formulation of it: reuse masks and recompute ids bit-exact, similarities within
    1e-5, no token within 1e-5 of the threshold on these seeds."""
    if case == "episode_merge2":
        fr = fcdata.episode_frames(2024, size=448, n_frames=5)
        prev, cur, m = fr[:4], fr[1:5], 2
    else:
        prev, cur, _ = fcdata.sel_pairs(1, batch=4)
        m = 1
    # thresholds chosen so that no similarity of these seeds lies within 1e-4 of them
    # (position-wise similarities crowd just below 1 on these frames)
    for tau in (0.94, 0.9675):
        prm = fc.SelectParams.naive(tau, merge=m)
        o = run_select(fc, ctx, prm, prev, cur)
        for b in range(cur.shape[0]):
            res = osel.naive_select(prev[b], cur[b], 14, m, tau)
            near = np.abs(res.sim - tau) < fcutil.MARGIN * tau
            assert not near.any(), f"tokens within 1e-5 of tau: {np.flatnonzero(near)}"
            fcutil._close(o["sim"][b], res.sim, "sim")
            np.testing.assert_array_equal(o["reuse_mask"][b], res.reuse_mask)
            n = res.n_recompute
            assert int(o["n_recompute"][b]) == n
            np.testing.assert_array_equal(o["recompute_idx"][b][:n], res.recompute_idx)
            assert tuple(o["shift"][b]) == (0, 0) and int(o["counts"][b][3]) == 0
            assert int(o["counts"][b][2]) == int(res.reuse_mask.sum())


def test_carried_spectra_match_pixels(fc, ctx):
    """fc_select_carry along two trajectories at once (448x448, 2x2 merge): the first
    step without a previous state is flushed, and every step's outputs are byte for
    byte those of fc_select on both frames' pixels; two steps are also checked against
    the oracle."""
    eps = [fcdata.episode_frames(40 + e, size=448, n_frames=5) for e in range(2)]
    fr = torch.from_numpy(np.ascontiguousarray(np.stack(eps, axis=1))).cuda()   # [5, 2, 3, H, W]
    prm = fc.SelectParams(merge=2)
    op = fcutil.oracle_select_params(prm)
    states = [fc.select_state_alloc(2, 448, 448), fc.select_state_alloc(2, 448, 448)]
    for s in range(5):
        got = fc.SelectOut.alloc(2, 256)
        ref = fc.SelectOut.alloc(2, 256)
        fc.fc_select_carry(ctx, prm, None if s == 0 else states[(s - 1) % 2], fr[s], states[s % 2],
                           got)
        fc.fc_select(ctx, prm, None if s == 0 else fr[s - 1], fr[s], ref)
        torch.cuda.synchronize()
        g, r = fcutil.select_out_np(got), fcutil.select_out_np(ref)
        for k, v in r.items():
            np.testing.assert_array_equal(g[k], v, err_msg=f"step {s}: {k}")
        if s == 0:
            assert (g["counts"][:, 3] == 1).all()
        if s in (1, 4):
            for b in range(2):
                res = osel.select_item(eps[b][s - 1], eps[b][s], op)
                mg, esc = fcutil.check_select(g, res, op, b)
                assert not esc
