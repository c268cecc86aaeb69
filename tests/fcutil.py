"""Shared helpers for the GPU parity tests: tensor conversion, the selection
comparison with its decision-margin audit, and layer comparisons."""
from __future__ import annotations

import numpy as np
import torch

import fcdata
from oracle import select as osel

# Tolerances (fixed by the benchmark spec of the hot path): fp32 scores within
# 1e-5 relative (plus an absolute floor of 1e-6 of the largest value, which only
# matters for values rounded to 0); bf16 layer outputs within 2e-2 relative L2
# of the fp32 oracle; decisions bit-exact unless the oracle's own margin is
# below 1e-5 (then the GPU result must still be a valid selection).
SCORE_RTOL, SCORE_ATOL_FRAC = 1e-5, 1e-6
LAYER_RTOL = 2e-2
MARGIN = 1e-5


def bf16_gpu(u16: np.ndarray, device="cuda") -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(u16).view(np.int16).copy()).view(
        torch.bfloat16).to(device)


def bf16_np(t: torch.Tensor) -> np.ndarray:
    return t.detach().contiguous().cpu().view(torch.int16).numpy().view(np.uint16)


def weights_gpu(wt: dict) -> dict:
    return {k: bf16_gpu(v) for k, v in wt.items()}


def layer_desc(shape: fcdata.LayerShape, wgpu: dict):
    import paper_2604_24391_amd as fc
    return fc.LayerDesc(shape.d, shape.n_heads, shape.n_kv, shape.hd, shape.ffn, wgpu,
                        rms_eps=shape.eps, rope_theta=shape.theta)


def rel_l2(a, b) -> float:
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def select_out_np(out) -> dict:
    return {k: (getattr(out, k).cpu().numpy() if getattr(out, k) is not None else None)
            for k in ("sim", "energy", "reuse_mask", "recompute_idx", "n_recompute", "shift",
                      "scalars", "counts", "flags")}


def _close(g, o, name):
    g = np.asarray(g, np.float64)
    o = np.asarray(o, np.float64)
    tol = SCORE_RTOL * np.abs(o) + SCORE_ATOL_FRAC * max(np.abs(o).max(), 1e-300)
    bad = np.abs(g - o) > tol
    assert not bad.any(), (f"{name}: {int(bad.sum())} values outside tolerance; worst "
                           f"|d|={np.abs(g - o).max():.3e} at {np.flatnonzero(bad)[:5]}")


def check_valid_selection(o: dict, b: int, N: int):
    """The GPU selection is a valid Algorithm-1 outcome of its own masks and keys."""
    flags = o["flags"][b]
    cand = (flags & 4) != 0
    reuse = o["reuse_mask"][b].astype(bool)
    k_reuse, k_cand, k_final, flushed = (int(x) for x in o["counts"][b])
    assert k_cand == int(cand.sum())
    assert not (reuse & ~cand).any(), "reused a non-candidate"
    assert int(reuse.sum()) == k_final == (0 if flushed else min(k_reuse, k_cand))
    e = o["energy"][b]
    if reuse.any() and (cand & ~reuse).any():
        worst_in = max((e[t], t) for t in np.flatnonzero(reuse))
        best_out = min((e[t], t) for t in np.flatnonzero(cand & ~reuse))
        assert worst_in < best_out, "reused set is not the ascending-energy top-K"
    n = int(o["n_recompute"][b])
    assert n == N - k_final
    ids = o["recompute_idx"][b][:n]
    np.testing.assert_array_equal(ids, np.flatnonzero(~reuse))


class Escapes(list):
    """Names of the decisions where the GPU and the oracle differ but the oracle's own
    margin is below MARGIN (the only mismatches the comparison can tolerate)."""


def check_select(o: dict, res: osel.SelectResult, prm: osel.SelectParams, b: int,
                 allow_escapes: bool = False):
    """Compare item b of the GPU outputs with the oracle; returns (margins, escapes).

    Scores must be within tolerance.  Every decision must agree bit for bit.  A
    mismatch is an "escape" only where the oracle's own margin for that decision is
    below MARGIN; any other mismatch fails at once.  Escapes also fail unless
    `allow_escapes` (no committed seed needs that: a seed that did would be marked
    xfail with the margin as its reason).  Decisions downstream of an escaped one are
    still compared wherever they do not depend on it."""
    N = res.energy.size
    esc = Escapes()
    check_valid_selection(o, b, N)
    _close(o["energy"][b], res.energy, "energy")
    _close(o["sim"][b], res.sim, "sim")
    sc = o["scalars"][b]
    want = [res.sim_freq, res.psi, res.alpha, res.mu, res.sigma, res.thr]
    for name, g, w in zip(("sim_freq", "psi", "alpha", "mu", "sigma", "thr"), sc, want):
        assert abs(g - w) <= SCORE_RTOL * abs(w) + 1e-12, f"{name}: gpu {g!r} oracle {w!r}"
    mg = osel.decision_margins(res, prm)
    k_reuse, k_cand, k_final, flushed = (int(x) for x in o["counts"][b])
    flags = o["flags"][b]

    def finish():
        assert allow_escapes or not esc, f"item {b}: tolerated mismatches {list(esc)}"
        return mg, esc

    # shift (argmax of Eq. 4-1): every alignment-dependent decision follows from it
    if tuple(o["shift"][b]) != res.shift:
        assert mg["shift"] < MARGIN, f"shift {tuple(o['shift'][b])} vs {res.shift}, margin {mg['shift']}"
        esc.append(f"shift (margin {mg['shift']:.2e})")
        return finish()
    np.testing.assert_array_equal((flags & 1) != 0, res.aligned, err_msg="Mask_align")
    # refresh (Eq. 4-3): token by token
    fresh = (flags & 2) != 0
    bad_f = np.flatnonzero(fresh != res.fresh)
    assert all(mg["threshold"][t] < MARGIN for t in bad_f), \
        f"refresh decisions differ at {bad_f[:8]} with margins {mg['threshold'][bad_f[:8]]}"
    if bad_f.size:
        esc.append(f"threshold at {bad_f[:8].tolist()}")
    # candidates: may differ only where the refresh or the similarity floor escaped
    cand = (flags & 4) != 0
    bad_c = np.flatnonzero(cand != res.cand)
    bad_s = np.setdiff1d(bad_c, bad_f)
    assert all(mg["tau_sim"][t] < MARGIN for t in bad_s), \
        f"candidates differ at {bad_s[:8]} with similarity-floor margins {mg['tau_sim'][bad_s[:8]]}"
    if bad_s.size:
        esc.append(f"tau_sim at {bad_s[:8].tolist()}")
    if bad_c.size == 0:
        assert k_cand == res.k_cand
    # gate and budget (scalars decided from fp64 sums)
    if bool(flushed) != res.flushed:
        assert mg["gate"] < MARGIN, f"flush decision differs, margin {mg['gate']}"
        esc.append(f"gate (margin {mg['gate']:.2e})")
        return finish()
    if k_reuse != res.k_reuse:
        assert mg["budget"] < MARGIN, f"K_reuse {k_reuse} vs {res.k_reuse}, margin {mg['budget']}"
        esc.append(f"budget (margin {mg['budget']:.2e})")
        return finish()
    if bad_c.size:
        return finish()
    # the ascending top-K and the compaction
    assert k_final == res.k_final
    diff = np.flatnonzero(o["reuse_mask"][b] != res.reuse_mask)
    if diff.size:
        assert mg["topk"] < MARGIN, f"reuse masks differ at {diff[:8]} (top-K margin {mg['topk']})"
        esc.append(f"topk (margin {mg['topk']:.2e})")
        return finish()
    n = res.n_recompute
    assert int(o["n_recompute"][b]) == n
    np.testing.assert_array_equal(o["recompute_idx"][b][:n], res.recompute_idx)
    return finish()


def oracle_select_params(prm) -> osel.SelectParams:
    return osel.SelectParams(patch=prm.patch, merge=prm.merge, tau_mig=prm.tau_mig, lam=prm.lam,
                             alpha_min=prm.alpha_min, alpha_max=prm.alpha_max,
                             adaptive=prm.adaptive, alpha_fixed=prm.alpha_fixed,
                             entropy_norm=prm.entropy_norm, tau_sim=prm.tau_sim,
                             align=prm.align, refresh=prm.refresh,
                             align_pixel=prm.align_pixel, align_rotation=prm.align_rotation)
