"""Pins of the selection oracle against things other than itself.

Each test pins one part of oracle/select.py to a library routine, a closed form,
an invariant the paper states, or brute force on tiny inputs, chosen so that a
plausible slip (a transposed matrix, a sign, a dropped term, a wrong estimator,
the wrong sort direction) fails at least one of them.
"""
import itertools
import json
import os

import numpy as np
import pytest
import scipy.fft

from oracle import select as osel

GOLD = os.path.join(os.path.dirname(__file__), "golden", "paper_constants.json")
RNG = np.random.default_rng(1234)


def _rel(a, b):
    return np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300)


# ------------------------------------------------------------------ paper constants
def test_defaults_are_the_papers_hyperparameters():
    """SelectParams defaults equal the values printed in Sec. 6.4 (golden fixture)."""
    g = json.load(open(GOLD))
    hp = g["hyperparameters"]
    p = osel.SelectParams()
    assert (p.tau_mig, p.lam, p.alpha_max, p.alpha_min) == \
        (hp["tau_mig"], hp["lambda"], hp["alpha_max"], hp["alpha_min"])
    hc = g["high_pass_cutoff"]
    h = osel.high_pass(hc["patch"])
    assert int((h == 0).sum()) == hc["zeroed_coefficients"]
    assert np.all(h[:hc["cutoff"], :hc["cutoff"]] == 0)
    assert h[hc["cutoff"], 0] == 1 and h[0, hc["cutoff"]] == 1


def test_high_pass_small_patches():
    """Eq. 3-4 cutoff c = max(1, floor(P/4)): P = 2, 3 keep c = 1 (only DC removed)."""
    for p, c in [(2, 1), (3, 1), (4, 1), (8, 2), (14, 3), (16, 4)]:
        h = osel.high_pass(p)
        assert int((h == 0).sum()) == c * c


# ------------------------------------------------------------------ PIN-1 DFT
@pytest.mark.parametrize("shape", [(14, 14), (16, 16), (8, 32), (7, 5)])
def test_dft2_matches_numpy_fft(shape):
    """PIN-1: the matrix DFT equals np.fft.fft2 and its inverse np.fft.ifft2."""
    x = RNG.standard_normal(shape)
    assert _rel(osel.dft2(x), np.fft.fft2(x)) < 1e-12
    z = RNG.standard_normal(shape) + 1j * RNG.standard_normal(shape)
    assert _rel(osel.idft2(z), np.fft.ifft2(z)) < 1e-12


def test_patch_amplitude_axes_are_not_transposed():
    """A horizontal cosine (varying along x) puts its energy at v, not at u."""
    x = np.arange(14)
    pt = np.tile(np.cos(2 * np.pi * 3 * x / 14), (14, 1))  # varies along x only
    a = osel.patch_amplitude(pt)
    assert a[0, 3] == pytest.approx(98.0) and a[0, 11] == pytest.approx(98.0)
    assert a[3, 0] < 1e-9


# ------------------------------------------------------------------ PIN-2 shift invariance
def test_amplitude_is_circular_shift_invariant():
    """PIN-2 (Fourier shift theorem, Sec. 2.3 / 3.1): a circular shift of a patch
    leaves its amplitude spectrum unchanged, so the token similarity is 1."""
    pt = RNG.uniform(size=(14, 14))
    a0 = osel.patch_amplitude(pt)
    for dy, dx in [(0, 1), (3, 0), (5, 9), (13, 13)]:
        a1 = osel.patch_amplitude(np.roll(pt, (dy, dx), axis=(0, 1)))
        assert _rel(a1, a0) < 1e-12
    aligned = np.ones((1, 1), bool)
    sim = osel.token_similarity(a0.reshape(1, 1, -1),
                                osel.patch_amplitude(np.roll(pt, (2, 7), (0, 1))).reshape(1, 1, -1),
                                0, 0, aligned)
    assert sim[0, 0] == pytest.approx(1.0, abs=1e-14)


# ------------------------------------------------------------------ PIN-3 constant patch
def test_constant_patch_has_only_dc():
    """PIN-3: a constant patch c has X(0,0) = P^2 c and every other bin 0; its
    high-pass energy is 0 (Sec. 3.2: smooth content sits in the DC term)."""
    c = 0.37
    pt = np.full((14, 14), c)
    a = osel.patch_amplitude(pt)
    assert a[0, 0] == pytest.approx(196 * c, rel=1e-14)
    a[0, 0] = 0
    assert a.max() < 1e-12
    assert osel.patch_energy(pt) < 1e-26


# ------------------------------------------------------------------ PIN-4 Parseval
def test_parseval_dft_and_two_routes_to_energy():
    """PIN-4: sum |X|^2 = P^2 sum p^2 (unnormalised DFT), and with the orthonormal DCT
    E = sum p^2 - sum_{u,v<3} D^2, D taken from scipy's DCT (an independent route)."""
    pt = RNG.uniform(size=(5, 14, 14))
    a = osel.patch_amplitude(pt)
    np.testing.assert_allclose((a ** 2).sum(axis=(1, 2)), 196 * (pt ** 2).sum(axis=(1, 2)),
                               rtol=1e-12)
    d = scipy.fft.dctn(pt, type=2, norm="ortho", axes=(1, 2))
    e2 = (pt ** 2).sum(axis=(1, 2)) - (d[:, :3, :3] ** 2).sum(axis=(1, 2))
    np.testing.assert_allclose(osel.patch_energy(pt), e2, rtol=1e-10)


# ------------------------------------------------------------------ PIN-5 DCT
def test_dct_matrix_matches_scipy_and_basis_images():
    """PIN-5: the DCT-II matrix equals scipy.fft.dctn(type=2, norm='ortho'); a DCT basis
    image inside the removed 3x3 block has E = 0, outside it E = amplitude^2."""
    pt = RNG.standard_normal((14, 14))
    c = osel.dct_matrix(14)
    assert _rel(c @ pt @ c.T, scipy.fft.dctn(pt, type=2, norm="ortho")) < 1e-12
    for (u, v) in [(0, 0), (2, 2), (1, 2), (3, 0), (0, 3), (7, 11), (13, 13)]:
        coef = np.zeros((14, 14))
        coef[u, v] = 0.8
        img = scipy.fft.idctn(coef, type=2, norm="ortho")
        e = osel.patch_energy(img)
        if u < 3 and v < 3:
            assert e < 1e-25
        else:
            assert e == pytest.approx(0.64, rel=1e-12)


# ------------------------------------------------------------------ PIN-6 Hermitian half
def test_hermitian_half_spectrum_cosine():
    """PIN-6: for real patches the amplitude is symmetric, A(u,v) = A(-u,-v), so the
    196-bin cosine equals a weighted cosine over the 100 unique bins."""
    p0, p1 = RNG.uniform(size=(2, 14, 14))
    a0, a1 = osel.patch_amplitude(p0), osel.patch_amplitude(p1)
    np.testing.assert_allclose(a0, np.roll(a0[::-1, ::-1], (1, 1), (0, 1)), rtol=1e-12)
    w = np.zeros((14, 14))
    w[:, 1:7] = 2
    w[[0, 7], 0] = 1
    w[1:7, 0] = 2
    w[[0, 7], 7] = 1
    w[1:7, 7] = 2
    assert int((w > 0).sum()) == 100 and w.sum() == 196
    half = (w * a0 * a1).sum() / np.sqrt((w * a0 * a0).sum() * (w * a1 * a1).sum())
    full = osel.token_similarity(a0.reshape(1, 1, -1), a1.reshape(1, 1, -1), 0, 0,
                                 np.ones((1, 1), bool))[0, 0]
    assert half == pytest.approx(full, rel=1e-13)


# ------------------------------------------------------------------ PIN-7 global similarity / gate
def test_global_similarity_special_cases():
    """PIN-7: Sim_freq = 1 for identical grids and for a circularly rolled grid, and
    0 against an all-zero grid; Sim < tau_mig flushes (Sec. 4.1, strict <)."""
    g = RNG.uniform(size=(16, 16))
    f = osel.dft2(g)
    assert osel.global_similarity(f, f) == pytest.approx(1.0, abs=1e-14)
    assert osel.global_similarity(osel.dft2(np.roll(g, (3, -5), (0, 1))), f) == \
        pytest.approx(1.0, abs=1e-13)
    assert osel.global_similarity(f, osel.dft2(np.zeros_like(g))) == 0.0
    frame = np.stack([np.tile(g.repeat(14, 0).repeat(14, 1), 1)] * 3)
    r = osel.select_item(np.zeros_like(frame), frame, osel.SelectParams())
    assert r.flushed and r.sim_freq == 0.0 and r.k_final == 0 and r.n_recompute == 256


# ------------------------------------------------------------------ PIN-8 phase correlation
def _direct_response(fp, fc):
    """Brute-force O(G^4) inverse transform of the normalised cross-power spectrum."""
    gh, gw = fp.shape
    x = fp * np.conj(fc)
    mag = np.abs(x)
    c = np.where(mag > 1e-9 * mag.max(), x / np.where(mag > 0, mag, 1), 0)
    r = np.zeros((gh, gw))
    for i in range(gh):
        for j in range(gw):
            acc = 0j
            for u in range(gh):
                for v in range(gw):
                    acc += c[u, v] * np.exp(2j * np.pi * (u * i / gh + v * j / gw))
            r[i, j] = acc.real / (gh * gw)
    return r


def test_phase_correlation_recovers_every_roll_small_grid():
    """PIN-8: g_t = roll(g_{t-1}, d) gives Delta = -d for every d in the signed range
    (exhaustive on an 8x8 grid), and the response equals the brute-force inverse."""
    g = RNG.uniform(size=(8, 8))
    fp = osel.dft2(g)
    for dy in range(-3, 5):
        for dx in range(-3, 5):
            fc = osel.dft2(np.roll(g, (dy, dx), (0, 1)))
            (di, dj), resp = osel.phase_correlation(fp, fc)
            wy, wx = (-dy) % 8, (-dx) % 8
            wy, wx = (wy if wy <= 4 else wy - 8), (wx if wx <= 4 else wx - 8)
            assert (di, dj) == (wy, wx)
            if (dy, dx) in [(0, 0), (1, -2), (4, 3)]:
                np.testing.assert_allclose(resp, _direct_response(fp, fc), atol=1e-12)
                assert resp.max() == pytest.approx(1.0, abs=1e-12)


def test_phase_correlation_half_grid_wrap_stays_positive():
    """Signed wrap: an index of exactly G/2 maps to +G/2."""
    g = RNG.uniform(size=(8, 16))
    (di, dj), _ = osel.phase_correlation(osel.dft2(g), osel.dft2(np.roll(g, (4, 8), (0, 1))))
    assert (di, dj) == (4, 8)


def test_frames_rolled_by_whole_tokens_give_the_shift():
    """PIN-8 (frames): rolling the frame by m*P*d px gives Delta = -d, with m = 1, 2."""
    for m in (1, 2):
        h = 14 * m * 8
        fr = RNG.uniform(size=(3, h, h))
        for d in [(1, 0), (0, -2), (-1, 3)]:
            cur = np.roll(fr, (14 * m * d[0], 14 * m * d[1]), (1, 2))
            r = osel.select_item(fr, cur, osel.SelectParams(merge=m))
            assert r.shift == (-d[0], -d[1])


# ------------------------------------------------------------------ PIN-9 entropy / budget
def test_entropy_and_budget_closed_forms():
    """PIN-9: a constant grid has Psi = 0 so alpha = alpha_max; an impulse grid has a
    flat power spectrum, raw Psi = ln M and normalised Psi = 1, so
    alpha = a_min + (a_max - a_min)/e (Eq. 4-4)."""
    p = osel.SelectParams()
    assert osel.spectral_entropy(osel.dft2(np.full((16, 16), 0.4)), True) == \
        pytest.approx(0.0, abs=1e-12)
    imp = np.zeros((16, 16))
    imp[5, 9] = 1.0
    f = osel.dft2(imp)
    assert osel.spectral_entropy(f, False) == pytest.approx(np.log(256), rel=1e-12)
    assert osel.spectral_entropy(f, True) == pytest.approx(1.0, rel=1e-12)
    a, k = osel.reuse_budget(1.0, 256, p)
    assert a == pytest.approx(0.08 + 0.42 / np.e, rel=1e-14)
    assert k == int(np.floor(256 * (0.08 + 0.42 / np.e))) == 60
    a0, k0 = osel.reuse_budget(0.0, 256, p)
    assert a0 == pytest.approx(0.5) and k0 == 128
    af, kf = osel.reuse_budget(0.7, 1000, osel.SelectParams(adaptive=False, alpha_fixed=0.3))
    assert (af, kf) == (0.3, 300)
    assert osel.spectral_entropy(np.zeros((4, 4)), True) == 0.0


def test_entropy_grows_with_detail():
    """Sec. 3.3: detail-rich scenes spread power into high bands -> higher entropy,
    hence a smaller reuse budget."""
    y, x = np.mgrid[0:32, 0:32]
    smooth = np.exp(-((y - 16) ** 2 + (x - 16) ** 2) / 200.0)
    detail = smooth + 0.3 * np.cos(2 * np.pi * 7 * x / 32) * np.cos(2 * np.pi * 5 * y / 32)
    noisy = detail + 0.3 * RNG.standard_normal((32, 32))
    ents = [osel.spectral_entropy(osel.dft2(g), True) for g in (smooth, detail, noisy)]
    assert ents[0] < ents[1] < ents[2]
    p = osel.SelectParams()
    ks = [osel.reuse_budget(e, 1024, p)[1] for e in ents]
    assert ks[0] > ks[1] > ks[2]


# ------------------------------------------------------------------ PIN-10 refresh rule
def test_refresh_mask_closed_form():
    """PIN-10: E = [0,0,0,1]: mu = 0.25, population sigma = sqrt(3)/4, thr = mu + 0.25
    sigma, so only the last token refreshes (Eq. 4-3, strict >).  The unbiased std
    would give sigma = 0.5 and thr = 0.375."""
    fresh, mu, sd, thr = osel.refresh_mask(np.array([0.0, 0.0, 0.0, 1.0]), 0.25)
    assert mu == 0.25 and sd == pytest.approx(np.sqrt(3) / 4, rel=1e-15)
    assert thr == pytest.approx(0.25 + 0.25 * np.sqrt(3) / 4, rel=1e-15)
    assert fresh.tolist() == [False, False, False, True]
    f2, _, s2, t2 = osel.refresh_mask(np.full(6, 0.3), 0.25)
    assert s2 == 0.0 and not f2.any()                 # sigma = 0 -> nothing refreshes


# ------------------------------------------------------------------ PIN-11 exhaustive top-K
def test_topk_exhaustive_small():
    """PIN-11: every key vector over {0,1,2}^N, candidate mask and k for N <= 5: the
    selection has min(k, |C|) members and every selected (key, id) precedes every
    unselected candidate's (key, id) -- the ascending order with ties to the lower id
    of Algorithm 1 / Sec. 4.4."""
    for n in range(1, 6):
        for keys in itertools.product((0.0, 1.0, 2.0), repeat=n):
            key = np.array(keys)
            for cmask in itertools.product((False, True), repeat=n):
                cand = np.array(cmask)
                for k in range(0, n + 2):
                    sel = set(osel.topk_ascending(cand, key, k).tolist())
                    c_ids = set(np.flatnonzero(cand).tolist())
                    assert len(sel) == min(k, len(c_ids)) and sel <= c_ids
                    for s in sel:
                        for u in c_ids - sel:
                            assert (key[s], s) < (key[u], u)


# ------------------------------------------------------------------ PIN-12 end to end
def _smooth_frame(h, w):
    y, x = np.mgrid[0:h, 0:w] / float(h)
    base = 0.5 + 0.3 * np.sin(2 * np.pi * x) * np.cos(2 * np.pi * y)
    return np.stack([base, base * 0.9, base * 0.8])


def test_identical_frames():
    """PIN-12a: identical frames: Delta = 0, every token aligned with similarity 1,
    K_final = min(K_reuse, |C|), reused tokens are the lowest-energy candidates."""
    fr = _smooth_frame(112, 112)
    fr[:, 20:60, 30:70] = 0.9                 # one hard-edged rectangle
    r = osel.select_item(fr, fr, osel.SelectParams())
    assert r.shift == (0, 0) and r.aligned.all() and not r.flushed
    np.testing.assert_allclose(r.sim, 1.0, atol=1e-12)
    assert r.sim_freq == pytest.approx(1.0, abs=1e-14)
    assert r.k_final == min(r.k_reuse, r.k_cand)
    reused = np.flatnonzero(r.reuse_mask)
    rest = np.setdiff1d(np.flatnonzero(r.cand), reused)
    if rest.size and reused.size:
        assert r.energy[reused].max() <= r.energy[rest].min()
    assert r.n_recompute == 64 - r.k_final


def test_missing_previous_frame_flushes():
    """PIN-12b: no previous frame -> flushed, K_final = 0, all N tokens recomputed
    (Sec. 4.1: the cache is flushed and all tokens recomputed)."""
    fr = _smooth_frame(112, 112)
    r = osel.select_item(None, fr, osel.SelectParams())
    assert r.flushed and r.k_final == 0
    assert r.recompute_idx.tolist() == list(range(64))


def test_one_token_roll_unaligns_one_row_and_column():
    """PIN-12c: a frame rolled by one token down and right gives Delta = (-1, -1);
    exactly the first token row and column are unaligned; aligned tokens see their
    exact source patch, so their similarity is 1; unaligned ones are 0 and never
    reused."""
    fr = RNG.uniform(size=(3, 112, 112))
    cur = np.roll(fr, (14, 14), (1, 2))
    r = osel.select_item(fr, cur, osel.SelectParams())
    assert r.shift == (-1, -1)
    al = r.aligned.reshape(8, 8)
    assert not al[0].any() and not al[:, 0].any() and al[1:, 1:].all()
    np.testing.assert_allclose(r.sim.reshape(8, 8)[1:, 1:], 1.0, atol=1e-12)
    assert np.all(r.sim.reshape(8, 8)[0] == 0) and np.all(r.reuse_mask.reshape(8, 8)[0] == 0)


def test_refresh_marks_the_edge_tokens():
    """Sec. 4.2: on a smooth frame with one hard vertical edge, the tokens holding the
    edge have the largest energy and are refreshed; the smooth ones are not."""
    fr = np.full((3, 112, 112), 0.2)
    fr[:, :, 61:] = 0.8                       # edge inside token column 4 (x = 56..69)
    r = osel.select_item(fr, fr, osel.SelectParams())
    fresh = r.fresh.reshape(8, 8)
    assert fresh[:, 4].all() and fresh.sum() == 8
    assert np.all(r.energy.reshape(8, 8)[:, [0, 1, 2, 3, 5, 6, 7]] == 0.0)   # flat -> snapped


def test_merge_token_energy_and_similarity_are_patch_aggregates():
    """With a 2x2 merge a token's energy is the sum of its four patch energies and its
    amplitude vector is the concatenation of theirs (row-major)."""
    fr = RNG.uniform(size=(3, 56, 56))
    r = osel.select_item(fr, fr, osel.SelectParams(merge=2))
    pe = osel.patch_energy(osel.patches(osel.luma(fr), 14))        # [4, 4]
    tok = pe.reshape(2, 2, 2, 2).transpose(0, 2, 1, 3).reshape(2, 2, 4).sum(-1)
    np.testing.assert_allclose(r.energy, tok.ravel(), rtol=1e-14)
    assert r.energy.size == 4


def test_fixed_budget_mode():
    """Ablation 'w/o Module III' (Sec. 6.3): a fixed reuse ratio gives
    K_reuse = floor(alpha_fixed * N) whatever the entropy."""
    fr = RNG.uniform(size=(3, 112, 112))
    r = osel.select_item(fr, fr, osel.SelectParams(adaptive=False, alpha_fixed=0.3))
    assert r.alpha == 0.3 and r.k_reuse == 19


def test_ablation_without_alignment_matches_positions():
    """Ablation 'w/o Module I' (Table 3, Sec. 6.3): position-wise matching.  On a frame
    rolled by one token the full method finds Delta = (-1, -1) and gives the aligned
    tokens similarity 1; without alignment Delta = (0, 0), every token counts as
    aligned, and each token is compared with the previous frame's token at its own
    position, which for a roll of random content is not the same patch (similarity
    below 1).  Identical frames give the same result either way."""
    fr = RNG.uniform(size=(3, 112, 112))
    cur = np.roll(fr, (14, 14), (1, 2))
    full = osel.select_item(fr, cur, osel.SelectParams())
    pos = osel.select_item(fr, cur, osel.SelectParams(align=False))
    assert full.shift == (-1, -1) and pos.shift == (0, 0)
    assert pos.aligned.all()
    assert np.all(pos.sim < 1.0 - 1e-3)
    # the source of token (I, J) without alignment is token (I, J): rolling the previous
    # frame by the same whole tokens makes every position-wise pair identical
    same = osel.select_item(cur, cur, osel.SelectParams(align=False))
    np.testing.assert_allclose(same.sim, 1.0, atol=1e-12)
    ref = osel.select_item(cur, cur, osel.SelectParams())
    np.testing.assert_array_equal(same.reuse_mask, ref.reuse_mask)
    # the global gate, energies and budget do not depend on the alignment
    assert pos.sim_freq == full.sim_freq and pos.k_reuse == full.k_reuse
    np.testing.assert_array_equal(pos.energy, full.energy)


def test_ablation_without_refresh_keeps_edge_tokens_as_candidates():
    """Ablation 'w/o Module II' (Table 3, Sec. 6.3): the edge tokens that the full
    method refreshes become candidates again; mu, sigma and the threshold are still
    reported.  With a budget above the candidate count every token is reused."""
    fr = np.full((3, 112, 112), 0.2)
    fr[:, :, 61:] = 0.8
    prm = dict(adaptive=False, alpha_fixed=1.0)
    full = osel.select_item(fr, fr, osel.SelectParams(**prm))
    nof = osel.select_item(fr, fr, osel.SelectParams(refresh=False, **prm))
    assert full.fresh.sum() == 8 and not nof.fresh.any()
    assert nof.k_cand == full.k_cand + 8 == 64
    assert (nof.mu, nof.sigma, nof.thr) == (full.mu, full.sigma, full.thr)
    assert full.k_final == 56 and nof.k_final == 64 and nof.n_recompute == 0


def test_luma_weights():
    """O1 reading: BT.601 luma, Y = 0.299 R + 0.587 G + 0.114 B (ITU-R BT.601).  Each
    primary alone gives its own weight, so a swap of any two weights fails; white
    and any grey map to their level (the weights sum to 1)."""
    g = np.full((3, 14, 14), 0.25)
    np.testing.assert_allclose(osel.luma(g), 0.25, rtol=1e-15)
    for ch, w in enumerate((0.299, 0.587, 0.114)):
        prim = np.zeros((3, 14, 14))
        prim[ch] = 1.0
        np.testing.assert_allclose(osel.luma(prim), w, rtol=1e-15)
    np.testing.assert_allclose(osel.luma(np.ones((3, 4, 4))), 1.0, rtol=1e-15)
    # a frame that is pure green in one half and pure blue in the other: the half
    # means of the token-grid map carry the two weights
    fr = np.zeros((3, 28, 56))
    fr[1, :, :28] = 1.0
    fr[2, :, 28:] = 1.0
    y = osel.luma(fr)
    assert y[:, :28].mean() == pytest.approx(0.587, abs=1e-15)
    assert y[:, 28:].mean() == pytest.approx(0.114, abs=1e-15)


# ------------------------------------------------------------------ zero-norm similarity
def test_token_similarity_zero_norm_rules():
    """O13 reading R13: two all-zero amplitude vectors are the same content (sim = 1);
    exactly one all-zero vector has nothing in common with the other (sim = 0); an
    unaligned token is 0 whatever its content."""
    a_cur = np.zeros((1, 3, 5))
    a_prev = np.zeros((1, 3, 5))
    a_cur[0, 1] = [1.0, 2.0, 0.0, 0.0, 1.0]       # token 1: current has content, previous none
    a_prev[0, 2] = [0.5, 0.0, 0.0, 3.0, 0.0]      # token 2: previous has content, current none
    sim = osel.token_similarity(a_cur, a_prev, 0, 0, np.ones((1, 3), bool))
    assert sim[0, 0] == 1.0 and sim[0, 1] == 0.0 and sim[0, 2] == 0.0
    sim = osel.token_similarity(a_cur, a_prev, 0, 0, np.array([[False, True, True]]))
    assert sim[0, 0] == 0.0


def test_black_tokens_end_to_end():
    """R13 through select_item: a token that is black in both frames has similarity 1;
    one that turns black has similarity 0 (the other tokens are identical, so the
    shift stays 0 and their similarity is 1)."""
    fr = RNG.uniform(0.2, 1.0, size=(3, 112, 112))
    fr[:, :14, :14] = 0.0                      # token 0 black in both frames
    cur = fr.copy()
    cur[:, 14:28, 28:42] = 0.0                 # token 10 = (1, 2) turns black
    r = osel.select_item(fr, cur, osel.SelectParams())
    assert r.shift == (0, 0)
    assert r.sim[0] == 1.0 and r.sim[10] == 0.0
    others = np.setdiff1d(np.arange(64), [0, 10])
    np.testing.assert_allclose(r.sim[others], 1.0, atol=1e-12)


# ------------------------------------------------------------------ energy snap (R15)
@pytest.mark.parametrize("m", [1, 2])
def test_energy_snap_constant(m):
    """R15: token energies below 1e-8 m^2 snap to exactly 0, larger ones are kept.  A
    patch 0.5 + c B_55 (B_55 the orthonormal DCT basis image (5, 5), outside the
    removed 3x3 block) has E = c^2 exactly: c = 1e-3 (E = 1e-6, a faint texture) must
    survive, c = 3e-5 (E = 9e-10, rounding-noise level) must snap."""
    coef = np.zeros((14, 14))
    coef[5, 5] = 1.0
    basis = scipy.fft.idctn(coef, type=2, norm="ortho")
    side = 14 * m * 2
    for c, keep in [(1e-3, True), (3e-5, False)]:
        y = np.full((side, side), 0.5)
        for i in range(0, side, 14):
            for j in range(0, side, 14):
                y[i:i + 14, j:j + 14] += c * basis
        fr = np.stack([y, y, y])
        r = osel.select_item(fr, fr, osel.SelectParams(merge=m))
        want = m * m * c * c
        if keep:
            np.testing.assert_allclose(r.energy, want, rtol=1e-6)
        else:
            assert np.all(r.energy == 0.0)


# ------------------------------------------------------------------ decision margins
def _hand_result(**kw):
    base = dict(reuse_mask=np.zeros(4, np.uint8), recompute_idx=np.arange(4, dtype=np.int32),
                shift=(0, 0), sim=np.array([0.95, 0.90, 0.80, 0.0]),
                energy=np.array([1.0, 2.0, 3.0, 4.0]),
                aligned=np.array([True, True, True, False]),
                fresh=np.array([False, False, False, True]),
                cand=np.array([True, True, True, False]), sim_freq=0.13, psi=0.5, alpha=0.30,
                mu=2.5, sigma=1.118, thr=2.5, k_reuse=1, k_cand=3, k_final=2, flushed=False,
                response=np.array([[1.0, 0.25], [-0.1, 0.0]]))
    base.update(kw)
    return osel.SelectResult(**base)


def test_decision_margins_hand_built():
    """Each margin of the mismatch audit on a result with known gaps:
    threshold |E - 2.5| / 2.5, top-K gap between the 2nd and 3rd candidate keys
    (3 - 2) / 3, budget |0.3 * 4 - 1| / 1.2, gate |0.13 - 0.12| / 0.12, shift peak
    minus runner-up (1 - 0.25) / 1, and the similarity floor |sim - 0.85| / 0.85 on
    aligned tokens only."""
    prm = osel.SelectParams(tau_sim=0.85)
    mg = osel.decision_margins(_hand_result(), prm)
    np.testing.assert_allclose(mg["threshold"], [0.6, 0.2, 0.2, 0.6], rtol=1e-14)
    assert mg["topk"] == pytest.approx(1.0 / 3.0, rel=1e-14)
    assert mg["budget"] == pytest.approx(0.2 / 1.2, rel=1e-12)
    assert mg["gate"] == pytest.approx(0.01 / 0.12, rel=1e-12)
    assert mg["shift"] == pytest.approx(0.75, rel=1e-14)
    np.testing.assert_allclose(mg["tau_sim"][:3], np.abs([0.95, 0.90, 0.80] - np.float64(0.85)) / 0.85,
                               rtol=1e-12)
    assert mg["tau_sim"][3] == np.inf


def test_decision_margins_degenerate_cases():
    """No top-K boundary when every candidate (or none) is taken; a fixed budget has no
    rounding decision; without a similarity floor no token has a floor margin; a tie
    of the two largest phase-correlation values has margin 0."""
    prm = osel.SelectParams(adaptive=False)
    mg = osel.decision_margins(_hand_result(k_final=3), prm)
    assert mg["topk"] == np.inf and mg["budget"] == np.inf and np.all(mg["tau_sim"] == np.inf)
    mg = osel.decision_margins(_hand_result(k_final=0), prm)
    assert mg["topk"] == np.inf
    mg = osel.decision_margins(_hand_result(response=np.array([[0.5, 0.5], [0.1, 0.0]])), prm)
    assert mg["shift"] == 0.0
    # a budget exactly on an integer has margin 0 (alpha N = 2)
    mg = osel.decision_margins(_hand_result(alpha=0.5), osel.SelectParams())
    assert mg["budget"] == 0.0


def test_decision_margins_on_a_real_result_bound_the_decisions():
    """On a computed selection every margin is consistent with the decision it audits:
    no token sits exactly on the threshold, the K-th reused key is below the first
    unused candidate's by the top-K margin, and the argmax of the response is unique."""
    prev, cur, _ = _tiny()
    r = osel.select_item(prev, cur, osel.SelectParams())
    mg = osel.decision_margins(r, osel.SelectParams())
    assert np.all(mg["threshold"] > 0)
    assert (r.energy > r.thr).tolist() == r.fresh.tolist()
    keys = np.sort(r.energy[r.cand])
    if 0 < r.k_final < keys.size:
        assert keys[r.k_final] - keys[r.k_final - 1] == pytest.approx(mg["topk"] * keys[r.k_final])
    assert mg["shift"] > 0


def _tiny():
    import fcdata
    prev, cur, _ = fcdata.tiny_pair(0)
    return prev[0], cur[0], None


# ------------------------------------------------------------------ naive baseline (Sec. 6.1)
def test_naive_selector_position_wise():
    """The naive baseline compares each token with the previous frame's token at the same
    position: identical frames reuse everything; a whole-token roll of random content
    (which the full method aligns) leaves almost nothing above a strict threshold; a
    missing previous frame reuses nothing."""
    fr = RNG.uniform(size=(3, 112, 112))
    r = osel.naive_select(fr, fr, 14, 1, 0.999)
    assert r.reuse_mask.all() and r.n_recompute == 0
    np.testing.assert_allclose(r.sim, 1.0, atol=1e-12)
    cur = np.roll(fr, (14, 14), (1, 2))
    r = osel.naive_select(fr, cur, 14, 1, 0.999)
    assert r.reuse_mask.sum() == 0 and np.all(r.sim < 0.999)
    full = osel.select_item(fr, cur, osel.SelectParams())
    assert full.shift == (-1, -1) and full.k_final > 0
    r = osel.naive_select(None, fr, 14, 1, 0.0)
    # a zero previous spectrum: cosine 0, which still reaches tau = 0
    assert r.reuse_mask.all() and np.all(r.sim == 0)
    r = osel.naive_select(None, fr, 14, 1, 1e-9)
    assert not r.reuse_mask.any()


def test_naive_selector_amplitude_invariances_and_threshold():
    """Amplitude spectra ignore a circular shift inside a patch (Fourier shift theorem):
    such a change keeps similarity 1 and the token is reused, while a token whose
    content is replaced falls below the threshold.  The threshold is inclusive (>=)
    and the recompute list is ascending."""
    prev = RNG.uniform(size=(3, 28, 56))                     # 2 x 4 tokens of 14 px
    cur = prev.copy()
    cur[:, 0:14, 14:28] = np.roll(prev[:, 0:14, 14:28], (3, 5), (1, 2))   # token 1: rolled
    cur[:, 14:28, 28:42] = RNG.uniform(size=(3, 14, 14))                   # token 6: replaced
    r = osel.naive_select(prev, cur, 14, 1, 0.999)
    assert r.sim[1] == pytest.approx(1.0, abs=1e-12) and r.reuse_mask[1] == 1
    assert r.sim[6] < 0.999 and r.reuse_mask[6] == 0
    assert r.recompute_idx.tolist() == [6]
    r2 = osel.naive_select(prev, cur, 14, 1, float(r.sim[6]))
    assert r2.reuse_mask[6] == 1                              # sim == tau is reused
    # brute force: the cosine of the flattened amplitude spectra, token 6
    a = np.abs(np.fft.fft2(osel.luma(cur)[14:28, 28:42]))
    b = np.abs(np.fft.fft2(osel.luma(prev)[14:28, 28:42]))
    assert r.sim[6] == pytest.approx(np.sum(a * b) / np.linalg.norm(a) / np.linalg.norm(b), rel=1e-12)


def test_naive_selector_equals_the_module_ablation_combination():
    """With alignment, refresh, the adaptive budget and the gate all switched off
    (shift 0, no fresh token, a 100 % budget, tau_mig = 0) Algorithm 1 reduces to the
    naive baseline: the candidates are the tokens whose position-wise similarity
    reaches tau_sim, and all of them are reused."""
    fr = fcdata_frames()
    for b in range(1, 3):
        naive = osel.naive_select(fr[b - 1], fr[b], 14, 2, 0.99)
        alg1 = osel.select_item(fr[b - 1], fr[b], osel.SelectParams(
            merge=2, align=False, refresh=False, adaptive=False, alpha_fixed=1.0, tau_sim=0.99,
            tau_mig=0.0))
        np.testing.assert_array_equal(naive.reuse_mask, alg1.reuse_mask)
        np.testing.assert_allclose(naive.sim, alg1.sim, rtol=1e-14)


def fcdata_frames():
    import fcdata
    return fcdata.episode_frames(2024, size=448, n_frames=3)
