"""Pins of the oracle's pixel-resolution phase correlation (Eq. 4-1 on full-resolution
luma, the align_pixel variant of Module I) against facts that do not come from the
oracle itself: circular shifts, a brute-force transform, the Fourier shift theorem for
fractional shifts, a parabola's vertex, a camera trajectory with known motion, and the
token-grid path on whole-token shifts."""
import numpy as np
import pytest

import fcdata
from oracle import select as osel


def rand_luma(rng, h, w):
    return rng.random((h, w))


@pytest.mark.parametrize("shape,shift", [((28, 42), (3, -5)), ((56, 56), (-27, 28)),
                                         ((42, 28), (0, 13)), ((28, 28), (14, 14))])
def test_circular_integer_shift(shape, shift):
    """Content rolled by d: the displacement is -d (token (I, J) takes its source at
    (I - d)), wrapped into (-N/2, N/2], with no sub-pixel correction."""
    rng = np.random.default_rng(1)
    h, w = shape
    y0 = rand_luma(rng, h, w)
    y1 = np.roll(y0, shift, axis=(0, 1))
    (di, dj), (pi, pj), r = osel.pixel_phase_correlation(y0, y1)

    def wrap(v, n):
        v %= n
        return v if v <= n // 2 else v - n
    assert (pi, pj) == (wrap(-shift[0], h), wrap(-shift[1], w))
    assert abs(di - pi) < 1e-9 and abs(dj - pj) < 1e-9
    assert r.max() == pytest.approx(1.0, abs=1e-9)


def test_response_against_brute_force_sums():
    """The response surface equals the explicit double sums of Eq. 4-1 on a 6 x 8
    pair: X(u,v) = F1(u,v) conj(F2(u,v)) with F(u,v) = sum_yx f e^{-2 pi i (uy/H + vx/W)},
    C = X / |X|, r(y,x) = Re (1/HW) sum_uv C e^{+2 pi i (uy/H + vx/W)}."""
    rng = np.random.default_rng(2)
    h, w = 6, 8
    a, b = rand_luma(rng, h, w), rand_luma(rng, h, w)

    def dft(f):
        out = np.zeros((h, w), complex)
        for u in range(h):
            for v in range(w):
                for y in range(h):
                    for x in range(w):
                        out[u, v] += f[y, x] * np.exp(-2j * np.pi * (u * y / h + v * x / w))
        return out
    x = dft(a) * np.conj(dft(b))
    c = x / np.abs(x)
    r = np.zeros((h, w))
    for y in range(h):
        for xx in range(w):
            acc = 0j
            for u in range(h):
                for v in range(w):
                    acc += c[u, v] * np.exp(2j * np.pi * (u * y / h + v * xx / w))
            r[y, xx] = (acc / (h * w)).real
    _, _, resp = osel.pixel_phase_correlation(a, b)
    np.testing.assert_allclose(resp, r, atol=1e-12)


@pytest.mark.parametrize("t0", [-0.5, -0.3, 0.0, 0.17, 0.5])
def test_parabolic_offset_is_the_vertex(t0):
    f = lambda t: 3.0 - 2.0 * (t - t0) ** 2          # noqa: E731
    assert osel.parabolic_offset(f(-1), f(0), f(1)) == pytest.approx(t0, abs=1e-12)


def test_parabolic_offset_flat_and_valley():
    assert osel.parabolic_offset(1.0, 1.0, 1.0) == 0.0
    assert osel.parabolic_offset(2.0, 1.0, 2.0) == 0.0        # not a peak
    assert osel.parabolic_offset(0.0, 1.0, 0.0) == 0.0


@pytest.mark.parametrize("s", [(0.3, -0.2), (-0.45, 0.4), (2.25, -3.4)])
def test_fractional_shift_sign_and_size(s):
    """A band-limited circular shift by s (phase ramp, Fourier shift theorem) gives a
    sub-pixel estimate on the right side of the integer peak: within 0.25 px of -s."""
    rng = np.random.default_rng(3)
    h = w = 56
    y0 = rand_luma(rng, h, w)
    u = np.fft.fftfreq(h)[:, None]
    v = np.fft.fftfreq(w)[None, :]
    y1 = np.real(np.fft.ifft2(np.fft.fft2(y0) * np.exp(-2j * np.pi * (u * s[0] + v * s[1]))))
    (di, dj), _, _ = osel.pixel_phase_correlation(y0, y1)
    assert abs(di + s[0]) < 0.25 and abs(dj + s[1]) < 0.25


def test_constant_and_missing_frames():
    """Spectra that are zero outside DC give a flat or zero surface: displacement
    (0, 0), no sub-pixel correction."""
    y = np.full((28, 28), 0.5)
    (di, dj), (pi, pj), r = osel.pixel_phase_correlation(y, y * 0.3)
    assert (pi, pj) == (0, 0) and (di, dj) == (0.0, 0.0)
    (di, dj), (pi, pj), r = osel.pixel_phase_correlation(np.zeros((28, 28)),
                                                         rand_luma(np.random.default_rng(4), 28, 28))
    assert (pi, pj) == (0, 0) and (di, dj) == (0.0, 0.0) and not r.any()


def test_token_shift_rounding():
    assert osel.token_shift(13.9, 28) == 0
    assert osel.token_shift(14.0, 28) == 1
    assert osel.token_shift(-14.0, 28) == -1
    assert osel.token_shift(-41.99, 28) == -1
    assert osel.token_shift(42.0, 28) == 2
    assert osel.token_shift(0.0, 14) == 0


def test_camera_trajectory_motion_recovered():
    """Consecutive frames of the seeded camera walk without shear (pure translation,
    new content entering at the borders): the camera moved by dpos pixels of texture,
    so content moved by -dpos and the displacement is +dpos, to a tenth of a pixel."""
    frames = fcdata.episode_frames(77, size=224, n_frames=6, shear=0.0)
    rng = np.random.default_rng(77)
    # replay the generator's random walk to get the true positions
    texture, max_step, shear = fcdata.EPISODE["texture"], fcdata.EPISODE["max_step"], 0.0
    area = (texture / 576.0) ** 2
    fcdata.frames.canvas(rng, texture, texture, n_blobs=int(32 * area), n_rects=int(8 * area),
                         n_bars=int(4 * area))
    pad = int(np.ceil(shear * 224 / 2)) + 2
    lo, hi = pad, texture - 224 - pad
    pos = np.array([(lo + hi) // 2, (lo + hi) // 2], dtype=np.int64)
    prev_pos = None
    for k in range(6):
        if k > 0:
            pos = np.clip(pos + rng.integers(-max_step, max_step + 1, 2), lo, hi)
        rng.uniform(-shear, shear)
        if k > 0:
            d = pos - prev_pos
            (di, dj), _, _ = osel.pixel_phase_correlation(osel.luma(frames[k - 1]),
                                                          osel.luma(frames[k]))
            assert abs(di - d[0]) < 0.1 and abs(dj - d[1]) < 0.1, (k, (di, dj), d)
        prev_pos = pos.copy()


@pytest.mark.parametrize("rolls", [(28, -56), (-28, 0), (0, 0)])
def test_pixel_mode_matches_grid_mode_on_whole_token_rolls(rolls):
    """Rolled by whole tokens (28 px at merge 2), both Module I readings find the same
    token displacement, so the whole selection agrees."""
    rng = np.random.default_rng(5)
    prev = rng.random((3, 112, 112)).astype(np.float32)
    cur = np.roll(prev, rolls, axis=(1, 2))
    base = osel.SelectParams(merge=2)
    pix = osel.SelectParams(merge=2, align_pixel=True)
    a = osel.select_item(prev, cur, base)
    b = osel.select_item(prev, cur, pix)
    assert a.shift == b.shift == (-rolls[0] // 28, -rolls[1] // 28)
    assert b.shift_px == pytest.approx((-rolls[0], -rolls[1]), abs=1e-9)
    np.testing.assert_array_equal(a.reuse_mask, b.reuse_mask)


def test_pixel_mode_margins():
    """The shift margin of the pixel mode is the rounding distance (token units) when no
    far peak competes."""
    rng = np.random.default_rng(6)
    prev = rng.random((3, 112, 112)).astype(np.float32)
    cur = np.roll(prev, (0, 21), axis=(1, 2))          # -21 px = -0.75 tokens
    prm = osel.SelectParams(merge=2, align_pixel=True)
    res = osel.select_item(prev, cur, prm)
    assert res.shift == (0, -1)
    mg = osel.decision_margins(res, prm)
    assert mg["shift"] == pytest.approx(0.25, abs=1e-9)


# ------------------------------------------------- rotation (log-polar, Fourier-Mellin)
def test_highpass_weight_closed_forms():
    hp = osel.highpass_weight(8, 12)
    assert hp[0, 0] == 0.0                                   # DC
    assert hp[4, 6] == pytest.approx(2.0, abs=1e-15)         # both Nyquist: X = 0
    x = np.cos(np.pi * 1 / 8) * np.cos(np.pi * 2 / 12)
    assert hp[1, 2] == pytest.approx((1 - x) * (2 - x), rel=1e-14)
    np.testing.assert_allclose(hp[1:, 1:], hp[1:, 1:][::-1, ::-1], rtol=1e-14)   # central symmetry


def test_bilinear_exact_on_affine_and_zero_outside():
    yy, xx = np.meshgrid(np.arange(6.0), np.arange(7.0), indexing="ij")
    img = 0.5 * yy - 0.25 * xx + 2.0
    ys, xs = np.array([0.3, 2.75, 4.5]), np.array([1.2, 5.9, 0.0])
    np.testing.assert_allclose(osel.bilinear(img, ys, xs, wrap=False), 0.5 * ys - 0.25 * xs + 2.0,
                               rtol=1e-14)
    assert osel.bilinear(img, np.array([-1.5]), np.array([2.0]), wrap=False)[0] == 0.0
    assert osel.bilinear(img, np.array([-1.0]), np.array([0.0]), wrap=True)[0] == img[5, 0]


def test_rotate_image_quarter_turn_is_rot90():
    y = np.random.default_rng(7).random((9, 9))
    np.testing.assert_allclose(osel.rotate_image(y, np.pi / 2), np.rot90(y), atol=1e-12)
    np.testing.assert_allclose(osel.rotate_image(y, 0.0), y, atol=0)


def test_log_polar_of_radial_spectrum_is_constant_in_angle():
    """A spectrum that depends on the radius only resamples to rows equal across angles
    (up to the bilinear error of a smooth function)."""
    h = w = 64
    fu = np.fft.fftfreq(h)[:, None] * h
    fv = np.fft.fftfreq(w)[None, :] * w
    mag = np.exp(-(fu ** 2 + fv ** 2) / 200.0)
    lp = osel.log_polar(mag, 32, 16)
    assert np.abs(lp - lp.mean(axis=0, keepdims=True)).max() < 0.02
    # column j samples radius R^(j / n_rho): compare with the function itself
    r = (31.0) ** (np.arange(16) / 16)
    np.testing.assert_allclose(lp.mean(axis=0), np.exp(-r ** 2 / 200.0), atol=0.02)


def trajectory_luma(size=224):
    return osel.luma(fcdata.episode_frames(11, size=size, n_frames=1, shear=0.0)[0])


@pytest.mark.parametrize("a", [0.05, -0.1, 0.2])
def test_rotation_recovered_with_its_sign(a):
    """The current frame is the previous one rotated by a (about the centre): the
    estimated angle is within 0.01 rad of a (the angular bins are pi / 224 = 0.014 rad),
    and the centre's displacement after rotating back under 0.5 px."""
    y0 = trajectory_luma()
    y1 = osel.rotate_image(y0, -a)
    ang, (di, dj), _ = osel.rotation_phase_correlation(y0, y1)
    assert abs(ang - a) < 0.01
    assert abs(di) < 0.5 and abs(dj) < 0.5


def test_rotation_then_translation():
    """Rotated by 0.1 rad and then moved by (6, -9) px: the angle is found and the
    centre's displacement is the move back, (-6, 9), within a pixel."""
    y0 = trajectory_luma()
    y1 = np.roll(osel.rotate_image(y0, -0.1), (6, -9), axis=(0, 1))
    ang, (di, dj), _ = osel.rotation_phase_correlation(y0, y1)
    assert abs(ang - 0.1) < 0.01
    assert abs(di + 6) < 1.0 and abs(dj - 9) < 1.0


def test_pure_roll_has_no_rotation():
    """A circular roll leaves the magnitude spectra equal (up to rounding): angle 0, and
    the displacement is the plain pixel-resolution one."""
    y0 = trajectory_luma()
    y1 = np.roll(y0, (-5, 12), axis=(0, 1))
    ang, d, _ = osel.rotation_phase_correlation(y0, y1)
    assert abs(ang) < 1e-12
    assert d == pytest.approx(osel.pixel_phase_correlation(y0, y1)[0], abs=1e-12)


def test_rotation_mode_in_the_selection():
    """select_item with align_rotation on a rotated-then-moved pair: the rotation is
    reported and the token displacement is that of the image centre after undoing it;
    on a pure whole-token roll it equals the plain pixel mode."""
    frames = fcdata.episode_frames(11, size=224, n_frames=1, shear=0.0)
    prev = frames[0]
    cur = np.stack([np.roll(osel.rotate_image(prev[c].astype(np.float64), -0.08), (28, 0),
                            axis=(0, 1)) for c in range(3)]).astype(np.float32)
    prm = osel.SelectParams(merge=2, align_pixel=True, align_rotation=True)
    res = osel.select_item(prev, cur, prm)
    assert abs(res.angle - 0.08) < 0.01 and res.shift == (-1, 0)
    rolled = np.roll(prev, (0, -56), axis=(1, 2))
    a = osel.select_item(prev, rolled, prm)
    b = osel.select_item(prev, rolled, osel.SelectParams(merge=2, align_pixel=True))
    assert a.shift == b.shift == (0, 2) and abs(a.angle) < 1e-12
    np.testing.assert_array_equal(a.reuse_mask, b.reuse_mask)
