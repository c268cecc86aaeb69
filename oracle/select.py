"""FreqCache cacheable-token selection -- CPU oracle, float64.

TEST INFRASTRUCTURE ONLY.  This module is the plain, slow reference that the
HIP path is checked against.  Only tests/, __graft_entry__.smoke() and the
cpu_baseline leg of bench.py may import it; the product path never does.  It
shares no code, tables or constants with the HIP sources.

Every transform is written as its textbook definition (matrix DFT, matrix
DCT-II), not as a fast algorithm.  Step names (O1..O19) follow the order in
which the paper computes things:

  Module I   (Sec. 4.1, Eqs. 3-2, 3-3, 4-1, 4-2): amplitude spectra, global
             spectral similarity and the migration gate, phase correlation for
             the displacement, alignment mask;
  Module II  (Sec. 4.2, Eqs. 3-4, 3-5, 4-3): block DCT, high-pass energy, the
             mean + lambda * std refresh rule;
  Module III (Sec. 4.3, Eqs. 3-6, 4-4): spectral entropy and adaptive budget;
  Fusion     (Sec. 4.4, Algorithm 1): candidates, ascending-energy top-K.

Readings where the paper is silent or garbled:
  * colour -> one channel: BT.601 luma of the [0,1] RGB frame;
  * DFT unnormalised; DCT-II orthonormal;
  * "feature maps" of Modules I/III: the token-grid map of mean luma;
  * the entropy formula missing from Eq. 3-6: Shannon entropy of the
    normalised power, divided by ln(M) (M = grid bins) when entropy_norm;
  * std is the population std; E below 1e-8 * m^2 is snapped to exactly 0;
  * phase-correlation guard |X| <= 1e-9 max|X| -> 0, real part, first
    (lowest row-major) index on ties, signed wrap keeping +G/2 positive;
  * a missing previous frame is treated as an all-zero previous frame;
  * align_pixel (a Module I variant): F of Eq. 4-1 is the full-resolution luma,
    the integer peak is refined per axis by a three-point parabola, and the
    displacement is rounded to whole tokens (halves away from zero);
  * align_rotation (with align_pixel): the rotation comes first from Eq. 4-1 on
    log-polar resampled, high-pass weighted magnitude spectra (Fourier-Mellin) and is
    undone by bilinear resampling about the frame centre before the displacement.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np


@dataclass
class SelectParams:
    """Selection hyper-parameters.  Defaults are the paper's chosen values
    (Sec. 6.4: tau_mig = 0.12, lambda = 0.25, alpha_max = 0.5, alpha_min = 0.08)."""
    patch: int = 14
    merge: int = 1
    tau_mig: float = 0.12
    lam: float = 0.25
    alpha_min: float = 0.08
    alpha_max: float = 0.5
    adaptive: bool = True          # False: fixed reuse ratio alpha_fixed (ablation "w/o III")
    alpha_fixed: float = 0.5
    entropy_norm: bool = True
    tau_sim: float = 0.0           # per-token similarity floor; 0 is exact Algorithm 1
    # Module ablations of Table 3 (Sec. 6.3):
    align: bool = True             # False: "w/o Module I", position-wise matching (Delta = 0)
    align_pixel: bool = False      # True: Eq. 4-1 on full-resolution luma, sub-pixel peak,
                                   # displacement rounded to whole tokens
    align_rotation: bool = False   # with align_pixel: the current frame's rotation found
                                   # and undone first (log-polar spectra)
    refresh: bool = True           # False: "w/o Module II", no high-frequency refresh


# ---------------------------------------------------------------- O1, O2: luma and tiling
def luma(frame: np.ndarray) -> np.ndarray:
    """O1: BT.601 luma of a [3, H, W] RGB frame, float64."""
    f = np.asarray(frame, dtype=np.float64)
    return 0.299 * f[0] + 0.587 * f[1] + 0.114 * f[2]


def patches(y: np.ndarray, p: int) -> np.ndarray:
    """O2: non-overlapping P x P patches p_(i,j) of an [H, W] map -> [H/P, W/P, P, P]
    (grid partition of Sec. 3.2)."""
    h, w = y.shape
    return y.reshape(h // p, p, w // p, p).transpose(0, 2, 1, 3)


# ---------------------------------------------------------------- transforms (definitions)
def dft_matrix(n: int) -> np.ndarray:
    """W[u, y] = exp(-2 pi i u y / n), the 1-D DFT as a matrix (exact phase index)."""
    k = np.arange(n)
    ang = 2.0 * np.pi * ((k[:, None] * k[None, :]) % n) / n
    return np.cos(ang) - 1j * np.sin(ang)


def dft2(x: np.ndarray) -> np.ndarray:
    """2-D DFT of the last two axes, X(u,v) = sum_{y,x} x(y,x) e^{-2 pi i (uy/H + vx/W)}."""
    wh = dft_matrix(x.shape[-2])
    ww = dft_matrix(x.shape[-1])
    return wh @ x @ ww.T


def idft2(x: np.ndarray) -> np.ndarray:
    """Inverse 2-D DFT (with the 1/(H W) factor)."""
    h, w = x.shape[-2:]
    wh = np.conj(dft_matrix(h))
    ww = np.conj(dft_matrix(w))
    return (wh @ x @ ww.T) / (h * w)


def dct_matrix(n: int) -> np.ndarray:
    """Orthonormal DCT-II: C[k, j] = s_k cos(pi (2j + 1) k / (2n)), s_0 = sqrt(1/n),
    s_k = sqrt(2/n)."""
    k = np.arange(n)[:, None]
    j = np.arange(n)[None, :]
    c = np.cos(np.pi * (2 * j + 1) * k / (2 * n))
    s = np.full((n, 1), np.sqrt(2.0 / n))
    s[0, 0] = np.sqrt(1.0 / n)
    return s * c


def high_pass(p: int) -> np.ndarray:
    """Eq. 3-4: H(u,v) = 0 iff u < c and v < c, c = max(1, floor(P/4)); else 1."""
    c = max(1, p // 4)
    h = np.ones((p, p))
    h[:c, :c] = 0.0
    return h


# ---------------------------------------------------------------- per-patch quantities
def patch_amplitude(pt: np.ndarray) -> np.ndarray:
    """O3, Eq. 3-2: amplitude spectrum A = sqrt(R^2 + I^2) of each patch's 2-D DFT."""
    return np.abs(dft2(pt))


def patch_energy(pt: np.ndarray) -> np.ndarray:
    """O14-O15, Eqs. 3-4/3-5: E = sum_{u,v} (H(u,v) D(u,v))^2 with D the patch's
    2-D DCT-II."""
    p = pt.shape[-1]
    c = dct_matrix(p)
    d = c @ pt @ c.T
    return np.sum((high_pass(p) * d) ** 2, axis=(-1, -2))


def token_view(a: np.ndarray, m: int) -> np.ndarray:
    """Group a per-patch array [Gp_h, Gp_w, ...] into tokens of m x m patches:
    -> [Gp_h/m, Gp_w/m, m*m, ...] with the m*m sub-patches in row-major order."""
    gh, gw = a.shape[:2]
    rest = a.shape[2:]
    t = a.reshape(gh // m, m, gw // m, m, *rest)
    t = np.moveaxis(t, 2, 1)           # [I, J, a, b, ...]
    return t.reshape(gh // m, gw // m, m * m, *rest)


# ---------------------------------------------------------------- Module III
def spectral_entropy(f_cur: np.ndarray, normalise: bool) -> float:
    """O9, Eq. 3-6: P = |F|^2 / sum |F|^2 and Psi = -sum P ln P (0 ln 0 = 0),
    divided by ln(M) when `normalise` (M = number of bins)."""
    pw = np.abs(f_cur) ** 2
    tot = pw.sum()
    if tot <= 0.0:
        return 0.0
    pr = (pw / tot).ravel()
    nz = pr[pr > 0]
    psi = float(-np.sum(nz * np.log(nz)))
    if normalise:
        m = pr.size
        psi = psi / np.log(m) if m > 1 else 0.0
    return psi


def reuse_budget(psi: float, n_tokens: int, prm: SelectParams):
    """O10, Eq. 4-4: alpha_t = a_min + (a_max - a_min) e^{-Psi}; K_reuse = floor(alpha_t N)."""
    if prm.adaptive:
        alpha = prm.alpha_min + (prm.alpha_max - prm.alpha_min) * np.exp(-psi)
    else:
        alpha = prm.alpha_fixed
    return float(alpha), int(np.floor(alpha * n_tokens))


# ---------------------------------------------------------------- Module I
def global_similarity(f_cur: np.ndarray, f_prev: np.ndarray) -> float:
    """O7, Eq. 3-3 on the global spectra: cosine of the amplitude spectra
    (all bins, DC included); 0 if either spectrum is zero."""
    a = np.abs(f_cur).ravel()
    b = np.abs(f_prev).ravel()
    na, nb = np.sqrt(np.sum(a * a)), np.sqrt(np.sum(b * b))
    if na == 0.0 or nb == 0.0:
        return 0.0
    return float(np.sum(a * b) / (na * nb))


def phase_correlation(f_prev: np.ndarray, f_cur: np.ndarray):
    """O11, Eq. 4-1: C = X / |X| with X = F(F_{t-1}) . conj(F(F_t)); the displacement
    is the argmax of Re F^{-1}(C), wrapped to signed offsets.

    Returns ((di, dj), response) where response is the real inverse transform.
    """
    x = f_prev * np.conj(f_cur)
    mag = np.abs(x)
    mx = mag.max()
    c = np.zeros_like(x)
    if mx > 0.0:
        keep = mag > 1e-9 * mx
        c[keep] = x[keep] / mag[keep]
    r = np.real(idft2(c))
    k = int(np.argmax(r))          # first maximum in row-major order
    gh, gw = r.shape
    ki, kj = divmod(k, gw)
    di = ki if ki <= gh // 2 else ki - gh
    dj = kj if kj <= gw // 2 else kj - gw
    return (di, dj), r


def parabolic_offset(a: float, b: float, c: float) -> float:
    """Vertex of the parabola through (-1, a), (0, b), (+1, c), relative to 0:
    (a - c) / (2 (a - 2b + c)); 0 when the three points are not a strict peak
    (a - 2b + c >= 0).  With b the maximum of the three, |offset| <= 1/2."""
    den = a - 2.0 * b + c
    if den >= 0.0:
        return 0.0
    return float((a - c) / (2.0 * den))


def pixel_phase_correlation(y_prev: np.ndarray, y_cur: np.ndarray):
    """Eq. 4-1 with the feature maps F taken as the frames' full-resolution luma: the
    integer displacement (pixels) is the argmax of the phase-correlation surface (same
    guard, tie and wrap rules as on the token grid), refined per axis by the vertex of
    the parabola through the peak and its two circular neighbours along that axis.

    Returns ((di, dj) sub-pixel floats, (pi, pj) integer peak, response)."""
    (pi, pj), r = phase_correlation(dft2(y_prev), dft2(y_cur))
    h, w = r.shape
    ki, kj = pi % h, pj % w
    di = pi + parabolic_offset(r[(ki - 1) % h, kj], r[ki, kj], r[(ki + 1) % h, kj])
    dj = pj + parabolic_offset(r[ki, (kj - 1) % w], r[ki, kj], r[ki, (kj + 1) % w])
    return (float(di), float(dj)), (int(pi), int(pj)), r


def token_shift(d_px: float, tp: int) -> int:
    """A pixel displacement in whole tokens of tp pixels: d / tp rounded to the
    nearest integer, halves away from zero."""
    q = abs(d_px) / tp
    return int(np.floor(q + 0.5)) * (1 if d_px >= 0 else -1)


def highpass_weight(h: int, w: int) -> np.ndarray:
    """High-pass emphasis of a magnitude spectrum before log-polar resampling:
    (1 - X)(2 - X) with X = cos(pi f_u) cos(pi f_v), f the signed frequency in cycles per
    sample (0 at DC, 2 at the Nyquist corners)."""
    fu = np.fft.fftfreq(h)[:, None]
    fv = np.fft.fftfreq(w)[None, :]
    x = np.cos(np.pi * fu) * np.cos(np.pi * fv)
    return (1.0 - x) * (2.0 - x)


def bilinear(img: np.ndarray, y: np.ndarray, x: np.ndarray, wrap: bool) -> np.ndarray:
    """Bilinear interpolation of img at (y, x); wrap: circular indices, otherwise 0
    outside the image."""
    h, w = img.shape
    y0, x0 = np.floor(y).astype(np.int64), np.floor(x).astype(np.int64)
    fy, fx = y - y0, x - x0
    out = np.zeros(np.broadcast(y, x).shape)
    for a, wa in ((0, 1.0 - fy), (1, fy)):
        for b, wb in ((0, 1.0 - fx), (1, fx)):
            yy, xx = y0 + a, x0 + b
            if wrap:
                v = img[yy % h, xx % w]
            else:
                ok = (yy >= 0) & (yy < h) & (xx >= 0) & (xx < w)
                v = np.where(ok, img[np.clip(yy, 0, h - 1), np.clip(xx, 0, w - 1)], 0.0)
            out = out + wa * wb * v
    return out


def log_polar(mag: np.ndarray, n_theta: int, n_rho: int) -> np.ndarray:
    """Samples a (centrally symmetric) magnitude spectrum at angles theta_i = pi i / n_theta
    and radii r_j = R^(j / n_rho), R = min(H, W) / 2 - 1, i.e. at frequency
    (r sin theta, r cos theta) with circular indexing; bilinear."""
    h, w = mag.shape
    big_r = min(h, w) / 2.0 - 1.0
    th = np.pi * np.arange(n_theta)[:, None] / n_theta
    r = big_r ** (np.arange(n_rho)[None, :] / n_rho)
    return bilinear(mag, r * np.sin(th), r * np.cos(th), wrap=True)


def rotate_image(y: np.ndarray, angle: float) -> np.ndarray:
    """y sampled at the points q rotated by `angle` about the image centre,
    out(q) = y(R(angle) (q - c) + c) with (x', y') = (x cos a - y sin a, x sin a + y cos a)
    in (column, row) coordinates; bilinear, 0 outside."""
    h, w = y.shape
    cy, cx = (h - 1) / 2.0, (w - 1) / 2.0
    qy, qx = np.meshgrid(np.arange(h) - cy, np.arange(w) - cx, indexing="ij")
    ca, sa = np.cos(angle), np.sin(angle)
    return bilinear(y, qx * sa + qy * ca + cy, qx * ca - qy * sa + cx, wrap=False)


def rotation_phase_correlation(y_prev: np.ndarray, y_cur: np.ndarray):
    """Fourier-Mellin step of the pixel-resolution Module I: Eq. 4-1 on the log-polar
    resampled, high-pass weighted magnitude spectra (n_theta = H angles over [0, pi),
    n_rho = min(H, W) / 2 radii) gives the rotation of the current frame relative to the
    previous one from the angular coordinate of the peak (sub-sample peak as in
    pixel_phase_correlation; its radial coordinate, the scale, is not used); the current
    frame is rotated back and Eq. 4-1 on the pair gives the displacement of the image
    centre.

    Returns (angle, (di, dj) sub-pixel floats, response of the final correlation)."""
    h, w = y_prev.shape
    n_theta, n_rho = h, min(h, w) // 2
    hp = highpass_weight(h, w)
    lp_prev = log_polar(np.abs(dft2(y_prev)) * hp, n_theta, n_rho)
    lp_cur = log_polar(np.abs(dft2(y_cur)) * hp, n_theta, n_rho)
    (d_th, _), _, _ = pixel_phase_correlation(lp_prev, lp_cur)
    angle = -d_th * np.pi / n_theta
    (di, dj), _, resp = pixel_phase_correlation(y_prev, rotate_image(y_cur, angle))
    return float(angle), (float(di), float(dj)), resp


def align_mask(gh: int, gw: int, di: int, dj: int) -> np.ndarray:
    """O12, Eq. 4-2: token (I, J) is aligned iff its source (I + di, J + dj) lies in
    the previous token grid."""
    i = np.arange(gh)[:, None] + di
    j = np.arange(gw)[None, :] + dj
    return ((i >= 0) & (i < gh) & (j >= 0) & (j < gw))


def token_similarity(a_cur: np.ndarray, a_prev: np.ndarray, di: int, dj: int,
                     aligned: np.ndarray) -> np.ndarray:
    """O13: per-token Eq. 3-3 -- cosine between the current token's amplitude vector and
    that of its source token in the previous frame; 0 when not aligned.  Both norms
    zero -> 1, exactly one zero -> 0.  a_*: [Gh, Gw, L] token amplitude vectors."""
    gh, gw = aligned.shape
    sim = np.zeros((gh, gw))
    for i in range(gh):
        for j in range(gw):
            if not aligned[i, j]:
                continue
            u = a_cur[i, j]
            v = a_prev[i + di, j + dj]
            nu, nv = np.sqrt(np.sum(u * u)), np.sqrt(np.sum(v * v))
            if nu == 0.0 and nv == 0.0:
                sim[i, j] = 1.0
            elif nu == 0.0 or nv == 0.0:
                sim[i, j] = 0.0
            else:
                sim[i, j] = np.sum(u * v) / (nu * nv)
    return sim


# ---------------------------------------------------------------- Module II
def refresh_mask(e_tok: np.ndarray, lam: float):
    """O16, Eq. 4-3: Mask_fresh = 1(E > mu_E + lambda sigma_E), population statistics
    over all N tokens."""
    mu = float(np.mean(e_tok))
    sd = float(np.sqrt(np.mean((e_tok - mu) ** 2)))
    thr = mu + lam * sd
    return e_tok > thr, mu, sd, thr


# ---------------------------------------------------------------- Fusion (Algorithm 1)
def topk_ascending(cand: np.ndarray, key: np.ndarray, k: int) -> np.ndarray:
    """O18: the k candidates with the smallest key, ties to the lower token id."""
    ids = np.flatnonzero(cand)
    order = sorted(ids.tolist(), key=lambda t: (key[t], t))
    return np.asarray(order[:k], dtype=np.int64)


@dataclass
class SelectResult:
    reuse_mask: np.ndarray        # [N] uint8, 1 = reuse cached token
    recompute_idx: np.ndarray     # [N - K_final] int32, ascending
    shift: tuple                  # (di, dj): token (I,J) reuses source (I+di, J+dj)
    sim: np.ndarray               # [N] per-token aligned spectral similarity
    energy: np.ndarray            # [N] token high-frequency energy
    aligned: np.ndarray           # [N] bool
    fresh: np.ndarray             # [N] bool
    cand: np.ndarray              # [N] bool
    sim_freq: float
    psi: float
    alpha: float
    mu: float
    sigma: float
    thr: float
    k_reuse: int
    k_cand: int
    k_final: int
    flushed: bool
    response: np.ndarray = field(repr=False, default=None)   # phase-correlation surface
    shift_px: tuple = None        # sub-pixel displacement (align_pixel only)
    angle: float = 0.0            # rotation of the current frame (align_rotation only)

    @property
    def n_recompute(self) -> int:
        return int(self.recompute_idx.size)


def select_item(prev: np.ndarray | None, cur: np.ndarray, prm: SelectParams) -> SelectResult:
    """Algorithm 1 for one frame pair ([3, H, W] each; prev may be None)."""
    p, m = prm.patch, prm.merge
    y_cur = luma(cur)
    y_prev = luma(prev) if prev is not None else np.zeros_like(y_cur)
    h, w = y_cur.shape
    if h % (p * m) or w % (p * m):
        raise ValueError("frame size must be a multiple of patch * merge")
    pc, pp = patches(y_cur, p), patches(y_prev, p)
    # O3/O4: per-patch amplitude spectra, grouped into token vectors
    a_cur = token_view(patch_amplitude(pc), m)
    a_prev = token_view(patch_amplitude(pp), m)
    gh, gw = a_cur.shape[:2]
    n = gh * gw
    a_cur = a_cur.reshape(gh, gw, -1)
    a_prev = a_prev.reshape(gh, gw, -1)
    # O5/O6: token-grid mean-luma maps and their spectra
    g_cur = token_view(pc.mean(axis=(-1, -2)), m).mean(axis=-1)
    g_prev = token_view(pp.mean(axis=(-1, -2)), m).mean(axis=-1)
    f_cur, f_prev = dft2(g_cur), dft2(g_prev)
    # Module I
    sim_freq = global_similarity(f_cur, f_prev)
    flushed = sim_freq < prm.tau_mig
    shift_px = None
    angle = 0.0
    if prm.align_pixel:
        if prm.align_rotation:
            angle, shift_px, resp = rotation_phase_correlation(y_prev, y_cur)
        else:
            shift_px, _, resp = pixel_phase_correlation(y_prev, y_cur)
        di, dj = token_shift(shift_px[0], p * m), token_shift(shift_px[1], p * m)
    else:
        (di, dj), resp = phase_correlation(f_prev, f_cur)
    if not prm.align:
        # "w/o Module I": tokens are matched at their own positions
        di, dj = 0, 0
    aligned = align_mask(gh, gw, di, dj)
    sim = token_similarity(a_cur, a_prev, di, dj, aligned)
    # Module II
    e_tok = token_view(patch_energy(pc), m).sum(axis=-1)
    e_tok = np.where(e_tok < 1e-8 * m * m, 0.0, e_tok)
    fresh, mu, sd, thr = refresh_mask(e_tok, prm.lam)
    if not prm.refresh:
        # "w/o Module II": no token is forced to recompute by its edge energy
        fresh = np.zeros_like(fresh)
    # Module III
    psi = spectral_entropy(f_cur, prm.entropy_norm)
    alpha, k_reuse = reuse_budget(psi, n, prm)
    # Fusion
    e_flat = e_tok.ravel()
    cand = (aligned & ~fresh & (sim >= prm.tau_sim)).ravel()
    k_cand = int(cand.sum())
    reuse = np.zeros(n, np.uint8)
    k_final = 0
    if not flushed:
        k_final = min(k_reuse, k_cand)
        reuse[topk_ascending(cand, e_flat, k_final)] = 1
    return SelectResult(
        reuse_mask=reuse, recompute_idx=np.flatnonzero(reuse == 0).astype(np.int32),
        shift=(int(di), int(dj)), sim=sim.ravel(), energy=e_flat, aligned=aligned.ravel(),
        fresh=fresh.ravel(), cand=cand, sim_freq=sim_freq, psi=psi, alpha=alpha, mu=mu,
        sigma=sd, thr=thr, k_reuse=k_reuse, k_cand=k_cand, k_final=k_final,
        flushed=bool(flushed), response=resp, shift_px=shift_px, angle=angle)


@dataclass
class NaiveResult:
    reuse_mask: np.ndarray        # [N] uint8
    recompute_idx: np.ndarray     # ascending int32
    sim: np.ndarray               # [N] position-wise amplitude-spectrum cosine

    @property
    def n_recompute(self) -> int:
        return int(self.recompute_idx.size)


def naive_select(prev: np.ndarray | None, cur: np.ndarray, patch: int, merge: int,
                 tau: float) -> NaiveResult:
    """The naive frequency baseline the paper compares against (Sec. 6.1): the frame is
    cut into patches, each token's 2-D FFT amplitude spectrum is compared with the
    previous frame's at the same position (cosine, Eq. 3-3 per token), and every token
    whose similarity reaches the fixed threshold tau is reused -- no alignment, no
    refresh, no adaptive budget and no migration gate.  A missing previous frame is an
    all-zero frame (similarity 0: nothing is reused)."""
    y_cur = luma(cur)
    y_prev = luma(prev) if prev is not None else np.zeros_like(y_cur)
    a_cur = token_view(patch_amplitude(patches(y_cur, patch)), merge)
    a_prev = token_view(patch_amplitude(patches(y_prev, patch)), merge)
    gh, gw = a_cur.shape[:2]
    sim = np.zeros((gh, gw))
    for i in range(gh):
        for j in range(gw):
            u = a_cur[i, j].ravel()
            v = a_prev[i, j].ravel()
            nu, nv = np.sqrt(np.sum(u * u)), np.sqrt(np.sum(v * v))
            if nu == 0.0 and nv == 0.0:
                sim[i, j] = 1.0
            elif nu > 0.0 and nv > 0.0:
                sim[i, j] = np.sum(u * v) / (nu * nv)
    reuse = (sim.ravel() >= tau).astype(np.uint8)
    return NaiveResult(reuse_mask=reuse,
                       recompute_idx=np.flatnonzero(reuse == 0).astype(np.int32),
                       sim=sim.ravel())


def select_batch(prev: np.ndarray | None, cur: np.ndarray, prm: SelectParams) -> list:
    """select_item over a [B, 3, H, W] batch."""
    return [select_item(None if prev is None else prev[b], cur[b], prm)
            for b in range(cur.shape[0])]


def decision_margins(res: SelectResult, prm: SelectParams) -> dict:
    """How close each of the oracle's decisions came to flipping (relative), for
    auditing any mismatch against the GPU: a mismatch is tolerated only where the
    oracle's own margin is below 1e-5.

      threshold  per token, |E - thr| / |thr|            (refresh rule, Eq. 4-3)
      topk       (key_(K+1) - key_K) / key_(K+1) over the sorted candidate keys
                 (the ascending top-K boundary of Algorithm 1); inf without one
      budget     |alpha N - round(alpha N)| / (alpha N)  (floor of Eq. 4-4);
                 inf for a fixed ratio
      gate       |Sim_freq - tau_mig| / tau_mig          (migration gate)
      shift      (r_1 - r_2) / |r_1| of the two largest phase-correlation values
                 (argmax of Eq. 4-1); with align_pixel the smaller of the distance of
                 each axis' d / (P m) to the nearest rounding boundary (a half-integer)
                 and (r_1 - r_far) / |r_1|, r_far the largest value outside the 3 x 3
                 neighbourhood of the peak (a flip between neighbours moves the
                 sub-pixel estimate only slightly)
      tau_sim    per token, |sim - tau_sim| / tau_sim where the similarity floor
                 is active (tau_sim > 0 and the token aligned); inf elsewhere
    """
    n = res.energy.size
    thr = res.thr
    thr_m = np.abs(res.energy - thr) / max(abs(thr), 1e-300)
    ids = np.flatnonzero(res.cand)
    keys = np.sort(res.energy[ids])
    if 0 < res.k_final < keys.size:
        a, b = keys[res.k_final - 1], keys[res.k_final]
        topk_m = (b - a) / max(abs(b), 1e-300)
    else:
        topk_m = np.inf
    an = res.alpha * n
    budget_m = abs(an - np.round(an)) / max(an, 1e-300) if prm.adaptive else np.inf
    gate_m = abs(res.sim_freq - prm.tau_mig) / prm.tau_mig
    if res.shift_px is None:
        r = np.sort(res.response.ravel())
        shift_m = (r[-1] - r[-2]) / max(abs(r[-1]), 1e-300) if r.size > 1 else np.inf
    else:
        tp = prm.patch * prm.merge
        rnd = min(abs(abs(d) / tp - np.floor(abs(d) / tp) - 0.5) for d in res.shift_px)
        resp = res.response
        h, w = resp.shape
        ki, kj = divmod(int(np.argmax(resp)), w)
        far = resp.copy()
        for a in (-1, 0, 1):
            for b in (-1, 0, 1):
                far[(ki + a) % h, (kj + b) % w] = -np.inf
        r1 = resp[ki, kj]
        far_m = (r1 - far.max()) / max(abs(r1), 1e-300) if np.isfinite(far.max()) else np.inf
        shift_m = min(rnd, far_m)
    if prm.tau_sim > 0:
        sim_m = np.where(res.aligned, np.abs(res.sim - prm.tau_sim) / prm.tau_sim, np.inf)
    else:
        sim_m = np.full(n, np.inf)
    return dict(threshold=thr_m, topk=float(topk_m), budget=float(budget_m),
                gate=float(gate_m), shift=float(shift_m), tau_sim=sim_m)
