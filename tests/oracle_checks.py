"""Independent pins of the float64 oracle.

Each check returns an error measure that must be small for a correct
oracle.  None of them re-types the oracle's own formulas: they compare with
numpy's FFT (the DFT is a special case of a library routine), closed forms of
wave optics, invariants the mathematics guarantees, a brute-force
Rayleigh-Sommerfeld sum and central finite differences.  The same checks are
run against deliberately broken copies of the oracle in
``test_oracle_mutations.py`` to show that each plausible mistake is caught.
"""

from __future__ import annotations

import numpy as np

import oracle.donn as od

LAM = 532e-9
DX = 36e-6


def rel(a, b):
    a = np.asarray(a)
    b = np.asarray(b)
    return float(np.linalg.norm((a - b).ravel()) / max(np.linalg.norm(b.ravel()), 1e-300))


def crand(g, shape):
    return g.standard_normal(shape) + 1j * g.standard_normal(shape)


# --- DFT ------------------------------------------------------------------

def dft_vs_numpy():
    g = np.random.default_rng(1)
    x = crand(g, (3, 12, 20))
    return max(rel(od.dft2(x), np.fft.fft2(x)), rel(od.idft2(x), np.fft.ifft2(x)))


def dft_delta_parseval():
    m0, m1 = 10, 16
    x = np.zeros((m0, m1), complex)
    x[3, 5] = 1.0
    k0 = np.arange(m0)[:, None]
    k1 = np.arange(m1)[None, :]
    expect = np.exp(-2j * np.pi * (3 * k0 / m0 + 5 * k1 / m1))
    e1 = rel(od.dft2(x), expect)
    g = np.random.default_rng(2)
    y = crand(g, (m0, m1))
    f = od.dft2(y)
    e2 = abs(np.sum(abs(f) ** 2) / (m0 * m1 * np.sum(abs(y) ** 2)) - 1.0)
    e3 = rel(od.idft2(od.dft2(y)), y)
    return max(e1, e2, e3)


def frequencies_vs_numpy():
    return max(float(np.max(np.abs(od.frequencies(m, DX) - np.fft.fftfreq(m, DX))))
               * DX for m in (7, 8, 64, 200, 1000))


# --- propagation invariants --------------------------------------------------

def z0_identity():
    g = np.random.default_rng(3)
    u = crand(g, (2, 24, 24))
    err = 0.0
    for approx in (od.FRESNEL, od.ANGULAR_SPECTRUM):
        for m in (24, 40):
            h = od.transfer_function(LAM, DX, 0.0, approx, m)
            err = max(err, rel(od.propagate(u, h), u))
    return err


def parseval_unpadded():
    g = np.random.default_rng(4)
    u = crand(g, (2, 32, 32))
    err = 0.0
    for approx, lam, dx, z in ((od.FRESNEL, LAM, DX, 0.3), (od.ANGULAR_SPECTRUM, 1550e-9, 8e-6, 0.05)):
        h = od.transfer_function(lam, dx, z, approx, 32)
        v = od.propagate(u, h)
        err = max(err, abs(np.sum(abs(v) ** 2) / np.sum(abs(u) ** 2) - 1.0))
    return err


def composition():
    g = np.random.default_rng(5)
    u = crand(g, (1, 128, 128))
    err = 0.0
    for approx, lam, dx in ((od.FRESNEL, LAM, DX), (od.ANGULAR_SPECTRUM, 1550e-9, 8e-6)):
        h1 = od.transfer_function(lam, dx, 0.1, approx, 128)
        h2 = od.transfer_function(lam, dx, 0.2, approx, 128)
        h3 = od.transfer_function(lam, dx, 0.3, approx, 128)
        err = max(err, rel(od.propagate(od.propagate(u, h1), h2), od.propagate(u, h3)))
    return err


def reciprocity():
    """P_{-z} undoes P_z, and P_{-z} equals the adjoint of P_z."""
    g = np.random.default_rng(6)
    u = crand(g, (2, 20, 20))
    v = crand(g, (2, 20, 20))
    err = 0.0
    for approx in (od.FRESNEL, od.ANGULAR_SPECTRUM):
        hp = od.transfer_function(LAM, DX, 0.25, approx, 20)
        hm = od.transfer_function(LAM, DX, -0.25, approx, 20)
        err = max(err, rel(od.propagate(od.propagate(u, hp), hm), u))
        err = max(err, rel(od.propagate(v, hm), od.propagate(v, hp, adjoint=True)))
    return err


def gaussian_field(m, w0_px, z, lam=LAM, dx=DX, center=None):
    """Closed-form Fresnel propagation of exp(-r^2/w0^2) to distance z (exact for the Fresnel TF)."""
    c = m / 2 if center is None else center
    yy, xx = np.meshgrid((np.arange(m) - c) * dx, (np.arange(m) - c) * dx, indexing="ij")
    r2 = xx ** 2 + yy ** 2
    w0 = w0_px * dx
    zr = np.pi * w0 * w0 / lam
    q = 1.0 + 1j * z / zr
    return np.exp(1j * 2 * np.pi / lam * z) / q * np.exp(-r2 / (w0 * w0 * q))


def fresnel_gaussian():
    m = 128
    u0 = gaussian_field(m, 4.0, 0.0)
    h = od.transfer_function(LAM, DX, 0.3, od.FRESNEL, m)
    return rel(od.propagate(u0[None], h)[0], gaussian_field(m, 4.0, 0.3))


def fresnel_gaussian_padded():
    """Same closed form with the beam inside an n=64 aperture padded to m=128."""
    n, m = 64, 128
    u0 = gaussian_field(n, 4.0, 0.0)
    h = od.transfer_function(LAM, DX, 0.1, od.FRESNEL, m)
    return rel(od.propagate(u0[None], h)[0], gaussian_field(n, 4.0, 0.1))


def fresnel_separable():
    """2-D Fresnel propagation equals 1-D propagations along x then y (times exp(jkz))."""
    g = np.random.default_rng(7)
    n = 30
    u = crand(g, (2, n, n))
    z = 0.3
    h = od.transfer_function(LAM, DX, z, od.FRESNEL, n)
    f = np.fft.fftfreq(n, DX)
    h1 = np.exp(-1j * np.pi * LAM * z * f ** 2)
    v = np.fft.ifft(np.fft.fft(u, axis=-1) * h1, axis=-1)
    v = np.fft.ifft(np.fft.fft(v, axis=-2) * h1[:, None], axis=-2)
    v = v * np.exp(1j * 2 * np.pi / LAM * z)
    return rel(od.propagate(u, h), v)


def rs_bruteforce(exact_kernel=True, smooth=True):
    """Angular spectrum vs a direct O(16^4) Rayleigh-Sommerfeld sum (Eqs. (sommerfeld), (r01))."""
    lam, dx, z = 532e-9, 4e-6, 0.01
    n, m = 16, 512
    k = 2 * np.pi / lam
    c = (n - 1) / 2
    yy, xx = np.meshgrid(np.arange(n) - c, np.arange(n) - c, indexing="ij")
    if smooth:
        u0 = np.exp(-(xx ** 2 + yy ** 2) / 9.0).astype(complex)
    else:
        u0 = crand(np.random.default_rng(8), (n, n))
    h = od.transfer_function(lam, dx, z, od.ANGULAR_SPECTRUM, m)
    v_as = od.propagate(u0[None], h)[0]
    py, px = np.meshgrid(np.arange(n), np.arange(n), indexing="ij")
    dyy = (py[:, :, None, None] - py[None, None]) * dx
    dxx = (px[:, :, None, None] - px[None, None]) * dx
    r = np.sqrt(z * z + dyy ** 2 + dxx ** 2)
    if exact_kernel:
        kern = z / (2 * np.pi) * (1.0 / r - 1j * k) * np.exp(1j * k * r) / r ** 2
    else:
        kern = z / (1j * lam) * np.exp(1j * k * r) / r ** 2
    v_bf = np.einsum("yxab,ab->yx", kern, u0) * dx * dx
    return rel(v_as, v_bf)


def fresnel_as_bound():
    """||P_F u - P_AS u|| <= max|H_F - H_AS| * ||u|| (Parseval), unpadded 200^2."""
    g = np.random.default_rng(9)
    u = crand(g, (1, 200, 200))
    hf = od.transfer_function(LAM, DX, 0.3, od.FRESNEL, 200)
    ha = od.transfer_function(LAM, DX, 0.3, od.ANGULAR_SPECTRUM, 200)
    lhs = np.linalg.norm(od.propagate(u, hf) - od.propagate(u, ha))
    bound = np.max(np.abs(hf - ha)) * np.linalg.norm(u)
    return lhs, bound


# --- network ---------------------------------------------------------------

def donn_zero_phase_gaussian():
    """phi = 0, gamma = 1: the L-layer network is one hop of (L+1)z; closed form."""
    m, L, z = 128, 2, 0.1
    amp = np.abs(gaussian_field(m, 4.0, 0.0))[None]
    phi = np.zeros((L, m, m))
    h = od.transfer_function(LAM, DX, z, od.FRESNEL, m)
    out = od.donn_forward(amp, phi, h, 1.0)
    e1 = rel(out["field"][0], gaussian_field(m, 4.0, (L + 1) * z))
    e2 = rel(out["intensity"][0], np.abs(gaussian_field(m, 4.0, (L + 1) * z)) ** 2)
    return max(e1, e2)


def donn_energy(gamma=0.8):
    g = np.random.default_rng(10)
    n, L = 24, 3
    amp = g.uniform(0, 1, (2, n, n))
    phi = g.uniform(0, 2 * np.pi, (L, n, n))
    h = od.transfer_function(LAM, DX, 0.3, od.FRESNEL, n)
    out = od.donn_forward(amp, phi, h, gamma)
    e_unpadded = abs(out["intensity"].sum() / (gamma ** (2 * L) * (amp ** 2).sum()) - 1.0)
    hp = od.transfer_function(LAM, DX, 0.3, od.FRESNEL, 2 * n)
    outp = od.donn_forward(amp, phi, hp, 1.0)
    padded_ok = outp["intensity"].sum() <= (amp ** 2).sum() * (1 + 1e-12)
    return e_unpadded, padded_ok


def readout_tiling():
    g = np.random.default_rng(11)
    i_map = g.uniform(0, 1, (3, 20, 20))
    tiles = od.Detector(5, tuple(y for y in range(0, 20, 5) for _ in range(4)),
                        tuple(x for _ in range(4) for x in range(0, 20, 5)))
    e1 = rel(od.detector_readout(i_map, tiles).sum(axis=1), i_map.sum(axis=(1, 2)))
    point = od.Detector(1, (7, 2), (3, 19))
    s = od.detector_readout(i_map, point)
    e2 = rel(s, np.stack([i_map[:, 7, 3], i_map[:, 2, 19]], axis=1))
    # a region read = sum of I on the window, written out by slicing here
    reg = od.Detector(4, (3,), (11,))
    e3 = rel(od.detector_readout(i_map, reg)[:, 0], i_map[:, 3:7, 11:15].sum(axis=(1, 2)))
    return max(e1, e2, e3)


def ce_known_values():
    loss, grad = od.softmax_cross_entropy(np.array([[0.0, np.log(2.0)]]), np.array([1]))
    e1 = abs(loss - np.log(1.5))
    e2 = float(np.max(np.abs(grad - np.array([[1 / 3, -1 / 3]]))))
    loss_u, _ = od.softmax_cross_entropy(np.full((4, 10), 3.7), np.arange(4))
    e3 = abs(loss_u - np.log(10.0))
    g = np.random.default_rng(12)
    s = g.normal(0, 3, (5, 10))
    t = g.integers(0, 10, 5)
    _, gr = od.softmax_cross_entropy(s, t)
    e4 = float(np.max(np.abs(gr.sum(axis=1))))
    return max(e1, e2, e3, e4)


def mse_known_values():
    """Equal sums give p = 1/K: loss (K-1)/K for any label, dL/dS_j =
    2/(B K) (1/K - t_j) (the softmax-Jacobian term vanishes); a dominant
    correct class gives a loss near 0."""
    b, k = 3, 10
    labels = np.array([0, 4, 9])
    loss, grad = od.mse_softmax_loss(np.full((b, k), 2.5), labels)
    t = np.zeros((b, k))
    t[np.arange(b), labels] = 1.0
    e1 = abs(loss - (k - 1) / k)
    e2 = np.abs(grad - 2.0 / (b * k) * (1.0 / k - t)).max()
    s = np.zeros((b, k))
    s[np.arange(b), labels] = 60.0
    e3 = od.mse_softmax_loss(s, labels)[0]
    return max(e1, e2, e3)


def adam_first_step():
    """With m = v = 0 the first bias-corrected step is lr * g / (|g| + eps)."""
    g = np.random.default_rng(21).normal(0, 3, (4, 5))
    phi = np.random.default_rng(22).uniform(0, 6, (4, 5))
    lr, eps = 0.5, 1e-8
    p1, m1, v1 = od.adam_update(phi, g, np.zeros_like(g), np.zeros_like(g), 1, lr=lr, eps=eps)
    return np.abs(p1 - (phi - lr * g / (np.abs(g) + eps))).max()


def adam_constant_gradient():
    """A constant gradient keeps m-hat = g and v-hat = g^2 at every step, so
    every step moves phi by lr * g / (|g| + eps)."""
    g = np.array([[2.0, -0.5, 1e-3]])
    phi = np.zeros_like(g)
    m = np.zeros_like(g)
    v = np.zeros_like(g)
    err = 0.0
    for t in range(1, 40):
        before = phi
        phi, m, v = od.adam_update(phi, g, m, v, t, lr=0.1, eps=1e-8)
        err = max(err, np.abs((before - phi) - 0.1 * g / (np.abs(g) + 1e-8)).max())
    return err


def adam_vs_torch():
    """Three steps with changing gradients agree with torch.optim.Adam (float64, CPU)."""
    import torch
    g = np.random.default_rng(23)
    phi0 = g.uniform(0, 6, (3, 4))
    grads = [g.normal(0, 1, (3, 4)) for _ in range(3)]
    p = torch.tensor(phi0.copy(), dtype=torch.float64, requires_grad=True)
    opt = torch.optim.Adam([p], lr=0.5, betas=(0.9, 0.999), eps=1e-8)
    phi, m, v = phi0, np.zeros_like(phi0), np.zeros_like(phi0)
    for t, gr in enumerate(grads, start=1):
        opt.zero_grad()
        p.grad = torch.tensor(gr, dtype=torch.float64)
        opt.step()
        phi, m, v = od.adam_update(phi, gr, m, v, t, lr=0.5)
    return np.abs(p.detach().numpy() - phi).max()


def loss_fd(loss_fn):
    g = np.random.default_rng(13)
    s = g.normal(0, 2, (4, 6))
    t = g.integers(0, 6, 4)
    _, grad = loss_fn(s, t)
    fd = np.zeros_like(s)
    eps = 1e-6
    for idx in np.ndindex(s.shape):
        sp = s.copy()
        sp[idx] += eps
        sm = s.copy()
        sm[idx] -= eps
        fd[idx] = (loss_fn(sp, t)[0] - loss_fn(sm, t)[0]) / (2 * eps)
    return rel(grad, fd)


def adjoint_dot():
    """<P u, v> = <u, P^H v> for padded and unpadded grids, both approximations."""
    g = np.random.default_rng(14)
    err = 0.0
    for approx in (od.FRESNEL, od.ANGULAR_SPECTRUM):
        for n, m in ((16, 16), (10, 16)):
            h = od.transfer_function(LAM, DX, 0.3, approx, m)
            u = crand(g, (2, n, n))
            v = crand(g, (2, n, n))
            a = np.vdot(v, od.propagate(u, h))
            b = np.vdot(od.propagate(v, h, adjoint=True), u)
            err = max(err, abs(a - b) / abs(a))
    return err


def _tiny_net(n=12, m=12, L=2, B=3, approx=None, gamma=1.0, seed=15):
    g = np.random.default_rng(seed)
    amp = g.uniform(0, 1, (B, n, n))
    phi = g.uniform(0, 2 * np.pi, (L, n, n))
    ap = od.FRESNEL if approx is None else approx
    h = od.transfer_function(LAM, DX, 0.05, ap, m)
    det = od.Detector(3, (2, 6), (1, 7))
    t = g.integers(0, 2, B)
    gi = g.standard_normal((B, n, n))
    return amp, phi, h, gamma, det, t, gi


def _loss(amp, phi, h, gamma, det, t, gi, mode):
    out = od.donn_forward(amp, phi, h, gamma, det)
    if mode == "ce":
        return od.softmax_cross_entropy(out["sums"], t)[0]
    return float(np.sum(gi * out["intensity"]))


def grad_fd(mode="ce", n=12, m=12, approx=None, gamma=1.0):
    """Central finite differences of the loss against donn_backward, every phase entry."""
    amp, phi, h, gamma, det, t, gi = _tiny_net(n=n, m=m, approx=approx, gamma=gamma)
    out = od.donn_forward(amp, phi, h, gamma, det)
    if mode == "ce":
        _, gs = od.softmax_cross_entropy(out["sums"], t)
        dphi = od.donn_backward(out, phi, h, gamma, det, grad_sums=gs)
    else:
        dphi = od.donn_backward(out, phi, h, gamma, grad_intensity=gi)
    eps = 1e-6
    fd = np.zeros_like(phi)
    for idx in np.ndindex(phi.shape):
        pp = phi.copy()
        pp[idx] += eps
        pm = phi.copy()
        pm[idx] -= eps
        fd[idx] = (_loss(amp, pp, h, gamma, det, t, gi, mode) - _loss(amp, pm, h, gamma, det, t, gi, mode)) / (2 * eps)
    return rel(dphi, fd), dphi


def global_phase_invariance():
    """The loss depends on intensities only, so sum over pixels of dL/dphi_l is 0 for each l."""
    worst = 0.0
    for mode in ("ce", "map"):
        amp, phi, h, gamma, det, t, gi = _tiny_net(n=10, m=16, L=3)
        out = od.donn_forward(amp, phi, h, gamma, det)
        if mode == "ce":
            _, gs = od.softmax_cross_entropy(out["sums"], t)
            d = od.donn_backward(out, phi, h, gamma, det, grad_sums=gs)
        else:
            d = od.donn_backward(out, phi, h, gamma, grad_intensity=gi)
        worst = max(worst, float(np.max(np.abs(d.sum(axis=(1, 2))) / np.abs(d).sum(axis=(1, 2)))))
    return worst


# --- sampled impulse response and Fraunhofer far field ----------------------

def _kernel_direct(lam, z, approx, ddy, ddx):
    """The diffraction kernels of Eqs. (fresnel) and (sommerfeld)/(r01) at one
    displacement, evaluated directly (one point at a time)."""
    k = 2.0 * np.pi / lam
    rho2 = ddy * ddy + ddx * ddx
    ekz = np.exp(1j * 2.0 * np.pi * np.fmod(z / lam, 1.0))
    if approx == od.FRESNEL_IR:
        return ekz / (1j * lam * z) * np.exp(1j * k * rho2 / (2.0 * z))
    r = np.sqrt(z * z + rho2)
    return z / (1j * lam) * ekz * np.exp(1j * k * rho2 / (r + z)) / (r * r)


def ir_linear_convolution(approx, lam=LAM, dx=DX, z=0.05, n=6, m=12):
    """The spectral hop with the sampled-kernel H equals the brute-force linear
    convolution sum_xi U(xi) h(x - xi) dx^2 of Eq. (forward_diff) on the
    aperture (m >= 2n - 1, so no displacement wraps)."""
    g = np.random.default_rng(31)
    u = crand(g, (n, n))
    h = od.transfer_function(lam, dx, z, approx, m)
    got = od.propagate(u[None], h)[0]
    ref = np.zeros((n, n), complex)
    for y in range(n):
        for x in range(n):
            acc = 0.0 + 0.0j
            for eta in range(n):
                for xi in range(n):
                    acc += u[eta, xi] * _kernel_direct(lam, z, approx, (y - eta) * dx, (x - xi) * dx)
            ref[y, x] = acc * dx * dx
    return rel(got, ref)


def fresnel_ir_gaussian(lam=LAM, dx=DX, n=64, m=128, z=0.35, w0_px=6.0):
    """A Gaussian beam through the sampled Fresnel kernel against the
    closed-form Gaussian beam (tolerance: Riemann-sum and kernel-truncation
    error of the discrete convolution, about 1e-4 here)."""
    u0 = gaussian_field(n, w0_px, 0.0, lam, dx)
    ref = gaussian_field(n, w0_px, z, lam, dx)
    h = od.transfer_function(lam, dx, z, od.FRESNEL_IR, m)
    return rel(od.propagate(u0[None], h)[0], ref)


def rs_ir_paraxial_bound(lam=1550e-9, dx=8e-6, z=0.05, n=16, m=32):
    """Rayleigh-Sommerfeld against Fresnel sampled kernels: pointwise
    |h_RS/h_F - 1| <= eps = rho^2/z^2 + k rho^4/(8 z^3) (binomial expansion of
    r in Eq. (r01) and the r^2 -> z^2 of the denominator), so
    |U_RS - U_F| <= eps dx^2/(lambda z) sum|U|.  Returns the ratio of the
    largest difference to that bound (must be <= 1) and the size of the
    difference relative to the field (must not vanish: the kernels differ)."""
    g = np.random.default_rng(32)
    u = crand(g, (n, n))
    a = od.propagate(u[None], od.transfer_function(lam, dx, z, od.RS_IR, m))[0]
    b = od.propagate(u[None], od.transfer_function(lam, dx, z, od.FRESNEL_IR, m))[0]
    rho2 = 2.0 * ((n - 1) * dx) ** 2
    k = 2.0 * np.pi / lam
    eps = rho2 / z ** 2 + k * rho2 ** 2 / (8.0 * z ** 3)
    bound = eps * dx * dx / (lam * z) * np.sum(np.abs(u))
    return float(np.max(np.abs(a - b)) / bound), rel(a, b)


def fresnel_ir_separable(lam=LAM, dx=DX, z=0.3, m=40):
    """The Fresnel kernel factors in x and y, so its 2-D DFT has rank one:
    H[ky,kx] H[0,0] = H[ky,0] H[0,kx]."""
    h = od.transfer_function(lam, dx, z, od.FRESNEL_IR, m)
    return rel(h * h[0, 0], np.outer(h[:, 0], h[0, :]))


def fraunhofer_vs_fresnel_sum(lam=LAM, dx=DX, m=32, n=16):
    """Expanding (x - xi)^2 in Eq. (fresnel) turns the Fresnel sum into the
    Fraunhofer sum of U(xi) exp(jk xi^2/(2z)) at the same x.  At
    z = m dx^2/lambda the Fraunhofer output pitch lambda z/(m dx) equals dx,
    so the sampled-kernel Fresnel hop and Eq. (fraunhofer) must agree exactly
    on the aperture."""
    z = m * dx * dx / lam
    g = np.random.default_rng(33)
    u = crand(g, (n, n))
    k = 2.0 * np.pi / lam
    c = (np.arange(n) - n / 2.0) * dx           # the n-window's coordinates in the centred m grid
    chirp = np.exp(1j * k * (c[:, None] ** 2 + c[None, :] ** 2) / (2.0 * z))
    far = od.fraunhofer((u * chirp)[None], lam, dx, z, m)[0]
    o = (m - n) // 2
    near = od.propagate(u[None], od.transfer_function(lam, dx, z, od.FRESNEL_IR, m))[0]
    return rel(far[o:o + n, o:o + n], near)


def fraunhofer_rectangle(lam=LAM, dx=DX, z=5.0, m=64, a=6, b=10):
    """Far field of a uniform a x b rectangle centred in the grid: the
    Fourier sum is a product of geometric series, |sum_i exp(-2 pi i u i / m)|
    = |sin(pi u a / m) / sin(pi u / m)|, u = k - m/2; the magnitude of
    Eq. (fraunhofer) is that product times dx^2/(lambda z)."""
    n = max(a, b) + (max(a, b) % 2)
    u = np.zeros((n, n))
    oy, ox = (n - a) // 2, (n - b) // 2
    u[oy:oy + a, ox:ox + b] = 1.0
    got = np.abs(od.fraunhofer(u[None], lam, dx, z, m)[0])

    def dirichlet(cnt):
        v = np.arange(m) - m // 2
        out = np.full(m, float(cnt))
        nz = v % m != 0
        out[nz] = np.abs(np.sin(np.pi * v[nz] * cnt / m) / np.sin(np.pi * v[nz] / m))
        return out

    ref = np.outer(dirichlet(a), dirichlet(b)) * dx * dx / (lam * z)
    return rel(got, ref)


def multichannel_grad_fd(channels=3):
    """Central finite differences of the cross-entropy of the merged sums of a
    multi-channel DONN against multichannel_backward, over every phase entry
    of every channel."""
    amp, phi, h, gamma, det, t, gi = _tiny_net(n=10, m=10, L=2, B=3)
    g = np.random.default_rng(41)
    amps = [amp] + [g.uniform(0, 1, amp.shape) for _ in range(channels - 1)]
    phis = [phi] + [g.uniform(0, 2 * np.pi, phi.shape) for _ in range(channels - 1)]

    def loss(ph):
        return od.softmax_cross_entropy(od.multichannel_forward(amps, ph, h, gamma, det)[1], t)[0]

    fwds, merged = od.multichannel_forward(amps, phis, h, gamma, det)
    _, gs = od.softmax_cross_entropy(merged, t)
    grads = od.multichannel_backward(fwds, phis, h, gamma, det, gs)
    eps = 1e-6
    worst = 0.0
    for c in range(channels):
        fd = np.zeros_like(phis[c])
        for idx in np.ndindex(phis[c].shape):
            pp = [p.copy() for p in phis]
            pm = [p.copy() for p in phis]
            pp[c][idx] += eps
            pm[c][idx] -= eps
            fd[idx] = (loss(pp) - loss(pm)) / (2 * eps)
        worst = max(worst, rel(grads[c], fd))
    return worst


def multichannel_sums_add():
    """The merged sums are the channels' sums added, and one channel is the plain network."""
    amp, phi, h, gamma, det, t, gi = _tiny_net(n=10, m=12, L=2, B=2)
    g = np.random.default_rng(42)
    amps = [amp, g.uniform(0, 1, amp.shape)]
    phis = [phi, g.uniform(0, 2 * np.pi, phi.shape)]
    _, merged = od.multichannel_forward(amps, phis, h, gamma, det)
    parts = [od.detector_readout(od.intensity(od.donn_forward(a, p, h, gamma)["field"]), det) for a, p in zip(amps, phis)]
    one = od.multichannel_forward(amps[:1], phis[:1], h, gamma, det)[1]
    return max(rel(merged, parts[0] + parts[1]), rel(one, od.donn_forward(amp, phi, h, gamma, det)["sums"]))


# --- codesign layer (Gumbel-Softmax over device levels) ---------------------

def _codesign_case(K=16, shape=(3, 5), seed=51):
    g = np.random.default_rng(seed)
    logits = g.standard_normal(shape + (K,))
    u = g.uniform(1e-12, 1.0, shape + (K,))
    noise = -np.log(-np.log(u))
    levels = np.sort(g.uniform(0.0, 2.0 * np.pi, K))
    return logits, noise, levels


def codesign_limits():
    """Uniform scores give the mean level; a low temperature gives the level
    of the largest score (the hard layer); the soft phase stays in the
    levels' range; the gradient over the K scores of a pixel sums to zero
    (softmax is invariant to a common shift)."""
    logits, noise, levels = _codesign_case()
    e1 = abs(od.codesign_phase(np.zeros(8), np.zeros(8), levels[:8], 1.0)[0] - np.mean(levels[:8]))
    soft, _ = od.codesign_phase(logits, noise, levels, 1e-4)
    hard, _ = od.codesign_phase(logits, noise, levels, 1.0, hard=True)
    e2 = float(np.max(np.abs(soft - hard)))
    phi, w = od.codesign_phase(logits, noise, levels, 0.7)
    e3 = float(max(0.0, levels.min() - phi.min(), phi.max() - levels.max()))
    gl = od.codesign_backward(w, levels, 0.7, np.ones(phi.shape))
    e4 = float(np.max(np.abs(gl.sum(axis=-1))))
    return max(e1, e2, e3, e4)


def codesign_hard_near_ties():
    """The hard choice is the device's float32 decision (reading R10): scores
    that differ below float32 resolution tie, and the first level wins.  The
    expected levels are worked out by hand from float32 rounding:
      - logits (1, 1), noise (0, 2^-30): 1 + 2^-30 rounds to 1 in float32 (ulp
        2^-23), so the scores tie and level 0 wins, where the float64 sums
        would pick level 1;
      - logits (1, 1), noise (0, 2^-22): 1 + 2^-22 is a float32 number, level 1;
      - logits (0.5, 0.5, 0.5), noise (0, 0, 0): an exact three-way tie, level 0;
      - logits (-3, 2, 2 + 2^-21), noise (0, 0, 0): level 2 by one float32 step.
    Returns the number of wrong choices."""
    levels = np.array([0.25, 1.5, 2.75])
    cases = [
        (np.array([1.0, 1.0, -9.0]), np.array([0.0, 2.0 ** -30, 0.0]), 0),
        (np.array([1.0, 1.0, -9.0]), np.array([0.0, 2.0 ** -22, 0.0]), 1),
        (np.array([0.5, 0.5, 0.5]), np.zeros(3), 0),
        (np.array([-3.0, 2.0, 2.0 + 2.0 ** -21]), np.zeros(3), 2),
    ]
    wrong = 0
    for logits, noise, k in cases:
        phi, _ = od.codesign_phase(logits, noise, levels, 1.0, hard=True)
        wrong += int(float(phi) != levels[k])
    return wrong


def codesign_grad_fd(tau=0.7):
    """Central finite differences of L = sum c * phi against codesign_backward."""
    logits, noise, levels = _codesign_case(K=6, shape=(2, 3))
    c = np.random.default_rng(52).standard_normal((2, 3))
    _, w = od.codesign_phase(logits, noise, levels, tau)
    got = od.codesign_backward(w, levels, tau, c)
    eps = 1e-6
    fd = np.zeros_like(logits)
    for idx in np.ndindex(logits.shape):
        lp = logits.copy()
        lm = logits.copy()
        lp[idx] += eps
        lm[idx] -= eps
        fd[idx] = (np.sum(c * od.codesign_phase(lp, noise, levels, tau)[0]) -
                   np.sum(c * od.codesign_phase(lm, noise, levels, tau)[0])) / (2 * eps)
    return rel(got, fd)


# ---------------------------------------------------------------------------
# Segmentation DONN (§5.6.2): optical skip connection and layer normalisation
# ---------------------------------------------------------------------------

def _skip_case(n=12, m=12, L=2, B=3, seed=61):
    amp, phi, h, gamma, det, t, gi = _tiny_net(n=n, m=m, L=L, B=B, seed=seed)
    skip = od.encode_amplitude(amp)   # the residual reading: the input field itself
    return amp, phi, h, gamma, det, gi, skip


def skip_adds_at_detector():
    """The detector field with the skip minus the field without it is the skip
    field itself (it is added after the last hop), and with gamma = 0 (no
    light through the layers) the intensity is |skip|^2."""
    amp, phi, h, gamma, det, gi, skip = _skip_case()
    with_skip = od.donn_forward(amp, phi, h, gamma, det, skip=skip)
    without = od.donn_forward(amp, phi, h, gamma, det)
    e1 = rel(with_skip["field"] - without["field"], skip)
    dark = od.donn_forward(amp, phi, h, 0.0, det, skip=skip)
    e2 = rel(dark["intensity"], np.abs(skip) ** 2)
    return max(e1, e2)


def layer_norm_moments(eps=1e-5):
    """Each normalised map has mean 0 and variance var / (var + eps); a
    constant map normalises to zero."""
    g = np.random.default_rng(62)
    x = g.uniform(0, 3, (4, 7, 5)) ** 2
    y, mean, rstd = od.layer_norm(x, eps)
    var = x.var(axis=(1, 2))
    e_mean = np.abs(y.mean(axis=(1, 2))).max()
    e_var = rel(y.var(axis=(1, 2)), var / (var + eps))
    e_stats = max(rel(mean, x.mean(axis=(1, 2))), rel(rstd, 1.0 / np.sqrt(var + eps)))
    const, _, _ = od.layer_norm(np.full((2, 3, 3), 5.0), eps)
    return max(e_mean, e_var, e_stats, np.abs(const).max())


def layer_norm_affine_invariance():
    """With eps = 0 the normalised map does not change under x -> a x + c, a > 0."""
    g = np.random.default_rng(63)
    x = g.standard_normal((3, 6, 6))
    y0, _, _ = od.layer_norm(x, 0.0)
    y1, _, _ = od.layer_norm(2.5 * x - 7.0, 0.0)
    return rel(y1, y0)


def layer_norm_grad_fd(eps=1e-5):
    """Central finite differences of L = sum G * LN(x) against layer_norm_backward."""
    g = np.random.default_rng(64)
    x = g.uniform(0, 2, (2, 4, 5))
    G = g.standard_normal(x.shape)
    y, _, rstd = od.layer_norm(x, eps)
    dx = od.layer_norm_backward(G, y, rstd)
    h = 1e-6
    fd = np.zeros_like(x)
    for idx in np.ndindex(x.shape):
        xp = x.copy()
        xp[idx] += h
        xm = x.copy()
        xm[idx] -= h
        fd[idx] = (np.sum(G * od.layer_norm(xp, eps)[0]) - np.sum(G * od.layer_norm(xm, eps)[0])) / (2 * h)
    return rel(dx, fd)


def segmentation_grad_fd(eps=1e-5):
    """Whole segmentation training chain, L = sum G * LN(|P(U_L) + U_0|^2):
    central finite differences in every phase entry against donn_backward
    seeded with the layer norm's backward."""
    amp, phi, h, gamma, det, gi, skip = _skip_case(n=8, m=8)

    def loss(p):
        out = od.donn_forward(amp, p, h, gamma, None, skip=skip)
        return float(np.sum(gi * od.layer_norm(out["intensity"], eps)[0]))

    out = od.donn_forward(amp, phi, h, gamma, None, skip=skip)
    y, _, rstd = od.layer_norm(out["intensity"], eps)
    dphi = od.donn_backward(out, phi, h, gamma, grad_intensity=od.layer_norm_backward(gi, y, rstd))
    step = 1e-6
    fd = np.zeros_like(phi)
    for idx in np.ndindex(phi.shape):
        pp = phi.copy()
        pp[idx] += step
        pm = phi.copy()
        pm[idx] -= step
        fd[idx] = (loss(pp) - loss(pm)) / (2 * step)
    return rel(dphi, fd)
