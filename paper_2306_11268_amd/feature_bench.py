"""Timings of the features beyond the headline training step, on one GPU.

    python -m paper_2306_11268_amd.feature_bench [--steps K] [--warmup W]

One JSON line per feature: milliseconds per call from HIP events around K
calls on the launch stream, a throughput, and for the memory-bound kernels
the bytes one call must move and the rate that gives.  Inputs are the
seeded synthetic workloads; the optics are those of the workloads named.

  loss modes / optimiser (§2.1, §5.1): the training step with the paper's
      softmax-MSE loss next to the cross-entropy one (5-layer 200x200
      Fresnel, batch 500), and the Adam step over the five masks;
  other approximations (§3.1.1): one hop with the sampled Fresnel and
      Rayleigh-Sommerfeld kernels (200 in a 400-point grid, batch 64), and
      the Fraunhofer far field (512 in a 1024-point grid, batch 64);
  architectures (§5.6): the 3-channel DONN's training step (batch 500), the
      codesign layer over 5x200x200 pixels and 256 device levels, and the
      segmentation DONN's training step (5 layers on the paper's 350x350
      grid, skip field and layer norm, batch 64).
"""

from __future__ import annotations

import argparse
import json

import numpy as np


def _time(fn, steps: int, warmup: int) -> float:
    import torch

    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(steps):
        fn()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / steps


def _line(name: str, ms: float, **kw) -> dict:
    d = {"feature": name, "ms": round(ms, 4)}
    for k, v in kw.items():
        d[k] = round(v, 1) if isinstance(v, float) else v
    print(json.dumps(d), flush=True)
    return d


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=5)
    args = ap.parse_args(argv)

    import torch

    from . import binding as lb
    from . import workloads as wl

    if not torch.cuda.is_available():
        raise SystemExit("no GPU visible")
    lb.load()
    dev = lambda x: torch.from_numpy(np.ascontiguousarray(x)).cuda()  # noqa: E731
    K, W = args.steps, args.warmup

    # ---- loss modes and the optimiser (workload 3 optics, batch 500)
    w = wl.WORKLOADS[3]
    B = w.batch
    det = lb.Detector(w.detector.size, w.detector.y0, w.detector.x0)
    net = lb.Network(w.wavelength, w.pixel_pitch, w.distance, w.approx, w.n, w.n_fft, w.layers, 1.0, det)
    amp, phi = dev(wl.amplitudes(w, B)), dev(wl.phases(w))
    labels = dev(wl.labels(w, B))
    saved = net.new_saved(B)
    for kind, name in ((lb.LR_LOSS_SOFTMAX_CE, "train_step_cross_entropy"), (lb.LR_LOSS_SOFTMAX_MSE, "train_step_softmax_mse")):
        def step(kind=kind):
            s = lb.lr_donn_forward(net, amp, phi, saved=saved, sums=True)["sums"]
            _, gs = lb.lr_loss(s, labels, kind=kind, want_loss=False)
            lb.lr_donn_backward(net, phi, saved, grad_sums=gs)
        ms = _time(step, K, W)
        _line(name, ms, workload=w.name, samples_per_s=B / ms * 1e3)
    m, v = torch.zeros_like(phi), torch.zeros_like(phi)
    g = torch.ones_like(phi) * 1e-3
    p = phi.clone()
    count = p.numel()
    ms = _time(lambda: lb.lr_adam_update(p, g, m, v, 1), K, W)
    nbytes = count * 4 * 7  # read phi, g, m, v; write phi, m, v
    _line("adam_step", ms, elements=count, bytes=nbytes, gbps=nbytes / ms / 1e6)

    # ---- other approximations: one hop, batch 64
    for approx, name, lam, dx, z in ((lb.LR_FRESNEL_IR, "hop_fresnel_kernel_200_in_400", 532e-9, 36e-6, 0.3),
                                     (lb.LR_RS_IR, "hop_rayleigh_sommerfeld_kernel_200_in_400", 1550e-9, 8e-6, 0.05)):
        pnet = lb.Network(lam, dx, z, approx, 200, 400, 1)
        u = dev((np.random.default_rng(81).standard_normal((64, 200, 200)) + 0j).astype(np.complex64))
        ms = _time(lambda: lb.lr_propagate(pnet, u), K, W)
        _line(name, ms, batch=64, samples_per_s=64 / ms * 1e3)
    fnet = lb.Network(532e-9, 36e-6, 20.0, lb.LR_FRAUNHOFER, 512, 1024, 1)
    u = dev((np.random.default_rng(82).standard_normal((64, 512, 512)) + 0j).astype(np.complex64))
    ms = _time(lambda: lb.lr_propagate(fnet, u), K, W)
    _line("fraunhofer_512_in_1024", ms, batch=64, samples_per_s=64 / ms * 1e3)

    # ---- multi-channel DONN (3 channels, workload 3 optics, batch 500)
    nets = [lb.Network(w.wavelength, w.pixel_pitch, w.distance, w.approx, w.n, w.n_fft, w.layers, 1.0, det)
            for _ in range(3)]
    amps = [dev(wl.amplitudes(w, B) * (0.5 + 0.25 * c)) for c in range(3)]
    phis = [dev(wl.phases(w)[::-1].copy() if c else wl.phases(w)) for c in range(3)]
    saveds = [n_.new_saved(B) for n_ in nets]
    ms = _time(lambda: lb.multichannel_train_step(nets, amps, phis, saveds, labels), K, W)
    _line("multichannel_3_train_step", ms, workload=w.name, samples_per_s=B / ms * 1e3)

    # ---- codesign layer: 5 x 200 x 200 pixels, 256 levels
    lev = 256
    shape = (w.layers, w.n, w.n)
    levels = dev(wl.device_levels(3, lev))
    scores = dev(wl.codesign_scores(3, shape, lev))
    noise = dev(wl.gumbel_draws(3, shape, lev))
    px = int(np.prod(shape))
    ms = _time(lambda: lb.lr_codesign_phase(scores, noise, levels, 0.5), K, W)
    nbytes = px * lev * 8 + px * 4
    _line("codesign_phase_256_levels", ms, pixels=px, bytes=nbytes, gbps=nbytes / ms / 1e6)
    gphi = torch.ones(shape, dtype=torch.float32, device="cuda")
    ms = _time(lambda: lb.lr_codesign_backward(scores, noise, levels, 0.5, gphi), K, W)
    nbytes = px * lev * 12 + px * 4
    _line("codesign_backward_256_levels", ms, pixels=px, bytes=nbytes, gbps=nbytes / ms / 1e6)

    # ---- segmentation DONN: 5 layers on the 350 x 350 grid, batch 64
    ws = wl.scaled(wl.WORKLOADS[3], n=350)
    Bs = 64
    snet = lb.Network(ws.wavelength, ws.pixel_pitch, ws.distance, ws.approx, ws.n, ws.n_fft, ws.layers, 1.0, None)
    samp = wl.amplitudes(ws, Bs)
    a_s, p_s = dev(samp), dev(wl.phases(ws))
    skip = dev(samp.astype(np.complex64))
    G = dev(np.random.default_rng(83).standard_normal((Bs, 350, 350)).astype(np.float32))
    s_saved = snet.new_saved(Bs)

    def seg_step():
        out = lb.lr_donn_forward(snet, a_s, p_s, saved=s_saved, sums=False, intensity=True, skip=skip)
        y, st = lb.lr_layer_norm(out["intensity"])
        gi = lb.lr_layer_norm_backward(G, y, st)
        lb.lr_donn_backward(snet, p_s, s_saved, grad_intensity=gi, skip=skip)

    ms = _time(seg_step, K, W)
    _line("segmentation_350_train_step", ms, batch=Bs, samples_per_s=Bs / ms * 1e3)
    inten = torch.rand((Bs, 350, 350), device="cuda")
    ms = _time(lambda: lb.lr_layer_norm(inten), K, W)
    nbytes = Bs * 350 * 350 * 12
    _line("layer_norm_350_b64", ms, bytes=nbytes, gbps=nbytes / ms / 1e6)


if __name__ == "__main__":
    main()
