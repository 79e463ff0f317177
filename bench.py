#!/usr/bin/env python3
"""Benchmark: BigGAN-128 G+D train step on one MI355X.

One step = one paragan_train_step call: n_D = 2 discriminator updates on
concat(real, fake) batches of 2 x 256 images and one generator update on
256 images (hinge loss; AdaBelief for G, Adam for D, the paper's asymmetric
policy), the configuration the paper trains BigGAN with at 2048 images per
step over 8 accelerators (Evaluation, Table tab:abl_study).  images/sec =
batch x steps / seconds (the generator batch, one step per generator
update).

Inputs are synthetic and seeded (real images uniform in [-1, 1], z ~ N(0, 1),
labels uniform over 1000 classes), generated on the GPU and resident in HBM
before the timed region.  Weights are random (N(0, 1/fan_in)); spectral
normalisation makes the scale immaterial.

value and ms_per_step come from the timed steps, run without
instrumentation.  The same number of steps then runs again with the
library's per-launch HIP event pairs on (profiled_ms_per_step: the events
cost the step a few percent); the kernel rates come from that pass.

The JSON line also carries:
  roofline      the dominant kernel (most GPU time in the profiled steps),
                timed live with HIP events on the library's stream:
                algorithmic FLOPs (real channels) / its launch time, against
                the bf16 dense MFMA peak;
  conv_mfma     all implicit-GEMM convolution launches together;
  bandwidth     the bandwidth-bound kernel families (SN power iteration
                and backward, weight packing, BN statistics / apply /
                backward, column sums, pooling, optimisers): algorithmic
                bytes / launch time against the 8 TB/s HBM peak (the SN and
                packing launches run on the second stream beside the
                convolutions, so theirs include waiting for CUs);
  cpu_baseline  the float64 CPU oracle timed on this host on a bounded
                sample (one train step at batch 2 on the same architecture);
  extras        the other workloads, each timed the same way after the main
                one: the BigGAN-128 discriminator step on 32 real + 32 fake
                images (paragan_d_step), the asynchronous update scheme at
                B = 256, n_D = 2 (generator batch 512, paragan_async_step),
                the BigGAN-512 train step at batch 16, n_D = 2, the main
                step fed by the host pipeline (pipeline_fed) and the main
                step with the weight gradients overlapped (overlap_wgrad).
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA (published)
PEAK_HBM_GBS = 8000.0         # MI355X HBM3E (published)

# HBM bytes per launch of a kernel, from two rocprofv3 --pmc passes over
# "bench.py --steps 1 --warmup 1 --no-cpu-baseline --no-extras --copy-probe" (FETCH_SIZE,
# then WRITE_SIZE, KiB per dispatch, averaged over the kernel's dispatches),
# each scaled by what the counter reads for the 1 GiB copy probe (FETCH_SIZE
# reads 0.5 GiB for it: x2.0; WRITE_SIZE reads 1 GiB: x1.0).  Valid only for
# the kernel source they were taken on (sha1 prefix of the file).
TRAFFIC = {
    "k_conv_halo<192x128,false>": {"fetch": 2.0 * 301623.0 * 1024, "write": 263315.0 * 1024,
                                   "source": "paragan_2411_03999_amd/csrc/convfwd.hip",
                                   "sha1": "2dcb2f927810"},
}


def traffic_of(name):
    """Measured HBM bytes per launch of kernel `name`, or None when none were
    taken or its source has changed since."""
    import hashlib
    t = TRAFFIC.get(name)
    if not t:
        return None
    with open(os.path.join(ROOT, t["source"]), "rb") as f:
        if hashlib.sha1(f.read()).hexdigest()[:12] != t["sha1"]:
            return None
    return t["fetch"] + t["write"]
METRIC = "images/sec/GPU, BigGAN-128 G+D train step; conv MFMA util % of peak"

ARCHS = {
    # img, ch, g_mult, d_mult, d_down, attn_res, n_classes, dz, shared_dim
    "biggan128": (128, 96, (16, 16, 8, 4, 2, 1), (1, 2, 4, 8, 16, 16), (1, 1, 1, 1, 1, 0), 64, 1000, 120, 128),
    "biggan512": (512, 64, (16, 16, 8, 8, 4, 2, 1, 1), (1, 1, 2, 4, 8, 8, 16, 16), (1, 1, 1, 1, 1, 1, 1, 0), 64,
                  1000, 128, 128),
}


# (lr, beta1, beta2, eps) of the generator's AdaBelief and the discriminator's Adam
OPT_G = (1e-4, 0.5, 0.999, 1e-12)
OPT_D = (4e-4, 0.0, 0.999, 1e-6)


def make_desc(lib, arch, B):
    img, ch, gm, dm, dd, attn, ncls, dz, sd = ARCHS[arch]
    d = lib.BigganDesc()
    d.img, d.ch, d.n_g, d.n_d = img, ch, len(gm) - 1, len(dm)
    for i, m in enumerate(gm):
        d.g_mult[i] = m
    for j, (m, dn) in enumerate(zip(dm, dd)):
        d.d_mult[j], d.d_down[j] = m, dn
    d.attn_res, d.n_classes, d.dz, d.shared_dim, d.B = attn, ncls, dz, sd, B
    d.n_power_iter, d.bn_eps, d.sn_eps = 1, 1e-5, 1e-12
    # the paper's asymmetric policy: AdaBelief for G, Adam for D
    d.opt_g = lib.Optim(lib.ADABELIEF, *OPT_G)
    d.opt_d = lib.Optim(lib.ADAM, *OPT_D)
    return d


def model_flops(arch):
    """Model FLOPs per image of one G fwd (g) and one D fwd (d), as the network
    defines them: 2 MACs per multiply-add of every conv and linear at its own
    resolution (G skips at the upsampled resolution, D skips conv-then-pool),
    the attention matmuls and the output conv; padding not counted.  Returns
    (g, d, conv_g, conv_d), the last two over conv layers only."""
    img, ch, gm, dm, dd, attn, ncls, dz, sd = ARCHS[arch]
    conv_g = 0.0
    H = 4
    for i in range(len(gm) - 1):
        cin, cout = gm[i] * ch, gm[i + 1] * ch
        Ho = 2 * H
        conv_g += 2.0 * Ho * Ho * cout * (9 * cin + 9 * cout + cin)
        H = Ho
    conv_g += 2.0 * img * img * 3 * 9 * gm[-1] * ch           # output conv (fp32)
    conv_d = 0.0
    H, cin = img, 3
    for m, down in zip(dm, dd):
        cout = m * ch
        skip = cin if (cin != cout or down) else 0
        conv_d += 2.0 * H * H * cout * (9 * cin + 9 * cout + skip)
        H, cin = (H // 2 if down else H), cout
    def attn_flops(c, hw):
        L = hw // 4
        return 2.0 * hw * (2 * (c // 8) * c + (c // 2) * c + c * (c // 2)) + 2.0 * hw * L * (c // 8 + c // 2)
    # attention at attn x attn: in G after the block producing that resolution, in D after the first block
    gc = [gm[i + 1] * ch for i in range(len(gm) - 1)]
    gres = [8 * 2 ** i for i in range(len(gm) - 1)]
    g = conv_g + (attn_flops(gc[gres.index(attn)], attn * attn) if attn in gres else 0.0)
    d = conv_d + attn_flops(dm[0] * ch, attn * attn)
    g += 2.0 * (dz // len(gm)) * 16 * gm[0] * ch                # z linear
    d += 2.0 * 2 * dm[-1] * ch                                  # head + projection
    return g, d, conv_g, conv_d


def device_net(torch, lib, ents, npar, nu, gen):
    """Seeded random parameters, u vectors and zeroed optimiser state on the GPU."""
    P = torch.empty(npar, dtype=torch.float32, device="cuda")
    for e in ents:
        n = 1
        for s in e["shape"]:
            n *= s
        view = P[e["offset"]:e["offset"] + n]
        name = e["name"]
        if name.endswith("gamma"):
            view.fill_(0.5)
        elif name.endswith("out_bn.gain"):
            view.fill_(1.0)
        elif len(e["shape"]) >= 2:
            fan = n // e["shape"][0]
            view.normal_(0.0, fan ** -0.5, generator=gen)
        else:
            view.normal_(0.0, 0.02, generator=gen)
    U = torch.empty(max(nu, 1), dtype=torch.float32, device="cuda").normal_(generator=gen)
    G = torch.zeros(npar, dtype=torch.float32, device="cuda")
    M = torch.zeros(npar, dtype=torch.float32, device="cuda")
    V = torch.zeros(npar, dtype=torch.float32, device="cuda")
    st = lib.NetState(P.data_ptr(), U.data_ptr(), G.data_ptr(), M.data_ptr(), V.data_ptr(), 0)
    return dict(P=P, U=U, G=G, M=M, V=V, state=st)


def timed(torch, fn, steps, warmup):
    """Milliseconds per call of fn over `steps` calls after `warmup`, on the
    device clock, bracketed by synchronisations."""
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        fn()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / steps


def extras(torch, lib, C, ctx, gen, Dn, real, labels, steps=5):
    """The discriminator step (32 + 32), the asynchronous iteration and the
    BigGAN-512 step; each from its own seeded state."""
    out = {}
    # BigGAN-128 D step on 32 real + 32 fake images
    d32 = make_desc(lib, "biggan128", 32)
    ws = lib.workspace(lib.paragan_train_step_ws_size(d32))
    xr, xf = real[0][:32].contiguous(), real[1][:32].contiguous()
    yr, yf = labels[0][:32].contiguous(), labels[1][:32].contiguous()
    loss = (C.c_float * 1)()

    def dstep():
        ctx.check(lib.paragan_d_step(ctx, d32, Dn["state"], xr, yr, xf, yf, ws, loss))
    ms = timed(torch, dstep, 4 * steps, 2)
    out["d_step_32_32"] = {"workload": "BigGAN-128 discriminator step, 32 real + 32 fake images",
                           "ms_per_step": ms, "images_per_sec": 64 / (ms / 1e3)}
    del ws
    # the asynchronous update scheme at B = 256, n_D = 2 (generator batch 512)
    B, n_D = 256, 2
    d = make_desc(lib, "biggan128", B)
    gents, gn, gnu = lib.paragan_net_layout(d, 0)
    dents, dn, dnu = lib.paragan_net_layout(d, 1)
    Ga = device_net(torch, lib, gents, gn, gnu, gen)
    Da = device_net(torch, lib, dents, dn, dnu, gen)
    z = torch.randn((n_D * B, d.dz), device="cuda", generator=gen)
    y = torch.randint(0, d.n_classes, (n_D * B,), device="cuda", generator=gen, dtype=torch.int32)
    img = torch.rand((n_D * B, d.img, d.img, 3), device="cuda", generator=gen) * 2 - 1
    lab = torch.randint(0, d.n_classes, (n_D * B,), device="cuda", generator=gen, dtype=torch.int32)
    pred = torch.empty(n_D * B, device="cuda")
    arr = lambda lst: (C.c_void_p * n_D)(*[t.data_ptr() for t in lst])
    inp = lib.AsyncInputs(arr(real[:n_D]), arr(labels[:n_D]), z.data_ptr(), y.data_ptr(), img.data_ptr(),
                          lab.data_ptr(), pred.data_ptr())
    ws = lib.workspace(lib.paragan_async_ws_size(d, n_D))
    losses = (C.c_float * (n_D + 1))()

    def astep():
        ctx.check(lib.paragan_async_step(ctx, d, Ga["state"], Da["state"], inp, n_D, ws, losses))
    ms = timed(torch, astep, steps, 1)
    out["async"] = {"workload": "BigGAN-128 asynchronous iteration: G step on 512 images against a D snapshot "
                                "(second stream) beside 2 D steps of 256 + 256 on the previous samples",
                    "ms_per_iteration": ms, "g_images_per_sec": n_D * B / (ms / 1e3),
                    "d_images_per_sec": 2 * n_D * B / (ms / 1e3)}
    del ws, Ga, Da, img
    torch.cuda.empty_cache()
    # BigGAN-512 train step at batch 16, n_D = 2
    B = 16
    d = make_desc(lib, "biggan512", B)
    gents, gn, gnu = lib.paragan_net_layout(d, 0)
    dents, dn, dnu = lib.paragan_net_layout(d, 1)
    G5 = device_net(torch, lib, gents, gn, gnu, gen)
    D5 = device_net(torch, lib, dents, dn, dnu, gen)
    keep = [torch.rand((B, d.img, d.img, 3), device="cuda", generator=gen) * 2 - 1 for _ in range(n_D)]
    keep += [torch.randint(0, d.n_classes, (B,), device="cuda", generator=gen, dtype=torch.int32)
             for _ in range(n_D)]
    keep += [torch.randn((B, d.dz), device="cuda", generator=gen) for _ in range(n_D)]
    keep += [torch.randint(0, d.n_classes, (B,), device="cuda", generator=gen, dtype=torch.int32)
             for _ in range(n_D)]
    keep += [torch.randn((B, d.dz), device="cuda", generator=gen),
             torch.randint(0, d.n_classes, (B,), device="cuda", generator=gen, dtype=torch.int32)]
    ptr = [t.data_ptr() for t in keep]
    arr = lambda lst: (C.c_void_p * n_D)(*lst)
    inp5 = lib.StepInputs(arr(ptr[0:n_D]), arr(ptr[n_D:2 * n_D]), arr(ptr[2 * n_D:3 * n_D]),
                          arr(ptr[3 * n_D:4 * n_D]), ptr[4 * n_D], ptr[4 * n_D + 1])
    ws = lib.workspace(lib.paragan_train_step_ws_size(d))

    def step5():
        ctx.check(lib.paragan_train_step(ctx, d, G5["state"], D5["state"], inp5, n_D, ws, losses))
    ms = timed(torch, step5, steps, 1)
    out["biggan512"] = {"workload": "BigGAN-512 G+D train step, batch 16, 2 D steps per G step",
                        "ms_per_step": ms, "images_per_sec": B / (ms / 1e3)}
    return out


def pipeline_fed(torch, lib, C, step, d, keep, n_D, steps=6, warmup=2):
    """The same train step with each D step's real batch arriving through the
    congestion-aware host pipeline: synthetic batches (SplitMix64) made by
    host threads into pinned slots, copied to the step's device buffers
    before each call.  Wall-clock rate, so host waits and PCIe copies count."""
    B, img = d.B, d.img
    src = lib.SynthSource()
    src.seed, src.B, src.img, src.n_classes = 2024, B, img, d.n_classes
    nbytes = lib.load().paragan_synth_batch_bytes(C.byref(src))
    nslot = 8
    slots = [torch.empty(nbytes, dtype=torch.uint8, pin_memory=True) for _ in range(nslot)]
    cfg = lib.PipelineCfg()
    # prefetch depth of at least two steps' batches, so the next step's
    # batches are made while the GPU runs this one
    cfg.min_threads, cfg.max_threads, cfg.min_depth, cfg.max_depth, cfg.window, cfg.threshold_ms = \
        1, 8, 2 * n_D, nslot, 4, 20.0
    pipe = lib.Pipeline(cfg, [t.data_ptr() for t in slots], nbytes, synth=src)
    n = B * img * img * 3

    def fed_step():
        for k in range(n_D):
            rc, seq, s = pipe.next(120000)
            if rc != lib.OK:
                raise lib.ParaganError(rc, pipe.error())
            buf = slots[s]
            keep[k].copy_(buf[:4 * n].view(torch.float32).view(B, img, img, 3), non_blocking=True)
            keep[n_D + k].copy_(buf[4 * n:4 * n + 4 * B].view(torch.int32), non_blocking=True)
            # the slot goes back to the pipeline once its copy has landed
            torch.cuda.current_stream().synchronize()
            pipe.release(s)
        step()

    try:
        for _ in range(warmup):
            fed_step()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            fed_step()
        torch.cuda.synchronize()
        secs = time.perf_counter() - t0
        st = pipe.stats()
    finally:
        pipe.close()
    return {"workload": "BigGAN-128 train step (B=256, n_D=2) with the real batches from the host pipeline "
                        "(synthetic SplitMix64 batches in pinned memory, copied to HBM before each step)",
            "images_per_sec": B * steps / secs, "ms_per_step": secs / steps * 1e3,
            "pipeline": {"threads": st["threads"], "depth": st["depth"], "grows": st["grows"],
                         "shrinks": st["shrinks"], "window_mean_ms": st["window_mean_ms"],
                         "consumer_wait_ms_total": st["consumer_wait_ms"]}}


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def cpu_baseline(arch, B=1, n_D=2):
    """Time the oracle (float64 numpy) on one train step at batch B."""
    import numpy as np
    from threadpoolctl import threadpool_info

    from oracle import biggan as O
    from paragan_2411_03999_amd.synth import Stream, init_params, init_u
    img, ch, gm, dm, dd, attn, ncls, dz, sd = ARCHS[arch]
    a = O.Arch(img, ch, gm, dm, dd, attn, ncls, dz, sd)
    s = Stream(4004)
    glay, gsn = O.g_layout(a)
    dlay, dsn = O.d_layout(a)
    gp, gu = init_params(glay, s, weights="gaussian"), init_u(glay, gsn, s)
    dp, du = init_params(dlay, s, weights="gaussian"), init_u(dlay, dsn, s)
    d_in = [(s.uniform((B, img, img, 3)), s.labels(B, ncls), s.normal((B, dz)), s.labels(B, ncls))
            for _ in range(n_D)]
    g_in = (s.normal((B, dz)), s.labels(B, ncls))
    hp = O.HParams(opt_g=O.OptSpec("adabelief", *OPT_G), opt_d=O.OptSpec("adam", *OPT_D))
    optG, optD = O.opt_init(gp), O.opt_init(dp)
    t0 = time.perf_counter()
    _, _, losses, _, _ = O.train_step(a, hp, (gp, gu), (dp, du), optG, optD, d_in, g_in)
    dt = time.perf_counter() - t0
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    return {"value": B / dt, "unit": "images/sec", "cores": int(threads), "kind": "oracle",
            "cpu_model": cpu_model(), "host_cpus": os.cpu_count(),
            "sample": "one %s G+D train step (n_D=%d) at batch %d, float64 numpy, %.1f s; finite losses: %s"
                      % (arch, n_D, B, dt, bool(np.all(np.isfinite(losses))))}


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--batch", type=int, default=256)
    ap.add_argument("--n-d", type=int, default=2)
    ap.add_argument("--arch", default="biggan128", choices=sorted(ARCHS))
    ap.add_argument("--seed", type=int, default=1004)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extras", action="store_true", help="skip the D-step, async and BigGAN-512 timings")
    ap.add_argument("--cpu-batch", type=int, default=2)
    ap.add_argument("--kernels-out", default=None, help="write the per-kernel table (JSON) here")
    ap.add_argument("--copy-probe", action="store_true",
                    help="before the timed steps, copy 1 GiB device to device once: the known-size "
                         "reference for scaling the FETCH_SIZE / WRITE_SIZE counters")
    ap.add_argument("--detail", action="store_true",
                    help="profile per GEMM shape (names carry [M,N,K]); the roofline is then per shape")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py: this build runs on one GPU only (--gpus %d requested); the multi-GPU data-parallel "
              "path is a design, not code" % args.gpus, file=sys.stderr)
        sys.exit(2)

    import ctypes as C

    import torch

    from paragan_2411_03999_amd import lib
    lib.load()
    torch.cuda.set_device(0)
    B, n_D = args.batch, args.n_d
    d = make_desc(lib, args.arch, B)
    assert lib.paragan_biggan_check(d) == lib.OK
    gen = torch.Generator(device="cuda")
    gen.manual_seed(args.seed)
    gents, gn, gnu = lib.paragan_net_layout(d, 0)
    dents, dn, dnu = lib.paragan_net_layout(d, 1)
    Gn = device_net(torch, lib, gents, gn, gnu, gen)
    Dn = device_net(torch, lib, dents, dn, dnu, gen)
    img = d.img
    keep = []
    for _ in range(n_D):
        keep.append(torch.rand((B, img, img, 3), device="cuda", generator=gen) * 2 - 1)
    for _ in range(n_D):
        keep.append(torch.randint(0, d.n_classes, (B,), device="cuda", generator=gen, dtype=torch.int32))
    for _ in range(n_D):
        keep.append(torch.randn((B, d.dz), device="cuda", generator=gen))
    for _ in range(n_D):
        keep.append(torch.randint(0, d.n_classes, (B,), device="cuda", generator=gen, dtype=torch.int32))
    keep.append(torch.randn((B, d.dz), device="cuda", generator=gen))
    keep.append(torch.randint(0, d.n_classes, (B,), device="cuda", generator=gen, dtype=torch.int32))
    ptr = [t.data_ptr() for t in keep]
    arr = lambda lst: (C.c_void_p * n_D)(*lst)
    inp = lib.StepInputs(arr(ptr[0:n_D]), arr(ptr[n_D:2 * n_D]), arr(ptr[2 * n_D:3 * n_D]),
                         arr(ptr[3 * n_D:4 * n_D]), ptr[4 * n_D], ptr[4 * n_D + 1])
    ws_bytes = lib.paragan_train_step_ws_size(d)
    ws = lib.workspace(ws_bytes)
    ctx = lib.Context()
    losses = (C.c_float * (n_D + 1))()

    def step():
        rc = lib.paragan_train_step(ctx, d, Gn["state"], Dn["state"], inp, n_D, ws, losses)
        if rc != lib.OK:
            raise lib.ParaganError(rc, lib.load().paragan_last_error(ctx.h).decode())

    print("bench: %s B=%d n_D=%d workspace %.1f GB, G %d params, D %d params"
          % (args.arch, B, n_D, ws_bytes / 2 ** 30, gn, dn), file=sys.stderr, flush=True)
    for i in range(args.warmup):
        step()
        print("bench: warmup step %d losses %s" % (i, list(losses)), file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    if args.copy_probe:
        src = torch.ones(1 << 28, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    # an event after every step as well (each step ends with its losses on
    # the host), for the spread of the step time
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    ev0.record()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step()
        evs[i].record()
    ev1.record()
    torch.cuda.synchronize()
    step_ms = sorted([ev0.elapsed_time(evs[0])] + [evs[i - 1].elapsed_time(evs[i]) for i in range(1, args.steps)])
    pct = lambda q: step_ms[min(len(step_ms) - 1, int(round(q * (len(step_ms) - 1))))]
    wall = time.perf_counter() - t0
    gpu_ms = ev0.elapsed_time(ev1)
    secs = gpu_ms / 1e3
    print("bench: %d steps in %.3f s (wall %.3f s), last losses %s" % (args.steps, secs, wall, list(losses)),
          file=sys.stderr, flush=True)
    # the same number of steps again with the library's per-launch event
    # pairs on, for the kernel rates (roofline, conv_mfma, bandwidth); the
    # events cost the step a few percent, so `value` comes from the pass above
    lib.paragan_profile(ctx, 2 if args.detail else 1)
    pe0 = torch.cuda.Event(enable_timing=True)
    pe1 = torch.cuda.Event(enable_timing=True)
    pe0.record()
    for i in range(args.steps):
        step()
    pe1.record()
    torch.cuda.synchronize()
    lib.paragan_profile(ctx, False)
    stats = lib.paragan_profile_read(ctx)
    prof_ms = pe0.elapsed_time(pe1) / args.steps
    print("bench: profiled pass %.1f ms/step, last losses %s" % (prof_ms, list(losses)), file=sys.stderr, flush=True)

    stats.sort(key=lambda s: -s["total_ms"])
    # the dominant kernel: most time among the MFMA (FLOP-tagged) launches
    dom = next(s for s in stats if s["flops"] > 0)
    achieved = dom["flops"] / (dom["total_ms"] / 1e3) / 1e12
    conv = [s for s in stats if s["name"].startswith(("k_conv_", "k_wgrad_")) and s["flops"] > 0
            and "f32mfma" not in s["name"]]
    conv_ms = sum(s["total_ms"] for s in conv)
    conv_tf = sum(s["flops"] for s in conv) / (conv_ms / 1e3) / 1e12 if conv_ms else 0.0
    all_ms = sum(s["total_ms"] for s in stats)
    bw = {}
    for s in stats:
        if s.get("bytes", 0) > 0:
            gbs = s["bytes"] / (s["total_ms"] / 1e3) / 1e9
            bw[s["name"]] = {"GB_per_s": gbs, "frac_of_hbm": gbs / PEAK_HBM_GBS,
                             "ms_per_step": s["total_ms"] / args.steps, "launches_per_step": s["launches"] / args.steps,
                             "bytes_per_launch": s["bytes"] / s["launches"]}
    if args.kernels_out:
        with open(args.kernels_out, "w") as f:
            json.dump(stats, f, indent=1)
    for s in stats[:(60 if args.detail else 16)]:
        rate = ("%8.1f TFLOP/s" % (s["flops"] / max(s["total_ms"], 1e-9) / 1e9) if s["flops"] > 0 else
                "%8.1f GB/s" % (s.get("bytes", 0) / max(s["total_ms"], 1e-9) / 1e6))
        print("bench: %-62s %6d launches %9.2f ms %s" % (s["name"], s["launches"], s["total_ms"], rate),
              file=sys.stderr)
    # model FLOPs of one step per image: G fwd in each D step and in the G
    # step, G bwd (2x fwd); D fwd+bwd on 2 images per D step, D fwd + input
    # gradient (1x fwd) in the G step
    g, dfw, conv_g, conv_d = model_flops(args.arch)
    per_img = (n_D + 3) * g + (6 * n_D + 2) * dfw
    conv_per_img = (n_D + 3) * conv_g + (6 * n_D + 2) * conv_d
    model_tf = per_img * B * args.steps / secs / 1e12
    conv_model_tf = conv_per_img * B * args.steps / (conv_ms / 1e3) / 1e12 if conv_ms else 0.0
    out = {
        "metric": METRIC,
        "value": B * args.steps / secs,
        "unit": "images/sec",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": gpu_ms / args.steps,
        "step_ms": {"median": pct(0.5), "p10": pct(0.1), "p90": pct(0.9)},
        # the second pass (same steps, per-launch event pairs on) that the
        # kernel rates below come from
        "profiled_ms_per_step": prof_ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded uniform images, N(0,1) latents, uniform labels; random weights)",
        "config": {"workload": "%s G+D train step, batch %d, %d D steps per G step, bf16 activations with fp32 "
                               "accumulation, fp32 heads" % (args.arch, B, n_D),
                   "batch": B, "n_D": n_D, "resolution": d.img},
        "roofline": {"bound": "mfma", "kernel": dom["name"], "achieved": achieved, "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": achieved / PEAK_BF16_TFLOPS, "traffic": traffic_of(dom["name"]),
                     "launches_per_step": dom["launches"] / args.steps,
                     "avg_launch_us": dom["total_ms"] / dom["launches"] * 1e3,
                     "flops_per_launch": dom["flops"] / dom["launches"]},
        "conv_mfma": {"achieved": conv_tf, "unit": "TFLOP/s", "frac_of_peak": conv_tf / PEAK_BF16_TFLOPS,
                      "share_of_profiled_time": conv_ms / max(all_ms, 1e-9),
                      "flops": "executed (the folded pool / upsample filters do fewer MACs than the model)"},
        "bandwidth": bw,
        "model": {"gflop_per_image": per_img / 1e9, "step_tflops": model_tf, "step_frac_of_peak":
                  model_tf / PEAK_BF16_TFLOPS, "conv_gflop_per_image": conv_per_img / 1e9,
                  "conv_tflops": conv_model_tf, "conv_frac_of_peak": conv_model_tf / PEAK_BF16_TFLOPS},
    }
    if not args.no_extras and args.arch == "biggan128" and B >= 32 and n_D >= 2:
        print("bench: timing the extra workloads ...", file=sys.stderr, flush=True)
        # the same step with the block backwards' weight gradients on a
        # further stream beside their data gradients (opt-in; the kernel
        # rates above are measured with it off, as they share the CUs on)
        ctx.set_overlap_wgrad(1)
        ms_ov = timed(torch, step, args.steps, 1)
        ctx.set_overlap_wgrad(0)
        overlap = {"workload": "the same train step with each block backward's weight gradients on a further "
                               "stream beside its data gradients (paragan_set_overlap_wgrad; bit-identical)",
                   "ms_per_step": ms_ov, "images_per_sec": B / (ms_ov / 1e3)}
        fed = pipeline_fed(torch, lib, C, step, d, keep, n_D)
        del ws
        torch.cuda.empty_cache()
        out["extras"] = extras(torch, lib, C, ctx, gen, Dn, keep[0:n_D], keep[n_D:2 * n_D])
        out["extras"]["pipeline_fed"] = fed
        out["extras"]["overlap_wgrad"] = overlap
        print("bench: extras %s" % json.dumps(out["extras"]), file=sys.stderr, flush=True)
    if not args.no_cpu_baseline:
        print("bench: timing the CPU oracle sample ...", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(args.arch, B=args.cpu_batch, n_D=n_D)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
