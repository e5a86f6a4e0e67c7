"""Benchmark of the PQ layer forward on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu] [--configs small_conv_n1,alexnet_fc6_n128,...]

Headline workload: the AlexNet-conv3-shaped PQ conv layer (32 x 256 x 13 x 13
-> 384 channels, 3x3, pad 1, C'_s = 4, K = 128), synthetic seeded inputs
resident in HBM before timing.  One step = one forward of the layer through
its prepared plan (qcnn_conv_plan_create once, before timing: the codebooks
and codes are the model, fixed at test time; then qcnn_plan_forward per
step), i.e. the whole hot path of a PQ conv layer: table build,
gather-accumulate and epilogue in the library's HIP kernel, and the sum of
the subspace splits.  `per_call` reports the same layer through
qcnn_conv_forward, which also re-lays the codes on every call.  Prints ONE
JSON line.

Timing: the step runs back to back for 100 ms of wall time (the GPU's
clocks settle over tens of milliseconds of load: right after an idle spell
the headline kernel runs ~14 % longer), then W untimed warm-up steps, then
K steps between two HIP events on the stream the kernels run on, with a
device synchronize on both sides; that gives `value` and `ms_per_step`.
Then max(50, K) groups of 10 steps with an event between groups give the
per-step median and minimum (`step_ms_stats`; an event between every two
steps would add ~5.6 us of idle GPU to each), and max(50, K) steps with the
library's kernel timing on
(HIP events recorded by the library on the same stream around the main
gather kernel of each call) give every launch's duration: the roofline's
`achieved` uses their mean (what a rocprofv3 kernel trace averages), and
their median and minimum are reported beside it.  When the subspaces are
split over workgroups a step also runs a split-sum kernel, outside the
kernel timing but inside the step.

Before the headline, the library's peak probes measure this device's LDS
read rate (bytes per clock per CU, and the shader clock under that load)
and HBM stream rates; `peaks` reports them beside the published figures and
the roofline also gives its fraction of the measured LDS peak.

The other four workloads (the small conv, the fc6-shaped FC layer, the
VGG-conv3-shaped conv and the AlexNet-shaped forward, with a row per layer)
are timed the same way and reported under "per_config"; `lut_build` times
the exported table of the headline layer against its HBM roofline; the CPU
baseline times the oracle on all threads and on one.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--configs", default="small_conv_n1,alexnet_fc6_n128,vgg16_conv3_n16,alexnet_n64",
                    help="extra workloads to time besides the headline (comma list, or 'none')")
    ap.add_argument("--only", default=None, help="time only this workload and exit (profiling runs)")
    return ap.parse_args()


def measured_traffic(name: str, sources, field: str = "hbm_bytes_per_launch"):
    """HBM bytes (per launch of the main kernel, or per step) from the
    committed rocprofv3 counter summary profiles/<name>_traffic.txt, or None
    when there is none or when a kernel source it was taken on has changed
    since (its sha256 is recorded in the summary)."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "%s_traffic.txt" % name)
    if not os.path.exists(path):
        return None
    fields, shas = {}, {}
    for line in open(path):
        if ":" not in line or line.startswith(" "):
            continue
        k, v = line.split(":", 1)
        k = k.strip()
        if k == "source_sha256":
            shas[sources[0]] = v.strip()
        elif k.startswith("source_sha256 "):
            shas[k.split(" ", 1)[1].strip()] = v.strip()
        else:
            fields[k] = v.strip()
    for src in sources:
        f = os.path.join(ROOT, "paper_1512_06473_amd", "csrc", src)
        if not os.path.exists(f) or shas.get(src) != hashlib.sha256(open(f, "rb").read()).hexdigest():
            return None
    try:
        return float(fields[field])
    except (KeyError, ValueError):
        return None


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the PQ forward shards over images with no exchange, so one "
              "MI355X's share is the whole measurement; --gpus %d is not supported" % args.gpus, file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_1512_06473_amd import api, workloads, workmodel
    from paper_1512_06473_amd.network import Network

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    dev = torch.device("cuda:0")

    def T(a):
        return torch.from_numpy(np.ascontiguousarray(a)).to(dev)

    def make_step(cfg, plans=True):
        """One forward of workload `cfg`: through plans prepared here, before
        any timing (plans=True), or through the per-call entry points."""
        d = workloads.generate(cfg)
        wl = d["spec"]
        if cfg == "alexnet_n64":
            net = Network(d["layers"], dev, use_plans=plans)
            x = T(d["x"])
            return (lambda: net.forward(x)), wl, d
        L = d["layers"][0]
        x, D, c = T(d["x"]), T(L["D"]), T(L["codes"])
        if L["kind"] == "conv":
            y = torch.empty((wl.N, L["spec"].Ct, api.out_size(wl.in_shape[1], L["spec"].dk, L["stride"], L["pad"]),
                             api.out_size(wl.in_shape[2], L["spec"].dk, L["stride"], L["pad"])),
                            dtype=torch.float32, device=dev)
            if plans:
                plan = api.ConvPlan(tuple(x.shape), D, c, L["stride"], L["pad"])
                return (lambda: plan(x, out=y)), wl, d
            return (lambda: api.conv_forward(x, D, c, L["stride"], L["pad"], out=y)), wl, d
        y = torch.empty((wl.N, L["spec"].Ct), dtype=torch.float32, device=dev)
        if plans:
            plan = api.FcPlan(wl.N, D, c)
            return (lambda: plan(x, out=y)), wl, d
        return (lambda: api.fc_forward(x, D, c, out=y)), wl, d

    def spin_up(step, ms):
        """Runs `step` back to back for `ms` milliseconds of wall time: under
        load the GPU's clocks take tens of milliseconds to settle (a headline
        kernel launched right after an idle spell runs ~14 % longer, falling
        over ~200 steps to its steady time)."""
        t0 = time.perf_counter()
        while (time.perf_counter() - t0) * 1e3 < ms:
            for _ in range(8):
                step()
            torch.cuda.synchronize(dev)

    def time_steps(step, steps, warmup, spin_ms=100.0):
        stream = torch.cuda.current_stream(dev)
        spin_up(step, spin_ms)
        for _ in range(warmup):
            step()
        torch.cuda.synchronize(dev)
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        t0 = time.perf_counter()
        e0.record(stream)
        for _ in range(steps):
            step()
        e1.record(stream)
        torch.cuda.synchronize(dev)
        wall = time.perf_counter() - t0
        return e0.elapsed_time(e1) / steps, wall * 1e3 / steps

    def work_of(wl):
        # per library call: a conv and its max-pool are one call whose full
        # output map never reaches HBM
        per_layer = workmodel.call_work(wl)
        tot = dict(dense_flops=0, gathers=0, lut=0, lds=0, hbm=0)
        for _, w in per_layer:
            tot["dense_flops"] += w.dense_flops
            tot["gathers"] += w.gathers
            tot["lut"] += w.lut_entries
            tot["lds"] += w.lds_bytes
            tot["hbm"] += w.hbm_bytes
        return tot

    def kernel_ms(step, steps):
        """Average duration of the main kernel of a step, from the library's
        own HIP events on the launch stream (a second pass of `steps` steps)."""
        api.timing_read()  # drop anything recorded earlier
        api.timing_enable(True)
        try:
            for _ in range(steps):
                step()
        finally:
            api.timing_enable(False)
        total, n = api.timing_read()
        return total / n, n

    def kernel_launches(step, n):
        """Per-launch durations (ms) of the main kernels of `n` back-to-back
        steps, from the library's HIP events on the launch stream."""
        api.timing_read_each(1)  # drop anything recorded earlier
        api.timing_enable(True)
        try:
            for _ in range(n):
                step()
        finally:
            api.timing_enable(False)
        return api.timing_read_each(64 * n)

    def step_times(step, n, warmup, group=10):
        """GPU time per step of `n` groups of `group` back-to-back steps (an
        event between groups: a timing event between every two steps would
        add ~5.6 us of idle GPU to each)."""
        spin_up(step, 50.0)
        for _ in range(warmup):
            step()
        torch.cuda.synchronize(dev)
        stream = torch.cuda.current_stream(dev)
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(n + 1)]
        ev[0].record(stream)
        for i in range(n):
            for _ in range(group):
                step()
            ev[i + 1].record(stream)
        torch.cuda.synchronize(dev)
        return [ev[i].elapsed_time(ev[i + 1]) / group for i in range(n)]

    def stats(xs, scale=1.0):
        a = np.asarray(xs, dtype=np.float64) * scale
        return {"mean": float(a.mean()), "median": float(np.median(a)), "min": float(a.min()), "n": int(a.size)}

    if args.only == "copy":
        # Plain device-to-device copy of a known size: the calibration run for
        # the FETCH_SIZE / WRITE_SIZE counters.
        nbytes = 256 << 20
        src = torch.ones(nbytes // 4, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        ms, _ = time_steps(lambda: dst.copy_(src), args.steps, args.warmup)
        print(json.dumps({"only": "copy", "bytes_read": nbytes, "bytes_written": nbytes, "ms_per_step": ms,
                          "GB_s": 2 * nbytes / ms / 1e6}))
        return
    def make_quant_step(name):
        """One k-means iteration (assignment then update) of the parameter
        quantizer on a dense synthetic layer of the named AlexNet shape."""
        Ct, Cs, dk, Csp, K = workloads.QUANT_LAYERS[name]
        W, D0 = workloads.random_quant(np.random.Generator(np.random.PCG64(7)), Ct, Cs, dk, Csp, K)
        Wd, D = T(W), T(D0)
        M = Cs // Csp
        codes = torch.empty((Ct, M) if dk == 1 else (Ct, dk, dk, M), dtype=torch.uint8, device=dev)
        obj = torch.empty(M, dtype=torch.float64, device=dev)
        cnt = torch.empty((M, K), dtype=torch.int32, device=dev)

        def step():
            api.pq_assign(Wd, D, codes=codes, objective=obj)
            api.pq_update(Wd, codes, D, counts=cnt)
        # HBM bytes an iteration must move: W read by both steps, the codes
        # written then read, the codebooks read and written.
        nbytes = 2 * W.nbytes + 2 * codes.numel() + 2 * D0.nbytes
        return step, nbytes, (Ct, Cs, dk, Csp, K)

    def make_ec_step():
        """One error-correction sweep over the 2304 subspaces of a 9216 -> 4096
        layer (C's = 4, K = 32) from the k-means solution, on 256 synthetic
        calibration images: S = |N(0,1)|, T = S W^T for W = 0.01 N(0,1).  Each
        call restarts from the k-means codebooks and codes (a device copy)."""
        rng = np.random.Generator(np.random.PCG64(31))
        Nimg, Cs, Ct, Csp, K = 256, 9216, 4096, 4, 32
        S = np.abs(rng.standard_normal((Nimg, Cs))).astype(np.float32)
        W = (0.01 * rng.standard_normal((Ct, Cs))).astype(np.float32)
        Sd, Td, Wd = T(S), T(S @ W.T), T(W)
        D0 = T((0.01 * rng.standard_normal((Cs // Csp, K, Csp))).astype(np.float32))
        Dk, ck, _ = api.pq_kmeans(Wd, D0, 4)
        D, c = Dk.clone(), ck.clone()
        torch.cuda.synchronize(dev)

        def step():
            D.copy_(Dk)
            c.copy_(ck)
            return api.ec_fc(Sd, Td, D, c, 1, 1)
        # HBM bytes a sweep must move: the float64 residual read and written
        # once per subspace step, plus the subspace's inputs
        M = Cs // Csp
        nbytes = M * (16.0 * Nimg * Ct + 4.0 * Nimg * Csp)
        return step, nbytes, "fc6 9216 -> 4096, C's=4, K=32, 256 images"

    def make_ecc_step():
        """One error-correction sweep over the 64 subspaces of the AlexNet conv3
        layer shape (256 -> 384, 3x3, pad 1, 13x13 maps, C's = 4, K = 128) from
        the k-means solution, on 32 synthetic calibration images: S = |N(0,1)|,
        T = the dense conv of S with W = 0.02 N(0,1).  Each call restarts from
        the k-means codebooks and codes (a device copy)."""
        rng = np.random.Generator(np.random.PCG64(37))
        Nimg, Cs, Hs, Ct, dk, Csp, K = 32, 256, 13, 384, 3, 4, 128
        S = np.abs(rng.standard_normal((Nimg, Cs, Hs, Hs))).astype(np.float32)
        Wt = (0.02 * rng.standard_normal((Ct, Cs, dk, dk))).astype(np.float32)
        Sd, Wd = T(S), T(Wt)
        Td = torch.nn.functional.conv2d(Sd, Wd, padding=1).contiguous()
        D0 = T((0.02 * rng.standard_normal((Cs // Csp, K, Csp))).astype(np.float32))
        Dk, ck, _ = api.pq_kmeans(Wd, D0, 3)
        D, c = Dk.clone(), ck.clone()
        torch.cuda.synchronize(dev)

        def step():
            D.copy_(Dk)
            c.copy_(ck)
            return api.ec_conv(Sd, Td, D, c, 1, 1, 1, 1)
        # HBM bytes a sweep must move: the float64 residual read twice (the
        # correlation pass and the update pass) and written once per subspace
        M = Cs // Csp
        nbytes = M * 24.0 * Nimg * Ct * Hs * Hs
        return step, nbytes, "conv3 256 -> 384, 3x3 p1, 13x13, C's=4, K=128, 32 images"

    def make_ecn_step():
        """Multi-layer error correction (Sec. 3.3.3) of the AlexNet conv3 ->
        conv4 -> conv5 stack (13x13 maps, 3x3, pad 1, ReLU; C's = 4, K = 128)
        on 32 synthetic images: per layer, k-means on dense synthetic weights
        W = 0.02 N(0,1), then one error-correction sweep against the original
        stack's responses, with the quantized stack's own inputs."""
        from paper_1512_06473_amd import quantize_net
        rng = np.random.Generator(np.random.PCG64(41))
        x = T(np.abs(rng.standard_normal((32, 256, 13, 13))).astype(np.float32))
        specs = []
        for Cs, Ct in ((256, 384), (384, 384), (384, 256)):
            specs.append({"kind": "conv", "stride": 1, "pad": 1, "relu": True,
                          "W": T((0.02 * rng.standard_normal((Ct, Cs, 3, 3))).astype(np.float32)),
                          "bias": T((0.01 * rng.standard_normal(Ct)).astype(np.float32)),
                          "D0": T((0.02 * rng.standard_normal((Cs // 4, 128, 4))).astype(np.float32))})
        # The original stack's responses T (the method's input): its dense
        # layers in float64 (unfold + matmul), rounded to fp32, made once.
        targets, ho = [], x
        for sp in specs:
            Wt = sp["W"].double()
            N, _, H, Wd = ho.shape
            cols = torch.nn.functional.unfold(ho.double(), 3, padding=1)
            lin = torch.matmul(Wt.reshape(Wt.shape[0], -1), cols).reshape(N, Wt.shape[0], H, Wd)
            targets.append(lin.float().contiguous())
            ho = torch.clamp_min(lin + sp["bias"].double()[None, :, None, None], 0.0).float()
        torch.cuda.synchronize(dev)
        return (lambda: quantize_net.quantize_network(x, specs, targets, sweeps=1, inner=1, kmeans_iters=3),
                "AlexNet conv3-conv5 (256->384->384->256, 3x3 p1, 13x13, C's=4, K=128), 32 images")

    if args.only == "ec_net":
        step, _ = make_ecn_step()
        ms, _ = time_steps(step, args.steps, args.warmup, 0.0)
        print(json.dumps({"only": args.only, "ms_per_step": ms}))
        return
    if args.only == "ec_conv3":
        step, nbytes, _ = make_ecc_step()
        ms, _ = time_steps(step, args.steps, args.warmup, 0.0)
        print(json.dumps({"only": args.only, "ms_per_step": ms, "hbm_bytes_per_step": nbytes}))
        return
    if args.only == "ec_fc6":
        step, nbytes, _ = make_ec_step()
        ms, _ = time_steps(step, args.steps, args.warmup, 0.0)
        print(json.dumps({"only": args.only, "ms_per_step": ms, "hbm_bytes_per_step": nbytes}))
        return
    if args.only and args.only.startswith("quant_"):
        step, nbytes, _ = make_quant_step(args.only[len("quant_"):])
        ms, _ = time_steps(step, args.steps, args.warmup)
        print(json.dumps({"only": args.only, "ms_per_step": ms, "hbm_bytes_per_step": nbytes}))
        return
    if args.only:
        if args.only == "lut_build":
            d = workloads.generate("alexnet_conv3_n32")
            xl, Dl = T(d["x"]), T(d["layers"][0]["D"])
            lut = api.lut_build(xl, Dl)
            step = lambda: api.lut_build(xl, Dl, out=lut)  # noqa: E731
        else:
            step, wl, _ = make_step(args.only)
        ms, _ = time_steps(step, args.steps, args.warmup)
        kms, kn = kernel_ms(step, args.steps)
        print(json.dumps({"only": args.only, "ms_per_step": ms, "main_kernel_us": kms * 1e3,
                          "main_kernel_launches": kn}))
        return

    # ------------------------------------------------------ measured peaks
    # The roofline denominators measured on this device: conflict-free 128-bit
    # LDS reads on every CU (with the shader clock under that load) and HBM
    # stream rates, reported beside the published figures.
    lds_peak = api.probe_lds(dev)
    hbm_peak = api.probe_hbm(2 << 30, dev)
    valu = api.probe_valu(dev)
    # The headline gather's VALU work per 1 KB table read (from its code: 300
    # plain and 132 DPP adds and 108 address multiply-adds per 108 reads).
    read_clk = (300 * valu["add_clk"] + 132 * valu["dpp_add_clk"] + 108 * valu["mad_clk"]) / 108 / 4
    peaks = {
        "lds": {"measured_bytes_per_clk_cu": lds_peak["bytes_per_clk_cu"],
                "measured_shader_clock_ghz": lds_peak["clock_ghz"],
                "measured_GB_s": lds_peak["bytes_per_s"] / 1e9,
                "spec_bytes_per_clk_cu": workmodel.LDS_READ_BYTES_PER_CLK_PER_CU,
                "spec_clock_ghz": workmodel.CLOCK_HZ / 1e9,
                "spec_GB_s": workmodel.LDS_PEAK_BPS / 1e9,
                "probe": "qcnn_probe_lds: one 1024-thread workgroup per CU, ds_read_b128 in 1 KB contiguous runs"},
        "valu": {"clk_per_wave_instr_per_simd": valu,
                 "headline_gather_cu_clk_per_read": read_clk,
                 "headline_gather_valu_bound_bytes_per_clk_cu": 1024.0 / read_clk,
                 "probe": "qcnn_probe_valu: 16 waves per CU, independent v_add_f32 / DPP v_add_f32 / v_mad_u32_u24"},
        "hbm": {"measured_read_GB_s": hbm_peak["read_bytes_per_s"] / 1e9,
                "measured_write_GB_s": hbm_peak["write_bytes_per_s"] / 1e9,
                "measured_copy_GB_s": hbm_peak["copy_bytes_per_s"] / 1e9,
                "spec_GB_s": workmodel.HBM_PEAK_BPS / 1e9,
                "probe": "qcnn_probe_hbm: 16-byte loads, stores, and both, over 2 GiB buffers"},
    }

    # ---------------------------------------------------------------- headline
    step, wl, data = make_step("alexnet_conv3_n32")
    ms, wall_ms = time_steps(step, args.steps, args.warmup)
    nl = max(50, args.steps)
    steps_ms = step_times(step, nl, 2)
    kl = kernel_launches(step, nl)
    kms = float(np.mean(kl))
    w = work_of(wl)
    sec = ms * 1e-3
    images_s = wl.N / sec
    lds_achieved = w["lds"] / (kms * 1e-3)
    traffic = measured_traffic("conv_flat_alexnet_conv3_n32", ["conv_flat.hip"])
    frac = lds_achieved / workmodel.LDS_PEAK_BPS
    line = {
        "metric": "images/s (AlexNet-conv3-shaped PQ conv layer; also effective dense GFLOP/s and LDS roofline %)",
        "value": images_s,
        "unit": "images/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (seeded |N(0,1)| activations, N(0,0.05^2) codebooks, uniform uint8 codes)",
        "config": {"workload": "alexnet_conv3_n32: PQ conv 32x256x13x13 -> 384, 3x3 s1 p1, C's=4 (M=64), K=128",
                   "global_batch": wl.N, "parallelism": "none (1 GPU)"},
        "effective_dense_gflops": w["dense_flops"] / sec / 1e9,
        "step_ms_stats": stats(steps_ms),
        "roofline": {
            "bound": "lds",
            "achieved": lds_achieved / 1e9,
            "peak": workmodel.LDS_PEAK_BPS / 1e9,
            "unit": "GB/s",
            "frac": frac,
            "traffic": traffic,
            "kernel": "conv_flat_kernel (fused table build + gather-accumulate)",
            "kernel_us": kms * 1e3,
            "kernel_us_stats": stats(kl, 1e3),
            "frac_at_median_kernel": w["lds"] / (float(np.median(kl)) * 1e-3) / workmodel.LDS_PEAK_BPS,
            "frac_at_best_kernel": w["lds"] / (float(np.min(kl)) * 1e-3) / workmodel.LDS_PEAK_BPS,
            "frac_of_measured_peak": lds_achieved / lds_peak["bytes_per_s"],
            "step_frac": w["lds"] / sec / workmodel.LDS_PEAK_BPS,
            "target_frac": 0.5,
            "target_met": bool(frac >= 0.5),
            "kernel_launches_timed": len(kl),
            "algorithmic_bytes_per_launch": w["lds"],
            "hbm_frac": w["hbm"] / (kms * 1e-3) / workmodel.HBM_PEAK_BPS,
        },
        "peaks": peaks,
        "wall_ms_per_step": wall_ms,
    }
    # The same layer through qcnn_conv_forward (codes re-laid on every call).
    pc_step, _, _ = make_step("alexnet_conv3_n32", plans=False)
    pc_ms, _ = time_steps(pc_step, args.steps, args.warmup)
    line["per_call"] = {"entry": "qcnn_conv_forward", "ms_per_step": pc_ms, "images_s": wl.N / (pc_ms * 1e-3),
                        "step_ms_stats": stats(step_times(pc_step, nl, 2))}

    # ------------------------------------------------------------ other configs
    per = {}
    extra = [] if args.configs == "none" else [c for c in args.configs.split(",") if c]
    main_kernel = {"small_conv_n1": "conv_flat", "alexnet_fc6_n128": "fc_tiled", "vgg16_conv3_n16": "conv_flat"}
    for cfg in extra:
        st, wlc, dc = make_step(cfg)
        steps = max(5, args.steps // (10 if cfg in ("vgg16_conv3_n16", "alexnet_n64") else 1))
        m, _ = time_steps(st, steps, max(2, args.warmup // 2))
        nlc = max(50, steps)
        kl = kernel_launches(st, nlc)
        per_step = max(1, len(kl) // nlc)
        wc = work_of(wlc)
        s_ = m * 1e-3
        row = {"ms_per_step": m, "images_s": wlc.N / s_, "effective_dense_gflops": wc["dense_flops"] / s_ / 1e9,
               "lds_frac": wc["lds"] / s_ / workmodel.LDS_PEAK_BPS,
               "hbm_frac": wc["hbm"] / s_ / workmodel.HBM_PEAK_BPS, "steps": steps,
               "step_ms_stats": stats(step_times(st, nlc, 1)),
               "main_kernels_ms_per_step": float(np.sum(kl)) / nlc, "main_kernel_launches_per_step": per_step}
        if cfg in main_kernel:
            row["kernel_us_stats"] = stats(kl, 1e3)
            row["kernel_lds_frac"] = wc["lds"] / (float(np.mean(kl)) * 1e-3) / workmodel.LDS_PEAK_BPS
            row["traffic"] = measured_traffic("%s_%s" % (main_kernel[cfg], cfg), [main_kernel[cfg] + ".hip"])
        if cfg == "alexnet_n64":
            # Table 1 per layer: the main kernel of every PQ layer (launch order
            # = layer order) and each layer's whole GPU time (its split-sum or
            # pooling kernels included; a pool after an unsplit conv is a layer
            # of its own).
            net = Network(dc["layers"], dev)
            xin = T(dc["x"])
            nlayers = len(net.layers)
            stream = torch.cuda.current_stream(dev)
            reps = 20
            acc = np.zeros(nlayers)
            for r in range(reps + 2):
                ev = [torch.cuda.Event(enable_timing=True) for _ in range(nlayers + 1)]
                h = xin
                ev[0].record(stream)
                for i, Lyr in enumerate(net.layers):
                    h = Lyr(h)
                    ev[i + 1].record(stream)
                torch.cuda.synchronize(dev)
                if r >= 2:
                    acc += [ev[i].elapsed_time(ev[i + 1]) for i in range(nlayers)]
            layer_ms = acc / reps
            karr = np.asarray(kl[: per_step * nlc]).reshape(nlc, per_step)
            rows, ki = [], 0
            names = {"conv": 0, "fc": 5, "pool": 0}
            cw = workmodel.call_work(wlc)
            assert [k for k, _ in cw] == [Lyr.name for Lyr in net.layers]
            for i, (kind, lw) in enumerate(cw):
                label = []
                for part in kind.split("+"):
                    names[part] += 1
                    label.append("%s%d" % (part, names[part]))
                r_ = {"layer": "+".join(label), "kind": kind, "layer_ms": float(layer_ms[i]),
                      "lds_bytes": lw.lds_bytes, "dense_flops": lw.dense_flops, "hbm_bytes": lw.hbm_bytes}
                if kind != "pool":
                    kk = karr[:, ki]
                    ki += 1
                    r_["kernel_us_stats"] = stats(kk, 1e3)
                    r_["kernel_lds_frac"] = lw.lds_bytes / (float(np.mean(kk)) * 1e-3) / workmodel.LDS_PEAK_BPS
                    r_["layer_lds_frac"] = lw.lds_bytes / (layer_ms[i] * 1e-3) / workmodel.LDS_PEAK_BPS
                else:
                    r_["layer_hbm_frac"] = lw.hbm_bytes / (layer_ms[i] * 1e-3) / workmodel.HBM_PEAK_BPS
                rows.append(r_)
            row["per_layer"] = rows
            row["traffic_per_step"] = measured_traffic("alexnet_n64", ["conv_flat.hip", "fc_tiled.hip", "glue.hip"],
                                                       "hbm_bytes_per_step")
            row["step_lds_frac"] = row["lds_frac"]
            row["target_step_lds_frac"] = 0.35
            row["target_met"] = bool(row["lds_frac"] >= 0.35)
            del net, xin, h
        per[cfg] = row
        del st
    line["per_config"] = per

    # ------------------------------------------- exported table (qcnn_lut_build)
    # The table of Sec. 3.1's test phase written to HBM for the headline
    # layer's input: N M K H W fp32 values, bound by HBM writes.
    if args.configs != "none":
        Ld = data["layers"][0]
        xl, Dl = T(data["x"]), T(Ld["D"])
        lut = api.lut_build(xl, Dl)
        nl_ = 50
        kl = kernel_launches(lambda: api.lut_build(xl, Dl, out=lut), nl_)
        wbytes = lut.numel() * 4
        rbytes = xl.numel() * 4 + Dl.numel() * 4
        km = float(np.mean(kl)) * 1e-3
        line["lut_build"] = {"table_bytes": wbytes, "input_bytes": rbytes, "kernel_us_stats": stats(kl, 1e3),
                             "hbm_write_roofline_us": wbytes / workmodel.HBM_PEAK_BPS * 1e6,
                             "hbm_frac": (wbytes + rbytes) / km / workmodel.HBM_PEAK_BPS,
                             "write_frac_of_measured_write_peak": wbytes / km / hbm_peak["write_bytes_per_s"]}
        del lut, xl, Dl

    # ---------------------------------------------- parameter quantizer (k-means)
    quant = {}
    for name in ([] if args.configs == "none" else list(workloads.QUANT_LAYERS)):
        st, nbytes, shape = make_quant_step(name)
        m, _ = time_steps(st, 20, 3)
        quant[name] = {"layer": "C_t=%d C_s=%d d_k=%d C's=%d K=%d" % shape, "ms_per_iteration": m,
                       "hbm_bytes_per_iteration": nbytes,
                       "hbm_frac": nbytes / (m * 1e-3) / workmodel.HBM_PEAK_BPS}
        del st
    line["quantizer"] = quant

    # ------------------------------------------ packed codes (Table 1 storage)
    # The same layers with their codes in the packed log2 K-bit form; the
    # forward reads the packed stream directly.  fc6 at N = 1 is where code
    # streaming dominates a step.
    packed = {}
    if args.configs != "none":
        def packed_case(cfg, n_images=None):
            d = workloads.generate(cfg)
            L = d["layers"][0]
            x = T(d["x"] if n_images is None else d["x"][:n_images])
            D, c = T(L["D"]), T(L["codes"])
            K = L["D"].shape[1]
            pc = api.pack_codes(c, K)
            Ct = L["codes"].shape[0]
            if L["kind"] == "conv":
                dk = L["codes"].shape[1]
                y = api.conv_forward(x, D, c, L["stride"], L["pad"])
                f8 = lambda: api.conv_forward(x, D, c, L["stride"], L["pad"], out=y)
                fp = lambda: api.conv_forward_packed(x, D, pc, Ct, dk, L["stride"], L["pad"], out=y)
            else:
                y = api.fc_forward(x, D, c)
                f8 = lambda: api.fc_forward(x, D, c, out=y)
                fp = lambda: api.fc_forward_packed(x, D, pc, Ct, out=y)
            m8, _ = time_steps(f8, 100, 5)
            mp, _ = time_steps(fp, 100, 5)
            return {"code_bytes": int(L["codes"].size), "packed_bytes": int(pc.numel()),
                    "bits_per_code": api.code_bits(K), "ms_byte_codes": m8, "ms_packed_codes": mp}
        packed["alexnet_conv3_n32"] = packed_case("alexnet_conv3_n32")
        packed["alexnet_fc6_n128"] = packed_case("alexnet_fc6_n128")
        packed["fc6_one_image"] = packed_case("alexnet_fc6_n128", 1)
    line["packed_codes"] = packed

    # -------------------------- error-corrected quantization of fc6 (Eq. (8)-(12))
    ecr = {}
    if args.configs != "none":
        step_ec, nbytes, meta = make_ec_step()
        times, objs = [], None
        for _ in range(3):
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record()
            objs = step_ec()
            e1.record()
            torch.cuda.synchronize(dev)
            times.append(e0.elapsed_time(e1))
        o = objs.cpu().numpy()
        ecr = {"layer": meta, "ms_per_sweep": min(times),
               "hbm_bytes_per_sweep": nbytes, "hbm_frac": nbytes / (min(times) * 1e-3) / workmodel.HBM_PEAK_BPS,
               "response_error_kmeans": float(o[0]), "response_error_after_sweep": float(o[-1])}
        del step_ec
    line["error_correction_fc"] = ecr

    # ------------------------ error-corrected quantization of conv3 (App. B)
    eccr = {}
    if args.configs != "none":
        step_ecc, nbytes, meta = make_ecc_step()
        times, objs = [], None
        for _ in range(3):
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record()
            objs = step_ecc()
            e1.record()
            torch.cuda.synchronize(dev)
            times.append(e0.elapsed_time(e1))
        o = objs.cpu().numpy()
        eccr = {"layer": meta, "ms_per_sweep": min(times), "hbm_bytes_per_sweep": nbytes,
                "hbm_frac": nbytes / (min(times) * 1e-3) / workmodel.HBM_PEAK_BPS,
                "response_error_kmeans": float(o[0]), "response_error_after_sweep": float(o[-1])}
        del step_ecc
    line["error_correction_conv"] = eccr

    # ------------------- multi-layer error correction of conv3-conv5 (Sec. 3.3.3)
    ecnr = {}
    if args.configs != "none":
        step_ecn, meta = make_ecn_step()
        times, res = [], None
        for _ in range(2):
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record()
            res = step_ecn()
            e1.record()
            torch.cuda.synchronize(dev)
            times.append(e0.elapsed_time(e1))
        ecnr = {"network": meta, "ms_per_network": min(times),
                "response_error_per_layer": [[float(r["objective"][0]), float(r["objective"][-1])] for r in res]}
        del step_ecn, res
    line["error_correction_network"] = ecnr

    # ------------------------------------------------------------ CPU baseline
    if not args.no_cpu:
        from oracle import oracle
        L = data["layers"][0]
        cpu_model = "unknown"
        try:
            for ln in open("/proc/cpuinfo"):
                if ln.startswith("model name"):
                    cpu_model = ln.split(":", 1)[1].strip()
                    break
        except OSError:
            pass
        all_threads = oracle.threads()

        def oracle_rate(threads, n_images, seconds):
            oracle.set_threads(threads)
            xs = data["x"][:n_images]
            t0 = time.perf_counter()
            reps = 0
            while True:
                oracle.conv_lut(xs, L["D"], L["codes"], L["stride"], L["pad"])
                reps += 1
                if time.perf_counter() - t0 >= seconds:
                    break
            el = time.perf_counter() - t0
            return reps * n_images / el, reps, el

        r_all, reps, el = oracle_rate(all_threads, wl.N, 10.0)
        r_one, reps1, el1 = oracle_rate(1, 4, 5.0)
        oracle.set_threads(all_threads)
        line["cpu_baseline"] = {"value": r_all, "unit": "images/s", "cores": all_threads,
                                "kind": "oracle", "cpu_model": cpu_model,
                                "sample": "%d full passes of the 32-image batch through the oracle's table path "
                                          "(float64, OpenMP over images, %d threads), %.1f s" % (reps, all_threads, el),
                                "one_thread": {"value": r_one, "unit": "images/s", "cores": 1,
                                               "sample": "%d passes of 4 of the 32 images on one thread, %.1f s"
                                                         % (reps1, el1)}}
        # the error-correction oracles on bounded samples of the same layers,
        # scaled to one sweep (their cost is linear in the subspace steps and,
        # for the conv oracle, in the images)
        if line.get("error_correction_fc"):
            from oracle import ec as OE
            rng = np.random.Generator(np.random.PCG64(31))
            Nimg, Cs, Ct, Csp, K = 256, 9216, 4096, 4, 32
            S = np.abs(rng.standard_normal((Nimg, Cs)))
            W = 0.01 * rng.standard_normal((Ct, Cs))
            Tn = S @ W.T
            D = 0.01 * rng.standard_normal((Cs // Csp, K, Csp))
            codes = rng.integers(0, K, (Ct, Cs // Csp)).astype(np.uint8)
            t0 = time.perf_counter()
            Y = OE.forward(S, D, codes)
            t_start = time.perf_counter() - t0
            steps = 8
            t0 = time.perf_counter()
            for m in range(steps):
                Sm = S[:, m * Csp:(m + 1) * Csp]
                old = Sm @ D[m][codes[:, m]].T
                D[m], codes[:, m] = OE.subspace_step(Sm, Tn - Y + old, D[m], codes[:, m], 1)
                Y = Y - old + Sm @ D[m][codes[:, m]].T
            t_step = (time.perf_counter() - t0) / steps
            line["error_correction_fc"]["cpu_oracle"] = {
                "ms_per_sweep": (t_start + (Cs // Csp) * t_step) * 1e3, "kind": "oracle",
                "sample": "the starting residual and %d of the %d subspace steps of the same layer (float64 "
                          "numpy), scaled to the sweep" % (steps, Cs // Csp)}
        if line.get("error_correction_conv"):
            from oracle import ec_conv as OC
            rng = np.random.Generator(np.random.PCG64(37))
            Ns, Nimg, Cs, Hs, Ct, dk, Csp, K = 2, 32, 256, 13, 384, 3, 4, 128
            S = np.abs(rng.standard_normal((Ns, Cs, Hs, Hs)))
            Wt = 0.02 * rng.standard_normal((Ct, Cs, dk, dk))
            D = 0.02 * rng.standard_normal((Cs // Csp, K, Csp))
            codes = rng.integers(0, K, (Ct, dk * dk)).astype(np.uint8)
            t0 = time.perf_counter()
            ss = [OC.shifted(S[:, m * Csp:(m + 1) * Csp], dk, 1, 1) for m in range(Cs // Csp)]
            Y = sum(OC.contribution(ss[m], D[m], codes) for m in range(Cs // Csp))
            t_start = time.perf_counter() - t0
            t0 = time.perf_counter()
            OC.subspace_step(ss[0], Y, D[0], codes, 1)  # any residual of the right shape times the same
            t_step = time.perf_counter() - t0
            scale = Nimg / Ns
            line["error_correction_conv"]["cpu_oracle"] = {
                "ms_per_sweep": scale * (t_start + (Cs // Csp) * t_step) * 1e3, "kind": "oracle",
                "sample": "the starting residual and one of the %d subspace steps of the same layer on %d of the "
                          "%d images (float64 numpy), scaled to the sweep and the images" % (Cs // Csp, Ns, Nimg)}
    print(json.dumps(line))


if __name__ == "__main__":
    main()
