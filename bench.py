#!/usr/bin/env python3
"""Throughput of the DeRF render path on one MI355X.

A step is one full render of a frame through the whole path -- sample and
encode, nearest-site assignment, per-head bucketing, grouped per-head MLP,
segment integration and Painter's merge -- with the rays already resident in
HBM.  The default workload is the paper-shaped headline frame: 504x378
forward-facing rays, 192 stratified samples per ray, 16 Voronoi heads of
8x128 (bf16 operands, fp32 accumulate).

Prints one JSON line (the last line on stdout).  `value` is rays/s over the
timed steps.  `roofline` rates the dominant kernel (the grouped MLP) with
algorithmic FLOPs (no padding) over its average duration, measured with HIP
events on the render's stream inside the timed region.  `cpu_baseline` times
the CPU oracle on a bounded ray sample of the same frame.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_TFLOPS = {"bf16": 2500.0, "fp32": 157.3}  # MI355X dense matrix peaks
PEAK_HBM_GBPS = 8000.0
METRIC = "rays/sec on 1 MI355X (504x378, 192 spp, K=16); MFMA util % of bf16 peak"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def workload_text(cfg, precision):
    a = cfg.arch
    rgb = ("%d->%d->3" % (a.width + a.dir_dim, a.rgb_hidden)) if a.rgb_hidden else (
        "%d->3" % (a.width + a.dir_dim))
    fine = (" + %d inverse-CDF fine (coarse outputs reused)" % cfg.n_fine) if cfg.n_fine else ""
    return ("%s: %dx%d %s rays, %d stratified%s samples/ray on [%g,%g], K=%d Voronoi heads of "
            "%dx%d (posenc L=%d, skip@%d, rgb %s), %s"
            % (cfg.name, cfg.width, cfg.height,
               "forward-facing NDC" if cfg.camera == "forward" else "object-centric",
               cfg.n_coarse, fine, cfg.near, cfg.far, cfg.num_sites, a.depth, a.width,
               a.pos_freqs, a.skip_layer, rgb, precision))


def kernel_source_hash():
    """Hash of the MLP kernel's source with comments and whitespace removed:
    a code change alters it, an edit of comments does not."""
    import hashlib
    import re
    text = "".join(open(os.path.join(ROOT, "paper_2011_12490_amd", "csrc", f)).read()
                   for f in ("mlp_kernel.h", "mlp_8x128.hip"))
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    text = re.sub(r"\s+", " ", text)
    return hashlib.sha256(text.encode()).hexdigest()[:16]


def measured_traffic():
    """HBM bytes per MLP launch from the committed counter summary, or None
    when the kernel code has changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", "mlp_kernel_derf_k16_hbm_counters.md")
    try:
        line = [l for l in open(path) if l.startswith("traffic-json:")][0]
        rec = json.loads(line.split(":", 1)[1])
        if kernel_source_hash() != rec["source_code_hash"]:
            return None
        return rec["traffic_bytes"]
    except (OSError, IndexError, ValueError, KeyError):
        return None


def cpu_baseline(sc, n_rays, nthreads):
    """The oracle timed on a seeded ray subset of the frame; also returns the
    subset's ids and the oracle's outputs (for the parity record)."""
    import numpy as np
    import oracle
    from paper_2011_12490_amd import scenes
    cfg = sc.cfg
    ids = scenes.ray_subset(n_rays, cfg.num_rays)
    t0 = time.perf_counter()
    ref = oracle.render(sc.sites, cfg.arch, sc.weights, sc.rays_o[ids], sc.rays_d[ids], cfg.near,
                        cfg.far, cfg.n_coarse, cfg.n_fine, seed=scenes.SEED_RENDER, ray_ids=ids,
                        nthreads=nthreads)
    dt = time.perf_counter() - t0
    # one thread on a sixteenth of the sample (about the same wall time)
    ids1 = ids[::16]
    t1 = time.perf_counter()
    oracle.render(sc.sites, cfg.arch, sc.weights, sc.rays_o[ids1], sc.rays_d[ids1], cfg.near,
                  cfg.far, cfg.n_coarse, cfg.n_fine, seed=scenes.SEED_RENDER, ray_ids=ids1,
                  nthreads=1)
    dt1 = time.perf_counter() - t1
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"value": len(ids) / dt, "unit": "rays/s", "cores": nthreads, "kind": "oracle",
            "sample": "%d seeded rays of the same frame (%d head evaluations, fp64 heads), %.1f s"
                      % (len(ids), len(ids) * (cfg.n_coarse + cfg.n_fine), dt),
            "cpu_model": model,
            "single_thread": {"value": len(ids1) / dt1, "unit": "rays/s",
                              "sample": "%d of those rays, %.1f s" % (len(ids1), dt1)}}, ids, ref


def parity_record(sc, precision, out, ids, ref, nthreads):
    """Parity of the benchmarked frame against the oracle, outside the timed
    region: the cells of every sample of the frame (a debug render that
    returns each sample's depth and cell; the oracle assigns the same depths,
    in blocks of rays) -- bit-exact except within 1e-5 of a bisector, whose
    count is reported -- and the largest pixel differences on the seeded ray
    subset the CPU baseline rendered (ids, ref; None without it)."""
    import numpy as np
    import torch
    import oracle
    from paper_2011_12490_amd import derf, scenes
    cfg = sc.cfg
    R, N = cfg.num_rays, cfg.n_coarse + cfg.n_fine
    rec = {"samples": R * N}
    o = torch.from_numpy(sc.rays_o).cuda()
    d = torch.from_numpy(sc.rays_d).cuda()
    cell = torch.empty((R, N), dtype=torch.int32, device="cuda")
    t = torch.empty((R, N), dtype=torch.float32, device="cuda")
    res = (torch.empty((R, 3), device="cuda"), torch.empty(R, device="cuda"),
           torch.empty(R, device="cuda"))
    r = derf.Renderer(sc.sites, cfg.arch, sc.weights, precision)
    derf.derf_render(r.handle, o, d, cfg.near, cfg.far,
                     derf.derf_sampling(cfg.n_coarse, cfg.n_fine, scenes.SEED_RENDER, 1, 0), *res,
                     debug=derf.derf_debug_out(derf._dptr(cell), derf._dptr(t), None, None))
    torch.cuda.synchronize()
    st = derf.derf_get_stats(r.handle)
    r.close()
    # the debug render is the benchmarked render: same outputs, bit for bit
    rec["debug_render_equals_timed"] = all(bool(torch.equal(a, b)) for a, b in zip(res, out))
    cell_h, t_h = cell.cpu().numpy(), t.cpu().numpy()
    del cell, t, res
    near = mism = unexplained = 0
    depths_exact = True
    block = max(1, (1 << 24) // N)
    for a in range(0, R, block):
        b = min(R, a + block)
        if cfg.n_fine == 0:
            # single pass: the stratified depths themselves are bit-exact too
            t_ref, c_ref, m = oracle.sample_assign(sc.sites, sc.rays_o[a:b], sc.rays_d[a:b],
                                                   cfg.near, cfg.far, N, scenes.SEED_RENDER,
                                                   ray_offset=a, margin=True, nthreads=nthreads)
            depths_exact = depths_exact and bool(np.array_equal(t_ref, t_h[a:b]))
        else:
            c_ref, m = oracle.assign_depths(sc.sites, sc.rays_o[a:b], sc.rays_d[a:b], t_h[a:b],
                                            margin=True, nthreads=nthreads)
        nb = m < 1e-5
        diff = c_ref != cell_h[a:b]
        near += int(nb.sum())
        mism += int(diff.sum())
        unexplained += int((diff & ~nb).sum())
    rec.update({"cells": "every sample of the frame, at the GPU's depths",
                "depths_bit_exact": depths_exact if cfg.n_fine == 0 else None,
                "near_bisector_samples": near, "cell_mismatches": mism,
                "mismatches_off_bisector": unexplained,
                "walk_fallback_rays": int(st.walk_fallback_rays)})
    if ids is not None:
        g = [x.cpu().numpy()[ids] for x in out]
        rec.update({"pixel_rays": int(len(ids)),
                    "max_abs_rgb": float(np.abs(g[0] - ref.rgb).max()),
                    "max_abs_depth": float(np.abs(g[1] - ref.depth).max()),
                    "max_abs_opacity": float(np.abs(g[2] - ref.opacity).max()),
                    "tol": 2e-2 if precision == "bf16" else 1e-4})
    return rec


def mfma_ceiling(iters=12000):
    """Throughput of back-to-back 32x32x16 bf16 MFMAs on every SIMD (two waves
    each, four independent accumulator chains per wave) for operand patterns
    random / constant / zero / random A with equal B columns (samples alike)
    and 0, 2 or 4 bf16-pack + packed-max vector
    instructions beside each MFMA (the head MLP's epilogue mix): the clock-
    and power-limited ceiling against which the MLP's fraction of the
    nominal 2.5 PFLOP/s is read.  Timed with events on torch's stream, which
    the probe is launched on."""
    import ctypes
    import torch
    from paper_2011_12490_amd import build as hipbuild
    if not os.path.exists(hipbuild.PROBE_LIB):
        raise SystemExit("libderf_probe.so is not built (run __graft_entry__.build())")
    L = ctypes.CDLL(hipbuild.PROBE_LIB)
    L.derf_probe_mfma.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_uint, ctypes.c_int,
                                  ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]
    L.derf_probe_mfma.restype = ctypes.c_int
    chains = L.derf_probe_chains()
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    grid = 2 * cus
    out = torch.empty(grid * 256, device="cuda")
    stream = torch.cuda.current_stream()
    res = []
    for mode, name in ((0, "random"), (1, "constant"), (2, "zero"), (3, "random, equal columns")):
        for valu in (0, 2, 4):
            def launch():
                rc = L.derf_probe_mfma(grid, iters, 1234, mode, valu, ctypes.c_void_p(out.data_ptr()),
                                       ctypes.c_void_p(stream.cuda_stream))
                if rc != 0:
                    raise RuntimeError("probe launch failed (%d)" % rc)
            launch()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for _ in range(3):
                launch()
            e1.record(stream)
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1) / 3
            flop = 2.0 * grid * 4 * iters * chains * 32 * 32 * 16
            tf = flop / (ms * 1e-3) / 1e12
            res.append({"operands": name, "valu_per_mfma": valu, "ms": ms, "tflops": tf,
                        "frac_of_peak": tf / PEAK_TFLOPS["bf16"]})
            log("bench: mfma ceiling %-8s valu %d: %.0f TFLOP/s (%.3f of peak)"
                % (name, valu, tf, tf / PEAK_TFLOPS["bf16"]))
    return res


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="derf_k16")
    ap.add_argument("--precision", default=None, choices=[None, "bf16", "fp32"])
    ap.add_argument("--sites", type=int, default=None, help="override the number of heads")
    ap.add_argument("--cpu-rays", type=int, default=24576)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-parity", action="store_true",
                    help="skip the parity record (cells of every sample and pixels of the CPU "
                         "sample against the oracle, after the timed steps)")
    ap.add_argument("--k-sweep", default=None,
                    help="comma-separated head counts: the same frame with K k-means sites each")
    ap.add_argument("--empty-heads", default=None, metavar="K1,K2,...",
                    help="mark these heads 0-capacity (empty space): never evaluated")
    ap.add_argument("--mixed", action="store_true",
                    help="heads of different capacities: head k gets the 8x128, 6x64 and 4x64 "
                         "architectures in turn (k mod 3), with their own weights")
    ap.add_argument("--soft", type=float, default=None, metavar="BETA",
                    help="also time the soft decomposition (every head on every sample) at "
                         "temperature BETA, with the per-ray head contributions")
    ap.add_argument("--gate", type=int, default=0, metavar="H",
                    help="also time the MLP-gating decomposition with a seeded gate of H "
                         "hidden units (16, 32 or 64) on the heads' position encoding")
    ap.add_argument("--cull", default=None, metavar="EPS[,LEVELS[,PIECE]]",
                    help="also time the Painter's-order render with transmittance culling "
                         "(stop below transmittance EPS, LEVELS levels, default 4; segments "
                         "cut into pieces of at most PIECE samples, default 0: whole)")
    ap.add_argument("--mfma-ceiling", action="store_true",
                    help="also run the matrix-core throughput probe (operand patterns x vector "
                         "instructions per MFMA) and report it under mfma_ceiling")
    ap.add_argument("--encoding", choices=["fused", "stored"], default="fused",
                    help="where gamma(x) is formed: inside the MLP (fused, the default) or by "
                         "its own pass into a table the MLP reads back (stored; heads without "
                         "a skip layer)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run a plain 1 GiB device copy (to scale HBM counters)")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py renders on one GPU only: the frame is not sharded across GPUs "
              "(rays are independent; see the sharding notes). Run with --gpus 1.",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2011_12490_amd import derf, scenes

    cfg = scenes.CONFIGS[args.workload]
    if args.sites is not None:
        cfg = scenes.with_changes(cfg, num_sites=args.sites)
    precision = args.precision or cfg.precision
    empty_heads = set(int(k) for k in args.empty_heads.split(",")) if args.empty_heads else set()
    head_archs = ([(scenes.ARCH_128, scenes.ARCH_SMALL, scenes.ARCH_TINY)[k % 3]
                   for k in range(cfg.num_sites)] if args.mixed else None)
    torch.cuda.set_device(0)

    def run(cfg, steps, warmup, copy_calibration=False):
        """Time `steps` renders of the workload; per-stage times from the
        library's HIP events on the render stream."""
        log("bench: building scene %s (%d rays x %d samples, K=%d, %s)"
            % (cfg.name, cfg.num_rays, cfg.n_coarse + cfg.n_fine, cfg.num_sites, precision))
        sc = scenes.make_scene(cfg)
        o = torch.from_numpy(sc.rays_o).cuda()
        d = torch.from_numpy(sc.rays_d).cuda()
        R = cfg.num_rays
        out = (torch.empty((R, 3), device="cuda"), torch.empty((R,), device="cuda"),
               torch.empty((R,), device="cuda"))
        if head_archs:
            ws = [scenes.make_weights(a, 1, seed=300 + k, sigma_bias=cfg.sigma_bias)[0]
                  for k, a in enumerate(head_archs)]
            r = derf.Renderer(sc.sites, head_archs, ws, precision)
        else:
            r = derf.Renderer(sc.sites, cfg.arch, sc.weights, precision)
        if empty_heads:
            r.set_empty_heads([k in empty_heads for k in range(cfg.num_sites)])
        if args.encoding == "stored":
            r.set_encoding(True)
        stream = torch.cuda.current_stream()

        def step():
            r.render(o, d, cfg.near, cfg.far, cfg.n_coarse, cfg.n_fine, scenes.SEED_RENDER,
                     out=out, stream=stream)

        for _ in range(warmup):
            step()
        torch.cuda.synchronize()
        log("bench: warmup done (%d steps)" % warmup)
        if copy_calibration:
            # a plain copy of known size: its FETCH_SIZE / WRITE_SIZE scale the
            # counters of the render kernels (1 GiB read + 1 GiB written)
            src = torch.ones(1 << 28, dtype=torch.float32, device="cuda")
            dst = torch.empty_like(src)
            dst.copy_(src)
            torch.cuda.synchronize()
            del src, dst
        derf.derf_reset_stats(r.handle)
        derf.derf_set_timing(r.handle, True)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            step()
        torch.cuda.synchronize()
        elapsed = time.perf_counter() - t0
        st = derf.derf_get_stats(r.handle)
        derf.derf_set_timing(r.handle, False)
        log("bench: timed %d steps in %.3f s" % (steps, elapsed))
        stage_ms = {name: st.stage_ms[i] / max(1, st.stage_launches[i])
                    for i, name in enumerate(derf.STAGE_NAMES)}
        heads = np.array(st.head_samples[:cfg.num_sites], dtype=np.int64)
        r.close()
        return sc, elapsed * 1e3 / steps, stage_ms, heads, out

    def run_soft(cfg, beta, steps, warmup):
        """Time `steps` soft-decomposition renders (with contributions)."""
        sc = scenes.make_scene(cfg)
        o = torch.from_numpy(sc.rays_o).cuda()
        d = torch.from_numpy(sc.rays_d).cuda()
        r = derf.Renderer(sc.sites, cfg.arch, sc.weights, precision)
        for _ in range(warmup):
            r.render_soft(o, d, cfg.near, cfg.far, cfg.n_coarse, beta, scenes.SEED_RENDER,
                          contrib=True)
        torch.cuda.synchronize()
        derf.derf_reset_stats(r.handle)
        derf.derf_set_timing(r.handle, True)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            r.render_soft(o, d, cfg.near, cfg.far, cfg.n_coarse, beta, scenes.SEED_RENDER,
                          contrib=True)
        torch.cuda.synchronize()
        elapsed = time.perf_counter() - t0
        st = derf.derf_get_stats(r.handle)
        stages = {name: st.stage_ms[i] / max(1, st.stage_launches[i])
                  for i, name in enumerate(derf.STAGE_NAMES) if st.stage_launches[i]}
        r.close()
        return elapsed * 1e3 / steps, stages

    def run_culled(cfg, eps, levels, piece, steps, warmup, ref_out):
        """Time `steps` culled renders; evaluated samples and the largest
        difference from the plain render's outputs ref_out."""
        sc = scenes.make_scene(cfg)
        o = torch.from_numpy(sc.rays_o).cuda()
        d = torch.from_numpy(sc.rays_d).cuda()
        r = derf.Renderer(sc.sites, cfg.arch, sc.weights, precision)
        for _ in range(warmup):
            out = r.render_culled(o, d, cfg.near, cfg.far, cfg.n_coarse, eps, levels,
                                  scenes.SEED_RENDER, piece=piece)
        torch.cuda.synchronize()
        derf.derf_reset_stats(r.handle)
        derf.derf_set_timing(r.handle, True)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            out = r.render_culled(o, d, cfg.near, cfg.far, cfg.n_coarse, eps, levels,
                                  scenes.SEED_RENDER, piece=piece)
        torch.cuda.synchronize()
        elapsed = time.perf_counter() - t0
        st = derf.derf_get_stats(r.handle)
        stages = {name: st.stage_ms[i] / max(1, st.stage_launches[i])
                  for i, name in enumerate(derf.STAGE_NAMES) if st.stage_launches[i]}
        evaluated = int(out[3].to(torch.int64).sum().item())
        diff = {"rgb": (out[0] - ref_out[0]).abs().max().item(),
                "depth": (out[1] - ref_out[1]).abs().max().item(),
                "opacity": (out[2] - ref_out[2]).abs().max().item()}
        r.close()
        return elapsed * 1e3 / steps, stages, evaluated, diff

    def run_gated(cfg, hidden, steps, warmup):
        """Time `steps` renders with the MLP-gating assignment (a seeded
        random gate on the heads' encoding; head evaluations per head and the
        mean number of one-head runs per ray come back too)."""
        sc = scenes.make_scene(cfg)
        o = torch.from_numpy(sc.rays_o).cuda()
        d = torch.from_numpy(sc.rays_d).cuda()
        L = cfg.arch.pos_freqs
        rng = np.random.Generator(np.random.PCG64(scenes.S0 + 9))
        count = derf.lib().derf_gate_weights_count(cfg.num_sites, L, hidden)
        gw = (rng.uniform(-1.0, 1.0, count) * 4.0 / np.sqrt(3 + 6 * L)).astype(np.float32)
        r = derf.Renderer(sc.sites, cfg.arch, sc.weights, precision)
        r.set_gate(L, hidden, gw)
        for _ in range(warmup):
            r.render_gated(o, d, cfg.near, cfg.far, cfg.n_coarse, scenes.SEED_RENDER)
        torch.cuda.synchronize()
        derf.derf_reset_stats(r.handle)
        derf.derf_set_timing(r.handle, True)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            r.render_gated(o, d, cfg.near, cfg.far, cfg.n_coarse, scenes.SEED_RENDER)
        torch.cuda.synchronize()
        elapsed = time.perf_counter() - t0
        st = derf.derf_get_stats(r.handle)
        stages = {name: st.stage_ms[i] / max(1, st.stage_launches[i])
                  for i, name in enumerate(derf.STAGE_NAMES) if st.stage_launches[i]}
        cell = r.render_gated(o, d, cfg.near, cfg.far, cfg.n_coarse, scenes.SEED_RENDER,
                              cells=True)[3]
        runs = float(((cell[:, 1:] != cell[:, :-1]).sum(1) + 1).double().mean().item())
        heads_g = [int(st.head_samples[k]) for k in range(cfg.num_sites)]
        r.close()
        return elapsed * 1e3 / steps, stages, runs, heads_g

    sc, ms_per_step, stage_ms, heads, frame_out = run(cfg, args.steps, args.warmup,
                                                      args.copy_calibration)
    plain_out = None
    if args.cull:
        # the plain render's outputs, for the culled render's difference
        pr = derf.Renderer(sc.sites, cfg.arch, sc.weights, precision)
        plain_out = [x.clone() for x in pr.render(torch.from_numpy(sc.rays_o).cuda(),
                                                  torch.from_numpy(sc.rays_d).cuda(), cfg.near,
                                                  cfg.far, cfg.n_coarse, cfg.n_fine,
                                                  scenes.SEED_RENDER)]
        torch.cuda.synchronize()
        pr.close()
    R = cfg.num_rays
    S = R * (cfg.n_coarse + cfg.n_fine)   # head evaluations (both passes when hierarchical)
    mlp_ms = stage_ms["mlp"]
    # head evaluations: every sample, less those owned by 0-capacity heads,
    # each at its owning head's multiply-adds
    evaluated = S - int(sum(heads[k] for k in empty_heads if k < cfg.num_sites))
    if head_archs:
        mlp_flop = 2.0 * sum(float(heads[k]) * head_archs[k].macs_per_sample()
                             for k in range(cfg.num_sites) if k not in empty_heads)
    else:
        mlp_flop = 2.0 * cfg.arch.macs_per_sample() * evaluated
    achieved = mlp_flop / (mlp_ms * 1e-3) / 1e12
    peak = PEAK_TFLOPS[precision]
    # t + cell + sigma/rgb per sample (coarse and fine lists when hierarchical), outputs per ray
    comp_bytes = 21.0 * S + 20.0 * R
    comp_gbps = comp_bytes / (stage_ms["composite"] * 1e-3) / 1e9

    k_sweep = None
    if args.k_sweep:
        k_sweep = []
        for K in [int(k) for k in args.k_sweep.split(",")]:
            ck = scenes.with_changes(cfg, num_sites=K)
            _, ms_k, st_k, heads_k, _ = run(ck, max(3, args.steps // 2), 2)
            k_sweep.append({"K": K, "rays_per_s": R / (ms_k * 1e-3), "ms_per_step": ms_k,
                            "mlp_ms": st_k["mlp"],
                            "mlp_frac": mlp_flop / (st_k["mlp"] * 1e-3) / 1e12 / peak,
                            "stage_ms": st_k,
                            "head_samples_min_max": [int(heads_k.min()), int(heads_k.max())]})
            log("bench: K=%d %.4g rays/s" % (K, k_sweep[-1]["rays_per_s"]))

    soft = None
    if args.soft is not None:
        if cfg.n_fine:
            raise SystemExit("--soft needs a single-pass workload")
        ms_s, st_s = run_soft(cfg, args.soft, max(3, args.steps // 4), 1)
        soft_flop = mlp_flop * cfg.num_sites
        soft = {"beta": args.soft, "rays_per_s": R / (ms_s * 1e-3), "ms_per_step": ms_s,
                "head_evaluations": S * cfg.num_sites, "mlp_ms": st_s["mlp"],
                "mlp_frac": soft_flop / (st_s["mlp"] * 1e-3) / 1e12 / peak, "stage_ms": st_s}
        log("bench: soft beta=%g %.4g rays/s" % (args.soft, soft["rays_per_s"]))

    culled = None
    if args.cull:
        if cfg.n_fine or head_archs or empty_heads:
            raise SystemExit("--cull needs a single-pass workload with one architecture")
        parts = args.cull.split(",")
        eps, levels = float(parts[0]), int(parts[1]) if len(parts) > 1 else 4
        piece = int(parts[2]) if len(parts) > 2 else 0
        ms_c, st_c, ev_c, diff_c = run_culled(cfg, eps, levels, piece, args.steps, 2, plain_out)
        culled = {"eps": eps, "levels": levels, "piece": piece, "rays_per_s": R / (ms_c * 1e-3),
                  "ms_per_step": ms_c, "speedup_vs_plain": ms_per_step / ms_c,
                  "evaluated_samples": ev_c, "evaluated_frac": ev_c / S,
                  "level_loop_ms": st_c.get("mlp"), "sample_ms": st_c.get("sample_assign"),
                  "max_abs_diff_vs_plain": diff_c}
        log("bench: culled eps=%g levels=%d piece=%d %.4g rays/s (%.3f of samples evaluated)"
            % (eps, levels, piece, culled["rays_per_s"], culled["evaluated_frac"]))

    gated = None
    if args.gate:
        if cfg.n_fine or head_archs or empty_heads:
            raise SystemExit("--gate needs a single-pass workload with one architecture")
        ms_g, st_g, runs_g, heads_g = run_gated(cfg, args.gate, args.steps, 2)
        gated = {"hidden": args.gate, "gate_input": "gamma_%d(x)" % cfg.arch.pos_freqs,
                 "rays_per_s": R / (ms_g * 1e-3), "ms_per_step": ms_g,
                 "vs_voronoi": ms_per_step / ms_g, "runs_per_ray": runs_g,
                 "sample_gate_ms": st_g.get("sample_assign"), "mlp_ms": st_g.get("mlp"),
                 "composite_ms": st_g.get("composite"),
                 "head_samples": {"min": min(heads_g), "max": max(heads_g)}}
        log("bench: gated H=%d %.4g rays/s (%.2f runs per ray)"
            % (args.gate, gated["rays_per_s"], runs_g))

    ceiling = mfma_ceiling() if args.mfma_ceiling else None

    cpu = None
    cpu_ids = cpu_ref = None
    nthreads = min(16, len(os.sched_getaffinity(0)))
    if not args.no_cpu_baseline:
        log("bench: timing the CPU oracle on %d rays with %d threads" % (args.cpu_rays, nthreads))
        cpu, cpu_ids, cpu_ref = cpu_baseline(sc, args.cpu_rays, nthreads)
    parity = None
    if not args.no_parity and not head_archs and not empty_heads:
        log("bench: parity record (cells of every sample, pixels of the CPU sample)")
        parity = parity_record(sc, precision, frame_out, cpu_ids, cpu_ref, nthreads)

    res = {
        "metric": METRIC,
        "value": R / (ms_per_step * 1e-3),
        "unit": "rays/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": precision,
        "data": "synthetic (seeded scene, Glorot-uniform random heads)",
        "config": {"workload": workload_text(cfg, precision), "rays": R,
                   "samples_per_ray": cfg.n_coarse + cfg.n_fine, "heads": cfg.num_sites,
                   "samples": S, "encoding": args.encoding},
        "evaluated_samples": evaluated,
        "roofline": {"bound": "mfma", "kernel": "mlp_kernel (grouped per-head MLP)",
                     "achieved": achieved, "peak": peak, "unit": "TFLOP/s",
                     "frac": achieved / peak,
                     "traffic": measured_traffic() if (cfg.name == "derf_k16" and cfg.num_sites == 16
                                                       and precision == "bf16" and not empty_heads
                                                       and not head_archs)
                     else None,
                     "flop_per_step": mlp_flop, "mlp_ms_per_step": mlp_ms,
                     "launches_per_step": 2 if cfg.n_fine else 1},
        "cpu_baseline": cpu,
        "parity": parity,
        "samples_per_s": S / (ms_per_step * 1e-3),
        "stage_ms": stage_ms,
        "composite": {"bound": "hbm", "achieved": comp_gbps, "peak": PEAK_HBM_GBPS,
                      "unit": "GB/s", "frac": comp_gbps / PEAK_HBM_GBPS,
                      "bytes_per_launch": comp_bytes},
        "head_samples": {"min": int(heads.min()), "median": float(np.median(heads)),
                         "max": int(heads.max())},
    }
    if k_sweep is not None:
        res["k_sweep"] = k_sweep
    if soft is not None:
        res["soft"] = soft
    if culled is not None:
        res["culled"] = culled
    if gated is not None:
        res["gated"] = gated
    if ceiling is not None:
        res["mfma_ceiling"] = ceiling
    print(json.dumps(res))


if __name__ == "__main__":
    main()
