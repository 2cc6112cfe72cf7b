"""Throughput of the tiled Newton–Schulz map on one MI355X.

    python bench.py [--steps 60] [--warmup 10] [--T 128] [--K 5] [--workload stack7b]

One step is one ``himuon_ns_tiled`` call over the whole workload (every tile
of every matrix: gather, normalise, K Newton–Schulz steps, write back), with
the inputs already resident in HBM. The default workload is a 32-layer stack
of 7B-style projection matrices (q, k, v, o 4096x4096; gate, up 11008x4096;
down 4096x11008; 224 matrices, 6.48e9 bf16 entries), synthetic low-rank(64)
plus noise, T=128, K=5, under a 16 GB chunk budget (two chunk launches).

Throughput counts 6·H·W·T·K flops per matrix (three T³ products per tile per
step). Rank 0 prints one JSON line on stdout; progress goes to stderr.
The JSON also carries:
  roofline      the fused kernel's algorithmic flops per launch over its mean
                launch duration (one pair of HIP events on the launch stream
                around the timed region, whose launches run back to back; the
                per-step spread in `step_ms` comes from a second, untimed pass
                with an event pair around each step), against the
                published dense fp16/bf16 MFMA peak (2.5 PFLOP/s); the MFMA
                work actually issued (less than 6T^3 per tile-step where a
                kernel exploits the symmetry of H and aI + P) is reported
                beside it as mfma_issued_*; `traffic` is
                the HBM bytes per launch from rocprofv3 FETCH_SIZE/WRITE_SIZE
                counters (profiles/ns_tiled_traffic.json) when they were taken
                on the current kernel source, else null;
  cpu_baseline  the fp64 oracle timed on the host cores (and on one core) on a
                bounded random sample of the same workload's tiles (read back
                from the GPU), with the CPU model; its `parity` field compares
                those oracle tiles with the GPU's outputs of the last step;
  power         socket power and graphics clock sampled from the driver's sysfs
                files during the timed region (null where they cannot be read):
                the fused kernels run at the board's power cap, below the clock
                on which the published peak is quoted.

`--calib-gemm N` times the GEMM library's N x N x N fp16 product instead (the
same power and clock fields), as a reference for what dense MFMA work
sustains under the same power cap; `--calib-mfma f16|bf16` times a launch of
nothing but 32x32x16 MFMA products (himuon_calib_mfma), the device's ceiling
for the tile kernels' own instruction.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import threading
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_TFLOPS = {"f16": 2500.0, "bf16": 2500.0, "f32": 157.3}  # MI355X dense MFMA, published
HBM_PEAK_GBS = 8000.0
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2606_27216_amd", "csrc", f)
                  for f in ("ns_device.h", "ns_tiled_kernels.hip", "ns_tiled_f16.hip")]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "ns_tiled_traffic.json")
METRIC = "tiled-NS TFLOP/s (6·H·W·T·K) + % bf16 MFMA peak, 7B layer stack T=128 K=5"


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


class PowerSampler:
    """Samples the GPU's socket power (hwmon power1_input, microwatts) and
    current graphics clock (the marked line of pp_dpm_sclk) every `period`
    seconds in a thread, while used as a context manager. Only a machine with
    exactly one GPU card in sysfs is sampled (no mapping from device to card
    is needed then); elsewhere summary() is None."""

    def __init__(self, period: float = 0.05):
        import glob
        self.period = period
        self.power_w, self.mhz = [], []
        self._stop = threading.Event()
        self._thread = None
        self.power_file = self.sclk_file = None
        cards = [d for d in sorted(glob.glob("/sys/class/drm/card*/device"))
                 if glob.glob(os.path.join(d, "hwmon", "hwmon*", "power1_input"))]
        if len(cards) == 1:
            self.power_file = glob.glob(os.path.join(cards[0], "hwmon", "hwmon*", "power1_input"))[0]
            sclk = os.path.join(cards[0], "pp_dpm_sclk")
            self.sclk_file = sclk if os.path.exists(sclk) else None

    def _read(self):
        try:
            with open(self.power_file) as f:
                self.power_w.append(int(f.read().strip()) / 1e6)
        except (OSError, ValueError):
            pass
        if self.sclk_file:
            try:
                with open(self.sclk_file) as f:
                    for line in f:
                        if "*" in line:
                            m = re.search(r"(\d+)\s*[Mm]hz", line)
                            if m:
                                self.mhz.append(int(m.group(1)))
            except OSError:
                pass

    def _run(self):
        while not self._stop.wait(self.period):
            self._read()

    def __enter__(self):
        if self.power_file:
            self._thread = threading.Thread(target=self._run, daemon=True)
            self._thread.start()
        return self

    def restart(self):
        """Drops the samples taken so far (those of a warm-up)."""
        self.power_w.clear()
        self.mhz.clear()

    def stop(self):
        """Ends the sampling; summary() then covers what was sampled so far."""
        if self._thread:
            self._stop.set()
            self._thread.join()
            self._thread = None

    def __exit__(self, *exc):
        self.stop()
        return False

    def summary(self):
        if not self.power_w:
            return None
        import statistics
        return {"socket_w_median": round(statistics.median(self.power_w), 1),
                "gfx_mhz_median": statistics.median(self.mhz) if self.mhz else None,
                "samples": len(self.power_w), "period_s": self.period,
                "source": "sysfs hwmon power1_input, pp_dpm_sclk"}


def timed_steps(torch, np, step, stream, steps, warmup, ps=None, jitter_steps=30):
    """Runs `warmup` untimed steps, then times exactly `steps` steps back to back.

    The timed region holds one pair of HIP events on the launch stream (start
    and end) and nothing else: with an event pair between two launches the
    kernel trace shows a gap of about 11 us before each launch, a few percent
    of a call of a few hundred microseconds. Step-to-step spread comes from
    a second, untimed pass of up to `jitter_steps` steps with an event pair
    around each. `ps` (a PowerSampler) is restarted with the timed region and
    stopped at its end.

    Returns (wall seconds, event-timed ms of the timed region, per-step ms of
    the second pass)."""
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    if ps is not None:
        ps.restart()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record(stream)
    for _ in range(steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    if ps is not None:
        ps.stop()
    region_ms = e0.elapsed_time(e1)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(min(steps, jitter_steps))]
    for a, b in ev:
        a.record(stream)
        step()
        b.record(stream)
    torch.cuda.synchronize()
    return wall, region_ms, np.array([a.elapsed_time(b) for a, b in ev])


def bench_calib_gemm(args, torch, np, dev):
    """The GEMM library's N x N x N fp16 product, timed like a bench step."""
    n = args.calib_gemm
    a = torch.randn(n, n, device=dev, dtype=torch.float16)
    b = torch.randn(n, n, device=dev, dtype=torch.float16)
    c = torch.empty(n, n, device=dev, dtype=torch.float16)
    with PowerSampler() as ps:
        wall, _, ms = timed_steps(torch, np, lambda: torch.matmul(a, b, out=c), torch.cuda.current_stream(dev),
                                  args.steps, args.warmup, ps)
    rec = {"metric": "library GEMM fp16 TFLOP/s (2N^3)", "value": round(2.0 * n ** 3 / (wall / args.steps) / 1e12, 1),
           "unit": "TFLOP/s", "n": n, "steps": args.steps, "warmup": args.warmup,
           "median_ms": round(float(np.median(ms)), 4), "peak": PEAK_TFLOPS["f16"], "power": ps.summary()}
    print(json.dumps(rec), flush=True)


def bench_calib_mfma(args, torch, np, dev, hm):
    """Dense 32x32x16 MFMA products and nothing else (himuon_calib_mfma):
    the rate the device sustains for the tile kernels' own instruction,
    timed like a bench step, with the power sampler."""
    compute = hm.COMPUTE_BF16 if args.calib_mfma == "bf16" else hm.COMPUTE_F16
    cus = torch.cuda.get_device_properties(dev).multi_processor_count
    grid, iters = 8 * cus, 20000  # eight waves per SIMD
    g = torch.Generator(device=dev)
    g.manual_seed(11)
    x = torch.randn(4096 * 8, device=dev, generator=g, dtype=torch.float32)
    ops = (x.to(torch.bfloat16) if args.calib_mfma == "bf16" else x.to(torch.float16)).contiguous()
    out = torch.empty(grid * 256, device=dev, dtype=torch.float32)
    stream = torch.cuda.current_stream(dev).cuda_stream

    def launch():
        st = hm.himuon_calib_mfma(compute, ops.data_ptr(), out.data_ptr(), grid, iters, stream)
        if st != hm.OK:
            raise RuntimeError(f"himuon_calib_mfma: {hm.himuon_status_string(st)}")

    flops = grid * 4 * 4 * iters * 32 * 32 * 16 * 2.0
    with PowerSampler() as ps:
        wall, _, ms = timed_steps(torch, np, launch, torch.cuda.current_stream(dev), args.steps, args.warmup, ps)
    assert torch.isfinite(out).all().item()
    rec = {"metric": f"MFMA-only 32x32x16 {args.calib_mfma} TFLOP/s", "value": round(flops / (wall / args.steps) / 1e12, 1),
           "unit": "TFLOP/s", "steps": args.steps, "warmup": args.warmup, "grid": grid, "iters": iters,
           "median_launch_ms": round(float(np.median(ms)), 4),
           "median_launch_tflops": round(flops / float(np.median(ms)) / 1e9, 1),
           "peak": PEAK_TFLOPS["f16"], "power": ps.summary()}
    print(json.dumps(rec), flush=True)


def kernel_source_hash() -> str:
    """Hash of the kernel sources' code: comments and whitespace removed, so
    that only a change of the code invalidates recorded counters."""
    src = "".join(open(f, encoding="utf-8").read() for f in KERNEL_SOURCES)
    src = re.sub(r"/\*.*?\*/", " ", src, flags=re.S)
    src = re.sub(r"//[^\n]*", " ", src)
    return hashlib.sha256("".join(src.split()).encode()).hexdigest()[:16]


def build_workload(name, device, dtype):
    import workloads
    if name == "stack7b":
        desc = ("7B layer stack: 32 layers x (q,k,v,o 4096x4096; gate,up 11008x4096; down 4096x11008), "
                "224 matrices, low-rank(64, sigma_i=1/i)+0.01 N(0,1)")
        return desc, workloads.stack_7b(32, dtype, device)
    if name == "layer7b":
        return "one 7B layer: 7 matrices, low-rank(64)+noise", workloads.layer_7b(3000, dtype, device)
    if name == "square4096":
        return "one 4096x4096 low-rank(64)+noise", [workloads.lowrank_plus_noise(4096, 4096, 2, dtype, device)]
    if name == "hetero":
        return ("heterogeneous: 8 each of 1024x4096, 4096x1024, 2048x2048, 0.02 t(3)",
                workloads.heterogeneous(dtype, device))
    raise SystemExit(f"unknown workload {name}")


def traffic_for_launch(T, K, dtype, compute, tiles_per_launch):
    """HBM bytes per launch from the committed counter summary, if it was
    taken on this kernel source and this configuration."""
    try:
        rec = json.load(open(TRAFFIC_FILE))
    except (OSError, ValueError):
        return None
    if rec.get("kernel_source_sha256_16") != kernel_source_hash():
        return None
    key = f"T{T}_K{K}_{dtype}_{compute}_tiles{tiles_per_launch}"
    ent = rec.get("launches", {}).get(key)
    if not ent:
        return None
    return ent["fetch_bytes"] + ent["write_bytes"]


def issued_fraction(T, op_name, c):
    """MFMA work a launch issues, as a fraction of the 6T^3 per tile-step the
    metric counts. The fp16 128-tile kernel evaluates only the ten upper
    32x32 blocks of the symmetric H and aI + P (of 16 each) plus the full PZ
    product, the fp16 64-tile kernel the three upper blocks (of 4) of each
    when c != 0; with c = 0 there is no P product (aI + P = aI + bH)."""
    if op_name == "f16" and T == 128:
        return (10 + (10 if c != 0 else 0) + 16) / 48.0
    if op_name == "f16" and T == 64 and c != 0:
        return (3 + 3 + 4) / 12.0
    return 1.0 if c != 0 else 2.0 / 3.0


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo", encoding="utf-8"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(mats, outs, T, K, coeffs, budget_s, seed=0):
    """The fp64 oracle on a random sample of tiles of the workload (host
    cores), timed; its tiles are also compared with the GPU's outputs of the
    last step (per-tile relative Frobenius error). A second, smaller
    sample runs on one core."""
    import numpy as np
    import oracle

    rng = np.random.default_rng(seed)
    counts = [oracle.tile_count(x.shape[0], x.shape[1], T) for x in mats]
    errs = []

    def sample(seconds, batch):
        # each round: up to `batch` random tiles of one random row of tiles,
        # so that one oracle call spreads them over its threads
        done, elapsed = 0, 0.0
        while elapsed < seconds:
            i = int(rng.integers(len(mats)))
            x, y = mats[i], outs[i]
            C = -(-x.shape[1] // T)
            r0 = int(rng.integers(counts[i] // C))
            ids = r0 * C + np.sort(rng.choice(C, min(batch, C), replace=False))
            # read back only the rows of tiles those ids touch
            rows = sorted({int(t) // C for t in ids})
            sub = {r: x[r * T:(r + 1) * T].float().cpu().double().numpy() for r in rows}
            got = {r: y[r * T:(r + 1) * T].float().cpu().double().numpy() for r in rows}
            refs = {}
            t0 = time.perf_counter()
            for r in rows:
                loc = [int(t) % C for t in ids if int(t) // C == r]
                refs[r] = (loc, oracle.ns_tiles(sub[r], T, K, *coeffs, loc))
            elapsed += time.perf_counter() - t0
            done += len(ids)
            for r, (loc, ref) in refs.items():
                for c, tile in zip(loc, ref):
                    g = got[r][:, c * T:(c + 1) * T]
                    rt = tile[:g.shape[0], :g.shape[1]]
                    n = np.linalg.norm(rt)
                    errs.append(np.linalg.norm(g - rt) / n if n > 0 else (0.0 if not np.any(g) else np.inf))
        return done, elapsed

    cores = oracle.num_threads()
    done, elapsed = sample(budget_s, 2 * cores)
    flops = 6.0 * T ** 3 * K
    oracle.set_num_threads(1)
    try:
        done1, elapsed1 = sample(budget_s / 4, 4)
    finally:
        oracle.set_num_threads(cores)
    e = np.array(errs)
    return {"value": flops * done / elapsed / 1e12, "unit": "TFLOP/s", "cores": cores, "kind": "oracle",
            "sample": f"{done} random {T}x{T} tiles of the same workload (fp64 oracle, {elapsed:.1f} s on {cores} "
                      f"threads); one core: {done1} tiles in {elapsed1:.1f} s",
            "one_core_value": flops * done1 / elapsed1 / 1e12, "cpu_model": cpu_model(),
            "parity": {"tiles": int(e.size), "max": float(e.max()), "p50": float(np.median(e)),
                       "bar": 2e-2 if mats[0].dtype.itemsize == 2 else 1e-5,
                       "what": "per-tile relative Frobenius error of the last step's output against these "
                               "oracle tiles"}}


def bench_gemm(args, hm, torch, np, mats, outs, desc, coeffs, compute, code, stream):
    """The library-GEMM path: whole matrices (T = 0, the full-matrix branch)
    or large tiles (T >= 1). Work counted: for T >= 1 the tiled metric
    6*H*W*T*K; for T = 0 the three products of each step on the m x n
    iterate (m = min(H, W)): (2 m^2 n + 2 m^3 + 2 m^2 n) K. Both are what
    the GEMMs issue (no symmetry is exploited on this path)."""
    rows = [x.shape[0] for x in mats]
    cols = [x.shape[1] for x in mats]
    Th, Tw = args.T, (args.T if args.Tw is None else args.Tw)
    if args.T == 0:
        flops_step = sum((4.0 * min(h, w) ** 2 * max(h, w) + 2.0 * min(h, w) ** 3) * args.K for h, w in zip(rows, cols))
        metric = "full-matrix NS TFLOP/s ((4m^2n + 2m^3)K, m = min(H,W)), 7B layer stack K=%d" % args.K
    elif Th == Tw:
        flops_step = sum(6.0 * h * w * args.T * args.K for h, w in zip(rows, cols))
        metric = "tiled-NS TFLOP/s (6*H*W*T*K) + %% bf16 MFMA peak, 7B layer stack T=%d K=%d (library GEMMs)" % (args.T, args.K)
    else:
        # per tile and step (4 m^2 n + 2 m^3), m = min(Th, Tw), n = max: per entry (4m + 2m^2/n)
        m, n = min(Th, Tw), max(Th, Tw)
        flops_step = sum((4.0 * m + 2.0 * m * m / n) * h * w * args.K for h, w in zip(rows, cols))
        metric = ("tiled-NS TFLOP/s ((4m^2n + 2m^3)K per tile), 7B layer stack %dx%d tiles K=%d (library GEMMs)"
                  % (Th, Tw, args.K))
    need = hm.himuon_ns_gemm_hw_workspace_size(rows, cols, Th, Tw, code, compute, args.K, *coeffs, int(args.budget))
    if need == 0:
        raise SystemExit("no plan for this call (budget below one problem?)")
    log(f"gemm path workspace {need / 2**30:.2f} GiB")
    ws = torch.empty(need, dtype=torch.uint8, device=mats[0].device)
    if args.tune:
        t0 = time.perf_counter()
        hm.gemm_tune(list(zip(rows, cols)), Th, code, K=args.K, coeffs=coeffs, compute=compute,
                     chunk_budget_bytes=int(args.budget), workspace=ws, stream=stream, Tw=Tw)
        log(f"GEMM candidates timed in {time.perf_counter() - t0:.1f} s")

    def step():
        hm.ns_gemm(mats, outputs=outs, T=Th, K=args.K, coeffs=coeffs, compute=compute,
                   chunk_budget_bytes=int(args.budget), workspace=ws, stream=stream, Tw=Tw)

    wall, region_ms, step_ms = timed_steps(torch, np, step, stream, args.steps, args.warmup)
    op_name = "f32" if code == hm.F32 else ("bf16" if compute == hm.COMPUTE_BF16 else "f16")
    peak = PEAK_TFLOPS[op_name]
    achieved = flops_step / (region_ms / args.steps * 1e-3) / 1e12
    rec = {
        "metric": metric, "value": round(flops_step / (wall / args.steps) / 1e12, 3), "unit": "TFLOP/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(wall * 1e3 / args.steps, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": op_name, "data": "synthetic",
        "config": {"workload": desc, "path": "gemm", "T": args.T, "Tw": Tw, "K": args.K, "matrices": len(mats),
                   "storage": args.dtype, "mfma_operands": op_name, "accumulate": "f32",
                   "chunk_budget_bytes": int(args.budget), "workspace_bytes": need, "gemm_tuned": bool(args.tune)},
        "roofline": {"bound": "mfma", "achieved": round(achieved, 3), "peak": peak, "unit": "TFLOP/s",
                     "frac": round(achieved / peak, 4), "traffic": None, "flops_per_step": flops_step,
                     "mean_step_ms": round(region_ms / args.steps, 4)},
        "step_ms": {"median": round(float(np.median(step_ms)), 4),
                    "iqr": round(float(np.percentile(step_ms, 75) - np.percentile(step_ms, 25)), 4),
                    "steps": len(step_ms)},
    }
    print(json.dumps(rec), flush=True)


def bench_rect(args, hm, torch, np, mats, outs, desc, coeffs, compute, code, stream, op_name):
    """The fused rectangular-tile kernels (himuon_ns_tiled_hw): T x Tw tiles,
    work counted as the GEMM path's rectangular tiles, (4 m^2 n + 2 m^3) K
    per tile with m = min, n = max of the tile sides (padding included, as
    the tiles run)."""
    Th, Tw = args.T, args.Tw
    m, n = min(Th, Tw), max(Th, Tw)
    tiles = sum(-(-h // Th) * -(-w // Tw) for h, w in ((x.shape[0], x.shape[1]) for x in mats))
    flops_step = tiles * (4.0 * m * m * n + 2.0 * m ** 3) * args.K
    ws = torch.empty(hm.himuon_ns_tiled_workspace_size(len(mats)), dtype=torch.uint8, device=mats[0].device)

    def step():
        hm.ns_tiled(mats, outputs=outs, T=Th, Tw=Tw, K=args.K, coeffs=coeffs, compute=compute,
                    chunk_budget_bytes=int(args.budget), workspace=ws, stream=stream)

    wall, region_ms, step_ms = timed_steps(torch, np, step, stream, args.steps, args.warmup)
    peak = PEAK_TFLOPS[op_name]
    achieved = flops_step / (region_ms / args.steps * 1e-3) / 1e12
    rec = {
        "metric": "tiled-NS TFLOP/s ((4m^2n + 2m^3)K per tile), 7B layer stack %dx%d tiles K=%d (fused kernel)"
                  % (Th, Tw, args.K),
        "value": round(flops_step / (wall / args.steps) / 1e12, 3), "unit": "TFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(wall * 1e3 / args.steps, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": op_name, "data": "synthetic",
        "config": {"workload": desc, "path": "tiled_hw", "T": Th, "Tw": Tw, "K": args.K, "matrices": len(mats),
                   "tiles": tiles, "storage": args.dtype, "mfma_operands": op_name, "accumulate": "f32",
                   "chunk_budget_bytes": int(args.budget)},
        "roofline": {"bound": "mfma", "achieved": round(achieved, 3), "peak": peak, "unit": "TFLOP/s",
                     "frac": round(achieved / peak, 4), "traffic": None, "flops_per_step": flops_step,
                     "mean_step_ms": round(region_ms / args.steps, 4)},
        "step_ms": {"median": round(float(np.median(step_ms)), 4),
                    "iqr": round(float(np.percentile(step_ms, 75) - np.percentile(step_ms, 25)), 4),
                    "steps": len(step_ms)},
    }
    print(json.dumps(rec), flush=True)


def bench_optstep(args, hm, torch, np, dev):
    """The optimizer-step benchmark of Sec. 6.4 (cross-layer batching): 8
    stacked bias-free Linear(H, H) layers in bf16, fresh Gaussian gradients
    before every step (outside the timed region), HiMuon with T = 512, K = 5
    against full-matrix Muon (T = 0: the same Alg. 1 step with Phi_K of the
    whole matrix), each as one call per layer and as one batched call over
    all layers; for HiMuon also the batched call recorded once into a plan (a
    HIP graph) and replayed each step, the study's graph-captured variant.
    Per-step time is the median of the HIP-event times of
    `--steps` steps after `--warmup` (the paper: 50 after 20), beside the
    median host time the step's calls take to enqueue, and the mean of the
    same number of steps run back to back between one event pair
    (`back_to_back_ms`: no event or gradient kernel between the steps); peak
    memory is torch's peak allocation over the variant's run, workspace
    included."""
    coeffs = tuple(float(np.float32(v)) for v in hm.QUINTIC)
    hs = [int(h) for h in args.hidden.split(",")]
    stream = torch.cuda.current_stream(dev)
    out = {}
    for H in hs:
        gen = torch.Generator(device=dev)
        gen.manual_seed(H)
        Ws = [(torch.randn(H, H, device=dev, generator=gen) * 0.02).to(torch.bfloat16) for _ in range(8)]
        Gs = [torch.empty(H, H, dtype=torch.bfloat16, device=dev) for _ in range(8)]
        res = {}
        variants = [("muon_full_per_layer", 0, False, False), ("muon_full_batched", 0, True, False)]
        for t in (int(v) for v in args.optstep_T.split(",")):
            variants += [(f"himuon_T{t}_per_layer", t, False, False), (f"himuon_T{t}_batched", t, True, False),
                         (f"himuon_T{t}_batched_graph", t, True, True)]
        if args.variants != "all":
            keep = args.variants.split(",")
            variants = [v for v in variants if v[0] in keep]
        for name, T, batched, graph in variants:
            Ms = [torch.zeros_like(w) for w in Ws]
            torch.cuda.synchronize()
            torch.cuda.reset_peak_memory_stats(dev)
            groups = [list(range(8))] if batched else [[i] for i in range(8)]
            opts = [hm.HiMuon([Ws[i] for i in g], T=T, K=5, coeffs=coeffs, lr=0.02, momentum=0.95,
                              weight_decay=0.0, nesterov=True, scale_c=0.2, tune=args.tune, capture=graph)
                    for g in groups]
            for o, g in zip(opts, groups):
                o.moms = [Ms[i] for i in g]
            ws_bytes = sum(o._workspace.numel() for o in opts)

            def one_step():
                for o, g in zip(opts, groups):
                    o.step([Gs[i] for i in g], stream=stream)

            times, host = [], []
            for it in range(args.warmup + args.steps):
                for g in Gs:
                    g.normal_(generator=gen)
                a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                a.record(stream)
                h0 = time.perf_counter()
                one_step()
                h1 = time.perf_counter()
                b.record(stream)
                if it >= args.warmup:
                    times.append((a, b))
                    host.append(h1 - h0)
            torch.cuda.synchronize()
            ms = np.array([a.elapsed_time(b) for a, b in times])
            # the same steps back to back between one event pair (the last
            # gradients reused): no event or gradient kernel between steps
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for _ in range(args.steps):
                one_step()
            e1.record(stream)
            torch.cuda.synchronize()
            b2b = e0.elapsed_time(e1) / args.steps
            flops = 8 * (6.0 * H * H * min(T, H) * 5 if T else 6.0 * H ** 3 * 5)
            res[name] = {"median_ms": round(float(np.median(ms)), 4),
                         "back_to_back_ms": round(b2b, 4),
                         "host_us_per_step": round(float(np.median(host)) * 1e6, 1),
                         "iqr_ms": round(float(np.percentile(ms, 75) - np.percentile(ms, 25)), 4),
                         "ns_tflops": round(flops / (float(np.median(ms)) * 1e-3) / 1e12, 2),
                         "peak_mem_MiB": round(torch.cuda.max_memory_allocated(dev) / 2 ** 20, 1),
                         "workspace_MiB": round(ws_bytes / 2 ** 20, 1)}
            log(f"H={H} {name}: {res[name]}")
            del opts
        if "muon_full_per_layer" in res:
            base = res["muon_full_per_layer"]["median_ms"]
            for name in res:
                res[name]["speedup_vs_full_per_layer"] = round(base / res[name]["median_ms"], 3)
        out[str(H)] = res
        del Ws, Gs
        torch.cuda.empty_cache()
    h_last = str(hs[-1])
    headline = "himuon_T512_batched" if "himuon_T512_batched" in out[h_last] else next(iter(out[h_last]))
    rec = {
        "metric": "optimizer-step time, 8 x Linear(H,H) bf16, K=5, median [ms]",
        "value": out[h_last][headline]["median_ms"],
        "unit": "ms", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "higher_is_better": False, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"8 x Linear({h_last},{h_last}) bf16, fresh N(0,1) gradients each step",
                   "variant": headline, "T": 0 if headline.startswith("muon_full") else 512, "K": 5, "momentum": 0.95, "nesterov": True, "scale_c": 0.2,
                   "gemm_tuned": bool(args.tune)},
        "results": out,
    }
    print(json.dumps(rec), flush=True)


def bench_layershapes(args, hm, torch, np, dev):
    """Per-layer speedup of the tiled map over the full-matrix map on the
    Qwen3 Block-0 shapes (Sec. 6.3): one random bf16 Gaussian matrix per
    shape, Phi_K (T = 0) and Phi_{K,512} through the library-GEMM path, K = 5,
    one call per matrix; the paired ratio t_full / t_tile is the median over
    `--steps` timed calls after `--warmup` (the paper: 30 after 3). The fused
    T = 128 kernel is timed beside them, and every call again as a recorded
    plan (one HIP graph launch per call, field `graph`)."""
    import workloads
    coeffs = tuple(float(np.float32(v)) for v in hm.QUINTIC)
    stream = torch.cuda.current_stream(dev)
    out = {}

    def timed(fn):
        for _ in range(args.warmup):
            fn()
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
        for a, b in ev:
            a.record(stream)
            fn()
            b.record(stream)
        torch.cuda.synchronize()
        return np.array([a.elapsed_time(b) for a, b in ev])

    for model, shapes in workloads.QWEN3_BLOCK0.items():
        res = {}
        for j, (name, H, W) in enumerate(shapes):
            x = workloads.gaussian(H, W, 7000 + j, "bf16", dev)
            y = torch.empty_like(x)
            for T in (0, 512):
                hm.gemm_tune([(H, W)], T, hm.BF16, K=5, coeffs=coeffs)
            t_full = timed(lambda: hm.ns_gemm([x], outputs=[y], T=0, K=5, coeffs=coeffs, stream=stream))
            t_tile = timed(lambda: hm.ns_gemm([x], outputs=[y], T=512, K=5, coeffs=coeffs, stream=stream))
            t_128 = timed(lambda: hm.ns_tiled([x], outputs=[y], T=128, K=5, coeffs=coeffs, stream=stream))
            # the same calls recorded once into HIP graphs (plans), one graph launch per call
            plans = {"full": hm.plan_ns_gemm([x], [y], T=0, K=5, coeffs=coeffs),
                     "512": hm.plan_ns_gemm([x], [y], T=512, K=5, coeffs=coeffs),
                     "128": hm.plan_ns_tiled([x], [y], T=128, K=5, coeffs=coeffs)}
            g = {k: timed(lambda p=p: p.launch(stream)) for k, p in plans.items()}
            for p in plans.values():
                p.close()
            res[name] = {"shape": [H, W], "full_ms": round(float(np.median(t_full)), 4),
                         "tiled512_ms": round(float(np.median(t_tile)), 4),
                         "speedup_512": round(float(np.median(t_full / t_tile)), 3),
                         "fused128_ms": round(float(np.median(t_128)), 4),
                         "speedup_128": round(float(np.median(t_full / t_128)), 3),
                         "graph": {"full_ms": round(float(np.median(g["full"])), 4),
                                   "tiled512_ms": round(float(np.median(g["512"])), 4),
                                   "fused128_ms": round(float(np.median(g["128"])), 4),
                                   "speedup_512": round(float(np.median(g["full"] / g["512"])), 3),
                                   "speedup_128": round(float(np.median(g["full"] / g["128"])), 3)}}
            log(f"{model} {name} {H}x{W}: {res[name]}")
        out[model] = res
    sp = [r["speedup_512"] for m in out.values() for r in m.values()]
    rec = {
        "metric": "per-layer tiled/full NS speedup t_full/t_tile, Qwen3 Block-0 shapes, T=512 K=5 (median of paired ratios)",
        "value": round(float(np.median(sp)), 3), "unit": "x", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "Qwen3 0.6B/1.7B/4B Block-0 shapes, one N(0,1) bf16 matrix each", "T": 512, "K": 5},
        "results": out,
    }
    print(json.dumps(rec), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=60)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="stack7b", choices=["stack7b", "layer7b", "square4096", "hetero"])
    ap.add_argument("--T", type=int, default=128)
    ap.add_argument("--K", type=int, default=5)
    ap.add_argument("--Tw", type=int, default=None,
                    help="tile width (tiles are T x Tw; default square): the fused rectangular kernels "
                         "(--path tiled) or the library GEMMs (--path gemm)")
    ap.add_argument("--dtype", default="bf16", choices=["bf16", "f32"])
    ap.add_argument("--compute", default="default", choices=["default", "f16", "bf16", "f32"])
    ap.add_argument("--budget", type=float, default=16e9, help="chunk budget in bytes (0: one chunk)")
    ap.add_argument("--cpu-seconds", type=float, default=12.0, help="oracle time budget (0: skip)")
    ap.add_argument("--path", default="tiled", choices=["tiled", "gemm"],
                    help="tiled: the fused per-tile kernels (T <= 256); gemm: himuon_ns_gemm, whole matrices "
                         "(--T 0) or large tiles (e.g. --T 512) through batched library GEMMs")
    ap.add_argument("--layershapes", action="store_true",
                    help="run the per-layer tiled (T=512) vs full-matrix comparison on Qwen3 Block-0 shapes instead")
    ap.add_argument("--optstep", action="store_true",
                    help="run the optimizer-step benchmark (8 x Linear(H,H), HiMuon T=512 vs full Muon) instead")
    ap.add_argument("--tune", type=int, default=1,
                    help="time the GEMM library's candidates for the GEMM path before the run (1) or not (0)")
    ap.add_argument("--hidden", default="1024,2048,4096", help="H values of --optstep")
    ap.add_argument("--optstep-T", dest="optstep_T", default="512",
                    help="--optstep: HiMuon tile sizes to run (comma-separated; the paper's is 512)")
    ap.add_argument("--variants", default="all",
                    help="--optstep variants to run (comma-separated names, or all)")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="only run a plain device copy of this many MiB per launch (counter calibration)")
    ap.add_argument("--calib-mfma", choices=["f16", "bf16"], default=None,
                    help="only run dense MFMA products (himuon_calib_mfma): the device's MFMA ceiling")
    ap.add_argument("--calib-gemm", type=int, default=0,
                    help="only time the GEMM library's N x N x N fp16 product (power-cap reference)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on one GPU only: the tiled map needs no communication between GPUs, and the "
              "figure is one GPU's share of the work (use --gpus 1).", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    import paper_2606_27216_amd as hm

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    if args.calib_copy_mib:
        n = args.calib_copy_mib << 20
        src = torch.empty(n, dtype=torch.uint8, device=dev).fill_(1)
        dst = torch.empty_like(src)
        for _ in range(args.warmup + args.steps):
            dst.copy_(src)
        torch.cuda.synchronize()
        log(f"copied {args.calib_copy_mib} MiB x {args.warmup + args.steps}")
        return

    if args.calib_gemm:
        return bench_calib_gemm(args, torch, np, dev)
    if args.calib_mfma:
        return bench_calib_mfma(args, torch, np, dev, hm)
    if args.optstep:
        return bench_optstep(args, hm, torch, np, dev)
    if args.layershapes:
        return bench_layershapes(args, hm, torch, np, dev)

    coeffs = tuple(float(np.float32(v)) for v in hm.QUINTIC)
    compute = {"default": hm.COMPUTE_DEFAULT, "f16": hm.COMPUTE_F16, "bf16": hm.COMPUTE_BF16,
               "f32": hm.COMPUTE_F32}[args.compute]
    resolved = hm.himuon_select_compute(hm.BF16 if args.dtype == "bf16" else hm.F32, compute, args.K, *coeffs)
    op_name = {hm.COMPUTE_F32: "f32", hm.COMPUTE_F16: "f16", hm.COMPUTE_BF16: "bf16"}[resolved]

    t0 = time.perf_counter()
    desc, mats = build_workload(args.workload, dev, args.dtype)
    torch.cuda.synchronize()
    outs = [torch.empty_like(x) for x in mats]
    log(f"workload ready in {time.perf_counter() - t0:.1f} s: {len(mats)} matrices")

    rows = [x.shape[0] for x in mats]
    cols = [x.shape[1] for x in mats]
    code = hm.BF16 if args.dtype == "bf16" else hm.F32
    stream = torch.cuda.current_stream(dev)
    if args.path == "gemm":
        return bench_gemm(args, hm, torch, np, mats, outs, desc, coeffs, compute, code, stream)
    if args.Tw is not None and args.Tw != args.T:
        return bench_rect(args, hm, torch, np, mats, outs, desc, coeffs, compute, code, stream, op_name)
    total, bounds = hm.himuon_plan_chunks(rows, cols, args.T, code, int(args.budget))
    launches = len(bounds) - 1
    flops_step = sum(6.0 * h * w * args.T * args.K for h, w in zip(rows, cols))
    elem = 2 if args.dtype == "bf16" else 4
    bytes_step = sum(2.0 * h * w * elem for h, w in zip(rows, cols))

    need = hm.himuon_ns_tiled_call_workspace_size(rows, cols, args.T, code, compute, args.K, *coeffs, int(args.budget))
    if need == 0:
        raise SystemExit("himuon_ns_tiled would reject this call (tile size, dtype/compute or budget)")
    ws = torch.empty(need, dtype=torch.uint8, device=dev)

    def step():
        hm.ns_tiled(mats, outputs=outs, T=args.T, K=args.K, coeffs=coeffs, compute=compute,
                    chunk_budget_bytes=int(args.budget), workspace=ws, stream=stream)

    with PowerSampler() as ps:
        wall, region_ms, step_ms = timed_steps(torch, np, step, stream, args.steps, args.warmup, ps)
    log(f"timed {args.steps} steps: wall {wall * 1e3:.2f} ms, events {region_ms:.2f} ms; "
        f"per-step median {np.median(step_ms):.3f} ms")
    power = ps.summary()
    if power:
        log(f"socket power {power['socket_w_median']} W, graphics clock {power['gfx_mhz_median']} MHz "
            f"({power['samples']} samples)")

    ms_per_step = wall * 1e3 / args.steps
    value = flops_step / (wall / args.steps) / 1e12
    # per launch: a step is one call of `launches` kernel launches
    launch_ms = region_ms / args.steps / launches
    flops_launch = flops_step / launches
    achieved = flops_launch / (launch_ms * 1e-3) / 1e12
    peak = PEAK_TFLOPS[op_name]
    issued = issued_fraction(args.T, op_name, coeffs[2])
    tiles_launch = total // launches
    traffic = traffic_for_launch(args.T, args.K, args.dtype, op_name, tiles_launch)

    rec = {
        "metric": METRIC,
        "value": round(value, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": op_name,
        "data": "synthetic",
        "config": {
            "workload": desc, "T": args.T, "K": args.K, "matrices": len(mats), "tiles": total,
            "storage": args.dtype, "mfma_operands": op_name, "accumulate": "f32",
            "chunk_budget_bytes": int(args.budget), "launches_per_step": launches,
            "hbm_bytes_per_step": bytes_step, "hbm_GBps_algorithmic": round(bytes_step / (wall / args.steps) / 1e9, 1),
        },
        "roofline": {
            "bound": "mfma", "achieved": round(achieved, 3), "peak": peak, "unit": "TFLOP/s",
            "frac": round(achieved / peak, 4), "traffic": traffic,
            "flops_per_launch": flops_launch, "mean_launch_ms": round(launch_ms, 4),
            "mfma_issued_fraction": round(issued, 4),
            "mfma_issued_tflops": round(achieved * issued, 3),
            "mfma_issued_frac": round(achieved * issued / peak, 4),
        },
        "step_ms": {"median": round(float(np.median(step_ms)), 4),
                    "iqr": round(float(np.percentile(step_ms, 75) - np.percentile(step_ms, 25)), 4),
                    "steps": len(step_ms)},
        "power": power,
    }
    if args.cpu_seconds > 0:
        log(f"cpu baseline: oracle on sampled tiles for ~{args.cpu_seconds:.0f} s")
        rec["cpu_baseline"] = cpu_baseline(mats, outs, args.T, args.K, coeffs, args.cpu_seconds)
        par = rec["cpu_baseline"]["parity"]
        log(f"parity on {par['tiles']} sampled tiles: max {par['max']:.3e} p50 {par['p50']:.3e} (bar {par['bar']:.0e})")
        if not par["max"] <= par["bar"]:
            log("PARITY FAILURE: sampled tiles exceed the bar")
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
