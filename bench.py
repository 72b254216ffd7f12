"""Throughput of the fused attention forward on one MI355X.

Default workload: B=2, H=32, N=8192, d=128, bf16, Q/K/V i.i.d. N(0,1) (seed 0),
scale = 1/sqrt(d).  One step = one unmasked forward plus one causal forward
over that batch (the two runs the workload is quoted on).  Inputs are resident
in HBM before the timed region starts.  ``--workload NAME`` measures another
named workload of ``seeded_inputs.WORKLOADS`` the same way (one forward per
mask it lists), e.g. the grouped-query ones.

Metric: TFLOPS with the paper's count, 4*B*H*N^2*d per forward (Evaluation
section, "Benchmark setting"), halved for the causal run, summed over the
step and divided by the wall time of the step.

Prints one JSON line.  Extra objects:
  roofline      the dominant kernel (the first mask's forward: unmasked for
                the default workload): its algorithmic
                flops per launch over its mean launch duration, timed with
                HIP events on the launch stream inside the timed region,
                against the dense MFMA peak of the input type (bf16/fp16 2.5, FP8 5.0 PFLOP/s); ``traffic`` is the HBM bytes
                per launch from rocprofv3 FETCH_SIZE + WRITE_SIZE counters
                (scaled by a plain copy of known size), read from the
                workload's committed profile summary (every quoted 16-bit
                workload, FP8, GQA 64/8 and MLA), or null without one or once the
                kernel source has changed since those counters were taken;
  hbm           those bytes over the same launch's duration, in GB/s, against
                the published 8 TB/s (null with traffic);
  cpu_baseline  the fp64 CPU oracle timed on this host on a bounded sample of
                the same workload (whole heads, both masks), in the same unit;
  cpu_single_core  the oracle on one core over the two small workloads
                (B=1 H=2 N=128 d=64 and B=8 H=16 N=1024 d=64, fp16, unmasked).

``--sustain SECONDS`` replaces the timed steps by each launch run back to back
for that long while rocm-smi samples the shader clock, one JSON line per
launch; with ``--library PATH`` (another build of the library) two builds can
be compared one after the other on one machine, which is the fair comparison
on a power-limited part.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import seeded_inputs as si  # noqa: E402

METRIC = "attention fwd TFLOPS (4·B·H·N²·d, ½ if causal) and % of MFMA peak"
PEAK_TFLOPS = 2500.0          # MI355X dense bf16/fp16 MFMA, published
PEAK_FLOP_PER_CLK = 256 * 4096  # 256 CUs x 4096 dense bf16 flop per clock
# FP8 (E4M3) MFMA: twice the 16-bit rate, 5.0 PFLOP/s dense, published
PEAK_HBM_GBPS = 8000.0          # MI355X HBM3E, published
PEAK_TFLOPS_FP8 = 5000.0
PEAK_FLOP_PER_CLK_FP8 = 256 * 8192
KERNEL_SOURCE = os.path.join(ROOT, "paper_2506_12355_amd", "csrc", "attn_fwd_gfx950.hip")
PROFILES = os.path.join(ROOT, "profiles")
# rocprofv3 HBM-counter summaries ([B][H][N][d] layout): workload -> file; each
# gives the HBM bytes of one launch of the workload's dominant instance (the
# unmasked one when the workload runs both masks)
TRAFFIC_SUMMARIES = {
    "mha_b2_h32_n8192_d128_bf16": "attn_fwd_bf16_d128_n8192_hbm_traffic.md",
    "fp8_b2_h32_n8192_d128": "attn_fwd_fp8_e4m3_d128_n8192_hbm_traffic.md",
    "gqa_b2_h64_kv8_n8192_d128_bf16_causal":
        "attn_fwd_gqa_h64_kv8_bf16_d128_n8192_causal_hbm_traffic.md",
    "mla_b2_h128_n8192_d192_dv128_bf16_causal":
        "attn_fwd_mla_h128_bf16_d192_dv128_n8192_causal_hbm_traffic.md",
    "mha_b8_h16_n1024_d64_f16": "attn_fwd_f16_d64_n1024_b8_h16_hbm_traffic.md",
    "mha_b4_h32_n2048_d128_f16_causal": "attn_fwd_f16_d128_n2048_b4_h32_causal_hbm_traffic.md",
    "mha_b1_h32_n32768_d128_bf16_causal_qk2": "attn_fwd_bf16_d128_n32768_causal_qk2_hbm_traffic.md",
}
TRAFFIC_SUMMARY = os.path.join(PROFILES, TRAFFIC_SUMMARIES["mha_b2_h32_n8192_d128_bf16"])


def flops(B, H, N, d, causal, dv=None):
    """The paper's count, 4*B*H*N^2*d, halved for causal; with a value head
    dimension dv != d (the MLA shape) the two products count 2*B*H*N^2*d and
    2*B*H*N^2*dv."""
    dv = d if dv is None else dv
    f = 2.0 * B * H * N * N * (d + dv)
    return f / 2 if causal else f


def kernel_source_sha256() -> str:
    with open(KERNEL_SOURCE, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def committed_traffic(workload: str = si.BENCH_WORKLOAD):
    """HBM bytes per launch of the workload's dominant instance from its
    committed counter summary, if there is one for the current kernel source."""
    name = TRAFFIC_SUMMARIES.get(workload)
    path = os.path.join(PROFILES, name) if name else None
    if path is None or not os.path.exists(path):
        return None
    text = open(path).read()
    sha = re.search(r"kernel_source_sha256:\s*([0-9a-f]{64})", text)
    val = re.search(r"traffic_bytes_per_launch:\s*([0-9.eE+]+)", text)
    if not sha or not val or sha.group(1) != kernel_source_sha256():
        return None
    return float(val.group(1))


# --------------------------------------------------------------------------
# shader clock during the timed region (rocm-smi, sampled from a thread)
# --------------------------------------------------------------------------
class SclkSampler:
    """Samples the current SCLK (and the package power, where rocm-smi reports
    it) with rocm-smi from a thread while GPU work runs."""

    def __init__(self, period_s=0.2, enabled=True):
        import threading
        self.enabled = enabled
        self.period_s = period_s
        self.samples = []
        self.power = []
        self._stop = threading.Event()
        self._thread = threading.Thread(target=self._run, daemon=True)

    @staticmethod
    def parse(text):
        """(SCLK MHz or None, package power W or None) from rocm-smi's JSON."""
        data = json.loads(text)
        sclk = watts = None
        for card in data.values():
            if not isinstance(card, dict):
                continue
            m = re.search(r"(\d+)\s*Mhz", str(card.get("sclk clock speed:", "")), re.I)
            if m and sclk is None:
                sclk = int(m.group(1))
            for key, val in card.items():
                if watts is None and re.search(r"power", key, re.I) and "(W)" in key:
                    try:
                        watts = float(str(val).split()[0])
                    except ValueError:
                        pass
        return sclk, watts

    def _read(self):
        import subprocess
        out = subprocess.run(["rocm-smi", "--showclocks", "--showpower", "--json"],
                             capture_output=True, text=True, timeout=10).stdout
        return self.parse(out)

    def _run(self):
        while not self._stop.is_set():
            try:
                v, w = self._read()
                if v:
                    self.samples.append(v)
                if w:
                    self.power.append(w)
            except Exception:
                pass
            self._stop.wait(self.period_s)

    def __enter__(self):
        if self.enabled:
            self._thread.start()
        return self

    def __exit__(self, *exc):
        self._stop.set()
        if self.enabled:
            self._thread.join(timeout=15)

    def median(self):
        # fewer than three readings: too few to trust (a reading may straddle
        # the start or the end of the load)
        if len(self.samples) < 3:
            return None
        v = sorted(self.samples)
        return v[len(v) // 2]


def sustained_sclk(step, sync, seconds=3.0, max_steps=1_000_000, enabled=True):
    """The shader clock under this workload: rocm-smi readings (every 0.1 s)
    over an untimed pass that keeps running the same step for ``seconds``,
    started right after the timed steps.  (The timed region can be far
    shorter than one rocm-smi call.)  Returns (median MHz or None, readings,
    steps run, median package power in W or None: not every host's rocm-smi
    reports one)."""
    if not enabled:
        return None, 0, 0, None
    n = 0
    with SclkSampler(period_s=0.1) as sclk:
        t0 = time.perf_counter()
        while time.perf_counter() - t0 < seconds and n < max_steps:
            for _ in range(8):
                step()
            sync()
            n += 8
    watts = sorted(sclk.power)[len(sclk.power) // 2] if len(sclk.power) >= 3 else None
    return sclk.median(), len(sclk.samples), n, watts


# --------------------------------------------------------------------------
# CPU baseline: the fp64 oracle on whole heads of the same workload
# --------------------------------------------------------------------------
def _oracle_head(args):
    from threadpoolctl import threadpool_limits
    from oracle import attention_fp64
    q, k, v, scale, dtype, masks, descale = args
    with threadpool_limits(limits=1):
        t0 = time.perf_counter()
        for causal in masks:
            attention_fp64(q, k, v, scale, causal, dtype, descale=descale)
        return time.perf_counter() - t0


# CPUs one GPU's share of a shared GPU host may keep busy: worker pools never
# exceed it, whatever the affinity mask shows
CPU_SHARE_PER_GPU = 16


def usable_cpus():
    """(CPUs this process may run on, CPUs it may keep busy at once): the
    scheduler affinity, and that count capped by the cgroup's CPU quota
    (cgroup v2 ``cpu.max``, or v1 ``cpu.cfs_quota_us`` / ``cpu.cfs_period_us``)
    when one is set, and by one GPU's CPU share of the host (16)."""
    import math
    affinity = len(os.sched_getaffinity(0))
    quota = None
    try:
        with open("/sys/fs/cgroup/cpu.max") as f:
            q, period = f.read().split()[:2]
        if q != "max":
            quota = int(q) / int(period)
    except (OSError, ValueError):
        try:
            with open("/sys/fs/cgroup/cpu/cpu.cfs_quota_us") as f:
                q = int(f.read())
            with open("/sys/fs/cgroup/cpu/cpu.cfs_period_us") as f:
                period = int(f.read())
            if q > 0:
                quota = q / period
        except (OSError, ValueError):
            pass
    usable = affinity if quota is None else max(1, min(affinity, math.ceil(quota)))
    return affinity, min(usable, CPU_SHARE_PER_GPU)


def cpu_baseline(w, q, k, v, descale=None):
    import multiprocessing as mp
    affinity, cores = usable_cpus()
    n_heads = min(w.B * w.H, 4 * cores)
    group = w.H // w.kv_heads
    heads = [(i // w.H, i % w.H) for i in range(n_heads)]
    jobs = [(q[b:b + 1, h:h + 1].copy(), k[b:b + 1, h // group:h // group + 1].copy(),
             v[b:b + 1, h // group:h // group + 1].copy(), w.scale, w.dtype, w.causal, descale)
            for b, h in heads]
    ctx = mp.get_context("fork")
    t0 = time.perf_counter()
    with ctx.Pool(cores) as pool:
        pool.map(_oracle_head, jobs, chunksize=1)
    wall = time.perf_counter() - t0
    work = len(heads) * sum(flops(1, 1, w.N, w.d, c, w.d_v) for c in w.causal)
    masks = "both masks" if len(w.causal) == 2 else ("causal" if w.causal[0] else "unmasked")
    model = "unknown CPU"
    try:
        with open("/proc/cpuinfo") as f:
            model = next((ln.split(":", 1)[1].strip() for ln in f if ln.startswith("model name")),
                         model)
    except OSError:
        pass
    return {
        "value": round(work / wall / 1e12, 6),
        "unit": "TFLOPS",
        "cores": cores,
        "cores_in_affinity": affinity,
        "kind": "oracle",
        "sample": (f"{len(heads)} of {w.B * w.H} (batch, head) slices of {w.name}, {masks}, "
                   f"spread over {cores} processes with single-threaded BLAS (every CPU this "
                   f"process may keep busy: {affinity} in its affinity mask, capped by the "
                   f"cgroup CPU quota and by one GPU's share of the host, "
                   f"{CPU_SHARE_PER_GPU}) on {model}; "
                   f"wall {wall:.1f} s"),
    }


def cpu_single_core(names=("mha_b1_h2_n128_d64_f16", "mha_b8_h16_n1024_d64_f16")):
    """The oracle on one core (single-threaded BLAS) over whole small workloads,
    unmasked: seconds and fp64 GFLOP/s by the metric's count."""
    from threadpoolctl import threadpool_limits
    from oracle import attention_fp64
    out = {}
    for name in names:
        w = si.WORKLOADS[name]
        q, k, v = w.inputs()
        with threadpool_limits(limits=1):
            t0 = time.perf_counter()
            attention_fp64(q, k, v, w.scale, False, w.dtype)
            dt = time.perf_counter() - t0
        out[name] = {"seconds": round(dt, 4),
                     "gflops": round(flops(w.B, w.H, w.N, w.d, False) / dt / 1e9, 3)}
    return out


# --------------------------------------------------------------------------
# the paper's benchmark grid: 16k tokens per batch, hidden 2048, d 64 / 128
# --------------------------------------------------------------------------
def run_grid(args, qa, torch, np):
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream(dev)
    for name, w in list(si.GRID.items()) + list(si.GRID_FP8.items()):
        fp8 = w.dtype == "e4m3"
        if fp8:
            q, k, v, scales = w.fp8_inputs()
            tq, tk, tv = (torch.from_numpy(x).to(dev) for x in (q, k, v))
        else:
            q, k, v = w.inputs()
            tq, tk, tv = (torch.from_numpy(x.view(np.int16)).to(dev).view(torch.bfloat16)
                          for x in (q, k, v))
        del q, k, v
        o = torch.empty((w.B, w.H, w.N, w.d), dtype=torch.bfloat16, device=dev)
        lse = torch.empty((w.B, w.H, w.N), dtype=torch.float32, device=dev)
        peak = PEAK_TFLOPS_FP8 if fp8 else PEAK_TFLOPS
        per = {}
        for causal in w.causal:
            # the C entry points directly: short launches must not wait on
            # Python-side argument checks
            ptrs = (tq.data_ptr(), tk.data_ptr(), tv.data_ptr(), o.data_ptr(), lse.data_ptr())
            if fp8:
                entry = qa.qm_attn_fwd_fp8
                call = ptrs + (w.B, w.H, w.N, w.d) + scales + (w.scale, int(causal),
                                                               stream.cuda_stream)
            else:
                entry = qa.qm_attn_fwd
                call = ptrs + (w.B, w.H, w.N, w.d, w.scale, int(causal), stream.cuda_stream,
                               qa.QM_BF16)
            for _ in range(args.warmup):
                assert entry(*call) == qa.QM_OK
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
            ev[0].record(stream)
            for _ in range(args.steps):
                entry(*call)
            ev[1].record(stream)
            torch.cuda.synchronize(dev)
            ms = ev[0].elapsed_time(ev[1]) / args.steps
            tf = flops(w.B, w.H, w.N, w.d, causal) / (ms * 1e-3) / 1e12
            per["causal" if causal else "unmasked"] = {
                "ms": round(ms, 4), "tflops": round(tf, 2),
                "pct_of_peak": round(100.0 * tf / peak, 2)}
        print(json.dumps({"metric": METRIC, "grid": True, "workload": name,
                          "B": w.B, "H": w.H, "N": w.N, "d": w.d, "dtype": w.dtype,
                          "peak_tflops": peak, "steps": args.steps, "warmup": args.warmup,
                          "tile_rows": args.tile_rows or "auto", "per_launch": per}),
              flush=True)
        del tq, tk, tv, o, lse


# --------------------------------------------------------------------------
def sustain(args, w, masks, step_one, dev, stream, torch, peak_per_clk):
    """Each launch of the workload back to back for args.sustain seconds (after
    its own warm-up) while rocm-smi samples the shader clock: the throughput a
    launch holds at the clock it settles to.  The part is power-limited with
    random operands, so two builds of the kernel compare fairly only like this,
    one after the other on one machine."""
    for m, causal in enumerate(masks):
        for _ in range(20):
            step_one(m)
        torch.cuda.synchronize(dev)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        n = 0
        with SclkSampler(period_s=0.1) as sclk:
            e0.record(stream)
            t0 = time.perf_counter()
            while time.perf_counter() - t0 < args.sustain:
                for _ in range(16):
                    step_one(m)
                n += 16
                torch.cuda.synchronize(dev)
            e1.record(stream)
            torch.cuda.synchronize(dev)
        ms = e0.elapsed_time(e1) / n
        tflops = flops(w.B, w.H, w.N, w.d, causal, w.d_v) / (ms * 1e-3) / 1e12
        mhz = sclk.median()
        print(json.dumps({
            "sustained": True, "workload": w.name, "launch": "causal" if causal else "unmasked",
            "library": os.path.abspath(args.library) if args.library else "in-tree",
            "seconds": args.sustain, "launches": n, "ms": round(ms, 4), "tflops": round(tflops, 2),
            "sclk_mhz": mhz,
            "tflops_per_ghz": round(tflops / (mhz / 1000.0), 1) if mhz else None,
            "pct_of_peak_at_sclk": (round(100.0 * tflops / (peak_per_clk * mhz * 1e6 / 1e12), 2)
                                    if mhz else None),
        }), flush=True)
        time.sleep(1.0)


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--no-cpu-baseline", action="store_true",
                    help="skip the CPU oracle leg (for profiler runs)")
    ap.add_argument("--no-sclk", action="store_true",
                    help="do not sample the shader clock (rocm-smi child processes); for runs "
                         "under a profiler that initialises the GPU in every process")
    ap.add_argument("--workload", default=si.BENCH_WORKLOAD, choices=sorted(si.WORKLOADS),
                    help="named workload (default: the one the metric is quoted on)")
    ap.add_argument("--layout", default="bhnd", choices=("bhnd", "bnhd"),
                    help="memory layout of q, k, v and o: [B][H][N][d] "
                         "(default) or [B][N][H][d]")
    ap.add_argument("--grid", action="store_true",
                    help="measure the paper's benchmark grid instead (one JSON line per shape; "
                         "bf16 at d = 64 and 128 with both masks, then FP8 at d = 128, causal)")
    ap.add_argument("--tile-rows", type=int, default=0, choices=(0, 128, 256),
                    help="query rows per workgroup (qm_attn_set_tile_rows): 0 chooses per call "
                         "from the shape (default); outputs are identical either way")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run a plain 1 GiB device copy (HBM counter calibration)")
    ap.add_argument("--sustain", type=float, default=0.0, metavar="SECONDS",
                    help="instead of the timed steps, run each launch of the workload back to "
                         "back for SECONDS while rocm-smi samples the shader clock, and print "
                         "one JSON line per launch (throughput, clock, throughput per GHz)")
    ap.add_argument("--library", default=None, metavar="PATH",
                    help="load this build of libqm_attn.so instead of the in-tree one "
                         "(to compare builds on one machine)")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the attention forward shards over heads without communication, "
              "so per-GPU throughput is the single-GPU figure)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2506_12355_amd as qa

    if not torch.cuda.is_available():
        print("bench.py needs a ROCm GPU", file=sys.stderr)
        sys.exit(1)
    if args.library:
        qa.load_library(os.path.abspath(args.library))
    else:
        qa.load_library()
    qa.set_tile_rows(args.tile_rows)

    if args.grid:
        run_grid(args, qa, torch, np)
        return

    w = si.WORKLOADS[args.workload]
    fp8 = w.dtype == "e4m3"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if fp8:
        # E4M3 codes with per-tensor scales; the output is bf16
        q, k, v, scales = w.fp8_inputs()
        tdtype = torch.bfloat16
        tq, tk, tv = (torch.from_numpy(x).to(dev) for x in (q, k, v))   # uint8 codes
    else:
        q, k, v = w.inputs()
        scales = None
        tdtype = torch.bfloat16 if w.dtype == "bf16" else torch.float16
        tq, tk, tv = (torch.from_numpy(x.view(np.int16)).to(dev).view(tdtype) for x in (q, k, v))
    if args.layout == "bnhd":
        tq, tk, tv = (t.transpose(1, 2).contiguous() for t in (tq, tk, tv))
    if fp8:
        tq, tk, tv = (t.view(torch.float8_e4m3fn) for t in (tq, tk, tv))
    peak = PEAK_TFLOPS_FP8 if fp8 else PEAK_TFLOPS
    peak_per_clk = PEAK_FLOP_PER_CLK_FP8 if fp8 else PEAK_FLOP_PER_CLK
    masks = list(w.causal)
    oshape = (w.B, w.N, w.H, w.d_v) if args.layout == "bnhd" else (w.B, w.H, w.N, w.d_v)
    outs = [(torch.empty(oshape, dtype=tdtype, device=dev),
             torch.empty((w.B, w.H, w.N), dtype=torch.float32, device=dev))
            for _ in masks]
    stream = torch.cuda.current_stream(dev)

    def launch(m):
        causal = masks[m]
        if fp8:
            qa.fwd_fp8(tq, tk, tv, scales, causal=causal, scale=w.scale, out=outs[m][0],
                       lse=outs[m][1], stream=stream, layout=args.layout)
        else:
            qa.fwd(tq, tk, tv, causal=causal, scale=w.scale, out=outs[m][0],
                   lse=outs[m][1], stream=stream, layout=args.layout)

    def step(ev=None):
        for m in range(len(masks)):
            if ev is not None:
                ev[m].record(stream)
            launch(m)
        if ev is not None:
            ev[len(masks)].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize(dev)

    if args.sustain > 0:
        sustain(args, w, masks, step_one=lambda m: launch(m), dev=dev, stream=stream, torch=torch,
                peak_per_clk=peak_per_clk)
        return

    events = [[torch.cuda.Event(enable_timing=True) for _ in range(len(masks) + 1)]
              for _ in range(args.steps)]
    torch.cuda.synchronize(dev)
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(events[i])
    torch.cuda.synchronize(dev)
    wall = time.perf_counter() - t0
    sclk_mhz, sclk_n, sclk_steps, watts = sustained_sclk(
        step, lambda: torch.cuda.synchronize(dev), enabled=not args.no_sclk)

    launch_ms = [sum(e[m].elapsed_time(e[m + 1]) for e in events) / len(events)
                 for m in range(len(masks))]
    launch_flops = [flops(w.B, w.H, w.N, w.d, c, w.d_v) for c in masks]
    ms_per_step = wall * 1e3 / args.steps
    value = sum(launch_flops) / (ms_per_step * 1e-3) / 1e12
    achieved = launch_flops[0] / (launch_ms[0] * 1e-3) / 1e12
    mask_name = ["causal" if c else "unmasked" for c in masks]
    # the committed counters belong to the in-tree kernel source
    traffic = committed_traffic(w.name) if args.layout == "bhnd" and not args.library else None

    if args.copy_calibration:
        src = torch.empty(1 << 29, dtype=torch.int16, device=dev).fill_(1)
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize(dev)

    result = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "TFLOPS",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {
            "workload": f"{w.name}: {' + '.join(mask_name)} forward per step",
            "B": w.B, "H": w.H, "Hkv": w.kv_heads, "N": w.N, "d": w.d, "d_v": w.d_v,
            "dtype": w.dtype,
            "layout": "[B][N][H][d]" if args.layout == "bnhd" else "[B][H][N][d]",
            "flop_count": ("4·B·H·N²·d" if w.d_v == w.d else "2·B·H·N²·(d + d_v)") + ", ½ if causal",
            "masks": ["causal" if c else "none" for c in masks], "seed": w.seed,
            "tile_rows": args.tile_rows or "auto",
        },
        "pct_of_peak": round(100.0 * value / peak, 2),
        "sclk_mhz": sclk_mhz,
        "pct_of_peak_at_sclk": (round(100.0 * value / (peak_per_clk * sclk_mhz * 1e6 / 1e12), 2)
                                if sclk_mhz else None),
        "package_power_w": watts,
        "sclk_source": (f"median of {sclk_n} rocm-smi readings over {sclk_steps} more steps "
                        "of the same workload, untimed, right after the timed steps"
                        if sclk_mhz else None),
        "per_launch": {
            name: {"ms": round(ms, 4), "tflops": round(f / (ms * 1e-3) / 1e12, 2)}
            for name, ms, f in zip(mask_name, launch_ms, launch_flops)
        },
        "roofline": {
            "bound": "mfma",
            "kernel": f"attn_fwd_kernel<{w.d}, {w.d_v}, {w.dtype}, {mask_name[0]}>",
            "achieved": round(achieved, 2),
            "peak": peak,
            "unit": "TFLOP/s",
            "frac": round(achieved / peak, 4),
            "traffic": traffic,
        },
        # HBM bandwidth of the same launch: the committed counter bytes over this
        # run's launch time (null without a counter summary for this source)
        "hbm": ({"achieved": round(traffic / (launch_ms[0] * 1e-3) / 1e9, 1),
                 "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                 "frac": round(traffic / (launch_ms[0] * 1e-3) / 1e9 / PEAK_HBM_GBPS, 4)}
                if traffic else None),
    }
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(w, q, k, v, descale=scales)
        result["cpu_single_core"] = cpu_single_core()
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
