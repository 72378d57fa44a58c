"""Throughput of the PAM matrix-product hot path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload w5]

One step runs every product of the workload once (for the default large
linear layer: forward Y = X .^ W^T, dX = dY .^ W and dW = dY^T .^ X) on
seeded synthetic inputs already resident in HBM.  K steps are timed between
device synchronisations; the printed JSON line reports whole-job PAM-MAC/s
(one PAM-MAC = one piecewise affine product + one float32 accumulate), the
vector-ALU roofline of the dominant kernel measured with HIP events on the
launch stream, and the CPU oracle timed on a bounded sample of the same
workload.
"""
from __future__ import annotations

import argparse
import ctypes
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

# Minimum vector-ALU lane operations per PAM-MAC on gfx950: one int32 add of
# the two encodings (one operand pre-biased once per LDS chunk) and one
# float32 add.
ALGO_LANE_OPS_PER_MAC = 2
# MI355X nominal: 256 CUs x 4 SIMDs x 32 lanes per clock x 2.4 GHz for the
# full-rate ops (int32 add, float32 add/mul/fma) = the 157.3 TFLOP/s
# float32-vector figure counted as one lane op per fma.
NOMINAL_VALU_LANE_OPS = 256 * 4 * 32 * 2.4e9
# Default warm-up: at least this much wall time of untimed steps.  After
# three warm-up steps, w4's first 20 timed steps (0.3-0.4 ms each) ran 4-13%
# slower than the same 20 steps repeated right after them: the GPU had not
# yet left the clock it idled at.
WARMUP_MIN_S = 0.5
# The GEMM kernel's sources: a committed traffic summary is valid only for these bytes.
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2305_17190_amd", "csrc", f)
                  for f in ("pam_kernels.hip", "pam_gemm_dma.hip", "pam_scalar.h")]


def log(msg: str) -> None:
    sys.stderr.write(msg + "\n")
    sys.stderr.flush()


def kernel_source_digest() -> str:
    h = hashlib.sha256()
    for path in KERNEL_SOURCES:
        with open(path, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def committed_counter(workload: str, form: str, key: str):
    """A per-launch figure from the committed rocprofv3 counter summary of one
    product (``traffic_bytes_per_launch``: HBM bytes; ``sustained_clock_ghz``:
    the engine clock the counters saw while the kernel ran).

    Returns None when there is no summary for this kernel or the kernel
    source changed since the counters were taken.
    """
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}_{form}.md")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        text = f.read()
    sha = re.search(r"kernel_source_sha256_16:\s*([0-9a-f]+)", text)
    val = re.search(key + r":\s*([0-9.eE+]+)", text)
    if not sha or not val or sha.group(1) != kernel_source_digest():
        return None
    return float(val.group(1))


class TimingEvents:
    """HIP events used only for timing, recorded on the launch stream.

    They are created with hipEventDisableSystemFence: recording a default
    event ends with a system-scope fence (cache write-back and invalidate),
    which between products as short as w4's (~0.05 ms) added ~3.5 us per
    event to the step and to the bracketed launch itself.  The elapsed times
    are read only after a device synchronisation.
    """
    DISABLE_SYSTEM_FENCE = 0x20000000

    def __init__(self, stream_handle: int):
        # The HIP runtime the process already loaded (torch's; the library
        # links the same soname), never a second copy.
        path = None
        with open("/proc/self/maps") as fh:
            for line in fh:
                if "libamdhip64" in line:
                    path = line.split()[-1]
                    break
        if path is None:
            raise RuntimeError("the HIP runtime is not loaded")
        hip = ctypes.CDLL(path)
        vp = ctypes.c_void_p
        hip.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(vp), ctypes.c_uint]
        hip.hipEventRecord.argtypes = [vp, vp]
        hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), vp, vp]
        hip.hipEventDestroy.argtypes = [vp]
        self.hip = hip
        self.stream = vp(stream_handle)
        self.events = []

    def _check(self, status: int, what: str) -> None:
        if status != 0:
            raise RuntimeError(f"{what} failed with HIP error {status}")

    def new(self):
        ev = ctypes.c_void_p()
        self._check(self.hip.hipEventCreateWithFlags(ctypes.byref(ev), self.DISABLE_SYSTEM_FENCE),
                    "hipEventCreateWithFlags")
        self.events.append(ev)
        return ev

    def record(self, ev) -> None:
        self._check(self.hip.hipEventRecord(ev, self.stream), "hipEventRecord")

    def elapsed_ms(self, start, end) -> float:
        ms = ctypes.c_float()
        self._check(self.hip.hipEventElapsedTime(ctypes.byref(ms), start, end), "hipEventElapsedTime")
        return ms.value

    def close(self) -> None:
        for ev in self.events:
            self.hip.hipEventDestroy(ev)
        self.events = []


def cpu_baseline(workload_id: int, host, forms, target_s: float) -> dict:
    """Time the C oracle on a bounded slice of every product of the workload."""
    import numpy as np
    from oracle import pam_c

    pam_c.load()
    threads = pam_c.num_threads()

    def run(form, count):
        a, b = host[form.a], host[form.b]
        if form.batch > 1:
            bats = list(range(count))
            t0 = time.perf_counter()
            pam_c.pam_gemm(a, b, form.trans_a, form.trans_b, form.m, form.n, form.k, form.lda, form.ldb,
                           form.stride_a, form.stride_b, batches=bats)
            return time.perf_counter() - t0, count * form.m * form.n * form.k
        rows = list(range(count))
        t0 = time.perf_counter()
        pam_c.pam_gemm(a, b, form.trans_a, form.trans_b, form.m, form.n, form.k, form.lda, form.ldb, rows=rows)
        return time.perf_counter() - t0, count * form.n * form.k

    def sample(target, start):
        # Probe with a small slice per product, then scale the slice to the target time.
        per_form = target / len(forms)
        total_t, total_macs, parts = 0.0, 0, []
        for form in forms:
            limit = form.batch if form.batch > 1 else form.m
            count = min(limit, max(1, start))
            t, macs = run(form, count)
            if t < per_form / 4:
                count = min(limit, max(count, int(count * per_form / max(t, 1e-3))))
                t, macs = run(form, count)
            total_t += t
            total_macs += macs
            parts.append(f"{form.name}: {count} {'batch entries' if form.batch > 1 else 'rows'}")
        return total_macs, total_t, parts

    total_macs, total_t, parts = sample(target_s, threads)
    # The same oracle on one core, on a smaller sample.
    pam_c.set_threads(1)
    try:
        one_macs, one_t, one_parts = sample(max(1.0, target_s / 8), 1)
    finally:
        pam_c.set_threads(threads)
    return {
        "value": total_macs / total_t / 1e9,
        "unit": "GPAM-MAC/s",
        "cores": threads,
        "kind": "oracle",
        "sample": f"workload {workload_id} ({'; '.join(parts)}), C oracle, float64 accumulate, "
                  f"{total_macs:.3e} PAM-MACs in {total_t:.1f} s",
        "one_core": {"value": one_macs / one_t / 1e9, "unit": "GPAM-MAC/s",
                     "sample": f"{'; '.join(one_parts)}, {one_macs:.3e} PAM-MACs in {one_t:.1f} s"},
    }


ELEMENTWISE_OPS = {
    # op: (binding name, kernel, bytes per element, input description)
    "mul": ("mul", "binary_vec4_kernel<PamOp>", 12, "N(0,1) with 1% zeros and 1% powers of two"),
    "pad": ("pad", "binary_vec4_kernel<PadOp>", 12, "N(0,1) with 1% zeros and 1% powers of two"),
    "palog2": ("palog2", "unary_vec4_kernel<Palog2Op>", 8, "|N(0,1)| with 1% zeros and 1% powers of two"),
    "paexp2": ("paexp2", "unary_vec4_kernel<Paexp2Op>", 8, "softmax-shaped arguments"),
}


def warm_up(args, torch, step) -> None:
    """Untimed steps before the timed region: args.warmup of them, or, when
    --warmup is not given, at least three and at least WARMUP_MIN_S seconds
    (synchronising after each, so that the GPU has left its idle clock);
    args.warmup is set to the number run."""
    t_warm = time.perf_counter()
    done = 0
    while done < args.warmup or (args.warmup_auto and time.perf_counter() - t_warm < WARMUP_MIN_S):
        step()
        done += 1
        if args.warmup_auto:
            torch.cuda.synchronize()
    args.warmup = done
    torch.cuda.synchronize()


def bench_elementwise(args, torch, wl, pam, dev) -> int:
    """One elementwise op on N elements: 8 bytes read and 4 written per element
    (two-operand ops), or 4 read and 4 written (one-operand ops)."""
    n = args.elementwise
    name, kernel, nbytes, desc = ELEMENTWISE_OPS[args.elementwise_op]
    fn = getattr(pam, name)
    if args.elementwise_op == "paexp2":
        a = wl.paexp2_arguments(n, 1000 + 4)
        ins = (torch.from_numpy(a).to(dev),)
    else:
        a, b = wl.pam_mul_inputs(n, 1000 + 3)
        ins = (torch.from_numpy(a).to(dev), torch.from_numpy(b).to(dev))
        if args.elementwise_op == "palog2":
            ins = (ins[0].abs(),)
    out = torch.empty_like(ins[0])
    warm_up(args, torch, lambda: fn(*ins, out=out))
    s = torch.cuda.Event(enable_timing=True)
    e = torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    s.record()
    for _ in range(args.steps):
        fn(*ins, out=out)
    e.record()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    launch_s = s.elapsed_time(e) / 1e3 / args.steps
    gbs = float(nbytes) * n / launch_s / 1e9
    result = {
        "metric": f"elementwise {args.elementwise_op} throughput",
        "value": round(n / launch_s / 1e9, 3),
        "unit": "G elements/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(elapsed / args.steps * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u32",
        "data": "synthetic",
        "config": {"workload": f"{args.elementwise_op} n={n}, {desc}"},
        "roofline": {"bound": "hbm", "kernel": kernel, "achieved": round(gbs, 1),
                     "peak": 8000.0, "unit": "GB/s", "frac": round(gbs / 8000.0, 4), "traffic": None,
                     "bytes_per_element": nbytes, "avg_launch_ms": round(launch_s * 1e3, 5)},
    }
    print(json.dumps(result), flush=True)
    return 0


def bench_autograd(args, torch, wl, pam, dev) -> int:
    """One PAM linear layer through autograd: forward Y = X .^ W^T, then
    backward with the approximate derivative (dX = dY .^ W, dW = dY^T .^ X)
    on the workload's tensors -- the same three products as the default step,
    plus the wrapper's own work."""
    from paper_2305_17190_amd.autograd import pam_linear

    wid = int(args.workload[1:])
    spec = wl.WORKLOADS[wid]
    names = [f.name for f in spec["forms"]]
    if names != ["fwd", "dX", "dW"]:
        print(f"--autograd needs a single-linear-layer workload (w2 or w5), not {args.workload}", file=sys.stderr)
        return 2
    host = wl.workload_inputs(wid)
    x = torch.from_numpy(host["X"]).to(dev).requires_grad_()
    w = torch.from_numpy(host["W"]).to(dev).requires_grad_()
    dy = torch.from_numpy(host["dY"]).to(dev)
    macs = sum(f.macs for f in spec["forms"])

    derivative = "exact" if args.exact_grad else "approximate"

    def step():
        x.grad = None
        w.grad = None
        pam_linear(x, w, derivative=derivative).backward(dy)

    warm_up(args, torch, step)
    s = torch.cuda.Event(enable_timing=True)
    e = torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    s.record()
    for _ in range(args.steps):
        step()
    e.record()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    step_s = s.elapsed_time(e) / 1e3 / args.steps
    log(f"autograd step {step_s * 1e3:.3f} ms ({macs / step_s / 1e9:.1f} GPAM-MAC/s)")
    result = {
        "metric": "PAM linear layer forward + backward through autograd, G PAM-MAC/s",
        "value": round(macs / step_s / 1e9, 3),
        "unit": "GPAM-MAC/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(elapsed / args.steps * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": spec["name"], "layer": "paper_2305_17190_amd.autograd.pam_linear, no bias",
                   "derivative": derivative, "pam_macs_per_step": macs},
    }
    print(json.dumps(result), flush=True)
    return 0


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=None,
                    help="untimed warm-up steps (default: at least 3, and at least 0.5 s of them, so that short "
                         "steps are not timed while the GPU's clock is still rising from idle)")
    ap.add_argument("--workload", default="w5", choices=["w1", "w2", "w3", "w4", "w5"])
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 1 GiB device-to-device copy (reference kernel for HBM counters)")
    ap.add_argument("--elementwise", type=int, default=0, metavar="N",
                    help="time only one elementwise op on N elements (HBM roofline) and print its line")
    ap.add_argument("--mantissa-bits", type=int, default=23,
                    help="round every operand to this many mantissa bits first (narrow products; default 23 = none)")
    ap.add_argument("--bf16", action="store_true",
                    help="the workload's operands stored as bfloat16 (rounded once, before timing), products of "
                         "the bfloat16 operands with float32 results")
    ap.add_argument("--autograd", action="store_true",
                    help="time one PAM linear layer forward + backward through autograd (w2, w5)")
    ap.add_argument("--exact-grad", action="store_true",
                    help="with --autograd: backward with the exact derivative (Table 1) instead of the approximate one")
    ap.add_argument("--elementwise-op", default="mul", choices=sorted(ELEMENTWISE_OPS),
                    help="the elementwise op --elementwise times (default mul)")
    args = ap.parse_args()
    args.warmup_auto = args.warmup is None
    if args.warmup is None:
        args.warmup = 3

    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}); the PAM matrix product is "
              "built and measured on a single MI355X.", file=sys.stderr)
        return 2

    import torch

    import pam_workloads as wl
    import paper_2305_17190_amd as pam

    if not torch.cuda.is_available():
        print("bench.py needs a HIP device", file=sys.stderr)
        return 1
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.copy_calibration:
        src = torch.ones(1 << 28, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        log(f"copied 3 x {src.numel() * 4} bytes")
        return 0
    pam.load()
    if args.elementwise:
        return bench_elementwise(args, torch, wl, pam, dev)
    if args.autograd:
        return bench_autograd(args, torch, wl, pam, dev)

    wid = int(args.workload[1:])
    spec = wl.WORKLOADS[wid]
    forms = spec["forms"]
    log(f"generating workload {wid} ({spec['desc']})")
    host = wl.workload_inputs(wid)
    dt = {k: torch.from_numpy(v).to(dev) for k, v in host.items()}
    if args.bf16:
        dt = {k: v.to(torch.bfloat16) for k, v in dt.items()}
    outs = {}
    for f in forms:
        shape = (f.batch, f.m, f.n) if f.batch > 1 else (f.m, f.n)
        outs[f.name] = torch.empty(shape, dtype=torch.float32, device=dev)

    def launch(f):
        if f.batch > 1:
            pam.bmm(dt[f.a], dt[f.b], trans_a=f.trans_a, trans_b=f.trans_b, out=outs[f.name],
                    mantissa_bits=args.mantissa_bits)
        else:
            pam.gemm(dt[f.a], dt[f.b], trans_a=f.trans_a, trans_b=f.trans_b, out=outs[f.name],
                     mantissa_bits=args.mantissa_bits)

    macs_per_step = sum(f.macs for f in forms)
    def one_step():
        for f in forms:
            launch(f)

    warm_up(args, torch, one_step)

    # Per-product events on the stream the products are launched on,
    # created before the timed region.
    timer = TimingEvents(torch.cuda.current_stream().cuda_stream)
    events = {f.name: [(timer.new(), timer.new()) for _ in range(args.steps)] for f in forms}
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        for f in forms:
            s, e = events[f.name][i]
            timer.record(s)
            launch(f)
            timer.record(e)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0

    per_form, med_form = {}, {}
    for f in forms:
        ms = sorted(timer.elapsed_ms(s, e) for s, e in events[f.name])
        per_form[f.name] = sum(ms) / len(ms)
        med_form[f.name] = ms[len(ms) // 2] if len(ms) % 2 else 0.5 * (ms[len(ms) // 2 - 1] + ms[len(ms) // 2])
        log(f"  {f.name:6s} m={f.m} n={f.n} k={f.k} batch={f.batch} plan={pam.plan(f.m, f.n, f.k, f.batch)} "
            f"avg {per_form[f.name]:.3f} ms median {med_form[f.name]:.3f} ms  "
            f"{f.macs / med_form[f.name] / 1e9:.1f} GPAM-MAC/s")
    timer.close()

    info = pam.device_info(0)
    peak = NOMINAL_VALU_LANE_OPS
    dom = max(forms, key=lambda f: per_form[f.name] * 1.0)
    dom_s = per_form[dom.name] / 1e3
    achieved = ALGO_LANE_OPS_PER_MAC * dom.macs / dom_s
    achieved_median = ALGO_LANE_OPS_PER_MAC * dom.macs / (med_form[dom.name] / 1e3)
    clock_ghz = committed_counter(spec["name"], dom.name, "sustained_clock_ghz")
    value = macs_per_step * args.steps / elapsed / 1e9
    log(f"device: {info}")
    log(f"step {elapsed / args.steps * 1e3:.3f} ms, {value:.1f} GPAM-MAC/s; dominant {dom.name}: "
        f"{achieved / 1e12:.2f} of {peak / 1e12:.2f} Tlane-op/s (device-read peak "
        f"{info['valu_lane_ops_per_s'] / 1e12:.2f})")

    result = {
        "metric": "PAM-GEMM G PAM-MAC/s on one MI355X; % of VALU op-rate peak",
        "value": round(value, 3),
        "unit": "GPAM-MAC/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(elapsed / args.steps * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": spec["name"],
            "products": [f"{f.name} ({'T' if f.trans_a else 'N'}{'T' if f.trans_b else 'N'}) "
                         f"{f.batch}x{f.m}x{f.n}x{f.k}" for f in forms],
            "pam_macs_per_step": macs_per_step,
            "parallelism": "single GPU",
            **({"mantissa_bits": args.mantissa_bits} if args.mantissa_bits != 23 else {}),
            **({"operands": "bfloat16"} if args.bf16 else {}),
        },
        "roofline": {
            "bound": "alu",
            "kernel": f"pam_gemm_dma_kernel {dom.name} "
                      f"({'T' if dom.trans_a else 'N'}{'T' if dom.trans_b else 'N'})",
            "achieved": round(achieved / 1e12, 3),
            "peak": round(peak / 1e12, 3),
            "unit": "Tlane-op/s",
            "frac": round(achieved / peak, 4),
            "traffic": committed_counter(spec["name"], dom.name, "traffic_bytes_per_launch"),
            "lane_ops_per_mac": ALGO_LANE_OPS_PER_MAC,
            "avg_launch_ms": round(per_form[dom.name], 4),
            "median_launch_ms": round(med_form[dom.name], 4),
            "frac_median": round(achieved_median / peak, 4),
            "device_peak": round(info["valu_lane_ops_per_s"] / 1e12, 3),
            # the engine clock rocprofv3's counters saw for this kernel (the
            # chip runs below its 2.4 GHz peak under this load), and the
            # fraction of the peak priced at that clock
            "sustained_clock_ghz": clock_ghz,
            "frac_at_sustained_clock": (round(achieved / (peak * clock_ghz / 2.4), 4) if clock_ghz else None),
        },
        "products": {f.name: {"median_ms": round(med_form[f.name], 4), "avg_ms": round(per_form[f.name], 4),
                              "gpam_mac_s": round(f.macs / med_form[f.name] / 1e6, 1),
                              "frac": round(ALGO_LANE_OPS_PER_MAC * f.macs / (med_form[f.name] / 1e3) / peak, 4)}
                     for f in forms},
    }
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on a bounded sample")
        result["cpu_baseline"] = cpu_baseline(wid, host, forms, args.cpu_seconds)
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
