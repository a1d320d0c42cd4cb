"""Benchmark: one codec round trip (sender encode + receiver decode) of a
synthetic gradient per step, on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]

Prints one JSON line.  `value` is Gelem/s of dense gradient (d / step time)
with the inputs already in device memory; `ms_median`, `ms_p10` and `ms_p90`
are over the timed steps; `hbm_frac` is the round trip's algorithmic bytes
(read g, write and read the payload, write the dense gradient) per step
time over the 8 TB/s HBM peak, and `hbm_frac_of_copy` the same over the
bandwidth a plain 1 GiB device copy reaches on the same GPU
(`copy_ceiling_GBps`, read plus written bytes); `roofline` describes the
kernel that takes the largest share of the step, timed with HIP events on
the library's stream; `cpu_baseline` times the CPU oracle on the same
workload on one host core.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "codec round-trip Gelem/s of dense gradient + % HBM peak; bits/element"
HBM_PEAK = 8.0e12            # B/s, MI355X HBM3E
INT_PEAK = 256 * 64 * 2.4e9  # 32-bit integer lane-ops/s: 256 CUs x 64 lanes/clk x 2.4 GHz
MALL_BYTES = 256 << 20       # last-level cache; inputs rotate through more than this


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_models(d, payload_bytes, n_sel, n_val, k, fill):
    """Algorithmic work of the dominant-kernel candidates, per launch.

    Streaming kernels are priced in the bytes they must move.  The two
    full-range queries are priced in 32-bit integer lane operations: each
    index costs the seed-free half of MurmurHash3 (multiply, rotate,
    multiply: 3 ops) and each probe the seeded half plus the bit test (seed
    xor, rotate, multiply-add, length xor, three xor-shifts, two multiplies,
    the range multiply, word shift, bit shift and mask: 16 ops).  A
    non-member is probed until its first clear bit, (1 - f^k)/(1 - f) probes
    at filter fill f; a positive takes all k.  The sender skips the selected
    set S, whose members it already knows."""
    pn = (1 - fill**k) / (1 - fill) if fill < 1 else k
    enc_ops = (d - n_sel) * 3 + (d - n_val) * 16 * pn + (n_val - n_sel) * 16 * k
    dec_ops = d * 3 + (d - n_val) * 16 * pn + n_val * 16 * k
    return {
        "k_probe<Q_ENCODE>": ("alu", enc_ops),
        "k_probe<Q_DECODE>": ("alu", dec_ops),
        "k_topr_hist": ("hbm", 4.0 * d),
        "k_select_filter": ("hbm", 4.0 * d + d / 8.0),
        "k_emit<Q_DECODE>": ("hbm", 4.0 * d + d / 8.0 + payload_bytes),
    }


def read_profile(kernel, workload):
    """Counter figures of `kernel` on `workload` from the committed rocprofv3
    summary (profiles/pmc_<kernel>_<workload>.txt): HBM bytes per launch and
    the VALU-busy fraction, if that summary was taken on the current kernel
    sources; {} otherwise."""
    import hashlib

    path = os.path.join(ROOT, "profiles", f"pmc_{_slug(kernel)}_{workload}.txt")
    if not os.path.exists(path):
        return {}
    fields = {}
    for line in open(path):
        if ":" in line and not line.startswith(" "):
            key, val = line.split(":", 1)
            fields[key.strip()] = val.strip()
    h = hashlib.sha256()
    for f in sorted(os.listdir(os.path.join(ROOT, "paper_2102_03112_amd", "csrc"))):
        h.update(open(os.path.join(ROOT, "paper_2102_03112_amd", "csrc", f), "rb").read())
    if fields.get("csrc_sha256") != h.hexdigest()[:16]:
        return {}
    out = {}
    for key in ("traffic_bytes_per_launch", "valu_busy"):
        if key in fields:
            out[key] = float(fields[key])
    return out


def copy_ceiling(stream, n_bytes=1 << 30, reps=5):
    """Achievable HBM bandwidth on this part: bytes read plus bytes written
    per second by a plain 1 GiB device-to-device copy (best of `reps`)."""
    import torch

    x = torch.ones(n_bytes // 4, dtype=torch.float32, device="cuda")
    y = torch.empty_like(x)
    y.copy_(x)
    best = float("inf")
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        y.copy_(x)
        e1.record(stream)
        torch.cuda.synchronize()
        best = min(best, e0.elapsed_time(e1) * 1e-3)
    del x, y
    torch.cuda.empty_cache()
    return 2.0 * n_bytes / best


def _slug(kernel):
    return kernel.replace("<", "_").replace(">", "").replace("Q_", "").lower()


def copy_calibration(n_bytes=1 << 30, reps=5):
    """A plain device copy of known size, for scaling the HBM counters."""
    import torch

    x = torch.ones(n_bytes // 4, dtype=torch.float32, device="cuda")
    y = torch.empty_like(x)
    for _ in range(reps):
        y.copy_(x)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": n_bytes, "copy_bytes_written": n_bytes, "reps": reps}), flush=True)


POLICY_NAMES = {0: "P0", 1: "P1", 2: "leftmost", 3: "middle", 4: "rightmost"}


def decode_sum_bench(w, n, steps, warmup, policy, seed):
    """Receiver of an n-worker step: n payloads of the workload (from n
    differently seeded gradients) decoded into one averaged dense gradient by
    dr_payload_decode_sum, against n dr_payload_decode calls whose outputs
    are added by torch on the same stream.  Prints its own JSON line."""
    import dataclasses

    import numpy as np
    import torch

    from paper_2102_03112_amd import binding as B
    from paper_2102_03112_amd import workloads as W

    cfg = B.Config.from_workload(w, policy, seed)
    total, _ = B.payload_layout(cfg)
    ws = B.workspace(w.d, w.n_tensors)
    stream = torch.cuda.current_stream()
    pays = []
    for p in range(n):
        g = torch.from_numpy(W.generate(dataclasses.replace(w, seed=w.seed + 1000 * p))).cuda()
        pay = torch.zeros(total, dtype=torch.uint8, device="cuda")
        B.payload_encode(g, cfg, pay, None, ws, stream)
        pays.append(pay)
        del g
    torch.cuda.synchronize()
    dense = torch.empty(w.d, dtype=torch.float32, device="cuda")
    one = torch.empty(w.d, dtype=torch.float32, device="cuda")

    def fused():
        B.payload_decode_sum(pays, cfg, 1.0 / n, dense, None, ws, stream)

    def separate():
        dense.zero_()
        for pay in pays:
            B.payload_decode(pay, cfg, one, None, None, None, ws, stream)
            dense.add_(one)
        dense.mul_(1.0 / n)

    def timed(fn):
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(steps):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / steps

    ms_f, ms_s = timed(fused), timed(separate)
    log(f"decode_sum: {n} payloads fused {ms_f:.4f} ms, separate {ms_s:.4f} ms")
    print(json.dumps({
        "metric": "receiver Gelem/s of decoded payload elements (n payloads x d)", "value": round(n * w.d / ms_f / 1e6, 4),
        "unit": "Gelem/s", "n_gpus": 1, "steps": steps, "warmup": warmup, "ms_per_step": round(ms_f, 5),
        "separate_ms_per_step": round(ms_s, 5), "speedup_vs_separate": round(ms_s / ms_f, 3),
        "higher_is_better": True, "dtype": "f32", "data": "synthetic",
        "config": {"workload": w.name, "d": w.d, "tensors": w.n_tensors, "payloads": n,
                   "policy": POLICY_NAMES[policy]},
    }), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="resnet50_25m")
    ap.add_argument("--policy", type=int, default=0, help="index policy: 0 = P0 (no error), 1 = P1 (random r of P), "
                                                      "2/3/4 = leftmost/middle/rightmost r of P")
    ap.add_argument("--policy-seed", type=int, default=20210205, help="key of policy 1")
    ap.add_argument("--segmentation", type=int, default=0, help="0 = equal-count runs, 1 = chord splits")
    ap.add_argument("--fit-model", type=int, default=0, help="0 = polynomial, 1 = double exponential")
    ap.add_argument("--n-seg", type=int, default=None, help="runs per tensor (0 = heuristic); default: the "
                                                            "workload's")
    ap.add_argument("--layout", type=int, default=0, help="filter layout: 0 = standard (every hash over the whole "
                                                          "array), 1 = partitioned (hash j over part j of k)")
    ap.add_argument("--no-variants", action="store_true",
                    help="skip timing the partitioned filter layout beside the standard one")
    ap.add_argument("--decode-sum", type=int, default=0, metavar="N",
                    help="instead: time the summing receiver over N payloads of the workload")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget-s", type=float, default=30.0, help="bound on the oracle's CPU time")
    ap.add_argument("--cpu-min-s", type=float, default=10.0,
                    help="the oracle's sample is repeated until it has run this long (at most 8 times)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a 1 GiB device copy (the reference kernel for HBM counter scaling)")
    args = ap.parse_args()

    if args.gpus != 1:
        print(json.dumps({"error": "this codec benchmark runs on one GPU; --gpus must be 1 (the exchange of "
                                   "payloads between GPUs is not part of this build)"}), flush=True)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2102_03112_amd import binding as B
    from paper_2102_03112_amd import workloads as W

    if not torch.cuda.is_available():
        raise SystemExit("bench.py needs a GPU")
    if args.copy_calibration:
        copy_calibration()
        return
    B.lib()  # fail loudly if the HIP library is missing
    w = W.WORKLOADS[args.workload]
    if args.decode_sum:
        decode_sum_bench(w, args.decode_sum, args.steps, args.warmup, args.policy, args.policy_seed)
        return
    d = w.d
    log(f"bench: workload {w.name} d={d} tensors={w.n_tensors}")
    t0 = time.time()
    g_host = W.generate(w)
    log(f"bench: generated input in {time.time() - t0:.1f}s sha256={W.sha256(g_host)[:16]}")

    cfg = B.Config.from_workload(w, args.policy, args.policy_seed, args.segmentation, args.n_seg, args.fit_model,
                                 filter_layout=args.layout)
    total, rec_off = B.payload_layout(cfg)
    n_copies = max(1, min(64, math.ceil(3 * MALL_BYTES / max(1, 4 * d)))) if 4 * d < 2 * MALL_BYTES else 1
    g_dev = [torch.from_numpy(g_host).cuda()]
    for _ in range(n_copies - 1):
        g_dev.append(g_dev[0].clone())
    payload = torch.zeros(total, dtype=torch.uint8, device="cuda")
    dense = torch.empty(d, dtype=torch.float32, device="cuda")
    counts = torch.zeros(4 * w.n_tensors, dtype=torch.int64, device="cuda")
    ws = B.workspace(d, w.n_tensors)
    stream = torch.cuda.current_stream()

    def step(i):
        B.roundtrip(g_dev[i % n_copies], cfg, payload, dense, None, None, counts, ws, stream)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()

    # timed region: an event between consecutive steps gives each step's time
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    evs[0].record(stream)
    for i in range(args.steps):
        step(i)
        evs[i + 1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms = evs[0].elapsed_time(evs[-1]) / args.steps
    per = sorted(evs[i].elapsed_time(evs[i + 1]) for i in range(args.steps))
    pct = lambda q: per[min(len(per) - 1, int(round(q * (len(per) - 1))))]
    log(f"bench: {args.steps} steps, {ms:.4f} ms/step (median {pct(0.5):.4f}, p10 {pct(0.1):.4f}, "
        f"p90 {pct(0.9):.4f}; wall {1e3 * wall / args.steps:.4f} ms/step)")

    # payload accounting from the records
    pay = payload.cpu().numpy()
    cnt = counts.cpu().numpy().reshape(w.n_tensors, 4)
    flags = int(np.bitwise_or.reduce(cnt[:, 3])) if w.n_tensors else 0
    used = idx_bits = val_bits = sig_bits = 0
    fills = []
    n_sel = n_val = 0
    kk = 0
    for t in range(w.n_tensors):
        rec = B.parse_record(pay, rec_off[t])
        used += rec.rec_bytes
        idx_bits += rec.m_bits
        val_bits += 32 * rec.seg_eff * (rec.deg_eff + 1)
        sig_bits += rec.n_values * rec.sigma_b
        n_sel += rec.n_selected
        n_val += rec.n_values
        kk = rec.k
        fills.append(float(np.unpackbits(rec.bits.view(np.uint8)).mean()))
    fill = float(np.mean(fills)) if fills else 0.0
    b_alg = 4.0 * d + 2.0 * used + 4.0 * d
    value = d / (ms * 1e-3) / 1e9

    # per-kernel durations from HIP events on the library's stream
    B.trace_begin(stream)
    for i in range(args.steps):
        step(i)
    tr = B.trace_end()
    kern = {name: (cnt_, tot / cnt_) for name, (cnt_, tot) in tr.items()}  # avg ms per launch
    per_step = {name: tot / args.steps for name, (cnt_, tot) in tr.items()}
    dom = max(per_step, key=per_step.get)
    models = kernel_models(d, used, n_sel, n_val, kk, fill)
    roof = {"kernel": dom, "bound": None, "achieved": None, "peak": None, "unit": None, "frac": None,
            "traffic": None}
    if dom in models:
        bound, work = models[dom]
        avg_s = kern[dom][1] * 1e-3
        ach = work / avg_s / 1e9
        peak = HBM_PEAK / 1e9 if bound == "hbm" else INT_PEAK / 1e9
        roof.update(bound=bound, achieved=round(ach, 1), peak=peak, unit="GB/s" if bound == "hbm" else "Gop/s",
                    frac=round(ach / peak, 4), work_per_launch=work, avg_launch_ms=round(kern[dom][1], 5),
                    launches_per_step=kern[dom][0] / args.steps)
    prof = read_profile(dom, w.name)
    roof["traffic"] = prof.get("traffic_bytes_per_launch")
    roof["valu_busy"] = prof.get("valu_busy")
    ceiling = copy_ceiling(stream)
    log("bench: kernel ms per step: " + ", ".join(f"{k}={v:.4f}" for k, v in sorted(per_step.items(),
                                                                                      key=lambda x: -x[1])))

    # the other filter layout on the same input, timed the same way (a
    # variant beside the headline figure, not the headline)
    variants = {}
    if not args.no_variants and args.layout == 0:
        cfg_p = B.Config.from_workload(w, args.policy, args.policy_seed, args.segmentation, args.n_seg, args.fit_model,
                                       filter_layout=1)

        def step_p(i):
            B.roundtrip(g_dev[i % n_copies], cfg_p, payload, dense, None, None, counts, ws, stream)

        for i in range(args.warmup):
            step_p(i)
        torch.cuda.synchronize()
        pe = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
        pe[0].record(stream)
        for i in range(args.steps):
            step_p(i)
            pe[i + 1].record(stream)
        torch.cuda.synchronize()
        ms_p = pe[0].elapsed_time(pe[-1]) / args.steps
        per_p = sorted(pe[i].elapsed_time(pe[i + 1]) for i in range(args.steps))
        B.trace_begin(stream)
        for i in range(args.steps):
            step_p(i)
        trp = {name: tot / args.steps for name, (cnt_, tot) in B.trace_end().items()}
        cp = counts.cpu().numpy().reshape(w.n_tensors, 4)
        variants["filter_layout_partitioned"] = {
            "ms_per_step": round(ms_p, 5), "ms_median": round(per_p[len(per_p) // 2], 5),
            "value": round(d / (ms_p * 1e-3) / 1e9, 4), "unit": "Gelem/s",
            "hbm_frac": round(b_alg / (ms_p * 1e-3) / HBM_PEAK, 4),
            "flags": int(np.bitwise_or.reduce(cp[:, 3])) if w.n_tensors else 0,
            "positives": int(cp[:, 1].sum()),
            "kernels_ms_per_step": {k: round(v, 5) for k, v in trp.items()},
        }
        log(f"bench: partitioned filter layout {ms_p:.4f} ms/step")

    # CPU oracle baseline on one host core
    cpu = None
    if not args.no_cpu_baseline:
        import oracle

        # a prefix of the gradient with the same per-tensor settings, sized so
        # the oracle (about 3 Melem/s on one core) stays within the budget
        elems = min(d, int(args.cpu_budget_s * 2.5e6))
        off = [o for o in w.offsets() if o < elems] + [elems]
        t0 = time.perf_counter()
        reps = 0
        while True:
            oracle.roundtrip(g_host[:elems], off, w.ratio, w.fpr, w.degree, cfg.n_seg, policy=args.policy,
                             seed=args.policy_seed, seg_mode=args.segmentation, model=args.fit_model)
            reps += 1
            tc = time.perf_counter() - t0
            if tc >= args.cpu_min_s or reps >= 8:
                break
        sample = "full workload" if elems == d else f"first {elems} elements ({len(off) - 1} tensors) of the workload"
        cpu = {"value": round(elems * reps / tc / 1e9, 6), "unit": "Gelem/s", "cores": 1, "kind": "oracle",
               "sample": f"{sample}, {reps} round trip{'s' if reps > 1 else ''}, {tc:.2f} s", "cpu": _cpu_model()}
        log(f"bench: oracle {elems} elements x {reps} in {tc:.2f}s")

    out = {
        "metric": METRIC,
        "value": round(value, 4),
        "unit": "Gelem/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": w.name, "d": d, "tensors": w.n_tensors,
                   "ratio": None if w.ratio is None else f"{w.ratio[0]}/{w.ratio[1]}", "fpr": w.fpr,
                   "degree": w.degree, "n_seg": cfg.n_seg, "policy": POLICY_NAMES[args.policy],
                   "segmentation": ["equal", "chord"][args.segmentation],
                   "fit_model": ["poly", "dexp"][args.fit_model],
                   "filter_layout": ["standard", "partitioned"][args.layout],
                   "input_copies": n_copies},
        "ms_median": round(pct(0.5), 5),
        "ms_p10": round(pct(0.1), 5),
        "ms_p90": round(pct(0.9), 5),
        "hbm_frac": round(b_alg / (ms * 1e-3) / HBM_PEAK, 4),
        "copy_ceiling_GBps": round(ceiling / 1e9, 1),
        "hbm_frac_of_copy": round(b_alg / (ms * 1e-3) / ceiling, 4),
        "bytes_alg": int(b_alg),
        "bits_per_elem": round(8.0 * used / d, 4),
        "bits_split": {"index": round(idx_bits / d, 4), "values": round(val_bits / d, 6),
                       "sigma": round(sig_bits / d, 4)},
        "selected": n_sel,
        "positives": n_val,
        "flags": flags,
        "roofline": roof,
        "kernels_ms_per_step": {k: round(v, 5) for k, v in per_step.items()},
        "variants": variants,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


def _cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip() + f" ({os.cpu_count()} threads visible)"
    except OSError:
        pass
    return None


if __name__ == "__main__":
    main()
