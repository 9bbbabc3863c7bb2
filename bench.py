"""DPB benchmark on one MI355X: encode + decode + decode-backward per step.

    python bench.py [--steps K] [--warmup W] [--workload train]

A step is one pass of the whole path over one batch: encode x -> (idx, coef),
decode -> y, and decode-backward of an upstream gradient g -> (grad_coef,
grad_x).  The three kernels are timed separately with HIP events between
them (dpb_forward, the encode + decode call, enqueues the same two kernels).
Inputs are seeded synthetic activations resident in HBM before the timed
region; three input sets rotate so that their total (>600 MB at the default
workload) exceeds the 256 MB Infinity Cache.

Prints ONE JSON line.  `roofline` describes the kernel with the largest average
launch time, timed with HIP events on the stream the kernels run on;
`extras` times the layer epilogues (normalization and its backward), the code
edits, the variance auxiliary loss and the whole autograd layer at the same
shape, after the timed steps; `cpu_baseline` times the CPU oracle on a bounded
sample of the same workload.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_2607_20652_amd import binding as dpb  # noqa: E402
from paper_2607_20652_amd import inputs  # noqa: E402

METRIC = "DPB fwd+bwd tokens/sec at d=768,N=2^20,k=64; % of HBM/VALU roofline"
HBM_PEAK_GBS = 8000.0
VALU_PEAK_TFLOPS = 157.3    # fp32 vector, 256 CUs at 2.4 GHz
MFMA_BF16_PEAK_TFLOPS = 2500.0
CSRC = os.path.join(ROOT, "paper_2607_20652_amd", "csrc")
COPY_BYTES = 256 << 20      # size of the plain copy that calibrates the HBM byte counters
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic.json")


def kernel_source_digest() -> str:
    """Digest of every source the encode / decode / backward kernels and their
    plan tables are built from (the row epilogues and code utilities in
    extras.hip do not affect them)."""
    h = hashlib.sha256()
    for f in sorted(os.listdir(CSRC)):
        if f.endswith((".hip", ".hpp", ".cpp")) and f != "extras.hip":
            h.update(f.encode())
            h.update(open(os.path.join(CSRC, f), "rb").read())
    return h.hexdigest()[:16]


KERNEL_SYMBOLS = {"encode": "encode3_kernel", "decode": "decode2_kernel", "decode_bwd": "decode_bwd2_kernel"}


def ingest_counters(fetch_csv: str, write_csv: str, workload: str) -> dict:
    """HBM bytes per launch from two rocprofv3 --pmc runs (FETCH_SIZE, WRITE_SIZE,
    KiB per dispatch) of `bench.py --only K --with-copy`, each scaled by what the
    same counter reads for the plain copy of COPY_BYTES in the same run."""
    import csv

    def per_kernel(path, counter):
        acc = {}
        for r in csv.DictReader(open(path)):
            if r["Counter_Name"] != counter:
                continue
            name = r["Kernel_Name"]
            key = "copy"  # runtime copies and fills
            for k, sym in KERNEL_SYMBOLS.items():
                if sym in name:
                    key = k
            acc.setdefault(key, []).append(float(r["Counter_Value"]) * 1024.0)
        if not acc.get("copy"):
            raise SystemExit(f"{path}: no calibrating copy dispatch")
        out = {k: float(np.median(v)) for k, v in acc.items() if k != "copy"}
        # plan set-up also issues KB-sized runtime copies; the calibrating copy is the largest
        out["copy"] = max(acc["copy"])
        return out

    fetch, write = per_kernel(fetch_csv, "FETCH_SIZE"), per_kernel(write_csv, "WRITE_SIZE")
    f_scale = COPY_BYTES / fetch["copy"]
    w_scale = COPY_BYTES / write["copy"]
    T = inputs.workload(workload).tokens
    rec = {"kernel_source_digest": kernel_source_digest(), "workload": workload,
           "copy_bytes": COPY_BYTES, "fetch_scale": f_scale, "write_scale": w_scale, "kernels": {}}
    for k in KERNEL_SYMBOLS:
        if k in fetch and k in write:
            rec["kernels"][k] = {"tokens": T, "fetch_bytes": fetch[k] * f_scale, "write_bytes": write[k] * w_scale,
                                 "hbm_bytes_per_launch": fetch[k] * f_scale + write[k] * w_scale}
    return rec


def algorithmic_bytes_per_token(w, k_tot: int) -> dict:
    """HBM bytes each kernel must move per token (inputs read once, outputs written once)."""
    xb = 2 if w.dtype == "bf16" else 4
    return {
        "forward": w.d * xb + k_tot * 8 + w.d * xb,        # read x, write (idx, coef), write y
        "encode": w.d * xb + k_tot * 8,                    # read x, write (idx, coef)
        "decode": k_tot * 8 + w.d * xb,                    # read (idx, coef), write y
        "decode_bwd": k_tot * 4 + w.d * xb + k_tot * 4 + w.d * xb,  # read idx, g; write grad_coef, grad_x
    }


def algorithmic_flops_per_token(w, plan_k_tot: int, hier) -> dict:
    """Arithmetic the method must do per token, 2 flops per multiply-add.

    encode: child scoring, sum over levels l >= 1 of K_{l-1} Delta_l d +-1 products
    (a dense contraction, on the matrix cores); decode: one signed add per hashed
    slot and coordinate; decode_bwd: the same for grad_coef and again for grad_x.
    """
    nbits, delta, active = hier
    hashed = plan_k_tot - active[0]
    score = sum(active[l - 1] * delta[l] for l in range(1, len(active))) * w.d
    return {"forward": 2 * score + 2 * hashed * w.d, "encode": 2 * score, "decode": 2 * hashed * w.d,
            "decode_bwd": 4 * hashed * w.d}


def load_traffic(kernel: str, tokens: int):
    """Measured HBM bytes per launch from the committed rocprofv3 counter runs,
    if they were taken on the current kernel sources; else None."""
    try:
        rec = json.load(open(TRAFFIC_FILE))
    except (OSError, ValueError):
        return None
    if rec.get("kernel_source_digest") != kernel_source_digest():
        return None
    k = rec.get("kernels", {}).get(kernel)
    if not k or k.get("tokens") != tokens:
        return None
    return k.get("hbm_bytes_per_launch")


def time_extras(plan, w, sets, act, steps: int) -> dict:
    """Times the layer epilogues and code utilities at the workload's shape
    (inputs resident in HBM, HIP events on the current stream) and the whole
    DPB layer (encode, decode, normalization, variance loss and their
    backward) as an autograd Function.  Bytes are what each kernel must move:
    every input read once, every output written once."""
    from paper_2607_20652_amd import autograd as dpb_autograd

    T, d, k = w.tokens, w.d, plan.k_tot
    xb = 2 if act == torch.bfloat16 else 4
    dev = sets[0][0].device
    x, g = sets[0]
    idx, coef = dpb.encode(plan, x)
    u = dpb.decode(plan, idx, coef, act)
    y = torch.empty_like(u)
    gref = torch.empty_like(u)
    ws = dpb.variance_workspace(plan, T, dev)
    gen = torch.Generator().manual_seed(5)
    rows = torch.arange(T, dtype=torch.int32).to(dev)
    slots = torch.randint(0, k, (T,), generator=gen, dtype=torch.int32).to(dev)
    ops = torch.randint(0, 3, (T,), generator=gen, dtype=torch.int32).to(dev)
    tidx, tcoef = dpb.encode(plan, sets[1][0])
    n_min = 2
    xg = x.detach().clone().requires_grad_(True)

    def layer():
        yy, lv = dpb_autograd.dpb_layer(xg, plan, True, n_min)
        torch.autograd.backward([yy, lv], [g, torch.ones((), device=dev)])
        xg.grad = None

    stats, m2 = dpb.std_state(plan, dev)
    stats.copy_(torch.stack([0.1 * torch.randn(stats.shape[0], generator=gen),
                             torch.rand(stats.shape[0], generator=gen) + 0.5], dim=1))
    sidx = torch.empty_like(idx)
    scoef = torch.empty_like(coef)
    sws = dpb.std_workspace(plan, dev)
    cases = {
        "encode_std": (lambda: dpb.encode_std(plan, x, stats, sidx, scoef), d * xb + 8 * k),
        "std_update": (lambda: dpb.std_update(plan, x, sidx, stats, m2, 0.0, 1e-6, sws), d * xb),
        "normalize": (lambda: dpb.normalize(plan, u, x, y=y), 3 * d * xb),
        "normalize_bwd": (lambda: dpb.normalize_bwd(plan, g, u, x, grad_ref=gref), 5 * d * xb),
        "variance_loss": (lambda: dpb.variance_loss(plan, idx, coef, n_min, workspace=ws), 12 * k),
        "edit_codes": (lambda: dpb.edit_codes(plan, idx, coef, rows, slots, ops, tidx, tcoef), 16 * k),
        "layer_fwd_bwd": (layer, None),
    }
    res = {}
    for name, (fn, bpt) in cases.items():
        try:
            fn()
        except dpb.DPBError as e:        # a call outside the library's limits for this hierarchy
            res[name] = {"unsupported": str(e)}
            continue
        for _ in range(2):
            fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(steps):
            fn()
        b.record()
        torch.cuda.synchronize()
        ms = a.elapsed_time(b) / steps
        rec = {"ms": round(ms, 4)}
        if bpt is not None:
            gbs = bpt * T / (ms * 1e-3) / 1e9
            rec.update({"bytes_per_launch": bpt * T, "hbm_GBps": round(gbs, 1), "hbm_frac": round(gbs / HBM_PEAK_GBS, 4)})
        else:
            rec["tokens_per_s"] = round(T / (ms * 1e-3), 1)
        res[name] = rec
    notes = {"variance_loss": {"n_min": n_min}, "edit_codes": {"edits": T},
             "layer_fwd_bwd": {"what": "autograd DPB layer: encode, decode, normalization, variance loss and backward"},
             "encode_std": {"what": "encode on standardized scores (random EMA statistics)"},
             "std_update": {"what": "EMA statistics update (all tokens for level 0, 64 sampled tokens above; "
                                    "momentum 0)"}}
    for k2, v in notes.items():
        if "ms" in res.get(k2, {}):
            res[k2].update(v)
    return res


def cpu_baseline(name: str, target_s: float = 12.0) -> dict:
    """The oracle (fp64 C, OpenMP over tokens) on a bounded sample of the workload."""
    import oracle

    w = inputs.workload(name)
    h = w.hierarchy()
    nb, dl, K = h if h is not None else oracle.hierarchy(w.d, w.n, w.levels, w.branching, w.beam, w.k)
    m = oracle.masks(w.d, w.n)
    gens = oracle.generators(nb, dl, 0)

    def run(T):
        x = inputs.activations(name, T).double().numpy()
        g = inputs.upstream_grad(name, T).double().numpy()
        t = time.perf_counter()
        idx, coef, _, _ = oracle.encode(w.d, m, nb, K, dl, gens, x)
        oracle.decode(w.d, m, idx, coef)
        oracle.decode_bwd(w.d, m, idx, g)
        return time.perf_counter() - t

    probe = 256
    t_probe = run(probe)
    T = int(min(w.tokens, max(probe, probe * target_s / max(t_probe, 1e-3))))
    t = run(T)
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    out = {
        "value": T / t,
        "unit": "tokens/s",
        "cores": oracle.num_threads(),
        "kind": "oracle",
        "sample": f"first {T} of {w.tokens} tokens of '{name}' (encode+decode+decode_bwd), {t:.1f} s",
        "cpu_model": model,
        "logical_cpus": os.cpu_count(),
    }
    # the same oracle on one thread, on the first tokens: the OpenMP
    # runtime the oracle runs on is set to one thread and back
    import ctypes
    try:
        gomp = ctypes.CDLL("libgomp.so.1")
        before = gomp.omp_get_max_threads()
        gomp.omp_set_num_threads(1)
        try:
            used = oracle.num_threads()
            # up to 1,024 tokens, fewer where one thread would take more than ~10 s
            T1 = int(max(64, min(1024, 10.0 * out["value"] / max(out["cores"], 1))))
            t1 = cpu_oracle_seconds(name, T1)
        finally:
            gomp.omp_set_num_threads(before)
        out["single_thread"] = {"value": T1 / t1, "unit": "tokens/s", "tokens": T1, "seconds": round(t1, 2),
                                "threads": used}
    except OSError:
        out["single_thread"] = None
    return out


def cpu_oracle_seconds(name: str, T: int) -> float:
    """Seconds the oracle takes for encode + decode + decode_bwd of the first T
    tokens of the workload (the threads OpenMP gives it)."""
    import oracle

    w = inputs.workload(name)
    h = w.hierarchy()
    nb, dl, K = h if h is not None else oracle.hierarchy(w.d, w.n, w.levels, w.branching, w.beam, w.k)
    m = oracle.masks(w.d, w.n)
    gens = oracle.generators(nb, dl, 0)
    x = inputs.activations(name, T).double().numpy()
    g = inputs.upstream_grad(name, T).double().numpy()
    t = time.perf_counter()
    idx, coef, _, _ = oracle.encode(w.d, m, nb, K, dl, gens, x)
    oracle.decode(w.d, m, idx, coef)
    oracle.decode_bwd(w.d, m, idx, g)
    return time.perf_counter() - t


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="train")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extras", action="store_true",
                    help="skip timing the normalization, edit and variance-loss kernels and the autograd layer")
    ap.add_argument("--only", choices=["encode", "decode", "decode_bwd"], default=None,
                    help="time a single kernel (for counter runs)")
    ap.add_argument("--with-copy", action="store_true",
                    help="also run one plain device copy of a known size (calibrates byte counters)")
    ap.add_argument("--ingest-counters", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="write the committed HBM-traffic record from two counter runs and exit")
    args = ap.parse_args()

    if args.ingest_counters:
        rec = ingest_counters(*args.ingest_counters, args.workload)
        with open(TRAFFIC_FILE, "w") as f:
            json.dump(rec, f, indent=1)
        print(json.dumps(rec))
        return 0

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py: measures one GPU only; the DPB shards by tokens with no "
              "communication, so a multi-GPU figure is N times the one-GPU value (not measured).",
              file=sys.stderr)
        return 2
    if not torch.cuda.is_available():
        print("bench.py: no GPU", file=sys.stderr)
        return 2
    if not os.path.exists(dpb.lib_path):
        from paper_2607_20652_amd import build
        build.build()

    w = inputs.workload(args.workload)
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    plan = dpb.Plan(w.d, seed=0, **w.plan_kwargs())
    T, k = w.tokens, plan.k_tot
    act = torch.bfloat16 if w.dtype == "bf16" else torch.float32

    # three rotating input sets, resident in HBM before timing
    x0, g0 = inputs.activations(args.workload), inputs.upstream_grad(args.workload)
    sets = []
    for r in range(3):
        sets.append((torch.roll(x0, shifts=r * 7919, dims=0).to(dev).contiguous(),
                     torch.roll(g0, shifts=r * 7919, dims=0).to(dev).contiguous()))
    idx = torch.empty((T, k), dtype=torch.int32, device=dev)
    coef = torch.empty((T, k), dtype=torch.float32, device=dev)
    y = torch.empty((T, w.d), dtype=act, device=dev)
    gc = torch.empty((T, k), dtype=torch.float32, device=dev)
    gx = torch.empty((T, w.d), dtype=act, device=dev)

    names = ["encode", "decode", "decode_bwd"]
    run = {n: (args.only is None or args.only == n) for n in names}

    def step(i, ev=None):
        x, g = sets[i % 3]
        for j, n in enumerate(names):
            if ev is not None:
                ev[j].record()
            if not run[n]:
                continue
            if n == "encode":
                dpb.encode(plan, x, idx, coef)
            elif n == "decode":
                dpb.decode(plan, idx, coef, act, y)
            else:
                dpb.decode_bwd(plan, idx, g, act, gc, gx)
        if ev is not None:
            ev[len(names)].record()

    if args.only in ("decode", "decode_bwd"):
        dpb.encode(plan, sets[0][0], idx, coef)  # codes for the kernels under test
    if args.with_copy:
        src = torch.empty(COPY_BYTES // 4, dtype=torch.float32, device=dev)  # contents are irrelevant
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()

    nev = len(names) + 1
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(nev)] for _ in range(args.steps)]
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for i in range(args.steps):
        step(i, evs[i])
    end.record()
    torch.cuda.synchronize()
    ms_total = start.elapsed_time(end)
    ms_step = ms_total / args.steps
    step_ms = [evs[i][0].elapsed_time(evs[i][nev - 1]) for i in range(args.steps)]
    launch_ms = {n: [evs[i][j].elapsed_time(evs[i][j + 1]) for i in range(args.steps)] for j, n in enumerate(names)}
    per_kernel_ms = {n: float(np.mean(v)) for n, v in launch_ms.items()}

    bpt = algorithmic_bytes_per_token(w, k)
    fpt = algorithmic_flops_per_token(w, k, (plan.level_bits, plan.branching, plan.active))
    timed = [n for n in names if run[n]]
    dom = max(timed, key=lambda n: per_kernel_ms[n])
    per_kernel = {}
    for n in timed:
        sec = per_kernel_ms[n] * 1e-3
        hbm = bpt[n] * T / sec / 1e9
        tfl = fpt[n] * T / sec / 1e12
        peak = MFMA_BF16_PEAK_TFLOPS if n == "encode" else VALU_PEAK_TFLOPS
        per_kernel[n] = {"ms": round(per_kernel_ms[n], 4), "ms_median": round(float(np.median(launch_ms[n])), 4),
                         "hbm_GBps": round(hbm, 1),
                         "hbm_frac": round(hbm / HBM_PEAK_GBS, 4), "tflops": round(tfl, 2),
                         "compute_peak_tflops": peak, "compute_frac": round(tfl / peak, 4)}
    # decode and decode-backward are bound by the vector ALU (sign generation and
    # signed accumulation); the encoder's contraction runs on the matrix cores
    bound = "mfma" if dom == "encode" else "alu"
    roofline = {
        "kernel": dom,
        "bound": bound,
        "achieved": per_kernel[dom]["tflops"],
        "peak": per_kernel[dom]["compute_peak_tflops"],
        "unit": "TFLOP/s",
        "frac": per_kernel[dom]["compute_frac"],
        "traffic": load_traffic(dom, T),
        "algorithmic_flops_per_launch": fpt[dom] * T,
        "algorithmic_bytes_per_launch": bpt[dom] * T,
        "hbm_achieved_GBps": per_kernel[dom]["hbm_GBps"],
        "hbm_frac": per_kernel[dom]["hbm_frac"],
        "avg_launch_ms": round(per_kernel_ms[dom], 4),
        "per_kernel": per_kernel,
    }

    out = {
        "metric": METRIC if args.workload == "train" else f"DPB fwd+bwd tokens/sec ({w.name})",
        "value": T / (ms_step * 1e-3),
        "value_median": T / (float(np.median(step_ms)) * 1e-3),
        # forward alone (encode + decode), from the per-launch means, and the
        # forward's HBM ceiling (read x, write the code and y once)
        "fwd_tokens_per_s": (T / ((per_kernel_ms["encode"] + per_kernel_ms["decode"]) * 1e-3)
                             if run["encode"] and run["decode"] else None),
        "fwd_hbm_ceiling_tokens_per_s": HBM_PEAK_GBS * 1e9 / bpt["forward"],
        # backward alone (decode-backward), and its HBM ceiling (read the code
        # indices and g, write grad_coef and grad_x once)
        "bwd_tokens_per_s": T / (per_kernel_ms["decode_bwd"] * 1e-3) if run["decode_bwd"] else None,
        "bwd_hbm_ceiling_tokens_per_s": HBM_PEAK_GBS * 1e9 / bpt["decode_bwd"],
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "ms_per_step_median": float(np.median(step_ms)),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if w.dtype == "bf16" else "f32",
        "data": "synthetic",
        "config": {
            "workload": (f"{w.name}: DPB d={w.d}, N=2^{w.n} ({w.levels} levels x {w.branching}-way), "
                         f"beam {w.beam}, k={w.k}, {T} tokens {w.dtype}; encode+decode+decode_bwd per step"
                         if w.hierarchy() is None else
                         f"{w.name}: DPB d={w.d}, levels n={plan.level_bits}, K={plan.active}, "
                         f"{w.branching} children per parent, {T} tokens {w.dtype}; encode+decode+decode_bwd per step"),
            "step_calls": "dpb_encode + dpb_decode + dpb_decode_bwd",
            "tokens_per_step": T, "d": w.d, "n_bits": w.n, "levels": w.levels, "branching": w.branching,
            "beam": w.beam, "k": w.k, "k_tot": k, "only": args.only,
        },
        "roofline": roofline,
    }
    if args.only is None and not args.no_extras:
        out["extras"] = time_extras(plan, w, sets, act, args.steps)
    if not args.no_cpu_baseline and args.only is None:
        out["cpu_baseline"] = cpu_baseline(args.workload)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
