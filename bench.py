"""Benchmark of the QuantEase hot path on one MI355X.

One step = one layer of the 4096 x 4096 attention-projection workload, 4-bit,
inputs resident in HBM:  Sigma = X X^T + 0.01 mean(diag) I over 128 x 2048
heavy-tailed tokens -> per-row grid -> 10 CD sweeps (objective after each)
-> exact objective.  value = column updates per second of the whole step
(p x 10 per step).  The outlier-aware path (3-bit, 1% outliers: lambda_max,
P_s(W), outlier grid, 10 CD + IHT iterations) is timed in the same run and
reported under "outlier"; the CPU oracle is timed on a bounded sample under
"cpu_baseline".

    python bench.py [--gpus 1] [--steps K] [--warmup W]
"""
import argparse
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "CD sweep time per layer (s) and column-updates/s at 4096×4096 4-bit"
HBM_PEAK_GBS = 8000.0
FP32_MFMA_PEAK_TFLOPS = 157.3
BF16_MFMA_PEAK_TFLOPS = 2500.0
SPLIT_PRODUCTS = 6             # bf16 products per fp32 product (exact three-way split)
TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "hbm_traffic_c2_4096x4096.md")
CALIB_COPY_BYTES = 256 << 20


# HIP sources each measured kernel is compiled from
KERNEL_SOURCES = {
    "gram_x3w_kernel": ["gram.hip", "nt_x3.h", "qe_internal.h"],
    "cd_step_kernel": ["cd.hip", "nt_x3.h", "qe_internal.h"],
}


def kernel_source_hash(kernel):
    """sha256 over the HIP sources `kernel` is compiled from (and the ABI header)."""
    import hashlib
    h = hashlib.sha256()
    files = [os.path.join(ROOT, "paper_2309_01885_amd", "csrc", f) for f in KERNEL_SOURCES[kernel]]
    files.append(os.path.join(ROOT, "include", "qe.h"))
    for path in files:
        h.update(os.path.basename(path).encode())
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic():
    """HBM bytes per launch from the committed FETCH_SIZE / WRITE_SIZE summary
    (copy-calibrated), keyed by kernel; a kernel is left out when its sources
    changed since the counters were taken."""
    try:
        with open(TRAFFIC_PROFILE) as f:
            text = f.read()
    except OSError:
        return {}
    m = re.search(r"```json\n(.*?)\n```", text, re.S)
    if not m:
        return {}
    data = json.loads(m.group(1))
    return {k: v["hbm_bytes_per_launch"] for k, v in data["kernels"].items()
            if k in KERNEL_SOURCES and v.get("source_sha256") == kernel_source_hash(k)}


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


CPU_GRAM_TOKENS = 32768      # oracle Gram sample (about 10 s on 16 host threads)
CPU_SWEEP_ROWS = 1024        # oracle sweep sample
CPU_ONE_THREAD_ROWS = 64     # single-thread sweep sample

# Child process for the single-thread figure: OpenMP's thread count is fixed
# when the oracle library loads, so it runs in a fresh interpreter.
_ONE_THREAD = """
import sys, numpy as np
sys.path.insert(0, sys.argv[1])
import oracle
d = sys.argv[2]
a = {k: np.load(d + "/" + k + ".npy") for k in ("W", "S", "scale", "zero")}
print(oracle.num_threads(), oracle.cd_sweep_timed(a["W"], a["S"], int(sys.argv[3]), a["scale"],
                                                  a["zero"]))
"""


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def one_thread_sweep(S, W, scale, zero, bits):
    """Seconds of one oracle sweep over W's rows with one OpenMP thread."""
    import subprocess
    import tempfile
    with tempfile.TemporaryDirectory(dir="/tmp") as d:
        for k, v in (("W", W), ("S", S), ("scale", scale), ("zero", zero)):
            np.save(os.path.join(d, k + ".npy"), np.ascontiguousarray(v))
        env = dict(os.environ, OMP_NUM_THREADS="1")
        out = subprocess.run([sys.executable, "-c", _ONE_THREAD, ROOT, d, str(bits)], env=env,
                             capture_output=True, text=True, timeout=600, check=True).stdout
    threads, secs = out.split()
    assert int(threads) == 1, out
    return float(secs)


def cpu_baseline(spec, X_head, W, scale, zero, sweeps):
    """The oracle as it stands on the host cores, on a bounded sample of the
    same step: Gram on the first n' tokens (scaled by n/n'), one CD sweep on r
    seeded rows (scaled by q/r rows and by the sweep count); plus the sweep on
    fewer rows with a single thread."""
    import oracle
    q, p, n = spec.q, spec.p, spec.n
    n_s = X_head.shape[1]
    t0 = time.perf_counter()
    S = oracle.damp(oracle.gram(X_head), spec.damp)
    t_gram = time.perf_counter() - t0
    rows = __import__("synth").row_sample(q, CPU_SWEEP_ROWS, spec.cfg)
    t_sweep = oracle.cd_sweep_timed(W[rows], S, spec.bits, scale[rows], zero[rows])
    t_step = t_gram * (n / n_s) + t_sweep * (q / len(rows)) * sweeps
    r1 = rows[:CPU_ONE_THREAD_ROWS]
    t_one = one_thread_sweep(S, W[r1], scale[r1], zero[r1], spec.bits)
    return {
        "value": p * sweeps / t_step,
        "unit": "column-updates/s",
        "cores": oracle.num_threads(),
        "cpu_model": cpu_model(),
        "kind": "oracle",
        "sample": (f"Gram over {n_s} of {n} tokens (x{n / n_s:.0f}), one Lemma-1 sweep over "
                   f"{len(rows)} of {q} rows (x{q / len(rows):.0f} rows, x{sweeps} sweeps); "
                   f"measured {t_gram:.2f} s + {t_sweep:.2f} s"),
        "step_s_extrapolated": t_step,
        "one_thread_sweep": {"rows": len(r1), "seconds": t_one,
                             "coordinate_updates_per_s": len(r1) * p / t_one,
                             "speedup_of_all_threads": (t_one / len(r1)) / (t_sweep / len(rows))},
    }


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-outlier", action="store_true", help="skip the outlier-aware timing")
    ap.add_argument("--no-peaks", action="store_true",
                    help="skip the matrix-core / copy peak checks (libqe_peak.so)")
    ap.add_argument("--calib-copy", action="store_true",
                    help="end with a plain 256 MiB device copy (HBM counter calibration)")
    ap.add_argument("--configs", action="store_true",
                    help="instead of the c2 step: Gram and CD timings of every workload "
                         "configuration at its full size (one JSON line)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on exactly one GPU: --gpus {args.gpus} is not supported "
              "(the CD sweep would shard by rows with no communication)",
              file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2309_01885_amd as P
    import synth

    if args.configs:
        print(json.dumps(configs_bench(P, torch, synth)), flush=True)
        return

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    spec = synth.CONFIGS["c2"]
    q, p, n, bits, sweeps = spec.q, spec.p, spec.n, spec.bits, spec.sweeps
    block = 128

    log(f"generating inputs: W {q}x{p}, X {p}x{n}")
    W_h = synth.weights(spec)
    X_h = synth.activations(spec)
    X = torch.from_numpy(X_h).to(dev)
    X_head = np.ascontiguousarray(X_h[:, :CPU_GRAM_TOKENS])
    del X_h
    W = torch.from_numpy(W_h).to(dev)
    Sigma = torch.empty((p, p), dtype=torch.float32, device=dev)
    Wh = torch.empty_like(W)
    codes = torch.empty((q, p), dtype=torch.uint8, device=dev)
    R = torch.empty_like(W)
    obj = torch.zeros(sweeps, dtype=torch.float64, device=dev)
    ws_gram = P.workspace(P.load().qe_gram_workspace_size(p, n), dev)
    ws_cd = P.workspace(P.cd_workspace_size(q, p, block), dev)
    ws_obj = P.workspace(P.load().qe_objective_workspace_size(q, p), dev)
    stream = torch.cuda.current_stream()

    ev = {k: [torch.cuda.Event(enable_timing=True) for _ in range(2)]
          for k in ("gram", "grid", "cd", "exact")}

    def step(timed=False):
        def mark(k, i):
            if timed:
                ev[k][i].record(stream)
        mark("gram", 0)
        P.gram(X, Sigma=Sigma, damp=spec.damp, ws=ws_gram, check=False)
        mark("gram", 1)
        mark("grid", 0)
        scale, zero = P.grid_minmax(W, bits)
        mark("grid", 1)
        mark("cd", 0)
        P.cd_sweep(W, Sigma, bits, scale, zero, Wh, codes, R, sweeps, block=block,
                   flags=P.QE_INIT_FROM_W, obj=obj, ws=ws_cd, check=False)
        mark("cd", 1)
        mark("exact", 0)
        out = P.objective(W, Wh, Sigma, ws=ws_obj, check=False)
        mark("exact", 1)
        return scale, zero, out

    log(f"warmup x{args.warmup}")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    for w in (ws_gram, ws_cd, ws_obj):
        st = P.sync_status(w)
        assert st == 0, f"device status {st}"

    log(f"timing x{args.steps}")
    phase = {k: [] for k in ev}
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        scale, zero, exact = step(timed=True)
        torch.cuda.synchronize()
        for k in ev:
            phase[k].append(ev[k][0].elapsed_time(ev[k][1]) * 1e-3)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    for w in (ws_gram, ws_cd, ws_obj):
        st = P.sync_status(w)
        assert st == 0, f"device status {st}"
    ms_per_step = wall / args.steps * 1e3
    value = p * sweeps / (wall / args.steps)
    f_sweeps = obj.cpu().numpy()
    exact = exact.cpu().numpy()

    # ---- dominant kernels, measured live on this stream
    # block-update step kernel: sweeps resumed from a valid R, no objective,
    # so the region holds only the step launches (+2 tiny setup kernels)
    super_w = max(256, block)                     # columns per step launch (super-block)
    nb = (p + super_w - 1) // super_w
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    P.cd_sweep(W, Sigma, bits, scale, zero, Wh, codes, R, sweeps, block=block,
               flags=P.QE_R_VALID | P.QE_CODES_VALID, obj=None, ws=ws_cd, check=False)
    e1.record(stream)
    torch.cuda.synchronize()
    t_steps = e0.elapsed_time(e1) * 1e-3
    # one sweep per call from W = What: events around each of sweeps 2..K
    # (with its objective, as in the step), median
    per_sweep = []
    for k in range(sweeps):
        a0, a1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a0.record(stream)
        P.cd_sweep(W, Sigma, bits, scale, zero, Wh, codes, R, 1, block=block,
                   flags=P.QE_INIT_FROM_W if k == 0 else P.QE_R_VALID | P.QE_CODES_VALID,
                   obj=obj[k:], ws=ws_cd, check=False)
        a1.record(stream)
        per_sweep.append((a0, a1))
    torch.cuda.synchronize()
    sweep_median_2_k = float(np.median([a.elapsed_time(b) * 1e-3 for a, b in per_sweep[1:]]))
    launches = sweeps * (nb + 1)
    cd_flops_per_launch = 2.0 * q * p * p / (nb + 1)      # 2qp^2 per sweep over nb + 1 launches
    cd_avg = t_steps / launches
    cd_tflops = cd_flops_per_launch / cd_avg / 1e12
    cd_mfma_flops = SPLIT_PRODUCTS * cd_flops_per_launch
    cd_bf16_tflops = cd_mfma_flops / cd_avg / 1e12
    gram_t = float(np.median(phase["gram"]))
    gram_flops = float(p) * (p + 1) * n                      # fp32 products (symmetric half)
    gram_tflops = gram_flops / gram_t / 1e12
    gram_mfma_flops = SPLIT_PRODUCTS * gram_flops            # the split algorithm's bf16 flops
    gram_bf16_tflops = gram_mfma_flops / gram_t / 1e12
    sweep_t = float(np.median(phase["cd"])) / sweeps
    traffic = measured_traffic()
    roof_cd = {"kernel": "cd_step_kernel<8>", "bound": "mfma", "achieved": cd_bf16_tflops,
               "peak": BF16_MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
               "frac": cd_bf16_tflops / BF16_MFMA_PEAK_TFLOPS,
               "traffic": traffic.get("cd_step_kernel"),
               "avg_launch_s": cd_avg, "flops_per_launch": cd_mfma_flops,
               "products": "bf16, 6 per fp32 product (exact 3-way split)",
               "fp32_equivalent_tflops": cd_tflops,
               "fp32_equivalent_frac": cd_tflops / FP32_MFMA_PEAK_TFLOPS}
    roof_gram = {"kernel": "gram_x3w_kernel", "bound": "mfma", "achieved": gram_bf16_tflops,
                 "peak": BF16_MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
                 "frac": gram_bf16_tflops / BF16_MFMA_PEAK_TFLOPS,
                 "traffic": traffic.get("gram_x3w_kernel"),
                 "call_s": gram_t, "flops_per_call": gram_mfma_flops,
                 "products": "bf16, 6 per fp32 product (exact 3-way split)",
                 "fp32_equivalent_tflops": gram_tflops,
                 "fp32_equivalent_frac": gram_tflops / FP32_MFMA_PEAK_TFLOPS}
    dominant = roof_gram if gram_t > sweeps * sweep_t else roof_cd

    result = {
        "metric": METRIC,
        "value": value,
        "unit": "column-updates/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32 (matrix products: bf16x3 split, f32 accumulate)",
        "data": "synthetic",
        "config": {"workload": spec.name, "q": q, "p": p, "n": n, "bits": bits,
                   "sweeps": sweeps, "block": block, "damp": spec.damp},
        "roofline": dominant,
        "rooflines": [roof_cd, roof_gram],
        "breakdown_s": {"gram": gram_t, "grid": float(np.median(phase["grid"])),
                        "cd_10_sweeps": float(np.median(phase["cd"])),
                        "exact_objective": float(np.median(phase["exact"]))},
        "sweep_time_s": sweep_t,
        "sweep_time_median_2_to_k_s": sweep_median_2_k,
        "cd_column_updates_per_s": p / sweep_t,
        "coordinate_updates_per_s": q * value,           # q * p * sweeps per step time
        "cd_coordinate_updates_per_s": q * p / sweep_t,
        "layer_time_s": ms_per_step / 1e3,
        "objective_per_sweep": [float(x) for x in f_sweeps],
        "rel_calibration_error": float(exact[0] / exact[1]),
    }

    if not args.no_outlier:
        log("outlier-aware path")
        result["outlier"] = outlier_bench(P, torch, synth, W, Sigma, dev, block)

    if not args.no_peaks:
        log("peak checks")
        from paper_2309_01885_amd import peaks
        mp = peaks.measure(torch)
        result["measured_peaks"] = mp
        for r in result["rooflines"]:
            r["frac_of_measured_bf16_peak"] = r["achieved"] / mp["mfma_bf16_tflops"]

    if not args.no_cpu:
        log("CPU oracle baseline")
        result["cpu_baseline"] = cpu_baseline(spec, X_head, W_h, scale.cpu().numpy(),
                                              zero.cpu().numpy(), sweeps)
    if args.calib_copy:
        a = torch.ones(CALIB_COPY_BYTES // 4, dtype=torch.float32, device=dev)
        b = torch.empty_like(a)
        b.copy_(a)
        torch.cuda.synchronize()
    print(json.dumps(result), flush=True)


def configs_bench(P, torch, synth):
    """Every workload configuration at its full size: the Gram over all
    n = 262144 device-drawn tokens (one call when X fits comfortably, else
    token chunks accumulated into Sigma), damping, the per-row grid and the
    configured number of CD sweeps from What = W.  Times from HIP events on
    the library's stream (c1 timed on its second pass, after the code objects
    are loaded)."""
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    out = {}
    # the first (c1) pass also loads the code objects; it is repeated and the
    # repeat is reported
    for key in ("c1", "c1", "c2", "c3up", "c3down", "c5"):
        spec = synth.CONFIGS[key]
        q, p, n = spec.q, spec.p, spec.n
        log(f"{key}: {q}x{p}, {n} tokens")
        chunk = n if p * n * 4 <= (16 << 30) else 32768
        Sigma = torch.empty((p, p), dtype=torch.float32, device=dev)
        gram_s = 0.0
        for c in range(n // chunk):
            Xc = synth.activation_chunk_device(spec, c, chunk, dev)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            P.gram(Xc, Sigma=Sigma, accumulate=c > 0, damp=spec.damp if c == n // chunk - 1 else 0.0)
            e1.record(stream)
            torch.cuda.synchronize()
            gram_s += e0.elapsed_time(e1) * 1e-3
            del Xc
        torch.cuda.empty_cache()
        W = torch.from_numpy(synth.weights(spec)).to(dev)
        scale, zero = P.grid_minmax(W, spec.bits)
        Wh = torch.empty_like(W)
        R = torch.empty_like(W)
        codes = torch.empty((q, p), dtype=torch.uint8, device=dev)
        ws = P.workspace(P.cd_workspace_size(q, p, 128), dev)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        P.cd_sweep(W, Sigma, spec.bits, scale, zero, Wh, codes, R, spec.sweeps, block=128,
                   flags=P.QE_INIT_FROM_W, ws=ws, check=False)
        e1.record(stream)
        torch.cuda.synchronize()
        cd_s = e0.elapsed_time(e1) * 1e-3
        out[spec.name] = {"q": q, "p": p, "n": n, "bits": spec.bits, "sweeps": spec.sweeps,
                          "gram_s": gram_s, "gram_chunks": n // chunk,
                          "gram_fp32_equivalent_tflops": float(p) * (p + 1) * n / gram_s / 1e12,
                          "sweep_s": cd_s / spec.sweeps,
                          "cd_fp32_equivalent_tflops": 2.0 * q * p * p * spec.sweeps / cd_s / 1e12,
                          "layer_s": gram_s + cd_s,
                          "column_updates_per_s": p * spec.sweeps / (gram_s + cd_s)}
        del Sigma, W, Wh, R, codes, ws
        torch.cuda.empty_cache()
    return {"configs": out}


def outlier_bench(P, torch, synth, W, Sigma, dev, block):
    spec = synth.CONFIGS["c4"]
    q, p, bits, iters, s = spec.q, spec.p, spec.bits, spec.sweeps, spec.s_budget
    stream = torch.cuda.current_stream()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(6)]
    ws_o = P.workspace(P.outlier_workspace_size(q, p, block, s), dev)
    Wh = torch.empty_like(W)
    codes = torch.empty((q, p), dtype=torch.uint8, device=dev)
    E = torch.empty_like(W)
    obj = torch.zeros(2 * iters, dtype=torch.float64, device=dev)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    lam = P.lambda_max(Sigma)
    t_lam = time.perf_counter() - t0

    def run(timed):
        if timed:
            ev[0].record(stream)
        H, sup, nnz = P.topk_abs(W, s, check=False)
        scale, zero = P.grid_minmax(W, bits, H)
        if timed:
            ev[1].record(stream)
        P.cd_outlier_sweep(W, Sigma, bits, scale, zero, Wh, codes, H, E, s, lam, sup, nnz, iters,
                           block=block, flags=P.QE_INIT_FROM_W, obj=obj, ws=ws_o, check=False)
        if timed:
            ev[2].record(stream)
        return nnz

    run(False)
    torch.cuda.synchronize()
    nnz = run(True)
    torch.cuda.synchronize()
    assert P.sync_status(ws_o) == 0
    g = obj.cpu().numpy()
    t_init = ev[0].elapsed_time(ev[1]) * 1e-3
    t_iters = ev[1].elapsed_time(ev[2]) * 1e-3
    res = {"workload": spec.name, "s": s, "lambda_max": lam, "lambda_time_s": t_lam,
           "init_time_s": t_init, "iter_time_s": t_iters / iters,
           "support_nnz": int(nnz.cpu().item()),
           "g_after_cd": [float(x) for x in g[0::2]], "g_after_iht": [float(x) for x in g[1::2]]}

    # structured outliers (Sec. 4.3): floor(s / q) whole columns
    ncols = s // q
    sup = torch.zeros(s, dtype=torch.int64, device=dev)

    def run_cols(timed):
        if timed:
            ev[3].record(stream)
        H, _, sup_c, n = P.topk_columns(W, ncols, check=False)
        sup[:q * ncols] = sup_c[:q * ncols]
        scale, zero = P.grid_minmax(W, bits, H)
        if timed:
            ev[4].record(stream)
        P.cd_outlier_sweep(W, Sigma, bits, scale, zero, Wh, codes, H, E, s, lam, sup, n, iters,
                           block=block, flags=P.QE_INIT_FROM_W | P.QE_OUTLIER_COLUMNS, obj=obj,
                           ws=ws_o, check=False)
        if timed:
            ev[5].record(stream)

    run_cols(False)
    torch.cuda.synchronize()
    run_cols(True)
    torch.cuda.synchronize()
    assert P.sync_status(ws_o) == 0
    g = obj.cpu().numpy()
    res["structured"] = {"columns": ncols, "init_time_s": ev[3].elapsed_time(ev[4]) * 1e-3,
                         "iter_time_s": ev[4].elapsed_time(ev[5]) * 1e-3 / iters,
                         "g_after_iht": [float(x) for x in g[1::2]]}
    return res


if __name__ == "__main__":
    main()
