"""Benchmark of the modality-aware W8A8 + low-rank linear on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload I] [--no-cpu]
                    [--method masquant|smoothquant|mas] [--weight-bits 8|4]

A step is one pass of the hot path over every projection of the workload:
per projection, smoothing + per-token int8 quantisation + the rank-r
down-projection (stage 1), then the int8 MFMA GEMM with the fused
dequantisation and Cross-Modal Compensation epilogue (stage 2), over one
batch of seeded synthetic mixed-modality tokens already resident in HBM.
Default workload: 4096 tokens (1024 text + 3072 vision), 3584 -> 18944,
rank 64, bf16 activations and outputs, int8 shared weight.

Prints one JSON line.  value = effective TOPS = sum of 2 T C_in C_out over
the step time (dense-equivalent int8 operations; quantisation and
compensation are not credited), from exactly K timed steps with nothing
recorded inside the timed region.  roofline: the stage-2 GEMM kernel, its
average launch duration from K rounds of the stage-2 launches back to back
(one event pair on the launch stream), against the 5.0 POPS dense int8
peak (algorithmic int8 ops) or, below the ridge point (the decode
workload), against 8 TB/s HBM (algorithmic bytes of the kernel), and
against the measured peaks (an int8 MFMA issue loop, a linear HBM read).
step_percentiles_ms: median, p10, p90 over max(K, 100) steps with an event
between consecutive steps.  sclk_under_load: the shader clock rocm-smi
reports while the headline step runs back to back for 1.5 s (after the
timed regions).  configs: the same summary for every workload
(at least 100 steps each).  cpu_baseline: the CPU oracle on the headline
workload.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

INT8_PEAK_TOPS = 5000.0      # MI355X dense int8 MFMA
HBM_PEAK_GBS = 8000.0        # MI355X HBM3E
KERNEL_SOURCES = ("paper_2603_04800_amd/csrc/masq_kernels.hip",)


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", type=int, default=1)
    ap.add_argument("--weight-bits", type=int, default=8, choices=(8, 4),
                    help="4: the W4A8 setting (shared weight as packed 4-bit codes)")
    ap.add_argument("--method", default="masquant", choices=("masquant", "smoothquant", "mas"),
                    help="comparators on the same kernels: smoothquant (one unified smoothing "
                         "factor, no compensation) or mas (MAS-only: a weight per modality, no "
                         "compensation)")
    ap.add_argument("--copies", type=int, default=2,
                    help="rotating input/output sets so no step reuses the last one's cache")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--no-peaks", action="store_true",
                    help="skip the measured-peak probes (int8 MFMA loop, HBM read and copy)")
    ap.add_argument("--only-headline", action="store_true",
                    help="time only --workload, not every workload's summary object")
    ap.add_argument("--no-sclk", action="store_true",
                    help="skip reading the shader clock (rocm-smi) while the headline "
                         "workload runs back to back")
    ap.add_argument("--summarize-profiles", metavar="DIR", default=None,
                    help="write the profiles/ summaries of the rocprofv3 runs under DIR "
                         "(trace/, fetch/, write/, copy_fetch/, copy_write/ and their .log; "
                         "mfma/ and lds/ for the counter summary)")
    ap.add_argument("--calibrate", action="store_true",
                    help="only time the calibration's exact steps (channel ranges, MAS factors, "
                         "Q(S_t W)) on the GPU against the host implementation, on the "
                         "workload's first projection")
    ap.add_argument("--cmc-study", action="store_true",
                    help="only print the compensation study of the workload's first projection: "
                         "effective rank of dW before and after whitening, and SQNR against "
                         "the rank ratio, whitened and not, beside the comparators "
                         "(weights at --weight-bits)")
    ap.add_argument("--mas-opt", action="store_true",
                    help="only run the MAS factor optimisation (2 epochs, batches of 256 rows) on "
                         "the workload's first projection: the objective of each modality "
                         "before and after, and the time per step")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="only run a plain device-to-device copy of MIB MiB (5 times): the "
                         "reference for scaling HBM traffic counters")
    return ap.parse_args()


def copy_probe(mib: int):
    """A plain copy of known size, profiled with the same counters as the GEMM
    so that FETCH_SIZE / WRITE_SIZE can be scaled to bytes."""
    import torch
    n = mib * (1 << 20)
    src = torch.empty(n, dtype=torch.uint8, device="cuda:0").fill_(1)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes_read": n, "copy_probe_bytes_written": n, "launches": 5}))


def calibration_timing(workload: int, reps: int = 20):
    """GPU (masq_channel_range, masq_smoothing_factors, masq_quantize_weight)
    against the host calibration (calibrate.smoothing_factors and
    quantize_shared_weight) on one projection's X and float weight."""
    import numpy as np
    import torch

    import synth
    from paper_2603_04800_amd import calibrate, ops
    cfg = synth.CONFIGS[workload]
    p = cfg.projections[0]
    li = synth.make_layer_inputs(cfg, 0, projections=[p.name])
    x, w = np.asarray(li.x[p.input_key], np.float32), np.asarray(li.w[p.name], np.float32)
    dev = torch.device("cuda:0")
    xt = torch.from_numpy(x).to(dev, torch.bfloat16 if cfg.act_dtype == "bf16" else torch.float32)
    mt = torch.from_numpy(np.asarray(li.modality, np.int32)).to(dev)
    wt = torch.from_numpy(np.ascontiguousarray(w)).to(dev)

    def gpu():
        r = ops.channel_range(xt, mt, cfg.n_mod)
        s, _ = ops.smoothing_factors(r, wt)
        return ops.quantize_weight(wt, s[0].contiguous())

    for _ in range(3):
        gpu()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        gpu()
    e1.record()
    torch.cuda.synchronize()
    gpu_ms = e0.elapsed_time(e1) / reps
    t0 = time.perf_counter()
    s32, _ = calibrate.smoothing_factors(x, li.modality, w, cfg.n_mod)
    calibrate.quantize_shared_weight(w, s32[0])
    host_ms = (time.perf_counter() - t0) * 1e3
    print(json.dumps({"metric": "calibration: channel ranges, MAS factors, Q(S_t W)",
                      "workload": cfg.name, "c_in": int(w.shape[0]), "c_out": int(w.shape[1]),
                      "tokens": int(x.shape[0]), "gpu_ms": round(gpu_ms, 4),
                      "host_ms": round(host_ms, 1), "host_threads": torch.get_num_threads()}),
          flush=True)
    if cfg.n_mod < 2 or cfg.rank == 0:
        return
    # the compensation factors of the first non-text modality (Sec. 4.3):
    # the GPU path (smoothed rows, dW and every large product on the GPU,
    # the small decompositions on the host) against the host calibration
    m = 1
    wq_h, ws_h = calibrate.quantize_shared_weight(w, s32[0])
    r = ops.channel_range(xt, mt, cfg.n_mod)
    s_t, _ = ops.smoothing_factors(r, wt)
    wq_t, ws_t = ops.quantize_weight(wt, s_t[0].contiguous())
    sm = s_t[m].contiguous()
    rows = torch.from_numpy(np.flatnonzero(li.modality == m).astype(np.int32)).to(dev)
    gpu_cmc_runs = []
    for _ in range(2):                     # the first run includes loading the kernels
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        z = ops.gather_smoothed(xt, rows, sm)
        dw = ops.weight_difference(wt, sm, wq_t, ws_t)
        l1, l2 = calibrate.cmc_factors_gpu(z, dw, cfg.rank, seed=m)
        gpu_cmc_runs.append(time.perf_counter() - t0)
    gpu_cmc_s = gpu_cmc_runs[-1]
    # the Gram product Z^T Z alone (the whitening's largest GEMM) and its
    # Cholesky factorisation, timed with events
    def gram():
        return ops.dgemm(z.T, z)

    gram()
    torch.cuda.synchronize()
    e0.record()
    for _ in range(5):
        gram()
    e1.record()
    torch.cuda.synchronize()
    gram_ms = e0.elapsed_time(e1) / 5
    n_r, k_c = z.shape
    gram_flops = 2.0 * k_c * k_c * n_r
    c = gram()
    chol_ms = []
    for _ in range(3):
        cc = c.clone()
        e0.record()
        ops.cholesky(cc, 1e-6)
        e1.record()
        torch.cuda.synchronize()
        chol_ms.append(e0.elapsed_time(e1))
    del z, dw, c, cc
    t0 = time.perf_counter()
    zh = x[li.modality == m].astype(np.float64) / s32[m].astype(np.float64)[None, :]
    dwh = calibrate._weight_difference(w, s32[m], wq_h, ws_h)
    h1, h2 = calibrate.cmc_factors(zh, dwh, cfg.rank, seed=m)
    host_cmc_s = time.perf_counter() - t0
    rel = float(np.linalg.norm(l1 @ l2 - h1 @ h2) / max(np.linalg.norm(h1 @ h2), 1e-300))
    print(json.dumps({"metric": "calibration: compensation factors of one modality",
                      "workload": cfg.name, "modality": m, "rows": int(n_r),
                      "c_in": int(w.shape[0]), "c_out": int(w.shape[1]), "rank": cfg.rank,
                      "gram": "Z^T Z", "gram_ms": round(gram_ms, 3),
                      "cholesky_ms": round(min(chol_ms), 3),
                      "gram_tflops": round(gram_flops / gram_ms / 1e9, 2),
                      "gram_frac_fp64_peak": round(gram_flops / gram_ms / 1e9 / 78.6, 4),
                      "gpu_s": round(gpu_cmc_s, 3), "gpu_s_first_run": round(gpu_cmc_runs[0], 3),
                      "host_s": round(host_cmc_s, 2),
                      "l1l2_relative_difference": rel}), flush=True)


def mas_opt_timing(workload: int, bits: int):
    """The MAS factor optimisation (Sec. 4.2) from the MAS initial factors:
    each modality's objective over all its rows before and after two epochs,
    and the wall time of the optimisation (every step's products, quantizers
    and reductions on the GPU; Adam on the host)."""
    import numpy as np
    import torch

    import synth
    from paper_2603_04800_amd import calibrate, mas_opt
    cfg = synth.CONFIGS[workload]
    p = cfg.projections[0]
    li = synth.make_layer_inputs(cfg, 0, projections=[p.name])
    x = np.asarray(li.x[p.input_key], np.float32)
    mod = np.asarray(li.modality, np.int32)
    w = np.asarray(li.w[p.name], np.float32)
    s0, _ = calibrate.smoothing_factors(x, mod, w, cfg.n_mod)
    dev = torch.device("cuda:0")
    wt = torch.from_numpy(np.ascontiguousarray(w)).to(dev)

    def objective(s):
        out = {}
        for m in range(cfg.n_mod):
            rows = x[mod == m]
            if rows.shape[0]:
                st = mas_opt._Step(torch.from_numpy(np.ascontiguousarray(rows)).to(dev),
                                   wt.double(), wt, bits)
                out[str(m)] = st(s[m])[0]
                del st
        return out

    before = objective(s0)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    s1, hist = mas_opt.optimise(x, mod, w, s0, epochs=2, batch=256, bits=bits)
    torch.cuda.synchronize()
    secs = time.perf_counter() - t0
    after = objective(s1)
    steps = sum(len(h) for h in hist)
    print(json.dumps({"metric": "MAS factor optimisation (2 epochs, batches of 256 rows)",
                      "workload": cfg.name, "weight_bits": bits, "c_in": int(w.shape[0]),
                      "c_out": int(w.shape[1]), "steps": steps, "seconds": round(secs, 2),
                      "ms_per_step": round(secs * 1e3 / max(steps, 1), 2),
                      "mae_before": before, "mae_after": after,
                      "factor_change_max_ratio": float(np.max(np.maximum(s1 / s0, s0 / s1)))}),
          flush=True)


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def _weight_bytes(L) -> int:
    """Bytes of the weight(s) a step reads: the shared weight at its bit width,
    or, for the MAS-only comparator, the weight of every modality present."""
    wq = L["wq"]
    if wq.ndim == 3:
        return len(set(L["modality"].tolist())) * wq.shape[1] * wq.shape[2]
    return wq.shape[0] * wq.shape[1] * int(L.get("weight_bits", 8)) // 8


def algorithmic_bytes(L) -> int:
    """Bytes the layer itself must move: X, Y, Wq, scales, smoothing vectors,
    factors of the non-text modalities present, modality ids."""
    T, K = L["x"].shape
    N = L["wq"].shape[-2]
    act = 2 if L["act_dtype"] == "bf16" else 4
    lr = 2 if L["lr_dtype"] == "bf16" else 4
    present = len(set(L["modality"].tolist()) - {0})
    wbytes = _weight_bytes(L)
    return (T * K * act + T * N * act + wbytes + N * 4 + L["n_mod"] * K * 4
            + present * L["rank"] * (K + N) * lr + T * 4)


GEMM_KERNEL = "k_gemm"          # name stem of the stage-2 GEMM kernels
COPY_KERNEL = "copyBuffer"      # the runtime's device-to-device copy (the probe)

# The rocprofv3 runs whose output --summarize-profiles reads; <repo> is the
# repository root, <out> the directory given to --summarize-profiles.
PROFILE_COMMANDS = {
    "trace": "cd /tmp && TMPDIR=/tmp rocprofv3 --kernel-trace --stats --output-format csv "
             "-d <out>/trace -o run -- python3 <repo>/bench.py --workload {w} --steps 30 "
             "--warmup 5 --no-cpu --no-peaks --only-headline",
    "fetch": "cd /tmp && TMPDIR=/tmp rocprofv3 --pmc FETCH_SIZE --output-format csv "
             "-d <out>/fetch -o run -- python3 <repo>/bench.py --workload {w} --steps 3 "
             "--warmup 1 --no-cpu --no-peaks --only-headline",
    "write": "cd /tmp && TMPDIR=/tmp rocprofv3 --pmc WRITE_SIZE --output-format csv "
             "-d <out>/write -o run -- python3 <repo>/bench.py --workload {w} --steps 3 "
             "--warmup 1 --no-cpu --no-peaks --only-headline",
    "mfma": "cd /tmp && TMPDIR=/tmp rocprofv3 --pmc MfmaUtil SQ_INSTS_VALU_MFMA_MOPS_I8 "
            "GRBM_GUI_ACTIVE --kernel-trace --output-format csv -d <out>/mfma -o run -- python3 "
            "<repo>/bench.py --workload {w} --steps 3 --warmup 1 --no-cpu --no-peaks "
            "--only-headline",
    "lds": "cd /tmp && TMPDIR=/tmp rocprofv3 --pmc SQ_LDS_BANK_CONFLICT SQ_LDS_IDX_ACTIVE "
           "SQ_INSTS_LDS SQ_WAVES --kernel-trace --output-format csv -d <out>/lds -o run -- "
           "python3 <repo>/bench.py --workload {w} --steps 3 --warmup 1 --no-cpu --no-peaks "
           "--only-headline",
    "copy_fetch": "cd /tmp && TMPDIR=/tmp rocprofv3 --pmc FETCH_SIZE --output-format csv "
                  "-d <out>/copy_fetch -o run -- python3 <repo>/bench.py --copy-probe 512",
    "copy_write": "cd /tmp && TMPDIR=/tmp rocprofv3 --pmc WRITE_SIZE --output-format csv "
                  "-d <out>/copy_write -o run -- python3 <repo>/bench.py --copy-probe 512",
}


def _profile_path(kind: str, workload_name: str) -> str:
    return os.path.join(ROOT, "profiles", f"k_gemm_{kind}_{workload_name}.txt")


def traffic_from_profiles(workload_name: str, src_hash: str):
    """HBM bytes per GEMM launch from the committed rocprofv3 counter summary,
    only if it was taken on the current kernel source."""
    path = _profile_path("traffic", workload_name)
    if not os.path.exists(path):
        return None
    kv = {}
    with open(path) as f:
        for line in f:
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                kv[k.strip()] = v.strip()
    if kv.get("kernel_source_sha256_16") != src_hash:
        return None
    return int(kv["bytes_per_launch"])


def _csv_rows(directory: str, suffix: str):
    import csv
    import glob
    paths = sorted(glob.glob(os.path.join(directory, "**", f"*{suffix}"), recursive=True))
    if not paths:
        raise FileNotFoundError(f"no *{suffix} under {directory}")
    with open(paths[0], newline="") as f:
        return list(csv.DictReader(f))


def _per_dispatch(directory: str, counter: str, name_part: str):
    """{dispatch id: summed counter value} of the dispatches whose kernel name
    contains name_part, from a rocprofv3 --pmc csv run."""
    vals = {}
    for r in _csv_rows(directory, "counter_collection.csv"):
        if r["Counter_Name"] != counter or name_part not in r["Kernel_Name"]:
            continue
        d = r["Dispatch_Id"]
        vals[d] = vals.get(d, 0.0) + float(r["Counter_Value"])
    if not vals:
        raise ValueError(f"no {counter} for kernels matching {name_part!r} in {directory}")
    return vals


def _per_dispatch_all(directory: str, name_part: str):
    """{dispatch id: {counter: value summed over instances, "us": duration}}
    of the dispatches whose kernel name contains name_part."""
    out = {}
    for r in _csv_rows(directory, "counter_collection.csv"):
        if name_part not in r["Kernel_Name"]:
            continue
        d = out.setdefault(r["Dispatch_Id"], {
            "us": (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3})
        d[r["Counter_Name"]] = d.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    return out


def summarize_counters(out: str, workload: int, cfg, src_hash: str, cmds: dict):
    """profiles/k_gemm_counters_<workload>.txt from the mfma/ and lds/ runs:
    MFMA utilisation of the GEMM and of stage 1 (rocprofv3's MfmaUtil: MFMA
    busy cycles over the kernel's GPU-active cycles times the SIMD count),
    the int8 MFMA operations counted (SQ_INSTS_VALU_MFMA_MOPS_I8 x 512), the
    clock implied by GRBM_GUI_ACTIVE (summed over the 8 XCDs) and the
    kernel time, and the LDS bank-conflict share."""
    for kind in ("mfma", "lds"):
        h = _bench_hash_in_log(os.path.join(out, f"{kind}.log"))
        if h != src_hash:
            raise SystemExit(f"{kind} run was taken on kernel source {h}, tree is {src_hash}")
    lines = [f"# rocprofv3 counters of the GEMM (k_gemm*) and stage-1 kernels (k_stage1*, or "
             f"k_down_lds and k_smooth_quant*), workload {cfg.name}",
             f"# command (mfma): {cmds['mfma']}", f"# command (lds): {cmds['lds']}",
             "# per-dispatch means; gemm_clock_ghz = GRBM_GUI_ACTIVE / 8 XCDs / kernel time; "
             "lds_conflict_share = SQ_LDS_BANK_CONFLICT / SQ_LDS_IDX_ACTIVE",
             f"kernel_source_sha256_16: {src_hash}"]
    # stage 1 is k_stage1_* or, in its split form, k_down_lds then the row quantiser
    for label, part in (("gemm", GEMM_KERNEL), ("stage1", "stage1"), ("down_lds", "k_down_lds"),
                        ("quant", "k_smooth_quant")):
        m = list(_per_dispatch_all(os.path.join(out, "mfma"), part).values())
        l = list(_per_dispatch_all(os.path.join(out, "lds"), part).values())
        if not m or not l:
            continue
        mean = lambda rows, k: sum(r.get(k, 0.0) for r in rows) / len(rows)
        us = mean(m, "us")
        if label == "gemm":      # GRBM_GUI_ACTIVE also counts time around a dispatch:
            lines.append(f"gemm_clock_ghz: "   # only meaningful for the long GEMM
                         f"{mean(m, 'GRBM_GUI_ACTIVE') / 8 / (mean(m, 'us') * 1e3):.3f}")
        lines += [f"{label}_dispatches: {len(m)}",
                  f"{label}_kernel_us: {us:.2f}",
                  f"{label}_mfma_util_percent: {mean(m, 'MfmaUtil'):.2f}",
                  f"{label}_int8_mfma_ops: {mean(m, 'SQ_INSTS_VALU_MFMA_MOPS_I8') * 512:.6e}",
                  f"{label}_lds_instructions: {mean(l, 'SQ_INSTS_LDS'):.0f}",
                  f"{label}_lds_conflict_share: "
                  f"{mean(l, 'SQ_LDS_BANK_CONFLICT') / max(mean(l, 'SQ_LDS_IDX_ACTIVE'), 1):.4f}",
                  f"{label}_waves: {mean(l, 'SQ_WAVES'):.0f}"]
    path = os.path.join(ROOT, "profiles", f"k_gemm_counters_{cfg.name}.txt")
    with open(path, "w") as f:
        f.write("\n".join(lines) + "\n")
    print(open(path).read())


def _bench_hash_in_log(path: str):
    with open(path) as f:
        for line in f:
            if line.startswith('{"metric"'):
                return json.loads(line).get("kernel_source_sha256_16")
    return None


def summarize_profiles(out: str, workload: int):
    """Write the committed text summaries of the rocprofv3 runs listed in
    PROFILE_COMMANDS (run beforehand, output under `out`)."""
    from synth.workloads import CONFIGS
    cfg = CONFIGS[workload]
    src_hash = kernel_source_hash()
    cmds = {k: v.format(w=workload) for k, v in PROFILE_COMMANDS.items()}
    os.makedirs(os.path.join(ROOT, "profiles"), exist_ok=True)
    if os.path.isdir(os.path.join(out, "mfma")) and os.path.isdir(os.path.join(out, "lds")):
        summarize_counters(out, workload, cfg, src_hash, cmds)
    if not os.path.isdir(os.path.join(out, "trace")):
        return
    for kind in ("trace", "fetch", "write"):
        h = _bench_hash_in_log(os.path.join(out, f"{kind}.log"))
        if h != src_hash:
            raise SystemExit(f"{kind} run was taken on kernel source {h}, tree is {src_hash}")

    stats = _csv_rows(os.path.join(out, "trace"), "kernel_stats.csv")
    with open(_profile_path("trace", cfg.name), "w") as f:
        f.write(f"# rocprofv3 kernel trace statistics, workload {cfg.name}\n")
        f.write(f"# command: {cmds['trace']}\n")
        f.write(f"# kernel_source_sha256_16: {src_hash}\n")
        f.write("# calls  avg_us  min_us  max_us  share%  kernel\n")
        for r in stats:
            name = r["Name"]
            short = name.replace("(anonymous namespace)::", "").replace("void ", "")
            short = short.split("(")[0][:110]
            f.write(f"{int(r['Calls']):6d} {float(r['AverageNs']) / 1e3:8.2f} "
                    f"{float(r['MinNs']) / 1e3:8.2f} {float(r['MaxNs']) / 1e3:8.2f} "
                    f"{float(r['Percentage']):6.2f}  {short}\n")

    copy_bytes = 512 << 20
    cf = max(_per_dispatch(os.path.join(out, "copy_fetch"), "FETCH_SIZE", COPY_KERNEL).values())
    cw = max(_per_dispatch(os.path.join(out, "copy_write"), "WRITE_SIZE", COPY_KERNEL).values())
    fetch_scale = copy_bytes / (cf * 1024.0)
    write_scale = copy_bytes / (cw * 1024.0)
    gf = _per_dispatch(os.path.join(out, "fetch"), "FETCH_SIZE", GEMM_KERNEL)
    gw = _per_dispatch(os.path.join(out, "write"), "WRITE_SIZE", GEMM_KERNEL)
    fkib = sum(gf.values()) / len(gf)
    wkib = sum(gw.values()) / len(gw)
    nbytes = int(round(fkib * 1024 * fetch_scale + wkib * 1024 * write_scale))
    with open(_profile_path("traffic", cfg.name), "w") as f:
        f.write(f"# HBM traffic of the stage-2 GEMM kernel (k_gemm*), workload {cfg.name}\n")
        for k in ("fetch", "write", "copy_fetch", "copy_write"):
            f.write(f"# command ({k}): {cmds[k]}\n")
        f.write("# bytes = FETCH_SIZE KiB * 1024 * fetch_scale + WRITE_SIZE KiB * 1024 * "
                "write_scale; the scales make a 512 MiB device copy read and write 512 MiB\n")
        f.write(f"kernel_source_sha256_16: {src_hash}\n")
        f.write(f"gemm_dispatches_fetch: {len(gf)}\n")
        f.write(f"gemm_dispatches_write: {len(gw)}\n")
        f.write(f"fetch_size_kib_per_launch: {fkib:.1f}\n")
        f.write(f"write_size_kib_per_launch: {wkib:.1f}\n")
        f.write(f"copy_probe_fetch_size_kib: {cf:.1f}\n")
        f.write(f"copy_probe_write_size_kib: {cw:.1f}\n")
        f.write(f"fetch_scale: {fetch_scale:.4f}\n")
        f.write(f"write_scale: {write_scale:.4f}\n")
        f.write(f"bytes_per_launch: {nbytes}\n")
    print(open(_profile_path("trace", cfg.name)).read())
    print(open(_profile_path("traffic", cfg.name)).read())


def cpu_baseline(layers, min_seconds=10.0, max_runs=64):
    """The CPU oracle (oracle.inference.linear, fp64) on the whole batch of the
    same workload (every projection), repeated until at least `min_seconds`
    of CPU work; the value is the mean over the runs."""
    import numpy as np
    from threadpoolctl import threadpool_info

    from oracle import inference as oinf
    runs, dt = 0, 0.0
    while runs < max_runs and (runs == 0 or dt < min_seconds):
        t0 = time.perf_counter()
        for L in layers:
            oinf.linear(L["x"], L["modality"], L["inv_smooth"], L["wq"], L["w_scale"],
                        L["l_down"], L["r_up"])
        dt += time.perf_counter() - t0
        runs += 1
    ops = sum(2.0 * L["x"].shape[0] * L["x"].shape[1] * L["wq"].shape[-2] for L in layers)
    T = layers[0]["x"].shape[0]
    n_text = int((np.asarray(layers[0]["modality"]) == 0).sum())
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    return {"value": round(ops * runs / dt / 1e12, 4), "unit": "TOPS",
            "cores": int(threads), "kind": "oracle",
            "host_cpus": os.cpu_count(), "affinity_cpus": len(os.sched_getaffinity(0)),
            "threads_note": "cores = the BLAS threads of the fp64 integer GEMM (the elementwise "
                            "steps run on one thread)",
            "sample": f"the whole {T}-token batch ({n_text} text), {len(layers)} projection(s), "
                      f"through oracle.inference.linear (fp64), {runs} runs, {dt:.1f} s total"}


def gemm_kernel_label(layers) -> str:
    """Name of the stage-2 kernel(s) the layers dispatch to: batches of at
    most 16 tokens with K % 64 == 0 take the k-sliced decode kernel (K up to
    8 slices of 40 64-byte steps; longer rows the single-pass one), other
    K % 64 == 0 shapes the LDS-DMA tile kernel, the rest the general-K one."""
    names = []
    for L in layers:
        T, K = L["x"].shape
        n = (("k_gemm_decode" if K <= 8 * 40 * 64 else "k_gemm_small") if T <= 16 and K % 64 == 0
             else "k_gemm_dma" if K % 64 == 0 else "k_gemm")
        if n not in names:
            names.append(n)
    return " + ".join(names) + " (stage 2: int8 GEMM + dequant + compensation)"


def gemm_bytes(L) -> int:
    """Bytes the stage-2 kernel must move at least: q codes, Wq, scales, the
    rank-r rows u, the factors of the non-text modalities present, modality
    ids and the output."""
    T, K = L["x"].shape
    N = L["wq"].shape[-2]
    out = 2 if L["act_dtype"] == "bf16" else 4
    lr = 2 if L["lr_dtype"] == "bf16" else 4
    present = len(set(L["modality"].tolist()) - {0})
    wbytes = _weight_bytes(L)
    return (T * K + wbytes + T * N * out + N * 4 + T * 4 + T * 4
            + (T * L["rank"] * 4 + present * L["rank"] * N * lr if present else 0))


def _probe_lib():
    """The peak probes (libmasq_probe.so, include/masq_probe.h)."""
    import ctypes
    path = os.path.join(ROOT, "paper_2603_04800_amd", "_lib", "libmasq_probe.so")
    if not os.path.exists(path):
        raise ImportError(f"{path} is missing: build first (python -m paper_2603_04800_amd.build)")
    lib = ctypes.CDLL(path)
    p, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    lib.masq_probe_mfma_i8.argtypes = [i32, i32, p, p]
    lib.masq_probe_mfma_i8.restype = ctypes.c_int
    lib.masq_probe_mfma_i8_ops.argtypes = [i32, i32]
    lib.masq_probe_mfma_i8_ops.restype = i64
    lib.masq_probe_read.argtypes = [p, i64, i32, p, p]
    lib.masq_probe_read.restype = ctypes.c_int
    lib.masq_probe_lds_dma.argtypes = [p, i64, i32, i32, p, p]
    lib.masq_probe_lds_dma.restype = ctypes.c_int
    lib.masq_probe_lds_dma_bytes.argtypes = [i32, i32]
    lib.masq_probe_lds_dma_bytes.restype = i64
    return lib


def measured_peaks(dev, reps: int = 7):
    """What this GPU sustains, median over `reps` timed launches each: int8
    MFMA operations per second of a pure-issue loop (no memory traffic, at the
    clock the chip holds under that load), the HBM read rate of a linear
    16-byte read of 4 GiB, and the rate of a 2 GiB device copy (read + write)."""
    import ctypes

    import torch
    lib = _probe_lib()
    st = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)

    def timed(fn):
        fn()
        fn()
        ts = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            e1.synchronize()
            ts.append(e0.elapsed_time(e1) * 1e-3)
        return sorted(ts)[len(ts) // 2]

    blocks, iters = 2048, 2500
    out = torch.empty(blocks * 256, dtype=torch.int32, device=dev)

    def mfma():
        if lib.masq_probe_mfma_i8(blocks, iters, ctypes.c_void_p(out.data_ptr()), st) != 0:
            raise RuntimeError("masq_probe_mfma_i8 failed")
    t_mfma = timed(mfma)
    ops = lib.masq_probe_mfma_i8_ops(blocks, iters)

    nbytes = 4 << 30
    buf = torch.zeros(nbytes, dtype=torch.uint8, device=dev)
    rblocks = 4096
    rout = torch.empty(rblocks * 256, dtype=torch.int32, device=dev)

    def read():
        if lib.masq_probe_read(ctypes.c_void_p(buf.data_ptr()), nbytes, rblocks,
                               ctypes.c_void_p(rout.data_ptr()), st) != 0:
            raise RuntimeError("masq_probe_read failed")
    t_read = timed(read)
    half = nbytes // 2
    src, dst = buf[:half], buf[half:]
    t_copy = timed(lambda: dst.copy_(src))
    # L2 -> LDS by LDS DMA, rows spread over 3 MB (L2-resident on every XCD)
    dblocks, diters = 256, 4000
    dout = torch.empty(dblocks, dtype=torch.int32, device=dev)

    def dma():
        if lib.masq_probe_lds_dma(ctypes.c_void_p(buf.data_ptr()), 3 << 20, dblocks, diters,
                                  ctypes.c_void_p(dout.data_ptr()), st) != 0:
            raise RuntimeError("masq_probe_lds_dma failed")
    t_dma = timed(dma)
    dma_bytes = lib.masq_probe_lds_dma_bytes(dblocks, diters)
    del buf, out, rout, dout
    torch.cuda.empty_cache()
    return {"int8_mfma_tops": round(ops / t_mfma / 1e12, 1),
            "hbm_read_gbps": round(nbytes / t_read / 1e9, 1),
            "hbm_copy_gbps": round(2 * half / t_copy / 1e9, 1),
            "l2_to_lds_dma_gbps": round(dma_bytes / t_dma / 1e9, 1),
            "method": "median of 7 launches: v_mfma_i32_32x32x32_i8 issue loop (8 chains a "
                      "wave, 2048 x 4 waves, no memory traffic); linear 16-byte read of 4 GiB; "
                      "2 GiB device copy; LDS DMA of 16-row x 64-byte pieces from an "
                      "L2-resident 3 MB region (256 x 8 waves)"}


def _pct(vals, q):
    v = sorted(vals)
    if not v:
        return None
    k = (len(v) - 1) * q
    lo, hi = int(k), min(int(k) + 1, len(v) - 1)
    return v[lo] + (v[hi] - v[lo]) * (k - lo)


def read_sclk(timeout_s: float = 20.0) -> dict:
    """The shader clock rocm-smi reports for every card it sees (MHz), run as
    a child process."""
    import re
    import subprocess
    try:
        out = subprocess.run(["rocm-smi", "--showclocks", "--json"], capture_output=True,
                             text=True, timeout=timeout_s)
        data = json.loads(out.stdout)
    except Exception as e:              # the clock is a report, never the measurement
        return {"error": repr(e)}
    cards = {}
    for card, fields in data.items():
        if not isinstance(fields, dict):
            continue
        for k, v in fields.items():
            m = re.search(r"(\d+)\s*mhz", str(v), re.I)
            if "sclk" in k.lower() and "speed" in k.lower() and m:
                cards[card] = int(m.group(1))
    return {"sclk_mhz": cards} if cards else {"error": "no sclk field", "raw": out.stdout[:300]}


def measure_workload(cfg_index, method, bits, steps, warmup, copies_min, dev, pct_steps=100,
                     keep_layers=False, min_warm_s=0.1, sclk_s=0.0):
    """Time one workload.  Three regions, each bracketed by events on the
    launch stream after a synchronisation, on rotating copies of every
    input, weight, output and workspace:
      A  `steps` whole steps with nothing recorded inside (the step time);
      B  `steps` rounds of the stage-2 launches alone, back to back (the
         GEMM kernels' average launch duration, inter-launch gaps included);
      C  max(steps, pct_steps) steps with an event between consecutive steps
         (per-step median, p10 and p90; each boundary record costs GPU time).
    """
    import torch

    from paper_2603_04800_amd import workload
    from synth.workloads import CONFIGS
    t0 = time.time()
    cfg = CONFIGS[cfg_index]
    layers = [workload.layer(cfg, p.name, method=method, weight_bits=bits)
              for p in cfg.projections]
    log(f"[bench] workload {cfg.name}: {len(layers)} projection(s), inputs + calibration "
        f"{time.time() - t0:.1f}s")
    out_dtype = torch.bfloat16 if cfg.act_dtype == "bf16" else torch.float32
    T = cfg.T
    # enough rotating copies that one step's data is not still in the 256 MB
    # Infinity Cache from the previous step
    per_copy = sum(algorithmic_bytes(L) for L in layers)
    copies = max(copies_min, min(16, -(-512 * 2**20 // per_copy)))
    sets = []
    for _ in range(copies):
        xs = {}
        projs = []
        for p, L in zip(cfg.projections, layers):
            x, mod, lin = workload.to_device(L, dev)
            if p.input_key in xs:                  # projections that read the same activations
                x = xs[p.input_key]
            xs[p.input_key] = x
            y = torch.empty((T, lin.c_out), dtype=out_dtype, device=dev)
            # arguments marshalled once, so the host keeps ahead of the GPU
            projs.append(lin.bind(x, mod, y, lin.workspace(T, dev)))
        sets.append(projs)
    torch.cuda.synchronize()

    def step(i):
        for b in sets[i % len(sets)]:
            b.stage1()
            b.stage2()

    def gemms(i):
        for b in sets[i % len(sets)]:
            b.stage2()

    # W warm-up steps, then more until the GPU has been busy for
    # min_warm_s: its clocks ramp up over several milliseconds after idle
    t_w = time.perf_counter()
    done = 0
    for i in range(warmup):
        step(i)
    done = warmup
    torch.cuda.synchronize()
    while time.perf_counter() - t_w < min_warm_s:
        for _ in range(8):
            step(done)
            done += 1
        torch.cuda.synchronize()
    warmup = done

    def region(fn, n, first):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for i in range(n):
            fn(first + i)
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1)

    step_ms = region(step, steps, warmup) / steps
    gemm_ms = region(gemms, steps, warmup + steps) / steps
    n_pct = max(steps, pct_steps)
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(n_pct + 1)]
    torch.cuda.synchronize()
    evs[0].record()
    for i in range(n_pct):
        step(warmup + 2 * steps + i)
        evs[i + 1].record()
    torch.cuda.synchronize()
    per = [evs[i].elapsed_time(evs[i + 1]) for i in range(n_pct)]
    sclk = None
    if sclk_s > 0:
        # the clock under this load: steps back to back for sclk_s seconds
        # while a thread asks rocm-smi once, half a second in
        import threading
        box = {}

        def probe():
            time.sleep(0.5)
            box.update(read_sclk())

        th = threading.Thread(target=probe)
        th.start()
        t_s, i = time.perf_counter(), 0
        while th.is_alive() or time.perf_counter() - t_s < sclk_s:
            for _ in range(8):
                step(i)
                i += 1
            torch.cuda.synchronize()
        th.join()
        sclk = dict(box, seconds=round(time.perf_counter() - t_s, 2), steps=i,
                    source="rocm-smi --showclocks, while the steps ran back to back")
    log(f"[bench] {cfg.name}: {step_ms:.4f} ms/step over {steps} steps, stage 2 "
        f"{gemm_ms:.4f} ms; per-step median {_pct(per, 0.5):.4f} ms over {n_pct}")
    res = {"cfg": cfg, "layers": layers if keep_layers else None, "copies": copies,
           "warmup_steps_run": warmup,
           "step_ms": step_ms, "gemm_ms": gemm_ms, "n_pct": n_pct,
           "median_ms": _pct(per, 0.5), "p10_ms": _pct(per, 0.1), "p90_ms": _pct(per, 0.9),
           "sclk": sclk,
           "ops": sum(2.0 * T * L["x"].shape[1] * L["wq"].shape[-2] for L in layers),
           "bytes": sum(algorithmic_bytes(L) for L in layers),
           "gemm_bytes": sum(gemm_bytes(L) for L in layers),
           "kernel": (gemm_kernel_label(layers) if method != "mas" else
                      "masq_mas_only_linear (rows grouped by modality on the device, "
                      "quantisation, grouped int8 GEMM with a weight per modality)")}
    del sets
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return res


def roofline_of(r, peaks):
    """The stage-2 kernels against their bound: int8 MFMA (algorithmic int8
    ops) or, below the ridge point, HBM (algorithmic bytes of the kernel)."""
    hbm_bound = r["ops"] / r["gemm_bytes"] < INT8_PEAK_TOPS / HBM_PEAK_GBS * 1e3
    if hbm_bound:
        achieved = r["gemm_bytes"] / (r["gemm_ms"] * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4)}
        if peaks:
            roof["measured_peak"] = peaks["hbm_read_gbps"]
            roof["frac_measured_peak"] = round(achieved / peaks["hbm_read_gbps"], 4)
    else:
        achieved = r["ops"] / (r["gemm_ms"] * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 2), "peak": INT8_PEAK_TOPS,
                "unit": "TOPS", "frac": round(achieved / INT8_PEAK_TOPS, 4)}
        if peaks:
            roof["measured_peak"] = peaks["int8_mfma_tops"]
            roof["frac_measured_peak"] = round(achieved / peaks["int8_mfma_tops"], 4)
    return roof


def config_summary(r, peaks):
    """The per-workload object of the bench line."""
    tops = r["ops"] / (r["step_ms"] * 1e-3) / 1e12
    gbps = r["bytes"] / (r["step_ms"] * 1e-3) / 1e9
    roof = roofline_of(r, peaks)
    out = {"workload": r["cfg"].name, "ms_per_step": round(r["step_ms"], 5),
           "median_ms": round(r["median_ms"], 5), "p10_ms": round(r["p10_ms"], 5),
           "p90_ms": round(r["p90_ms"], 5), "percentile_steps": r["n_pct"],
           "tops": round(tops, 2), "gbps": round(gbps, 1),
           "frac_int8_spec": round(tops / INT8_PEAK_TOPS, 4),
           "frac_hbm_spec": round(gbps / HBM_PEAK_GBS, 4),
           "gemm_ms": round(r["gemm_ms"], 5), "gemm_bound": roof["bound"],
           "gemm_achieved": roof["achieved"], "gemm_frac_spec": roof["frac"]}
    if peaks:
        out["frac_int8_measured"] = round(tops / peaks["int8_mfma_tops"], 4)
        out["frac_hbm_measured"] = round(gbps / peaks["hbm_read_gbps"], 4)
        out["gemm_frac_measured"] = roof["frac_measured_peak"]
    return out


def main():
    args = parse()
    if args.copy_probe:
        copy_probe(args.copy_probe)
        return
    if args.calibrate:
        calibration_timing(args.workload)
        return
    if args.mas_opt:
        mas_opt_timing(args.workload, args.weight_bits)
        return
    if args.cmc_study:
        from paper_2603_04800_amd import study
        for row in study.cmc_study(args.workload, weight_bits=args.weight_bits):
            print(json.dumps(row), flush=True)
        return
    if args.summarize_profiles:
        summarize_profiles(args.summarize_profiles, args.workload)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import torch

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    peaks = None
    if not args.no_peaks:
        peaks = measured_peaks(dev)
        log(f"[bench] measured peaks: {peaks['int8_mfma_tops']} int8 TOPS, "
            f"{peaks['hbm_read_gbps']} GB/s read, {peaks['hbm_copy_gbps']} GB/s copy")

    # every workload's summary first (this also brings the chip to its
    # sustained state), then the headline workload: W warm-up steps and
    # exactly --steps timed steps (region A)
    from synth.workloads import CONFIGS
    per = {}
    if not args.only_headline:
        for ci in range(len(CONFIGS)):
            r = measure_workload(ci, args.method, args.weight_bits, max(args.steps, 100),
                                 args.warmup, args.copies, dev)
            per[str(ci)] = config_summary(r, peaks)
    head = measure_workload(args.workload, args.method, args.weight_bits, args.steps,
                            args.warmup, args.copies, dev, keep_layers=True,
                            sclk_s=0.0 if args.no_sclk else 1.5)
    cfg, layers = head["cfg"], head["layers"]
    log(f"[bench] timed {args.steps} steps: {head['step_ms']:.4f} ms/step, stage 2 "
        f"{head['gemm_ms']:.4f} ms")
    ms = head["step_ms"]
    tops = head["ops"] / (ms * 1e-3) / 1e12
    roof = roofline_of(head, peaks)
    src_hash = kernel_source_hash()
    traffic = (traffic_from_profiles(cfg.name, src_hash)
               if args.weight_bits == 8 and args.method == "masquant" else None)
    roof.update({
        "kernel": head["kernel"],
        "traffic": traffic,
        "gemm_ms": round(head["gemm_ms"], 5),
        "gemm_timing": f"{args.steps} rounds of the stage-2 launches back to back on rotating "
                       "copies, one event pair on the launch stream (inter-launch gaps included)",
        "ops_per_step": int(head["ops"]), "algorithmic_bytes_per_step": int(head["gemm_bytes"]),
    })
    record = {
        "metric": "effective TOPS of modality-aware W8A8+low-rank linear; % int8 MFMA / HBM peak",
        "value": round(tops, 2),
        "unit": "TOPS",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "warmup_steps_run": head["warmup_steps_run"],
        "warmup_rule": "W untimed steps, then more until 0.1 s of steps have run (GPU clocks "
                       "ramp up over milliseconds after idle)",
        "ms_per_step": round(ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int8",
        "data": "synthetic (seeded; text N(0,1), vision N(0,1)x30, audio N(0,1)x2, "
                "1% outlier channels)",
        "config": {
            "workload": cfg.name, "tokens": int(cfg.T),
            "projections": [[p.name, int(p.c_in), int(p.c_out)] for p in cfg.projections],
            "method": args.method, "rank": int(layers[0]["rank"]),
            "modality_counts": list(map(int, cfg.counts)),
            "io_dtype": cfg.act_dtype,
            "weight_dtype": "int8" if args.weight_bits == 8 else "int4 (packed, W4A8)",
            "factor_dtype": cfg.lr_dtype,
            "rotating_copies": head["copies"],
        },
        "effective_GBps": round(head["bytes"] / (ms * 1e-3) / 1e9, 1),
        "frac_hbm_peak_step": round(head["bytes"] / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        "frac_int8_peak_step": round(tops / INT8_PEAK_TOPS, 4),
        "step_percentiles_ms": {"median": round(head["median_ms"], 5),
                                "p10": round(head["p10_ms"], 5), "p90": round(head["p90_ms"], 5),
                                "steps": head["n_pct"]},
        "roofline": roof,
        "measured_peaks": peaks,
        "sclk_under_load": head["sclk"],
        "kernel_source_sha256_16": src_hash,
    }
    if not args.no_cpu and args.method == "masquant":
        try:
            record["cpu_baseline"] = cpu_baseline(layers)
        except Exception as e:          # the baseline is a report, never the measurement
            record["cpu_baseline"] = {"error": repr(e)}
    if per:
        record["configs"] = per
    print(json.dumps(record), flush=True)


if __name__ == "__main__":
    main()
