"""Decode-step benchmark of the fused dequant-GEMV over packed VBQ weights.

A step is every linear GEMV of one decode token of the chosen synthetic
workload, in call order, on one stream (Q|K|V and gate|up are stored as one
row-concatenated matrix each, since they read the same input).  Inputs are
resident in HBM before timing starts.  Default workload: the 9B-class step
(d_model 4096, 32 layers, GQA K/V 1024, MLP 14336, vocab 128256, widths drawn
from the {1:.69, 2:.15, 4:.12, 8:.04} mix), 129 GEMVs, ~1.95 GB streamed.

    python bench.py [--steps K] [--warmup W] [--workload 0..4] [--gpus 1]
    python bench.py --qat     # the selection-path forward (training), its own JSON line

Prints one JSON line.  `value` is effective GB/s = algorithmic bytes of the
step / wall time per step (HIP-graph replay of the step, or eager launches if
faster).  `roofline` is the dominant kernel of the step (the one with the most
GPU time): algorithmic bytes per launch / its average launch duration, timed
with HIP events on the launch stream around replays of a graph of its launches;
`traffic` is its HBM bytes per launch from the committed rocprofv3 counter
summary when that was taken on the current kernel source.  `step_roofline`
lists every kernel of the step the same way.  The default run also times the
one-GEMV and 131M-class workloads hot and cold and the device's plain
streaming-read ceiling.  cpu_baseline times the double-precision oracle on a
bounded sample of the same workload (host cores; a baseline only).
"""

import argparse
import ctypes
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0
METRIC = "fused dequant-GEMV effective HBM GB/s (% of peak) and µs per decode step"
# the kernels and the packer's layout choices (tile and chunk sizes) decide the traffic
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2607_02893_amd", "csrc", f)
                  for f in ("vbq_kernels.hip", "vbq_layout.hpp", "vbq_pack.cpp")]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "vbq_mv_kernel_9b_step_traffic.md")
TRAFFIC_CONFIG = "workload 3, M 1, widths mixed"  # the only configuration the counters were taken on
CALIB_BYTES = 256 << 20  # plain copy used to scale the HBM byte counters


# the selection-path forward (--qat): its own kernel source and counter summary
QAT_SOURCES = [os.path.join(ROOT, "paper_2607_02893_amd", "csrc", "vbq_select.hip")]
QAT_TRAFFIC_FILE = os.path.join(ROOT, "profiles", "vbq_qat_forward_kernel_131m_step_traffic.md")
QAT_TRAFFIC_CONFIG = "selection forward, 131M-class linear weights"
QAT_METRIC = ("selection-path forward (four candidate reconstructions + Gumbel-Softmax mix per 64-weight group) "
              "effective HBM GB/s and µs per training step")
# bytes per group: W and w_soft (64 fp32 each), logits, noise and pi (4 fp32 each), hardened width (1 byte)
QAT_BYTES_PER_GROUP = 256 + 256 + 16 + 16 + 16 + 1


def kernel_source_hash(sources=None):
    import hashlib
    h = hashlib.sha256()
    for path in (KERNEL_SOURCES if sources is None else sources):
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def _traffic_fields(config, path, expected_config, sources):
    """The `- key: value` fields of a committed counter summary, or None when it
    is missing, was taken on another kernel source, or on another configuration
    than `config`."""
    if config != expected_config:
        return None
    try:
        fields = {}
        with open(path) as f:
            for line in f:
                if ":" in line and line.startswith("- "):
                    k, v = line[2:].split(":", 1)
                    v = v.strip()
                    fields[k.strip()] = v.split("`")[1] if v.startswith("`") else v
    except OSError:
        return None
    if fields.get("kernel_source_sha256") != kernel_source_hash(sources) or fields.get("config") != expected_config:
        return None
    return fields


def measured_traffic(config, path=None, expected_config=None, sources=None):
    """HBM bytes per launch (every launch of the run) from a committed counter
    summary, or None (see _traffic_fields)."""
    path = TRAFFIC_FILE if path is None else path
    expected_config = TRAFFIC_CONFIG if expected_config is None else expected_config
    fields = _traffic_fields(config, path, expected_config, sources)
    try:
        return None if fields is None else int(fields["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def measured_traffic_per_kernel(config, path=None):
    """{kernel name: HBM bytes per launch} from the committed counter summary of
    the decode step, or None (see _traffic_fields)."""
    fields = _traffic_fields(config, TRAFFIC_FILE if path is None else path, TRAFFIC_CONFIG, None)
    try:
        return None if fields is None else {k: int(v["hbm_bytes_per_launch"])
                                            for k, v in json.loads(fields["per_kernel"]).items()}
    except (KeyError, ValueError, TypeError):
        return None


def canonical_kernel(name):
    """A profiler's kernel name in vbq_kernel_name's form: template arguments
    without spaces, the default last argument of vbq_mv_kernel dropped."""
    n = name.replace("void ", "").replace("(anonymous namespace)::", "").split("(")[0].replace(" ", "")
    return n[:-4] + ">" if n.endswith(",-1>") else n


def pmc_summary(fetch_dir, write_dir, kernel="vbq_mv_", sources=None):
    """Summarise two rocprofv3 --pmc runs of `bench.py --profile` (FETCH_SIZE,
    then WRITE_SIZE): per-launch KiB of the kernels whose name contains
    `kernel`, scaled by what the same counters read for the calibration copy
    of CALIB_BYTES."""
    import csv
    import glob

    def per_kernel(d, counter, by_name=False):
        path = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)[0]
        acc = {}
        for r in csv.DictReader(open(path)):
            if r["Counter_Name"] != counter:
                continue
            name = r["Kernel_Name"]
            # e.g. every one-row GEMV kernel of the decode step (per-unit and two-waves-per-unit)
            key = ("vbq" if not by_name else canonical_kernel(name)) if kernel in name else \
                ("copy" if "MulFunctor" in name and not by_name else None)
            if key is None:
                continue
            acc.setdefault(key, {}).setdefault(r["Dispatch_Id"], 0.0)
            acc[key][r["Dispatch_Id"]] += float(r["Counter_Value"])
        return {k: list(v.values()) for k, v in acc.items()}

    f, w = per_kernel(fetch_dir, "FETCH_SIZE"), per_kernel(write_dir, "WRITE_SIZE")
    calib_kib = CALIB_BYTES / 1024.0
    f_copy, w_copy = float(np.median(f["copy"])), float(np.median(w["copy"]))
    f_scale, w_scale = calib_kib / f_copy, calib_kib / w_copy
    fv, wv = np.array(f["vbq"]), np.array(w["vbq"])
    fetch_b = float(np.mean(fv)) * f_scale * 1024
    write_b = float(np.mean(wv)) * w_scale * 1024
    per = {}
    fk, wk = per_kernel(fetch_dir, "FETCH_SIZE", by_name=True), per_kernel(write_dir, "WRITE_SIZE", by_name=True)
    for name in sorted(fk):
        if name in wk:
            b = float(np.mean(fk[name])) * f_scale * 1024 + float(np.mean(wk[name])) * w_scale * 1024
            per[name] = {"launches": len(fk[name]), "hbm_bytes_per_launch": int(round(b))}
    return {"launches": int(fv.size), "fetch_kib_per_launch_raw": float(np.mean(fv)),
            "write_kib_per_launch_raw": float(np.mean(wv)), "copy_fetch_kib": f_copy, "copy_write_kib": w_copy,
            "fetch_scale": f_scale, "write_scale": w_scale, "fetch_bytes_per_launch": fetch_b,
            "write_bytes_per_launch": write_b, "hbm_bytes_per_launch": int(round(fetch_b + write_b)),
            "per_kernel": per, "kernel_source_sha256": kernel_source_hash(sources)}


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def algorithmic_bytes(bits, N, K, M=1):
    """Codes (8*b per group) + fp16 scales + 2-bit width map + x (fp16) + y (fp32)."""
    groups = bits.size
    codes = int(np.sum(8 * bits.astype(np.int64)))
    wmap = groups / 4.0 if np.unique(bits).size > 1 else 0.0
    return codes + 2 * groups + wmap + 2 * M * K + 4 * M * N


def _gen_pack(task):
    """Worker: draw one matrix and pack it with libvbq (host only).  A matrix
    with per-row widths (the recipe's tiered head) is packed as one row bucket
    per width; every other matrix as one blob.  Returns its parts as
    (output rows or None, blob, descriptor bytes, algorithmic bytes)."""
    idx, cfg, seed, spec = task
    from paper_2607_02893_amd import synth, vbq
    bits, q, s = synth.make_matrix(spec, seed)
    whole = None
    if spec.row_tiers is not None:
        rb = vbq.pack_row_buckets(q, s, bits, n_threads=1)
        parts = [(rows, np.asarray(blob).copy(), bytes(d), algorithmic_bytes(bits[rows], len(rows), spec.K))
                 for _, rows, blob, d in rb]
        # the whole blob, bucket table and row index: one vbq_gemv_buckets call
        whole = (np.asarray(rb.blob).copy(), [bytes(b) for b in rb.buckets], rb.row_index.copy())
    else:
        blob, desc = vbq.pack_codes(q, s, bits, n_threads=1)
        parts = [(None, np.asarray(blob).copy(), bytes(desc), algorithmic_bytes(bits, spec.N, spec.K))]
    return idx, parts, spec.N * spec.K, whole


def prepare(cfg, workers, uniform_bits=0, recipe=False):
    from paper_2607_02893_amd import synth
    wl = synth.workload(cfg, uniform_bits, recipe=recipe)
    tasks = [(i, cfg, wl.seed, m) for i, m in enumerate(wl.matrices)]
    out = [None] * len(tasks)
    t0 = time.time()
    if workers > 1:
        import multiprocessing as mp
        # fork before anything touches the GPU
        with mp.get_context("fork").Pool(workers) as pool:
            for r in pool.imap_unordered(_gen_pack, sorted(tasks, key=lambda t: -t[3].N * t[3].K)):
                out[r[0]] = r
    else:
        for t in tasks:
            r = _gen_pack(t)
            out[r[0]] = r
    log(f"generated + packed {len(tasks)} matrices in {time.time() - t0:.1f}s")
    return wl, out


def cpu_baseline(wl, budget_s=20.0):
    """Oracle (numpy fp64 dequant + matvec) on the first matrices of the step
    until the time budget is spent, scaled by weight count to a full step."""
    from oracle import matmul as omatmul
    from paper_2607_02893_amd import synth
    try:
        from threadpoolctl import threadpool_info
        blas_threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:
        blas_threads = None
    total_w = sum(m.N * m.K for m in wl.matrices)
    done_w, spent, names = 0, 0.0, []
    for spec in wl.matrices:
        bits, q, s = synth.make_matrix(spec, wl.seed)
        x = synth.make_x(spec, wl.seed)[0]
        t0 = time.perf_counter()
        rows = max(1, (1 << 25) // spec.K)  # row blocks keep the fp64 matrix bounded
        y = np.empty(spec.N)
        for r0 in range(0, spec.N, rows):
            y[r0:r0 + rows] = omatmul.gemv(q[r0:r0 + rows], s[r0:r0 + rows], x)
        spent += time.perf_counter() - t0
        done_w += spec.N * spec.K
        names.append(f"{spec.name}{spec.layer}")
        if spent >= budget_s:
            break
    s_per_step = spent * total_w / done_w
    cores = len(os.sched_getaffinity(0))
    return {"value": round(1e3 * s_per_step, 1), "unit": "ms/step", "cores": blas_threads or cores,
            "host_cores_visible": cores, "kind": "oracle",
            "sample": f"{len(names)} of {len(wl.matrices)} matrices ({done_w / 1e6:.0f}M of {total_w / 1e6:.0f}M "
                      f"weights: {', '.join(names[:6])}{'...' if len(names) > 6 else ''}), "
                      f"{spent:.1f}s, scaled by weight count",
            "gb_per_s_equiv": None}


def write_traffic_file(path, summ):
    """The committed form of the counter summary that measured_traffic() reads."""
    lines = [
        "# HBM traffic of vbq_mv_kernel<1>: 9B-class decode step (129 GEMVs, M=1)",
        "",
        "Two counter passes over `bench.py --profile --workers 1 --steps 2 --warmup 1` (the step's HIP graph",
        "replayed 3 times; the weights packed in the process itself, since a worker process of the packing",
        "pool that receives the pool's SIGTERM stalls in the counter tool's shutdown), then a plain copy of",
        "256 MiB (torch.mul by 1.0) to scale the counters to bytes:",
        "",
        "```",
        "cd /tmp && export TMPDIR=/tmp",
        "timeout -s KILL 300 rocprofv3 --pmc FETCH_SIZE --output-format csv -d $OUT/pmc_fetch -o run -- "
        "python3 $R/bench.py --profile --workers 1 --steps 2 --warmup 1",
        "timeout -s KILL 300 rocprofv3 --pmc WRITE_SIZE --output-format csv -d $OUT/pmc_write -o run -- "
        "python3 $R/bench.py --profile --workers 1 --steps 2 --warmup 1",
        "python3 bench.py --pmc-summary $OUT/pmc_fetch $OUT/pmc_write --write-traffic <this file>",
        "```",
        "",
        "(`$R` is the repository root, `$OUT` an output directory.)  Per-launch figures, averaged over every GEMV launch of the step:",
        "",
        f"- config: {TRAFFIC_CONFIG}",
        f"- launches: {summ['launches']}",
        f"- fetch_kib_per_launch_raw: {summ['fetch_kib_per_launch_raw']:.1f}",
        f"- write_kib_per_launch_raw: {summ['write_kib_per_launch_raw']:.1f}",
        f"- copy_fetch_kib (256 MiB read): {summ['copy_fetch_kib']:.0f}",
        f"- copy_write_kib (256 MiB written): {summ['copy_write_kib']:.0f}",
        f"- fetch_scale: {summ['fetch_scale']:.4f}",
        f"- write_scale: {summ['write_scale']:.4f}",
        f"- fetch_bytes_per_launch: {summ['fetch_bytes_per_launch']:.0f}",
        f"- write_bytes_per_launch: {summ['write_bytes_per_launch']:.0f}",
        f"- hbm_bytes_per_launch: {summ['hbm_bytes_per_launch']}",
        f"- per_kernel: `{json.dumps(summ.get('per_kernel', {}), sort_keys=True)}`",
        f"- kernel_source_sha256: `{summ['kernel_source_sha256']}` (vbq_kernels.hip, vbq_layout.hpp, "
        "vbq_pack.cpp)",
        "",
        "bench.py reports hbm_bytes_per_launch as roofline.traffic while the kernel source still has this hash.",
    ]
    with open(path, "w") as f:
        f.write("\n".join(lines) + "\n")


def write_qat_traffic_file(path, summ):
    """Counter summary of the selection-path forward kernel (read back by measured_traffic)."""
    lines = [
        "# HBM traffic of vbq_qat_forward_kernel: 131M-class training step (one launch)",
        "",
        "Two counter passes over `bench.py --qat --profile --steps 2 --warmup 1` (3 forward launches over the",
        "131M-class model's 137.8M linear weights), then a plain copy of 256 MiB (torch.mul by 1.0) to",
        "scale the counters to bytes:",
        "",
        "```",
        "cd /tmp && export TMPDIR=/tmp",
        "timeout -s KILL 300 rocprofv3 --pmc FETCH_SIZE --output-format csv -d $OUT/pmc_qat_fetch -o run -- "
        "python3 $R/bench.py --qat --profile --steps 2 --warmup 1",
        "timeout -s KILL 300 rocprofv3 --pmc WRITE_SIZE --output-format csv -d $OUT/pmc_qat_write -o run -- "
        "python3 $R/bench.py --qat --profile --steps 2 --warmup 1",
        "python3 bench.py --qat --pmc-summary $OUT/pmc_qat_fetch $OUT/pmc_qat_write "
        "--write-traffic <this file>",
        "```",
        "",
        "(`$R` is the repository root, `$OUT` an output directory.)  Per-launch figures, averaged over the forward launches:",
        "",
        f"- config: {QAT_TRAFFIC_CONFIG}",
        f"- launches: {summ['launches']}",
        f"- fetch_kib_per_launch_raw: {summ['fetch_kib_per_launch_raw']:.1f}",
        f"- write_kib_per_launch_raw: {summ['write_kib_per_launch_raw']:.1f}",
        f"- copy_fetch_kib (256 MiB read): {summ['copy_fetch_kib']:.0f}",
        f"- copy_write_kib (256 MiB written): {summ['copy_write_kib']:.0f}",
        f"- fetch_scale: {summ['fetch_scale']:.4f}",
        f"- write_scale: {summ['write_scale']:.4f}",
        f"- fetch_bytes_per_launch: {summ['fetch_bytes_per_launch']:.0f}",
        f"- write_bytes_per_launch: {summ['write_bytes_per_launch']:.0f}",
        f"- hbm_bytes_per_launch: {summ['hbm_bytes_per_launch']}",
        f"- kernel_source_sha256: `{summ['kernel_source_sha256']}` (vbq_select.hip)",
        "",
        "bench.py --qat reports hbm_bytes_per_launch as roofline.traffic while the kernel source still has this hash.",
    ]
    with open(path, "w") as f:
        f.write("\n".join(lines) + "\n")


def qat_cpu_baseline(W, logits, noise, tau, n, budget_s=20.0):
    """Oracle (numpy fp64) forward on consecutive chunks of groups until the
    time budget is spent, scaled by group count to the whole step."""
    from oracle import qat as oqat
    chunk = 16384
    done, spent = 0, 0.0
    while done < n and spent < budget_s:
        c = min(chunk, n - done)
        w = W[64 * done:64 * (done + c)].reshape(c, 64)
        t0 = time.perf_counter()
        oqat.forward(w, logits[done:done + c].reshape(c, 1, 4), noise[done:done + c].reshape(c, 1, 4), tau)
        spent += time.perf_counter() - t0
        done += c
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:
        threads = None
    s_per_step = spent * n / done
    cores = len(os.sched_getaffinity(0))
    return {"value": round(1e3 * s_per_step, 1), "unit": "ms/step", "cores": threads or cores,
            "host_cores_visible": cores, "kind": "oracle",
            "sample": f"first {done} of {n} groups ({done * 64 / 1e6:.1f}M of {n * 64 / 1e6:.1f}M weights) in "
                      f"chunks of {chunk}, {spent:.1f}s, scaled by group count"}


def main_qat(args):
    """--qat: the selection-path forward over the 131M-class model's linear
    weights laid end to end (paper section 3.2, Algorithm 1), one launch of the
    forward kernel plus the bbar reduction per step."""
    from paper_2607_02893_amd import synth
    name, mats, n = synth.selection_workload(1)
    tau = 0.5
    t0 = time.time()
    W, logits, noise = synth.selection_inputs(n, part=1)
    log(f"{name}: {len(mats)} matrices, {n} groups ({n * 64 / 1e6:.1f}M weights), inputs drawn in "
        f"{time.time() - t0:.1f}s")

    import torch
    from paper_2607_02893_amd import vbq
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    Wd = torch.from_numpy(W).to(dev)
    ld = torch.from_numpy(logits).to(dev)
    nd = torch.from_numpy(noise).to(dev)
    ws = torch.empty_like(Wd)
    pi = torch.empty((n, 4), dtype=torch.float32, device=dev)
    hard = torch.empty(n, dtype=torch.uint8, device=dev)
    bbar = torch.empty(1, dtype=torch.float64, device=dev)
    ws_bytes = vbq.qat_workspace_size(n)
    work = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream()
    sptr = stream.cuda_stream
    blocks = ws_bytes // 8
    alg_kernel = n * QAT_BYTES_PER_GROUP + 8 * blocks          # the forward kernel (its partial sums included)
    alg_step = alg_kernel + 8 * blocks + 8                      # + the bbar reduction

    def fwd(with_bbar=True):
        st = vbq.raw_qat_forward(n, Wd.data_ptr(), ld.data_ptr(), nd.data_ptr(), tau, ws.data_ptr(), pi.data_ptr(),
                                 hard.data_ptr(), bbar.data_ptr() if with_bbar else 0,
                                 work.data_ptr() if with_bbar else 0, ws_bytes if with_bbar else 0, sptr)
        if st != 0:
            raise vbq.VbqError(st, "vbq_qat_forward")

    for _ in range(args.warmup):
        fwd()
    torch.cuda.synchronize()
    if args.profile:
        # the launches the roofline times (the forward kernel alone, back to back),
        # then a few whole steps (forward + bbar)
        t0 = time.perf_counter()
        for _ in range(args.steps):
            fwd(False)
        torch.cuda.synchronize()
        dt = (time.perf_counter() - t0) / args.steps
        for _ in range(3):
            fwd()
        torch.cuda.synchronize()
        src = torch.ones(CALIB_BYTES // 4, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.mul(src, 1.0, out=dst)
        torch.cuda.synchronize()
        print(json.dumps({"profile_run": True, "us_per_step_eager": round(1e6 * dt, 2)}), flush=True)
        return

    def timed(run, k):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        e0.record(stream)
        for _ in range(k):
            run()
        e1.record(stream)
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) / k, e0.elapsed_time(e1) * 1e-3 / k

    wall_s, gpu_s = timed(fwd, args.steps)
    log(f"step (forward + bbar): {1e6 * wall_s:.1f} us wall, {1e6 * gpu_s:.1f} us events")
    # the forward kernel alone, K launches back to back on the same stream
    _, kern_s = timed(lambda: fwd(False), args.steps)
    log(f"forward kernel alone: {1e6 * kern_s:.1f} us per launch")
    # the same forward writing w_soft as bf16 (6 bytes per weight instead of 8)
    ws16 = torch.empty(n * 64, dtype=torch.bfloat16, device=dev)

    def fwd16():
        st = vbq.raw_qat_forward(n, Wd.data_ptr(), ld.data_ptr(), nd.data_ptr(), tau, ws16.data_ptr(), pi.data_ptr(),
                                 hard.data_ptr(), 0, 0, 0, sptr, flags=vbq.QAT_WSOFT_BF16)
        if st != 0:
            raise vbq.VbqError(st, "vbq_qat_forward (bf16)")
    for _ in range(3):
        fwd16()
    _, k16_s = timed(fwd16, args.steps)
    alg16 = alg_kernel - n * 64 * 2
    log(f"forward kernel, bf16 w_soft: {1e6 * k16_s:.1f} us per launch, {alg16 / k16_s / 1e9:.0f} GB/s")
    del ws16
    # the logit step's gradient (Algorithm 1, every m-th step): same weights, a
    # seeded dL/dw_soft, the forward's pi
    grad = torch.from_numpy(synth.rng_for(synth.SELECTION_SEED, 3004, 1).standard_normal(
        n * 64, dtype=np.float32)).to(dev)
    dlog = torch.empty((n, 4), dtype=torch.float32, device=dev)

    def lgrad():
        st = vbq.raw_qat_logit_grad(n, Wd.data_ptr(), grad.data_ptr(), pi.data_ptr(), tau, 0.05, n,
                                    dlog.data_ptr(), sptr)
        if st != 0:
            raise vbq.VbqError(st, "vbq_qat_logit_grad")
    for _ in range(3):
        lgrad()
    _, grad_s = timed(lgrad, args.steps)
    alg_grad = n * (256 + 256 + 16 + 16)
    log(f"logit-step gradient: {1e6 * grad_s:.1f} us per launch, {alg_grad / grad_s / 1e9:.0f} GB/s")
    del grad
    torch.cuda.synchronize()
    value = alg_step / wall_s / 1e9
    achieved = alg_kernel / kern_s / 1e9
    traffic = measured_traffic(QAT_TRAFFIC_CONFIG, QAT_TRAFFIC_FILE, QAT_TRAFFIC_CONFIG, QAT_SOURCES)
    # plain copy of the same bytes through torch (context: what the chip streams)
    cp_src = torch.empty(n * 64 + n * 12, dtype=torch.float32, device=dev)
    cp_dst = torch.empty_like(cp_src)
    for _ in range(3):
        cp_dst.copy_(cp_src)
    _, copy_s = timed(lambda: cp_dst.copy_(cp_src), max(5, args.steps // 4))
    copy_gbs = 2 * cp_src.numel() * 4 / copy_s / 1e9
    log(f"torch copy of {2 * cp_src.numel() * 4 / 1e6:.0f} MB (read + write): {1e6 * copy_s:.1f} us, {copy_gbs:.0f} GB/s")
    del cp_src, cp_dst
    cpu = None
    if not args.no_cpu:
        cpu = qat_cpu_baseline(W, logits, noise, tau, n)
        log(f"cpu oracle: {cpu['value']} ms/step ({cpu['sample']})")
    out = {
        "metric": QAT_METRIC,
        "value": round(value, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(1e3 * wall_s, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "precision": "fp32 weights in and out, fp16-rounded scales, double-precision group statistics",
        "data": "synthetic (seeded draws; no trained weights)",
        "config": {"workload": f"{name} selection-path forward: the linear weights of {len(mats)} matrices "
                               f"end to end, {n * 64 / 1e6:.1f}M weights, {n} groups, tau {tau}",
                   "algorithmic_bytes_per_step": int(alg_step)},
        "us_per_step": round(1e6 * wall_s, 2),
        "pct_of_peak_hbm": round(100 * value / PEAK_HBM_GBS, 1),
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": round(achieved / PEAK_HBM_GBS, 4), "traffic": traffic,
                     "kernel": "vbq_qat_forward_kernel",
                     "launches_per_step": 1,
                     "algorithmic_bytes_per_launch": int(alg_kernel),
                     "avg_launch_us": round(1e6 * kern_s, 3),
                     "timing": "HIP events on the launch stream around K launches of the kernel alone",
                     "traffic_unit": "HBM bytes per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, copy-calibrated)",
                     "traffic_vs_algorithmic": round(traffic / alg_kernel, 3) if traffic else None},
        "w_soft_bf16": {"kernel": "vbq_qat_forward_kernel<bf16>", "us_per_launch": round(1e6 * k16_s, 2),
                        "algorithmic_bytes": int(alg16), "GBps": round(alg16 / k16_s / 1e9, 1),
                        "frac": round(alg16 / k16_s / 1e9 / PEAK_HBM_GBS, 4),
                        "note": "the same forward writing w_soft as bf16 (rounded to nearest even)"},
        "logit_grad": {"kernel": "vbq_qat_grad_kernel", "us_per_launch": round(1e6 * grad_s, 2),
                       "algorithmic_bytes": int(alg_grad), "GBps": round(alg_grad / grad_s / 1e9, 1),
                       "frac": round(alg_grad / grad_s / 1e9 / PEAK_HBM_GBS, 4),
                       "note": "W and dL/dw_soft read, pi read, dL/dlogits written (Algorithm 1 logit step)"},
        "copy_GBps": round(copy_gbs, 1),
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", type=int, default=3)
    ap.add_argument("--batch", type=int, default=1, help="activation rows M (M > 1 times vbq_gemm_small)")
    ap.add_argument("--uniform", type=int, default=0, choices=(0, 1, 2, 4, 8),
                    help="every group of every matrix at this width (the 1.46B workload's roofline variants)")
    ap.add_argument("--recipe", action="store_true",
                    help="the deployed recipe's widths (one width per projection, the LM head as row buckets)")
    ap.add_argument("--workers", type=int, default=min(12, len(os.sched_getaffinity(0))))
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--no-dense", action="store_true")
    ap.add_argument("--no-small", action="store_true",
                    help="skip the hot / cold timing of workloads 0 and 1 that the default run adds")
    ap.add_argument("--cold", type=int, default=0, metavar="K",
                    help="also time K steps one by one, each after a 1 GiB write that evicts L2 and the "
                         "Infinity Cache (the write is outside the timed region)")
    ap.add_argument("--profile", action="store_true",
                    help="short run for rocprofv3: the step's graph replayed --steps times, then a calibration copy")
    ap.add_argument("--pmc-summary", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="summarise two rocprofv3 --pmc runs of --profile (FETCH_SIZE, WRITE_SIZE) and exit")
    ap.add_argument("--write-traffic", metavar="PATH", help="with --pmc-summary: write the traffic summary file")
    ap.add_argument("--persistent", action="store_true",
                    help="time the step as one launch (vbq_step_run) instead of one launch per GEMV")
    ap.add_argument("--qat", action="store_true",
                    help="time the selection-path forward (training) over the 131M-class weights instead")
    args = ap.parse_args()
    if args.pmc_summary:
        if args.qat:
            summ = pmc_summary(*args.pmc_summary, kernel="vbq_qat_forward_kernel", sources=QAT_SOURCES)
        else:
            summ = pmc_summary(*args.pmc_summary)
        print(json.dumps(summ), flush=True)
        if args.write_traffic:
            (write_qat_traffic_file if args.qat else write_traffic_file)(args.write_traffic, summ)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the fused GEMV path has no multi-GPU mode "
              "(the row / K split that would shard it is described in the design notes).", file=sys.stderr)
        sys.exit(2)
    if args.qat:
        return main_qat(args)

    if args.recipe and (args.batch != 1 or args.uniform):
        print("--recipe runs one activation row with the recipe's own widths", file=sys.stderr)
        sys.exit(2)
    wl, packed = prepare(args.workload, args.workers, args.uniform, args.recipe)

    import torch
    from paper_2607_02893_amd import vbq

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()
    M = args.batch
    st = build_step(wl, packed, M, dev)
    del packed
    log(f"{len(st.mats)} matrices in {len(st.calls)} launches, {st.total_w / 1e9:.2f}G weights, "
        f"algorithmic {st.total_alg / 1e6:.1f} MB/step, blobs {st.blob_bytes / 1e6:.1f} MB")
    for _ in range(args.warmup):
        st.run(stream.cuda_stream)
    torch.cuda.synchronize()
    if args.persistent:
        return main_persistent(args, wl, st, stream)
    g = st.graph(stream)

    if args.profile:
        # the timed loop itself (graph replay) for the profiler, then the
        # calibration copy of known size for the HBM byte counters
        for _ in range(args.warmup):
            g.replay()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            g.replay()
        torch.cuda.synchronize()
        dt = (time.perf_counter() - t0) / args.steps
        log(f"profile run: {args.steps} graph replays, {1e6 * dt:.1f} us/step")
        src = torch.ones(CALIB_BYTES // 4, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.mul(src, 1.0, out=dst)
        torch.cuda.synchronize()
        print(json.dumps({"profile_run": True, "us_per_step_graph": round(1e6 * dt, 2)}), flush=True)
        return

    # eager launches and graph replay of the same launches; the faster is reported
    eager_s, eager_gpu_s = timed(lambda: st.run(stream.cuda_stream), args.steps, stream)
    log(f"eager: {1e6 * eager_s:.1f} us/step (events {1e6 * eager_gpu_s:.1f})")
    for _ in range(args.warmup):
        g.replay()
    graph_s, graph_gpu_s = timed(g.replay, args.steps, stream)
    log(f"graph: {1e6 * graph_s:.1f} us/step (events {1e6 * graph_gpu_s:.1f})")
    ref = [m[2].clone() for m in st.mats[:3] + st.mats[-1:]]
    st.run(stream.cuda_stream)
    torch.cuda.synchronize()
    for r, m in zip(ref, st.mats[:3] + st.mats[-1:]):
        assert torch.equal(r, m[2]), "graph replay differs from eager launch"
    use_graph = graph_s <= eager_s
    wall_s = graph_s if use_graph else eager_s
    run_one = g.replay if use_graph else (lambda: st.run(stream.cuda_stream))
    step_dist = distribution(run_one, min(100, args.steps), stream)
    log(f"single steps: median {step_dist['median']} us, p10 {step_dist['p10']}, p90 {step_dist['p90']}")

    flush = torch.empty(1 << 28, dtype=torch.float32, device=dev)  # 1 GiB: evicts L2 and the Infinity Cache
    cold_us = cold_steps(run_one, args.cold, flush, stream) if args.cold > 0 else None
    if cold_us:
        log(f"cold: {cold_us['median']:.1f} us/step (median of {args.cold}, caches flushed before each)")

    # every kernel of the step alone: its launches, in step order, as one graph
    # replayed back to back on the launch stream (HIP events around the loop)
    kern = per_kernel_timing(st, stream, args.steps, args.warmup)
    dominant = max(kern, key=lambda k: kern[k]["launches"] * kern[k]["avg_launch_us"])
    sum_kernel_us = sum(v["launches"] * v["avg_launch_us"] for v in kern.values())
    log("kernels: " + ", ".join(f"{k} x{v['launches']} {v['avg_launch_us']:.2f} us {v['GBps']:.0f} GB/s"
                                for k, v in kern.items()))
    per_shape = per_shape_timing(st, stream, min(5, args.steps))
    log(f"per shape (launch bracketed by events): {per_shape}")

    dense = None if args.no_dense else dense_baseline(st, M, args.steps, dev, min(eager_s, graph_s))
    if dense:
        log(f"dense fp16: {dense['us_per_step']:.1f} us/step")

    config_key = (f"workload {args.workload}, M {M}, "
                  f"widths {'recipe' if args.recipe else 'uniform ' + str(args.uniform) if args.uniform else 'mixed'}")
    traffic_all = measured_traffic(config_key)
    traffic_k = measured_traffic_per_kernel(config_key)
    dk = kern[dominant]
    t_dom = traffic_k.get(dominant) if traffic_k else None
    achieved = dk["alg_bytes_per_launch"] / (1e-6 * dk["avg_launch_us"]) / 1e9
    value = st.total_alg / wall_s / 1e9
    step_counters = None
    if traffic_k and all(k in traffic_k for k in kern):
        hbm = sum(traffic_k[k] * v["launches"] for k, v in kern.items())
        step_counters = {"hbm_bytes_per_step": hbm, "vs_algorithmic": round(hbm / st.total_alg, 3),
                         "frac_of_sum_kernel_time": round(hbm / (1e-6 * sum_kernel_us) / 1e9 / PEAK_HBM_GBS, 4),
                         "frac_of_step_time": round(hbm / wall_s / 1e9 / PEAK_HBM_GBS, 4)}

    small = None
    if not args.no_small and args.workload == 3 and M == 1 and not args.recipe and not args.uniform:
        small = {f"workload {c}": small_workload(c, args, dev, stream, flush) for c in (0, 1)}
    ceiling = read_ceiling(flush, stream)
    log(f"streaming-read ceiling: {ceiling['GBps']:.0f} GB/s ({ceiling['blocks']} blocks)")
    del flush
    torch.cuda.empty_cache()

    cpu = None
    if not args.no_cpu:
        cpu = cpu_baseline(wl)
        log(f"cpu oracle: {cpu['value']} ms/step ({cpu['sample']})")
    n_launch = len(st.calls)
    out = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(1e3 * wall_s, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "precision": "fp16 activations x {1,2,4,8}-bit codes with fp16 group scales, fp32 accumulation",
        "data": "synthetic (seeded draws; no trained weights)",
        "config": {"workload": f"{wl.name} decode step (workload {args.workload}): {len(st.mats)} GEMVs"
                               f"{f' in {n_launch} launches' if n_launch != len(st.mats) else ''}, "
                               f"{st.total_w / 1e9:.2f}G weights", "M": M,
                   "uniform_bits": args.uniform or None, "recipe": bool(args.recipe),
                   "algorithmic_bytes_per_step": int(st.total_alg), "blob_bytes": int(st.blob_bytes),
                   "timing": "HIP-graph replay of the step" if use_graph else "eager launches"},
        "us_per_step": round(1e6 * wall_s, 2),
        "us_per_step_eager": round(1e6 * eager_s, 2),
        "us_per_step_graph": round(1e6 * graph_s, 2),
        "us_per_step_cold": cold_us,
        "us_per_step_distribution": step_dist,
        "pct_of_peak_hbm": round(100 * value / PEAK_HBM_GBS, 1),
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": round(achieved / PEAK_HBM_GBS, 4), "traffic": t_dom,
                     "kernel": dominant,
                     "launches_per_step": dk["launches"],
                     "share_of_step_kernel_time": round(dk["launches"] * dk["avg_launch_us"] / sum_kernel_us, 3),
                     "algorithmic_bytes_per_launch": round(dk["alg_bytes_per_launch"]),
                     "avg_launch_us": dk["avg_launch_us"],
                     "timing": "HIP events on the launch stream around K replays of a graph of this kernel's "
                               "launches of one step (step order, back to back)",
                     "traffic_unit": "HBM bytes per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, copy-calibrated)",
                     "traffic_vs_algorithmic": round(t_dom / dk["alg_bytes_per_launch"], 3) if t_dom else None,
                     "frac_from_counters": round(t_dom / (1e-6 * dk["avg_launch_us"]) / 1e9 / PEAK_HBM_GBS, 4)
                     if t_dom else None},
        "step_roofline": {"sum_kernel_us": round(sum_kernel_us, 1),
                          "frac_algorithmic_of_step_time": round(value / PEAK_HBM_GBS, 4),
                          "frac_algorithmic_of_sum_kernel_time":
                              round(st.total_alg / (1e-6 * sum_kernel_us) / 1e9 / PEAK_HBM_GBS, 4),
                          "counters": step_counters,
                          "traffic_all_launches_per_launch": traffic_all,
                          "kernels": kern},
        "read_ceiling": ceiling,
        "small_workloads": small,
        "per_shape": per_shape,
        "cpu_baseline": cpu,
        "dense_fp16_baseline": dense,
    }
    print(json.dumps(out), flush=True)


def main_persistent(args, wl, st, stream):
    """--persistent: the same step as ONE launch (vbq_step_run): the GEMVs in
    order, each waiting for the previous one inside the kernel."""
    import torch
    from paper_2607_02893_amd import vbq
    ps = vbq.Step(st.launch_args)
    ref = [m[2].clone() for m in st.mats]  # per-GEMV launches (warm-up above)
    for m in st.mats:
        m[2].fill_(float("nan"))

    def run():
        r = ps.run(stream)
        if r != 0:
            raise vbq.VbqError(r, "vbq_step_run")
    run()
    torch.cuda.synchronize()
    if ps.status() != 0:
        raise RuntimeError("vbq_step_run: a wait timed out")
    same = all(torch.equal(r, m[2]) for r, m in zip(ref, st.mats))
    log(f"one-launch step equals the per-GEMV launches bit for bit: {same}")
    if not same:
        raise RuntimeError("one-launch step differs from the per-GEMV launches")
    for _ in range(args.warmup):
        run()
    if args.profile:
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            run()
        torch.cuda.synchronize()
        dt = (time.perf_counter() - t0) / args.steps
        print(json.dumps({"profile_run": True, "persistent": True, "us_per_step": round(1e6 * dt, 2)}), flush=True)
        return
    wall_s, gpu_s = timed(run, args.steps, stream)
    dist = distribution(run, min(100, args.steps), stream)
    torch.cuda.synchronize()
    assert ps.status() == 0
    # the per-GEMV path on the same tree, for comparison
    g = st.graph(stream)
    for _ in range(args.warmup):
        g.replay()
    per_s, _ = timed(g.replay, args.steps, stream)
    log(f"one launch: {1e6 * wall_s:.1f} us/step (events {1e6 * gpu_s:.1f}); one launch per GEMV "
        f"(graph): {1e6 * per_s:.1f} us/step")
    value = st.total_alg / wall_s / 1e9
    out = {
        "metric": METRIC, "value": round(value, 1), "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(1e3 * wall_s, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32",
        "precision": "fp16 activations x {1,2,4,8}-bit codes with fp16 group scales, fp32 accumulation",
        "data": "synthetic (seeded draws; no trained weights)",
        "config": {"workload": f"{wl.name} decode step (workload {args.workload}) as one launch: "
                               f"{len(st.launch_args)} GEMVs, {st.total_w / 1e9:.2f}G weights", "M": 1,
                   "algorithmic_bytes_per_step": int(st.total_alg),
                   "timing": "eager vbq_step_run calls (a clearing kernel + one cooperative launch)"},
        "us_per_step": round(1e6 * wall_s, 2), "us_per_step_distribution": dist,
        "us_per_step_per_gemv_launches": round(1e6 * per_s, 2),
        "pct_of_peak_hbm": round(100 * value / PEAK_HBM_GBS, 1),
        "roofline": {"bound": "hbm", "achieved": round(st.total_alg / gpu_s / 1e9, 1), "peak": PEAK_HBM_GBS,
                     "unit": "GB/s", "frac": round(st.total_alg / gpu_s / 1e9 / PEAK_HBM_GBS, 4), "traffic": None,
                     "kernel": "vbq_step_kernel", "launches_per_step": 1,
                     "algorithmic_bytes_per_launch": int(st.total_alg), "avg_launch_us": round(1e6 * gpu_s, 2),
                     "timing": "HIP events on the launch stream around K steps"},
        "bitwise_equal_to_per_gemv_launches": same,
        "cpu_baseline": None,
    }
    print(json.dumps(out), flush=True)


class Step:
    """The launches of one decode step on device.  launch_args: per GEMV (one per
    bucket of a bucketed matrix) (desc, blob, x, y, output-row map or 0, len(y)),
    what the one-launch step takes.  calls: the launches the step makes, each
    ("gemv", launch_args index) or ("buckets", table, n, blob, row index, x, y,
    len(y)) for a bucketed matrix in one vbq_gemv_buckets call; with each call's
    algorithmic bytes, kernel name and shape label."""

    def __init__(self, M):
        self.M = M
        self.mats = []        # per matrix: ([(PackedMatrix, rows or None)], x, y, algorithmic bytes)
        self.launch_args = []
        self.calls = []
        self.launch_alg = []  # per call
        self.kernels = []     # per call
        self.labels = []      # per call
        self.total_alg = 0.0
        self.total_w = 0
        self.blob_bytes = 0
        self._keep = []       # device buffers and ctypes tables the calls point at

    def launch(self, i, stream_ptr):
        from paper_2607_02893_amd import vbq
        c = self.calls[i]
        if c[0] == "buckets":
            return vbq.raw_gemv_buckets(*c[1:], stream_ptr)
        d, b, x, y, rows, ylen = self.launch_args[c[1]]
        if rows:
            return vbq.raw_gemv_rows(d, b, x, y, ylen, rows, stream_ptr)
        if self.M == 1:
            return vbq.raw_gemv(d, b, x, y, stream_ptr)
        return vbq.raw_gemm_small(d, b, self.M, x, d.K, y, d.N, stream_ptr)

    def run(self, stream_ptr, idx=None):
        from paper_2607_02893_amd import vbq
        for i in (range(len(self.calls)) if idx is None else idx):
            r = self.launch(i, stream_ptr)
            if r != 0:
                raise vbq.VbqError(r, "vbq_gemv / vbq_gemv_rows / vbq_gemv_buckets / vbq_gemm_small")

    def graph(self, stream, idx=None, reps=1):
        """The launches (all, or those in idx) captured as one HIP graph, reps
        times in a row (a graph of a few short kernels replayed back to back
        would otherwise time the host's graph launches)."""
        import torch
        g = torch.cuda.CUDAGraph()
        cap = torch.cuda.Stream()
        cap.wait_stream(stream)
        with torch.cuda.stream(cap):
            g.capture_begin()
            for _ in range(reps):
                self.run(cap.cuda_stream, idx)
            g.capture_end()
        stream.wait_stream(cap)
        return g


def build_step(wl, packed, M, dev):
    import torch
    from paper_2607_02893_amd import synth, vbq
    st = Step(M)
    for idx, parts, nw, whole in packed:
        spec = wl.matrices[idx]
        xm = synth.make_x(spec, wl.seed, M)
        x = torch.from_numpy(np.ascontiguousarray(xm[0] if M == 1 else xm)).to(dev)
        y = torch.empty(spec.N if M == 1 else (M, spec.N), dtype=torch.float32, device=dev)
        table = None
        if whole is not None and M == 1:
            blob_all = torch.from_numpy(whole[0]).to(dev)
            rows_all = torch.from_numpy(whole[2]).to(dev)
            bks = [vbq.VbqBucket.from_buffer_copy(b) for b in whole[1]]
            if vbq.buckets_kernel_name(bks) != "per bucket":
                table = (vbq.VbqBucket * vbq.MAX_BUCKETS)(*bks)
                st._keep += [blob_all, rows_all, table]
        dev_parts, alg = [], 0.0
        for k, (rows, blob, dbytes, palg) in enumerate(parts):
            desc = vbq.VbqDesc.from_buffer_copy(dbytes)
            if table is not None:  # the bucket's bytes and rows inside the whole buffers
                off, r0 = int(table[k].blob_offset), int(table[k].row_begin)
                Wp = vbq.PackedMatrix.on_device(blob_all[off:off + int(desc.total_bytes)], desc)
                rt = rows_all[r0:r0 + len(rows)]
            else:
                Wp = vbq.PackedMatrix(blob, desc, device=dev)
                rt = None if rows is None else torch.from_numpy(rows).to(dev)
            dev_parts.append((Wp, rt))
            palg += (2 * spec.K + 4 * desc.N) * (M - 1)  # x and y of the extra rows
            st.launch_args.append((desc, Wp.blob.data_ptr(), x.data_ptr(), y.data_ptr(),
                                   0 if rt is None else rt.data_ptr(), spec.N))
            if table is None:
                st.calls.append(("gemv", len(st.launch_args) - 1))
                st.launch_alg.append(palg)
                st.kernels.append(vbq.kernel_name(desc, M))
                st.labels.append(f"{desc.N}x{desc.K}" + (" (row bucket)" if rt is not None else ""))
            alg += palg
            st.blob_bytes += desc.total_bytes
        if table is not None:
            st.calls.append(("buckets", table, len(parts), blob_all.data_ptr(), rows_all.data_ptr(),
                             x.data_ptr(), y.data_ptr(), spec.N))
            st.launch_alg.append(alg)
            st.kernels.append(vbq.buckets_kernel_name(list(table)[:len(parts)]))
            st.labels.append(f"{spec.N}x{spec.K} ({len(parts)} row buckets, one launch)")
        st.mats.append((dev_parts, x, y, alg))
        st.total_alg += alg
        st.total_w += nw
    return st


def timed(run, n, stream):
    """Wall time per call (host clock, synchronized on both sides) and GPU time
    per call (HIP events recorded on the launch stream around the same region)."""
    import torch
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    e0.record(stream)
    for _ in range(n):
        run()
    e1.record(stream)
    torch.cuda.synchronize()
    return (time.perf_counter() - t0) / n, e0.elapsed_time(e1) * 1e-3 / n


def distribution(run, n, stream):
    """Median / p10 / p90 of single calls, each bracketed by its own events."""
    import torch
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n)]
    for e0, e1 in ev:
        e0.record(stream)
        run()
        e1.record(stream)
    torch.cuda.synchronize()
    us = np.array([e0.elapsed_time(e1) * 1e3 for e0, e1 in ev])
    return {"median": round(float(np.median(us)), 2), "p10": round(float(np.percentile(us, 10)), 2),
            "p90": round(float(np.percentile(us, 90)), 2), "steps": n,
            "timing": "HIP events around each step, on the launch stream"}


def cold_steps(run, n, flush, stream):
    """Steps timed one by one, each after a 1 GiB write that evicts L2 and the
    Infinity Cache (the write is outside the timed region)."""
    import torch
    ts = []
    for _ in range(n):
        flush.fill_(1.0)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        run()
        e1.record(stream)
        torch.cuda.synchronize()
        ts.append(e0.elapsed_time(e1) * 1e3)
    return {"median": round(float(np.median(ts)), 2), "p10": round(float(np.percentile(ts, 10)), 2),
            "p90": round(float(np.percentile(ts, 90)), 2), "steps": n,
            "timing": "HIP events around each step after a 1 GiB flush write"}


def per_kernel_timing(st, stream, steps, warmup):
    """Per kernel of the step: its launches (step order, repeated up to at least
    64) as one graph, replayed back to back; average launch duration from HIP
    events around the loop."""
    out = {}
    for name in dict.fromkeys(st.kernels):
        idx = [i for i, k in enumerate(st.kernels) if k == name]
        reps = -(-64 // len(idx))  # at least 64 launches per replay
        g = st.graph(stream, idx, reps)
        for _ in range(max(2, warmup)):
            g.replay()
        _, gpu_s = timed(g.replay, max(5, steps // reps), stream)
        avg = gpu_s / (len(idx) * reps)
        alg = float(np.mean([st.launch_alg[i] for i in idx]))
        out[name] = {"launches": len(idx), "avg_launch_us": round(1e6 * avg, 3),
                     "alg_bytes_per_launch": round(alg), "GBps": round(alg / avg / 1e9, 1)}
    return out


def per_shape_timing(st, stream, n_ev):
    """Diagnostic: each launch bracketed by its own events (adds event overhead)."""
    import torch
    n = len(st.calls)
    starts = [[torch.cuda.Event(enable_timing=True) for _ in range(n)] for _ in range(n_ev)]
    ends = [[torch.cuda.Event(enable_timing=True) for _ in range(n)] for _ in range(n_ev)]
    for r in range(n_ev):
        for i in range(n):
            starts[r][i].record(stream)
            st.launch(i, stream.cuda_stream)
            ends[r][i].record(stream)
    torch.cuda.synchronize()
    dur = np.median(np.array([[starts[r][i].elapsed_time(ends[r][i]) * 1e-3 for i in range(n)]
                              for r in range(n_ev)]), axis=0)
    per = {}
    for i in range(n):
        key = st.labels[i]
        e = per.setdefault(key, {"count": 0, "us": [], "alg_bytes": st.launch_alg[i], "kernel": st.kernels[i]})
        e["count"] += 1
        e["us"].append(1e6 * dur[i])
    return {k: {"count": v["count"], "kernel": v["kernel"], "us_median": round(float(np.median(v["us"])), 2),
                "GBps": round(v["alg_bytes"] / (1e-6 * float(np.median(v["us"]))) / 1e9, 1)}
            for k, v in per.items()}


def dense_baseline(st, M, steps, dev, vbq_s):
    """Dense fp16 F.linear over the dequantized weights (context: the paper's
    FP16 comparison), eager launches."""
    import torch
    try:
        ws = []
        for parts, x, y, _ in st.mats:
            if parts[0][1] is None:
                ws.append(parts[0][0].dequant().half())
            else:  # row buckets: scatter each bucket's rows back into place
                w = torch.empty((y.shape[-1], parts[0][0].K), dtype=torch.float16, device=dev)
                for Wp, rows in parts:
                    w[rows.long()] = Wp.dequant().half()
                ws.append(w)
        torch.cuda.synchronize()
        xs = [m[1].view(M, -1) for m in st.mats]

        def dense_step():
            for w, xx in zip(ws, xs):
                torch.nn.functional.linear(xx, w)
        for _ in range(3):
            dense_step()
        torch.cuda.synchronize()
        nd = max(5, steps // 10)
        t0 = time.perf_counter()
        for _ in range(nd):
            dense_step()
        torch.cuda.synchronize()
        dense_s = (time.perf_counter() - t0) / nd
        del ws
        torch.cuda.empty_cache()
        return {"us_per_step": round(1e6 * dense_s, 1), "weight_bytes": 2 * st.total_w,
                "speedup_vbq": round(dense_s / vbq_s, 2),
                "note": "torch F.linear (fp16) over the dequantized weights, eager launches"}
    except Exception as e:
        log(f"dense baseline skipped: {e}")
        return None


def small_workload(cfg, args, dev, stream, flush):
    """A small decode workload (one GEMV, or the 131M-class step) timed hot
    (graph replays back to back, weights resident in the caches) and cold
    (each step after a 1 GiB flush write)."""
    wl, packed = prepare(cfg, args.workers)
    st = build_step(wl, packed, 1, dev)
    g = st.graph(stream)
    reps = -(-512 // len(st.calls))  # hot: the step repeated in one graph, >= 512 launches
    gr = st.graph(stream, reps=reps)
    for _ in range(max(5, args.warmup)):
        gr.replay()
    _, hot_gpu = timed(gr.replay, max(10, args.steps // reps), stream)
    hot_gpu /= reps
    cold = cold_steps(g.replay, max(20, min(100, args.steps)), flush, stream)
    out = {"name": wl.name, "launches": len(st.calls), "algorithmic_bytes": int(st.total_alg),
           "hot_us": round(1e6 * hot_gpu, 2),
           "hot_timing": f"HIP events around replays of a graph holding the step {reps} times in a row",
           "cold_us": cold,
           "hot_GBps": round(st.total_alg / hot_gpu / 1e9, 1),
           "cold_GBps": round(st.total_alg / (1e-6 * cold["median"]) / 1e9, 1),
           "kernels": sorted(set(st.kernels))}
    log(f"workload {cfg} ({wl.name}): hot {out['hot_us']} us, cold median {cold['median']} us")
    return out


def read_ceiling(buf, stream, reps=10):
    """The device's plain streaming-read rate (vbq_read_ceiling over a 1 GiB
    buffer), best over a few grid sizes."""
    import torch
    from paper_2607_02893_amd import vbq
    nbytes = buf.numel() * buf.element_size()
    best = None
    for blocks in (4096, 8192, 16384, 32768, 65536, 131072):
        sink = torch.empty(4 * blocks, dtype=torch.int32, device=buf.device)  # 4 words per block

        def rd():
            r = vbq.raw_read_ceiling(buf.data_ptr(), nbytes, blocks, sink.data_ptr(), stream.cuda_stream)
            if r != 0:
                raise vbq.VbqError(r, "vbq_read_ceiling")
        rd()
        _, s = timed(rd, reps, stream)
        gbs = nbytes / s / 1e9
        if best is None or gbs > best["GBps"]:
            best = {"GBps": round(gbs, 1), "blocks": blocks, "bytes": nbytes, "us": round(1e6 * s, 1),
                    "frac_of_peak": round(gbs / PEAK_HBM_GBS, 4),
                    "timing": f"HIP events around {reps} back-to-back reads of the buffer"}
    return best


if __name__ == "__main__":
    main()
