#!/usr/bin/env python3
"""Benchmark of the RKSC verify pass on one MI355X.

One step = one rksc_verify_forward call over the whole workload: every layer of
the multi-branch forward over the shared prefix cache, the fused
lm_head-entropy probe of every layer (one stream per exit window of layers)
and the exit rule (branches that exit stop being computed). Inputs (random-init bf16 weights, synthetic prefix K/V,
uniform tokens) are generated on the GPU and are resident in HBM before the
timed region, with the pre-tiled gate|up copy of every layer (rksc_tile_gate_up,
built once with the weights: a storage layout the library reads where the
gate|up projection runs on 128-row tiles); the workspace and outputs are
allocated once.

Prints ONE JSON line on stdout (progress goes to stderr):
  value        verify tokens/s = n_branches * branch_len / step time
  roofline     the dominant kernel class (most time per call; the gate|up
               projection at the default workload) against its roof, timed
               with HIP events recorded around its launches inside the timed
               steps, at every 4th layer for a per-layer class (the only
               events in that region: every recorded event opens a gap in
               the stream)
  kernels      every kernel class timed the same way in a separate breakdown
               pass before the timed region ("pass" says which)
  exit_histogram, live_layer_fraction   exit layers of the timed calls
  full_depth   the same workload with tau = 0 (no exit)
  tau_sweep    exit layers and call time at tau in {0.02, 0.05, 0.1, 0.2}
  prefill      the root forward (Eq. prefix_fwd) over the workload's prefix
  decode       batched greedy decode of 8 branches over the same prefix cache
               (suffix prefill, one-token steps, the CGEE gate), per step
               against the HBM bytes it must stream (weights, lm_head, prefix KV)
  kv_probe     the library's KV probe at 8 branches over the same prefix: the
               batched full recompute, the root forward and the batched suffix
               decode over the shared cache (min of 3 each), and its verdict
  tree         a 64-token search-tree node built once over the prefix cache
               (rksc_prefix_extend) against 8 children recomputing it, and the
               device ASKS gate over 8 branches
  asks_similarity  the pairwise ASKS similarity at B = 1, 8, 16, 32 (time only)
  cpu_baseline the float64 CPU oracle on a bounded sample of the workload

    python bench.py [--steps K] [--warmup W] [--workload 7b_single]
"""
import argparse
import ctypes
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "verify tokens/s at 7B shape w/ entropy exit; % peak HBM BW and MFMA util"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
FP32_PEAK_TFLOPS = 157.3       # MI355X fp32 vector / MFMA


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


class HipEvents:
    """hipEvent_t handles through the HIP runtime (events recorded by librksc on the call's stream)."""

    # Timing-only events: no system-scope fence on record. A fenced record writes
    # back and invalidates the caches, which opens a ~5 us gap in the stream and
    # leaves the next kernel cold.
    DISABLE_SYSTEM_FENCE = 0x20000000

    def __init__(self):
        self.lib = ctypes.CDLL("libamdhip64.so")
        self.lib.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.lib.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
        self.lib.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
        self.lib.hipEventDestroy.argtypes = [ctypes.c_void_p]

    def create(self, n, fenced=True):
        evs = []
        for _ in range(n):
            e = ctypes.c_void_p()
            if fenced:
                rc = self.lib.hipEventCreate(ctypes.byref(e))
            else:
                rc = self.lib.hipEventCreateWithFlags(ctypes.byref(e), self.DISABLE_SYSTEM_FENCE)
            if rc != 0:
                raise RuntimeError(f"hipEventCreate failed ({rc})")
            evs.append(e.value)
        return evs

    def elapsed_ms(self, a, b):
        ms = ctypes.c_float()
        rc = self.lib.hipEventElapsedTime(ctypes.byref(ms), ctypes.c_void_p(a), ctypes.c_void_p(b))
        if rc != 0:
            raise RuntimeError(f"hipEventElapsedTime failed ({rc})")
        return ms.value

    def destroy(self, evs):
        for e in evs:
            self.lib.hipEventDestroy(ctypes.c_void_p(e))


def kernel_work(shape, B_live, n, s, win=1):
    """Algorithmic bytes and flops per launch of each timed kernel class at B_live live branches
    (the lm_head stream serves an exit window of `win` layers: B_live * win columns)."""
    d, H, Hkv, hd, F, V = shape.d_model, shape.n_heads, shape.n_kv_heads, shape.head_dim, shape.d_ff, shape.vocab
    T = 2 if shape.dtype == "bf16" else 4
    M = B_live * s
    Nqkv = (H + 2 * Hkv) * hd

    def gemm(N, K, out_bytes):
        # What the method moves (not this library's split partials): the weights, the
        # activation once in the storage type, and the method's output of the step.
        return {"bytes": N * K * T + M * K * T + out_bytes, "flops": 2.0 * M * N * K}

    attn_flops = 4.0 * hd * H * B_live * (s * n + s * (s + 1) / 2)
    attn_bytes = 2 * Hkv * n * hd * T + B_live * 2 * Hkv * s * hd * T + 2 * M * H * hd * T
    return {
        # q, k, v in the storage type; the O and down outputs are added to the fp32 residual;
        # the gate|up step's output is the SwiGLU product [M, F]
        "qkv_proj": gemm(Nqkv, d, M * Nqkv * T), "o_proj": gemm(d, H * hd, M * d * 4),
        "gate_up_proj": gemm(2 * F, d, M * F * T), "down_proj": gemm(d, F, M * d * 4),
        "attention": {"bytes": attn_bytes, "flops": attn_flops},
        # W_lm once, the hi+lo bf16 normalised rows, the per-workgroup statistics
        "lm_head_entropy": {"bytes": V * d * T + B_live * win * d * 4, "flops": 2.0 * B_live * win * V * d},
    }


EVENT_SLOTS = {"qkv_proj": 0, "attention": 2, "o_proj": 4, "gate_up_proj": 6, "down_proj": 8, "lm_head_entropy": 10}

# Device code each timed kernel class is built from (hashed to tell whether a
# stored counter measurement still describes the current kernel).
KERNEL_SOURCES = {
    "lm_head_entropy": ["k_entropy.hip", "common.h"],
    "qkv_proj": ["k_gemm.hip", "common.h"], "o_proj": ["k_gemm.hip", "common.h"],
    "gate_up_proj": ["k_gemm.hip", "common.h"], "down_proj": ["k_gemm.hip", "common.h"],
    "attention": ["k_attn.hip", "common.h"],
}
# Name fragments of the device kernels behind each class in rocprofv3 output.
# At 7b_single: QKV uses 192-column tiles, gate|up 256, O and down 128.
KERNEL_NAMES = {"lm_head_entropy": "k_entropy_bf16", "attention": "k_attn_bf16", "qkv_proj": "k_gemm_dmaILi192",
                "o_proj": "k_gemm_dmaILi128", "gate_up_proj": "k_gemm_dmaILi256", "down_proj": "k_gemm_dmaILi128"}
# The decode measurement: the paper's B = 8 branches and t = 32 decode steps of
# its throughput table, after a 32-token suffix per branch.
DECODE_BRANCHES, DECODE_SUFFIX, DECODE_TOKENS = 8, 32, 32
TREE_NODE = 64   # tokens of a search-tree node (one reasoning step) in the tree-sharing measurement
COPY_BYTES = 1 << 29   # calibration copy: 512 MiB read + 512 MiB written


def source_digest(kernel):
    """SHA-256 of the kernel's sources with comments and whitespace runs removed, so
    that a stored counter record goes stale when the code changes, not its comments."""
    import hashlib
    import re
    h = hashlib.sha256()
    for fn in KERNEL_SOURCES[kernel]:
        with open(os.path.join(ROOT, "paper_2606_09937_amd", "csrc", fn), encoding="utf-8") as f:
            text = f.read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        h.update(" ".join(text.split()).encode())
    return h.hexdigest()


def traffic_record_path(kernel, workload):
    return os.path.join(ROOT, "profiles", f"{kernel}_{workload}_traffic.json")


def stored_traffic(kernel, workload):
    """HBM bytes per launch from the committed counter runs, or None if absent or stale."""
    path = traffic_record_path(kernel, workload)
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("source_sha256") != source_digest(kernel):
        return None
    return rec["hbm_bytes_per_launch"]


def _read_counter_csv(directory):
    """(kernel name, counter name, value) rows of every *counter_collection.csv under directory."""
    import csv
    rows = []
    for dp, _, files in os.walk(directory):
        for fn in files:
            if fn.endswith("counter_collection.csv"):
                with open(os.path.join(dp, fn)) as f:
                    for r in csv.DictReader(f):
                        rows.append((r["Kernel_Name"], r["Counter_Name"], float(r["Counter_Value"]), r["Dispatch_Id"]))
    return rows


def _per_dispatch(rows, name_part, counter):
    """Counter value per dispatch (summed over its per-agent/per-instance records)."""
    per = {}
    for kname, cname, val, disp in rows:
        if name_part in kname and cname == counter:
            per[disp] = per.get(disp, 0.0) + val
    return list(per.values())


def summarize_pmc(args):
    """Writes the traffic record and prints a text summary from four rocprofv3 --pmc runs."""
    import statistics
    fetch, write = _read_counter_csv(args.pmc_fetch), _read_counter_csv(args.pmc_write)
    cfetch, cwrite = _read_counter_csv(args.pmc_copy_fetch), _read_counter_csv(args.pmc_copy_write)
    kname = KERNEL_NAMES[args.kernel]
    k_f = _per_dispatch(fetch, kname, "FETCH_SIZE")
    k_w = _per_dispatch(write, kname, "WRITE_SIZE")
    c_f = _per_dispatch(cfetch, "neg_kernel", "FETCH_SIZE")
    c_w = _per_dispatch(cwrite, "neg_kernel", "WRITE_SIZE")
    if not (k_f and k_w and c_f and c_w):
        raise SystemExit(f"missing dispatches: kernel fetch {len(k_f)} write {len(k_w)}, "
                         f"copy fetch {len(c_f)} write {len(c_w)}")
    # bytes per counter unit, from the copy of known size (counters read KiB nominally)
    sf = COPY_BYTES / statistics.median(c_f)
    sw = COPY_BYTES / statistics.median(c_w)
    fb = statistics.median(k_f) * sf
    wb = statistics.median(k_w) * sw
    rec = {
        "kernel": args.kernel, "workload": args.workload, "device_kernel": kname,
        "fetch_bytes_per_launch": fb, "write_bytes_per_launch": wb, "hbm_bytes_per_launch": fb + wb,
        "fetch_scale_bytes_per_unit": sf, "write_scale_bytes_per_unit": sw,
        "dispatches": {"kernel_fetch": len(k_f), "kernel_write": len(k_w), "copy_fetch": len(c_f),
                       "copy_write": len(c_w)},
        "source_sha256": source_digest(args.kernel),
    }
    with open(traffic_record_path(args.kernel, args.workload), "w") as f:
        json.dump(rec, f, indent=1)
    print(f"{args.kernel} ({kname}) at {args.workload}: FETCH_SIZE median {statistics.median(k_f):.0f} over "
          f"{len(k_f)} dispatches, WRITE_SIZE median {statistics.median(k_w):.0f} over {len(k_w)}")
    print(f"copy calibration ({COPY_BYTES} B read + written): FETCH_SIZE {statistics.median(c_f):.0f}, "
          f"WRITE_SIZE {statistics.median(c_w):.0f} -> {sf:.1f} / {sw:.1f} bytes per counter unit")
    print(f"HBM traffic per launch: read {fb / 1e6:.1f} MB + write {wb / 1e6:.3f} MB = {(fb + wb) / 1e6:.1f} MB")


def summarize_mfma(args):
    """Prints the MFMA counters of a rocprofv3 --pmc MfmaUtil SQ_INSTS_VALU_MFMA_MOPS_BF16 run per
    projection class: MfmaUtil (MFMA-busy cycles over active cycles x SIMDs, %) and the bf16 MFMA
    flops issued (MOPS x 512) against the class's algorithmic flops (the hi/lo operand split issues
    two products per algorithmic one). Dispatches are assigned to classes by their issued flops."""
    import re
    import statistics

    import workloads
    rows = _read_counter_csv(args.pmc_mfma)
    per = {}
    for kname, cname, val, disp in rows:
        d = per.setdefault(disp, {"name": kname})
        d[cname] = d.get(cname, 0.0) + val
    wl = workloads.get(args.workload)
    shape = wl.model
    work = kernel_work(shape, wl.n_branches, wl.prefix_len, wl.branch_len, 1)
    classes = {c: work[c]["flops"] for c in PROJECTIONS}
    got = {c: [] for c in classes}
    other = {}
    for d in per.values():
        if "MfmaUtil" not in d or "SQ_INSTS_VALU_MFMA_MOPS_BF16" not in d:
            continue
        issued = d["SQ_INSTS_VALU_MFMA_MOPS_BF16"] * 512
        best = min(classes, key=lambda c: abs(issued / classes[c] - 2.0))
        if "k_gemm" in d["name"] and abs(issued / classes[best] - 2.0) < 0.1:
            got[best].append((d["MfmaUtil"], issued, d["name"]))
        else:
            m = re.search(r"(k_[a-z0-9_]+)", d["name"])
            other.setdefault(m.group(1) if m else d["name"][:40], []).append((d["MfmaUtil"], issued))
    print(f"MFMA counters at {wl.name} (M = {wl.n_branches * wl.branch_len} rows): per projection class")
    print(f"{'class':14s} {'launches':>8s} {'MfmaUtil %':>11s} {'issued GFLOP':>13s} {'algorithmic GFLOP':>18s}  kernel")
    for c, lst in got.items():
        if not lst:
            continue
        u = statistics.median(x[0] for x in lst)
        iss = statistics.median(x[1] for x in lst)
        print(f"{c:14s} {len(lst):8d} {u:11.1f} {iss / 1e9:13.1f} {classes[c] / 1e9:18.1f}  {lst[0][2][:70]}")
    for k, lst in sorted(other.items()):
        u = statistics.median(x[0] for x in lst)
        iss = statistics.median(x[1] for x in lst)
        print(f"{'(other)':14s} {len(lst):8d} {u:11.1f} {iss / 1e9:13.2f} {'':>18s}  {k}")


def summarize_stats(args):
    """Prints the per-kernel table of a rocprofv3 --stats run (kernel_stats.csv)."""
    import csv
    path = None
    for dp, _, files in os.walk(args.stats):
        for fn in files:
            if fn.endswith("kernel_stats.csv"):
                path = os.path.join(dp, fn)
    if path is None:
        raise SystemExit(f"no kernel_stats.csv under {args.stats}")
    with open(path) as f:
        rows = list(csv.DictReader(f))
    print(f"{'calls':>6} {'avg us':>9} {'min us':>9} {'max us':>9} {'total %':>8}  kernel")
    for r in rows:
        print(f"{int(r['Calls']):6d} {float(r['AverageNs']) / 1e3:9.2f} {float(r['MinNs']) / 1e3:9.2f} "
              f"{float(r['MaxNs']) / 1e3:9.2f} {float(r['Percentage']):8.2f}  {r['Name'][:110]}")


def copy_calibration():
    """One plain copy kernel (dst = -src, fp32) of COPY_BYTES, three times, for counter scaling."""
    import torch
    src = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(3):
        torch.neg(src, out=dst)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": COPY_BYTES, "copy_bytes_written": COPY_BYTES, "launches": 3}))


def cpu_model():
    """The host CPU's model name and the cores this process may run on."""
    name = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    name = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        avail = len(os.sched_getaffinity(0))
    except AttributeError:
        avail = os.cpu_count() or 1
    return name, avail


def blas_threads():
    from threadpoolctl import threadpool_info
    return max([i.get("num_threads", 1) for i in threadpool_info()] + [1])


def cpu_baseline(mw, kv, toks, wl, layers, branches=None):
    """Float64 oracle on the first `layers` layers (and the first `branches` branches) of the
    same workload; the time is scaled to all layers and all branches (branches are independent
    given the prefix, and every layer costs the same)."""
    import dataclasses

    import oracle

    shape = mw.shape
    B = wl.n_branches
    nb = B if branches is None else min(branches, B)
    sub = dataclasses.replace(shape, n_layers=layers)

    class Host:
        pass

    host = Host()
    host.embed = mw.embed.cpu()
    host.layers = [{k: v.cpu() for k, v in mw.layers[i].items() if k != "w_gate_up_tiled"} for i in range(layers)]
    host.final_norm = mw.final_norm.cpu()
    host.lm_head = mw.lm_head.cpu()
    pk, pv = kv.k[:layers].cpu(), kv.v[:layers].cpu()
    t_np = toks.cpu().numpy()[:nb]
    t0 = time.perf_counter()
    oracle.verify_forward(host, sub, pk, pv, t_np, wl.tau, wl.patience)
    dt = time.perf_counter() - t0
    scale = (shape.n_layers / layers) * (B / nb)
    per_step = dt * scale
    tokens = B * wl.branch_len
    exact = layers == shape.n_layers and nb == B
    return {
        "value": tokens / per_step, "unit": "tokens/s", "cores": blas_threads(), "kind": "oracle",
        "extrapolated": not exact,
        "sample": (f"float64 oracle verify pass over {'all' if layers == shape.n_layers else f'the first {layers} of'} "
                   f"{shape.n_layers} layers and {'all' if nb == B else f'{nb} of the'} {B} branch(es) of "
                   f"{wl.name} ({wl.branch_len} tokens each, {kv.k.shape[2]}-token prefix), {dt:.1f} s"
                   + ("" if exact else f"; time scaled by {scale:g} (layers x branches)")),
        "sample_seconds": dt,
    }


def cpu_single_thread_tiny(seed):
    """The oracle on the tiny workload (2 layers, 4 branches x 16 tokens over 64 prefix tokens)
    with BLAS limited to one thread: tokens/s."""
    import oracle
    import workloads
    from threadpoolctl import threadpool_limits

    wl = workloads.get("tiny")
    shape = wl.model
    mw = workloads.make_model(shape, seed=seed)
    kv = workloads.make_prefix_kv(shape, wl.prefix_len, seed=seed)
    toks = workloads.make_tokens(wl.n_branches * wl.branch_len, shape.vocab, seed=seed).reshape(
        wl.n_branches, wl.branch_len).numpy()
    with threadpool_limits(1):
        oracle.verify_forward(mw, shape, kv.k, kv.v, toks, wl.tau, wl.patience)   # warm
        reps, t0 = 0, time.perf_counter()
        while reps < 3 or time.perf_counter() - t0 < 1.0:
            oracle.verify_forward(mw, shape, kv.k, kv.v, toks, wl.tau, wl.patience)
            reps += 1
        dt = (time.perf_counter() - t0) / reps
    return {"workload": "tiny", "value": wl.n_branches * wl.branch_len / dt, "unit": "tokens/s", "cores": 1,
            "ms_per_call": dt * 1e3, "calls": reps}


def measure_decode(mw, kv, shape, n, args, hip, sp, stream, dev):
    """Batched decode over the prefix cache (Sec. 2.2; Eq. gen_conf, Eq. cgee_gate):
    DECODE_BRANCHES branches, a DECODE_SUFFIX-token suffix prefill, then greedy
    one-token steps (each feeds its argmax back) until DECODE_TOKENS tokens per
    branch are generated, then the Level-1 gate. The steps are timed with HIP
    events on `stream`; the solve time spans the suffix, the steps and the gate."""
    import torch

    import paper_2606_09937_amd as rk
    import workloads

    L = shape.n_layers
    Bd, sd, td = DECODE_BRANCHES, DECODE_SUFFIX, DECODE_TOKENS
    stoks = workloads.make_tokens(Bd * sd, shape.vocab, seed=args.seed, name="suffix",
                                  device=dev).reshape(Bd, sd).contiguous()
    dec = rk.Decoder(mw, kv.k, kv.v, Bd, sd, capacity=sd + td, device=dev)

    def run_decode(ev=None):
        dec.cache.struct.length = 0
        dec.suffix(stoks, stream)
        if ev:
            hip.lib.hipEventRecord(ctypes.c_void_p(ev[0]), sp)
        for _ in range(td - 1):
            dec.step(None, stream)
        if ev:
            hip.lib.hipEventRecord(ctypes.c_void_p(ev[1]), sp)
        return dec.gate(0.70, 0.06, stream)

    run_decode()
    torch.cuda.synchronize()
    k_d = max(1, min(args.steps, 3))
    a, b = hip.create(2)
    tot = []
    steps_ms = []
    for _ in range(k_d):
        m0, m1 = hip.create(2)
        hip.lib.hipEventRecord(ctypes.c_void_p(a), sp)
        fired, winner, p_mean, _ = run_decode((m0, m1))
        hip.lib.hipEventRecord(ctypes.c_void_p(b), sp)
        torch.cuda.synchronize()
        tot.append(hip.elapsed_ms(a, b))
        steps_ms.append(hip.elapsed_ms(m0, m1))
        hip.destroy([m0, m1])
    hip.destroy([a, b])
    d_, H_, Hkv_, hd_, F_ = shape.d_model, shape.n_heads, shape.n_kv_heads, shape.head_dim, shape.d_ff
    T_ = 2 if shape.dtype == "bf16" else 4
    P_ = d_ * (H_ + 2 * Hkv_) * hd_ + H_ * hd_ * d_ + 3 * d_ * F_
    step_bytes = T_ * (L * P_ + shape.vocab * d_ + L * 2 * Hkv_ * n * hd_)
    step_ms = float(sorted(steps_ms)[len(steps_ms) // 2]) / (td - 1)
    total_ms = float(sorted(tot)[len(tot) // 2])
    decode = {"n_branches": Bd, "suffix_len": sd, "tokens_per_branch": td, "prefix_len": n,
              "ms_per_solve": total_ms, "suffix_and_gate_ms": total_ms - step_ms * (td - 1),
              "ms_per_step": step_ms, "step_tokens_per_s": Bd / (step_ms / 1e3),
              "solve_tokens_per_s": Bd * td / (total_ms / 1e3),
              "step_algorithmic_bytes": step_bytes, "step_hbm_gbs": step_bytes / (step_ms / 1e3) / 1e9,
              "step_hbm_frac": step_bytes / (step_ms / 1e3) / 1e9 / HBM_PEAK_GBS,
              "gate": {"tau_conf": 0.70, "r_gap": 0.06, "fired": int(fired.item()),
                       "winner": int(winner.item()), "p_mean": [round(x, 4) for x in p_mean.tolist()]},
              "runs_timed": k_d}
    log(f"decode B={Bd} suffix={sd} tokens={td}: {total_ms:.2f} ms/solve, {step_ms:.3f} ms/step "
        f"({decode['step_hbm_gbs']:.0f} GB/s weight+KV stream), gate fired={decode['gate']['fired']}")
    del dec
    return decode


def measure_prefill(mw, shape, n, args, hip, sp, stream, dev):
    """Root forward (Eq. prefix_fwd) over n tokens: ms per call and algorithmic TFLOP/s."""
    import torch
    import paper_2606_09937_amd as rk
    import workloads
    L = shape.n_layers
    ptoks = workloads.make_tokens(n, shape.vocab, seed=args.seed, name="prefix", device=dev)
    pws = torch.empty(rk.rksc_prefill_workspace_size(shape, n), dtype=torch.uint8, device=dev)
    dt_kv = torch.bfloat16 if shape.dtype == "bf16" else torch.float32
    pk = torch.empty((L, shape.n_kv_heads, n, shape.head_dim), dtype=dt_kv, device=dev)
    pv = torch.empty_like(pk)
    hr = torch.empty((L, shape.d_model), dtype=torch.float32, device=dev)
    pstep = lambda: rk.rksc_prefill(mw, ptoks, pk, pv, hr, pws, stream)   # noqa: E731
    for _ in range(max(1, args.warmup)):
        pstep()
    torch.cuda.synchronize()
    k_p = max(1, min(args.steps, 10))
    a, b = hip.create(2)
    hip.lib.hipEventRecord(ctypes.c_void_p(a), sp)
    for _ in range(k_p):
        pstep()
    hip.lib.hipEventRecord(ctypes.c_void_p(b), sp)
    torch.cuda.synchronize()
    p_ms = hip.elapsed_ms(a, b) / k_p
    hip.destroy([a, b])
    d_, H_, Hkv_, hd_, F_ = shape.d_model, shape.n_heads, shape.n_kv_heads, shape.head_dim, shape.d_ff
    P_ = d_ * (H_ + 2 * Hkv_) * hd_ + H_ * hd_ * d_ + 3 * d_ * F_
    p_flops = L * (2.0 * n * P_ + 4.0 * hd_ * H_ * n * (n + 1) / 2)
    peak = BF16_PEAK_TFLOPS if shape.dtype == "bf16" else FP32_PEAK_TFLOPS
    prefill = {"n_prefix": n, "ms_per_call": p_ms, "tokens_per_s": n / (p_ms / 1e3), "calls_timed": k_p,
               "algorithmic_tflops": p_flops / (p_ms / 1e3) / 1e12,
               "mfma_frac": p_flops / (p_ms / 1e3) / 1e12 / peak}
    log(f"prefill n={n}: {p_ms:.3f} ms/call, {prefill['tokens_per_s']:.0f} tokens/s, "
        f"{prefill['algorithmic_tflops']:.1f} TFLOP/s algorithmic")
    del pws, pk, pv, hr
    return prefill


def measure_kv_probe(mw, shape, n, args, stream, dev):
    """The KV probe (Sec. 2.2) at the paper's cost-constants setting: B = 8 branches
    over the workload's prefix with a DECODE_SUFFIX-token suffix; the three paths
    are timed as the minimum of 3 runs each by the library's probe."""
    import paper_2606_09937_amd as rk
    import workloads

    Bd, sd = DECODE_BRANCHES, DECODE_SUFFIX
    ptoks = workloads.make_tokens(n, shape.vocab, seed=args.seed, name="prefix", device=dev)
    stoks = workloads.make_tokens(Bd * sd, shape.vocab, seed=args.seed, name="suffix",
                                  device=dev).reshape(Bd, sd).contiguous()
    probe = rk.KVProbe(3)
    share, t, _ = probe.decide(mw, ptoks, stoks, stream=stream)
    out = {"n_branches": Bd, "prefix_len": n, "suffix_len": sd, "reps": 3,
           "batch_full_ms": t[0], "prefix_fwd_ms": t[1], "sfx_kv_ms": t[2], "net_saved_ms": t[0] - t[1] - t[2],
           "share": share}
    log(f"kv probe B={Bd} n={n} s={sd}: full {t[0]:.1f} ms, prefix {t[1]:.1f} ms, suffix {t[2]:.1f} ms, "
        f"net saved {t[0] - t[1] - t[2]:.1f} ms, share={share}")
    return out


def measure_tree(mw, kv, shape, n, args, hip, sp, stream, dev):
    """Tree sharing and the ASKS gate at the workload's prefix: one search-tree node
    of TREE_NODE tokens built once over the root cache (rksc_prefix_extend: the root is
    read in place and only the node's entries are written), against
    its DECODE_BRANCHES children each recomputing the node's tokens over the root cache
    (one batched suffix pass); and the device ASKS gate over DECODE_BRANCHES rows."""
    import torch

    import paper_2606_09937_amd as rk
    import workloads

    m, Bd = TREE_NODE, DECODE_BRANCHES
    L = shape.n_layers
    node = workloads.make_tokens(m, shape.vocab, seed=args.seed, name="node", device=dev)
    dtype = torch.bfloat16 if shape.dtype == "bf16" else torch.float32
    ws = torch.empty(rk.rksc_prefix_extend_workspace_size(shape, n, m), dtype=torch.uint8, device=dev)
    ck = torch.empty((L, shape.n_kv_heads, m, shape.head_dim), dtype=dtype, device=dev)
    cv = torch.empty_like(ck)
    hn = torch.empty((L, shape.d_model), dtype=torch.float32, device=dev)
    dec = rk.Decoder(mw, kv.k, kv.v, Bd, m, capacity=m, device=dev)
    rows = node.repeat(Bd, 1).contiguous()

    def timed(fn, reps=3):
        fn()
        torch.cuda.synchronize()
        best = float("inf")
        for _ in range(reps):
            a, b = hip.create(2)
            hip.lib.hipEventRecord(ctypes.c_void_p(a), sp)
            fn()
            hip.lib.hipEventRecord(ctypes.c_void_p(b), sp)
            torch.cuda.synchronize()
            best = min(best, hip.elapsed_ms(a, b))
            hip.destroy([a, b])
        return best

    def unshared():
        dec.cache.struct.length = 0
        dec.suffix(rows, stream)

    t_ext = timed(lambda: rk.rksc_prefix_extend(mw, kv.k, kv.v, node, ck, cv, hn, ws, stream))
    t_all = timed(unshared)
    hid = workloads.make_hidden(L, Bd, shape.d_model, seed=args.seed, device=dev)
    t_gate = timed(lambda: rk.asks_gate(hid, hn, 1.5, 0.82, stream))
    out = {"parent_len": n, "node_tokens": m, "children": Bd, "extend_ms": t_ext,
           "children_recompute_ms": t_all, "asks_gate_us": t_gate * 1e3}
    log(f"tree: node of {m} tokens over {n}: extend {t_ext:.2f} ms once vs {t_all:.2f} ms for {Bd} children "
        f"recomputing it; ASKS gate {t_gate * 1e3:.1f} us")
    del dec, ws, ck, cv
    return out


def measure_asks(shape, args, hip, sp, stream, dev):
    """The ASKS pairwise similarity (Eq. asks_sim over all branch pairs) at the
    workload's layer count and width for the branch counts of the configs
    (1, 8, 16, 32): latency-bound, reported as time only."""
    import torch

    import paper_2606_09937_amd as rk
    import workloads

    L, d = shape.n_layers, shape.d_model
    out = {}
    for B in (1, 8, 16, 32):
        hid = workloads.make_hidden(L, B, d, seed=args.seed, device=dev)
        S = torch.empty((B, B), dtype=torch.float32, device=dev)
        rk.rksc_asks_similarity(hid, 1.5, S, stream)
        torch.cuda.synchronize()
        best = float("inf")
        for _ in range(5):
            a, b = hip.create(2)
            hip.lib.hipEventRecord(ctypes.c_void_p(a), sp)
            rk.rksc_asks_similarity(hid, 1.5, S, stream)
            hip.lib.hipEventRecord(ctypes.c_void_p(b), sp)
            torch.cuda.synchronize()
            best = min(best, hip.elapsed_ms(a, b))
            hip.destroy([a, b])
        out[str(B)] = {"us": best * 1e3, "bytes": 4 * L * B * d}
    log("asks similarity: " + ", ".join(f"B={k} {v['us']:.1f} us" for k, v in out.items()))
    return out


# The other configurations of the verify pass, each timed in the default run
# after the headline (one record each): the tree of thoughts, the large
# vocabulary, the long prefix and its one-token decode regime.
CONFIG_RECORDS = ("7b_tot", "7b_large_vocab", "10b_long", "10b_decode")
PROJECTIONS = ("qkv_proj", "o_proj", "gate_up_proj", "down_proj")


def class_roof(work, avg_us, dtype):
    """One kernel class against its binding roof: MFMA when its algorithmic intensity is
    above the bf16 ridge (2.5 PFLOP/s / 8 TB/s = 312 flop/B), else HBM."""
    sec = avg_us * 1e-6
    gbs = work["bytes"] / sec / 1e9
    tf = work["flops"] / sec / 1e12
    peak = BF16_PEAK_TFLOPS if dtype == "bf16" else FP32_PEAK_TFLOPS
    mfma = work["flops"] / work["bytes"] > BF16_PEAK_TFLOPS / HBM_PEAK_GBS * 1e3
    return {"avg_us": avg_us, "hbm_gbs": gbs, "hbm_frac": gbs / HBM_PEAK_GBS, "tflops": tf, "mfma_frac": tf / peak,
            "bound": "mfma" if mfma else "hbm", "frac": tf / peak if mfma else gbs / HBM_PEAK_GBS,
            "algorithmic_bytes": work["bytes"], "algorithmic_flops": work["flops"]}


def event_arrays(hip, L, k_steps, slots, stream_layers):
    """HIP events for k_steps profiled calls at the given per-layer slots (the lm_head slots only
    at the layers where the stream runs). Returns (events, per-call host arrays)."""
    per_step = 12 * L
    evs = hip.create(per_step * k_steps, fenced=False)
    ptrs = []
    for k in range(k_steps):
        arr = (ctypes.c_void_p * per_step)()
        for l in range(L):
            for sl in slots:
                if sl in (EVENT_SLOTS["lm_head_entropy"], EVENT_SLOTS["lm_head_entropy"] + 1) and \
                        l not in stream_layers:
                    continue
                arr[12 * l + sl] = evs[k * per_step + 12 * l + sl]
        ptrs.append(ctypes.cast(arr, ctypes.c_void_p))
        ptrs[-1]._keep = arr
    return evs, ptrs


def measure_workload(name, args, hip, dev):
    """One configuration of the verify pass: ms per call at its (tau, patience) and at tau = 0
    (full depth), each the median of `reps` calls timed with HIP events; the per-class kernel
    times from a profiled full-depth call; each class against its binding roof; and the
    projections' algorithmic MFMA fraction over their summed time."""
    import torch

    import paper_2606_09937_amd as rk
    import workloads

    wl = workloads.get(name)
    shape = wl.model
    B, n, s, L = wl.n_branches, wl.prefix_len, wl.branch_len, shape.n_layers
    t0 = time.perf_counter()
    mw = workloads.make_model(shape, seed=args.seed, device=dev)
    rk.tile_gate_up(mw)
    kv = workloads.make_prefix_kv(shape, n, seed=args.seed, device=dev)
    toks = workloads.make_tokens(B * s, shape.vocab, seed=args.seed, device=dev).reshape(B, s).contiguous()
    ws = torch.empty(rk.rksc_verify_workspace_size(shape, B, s, n), dtype=torch.uint8, device=dev)
    ent = torch.empty((L, B), dtype=torch.float32, device=dev)
    ex = torch.empty((B,), dtype=torch.int32, device=dev)
    torch.cuda.synchronize()
    lib = rk.load_library()
    w_struct, keep = rk._weights_struct(mw)
    kv_struct = rk.PrefixKV(n, rk._ptr(kv.k), rk._ptr(kv.v))
    stream = torch.cuda.current_stream()
    sp = ctypes.c_void_p(stream.cuda_stream)
    common = (ctypes.byref(w_struct), ctypes.byref(kv_struct), rk._ptr(toks), B, s)

    def call(tau, patience, events=None):
        if events is None:
            st = lib.rksc_verify_forward(*common, float(tau), int(patience), rk._ptr(ent), rk._ptr(ex), None,
                                         rk._ptr(ws), ws.numel(), sp)
        else:
            st = lib.rksc_verify_forward_profiled(*common, float(tau), int(patience), rk._ptr(ent), rk._ptr(ex),
                                                  None, rk._ptr(ws), ws.numel(), sp, events)
        if st != 0:
            raise RuntimeError(f"rksc_verify_forward failed at {name}: {rk.rksc_last_error()}")

    call(wl.tau, wl.patience)
    torch.cuda.synchronize()
    reps = 3

    def timed(tau, patience):
        out = []
        for _ in range(reps):
            a, b = hip.create(2)
            hip.lib.hipEventRecord(ctypes.c_void_p(a), sp)
            call(tau, patience)
            hip.lib.hipEventRecord(ctypes.c_void_p(b), sp)
            torch.cuda.synchronize()
            out.append(hip.elapsed_ms(a, b))
            hip.destroy([a, b])
        return sorted(out)[len(out) // 2]

    ms_tau = timed(wl.tau, wl.patience)
    exits = ex.cpu().tolist()
    ms_full = timed(0.0, 1)

    # Per-class times from one profiled full-depth call (every layer live).
    win = rk.rksc_verify_window(shape, B, s, n)
    stream_layers = [l for l in range(L) if l % win == win - 1 or l == L - 1]
    slots = sorted(set(v for s0 in EVENT_SLOTS.values() for v in (s0, s0 + 1)))
    evs, ptrs = event_arrays(hip, L, 1, slots, stream_layers)
    call(0.0, 1, ptrs[0])
    torch.cuda.synchronize()
    work = kernel_work(shape, B, n, s, win)
    kernels = {}
    for cls, slot in EVENT_SLOTS.items():
        ls = stream_layers if cls == "lm_head_entropy" else range(L)
        d = [hip.elapsed_ms(evs[12 * l + slot], evs[12 * l + slot + 1]) for l in ls]
        rec = class_roof(work[cls], sum(d) / len(d) * 1e3, shape.dtype)
        rec["launches_per_call"] = len(d)
        rec["us_per_call"] = sum(d) * 1e3
        kernels[cls] = rec
    hip.destroy(evs)
    g_us = sum(kernels[c]["us_per_call"] for c in PROJECTIONS)
    g_flops = sum(work[c]["flops"] * kernels[c]["launches_per_call"] for c in PROJECTIONS)
    peak = BF16_PEAK_TFLOPS if shape.dtype == "bf16" else FP32_PEAK_TFLOPS
    dom = max(kernels, key=lambda k: kernels[k]["us_per_call"])
    rec = {
        "workload": name, "description": wl.description, "n_branches": B, "prefix_len": n, "branch_len": s,
        "layers": L, "tau": wl.tau, "patience": wl.patience, "exit_window": win,
        "ms_per_call": ms_tau, "tokens_per_s": B * s / (ms_tau / 1e3), "exit_layers": exits,
        "full_depth": {"ms_per_call": ms_full, "tokens_per_s": B * s / (ms_full / 1e3)},
        "calls_timed": reps,
        "kernels": kernels,
        "dominant": dom,
        "roofline": {"kernel": dom, "bound": kernels[dom]["bound"], "frac": kernels[dom]["frac"]},
        "projections": {"us_per_call": g_us, "algorithmic_tflops": g_flops / (g_us * 1e-6) / 1e12,
                        "mfma_frac": g_flops / (g_us * 1e-6) / 1e12 / peak},
    }
    log(f"{name}: {ms_tau:.2f} ms/call ({rec['tokens_per_s']:.0f} tokens/s, exits {sorted(set(exits))}), full depth "
        f"{ms_full:.2f} ms; projections {rec['projections']['mfma_frac']:.3f} of bf16 peak, attention "
        f"{kernels['attention']['avg_us']:.0f} us/layer ({kernels['attention']['bound']} "
        f"{kernels['attention']['frac']:.3f}), lm_head {kernels['lm_head_entropy']['hbm_frac']:.3f} of HBM "
        f"[{time.perf_counter() - t0:.1f} s]")
    cpu = None
    if args.cpu_extrapolate:
        cpu = cpu_baseline(mw, kv, toks, wl, min(2, L), branches=2)
        log(f"{name}: cpu oracle {cpu['value']:.4f} tokens/s extrapolated ({cpu['sample_seconds']:.1f} s sample)")
    rec["cpu_baseline"] = cpu
    del mw, kv, toks, ws, ent, ex, keep
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return rec


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="7b_single")
    ap.add_argument("--tau", type=float, default=None)
    ap.add_argument("--patience", type=int, default=None)
    ap.add_argument("--seed", type=int, default=42)
    ap.add_argument("--cpu-layers", type=int, default=0,
                    help="layers in the oracle's sample (0: all layers, the whole verify pass)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the records of the other configurations (7b_tot, 7b_large_vocab, 10b_long, 10b_decode)")
    ap.add_argument("--configs", default=",".join(CONFIG_RECORDS),
                    help="comma-separated configurations to record after the headline")
    ap.add_argument("--no-cpu-extrapolate", dest="cpu_extrapolate", action="store_false",
                    help="skip the oracle's 2-branch, 2-layer samples of the other configurations")
    ap.add_argument("--no-full-depth", action="store_true")
    ap.add_argument("--no-tau-sweep", action="store_true")
    ap.add_argument("--no-prefill", action="store_true", help="skip the root-forward (prefill) timing")
    ap.add_argument("--no-decode", action="store_true", help="skip the batched-decode timing")
    ap.add_argument("--no-probe", action="store_true", help="skip the KV probe timing")
    ap.add_argument("--no-tree", action="store_true",
                    help="skip the tree-sharing, ASKS-gate and ASKS-similarity timings")
    ap.add_argument("--decode-only", action="store_true",
                    help="time only the batched decode (for a kernel trace of it) and print its JSON")
    ap.add_argument("--prefill-only", action="store_true",
                    help="time only the root forward (for a kernel trace of it) and print its JSON")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run the plain copy kernel used to scale HBM counters")
    ap.add_argument("--summarize-stats", dest="stats", metavar="DIR",
                    help="print the kernel table of a rocprofv3 --stats output directory and exit")
    ap.add_argument("--summarize-pmc", action="store_true",
                    help="write profiles/<kernel>_<workload>_traffic.json from four --pmc output directories")
    ap.add_argument("--kernel", default="lm_head_entropy")
    ap.add_argument("--pmc-fetch")
    ap.add_argument("--pmc-write")
    ap.add_argument("--pmc-copy-fetch")
    ap.add_argument("--pmc-copy-write")
    ap.add_argument("--summarize-mfma", dest="pmc_mfma", metavar="DIR",
                    help="print the per-class MFMA counters of a rocprofv3 --pmc MfmaUtil "
                         "SQ_INSTS_VALU_MFMA_MOPS_BF16 output directory (for --workload) and exit")
    args = ap.parse_args()
    if args.stats:
        return summarize_stats(args)
    if args.summarize_pmc:
        return summarize_pmc(args)
    if args.pmc_mfma:
        return summarize_mfma(args)

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: the verify pass runs on a single MI355X (no multi-GPU path); "
              "run it with --gpus 1", file=sys.stderr)
        sys.exit(2)

    if args.copy_calibration:
        return copy_calibration()

    import torch

    import paper_2606_09937_amd as rk
    import workloads

    wl = workloads.get(args.workload)
    if args.tau is not None or args.patience is not None:
        wl = wl.with_(tau=wl.tau if args.tau is None else args.tau,
                      patience=wl.patience if args.patience is None else args.patience)
    shape = wl.model
    B, n, s, L = wl.n_branches, wl.prefix_len, wl.branch_len, shape.n_layers
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)

    log(f"workload {wl.name}: {wl.description}; generating inputs on {torch.cuda.get_device_name(0)}")
    t0 = time.perf_counter()
    mw = workloads.make_model(shape, seed=args.seed, device=dev)
    tiled = rk.tile_gate_up(mw)
    kv = workloads.make_prefix_kv(shape, n, seed=args.seed, device=dev)
    toks = workloads.make_tokens(B * s, shape.vocab, seed=args.seed, device=dev).reshape(B, s).contiguous()
    ws = torch.empty(rk.rksc_verify_workspace_size(shape, B, s, n), dtype=torch.uint8, device=dev)
    ent = torch.empty((L, B), dtype=torch.float32, device=dev)
    ex = torch.empty((B,), dtype=torch.int32, device=dev)
    torch.cuda.synchronize()
    log(f"inputs ready in {time.perf_counter() - t0:.1f} s; workspace {ws.numel() / 2**20:.1f} MiB")

    lib = rk.load_library()
    w_struct, keep = rk._weights_struct(mw)
    kv_struct = rk.PrefixKV(n, rk._ptr(kv.k), rk._ptr(kv.v))
    stream = torch.cuda.current_stream()
    sp = ctypes.c_void_p(stream.cuda_stream)
    common = (ctypes.byref(w_struct), ctypes.byref(kv_struct), rk._ptr(toks), B, s)

    def step(tau, patience, events=None):
        if events is None:
            st = lib.rksc_verify_forward(*common, float(tau), int(patience), rk._ptr(ent), rk._ptr(ex), None,
                                         rk._ptr(ws), ws.numel(), sp)
        else:
            st = lib.rksc_verify_forward_profiled(*common, float(tau), int(patience), rk._ptr(ent), rk._ptr(ex),
                                                  None, rk._ptr(ws), ws.numel(), sp, events)
        if st != 0:
            raise RuntimeError(f"rksc_verify_forward failed: {rk.rksc_last_error()}")

    if args.prefill_only:
        hip = HipEvents()
        hip.lib.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        prefill = measure_prefill(mw, shape, n, args, hip, sp, stream, dev)
        print(json.dumps({"metric": "root forward (prefill) at 7B shape", "unit": "tokens/s",
                          "value": prefill["tokens_per_s"], "dtype": shape.dtype, "data": "synthetic",
                          "config": {"workload": wl.name, "prefix_len": n}, "prefill": prefill}), flush=True)
        return

    if args.decode_only:
        hip = HipEvents()
        hip.lib.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        decode = measure_decode(mw, kv, shape, n, args, hip, sp, stream, dev)
        print(json.dumps({"metric": "batched decode (8 branches, greedy) at 7B shape", "unit": "tokens/s",
                          "value": decode["step_tokens_per_s"], "dtype": shape.dtype, "data": "synthetic",
                          "config": {"workload": wl.name, "prefix_len": n}, "decode": decode}), flush=True)
        return

    lib.rksc_verify_forward_profiled.restype = ctypes.c_int32
    lib.rksc_verify_forward_profiled.argtypes = list(lib.rksc_verify_forward.argtypes) + [ctypes.c_void_p]

    for i in range(args.warmup):
        step(wl.tau, wl.patience)
    torch.cuda.synchronize()
    log(f"warmup done ({args.warmup} steps)")

    hip = HipEvents()
    hip.lib.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
    per_step = 12 * L
    tokens = B * s

    def profiled_steps(k_steps, slots, layer_stride=1):
        """Event arrays for k_steps calls with timing events at the given per-layer
        slots, at every layer_stride-th layer (layer 0, layer_stride, ...)."""
        evs = hip.create(per_step * k_steps, fenced=False)
        arrays = []
        for k in range(k_steps):
            arr = (ctypes.c_void_p * per_step)()
            for l in range(0, L, layer_stride):
                for sl in slots:
                    if sl in (EVENT_SLOTS["lm_head_entropy"], EVENT_SLOTS["lm_head_entropy"] + 1) and \
                            l not in stream_layers:
                        continue   # no stream at this layer: the library records nothing there
                    arr[12 * l + sl] = evs[k * per_step + 12 * l + sl]
            arrays.append(arr)
        ptrs = [ctypes.cast(a, ctypes.c_void_p) for a in arrays]
        return evs, ptrs

    # The probe's lm_head stream runs once per exit window, at the window's last layer.
    win = rk.rksc_verify_window(shape, B, s, n)
    stream_layers = [l for l in range(L) if l % win == win - 1 or l == L - 1]

    def durations(evs, k_steps, slot, layers, layer_stride=1):
        ls = ([l for l in stream_layers if l < layers] if slot == EVENT_SLOTS["lm_head_entropy"]
              else range(0, layers, layer_stride))
        return [hip.elapsed_ms(evs[k * per_step + 12 * l + slot], evs[k * per_step + 12 * l + slot + 1])
                for k in range(k_steps) for l in ls]

    # 1) Breakdown pass (untimed): events around every kernel class. Each recorded
    #    event opens a few-microsecond gap in the stream, so these steps are not
    #    the ones the headline is measured on.
    kb_steps = max(2, min(args.steps, 5))
    evs_b, ptrs_b = profiled_steps(kb_steps, sorted(set(v for s0 in EVENT_SLOTS.values() for v in (s0, s0 + 1))))
    for k in range(kb_steps):
        step(wl.tau, wl.patience, ptrs_b[k])
    torch.cuda.synchronize()
    exits = ex.cpu().tolist()
    live_layers = max(exits)   # layers past every branch's exit run kernels that return at once
    kernels = {}
    for name, slot in EVENT_SLOTS.items():
        d = durations(evs_b, kb_steps, slot, live_layers)
        kernels[name] = {"avg_us": sum(d) / len(d) * 1e3, "launches_timed": len(d), "pass": "breakdown"}
    hip.destroy(evs_b)
    live_per_layer = [sum(1 for e in exits if e >= l + 1) for l in range(L)]
    mean_live = sum(live_per_layer[:live_layers]) / live_layers
    work = kernel_work(shape, max(1, round(mean_live)), n, s, win)
    # Dominant class: the most time per call (per-launch time x launches per call).
    launches = {k: (len([l for l in stream_layers if l < live_layers]) if k == "lm_head_entropy" else live_layers)
                for k in kernels}
    shares = {k: v["avg_us"] * launches[k] for k, v in kernels.items()}
    for k, v in kernels.items():
        v["launches_per_call"] = launches[k]
        v["us_per_call"] = shares[k]
    dom = max(shares, key=shares.get)

    # 2) Timed region: K calls, events only around the dominant kernel class, and
    #    (for a per-layer class) only at every 4th layer: each recorded pair
    #    stretches the call by ~2 us, and the layers' launches of a class are the
    #    same work, so 8 of 32 per call time it as well at a quarter of the cost.
    stride_t = 1 if dom == "lm_head_entropy" or L < 16 else 4
    evs_t, ptrs_t = profiled_steps(args.steps, [EVENT_SLOTS[dom], EVENT_SLOTS[dom] + 1], stride_t)
    start, stop = hip.create(2)
    torch.cuda.synchronize()
    hip.lib.hipEventRecord(ctypes.c_void_p(start), sp)
    t_wall = time.perf_counter()
    for k in range(args.steps):
        step(wl.tau, wl.patience, ptrs_t[k])
    hip.lib.hipEventRecord(ctypes.c_void_p(stop), sp)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_wall
    total_ms = hip.elapsed_ms(start, stop)
    ms_per_step = total_ms / args.steps
    value = tokens / (ms_per_step / 1e3)
    log(f"timed {args.steps} steps: {ms_per_step:.3f} ms/step (wall {wall / args.steps * 1e3:.3f} ms), "
        f"{value:.1f} tokens/s, exit layers {exits}")
    d = durations(evs_t, args.steps, EVENT_SLOTS[dom], live_layers, stride_t)
    kernels[dom].update({"avg_us": sum(d) / len(d) * 1e3, "launches_timed": len(d), "pass": "timed"})
    hip.destroy(evs_t + [start, stop])

    for name, rec in kernels.items():
        wk = work[name]
        sec = rec["avg_us"] * 1e-6
        rec["hbm_gbs"] = wk["bytes"] / sec / 1e9
        rec["tflops"] = wk["flops"] / sec / 1e12
        rec["hbm_frac"] = rec["hbm_gbs"] / HBM_PEAK_GBS
        peak = BF16_PEAK_TFLOPS if shape.dtype == "bf16" else FP32_PEAK_TFLOPS
        rec["mfma_frac"] = rec["tflops"] / peak
        rec["algorithmic_bytes"] = wk["bytes"]
        rec["algorithmic_flops"] = wk["flops"]
        # HBM bytes per launch from the committed rocprofv3 counter passes, where taken
        traffic = stored_traffic(name, wl.name)
        if traffic is not None:
            rec["hbm_traffic_bytes"] = traffic
            rec["hbm_traffic_gbs"] = traffic / sec / 1e9
    dk = kernels[dom]
    # Compute-bound when the class's arithmetic intensity is above the bf16 ridge
    # (2.5 PFLOP/s / 8 TB/s = 312 flop/B): the projections at many rows, and the
    # shared-prefix attention at long prefixes with many query rows.
    gemm_like = work[dom]["flops"] / work[dom]["bytes"] > BF16_PEAK_TFLOPS / HBM_PEAK_GBS * 1e3
    roofline = {
        "kernel": dom,
        "bound": "mfma" if gemm_like else "hbm",
        "achieved": dk["tflops"] if gemm_like else dk["hbm_gbs"],
        "peak": BF16_PEAK_TFLOPS if gemm_like else HBM_PEAK_GBS,
        "unit": "TFLOP/s" if gemm_like else "GB/s",
        "traffic": stored_traffic(dom, wl.name),
        "avg_launch_us": dk["avg_us"],
        "algorithmic_bytes_per_launch": work[dom]["bytes"],
    }
    roofline["frac"] = roofline["achieved"] / roofline["peak"]
    exit_hist = {str(l): exits.count(l) for l in sorted(set(exits))}
    live_fraction = sum(min(e, L) for e in exits) / (L * B)

    full_depth = None
    if not args.no_full_depth:
        for _ in range(max(1, args.warmup)):
            step(0.0, 1)
        torch.cuda.synchronize()
        a, b = hip.create(2)
        hip.lib.hipEventRecord(ctypes.c_void_p(a), sp)
        for _ in range(args.steps):
            step(0.0, 1)
        hip.lib.hipEventRecord(ctypes.c_void_p(b), sp)
        torch.cuda.synchronize()
        fd_ms = hip.elapsed_ms(a, b) / args.steps
        hip.destroy([a, b])
        full_depth = {"tau": 0.0, "ms_per_step": fd_ms, "value": tokens / (fd_ms / 1e3), "unit": "tokens/s"}
        log(f"full depth (tau=0): {fd_ms:.3f} ms/step, {full_depth['value']:.1f} tokens/s")

    # Functional sweep of the exit threshold (same inputs): random-init weights
    # rarely stabilise within tau = 0.02, so larger taus show the exit path at work.
    tau_sweep = None
    if not args.no_tau_sweep:
        tau_sweep = []
        for tau in (0.02, 0.05, 0.1, 0.2):
            step(tau, wl.patience)
            torch.cuda.synchronize()
            a, b = hip.create(2)
            hip.lib.hipEventRecord(ctypes.c_void_p(a), sp)
            for _ in range(3):
                step(tau, wl.patience)
            hip.lib.hipEventRecord(ctypes.c_void_p(b), sp)
            torch.cuda.synchronize()
            t_ms = hip.elapsed_ms(a, b) / 3
            hip.destroy([a, b])
            ex_t = ex.cpu().tolist()
            tau_sweep.append({"tau": tau, "patience": wl.patience, "exit_layers": ex_t, "ms_per_step": t_ms,
                              "value": tokens / (t_ms / 1e3)})
            log(f"tau {tau}: exit layers {ex_t}, {t_ms:.3f} ms/step")

    # Root forward over the same prefix length (Eq. prefix_fwd): the step before
    # the verify pass, which writes the cache the verify pass reads.
    prefill = None
    if not args.no_prefill:
        prefill = measure_prefill(mw, shape, n, args, hip, sp, stream, dev)

    decode = None if args.no_decode else measure_decode(mw, kv, shape, n, args, hip, sp, stream, dev)
    kv_probe = None if args.no_probe else measure_kv_probe(mw, shape, n, args, stream, dev)
    tree = None if args.no_tree else measure_tree(mw, kv, shape, n, args, hip, sp, stream, dev)
    asks = None if args.no_tree else measure_asks(shape, args, hip, sp, stream, dev)

    cpu = None
    if not args.no_cpu_baseline:
        cpu_layers = L if args.cpu_layers <= 0 else min(args.cpu_layers, L)
        log(f"cpu baseline: oracle on {cpu_layers} layer(s)")
        cpu = cpu_baseline(mw, kv, toks, wl, cpu_layers)
        name_cpu, avail = cpu_model()
        cpu["cpu_model"] = name_cpu
        cpu["cores_available"] = avail
        cpu["single_thread_tiny"] = cpu_single_thread_tiny(args.seed)
        log(f"cpu baseline: {cpu['value']:.3f} tokens/s on {cpu['cores']} threads ({name_cpu}, {avail} cores "
            f"available); tiny on one thread {cpu['single_thread_tiny']['value']:.0f} tokens/s")

    # The other configurations, one record each (their models replace the headline's in HBM).
    configs = None
    if not args.no_configs and args.configs:
        del mw, kv, toks, ws, keep, w_struct
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        configs = {}
        for cname in [c for c in args.configs.split(",") if c]:
            configs[cname] = measure_workload(cname, args, hip, dev)
        if cpu is not None:
            cpu["extrapolated_configs"] = {k: v["cpu_baseline"] for k, v in configs.items() if v["cpu_baseline"]}
            for v in configs.values():
                v.pop("cpu_baseline", None)

    out = {
        "metric": METRIC,
        "value": value,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": shape.dtype,
        "data": "synthetic: random-init weights N(0,0.02^2), synthetic prefix K/V, uniform tokens (seeded)",
        "config": {
            "workload": wl.name,
            "description": wl.description,
            "layers": L, "d_model": shape.d_model, "heads": shape.n_heads, "kv_heads": shape.n_kv_heads,
            "head_dim": shape.head_dim, "d_ff": shape.d_ff, "vocab": shape.vocab,
            "n_branches": B, "prefix_len": n, "branch_len": s, "tau": wl.tau, "patience": wl.patience,
            "exit_layers": exits, "parallelism": "single GPU", "gate_up_tiled": tiled,
        },
        "roofline": roofline,
        "exit_histogram": exit_hist,
        "live_layer_fraction": live_fraction,
        "kernels": kernels,
        "full_depth": full_depth,
        "tau_sweep": tau_sweep,
        "prefill": prefill,
        "decode": decode,
        "kv_probe": kv_probe,
        "tree": tree,
        "asks_similarity": asks,
        "cpu_baseline": cpu,
        "configs": configs,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
