"""Benchmark of one target-model tree-verification step on one MI355X.

A step is the whole hot path on one batch: tree_verify_attention (every
draft-tree node over its paged prefix plus its root path), tree_argmax_accept
(vocabulary argmax, greedy longest accepted path, bonus token) and
kv_compact_accepted (accepted rows into the cache), all through the C ABI on
one HIP stream. Inputs are resident in HBM before timing starts; consecutive
steps rotate over several copies of the inputs (more than 1 GB apart) so no
step finds its data in the 256 MB Infinity Cache.

Prints ONE JSON line. `value` is verified tree-tokens per second (tree nodes
verified per step / wall time per step; B * N, or the real nodes of a ragged
verification-fusion batch). `roofline` describes the
kernel call that takes the most time; `roofline_attention` the attention
call. `cpu_baseline` times the fp64 CPU oracle on a bounded sample.
"""
from __future__ import annotations

import argparse
import hashlib
import glob
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0
METRIC = "verified tree-tokens/sec + achieved HBM GB/s (% of peak), 8B-shaped, 1 GPU"


def source_digest() -> str:
    h = hashlib.sha256()
    for f in sorted(glob.glob(os.path.join(ROOT, "paper_2602_21224_amd", "csrc", "*"))):
        with open(f, "rb") as fh:
            h.update(os.path.basename(f).encode())
            h.update(fh.read())
    return h.hexdigest()[:16]


def real_nodes(w) -> np.ndarray:
    """Nodes per sequence that the step verifies (all N unless the batch is ragged)."""
    if w.num_nodes is None:
        return np.full(w.B, w.N, dtype=np.int64)
    return np.clip(w.num_nodes.astype(np.int64), 0, w.N)


def algorithmic(w):
    """Bytes (and FLOP) the method itself must move (and do) per call. Padding
    nodes of a ragged batch are not counted: only real nodes are verified."""
    from paper_2602_21224_amd.workloads import tree_depths
    L = w.kv_len.astype(np.int64)
    nn = real_nodes(w)
    R = int(nn.sum())
    live = nn > 0                                             # sequences with work
    row = w.Hkv * w.D * 2                                     # one K or V row, bf16
    anc = sum(int((tree_depths(w.parent[b][:nn[b]]) + 1).sum()) for b in range(w.B) if nn[b])
    pages_used = int(sum((int(l) + w.P - 1) // w.P for l in L[live]))
    attn_bytes = (int(L[live].sum()) * row * 2                # prefix K + V
                  + R * row * 2                               # tree K + V
                  + 2 * R * w.Hq * w.D * 2                    # q in, out
                  + R * w.Hq * 4                              # lse out
                  + pages_used * 4 + R * 4 + w.B * 4)         # page ids, parent, kv_len
    attn_flop = 4 * w.Hq * w.D * int((nn * L).sum()) + 4 * w.Hq * w.D * anc
    accept_bytes = R * w.V * 4 + 3 * R * 4 + R * 4 + 2 * w.B * 4
    if w.num_nodes is not None:
        attn_bytes += w.B * 4                                 # node counts
        accept_bytes += w.B * 4
    return attn_bytes, attn_flop, accept_bytes


def compact_bytes(w, accept_len):
    return 2 * int(accept_len.sum()) * w.Hkv * w.D * 2 * 2    # K and V rows, read + write


def warm_up(step, n_steps: int, min_seconds: float, torch):
    """Run the W requested warm-up steps, then more until min_seconds have
    passed (a short warm-up leaves the GPU below its sustained clocks); returns
    the number of steps run. None of them is timed."""
    t0 = time.perf_counter()
    i = 0
    while i < n_steps:
        step(i)
        i += 1
    torch.cuda.synchronize()
    while time.perf_counter() - t0 < min_seconds:
        for _ in range(8):
            step(i)
            i += 1
        torch.cuda.synchronize()
    return i


def pct(a, q):
    return round(float(np.percentile(a, q)) * 1e6, 2)


class TimingEvents:
    """HIP events used for timing only, created with hipEventDisableSystemFence:
    a default event makes a system-scope release (cache write-back) when it is
    recorded, which costs the stream several microseconds per event and is
    counted inside the intervals it brackets. Uses the HIP runtime that torch
    has loaded."""
    FLAGS = 0x20000000       # hipEventDisableSystemFence

    def __init__(self):
        import ctypes
        path = None
        with open("/proc/self/maps") as fh:
            for line in fh:
                if "libamdhip64" in line:
                    path = line.split()[-1]
                    break
        if path is None:
            raise RuntimeError("the HIP runtime is not loaded")
        self.ct = ctypes
        self.hip = ctypes.CDLL(path)
        self.hip.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
        self.hip.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        self.hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                                 ctypes.c_void_p]
        self.hip.hipEventDestroy.argtypes = [ctypes.c_void_p]

    def create(self):
        e = self.ct.c_void_p()
        if self.hip.hipEventCreateWithFlags(self.ct.byref(e), self.FLAGS) != 0:
            raise RuntimeError("hipEventCreateWithFlags failed")
        return e

    def record(self, e, stream):
        if self.hip.hipEventRecord(e, self.ct.c_void_p(stream.cuda_stream)) != 0:
            raise RuntimeError("hipEventRecord failed")

    def seconds(self, a, b) -> float:
        ms = self.ct.c_float()
        if self.hip.hipEventElapsedTime(self.ct.byref(ms), a, b) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return ms.value * 1e-3

    def destroy(self, e):
        self.hip.hipEventDestroy(e)


def load_traffic(kernel: str, workload: str):
    """HBM bytes per launch from committed rocprofv3 counter runs, if they were
    taken on the current kernel sources; else None."""
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel}_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        t = json.load(f)
    if t.get("source_digest") != source_digest():
        return None
    return t.get("hbm_bytes_per_launch")


CALL_KERNELS = {
    "tree_verify_attention": ("tree_attention_kernel", "tree_attention_merge_kernel"),
    "tree_argmax_accept": ("argmax_segments_kernel", "accept_kernel"),
    "kv_compact_accepted": ("kv_compact_kernel",),
    "tree_build": ("tb_rows_kernel", "tb_expand_kernel", "tb_select_kernel", "tb_prune_kernel"),
    "tree_lm_head_argmax_accept": ("lm_keys_clear_kernel", "lm_head_argmax_kernel", "accept_kernel"),
}


def _counter_means(run_dir: str, counter: str):
    """Mean value per dispatch of one rocprofv3 counter, by kernel base name."""
    import csv
    files = glob.glob(os.path.join(run_dir, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise SystemExit(f"no counter_collection.csv under {run_dir}")
    vals = {}
    for fn in files:
        with open(fn) as fh:
            for r in csv.DictReader(fh):
                if r["Counter_Name"] != counter:
                    continue
                name = r["Kernel_Name"].replace("(anonymous namespace)", "")
                base = name.split("(")[0].split("<")[0].split("::")[-1].split()[-1]
                vals.setdefault(base, []).append(float(r["Counter_Value"]))
    return vals


def write_traffic(workload: str, fetch_dir: str, write_dir: str, copy_fetch_dir: str,
                  copy_write_dir: str):
    """Turn rocprofv3 FETCH_SIZE / WRITE_SIZE runs (KiB per dispatch) of this
    benchmark and of --copy-calibration into HBM bytes per call, scaled by what
    the same counters read for a device copy of known size, and store them under
    profiles/ with the digest of the kernel sources they were taken on."""
    cf = _counter_means(copy_fetch_dir, "FETCH_SIZE")["__amd_rocclr_copyBuffer"]
    cw = _counter_means(copy_write_dir, "WRITE_SIZE")["__amd_rocclr_copyBuffer"]
    copy_kib = float(1 << 30) / 1024.0
    fetch_scale = copy_kib / max(cf)
    write_scale = copy_kib / max(cw)
    fv = _counter_means(fetch_dir, "FETCH_SIZE")
    wv = _counter_means(write_dir, "WRITE_SIZE")
    for call, kernels in CALL_KERNELS.items():
        per = {}
        total = 0.0
        calls = len(fv.get(kernels[0], []))          # the first kernel runs once per call
        for k in kernels:
            if k not in fv or k not in wv or calls == 0:
                continue
            # bytes per call: a kernel may run several times per call
            fb = np.sum(fv[k]) / calls * 1024.0 * fetch_scale
            wb = np.sum(wv[k]) / calls * 1024.0 * write_scale
            per[k] = {"fetch_bytes": int(round(fb)), "write_bytes": int(round(wb)),
                      "dispatches": len(fv[k])}
            total += fb + wb
        if not per:
            continue
        out = {"call": call, "workload": workload, "hbm_bytes_per_launch": int(round(total)),
               "kernels": per, "fetch_scale": round(fetch_scale, 4),
               "write_scale": round(write_scale, 4),
               "calibration": f"1 GiB device copy: FETCH_SIZE {max(cf):.1f} KiB, "
                              f"WRITE_SIZE {max(cw):.1f} KiB per launch",
               "source_digest": source_digest()}
        path = os.path.join(ROOT, "profiles", f"traffic_{call}_{workload}.json")
        with open(path, "w") as fh:
            json.dump(out, fh, indent=1)
            fh.write("\n")
        print(f"{call}: {total / 1e6:.2f} MB per call -> {os.path.relpath(path, ROOT)}")
        for k, v in per.items():
            print(f"   {k:30s} read {v['fetch_bytes'] / 1e6:9.2f} MB  written "
                  f"{v['write_bytes'] / 1e6:8.2f} MB  ({v['dispatches']} dispatches)")


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _oracle_step_rate(w, sl, min_seconds):
    """Verified tree-tokens/s of the oracle's whole step on sequences `sl`,
    repeated until about min_seconds of CPU work."""
    import oracle
    nn = None if w.num_nodes is None else w.num_nodes[sl]
    reps, t0 = 0, time.perf_counter()
    while True:
        oracle.tree_attention(w.q[sl], w.k_tree[sl], w.v_tree[sl], w.k_cache, w.v_cache,
                              w.page_table[sl], w.kv_len[sl], w.parent[sl], num_nodes=nn)
        a = oracle.argmax(w.logits[sl])
        alen, aidx, _ = oracle.accept(w.draft[sl], w.parent[sl], a, num_nodes=nn)
        oracle.kv_compact(w.k_tree[sl], w.v_tree[sl], w.k_cache, w.v_cache, w.page_table[sl],
                          w.kv_len[sl], aidx, alen)
        reps += 1
        dt = time.perf_counter() - t0
        if dt >= min_seconds or reps >= 50:
            break
    tokens = int(real_nodes(w)[sl].sum())
    return reps * tokens / dt, reps, dt


def cpu_baseline(w, sample_b: int, min_seconds: float = 10.0, single_thread: bool = False):
    """The fp64 CPU oracle on the first `sample_b` sequences of the same
    workload, on every host thread; with `single_thread`, also on one."""
    import oracle
    sl = slice(0, sample_b)
    threads = oracle.num_threads()
    rate, reps, dt = _oracle_step_rate(w, sl, min_seconds)
    out = {"value": round(rate, 2), "unit": "verified tree-tokens/s", "cores": threads,
           "kind": "oracle", "cpu_model": cpu_model(),
           "sample": f"{sample_b} of {w.B} sequences of the same workload, {reps} passes "
                     f"(fp64 C, OpenMP, {threads} threads), {dt:.2f} s"}
    if single_thread:
        oracle.set_num_threads(1)
        try:
            rate1, reps1, dt1 = _oracle_step_rate(w, sl, min_seconds / 2)
        finally:
            oracle.set_num_threads(threads)
        out["value_1_thread"] = round(rate1, 2)
        out["sample_1_thread"] = f"the same sample on one thread, {reps1} passes, {dt1:.2f} s"
    return out


def tree_build_bytes(x, accept_len=None, r_min: int = 0) -> int:
    """Bytes the tree builder must move per call: the logits rows it uses once,
    the hot map once, one table row per expanded node, the outputs. With
    accept_len (re-sampling) only the remaining rows of each sequence count."""
    steps = np.full(x.B, x.S) if accept_len is None else np.maximum(x.S - accept_len, 0)
    if accept_len is not None:
        steps = np.where(steps > r_min, steps, 0)
    rows = int(steps.sum())
    expanded = int(sum(1 + (s - 1) * x.k for s in steps if s > 0))
    return (rows * x.V * 4 + (x.V * 4 + x.H * 4 if x.H else 0) + expanded * x.H * 2
            + x.B * x.budget * 12 + x.B * 8)


def run_tree_build(args, T, torch):
    """The draft-tree builder (token-info sampling, Alg. 1, and budget
    pruning) on one batch per step; value = draft trees per second."""
    from paper_2602_21224_amd import workloads as W
    x = W.tree_build_preset(args.workload)
    resample = args.workload.startswith("rs_")
    r_min = 1
    dev = torch.device("cuda:0")
    print(f"# workload {args.workload}: B={x.B} S={x.S} V={x.V} H={x.H} k={x.k} "
          f"budget={x.budget}", file=sys.stderr, flush=True)
    up = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    table = up(x.table.view(np.int16)).view(torch.bfloat16) if x.H else None
    hot_vocab = up(x.hot_vocab) if x.H else None
    hot_index = up(x.hot_index) if x.H else None
    copies = [dict(logits=up(x.logits), root=up(x.root))]
    if resample:
        bonus, alen = W.resample_inputs(x, 7)
        copies[0].update(bonus=up(bonus), alen=up(alen))
    copies += [{k: v.clone() for k, v in copies[0].items()} for _ in range(args.copies - 1)]
    ws = torch.empty(T.tree_build_workspace_size(x.B, x.S, x.V, x.H, x.k), dtype=torch.uint8,
                     device=dev)
    outs = [dict(parent=torch.empty((x.B, x.budget), dtype=torch.int32, device=dev),
                 token=torch.empty((x.B, x.budget), dtype=torch.int32, device=dev),
                 joint=torch.empty((x.B, x.budget), dtype=torch.float32, device=dev),
                 nn=torch.empty((x.B,), dtype=torch.int32, device=dev)) for _ in copies]
    stream = torch.cuda.current_stream()
    tev = TimingEvents()

    def step(i, ev=None):
        c, o = copies[i % len(copies)], outs[i % len(copies)]
        if ev: tev.record(ev[0], stream)
        if resample:
            T.tree_resample(c["logits"], c["bonus"], c["alen"], table, hot_vocab, hot_index,
                            k=x.k, r=r_min, budget=x.budget, parent=o["parent"],
                            token=o["token"], joint=o["joint"], num_nodes=o["nn"], workspace=ws)
        else:
            T.tree_build(c["logits"], c["root"], table, hot_vocab, hot_index, k=x.k,
                         budget=x.budget, parent=o["parent"], token=o["token"], joint=o["joint"],
                         num_nodes=o["nn"], workspace=ws)
        if ev: tev.record(ev[1], stream)

    warm_steps = warm_up(step, args.warmup, args.min_warmup_s, torch)
    ev_every = max(1, min(4, args.steps // 8))
    evs = [[tev.create() for _ in range(2)] if i % ev_every == 0 else None
           for i in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(warm_steps + i, evs[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    sampled = [e for e in evs if e is not None]
    t_call = np.array([tev.seconds(e[0], e[1]) for e in sampled])
    for e in sampled:
        for q in e:
            tev.destroy(q)
    nbytes = tree_build_bytes(x, alen if resample else None, r_min)
    ach = nbytes / t_call.mean() / 1e9
    cpu = None
    if args.cpu_sample != 0:
        import oracle
        nb = x.B if args.cpu_sample < 0 else min(args.cpu_sample, x.B)
        reps, c0 = 0, time.perf_counter()
        while True:
            if resample:
                oracle.resample(x.logits[:nb], bonus[:nb], alen[:nb], x.table, x.hot_vocab, x.k,
                                r_min, x.budget)
            else:
                oracle.tree_build(x.logits[:nb], x.root[:nb], x.table, x.hot_vocab, x.k,
                                  x.budget)
            reps += 1
            dt = time.perf_counter() - c0
            if dt >= 10.0 or reps >= 50:
                break
        cpu = {"value": round(reps * nb / dt, 2), "unit": "draft trees/s", "cores": 1,
               "kind": "oracle", "cpu_model": cpu_model(),
               "sample": f"{nb} of {x.B} sequences of the same workload, {reps} passes "
                         f"(numpy, one thread), {dt:.2f} s"}
    line = {
        "metric": ("re-sampled draft trees/sec (Alg. 2 + budget pruning), 1 GPU" if resample else
                   "draft trees/sec (token-info sampling + budget pruning), 1 GPU"),
        "value": round(x.B / (wall / args.steps), 1), "unit": "draft trees/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(wall / args.steps * 1e3, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32+f64", "data": "synthetic",
        "config": {"workload": args.workload, "batch": x.B, "steps": x.S, "vocab": x.V,
                   "hot_tokens": x.H, "branch": x.k, "budget": x.budget,
                   "input_copies_rotated": len(copies)},
        "roofline": {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(ach / HBM_PEAK_GBS, 4),
                     "traffic": load_traffic("tree_build", args.workload), "kernel": "tree_build",
                     "avg_us": round(t_call.mean() * 1e6, 2), "algorithmic_bytes": int(nbytes),
                     "launches_per_call": 2 * x.S + 2},
        "call_us_p10_p50_p90": [pct(t_call, 10), pct(t_call, 50), pct(t_call, 90)],
        "warmup_steps_run": warm_steps,
        "timed_steps_with_events": len(sampled),
        "cpu_baseline": cpu,
        "source_digest": source_digest(),
    }
    print(json.dumps(line), flush=True)


def run_lm_head(args, T, torch):
    """The LM head fused with greedy verification (hidden states x head
    weight, per-node argmax, acceptance) on one batch per step; value =
    verified tree-tokens per second. The roofline is the matrix cores'
    (2 R V d flops per call against the dense bf16 peak)."""
    from paper_2602_21224_amd import workloads as W
    x = W.lm_head_preset(args.workload)
    dev = torch.device("cuda:0")
    R = x.B * x.N
    print(f"# workload {args.workload}: B={x.B} N={x.N} V={x.V} d={x.d}", file=sys.stderr,
          flush=True)
    up = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    w_head = up(x.w_head.view(np.int16)).view(torch.bfloat16)
    copies = [dict(hidden=up(x.hidden.view(np.int16)).view(torch.bfloat16), draft=up(x.draft),
                   parent=up(x.parent))]
    copies += [{k: v.clone() for k, v in copies[0].items()} for _ in range(args.copies - 1)]
    ws = torch.empty(T.lm_head_workspace_size(x.B, x.N, x.V, x.d), dtype=torch.uint8, device=dev)
    mk = lambda *shape: torch.empty(shape, dtype=torch.int32, device=dev)
    outs = [dict(amax=mk(x.B, x.N), alen=mk(x.B), aidx=mk(x.B, x.N), bonus=mk(x.B))
            for _ in copies]
    stream = torch.cuda.current_stream()
    tev = TimingEvents()

    def step(i, ev=None):
        c, o = copies[i % len(copies)], outs[i % len(copies)]
        if ev: tev.record(ev[0], stream)
        T.tree_lm_head_argmax_accept(c["hidden"], w_head, c["draft"], c["parent"],
                                     argmax_out=o["amax"], accept_len=o["alen"],
                                     accept_idx=o["aidx"], bonus_token=o["bonus"], workspace=ws)
        if ev: tev.record(ev[1], stream)

    warm_steps = warm_up(step, args.warmup, args.min_warmup_s, torch)
    ev_every = max(1, min(4, args.steps // 8))
    evs = [[tev.create() for _ in range(2)] if i % ev_every == 0 else None
           for i in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(warm_steps + i, evs[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    sampled = [e for e in evs if e is not None]
    t_call = np.array([tev.seconds(e[0], e[1]) for e in sampled])
    # Context: the library GEMM of the same product (bf16 logits written to HBM,
    # no argmax), timed the same way.
    hid2 = copies[0]["hidden"].reshape(R, x.d)
    for _ in range(5):
        torch.nn.functional.linear(hid2, w_head)
    torch.cuda.synchronize()
    t_lib = []
    for e in sampled[:8]:
        tev.record(e[0], stream)
        torch.nn.functional.linear(hid2, w_head)
        tev.record(e[1], stream)
        torch.cuda.synchronize()
        t_lib.append(tev.seconds(e[0], e[1]))
    for e in sampled:
        for q in e:
            tev.destroy(q)
    alen = outs[(warm_steps + args.steps - 1) % len(copies)]["alen"].cpu().numpy()
    flop = 2.0 * R * x.V * x.d
    tflops = flop / t_call.mean() / 1e12
    cpu = None
    if args.cpu_sample != 0:
        import oracle
        nr = 16
        reps, c0 = 0, time.perf_counter()
        while True:
            oracle.lm_head_argmax(x.hidden.reshape(R, x.d)[:nr], x.w_head)
            reps += 1
            dt = time.perf_counter() - c0
            if dt >= 10.0:
                break
        cpu = {"value": round(reps * nr / dt, 2), "unit": "verified tree-tokens/s",
               "cores": int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1)),
               "kind": "oracle", "cpu_model": cpu_model(),
               "sample": f"LM-head argmax of the first {nr} of {R} node rows over the whole "
                         f"vocabulary, {reps} passes (numpy fp64 matmul), {dt:.2f} s"}
    line = {
        "metric": "verified tree-tokens/sec (LM head fused with argmax + accept), 8B-shaped, "
                  "1 GPU",
        "value": round(R / (wall / args.steps), 1), "unit": "verified tree-tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(wall / args.steps * 1e3, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": args.workload, "batch": x.B, "tree_nodes": x.N, "vocab": x.V,
                   "hidden": x.d, "input_copies_rotated": len(copies)},
        "roofline": {"bound": "mfma", "achieved": round(tflops, 1),
                     "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(tflops / MFMA_BF16_PEAK_TFLOPS, 4),
                     "traffic": load_traffic("tree_lm_head_argmax_accept", args.workload),
                     "kernel": "tree_lm_head_argmax_accept",
                     "avg_us": round(t_call.mean() * 1e6, 2), "algorithmic_flop": flop,
                     "launches_per_call": 3},
        "call_us_p10_p50_p90": [pct(t_call, 10), pct(t_call, 50), pct(t_call, 90)],
        "warmup_steps_run": warm_steps,
        "library_gemm_bf16_out_us": round(float(np.median(t_lib)) * 1e6, 2) if t_lib else None,
        "accept_len_hist": np.bincount(alen, minlength=1).tolist(),
        "timed_steps_with_events": len(sampled),
        "cpu_baseline": cpu,
        "source_digest": source_digest(),
    }
    print(json.dumps(line), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=100)
    ap.add_argument("--min-warmup-s", type=float, default=1.5,
                    help="keep warming up (untimed) until this many seconds have passed")
    ap.add_argument("--workload", default="llama8b_bs16")
    ap.add_argument("--copies", type=int, default=3)
    ap.add_argument("--cpu-sample", type=int, default=-1,
                    help="sequences in the CPU-oracle sample (-1: all, 0: skip)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB a few times (calibrates "
                         "the HBM byte counters against a known size) and exit")
    ap.add_argument("--write-traffic", nargs=4, metavar=("FETCH_DIR", "WRITE_DIR", "COPY_FETCH_DIR",
                                                      "COPY_WRITE_DIR"),
                    help="convert rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE output directories "
                         "(this benchmark, then --copy-calibration 1024) into "
                         "profiles/traffic_*.json and exit; needs no GPU")
    args = ap.parse_args()
    if args.write_traffic:
        write_traffic(args.workload, *args.write_traffic)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); the verification "
              "step shards by sequence with no exchange, so N GPUs run N independent copies.",
              file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2602_21224_amd as T
    from paper_2602_21224_amd import workloads as W

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.copy_calibration > 0:
        n = args.copy_calibration << 20
        src = torch.ones(n, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes": n, "launches": 3}), flush=True)
        return
    T.load()
    if args.workload in W.TREE_BUILD_PRESETS:
        run_tree_build(args, T, torch)
        return
    if args.workload in W.LM_HEAD_PRESETS:
        run_lm_head(args, T, torch)
        return
    w = W.preset(args.workload)
    print(f"# workload {args.workload}: B={w.B} N={w.N} Hq={w.Hq} Hkv={w.Hkv} D={w.D} "
          f"V={w.V} kv_len sum={int(w.kv_len.sum())}", file=sys.stderr, flush=True)

    def up(a, bf16=False):
        t = torch.from_numpy(np.ascontiguousarray(a.view(np.int16) if bf16 else a))
        t = t.to(dev)
        return t.view(torch.bfloat16) if bf16 else t

    base = dict(q=up(w.q, True), k_tree=up(w.k_tree, True), v_tree=up(w.v_tree, True),
                k_cache=up(w.k_cache, True), v_cache=up(w.v_cache, True),
                page_table=up(w.page_table), kv_len=up(w.kv_len), parent=up(w.parent),
                draft=up(w.draft), logits=up(w.logits))
    if w.num_nodes is not None:
        base["num_nodes"] = up(w.num_nodes)
    copies = [base] + [{k: v.clone() for k, v in base.items()} for _ in range(args.copies - 1)]
    ws_attn = torch.empty(T.attention_workspace_size(w.B, w.N, w.Hq, w.Hkv, w.D),
                          dtype=torch.uint8, device=dev)
    ws_acc = torch.empty(T.argmax_workspace_size(w.B, w.N, w.V), dtype=torch.uint8, device=dev)
    outs = [dict(out=torch.empty((w.B, w.N, w.Hq, w.D), dtype=torch.bfloat16, device=dev),
                 lse=torch.empty((w.B, w.N, w.Hq), dtype=torch.float32, device=dev),
                 amax=torch.empty((w.B, w.N), dtype=torch.int32, device=dev),
                 alen=torch.empty((w.B,), dtype=torch.int32, device=dev),
                 aidx=torch.empty((w.B, w.N), dtype=torch.int32, device=dev),
                 bonus=torch.empty((w.B,), dtype=torch.int32, device=dev))
            for _ in copies]
    stream = torch.cuda.current_stream()

    tev = TimingEvents()

    def step(i, ev=None):
        c, o = copies[i % len(copies)], outs[i % len(copies)]
        if ev: tev.record(ev[0], stream)
        T.tree_verify_attention(c["q"], c["k_tree"], c["v_tree"], c["k_cache"], c["v_cache"],
                                c["page_table"], c["kv_len"], c["parent"],
                                max_kv_len=w.max_kv_len, out=o["out"], lse=o["lse"],
                                workspace=ws_attn, num_nodes=c.get("num_nodes"))
        if ev: tev.record(ev[1], stream)
        T.tree_argmax_accept(c["logits"], c["draft"], c["parent"], argmax_out=o["amax"],
                             accept_len=o["alen"], accept_idx=o["aidx"], bonus_token=o["bonus"],
                             workspace=ws_acc, num_nodes=c.get("num_nodes"))
        if ev: tev.record(ev[2], stream)
        T.kv_compact_accepted(c["k_tree"], c["v_tree"], c["k_cache"], c["v_cache"],
                              c["page_table"], c["kv_len"], o["aidx"], o["alen"])
        if ev: tev.record(ev[3], stream)

    warm_steps = warm_up(step, args.warmup, args.min_warmup_s, torch)

    # Even a fence-free event record costs the stream about a microsecond, so
    # the per-call durations are taken on every ev_every-th timed step only.
    ev_every = max(1, min(4, args.steps // 8))
    evs = [[tev.create() for _ in range(4)] if i % ev_every == 0 else None
           for i in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(warm_steps + i, evs[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0

    sampled = [e for e in evs if e is not None]
    t_attn = np.array([tev.seconds(e[0], e[1]) for e in sampled])
    t_acc = np.array([tev.seconds(e[1], e[2]) for e in sampled])
    t_cmp = np.array([tev.seconds(e[2], e[3]) for e in sampled])
    for e in sampled:
        for x in e:
            tev.destroy(x)
    ms_per_step = wall / args.steps * 1e3
    tokens = int(real_nodes(w).sum())
    value = tokens / (wall / args.steps)

    alen = outs[(warm_steps + args.steps - 1) % len(copies)]["alen"].cpu().numpy()
    attn_bytes, attn_flop, acc_bytes = algorithmic(w)
    cmp_bytes = compact_bytes(w, alen)
    a_attn = attn_bytes / t_attn.mean() / 1e9
    a_acc = acc_bytes / t_acc.mean() / 1e9

    ridge = MFMA_BF16_PEAK_TFLOPS * 1e12 / (HBM_PEAK_GBS * 1e9)     # FLOP per byte

    def roof(kernel, bytes_, ts, flop=None):
        """Roofline of one call from its per-call event times `ts`: HBM-bound
        (GB/s against 8 TB/s) unless its algorithmic FLOP per byte is above the
        ridge, then matrix-bound (TFLOP/s against the dense bf16 peak)."""
        t = ts.mean()
        gbs = bytes_ / t / 1e9
        r = {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS,
             "unit": "GB/s", "frac": round(gbs / HBM_PEAK_GBS, 4),
             "traffic": load_traffic(kernel, args.workload),
             "kernel": kernel, "avg_us": round(t * 1e6, 2), "p10_us": pct(ts, 10),
             "p50_us": pct(ts, 50), "p90_us": pct(ts, 90), "algorithmic_bytes": int(bytes_)}
        if flop is not None:
            tf = flop / t / 1e12
            r["tflops"] = round(tf, 1)
            r["mfma_frac"] = round(tf / MFMA_BF16_PEAK_TFLOPS, 4)
            r["hbm_gbs"] = round(gbs, 1)
            r["hbm_frac"] = round(gbs / HBM_PEAK_GBS, 4)
            r["algorithmic_flop"] = int(flop)
            if flop / bytes_ > ridge:
                r.update(bound="mfma", achieved=round(tf, 1), peak=MFMA_BF16_PEAK_TFLOPS,
                         unit="TFLOP/s", frac=round(tf / MFMA_BF16_PEAK_TFLOPS, 4))
        return r

    r_attn = roof("tree_verify_attention", attn_bytes, t_attn, attn_flop)
    r_acc = roof("tree_argmax_accept", acc_bytes, t_acc)
    dominant = r_acc if t_acc.mean() >= t_attn.mean() else r_attn

    cpu = None
    if args.cpu_sample != 0:
        nb = w.B if args.cpu_sample < 0 else min(args.cpu_sample, w.B)
        cpu = cpu_baseline(w, nb, single_thread=args.workload in ("tiny", "llama8b_bs1"))

    line = {
        "metric": METRIC, "value": round(value, 1), "unit": "verified tree-tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": args.workload, "batch": w.B, "tree_nodes": w.N,
                   "q_heads": w.Hq, "kv_heads": w.Hkv, "head_dim": w.D, "page_size": w.P,
                   "vocab": w.V, "kv_len_sum": int(w.kv_len.sum()),
                   "kv_len_range": [int(w.kv_len.min()), int(w.kv_len.max())],
                   "input_copies_rotated": len(copies),
                   "verified_nodes_per_step": tokens},
        "roofline": dominant,
        "roofline_attention": r_attn,
        "step_breakdown_us": {"attention": round(t_attn.mean() * 1e6, 2),
                              "argmax_accept": round(t_acc.mean() * 1e6, 2),
                              "compact": round(t_cmp.mean() * 1e6, 2),
                              "attention_p10_p50_p90": [pct(t_attn, 10), pct(t_attn, 50),
                                                        pct(t_attn, 90)],
                              "argmax_accept_p10_p50_p90": [pct(t_acc, 10), pct(t_acc, 50),
                                                            pct(t_acc, 90)],
                              "compact_p10_p50_p90": [pct(t_cmp, 10), pct(t_cmp, 50),
                                                      pct(t_cmp, 90)],
                              "timed_steps_with_events": len(sampled)},
        "warmup_steps_run": warm_steps,
        "kernel_tokens_per_s": round(tokens / (t_attn.mean() + t_acc.mean() + t_cmp.mean()), 1),
        "accept_len_hist": np.bincount(alen).tolist(),
        "compact_bytes": cmp_bytes,
        "cpu_baseline": cpu,
        "source_digest": source_digest(),
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
