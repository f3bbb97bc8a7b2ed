"""Benchmark of the paged-attention hot path on one MI355X.

A step is one pass of the whole path over one batch: the KV-cache write of
the batch's new tokens followed by attention, i.e. the phases of
vd_attn_forward -- plan (launched only when the batch needs it: prefill rows,
whose new tokens it writes, or more than 256 requests), split, chunk and merge
-- on synthetic bf16 inputs already resident in HBM; on a decode batch the
split items write the new tokens themselves.  R replicas of the inputs (pools,
page tables, queries) are cycled so that no step finds its K/V in the 256 MB
last-level cache left behind by the previous step.

Prints one JSON line: whole-step KV GB/s (algorithmic K+V bytes of the batch
over the step time), the roofline of the dominant kernel measured with HIP
events on the launch stream (recorded by that kernel's own dispatch, so that
no marker packet sits between the step's kernels), and the CPU oracle timed
on the host as a reported baseline.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0        # MI355X HBM3E, vendor figure
MFMA_BF16_PEAK_TFS = 2500.0  # MI355X dense bf16 matrix peak, vendor figure


def log(msg):
    print("[bench] " + msg, file=sys.stderr, flush=True)


def workloads():
    from paper_2609_38981_amd import workloads as W
    return {
        "decode8b": (lambda: W.config2(pool_factor=1.5),
                     "Llama-3-8B paged decode: 64 requests, context U[512,4096], Hq 32 / Hkv 8, "
                     "head_dim 128, page 16, pool 1.5x need"),
        "mixed8b": (lambda: W.config3(),
                    "Llama-3-8B mixed batch: 8 prefill chunks of 512 at offsets U[0,8192] + 120 "
                    "decodes with context U[256,8192], Hq 32 / Hkv 8, head_dim 128, page 16"),
        "longdecode8b": (lambda: W.config4(),
                         "Llama-3-8B long-context decode: 8 requests, context U[32768,131072], "
                         "Hq 32 / Hkv 8, head_dim 128, page 16"),
        "verify70b": (lambda: W.config5(),
                      "Llama-70B prefix-shared verify: 256 requests on a shared 2048-token prefix "
                      "+ suffix U[64,512], s=4 (even) / s=1 (odd), Hq 64 / Hkv 8, head_dim 128"),
        "tiny": (lambda: W.config1(), "tiny: 2 requests (n 37 s 1, n 100 s 8), Hq 4 / Hkv 2, D 64"),
        "swa8b": (lambda: W.config2(batch=32, lo=8192, hi=32768, shape=W.LLAMA8B_SWA4K, cfg=6,
                                    pool_factor=1.5),
                  "Llama-3-8B geometry with a 4096-key sliding window, paged decode: 32 requests, "
                  "context U[8192,32768], Hq 32 / Hkv 8, head_dim 128, page 16, pool 1.5x need"),
    }


def kernel_code_digest() -> str:
    """SHA-256 of the attention kernels' code: the sources with comments
    removed and whitespace collapsed, so that an edit of a comment does not
    count as a change of the kernel."""
    import hashlib
    import re

    csrc = os.path.join(ROOT, "paper_2609_38981_amd", "csrc")
    code = []
    for n in ("vd_attn.hip", "vd_cas.hpp", "vd_hw.hpp"):
        with open(os.path.join(csrc, n)) as f:
            t = f.read()
        t = re.sub(r"/\*.*?\*/", " ", t, flags=re.S)
        t = re.sub(r"//[^\n]*", " ", t)
        code.append(" ".join(t.split()))
    return hashlib.sha256("\n".join(code).encode()).hexdigest()


def measured_traffic(kernel: str, workload: str):
    """HBM bytes per launch from the committed rocprofv3 counter summaries
    (profiles/hbm_traffic.json: one entry per (kernel, workload)), or None when
    no entry covers this kernel and workload or the kernels' code changed since
    its counters were taken.  ``kernel`` may name several kernels joined by
    "+" (a phase that launches them back to back): the sum of their entries,
    or None unless every one has a current entry."""
    path = os.path.join(ROOT, "profiles", "hbm_traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        entries = json.load(f).get("entries", [])
    digest = kernel_code_digest()
    total = 0
    for k in kernel.split("+"):
        hit = [e for e in entries if e.get("kernel") == k and e.get("workload") == workload
               and e.get("code_sha256") == digest]
        if not hit:
            return None
        total += int(hit[-1]["bytes_per_launch"])
    return total


def host_threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    cap = os.environ.get("OMP_NUM_THREADS")
    if cap and cap.isdigit():
        n = min(n, int(cap))
    return max(n, 1)


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def err_vs_gpu(got, ref) -> dict:
    """The GPU output against the oracle: the largest absolute difference, and
    that difference relative to the largest oracle magnitude of the sample (the
    bf16 rounding of an output alone accounts for up to 2^-9 of its own
    magnitude)."""
    diff = np.abs(got - ref)
    scale = float(np.abs(ref).max())
    return {"max_abs_err_vs_gpu": float(diff.max()),
            "max_err_rel_to_max_abs": float(diff.max()) / scale if scale > 0 else 0.0}


def cpu_baseline(call, gpu_bits=None, min_seconds: float = 10.0, max_requests: int = 64):
    """The oracle on the host on a bounded sample of the same workload: the
    first requests of the batch (whole requests), repeated until at least
    ``min_seconds`` of wall time.  Returns KV GB/s of the sample and, with the
    GPU output of the whole call (``gpu_bits``, uint16 [T, Hq, D]), the largest
    difference between the oracle and the GPU on the sample's rows."""
    import oracle
    from paper_2609_38981_amd import workloads as W

    sh = call.shape
    # bound the sample: whole requests until ~4 G multiply-adds of attention work
    reqs, work = [], 0
    for r in call.reqs[:max_requests]:
        cost = r.s * r.n * sh.num_q_heads * sh.head_dim * 2
        if reqs and work + cost > 4e9:
            break
        reqs.append(r)
        work += cost
    sub = W.Call(sh, call.prompts, reqs, call.page_table[:len(reqs)], call.num_pages,
                 call.page_owner)
    kp, vp = call.std_pool(poison=False)
    args = (sub.q_bits(), sub.cu_q_lens, sub.context_lens, sub.page_table, kp, vp)
    kw = dict(num_q_heads=sh.num_q_heads, num_kv_heads=sh.num_kv_heads, head_dim=sh.head_dim,
              page_size=sh.page_size, window=sh.window)
    threads = host_threads()
    reps, t0 = 0, time.perf_counter()
    while True:
        ref = oracle.paged_attention(*args, threads=threads, **kw)
        reps += 1
        el = time.perf_counter() - t0
        if el >= min_seconds or reps >= 1000:
            break
    sec = el / reps
    res = {"value": round(sub.kv_bytes() / sec / 1e9, 4), "unit": "GB/s", "cores": threads,
           "kind": "oracle", "cpu_model": cpu_model(),
           "sample": "%d of %d requests (%d query rows, %.1f MB K+V), %d repetitions, %.2f s "
                     "per repetition" % (len(reqs), call.num_seqs, sub.total_q_tokens,
                                         sub.kv_bytes() / 1e6, reps, sec)}
    if gpu_bits is not None:
        # the sample's rows are the call's first rows
        got = W.bf16_to_f32(gpu_bits[:sub.total_q_tokens]).astype(np.float64)
        res.update(err_vs_gpu(got, ref))
    return res


# The batch-invariant linear layer (vd_linear): (M tokens, N outputs, K inputs)
LINEAR_WORKLOADS = {
    "linear8b": ((4096, 6144, 4096),
                 "Llama-3-8B QKV projection: 4096 tokens, 4096 -> 6144 (q 4096, k 1024, v 1024), "
                 "bf16 activations and weights, fp32 accumulation"),
}


def linear_cpu_baseline(a_bits, b_bits, gpu_bits=None, min_seconds: float = 10.0):
    """The oracle (fp64 plain loops) on a bounded sample of the same layer: the
    first rows of the activations, repeated until at least ``min_seconds``;
    with the GPU output (``gpu_bits``, uint16 [M, N]), the largest absolute
    difference from the oracle on the sample's rows."""
    from paper_2609_38981_amd import workloads as W

    import oracle

    M, K = a_bits.shape
    N = b_bits.shape[0]
    rows = max(1, min(M, int(4e9 // (2 * N * K))))  # ~4 GFLOP of work per repetition
    threads = host_threads()
    reps, t0 = 0, time.perf_counter()
    while True:
        ref = oracle.linear(a_bits[:rows], b_bits, threads=threads)
        reps += 1
        el = time.perf_counter() - t0
        if el >= min_seconds or reps >= 1000:
            break
    sec = el / reps
    res = {"value": round(2.0 * rows * N * K / sec / 1e12, 6), "unit": "TFLOP/s",
           "cores": threads, "kind": "oracle", "cpu_model": cpu_model(),
           "sample": "%d of %d rows (%d x %d x %d), %d repetitions, %.2f s per repetition"
                     % (rows, M, rows, N, K, reps, sec)}
    if gpu_bits is not None:
        got = W.bf16_to_f32(gpu_bits[:rows]).astype(np.float64)
        res.update(err_vs_gpu(got, ref))
    return res


def bench_linear(args):
    """One step = one vd_linear call over the whole layer (inputs resident in
    HBM, R replicas cycled); the kernel is the whole step."""
    import torch

    from paper_2609_38981_amd import staging as S
    from paper_2609_38981_amd import vdattn as V
    from paper_2609_38981_amd import workloads as W

    (M, N, K), desc = LINEAR_WORKLOADS[args.workload]
    rng = W.rng_for(7, 1)
    a_bits, b_bits = W.normal_bf16(rng, (M, K)), W.normal_bf16(rng, (N, K))
    reps = []
    for _ in range(max(args.replicas, 1)):
        a, b = S.bf16_tensor(a_bits, "cuda"), S.bf16_tensor(b_bits, "cuda")
        reps.append((a, b, torch.empty((M, N), dtype=torch.bfloat16, device="cuda")))
    stream = torch.cuda.current_stream()
    for i in range(args.warmup):
        V.linear(*reps[i % len(reps)])
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(args.steps)]
    t0 = time.perf_counter()
    for i in range(args.steps):
        a, b, c = reps[i % len(reps)]
        evs[i][0].record(stream)
        V.linear(a, b, c)
        evs[i][1].record(stream)
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / args.steps
    k_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in evs]))
    gpu_bits = S.bits_of(reps[0][2])  # before torch.matmul below overwrites it
    flop = 2.0 * M * N * K
    ach = flop / (k_ms * 1e-3) / 1e12
    # context: the vendor library GEMM on the same shapes (not batch-invariant in general)
    a, b, c = reps[0]
    bt = b.t()
    for _ in range(3):
        torch.matmul(a, bt, out=c)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(20):
        torch.matmul(a, bt, out=c)
    e1.record(stream)
    torch.cuda.synchronize()
    lib_ms = e0.elapsed_time(e1) / 20
    log("linear %s: %.4f ms/step, kernel %.4f ms = %.1f TFLOP/s; torch.matmul %.4f ms"
        % (args.workload, ms, k_ms, ach, lib_ms))
    res = {
        "metric": "batch-invariant linear TFLOP/s (bf16, fp32 accumulation)",
        "value": round(flop / (ms * 1e-3) / 1e12, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms, 5), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": desc, "M": M, "N": N, "K": K, "replicas": len(reps)},
        "roofline": {"kernel": "linear_kernel", "bound": "mfma", "achieved": round(ach, 2),
                     "peak": MFMA_BF16_PEAK_TFS, "unit": "TFLOP/s",
                     "frac": round(ach / MFMA_BF16_PEAK_TFS, 4), "traffic": None,
                     "avg_ms": round(k_ms, 5), "timed_launches": args.steps,
                     "algorithmic_flop": int(flop)},
        "torch_matmul_tflops": round(flop / (lib_ms * 1e-3) / 1e12, 2),
    }
    if not args.no_cpu_baseline:
        log("timing the CPU oracle baseline")
        res["cpu_baseline"] = linear_cpu_baseline(a_bits, b_bits, gpu_bits)
    print(json.dumps(res), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="longdecode8b",
                    choices=sorted(workloads()) + sorted(LINEAR_WORKLOADS))
    ap.add_argument("--replicas", type=int, default=4)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--time-every", type=int, default=4,
                    help="time the dominant kernel with HIP events on every N-th timed step "
                         "(each timed launch costs the stream a few microseconds)")
    ap.add_argument("--copy-calibration-mb", type=int, default=0,
                    help="run one plain copy kernel of this many MiB (float32 negate: reads "
                         "and writes that many bytes) before timing, to calibrate HBM counters")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the library has no multi-GPU path (the kernels "
              "run on one GPU's share of the work). Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2609_38981_amd import staging as S
    from paper_2609_38981_amd import vdattn as V

    torch.cuda.set_device(0)
    if args.workload in LINEAR_WORKLOADS:
        return bench_linear(args)
    make, desc = workloads()[args.workload]
    t0 = time.perf_counter()
    call = make()
    sh = call.shape
    log("workload %s: %d requests, %d query rows, %.1f MB K+V (%.1fs to generate)" % (
        args.workload, call.num_seqs, call.total_q_tokens, call.kv_bytes() / 1e6,
        time.perf_counter() - t0))
    attn = S.handle_for(sh)

    # replicas of every device input: the first staged from the host, the others
    # device copies of it
    reps = []
    dc0 = S.to_device(attn, call, poison=False)
    for i in range(max(args.replicas, 1)):
        dc = dc0 if i == 0 else S.clone_device_call(dc0)
        ws = attn.new_workspace(call.num_seqs, dc.batch.max_q_len, dc.batch.max_context_len)
        reps.append((dc, ws, torch.empty_like(dc.batch.q)))
    P = sh.page_size
    # this step's new tokens (the K/V of the query rows, positions n - s .. n - 1
    # of every request): the call writes them into the pool before attention
    # reads it (the split items themselves, or the plan launch)
    kn, vn = call.query_kv()
    k_new, v_new = S.bf16_tensor(kn, "cuda"), S.bf16_tensor(vn, "cuda")
    for dc, _, _ in reps:
        dc.batch.k_new, dc.batch.v_new = k_new, v_new
    torch.cuda.synchronize()
    log("staged %d replicas" % len(reps))

    stream = torch.cuda.current_stream()
    G = sh.group
    # visible keys of the row at p: p + 1, or at most the window
    vis = (lambda p: min(p + 1, sh.window)) if sh.window > 0 else (lambda p: p + 1)
    chunk_flops = sum(sum(vis(p) for p in r.positions) for r in call.reqs
                      if r.s * G > 32) * sh.num_q_heads * sh.head_dim * 4
    split_idx = [i for i, r in enumerate(call.reqs) if r.s * G <= 32]
    split_reqs = [call.reqs[i] for i in split_idx]
    # bytes the split kernel must read at least once: distinct cache slots
    # (pages shared by several requests count once)
    split_bytes = call.unique_kv_bytes(split_idx)
    # the kernel that bounds the step: compare ideal times on its roofline
    dominant = "chunks" if chunk_flops / (MFMA_BF16_PEAK_TFS * 1e12) > \
        split_bytes / (HBM_PEAK_GBS * 1e9) else "splits"

    # each replica's call marshalled once: a phase is then a single C call
    prepared = [attn.prepare(dc.batch, out, ws, stream) for dc, ws, out in reps]

    def step(i, ev=None, all_ev=None, timed=None):
        pc = prepared[i % len(prepared)]
        phases = [pc.plan, pc.splits, pc.chunks, pc.merge]
        names = ["plan_and_kv_write", "splits", "chunks", "merge"]
        for j, (name, fn) in enumerate(zip(names, phases)):
            if all_ev is not None:
                all_ev[j].record(stream)
            if ev is not None and name == (timed or dominant):
                fn(events=ev)  # recorded by the kernel's own dispatch
            else:
                fn()
        if all_ev is not None:
            all_ev[len(phases)].record(stream)

    if args.copy_calibration_mb:
        # one plain copy kernel of known size, for scaling the HBM counters
        n = (args.copy_calibration_mb << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        torch.neg(src, out=dst)
        torch.cuda.synchronize()
        del src, dst
    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    every = max(args.time_every, 1)
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(2)]
           for _ in range(0, args.steps, every)]
    for pair in evs:  # create the HIP events before the timed region
        for e in pair:
            e.record(stream)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(args.warmup + i, ev=evs[i // every] if i % every == 0 else None)
    enqueued = time.perf_counter() - t0
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ms = elapsed * 1e3 / args.steps
    dom_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in evs]))
    # diagnostic pass (not the timed region): every phase bracketed
    diag = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(10)]
    for i in range(10):
        step(i, all_ev=diag[i])
    torch.cuda.synchronize()
    ph_ms = np.mean([[e[j].elapsed_time(e[j + 1]) for j in range(4)] for e in diag], axis=0)
    log("timed: %.4f ms/step (enqueue %.4f), %s kernel %.4f ms; diagnostic phases (ms): "
        "plan+kv_write %.4f splits %.4f chunks %.4f merge %.4f"
        % (ms, enqueued * 1e3 / args.steps, dominant, dom_ms, *ph_ms))

    # outside the timed region: a call with both kinds of rows also times the
    # other phase's kernel by its own dispatches
    other = "chunks" if dominant == "splits" else "splits"
    other_ms = None
    if chunk_flops > 0 and split_reqs:
        oev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(8)]
        for pair in oev:
            for e in pair:
                e.record(stream)
        torch.cuda.synchronize()
        for i in range(len(oev)):
            step(i, ev=oev[i], timed=other)
        torch.cuda.synchronize()
        other_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in oev]))

    kv_bytes = call.kv_bytes()
    uniq_bytes = call.unique_kv_bytes()
    T = call.total_q_tokens
    hq, hkv, D = sh.num_q_heads, sh.num_kv_heads, sh.head_dim
    value = kv_bytes / (ms * 1e-3) / 1e9

    def roofline(kind, k_ms, launches):
        if kind == "chunks":
            ach = chunk_flops / (k_ms * 1e-3) / 1e12
            return {"kernel": "chunk_kernel", "bound": "mfma", "achieved": round(ach, 3),
                    "peak": MFMA_BF16_PEAK_TFS, "unit": "TFLOP/s",
                    "frac": round(ach / MFMA_BF16_PEAK_TFS, 4),
                    "traffic": measured_traffic("chunk_kernel", args.workload),
                    "avg_ms": round(k_ms, 5), "timed_launches": launches,
                    "algorithmic_flop": int(chunk_flops)}
        # K+V of the visible keys, Q, the page-table entries read; and when the
        # split launch writes the call's new tokens (at most 256 requests, and
        # at most 16 query rows per split-path request: groups of two or more
        # query heads, or max_q_len <= 16), every query row's K+V read from
        # k_new / v_new and written to the pool
        alg = split_bytes + sum(r.s for r in split_reqs) * hq * D * 2 + \
            sum(-(-r.n // P) - call.first_key(i) // P for i, r in zip(split_idx, split_reqs)) * 4
        if call.num_seqs <= 256 and (G >= 2 or call.max_q_len <= 16):
            alg += 2 * T * hkv * D * 2 * 2
        ach = alg / (k_ms * 1e-3) / 1e9
        # with the shared_pages hint the library's shared-prefix pass runs
        # (no window, 2 .. 1024 requests, contexts past one split): the timed
        # phase is the shared-prefix kernel and the split kernel together
        casc = bool(reps[0][0].batch.shared_pages) and sh.window == 0 and \
            2 <= call.num_seqs <= 1024 and call.max_context_len > V.SPLIT_KEYS
        return {"kernel": "prefix_kernel+split_kernel" if casc else "split_kernel",
                "bound": "hbm", "achieved": round(ach, 1),
                "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(ach / HBM_PEAK_GBS, 4),
                "traffic": measured_traffic("prefix_kernel+split_kernel" if casc else "split_kernel",
                                            args.workload),
                "avg_ms": round(k_ms, 5), "timed_launches": launches,
                "algorithmic_bytes": int(alg)}

    roof = roofline(dominant, dom_ms, len(evs))

    res = {
        "metric": "paged-attn KV GB/s (% HBM peak) at bitwise batch/chunk/page invariance",
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": desc, "num_seqs": call.num_seqs, "query_rows": T,
                   "kv_bytes": kv_bytes, "kv_bytes_distinct": uniq_bytes,
                   "replicas": len(reps)},
        # distinct K+V bytes of the call over the step time, against HBM peak
        "hbm_frac_whole_step": round(uniq_bytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        "tokens_per_s": round(T / (ms * 1e-3), 1),
        # host time to enqueue the timed steps: well below ms_per_step means
        # the GPU, not the launch path, set the pace
        "enqueue_ms_per_step": round(enqueued * 1e3 / args.steps, 5),
        "phase_ms_diagnostic": {k: round(float(v), 5) for k, v in
                                zip(["plan_and_kv_write", "splits", "chunks", "merge"], ph_ms)},
        "roofline": roof,
    }
    if other_ms is not None:
        # the other kind of rows' kernel (the dominant one is the kernel whose
        # ideal time on its own roofline is the longer)
        res["roofline_other_kernel"] = roofline(other, other_ms, len(oev))
    # outside the timed region: the output of the timed call, and the first and
    # last requests run alone, whose rows must be bit-identical to the batched ones
    gpu_bits = S.bits_of(reps[0][2])
    probe = sorted({0, call.num_seqs - 1})
    alone = call.subcall(probe)
    dca = S.to_device(attn, alone, poison=False)
    wsa = attn.new_workspace(alone.num_seqs, dca.batch.max_q_len, dca.batch.max_context_len)
    outa = torch.empty_like(dca.batch.q)
    attn.forward(dca.batch, out=outa, workspace=wsa)
    torch.cuda.synchronize()
    bits_a = S.bits_of(outa)
    same = 0
    for k, ri in enumerate(probe):
        for p in call.reqs[ri].positions:
            same += int(np.array_equal(bits_a[alone.row_of(k, p)], gpu_bits[call.row_of(ri, p)]))
    res["invariance"] = {"rows": int(alone.total_q_tokens), "bit_identical": same,
                         "variant": "requests %s alone vs in the timed batch" % probe}
    if not args.no_cpu_baseline:
        log("timing the CPU oracle baseline")
        res["cpu_baseline"] = cpu_baseline(call, gpu_bits)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
