"""Benchmark of the SegPagedAttention hot path on one MI355X.

A step is one pass of the hot path over one batch of synthetic input: page
selection (seg_paged_attn_select) and the attention forward with its split
combine (seg_paged_attn_fwd). The default workload is the largest
single-GPU decode: the variable-length sparse decode (64 requests, 32 query /
8 KV heads, head dim 128, contexts log-uniform in [4096, 131072] tokens in
4096-token segments, page 16, a per-request budget of 5-50% of the pages,
keys of each page scaled by LogNormal(0, 0.5)).

Output: one JSON line. `value` is attended KV tokens per second for the whole
step (inputs resident in HBM). `roofline` is the dominant kernel
(decode_attn): algorithmic bytes per launch over its mean launch time,
measured with HIP events attached to each dispatch on the launch stream.
`cpu_baseline` is the fp64 oracle timed on this host's cores (a pool of
single-threaded processes) on a sample of the same step.
`config.sub_records` holds the same measurement, from the same run, for the
Llama-3-8B-shaped decode (2), the chunked prefill (4, matrix-core bound) and
the top-k selection + attention workload (5, with its page-summary build
timed on its own).

python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload N] [--no-cpu-baseline]
                [--sub-records 2,4,5 | --no-sub-records]
"""
from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "attended KV tokens/s and achieved HBM GB/s (% of peak) for sparse decode"
HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0

# HBM bytes per launch from rocprofv3 FETCH_SIZE / WRITE_SIZE passes, scaled by
# what the same counters read for a device copy of known size. An entry counts
# only while the kernel's sources hash to the recorded value.
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic.json")
CSRC = os.path.join(ROOT, "paper_2606_06256_amd", "csrc")
KERNELS = {  # bench name -> (kernel symbol fragment, sources that build it)
    "decode_attn": ("decode_attn_kernel", ["common.hpp", "kernels.hpp", "decode.hip"]),
    "prefill_attn": ("prefill_kernel", ["common.hpp", "kernels.hpp", "prefill.hip"]),
    "token_mass": ("token_mass_kernel", ["common.hpp", "kernels.hpp", "mass.hip"]),
}
OP_OF_KERNEL = {"token_mass": "--op token_mass "}   # bench arguments that run the kernel
COPY_KERNEL = "copyBuffer"


def _code_text(src):
    """Source text without comments and with whitespace runs collapsed, so a
    comment edit does not void a recorded figure (string literals in kernel
    sources hold no comment markers)."""
    src = re.sub(r"/\*.*?\*/", " ", src, flags=re.S)
    src = re.sub(r"//[^\n]*", " ", src)
    return " ".join(src.split())


def kernel_sources_sha256(kname):
    h = hashlib.sha256()
    for f in KERNELS[kname][1]:
        with open(os.path.join(CSRC, f)) as fh:
            h.update(_code_text(fh.read()).encode())
    return h.hexdigest()


def recorded_traffic(kname, workload):
    """HBM bytes per launch of `kname` on `workload`, or None when no counter
    entry exists or the kernel has changed since the counters were taken."""
    try:
        with open(TRAFFIC_FILE) as f:
            d = json.load(f)
    except FileNotFoundError:
        return None
    e = d.get("kernels", {}).get(f"{kname}/{workload}")
    if not e or e.get("sources_sha256") != kernel_sources_sha256(kname):
        return None
    return e["hbm_bytes_per_launch"]


def pmc_mean_kib(out_dir, counter, fragment):
    """Mean per-dispatch value of `counter` (KiB) over dispatches of kernels
    whose name contains `fragment`, from a rocprofv3 --pmc csv output dir."""
    per_dispatch = {}
    for path in glob.glob(os.path.join(out_dir, "**", "*counter_collection.csv"), recursive=True):
        with open(path) as f:
            for row in csv.DictReader(f):
                if row.get("Counter_Name") != counter or fragment not in row.get("Kernel_Name", ""):
                    continue
                key = (path, row.get("Dispatch_Id"))
                per_dispatch[key] = per_dispatch.get(key, 0.0) + float(row["Counter_Value"])
    if not per_dispatch:
        raise RuntimeError(f"no {counter} rows for '{fragment}' under {out_dir}")
    return sum(per_dispatch.values()) / len(per_dispatch), len(per_dispatch)


def pmc_command(bench_args):
    """The counter runs behind an entry: one pass per counter, from /tmp on
    the GPU host, with the repository root in $R."""
    return ("cd /tmp && export TMPDIR=/tmp && rocprofv3 --pmc {FETCH_SIZE|WRITE_SIZE} "
            "--kernel-include-regex 'decode_attn|prefill_kernel|token_mass|copyBuffer' --output-format csv "
            f"-d <out_dir> -o run -- python3 $R/bench.py {bench_args}")


def write_traffic_entry(args):
    """Record one kernel's HBM traffic from four rocprofv3 --pmc output dirs."""
    from paper_2606_06256_amd import inputs as I
    copy_bytes = 1 << 30
    cf, _ = pmc_mean_kib(args.calib_fetch, "FETCH_SIZE", COPY_KERNEL)
    cw, _ = pmc_mean_kib(args.calib_write, "WRITE_SIZE", COPY_KERNEL)
    fetch_scale = copy_bytes / (cf * 1024)
    write_scale = copy_bytes / (cw * 1024)
    frag = KERNELS[args.kernel][0]
    kf, nf = pmc_mean_kib(args.fetch, "FETCH_SIZE", frag)
    kw, nw = pmc_mean_kib(args.write, "WRITE_SIZE", frag)
    read_b = kf * 1024 * fetch_scale
    write_b = kw * 1024 * write_scale
    try:
        with open(TRAFFIC_FILE) as f:
            d = json.load(f)
    except FileNotFoundError:
        d = {"kernels": {}}
    d["calibration"] = {"kernel": "__amd_rocclr_copyBuffer (torch device copy)",
                        "bytes_read": copy_bytes, "bytes_written": copy_bytes,
                        "FETCH_SIZE_kib": round(cf, 3), "WRITE_SIZE_kib": round(cw, 3),
                        "fetch_scale": round(fetch_scale, 6), "write_scale": round(write_scale, 6),
                        "command": pmc_command("--copy-calibration --steps 3")}
    name = I.config(args.workload).spec.name
    d["kernels"][f"{args.kernel}/{name}"] = {
        "kernel": frag, "workload": name,
        "FETCH_SIZE_kib": round(kf, 3), "WRITE_SIZE_kib": round(kw, 3), "dispatches": [nf, nw],
        "hbm_read_bytes": int(read_b), "hbm_write_bytes": int(write_b),
        "hbm_bytes_per_launch": int(read_b + write_b),
        "sources_sha256": kernel_sources_sha256(args.kernel),
        "command": pmc_command(OP_OF_KERNEL.get(args.kernel, "")
                               + f"--steps 5 --warmup 2 --no-cpu-baseline --no-sub-records "
                               f"--workload {args.workload}"),
    }
    os.makedirs(os.path.dirname(TRAFFIC_FILE), exist_ok=True)
    with open(TRAFFIC_FILE, "w") as f:
        json.dump(d, f, indent=1, sort_keys=True)
        f.write("\n")
    print(json.dumps(d["kernels"][f"{args.kernel}/{name}"]), flush=True)


def algorithmic_bytes(wl, sel_indptr, sel_pages):
    """Bytes the attention launch must move: selected valid K and V, Q, O,
    and the index reads (page id, page-table entry) of every selected page."""
    tokens = wl.attended_tokens(sel_indptr, sel_pages)
    kv = tokens * 2 * wl.D * 2
    rows = wl.total_q * wl.Hq
    qo = rows * wl.D * 2 * 2
    idx = int(sel_indptr[-1]) * 8
    return tokens, kv + qo + idx


def attention_flops(wl, sel_indptr, sel_pages):
    """2 * 2 * D flops per visible (query row, key) pair (QK^T and PV)."""
    tot = 0
    P = wl.P
    for u in range(wl.num_units):
        r = u // wl.Hkv
        L = int(wl.ctx_lens[r])
        nq = int(wl.q_indptr[r + 1] - wl.q_indptr[r])
        pg = sel_pages[sel_indptr[u]:sel_indptr[u + 1]].astype(np.int64)
        tok = (pg[:, None] * P + np.arange(P)[None, :]).reshape(-1)
        tok = tok[tok < L]
        for i in range(nq):
            tot += int(np.sum(tok <= L - nq + i)) * wl.G
    return 4 * wl.D * tot


def _cpu_worker(args):
    """One process of the CPU baseline: the fp64 oracle (select + attention)
    over its units, repeated until `seconds` have passed; single-threaded.
    Also returns each unit's first result (page list, O, LSE), which the
    parity entry of the bench line compares with the GPU's."""
    cfg, units, seconds = args
    from threadpoolctl import threadpool_limits

    from oracle import segpa_oracle as O
    from paper_2606_06256_amd import inputs as I
    wl = I.config(cfg)
    sp = wl.spec
    with threadpool_limits(limits=1):
        q64 = wl.q("cpu").double().numpy()
        kv = {}
        for u in units:                     # input generation is not timed
            K, V = wl.unit_kv(*divmod(u, wl.Hkv), "cpu")
            kv[u] = (K.double().numpy(), V.double().numpy())
        tokens = 0
        done = 0
        first = {}
        t0 = time.perf_counter()
        while time.perf_counter() - t0 < seconds:
            for u in units:
                K, V = kv[u]
                sel = O.select(sp.sel_mode, wl.ctx_lens, wl.q_indptr, wl.Hq, wl.Hkv, wl.P,
                               budgets=wl.budgets, forced_head=sp.forced_head,
                               forced_tail=sp.forced_tail, seed=sp.sel_seed,
                               head_policy=wl.head_policy, n_sink=sp.n_sink, window=sp.window,
                               q=q64, kv_of_unit=lambda rr, gg: (K, V), units=[u])[u]
                res = O.forward_unit(q64, wl.q_indptr, wl.ctx_lens, wl.Hq, wl.Hkv, wl.P, u, sel, K, V)
                if u not in first:
                    first[u] = ([int(p) for p in sel], res[0], res[1])
                L = int(wl.ctx_lens[u // wl.Hkv])
                tokens += int(sum(min(wl.P, L - p * wl.P) for p in sel))
                done += 1
        return tokens, time.perf_counter() - t0, done, first


def cpu_baseline(cfg, wl, seconds=12.0, max_procs=16):
    """fp64 oracle (select + attention) on a sample of the step's units, in a
    pool of single-threaded processes over the host cores available to this
    process (at most max_procs), all timed over the same interval."""
    import multiprocessing as mp
    cores = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else os.cpu_count()
    procs = max(1, min(max_procs, cores))
    U = wl.num_units
    n_sample = min(U, 2 * procs)
    units = sorted({int(x) for x in np.linspace(0, U - 1, n_sample)})
    shares = [units[i::procs] for i in range(procs)]
    shares = [sh for sh in shares if sh]
    ctx = mp.get_context("spawn")
    with ctx.Pool(len(shares)) as pool:
        res = pool.map(_cpu_worker, [(cfg, sh, seconds) for sh in shares])
    tokens = sum(r[0] for r in res)
    wall = max(r[1] for r in res)
    done = sum(r[2] for r in res)
    first = {u: v for r in res for u, v in r[3].items()}
    return {"value": tokens / wall, "unit": "tokens/s", "cores": len(shares), "kind": "oracle",
            "sample": f"{len(units)} of {U} (request, KV head) units of one step, {done} unit "
                      f"evaluations in {wall:.1f} s by {len(shares)} single-threaded fp64 numpy "
                      f"processes (host cores available: {cores})"}, first


def parity_of_sample(wl, first, ind, pages, out, lse):
    """The GPU's selection and outputs of the last timed step against the
    oracle's results for the CPU baseline's sampled units."""
    G = wl.G
    mism = 0
    max_abs = 0.0
    sum_abs = 0.0
    n_el = 0
    lse_max = 0.0
    for u, (sel, Oo, LSE) in first.items():
        got = [int(p) for p in pages[int(ind[u]):int(ind[u + 1])]]
        mism += got != sel
        r, g = divmod(u, wl.Hkv)
        q0, q1 = int(wl.q_indptr[r]), int(wl.q_indptr[r + 1])
        if q1 == q0:
            continue
        d = np.abs(out[q0:q1, g * G:(g + 1) * G].astype(np.float64) - Oo)
        max_abs = max(max_abs, float(d.max()))
        sum_abs += float(d.sum())
        n_el += d.size
        a, b = lse[q0:q1, g * G:(g + 1) * G].astype(np.float64), LSE
        fin = np.isfinite(a) & np.isfinite(b)
        if fin.any():
            lse_max = max(lse_max, float(np.abs(a - b)[fin].max()))
    return {"units": len(first), "selection_mismatches": int(mism), "o_max_abs": max_abs,
            "o_mean_abs": sum_abs / max(1, n_el), "lse_max_abs": lse_max,
            "compared": "the last timed step's page lists, O (bf16) and LSE of the sampled "
                        "units against the fp64 oracle"}


def device_copy_gbs(torch, nbytes=1 << 30, reps=5):
    """Bytes moved per second (read + write) by a plain 1 GiB device-to-device
    copy on this machine, median of 5: a practical HBM ceiling the decode kernel is
    compared with beside the 8 TB/s specification."""
    src = torch.ones(nbytes, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    ts = []
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        dst.copy_(src)
        e1.record()
        torch.cuda.synchronize()
        ts.append(e0.elapsed_time(e1))
    del src, dst
    return 2 * nbytes / (float(np.median(ts)) * 1e-3) / 1e9


def cold_steps(dw, torch, binding, kname, n=9, evict_bytes=1 << 30):
    """Median step and dominant-kernel time with the caches cold: each step is
    queued right behind a read of 1 GiB, more than the L2s and the 256 MB
    Infinity Cache hold (no host synchronisation in between, so no launch gap
    enters the step). The buffer is read, not written: evicting with writes
    leaves dirty lines whose write-back then competes with the measured
    kernel."""
    scratch = torch.ones(evict_bytes // 4, dtype=torch.int32, device="cuda")
    for _ in range(2):                        # its own dirty lines leave the caches first
        scratch.sum()
    dw.step()
    torch.cuda.synchronize()
    steps, kern = [], {}
    for _ in range(n):                        # step time (no per-launch events)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        scratch.sum()
        e0.record()
        dw.step()
        e1.record()
        torch.cuda.synchronize()
        steps.append(e0.elapsed_time(e1))
    for _ in range(n):                        # per-kernel times
        binding.profile_begin()
        scratch.sum()
        dw.step()
        torch.cuda.synchronize()
        for k, (c, t) in binding.profile_end().items():
            kern.setdefault(k, []).append(t / c)
    del scratch
    out = {"evict_read_bytes": evict_bytes, "steps": n, "median_step_ms": round(float(np.median(steps)), 5)}
    for k, v in kern.items():
        out[f"median_{k}_ms"] = round(float(np.median(v)), 5)
    return out


def bench_rope_align(args, wl):
    """RoPE alignment (Section 4.2) of every key page of the workload's pool,
    each page by a seeded shift: one read and one write of the K pool."""
    import torch

    from paper_2606_06256_amd import binding, build_lib
    from paper_2606_06256_amd.device import DeviceWorkload
    if not os.path.exists(binding.LIB_PATH):
        build_lib.build()
    if not torch.cuda.is_available():
        raise RuntimeError("bench.py needs a GPU")
    torch.cuda.set_device(0)
    dw = DeviceWorkload(wl)
    n = int(dw.k_pool.shape[0])
    pages = torch.arange(n, dtype=torch.int32, device="cuda")
    g = torch.Generator().manual_seed(7)
    deltas = torch.randint(-131072, 131072, (n,), generator=g, dtype=torch.int32).cuda()
    run = lambda: binding.seg_paged_attn_rope_align(dw.dims, dw.k_pool, pages, deltas, 10000.0)
    for _ in range(args.warmup):
        run()
    torch.cuda.synchronize()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(args.steps):
        run()
    stop.record()
    torch.cuda.synchronize()
    ms = start.elapsed_time(stop) / args.steps
    binding.profile_begin()
    for _ in range(args.steps):
        run()
    torch.cuda.synchronize()
    prof = binding.profile_end()
    nl, tl = prof["rope_align"]
    launch_ms = tl / nl
    nbytes = 2 * n * wl.P * wl.D * 2          # every key page read and written once
    gbs = nbytes / (launch_ms * 1e-3) / 1e9
    # the same bytes moved by a plain device copy (read + write), for scale
    src = dw.k_pool.view(-1)
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    c0.record()
    for _ in range(args.steps):
        dst.copy_(src)
    c1.record()
    torch.cuda.synchronize()
    copy_gbs = nbytes / (c0.elapsed_time(c1) / args.steps * 1e-3) / 1e9
    del dst
    print(json.dumps({
        "metric": "RoPE alignment of cached key pages: HBM GB/s", "value": round(nbytes / (ms * 1e-3) / 1e9, 1),
        "unit": "GB/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms, 5), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f64", "data": "synthetic",
        "config": {"workload": wl.spec.name + " key pool", "pages": n, "page_size": wl.P, "head_dim": wl.D,
                   "bytes_per_launch": nbytes, "device_copy_gbs_same_bytes": round(copy_gbs, 1)},
        "roofline": {"kernel": "rope_align", "bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(gbs / HBM_PEAK_GBS, 4), "traffic": None,
                     "launch_ms": round(launch_ms, 5)},
    }), flush=True)


def bench_append(args, wl):
    """Appending each request's n_q new tokens (the workload's query chunk, at
    the end of its context) into their pages, with the key-sum refresh of
    every page written."""
    import torch

    from paper_2606_06256_amd import binding, build_lib
    from paper_2606_06256_amd.device import DeviceWorkload
    if not os.path.exists(binding.LIB_PATH):
        build_lib.build()
    if not torch.cuda.is_available():
        raise RuntimeError("bench.py needs a GPU")
    torch.cuda.set_device(0)
    dw = DeviceWorkload(wl)
    nq = np.diff(wl.q_indptr).astype(np.int64)
    L0 = (wl.ctx_lens - nq).astype(np.int32)
    n_new = int(nq.sum())
    g = torch.Generator().manual_seed(11)
    kn = torch.randn(n_new, wl.Hkv, wl.D, generator=g).to(torch.bfloat16).cuda()
    vn = torch.randn(n_new, wl.Hkv, wl.D, generator=g).to(torch.bfloat16).cuda()
    ks = torch.zeros(wl.num_phys, wl.D, dtype=torch.float32, device="cuda")
    l0 = torch.from_numpy(L0).cuda()
    ind = torch.from_numpy(wl.q_indptr.astype(np.int32)).cuda()
    run = lambda: binding.seg_paged_attn_append(dw.dims, l0, ind, kn, vn, dw.seg_table, dw.page_table,
                                                dw.k_pool, dw.v_pool, ks)
    for _ in range(args.warmup):
        run()
    torch.cuda.synchronize()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(args.steps):
        run()
    stop.record()
    torch.cuda.synchronize()
    ms = start.elapsed_time(stop) / args.steps
    # bytes: new K and V read and written; every written page's valid keys
    # read back for its sum, and the sum written
    touched_tokens = 0
    touched_pages = 0
    for r in range(wl.B):
        if nq[r] == 0:
            continue
        j0, j1 = int(L0[r]) // wl.P, (int(wl.ctx_lens[r]) - 1) // wl.P
        for j in range(j0, j1 + 1):
            touched_pages += wl.Hkv
            touched_tokens += wl.Hkv * min(wl.P, int(wl.ctx_lens[r]) - j * wl.P)
    nbytes = 4 * n_new * wl.Hkv * wl.D * 2 + touched_tokens * wl.D * 2 + touched_pages * wl.D * 4
    gbs = nbytes / (ms * 1e-3) / 1e9
    print(json.dumps({
        "metric": "KV append with key-sum refresh: HBM GB/s", "value": round(gbs, 1), "unit": "GB/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": wl.spec.name + " chunk append", "new_tokens": n_new, "kv_heads": wl.Hkv,
                   "pages_touched": touched_pages, "bytes_per_call": nbytes},
        "roofline": {"kernel": "append + key_refresh", "bound": "hbm", "achieved": round(gbs, 1),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(gbs / HBM_PEAK_GBS, 4),
                     "traffic": None},
    }), flush=True)


def bench_token_mass(args, wl, tau=0.2, recent=128):
    """The attention-mass token selection after a chunked-prefill forward:
    the probability pass (token_mass) and the per-request selection
    (select_tokens), at the sparse-FFN setting the paper gives for Qwen3-32B
    (mass threshold 0.2, the most recent 128 tokens always kept)."""
    import torch

    from paper_2606_06256_amd import binding, build_lib
    from paper_2606_06256_amd.device import DeviceWorkload
    if not os.path.exists(binding.LIB_PATH):
        build_lib.build()
    if not torch.cuda.is_available():
        raise RuntimeError("bench.py needs a GPU")
    torch.cuda.set_device(0)
    dw = DeviceWorkload(wl)
    if wl.spec.sel_mode == 3:
        dw.summary()
    dw.select()
    dw.fwd()                                  # the lse the masses are normalised by

    def run():
        dw.token_mass()
        dw.select_tokens(tau, recent)
    for _ in range(args.warmup):
        run()
    torch.cuda.synchronize()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(args.steps):
        run()
    stop.record()
    torch.cuda.synchronize()
    ms = start.elapsed_time(stop) / args.steps
    binding.profile_begin()
    for _ in range(args.steps):
        run()
    torch.cuda.synchronize()
    prof = binding.profile_end()
    n_m, t_m = prof["token_mass"]
    n_s, t_s = prof["select_tokens"]
    mass_ms, sel_ms = t_m / n_m, t_s / n_s
    # algorithmic bytes of token_mass: every chunk row of q and its lse read
    # once, the chunk's selected keys read once, the masses written; flops:
    # 2 D per visible (row, chunk key) pair
    ind, pages = dw.selection()
    nq = np.diff(wl.q_indptr).astype(np.int64)
    chunk_keys, pairs = 0, 0
    for u in range(wl.num_units):
        r = u // wl.Hkv
        L, n = int(wl.ctx_lens[r]), int(nq[r])
        pg = set(pages[ind[u]:ind[u + 1]].tolist())
        ks = [k for k in range(n) if (L - n + k) >= 0 and (L - n + k) // wl.P in pg]
        chunk_keys += len(ks)
        pairs += wl.G * sum(n - k for k in ks)
    abytes = wl.total_q * wl.Hq * (wl.D * 2 + 4) + chunk_keys * wl.D * 2 + wl.total_q * wl.Hkv * 4
    flops = 2 * wl.D * pairs
    gbs = abytes / (mass_ms * 1e-3) / 1e9
    tfs = flops / (mass_ms * 1e-3) / 1e12
    keep_frac = float(dw.keep_count.sum().item()) / max(1, wl.total_q)
    print(json.dumps({
        "metric": "attention-mass token selection: chunk tokens/s", "value": round(wl.total_q / (ms * 1e-3), 1),
        "unit": "tokens/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms, 5), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": wl.spec.name + " token selection", "chunk_tokens": wl.total_q,
                   "q_heads": wl.Hq, "kv_heads": wl.Hkv, "tau": tau, "recent": recent,
                   "kept_fraction": round(keep_frac, 4), "token_mass_ms": round(mass_ms, 5),
                   "select_tokens_ms": round(sel_ms, 5), "token_mass_tflops": round(tfs, 2),
                   "token_mass_mfma_frac": round(tfs / MFMA_BF16_PEAK_TFLOPS, 4)},
        "roofline": {"kernel": "token_mass", "bound": "hbm", "achieved": round(gbs, 1),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(gbs / HBM_PEAK_GBS, 4),
                     "traffic": recorded_traffic("token_mass", wl.spec.name), "bytes_per_launch": abytes,
                     "flops_per_launch": flops, "launch_ms": round(mass_ms, 5)},
    }), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", type=int, default=None,
                    help="named workload 1..10 (default 3, the varlen sparse decode; 9 for --op token_mass)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--sub-records", default="2,4,5",
                    help="workloads also measured in the same run (step time, dominant-kernel "
                         "roofline), reported under config.sub_records")
    ap.add_argument("--no-sub-records", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 1 GiB device-to-device copy (scale for HBM byte counters)")
    ap.add_argument("--op", choices=["step", "rope_align", "append", "token_mass"], default="step",
                    help="step: the hot path (default); rope_align: RoPE alignment of every "
                         "key page of the workload's pool; append: writing each request's "
                         "query chunk of new tokens into its pages with the key-sum refresh; "
                         "token_mass: attention-mass token selection after a chunked prefill")
    ap.add_argument("--record-traffic", choices=sorted(KERNELS),
                    help="write the kernel's HBM traffic entry from rocprofv3 --pmc output dirs "
                         "(--fetch, --write, --calib-fetch, --calib-write); runs nothing on the GPU")
    ap.add_argument("--fetch")
    ap.add_argument("--write")
    ap.add_argument("--calib-fetch")
    ap.add_argument("--calib-write")
    args = ap.parse_args()
    if args.workload is None:
        args.workload = 9 if args.op == "token_mass" else 3
    if args.record_traffic:
        args.kernel = args.record_traffic
        write_traffic_entry(args)
        return
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    if args.copy_calibration:
        import torch
        n = 1 << 30
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(args.steps):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes_read": n, "bytes_written": n,
                          "launches": args.steps}), flush=True)
        return

    from paper_2606_06256_amd import inputs as I
    wl = I.config(args.workload)
    if args.op == "rope_align":
        bench_rope_align(args, wl)
        return
    if args.op == "append":
        bench_append(args, wl)
        return
    if args.op == "token_mass":
        bench_token_mass(args, wl)
        return

    # CPU baseline first, before anything initialises the GPU (a failure there
    # is reported in the line rather than losing the GPU measurement)
    cpu, first = None, None
    if not args.no_cpu_baseline:
        try:
            cpu, first = cpu_baseline(args.workload, wl)
        except Exception as e:  # noqa: BLE001
            cpu = {"kind": "oracle", "error": f"{type(e).__name__}: {e}"}

    import torch
    from paper_2606_06256_amd import binding, build_lib
    if not os.path.exists(binding.LIB_PATH):
        build_lib.build()
    if not torch.cuda.is_available():
        raise RuntimeError("bench.py needs a GPU")
    torch.cuda.set_device(0)

    head = measure_step(wl, args, torch, binding, cold=True, with_copy=True, check=first)
    if cpu is not None and first:
        cpu["parity"] = head.pop("parity")
    subs = []
    if not args.no_sub_records:
        for i in [int(x) for x in args.sub_records.split(",") if x.strip()]:
            if i == args.workload:
                continue
            torch.cuda.empty_cache()
            try:
                r = measure_step(I.config(i), args, torch, binding, cold=False, with_copy=False)
            except Exception as e:  # noqa: BLE001  (the headline stands on its own)
                subs.append({"workload": I.config_spec(i).name, "error": f"{type(e).__name__}: {e}"})
                continue
            subs.append({k: r[k] for k in ("ms_per_step", "value", "unit")} |
                        {"workload": r["config"]["workload"], "roofline": r["roofline"],
                         "kernels": r["config"]["kernels"],
                         "attended_kv_tokens_per_step": r["config"]["attended_kv_tokens_per_step"]} |
                        ({"page_summary_ms": r["config"]["page_summary_ms"]}
                         if "page_summary_ms" in r["config"] else {}))
    line = {
        "metric": METRIC,
        "value": head["value"],
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": head["config"],
        "roofline": head["roofline"],
        "cpu_baseline": cpu,
    }
    if subs:
        line["config"]["sub_records"] = subs
    print(json.dumps(line), flush=True)


def measure_step(wl, args, torch, binding, *, cold, with_copy, check=None):
    """Warm-up, then exactly args.steps timed steps of `wl` (inputs resident in
    HBM), then the same number of steps with per-kernel dispatch timing.
    With `check` (the oracle's results for some units), the timed steps'
    outputs are compared with it."""
    from paper_2606_06256_amd import inputs as I
    from paper_2606_06256_amd.device import DeviceWorkload

    dw = DeviceWorkload(wl)
    summary_ms = None
    if wl.spec.sel_mode == I.SEL_TOPK_MEANKEY:
        # page key sums are built once when pages are written; timed on their own
        dw.summary()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(3):
            dw.summary()
        e1.record()
        torch.cuda.synchronize()
        summary_ms = e0.elapsed_time(e1) / 3

    for _ in range(args.warmup):
        dw.step()
    torch.cuda.synchronize()
    ind, pages = dw.selection()
    tokens, abytes = algorithmic_bytes(wl, ind, pages)

    # timed region: exactly K steps
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for _ in range(args.steps):
        dw.step()
    stop.record()
    torch.cuda.synchronize()
    ms_per_step = start.elapsed_time(stop) / args.steps
    parity = None
    if check:
        parity = parity_of_sample(wl, check, *dw.selection(), dw.out.float().cpu().numpy(),
                                  dw.lse.cpu().numpy())

    # per-kernel launch times: HIP events attached to each kernel dispatch on
    # the stream it is launched on (the kernel's own start and end)
    binding.profile_begin()
    for _ in range(args.steps):
        dw.step()
    torch.cuda.synchronize()
    prof = binding.profile_end()
    prefill = "prefill_attn" in prof
    kname = "prefill_attn" if prefill else "decode_attn"
    n_attn, ms_attn = prof[kname]
    attn_ms = ms_attn / n_attn
    achieved = abytes / (attn_ms * 1e-3) / 1e9
    traffic = recorded_traffic(kname, wl.spec.name)
    if prefill:
        # the chunk's attention is a dense contraction: matrix-core bound
        flops = attention_flops(wl, ind, pages)
        tf = flops / (attn_ms * 1e-3) / 1e12
        roofline = {"kernel": kname, "bound": "mfma", "achieved": round(tf, 2),
                    "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                    "frac": round(tf / MFMA_BF16_PEAK_TFLOPS, 4), "traffic": traffic,
                    "flops_per_launch": flops, "launch_ms": round(attn_ms, 5),
                    "hbm_gbs": round(achieved, 1)}
    else:
        roofline = {"kernel": kname, "bound": "hbm", "achieved": round(achieved, 1),
                    "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                    "traffic": traffic, "bytes_per_launch": abytes, "launch_ms": round(attn_ms, 5)}
    roofline["launch_timing"] = "HIP events attached to the kernel dispatch"
    if traffic is not None:
        roofline["traffic_over_algorithmic_bytes"] = round(traffic / abytes, 4)
        roofline["traffic_source"] = ("recorded rocprofv3 FETCH_SIZE/WRITE_SIZE passes "
                                      "(profiles/hbm_traffic.json), valid for the current kernel sources")
    if with_copy and not prefill:
        copy = device_copy_gbs(torch)
        roofline["measured_device_copy_gbs"] = round(copy, 1)
        roofline["frac_of_measured_device_copy"] = round(achieved / copy, 4)
    kernels = {k: {"launches": n, "mean_ms": round(t / n, 5)} for k, (n, t) in prof.items()}
    config = {"workload": wl.spec.name, "description": wl.spec.description,
              "requests": wl.B, "q_heads": wl.Hq, "kv_heads": wl.Hkv, "head_dim": wl.D,
              "page_size": wl.P, "segment_tokens": wl.spec.seg_tokens,
              "attended_kv_tokens_per_step": tokens,
              "step_gbs": round(abytes / (ms_per_step * 1e-3) / 1e9, 1),
              "kernels": kernels}
    if cold:
        config["cold_cache"] = cold_steps(dw, torch, binding, kname)
    if summary_ms is not None:
        config["page_summary_ms"] = round(summary_ms, 4)
    del dw
    out = {"value": round(tokens / (ms_per_step * 1e-3), 1), "unit": "tokens/s",
           "ms_per_step": round(ms_per_step, 5), "config": config, "roofline": roofline}
    if check:
        out["parity"] = parity
    return out

if __name__ == "__main__":
    main()
