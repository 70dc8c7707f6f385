#!/usr/bin/env python3
"""SPLA decode-step benchmark on one MI355X.

    python bench.py [--steps K] [--warmup W] [--config 3] [--replicas R]

A step is one spla_decode call over the whole batch of the workload (for
the appending workload, one spla_step): block scoring over every block's
statistics, top-k selection, the fused exact + selected-linear pass over the
selected blocks, and the merge. The cache is filled once through spla_append
from the seeded synthetic generators (untimed). R identical copies of the
cache are decoded in rotation so that the 256 MB last-level cache cannot
serve a step from the previous visit; inputs are resident in HBM when the
timed region starts.

Prints one JSON line: whole-step throughput as algorithmic HBM bytes per
second (value, GB/s), latency (ms_per_step), the roofline of the dominant
kernel (the single-launch decode kernel at this shape: the timed region over
the launches, with its counter traffic when the committed counter summary
matches the kernel sources) and the fp64 CPU oracle timed on a bounded
sample. Three more objects measure the same workload with the library's
options: strided selection windows (C = 32, s = 16; roofline of its scoring
kernel), a paged K/V pool behind a shuffled block table, and a causal
prefill of 16 positions per sequence. --no-strided skips them.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "SPLA decode-step latency (µs) + achieved HBM GB/s vs peak at 128K ctx"
PEAK_HBM_GBS = 8000.0
KERNEL_SOURCES = sorted("paper_2601_22379_amd/csrc/" + f
                        for f in os.listdir(os.path.join(ROOT, "paper_2601_22379_amd", "csrc"))
                        if f.endswith((".hip", ".h")))


STRIDED_TAG = "_strided_c32_s16"


def traffic_file(kernel, variant=""):
    return os.path.join(ROOT, "profiles", f"{kernel}{variant}_kernel_traffic.json")


def traffic_of(kernel, workload, variant=""):
    """Calibrated HBM bytes per launch of `kernel` from its committed counter
    summary, or None when there is none or the kernel sources changed since."""
    tfile = traffic_file(kernel, variant)
    if not os.path.exists(tfile):
        return None
    with open(tfile) as f:
        tr = json.load(f)
    if tr.get("source_sha") == source_hash(KERNEL_SOURCES) and tr.get("workload") == workload:
        return tr["hbm_bytes_per_launch"]
    return None


def copy_calibration(dev):
    """A plain elementwise kernel over 1 GiB (1 GiB read, 1 GiB written): the
    reference the counter passes are scaled by."""
    import torch

    n = 1 << 28
    src = torch.ones(n, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    torch.mul(src, 1.0, out=dst)
    torch.cuda.synchronize()
    log("copy calibration: 1 GiB read + 1 GiB written by one elementwise kernel")


def dominant_bytes(w, ab, kernel):
    """Algorithmic bytes one launch of the dominant kernel moves: the whole
    decode (everything but the append) for the single-launch kernel, the
    statistics plus the queries for the scoring kernel, the selected rows,
    the state and the queries for the sparse pass."""
    q = w.batch * w.n_q_heads * w.head_dim * (4 if w.dtype == "f32" else 2)
    if kernel == "decode":
        return ab["total"] - ab["append"]
    if kernel == "sparse":  # selected rows, the state (written back too by a step), queries
        return ab["selected_kv"] + ab["state"] * (2 if w.appends_per_step else 1) + q
    return ab["stats"] + q



def log(msg):
    sys.stderr.write(f"[bench {time.strftime('%H:%M:%S')}] {msg}\n")
    sys.stderr.flush()


def source_hash(paths):
    h = hashlib.sha256()
    for p in paths:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def shuffled_block_table(w, seed=7):
    """A paged pool of batch * nb_cap + 64 pages and a seeded shuffle of it
    as the block table (int32 [batch][nb_cap])."""
    import numpy as np

    nb = w.capacity // w.block_size
    pages = w.batch * nb + 64
    rng = np.random.default_rng([seed, w.code])
    return pages, rng.permutation(pages)[:w.batch * nb].reshape(w.batch, nb).astype(np.int32)


def build_workload(w, replicas, dev, sel_window=0, sel_stride=0, paged=False):
    import torch

    from paper_2601_22379_amd import spla
    import spla_inputs as si

    pages, table = shuffled_block_table(w) if paged else (0, None)
    cfg = spla.make_config(w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.block_size,
                           w.top_k, w.capacity, w.dtype, n_sink=w.n_sink, n_local=w.n_local,
                           sel_window=sel_window, sel_stride=sel_stride, kv_pages=pages)
    tab = None if table is None else torch.from_numpy(table).to(dev)
    first = spla.SplaCache(cfg, dev, block_table=tab)
    dt = torch.float32 if w.dtype == "f32" else torch.bfloat16
    lens = [w.prefill_length(b) for b in range(w.batch)]
    per_tok = w.batch * w.n_kv_heads * w.head_dim * 8
    T = int(min(w.capacity, max(256, 1 << (int((1 << 29) // per_tok).bit_length() - 1))))
    t0 = time.time()
    for a in range(0, max(lens), T):
        K, V, n = si.gen_kv_slab(w, a, min(a + T, max(lens)), lengths=lens, threads=16)
        first.append(torch.from_numpy(K).to(dt).to(dev), torch.from_numpy(V).to(dt).to(dev),
                     torch.from_numpy(n).to(dev))
    torch.cuda.synchronize()
    log(f"filled {w.name} in {time.time() - t0:.1f}s")
    caches = [first]
    for _ in range(replicas - 1):
        c = spla.SplaCache(cfg, dev, block_table=tab)
        for name in ("k", "v", "stats", "state", "norm", "seq_lens"):
            getattr(c, name).copy_(getattr(first, name))
        caches.append(c)
    torch.cuda.synchronize()
    return cfg, caches


def strided_leg(w, R, dev, qs, gamma, outs, sels, K, W, C=32, s=16, paged=False):
    """The same decode with strided selection windows (C tokens every s,
    max-pooled into blocks; the paper's C = 32, s = 16), or (C = s = B,
    paged) with the K/V caches in a paged pool behind a shuffled block
    table: a cache of its own, K timed steps, then the same steps with every
    phase bracketed by HIP events. Returns a dict for the JSON line; the
    scoring kernel, which streams the statistics, is the dominant one."""
    import numpy as np
    import torch

    from paper_2601_22379_amd import spla
    import spla_inputs as si

    win = (C, s) != (w.block_size, w.block_size)
    cfg, caches = build_workload(w, R, dev, C if win else 0, s if win else 0, paged)

    def one(i, events=None):
        r = i % R
        return caches[r].decode(qs[i % qs.shape[0]], gamma, outs[r], sels[r], events)

    for i in range(W):
        one(i)
    t_a = torch.cuda.Event(enable_timing=True)
    t_b = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_a.record()
    for i in range(K):
        one(W + i)
    t_b.record()
    torch.cuda.synchronize()
    lat_us = t_a.elapsed_time(t_b) / K * 1e3
    names = spla.decode_phases(cfg)
    ev = [spla.make_events(names) for _ in range(K)]
    for i in range(K):
        one(W + K + i, ev[i][0])
    torch.cuda.synchronize()
    phases = {n: float(np.mean([e[1][n][0].elapsed_time(e[1][n][1]) for e in ev])) * 1e3
              for n in names}
    lens = caches[0].seq_lens.cpu().numpy()
    sel_np = sels[0].cpu().numpy()
    sel_counts = [[sum(min(w.block_size, int(lens[b]) - int(i) * w.block_size)
                       for i in sel_np[b, h] if i >= 0) for h in range(w.n_kv_heads)]
                  for b in range(w.batch)]
    ab = si.algorithmic_bytes(w, sel_counts)
    if win:
        ab["stats"] = sum(-(-int(L) // s) for L in lens) * w.n_kv_heads * 2 * w.head_dim * 4
    ab["total"] = ab["q_out"] + ab["stats"] + ab["selected_kv"] + ab["state"] + ab["append"]
    # dominant kernel: the single-launch decode kernel where the variant runs
    # as one (its average launch: the timed region over the launches), else
    # the statistics scan
    dom = "decode" if names == ["decode"] else "score"
    sb = dominant_bytes(w, ab, dom)
    dom_us = lat_us if dom == "decode" else phases["score"]
    del caches
    torch.cuda.synchronize()
    log(f"{'paged KV' if paged else 'strided selection'} (C={C}, s={s}): {lat_us:.2f} us/step, "
        "phases us: " + ", ".join(f"{k}={v:.2f}" for k, v in phases.items()))
    head = {"kv_pages": int(cfg.kv_pages)} if paged else {"window": C, "stride": s}
    # counter passes exist for the strided variant's scoring kernel only
    traffic = None if paged else traffic_of(dom, w.name, STRIDED_TAG)
    return {**head, "latency_us": round(lat_us, 3),
            "value": round(ab["total"] / (lat_us * 1e-6) / 1e9, 1), "unit": "GB/s",
            "algorithmic_bytes": ab, "phases_us": {k: round(v, 3) for k, v in phases.items()},
            "roofline": {"kernel": dom, "bound": "hbm",
                         "achieved": round(sb / (dom_us * 1e-6) / 1e9, 1),
                         "peak": PEAK_HBM_GBS, "unit": "GB/s",
                         "frac": round(sb / (dom_us * 1e-6) / 1e9 / PEAK_HBM_GBS, 4),
                         "traffic": traffic,
                         "algorithmic_bytes_per_launch": sb,
                         "avg_launch_us": round(dom_us, 3),
                         "avg_launch_method": ("timed region / launches" if dom == "decode"
                                               else "per-launch events")}}


def prefill_leg(w, dev, K, T=32):
    """Causal prefill (spla_prefill) of T tokens per sequence at the
    workload's context: the cache is filled to capacity - T (2 K + 1) tokens,
    then K timed calls each prefill T positions (one chunk of the chunked
    kernels for bf16, G <= 8). Returns a dict for the JSON line: latency per
    call and per position, tokens per second over the whole batch, and the
    bytes the chunk's kernels must move (the statistics once per chunk, every
    query's selected K/V rows, S_bar read and written, the new rows)."""
    import numpy as np
    import torch

    from paper_2601_22379_amd import spla
    import spla_inputs as si

    lens = [w.capacity - T * (2 * K + 1)] * w.batch  # room for every call below
    cfg = spla.make_config(w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.block_size,
                           w.top_k, w.capacity, w.dtype, n_sink=w.n_sink, n_local=w.n_local)
    cache = spla.SplaCache(cfg, dev)
    dt = torch.float32 if w.dtype == "f32" else torch.bfloat16
    per_tok = w.batch * w.n_kv_heads * w.head_dim * 8
    S = int(min(w.capacity, max(256, 1 << (int((1 << 29) // per_tok).bit_length() - 1))))
    for a in range(0, lens[0], S):
        Kt, Vt, n = si.gen_kv_slab(w, a, min(a + S, lens[0]), lengths=lens, threads=16)
        cache.append(torch.from_numpy(Kt).to(dt).to(dev), torch.from_numpy(Vt).to(dt).to(dev),
                     torch.from_numpy(n).to(dev))
    rng = np.random.default_rng([w.code, 5])
    kn = torch.from_numpy(rng.standard_normal((T, w.batch, w.n_kv_heads, w.head_dim))
                          .astype(np.float32)).to(dt).to(dev)
    vn = torch.from_numpy(rng.standard_normal(kn.shape).astype(np.float32)).to(dt).to(dev)
    q = torch.from_numpy(np.stack([si.gen_q_batch(w, t) for t in range(T)])).to(dt).to(dev)
    gamma = torch.from_numpy(si.gen_gamma(w)).to(dev)
    out, sel = cache.prefill(kn, vn, q, gamma)  # warm-up call (T positions)
    torch.cuda.synchronize()
    a = torch.cuda.Event(enable_timing=True)
    b = torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(K):
        cache.prefill(kn, vn, q, gamma, out, sel)
    b.record()
    torch.cuda.synchronize()
    us = a.elapsed_time(b) / K * 1e3
    # the same calls with every phase bracketed by events (recorded by the
    # library on its stream): the split between the chunk's kernels
    names = ["append", "linear", "score", "select", "sparse", "merge"]
    evs = [spla.make_events(names) for _ in range(K)]
    torch.cuda.synchronize()
    for i in range(K):
        cache.prefill(kn, vn, q, gamma, out, sel, events=evs[i][0])
    torch.cuda.synchronize()
    phases = {n: float(np.mean([e[1][n][0].elapsed_time(e[1][n][1]) for e in evs])) * 1e3
              for n in names}
    assert cache.device_errors() == 0
    e = 4 if w.dtype == "f32" else 2
    d, B = w.head_dim, w.block_size
    L_end = int(cache.seq_lens[0].item())
    nb = -(-L_end // B)
    sel_np = sel.cpu().numpy()
    sel_tok = int(sum(min(B, L_end - int(i) * B) for i in sel_np.reshape(-1) if i >= 0))
    bh = w.batch * w.n_kv_heads
    ab = {"stats": bh * nb * 2 * d * 4, "selected_kv_all_queries": sel_tok * d * 2 * e,
          "state_rw": 2 * bh * (d * d + d) * 4, "new_rows": bh * T * 2 * d * e,
          "q_out": 2 * T * w.batch * w.n_q_heads * d * e}
    ab["total"] = sum(ab.values())
    tok_s = w.batch * T / (us * 1e-6)
    # dominant kernel: the per-query fused sparse pass, whose bytes are every
    # query's selected K/V rows plus its query rows
    sp_bytes = ab["selected_kv_all_queries"] + T * w.batch * w.n_q_heads * d * e
    sp_ach = sp_bytes / (phases["sparse"] * 1e-6) / 1e9
    log(f"prefill: {T} positions in {us:.1f} us ({us / T:.2f} us per position, "
        f"{tok_s / 1e6:.2f} M tokens/s) from {lens[0]} tokens; phases us: "
        + ", ".join(f"{k}={v:.1f}" for k, v in phases.items()))
    return {"tokens_per_call": T, "calls": K, "context_start": lens[0],
            "latency_us_per_call": round(us, 2), "latency_us_per_position": round(us / T, 3),
            "tokens_per_s": round(tok_s, 1), "algorithmic_bytes_per_call": ab,
            "achieved_GBs_per_call": round(ab["total"] / (us * 1e-6) / 1e9, 1),
            "phases_us": {k: round(v, 2) for k, v in phases.items()},
            "roofline": {"kernel": "prefill_sparse", "bound": "hbm", "achieved": round(sp_ach, 1),
                         "peak": PEAK_HBM_GBS, "unit": "GB/s",
                         "frac": round(sp_ach / PEAK_HBM_GBS, 4),
                         "algorithmic_bytes_per_launch": sp_bytes,
                         "avg_launch_us": round(phases["sparse"], 3),
                         "avg_launch_method": "per-launch events"},
            "method": "chunked prefill (spla_prefill, one chunk of T positions per call)"}


def append_leg(w, dev, K, T=16384):
    """Bulk append (spla_append) of T tokens per (sequence, KV head) into an
    empty cache of the workload's shape: K calls, each after spla_reset
    (outside the timed events). Returns a dict for the JSON line: latency per
    call, tokens per second, and the bytes the append must move (the new K
    and V rows read and written into the cache, the block statistics
    written, S_bar and z_bar read and written)."""
    import numpy as np
    import torch

    from paper_2601_22379_amd import spla
    import spla_inputs as si

    T = min(T, w.capacity)
    cfg = spla.make_config(w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.block_size,
                           w.top_k, w.capacity, w.dtype, n_sink=w.n_sink, n_local=w.n_local)
    cache = spla.SplaCache(cfg, dev)
    dt = torch.float32 if w.dtype == "f32" else torch.bfloat16
    lens = [T] * w.batch
    Kt, Vt, n = si.gen_kv_slab(w, 0, T, lengths=lens, threads=16)
    kd = torch.from_numpy(Kt).to(dt).to(dev)
    vd = torch.from_numpy(Vt).to(dt).to(dev)
    del Kt, Vt
    times = []
    for i in range(K + 1):
        cache.reset()
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record()
        cache.append(kd, vd)
        b.record()
        torch.cuda.synchronize()
        if i > 0:
            times.append(a.elapsed_time(b) * 1e3)
    assert cache.device_errors() == 0
    us = float(np.median(times))
    e = 4 if w.dtype == "f32" else 2
    bh, d = w.batch * w.n_kv_heads, w.head_dim
    nb = -(-T // w.block_size)
    ab = {"kv_read": bh * T * 2 * d * e, "kv_written": bh * T * 2 * d * e,
          "stats_written": bh * nb * 2 * d * 4, "state_rw": 2 * bh * (d * d + d) * 4}
    ab["total"] = sum(ab.values())
    ach = ab["total"] / (us * 1e-6) / 1e9
    log(f"append: {T} tokens per (sequence, KV head) in {us:.1f} us "
        f"({bh * T / (us * 1e-6) / 1e9:.2f} G token-rows/s, {ach:.0f} GB/s algorithmic)")
    return {"tokens_per_sequence": T, "calls": K, "latency_us_median": round(us, 2),
            "token_rows_per_s": round(bh * T / (us * 1e-6), 1), "algorithmic_bytes": ab,
            "achieved_GBs": round(ach, 1), "frac_of_peak_hbm": round(ach / PEAK_HBM_GBS, 4),
            "method": "spla_append into an empty cache (events around the call)"}


def cpu_baseline(w, seconds, n_units=8):
    """The fp64 oracle's decode on a bounded sample of the workload: n_units
    (sequence, KV head) units with their state prebuilt (untimed), decoded
    round-robin for `seconds` of wall time by as many threads as the process
    may use (at most 16, the host share of one GPU; BLAS single-threaded in
    each), then by one thread for the 1-core figure."""
    import numpy as np
    from concurrent.futures import ThreadPoolExecutor
    from threadpoolctl import threadpool_limits

    import oracle as O
    import spla_inputs as si

    cores = max(1, min(16, len(os.sched_getaffinity(0))))
    p = O.SplaParams(block_size=w.block_size, top_k=w.top_k, n_sink=w.n_sink, n_local=w.n_local)
    rng = np.random.default_rng([w.code, 99])
    allp = [(b, h) for b in range(w.batch) for h in range(w.n_kv_heads)]
    pick = [allp[i] for i in rng.choice(len(allp), size=min(n_units, len(allp)), replace=False)]
    gamma = si.gen_gamma(w)

    def make(bh):
        b, h = bh
        L = int(w.lengths[b])
        K, V = si.gen_kv(w, b, h, 0, L)
        st = O.build_state(K, V, L, w.block_size)
        q = si.gen_q(w, b)[h * w.group:(h + 1) * w.group]
        return (q, st, K, V, gamma[h * w.group:(h + 1) * w.group])

    def timed(n_threads):
        t0 = time.perf_counter()
        counts = [0] * n_threads

        def work(i):
            j = 0
            while time.perf_counter() - t0 < seconds:
                u = units[(i + j) % len(units)]
                O.decode_kv_head(u[0], u[1], u[2], u[3], u[4], p)
                j += 1
            counts[i] = j

        with ThreadPoolExecutor(n_threads) as ex:
            list(ex.map(work, range(n_threads)))
        return sum(counts), time.perf_counter() - t0

    with threadpool_limits(1):
        with ThreadPoolExecutor(cores) as ex:
            units = list(ex.map(make, pick))
        n_all, t_all = timed(cores)
        n_one, t_one = timed(1)
    per_unit = si.algorithmic_bytes(w)["total"] / (w.batch * w.n_kv_heads)
    return {"value": round(per_unit * n_all / t_all / 1e9, 4), "unit": "GB/s", "cores": cores,
            "kind": "oracle",
            "value_1core": round(per_unit * n_one / t_one / 1e9, 4),
            "sample": f"fp64 oracle decode of {len(units)} of {len(allp)} (sequence, KV head) "
                      f"units of {w.name} (state prebuilt, untimed), round-robin for "
                      f"{seconds:.0f}s wall on {cores} threads ({n_all} unit decodes, "
                      f"{t_all / n_all * cores * 1e3:.1f} ms each) and on 1 thread "
                      f"({n_one} decodes, {t_one / max(n_one, 1) * 1e3:.1f} ms each)",
            "cpu": _cpu_model()}


def _cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


# ---------------------------------------------------------------------------
# rocprofv3 summaries (CSV output of the passes listed in the summaries)

def _kernel_short(name):
    return name.split("(")[0].replace("void ", "")


def trace_summary(trace_dir, workload, command, out_path, path="decode"):
    """Per-kernel averages of a `rocprofv3 --kernel-trace --stats` pass."""
    import csv
    rows = list(csv.DictReader(open(os.path.join(trace_dir, "run_kernel_stats.csv"))))
    lines = [f"# SPLA {path}, {workload}: kernel trace", "",
             f"command: `{command}`", "",
             "| kernel | calls | avg us | min us | max us |", "|---|---|---|---|---|"]
    for r in rows:
        n = r["Name"]
        if "spla" not in n:
            continue
        lines.append(f"| {_kernel_short(n)} | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
                     f"{float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} |")
    with open(out_path, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def traffic_summary(fetch_dir, write_dir, workload, commands, out_md, kernel, kernel_bytes,
                    variant=""):
    """Calibrated HBM bytes per dispatch from FETCH_SIZE / WRITE_SIZE passes.

    Both counters are in KiB per dispatch. Each is scaled by what it reads for
    the 1 GiB elementwise copy (--copy-calibration: 1 GiB read, 1 GiB written).
    The figures of `kernel` (the dominant kernel) also go to its JSON file,
    which bench.py reports while the kernel sources are unchanged.
    """
    import csv
    import collections

    def per_kernel(d, counter):
        acc = collections.defaultdict(list)
        for r in csv.DictReader(open(os.path.join(d, "run_counter_collection.csv"))):
            if r["Counter_Name"] == counter:
                acc[r["Kernel_Name"]].append(float(r["Counter_Value"]))
        return {k: sum(v) / len(v) for k, v in acc.items()}

    fetch, write = per_kernel(fetch_dir, "FETCH_SIZE"), per_kernel(write_dir, "WRITE_SIZE")
    copy = [k for k in fetch if "AUnaryFunctor" in k or "MulFunctor" in k]
    assert copy, "no calibration copy kernel in the FETCH_SIZE pass"
    gib_kib = float(1 << 20)
    f_scale = gib_kib / fetch[copy[0]]
    w_scale = gib_kib / write[copy[0]]
    label = workload + (", strided selection windows C = 32, s = 16" if variant else "")
    lines = [f"# SPLA decode, {label}: HBM traffic per dispatch (rocprofv3 counters)", ""]
    lines += [f"command: `{c}`" for c in commands]
    lines += ["", f"calibration (1 GiB read + 1 GiB written by one elementwise kernel): "
              f"FETCH_SIZE reads {fetch[copy[0]]:.1f} KiB -> scale {f_scale:.4f}; "
              f"WRITE_SIZE reads {write[copy[0]]:.1f} KiB -> scale {w_scale:.4f}", "",
              "| kernel | FETCH_SIZE KiB | WRITE_SIZE KiB | calibrated read MB | calibrated write MB |",
              "|---|---|---|---|---|"]
    dom = None
    for k in sorted(fetch):
        if "spla" not in k or "append" in k:
            continue
        fr, wr = fetch[k] * f_scale * 1024, write.get(k, 0.0) * w_scale * 1024
        lines.append(f"| {_kernel_short(k)} | {fetch[k]:.1f} | {write.get(k, 0.0):.1f} | "
                     f"{fr / 1e6:.3f} | {wr / 1e6:.3f} |")
        if f"::{kernel}_" in k:
            assert dom is None, f"several {kernel} kernels in the counter passes"
            dom = (fr, wr)
    assert dom is not None, f"no {kernel} kernel in the counter passes"
    lines += ["", f"{kernel} kernel: algorithmic {kernel_bytes / 1e6:.3f} MB per dispatch, counted "
              f"{(dom[0] + dom[1]) / 1e6:.3f} MB (read {dom[0] / 1e6:.3f} + write "
              f"{dom[1] / 1e6:.3f})"]
    with open(out_md, "w") as f:
        f.write("\n".join(lines) + "\n")
    with open(traffic_file(kernel, variant), "w") as f:
        json.dump({"workload": workload, "kernel": kernel,
                   "source_sha": source_hash(KERNEL_SOURCES),
                   "hbm_bytes_per_launch": int(round(dom[0] + dom[1])),
                   "read_bytes": int(round(dom[0])), "write_bytes": int(round(dom[1])),
                   "fetch_scale": f_scale, "write_scale": w_scale}, f, indent=1)
    print("\n".join(lines))


def percentiles(xs):
    import numpy as np

    a = np.asarray(xs, dtype=np.float64)
    return {"median": round(float(np.median(a)), 3), "p10": round(float(np.percentile(a, 10)), 3),
            "p90": round(float(np.percentile(a, 90)), 3), "n": int(a.size)}


def clone_cache(c):
    """A second cache with the same contents (device copies)."""
    from paper_2601_22379_amd import spla

    d = spla.SplaCache(c.cfg, c.device, block_table=c.block_table)
    for name in ("k", "v", "stats", "state", "norm", "seq_lens"):
        getattr(d, name).copy_(getattr(c, name))
    return d


def replicas_for(w, requested):
    """Cache copies decoded in rotation: one for the appending workload
    (each step's working set, about 0.8 GB, is already well above the 256 MB
    last-level cache, and its separate-launch replay needs a clone of the
    cache), else `requested`."""
    import spla_inputs as si

    big = si.algorithmic_bytes(w)["total"] > (1 << 29)
    return 1 if (w.appends_per_step > 0 or big) else requested


def run_workload(w, R, dev, K, W, headline=False, no_graph=False):
    """Fills R copies of the workload's cache and times K steps (after W
    untimed ones) on them in rotation. Every timed step writes an output of
    its own; afterwards the same steps are replayed on the separate-launch
    path and every output must match bit for bit, and every cache's device
    error word must be clear. A second pass brackets each step with events
    (median / p10 / p90), a third the dominant kernel. Returns the dict of
    the workload's JSON object and the extras (separate-launch latency and
    phases, graph replay; None for an appending workload that is not the
    headline)."""
    import numpy as np
    import torch

    from paper_2601_22379_amd import spla
    import spla_inputs as si

    cfg, caches = build_workload(w, R, dev)
    dt = torch.float32 if w.dtype == "f32" else torch.bfloat16
    gamma = torch.from_numpy(si.gen_gamma(w)).to(dev)
    appending = w.appends_per_step > 0
    n_steps = 4 * K + W + 2 * R + 1
    if appending:
        # per-step token rows and queries, generated before timing: step s
        # appends position lengths[b] - 1 + s // R of each sequence (each
        # replica advances on its own)
        n_pos = (n_steps - 1) // R + 1
        assert max(w.lengths) - 1 + n_pos <= w.capacity, "appending steps exceed the capacity"
        kn = np.zeros((n_steps, w.batch, w.n_kv_heads, w.head_dim), np.float32)
        vn = np.zeros_like(kn)
        steps = np.arange(n_steps)
        for b in range(w.batch):
            p0 = w.lengths[b] - 1
            for h in range(w.n_kv_heads):
                kk, vv = si.gen_kv(w, b, h, p0, p0 + n_pos)
                kn[:, b, h], vn[:, b, h] = kk[steps // R], vv[steps // R]
        kn_d = torch.from_numpy(kn).to(dt).to(dev)
        vn_d = torch.from_numpy(vn).to(dt).to(dev)
        qs = torch.from_numpy(np.stack([si.gen_q_batch(w, s) for s in range(min(n_steps, 64))])).to(
            dt).to(dev)
    else:
        qs = torch.from_numpy(si.gen_q_batch(w)[None]).to(dt).to(dev)
    outs = torch.empty((K, w.batch, w.n_q_heads, w.head_dim), dtype=dt, device=dev)
    sels = [torch.empty((w.batch, w.n_kv_heads, w.top_k), dtype=torch.int32, device=dev)
            for _ in range(R)]

    def one(s, out, cache=None, events=None):
        r = s % R
        c = caches[r] if cache is None else cache
        q = qs[s % qs.shape[0]]
        if appending:
            return c.step(kn_d[s], vn_d[s], q, gamma, out, sels[r], events)
        return c.decode(q, gamma, out, sels[r], events)

    launched = spla.decode_phases(cfg)
    # dominant kernel: the single launch, else the longer of the statistics
    # scan and the sparse pass (decided from their per-launch events below)
    cands = ["decode"] if "decode" in launched else ["score", "sparse"]
    for s in range(W):
        one(s, outs[0])
    torch.cuda.synchronize()
    ref_cache = clone_cache(caches[0]) if appending else None

    # timed region: exactly K steps, no instrumentation inside
    t_a = torch.cuda.Event(enable_timing=True)
    t_b = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_a.record()
    for s in range(K):
        one(W + s, outs[s])
    t_b.record()
    torch.cuda.synchronize()
    ms_per_step = t_a.elapsed_time(t_b) / K
    errs = [c.device_errors() for c in caches]
    assert all(e == 0 for e in errs), f"device error word set: {errs}"

    # the same steps on the separate launches, compared bit for bit
    ref = torch.empty_like(outs[0])
    mism = 0
    for c in caches + ([ref_cache] if ref_cache is not None else []):
        c.cfg.flags |= spla.FLAG_SEPARATE_KERNELS
    try:
        if appending:
            for s in range(K):
                # replica 0 only (R = 1 for the appending workload)
                one(W + s, ref, cache=ref_cache)
                mism += int(not torch.equal(ref, outs[s]))
        else:
            for r in range(min(R, K)):
                one(W + r, ref)
                for s in range(r, K, R):
                    mism += int(not torch.equal(ref, outs[s]))
        torch.cuda.synchronize()
    finally:
        for c in caches + ([ref_cache] if ref_cache is not None else []):
            c.cfg.flags &= ~spla.FLAG_SEPARATE_KERNELS
    assert mism == 0, f"{mism} of {K} timed steps differ from the separate-launch path"
    if ref_cache is not None:
        assert ref_cache.device_errors() == 0
        del ref_cache

    # each step bracketed by its own events: the distribution
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(K)]
    off = W + K if appending else W
    for s in range(K):
        ev[s][0].record()
        one(off + s, outs[s])
        ev[s][1].record()
    torch.cuda.synchronize()
    dist = percentiles([a.elapsed_time(b) * 1e3 for a, b in ev])

    # events around the candidate kernels only, recorded by the library
    dev_ev = [spla.make_events(cands) for _ in range(K)]
    off += K if appending else 0
    torch.cuda.synchronize()
    for s in range(K):
        one(off + s, outs[s], events=dev_ev[s][0])
    torch.cuda.synchronize()
    ev_us = {c: float(np.mean([e[1][c][0].elapsed_time(e[1][c][1]) for e in dev_ev])) * 1e3
             for c in cands}
    dom = max(cands, key=lambda c: ev_us[c])
    dom_us_events = ev_us[dom]
    # a step that is one launch of the dominant kernel and nothing else: the
    # timed region over the launches is its average launch duration, without
    # per-launch event records (whose own cost lengthens each launch)
    only_dom = launched == [dom] and not appending
    dom_us = ms_per_step * 1e3 if only_dom else dom_us_events
    dom_method = "timed region / launches" if only_dom else "per-launch events"

    sel_counts = None
    if not appending:
        lens = caches[0].seq_lens.cpu().numpy()
        sel_np = sels[0].cpu().numpy()
        sel_counts = [[sum(min(w.block_size, int(lens[b]) - int(i) * w.block_size)
                           for i in sel_np[b, h] if i >= 0) for h in range(w.n_kv_heads)]
                      for b in range(w.batch)]
    ab = si.algorithmic_bytes(w, sel_counts)
    dom_bytes = dominant_bytes(w, ab, dom)
    achieved = dom_bytes / (dom_us * 1e-6) / 1e9
    prof_us = None
    trace_md = os.path.join(ROOT, "profiles", f"decode_{w.name}_kernel_trace.md")
    if os.path.exists(trace_md):
        for ln in open(trace_md):
            if ln.startswith(f"| spla::{dom}_"):
                prof_us = float(ln.split("|")[3])
                break
    leg = {"latency_us": round(ms_per_step * 1e3, 3),
           "latency_us_per_step_events": dist,
           "value": round(ab["total"] / (ms_per_step * 1e-3) / 1e9, 1), "unit": "GB/s",
           "frac_of_peak_hbm": round(ab["total"] / (ms_per_step * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
           "algorithmic_bytes": ab, "kernels": launched + (["append"] if appending else []),
           "cache_replicas": R, "steps": K,
           "checked": f"{K} timed steps equal to the separate launches bit for bit; "
                      "device error word clear",
           "roofline": {"kernel": dom, "bound": "hbm", "achieved": round(achieved, 1),
                        "peak": PEAK_HBM_GBS, "unit": "GB/s",
                        "frac": round(achieved / PEAK_HBM_GBS, 4),
                        "traffic": traffic_of(dom, w.name),
                        "algorithmic_bytes_per_launch": dom_bytes,
                        "avg_launch_us": round(dom_us, 3), "avg_launch_method": dom_method,
                        "avg_launch_us_per_launch_events": round(dom_us_events, 3),
                        "profiled_avg_us": prof_us}}
    log(f"{w.name}: {ms_per_step * 1e3:.2f} us/step (per-step events median {dist['median']:.2f}, "
        f"p10 {dist['p10']:.2f}, p90 {dist['p90']:.2f}); {dom} kernel {dom_us:.2f} us "
        f"({dom_method}), {achieved:.0f} GB/s algorithmic")
    if not headline and appending:
        del caches
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        return leg, None

    # extras: the separate-kernel path's plain latency and phases, and a graph
    # replay of the steps
    sep_names = ["score", "select", "sparse", "merge"] + (["append"] if appending else [])
    for c in caches:
        c.cfg.flags |= spla.FLAG_SEPARATE_KERNELS
    sep_launched = set(spla.decode_phases(caches[0].cfg)) | {"append"}
    try:
        for s in range(W):
            one(s, outs[0])
        torch.cuda.synchronize()
        t_a.record()
        for s in range(K):
            one(W + s, outs[s])
        t_b.record()
        torch.cuda.synchronize()
        sep_ms = t_a.elapsed_time(t_b) / K
        evp = [spla.make_events(sep_names) for _ in range(K)]
        torch.cuda.synchronize()
        for s in range(K):
            one(W + 2 * K + s, outs[s], events=evp[s][0])
        torch.cuda.synchronize()
    finally:
        for c in caches:
            c.cfg.flags &= ~spla.FLAG_SEPARATE_KERNELS
    phases = {}
    for name in sep_names:
        if name in sep_launched:
            phases[name] = float(np.mean([e[1][name][0].elapsed_time(e[1][name][1])
                                          for e in evp])) * 1e3
    log(f"separate kernels {sep_ms * 1e3:.2f} us/step, phases us: "
        + ", ".join(f"{k}={v:.2f}" for k, v in phases.items()))
    graph_us = None
    if not no_graph and not appending:
        try:
            # one graph holding NG consecutive steps (over the replicas), so
            # that the graph's own launch cost is shared by NG steps
            NG = R * max(1, 12 // R)
            side = torch.cuda.Stream()
            side.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(side):
                g = torch.cuda.CUDAGraph()
                with torch.cuda.graph(g, stream=side):
                    for r in range(NG):
                        one(r, outs[r % K])
            torch.cuda.current_stream().wait_stream(side)
            torch.cuda.synchronize()
            for r in range(NG):
                one(r, outs[r % K])
            torch.cuda.synchronize()
            eager = [outs[r % K].clone() for r in range(min(NG, K))]
            for _ in range(3):
                g.replay()
                torch.cuda.synchronize()
                for r in range(min(NG, K)):
                    assert torch.equal(outs[r % K], eager[r]), "graph replay differs from eager"
            n_rep = max(1, K // NG)
            t_a.record()
            for _ in range(n_rep):
                g.replay()
            t_b.record()
            torch.cuda.synchronize()
            graph_us = t_a.elapsed_time(t_b) / (n_rep * NG) * 1e3
        except Exception as e:  # graph capture is an extra measurement only
            log(f"graph measurement skipped: {e!r}")
    extras = {"latency_us_separate_kernels": round(sep_ms * 1e3, 3),
              "phases_us_separate_kernels": {k: round(v, 3) for k, v in phases.items()},
              "latency_us_hip_graph": None if graph_us is None else round(graph_us, 3)}
    del caches
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return leg, extras


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", default="3")
    ap.add_argument("--replicas", type=int, default=6)
    ap.add_argument("--cpu-seconds", type=float, default=6.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-graph", action="store_true")
    ap.add_argument("--legs", default="1,2,4,5,g5",
                    help="other workloads measured after the headline one ('' for none)")
    ap.add_argument("--no-strided", action="store_true",
                    help="skip the strided-selection (C = 32, s = 16), paged-KV and prefill legs")
    ap.add_argument("--strided-only", action="store_true",
                    help="run only the strided-selection leg and print its JSON (profiling)")
    ap.add_argument("--prefill-only", action="store_true",
                    help="run only the prefill leg and print its JSON (profiling)")
    ap.add_argument("--append-only", action="store_true",
                    help="run only the bulk-append leg and print its JSON (profiling)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run a plain 1 GiB copy kernel (for counter scaling)")
    ap.add_argument("--trace-summary", metavar="DIR",
                    help="write the profiles/ summary of a kernel-trace pass in DIR and exit")
    ap.add_argument("--traffic-summary", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="write the profiles/ traffic summary of two counter passes and exit")
    ap.add_argument("--kernel", default="decode", choices=["decode", "score", "sparse"],
                    help="dominant kernel of a --traffic-summary")
    ap.add_argument("--command", action="append", default=[],
                    help="profiling command quoted in a summary (repeatable)")
    args = ap.parse_args()
    if args.trace_summary or args.traffic_summary:
        import spla_inputs as si
        w = si.config(args.config)
        path = "prefill" if args.prefill_only else ("append" if args.append_only else "decode")
        tag = f"{path}_{w.name}" + (STRIDED_TAG if args.strided_only else "")
        if args.trace_summary:
            label = w.name + (", strided selection windows C = 32, s = 16"
                              if args.strided_only else "")
            trace_summary(args.trace_summary, label, " && ".join(args.command),
                          os.path.join(ROOT, "profiles", f"{tag}_kernel_trace.md"), path)
        if args.traffic_summary:
            ab = si.algorithmic_bytes(w, None)
            variant = STRIDED_TAG if args.strided_only else ""
            if args.strided_only:  # window statistics: one entry per 16 tokens
                ab["stats"] = sum(-(-int(L) // 16) for L in w.lengths) * w.n_kv_heads * 2 * \
                    w.head_dim * 4
            traffic_summary(args.traffic_summary[0], args.traffic_summary[1], w.name,
                            args.command, os.path.join(ROOT, "profiles", f"{tag}_traffic.md"),
                            args.kernel, dominant_bytes(w, ab, args.kernel), variant)
        return
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py: --gpus {args.gpus} (world size {world}) requested; this SPLA decode "
              "library runs on a single GPU only (no multi-GPU path is built).", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2601_22379_amd import spla
    import spla_inputs as si

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    spla.lib()  # fail loudly if the HIP library is missing
    dev = torch.device("cuda:0")
    w = si.config(args.config)
    R = max(1, args.replicas)
    K, W = args.steps, args.warmup
    dt = torch.float32 if w.dtype == "f32" else torch.bfloat16
    if args.strided_only:
        qs = torch.from_numpy(si.gen_q_batch(w)[None]).to(dt).to(dev)
        gamma = torch.from_numpy(si.gen_gamma(w)).to(dev)
        outs = [torch.empty((w.batch, w.n_q_heads, w.head_dim), dtype=dt, device=dev)
                for _ in range(R)]
        sels = [torch.empty((w.batch, w.n_kv_heads, w.top_k), dtype=torch.int32, device=dev)
                for _ in range(R)]
        line = strided_leg(w, R, dev, qs, gamma, outs, sels, K, W)
        if args.copy_calibration:
            copy_calibration(dev)
        print(json.dumps(line), flush=True)
        return
    if args.prefill_only:
        print(json.dumps(prefill_leg(w, dev, K=K)), flush=True)
        return
    if args.append_only:
        print(json.dumps(append_leg(w, dev, K=min(K, 20))), flush=True)
        return
    wall0 = time.perf_counter()
    head, extras = run_workload(w, replicas_for(w, R), dev, K, W, headline=True,
                                no_graph=args.no_graph)
    strided = paged = prefill = append = None
    if w.appends_per_step == 0 and not args.no_strided:
        qs = torch.from_numpy(si.gen_q_batch(w)[None]).to(dt).to(dev)
        gamma = torch.from_numpy(si.gen_gamma(w)).to(dev)
        outs = [torch.empty((w.batch, w.n_q_heads, w.head_dim), dtype=dt, device=dev)
                for _ in range(R)]
        sels = [torch.empty((w.batch, w.n_kv_heads, w.top_k), dtype=torch.int32, device=dev)
                for _ in range(R)]
        strided = strided_leg(w, R, dev, qs, gamma, outs, sels, K, W)
        paged = strided_leg(w, R, dev, qs, gamma, outs, sels, K, W, C=w.block_size,
                            s=w.block_size, paged=True)
        prefill = prefill_leg(w, dev, K=20)
        torch.cuda.empty_cache()
        append = append_leg(w, dev, K=10)
        torch.cuda.empty_cache()
    legs = {}
    for cid in [c for c in args.legs.split(",") if c.strip() and c.strip() != args.config]:
        wl = si.config(cid.strip())
        # the appending workload has 512 positions of room for all its steps
        kl = min(K, 100) if wl.appends_per_step else K
        leg, ex = run_workload(wl, replicas_for(wl, R), dev, kl, W)
        legs[wl.name] = {**leg, **(ex or {})}
    if args.copy_calibration:
        copy_calibration(dev)
    cpu = None
    if not args.no_cpu_baseline:
        log("timing the CPU oracle")
        cpu = cpu_baseline(w, args.cpu_seconds)
    ms_per_step = head["latency_us"] / 1e3
    line = {
        "metric": METRIC,
        "value": head["value"],
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": round(ms_per_step, 6),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic (seeded generators; no dataset)",
        "config": {"workload": w.name, "batch": w.batch, "n_q_heads": w.n_q_heads,
                   "n_kv_heads": w.n_kv_heads, "head_dim": w.head_dim,
                   "context": int(max(w.lengths)), "block_size": w.block_size,
                   "top_k": w.top_k, "n_sink": w.n_sink, "n_local": w.n_local,
                   "cache_replicas": head["cache_replicas"],
                   "appends_per_step": w.appends_per_step},
        "latency_us": head["latency_us"],
        "latency_us_per_step_events": head["latency_us_per_step_events"],
        "frac_of_peak_hbm": head["frac_of_peak_hbm"],
        "algorithmic_bytes": head["algorithmic_bytes"],
        "checked": head["checked"],
        **extras,
        "roofline": head["roofline"],
        "cpu_baseline": cpu,
        "workloads": legs,
        "strided_selection": strided,
        "paged_kv": paged,
        "prefill": prefill,
        "append": append,
        "bench_wall_s": round(time.perf_counter() - wall0, 1),
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
