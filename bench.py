#!/usr/bin/env python3
"""Benchmark of the f-gram embedding hot path on one MI355X.

One step is one pass of the whole path over one [B, T] batch's worth of work,
inputs already resident on the device: the longest-suffix lookup and the row
gather.  The headline schedule is the library's pipelined step
(scone_embed_pipelined): each launch gathers the rows of batch k while it
looks up batch k+1, so K timed steps run K lookups and K gathers.  The serial
schedule (scone_lookup then scone_gather) and the fused kernel (scone_embed)
are timed beside it.  The table build is offline and not timed.  Prints one
JSON line with tokens/s, the step kernel's achieved bandwidth against its
roofline (HBM, or PCIe when the rows live in host-pinned memory), and the CPU
oracle timed on a bounded sample of the same workload.

Workloads (``--config``): c3_10m_k5 (default: 10M f-grams of length 2..5,
4 KiB rows, 41 GB in HBM, the largest workload one GPU holds), c2_1m, tiny
(HBM prefill), c4_host (rows in host-pinned memory read over PCIe), c5_decode
(256 sequences x 1024 decoding steps of one token each).

The headline roofline fraction is cache-assisted: Zipf-distributed ids repeat
rows that the L2s and the 256 MB last-level cache then serve.  The same
pipelined step over uniform random ids (no repeated rows) is reported beside
it as ``roofline.no_reuse``.

Profiling: ``--plan-out FILE`` records which library kernel each dispatch of
the run is and to which phase it belongs; ``--reduce-trace`` and
``--reduce-counters`` turn rocprofv3 csv output of such a run into the
summaries under profiles/ (see ``reduce_main``).

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--config NAME]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "tokens/sec and gather GB/s (% of HBM peak) for f-gram lookup+gather, 1 MI355X"
HBM_PEAK_GBPS = 8000.0
PCIE_PEAK_GBPS = 63.0    # PCIe 5.0 x16, one direction
MFMA_BF16_PEAK_TFLOPS = 2500.0  # dense bf16 matrix-core peak
DEFAULT_CONFIG = "c3_10m_k5"
N_BATCHES = 4
SAMPLE_EVERY = 8
COLD_REPS = 10


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def describe(cfg) -> str:
    where = "host-pinned memory" if cfg.placement == "host" else "HBM"
    shape = (f"{cfg.B} sequences x {cfg.T} decode steps" if cfg.decode
             else f"queries {cfg.B}x{cfg.T}")
    return (f"{cfg.name}: vocab {cfg.V} Zipf(1.1), {cfg.n_fgrams} f-grams of length "
            f"{cfg.min_len}..{cfg.max_len}, table {cfg.n_rows}x{cfg.d} {cfg.dtype} in "
            f"{where}, {shape}, {int(cfg.coverage * 100)}% planted coverage, "
            f"max_n={cfg.max_n}")


# The sources of each measured kernel (its file and the headers that hold its
# device code): a traffic summary is used only while they are unchanged.
KERNEL_SOURCES = {
    "gather": ("gather.hip", "row_copy.h", "scone_internal.h"),
    "embed": ("embed.hip", "tile_lookup.h", "scone_internal.h", "table_build.hip"),
    "pipelined": ("pipeline.hip", "row_copy.h", "tile_lookup.h", "scone_internal.h",
                  "table_build.hip"),
}


def source_sha(*names: str) -> str:
    h = hashlib.sha1()
    for name in names:
        h.update(open(os.path.join(ROOT, "paper_2502_01637_amd", "csrc", name), "rb").read())
    return h.hexdigest()[:12]


def measured_traffic(config: str, kernel: str):
    """HBM bytes per launch of `kernel` from the committed rocprofv3 counter
    summary, or None when there is none for the kernel's current sources."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{config}_traffic.md")
    if not os.path.exists(path):
        return None
    m = re.search(r"^TRAFFIC (\{.*\})\s*$", open(path).read(), re.M)
    if not m:
        return None
    rec = json.loads(m.group(1))
    if rec.get("source_sha1") != source_sha(*KERNEL_SOURCES[kernel]):
        return None
    return rec


def build_table(S, torch, w, dev, max_load):
    fg = torch.from_numpy(w.fgrams).to(dev)
    ln = torch.from_numpy(w.lengths).to(dev)
    idv = torch.from_numpy(w.ids).to(dev)
    torch.cuda.synchronize()
    t = time.perf_counter()
    table = S.build_fgram_table(fg, ln, idv, max_load=max_load)
    return table, time.perf_counter() - t


def host_rows(S, torch, cfg, dev):
    """The whole row table in pinned host memory, filled chunk by chunk from
    the generator on the device."""
    from workloads import fill_table, torch_dtype
    t = time.perf_counter()
    host = S.HostRows(cfg.n_rows, (cfg.d,), torch_dtype(cfg))
    log(f"pinned {host.nbytes / 1e9:.1f} GB of host memory in {time.perf_counter() - t:.1f} s")
    ht = host.tensor()
    chunk = max(1, (1 << 30) // cfg.row_bytes)
    stage = torch.empty((chunk, cfg.d), dtype=torch_dtype(cfg), device=dev)
    t = time.perf_counter()
    for r0 in range(0, cfg.n_rows, chunk):
        n = min(chunk, cfg.n_rows - r0)
        fill_table(cfg, stage[:n], row0=r0)
        ht[r0:r0 + n].copy_(stage[:n])
        if (r0 // chunk) % 16 == 0:
            log(f"  filled rows {r0 + n}/{cfg.n_rows}")
    torch.cuda.synchronize()
    log(f"filled in {time.perf_counter() - t:.1f} s")
    del stage
    return host


def h2d_ceiling(torch, dev, nbytes=1 << 30, reps=5):
    """Measured host-to-device copy rate from pinned memory (GB/s)."""
    src = torch.empty(nbytes, dtype=torch.uint8, pin_memory=True)
    dst = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    dst.copy_(src, non_blocking=True)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        dst.copy_(src, non_blocking=True)
    e1.record()
    torch.cuda.synchronize()
    return nbytes * reps / (e0.elapsed_time(e1) * 1e-3) / 1e9


def split_placement(S, torch, cfg, table, rows, X, fid, outs, K, warmup):
    """Token rows in HBM, f-gram rows in pinned host memory, each distinct
    f-gram row of a batch read over PCIe once (scone_gather_split)."""
    dev = outs[0].device
    near = rows.tensor()[:cfg.V].to(dev)          # the token rows, copied into HBM
    far = rows.rows(cfg.V, cfg.n_rows)            # the f-gram rows, in place
    ws = torch.empty(S.split_workspace_bytes(cfg.n_tok, cfg.row_bytes), dtype=torch.uint8,
                     device=dev)
    nu = torch.zeros(1, dtype=torch.int32, device=dev)
    SPLIT = ("k_split_clear", "k_split_insert", "k_split_number", "k_split_fetch",
             "k_split_gather")
    for k in range(warmup):
        S.lookup(table, X[k % N_BATCHES], cfg.max_n, fgram_ids=fid)
        S.gather_split(fid, near, far, ws, out=outs[k % N_BATCHES], n_unique=nu)
        for kern in ("k_lookup",) + SPLIT:
            PLAN.add("split_warmup", kern)
    if S.check() != 0:
        raise SystemExit("device error in split-placement warm-up")
    ev, uniq = [], []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(K):
        e = None
        if k % SAMPLE_EVERY == 0:
            e = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
            ev.append(e)
        S.lookup(table, X[k % N_BATCHES], cfg.max_n, fgram_ids=fid)
        if e:
            e[0].record()
        S.gather_split(fid, near, far, ws, out=outs[k % N_BATCHES], n_unique=nu)
        for kern in ("k_lookup",) + SPLIT:
            PLAN.add("split_timed", kern)
        if e:
            e[1].record()
            uniq.append(nu.clone())
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    if S.check() != 0:
        raise SystemExit("device error in split placement")
    ms = float(np.mean([a.elapsed_time(b) for a, b in ev]))
    n_unique = float(np.mean([int(u.item()) for u in uniq]))
    # parity of batch 0 against the plain gather over the whole host table
    ids0, _ = S.lookup(table, X[0], cfg.max_n)
    a = S.gather(ids0, rows)
    b = S.gather_split(ids0, near, far, ws)
    for kern in ("k_lookup", "k_gather") + SPLIT:
        PLAN.add("split_parity", kern)
    same = bool(torch.equal(a.view(torch.int16), b.view(torch.int16)))
    del near, ws
    return {"tokens_per_s": cfg.n_tok * K / wall, "ms_per_step": wall * 1e3 / K,
            "gather_split_us": ms * 1e3, "distinct_far_rows_per_batch": n_unique,
            "pcie_bytes_per_batch": n_unique * cfg.row_bytes,
            "rows_equal_plain_gather": same}


class Plan:
    """The library kernels a run launches, one entry per dispatch, in order,
    each with the phase it belongs to.  ``--plan-out`` writes it next to a
    rocprofv3 run so that the reducers can tell the timed dispatches of each
    phase apart from warm-up, control and parity launches."""

    def __init__(self):
        self.entries = []

    def add(self, phase: str, kernel: str, n: int = 1):
        self.entries.extend([[phase, kernel]] * n)


PLAN = Plan()


def host_info() -> dict:
    """CPU model and the cores this process may run on."""
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    cores = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else os.cpu_count()
    return {"cpu_model": model, "cores_available": int(cores or 1)}


def oracle_threads() -> int:
    """Threads for the all-core oracle timing: the cores this process may use,
    capped by OMP_NUM_THREADS when the environment sets it."""
    n = host_info()["cores_available"]
    env = os.environ.get("OMP_NUM_THREADS", "")
    if env.isdigit() and int(env) > 0:
        n = min(n, int(env))
    return max(1, n)


def probes_per_position(cfg, w, X: np.ndarray) -> float:
    """Mean hash probes per position of the kernels' tile lookup, counted on
    the host by replaying its schedule (not read off the device): lengths 3
    and 2 in the first round (only 2 when max_n = 2), 5 and 4 in the second
    where the length-3 suffix ends some f-gram of length 4 or more, 7 and 6 in
    the third where the length-5 suffix ends one of length 6 or more; a length
    is probed only when it fits the window (n <= min(max_n, t + 1))."""
    B, T = X.shape
    max_n = min(cfg.max_n, cfg.max_len)     # the library clamps the window to K
    top = np.broadcast_to(np.minimum(max_n, np.arange(T) + 1), (B, T))

    def fits(n):
        return (top >= n) if n >= 2 else np.zeros_like(top, dtype=bool)

    def windows(n):
        """The length-n window ending at every position, as n int32 tokens in
        one opaque value (positions before t = n - 1 get zeros, and fits()
        masks them)."""
        win = np.zeros((B, T, n), dtype=np.int32)
        for i in range(n):
            lag = n - 1 - i                       # token i of the window is X[t - lag]
            win[:, lag:, i] = X[:, :T - lag]
        return win.reshape(B * T, n).view(np.dtype((np.void, 4 * n))).reshape(B, T)

    def flagged(n):
        """Positions whose length-n suffix ends an f-gram of length n + 1 or more."""
        long_ = w.lengths >= n + 1
        if not long_.any():
            return np.zeros((B, T), dtype=bool)
        sel = w.fgrams[long_]
        L = w.lengths[long_].astype(np.int64)
        cols = L[:, None] - n + np.arange(n)[None, :]
        ends = np.ascontiguousarray(np.take_along_axis(sel, cols, axis=1), dtype=np.int32)
        ends = ends.view(np.dtype((np.void, 4 * n))).ravel()
        return np.isin(windows(n), np.unique(ends)) & fits(n)

    if max_n <= 2:
        return float(fits(2).sum()) / X.size
    probes = fits(3).astype(np.int64) + fits(2).astype(np.int64)
    if max_n >= 4:
        go = flagged(3)
        probes += go * (fits(5).astype(np.int64) + fits(4))
        if max_n >= 6:
            probes += (go & flagged(5)) * (fits(7).astype(np.int64) + fits(6))
    return float(probes.sum()) / X.size


def oracle_all_cores(one_pass, X: np.ndarray, min_seconds: float) -> dict:
    """The oracle's passes over X with its rows split into one slice per host
    thread (the oracle's calls release the interpreter lock, so the slices
    run in parallel on its shared read-only dictionary), repeated for at least
    min_seconds: a labelled all-core figure beside the single-core baseline."""
    import threading
    nthr = min(oracle_threads(), X.shape[0])
    slices = np.array_split(np.arange(X.shape[0]), nthr)
    passes, elapsed = 0, 0.0
    while elapsed < min_seconds or passes == 0:
        t = time.perf_counter()
        th = [threading.Thread(target=one_pass, args=(X[sl],)) for sl in slices]
        for x in th:
            x.start()
        for x in th:
            x.join()
        elapsed += time.perf_counter() - t
        passes += 1
    return {"value": passes * X.size / elapsed, "unit": "tokens/s", "threads": nthr,
            "passes": passes, "seconds": round(elapsed, 3),
            "how": f"the same passes with the rows split over {nthr} threads sharing the "
                   "oracle's dictionary"}


def cpu_baseline(cfg, w, X0, host_np_full, E, gpu_ids, gpu_outs, min_seconds: float):
    """Time the oracle (single-threaded) on batch 0, repeated until min_seconds,
    then the same passes split by rows over all host cores (labelled), and
    check the GPU results of batch 0 against it."""
    import torch
    import oracle
    from workloads import table_rows
    t0 = time.perf_counter()
    o = oracle.OracleTable(w.fgrams, w.lengths, w.ids)
    build_s = time.perf_counter() - t0
    exp_ids, exp_len = o.lookup(X0, cfg.max_n)
    queries = o.queries
    uniq = None
    if host_np_full is not None:
        host_np, what = host_np_full, "the full host-pinned table"
    elif cfg.n_rows * cfg.row_bytes <= (4 << 30):
        host_np, what = E.cpu().view(torch.uint8).numpy(), "the full host table"
    else:
        # only the rows this batch references (the full table is not copied to
        # the host); the id remap to that compact table is timed with the gather
        uniq = np.unique(exp_ids)
        host = table_rows(cfg, torch.from_numpy(uniq.astype(np.int64)), device="cuda").cpu()
        host_np = host.view(torch.uint8).numpy()
        what = f"a compact host table of the {len(uniq)} referenced rows (id remap timed)"

    def one_pass(rows):
        ids_p, _ = o.lookup(rows, cfg.max_n)
        if uniq is not None:
            ids_p = np.searchsorted(uniq, ids_p).astype(np.int32)
        return oracle.gather(ids_p, host_np)

    passes, elapsed = 0, 0.0
    while elapsed < min_seconds or passes == 0:
        t = time.perf_counter()
        out = one_pass(X0)
        elapsed += time.perf_counter() - t
        passes += 1
    all_cores = oracle_all_cores(one_pass, X0, min_seconds / 2)
    parity_rows = [bool(g.view(torch.uint8).cpu().numpy().reshape(out.shape).tobytes()
                        == out.tobytes()) for g in gpu_outs]
    info = host_info()
    return ({"value": passes * cfg.n_tok / elapsed, "unit": "tokens/s", "cores": 1,
             "kind": "oracle",
             "sample": f"batch 0 ({cfg.n_tok} tokens) of {describe(cfg)}; {passes} full "
                       f"passes of lookup + memcpy gather from {what}; dictionary build "
                       f"({build_s:.1f} s) not timed",
             "seconds": round(elapsed, 3), "build_seconds": round(build_s, 3),
             "cpu_model": info["cpu_model"], "cores_available": info["cores_available"],
             "all_cores": all_cores},
            {"ids_bit_exact": bool(np.array_equal(gpu_ids, exp_ids)),
             "split_rows_bit_exact": parity_rows[0], "fused_rows_bit_exact": parity_rows[1],
             "pipelined_rows_bit_exact": parity_rows[2],
             "positions": int(cfg.n_tok)}, exp_len, queries)


def run_prefill(args, cfg):
    import torch
    import paper_2502_01637_amd as S
    from workloads import make_workload, query_batches, fill_table, torch_dtype, match_stats

    dev = torch.device("cuda", 0)
    host = cfg.placement == "host"
    t = time.perf_counter()
    w = make_workload(cfg)
    batches_np = query_batches(w, N_BATCHES)
    log(f"generated in {time.perf_counter() - t:.1f} s")
    table, build_s = build_table(S, torch, w, dev, args.max_load)
    if host:
        rows = host_rows(S, torch, cfg, dev)
        E = None
    else:
        E = torch.empty((cfg.n_rows, cfg.d), dtype=torch_dtype(cfg), device=dev)
        fill_table(cfg, E)
        rows = E
    X = [torch.from_numpy(b).to(dev) for b in batches_np]
    fid = torch.empty((cfg.B, cfg.T), dtype=torch.int32, device=dev)
    # the pipelined schedule's two id buffers: step g gathers pid[g % 2] (batch
    # g's ids, looked up by step g - 1) and looks up batch g + 1 into the other
    pid = [torch.empty((cfg.B, cfg.T), dtype=torch.int32, device=dev) for _ in range(2)]
    # Step k writes outs[k % N_BATCHES]: together the outputs exceed the 256 MB
    # last-level cache, so no step overwrites lines the previous one left
    # dirty there and every step's writes reach HBM.
    outs = [torch.empty((cfg.B, cfg.T, cfg.d), dtype=torch_dtype(cfg), device=dev)
            for _ in range(N_BATCHES)]
    torch.cuda.synchronize()
    log(f"table: {table.n} f-grams, {table.entries} entries in {table.capacity} slots x "
        f"{table.slot_bytes} B, build {build_s * 1e3:.1f} ms")

    K = args.steps
    G = "k_gather"      # k_gather_rows for whole-KiB rows, k_gather otherwise

    def pipelined_step(g):
        S.embed_pipelined(table, X[(g + 1) % N_BATCHES], cfg.max_n, pid[(g + 1) % 2],
                          pid[g % 2], rows, out=outs[g % N_BATCHES])

    def timed(path):
        """W warm-up steps, then K timed steps between two synchronisations.
        HIP events around each kernel are recorded on every 8th step only, so
        that they barely perturb the wall clock.  Returns (wall seconds,
        per-kernel mean ms list, device ms per step over the timed region)."""
        if path == "pipelined":   # first lookup, before the warm-up steps
            S.embed_pipelined(table, X[0], cfg.max_n, pid[0], None, rows)
            PLAN.add("pipelined_first_lookup", "k_lookup")
        for k in range(args.warmup):
            if path == "split":
                S.lookup(table, X[k % N_BATCHES], cfg.max_n, fgram_ids=fid)
                S.gather(fid, rows, out=outs[k % N_BATCHES])
                PLAN.add("serial_warmup", "k_lookup")
                PLAN.add("serial_warmup", G)
            elif path == "pipelined":
                pipelined_step(k)
                PLAN.add("pipelined_warmup", "k_pipelined")
            else:
                S.embed(table, X[k % N_BATCHES], cfg.max_n, rows, out=outs[k % N_BATCHES])
                PLAN.add("fused_warmup", "k_embed")
        rc = S.check()
        if rc != 0:
            raise SystemExit(f"device error after warmup ({path}): status {rc}")
        nk = 2 if path == "split" else 1
        ev = []
        span = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        span[0].record()
        for k in range(K):
            e = None
            if k % SAMPLE_EVERY == 0:
                e = [torch.cuda.Event(enable_timing=True) for _ in range(nk + 1)]
                ev.append(e)
                e[0].record()
            if path == "split":
                S.lookup(table, X[k % N_BATCHES], cfg.max_n, fgram_ids=fid)
                if e:
                    e[1].record()
                S.gather(fid, rows, out=outs[k % N_BATCHES])
                PLAN.add("serial_timed", "k_lookup")
                PLAN.add("serial_timed", G)
            elif path == "pipelined":
                pipelined_step(args.warmup + k)
                PLAN.add("pipelined_timed", "k_pipelined")
            else:
                S.embed(table, X[k % N_BATCHES], cfg.max_n, rows, out=outs[k % N_BATCHES])
                PLAN.add("fused_timed", "k_embed")
            if e:
                e[nk].record()
        span[1].record()
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        rc = S.check()
        if rc != 0:
            raise SystemExit(f"device error in timed region ({path}): status {rc}")
        per = [float(np.mean([e[i].elapsed_time(e[i + 1]) for e in ev])) for i in range(nk)]
        return wall, per, span[0].elapsed_time(span[1]) / K

    # The headline is the pipelined schedule (one launch per step); the serial
    # schedule, scone_lookup then scone_gather, and the fused scone_embed are
    # timed the same way beside it.
    # The pipelined path launches one kernel per step, so its launch duration
    # is the device time of the whole timed region (two events around it) per
    # step; the events around single sampled launches (also reported) read a
    # few microseconds high, as each adds its own marker packets.
    wall, (pipe_sampled_ms,), pipe_ms = timed("pipelined")
    serial_wall, (lookup_ms, gather_ms), _ = timed("split")
    fused_wall, (embed_ms,), _ = timed("fused")

    gather_bytes = cfg.gather_bytes()
    # one pipelined launch: the gather's bytes plus the lookup's token read
    # and id write (hash probes are the lookup's cost, not the problem's)
    pipe_bytes = gather_bytes + cfg.n_tok * 8
    pipe_achieved = pipe_bytes / (pipe_ms * 1e-3) / 1e9
    value = cfg.n_tok * K / wall

    # Id sets without reuse, rotated like the query batches (one set reused
    # every step would leave its rows in the 256 MB last-level cache):
    # uniform random ids over the whole table, and contiguous rows (the
    # kernel's streaming rate with neither reuse nor random access).
    gen = torch.Generator(device=dev)
    gen.manual_seed(cfg.seed)
    uids = [torch.randint(0, cfg.n_rows, (cfg.B, cfg.T), dtype=torch.int32, device=dev,
                          generator=gen) for _ in range(N_BATCHES)]
    sids = [(torch.arange(k * cfg.n_tok, (k + 1) * cfg.n_tok, dtype=torch.int64, device=dev)
             % cfg.n_rows).to(torch.int32).view(cfg.B, cfg.T) for k in range(N_BATCHES)]

    # The headline kernel without cache help: the same pipelined steps, each
    # looking up the next real batch while it gathers one of the uniform id
    # sets.  Its rate is HBM's alone.
    nr_next = torch.empty_like(pid[0])
    for k in range(2):
        S.embed_pipelined(table, X[(k + 1) % N_BATCHES], cfg.max_n, nr_next,
                          uids[k % N_BATCHES], rows, out=outs[k % N_BATCHES])
    PLAN.add("noreuse_warmup", "k_pipelined", 2)
    torch.cuda.synchronize()
    ne = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    ne[0].record()
    for k in range(K):
        S.embed_pipelined(table, X[(k + 1) % N_BATCHES], cfg.max_n, nr_next,
                          uids[k % N_BATCHES], rows, out=outs[k % N_BATCHES])
    ne[1].record()
    torch.cuda.synchronize()
    PLAN.add("noreuse_timed", "k_pipelined", K)
    if S.check() != 0:
        raise SystemExit("device error in the no-reuse pipelined steps")
    noreuse_ms = ne[0].elapsed_time(ne[1]) / K

    def control_ms(idsets, phase):
        for k in range(2):
            S.gather(idsets[k % N_BATCHES], rows, out=outs[k % N_BATCHES])
        PLAN.add(phase + "_warmup", G, 2)
        torch.cuda.synchronize()
        ue = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        ue[0].record()
        for k in range(K):
            S.gather(idsets[k % N_BATCHES], rows, out=outs[k % N_BATCHES])
        ue[1].record()
        torch.cuda.synchronize()
        PLAN.add(phase + "_timed", G, K)
        return ue[0].elapsed_time(ue[1]) / K

    uniform_ms = control_ms(uids, "uniform")
    sequential_ms = control_ms(sids, "contiguous")
    del uids, sids, nr_next

    # Cold caches: reading a 1 GiB buffer between repetitions evicts the L2s
    # and the 256 MB last-level cache, so table, hash slots and tokens all come
    # from HBM.  The buffer is read, not written, so the caches hold clean
    # lines and the timed kernels pay no write-back of the flush itself.
    cold = None
    if not host:
        flush = torch.ones(1 << 28, dtype=torch.float32, device=dev)
        ce, pe = [], []
        for k in range(COLD_REPS):
            flush.amax()
            e = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
            e[0].record()
            S.lookup(table, X[k % N_BATCHES], cfg.max_n, fgram_ids=fid)
            e[1].record()
            S.gather(fid, rows, out=outs[k % N_BATCHES])
            e[2].record()
            ce.append(e)
            PLAN.add("cold_serial", "k_lookup")
            PLAN.add("cold_serial", G)
        S.embed_pipelined(table, X[0], cfg.max_n, pid[0], None, rows)
        PLAN.add("cold_first_lookup", "k_lookup")
        for k in range(COLD_REPS):
            flush.amax()
            e = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
            e[0].record()
            pipelined_step(k)
            e[1].record()
            pe.append(e)
            PLAN.add("cold_pipelined", "k_pipelined")
        torch.cuda.synchronize()
        del flush
        c_look = float(np.mean([e[0].elapsed_time(e[1]) for e in ce]))
        c_gath = float(np.mean([e[1].elapsed_time(e[2]) for e in ce]))
        c_pipe = float(np.mean([e[0].elapsed_time(e[1]) for e in pe]))
        cold = {"reps": COLD_REPS, "flush_bytes": 1 << 30, "lookup_us": c_look * 1e3,
                "gather_us": c_gath * 1e3,
                "gather_GBps": gather_bytes / (c_gath * 1e-3) / 1e9,
                "device_tokens_per_s": cfg.n_tok / ((c_look + c_gath) * 1e-3),
                "pipelined_us": c_pipe * 1e3,
                "pipelined_GBps": pipe_bytes / (c_pipe * 1e-3) / 1e9,
                "pipelined_device_tokens_per_s": cfg.n_tok / (c_pipe * 1e-3)}

    if args.copy_calibration:
        n = args.copy_calibration << 20
        src = torch.empty(n, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    # Batch 0 once more for the parity check and the match statistics.
    fid0, ml0 = S.lookup(table, X[0], cfg.max_n, want_len=True)
    out0 = S.gather(fid0, rows)
    out0f = S.embed(table, X[0], cfg.max_n, rows)
    S.embed_pipelined(table, X[0], cfg.max_n, pid[0], None, rows)
    out0p = S.embed_pipelined(table, X[1], cfg.max_n, pid[1], pid[0], rows)
    PLAN.add("parity", "k_lookup")
    PLAN.add("parity", G)
    PLAN.add("parity", "k_embed")
    PLAN.add("parity", "k_lookup")
    PLAN.add("parity", "k_pipelined")
    if S.check() != 0:
        raise SystemExit("device error in parity pass")
    torch.cuda.synchronize()

    if host:
        split = split_placement(S, torch, cfg, table, rows, X, fid, outs, K, args.warmup)
    if host:
        # rows cross PCIe once; the output is written to HBM
        read_bytes = cfg.n_tok * cfg.row_bytes
        pcie = read_bytes / (pipe_ms * 1e-3) / 1e9
        ceiling = h2d_ceiling(torch, dev)
        bound, peak, rate = "pcie", PCIE_PEAK_GBPS, pcie
        extra = {"pcie_read_GBps": pcie, "h2d_copy_ceiling_GBps": ceiling,
                 "pct_of_h2d_ceiling": 100.0 * pcie / ceiling,
                 "pcie_inclusive_tokens_per_s": value, "split_placement": split}
        alg_bytes = read_bytes
        nr_rate = read_bytes / (noreuse_ms * 1e-3) / 1e9
    else:
        bound, peak, rate = "hbm", HBM_PEAK_GBPS, pipe_achieved
        extra = {}
        alg_bytes = pipe_bytes
        nr_rate = pipe_bytes / (noreuse_ms * 1e-3) / 1e9

    def control(ms):
        """A gather control's rate: HBM bytes against the HBM peak, or for
        host-pinned rows the bytes read over PCIe against the PCIe peak."""
        if host:
            rate = cfg.n_tok * cfg.row_bytes / (ms * 1e-3) / 1e9
            return {"us": ms * 1e3, "pcie_read_GBps": rate,
                    "pct_pcie_peak": 100.0 * rate / PCIE_PEAK_GBPS, "id_sets": N_BATCHES}
        rate = gather_bytes / (ms * 1e-3) / 1e9
        return {"us": ms * 1e3, "GBps": rate, "pct_hbm_peak": 100.0 * rate / HBM_PEAK_GBPS,
                "id_sets": N_BATCHES}

    result = {
        "metric": METRIC,
        "value": value,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": wall * 1e3 / K,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if cfg.dtype == "bf16" else "f32",
        "data": "synthetic (seeded Zipf(1.1) tokens, planted f-grams, counter-based rows)",
        "config": {"workload": describe(cfg), "B": cfg.B, "T": cfg.T, "tokens": cfg.n_tok,
                   "n_fgrams": cfg.n_fgrams, "max_n": cfg.max_n, "d": cfg.d,
                   "row_bytes": cfg.row_bytes, "placement": cfg.placement,
                   "hash_slots": table.capacity, "slot_bytes": table.slot_bytes,
                   "max_load": args.max_load, "rotating_batches": N_BATCHES},
        "path": "scone_embed_pipelined (one launch per step: gather of batch k, lookup of "
                "batch k+1)",
        "pipelined_us": pipe_ms * 1e3,
        "pipelined_us_sampled_single_launch": pipe_sampled_ms * 1e3,
        "serial_path": {"path": "scone_lookup + scone_gather",
                        "tokens_per_s": cfg.n_tok * K / serial_wall,
                        "ms_per_step": serial_wall * 1e3 / K},
        "lookup_us": lookup_ms * 1e3,
        "gather_us": gather_ms * 1e3,
        "gather": control(gather_ms),
        "fused_path": {"tokens_per_s": cfg.n_tok * K / fused_wall,
                       "ms_per_step": fused_wall * 1e3 / K, **control(embed_ms)},
        "warm_device_tokens_per_s": cfg.n_tok / ((lookup_ms + gather_ms) * 1e-3),
        "cold_caches": cold,
        "uniform_id_gather": control(uniform_ms),
        "sequential_row_gather": control(sequential_ms),
    }
    result.update(extra)
    traffic = measured_traffic(cfg.name, "pipelined")
    result["roofline"] = {
        "bound": bound, "achieved": rate, "peak": peak, "unit": "GB/s", "frac": rate / peak,
        "traffic": None if traffic is None else traffic["traffic_bytes_per_launch"],
        "kernel": "scone_embed_pipelined (k_pipelined)",
        "algorithmic_bytes_per_launch": alg_bytes,
        "cache_assisted": not host,
        "note": ("frac counts the row bytes read over PCIe (the host-pinned table is not "
                 "cached on the device) over the step time; no_reuse is the same kernel over "
                 "uniform random ids" if host else
                 "frac counts algorithmic bytes over the step time on the Zipf workload, whose "
                 "repeated rows the L2s and the 256 MB last-level cache serve in part; "
                 "no_reuse is the same kernel over uniform random ids; traffic is L2-miss "
                 "bytes (FETCH_SIZE + WRITE_SIZE, calibrated), which include last-level-cache "
                 "hits: gfx950's counters do not separate DRAM from that cache"),
        "no_reuse": {"achieved": nr_rate, "frac": nr_rate / peak, "us": noreuse_ms * 1e3,
                     "traffic": None if traffic is None
                     else traffic.get("noreuse_traffic_bytes_per_launch"),
                     "ids": f"uniform random over all {cfg.n_rows} rows, {N_BATCHES} "
                            "rotating sets; the lookup half runs on the real next batch"},
    }
    gtraffic = measured_traffic(cfg.name, "gather")
    result["serial_path"]["gather_traffic"] = (None if gtraffic is None
                                               else gtraffic["traffic_bytes_per_launch"])
    result["uniform_id_gather"]["traffic"] = (None if gtraffic is None
                                              else gtraffic.get("uniform_traffic_bytes_per_launch"))
    etraffic = measured_traffic(cfg.name, "embed")
    result["fused_path"]["traffic"] = (None if etraffic is None
                                       else etraffic["traffic_bytes_per_launch"])
    # Space of the f-gram layer as served: the row table plus the dictionary
    # (the paper's in-memory layout, a dense matrix and a hash index).
    result["space"] = {"row_table_bytes": cfg.n_rows * cfg.row_bytes,
                       "hash_table_bytes": table.capacity * table.slot_bytes,
                       "total_bytes": cfg.n_rows * cfg.row_bytes
                       + table.capacity * table.slot_bytes,
                       "hash_load": table.entries / table.capacity,
                       "hash_entries": table.entries, "fgrams": table.n,
                       "suffix_entries": table.entries - table.n}
    ml = ml0.cpu().numpy()
    result["match"] = match_stats(ml, cfg.max_n)
    result["build_ms"] = build_s * 1e3
    host_pp = probes_per_position(cfg, w, batches_np[0])
    _, _, dev_probes = S.lookup_counted(table, X[0], cfg.max_n)
    PLAN.add("probe_count", "k_lookup", 1)
    result["probes"] = {
        "per_position_kernel_schedule": host_pp,
        "counted": "on the host, replaying the tile lookup's pruned two-lane schedule over "
                   "batch 0 (each probe reads one 64-byte bucket, more only when it is full)",
        "per_position_device": dev_probes / cfg.n_tok,
        "device_counted": "on the device: scone_lookup_counted over batch 0 (the same kernel "
                          "instantiated with a probe counter)",
        "device_equals_host_replay": dev_probes == round(host_pp * cfg.n_tok),
        "max_per_position": max(cfg.max_n - 1, 0)}

    if not args.no_cpu_baseline:
        host_np = rows.tensor().view(torch.uint8).numpy() if host else None
        cb, parity, exp_len, queries = cpu_baseline(cfg, w, batches_np[0], host_np, E,
                                                    fid0.cpu().numpy(), [out0, out0f, out0p],
                                                    args.cpu_seconds)
        parity["match_len_bit_exact"] = bool(np.array_equal(ml, exp_len))
        result["cpu_baseline"] = cb
        result["parity"] = parity
        result["probes"]["oracle_queries_per_position"] = queries / cfg.n_tok
        result["probes"]["oracle_order"] = "longest first, stop at the first hit"
    else:
        result["cpu_baseline"] = None
    if host:
        rows.close()
    return result


def run_decode(args, cfg):
    """Decoding: every step appends one token to each of cfg.B sequences and
    embeds it (scone_decode_step), cfg.T steps in all, eagerly and replayed
    from a HIP graph."""
    import torch
    import paper_2502_01637_amd as S
    from workloads import make_workload, fill_table, torch_dtype, match_stats

    dev = torch.device("cuda", 0)
    t = time.perf_counter()
    w = make_workload(cfg)
    log(f"generated in {time.perf_counter() - t:.1f} s")
    table, build_s = build_table(S, torch, w, dev, args.max_load)
    E = torch.empty((cfg.n_rows, cfg.d), dtype=torch_dtype(cfg), device=dev)
    fill_table(cfg, E)
    Sq, steps = cfg.B, cfg.T
    cap = cfg.max_n - 1
    Xs = torch.from_numpy(np.ascontiguousarray(w.tokens.T)).to(dev)   # [steps, Sq]
    ctx = torch.zeros((Sq, cap), dtype=torch.int32, device=dev)
    clen = torch.zeros(Sq, dtype=torch.int32, device=dev)
    ids = torch.empty((steps, Sq), dtype=torch.int32, device=dev)
    lens = torch.empty((steps, Sq), dtype=torch.int8, device=dev)
    out = torch.empty((Sq, cfg.d), dtype=E.dtype, device=dev)
    torch.cuda.synchronize()

    def run_all(phase):
        clen.fill_(0)
        for s in range(steps):
            S.decode_step(table, ctx, clen, Xs[s], cfg.max_n, E, out, fgram_ids=ids[s],
                          match_len=lens[s])
        PLAN.add(phase, "k_decode", steps)

    # warm-up pass, then the timed eager pass (the host launches every step)
    run_all("decode_warmup")
    if S.check() != 0:
        raise SystemExit("device error in decode warm-up")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    run_all("decode_eager")
    torch.cuda.synchronize()
    eager_wall = time.perf_counter() - t0
    if S.check() != 0:
        raise SystemExit("device error in decode")
    ids_eager = ids.cpu().numpy()

    # the same steps captured once in a HIP graph and replayed
    g = torch.cuda.CUDAGraph()
    clen.fill_(0)
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        for s in range(steps):
            S.decode_step(table, ctx, clen, Xs[s], cfg.max_n, E, out, fgram_ids=ids[s],
                          match_len=lens[s])
    replays, graph_times, graph_ev_ms = 3, [], []
    for r in range(replays):
        clen.fill_(0)
        ids.fill_(-1)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0 = time.perf_counter()
        e0.record()
        g.replay()
        e1.record()
        torch.cuda.synchronize()
        PLAN.add("decode_graph", "k_decode", steps)
        graph_times.append(time.perf_counter() - t0)
        graph_ev_ms.append(e0.elapsed_time(e1))
        if S.check() != 0:
            raise SystemExit("device error in graph replay")
        if not np.array_equal(ids.cpu().numpy(), ids_eager):
            raise SystemExit(f"graph replay {r} differs from the eager decode")
    graph_wall = min(graph_times)
    # per step on the device: HIP events around the whole replay (per-launch
    # events would dominate a step this short)
    step_us = min(graph_ev_ms) * 1e3 / steps

    # Latency against batch size (the paper's inference study reports
    # per-token embedding latency for batches of 1 to 16): the first sq
    # sequences, 256 steps captured in a graph, device time per step.
    sweep = []
    st_n = min(steps, 256)
    for sq in (1, 2, 4, 8, 16, 32, 64, 128, 256):
        if sq > Sq:
            break
        Xq = Xs[:st_n, :sq].contiguous()
        ctx_q = torch.zeros((sq, cap), dtype=torch.int32, device=dev)
        clen_q = torch.zeros(sq, dtype=torch.int32, device=dev)
        out_q = torch.empty((sq, cfg.d), dtype=E.dtype, device=dev)
        ids_q = torch.empty((st_n, sq), dtype=torch.int32, device=dev)
        gq = torch.cuda.CUDAGraph()
        torch.cuda.synchronize()
        with torch.cuda.graph(gq):
            for s in range(st_n):
                S.decode_step(table, ctx_q, clen_q, Xq[s], cfg.max_n, E, out_q,
                              fgram_ids=ids_q[s])
        ev_ms = []
        for r in range(3):
            clen_q.fill_(0)
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            gq.replay()
            e1.record()
            torch.cuda.synchronize()
            PLAN.add(f"decode_sweep_{sq}", "k_decode", st_n)
            ev_ms.append(e0.elapsed_time(e1))
        if S.check() != 0 or not np.array_equal(ids_q.cpu().numpy(), ids_eager[:st_n, :sq]):
            raise SystemExit(f"batch-size sweep at {sq} sequences differs from the eager decode")
        us = min(ev_ms) * 1e3 / st_n
        sweep.append({"sequences": sq, "us_per_step": us, "us_per_token": us / sq})
        del gq

    tokens = Sq * steps
    per_step_bytes = Sq * (2 * cfg.row_bytes + 4)
    kernel_GBps = per_step_bytes / (step_us * 1e-6) / 1e9
    result = {
        "metric": METRIC,
        "value": tokens / graph_wall,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": steps,
        "ms_per_step": graph_wall * 1e3 / steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded Zipf(1.1) tokens, planted f-grams, counter-based rows)",
        "config": {"workload": describe(cfg), "sequences": Sq, "decode_steps": steps,
                   "tokens": tokens, "n_fgrams": cfg.n_fgrams, "max_n": cfg.max_n,
                   "d": cfg.d, "row_bytes": cfg.row_bytes, "placement": "hbm",
                   "context_capacity": cap, "hash_slots": table.capacity},
        "path": "scone_decode_step, one launch per step, replayed from a HIP graph",
        "graph_us_per_step": graph_wall * 1e6 / steps,
        "eager_us_per_step": eager_wall * 1e6 / steps,
        "eager_tokens_per_s": tokens / eager_wall,
        "device_us_per_step": step_us,
        "roofline": {"bound": "hbm", "achieved": kernel_GBps, "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": kernel_GBps / HBM_PEAK_GBPS, "traffic": None,
                     "kernel": "scone_decode_step (k_decode)",
                     "algorithmic_bytes_per_launch": per_step_bytes,
                     "note": "2.1 MB per step: launch-latency bound, not bandwidth bound"},
        "match": match_stats(lens.cpu().numpy(), cfg.max_n),
        "build_ms": build_s * 1e3,
        "batch_sweep": sweep,
    }
    if not args.no_cpu_baseline:
        import oracle
        from workloads import table_rows
        t0 = time.perf_counter()
        o = oracle.OracleTable(w.fgrams, w.lengths, w.ids)
        build_o = time.perf_counter() - t0
        # decode step s of a sequence equals the prefill lookup at position s
        exp_ids, exp_len = o.lookup(w.tokens, cfg.max_n)
        uniq = np.unique(exp_ids)
        compact = table_rows(cfg, torch.from_numpy(uniq.astype(np.int64)),
                             device="cuda").cpu().view(torch.uint8).numpy()
        def one_pass(rows):
            ids_p, _ = o.lookup(rows, cfg.max_n)
            oracle.gather(np.searchsorted(uniq, ids_p).astype(np.int32), compact)

        passes, elapsed = 0, 0.0
        while elapsed < args.cpu_seconds or passes == 0:
            t = time.perf_counter()
            one_pass(w.tokens)
            elapsed += time.perf_counter() - t
            passes += 1
        all_cores = oracle_all_cores(one_pass, w.tokens, args.cpu_seconds / 2)
        # rows of the last step (left in `out` by the graph replay), byte for byte
        last = oracle.gather(np.searchsorted(uniq, exp_ids[:, -1]).astype(np.int32), compact)
        clen.fill_(0)
        g.replay()
        torch.cuda.synchronize()
        PLAN.add("decode_parity", "k_decode", steps)
        result["cpu_baseline"] = {
            "value": passes * tokens / elapsed, "unit": "tokens/s", "cores": 1,
            "kind": "oracle",
            "sample": f"all {tokens} tokens of {describe(cfg)} as one prefill lookup "
                      f"(equal to decoding them), {passes} passes, memcpy gather from a compact "
                      f"host table of the {len(uniq)} referenced rows (id remap timed); "
                      f"dictionary build ({build_o:.1f} s) not timed",
            "seconds": round(elapsed, 3), **host_info(), "all_cores": all_cores}
        result["parity"] = {
            "ids_bit_exact": bool(np.array_equal(ids_eager.T, exp_ids)),
            "match_len_bit_exact": bool(np.array_equal(lens.cpu().numpy().T, exp_len)),
            "last_step_rows_bit_exact": bool(out.cpu().view(torch.uint8).numpy().tobytes()
                                             == last.tobytes()),
            "positions": tokens}
    else:
        result["cpu_baseline"] = None
    return result


def run_tag(args, cfg):
    """Pre-scan tagging of a corpus of many query batches: match length per
    token and the histogram, scone_tag (no ids, no rows)."""
    import torch
    import paper_2502_01637_amd as S
    from workloads import make_workload, query_batches

    dev = torch.device("cuda", 0)
    w = make_workload(cfg)
    corpus_np = np.concatenate(query_batches(w, args.tag_batches))
    table, build_s = build_table(S, torch, w, dev, args.max_load)
    X = torch.from_numpy(corpus_np).to(dev)
    n = X.numel()
    ml = torch.empty(X.shape, dtype=torch.int8, device=dev)
    hist = torch.zeros(S.scone.MAX_FGRAM_LEN + 1, dtype=torch.int64, device=dev)
    for _ in range(args.warmup):
        S.tag(table, X, cfg.max_n, match_len=ml, hist=hist)
    hist.zero_()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record()
    for _ in range(args.steps):
        S.tag(table, X, cfg.max_n, match_len=ml, hist=hist)
    e1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    if S.check() != 0:
        raise SystemExit("device error in tagging")
    h = hist.cpu().numpy() // args.steps
    mean_len = float((h * np.arange(len(h))).sum() / max(h.sum(), 1))
    result = {"metric": "pre-scan tagging tokens/s (longest f-gram length per token), 1 MI355X",
              "value": n * args.steps / wall, "unit": "tokens/s", "n_gpus": 1,
              "steps": args.steps, "warmup": args.warmup,
              "ms_per_step": wall * 1e3 / args.steps, "higher_is_better": True,
              "scaling": "weak", "vs_baseline": None, "dtype": "int32",
              "data": "synthetic corpus (seeded Zipf(1.1) tokens, planted f-grams)",
              "config": {"workload": describe(cfg), "corpus_tokens": n,
                         "sequences": int(X.shape[0]), "T": int(X.shape[1])},
              "device_ms_per_pass": e0.elapsed_time(e1) / args.steps,
              "histogram": {int(k): int(v) for k, v in enumerate(h) if v},
              "average_match_length": mean_len, "build_ms": build_s * 1e3}
    if not args.no_cpu_baseline:
        import oracle
        o = oracle.OracleTable(w.fgrams, w.lengths, w.ids)
        sample = corpus_np[:cfg.B]
        t0 = time.perf_counter()
        passes = 0
        while time.perf_counter() - t0 < args.cpu_seconds or passes == 0:
            _, exp_len = o.lookup(sample, cfg.max_n)
            passes += 1
        el = time.perf_counter() - t0
        result["cpu_baseline"] = {"value": passes * sample.size / el, "unit": "tokens/s",
                                  "cores": 1, "kind": "oracle",
                                  "sample": f"the first {sample.shape[0]} sequences "
                                            f"({sample.size} tokens), {passes} passes",
                                  **host_info()}
        result["parity"] = {"match_len_bit_exact": bool(np.array_equal(
            ml[:cfg.B].cpu().numpy(), exp_len))}
    return result


def run_discover(args, cfg):
    """F-gram discovery over a corpus of many query batches (scone_discover_fgrams)."""
    import torch
    import paper_2502_01637_amd as S
    from workloads import make_workload, query_batches

    dev = torch.device("cuda", 0)
    w = make_workload(cfg)
    corpus_np = np.concatenate(query_batches(w, args.tag_batches))
    X = torch.from_numpy(corpus_np).to(dev)
    n = X.numel()
    K, Sn, mc = cfg.max_len, args.discover_s, 5
    for _ in range(max(1, args.warmup // 5)):
        S.discover_fgrams(X, K, Sn, mc)
    torch.cuda.synchronize()
    times = []
    for _ in range(max(1, args.steps // 10)):
        t0 = time.perf_counter()
        fg, ln, ct = S.discover_fgrams(X, K, Sn, mc)
        torch.cuda.synchronize()
        times.append(time.perf_counter() - t0)
    wall = min(times)
    lens = np.bincount(ln.cpu().numpy(), minlength=K + 1)
    result = {"metric": "f-gram discovery corpus tokens/s (Algorithm 3, K-1 scans), 1 MI355X",
              "value": n / wall, "unit": "tokens/s", "n_gpus": 1, "steps": len(times),
              "warmup": 1, "ms_per_step": wall * 1e3, "higher_is_better": True,
              "scaling": "weak", "vs_baseline": None, "dtype": "int32",
              "data": "synthetic corpus (seeded Zipf(1.1) tokens, planted f-grams)",
              "config": {"workload": describe(cfg), "corpus_tokens": n, "K": K, "S": Sn,
                         "min_count": mc},
              "found": int(len(ln)), "lengths": {int(k): int(v) for k, v in enumerate(lens) if v},
              "min_kept_count": int(ct.min().item()) if len(ct) else 0}
    if not args.no_cpu_baseline:
        from oracle import discovery
        sample = corpus_np[:max(1, (1 << 20) // corpus_np.shape[1])]
        t0 = time.perf_counter()
        cands = discovery.candidates(sample, K, mc)
        el = time.perf_counter() - t0
        result["cpu_baseline"] = {"value": sample.size / el, "unit": "tokens/s", "cores": 1,
                                  "kind": "oracle",
                                  "sample": f"the first {sample.shape[0]} sequences "
                                            f"({sample.size} tokens), counting with numpy",
                                  **host_info()}
        fg2, ln2, ct2 = S.discover_fgrams(torch.from_numpy(sample).to(dev), K, Sn, mc)
        got = {tuple(int(v) for v in r[:L]): int(c) for r, L, c in
               zip(fg2.cpu().numpy(), ln2.cpu().numpy(), ct2.cpu().numpy())}
        oc = dict(cands)
        cmin = min(got.values()) if got else 0
        valid = (len(got) == min(Sn, len(cands)) and all(oc.get(g) == c for g, c in got.items())
                 and all(g in got for g, c in cands if c > cmin))
        result["parity"] = {"sample_top_s_valid": bool(valid)}
    return result


def blas_threads() -> int:
    """Threads of numpy's BLAS pool (the oracle's matrix products run there)."""
    try:
        from threadpoolctl import threadpool_info
        n = [i["num_threads"] for i in threadpool_info() if i.get("user_api") == "blas"]
        return int(max(n)) if n else 1
    except ImportError:
        return 1


def fgram_model_flops(lengths: np.ndarray, d: int, d_ff: int, n_layers: int,
                      products_only: bool = False) -> float:
    """Algorithmic flops of precomputing F for f-grams of these lengths.  A
    full layer costs, per token, 2 (3d^2 + d^2 + 2 d d_ff) for its four
    products and 4 (i + 1) d for position i's scores and weighted sum.  F
    needs only the last token's output, so the last layer computes q, k, v
    for every token but attention, the output projection and the MLP for the
    last position alone.  products_only leaves out the attention terms (the
    flops of the matrix products alone)."""
    if n_layers == 0:
        return 0.0
    n = lengths.astype(np.float64)
    att = 0.0 if products_only else 1.0
    full = n * 2.0 * (4.0 * d * d + 2.0 * d * d_ff) + att * 4.0 * d * n * (n + 1) / 2
    last = n * 2.0 * 3.0 * d * d + 2.0 * (d * d + 2.0 * d * d_ff) + att * 4.0 * d * n
    return float((n_layers - 1) * full.sum() + last.sum())


def run_precompute(args, cfg):
    """Precompute of the f-gram rows (scone_fgram_model_forward) for the whole
    f-gram set of a workload, through a 6-layer d_model 1024 f-gram model."""
    import torch
    import paper_2502_01637_amd as S
    from workloads import make_workload, fill_table, torch_dtype
    from workloads.fgram_model import GPT2_128M, make_params, bf16_bits_to_f64

    if cfg.dtype != "bf16" or cfg.d != GPT2_128M.d or cfg.max_len > GPT2_128M.max_len:
        raise SystemExit("--precompute needs a bf16 workload with d = 1024 and f-grams up to 3")
    mc = GPT2_128M
    dev = torch.device("cuda", 0)
    w = make_workload(cfg)
    fg_np = np.ascontiguousarray(w.fgrams[:, :mc.max_len])
    P = make_params(mc, seed=cfg.seed + 7, recipe="gpt2")
    model = S.FgramModel(P, mc.d, mc.n_heads, mc.d_ff, mc.n_layers, mc.max_len, device=dev)
    E = torch.empty((cfg.n_rows, cfg.d), dtype=torch_dtype(cfg), device=dev)
    fill_table(cfg, E)
    fg, ln, ids = (torch.from_numpy(a).to(dev) for a in (fg_np, w.lengths, w.ids))
    tok = E[:cfg.V]
    for _ in range(args.warmup):
        S.precompute_fgram_rows(model, fg, ln, ids, tok, E)
    torch.cuda.synchronize()
    st = torch.cuda.current_stream()
    evs = []
    t0 = time.perf_counter()
    for _ in range(args.steps):
        e = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        e[0].record(st)
        S.precompute_fgram_rows(model, fg, ln, ids, tok, E)
        e[1].record(st)
        evs.append(e)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    dev_ms = float(np.mean([a.elapsed_time(b) for a, b in evs]))
    flops = fgram_model_flops(w.lengths, mc.d, mc.d_ff, mc.n_layers)
    tflops = flops / (dev_ms * 1e-3) / 1e12
    n = len(w.lengths)
    result = {"metric": "f-gram rows precomputed/s (F = A_fgram over every f-gram), 1 MI355X",
              "value": n * args.steps / wall, "unit": "f-grams/s", "n_gpus": 1,
              "steps": args.steps, "warmup": args.warmup, "ms_per_step": wall * 1e3 / args.steps,
              "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
              "data": "synthetic f-gram set (seeded Zipf(1.1)), random GPT-2-style weights",
              "config": {"workload": f"{describe(cfg)}; f-gram model d_model {mc.d}, "
                                     f"{mc.n_heads} heads, ffw {mc.d_ff}, {mc.n_layers} layers",
                         "n_fgrams": n, "tokens": int(w.lengths.sum()), "d": mc.d,
                         "d_ff": mc.d_ff, "n_layers": mc.n_layers, "n_heads": mc.n_heads},
              "device_ms_per_step": dev_ms, "flops_per_step": flops, "TFLOPs": tflops,
              "product_flops_per_step": fgram_model_flops(w.lengths, mc.d, mc.d_ff,
                                                          mc.n_layers, products_only=True),
              "roofline": {"bound": "mfma", "achieved": tflops, "peak": MFMA_BF16_PEAK_TFLOPS,
                           "unit": "TFLOP/s", "frac": tflops / MFMA_BF16_PEAK_TFLOPS,
                           "traffic": None,
                           "kernel": "scone_fgram_model_forward (all kernels of one call)",
                           "algorithmic_flops_per_launch": flops}}
    result["cpu_baseline"] = None
    if not args.no_cpu_baseline:
        # The CPU-baseline leg: parity of a sample of rows with the oracle (the
        # bar of the GPU parity tests, 3 eps(L) per row), then the oracle timed.
        from oracle import fgram_model as orc
        rng = np.random.default_rng(0)
        sample = rng.choice(n, 32, replace=False)
        T64 = E[:cfg.V].float().cpu().numpy().astype(np.float64)
        P64 = {k: bf16_bits_to_f64(v) for k, v in P.items()}
        ref = orc.forward(fg_np[sample], w.lengths[sample], T64, P64, mc.n_layers, mc.n_heads)
        got = E[torch.from_numpy(w.ids[sample].astype(np.int64)).to(dev)].float().cpu().numpy()
        rel = np.linalg.norm(got - ref, axis=1) / np.linalg.norm(ref, axis=1)
        bar = 3 * 2.0 ** -9 * np.sqrt((5 * mc.n_layers + 2) / 3)
        result["parity"] = {"sample_rows": len(sample), "max_row_rel_err": float(rel.max()),
                            "bar": bar, "ok": bool(rel.max() <= bar)}
        cs = rng.choice(n, 64, replace=False)
        t0 = time.perf_counter()
        reps = 0
        while True:
            orc.forward(fg_np[cs], w.lengths[cs], T64, P64, mc.n_layers, mc.n_heads)
            reps += 1
            if time.perf_counter() - t0 >= min(args.cpu_seconds, 10.0):
                break
        el = time.perf_counter() - t0
        result["cpu_baseline"] = {"value": reps * len(cs) / el, "unit": "f-grams/s",
                                  "cores": blas_threads(), "kind": "oracle",
                                  "sample": f"{len(cs)} f-grams, repeated {reps} times, "
                                            "float64 numpy (BLAS threads)",
                                  "cpu_model": host_info()["cpu_model"]}
    return result


# ------------------------------------------------------------ profiles ----
# rocprofv3 writes one csv row per dispatch (kernel trace) or per dispatch and
# counter (counter collection).  A run made with --plan-out also leaves the
# plan of its library dispatches; the reducers below walk the csv's library
# kernels in dispatch order against that plan, so each figure is taken over
# the timed dispatches of one phase only.

BUILD_KERNELS = ("k_count_long", "k_insert", "k_verify", "k_mark", "k_count_used")


def _short(name: str) -> str:
    n = re.sub(r"\(anonymous namespace\)::", "", name)
    return n.split("(")[0].replace("void ", "").replace("scone::", "").strip()


def _library_dispatches(rows):
    """This library's dispatches after the table build, in dispatch order."""
    lib = sorted((r for r in rows if "scone::" in r["Kernel_Name"]),
                 key=lambda r: int(r["Dispatch_Id"]))
    i = 0
    while i < len(lib) and _short(lib[i]["Kernel_Name"]).startswith(BUILD_KERNELS):
        i += 1
    return lib[i:]


def _by_phase(rows, plan):
    """{phase: [row, ...]} after checking every dispatch against the plan."""
    lib = _library_dispatches(rows)
    if len(lib) < len(plan["entries"]):
        raise SystemExit(f"the csv has {len(lib)} library dispatches after the build, "
                         f"the plan {len(plan['entries'])}")
    out = {}
    for (phase, kernel), r in zip(plan["entries"], lib):
        if not _short(r["Kernel_Name"]).startswith(kernel):
            raise SystemExit(f"dispatch {r['Dispatch_Id']} is {_short(r['Kernel_Name'])}, "
                             f"the plan expects {kernel} ({phase})")
        out.setdefault(phase, []).append(r)
    return out


def _read_csv(path):
    import csv
    with open(path) as f:
        return list(csv.DictReader(f))


def reduce_trace(trace_csv, plan_path, bench_json, out_md, profile_cmd, bench_plain=False):
    """profiles/<workload>_kernel_trace.md from a --kernel-trace run."""
    import statistics as st
    plan = json.load(open(plan_path))
    rows = _read_csv(trace_csv)
    for r in rows:
        r["ns"] = int(r["End_Timestamp"]) - int(r["Start_Timestamp"])
    ph = _by_phase(rows, plan)
    bench = None
    for line in (open(bench_json) if bench_json else []):
        if line.startswith('{"metric"'):
            bench = json.loads(line)
    lib = [r for r in rows if "scone::" in r["Kernel_Name"]]
    by = {}
    for r in lib:
        by.setdefault(_short(r["Kernel_Name"]), []).append(r)
    us = lambda L: st.mean(x["ns"] for x in L) / 1e3
    med = lambda L: st.median(x["ns"] for x in L) / 1e3
    span = lambda L: f"{L[0]['Dispatch_Id']}-{L[-1]['Dispatch_Id']}"
    cfgname = plan["config"]
    srcs = kernel_sources(set(by))
    L = [f"# Kernel trace: {cfgname} ({plan['workload']})\n",
         "Command (one MI355X, `<repo>` the repository root):\n", f"    {profile_cmd}\n",
         "Reduced with `python bench.py --reduce-trace <out>/run_kernel_trace.csv "
         "--plan <plan.json> --bench-json <bench stdout> --out <this file>`.\n",
         "Per-kernel durations from the kernel-trace csv (ns); only this library's kernels.",
         "Sources (sha1): " + ", ".join(f"{s} {source_sha(s)}" for s in srcs) + ".\n", "```"]
    for name, rs in sorted(by.items(), key=lambda kv: -sum(x["ns"] for x in kv[1])):
        ns = [x["ns"] for x in rs]
        r0 = rs[0]
        L.append(f"{name[:58]:58s} calls={len(rs):4d} avg_ns={st.mean(ns):11.1f} "
                 f"med_ns={st.median(ns):10.1f} min_ns={min(ns):9d} max_ns={max(ns):9d} "
                 f"grid={r0['Grid_Size_X']} wg={r0['Workgroup_Size_X']} vgpr={r0['VGPR_Count']} "
                 f"lds={r0['LDS_Block_Size']}")
    L += ["```\n", "By phase (dispatch numbers from the csv; warm-up and parity launches "
                    "left out):\n", "```"]
    for phase, rs_all in ph.items():
        if phase.endswith(("_warmup", "_first_lookup", "parity")):
            continue
        groups = {}
        for r in rs_all:
            groups.setdefault(_short(r["Kernel_Name"]), []).append(r)
        for name, rs in groups.items():
            L.append(f"{phase:17s} {name[:40]:40s} n={len(rs):5d} (dispatches {span(rs)}) "
                     f"mean {us(rs):9.2f} us  median {med(rs):9.2f} us")
    L.append("```\n")
    where = ("a run of the same command without the profiler, in the same call" if bench_plain
             else "HIP events in the same run, under the profiler")
    if bench and "pipelined_us" in bench:
        L.append(f"bench.py's own figures ({where}): "
                 f"pipelined step {bench['pipelined_us']:.1f} us (device time of the timed "
                 f"region per step), no-reuse pipelined step "
                 f"{bench['roofline']['no_reuse']['us']:.1f} us, serial lookup "
                 f"{bench['lookup_us']:.1f} us + gather {bench['gather_us']:.1f} us, "
                 f"uniform-id gather {bench['uniform_id_gather']['us']:.1f} us, contiguous "
                 f"rows {bench['sequential_row_gather']['us']:.1f} us; headline "
                 f"{bench['value'] / 1e6:.1f} M tokens/s, roofline frac "
                 f"{bench['roofline']['frac']:.3f} (no reuse "
                 f"{bench['roofline']['no_reuse']['frac']:.3f}).\n")
    elif bench and "graph_us_per_step" in bench:
        sweep = ", ".join(f"{x['sequences']}: {x['us_per_step']:.2f}" for x in bench["batch_sweep"])
        L.append(f"bench.py's own figures ({where}): "
                 f"{bench['device_us_per_step']:.2f} us per step on the device (HIP events "
                 f"around each graph replay), {bench['eager_us_per_step']:.1f} us per step when "
                 f"the host launches every step; batch-size sweep (sequences: us per step) "
                 f"{sweep}.  The tracer adds its own work between dispatches, so for steps "
                 "this short the figures of a run without it are the ones to quote.\n")
    open(out_md, "w").write("\n".join(L) + "\n")
    print(f"wrote {out_md}")


def reduce_counters(fetch_csv, write_csv, plan_path, fetch_cmd, write_cmd, out_dir):
    """profiles/<kernel>_<workload>_traffic.md from a FETCH_SIZE run and a
    WRITE_SIZE run of the same bench.py command (with --copy-calibration)."""
    import statistics as st
    from workloads import CONFIGS
    plan = json.load(open(plan_path))
    cfgname = plan["config"]
    cfg = CONFIGS[cfgname]
    per = {}
    copies = {}
    for ctr, path in (("FETCH_SIZE", fetch_csv), ("WRITE_SIZE", write_csv)):
        rows = [r for r in _read_csv(path) if r["Counter_Name"] == ctr]
        per[ctr] = _by_phase(rows, plan)
        cp = sorted((r for r in rows if "copyBuffer" in r["Kernel_Name"]),
                    key=lambda r: int(r["Dispatch_Id"]))
        big = max(int(r["Grid_Size"]) for r in cp)
        copies[ctr] = [float(r["Counter_Value"]) for r in cp if int(r["Grid_Size"]) == big][-5:]
    kib = plan["copy_calibration_mib"] * 1024.0
    fscale = kib / st.mean(copies["FETCH_SIZE"])
    wscale = kib / st.mean(copies["WRITE_SIZE"])

    def mean_kib(ctr, phase, kernel):
        v = [float(r["Counter_Value"]) for r in per[ctr].get(phase, [])
             if _short(r["Kernel_Name"]).startswith(kernel)]
        return st.mean(v) if v else None

    def traffic(phase, kernel):
        f, w = mean_kib("FETCH_SIZE", phase, kernel), mean_kib("WRITE_SIZE", phase, kernel)
        if f is None or w is None:
            return None, None, None
        return f, w, int(round(f * 1024 * fscale + w * 1024 * wscale))

    G = "k_gather"
    specs = {
        "pipelined": ("k_pipelined", [("pipelined_timed", "traffic_bytes_per_launch", "Zipf workload"),
                                      ("noreuse_timed", "noreuse_traffic_bytes_per_launch",
                                       "uniform random ids (no reuse)")],
                      cfg.gather_bytes() + cfg.n_tok * 8,
                      f"2 x {cfg.row_bytes} B rows + 4 B id read + 4 B token read + 4 B id written"),
        "gather": (G, [("serial_timed", "traffic_bytes_per_launch", "Zipf workload"),
                       ("uniform_timed", "uniform_traffic_bytes_per_launch",
                        "uniform random ids (no reuse)"),
                       ("contiguous_timed", "contiguous_traffic_bytes_per_launch",
                        "contiguous rows")],
                   cfg.gather_bytes(), f"2 x {cfg.row_bytes} B rows + 4 B id"),
        "embed": ("k_embed", [("fused_timed", "traffic_bytes_per_launch", "Zipf workload")],
                  cfg.gather_bytes(), f"4 B token + 2 x {cfg.row_bytes} B rows"),
    }
    lf, lw, lt = traffic("serial_timed", "k_lookup")
    for key, (kernel, phases, alg, algtxt) in specs.items():
        rec = {"config": cfgname, "kernel": kernel, "source_sha1": source_sha(*KERNEL_SOURCES[key]),
               "fetch_scale": round(fscale, 5), "write_scale": round(wscale, 5)}
        lines = []
        for phase, field, what in phases:
            f, w, t = traffic(phase, kernel)
            if t is None:
                continue
            rec[field] = t
            if field == "traffic_bytes_per_launch":
                rec["fetch_kib_per_dispatch"] = round(f, 1)
                rec["write_kib_per_dispatch"] = round(w, 1)
            lines.append(f"{phase:17s} ({what}): FETCH_SIZE {f:10.1f} KiB x {fscale:.4f} + "
                         f"WRITE_SIZE {w:10.1f} KiB x {wscale:.4f} = {t / 1e6:8.1f} MB per launch")
        L = [f"# L2-miss traffic of {kernel} on {cfgname} ({plan['workload']})\n",
             "Two counter passes, each its own run of the same command (one MI355X):\n",
             f"    {fetch_cmd}", f"    {write_cmd}\n",
             "Reduced with `python bench.py --reduce-counters <fetch csv> <write csv> "
             "--plan <plan.json>`.\n",
             "FETCH_SIZE and WRITE_SIZE count the bytes the L2s request from and write to "
             "the memory fabric.  On MI355X the 256 MB last-level cache (Infinity Cache) sits "
             "behind that fabric, so these are L2-miss bytes: they include last-level-cache "
             "hits, and no counter gfx950 exposes to rocprofv3 separates DRAM traffic from "
             "them (its counter list has no data-fabric or memory-controller block).  With "
             "uniform random ids over a table far larger than that cache the two coincide.\n",
             f"Calibration: the run's last five plain device copies of "
             f"{plan['copy_calibration_mib']} MiB read FETCH_SIZE = "
             f"{st.mean(copies['FETCH_SIZE']):.1f} KiB and WRITE_SIZE = "
             f"{st.mean(copies['WRITE_SIZE']):.1f} KiB for {kib:.0f} KiB moved each way, so "
             f"FETCH_SIZE is scaled by {fscale:.4f} and WRITE_SIZE by {wscale:.4f}.\n",
             f"Means over each phase's {plan['steps']} timed dispatches:\n", "```"] + lines + [
             "```\n",
             f"Algorithmic bytes per launch: {alg / 1e6:.1f} MB ({cfg.n_tok} tokens x "
             f"({algtxt})).",
             (f"The standalone lookup kernel moves {lt / 1e6:.1f} MB per launch in the same run "
              f"(FETCH {lf:.1f} KiB, WRITE {lw:.1f} KiB).\n" if lt else ""),
             "TRAFFIC " + json.dumps(rec)]
        out = os.path.join(out_dir, f"{key}_{cfgname}_traffic.md")
        open(out, "w").write("\n".join(L) + "\n")
        print(f"wrote {out}")


def reduce_precompute(trace_csv, bench_json, pmc_csv, out_md, trace_cmd, pmc_cmd):
    """profiles/fgram_model_<workload>_kernel_trace.md from a --kernel-trace run
    of `bench.py --precompute` (one warm-up and two timed calls) and, when
    given, a counter run with GRBM_GUI_ACTIVE, SQ_VALU_MFMA_BUSY_CYCLES,
    SQ_INSTS_MFMA and SQ_BUSY_CYCLES."""
    import collections
    import statistics as st
    bench = [json.loads(ln) for ln in open(bench_json) if ln.startswith('{"metric"')][0]
    calls = bench["steps"] + bench["warmup"]
    rows = [r for r in _read_csv(trace_csv) if "scone::" in r["Kernel_Name"]]
    for r in rows:
        r["ns"] = int(r["End_Timestamp"]) - int(r["Start_Timestamp"])
        r["short"] = _short(r["Kernel_Name"]).replace("gemm::", "")

    def cls(name):
        return {"k_gemm<0": "products: q/k/v (bias)", "k_gemm<1": "products: fc1 (bias+GELU)",
                "k_gemm<2": "products: o-proj / fc2 (residual)"}.get(name[:8], name.split("<")[0])

    by, tot = collections.defaultdict(list), collections.defaultdict(float)
    for r in rows:
        by[(r["short"], r["Grid_Size_X"])].append(r)
        tot[cls(r["short"])] += r["ns"]
    prod_ns = sum(v for k, v in tot.items() if k.startswith("products")) / calls
    all_ns = sum(tot.values()) / calls
    L = ["# Kernel trace: precompute of F (scone_fgram_model_forward)\n",
         f"Workload: {bench['config']['workload']}; {bench['config']['n_fgrams']} f-grams, "
         f"{bench['config']['tokens']} tokens; {bench['warmup']} warm-up and "
         f"{bench['steps']} timed calls.\n",
         "Commands (one MI355X, `<repo>` the repository root):\n", f"    {trace_cmd}"]
    if pmc_csv:
        L.append(f"    {pmc_cmd}")
    L += ["", "Reduced with `python bench.py --reduce-precompute <trace csv> --bench-json "
          "<bench stdout> [--pmc <counter csv>] --out <this file>`.\n",
          "Sources (sha1): " + ", ".join(f"{x} {source_sha(x)}" for x in
                                         ("fgram_model.hip", "gemm_bf16.h")) + ".\n",
          "Per-kernel durations (ns), one line per (kernel, grid):\n", "```"]
    for (name, grid), rs in sorted(by.items(), key=lambda kv: -sum(x["ns"] for x in kv[1])):
        v = [x["ns"] for x in rs]
        L.append(f"{name[:40]:40s} calls={len(rs):5d} avg_ns={st.mean(v):10.1f} "
                 f"med_ns={st.median(v):10.1f} min_ns={min(v):9d} max_ns={max(v):9d} "
                 f"grid={grid} wg={rs[0]['Workgroup_Size_X']} vgpr={rs[0]['VGPR_Count']} "
                 f"lds={rs[0]['LDS_Block_Size']}")
    L += ["```\n", f"Device time per call by kernel class (sum over the {calls} calls / "
                   f"{calls}):\n", "```"]
    for k, v in sorted(tot.items(), key=lambda kv: -kv[1]):
        L.append(f"{k:36s} {v / calls / 1e6:8.2f} ms/call {100 * v / sum(tot.values()):6.1f}%")
    L += [f"{'total':36s} {all_ns / 1e6:8.2f} ms/call", "```\n"]
    pf = bench["product_flops_per_step"]
    L.append(f"Matrix products: {pf / 1e12:.1f} TFLOP of algorithmic work per call in "
             f"{prod_ns / 1e6:.1f} ms of k_gemm time, {pf / prod_ns / 1e3:.0f} TFLOP/s "
             f"({100 * pf / prod_ns / 1e3 / 2500:.1f}% of the 2.5 PFLOP/s dense bf16 peak).  "
             f"Whole call: {bench['flops_per_step'] / 1e12:.1f} TFLOP in {all_ns / 1e6:.1f} ms "
             f"of kernel time, {bench['flops_per_step'] / all_ns / 1e3:.0f} TFLOP/s; bench.py's "
             f"HIP events around each call read {bench['device_ms_per_step']:.1f} ms "
             f"({bench['TFLOPs']:.0f} TFLOP/s).\n")
    if pmc_csv:
        pm = collections.defaultdict(dict)
        for r in _read_csv(pmc_csv):
            if "k_gemm" not in r["Kernel_Name"]:
                continue
            pm[int(r["Dispatch_Id"])][r["Counter_Name"]] = float(r["Counter_Value"])
        # GRBM_GUI_ACTIVE counts each of the 8 XCDs' active cycles;
        # SQ_VALU_MFMA_BUSY_CYCLES sums the matrix-core busy cycles of all
        # 1,024 SIMDs (256 compute units x 4).
        gui = sum(d.get("GRBM_GUI_ACTIVE", 0) for d in pm.values()) / 8
        busy = sum(d.get("SQ_VALU_MFMA_BUSY_CYCLES", 0) for d in pm.values()) / 1024
        mf = sum(d.get("SQ_INSTS_MFMA", 0) for d in pm.values())
        L.append(f"Counter run over the products' {len(pm)} dispatches: the matrix cores are "
                 f"busy {100 * busy / max(gui, 1):.1f}% of the active cycles "
                 f"(SQ_VALU_MFMA_BUSY_CYCLES / 1,024 SIMDs over GRBM_GUI_ACTIVE / 8 XCDs); "
                 f"{mf:.4g} MFMA instructions.\n")
    open(out_md, "w").write("\n".join(L) + "\n")
    print(f"wrote {out_md}")


def kernel_sources(names):
    """The library sources a set of kernels is built from: each file that
    defines one of them (``name<...>`` or ``name``), the local headers those
    files include, and the runtime (the error word)."""
    import re
    csrc = os.path.join(ROOT, "paper_2502_01637_amd", "csrc")
    files = sorted(f for f in os.listdir(csrc) if f.endswith((".hip", ".h")))
    text = {f: open(os.path.join(csrc, f)).read() for f in files}
    base = {n.split("<")[0] for n in names}
    out = {"runtime.hip"}
    for f in files:
        if any(re.search(r"\bvoid\s+" + re.escape(b) + r"\s*\(", text[f]) for b in base):
            out.add(f)
    todo = list(out)
    while todo:
        for h in re.findall(r'#include "([\w.]+)"', text[todo.pop()]):
            if h in text and h not in out:
                out.add(h)
                todo.append(h)
    return sorted(out)


def reduce_kernels(trace_csv, bench_json, plain_json, out_md, title, desc, cmd):
    """A per-kernel summary of a --kernel-trace run of any bench.py mode (the
    tagger and discovery summaries): this library's kernels by (name, grid),
    their time per call, and bench.py's own figures from the profiled run and
    from a run without the profiler."""
    import collections
    import statistics as st
    rows = [r for r in _read_csv(trace_csv) if "scone::" in r["Kernel_Name"]]
    by = collections.defaultdict(list)
    for r in rows:
        r["ns"] = int(r["End_Timestamp"]) - int(r["Start_Timestamp"])
        by[(_short(r["Kernel_Name"]), r["Grid_Size_X"])].append(r)
    srcs = kernel_sources({name for name, _ in by})
    L = [f"# Kernel trace: {title}\n", f"{desc}\n", "Command (one MI355X, `<repo>` the repository root):\n",
         f"    {cmd}\n", "Reduced with `python bench.py --reduce-kernels <trace csv> --bench-json "
         "<profiled run's stdout> --plain-json <stdout of a run without the profiler> ...`.\n",
         "Sources (sha1): " + ", ".join(f"{x} {source_sha(x)}" for x in srcs) + ".\n",
         "Per-kernel durations (ns), this library's kernels only:\n", "```"]
    for (name, grid), rs in sorted(by.items(), key=lambda kv: -sum(x["ns"] for x in kv[1])):
        v = [x["ns"] for x in rs]
        L.append(f"{name[:48]:48s} calls={len(rs):5d} avg_ns={st.mean(v):11.1f} "
                 f"med_ns={st.median(v):10.1f} min_ns={min(v):9d} max_ns={max(v):9d} "
                 f"grid={grid} wg={rs[0]['Workgroup_Size_X']} vgpr={rs[0]['VGPR_Count']} "
                 f"lds={rs[0]['LDS_Block_Size']}")
    L.append("```\n")

    def figures(path, where):
        if not path:
            return
        b = [json.loads(ln) for ln in open(path) if ln.startswith('{"metric"')][0]
        extra = "".join(f", {k} {b[k]:.4g}" for k in ("device_ms_per_pass", "ms_per_step")
                        if k in b)
        L.append(f"bench.py {where}: {b['value']:.4g} {b['unit']}{extra}.")

    figures(bench_json, "under the profiler")
    figures(plain_json, "without the profiler (a separate run in the same call)")
    L.append("")
    open(out_md, "w").write("\n".join(L) + "\n")
    print(f"wrote {out_md}")


CACHE_COUNTERS = ("TCC_HIT_sum", "TCC_MISS_sum", "TCP_UTCL1_TRANSLATION_MISS_sum",
                  "TCP_UTCL1_TRANSLATION_HIT_sum")


def reduce_cache(pmc_csv, plan_path, out_md, profile_cmd):
    """profiles/probe_cache_<workload>.md from one counter pass with the L2
    hit/miss and first-level translation counters."""
    import statistics as st
    plan = json.load(open(plan_path))
    rows = _read_csv(pmc_csv)
    per = {c: _by_phase([r for r in rows if r["Counter_Name"] == c], plan)
           for c in CACHE_COUNTERS}
    n_tok = None
    from workloads import CONFIGS
    cfg = CONFIGS[plan["config"]]
    n_tok = cfg.n_tok
    labels = [("serial_timed", "k_lookup", "lookup (serial)"),
              ("pipelined_timed", "k_pipelined", "pipelined step, Zipf ids"),
              ("noreuse_timed", "k_pipelined", "pipelined step, uniform ids"),
              ("serial_timed", "k_gather", "gather, Zipf ids (serial)"),
              ("fused_timed", "k_embed", "fused lookup+gather"),
              ("uniform_timed", "k_gather", "gather, uniform ids"),
              ("contiguous_timed", "k_gather", "gather, contiguous rows")]
    L = [f"# L2 hit rate and address-translation misses: {plan['config']} ({plan['workload']})\n",
         "One counter pass (one MI355X; TCC_HIT/TCC_MISS are L2 requests summed over all "
         "channels of the eight XCDs, TCP_UTCL1_TRANSLATION_* the first-level address "
         "translation caches of the compute units):\n", f"    {profile_cmd}\n",
         "Reduced with `python bench.py --reduce-cache <counter csv> --plan <plan.json> "
         "--out <this file>`.\n",
         f"Means per dispatch over each phase's {plan['steps']} timed launches "
         f"({n_tok} tokens per launch):\n", "```"]
    for phase, kern, label in labels:
        vals = {}
        for c in CACHE_COUNTERS:
            v = [float(r["Counter_Value"]) for r in per[c].get(phase, [])
                 if _short(r["Kernel_Name"]).startswith(kern)]
            vals[c] = st.mean(v) if v else None
        if any(v is None for v in vals.values()):
            continue
        h, mi = vals["TCC_HIT_sum"], vals["TCC_MISS_sum"]
        tm = vals["TCP_UTCL1_TRANSLATION_MISS_sum"]
        L.append(f"{label:30s} {kern:12s} L2 requests {h + mi:11.0f}  L2 hit "
                 f"{h / max(h + mi, 1):6.1%}  UTCL1 misses {tm:9.0f} ({tm / n_tok:.3f} per token)")
    L.append("```\n")
    open(out_md, "w").write("\n".join(L) + "\n")
    print(f"wrote {out_md}")


def reduce_main(argv):
    ap = argparse.ArgumentParser(description="reduce rocprofv3 csv output of a bench.py run")
    ap.add_argument("--reduce-trace", metavar="KERNEL_TRACE_CSV")
    ap.add_argument("--reduce-counters", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"))
    ap.add_argument("--reduce-cache", metavar="COUNTER_CSV")
    ap.add_argument("--reduce-precompute", metavar="KERNEL_TRACE_CSV")
    ap.add_argument("--reduce-kernels", metavar="KERNEL_TRACE_CSV")
    ap.add_argument("--plain-json")
    ap.add_argument("--title", default="")
    ap.add_argument("--desc", default="")
    ap.add_argument("--pmc", metavar="COUNTER_CSV")
    ap.add_argument("--pmc-cmd", default="")
    ap.add_argument("--plan")
    ap.add_argument("--bench-json")
    ap.add_argument("--out")
    ap.add_argument("--profile-cmd", default="", help="the profiler command (trace)")
    ap.add_argument("--bench-plain", action="store_true",
                    help="--bench-json comes from a run without the profiler")
    ap.add_argument("--fetch-cmd", default="")
    ap.add_argument("--write-cmd", default="")
    ap.add_argument("--out-dir", default=os.path.join(ROOT, "profiles"))
    a = ap.parse_args(argv)
    if a.reduce_trace:
        reduce_trace(a.reduce_trace, a.plan, a.bench_json, a.out, a.profile_cmd, a.bench_plain)
    if a.reduce_counters:
        reduce_counters(a.reduce_counters[0], a.reduce_counters[1], a.plan, a.fetch_cmd,
                        a.write_cmd, a.out_dir)
    if a.reduce_cache:
        reduce_cache(a.reduce_cache, a.plan, a.out, a.profile_cmd)
    if a.reduce_kernels:
        reduce_kernels(a.reduce_kernels, a.bench_json, a.plain_json, a.out, a.title, a.desc,
                       a.profile_cmd)
    if a.reduce_precompute:
        reduce_precompute(a.reduce_precompute, a.bench_json, a.pmc, a.out, a.profile_cmd,
                          a.pmc_cmd)


def main():
    if any(a in ("--reduce-trace", "--reduce-counters", "--reduce-cache", "--reduce-precompute",
                 "--reduce-kernels") for a in sys.argv[1:]):
        reduce_main(sys.argv[1:])
        return
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default=DEFAULT_CONFIG)
    ap.add_argument("--max-load", type=float, default=0.25,
                    help="hash-table load target (slots >= entries / max_load)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--tag", action="store_true",
                    help="pre-scan tagging of a corpus of --tag-batches query batches")
    ap.add_argument("--tag-batches", type=int, default=64)
    ap.add_argument("--discover", action="store_true",
                    help="f-gram discovery over a corpus of --tag-batches query batches")
    ap.add_argument("--discover-s", type=int, default=1_000_000)
    ap.add_argument("--precompute", action="store_true",
                    help="time the precompute of the f-gram rows by the f-gram model")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="also run a plain device copy of MIB MiB (counter calibration)")
    ap.add_argument("--plan-out", metavar="FILE",
                    help="write the run's library dispatches by phase (for the reducers)")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              f"(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import torch
    from workloads import CONFIGS
    if args.config not in CONFIGS:
        raise SystemExit(f"unknown config {args.config}; choose from {sorted(CONFIGS)}")
    cfg = CONFIGS[args.config]
    torch.cuda.set_device(0)
    log("workload:", describe(cfg))
    if args.precompute:
        if "--steps" not in sys.argv:
            args.steps = 5
        if "--warmup" not in sys.argv:
            args.warmup = 1
        result = run_precompute(args, cfg)
    elif args.discover:
        result = run_discover(args, cfg)
    elif args.tag:
        result = run_tag(args, cfg)
    elif cfg.decode:
        result = run_decode(args, cfg)
    else:
        result = run_prefill(args, cfg)
    if args.plan_out:
        json.dump({"config": cfg.name, "workload": describe(cfg), "steps": args.steps,
                   "warmup": args.warmup, "copy_calibration_mib": args.copy_calibration,
                   "argv": sys.argv, "entries": PLAN.entries}, open(args.plan_out, "w"))
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
