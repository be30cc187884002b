"""Throughput of FineMoE expert-map matching + prefetch selection on one MI355X.

One step = one pass of the whole hot path over one query batch that is
already resident in HBM: the batched cosine search over the store (trajectory
search, Eq. 5, and/or semantic search, Eq. 4, with ranking fused in), then the
prefetch-set selection (Section 4.3, Eq. 6-8) for every (query, layer) row,
each half of the batch through its match-and-select call (the merge of the
search's partial lists and the selection in one launch).

Default workload: the largest one that fits one GPU, the mixed Qwen1.5-MoE
batch (1,000,000 stored maps of 24 x 60 bfloat16, each with a 2048-dimension
bfloat16 embedding; 1,024 queries, 512 semantic at full depth and 512
trajectory with prefix depths U{1..23}; top-1, threshold 0.8, at most 8
experts), both searches and the selection in one step.  ``--config`` selects
another workload.

Prints ONE JSON line.  ``roofline`` refers to the dominant kernel (the scan
kernel of the match call; for the mixed workload the slower of the two
scans, the other one's figures under ``roofline.other``), timed by HIP events
that the library records right around its launch on the stream it runs on
(fm_debug_scan_events); ``calls_us`` is a step's match-and-select calls
(staging, scan, merge and selection).  ``cpu_baseline`` is the CPU oracle timed on a bounded sample of
the same batch.

``--path dedup`` measures the deduplicating insert instead (Section 4.4):
batches of 256 new iterations into the full 100,000-entry store of d = 4096
embeddings, prefetch distance 3; one step = one insert call.

``--path step`` measures the incremental per-layer trajectory re-search
(Section 4.2.2): 64 queries against the 50,000-map Qwen store, one step = one
pass of L - d = 18 searches (prefix depths 1 .. 18), each an fm_traj_step
call; the same searches as full re-scans are timed for reference.

``--path order`` measures the Section 4.5 prefetch ordering of a workload's
selected sets (``--config``; one step = one fm_priority_order call).

``--path capacity`` runs the store-capacity study (Section 6 sensitivity):
mean best-match similarity, the misses of the selected sets and the full-map
similarity at the sphere-covering sizes 2LJ and LJ ln(LJ) / 2 (Section 4.4),
for stores of 1,000 .. 1,000,000 Qwen-shaped iterations.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
BF16_MFMA_PEAK_TFS = 2500.0    # dense bf16 MFMA
FP32_MFMA_PEAK_TFS = 157.3     # dense fp32 MFMA

# HBM traffic of the dominant kernel per launch, from two rocprofv3 --pmc runs
# (FETCH_SIZE, then WRITE_SIZE, KiB per dispatch) of this bench, each scaled by
# what the same counter reads for a plain copy kernel of 256 MiB
# (profiles/traffic_counters.md).  Only for kernels unchanged since.
COPY_BYTES_KIB = 262144.0
COPY_COUNTERS_KIB = {"FETCH_SIZE": 131083.5, "WRITE_SIZE": 262144.0}
COUNTERS_KIB = {
    # workload: {kernel: (FETCH_SIZE KiB, WRITE_SIZE KiB) per dispatch}
    "mixtral_traj_n1k": {"k_traj_scan": (610.1, 10.9)},
    "qwen_traj_n50k_b64": {"k_traj_scan": (138797.4, 128.0)},
    "semantic_d4096_n100k_b256": {"k_sem_mm": (417145.2, 512.0)},
    "phi_traj_top4_n200k_b512": {"k_traj_scan": (333131.3, 1012.0)},
    "qwen_mixed_bf16_n1m_b1024": {"k_sem_mm": (2657013.4, 512.0), "k_traj_mm": (2276903.6, 557.0)},
}


def counter_traffic(workload, kernel):
    fw = COUNTERS_KIB.get(workload, {}).get(kernel)
    if fw is None:
        return None
    fetch, write = fw
    kib = (fetch * COPY_BYTES_KIB / COPY_COUNTERS_KIB["FETCH_SIZE"]
           + write * COPY_BYTES_KIB / COPY_COUNTERS_KIB["WRITE_SIZE"])
    return kib * 1024.0


def scan_kernels(s):
    """The scan kernel the library launches for each half of workload s's
    batch (the same rules as the library's dispatch): the semantic top-1
    scan k_sem_mm for k = 1, else k_sem_scan; the bf16 top-1 trajectory scan
    k_traj_mm for bf16 stores, k = 1 and more than 128 queries per launch,
    else k_traj_scan."""
    sem = ("k_sem_mm" if s.k == 1 else "k_sem_scan") if s.B_sem else None
    traj = None
    if s.B_traj:
        traj = "k_traj_mm" if (s.map_dtype == "bf16" and s.k == 1 and min(s.B_traj, 1024) > 128) else "k_traj_scan"
    return sem, traj


def hip_runtime():
    """The HIP runtime this process already uses (torch's), for raw events."""
    import ctypes
    import re
    paths = sorted(set(re.findall(r"(/\S*libamdhip64\.so\S*)", open("/proc/self/maps").read())))
    if not paths:
        raise RuntimeError("the HIP runtime is not loaded")
    hip = ctypes.CDLL(paths[0])
    hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
    hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
    hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
    return hip


class ScanTimer:
    """HIP event pairs that the library records around its scan kernel launch
    (fm_debug_scan_events), one pair per timed call."""

    def __init__(self, hip, lib, n):
        import ctypes
        self.hip, self.lib, self.C = hip, lib, ctypes
        self.pairs = []
        for _ in range(n):
            a, b = ctypes.c_void_p(), ctypes.c_void_p()
            assert hip.hipEventCreate(ctypes.byref(a)) == 0 and hip.hipEventCreate(ctypes.byref(b)) == 0
            self.pairs.append((a, b))

    def arm(self, i):
        a, b = self.pairs[i]
        assert self.lib.fm_debug_scan_events(a, b) == 0

    def disarm(self):
        assert self.lib.fm_debug_scan_events(None, None) == 0

    def mean_ms(self, n):
        vals = []
        for a, b in self.pairs[:n]:
            ms = self.C.c_float()
            assert self.hip.hipEventElapsedTime(self.C.byref(ms), a, b) == 0
            vals.append(ms.value)
        return float(np.mean(vals))


def parse():
    p = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=50)
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--config", type=int, default=5, choices=[1, 2, 3, 4, 5])
    p.add_argument("--cpu-seconds", type=float, default=15.0, help="budget of the CPU-oracle sample")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cold-reps", type=int, default=10,
                   help="untimed steps after the timed region, each after a 512 MiB read that flushes the "
                        "256 MB memory-side cache, whose scan events give the cold scan time (0: skip)")
    p.add_argument("--path", default="match", choices=["match", "dedup", "step", "order", "capacity"],
                   help="match: search + selection (default); dedup: deduplicating inserts (Section 4.4); "
                        "step: incremental per-layer trajectory re-search passes (Section 4.2.2); "
                        "order: prefetch priority ordering of the selected sets (Section 4.5); "
                        "capacity: similarity and misses against store capacity (Section 6 sensitivity)")
    p.add_argument("--copy-probe", action="store_true",
                   help="only copy 256 MiB device-to-device three times (reference for HBM traffic counters)")
    return p.parse_args()


def algorithmic_cost(s, a):
    """Bytes and flops the method itself must move/compute for one batch."""
    esz = 2 if s.map_dtype == "bf16" else 4
    out = {"traj_bytes": 0, "traj_flops": 0, "sem_bytes": 0, "sem_flops": 0}
    if s.B_traj:
        d = np.clip(a["depth"], 1, s.L)
        dmax = int(d.max())
        out["traj_bytes"] = s.n * dmax * s.E * esz
        # the stored prefix norms are computed at insert, not per batch
        out["traj_flops"] = int(2 * s.n * s.E * int(d.sum()))
    if s.B_sem:
        out["sem_bytes"] = s.n * s.d_emb * 2 + 4 * s.n
        out["sem_flops"] = 2 * s.B_sem * s.n * s.d_emb
    return out


def _oracle_step(s, a, sem_rows, traj_rows):
    """One step of the oracle on the given queries: each kind's queries as one
    batch against the whole store, then their prefetch sets."""
    import oracle
    idx = np.full((len(sem_rows) + len(traj_rows), s.k), -1, dtype=np.int64)
    sc = np.full(idx.shape, -np.inf)
    if len(sem_rows):
        idx[:len(sem_rows)], sc[:len(sem_rows)] = oracle.match_semantic(a["embs"], a["q_sem"][sem_rows], s.k)
    if len(traj_rows):
        b = np.asarray(traj_rows) - s.B_sem
        idx[len(sem_rows):], sc[len(sem_rows):] = oracle.match_trajectory(a["maps"], s.map_dtype, a["q_traj"][b],
                                                                         a["depth"][b], s.k)
    rows = np.r_[np.asarray(sem_rows, dtype=np.int64), np.asarray(traj_rows, dtype=np.int64)]
    oracle.select_prefetch(a["maps"], s.map_dtype, idx, sc, a["lb"][rows], a["le"][rows], s.tau_mode, s.tau,
                           s.k_min, s.k_max, s.blend)
    return rows, idx


def cpu_baseline(s, a, gpu_idx, budget_s):
    """The oracle on a bounded sample of the same batch: the first m queries of
    each kind, each kind as one batch against the whole store (the oracle
    widens every store chunk once per batch), then the selection.  m starts
    at 8 and grows fourfold while the next run is predicted to fit the
    budget; the largest run is reported."""
    from threadpoolctl import threadpool_info
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    per_kind = max(s.B_sem, s.B_traj)
    m, best = 8, None
    while True:
        m = min(m, per_kind)
        sem_rows = list(range(min(m, s.B_sem)))
        traj_rows = list(range(s.B_sem, s.B_sem + min(m, s.B_traj)))
        t0 = time.perf_counter()
        rows, idx = _oracle_step(s, a, sem_rows, traj_rows)
        dt = time.perf_counter() - t0
        best = (rows, idx, dt)
        if m >= per_kind or 4 * dt > budget_s:
            break
        m *= 4
    rows, idx, dt = best
    mism = int(np.sum(idx[:, 0] != gpu_idx[rows, 0]))
    kinds = []
    if s.B_sem:
        kinds.append(f"{min(m, s.B_sem)} of {s.B_sem} semantic")
    if s.B_traj:
        kinds.append(f"{min(m, s.B_traj)} of {s.B_traj} trajectory")
    return {"value": len(rows) / dt, "unit": "queries/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{' + '.join(kinds)} queries (the first of each kind), each kind one batch against the "
                      f"full {s.n}-map store in {dt:.1f} s, then their prefetch sets",
            "top1_index_mismatches_vs_gpu": mism}


# Deduplicating-insert workload: the Mixtral-shaped store with d = 4096
# embeddings at capacity (100,000 iterations), batches of 256 new iterations
# (one in eight an exact copy of a stored one), prefetch distance 3 (the
# paper's setting for Mixtral, Section 6).
DEDUP_CONFIG = 3
DEDUP_BATCH = 256
DEDUP_D = 3
DEDUP_BATCHES = 8


def dedup_cost(s, m):
    """Algorithmic bytes and flops of one deduplicating insert of m new
    iterations into a full store: every stored embedding and map is read once
    and scored against every new iteration (the dense score matrices are this
    implementation's choice and are not counted)."""
    esz = 2 if s.map_dtype == "bf16" else 4
    return {"sem_bytes": s.n * s.d_emb * 2 + 4 * s.n, "sem_flops": 2 * m * s.n * s.d_emb,
            "traj_bytes": s.n * s.L * s.E * esz + 4 * s.n, "traj_flops": 2 * m * s.n * s.L * s.E}


def dedup_cpu_baseline(s, a, b, d, gpu_slots, budget_s):
    """Oracle RDY rows and victim choice for the first new iterations of the
    batch (all of them find the store full), one at a time."""
    import oracle
    from threadpoolctl import threadpool_info
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    taken = np.zeros(s.n, dtype=bool)
    t_total, rows, mism = 0.0, 0, 0
    m = b["new_maps"].shape[0]
    for x in range(m):
        t0 = time.perf_counter()
        r = oracle.redundancy(a["maps"], a["embs"], b["new_maps"][x:x + 1], b["new_embs"][x:x + 1], s.map_dtype, d)
        cand = np.flatnonzero(~taken)
        y = int(oracle.rank(r[0, cand], 1, cand)[0][0])
        taken[y] = True
        t_total += time.perf_counter() - t0
        rows += 1
        mism += int(y != int(gpu_slots[x]))
        if t_total >= budget_s:
            break
    return {"value": rows / t_total, "unit": "new iterations/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{rows} of {m} new iterations against the full {s.n}-entry store (RDY row + victim), "
                      "one at a time", "victim_mismatches_vs_gpu": mism}


def bench_dedup(args):
    import torch
    import synth
    import paper_2502_05370_amd as fm
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    from parity import to_device

    s = synth.spec(DEDUP_CONFIG).scaled(B_traj=0, B_sem=0)
    a = synth.generate(s)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    store = fm.Store(s.n, s.L, s.E, s.d_emb, s.map_dtype, device=dev)
    store.insert(to_device(a["maps"], s.map_dtype), to_device(a["embs"], "bf16"))
    big = synth.generate_new(s, DEDUP_BATCH * DEDUP_BATCHES, a)
    maps = to_device(big["new_maps"], s.map_dtype)
    embs = to_device(big["new_embs"], "bf16")
    batches = [(maps[i * DEDUP_BATCH:(i + 1) * DEDUP_BATCH], embs[i * DEDUP_BATCH:(i + 1) * DEDUP_BATCH])
               for i in range(DEDUP_BATCHES)]
    ws = fm.Workspace(store)
    scratch = fm._aligned_bytes(fm.dedup_scratch_bytes(s.n, DEDUP_BATCH), dev)
    stream = torch.cuda.current_stream()
    hip = hip_runtime()
    lib = fm._lib.load()
    timer = ScanTimer(hip, lib, args.steps)

    # the first batch against the untouched store, kept for the CPU baseline
    first = store.insert_dedup(*batches[0], DEDUP_D, workspace=ws, scratch=scratch, stream=stream)
    first = first.cpu().numpy()
    for i in range(args.warmup):
        store.insert_dedup(*batches[(i + 1) % DEDUP_BATCHES], DEDUP_D, workspace=ws, scratch=scratch, stream=stream)
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    t0 = time.perf_counter()
    for i in range(args.steps):
        ev[i][0].record(stream)
        timer.arm(i)
        store.insert_dedup(*batches[(i + 1 + args.warmup) % DEDUP_BATCHES], DEDUP_D, workspace=ws, scratch=scratch,
                           stream=stream)
        timer.disarm()
        ev[i][1].record(stream)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    call_ms = float(np.mean([e0.elapsed_time(e1) for e0, e1 in ev]))
    scan_ms = timer.mean_ms(args.steps)

    # the events bracket the last scan kernel of each call: the semantic one
    cost = dedup_cost(s, DEDUP_BATCH)
    byts, flops = cost["sem_bytes"], cost["sem_flops"]
    dur_s = scan_ms * 1e-3
    if flops / (BF16_MFMA_PEAK_TFS * 1e12) > byts / (HBM_PEAK_GBS * 1e9):
        achieved = flops / dur_s / 1e12
        roof = {"bound": "mfma", "achieved": achieved, "peak": BF16_MFMA_PEAK_TFS, "unit": "TFLOP/s",
                "frac": achieved / BF16_MFMA_PEAK_TFS}
    else:
        achieved = byts / dur_s / 1e9
        roof = {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": achieved / HBM_PEAK_GBS}
    # (the dense semantic pass runs on the top-1 scan's dense form, k_sem_mm)
    roof.update({"traffic": None, "kernel": "k_sem_mm", "mfma_dtype": "bf16", "duration_us": scan_ms * 1e3,
                 "algorithmic_bytes": byts, "algorithmic_flops": flops, "call_us": call_ms * 1e3})
    cpu = None
    if not args.no_cpu_baseline:
        b0 = {"new_maps": big["new_maps"][:DEDUP_BATCH], "new_embs": big["new_embs"][:DEDUP_BATCH]}
        cpu = dedup_cpu_baseline(s, a, b0, DEDUP_D, first, args.cpu_seconds)
    line = {
        "metric": "new iterations/sec inserted with deduplication (RDY, Section 4.4) at 1 GPU",
        "value": DEDUP_BATCH * args.steps / elapsed, "unit": "new iterations/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": elapsed / args.steps * 1e3,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32+bf16",
        "data": "synthetic",
        "config": {"workload": f"dedup_semantic_d{s.d_emb}_n{s.n // 1000}k_b{DEDUP_BATCH}", "store_maps": s.n,
                   "capacity": s.n, "layers": s.L, "experts": s.E, "map_dtype": s.map_dtype, "d_emb": s.d_emb,
                   "batch": DEDUP_BATCH, "prefetch_distance": DEDUP_D},
        "roofline": roof,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


# Incremental re-search workload: the Qwen-shaped store (50,000 maps of
# 24 x 60 float32) and 64 queries; one pass observes layers 1 .. L-d and
# searches after each (d = 6, the paper's setting for Qwen, Section 6), i.e.
# L - d = 18 searches at prefix depths 1 .. 18.
STEP_CONFIG = 2
STEP_D = 6


def bench_step(args):
    import torch
    import synth
    import paper_2502_05370_amd as fm
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    from parity import to_device

    s = synth.spec(STEP_CONFIG)
    a = synth.generate(s)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    store = fm.Store(s.n, s.L, s.E, s.d_emb, s.map_dtype, device=dev)
    store.insert(to_device(a["maps"], s.map_dtype))
    B, n_layers = s.B_traj, s.L - STEP_D
    q = to_device(a["q_traj"], s.map_dtype)
    q_layers = [q[:, l].contiguous() for l in range(n_layers)]
    ws = fm.Workspace(store)
    tp = fm.TrajPass(store, B)
    idx = torch.empty((B, s.k), dtype=torch.int32, device=dev)
    score = torch.empty((B, s.k), dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream()
    hip = hip_runtime()
    lib = fm._lib.load()
    timer = ScanTimer(hip, lib, args.steps * n_layers)

    def one_pass(i=None):
        for l in range(n_layers):
            if i is not None:
                timer.arm(i * n_layers + l)
            tp.step(q_layers[l], l, s.k, out=(idx, score), workspace=ws, stream=stream)
        if i is not None:
            timer.disarm()

    for _ in range(args.warmup):
        one_pass()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        one_pass(i)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    step_ms = timer.mean_ms(args.steps * n_layers)

    # reference: the same searches as full re-scans (fm_match_trajectory at
    # each depth), timed the same way
    depths = [torch.full((B,), l + 1, dtype=torch.int32, device=dev) for l in range(n_layers)]

    def rescan_pass():
        for l in range(n_layers):
            fm.match_trajectory(store, q, depths[l], s.k, max_depth=l + 1, out=(idx, score), workspace=ws,
                                stream=stream)

    rescan_pass()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    for _ in range(args.steps):
        rescan_pass()
    torch.cuda.synchronize()
    rescan_s = (time.perf_counter() - t1) / args.steps

    # algorithmic cost of one step launch, averaged over the pass: the new
    # layer's plane and inverse norms, and the running dots (written at the
    # first layer, read and written after)
    esz = 2 if s.map_dtype == "bf16" else 4
    plane = s.n * s.E * esz + 4 * s.n
    dots = [4 * B * s.n] + [8 * B * s.n] * (n_layers - 1)
    byts = plane + float(np.mean(dots))
    flops = 2 * B * s.n * s.E
    dur_s = step_ms * 1e-3
    if flops / (FP32_MFMA_PEAK_TFS * 1e12) > byts / (HBM_PEAK_GBS * 1e9):
        achieved = flops / dur_s / 1e12
        roof = {"bound": "mfma", "achieved": achieved, "peak": FP32_MFMA_PEAK_TFS, "unit": "TFLOP/s",
                "frac": achieved / FP32_MFMA_PEAK_TFS}
    else:
        achieved = byts / dur_s / 1e9
        roof = {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": achieved / HBM_PEAK_GBS}
    roof.update({"traffic": None, "kernel": "k_traj_step", "mfma_dtype": "f32", "duration_us": step_ms * 1e3,
                 "algorithmic_bytes": byts, "algorithmic_flops": flops,
                 "pass_us": elapsed / args.steps * 1e6, "rescan_pass_us": rescan_s * 1e6})
    cpu = None
    if not args.no_cpu_baseline:
        cpu = step_cpu_baseline(s, a, n_layers, idx.cpu().numpy(), args.cpu_seconds)
    line = {
        "metric": "per-layer trajectory re-searches/sec (queries x searched layers, Section 4.2.2) at 1 GPU",
        "value": B * n_layers * args.steps / elapsed, "unit": "query-layer searches/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": elapsed / args.steps * 1e3,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": f"step_qwen_n{s.n // 1000}k_b{B}_d{STEP_D}", "store_maps": s.n, "layers": s.L,
                   "experts": s.E, "map_dtype": s.map_dtype, "batch": B, "prefetch_distance": STEP_D,
                   "searches_per_pass": n_layers, "top_k": s.k},
        "roofline": roof,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


def step_cpu_baseline(s, a, n_layers, gpu_idx_last, budget_s):
    """Oracle passes (Section 4.2.2 schedule: a search at every depth
    1 .. L-d) for one query at a time."""
    import oracle
    from threadpoolctl import threadpool_info
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    t_total, done, mism = 0.0, 0, 0
    for b in range(s.B_traj):
        t0 = time.perf_counter()
        res = oracle.research_schedule(a["maps"], s.map_dtype, a["q_traj"][b:b + 1], s.k, STEP_D)
        t_total += time.perf_counter() - t0
        done += 1
        mism += int(res[s.L][0][0, 0] != gpu_idx_last[b, 0])
        if t_total >= budget_s:
            break
    return {"value": done * n_layers / t_total, "unit": "query-layer searches/s", "cores": int(threads),
            "kind": "oracle", "sample": f"{done} of {s.B_traj} queries, each a whole pass of {n_layers} searches "
                                        f"against the full {s.n}-map store", "last_layer_mismatches_vs_gpu": mism}


def bench_order(args):
    """Section 4.5 prefetch ordering of workload ``--config``'s batch: the
    matches and prefetch sets are computed once (resident), then each step
    orders every query's set by p / (l - l_now) with l_now = the layer before
    its first selected one."""
    import torch
    import synth
    import paper_2502_05370_amd as fm
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    from parity import to_device

    s = synth.spec(args.config)
    a = synth.generate(s)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    store = fm.Store(s.n, s.L, s.E, s.d_emb, s.map_dtype, device=dev)
    store.insert(to_device(a["maps"], s.map_dtype), to_device(a["embs"], "bf16") if s.d_emb else None)
    idx = torch.empty((s.B, s.k), dtype=torch.int32, device=dev)
    score = torch.empty((s.B, s.k), dtype=torch.float32, device=dev)
    max_depth = int(np.clip(a["depth"], 1, s.L).max()) if s.B_traj else s.L
    if s.B_sem:
        fm.match_semantic(store, to_device(a["q_sem"], "bf16"), s.k, out=(idx[:s.B_sem], score[:s.B_sem]))
    if s.B_traj:
        fm.match_trajectory(store, to_device(a["q_traj"], s.map_dtype), to_device(a["depth"], "i32"), s.k,
                            max_depth=max_depth, out=(idx[s.B_sem:], score[s.B_sem:]))
    mask, count = fm.select_prefetch(store, idx, score, to_device(a["lb"], "i32"), to_device(a["le"], "i32"),
                                     tau=s.tau, k_min=s.k_min, k_max=s.k_max, mode=s.tau_mode, blend=s.blend)
    l_now = to_device(a["lb"].astype(np.int32) - 1, "i32")
    cap = s.L * s.E
    out = (torch.empty((s.B, cap), dtype=torch.int32, device=dev), torch.empty((s.B, cap), dtype=torch.float32, device=dev),
           torch.empty((s.B,), dtype=torch.int32, device=dev))
    stream = torch.cuda.current_stream()

    def order():
        fm.priority_order(store, idx, score, mask, l_now=l_now, blend=s.blend, cap=cap, out=out, stream=stream)

    for _ in range(args.warmup):
        order()
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    t0 = time.perf_counter()
    for i in range(args.steps):
        ev[i][0].record(stream)
        order()
        ev[i][1].record(stream)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    call_ms = float(np.mean([e0.elapsed_time(e1) for e0, e1 in ev]))
    cnt = out[2].cpu().numpy()
    # algorithmic bytes: the prefetch sets, each candidate's stored
    # probabilities (k rows when blending) and the ordered lists written
    esz = 2 if s.map_dtype == "bf16" else 4
    k_rows = s.k if s.blend else 1
    byts = s.B * s.L * 8 + int(cnt.sum()) * k_rows * esz + s.B * cap * 8
    achieved = byts / (call_ms * 1e-3) / 1e9
    roof = {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
            "traffic": None, "kernel": "k_priority", "duration_us": call_ms * 1e3, "algorithmic_bytes": byts,
            "candidates_per_query": float(cnt.mean())}
    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
        gi, gs, gm = idx.cpu().numpy(), score.cpu().numpy(), mask.cpu().numpy().view(np.uint64)
        ln = a["lb"].astype(np.int64) - 1
        t_total, done, mism = 0.0, 0, 0
        go = out[0].cpu().numpy()
        for b in range(s.B):
            t1 = time.perf_counter()
            o, _, _ = oracle.priority_order(a["maps"], s.map_dtype, gi[b:b + 1], gs[b:b + 1], s.blend,
                                            oracle.PRI_PREFETCH, gm[b:b + 1], l_now=ln[b:b + 1], cap=cap)
            t_total += time.perf_counter() - t1
            done += 1
            mism += int(not np.array_equal(o[0], go[b]))
            if t_total >= args.cpu_seconds:
                break
        cpu = {"value": done / t_total, "unit": "ordered queries/s", "cores": int(threads), "kind": "oracle",
               "sample": f"{done} of {s.B} queries, one at a time", "order_mismatches_vs_gpu": mism}
    line = {
        "metric": "prefetch-ordered queries/sec (Section 4.5 priorities of the selected sets) at 1 GPU",
        "value": s.B * args.steps / elapsed, "unit": "queries/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": elapsed / args.steps * 1e3, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": f"order_{s.name}", "store_maps": s.n, "layers": s.L, "experts": s.E, "batch": s.B,
                   "list_capacity": cap},
        "roofline": roof,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


# Capacity study: the Qwen-shaped bf16 store with d = 2048 embeddings
# (workload 5's generator), read at growing capacities; 1024 fresh iterations
# as queries (half by embedding, guiding layers 1..d; half by trajectory at
# depth p ~ U{1..L-d}, guiding layer p + d), prefetch distance d = 6.
CAP_CONFIG = 5
CAP_D = 6
CAP_SIZES = (1_000, 2_000, 2_880, 5_000, 5_236, 10_000, 20_000, 50_000, 100_000, 200_000, 500_000, 1_000_000)


def bench_capacity(args):
    import math
    import torch
    import synth
    import paper_2502_05370_amd as fm
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    from parity import to_device

    s = synth.spec(CAP_CONFIG).scaled(B_traj=0, B_sem=0)
    print("generating the store", file=sys.stderr, flush=True)
    a = synth.generate(s)
    m = 1024
    new = synth.generate_new(s, m, a, dup_frac=0.0)
    with open(os.path.join(ROOT, "tests", "golden", "models.json")) as f:
        K = json.load(f)["models"]["qwen1.5_moe"]["K"]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    store = fm.Store(s.n, s.L, s.E, s.d_emb, s.map_dtype, device=dev)
    maps, embs = to_device(a["maps"], s.map_dtype), to_device(a["embs"], "bf16")
    h = m // 2
    rng = np.random.default_rng(250205370)
    depth = rng.integers(1, s.L - CAP_D + 1, size=m - h).astype(np.int32)
    q_maps = to_device(new["new_maps"], s.map_dtype)
    q_sem = to_device(new["new_embs"][:h], "bf16")
    q_traj = q_maps[h:]
    lb = np.concatenate([np.zeros(h, np.int32), depth + CAP_D - 1])
    le = np.concatenate([np.full(h, CAP_D, np.int32), depth + CAP_D])
    lbt, let = to_device(lb, "i32"), to_device(le, "i32")
    depth_t = to_device(depth, "i32")
    full_depth = torch.full((m,), s.L, dtype=torch.int32, device=dev)
    ws = fm.Workspace(store)
    idx = torch.empty((m, 1), dtype=torch.int32, device=dev)
    score = torch.empty((m, 1), dtype=torch.float32, device=dev)
    fidx = torch.empty((m, 1), dtype=torch.int32, device=dev)
    fscore = torch.empty((m, 1), dtype=torch.float32, device=dev)
    hip = hip_runtime()
    lib = fm._lib.load()
    rows = []
    inserted = 0
    for C in CAP_SIZES:
        store.insert(maps[inserted:C], embs[inserted:C])
        inserted = C
        timer = ScanTimer(hip, lib, 2 * args.steps)
        # one untimed search per capacity (launch shapes change with the size)
        fm.match_semantic(store, q_sem, 1, out=(idx[:h], score[:h]), workspace=ws)
        fm.match_trajectory(store, q_traj, depth_t, 1, max_depth=s.L - CAP_D, out=(idx[h:], score[h:]),
                            workspace=ws)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(args.steps):
            timer.arm(2 * i)
            fm.match_semantic(store, q_sem, 1, out=(idx[:h], score[:h]), workspace=ws)
            timer.arm(2 * i + 1)
            fm.match_trajectory(store, q_traj, depth_t, 1, max_depth=s.L - CAP_D,
                                out=(idx[h:], score[h:]), workspace=ws)
            timer.disarm()
        torch.cuda.synchronize()
        match_s = (time.perf_counter() - t0) / args.steps
        durs = []
        for i in range(2 * args.steps):
            ms = timer.C.c_float()
            assert hip.hipEventElapsedTime(timer.C.byref(ms), *timer.pairs[i]) == 0
            durs.append(ms.value)
        sem_ms, traj_ms = float(np.mean(durs[0::2])), float(np.mean(durs[1::2]))
        mask, _ = fm.select_prefetch(store, idx, score, lbt, let, tau=s.tau, k_min=s.k_min, k_max=s.k_max,
                                     mode=s.tau_mode, blend=s.blend)
        miss = fm.miss_count(store, q_maps, mask, K, lbt, let)
        # the covering claim concerns whole maps: full-depth trajectory search
        fm.match_trajectory(store, q_maps, full_depth, 1, max_depth=s.L, out=(fidx, fscore), workspace=ws)
        torch.cuda.synchronize()
        sc = score.cpu().numpy()[:, 0].astype(np.float64)
        fsc = fscore.cpu().numpy()[:, 0].astype(np.float64)
        n_rows = int((le - lb).sum())
        rows.append({"capacity": C, "mean_semantic": float(sc[:h].mean()), "mean_trajectory": float(sc[h:].mean()),
                     "mean_full_map": float(fsc.mean()), "min_full_map": float(fsc.min()),
                     "hit_rate": 1.0 - float(miss.cpu().numpy().sum()) / (K * n_rows),
                     "sem_scan_us": sem_ms * 1e3, "traj_scan_us": traj_ms * 1e3, "match_us": match_s * 1e6})
        print(json.dumps(rows[-1]), file=sys.stderr, flush=True)
    LJ = s.L * s.E
    bound = {"LJ": LJ, "2LJ": 2 * LJ, "half_LJ_lnLJ": round(0.5 * LJ * math.log(LJ)),
             "min_full_map_at_2LJ": next(r["min_full_map"] for r in rows if r["capacity"] == 2 * LJ),
             "min_full_map_at_half_LJ_lnLJ": next(r["min_full_map"] for r in rows
                                                  if r["capacity"] == round(0.5 * LJ * math.log(LJ)))}
    last = rows[-1]
    sem_bytes = s.n * s.d_emb * 2 + 4 * s.n
    sem_flops = 2 * h * s.n * s.d_emb
    dur_s = last["sem_scan_us"] * 1e-6
    if sem_flops / (BF16_MFMA_PEAK_TFS * 1e12) > sem_bytes / (HBM_PEAK_GBS * 1e9):
        achieved = sem_flops / dur_s / 1e12
        roof = {"bound": "mfma", "achieved": achieved, "peak": BF16_MFMA_PEAK_TFS, "unit": "TFLOP/s",
                "frac": achieved / BF16_MFMA_PEAK_TFS}
    else:
        achieved = sem_bytes / dur_s / 1e9
        roof = {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": achieved / HBM_PEAK_GBS}
    roof.update({"traffic": None, "kernel": "k_sem_mm", "mfma_dtype": "bf16", "duration_us": last["sem_scan_us"],
                 "algorithmic_bytes": sem_bytes, "algorithmic_flops": sem_flops})
    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
        t_total, done, mism = 0.0, 0, 0
        gi = idx.cpu().numpy()
        for b in range(h):
            t1 = time.perf_counter()
            oi, _ = oracle.match_semantic(a["embs"], new["new_embs"][b:b + 1], 1)
            t_total += time.perf_counter() - t1
            done += 1
            mism += int(oi[0, 0] != gi[b, 0])
            if t_total >= args.cpu_seconds:
                break
        cpu = {"value": done / t_total, "unit": "queries/s", "cores": int(threads), "kind": "oracle",
               "sample": f"{done} semantic queries against the full {s.n}-entry store, one at a time",
               "top1_index_mismatches_vs_gpu": mism}
    line = {
        "metric": "expert-map queries/sec at the largest store capacity, with similarity and misses vs capacity "
                  "(Section 6 sensitivity)",
        "value": m / (last["match_us"] * 1e-6), "unit": "queries/s", "n_gpus": 1, "steps": args.steps,
        "warmup": 0, "ms_per_step": last["match_us"] * 1e-3, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"capacity_qwen_bf16_d{s.d_emb}_to{s.n // 1000}k_b{m}", "layers": s.L,
                   "experts": s.E, "K": K, "prefetch_distance": CAP_D, "queries": m,
                   "capacities": list(CAP_SIZES)},
        "study": rows,
        "covering_bound": bound,
        "roofline": roof,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}, WORLD_SIZE {world}); "
              "the store would shard by rows across GPUs but that path is not built", file=sys.stderr)
        sys.exit(2)

    import torch
    if args.copy_probe:
        src = torch.ones(64 << 20, dtype=torch.float32, device="cuda:0")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes": src.numel() * 4, "launches": 3}))
        return
    if args.path == "dedup":
        bench_dedup(args)
        return
    if args.path == "step":
        bench_step(args)
        return
    if args.path == "order":
        bench_order(args)
        return
    if args.path == "capacity":
        bench_capacity(args)
        return
    import synth
    import paper_2502_05370_amd as fm
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    from parity import to_device

    s = synth.spec(args.config)
    a = synth.generate(s)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    store = fm.Store(s.n, s.L, s.E, s.d_emb, s.map_dtype, device=dev)
    store.insert(to_device(a["maps"], s.map_dtype), to_device(a["embs"], "bf16") if s.d_emb else None)
    ws_sem = fm.Workspace(store)
    ws_traj = fm.Workspace(store)
    q_sem = to_device(a["q_sem"], "bf16") if s.B_sem else None
    q_traj = to_device(a["q_traj"], s.map_dtype) if s.B_traj else None
    depth = to_device(a["depth"], "i32") if s.B_traj else None
    lb = to_device(a["lb"], "i32")
    le = to_device(a["le"], "i32")
    idx = torch.empty((s.B, s.k), dtype=torch.int32, device=dev)
    score = torch.empty((s.B, s.k), dtype=torch.float32, device=dev)
    mask = torch.empty((s.B, s.L), dtype=torch.int64, device=dev)
    count = torch.empty((s.B, s.L), dtype=torch.uint8, device=dev)
    max_depth = int(np.clip(a["depth"], 1, s.L).max()) if s.B_traj else s.L
    stream = torch.cuda.current_stream()

    hip = hip_runtime()
    lib = fm._lib.load()
    sem_k, traj_k = scan_kernels(s)
    timers = {}
    if sem_k:
        timers[sem_k] = ScanTimer(hip, lib, args.steps)
    if traj_k:
        timers[traj_k] = ScanTimer(hip, lib, args.steps)

    sel = dict(tau=s.tau, k_min=s.k_min, k_max=s.k_max, mode=s.tau_mode, blend=s.blend)
    h = s.B_sem

    def step(i=None, tm=timers):
        """One step: each half of the batch through its match-and-select call
        (search, merge and selection of its rows)."""
        if s.B_sem:
            if i is not None:
                tm[sem_k].arm(i)
            fm.match_semantic_select(store, q_sem, lb[:h], le[:h], k=s.k, out=(idx[:h], score[:h], mask[:h],
                                     count[:h]), workspace=ws_sem, stream=stream, **sel)
        if s.B_traj:
            if i is not None:
                tm[traj_k].arm(i)
            fm.match_trajectory_select(store, q_traj, depth, lb[h:], le[h:], k=s.k, max_depth=max_depth,
                                       out=(idx[h:], score[h:], mask[h:], count[h:]), workspace=ws_traj,
                                       stream=stream, **sel)
        if i is not None:
            lib.fm_debug_scan_events(None, None)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # Timed region: K steps of the match-and-select calls on one stream.  HIP
    # events bracket the calls of every step, and the library records a
    # second pair right around each scan kernel launch on the same stream.
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        ev[i][0].record(stream)
        step(i)
        ev[i][1].record(stream)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    elapsed = t1 - t0
    calls_ms = float(np.mean([e0.elapsed_time(e1) for e0, e1 in ev]))
    scan_ms = {k: t.mean_ms(args.steps) for k, t in timers.items() if t is not None}

    # Cold scans (outside the timed region): before each of these steps a
    # read of 512 MiB, twice the 256 MB memory-side cache, evicts the store's
    # lines (with clean ones, so no write-back competes with the scan), and
    # the scan events time reads that come from HBM.
    cold_ms = {}
    if args.cold_reps > 0:
        flush = torch.ones(128 << 20, dtype=torch.int32, device=dev)
        cold = {k: ScanTimer(hip, lib, args.cold_reps) if t is not None else None for k, t in timers.items()}
        sink = torch.zeros((), dtype=torch.int32, device=dev)
        torch.cuda.synchronize()
        for i in range(args.cold_reps):
            torch.amax(flush, dim=0, out=sink)
            step(i, cold)
        torch.cuda.synchronize()
        cold_ms = {k: t.mean_ms(args.cold_reps) for k, t in cold.items() if t is not None}
        del flush

    # Dominant kernel and its binding roofline: the larger of its algorithmic
    # bytes at the HBM peak and its algorithmic flops at the MFMA peak of the
    # arithmetic it implements (float32 products for float32 maps, bf16
    # otherwise).
    cost = algorithmic_cost(s, a)
    kernel = max(scan_ms, key=scan_ms.get)
    if kernel == traj_k:
        byts, flops = cost["traj_bytes"], cost["traj_flops"]
        fpeak, fdt = (FP32_MFMA_PEAK_TFS, "f32") if s.map_dtype == "f32" else (BF16_MFMA_PEAK_TFS, "bf16")
    else:
        byts, flops = cost["sem_bytes"], cost["sem_flops"]
        fpeak, fdt = BF16_MFMA_PEAK_TFS, "bf16"
    dur_s = scan_ms[kernel] * 1e-3
    if flops / (fpeak * 1e12) > byts / (HBM_PEAK_GBS * 1e9):
        achieved = flops / dur_s / 1e12
        roof = {"bound": "mfma", "achieved": achieved, "peak": fpeak, "unit": "TFLOP/s", "frac": achieved / fpeak}
    else:
        achieved = byts / dur_s / 1e9
        roof = {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": achieved / HBM_PEAK_GBS}
    roof["traffic"] = counter_traffic(s.name, kernel)
    roof["kernel"] = kernel
    roof["mfma_dtype"] = fdt
    roof["duration_us"] = scan_ms[kernel] * 1e3
    roof["algorithmic_bytes"] = byts
    roof["algorithmic_flops"] = flops
    roof["scan_us"] = {k: v * 1e3 for k, v in scan_ms.items()}
    roof["calls_us"] = calls_ms * 1e3
    for other in scan_ms:
        if other == kernel:
            continue
        # the other scan of a mixed batch against its own binding roofline
        if other == traj_k:
            ob, of = cost["traj_bytes"], cost["traj_flops"]
            op = FP32_MFMA_PEAK_TFS if s.map_dtype == "f32" else BF16_MFMA_PEAK_TFS
        else:
            ob, of, op = cost["sem_bytes"], cost["sem_flops"], BF16_MFMA_PEAK_TFS
        od = scan_ms[other] * 1e-3
        if of / (op * 1e12) > ob / (HBM_PEAK_GBS * 1e9):
            roof["other"] = {"kernel": other, "bound": "mfma", "achieved": of / od / 1e12, "peak": op,
                             "unit": "TFLOP/s", "frac": of / od / 1e12 / op}
        else:
            roof["other"] = {"kernel": other, "bound": "hbm", "achieved": ob / od / 1e9, "peak": HBM_PEAK_GBS,
                             "unit": "GB/s", "frac": ob / od / 1e9 / HBM_PEAK_GBS}
        roof["other"].update({"duration_us": scan_ms[other] * 1e3, "algorithmic_bytes": ob,
                              "algorithmic_flops": of, "traffic": counter_traffic(s.name, other)})
    if cold_ms:
        # the same kernel's cold average and the fraction it reaches
        cold_s = cold_ms[kernel] * 1e-3
        roof["cold_duration_us"] = cold_ms[kernel] * 1e3
        roof["cold_frac"] = ((flops / cold_s / 1e12) / fpeak if roof["bound"] == "mfma"
                             else (byts / cold_s / 1e9) / HBM_PEAK_GBS)
        roof["cold_scan_us"] = {k: v * 1e3 for k, v in cold_ms.items()}

    value = s.B * args.steps / elapsed
    gpu_idx = idx.cpu().numpy()
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(s, a, gpu_idx, args.cpu_seconds)

    line = {
        "metric": "expert-map queries/sec (match + prefetch select) at 1 GPU; % HBM/MFMA peak",
        "value": value, "unit": "queries/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": elapsed / args.steps * 1e3, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32" if s.map_dtype == "f32" and not s.B_sem else
        ("bf16" if s.map_dtype == "bf16" or not s.B_traj else "f32+bf16"),
        "data": "synthetic",
        "config": {"workload": s.name, "store_maps": s.n, "layers": s.L, "experts": s.E,
                   "map_dtype": s.map_dtype, "d_emb": s.d_emb, "batch": s.B, "batch_semantic": s.B_sem,
                   "batch_trajectory": s.B_traj, "top_k": s.k, "tau": s.tau, "k_max": s.k_max},
        "roofline": roof,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
