"""Throughput of exact dense top-k on one MI355X.

Workload: exact top-5 by inner product for batches of 256 queries over 32,768 x 1,024 bf16
unit rows (256-component Gaussian mixture, sigma 0.3; queries are noisy copies of rows),
fp32 accumulation.  A step is one oprag_search_dense call over one batch: the scoring
kernel (per-chunk top-k lists) plus the merge of the lists.

Protocol: the index is replicated into 16 slabs (1 GiB in all, more than the 256 MB
Infinity Cache) and steps rotate over them, so every step streams its slab from HBM.
Steps are captured into HIP graphs (16 searches, one per slab) and replayed.  The same
searches launched one by one from Python give ``eager_queries_per_s`` and per-call
percentiles; a single slab reused every step gives ``warm_queries_per_s``.

Roofline: the scoring kernel carries a pair of HIP events in its own dispatch on the stream
it runs on (oprag_time_next_dense_kernel), stamped when the kernel starts and ends; its
average duration over a pass of 512 timed eager calls of the same workload gives
achieved = algorithmic bytes per launch (rows + queries + output lists) / that duration.  ``traffic`` is the HBM traffic per launch measured with
rocprofv3 counters (see --pmc-pass / --pmc-summarize), used only while the kernel source is
unchanged since the counters were taken.

Also reported: the CPU oracle's own throughput on a bounded sample of the same workload
(fp64 scores with a multithreaded BLAS, full stable sort per query).
"""
from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

N_ROWS, DIM, BATCH, K = 32768, 1024, 256, 5
COPIES = 16
HBM_PEAK_GBS = 8000.0
BF16_PEAK_TFLOPS = 2500.0
METRIC = "queries/s exact top-k (32K×1024 bf16, batch 256) + % of HBM/MFMA roofline"
KERNEL_SRC = os.path.join(ROOT, "paper_2608_08340_amd", "csrc", "dense.hip")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "dense_scoring_32k_x_1024_bf16_b256_traffic.json")
COPY_ROWS = 65536  # reference copy for counter scaling: 65,536 x 1,024 bf16 = 128 MiB each way


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or "unknown"


KERNEL_UNITS = {"dense.hip": ("dense.hip", "dense_ilp.hip"), "bm25.hip": ("bm25.hip",)}


def kernel_source_sha(name: str = "dense.hip") -> str:
    """sha256[:16] of what a kernel is built from: its source files (the scoring kernel's
    second compile unit included) and the compile flags."""
    from paper_2608_08340_amd import build as B
    h = hashlib.sha256()
    for f in KERNEL_UNITS.get(name, (name,)):
        h.update(open(os.path.join(os.path.dirname(KERNEL_SRC), f), "rb").read())
    h.update(repr((B.FLAGS, B.SOURCE_FLAGS)).encode())
    return h.hexdigest()[:16]


def kernel_sha_label(name: str = "dense.hip") -> str:
    return f"kernel build sha256[:16] ({' + '.join(KERNEL_UNITS.get(name, (name,)))} + compile flags): " \
           f"{kernel_source_sha(name)}"


def algorithmic_bytes(n_rows: int, dim: int, batch: int, k: int, elem: int = 2) -> int:
    """Index rows + queries + the k (score, id) results per query."""
    return n_rows * dim * elem + batch * dim * elem + batch * k * 12


def cpu_baseline(rows, queries, budget_s: float) -> dict:
    """The oracle as it stands: fp64 GEMM (multithreaded BLAS) + full stable sort per query,
    the sorts spread over a thread pool of the visible cores, timed on the host."""
    import concurrent.futures as cf

    from threadpoolctl import threadpool_info

    import synth
    from oracle import dense as od
    from oracle.storage import decode

    X = decode(synth.storage_bits(rows), "bf16")
    Qall = decode(synth.storage_bits(queries), "bf16")
    n_threads = max(1, len(os.sched_getaffinity(0)))
    per = max(1, BATCH // n_threads)
    done, t0 = 0, time.perf_counter()
    with cf.ThreadPoolExecutor(n_threads) as pool:
        while True:
            q = Qall[(done % Qall.shape[0]):(done % Qall.shape[0]) + BATCH]
            S = od.scores(X, q)
            list(pool.map(lambda i: od.topk_from_scores(S[i:i + per], K), range(0, S.shape[0], per)))
            done += q.shape[0]
            el = time.perf_counter() - t0
            if el >= budget_s or done >= 256 * Qall.shape[0]:  # the queries repeat cyclically
                break
    blas = [i for i in threadpool_info() if i.get("user_api") == "blas"]
    threads = max([i.get("num_threads", 1) for i in blas] or [1])
    return {"value": round(done / el, 2), "unit": "queries/s", "cores": int(max(threads, n_threads)), "kind": "oracle",
            "sample": f"{done} queries in batches of {BATCH} over the same 32,768 x 1,024 bf16 rows, top-{K}: "
                      f"fp64 numpy GEMM ({threads} BLAS threads) + per-query full stable sort ({n_threads} pool "
                      f"threads, {per} queries per task); {el:.1f} s; host {cpu_model()}, "
                      f"{len(os.sched_getaffinity(0))} cores visible"}


# The paper's only retrieval numbers are end-to-end latencies on other hardware: quoted beside
# the measurement as context, never as the target.
PAPER_CONTEXT = {
    "hybrid_retrieval_latency_reduction_pct": [59.20, 59.62],
    "what": "OpRAG's dense-first hybrid retrieval (top-128 candidates, lexical rerank) against full hybrid "
            "retrieval: 69.87 -> 28.21 ms (Llama3-8B run) and 68.63 -> 28.00 ms (Mistral-7B run), Recall@5 1.000",
    "hardware": "2x NVIDIA A100 (the paper's query-serving platform; retrieval device not stated), "
                "FAISS with float32 vectors",
    "source": "paper Section 5.5, table of Higress-style GPU query serving",
    "note": "context only: a different metric (end-to-end latency of a serving pipeline), workload and machine",
}


def traffic_record():
    """HBM bytes per scoring launch from the committed counter summary, if still current."""
    try:
        rec = json.load(open(TRAFFIC_FILE))
    except (OSError, ValueError):
        return None, "no counter summary"
    if rec.get("kernel_source_sha") != kernel_source_sha():
        return None, "kernel changed since the counters were taken"
    return rec.get("traffic_bytes_per_launch"), rec.get("command", "")


def pmc_summarize(out_dir: str) -> int:
    """Turn two rocprofv3 --pmc runs of --pmc-pass (FETCH_SIZE, WRITE_SIZE) into the traffic record."""
    vals = {}
    for counter in ("FETCH_SIZE", "WRITE_SIZE"):
        files = glob.glob(os.path.join(out_dir, counter.lower(), "**", "*counter_collection.csv"), recursive=True)
        if not files:
            print(f"no counter file for {counter} under {out_dir}", file=sys.stderr)
            return 1
        if len(files) != 1:
            print(f"{counter}: expected one counter file, found {len(files)}", file=sys.stderr)
            return 1
        copies, score = [], []
        for r in csv.DictReader(open(files[0])):
            if r["Counter_Name"] != counter:
                continue
            name = r["Kernel_Name"]
            if "copy16_kernel" in name:
                copies.append((int(r["Dispatch_Id"]), float(r["Counter_Value"])))
            elif "dense_mfma_kernel" in name:
                score.append(float(r["Counter_Value"]))
        if not copies or not score:
            print(f"{counter}: missing dispatches (copy {len(copies)}, scoring {len(score)})", file=sys.stderr)
            return 1
        # the reference copy is the pass's first copy (the index uploads that follow are copies too)
        vals[counter] = {"copy": min(copies)[1], "score": float(np.median(score)),
                         "n": {"copy": 1, "score": len(score)}}
    copy_kib = COPY_ROWS * DIM * 2 / 1024.0
    f_fetch = copy_kib / vals["FETCH_SIZE"]["copy"]
    f_write = copy_kib / vals["WRITE_SIZE"]["copy"]
    fetch = vals["FETCH_SIZE"]["score"] * f_fetch * 1024.0
    write = vals["WRITE_SIZE"]["score"] * f_write * 1024.0
    rec = {
        "kernel": "dense_mfma_kernel (scoring, 32,768 x 1,024 bf16, batch 256, k 5)",
        "kernel_source_sha": kernel_source_sha(),
        "fetch_kib_raw": vals["FETCH_SIZE"]["score"], "write_kib_raw": vals["WRITE_SIZE"]["score"],
        "copy_fetch_kib_raw": vals["FETCH_SIZE"]["copy"], "copy_write_kib_raw": vals["WRITE_SIZE"]["copy"],
        "copy_bytes_each_way": COPY_ROWS * DIM * 2,
        "fetch_scale": f_fetch, "write_scale": f_write,
        "traffic_bytes_per_launch": round(fetch + write),
        "algorithmic_bytes_per_launch": algorithmic_bytes(N_ROWS, DIM, BATCH, K),
        "dispatches": {c: vals[c]["n"] for c in vals},
        "command": "cd /tmp && export TMPDIR=/tmp && for c in FETCH_SIZE WRITE_SIZE; do timeout -s KILL 120 "
                   "rocprofv3 --pmc $c --output-format csv -d $GRAFT_REPO_ROOT/gpurun_out/pmc/$(echo $c | tr A-Z a-z) "
                   "-- python3 $GRAFT_REPO_ROOT/bench.py --pmc-pass; done && python3 $GRAFT_REPO_ROOT/bench.py "
                   "--pmc-summarize $GRAFT_REPO_ROOT/gpurun_out/pmc",
    }
    os.makedirs(os.path.dirname(TRAFFIC_FILE), exist_ok=True)
    json.dump(rec, open(TRAFFIC_FILE, "w"), indent=1)
    print(json.dumps(rec))
    return 0


# Counter passes for the MFMA-bound workloads: one rocprofv3 --pmc run per group (each within
# the per-block counter limits), each over a short run of `bench.py --pmc-workload NAME`.
PMC_GROUPS = {"fetch": "FETCH_SIZE", "write": "WRITE_SIZE", "l2": "TCC_HIT_sum TCC_MISS_sum",
              "mfma": "SQ_VALU_MFMA_BUSY_CYCLES SQ_INSTS_VALU_MFMA_MOPS_BF16 SQ_BUSY_CYCLES GRBM_GUI_ACTIVE",
              "lat": "TCP_TCC_READ_REQ_LATENCY_sum TCP_TCC_READ_REQ_sum TCC_EA0_RDREQ_LEVEL_sum TCC_EA0_RDREQ_sum",
              "wait": "SQ_WAIT_INST_ANY SQ_WAVE_CYCLES SQ_INSTS_LDS SQ_LDS_BANK_CONFLICT SQ_INSTS_VMEM_RD TA_BUSY_avr"}
PMC_WORKLOADS = {
    "b256": {"title": "32,768 x 1,024 bf16, batch 256, top-5 (8 cold slabs)", "n": N_ROWS, "d": DIM,
             "batch": 256, "k": 5},
    "b1024": {"title": "32,768 x 1,024 bf16, batch 1,024, top-5 (8 cold slabs)", "n": N_ROWS, "d": DIM,
              "batch": 1024, "k": 5},
    "c4": {"title": "1,048,576 x 768 bf16, batch 1,024, top-10", "n": 1 << 20, "d": 768, "batch": 1024, "k": 10},
    "bm25": {"title": "BM25 top-100 over the 32,768-chunk Zipf corpus (head rows and tail postings), batch 256, "
                      "8 searches on one index", "kernel": "bm25_kernel", "groups": ("fetch", "write", "l2"),
             "file": "bm25_32k_zipf_b256_counters.txt", "batch": 256, "k": 100},
}


def pmc_file(name: str) -> str:
    return os.path.join(ROOT, "profiles", PMC_WORKLOADS[name].get("file", f"dense_scoring_{name}_counters.txt"))


def pmc_groups(name: str) -> dict:
    return {g: PMC_GROUPS[g] for g in PMC_WORKLOADS[name].get("groups", PMC_GROUPS)}


def bm25_algorithmic_bytes(hw) -> int:
    """Distinct postings of the batch's terms (chunk id + weight, 8 bytes each), one 4-byte
    statistic per chunk and per term offset: each read once."""
    postings = int(sum(int(hw.csr.term_indptr[u + 1] - hw.csr.term_indptr[u]) for u in set(hw.qterms.tolist())))
    return postings * 8 + 4 * N_ROWS + 4 * hw.csr.term_indptr.size


def pmc_command(name: str) -> str:
    parts = [f"timeout -s KILL 120 rocprofv3 --pmc {c} --output-format csv -d $GRAFT_REPO_ROOT/gpurun_out/pmc_{name}/{g} "
             f"-- python3 $GRAFT_REPO_ROOT/bench.py --pmc-workload {name}" for g, c in pmc_groups(name).items()]
    return ("cd /tmp && export TMPDIR=/tmp && " + " && ".join(parts) +
            f" && python3 $GRAFT_REPO_ROOT/bench.py --pmc-workload {name} --pmc-summarize $GRAFT_REPO_ROOT/gpurun_out/pmc_{name}")


def pmc_workload_run(name: str) -> int:
    """A short run for counter collection: one reference copy of known size, then searches."""
    import torch

    import synth
    from paper_2608_08340_amd import Index

    wl = PMC_WORKLOADS[name]
    dev = torch.device("cuda", 0)
    ref = Index(DIM, COPY_ROWS, torch.bfloat16)
    ref.upsert(torch.zeros((COPY_ROWS, DIM), dtype=torch.bfloat16, device=dev))
    torch.cuda.synchronize()
    if name == "bm25":
        import numpy as np
        hw = synth.hybrid_32k()
        t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
        ix = Index(DIM, N_ROWS, torch.bfloat16)
        ix.upsert(hw.dense.rows.to(dev))
        ix.attach_sparse(t(hw.csr.term_indptr), t(hw.csr.post_chunk), t(hw.csr.post_tf), t(hw.csr.doc_len))
        qi, qt = t(hw.qterm_indptr), t(hw.qterms)
        torch.cuda.synchronize()
        for _ in range(8):
            ix.search_sparse(qi, qt, wl["k"])
        torch.cuda.synchronize()
        print("pmc workload done", flush=True)
        return 0
    if name == "c4":
        w = synth.mixture_dense(4, wl["n"], wl["d"], 4096, wl["batch"], wl["k"], "bf16")
        idxs = [Index(wl["d"], wl["n"], torch.bfloat16)]
    else:
        w = synth.dense_32k()
        idxs = [Index(wl["d"], wl["n"], torch.bfloat16) for _ in range(8)]
    rows = w.rows.to(dev)
    for ix in idxs:
        ix.upsert(rows)
    q = w.queries[:wl["batch"]].contiguous().to(dev)
    torch.cuda.synchronize()
    for r in range(3 if name == "c4" else 1):
        for ix in idxs:
            ix.search_dense(q, wl["k"])
    torch.cuda.synchronize()
    print("pmc workload done", flush=True)
    return 0


def pmc_workload_summarize(name: str, out_dir: str) -> int:
    """Per-dispatch counter values of the workload's kernel (median over its dispatches) and the
    derived HBM bytes, L2 hit rate and MFMA utilisation, written under profiles/."""
    wl = PMC_WORKLOADS[name]
    kernel = wl.get("kernel", "dense_mfma_kernel")
    vals, copy, durs = {}, {}, []
    agent = {}
    for f in glob.glob(os.path.join(out_dir, "**", "*agent_info.csv"), recursive=True):
        for r in csv.DictReader(open(f)):
            if r.get("Agent_Type", "").upper().endswith("GPU") or int(r.get("Simd_Count", "0") or 0) > 0:
                agent = r
        break
    n_xcc = int(agent.get("Num_Xcc", 8) or 8)
    n_simd = int(agent.get("Cu_Count", 256) or 256) * int(agent.get("Simd_Per_Cu", 4) or 4)
    for g in pmc_groups(name):
        files = glob.glob(os.path.join(out_dir, g, "**", "*counter_collection.csv"), recursive=True)
        if len(files) != 1:
            print(f"{g}: expected one counter file under {out_dir}/{g}, found {len(files)}", file=sys.stderr)
            return 1
        per = {}
        for r in csv.DictReader(open(files[0])):
            key = (r["Kernel_Name"], int(r["Dispatch_Id"]), r["Counter_Name"])
            per.setdefault(key, []).append(float(r["Counter_Value"]))
        for (kname, disp, cname), v in per.items():
            agg = max(v) if cname == "GRBM_GUI_ACTIVE" else sum(v)
            if "copy16_kernel" in kname:
                copy.setdefault(cname, []).append((disp, agg))
            elif kernel in kname:
                vals.setdefault(cname, []).append(agg)
        if g == "mfma":
            for r in csv.DictReader(open(files[0])):
                if kernel in r["Kernel_Name"] and r["Counter_Name"] == "GRBM_GUI_ACTIVE":
                    durs.append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
    med = {c: float(np.median(v)) for c, v in vals.items()}
    n_disp = {c: len(v) for c, v in vals.items()}
    ref = {c: min(v)[1] for c, v in copy.items()}  # the pass's first copy is the reference
    src = "bm25.hip" if kernel == "bm25_kernel" else "dense.hip"
    lines = [f"rocprofv3 counters of {kernel}, {wl['title']}",
             f"command: {pmc_command(name)}",
             kernel_sha_label(src), "",
             "median per dispatch (dispatches counted):"]
    for c in sorted(med):
        lines.append(f"  {c:32s} {med[c]:16.1f}   ({n_disp[c]})")
    if kernel == "bm25_kernel":
        import synth
        abytes = bm25_algorithmic_bytes(synth.hybrid_32k())
        flops = 0.0
    else:
        abytes = algorithmic_bytes(wl["n"], wl["d"], wl["batch"], wl["k"])
        flops = 2.0 * wl["batch"] * wl["n"] * wl["d"]
    lines.append("derived:")
    copy_kib = COPY_ROWS * DIM * 2 / 1024.0
    if "FETCH_SIZE" in med and "WRITE_SIZE" in med and "FETCH_SIZE" in ref and "WRITE_SIZE" in ref:
        fetch = med["FETCH_SIZE"] * copy_kib / ref["FETCH_SIZE"] * 1024.0
        write = med["WRITE_SIZE"] * copy_kib / ref["WRITE_SIZE"] * 1024.0
        lines.append(f"  HBM bytes per launch (FETCH_SIZE + WRITE_SIZE, each scaled by a {COPY_ROWS * DIM * 2} B copy: "
                     f"x{copy_kib / ref['FETCH_SIZE']:.4f} / x{copy_kib / ref['WRITE_SIZE']:.4f}): {fetch + write:.0f}")
        lines.append(f"  algorithmic bytes per launch: {abytes}  (traffic / algorithmic = {(fetch + write) / abytes:.3f})")
    if "TCC_HIT_sum" in med and "TCC_MISS_sum" in med:
        h, m = med["TCC_HIT_sum"], med["TCC_MISS_sum"]
        lines.append(f"  L2 hit rate TCC_HIT / (TCC_HIT + TCC_MISS): {h / (h + m):.4f}")
    if "SQ_VALU_MFMA_BUSY_CYCLES" in med and "GRBM_GUI_ACTIVE" in med:
        gui = med["GRBM_GUI_ACTIVE"] / n_xcc  # the CSV sums the counter over the XCDs
        lines.append(f"  GPU-active cycles per XCD (GRBM_GUI_ACTIVE / {n_xcc} XCDs): {gui:.0f}")
        if durs:
            d_us = float(np.median(durs))
            lines.append(f"  dispatch duration under the profiler (median): {d_us:.2f} us; "
                         f"active cycles / duration = {gui / d_us / 1e3:.3f} GHz")
        lines.append(f"  MFMA utilisation SQ_VALU_MFMA_BUSY_CYCLES / (cycles per XCD x {n_simd} SIMDs): "
                     f"{med['SQ_VALU_MFMA_BUSY_CYCLES'] / (gui * n_simd):.4f}")
    if "TCP_TCC_READ_REQ_LATENCY_sum" in med and med.get("TCP_TCC_READ_REQ_sum"):
        lines.append(f"  L1 -> L2 read latency (TCP_TCC_READ_REQ_LATENCY / TCP_TCC_READ_REQ): "
                     f"{med['TCP_TCC_READ_REQ_LATENCY_sum'] / med['TCP_TCC_READ_REQ_sum']:.0f} cycles per request")
    if "TCC_EA0_RDREQ_LEVEL_sum" in med and med.get("TCC_EA0_RDREQ_sum"):
        lines.append(f"  L2 -> memory read latency (TCC_EA0_RDREQ_LEVEL / TCC_EA0_RDREQ): "
                     f"{med['TCC_EA0_RDREQ_LEVEL_sum'] / med['TCC_EA0_RDREQ_sum']:.0f} cycles per request")
    if "SQ_WAIT_INST_ANY" in med and med.get("SQ_WAVE_CYCLES"):
        lines.append(f"  wave time waiting on a dependency (SQ_WAIT_INST_ANY / SQ_WAVE_CYCLES): "
                     f"{med['SQ_WAIT_INST_ANY'] / med['SQ_WAVE_CYCLES']:.3f}")
    if "SQ_LDS_BANK_CONFLICT" in med and med.get("SQ_INSTS_LDS"):
        lines.append(f"  LDS bank-conflict cycles per LDS instruction: {med['SQ_LDS_BANK_CONFLICT'] / med['SQ_INSTS_LDS']:.3f}")
    if "SQ_INSTS_VALU_MFMA_MOPS_BF16" in med and flops:
        lines.append(f"  MFMA flops SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512: {med['SQ_INSTS_VALU_MFMA_MOPS_BF16'] * 512:.4g} "
                     f"(algorithmic 2 B N d = {flops:.4g})")
    out = pmc_file(name)
    os.makedirs(os.path.dirname(out), exist_ok=True)
    open(out, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))
    return 0


STATS_FILE = os.path.join(ROOT, "profiles", "dense_scoring_32k_x_1024_bf16_b256_kernel_stats.txt")


SUITE_STATS_FILE = os.path.join(ROOT, "profiles", "suite_every_workload_kernel_stats.txt")


def trace_summarize(out_dir: str, suite: bool = False) -> int:
    """Write the kernel-trace statistics of a rocprofv3 --kernel-trace --stats run of bench.py
    (of ``bench.py --suite`` when suite is set)."""
    files = glob.glob(os.path.join(out_dir, "**", "*kernel_stats.csv"), recursive=True)
    if not files:
        print(f"no kernel_stats.csv under {out_dir}", file=sys.stderr)
        return 1
    rows = list(csv.DictReader(open(files[0])))
    if suite:
        head = [
            "rocprofv3 kernel statistics of bench.py --suite (every workload: 32K x 1,024 bf16 batches 1 / 16 / 100 / 256 / "
            "1,024, hybrid dense / BM25 / RRF / full, dense-first, weighted fusion, embedding tail, 1M x 768, "
            "streaming upsert and search); calls include warm-up and the eager timing passes",
            "command: cd /tmp && export TMPDIR=/tmp && timeout -k 10 600 rocprofv3 --kernel-trace --stats "
            "--output-format csv -d $GRAFT_REPO_ROOT/gpurun_out/kt_suite -o suite -- python3 $GRAFT_REPO_ROOT/bench.py "
            "--suite && python3 $GRAFT_REPO_ROOT/bench.py --suite-trace-summarize $GRAFT_REPO_ROOT/gpurun_out/kt_suite",
        ]
        out_file, n_show = SUITE_STATS_FILE, 40
    else:
        head = [
            "rocprofv3 kernel statistics of the default bench.py run (32,768 x 1,024 bf16, batch 256, k 5; "
            "the CPU oracle leg left out)",
            "command: cd /tmp && export TMPDIR=/tmp && timeout -k 10 400 rocprofv3 --kernel-trace --stats "
            "--output-format csv -d $GRAFT_REPO_ROOT/gpurun_out/kt_bench -o bench -- python3 $GRAFT_REPO_ROOT/bench.py "
            "--no-cpu && python3 $GRAFT_REPO_ROOT/bench.py --trace-summarize $GRAFT_REPO_ROOT/gpurun_out/kt_bench",
        ]
        out_file, n_show = STATS_FILE, 12
    lines = head + [
        kernel_sha_label(),
        "",
        f"{'calls':>7} {'avg_us':>9} {'min_us':>9} {'max_us':>9} {'share%':>7}  kernel",
    ]
    for r in rows[:n_show]:
        name = r["Name"].replace("(anonymous namespace)::", "")
        lines.append(f"{int(r['Calls']):7d} {float(r['AverageNs']) / 1e3:9.2f} {float(r['MinNs']) / 1e3:9.2f} "
                     f"{float(r['MaxNs']) / 1e3:9.2f} {float(r['Percentage']):7.2f}  {name[:150]}")
    os.makedirs(os.path.dirname(out_file), exist_ok=True)
    open(out_file, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))
    return 0


def _timed(fn, reps: int, stream, warm: int = 1) -> float:
    """Mean milliseconds per call of fn() over reps calls on the stream, after `warm` untimed
    calls (as many as the indexes fn rotates over, so each has its workspace before timing)."""
    import torch
    for _ in range(warm):
        fn()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record(stream)
    for _ in range(reps):
        fn()
    b.record(stream)
    torch.cuda.synchronize()
    return a.elapsed_time(b) / reps


def _kernel_ms(fn, reps: int, stream) -> float:
    """Mean duration of the scoring kernel of the dense search fn() performs (dispatch events)."""
    import torch
    import paper_2608_08340_amd as P
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
    for a, b in evs:
        a.record(stream)
        b.record(stream)
    torch.cuda.synchronize()
    for a, b in evs:
        P.time_next_dense_kernel(a, b)
        fn()
    torch.cuda.synchronize()
    return float(np.mean([a.elapsed_time(b) for a, b in evs]))


def suite() -> int:
    """Every workload once: per-call time, throughput and roofline fractions (one JSON line each)."""
    import torch

    import synth
    from paper_2608_08340_amd import Index, rrf_fuse

    dev = torch.device("cuda", 0)
    stream = torch.cuda.current_stream(dev)
    out = []

    def report(name, ms, batch, abytes, flops, kern_ms=None, **extra):
        r = {"workload": name, "us_per_call": round(ms * 1e3, 2), "queries_per_s": round(batch / (ms / 1e3), 1),
             "hbm_frac_call": round(abytes / (ms / 1e3) / 1e9 / HBM_PEAK_GBS, 4),
             "mfma_frac_call": round(flops / (ms / 1e3) / 1e12 / BF16_PEAK_TFLOPS, 4)}
        if kern_ms is not None:
            r.update({"scoring_kernel_us": round(kern_ms * 1e3, 2),
                      "hbm_frac_kernel": round(abytes / (kern_ms / 1e3) / 1e9 / HBM_PEAK_GBS, 4),
                      "mfma_frac_kernel": round(flops / (kern_ms / 1e3) / 1e12 / BF16_PEAK_TFLOPS, 4)})
        r.update(extra)
        out.append(r)
        print(json.dumps(r), flush=True)

    # tiny: 1,024 x 384 fp32, 16 queries, top-5 (launch-bound)
    w = synth.tiny_dense()
    ix = Index(384, 1024, torch.float32)
    ix.upsert(w.rows.to(dev))
    qt = w.queries.to(dev)
    ms = _timed(lambda: ix.search_dense(qt, 5), 200, stream)
    report("tiny 1,024 x 384 fp32, 16 queries, top-5", ms, 16, algorithmic_bytes(1024, 384, 16, 5, 4),
           2.0 * 16 * 1024 * 384, _kernel_ms(lambda: ix.search_dense(qt, 5), 100, stream))
    ix.close()

    # 32K x 1,024 bf16, batches 1 / 16 / 100 / 256 / 1,024 top-5 and 1 / 16 top-10, HBM-cold (16 slab
    # copies rotated)
    w = synth.dense_32k()
    rows = w.rows.to(dev)
    idxs = []
    for _ in range(COPIES):
        ix = Index(DIM, N_ROWS, torch.bfloat16)
        ix.upsert(rows)
        idxs.append(ix)
    # A plain cold streaming read of the same 64 MiB (the library's read probe: 16-byte loads,
    # eight in flight per thread; 16 copies rotated so every read comes from HBM), over a sweep
    # of grid sizes: how fast one cold pass over a slab goes on this part, the ceiling for the
    # HBM-bound batches.
    from paper_2608_08340_amd import probe_read
    sink = torch.empty(4096, dtype=torch.int32, device=dev)
    itr = [0]
    rd = {"workload": "plain cold read of 64 MiB (read probe: 16-byte loads, eight in flight per thread, "
                      "16 copies rotated), best grid", "grids": {}}
    for blocks in (256, 512, 1024, 2048, 4096):
        def cold_read():
            c = itr[0] % COPIES
            itr[0] += 1
            probe_read(idxs[c].slab, blocks, sink)
        ms_rd = _timed(cold_read, 256, stream)
        rd["grids"][blocks] = round(ms_rd * 1e3, 2)
    best = min(rd["grids"].values()) / 1e3
    rd.update({"us_per_call": round(best * 1e3, 2), "gb_per_s": round(N_ROWS * DIM * 2 / (best / 1e3) / 1e9, 1),
               "hbm_frac": round(N_ROWS * DIM * 2 / (best / 1e3) / 1e9 / HBM_PEAK_GBS, 4)})
    out.append(rd)
    print(json.dumps(rd), flush=True)
    sweep = []
    for b, kk in ((1, K), (16, K), (100, K), (256, K), (1024, K), (1, 10), (16, 10)):
        q = w.queries[:b].contiguous().to(dev)
        outs = [(torch.empty((b, kk), device=dev), torch.empty((b, kk), dtype=torch.int64, device=dev))
                for _ in range(COPIES)]
        it = [0]

        def step():
            c = it[0] % COPIES
            it[0] += 1
            idxs[c].search_dense(q, kk, out=outs[c])
        ms = _timed(step, 256, stream, COPIES)
        if kk == K:
            sweep.append((b, ms))
        report(f"32,768 x 1,024 bf16, batch {b}, top-{kk}, cold", ms, b, algorithmic_bytes(N_ROWS, DIM, b, kk),
               2.0 * b * N_ROWS * DIM, _kernel_ms(step, 128, stream))
    # cost model t(B) = alpha + beta * B over the batch sweep (least squares)
    bs = np.array([b for b, _ in sweep], dtype=np.float64)
    ts = np.array([m * 1e3 for _, m in sweep], dtype=np.float64)
    beta, alpha = np.polyfit(bs, ts, 1)
    fit = {"workload": "32,768 x 1,024 bf16 batch sweep, fit t(B) = alpha + beta * B", "alpha_us": round(float(alpha), 2),
           "beta_us_per_query": round(float(beta), 4),
           "max_rel_residual": round(float(np.max(np.abs(alpha + beta * bs - ts) / ts)), 3)}
    out.append(fit)
    print(json.dumps(fit), flush=True)

    # hybrid: the same index + 32,768-chunk Zipf corpus; dense 100 + BM25 100 -> RRF(60) -> 5
    hw = synth.hybrid_32k(dense=w)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    csr = [t(hw.csr.term_indptr), t(hw.csr.post_chunk), t(hw.csr.post_tf), t(hw.csr.doc_len)]
    for ix in idxs:
        ix.attach_sparse(*csr)
    qd = hw.dense.queries.to(dev)
    qi, qterms = t(hw.qterm_indptr), t(hw.qterms)
    nq = qd.shape[0]
    it = [0]

    def nxt():
        it[0] += 1
        return idxs[it[0] % COPIES]
    postings = int(sum(int(hw.csr.term_indptr[u + 1] - hw.csr.term_indptr[u]) for u in set(hw.qterms.tolist())))
    sparse_bytes = postings * 8 + 4 * N_ROWS + 4 * hw.csr.term_indptr.size
    ms_d = _timed(lambda: nxt().search_dense(qd, 100), 64, stream, COPIES)
    report("hybrid: dense top-100, batch 256, cold", ms_d, nq, algorithmic_bytes(N_ROWS, DIM, nq, 100),
           2.0 * nq * N_ROWS * DIM, _kernel_ms(lambda: nxt().search_dense(qd, 100), 64, stream))
    ms_s = _timed(lambda: nxt().search_sparse(qi, qterms, 100), 64, stream, COPIES)
    report("hybrid: BM25 top-100 over CSR postings, batch 256", ms_s, nq, sparse_bytes, 0.0,
           distinct_postings=postings)
    dl = nxt().search_dense(qd, 100)[1]
    sl = nxt().search_sparse(qi, qterms, 100)[1]
    ms_r = _timed(lambda: rrf_fuse(dl, sl, 60, 5), 256, stream)
    report("hybrid: RRF(60) of 100 + 100 -> 5, batch 256", ms_r, nq, nq * 200 * 8 + nq * 5 * 12, 0.0)
    ms_h = _timed(lambda: nxt().search_hybrid(qd, qi, qterms, 100, 100, 60, 5), 64, stream, COPIES)
    report("hybrid: full oprag_search_hybrid, batch 256, cold", ms_h, nq,
           algorithmic_bytes(N_ROWS, DIM, nq, 5) + sparse_bytes, 2.0 * nq * N_ROWS * DIM)
    # dense-first: dense top-128, BM25 of those candidates only, RRF(60) -> 5; quality against
    # the full hybrid result as Recall@5 and Jaccard overlap
    ms_f = _timed(lambda: nxt().search_hybrid_dense_first(qd, qi, qterms, 128, 60, 5), 64, stream, COPIES)
    a = nxt().search_hybrid_dense_first(qd, qi, qterms, 128, 60, 5)[1].cpu().numpy()
    b = nxt().search_hybrid(qd, qi, qterms, 100, 100, 60, 5)[1].cpu().numpy()
    inter = [len(set(a[i]) & set(b[i])) for i in range(nq)]
    report("hybrid dense-first: dense top-128 -> BM25 of the candidates -> RRF(60) -> 5, batch 256, cold", ms_f, nq,
           algorithmic_bytes(N_ROWS, DIM, nq, 128), 2.0 * nq * N_ROWS * DIM,
           recall_at_5_vs_full=round(float(np.mean(inter)) / 5, 3),
           jaccard_vs_full=round(float(np.mean([x / len(set(a[i]) | set(b[i])) for i, x in enumerate(inter)])), 3))
    # the paper's weighted fusion over every chunk (min-max normalised, 0.5 / 0.5), top-5
    ms_w = _timed(lambda: nxt().search_hybrid_weighted(qd, qi, qterms, 0.5, 0.5, 5), 64, stream, COPIES)
    report("hybrid weighted: 0.5 minmax(dense) + 0.5 minmax(BM25) over all chunks -> 5, batch 256, cold", ms_w, nq,
           algorithmic_bytes(N_ROWS, DIM, nq, 5) + sparse_bytes, 2.0 * nq * N_ROWS * DIM)
    for ix in idxs:
        ix.close()
    del idxs, rows

    # embedding tail fused with the upsert: 256 chunks x 512 tokens of 1,024-wide bf16 hidden
    # states (seeded synthetic; lengths uniform in [64, 512]) -> mean pool -> L2 -> bf16 rows
    g = np.random.default_rng(11)
    m_e, t_e = 256, 512
    hid = torch.randn((m_e, t_e, DIM), generator=torch.Generator().manual_seed(11)).to(torch.bfloat16).to(dev)
    lens = torch.from_numpy(g.integers(64, t_e + 1, size=m_e).astype(np.int32)).to(dev)
    ixe = Index(DIM, m_e * 40, torch.bfloat16)
    ms_e = _timed(lambda: ixe.upsert_pooled(hid, lens), 32, stream)
    tok = int(lens.sum().item())
    report("embedding tail: mean pool + L2 + upsert, 256 chunks x <=512 tokens x 1,024 bf16 hidden", ms_e, m_e,
           tok * DIM * 2 + m_e * DIM * 2, 0.0, valid_tokens=tok)
    ixe.close()
    del hid

    # 1,048,576 x 768 bf16, batch 1,024, top-10 (larger than the Infinity Cache)
    w4 = synth.mixture_dense(4, 1 << 20, 768, 4096, 1024, 10, "bf16")
    ix = Index(768, 1 << 20, torch.bfloat16)
    ix.upsert(w4.rows.to(dev))
    q4 = w4.queries.to(dev)
    ms = _timed(lambda: ix.search_dense(q4, 10), 10, stream)
    report("1,048,576 x 768 bf16, batch 1,024, top-10", ms, 1024, algorithmic_bytes(1 << 20, 768, 1024, 10),
           2.0 * 1024 * (1 << 20) * 768, _kernel_ms(lambda: ix.search_dense(q4, 10), 10, stream))
    ix.close()
    del w4

    # streaming: 8,388,608 x 384 fp16 (+65,536 fp32 rows per upsert), batch 4,096, top-100
    n0, m, d = 8388608, 65536, 384
    cen = synth.mixture_centres(synth.rng(5, 0), 8192, d)
    base = synth.to_storage(synth.mixture_rows_chunked(5, 1, cen, n0, 0.3), "f16")
    ix = Index(d, n0 + 16 * m, torch.float16)
    ix.upsert(base.to(dev))
    del base
    new = torch.from_numpy(synth.mixture_rows_chunked(5, 10, cen, m, 0.3)).to(dev)
    ms_u = _timed(lambda: ix.upsert(new), 1, stream)  # two appends (warm-up + one timed)
    report("streaming: upsert of 65,536 fp32 rows -> fp16 slab", ms_u, m, m * d * (4 + 2), 0.0)
    cur = ix.slab[torch.from_numpy(np.random.default_rng(0).integers(0, ix.n_rows, 4096)).to(dev)].clone()
    ms = _timed(lambda: ix.search_dense(cur, 100), 3, stream)
    n5 = ix.n_rows
    report(f"streaming: {n5:,} x 384 fp16, batch 4,096, top-100", ms, 4096, algorithmic_bytes(n5, d, 4096, 100),
           2.0 * 4096 * n5 * d, _kernel_ms(lambda: ix.search_dense(cur, 100), 3, stream))
    ix.close()
    return 0


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=2048)
    ap.add_argument("--warmup", type=int, default=64)
    ap.add_argument("--copies", type=int, default=COPIES)
    ap.add_argument("--cpu-budget", type=float, default=12.0)
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--pmc-pass", action="store_true",
                    help="a short run for counter collection: one reference copy, then 8 cold searches")
    ap.add_argument("--pmc-summarize", metavar="DIR", help="write the traffic record from two --pmc runs")
    ap.add_argument("--trace-summarize", metavar="DIR", help="write the kernel statistics of a traced run")
    ap.add_argument("--suite-trace-summarize", metavar="DIR",
                    help="write the kernel statistics of a traced --suite run")
    ap.add_argument("--suite", action="store_true", help="time every workload (one JSON line each)")
    ap.add_argument("--pmc-workload", choices=sorted(PMC_WORKLOADS),
                    help="a short run of one workload for counter collection (with --pmc-summarize: summarise)")
    args = ap.parse_args()
    if args.pmc_workload and args.pmc_summarize:
        return pmc_workload_summarize(args.pmc_workload, args.pmc_summarize)
    if args.pmc_summarize:
        return pmc_summarize(args.pmc_summarize)
    if args.pmc_workload:
        return pmc_workload_run(args.pmc_workload)
    if args.trace_summarize:
        return trace_summarize(args.trace_summarize)
    if args.suite_trace_summarize:
        return trace_summarize(args.suite_trace_summarize, suite=True)
    if args.suite:
        if args.gpus != 1:
            print("the suite runs on one GPU only", file=sys.stderr)
            return 2
        return suite()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: --gpus {args.gpus} is not supported (the multi-GPU sharding "
              f"of the index is a design, not code, in this library)", file=sys.stderr)
        return 2

    import torch

    import synth
    import paper_2608_08340_amd as P
    from paper_2608_08340_amd import Index

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 2
    dev = torch.device("cuda", 0)
    log("generating 32,768 x 1,024 bf16 rows")
    w = synth.dense_32k()
    rows_dev = w.rows.to(dev)
    q = w.queries[:BATCH].contiguous().to(dev)
    copies = max(1, args.copies)

    if args.pmc_pass:
        ref = Index(DIM, COPY_ROWS, torch.bfloat16)
        src = torch.zeros((COPY_ROWS, DIM), dtype=torch.bfloat16, device=dev)
        ref.upsert(src)  # one same-dtype copy of known size: the scale reference
        torch.cuda.synchronize()
        idxs = []
        for c in range(8):
            ix = Index(DIM, N_ROWS, torch.bfloat16)
            ix.upsert(rows_dev)
            idxs.append(ix)
        torch.cuda.synchronize()
        for ix in idxs:
            ix.search_dense(q, K)
        torch.cuda.synchronize()
        print("pmc pass done", flush=True)
        return 0

    idxs = []
    for c in range(copies):
        ix = Index(DIM, N_ROWS, torch.bfloat16)
        ix.upsert(rows_dev)
        idxs.append(ix)
    del rows_dev
    outs = [(torch.empty((BATCH, K), dtype=torch.float32, device=dev),
             torch.empty((BATCH, K), dtype=torch.int64, device=dev)) for _ in range(copies)]
    for c in range(copies):
        idxs[c].workspace(0, BATCH, K)
        idxs[c].search_dense(q, K, out=outs[c])
    torch.cuda.synchronize()
    for c in range(1, copies):  # every copy returns the same lists
        assert torch.equal(outs[c][1], outs[0][1])

    steps = max(1, args.steps)
    warm = max(0, args.warmup)
    stream = torch.cuda.current_stream(dev)
    def capture(n):
        """A HIP graph of n consecutive steps over slabs 0 .. n-1."""
        gr = torch.cuda.CUDAGraph()
        with torch.cuda.graph(gr):
            for c in range(n):
                idxs[c].search_dense(q, K, out=outs[c])
        torch.cuda.synchronize()
        return gr

    g_full = capture(copies)
    rem = steps % copies
    g_rem = capture(rem) if rem else None

    def run(n):
        for _ in range(n // copies):
            g_full.replay()
        if n % copies:
            g_rem.replay()

    log(f"warmup {warm} steps")
    run(warm)
    torch.cuda.synchronize()
    ref_ids = outs[0][1].clone()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    log(f"timing {steps} steps (graph replay over {copies} slabs)")
    torch.cuda.synchronize()
    e0.record(stream)
    t0 = time.perf_counter()
    run(steps)
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = e0.elapsed_time(e1) / steps
    for c in range(min(copies, steps)):
        assert torch.equal(outs[c][1], ref_ids), "graph replay changed the result"

    # ---- eager calls: per-call percentiles, and the scoring kernel's own duration from the
    # events its dispatch carries
    n_eager = min(steps, 512)
    cev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n_eager)]
    kev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n_eager)]
    for a, b in kev:  # create the events (torch makes them on first record) before the library records them
        a.record(stream)
        b.record(stream)
    torch.cuda.synchronize()
    for i in range(n_eager):
        cev[i][0].record(stream)
        P.time_next_dense_kernel(*kev[i])
        idxs[i % copies].search_dense(q, K, out=outs[i % copies])
        cev[i][1].record(stream)
    torch.cuda.synchronize()
    call_ms = np.array([a.elapsed_time(b) for a, b in cev])
    kern_ms = np.array([a.elapsed_time(b) for a, b in kev])
    kernel_ms = float(kern_ms.mean())
    kernel_src = f"HIP events carried by the kernel's dispatch, mean of {n_eager} eager calls"

    # ---- warm: one slab, graph of 16 searches on it
    gw = torch.cuda.CUDAGraph()
    with torch.cuda.graph(gw):
        for c in range(copies):
            idxs[0].search_dense(q, K, out=outs[0])
    torch.cuda.synchronize()
    gw.replay()
    torch.cuda.synchronize()
    reps = max(1, 256 // copies)
    e0.record(stream)
    for _ in range(reps):
        gw.replay()
    e1.record(stream)
    torch.cuda.synchronize()
    warm_ms = e0.elapsed_time(e1) / (reps * copies)

    value = BATCH / (ms / 1e3)
    abytes = algorithmic_bytes(N_ROWS, DIM, BATCH, K)
    flops = 2.0 * BATCH * N_ROWS * DIM
    achieved = abytes / (kernel_ms / 1e3) / 1e9
    traffic, traffic_note = traffic_record()
    result = {
        "metric": METRIC, "value": round(value, 1), "unit": "queries/s", "n_gpus": 1,
        "steps": steps, "warmup": warm, "ms_per_step": round(ms, 5), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "dense exact top-5 over 32,768 x 1,024 bf16 unit rows (256-cluster mixture), "
                               "batch 256, fp32 accumulation; 16 slab copies rotated (HBM-cold), HIP-graph replay",
                   "n_rows": N_ROWS, "dim": DIM, "batch": BATCH, "k": K, "slab_copies": copies},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic},
        "kernel": {"name": "dense_mfma_kernel (scoring; BN=128 queries x 256 rows per workgroup)",
                   "avg_us": round(kernel_ms * 1e3, 2), "timing": kernel_src,
                   "p10_p50_p90_us": [round(float(np.percentile(kern_ms, p)) * 1e3, 2) for p in (10, 50, 90)],
                   "algorithmic_bytes_per_launch": abytes, "flops_per_launch": flops,
                   "mfma_tflops": round(flops / (kernel_ms / 1e3) / 1e12, 1),
                   "mfma_frac": round(flops / (kernel_ms / 1e3) / 1e12 / BF16_PEAK_TFLOPS, 4),
                   "traffic_note": traffic_note},
        "call_us_p10_p50_p90": [round(float(np.percentile(call_ms, p)) * 1e3, 2) for p in (10, 50, 90)],
        "eager_queries_per_s": round(BATCH / (float(np.median(call_ms)) / 1e3), 1),
        "warm_queries_per_s": round(BATCH / (warm_ms / 1e3), 1),
        "wall_s_timed": round(wall, 3),
    }
    if not args.no_cpu:
        log("timing the CPU oracle")
        result["cpu_baseline"] = cpu_baseline(w.rows, w.queries, args.cpu_budget)
    result["paper_context"] = PAPER_CONTEXT
    print(json.dumps(result), flush=True)
    for ix in idxs:
        ix.close()
    return 0


if __name__ == "__main__":
    sys.exit(main())
