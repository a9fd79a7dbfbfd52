"""Benchmark of the FlashLoop per-loop step on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload C4] [--no-cpu-baseline]
    python bench.py --copy-calib        # plain copy kernel of known size (HBM counter calibration)

One step = every sparse loop r = 2..R of one layer over one batch of synthetic input, each loop being
the whole hot path: token scoring + top-k, K and V residual quantization (with the reconstructed new
rows), the mass-corrected sparse attention update, and the in-place dequantization that commits the new
rows into the K/V caches.  Loop 2 computes both passes of the update and keeps its add terms; loops 3..R
take the previous loop's add terms as their subtract terms (the column sets are fixed and the active rows
nested, so the two are equal in exact arithmetic) and keep their own.  The dense loop-1 set-up (base codec, dense attention, fp64 column statistic,
column lists) runs once before timing.  Inputs are resident in HBM before the timed region; every step
re-runs loops 2..R on the state the previous step left (the work of each call depends only on the
fixed budgets, not on the values).

Prints ONE JSON line with the metric (updated rows per second per layer-loop), the roofline of the
dominant kernel measured with HIP events on the launch stream, and the CPU oracle timed on a bounded
sample of the same workload.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "updated-token attn rows/s per layer-loop + achieved HBM GB/s & MFMA % at 32K"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
MFMA_BF16_TFLOPS = 2500.0      # dense bf16/fp16 MFMA
FP64_VECTOR_TFLOPS = 78.6      # fp64 vector FMA (the pruning statistic)
PROFILE_DIR = os.path.join(ROOT, "profiles")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


# ---- algorithmic work of each call (what the method itself must move / compute) ----------------------
def attn_work(idx, cols, slot, N, H, d, window, B, reuse=False, keep_terms=True, current=False, sub_only=False):
    """Exact algorithmic bytes and flops of one sparse attention launch.

    flops = 8 d * sum over (b, h, i in A) |S_i|  (two passes, each q.k and p.v), or 4 d * ... when the
            subtract terms are the previous loop's stored add terms (reuse: the add pass only);
    bytes = Q rows of loops r and r-1 (r only with reuse), o in/out and lse in/out (out only with reuse)
            of the updated rows, every distinct column of K/V touched by some S_i (cache rows, plus the
            new rows of updated columns), the column list and the slot entries of the touched columns;
            with reuse the previous terms, masses and slot entries of the rows are read, and with
            keep_terms this loop's terms and masses are written.  current: the caches already hold the
            new rows (reuse only), so every touched column is one cache row and no slot entry is read.
            sub_only: the subtract pass alone over the previous loop's caches (4 d flops per column; q_prev
            rows, lse in, the touched cache rows and the list read; the terms and masses written).
    """
    if sub_only:
        reuse, current = True, True
    flops = 0.0
    nbytes = 0.0
    for b in range(B):
        rows = idx[b].astype(np.int64)
        k = rows.size
        upd = slot[b] >= 0
        for h in range(H):
            g = np.sort(cols[b, h].astype(np.int64))
            n_list = np.searchsorted(g, rows - window, side="right")         # list columns j <= i - w
            n_band = np.minimum(window, rows + 1) if window > 0 else 0
            flops += (4.0 if reuse else 8.0) * d * float(np.sum(n_list + n_band))
            used = np.zeros(N, dtype=bool)
            if rows.size:
                used[g[g <= rows.max() - window]] = True
                if window > 0:
                    diff = np.zeros(N + 1, dtype=np.int64)
                    np.add.at(diff, np.maximum(rows - window + 1, 0), 1)
                    np.add.at(diff, rows + 1, -1)
                    used |= np.cumsum(diff[:N]) > 0
            n_used = int(used.sum())
            n_new = 0 if current else int((used & upd).sum())
            nbytes += (n_used + n_new) * d * 2 * 2          # K and V rows, bf16
            nbytes += (0 if current else n_used * 4) + g.size * 4   # slot lookups and the column list
        nbytes += k * H * d * 2 * (1 if reuse else 2)       # q_cur (and q_prev) rows
        nbytes += k * 4
        if sub_only:                                        # lse in, terms and masses out
            nbytes += k * H * 4 + k * H * d * 4 + k * H * 4
            continue
        nbytes += k * H * d * 4 * 2 + k * H * 4 * (1 if reuse else 2)   # o in/out, lse (in/)out
        if reuse:
            nbytes += k * H * d * 4 + k * H * 4 + k * 4     # previous terms, masses, slot entries
        if keep_terms:
            nbytes += k * H * d * 4 + k * H * 4             # this loop's terms and masses
    return nbytes, flops


def codec_bytes(k, H, d, bits, group, axis_token, B):
    """quantize: read cur + ref rows, write codes + metadata + reconstructed rows (compact, or committed
    into the cache in place: the same bytes)."""
    rows = B * k * H * d
    meta = B * (math.ceil(k / group) * H * d if axis_token else k * H * (d // group)) * 2 * 2
    return rows * 2 * 2 + rows * bits / 8 + meta + rows * 2 + B * k * 4


def commit_bytes(k, H, d, bits, group, axis_token, B):
    """dequantize in place: read codes + metadata + cache rows, write cache rows."""
    rows = B * k * H * d
    meta = B * (math.ceil(k / group) * H * d if axis_token else k * H * (d // group)) * 2 * 2
    return rows * bits / 8 + meta + rows * 2 * 2 + B * k * 4


def select_bytes(n_cand, N, D, k, B):
    return B * (n_cand * D * 2 * 4 + n_cand * 4 * 2 + k * 4 + N * 4 + n_cand * 4)


# ---- the timed step ------------------------------------------------------------------------------------
class Step:
    def __init__(self, w, dev, gs, fl, torch):
        from paper_2609_29812_amd import driver
        self.w, self.dev, self.gs, self.fl, self.torch, self.driver = w, dev, gs, fl, torch, driver

    def run(self, events=None):
        """One step (loops 2..R).  events: optional dict name -> list of (start, end) event pairs."""
        w, dev, gs, fl, driver = self.w, self.dev, self.gs, self.fl, self.driver
        torch = self.torch
        gs.cand = None
        trace = []

        def timed(name, fn):
            if events is None:
                return fn()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            out = fn()
            e1.record()
            events.setdefault(name, []).append((e0, e1))
            return out

        for r in range(2, w.loops + 1):
            qr, qp = dev["q"][r - 1], dev["q"][r - 2]
            kr, kp = dev["k"][r - 1], dev["k"][r - 2]
            vr, vp = dev["v"][r - 1], dev["v"][r - 2]
            bits, kk = w.bits_at(r), w.k(r)
            idx, slot, _ = timed(f"select r{r}", lambda: fl.select_tokens(kr, kp, vr, vp, kk, cand=gs.cand))
            B, N, H, d = kr.shape
            term = torch.empty(B, kk, H, d, dtype=torch.float32, device=kr.device)
            mass = torch.empty(B, kk, H, dtype=torch.float32, device=kr.device)
            split = r == 2 and driver.subtract_pass_first(kk, gs.cols.shape[2], gs.window, B, N, H, d)
            if split:
                # the subtract pass over the loop-1 state, then as loops 3, 4: quantize and commit in one
                # pass, and the add pass over the caches with the just-computed subtract terms
                sub, msub = timed(f"sub r{r}", lambda: fl.subtract_terms(qp, gs.k_hat, gs.v_hat, idx, gs.cols,
                                                                         gs.window, gs.lse, v16=gs.v16))
                timed(f"quant_kv r{r}", lambda: fl.kv_residual_quant_kv(
                    kr, gs.k_hat, vr, gs.v_hat, idx, bits, gs.group, mode=fl.DQ_COMMIT, v_f16=gs.v16))
                timed(f"attn r{r}", lambda: fl.loop_sparse_attn(
                    qr, None, gs.k_hat, gs.v_hat, None, None, slot, idx, gs.cols, gs.window, gs.lse, gs.o,
                    term_prev=sub, mass_prev=msub, slot_prev=slot, term_out=term, mass_out=mass, v16=gs.v16))
            elif r == 2:
                # both passes: quantize (compact new rows), attend, then commit into the caches
                (ck, sk, zk, k_new), (cv, sv, zv, v_new) = timed(f"quant_kv r{r}", lambda: fl.kv_residual_quant_kv(
                    kr, gs.k_hat, vr, gs.v_hat, idx, bits, gs.group))
                timed(f"attn r{r}", lambda: fl.loop_sparse_attn(
                    qr, qp, gs.k_hat, gs.v_hat, k_new, v_new, slot, idx, gs.cols, gs.window, gs.lse, gs.o,
                    term_out=term, mass_out=mass))
                timed(f"commit_kv r{r}", lambda: fl.kv_residual_dequant_kv(
                    (ck, sk, zk), (cv, sv, zv), idx, bits, gs.group, gs.k_hat, gs.v_hat, mode=fl.DQ_COMMIT))
                if gs.v16 is not None:
                    timed(f"v16 r{r}", lambda: fl.kv_f16_rows(gs.v_hat, idx, out=gs.v16))
            else:
                # the add pass alone: quantize and commit in one pass, then attend over the caches
                timed(f"quant_kv r{r}", lambda: fl.kv_residual_quant_kv(
                    kr, gs.k_hat, vr, gs.v_hat, idx, bits, gs.group, mode=fl.DQ_COMMIT, v_f16=gs.v16))
                timed(f"attn r{r}", lambda: fl.loop_sparse_attn(
                    qr, None, gs.k_hat, gs.v_hat, None, None, slot, idx, gs.cols, gs.window, gs.lse, gs.o,
                    term_prev=gs.term, mass_prev=gs.mass, slot_prev=gs.slot_prev, term_out=term, mass_out=mass,
                    v16=gs.v16))
            gs.term, gs.mass, gs.slot_prev = term, mass, slot
            trace.append((r, idx, slot))
            gs.cand = idx
        return trace


def capture_step(step, torch):
    """One step captured in a HIP graph (torch.cuda.CUDAGraph on ROCm): every launch of loops 2..R on the
    capture stream, its buffers from the graph's pool.  Replays redo the step on the layer state as it
    stands, as the eager loop does.  None if capture fails (the eager number stands then)."""
    try:
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            step.run()
        torch.cuda.synchronize()
        return g
    except Exception as e:   # (reported; the bench keeps the eager timing)
        log(f"[bench] graph capture failed: {e}")
        return None


def source_sha(path):
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


KERNEL_SRC = {"seg_cur_kernel": "fl_seg_attn.hip", "seg_sub_kernel": "fl_seg_attn.hip", "seg1_cur_kernel": "fl_seg_attn.hip",
              "seg1_sub_kernel": "fl_seg_attn.hip", "loop_attn_kernel": "fl_attn.hip", "cur_attn_kernel": "fl_attn.hip",
              "cur_sub_kernel": "fl_attn.hip", "reuse_attn_kernel": "fl_attn.hip"}


def load_counters(kernel, workload):
    """HBM traffic and MFMA busy fraction per launch from committed rocprofv3 counter runs
    (profiles/<kernel>_<workload>_counters.json), used only when taken on the kernel's current source:
    traffic = FETCH_SIZE and WRITE_SIZE scaled by a 1 GiB copy's; traffic_dram = the DRAM request counters
    times their request sizes."""
    none = {"traffic": None, "traffic_dram": None, "traffic_dram_read": None, "traffic_dram_write": None,
            "mfma_busy": None}
    path = os.path.join(PROFILE_DIR, f"{kernel}_{workload}_counters.json")
    src = os.path.join(ROOT, "paper_2609_29812_amd", "csrc", KERNEL_SRC.get(kernel, "fl_attn.hip"))
    if not os.path.exists(path):
        return none
    with open(path) as f:
        rec = json.load(f)
    if rec.get("source_sha") != source_sha(src):
        return none
    rd, wr = rec.get("dram_read_bytes_per_launch"), rec.get("dram_write_bytes_per_launch")
    return {"traffic": rec.get("fetch_write_bytes_per_launch"),
            "traffic_dram": None if rd is None or wr is None else int(rd + wr), "traffic_dram_read": rd,
            "traffic_dram_write": wr, "mfma_busy": rec.get("mfma_busy")}


# ---- CPU oracle leg ------------------------------------------------------------------------------------
def cpu_baseline(w, st, threads_note):
    """The oracle's per-loop step (select + codec for every head, the update for every active row of
    head 0, scaled by the head count) on the host cores; the dense loop-1 set-up for head 0 is untimed."""
    from oracle import attention as att
    from oracle import chain as och
    from oracle import codec, select
    from oracle.numerics import bf16_to_f64

    t0 = time.time()
    rec = och.loop1(st, heads=[0])
    log(f"[cpu] oracle loop-1 setup (head 0, untimed) {time.time() - t0:.1f}s")
    t_est = 0.0
    t_cpu = 0.0
    rows_total = 0
    reps = 0
    while reps < 1 or (t_cpu < 10.0 and reps < 8):     # about 10 s of CPU work, whole steps only
        reps += 1
        o = {key: v.copy() for key, v in rec.o1.items()}
        lse = {key: v.copy() for key, v in rec.lse1.items()}
        k_hat, v_hat = rec.k_hat1, rec.v_hat1
        cand = None
        for r in range(2, w.loops + 1):
            ta = time.perf_counter()
            keys = select.token_keys([(st.k[r - 1], st.k[r - 2]), (st.v[r - 1], st.v[r - 2])], cand)
            idx, slot = select.nested_topk(keys, cand, w.k(r), w.seq)
            bits = w.bits_at(r)
            ek = codec.quantize(st.k[r - 1], k_hat, idx, bits, w.group, codec.AXIS_TOKEN)
            k_new_hat, _ = codec.reconstruct(k_hat, st.k[r - 1], idx, ek, bits, w.group, codec.AXIS_TOKEN)
            ev = codec.quantize(st.v[r - 1], v_hat, idx, bits, w.group, codec.AXIS_CHANNEL)
            v_new_hat, _ = codec.reconstruct(v_hat, st.v[r - 1], idx, ev, bits, w.group, codec.AXIS_CHANNEL)
            tb = time.perf_counter()
            for b in range(w.batch):
                kp, vp = bf16_to_f64(k_hat[b, :, 0]), bf16_to_f64(v_hat[b, :, 0])
                kc, vc = bf16_to_f64(k_new_hat[b, :, 0]), bf16_to_f64(v_new_hat[b, :, 0])
                qc, qp = bf16_to_f64(st.q[r - 1][b, :, 0]), bf16_to_f64(st.q[r - 2][b, :, 0])
                for i in idx[b]:
                    S = att.row_columns(rec.cols[b, 0], int(i), w.window)
                    o[b, 0][i], lse[b, 0][i], _ = att.correct_row(S, qc[i], qp[i], kp, vp, kc, vc, lse[b, 0][i],
                                                                  o[b, 0][i], w.sm_scale)
            tc = time.perf_counter()
            t_est += (tb - ta) + (tc - tb) * w.heads
            t_cpu += tc - ta
            rows_total += w.batch * w.k(r)
            k_hat, v_hat, cand = k_new_hat, v_new_hat, idx
    return {
        "value": rows_total / t_est,
        "unit": "rows/s",
        "cores": threads_note,
        "host_cores": len(os.sched_getaffinity(0)),
        "cores_note": "cores = the BLAS threads the oracle's matrix products use; its elementwise numpy work is "
                      "single-threaded; host_cores = the cores this process may run on",
        "kind": "oracle",
        "sample": (f"{w.name} loops 2-{w.loops}: token scoring, top-k and the K/V residual codec for all "
                   f"{w.heads} heads, the mass-corrected update for every active row of head 0 only "
                   f"(its time x{w.heads}); {reps} repetition(s), {t_cpu:.1f}s of CPU work, estimated full "
                   f"steps {t_est:.1f}s"),
    }


def blas_threads():
    try:
        from threadpoolctl import threadpool_info
        n = [i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"]
        return max(n) if n else 1
    except Exception:
        return 1


# ---- copy calibration ----------------------------------------------------------------------------------
def copy_calib():
    import torch
    nbytes = 1 << 30
    src = torch.empty(nbytes // 4, dtype=torch.float32, device="cuda").fill_(1.0)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(5):
        torch.mul(src, 1.0, out=dst)      # one elementwise kernel: reads and writes nbytes each
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": nbytes, "copy_bytes_written": nbytes, "dispatches": 5}), flush=True)


# ---- counter summaries -------------------------------------------------------------------------------------
# Per-dispatch request sizes of the L2 -> memory interface: writes are 64-byte requests (a 1 GiB copy
# writes exactly 2^24 of them); reads are 128-byte requests (the TCC_EA0_RDREQ_{32B,64B,128B} split of the
# same runs), and a 1 GiB copy issues 0.83 GiB of them: the rest of its source is served from the
# last-level cache (MALL) in front of HBM, whose hits are no HBM traffic.
DRAM_READ_REQ_BYTES = 128
DRAM_WRITE_REQ_BYTES = 64


def _pmc_means(dirs, kernel):
    import collections
    import csv
    import glob
    per = collections.defaultdict(lambda: collections.defaultdict(float))   # counter -> dispatch -> sum
    names = set()
    for d in dirs:
        for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
            with open(f) as fh:
                for r in csv.DictReader(fh):
                    if kernel not in r["Kernel_Name"]:
                        continue
                    names.add(r["Kernel_Name"])
                    per[r["Counter_Name"]][(f, r["Dispatch_Id"])] += float(r["Counter_Value"])
    return {c: sum(v.values()) / len(v) for c, v in per.items()}, {c: len(v) for c, v in per.items()}, names


def pmc_summary(kernel, workload, dirs, commands, copy_dirs=()):
    """Summarize rocprofv3 --pmc runs (counter_collection.csv under each dir) of one kernel into
    profiles/<kernel>_<workload>_counters.json: per-dispatch means of every counter (summed over its
    dimensions), the DRAM bytes they imply, and the MFMA busy fraction."""
    mean, n_disp, names = _pmc_means(dirs, kernel)
    if not mean:
        raise SystemExit(f"no dispatches of {kernel} under {dirs}")
    rec = {"kernel": sorted(names), "workload": workload,
           "source_sha": source_sha(os.path.join(ROOT, "paper_2609_29812_amd", "csrc", KERNEL_SRC[kernel])),
           "counters_per_dispatch": {c: round(v, 1) for c, v in sorted(mean.items())},
           "dispatches": n_disp}
    rd, wr = mean.get("TCC_EA0_RDREQ_DRAM_sum"), mean.get("TCC_EA0_WRREQ_DRAM_sum")
    rec["dram_read_bytes_per_launch"] = None if rd is None else int(rd * DRAM_READ_REQ_BYTES)
    rec["dram_write_bytes_per_launch"] = None if wr is None else int(wr * DRAM_WRITE_REQ_BYTES)
    tot = mean.get("TCC_EA0_RDREQ_sum")
    if tot:
        rec["read_request_mix"] = {sz: round(mean.get(f"TCC_EA0_RDREQ_{sz}_sum", 0.0) / tot, 4)
                                   for sz in ("32B", "64B", "128B")}
    busy, active = mean.get("SQ_VALU_MFMA_BUSY_CYCLES"), mean.get("SQ_BUSY_CU_CYCLES")
    # both sum over the chip: MFMA busy cycles over the SIMDs (four per CU), busy cycles over the CUs
    rec["mfma_busy"] = None if not busy or not active else round(busy / (4 * active), 4)
    if copy_dirs:
        # FETCH_SIZE / WRITE_SIZE (KiB) scaled by what they read for a copy of 1 GiB each way
        cm, _, _ = _pmc_means(copy_dirs, "elementwise")
        fs, ws = cm.get("FETCH_SIZE"), cm.get("WRITE_SIZE")
        rec["copy_calibration"] = {
            "kernel": "elementwise copy (torch.mul(src, 1.0, out=dst)), 1 GiB read + 1 GiB written",
            "counters_per_dispatch": {c: round(v, 1) for c, v in sorted(cm.items())}}
        if fs and ws and "FETCH_SIZE" in mean and "WRITE_SIZE" in mean:
            f_scale, w_scale = (1 << 20) / fs, (1 << 20) / ws
            rec["copy_calibration"].update(fetch_scale=round(f_scale, 4), write_scale=round(w_scale, 4))
            rec["fetch_write_bytes_per_launch"] = int((mean["FETCH_SIZE"] * f_scale + mean["WRITE_SIZE"] * w_scale) * 1024)
    rec["commands"] = commands
    rec["note"] = ("R = repository root.  dram bytes = TCC_EA0_RDREQ_DRAM_sum x 128 + TCC_EA0_WRREQ_DRAM_sum x 64 "
                   "per dispatch; mfma_busy = SQ_VALU_MFMA_BUSY_CYCLES / (4 SIMDs per CU x SQ_BUSY_CU_CYCLES)")
    out = os.path.join(PROFILE_DIR, f"{kernel}_{workload}_counters.json")
    with open(out, "w") as fh:
        json.dump(rec, fh, indent=1)
    print(json.dumps({k: rec[k] for k in ("dram_read_bytes_per_launch", "dram_write_bytes_per_launch",
                                          "mfma_busy")}), flush=True)


def trace_summary(title, command, trace_dir, out_name):
    """Markdown table of a rocprofv3 --kernel-trace run (kernel_trace.csv under trace_dir) into
    profiles/<out_name>.md: per kernel and grid, the calls and their durations."""
    import collections
    import csv
    import glob
    files = glob.glob(os.path.join(trace_dir, "**", "*kernel_trace.csv"), recursive=True)
    if not files:
        raise SystemExit(f"no kernel_trace.csv under {trace_dir}")
    groups = collections.defaultdict(list)
    meta = {}
    for f in files:
        with open(f) as fh:
            for r in csv.DictReader(fh):
                grid = "x".join(r.get(f"Grid_Size_{a}", "1") for a in "XYZ")
                key = (r["Kernel_Name"], grid)
                groups[key].append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
                meta[key] = (r.get("Workgroup_Size_X", ""), r.get("Arch_VGPR_Count", r.get("VGPR_Count", "")),
                             r.get("Accum_VGPR_Count", ""), r.get("LDS_Block_Size", r.get("Group_Segment_Size", "")),
                             r.get("Scratch_Size", r.get("Private_Segment_Size", "")))
    total = sum(sum(v) for v in groups.values())
    lines = [f"# {title}", "", "Command (run from the repository root on the MI355X box; R = repository root):", "",
             "```", command, "```", "",
             "Durations of one kernel drift upward over a sustained run of back-to-back steps (the graph replays "
             "come last) and recover after a pause, which is the chip's clock management; the minimum and the "
             "median bracket what the benchmark's shorter per-kernel HIP-event pass measures.", "",
             "| kernel | grid (work-items) | wg | vgpr/agpr | LDS B | scratch | calls | avg us | median us | min us | "
             "max us | % time |",
             "|---|---|---|---|---|---|---|---|---|---|---|---|"]
    for key, v in sorted(groups.items(), key=lambda kv: -sum(kv[1])):
        wg, vg, ag, lds, scr = meta[key]
        name = key[0].replace("void ", "").split("(")[0].replace("|", "\\|")
        lines.append(f"| {name} | {key[1]} | {wg} | {vg}/{ag} | {lds} | {scr} | {len(v)} | {sum(v) / len(v):.2f} | "
                     f"{float(np.median(v)):.2f} | {min(v):.2f} | {max(v):.2f} | {100 * sum(v) / total:.1f} |")
    with open(os.path.join(PROFILE_DIR, f"{out_name}.md"), "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print("\n".join(lines[8:]), flush=True)


def gpu_sleep_cycles(ms, torch):
    """Cycles for torch.cuda._sleep (a spin kernel) to last about `ms` milliseconds, measured here."""
    n = 1 << 20
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    a.record()
    torch.cuda._sleep(n)
    b.record()
    torch.cuda.synchronize()
    per_ms = n / max(a.elapsed_time(b), 1e-3)
    return int(min(max(ms * per_ms, 1e4), 1e10))


def workload_config(w):
    return {"workload": w.name, "batch": w.batch, "seq": w.seq, "heads": w.heads, "head_dim": w.head_dim,
            "loops": w.loops, "sparse_loops": f"2-{w.loops}",
            "rows_per_step": sum(w.batch * w.k(r) for r in range(2, w.loops + 1)),
            "k_per_loop": [w.k(r) for r in range(2, w.loops + 1)], "column_budget": w.col_budget,
            "window": w.window, "residual_bits": list(w.bits), "group": w.group}


def measure(w, dev, driver, fl, torch, steps, warmup, log_calls=False):
    """Set-up, then W warm-up steps and K timed steps (HIP events on the launch stream around the K steps);
    then a separate pass with events around every call, for the per-call durations and the rooflines."""
    t0 = time.time()
    gs = driver.setup(dev["q"][0], dev["k"][0], dev["v"][0], w.base_bits, w.group, w.n_sink, w.top_cols,
                      w.window)
    torch.cuda.synchronize()
    log(f"[bench] {w.name}: loop-1 setup on GPU {time.time() - t0:.2f}s")
    step = Step(w, dev, gs, fl, torch)
    for _ in range(warmup):
        step.run()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t_wall = time.perf_counter()
    e0.record()
    for _ in range(steps):
        step.run()
    e1.record()
    torch.cuda.synchronize()
    t_wall = time.perf_counter() - t_wall
    ms_eager = e0.elapsed_time(e1) / steps
    rows_per_step = sum(w.batch * w.k(r) for r in range(2, w.loops + 1))
    log(f"[bench] {w.name}: {steps} steps: {ms_eager:.4f} ms/step (wall {t_wall / steps * 1e3:.4f} ms)")

    # the same step captured once in a graph and replayed; the step time is the faster of the two (the replay
    # pays off where the step is launch-bound: the small workloads; at 32K the eager launches keep ahead)
    ms_graph = None
    graph = capture_step(step, torch)
    if graph is not None:
        for _ in range(warmup):
            graph.replay()
        torch.cuda.synchronize()
        e0.record()
        for _ in range(steps):
            graph.replay()
        e1.record()
        torch.cuda.synchronize()
        ms_graph = e0.elapsed_time(e1) / steps
        log(f"[bench] {w.name}: {steps} graph replays: {ms_graph:.4f} ms/step")
    mode = "graph replay" if ms_graph is not None and ms_graph < ms_eager else "eager"
    ms_step = ms_graph if mode == "graph replay" else ms_eager

    # per-call durations with events on the launch stream (a separate pass, same work).  The GPU sleeps
    # before each step of this pass, so that the host has queued the step's calls by the time it wakes and
    # every event pair brackets kernels that run back to back (otherwise the GPU can idle inside an interval
    # while Python issues the next call after a short kernel).
    sleep_cycles = gpu_sleep_cycles(2.0, torch)
    events = {}
    reps = max(3, min(steps, 10))
    trace = None
    for _ in range(reps):
        torch.cuda._sleep(sleep_cycles)
        trace = step.run(events)
    torch.cuda.synchronize()
    dur_us = {name: float(np.mean([a.elapsed_time(b) for a, b in pairs])) * 1e3 for name, pairs in events.items()}

    cols = gs.cols.cpu().numpy()
    B, N, H, d = w.batch, w.seq, w.heads, w.head_dim
    kernels = {}
    attn_us = 0.0
    per_kernel = {}               # kernel -> [bytes, flops, us, launches]
    total_bytes = 0.0
    n_cand = N
    for r, idx_t, slot_t in trace:
        idx, slot = idx_t.cpu().numpy(), slot_t.cpu().numpy()
        kr, bits = w.k(r), w.bits_at(r)
        split = r == 2 and f"sub r{r}" in dur_us
        by, fl_ = attn_work(idx, cols, slot, N, H, d, w.window, B, reuse=r > 2 or split, current=r > 2 or split)
        # the fp16 copy of the committed value rows (written by the quantizer, or after the separate commit)
        v16_bytes = B * kr * H * d * 2 if gs.v16 is not None else 0
        two_pass = r == 2 and not split
        work = {
            f"select r{r}": (select_bytes(n_cand, N, H * d, kr, B), 0.0),
            f"quant_kv r{r}": (codec_bytes(kr, H, d, bits, w.group, True, B)
                               + codec_bytes(kr, H, d, bits, w.group, False, B) - B * kr * 4
                               + (0 if two_pass else v16_bytes), 0.0),
            f"attn r{r}": (by, fl_),
        }
        if split:
            work[f"sub r{r}"] = attn_work(idx, cols, slot, N, H, d, w.window, B, sub_only=True)
        elif r == 2:
            work[f"commit_kv r{r}"] = (commit_bytes(kr, H, d, bits, w.group, True, B)
                                       + commit_bytes(kr, H, d, bits, w.group, False, B) - B * kr * 4, 0.0)
            if f"v16 r{r}" in dur_us:
                work[f"v16 r{r}"] = (2 * v16_bytes + B * kr * 4, 0.0)   # bf16 rows read, fp16 rows written
        for name, (nb, nf) in work.items():
            us = dur_us[name]
            kernels[name] = {"us": round(us, 2), "GB/s": round(nb / us / 1e3, 1),
                             "TFLOP/s": round(nf / us / 1e6, 2) if nf else None,
                             "alg_MB": round(nb / 1e6, 2), "alg_GF": round(nf / 1e9, 3) if nf else None}
            total_bytes += nb
        attn_us += dur_us[f"attn r{r}"]
        c_list = cols.shape[2]
        kname = fl.attn_kernel_name(fl.PASS_BOTH if (r == 2 and not split) else fl.PASS_ADD, kr, c_list, w.window,
                                    B, N, H, d)
        launches = [(kname, by, fl_, dur_us[f"attn r{r}"])]
        if split:
            attn_us += dur_us[f"sub r{r}"]
            launches.append((fl.attn_kernel_name(fl.PASS_SUBTRACT, kr, c_list, w.window, B, N, H, d),
                             *work[f"sub r{r}"], dur_us[f"sub r{r}"]))
        for kn, nb, nf, us in launches:
            acc = per_kernel.setdefault(kn, [0.0, 0.0, 0.0, 0])
            acc[0] += nb
            acc[1] += nf
            acc[2] += us
            acc[3] += 1
        n_cand = kr
    if log_calls:
        for name, kv in kernels.items():
            log(f"  {name:12s} {kv['us']:9.2f} us  {kv['GB/s']:8.1f} GB/s  alg {kv['alg_MB']:8.2f} MB"
                + (f"  {kv['TFLOP/s']:7.2f} TFLOP/s" if kv["TFLOP/s"] else ""))

    def roofline_of(kname):
        nb, nf, us, n = per_kernel[kname]
        t_hbm = nb / (HBM_PEAK_GBS * 1e9)
        t_mfma = nf / (MFMA_BF16_TFLOPS * 1e12)
        bound = "hbm" if t_hbm >= t_mfma else "mfma"
        if bound == "hbm":
            achieved, peak, unit = nb / (us * 1e-6) / 1e9, HBM_PEAK_GBS, "GB/s"
        else:
            achieved, peak, unit = nf / (us * 1e-6) / 1e12, MFMA_BF16_TFLOPS, "TFLOP/s"
        out = {"kernel": kname, "bound": bound, "achieved": round(achieved, 2), "peak": peak, "unit": unit,
               "frac": round(achieved / peak, 4), "traffic": None,
               "launches_per_step": n, "alg_bytes_per_launch": round(nb / n), "alg_flops_per_launch": round(nf / n),
               "avg_launch_us": round(us / n, 2),
               "mfma_frac": round(nf / (us * 1e-6) / 1e12 / MFMA_BF16_TFLOPS, 4),
               "hbm_frac": round(nb / (us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)}
        out.update(load_counters(kname, w.name))
        return out

    # the dominant kernel is the one with the most time per step
    order = sorted(per_kernel, key=lambda kn: -per_kernel[kn][2])
    return {"state": gs, "ms_per_step": ms_step, "ms_per_step_graph": ms_graph, "ms_per_step_eager": ms_eager,
            "step_mode": mode,
            "rows_per_step": rows_per_step,
            "step_hbm_GBps": round(total_bytes / (ms_step * 1e-3) / 1e9, 1),
            "attn_rows_per_s": round(rows_per_step / (attn_us * 1e-6), 1),
            "roofline": roofline_of(order[0]),
            "roofline_other_kernels": {kn: roofline_of(kn) for kn in order[1:]},
            "kernels": kernels}


# ---- main ----------------------------------------------------------------------------------------------
def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="C4")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-decode", action="store_true")
    ap.add_argument("--no-prune", action="store_true")
    ap.add_argument("--no-configs", action="store_true", help="only the 32K workload (no per-workload summaries)")
    ap.add_argument("--decode-only", action="store_true", help="only the decode measurement (for traces)")
    ap.add_argument("--copy-calib", action="store_true")
    ap.add_argument("--pmc-summary", nargs="+", metavar="ARG",
                    help="KERNEL WORKLOAD DIR [DIR ...]: summarize rocprofv3 --pmc runs into profiles/ (no GPU)")
    ap.add_argument("--pmc-command", action="append", default=[], help="a command recorded in the summary")
    ap.add_argument("--pmc-copy", nargs="*", default=[], help="counter dirs of the copy calibration runs")
    ap.add_argument("--trace-summary", nargs=4, metavar=("TITLE", "COMMAND", "TRACE_DIR", "OUT_NAME"),
                    help="summarize a rocprofv3 --kernel-trace run into profiles/OUT_NAME.md (no GPU)")
    args = ap.parse_args()
    if args.trace_summary:
        trace_summary(*args.trace_summary)
        return
    if args.pmc_summary:
        if len(args.pmc_summary) < 3:
            ap.error("--pmc-summary needs KERNEL WORKLOAD DIR [DIR ...]")
        pmc_summary(args.pmc_summary[0], args.pmc_summary[1], args.pmc_summary[2:], args.pmc_command, args.pmc_copy)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; there is no multi-GPU path (asked for {args.gpus}): "
              "the step would shard by head with one small all-gather of row-score partials.", flush=True)
        sys.exit(2)
    import torch
    torch.cuda.set_device(0)
    if args.copy_calib:
        copy_calib()
        return

    from paper_2609_29812_amd import driver
    from paper_2609_29812_amd import flashloop as fl
    from workloads import get, make_layer
    from workloads.gen_device import make_layer_device

    fl.load()
    w = get(args.workload)
    t0 = time.time()
    st = make_layer(w)
    log(f"[bench] generated {w.name} in {time.time() - t0:.1f}s")

    def up(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda().view(torch.bfloat16)

    dev = {n: [up(a) for a in getattr(st, n)] for n in "qkv"}
    if args.decode_only:
        gs = driver.setup(dev["q"][0], dev["k"][0], dev["v"][0], w.base_bits, w.group, w.n_sink, w.top_cols,
                          w.window)
        print(json.dumps({"decode": decode_bench(w, gs, fl, torch)}), flush=True)
        return
    m = measure(w, dev, driver, fl, torch, args.steps, args.warmup, log_calls=True)
    gs = m["state"]
    ms_step = m["ms_per_step"]
    rows_per_step = m["rows_per_step"]
    result = {
        "metric": METRIC,
        "value": round(rows_per_step / (ms_step * 1e-3), 1),
        "unit": "rows/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "step_mode": m["step_mode"],
        "ms_per_step_eager": round(m["ms_per_step_eager"], 4),
        "ms_per_step_graph_replay": None if m["ms_per_step_graph"] is None else round(m["ms_per_step_graph"], 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": workload_config(w),
        "step_hbm_GBps": m["step_hbm_GBps"],
        "attn_rows_per_s": m["attn_rows_per_s"],
        "roofline": m["roofline"],
        "roofline_other_kernels": m["roofline_other_kernels"],
        "kernels": m["kernels"],
    }
    if not args.no_configs:
        result["configs"] = {}
        for name in ("C1", "C2", "C3", "C5"):
            wc = get(name)
            t0 = time.time()
            devc = make_layer_device(wc)
            torch.cuda.synchronize()
            log(f"[bench] generated {wc.name} on the device in {time.time() - t0:.1f}s")
            mc = measure(wc, devc, driver, fl, torch, max(5, args.steps // 2), max(2, args.warmup // 2))
            rec = {"workload": wc.name, "config": workload_config(wc), "rows_per_step": mc["rows_per_step"],
                   "ms_per_step": round(mc["ms_per_step"], 4),
                   "step_mode": mc["step_mode"], "ms_per_step_eager": round(mc["ms_per_step_eager"], 4),
                   "ms_per_step_graph_replay": (None if mc["ms_per_step_graph"] is None
                                                else round(mc["ms_per_step_graph"], 4)),
                   "rows_per_s": round(mc["rows_per_step"] / (mc["ms_per_step"] * 1e-3), 1),
                   "attn_rows_per_s": mc["attn_rows_per_s"], "step_hbm_GBps": mc["step_hbm_GBps"],
                   "roofline": mc["roofline"], "roofline_other_kernels": mc["roofline_other_kernels"],
                   "attn_us_per_loop": {k_: v_["us"] for k_, v_ in mc["kernels"].items() if k_.startswith("attn")},
                   "data": "synthetic, drawn on the device with the same recipe (throughput does not depend on "
                           "the values)"}
            if wc.layers > 1:
                rec["stack"] = {"layers": wc.layers, "ms_per_step": round(mc["ms_per_step"] * wc.layers, 3),
                                "note": f"{wc.layers} x the layer-0 step (every layer has the same shapes and "
                                        "budgets; only the seeds differ)"}
            result["configs"][name] = rec
            del devc, mc
            torch.cuda.empty_cache()
    result["kv_footprint"] = kv_footprint(w)
    if not args.no_decode:
        result["decode"] = decode_bench(w, gs, fl, torch)
    if not args.no_prune:
        result["prune"] = prune_bench(w, gs, dev["q"][w.loops - 1], fl, torch)
        result["keep_recent"] = tail_bench(w, gs, dev["k"][w.loops - 1], fl, torch)
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(w, st, blas_threads())
    print(json.dumps(result), flush=True)


def kv_footprint(w):
    """Bytes of one layer's K and V state after the workload's last loop, stored three ways (Section 4.3, Eq. 4;
    Appendix E): a bf16 cache per loop (a looped model without the method); the packed streams the paper's
    engine keeps (int4 base codes and fp16 metadata, then each sparse loop's residual codes and metadata);
    and the one in-place bf16 cache pair this implementation keeps, with the fp16 copy of the value cache
    the attention reads."""
    B, N, H, d, G = w.batch, w.seq, w.heads, w.head_dim, w.group
    el = B * N * H * d
    per_loop_bf16 = w.loops * 2 * el * 2
    base = 2 * el * w.base_bits // 8
    base_meta = B * -(-N // G) * H * d * 4 + B * N * H * (d // G) * 4     # K per-channel, V per-token; z and s
    res = res_meta = 0
    for r in range(2, w.loops + 1):
        k = w.k(r)
        res += 2 * B * k * H * d * w.bits_at(r) // 8
        res_meta += B * -(-k // G) * H * d * 4 + B * k * H * (d // G) * 4
    packed = base + base_meta + res + res_meta
    working = 2 * el * 2 + el * 2          # bf16 K and V caches, fp16 copy of the values
    mb = lambda x: round(x / 1e6, 1)
    return {"workload": w.name, "bf16_cache_per_loop_MB": mb(per_loop_bf16),
            "packed_MB": mb(packed), "packed_bytes": packed, "packed_parts_MB": {"base_codes": mb(base), "base_metadata": mb(base_meta),
                                                       "residual_codes": mb(res), "residual_metadata": mb(res_meta)},
            "working_caches_MB": mb(working), "packed_reduction": round(per_loop_bf16 / packed, 2),
            "working_reduction": round(per_loop_bf16 / working, 2)}


def decode_work(B, T, H, d, c, c_next):
    """Algorithmic bytes of one decode step: the K and V rows of the attended columns, the query, the
    output (read unless dense, written), the column list, the cached subtract term, the next loop's
    columns and subtract term, and the V rows of the selected columns when the next loop keeps fewer than
    all of them (keeping all, its subtract term is this loop's add term)."""
    n = T if c == 0 else c
    nb = B * H * n * d * 2 * 2 + B * H * d * 2 + B * H * d * 4 * (1 if c == 0 else 3) + B * H * 4 * 2
    if c:
        nb += B * H * c * 4
    if c_next:
        nb += B * H * c_next * 4 + B * H * d * 4
        if c_next < n:
            nb += B * H * c_next * d * 2
    return nb


def decode_bench(w, gs, fl, torch):
    """The decode step for one new position of the workload's context: a dense source loop over every
    position, then the sparse loops over the column budget (sinks and window forced), timed per loop with
    HIP events (separate from the prefill step above)."""
    B, T, H, d = gs.k_hat.shape
    c = w.col_budget
    g = torch.Generator(device="cuda").manual_seed(11)
    q = torch.randn(B, H, d, device="cuda", generator=g).to(torch.bfloat16)
    o = torch.zeros(B, H, d, dtype=torch.float32, device="cuda")
    reps = 20

    def timed(fn):
        for _ in range(3):
            out = fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            out = fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps * 1e3, out

    # outputs and workspaces allocated once: the timed calls allocate nothing
    out_d = (torch.empty(B, H, c, dtype=torch.int32, device="cuda"), torch.empty(B, H, device="cuda"),
             torch.empty(B, H, d, device="cuda"))
    out_s = tuple(torch.empty_like(t) for t in out_d)
    ws_d = fl.decode_ws(gs.k_hat, None, c)
    us_dense, (cols, mass, sub) = timed(lambda: fl.decode_step(q, gs.k_hat, gs.v_hat, None, None, None, o, c,
                                                               n_sink=w.n_sink, window=w.window, out=out_d,
                                                               ws=ws_d))
    ws_s = fl.decode_ws(gs.k_hat, cols, c)
    us_sparse, _ = timed(lambda: fl.decode_step(q, gs.k_hat, gs.v_hat, cols, mass, sub, o, c,
                                                n_sink=w.n_sink, window=w.window, out=out_s, ws=ws_s))
    nb_dense = decode_work(B, T, H, d, 0, c)
    nb_sparse = decode_work(B, T, H, d, c, c)
    log(f"[bench] decode: dense loop {us_dense:.1f} us ({nb_dense / us_dense / 1e3:.0f} GB/s), "
        f"sparse loop {us_sparse:.1f} us ({nb_sparse / us_sparse / 1e3:.0f} GB/s)")
    return {"workload": f"{w.name} decode position {T - 1}", "columns_dense": T, "columns_sparse": c,
            "dense_loop_us": round(us_dense, 2), "sparse_loop_us": round(us_sparse, 2),
            "dense_alg_MB": round(nb_dense / 1e6, 2), "sparse_alg_MB": round(nb_sparse / 1e6, 2),
            "dense_GBps": round(nb_dense / us_dense / 1e3, 1), "sparse_GBps": round(nb_sparse / us_sparse / 1e3, 1),
            "timing": f"HIP events, mean of {reps} calls (two launches each, nothing allocated)"}


def prune_work(rows, cols, n_sink, H, d):
    """Algorithmic work of one fl_prune_columns call: bytes = the list entries' K rows, the updated rows'
    queries and lse_ref, the keys written, the lists read and written; fp64 flops = 2 d per (updated row i,
    list entry j >= sinks) pair with i >= j (one dot product each; the exponentials are not counted)."""
    B, k = rows.shape
    c_list = cols.shape[2]
    ns = min(n_sink, c_list)
    nb = B * H * (c_list - ns) * (d * 2 + 4) + B * k * H * (d * 2 + 4) + B * H * c_list * 4 * 2
    pairs = 0
    for b in range(B):
        rb = np.sort(rows[b])
        for h in range(H):
            js = cols[b, h, ns:]
            pairs += int(np.sum(len(rb) - np.searchsorted(rb, js, side="left")))
    return nb, 2.0 * d * pairs


def prune_bench(w, gs, q_last, fl, torch):
    """The list pruning after the last sparse loop of the step, to half the ranked entries (one step of a
    decaying budget), timed with HIP events (not part of the step: the workload's budget is constant)."""
    t_next = w.top_cols // 2
    reps = 10
    for _ in range(2):
        fl.prune_columns(q_last, gs.k_hat, gs.cand, gs.cols, gs.lse, w.n_sink, t_next)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        fl.prune_columns(q_last, gs.k_hat, gs.cand, gs.cols, gs.lse, w.n_sink, t_next)
    e1.record()
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) / reps * 1e3
    B, N, H, d = gs.k_hat.shape
    nb, nf = prune_work(gs.cand.cpu().numpy(), gs.cols.cpu().numpy(), w.n_sink, H, d)
    achieved = nf / (us * 1e-6) / 1e12
    log(f"[bench] prune: {us:.1f} us, {achieved:.2f} fp64 TFLOP/s")
    return {"workload": f"{w.name} list {gs.cols.shape[2]} -> {min(w.n_sink, gs.cols.shape[2]) + t_next} entries "
                        f"over {gs.cand.shape[1]} updated rows", "us": round(us, 2),
            "bound": "alu", "achieved": round(achieved, 2), "peak": FP64_VECTOR_TFLOPS, "unit": "TFLOP/s (fp64)",
            "frac": round(achieved / FP64_VECTOR_TFLOPS, 4), "alg_MB": round(nb / 1e6, 2),
            "alg_GF": round(nf / 1e9, 3), "timing": f"HIP events, mean of {reps} calls (two launches each)"}


def tail_bench(w, gs, k_last, fl, torch, tail=64):
    """The recent-token bf16 tail (Appendix E, 64 positions) applied to the cache after the step's last
    loop, for its active rows; timed with HIP events (the workload itself runs without a tail)."""
    reps = 20
    cache = gs.k_hat.clone()
    for _ in range(2):
        fl.kv_keep_recent(k_last, gs.cand, tail, cache=cache)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        fl.kv_keep_recent(k_last, gs.cand, tail, cache=cache)
    e1.record()
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) / reps * 1e3
    B, N, H, d = cache.shape
    idx = gs.cand.cpu().numpy()
    n_tail = int(np.sum(idx >= N - tail))
    nb = n_tail * H * d * 2 * 2 + B * min(idx.shape[1], tail) * 4
    return {"workload": f"{w.name} tail {tail}: {n_tail} active tail rows of one tensor", "us": round(us, 2),
            "alg_KB": round(nb / 1e3, 2), "timing": f"HIP events, mean of {reps} calls (launch-bound)"}


if __name__ == "__main__":
    main()
