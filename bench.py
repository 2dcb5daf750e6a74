"""Benchmark of the block-sparse linear layer on one MI355X.

Workload (default): DeiT-B fc1 at batch 256 -- X bf16 [50432 x 768] ~ N(0,1),
W bf16 [3072 x 768] ~ N(0, 0.02), bias, 32x32 blocks, 50% of the blocks kept
uniformly at random (exactly 1152 of 2304), no GELU.

A step is one lpv_bsr_linear call over the whole batch (X staging, kept-block
contraction, epilogue); the weight is packed once before timing (weights are
static at inference) and the pack is timed on its own.  Before any timing the
GPU runs block-sparse and dense launches alternately for a fixed time, so the
clock has settled whatever --warmup is; then W untimed and K timed steps give
`value`.  The speed-up over the dense path (lpv_dense_linear, same shape, same
epilogue) comes from interleaved rounds (block-sparse, dense, block-sparse,
...), so both see the same clock; the GPU clock during those rounds is sampled
and reported.  Prints ONE JSON line on stdout; details go to stderr.

    python bench.py [--steps K] [--warmup W] [--gpus 1] [--no-cpu] [--gelu]
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16/fp16 matrix-core peak (published)
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E (published)
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "bsr_linear_fc1_hbm_traffic.json")
CLOCK_FILE = os.path.join(ROOT, "profiles", "bsr_linear_fc1_gpu_clock.md")
STATS_FILE = os.path.join(ROOT, "profiles", "bsr_linear_deit_b_fc1_bf16_kernel_stats.md")
STATS_FILE_BACKWARD = os.path.join(ROOT, "profiles", "backward_delta_deit_b_fc1_bf16_kernel_stats.md")
KERNEL_SOURCES = ("paper_2407_02068_amd/csrc/linear.hip", "paper_2407_02068_amd/csrc/lpv_device.h",
                  "paper_2407_02068_amd/csrc/lpv_internal.h")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_source_hash():
    h = hashlib.sha256()
    for p in KERNEL_SOURCES:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic():
    """HBM bytes per launch of the block-sparse kernel from the committed
    rocprofv3 counter summary, if it was taken on the current kernel source."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("kernel_source_sha256_16") != kernel_source_hash():
        return None
    return t.get("hbm_bytes_per_launch")


def algorithmic_bytes(M, N, K, nnzb, b_r, b_c, kused_cols, es=2):
    """X (used columns only) + Y + kept W + bias + BSR indices, each once."""
    return es * (M * kused_cols + M * N + nnzb * b_r * b_c + N) + 4 * (N // b_r + 1 + nnzb)


# bf16, no GELU, block-sparse with 32-wide blocks / dense; 12 groups of 256
# outputs, so the pair's last k-step is multiplied after its barrier
SPARSE_KERNEL = "k_linear16<2, false, false, false, false, true>"
DENSE_KERNEL = "k_linear16<2, false, true, false, false, true>"
CALIB_BYTES = 1 << 30                        # the calibration copy reads and writes this much


def write_traffic(fetch_csv, write_csv, command):
    """HBM bytes per launch of the block-sparse kernel from two rocprofv3
    counter runs of ``--profile-pass`` (FETCH_SIZE, then WRITE_SIZE, KiB per
    dispatch), each scaled by what the same counter reads for the 1 GiB
    device-to-device copy of that pass; written next to the other profiles."""
    import csv

    def per_dispatch(path, counter):
        rows = [r for r in csv.DictReader(open(path)) if r["Counter_Name"] == counter]
        kern = [float(r["Counter_Value"]) for r in rows if SPARSE_KERNEL in r["Kernel_Name"]]
        copies = [float(r["Counter_Value"]) for r in rows if "copyBuffer" in r["Kernel_Name"]]
        if not kern or not copies:
            raise SystemExit("%s: no %s rows for the kernel or the copy" % (path, counter))
        return sum(kern) / len(kern), max(copies)

    fk, fc = per_dispatch(fetch_csv, "FETCH_SIZE")
    wk, wc = per_dispatch(write_csv, "WRITE_SIZE")
    f_scale = CALIB_BYTES / (fc * 1024.0)
    w_scale = CALIB_BYTES / (wc * 1024.0)
    out = {"kernel": "k_linear16 (lpv_bsr_linear), bf16, no GELU",
           "workload": "DeiT-B fc1 batch 256, 32x32 blocks, 50% block sparsity",
           "kernel_source_sha256_16": kernel_source_hash(),
           "fetch_kib_per_dispatch": round(fk, 1), "write_kib_per_dispatch": round(wk, 1),
           "copy_1GiB_fetch_kib": round(fc, 1), "copy_1GiB_write_kib": round(wc, 1),
           "fetch_scale": round(f_scale, 4), "write_scale": round(w_scale, 4),
           "hbm_read_bytes_per_launch": int(fk * 1024 * f_scale),
           "hbm_write_bytes_per_launch": int(wk * 1024 * w_scale),
           "hbm_bytes_per_launch": int(fk * 1024 * f_scale + wk * 1024 * w_scale),
           "counter_runs": [
               "rocprofv3 --pmc FETCH_SIZE -d gpurun_out/pmc_fetch -o fetch --output-format csv "
               "-- python bench.py --profile-pass",
               "rocprofv3 --pmc WRITE_SIZE -d gpurun_out/pmc_write -o write --output-format csv "
               "-- python bench.py --profile-pass"],
           "command": command}
    with open(TRAFFIC_FILE, "w") as f:
        json.dump(out, f, indent=1)
        f.write("\n")
    print(json.dumps(out, indent=1))


def kernel_label(name):
    """A short name for a kernel of the rocprofv3 statistics."""
    import re
    m = re.search(r"k_linear16<(\d), (true|false), (true|false), (true|false), (true|false), (true|false)>",
                  name)
    if m:
        return "k_linear16 %s %s%s%s%s%s (%s)" % (
            {"2": "bf16", "1": "fp16"}[m.group(1)],
            "dense" if m.group(3) == "true" else "block-sparse",
            " + GELU" if m.group(2) == "true" else "", ", K tail" if m.group(4) == "true" else "",
            ", 16-column halves" if m.group(5) == "true" else "",
            ", DMA before the last k-step" if m.group(6) == "false" else "",
            "lpv_dense_linear" if m.group(3) == "true" else "lpv_bsr_linear")
    labels = (("k_block_scores_lds<2, true", "k_block_scores_lds, Taylor (lpv_delta_curve)"),
              ("k_block_scores_lds<2, false", "k_block_scores_lds, sum of squares (lpv_mask_topk)"),
              ("k_block_scores<2, true", "k_block_scores, Taylor (lpv_delta_curve)"),
              ("k_block_scores<2, false", "k_block_scores, sum of squares (lpv_mask_topk)"),
              ("k_block_scores", "k_block_scores (lpv_mask_topk)"),
              ("k_delta_dots", "k_delta_dots (lpv_delta_curve)"),
              ("k_rank", "k_rank (lpv_delta_curve)"),
              ("k_delta_steps", "k_delta_steps (lpv_delta_curve)"),
              ("k_delta_finish", "k_delta_finish (lpv_delta_curve)"),
              ("k_mask_topk", "k_mask_topk (lpv_mask_topk)"),
              ("k_attention", "k_attention (lpv_attention)"),
              ("k_add_layernorm", "k_add_layernorm (lpv_add_layernorm)"),
              ("FillFunctor", "torch fill (cache flush between cold launches)"),
              ("copyBuffer", "HIP runtime copy"),
              ("direct_copy_kernel", "torch copy"))
    for key, label in labels:
        if key in name:
            return label
    for key in ("k_pack_plan", "k_pack_compact", "k_sched_fill", "k_stream_fill", "k_walk_fill"):
        if key in name:
            return key + " (lpv_bsr_pack)"
    for key, api in (("k_gradw_tiles", "lpv_bsr_grad_w"), ("k_gradw_reduce", "lpv_bsr_grad_w"),
                     ("k_gradw_plain", "lpv_bsr_grad_w"), ("k_bias_partial", "lpv_bias_grad"),
                     ("k_bias_reduce", "lpv_bias_grad"), ("k_transpose_blocks", "lpv_bsr_transpose"),
                     ("k_unpack", "lpv_bsr_unpack")):
        if key in name:
            return "%s (%s)" % (key, api)
    if name.startswith("Cijk") or name.startswith("Custom_Cijk"):
        return "hipBLASLt " + name.split("_UserArgs")[0][:48]
    return name.split("(")[0][:72]


STATS_RUN = ("rocprofv3 --kernel-trace --stats -d gpurun_out/prof_bench -o bench --output-format csv "
             "-- python bench.py --steps 20 --warmup 5 2> gpurun_out/prof_bench.log")
STATS_RUN_BACKWARD = ("rocprofv3 --kernel-trace --stats -d gpurun_out/prof_bw -o bw --output-format "
                      "csv -- python bench.py --no-cpu --no-flushed --no-power --no-stack --no-sweep")


def timed_window(trace_csv, bench_log):
    """Durations (us) of the block-sparse launches inside bench.py's timed
    steps, from the rocprofv3 kernel trace: the run's stderr names the window
    (``STATS_WINDOW first=F steps=K``: the K launches after the first F of the
    headline kernel), and the trace lists every dispatch with its start and
    end time."""
    import csv
    import re
    m = None
    for line in open(bench_log):
        m = re.search(r"STATS_WINDOW first=(\d+) steps=(\d+)", line) or m
    if m is None:
        raise SystemExit("%s: no STATS_WINDOW line" % bench_log)
    first, steps = int(m.group(1)), int(m.group(2))
    rows = [r for r in csv.DictReader(open(trace_csv)) if SPARSE_KERNEL in r["Kernel_Name"]]
    rows.sort(key=lambda r: int(r["Start_Timestamp"]))
    win = rows[first:first + steps]
    if len(win) != steps:
        raise SystemExit("%s: %d launches of the kernel, window %d+%d" % (trace_csv, len(rows),
                                                                         first, steps))
    return [(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3 for r in win]


def write_stats(stats_csv, command, backward=False, trace_csv=None, bench_log=None):
    """The rocprofv3 --kernel-trace --stats summary of a bench.py run as a
    short table next to the other profiles: the run the driver makes (forward,
    sweep, encoder, ...), or (backward) the run with the backward and
    delta-curve legs.  For the forward run the block-sparse kernel's launches
    inside the timed steps are averaged on their own (the stats table mixes
    every shape the run launches the same kernel at)."""
    import csv
    rows = list(csv.DictReader(open(stats_csv)))
    text = ["# rocprofv3 kernel statistics: DeiT-B fc1 (X 50432 x 768 -> 3072), bf16, 32x32 blocks, "
            "50%% block sparsity, %s" % ("forward, backward and delta curve" if backward else
                                         "the default bench.py run"), "",
            "Profiled run, then this summary (from the repository root on one MI355X):", "", "```",
            STATS_RUN_BACKWARD if backward else STATS_RUN, command, "```", ""]
    if not backward and trace_csv:
        win = timed_window(trace_csv, bench_log)
        avg_us = sum(win) / len(win)
        text += ["Block-sparse kernel inside the %d timed steps (from the kernel trace): mean "
                 "%.1f us, min %.1f us, max %.1f us: %.0f TFLOP/s on the 118.98 GFLOP of kept "
                 "work (%.1f%% of the 2.5 PFLOP/s bf16 matrix-core peak).  `bench.py` times the "
                 "same launches with HIP events on their stream and reports that mean as "
                 "`roofline.achieved`." % (len(win), avg_us, min(win), max(win),
                                           118.98e9 / (avg_us * 1e-6) / 1e12,
                                           118.98e9 / (avg_us * 1e-6) / 1e12 / 25.0), ""]
    text += ["| kernel | calls | avg us | min us | max us | % of GPU time |",
             "|---|---:|---:|---:|---:|---:|"]
    for r in rows:
        text.append("| %s | %s | %.1f | %.1f | %.1f | %.2f |" % (
            kernel_label(r["Name"]), r["Calls"], float(r["AverageNs"]) / 1e3,
            float(r["MinNs"]) / 1e3, float(r["MaxNs"]) / 1e3, float(r["Percentage"])))
    if backward:
        text += ["", "The block-sparse k_linear16 row counts the forward launches and the dX "
                 "launches (the same kernel on the transposed handle).  dW is k_gradw_tiles + "
                 "k_gradw_reduce, db k_bias_partial + k_bias_reduce, the delta curve "
                 "k_block_scores_lds + k_rank + k_delta_dots + "
                 "k_delta_steps + k_delta_finish; Cijk_Ailk is hipBLASLt's dense G^T X "
                 "reference, Custom_Cijk_Alik its dense forward."]
    else:
        text += ["", "Rows of one kernel name cover every shape the run launches it at (the "
                 "headline, the sweep, the encoder's linears).  The encoder leg (12-block DeiT-B, "
                 "batch 256: chains with block-sparse and with dense linears, attention and layer "
                 "norm timed alone, the power windows) accounts for the k_attention and "
                 "k_add_layernorm rows.  The hipBLASLt rows (Cijk) are "
                 "`torch.addmm` at the headline shape, a check on the dense path."]
    with open(STATS_FILE_BACKWARD if backward else STATS_FILE, "w") as f:
        f.write("\n".join(text) + "\n")
    print("\n".join(text))


COUNTER_FILE = os.path.join(ROOT, "profiles", "bsr_linear_fc1_counters.md")
COUNTER_PASSES = (
    "SQ_WAVE_CYCLES SQ_BUSY_CYCLES SQ_WAIT_ANY SQ_WAIT_INST_ANY SQ_ACTIVE_INST_ANY "
    "SQ_ACTIVE_INST_LDS SQ_INSTS_LDS SQ_LDS_BANK_CONFLICT",
    "SQ_VALU_MFMA_BUSY_CYCLES SQ_WAIT_INST_LDS SQ_LDS_IDX_ACTIVE SQ_INSTS_MFMA SQ_INSTS_SALU "
    "SQ_INSTS_VALU SQ_INSTS_VMEM SQ_WAVES GRBM_GUI_ACTIVE",
    "TCC_HIT_sum TCC_MISS_sum GRBM_GUI_ACTIVE")


def write_counters(csvs, command):
    """Derived figures of the block-sparse (and dense) kernel from three
    rocprofv3 --pmc passes of ``--profile-pass`` (COUNTER_PASSES, one CSV per
    pass): matrix-core busy share, wave-cycle shares waiting / issuing, LDS
    activity and bank conflicts, L2 hit rate.  Counter values are summed over
    the device by rocprofv3; GRBM_GUI_ACTIVE is summed over the XCDs."""
    import csv
    vals = {}
    n_xcc = 8
    for path in csvs:
        agents = os.path.join(os.path.dirname(path),
                              os.path.basename(path).replace("counter_collection", "agent_info"))
        try:
            n_xcc = max(int(a.get("Num_Xcc") or 0) for a in csv.DictReader(open(agents))) or n_xcc
        except (OSError, ValueError):
            pass
        for r in csv.DictReader(open(path)):
            for key, tag in ((SPARSE_KERNEL, "bsr"), (DENSE_KERNEL, "dense")):
                if key in r["Kernel_Name"]:
                    vals.setdefault((tag, r["Counter_Name"]), []).append(float(r["Counter_Value"]))
    avg = {k: sum(v) / len(v) for k, v in vals.items()}

    def derived(tag):
        g = lambda c: avg.get((tag, c))
        cyc = g("GRBM_GUI_ACTIVE") / n_xcc  # cycles of the dispatch, per XCD
        cus, simds = 256, 1024
        out = [("dispatch cycles (GRBM_GUI_ACTIVE per XCD)", "%.0f" % cyc),
               ("matrix cores busy (SQ_VALU_MFMA_BUSY_CYCLES / (cycles x %d SIMDs))" % simds,
                "%.1f%%" % (100 * g("SQ_VALU_MFMA_BUSY_CYCLES") / (cyc * simds))),
               ("wave cycles waiting on anything (SQ_WAIT_ANY / SQ_WAVE_CYCLES)",
                "%.1f%%" % (100 * g("SQ_WAIT_ANY") / g("SQ_WAVE_CYCLES"))),
               ("wave cycles waiting on a dependency, s_waitcnt (SQ_WAIT_INST_ANY / SQ_WAVE_CYCLES)",
                "%.1f%%" % (100 * g("SQ_WAIT_INST_ANY") / g("SQ_WAVE_CYCLES"))),
               ("wave cycles issuing (SQ_ACTIVE_INST_ANY / SQ_WAVE_CYCLES)",
                "%.1f%%" % (100 * g("SQ_ACTIVE_INST_ANY") / g("SQ_WAVE_CYCLES"))),
               ("LDS busy (SQ_LDS_IDX_ACTIVE / (cycles x %d CUs))" % cus,
                "%.1f%%" % (100 * g("SQ_LDS_IDX_ACTIVE") / (cyc * cus))),
               ("LDS bank-conflict cycles / LDS active cycles",
                "%.2f%%" % (100 * g("SQ_LDS_BANK_CONFLICT") / g("SQ_LDS_IDX_ACTIVE"))),
               ("instructions per wave: MFMA / SALU / VALU / LDS / VMEM", "%.0f / %.0f / %.0f / %.0f / %.0f" % (
                   g("SQ_INSTS_MFMA") / g("SQ_WAVES"), g("SQ_INSTS_SALU") / g("SQ_WAVES"),
                   g("SQ_INSTS_VALU") / g("SQ_WAVES"), g("SQ_INSTS_LDS") / g("SQ_WAVES"),
                   g("SQ_INSTS_VMEM") / g("SQ_WAVES"))),
               ("L2 hit rate (TCC_HIT / (TCC_HIT + TCC_MISS))",
                "%.1f%%" % (100 * g("TCC_HIT_sum") / (g("TCC_HIT_sum") + g("TCC_MISS_sum"))))]
        return out

    text = ["# rocprofv3 counters: DeiT-B fc1 (X 50432 x 768 -> 3072), bf16, 32x32 blocks, "
            "50% block sparsity", "",
            "Three counter passes over `bench.py --profile-pass` (three launches of each path), "
            "then this summary (from the repository root on one MI355X):", "", "```"]
    for i, c in enumerate(COUNTER_PASSES):
        text.append("rocprofv3 --pmc %s -d gpurun_out/pmc_c%d -o c%d --output-format csv -- "
                    "python bench.py --profile-pass" % (c, i + 1, i + 1))
    text += [command, "```", "",
             "| figure | k_linear16 block-sparse | k_linear16 dense |", "|---|---:|---:|"]
    for (name, a), (_, b) in zip(derived("bsr"), derived("dense")):
        text.append("| %s | %s | %s |" % (name, a, b))
    text += ["", "Counter values are per dispatch, averaged over the three launches; SQ counters "
             "are summed over the device, GRBM_GUI_ACTIVE over the %d XCDs." % n_xcc]
    with open(COUNTER_FILE, "w") as f:
        f.write("\n".join(text) + "\n")
    print("\n".join(text))


def write_clock(csv_path, command):
    """The GPU clock achieved during each kernel of a ``--profile-pass`` run:
    GRBM_GUI_ACTIVE cycles of the dispatch (rocprofv3 sums the counter over
    the XCDs, so per XCD: divided by their number, from the agent record) over
    its duration (counter timestamps, ns); written next to the other profiles."""
    import csv
    agents = os.path.join(os.path.dirname(csv_path),
                          os.path.basename(csv_path).replace("counter_collection", "agent_info"))
    n_xcc = max(int(a.get("Num_Xcc") or 0) for a in csv.DictReader(open(agents)))
    rows = [r for r in csv.DictReader(open(csv_path)) if r["Counter_Name"] == "GRBM_GUI_ACTIVE"]
    lines = []
    for name, key in (("k_linear16 bf16 block-sparse (lpv_bsr_linear)", SPARSE_KERNEL),
                      ("k_linear16 bf16 dense (lpv_dense_linear)", DENSE_KERNEL)):
        sel = [r for r in rows if key in r["Kernel_Name"]]
        if not sel:
            raise SystemExit("%s: no GRBM_GUI_ACTIVE rows for %s" % (csv_path, key))
        for r in sel:
            ns = float(r["End_Timestamp"]) - float(r["Start_Timestamp"])
            cyc = float(r["Counter_Value"])
            lines.append("| %s | %s | %.1f | %.0f | %.0f |" % (name, r["Dispatch_Id"], ns / 1e3, cyc,
                                                               cyc / n_xcc / ns * 1e3))
    text = ["# GPU clock during the kernels: DeiT-B fc1 (X 50432 x 768 -> 3072), bf16, "
            "32x32 blocks, 50% block sparsity", "",
            "Counter run (from the repository root on one MI355X), then this summary:", "", "```",
            "rocprofv3 --pmc GRBM_GUI_ACTIVE -d gpurun_out/pmc_clock -o clock --output-format csv "
            "-- python bench.py --profile-pass", command, "```", "",
            "Each row is one dispatch of the profile pass (three launches of each path, "
            "serialised by the counter collection): the active cycles, summed over the "
            "%d XCDs, divided by their number and by the dispatch's duration." % n_xcc, "",
            "| kernel | dispatch | us | GRBM_GUI_ACTIVE cycles | MHz |",
            "|---|---:|---:|---:|---:|"] + lines
    with open(CLOCK_FILE, "w") as f:
        f.write("\n".join(text) + "\n")
    print("\n".join(text))


def time_launches(fn, steps, warmup):
    import torch
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        starts[i].record()
        fn()
        ends[i].record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = sorted(s.elapsed_time(e) for s, e in zip(starts, ends))
    return wall, ms


def prewarm(fns, seconds):
    """Run the launch functions in turn until ``seconds`` have passed (the GPU
    clock and power state settle); returns the number of calls of each."""
    import torch
    n = [0] * len(fns)
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < seconds:
        for i, fn in enumerate(fns):
            for _ in range(20):
                fn()
            n[i] += 20
        torch.cuda.synchronize()
    return n


def interleaved(fa, fb, rounds, per_round):
    """Rounds of ``per_round`` launches of fa, then of fb, each launch between
    its own pair of events on the launching stream; returns (a_ms, b_ms), the
    per-launch times of each, so both sides are measured on the same clock."""
    import torch
    a, b = [], []
    for _ in range(rounds):
        for fn, out in ((fa, a), (fb, b)):
            ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                  for _ in range(per_round)]
            for e0, e1 in ev:
                e0.record()
                fn()
                e1.record()
            torch.cuda.synchronize()
            out.extend(e0.elapsed_time(e1) for e0, e1 in ev)
    return a, b


class ClockSampler:
    """The GPU's graphics clock (MHz) sampled every 10 ms through amd-smi while
    a block runs (``with ClockSampler() as c: ...``; then c.summary())."""

    def __init__(self):
        self.samples, self.error, self._stop, self._th, self._h = [], None, None, None, None

    def _read(self):
        import amdsmi
        v = amdsmi.amdsmi_get_clock_info(self._h, amdsmi.AmdSmiClkType.GFX).get("clk")
        return float(v) if isinstance(v, (int, float)) and v > 0 else None

    def __enter__(self):
        import threading
        try:
            import amdsmi
            amdsmi.amdsmi_init()
            self._h = _smi_handle(amdsmi)
            if self._h is None:
                raise RuntimeError("no amd-smi device matches the benchmarked GPU")
            self._read()
        except Exception as e:  # no amd-smi access: reported as such
            self.error = "amdsmi: %s" % e
            return self
        self._stop = threading.Event()

        def poll():
            while not self._stop.is_set():
                try:
                    v = self._read()
                except Exception:
                    v = None
                if v is not None:
                    self.samples.append(v)
                self._stop.wait(0.01)
        self._th = threading.Thread(target=poll)
        self._th.start()
        return self

    def __exit__(self, *a):
        if self._th is not None:
            self._stop.set()
            self._th.join()
        try:
            import amdsmi
            amdsmi.amdsmi_shut_down()
        except Exception:
            pass

    def summary(self):
        if not self.samples:
            return {"unavailable": self.error or "no samples"}
        v = sorted(self.samples)
        return {"median_MHz": v[len(v) // 2], "min_MHz": v[0], "max_MHz": v[-1],
                "samples": len(v), "source": "amd-smi GFX clock every 10 ms"}


def _smi_handle(amdsmi):
    """The amd-smi handle of the GPU torch uses (device 0)."""
    import torch
    handles = amdsmi.amdsmi_get_processor_handles()
    if len(handles) == 1:
        return handles[0]
    p = torch.cuda.get_device_properties(0)
    want = (getattr(p, "pci_domain_id", None), getattr(p, "pci_bus_id", None),
            getattr(p, "pci_device_id", None))
    for c in handles:
        dom, bus, rest = amdsmi.amdsmi_get_gpu_device_bdf(c).split(":")
        if (int(dom, 16), int(bus, 16), int(rest.split(".")[0], 16)) == want:
            return c
    return None


def time_flushed(fn, steps, flush_buf):
    """Each launch timed alone after writing flush_buf (larger than L2 and the
    256 MB MALL together), so that X, W and Y start outside the caches."""
    import torch
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
    fn()
    for i in range(steps):
        flush_buf.fill_(i & 0x7f)
        starts[i].record()
        fn()
        ends[i].record()
    torch.cuda.synchronize()
    return sorted(s.elapsed_time(e) for s, e in zip(starts, ends))


def time_backward(w, h, W, X, steps, tt, to_dev):
    """The layer's backward at the same workload (finetuning): dX = G W~ by the
    forward kernel on the transposed handle, dW = G^T X on the kept blocks,
    db = the column sums of G; G is a seeded N(0, 1) gradient.  Dense
    references: the library's dense kernel for dX (on W~^T) and hipBLASLt's
    full G^T X for dW."""
    import torch

    import workloads as wl
    from paper_2407_02068_amd import lpv
    G = to_dev(wl.grad_output(4, 0, w.M, w.N, w.dtype))
    ht = lpv.bsr_transpose(h)
    dX = torch.empty((w.M, w.K), dtype=tt, device="cuda")
    dXd = torch.empty_like(dX)
    dW = torch.empty((w.nnzb, w.b_r, w.b_c), dtype=tt, device="cuda")
    db = torch.empty(w.N, dtype=tt, device="cuda")
    WT = lpv.bsr_unpack(h).t().contiguous()        # W~^T, K x N, for the dense dX
    Gt = G.t().contiguous()                        # for hipBLASLt's G^T X
    steps = max(10, steps // 2)
    _, xms = time_launches(lambda: lpv.bsr_linear(ht, G, None, dX), steps, 10)
    _, xdms = time_launches(lambda: lpv.dense_linear(WT, G, None, dXd), steps, 10)
    _, wms = time_launches(lambda: lpv.grad_w(h, G, X, dW), steps, 10)
    _, wbms = time_launches(lambda: torch.mm(Gt, X), steps, 5)
    _, bms = time_launches(lambda: lpv.bias_grad_noalloc(G, db), steps, 10)
    _, bams = time_launches(lambda: lpv.bias_grad(G, db), steps, 10)
    ht.close()
    kept = w.kept_flops()
    avg = lambda ms: sum(ms) / len(ms)
    return {"dx_ms": round(avg(xms), 5), "dx_dense_ms": round(avg(xdms), 5),
            "dx_tflops": round(kept / (avg(xms) * 1e-3) / 1e12, 1),
            "dw_ms": round(avg(wms), 5), "dw_tflops": round(kept / (avg(wms) * 1e-3) / 1e12, 1),
            "dw_frac_of_peak": round(kept / (avg(wms) * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
            "dw_hipblaslt_dense_ms": round(avg(wbms), 5), "db_ms": round(avg(bms), 5),
            "db_stream_alloc_ms": round(avg(bams), 5),
            "note": "event averages; dW includes its chunk reduction (the workspace is the "
                    "handle's, allocated once); db by the call that allocates nothing, "
                    "db_stream_alloc_ms by the one with a stream-ordered workspace; "
                    "G seeded N(0, 1)"}


def time_delta_curve(w, W, steps, to_dev):
    """The delta curve of the same layer (Sec. 3.3): 64 seeded per-sample
    gradients of the weight, the 21 sparsity points 0, 5, .., 100.  The pass
    over the per-sample gradients bounds it: reported against HBM."""
    import numpy as np
    import torch

    import workloads as wl
    from paper_2407_02068_amd import lpv
    n_s = 64
    g = wl.rng(4, 0, wl.T_GRAD)
    grad = to_dev(wl.quantize(g.normal(0, 1e-3, (w.N, w.K)).astype(np.float32), w.dtype))
    S = torch.empty((n_s, w.N, w.K), dtype=W.dtype, device="cuda")
    for i in range(n_s):  # generated per sample to bound host memory
        S[i] = to_dev(wl.quantize(g.normal(0, 1e-2, (w.N, w.K)).astype(np.float32), w.dtype))
    pcts = list(range(0, 101, 5))
    out = torch.empty(len(pcts), dtype=torch.float64, device="cuda")
    ws = torch.empty(lpv.delta_curve_workspace_size(w.N, w.K, w.b_r, w.b_c, n_s, len(pcts)),
                     dtype=torch.uint8, device="cuda")
    _, ms = time_launches(lambda: lpv.delta_curve(W, grad, S, w.b_r, w.b_c, 1e-4, pcts, out,
                                                  workspace=ws), max(10, steps // 2), 5)
    avg = sum(ms) / len(ms)
    alg = (n_s + 2) * w.N * w.K * 2  # every vector (samples, grad, W) read once
    return {"ms": round(avg, 5), "n_samples": n_s, "points": len(pcts),
            "hbm_alg_bytes": alg, "hbm_achieved_GBs": round(alg / (avg * 1e-3) / 1e9, 1),
            "hbm_frac": round(alg / (avg * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
            "note": "event average; block scores, ranking, float64 block dot products and the "
                    "ratio steps, in a caller-owned workspace; per-sample gradients seeded "
                    "N(0, 1e-2)"}


def measure_power(sparse, dense, seconds=2.0, settle=0.6, pairs=3, unit="launch"):
    """Board power in the manner of the paper's measurement (the power meter
    averaged over a period, idle subtracted): amd-smi's socket power sampled
    every 20 ms over windows of idle, a loop of block-sparse calls and a loop
    of dense calls -- idle, one block-sparse window that only brings the board
    from idle to load (discarded: the meter's average lags), then ``pairs`` x
    (block-sparse, dense), then idle -- the samples of each window's first
    ``settle`` seconds dropped.  Energy
    per call above idle = (window power - idle) x time per call, per window;
    reported as the mean over the windows with their spread.  (amd-smi's
    energy counter lags the windows on this machine, so it is not used.)"""
    import threading

    import torch
    try:
        import amdsmi
        amdsmi.amdsmi_init()
    except Exception as e:  # no amd-smi access on this machine
        return {"unavailable": "amdsmi: %s" % e}
    try:
        h = _smi_handle(amdsmi)
        if h is None:
            return {"unavailable": "no amd-smi device matches the benchmarked GPU"}

        def socket_w():
            v = amdsmi.amdsmi_get_power_info(h).get("current_socket_power")
            return float(v) if isinstance(v, (int, float)) and v > 0 else None

        def window(fn):
            samples, stop = [], threading.Event()
            t0 = time.perf_counter()

            def poll():
                while not stop.is_set():
                    v = socket_w()
                    if v is not None and time.perf_counter() - t0 >= settle:
                        samples.append(v)
                    stop.wait(0.02)
            th = threading.Thread(target=poll)
            torch.cuda.synchronize()
            th.start()
            n = 0
            if fn is None:
                time.sleep(seconds)
            else:
                while time.perf_counter() - t0 < seconds:
                    for _ in range(10):
                        fn()
                    n += 10
                    torch.cuda.synchronize()
            el = time.perf_counter() - t0
            stop.set()
            th.join()
            if not samples:
                raise RuntimeError("no power samples")
            return sum(samples) / len(samples), n, el

        runs = {"idle": [], "bsr": [], "dense": [], "ramp": []}
        order = [("idle", None), ("ramp", sparse)] + [("bsr", sparse), ("dense", dense)] * pairs \
            + [("idle", None)]
        for kind, fn in order:
            runs[kind].append(window(fn))
        del runs["ramp"]
        idle = sum(r[0] for r in runs["idle"]) / len(runs["idle"])
        # energy per call above idle, one value per window (mJ)
        e = {k: [(wt - idle) * el / n * 1e3 for wt, n, el in runs[k]] for k in ("bsr", "dense")}
        watts = {k: sum(r[0] for r in v) / len(v) for k, v in runs.items()}
        mean = lambda v: sum(v) / len(v)
        red = [100.0 * (1.0 - b / d) for b, d in zip(e["bsr"], e["dense"]) if d > 0]
        return {"idle_W": round(idle, 1), "bsr_W": round(watts["bsr"], 1),
                "dense_W": round(watts["dense"], 1),
                "bsr_mJ_per_%s_above_idle" % unit: round(mean(e["bsr"]), 2),
                "dense_mJ_per_%s_above_idle" % unit: round(mean(e["dense"]), 2),
                "bsr_mJ_windows": [round(v, 2) for v in e["bsr"]],
                "dense_mJ_windows": [round(v, 2) for v in e["dense"]],
                "energy_reduction_pct": round(100.0 * (1.0 - mean(e["bsr"]) / mean(e["dense"])), 1)
                if mean(e["dense"]) > 0 else None,
                "energy_reduction_pct_min_max": [round(min(red), 1), round(max(red), 1)] if red else None,
                "method": "amd-smi current socket power every 20 ms over %.1f s windows (idle, a "
                          "discarded block-sparse ramp window, %d x (block-sparse, dense), idle; "
                          "first %.1f s of each dropped); "
                          "energy per %s = (window power - idle) x time per %s"
                          % (seconds, pairs, settle, unit, unit)}
    except Exception as e:
        return {"unavailable": "amdsmi: %s" % e}
    finally:
        try:
            amdsmi.amdsmi_shut_down()
        except Exception:
            pass


def time_stack(steps, to_dev, power=True):
    """The DeiT-B encoder at batch 256 (256 x 197 tokens): 12 pre-norm blocks of
    LN -> qkv -> multi-head attention (12 heads of 64) -> proj -> residual ->
    LN -> fc1 + GELU -> fc2 -> residual, the four linear layers of each block
    at their own sparsity (uniform in [30, 80]%, Zipf-skewed rows), chained on
    the GPU by paper_2407_02068_amd.encoder (the composition the encoder
    tests check link by link); beside it the same chain with the library's
    dense kernel for the linear layers.  The linear layers' own time is the
    sum of their launches' event times inside the chain.  With ``power``, the
    board energy per 256 images above idle, block-sparse against dense."""
    import torch

    import workloads as wl
    from paper_2407_02068_amd.encoder import deit_chain
    layers = wl.b_stack()
    T, H = 197, 12
    n_seq = layers[0].M // T
    chain = deit_chain(layers, to_dev, n_seq, T, H)
    X0 = to_dev(layers[0].X)
    sparse = lambda: chain.run(X0, sparse=True)
    dense = lambda: chain.run(X0, sparse=False)
    n = max(5, steps // 4)
    prewarm([sparse, dense], 0.5)
    sms, dms = interleaved(sparse, dense, 3, n)
    ev_s, ev_d = [], []
    for _ in range(3):  # the linear launches alone, inside the chain
        chain.run(X0, sparse=True, linear_events=ev_s)
        chain.run(X0, sparse=False, linear_events=ev_d)
    torch.cuda.synchronize()
    lin_s = sum(a.elapsed_time(b) for a, b in ev_s) / 3
    lin_d = sum(a.elapsed_time(b) for a, b in ev_d) / 3
    from paper_2407_02068_amd import lpv
    A, O, qkv, R, P = chain.A, chain.O, chain.qkv, chain.R, chain.P
    g1, b0 = chain.gamma, chain.beta
    _, ams = time_launches(lambda: lpv.attention(qkv, n_seq, T, H, out=O), max(10, steps // 2), 5)
    _, lms = time_launches(lambda: lpv.add_layernorm(R[0], P, g1, b0, 1e-6, S=R[1], out=A),
                           max(10, steps // 2), 5)
    pw = measure_power(sparse, dense, unit="256_images") if power else None
    # the same chains captured into HIP graphs (one replay = one forward pass)
    g_s, _ = chain.capture(X0, sparse=True)
    g_d, _ = chain.capture(X0, sparse=False)
    gms, gdms = interleaved(g_s.replay, g_d.replay, 3, n)
    del g_s, g_d
    chain.close()
    kept = sum(w.kept_flops() for w in layers)
    dense_fl = sum(w.dense_flops() for w in layers)
    att_flops = 4.0 * n_seq * H * T * T * 64          # QK^T and PV, per block
    ln_bytes = 4.0 * layers[0].M * 768 * 2              # x, y read; S, out written
    avg = lambda ms: sum(ms) / len(ms)
    return {"blocks": len(layers) // 4, "linears": len(layers),
            "kept_gflop": round(kept / 1e9, 1), "dense_gflop": round(dense_fl / 1e9, 1),
            "ms": round(avg(sms), 4), "images_per_s": round(n_seq / (avg(sms) * 1e-3), 1),
            "dense_ms": round(avg(dms), 4), "speedup_vs_dense": round(avg(dms) / avg(sms), 3),
            "graph_ms": round(avg(gms), 4), "graph_dense_ms": round(avg(gdms), 4),
            "graph_images_per_s": round(n_seq / (avg(gms) * 1e-3), 1),
            "linear_ms": round(lin_s, 4), "linear_dense_ms": round(lin_d, 4),
            "linear_tflops": round(kept / (lin_s * 1e-3) / 1e12, 1),
            "linear_speedup_vs_dense": round(lin_d / lin_s, 3),
            "attention_ms": round(avg(ams), 5),
            "attention_tflops": round(att_flops / (avg(ams) * 1e-3) / 1e12, 1),
            "add_layernorm_ms": round(avg(lms), 5),
            "add_layernorm_GBs": round(ln_bytes / (avg(lms) * 1e-3) / 1e9, 1),
            "power": pw,
            "note": "event averages of the whole encoder (12 blocks, 25 LN, 12 attention, 48 "
                    "linear launches), block-sparse and dense chains interleaved; linear_ms = the "
                    "48 linear launches' event times inside the chain (linear_tflops = kept "
                    "FLOPs / linear_ms); graph_ms / graph_dense_ms: the same chains captured "
                    "once into HIP graphs and replayed; DeiT-B, 256 x 197 tokens, 32x32 blocks; "
                    "attention and LN timed alone at the same shape"}


def sweep(steps, cfgs=("fc1", "s_fc1", "b_layer")):
    """Every measured point besides the headline: the DeiT-B fc1 sweep (blocks
    16/32/64 x sparsity 0/25/50/75/90% x bf16/fp16, exact-count uniform masks),
    DeiT-S fc1 with bias + GELU (batch 64, top-half L2 masks) and the four
    linears of one DeiT-B layer (batch 128).  Each point: block-sparse and
    dense launches interleaved (3 rounds), kept TFLOP/s, the fraction of the
    bf16/fp16 matrix-core peak and the speed-up over lpv_dense_linear."""
    import numpy as np
    import torch

    import workloads as wl
    from paper_2407_02068_amd import lpv
    pts = []

    def todev(a, dtype):
        a = np.ascontiguousarray(a)
        if dtype == "bf16":
            return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).cuda()
        return torch.from_numpy(a).cuda()

    def point(w, X, cfg):
        W, b = todev(w.W, w.dtype), todev(w.bias, w.dtype)
        h = lpv.bsr_pack(W, torch.from_numpy(w.mask).cuda(), w.b_r, w.b_c)
        Y = torch.empty((X.shape[0], w.N), dtype=X.dtype, device="cuda")
        Yd = torch.empty_like(Y)
        epi = "gelu" if w.gelu else None
        fs = lambda: lpv.bsr_linear(h, X, b, Y, epi=epi)
        fd = lambda: lpv.dense_linear(W, X, b, Yd, epi=epi)
        prewarm([fs, fd], 0.05)
        n = max(5, min(20, steps))
        a, d = interleaved(fs, fd, 3, n)
        h.close()
        ts, td = pct(sorted(a), .5), pct(sorted(d), .5)
        kept = w.kept_flops(X.shape[0])
        pts.append({"config": cfg, "workload": w.name, "M": X.shape[0], "N": w.N, "K": w.K,
                    "block": [w.b_r, w.b_c], "sparsity_pct": w.meta.get("sparsity"),
                    "dtype": w.dtype, "gelu": w.gelu, "kept_gflop": round(kept / 1e9, 3),
                    "bsr_us": round(ts * 1e3, 1), "dense_us": round(td * 1e3, 1),
                    "tflops": round(kept / (ts * 1e-3) / 1e12, 1),
                    "frac_of_peak": round(kept / (ts * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
                    "speedup_vs_dense": round(td / ts, 3)})
        log("sweep %-28s %7.1f us (dense %7.1f us) %6.1f TFLOP/s  x%.2f" % (
            w.name, ts * 1e3, td * 1e3, pts[-1]["tflops"], pts[-1]["speedup_vs_dense"]))

    if "fc1" in cfgs:
        for dtype in ("bf16", "f16"):
            X = todev(wl.activations(4, 0, 256 * 197, 768, dtype), dtype)
            for block in wl.FC1_SWEEP_BLOCKS:
                for sp in wl.FC1_SWEEP_SPARSITY:
                    point(wl.b_fc1(block=block, sparsity=sp, dtype=dtype, with_x=False), X,
                          "b_fc1_sweep")
            del X
    if "s_fc1" in cfgs:
        w = wl.s_fc1_gelu()
        point(w, todev(w.X, w.dtype), "s_fc1_gelu")
    if "b_layer" in cfgs:
        for w in wl.b_layer():
            point(w, todev(w.X, w.dtype), "b_layer")
    torch.cuda.synchronize()
    return {"points": pts,
            "note": "median event time of 3 interleaved rounds per point (block-sparse, dense); "
                    "frac_of_peak against the 2.5 PFLOP/s dense bf16/fp16 matrix-core peak"}


def pct(ms, q):
    return ms[min(len(ms) - 1, int(q * (len(ms) - 1) + 0.5))]


def cpu_baseline(w, target_s=12.0):
    """The float64 oracle on the host cores, on a bounded sample of token
    rows of the same workload; reported as effective TFLOP/s on kept blocks."""
    import numpy as np
    import oracle
    nt = oracle.default_threads()
    rows = 64
    t = 0.0
    while True:
        X = w.X[:rows]
        t0 = time.perf_counter()
        oracle.linear(X, w.W, w.dtype, w.b_r, w.b_c, w.mask, w.bias, gelu=w.gelu, nthreads=nt)
        t = time.perf_counter() - t0
        if t >= target_s / 4 or rows >= w.M:
            break
        rows = min(w.M, int(rows * max(2.0, target_s / 4 / max(t, 1e-3))))
    reps, total = 1, t
    while rows >= w.M and total < target_s and reps < 10:  # the whole workload: repeat it
        X = w.X[:rows]
        t0 = time.perf_counter()
        oracle.linear(X, w.W, w.dtype, w.b_r, w.b_c, w.mask, w.bias, gelu=w.gelu, nthreads=nt)
        total += time.perf_counter() - t0
        reps += 1
    t = total / reps
    flops = w.kept_flops(rows)
    return {"value": flops / t / 1e12, "unit": "TFLOP/s", "cores": nt, "kind": "oracle",
            "sample": "first %d of %d token rows of the same workload (float64 mask expansion + "
                      "triple loop), mean of %d runs, %.1f s each" % (rows, w.M, reps, t)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--prewarm-s", type=float, default=1.5,
                    help="seconds of alternating block-sparse and dense launches before any timing")
    ap.add_argument("--rounds", type=int, default=8,
                    help="interleaved block-sparse / dense rounds for the speed-up")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-backward", action="store_true",
                    help="skip the backward and delta-curve timings")
    ap.add_argument("--no-power", action="store_true", help="skip the amd-smi power legs")
    ap.add_argument("--no-stack", action="store_true", help="skip the 12-block DeiT-B encoder")
    ap.add_argument("--no-sweep", action="store_true", help="skip the sweep of the other configs")
    ap.add_argument("--no-flushed", action="store_true",
                    help="skip the cold-cache timing (kernel statistics of warm launches only)")
    ap.add_argument("--gelu", action="store_true", help="fused GELU epilogue (secondary point)")
    ap.add_argument("--dtype", default="bf16", choices=["bf16", "f16"])
    ap.add_argument("--block", type=int, default=32)
    ap.add_argument("--sparsity", type=int, default=50)
    ap.add_argument("--profile-pass", action="store_true",
                    help="only 3 launches of each path and a 1 GiB device copy (rocprofv3 counter runs)")
    ap.add_argument("--write-traffic", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="turn two --profile-pass counter CSVs into the HBM traffic summary")
    ap.add_argument("--write-stats", nargs=3, metavar=("STATS_CSV", "TRACE_CSV", "BENCH_LOG"),
                    help="turn a rocprofv3 --kernel-trace --stats run of this script (its stats "
                         "and kernel-trace CSVs and the run's stderr) into the statistics summary")
    ap.add_argument("--write-stats-backward", metavar="STATS_CSV",
                    help="the same for the run with the backward and delta-curve legs")
    ap.add_argument("--write-counters", nargs=3, metavar="PASS_CSV",
                    help="turn the three --profile-pass counter CSVs (COUNTER_PASSES) into the "
                         "counter summary")
    ap.add_argument("--write-clock", metavar="CLOCK_CSV",
                    help="turn a --profile-pass GRBM_GUI_ACTIVE counter CSV into the clock summary")
    args = ap.parse_args()

    if args.write_traffic:
        write_traffic(*args.write_traffic, command=" ".join(["python bench.py"] + sys.argv[1:]))
        return
    if args.write_stats:
        write_stats(args.write_stats[0], " ".join(["python bench.py"] + sys.argv[1:]),
                    trace_csv=args.write_stats[1], bench_log=args.write_stats[2])
        return
    if args.write_stats_backward:
        write_stats(args.write_stats_backward,
                    command=" ".join(["python bench.py"] + sys.argv[1:]), backward=True)
        return
    if args.write_clock:
        write_clock(args.write_clock, command=" ".join(["python bench.py"] + sys.argv[1:]))
        return
    if args.write_counters:
        write_counters(args.write_counters, command=" ".join(["python bench.py"] + sys.argv[1:]))
        return

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the block-sparse layer shards over tokens with no "
              "exchange, so a multi-GPU run is N independent copies; run with --gpus 1",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import workloads as wl
    from paper_2407_02068_amd import lpv

    lpv.lib()
    torch.cuda.set_device(0)
    w = wl.b_fc1(block=args.block, sparsity=args.sparsity, dtype=args.dtype, gelu=args.gelu)
    M, N, K = w.M, w.N, w.K
    tt = torch.bfloat16 if w.dtype == "bf16" else torch.float16

    def to_dev(a):
        a = np.ascontiguousarray(a)
        if a.dtype == np.uint16:
            return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).cuda()
        return torch.from_numpy(a).cuda()

    X, W, b = to_dev(w.X), to_dev(w.W), to_dev(w.bias)
    mask = torch.from_numpy(w.mask).cuda()
    Y = torch.empty((M, N), dtype=tt, device="cuda")
    Yd = torch.empty((M, N), dtype=tt, device="cuda")
    epi = "gelu" if w.gelu else None
    log("workload %s: M=%d N=%d K=%d nnzb=%d" % (w.name, M, N, K, w.nnzb))

    torch.cuda.synchronize()
    t0 = time.perf_counter()
    h = lpv.bsr_pack(W, mask, w.b_r, w.b_c)
    pack_ms = (time.perf_counter() - t0) * 1e3

    n_sparse = [0]  # launches of the block-sparse kernel at this shape so far

    def sparse():
        n_sparse[0] += 1
        lpv.bsr_linear(h, X, b, Y, epi=epi)

    dense = lambda: lpv.dense_linear(W, X, b, Yd, epi=epi)
    if args.profile_pass:
        for _ in range(3):
            sparse()
        for _ in range(3):
            dense()
        src = torch.empty(CALIB_BYTES // 2, dtype=torch.bfloat16, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        log("profile pass done")
        h.close()
        return
    # the block mask of the same weight on the GPU (scores + top-k), one-time per weight
    maskgen = lambda: lpv.mask_topk(W, w.b_r, w.b_c, args.sparsity)
    _, mgms = time_launches(maskgen, 20, 3)
    # settle the clock (independent of --warmup), then the contract's W + K steps
    prewarm([sparse, dense], args.prewarm_s)
    for _ in range(args.warmup):
        sparse()
    torch.cuda.synchronize()
    log("STATS_WINDOW first=%d steps=%d" % (n_sparse[0], args.steps))
    wall, ms = time_launches(sparse, args.steps, 0)
    # the speed-up: block-sparse and dense rounds interleaved on the same clock
    with ClockSampler() as clock:
        ims, dms = interleaved(sparse, dense, args.rounds, max(10, args.steps // 4))
    # torch.addmm (hipBLASLt) at the same shape, as a check on the dense path only
    bl = lambda: torch.addmm(b, X, W.t())
    _, bms = time_launches(bl, max(20, args.steps // 2), 5)
    sw = None if args.no_sweep else sweep(args.steps)
    back = None if args.no_backward else time_backward(w, h, W, X, args.steps, tt, to_dev)
    dcurve = None if args.no_backward else time_delta_curve(w, W, args.steps, to_dev)
    power = None if args.no_power else measure_power(sparse, dense)
    stack = None if args.no_stack else time_stack(args.steps, to_dev, power=not args.no_power)
    # cold caches: the same launches after a 1 GiB write each
    fms = fdms = None
    if not args.no_flushed:
        flush_buf = torch.empty(CALIB_BYTES, dtype=torch.uint8, device="cuda")
        fms = time_flushed(sparse, 20, flush_buf)
        fdms = time_flushed(dense, 20, flush_buf)
        del flush_buf

    kept_flops = w.kept_flops()
    ms_step = wall / args.steps * 1e3
    value = kept_flops / (wall / args.steps) / 1e12
    ev_avg = sum(ms) / len(ms)
    achieved = kept_flops / (ev_avg * 1e-3) / 1e12
    kused = int((w.mask.sum(axis=0) > 0).sum()) * w.b_c
    alg_bytes = algorithmic_bytes(M, N, K, w.nnzb, w.b_r, w.b_c, kused)
    hbm_gbs = alg_bytes / (ev_avg * 1e-3) / 1e9
    traffic = measured_traffic()
    ims, dms = sorted(ims), sorted(dms)
    i_med, d_med = pct(ims, .5), pct(dms, .5)
    log("bsr_linear (timed steps): mean %.1f us, median %.1f us (p10 %.1f, p90 %.1f), %.0f TFLOP/s "
        "effective, %.0f GB/s alg." % (ev_avg * 1e3, pct(sorted(ms), .5) * 1e3,
                                       pct(sorted(ms), .1) * 1e3, pct(sorted(ms), .9) * 1e3,
                                       achieved, hbm_gbs))
    log("interleaved: bsr_linear median %.1f us, dense_linear median %.1f us (%.0f TFLOP/s), "
        "speedup %.3fx; clock %s" % (i_med * 1e3, d_med * 1e3,
                                      w.dense_flops() / (d_med * 1e-3) / 1e12, d_med / i_med,
                                      json.dumps(clock.summary())))
    log("hipBLASLt addmm median %.1f us" % (pct(bms, .5) * 1e3))
    if back:
        log("backward: dX %.1f us (dense %.1f us), dW %.1f us (hipBLASLt full G^T X %.1f us), "
            "db %.1f us" % (back["dx_ms"] * 1e3, back["dx_dense_ms"] * 1e3, back["dw_ms"] * 1e3,
                            back["dw_hipblaslt_dense_ms"] * 1e3, back["db_ms"] * 1e3))
    if power:
        log("power: %s" % json.dumps(power))
    if stack:
        log("DeiT-B encoder (12 blocks, batch 256): %.2f ms (%.0f images/s), dense linears "
            "%.2f ms (speedup %.2fx); linears alone %.2f ms vs %.2f ms (%.0f TFLOP/s); "
            "attention %.1f us (%.0f TFLOP/s), add+LN %.1f us (%.0f GB/s)"
            % (stack["ms"], stack["images_per_s"], stack["dense_ms"], stack["speedup_vs_dense"],
               stack["linear_ms"], stack["linear_dense_ms"], stack["linear_tflops"],
               stack["attention_ms"] * 1e3, stack["attention_tflops"],
               stack["add_layernorm_ms"] * 1e3, stack["add_layernorm_GBs"]))
        log("DeiT-B encoder as HIP graph replays: %.2f ms (%.0f images/s), dense linears %.2f ms"
            % (stack["graph_ms"], stack["graph_images_per_s"], stack["graph_dense_ms"]))
        if stack.get("power"):
            log("encoder power: %s" % json.dumps(stack["power"]))
    if dcurve:
        log("delta curve: %.1f us for %d samples x %d points (%.0f GB/s of %d MB)"
            % (dcurve["ms"] * 1e3, dcurve["n_samples"], dcurve["points"],
               dcurve["hbm_achieved_GBs"], dcurve["hbm_alg_bytes"] // 1000000))
    if fms:
        log("flushed caches: bsr_linear median %.1f us, dense_linear median %.1f us (speedup %.2fx)"
            % (pct(fms, .5) * 1e3, pct(fdms, .5) * 1e3, pct(fdms, .5) / pct(fms, .5)))
    log("pack: %.2f ms (one-time); mask_topk median %.1f us (one-time)"
        % (pack_ms, pct(mgms, .5) * 1e3))

    out = {
        "metric": "effective TFLOP/s + speedup vs dense, DeiT-B fc1 at 50% block sparsity",
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {"workload": "DeiT-B fc1 batch 256: X [%d x %d] -> %d, %dx%d blocks, %d%% block "
                               "sparsity (uniform, exact count), %s, bias%s"
                               % (M, K, N, w.b_r, w.b_c, args.sparsity, w.dtype,
                                  " + GELU" if w.gelu else ", no GELU"),
                   "M": M, "N": N, "K": K, "block": [w.b_r, w.b_c], "sparsity_pct": args.sparsity,
                   "nnzb": w.nnzb, "kept_gflop": round(kept_flops / 1e9, 2)},
        "speedup_vs_dense": round(d_med / i_med, 3),
        "interleaved": {"rounds": args.rounds, "per_round": max(10, args.steps // 4),
                        "bsr_ms_median": round(i_med, 5), "bsr_ms_p10": round(pct(ims, .1), 5),
                        "bsr_ms_p90": round(pct(ims, .9), 5),
                        "dense_ms_median": round(d_med, 5), "dense_ms_p10": round(pct(dms, .1), 5),
                        "dense_ms_p90": round(pct(dms, .9), 5),
                        "dense_tflops": round(w.dense_flops() / (d_med * 1e-3) / 1e12, 1),
                        "gpu_clock": clock.summary()},
        "prewarm_s": args.prewarm_s,
        "bsr_ms_median": round(pct(sorted(ms), .5), 5),
        "bsr_ms_p10": round(pct(sorted(ms), .1), 5),
        "bsr_ms_p90": round(pct(sorted(ms), .9), 5),
        "hipblaslt_addmm_ms": round(pct(bms, .5), 5),
        "speedup_vs_hipblaslt": round(pct(bms, .5) / i_med, 3),
        "flushed": None if not fms else {
            "bsr_ms_median": round(pct(fms, .5), 5), "bsr_ms_p90": round(pct(fms, .9), 5),
            "dense_ms_median": round(pct(fdms, .5), 5),
            "speedup_vs_dense": round(pct(fdms, .5) / pct(fms, .5), 3),
            "note": "each launch after a 1 GiB device write (L2 and MALL evicted)"},
        "sweep": sw,
        "backward": back,
        "delta_curve": dcurve,
        "power": power,
        "encoder": stack,
        "pack_ms": round(pack_ms, 3),
        "mask_topk_ms_median": round(pct(mgms, .5), 5),
        "roofline": {"bound": "mfma", "achieved": round(achieved, 1), "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                     "traffic": traffic,
                     "kernel": "k_linear16 (lpv_bsr_linear)",
                     "achieved_from": "kept FLOPs / mean HIP-event duration of the %d timed steps"
                                      % args.steps,
                     "hbm_alg_bytes": alg_bytes, "hbm_achieved_GBs": round(hbm_gbs, 1),
                     "hbm_peak_GBs": PEAK_HBM_GBS, "hbm_frac": round(hbm_gbs / PEAK_HBM_GBS, 4)},
    }
    if not args.no_cpu:
        log("timing the CPU oracle on a sample ...")
        out["cpu_baseline"] = cpu_baseline(w)
    else:
        out["cpu_baseline"] = None
    h.close()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
