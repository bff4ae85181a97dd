#!/usr/bin/env python3
"""Throughput of the fused compress + decompress + error-update step on one MI355X.

Default workload: the 8192x4096 bf16 inter-stage activation gradient, rank 16,
one power iteration, error buffer and Q carried from step to step, a fresh
seeded input each step (8 distinct inputs, cycled).  A step is one
occ_step call: error-feedback add, left product, CholeskyQR, right product,
reconstruction and residual.

Prints ONE JSON line.  `value` is input GB/s (bytes of M as stored, per step,
over the measured step time) with every input already resident in HBM, from
K back-to-back steps between two synchronisations.  `cold` repeats the step
at least 20 times, each with its own event pair after a read of an unrelated
2 GiB buffer outside the events (the caches then hold clean, unrelated data),
and reports the median; `step_roofline` and `cold.step_roofline_frac` are the
two step-level fractions of the 8 TB/s HBM roofline.
`roofline` is measured for the kernel that takes the most time, from HIP
events bracketing each of its launches on the library's stream, against the
8 TB/s HBM3E peak; `traffic` comes from the committed rocprofv3 counter
summary in profiles/ when it matches the current kernel sources.
`cpu_baseline` times the float64 oracle on this host on a bounded sample of
the same workload.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload 1..5]
"""

from __future__ import annotations

import argparse
import glob
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "compress+decompress+err-update input GB/s and % of HBM roofline, 1 MI355X"
HBM_PEAK_GBS = 8000.0
FP32_MFMA_PEAK_TFLOPS = 157.3     # dense fp32 matrix-core peak of the MI355X
BF16_MFMA_PEAK_TFLOPS = 2500.0    # dense bf16 matrix-core peak of the MI355X
PROFILES = os.path.join(ROOT, "profiles")
CSRC = os.path.join(ROOT, "paper_2301_09830_amd", "csrc")


def code_lines(text: str) -> str:
    """C++ source without its line comments, trailing blanks and empty lines
    (the library's sources hold no "//" inside string literals)."""
    out = []
    for line in text.splitlines():
        line = line.split("//", 1)[0].rstrip()
        if line:
            out.append(line)
    return "\n".join(out)


def kernel_source_digest() -> str:
    """Digest of the library's code (comments excluded); counter summaries
    apply only to it."""
    h = hashlib.sha256()
    for path in sorted(glob.glob(os.path.join(CSRC, "*.hpp")) + glob.glob(os.path.join(CSRC, "*.hip"))):
        with open(path, encoding="utf-8") as f:
            h.update(os.path.basename(path).encode())
            h.update(code_lines(f.read()).encode())
    return h.hexdigest()[:16]


# ----------------------------------------------------------------------------
# algorithmic byte accounting (bytes that must cross HBM, per element of M)
# ----------------------------------------------------------------------------
def kernel_alg_bytes(kernel: str, elements: int, m_bytes: int) -> int | None:
    """Bytes one launch of a streaming kernel must move for `elements` of M.

    Passes named without a suffix read M and err_prev (m_bytes + 4 per
    element); pass_p_first also stores A = M + err_prev over err (+4); the
    passes named *_a read that stored A back (4).  The reconstruction pass
    writes err (+4) and M_hat (+4) on top of its reads.
    """
    per = {"pass_p": m_bytes + 4, "pass_q": m_bytes + 4, "mhat_err": m_bytes + 12,
           "err_only": m_bytes + 8, "pass_p_first": m_bytes + 8, "pass_p_a": 4,
           "pass_q_a": 4, "mhat_err_a": 12, "err_only_a": 8}.get(kernel)
    return None if per is None else per * elements


def product_engine(kernel: str, m_dtype: str, rank: int) -> tuple:
    """(matrix-core peak in TFLOP/s of ALGORITHMIC flops, engine) of a product kernel.

    Ranks padded to <= 16 and fp32 inputs run fp32 products on fp32 matrix
    cores.  For bf16 M at padded ranks 32..128 the left and right products
    and the reconstruction run on bf16 matrix cores with split operands,
    three bf16 products per algorithmic product, so the algorithmic flops
    have a third of the bf16 peak."""
    split = kernel.startswith(("pass_", "mhat_err", "err_only"))
    if m_dtype == "bf16" and rank > 16 and split:
        return BF16_MFMA_PEAK_TFLOPS / 3.0, "bf16 matrix cores, split operands (3 products)"
    return FP32_MFMA_PEAK_TFLOPS, "fp32 matrix cores"


def kernel_alg_flops(kernel: str, elements: int, rank: int) -> int | None:
    """Flops of one launch of a product kernel: 2 r per element of M (the
    left and right products and the reconstruction each do r FMAs)."""
    if kernel.split("_")[0] in ("pass", "mhat") or kernel.startswith("err_only"):
        return 2 * rank * elements
    return None


def step_alg_bytes(elements: int, m_bytes: int, iters: int, write_mhat: bool = True) -> int:
    """Algorithmic bytes of one step: the cheaper of re-reading M and err in
    each of the 2t+1 passes (X) and storing A in the first pass to read it
    back afterwards (Y), plus the err and M_hat writes."""
    out = 4 + (4 if write_mhat else 0)
    x = (2 * iters + 1) * (m_bytes + 4) + out
    y = (m_bytes + 8) + 4 * (2 * iters - 1) + 4 + out
    return elements * min(x, y)


def load_profile(kernel: str, workload: str) -> dict | None:
    """The committed counter summary of a kernel on a workload, if it was
    taken on the current kernel sources."""
    path = os.path.join(PROFILES, f"{kernel}__{workload}__pmc.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    start = text.find("```json")
    if start < 0:
        return None
    end = text.find("```", start + 7)
    try:
        rec = json.loads(text[start + 7:end])
    except ValueError:
        return None
    if rec.get("kernel_source_sha") != kernel_source_digest():
        return None
    return rec


def load_traffic(kernel: str, workload: str, launches_elements: int):
    """HBM bytes per launch from the committed counter summary, or None."""
    rec = load_profile(kernel, workload)
    return None if rec is None else rec.get("hbm_bytes_per_launch")


# ----------------------------------------------------------------------------
# workload setup
# ----------------------------------------------------------------------------
def gen_inputs(w, n_inputs: int):
    """Stored-dtype host matrices: n_inputs steps x len(w.shapes) matrices."""
    from concurrent.futures import ThreadPoolExecutor
    jobs = [(s, j) for s in range(n_inputs) for j in range(len(w.shapes))]
    with ThreadPoolExecutor(max_workers=min(8, len(jobs))) as ex:
        mats = list(ex.map(lambda sj: w.matrix(*sj), jobs))
    return {sj: m for sj, m in zip(jobs, mats)}


def to_device(x, dtype: str):
    import numpy as np
    import torch
    if dtype == "f32":
        return torch.from_numpy(np.ascontiguousarray(x)).cuda()
    return torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(torch.bfloat16).cuda()


def host_info() -> dict:
    """CPU model of this host and the BLAS library numpy runs on."""
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    blas, threads = "unknown", 1
    try:
        from threadpoolctl import threadpool_info
        for i in threadpool_info():
            if i.get("user_api") == "blas":
                blas = f"{i.get('internal_api')} {i.get('version')} ({i.get('architecture')})"
                threads = int(i.get("num_threads", 1))
                break
    except Exception:
        threads = int(os.environ.get("OMP_NUM_THREADS", "1"))
    return {"cpu_model": model, "blas": blas, "cores": threads}


def cpu_baseline(w, host, seconds: float, runs: int = 3):
    """Time oracle.step on this host's cores: `runs` runs of about
    seconds / runs each over the same bounded sample (whole matrix steps,
    err and Q carried from the workload's initial state), reporting the
    median input GB/s."""
    import numpy as np
    import oracle
    info = host_info()
    count = len(w.shapes)
    n_inputs = len({s for (s, _) in host})
    rates, mats_done, spent = [], [], 0.0
    for _ in range(runs):
        state = {j: (np.zeros(w.shapes[j]), w.q0(j).astype(np.float64)) for j in range(count)}
        done_bytes, steps, mats = 0, 0, 0
        t0 = time.perf_counter()
        while True:
            s = steps % n_inputs
            for j in range(count):
                e, q = state[j]
                out = oracle.step(host[(s, j)], w.m_dtype, e, q, w.rank, w.iters)
                state[j] = (out["err"], out["Q"])
                done_bytes += host[(s, j)].nbytes
                mats += 1
                if time.perf_counter() - t0 > seconds / runs:
                    break
            steps += 1
            if time.perf_counter() - t0 > seconds / runs:
                break
        dt = time.perf_counter() - t0
        spent += dt
        rates.append(done_bytes / dt / 1e9)
        mats_done.append(mats)
    med = sorted(rates)[len(rates) // 2]
    return {"value": round(med, 4), "unit": "GB/s", "cores": info["cores"],
            "kind": "oracle", "seconds": round(spent, 2),
            "runs_gbs": [round(r, 4) for r in rates],
            "cpu_model": info["cpu_model"], "blas": info["blas"],
            "sample": f"median of {runs} runs of {'/'.join(str(x) for x in mats_done)} matrix "
                      f"steps of {w.name} (oracle.step, float64, err/Q carried from the initial "
                      f"state) on {info['cores']} BLAS threads"}


# ----------------------------------------------------------------------------
# rocprofv3 summaries -> profiles/ (host-side text processing, no GPU)
# ----------------------------------------------------------------------------
def profile_name(kname: str) -> str | None:
    """Launch name (as in the per-kernel timings) of a library kernel, from its
    demangled name as rocprofv3 reports it."""
    base = kname.split("(")[0].replace("void ", "").replace("occ::", "").strip()
    short = base.split("<")[0]
    args = [a.strip() for a in base[len(short) + 1:-1].split(",")] if "<" in base else []
    fixed = {"k_pm": "pass_p", "k_qm": "pass_q", "k_qfin16": "q_finish", "k_qpad": "qpad",
             "k_qredl": "q_reduce", "k_qpadl": "qpad"}
    if short in fixed:
        return fixed[short]
    if short == "k_mh16":
        if args[3] == "1":
            return "decompress"
        return "mhat_err" if args[4] == "true" else "err_only"
    if short == "k_lp":
        return {"0": "pass_p", "1": "pass_p_first", "2": "pass_p_a"}[args[2]]
    if short == "k_lq":
        return {"0": "pass_q", "2": "pass_q_a"}[args[2]]
    if short == "k_ml":
        if args[3] == "1":
            return "decompress"
        return "mhat_err_a" if args[4] == "true" else "err_only_a"
    if short == "k_mlx":
        if args[1] == "1":
            return "decompress"
        return "mhat_err_a" if args[2] == "true" else "err_only_a"
    if short == "k_lqx":
        return {"0": "pass_q", "2": "pass_q_a"}[args[2]]
    pair = {"k_lg": "gram", "k_gsum": "gram_sum", "k_lchol": "chol", "k_lapply": "apply"}
    if short in pair:
        return pair[short] + ("2" if args[-1] == "1" else "")
    return None


XCDS = 8        # accelerator complex dies of the MI355X (GRBM_GUI_ACTIVE is summed over them)
SIMDS = 1024    # 256 compute units x 4 SIMDs


def write_profiles(workload: str, trace_dir: str, fetch_dir: str, write_dir: str,
                   commands: dict, elements: int, m_bytes: int, mfma_dir: str | None = None,
                   streaming_only: bool = False) -> list:
    """Summaries of one rocprofv3 kernel trace and two counter runs (plus, with
    mfma_dir, a run of matrix-core counters)."""
    import csv
    out = []
    stats = glob.glob(os.path.join(trace_dir, "*kernel_stats.csv"))[0]
    rows = list(csv.DictReader(open(stats)))
    lines = ["| kernel | calls | avg us | min us | max us | share % |", "|---|---|---|---|---|---|"]
    for r in rows:
        lines.append(f"| `{r['Name'].split('(')[0]}` | {r['Calls']} | {float(r['AverageNs'])/1e3:.2f} | "
                     f"{float(r['MinNs'])/1e3:.2f} | {float(r['MaxNs'])/1e3:.2f} | {float(r['Percentage']):.1f} |")

    def counters(d):
        agg = {}
        for r in csv.DictReader(open(glob.glob(os.path.join(d, "*counter_collection.csv"))[0])):
            agg.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]))
        return {k: sum(v) / len(v) for k, v in agg.items()}
    fetch, write = counters(fetch_dir), counters(write_dir)
    mf = {}
    if mfma_dir:
        for r in csv.DictReader(open(glob.glob(os.path.join(mfma_dir, "*counter_collection.csv"))[0])):
            mf.setdefault(r["Kernel_Name"].split("(")[0], {}).setdefault(r["Counter_Name"], []).append(
                float(r["Counter_Value"]))
        mf = {k: {c: sum(v) / len(v) for c, v in d.items()} for k, d in mf.items()}
    copy = [k for k in fetch if "copyBuffer" in k or "copy" in k.lower()]
    cal_read = cal_write = None
    calib_bytes = commands.get("calibration_bytes")
    if copy and calib_bytes:
        k = copy[0]
        cal_read = calib_bytes / (fetch[k] * 1024.0)
        cal_write = calib_bytes / (write[k] * 1024.0)
    digest = kernel_source_digest()
    for r in rows:
        name = profile_name(r["Name"])
        if name is None or (streaming_only and kernel_alg_bytes(name, 1, m_bytes) is None):
            continue
        fk = next((k for k in fetch if k.split("(")[0] == r["Name"].split("(")[0]), None)
        rec = {"kernel": name, "hip_kernel": r["Name"].split("(")[0], "workload": workload,
               "avg_duration_us": round(float(r["AverageNs"]) / 1e3, 3),
               "kernel_source_sha": digest}
        if fk is not None and cal_read:
            rb = fetch[fk] * 1024.0 * cal_read
            wb = write[fk] * 1024.0 * cal_write
            rec.update(fetch_kib_per_dispatch=round(fetch[fk], 3), write_kib_per_dispatch=round(write[fk], 3),
                       read_calibration=round(cal_read, 4), write_calibration=round(cal_write, 4),
                       hbm_bytes_per_launch=int(rb + wb))
            alg = kernel_alg_bytes(name, elements, m_bytes)
            if alg:
                rec["alg_bytes_per_launch"] = alg
        mk = mf.get(r["Name"].split("(")[0])
        if mk and mk.get("GRBM_GUI_ACTIVE"):
            busy = mk.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0)
            gui = mk["GRBM_GUI_ACTIVE"]
            mops = sum(mk.get(c, 0.0) for c in ("SQ_INSTS_VALU_MFMA_MOPS_F32", "SQ_INSTS_VALU_MFMA_MOPS_BF16",
                                                   "SQ_INSTS_VALU_MFMA_MOPS_F64"))
            rec["mfma"] = {
                "busy_cycles": busy, "gui_active": gui,
                "util": round(busy / (gui / XCDS * SIMDS), 4),
                "flops_per_launch": mops * 512,
                "mops_f32": mk.get("SQ_INSTS_VALU_MFMA_MOPS_F32", 0.0),
                "mops_bf16": mk.get("SQ_INSTS_VALU_MFMA_MOPS_BF16", 0.0),
                "mops_f64": mk.get("SQ_INSTS_VALU_MFMA_MOPS_F64", 0.0),
                "tflops": round(mops * 512 / (rec["avg_duration_us"] * 1e-6) / 1e12, 1)}
        text = [f"# `{name}` on {workload}: rocprofv3 summary", "",
                f"Kernel `{rec['hip_kernel']}`; average duration {rec['avg_duration_us']} us "
                f"over {r['Calls']} dispatches.", "",
                "Commands (run from the repository root on the MI355X box):", ""]
        for key in ("trace", "fetch", "write", "mfma"):
            if key in commands:
                text.append(f"- {key}: `{commands[key]}`")
        text += ["", "Kernel trace statistics of the same run (all kernels of the step):", ""] + lines
        if "hbm_bytes_per_launch" in rec:
            text += ["", f"HBM traffic per dispatch: FETCH_SIZE {rec['fetch_kib_per_dispatch']} KiB x "
                         f"{rec['read_calibration']} + WRITE_SIZE {rec['write_kib_per_dispatch']} KiB x "
                         f"{rec['write_calibration']} = {rec['hbm_bytes_per_launch']} bytes. The calibration "
                         "factors are (bytes a plain device copy of known size moves) / (what the counter "
                         "reports for that copy)."]
        if "mfma" in rec:
            m_ = rec["mfma"]
            text += ["", f"Matrix cores: SQ_VALU_MFMA_BUSY_CYCLES {m_['busy_cycles']:.0f} over GRBM_GUI_ACTIVE "
                         f"{m_['gui_active']:.0f} (summed over the {XCDS} XCDs) and {SIMDS} SIMDs: busy "
                         f"{100 * m_['util']:.1f} % of the kernel's cycles; MFMA MOPS x 512 = "
                         f"{m_['flops_per_launch'] / 1e9:.1f} GFLOP per dispatch of matrix-core work, "
                         f"{m_['tflops']} TFLOP/s over the average duration."]
        text += ["", "```json", json.dumps(rec, indent=1), "```", ""]
        path = os.path.join(PROFILES, f"{name}__{workload}__pmc.md")
        with open(path, "w") as f:
            f.write("\n".join(text))
        out.append(path)
    return out


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=400)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", type=int, default=2, choices=[1, 2, 3, 4, 5])
    ap.add_argument("--inputs", type=int, default=0,
                    help="distinct seeded inputs cycled through (default: the workload's steps)")
    ap.add_argument("--rows", action="store_true",
                    help="embedding workload: the row-sparse step over the union of the "
                         "inputs' nonzero rows (bytes accounted by rows touched)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--cold-reps", type=int, default=30,
                    help="flushed repetitions (median reported; at least 20)")
    ap.add_argument("--flush-gib", type=float, default=2.0,
                    help="bytes read between flushed repetitions, GiB (at least 1)")
    ap.add_argument("--no-kernel-timing", action="store_true")
    ap.add_argument("--calibrate-copy-mib", type=int, default=0,
                    help="also run a plain device copy of this size (counter calibration)")
    ap.add_argument("--mfma-dir", default=None,
                    help="with --write-profiles: rocprofv3 csv output of the matrix-core counter run")
    ap.add_argument("--write-profiles", nargs=3, metavar=("TRACE_DIR", "FETCH_DIR", "WRITE_DIR"),
                    help="host only: turn rocprofv3 csv output into profiles/*.md summaries")
    ap.add_argument("--profile-commands", default="",
                    help="json {trace, fetch, write, calibration_bytes} recorded in the summaries")
    args = ap.parse_args()

    if args.write_profiles:
        from workloads import WORKLOADS
        w = WORKLOADS[args.workload]
        name, elements = w.name, w.elements
        if args.rows:
            # the rows the row-sparse step touches: the union over the inputs
            import numpy as np
            live = np.zeros(w.shapes[0][0], dtype=bool)
            for s in range(args.inputs or w.steps):
                live |= (w.matrix(s, 0) != 0).any(axis=1)
            name, elements = w.name + "_rows", int(live.sum()) * w.shapes[0][1]
        paths = write_profiles(name, *args.write_profiles, json.loads(args.profile_commands),
                               elements, 2 if w.m_dtype == "bf16" else 4, mfma_dir=args.mfma_dir,
                               streaming_only=w.rank > 16)
        print("\n".join(paths))
        return 0

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print(json.dumps({"metric": METRIC, "error": "liboptcc runs on one GPU; "
                          "multi-GPU runs are not part of this benchmark (use --gpus 1)"}))
        return 2

    import numpy as np
    import torch

    from paper_2301_09830_amd import optcc
    from workloads import WORKLOADS

    w = WORKLOADS[args.workload]
    n_inputs = args.inputs or w.steps
    host = gen_inputs(w, n_inputs)
    count = len(w.shapes)
    dev_M = {k: to_device(v, w.m_dtype) for k, v in host.items()}
    errs = [torch.zeros(s, dtype=torch.float32, device="cuda") for s in w.shapes]
    Qs = [torch.from_numpy(w.q0(j)).cuda() for j in range(count)]
    Ps = [torch.empty((s[0], w.rank), dtype=torch.float32, device="cuda") for s in w.shapes]
    Mhs = [torch.empty(s, dtype=torch.float32, device="cuda") for s in w.shapes]
    L = optcc.lib()
    arrays = []
    for s in range(n_inputs):
        arr = (optcc.occ_mat_t * count)()
        for j in range(count):
            mat = optcc.make_mat(dev_M[(s, j)], errs[j], Ps[j], Qs[j], Mhs[j])
            arr[j] = mat
        arrays.append(arr)
    n_live = None
    if args.rows:
        # Row-sparse step: one list for every timed step, the union of the
        # nonzero rows of all the inputs cycled through (the carried error
        # stays inside it: its rows are those of earlier inputs).
        if w.kind != "zipf" or count != 1:
            raise SystemExit("--rows applies to the embedding workload (--workload 4)")
        live = np.zeros(w.shapes[0][0], dtype=bool)
        for v in host.values():
            live |= (v != 0).any(axis=1)
        rows_t = torch.from_numpy(np.nonzero(live)[0].astype(np.int32)).cuda()
        n_live = int(rows_t.numel())
        Ps = [torch.empty((n_live, w.rank), dtype=torch.float32, device="cuda")]
        Mhs = [torch.zeros(w.shapes[0], dtype=torch.float32, device="cuda")]
        for s in range(n_inputs):
            arrays[s][0].P = Ps[0].data_ptr()
            arrays[s][0].M_hat = Mhs[0].data_ptr()
        dt_code = optcc.OCC_BF16 if w.m_dtype == "bf16" else optcc.OCC_F32
        ws_bytes = L.occ_step_rows_workspace_bytes(n_live, w.shapes[0][1], dt_code, w.rank,
                                                   w.iters)
    else:
        ws_bytes = L.occ_workspace_bytes(arrays[0], count, w.rank, w.iters)
    ws = optcc.alloc_workspace(ws_bytes)
    stream = torch.cuda.current_stream()
    sptr = int(stream.cuda_stream)
    wsp = int(ws.data_ptr())

    def step(k: int) -> None:
        if n_live is not None:
            st = L.occ_step_rows(arrays[k % n_inputs], int(rows_t.data_ptr()), n_live, w.rank,
                                 w.iters, 0, wsp, ws_bytes, sptr)
        else:
            st = L.occ_step_batched(arrays[k % n_inputs], count, w.rank, w.iters, 0, wsp,
                                    ws_bytes, sptr)
        if st != 0:
            raise optcc.OccError("occ_step_rows" if n_live is not None else "occ_step_batched", st)

    for k in range(args.warmup):
        step(k)
    torch.cuda.synchronize()

    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record(stream)
    for k in range(args.steps):
        step(args.warmup + k)
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_events = ev0.elapsed_time(ev1)
    ms_per_step = ms_events / args.steps

    wname = w.name + ("_rows" if n_live is not None else "")
    # bytes accounted by the rows the step touches (all rows unless --rows)
    elements = w.elements if n_live is None else n_live * w.shapes[0][1]
    m_bytes = 2 if w.m_dtype == "bf16" else 4
    input_bytes = elements * m_bytes
    value = input_bytes / (ms_per_step * 1e-3) / 1e9
    step_bytes = step_alg_bytes(elements, m_bytes, w.iters)

    # Flushed ("cold") steps: before each repetition, outside its events, read
    # a buffer of flush_gib GiB (larger than the 256 MiB memory-side cache and
    # the 8 x 4 MiB L2), so every repetition starts with caches holding clean,
    # unrelated data; median over the repetitions.
    cold = None
    if args.cold_reps > 0:
        reps = max(20, args.cold_reps)
        flush = torch.empty(int(max(1.0, args.flush_gib) * (1 << 30)) // 4, dtype=torch.float32,
                            device="cuda").fill_(1.0)
        sink = torch.zeros((), dtype=torch.float32, device="cuda")
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(reps)]
        torch.cuda.synchronize()
        for k in range(reps):
            sink += flush.sum()
            evs[k][0].record(stream)
            step(args.warmup + args.steps + k)
            evs[k][1].record(stream)
        torch.cuda.synchronize()
        times = sorted(a.elapsed_time(b) for a, b in evs)
        med = times[len(times) // 2]
        cold = {"ms_per_step_median": round(med, 5), "ms_min": round(times[0], 5),
                "ms_max": round(times[-1], 5), "reps": reps,
                "value": round(input_bytes / (med * 1e-3) / 1e9, 2),
                "step_roofline_frac": round(step_bytes / (med * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                "flush": f"{flush.numel() * 4 / (1 << 30):.1f} GiB read (torch sum) before each "
                         "repetition, outside its events"}
        del flush

    kernels = {}
    roofline = None
    if not args.no_kernel_timing:
        optcc.occ_profile_begin()
        for k in range(args.steps):
            step(k)
        prof = optcc.occ_profile_end()
        for name, (launches, total_ms) in prof.items():
            kernels[name] = {"launches_per_step": round(launches / args.steps, 3),
                             "avg_us": round(total_ms / launches * 1e3, 3),
                             "share": None}
        tot = sum(v[1] for v in prof.values())
        for name in kernels:
            kernels[name]["share"] = round(prof[name][1] / tot, 4) if tot else None
        streaming = {k: v for k, v in prof.items() if kernel_alg_bytes(k, 1, m_bytes)}
        if streaming:
            dom = max(streaming, key=lambda k: streaming[k][1])
            launches, total_ms = prof[dom]
            avg_s = total_ms / launches * 1e-3
            per_launch = kernel_alg_bytes(dom, elements, m_bytes)  # one launch covers the batch
            flops = kernel_alg_flops(dom, elements, w.rank)
            prof_rec = load_profile(dom, wname)
            traffic = None if prof_rec is None else prof_rec.get("hbm_bytes_per_launch")
            # the bound is whichever resource the kernel's algorithmic work
            # needs longer on: HBM bytes at 8 TB/s or its flops on the matrix
            # cores it runs on
            mfma_peak, engine = product_engine(dom, w.m_dtype, w.rank)
            mfma_bound = flops is not None and flops / mfma_peak > per_launch / HBM_PEAK_GBS * 1e3
            if mfma_bound:
                achieved, peak, unit = flops / avg_s / 1e12, round(mfma_peak, 1), "TFLOP/s"
            else:
                achieved, peak, unit = per_launch / avg_s / 1e9, HBM_PEAK_GBS, "GB/s"
            # the committed kernel trace of the same kernel and workload, side by side
            trace_us = None if prof_rec is None else prof_rec.get("avg_duration_us")
            trace_frac = None
            if trace_us:
                t_s = trace_us * 1e-6
                trace_frac = round((flops / t_s / 1e12 if mfma_bound else per_launch / t_s / 1e9)
                                   / (mfma_peak if mfma_bound else HBM_PEAK_GBS), 4)
            roofline = {"kernel": dom, "bound": "mfma" if mfma_bound else "hbm",
                        "achieved": round(achieved, 1), "peak": peak, "unit": unit,
                        "frac": round(achieved / peak, 4),
                        "frac_source": "HIP events bracketing each launch in this run",
                        "trace_avg_us": trace_us, "trace_frac": trace_frac,
                        "traffic": traffic, "alg_bytes_per_launch": int(per_launch),
                        "alg_flops_per_launch": flops, "engine": engine,
                        "mfma_util": (prof_rec or {}).get("mfma", {}).get("util"),
                        "hbm_achieved_gbs": round(per_launch / avg_s / 1e9, 1),
                        "avg_launch_us": round(avg_s * 1e6, 3)}

    if args.calibrate_copy_mib:
        n = args.calibrate_copy_mib * (1 << 20) // 4
        a = torch.empty(n, dtype=torch.float32, device="cuda").normal_()
        b = torch.empty_like(a)
        for _ in range(5):
            b.copy_(a)
        torch.cuda.synchronize()

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(w, host, args.cpu_seconds)

    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": wname,
                   "shapes": [list(s) for s in w.shapes],
                   "m_dtype": w.m_dtype, "rank": w.rank, "iters": w.iters,
                   "distinct_inputs": n_inputs, "state": "err and Q carried across steps",
                   **({"live_rows": n_live, "live_fraction": round(n_live / w.shapes[0][0], 4),
                       "entry_point": "occ_step_rows"} if n_live is not None else {})},
        "step_roofline": {"alg_bytes_per_step": step_bytes,
                          "achieved": round(step_bytes / (ms_per_step * 1e-3) / 1e9, 1),
                          "frac": round(step_bytes / (ms_per_step * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                          "timing": "back-to-back steps (warm caches)"},
        "cold": cold,
        "roofline": roofline,
        "cpu_baseline": cpu,
        "kernels": kernels,
        "wall_s": round(wall, 3),
    }
    print(json.dumps(out))
    return 0


if __name__ == "__main__":
    sys.exit(main())
