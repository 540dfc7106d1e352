#!/usr/bin/env python3
"""Benchmark: tril(A A^T) on one MI355X.

A step is one pass of the hot path over the workload with its inputs already
resident in HBM: spsyrk_lower (validation, column index, symbolic pass, row
pointers, numeric pass with the semiring's finalisation), plus spsyrk_mirror
or spsyrk_offdiag where the workload asks for them.  The default workload is
the largest one: 2^23 x 2^28, 16 Zipf(0.9) columns per row with columns of
more than 50 entries dropped, int32 overlap counts finalised to fp32 Jaccard.

Prints one JSON line: useful GFLOP/s (2 per lower-triangle multiply-add,
integer semirings counted the same way), output nnz/s, the HBM roofline of the
dominant kernel (measured with HIP events on the library's stream inside the
timed region) and of the whole call, and the CPU oracle timed on a bounded
sample of the same workload.
"""
import argparse
import hashlib
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0   # MI355X HBM3E peak, GB/s
METRIC = "useful GFLOP/s + output nnz/s for tril(A*A^T); % of HBM roofline, 1 GPU"
V_IN = {"f64": 8, "f32": 4, "count": 0, "jaccard": 0}       # bytes per value of A
V_OUT = {"f64": 8, "f32": 4, "count": 4, "jaccard": 4}      # bytes per value of C
V_CX = {"f64": 8, "f32": 4, "count": 0, "jaccard": 0}       # bytes per value in the column index
# (Jaccard keys carry the partner's row length; no value array)


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=10)
    p.add_argument("--warmup", type=int, default=2)
    p.add_argument("--workload", default="jaccard_large")
    p.add_argument("--seed", type=int, default=1)
    p.add_argument("--scale-shift", type=int, default=0, help="shrink the workload by 2^k (testing only)")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-rows", type=int, default=0, help="rows in the oracle sample (0: automatic)")
    p.add_argument("--cpu-full", action="store_true",
                   help="also time the oracle over every row, on one thread and on all host threads")
    p.add_argument("--copy-calibration", action="store_true",
                   help="also run a plain 1 GiB device copy (reference for HBM byte counters)")
    p.add_argument("--json-out", default="")
    p.add_argument("--no-side", action="store_true",
                   help="skip the side measurements (copy bandwidth, lower vs offdiag(A, A), half blocks)")
    return p.parse_args()


def kernel_source_hash():
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2608_09713_amd", "csrc")
    for f in sorted(os.listdir(csrc)):
        if f.endswith((".hip", ".h")):
            h.update(open(os.path.join(csrc, f), "rb").read())
    return h.hexdigest()[:16]


def traffic_from_profiles(kernel_phase, workload):
    """HBM bytes per launch from the committed counter summary, if it was taken
    on the current kernel sources; else None."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    try:
        t = json.load(open(path))
    except Exception:
        return None
    if t.get("source_hash") != kernel_source_hash():
        return None
    k = t.get("workloads", {}).get(workload, {}).get("kernels", {}).get(kernel_phase)
    if not k:
        return None
    return k.get("hbm_bytes_per_launch")


def column_stats(A):
    c = np.bincount(A.col_idx, minlength=A.ncols)
    c = c.astype(np.int64)
    F_L = int((c * (c + 1) // 2).sum())
    n_ne = int(np.count_nonzero(c))
    return F_L, n_ne


def alg_bytes_phase(phase, sz, sr):
    """Algorithmic bytes of one launch of a one-kernel phase: every array the
    kernel must touch, counted once (per-product gathers of partner keys are
    not counted; each key of the column index counts once).

    light_numeric (the single-pass light-row kernel) reads the row pointers,
    the per-row product counts and staging slots (8 B each per row), the
    packed partner-run word of every entry (4 B; the rare run too long for its
    word is read from the full table and not counted), the values of A (fp
    semirings), every kept column-index key and value once; it writes every
    light output entry at its staging slot (column + value, or one packed 4-B
    word for counts and Jaccard values when the stats say so) and the exact
    row lengths (8 B per row).  compact reads every staged entry and writes it
    as column + value once, plus three 8-B words per row (and, unpacking
    Jaccard words, the row pointers of A).  colindex_pack (the local sort that
    writes the column index) reads every sorted record (column, row field,
    entry index: 12 B), writes every entry's key and index value at its sorted
    position and the packed partner-run word (4 B) of every entry that has
    partners (all but the first of each column).  heavy_symbolic reads the
    heavy-row list, their row pointers, their entries' run words, cursors and
    run ends (12 B), every kept index key once, and writes a length per heavy
    row; heavy_numeric reads the same plus the output row pointers, A's values
    and the index values, and writes the heavy rows' output entries."""
    m, nnz = sz["m"], sz["nnz_A"]
    vo = 4 + V_OUT[sr]
    nh, he, hout = sz["heavy_rows"], sz["heavy_entries"], sz["heavy_nnz_out"]
    light_out = sz["nnz_C"] - hout
    packed = bool(sz.get("packed_staging"))
    staged = 4 if packed else vo
    if phase == "light_numeric":
        return (8 * (m + 1) + 8 * m + 8 * m + 4 * nnz + nnz * V_IN[sr]
                + sz["csc_entries"] * (4 + V_CX[sr]) + light_out * staged + 8 * m)
    if phase == "compact":
        return light_out * (staged + vo) + 3 * 8 * m + (8 * (m + 1) if packed and sr == "jaccard" else 0)
    if phase == "colindex_pack":
        return 12 * nnz + nnz * (4 + V_CX[sr]) + 4 * (nnz - sz["n_ne"])
    if phase == "heavy_symbolic":
        return 4 * nh + 16 * nh + 12 * he + 4 * sz["csc_entries"] + 8 * nh
    if phase == "heavy_numeric":
        return (4 * nh + 16 * nh + 8 * nh + he * (12 + V_IN[sr]) + sz["csc_entries"] * (4 + V_CX[sr])
                + hout * vo)
    return None


# phases that are one kernel launch each (a roofline is quoted for one kernel)
SINGLE_KERNEL_PHASES = ("light_numeric", "compact", "colindex_pack", "heavy_symbolic", "heavy_numeric")


def whole_call_bytes(sz, sr, mirror_nnz=None):
    """B_alg of the call: A read once, A's column-major copy written and read
    once, C_L written once (and, with the mirror, C_L read and C written)."""
    m, nnz, v = sz["m"], sz["nnz_A"], V_IN[sr]
    B_A = 8 * (m + 1) + nnz * (4 + v)
    B_AT = 2 * (8 * (sz["n_ne"] + 1) + nnz * (4 + v))
    B_C = 8 * (m + 1) + sz["nnz_C"] * (4 + V_OUT[sr])
    b = B_A + B_AT + B_C
    if mirror_nnz is not None:
        b += B_C + 8 * (m + 1) + mirror_nnz * (4 + V_OUT[sr])
    return b


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor()


ORACLE_PRODUCTS_PER_S = 5e6   # rough single-thread oracle speed (map updates per second), for sizing samples


def _oracle_leg(A, sr, rows, threads):
    """Time the oracle over the given rows (None: all) on ``threads`` threads;
    the column-major copy of A is built inside the timed call."""
    import oracle
    Ain = A if sr in ("f64", "f32") else A.with_values(None)
    t0 = time.perf_counter()
    R = oracle.lower(Ain, sr, rows=rows, threads=threads)
    t = time.perf_counter() - t0
    flops = 2 * int(R.count.astype(np.int64).sum())
    nrows = A.nrows if rows is None else len(rows)
    out = {"value": flops / t / 1e9, "unit": "GFLOP/s", "cores": threads, "kind": "oracle",
           "nnz_per_s": R.nnz / t, "seconds": t, "rows": nrows, "flops": flops}
    del R
    return out


def _sample(A, frac, seed):
    if frac >= 1.0:
        return None
    rng = np.random.default_rng(seed + 1000)
    k = max(1, int(A.nrows * frac))
    return np.sort(rng.choice(A.nrows, size=k, replace=False))


def cpu_baseline(A, sr, F_L, seed, rows_override=0):
    """The oracle as it stands, timed on this host beside the GPU run, on a
    bounded seeded row sample: on all host threads (the headline figure;
    blocks of rows through the same per-row code) over a sample of about
    25 s of single-thread work, and on one thread over about 8 s of work."""
    import oracle
    oracle.build()
    threads = oracle.host_threads()
    if rows_override:
        f_multi = f_single = min(1.0, rows_override / A.nrows)
    else:
        f_multi = min(1.0, 25.0 * ORACLE_PRODUCTS_PER_S / max(1, F_L))
        f_single = min(1.0, 8.0 * ORACLE_PRODUCTS_PER_S / max(1, F_L))
    multi = _oracle_leg(A, sr, _sample(A, f_multi, seed), threads)
    single = _oracle_leg(A, sr, _sample(A, f_single, seed + 1), 1)
    host = f"host {cpu_model()} with {os.cpu_count()} logical CPUs ({threads} used)"
    multi["sample"] = (f"{multi['rows']} of {A.nrows} rows (seeded), computed in blocks of rows on {threads} "
                       f"threads, column-major copy of A built inside the timed call (one thread); {host}")
    single["sample"] = f"{single['rows']} of {A.nrows} rows (seeded), one thread; {host}"
    multi["single_thread"] = single
    return multi


def cpu_full(A, sr, seed, skip_single):
    """Every row: one thread (unless skip_single) and all host threads."""
    import oracle
    oracle.build()
    out = {"threads": oracle.host_threads(), "cpu": cpu_model(), "logical_cpus": os.cpu_count()}
    out["all_threads"] = _oracle_leg(A, sr, None, out["threads"])
    if not skip_single:
        out["one_thread"] = _oracle_leg(A, sr, None, 1)
    return out


def timed_call(torch, fn, reps=3):
    """Median wall time (ms) of a whole library call, device work included."""
    out = fn()
    del out
    torch.cuda.synchronize()
    ts = []
    for _ in range(reps):
        t0 = time.perf_counter()
        out = fn()
        torch.cuda.synchronize()
        ts.append((time.perf_counter() - t0) * 1e3)
        del out
    return float(np.median(ts))


def side_measurements(sp, torch, dev, Ad, Bd, sr, w, whole_call_GBs):
    """Figures reported beside the metric (outside the timed steps): a plain
    device copy's bandwidth and the whole call against it; t(lower(A)) over
    t(offdiag(A, A)) (ideal about 0.5: half the products and about half the
    output); a planned product for new values of the same pattern; Y = C X
    for 1 and 8 columns from C_L alone (Eq. (spmv)), with its
    HBM figure; two stages (A's columns split in half) accumulated one call
    at a time against the one-shot lower part; for a workload with a right
    operand, the two half blocks of Algorithm 3 against the full block."""
    side = {}
    src = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    src.fill_(1)
    ms = timed_call(torch, lambda: dst.copy_(src), reps=5)
    del src, dst
    copy_GBs = 2 * (1 << 30) / (ms / 1e3) / 1e9
    side["copy_GBs"] = copy_GBs
    side["whole_call_vs_copy"] = whole_call_GBs / copy_GBs
    t_low = timed_call(torch, lambda: sp.lower(Ad, sr))
    t_full = timed_call(torch, lambda: sp.offdiag(Ad, Ad, sr))
    side["lower_ms"] = t_low
    side["offdiag_AA_ms"] = t_full
    side["lower_over_offdiag_AA"] = t_low / t_full
    # the two-phase use: a plan, then products for new values of the pattern
    plan, C0 = sp.lower_plan(Ad, sr)
    del C0
    side["plan_execute_ms"] = timed_call(torch, lambda: plan.execute(Ad.values))
    plan.close()
    # Y = C X from C_L alone (Eq. (spmv) / (spgemm)): algorithmic bytes are
    # C_L read once, X read once and Y written once
    C = sp.lower(Ad, sr)
    xdt = torch.float64 if sr in ("f64", "count") else torch.float32
    vC = 8 if sr == "f64" else 4
    gen = torch.Generator(device=dev).manual_seed(7)
    for k in (1, 8):
        X = torch.randn((C.nrows, k), dtype=xdt, device=dev, generator=gen)
        ms = timed_call(torch, lambda: sp.symm(C, X, sr))
        B = 8 * (C.nrows + 1) + C.nnz * (4 + vC) + 2 * C.nrows * k * X.element_size()
        side[f"symm_k{k}_ms"] = ms
        side[f"symm_k{k}_GBs"] = B / (ms / 1e3) / 1e9
        side[f"symm_k{k}_frac"] = B / (ms / 1e3) / 1e9 / HBM_PEAK_GBS
        del X
    del C
    # two stages (the columns of A split in half) accumulated one at a time
    # (Sec. III-A, C = sum over stages of SYRK(A_s)); Jaccard values do not
    # add, so that workload accumulates its overlap counts
    A = w["A"]
    sa = "count" if sr == "jaccard" else sr
    vdt = {"f64": np.float64, "f32": np.float32}.get(sa)
    half = A.ncols // 2
    rows = np.repeat(np.arange(A.nrows), np.diff(A.row_ptr))
    stages = []
    for lo, hi in ((0, half), (half, A.ncols)):
        sel = (A.col_idx >= lo) & (A.col_idx < hi)
        rp = np.zeros(A.nrows + 1, dtype=np.int64)
        np.cumsum(np.bincount(rows[sel], minlength=A.nrows), out=rp[1:])
        vals = A.values[sel].astype(vdt) if (vdt is not None and A.values is not None) else None
        S = type(A)(A.nrows, hi - lo, rp, (A.col_idx[sel] - lo).astype(np.int32), vals)
        stages.append(sp.DeviceCSR.from_host(S, dev, vdt))
    Afull = sp.DeviceCSR.from_host(A if vdt else A.with_values(None), dev, vdt)
    C1 = sp.lower(stages[0], sa)
    side["stage_semiring"] = sa
    side["stage1_lower_ms"] = timed_call(torch, lambda: sp.lower(stages[0], sa))
    side["stage2_accumulate_ms"] = timed_call(torch, lambda: sp.lower_accumulate(C1, stages[1], sa))
    side["one_shot_lower_ms"] = timed_call(torch, lambda: sp.lower(Afull, sa))
    del C1, stages, Afull
    if Bd is not None:
        side["offdiag_ms"] = timed_call(torch, lambda: sp.offdiag(Ad, Bd, sr))
        side["half_top_ms"] = timed_call(torch, lambda: sp.offdiag_half(Ad, Bd, "top", sr))
        side["half_right_ms"] = timed_call(torch, lambda: sp.offdiag_half(Ad, Bd, "right", sr))
    print(f"[bench] side: {side}", file=sys.stderr, flush=True)
    return side


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1",
                          "gpus_requested": args.gpus}))
        sys.exit(2)
    import torch
    import paper_2608_09713_amd as sp
    from paper_2608_09713_amd import workloads as W

    sp.library()  # fails loudly if the HIP library is not built
    dev = "cuda:0"
    t0 = time.perf_counter()
    w = W.make(args.workload, args.seed, args.scale_shift)
    A = w["A"]
    sr = w["semiring"]
    print(f"[bench] generated {args.workload} m={A.nrows} n={A.ncols} nnz={A.nnz} in "
          f"{time.perf_counter() - t0:.1f}s", file=sys.stderr, flush=True)
    vdt = {"f64": np.float64, "f32": np.float32}.get(sr)
    Ad = sp.DeviceCSR.from_host(A if vdt else A.with_values(None), dev, vdt)
    Bd = sp.DeviceCSR.from_host(w["B"] if vdt else w["B"].with_values(None), dev, vdt) if "B" in w else None
    F_L, n_ne = column_stats(A)

    def step():
        C = sp.lower(Ad, sr)
        st = sp.stats()
        M = sp.mirror(C, sr) if "mirror" in w["ops"] else None
        O = sp.offdiag(Ad, Bd, sr) if "offdiag" in w["ops"] else None
        return C, st, M, O

    for _ in range(args.warmup):
        out = step()
        del out
    torch.cuda.synchronize()

    if args.copy_calibration:
        src = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        src.fill_(1)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    # The phase breakdown comes from untimed steps with events around every
    # phase (each recorded event idles the device for a few microseconds);
    # the timed steps then record events around the dominant one-kernel phase
    # only, which gives its roofline.
    survey = max(1, min(args.steps, 3))
    sp.timing_begin()
    for _ in range(survey):
        out = None
        out = step()
    torch.cuda.synchronize()
    phases = sp.timing_end()
    C, st, M, O = out
    del out
    sz = {"m": A.nrows, "nnz_A": A.nnz, "nnz_C": C.nnz, "csc_entries": st["csc_entries"],
          "ngroups": (A.ncols + (1 << st["group_shift"]) - 1) >> st["group_shift"], "n_ne": n_ne,
          "heavy_rows": st["heavy_rows"], "heavy_entries": st["heavy_entries"],
          "heavy_nnz_out": st["heavy_nnz_out"], "packed_staging": st["packed_staging"]}

    def kernel_roof(k, ph, steps):
        ms, n = ph[k]
        ab = alg_bytes_phase(k, sz, sr)
        if not (n and ab):
            return None
        ach = ab / (ms / n / 1e3) / 1e9
        return {"avg_ms": ms / n, "ms_per_step": ms / steps, "alg_bytes_per_launch": ab, "achieved_GBs": ach,
                "frac": ach / HBM_PEAK_GBS}

    # every one-kernel phase's figure (from the survey), and the dominant one
    kernel_roofs = {}
    for k in SINGLE_KERNEL_PHASES:
        if k not in phases or k == "light_numeric" and sz["m"] == sz["heavy_rows"]:
            continue
        kr = kernel_roof(k, phases, survey)
        if kr:
            kernel_roofs[k] = kr
    dom = max(kernel_roofs, key=lambda k: kernel_roofs[k]["ms_per_step"]) if kernel_roofs else None
    del C, M, O

    sp.timing_begin([dom] if dom else [])
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    last = None
    for _ in range(args.steps):
        last = None
        last = step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    timed_phases = sp.timing_end()
    C, st, M, O = last
    ms_step = (t1 - t0) * 1e3 / args.steps
    t_step = ms_step / 1e3
    flops = 2 * F_L
    value = flops / t_step / 1e9
    mirror_nnz = M.nnz if M is not None else None
    B_alg = whole_call_bytes(sz, sr, mirror_nnz)

    roof = None
    if dom and dom in timed_phases:
        kernel_roofs[dom] = kernel_roof(dom, timed_phases, args.steps)
        kr = kernel_roofs[dom]
        roof = {"bound": "hbm", "achieved": kr["achieved_GBs"], "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": kr["frac"], "traffic": traffic_from_profiles(dom, args.workload), "kernel": dom,
                "kernel_avg_ms": kr["avg_ms"], "alg_bytes_per_launch": kr["alg_bytes_per_launch"]}
    phase_ms = {k: v[0] / v[1] for k, v in phases.items()}          # per launch of the phase
    phase_ms_step = {k: v[0] / survey for k, v in phases.items()}  # per step (all its launches)

    line = {
        "metric": METRIC,
        "value": value,
        "unit": "GFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": {"f64": "f64", "f32": "f32 in, f64 accumulate", "count": "i32",
                  "jaccard": "i32 counts, f32 Jaccard"}[sr],
        "data": "synthetic (seeded generator)",
        "config": {"workload": f"{args.workload}: {W.WORKLOADS[args.workload]}" +
                               (f" (scaled down by 2^{args.scale_shift})" if args.scale_shift else ""),
                   "nrows": A.nrows, "ncols": A.ncols, "nnz_A": A.nnz, "F_L": F_L, "nnz_C_L": C.nnz,
                   "ops": w["ops"], "seed": args.seed},
        "nnz_per_s": C.nnz / t_step,
        "hbm_roofline_whole_call": {"B_alg": B_alg, "achieved_GBs": B_alg / t_step / 1e9,
                                    "frac": B_alg / t_step / 1e9 / HBM_PEAK_GBS},
        "roofline": roof,
        "kernel_rooflines": kernel_roofs,
        "phase_ms": phase_ms,
        "phase_ms_per_step": phase_ms_step,
        "library_stats": st,
        "kernel_source_hash": kernel_source_hash(),
    }
    if mirror_nnz is not None:
        line["config"]["nnz_C_full"] = mirror_nnz
    if O is not None:
        line["config"]["nnz_offdiag"] = O.nnz
    del C, M, O, last
    torch.cuda.empty_cache()
    if not args.no_side:
        line["side"] = side_measurements(sp, torch, dev, Ad, Bd, sr, w, B_alg / t_step / 1e9)
        torch.cuda.empty_cache()
    if not args.no_cpu_baseline:
        print("[bench] oracle on a row sample ...", file=sys.stderr, flush=True)
        line["cpu_baseline"] = cpu_baseline(A, sr, F_L, args.seed, args.cpu_rows)
    else:
        line["cpu_baseline"] = None
    if args.cpu_full:
        print("[bench] oracle over every row ...", file=sys.stderr, flush=True)
        line["cpu_full"] = cpu_full(A, sr, args.seed, skip_single=F_L > 2e9)
    s = json.dumps(line)
    print(s, flush=True)
    if args.json_out:
        with open(args.json_out, "w") as f:
            f.write(s + "\n")


if __name__ == "__main__":
    main()
