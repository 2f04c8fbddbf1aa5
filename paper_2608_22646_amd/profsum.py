"""Summaries of rocprofv3 CSV output for profiles/ (kernel times, HBM counters).

  python -m paper_2608_22646_amd.profsum stats <kernel_stats.csv> <command> > profiles/<name>.txt
  python -m paper_2608_22646_amd.profsum traffic <fetch.csv> <write.csv> <copy_fetch.csv> <copy_write.csv>
        <kernel-name-substring> <copy-bytes> <command...> > profiles/<name>_traffic.txt

  python -m paper_2608_22646_amd.profsum util <counters.csv> <compute-units> <xcds> <command...> > profiles/<name>_util.txt

The traffic summary scales each counter (KiB per dispatch) by the ratio of the
known traffic of a plain copy kernel to what the same counter reads for it.
The utilisation summary reads one pass of GRBM_GUI_ACTIVE,
SQ_VALU_MFMA_BUSY_CYCLES, TA_TA_BUSY_sum, SQ_WAIT_INST_ANY and SQ_WAVE_CYCLES
and gives, per kernel, the clock (busy cycles over the dispatch's duration;
GRBM_GUI_ACTIVE is summed over the XCDs), the MFMA busy fraction (per SIMD,
four per compute unit), the texture-address busy fraction (per compute unit)
and the waves' share of cycles spent waiting.
"""
import csv
import hashlib
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))


def short(name, n=110):
    name = name.replace("dllm::(anonymous namespace)::", "").replace("(anonymous namespace)::", "")
    return name if len(name) <= n else name[:n - 3] + "..."


def stats(path, command):
    rows = list(csv.DictReader(open(path)))
    rows.sort(key=lambda r: -float(r["TotalDurationNs"]))
    tot = sum(float(r["TotalDurationNs"]) for r in rows)
    print(f"# rocprofv3 kernel statistics\n# command: {command}\n")
    print(f"{'share':>6} {'calls':>7} {'avg_us':>10} {'min_us':>9} {'max_us':>9}  kernel")
    for r in rows[:25]:
        print(f"{100 * float(r['TotalDurationNs']) / tot:5.1f}% {int(r['Calls']):7d} {float(r['AverageNs']) / 1e3:10.1f} "
              f"{float(r['MinNs']) / 1e3:9.1f} {float(r['MaxNs']) / 1e3:9.1f}  {short(r['Name'])}")


def per_dispatch(path, substr):
    vals = [float(r["Counter_Value"]) for r in csv.DictReader(open(path)) if substr in r["Kernel_Name"]]
    return sum(vals) / len(vals), len(vals)


def copy_reading(path):
    vals = [float(r["Counter_Value"]) for r in csv.DictReader(open(path)) if "copyBuffer" in r["Kernel_Name"]
            or "copy" in r["Kernel_Name"].lower() and "Fill" not in r["Kernel_Name"]]
    return max(vals)


def traffic(fetch, write, cfetch, cwrite, substr, copy_bytes, command):
    f_kib, nf = per_dispatch(fetch, substr)
    w_kib, nw = per_dispatch(write, substr)
    exp_kib = copy_bytes / 1024.0
    ff = exp_kib / copy_reading(cfetch)
    fw = exp_kib / copy_reading(cwrite)
    tb = (f_kib * ff + w_kib * fw) * 1024.0
    # the source the counted kernel is built from, hashed so that a reader of
    # the summary can tell when the kernel has changed since
    name, fname = (("head", "k_head_bf16.hip") if "head_stream" in substr else
                   ("misc", "k_misc.hip") if "rmsnorm" in substr else ("gemm", "k_gemm_bf16.hip"))
    src = os.path.join(HERE, "csrc", fname)
    sha = hashlib.sha256(open(src, "rb").read()).hexdigest()
    print(f"# HBM traffic of one launch from rocprofv3 --pmc counters\n# command: {command}")
    print(f"# kernel: launches whose name contains '{substr}'")
    print(f"# calibration: a plain copy of {copy_bytes} bytes reads FETCH_SIZE {copy_reading(cfetch):.0f} KiB and "
          f"WRITE_SIZE {copy_reading(cwrite):.0f} KiB (expected {exp_kib:.0f} KiB each)")
    print(f"fetch_kib_per_dispatch={f_kib:.1f}")
    print(f"write_kib_per_dispatch={w_kib:.1f}")
    print(f"dispatches={nf}")
    print(f"fetch_scale={ff:.4f}")
    print(f"write_scale={fw:.4f}")
    print(f"traffic_bytes_per_launch={tb:.0f}")
    print(f"{name}_source_sha256={sha}")


def util(path, cus, xcds, command):
    import collections
    import statistics
    keys = ("gemm_wd_kernel", "gemm_bf16_kernel", "gemm_rows_kernel", "attn_", "head_")
    per = collections.defaultdict(lambda: collections.defaultdict(list))
    dur = collections.defaultdict(dict)
    for r in csv.DictReader(open(path)):
        name = r["Kernel_Name"]
        if not any(k in name for k in keys):
            continue
        k = short(name, 400).split("(")[0]
        per[k][r["Counter_Name"]].append(float(r["Counter_Value"]))
        dur[k][r.get("Dispatch_Id", len(dur[k]))] = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
    print(f"# MFMA and texture-address utilisation per kernel from one rocprofv3 --pmc pass\n# command: {command}")
    print(f"# per dispatch, with cycles = GRBM_GUI_ACTIVE / {xcds} XCDs: clock = cycles / duration; mfma_busy = "
          f"SQ_VALU_MFMA_BUSY_CYCLES / (cycles x {cus} CUs x 4 SIMDs); ta_busy = TA_TA_BUSY_sum / (cycles x {cus}); "
          f"wait = SQ_WAIT_INST_ANY / SQ_WAVE_CYCLES\n")
    print(f"{'dispatches':>10} {'us':>8} {'GHz':>6} {'mfma_busy':>10} {'ta_busy':>8} {'wait':>6}  kernel")
    rows = []
    for k, c in per.items():
        if not all(n in c for n in ("GRBM_GUI_ACTIVE", "SQ_VALU_MFMA_BUSY_CYCLES", "TA_TA_BUSY_sum",
                                    "SQ_WAIT_INST_ANY", "SQ_WAVE_CYCLES")):
            continue
        mean = {n: sum(v) / len(v) for n, v in c.items()}
        us = statistics.median(dur[k].values())
        cyc = mean["GRBM_GUI_ACTIVE"] / xcds
        rows.append((len(dur[k]) * us, len(dur[k]), us, cyc / (us * 1e3),
                     mean["SQ_VALU_MFMA_BUSY_CYCLES"] / (cyc * cus * 4), mean["TA_TA_BUSY_sum"] / (cyc * cus),
                     mean["SQ_WAIT_INST_ANY"] / mean["SQ_WAVE_CYCLES"], k))
    for _, n, us, ghz, mf, ta, wt, k in sorted(rows, reverse=True):
        print(f"{n:10d} {us:8.1f} {ghz:6.2f} {mf:10.3f} {ta:8.3f} {wt:6.3f}  {short(k)}")


if __name__ == "__main__":
    if sys.argv[1] == "stats":
        stats(sys.argv[2], " ".join(sys.argv[3:]))
    elif sys.argv[1] == "traffic":
        traffic(*sys.argv[2:6], sys.argv[6], int(sys.argv[7]), " ".join(sys.argv[8:]))
    elif sys.argv[1] == "util":
        util(sys.argv[2], int(sys.argv[3]), int(sys.argv[4]), " ".join(sys.argv[5:]))
    else:
        raise SystemExit(__doc__)
