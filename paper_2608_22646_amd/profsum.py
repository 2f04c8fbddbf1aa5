"""Summaries of rocprofv3 CSV output for profiles/ (kernel times, HBM counters).

  python -m paper_2608_22646_amd.profsum stats <kernel_stats.csv> <command> > profiles/<name>.txt
  python -m paper_2608_22646_amd.profsum traffic <fetch.csv> <write.csv> <copy_fetch.csv> <copy_write.csv>
        <kernel-name-substring> <copy-bytes> <command...> > profiles/<name>_traffic.txt

The traffic summary scales each counter (KiB per dispatch) by the ratio of the
known traffic of a plain copy kernel to what the same counter reads for it.
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


if __name__ == "__main__":
    if sys.argv[1] == "stats":
        stats(sys.argv[2], " ".join(sys.argv[3:]))
    elif sys.argv[1] == "traffic":
        traffic(*sys.argv[2:6], sys.argv[6], int(sys.argv[7]), " ".join(sys.argv[8:]))
    else:
        raise SystemExit(__doc__)
