"""Summaries of rocprofv3 output for the committed profiles.

kernels   rocprofv3 --kernel-trace --stats: a markdown table per kernel.
traffic   two rocprofv3 --pmc runs (FETCH_SIZE, then WRITE_SIZE; KiB per
          dispatch): each counter is scaled by what it reads for copy16, a
          plain copy kernel of known size in the same run, and the HBM bytes
          per launch of every kernel family of the stage are totalled. The
          record it prints carries a hash of the kernel sources it was
          measured on; bench.py reports the traffic only while the sources
          still hash the same.

usage: python -m paper_2606_07881_amd.profile_summary kernels STATS_CSV
       python -m paper_2606_07881_amd.profile_summary traffic FETCH_CSV WRITE_CSV [COPY_BYTES]
"""
import csv
import collections
import hashlib
import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
COPY_KERNEL = "copy16"
COPY_BYTES = 256 * 2 ** 20   # read and written by one copy16 dispatch of stage_bench --copy-probe

# Kernel families of the stage library (paci_kernel_family_name) and the
# kernels (demangled name fragments) one launch of the family runs.
FAMILIES = {
    "gemm_fwd": ["gemm_pipe_kernel<bool _Accum, bool, E, true, 1", "gemm_pipe_kernel<bool _Accum, bool, E, true, 2",
                 "gemm_pipe_kernel<bool _Accum, bool, E, true, 3"],
    "gemm_dgrad": ["gemm_pipe_kernel<bool _Accum, bool, E, true, 0", "gemm_pipe_kernel<bool _Accum, bool, E, true, 4",
                   "gemm_pipe_kernel<bool _Accum, bool, E, false, 0", "gemm_pipe_kernel<bool _Accum, bool, E, false, 4"],
    "gemm_wgrad_acc": ["gemm_pipe_kernel<float, false, false, 5", "gemm_pipe_kernel<float, false, false, 6",
                       "gemm_pipe_kernel<float, false, false, 0"],
    "attn_fwd": ["attn_fwd_ring_kernel"],
    "attn_bwd": ["attn_pairs_kernel", "attn_bwd_ring_kernel"],
    "layernorm_fwd": ["ln_fwd_kernel"],
    "layernorm_bwd": ["ln_bwd_kernel", "colsum_atomic_kernel<bool _Accum, bool, E>"],
    "bias_grad": ["colsum_atomic_kernelIDF16bLb0E"],
    "adamw": ["adamw_kernel", "guard_kernel", "guard_ranges_kernel", "ctl_kernel", "transpose16_kernel"],
    "copy": ["fill_f32_kernel"],
}
# families whose launch runs each of its kernels once; every other family runs
# one of its kernels (an epilogue or shape variant) per launch
SEQUENCES = {"attn_bwd", "layernorm_bwd"}
# families whose launch can run a second kernel of another tile shape (the
# grouped weight gradients: a 256 x 256 part, then the 256 x 128 rest): a launch
# is counted once, by its 256 x 128 kernel when the run has one
SPLIT_LAUNCH = {"gemm_wgrad_acc": "PipeTile<256, 128"}


def sources_sha256():
    """Hash of every kernel source of the library (csrc/*.hip, *.hpp), in name order."""
    h = hashlib.sha256()
    for name in sorted(os.listdir(CSRC)):
        if name.endswith((".hip", ".hpp")) and name != "stage_bench.hip":
            h.update(name.encode())
            with open(os.path.join(CSRC, name), "rb") as f:
                h.update(f.read())
    return h.hexdigest()


def family_of(kernel):
    for fam, frags in FAMILIES.items():
        if any(fr in kernel for fr in frags):
            return fam
    return None


def kernels_md(stats_csv, top=24):
    rows = list(csv.DictReader(open(stats_csv)))
    rows.sort(key=lambda r: -float(r["TotalDurationNs"]))
    out = ["| kernel | family | calls | total ms | avg us | min us | max us | % |", "|---|---|---|---|---|---|---|---|"]
    for r in rows[:top]:
        name = r["Name"].replace("|", "/")
        out.append(f"| `{name[:130]}` | {family_of(name) or '-'} | {r['Calls']} | {float(r['TotalDurationNs']) / 1e6:.1f} | "
                   f"{float(r['AverageNs']) / 1e3:.1f} | {float(r['MinNs']) / 1e3:.1f} | {float(r['MaxNs']) / 1e3:.1f} | "
                   f"{float(r['Percentage']):.2f} |")
    return "\n".join(out)


def _per_kernel(path):
    agg = collections.defaultdict(list)
    for r in csv.DictReader(open(path)):
        agg[r["Kernel_Name"]].append(float(r["Counter_Value"]))
    return agg


def traffic(fetch_csv, write_csv, copy_bytes=COPY_BYTES):
    """Returns (markdown, record). Byte counts per dispatch are scaled so that
    copy16 reads and writes copy_bytes; a family's bytes per launch are the
    bytes of all its dispatches over its launches (the dispatches of its first
    kernel for a SEQUENCES family, all its dispatches otherwise)."""
    f, w = _per_kernel(fetch_csv), _per_kernel(write_csv)
    copy = [k for k in f if COPY_KERNEL in k]
    if not copy:
        raise ValueError("no copy16 dispatch in the counter run (run stage_bench with --copy-probe)")
    f_scale = copy_bytes / (1024.0 * sum(f[copy[0]]) / len(f[copy[0]]))
    w_scale = copy_bytes / (1024.0 * sum(w[copy[0]]) / len(w[copy[0]]))
    fams = collections.defaultdict(float)
    launches = collections.defaultdict(int)
    split = {fam for fam, tag in SPLIT_LAUNCH.items() if any(tag in k and family_of(k) == fam for k in f)}
    lines = [f"Scale factors from {COPY_KERNEL} ({copy_bytes / 2 ** 20:.0f} MiB read and written per dispatch): "
             f"FETCH_SIZE x {f_scale:.3f}, WRITE_SIZE x {w_scale:.3f}.", "",
             "| kernel | family | dispatches | FETCH_SIZE KiB/dispatch | WRITE_SIZE KiB/dispatch | HBM MiB/dispatch (scaled) |",
             "|---|---|---|---|---|---|"]
    for k in sorted(f, key=lambda k: -sum(f[k]) / len(f[k])):
        fk = sum(f[k]) / len(f[k])
        wk = sum(w.get(k, [0.0])) / max(len(w.get(k, [])), 1)
        b = 1024.0 * (fk * f_scale + wk * w_scale)
        fam = family_of(k)
        if fam:
            fams[fam] += b * len(f[k])
            if fam in split:
                if SPLIT_LAUNCH[fam] in k:
                    launches[fam] += len(f[k])
            elif fam not in SEQUENCES or FAMILIES[fam][0] in k:
                launches[fam] += len(f[k])
        lines.append(f"| `{k.replace('|', '/')[:130]}` | {fam or '-'} | {len(f[k])} | {fk:.1f} | {wk:.1f} | {b / 2 ** 20:.1f} |")
    record = {"sources_sha256": sources_sha256(), "fetch_scale": f_scale, "write_scale": w_scale,
              "bytes_per_launch": {k: round(v / max(launches[k], 1)) for k, v in sorted(fams.items())}}
    return "\n".join(lines), record


SIMD_NUM = 256 * 4   # MI355X: 256 CUs of 4 SIMDs
XCC_NUM = 8          # GRBM_GUI_ACTIVE comes summed over the 8 XCDs (each counts the same cycles)


def mfma(counters_csv):
    """Per-kernel MFMA busy fraction SQ_VALU_MFMA_BUSY_CYCLES (summed over
    SIMDs) / (GPU-active cycles x SIMD_NUM), GPU-active cycles being
    GRBM_GUI_ACTIVE / XCC_NUM; the executed bf16 MFMA FLOP
    (SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512) and their rate against the dense
    peak of 1024 FLOP per SIMD and cycle; and the same per family (summed
    over its dispatches). Returns markdown."""
    rows = collections.defaultdict(lambda: collections.defaultdict(list))
    for r in csv.DictReader(open(counters_csv)):
        rows[r["Kernel_Name"]][r["Counter_Name"]].append(float(r["Counter_Value"]))
    need = ("SQ_VALU_MFMA_BUSY_CYCLES", "GRBM_GUI_ACTIVE", "SQ_INSTS_VALU_MFMA_MOPS_BF16")
    fam_busy, fam_active, fam_flop = (collections.defaultdict(float) for _ in range(3))
    lines = ["| kernel | family | dispatches | MFMA busy % | bf16 MFMA GFLOP / dispatch | GPU-active kcycles / dispatch |",
             "|---|---|---|---|---|---|"]
    order = sorted(rows, key=lambda k: -sum(rows[k].get("GRBM_GUI_ACTIVE", [0.0])))
    for k in order:
        c = rows[k]
        if any(n not in c for n in need):
            continue
        n = len(c["GRBM_GUI_ACTIVE"])
        busy, active, mops = sum(c[need[0]]), sum(c[need[1]]) / XCC_NUM, sum(c[need[2]])
        if mops == 0:
            continue
        fam = family_of(k)
        if fam:
            fam_busy[fam] += busy
            fam_active[fam] += active
            fam_flop[fam] += mops * 512
        lines.append(f"| `{k.replace('|', '/')[:130]}` | {fam or '-'} | {n} | {100 * busy / (active * SIMD_NUM):.1f} | "
                     f"{mops * 512 / n / 1e9:.1f} | {active / n / 1e3:.0f} |")
    lines += ["", "| family | MFMA busy % | executed bf16 MFMA FLOP per GPU-active cycle, fraction of the dense peak |",
              "|---|---|---|"]
    for fam in sorted(fam_busy, key=lambda f: -fam_active[f]):
        lines.append(f"| {fam} | {100 * fam_busy[fam] / (fam_active[fam] * SIMD_NUM):.1f} | "
                     f"{fam_flop[fam] / (fam_active[fam] * SIMD_NUM * 1024) * 100:.1f}% |")
    return "\n".join(lines)


def read_record(md_path):
    """The traffic record line of a committed summary, or None."""
    try:
        with open(md_path) as fh:
            for line in fh:
                if line.startswith("traffic-record: "):
                    return json.loads(line[len("traffic-record: "):])
    except OSError:
        return None
    return None


if __name__ == "__main__":
    if len(sys.argv) >= 3 and sys.argv[1] == "kernels":
        print(kernels_md(sys.argv[2]))
    elif len(sys.argv) >= 3 and sys.argv[1] == "mfma":
        print(mfma(sys.argv[2]))
    elif len(sys.argv) >= 4 and sys.argv[1] == "traffic":
        md, rec = traffic(sys.argv[2], sys.argv[3], float(sys.argv[4]) if len(sys.argv) > 4 else COPY_BYTES)
        print(md)
        print()
        print("traffic-record: " + json.dumps(rec))
    else:
        print(__doc__)
        sys.exit(2)
