"""Turns rocprofv3 output of ``bench.py --steps-only`` into the short text
summaries kept under ``profiles/``.

    python profile_summary.py stats <kernel_stats.csv> <out.md> <command...>
    python profile_summary.py traffic <fetch.csv> <write.csv> \\
        <copy_fetch.csv> <copy_write.csv> <copy_mib> <kernel> <out.txt> <command...>

    python profile_summary.py counters <out.md> <n_cu> <n_xcd> \\
        <pass1.csv> [<pass2.csv> ...] -- <command...>

The traffic summary scales FETCH_SIZE and WRITE_SIZE (KiB per dispatch) by
what the same counters read for a plain device copy of known size, and
records the hash of the kernel sources it was taken on.  The counter summary
gives every counter's mean per dispatch for each kernel, and the derived
ratios: MFMA busy (SQ_VALU_MFMA_BUSY_CYCLES over GRBM_GUI_ACTIVE times four
SIMDs per CU), and the shares of wave cycles spent waiting or issuing LDS,
VALU and vector-memory instructions.
"""
from __future__ import annotations

import collections
import csv
import hashlib
import os
import sys

ROOT = os.path.dirname(os.path.abspath(__file__))


def sources_of(kernel=None):
    """The source files a kernel is built from (the linear-attention kernels
    by default)."""
    if kernel and kernel.startswith("k_logp"):
        return ("logp.hip",)
    if kernel and kernel.startswith("k_conv"):
        return ("conv.hip",)
    if kernel and kernel.startswith("k_attn"):
        return ("attn.hip", "la_common.hpp")
    if kernel and kernel.startswith("k_kda"):
        return ("kda.hip",)
    return ("la.hip", "la_common.hpp")


def source_sha(kernel=None):
    h = hashlib.sha256()
    for name in sources_of(kernel):
        with open(os.path.join(ROOT, "paper_2608_28158_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def short(name):
    n = name.split("(")[0]
    for key in ("k_bwd_revorder", "k_bwd_fwdorder", "k_blocksum", "k_fwd_blockscan",
                "k_fwd_block", "k_bwd_blockscan", "k_dg_carry", "k_gather", "k_scatter_add",
                "k_replay_reduce", "k_logp_lse", "k_logp_gather", "k_logp_rowsum",
                "k_logp_grad", "k_logp_onehot", "k_conv_fwd", "k_conv_bwd",
                "k_conv_dw_sum", "k_attn_fwd", "k_attn_dq", "k_attn_dkdv", "k_attn_delta",
                "k_attn_gather", "k_attn_scatter", "k_kda_prep", "k_kda_seq", "k_kda_out",
                "k_kda_bwd_prep", "k_kda_bwd_prod", "k_kda_bwd_tm", "k_kda_bwd_local", "k_kda_reduce",
                "k_kda_bank_add"):
        if key in name:
            return key
    return n.replace("void ", "")[:48]


def stats(src, out, cmd):
    rows = list(csv.DictReader(open(src)))
    tot = sum(float(r["TotalDurationNs"]) for r in rows)
    lines = ["# rocprofv3 kernel statistics", "", "Command:", "", "    " + " ".join(cmd), "",
             f"Kernel source hashes: la.hip + la_common.hpp {source_sha()}, "
             f"logp.hip {source_sha('k_logp')}, conv.hip {source_sha('k_conv')}, "
             f"attn.hip + la_common.hpp {source_sha('k_attn')}, kda.hip {source_sha('k_kda')}", "",
             "| kernel | calls | total ms | avg us | min us | max us | share |",
             "|---|---|---|---|---|---|---|"]
    for r in sorted(rows, key=lambda r: -float(r["TotalDurationNs"])):
        lines.append("| %s | %s | %.3f | %.1f | %.1f | %.1f | %.1f%% |" % (
            short(r["Name"]), r["Calls"], float(r["TotalDurationNs"]) / 1e6,
            float(r["AverageNs"]) / 1e3, float(r["MinNs"]) / 1e3, float(r["MaxNs"]) / 1e3,
            100 * float(r["TotalDurationNs"]) / tot))
    open(out, "w").write("\n".join(lines) + "\n")


def per_kernel(path, counter):
    agg, disp = collections.defaultdict(float), collections.defaultdict(set)
    for r in csv.DictReader(open(path)):
        if r["Counter_Name"] != counter:
            continue
        k = short(r["Kernel_Name"])
        agg[k] += float(r["Counter_Value"])
        disp[k].add(r["Dispatch_Id"])
    return {k: agg[k] / len(disp[k]) for k in agg}


def traffic(fetch, write, cfetch, cwrite, copy_mib, kernel, out, cmd):
    """HBM bytes per dispatch of one kernel, FETCH_SIZE and WRITE_SIZE each
    scaled by what it reads for a plain copy of copy_mib MiB."""
    f, w = per_kernel(fetch, "FETCH_SIZE"), per_kernel(write, "WRITE_SIZE")
    cf = max(v for k, v in per_kernel(cfetch, "FETCH_SIZE").items() if "copy" in k.lower())
    cw = max(v for k, v in per_kernel(cwrite, "WRITE_SIZE").items() if "copy" in k.lower())
    kib = float(copy_mib) * 1024
    sf, sw = kib / cf, kib / cw
    hbm = (f[kernel] * sf + w[kernel] * sw) * 1024
    lines = [f"# HBM traffic of {kernel} (rocprofv3 --pmc, per dispatch)",
             "command: " + " ".join(cmd),
             f"copy probe: {copy_mib} MiB read and written; FETCH_SIZE reads {cf:.0f} KiB "
             f"(scale {sf:.3f}), WRITE_SIZE reads {cw:.0f} KiB (scale {sw:.3f})",
             f"fetch_kib_per_launch: {f[kernel]:.0f}",
             f"write_kib_per_launch: {w[kernel]:.0f}",
             f"hbm_bytes_per_launch: {hbm:.0f}",
             f"sources: {' + '.join(sources_of(kernel))}",
             f"source_sha: {source_sha(kernel)}"]
    open(out, "w").write("\n".join(lines) + "\n")


def counters(out, n_cu, n_xcd, paths, cmd):
    """Per-kernel means per dispatch of every counter in the given pass
    files, with derived ratios.  GRBM_GUI_ACTIVE reads as the sum over the
    XCDs, so the MFMA busy share is SQ_VALU_MFMA_BUSY_CYCLES over
    GRBM_GUI_ACTIVE / n_xcd * n_cu * 4 SIMDs; the bf16 (fp32) MFMA rate is
    SQ_INSTS_VALU_MFMA_MOPS_BF16 (_F32) * 512 FLOP over the dispatch duration."""
    vals = collections.defaultdict(dict)   # kernel -> counter -> mean per dispatch
    dur = collections.defaultdict(list)    # kernel -> dispatch durations (ns)
    for path in paths:
        agg = collections.defaultdict(float)
        disp = collections.defaultdict(set)
        seen = set()
        for r in csv.DictReader(open(path)):
            k = short(r["Kernel_Name"])
            agg[(k, r["Counter_Name"])] += float(r["Counter_Value"])
            disp[(k, r["Counter_Name"])].add(r["Dispatch_Id"])
            if (k, r["Dispatch_Id"]) not in seen:
                seen.add((k, r["Dispatch_Id"]))
                dur[k].append(float(r["End_Timestamp"]) - float(r["Start_Timestamp"]))
        for (k, c), v in agg.items():
            vals[k][c] = v / len(disp[(k, c)])
    names = sorted({c for d in vals.values() for c in d})
    kernels = sorted(vals, key=lambda k: -vals[k].get("SQ_WAVE_CYCLES", vals[k].get("GRBM_GUI_ACTIVE", 0)))
    lines = ["# rocprofv3 counters per kernel (mean per dispatch)", "", "Command (one run per pass):",
             "", "    " + " ".join(cmd), "",
             "Kernel source hashes: " + ", ".join(sorted({" + ".join(sources_of(k)) + " " + source_sha(k)
                                                         for k in vals if k.startswith("k_")})), "",
             f"MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE / {n_xcd} XCDs x {n_cu} CUs "
             "x 4 SIMDs); MFMA rates = SQ_INSTS_VALU_MFMA_MOPS_BF16 (_F32) x 512 FLOP / dispatch "
             "duration (peaks 2500 and 157.3 TFLOP/s); wait, issue and LDS shares are of SQ_WAVE_CYCLES "
             "(all in quad-cycles); LDS busy = SQ_LDS_IDX_ACTIVE / (GRBM_GUI_ACTIVE / "
             f"{n_xcd} x {n_cu}).", ""]

    def ratio(d, a, b, f=1.0):
        return "%.1f%%" % (100.0 * d[a] / (d[b] * f)) if a in d and d.get(b) else "-"

    lines += ["| kernel | MFMA busy | bf16 MFMA TFLOP/s | fp32 MFMA TFLOP/s | LDS busy | LDS conflict share | "
              "wait any | VALU issue | LDS issue |",
              "|---|---|---|---|---|---|---|---|---|"]

    def rate(d, k, counter):
        if not d.get(counter) or not dur.get(k):
            return "-"
        ns = sum(dur[k]) / len(dur[k])
        return "%.1f" % (d[counter] * 512 / ns / 1e3)

    for k in kernels:
        d = vals[k]
        lines.append("| %s | %s | %s | %s | %s | %s | %s | %s | %s |" % (
            k, ratio(d, "SQ_VALU_MFMA_BUSY_CYCLES", "GRBM_GUI_ACTIVE", 4.0 * n_cu / n_xcd),
            rate(d, k, "SQ_INSTS_VALU_MFMA_MOPS_BF16"), rate(d, k, "SQ_INSTS_VALU_MFMA_MOPS_F32"),
            ratio(d, "SQ_LDS_IDX_ACTIVE", "GRBM_GUI_ACTIVE", 1.0 * n_cu / n_xcd),
            ratio(d, "SQ_LDS_BANK_CONFLICT", "SQ_LDS_IDX_ACTIVE"),
            ratio(d, "SQ_WAIT_ANY", "SQ_WAVE_CYCLES"),
            ratio(d, "SQ_ACTIVE_INST_VALU", "SQ_WAVE_CYCLES"),
            ratio(d, "SQ_ACTIVE_INST_LDS", "SQ_WAVE_CYCLES")))
    lines += ["", "Raw means per dispatch:", "", "| counter | " + " | ".join(kernels) + " |",
              "|---" * (len(kernels) + 1) + "|"]
    for c in names:
        lines.append("| %s | " % c + " | ".join(
            "%.4g" % vals[k][c] if c in vals[k] else "-" for k in kernels) + " |")
    open(out, "w").write("\n".join(lines) + "\n")


if __name__ == "__main__":
    if sys.argv[1] == "stats":
        stats(sys.argv[2], sys.argv[3], sys.argv[4:])
    elif sys.argv[1] == "counters":
        rest = sys.argv[5:]
        cut = rest.index("--")
        counters(sys.argv[2], int(sys.argv[3]), int(sys.argv[4]), rest[:cut], rest[cut + 1:])
    else:
        traffic(*sys.argv[2:9], sys.argv[9:])
