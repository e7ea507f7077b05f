"""Summaries of rocprofv3 CSV output for the cold-start path (markdown on stdout).

  python -m paper_2503_17707_amd.profsum overlap DIR LABEL [GAP_MS]
      DIR from `rocprofv3 --kernel-trace --memory-copy-trace -f csv -d DIR -o ov
      -- python bench.py ...`: for every cold start in the run (a burst of
      host-to-device copies followed by the library's kernels), how much of the
      compute ran while weights were still being copied, and the compute tail
      left after the last copy.  Copies further apart than GAP_MS (default
      0.35) start a new load: raise it when staged copies of pageable blobs
      leave longer gaps inside one load.

  python -m paper_2503_17707_amd.profsum mfma DIR LABEL
      DIR from `rocprofv3 --pmc SQ_INSTS_VALU_MFMA_MOPS_F16 SQ_VALU_MFMA_BUSY_CYCLES
      SQ_BUSY_CU_CYCLES GRBM_GUI_ACTIVE -f csv -d DIR -o mf -- python bench.py ...`:
      per kernel, the MFMA work executed and the fraction of SIMD cycles the
      matrix units were busy.

  python -m paper_2503_17707_amd.profsum kernels DIR LABEL
      DIR from `rocprofv3 --kernel-trace --stats -f csv -d DIR -o bench -- python
      bench.py ...`: the per-kernel statistics, and the average duration per
      launch of each kernel kind with its split-K reduce counted in (the unit
      bench.py times with HIP events).

  python -m paper_2503_17707_amd.profsum traffic FETCH WRITE CAL_FETCH CAL_WRITE LABEL
      FETCH / WRITE from `rocprofv3 --pmc FETCH_SIZE` / `--pmc WRITE_SIZE -f csv
      -d DIR -o bench -- python bench.py ...`, CAL_* the same counters over
      `python bench.py --calibrate-copy-mib 1024` (a plain device copy of
      1 GiB, three times): each counter is scaled by what it reads for the
      copy, and the bytes of every dispatch of a kernel kind are divided by
      that kind's launches.  Ends with the block bench.py reads (bytes per
      launch, valid while the kernel sources keep the printed hash).

  python -m paper_2503_17707_amd.profsum stalls DIR_A DIR_B LABEL
      DIR_A from `rocprofv3 --pmc SQ_WAVE_CYCLES SQ_BUSY_CYCLES SQ_WAIT_ANY
      SQ_WAIT_INST_ANY SQ_ACTIVE_INST_ANY SQ_VALU_MFMA_BUSY_CYCLES SQ_ACTIVE_INST_LDS
      SQ_ACTIVE_INST_VMEM GRBM_GUI_ACTIVE -f csv -d DIR_A -o c -- python bench.py
      --workload W --gemm-reference`, DIR_B the same with SQ_WAIT_INST_LDS
      SQ_LDS_BANK_CONFLICT SQ_LDS_IDX_ACTIVE SQ_LDS_DATA_FIFO_FULL SQ_LDS_CMD_FIFO_FULL
      SQ_ACTIVE_INST_VALU SQ_ACTIVE_INST_SCA SQ_INSTS_LDS GRBM_GUI_ACTIVE: where the
      GEMM waves' cycles go, for this library's GEMM kernels (by tile and role)
      and the vendor library's, side by side.  With `bench.py --attention-only`
      runs instead, the same columns for the prefill attention kernels.

Only reads files; used to write the summaries kept with the profiles.
"""
import collections
import csv
import glob
import hashlib
import os
import re
import sys

N_XCD = 8           # GRBM_GUI_ACTIVE is summed over the 8 XCDs
N_SIMD = 256 * 4    # SQ_VALU_MFMA_BUSY_CYCLES is summed over every SIMD
GAP_NS = 350_000  # default: copies further apart start a new load (pinned loads: gaps < 0.25 ms)


def _one(d, pattern):
    files = glob.glob(os.path.join(d, pattern))
    if len(files) != 1:
        raise SystemExit("expected one %s in %s, found %d" % (pattern, d, len(files)))
    return files[0]


def kind_of(name):
    """Kernel family of a mangled kernel name (GEMM role from its template arguments)."""
    roles = {0: "gemm_qkv", 1: "gemm_o", 2: "gemm_fc1", 3: "gemm_fc2", 4: "lora_shrink"}
    m = re.search(r"gemm_kernelIDF16b?_((?:Li\d+E)+)", name) or \
        re.search(r"gemm_kernelIDF16_((?:Li\d+E)+)", name)
    if m:
        a = [int(x) for x in re.findall(r"Li(\d+)E", m.group(1))]
        return roles.get(a[5], "gemm")
    if "splitk_resid_ln_kernel" in name:
        return roles[int(re.search(r"splitk_resid_ln_kernelIDF16b?_Li(\d+)E", name).group(1))] + " reduce"
    if "tail_reduce_kernel" in name:
        return roles[int(re.search(r"tail_reduce_kernelIDF16b?_Li\d+ELi(\d+)E", name).group(1))] + " reduce"
    if "splitk_reduce_kernel" in name:
        return roles[int(re.search(r"splitk_reduce_kernelIDF16b?_Li\d+ELi(\d+)E", name).group(1))] + " reduce"
    m = re.search(r"gemv_kernelIDF16b?_Li(\d+)E", name)
    if m:  # decode steps: named by epilogue (o and fc2 share the residual one)
        return {0: "gemv_qkv", 1: "gemv_fc1", 2: "gemv_o_fc2", 3: "gemv_shrink"}[int(m.group(1))]
    if "decode_attention" in name:
        return "decode_attention"
    for k in ("attention", "layernorm", "lm_head", "argmax", "embed", "lora_pack", "lora_merge"):
        if k in name:
            return k
    return None


def _union(iv):
    out = []
    for s, e in sorted(iv):
        if out and s <= out[-1][1]:
            out[-1][1] = max(out[-1][1], e)
        else:
            out.append([s, e])
    return out


def _inter(u, lo, hi):
    return sum(max(0, min(e, hi) - max(s, lo)) for s, e in u)


def overlap(d, label, gap_ns=GAP_NS):
    copies = [(int(r["Start_Timestamp"]), int(r["End_Timestamp"]))
              for r in csv.DictReader(open(_one(d, "*memory_copy_trace.csv")))
              if r["Direction"].endswith("HOST_TO_DEVICE")]
    kernels = [(int(r["Start_Timestamp"]), int(r["End_Timestamp"]), r["Kernel_Name"])
               for r in csv.DictReader(open(_one(d, "*kernel_trace.csv")))]
    copies.sort()
    loads = []
    for s, e in copies:
        if loads and s - loads[-1][1] < gap_ns:
            loads[-1][1] = max(loads[-1][1], e)
            loads[-1][2] += 1
        else:
            loads.append([s, e, 1])
    rows = []
    for i, (cs, ce, n) in enumerate(loads):
        nxt = loads[i + 1][0] if i + 1 < len(loads) else float("inf")
        ends = [e for s, e, name in kernels if cs <= s < nxt and kind_of(name) == "argmax"]
        if not ends:
            continue  # a load with no prefill behind it (bandwidth measurement)
        end = min(ends)  # the first prefill after the load ends at its argmax
        ks = [(s, e) for s, e, name in kernels if cs <= s and e <= end and kind_of(name)]
        u = _union(ks)
        busy = sum(e - s for s, e in u)
        rows.append((n, (ce - cs) / 1e6, busy / 1e6, _inter(u, cs, ce) / max(busy, 1),
                     max(0, end - ce) / 1e6, (end - cs) / 1e6))
    out = ["# Copy / compute overlap during cold starts, %s\n" % label,
           "Each row is one cold start of the run (the first is the warm-up): host-to-device "
           "copies of the layer stream and the LoRA staging, then the prefill, whose kernels "
           "each wait for their layer's copy event.  Overlap = share of the prefill's kernel "
           "busy time that falls inside the copy window; tail = time from the last copy's end "
           "to the argmax's end.\n",
           "| cold start | copies | copy window ms | kernel busy ms | overlap | tail ms | "
           "first copy -> argmax ms |", "|---|---|---|---|---|---|---|"]
    for i, (n, win, busy, ov, tail, span) in enumerate(rows):
        out.append("| %d%s | %d | %.2f | %.2f | %.3f | %.2f | %.2f |" % (
            i, " (warm-up)" if i == 0 else "", n, win, busy, ov, tail, span))
    return "\n".join(out)


def mfma(d, label):
    per = collections.defaultdict(lambda: collections.defaultdict(list))
    dur = collections.defaultdict(dict)  # kind -> dispatch -> ns
    for r in csv.DictReader(open(_one(d, "*counter_collection.csv"))):
        k = kind_of(r["Kernel_Name"])
        if k:
            per[k][r["Counter_Name"]].append(float(r["Counter_Value"]))
            dur[k][r["Dispatch_Id"]] = int(r["End_Timestamp"]) - int(r["Start_Timestamp"])
    out = ["# MFMA work and matrix-unit busy fraction per kernel kind, %s\n" % label,
           "Counters per dispatch, averaged over the run's dispatches of each kind.  MFMA "
           "FLOPs = SQ_INSTS_VALU_MFMA_MOPS_F16 x 512.  Busy = SQ_VALU_MFMA_BUSY_CYCLES / "
           "(GRBM_GUI_ACTIVE / %d XCDs x %d SIMDs): the share of all SIMD cycles, over the "
           "dispatch, in which the matrix unit was busy.  Counter runs serialize dispatches, so "
           "launch gaps are absent here.  Clock = GRBM_GUI_ACTIVE / %d XCDs / the dispatch's "
           "duration: the sustained shader clock, read from the long dispatches (GRBM_GUI_ACTIVE also counts "
           "the counters' own start and stop, which dominates dispatches of a few microseconds and "
           "inflates their clock and deflates their busy share).\n" % (N_XCD, N_SIMD, N_XCD),
           "| kind | dispatches | MFMA GFLOP per dispatch | GPU cycles per dispatch | "
           "clock GHz | MFMA busy |", "|---|---|---|---|---|---|"]
    for k in sorted(per):
        c = per[k]
        if not c.get("GRBM_GUI_ACTIVE"):
            continue
        n = len(c["GRBM_GUI_ACTIVE"])
        mops = sum(c.get("SQ_INSTS_VALU_MFMA_MOPS_F16", [0])) / n
        busy = sum(c.get("SQ_VALU_MFMA_BUSY_CYCLES", [0])) / n
        gui = sum(c["GRBM_GUI_ACTIVE"]) / n / N_XCD
        ns = sum(dur[k].values()) / max(1, len(dur[k]))
        out.append("| %s | %d | %.3f | %.0f | %.2f | %.3f |" % (
            k, n, mops * 512 / 1e9, gui, gui / ns if ns else 0.0, busy / (gui * N_SIMD) if gui else 0.0))
    return "\n".join(out)


def source_sha256():
    """Hash of the kernel sources, as bench.py computes it."""
    here = os.path.dirname(os.path.abspath(__file__))
    h = hashlib.sha256()
    for f in sorted(glob.glob(os.path.join(here, "csrc", "*"))):
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def _base(kind):
    return kind[:-len(" reduce")] if kind and kind.endswith(" reduce") else kind


def kernels(d, label):
    rows = list(csv.DictReader(open(_one(d, "*kernel_stats.csv"))))
    out = ["# Kernel durations, %s\n" % label,
           "Kernel sources (paper_2503_17707_amd/csrc/*) sha256: `%s`\n" % source_sha256(),
           "| kernel | kind | calls | avg us | total ms | % |", "|---|---|---|---|---|---|"]
    total, launches = collections.defaultdict(float), collections.defaultdict(int)
    for r in rows:
        k = kind_of(r["Name"])
        if len(out) < 26:
            out.append("| `%s` | %s | %s | %.2f | %.2f | %.2f |" % (
                r["Name"][:100], k or "-", r["Calls"], float(r["AverageNs"]) / 1e3,
                float(r["TotalDurationNs"]) / 1e6, float(r["Percentage"])))
        if k:
            total[_base(k)] += float(r["TotalDurationNs"])
            if not k.endswith(" reduce"):
                launches[k] += int(r["Calls"])
    out += ["\nAverage duration per launch by kind (a GEMM kind includes its split-K reduce):\n",
            "| kind | launches | avg us |", "|---|---|---|"]
    for k in sorted(total):
        if launches[k]:
            out.append("| %s | %d | %.2f |" % (k, launches[k], total[k] / launches[k] / 1e3))
    return "\n".join(out)


def _counter(d, name):
    per = collections.defaultdict(list)
    for r in csv.DictReader(open(_one(d, "*counter_collection.csv"))):
        if r["Counter_Name"].startswith(name):
            per[r["Kernel_Name"]].append(float(r["Counter_Value"]))
    return per


def traffic(fetch, write, cal_fetch, cal_write, label):
    f, w = _counter(fetch, "FETCH_SIZE"), _counter(write, "WRITE_SIZE")
    copy = "__amd_rocclr_copyBuffer"
    cf = _counter(cal_fetch, "FETCH_SIZE")[copy]
    cw = _counter(cal_write, "WRITE_SIZE")[copy]
    kib = 1 << 20  # KiB in the 1 GiB copy
    sf, sw = kib / (sum(cf) / len(cf)), kib / (sum(cw) / len(cw))
    out = ["# HBM traffic per kernel launch, %s\n" % label,
           "FETCH_SIZE and WRITE_SIZE (KiB per dispatch) scaled by what the same counter reads "
           "for a plain 1 GiB device copy: FETCH_SIZE %.1f KiB -> x%.4f, WRITE_SIZE %.1f KiB -> x%.4f.\n"
           % (sum(cf) / len(cf), sf, sum(cw) / len(cw), sw),
           "| kernel | kind | dispatches | read MB / dispatch | write MB / dispatch |", "|---|---|---|---|---|"]
    tot, launches = collections.defaultdict(float), collections.defaultdict(int)
    for name, vals in f.items():
        k = kind_of(name)
        if not k:
            continue
        rb = sum(vals) * 1024 * sf
        wv = w.get(name, [])
        wb = sum(wv) * 1024 * sw
        out.append("| `%s` | %s | %d | %.2f | %.2f |" % (name[:90], k, len(vals), rb / len(vals) / 1e6,
                                                        (wb / len(wv) if wv else 0.0) / 1e6))
        tot[_base(k)] += rb + (wb * len(vals) / len(wv) if wv else 0.0)
        if not k.endswith(" reduce"):
            launches[k] += len(vals)
    out += ["\nHBM bytes per launch of each kind (all its dispatches, split-K reduces included, over "
            "its launches), read by bench.py while the kernel sources keep this hash:\n",
            "```traffic", "source_sha256 %s" % source_sha256()]
    for k in sorted(tot):
        if launches[k]:
            out.append("%s %.0f" % (k, tot[k] / launches[k]))
    out.append("```")
    return "\n".join(out)


def _gemm_key(name):
    m = re.search(r"attention_kernelIDF16b?_((?:Li\d+E)+)", name)
    if m and "decode" not in name:
        a = [int(x) for x in re.findall(r"Li(\d+)E", m.group(1))]
        return "attention hd %d, %d queries/wave, %d key group(s)" % (a[0], a[1], a[2])
    m = re.search(r"gemm_kernelIDF16b?_((?:Li\d+E)+)", name)
    if m:
        a = [int(x) for x in re.findall(r"Li(\d+)E", m.group(1))]
        return "this library %dx%d, %d waves, %s" % (a[1], a[2], 64 * a[3] * a[4] // 64,
                                                    {0: "qkv", 1: "o", 2: "fc1", 3: "o/fc2"}.get(a[5], "?"))
    m = re.search(r"(MT\d+x\d+x\d+)", name)
    if "Cijk" in name and m:
        return "vendor library " + m.group(1)
    return None


def stalls(dir_a, dir_b, label):
    per = collections.defaultdict(lambda: collections.defaultdict(list))
    for d in (dir_a, dir_b):
        for r in csv.DictReader(open(_one(d, "*counter_collection.csv"))):
            k = _gemm_key(r["Kernel_Name"])
            if k:
                per[k][r["Counter_Name"]].append(float(r["Counter_Value"]))
    out = ["# Where the waves' cycles go, %s\n" % label,
           "Kernel sources (paper_2503_17707_amd/csrc/*) sha256: `%s`\n" % source_sha256(),
           "Counters per dispatch (dispatches serialized by the counter runs), averaged per kernel.  "
           "Per wave-cycle: SQ_WAIT_ANY (waiting at a wait-count or barrier), SQ_WAIT_INST_ANY "
           "(ready but waiting to issue), SQ_ACTIVE_INST_ANY / _LDS / _VMEM / _VALU, each over "
           "SQ_WAVE_CYCLES.  MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE / 8 XCDs x 1024 "
           "SIMDs); LDS active = SQ_LDS_IDX_ACTIVE / (GRBM_GUI_ACTIVE / 8), summed over the shader "
           "engines; bank conflicts as a share of it.\n",
           "| kernel | dispatches | MFMA busy | wait | wait to issue | active | LDS instr active | VMEM instr "
           "active | VALU active | LDS active | LDS bank conflict share |",
           "|---|---|---|---|---|---|---|---|---|---|---|"]
    for k in sorted(per):
        c = {n: sum(v) / len(v) for n, v in per[k].items()}
        wc = c.get("SQ_WAVE_CYCLES", 0.0)
        g = c.get("GRBM_GUI_ACTIVE", 0.0) / N_XCD
        if not wc or not g:
            continue
        out.append("| %s | %d | %.3f | %.2f | %.2f | %.2f | %.2f | %.2f | %.2f | %.1f | %.2f |" % (
            k, len(per[k].get("SQ_WAVE_CYCLES", [])), c.get("SQ_VALU_MFMA_BUSY_CYCLES", 0) / (g * N_SIMD),
            c.get("SQ_WAIT_ANY", 0) / wc, c.get("SQ_WAIT_INST_ANY", 0) / wc, c.get("SQ_ACTIVE_INST_ANY", 0) / wc,
            c.get("SQ_ACTIVE_INST_LDS", 0) / wc, c.get("SQ_ACTIVE_INST_VMEM", 0) / wc,
            c.get("SQ_ACTIVE_INST_VALU", 0) / wc, c.get("SQ_LDS_IDX_ACTIVE", 0) / g,
            c.get("SQ_LDS_BANK_CONFLICT", 0) / max(1.0, c.get("SQ_LDS_IDX_ACTIVE", 0))))
    return "\n".join(out)


def main(argv):
    usage = {"overlap": (3, 4), "mfma": (3, 3), "kernels": (3, 3), "traffic": (6, 6), "stalls": (4, 4)}
    if not argv or argv[0] not in usage or not usage[argv[0]][0] <= len(argv) <= usage[argv[0]][1]:
        raise SystemExit(__doc__)
    if argv[0] == "overlap":
        gap = int(float(argv[3]) * 1e6) if len(argv) > 3 else GAP_NS
        print(overlap(argv[1], argv[2], gap))
    elif argv[0] == "mfma":
        print(mfma(argv[1], argv[2]))
    elif argv[0] == "kernels":
        print(kernels(argv[1], argv[2]))
    elif argv[0] == "stalls":
        print(stalls(argv[1], argv[2], argv[3]))
    else:
        print(traffic(*argv[1:6]))


if __name__ == "__main__":
    main(sys.argv[1:])
