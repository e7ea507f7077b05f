"""Benchmark of the cold-start prefill path on one MI355X.

Prints one JSON line on stdout.  The headline workload (default: the OPT-66B
shape, 64 layers, d_model 9216, B=2, T=2048, LoRA rank 16 on q and v, fp16
weights, random init: the largest configuration that fits one GPU) is
synthetic; a smaller one (default: the OPT-1.3B shape, B=1, T=512) is measured
first and reported under "extra".  OPT-66B's 131 GB exceed the host memory a
process may pin on the GPU machines, so part of its layer blobs are pageable
and staged through the loader's pinned ring; the line states how many.

* value: warm prefill throughput (TFLOP/s of algorithmic FLOPs) with every
  input already resident in HBM: K timed steps, each one full pass of the
  prefill (embedding, all layers with LoRA, final LayerNorm, LM head, argmax).
* cold_start: the paper's metric, time to first token from pinned host
  weights (poisoned device weights, then LoRA attach + layer streaming +
  prefill), PCIe-inclusive; with the H2D rate of the copy stream.
* roofline: the dominant kernel's average duration from per-kernel HIP events
  on the compute stream (a separate pass of the same K steps), against the
  dense fp16 MFMA peak.
* merged_lora: the same prefill after folding the adapter into the base
  weights (when the workload uses one adapter), against the unmerged time.
* decode: greedy decode steps with the KV cache after a prefill (ms per step,
  weight bytes read per second against HBM), checked against the oracle's
  stored decode logits when present.
* cpu_baseline: the CPU oracle timed on a bounded sample of the same workload.
* paper_context: the paper's own latency figures with the hardware it states.

Separate modes (each prints its own JSON line and exits): --h2d-sweep (pinned
copy rates), --calibrate-copy-mib (the reference copy for HBM byte counters),
--gemm-reference (the projection GEMMs through these kernels and through the
vendor library on the same operands, as a reference point).
"""
import argparse
import gc
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

MFMA_PEAK_TFLOPS = 2500.0     # MI355X dense fp16/bf16
HBM_PEAK_GBPS = 8000.0
PCIE5_X16_GBPS = 63.0         # 32 GT/s x 16 lanes x 128/130 / 8, per direction
METRIC = "cold-start TTFT ms (host weights→first token); prefill TFLOP/s; H2D GB/s"

# The paper's own figures (PipeBoost, arXiv 2503.17707), context only: they come
# from a two-GPU system loading from NVMe, not from this single-GPU path.
PAPER_CONTEXT = {
    "hardware": "2x NVIDIA A100-40GB (PCIe 4.0 x16 per GPU, up to 32 GB/s), Intel Xeon 8338C, "
                "512 GB DDR4; models loaded from NVMe (Section 5.1)",
    "opt_1_3b_first_token": "under 1 s, of which 0.64 s model loading (Section 1); the abstract's "
                            "'few hundred microseconds' cannot include moving 2.63 GB over PCIe",
    "latency_reduction_vs_state_of_the_art": "31% to 49.8% (abstract)",
    "ttft_reduction_vs_serverlessllm": "30% to 47% (Section 1); OPT-1.3B -30.2%, OPT-13B -40.3% "
                                       "(Section 5.2), prompt 64 x batch 64",
    "table1_opt13b_lora_s": {"load_model_params": 3.989, "load_lora_params": 0.021,
                             "prefill": 0.141, "total": 5.547},
    "precision": "not stated by the paper",
}


def err(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_flops(w, kind):
    """Algorithmic FLOPs of one launch of a kernel kind (see the design notes)."""
    d, f, B, T = w.d_model, w.d_ffn, w.batch, w.seq_len
    n = B * T
    rows_lora = sum(T for a in w.adapters() if a >= 0)
    r = w.lora_rank
    tg = set(w.lora_targets) if rows_lora else set()
    if kind == "gemm_qkv":
        return 2 * n * 3 * d * d + 2 * rows_lora * r * d * len(tg & {"q", "k", "v"})
    if kind == "gemm_o":
        return 2 * n * d * d + (2 * rows_lora * r * d if "o" in tg else 0)
    if kind in ("gemm_fc1", "gemm_fc2"):
        return 2 * n * d * f
    if kind == "attention":
        return 2 * B * d * T * (T + 1)
    return None


def source_sha256():
    import glob
    import hashlib

    h = hashlib.sha256()
    for f in sorted(glob.glob(os.path.join(ROOT, "paper_2503_17707_amd", "csrc", "*"))):
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def profiled_traffic(workload, kind):
    """HBM bytes per launch of a kernel kind from the committed rocprofv3 counter
    summary, or None when absent or taken from other kernel sources."""
    path = os.path.join(ROOT, "profiles", "hbm_traffic_%s.md" % workload)
    if not os.path.exists(path):
        return None
    block, inside = {}, False
    for line in open(path):
        line = line.strip()
        if line.startswith("```traffic"):
            inside = True
            continue
        if inside and line.startswith("```"):
            break
        if inside and line:
            k, v = line.split()
            block[k] = v
    if block.get("source_sha256") != source_sha256() or kind not in block:
        return None
    return float(block[kind])


def oracle_baseline(w, n_layers):
    """Time the CPU oracle on the first n_layers of the workload (plus the LM head)."""
    import numpy as np

    import oracle
    import synth

    class Pregenerated(oracle.WeightSource):
        # draws stored first so the timed region holds the oracle's own work
        def __init__(self, w, n):
            super().__init__(w)
            k = self.kind
            self.g = {t: synth.base_tensor(w, -1, t, k) for t in synth.GLOBAL_TENSORS}
            self.ls = [{t: synth.base_tensor(w, l, t, k) for t in synth.LAYER_TENSORS}
                       for l in range(n)]
            self.lo = {}
            for a in {a for a in w.adapters() if a >= 0}:
                self.lo[a] = [{t: {x: synth.lora_tensor(w, a, l, t, x, k) for x in ("A", "B")}
                               for t in w.lora_targets} for l in range(n)]

        def globals(self):
            return {t: oracle.widen(v, self.kind) for t, v in self.g.items()}

        def layer(self, l):
            return {t: oracle.widen(v, self.kind) for t, v in self.ls[l].items()}

        def lora(self, a, l):
            return {t: {x: oracle.widen(v, self.kind) for x, v in d.items()}
                    for t, d in self.lo[a][l].items()}

    src = Pregenerated(w, n_layers)
    toks = synth.tokens(w)
    t0 = time.perf_counter()
    oracle.prefill_first_token(w, tokens=toks, source=src, n_layers=n_layers)
    dt = time.perf_counter() - t0
    fl = w.prefill_flops()
    per_layer = (fl["gemm"] + fl["attn"] + fl["lora"]) / w.n_layers
    flops = per_layer * n_layers + fl["lm_head"]
    cores = len(os.sched_getaffinity(0))
    threads = int(os.environ.get("OMP_NUM_THREADS", cores))
    cpu_model = ""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                cpu_model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    try:
        b = np.show_config(mode="dicts")["Build Dependencies"]["blas"]
        blas = ("%s %s" % (b.get("name", ""), b.get("version", ""))).strip()
    except Exception:
        blas = "unknown"
    return {"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": min(cores, threads),
            "kind": "oracle", "seconds": dt, "cpu_model": cpu_model, "blas": blas,
            "sample": "float64 numpy oracle, first %d of %d layers of the same workload "
                      "(B=%d, T=%d) plus final LayerNorm and LM head; weight draws made before "
                      "timing, widening to float64 timed" % (n_layers, w.n_layers, w.batch,
                                                             w.seq_len)}


def h2d_sweep(w, pb, torch, np):
    """Best sustained pinned host -> device rate: the loader over the workload's
    layer blobs at several chunk sizes, and plain pinned copies of 1 MiB .. 1 GiB
    on one and on two streams (median of 3 after a warm-up)."""
    cfg = pb.make_config(w)
    hw = pb.HostWeights(w, cfg)
    m = pb.Model(cfg, "cuda:0")
    loader = {}
    for mib in (1, 4, 16, 64, 256, 1024):
        m.set_chunk_bytes(mib << 20)
        rates = []
        for rep in range(4):
            m.stream_layers(hw, w.order())
            torch.cuda.synchronize()
            b, ms = m.load_stats()
            if rep:
                rates.append(b / ms / 1e6)
        loader[str(mib)] = float(np.median(rates))
    m.set_chunk_bytes(256 << 20)
    m.destroy()
    hw.free()
    plain = {}
    for mib in (1, 4, 16, 64, 256, 1024):
        n = mib << 20
        reps = max(1, (2 << 30) // n)  # about 2 GiB per timing
        for ns in (1, 2):
            srcs = [torch.empty(n, dtype=torch.uint8, pin_memory=True) for _ in range(ns)]
            dsts = [torch.empty(n, dtype=torch.uint8, device="cuda:0") for _ in range(ns)]
            streams = [torch.cuda.Stream() for _ in range(ns)]
            rates = []
            for rep in range(4):
                torch.cuda.synchronize()
                t0 = time.perf_counter()
                for i in range(reps):
                    with torch.cuda.stream(streams[i % ns]):
                        dsts[i % ns].copy_(srcs[i % ns], non_blocking=True)
                torch.cuda.synchronize()
                if rep:
                    rates.append(n * reps / (time.perf_counter() - t0) / 1e9)
            plain["%d MiB x %d stream%s" % (mib, ns, "s" if ns > 1 else "")] = float(np.median(rates))
            del srcs, dsts
    best = max(list(loader.values()) + list(plain.values()))
    return {"h2d_sweep": {"workload": w.name, "loader_GBps_by_chunk_MiB": loader,
                          "plain_pinned_copy_GBps": plain, "best_GBps": best,
                          "pcie_gen5_x16_GBps": PCIE5_X16_GBPS,
                          "best_frac_of_pcie": best / PCIE5_X16_GBPS}}


def gemm_reference(w, pb, torch, reps=40):
    """The workload's four projection GEMMs (no LoRA tiles) through this
    library's kernels (pb_op_gemm: the model's tile plan and epilogues; o and
    fc2 with their plain split-K reduce, without the LayerNorm the model fuses
    into it) and through the vendor library behind torch's linear (bias
    added), on the same device operands: events around `reps` back-to-back
    launches, after a warm-up.  A reference point for the kernels' rate, not
    part of the path."""
    d, f, n = w.d_model, w.d_ffn, w.batch * w.seq_len
    dt = torch.float16 if w.dtype == "f16" else torch.bfloat16
    dcode = 1 if w.dtype == "f16" else 0
    ws_bytes = max(64 << 20, min(1 << 30, 4 * n * d * 4))
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda:0")
    g = torch.Generator(device="cuda:0").manual_seed(5)
    shapes = [("qkv", 3 * d, d, 0), ("o", d, d, 2), ("fc1", f, d, 1), ("fc2", d, f, 2)]
    out = {}
    for name, N, K, epi in shapes:
        X = torch.randn(n, K, device="cuda:0", generator=g).to(dt)
        W = (torch.randn(N, K, device="cuda:0", generator=g) * 0.02).to(dt)
        b = (torch.randn(N, device="cuda:0", generator=g) * 0.02).to(dt)
        C = torch.empty(n, N, dtype=dt, device="cuda:0") if epi != 2 else None
        R = torch.zeros(n, N, dtype=torch.float32, device="cuda:0") if epi == 2 else None

        def ours():
            pb.op_gemm(dcode, epi, X, W, b, C=C, R=R, qscale=d ** -0.5 if epi == 0 else 1.0,
                       qcols=d if epi == 0 else 0, workspace=ws)

        def library():
            torch.nn.functional.linear(X, W, b)

        row = {"M": n, "N": N, "K": K}
        for label, fn in (("this_library", ours), ("vendor_library", library)):
            for _ in range(5):
                fn()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(reps):
                fn()
            e1.record()
            torch.cuda.synchronize()
            us = e0.elapsed_time(e1) * 1e3 / reps
            row[label] = {"us": us, "tflops": 2.0 * n * N * K / us / 1e6}
        row["this_over_vendor_time"] = row["this_library"]["us"] / row["vendor_library"]["us"]
        out[name] = row
        del X, W, b, C, R
    return {"gemm_reference": {"workload": w.name, "dtype": w.dtype, "launches_timed": reps,
                               "shapes": out}}


def measure(w, steps, warmup, cold_reps, decode_steps, pb, torch, np):
    """One workload: H2D alone, cold starts, warm prefill, per-kernel events,
    decode and merged LoRA where the workload has room for them.  Returns the
    result sections (everything of the JSON line but the CPU baseline)."""
    import synth

    dev = torch.device("cuda:0")
    t0 = time.perf_counter()
    # room for decode steps after the prompt (none when the prompt fills max_pos)
    dec_steps = max(0, min(decode_steps, w.max_pos - w.seq_len))
    # with a shadow of the unmerged attention weights, so that the merged-LoRA
    # section can also time an adapter switch
    cfg = pb.make_config(w, max_new_tokens=dec_steps, merge_shadow=True)
    hw = pb.HostWeights(w, cfg)
    for a in sorted({a for a in w.adapters() if a >= 0}):
        hw.add_lora(a)
    err("%s host weights: %.1f GB (%d of %d layer blobs pinned, the rest staged) in %.1f s" % (
        w.name, (hw.globals_bytes + len(hw.layers) * hw.layer_bytes) / 1e9, hw.pinned_layers,
        len(hw.layers), time.perf_counter() - t0))
    hw_pinned = (hw.pinned_layers, len(hw.layers))
    try:
        nodes_online = open("/sys/devices/system/node/online").read().strip()
    except OSError:
        nodes_online = "unknown"
    numa = {"gpu_numa_node": hw.numa_node, "host_nodes_online": nodes_online,
            "pageable_blobs_bound": sum(1 for b in hw.layers if getattr(b, "bound", False)),
            "binding": "pinned and pageable host blobs placed on the GPU's NUMA node (preferred policy)"
                       if hw.numa_node >= 0 else "runtime default placement"}
    t0 = time.perf_counter()
    m = pb.Model(cfg, "cuda:0")
    init_ms = (time.perf_counter() - t0) * 1e3
    toks = synth.tokens(w)
    ad = list(w.adapters())
    # no collection passes of the interpreter inside timed regions (as timeit
    # does): with torch loaded one pass stalls the host for tens of ms
    gc.collect()
    gc.disable()

    # ---- H2D alone (the bandwidth the loader can get): copies only, median of 3
    # after one warm-up transfer --------------------------------------------------
    rates = []
    for rep in range(4):
        m.poison(0xFF)
        m.stream_layers(hw, w.order())
        torch.cuda.synchronize(dev)
        h2d_bytes, h2d_ms = m.load_stats()
        if rep:
            rates.append(h2d_bytes / h2d_ms / 1e6)
    b_meas = float(np.median(rates))
    err("H2D alone: %.2f GB at %.2f GB/s (median of %d)" % (h2d_bytes / 1e9, b_meas, len(rates)))

    # ---- cold start: pinned host weights -> first token ---------------------
    lora_bytes = sum(b.nbytes for bl in hw.loras.values() for b in bl)
    ttft, loads, first = [], [], None
    for rep in range(cold_reps + 1):
        m.poison(0xFF)
        m.set_stream_delay_us(0)
        torch.cuda.synchronize(dev)
        t0 = time.perf_counter()
        pb.attach_all(m, hw)
        m.stream_layers(hw, w.order())
        tok, logits = m.prefill(toks, ad)
        t1 = time.perf_counter()
        b, ms = m.load_stats()
        if rep == 0:
            first = (tok.copy(), logits.copy())
            continue  # warm-up of code objects and first touches
        ttft.append((t1 - t0) * 1e3)
        loads.append(b / ms / 1e6)
    ttft_med = float(np.median(ttft))
    total_h2d = h2d_bytes + lora_bytes
    bound_ms = total_h2d / (b_meas * 1e6)
    err("cold TTFT median %.2f ms (min %.2f max %.2f), bound %.2f ms" % (
        ttft_med, min(ttft), max(ttft), bound_ms))

    # ---- parity of the first token against the stored oracle logits ---------
    parity = None
    gp = os.path.join(ROOT, "tests", "golden", w.name + ".npz")
    if os.path.exists(gp) and w == synth.WORKLOADS.get(w.name):
        g = np.load(gp, allow_pickle=False)
        ref = g["logits"].astype(np.float64)
        rows = np.linalg.norm(first[1] - ref, axis=-1) / np.linalg.norm(ref, axis=-1)
        parity = {"tokens_equal": bool(np.array_equal(first[0], g["tokens"])),
                  "max_abs": float(np.max(np.abs(first[1] - ref))),
                  "rel_l2_worst_sequence": float(np.max(rows)),
                  "rel_l2_per_sequence": [float(x) for x in rows]}

    # ---- warm prefill: weights resident in HBM -----------------------------
    for _ in range(warmup):
        m.prefill(toks, ad)
    torch.cuda.synchronize(dev)
    t0 = time.perf_counter()
    for _ in range(steps):
        m.prefill(toks, ad)
    torch.cuda.synchronize(dev)
    dt = time.perf_counter() - t0
    ms_step = dt / steps * 1e3
    flops = w.prefill_flops()["total"]
    tflops = flops / (ms_step / 1e3) / 1e12

    # ---- per-kernel durations: same steps, events from the kernels' dispatch packets --
    m.reset_timing()
    m.set_timing(True)
    for _ in range(steps):
        m.prefill(toks, ad)
    m.set_timing(False)
    kt = m.timing()

    # ---- decode: greedy steps with the KV cache after a prefill -----------
    decode = None
    if dec_steps:
        gd = os.path.join(ROOT, "tests", "golden", w.name + "-decode.npz")
        tok, _ = m.prefill(toks, ad)
        dec_parity = None
        if os.path.exists(gd) and w == synth.WORKLOADS.get(w.name):
            g = np.load(gd, allow_pickle=False)
            k = min(dec_steps, g["tokens"].shape[0])
            t_ok, worst, rel = True, 0.0, 0.0
            cur = tok
            for i in range(k):
                cur, lg = m.decode(cur, ad)
                ref = g["logits"][i].astype(np.float64)
                t_ok &= bool(np.array_equal(cur, g["tokens"][i]))
                worst = max(worst, float(np.max(np.abs(lg - ref))))
                rel = max(rel, float(np.max(np.linalg.norm(lg - ref, axis=-1)
                                            / np.linalg.norm(ref, axis=-1))))
            dec_parity = {"steps": k, "tokens_equal": t_ok, "max_abs": worst,
                          "rel_l2_worst_sequence": rel}
            tok, _ = m.prefill(toks, ad)
        torch.cuda.synchronize(dev)
        t0 = time.perf_counter()
        cur = tok
        for _ in range(dec_steps):
            cur, _ = m.decode(cur, ad, want_logits=False)
        dt_dec = time.perf_counter() - t0
        ms_tok = dt_dec / dec_steps * 1e3
        wbytes = h2d_bytes + lora_bytes  # every step reads every weight once
        decode = {"steps": dec_steps, "ms_per_step": ms_tok,
                  "tokens_per_s": w.batch * dec_steps / dt_dec,
                  "weight_GBps": wbytes / (ms_tok / 1e3) / 1e9,
                  "frac_of_hbm": wbytes / (ms_tok / 1e3) / 1e9 / HBM_PEAK_GBPS,
                  "parity": dec_parity}
    kernels = {k: {"avg_ms": (v[0] / v[1]) if v[1] else None, "launches_per_step": v[1] / steps,
                   "ms_per_step": v[0] / steps} for k, v in kt.items()}
    cand = [k for k in kt if kernel_flops(w, k) is not None and kt[k][1]]
    dom = max(cand, key=lambda k: kt[k][0])
    avg_ms = kt[dom][0] / kt[dom][1]
    achieved = kernel_flops(w, dom) / (avg_ms / 1e3) / 1e12
    roofline = {"bound": "mfma", "kernel": dom, "achieved": achieved, "peak": MFMA_PEAK_TFLOPS,
                "unit": "TFLOP/s", "frac": achieved / MFMA_PEAK_TFLOPS,
                "traffic": profiled_traffic(w.name, dom), "traffic_unit": "bytes per launch",
                "avg_launch_ms": avg_ms, "flops_per_launch": kernel_flops(w, dom)}
    # ---- merged LoRA (the paper's choice for pipeline inference): the adapter
    # folded into the base weights, every sequence run as the base model ----
    merged = None
    used = sorted({a for a in ad if a >= 0})
    if len(used) == 1:
        t0 = time.perf_counter()
        m.merge_lora(used[0])
        merge_ms = (time.perf_counter() - t0) * 1e3
        base_ad = [-1] * len(ad)
        mt, ml = m.prefill(toks, base_ad)
        for _ in range(warmup):
            m.prefill(toks, base_ad)
        torch.cuda.synchronize(dev)
        t0 = time.perf_counter()
        for _ in range(steps):
            m.prefill(toks, base_ad)
        torch.cuda.synchronize(dev)
        ms_m = (time.perf_counter() - t0) / steps * 1e3
        # an epoch boundary's switch: restore the shadow, merge again
        t0 = time.perf_counter()
        m.merge_lora(used[0])
        switch_ms = (time.perf_counter() - t0) * 1e3
        t0 = time.perf_counter()
        m.unmerge_lora()
        unmerge_ms = (time.perf_counter() - t0) * 1e3
        merged = {"slot": used[0], "merge_ms": merge_ms, "switch_ms": switch_ms, "unmerge_ms": unmerge_ms,
                  "ms_per_step": ms_m,
                  "unmerged_over_merged": ms_step / ms_m,
                  "tokens_equal_unmerged": bool(np.array_equal(mt, first[0])),
                  "max_abs_vs_unmerged": float(np.max(np.abs(ml - first[1])))}
    m.destroy()
    hw.free()
    gc.enable()

    return {
        "tflops": tflops, "ms_step": ms_step, "flops": flops, "ttft": ttft, "loads": loads,
        "b_meas": b_meas, "total_h2d": total_h2d, "bound_ms": bound_ms, "init_ms": init_ms,
        "roofline": roofline, "kernels": kernels, "decode": decode, "merged": merged,
        "parity": parity, "pinned_layers": hw_pinned[0], "layer_blobs": hw_pinned[1], "numa": numa,
    }



def attention_only(names, pb, torch, reps=20):
    """The prefill attention kernel alone (pb_op_attention) at each workload's
    shape (B sequences of T tokens, H heads of head_dim hd) on random q, k, v:
    events around `reps` back-to-back launches after a warm-up.  FLOPs count
    the causal products only (QK^T and PV over keys <= query)."""
    out = {}
    g = torch.Generator(device="cuda:0").manual_seed(7)
    for name in names:
        import synth

        w = synth.WORKLOADS[name]
        B, T, H, hd = w.batch, w.seq_len, w.n_heads, w.head_dim
        dt = torch.float16 if w.dtype == "f16" else torch.bfloat16
        dcode = 1 if w.dtype == "f16" else 0
        qkv = torch.randn(B * T, 3 * H * hd, device="cuda:0", generator=g).to(dt)
        o = torch.empty(B * T, H * hd, dtype=dt, device="cuda:0")
        for _ in range(3):
            pb.op_attention(dcode, qkv, o, B, T, H, hd)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            pb.op_attention(dcode, qkv, o, B, T, H, hd)
        e1.record()
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1e3 / reps
        fl = 2.0 * B * H * hd * T * (T + 1)
        out[name] = {"B": B, "T": T, "H": H, "head_dim": hd, "us": us, "tflops": fl / us / 1e6,
                     "frac_of_mfma_peak": fl / us / 1e6 / MFMA_PEAK_TFLOPS}
        del qkv, o
    return {"attention_only": out, "launches_timed": reps}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="opt-66b",
                    help="the headline workload (default: the OPT-66B shape, the largest that "
                         "fits one GPU)")
    ap.add_argument("--extra-workload", default="opt-1.3b",
                    help="a second, smaller workload measured first and reported under "
                         "'extra' ('' or 'none' = none)")
    ap.add_argument("--cold-reps", type=int, default=5)
    ap.add_argument("--layers", type=int, default=0,
                    help="run only the first N layers of the headline workload's shape (for "
                         "counter passes, whose figures are per kernel launch; 0 = all)")
    ap.add_argument("--oracle-layers", type=int, default=-1,
                    help="layers of the CPU-oracle sample (0 = all; default: all layers up to "
                         "about 1e13 FLOPs of work, at least one)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-numa", action="store_true",
                    help="leave host blobs where the runtime and the kernel put them instead of on "
                         "the GPU's NUMA node")
    ap.add_argument("--calibrate-copy-mib", type=int, default=0,
                    help="only run a plain device copy of this many MiB (3 times) and exit: "
                         "the reference kernel for scaling HBM byte counters")
    ap.add_argument("--decode-steps", type=int, default=32,
                    help="greedy decode steps timed after the prefill (0 = none)")
    ap.add_argument("--gemm-reference", action="store_true",
                    help="only time the workload's four projection GEMMs through this library's "
                         "kernels and through the vendor library (torch's linear), then exit")
    ap.add_argument("--attention-only", default="",
                    help="only time the prefill attention kernel at these workloads' shapes "
                         "(comma-separated names), then exit")
    ap.add_argument("--h2d-sweep", action="store_true",
                    help="only measure the loader's H2D rate over chunk sizes, and plain pinned "
                         "copies on one and two streams, then exit")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(the sharding design is described with the design notes); run with --gpus 1",
              file=sys.stderr)
        sys.exit(2)

    if args.no_numa:
        os.environ["PIPEBOOST_NUMA"] = "0"
    import numpy as np
    import torch

    if args.calibrate_copy_mib:
        n = args.calibrate_copy_mib << 20
        src = torch.empty(n, dtype=torch.uint8, device="cuda:0").fill_(1)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibration_copy_bytes": n, "copies": 3}), flush=True)
        return

    import synth
    from paper_2503_17707_amd import binding as pb

    pb.lib()  # fails loudly if the HIP library is missing
    if args.attention_only:
        print(json.dumps(attention_only(args.attention_only.split(","), pb, torch)), flush=True)
        return
    w = synth.WORKLOADS[args.workload]
    if args.layers:
        w = w.with_(n_layers=min(args.layers, w.n_layers), layer_order=None)
    if args.h2d_sweep:
        print(json.dumps(h2d_sweep(w, pb, torch, np)), flush=True)
        return
    if args.gemm_reference:
        print(json.dumps(gemm_reference(w, pb, torch)), flush=True)
        return
    out_extra = None
    if args.extra_workload and args.extra_workload not in ("none", args.workload):
        we = synth.WORKLOADS[args.extra_workload]
        r = measure(we, max(args.steps, 50), args.warmup, args.cold_reps, args.decode_steps,
                    pb, torch, np)
        out_extra = sections(we, r)
        out_extra["steps"] = max(args.steps, 50)
        del r
        gc.collect()
    res = measure(w, args.steps, args.warmup, args.cold_reps, args.decode_steps, pb, torch, np)

    cpu = None
    if not args.no_cpu_baseline:
        n_or = args.oracle_layers
        if n_or < 0:
            fl = w.prefill_flops()
            per_layer = (fl["gemm"] + fl["attn"] + fl["lora"]) / w.n_layers
            n_or = int(max(1, min(w.n_layers, 1e13 // per_layer)))
        n_or = n_or or w.n_layers
        err("timing the CPU oracle on %d layers ..." % n_or)
        cpu = oracle_baseline(w, n_or)

    out = {
        "metric": METRIC,
        "value": res["tflops"],
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": res["ms_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic (seeded random-init weights and uniform prompt tokens)",
        "config": config_of(w),
    }
    out.update(sections(w, res))
    out["cpu_baseline"] = cpu
    out["extra"] = out_extra
    out["paper_context"] = PAPER_CONTEXT
    print(json.dumps(out), flush=True)


def config_of(w):
    return {"workload": "%s: %d layers, d_model %d, %d heads, FFN %d, vocab %d; batch %d x "
                        "%d tokens; LoRA rank %d alpha %g on %s, %d adapter(s); %s weights"
                        % (w.name, w.n_layers, w.d_model, w.n_heads, w.d_ffn, w.vocab,
                           w.batch, w.seq_len, w.lora_rank, w.lora_alpha,
                           ",".join(w.lora_targets), w.n_adapters, w.dtype),
            "global_batch": w.batch, "seq_len": w.seq_len, "parallelism": "single GPU"}


def sections(w, r):
    """The per-workload sections of the JSON line from measure()'s results."""
    ttft = r["ttft"]
    ttft_med = float(sorted(ttft)[len(ttft) // 2]) if len(ttft) % 2 else float(
        sum(sorted(ttft)[len(ttft) // 2 - 1:len(ttft) // 2 + 1]) / 2)
    total_h2d, bound_ms, b_meas, ms_step = r["total_h2d"], r["bound_ms"], r["b_meas"], r["ms_step"]
    loads = sorted(r["loads"])
    staged = r["layer_blobs"] - r["pinned_layers"]
    return {
        "workload": w.name,
        "prefill": {"tflops": r["tflops"], "frac_of_mfma_peak": r["tflops"] / MFMA_PEAK_TFLOPS,
                    "flops_per_step": r["flops"], "ms_per_step": ms_step},
        "cold_start": {"ttft_ms": ttft_med, "ttft_min_ms": min(ttft), "ttft_max_ms": max(ttft),
                       "reps": len(ttft), "h2d_bytes": total_h2d,
                       "h2d_GBps_during_cold_start": loads[len(loads) // 2],
                       "h2d_GBps_alone": b_meas, "pcie_gen5_x16_GBps": PCIE5_X16_GBPS,
                       "bound_ms": bound_ms, "frac_of_bound": bound_ms / ttft_med,
                       # the same bytes at the link rate (32 GT/s x 16 lanes, 128b/130b)
                       "link_bound_ms": total_h2d / (PCIE5_X16_GBPS * 1e6),
                       "frac_of_link_bound": total_h2d / (PCIE5_X16_GBPS * 1e6) / ttft_med,
                       "bound_terms_ms": {"h2d_bytes_over_B_meas": bound_ms,
                                          "flops_over_warm_rate": ms_step},
                       "ttft_over_max_bound": ttft_med / max(bound_ms, ms_step),
                       "init_ms": r["init_ms"],
                       "host_numa": r["numa"],
                       "layer_blobs_pinned": r["pinned_layers"],
                       "layer_blobs_staged": staged,
                       "host_memory": ("all layer blobs in pinned host memory" if not staged else
                                       "%d of %d layer blobs pinned; the other %d are pageable and "
                                       "copied through the loader's pinned ring (the machine caps "
                                       "pinned memory per process)" % (
                                           r["pinned_layers"], r["layer_blobs"], staged))},
        "h2d": {"GBps": b_meas, "frac_of_pcie_gen5_x16": b_meas / PCIE5_X16_GBPS},
        "roofline": r["roofline"],
        "kernels": r["kernels"],
        "decode": r["decode"],
        "merged_lora": r["merged"],
        "parity": r["parity"],
    }


if __name__ == "__main__":
    main()
