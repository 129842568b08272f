"""Benchmark: mixed-policy KV decode attention at 64k context on one MI355X.

One timed step is one pass of the whole hot path over one batch of the
64k-context long-document workload (batch 16, 28 query / 4 KV heads, head dim
128, bf16; 4096 text + 15 x 4096 ViT tokens under a 5x storage budget):
  importance scoring over the full context (observation window 32),
  top-k eviction + compaction of the ViT segment (11735 rows per KV head),
  4-bit group quantization of the text segment (group 64),
  512 decode steps, each appending the step's K/V to the protected tail and
  attending over text (packed) + ViT (compacted) + tail.
value = decoded tokens per second of that whole job (B * 512 per step).
Inputs are synthetic (seeded), resident in HBM before timing starts.

The roofline object covers the decode attention call (the dominant kernel
pair: matrix-core split-K pass + log-sum-exp combine), timed with HIP events
on the stream it runs on, against the 8 TB/s HBM peak; cpu_baseline times the
CPU oracle on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import glob
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
METRIC = "mixed-policy KV decode attention tokens/s and achieved HBM GB/s @64k ctx"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5, help="timed jobs")
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--decode-steps", type=int, default=None,
                    help="decode steps per job (default: the workload's 512)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--event-every", type=int, default=8,
                    help="decode steps between timed ones: every event record on the stream "
                         "costs the GPU about 3 us, so the kernel and call events bracket "
                         "steps 0, n, 2n, ... of each job and the rest run unobserved")
    ap.add_argument("--cpu-sample-heads", type=int, default=32)
    ap.add_argument("--cpu-sample-steps", type=int, default=64)
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="after the run, copy a 1 GiB device buffer 3 times (a plain copy "
                         "kernel of known size, for scaling HBM byte counters)")
    ap.add_argument("--summarize-profiles", metavar="DIR", default=None,
                    help="no benchmark: read rocprofv3 output under DIR/trace (kernel trace "
                         "stats), DIR/fetch and DIR/write (FETCH_SIZE / WRITE_SIZE counters of "
                         "runs with --calibrate-copy) and write the summaries under profiles/")
    ap.add_argument("--prefill", action="store_true",
                    help="instead of the decode job: time the multi-query attention of the "
                         "image-editing and text-to-image workloads and report "
                         "matrix-core utilisation (one JSON line each)")
    ap.add_argument("--streaming", action="store_true",
                    help="the decode job with the decode rows streamed into the int4 text "
                         "segment's residual tail (groups of 64 quantised as they fill)")
    ap.add_argument("--batch", action="store_true",
                    help="instead of the decode job: 16 decode requests of different lengths, "
                         "one batched call against one call per request (one JSON line)")
    ap.add_argument("--mall-check", action="store_true",
                    help="decode kernel time on one copy of the compressed 64k cache vs "
                         "alternating between two copies (reuse distance above the 256 MB "
                         "last-level cache)")
    ap.add_argument("--read-ceiling", action="store_true",
                    help="streaming-read rate of HBM in the decode kernel's launch shape: "
                         "whole-line loads and the matrix-core operand pattern (one JSON line)")
    ap.add_argument("--understanding", action="store_true",
                    help="the 7B-shaped understanding workload (4 requests, 4608-row context, "
                         "256 decode steps): whole job, and the decode steps issued one by one "
                         "and replayed as one HIP graph (one JSON line)")
    ap.add_argument("--no-secondary", action="store_true",
                    help="default run only: skip the secondary measurements (prefill, dynamic "
                         "budget, understanding workload) reported under 'secondary'")
    ap.add_argument("--dynamic", action="store_true",
                    help="instead of the decode job: the editing workload under the dynamic "
                         "budget (Eq. 1-3), reporting the chunk-boundary overhead (one JSON line)")
    ap.add_argument("--profile-command", default="",
                    help="with --summarize-profiles: the commands that produced DIR (recorded)")
    return ap.parse_args()


DECODE_KERNELS = ("decode_mfma_kernel", "decode_merge_kernel")
COPY_BYTES = 1 << 30


def _csv(path_glob):
    import csv
    import glob
    files = sorted(glob.glob(path_glob, recursive=True))
    if not files:
        raise FileNotFoundError(path_glob)
    with open(files[0]) as f:
        return list(csv.DictReader(f))


class HipEvents:
    """n timing events created with hipEventDisableSystemFence: recording one
    skips the system-scope cache writeback and invalidation that a default
    event performs, so per-step events do not slow the work they time.  They
    come from the HIP runtime torch has loaded (same soname)."""

    FLAGS = 0x20000000  # hipEventDisableSystemFence

    def __init__(self, n: int):
        import ctypes
        self._c = ctypes
        self.hip = ctypes.CDLL("libamdhip64.so.7")
        self.ev = [ctypes.c_void_p() for _ in range(n)]
        for e in self.ev:
            self._check(self.hip.hipEventCreateWithFlags(ctypes.byref(e), ctypes.c_uint(self.FLAGS)),
                        "hipEventCreateWithFlags")

    def _check(self, rc: int, what: str):
        if rc != 0:
            raise RuntimeError(f"{what} failed with HIP error {rc}")

    def handle(self, i: int) -> int:
        return self.ev[i].value

    def record(self, i: int, stream) -> None:
        self._check(self.hip.hipEventRecord(self.ev[i], self._c.c_void_p(stream.cuda_stream)),
                    "hipEventRecord")

    def elapsed_ms(self, i: int, j: int) -> float:
        ms = self._c.c_float()
        self._check(self.hip.hipEventElapsedTime(self._c.byref(ms), self.ev[i], self.ev[j]),
                    "hipEventElapsedTime")
        return ms.value

    def close(self) -> None:
        for e in self.ev:
            self.hip.hipEventDestroy(e)
        self.ev = []


def _counters(path: str, kernel: str, per_dispatch: bool = False):
    """Counter values of one kernel from a rocprofv3 counter_collection.csv:
    the average per dispatch, or one dict per dispatch (with its grid size)."""
    import csv
    rows = {}
    with open(path) as f:
        for r in csv.DictReader(f):
            name = r["Kernel_Name"].replace("(anonymous namespace)::", "")
            if kernel not in name.split("(")[0]:
                continue
            e = rows.setdefault(r["Dispatch_Id"], {"_grid": int(r["Grid_Size"])})
            e[r["Counter_Name"]] = float(r["Counter_Value"])
    if per_dispatch:
        return [rows[k] for k in sorted(rows, key=int)]
    out = {"_dispatches": len(rows)}
    for e in rows.values():
        for k, v in e.items():
            if not k.startswith("_"):
                out[k] = out.get(k, 0.0) + v / len(rows)
    return out


def summarize_prefill(d: str, command: str):
    """Kernel statistics of the prefill benchmark and matrix-core counters of
    its attention kernel, written to profiles/prefill_attend_4096q.md.
    SQ_VALU_MFMA_BUSY_CYCLES is summed over the chip's SIMDs and
    GRBM_GUI_ACTIVE over its XCDs, so utilisation = busy / (SIMDs x
    GRBM_GUI_ACTIVE / XCDs)."""
    import workloads as gen
    CUS, XCDS = 256, 8
    stats = _csv(os.path.join(d, "ptrace", "**", "*kernel_stats.csv"))
    lines = ["# Kernel statistics and matrix-core counters of the 4096-query prefill benchmark",
             "", "Commands (rocprofv3 on one MI355X):", "", "```", command, "```", "",
             "| kernel | calls | avg us | min us | max us | % |", "|---|---|---|---|---|---|"]
    for r in sorted(stats, key=lambda r: -float(r["TotalDurationNs"]))[:10]:
        name = r["Name"].replace("(anonymous namespace)::", "").split("(")[0]
        name = name.replace("void ", "").replace("uc::", "")
        lines.append(f"| {name[:80]} | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
                     f"{float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} | "
                     f"{float(r['Percentage']):.2f} |")
    grids = {}
    for w in (gen.IMAGE_EDITING, gen.TEXT_TO_IMAGE):
        qb = (w.group_size * w.M + 127) // 128
        grids[((qb * w.B * w.Hkv + 7) // 8 * 8) * 256] = w
    pm = glob.glob(os.path.join(d, "ppmc", "**", "*counter_collection.csv"), recursive=True)
    if pm:
        lines += ["", "Counters of prefill_mfma_kernel per workload (one counter pass; "
                      "dispatches run serialised under counter collection; per-dispatch "
                      "counts, utilisation as mean and range over the dispatches):", "",
                  "| workload | dispatches | MFMA busy cycles | x 1024 flop | algorithmic flop | "
                  "MFMA utilisation | VALU insts | LDS insts | LDS conflict cycles |",
                  "|---|---|---|---|---|---|---|---|---|"]
        rows = {}
        for e in _counters(pm[0], "prefill_mfma_kernel", per_dispatch=True):
            rows.setdefault(e["_grid"], []).append(e)
        for grid, es in rows.items():
            w = grids.get(grid)
            alg = float("nan")
            if w is not None:  # attended rows: fixed-fraction evictions keep floor(ratio * n)
                n_att = sum(int(sg.n * sg.keep_ratio) if sg.policy == "evict" else sg.n
                            for sg in w.segments)
                alg = 4.0 * w.M * n_att * w.D * w.Hq * w.B
            utils = []
            for e in es:
                act = e.get("GRBM_GUI_ACTIVE", 0.0) / XCDS
                utils.append(e.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0) / (4 * CUS * act)
                             if act else float("nan"))
            mean = lambda k: sum(e.get(k, 0.0) for e in es) / len(es)  # noqa: E731
            busy = mean("SQ_VALU_MFMA_BUSY_CYCLES")
            lines.append(f"| {w.name if w else grid} | {len(es)} | {busy:.4g} | "
                         f"{busy * 1024:.4g} | {alg:.4g} | {sum(utils) / len(utils):.3f} "
                         f"({min(utils):.3f}-{max(utils):.3f}) | {mean('SQ_INSTS_VALU'):.4g} | "
                         f"{mean('SQ_INSTS_LDS'):.4g} | {mean('SQ_LDS_BANK_CONFLICT'):.4g} |")
        lines += ["", "The busy-cycle count times 1024 matches the algorithmic flop count "
                      "4 M N D Hq B of each step (one 16x16x32 product = 16384 flop = 16 busy "
                      "cycles) to within 1 %: no padded products; the extra work is the one tile "
                      "of scores per workgroup that the pipelined loop computes past its last "
                      "tile and the scores that a rare raise of the reference maximum recomputes "
                      "from the tile's K rows.  Utilisation is busy cycles over the SIMD-cycles "
                      "of the dispatch."]
    with open(os.path.join(ROOT, "profiles", "prefill_attend_4096q.md"), "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def summarize_profiles(d: str, command: str):
    """Per-dispatch HBM bytes of the decode attention call from FETCH_SIZE /
    WRITE_SIZE (KiB per dispatch), each scaled by the factor that makes the
    counter read exactly 1 GiB for a plain 1 GiB device copy; plus the kernel
    trace statistics.  Writes profiles/decode_attend_64k_traffic.json (read by
    the benchmark while the library sources are unchanged) and a text summary."""
    from paper_2609_32831_amd.build import source_digest

    def per_kernel(rows, counter):
        acc = {}
        for r in rows:
            if r["Counter_Name"] != counter:
                continue
            acc.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]))
        return acc

    out = {"source_digest": source_digest(), "command": command}
    for counter, sub in (("FETCH_SIZE", "fetch"), ("WRITE_SIZE", "write")):
        acc = per_kernel(_csv(os.path.join(d, sub, "**", "*counter_collection.csv")), counter)
        copies = [max(v) for k, v in acc.items() if "copy" in k.lower()]
        if not copies:
            raise RuntimeError(f"{sub}: no copy kernel found (run with --calibrate-copy)")
        factor = (COPY_BYTES / 1024.0) / max(copies)
        out[f"{counter.lower()}_copy_kib"] = max(copies)
        out[f"{counter.lower()}_factor"] = factor
        for kn in DECODE_KERNELS:
            vals = [v for k, vs in acc.items() if kn in k for v in vs]
            out[f"{kn}_{counter.lower()}_kib_avg"] = sum(vals) / len(vals)
            out[f"{kn}_dispatches"] = len(vals)
    per = {kn: (out[f"{kn}_fetch_size_kib_avg"] * out["fetch_size_factor"] +
                out[f"{kn}_write_size_kib_avg"] * out["write_size_factor"]) * 1024.0
           for kn in DECODE_KERNELS}
    # the roofline is taken on the attention kernel; the call adds the merge
    out["traffic_bytes_per_launch"] = int(round(per[DECODE_KERNELS[0]]))
    out["traffic_bytes_per_call"] = int(round(sum(per.values())))
    stats = _csv(os.path.join(d, "trace", "**", "*kernel_stats.csv"))
    lines = ["# Kernel statistics and HBM traffic of the 64k-context decode benchmark", "",
             "Commands (rocprofv3 on one MI355X):", "", "```", command, "```", "",
             "| kernel | calls | avg us | min us | max us | % |", "|---|---|---|---|---|---|"]
    for r in sorted(stats, key=lambda r: -float(r["TotalDurationNs"]))[:10]:
        name = r["Name"].replace("(anonymous namespace)::", "").split("(")[0]
        name = name.replace("void ", "").replace("uc::", "")
        lines.append(f"| {name[:80]} | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
                     f"{float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} | "
                     f"{float(r['Percentage']):.2f} |")
    avg = {kn: next(float(r["AverageNs"]) / 1e3 for r in stats if kn in r["Name"])
           for kn in DECODE_KERNELS}
    out["avg_us"] = avg
    lines += ["", f"decode attention call (sum of the two kernels' averages): "
                  f"{sum(avg.values()):.2f} us", "",
              "HBM bytes per dispatch (FETCH_SIZE x {:.4f}, WRITE_SIZE x {:.4f}; the factors make a "
              "plain 1 GiB copy read 1 GiB):".format(out["fetch_size_factor"],
                                                     out["write_size_factor"])]
    for kn in DECODE_KERNELS:
        fb = out[f"{kn}_fetch_size_kib_avg"] * out["fetch_size_factor"] * 1024
        wb = out[f"{kn}_write_size_kib_avg"] * out["write_size_factor"] * 1024
        lines.append(f"- {kn}: read {fb / 1e6:.2f} MB, written {wb / 1e6:.2f} MB "
                     f"({out[f'{kn}_dispatches']} dispatches)")
    lines.append(f"- per call (both kernels): {out['traffic_bytes_per_call'] / 1e6:.2f} MB")
    # counter passes dpmc, dpmc2, ...: one rocprofv3 --pmc run each (the
    # hardware takes at most 8 SQ, 4 TCC, 4 TCP, 2 TA and 2 GRBM counters
    # per run); their per-dispatch averages are merged
    dps = sorted(glob.glob(os.path.join(d, "dpmc*", "**", "*counter_collection.csv"),
                           recursive=True))
    if dps:
        c, n_disp = {}, []
        for path in dps:
            ci = _counters(path, DECODE_KERNELS[0])
            n_disp.append(ci.pop("_dispatches"))
            c.update(ci)
        hit, miss = c.get("TCC_HIT_sum"), c.get("TCC_MISS_sum")
        lines += ["", f"Counters of {DECODE_KERNELS[0]} (average per dispatch over "
                      f"{'/'.join(str(x) for x in n_disp)} dispatches, {len(dps)} counter "
                      f"passes):", ""]
        for k in sorted(c):
            lines.append(f"- {k}: {c[k]:.4g}")
        lines += ["", "Derived:"]
        if hit is not None and miss is not None:
            lines.append(f"- L2 hit fraction: {hit / (hit + miss):.3f} "
                         f"(misses x 128 B = {miss * 128 / 1e6:.1f} MB)")
        if c.get("SQ_INSTS_LDS"):
            lines.append(f"- LDS bank-conflict cycles per LDS instruction: "
                         f"{c.get('SQ_LDS_BANK_CONFLICT', 0.0) / c['SQ_INSTS_LDS']:.3f}")
        if c.get("TCC_EA0_RDREQ_sum") and c.get("TCC_EA0_RDREQ_LEVEL_sum"):
            lines.append(f"- memory read latency at the L2 (EA read requests in flight summed "
                         f"per cycle / requests): "
                         f"{c['TCC_EA0_RDREQ_LEVEL_sum'] / c['TCC_EA0_RDREQ_sum']:.0f} cycles")
        if c.get("TCP_TCC_READ_REQ_sum") and c.get("TCP_TCC_READ_REQ_LATENCY_sum"):
            lines.append(f"- L1-to-L2 read latency (TCP_TCC_READ_REQ_LATENCY / "
                         f"TCP_TCC_READ_REQ): "
                         f"{c['TCP_TCC_READ_REQ_LATENCY_sum'] / c['TCP_TCC_READ_REQ_sum']:.0f} "
                         f"cycles")
        if c.get("SQ_WAVE_CYCLES"):
            for k, what in (("SQ_WAIT_INST_ANY", "waiting for an issued instruction's result"),
                            ("SQ_WAIT_ANY", "waiting for anything"),
                            ("SQ_ACTIVE_INST_VALU", "issuing vector ALU instructions"),
                            ("SQ_ACTIVE_INST_VMEM", "issuing memory instructions")):
                if c.get(k) is not None:
                    lines.append(f"- {k} / SQ_WAVE_CYCLES ({what}): "
                                 f"{c[k] / c['SQ_WAVE_CYCLES']:.3f}")
        if c.get("SQ_INST_LEVEL_VMEM") and c.get("SQ_INSTS_VMEM_RD"):
            lines.append(f"- vector memory instructions in flight per issued one "
                         f"(SQ_INST_LEVEL_VMEM / SQ_INSTS_VMEM): "
                         f"{c['SQ_INST_LEVEL_VMEM'] / c.get('SQ_INSTS_VMEM', c['SQ_INSTS_VMEM_RD']):.0f}")
    os.makedirs(os.path.join(ROOT, "profiles"), exist_ok=True)
    with open(os.path.join(ROOT, "profiles", "decode_attend_64k_traffic.json"), "w") as f:
        json.dump(out, f, indent=1)
    with open(os.path.join(ROOT, "profiles", "decode_attend_64k.md"), "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def cpu_baseline(w, n_heads: int, n_steps: int, T: int):
    """Time the CPU oracle on n_heads KV heads (full 64k context, full
    compression) and n_steps decode steps; extrapolate linearly to the whole
    job (all B*Hkv heads, T steps) and express it in decode tokens/s."""
    import numpy as np

    import oracle as ref
    import workloads as gen

    cores = ref.set_threads(0)
    D, G = w.D, w.group_size
    nb = max(1, n_heads // w.Hkv)
    BHs = nb * w.Hkv
    sm = float(np.float32(1.0 / np.sqrt(D)))
    pols = None
    import oracle.pipeline as op
    pols = op.plan(w)
    text, vit = 0, 1
    t0 = time.perf_counter()
    kt = gen.segment_kv(w, text, "k", 0, BHs)
    vt = gen.segment_kv(w, text, "v", 0, BHs)
    kv_ = gen.segment_kv(w, vit, "k", 0, BHs)
    vv_ = gen.segment_kv(w, vit, "v", 0, BHs)
    q_obs = gen.queries(w, gen.T_QOBS, w.W, bh0=0, nbh=nb * w.Hq)
    qd = gen.queries(w, gen.T_QDEC, n_steps, bh0=0, nbh=nb * w.Hq)
    kd = gen.decode_kv(w, "k", 0, n_steps, 0, BHs)
    vd = gen.decode_kv(w, "v", 0, n_steps, 0, BHs)
    t_gen = time.perf_counter() - t0

    t0 = time.perf_counter()
    n_t, n_v = w.segments[text].n, w.segments[vit].n
    K = np.concatenate([ref.widen(kt, "bf16"), ref.widen(kv_, "bf16")], axis=1).reshape(nb, w.Hkv, -1, D)
    seg = np.concatenate([np.zeros(n_t, np.int32), np.ones(n_v, np.int32)])
    sc, _ = ref.score(ref.widen(q_obs, "bf16").reshape(nb, w.Hq, w.W, D), K, seg, 2, sm)
    t1 = time.perf_counter()
    keep = ref.select(sc.reshape(BHs, -1)[:, n_t:], pols[vit]["k"], 0)
    t2 = time.perf_counter()
    pk = ref.quantize(kt, vt, "bf16", pols[text]["group"], [pols[text]["bits"]] * BHs)
    kh, vh = ref.dequant(pk, n_t, D, pols[text]["group"], "bf16")
    t3 = time.perf_counter()
    t_compress = t3 - t0
    stages = {"score_s": round(t1 - t0, 3), "select_s": round(t2 - t1, 3),
              "quantize_s": round(t3 - t2, 3)}

    present = np.zeros((BHs, n_v), np.uint8)
    for i in range(BHs):
        present[i, keep[i]] = 1
    Kl = np.concatenate([kh, ref.widen(kv_, "bf16")], axis=1)
    Vl = np.concatenate([vh, ref.widen(vv_, "bf16")], axis=1)
    del K
    t_att = 0.0
    for t in range(n_steps):
        Kt = np.concatenate([Kl, ref.widen(kd[:, : t + 1], "bf16")], axis=1).reshape(nb, w.Hkv, -1, D)
        Vt = np.concatenate([Vl, ref.widen(vd[:, : t + 1], "bf16")], axis=1).reshape(nb, w.Hkv, -1, D)
        pr = np.concatenate([np.ones((BHs, n_t), np.uint8), present, np.ones((BHs, t + 1), np.uint8)],
                            axis=1).reshape(nb, w.Hkv, -1)
        segs = np.concatenate([seg, np.full(t + 1, 2, np.int32)])
        q = ref.widen(qd[:, t:t + 1], "bf16").reshape(nb, w.Hq, 1, D)
        t0 = time.perf_counter()
        ref.attend(q, Kt, Vt, pr, segs, 3, sm)
        t_att += time.perf_counter() - t0
    stages["attend_s_per_step"] = round(t_att / n_steps, 4)
    # one representative step (decode step 0's attention over the sampled
    # heads) again on a single thread
    Kt = np.concatenate([Kl, ref.widen(kd[:, :1], "bf16")], axis=1).reshape(nb, w.Hkv, -1, D)
    Vt = np.concatenate([Vl, ref.widen(vd[:, :1], "bf16")], axis=1).reshape(nb, w.Hkv, -1, D)
    pr = np.concatenate([np.ones((BHs, n_t), np.uint8), present, np.ones((BHs, 1), np.uint8)],
                        axis=1).reshape(nb, w.Hkv, -1)
    segs = np.concatenate([seg, np.full(1, 2, np.int32)])
    q = ref.widen(qd[:, 0:1], "bf16").reshape(nb, w.Hq, 1, D)
    ref.set_threads(1)
    t0 = time.perf_counter()
    ref.attend(q, Kt, Vt, pr, segs, 3, sm)
    t_one = time.perf_counter() - t0
    ref.set_threads(cores)
    scale = (w.B * w.Hkv) / BHs
    t_job = (t_compress + t_att / n_steps * T) * scale
    return {
        "value": round(w.B * T / t_job, 3),
        "unit": "tokens/s",
        "cores": int(cores),
        "kind": "oracle",
        "cpu": cpu_model(),
        "sample": (f"{BHs} of {w.B * w.Hkv} KV heads at full 65536-token context: "
                   f"scoring + selection + quantization ({t_compress:.2f} s) and "
                   f"{n_steps} of {T} decode steps ({t_att:.2f} s), extrapolated "
                   f"linearly to all heads and steps"),
        "stages": stages,
        "single_thread": {"step": f"decode step 0 attention over {BHs} KV heads",
                          "s": round(t_one, 4), "threads": 1},
    }


BF16_PEAK_TFLOPS = 2500.0


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_prefill_baseline(w, stride: int = 16):
    """The CPU oracle's attention for one prefill step of workload w, timed on
    KV head (0, 0) over every stride-th query row of its block and
    extrapolated linearly to all query rows and KV heads.  The logical
    sequence is built as the oracle defines it (kept rows masked in place,
    packed rows quantised and dequantised, 4-bit where the widths are chosen
    per head); which rows are kept does not change the oracle's work."""
    import numpy as np

    import oracle as ref
    import oracle.pipeline as op
    import workloads as gen

    cores = ref.set_threads(0)
    pols = op.plan(w)
    hi = op.head_inputs(w, 0, 0)
    comp = {"khat": [], "vhat": [], "present": []}
    for i, (sg, p) in enumerate(zip(w.segments, pols)):
        k_i, v_i = hi["seg_k"][i], hi["seg_v"][i]
        pres = np.ones(sg.n, np.uint8)
        if p["kind"] == "quant":
            pk = ref.quantize(k_i[None], v_i[None], sg.dtype, p["group"], [p["bits"] or 4])
            kh, vh = ref.dequant(pk, sg.n, w.D, p["group"], sg.dtype)
            kh, vh = kh[0], vh[0]
        else:
            kh, vh = ref.widen(k_i, sg.dtype), ref.widen(v_i, sg.dtype)
            if p["kind"] == "evict":
                pres[:] = 0
                pres[np.linspace(0, sg.n - 1, p["k"]).astype(np.int64)] = 1
        comp["khat"].append(kh)
        comp["vhat"].append(vh)
        comp["present"].append(pres)
    q = gen.queries(w, gen.T_QPRE, w.M, bh0=0, nbh=w.group_size, step=1)[:, ::stride]
    t0 = time.perf_counter()
    op.attend_head(w, comp, q, w.q_dtype)
    t = time.perf_counter() - t0
    rows = q.shape[1]
    ms = t * (w.M / rows) * (w.B * w.Hkv) * 1e3
    return {"value": round(ms, 1), "unit": "ms per step", "cores": int(cores), "kind": "oracle",
            "cpu": cpu_model(),
            "sample": (f"KV head (0, 0): {rows} of {w.M} query rows of each of its "
                       f"{w.group_size} query heads over all {w.n_context} context rows "
                       f"({t:.2f} s), extrapolated linearly to all rows and "
                       f"{w.B * w.Hkv} KV heads")}


def t2i_stored_per_head(w, bits) -> float:
    """Mean stored bytes per KV head of the text-to-image cache: kept text plus
    the latent at each head's width."""
    from paper_2609_32831_amd import NAME_DT, uc_dense_bytes, uc_packed_bytes
    text, lat = w.segments
    per = [uc_dense_bytes(text.n, w.D, NAME_DT[text.dtype])
           + uc_packed_bytes(lat.n, w.D, lat.group, b, NAME_DT[lat.dtype]) for b in bits]
    return sum(per) / len(per)


def static_compression(w, stored_per_head: float) -> dict:
    """Target and realized compression of a workload's cache (original bytes
    at the I/O element type over stored bytes per KV head; protected decode
    tails are no part of either)."""
    from paper_2609_32831_amd import NAME_DT, uc_dense_bytes
    orig = sum(uc_dense_bytes(s.n, w.D, NAME_DT[w.q_dtype]) for s in w.segments)
    return {"target_x": w.budget_ratio, "realized_x": round(orig / stored_per_head, 5)}


def prefill_bench(args):
    """Multi-query attention steps of the editing (4096-query blocks against
    text + compacted ViT + int4 VAE, fixed cache, fresh queries) and
    text-to-image (4096-query blocks against text + int2/int4 latent that is
    requantised every step) workloads.  Utilisation = algorithmic flops
    4 * M * N_attended * D * Hq * B per step over the bf16 dense peak."""
    import torch

    import workloads as gen
    import paper_2609_32831_amd as uc
    results = []
    from paper_2609_32831_amd import uc_attend_mixed, uc_set_kernel_events
    from paper_2609_32831_amd.runner import DenoiseRun, Run
    from workloads.device import DenoiseInputs, device_inputs

    def timed_kernel(fn, n):
        """Average duration of the attention kernel alone (the library
        records the events around it)."""
        evs = HipEvents(2 * n)
        for i in range(n):
            uc_set_kernel_events(evs.handle(2 * i), evs.handle(2 * i + 1))
            fn(i)
        torch.cuda.synchronize()
        ms = sum(evs.elapsed_ms(2 * i, 2 * i + 1) for i in range(n)) / n
        evs.close()
        return ms

    def timed(fn, n):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        # a few untimed steps first: the clocks settle under sustained load
        for _ in range(max(3, args.warmup)):
            fn(0)
        torch.cuda.synchronize()
        a.record()
        for i in range(n):
            fn(i)
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / n

    n = max(10, args.steps)
    # image editing: scoring on the first latent block, 25% ViT, int4 VAE
    w = gen.IMAGE_EDITING
    inp = device_inputs(w, "cuda")
    run = Run(w, inp)
    qs = [inp["q_pre"](t) for t in range(2)]
    torch.cuda.synchronize()
    t_c = timed(lambda i: (run.score(q_obs=qs[0], W=w.M), run.select(), run.quantize()), 1)
    o = torch.empty(w.B, w.Hq, w.M, w.D, device="cuda")
    t_p = timed(lambda i: run.prefill_step(qs[i % 2], o), n)
    t_k = timed_kernel(lambda i: run.prefill_step(qs[i % 2], o), n)
    # the same steps through an execution plan of the frozen cache: the
    # packed rows are dequantised and V converted once, by the first call
    plan = uc.AttendPlan(run.shape, run.mixed, None, qs[0].dtype, w.M, run.sm)
    t_plan = timed(lambda i: plan.attend(qs[i % 2], o), n)
    plan.close()
    n_att = sum(p.k if p.kind == "evict" else s.n for s, p in zip(w.segments, run.pol))
    fl = 4.0 * w.M * n_att * w.D * w.Hq * w.B
    results.append({"metric": "prefill attention step (matrix cores)", "workload": w.name,
                      "ms_per_step": round(t_p, 4), "tflops": round(fl / t_p / 1e9, 1),
                      "frac_of_bf16_peak": round(fl / t_p / 1e9 / BF16_PEAK_TFLOPS, 4),
                      "kernel_ms": round(t_k, 4),
                      "kernel_frac_of_bf16_peak": round(fl / t_k / 1e9 / BF16_PEAK_TFLOPS, 4),
                      "ms_per_step_plan": round(t_plan, 4),
                      "plan_frac_of_bf16_peak": round(fl / t_plan / 1e9 / BF16_PEAK_TFLOPS, 4),
                      "gflop_per_step": round(fl / 1e9, 1), "attended_rows": n_att,
                      "compression": static_compression(w, run.stored_bytes_per_head()),
                      "compress_ms": round(t_c, 3), "steps": n,
                      "cpu_baseline": None if args.no_cpu_baseline else cpu_prefill_baseline(w)})
    del run, inp, qs, o
    torch.cuda.empty_cache()
    # text-to-image: widths from the first (dense) step, then requantise + attend
    w = gen.TEXT_TO_IMAGE
    di = DenoiseInputs(w, "cuda")
    run = DenoiseRun(w, di.seg_k, di.seg_v)
    o = torch.empty(w.B, w.Hq, w.M, w.D, device="cuda")
    run.step(0, di.q, o)
    torch.cuda.synchronize()
    segs = run._segs_packed()
    t_s = timed(lambda i: run.step(1 + i, di.q, o), n)  # requantise + attend (no rescoring)
    t_a = timed(lambda i: uc_attend_mixed(run.shape, segs, di.q, w.M, run.sm, o, ws=run.ws), n)
    t_k = timed_kernel(lambda i: uc_attend_mixed(run.shape, segs, di.q, w.M, run.sm, o,
                                                 ws=run.ws), n)
    fl = 4.0 * w.M * w.n_context * w.D * w.Hq * w.B
    results.append({"metric": "prefill attention step (matrix cores)", "workload": w.name,
                      "ms_per_step": round(t_a, 4), "tflops": round(fl / t_a / 1e9, 1),
                      "frac_of_bf16_peak": round(fl / t_a / 1e9 / BF16_PEAK_TFLOPS, 4),
                      "kernel_ms": round(t_k, 4),
                      "kernel_frac_of_bf16_peak": round(fl / t_k / 1e9 / BF16_PEAK_TFLOPS, 4),
                      "gflop_per_step": round(fl / 1e9, 1), "attended_rows": w.n_context,
                      "step_with_requantise_ms": round(t_s, 4), "bits": run.bits[:8],
                      "compression": static_compression(w, t2i_stored_per_head(w, run.bits)),
                      "steps": n,
                      "cpu_baseline": None if args.no_cpu_baseline else cpu_prefill_baseline(w)})
    del run, di, o
    torch.cuda.empty_cache()
    return results


def _clone_segment(seg):
    """A copy of a segment (descriptor and every buffer it points into)."""
    import ctypes

    import torch

    import paper_2609_32831_amd as uc
    t2 = {k: (v.clone() if isinstance(v, torch.Tensor) else v) for k, v in seg.t.items()}
    d = uc.uc_segment()
    ctypes.memmove(ctypes.byref(d), ctypes.byref(seg.desc), ctypes.sizeof(d))
    for f in ("k", "v", "idx", "head_bits", "code_off", "codes_k", "codes_v", "scale_k", "min_k",
              "scale_v", "min_v", "tail_k", "tail_v"):
        if getattr(seg.desc, f) and t2.get(f) is not None:
            setattr(d, f, t2[f].data_ptr())
    return uc.Segment(d, t2)


def mall_check(args):
    """The decode kernel on the 64k cache (tail of 256 rows) timed on one copy
    of the compressed cache, and alternating between two identical copies:
    each call reads 435 MB, more than the 256 MB last-level cache, and with
    two copies a row is read again only after 870 MB of other rows.  Equal
    times mean that the single-copy figure is not helped by cache reuse."""
    import torch

    import paper_2609_32831_amd as uc
    import workloads as gen
    from paper_2609_32831_amd.runner import Run
    from workloads.device import device_inputs

    w = gen.LONG_CONTEXT_64K
    inp = device_inputs(w, "cuda", steps=w.steps)
    run = Run(w, inp)
    run.compress()
    o = torch.empty(w.B, w.Hq, 1, w.D, device="cuda")
    for t in range(256):
        uc.uc_attend_append(run.shape, run.mixed, len(run.mixed) - 1, inp["k_dec"][t],
                            inp["v_dec"][t], 1, inp["q_dec"][t], 1, run.sm, o, ws=run.ws_attend)
    copies = [run.mixed, [_clone_segment(sg) for sg in run.mixed]]
    torch.cuda.synchronize()
    q = inp["q_dec"][300]
    n = 64
    evs = HipEvents(2 * n)

    def timed(order):
        for i in range(8):
            uc.uc_attend_mixed(run.shape, copies[order[i % len(order)]], q, 1, run.sm, o,
                               ws=run.ws_attend)
        for i in range(n):
            uc.uc_set_kernel_events(evs.handle(2 * i), evs.handle(2 * i + 1))
            uc.uc_attend_mixed(run.shape, copies[order[i % len(order)]], q, 1, run.sm, o,
                               ws=run.ws_attend)
        torch.cuda.synchronize()
        return sum(evs.elapsed_ms(2 * i, 2 * i + 1) for i in range(n)) / n * 1e3

    res = {"one": [], "two": []}
    for _ in range(3):
        res["one"].append(timed([0]))
        res["two"].append(timed([0, 1]))
    nbytes = run.attended_bytes(256)
    one, two = min(res["one"]), min(res["two"])
    print(json.dumps({"metric": "decode kernel, one cache copy vs two alternating copies",
                      "workload": w.name, "bytes_per_call": int(nbytes),
                      "one_copy_us": round(one, 2), "two_copies_us": round(two, 2),
                      "one_copy_frac": round(nbytes / one / 1e3 / HBM_PEAK_GBPS, 4),
                      "two_copies_frac": round(nbytes / two / 1e3 / HBM_PEAK_GBPS, 4),
                      "ratio": round(two / one, 4)}), flush=True)
    evs.close()


def understanding_bench(args):
    """The 7B-shaped understanding workload: compression (scores of a 32-row
    observation window over all 4608 context rows, the top 406 ViT rows per
    KV head kept and gathered) and 256 decode steps, each appending its K/V to
    the protected tail inside one fused attention launch plus the combine.
    Each step reads about 8.65 MB, which stays in the 256 MB last-level cache,
    so the steps are bound by launches and latency: they are timed issued one
    by one (the whole job, as the 64k benchmark times it) and captured once as
    a HIP graph of all 256 steps and replayed; every replay's outputs are
    compared with the steps issued one by one."""
    import torch

    import paper_2609_32831_amd as uc
    import workloads as gen
    from paper_2609_32831_amd.runner import Run
    from workloads.device import device_inputs

    w = gen.UNDERSTANDING_7B
    T = w.steps
    inp = device_inputs(w, "cuda", steps=T)
    run = Run(w, inp)
    o = torch.empty(T, w.B, w.Hq, 1, w.D, device="cuda")

    def steps():
        for t in range(T):
            uc.uc_attend_append(run.shape, run.mixed, len(run.mixed) - 1, inp["k_dec"][t],
                                inp["v_dec"][t], 1, inp["q_dec"][t], 1, run.sm, o[t],
                                ws=run.ws_attend)

    def job():
        run.compress()
        steps()

    # the same steps through an execution plan of the frozen layout: created
    # once per job after compression, then each step passes only pointers
    # (App. E, "Cached metadata and execution plans")
    step_ptrs = [(x.data_ptr(), x.stride(0) * x.element_size())
                 for x in (inp["k_dec"], inp["v_dec"], inp["q_dec"], o)]
    ws_plan = None

    def plan_steps():
        plan = uc.AttendPlan(run.shape, run.mixed, len(run.mixed) - 1, inp["q_dec"].dtype, 1,
                             run.sm, ws=ws_plan)
        step = plan.attend_append
        (kb, ks), (vb, vs), (qb, qs), (ob, os_) = step_ptrs
        for t in range(T):
            step(kb + t * ks, vb + t * vs, 1, qb + t * qs, ob + t * os_)
        plan.close()

    stream = torch.cuda.current_stream()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
    for _ in range(max(1, args.warmup)):
        job()
    torch.cuda.synchronize()
    n = max(1, args.steps)
    job_ms, step_ms = 0.0, 0.0
    for _ in range(n):
        ev[0].record(stream)
        run.compress()
        ev[1].record(stream)
        steps()
        ev[2].record(stream)
        torch.cuda.synchronize()
        job_ms += ev[0].elapsed_time(ev[2])
        step_ms += ev[1].elapsed_time(ev[2])
    job_ms /= n
    step_ms /= n
    o_eager = o.clone()
    run.compress()
    p0 = uc.AttendPlan(run.shape, run.mixed, len(run.mixed) - 1, inp["q_dec"].dtype, 1, run.sm)
    ws_plan = p0.ws
    p0.close()
    plan_ms, plan_job_ms, plan_ok = 0.0, 0.0, True
    for _ in range(n):
        o.zero_()
        torch.cuda.synchronize()
        ev[0].record(stream)
        run.compress()
        ev[1].record(stream)
        plan_steps()
        ev[2].record(stream)
        torch.cuda.synchronize()
        plan_job_ms += ev[0].elapsed_time(ev[2])
        plan_ms += ev[1].elapsed_time(ev[2])
        plan_ok = plan_ok and bool(torch.equal(o, o_eager))
    plan_ms /= n
    plan_job_ms /= n
    # the same 256 steps as one graph: the tail restarts at row 0, and each
    # replay appends and attends exactly as the steps above did
    run.tail.n_rows = 0
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(stream)
    with torch.cuda.graph(g, stream=side):
        steps()
    torch.cuda.synchronize()
    graph_ms, ok = 0.0, True
    for _ in range(n):
        o.zero_()
        torch.cuda.synchronize()
        ev[0].record(stream)
        g.replay()
        ev[3].record(stream)
        torch.cuda.synchronize()
        graph_ms += ev[0].elapsed_time(ev[3])
        ok = ok and bool(torch.equal(o, o_eager))
    graph_ms /= n
    nbytes = sum(run.attended_bytes(t + 1) for t in range(T)) / T
    tokens = w.B * T
    return ({"metric": "understanding decode", "workload": w.name,
                      "tokens_per_s": round(tokens / (job_ms / 1e3), 1), "ms_per_job": round(job_ms, 3),
                      "compress_ms": round(job_ms - step_ms, 3),
                      "decode_step_us": round(step_ms / T * 1e3, 2),
                      "decode_step_us_plan": round(plan_ms / T * 1e3, 2),
                      "tokens_per_s_plan": round(tokens / (plan_job_ms / 1e3), 1),
                      "plan_matches_steps": plan_ok,
                      "decode_step_us_graph": round(graph_ms / T * 1e3, 2),
                      "decode_tokens_per_s_graph": round(tokens / (graph_ms / 1e3), 1),
                      "bytes_per_step": int(nbytes), "graph_matches_steps": ok, "jobs": n})


def dynamic_bench(args):
    """The editing workload under the dynamic budget (Sec. 3.3 Eq. 1-3): per
    request, timestep 0 on the full cache plus the initial compression, then
    24 compressed timesteps with a budget decision after every 5.  Reports
    the attention time, the time of the chunk-boundary work (type masses to
    the host, Eq. 2/3, re-scoring and top-k inside the kept rows, index
    composition, re-quantisation) and its fraction of the attention time."""
    import torch

    import workloads as gen
    from paper_2609_32831_amd.runner import DynamicRun
    from workloads.device import device_inputs

    from paper_2609_32831_amd.calibrate import calibrate_rho_min, realized_compression

    w = gen.IMAGE_EDITING_DYNAMIC
    inp = device_inputs(w, "cuda")
    # rho_min calibrated to the workload's target average compression (App. B)
    cal = calibrate_rho_min(w, inp, w.target_compression, requests=list(range(w.B)))
    w = gen.scaled(w, rho_min=cal["rho_min"])
    qs = [inp["q_pre"](t) for t in range(w.steps)]
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    res = []
    for b in range(w.B):
        seg_k = [t[b:b + 1].contiguous() for t in inp["seg_k"]]
        seg_v = [t[b:b + 1].contiguous() for t in inp["seg_v"]]
        q_b = [q[b:b + 1].contiguous() for q in qs]
        o = torch.empty(1, w.Hq, w.M, w.D, device="cuda")
        for rep in range(max(1, args.warmup) + 1):  # the last repetition is timed
            run = DynamicRun(w, seg_k, seg_v)
            ev = HipEvents(3 * w.steps)
            torch.cuda.synchronize()
            bsteps = []
            for t in range(w.steps):
                ev.record(3 * t, stream)
                # the attention (on the layout's execution plan) and the
                # per-step type masses
                run.attend(t, q_b[t], o)
                ev.record(3 * t + 1, stream)
                if run.after_step(t, q_b[t]) is not None:
                    # a boundary: its work is bracketed by one more event (the
                    # other steps have none: an event costs the GPU a few us)
                    ev.record(3 * t + 2, stream)
                    bsteps.append(t)
            torch.cuda.synchronize()
        att = [ev.elapsed_ms(3 * t, 3 * t + 1) for t in range(w.steps)]
        bnd = [ev.elapsed_ms(3 * t + 1, 3 * t + 2) if t in bsteps else 0.0
               for t in range(w.steps)]
        ev.close()
        d = run.decisions
        res.append({"att": att, "bnd": bnd, "dec": d})
    att0 = sum(r["att"][0] for r in res)
    init = sum(r["bnd"][0] for r in res)
    att = sum(sum(r["att"][1:]) for r in res)
    bnd = sum(sum(r["bnd"][1:]) for r in res)
    last = res[0]["dec"][max(res[0]["dec"])]
    realized = sum(realized_compression(w, r["dec"]) for r in res) / len(res)
    return ({"metric": "dynamic budget overhead (Eq. 1-3 at chunk boundaries)",
                      "workload": w.name, "requests": w.B, "timesteps": w.steps,
                      "chunk_steps": w.chunk_steps,
                      "compression": {"target": w.target_compression,
                                      "realized": round(realized, 5),
                                      "rho_init": w.rho_init,
                                      "rho_min_calibrated": round(w.rho_min, 6),
                                      "calibration_probes": len(cal["probes"])},
                      "full_kv_step_ms": round(att0 / w.B, 4),
                      "initial_compression_ms": round(init / w.B, 4),
                      "compressed_step_ms": round(att / w.B / (w.steps - 1), 4),
                      "boundary_ms_total": round(bnd / w.B, 4),
                      "boundary_frac_of_attention": round(bnd / att, 4),
                      "decisions_request0": {str(t): {"rho": round(x["rho"], 5), "k": x["k"],
                                                      "bits": x["bits"], "group": x["group"]}
                                             for t, x in res[0]["dec"].items()},
                      "final_k": last["k"], "final_bits": last["bits"],
                      "final_group": last["group"]})


def batch_bench(args):
    """Requests of different context lengths decoded together: 16 requests of
    the 64k workload's shape (4 KV heads, 28 query heads, head dim 128), each
    with the int4 g64 text segment (4096 rows) and its own number of kept ViT
    rows (2000 + 700 r) and protected tail rows (r + 1).  One uc_attend_batch
    call (one attention launch for all requests) against one uc_attend_mixed
    call per request; each captured in a graph and replayed (fence-free
    events around every replay).  Roofline of the batched attention kernel on
    the bytes all requests read."""
    import torch

    import paper_2609_32831_amd as uc
    from paper_2609_32831_amd.runner import sm_scale

    torch.manual_seed(0)
    Hq, Hkv, D, R = 28, 4, 128, 16
    dev = "cuda"
    shape1 = uc.make_shape(1, Hq, Hkv, D)
    reqs, n_bytes = [], 0
    for r in range(R):
        n_vit, n_tail = 2000 + 700 * r, r + 1
        kt = torch.randn(1, Hkv, 4096, D, device=dev).to(torch.bfloat16)
        vt = torch.randn(1, Hkv, 4096, D, device=dev).to(torch.bfloat16)
        text = uc.packed_segment(1, Hkv, 4096, D, 64, torch.bfloat16, bits=4, device=dev)
        uc.uc_quantize_segment(shape1, kt, vt, 4096, text)
        vit = uc.dense_segment(torch.randn(1, Hkv, n_vit, D, device=dev).to(torch.bfloat16),
                               torch.randn(1, Hkv, n_vit, D, device=dev).to(torch.bfloat16))
        tk = torch.randn(1, Hkv, n_tail, D, device=dev).to(torch.bfloat16)
        tail = uc.dense_segment(tk, torch.randn_like(tk))
        reqs.append([text, vit, tail])
        n_bytes += Hkv * (uc.uc_packed_bytes(4096, D, 64, 4, uc.UC_BF16) + (n_vit + n_tail) * 2 * D * 2)
    n_bytes += R * Hq * D * (2 + 4)
    shape = uc.make_shape(R, Hq, Hkv, D)
    q = torch.randn(R, Hq, 1, D, device=dev).to(torch.bfloat16)
    o = torch.empty(R, Hq, 1, D, device=dev)
    sm = sm_scale(D)
    ws = torch.empty(max(uc.uc_attend_batch_workspace_size(shape, reqs, uc.UC_BF16, 1), 256),
                     dtype=torch.uint8, device=dev)
    ws1 = torch.empty(max(max(uc.uc_attend_workspace_size(shape1, rq, uc.UC_BF16, 1) for rq in reqs),
                          256), dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream()
    n = max(20, args.steps * 20)

    def batched():
        uc.uc_attend_batch(shape, reqs, q, 1, sm, o, ws=ws)

    def looped():
        for r in range(R):
            uc.uc_attend_mixed(shape1, reqs[r], q[r:r + 1], 1, sm, o[r:r + 1], ws=ws1)

    res = {}
    # kernel time of the batched launch (eager calls, library-recorded events)
    for _ in range(3):
        batched()
    evk = HipEvents(2 * n)
    torch.cuda.synchronize()
    for i in range(n):
        uc.uc_set_kernel_events(evk.handle(2 * i), evk.handle(2 * i + 1))
        batched()
    torch.cuda.synchronize()
    res["kernel"] = sum(evk.elapsed_ms(2 * i, 2 * i + 1) for i in range(n)) / n * 1e3
    evk.close()
    # whole-call GPU time: each variant captured once in a graph (kernels only)
    # and replayed, so host-side marshalling does not starve the GPU; every
    # replay's output is checked against the eager result
    batched()
    torch.cuda.synchronize()
    o_ref = o.clone()
    for name, fn in (("batched", batched), ("per_request", looped)):
        g = torch.cuda.CUDAGraph()
        cs = torch.cuda.Stream()
        cs.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(cs):
            fn()  # warm-up on the capture stream
        torch.cuda.current_stream().wait_stream(cs)
        torch.cuda.synchronize()
        with torch.cuda.graph(g):
            fn()
        ev = HipEvents(2 * n)
        for i in range(n):
            o.zero_()
            ev.record(2 * i, stream)
            g.replay()
            ev.record(2 * i + 1, stream)
            if i < 3:
                torch.cuda.synchronize()
                if (o - o_ref).abs().max().item() > 5e-4:
                    raise RuntimeError(f"graph replay {i} of {name} differs from the eager result")
        torch.cuda.synchronize()
        res[name] = sum(ev.elapsed_ms(2 * i, 2 * i + 1) for i in range(n)) / n * 1e3
        ev.close()
        del g
    ach = n_bytes / (res["kernel"] * 1e-6) / 1e9
    return {"metric": "batched decode over requests of different layouts",
            "requests": R, "bytes_per_step": n_bytes,
            "batched_call_us": round(res["batched"], 2),
            "per_request_calls_us": round(res["per_request"], 2),
            "speedup": round(res["per_request"] / res["batched"], 3),
            "roofline": {"bound": "hbm", "kernel": "decode_batch_args_kernel",
                         "avg_launch_us": round(res["kernel"], 2),
                         "achieved": round(ach, 1), "peak": HBM_PEAK_GBPS,
                         "unit": "GB/s", "frac": round(ach / HBM_PEAK_GBPS, 4)}}


def read_ceiling(args) -> dict:
    """The streaming-read probe (uc_read_probe) over a 2 GiB buffer, both load
    patterns, 20 timed calls each after 3 warm-up calls (fence-free events
    around each call): the rate a plain read of HBM reaches in the decode
    kernel's launch shape, which the decode kernel's achieved bandwidth is
    compared with."""
    import torch

    import paper_2609_32831_amd as uc

    unit = uc.uc_read_probe_unit()
    nbytes = (2 << 30) // unit * unit
    buf = torch.ones(nbytes, dtype=torch.uint8, device="cuda")
    sink = torch.empty(uc.uc_read_probe_sink_bytes(), dtype=torch.uint8, device="cuda")
    n = 20
    res = {"metric": "streaming read of HBM (probe)", "bytes": nbytes,
           "launch": "2 x 256-thread workgroups per CU, non-temporal 16-byte loads"}
    for name, pat in (("lines", uc.UC_PROBE_LINES), ("operand_pattern", uc.UC_PROBE_OPERAND)):
        for _ in range(3):
            uc.uc_read_probe(buf, pat, sink)
        ev = HipEvents(2 * n)
        torch.cuda.synchronize()
        stream = torch.cuda.current_stream()
        for i in range(n):
            ev.record(2 * i, stream)
            uc.uc_read_probe(buf, pat, sink)
            ev.record(2 * i + 1, stream)
        torch.cuda.synchronize()
        ts = sorted(ev.elapsed_ms(2 * i, 2 * i + 1) for i in range(n))
        ev.close()
        res[name + "_tbs"] = round(nbytes / (ts[n // 2] * 1e-3) / 1e12, 3)
        res[name + "_best_tbs"] = round(nbytes / (ts[0] * 1e-3) / 1e12, 3)
    del buf
    return res


def secondary(args) -> dict:
    """The other workloads' figures, measured in the same run as the headline
    line (no CPU baselines): the two prefill workloads, the dynamic budget's
    boundary overhead, the understanding workload's decode, the batched
    decode of requests of different layouts and the streaming-read ceiling
    of HBM.  A part that
    fails is reported with its error instead of its figures."""
    import copy
    import traceback
    a = copy.copy(args)
    a.no_cpu_baseline = True
    res = {}
    for name, fn in (("prefill", prefill_bench), ("dynamic", dynamic_bench),
                     ("understanding", understanding_bench), ("batch", batch_bench),
                     ("read_ceiling", read_ceiling)):
        t0 = time.perf_counter()
        try:
            res[name] = fn(a)
        except Exception as e:  # keep the headline line whatever happens here
            traceback.print_exc()
            res[name] = {"error": f"{type(e).__name__}: {e}"}
        print(f"# secondary {name} took {time.perf_counter() - t0:.1f} s", file=sys.stderr,
              flush=True)
    return res


def main():
    args = parse()
    if args.summarize_profiles:
        if args.prefill:
            summarize_prefill(args.summarize_profiles, args.profile_command)
        else:
            summarize_profiles(args.summarize_profiles, args.profile_command)
        return
    if args.prefill:
        if args.gpus != 1:
            sys.exit(2)
        for r in prefill_bench(args):
            print(json.dumps(r), flush=True)
        return
    if args.dynamic:
        if args.gpus != 1:
            sys.exit(2)
        print(json.dumps(dynamic_bench(args)), flush=True)
        return
    if args.mall_check:
        if args.gpus != 1:
            sys.exit(2)
        mall_check(args)
        return
    if args.read_ceiling:
        if args.gpus != 1:
            sys.exit(2)
        print(json.dumps(read_ceiling(args)), flush=True)
        return
    if args.understanding:
        if args.gpus != 1:
            sys.exit(2)
        print(json.dumps(understanding_bench(args)), flush=True)
        return
    if args.batch:
        if args.gpus != 1:
            sys.exit(2)
        print(json.dumps(batch_bench(args)), flush=True)
        return
    if args.gpus != 1:
        print(f"bench.py: this build runs on one GPU; --gpus {args.gpus} is not supported "
              "(the path would shard over (b, h_kv) with no exchange, see the design notes)",
              file=sys.stderr, flush=True)
        sys.exit(2)
    import numpy as np
    import torch

    import paper_2609_32831_amd as uc
    import workloads as gen
    from paper_2609_32831_amd.runner import Run
    from workloads.device import device_inputs

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    w = gen.LONG_CONTEXT_64K_STREAMING if args.streaming else gen.LONG_CONTEXT_64K
    T = w.steps if args.decode_steps is None else args.decode_steps
    t0 = time.perf_counter()
    inp = device_inputs(w, "cuda", steps=T)
    run = Run(w, inp)
    torch.cuda.synchronize()
    print(f"# inputs ready in {time.perf_counter() - t0:.1f} s", file=sys.stderr, flush=True)

    stream = torch.cuda.current_stream()
    o = torch.empty(T, w.B, w.Hq, 1, w.D, device="cuda")
    # sampled steps: 4t+2, 4t+3, which the library records around its
    # attention kernel alone (the merge of partial results falls outside
    # them), on steps t % every == 0; 4t, 4t+1 around the whole attention call
    # on steps t % every == every // 2 (so that no call bracket holds the
    # kernel pair's records, unless every == 1)
    every = max(1, args.event_every)
    sampled = [t for t in range(T) if t % every == 0]
    sampled_call = [t for t in range(T) if t % every == every // 2]
    ev = HipEvents(4 * T)
    ev_c = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))

    def job(record: bool):
        if record:
            ev_c[0].record(stream)
        run.compress()
        if record:
            ev_c[1].record(stream)
        for t in range(T):
            if run.tail is None:  # the row joins the quantised text segment's residual tail
                uc.uc_stream_append(run.shape, run.mixed[run.stream], inp["k_dec"][t],
                                    inp["v_dec"][t], 1)
            kern_t = record and t % every == 0
            call_t = record and t % every == every // 2
            if call_t:
                ev.record(4 * t, stream)
            if kern_t:
                uc.uc_set_kernel_events(ev.handle(4 * t + 2), ev.handle(4 * t + 3))
            if run.tail is not None:  # row t joins the protected tail inside the attention launch
                uc.uc_attend_append(run.shape, run.mixed, len(run.mixed) - 1, inp["k_dec"][t],
                                    inp["v_dec"][t], 1, inp["q_dec"][t], 1, run.sm, o[t],
                                    ws=run.ws_attend)
            else:
                uc.uc_attend_mixed(run.shape, run.mixed, inp["q_dec"][t], 1, run.sm, o[t],
                                   ws=run.ws_attend)
            if call_t:
                ev.record(4 * t + 1, stream)

    for _ in range(args.warmup):
        job(False)
    torch.cuda.synchronize()
    print("# warmup done", file=sys.stderr, flush=True)
    attend_ms = 0.0
    kernel_ms = 0.0
    compress_ms = 0.0
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    for k in range(args.steps):
        job(True)
        torch.cuda.synchronize()
        attend_ms += sum(ev.elapsed_ms(4 * t, 4 * t + 1) for t in sampled_call)
        kernel_ms += sum(ev.elapsed_ms(4 * t + 2, 4 * t + 3) for t in sampled)
        compress_ms += ev_c[0].elapsed_time(ev_c[1])
        print(f"# job {k + 1}/{args.steps} done", file=sys.stderr, flush=True)
    end.record(stream)
    torch.cuda.synchronize()
    total_ms = start.elapsed_time(end)
    ms_per_step = total_ms / args.steps
    tokens = w.B * T
    value = tokens / (ms_per_step / 1e3)
    att_us = attend_ms / (args.steps * len(sampled_call)) * 1e3
    kern_us = kernel_ms / (args.steps * len(sampled)) * 1e3
    # algorithmic bytes per attend call, averaged over the sampled steps'
    # tail lengths
    avg_bytes = sum(run.attended_bytes(t + 1) for t in sampled) / len(sampled)
    call_bytes = sum(run.attended_bytes(t + 1) for t in sampled_call) / len(sampled_call)
    achieved = avg_bytes / (kern_us * 1e-6) / 1e9
    # the decode steps alone: the timed jobs less their compression
    decode_ms = ms_per_step - compress_ms / args.steps
    traffic = None
    tp = os.path.join(ROOT, "profiles", "decode_attend_64k_traffic.json")
    if os.path.exists(tp) and not args.streaming:
        try:
            with open(tp) as f:
                tr = json.load(f)
            from paper_2609_32831_amd.build import source_digest
            if tr.get("source_digest") == source_digest():
                traffic = tr.get("traffic_bytes_per_launch")
        except Exception:  # stale or unreadable counters: report none
            traffic = None
    out = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "batch": w.B, "q_heads": w.Hq,
                   "kv_heads": w.Hkv, "head_dim": w.D, "context": w.n_context,
                   "segments": ("text 4096 int4 g64 + decode rows streamed into its tail | "
                                "vit 61440 -> 11735 kept per kv head" if args.streaming else
                                "text 4096 int4 g64 | vit 61440 -> 11735 kept per kv head | "
                                "protected decode tail"), "budget": "5x",
                   "decode_steps": T, "observation_window": w.W},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4),
                     "traffic": traffic,
                     "kernel": "decode_mfma_kernel",
                     "avg_launch_us": round(kern_us, 2),
                     "algorithmic_bytes_per_launch": int(avg_bytes),
                     # the whole attention call: the kernel and the merge of
                     # its partial records
                     "call_frac": round(call_bytes / (att_us * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4)},
        "compression": static_compression(w, run.stored_bytes_per_head()),
        "attend_call_us": round(att_us, 2),
        "attend_call_frac": round(call_bytes / (att_us * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4),
        "decode_step_us": round(decode_ms / T * 1e3, 2),
        "decode_only_tokens_per_s": round(tokens / (decode_ms / 1e3), 1),
        "compress_ms": round(compress_ms / args.steps, 3),
    }
    if args.calibrate_copy:
        src = torch.empty(1 << 30, dtype=torch.uint8, device="cuda").fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    if not args.no_secondary and not args.streaming:
        del run, inp, o, ev
        torch.cuda.empty_cache()
        out["secondary"] = secondary(args)
    if not args.no_cpu_baseline and not args.streaming:  # the baseline models the headline job
        t0 = time.perf_counter()
        out["cpu_baseline"] = cpu_baseline(w, args.cpu_sample_heads, args.cpu_sample_steps, T)
        print(f"# cpu baseline took {time.perf_counter() - t0:.1f} s", file=sys.stderr, flush=True)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
