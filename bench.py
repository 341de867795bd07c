#!/usr/bin/env python3
"""Benchmark of the Lynx hot path on one MI355X.

Workload (Llama-3-8B-shaped single sequence): 32 layers x (32 query heads,
8 kv heads, head_dim 128), context 32768 tokens, batch 1, BF16 K/V ~ N(0,1)
with 1% of K (kv head, channel) columns x8; k = 8 draft queries per layer for
verification.  Synthetic data, seeded.

One step = the whole hot path over all 32 layers:
  1. encode (quantize, split, pack) every layer's K/V       [main stream]
  2. residual transport: H2D copy of the residual planes of all layers (one
     allocation per plane kind) from pinned host memory, standing in for
     the network                                              [side stream]
     overlapped with
  3. anchor-only decode attention, one query token per layer   [main stream]
  4. wait for the residual, merge anchor + residual -> codes, one call per
     plane kind over all layers                               [main stream]
  5. verification attention of the 8 drafts over the codes    [main stream]

After the timed steps, further stages are timed on their own (reported
under "stages"): the same decode calls with no transport running, and in
the four transport conditions; the stream ceilings (a device copy and a
uint8 add); the verification of k = 8 drafts at 128K context (32 q / 8 kv
heads, one layer, merged codes + causal BF16 tail), the configuration the
paper's verification latency is quoted for; the decode calls once more with
the 8 BF16 tokens the speculative decoder generated; greedy and sampled
acceptance of 8 drafts over a 128256-entry vocabulary; the batched paged
decode of 16 sequences of 16K-64K tokens in 16-token blocks; the 70B-shaped
overlap run (4 x 128K tokens, 64 q / 8 kv heads: 16 decode steps against
the residual H2D, then merge and verification of 4 drafts, with the overlap
fraction and end-to-end time); the serializer pipeline; the hierarchical
codec; and the 2 + 6 / 6 + 2 split widths.

Every stage is timed with a pair of HIP events around each call (or block of
per-layer calls) after untimed warm-ups (at least 5 calls and at least 50 ms
of them) and reported as the median, with min, max and count: 50 samples
unless stated (50 steps by default; 50 runs of the millisecond-long
transport pipelines).

Printed: one JSON line.  `value` is the anchor-decode attention throughput in
GB/s of algorithmic KV bytes (144 bytes per token per kv head) over all the
timed steps, from HIP events on the stream the kernels run on.

Offline helpers (no GPU) turn rocprofv3 output of this script into the text
summaries kept under profiles/:
  --summarize-trace DIR          kernel-trace CSVs -> per-kernel durations
  --summarize-pmc FETCH WRITE    FETCH_SIZE / WRITE_SIZE CSVs of a run with
                                 --copy-calibration -> HBM bytes per call
  --summarize-copies DIR         kernel + memory-copy trace -> the kernels
                                 inside each host-to-device copy
  --summarize-conditions DIR...  counter runs of the transport conditions
"""
from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import json
import os
import re
import sys
import time
from pathlib import Path

ROOT = Path(__file__).resolve().parent
sys.path.insert(0, str(ROOT))

HBM_PEAK_GBPS = 8000.0
METRIC = "anchor decode-attn KV GB/s (% HBM peak); encode/merge GB/s; verify µs @128k"
WORKLOAD = "llama3-8b-32k"
COPY_CALIBRATION_BYTES = 640 << 20
TRAFFIC_SUMMARY = ROOT / "profiles" / "anchor_decode_llama3-8b-32k_traffic.md"
# sources whose kernels make up one anchor-decode call
DECODE_SOURCES = ["anchor_decode.hip", "split_merge.h", "attention.hip", "lynx_internal.h", "lane_ops.h"]

# algorithmic bytes per unit
ENC_BYTES_PER_ELEM = 2.0 + 0.5 + 0.5 + 0.0625   # read BF16, write 2 nibbles, metadata
MERGE_BYTES_PER_ELEM = 2.0                      # read 0.5 + 0.5, write 1
DECODE_BYTES_PER_TOKEN_HEAD = 64 + 64 + 8 + 8   # K, V nibble rows + V meta + K meta (amortised)
VERIFY_BYTES_PER_TOKEN_HEAD = 128 + 128 + 8 + 8  # K, V code rows + metadata

# timed samples per stage, after untimed warm-ups: at least WARM calls and
# at least WARM_S seconds of them (the part's clocks take tens of ms of
# sustained load to settle: the paged batch decode, 50 calls at a time on one
# pool, runs 157, 143, 141, 140, 138, 137, 135, 133 us from a cold start)
REPS, WARM, WARM_S = 50, 5, 0.05


def summary(samples):
    """Median, min, max and count of a list of timings (us)."""
    s = sorted(samples)
    n = len(s)
    med = s[n // 2] if n % 2 else 0.5 * (s[n // 2 - 1] + s[n // 2])
    return {"median": round(med, 3), "min": round(s[0], 3), "max": round(s[-1], 3), "n": n}


def call_samples(fn, n=REPS, warm=WARM, per=1):
    """us per unit of `fn` (which covers `per` units), one pair of HIP events
    on the current stream around each of n timed calls after untimed ones: at
    least `warm` calls and at least WARM_S seconds of calls."""
    import torch

    t0 = time.perf_counter()
    for _ in range(warm):
        fn()
    torch.cuda.synchronize()
    while time.perf_counter() - t0 < WARM_S:
        for _ in range(max(warm, 1)):
            fn()
        torch.cuda.synchronize()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(n)]
    for a, b in evs:
        a.record()
        fn()
        b.record()
    torch.cuda.synchronize()
    return [a.elapsed_time(b) * 1e3 / per for a, b in evs]


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=50)
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--layers", type=int, default=None, help="override layer count (testing only)")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-layers", type=int, default=24,
                   help="layers of the CPU oracle's decode sample (encode and merge: half, verify: a quarter)")
    p.add_argument("--copy-calibration", action="store_true",
                   help="run one plain device copy of 640 MiB before the steps (counter calibration)")
    p.add_argument("--summarize-trace", metavar="DIR")
    p.add_argument("--summarize-pmc", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"))
    p.add_argument("--summarize-conditions", nargs="+", metavar="DIR",
                   help="per-condition counters of the transport-interference stage from --pmc runs")
    p.add_argument("--transport-trials", type=int, default=8,
                   help="trials per condition of the transport-interference stage (0: skip it)")
    p.add_argument("--summarize-copies", metavar="DIR",
                   help="kernel + memory-copy trace CSVs -> kernels inside each H2D copy")
    p.add_argument("--no-spec-stages", dest="spec_stages", action="store_false",
                   help="skip the decode-with-tail and draft-acceptance stages")
    p.add_argument("--paged-calls", type=int, default=REPS,
                   help="timed paged batch-decode calls (paged-b16-16k-64k; 0 skips the stage)")
    p.add_argument("--no-hier", dest="hier", action="store_false",
                   help="skip the hierarchical-codec stage")
    p.add_argument("--no-split-widths", dest="split_widths", action="store_false",
                   help="skip the 2 + 6 / 6 + 2 split stage")
    p.add_argument("--no-serdes", dest="serdes", action="store_false",
                   help="skip the serializer / deserializer pipeline stage")
    p.add_argument("--no-overlap-70b", dest="overlap_70b", action="store_false",
                   help="skip the 70B-shaped overlap run (70b-overlap-b4-128k)")
    p.add_argument("--verify-128k-calls", type=int, default=REPS,
                   help="timed verification calls at 128K context (0 skips the stage)")
    p.add_argument("--no-ceilings", dest="ceilings", action="store_false",
                   help="skip the plain copy / add stream-rate stage")
    return p.parse_args()


def decode_sources_hash() -> str:
    h = hashlib.sha256()
    for name in DECODE_SOURCES:
        h.update((ROOT / "paper_2607_01831_amd" / "csrc" / name).read_bytes())
    return h.hexdigest()


def stored_traffic():
    """HBM bytes per anchor-decode call from the committed counter summary,
    or None when the decode kernels changed since it was taken."""
    try:
        text = TRAFFIC_SUMMARY.read_text()
    except OSError:
        return None
    fields = {}
    for line in text.splitlines():
        line = line.strip().strip("`")
        if line.startswith(("kernel_sources_sha256:", "traffic_bytes_per_call:")):
            k, v = line.split(":", 1)
            fields[k.strip()] = v.strip()
    if fields.get("kernel_sources_sha256") != decode_sources_hash():
        return None
    try:
        return int(fields["traffic_bytes_per_call"])
    except (KeyError, ValueError):
        return None


# ------------------------------------------------------------ rocprof summaries --

def _csv(dirname, suffix):
    files = glob.glob(os.path.join(dirname, "**", f"*{suffix}"), recursive=True)
    if not files:
        raise SystemExit(f"no *{suffix} under {dirname}")
    with open(files[0], newline="") as f:
        return list(csv.DictReader(f))


def _short(name: str) -> str:
    for key in ("anchor_split_decode_kernel", "anchor_decode_kernel", "attn_combine_kernel", "verify_kernel", "encode_kernel",
                "merge_kernel", "copyBuffer", "hencode_kernel", "hdequant_kernel",
                "deserialize_anchor_kernel", "deserialize_residual_kernel", "merge_split_kernel",
                "dequant_anchor_split_kernel", "argmax_chunk_kernel", "accept_kernel",
                "sample_chunk_kernel", "sample_pick_kernel"):
        if key in name:
            return key
    if "vectorized_elementwise_kernel" in name and "CUDAFunctor_add" in name:
        return "torch add (uint8)"
    return name.split("(")[0][:60]


def _variant(name: str) -> str:
    """A library kernel with its template arguments (the decode of a 32K layer,
    anchor_decode_kernel<4, 0, 4>, and the 70B-shaped one-round decode,
    anchor_decode_kernel<8, 0, 64>, launch the same number of work-items);
    any other kernel by its short name."""
    m = re.search(r"(\w+_kernel)(<[^()]*>)\(", name)
    if m and "lynx::" in name:
        return m.group(1) + m.group(2)
    return _short(name)


# the roofline's call: one 32K-token layer of 8 kv heads, one round of 512
# workgroups of 4 groups each
DECODE_32K_VARIANT = "anchor_decode_kernel<4, 0, 4>"
DECODE_32K_GRID = 512 * 256


def _us(r):
    return (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3


def _grid(r):
    """Work-items of a dispatch (counter CSVs give Grid_Size, trace CSVs X/Y/Z)."""
    if r.get("Grid_Size"):
        return int(r["Grid_Size"])
    return int(r["Grid_Size_X"]) * int(r["Grid_Size_Y"]) * int(r["Grid_Size_Z"])


def _calls(rows, first):
    """Every `first` dispatch (anchor_decode_kernel or verify_kernel) with the
    attn_combine_kernel dispatch right after it on the same queue, if there
    is one (a fused decode has none): one lynx_attn_* call each."""
    rows = sorted(rows, key=lambda r: int(r["Dispatch_Id"]))
    nxt = {}
    for i, r in enumerate(rows):
        for r2 in rows[i + 1:]:
            if r2["Queue_Id"] == r["Queue_Id"]:
                nxt[id(r)] = r2
                break
    calls = []
    for r in rows:
        if _short(r["Kernel_Name"]) == first:
            n = nxt.get(id(r))
            calls.append((r, n if n is not None and _short(n["Kernel_Name"]) == "attn_combine_kernel"
                          else None))
    return calls


def _stats(xs):
    xs = sorted(xs)
    n = len(xs)
    med = xs[n // 2] if n % 2 else 0.5 * (xs[n // 2 - 1] + xs[n // 2])
    return med, xs[0], xs[-1], sum(xs) / n


def summarize_trace(dirname):
    """Kernel durations of a rocprofv3 --kernel-trace run, per kernel and grid
    size (work-items), and per API call (decode or verify kernel plus its
    combine kernel, when there is one)."""
    rows = _csv(dirname, "kernel_trace.csv")
    by = {}
    for r in rows:
        by.setdefault((_variant(r["Kernel_Name"]), _grid(r)), []).append(_us(r))
    print("| kernel | grid (work-items) | dispatches | median us | min us | max us | mean us |")
    print("|---|---|---|---|---|---|---|")
    for (n, g), ds in sorted(by.items(), key=lambda kv: -sum(kv[1])):
        med, lo, hi, mean = _stats(ds)
        print(f"| {n} | {g} | {len(ds)} | {med:.2f} | {lo:.2f} | {hi:.2f} | {mean:.2f} |")
    print()
    print("| first kernel of the call | grid (work-items) | calls | first kernel median us | combine median us | "
          "call (first start to last end) median us |")
    print("|---|---|---|---|---|---|")
    for first in ("anchor_decode_kernel", "anchor_split_decode_kernel", "verify_kernel"):
        groups = {}
        for a, b in _calls(rows, first):
            groups.setdefault((_variant(a["Kernel_Name"]), _grid(a)), []).append((a, b))
        for (v, g), cs in sorted(groups.items()):
            k = _stats([_us(a) for a, _ in cs])[0]
            comb = [_us(b) for _, b in cs if b is not None]
            c = f"{_stats(comb)[0]:.2f}" if comb else "(fused)"
            span = _stats([(int((b or a)["End_Timestamp"]) - int(a["Start_Timestamp"])) / 1e3
                           for a, b in cs])[0]
            print(f"| {v} | {g} | {len(cs)} | {k:.2f} | {c} | {span:.2f} |")


def summarize_pmc(fetch_dir, write_dir):
    """HBM bytes per dispatch from two rocprofv3 --pmc runs (FETCH_SIZE, then
    WRITE_SIZE, KiB per dispatch) of a run with --copy-calibration: each
    counter scaled by what it reads for the plain copy of known size.  Per
    kernel and grid size, and per 32K-layer anchor-decode call (the
    roofline's kernel: 8 kv heads x 32768 tokens, one round of 512
    workgroups)."""
    def per_dispatch(dirname, counter):
        return {int(r["Dispatch_Id"]): (r, float(r["Counter_Value"]))
                for r in _csv(dirname, "counter_collection.csv") if r["Counter_Name"] == counter}

    fetch = per_dispatch(fetch_dir, "FETCH_SIZE")
    write = per_dispatch(write_dir, "WRITE_SIZE")

    def copy_kib(table):
        cands = [v for r, v in table.values() if _short(r["Kernel_Name"]) == "copyBuffer"]
        if not cands:
            raise SystemExit("no copy kernel in the counter run (use --copy-calibration)")
        return max(cands)

    known_kib = COPY_CALIBRATION_BYTES / 1024
    f_fetch = known_kib / copy_kib(fetch)
    f_write = known_kib / copy_kib(write)
    print(f"copy calibration: a plain copy of {COPY_CALIBRATION_BYTES} bytes reads FETCH_SIZE "
          f"{copy_kib(fetch):.0f} KiB and WRITE_SIZE {copy_kib(write):.0f} KiB; scale factors "
          f"fetch {f_fetch:.4f}, write {f_write:.4f}")
    print()

    def grouped(table, f):
        g = {}
        for r, v in table.values():
            g.setdefault((_variant(r["Kernel_Name"]), _grid(r)), []).append(v * 1024 * f)
        return g

    gf, gw = grouped(fetch, f_fetch), grouped(write, f_write)
    print("| kernel | grid (work-items) | dispatches | read MB per dispatch | written MB per dispatch |")
    print("|---|---|---|---|---|")
    for key in sorted(gf, key=lambda k: -sum(gf[k])):
        if key[0] == "copyBuffer" or key not in gw:
            continue
        rd = sum(gf[key]) / len(gf[key]) / 1e6
        wr = sum(gw[key]) / len(gw[key]) / 1e6
        print(f"| {key[0]} | {key[1]} | {len(gf[key])} | {rd:.2f} | {wr:.2f} |")
    # one 32K-layer decode call: the decode kernel with the 32K layer's grid
    # (and its combine, when the call has one)
    rows_f = [r for r, _ in fetch.values()]
    per = []
    for a, b in _calls(rows_f, "anchor_decode_kernel"):
        if _variant(a["Kernel_Name"]) != DECODE_32K_VARIANT or _grid(a) != DECODE_32K_GRID:
            continue
        ids = [int(a["Dispatch_Id"])] + ([int(b["Dispatch_Id"])] if b is not None else [])
        if all(i in write for i in ids):
            per.append(sum(fetch[i][1] * 1024 * f_fetch + write[i][1] * 1024 * f_write for i in ids))
    print()
    if per:
        print(f"32K-layer anchor-decode calls measured: {len(per)}")
        print(f"kernel_sources_sha256: {decode_sources_hash()}")
        print(f"traffic_bytes_per_call: {int(round(sum(per) / len(per)))}")


def summarize_copies(dirname):
    """Host-to-device copies longer than 1 ms in a rocprofv3 --kernel-trace
    --memory-copy-trace run, grouped by what ran while each was in flight
    (kernel variants and their dispatch counts) and by duration to the
    millisecond: copies per group, median duration, median time each kernel
    spent inside the copy's window."""
    kt = _csv(dirname, "kernel_trace.csv")
    mc = _csv(dirname, "memory_copy_trace.csv")
    big = [r for r in mc if r["Direction"].endswith("HOST_TO_DEVICE")
           and int(r["End_Timestamp"]) - int(r["Start_Timestamp"]) > 1_000_000]
    groups, order = {}, []
    for r in big:
        s0, e0 = int(r["Start_Timestamp"]), int(r["End_Timestamp"])
        inside = {}
        for k in kt:
            ov = min(int(k["End_Timestamp"]), e0) - max(int(k["Start_Timestamp"]), s0)
            if ov > 0:
                c = inside.setdefault((_variant(k["Kernel_Name"]), _grid(k)), [0, 0.0])
                c[0] += 1
                c[1] += ov / 1e3
        key = ((e0 - s0) // 1_000_000, tuple(sorted((n, g, c) for (n, g), (c, _) in inside.items())))
        if key not in groups:
            groups[key] = []
            order.append(key)
        groups[key].append(((e0 - s0) / 1e3, {(n, g): t for (n, g), (_, t) in inside.items()}))
    print("| H2D copies | median duration us | kernels inside each copy's window (kernel [grid] x dispatches: "
          "median us inside) |")
    print("|---|---|---|")
    for key in order:
        cs = groups[key]
        desc = "; ".join(f"{n} [{g}] x{c}: {_stats([t[(n, g)] for _, t in cs])[0]:.1f}"
                         for n, g, c in key[1]) or "none"
        print(f"| {len(cs)} | {_stats([d for d, _ in cs])[0]:.1f} | {desc} |")


TRANSPORT_CONDITIONS = ("alone", "h2d running", "after encode", "after encode, h2d running")


def transport_interference(encode_all, decode_all, start_h2d, trials):
    """The 32 decode calls in four conditions, interleaved trial by trial:
    alone; with the residual H2D running on the side stream; right after the
    encode of every layer; right after the encode with the H2D running (the
    step's own order).  Before each decode run a marker kernel (a fill of
    (c + 1) << 16 int16 values) names condition c for a counter run.  Returns
    us per call (median, min, max) per condition."""
    import torch

    main_s = torch.cuda.current_stream()
    res = {c: [] for c in TRANSPORT_CONDITIONS}
    for t in range(trials + 1):
        for c, name in enumerate(TRANSPORT_CONDITIONS):
            torch.cuda.synchronize()
            if c >= 2:
                encode_all()
            if c in (1, 3):
                done = torch.cuda.Event()
                done.record(main_s)
                start_h2d(done)
            torch.full(((c + 1) << 16,), c, dtype=torch.int16, device=main_s.device)
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(main_s)
            n = decode_all()
            b.record(main_s)
            torch.cuda.synchronize()
            if t > 0:  # the first round warms up
                res[name].append(a.elapsed_time(b) * 1e3 / n)
    return {name: summary(v) for name, v in res.items()}


def summarize_conditions(dirs):
    """Counters of the anchor-decode dispatches of a --pmc run per condition of
    the transport-interference stage (the condition is named by the int16 fill
    before its decode run), mean per dispatch; then the derived latencies."""
    per = {}
    for d in dirs:
        rows = sorted(_csv(d, "counter_collection.csv"), key=lambda r: int(r["Dispatch_Id"]))
        disp = {}
        for r in rows:
            disp.setdefault(int(r["Dispatch_Id"]), []).append(r)
        markers = sorted({_grid(rs[0]) for rs in disp.values()
                          if "FillFunctor<short>" in rs[0]["Kernel_Name"]})
        if len(markers) != len(TRANSPORT_CONDITIONS):
            raise SystemExit(f"{d}: expected {len(TRANSPORT_CONDITIONS)} marker sizes, found {markers}")
        cond = None
        for i in sorted(disp):
            rs = disp[i]
            name = rs[0]["Kernel_Name"]
            if "FillFunctor<short>" in name:
                cond = markers.index(_grid(rs[0]))
            elif cond is not None and _variant(name) == DECODE_32K_VARIANT and _grid(rs[0]) == DECODE_32K_GRID:
                for r in rs:
                    per.setdefault(r["Counter_Name"], {}).setdefault(cond, []).append(
                        float(r["Counter_Value"]))
                per.setdefault("duration_us", {}).setdefault(cond, []).append(_us(rs[0]))
    names = sorted(per)
    print("| counter (mean per 32K decode dispatch) | " + " | ".join(TRANSPORT_CONDITIONS) + " |")
    print("|---|" + "---|" * len(TRANSPORT_CONDITIONS))
    mean = lambda xs: sum(xs) / len(xs) if xs else float("nan")
    for n in names:
        print(f"| {n} | " + " | ".join(f"{mean(per[n].get(c, [])):.1f}"
                                      for c in range(len(TRANSPORT_CONDITIONS))) + " |")
    for num, den, label in (("TCC_EA0_RDREQ_LEVEL_sum", "TCC_EA0_RDREQ_sum", "L2 -> memory read latency (cycles)"),
                            ("TCC_EA0_WRREQ_LEVEL_sum", "TCC_EA0_WRREQ_sum", "L2 -> memory write latency (cycles)"),
                            ("TCP_TCC_READ_REQ_LATENCY_sum", "TCP_TCC_READ_REQ_sum", "L1 -> L2 read latency (cycles)")):
        if num in per and den in per:
            print(f"| {label} | " + " | ".join(
                f"{mean(per[num].get(c, [])) / max(mean(per[den].get(c, [])), 1e-9):.0f}"
                for c in range(len(TRANSPORT_CONDITIONS))) + " |")


def stream_ceilings(dev):
    """Practical HBM stream rates on this part, with torch's own kernels over
    buffers larger than the 256 MB last-level cache: a device-to-device copy
    (reads and writes one byte per byte, as the merge does) and a uint8 add
    c = a + b (reads two bytes per byte written, as the encode does); median
    over REPS calls, bytes read + written per second."""
    import torch

    n = 512 << 20
    a = torch.ones(n, dtype=torch.uint8, device=dev)
    b = torch.ones(n, dtype=torch.uint8, device=dev)
    c = torch.empty(n, dtype=torch.uint8, device=dev)
    copy = summary(call_samples(lambda: c.copy_(a)))
    add = summary(call_samples(lambda: torch.add(a, b, out=c)))
    del a, b, c
    return {"stream_ceilings": {
        "copy_512MiB_us": copy["median"], "copy_GBps": round(2 * n / (copy["median"] * 1e-6) / 1e9, 1),
        "add_u8_512MiB_us": add["median"], "add_u8_GBps": round(3 * n / (add["median"] * 1e-6) / 1e9, 1)}}


# --------------------------------------------------------------- CPU baseline --

def verify_128k(calls, dev):
    """Verification at 128K context (32 q / 8 kv heads, k = 8 drafts with
    their causal BF16 tail) over merged codes: two encoded layers, used in
    turn so that no call finds the previous one's bytes in the 256 MB
    last-level cache; a pair of HIP events around each call.  Then, on the
    same layer, the anchor-only decode of draft 0 against the verification of
    draft 0 over the merged codes without the tail: the deviation the
    residual removes (vNMSE = E ||o_anchor - o_full||^2 / ||o_full||^2 over
    the query heads, and the largest absolute difference)."""
    import torch

    from paper_2607_01831_amd import inputs, lynx

    w3 = inputs.WORKLOADS["llama3-8b-verify-128k"]
    T3, Hkv, Hq, nq = w3.context, w3.Hkv, w3.Hq, w3.drafts
    L3 = lynx.contiguous_layout(Hkv, 1, T3)
    table = torch.zeros(1, 1, dtype=torch.int32, device=dev)
    lens = torch.tensor([T3], dtype=torch.int32, device=dev)
    pools, qs, kns, vns = [], [], [], []
    for layer in range(2):
        pool = lynx.KVPool.allocate(L3, 1, device=dev)
        k = inputs.kv(w3, "k", layer=layer, device=dev)
        v = inputs.kv(w3, "v", layer=layer, device=dev)
        pool.encode(0, T3, table, k, v)
        pool.merge()
        del k, v
        pools.append(pool)
        qs.append(inputs.queries(w3, layer=layer, nq=nq, device=dev))
        kn, vn = inputs.drafts_kv(w3, layer=layer, device=dev)
        kns.append(kn)
        vns.append(vn)
    out = torch.empty(1, nq, Hq, 128, dtype=torch.bfloat16, device=dev)
    ws = lynx.workspace(L3, 1, Hq, nq, T3)
    turn = [0]

    def call():
        i = turn[0]
        turn[0] += 1
        p = pools[i % 2]
        lynx.lynx_attn_verify(L3, 1, Hq, nq, T3, lens, table, p.k_codes, p.v_codes, p.meta,
                              qs[i % 2], kns[i % 2], vns[i % 2], out, ws)

    st = summary(call_samples(call, n=calls))
    us = st["median"]
    gbps = T3 * Hkv * VERIFY_BYTES_PER_TOKEN_HEAD / (us * 1e-6) / 1e9
    # anchor-only decode vs the merged-code verification, draft 0, no tail
    p = pools[0]
    q0 = qs[0][:, 0].contiguous()                      # [1][Hq][128]
    o_anc = torch.empty(1, Hq, 128, dtype=torch.bfloat16, device=dev)
    o_full = torch.empty(1, 1, Hq, 128, dtype=torch.bfloat16, device=dev)
    lynx.lynx_attn_anchor_decode(L3, 1, Hq, T3, lens, table, p.k_anc, p.v_anc, p.meta, q0, o_anc,
                                 None, ws)
    lynx.lynx_attn_verify(L3, 1, Hq, 1, T3, lens, table, p.k_codes, p.v_codes, p.meta,
                          q0.view(1, 1, Hq, 128), None, None, o_full, ws)
    torch.cuda.synchronize()
    oa, of = o_anc[0].float(), o_full[0, 0].float()
    vn = float(((oa - of).pow(2).sum(dim=-1) / of.pow(2).sum(dim=-1)).mean())
    del pools
    return {"verify_128k_us": round(us, 2), "verify_128k_us_min": st["min"],
            "verify_128k_us_max": st["max"], "verify_128k_calls": st["n"],
            "verify_128k_GBps": round(gbps, 2), "verify_128k_frac": round(gbps / HBM_PEAK_GBPS, 4),
            "anchor_vs_full_128k": {"query": "draft 0, no tail", "vnmse": float(f"{vn:.3g}"),
                                    "max_abs_diff": round(float((oa - of).abs().max()), 5)}}


def paged_decode_stage(calls, dev):
    """Batched paged anchor decode (paged-b16-16k-64k): 16 sequences with
    lengths uniform on [16384, 65536] in 16-token blocks under a random block
    table over one pool, 32 q / 8 kv heads, one query token per sequence.  The
    pool's anchor planes (about 755 MB) exceed the 256 MB last-level cache, so
    every call reads them from HBM; HIP events around the timed calls."""
    import torch

    from paper_2607_01831_amd import inputs, lynx

    w = inputs.WORKLOADS["paged-b16-16k-64k"]
    lens = inputs.seq_lengths(w)
    table, n_blocks = inputs.paged_block_table(lens, w.block_tokens,
                                               inputs.seed_of(w.wid, inputs.T_BLOCKS))
    L = lynx.Layout(num_kv_heads=w.Hkv, block_tokens=w.block_tokens,
                    max_blocks_per_seq=table.shape[1], num_blocks=n_blocks, max_tokens=w.context)
    pool = lynx.KVPool.allocate(L, w.batch, device=dev, codes=False)
    tdev, ldev = table.to(dev), lens.to(dev)
    for b in range(w.batch):
        T = int(lens[b])
        k = inputs.kv(w, "k", seq=b, T=T, device=dev)
        v = inputs.kv(w, "v", seq=b, T=T, device=dev)
        pool.encode(b, T, tdev, k, v)
        del k, v
    q = inputs.queries(w, device=dev)
    out = torch.empty(w.batch, w.Hq, 128, dtype=torch.bfloat16, device=dev)
    max_len = int(lens.max())
    ws = lynx.workspace(L, w.batch, w.Hq, 1, max_len, device=dev)

    def call():
        lynx.lynx_attn_anchor_decode(L, w.batch, w.Hq, max_len, ldev, tdev, pool.k_anc, pool.v_anc,
                                     pool.meta, q, out, None, ws)

    st = summary(call_samples(call, n=calls))
    us = st["median"]
    nbytes = int(lens.sum()) * w.Hkv * DECODE_BYTES_PER_TOKEN_HEAD
    gbps = nbytes / (us * 1e-6) / 1e9
    del pool
    return {"paged_b16_decode_us": round(us, 2), "paged_b16_decode_us_min": st["min"],
            "paged_b16_decode_us_max": st["max"], "paged_b16_decode_calls": st["n"],
            "paged_b16_decode_MB": round(nbytes / 1e6, 1),
            "paged_b16_decode_GBps": round(gbps, 2),
            "paged_b16_decode_frac": round(gbps / HBM_PEAK_GBPS, 4)}


def overlap_70b_stage(dev):
    """The 70B-shaped overlap run (70b-overlap-b4-128k): 4 sequences x 131072
    tokens, 64 q / 8 kv heads.  Timed with HIP events over REPS runs (medians;
    every decode step also alone), each part alone and then overlapped: 16 anchor-decode steps (a fresh query per step); the
    H2D of the residual planes (512 MiB) from pinned host memory on a side
    stream; both at once; then merge of both planes and verification of
    k = 4 drafts with their causal BF16 tail.  overlap = (t_dec + t_h2d -
    t_both) / min(t_dec, t_h2d) (1 = the shorter one fully hidden);
    end_to_end = t_both + merge + verify."""
    import torch

    from paper_2607_01831_amd import inputs, lynx

    w = inputs.WORKLOADS["70b-overlap-b4-128k"]
    B, T, Hkv, Hq, nq, steps = w.batch, w.context, w.Hkv, w.Hq, w.drafts, w.decode_steps
    L = lynx.contiguous_layout(Hkv, B, T)
    pool = lynx.KVPool.allocate(L, B, device=dev)
    table = inputs.contiguous_block_table(B).to(dev)
    lens = torch.full((B,), T, dtype=torch.int32, device=dev)
    for b in range(B):
        k = inputs.kv(w, "k", seq=b, device=dev)
        v = inputs.kv(w, "v", seq=b, device=dev)
        pool.encode(b, T, table, k, v)
        del k, v
    host_k = pool.k_res.cpu().pin_memory()
    host_v = pool.v_res.cpu().pin_memory()
    recv_k, recv_v = torch.empty_like(pool.k_res), torch.empty_like(pool.v_res)
    qs = [inputs.queries(w, step=s, device=dev) for s in range(steps)]
    qv = inputs.queries(w, step=steps, nq=nq, device=dev)
    kn, vn = inputs.drafts_kv(w, device=dev)
    out = torch.empty(B, Hq, 128, dtype=torch.bfloat16, device=dev)
    outv = torch.empty(B, nq, Hq, 128, dtype=torch.bfloat16, device=dev)
    nws = max(lynx.lynx_attn_workspace_bytes(L, B, Hq, 1, T), lynx.lynx_attn_workspace_bytes(L, B, Hq, nq, T))
    # zero-filled: the arrival counters at the workspace's head start at zero
    ws = torch.zeros(nws, dtype=torch.uint8, device=dev)
    main_s, side = torch.cuda.current_stream(), torch.cuda.Stream()
    ev = lambda: torch.cuda.Event(enable_timing=True)

    def decode_steps(step_evs=None):
        for s in range(steps):
            if step_evs is not None:
                step_evs[s][0].record(main_s)
            lynx.lynx_attn_anchor_decode(L, B, Hq, T, lens, table, pool.k_anc, pool.v_anc, pool.meta,
                                         qs[s], out, None, ws)
            if step_evs is not None:
                step_evs[s][1].record(main_s)

    def transport(after):
        side.wait_event(after)
        with torch.cuda.stream(side):
            recv_k.copy_(host_k, non_blocking=True)
            recv_v.copy_(host_v, non_blocking=True)
            done = ev()
            done.record(side)
        return done

    def merge_verify():
        lynx.lynx_kv_merge(pool.k_anc, recv_k, pool.k_codes)
        lynx.lynx_kv_merge(pool.v_anc, recv_v, pool.v_codes)
        m = ev()
        m.record(main_s)
        lynx.lynx_attn_verify(L, B, Hq, nq, T, lens, table, pool.k_codes, pool.v_codes, pool.meta,
                              qv, kn, vn, outv, ws)
        return m

    t0 = time.perf_counter()
    decode_steps()
    merge_verify()
    torch.cuda.synchronize()
    while time.perf_counter() - t0 < WARM_S:
        decode_steps()
        torch.cuda.synchronize()
    runs, step_us = [], []
    for _ in range(REPS):
        # decode alone (a pair of events around each step too)
        a0, a1 = ev(), ev()
        sev = [(ev(), ev()) for _ in range(steps)]
        a0.record(main_s); decode_steps(sev); a1.record(main_s)
        torch.cuda.synchronize()
        step_us += [x.elapsed_time(y) * 1e3 for x, y in sev]
        # transport alone
        h0 = ev(); h0.record(main_s)
        h1 = transport(h0)
        torch.cuda.synchronize()
        # both, then merge + verify
        b0 = ev(); b0.record(main_s)
        hb = transport(b0)
        decode_steps()
        main_s.wait_event(hb)
        b1 = ev(); b1.record(main_s)
        m1 = merge_verify()
        v1 = ev(); v1.record(main_s)
        torch.cuda.synchronize()
        runs.append({"t_dec": a0.elapsed_time(a1), "t_h2d": h0.elapsed_time(h1),
                     "t_both": b0.elapsed_time(b1), "merge": b1.elapsed_time(m1),
                     "verify": m1.elapsed_time(v1), "e2e": b0.elapsed_time(v1)})
    # the decode step on its own, called back to back after the warm-up: the
    # kernel's sustained rate, beside the in-run figure above (whose steps start
    # after the merge, the verification and the transport's wait)
    sustained = summary(call_samples(lambda: decode_steps(), n=REPS, per=steps))
    # medians over the runs (ms)
    best = {k: summary([r_[k] for r_ in runs])["median"] for k in runs[0]}
    t_dec, t_h2d, t_both = best["t_dec"], best["t_h2d"], best["t_both"]
    st_step = summary(step_us)
    dec_bytes = B * T * Hkv * DECODE_BYTES_PER_TOKEN_HEAD
    res_bytes = host_k.numel() + host_v.numel()
    merge_bytes = 2 * B * T * Hkv * 128 * MERGE_BYTES_PER_ELEM
    ver_bytes = B * T * Hkv * VERIFY_BYTES_PER_TOKEN_HEAD
    us_step = st_step["median"]
    r = {
        "runs": len(runs),
        "decode_us_per_step": round(us_step, 2),
        "decode_us_per_step_min": st_step["min"],
        "decode_us_per_step_max": st_step["max"],
        "decode_steps_timed": st_step["n"],
        "decode_us_per_step_sustained": sustained["median"],
        "decode_frac_sustained": round(dec_bytes / (sustained["median"] * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4),
        "decode_GBps": round(dec_bytes / (us_step * 1e-6) / 1e9, 2),
        "decode_frac": round(dec_bytes / (us_step * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4),
        "decode_16_steps_us": round(t_dec * 1e3, 1),
        "h2d_us": round(t_h2d * 1e3, 1),
        "h2d_GBps": round(res_bytes / (t_h2d * 1e-3) / 1e9, 2),
        "both_us": round(t_both * 1e3, 1),
        "overlap": round(max(0.0, min(1.0, (t_dec + t_h2d - t_both) / min(t_dec, t_h2d))), 3),
        "merge_us": round(best["merge"] * 1e3, 1),
        "merge_GBps": round(merge_bytes / (best["merge"] * 1e-3) / 1e9, 2),
        "verify_k4_us": round(best["verify"] * 1e3, 1),
        "verify_k4_GBps": round(ver_bytes / (best["verify"] * 1e-3) / 1e9, 2),
        "end_to_end_us": round(best["e2e"] * 1e3, 1),
    }
    del pool, host_k, host_v
    return {"overlap_70b_b4_128k": r}


def serdes_pipeline_stage(dev, T, Hkv, K, V, n_layers, side):
    """The prioritized transmission of Sec. 4.2 over the workload's layers, one
    KV object per layer, on one GPU standing in for both instances:

      sender compute   lynx_kv_serialize of layer l into one of three anchor
                       buffers (reused once layer l - 3's anchor has left) and
                       its own residual buffer
      sender NIC       D2H of every anchor buffer, in layer order, through a
                       ring of four pinned host slots (the wire); the residual
                       buffers follow once every anchor has arrived (strict
                       priority)
      receiver NIC     H2D of each buffer into one of two receive buffers
      receiver compute lynx_kv_deserialize_anchor of every layer (the Anchor
                       phase: decoding could start when it ends), then
                       lynx_kv_deserialize_residual (the Residual phase)

    Three streams at the default priority: every kernel on the main stream
    (the receiver's kernel for transfer m - 2 issued after the sender's for
    m, so neither waits behind the other), the sends on the side stream, the
    receives on a third.  The send and receive of this loopback share one PCIe link, which
    carries both directions at once (≈56 GB/s each).  HIP events give the
    times, relative to the first serialize, medians over ten runs; the same pipeline without its
    kernels gives the wire alone.  The received pool is checked against the
    direct encode + merge of the same layers."""
    import torch

    from paper_2607_01831_amd import lynx

    na, nr = lynx.lynx_serialized_bytes(Hkv, T)
    L = lynx.contiguous_layout(Hkv, 1, T)
    table = torch.zeros(1, 1, dtype=torch.int32, device=dev)
    u8 = dict(dtype=torch.uint8, device=dev)
    n_tx, n_wire = 3, 4
    tx_anc = [torch.empty(na, **u8) for _ in range(n_tx)]
    tx_res = [torch.empty(nr, **u8) for _ in range(n_layers)]
    rx = {"a": [torch.empty(na, **u8) for _ in range(2)], "r": [torch.empty(nr, **u8) for _ in range(2)]}
    # the wire: a ring of pinned host slots, as a NIC's registered buffers
    ring = [torch.empty(max(na, nr), dtype=torch.uint8).pin_memory() for _ in range(n_wire)]
    recv, _ = lynx.KVPool.allocate_layers(L, 1, n_layers, device=dev)
    main_s, s_send, s_recv = torch.cuda.current_stream(), side, torch.cuda.Stream()
    ev = lambda: torch.cuda.Event(enable_timing=True)

    def run(kernels=True):
        # transfers in wire order: every anchor, then every residual; every
        # event is recorded (enqueued) before any stream waits on it
        N = n_layers
        xfers = [("a", l) for l in range(N)] + [("r", l) for l in range(N)]
        M = len(xfers)
        ser = [ev() for _ in range(N)]
        sent, got, des = ([ev() for _ in range(M)] for _ in range(3))
        t0 = ev()
        t0.record(main_s)

        def deserialize(m):
            kind, l = xfers[m]
            main_s.wait_event(got[m])
            if kernels:
                p = recv[l]
                if kind == "a":
                    lynx.lynx_kv_deserialize_anchor(L, 0, 0, T, table, rx["a"][l % 2], p.k_anc, p.v_anc, p.meta)
                else:
                    lynx.lynx_kv_deserialize_residual(L, 0, 0, T, table, rx["r"][l % 2], p.k_anc, p.v_anc,
                                                      p.k_codes, p.v_codes)
            des[m].record(main_s)

        for m, (kind, l) in enumerate(xfers):
            nbytes = na if kind == "a" else nr
            if kind == "a":                          # sender compute
                if l >= n_tx:
                    main_s.wait_event(sent[l - n_tx])    # its send buffer has left
                if kernels:
                    lynx.lynx_kv_serialize(Hkv, T, K[l], V[l], tx_anc[l % n_tx], tx_res[l])
                ser[l].record(main_s)
                s_send.wait_event(ser[l])
            elif l == 0:
                s_send.wait_event(got[N - 1])            # residuals once every anchor is in
            if m >= n_wire:
                s_send.wait_event(got[m - n_wire])       # its wire slot has been read
            with torch.cuda.stream(s_send):              # sender NIC
                src = tx_anc[l % n_tx] if kind == "a" else tx_res[l]
                ring[m % n_wire][:nbytes].copy_(src, non_blocking=True)
                sent[m].record(s_send)
            if m >= 2:                                   # receiver compute, two transfers behind
                deserialize(m - 2)
            s_recv.wait_event(sent[m])
            if m >= 2 and xfers[m - 2][0] == kind:
                s_recv.wait_event(des[m - 2])            # its receive buffer is free
            with torch.cuda.stream(s_recv):              # receiver NIC
                rx[kind][l % 2].copy_(ring[m % n_wire][:nbytes], non_blocking=True)
                got[m].record(s_recv)
        deserialize(M - 2)
        deserialize(M - 1)
        torch.cuda.synchronize()
        ms = lambda e: t0.elapsed_time(e)
        return {"serialized": ms(ser[-1]), "anchors_sent": ms(sent[N - 1]), "anchor_ready": ms(des[N - 1]),
                "residuals_sent": ms(sent[-1]), "full_ready": ms(des[-1])}

    run()
    piped, wires = [], []
    for _ in range(REPS):
        piped.append(run())
        wires.append(run(kernels=False))
    # medians over the runs (the pinned-host copy rate varies run to run)
    best = {k: summary([r_[k] for r_ in piped])["median"] for k in piped[0]}
    wire = {k: summary([r_[k] for r_ in wires])["median"] for k in wires[0]}
    full_spread = summary([r_["full_ready"] for r_ in piped])
    run()
    # each kernel alone: median over blocks of all layers (ms per block)
    def alone(fn):
        return summary(call_samples(fn, n=REPS, warm=2))["median"] * 1e-3
    t_ser = alone(lambda: [lynx.lynx_kv_serialize(Hkv, T, K[l], V[l], tx_anc[l % n_tx], tx_res[l])
                           for l in range(n_layers)])
    t_da = alone(lambda: [lynx.lynx_kv_deserialize_anchor(L, 0, 0, T, table, rx["a"][l % 2], recv[l].k_anc,
                                                          recv[l].v_anc, recv[l].meta) for l in range(n_layers)])
    run()  # the loop above scattered the last receive buffers into every layer
    t_dr = alone(lambda: [lynx.lynx_kv_deserialize_residual(L, 0, 0, T, table, rx["r"][l % 2], recv[l].k_anc,
                                                            recv[l].v_anc, recv[l].k_codes, recv[l].v_codes)
                          for l in range(n_layers)])
    run()
    elems = T * Hkv * 128 * 2
    us_l = lambda t: t * 1e3 / n_layers
    r = {
        "objects": n_layers,
        "anchor_MB_per_object": round(na / 1e6, 2),
        "residual_MB_per_object": round(nr / 1e6, 2),
        "serialize_us_per_object": round(us_l(t_ser), 2),
        "serialize_GBps": round(elems * ENC_BYTES_PER_ELEM * n_layers / (t_ser * 1e-3) / 1e9, 1),
        "deserialize_anchor_us_per_object": round(us_l(t_da), 2),
        "deserialize_anchor_GBps": round(2 * na * n_layers / (t_da * 1e-3) / 1e9, 1),
        "deserialize_residual_us_per_object": round(us_l(t_dr), 2),
        "deserialize_residual_GBps": round(T * Hkv * 512 * n_layers / (t_dr * 1e-3) / 1e9, 1),
        "runs": len(piped),
        "pipelined_ms": {k: round(v, 3) for k, v in best.items()},
        "pipelined_full_ready_ms_min_max": [full_spread["min"], full_spread["max"]],
        "wire_only_ms": {k: round(v, 3) for k, v in wire.items()},
        "wire_GBps_per_direction": round((na + nr) * n_layers / (wire["full_ready"] * 1e-3) / 1e9, 2),
        "anchor_ready_over_full": round(best["anchor_ready"] / best["full_ready"], 3),
        # share of the serialize + anchor-phase kernel time hidden behind the wire
        "compute_hidden": round(max(0.0, min(1.0, 1.0 - (best["anchor_ready"] - wire["anchor_ready"])
                                             / max(t_ser + t_da, 1e-9))), 3),
    }
    # the receiver's pool equals the direct encode + merge of the same layers
    direct = lynx.KVPool.allocate(L, 1, device=dev)
    ok = True
    for l in (0, n_layers // 2, n_layers - 1):
        direct.encode(0, T, table, K[l], V[l])
        direct.merge()
        for name in ("k_anc", "v_anc", "k_codes", "v_codes"):
            ok &= bool(torch.equal(getattr(recv[l], name), getattr(direct, name)))
        for name in ("k_scale", "k_zero", "v_scale", "v_zero"):
            ok &= bool(torch.equal(getattr(recv[l].meta, name), getattr(direct.meta, name)))
    r["received_equals_encode"] = ok
    del tx_anc, tx_res, rx, ring, recv, direct
    return {"serdes_pipeline": r}


def hier_codec_stage(dev, T, Hkv, Hq, K, V, Q, pools, L, n_layers, alphas=(255.0, 1.0)):
    """The paper's own hierarchical codec (Alg. 1) on the workload's layers,
    in its three variants (Alg. 1's biased split, the centred split that
    keeps every code, the single 4-bit code): encode, and dequantization of
    the anchor alone and of the merged codes to BF16 pages, each timed over
    all layers in turn (HIP events); then the compression error
    vNMSE = E ||o_hat - o||^2 / ||o||^2, o the attention output of each
    layer's decode query (first four layers, every query head) over the
    exact BF16 cache and o_hat the same over a compressed one: the uniform
    codec through the anchor-decode and verify kernels, the hierarchical one
    through its BF16 pages and plain fp32 attention.  alpha is not given by
    the paper; the first value is the one timed."""
    import torch

    from paper_2607_01831_amd import lynx

    table = torch.zeros(1, 1, dtype=torch.int32, device=dev)
    lens = torch.tensor([T], dtype=torch.int32, device=dev)
    # layer l encodes into pool l % R and is dequantized from there: R pools
    # hold more than the last-level cache, so every timed call starts cold
    R = 12
    hps = [lynx.KVPool.allocate(L, 1, device=dev) for _ in range(R)]
    hms = [lynx.HMeta.empty(L, 1, device=dev) for _ in range(R)]
    hp, hm = hps[0], hms[0]
    ko = torch.empty(T, Hkv, 128, dtype=torch.bfloat16, device=dev)
    vo = torch.empty_like(ko)
    ev = lambda: torch.cuda.Event(enable_timing=True)
    a0 = alphas[0]
    variants = {"biased": lynx.LYNX_HQ_BIASED, "centred": lynx.LYNX_HQ_CENTRED, "int4": lynx.LYNX_HQ_INT4}

    def timed(fn):
        """Median us per layer over REPS blocks of all layers."""
        return summary(call_samples(fn, n=REPS, warm=2, per=n_layers))["median"]

    def encode(l, a, vid, into=None):
        res = vid != lynx.LYNX_HQ_INT4
        p, m = (hps[l % R], hms[l % R]) if into is None else into
        lynx.lynx_hkv_encode(L, 0, T, table, K[l], V[l], a, vid, p.k_anc, p.v_anc,
                             p.k_res if res else None, p.v_res if res else None, m)

    elems = T * Hkv * 128 * 2
    meta_b = 4.0 * 2 * (1 / 256 + 1 / 32)          # page and chunk fp32 pairs per element
    r = {"alpha": a0, "timed": {}}
    for name, vid in variants.items():
        res = vid != lynx.LYNX_HQ_INT4
        t_enc = timed(lambda: [encode(l, a0, vid) for l in range(n_layers)])
        t_da = timed(lambda: [lynx.lynx_hkv_dequant(L, 0, T, table, False, hps[l % R].k_anc, hps[l % R].v_anc,
                                                    a0, vid, hms[l % R], ko, vo) for l in range(n_layers)])
        t = {"encode_us_per_layer": round(t_enc, 2),
             "encode_GBps": round(elems * (2 + (1 if res else 0.5) + meta_b) / (t_enc * 1e-6) / 1e9, 1),
             "dequant_anchor_us_per_layer": round(t_da, 2),
             "dequant_anchor_GBps": round(elems * (0.5 + meta_b + 2) / (t_da * 1e-6) / 1e9, 1)}
        if res:
            for p in hps:
                p.merge()
            t_df = timed(lambda: [lynx.lynx_hkv_dequant(L, 0, T, table, True, hps[l % R].k_codes,
                                                        hps[l % R].v_codes, a0, vid, hms[l % R], ko, vo)
                                  for l in range(n_layers)])
            t["dequant_full_us_per_layer"] = round(t_df, 2)
            t["dequant_full_GBps"] = round(elems * (1 + meta_b + 2) / (t_df * 1e-6) / 1e9, 1)
        r["timed"][name] = t

    G = Hq // Hkv

    def attn(q, k, v):
        """fp32 attention of one decode query [Hq][128] over BF16 k, v [T][Hkv][128]."""
        kf = k.float().repeat_interleave(G, dim=1).permute(1, 0, 2)   # [Hq][T][128]
        vf = v.float().repeat_interleave(G, dim=1).permute(1, 0, 2)
        s = torch.einsum("hd,htd->ht", q.float(), kf) / 128 ** 0.5
        return torch.einsum("ht,htd->hd", torch.softmax(s, dim=1), vf)

    def vnmse(o_hat, o):
        return float(((o_hat - o).pow(2).sum(dim=-1) / o.pow(2).sum(dim=-1)).mean())

    acc = {}
    out = torch.empty(1, Hq, 128, dtype=torch.bfloat16, device=dev)
    outv = torch.empty(1, 1, Hq, 128, dtype=torch.bfloat16, device=dev)
    ws = lynx.workspace(L, 1, Hq, 1, T, device=dev)
    layers = range(min(4, n_layers))
    for l in layers:
        q = Q[l][0]
        o = attn(q, K[l], V[l])
        p = pools[l]
        lynx.lynx_attn_anchor_decode(L, 1, Hq, T, lens, table, p.k_anc, p.v_anc, p.meta, Q[l], out, None, ws)
        acc.setdefault("uniform_anchor", []).append(vnmse(out[0].float(), o))
        lynx.lynx_attn_verify(L, 1, Hq, 1, T, lens, table, p.k_codes, p.v_codes, p.meta,
                              Q[l].view(1, 1, Hq, 128), None, None, outv, ws)
        acc.setdefault("uniform_full", []).append(vnmse(outv[0, 0].float(), o))
        for a in alphas:
            for name, vid in variants.items():
                encode(l, a, vid, into=(hp, hm))
                modes = [("anchor", False, (hp.k_anc, hp.v_anc))]
                if vid != lynx.LYNX_HQ_INT4:
                    hp.merge()
                    modes.append(("full", True, (hp.k_codes, hp.v_codes)))
                for mode, full, (kp, vp) in modes:
                    lynx.lynx_hkv_dequant(L, 0, T, table, full, kp, vp, a, vid, hm, ko, vo)
                    key = f"{name}_alpha{a:g}" if vid == lynx.LYNX_HQ_INT4 else f"{name}_{mode}_alpha{a:g}"
                    acc.setdefault(key, []).append(vnmse(attn(q, ko, vo), o))
    torch.cuda.synchronize()
    r["vnmse"] = {k: float(f"{sum(v) / len(v):.3g}") for k, v in acc.items()}
    r["vnmse_layers"] = len(layers)
    del hp, hm, hps, hms, ko, vo
    return {"hier_codec": r}


def split_widths_stage(dev, T, Hkv, K, V, n_layers, Q=None, Hq=None):
    """The 2 + 6 and 6 + 2 splits on the workload's layers: encode of every
    layer into its own planes (so the merge below reads cold planes), merge of
    the whole cache (one call per plane kind), the anchor phase's BF16
    pages and the anchor decode straight from the A-bit planes (layers in
    turn, one query per layer), HIP events; bytes as for the 4 + 4 codec, with
    A / 8 and (8 - A) / 8 bytes per element for the two planes, and for the
    decode 32 A + 16 bytes per token and kv head (K and V anchors, V scale and
    zero, K scales and zeros over the group's 128 tokens)."""
    import torch

    from paper_2607_01831_amd import lynx

    table = torch.zeros(1, 1, dtype=torch.int32, device=dev)
    L = lynx.contiguous_layout(Hkv, 1, T)
    rows = T * Hkv
    elems = rows * 128 * 2
    ev = lambda: torch.cuda.Event(enable_timing=True)
    r = {}
    for A in (2, 6):
        R = 8 - A
        anc = torch.empty(2, n_layers, rows * 16 * A, dtype=torch.uint8, device=dev)
        res = torch.empty(2, n_layers, rows * 16 * R, dtype=torch.uint8, device=dev)
        codes = torch.empty(2, n_layers, rows * 128, dtype=torch.uint8, device=dev)
        metas = [lynx.Meta.empty(L, 1, device=dev) for _ in range(n_layers)]
        ko = torch.empty(T, Hkv, 128, dtype=torch.bfloat16, device=dev)
        vo = torch.empty_like(ko)

        def enc():
            for l in range(n_layers):
                lynx.lynx_kv_encode_split(L, A, 0, T, table, K[l], V[l], anc[0, l], anc[1, l], res[0, l],
                                          res[1, l], metas[l])

        def merge():
            for w in range(2):
                lynx.lynx_kv_merge_split(A, anc[w], res[w], codes[w])

        def deq():
            for l in range(n_layers):
                lynx.lynx_kv_dequant_anchor_split(L, A, 0, T, table, anc[0, l], anc[1, l], metas[l], ko, vo)

        lens = torch.tensor([T], dtype=torch.int32, device=dev)
        dec_out = torch.empty(1, Hq or 1, 128, dtype=torch.bfloat16, device=dev)
        ws = lynx.workspace(L, 1, Hq or 1, 1, T)

        def dec():
            for l in range(n_layers):
                lynx.lynx_attn_anchor_decode_split(A, L, 1, Hq, T, lens, table, anc[0, l], anc[1, l], metas[l],
                                                   Q[l], dec_out, None, ws)

        out = {}
        for name, fn, per_elem in (("encode", enc, 2 + 1 + 0.0625), ("merge", merge, 2.0),
                                   ("dequant_anchor", deq, A / 8 + 2 + 0.0625)):
            # median us per layer over REPS blocks of all layers
            us = summary(call_samples(fn, n=REPS, warm=2, per=n_layers))["median"]
            out[f"{name}_us_per_layer"] = round(us, 2)
            out[f"{name}_GBps"] = round(elems * per_elem / (us * 1e-6) / 1e9, 1)
        if Q is not None:
            enc()
            st = summary(call_samples(dec, n=REPS, warm=2, per=n_layers))
            out["anchor_decode_us_per_layer"] = st
            gbps = rows * (32 * A + 16) / (st["median"] * 1e-6) / 1e9
            out["anchor_decode_GBps"] = round(gbps, 1)
            out["anchor_decode_frac"] = round(gbps / HBM_PEAK_GBPS, 4)
        r[f"split_{A}_{R}"] = out
        del anc, res, codes, metas
    return {"split_widths": r}


def host_cpu():
    """The host CPU's model name and logical core count."""
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.lower().startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {"cpu": model, "nproc": os.cpu_count()}


def cpu_baseline(w, layer_inputs, n_dec=8, n_enc=4, n_ver=2):
    """The CPU oracle, untuned, timed on this host on bounded samples of the
    workload's step: its encode (single-threaded) and merge (single-threaded)
    of n_enc layers, its anchor decode of n_dec layers and its verification
    (k drafts with the causal BF16 tail) of n_ver layers, both threaded over
    the kv heads on every core this process may use.  GB/s with the GPU's
    algorithmic bytes; `value` is the anchor decode's (the metric's step)."""
    import numpy as np
    import torch

    import oracle

    def bits(t):
        return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)

    threads = oracle.default_threads()
    T, Hkv = w.context, w.Hkv
    OL = oracle.Layout(Hkv=Hkv, bt=T, max_blocks=1, max_tokens=T)
    table = np.zeros((1, 1), np.int32)
    t = {"encode": 0.0, "merge": 0.0, "decode": 0.0, "verify": 0.0}
    for l in range(max(n_dec, n_enc, n_ver)):
        k, v, q, qv, kn, vn = layer_inputs(l)
        t0 = time.perf_counter()
        planes, meta = oracle.encode_batch(OL, [T], table, [bits(k)], [bits(v)], 1)
        t1 = time.perf_counter()
        kc = oracle.merge(planes["k_anc"], planes["k_res"])
        vc = oracle.merge(planes["v_anc"], planes["v_res"])
        t2 = time.perf_counter()
        if l < n_enc:
            t["encode"] += t1 - t0
            t["merge"] += t2 - t1
        if l < n_dec:
            t0 = time.perf_counter()
            oracle.anchor_decode(OL, w.Hq, np.array([T]), table, planes["k_anc"], planes["v_anc"],
                                 meta, bits(q), nthreads=threads)
            t["decode"] += time.perf_counter() - t0
        if l < n_ver:
            t0 = time.perf_counter()
            oracle.verify(OL, w.Hq, np.array([T]), table, kc, vc, meta, bits(qv), bits(kn), bits(vn),
                          nthreads=threads)
            t["verify"] += time.perf_counter() - t0
    elems = T * Hkv * 128 * 2
    gb = lambda nbytes, secs: round(nbytes / secs / 1e9, 4)
    steps = {
        "encode": {"GBps": gb(n_enc * elems * ENC_BYTES_PER_ELEM, t["encode"]), "cores": 1,
                   "layers": n_enc, "s": round(t["encode"], 2)},
        "merge": {"GBps": gb(n_enc * elems * MERGE_BYTES_PER_ELEM, t["merge"]), "cores": 1,
                  "layers": n_enc, "s": round(t["merge"], 2)},
        "anchor_decode": {"GBps": gb(n_dec * T * Hkv * DECODE_BYTES_PER_TOKEN_HEAD, t["decode"]),
                          "cores": threads, "layers": n_dec, "s": round(t["decode"], 2)},
        "verify": {"GBps": gb(n_ver * T * Hkv * VERIFY_BYTES_PER_TOKEN_HEAD, t["verify"]),
                   "us_per_layer": round(t["verify"] * 1e6 / n_ver, 1), "cores": threads,
                   "layers": n_ver, "s": round(t["verify"], 2)},
    }
    return {"value": steps["anchor_decode"]["GBps"], "unit": "GB/s", "cores": threads,
            "kind": "oracle",
            "sample": f"fp64 oracle on the same seeded inputs, {T} tokens, all {Hkv} kv heads: "
                      f"anchor decode of {n_dec} of {w.layers} layers on {threads} threads "
                      f"({t['decode']:.2f} s); also encode and merge of {n_enc} layers (one "
                      f"thread, {t['encode'] + t['merge']:.2f} s) and verification of k={w.drafts} drafts "
                      f"of {n_ver} layers ({t['verify']:.2f} s)",
            "steps": steps, "host": host_cpu()}


# ----------------------------------------------------------------------- main --

def main():
    args = parse()
    if args.summarize_trace:
        summarize_trace(args.summarize_trace)
        return
    if args.summarize_pmc:
        summarize_pmc(*args.summarize_pmc)
        return
    if args.summarize_conditions:
        summarize_conditions(args.summarize_conditions)
        return
    if args.summarize_copies:
        summarize_copies(args.summarize_copies)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the library has no "
              "multi-GPU path; it would shard by kv head or along the context.", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2607_01831_amd import inputs, lynx

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    lynx.load()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    w = inputs.WORKLOADS[WORKLOAD]
    n_layers = args.layers or w.layers
    T, Hkv, Hq, nq = w.context, w.Hkv, w.Hq, w.drafts
    L = lynx.contiguous_layout(Hkv, 1, T)
    table = torch.zeros(1, 1, dtype=torch.int32, device=dev)
    lens = torch.tensor([T], dtype=torch.int32, device=dev)

    # ---------------- set-up (untimed) ----------------
    t_setup = time.perf_counter()
    K, V, Q, QV, KN, VN = [], [], [], [], [], []
    for l in range(n_layers):
        K.append(inputs.kv(w, "k", layer=l, device=dev))
        V.append(inputs.kv(w, "v", layer=l, device=dev))
        Q.append(inputs.queries(w, layer=l, device=dev))
        QV.append(inputs.queries(w, layer=l, step=1, nq=nq, device=dev))
        kn, vn = inputs.drafts_kv(w, layer=l, device=dev)
        KN.append(kn)
        VN.append(vn)
    # every layer's planes are slices of one allocation per plane kind: the
    # residual stream of the whole cache moves and merges in one call each
    pools, whole = lynx.KVPool.allocate_layers(L, 1, n_layers, device=dev)
    # decode-side residual buffers, filled only by the H2D transport
    recv_k = torch.empty_like(whole.k_res)
    recv_v = torch.empty_like(whole.v_res)
    # the residual stream as it leaves the prefill side: pinned host staging
    for l in range(n_layers):
        pools[l].encode(0, T, table, K[l], V[l])
    host_k = whole.k_res.cpu().pin_memory()
    host_v = whole.v_res.cpu().pin_memory()
    out = torch.empty(1, Hq, 128, dtype=torch.bfloat16, device=dev)
    outv = torch.empty(1, nq, Hq, 128, dtype=torch.bfloat16, device=dev)
    ws = lynx.workspace(L, 1, Hq, nq, T)
    torch.cuda.synchronize()
    if args.copy_calibration:
        # one plain device-to-device copy of known size, for the HBM counters
        src = torch.ones(COPY_CALIBRATION_BYTES, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    t_setup = time.perf_counter() - t_setup

    main_s = torch.cuda.current_stream()
    side = torch.cuda.Stream()
    ev = lambda: torch.cuda.Event(enable_timing=True)

    def step(rec):
        e = {k: ev() for k in ("start", "enc", "dec0", "dec", "merge0", "merge", "ver")}
        e["h2d0"], e["h2d"] = ev(), ev()
        e["start"].record(main_s)
        for l in range(n_layers):
            pools[l].encode(0, T, table, K[l], V[l])
        e["enc"].record(main_s)
        # residual transport on the side stream, after the prefill side is done
        side.wait_event(e["enc"])
        with torch.cuda.stream(side):
            e["h2d0"].record(side)
            recv_k.copy_(host_k, non_blocking=True)
            recv_v.copy_(host_v, non_blocking=True)
            e["h2d"].record(side)
        e["dec0"].record(main_s)
        for l in range(n_layers):
            p = pools[l]
            lynx.lynx_attn_anchor_decode(L, 1, Hq, T, lens, table, p.k_anc, p.v_anc, p.meta,
                                         Q[l], out, None, ws)
        e["dec"].record(main_s)
        main_s.wait_event(e["h2d"])
        e["merge0"].record(main_s)
        lynx.lynx_kv_merge(whole.k_anc, recv_k, whole.k_codes)
        lynx.lynx_kv_merge(whole.v_anc, recv_v, whole.v_codes)
        e["merge"].record(main_s)
        for l in range(n_layers):
            p = pools[l]
            lynx.lynx_attn_verify(L, 1, Hq, nq, T, lens, table, p.k_codes, p.v_codes, p.meta,
                                  QV[l], KN[l], VN[l], outv, ws)
        e["ver"].record(main_s)
        rec.append(e)

    for _ in range(args.warmup):
        step([])
    torch.cuda.synchronize()
    recs = []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step(recs)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0

    # The same decode calls once more with no residual transport running
    # (reported beside the step's figure, which overlaps the transport).
    def decode_layers():
        for l in range(n_layers):
            p = pools[l]
            lynx.lynx_attn_anchor_decode(L, 1, Hq, T, lens, table, p.k_anc, p.v_anc, p.meta,
                                         Q[l], out, None, ws)

    st_dec_alone = summary(call_samples(decode_layers, n=max(args.steps, 1), warm=1, per=n_layers))

    def encode_layers():
        for l in range(n_layers):
            pools[l].encode(0, T, table, K[l], V[l])

    def start_h2d(after):
        side.wait_event(after)
        with torch.cuda.stream(side):
            recv_k.copy_(host_k, non_blocking=True)
            recv_v.copy_(host_v, non_blocking=True)

    def decode_counted():
        decode_layers()
        return n_layers

    transport = (transport_interference(encode_layers, decode_counted, start_h2d, args.transport_trials)
                 if args.transport_trials > 0 else None)
    ceil = stream_ceilings(dev) if args.ceilings else None
    ver128 = verify_128k(args.verify_128k_calls, dev) if args.verify_128k_calls > 0 else None
    paged = paged_decode_stage(args.paged_calls, dev) if args.paged_calls > 0 else None
    ovl = overlap_70b_stage(dev) if args.overlap_70b else None
    serdes = serdes_pipeline_stage(dev, T, Hkv, K, V, n_layers, side) if args.serdes else None
    hier = hier_codec_stage(dev, T, Hkv, Hq, K, V, Q, pools, L, n_layers) if args.hier else None
    split = split_widths_stage(dev, T, Hkv, K, V, n_layers, Q, Hq) if args.split_widths else None

    # The speculative decoder's own pieces, timed alone: decode over the
    # anchors plus the 8 BF16 tokens it generated (32 layers), and greedy
    # acceptance of 8 drafts over a 128256-entry vocabulary.
    spec = {}
    if args.spec_stages:
        def decode_tail_layers():
            for l in range(n_layers):
                p = pools[l]
                lynx.lynx_attn_anchor_decode_tail(L, 1, Hq, T, lens, table, p.k_anc, p.v_anc, p.meta,
                                                  Q[l], KN[l], VN[l], out, None, ws)

        spec["anchor_decode_tail8_us_per_layer"] = summary(
            call_samples(decode_tail_layers, n=max(args.steps, 1), warm=1, per=n_layers))["median"]
        vocab = 128256
        g = torch.Generator().manual_seed(7)
        logits = torch.randn(1, nq + 1, vocab, generator=g).to(dev)
        drafts = logits[:, :nq].argmax(dim=2).to(torch.int32)
        acc = torch.empty(1, dtype=torch.int32, device=dev)
        nxt = torch.empty(1, dtype=torch.int32, device=dev)
        aws = torch.empty(max(lynx.lynx_spec_accept_workspace_bytes(1, nq, vocab), 16),
                          dtype=torch.uint8, device=dev)
        spec["accept_greedy_k8_vocab128256_us"] = summary(call_samples(
            lambda: lynx.lynx_spec_accept_greedy(logits, drafts, acc, nxt, aws)))["median"]
        spec["accept_greedy_all_kept"] = int(acc.item()) == nq
        # acceptance of sampled drafts over the same vocabulary: target and
        # draft distributions (softmax of the scores and of perturbed ones)
        probs = torch.softmax(logits, dim=2).contiguous()
        qprobs = torch.softmax(logits[:, :nq] + 0.5 * torch.randn(1, nq, vocab, generator=g).to(dev),
                               dim=2).contiguous()
        uni = torch.rand(1, nq + 1, generator=g).to(dev)
        spec["accept_sample_k8_vocab128256_us"] = summary(call_samples(
            lambda: lynx.lynx_spec_accept_sample(probs, qprobs, drafts, uni, acc, nxt, aws)))["median"]

    def ms(a, b):
        return sum(r[a].elapsed_time(r[b]) for r in recs) / len(recs)

    def per_layer(a, b):
        """median, min, max over the timed steps of one stage, us per layer"""
        return summary([r[a].elapsed_time(r[b]) * 1e3 / n_layers for r in recs])

    t_step = ms("start", "ver")
    t_enc = ms("start", "enc")
    t_dec = ms("dec0", "dec")
    t_h2d = ms("h2d0", "h2d")
    t_merge = ms("merge0", "merge")
    t_ver = ms("merge", "ver")

    elems = n_layers * T * Hkv * 128 * 2  # K and V elements
    enc_gbps = elems * ENC_BYTES_PER_ELEM / (t_enc * 1e-3) / 1e9
    merge_gbps = elems * MERGE_BYTES_PER_ELEM / (t_merge * 1e-3) / 1e9
    dec_bytes = n_layers * T * Hkv * DECODE_BYTES_PER_TOKEN_HEAD
    dec_gbps = dec_bytes / (t_dec * 1e-3) / 1e9
    ver_bytes = n_layers * T * Hkv * VERIFY_BYTES_PER_TOKEN_HEAD
    ver_gbps = ver_bytes / (t_ver * 1e-3) / 1e9
    h2d_gbps = (host_k.numel() + host_v.numel()) / (t_h2d * 1e-3) / 1e9
    ver_us = t_ver * 1e3 / n_layers
    overlap = max(0.0, min(1.0, (t_dec + t_h2d - (ms("dec0", "merge0"))) / min(t_dec, t_h2d)))

    per_call_bytes = T * Hkv * DECODE_BYTES_PER_TOKEN_HEAD
    per_call_s = t_dec * 1e-3 / n_layers
    result = {
        "metric": METRIC,
        "value": round(dec_gbps, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(t_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{WORKLOAD}: {n_layers} layers x ({Hq} q / {Hkv} kv heads, d=128), "
                               f"context {T}, batch 1, k={nq} drafts", "layers": n_layers,
                   "q_heads": Hq, "kv_heads": Hkv, "head_dim": 128, "context": T, "batch": 1,
                   "drafts": nq},
        "hbm_frac": round(dec_gbps / HBM_PEAK_GBPS, 4),
        "stages": {
            "encode_GBps": round(enc_gbps, 2), "encode_frac": round(enc_gbps / HBM_PEAK_GBPS, 4),
            "encode_us_per_layer": round(t_enc * 1e3 / n_layers, 2),
            "anchor_decode_GBps": round(dec_gbps, 2),
            "anchor_decode_us_per_layer": round(t_dec * 1e3 / n_layers, 3),
            "anchor_decode_GBps_without_transport": round(
                T * Hkv * DECODE_BYTES_PER_TOKEN_HEAD / (st_dec_alone["median"] * 1e-6) / 1e9, 2),
            "anchor_decode_us_per_layer_without_transport": st_dec_alone["median"],
            "per_layer_us": {"encode": per_layer("start", "enc"),
                             "anchor_decode": per_layer("dec0", "dec"),
                             "anchor_decode_without_transport": st_dec_alone,
                             "merge": per_layer("merge0", "merge"),
                             "verify": per_layer("merge", "ver")},
            "merge_GBps": round(merge_gbps, 2), "merge_frac": round(merge_gbps / HBM_PEAK_GBPS, 4),
            "merge_us_per_layer": round(t_merge * 1e3 / n_layers, 2),
            "verify_us_per_layer": round(ver_us, 2),
            "verify_GBps": round(ver_gbps, 2),
            "residual_h2d_GBps": round(h2d_gbps, 2),
            **(ceil or {}),
            **(ver128 or {}),
            **(paged or {}),
            **(ovl or {}),
            **(serdes or {}),
            **(hier or {}),
            **(split or {}),
            **spec,
            "decode_hidden_behind_h2d": round(overlap, 3),
            **({"anchor_decode_us_per_layer_by_condition": transport} if transport else {}),
            "wall_ms_per_step": round(wall * 1e3 / args.steps, 3),
            "setup_s": round(t_setup, 1),
        },
        "roofline": {
            "kernel": "anchor_decode_kernel: one launch per lynx_attn_anchor_decode call on a 32K layer "
                      "(the split merge runs in the same launch)",
            "bound": "hbm",
            "achieved": round(per_call_bytes / per_call_s / 1e9, 2),
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": round(per_call_bytes / per_call_s / 1e9 / HBM_PEAK_GBPS, 4),
            "traffic": stored_traffic(),
            "algorithmic_bytes_per_call": per_call_bytes,
            "us_per_call": round(per_call_s * 1e6, 3),
        },
    }
    if not args.no_cpu_baseline:
        def layer_inputs(l):
            kn, vn = inputs.drafts_kv(w, layer=l)
            return (inputs.kv(w, "k", layer=l), inputs.kv(w, "v", layer=l),
                    inputs.queries(w, layer=l), inputs.queries(w, layer=l, step=1, nq=nq), kn, vn)
        nl = min(args.cpu_layers, n_layers)
        result["cpu_baseline"] = cpu_baseline(w, layer_inputs, n_dec=nl, n_enc=max(1, nl // 2),
                                              n_ver=max(1, nl // 4))
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
