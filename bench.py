"""Benchmark of the TurboAngle KV-cache codec on one MI355X.

One step = one pass of the whole hot path over the Mistral-7B-shaped cache (32 layers, 8 KV
heads, 4096 tokens, d = 128, bf16, n = 64 angle bins, K 8-bit linear / V 4-bit log norms):
encode all of K and V into the compressed cache, then decode a whole compressed cache back to
bf16.  Inputs are seeded synthetic tensors resident in HBM before the timed region.  Two caches
and two output sets alternate between steps, so a decode never reads the cache the encode
before it has just written (the working set of a step exceeds the last-level cache, and the
cache a decode reads was written a full step earlier).

    python bench.py [--steps K] [--warmup W] [--workload C2|C3|C4|C5] [--no-cpu-baseline]
    python bench.py --summarize-profiles TRACE FETCH WRITE SQ VALU --commands ...

Prints one JSON line.  `value` is bf16 KV bytes through the codec per second, counting the
bytes encoded and the bytes decoded in a step (2 x 512 MiB at the default workload), divided
by the step time.  The roofline object is the HBM roofline of the slower direction, with the
algorithmic bytes of one launch (every bf16 element and every cache byte once); the counter
evidence it quotes (HBM bytes per launch, VALU instructions and busy fraction) comes from the
rocprofv3 summary committed under profiles/ for the same kernel sources.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import workloads  # noqa: E402

METRIC = "encode+decode GB/s of bf16 KV and % of HBM peak, d=128, 1 MI355X"
HBM_PEAK_GBPS = 8000.0
PROFILE_COUNTERS = os.path.join(ROOT, "profiles", "mistral7b_c2_encode_decode_counters.json")
# the codec counter summary of each workload that has one
CODEC_COUNTER_FILES = {"C2": "mistral7b_c2_encode_decode_counters.json",
                       "C3": "c3_early_boost_encode_decode_counters.json",
                       "C4": "d64_batch8_c4_encode_decode_counters.json"}


def codec_counters(workload_key: str):
    name = CODEC_COUNTER_FILES.get(workload_key)
    return None if name is None else os.path.join(ROOT, "profiles", name)
# fp32 VALU issue peak without packed-fp32 instructions: 256 CUs x 4 SIMDs, one wave64
# instruction per SIMD every 4 cycles, 2.4 GHz
VALU_ISSUE_PEAK = 256 * 4 * 2.4e9 / 4
# kernel sources each counter summary depends on: a summary is quoted only while they are
# unchanged
CODEC_SOURCES = ["tvq_encode.hip", "tvq_decode.hip", "tvq_codes.h", "tvq_device.h",
                 "tvq_internal.h"]
ATTENTION_SOURCES = ["tvq_attention.hip", "tvq_codes.h", "tvq_device.h", "tvq_internal.h"]
# the attention counter summary of each workload the attention step runs on
ATTENTION_COUNTER_FILES = {"C5": "longctx_c5_attention_counters.json",
                           "C4": "d64_batch8_c4_attention_counters.json"}


LONGCTX_DECODE_COUNTERS = os.path.join(ROOT, "profiles", "longctx_c5_decode_counters.json")


def attention_counters(workload_key: str):
    name = ATTENTION_COUNTER_FILES.get(workload_key)
    return None if name is None else os.path.join(ROOT, "profiles", name)
ATTN_GROUP = 4          # query heads per KV head (32 query heads over 8 KV heads)
PAGE_TOKENS = 256       # slots per block of the paged pool


# HIP event flag: no system-scope fence (cache write-back and invalidation) when the event is
# recorded.  The HIP runtime documents it for events that only time work: the default fence
# writes the GPU's caches back between the timed kernels and slows the one that follows.
HIP_EVENT_DISABLE_SYSTEM_FENCE = 0x20000000


class TimingEvent:
    """A HIP timing event created with HIP_EVENT_DISABLE_SYSTEM_FENCE, recorded on a stream;
    the interface of torch.cuda.Event that the bench uses (record, elapsed_time in ms)."""
    _hip = None

    @classmethod
    def _lib(cls):
        if cls._hip is None:
            import ctypes
            lib = ctypes.CDLL("libamdhip64.so")
            lib.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
            lib.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
            lib.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                                ctypes.c_void_p]
            lib.hipEventDestroy.argtypes = [ctypes.c_void_p]
            cls._hip = lib
        return cls._hip

    def __init__(self):
        import ctypes
        self._ev = ctypes.c_void_p()
        if self._lib().hipEventCreateWithFlags(ctypes.byref(self._ev),
                                               HIP_EVENT_DISABLE_SYSTEM_FENCE) != 0:
            raise RuntimeError("hipEventCreateWithFlags failed")

    def record(self, stream=None):
        import torch
        s = stream if stream is not None else torch.cuda.current_stream()
        if self._lib().hipEventRecord(self._ev, s.cuda_stream) != 0:
            raise RuntimeError("hipEventRecord failed")

    def elapsed_time(self, end) -> float:
        import ctypes
        ms = ctypes.c_float()
        if self._lib().hipEventElapsedTime(ctypes.byref(ms), self._ev, end._ev) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return float(ms.value)

    def __del__(self):
        if self._hip is not None and self._ev:
            self._hip.hipEventDestroy(self._ev)


def kernel_source_hash(names=None) -> str:
    h = hashlib.sha256()
    for name in names or CODEC_SOURCES:
        with open(os.path.join(ROOT, "paper_2603_27467_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def algorithmic_bytes(w: workloads.Workload) -> dict:
    """Bytes a launch must move: every bf16 input element once and every cache byte once
    (angle codes, norm codes, 8-byte headers), per direction."""
    P = w.d // 2
    elem_bytes = 2 if w.dtype == "bf16" else 4
    kv = 2 * w.L * w.B * w.H * w.T * w.d * elem_bytes
    comp = 0
    for t in w.table:
        for n, mode, bits in ((t.n_k, t.norm_mode_k, t.norm_bits_k),
                              (t.n_v, t.norm_mode_v, t.norm_bits_v)):
            wbits = int(np.ceil(np.log2(n)))
            rec = P * wbits // 8 + (4 * P if mode == 0 else P * bits // 8 + 8)
            comp += rec * w.B * w.H * w.T
    return {"kv": kv, "compressed": comp, "per_launch": kv + comp,
            "vectors": 2 * w.L * w.B * w.H * w.T}


def profile_entry(kernel: str, workload: str, path: str = PROFILE_COUNTERS, sources=None):
    """The committed counter summary of `kernel` ("tvq_encode" / "tvq_decode" in the codec
    summary, "tvq_attention" in the long-context one): HBM bytes per launch from rocprofv3
    FETCH_SIZE / WRITE_SIZE scaled by the same counters on a copy of known size, VALU
    instructions per launch and VALU busy.  None when absent, when the counters were taken on
    another workload, or when the kernel sources have changed since they were taken."""
    try:
        with open(path) as f:
            d = json.load(f)
    except (OSError, ValueError):
        return None
    if d.get("kernel_source_hash") != kernel_source_hash(sources) or d.get("workload") != workload:
        return None
    return d.get("kernels", {}).get(kernel)


def cpu_baseline(w: workloads.Workload, budget_s: float = 15.0) -> dict:
    """The oracle (plain C, untuned) on a bounded sample of the same workload: chunks of
    consecutive tokens of every (batch, head) row, K and V, layer by layer, encoded and decoded
    (fixed-order fp32 decode + bf16 rounding), sharded over all host cores by a thread pool
    (ctypes releases the GIL).  Inputs are drawn before the timed region."""
    import oracle
    from concurrent.futures import ThreadPoolExecutor

    cores = os.cpu_count() or 1
    signs = workloads.sign_table(w.sign_seed, w.L, w.d)
    chunk = 64

    def prepare_layer(l: int, spans):
        """Draw layer l once up to the last token needed and cut it into the chunks."""
        t = w.table[l]
        kinds = [oracle.Kind(t.n_k, t.norm_mode_k, t.norm_bits_k),
                 oracle.Kind(t.n_v, t.norm_mode_v, t.norm_bits_v)]
        c = oracle.Codec(1, w.H, w.d, kinds, signs[l:l + 1])
        top = max(t1 for _, t1 in spans)
        k = workloads.generate(w, "K", layers=range(l, l + 1), tokens=range(0, top))
        v = workloads.generate(w, "V", layers=range(l, l + 1), tokens=range(0, top))
        out = []
        for t0, t1 in spans:
            total, _ = c.layout(w.B, t1 - t0)
            out.append((c, np.ascontiguousarray(k[:, :, :, t0:t1]),
                        np.ascontiguousarray(v[:, :, :, t0:t1]), np.zeros(total, np.uint8),
                        t1 - t0))
        return out

    def run(job):
        c, k, v, cache, T = job
        c.encode_cache(k, v, 0, T, cache, want_coords=False)
        out = c.decode_cache(cache, w.B, T, 0, T, "f32")
        oracle.f32_to_bf16(out)
        return 2 * w.B * w.H * T

    # a sample of whole 64-token chunks (every layer, K and V), passed over repeatedly until
    # about `budget_s` of wall time has been spent
    oracle.lib()
    n_jobs = 64 * cores
    tasks = []
    l, t0 = 0, 0
    while len(tasks) < n_jobs:
        tasks.append((l, t0, min(t0 + chunk, w.T)))
        l += 1
        if l >= w.L:
            l, t0 = 0, (t0 + chunk) % w.T
    by_layer = {}
    for l_, t0_, t1_ in tasks:
        by_layer.setdefault(l_, []).append((t0_, t1_))
    with ThreadPoolExecutor(max_workers=cores) as ex:
        jobs = [j for part in ex.map(lambda kv: prepare_layer(*kv), by_layer.items()) for j in part]
    vecs, passes = 0, 0
    s = time.perf_counter()
    with ThreadPoolExecutor(max_workers=cores) as ex:
        while time.perf_counter() - s < budget_s:
            vecs += sum(ex.map(run, jobs))
            passes += 1
    wall = time.perf_counter() - s
    # the same jobs on one thread, for about a fifth of the budget
    vecs1 = 0
    s1 = time.perf_counter()
    for job in jobs:
        vecs1 += run(job)
        if time.perf_counter() - s1 > budget_s / 5:
            break
    wall1 = time.perf_counter() - s1
    elem_bytes = 2 if w.dtype == "bf16" else 4
    kv_bytes = vecs * w.d * elem_bytes
    return {"value": round(2 * kv_bytes / wall / 1e9, 4), "unit": "GB/s", "cores": cores,
            "value_1core": round(2 * vecs1 * w.d * elem_bytes / wall1 / 1e9, 4),
            "kind": "oracle",
            "sample": f"{len(tasks)} chunks of {chunk} tokens x {w.B * w.H} (batch, head) rows "
                      f"x (K, V) spread over all {w.L} layers, {vecs // passes} vectors, encoded "
                      f"and decoded {passes} times: {vecs} vectors in {wall:.1f} s on {cores} "
                      f"threads; value_1core: {vecs1} vectors of the same jobs in {wall1:.1f} s "
                      f"on one thread; same unit as value (bf16 KV bytes encoded + decoded per "
                      f"second)"}


def cpu_baseline_attention(w: workloads.Workload, budget_s: float = 15.0,
                           tokens: int = 2048) -> dict:
    """The oracle's attention (plain C, fp64, untuned) on a bounded sample of the same cache:
    single (sequence, KV head) rows of `tokens` cached tokens, layers taken in turn, each
    encoded by the oracle beforehand (not timed), then attention of ATTN_GROUP query heads over
    the row, sharded over all host cores by a thread pool (ctypes releases the GIL).  The unit
    is the attention line's: bf16-equivalent K and V bytes consumed per second."""
    import oracle
    from concurrent.futures import ThreadPoolExecutor

    cores = os.cpu_count() or 1
    signs = workloads.sign_table(w.sign_seed, w.L, w.d)
    T = min(tokens, w.T)
    scale = 1.0 / float(np.sqrt(w.d))
    rng = np.random.default_rng(w.data_seed + 11)

    def prepare(l: int):
        t = w.table[l]
        kinds = [oracle.Kind(t.n_k, t.norm_mode_k, t.norm_bits_k),
                 oracle.Kind(t.n_v, t.norm_mode_v, t.norm_bits_v)]
        c = oracle.Codec(1, 1, w.d, kinds, signs[l:l + 1])
        k = workloads.generate(w, "K", layers=range(l, l + 1), tokens=range(0, T))
        v = workloads.generate(w, "V", layers=range(l, l + 1), tokens=range(0, T))
        total, _ = c.layout(1, T)
        cache = np.zeros(total, np.uint8)
        b, h = l % w.B, (l // w.B) % w.H
        c.encode_cache(np.ascontiguousarray(k[:, b:b + 1, h:h + 1]),
                       np.ascontiguousarray(v[:, b:b + 1, h:h + 1]), 0, T, cache,
                       want_coords=False)
        q = rng.standard_normal((1, ATTN_GROUP, w.d))
        return c, cache, q

    def run(job):
        c, cache, q = job
        c.attention_decode(cache, 1, T, 0, T, q, scale)
        return T

    oracle.lib()
    layers = [l % w.L for l in range(max(cores, 8))]
    with ThreadPoolExecutor(max_workers=cores) as ex:
        jobs = list(ex.map(prepare, layers))
    toks, passes = 0, 0
    s = time.perf_counter()
    with ThreadPoolExecutor(max_workers=cores) as ex:
        while time.perf_counter() - s < budget_s:
            toks += sum(ex.map(run, jobs))
            passes += 1
    wall = time.perf_counter() - s
    toks1 = 0
    s1 = time.perf_counter()
    while time.perf_counter() - s1 < budget_s / 5:
        for job in jobs:
            toks1 += run(job)
    wall1 = time.perf_counter() - s1
    per_tok = 2 * w.d * 2                     # bf16 K and V of one token of one KV head
    return {"value": round(toks * per_tok / wall / 1e9, 4), "unit": "GB/s", "cores": cores,
            "value_1core": round(toks1 * per_tok / wall1 / 1e9, 4), "kind": "oracle",
            "sample": f"{len(jobs)} (sequence, KV head) rows of {T} cached tokens, one layer "
                      f"each (layers in turn), {ATTN_GROUP} query heads, fp64 attention over "
                      f"the codes, {passes} passes: {toks} tokens in {wall:.1f} s on {cores} "
                      f"threads; value_1core: {toks1} tokens in {wall1:.1f} s on one thread; "
                      f"same unit as value (bf16-equivalent K and V bytes consumed per second)"}


def _csv(path):
    import csv
    with open(path) as f:
        return list(csv.DictReader(f))


def _short(name: str) -> str:
    """Map a rocprofv3 kernel name to the entry point it belongs to."""
    if "encode_" in name and "tvq" in name:
        return "tvq_encode"
    if "decode_" in name and "tvq" in name:
        return "tvq_decode"
    if "attn_" in name and "chunk_kernel" in name and "tvq" in name:
        return "tvq_attention_chunk"
    if "attn_merge" in name and "tvq" in name:
        return "tvq_attention_merge"
    if "copyBuffer" in name:
        return "copy"
    return name


def _kernel_label(name: str) -> str:
    """"void tvq::(anonymous namespace)::encode_fast_kernel<128, true>(tvq::EncodeArgs)" ->
    "encode_fast_kernel<128, true>"."""
    name = name.split("(tvq::")[0]
    return name.split("::")[-1]


def _find(dirpath: str, suffix: str) -> str:
    for root, _, files in os.walk(dirpath):
        for f in files:
            if f.endswith(suffix):
                return os.path.join(root, f)
    raise FileNotFoundError(f"no *{suffix} under {dirpath}")


# dispatches of each codec kernel in the kernel-trace run that are timed steps (the last 20 of
# `bench.py --steps 20 --warmup 3`: before them the encode fills two caches and both directions
# run the warm-up steps)
TRACE_TIMED_DISPATCHES = 20


def shader_engines(trace_dir):
    """(shader engines, XCDs) of the GPU agent (rocprofv3 agent_info.csv, the agent with
    compute units)."""
    try:
        rows = _csv(_find(trace_dir, "agent_info.csv"))
    except (OSError, FileNotFoundError, StopIteration):
        return 32, 8
    gpu = max(rows, key=lambda r: int(r.get("Cu_Count") or 0))
    return int(gpu.get("Array_Count") or 32) or 32, int(gpu.get("Num_Xcc") or 8) or 8


def dispatch_timeline(trace_dir) -> dict:
    """Per codec entry point, the durations (ns) of its dispatches in issue order
    (kernel_trace.csv)."""
    rows = _csv(_find(trace_dir, "kernel_trace.csv"))
    rows.sort(key=lambda r: int(r["Dispatch_Id"]))
    out = {}
    for r in rows:
        k = _short(r["Kernel_Name"])
        if k in ("tvq_encode", "tvq_decode", "tvq_attention"):
            out.setdefault(k, []).append(float(r["End_Timestamp"]) - float(r["Start_Timestamp"]))
    return out


def clock_fields(d: dict, topo, durations, timed: int) -> dict:
    """The shader clock of an entry point's kernel.  GRBM_GUI_ACTIVE counts the cycles the
    graphics engine is active, summed over the XCDs: per XCD over the duration of a counted
    dispatch (which runs alone in the counter run) it is the clock of that dispatch.  Over the
    mean of the timed dispatches of the kernel-trace run, where launches follow each other, the
    same cycle count gives the clock those launches sustained (the cycles of an issue-bound
    launch do not depend on the clock).  SQ_BUSY_CYCLES per shader engine (the cycles the
    shader arrays are busy, ~90% of the active ones) gives the same ratio and is recorded
    beside it."""
    n_se, n_xcc = topo
    sq = float(np.median(d["SQ_BUSY_CYCLES"])) / n_se
    pmc_ns = float(np.median(d["pmc_ns"]))
    grbm = float(np.median(d["GRBM_GUI_ACTIVE"])) / n_xcc if d.get("GRBM_GUI_ACTIVE") else float("nan")
    tl = list(durations)[-timed:] if durations else []
    t_avg = float(np.mean(tl)) if tl else float("nan")
    return {"grbm_active_cycles_per_xcd": int(round(grbm)) if grbm == grbm else None,
            "sq_busy_cycles_per_se": int(round(sq)), "pmc_dispatch_ns": pmc_ns,
            "clock_ghz_pmc": round(grbm / pmc_ns, 3), "clock_ghz_pmc_sq_busy": round(sq / pmc_ns, 3),
            "trace_timed_avg_ns": round(t_avg, 1), "trace_timed_dispatches": len(tl),
            "clock_ghz_sustained": round(grbm / t_avg, 3) if tl and grbm == grbm else None,
            "clock_ghz_sustained_sq_busy": round(sq / t_avg, 3) if tl else None,
            "dispatch_ns": [round(x) for x in durations]}


def summarize_profiles(trace_dir, fetch_dir, write_dir, sq_dir, valu_dir, commands,
                       workload_key: str = "C2") -> int:
    """Turn the rocprofv3 output of the profiling runs (kernel trace, FETCH_SIZE, WRITE_SIZE,
    SQ instruction counts, VALU busy) of the codec step on `workload_key` into the counter
    summary bench.py reads and a readable table, both under profiles/.  FETCH_SIZE and
    WRITE_SIZE (KiB per dispatch) are scaled by what they read for the 1 GiB device copy the
    profiled runs include (--copy-calibration)."""
    path = codec_counters(workload_key)
    if path is None:
        print(f"no codec counter summary is kept for {workload_key}", file=sys.stderr)
        return 2
    w = workloads.get(workload_key)
    ab = algorithmic_bytes(w)
    per = {}

    def add(kind, rows, counter):
        for r in rows:
            if r["Counter_Name"] != counter:
                continue
            k = _short(r["Kernel_Name"])
            per.setdefault(k, {}).setdefault(kind, []).append(float(r["Counter_Value"]))

    add("fetch_kib", _csv(_find(fetch_dir, "counter_collection.csv")), "FETCH_SIZE")
    add("write_kib", _csv(_find(write_dir, "counter_collection.csv")), "WRITE_SIZE")
    sq = _csv(_find(sq_dir, "counter_collection.csv"))
    for c in ("SQ_INSTS_VALU", "SQ_INSTS_SALU", "SQ_INSTS_LDS", "SQ_INSTS_VMEM_RD",
              "SQ_INSTS_VMEM_WR", "SQ_WAVES", "SQ_BUSY_CYCLES", "GRBM_GUI_ACTIVE"):
        add(c, sq, c)
    # the duration of each counted dispatch, for the clocks below
    for r in sq:
        if r["Counter_Name"] == "SQ_BUSY_CYCLES":
            per.setdefault(_short(r["Kernel_Name"]), {}).setdefault("pmc_ns", []).append(
                float(r["End_Timestamp"]) - float(r["Start_Timestamp"]))
    topo = shader_engines(trace_dir)
    timeline = dispatch_timeline(trace_dir)
    add("VALUBusy", _csv(_find(valu_dir, "counter_collection.csv")), "VALUBusy")
    stats = {}
    for r in _csv(_find(trace_dir, "kernel_stats.csv")):
        k = _short(r["Name"])
        if k in ("tvq_encode", "tvq_decode"):
            stats.setdefault(k, []).append(r)
    # the calibration copy is the largest copy dispatch (the others stage a few bytes)
    copy_bytes = float(1 << 30)
    fetch_scale = copy_bytes / 1024.0 / max(per["copy"]["fetch_kib"])
    write_scale = copy_bytes / 1024.0 / max(per["copy"]["write_kib"])
    out = {"kernel_source_hash": kernel_source_hash(), "workload": w.name,
           "algorithmic_bytes_per_launch": ab["per_launch"],
           "fetch_scale_from_copy": round(fetch_scale, 4),
           "write_scale_from_copy": round(write_scale, 4),
           "copy_bytes": int(copy_bytes), "commands": commands, "kernels": {}}
    lines = [f"# Counter summary: {w.name} (L={w.L}, B={w.B}, H={w.H}, T={w.T}, d={w.d}, bf16)",
             "", "Commands (run from /tmp, repository root $R):", ""]
    lines += [f"    {c}" for c in commands]
    lines += ["", f"FETCH_SIZE scale from the 1 GiB copy: {fetch_scale:.4f}; WRITE_SIZE scale: "
              f"{write_scale:.4f}", "",
              "| entry point | kernels (calls, avg ns, min ns) | HBM bytes/launch (counters) | "
              "algorithmic bytes/launch | VALU instr/launch | VALU instr/tile | VALUBusy % |",
              "|---|---|---|---|---|---|---|"]
    for k in ("tvq_encode", "tvq_decode"):
        d = per.get(k, {})
        # one launch of the entry point = one dispatch per kernel it starts; the profiled runs
        # start one kernel per call at this workload
        fetch = float(np.median(d["fetch_kib"])) * 1024.0 * fetch_scale
        write = float(np.median(d["write_kib"])) * 1024.0 * write_scale
        valu = float(np.median(d["SQ_INSTS_VALU"]))
        tiles = ab["vectors"] / (64 // (w.d // 32))
        ent = {"hbm_bytes_per_launch": int(round(fetch + write)),
               "fetch_bytes_per_launch": int(round(fetch)),
               "write_bytes_per_launch": int(round(write)),
               "valu_insts_per_launch": int(valu),
               "valu_insts_per_tile": round(valu / tiles, 1),
               "salu_insts_per_launch": int(np.median(d["SQ_INSTS_SALU"])),
               "lds_insts_per_launch": int(np.median(d["SQ_INSTS_LDS"])),
               "vmem_rd_insts_per_launch": int(np.median(d["SQ_INSTS_VMEM_RD"])),
               "vmem_wr_insts_per_launch": int(np.median(d["SQ_INSTS_VMEM_WR"])),
               "waves_per_launch": int(np.median(d["SQ_WAVES"])),
               "valu_busy_pct": round(float(np.median(d["VALUBusy"])), 2),
               **clock_fields(d, topo, timeline.get(k, []), TRACE_TIMED_DISPATCHES),
               "trace": [{"kernel": r["Name"], "calls": int(r["Calls"]),
                          "avg_ns": float(r["AverageNs"]), "min_ns": float(r["MinNs"]),
                          "max_ns": float(r["MaxNs"])} for r in stats.get(k, [])]}
        out["kernels"][k] = ent
        ks = "; ".join(f"{_kernel_label(t['kernel'])} ({t['calls']}, {t['avg_ns']:.0f}, "
                       f"{t['min_ns']:.0f})" for t in ent["trace"])
        lines.append(f"| {k} | {ks} | {ent['hbm_bytes_per_launch']} | {ab['per_launch']} | "
                     f"{ent['valu_insts_per_launch']} | {ent['valu_insts_per_tile']} | "
                     f"{ent['valu_busy_pct']} |")
    lines += ["", f"Clock and trace figures ({topo[1]} XCDs, {topo[0]} shader engines; "
              "GRBM_GUI_ACTIVE and SQ_BUSY_CYCLES from the counter run, whose dispatches run one "
              f"at a time; the trace mean over the last {TRACE_TIMED_DISPATCHES} dispatches of "
              "the kernel-trace run, the timed steps):", "",
              "| entry point | active cycles per XCD (busy per shader engine) | counted dispatch "
              "(us) | clock of the counted dispatch (GHz) | trace mean of the timed dispatches "
              "(us) | sustained clock = active cycles / trace mean (GHz) | fraction of the "
              "roofline at the trace mean |", "|---|---|---|---|---|---|---|"]
    for k in ("tvq_encode", "tvq_decode"):
        e = out["kernels"][k]
        lines.append(f"| {k} | {e['grbm_active_cycles_per_xcd']} ({e['sq_busy_cycles_per_se']}) | "
                     f"{e['pmc_dispatch_ns'] / 1e3:.1f} | {e['clock_ghz_pmc']} | "
                     f"{e['trace_timed_avg_ns'] / 1e3:.1f} | {e['clock_ghz_sustained']} | "
                     f"{ab['per_launch'] / (e['trace_timed_avg_ns'] * 1e-9) / 1e9 / HBM_PEAK_GBPS:.4f} |")
    lines += ["", "Dispatch durations of the kernel-trace run in issue order (us):", ""]
    for k in ("tvq_encode", "tvq_decode"):
        lines.append(f"    {k}: " + ", ".join(f"{x / 1e3:.1f}" for x in timeline.get(k, [])))
    lines += ["", "rocprofv3 --kernel-trace --stats summary of the first command "
              "(kernel_stats.csv):", "", "```"]
    with open(_find(trace_dir, "kernel_stats.csv")) as f:
        lines += [ln.rstrip("\n") for ln in f]
    lines += ["```"]
    os.makedirs(os.path.join(ROOT, "profiles"), exist_ok=True)
    with open(path, "w") as f:
        json.dump(out, f, indent=1)
    with open(path.replace("_counters.json", "_counters.md"), "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))
    return 0


def copy_calibration() -> None:
    """A plain 1 GiB device copy: what FETCH_SIZE and WRITE_SIZE read for it scales them."""
    import torch
    src = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst


def copy_peak(nbytes: int = 1 << 30, reps: int = 10) -> dict:
    """The achievable streaming rate on this GPU: a plain elementwise read + write pass
    (torch.add of 0 from one fp32 buffer of `nbytes` into another; it streams faster than the
    runtime's device-to-device blit), timed with events over `reps` runs after a warm-up run.
    Bytes moved per run = 2 * nbytes."""
    import torch
    src = torch.zeros(nbytes // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    torch.add(src, 0.0, out=dst)
    ev = [TimingEvent() for _ in range(reps + 1)]
    torch.cuda.synchronize()
    ev[0].record()
    for i in range(reps):
        torch.add(src, 0.0, out=dst)
        ev[i + 1].record()
    torch.cuda.synchronize()
    ms = np.array([ev[i].elapsed_time(ev[i + 1]) for i in range(reps)])
    del src, dst
    return {"kernel": "elementwise fp32 read + write (torch.add of 0)",
            "bytes_per_run": 2 * nbytes,
            "GBps_mean": round(2 * nbytes / (float(ms.mean()) * 1e-3) / 1e9, 1),
            "GBps_max": round(2 * nbytes / (float(ms.min()) * 1e-3) / 1e9, 1)}


def longctx_bytes(w: workloads.Workload):
    """(compressed bytes of one token position over all layers, kinds, sequences and KV heads;
    bf16 K + V bytes of one token position; bf16 query + output bytes of one attention step)."""
    P = w.d // 2
    rec_tok = 0
    for t in w.table:
        for n, mode, bits in ((t.n_k, t.norm_mode_k, t.norm_bits_k),
                              (t.n_v, t.norm_mode_v, t.norm_bits_v)):
            wbits = int(np.ceil(np.log2(n)))
            rec_tok += (P * wbits // 8 + (4 * P if mode == 0 else P * bits // 8 + 8)) * w.B * w.H
    kv_tok = 2 * w.L * w.B * w.H * w.d * 2
    qo = 2 * w.L * w.B * w.H * ATTN_GROUP * w.d * 2
    return rec_tok, kv_tok, qo


def summarize_longctx_decode(fetch_dir, write_dir, commands, steps_total: int) -> int:
    """HBM bytes of the long-context decode (C5: the whole cache decoded every step) from a
    FETCH_SIZE run and a WRITE_SIZE run of `commands` (`steps_total` = warmup + timed steps,
    with --copy-calibration): every decode dispatch's KiB scaled by what the counter reads for
    the 1 GiB copy, summed, per step; beside the algorithmic bytes of the same steps."""
    w = workloads.get("C5")
    rec_tok, kv_tok, _ = longctx_bytes(w)
    t_mean = w.T + (steps_total + 1) / 2            # tokens decoded per step, mean
    rows = {}
    for kind, d, counter in (("fetch_kib", fetch_dir, "FETCH_SIZE"),
                             ("write_kib", write_dir, "WRITE_SIZE")):
        for r in _csv(_find(d, "counter_collection.csv")):
            if r["Counter_Name"] != counter:
                continue
            k = _short(r["Kernel_Name"])
            if k == "tvq_decode":
                k = _kernel_label(r["Kernel_Name"])
            elif k != "copy":
                continue
            rows.setdefault(k, {}).setdefault(kind, []).append(float(r["Counter_Value"]))
    copy_bytes = float(1 << 30)
    fetch_scale = copy_bytes / 1024.0 / max(rows["copy"]["fetch_kib"])
    write_scale = copy_bytes / 1024.0 / max(rows["copy"]["write_kib"])
    kernels, total = {}, 0.0
    for k, d in rows.items():
        if k == "copy":
            continue
        fetch = np.array(d["fetch_kib"]) * 1024.0 * fetch_scale
        write = np.array(d["write_kib"]) * 1024.0 * write_scale
        total += float(fetch.sum() + write.sum())
        kernels[k] = {"dispatches": len(fetch), "fetch_bytes_median": int(np.median(fetch)),
                      "write_bytes_median": int(np.median(write))}
    alg = (rec_tok + kv_tok) * t_mean
    out = {"kernel_source_hash": kernel_source_hash(), "workload": w.name,
           "steps_total": steps_total, "tokens_decoded_per_step_mean": t_mean,
           "hbm_bytes_per_step": int(round(total / steps_total)),
           "algorithmic_bytes_per_step": int(round(alg)),
           "fetch_scale_from_copy": round(fetch_scale, 4),
           "write_scale_from_copy": round(write_scale, 4), "kernels": kernels,
           "commands": commands}
    lines = [f"# Long-context decode traffic: {w.name} (L={w.L}, B={w.B}, H={w.H}, "
             f"T={w.T} cached + 1 per step, d={w.d})", "",
             "Commands (run from /tmp, repository root $R):", ""]
    lines += [f"    {c}" for c in commands]
    lines += ["", f"FETCH_SIZE scale from the 1 GiB copy: {fetch_scale:.4f}; WRITE_SIZE scale: "
              f"{write_scale:.4f}", "",
              "| decode kernel | dispatches | median fetch bytes | median write bytes |",
              "|---|---|---|---|"]
    for k, e in kernels.items():
        lines.append(f"| {k} | {e['dispatches']} | {e['fetch_bytes_median']} | "
                     f"{e['write_bytes_median']} |")
    lines += ["", f"Per step ({steps_total} steps, {t_mean:.1f} tokens decoded per step on "
              f"average): HBM {out['hbm_bytes_per_step']} bytes by the counters, "
              f"{out['algorithmic_bytes_per_step']} algorithmic, ratio "
              f"{out['hbm_bytes_per_step'] / out['algorithmic_bytes_per_step']:.4f}."]
    with open(LONGCTX_DECODE_COUNTERS, "w") as f:
        json.dump(out, f, indent=1)
    with open(LONGCTX_DECODE_COUNTERS.replace(".json", ".md"), "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))
    return 0


def summarize_attention_profiles(trace_dir, fetch_dir, write_dir, sq_dir, valu_dir, commands,
                                 steps_total: int, workload_key: str = "C5") -> int:
    """Counter summary of the attention step over the cache of `workload_key` (the runs of
    `commands`, each with `steps_total` = warmup + timed steps): per chunk-kernel instantiation
    and for the merge kernel, HBM bytes per dispatch (FETCH_SIZE / WRITE_SIZE scaled by the
    1 GiB copy), VALU and LDS instructions, bank-conflict cycles and VALU busy; and the HBM
    bytes of one step."""
    w = workloads.get(workload_key)
    counters_path = attention_counters(workload_key)
    rec_tok, _, qo = longctx_bytes(w)
    t_mean = w.T + (steps_total + 1) / 2            # tokens attended per step, mean
    per = {}

    def add(kind, rows, counter):
        for r in rows:
            if r["Counter_Name"] != counter:
                continue
            k = _short(r["Kernel_Name"])
            if k.startswith("tvq_attention"):
                k = _kernel_label(r["Kernel_Name"])
            per.setdefault(k, {}).setdefault(kind, []).append(float(r["Counter_Value"]))

    add("fetch_kib", _csv(_find(fetch_dir, "counter_collection.csv")), "FETCH_SIZE")
    add("write_kib", _csv(_find(write_dir, "counter_collection.csv")), "WRITE_SIZE")
    sq = _csv(_find(sq_dir, "counter_collection.csv"))
    for c in ("SQ_INSTS_VALU", "SQ_INSTS_LDS", "SQ_LDS_BANK_CONFLICT", "SQ_WAVES", "SQ_INSTS_MFMA",
              "SQ_VALU_MFMA_BUSY_CYCLES", "GRBM_GUI_ACTIVE"):
        add(c, sq, c)
    n_se, n_xcc = shader_engines(trace_dir)
    try:
        agent = max(_csv(_find(trace_dir, "agent_info.csv")), key=lambda r: int(r.get("Cu_Count") or 0))
        n_simd = int(agent.get("Simd_Count") or 1024)
    except (OSError, FileNotFoundError, StopIteration):
        n_simd = 1024
    add("VALUBusy", _csv(_find(valu_dir, "counter_collection.csv")), "VALUBusy")
    fetch_scale = float(1 << 30) / 1024.0 / max(per["copy"]["fetch_kib"])
    write_scale = float(1 << 30) / 1024.0 / max(per["copy"]["write_kib"])
    trace = {}
    for r in _csv(_find(trace_dir, "kernel_stats.csv")):
        if _short(r["Name"]).startswith("tvq_attention"):
            trace[_kernel_label(r["Name"])] = {"calls": int(r["Calls"]),
                                              "avg_ns": float(r["AverageNs"]),
                                              "min_ns": float(r["MinNs"]),
                                              "max_ns": float(r["MaxNs"])}
    kernels, hbm_step, valu_step, conf_step, busy = {}, 0.0, 0.0, 0.0, []
    for k, d in sorted(per.items()):
        if "attn_" not in k:
            continue
        per_step = len(d["fetch_kib"]) / steps_total
        fetch = float(np.median(d["fetch_kib"])) * 1024.0 * fetch_scale
        write = float(np.median(d["write_kib"])) * 1024.0 * write_scale
        kernels[k] = {"dispatches_per_step": per_step,
                      "fetch_bytes_per_dispatch": int(round(fetch)),
                      "write_bytes_per_dispatch": int(round(write)),
                      "valu_insts_per_dispatch": int(np.median(d["SQ_INSTS_VALU"])),
                      "lds_insts_per_dispatch": int(np.median(d["SQ_INSTS_LDS"])),
                      "lds_bank_conflict_cycles_per_dispatch":
                          int(np.median(d["SQ_LDS_BANK_CONFLICT"])),
                      "waves_per_dispatch": int(np.median(d["SQ_WAVES"])),
                      "valu_busy_pct": round(float(np.median(d["VALUBusy"])), 2)}
        if d.get("SQ_INSTS_MFMA") and d.get("GRBM_GUI_ACTIVE"):
            # matrix-core busy cycles per SIMD over the dispatch's active cycles per XCD: the
            # share of the SIMDs' time the matrix instructions hold
            active = float(np.median(d["GRBM_GUI_ACTIVE"])) / n_xcc
            mf_busy = float(np.median(d["SQ_VALU_MFMA_BUSY_CYCLES"])) / n_simd
            kernels[k].update({"mfma_insts_per_dispatch": int(np.median(d["SQ_INSTS_MFMA"])),
                               "active_cycles_per_xcd": int(round(active)),
                               "mfma_busy_cycles_per_simd": int(round(mf_busy)),
                               "mfma_busy_pct": round(100.0 * mf_busy / active, 2) if active else None})
        hbm_step += per_step * (fetch + write)
        if "chunk" in k:
            valu_step += per_step * float(np.median(d["SQ_INSTS_VALU"]))
            conf_step += per_step * float(np.median(d["SQ_LDS_BANK_CONFLICT"]))
            busy += [float(np.median(d["VALUBusy"]))] * int(round(per_step))
    tiles_step = w.L * w.B * w.H * t_mean / (64 // (w.d // 32))
    ent = {"hbm_bytes_per_step": int(round(hbm_step)),
           "algorithmic_bytes_per_step": int(round(rec_tok * t_mean + qo)),
           "valu_insts_per_tile": round(valu_step / tiles_step, 1),
           "lds_bank_conflict_cycles_per_tile": round(conf_step / tiles_step, 1),
           "valu_busy_pct": round(float(np.mean(busy)), 2),
           "per_kernel": kernels, "trace": trace}
    out = {"kernel_source_hash": kernel_source_hash(ATTENTION_SOURCES), "workload": w.name,
           "query_heads_per_kv_head": ATTN_GROUP, "tokens_attended_mean": t_mean,
           "fetch_scale_from_copy": round(fetch_scale, 4),
           "write_scale_from_copy": round(write_scale, 4), "commands": commands,
           "kernels": {"tvq_attention": ent}}
    lines = [f"# Counter summary: attention over the compressed cache, {w.name} (L={w.L}, "
             f"B={w.B}, KV heads={w.H}, query heads={w.H * ATTN_GROUP}, T={w.T}, d={w.d})",
             "", "Commands (run from /tmp, repository root $R):", ""]
    lines += [f"    {c}" for c in commands]
    lines += ["", f"FETCH_SIZE scale from the 1 GiB copy: {fetch_scale:.4f}; WRITE_SIZE scale: "
              f"{write_scale:.4f}; tokens attended per step (mean): {t_mean}", "",
              f"Per step ({w.L} layer calls): HBM {ent['hbm_bytes_per_step']} B by counters vs "
              f"{ent['algorithmic_bytes_per_step']} B algorithmic; VALU {ent['valu_insts_per_tile']}"
              f" instructions per tile of {64 // (w.d // 32)} tokens; LDS bank-conflict cycles "
              f"per tile "
              f"{ent['lds_bank_conflict_cycles_per_tile']}; VALUBusy {ent['valu_busy_pct']} %", "",
              "| kernel | dispatches/step | avg ns (trace) | fetch B/dispatch | write B/dispatch | "
              "VALU/dispatch (incl. MFMA) | MFMA/dispatch | LDS/dispatch | bank-conflict cycles | "
              "VALUBusy % | MFMA busy % of active cycles |",
              "|---|---|---|---|---|---|---|---|---|---|---|"]
    for k, e in kernels.items():
        tr = trace.get(k, {})
        lines.append(f"| {k} | {e['dispatches_per_step']:.0f} | {tr.get('avg_ns', 0):.0f} | "
                     f"{e['fetch_bytes_per_dispatch']} | {e['write_bytes_per_dispatch']} | "
                     f"{e['valu_insts_per_dispatch']} | {e.get('mfma_insts_per_dispatch', '-')} | "
                     f"{e['lds_insts_per_dispatch']} | "
                     f"{e['lds_bank_conflict_cycles_per_dispatch']} | {e['valu_busy_pct']} | "
                     f"{e.get('mfma_busy_pct', '-')} |")
    lines += ["", "rocprofv3 --kernel-trace --stats summary of the first command "
              "(kernel_stats.csv, codec and attention kernels):", "", "```"]
    with open(_find(trace_dir, "kernel_stats.csv")) as f:
        rows = [ln.rstrip("\n") for ln in f]
    lines += [rows[0]] + [r for r in rows[1:] if "tvq::" in r]
    lines += ["```"]
    with open(counters_path, "w") as f:
        json.dump(out, f, indent=1)
    with open(counters_path.replace("_counters.json", "_counters.md"), "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))
    return 0


def run_longctx(w: workloads.Workload, args) -> dict:
    """Long-context step: the cache already holds T tokens of B sequences (every layer, K and
    V); one step encodes one new token per sequence and layer into slot T + i and decodes
    slots [0, T + i + 1) of the whole cache back to bf16.  Inputs are drawn on the GPU
    (workloads.fill_device); the initial draw is freed before the outputs are allocated."""
    import torch
    import paper_2603_27467_amd as tvq

    layers = [tvq.LayerCfg(t.n_k, t.n_v, t.norm_bits_k, t.norm_bits_v, t.norm_mode_k,
                           t.norm_mode_v) for t in w.table]
    codec = tvq.Codec(w.L, w.H, w.d, layers,
                      signs=workloads.sign_table(w.sign_seed, w.L, w.d))
    n_new = args.warmup + args.steps
    cap = w.T + n_new
    lay = codec.layout(w.B, cap)
    shape = (w.L, w.B, w.H, w.T, w.d)
    print(f"# workload {w.name}: drawing {2 * np.prod(shape) * 2 / 1e9:.1f} GB of bf16 on the "
          f"GPU, cache {lay.total_bytes / 1e9:.1f} GB", file=sys.stderr, flush=True)
    stream = torch.cuda.current_stream()
    if args.paged:
        # a pool of PAGE_TOKENS-slot blocks, handed to the sequences in a shuffled order
        max_blocks = -(-cap // PAGE_TOKENS)
        n_blocks = w.B * max_blocks
        pool_lay = codec.pool_layout(n_blocks, PAGE_TOKENS)
        perm = np.random.default_rng(w.data_seed).permutation(n_blocks).astype(np.int32)
        table = torch.from_numpy(perm.reshape(w.B, max_blocks)).cuda()
        cache = torch.empty(pool_lay.total_bytes, dtype=torch.uint8, device="cuda")
        pos = torch.zeros(w.B, dtype=torch.int32, device="cuda")
        ctx = torch.zeros(w.B, dtype=torch.int32, device="cuda")
    else:
        cache = torch.empty(lay.total_bytes, dtype=torch.uint8, device="cuda")
    k = torch.empty(shape, dtype=torch.bfloat16, device="cuda")
    workloads.fill_device(w, "K", k)
    v = torch.empty_like(k)
    workloads.fill_device(w, "V", v)
    if args.paged:
        codec.encode_paged(k, v, pos, table, cache, pool_lay, stream)
        pos.fill_(w.T)
    else:
        codec.encode(k, v, cache, lay, 0, stream)
    torch.cuda.synchronize()
    del k, v
    torch.cuda.empty_cache()
    kn = torch.empty((w.L, w.B, w.H, n_new, w.d), dtype=torch.bfloat16, device="cuda")
    workloads.fill_device(w, "K", kn, token_part=1)
    vn = torch.empty_like(kn)
    workloads.fill_device(w, "V", vn, token_part=1)
    if args.attention:
        Hq = w.H * ATTN_GROUP
        g = torch.Generator(device="cuda")
        g.manual_seed(w.data_seed + 7)
        qs = torch.randn((w.L, w.B, Hq, w.d), generator=g, device="cuda").to(torch.bfloat16)
        os_ = torch.empty_like(qs)
        ws_bytes = (codec.attention_paged_workspace_bytes(w.B, Hq, cap, PAGE_TOKENS)
                    if args.paged else codec.attention_workspace_bytes(w.B, Hq, cap))
        ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
        scale = 1.0 / float(np.sqrt(w.d))
    else:
        ko = torch.empty((w.L, w.B, w.H, cap, w.d), dtype=torch.bfloat16, device="cuda")
        vo = torch.empty_like(ko)

    if args.paged:
        # the serving step: every step-varying value (positions, context lengths) lives on
        # the device, so the step can be captured once and replayed
        kin = torch.empty((w.L, w.B, w.H, 1, w.d), dtype=torch.bfloat16, device="cuda")
        vin = torch.empty_like(kin)

        def paged_step():
            # stream=None: the current stream when called (the capture stream under capture)
            codec.encode_paged(kin, vin, pos, table, cache, pool_lay)
            torch.add(pos, 1, out=ctx)
            for layer in range(w.L):
                codec.attention_paged(cache, pool_lay, table, ctx, cap, layer, qs[layer],
                                      os_[layer], scale, ws)
            pos.add_(1)

        graph = None
        if args.graph:
            torch.cuda.synchronize()
            graph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(graph):
                paged_step()
            torch.cuda.synchronize()

    def step(i, ev=None):
        t = w.T + i
        if args.paged:
            if ev is not None:
                ev[0].record(stream)
            kin.copy_(kn[:, :, :, i:i + 1])
            vin.copy_(vn[:, :, :, i:i + 1])
            if ev is not None:
                ev[1].record(stream)
            if graph is not None:
                graph.replay()
            else:
                paged_step()
            if ev is not None:
                ev[2].record(stream)
            return
        if ev is not None:
            ev[0].record(stream)
        codec.encode(kn[:, :, :, i:i + 1], vn[:, :, :, i:i + 1], cache, lay, t, stream)
        if ev is not None:
            ev[1].record(stream)
        if args.attention:
            for layer in range(w.L):
                codec.attention(cache, lay, layer, t + 1, qs[layer], os_[layer], scale, ws,
                                stream)
        else:
            codec.decode(cache, lay, 0, t + 1, ko[:, :, :, :t + 1], vo[:, :, :, :t + 1],
                         stream)
        if ev is not None:
            ev[2].record(stream)

    print(f"# warmup {args.warmup}", file=sys.stderr, flush=True)
    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    if args.copy_calibration:
        copy_calibration()
    ev = [[TimingEvent() for _ in range(3)] for _ in range(args.steps)]
    print(f"# timing {args.steps} steps", file=sys.stderr, flush=True)
    t_wall = time.perf_counter()
    for i in range(args.steps):
        step(args.warmup + i, ev[i])
    torch.cuda.synchronize()
    wall_s = time.perf_counter() - t_wall
    enc = np.array([e[0].elapsed_time(e[1]) for e in ev])
    dec = np.array([e[1].elapsed_time(e[2]) for e in ev])
    span_ms = ev[0][0].elapsed_time(ev[-1][2]) / args.steps
    ms_per_step = max(span_ms, float(enc.mean() + dec.mean()))
    # bytes of the timed steps, per step on average (the decoded range grows by one token)
    rec_tok, kv_tok, qo = longctx_bytes(w)
    t_mean = w.T + args.warmup + (args.steps - 1) / 2 + 1    # tokens decoded per step, mean
    enc_bytes = rec_tok + kv_tok
    dec_ms = float(dec.mean())
    value = (kv_tok + kv_tok * t_mean) / (ms_per_step * 1e-3) / 1e9
    if args.attention:
        # codes of every cached token once, plus the bf16 queries and outputs of every layer
        att_bytes = rec_tok * t_mean + qo
        path = attention_counters(args.workload)
        prof = None if path is None else profile_entry("tvq_attention", w.name, path,
                                                       ATTENTION_SOURCES)
        att_gbs = att_bytes / (dec_ms * 1e-3) / 1e9
        return {
            "metric": "attention over the compressed cache: bf16-equivalent KV GB/s consumed",
            "value": round(value, 2), "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
            "warmup": args.warmup, "ms_per_step": round(ms_per_step, 5),
            "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
            "dtype": "f32", "data": "synthetic",
            "config": {"workload": w.name, "layers": w.L, "batch": w.B, "kv_heads": w.H,
                       "q_heads": w.H * ATTN_GROUP, "tokens_cached": w.T, "head_dim": w.d,
                       "io_dtype": w.dtype, "table": w.notes,
                       "step": ("paged pool of %d-slot blocks (shuffled block tables), "
                                "%s: append 1 token per sequence and layer at device-side "
                                "positions, then attention of every layer over device-side "
                                "context lengths" % (PAGE_TOKENS, "one graph replay"
                                                     if args.graph else "eager launches")
                                if args.paged else
                                "encode 1 token per sequence and layer, then attention of "
                                "one query token per sequence over the whole cache, every "
                                "layer"),
                       "compressed_bytes_per_token": rec_tok},
            "roofline": {"bound": "hbm", "kernel": "tvq_attention (chunk + merge)",
                         "achieved": round(att_gbs, 2), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                         "frac": round(att_gbs / HBM_PEAK_GBPS, 4),
                         "traffic": None if prof is None else prof["hbm_bytes_per_step"],
                         "algorithmic_bytes_per_step": int(att_bytes)},
            "encode": ({"input_copy_ms": round(float(enc.mean()), 5)} if args.paged else
                       {"ms": round(float(enc.mean()), 5),
                        "ms_min": round(float(enc.min()), 5)}),
            "attention": {"ms": round(dec_ms, 5), "ms_median": round(float(np.median(dec)), 5),
                          "ms_min": round(float(dec.min()), 5),
                          "ms_per_layer": round(dec_ms / w.L, 5),
                          "hbm_GBps_algorithmic": round(att_gbs, 2)},
            "counters": None if prof is None else {
                k: prof[k] for k in ("hbm_bytes_per_step", "algorithmic_bytes_per_step",
                                     "valu_insts_per_tile", "valu_busy_pct",
                                     "lds_bank_conflict_cycles_per_tile")},
            "wall_s_timed": round(wall_s, 4),
            "kernel_source_hash": kernel_source_hash(ATTENTION_SOURCES),
        }
    dec_bytes = (rec_tok + kv_tok) * t_mean
    dec_gbs = dec_bytes / (dec_ms * 1e-3) / 1e9
    # the committed decode traffic of this workload, scaled to this run's mean range
    traffic = None
    try:
        with open(LONGCTX_DECODE_COUNTERS) as f:
            cnt = json.load(f)
        if cnt.get("workload") == w.name and cnt.get("kernel_source_hash") == kernel_source_hash():
            traffic = int(round(cnt["hbm_bytes_per_step"] * t_mean /
                                cnt["tokens_decoded_per_step_mean"]))
    except (OSError, ValueError, KeyError):
        traffic = None
    return {
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
        "config": {"workload": w.name, "layers": w.L, "batch": w.B, "kv_heads": w.H,
                   "tokens_cached": w.T, "head_dim": w.d, "io_dtype": w.dtype,
                   "table": w.notes, "step": "encode 1 token per sequence and layer, then "
                                             "decode the whole cache",
                   "compressed_bytes_per_token": rec_tok},
        "roofline": {"bound": "hbm", "kernel": "tvq_decode",
                     "achieved": round(dec_gbs, 2), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(dec_gbs / HBM_PEAK_GBPS, 4), "traffic": traffic,
                     "algorithmic_bytes_per_launch": int(dec_bytes)},
        "encode": {"ms": round(float(enc.mean()), 5), "ms_min": round(float(enc.min()), 5),
                   "vectors": 2 * w.L * w.B * w.H, "algorithmic_bytes": enc_bytes},
        "decode": {"ms": round(dec_ms, 5), "ms_median": round(float(np.median(dec)), 5),
                   "ms_min": round(float(dec.min()), 5),
                   "hbm_GBps_algorithmic": round(dec_gbs, 2),
                   "frac_of_peak": round(dec_gbs / HBM_PEAK_GBPS, 4),
                   "vectors_per_s": round(2 * w.L * w.B * w.H * t_mean / (dec_ms * 1e-3), 1)},
        "wall_s_timed": round(wall_s, 4),
        "kernel_source_hash": kernel_source_hash(),
    }


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="C2")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--attention", action="store_true",
                    help="attention over the compressed cache in place of the full decode "
                         "(the long-context cache of C5, or the cache of the workload named)")
    ap.add_argument("--encode-mfma", action="store_true",
                    help="encode with the matrix-core transform schedule (comparison)")
    ap.add_argument("--paged", action="store_true",
                    help="long-context attention step over a paged pool (implies --attention)")
    ap.add_argument("--graph", action="store_true",
                    help="with --paged: capture the step once and replay it")
    ap.add_argument("--pool", action="store_true",
                    help="encode and decode through a paged pool (blocks of PAGE_TOKENS slots "
                         "handed out in a shuffled order) in place of a contiguous cache")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run a plain 1 GiB device copy (for counter scaling)")
    ap.add_argument("--summarize-profiles", nargs=5,
                    metavar=("TRACE", "FETCH", "WRITE", "SQ", "VALU"),
                    help="write the profiles/ counter summary of the --workload codec step "
                         "(C2, C3 or C4) from rocprofv3 output dirs")
    ap.add_argument("--summarize-attention-profiles", nargs=6,
                    metavar=("TRACE", "FETCH", "WRITE", "SQ", "VALU", "STEPS_TOTAL"),
                    help="write the profiles/ counter summary of the attention step over "
                         "the --workload cache (C5 or C4) from rocprofv3 output dirs")
    ap.add_argument("--summarize-longctx-decode", nargs=3,
                    metavar=("FETCH", "WRITE", "STEPS_TOTAL"),
                    help="write the profiles/ traffic summary of the long-context decode (C5)")
    ap.add_argument("--commands", nargs="*", default=[],
                    help="the profiling commands, recorded in the summary")
    args = ap.parse_args()
    if args.paged:
        args.attention = True
    if args.pool and (args.encode_mfma or args.attention or args.workload == "C5"):
        print("--pool runs the codec step of C1-C4 with the canonical encode only",
              file=sys.stderr)
        return 2
    if args.summarize_profiles:
        return summarize_profiles(*args.summarize_profiles, args.commands, args.workload)
    if args.summarize_longctx_decode:
        a = args.summarize_longctx_decode
        return summarize_longctx_decode(a[0], a[1], args.commands, int(a[2]))
    if args.summarize_attention_profiles:
        a = args.summarize_attention_profiles
        return summarize_attention_profiles(*a[:5], args.commands, int(a[5]), args.workload)
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on one GPU only: the codec is per-vector and the bench measures "
              "one GPU's share; --gpus above 1 is not supported", file=sys.stderr)
        return 2

    import torch
    import paper_2603_27467_amd as tvq

    if not torch.cuda.is_available():
        print("no GPU visible", file=sys.stderr)
        return 1
    w = workloads.get(args.workload)
    if args.workload == "C5" or args.attention:
        # the serving step over a cache of the workload's shape (C5: the long-context cache;
        # --attention on another workload: attention over that workload's cache, e.g. d = 64)
        out = run_longctx(w, args)
        if not args.no_cpu_baseline:
            print("# cpu baseline (oracle on host cores)", file=sys.stderr, flush=True)
            out["cpu_baseline"] = (cpu_baseline_attention(w) if args.attention
                                   else cpu_baseline(w))
        print(json.dumps(out), flush=True)
        return 0
    ab = algorithmic_bytes(w)
    print(f"# workload {w.name}: generating inputs", file=sys.stderr, flush=True)
    k = workloads.generate(w, "K")
    v = workloads.generate(w, "V")
    conv = (lambda a: torch.from_numpy(a.view(np.int16)).view(torch.bfloat16)) \
        if w.dtype == "bf16" else torch.from_numpy
    kd, vd = conv(k).cuda(), conv(v).cuda()
    del k, v
    layers = [tvq.LayerCfg(t.n_k, t.n_v, t.norm_bits_k, t.norm_bits_v, t.norm_mode_k,
                           t.norm_mode_v) for t in w.table]
    codec = tvq.Codec(w.L, w.H, w.d, layers,
                      signs=workloads.sign_table(w.sign_seed, w.L, w.d))
    stream = torch.cuda.current_stream()
    if args.pool:
        # the same records in a pool of PAGE_TOKENS-slot blocks, shuffled over the sequences
        max_blocks = -(-w.T // PAGE_TOKENS)
        n_blocks = w.B * max_blocks
        lay = codec.pool_layout(n_blocks, PAGE_TOKENS)
        perm = np.random.default_rng(w.data_seed).permutation(n_blocks).astype(np.int32)
        table = torch.from_numpy(perm.reshape(w.B, max_blocks)).cuda()
        pos0 = torch.zeros(w.B, dtype=torch.int32, device="cuda")

        def encode_to(c):
            codec.encode_paged(kd, vd, pos0, table, c, lay, stream)

        def decode_from(c, ko, vo):
            codec.decode_paged(c, lay, table, 0, w.T, ko, vo, stream)
    else:
        lay = codec.layout(w.B, w.T)
        encode = codec.encode_mfma if args.encode_mfma else codec.encode

        def encode_to(c):
            encode(kd, vd, c, lay, 0, stream)

        def decode_from(c, ko, vo):
            codec.decode(c, lay, 0, w.T, ko, vo, stream)
    caches = [torch.empty(lay.total_bytes, dtype=torch.uint8, device="cuda") for _ in range(2)]
    outs = [(torch.empty_like(kd), torch.empty_like(vd)) for _ in range(2)]
    for c in caches:                        # both caches hold the encoded workload
        encode_to(c)

    def step(i, ev=None):
        if ev is not None:
            ev[0].record(stream)
        encode_to(caches[i % 2])
        if ev is not None:
            ev[1].record(stream)
        ko, vo = outs[i % 2]
        decode_from(caches[(i + 1) % 2], ko, vo)
        if ev is not None:
            ev[2].record(stream)

    print(f"# warmup {args.warmup}", file=sys.stderr, flush=True)
    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()

    if args.copy_calibration:
        copy_calibration()

    ev = [[TimingEvent() for _ in range(3)] for _ in range(args.steps)]
    print(f"# timing {args.steps} steps", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    t_wall = time.perf_counter()
    for i in range(args.steps):
        step(args.warmup + i, ev[i])
    torch.cuda.synchronize()
    wall_s = time.perf_counter() - t_wall
    print("# streaming copy", file=sys.stderr, flush=True)
    copy = copy_peak()
    enc = np.array([e[0].elapsed_time(e[1]) for e in ev])
    dec = np.array([e[1].elapsed_time(e[2]) for e in ev])
    span_ms = ev[0][0].elapsed_time(ev[-1][2]) / args.steps
    ms_per_step = max(span_ms, float(enc.mean() + dec.mean()))

    def leg(ms_all, name):
        kern = f"tvq_{name}"
        ms = float(ms_all.mean())
        gbs = ab["per_launch"] / (ms * 1e-3) / 1e9
        # the committed counters cover the canonical-schedule encode of a contiguous cache
        path = codec_counters(args.workload)
        prof = (None if (args.encode_mfma and name == "encode") or args.pool or path is None
                else profile_entry(kern, w.name, path))
        out = {"ms": round(ms, 5), "ms_median": round(float(np.median(ms_all)), 5),
               "ms_min": round(float(ms_all.min()), 5),
               "kv_GBps": round(ab["kv"] / (ms * 1e-3) / 1e9, 2),
               "hbm_GBps_algorithmic": round(gbs, 2),
               "frac_of_peak": round(gbs / HBM_PEAK_GBPS, 4),
               "frac_of_peak_at_min": round(ab["per_launch"] / (ms_all.min() * 1e-3) / 1e9
                                            / HBM_PEAK_GBPS, 4),
               "frac_of_copy_peak": round(gbs / copy["GBps_mean"], 4),
               "vectors_per_s": round(ab["vectors"] / (ms * 1e-3), 1),
               "traffic_bytes_per_launch": None if prof is None else prof["hbm_bytes_per_launch"]}
        if prof is not None:
            # VALU issue: instructions of one launch (counters) over this run's launch time, at
            # the 2.4 GHz peak clock and at the clock the profiled launches sustained
            clk = prof.get("clock_ghz_sustained")
            out["valu"] = {"insts_per_launch": prof["valu_insts_per_launch"],
                           "insts_per_tile": prof["valu_insts_per_tile"],
                           "busy_pct_profiled": prof["valu_busy_pct"],
                           "issue_frac": round(prof["valu_insts_per_launch"] / (ms * 1e-3)
                                               / VALU_ISSUE_PEAK, 4)}
            if clk:
                out["valu"]["issue_frac_at_clock"] = round(
                    prof["valu_insts_per_launch"] / (ms * 1e-3) / (VALU_ISSUE_PEAK * clk / 2.4), 4)
                t_ns = prof["trace_timed_avg_ns"]
                out["profiled"] = {
                    "trace_timed_avg_us": round(t_ns / 1e3, 2),
                    "frac_of_peak_trace_timed": round(ab["per_launch"] / (t_ns * 1e-9) / 1e9
                                                      / HBM_PEAK_GBPS, 4),
                    "clock_ghz_sustained": clk, "clock_ghz_single_dispatch":
                        prof["clock_ghz_pmc"]}
        return out

    e_leg, d_leg = leg(enc, "encode"), leg(dec, "decode")
    dom_name, dom = ("encode", e_leg) if e_leg["ms"] >= d_leg["ms"] else ("decode", d_leg)
    value = 2 * ab["kv"] / (ms_per_step * 1e-3) / 1e9
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
        "config": {"workload": w.name, "layers": w.L, "batch": w.B, "kv_heads": w.H,
                   "tokens": w.T, "head_dim": w.d, "io_dtype": w.dtype,
                   "table": w.notes, "kv_bytes_per_direction": ab["kv"],
                   "compressed_bytes": ab["compressed"],
                   "encode_schedule": ("matrix-core stages, comparison (tvq_encode_mfma)"
                                       if args.encode_mfma else "canonical butterfly"),
                   "cache": (f"paged pool, {PAGE_TOKENS}-slot blocks in a shuffled order "
                             "(tvq_encode_paged / tvq_decode_paged)" if args.pool
                             else "contiguous")},
        "roofline": {"bound": "hbm", "kernel": f"tvq_{dom_name}",
                     "achieved": dom["hbm_GBps_algorithmic"], "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": dom["frac_of_peak"],
                     "traffic": dom["traffic_bytes_per_launch"],
                     "algorithmic_bytes_per_launch": ab["per_launch"]},
        "encode": e_leg,
        "decode": d_leg,
        "wall_s_timed": round(wall_s, 4),
        "copy_peak": copy,
        "kernel_source_hash": kernel_source_hash(),
    }
    if "valu" in dom:
        out["roofline"]["valu_issue_frac"] = dom["valu"]["issue_frac"]
        if "issue_frac_at_clock" in dom["valu"]:
            out["roofline"]["valu_issue_frac_at_clock"] = dom["valu"]["issue_frac_at_clock"]
    if "profiled" in dom:
        # the committed kernel trace of the same kernel: its timed dispatches' mean duration,
        # the fraction of the roofline at it, and the shader clock it implies
        out["roofline"]["frac_trace"] = dom["profiled"]["frac_of_peak_trace_timed"]
        out["roofline"]["trace_avg_us"] = dom["profiled"]["trace_timed_avg_us"]
        out["roofline"]["clock_ghz"] = dom["profiled"]["clock_ghz_sustained"]
    if not args.no_cpu_baseline:
        print("# cpu baseline (oracle on host cores)", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(w)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
