"""Benchmark of the TurboAngle KV-cache codec on one MI355X.

One step = one pass of the whole hot path over the Mistral-7B-shaped cache (32 layers, 8 KV
heads, 4096 tokens, d = 128, bf16, n = 64 angle bins, K 8-bit linear / V 4-bit log norms):
encode all of K and V into the compressed cache, then decode the whole cache back to bf16.
Inputs are seeded synthetic tensors resident in HBM before the timed region.

    python bench.py [--steps K] [--warmup W] [--workload C2|C3|C4] [--no-cpu-baseline]

Prints one JSON line.  `value` is bf16 KV bytes through the codec per second, counting the
bytes encoded and the bytes decoded in a step (2 x 512 MiB at the default workload), divided
by the step time.
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
PROFILE_COUNTERS = os.path.join(ROOT, "profiles", "hbm_traffic.json")
KERNEL_SOURCES = ["tvq_encode.hip", "tvq_decode.hip", "tvq_device.h", "tvq_internal.h"]


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for name in KERNEL_SOURCES:
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


def traffic_from_profiles(kernel: str):
    """HBM bytes per launch measured with rocprofv3 FETCH_SIZE / WRITE_SIZE and scaled by the
    same counters on a copy of known size; None when absent or when the kernel sources have
    changed since the counters were taken."""
    try:
        with open(PROFILE_COUNTERS) as f:
            d = json.load(f)
    except (OSError, ValueError):
        return None
    if d.get("kernel_source_hash") != kernel_source_hash():
        return None
    ent = d.get("kernels", {}).get(kernel)
    return None if ent is None else ent.get("hbm_bytes_per_launch")


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
    elem_bytes = 2 if w.dtype == "bf16" else 4
    kv_bytes = vecs * w.d * elem_bytes
    return {"value": round(2 * kv_bytes / wall / 1e9, 4), "unit": "GB/s", "cores": cores,
            "kind": "oracle",
            "sample": f"{len(tasks)} chunks of {chunk} tokens x {w.B * w.H} (batch, head) rows "
                      f"x (K, V) spread over all {w.L} layers, {vecs // passes} vectors, encoded "
                      f"and decoded {passes} times: {vecs} vectors in {wall:.1f} s on {cores} "
                      f"threads; same unit as value (bf16 KV bytes encoded + decoded per second)"}


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="C2")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run a plain device copy of known size (for counter scaling)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on one GPU only: the codec is per-vector and this build measures "
              "one GPU's share; --gpus above 1 is not supported", file=sys.stderr)
        return 2

    import torch
    import paper_2603_27467_amd as tvq

    if not torch.cuda.is_available():
        print("no GPU visible", file=sys.stderr)
        return 1
    w = workloads.get(args.workload)
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
    lay = codec.layout(w.B, w.T)
    cache = torch.empty(lay.total_bytes, dtype=torch.uint8, device="cuda")
    ko, vo = torch.empty_like(kd), torch.empty_like(vd)
    stream = torch.cuda.current_stream()

    def step():
        codec.encode(kd, vd, cache, lay, 0, stream)
        codec.decode(cache, lay, 0, w.T, ko, vo, stream)

    print(f"# warmup {args.warmup}", file=sys.stderr, flush=True)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    if args.copy_calibration:
        src = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()

    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    print(f"# timing {args.steps} steps", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    t_wall = time.perf_counter()
    for i in range(args.steps):
        ev[i][0].record(stream)
        codec.encode(kd, vd, cache, lay, 0, stream)
        ev[i][1].record(stream)
        codec.decode(cache, lay, 0, w.T, ko, vo, stream)
        ev[i][2].record(stream)
    torch.cuda.synchronize()
    wall_s = time.perf_counter() - t_wall
    enc_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in ev]))
    dec_ms = float(np.mean([e[1].elapsed_time(e[2]) for e in ev]))
    span_ms = ev[0][0].elapsed_time(ev[-1][2]) / args.steps
    ms_per_step = max(span_ms, enc_ms + dec_ms)

    def leg(ms, name):
        kern = f"tvq_{name}"
        bytes_per = ab["per_launch"]
        gbs = bytes_per / (ms * 1e-3) / 1e9
        return {"ms": round(ms, 5), "kv_GBps": round(ab["kv"] / (ms * 1e-3) / 1e9, 2),
                "hbm_GBps_algorithmic": round(gbs, 2), "frac_of_peak": round(gbs / HBM_PEAK_GBPS, 4),
                "vectors_per_s": round(ab["vectors"] / (ms * 1e-3), 1),
                "traffic_bytes_per_launch": traffic_from_profiles(kern)}

    enc, dec = leg(enc_ms, "encode"), leg(dec_ms, "decode")
    dom_name, dom = ("encode", enc) if enc_ms >= dec_ms else ("decode", dec)
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
                   "compressed_bytes": ab["compressed"]},
        "roofline": {"bound": "hbm", "kernel": f"tvq_{dom_name}",
                     "achieved": dom["hbm_GBps_algorithmic"], "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": dom["frac_of_peak"],
                     "traffic": dom["traffic_bytes_per_launch"],
                     "algorithmic_bytes_per_launch": ab["per_launch"]},
        "encode": enc,
        "decode": dec,
        "wall_s_timed": round(wall_s, 4),
        "kernel_source_hash": kernel_source_hash(),
    }
    if not args.no_cpu_baseline:
        print("# cpu baseline (oracle on host cores)", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(w)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
