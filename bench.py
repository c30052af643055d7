#!/usr/bin/env python3
"""Throughput benchmark: target tokens/s of whole-job batched translation on one MI355X.

One step = one nt_translate call over the whole synthetic workload (sorting, dynamic
batching, DLCL encoder, cached decoder steps, search, pruning, results back in host
memory), with inputs and weights generated beforehand.  Prints one JSON line.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload wide-30-6]

The default workload is the largest configuration, the wide teacher-size model (d = 1024,
30-layer DLCL encoder, 6-layer decoder, beam 4, 4096 sentences).  Batches are decoded four
at a time on their own streams (the library default), each decoder step replayed from a
captured HIP graph.  The line carries a roofline entry for the dominant kernel class,
timed with HIP events on the launch stream inside the timed region: up to 40 units
(decoder steps or batch encodes; at most 2 per timed step) are sampled, and each sample
runs alone on the GPU so that its kernel durations are the kernel's own.  Next to that per-launch rate the entry
gives the class's algorithmic work per translation over the timed step's wall time
(`in_pipeline`), and how much kernel time the concurrent batches overlap (`overlap`).
It also carries the CPU oracle's throughput on a bounded sample of the same workload
(the oracle as written, one process per core).
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import synth  # noqa: E402

PEAK = {  # MI355X published peaks (dense)
    "hbm_GBps": 8000.0,
    # FP8 weights are widened to fp16 inside the GEMM, whose contraction runs on the fp16 MFMA
    "mfma_TFLOPs": {"f16": 2500.0, "bf16": 2500.0, "f8": 2500.0, "f8w": 2500.0, "f32": 157.3},
}
GEMM_CLASSES = (0, 1, 2)

# HBM-side bytes per launch of a kernel class on a workload, from two rocprofv3 --pmc
# passes (FETCH_SIZE, WRITE_SIZE; KiB per dispatch averaged over every dispatch of the
# class) scaled by what the same counters read for a plain 512 MiB device copy (FETCH_SIZE
# reads half the bytes moved, WRITE_SIZE all of them).  Valid only for the kernel source
# the counters were taken on (sha256 over `files`); otherwise the bench reports null.
GEMM_FILES = ["paper_2109_08008_amd/csrc/nt_gemm.hip", "paper_2109_08008_amd/csrc/nt_common.h"]
TRAFFIC = {
    ("gemm_dec", "wide-30-6"): {
        "files": GEMM_FILES, "sha256": "8696ca14961f0c4ac045848f028eeab73e938a62840b3e44679dde3faaf0af44",
        "fetch_kib": 12662.90, "write_kib": 4063.62, "fetch_scale": 2.0, "write_scale": 1.0,
    },
    ("gemm_enc", "wide-30-6"): {
        "files": GEMM_FILES, "sha256": "8696ca14961f0c4ac045848f028eeab73e938a62840b3e44679dde3faaf0af44",
        "fetch_kib": 111992.06, "write_kib": 74738.06, "fetch_scale": 2.0, "write_scale": 1.0,
    },
    ("gemm_vocab", "wide-30-6"): {
        "files": GEMM_FILES, "sha256": "8696ca14961f0c4ac045848f028eeab73e938a62840b3e44679dde3faaf0af44",
        "fetch_kib": 44495.21, "write_kib": 5086.86, "fetch_scale": 2.0, "write_scale": 1.0,
    },
    ("gemm_dec", "base-6-6"): {
        "files": GEMM_FILES, "sha256": "8696ca14961f0c4ac045848f028eeab73e938a62840b3e44679dde3faaf0af44",
        "fetch_kib": 3929.49, "write_kib": 1303.11, "fetch_scale": 2.0, "write_scale": 1.0,
    },
    ("gemm_enc", "base-6-6"): {
        "files": GEMM_FILES, "sha256": "8696ca14961f0c4ac045848f028eeab73e938a62840b3e44679dde3faaf0af44",
        "fetch_kib": 15480.32, "write_kib": 19806.60, "fetch_scale": 2.0, "write_scale": 1.0,
    },
    ("gemm_vocab", "base-6-6"): {
        "files": GEMM_FILES, "sha256": "8696ca14961f0c4ac045848f028eeab73e938a62840b3e44679dde3faaf0af44",
        "fetch_kib": 13998.60, "write_kib": 3141.33, "fetch_scale": 2.0, "write_scale": 1.0,
    },
    ("gemm_enc", "deep-shallow-greedy"): {
        "files": GEMM_FILES, "sha256": "8696ca14961f0c4ac045848f028eeab73e938a62840b3e44679dde3faaf0af44",
        "fetch_kib": 15286.01, "write_kib": 17941.79, "fetch_scale": 2.0, "write_scale": 1.0,
    },
    ("gemm_dec", "deep-shallow-greedy"): {
        "files": GEMM_FILES, "sha256": "8696ca14961f0c4ac045848f028eeab73e938a62840b3e44679dde3faaf0af44",
        "fetch_kib": 2063.13, "write_kib": 411.51, "fetch_scale": 2.0, "write_scale": 1.0,
    },
    ("gemm_vocab", "deep-shallow-greedy"): {
        "files": GEMM_FILES, "sha256": "8696ca14961f0c4ac045848f028eeab73e938a62840b3e44679dde3faaf0af44",
        "fetch_kib": 17058.90, "write_kib": 945.94, "fetch_scale": 2.0, "write_scale": 1.0,
    },
    ("gemm_enc", "deep-shallow-beam"): {
        "files": GEMM_FILES, "sha256": "8696ca14961f0c4ac045848f028eeab73e938a62840b3e44679dde3faaf0af44",
        "fetch_kib": 34254.48, "write_kib": 36548.84, "fetch_scale": 2.0, "write_scale": 1.0,
    },
    ("gemm_vocab", "deep-shallow-beam"): {
        "files": GEMM_FILES, "sha256": "8696ca14961f0c4ac045848f028eeab73e938a62840b3e44679dde3faaf0af44",
        "fetch_kib": 22423.13, "write_kib": 6903.01, "fetch_scale": 2.0, "write_scale": 1.0,
    },
    ("gemm_dec", "deep-shallow-beam"): {
        "files": GEMM_FILES, "sha256": "8696ca14961f0c4ac045848f028eeab73e938a62840b3e44679dde3faaf0af44",
        "fetch_kib": 5920.51, "write_kib": 2873.06, "fetch_scale": 2.0, "write_scale": 1.0,
    },
}


def traffic_bytes(kernel: str, workload: str):
    import hashlib
    t = TRAFFIC.get((kernel, workload))
    if t is None:
        return None
    h = hashlib.sha256()
    for f in t["files"]:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    if h.hexdigest() != t["sha256"]:
        return None   # the kernel changed since the counters were taken
    return round((t["fetch_kib"] * t["fetch_scale"] + t["write_kib"] * t["write_scale"]) * 1024)
ENCODE_ONLY_CLASSES = (0, 3, 5)   # launched only by batch encodes (GEMM_ENC, DLCL, ATTN_ENC)


def parse_args():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="wide-30-6", choices=sorted(synth.WORKLOADS))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-graphs", action="store_true", help="launch decoder steps kernel by kernel")
    ap.add_argument("--no-beam-fused", action="store_true",
                    help="beam search stores the fp32 logits and scans them (the default keeps them out of HBM)")
    ap.add_argument("--streams", type=int, default=0, help="batches decoded concurrently (0: library default)")
    ap.add_argument("--samples", type=int, default=40,
                    help="timing samples (isolated units) in the timed region, at most 2 per timed step")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="target CPU work for the oracle sample")
    ap.add_argument("--cpu-procs", type=int, default=0, help="oracle processes (0: min(16, cores))")
    ap.add_argument("--cpu-full", action="store_true",
                    help="time the oracle on the whole sentence set instead of a bounded sample (slow)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run three 512 MiB device copies (the reference kernel that HBM counters are "
                         "scaled by) and exit")
    return ap.parse_args()


def calibrate_copy() -> dict:
    """Three plain device copies of 512 MiB (fp32 tensors of 128 Mi elements): the kernel of
    known traffic (512 MiB read and 512 MiB written each) that the FETCH_SIZE / WRITE_SIZE
    readings of the library's kernels are scaled by."""
    import torch
    n = 1 << 27
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    return {"copies": 3, "bytes_read_each": 4 * n, "bytes_written_each": 4 * n}


def roofline_entry(cls: int, prof: dict, dtype: str, workload: str) -> dict:
    """Roofline of one kernel class from its event timings and algorithmic work.  The
    bound follows the class's algorithmic intensity (flops over the bytes the method must
    move: weights, keys/values, logits) against the ridge of the peaks."""
    from paper_2109_08008_amd import nt
    n = max(prof["launches"], 1)
    sec = prof["ms"] / 1e3
    intensity = prof["flops"] / max(prof["bytes"], 1.0)
    ridge = PEAK["mfma_TFLOPs"][dtype] * 1e12 / (PEAK["hbm_GBps"] * 1e9)
    if cls in GEMM_CLASSES and intensity >= ridge:
        achieved = prof["flops"] / sec / 1e12
        peak = PEAK["mfma_TFLOPs"][dtype]
        bound, unit = "mfma", "TFLOP/s"
    else:
        achieved = prof["bytes"] / sec / 1e9
        peak = PEAK["hbm_GBps"]
        bound, unit = "hbm", "GB/s"
    return {
        "bound": bound, "achieved": round(achieved, 2), "peak": peak, "unit": unit,
        "frac": round(achieved / peak, 4), "traffic": traffic_bytes(nt.KERNEL_CLASSES[cls], workload),
        "traffic_unit": "HBM-side bytes per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, copy-calibrated)",
        "kernel": nt.KERNEL_CLASSES[cls], "launches": prof["launches"],
        "avg_us": round(prof["ms"] * 1e3 / n, 2),
        "alg_bytes_per_launch": round(prof["bytes"] / n), "alg_flops_per_launch": round(prof["flops"] / n),
    }


DECODE_CLASSES = (1, 2, 4, 6, 7, 8, 9)   # decoder-step kernels (LN also counts the encoder's LN2)


def phase_rooflines(breakdown: dict, dtype: str) -> dict:
    """The metric's two fractions from the all-class profile (every unit run alone):
    encoder GEMM MFMA utilisation and the decode step's effective HBM rate (algorithmic
    bytes / kernel time), both against MI355X's published peaks."""
    from paper_2109_08008_amd import nt
    enc = breakdown[nt.KERNEL_CLASSES[0]]
    dec = [breakdown[nt.KERNEL_CLASSES[c]] for c in DECODE_CLASSES]
    enc_tf = enc["flops"] / max(enc["ms"], 1e-9) / 1e9
    dec_gbs = sum(x["bytes"] for x in dec) / max(sum(x["ms"] for x in dec), 1e-9) / 1e6
    return {
        "encoder_gemm_mfma": {"achieved": round(enc_tf, 2), "peak": PEAK["mfma_TFLOPs"][dtype], "unit": "TFLOP/s",
                              "frac": round(enc_tf / PEAK["mfma_TFLOPs"][dtype], 4)},
        "decode_step_hbm": {"achieved": round(dec_gbs, 2), "peak": PEAK["hbm_GBps"], "unit": "GB/s",
                            "frac": round(dec_gbs / PEAK["hbm_GBps"], 4),
                            "note": "algorithmic bytes of the decoder-step kernel classes (weights, keys/values, "
                                    "logits) / their kernel time"},
    }


def achievable_peaks() -> dict:
    """Probes of what this GPU delivers: a 1 GiB device copy (GB/s of read + write) and a
    large fp16 matrix product through the vendor library (torch.matmul -> hipBLASLt)."""
    import torch
    n = 1 << 28
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    a = torch.randn(8192, 8192, dtype=torch.float16, device="cuda")
    b = torch.randn(8192, 8192, dtype=torch.float16, device="cuda")

    def timeit(fn, reps):
        fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / 1e3 / reps

    copy_s = timeit(lambda: dst.copy_(src), 10)
    mm_s = timeit(lambda: torch.matmul(a, b), 10)
    out = {"copy_GBps": round(2 * n * 4 / copy_s / 1e9, 1), "gemm_fp16_TFLOPs": round(2 * 8192 ** 3 / mm_s / 1e12, 1),
           "note": "1 GiB device copy; torch.matmul 8192^3 fp16"}
    del src, dst, a, b
    torch.cuda.empty_cache()
    return out


# ---- CPU oracle baseline ------------------------------------------------------------------
_ORACLE = {}


def _oracle_translate(src):
    import oracle
    from oracle.ensemble import translate_ensemble
    if isinstance(_ORACLE["model"], list):
        return translate_ensemble(_ORACLE["model"], src, _ORACLE["search"], _ORACLE["rule"])
    return oracle.translate(_ORACLE["model"], src, _ORACLE["search"])


def _oracle_worker(idx):
    from threadpoolctl import threadpool_limits
    with threadpool_limits(limits=1):
        return len(_oracle_translate(_ORACLE["srcs"][idx]).tokens)


def cpu_baseline(w: synth.Workload, blobs, ids, offs, seconds: float, procs: int, full: bool = False) -> dict:
    """The fp32 oracle on a length-stratified sample (or, with full, every sentence), split
    over processes (one BLAS thread each) the way the paper splits CPU decoding by lines."""
    import multiprocessing as mp
    import oracle
    from threadpoolctl import threadpool_limits

    P = procs or min(16, os.cpu_count() or 1)
    srcs = synth.sentence_list(ids, offs)
    if w.members:
        model = [oracle.OracleModel(mb.model, b, np.float32, hist_norm=mb.dlcl) for mb, b in zip(w.members, blobs)]
    else:
        model = oracle.OracleModel(w.model, blobs[0], np.float32)
    _ORACLE.update(model=model, srcs=srcs, search=w.search, rule=w.ensemble_rule)
    # calibrate on the median-length sentence, then size the sample to ~`seconds` of work
    order = synth.stratified_subset(offs, len(srcs))
    probe = int(order[len(order) // 2])
    with threadpool_limits(limits=1):
        t0 = time.perf_counter()
        _oracle_translate(srcs[probe])
        t_one = time.perf_counter() - t0
    n = len(srcs) if full else int(min(len(srcs), max(P, P * max(1, math.floor(seconds / max(t_one, 1e-3))))))
    sample = synth.stratified_subset(offs, n)
    ctx = mp.get_context("fork")
    with ctx.Pool(P) as pool:
        t0 = time.perf_counter()
        toks = pool.map(_oracle_worker, [int(i) for i in sample], chunksize=1)
        dt = time.perf_counter() - t0
    return {
        "value": round(sum(toks) / dt, 2), "unit": "tokens/s", "cores": P, "kind": "oracle",
        "sample": f"{n} of {len(srcs)} sentences, every ({len(srcs)}/{n})-th of the length-sorted order; "
                  f"fp32 NumPy oracle, {P} processes x 1 BLAS thread; {sum(toks)} target tokens in {dt:.1f} s",
        "host_cpu_count": os.cpu_count(),
    }


def main():
    args = parse_args()
    if args.calibrate_copy:
        print(json.dumps(calibrate_copy()), flush=True)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} is not supported by this build "
              "(sentences are independent: a multi-GPU run would shard batches across replicas)", file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2109_08008_amd import nt

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    peaks = achievable_peaks()
    w = synth.WORKLOADS[args.workload]
    blobs = synth.member_weights(w) if w.members else [synth.make_weights(w.model, seed=w.weights_seed)]
    ids, offs = synth.make_sentences(w.data, w.model.vocab, seed=w.data_seed)
    nt.nt_set_graphs(not args.no_graphs)
    nt.nt_set_beam_fused(not args.no_beam_fused)
    if args.streams:
        nt.nt_set_streams(args.streams)
    if w.members:   # ensemble decoding: every member scores each step
        model = nt.Ensemble([nt.Model(mb.model, b, w.dtype, hist_norm=mb.dlcl) for mb, b in zip(w.members, blobs)],
                            w.ensemble_rule)
    else:
        model = nt.Model(w.model, blobs[0], w.dtype)
    sc = nt.search_cfg(w.search)
    ws_bytes = nt.nt_translate_workspace_size(model.handle, sc, offs)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
    cap = int(sum(synth.max_target_len(w.search, int(L)) for L in np.diff(offs)))
    stream = torch.cuda.current_stream().cuda_stream

    def step():
        return nt.nt_translate(model.handle, sc, ids, offs, cap, ws.data_ptr(), ws_bytes, stream)

    # warmup; the last warmup step times every unit (decoder step or batch encode), each
    # run alone, to find the dominant kernel class and count the units of one step
    breakdown = {}
    for i in range(max(args.warmup, 1)):
        if i == max(args.warmup, 1) - 1:
            nt.nt_prof_reset()
            nt.nt_prof_enable((1 << len(nt.KERNEL_CLASSES)) - 1)
        step()
    torch.cuda.synchronize()
    enc_units, step_units = nt.nt_prof_units()
    for c, name in enumerate(nt.KERNEL_CLASSES):
        breakdown[name] = nt.nt_prof_get(c)
    nt.nt_prof_enable(0)
    dominant = max(range(len(nt.KERNEL_CLASSES)), key=lambda c: breakdown[nt.KERNEL_CLASSES[c]]["ms"])

    # timed region: events on the dominant class in about `samples` units, each run alone
    # (the other batches' streams drained first) so that they time the kernel by itself
    # A sample drains the other batches' streams and runs alone, which stalls the pipeline
    # for about one unit: at most 2 per timed step keeps that near 1% of the timed run.
    # The stride advances the sampled position within a translation by units / samples
    # from one timed step to the next, so the samples spread over the whole translation
    # (its long-sentence first batches and short-sentence last ones, early and late steps)
    # instead of landing on the same units in every timed step.
    units = enc_units if dominant in ENCODE_ONLY_CLASSES else step_units
    samples = max(1, min(args.samples, 2 * args.steps))
    per_step = max(1, samples // args.steps)
    stride = max(1, units // per_step + units // samples)
    nt.nt_prof_reset()
    nt.nt_prof_config(1 << dominant, stride)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        out, out_off, score, _ = step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    nt.nt_prof_enable(0)
    prof = nt.nt_prof_get(dominant)
    n_tokens = int(out_off[-1])
    elapsed = t1 - t0
    value = n_tokens * args.steps / elapsed

    # the dominant class inside the timed run: its algorithmic work per translation (every
    # launch, from the all-unit profile) over the timed step's wall time; and how much of
    # the kernels' own time the concurrent batches hide
    dom = breakdown[nt.KERNEL_CLASSES[dominant]]
    rl = roofline_entry(dominant, prof, w.dtype, w.name)
    step_s = elapsed / args.steps
    work = dom["flops"] if rl["bound"] == "mfma" else dom["bytes"]
    pipe = work / step_s / (1e12 if rl["bound"] == "mfma" else 1e9)
    rl["in_pipeline"] = {
        "achieved": round(pipe, 2), "frac": round(pipe / rl["peak"], 4),
        "note": "the class's algorithmic work per translation (all its launches) / the timed step's wall time",
    }
    rl["overlap"] = round(sum(v["ms"] for v in breakdown.values()) / (step_s * 1e3), 3)
    rl["sampled_units_stride"] = stride
    rl["timing"] = ("HIP events around every launch of the class in the sampled units of the timed region, "
                    "each unit run alone on the GPU")

    line = {
        "metric": "target tokens/sec translated (fp16, 1 GPU); encoder MFMA util; decode HBM GB/s",
        "value": round(value, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(elapsed / args.steps * 1e3, 2),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic (seeded token IDs and N(0,0.02) weights of the workload's shapes)",
        "config": {
            "workload": w.name, "description": w.description, "sentences": int(len(offs) - 1),
            "source_tokens": int(offs[-1]), "target_tokens_per_step": n_tokens,
            "beam": w.search.beam, "token_budget": w.search.token_budget,
            "d_model": w.model.d_model, "n_enc": w.model.n_enc, "n_dec": w.model.n_dec, "vocab": w.model.vocab,
            "decode_step_graphs": not args.no_graphs, "beam_logits_in_hbm": bool(args.no_beam_fused), "concurrent_batches": args.streams or 4,
            "workspace_GB": round(ws_bytes / 1e9, 2),
        },
        "roofline": rl,
        "phase_rooflines": phase_rooflines(breakdown, w.dtype),
        "achievable_peaks": peaks,
        "kernel_ms_per_step_alone": {k: round(v["ms"], 3) for k, v in breakdown.items()},
        "kernel_classes_per_step": {k: {"launches": v["launches"], "ms_alone": round(v["ms"], 3),
                                        "alg_MB": round(v["bytes"] / 1e6, 2), "alg_GFLOP": round(v["flops"] / 1e9, 2)}
                                    for k, v in breakdown.items()},
    }
    if w.members:
        line["config"]["members"] = [f"{mb.model.n_enc}-{mb.model.n_dec}{'+DLCL' if mb.dlcl else ''}"
                                     f"{f'+RPR{mb.model.rel_k}' if mb.model.rel_k else ''}" for mb in w.members]
        line["config"]["ensemble_rule"] = ["mean log-prob", "log mean prob"][w.ensemble_rule]
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(w, blobs, ids, offs, args.cpu_seconds, args.cpu_procs, args.cpu_full)
    else:
        line["cpu_baseline"] = None
    model.close()
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
