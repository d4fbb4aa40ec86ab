#!/usr/bin/env python
"""Throughput of DLM-based lossless compression on one MI355X.

A step is one masked-diffusion encode pass over one batch of chunks: the
bidirectional transformer forward over every position, entropy of every
masked position, the commitment schedule, integer CDFs of the committed
positions, range coding on the host and the reveal.  The default workload is
the 8B-shaped model (32 layers, d=4096, 32 heads, SwiGLU 12288, vocab 126464)
on 2048-token chunks with k=16 positions per pass; the input is a seeded
synthetic order-1 Zipf/Markov token stream (u32 tokens) standing in for the
paper's tokenised enwik8, and the weights are seeded random.

value = input bytes encoded per second over the timed steps (tokens are
resident in HBM before timing starts).  roofline = the dominant kernel's
algorithmic flops per launch / its average HIP-event duration in the timed
region, against the bf16 dense MFMA peak.  cpu_baseline = the fp64 CPU oracle
on a bounded sample of one pass, extrapolated to the same unit.
"""
import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_FP32_TFLOPS = 157.3    # MI355X fp32 vector
PEAK_HBM_GBS = 8000.0


def needed_tokens(w, steps):
    cd = w.codec
    T, B = cd.chunk_len, cd.batch
    min_passes = math.ceil(T / cd.m_max)          # a chunk lasts at least this many passes
    chunks = B * (math.ceil(steps / min_passes) + 1)
    return min(w.n_tokens, chunks * T)


def cpu_baseline(w, layers_timed=1, vocab_sample=4096):
    """Time the oracle on one pass of one chunk with half its positions masked:
    `layers_timed` of the model's layers at full width (x n_layers), the LM head
    against a `vocab_sample`-row slice of the head (x vocab / sample), entropy
    of the masked rows, selection, and k full-vocabulary CDF rows."""
    import numpy as np
    from threadpoolctl import threadpool_info

    import workloads as wl
    from oracle import cdf as OC
    from oracle import model as OM
    from oracle import schedule as OS
    from oracle import weights as OW

    sh, cd = w.model, w.codec
    T, V, k = cd.chunk_len, sh.vocab, cd.m_max
    W = OW.Weights(sh)
    st = np.full(T, sh.mask_id)
    st[::2] = wl.make_tokens(w, T)[::2]
    x = W.embed_rows(st)
    cos, sin = OM.rope_cos_sin(T, sh.d_head, sh.rope_theta)
    lw = [W.layer(l) for l in range(layers_timed)]           # generation is not timed
    vs = min(V, vocab_sample)
    head = W.head_rows(np.arange(vs))
    full_row = wl.random_logits(1, 1, V, 8.0)[0].astype(np.float64)

    t0 = time.perf_counter()
    for l in range(layers_timed):
        x = OM.block(sh, lw[l], x, cos, sin)
    t_layers = (time.perf_counter() - t0) / layers_timed
    t0 = time.perf_counter()
    pos = OM.masked_positions(sh, st)
    h = OM.norm(sh, x)[pos]
    lg = h @ head.T
    H = OS.entropy_bits(lg)
    t_head = (time.perf_counter() - t0) * V / vs
    t0 = time.perf_counter()
    OS.select(H, pos, cd.tau_bits, cd.m_min, cd.m_max)
    for _ in range(k):
        OC.cdf_row(full_row, cd.cdf_bits)
    t_rest = time.perf_counter() - t0
    t_pass = sh.n_layers * t_layers + t_head + t_rest
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    return {
        "value": k * w.token_bytes / t_pass,
        "unit": "B/s",
        "cores": threads,              # BLAS threads the oracle ran on
        "host_cpus": os.cpu_count(),   # logical CPUs of the host
        "kind": "oracle",
        "sample": (f"one pass of one {T}-token chunk, {T // 2} masked: {layers_timed} of "
                   f"{sh.n_layers} layers timed (x{sh.n_layers}), LM head on a {vs}-row vocab "
                   f"slice (x{V / vs:.1f}), entropy, selection, {k} CDF rows; "
                   f"fp64 NumPy, extrapolated pass time {t_pass:.1f} s"),
    }


def roundtrip_leg(model, w):
    """One batch of whole chunks encoded into a container (one streaming
    encoder step per pass), then decoded, each timed end to end (host tokens
    in, host bytes out): decode throughput, bits per input byte and the pass
    count, which the timed encode passes cannot give."""
    import numpy as np
    import torch

    import workloads as wl
    cd = w.codec
    toks = wl.make_tokens(w, cd.batch * cd.chunk_len)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    enc = model.encoder(cd, toks)
    passes = 0
    try:
        while not enc.step():
            passes += 1
        passes += 1
        data = enc.finish()
    finally:
        enc.close()
    t1 = time.perf_counter()
    print(f"roundtrip: encoded {len(toks)} tokens in {passes} passes, {t1 - t0:.1f} s",
          file=sys.stderr, flush=True)
    back = model.decode(data)
    t2 = time.perf_counter()
    print(f"roundtrip: decoded in {t2 - t1:.1f} s", file=sys.stderr, flush=True)
    if not np.array_equal(back, toks):
        raise RuntimeError("round trip mismatch")
    nb = len(toks) * w.token_bytes
    return {
        "tokens": int(len(toks)),
        "container_bytes": len(data),
        "bits_per_input_byte": round(8.0 * len(data) / nb, 4),
        # passes of the batch: every chunk starts at pass 0, so this is the
        # largest pass count of its chunks (all equal under a fixed k)
        "passes": passes,
        "encode_s": round(t1 - t0, 3),
        "decode_s": round(t2 - t1, 3),
        "encode_bytes_per_s": round(nb / (t1 - t0), 1),
        "decode_bytes_per_s": round(nb / (t2 - t1), 1),
        "note": "random-init weights: the ratio exercises the coder only",
    }


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "ffn_in_gemm_8b_traffic.md")
GEMM_SOURCE = os.path.join(ROOT, "paper_2608_11249_amd", "csrc", "gemm_bf16.hip")


def code_hash(path):
    """sha256[:16] of a C++ source with its // comments, trailing blanks and
    empty lines removed: the code the counters were taken on, so that an edit
    to comments alone keeps a summary valid."""
    import hashlib
    lines = []
    for line in open(path, encoding="utf-8"):
        line = line.split("//", 1)[0].rstrip()
        if line:
            lines.append(line)
    return hashlib.sha256("\n".join(lines).encode()).hexdigest()[:16]


def gemm_source_hash():
    return code_hash(GEMM_SOURCE)


def measured_traffic():
    """HBM bytes per launch of the FFN-in GEMM from the committed rocprofv3
    FETCH_SIZE / WRITE_SIZE summary, if it was taken on the current source."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    vals = {}
    for line in open(TRAFFIC_FILE):
        if ": " in line and line.startswith("- "):
            k, v = line[2:].split(": ", 1)
            vals[k.strip()] = v.strip().strip("`")
    if vals.get("gemm_bf16.hip code sha256[:16]") != gemm_source_hash():
        return None
    try:
        return float(vals["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def copy_calibration(nbytes):
    """A plain device-to-device copy of known size, run under rocprofv3 --pmc to
    scale FETCH_SIZE / WRITE_SIZE into bytes."""
    import torch
    x = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
    y = torch.empty_like(x)
    for _ in range(3):
        y.copy_(x)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": nbytes, "dispatches": 3}), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    # 128 passes = one chunk's worth at k = 16 (2048 / 16): with the warmup
    # passes, the timed passes see every masked-row count of a chunk once
    ap.add_argument("--steps", type=int, default=128)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="8b",
                    choices=["tiny", "small", "8b", "8b-throughput", "8b-long"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--profile-all", action="store_true",
                    help="time every stage inside the timed region (adds event overhead)")
    ap.add_argument("--no-decode", action="store_true",
                    help="skip the whole-chunk encode + decode leg (detail.roundtrip)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                    help="only run a plain device copy of BYTES (counter calibration)")
    args = ap.parse_args()
    if args.copy_calibration:
        copy_calibration(args.copy_calibration)
        return
    if args.gpus != 1:
        print("bench.py runs on one GPU only: chunks are independent, so several GPUs "
              "would each encode their own range of chunks; --gpus must be 1", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2608_11249_amd as dl
    import workloads as wl

    w = wl.WORKLOADS[args.workload]
    sh, cd = w.model, w.codec
    warmup = max(args.warmup, 1)
    toks = wl.make_tokens(w, needed_tokens(w, warmup + args.steps))
    torch.cuda.init()
    model = dl.Model(sh, max_chunk=cd.chunk_len, max_batch=cd.batch)
    enc = model.encoder(cd, toks)
    gemm_stages = ["qkv", "attn", "oproj", "ffn_in", "ffn_out", "head"]
    layer_stages = ["qkv", "attn", "oproj", "ffn_in", "ffn_out"]
    for _ in range(warmup - 1):
        enc.step()
    # the last warmup pass times every stage (per-stage breakdown, dominant kernel)
    model.profile(True)
    enc.step()
    prof_all = model.profile_read()
    dom = max(gemm_stages, key=lambda s: prof_all[s][0])
    # the timed passes carry events around the dominant stage (in one layer per
    # pass, rotating through the layers) and the LM head only
    model.profile(True, stages=None if args.profile_all else sorted({dom, "head"}),
                  one_layer=not args.profile_all)
    torch.cuda.synchronize()
    c0 = enc.coded
    t0 = time.perf_counter()
    steps = 0
    for _ in range(args.steps):
        done = enc.step()
        steps += 1
        if done:
            break
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    prof = model.profile_read()
    model.profile(False)
    coded = enc.coded - c0

    bf16 = sh.dtype == "bf16"
    ms, n, work = prof[dom]
    achieved = (work / n) / (ms / n * 1e-3) / 1e12
    peak = PEAK_BF16_TFLOPS if bf16 else PEAK_FP32_TFLOPS
    # flops of the timed passes: the layer stages do the same work every pass;
    # the head's work (masked rows only) was accumulated over the timed passes
    step_flops = sum(prof_all[s][2] for s in layer_stages) + prof["head"][2] / steps
    stages_ms = {s: round(v[0], 3) for s, v in prof_all.items() if v[1]}
    out = {
        "metric": "input bytes/s encoded per MI355X (8B-shaped DLM)",
        "value": coded * w.token_bytes / elapsed,
        "unit": "B/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": elapsed / steps * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": sh.dtype,
        "data": "synthetic (seeded order-1 Zipf/Markov token stream; seeded random weights)",
        "config": {
            "workload": f"{w.name}: L={sh.n_layers} d={sh.d_model} heads={sh.n_heads} "
                        f"ffn={sh.d_ffn} {sh.ffn} vocab={sh.vocab}, chunk {cd.chunk_len} x "
                        f"batch {cd.batch}, {'k=%d' % cd.m_max if cd.m_min == cd.m_max else 'H<=%.2g bits, %d..%d' % (cd.tau_bits, cd.m_min, cd.m_max)} per pass",
            "token_bytes": w.token_bytes,
            "cdf_bits": cd.cdf_bits,
            "coder_bits": cd.coder_bits,
        },
        "roofline": {
            "bound": "mfma" if bf16 else "alu",
            "kernel": f"{dom} GEMM" if dom != "attn" else "attention",
            "achieved": round(achieved, 1),
            "peak": peak,
            "unit": "TFLOP/s",
            "frac": round(achieved / peak, 4),
            "traffic": measured_traffic() if (dom == "ffn_in" and args.workload == "8b") else None,
            # the whole step: the algorithmic flops of one pass (every layer
            # GEMM and attention, the LM head at the masked rows, averaged over
            # the timed passes) over the measured time per step
            "step": {
                "flops_per_step": step_flops,
                "achieved": round(step_flops / (elapsed / steps) / 1e12, 1),
                "frac": round(step_flops / (elapsed / steps) / 1e12 / peak, 4),
            },
        },
        "detail": {
            "tokens_per_s": coded / elapsed,
            "forward_tokens_per_s": steps * cd.batch * cd.chunk_len / elapsed,
            "step_tflops": round(step_flops / (elapsed / steps) / 1e12, 1),
            "step_mfma_frac": round(step_flops / (elapsed / steps) / 1e12 / peak, 4),
            "stage_ms_one_profiled_pass": stages_ms,
        },
    }
    if not args.no_decode:
        out["detail"]["roundtrip"] = roundtrip_leg(model, w)
    model.close()
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
