"""Shared helpers of the GPU parity tests (imported by tests only)."""
import dataclasses
import math
import sys

import numpy as np

import workloads as wl


def log(*a):
    """Name the case before each GPU step, flushed, so a failing run says which."""
    print("[gpu-case]", *a, flush=True)
    sys.stdout.flush()


def shape(**kw):
    """A small model shape; weight-scale exponents follow d_model / d_ffn."""
    d = kw.get("d_model", 128)
    F = kw.get("d_ffn", 256)
    base = dict(name="t", n_layers=2, d_model=d, n_heads=2, d_ffn=F, vocab=500,
                ffn="gelu", norm="layernorm", dtype="bf16", embed_exp=0,
                attn_exp=wl.fan_in_exp(d), ffn_in_exp=wl.fan_in_exp(d),
                ffn_out_exp=wl.fan_in_exp(F), head_exp=wl.fan_in_exp(d), seed=3)
    base.update(kw)
    return wl.ModelShape(**base)


def codec(chunk, k=None, tau=float("-inf"), mmin=None, mmax=None, P=16, W=32, batch=1, **kw):
    if k is not None:
        mmin = mmax = k
    return wl.CodecParams(chunk, tau, mmin, mmax, P, W, batch, **kw)


def rel_err_rows(gpu, ref):
    """Per row max |gpu - ref| / max |ref|, maximised over rows."""
    num = np.abs(gpu - ref).max(axis=1)
    den = np.abs(ref).max(axis=1)
    return float((num / den).max())


FIXED_HEADER = 144  # container version 3


def payloads(container: bytes):
    """Per-chunk payloads held by a dlmc container (layout of include/dlmc.h)."""
    hdr = int.from_bytes(container[8:12], "little")
    nc = int.from_bytes(container[136:144], "little")
    offs = [int.from_bytes(container[FIXED_HEADER + 8 * c: FIXED_HEADER + 8 + 8 * c], "little")
            for c in range(nc + 1)]
    return [container[hdr + offs[c]: hdr + offs[c + 1]] for c in range(nc)]
