"""Python binding of libdlmc.so: DLM-based lossless compression on MI355X.

Argument marshalling only -- every step of the masked-diffusion pass runs in
the library's HIP kernels and host runtime.  The library is built in-tree by
``paper_2608_11249_amd.build.build()``; importing this module does not need a
GPU, but every call that does GPU work fails loudly when the library is
missing or no GPU is present.  torch is used only to hand device buffers and
streams to the stage hooks.
"""
from __future__ import annotations

import ctypes
import os
import re
from typing import Callable, Optional, Sequence

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libdlmc.so")
HEADER = os.path.join(os.path.dirname(HERE), "include", "dlmc.h")

FFN = {"gelu": 0, "swiglu": 1}
NORM = {"layernorm": 0, "rmsnorm": 1}
DTYPE = {"f32": 0, "bf16": 1}
FLAG_CRC = 1
STAGES = ["embed", "norm", "qkv", "attn", "oproj", "ffn_in", "ffn_out", "head", "entropy",
          "select", "cdf", "reveal", "compact"]
PROFILE_ONE_LAYER = 1 << 31  # DLMC_PROFILE_ONE_LAYER


class LibraryMissing(RuntimeError):
    pass


class DlmcError(RuntimeError):
    def __init__(self, code: int, what: str, detail: str):
        super().__init__(f"dlmc error {code} ({what}): {detail}")
        self.code = code


class ModelConfig(ctypes.Structure):
    _fields_ = [("struct_size", ctypes.c_uint32), ("n_layers", ctypes.c_int32),
                ("d_model", ctypes.c_int32), ("n_heads", ctypes.c_int32),
                ("d_ffn", ctypes.c_int32), ("vocab", ctypes.c_int32),
                ("ffn_kind", ctypes.c_int32), ("norm_kind", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("rope_theta", ctypes.c_float),
                ("norm_eps", ctypes.c_float), ("embed_exp", ctypes.c_int32),
                ("attn_exp", ctypes.c_int32), ("ffn_in_exp", ctypes.c_int32),
                ("ffn_out_exp", ctypes.c_int32), ("head_exp", ctypes.c_int32),
                ("max_chunk", ctypes.c_int32), ("max_batch", ctypes.c_int32)]


class CodecParams(ctypes.Structure):
    _fields_ = [("struct_size", ctypes.c_uint32), ("chunk_len", ctypes.c_int32),
                ("tau_bits", ctypes.c_float), ("m_min", ctypes.c_int32),
                ("m_max", ctypes.c_int32), ("cdf_bits", ctypes.c_int32),
                ("coder_bits", ctypes.c_int32), ("batch", ctypes.c_int32),
                ("flags", ctypes.c_int32), ("schedule", ctypes.c_int32),
                ("blocks", ctypes.c_int32), ("u1", ctypes.c_int32),
                ("growth", ctypes.c_double), ("coder", ctypes.c_int32),
                ("context", ctypes.c_int32), ("context_kind", ctypes.c_int32),
                ("rank_compressor", ctypes.c_int32), ("context_seed", ctypes.c_uint64),
                ("rank_level", ctypes.c_int32), ("reserved", ctypes.c_int32)]


SCHEDULE = {"entropy": 0, "uniform": 1, "progressive": 2}
CODER = {"range": 0, "rans": 1, "rank": 2}
RANK_COMPRESSOR = {"none": 0, "zlib": 1, "lzma": 2, "zstd": 3}
CONTEXT = {"contiguous": 0, "random": 1, "attention": 2}


TRACE_FN = ctypes.CFUNCTYPE(None, ctypes.c_void_p, ctypes.c_int32, ctypes.c_uint64,
                            ctypes.c_int32, ctypes.c_int32, ctypes.POINTER(ctypes.c_int32),
                            ctypes.POINTER(ctypes.c_float), ctypes.POINTER(ctypes.c_uint32),
                            ctypes.c_uint64)

_lib = None
P = ctypes.POINTER
vp, i32, u32, u64, f32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_uint32, ctypes.c_uint64, ctypes.c_float
_SIGS = {
    "dlmc_model_create": (i32, [P(ModelConfig), u64, i32, P(vp)]),
    "dlmc_model_destroy": (None, [vp]),
    "dlmc_set_stream": (i32, [vp, vp]),
    "dlmc_encode_bound": (i32, [vp, P(CodecParams), u64, P(u64)]),
    "dlmc_encode": (i32, [vp, P(CodecParams), vp, u64, vp, u64, P(u64)]),
    "dlmc_decode_size": (i32, [vp, u64, P(u64)]),
    "dlmc_decode": (i32, [vp, vp, u64, i32, vp, u64, P(u64)]),
    "dlmc_encoder_begin": (i32, [vp, P(CodecParams), vp, u64, P(vp)]),
    "dlmc_encoder_step": (i32, [vp, P(i32), P(u64)]),
    "dlmc_encoder_finish": (i32, [vp, vp, u64, P(u64)]),
    "dlmc_session_destroy": (None, [vp]),
    "dlmc_set_trace": (i32, [vp, TRACE_FN, vp]),
    "dlmc_forward_logits": (i32, [vp, vp, i32, i32, vp, vp, vp]),
    "dlmc_entropy_cdf": (i32, [vp, vp, i32, i32, vp, vp, vp, vp]),
    "dlmc_entropy_cdf_noalloc": (i32, [vp, vp, i32, i32, vp, vp, vp, vp]),
    "dlmc_select": (i32, [vp, vp, vp, i32, i32, i32, f32, i32, i32, vp, vp, vp]),
    "dlmc_weight_copy": (i32, [vp, i32, vp, u64]),
    "dlmc_profile_enable": (i32, [vp, ctypes.c_uint32]),
    "dlmc_profile_read": (i32, [vp, i32, P(ctypes.c_double), P(u64), P(ctypes.c_double)]),
    "dlmc_rc_encode": (i32, [vp, vp, u64, i32, i32, vp, u64, P(u64)]),
    "dlmc_rc_decode": (i32, [vp, u64, vp, u64, i32, i32, i32, vp]),
    "dlmc_rans_encode": (i32, [vp, vp, u64, i32, vp, u64, P(u64)]),
    "dlmc_rank_rows": (i32, [vp, vp, i32, vp, vp]),
    "dlmc_context_scores": (i32, [vp, vp, i32, vp]),
    "dlmc_select_rank_rows": (i32, [vp, vp, i32, vp, vp]),
    "dlmc_rans_decode": (i32, [vp, u64, vp, u64, i32, i32, vp]),
    "dlmc_encode_range": (i32, [vp, P(CodecParams), vp, u64, u64, u64, vp, u64, P(u64)]),
    "dlmc_encode_range_bound": (i32, [vp, P(CodecParams), u64, u64, u64, P(u64)]),
    "dlmc_merge": (i32, [P(vp), P(u64), i32, vp, u64, P(u64)]),
    "dlmc_numerics_id": (i32, [P(u64)]),
    "dlmc_test_inject_nonfinite": (i32, [vp, i32]),
    "dlmc_test_head_logits": (i32, [vp, i32]),
    "dlmc_test_gemm_tiles": (i32, [i32, i32, i32, i32, i32, ctypes.POINTER(ctypes.c_int32),
                                   ctypes.POINTER(ctypes.c_int32)]),
    "dlmc_status_string": (ctypes.c_char_p, [i32]),
    "dlmc_last_error": (ctypes.c_char_p, []),
}


def lib():
    """The loaded libdlmc.so (raises LibraryMissing if it was not built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise LibraryMissing(f"{LIB_PATH} is not built; run paper_2608_11249_amd.build.build()")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def header_symbols():
    """Function names declared in include/dlmc.h."""
    txt = open(HEADER).read()
    return sorted(set(re.findall(r"\b(dlmc_[a-z_0-9]+)\s*\(", txt)) - {"dlmc_trace_fn"})


def _check(st: int):
    if st != 0:
        L = lib()
        raise DlmcError(st, L.dlmc_status_string(st).decode(), L.dlmc_last_error().decode())


def _ptr(a) -> int:
    """Address of a numpy array or a torch tensor."""
    if a is None:
        return None
    if isinstance(a, np.ndarray):
        return a.ctypes.data
    return a.data_ptr()


def model_config(shape, max_chunk: int, max_batch: int) -> ModelConfig:
    return ModelConfig(ctypes.sizeof(ModelConfig), shape.n_layers, shape.d_model, shape.n_heads,
                       shape.d_ffn, shape.vocab, FFN[shape.ffn], NORM[shape.norm], DTYPE[shape.dtype],
                       shape.rope_theta, shape.norm_eps, shape.embed_exp, shape.attn_exp,
                       shape.ffn_in_exp, shape.ffn_out_exp, shape.head_exp, max_chunk, max_batch)


def codec_params(codec, batch: Optional[int] = None, crc: bool = False) -> CodecParams:
    return CodecParams(ctypes.sizeof(CodecParams), codec.chunk_len, codec.tau_bits, codec.m_min,
                       codec.m_max, codec.cdf_bits, codec.coder_bits,
                       codec.batch if batch is None else batch, FLAG_CRC if crc else 0,
                       SCHEDULE[codec.schedule], codec.blocks, codec.u1, float(codec.growth),
                       CODER[codec.coder], codec.context, CONTEXT[codec.context_kind],
                       RANK_COMPRESSOR[codec.rank_compressor], codec.context_seed,
                       codec.rank_level, 0)


class Encoder:
    """Streaming encoder: ``step()`` runs exactly one masked-diffusion pass."""

    def __init__(self, model: "Model", codec, tokens: np.ndarray, batch=None, crc=False):
        self.model = model
        self._tok = np.ascontiguousarray(tokens, dtype=np.int32)
        self._cp = codec_params(codec, batch, crc)
        h = vp()
        _check(lib().dlmc_encoder_begin(model.handle, ctypes.byref(self._cp), _ptr(self._tok),
                                        len(self._tok), ctypes.byref(h)))
        self.handle = h
        self.coded = 0
        self.done = False

    def step(self) -> bool:
        done, coded = i32(0), u64(0)
        _check(lib().dlmc_encoder_step(self.handle, ctypes.byref(done), ctypes.byref(coded)))
        self.coded += coded.value
        self.done = bool(done.value)
        return self.done

    def finish(self) -> bytes:
        bound = self.model.encode_bound(self._cp, len(self._tok))
        out = np.empty(bound, dtype=np.uint8)
        n = u64(0)
        _check(lib().dlmc_encoder_finish(self.handle, _ptr(out), bound, ctypes.byref(n)))
        return out[: n.value].tobytes()

    def close(self):
        if self.handle:
            lib().dlmc_session_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Model:
    """A masked diffusion LM with seeded random weights on one GPU."""

    def __init__(self, shape, max_chunk: int, max_batch: int = 1, device: int = 0):
        self.shape = shape
        self.cfg = model_config(shape, max_chunk, max_batch)
        h = vp()
        _check(lib().dlmc_model_create(ctypes.byref(self.cfg), shape.seed, device, ctypes.byref(h)))
        self.handle = h
        self._trace_cb = None

    def close(self):
        if getattr(self, "handle", None):
            lib().dlmc_model_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *a):
        self.close()

    # ---- compression
    def encode_bound(self, cp: CodecParams, n: int) -> int:
        out = u64(0)
        _check(lib().dlmc_encode_bound(self.handle, ctypes.byref(cp), n, ctypes.byref(out)))
        return out.value

    def encode(self, tokens, codec, batch=None, crc=False) -> bytes:
        tok = np.ascontiguousarray(tokens, dtype=np.int32)
        cp = codec_params(codec, batch, crc)
        bound = self.encode_bound(cp, len(tok))
        out = np.empty(max(bound, 1), dtype=np.uint8)
        n = u64(0)
        _check(lib().dlmc_encode(self.handle, ctypes.byref(cp), _ptr(tok), len(tok), _ptr(out),
                                 bound, ctypes.byref(n)))
        return out[: n.value].tobytes()

    def encode_range(self, tokens, codec, first_chunk: int, n_chunks: int, batch=None,
                     crc=False) -> bytes:
        """A partial container of chunks [first_chunk, first_chunk + n_chunks)."""
        tok = np.ascontiguousarray(tokens, dtype=np.int32)
        cp = codec_params(codec, batch, crc)
        bound = u64(0)
        _check(lib().dlmc_encode_range_bound(self.handle, ctypes.byref(cp), len(tok), first_chunk,
                                             n_chunks, ctypes.byref(bound)))
        out = np.empty(max(bound.value, 1), dtype=np.uint8)
        n = u64(0)
        _check(lib().dlmc_encode_range(self.handle, ctypes.byref(cp), _ptr(tok), len(tok),
                                       first_chunk, n_chunks, _ptr(out), bound.value,
                                       ctypes.byref(n)))
        return out[: n.value].tobytes()

    def inject_nonfinite(self, on: bool):
        """Test hook: every forward writes a NaN into its first logit while on."""
        _check(lib().dlmc_test_inject_nonfinite(self.handle, 1 if on else 0))

    def head_logits_mode(self, mode: int):
        """Test hook: 0 deferred logits chosen by cost, 1 always, 2 never."""
        _check(lib().dlmc_test_head_logits(self.handle, int(mode)))

    def decode(self, data: bytes, batch: int = 0) -> np.ndarray:
        buf = np.frombuffer(data, dtype=np.uint8).copy()
        n = decode_size(data)
        out = np.empty(max(n, 1), dtype=np.int32)
        got = u64(0)
        _check(lib().dlmc_decode(self.handle, _ptr(buf), len(buf), batch, _ptr(out), n,
                                 ctypes.byref(got)))
        return out[: got.value]

    def encoder(self, codec, tokens, batch=None, crc=False) -> Encoder:
        return Encoder(self, codec, tokens, batch, crc)

    def set_trace(self, fn: Optional[Callable], coded: bool = False):
        """fn(dir, chunk, pass, positions: list, entropies: list, cdf_hash) or
        None; with coded=True fn(dir, chunk, pass, positions, entropies,
        coded_pairs: list of (start, freq) / (rank, symbol), cdf_hash)."""
        if fn is None:
            self._trace_cb = None
            _check(lib().dlmc_set_trace(self.handle, TRACE_FN(), None))
            return

        def cb(_user, d, chunk, pas, n, pos, ent, iv, hsh):
            p = [pos[i] for i in range(n)]
            e = [ent[i] for i in range(n)]
            if coded:
                fn(int(d), int(chunk), int(pas), p, e,
                   [(int(iv[2 * i]), int(iv[2 * i + 1])) for i in range(n)], int(hsh))
            else:
                fn(int(d), int(chunk), int(pas), p, e, int(hsh))

        self._trace_cb = TRACE_FN(cb)
        _check(lib().dlmc_set_trace(self.handle, self._trace_cb, None))

    def profile(self, on: bool = True, stages: Optional[Sequence[str]] = None,
                one_layer: bool = False):
        """Enable (all stages, or the named ones) / disable per-stage event
        timing; every call resets the counters.  one_layer: time the per-layer
        stages in one layer per forward pass (rotating), not in every layer."""
        if not on:
            mask = 0
        elif stages is None:
            mask = (1 << len(STAGES)) - 1
        else:
            mask = 0
            for name in stages:
                mask |= 1 << STAGES.index(name)
        if on and one_layer:
            mask |= PROFILE_ONE_LAYER
        _check(lib().dlmc_profile_enable(self.handle, mask))

    def profile_read(self) -> dict:
        """{stage: (ms_total, launches, work)} since profiling was enabled."""
        out = {}
        for i, name in enumerate(STAGES):
            ms, n, wk = ctypes.c_double(0), u64(0), ctypes.c_double(0)
            _check(lib().dlmc_profile_read(self.handle, i, ctypes.byref(ms), ctypes.byref(n),
                                           ctypes.byref(wk)))
            out[name] = (ms.value, n.value, wk.value)
        return out

    def set_stream(self, stream_handle: Optional[int]):
        _check(lib().dlmc_set_stream(self.handle, stream_handle))

    # ---- stage hooks on torch device tensors
    def forward_logits(self, state):
        """state: int32 cuda tensor [B, T].  Returns (logits [n, V], rows [n])."""
        import torch
        B, T = state.shape
        V = self.shape.vocab
        logits = torch.empty(B * T * V, dtype=torch.float32, device=state.device)
        rows = torch.empty(B * T, dtype=torch.int32, device=state.device)
        n = torch.zeros(1, dtype=torch.int32, device=state.device)
        self.set_stream(torch.cuda.current_stream(state.device).cuda_stream)
        _check(lib().dlmc_forward_logits(self.handle, _ptr(state.contiguous()), B, T, _ptr(logits),
                                         _ptr(rows), _ptr(n)))
        k = int(n.item())
        return logits[: k * V].view(k, V), rows[:k]

    def entropy_cdf(self, logits, cdf_bits: int, want_cdf: bool = True):
        """Per row of logits [n, V]: (H bits, max, g, cdf) (g, cdf None if not wanted)."""
        import torch
        n, V = logits.shape
        dev = logits.device
        H = torch.empty(n, dtype=torch.float32, device=dev)
        mx = torch.empty(n, dtype=torch.float32, device=dev)
        g = cdf = None
        if want_cdf:
            g = torch.empty(n * V, dtype=torch.int32, device=dev)
            cdf = torch.empty(n * (V + 1), dtype=torch.int32, device=dev)
        self.set_stream(torch.cuda.current_stream(dev).cuda_stream)
        _check(lib().dlmc_entropy_cdf(self.handle, _ptr(logits.contiguous()), n, cdf_bits, _ptr(H),
                                      _ptr(mx), _ptr(g), _ptr(cdf)))
        if want_cdf:
            g, cdf = g.view(n, V), cdf.view(n, V + 1)
        return H, mx, g, cdf


    def entropy_cdf_noalloc(self, logits, cdf_bits: int, want_cdf: bool = True):
        """entropy_cdf through the allocation-free entry point (the library's
        static scratch); the outputs are torch tensors allocated here."""
        import torch
        n, V = logits.shape
        dev = logits.device
        H = torch.empty(n, dtype=torch.float32, device=dev)
        mx = torch.empty(n, dtype=torch.float32, device=dev)
        g = cdf = None
        if want_cdf:
            g = torch.empty(n * V, dtype=torch.int32, device=dev)
            cdf = torch.empty(n * (V + 1), dtype=torch.int32, device=dev)
        self.set_stream(torch.cuda.current_stream(dev).cuda_stream)
        _check(lib().dlmc_entropy_cdf_noalloc(self.handle, _ptr(logits.contiguous()), n, cdf_bits,
                                              _ptr(H), _ptr(mx), _ptr(g), _ptr(cdf)))
        if want_cdf:
            g, cdf = g.view(n, V), cdf.view(n, V + 1)
        return H, mx, g, cdf

    def context_scores(self, tokens) -> np.ndarray:
        """Attention-based context score of every position of one chunk."""
        t = np.ascontiguousarray(tokens, dtype=np.int32)
        out = np.empty(len(t), dtype=np.float32)
        _check(lib().dlmc_context_scores(self.handle, _ptr(t), len(t), _ptr(out)))
        return out

    def rank_rows(self, logits, sym):
        """Ranks of sym[i] in device logits row i (torch tensors on cuda)."""
        import torch
        n = int(sym.shape[0])
        out = torch.empty(n, dtype=torch.int32, device=logits.device)
        self.set_stream(torch.cuda.current_stream(logits.device).cuda_stream)
        _check(lib().dlmc_rank_rows(self.handle, _ptr(logits.contiguous()), n,
                                    _ptr(sym.contiguous()), _ptr(out)))
        return out

    def select_rank_rows(self, logits, rank):
        """The symbol of rank[i] in device logits row i."""
        import torch
        n = int(rank.shape[0])
        out = torch.empty(n, dtype=torch.int32, device=logits.device)
        self.set_stream(torch.cuda.current_stream(logits.device).cuda_stream)
        _check(lib().dlmc_select_rank_rows(self.handle, _ptr(logits.contiguous()), n,
                                           _ptr(rank.contiguous()), _ptr(out)))
        return out
    def select(self, H, rows, B: int, T: int, tau: float, m_min: int, m_max: int):
        """Schedule on device entropies; returns (sel_pos [B, m_max], sel_row, n_sel [B])."""
        import torch
        dev = H.device
        sel_pos = torch.full((B, m_max), -1, dtype=torch.int32, device=dev)
        sel_row = torch.full((B, m_max), -1, dtype=torch.int32, device=dev)
        n_sel = torch.zeros(B, dtype=torch.int32, device=dev)
        self.set_stream(torch.cuda.current_stream(dev).cuda_stream)
        _check(lib().dlmc_select(self.handle, _ptr(H.contiguous()), _ptr(rows.contiguous()),
                                 int(rows.numel()), B, T, tau, m_min, m_max, _ptr(sel_pos),
                                 _ptr(sel_row), _ptr(n_sel)))
        return sel_pos, sel_row, n_sel

    def weight(self, tensor_id: int, rows: int, cols: int) -> np.ndarray:
        """A weight tensor in canonical [out, in] layout (uint16 bf16 bits or float32)."""
        dt = np.uint16 if self.shape.dtype == "bf16" else np.float32
        out = np.empty((rows, cols), dtype=dt)
        _check(lib().dlmc_weight_copy(self.handle, tensor_id, _ptr(out), out.nbytes))
        return out


GEMM_EPI = {"store": 0, "residual": 1, "qkv": 2, "gelu": 3, "swiglu": 4}


def gemm_tiles(M: int, N: int, K: int, epi: str, d_model: int = 0):
    """(kind, split) the bf16 GEMM chooses (host only): kind "128x128",
    "192x128" or "4wave" with columns [0, split) on 256 x 256 tiles."""
    kind, split = ctypes.c_int32(), ctypes.c_int32()
    _check(lib().dlmc_test_gemm_tiles(M, N, K, GEMM_EPI[epi], d_model, ctypes.byref(kind),
                                      ctypes.byref(split)))
    return ("128x128", "192x128", "4wave")[kind.value], split.value


def decode_size(data: bytes) -> int:
    buf = np.frombuffer(data, dtype=np.uint8)
    n = u64(0)
    _check(lib().dlmc_decode_size(_ptr(buf) if len(buf) else None, len(buf), ctypes.byref(n)))
    return n.value


def merge(parts: Sequence[bytes]) -> bytes:
    """One complete container from partial containers of the same input."""
    bufs = [np.frombuffer(p, dtype=np.uint8).copy() for p in parts]
    ptrs = (vp * len(bufs))(*[b.ctypes.data if len(b) else None for b in bufs])
    lens = (u64 * len(bufs))(*[len(b) for b in bufs])
    n = u64(0)
    L = lib()
    st = L.dlmc_merge(ptrs, lens, len(bufs), None, 0, ctypes.byref(n))
    if st != -6:
        _check(st)
    out = np.empty(max(n.value, 1), dtype=np.uint8)
    _check(L.dlmc_merge(ptrs, lens, len(bufs), _ptr(out), n.value, ctypes.byref(n)))
    return out[: n.value].tobytes()


def numerics_id() -> int:
    """This build's numerics identity (recorded in every container)."""
    out = u64(0)
    _check(lib().dlmc_numerics_id(ctypes.byref(out)))
    return out.value


def rc_encode(start, freq, cdf_bits: int, coder_bits: int) -> bytes:
    s = np.ascontiguousarray(start, dtype=np.uint32)
    f = np.ascontiguousarray(freq, dtype=np.uint32)
    cap = len(s) * 8 + 64
    out = np.empty(cap, dtype=np.uint8)
    n = u64(0)
    _check(lib().dlmc_rc_encode(_ptr(s), _ptr(f), len(s), cdf_bits, coder_bits, _ptr(out), cap,
                                ctypes.byref(n)))
    return out[: n.value].tobytes()


def rc_decode(data: bytes, cdfs: np.ndarray, cdf_bits: int, coder_bits: int) -> np.ndarray:
    c = np.ascontiguousarray(cdfs, dtype=np.uint32)
    n, V1 = c.shape
    buf = np.frombuffer(data, dtype=np.uint8).copy()
    out = np.empty(max(n, 1), dtype=np.int32)
    _check(lib().dlmc_rc_decode(_ptr(buf), len(buf), _ptr(c), n, V1 - 1, cdf_bits, coder_bits,
                                _ptr(out)))
    return out[:n]


def rans_encode(start, freq, cdf_bits: int) -> bytes:
    s = np.ascontiguousarray(start, dtype=np.uint32)
    f = np.ascontiguousarray(freq, dtype=np.uint32)
    cap = len(s) * 4 + 16
    out = np.empty(cap, dtype=np.uint8)
    n = u64(0)
    _check(lib().dlmc_rans_encode(_ptr(s), _ptr(f), len(s), cdf_bits, _ptr(out), cap,
                                  ctypes.byref(n)))
    return out[: n.value].tobytes()


def rans_decode(data: bytes, cdfs: np.ndarray, cdf_bits: int) -> np.ndarray:
    c = np.ascontiguousarray(cdfs, dtype=np.uint32)
    n, V1 = c.shape
    buf = np.frombuffer(data, dtype=np.uint8).copy()
    out = np.empty(max(n, 1), dtype=np.int32)
    _check(lib().dlmc_rans_decode(_ptr(buf) if len(buf) else None, len(buf), _ptr(c), n, V1 - 1,
                                  cdf_bits, _ptr(out)))
    return out[:n]
