"""ctypes binding of libspecdec.so (include/spec.h).

Argument marshalling only: every step of the speculative path runs in the HIP
library.  Functions keep the C names and raise `SpecError` on a non-zero
status.  Device buffers are passed as integer addresses (e.g. a torch tensor's
data_ptr()); the stream as an integer hipStream_t (e.g. torch's
cuda_stream).  There is no CPU fallback: without the built library every call
raises.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, Structure, c_char_p, c_double, c_float, c_int32, c_int64, c_size_t, c_void_p

_HERE = os.path.dirname(os.path.abspath(__file__))
# SPECDEC_LIBRARY: another build of the same library (the host-sanitizer
# build of the ABI tests); by default the in-tree build.
LIB_PATH = os.environ.get("SPECDEC_LIBRARY") or os.path.join(_HERE, "libspecdec.so")

SPEC_MAX_K = 16
SPEC_MAX_BATCH = 16
SPEC_MAX_ROWS = 160
SPEC_KV_PAGE = 64
SPEC_SCRATCH_BYTES = 32 << 20
SPEC_FLAG_NO_GRAPHS = 1
SPEC_FLAG_ROWMAJOR = 8
SPEC_FLAG_DRAFT_MROPE = 16
SPEC_FLAG_BLOCK_DRAFT = 32
SPEC_FLAG_COND = 64
SPEC_FLAG_FULL_DRAFT_ROWS = 128
SPEC_FLAG_COND_CROSS = 256
STATUS = {0: "SPEC_OK", 1: "SPEC_E_INVAL", 2: "SPEC_E_STATE", 3: "SPEC_E_CAPACITY", 5: "SPEC_E_HIP",
          6: "SPEC_E_NUMERIC"}
KERNEL_KINDS = {"qkv": 0, "o": 1, "gateup": 2, "down": 3, "lmhead": 4, "attn": 5, "other": 6}


class spec_dims(Structure):
    _fields_ = [("layers", c_int32), ("hidden", c_int32), ("q_heads", c_int32), ("kv_heads", c_int32),
                ("head_dim", c_int32), ("ffn", c_int32), ("mrope_section", c_int32 * 3),
                ("interleaved", c_int32), ("rope_base", c_float), ("rms_eps", c_float)]


class spec_config(Structure):
    _fields_ = [("target", spec_dims), ("draft", spec_dims), ("vocab", c_int32), ("K", c_int32),
                ("batch", c_int32), ("max_new_tokens", c_int32), ("stop_token", c_int32), ("flags", c_int32),
                ("mask_token", c_int32), ("cond_layers", c_int32 * 3)]


class spec_layer_weights(Structure):
    _fields_ = [(n, c_void_p) for n in ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "w_gate", "w_up",
                                        "w_down")]


class spec_model_weights(Structure):
    _fields_ = [("layers", POINTER(spec_layer_weights)), ("final_norm", c_void_p), ("w_fuse", c_void_p),
                ("w_in", c_void_p)]


class spec_vision_block(Structure):
    _fields_ = [("start", c_int32), ("t", c_int32), ("h", c_int32), ("w", c_int32)]


class spec_seq_init(Structure):
    _fields_ = [("prefix_len", c_int32), ("n_blocks", c_int32), ("blocks", POINTER(spec_vision_block)),
                ("pending_token", c_int32), ("tgt_k", POINTER(c_void_p)), ("tgt_v", POINTER(c_void_p)),
                ("drf_k", POINTER(c_void_p)), ("drf_v", POINTER(c_void_p)), ("page_table", POINTER(c_int32))]


class SpecError(RuntimeError):
    def __init__(self, status: int, func: str, msg: str):
        self.status = status
        super().__init__(f"{func}: {STATUS.get(status, status)}: {msg}")


_lib = None


def lib():
    """Load libspecdec.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
        L = ctypes.CDLL(LIB_PATH)
        P = c_void_p
        sig = {
            "spec_workspace_bytes": [POINTER(spec_config), POINTER(spec_seq_init), POINTER(c_size_t)],
            "spec_init": [POINTER(spec_config), P, POINTER(spec_model_weights), POINTER(spec_model_weights),
                          POINTER(spec_seq_init), P, c_size_t, P, POINTER(P)],
            "draft_step": [P, P],
            "draft_steps": [P, c_int32, P],
            "spec_verify": [P, P, P],
            "spec_verify_scratch": [P, P, P],
            "spec_commit": [P, P, P, P, P],
            "spec_attn_readout": [P, c_int32, c_int32, P],
            "spec_sync": [P, POINTER(c_int32)],
            "spec_debug_positions": [P, c_int32, P, c_int32],
            "spec_debug_state": [P, c_int32, P],
            "spec_debug_kv": [P, c_int32, c_int32, c_int32, c_int32, c_int32, c_int32, P],
            "spec_timing": [P, c_int32],
            "spec_stream_read": [P, ctypes.c_size_t, P, c_int32, P],
            "spec_timing_read": [P, c_int32, POINTER(c_int64), POINTER(c_double), POINTER(c_double)],
            "spec_debug_path": [P, POINTER(c_int32)],
            "spec_debug_feature": [P, c_int32, c_int32, c_int32, P],
        }
        for name, args in sig.items():
            f = getattr(L, name)
            f.argtypes = args
            f.restype = c_int32
        L.spec_seq_pages.argtypes = [POINTER(spec_config), POINTER(spec_seq_init)]
        L.spec_seq_pages.restype = c_int32
        L.spec_destroy.argtypes = [P]
        L.spec_destroy.restype = None
        L.spec_last_error.argtypes = [P]
        L.spec_last_error.restype = c_char_p
        _lib = L
    return _lib


def spec_last_error(ctx) -> str:
    s = lib().spec_last_error(ctx)
    return s.decode() if s else ""


def _check(status: int, func: str, ctx=None) -> None:
    if status != 0:
        raise SpecError(status, func, spec_last_error(ctx))


def spec_seq_pages(cfg: spec_config, seq: spec_seq_init) -> int:
    n = lib().spec_seq_pages(ctypes.byref(cfg), ctypes.byref(seq))
    if n < 0:
        raise SpecError(1, "spec_seq_pages", "bad arguments")
    return n


def spec_workspace_bytes(cfg: spec_config, seqs) -> int:
    n = c_size_t(0)
    _check(lib().spec_workspace_bytes(ctypes.byref(cfg), seqs, ctypes.byref(n)), "spec_workspace_bytes")
    return n.value


def spec_init(cfg: spec_config, embed: int, target: spec_model_weights, draft, seqs, workspace: int,
              workspace_bytes: int, stream: int) -> c_void_p:
    ctx = c_void_p()
    st = lib().spec_init(ctypes.byref(cfg), c_void_p(embed), ctypes.byref(target),
                         ctypes.byref(draft) if draft is not None else None, seqs, c_void_p(workspace),
                         workspace_bytes, c_void_p(stream), ctypes.byref(ctx))
    _check(st, "spec_init")
    return ctx


def draft_step(ctx, d_draft_tokens: int = 0) -> None:
    _check(lib().draft_step(ctx, c_void_p(d_draft_tokens or None)), "draft_step", ctx)


def draft_steps(ctx, n: int, d_draft_tokens: int = 0) -> None:
    _check(lib().draft_steps(ctx, n, c_void_p(d_draft_tokens or None)), "draft_steps", ctx)


def spec_verify(ctx, d_draft_tokens: int = 0, d_logits: int = 0) -> None:
    _check(lib().spec_verify(ctx, c_void_p(d_draft_tokens or None), c_void_p(d_logits or None)), "spec_verify", ctx)


def spec_verify_scratch(ctx, d_draft_tokens: int = 0, d_logits: int = 0) -> None:
    _check(lib().spec_verify_scratch(ctx, c_void_p(d_draft_tokens or None), c_void_p(d_logits or None)),
           "spec_verify_scratch", ctx)


def spec_commit(ctx, d_accept_len: int = 0, d_committed: int = 0, d_n_committed: int = 0,
                d_finished: int = 0) -> None:
    _check(lib().spec_commit(ctx, *(c_void_p(p or None) for p in (d_accept_len, d_committed, d_n_committed,
                                                                    d_finished))), "spec_commit", ctx)


def spec_attn_readout(ctx, model: int, layer: int, d_out: int = 0) -> None:
    _check(lib().spec_attn_readout(ctx, model, layer, c_void_p(d_out or None)), "spec_attn_readout", ctx)


def spec_sync(ctx) -> int:
    n = c_int32(0)
    _check(lib().spec_sync(ctx, ctypes.byref(n)), "spec_sync", ctx)
    return n.value


def spec_destroy(ctx) -> None:
    lib().spec_destroy(ctx)


def spec_debug_positions(ctx, b: int, length: int):
    import numpy as np
    out = np.zeros((3, length), dtype=np.int32)
    _check(lib().spec_debug_positions(ctx, b, out.ctypes.data, length), "spec_debug_positions", ctx)
    return out


def spec_debug_state(ctx, b: int) -> dict:
    import numpy as np
    out = np.zeros(8, dtype=np.int32)
    _check(lib().spec_debug_state(ctx, b, out.ctypes.data), "spec_debug_state", ctx)
    keys = ("seq_len", "draft_len", "pending", "n_gen", "finished", "accept_len", "n_commit", "err")
    return {k: int(v) for k, v in zip(keys, out)}


def spec_debug_kv(ctx, b: int, model: int, layer: int, which: int, pos0: int, npos: int, kv_heads: int,
                  head_dim: int):
    """Returns uint16 bfloat16 bits [npos][kv_heads][head_dim]."""
    import numpy as np
    out = np.zeros((npos, kv_heads, head_dim), dtype=np.uint16)
    _check(lib().spec_debug_kv(ctx, b, model, layer, which, pos0, npos, out.ctypes.data), "spec_debug_kv", ctx)
    return out


PATHS = {0: "rowmajor", 1: "packed"}


def spec_debug_feature(ctx, b: int, slot0: int, n: int, hidden: int):
    """Fused target features of slots [slot0, slot0+n) as bf16 bits [n][hidden]."""
    import numpy as np
    out = np.zeros((n, hidden), dtype=np.uint16)
    _check(lib().spec_debug_feature(ctx, b, slot0, n, out.ctypes.data_as(c_void_p)), "spec_debug_feature", ctx)
    return out


def spec_debug_path(ctx) -> str:
    p = c_int32(-1)
    _check(lib().spec_debug_path(ctx, ctypes.byref(p)), "spec_debug_path", ctx)
    return PATHS[p.value]


def spec_stream_read(d_buf: int, nbytes: int, d_sink: int, sink_words: int, stream: int) -> None:
    _check(lib().spec_stream_read(c_void_p(d_buf), nbytes, c_void_p(d_sink), sink_words, c_void_p(stream or None)),
           "spec_stream_read")


def spec_timing(ctx, enable: bool) -> None:
    _check(lib().spec_timing(ctx, 1 if enable else 0), "spec_timing", ctx)


def spec_timing_read(ctx, kind: str):
    n, ms, by = c_int64(0), c_double(0), c_double(0)
    _check(lib().spec_timing_read(ctx, KERNEL_KINDS[kind], ctypes.byref(n), ctypes.byref(ms), ctypes.byref(by)),
           "spec_timing_read", ctx)
    return n.value, ms.value, by.value


def dims(shape, layers=None) -> spec_dims:
    """spec_dims from an object with layers, hidden, q_heads, kv_heads, head_dim,
    ffn, mrope_section, interleaved, rope_base, rms_eps attributes."""
    d = spec_dims()
    if shape is None:
        return d
    d.layers = shape.layers if layers is None else layers
    d.hidden, d.q_heads, d.kv_heads = shape.hidden, shape.q_heads, shape.kv_heads
    d.head_dim, d.ffn = shape.head_dim, shape.ffn
    for i in range(3):
        d.mrope_section[i] = shape.mrope_section[i]
    d.interleaved = 1 if shape.interleaved else 0
    d.rope_base, d.rms_eps = shape.rope_base, shape.rms_eps
    return d
