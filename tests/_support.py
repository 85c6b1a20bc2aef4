"""Shared test helpers: build oracle sequences from a workload, compare tokens
and logits with the tolerances the tests use."""
import numpy as np

import oracle
from oracle import model as OM
from oracle import spec as OS
import workloads as W

# Normwise relative tolerance on logits and on cached K/V values (fp32
# accumulation, bfloat16 storage of activations).
LOGIT_RTOL = 2e-2
# A row's argmax is "pinned" when the oracle's top-1 beats top-2 by more than
# this fraction of |top-1|: then the GPU must pick the same token.
MARGIN = 2e-2


# Session flags selecting the library's execution path (see include/spec.h).
PATH_FLAGS = {"packed": 0, "rowmajor": 8}


def capacity_for(w: W.Workload, b: int) -> int:
    return w.seqs[b].prefix_len + w.max_new_tokens + w.K + 2


def oracle_decoders(w: W.Workload, provider, mirror: bool = False, cache_weights: bool = True,
                    draft_rotary: str = OM.ROTARY_FLAT):
    T = OM.Decoder(provider, "target", w.target, w.vocab, OM.ROTARY_MROPE, mirror=mirror,
                   cache_weights=cache_weights)
    D = None
    if w.draft is not None:
        D = OM.Decoder(provider, "draft", w.draft, w.vocab, draft_rotary, mirror=mirror,
                       cache_weights=cache_weights)
    return T, D


def host_kv(w: W.Workload, b: int, model: str):
    return lambda li: (W.prefix_kv_host(w, b, model, li, "k"), W.prefix_kv_host(w, b, model, li, "v"))


def device_kv(w: W.Workload, b: int, model: str):
    """Prefix K/V drawn on the GPU by the device generator, read back as bf16 bits."""
    import torch

    def bits(t):
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return lambda li: (bits(W.prefix_kv_device(w, b, model, li, "k")),
                       bits(W.prefix_kv_device(w, b, model, li, "v")))


def conditioning(w: W.Workload, provider, layers, mirror: bool = False):
    """The oracle's target-hidden-state conditioning with the workload's seeded
    fusion weights."""
    from oracle import numerics as ON
    return OS.Conditioning(layers, ON.decode(provider.get("draft", -1, "w_fuse")),
                           ON.decode(provider.get("draft", -1, "w_in")), mirror=mirror)


def oracle_sequence(w: W.Workload, b: int, T, D, kv=None, capacity=None, pending=None,
                    with_draft: bool = True, cond=None):
    lay = w.seqs[b]
    cap = capacity or capacity_for(w, b)
    blocks = [(bl.start, bl.t, bl.h, bl.w) for bl in lay.blocks]
    kv = kv or host_kv
    pend = W.first_pending_token(w, b) if pending is None else pending
    dd = D if with_draft else None
    return OS.Sequence(T, dd, lay.prefix_len, blocks, pend, cap, kv(w, b, "target"),
                       kv(w, b, "draft") if dd is not None else None,
                       K=w.K, max_new_tokens=w.max_new_tokens, stop_token=w.stop_token, cond=cond)


def margin(z: np.ndarray) -> np.ndarray:
    """Relative top-1/top-2 gap per row of float logits."""
    s = np.sort(z, axis=-1)
    return (s[..., -1] - s[..., -2]) / np.abs(s[..., -1])


def normwise_err(a: np.ndarray, ref: np.ndarray) -> float:
    """max |a - ref| / max |ref| over the whole array."""
    a = np.asarray(a, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    return float(np.max(np.abs(a - ref)) / max(np.max(np.abs(ref)), 1e-30))


def check_argmax_rows(gpu_tokens, oracle_logits, tol: float = MARGIN):
    """Every GPU argmax must be the oracle argmax on pinned rows, and within
    `tol` (relative to |top-1|) of the oracle's top-1 on unpinned rows.
    Returns the boolean pinned mask."""
    z = np.asarray(oracle_logits, dtype=np.float64)
    ref = OM.greedy_argmax(z)
    pinned = margin(z) > tol
    for j, t in enumerate(np.asarray(gpu_tokens).ravel()):
        top = z[j, ref[j]]
        if pinned[j]:
            assert int(t) == int(ref[j]), f"row {j}: gpu {t} oracle {ref[j]} (pinned)"
        else:
            assert top - z[j, int(t)] <= tol * abs(top), f"row {j}: gpu {t} not near-max"
    return pinned
