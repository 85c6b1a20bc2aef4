"""Opens a speculative-decoding context on a seeded synthetic workload.

Plumbing only: weights and prompt K/V come from the `workloads` generators and
are placed in device memory with torch; the context, every kernel and every
length live in the HIP library behind include/spec.h.
"""
from __future__ import annotations

from typing import Optional

import numpy as np

from . import binding as B


def _require_gpu():
    import torch
    if not torch.cuda.is_available():
        raise RuntimeError("the speculative path needs a ROCm GPU (gfx950); no device is visible")
    return torch


class Session:
    """Device weights + prompt caches + an open spec_ctx for one workload.

    source='host'   weights drawn with numpy on the host (small shapes)
    source='device' weights drawn on the GPU with torch's seeded generator
    page_seed       None: each sequence's KV pages follow the previous
                    sequence's; an int: a seeded random permutation of the
                    page pool is handed over as the sequences' page tables
    pending_tokens  None: the workload's first pending token per sequence;
                    else one token id per sequence
    cond_cross      with cond_layers: the features are the draft's layer-0
                    cross-attention context (SPEC_FLAG_COND_CROSS)
    """

    def __init__(self, w, source: str = "host", flags: int = 0, with_draft: bool = True,
                 K: Optional[int] = None, max_new_tokens: Optional[int] = None, stop_token: Optional[int] = None,
                 provider=None, page_seed: Optional[int] = None, mask_token: Optional[int] = None,
                 cond_layers=None, pending_tokens=None, cond_cross: bool = False):
        torch = _require_gpu()
        import workloads as W
        self.torch = torch
        self.w = w
        self.K = w.K if K is None else K
        self.B = w.batch
        self.V = w.vocab
        self.dev = torch.device("cuda")
        if provider is not None:
            self.src = provider
        elif source == "host":
            self.src = W.HostWeights(w)
        else:
            self.src = W.DeviceWeights(w)
        self.source = source
        self.has_draft = with_draft and w.draft is not None

        self._keep = []
        self.embed = self._tensor("global", -1, "embed")
        self.tgt_w, self.tgt_struct = self._model("target", w.target)
        if self.has_draft:
            self.drf_w, self.drf_struct = self._model("draft", w.draft)

        cfg = B.spec_config()
        cfg.target = B.dims(w.target)
        cfg.draft = B.dims(w.draft if self.has_draft else None)
        cfg.vocab = w.vocab
        cfg.K = self.K
        cfg.batch = self.B
        cfg.max_new_tokens = w.max_new_tokens if max_new_tokens is None else max_new_tokens
        cfg.stop_token = w.stop_token if stop_token is None else stop_token
        cfg.flags = flags
        cfg.mask_token = w.vocab - 1 if mask_token is None else mask_token   # block proposal's MASK input
        if cond_layers is not None:   # the draft conditioned on these target layers' hidden states
            cfg.flags |= B.SPEC_FLAG_COND | (B.SPEC_FLAG_COND_CROSS if cond_cross else 0)
            for i in range(3):
                cfg.cond_layers[i] = int(cond_layers[i])
            self.w_fuse = self._tensor("draft", -1, "w_fuse")
            self.drf_struct.w_fuse = self.w_fuse.data_ptr()
            if not cond_cross:        # the cross-attention form has no input projection
                self.w_in = self._tensor("draft", -1, "w_in")
                self.drf_struct.w_in = self.w_in.data_ptr()
        self.cfg = cfg

        seqs = (B.spec_seq_init * self.B)()
        prefix = []
        for b, lay in enumerate(w.seqs):
            s = seqs[b]
            s.prefix_len = lay.prefix_len
            blocks = (B.spec_vision_block * max(1, len(lay.blocks)))()
            for i, bl in enumerate(lay.blocks):
                blocks[i].start, blocks[i].t, blocks[i].h, blocks[i].w = bl.start, bl.t, bl.h, bl.w
            s.n_blocks = len(lay.blocks)
            s.blocks = blocks
            s.pending_token = (W.first_pending_token(w, b) if pending_tokens is None
                               else int(pending_tokens[b]))
            kv = {}
            for model, shape in (("target", w.target), ("draft", w.draft if self.has_draft else None)):
                if shape is None:
                    continue
                ks = [self._prefix(b, model, li, "k") for li in range(shape.layers)]
                vs = [self._prefix(b, model, li, "v") for li in range(shape.layers)]
                kv[model] = (ks, vs)
                prefix += ks + vs
            arr = lambda ts: (ctypes_void_array(len(ts)))(*[t.data_ptr() for t in ts])
            s.tgt_k, s.tgt_v = arr(kv["target"][0]), arr(kv["target"][1])
            if self.has_draft:
                s.drf_k, s.drf_v = arr(kv["draft"][0]), arr(kv["draft"][1])
            self._keep += [blocks, s.tgt_k, s.tgt_v]
        if page_seed is not None:
            import ctypes
            npg = [B.spec_seq_pages(cfg, seqs[b]) for b in range(self.B)]
            perm = np.random.default_rng(page_seed).permutation(sum(npg)).astype(np.int32)
            self.page_tables = []
            off = 0
            for b in range(self.B):
                arr = (ctypes.c_int32 * npg[b])(*perm[off:off + npg[b]].tolist())
                off += npg[b]
                seqs[b].page_table = arr
                self.page_tables.append(arr)
            self._keep += self.page_tables
        self.seqs = seqs
        self.ws_bytes = B.spec_workspace_bytes(cfg, seqs)
        self.ws = torch.empty(self.ws_bytes, dtype=torch.uint8, device=self.dev)
        self.stream = torch.cuda.current_stream()
        self.ctx = B.spec_init(cfg, self.embed.data_ptr(), self.tgt_struct,
                               self.drf_struct if self.has_draft else None, seqs, self.ws.data_ptr(),
                               self.ws_bytes, self.stream.cuda_stream)
        del prefix     # spec_init waited for the uploads; prompt K/V are no longer needed
        K1 = self.K + 1
        self.dtok = torch.full((self.B, max(1, self.K)), -1, dtype=torch.int32, device=self.dev)
        self.vtok = torch.zeros((self.B, max(1, self.K)), dtype=torch.int32, device=self.dev)
        self.logits = torch.zeros((self.B, K1, self.V), dtype=torch.bfloat16, device=self.dev)
        self.acc = torch.zeros(self.B, dtype=torch.int32, device=self.dev)
        self.com = torch.zeros((self.B, K1), dtype=torch.int32, device=self.dev)
        self.ncom = torch.zeros(self.B, dtype=torch.int32, device=self.dev)
        self.fin = torch.zeros(self.B, dtype=torch.int32, device=self.dev)

    # -- tensors ---------------------------------------------------------------
    def _tensor(self, model, layer, name):
        torch = self.torch
        if self.source == "device" and hasattr(self.src, "tensor"):
            t = self.src.tensor(model, layer, name)
        else:
            bits = self.src.get(model, layer, name)
            t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(self.dev).view(torch.bfloat16)
        self._keep.append(t)
        return t

    def _prefix(self, b, model, layer, which):
        import workloads as W
        torch = self.torch
        if self.source == "device":
            return W.prefix_kv_device(self.w, b, model, layer, which)
        bits = W.prefix_kv_host(self.w, b, model, layer, which)
        return torch.from_numpy(bits.view(np.int16)).to(self.dev).view(torch.bfloat16)

    def _model(self, model, shape):
        layers = (B.spec_layer_weights * shape.layers)()
        tens = []
        for li in range(shape.layers):
            d = {}
            for n in ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "w_gate", "w_up", "w_down"):
                t = self._tensor(model, li, n)
                d[n] = t
                setattr(layers[li], n, t.data_ptr())
            tens.append(d)
        fn = self._tensor(model, -1, "final_norm")
        st = B.spec_model_weights()
        st.layers = layers
        st.final_norm = fn.data_ptr()
        self._keep += [layers]
        return tens, st

    # -- calls ---------------------------------------------------------------------
    def draft_step(self, out=None):
        B.draft_step(self.ctx, (out if out is not None else self.dtok).data_ptr())

    def draft_steps(self, n: int, out=None):
        B.draft_steps(self.ctx, n, (out if out is not None else self.dtok).data_ptr())

    def verify(self, drafts=None, logits: bool = False):
        """drafts: None (the draft's own proposals), or [B][K] ints (host or device)."""
        ptr = 0
        if drafts is not None:
            t = drafts if hasattr(drafts, "data_ptr") else self.torch.as_tensor(np.asarray(drafts, dtype=np.int32))
            self.vtok.copy_(t.reshape(self.B, -1).to(self.dev, self.torch.int32), non_blocking=False)
            ptr = self.vtok.data_ptr()
        B.spec_verify(self.ctx, ptr, self.logits.data_ptr() if logits else 0)

    def commit(self):
        B.spec_commit(self.ctx, self.acc.data_ptr(), self.com.data_ptr(), self.ncom.data_ptr(), self.fin.data_ptr())

    def attn_readout(self, model: int, layer: int):
        """Arms the attention-budget readout of `layer` for the next pass of
        `model` (0 target, 1 draft); returns the float32 [B, K+1, q_heads, 4]
        device tensor that pass fills (NaN where it writes nothing)."""
        shape = self.w.target if model == 0 else self.w.draft
        out = self.torch.full((self.B, self.K + 1, shape.q_heads, 4), float("nan"), dtype=self.torch.float32,
                              device=self.dev)
        self._readout = out
        B.spec_attn_readout(self.ctx, model, layer, out.data_ptr())
        return out

    def sync(self) -> int:
        return B.spec_sync(self.ctx)

    def state(self, b: int = 0) -> dict:
        return B.spec_debug_state(self.ctx, b)

    def positions(self, b: int, length: int):
        return B.spec_debug_positions(self.ctx, b, length)

    def feature(self, b, slot0, n):
        return B.spec_debug_feature(self.ctx, b, slot0, n, self.w.target.hidden)

    def kv(self, b, model, layer, which, pos0, npos):
        shape = self.w.target if model == 0 else self.w.draft
        return B.spec_debug_kv(self.ctx, b, model, layer, which, pos0, npos, shape.kv_heads, shape.head_dim)

    def committed(self):
        """Host copies of the last commit's outputs (synchronising)."""
        n = self.ncom.cpu().numpy()
        c = self.com.cpu().numpy()
        return [list(c[b, :n[b]]) for b in range(self.B)], self.acc.cpu().numpy(), self.fin.cpu().numpy()

    def close(self):
        if getattr(self, "ctx", None):
            B.spec_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def ctypes_void_array(n):
    import ctypes
    return ctypes.c_void_p * n
