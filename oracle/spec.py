"""Propose / verify / commit (Sec. 3.2) and greedy decoding (Eq. stage1).

One `Sequence` holds a prompt whose first P slots carry given (pre-rotation)
keys and values, followed by committed tokens.  The last committed token is
the *pending* token: it sits at index n = seq_len and its keys/values are not
yet in the target cache; it is row 0 of the next verify.

  Eq. verify  rows [pending, d_1..d_K] at slots n..n+K in one forward pass;
              r*_j = argmax of row j-1 (the target's token for index n+j).
  Eq. accept  l = max{ l <= K : d_j = r*_j for every j <= l }.
  Eq. commit  commit (d_1..d_l, r*_{l+1}); the target cache keeps slots
              0..n+l (older slots, the pending token, the l accepted drafts);
              the bonus r*_{l+1} becomes the next pending token; t <- t+l+1.
              The loop ends when a stop token is committed (Sec. 3.2) or the
              token budget is reached.  Slots past the new length are stale and
              are overwritten by the next verify (rollback).
  Eq. propose the routine reasoner proposes d_1..d_K; here as an
              autoregressive chain of single-token draft steps (Sec. 4.1 names
              a depth-bounded autoregressive chain as one draft family).

The draft keeps its own cache (FlatRoPE).  Its slot s is valid while every
token it has consumed up to s equals the committed sequence; after a commit
its length falls back to the first slot where they differ, and the next draft
step first consumes the committed tokens it has not seen (catch-up rows).
"""
from dataclasses import dataclass, field
from typing import Callable, List, Optional

import numpy as np

from . import model as M
from . import numerics
from . import positions


def accept_length(drafts, rstar) -> int:
    """Eq. accept: the longest l in {0..K} with drafts[j] == rstar[j] for all j < l."""
    K = len(drafts)
    best = 0
    for l in range(K + 1):
        if all(int(drafts[j]) == int(rstar[j]) for j in range(l)):
            best = l
    return best


def commit_tokens(drafts, rstar, l: int, stop_token: int = -1, budget: Optional[int] = None):
    """Eq. commit: (d_1..d_l, r*_{l+1}), cut after the first stop token and to
    at most `budget` tokens.  Returns (tokens, finished)."""
    toks = [int(t) for t in drafts[:l]] + [int(rstar[l])]
    finished = False
    if stop_token >= 0 and stop_token in toks:
        toks = toks[:toks.index(stop_token) + 1]
        finished = True
    if budget is not None and len(toks) >= budget:
        toks = toks[:budget]
        finished = True
    return toks, finished


@dataclass
class VerifyResult:
    logits: np.ndarray          # [K+1, V] float64
    rstar: np.ndarray           # [K+1]
    accept_len: int
    committed: List[int]
    finished: bool


class Conditioning:
    """The draft conditioned on target hidden states (Sec. 4.1: the target's
    hidden states from several layers feed the draft; fused EAGLE-3 style,
    Sec. 5).  Reading:

      f_t = W_fuse [h_a(t); h_b(t); h_c(t)]       (3H -> H)
      x_t = e(token_t) + W_in [e(token_t); f_{t-1}]  (2H -> H), the draft's layer-0 input

    where h_l(t) is the target's residual stream after layer l at slot t, taken
    from verify rows whose inputs are committed; f is zero where the target has
    not verified the slot (prompt slots, since prefill is not part of the
    path, and the draft's own proposal rows).

    cross=True is the form Sec. 4.1 states: the fused states are the draft's
    cross-attention keys and values instead of an input term.  The draft's
    layer 0 then attends only to a context whose slot s holds
    k = rot_s(W_k RMSNorm(f_s)), v = W_v RMSNorm(f_s) (its own layer-0 norm
    and projections), for the slots the target has verified, and the given
    prompt keys and values for the prompt slots; a draft row at slot t sees
    the context slots s < t that exist (s < seq_len), and its input is the
    plain embedding (W_in is not used)."""

    def __init__(self, layers, w_fuse: np.ndarray, w_in: Optional[np.ndarray], mirror: bool = False,
                 cross: bool = False):
        self.layers = tuple(int(l) for l in layers)
        self.w_fuse = np.asarray(w_fuse, dtype=np.float64)
        self.w_in = None if w_in is None else np.asarray(w_in, dtype=np.float64)
        self.mirror = mirror
        self.cross = cross

    def fuse(self, captured, j: int) -> np.ndarray:
        h = np.concatenate([captured[l][j] for l in self.layers])
        f = self.w_fuse @ h
        return numerics.mirror(f) if self.mirror else f

    def input(self, x: np.ndarray, slots, feat) -> np.ndarray:
        H = x.shape[1]
        out = np.empty_like(x)
        for i, t in enumerate(slots):
            f = feat.get(int(t) - 1, np.zeros(H))
            out[i] = x[i] + self.w_in @ np.concatenate([x[i], f])
        return out


class Sequence:
    """One scene: target (and optionally draft) caches plus committed tokens."""

    def __init__(self, target: M.Decoder, draft: Optional[M.Decoder], prefix_len: int, blocks,
                 pending_token: int, capacity: int, tgt_prefix_kv, drf_prefix_kv=None,
                 K: int = 4, max_new_tokens: int = 20, stop_token: int = -1,
                 cond: Optional[Conditioning] = None):
        """tgt_prefix_kv(layer) -> (k_bits, v_bits) [P, n_kv, D] uint16; likewise
        drf_prefix_kv for the draft.  `blocks` are (start, t, h, w) grids."""
        self.T, self.D = target, draft
        self.P = prefix_len
        self.K = K
        self.max_new = max_new_tokens
        self.stop = stop_token
        self.cap = capacity
        self.tpos = positions.target_positions(capacity, blocks)
        self.tc = target.new_cache(capacity, self.tpos)
        for li in range(target.s.layers):
            k, v = tgt_prefix_kv(li)
            target.fill_prefix(self.tc, li, k, v)
        self.cond = cond
        self.feat = {}                            # slot -> fused target feature (conditioning)
        self.committed = [int(pending_token)]     # tokens at indices P, P+1, ...
        self.finished = False
        self.history: List[int] = []              # accept length per verify
        if draft is not None:
            # FlatRoPE draft: every slot at its 1D index; an M-RoPE draft (the
            # comparison arm of the attention-budget readout, Sec. 4.2) uses
            # the target's 3D positions
            dpos = self.tpos if draft.rotary == M.ROTARY_MROPE else positions.flat_positions(capacity)
            self.dc = draft.new_cache(capacity, dpos)
            for li in range(draft.s.layers):
                k, v = drf_prefix_kv(li)
                draft.fill_prefix(self.dc, li, k, v)
            self.draft_len = prefix_len
            self.props: List[int] = []            # this round's proposals d_1, d_2, ...

    # index helpers ----------------------------------------------------------
    @property
    def seq_len(self) -> int:
        """Slots with target K/V = index of the pending token."""
        return self.P + len(self.committed) - 1

    @property
    def pending(self) -> int:
        return self.committed[-1]

    @property
    def generated(self) -> List[int]:
        return self.committed[1:]

    def token_at(self, i: int) -> int:
        return self.committed[i - self.P]

    # target ------------------------------------------------------------------
    def verify(self, drafts) -> VerifyResult:
        """Eq. verify + Eq. accept + Eq. commit for one iteration."""
        assert not self.finished
        n = self.seq_len
        K = len(drafts)
        rows = [self.pending] + [int(d) for d in drafts]
        slots = list(range(n, n + K + 1))
        if self.cond is not None:
            self.T.capture_layers = self.cond.layers
        z = self.T.forward(rows, slots, self.tc)
        self.T.capture_layers = ()
        rstar = M.greedy_argmax(z)
        l = accept_length(drafts, rstar)
        budget = self.max_new - len(self.generated)
        toks, fin = commit_tokens(drafts, rstar, l, self.stop, budget)
        if self.cond is not None:
            # rows 0..len(toks)-1 had committed inputs (the pending token and
            # the accepted proposals): their features are final
            for j in range(len(toks)):
                self.feat[n + j] = self.cond.fuse(self.T.captured, j)
            if self.cond.cross and self.D is not None:
                slots_c = list(range(n, n + len(toks)))
                self.D.context_kv(self.dc, 0, np.stack([self.feat[t] for t in slots_c]), slots_c)
        self._commit(n, toks)
        self.finished = fin
        self.history.append(l)
        return VerifyResult(z, rstar, l, toks, fin)

    def _commit(self, n_old: int, toks: List[int]) -> None:
        self.committed.extend(toks)
        if self.D is not None:
            s = n_old + 1
            while s < self.draft_len and (s - n_old - 1) < len(toks) \
                    and self.props[s - n_old - 1] == toks[s - n_old - 1]:
                s += 1
            # The pending token is always re-consumed, so a draft step has a row
            # to propose from.
            self.draft_len = min(self.draft_len, s, self.seq_len)
            self.props = []

    def greedy_step(self) -> int:
        """Eq. stage1 at temperature 0: one target row, commit its argmax."""
        return self.verify([]).committed[0]

    # draft -------------------------------------------------------------------
    def _draft_forward(self, tokens, slots, visible=None):
        if self.cond is not None and self.cond.cross:
            self.D.cross_layer, self.D.cross_len = 0, self.seq_len
        elif self.cond is not None:
            self.D.input_hook = lambda x, sl: self.cond.input(x, sl, self.feat)
        try:
            return self.D.forward(tokens, slots, self.dc, visible=visible)
        finally:
            self.D.input_hook = None
            self.D.cross_layer, self.D.cross_len = None, 0

    def draft_input(self, s: int) -> int:
        n = self.seq_len
        if s <= n:
            return self.token_at(s)
        return self.props[s - n - 1]

    def draft_step(self):
        """One draft step: consume slots draft_len .. n+len(props) and propose
        the next token from the last row.  Returns (token, logits of that row)."""
        n = self.seq_len
        last = n + len(self.props)
        slots = list(range(self.draft_len, last + 1))
        toks = [self.draft_input(s) for s in slots]
        z = self._draft_forward(toks, slots)
        d = int(M.greedy_argmax(z[-1:])[0])
        self.props.append(d)
        self.draft_len = last + 1
        return d, z[-1]

    def propose(self, K: Optional[int] = None) -> List[int]:
        """Eq. propose as K chained draft steps."""
        K = self.K if K is None else K
        return [self.draft_step()[0] for _ in range(K)]

    def block_propose(self, mask_token: int, K: Optional[int] = None):
        """Eq. propose in a single forward (the block-diffusion draft family of
        Sec. 4.1): rows [pending, MASK x K] at slots n..n+K, where the pending
        row attends causally and every MASK row attends to the prefix and to
        all rows of the block; MASK row i proposes d_i (greedy).  Committed
        tokens the draft has not consumed with their own inputs (accepted
        proposals, whose slots hold MASK rows' K/V) are first re-encoded
        causally.  Afterwards only the pending row's slot holds a real input.
        Returns (proposals, logits [K, V] of the MASK rows)."""
        K = self.K if K is None else K
        n = self.seq_len
        if self.draft_len < n:
            slots = list(range(self.draft_len, n))
            self._draft_forward([self.token_at(s) for s in slots], slots)
        rows = [self.pending] + [int(mask_token)] * K
        slots = list(range(n, n + K + 1))
        z = self._draft_forward(rows, slots, visible=[n] + [n + K] * K)
        props = [int(t) for t in M.greedy_argmax(z[1:])]
        self.props = props
        self.draft_len = n + 1
        return props, z[1:]


def greedy_trace(seq: Sequence, max_tokens: Optional[int] = None) -> List[int]:
    """Greedy decoding until stop / budget; returns the generated tokens."""
    limit = seq.max_new if max_tokens is None else max_tokens
    while not seq.finished and len(seq.generated) < limit:
        seq.greedy_step()
    return seq.generated


def spec_loop(seq: Sequence, proposer: Callable[[Sequence], List[int]]) -> List[int]:
    """Propose / verify / commit until finished; returns the generated tokens."""
    while not seq.finished:
        seq.verify(proposer(seq))
    return seq.generated
