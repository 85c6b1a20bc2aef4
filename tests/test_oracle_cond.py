"""Closed-form pins of the draft's conditioning on target hidden states
(Sec. 4.1: hidden states of several target layers feed the draft; Sec. 5:
the EAGLE-3 family fuses three of them).

The reading under test is
    f_t = W_fuse [h_a(t); h_b(t); h_c(t)]              (3H -> H)
    x_t = e(token_t) + W_in [e(token_t); f_{t-1}]      (2H -> H)
with h_l the target's residual stream after layer l.  Scaled identity blocks
make every term of both sums recognisable, so a swapped block, a wrong layer
or slot, or a dropped term changes the result."""
import dataclasses

import numpy as np

import workloads as W
from oracle import model as M
from oracle import spec as OS
from tests import _support as S

H = 4


def _cond(layers, fuse_scales=(1.0, 10.0, 100.0), in_scales=(2.0, 7.0), h=H):
    I = np.eye(h)
    w_fuse = np.concatenate([s * I for s in fuse_scales], axis=1)      # [H, 3H]
    w_in = np.concatenate([s * I for s in in_scales], axis=1)          # [H, 2H]
    return OS.Conditioning(layers, w_fuse, w_in)


def test_fuse_takes_the_named_layers_in_order():
    rng = np.random.default_rng(0)
    cap = {l: rng.standard_normal((3, H)) for l in range(4)}
    c = _cond((2, 0, 3))
    for j in range(3):
        want = cap[2][j] + 10.0 * cap[0][j] + 100.0 * cap[3][j]
        assert np.allclose(c.fuse(cap, j), want, rtol=0, atol=1e-12)
    # the same layer named twice counts twice
    c = _cond((1, 1, 0))
    assert np.allclose(c.fuse(cap, 1), 11.0 * cap[1][1] + 100.0 * cap[0][1], rtol=0, atol=1e-12)


def test_input_adds_embedding_and_previous_slot_feature():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((3, H))
    f = {9: rng.standard_normal(H), 10: rng.standard_normal(H), 11: rng.standard_normal(H)}
    c = _cond((0, 0, 0))
    out = c.input(x, [10, 11, 12], f)
    for i, t in enumerate((10, 11, 12)):
        # e + 2 e + 7 f_{t-1}: the feature of the slot before the row's own
        assert np.allclose(out[i], 3.0 * x[i] + 7.0 * f[t - 1], rtol=0, atol=1e-12)
    # no feature for the previous slot: the fused term is zero
    out = c.input(x[:1], [5], f)
    assert np.allclose(out[0], 3.0 * x[0], rtol=0, atol=1e-12)


def _w():
    base = W.get("C1")
    lay = W.SeqLayout(40, (W.VisionBlock(0, 1, 4, 6),))
    return base.with_(target=dataclasses.replace(base.target, layers=3), vocab=256, seqs=(lay,), K=3,
                      max_new_tokens=10)


def test_captured_state_is_the_residual_after_the_named_layer():
    # with a layer's output projections zeroed, the residual after it equals
    # the residual after the layer before: the capture is taken after the layer
    w = _w()
    hp = W.HostWeights(w)
    T, _ = S.oracle_decoders(w, hp)
    seq = S.oracle_sequence(w, 0, T, None, with_draft=False)
    rows, slots = [seq.pending, 3, 7], [seq.P, seq.P + 1, seq.P + 2]
    T.capture_layers = (0, 1, 2)
    T.forward(rows, slots, seq.tc)
    before = {l: T.captured[l].copy() for l in (0, 1, 2)}
    assert not np.allclose(before[0], before[1])
    Wl = T.layer(1)
    saved = (Wl["wo"].copy(), Wl["w_down"].copy())
    Wl["wo"][:] = 0.0
    Wl["w_down"][:] = 0.0
    try:
        T.forward(rows, slots, seq.tc)
        assert np.array_equal(T.captured[1], T.captured[0])
        assert np.array_equal(T.captured[0], before[0])
    finally:
        Wl["wo"][:], Wl["w_down"][:] = saved
        T.capture_layers = ()


def test_sequence_wires_features_to_committed_slots_and_draft_rows():
    # a verify stores f for the slots whose inputs it committed, from the rows
    # at those slots; a draft row at slot t then reads f_{t-1}
    w = _w()
    hp = W.HostWeights(w)
    T, D = S.oracle_decoders(w, hp)
    cond = _cond((2, 0, 1), h=w.target.hidden)
    trace = OS.greedy_trace(S.oracle_sequence(w, 0, T, None, with_draft=False))
    seq = S.oracle_sequence(w, 0, T, D, cond=cond)
    n = seq.seq_len
    drafts = [trace[0], trace[1], (trace[2] + 1) % w.vocab]    # two accepted
    T.capture_layers = (0, 1, 2)
    res = seq.verify(drafts)
    assert res.accept_len == 2 and len(res.committed) == 3
    assert sorted(seq.feat) == [n, n + 1, n + 2]
    # the same rows through an independent copy of the target cache
    ref = S.oracle_sequence(w, 0, T, None, with_draft=False)
    T.capture_layers = (0, 1, 2)
    T.forward([ref.pending] + drafts, list(range(n, n + 4)), ref.tc)
    cap = {l: T.captured[l].copy() for l in (0, 1, 2)}
    T.capture_layers = ()
    for j in range(3):
        assert np.allclose(seq.feat[n + j], cap[2][j] + 10.0 * cap[0][j] + 100.0 * cap[1][j],
                           rtol=1e-12, atol=1e-12)
    # the draft's next step: record the layer-0 input of each of its rows
    seen = []
    orig = D.forward

    def spy(tokens, slots, cache, **kw):
        hook = D.input_hook
        e = D.embed_rows(tokens)
        seen.append((list(slots), e, hook(e.copy(), np.asarray(slots))))
        return orig(tokens, slots, cache, **kw)

    D.forward = spy
    try:
        seq.draft_step()
    finally:
        D.forward = orig
    slots, e, x = seen[0]
    assert slots[-1] == seq.seq_len
    for i, t in enumerate(slots):
        f = seq.feat.get(t - 1, np.zeros(w.target.hidden))
        assert np.allclose(x[i], 3.0 * e[i] + 7.0 * f, rtol=1e-12, atol=1e-12), t


# --- the cross-attention form (Sec. 4.1: target states as the draft's K/V) ------------

def _cross_seq(mirror=False):
    w = _w()
    hp = W.HostWeights(w)
    T, D = S.oracle_decoders(w, hp)
    cond = S.conditioning(w, hp, (2, 0, 1), cross=True)
    trace = OS.greedy_trace(S.oracle_sequence(w, 0, T, None, with_draft=False))
    seq = S.oracle_sequence(w, 0, T, D, cond=cond)
    return w, T, D, seq, trace


def test_cross_context_rows_are_the_draft_layer0_projections_of_the_features():
    # after a verify that commits three rows, the draft's layer-0 cache holds,
    # at exactly those slots, rot_s(W_k RMSNorm(f_s) g) and W_v RMSNorm(f_s) g;
    # prompt slots keep the given keys and values, other slots stay untouched
    from oracle import rope
    w, T, D, seq, trace = _cross_seq()
    n, P = seq.seq_len, seq.P
    before_k, before_v = seq.dc.k[0].copy(), seq.dc.v[0].copy()
    res = seq.verify([trace[0], trace[1], (trace[2] + 1) % w.vocab])
    assert res.accept_len == 2
    Wd = D.layer(0)
    s = D.s
    for t in (n, n + 1, n + 2):
        a = M.rmsnorm(seq.feat[t], Wd["attn_norm"], s.rms_eps)
        k = (Wd["wk"] @ a).reshape(1, s.kv_heads, s.head_dim)
        want_k = rope.flatrope(k, np.array([t]), s.rope_base)[0]
        want_v = (Wd["wv"] @ a).reshape(s.kv_heads, s.head_dim)
        assert np.allclose(seq.dc.k[0][t], want_k, rtol=1e-10, atol=1e-12), t
        assert np.allclose(seq.dc.v[0][t], want_v, rtol=1e-10, atol=1e-12), t
    untouched = [i for i in range(seq.dc.cap) if i not in (n, n + 1, n + 2)]
    assert np.array_equal(seq.dc.k[0][untouched], before_k[untouched])
    assert np.array_equal(seq.dc.v[0][untouched], before_v[untouched])
    assert np.any(before_k[:P] != 0)


def test_cross_attention_with_zero_keys_averages_the_visible_context():
    # zero W_k and W_q in the draft's layer 0 make every score 0, so each head's
    # output is the plain mean of the values the row sees: the context slots
    # s < min(t, seq_len).  With that layer's down projection zeroed the
    # draft's final hidden row is RMSNorm(e + o W_o^T) g_final, a closed form
    # of that visible set.
    w, T, D, seq, trace = _cross_seq()
    seq.verify([trace[0], (trace[1] + 1) % w.vocab, 0])        # l = 1: two rows committed
    Wd = D.layer(0)
    saved = {k: Wd[k].copy() for k in ("wq", "wk", "w_down")}
    for k in saved:
        Wd[k][:] = 0.0
    try:
        n = seq.seq_len
        # the rows of the next draft step (catch-up rows before n, the pending row at n)
        slots = list(range(seq.draft_len, n + 1))
        toks = [seq.draft_input(t) for t in slots]
        D.cross_layer, D.cross_len = 0, n
        z, hid = D.forward(toks, slots, seq.dc, want_hidden=True)
        D.cross_layer, D.cross_len = None, 0
        s = D.s
        G = s.q_heads // s.kv_heads
        for i, t in enumerate(slots):
            m = min(t, n)                                          # visible: 0 .. m-1
            o = np.concatenate([seq.dc.v[0][:m, h // G, :].mean(axis=0) for h in range(s.q_heads)])
            x = D.embed_rows([toks[i]])[0] + Wd["wo"] @ o
            want = M.rmsnorm(x, D.final_norm(), s.rms_eps)
            assert np.allclose(hid[i], want, rtol=1e-10, atol=1e-12), t
    finally:
        for k, v in saved.items():
            Wd[k][:] = v


def test_cross_row_sees_neither_its_own_slot_nor_unverified_slots():
    w, T, D, seq, trace = _cross_seq()
    seq.verify([trace[0], trace[1], (trace[2] + 1) % w.vocab])   # three rows committed
    n = seq.seq_len

    def run(slot_tok):
        D.cross_layer, D.cross_len = 0, n
        try:
            return D.forward([slot_tok[1]], [slot_tok[0]], seq.dc)
        finally:
            D.cross_layer, D.cross_len = None, 0

    t = n - 1                       # a catch-up row at a verified slot
    row = (t, seq.token_at(t))
    z0 = run(row)
    for which in ("k", "v"):
        c = getattr(seq.dc, which)[0]
        keep = c.copy()
        c[t] += 3.0                 # the row's own slot: not visible
        assert np.array_equal(run(row), z0)
        c[:] = keep
        c[t - 1] += 3.0             # the slot before: visible
        assert not np.allclose(run(row), z0)
        c[:] = keep
    # a proposal row beyond seq_len sees no context at or after seq_len
    row = (n + 2, 5)
    z1 = run(row)
    c = seq.dc.v[0]
    keep = c.copy()
    c[n:n + 2] += 3.0
    assert np.array_equal(run(row), z1)
    c[n - 1] += 3.0
    assert not np.allclose(run(row), z1)
    c[:] = keep


def test_cross_conditioned_spec_loop_equals_greedy():
    w, T, D, seq, trace = _cross_seq()
    assert OS.spec_loop(seq, lambda sq: sq.propose()) == list(trace)
