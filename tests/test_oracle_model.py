"""Pins for the oracle's decoder stack: closed forms of RMSNorm and SiLU, an
online-softmax (split-KV) evaluation of attention, the MHA equivalence of the
GQA grouping, causality, shift invariance, and verify-of-K == K+1 sequential
decodes (Eq. verify)."""
import dataclasses
import math

import numpy as np
import pytest
import scipy.special

import workloads as W
from oracle import model as M
from oracle import numerics, positions, rope
from tests import _support as S


# --- numerics ---------------------------------------------------------------

def test_bf16_decode_known_patterns():
    bits = np.array([0x3F80, 0xC020, 0x0000, 0x8000, 0x4049, 0x7F80], dtype=np.uint16)
    v = numerics.decode(bits)
    assert v[0] == 1.0 and v[1] == -2.5 and v[2] == 0.0 and v[3] == 0.0
    assert v[4] == 3.140625 and np.isinf(v[5])


def test_bf16_mirror_rounding():
    x = np.array([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 1.0 + 2 ** -8 + 2 ** -20, -1.0 - 2 ** -8])
    assert list(numerics.mirror(x)) == [1.0, 1.0 + 2 ** -6, 1.0 + 2 ** -7, -1.0]
    assert np.isnan(numerics.mirror(np.array([np.nan])))[0]


# --- RMSNorm / SiLU -----------------------------------------------------------

def test_rmsnorm_unit_rms_and_scale_invariance():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((4, 300)) * 7.0
    y = M.rmsnorm(x, np.ones(300), 0.0)
    assert np.allclose(np.sqrt(np.mean(y * y, axis=-1)), 1.0, rtol=1e-13)
    assert np.allclose(M.rmsnorm(3.0 * x, np.ones(300), 0.0), y, rtol=1e-13)
    g = rng.standard_normal(300)
    assert np.allclose(M.rmsnorm(x, g, 0.0), y * g, rtol=1e-13)


def test_normed_pair_is_rmsnorm_times_gain():
    # the (x * g, 1/rms) pair the forward pass projects equals RMSNorm(x) * g
    w = _tiny()
    T, _ = S.oracle_decoders(w, W.HostWeights(w))
    rng = np.random.default_rng(14)
    x = rng.standard_normal((3, w.target.hidden)) * 5
    g = 1 + 0.1 * rng.standard_normal(w.target.hidden)
    a, inv = T._normed(x, g)
    assert np.allclose(a * inv, M.rmsnorm(x, g, w.target.rms_eps), rtol=1e-13, atol=1e-15)
    T.mirror = True
    am, _ = T._normed(x, g)
    assert np.array_equal(am, numerics.mirror(x * g))


def test_silu_is_x_times_logistic():
    x = np.linspace(-30, 30, 101)
    assert np.allclose(M.silu(x), x * scipy.special.expit(x), rtol=1e-13, atol=1e-300)
    assert M.silu(np.array([0.0]))[0] == 0.0


# --- attention ------------------------------------------------------------------

def _online_attention(q, kc, vc, slots, chunk):
    """Keys processed in chunks with running max / running sum (the split-KV
    log-sum-exp merge); an independent evaluation of softmax attention."""
    M_, nq, D = q.shape
    G = nq // kc.shape[1]
    out = np.zeros_like(q)
    for i in range(M_):
        for h in range(nq):
            m_run, l_run, acc = -math.inf, 0.0, np.zeros(D)
            n_vis = slots[i] + 1
            for c0 in range(0, n_vis, chunk):
                ks = kc[c0:min(n_vis, c0 + chunk), h // G]
                s = ks @ q[i, h] / math.sqrt(D)
                m_new = max(m_run, float(np.max(s)))
                scale = math.exp(m_run - m_new) if m_run > -math.inf else 0.0
                p = np.exp(s - m_new)
                l_run = l_run * scale + float(np.sum(p))
                acc = acc * scale + p @ vc[c0:c0 + len(s), h // G]
                m_run = m_new
            out[i, h] = acc / l_run
    return out


def test_attention_matches_online_softmax():
    rng = np.random.default_rng(1)
    q = rng.standard_normal((3, 6, 16))
    kc = rng.standard_normal((40, 2, 16)) * 2
    vc = rng.standard_normal((40, 2, 16))
    slots = [20, 33, 39]
    ref = M.attend(q, kc, vc, slots)
    for chunk in (1, 7, 64):
        assert np.allclose(_online_attention(q, kc, vc, slots, chunk), ref, rtol=1e-12, atol=1e-12)


def test_attention_closed_forms():
    rng = np.random.default_rng(2)
    q = rng.standard_normal((2, 2, 8))
    vc = rng.standard_normal((10, 1, 8))
    kc = np.tile(rng.standard_normal((1, 1, 8)), (10, 1, 1))    # identical keys
    out = M.attend(q, kc, vc, [9, 0])
    assert np.allclose(out[0, :], vc[:10, 0].mean(axis=0), rtol=1e-12)   # uniform weights
    assert np.allclose(out[1, :], vc[0, 0], rtol=1e-12)                   # one visible key


def test_gqa_equals_mha_with_repeated_kv_heads():
    # q head h reads kv head h // (n_q / n_kv): the same as MHA whose kv head h
    # is a copy of GQA kv head h // G.
    rng = np.random.default_rng(3)
    q = rng.standard_normal((2, 6, 8))
    kc = rng.standard_normal((12, 2, 8))
    vc = rng.standard_normal((12, 2, 8))
    rep = [0, 0, 0, 1, 1, 1]
    a = M.attend(q, kc, vc, [5, 11])
    b = M.attend(q, kc[:, rep], vc[:, rep], [5, 11])
    assert np.array_equal(a, b)


# --- whole stack ----------------------------------------------------------------

def _tiny(prefix=40, vocab=256, layers=2):
    base = W.get("C1")
    lay = W.SeqLayout(prefix, (W.VisionBlock(0, 1, 4, 6),))
    return base.with_(target=dataclasses.replace(base.target, layers=layers), vocab=vocab, seqs=(lay,))


def test_verify_rows_equal_sequential_decodes():
    # Eq. verify: row j of one batched pass equals a single-row pass after the
    # earlier rows were decoded one by one.
    w = _tiny()
    hp = W.HostWeights(w)
    T, _ = S.oracle_decoders(w, hp)
    rng = np.random.default_rng(4)
    toks = rng.integers(0, w.vocab, size=5)
    a = S.oracle_sequence(w, 0, T, None, with_draft=False)
    b = S.oracle_sequence(w, 0, T, None, with_draft=False)
    n = a.seq_len
    za = T.forward(list(toks), list(range(n, n + 5)), a.tc)
    for j in range(5):
        zb = T.forward([int(toks[j])], [n + j], b.tc)
        assert np.allclose(zb[0], za[j], rtol=1e-9, atol=1e-12)
    for li in range(w.target.layers):
        assert np.allclose(a.tc.k[li][:n + 5], b.tc.k[li][:n + 5], rtol=1e-9, atol=1e-12)


def test_causality_of_new_rows():
    w = _tiny()
    hp = W.HostWeights(w)
    T, _ = S.oracle_decoders(w, hp)
    a = S.oracle_sequence(w, 0, T, None, with_draft=False)
    b = S.oracle_sequence(w, 0, T, None, with_draft=False)
    n = a.seq_len
    za = T.forward([3, 4, 5, 6], list(range(n, n + 4)), a.tc)
    zb = T.forward([3, 4, 9, 11], list(range(n, n + 4)), b.tc)
    assert np.array_equal(za[:2], zb[:2])
    assert not np.allclose(za[2:], zb[2:])


def test_logits_invariant_to_shared_position_shift():
    # Every axis of every slot shifted by the same delta leaves all scores, hence
    # the logits, unchanged (relative-position property of the rotation).
    w = _tiny()
    hp = W.HostWeights(w)
    T, _ = S.oracle_decoders(w, hp)
    P = w.seqs[0].prefix_len
    cap = P + 8
    pos = positions.target_positions(cap, [(0, 1, 4, 6)])
    outs = []
    for delta in (0, 37, 1000):
        c = T.new_cache(cap, pos + delta)
        for li in range(w.target.layers):
            k, v = S.host_kv(w, 0, "target")(li)
            T.fill_prefix(c, li, k, v)
        outs.append(T.forward([1, 2, 3], [P, P + 1, P + 2], c))
    for z in outs[1:]:
        assert np.allclose(z, outs[0], rtol=1e-9, atol=1e-11)


def test_zero_output_projections_leave_residual_stream():
    # With W_o = W_down = 0 each layer is the identity on x, so the logits are
    # the final norm of the token embedding against the tied head.
    w = _tiny()
    hp = W.HostWeights(w)

    class ZeroProj:
        def get(self, model, layer, name):
            a = hp.get(model, layer, name)
            return np.zeros_like(a) if name in ("wo", "w_down") else a

    T, _ = S.oracle_decoders(w, ZeroProj())
    seq = S.oracle_sequence(w, 0, T, None, with_draft=False)
    z = T.forward([7], [seq.seq_len], seq.tc)
    E = numerics.decode(hp.get("global", -1, "embed"))
    g = numerics.decode(hp.get("target", -1, "final_norm"))
    x = E[7]
    h = x / np.sqrt(np.mean(x * x) + w.target.rms_eps) * g
    assert np.allclose(z[0], E @ h, rtol=1e-12, atol=1e-12)


def test_greedy_argmax_ties_and_nan():
    z = np.array([[1.0, 3.0, 3.0, 2.0], [np.nan, 0.5, np.nan, 0.5], [-1.0, -2.0, np.nan, -1.0]])
    assert list(M.greedy_argmax(z)) == [1, 1, 0]


def test_softmax_rows_sum_to_one_and_are_shift_invariant():
    rng = np.random.default_rng(12)
    s = rng.standard_normal((5, 37)) * 30
    p = M.softmax(s)
    assert np.allclose(p.sum(axis=-1), 1.0, rtol=0, atol=1e-14)
    assert np.all(p >= 0)
    assert np.allclose(M.softmax(s + 1234.5), p, rtol=1e-12, atol=1e-15)
    assert np.allclose(p, scipy.special.softmax(s, axis=-1), rtol=1e-12, atol=1e-15)


def test_chunked_lm_head_equals_one_product():
    # the LM head over vocabulary chunks (used for the 152064-row head) equals
    # one product with the whole decoded embedding, ragged last chunk included
    w = _tiny(vocab=1000)
    hp = W.HostWeights(w)
    E = numerics.decode(hp.get("global", -1, "embed"))
    h = np.random.default_rng(13).standard_normal((3, w.target.hidden))
    whole = M.Decoder(hp, "target", w.target, w.vocab, M.ROTARY_MROPE)
    assert whole.vocab <= whole.lm_chunk
    chunked = M.Decoder(hp, "target", w.target, w.vocab, M.ROTARY_MROPE, cache_weights=False, lm_chunk=96)
    ref = h @ E.T
    assert np.allclose(whole.lm_head(h), ref, rtol=1e-13, atol=1e-13)
    assert np.allclose(chunked.lm_head(h), ref, rtol=1e-13, atol=1e-13)
    assert chunked.lm_head(h).shape == (3, 1000)
