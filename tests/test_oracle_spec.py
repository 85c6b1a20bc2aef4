"""Pins for propose / verify / commit (Sec. 3.2).

The plain definition the method must reach is greedy decoding of the target
(Eq. stage1 at temperature 0): speculative decoding keeps the target's exact
greedy output (Sec. 2).  These tests check the oracle's loop against that,
against brute-force enumeration of the accept rule, against a fresh prefill of
the committed sequence, and the reporting formulas against Table main."""
import dataclasses
import itertools

import numpy as np
import pytest

import workloads as W
from oracle import model as M
from oracle import report
from oracle import spec as OS
from tests import _support as S


def _tiny(K=4, max_new=12, stop=-1, vocab=256, prefix=48):
    base = W.get("C1")
    lay = W.SeqLayout(prefix, (W.VisionBlock(0, 1, 5, 6),))
    return base.with_(vocab=vocab, seqs=(lay,), K=K, max_new_tokens=max_new, stop_token=stop)


@pytest.fixture(scope="module")
def tiny():
    w = _tiny()
    hp = W.HostWeights(w)
    T, D = S.oracle_decoders(w, hp)
    seq = S.oracle_sequence(w, 0, T, D)
    trace = list(OS.greedy_trace(seq))
    return w, hp, T, D, trace


# --- Eq. accept -------------------------------------------------------------------

def _first_mismatch(d, r):
    eq = np.asarray(d) == np.asarray(r)[:len(d)]
    return int(np.argmin(eq)) if not eq.all() else len(d)


def test_accept_length_bruteforce_small_vocab():
    # every draft in {0..7}^3 against several target argmax vectors
    for rstar in [(0, 1, 2, 3), (5, 5, 5, 5), (7, 0, 7, 1)]:
        for d in itertools.product(range(8), repeat=3):
            assert OS.accept_length(d, rstar) == _first_mismatch(d, rstar)


def test_accept_length_random_large_vocab():
    rng = np.random.default_rng(0)
    for _ in range(2000):
        K = int(rng.integers(0, 17))
        r = rng.integers(0, 1024, size=K + 1)
        d = np.where(rng.random(K) < 0.8, r[:K], rng.integers(0, 1024, size=K))
        assert OS.accept_length(d, r) == _first_mismatch(d, r)


def test_commit_rule_bonus_stop_and_budget():
    toks, fin = OS.commit_tokens([4, 5, 6], [4, 5, 9, 8], 2)
    assert toks == [4, 5, 9] and not fin
    toks, fin = OS.commit_tokens([4, 5, 6], [4, 5, 6, 8], 3)
    assert toks == [4, 5, 6, 8] and not fin                     # l = K commits K+1
    toks, fin = OS.commit_tokens([4, 5, 6], [4, 5, 6, 8], 3, stop_token=5)
    assert toks == [4, 5] and fin
    toks, fin = OS.commit_tokens([4, 5, 6], [4, 5, 6, 8], 3, budget=2)
    assert toks == [4, 5] and fin


# --- whole loop vs greedy decoding -----------------------------------------------

def test_trace_is_greedy_by_definition(tiny):
    # each greedy token is the argmax of a single-row pass over all earlier tokens
    w, hp, T, D, trace = tiny
    seq = S.oracle_sequence(w, 0, T, None, with_draft=False)
    toks = [seq.pending] + trace
    n0 = seq.seq_len
    for j in range(len(trace)):
        z = T.forward([toks[j]], [n0 + j], seq.tc)
        assert int(np.argmax(z[0])) == trace[j]


@pytest.mark.parametrize("p", [0.0, 0.5, 0.8, 1.0])
def test_spec_loop_equals_greedy_synthetic_drafts(tiny, p):
    w, hp, T, D, trace = tiny
    w2 = w.with_(p_accept=(p,))
    seq = S.oracle_sequence(w2, 0, T, None, with_draft=False)
    synth = W.DraftSynth(w2, 0)

    def proposer(s):
        i = len(s.generated)
        return list(synth.propose(np.array(trace[i:]), w.K))

    out = OS.spec_loop(seq, proposer)
    assert out == trace
    if p == 1.0:
        assert all(l == w.K for l in seq.history[:-1])
    if p == 0.0:
        assert max(seq.history) <= 1    # only accidental matches


def test_spec_loop_equals_greedy_with_draft_model(tiny):
    w, hp, T, D, trace = tiny
    seq = S.oracle_sequence(w, 0, T, D)
    out = OS.spec_loop(seq, lambda s: s.propose())
    assert out == trace


def test_accept_zero_is_one_greedy_step_and_full_accept(tiny):
    w, hp, T, D, trace = tiny
    seq = S.oracle_sequence(w, 0, T, None, with_draft=False)
    wrong = [(trace[0] + 1) % w.vocab] * w.K
    r = seq.verify(wrong)
    assert r.accept_len == 0 and r.committed == [trace[0]]
    r = seq.verify(trace[1:1 + w.K])
    assert r.accept_len == w.K and r.committed == trace[1:2 + w.K]


def test_commit_leaves_cache_equal_to_fresh_prefill(tiny):
    # After rounds with rejected drafts, every valid slot equals what a fresh
    # one-token-at-a-time pass over the committed tokens stores.
    w, hp, T, D, trace = tiny
    a = S.oracle_sequence(w, 0, T, D)
    rng = np.random.default_rng(5)
    for _ in range(3):
        a.propose()
        i = len(a.generated)
        d = [t if rng.random() < 0.6 else int(rng.integers(0, w.vocab)) for t in trace[i:i + w.K]]
        d += [0] * (w.K - len(d))
        a.verify(d)
    b = S.oracle_sequence(w, 0, T, D)
    for _ in range(len(a.generated)):
        b.greedy_step()
    assert a.generated == b.generated
    n = a.seq_len
    for li in range(w.target.layers):
        assert np.allclose(a.tc.k[li][:n], b.tc.k[li][:n], rtol=1e-9, atol=1e-12)
        assert np.allclose(a.tc.v[li][:n], b.tc.v[li][:n], rtol=1e-9, atol=1e-12)
    # draft: its valid slots equal a fresh draft pass over the committed tokens
    c = S.oracle_sequence(w, 0, T, D)
    toks = [c.pending] + a.generated
    P = c.P
    D.forward(toks[:a.draft_len - P], list(range(P, a.draft_len)), c.dc)
    for li in range(w.draft.layers):
        assert np.allclose(a.dc.k[li][:a.draft_len], c.dc.k[li][:a.draft_len], rtol=1e-9, atol=1e-12)
    assert a.draft_len <= a.seq_len


def test_draft_catch_up_rows_after_override(tiny):
    # Draft proposals overridden by the verifier: the next draft step re-consumes
    # the committed tokens it has not seen and proposes what a fresh draft would.
    w, hp, T, D, trace = tiny
    a = S.oracle_sequence(w, 0, T, D)
    props = a.propose()
    override = trace[:w.K]
    r = a.verify(override)
    d_next, z_next = a.draft_step()
    c = S.oracle_sequence(w, 0, T, D)
    toks = [c.pending] + a.generated
    z = D.forward(toks, list(range(c.P, a.seq_len + 1)), c.dc)
    assert d_next == int(np.argmax(z[-1]))
    assert np.allclose(z_next, z[-1], rtol=1e-9, atol=1e-12)


def test_stop_token_and_budget(tiny):
    w, hp, T, D, trace = tiny
    stop = trace[5]
    cut = trace.index(stop)
    w2 = w.with_(stop_token=stop)
    seq = S.oracle_sequence(w2, 0, T, D)
    assert OS.spec_loop(seq, lambda s: s.propose()) == trace[:cut + 1]
    w3 = w.with_(max_new_tokens=7)
    seq = S.oracle_sequence(w3, 0, T, D)
    assert OS.spec_loop(seq, lambda s: s.propose()) == trace[:7]


# --- reporting (Eq. L-and-speedup, Sec. 5.1, Table main) -------------------------

def test_table_main_speedups_from_L_and_c():
    # EAGLE-3 chain draft: c = 15 * 0.047 = 0.705; block-diffusion: c = 0.18.
    c_ar, c_bd = 15 * 0.047, 0.18
    rows = [  # (L, printed S, c, tolerance)
        (7.33, 4.30, c_ar, 0.015), (6.99, 4.11, c_ar, 0.015), (7.41, 4.36, c_ar, 0.015),
        (7.35, 4.32, c_ar, 0.015), (6.95, 4.08, c_ar, 0.015), (7.30, 4.29, c_ar, 0.015),
        (5.16, 4.39, c_bd, 0.03), (4.65, 3.97, c_bd, 0.03), (4.95, 4.21, c_bd, 0.03),
        (5.17, 4.40, c_bd, 0.03), (4.67, 3.97, c_bd, 0.03),
    ]
    for L, S_print, c, tol in rows:
        assert abs(report.theoretical_speedup(L, c) - S_print) <= tol
    # the tok/s column is the 34 tok/s target-only rate times off-shelf S
    for S_off, tps in [(4.23, 143.8), (4.36, 148.2), (4.29, 145.9), (4.21, 143.1)]:
        assert round(34.0 * S_off, 1) == tps
    # "L = 4.6 -> about 78% of tokens from the routine path": (L - 1) / L
    assert round((4.6 - 1) / 4.6, 2) == 0.78


def test_iid_expected_L_by_enumeration():
    # E[l+1] for independent matches, by enumerating every match pattern with
    # its probability and applying the accept rule to it.
    for p, K in [(0.75, 8), (0.5, 5), (0.9, 4)]:
        e = 0.0
        for pat in itertools.product([True, False], repeat=K):
            prob = np.prod([p if m else 1 - p for m in pat])
            d = [0 if m else 1 for m in pat]
            e += prob * (OS.accept_length(d, [0] * (K + 1)) + 1)
        assert e == pytest.approx(report.iid_expected_L(p, K), rel=1e-12)
        assert e == pytest.approx((1 - p ** (K + 1)) / (1 - p), rel=1e-12)
    assert report.mean_accepted_length([3, 0, 8]) == pytest.approx(14 / 3)


def test_mrope_draft_reduces_to_flatrope_on_text_and_differs_on_vision():
    # An M-RoPE draft gives every text slot (i, i, i), whose rotation is the 1D
    # one at i (Eq. rope-3d with equal axes), so on a prompt without vision
    # blocks it proposes exactly what the FlatRoPE draft does; with a vision
    # block the two see different key positions.
    for blocks, same in (((), True), ((W.VisionBlock(0, 1, 5, 6),), False)):
        w = _tiny(vocab=256).with_(seqs=(W.SeqLayout(48, blocks),))
        hp = W.HostWeights(w)
        outs = []
        for rot in (M.ROTARY_FLAT, M.ROTARY_MROPE):
            T, D = S.oracle_decoders(w, hp, draft_rotary=rot)
            seq = S.oracle_sequence(w, 0, T, D)
            d, z = seq.draft_step()
            outs.append((d, z, seq.dc.k[0][:48].copy()))
        assert np.allclose(outs[0][1], outs[1][1], rtol=1e-12, atol=1e-12) == same
        assert np.allclose(outs[0][2], outs[1][2], rtol=1e-12, atol=1e-12) == same


# --- block proposal (single-forward draft, Eq. propose) ---------------------------

def _block_seq(K=4, max_new=12):
    w = _tiny(K=K, max_new=max_new)
    hp = W.HostWeights(w)
    T, D = S.oracle_decoders(w, hp)
    return w, hp, T, D


def test_block_visibility_rules():
    w, hp, T, D = _block_seq()
    mask = w.vocab - 1
    seq = S.oracle_sequence(w, 0, T, D)
    n, K = seq.seq_len, w.K
    rows = [seq.pending] + [mask] * K
    slots = list(range(n, n + K + 1))
    ref = S.oracle_sequence(w, 0, T, D)
    # visible = slots is the default causal pass, bit for bit
    z_causal = ref.D.forward(rows, slots, ref.dc)
    fresh = S.oracle_sequence(w, 0, T, D)
    assert np.array_equal(fresh.D.forward(rows, slots, fresh.dc, visible=slots), z_causal)
    z_block = seq.D.forward(rows, slots, seq.dc, visible=[n] + [n + K] * K)
    # the pending row and the last MASK row see exactly what a causal pass shows them
    assert np.array_equal(z_block[0], z_causal[0])
    assert np.allclose(z_block[K], z_causal[K], rtol=1e-12, atol=1e-12)
    # an earlier MASK row also sees the MASK rows after it
    assert not np.allclose(z_block[1], z_causal[1], rtol=1e-6)


def test_spec_loop_with_block_drafts_equals_greedy():
    w, hp, T, D = _block_seq()
    trace = OS.greedy_trace(S.oracle_sequence(w, 0, T, None, with_draft=False))
    seq = S.oracle_sequence(w, 0, T, D)
    out = OS.spec_loop(seq, lambda sq: sq.block_propose(w.vocab - 1)[0])
    assert out == list(trace)


def test_block_catch_up_reencodes_accepted_tokens():
    # proposals that the verifier accepts were consumed as MASK inputs; the
    # next block proposal re-encodes them, so the draft cache over the
    # committed sequence equals a fresh causal pass over it
    w, hp, T, D = _block_seq(K=4, max_new=20)
    trace = OS.greedy_trace(S.oracle_sequence(w, 0, T, None, with_draft=False))
    seq = S.oracle_sequence(w, 0, T, D)
    P = seq.P
    for _ in range(3):
        seq.block_propose(w.vocab - 1)
        i = len(seq.generated)
        seq.verify(trace[i:i + w.K])          # all accepted (a bonus token too)
    seq.block_propose(w.vocab - 1)            # re-encodes the accepted tokens
    n = seq.seq_len
    fresh = S.oracle_sequence(w, 0, T, D)
    toks = [fresh.pending] + list(seq.generated)
    fresh.D.forward(toks, list(range(P, P + len(toks))), fresh.dc)
    for li in range(D.s.layers):
        assert np.allclose(seq.dc.k[li][P:n + 1], fresh.dc.k[li][P:n + 1], rtol=1e-10, atol=1e-12)
        assert np.allclose(seq.dc.v[li][P:n + 1], fresh.dc.v[li][P:n + 1], rtol=1e-10, atol=1e-12)


# --- conditioning on target hidden states -----------------------------------------

def test_conditioning_with_zero_input_weights_is_the_plain_draft():
    w, hp, T, D = _block_seq()
    cond = S.conditioning(w, hp, (0, 1, 1))
    cond.w_in[:] = 0.0
    a = S.oracle_sequence(w, 0, T, D, cond=cond)
    b = S.oracle_sequence(w, 0, T, D)
    for _ in range(2):
        da, za = a.draft_step()
        db, zb = b.draft_step()
        assert np.array_equal(za, zb)
    trace = OS.greedy_trace(S.oracle_sequence(w, 0, T, None, with_draft=False))
    a.verify(trace[:2] + [0, 0])
    b.verify(trace[:2] + [0, 0])
    assert a.feat and set(a.feat) == set(range(a.P, a.seq_len))
    assert np.array_equal(a.draft_step()[1], b.draft_step()[1])


def test_captured_last_layer_reproduces_the_logits():
    # the residual stream after the last layer, normalised and projected on
    # the tied embedding, is the forward pass's own logits
    w, hp, T, D = _block_seq()
    seq = S.oracle_sequence(w, 0, T, None, with_draft=False)
    L = T.s.layers
    T.capture_layers = (L - 1,)
    z = T.forward([seq.pending, 5, 9], [seq.P, seq.P + 1, seq.P + 2], seq.tc)
    T.capture_layers = ()
    h = M.rmsnorm(T.captured[L - 1], T.final_norm(), T.s.rms_eps)
    assert np.allclose(T.lm_head(h), z, rtol=1e-12, atol=1e-12)


def test_features_of_a_verify_equal_sequential_single_row_features():
    # a verify of K+1 rows yields, for each committed row, the feature that
    # one-row verifies of the same tokens yield (the target is causal)
    w, hp, T, D = _block_seq()
    cond = S.conditioning(w, hp, (0, 1, 1))
    trace = OS.greedy_trace(S.oracle_sequence(w, 0, T, None, with_draft=False))
    a = S.oracle_sequence(w, 0, T, None, with_draft=False, cond=cond)
    a.verify(trace[:w.K])                       # all accepted: K+1 committed rows
    b = S.oracle_sequence(w, 0, T, None, with_draft=False, cond=cond)
    for _ in range(w.K + 1):
        b.verify([])
    assert set(a.feat) == set(b.feat)
    for t in a.feat:
        assert np.allclose(a.feat[t], b.feat[t], rtol=1e-9, atol=1e-9)


def test_conditioned_spec_loop_equals_greedy():
    w, hp, T, D = _block_seq()
    cond = S.conditioning(w, hp, (0, 1, 1))
    trace = OS.greedy_trace(S.oracle_sequence(w, 0, T, None, with_draft=False))
    seq = S.oracle_sequence(w, 0, T, D, cond=cond)
    assert OS.spec_loop(seq, lambda sq: sq.propose()) == list(trace)
    seq = S.oracle_sequence(w, 0, T, D, cond=cond)
    assert OS.spec_loop(seq, lambda sq: sq.block_propose(w.vocab - 1)[0]) == list(trace)
