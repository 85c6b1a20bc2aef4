"""Pins for the attention-budget readout (Sec. 4.2, Table attn-budget): closed
forms (uniform scores, a single dominant key), the library entropy of a chosen
distribution, the attention probabilities recovered through attend() with
one-hot values, and the slot classes of a prompt layout."""
import math

import numpy as np
import scipy.stats

import workloads as W
from oracle import budget as B
from oracle import model as M


def _classes(n_vis, n_traj, n_gen):
    return np.array([B.VISUAL] * n_vis + [B.TRAJ_TEXT] * n_traj + [B.GENERATED] * n_gen, dtype=np.int8)


def test_uniform_scores_give_class_fractions_and_unit_entropy():
    # q = 0: every visible key scores 0, so each class holds n_c / n of the mass
    # and the renormalised trajectory distribution is uniform (entropy 1).
    cls = _classes(30, 7, 5)
    q = np.zeros((3, 4, 16))
    kc = np.random.default_rng(0).standard_normal((42, 2, 16))
    slots = [41, 36, 20]
    r = B.budget(q, kc, slots, cls)
    for i, s in enumerate(slots):
        n = s + 1
        c = cls[:n]
        want = [np.sum(c == 0) / n, np.sum(c == 1) / n, np.sum(c == 2) / n]
        assert np.allclose(r[i, :, :3], want, rtol=1e-14, atol=0)
        assert np.allclose(r[i, :, 3], 1.0, rtol=1e-14) if np.sum(c == 1) > 1 else np.all(r[i, :, 3] == 0)


def test_single_dominant_key():
    # q along key j with a huge score: all mass goes to j's class; when j is a
    # trajectory slot the entropy within the class tends to 0, otherwise the
    # (tiny) trajectory mass is spread evenly over its equal-score slots.
    D = 8
    cls = _classes(4, 5, 3)
    kc = np.zeros((12, 1, D))
    for j, c in ((6, B.TRAJ_TEXT), (1, B.VISUAL), (10, B.GENERATED)):
        kc[:] = 0.0
        kc[j, 0, 0] = 1.0
        q = np.zeros((1, 1, D))
        q[0, 0, 0] = 400.0 * math.sqrt(D)
        r = B.budget(q, kc, [11], cls)[0, 0]
        assert abs(r[c] - 1.0) < 1e-12 and abs(sum(r[:3]) - 1.0) < 1e-12
        assert r[3] < 1e-12 if c == B.TRAJ_TEXT else abs(r[3] - 1.0) < 1e-12


def test_entropy_matches_library_on_chosen_distribution():
    # scores log(w) give p proportional to w; the trajectory entropy is the
    # library entropy of w restricted to class 1, over ln(n_1).
    rng = np.random.default_rng(1)
    n = 20
    cls = rng.integers(0, 3, size=n).astype(np.int8)
    cls[:3] = B.TRAJ_TEXT
    w = rng.uniform(0.05, 3.0, size=n)
    p = w / w.sum()
    r = B.row_budget(p, cls)
    sel = w[cls == B.TRAJ_TEXT]
    assert abs(r[3] - scipy.stats.entropy(sel) / math.log(sel.size)) < 1e-13
    for c in range(3):
        assert abs(r[c] - w[cls == c].sum() / w.sum()) < 1e-13
    # a single trajectory slot (or none) has no spread
    assert B.row_budget(p[:5], np.array([1, 0, 2, 0, 2], dtype=np.int8))[3] == 0.0
    assert B.row_budget(p[:3], np.array([0, 2, 2], dtype=np.int8))[1] == 0.0


def test_probabilities_agree_with_attention_through_one_hot_values():
    # attend() with value k equal to the k-th unit vector returns the attention
    # probabilities themselves (GQA grouping, causal mask, 1/sqrt(D) included).
    rng = np.random.default_rng(2)
    cap, nq, nkv, D = 24, 6, 2, 16
    q = rng.standard_normal((3, nq, D)) * 2.0
    kc = rng.standard_normal((cap, nkv, D))
    slots = [23, 15, 9]
    cls = rng.integers(0, 3, size=cap).astype(np.int8)
    vc = np.zeros((cap, nkv, cap))
    for k in range(cap):
        vc[k, :, k] = 1.0
    # attend() takes the value width from q's last axis: pad q and keys with zeros
    qp = np.concatenate([q, np.zeros((3, nq, cap - D))], axis=-1)
    kp = np.concatenate([kc, np.zeros((cap, nkv, cap - D))], axis=-1)
    p = M.attend(qp * math.sqrt(cap / D), kp, vc, slots)     # same scores as width D
    r = B.budget(q, kc, slots, cls)
    for i, s in enumerate(slots):
        for h in range(nq):
            ph = p[i, h, :s + 1]
            assert abs(ph.sum() - 1.0) < 1e-12 and np.all(p[i, h, s + 1:] == 0)
            for c in range(3):
                assert abs(r[i, h, c] - ph[cls[:s + 1] == c].sum()) < 1e-12
            sel = ph[cls[:s + 1] == B.TRAJ_TEXT]
            if sel.size > 1:
                assert abs(r[i, h, 3] - scipy.stats.entropy(sel) / math.log(sel.size)) < 1e-12


def test_slot_classes_of_a_prompt_layout():
    w = W.get("C1")
    lay = w.seqs[0]
    blocks = [(b.start, b.t, b.h, b.w) for b in lay.blocks]
    total = lay.prefix_len + 9
    c = B.slot_classes(lay.prefix_len, blocks, total)
    assert np.sum(c == B.VISUAL) == sum(b.ntok for b in lay.blocks)
    assert np.sum(c == B.GENERATED) == 9
    for b in lay.blocks:
        assert np.all(c[b.start:b.start + b.ntok] == B.VISUAL)
    assert np.sum(c == B.TRAJ_TEXT) == lay.prefix_len - sum(b.ntok for b in lay.blocks)


def test_forward_readout_layer_leaves_logits_unchanged():
    import dataclasses
    from tests import _support as S
    base = W.get("C1")
    lay = W.SeqLayout(40, (W.VisionBlock(0, 1, 4, 6),))
    w = base.with_(target=dataclasses.replace(base.target, layers=2), vocab=256, seqs=(lay,))
    hp = W.HostWeights(w)
    T, _ = S.oracle_decoders(w, hp, cache_weights=True)
    seq_a = S.oracle_sequence(w, 0, T, None, with_draft=False)
    toks = [5, 17, 3]
    za = seq_a.T.forward(toks, [40, 41, 42], seq_a.tc)
    T.readout_layer = 1
    T.readout_classes = B.slot_classes(40, [(0, 1, 4, 6)], seq_a.tc.cap)
    seq_b = S.oracle_sequence(w, 0, T, None, with_draft=False)
    zb = seq_b.T.forward(toks, [40, 41, 42], seq_b.tc)
    assert np.array_equal(za, zb)
    r = T.readout
    assert r.shape == (3, w.target.q_heads, 4)
    assert np.allclose(r[:, :, :3].sum(-1), 1.0, rtol=1e-12)
    assert np.all((r[:, :, 3] >= 0) & (r[:, :, 3] <= 1 + 1e-12))
    assert np.all(r[:, :, 2] > 0)        # every new row sees at least itself
