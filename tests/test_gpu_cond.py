"""GPU parity of the draft conditioned on target hidden states (SPEC_FLAG_COND;
Sec. 4.1, fused EAGLE-3 style as in Sec. 5): each verify keeps the target's
residual stream after three chosen layers, the committed rows' fused
features f = W_fuse [h_a; h_b; h_c] become per-slot features, and a draft row
at slot t takes the input e + W_in [e; f(t-1)].

  * tiny workload, packed and row-major paths: the features of the committed
    slots (within 2e-2 normwise) and the draft's proposals (argmax on pinned
    rows) against the oracle over two rounds, with the K-step chain and with
    the block proposal;
  * the speculative loop with a conditioned draft commits exactly greedy
    decoding;
  * a 3-layer tiny target capturing three distinct layers (0, 1, 2);
  * the cross-attention form (SPEC_FLAG_COND_CROSS, Sec. 4.1): proposals,
    features and the draft's layer-0 context K/V against the oracle on both
    paths and at 7B width, greedy equivalence;
  * one target layer at 7B width with the 2-layer draft: features and
    proposals against the oracle.
"""
import numpy as np
import pytest

import workloads as W
from oracle import numerics as ON
from oracle import spec as OS
from tests import _support as S

pytestmark = pytest.mark.gpu

LAYERS_TINY = (0, 1, 1)


def _session(w, **kw):
    from paper_2606_31160_amd.harness import Session
    return Session(w, **kw)


@pytest.fixture(scope="module")
def c1():
    w = W.get("C1")
    hp = W.HostWeights(w)
    T, D = S.oracle_decoders(w, hp)
    trace = OS.greedy_trace(S.oracle_sequence(w, 0, T, None, with_draft=False))
    return w, hp, T, D, trace


def _rounds(w, s, seq, trace, block, rounds=2, cross=False):
    """Drive GPU and oracle through the same rounds (greedy drafts, so that
    proposals get accepted); check proposals and features (and, for the
    cross-attention form, the draft's layer-0 context K/V of the verified
    slots)."""
    P = w.seqs[0].prefix_len
    same_history = True   # proposals are compared while both sides' draft histories agree
    for _ in range(rounds):
        s.draft_steps(w.K)
        gpu = s.dtok[0].cpu().numpy()
        if block:
            props, z = seq.block_propose(w.vocab - 1)
        else:
            rec = []
            for _ in range(w.K):
                d, zz = seq.draft_step()
                rec.append(zz)
            props, z = seq.props, np.stack(rec)
        if same_history:
            pinned = S.check_argmax_rows(gpu, z)
            same_history = bool(pinned.all()) and list(gpu) == list(props)
        # the features come from the verify rows only (the drafts verified
        # are the greedy continuation), so they are compared in every round
        i = len(seq.generated)
        d = np.array(trace[i:i + w.K], dtype=np.int32)
        if len(d) < w.K:
            break
        s.verify(d[None, :])
        s.commit()
        seq.verify(d)
        coms, acc, fin = s.committed()
        assert coms[0] == seq.committed[-len(coms[0]):]
        n = seq.seq_len
        got = ON.decode(s.feature(0, P, n - P))
        ref = np.stack([seq.feat[t] for t in range(P, n)])
        for r in range(n - P):
            assert S.normwise_err(got[r], ref[r]) <= S.LOGIT_RTOL, r
        if cross:
            for which, ref_c in ((0, seq.dc.k[0]), (1, seq.dc.v[0])):
                ctx = ON.decode(s.kv(0, 1, 0, which, P, n - P))
                for r in range(n - P):
                    assert S.normwise_err(ctx[r], ref_c[P + r]) <= S.LOGIT_RTOL, (which, r)


@pytest.mark.parametrize("block", [False, True])
@pytest.mark.parametrize("path", ["packed", "rowmajor"])
def test_conditioned_draft_against_oracle(c1, path, block):
    from paper_2606_31160_amd import binding as B
    w, hp, T, D, trace = c1
    flags = S.PATH_FLAGS[path] | (B.SPEC_FLAG_BLOCK_DRAFT if block else 0)
    s = _session(w, provider=hp, flags=flags, cond_layers=LAYERS_TINY)
    seq = S.oracle_sequence(w, 0, T, D, cond=S.conditioning(w, hp, LAYERS_TINY))
    _rounds(w, s, seq, trace, block)
    s.close()


def test_conditioned_draft_three_distinct_target_layers():
    # a 3-layer tiny target capturing layers (0, 1, 2): every column block of
    # the fused operand comes from a different layer, so a swapped block or a
    # layer taken twice changes the features
    import dataclasses
    base = W.get("C1")
    w = base.with_(target=dataclasses.replace(base.target, layers=3))
    hp = W.HostWeights(w)
    T, D = S.oracle_decoders(w, hp)
    trace = OS.greedy_trace(S.oracle_sequence(w, 0, T, None, with_draft=False))
    s = _session(w, provider=hp, cond_layers=(0, 1, 2))
    seq = S.oracle_sequence(w, 0, T, D, cond=S.conditioning(w, hp, (0, 1, 2)))
    _rounds(w, s, seq, trace, block=False)
    s.close()


@pytest.mark.parametrize("path", ["packed", "rowmajor"])
def test_cross_attention_conditioned_draft_against_oracle(c1, path):
    # Sec. 4.1's form: the fused features are the draft's layer-0
    # cross-attention context; proposals, features and the context K/V of
    # every verified slot against the oracle over three rounds
    w, hp, T, D, trace = c1
    s = _session(w, provider=hp, flags=S.PATH_FLAGS[path], cond_layers=LAYERS_TINY, cond_cross=True)
    seq = S.oracle_sequence(w, 0, T, D, cond=S.conditioning(w, hp, LAYERS_TINY, cross=True))
    _rounds(w, s, seq, trace, block=False, rounds=3, cross=True)
    s.close()


def test_cross_attention_spec_loop_equals_greedy(c1):
    w, hp = c1[:2]
    s = _session(w, provider=hp, cond_layers=LAYERS_TINY, cond_cross=True)
    out = []
    while True:
        s.draft_steps(w.K)
        s.verify(None)
        s.commit()
        coms, acc, fin = s.committed()
        out += [int(t) for t in coms[0]]
        if fin[0]:
            break
    s.close()
    ar = _session(w, provider=hp, K=0, with_draft=False)
    ref = []
    while True:
        ar.verify(None)
        ar.commit()
        coms, acc, fin = ar.committed()
        ref += [int(t) for t in coms[0]]
        if fin[0]:
            break
    assert out == ref and len(out) == w.max_new_tokens


def test_conditioned_spec_loop_equals_greedy(c1):
    w, hp = c1[:2]
    s = _session(w, provider=hp, cond_layers=LAYERS_TINY)
    out = []
    while True:
        s.draft_steps(w.K)
        s.verify(None)
        s.commit()
        coms, acc, fin = s.committed()
        out += [int(t) for t in coms[0]]
        if fin[0]:
            break
    s.close()
    ar = _session(w, provider=hp, K=0, with_draft=False)
    ref = []
    while True:
        ar.verify(None)
        ar.commit()
        coms, acc, fin = ar.committed()
        ref += [int(t) for t in coms[0]]
        if fin[0]:
            break
    assert out == ref and len(out) == w.max_new_tokens


def test_cross_attention_conditioned_draft_7b_width():
    w = W.get("C2")
    src = W.DeviceWeights(w)
    T, D = S.oracle_decoders(w, src, cache_weights=True)
    trace = OS.greedy_trace(S.oracle_sequence(w, 0, T, None, kv=S.device_kv, with_draft=False), 2 * w.K + 4)
    s = _session(w, source="device", provider=src, cond_layers=(0, 0, 0), cond_cross=True)
    seq = S.oracle_sequence(w, 0, T, D, kv=S.device_kv, cond=S.conditioning(w, src, (0, 0, 0), cross=True))
    _rounds(w, s, seq, trace, block=False, rounds=2, cross=True)
    s.close()


def test_conditioned_draft_7b_width():
    w = W.get("C2")
    src = W.DeviceWeights(w)
    T, D = S.oracle_decoders(w, src, cache_weights=True)
    trace = OS.greedy_trace(S.oracle_sequence(w, 0, T, None, kv=S.device_kv, with_draft=False), 2 * w.K + 4)
    s = _session(w, source="device", provider=src, cond_layers=(0, 0, 0))
    seq = S.oracle_sequence(w, 0, T, D, kv=S.device_kv, cond=S.conditioning(w, src, (0, 0, 0)))
    _rounds(w, s, seq, trace, block=False, rounds=2)
    s.close()
