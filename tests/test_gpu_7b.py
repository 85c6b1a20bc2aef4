"""GPU parity at the 7B-class shapes (hidden 3584, 28 q / 4 kv heads, head_dim 128,
M-RoPE sections 16/24/24, SwiGLU 18944), in the launch configuration the
benchmark times (batch 1, K = 8, 9 verify rows).

  * one target layer over the 3328-token two-frame prompt, against the oracle
    (logits, greedy tokens, accept length, new K/V rows, position ids);
  * the 2-layer FlatRoPE draft at that width, against the oracle;
  * 4 target layers with the full 152064-token tied head over the 4096-token
    prompt, against the oracle;
  * the full 28-layer verify: the speculative output equals greedy decoding
    bit for bit (a property that holds at any size; the oracle would need
    minutes for 28 layers).
"""
import dataclasses

import numpy as np
import pytest

import workloads as W
from oracle import numerics as ON
from oracle import positions as OP
from oracle import spec as OS
from tests import _support as S

pytestmark = pytest.mark.gpu


# Every test runs on both execution paths of the library: one kernel per
# layer step over the tile-packed weight copy or over the caller's row-major
# weights.
_PATH = {"flags": 0}


@pytest.fixture(autouse=True, params=["packed", "rowmajor"])
def path(request):
    _PATH["flags"] = S.PATH_FLAGS[request.param]
    yield request.param


def _session(w, **kw):
    from paper_2606_31160_amd.harness import Session
    kw["flags"] = kw.get("flags", 0) | _PATH["flags"]
    return Session(w, **kw)


def _blocks(w, b=0):
    return [(x.start, x.t, x.h, x.w) for x in w.seqs[b].blocks]


@pytest.fixture(scope="module")
def c2():
    w = W.get("C2").with_(draft=None)
    hp = W.HostWeights(w)
    T, _ = S.oracle_decoders(w, hp, cache_weights=True)
    return w, hp, T


@pytest.mark.parametrize("K", [8, 15])
def test_one_layer_verify_against_oracle(c2, K):
    # K = 15: 16 verify rows, a full MFMA row block (every row of the packed
    # kernels' operands live, the streamed down-projection input at 16 rows)
    w, hp, T = c2
    w = w.with_(K=K)
    s = _session(w, provider=hp)
    P = w.seqs[0].prefix_len
    L = P + w.K + 1
    assert np.array_equal(s.positions(0, L), OP.target_positions(L, _blocks(w)))
    rng = np.random.default_rng(21)
    drafts = rng.integers(0, w.vocab, size=w.K).astype(np.int32)
    seq = S.oracle_sequence(w, 0, T, None, with_draft=False)
    # make the first three drafts the oracle's own greedy tokens so l > 0 is exercised
    probe = S.oracle_sequence(w, 0, T, None, with_draft=False)
    greedy = OS.greedy_trace(probe, 3)
    drafts[:3] = greedy
    s.verify(drafts[None, :], logits=True)
    s.commit()
    ref = seq.verify(drafts)
    gl = s.logits[0].float().cpu().numpy()
    for j in range(w.K + 1):
        assert S.normwise_err(gl[j], ref.logits[j]) <= S.LOGIT_RTOL, j
    coms, acc, fin = s.committed()
    l = int(acc[0])
    pinned = S.margin(ref.logits) > S.MARGIN
    if pinned[:ref.accept_len + 1].all():
        assert l == ref.accept_len and coms[0] == ref.committed
    assert coms[0][:l] == list(drafts[:l])
    for li in range(w.target.layers):
        for which, ref_c in ((0, seq.tc.k[li]), (1, seq.tc.v[li])):
            got = ON.decode(s.kv(0, 0, li, which, P, w.K + 1))
            assert S.normwise_err(got, ref_c[P:P + w.K + 1]) <= S.LOGIT_RTOL
    s.close()


def test_two_layer_flatrope_draft_against_oracle():
    """Draft steps at 7B width; tokens compared while the oracle's rows are
    pinned, the K/V rows each step writes compared for every step taken."""
    base = W.get("C2")
    w = base.with_(target=dataclasses.replace(base.target, layers=1), seed=1)
    hp = W.HostWeights(w)
    T, D = S.oracle_decoders(w, hp, cache_weights=True)
    s = _session(w, provider=hp)
    seq = S.oracle_sequence(w, 0, T, D)
    P = w.seqs[0].prefix_len
    steps = 0
    for step in range(4):
        s.draft_step()
        d_ref, z_ref = seq.draft_step()
        steps += 1
        pinned = S.check_argmax_rows([int(s.dtok[0, step].item())], z_ref[None, :])
        if not pinned[0]:
            break
    assert steps >= 2
    n = P + steps
    assert s.state(0)["draft_len"] == n == seq.draft_len
    for li in range(w.draft.layers):
        for which, ref_c in ((0, seq.dc.k[li]), (1, seq.dc.v[li])):
            got = ON.decode(s.kv(0, 1, li, which, P, steps))
            assert S.normwise_err(got, ref_c[P:n]) <= S.LOGIT_RTOL
    s.close()


def test_four_layers_with_full_vocabulary_against_oracle():
    base = W.get("C3")
    w = base.with_(target=dataclasses.replace(base.target, layers=4), draft=None)
    src = W.DeviceWeights(w)
    s = _session(w, source="device", provider=src)
    T, _ = S.oracle_decoders(w, src, cache_weights=False)
    seq = S.oracle_sequence(w, 0, T, None, kv=S.device_kv, with_draft=False)
    rng = np.random.default_rng(31)
    drafts = rng.integers(0, w.vocab, size=w.K).astype(np.int32)
    s.verify(drafts[None, :], logits=True)
    s.commit()
    ref = seq.verify(drafts)
    gl = s.logits[0].float().cpu().numpy()
    for j in range(w.K + 1):
        assert S.normwise_err(gl[j], ref.logits[j]) <= S.LOGIT_RTOL, j
    coms, acc, fin = s.committed()
    l = int(acc[0])
    assert coms[0][:l] == list(drafts[:l])
    S.check_argmax_rows(coms[0][l:l + 1], ref.logits[l:l + 1])
    s.close()


def test_full_verify_speculative_equals_greedy():
    w = W.get("C3").with_(max_new_tokens=40)
    src = W.DeviceWeights(w)
    ar = _session(w, source="device", provider=src, K=0, with_draft=False)
    trace = []
    while True:
        ar.verify(None)
        ar.commit()
        coms, acc, fin = ar.committed()
        trace += [int(t) for t in coms[0]]
        if fin[0]:
            break
    ar.close()
    assert len(trace) == w.max_new_tokens
    s = _session(w, source="device", provider=src)
    synth = W.DraftSynth(w, 0)
    out, accs = [], []
    while True:
        for _ in range(w.K):
            s.draft_step()
        s.verify(synth.propose(np.array(trace[len(out):]), w.K)[None, :])
        s.commit()
        coms, acc, fin = s.committed()
        out += [int(t) for t in coms[0]]
        accs.append(int(acc[0]))
        if fin[0]:
            break
    assert out == trace
    assert max(accs) >= 2
    st = s.state(0)
    assert st["seq_len"] == w.seqs[0].prefix_len + len(trace)
    s.close()
