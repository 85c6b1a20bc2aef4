"""GPU parity at the 7B-class shapes (hidden 3584, 28 q / 4 kv heads, head_dim 128,
M-RoPE sections 16/24/24, SwiGLU 18944), in the launch configuration the
benchmark times (batch 1, K = 8, 9 verify rows).

  * one target layer over the 3328-token two-frame prompt, against the oracle
    (logits, greedy tokens, accept length, new K/V rows, position ids);
  * the same layer with two sequences (18 rows: the two-row-block GEMV, and
    on the row-major path the GEMM's k-split q/k/v route), against the oracle;
  * the 2-layer FlatRoPE draft at that width, against the oracle;
  * 4 target layers with the full 152064-token tied head over the 4096-token
    prompt, against the oracle (l = 2 and the bonus token bit for bit);
  * the full 28-layer verify over the 4096-token prompt against the oracle
    (logits of every row, l and commits bit for bit, first and last layers'
    new K/V rows);
  * the full 28-layer speculative loop equals greedy decoding bit for bit.

Wherever l and the committed tokens are compared, the pending token is
reseeded until the oracle's rows 0..l are pinned, and that is asserted.
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
    # kernels' operands live, the streamed down-projection input at 16 rows).
    # The pending token is reseeded until the oracle's first four greedy rows
    # are pinned; the drafts copy three greedy tokens, so l = 3 is asserted
    # bit for bit together with the bonus token.
    w, hp, T = c2
    w = w.with_(K=K)
    pend, drafts, trace, _ = S.pinned_greedy_drafts(w, 0, T, k=3, seed=21)
    s = _session(w, provider=hp, pending_tokens=[pend])
    P = w.seqs[0].prefix_len
    L = P + w.K + 1
    assert np.array_equal(s.positions(0, L), OP.target_positions(L, _blocks(w)))
    seq = S.oracle_sequence(w, 0, T, None, with_draft=False, pending=pend)
    s.verify(drafts[None, :], logits=True)
    s.commit()
    ref = seq.verify(drafts)
    gl = s.logits[0].float().cpu().numpy()
    for j in range(w.K + 1):
        assert S.normwise_err(gl[j], ref.logits[j]) <= S.LOGIT_RTOL, j
    coms, acc, fin = s.committed()
    S.assert_verify_matches(ref, drafts, coms[0], acc[0], k=3)
    assert coms[0] == trace
    st = s.state(0)
    assert st["seq_len"] == P + 4 and st["pending"] == trace[3]
    for li in range(w.target.layers):
        for which, ref_c in ((0, seq.tc.k[li]), (1, seq.tc.v[li])):
            got = ON.decode(s.kv(0, 0, li, which, P, w.K + 1))
            assert S.normwise_err(got, ref_c[P:P + w.K + 1]) <= S.LOGIT_RTOL
    s.close()


def test_one_layer_two_sequences_18_rows_against_oracle(c2, path):
    # batch 2, K = 8: 18 rows per pass.  Packed: the two-row-block GEMV.
    # Row-major: 18 rows of a 3584-wide input do not fit the thin GEMV's LDS,
    # so the pass runs on the batched GEMM, whose q/k/v launch would cover
    # too few CUs in one split and takes the k-split route (partial sums, then
    # the rotary and cache-append finish).  Each sequence's pending token is
    # reseeded until its first three greedy rows are pinned (l = 2 each).
    w, hp, T = c2
    w = w.with_(seqs=(w.seqs[0], w.seqs[0]), p_accept=(0.75, 0.75))
    assert w.batch * (w.K + 1) == 18
    picks = [S.pinned_greedy_drafts(w, b, T, k=2, seed=31 + b) for b in range(2)]
    s = _session(w, provider=hp, pending_tokens=[p[0] for p in picks])
    P = w.seqs[0].prefix_len
    drafts = np.stack([p[1] for p in picks])
    s.verify(drafts, logits=True)
    s.commit()
    coms, acc, fin = s.committed()
    gl = s.logits.float().cpu().numpy()
    for b in range(2):
        seq = S.oracle_sequence(w, b, T, None, with_draft=False, pending=picks[b][0])
        ref = seq.verify(drafts[b])
        for j in range(w.K + 1):
            assert S.normwise_err(gl[b, j], ref.logits[j]) <= S.LOGIT_RTOL, (b, j)
        S.assert_verify_matches(ref, drafts[b], coms[b], acc[b], k=2)
        for which, ref_c in ((0, seq.tc.k[0]), (1, seq.tc.v[0])):
            got = ON.decode(s.kv(b, 0, 0, which, P, w.K + 1))
            assert S.normwise_err(got, ref_c[P:P + w.K + 1]) <= S.LOGIT_RTOL, (b, which)
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
    # full 152064-token head: the pending token is reseeded until the oracle's
    # first three greedy rows are pinned, so l = 2 and the bonus are asserted
    base = W.get("C3")
    w = base.with_(target=dataclasses.replace(base.target, layers=4), draft=None)
    src = W.DeviceWeights(w)
    T, _ = S.oracle_decoders(w, src, cache_weights=True)
    pend, drafts, trace, _ = S.pinned_greedy_drafts(w, 0, T, k=2, kv=S.device_kv, seed=31)
    s = _session(w, source="device", provider=src, pending_tokens=[pend])
    seq = S.oracle_sequence(w, 0, T, None, kv=S.device_kv, with_draft=False, pending=pend)
    s.verify(drafts[None, :], logits=True)
    s.commit()
    ref = seq.verify(drafts)
    gl = s.logits[0].float().cpu().numpy()
    for j in range(w.K + 1):
        assert S.normwise_err(gl[j], ref.logits[j]) <= S.LOGIT_RTOL, j
    coms, acc, fin = s.committed()
    S.assert_verify_matches(ref, drafts, coms[0], acc[0], k=2)
    assert coms[0] == trace
    s.close()


@pytest.fixture(scope="module")
def c3_oracle():
    """The oracle's verify of the 28-layer workload with random drafts, for a
    pending token whose row 0 is pinned (shared by both execution paths).

    Tolerance at this depth.  Any implementation that stores activations in
    bf16 (the projections' inputs, q/k/v and the KV cache, the attention and
    SwiGLU outputs) departs from exact arithmetic by the rounding noise of
    that format, and through 28 layers this noise alone exceeds 2e-2: the
    oracle's own mirror mode (bf16 at those points, float64 elsewhere) differs
    from the plain float64 oracle by d_fmt ~ 2.7e-2 on these rows.  (Rounding
    flips make it chaotic: a 1e-7 change of the input moves the mirror
    oracle's logits by ~2.8e-2, the plain oracle's by 7.6e-7.)  So the bar
    here is tau = max(2e-2, 1.5 d_fmt), computed from the oracle in this test,
    and a row is pinned when its top-1/top-2 margin exceeds tau."""
    import psutil
    w = W.get("C3").with_(draft=None)
    src = W.DeviceWeights(w)
    # the float64 layer cache (about 57 GB) only where the host has room
    big = psutil.virtual_memory().available > 150 * 2**30
    T, _ = S.oracle_decoders(w, src, cache_weights=big)
    rng = np.random.default_rng(41)
    drafts = rng.integers(0, w.vocab, size=w.K).astype(np.int32)
    pend, ref, seq, tau, _ = S.deep_verify_reference(w, 0, T, drafts, kv=S.device_kv)
    P = w.seqs[0].prefix_len
    kv = {(li, which): c[P:P + w.K + 1].copy() for li in (0, w.target.layers - 1)
          for which, c in ((0, seq.tc.k[li]), (1, seq.tc.v[li]))}
    return w, src, pend, drafts, ref, kv, tau


def test_full_28_layer_verify_against_oracle(c3_oracle):
    """The timed verify itself: 28 layers, the 152064-token head, the
    4096-token prompt, 9 rows, against the plain float64 oracle.  Logits of
    every row within tau (see c3_oracle), l and the committed tokens bit for
    bit (the pending token is reseeded until the oracle's row 0 is pinned at
    tau), the first layer's new K/V rows within 2e-2 and the last layer's
    within tau."""
    w, src, pend, drafts, ref, kv, tau = c3_oracle
    s = _session(w, source="device", provider=src, pending_tokens=[pend])
    s.verify(drafts[None, :], logits=True)
    s.commit()
    gl = s.logits[0].float().cpu().numpy()
    errs = [S.normwise_err(gl[j], ref.logits[j]) for j in range(w.K + 1)]
    print(f"28 layers: logit error max {max(errs):.3e} (tau {tau:.3e})", flush=True)
    for j in range(w.K + 1):
        assert errs[j] <= tau, (j, errs[j], tau)
    coms, acc, fin = s.committed()
    assert S.margin(ref.logits)[0] > tau
    assert int(acc[0]) == ref.accept_len == 0
    assert list(coms[0]) == list(ref.committed)
    P = w.seqs[0].prefix_len
    for (li, which), want in kv.items():
        got = ON.decode(s.kv(0, 0, li, which, P, w.K + 1))
        bar = S.LOGIT_RTOL if li == 0 else tau
        assert S.normwise_err(got, want) <= bar, (li, which)
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
