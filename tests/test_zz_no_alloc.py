"""spec_verify_scratch: the verify whose per-pass scratch lives in the library's
static per-device array (no allocation, no graph), checked against
spec_verify on twin contexts.

Two calls in a row on the static array: first a 7B-width one-layer verify of
9 rows over the 3328-token prompt, then the smaller tiny workload (5 rows, 320
tokens).  Each must give spec_verify's logits, greedy tokens, accept length,
commits, lengths and new K/V rows bit for bit (same kernels, same summation
order).  A context whose verify needs more scratch than the array holds is
refused with SPEC_E_CAPACITY and stays usable."""
import numpy as np
import pytest

import workloads as W
from oracle import spec as OS
from tests import _support as S

pytestmark = pytest.mark.gpu


def _pair(w, **kw):
    from paper_2606_31160_amd.harness import Session
    return Session(w, **kw), Session(w, **kw)


def _round(s, drafts, scratch):
    from paper_2606_31160_amd import binding as B
    s.vtok.copy_(s.torch.as_tensor(np.asarray(drafts, dtype=np.int32)).reshape(s.B, -1).to(s.dev))
    fn = B.spec_verify_scratch if scratch else B.spec_verify
    fn(s.ctx, s.vtok.data_ptr(), s.logits.data_ptr())
    s.commit()
    coms, acc, fin = s.committed()
    return s.logits.view(s.torch.int16).cpu().numpy().copy(), coms, acc.copy(), [s.state(b) for b in range(s.B)]


def _same(a, b):
    assert np.array_equal(a[0], b[0]), "logits differ"
    assert a[1] == b[1], (a[1], b[1])
    assert np.array_equal(a[2], b[2])
    assert a[3] == b[3]


def _kv_same(sa, sb, w, P, n):
    for li in range(w.target.layers):
        for which in (0, 1):
            assert np.array_equal(sa.kv(0, 0, li, which, P, n), sb.kv(0, 0, li, which, P, n)), (li, which)


def test_scratch_verify_equals_verify_on_two_calls_then_a_smaller_one():
    # call 1: 7B-width layer, 9 rows, 3328-token prompt (device weights)
    w = W.get("C2").with_(draft=None)
    src = W.DeviceWeights(w)
    ref, scr = _pair(w, source="device", provider=src)
    rng = np.random.default_rng(31)
    for r in range(2):
        drafts = rng.integers(0, w.vocab, size=(1, w.K))
        a = _round(ref, drafts, scratch=False)
        b = _round(scr, drafts, scratch=True)
        _same(a, b)
    P = w.seqs[0].prefix_len
    _kv_same(ref, scr, w, P, 2 * (w.K + 1))
    ref.close()
    scr.close()

    # call 2, smaller input: the tiny workload with its draft, a draft-then-
    # verify round with the draft's own proposals, then explicit proposals
    # whose first tokens are the oracle's greedy tokens (l > 0)
    w = W.get("C1")
    hp = W.HostWeights(w)
    ref, scr = _pair(w, provider=hp)
    from paper_2606_31160_amd import binding as B
    for s, scratch in ((ref, False), (scr, True)):
        s.draft_steps(w.K)
        (B.spec_verify_scratch if scratch else B.spec_verify)(s.ctx, 0, s.logits.data_ptr())
        s.commit()
    la = ref.logits.view(ref.torch.int16).cpu().numpy()
    lb = scr.logits.view(scr.torch.int16).cpu().numpy()
    assert np.array_equal(la, lb)
    assert ref.committed()[0] == scr.committed()[0]
    T, D = S.oracle_decoders(w, hp)
    probe = S.oracle_sequence(w, 0, T, None, with_draft=False)
    trace = OS.greedy_trace(probe, 12)
    n0 = len(ref.committed()[0][0])
    drafts = np.array(trace[n0:n0 + w.K])[None, :]
    a = _round(ref, drafts, scratch=False)
    b = _round(scr, drafts, scratch=True)
    _same(a, b)
    _kv_same(ref, scr, w, w.seqs[0].prefix_len, n0 + w.K + 1)
    assert ref.sync() == 0 and scr.sync() == 0
    ref.close()
    scr.close()


def test_scratch_verify_refuses_a_pass_larger_than_the_array():
    # 16 sequences of the two-frame 3328-token prompt at 7B width with the
    # 152064-token head, 144 rows: the logits staging alone (144 x 152064
    # bf16) exceeds the static array
    from paper_2606_31160_amd import binding as B
    from paper_2606_31160_amd.harness import Session
    c2 = W.get("C2")
    w = c2.with_(draft=None, vocab=152064, seqs=tuple([c2.seqs[0]] * 16), p_accept=tuple([0.75] * 16))
    assert w.batch * (w.K + 1) == 144
    s = Session(w, source="device", provider=W.DeviceWeights(w))
    with pytest.raises(B.SpecError) as e:
        B.spec_verify_scratch(s.ctx, s.vtok.data_ptr(), 0)
    assert e.value.status == 3
    assert "SPEC_SCRATCH_BYTES" in B.spec_last_error(s.ctx)
    # nothing was enqueued and the state is unchanged: a plain verify runs
    st = s.state(0)
    B.spec_verify(s.ctx, s.vtok.data_ptr(), 0)
    s.commit()
    assert s.state(0)["seq_len"] == st["seq_len"] + 1
    assert s.sync() == 0
    s.close()
