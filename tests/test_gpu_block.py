"""GPU parity of the single-forward block proposal (SPEC_FLAG_BLOCK_DRAFT; the
block-diffusion draft family of Sec. 4.1, Eq. propose): rows [pending,
MASK x K] through the draft, the pending row causal and every MASK row seeing
the prefix and the whole block, MASK row i proposing d_i; accepted proposals
are re-encoded causally in the next round.

  * tiny workload, packed and row-major paths: the K proposals against the
    oracle's block proposal (argmax on pinned rows), the pending row's draft
    K/V, and a second round after accepted proposals (the catch-up);
  * the speculative loop with block proposals commits exactly greedy decoding
    (tiny, and 16 tiny scenes whose 80-row passes run on the batched GEMM);
  * the 2-layer draft at 7B width over the 3328-token prompt against the oracle;
  * three scenes at the paper backbone's width with K = 16: the speculative loop
    with block proposals commits exactly greedy decoding.
"""
import numpy as np
import pytest

import workloads as W
from oracle import numerics as ON
from oracle import spec as OS
from tests import _support as S

pytestmark = pytest.mark.gpu


def _session(w, **kw):
    from paper_2606_31160_amd import binding as B
    from paper_2606_31160_amd.harness import Session
    kw["flags"] = kw.get("flags", 0) | B.SPEC_FLAG_BLOCK_DRAFT
    return Session(w, **kw)


def _loop(s):
    outs = [[] for _ in range(s.B)]
    done = [False] * s.B
    for _ in range(200):
        s.draft_steps(s.K)
        s.verify(None)
        s.commit()
        coms, acc, fin = s.committed()
        for b in range(s.B):
            if not done[b]:
                outs[b] += [int(t) for t in coms[b]]
                done[b] = bool(fin[b])
        if all(done):
            return outs
    raise AssertionError("loop did not finish")


@pytest.fixture(scope="module")
def c1():
    w = W.get("C1")
    hp = W.HostWeights(w)
    T, D = S.oracle_decoders(w, hp)
    trace = OS.greedy_trace(S.oracle_sequence(w, 0, T, None, with_draft=False))
    return w, hp, T, D, trace


@pytest.mark.parametrize("path", ["packed", "rowmajor"])
def test_block_proposals_against_oracle(c1, path):
    w, hp, T, D = c1[:4]
    trace = c1[4]
    mask = w.vocab - 1
    s = _session(w, provider=hp, flags=S.PATH_FLAGS[path])
    seq = S.oracle_sequence(w, 0, T, D)
    P = w.seqs[0].prefix_len
    for rnd in range(2):
        s.draft_steps(w.K)
        gpu = s.dtok[0].cpu().numpy()
        n = seq.seq_len
        props, z = seq.block_propose(mask)
        pinned = S.check_argmax_rows(gpu, z)
        st = s.state(0)
        assert st["draft_len"] == n + 1 and st["seq_len"] == n
        # the pending row's draft K/V (a real input) against the oracle's
        for which, ref in ((0, seq.dc.k[0]), (1, seq.dc.v[0])):
            got = ON.decode(s.kv(0, 1, 0, which, n, 1))
            assert S.normwise_err(got, ref[n:n + 1]) <= S.LOGIT_RTOL
        if not pinned.all():
            pytest.skip("an unpinned proposal: histories may diverge")
        # verify the greedy continuation so that every proposal of the next
        # round's catch-up is an accepted one
        i = len(seq.generated)
        d = np.array(trace[i:i + w.K], dtype=np.int32)
        if len(d) < w.K:
            break
        s.verify(d[None, :])
        s.commit()
        seq.verify(d)
        coms, acc, fin = s.committed()
        assert coms[0] == seq.committed[-len(coms[0]):]
    s.close()


def test_block_spec_loop_equals_greedy(c1):
    w, hp = c1[:2]
    spec = _loop(_session(w, provider=hp))[0]
    from paper_2606_31160_amd.harness import Session
    ar = Session(w, provider=hp, K=0, with_draft=False)
    out = []
    while True:
        ar.verify(None)
        ar.commit()
        coms, acc, fin = ar.committed()
        out += [int(t) for t in coms[0]]
        if fin[0]:
            break
    assert spec == out and len(spec) == w.max_new_tokens


def test_block_sixteen_scenes_gemm_equals_greedy():
    # 80-row passes run on the batched GEMM, whose sums are grouped differently
    # from smaller passes, so the greedy reference is taken at the same pass
    # shape: rounds whose drafts are random commit only greedy tokens
    base = W.get("C1")
    lens = np.random.default_rng(3).integers(430, 701, size=16)
    w = base.with_(seqs=tuple(W.c5_layout(int(p)) for p in lens), p_accept=tuple([0.8] * 16))
    assert w.batch * (w.K + 1) == 80
    hp = W.HostWeights(w)
    from paper_2606_31160_amd.harness import Session
    ref = Session(w, provider=hp, page_seed=21)
    rng = np.random.default_rng(4)
    outs = [[] for _ in range(w.batch)]
    done = [False] * w.batch
    while not all(done):
        ref.verify(rng.integers(0, w.vocab, size=(w.batch, w.K)).astype(np.int32))
        ref.commit()
        coms, acc, fin = ref.committed()
        for b in range(w.batch):
            if not done[b]:
                outs[b] += [int(t) for t in coms[b]]
                done[b] = bool(fin[b])
    ref.close()
    s = _session(w, provider=hp, page_seed=21)
    spec = _loop(s)
    s.close()
    assert spec == outs


def test_block_paper_width_three_scenes_equals_greedy():
    """Hidden 4096, 32/8 heads, K = 16, three scenes: every pass (verify,
    catch-up and block) has 51 rows and runs on the batched GEMM with q/k/v in
    one split.  The greedy reference is taken at the verify's pass shape, as
    above."""
    import dataclasses
    base = W.get("C6")
    w = base.with_(target=dataclasses.replace(base.target, layers=2), vocab=2048, max_new_tokens=24,
                   seqs=tuple(W.c5_layout(p) for p in (1100, 1400, 1700)), p_accept=(0.8, 0.8, 0.8))
    src = W.DeviceWeights(w)
    from paper_2606_31160_amd.harness import Session
    ref = Session(w, source="device", provider=src, page_seed=21)
    rng = np.random.default_rng(5)
    outs = [[] for _ in range(w.batch)]
    done = [False] * w.batch
    while not all(done):
        ref.verify(rng.integers(0, w.vocab, size=(w.batch, w.K)).astype(np.int32))
        ref.commit()
        coms, acc, fin = ref.committed()
        for b in range(w.batch):
            if not done[b]:
                outs[b] += [int(t) for t in coms[b]]
                done[b] = bool(fin[b])
    ref.close()
    assert all(len(o) == w.max_new_tokens for o in outs)
    s = _session(w, source="device", provider=src, page_seed=21)
    spec = _loop(s)
    s.close()
    assert spec == outs


def test_block_proposal_7b_width_draft():
    w = W.get("C2")
    src = W.DeviceWeights(w)
    T, D = S.oracle_decoders(w, src, cache_weights=True)
    s = _session(w, source="device", provider=src)
    s.draft_steps(w.K)
    gpu = s.dtok[0].cpu().numpy()
    s.close()
    seq = S.oracle_sequence(w, 0, T, D, kv=S.device_kv)
    props, z = seq.block_propose(w.vocab - 1)
    S.check_argmax_rows(gpu, z)
