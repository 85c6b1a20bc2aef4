"""GPU parity of passes over many sequences at once: more than 64 rows per
pass run on the batched-row GEMM, with caches in shuffled KV pages.

  * 16 tiny scenes of different prompt lengths, K = 4 (80 rows): one verify's
    logits, accept lengths, commits and new K/V rows against the oracle, then
    the speculative loop to the token budget, every committed token checked
    against the oracle's logits over the sequence's own history;
  * 8 tiny scenes with K = 16 and 4 q heads per kv head (136 rows, two
    attention row blocks);
  * the same 16 scenes with K = 6 and 9 (112 and 160 rows: 7 and 10 row
    blocks of the wide-unit GEMM), and passes of 32, 33 and 48 rows (the
    boundary of the packed GEMV);
  * 16 scenes of the 16-scene workload's prompt structure (prompts of
    2048..8192 tokens, four camera grids each) at the 7B-class width through
    one target layer, 144 rows and 48 rows: logits of every sequence against
    the oracle;
  * the 16-scene workload at full size (28 layers, the 152064-token head,
    one 144-row verify): its shortest- and longest-prompt scenes against the
    oracle;
  * chained draft steps compacted to one row per sequence: the 16-scene loop
    with and without compaction, and bit-equal proposals on the packed path.
"""
import dataclasses

import numpy as np
import pytest

import workloads as W
from oracle import numerics as ON
from oracle import spec as OS
from tests import _support as S

pytestmark = pytest.mark.gpu


def _session(w, **kw):
    from paper_2606_31160_amd.harness import Session
    return Session(w, **kw)


def _scenes(w, n, lo, hi, seed):
    # four (2, h, 16) camera grids fill about 85% of each prompt (lo >= 430)
    lens = np.random.default_rng(seed).integers(lo, hi + 1, size=n)
    seqs = tuple(W.c5_layout(int(p)) for p in lens)
    assert all(max(b.start + b.ntok for b in q.blocks) <= q.prefix_len for q in seqs)
    return w.with_(seqs=seqs, p_accept=tuple([0.8] * n))


def _verify_against_oracle(w, s, T, seed, check_kv=(0,), kv=None):
    """One verify of explicit drafts (the oracle's first greedy token, then
    random ids) for every sequence, with logits, against the oracle."""
    rng = np.random.default_rng(seed)
    seqs, drafts = [], np.zeros((w.batch, w.K), dtype=np.int32)
    for b in range(w.batch):
        probe = S.oracle_sequence(w, b, T, None, kv=kv, with_draft=False)
        d = rng.integers(0, w.vocab, size=w.K).astype(np.int32)
        d[:1] = OS.greedy_trace(probe, 1)
        drafts[b] = d
        seqs.append(S.oracle_sequence(w, b, T, None, kv=kv, with_draft=False))
    s.verify(drafts, logits=True)
    s.commit()
    coms, acc, fin = s.committed()
    gl = s.logits.float().cpu().numpy()
    for b in range(w.batch):
        ref = seqs[b].verify(drafts[b])
        for j in range(w.K + 1):
            assert S.normwise_err(gl[b, j], ref.logits[j]) <= S.LOGIT_RTOL, (b, j)
        l = int(acc[b])
        pinned = S.margin(ref.logits) > S.MARGIN
        if pinned[:ref.accept_len + 1].all():
            assert l == ref.accept_len and coms[b] == ref.committed, b
        assert coms[b][:l] == list(drafts[b][:l])
        S.check_argmax_rows(coms[b][l:l + 1], ref.logits[l:l + 1])
        st = s.state(b)
        assert st["seq_len"] == w.seqs[b].prefix_len + l + 1 and st["pending"] == coms[b][-1]
        if b in check_kv:
            P = w.seqs[b].prefix_len
            for li in range(w.target.layers):
                for which, cache in ((0, seqs[b].tc.k[li]), (1, seqs[b].tc.v[li])):
                    got = ON.decode(s.kv(b, 0, li, which, P, w.K + 1))
                    assert S.normwise_err(got, cache[P:P + w.K + 1]) <= S.LOGIT_RTOL, (b, li, which)


def _loop(s, max_rounds=100):
    outs = [[] for _ in range(s.B)]
    done = [False] * s.B
    for _ in range(max_rounds):
        for _ in range(s.K):
            s.draft_step()
        s.verify(None)
        s.commit()
        coms, acc, fin = s.committed()
        for b in range(s.B):
            if not done[b]:
                outs[b] += [int(t) for t in coms[b]]
                done[b] = bool(fin[b])
            else:
                assert coms[b] == []
        if all(done):
            break
    assert s.sync() == s.B
    return outs


def _check_history(w, T, outs):
    """Each committed token is the oracle's greedy token after the tokens
    committed before it (pinned rows), or within the tolerance of its top-1."""
    for b, toks in enumerate(outs):
        assert len(toks) == w.max_new_tokens
        seq = S.oracle_sequence(w, b, T, None, with_draft=False)
        P = w.seqs[b].prefix_len
        rows = [seq.pending] + toks[:-1]
        z = T.forward(rows, list(range(P, P + len(rows))), seq.tc)
        S.check_argmax_rows(toks, z)


@pytest.fixture(scope="module")
def tiny16():
    w = _scenes(W.get("C1"), 16, 430, 700, seed=3)
    hp = W.HostWeights(w)
    T, _ = S.oracle_decoders(w, hp)
    return w, hp, T


@pytest.mark.parametrize("path", ["packed", "rowmajor"])
def test_sixteen_scenes_one_verify(tiny16, path):
    # the GEMM streams the tile-packed weight copy by default, the caller's
    # row-major weights with SPEC_FLAG_ROWMAJOR
    from paper_2606_31160_amd import binding as B
    w, hp, T = tiny16
    assert w.batch * (w.K + 1) == 80
    s = _session(w, page_seed=11, flags=S.PATH_FLAGS[path])
    assert B.spec_debug_path(s.ctx) == path
    _verify_against_oracle(w, s, T, seed=5, check_kv=(0, 9, 15))
    s.close()


@pytest.mark.parametrize("K", [6, 9])
def test_sixteen_scenes_row_blocks_of_the_wide_gemm(tiny16, K):
    # 112 and 160 rows: 7 and 10 row blocks of the wide-unit GEMM (the other
    # tests cover 3 at 7B width, 4 at the paper width, 5 and 9; 10 blocks is
    # the pass-size limit)
    w, hp, T = tiny16
    w = w.with_(K=K)
    assert w.batch * (K + 1) in (112, 160)
    s = _session(w, page_seed=13)
    _verify_against_oracle(w, s, T, seed=6 + K, check_kv=(0, 15))
    s.close()


@pytest.mark.parametrize("B,K,path", [(16, 1, "packed"), (2, 15, "packed"), (3, 10, "rowmajor"),
                                      (16, 2, "rowmajor")])
def test_pass_size_boundary_of_the_packed_gemv(tiny16, B, K, path):
    # 32 rows (16 x 2 and 2 x 16): the packed GEMV with two full row blocks;
    # 33 and 48 rows: past it, which at this width the row-major thin GEMV
    # stages (wider models take the wide-unit GEMM there)
    w, hp, T = tiny16
    w = w.with_(K=K, seqs=w.seqs[:B], p_accept=w.p_accept[:B])
    s = _session(w, page_seed=16)
    from paper_2606_31160_amd import binding as B_
    assert B_.spec_debug_path(s.ctx) == path
    _verify_against_oracle(w, s, T, seed=9 + K, check_kv=(0, B - 1))
    s.close()


def test_sixteen_scenes_7b_width_one_layer_three_row_blocks():
    # 48 rows at the 7B-class width: the k-split q/k/v, o and down launches of
    # the wide-unit GEMM with one x block per wave
    c5 = W.get("C5")
    w = W.get("C2").with_(seqs=c5.seqs, p_accept=c5.p_accept, draft=None, K=2)
    assert w.batch * (w.K + 1) == 48 and w.target.hidden == 3584
    src = W.DeviceWeights(w)
    T, _ = S.oracle_decoders(w, src, cache_weights=True)
    s = _session(w, source="device", provider=src, page_seed=15)
    _verify_against_oracle(w, s, T, seed=8, check_kv=(0, 15), kv=S.device_kv)
    s.close()


@pytest.mark.parametrize("rows", ["one_row", "full"])
def test_sixteen_scenes_spec_loop(tiny16, rows):
    # chained draft steps after a round's first run as 16-row passes on the
    # packed GEMV (live-row compaction), or, with SPEC_FLAG_FULL_DRAFT_ROWS,
    # as the 80-row pass on the GEMM
    from paper_2606_31160_amd import binding as B
    w, hp, T = tiny16
    s = _session(w, page_seed=12, flags=B.SPEC_FLAG_FULL_DRAFT_ROWS if rows == "full" else 0)
    outs = _loop(s)
    s.close()
    _check_history(w, T, outs)


def test_sixteen_scenes_28_layer_verify_sampled_against_oracle():
    """The 16-scene workload at full size: 28 layers, the 152064-token head,
    prompts of 2048..8192 tokens in shuffled KV pages, one 144-row verify on
    the batched GEMM.  The scenes with the shortest and the longest prompt are
    checked against the plain float64 oracle: logits of their 9 rows within
    tau (tests/_support.deep_verify_reference), l and the committed token bit
    for bit (their pending tokens reseeded until row 0 is pinned at tau), and
    their first and last layers' new K/V rows."""
    import psutil
    w = W.get("C5").with_(draft=None)
    src = W.DeviceWeights(w)
    T, _ = S.oracle_decoders(w, src, cache_weights=psutil.virtual_memory().available > 150 * 2**30)
    drafts = np.random.default_rng(47).integers(0, w.vocab, size=(w.batch, w.K)).astype(np.int32)
    lens = [q.prefix_len for q in w.seqs]
    sample = sorted({int(np.argmin(lens)), int(np.argmax(lens))})
    picks = {b: S.deep_verify_reference(w, b, T, drafts[b], kv=S.device_kv, n=4) for b in sample}
    pend = [picks[b][0] if b in picks else W.first_pending_token(w, b) for b in range(w.batch)]
    s = _session(w, source="device", provider=src, page_seed=5, pending_tokens=pend)
    s.verify(drafts, logits=True)
    s.commit()
    gl = s.logits.float().cpu().numpy()
    coms, acc, fin = s.committed()
    for b in sample:
        _, ref, seq, tau, _ = picks[b]
        errs = [S.normwise_err(gl[b, j], ref.logits[j]) for j in range(w.K + 1)]
        print(f"scene {b} (prompt {lens[b]}): logit error max {max(errs):.3e} (tau {tau:.3e})", flush=True)
        assert max(errs) <= tau, b
        assert int(acc[b]) == ref.accept_len == 0
        assert list(coms[b]) == list(ref.committed)
        P = w.seqs[b].prefix_len
        for li in (0, w.target.layers - 1):
            for which, cache in ((0, seq.tc.k[li]), (1, seq.tc.v[li])):
                got = ON.decode(s.kv(b, 0, li, which, P, w.K + 1))
                bar = S.LOGIT_RTOL if li == 0 else tau
                assert S.normwise_err(got, cache[P:P + w.K + 1]) <= bar, (b, li, which)
    s.close()


def _proposal_rounds(w, flags, rounds=3):
    s = _session(w, page_seed=4, flags=flags)
    props, coms = [], []
    for _ in range(rounds):
        for _ in range(s.K):
            s.draft_step()
        props.append(s.dtok.cpu().numpy().copy())
        s.verify(None)
        s.commit()
        coms.append(s.committed()[0])
    s.sync()
    s.close()
    return props, coms


def test_one_row_draft_steps_equal_full_row_steps():
    # 3 scenes, K = 4: 15-row passes on the packed GEMV.  A draft row's
    # result does not depend on the pass's row count there, so compacted
    # draft steps propose exactly what the full passes propose.
    from paper_2606_31160_amd import binding as B
    w = _scenes(W.get("C1"), 3, 430, 520, seed=8).with_(max_new_tokens=64)
    a = _proposal_rounds(w, 0)
    b = _proposal_rounds(w, B.SPEC_FLAG_FULL_DRAFT_ROWS)
    for pa, pb in zip(a[0], b[0]):
        np.testing.assert_array_equal(pa, pb)
    assert a[1] == b[1]


def test_block_of_16_eight_scenes():
    base = W.get("C1")
    w = _scenes(base, 8, 430, 600, seed=4).with_(
        K=16, target=dataclasses.replace(base.target, q_heads=8, kv_heads=2),
        draft=dataclasses.replace(base.draft, q_heads=8, kv_heads=2))
    assert w.batch * (w.K + 1) == 136
    T, _ = S.oracle_decoders(w, W.HostWeights(w))
    s = _session(w, page_seed=13)
    _verify_against_oracle(w, s, T, seed=6, check_kv=(3,))
    s.close()
    s = _session(w)
    outs = _loop(s)
    s.close()
    _check_history(w, T, outs)


@pytest.mark.parametrize("path", ["packed", "rowmajor"])
def test_sixteen_scenes_7b_width_one_layer(path):
    c5 = W.get("C5")
    w = W.get("C2").with_(seqs=c5.seqs, p_accept=c5.p_accept, draft=None)
    assert w.batch * (w.K + 1) == 144 and w.target.hidden == 3584
    src = W.DeviceWeights(w)
    T, _ = S.oracle_decoders(w, src, cache_weights=True)
    s = _session(w, source="device", provider=src, page_seed=14, flags=S.PATH_FLAGS[path])
    _verify_against_oracle(w, s, T, seed=7, check_kv=(0, 15), kv=S.device_kv)
    s.close()
