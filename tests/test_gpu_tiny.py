"""GPU parity on the tiny workload: 2-layer target (hidden 256, 4 q / 2 kv heads,
head_dim 64, M-RoPE sections 8/12/12, SwiGLU 688, vocab 1024), 1-layer FlatRoPE
draft, prompt of 320 tokens (1x16x16 vision grid + 64 text), K = 4.

Bit-exact: position ids, accept lengths, committed tokens, lengths, the GPU's
speculative output against its own greedy decoding.  Within 2e-2 normwise:
logits and cached K/V against the float64 oracle.  Argmax decisions are
compared on rows whose oracle top-1 margin exceeds 2e-2; on the other rows
the GPU token must be within that margin of the oracle's top-1."""
import dataclasses

import numpy as np
import pytest

import workloads as W
from oracle import model as OM
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


@pytest.fixture(scope="module")
def c1():
    w = W.get("C1")
    hp = W.HostWeights(w)
    T, D = S.oracle_decoders(w, hp)
    seq = S.oracle_sequence(w, 0, T, D)
    trace = OS.greedy_trace(seq)
    return w, hp, T, D, trace


def _blocks(w, b=0):
    return [(x.start, x.t, x.h, x.w) for x in w.seqs[b].blocks]


def run_loop(s, mode, synth=None, trace=None, max_rounds=100):
    """Drive propose/verify/commit on sequence 0 until it finishes.
    mode 'draft': the draft model's own K proposals; 'synth': DraftSynth over
    `trace`; 'ar': K = 0.  Returns (tokens, accept lengths, proposals per round)."""
    out, accs, props = [], [], []
    for _ in range(max_rounds):
        if mode == "draft":
            for _ in range(s.K):
                s.draft_step()
            props.append(s.dtok[0].cpu().numpy().copy())
            s.verify(None)
        elif mode == "synth":
            i = len(out)
            s.verify(synth.propose(np.array(trace[i:]), s.K)[None, :])
        else:
            s.verify(None)
        s.commit()
        coms, acc, fin = s.committed()
        out += [int(t) for t in coms[0]]
        accs.append(int(acc[0]))
        if fin[0]:
            break
    assert s.sync() == s.B
    return out, accs, props


# ---------------------------------------------------------------------------

LAYOUTS = {
    "c1": None,
    "frames": W.SeqLayout(200, (W.VisionBlock(0, 2, 6, 8), W.VisionBlock(100, 1, 4, 5))),
    "interleaved": W.SeqLayout(150, (W.VisionBlock(10, 3, 5, 4),)),
}


@pytest.mark.parametrize("name", list(LAYOUTS))
def test_positions_bit_exact(c1, name):
    w = c1[0]
    if LAYOUTS[name] is not None:
        w = w.with_(seqs=(LAYOUTS[name],))
    if name == "interleaved":
        w = w.with_(target=dataclasses.replace(w.target, interleaved=True))
    s = _session(w)
    L = w.seqs[0].prefix_len + w.max_new_tokens + w.K + 1
    assert np.array_equal(s.positions(0, L), OP.target_positions(L, _blocks(w)))
    s.close()


def test_prefix_caches(c1):
    w, hp, T, D, trace = c1
    s = _session(w)
    seq = S.oracle_sequence(w, 0, T, D)
    P = w.seqs[0].prefix_len
    for model, dec, cache in ((0, T, seq.tc), (1, D, seq.dc)):
        for li in range(dec.s.layers):
            k = ON.decode(s.kv(0, model, li, 0, 0, P))
            assert S.normwise_err(k, cache.k[li][:P]) <= 1e-2, (model, li)
            v = s.kv(0, model, li, 1, 0, P)
            assert np.array_equal(v, W.prefix_kv_host(w, 0, "target" if model == 0 else "draft", li, "v"))
    s.close()


def test_one_verify_logits_accept_commit(c1):
    w, hp, T, D, trace = c1
    s = _session(w)
    seq = S.oracle_sequence(w, 0, T, D)
    drafts = W.DraftSynth(w, 0).propose(np.array(trace), w.K)
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
        assert l == ref.accept_len
        assert coms[0] == ref.committed
    assert coms[0][:l] == list(drafts[:l])
    S.check_argmax_rows(coms[0][l:l + 1], ref.logits[l:l + 1])
    st = s.state(0)
    assert st["seq_len"] == w.seqs[0].prefix_len + l + 1
    assert st["pending"] == coms[0][-1]
    # the new keys/values the verify appended, rows 0..K
    P = w.seqs[0].prefix_len
    for li in range(w.target.layers):
        k = ON.decode(s.kv(0, 0, li, 0, P, w.K + 1))
        v = ON.decode(s.kv(0, 0, li, 1, P, w.K + 1))
        assert S.normwise_err(k, seq.tc.k[li][P:P + w.K + 1]) <= S.LOGIT_RTOL
        assert S.normwise_err(v, seq.tc.v[li][P:P + w.K + 1]) <= S.LOGIT_RTOL
    s.close()


def test_spec_loop_equals_greedy_and_oracle(c1):
    w, hp, T, D, trace = c1
    spec_out, accs, props = run_loop(_session(w), "draft")
    ar_out, _, _ = run_loop(_session(w, K=0, with_draft=False), "ar")
    assert spec_out == ar_out                       # Eq. commit keeps greedy output exactly
    assert len(spec_out) == w.max_new_tokens
    # oracle check of every committed token, teacher-forced along the GPU sequence
    seq = S.oracle_sequence(w, 0, T, None, with_draft=False)
    P = w.seqs[0].prefix_len
    toks = [seq.pending] + spec_out[:-1]
    z = T.forward(toks, list(range(P, P + len(toks))), seq.tc)
    pinned = S.check_argmax_rows(spec_out, z)
    if pinned.all():
        assert spec_out == trace


def test_draft_proposals_match_oracle(c1):
    w, hp, T, D, trace = c1
    s = _session(w)
    gpu_out, _, gpu_props = run_loop(s, "draft")
    seq = S.oracle_sequence(w, 0, T, D)
    rec = []

    def proposer(sq):
        out = []
        for _ in range(w.K):
            d, z = sq.draft_step()
            out.append(d)
            rec.append(z)
        return out

    ref_out = OS.spec_loop(seq, proposer)
    if ref_out != gpu_out:
        pytest.skip("GPU and oracle histories diverged at an unpinned row")
    S.check_argmax_rows(np.concatenate(gpu_props), np.stack(rec))


def test_caches_and_lengths_after_rounds(c1):
    w, hp, T, D, trace = c1
    s = _session(w)
    seq = S.oracle_sequence(w, 0, T, D)
    rng = np.random.default_rng(11)
    for _ in range(3):
        for _ in range(w.K):
            s.draft_step()
        seq.propose()
        i = len(seq.generated)
        d = np.array([t if rng.random() < 0.6 else int(rng.integers(0, w.vocab)) for t in trace[i:i + w.K]],
                     dtype=np.int32)
        s.verify(d[None, :])
        s.commit()
        seq.verify(d)
    st = s.state(0)
    assert (st["seq_len"], st["draft_len"], st["pending"], st["n_gen"]) == \
        (seq.seq_len, seq.draft_len, seq.pending, len(seq.generated))
    n = seq.seq_len
    for li in range(w.target.layers):
        for which, ref in ((0, seq.tc.k[li]), (1, seq.tc.v[li])):
            got = ON.decode(s.kv(0, 0, li, which, 0, n))
            assert S.normwise_err(got, ref[:n]) <= S.LOGIT_RTOL
    for li in range(w.draft.layers):
        got = ON.decode(s.kv(0, 1, li, 0, 0, seq.draft_len))
        assert S.normwise_err(got, seq.dc.k[li][:seq.draft_len]) <= S.LOGIT_RTOL
    s.close()


def test_stop_token_and_budget(c1):
    w, hp, T, D, trace = c1
    ar, _, _ = run_loop(_session(w, K=0, with_draft=False), "ar")
    stop = ar[6]
    cut = ar.index(stop)
    out, _, _ = run_loop(_session(w, stop_token=stop), "draft")
    assert out == ar[:cut + 1]
    out, _, _ = run_loop(_session(w, max_new_tokens=7), "synth", synth=W.DraftSynth(w, 0), trace=ar)
    assert out == ar[:7]


def test_out_of_range_draft_token_is_flagged(c1):
    from paper_2606_31160_amd import binding as B
    w = c1[0]
    s = _session(w)
    s.verify(np.array([[1, 2, w.vocab + 5, 3]], dtype=np.int32))
    s.commit()
    with pytest.raises(B.SpecError) as e:
        s.sync()
    assert e.value.status == 1
    s.close()


def test_call_order_enforced(c1):
    from paper_2606_31160_amd import binding as B
    w = c1[0]
    s = _session(w)
    with pytest.raises(B.SpecError):
        s.commit()                      # nothing verified
    with pytest.raises(B.SpecError):
        s.verify(None)                  # no proposals yet
    with pytest.raises(B.SpecError):
        s.draft_steps(0)                # n must be at least 1
    s.draft_step()
    with pytest.raises(B.SpecError):
        s.draft_steps(w.K)              # more than the K - 1 steps left
    s.draft_steps(w.K - 1)
    with pytest.raises(B.SpecError):
        s.draft_step()                  # K steps already taken
    s.verify(None)
    with pytest.raises(B.SpecError):
        s.verify(None)                  # commit first
    s.commit()
    s.close()


def test_graphs_and_direct_launches_agree(c1):
    from paper_2606_31160_amd import binding as B
    w, hp, T, D, trace = c1
    outs = []
    for flags in (0, B.SPEC_FLAG_NO_GRAPHS):
        s = _session(w, flags=flags)
        for _ in range(w.K):
            s.draft_step()
        s.verify(None, logits=True)
        s.commit()
        lg = s.logits.clone()
        o, _, _ = run_loop(s, "draft")
        outs.append((o, lg))
    assert outs[0][0] == outs[1][0]
    assert bool((outs[0][1] == outs[1][1]).all())


def test_draft_steps_equals_single_steps(c1):
    """draft_steps(n) is n draft_step calls issued as one launch sequence: the
    same proposals (columns of the output), the same state, over several
    rounds that include verifier overrides, and a split of K into 1 + (K - 1)."""
    w, hp, T, D, trace = c1
    runs = []
    for how in ("single", "batched", "split"):
        s = _session(w)
        props, states = [], []
        for _ in range(4):
            if how == "single":
                for _ in range(w.K):
                    s.draft_step()
            elif how == "batched":
                s.draft_steps(w.K)
            else:
                s.draft_step()
                s.draft_steps(w.K - 1)
            props.append(s.dtok.cpu().numpy().copy())
            s.verify(None)
            s.commit()
            states.append(s.state(0))
        runs.append((props, states))
    for other in runs[1:]:
        for a, b in zip(runs[0][0], other[0]):
            assert np.array_equal(a, b)
        assert runs[0][1] == other[1]


def run_batch(s, mode, max_rounds=100):
    outs = [[] for _ in range(s.B)]
    done = [False] * s.B
    for _ in range(max_rounds):
        if mode == "draft":
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


def test_batch_of_two(c1):
    w, hp, T, D, trace = c1
    lay2 = W.SeqLayout(260, (W.VisionBlock(20, 2, 8, 8),))
    wb = w.with_(seqs=(w.seqs[0], lay2), p_accept=(0.8, 0.8))
    spec = run_batch(_session(wb), "draft")
    ar = run_batch(_session(wb, K=0, with_draft=False), "ar")
    assert spec == ar
    single, _, _ = run_loop(_session(w), "draft")
    assert spec[0] == single
    Tb, _ = S.oracle_decoders(wb, W.HostWeights(wb))
    seq = S.oracle_sequence(wb, 1, Tb, None, with_draft=False)
    P = lay2.prefix_len
    toks = [seq.pending] + spec[1][:-1]
    z = Tb.forward(toks, list(range(P, P + len(toks))), seq.tc)
    S.check_argmax_rows(spec[1], z)


def test_shuffled_page_tables(c1):
    """Caches in a seeded random permutation of the page pool (caller page
    tables) give the same tokens and bit-identical cached keys and values as
    the default in-order pages."""
    w = c1[0]
    lay2 = W.SeqLayout(260, (W.VisionBlock(20, 2, 8, 8),))
    wb = w.with_(seqs=(w.seqs[0], lay2), p_accept=(0.8, 0.8))
    plain, paged = _session(wb), _session(wb, page_seed=5)
    assert run_batch(plain, "draft") == run_batch(paged, "draft")
    for b in range(wb.batch):
        st = plain.state(b)
        assert st == paged.state(b)
        for model, shape, n in ((0, wb.target, st["seq_len"]), (1, wb.draft, st["draft_len"])):
            for li in range(shape.layers):
                for which in (0, 1):
                    assert np.array_equal(plain.kv(b, model, li, which, 0, n), paged.kv(b, model, li, which, 0, n))
    plain.close()
    paged.close()


def test_block_of_16_with_two_row_blocks(c1):
    # K = 16 (M = 17 rows, two 16-row MFMA blocks in every GEMV) and 4 q heads
    # per kv head (68 query rows per kv head: two attention row blocks).
    w = c1[0]
    w16 = w.with_(K=16, target=dataclasses.replace(w.target, q_heads=8, kv_heads=2),
                  draft=dataclasses.replace(w.draft, q_heads=8, kv_heads=2))
    ar, _, _ = run_loop(_session(w16, K=0, with_draft=False), "ar")
    out, accs, _ = run_loop(_session(w16), "synth", synth=W.DraftSynth(w16, 0), trace=ar)
    assert out == ar
    hp = W.HostWeights(w16)
    T, _ = S.oracle_decoders(w16, hp)
    seq = S.oracle_sequence(w16, 0, T, None, with_draft=False)
    P = w16.seqs[0].prefix_len
    toks = [seq.pending] + out[:-1]
    z = T.forward(toks, list(range(P, P + len(toks))), seq.tc)
    S.check_argmax_rows(out, z)


def test_interleaved_axis_assignment_rotation():
    """Interleaved M-RoPE (pair d reads axis d mod 3, Eq. axis-assign) on a
    prompt with a 3x5x4 vision grid: rotated prompt keys, one verify's logits
    and the new key rows against the oracle."""
    base = W.get("C1")
    w = base.with_(target=dataclasses.replace(base.target, interleaved=True),
                   seqs=(LAYOUTS["interleaved"],), draft=None)
    hp = W.HostWeights(w)
    T, _ = S.oracle_decoders(w, hp)
    s = _session(w, with_draft=False)
    seq = S.oracle_sequence(w, 0, T, None, with_draft=False)
    P = w.seqs[0].prefix_len
    for li in range(w.target.layers):
        k = ON.decode(s.kv(0, 0, li, 0, 0, P))
        assert S.normwise_err(k, seq.tc.k[li][:P]) <= 1e-2, li
    drafts = np.random.default_rng(3).integers(0, w.vocab, size=w.K).astype(np.int32)
    s.verify(drafts[None, :], logits=True)
    s.commit()
    ref = seq.verify(drafts)
    gl = s.logits[0].float().cpu().numpy()
    for j in range(w.K + 1):
        assert S.normwise_err(gl[j], ref.logits[j]) <= S.LOGIT_RTOL, j
    for li in range(w.target.layers):
        k = ON.decode(s.kv(0, 0, li, 0, P, w.K + 1))
        assert S.normwise_err(k, seq.tc.k[li][P:P + w.K + 1]) <= S.LOGIT_RTOL
    s.close()


def test_requested_execution_path_runs(c1, path):
    """The requested weight layout is the one the per-layer kernels stream,
    one launch per layer step (counted by the library's timing)."""
    from paper_2606_31160_amd import binding as B
    w = c1[0]
    s = _session(w)
    B.spec_timing(s.ctx, True)
    s.draft_step()
    for _ in range(w.K - 1):
        s.draft_step()
    s.verify(None)
    s.commit()
    n_qkv, _, _ = B.spec_timing_read(s.ctx, "qkv")
    B.spec_timing(s.ctx, False)
    assert s.sync() == 0
    assert B.spec_debug_path(s.ctx) == path
    assert n_qkv == w.target.layers + w.K * w.draft.layers
    s.close()


class _EditedEmbed:
    """The workload's weights with the tied embedding edited by `edit`."""

    def __init__(self, base, edit):
        self.base, self.edit = base, edit

    def get(self, model, layer, name):
        a = self.base.get(model, layer, name)
        return self.edit(a.copy()) if name == "embed" else a


@pytest.mark.parametrize("direction", ["copy_up", "copy_down"])
def test_exact_argmax_tie_goes_to_the_lowest_index(c1, direction):
    """Eq. verify's greedy argmax on exact ties (reading: lowest index wins).
    Copying the embedding row of row 0's greedy token v into another row u
    makes logits z[v] and z[u] bit-equal on both sides; the committed bonus
    token must then be min(u, v), with u in another LM-head tile and
    workgroup, above or below v."""
    w, hp = c1[0], c1[1]
    rng = np.random.default_rng(51)
    drafts = None
    for pend in S.pending_candidates(w, 0):
        T, _ = S.oracle_decoders(w, hp)
        z0 = S.oracle_sequence(w, 0, T, None, with_draft=False, pending=pend).verify([]).logits[0]
        v = int(np.argmax(z0))
        if S.margin(z0[None, :])[0] <= S.MARGIN:
            continue
        u = (v + 16 * 7 + 3) % w.vocab if direction == "copy_up" else (v - 16 * 7 - 3) % w.vocab
        if pend == u or (direction == "copy_up") != (u > v):
            continue
        drafts = rng.integers(0, w.vocab, size=w.K).astype(np.int32)
        drafts[drafts == u] = (u + 1) % w.vocab
        drafts[drafts == v] = (v + 1) % w.vocab
        break
    assert drafts is not None

    def edit(E):
        E[u] = E[v]
        return E

    prov = _EditedEmbed(hp, edit)
    T, _ = S.oracle_decoders(w, prov)
    ref = S.oracle_sequence(w, 0, T, None, with_draft=False, pending=pend).verify(drafts)
    assert ref.logits[0, u] == ref.logits[0, v]
    want = min(u, v)
    assert ref.rstar[0] == want and ref.accept_len == 0
    s = _session(w, provider=prov, pending_tokens=[pend])
    s.verify(drafts[None, :], logits=True)
    s.commit()
    zb = s.logits[0, 0].view(s.torch.int16).cpu().numpy()
    assert zb[u] == zb[v]
    coms, acc, fin = s.committed()
    assert int(acc[0]) == 0 and coms[0] == [want], (coms[0], u, v)
    assert s.sync() == 0
    s.close()


def test_nan_logits_are_reported_and_skipped(c1):
    """NaN logits count as -inf in the argmax and set SPEC_E_NUMERIC, which
    spec_sync reports (reading of Eq. verify's argmax on invalid values)."""
    from paper_2606_31160_amd import binding as B
    w, hp = c1[0], c1[1]
    pend = W.first_pending_token(w, 0)
    rng = np.random.default_rng(52)
    drafts = rng.integers(0, w.vocab, size=w.K).astype(np.int32)
    jn = next(j for j in range(w.vocab - 1, 0, -1) if j != pend and j not in set(drafts.tolist()))

    def edit(E):
        E[jn] = 0x7FC0            # a quiet NaN in every column of one row
        return E

    prov = _EditedEmbed(hp, edit)
    T, _ = S.oracle_decoders(w, prov)
    ref = S.oracle_sequence(w, 0, T, None, with_draft=False, pending=pend).verify(drafts)
    assert np.isnan(ref.logits[:, jn]).all() and not np.isnan(np.delete(ref.logits, jn, axis=1)).any()
    s = _session(w, provider=prov)
    s.verify(drafts[None, :])
    s.commit()
    with pytest.raises(B.SpecError) as e:
        s.sync()
    assert e.value.status == 6
    coms, acc, fin = s.committed()
    z = np.delete(ref.logits, jn, axis=1)
    if S.margin(z[:1])[0] > S.MARGIN:
        assert coms[0][-1] == ref.committed[-1] and int(acc[0]) == ref.accept_len
    assert jn not in coms[0]
    s.close()
