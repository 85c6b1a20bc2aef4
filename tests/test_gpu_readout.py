"""GPU parity of the attention-budget readout (Sec. 4.2, Table attn-budget):
attention mass on visual / trajectory-text / generated slots and the
normalised entropy within trajectory/text, per verify row and query head,
against the oracle's readout of the same layer (oracle.budget).

The oracle rounds activations to bfloat16 where the GPU stores them
(numerics.mirror), so both sides score the same bf16 queries and keys; the
remaining differences are fp32 accumulation order.  Tolerances: 2e-3 absolute
on each mass and on the entropy; the three masses sum to 1 within 1e-5.

  * tiny workload, target layers 0 and 1, packed and row-major paths;
  * the readout pass leaves logits and committed tokens as a plain pass does,
    applies to one pass only, and can be disarmed;
  * the draft's readout with FlatRoPE and with M-RoPE (SPEC_FLAG_DRAFT_MROPE),
    each against the oracle draft of that rotary, and the M-RoPE draft's
    speculative output still equals greedy decoding;
  * the draft's layer-0 cross-attention (SPEC_FLAG_COND_CROSS), the layer the
    paper's table reads, with FlatRoPE and with M-RoPE;
  * 7B-class width, one layer over the 3328-token two-frame prompt;
  * the paper backbone width (32 heads, interleaved M-RoPE), 17 verify rows.
"""
import dataclasses

import numpy as np
import pytest

import workloads as W
from oracle import budget as OB
from oracle import model as OM
from oracle import spec as OS
from tests import _support as S

pytestmark = pytest.mark.gpu

MASS_ATOL = 2e-3
ENT_ATOL = 2e-3


def _session(w, **kw):
    from paper_2606_31160_amd.harness import Session
    return Session(w, **kw)


def _blocks(w, b=0):
    return [(x.start, x.t, x.h, x.w) for x in w.seqs[b].blocks]


def _check(got, ref):
    """got/ref [rows, heads, 4]."""
    assert got.shape == ref.shape
    assert np.all(np.isfinite(got))
    assert np.max(np.abs(got[..., :3].sum(-1) - 1.0)) <= 1e-5
    assert np.all((got[..., 3] >= -1e-6) & (got[..., 3] <= 1.0 + 1e-5))
    assert np.max(np.abs(got[..., :3] - ref[..., :3])) <= MASS_ATOL
    assert np.max(np.abs(got[..., 3] - ref[..., 3])) <= ENT_ATOL


def _target_case(w, provider, layer, drafts, flags=0, device=False):
    """GPU readout of one verify and the oracle's, [K+1, q_heads, 4] each.
    device: weights and prompt K/V drawn by the device generator (the oracle
    reads the same seeded tensors back)."""
    s = _session(w, provider=provider, flags=flags, source="device" if device else "host")
    out = s.attn_readout(0, layer)
    s.verify(drafts[None, :])
    s.commit()
    got = out[0].cpu().numpy()
    s.close()
    T, _ = S.oracle_decoders(w, provider, mirror=True)
    seq = S.oracle_sequence(w, 0, T, None, kv=S.device_kv if device else None, with_draft=False)
    T.readout_layer = layer
    T.readout_classes = OB.slot_classes(w.seqs[0].prefix_len, _blocks(w), seq.cap)
    seq.verify(drafts)
    return got, T.readout


@pytest.fixture(scope="module")
def c1():
    w = W.get("C1")
    return w, W.HostWeights(w)


@pytest.mark.parametrize("path", ["packed", "rowmajor"])
@pytest.mark.parametrize("layer", [0, 1])
def test_target_readout_against_oracle(c1, layer, path):
    w, hp = c1
    drafts = np.random.default_rng(5).integers(0, w.vocab, size=w.K).astype(np.int32)
    got, ref = _target_case(w, hp, layer, drafts, flags=S.PATH_FLAGS[path])
    _check(got, ref)
    # the prompt is vision-dominated and every row sees itself: all three
    # classes receive mass
    assert np.all(got[..., 0] > 0) and np.all(got[..., 2] > 0)


def test_readout_pass_is_a_plain_pass_and_arms_once(c1):
    w, hp = c1
    drafts = np.random.default_rng(6).integers(0, w.vocab, size=w.K).astype(np.int32)
    res = []
    for arm in (False, True):
        s = _session(w, provider=hp)
        out = s.attn_readout(0, 1) if arm else None
        s.verify(drafts[None, :], logits=True)
        s.commit()
        res.append((s.logits[0].float().cpu().numpy(), s.committed()))
        if arm:
            first = out.clone()
            assert bool(first.isfinite().all())
            # later passes do not write it
            out.fill_(-7.0)
            s.verify(drafts[None, :])
            s.commit()
            assert bool((out == -7.0).all())
            # armed, then disarmed: nothing is written
            s.attn_readout(0, 0)
            from paper_2606_31160_amd import binding as B
            B.spec_attn_readout(s.ctx, 0, 0, 0)
            s.verify(drafts[None, :])
            s.commit()
            assert bool(s._readout.isnan().all())
        s.close()
    (z0, c0), (z1, c1_) = res
    assert S.normwise_err(z1, z0) <= 1e-5
    assert c0[0] == c1_[0] and list(c0[1]) == list(c1_[1])


def test_readout_rejects_bad_arguments(c1):
    from paper_2606_31160_amd import binding as B
    w, hp = c1
    s = _session(w, provider=hp)
    for model, layer in ((0, 2), (0, -1), (1, 1), (2, 0)):
        with pytest.raises(B.SpecError) as e:
            s.attn_readout(model, layer)
        assert e.value.status == 1
    s.close()


@pytest.mark.parametrize("rotary", [OM.ROTARY_FLAT, OM.ROTARY_MROPE])
def test_draft_readout_flatrope_and_mrope(c1, rotary):
    from paper_2606_31160_amd import binding as B
    w, hp = c1
    flags = B.SPEC_FLAG_DRAFT_MROPE if rotary == OM.ROTARY_MROPE else 0
    s = _session(w, provider=hp, flags=flags)
    out = s.attn_readout(1, 0)
    s.draft_step()
    got = out[0].cpu().numpy()
    tok = int(s.dtok[0, 0].cpu())
    s.close()
    T, D = S.oracle_decoders(w, hp, mirror=True, draft_rotary=rotary)
    seq = S.oracle_sequence(w, 0, T, D)
    D.readout_layer = 0
    D.readout_classes = OB.slot_classes(w.seqs[0].prefix_len, _blocks(w), seq.cap)
    d, z = seq.draft_step()
    # the first draft step of a round consumes one row (the pending token)
    assert np.all(np.isnan(got[1:]))
    _check(got[:1], D.readout)
    S.check_argmax_rows([tok], z[None, :])


@pytest.mark.parametrize("rotary", [OM.ROTARY_FLAT, OM.ROTARY_MROPE])
def test_draft_cross_attention_readout(c1, rotary):
    # Table attn-budget reads the draft's layer-0 cross-attention: with
    # SPEC_FLAG_COND_CROSS that layer attends to the target-state context
    # (prompt slots and the slots a verify committed).  One verify with two
    # accepted drafts, then the readout of the next draft step's rows.
    from paper_2606_31160_amd import binding as B
    w, hp = c1
    layers = (0, 1, 1)
    flags = B.SPEC_FLAG_DRAFT_MROPE if rotary == OM.ROTARY_MROPE else 0
    T, D = S.oracle_decoders(w, hp, mirror=True, draft_rotary=rotary)
    trace = OS.greedy_trace(S.oracle_sequence(w, 0, T, None, with_draft=False), 4)
    drafts = np.array([trace[0], trace[1], (trace[2] + 1) % w.vocab, 0], dtype=np.int32)
    s = _session(w, provider=hp, flags=flags, cond_layers=layers, cond_cross=True)
    s.verify(drafts[None, :])
    s.commit()
    coms = s.committed()[0][0]
    out = s.attn_readout(1, 0)
    s.draft_step()
    got = out[0].cpu().numpy()
    s.close()
    seq = S.oracle_sequence(w, 0, T, D, cond=S.conditioning(w, hp, layers, mirror=True, cross=True))
    res = seq.verify(drafts)
    assert list(coms) == list(res.committed) and res.accept_len == 2
    D.readout_layer = 0
    D.readout_classes = OB.slot_classes(w.seqs[0].prefix_len, _blocks(w), seq.cap)
    seq.draft_step()
    n = D.readout.shape[0]                      # the catch-up rows of the step
    assert n >= 1 and np.all(np.isnan(got[n:]))
    _check(got[:n], D.readout)


def test_mrope_draft_keeps_greedy_output(c1):
    from paper_2606_31160_amd import binding as B
    w, hp = c1

    def loop(s, K):
        out = []
        while True:
            if K:
                s.draft_steps(K)
            s.verify(None)
            s.commit()
            coms, acc, fin = s.committed()
            out += [int(t) for t in coms[0]]
            if fin[0]:
                return out
    spec = loop(_session(w, provider=hp, flags=B.SPEC_FLAG_DRAFT_MROPE), w.K)
    ar = loop(_session(w, provider=hp, K=0, with_draft=False), 0)
    assert spec == ar and len(spec) == w.max_new_tokens


def test_readout_7b_width_one_layer():
    w = W.get("C2").with_(draft=None)
    drafts = np.random.default_rng(8).integers(0, w.vocab, size=w.K).astype(np.int32)
    got, ref = _target_case(w, W.DeviceWeights(w), 0, drafts, device=True)
    _check(got, ref)


def test_readout_paper_backbone_width_17_rows():
    base = W.get("C6")
    w = base.with_(target=dataclasses.replace(base.target, layers=1), draft=None, vocab=1024)
    drafts = np.random.default_rng(9).integers(0, w.vocab, size=w.K).astype(np.int32)
    got, ref = _target_case(w, W.DeviceWeights(w), 0, drafts, device=True)
    _check(got, ref)
