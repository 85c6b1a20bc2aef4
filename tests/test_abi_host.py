"""Host-side checks of the C ABI: the library loads, exports every entry point
include/spec.h declares, and rejects invalid arguments on the host before any
work is enqueued.  No GPU is needed: the calls below fail validation first."""
import ctypes
import os
import re

import pytest

from paper_2606_31160_amd import binding as B
import workloads as W

HEADER = os.path.join(os.path.dirname(os.path.dirname(__file__)), "include", "spec.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b((?:spec|draft)_\w+)\s*\(", text)))


def test_library_loads_and_exports_every_declared_symbol():
    L = B.lib()
    names = _declared()
    assert "spec_init" in names and "draft_step" in names and "spec_verify" in names and "spec_commit" in names
    for n in names:
        assert hasattr(L, n), n


def test_struct_sizes_match_c_layout():
    # 64-bit SysV layout of the header's structs
    assert ctypes.sizeof(B.spec_dims) == 48
    assert ctypes.sizeof(B.spec_config) == 136
    assert ctypes.sizeof(B.spec_seq_init) == 64
    assert ctypes.sizeof(B.spec_layer_weights) == 72


def _cfg(w, K=None, batch=1):
    cfg = B.spec_config()
    cfg.target = B.dims(w.target)
    cfg.draft = B.dims(w.draft)
    cfg.vocab = w.vocab
    cfg.K = w.K if K is None else K
    cfg.batch = batch
    cfg.max_new_tokens = 20
    cfg.stop_token = -1
    return cfg


FAKE = 0x100000   # an aligned non-null address; validation never dereferences it


def _seqs(w, cfg, prefix=None, blocks=None, pending=3):
    seqs = (B.spec_seq_init * cfg.batch)()
    keep = []
    for b in range(cfg.batch):
        s = seqs[b]
        lay = w.seqs[0]
        s.prefix_len = lay.prefix_len if prefix is None else prefix
        bl = lay.blocks if blocks is None else blocks
        arr = (B.spec_vision_block * max(1, len(bl)))()
        for i, x in enumerate(bl):
            arr[i].start, arr[i].t, arr[i].h, arr[i].w = x
        s.blocks, s.n_blocks = arr, len(bl)
        s.pending_token = pending
        tk = (ctypes.c_void_p * cfg.target.layers)(*([FAKE] * cfg.target.layers))
        dk = (ctypes.c_void_p * max(1, cfg.draft.layers))(*([FAKE] * max(1, cfg.draft.layers)))
        s.tgt_k = s.tgt_v = tk
        s.drf_k = s.drf_v = dk
        keep += [arr, tk, dk]
    return seqs, keep


def _blocks(w):
    return [(b.start, b.t, b.h, b.w) for b in w.seqs[0].blocks]


def test_workspace_query_on_host():
    w = W.get("C1")
    cfg = _cfg(w)
    seqs, keep = _seqs(w, cfg, blocks=_blocks(w))
    n1 = B.spec_workspace_bytes(cfg, seqs)
    assert n1 > 0 and n1 % 256 == 0
    cfg.max_new_tokens = 500
    assert B.spec_workspace_bytes(cfg, seqs) > n1


@pytest.mark.parametrize("name", ["C3", "C6"])
def test_benchmark_and_paper_configs_validate_on_host(name):
    # the 7B-class benchmark configuration, and the paper's backbone at K = 16
    # (17 verify rows, interleaved axis assignment)
    w = W.get(name)
    cfg = _cfg(w)
    seqs, keep = _seqs(w, cfg, blocks=_blocks(w))
    n = B.spec_workspace_bytes(cfg, seqs)
    assert n > 0 and n % 256 == 0


@pytest.mark.parametrize("mutate,needle", [
    (lambda c, s: setattr(c, "K", 17), "K out of range"),
    (lambda c, s: setattr(c, "batch", 0), "batch"),
    (lambda c, s: setattr(c, "vocab", 1000), "vocab"),
    (lambda c, s: setattr(c, "max_new_tokens", 0), "max_new_tokens"),
    (lambda c, s: setattr(c, "stop_token", 5000), "stop_token"),
    (lambda c, s: c.target.mrope_section.__setitem__(0, 9), "mrope_section"),
    (lambda c, s: setattr(c.target, "head_dim", 96), "head_dim"),
    (lambda c, s: setattr(c.target, "q_heads", 3), "q_heads"),
    (lambda c, s: setattr(c.target, "ffn", 680), "ffn"),
    (lambda c, s: setattr(c.draft, "hidden", 128), "draft"),
    # an M-RoPE draft's sections are validated like the target's
    (lambda c, s: (setattr(c, "flags", B.SPEC_FLAG_DRAFT_MROPE), c.draft.mrope_section.__setitem__(0, 9)),
     "draft: mrope_section"),
    (lambda c, s: setattr(s[0], "pending_token", 1024), "pending_token"),
    (lambda c, s: setattr(s[0], "prefix_len", 0), "prefix_len"),
    (lambda c, s: (setattr(c, "flags", B.SPEC_FLAG_BLOCK_DRAFT), setattr(c, "mask_token", 1024)), "mask_token"),
    (lambda c, s: setattr(c, "flags", 2), "unknown bits in flags"),
    (lambda c, s: setattr(c, "flags", 4 | B.SPEC_FLAG_ROWMAJOR), "unknown bits in flags"),
    (lambda c, s: (setattr(c, "flags", B.SPEC_FLAG_BLOCK_DRAFT), setattr(c, "K", 0)), "BLOCK_DRAFT"),
    (lambda c, s: setattr(c, "flags", B.SPEC_FLAG_COND_CROSS), "needs SPEC_FLAG_COND"),
    (lambda c, s: setattr(c, "flags", B.SPEC_FLAG_COND | B.SPEC_FLAG_COND_CROSS | B.SPEC_FLAG_BLOCK_DRAFT),
     "does not combine with SPEC_FLAG_BLOCK_DRAFT"),
])
def test_invalid_config_rejected_on_host(mutate, needle):
    w = W.get("C1")
    cfg = _cfg(w)
    seqs, keep = _seqs(w, cfg, blocks=_blocks(w))
    mutate(cfg, seqs)
    with pytest.raises(B.SpecError) as e:
        B.spec_workspace_bytes(cfg, seqs)
    assert e.value.status == 1 and needle in str(e.value)


def test_vision_blocks_validated():
    w = W.get("C1")
    cfg = _cfg(w)
    for blocks, needle in [([(310, 1, 4, 4)], "outside"), ([(0, 1, 4, 4), (10, 1, 2, 2)], "overlap"),
                           ([(0, 0, 4, 4)], "outside")]:
        seqs, keep = _seqs(w, cfg, blocks=blocks)
        with pytest.raises(B.SpecError) as e:
            B.spec_workspace_bytes(cfg, seqs)
        assert needle in str(e.value)


def test_init_rejects_before_touching_the_device():
    w = W.get("C1")
    cfg = _cfg(w)
    seqs, keep = _seqs(w, cfg, blocks=_blocks(w))
    tl = (B.spec_layer_weights * cfg.target.layers)()
    for l in range(cfg.target.layers):
        for n, _ in B.spec_layer_weights._fields_:
            setattr(tl[l], n, FAKE)
    tw = B.spec_model_weights(tl, FAKE)
    dl = (B.spec_layer_weights * cfg.draft.layers)()
    for l in range(cfg.draft.layers):
        for n, _ in B.spec_layer_weights._fields_:
            setattr(dl[l], n, FAKE)
    dw = B.spec_model_weights(dl, FAKE)
    need = B.spec_workspace_bytes(cfg, seqs)
    # workspace too small
    with pytest.raises(B.SpecError) as e:
        B.spec_init(cfg, FAKE, tw, dw, seqs, FAKE, need - 256, 0)
    assert e.value.status == 3
    # misaligned workspace
    with pytest.raises(B.SpecError) as e:
        B.spec_init(cfg, FAKE, tw, dw, seqs, FAKE + 16, need, 0)
    assert e.value.status == 1 and "workspace" in str(e.value)
    # a null weight
    tl[1].w_up = None
    with pytest.raises(B.SpecError) as e:
        B.spec_init(cfg, FAKE, tw, dw, seqs, FAKE, need, 0)
    assert "layer 1" in str(e.value)
    tl[1].w_up = FAKE
    # draft weights given while draft.layers == 0
    cfg.draft.layers = 0
    with pytest.raises(B.SpecError) as e:
        B.spec_init(cfg, FAKE, tw, dw, seqs, FAKE, need, 0)
    assert "draft" in str(e.value)


def test_calls_on_null_context():
    L = B.lib()
    assert L.draft_step(None, None) == 1
    assert L.draft_steps(None, 1, None) == 1
    assert L.spec_attn_readout(None, 0, 0, None) == 1
    assert L.spec_verify(None, None, None) == 1
    assert L.spec_commit(None, None, None, None, None) == 1
    assert L.spec_sync(None, None) == 1
    L.spec_destroy(None)


def test_flatrope_draft_ignores_its_sections():
    w = W.get("C1")
    cfg = _cfg(w)
    seqs, keep = _seqs(w, cfg, blocks=_blocks(w))
    cfg.draft.mrope_section[0] = 9
    assert B.spec_workspace_bytes(cfg, seqs) > 0


def test_page_tables_validated_on_host():
    w = W.get("C1")
    cfg = _cfg(w, batch=2)
    seqs, keep = _seqs(w, cfg, blocks=_blocks(w))
    n = B.spec_seq_pages(cfg, seqs[0])
    # prompt + token budget + K + 2 slots, in pages of 64
    assert n == -(-(w.seqs[0].prefix_len + 20 + w.K + 2) // 64)
    plain = B.spec_workspace_bytes(cfg, seqs)

    def tables(t0, t1):
        a0 = (ctypes.c_int32 * len(t0))(*t0)
        a1 = (ctypes.c_int32 * len(t1))(*t1)
        keep.extend([a0, a1])
        seqs[0].page_table, seqs[1].page_table = a0, a1

    perm = list(range(2 * n))[::-1]
    tables(perm[:n], perm[n:])
    assert B.spec_workspace_bytes(cfg, seqs) == plain     # same pool, another order
    for t0, t1, needle in [(perm[:n], perm[:n], "used twice"),
                           (perm[:n - 1] + [2 * n], perm[n:], "out of range"),
                           (perm[:n - 1] + [-1], perm[n:], "out of range")]:
        tables(t0, t1)
        with pytest.raises(B.SpecError) as e:
            B.spec_workspace_bytes(cfg, seqs)
        assert needle in str(e.value)
    tables(perm[:n], perm[n:])
    seqs[1].page_table = None
    with pytest.raises(B.SpecError) as e:
        B.spec_workspace_bytes(cfg, seqs)
    assert "every sequence" in str(e.value)
