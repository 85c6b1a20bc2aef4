// Host runtime behind include/spec.h: validation, workspace carving, the 3D
// position table and the rotary (cos, sin) table, the call state machine,
// HIP-graph capture and per-kernel event timing.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <exception>
#include <new>
#include <string>
#include <vector>

#include "ctx.h"
#include "gemv.h"
#include "sgemv.h"

using namespace specdec;

struct spec_ctx {
  Ctx c;
};

namespace {

thread_local std::string g_init_error;

constexpr size_t kAlign = 256;
constexpr int32_t kKnownFlags = SPEC_FLAG_NO_GRAPHS | SPEC_FLAG_ROWMAJOR | SPEC_FLAG_BLOCK_DRAFT | SPEC_FLAG_COND |
                                SPEC_FLAG_DRAFT_MROPE | SPEC_FLAG_FULL_DRAFT_ROWS | SPEC_FLAG_COND_CROSS;

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

struct Carver {
  char* base;
  size_t off = 0;
  template <class T>
  T* take(size_t n) {
    off = align_up(off, kAlign);
    T* p = base ? reinterpret_cast<T*>(base + off) : nullptr;
    off += n * sizeof(T);
    return p;
  }
};

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// ---- validation -------------------------------------------------------------

bool check_dims(const spec_dims& d, bool is_target, std::string& err, const char* who) {
  char buf[256];
  auto bad = [&](const char* what) {
    snprintf(buf, sizeof buf, "%s: %s", who, what);
    err = buf;
    return false;
  };
  if (d.layers < 1 || d.layers > SPEC_MAX_LAYERS) return bad("layers out of range");
  if (d.hidden < 16 || d.hidden % 16) return bad("hidden must be a positive multiple of 16");
  if (d.head_dim != 64 && d.head_dim != 128) return bad("head_dim must be 64 or 128");
  if (d.kv_heads < 1 || d.q_heads < 1 || d.q_heads % d.kv_heads) return bad("q_heads must be a multiple of kv_heads");
  if ((d.q_heads * d.head_dim) % 16) return bad("q_heads*head_dim must be a multiple of 16");
  if (d.ffn < 16 || d.ffn % 16) return bad("ffn must be a positive multiple of 16");
  if (!(d.rope_base > 1.0f) || !std::isfinite(d.rope_base)) return bad("rope_base must be > 1");
  if (!(d.rms_eps >= 0.0f) || !std::isfinite(d.rms_eps)) return bad("rms_eps must be >= 0");
  if (is_target) {
    if (d.interleaved != 0 && d.interleaved != 1) return bad("interleaved must be 0 or 1");
    const int* s = d.mrope_section;
    if (s[0] < 0 || s[1] < 0 || s[2] < 0 || s[0] + s[1] + s[2] != d.head_dim / 2)
      return bad("mrope_section must be non-negative and sum to head_dim/2");
  }
  return true;
}

// KV pages of one sequence (include/spec.h, spec_seq_pages).
int seq_pages(const spec_config* cfg, const spec_seq_init& s) {
  return (int)((align_up((size_t)s.prefix_len + cfg->max_new_tokens + cfg->K + 2, kAttnChunk)) / kAttnChunk);
}

bool check_config(const spec_config* cfg, const spec_seq_init* seqs, bool has_draft, std::string& err) {
  if (!cfg || !seqs) {
    err = "null config or sequences";
    return false;
  }
  if (cfg->batch < 1 || cfg->batch > SPEC_MAX_BATCH) {
    err = "batch out of range";
    return false;
  }
  if (cfg->K < 0 || cfg->K > SPEC_MAX_K) {
    err = "K out of range";
    return false;
  }
  if (cfg->batch * (cfg->K + 1) > SPEC_MAX_ROWS) {
    err = "batch*(K+1) rows per pass must not exceed SPEC_MAX_ROWS";
    return false;
  }
  if (cfg->vocab < 16 || cfg->vocab % 16) {
    err = "vocab must be a positive multiple of 16";
    return false;
  }
  if (cfg->max_new_tokens < 1) {
    err = "max_new_tokens must be >= 1";
    return false;
  }
  if (cfg->stop_token < -1 || cfg->stop_token >= cfg->vocab) {
    err = "stop_token out of range";
    return false;
  }
  if (cfg->flags & ~kKnownFlags) {
    err = "unknown bits in flags";
    return false;
  }
  if (!check_dims(cfg->target, true, err, "target")) return false;
  if (cfg->flags & SPEC_FLAG_COND) {
    if (!has_draft) {
      err = "SPEC_FLAG_COND needs a draft";
      return false;
    }
    for (int i = 0; i < 3; ++i)
      if (cfg->cond_layers[i] < 0 || cfg->cond_layers[i] >= cfg->target.layers) {
        err = "cond_layers out of range";
        return false;
      }
  }
  if (cfg->flags & SPEC_FLAG_COND_CROSS) {
    if (!(cfg->flags & SPEC_FLAG_COND)) {
      err = "SPEC_FLAG_COND_CROSS needs SPEC_FLAG_COND";
      return false;
    }
    if (cfg->flags & SPEC_FLAG_BLOCK_DRAFT) {
      err = "SPEC_FLAG_COND_CROSS does not combine with SPEC_FLAG_BLOCK_DRAFT";
      return false;
    }
  }
  if (cfg->flags & SPEC_FLAG_BLOCK_DRAFT) {
    if (!has_draft || cfg->K < 1) {
      err = "SPEC_FLAG_BLOCK_DRAFT needs a draft and K >= 1";
      return false;
    }
    if (cfg->mask_token < 0 || cfg->mask_token >= cfg->vocab) {
      err = "mask_token out of range";
      return false;
    }
  }
  if (has_draft) {
    if (!check_dims(cfg->draft, (cfg->flags & SPEC_FLAG_DRAFT_MROPE) != 0, err, "draft")) return false;
    if (cfg->draft.hidden != cfg->target.hidden || cfg->draft.head_dim != cfg->target.head_dim ||
        cfg->draft.rope_base != cfg->target.rope_base) {
      err = "draft hidden, head_dim and rope_base must equal the target's";
      return false;
    }
  }
  for (int b = 0; b < cfg->batch; ++b) {
    const spec_seq_init& s = seqs[b];
    char buf[160];
    if (s.prefix_len < 1) {
      snprintf(buf, sizeof buf, "sequence %d: prefix_len must be >= 1", b);
      err = buf;
      return false;
    }
    if (s.pending_token < 0 || s.pending_token >= cfg->vocab) {
      snprintf(buf, sizeof buf, "sequence %d: pending_token out of range", b);
      err = buf;
      return false;
    }
    if (s.n_blocks < 0 || (s.n_blocks > 0 && !s.blocks)) {
      snprintf(buf, sizeof buf, "sequence %d: bad vision blocks", b);
      err = buf;
      return false;
    }
    std::vector<char> taken(s.prefix_len, 0);
    for (int i = 0; i < s.n_blocks; ++i) {
      const spec_vision_block& v = s.blocks[i];
      const long long n = (long long)v.t * v.h * v.w;
      if (v.t < 1 || v.h < 1 || v.w < 1 || v.start < 0 || v.start + n > s.prefix_len) {
        snprintf(buf, sizeof buf, "sequence %d: vision block %d outside [0, prefix_len)", b, i);
        err = buf;
        return false;
      }
      for (long long k = v.start; k < v.start + n; ++k) {
        if (taken[k]) {
          snprintf(buf, sizeof buf, "sequence %d: vision blocks overlap", b);
          err = buf;
          return false;
        }
        taken[k] = 1;
      }
    }
    if (!s.tgt_k || !s.tgt_v) {
      snprintf(buf, sizeof buf, "sequence %d: missing target prefix K/V", b);
      err = buf;
      return false;
    }
    for (int l = 0; l < cfg->target.layers; ++l)
      if (!s.tgt_k[l] || !s.tgt_v[l] || !aligned16(s.tgt_k[l]) || !aligned16(s.tgt_v[l])) {
        snprintf(buf, sizeof buf, "sequence %d: target prefix K/V of layer %d null or misaligned", b, l);
        err = buf;
        return false;
      }
    if (has_draft) {
      if (!s.drf_k || !s.drf_v) {
        snprintf(buf, sizeof buf, "sequence %d: missing draft prefix K/V", b);
        err = buf;
        return false;
      }
      for (int l = 0; l < cfg->draft.layers; ++l)
        if (!s.drf_k[l] || !s.drf_v[l] || !aligned16(s.drf_k[l]) || !aligned16(s.drf_v[l])) {
          snprintf(buf, sizeof buf, "sequence %d: draft prefix K/V of layer %d null or misaligned", b, l);
          err = buf;
          return false;
        }
    }
  }
  // page tables: all or none; together a permutation of the pool's pages
  int given = 0;
  long long pool = 0;
  for (int b = 0; b < cfg->batch; ++b) {
    given += seqs[b].page_table != nullptr;
    pool += seq_pages(cfg, seqs[b]);
  }
  if (given != 0 && given != cfg->batch) {
    err = "either every sequence gives a page_table or none does";
    return false;
  }
  if (pool >= (1ll << 31) / kAttnChunk) {
    err = "too many KV pages";
    return false;
  }
  if (given) {
    std::vector<char> used((size_t)pool, 0);
    for (int b = 0; b < cfg->batch; ++b) {
      const int n = seq_pages(cfg, seqs[b]);
      for (int i = 0; i < n; ++i) {
        const int32_t p = seqs[b].page_table[i];
        if (p < 0 || p >= pool || used[p]) {
          char buf[160];
          snprintf(buf, sizeof buf, "sequence %d: page_table[%d] = %d is out of range or used twice", b, i, p);
          err = buf;
          return false;
        }
        used[p] = 1;
      }
    }
  }
  return true;
}

bool check_weights(const spec_model_weights* w, const spec_dims& d, std::string& err, const char* who) {
  char buf[160];
  if (!w || !w->layers || !w->final_norm || !aligned16(w->final_norm)) {
    snprintf(buf, sizeof buf, "%s weights: null or misaligned", who);
    err = buf;
    return false;
  }
  for (int l = 0; l < d.layers; ++l) {
    const spec_layer_weights& L = w->layers[l];
    const void* ps[] = {L.attn_norm, L.wq, L.wk, L.wv, L.wo, L.ffn_norm, L.w_gate, L.w_up, L.w_down};
    for (const void* p : ps)
      if (!p || !aligned16(p)) {
        snprintf(buf, sizeof buf, "%s weights: layer %d has a null or misaligned tensor", who, l);
        err = buf;
        return false;
      }
  }
  return true;
}

// ---- layout -------------------------------------------------------------------

struct Layout {
  int B, K, R, M, Mpad, V, cap, chunk, splits, pool;
};


Layout make_layout(const spec_config* cfg, const spec_seq_init* seqs) {
  Layout L{};
  L.B = cfg->batch;
  L.K = cfg->K;
  L.R = cfg->K + 1;
  L.M = L.B * L.R;
  L.Mpad = (int)align_up(L.M, 16);
  L.V = cfg->vocab;
  int maxP = 0;
  for (int b = 0; b < L.B; ++b) maxP = std::max(maxP, seqs[b].prefix_len);
  L.cap = (int)align_up((size_t)maxP + cfg->max_new_tokens + cfg->K + 2, kAttnChunk);
  L.chunk = kAttnChunk;
  L.splits = L.cap / L.chunk;
  L.pool = 0;
  for (int b = 0; b < L.B; ++b) L.pool += seq_pages(cfg, seqs[b]);
  return L;
}

// wide: the context's passes have more than kSgMaxRows rows and run on the
// tile-packed copy (the wide-unit GEMM)
void set_splits(Model& m, int M, bool gemm_rows, bool wide) {
  if (wide) {
    m.s_down = gemm_wide_splits(m.d.hidden, m.d.ffn, num_cus());
    m.s_o = gemm_wide_splits(m.d.hidden, m.d.q_heads * m.d.head_dim, num_cus());
    return;
  }
  const int slots = gemm_rows ? num_cus() * gemm_wgs_per_cu(M) : num_cus();
  m.s_down = gemm_rows ? gemm_down_splits(m.d.hidden, m.d.ffn, slots) : down_splits(M, m.d.ffn, num_cus());
  m.s_o = gemm_rows ? gemm_down_splits(m.d.hidden, m.d.q_heads * m.d.head_dim, slots) : 1;
}

size_t part_elems_for(const Model& m, int M, bool wide) {
  // a pass of fewer rows may split the q/k/v GEMM where one of M rows does not
  const int nqkv = (m.d.q_heads + 2 * m.d.kv_heads) * m.d.head_dim;
  size_t qkv = 0;
  for (int r = 1; r <= M; ++r) {
    const int sq = gemm_qkv_splits_for(nqkv, m.d.hidden, r, num_cus(), wide);
    if (sq > 1) qkv = std::max(qkv, (size_t)sq * r * nqkv);
  }
  return std::max((size_t)std::max({m.s_down, m.s_o, kCondSplits}) * M * m.d.hidden, qkv);
}

// The q/k/v, o, gate/up and LM-head GEMVs keep a workgroup's whole reduction
// (one k-split): their x rows for the full reduction length must fit in LDS,
// and each wave streams at most kGemvSteps steps.
// Whether the thin GEMV kernels can stage M rows of every input width of a model.
bool thin_fits(const spec_dims& d, int M, int* bad_width = nullptr) {
  const int Ks[2] = {d.hidden, d.q_heads * d.head_dim};
  for (int Kd : Ks) {
    const int T = (Kd + 31) / 32;
    if (T > kGemvWaves * kGemvSteps || gemv_p_lds_bytes(M, T) > (size_t)gemv_lds_limit()) {
      if (bad_width) *bad_width = Kd;
      return false;
    }
  }
  return true;
}

bool check_fits(const spec_dims& d, int M, std::string& err, const char* who) {
  // more rows than one MFMA block: the batched-row GEMM, which streams x
  // through LDS in chunks, takes what the thin kernels cannot stage
  if (M > kSgMaxRowsGemm) return true;
  int Kd = 0;
  if (!thin_fits(d, M, &Kd)) {
    char buf[200];
    snprintf(buf, sizeof buf, "%s: %d rows per pass (batch*(K+1)) with width %d exceed one GEMV workgroup", who, M, Kd);
    err = buf;
    return false;
  }
  return true;
}

// Layered passes of this many rows run on the batched-row GEMM.
bool gemm_rows_for(const spec_config* cfg, bool has_draft, int M) {
  if (M > kThinRows) return true;
  return M > kSgMaxRowsGemm && (!thin_fits(cfg->target, M) || (has_draft && !thin_fits(cfg->draft, M)));
}

// The draft's packed-GEMV jobs for a pass of one row per sequence (B rows),
// kept in drf.sg_one; the context's pass shape is untouched on return.
bool sg_build_one(Ctx& c, bool fill) {
  const int R = c.R, M = c.M, Mpad = c.Mpad;
  c.R = 1;
  c.M = c.B;
  c.Mpad = c.Mpad1;
  std::vector<SgJob> host, block;
  host.swap(c.drf.sg_host);
  block.swap(c.drf.sg_block);
  const bool ok = sg_build_jobs(c, c.drf, true, fill);
  c.drf.sg_one.swap(c.drf.sg_host);
  c.drf.sg_host.swap(host);
  c.drf.sg_block.swap(block);
  c.R = R;
  c.M = M;
  c.Mpad = Mpad;
  return ok;
}

// Carves the workspace (base == nullptr only measures).  Returns total bytes.
size_t carve(Ctx& c, const spec_config* cfg, const spec_seq_init* seqs, bool has_draft, char* base) {
  const Layout L = make_layout(cfg, seqs);
  c.B = L.B;
  c.K = L.K;
  c.R = L.R;
  c.M = L.M;
  c.Mpad = L.Mpad;
  c.V = L.V;
  c.cap = L.cap;
  c.pps = L.splits;
  c.pool = L.pool;
  c.attn_chunk = L.chunk;
  c.ncu = num_cus();
  c.attn_splits = L.splits;
  // one page per attention workgroup gives a pass over one sequence of 4 kv
  // heads enough workgroups; with 8 or more (sequence, kv head) pairs three
  // pages per workgroup (a third of the partials to merge), from 8 sequences
  // on four.  The choice depends on the batch and the target's kv heads only,
  // so every pass of a context groups the attention sums the same way.
  c.attn_ppw = L.B >= 8 ? 4 : (L.B * cfg->target.kv_heads >= 8 ? 3 : 1);
  c.tgt.d = cfg->target;
  c.tgt.flat = false;
  c.block_draft = has_draft && (cfg->flags & SPEC_FLAG_BLOCK_DRAFT) != 0;
  c.mask_token = cfg->mask_token;
  c.cond = has_draft && (cfg->flags & SPEC_FLAG_COND) != 0;
  c.cross = c.cond && (cfg->flags & SPEC_FLAG_COND_CROSS) != 0;
  for (int i = 0; i < 3; ++i) c.cond_layers[i] = cfg->cond_layers[i];
  c.gemm_rows = gemm_rows_for(cfg, has_draft, L.M);
  // passes of more than kSgMaxRows rows never take the packed GEMV, so they
  // stream the packed copy on the wide-unit GEMM unless the caller asks for
  // row-major weights
  c.gemm_wide = c.gemm_rows && L.M > kSgMaxRows && !(cfg->flags & SPEC_FLAG_ROWMAJOR);
  set_splits(c.tgt, L.M, c.gemm_rows, c.gemm_wide);
  if (has_draft) {
    c.drf.d = cfg->draft;
    c.drf.flat = (cfg->flags & SPEC_FLAG_DRAFT_MROPE) == 0;
    set_splits(c.drf, L.M, c.gemm_rows, c.gemm_wide);
  }
  const spec_dims& t = cfg->target;
  const int H = t.hidden, D = t.head_dim;
  int nqD = t.q_heads * D, F = t.ffn, nq = t.q_heads;
  size_t part = part_elems_for(c.tgt, L.M, c.gemm_wide);
  if (has_draft) {
    nqD = std::max(nqD, cfg->draft.q_heads * D);
    F = std::max(F, cfg->draft.ffn);
    nq = std::max(nq, cfg->draft.q_heads);
    part = std::max(part, part_elems_for(c.drf, L.M, c.gemm_wide));
  }
  Carver cv{base};
  c.st = cv.take<SeqState>(L.B);
  c.hist = cv.take<int32_t>((size_t)L.B * L.cap);
  c.pt = cv.take<int32_t>((size_t)L.B * L.splits);
  c.pos3 = cv.take<int32_t>((size_t)L.B * 3 * L.cap);
  c.cs = cv.take<float2>((size_t)L.cap * (D / 2));
  c.tgt.axis = cv.take<int8_t>(D / 2);
  c.drf.axis = cv.take<int8_t>(D / 2);
  c.x = cv.take<float>((size_t)L.Mpad * H);
  c.q = cv.take<bf16_t>((size_t)L.Mpad * nqD);
  c.o = cv.take<bf16_t>((size_t)L.Mpad * nqD);
  c.u = cv.take<bf16_t>((size_t)L.Mpad * align_up(F, 32));   // row-major, or step-major for the packed path
  c.xg = cv.take<bf16_t>((size_t)L.Mpad * H);
  c.xgp = (c.gemm_wide && H % 32 == 0) ? cv.take<bf16_t>((size_t)L.Mpad * H) : nullptr;
  c.ss = cv.take<float>((size_t)(H / kTile) * L.Mpad);
  c.rcs = cv.take<float2>((size_t)L.Mpad * (D / 2));
  c.part = cv.take<float>(part);
  c.part_elems = part;
  const size_t attn_rows = (size_t)L.splits * L.B * nq * L.R;
  c.attn_rows = attn_rows;
  c.op = cv.take<bf16_t>(attn_rows * D);
  c.mp = cv.take<float>(attn_rows);
  c.lp = cv.take<float>(attn_rows);
  c.amax_v = cv.take<float>((size_t)(L.V / kTile) * L.Mpad);
  c.amax_i = cv.take<int32_t>((size_t)(L.V / kTile) * L.Mpad);
  c.logits = cv.take<bf16_t>((size_t)L.Mpad * L.V);
  c.cls = cv.take<int8_t>((size_t)L.B * L.cap);
  c.rp = cv.take<float>(attn_rows * 4);
  if (c.cond) {
    c.cat3 = cv.take<bf16_t>((size_t)L.Mpad * 3 * H);
    c.fusedp = cv.take<float>((size_t)kCondSplits * L.M * H);
    c.feat = cv.take<bf16_t>((size_t)L.B * L.cap * H);
    c.cat2 = cv.take<bf16_t>((size_t)L.Mpad * 2 * H);
  }
  c.tgt.kv_layer = (size_t)L.pool * t.kv_heads * kAttnChunk * D;
  c.tgt.kc = cv.take<bf16_t>(c.tgt.kv_layer * t.layers);
  c.tgt.vt = cv.take<bf16_t>(c.tgt.kv_layer * t.layers);
  if (has_draft) {
    c.drf.kv_layer = (size_t)L.pool * cfg->draft.kv_heads * kAttnChunk * D;
    c.drf.kc = cv.take<bf16_t>(c.drf.kv_layer * cfg->draft.layers);
    c.drf.vt = cv.take<bf16_t>(c.drf.kv_layer * cfg->draft.layers);
    if (c.cross) {
      c.junk_kc = cv.take<bf16_t>(c.drf.kv_layer);
      c.junk_vt = cv.take<bf16_t>(c.drf.kv_layer);
    }
  }
  // packed-weight path: passes of at most 32 rows on the layered path
  c.sg = false;
  const bool sg_ok = !(cfg->flags & SPEC_FLAG_ROWMAJOR) && L.M <= kSgMaxRows && sg_build_jobs(c, c.tgt, false, false) &&
                     (!has_draft || sg_build_jobs(c, c.drf, true, false));
  // passes on the batched-row GEMM stream the same tile-packed copy: every
  // wave load is then 1 KB of consecutive memory instead of 16 row pieces
  c.gemm_pk = !sg_ok && c.gemm_rows && !(cfg->flags & SPEC_FLAG_ROWMAJOR);
  // live-row compaction of chained draft steps (one row per sequence)
  c.Mpad1 = (int)align_up(L.B, 16);
  c.one_rows = has_draft && !c.block_draft && !c.cond && L.R > 1 && L.B <= kSgMaxRows && (sg_ok || c.gemm_pk) &&
               !(cfg->flags & SPEC_FLAG_FULL_DRAFT_ROWS) && sg_build_one(c, false);
  if (sg_ok || c.one_rows) {
    size_t pf = 0;
    int units = 0;
    auto fold = [&](const std::vector<SgJob>& js) {
      for (const SgJob& j : js) {
        pf = std::max(pf, sg_part_floats(j));
        units = std::max(units, j.units);
      }
    };
    if (sg_ok) {
      for (int k = 0; k < (has_draft ? 2 : 1); ++k) {
        const Model& mm = k ? c.drf : c.tgt;
        fold(mm.sg_host);
        fold(mm.sg_block);
      }
    }
    if (c.one_rows) fold(c.drf.sg_one);
    c.sg_part_floats = pf;
    c.sg_units = units;
    c.sg_part = cv.take<float>(pf);
    c.sg_cnt = cv.take<unsigned>((size_t)units + 1);   // + the LM head's fused-argmax counter
  }
  if (sg_ok || c.gemm_pk) {
    c.sg = sg_ok;
    pk_offsets(c.tgt);
    c.pk_head = cv.take<bf16_t>(sg_packed_elems(L.V / kTile, (H + 31) / 32));
    c.tgt.pk = cv.take<bf16_t>(c.tgt.pk_layer * t.layers);
    if (has_draft) {
      pk_offsets(c.drf);
      c.drf.pk = cv.take<bf16_t>(c.drf.pk_layer * cfg->draft.layers);
    }
  }
  return align_up(cv.off, kAlign);
}

// (p_T, p_H, p_W) per index: text -> (i, i, i); patch (t, h, w) of a block
// starting at s -> (s+t, s+h, s+w) (Sec. 3.3, Sec. 4.2).
void build_positions(const spec_seq_init& s, int cap, int32_t* out) {
  for (int i = 0; i < cap; ++i) out[i] = out[cap + i] = out[2 * cap + i] = i;
  for (int k = 0; k < s.n_blocks; ++k) {
    const spec_vision_block& v = s.blocks[k];
    int idx = v.start;
    for (int t = 0; t < v.t; ++t)
      for (int h = 0; h < v.h; ++h)
        for (int w = 0; w < v.w; ++w, ++idx) {
          out[idx] = v.start + t;
          out[cap + idx] = v.start + h;
          out[2 * cap + idx] = v.start + w;
        }
  }
}

// a(d) of Eq. axis-assign.
void build_axis(const spec_dims& d, bool flat, int8_t* out) {
  const int half = d.head_dim / 2;
  for (int i = 0; i < half; ++i) {
    if (flat) {
      out[i] = 0;
    } else if (d.interleaved) {
      out[i] = (int8_t)(i % 3);
    } else {
      out[i] = (int8_t)(i < d.mrope_section[0] ? 0 : (i < d.mrope_section[0] + d.mrope_section[1] ? 1 : 2));
    }
  }
}

spec_status fail_hip(Ctx& c, hipError_t e, const char* where) {
  c.poisoned = true;
  c.err = std::string(where) + ": " + hipGetErrorString(e);
  return SPEC_E_HIP;
}

spec_status set_err(Ctx& c, spec_status s, const char* msg) {
  c.err = msg;
  return s;
}

#define HIPCHK(c, expr, where)                       \
  do {                                               \
    hipError_t e_ = (expr);                          \
    if (e_ != hipSuccess) return fail_hip(c, e_, where); \
  } while (0)

// One pass; a block proposal is the draft's catch-up of accepted tokens and
// the block pass.
// A chained draft step after the first of a round, as a pass of one row per
// sequence on the packed GEMV: every live sequence consumes exactly its
// previous proposal then (draft_len == seq_len + dstep), so the rows
// b*(K+1)+1.. of the full pass would all be idle.
struct OneRowPass {
  Ctx& c;
  int R, M, Mpad;
  bool sg;
  explicit OneRowPass(Ctx& ctx) : c(ctx), R(ctx.R), M(ctx.M), Mpad(ctx.Mpad), sg(ctx.sg) {
    c.R = 1;
    c.M = c.B;
    c.Mpad = c.Mpad1;
    c.sg = true;
    c.drf.sg_host.swap(c.drf.sg_one);
  }
  ~OneRowPass() {
    c.R = R;
    c.M = M;
    c.Mpad = Mpad;
    c.sg = sg;
    c.drf.sg_host.swap(c.drf.sg_one);
  }
};

hipError_t launch_pass(Ctx& c, PassMode mode, bool one_row = false) {
  if (one_row) {
    OneRowPass shape(c);
    return launch_forward(c, PASS_DRAFT);
  }
  if (mode != PASS_BLOCK) return launch_forward(c, mode);
  const hipError_t e = launch_forward(c, PASS_CATCHUP);
  return e != hipSuccess ? e : launch_forward(c, PASS_BLOCK);
}

// Captures `launch` into `ge` on the capture stream (once; `ge` is reset by
// the caller when what the graph bakes in changes) and launches it.
template <class Launch>
spec_status run_graph(Ctx& c, hipGraphExec_t& ge, Launch&& launch) {
  if (!ge) {
    if (!c.cap_stream) HIPCHK(c, hipStreamCreateWithFlags(&c.cap_stream, hipStreamNonBlocking), "capture stream");
    hipStream_t user = c.stream;
    c.stream = c.cap_stream;
    hipGraph_t g = nullptr;
    hipError_t e = hipStreamBeginCapture(c.cap_stream, hipStreamCaptureModeThreadLocal);
    hipError_t el = hipSuccess;
    if (e == hipSuccess) {
      el = launch();
      e = hipStreamEndCapture(c.cap_stream, &g);
    }
    c.stream = user;
    if (el != hipSuccess) {
      if (g) (void)hipGraphDestroy(g);
      return fail_hip(c, el, "graph capture launch");
    }
    HIPCHK(c, e, "graph capture");
    e = hipGraphInstantiate(&ge, g, nullptr, nullptr, 0);
    (void)hipGraphDestroy(g);
    HIPCHK(c, e, "graph instantiate");
  }
  HIPCHK(c, hipGraphLaunch(ge, c.stream), "graph launch");
  return SPEC_OK;
}

// Runs one pass either directly or through its captured graph.  A draft
// pass's graph also writes the proposals to the caller's array, so it is
// captured again when that array changes.
spec_status run_pass(Ctx& c, PassMode mode) {
  const int mi = mode == PASS_VERIFY ? 0 : 1;
  const bool drafting = mode != PASS_VERIFY;
  if (c.ro_arm_out && c.ro_arm_model == mi) {
    // an armed readout: this pass is launched kernel by kernel with the
    // readout variants on its layer; graphs and later passes are unaffected
    c.ro_m = mi ? &c.drf : &c.tgt;
    c.ro_layer = c.ro_arm_layer;
    c.ro_out = c.ro_arm_out;
    c.ro_arm_out = nullptr;
    c.ro_arm_model = -1;
    const hipError_t e = launch_pass(c, mode);
    c.ro_m = nullptr;
    c.ro_out = nullptr;
    HIPCHK(c, e, "forward pass with readout");
    return SPEC_OK;
  }
  const bool one = c.one_rows && mode == PASS_DRAFT && c.dsteps > 0;
  const bool graphs = c.use_graphs && !c.timing;
  if (!graphs) {
    // timing mode: a head start so the timed kernels run back to back
    if (c.timing) HIPCHK(c, launch_hold(c, mode == PASS_VERIFY ? 4.0 : 1.0), "timing hold");
    HIPCHK(c, launch_pass(c, mode, one), "forward pass");
    return SPEC_OK;
  }
  if (drafting && c.g_draft_out != c.draft_out) {
    for (hipGraphExec_t* g : {&c.g_draft, &c.g_draft1})
      if (*g) {
        (void)hipGraphExecDestroy(*g);
        *g = nullptr;
      }
  }
  if (drafting) c.g_draft_out = c.draft_out;
  return run_graph(c, mode == PASS_VERIFY ? c.g_verify : (one ? c.g_draft1 : c.g_draft),
                   [&] { return launch_pass(c, mode, one); });
}

// The commit kernel runs through a graph of its own too: launched directly
// right after the verify graph it started about 8 us late on MI355X, while a
// graph after a graph starts at once.  Its output pointers are baked in.
spec_status run_commit(Ctx& c) {
  if (!c.use_graphs || c.timing) {
    HIPCHK(c, launch_commit(c, c.commit_out[0], c.commit_out[1], c.commit_out[2], c.commit_out[3]), "commit");
    return SPEC_OK;
  }
  if (c.g_commit && !std::equal(c.commit_out, c.commit_out + 4, c.g_commit_out)) {
    (void)hipGraphExecDestroy(c.g_commit);
    c.g_commit = nullptr;
  }
  std::copy(c.commit_out, c.commit_out + 4, c.g_commit_out);
  return run_graph(c, c.g_commit,
                   [&] { return launch_commit(c, c.commit_out[0], c.commit_out[1], c.commit_out[2], c.commit_out[3]); });
}

// Where spec_verify_scratch puts a verify's scratch inside the static array:
// the buffers spec_verify takes from the workspace for the duration of one
// pass (attention partials, partial sums and tiles, arrival counters, argmax
// pairs, logits staging).  Offsets are 256-byte aligned.
struct ScratchPlan {
  size_t op = 0, mp = 0, lp = 0, rp = 0, part = 0, sg_part = 0, sg_cnt = 0, amax_v = 0, amax_i = 0, logits = 0;
  size_t cnt_bytes = 0;   // counters to clear (a multiple of 16)
  size_t bytes = 0;
};

ScratchPlan scratch_plan(const Ctx& c) {
  ScratchPlan p;
  size_t off = 0;
  auto take = [&](size_t n) {
    off = align_up(off, kAlign);
    const size_t at = off;
    off += n;
    return at;
  };
  const int D = c.tgt.d.head_dim;
  const size_t amax = (size_t)(c.V / kTile) * c.Mpad;
  p.op = take(c.attn_rows * D * sizeof(bf16_t));
  p.mp = take(c.attn_rows * sizeof(float));
  p.lp = take(c.attn_rows * sizeof(float));
  p.rp = take(c.attn_rows * 4 * sizeof(float));
  p.part = take(c.part_elems * sizeof(float));
  p.sg_part = take(c.sg ? c.sg_part_floats * sizeof(float) : 0);
  p.cnt_bytes = c.sg ? align_up((size_t)(c.sg_units + 1) * sizeof(unsigned), 16) : 0;
  p.sg_cnt = take(p.cnt_bytes);
  p.amax_v = take(amax * sizeof(float));
  p.amax_i = take(amax * sizeof(int32_t));
  p.logits = take((size_t)c.Mpad * c.V * sizeof(bf16_t));
  p.bytes = align_up(off, kAlign);
  return p;
}

// Points the context's scratch buffers into the static array for the
// lifetime of the object, then restores the workspace's.
struct ScratchSwap {
  Ctx& c;
  bf16_t* op;
  float *mp, *lp, *rp, *part, *sg_part, *amax_v;
  unsigned* sg_cnt;
  int32_t* amax_i;
  bf16_t* logits;
  ScratchSwap(Ctx& ctx, char* base, const ScratchPlan& p)
      : c(ctx), op(ctx.op), mp(ctx.mp), lp(ctx.lp), rp(ctx.rp), part(ctx.part), sg_part(ctx.sg_part),
        amax_v(ctx.amax_v), sg_cnt(ctx.sg_cnt), amax_i(ctx.amax_i), logits(ctx.logits) {
    c.op = reinterpret_cast<bf16_t*>(base + p.op);
    c.mp = reinterpret_cast<float*>(base + p.mp);
    c.lp = reinterpret_cast<float*>(base + p.lp);
    c.rp = reinterpret_cast<float*>(base + p.rp);
    c.part = reinterpret_cast<float*>(base + p.part);
    c.sg_part = c.sg ? reinterpret_cast<float*>(base + p.sg_part) : nullptr;
    c.sg_cnt = c.sg ? reinterpret_cast<unsigned*>(base + p.sg_cnt) : nullptr;
    c.amax_v = reinterpret_cast<float*>(base + p.amax_v);
    c.amax_i = reinterpret_cast<int32_t*>(base + p.amax_i);
    c.logits = reinterpret_cast<bf16_t*>(base + p.logits);
  }
  ~ScratchSwap() {
    c.op = op;
    c.mp = mp;
    c.lp = lp;
    c.rp = rp;
    c.part = part;
    c.sg_part = sg_part;
    c.sg_cnt = sg_cnt;
    c.amax_v = amax_v;
    c.amax_i = amax_i;
    c.logits = logits;
  }
};

template <class F>
spec_status guarded(spec_ctx* ctx, F f) {
  if (!ctx) return SPEC_E_INVAL;
  if (ctx->c.poisoned) return SPEC_E_HIP;
  try {
    return f(ctx->c);
  } catch (const std::bad_alloc&) {
    ctx->c.err = "host out of memory";
    return SPEC_E_CAPACITY;
  } catch (const std::exception& ex) {
    ctx->c.err = ex.what();
    return SPEC_E_INVAL;
  }
}

}  // namespace

extern "C" {

int32_t spec_seq_pages(const spec_config* cfg, const spec_seq_init* seq) {
  if (!cfg || !seq || seq->prefix_len < 1 || cfg->max_new_tokens < 1 || cfg->K < 0) return -1;
  return seq_pages(cfg, *seq);
}

spec_status spec_workspace_bytes(const spec_config* cfg, const spec_seq_init* seqs, size_t* bytes) {
  if (!cfg || !seqs || !bytes) return SPEC_E_INVAL;
  try {
    std::string err;
    const bool has_draft = cfg->draft.layers > 0;
    if (!check_config(cfg, seqs, has_draft, err)) {
      g_init_error = err;
      return SPEC_E_INVAL;
    }
    const int M = cfg->batch * (cfg->K + 1);
    if (!check_fits(cfg->target, M, err, "target") || (has_draft && !check_fits(cfg->draft, M, err, "draft"))) {
      g_init_error = err;
      return SPEC_E_CAPACITY;
    }
    Ctx c;
    *bytes = carve(c, cfg, seqs, has_draft, nullptr);
    return SPEC_OK;
  } catch (...) {
    return SPEC_E_INVAL;
  }
}

spec_status spec_init(const spec_config* cfg, const void* embed, const spec_model_weights* target,
                      const spec_model_weights* draft, const spec_seq_init* seqs, void* workspace,
                      size_t workspace_bytes, hipStream_t stream, spec_ctx** out) {
  if (!out) return SPEC_E_INVAL;
  *out = nullptr;
  std::string err;
  const bool has_draft = cfg && cfg->draft.layers > 0;
  if (cfg && has_draft != (draft != nullptr)) {
    g_init_error = "draft weights must be given exactly when draft.layers > 0";
    return SPEC_E_INVAL;
  }
  if (!check_config(cfg, seqs, has_draft, err)) {
    g_init_error = err;
    return SPEC_E_INVAL;
  }
  if (!embed || !aligned16(embed)) {
    g_init_error = "embed: null or misaligned";
    return SPEC_E_INVAL;
  }
  if (!check_weights(target, cfg->target, err, "target") ||
      (has_draft && !check_weights(draft, cfg->draft, err, "draft")) ||
      ((cfg->flags & SPEC_FLAG_COND) && has_draft &&
       (!draft->w_fuse || !aligned16(draft->w_fuse) ||
        (!(cfg->flags & SPEC_FLAG_COND_CROSS) && (!draft->w_in || !aligned16(draft->w_in)))) &&
       (err = "SPEC_FLAG_COND: draft w_fuse / w_in null or misaligned", true))) {
    g_init_error = err;
    return SPEC_E_INVAL;
  }
  if (!workspace || (reinterpret_cast<uintptr_t>(workspace) % kAlign)) {
    g_init_error = "workspace: null or not 256-byte aligned";
    return SPEC_E_INVAL;
  }
  {
    const int M = cfg->batch * (cfg->K + 1);
    if (!check_fits(cfg->target, M, err, "target") || (has_draft && !check_fits(cfg->draft, M, err, "draft"))) {
      g_init_error = err;
      return SPEC_E_CAPACITY;
    }
  }
  spec_ctx* ctx = nullptr;
  try {
    ctx = new spec_ctx();
    Ctx& c = ctx->c;
    const size_t need = carve(c, cfg, seqs, has_draft, nullptr);
    if (workspace_bytes < need) {
      g_init_error = "workspace too small (query spec_workspace_bytes)";
      delete ctx;
      return SPEC_E_CAPACITY;
    }
    carve(c, cfg, seqs, has_draft, static_cast<char*>(workspace));
    c.cfg = *cfg;
    c.stream = stream;
    c.has_draft = has_draft;
    c.use_graphs = !(cfg->flags & SPEC_FLAG_NO_GRAPHS);
    c.embed = static_cast<const bf16_t*>(embed);
    auto load_model = [&](Model& m, const spec_model_weights* w) {
      m.final_norm = static_cast<const bf16_t*>(w->final_norm);
      m.L.resize(m.d.layers);
      for (int l = 0; l < m.d.layers; ++l) {
        const spec_layer_weights& s = w->layers[l];
        m.L[l] = LayerW{static_cast<const bf16_t*>(s.attn_norm), static_cast<const bf16_t*>(s.wq),
                        static_cast<const bf16_t*>(s.wk),        static_cast<const bf16_t*>(s.wv),
                        static_cast<const bf16_t*>(s.wo),        static_cast<const bf16_t*>(s.ffn_norm),
                        static_cast<const bf16_t*>(s.w_gate),    static_cast<const bf16_t*>(s.w_up),
                        static_cast<const bf16_t*>(s.w_down)};
      }
    };
    load_model(c.tgt, target);
    if (has_draft) load_model(c.drf, draft);
    if (c.cond) {
      c.w_fuse = static_cast<const bf16_t*>(draft->w_fuse);
      c.w_in = static_cast<const bf16_t*>(draft->w_in);
    }
    if (hipGetDevice(&c.device) != hipSuccess) c.device = 0;
    init_kernel_attributes();
    {
      // the static scratch array's address on this device (spec_verify_scratch)
      const hipError_t e = scratch_resolve(c.device);
      if (e != hipSuccess) {
        g_init_error = std::string("scratch symbol lookup: ") + hipGetErrorString(e);
        delete ctx;
        return SPEC_E_HIP;
      }
    }

    // host-built tables
    const int D = cfg->target.head_dim, half = D / 2;
    std::vector<int32_t> pos((size_t)c.B * 3 * c.cap);
    for (int b = 0; b < c.B; ++b) build_positions(seqs[b], c.cap, pos.data() + (size_t)b * 3 * c.cap);
    std::vector<float2> cs((size_t)c.cap * half);
    for (int p = 0; p < c.cap; ++p)
      for (int d = 0; d < half; ++d) {
        const double th = std::pow((double)cfg->target.rope_base, -2.0 * d / D);
        const double ang = th * (double)p;
        cs[(size_t)p * half + d] = make_float2((float)std::cos(ang), (float)std::sin(ang));
      }
    std::vector<int8_t> ax_t(half), ax_d(half);
    build_axis(cfg->target, false, ax_t.data());
    build_axis(cfg->draft, c.drf.flat, ax_d.data());
    c.pt_host.assign((size_t)c.B * c.pps, 0);
    c.npages.assign(c.B, 0);
    for (int b = 0, next = 0; b < c.B; ++b) {
      const int n = seq_pages(cfg, seqs[b]);
      c.npages[b] = n;
      for (int i = 0; i < n; ++i)
        c.pt_host[(size_t)b * c.pps + i] = seqs[b].page_table ? seqs[b].page_table[i] : next + i;
      next += n;
    }
    // token class of every slot for the attention-budget readout (Sec. 4.2):
    // vision-block slots, other prompt slots, generated slots
    std::vector<int8_t> cls((size_t)c.B * c.cap, 2);
    for (int b = 0; b < c.B; ++b) {
      int8_t* cb = cls.data() + (size_t)b * c.cap;
      std::fill(cb, cb + seqs[b].prefix_len, (int8_t)1);
      int ntraj = seqs[b].prefix_len;
      for (int i = 0; i < seqs[b].n_blocks; ++i) {
        const spec_vision_block& v = seqs[b].blocks[i];
        const int n = v.t * v.h * v.w;
        std::fill(cb + v.start, cb + v.start + n, (int8_t)0);
        ntraj -= n;
      }
      c.ro_inv_ln[b] = ntraj > 1 ? (float)(1.0 / std::log((double)ntraj)) : 0.f;
    }
    std::vector<SeqState> st(c.B);
    std::vector<int32_t> hist((size_t)c.B * c.cap, 0);
    for (int b = 0; b < c.B; ++b) {
      SeqState s{};
      s.seq_len = seqs[b].prefix_len;
      s.draft_len = seqs[b].prefix_len;
      s.pending = seqs[b].pending_token;
      s.prefix_len = seqs[b].prefix_len;
      st[b] = s;
      hist[(size_t)b * c.cap + seqs[b].prefix_len] = seqs[b].pending_token;
    }

    auto hip_fail = [&](hipError_t e, const char* where) {
      g_init_error = std::string(where) + ": " + hipGetErrorString(e);
      delete ctx;
      return SPEC_E_HIP;
    };
    hipError_t e;
    if ((e = launch_zero(c, workspace, need)) != hipSuccess) return hip_fail(e, "workspace clear");
    if ((e = hipMemcpyAsync(c.pos3, pos.data(), pos.size() * 4, hipMemcpyHostToDevice, stream)) != hipSuccess ||
        (e = hipMemcpyAsync(c.pt, c.pt_host.data(), c.pt_host.size() * 4, hipMemcpyHostToDevice, stream)) !=
            hipSuccess ||
        (e = hipMemcpyAsync(c.cs, cs.data(), cs.size() * sizeof(float2), hipMemcpyHostToDevice, stream)) !=
            hipSuccess ||
        (e = hipMemcpyAsync(c.tgt.axis, ax_t.data(), half, hipMemcpyHostToDevice, stream)) != hipSuccess ||
        (e = hipMemcpyAsync(c.drf.axis, ax_d.data(), half, hipMemcpyHostToDevice, stream)) != hipSuccess ||
        (e = hipMemcpyAsync(c.st, st.data(), st.size() * sizeof(SeqState), hipMemcpyHostToDevice, stream)) !=
            hipSuccess ||
        (e = hipMemcpyAsync(c.hist, hist.data(), hist.size() * 4, hipMemcpyHostToDevice, stream)) != hipSuccess ||
        (e = hipMemcpyAsync(c.cls, cls.data(), cls.size(), hipMemcpyHostToDevice, stream)) != hipSuccess)
      return hip_fail(e, "table upload");
    if (c.sg) {
      if (!sg_build_jobs(c, c.tgt, false, true) || (has_draft && !sg_build_jobs(c, c.drf, true, true))) {
        g_init_error = "packed GEMV plan changed between sizing and init";
        delete ctx;
        return SPEC_E_INVAL;
      }
      if ((e = sg_pack_head(c)) != hipSuccess || (e = sg_pack_model(c, c.tgt)) != hipSuccess ||
          (has_draft && (e = sg_pack_model(c, c.drf)) != hipSuccess))
        return hip_fail(e, "weight packing");
    }
    if (c.one_rows && !sg_build_one(c, true)) {
      g_init_error = "packed GEMV plan of the one-row draft pass changed between sizing and init";
      delete ctx;
      return SPEC_E_INVAL;
    }
    if (c.gemm_pk) {
      if ((e = sg_pack_head(c)) != hipSuccess || (e = sg_pack_model(c, c.tgt)) != hipSuccess ||
          (has_draft && (e = sg_pack_model(c, c.drf)) != hipSuccess))
        return hip_fail(e, "weight packing");
    }
    for (int b = 0; b < c.B; ++b) {
      for (int l = 0; l < c.tgt.d.layers; ++l)
        if ((e = launch_prefix_kv(c, c.tgt, l, b, seqs[b].prefix_len, static_cast<const bf16_t*>(seqs[b].tgt_k[l]),
                                  static_cast<const bf16_t*>(seqs[b].tgt_v[l]))) != hipSuccess)
          return hip_fail(e, "prefix K/V");
      if (has_draft)
        for (int l = 0; l < c.drf.d.layers; ++l)
          if ((e = launch_prefix_kv(c, c.drf, l, b, seqs[b].prefix_len,
                                    static_cast<const bf16_t*>(seqs[b].drf_k[l]),
                                    static_cast<const bf16_t*>(seqs[b].drf_v[l]))) != hipSuccess)
            return hip_fail(e, "prefix K/V");
    }
    // The host tables above are pageable and local: wait for the uploads.
    if ((e = hipStreamSynchronize(stream)) != hipSuccess) return hip_fail(e, "init sync");
    *out = ctx;
    return SPEC_OK;
  } catch (const std::bad_alloc&) {
    delete ctx;
    g_init_error = "host out of memory";
    return SPEC_E_CAPACITY;
  } catch (const std::exception& ex) {
    delete ctx;
    g_init_error = ex.what();
    return SPEC_E_INVAL;
  }
}

spec_status draft_step(spec_ctx* ctx, int32_t* d_draft_tokens) {
  return guarded(ctx, [&](Ctx& c) -> spec_status {
    if (!c.has_draft) return set_err(c, SPEC_E_STATE, "draft_step: no draft model");
    if (c.K < 1) return set_err(c, SPEC_E_STATE, "draft_step: K is 0");
    if (c.phase == Ctx::VERIFIED) return set_err(c, SPEC_E_STATE, "draft_step: commit the last verify first");
    if (c.dsteps >= c.K) return set_err(c, SPEC_E_STATE, "draft_step: K steps already taken this round");
    c.draft_out = d_draft_tokens;
    spec_status s = run_pass(c, c.block_draft ? PASS_BLOCK : PASS_DRAFT);
    if (s != SPEC_OK) return s;
    c.dsteps += c.block_draft ? c.K : 1;
    c.phase = Ctx::DRAFTING;
    return SPEC_OK;
  });
}

spec_status draft_steps(spec_ctx* ctx, int32_t n, int32_t* d_draft_tokens) {
  return guarded(ctx, [&](Ctx& c) -> spec_status {
    if (!c.has_draft) return set_err(c, SPEC_E_STATE, "draft_steps: no draft model");
    if (c.K < 1) return set_err(c, SPEC_E_STATE, "draft_steps: K is 0");
    if (c.phase == Ctx::VERIFIED) return set_err(c, SPEC_E_STATE, "draft_steps: commit the last verify first");
    if (n < 1 || n > c.K - c.dsteps) return set_err(c, SPEC_E_STATE, "draft_steps: n must be 1..K minus the steps taken");
    if (c.block_draft) {
      if (n != c.K) return set_err(c, SPEC_E_STATE, "draft_steps: the block proposal takes n = K");
      c.draft_out = d_draft_tokens;
      spec_status s = run_pass(c, PASS_BLOCK);
      if (s != SPEC_OK) return s;
      c.dsteps = c.K;
      c.phase = Ctx::DRAFTING;
      return SPEC_OK;
    }
    c.draft_out = d_draft_tokens;
    if (n == 1 || !c.use_graphs || c.timing || (c.ro_arm_out && c.ro_arm_model == 1)) {
      for (int i = 0; i < n; ++i) {
        spec_status s = run_pass(c, PASS_DRAFT);
        if (s != SPEC_OK) return s;
        c.dsteps += 1;
      }
    } else {
      const bool first = c.dsteps == 0;
      if (c.g_drafts && (c.g_drafts_n != n || c.g_drafts_out != d_draft_tokens || c.g_drafts_first != first)) {
        (void)hipGraphExecDestroy(c.g_drafts);
        c.g_drafts = nullptr;
      }
      c.g_drafts_n = n;
      c.g_drafts_out = d_draft_tokens;
      c.g_drafts_first = first;
      spec_status s = run_graph(c, c.g_drafts, [&]() -> hipError_t {
        for (int i = 0; i < n; ++i) {
          const hipError_t e = launch_pass(c, PASS_DRAFT, c.one_rows && (!first || i > 0));
          if (e != hipSuccess) return e;
        }
        return hipSuccess;
      });
      if (s != SPEC_OK) return s;
      c.dsteps += n;
    }
    c.phase = Ctx::DRAFTING;
    return SPEC_OK;
  });
}

spec_status spec_verify(spec_ctx* ctx, const int32_t* d_draft_tokens, void* d_logits) {
  return guarded(ctx, [&](Ctx& c) -> spec_status {
    if (c.phase == Ctx::VERIFIED) return set_err(c, SPEC_E_STATE, "spec_verify: commit the last verify first");
    if (!d_draft_tokens && c.K > 0 && c.dsteps != c.K)
      return set_err(c, SPEC_E_STATE, "spec_verify: no draft tokens given and fewer than K draft steps taken");
    HIPCHK(c, launch_stage_verify(c, c.K > 0 ? d_draft_tokens : nullptr, d_logits ? 1 : 0), "verify staging");
    spec_status s = run_pass(c, PASS_VERIFY);
    if (s != SPEC_OK) return s;
    HIPCHK(c, launch_logits_out(c, d_logits), "logits copy");
    c.phase = Ctx::VERIFIED;
    return SPEC_OK;
  });
}

spec_status spec_verify_scratch(spec_ctx* ctx, const int32_t* d_draft_tokens, void* d_logits) {
  return guarded(ctx, [&](Ctx& c) -> spec_status {
    if (c.phase == Ctx::VERIFIED)
      return set_err(c, SPEC_E_STATE, "spec_verify_scratch: commit the last verify first");
    if (!d_draft_tokens && c.K > 0 && c.dsteps != c.K)
      return set_err(c, SPEC_E_STATE,
                     "spec_verify_scratch: no draft tokens given and fewer than K draft steps taken");
    const ScratchPlan plan = scratch_plan(c);
    if (plan.bytes > scratch_capacity()) {
      char buf[200];
      snprintf(buf, sizeof buf,
               "spec_verify_scratch: this context's verify needs %zu bytes of scratch, more than the %zu-byte "
               "static array (SPEC_SCRATCH_BYTES)",
               plan.bytes, scratch_capacity());
      return set_err(c, SPEC_E_CAPACITY, buf);
    }
    char* base = static_cast<char*>(scratch_device_ptr(c.device));
    if (!base) return set_err(c, SPEC_E_STATE, "spec_verify_scratch: scratch address not resolved on this device");
    ScratchSwap swap(c, base, plan);
    // arrival counters start at zero (every launch leaves them at zero, but
    // the array is shared with every other context on this GPU)
    if (plan.cnt_bytes) HIPCHK(c, launch_zero(c, c.sg_cnt, plan.cnt_bytes), "scratch counter clear");
    HIPCHK(c, launch_stage_verify(c, c.K > 0 ? d_draft_tokens : nullptr, d_logits ? 1 : 0), "verify staging");
    if (c.ro_arm_out && c.ro_arm_model == 0) {
      c.ro_m = &c.tgt;
      c.ro_layer = c.ro_arm_layer;
      c.ro_out = c.ro_arm_out;
      c.ro_arm_out = nullptr;
      c.ro_arm_model = -1;
    }
    if (c.timing) HIPCHK(c, launch_hold(c, 4.0), "timing hold");
    const hipError_t e = launch_pass(c, PASS_VERIFY);
    c.ro_m = nullptr;
    c.ro_out = nullptr;
    HIPCHK(c, e, "forward pass");
    HIPCHK(c, launch_logits_out(c, d_logits), "logits copy");
    c.phase = Ctx::VERIFIED;
    return SPEC_OK;
  });
}

spec_status spec_commit(spec_ctx* ctx, int32_t* d_accept_len, int32_t* d_committed, int32_t* d_n_committed,
                        int32_t* d_finished) {
  return guarded(ctx, [&](Ctx& c) -> spec_status {
    if (c.phase != Ctx::VERIFIED) return set_err(c, SPEC_E_STATE, "spec_commit: no verify to commit");
    c.commit_out[0] = d_accept_len;
    c.commit_out[1] = d_committed;
    c.commit_out[2] = d_n_committed;
    c.commit_out[3] = d_finished;
    spec_status s = run_commit(c);
    if (s != SPEC_OK) return s;
    c.phase = Ctx::READY;
    c.dsteps = 0;
    return SPEC_OK;
  });
}

spec_status spec_attn_readout(spec_ctx* ctx, int32_t model, int32_t layer, float* d_out) {
  return guarded(ctx, [&](Ctx& c) -> spec_status {
    if (!d_out) {
      c.ro_arm_out = nullptr;
      c.ro_arm_model = -1;
      return SPEC_OK;
    }
    if (model != 0 && model != 1) return set_err(c, SPEC_E_INVAL, "spec_attn_readout: model must be 0 or 1");
    if (model == 1 && !c.has_draft) return set_err(c, SPEC_E_STATE, "spec_attn_readout: no draft model");
    const Model& m = model ? c.drf : c.tgt;
    if (layer < 0 || layer >= m.d.layers) return set_err(c, SPEC_E_INVAL, "spec_attn_readout: layer out of range");
    if (!aligned16(d_out)) return set_err(c, SPEC_E_INVAL, "spec_attn_readout: d_out must be 16-byte aligned");
    c.ro_arm_model = model;
    c.ro_arm_layer = layer;
    c.ro_arm_out = d_out;
    return SPEC_OK;
  });
}

spec_status spec_sync(spec_ctx* ctx, int32_t* n_finished) {
  return guarded(ctx, [&](Ctx& c) -> spec_status {
    std::vector<SeqState> st(c.B);
    HIPCHK(c, hipMemcpyAsync(st.data(), c.st, st.size() * sizeof(SeqState), hipMemcpyDeviceToHost, c.stream),
           "state read");
    HIPCHK(c, hipStreamSynchronize(c.stream), "sync");
    int fin = 0, err = 0;
    for (const SeqState& s : st) {
      fin += s.finished ? 1 : 0;
      err |= s.err;
    }
    if (n_finished) *n_finished = fin;
    if (err & ERR_NUMERIC) return set_err(c, SPEC_E_NUMERIC, "NaN logits seen on the device");
    if (err & ERR_TOKEN) return set_err(c, SPEC_E_INVAL, "a draft token id was out of range (replaced by 0)");
    if (err & ERR_STATE) return set_err(c, SPEC_E_STATE, "draft catch-up exceeded K+1 rows");
    return SPEC_OK;
  });
}

void spec_destroy(spec_ctx* ctx) {
  if (!ctx) return;
  Ctx& c = ctx->c;
  if (c.stream) (void)hipStreamSynchronize(c.stream);
  if (c.g_verify) (void)hipGraphExecDestroy(c.g_verify);
  if (c.g_draft) (void)hipGraphExecDestroy(c.g_draft);
  if (c.g_draft1) (void)hipGraphExecDestroy(c.g_draft1);
  if (c.g_commit) (void)hipGraphExecDestroy(c.g_commit);
  if (c.g_drafts) (void)hipGraphExecDestroy(c.g_drafts);
  if (c.cap_stream) (void)hipStreamDestroy(c.cap_stream);
  for (hipEvent_t e : c.ev_pool) (void)hipEventDestroy(e);
  delete ctx;
}

const char* spec_last_error(const spec_ctx* ctx) {
  if (!ctx) return g_init_error.c_str();
  return ctx->c.err.c_str();
}

spec_status spec_debug_positions(spec_ctx* ctx, int32_t b, int32_t* host_out, int32_t len) {
  return guarded(ctx, [&](Ctx& c) -> spec_status {
    if (b < 0 || b >= c.B || !host_out || len < 0 || len > c.cap) return set_err(c, SPEC_E_INVAL, "bad arguments");
    HIPCHK(c, hipStreamSynchronize(c.stream), "sync");
    for (int a = 0; a < 3; ++a)
      HIPCHK(c, hipMemcpy(host_out + (size_t)a * len, c.pos3 + ((size_t)b * 3 + a) * c.cap, (size_t)len * 4,
                          hipMemcpyDeviceToHost),
             "positions read");
    return SPEC_OK;
  });
}

spec_status spec_debug_state(spec_ctx* ctx, int32_t b, int32_t* host_out) {
  return guarded(ctx, [&](Ctx& c) -> spec_status {
    if (b < 0 || b >= c.B || !host_out) return set_err(c, SPEC_E_INVAL, "bad arguments");
    SeqState s;
    HIPCHK(c, hipStreamSynchronize(c.stream), "sync");
    HIPCHK(c, hipMemcpy(&s, c.st + b, sizeof s, hipMemcpyDeviceToHost), "state read");
    const int32_t v[8] = {s.seq_len, s.draft_len, s.pending, s.n_gen, s.finished, s.accept_len, s.n_commit, s.err};
    memcpy(host_out, v, sizeof v);
    return SPEC_OK;
  });
}

spec_status spec_debug_feature(spec_ctx* ctx, int32_t b, int32_t slot0, int32_t n, void* host_out) {
  return guarded(ctx, [&](Ctx& c) -> spec_status {
    if (!c.cond) return set_err(c, SPEC_E_STATE, "spec_debug_feature: the draft is not conditioned");
    if (b < 0 || b >= c.B || slot0 < 0 || n < 0 || slot0 + n > c.cap || (n > 0 && !host_out))
      return set_err(c, SPEC_E_INVAL, "bad arguments");
    HIPCHK(c, hipStreamSynchronize(c.stream), "sync");
    const size_t H = c.tgt.d.hidden;
    HIPCHK(c, hipMemcpy(host_out, c.feat + ((size_t)b * c.cap + slot0) * H, (size_t)n * H * sizeof(bf16_t),
                        hipMemcpyDeviceToHost),
           "feature copy");
    return SPEC_OK;
  });
}

spec_status spec_debug_path(const spec_ctx* ctx, int32_t* path) {
  if (!ctx || !path) return SPEC_E_INVAL;
  const Ctx& c = ctx->c;
  *path = (c.sg || c.gemm_pk) ? SPEC_PATH_PACKED : SPEC_PATH_ROWMAJOR;
  return SPEC_OK;
}

spec_status spec_debug_kv(spec_ctx* ctx, int32_t b, int32_t model, int32_t layer, int32_t which, int32_t pos0,
                          int32_t npos, void* host_out) {
  return guarded(ctx, [&](Ctx& c) -> spec_status {
    if (model != 0 && !(model == 1 && c.has_draft)) return set_err(c, SPEC_E_INVAL, "bad model");
    Model& m = model == 0 ? c.tgt : c.drf;
    if (b < 0 || b >= c.B || layer < 0 || layer >= m.d.layers || (which != 0 && which != 1) || pos0 < 0 ||
        npos < 0 || pos0 + npos > c.npages[b] * kAttnChunk || !host_out)
      return set_err(c, SPEC_E_INVAL, "bad arguments");
    HIPCHK(c, hipStreamSynchronize(c.stream), "sync");
    const int nkv = m.d.kv_heads, D = m.d.head_dim;
    bf16_t* out = static_cast<bf16_t*>(host_out);
    // one page (all kv heads) at a time: keys [nkv][page][D], values [nkv][D][page]
    const size_t page_elems = (size_t)nkv * kAttnChunk * D;
    std::vector<bf16_t> tmp(page_elems);
    for (int s = pos0; s < pos0 + npos;) {
      const int pi = s / kAttnChunk, off = s % kAttnChunk;
      const int n = std::min(kAttnChunk - off, pos0 + npos - s);
      const bf16_t* src = (which == 0 ? m.kc : m.vt) + m.kv_layer * layer +
                          (size_t)c.pt_host[(size_t)b * c.pps + pi] * page_elems;
      HIPCHK(c, hipMemcpy(tmp.data(), src, page_elems * 2, hipMemcpyDeviceToHost), "kv read");
      for (int i = 0; i < n; ++i)
        for (int h = 0; h < nkv; ++h)
          for (int d = 0; d < D; ++d)
            out[((size_t)(s - pos0 + i) * nkv + h) * D + d] =
                which == 0 ? tmp[((size_t)h * kAttnChunk + off + i) * D + d]
                           : tmp[((size_t)h * D + d) * kAttnChunk + off + i];
      s += n;
    }
    return SPEC_OK;
  });
}

spec_status spec_stream_read(const void* d_buf, size_t bytes, uint32_t* d_sink, int32_t sink_words,
                            hipStream_t stream) {
  if (!d_buf || !d_sink || bytes == 0 || bytes % 16 || !aligned16(d_buf) || sink_words < 4 || sink_words % 4)
    return SPEC_E_INVAL;
  return launch_stream_read(d_buf, bytes, d_sink, sink_words, stream) == hipSuccess ? SPEC_OK : SPEC_E_HIP;
}

spec_status spec_timing(spec_ctx* ctx, int32_t enable) {
  return guarded(ctx, [&](Ctx& c) -> spec_status {
    HIPCHK(c, hipStreamSynchronize(c.stream), "sync");
    c.timing = enable != 0;
    c.trec.clear();
    c.ev_used = 0;
    for (int k = 0; k < SPEC_KERNEL_KINDS; ++k) {
      c.t_launches[k] = 0;
      c.t_ms[k] = 0.0;
      c.t_bytes[k] = 0.0;
    }
    return SPEC_OK;
  });
}

spec_status spec_timing_read(spec_ctx* ctx, int32_t kind, int64_t* launches, double* ms, double* bytes) {
  return guarded(ctx, [&](Ctx& c) -> spec_status {
    if (kind < 0 || kind >= SPEC_KERNEL_KINDS) return set_err(c, SPEC_E_INVAL, "bad kernel kind");
    HIPCHK(c, hipStreamSynchronize(c.stream), "sync");
    for (const TimingRec& r : c.trec) {
      float t = 0.f;
      HIPCHK(c, hipEventElapsedTime(&t, r.e0, r.e1), "event time");
      c.t_launches[r.kind] += 1;
      c.t_ms[r.kind] += t;
      c.t_bytes[r.kind] += r.bytes;
    }
    c.trec.clear();
    c.ev_used = 0;
    if (launches) *launches = c.t_launches[kind];
    if (ms) *ms = c.t_ms[kind];
    if (bytes) *bytes = c.t_bytes[kind];
    return SPEC_OK;
  });
}

}  // extern "C"
