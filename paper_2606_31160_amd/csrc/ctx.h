// Internal definitions shared by the host runtime (runtime.cpp) and the
// gfx950 kernels (kernels.hip).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <string>
#include <vector>

#include "../../include/spec.h"

namespace specdec {

typedef uint16_t bf16_t;
struct SgJob;

constexpr int kMaxRows = SPEC_MAX_K + 1;     // rows per sequence in one pass
constexpr int kTile = 16;                    // output rows per GEMV tile (one MFMA block)
constexpr int kKeyBlock = 32;                // keys per attention inner step
constexpr int kAttnChunk = SPEC_KV_PAGE;     // keys per attention workgroup (split-KV chunk) = one cache page
constexpr int kGemvWaves = 16;               // waves per GEMV workgroup
constexpr int kGemvSteps = 8;                // max 32-wide k-steps per GEMV wave

// Per-sequence state, resident in device memory.  Only kernels change it
// between spec_init and spec_destroy, so a captured graph stays valid for
// every round.
struct SeqState {
  int32_t seq_len;      // slots holding target K/V = index of the pending token
  int32_t draft_len;    // slots holding draft K/V
  int32_t pending;      // token at index seq_len
  int32_t n_gen;        // committed tokens so far
  int32_t finished;
  int32_t dstep;        // draft steps taken this round
  int32_t accept_len;   // l of the last verify
  int32_t n_commit;     // tokens the last verify commits (after stop / budget cut)
  int32_t fin_pending;  // the last verify ends the sequence
  int32_t err;          // sticky ERR_* bits
  int32_t prefix_len;
  int32_t want_logits;  // the current verify copies bf16 logits out
  int32_t base;         // slot of row 0 of the current pass
  int32_t count;        // valid rows of the current pass (0 when idle)
  int32_t dcall;        // draft_step calls this round (the output column of the next one)
  int32_t causal;       // rows 0..causal-1 of the current pass attend causally; the rest see
                        // every row of the pass (a block proposal's MASK rows)
  int32_t vtok[kMaxRows];       // verify rows: pending, d_1..d_K
  int32_t rstar[kMaxRows];      // greedy token of each verify row
  int32_t committed[kMaxRows];  // tokens of the last verify to commit
  int32_t props[kMaxRows];      // the draft's own proposals this round
};

enum { ERR_TOKEN = 1, ERR_NUMERIC = 2, ERR_STATE = 4 };

constexpr int kCondSplits = 4;   // k-splits of the feature fusion (3H inputs) and of the input projection

// Passes: the target's verify; one draft step (consume, propose from the last
// row); for the single-forward block proposal, the draft's causal catch-up of
// committed tokens it has not consumed (no LM head) and the block pass itself.
enum PassMode { PASS_VERIFY = 0, PASS_DRAFT = 1, PASS_CATCHUP = 2, PASS_BLOCK = 3, PASS_CTX = 4 };

struct LayerW {
  const bf16_t *attn_norm, *wq, *wk, *wv, *wo, *ffn_norm, *wg, *wu, *wd;
};

struct Model {
  spec_dims d{};
  bool flat = false;                // FlatRoPE (draft) instead of 3D M-RoPE (target)
  std::vector<LayerW> L;
  const bf16_t* final_norm = nullptr;
  bf16_t* kc = nullptr;             // [layers][pool pages][kv_heads][kAttnChunk][head_dim], rotated keys
  bf16_t* vt = nullptr;             // [layers][pool pages][kv_heads][head_dim][kAttnChunk], values transposed
  int8_t* axis = nullptr;           // [head_dim/2] axis (0 T, 1 H, 2 W) of each rotary pair
  int s_down = 1;                  // k-splits of the down projection
  int s_o = 1;                     // k-splits of the o projection on the batched-row GEMM
  size_t kv_layer = 0;              // elements of one layer's key (or value) cache
  // tile-packed weights (sgemv.h) of every layer: q/k/v, o, gate/up pairs, down
  bf16_t* pk = nullptr;
  size_t pk_layer = 0, pk_o = 0, pk_gu = 0, pk_dn = 0;   // elements per layer; offsets inside a layer
  std::vector<SgJob> sg_host;       // [layers][4] (q/k/v, o, gate/up, down) + the LM head
  std::vector<SgJob> sg_block;      // draft, block proposal: the last layer's down for every row, the LM head over all rows
  std::vector<SgJob> sg_one;        // draft, steps after the first of a round: the sg_host jobs for one row per sequence
};

struct TimingRec {
  int kind;
  double bytes;
  hipEvent_t e0, e1;
};

struct Ctx {
  spec_config cfg{};
  int B = 1, K = 0, R = 1, M = 1, Mpad = 16, V = 0, cap = 0;
  int attn_chunk = kAttnChunk, attn_splits = 1;
  int attn_ppw = 1;                  // pages per attention workgroup (several for many sequences)
  int pps = 1;                       // page-table entries per sequence (cap / kAttnChunk)
  int pool = 0;                      // cache pages per layer
  std::vector<int32_t> pt_host;      // [B][pps] physical page of each sequence page
  std::vector<int32_t> npages;       // [B] pages each sequence owns
  int ncu = 256;                     // compute units of the device (GEMV grids)
  hipStream_t stream = nullptr;      // caller's stream
  hipStream_t cap_stream = nullptr;  // private stream used only for graph capture
  int device = 0;

  // workspace carve-out
  SeqState* st = nullptr;           // [B]
  int32_t* hist = nullptr;          // [B][cap] token at each index >= prefix_len
  int32_t* pt = nullptr;            // [B][pps] page table (slot s of sequence b: page pt[b][s / kAttnChunk])
  int32_t* pos3 = nullptr;          // [B][3][cap] target rotary positions
  float2* cs = nullptr;             // [cap][head_dim/2] (cos, sin) of theta_d * p
  float* x = nullptr;               // [Mpad][hidden] residual stream
  bf16_t* q = nullptr;              // [Mpad][q_heads*head_dim] rotated queries
  bf16_t* o = nullptr;              // [Mpad][q_heads*head_dim] attention output
  bf16_t* u = nullptr;              // [Mpad][ffn] SwiGLU output (max of both models)
  bf16_t* xg = nullptr;             // [Mpad][hidden] bf16(x * gain of the next RMSNorm)
  float* ss = nullptr;              // [hidden/16][Mpad] per-16-column sums of x^2
  float2* rcs = nullptr;            // [Mpad][head_dim/2] (cos, sin) of each row's rotary pairs
  float* part = nullptr;            // GEMV k-split partial sums
  size_t part_elems = 0;
  bf16_t* op = nullptr;             // [splits][B][q_heads][R][head_dim] attention partials (unnormalised)
  size_t attn_rows = 0;             // splits * B * q_heads * R (max over the models)
  float* mp = nullptr;              // [splits][B][q_heads][R] running max (log2 units)
  float* lp = nullptr;              // [splits][B][q_heads][R] running sum
  float* amax_v = nullptr;          // [vocab/16][Mpad] per-tile maximum logit
  int32_t* amax_i = nullptr;        // [vocab/16][Mpad] its index
  bf16_t* logits = nullptr;         // [Mpad][vocab] bf16 logits of the last verify
  int8_t* cls = nullptr;            // [B][cap] class of every slot: 0 visual, 1 trajectory/text, 2 generated
  float* rp = nullptr;              // [splits][B][q_heads][R][4] attention-budget readout partials

  const bf16_t* embed = nullptr;
  Model tgt, drf;

  // packed-weight path (passes of at most 16 rows)
  bool sg = false;
  bf16_t* pk_head = nullptr;        // tile-packed LM head (shared by both models)
  float* sg_part = nullptr;         // partial tiles of split units
  unsigned* sg_cnt = nullptr;       // arrival counters
  size_t sg_part_floats = 0;
  int sg_units = 0;
  bool has_draft = false;
  bool block_draft = false;          // SPEC_FLAG_BLOCK_DRAFT: draft_step proposes all K in one forward
  int mask_token = 0;                // input token of the block's MASK rows
  // SPEC_FLAG_COND: the draft conditioned on target hidden states
  bool cond = false;
  int cond_layers[3] = {};
  const bf16_t* w_fuse = nullptr;    // [H][3H]
  const bf16_t* w_in = nullptr;      // [H][2H]
  bf16_t* cat3 = nullptr;            // [Mpad][3H] verify rows' residual streams after cond_layers
  float* fusedp = nullptr;           // [kCondSplits][M][H] k-split partial sums of w_fuse . cat3
  bf16_t* feat = nullptr;            // [B][cap][H] fused feature of every verified slot
  bf16_t* cat2 = nullptr;            // [Mpad][2H] draft rows' [embedding; feature of the previous slot]
  // SPEC_FLAG_COND_CROSS: the features are the draft's layer-0 cross-attention
  // context instead of an input term; that layer's own K/V appends go to
  // these unread pools (one draft layer's worth each)
  bool cross = false;
  bf16_t* junk_kc = nullptr;
  bf16_t* junk_vt = nullptr;

  // host state machine
  enum Phase { READY = 0, DRAFTING = 1, VERIFIED = 2 } phase = READY;
  int dsteps = 0;
  bool one_rows = false;             // draft steps after a round's first run as passes of one row per sequence
  int Mpad1 = 16;                    // ... whose row count B is padded to this
  bool gemm_rows = false;              // layered row-major passes run on the batched-row GEMM
  bool gemm_pk = false;                // ... which streams the tile-packed weight copy
  bool gemm_wide = false;              // ... on the wide-unit kernel (passes of more than 32 rows)
  bf16_t* xgp = nullptr;               // wide contexts: step-major copy of xg [H/32][M][32] for that kernel
  bool poisoned = false;
  std::string err;

  // graphs
  bool use_graphs = true;
  hipGraphExec_t g_verify = nullptr, g_draft = nullptr, g_commit = nullptr;
  hipGraphExec_t g_draft1 = nullptr;             // the one-row-per-sequence draft pass
  int32_t* draft_out = nullptr;                  // draft_step's output array (baked into the draft graph)
  int32_t* g_draft_out = nullptr;                // ... the one the current draft graph writes
  hipGraphExec_t g_drafts = nullptr;             // n draft passes in one graph (draft_steps)
  int g_drafts_n = 0;
  bool g_drafts_first = false;                   // ... its first pass is a round's first (full rows)
  int32_t* g_drafts_out = nullptr;
  int32_t* commit_out[4] = {};                   // spec_commit's outputs (baked into the commit graph)
  int32_t* g_commit_out[4] = {};

  // attention-budget readout: armed by spec_attn_readout, active during the
  // one pass it applies to
  float ro_inv_ln[SPEC_MAX_BATCH] = {};   // 1 / ln(trajectory/text slots) per sequence, 0 if <= 1
  int ro_arm_model = -1, ro_arm_layer = 0;
  float* ro_arm_out = nullptr;
  const Model* ro_m = nullptr;
  int ro_layer = 0;
  float* ro_out = nullptr;

  // timing
  bool timing = false;
  std::vector<TimingRec> trec;
  std::vector<hipEvent_t> ev_pool;
  size_t ev_used = 0;
  int64_t t_launches[SPEC_KERNEL_KINDS] = {};
  double t_ms[SPEC_KERNEL_KINDS] = {}, t_bytes[SPEC_KERNEL_KINDS] = {};
};

// ---- launchers (kernels.hip) ------------------------------------------------
// Each returns hipSuccess or the launch error.

hipError_t launch_zero(Ctx& c, void* p, size_t bytes);
hipError_t launch_stream_read(const void* p, size_t bytes, uint32_t* sink, int sink_words, hipStream_t s);
hipError_t launch_hold(Ctx& c, double ms);   // bounded device-side wait (timing mode)
hipError_t launch_prefix_kv(Ctx& c, Model& m, int layer, int b, int prefix_len,
                            const bf16_t* k_pre, const bf16_t* v);
hipError_t launch_stage_verify(Ctx& c, const int32_t* d_override, int want_logits);
hipError_t launch_forward(Ctx& c, PassMode mode);   // embed .. accept / draft pick
hipError_t launch_commit(Ctx& c, int32_t* acc, int32_t* committed, int32_t* ncommit, int32_t* fin);
hipError_t launch_logits_out(Ctx& c, void* d_logits);
// Packed-weight path: plans (and, with fill, points) every GEMV job of a model;
// false if a shape does not fit.  Packs a model's weights / the LM head.
bool sg_build_jobs(Ctx& c, Model& m, bool draft, bool fill);
// Offsets of o, gate/up and down inside a layer of the tile-packed copy, and its elements per layer.
void pk_offsets(Model& m);
hipError_t sg_pack_model(Ctx& c, Model& m);
hipError_t sg_pack_head(Ctx& c);

// The library's static per-device scratch array (scratch.hip): its device
// address on the current device, resolved once per device (spec_init).
hipError_t scratch_resolve(int device);
void* scratch_device_ptr(int device);
size_t scratch_capacity();

// Dynamic LDS bytes one GEMV workgroup needs (TT tiles, M rows, span k-steps)
// and the device limit; k-splits of a GEMV whose workgroups cannot hold all
// of x.
size_t gemv_lds_bytes(int TT, int M, int span_steps);
int gemv_lds_limit();
size_t gemv_p_lds_bytes(int M, int span_steps);
int down_splits(int M, int Kd, int ncu);
int num_cus();
void init_kernel_attributes();

}  // namespace specdec
