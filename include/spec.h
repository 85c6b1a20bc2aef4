/*
 * spec.h -- C ABI of the MI355X speculative verify-and-commit library
 * (libspecdec.so, gfx950).
 *
 * The library runs the propose / verify / commit loop of two-reasoner
 * speculative decoding (Sec. 3.2 and Sec. 4.1 of "Reasoning-aware Speculative
 * Decoding for Efficient Vision-Language-Action Models in Autonomous
 * Driving"):
 *   draft_step   one step of the routine reasoner, which proposes the next token
 *                with FlatRoPE (Eq. propose, Eq. flatrope-proj); K calls give d_1..d_K.
 *   spec_verify  the deliberative reasoner (target, 3D M-RoPE, Eq. rope-3d)
 *                evaluates [pending, d_1..d_K] in one forward pass, takes the
 *                greedy token of every row (Eq. verify) and the longest matching
 *                prefix l (Eq. accept).
 *   spec_commit  commits (d_1..d_l, r*_{l+1}), advances the lengths by l+1 and
 *                rolls back both KV caches (Eq. commit).
 *
 * Conventions
 *   - Every entry point returns a spec_status; nothing throws or exits.
 *   - "device" pointers are HIP device memory on the device that is current at
 *     spec_init; "host" pointers are ordinary memory.
 *   - bf16 means IEEE bfloat16 stored as 16-bit words; matrices are row-major
 *     [out_features][in_features].  All row lengths must be multiples of 8
 *     elements and all device pointers 16-byte aligned.
 *   - All work is enqueued on the stream given to spec_init and returns
 *     without waiting, except the calls documented as synchronising.
 *   - Arguments are validated on the host before anything is enqueued; on an
 *     error the context is left unchanged.  A HIP runtime error poisons the
 *     context: afterwards only spec_last_error and spec_destroy are valid.
 *   - One context is not safe to use from two threads at once.
 */
#ifndef SPECDEC_SPEC_H
#define SPECDEC_SPEC_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SPEC_MAX_K      16   /* draft block size limit (the paper verifies blocks of 16) */
#define SPEC_MAX_BATCH  16   /* sequences per context */
#define SPEC_MAX_LAYERS 256
#define SPEC_MAX_ROWS   160  /* batch*(K+1): rows of one verify pass */
#define SPEC_KV_PAGE    64   /* KV slots per cache page */

typedef struct spec_ctx spec_ctx;   /* opaque; owned by the library */

typedef enum spec_status {
  SPEC_OK = 0,
  SPEC_E_INVAL = 1,     /* bad argument, or a token id out of range was seen on the device */
  SPEC_E_STATE = 2,     /* call out of order (see the state machine below) */
  SPEC_E_CAPACITY = 3,  /* workspace too small or sequence capacity exceeded */
  SPEC_E_HIP = 5,       /* HIP runtime error; the context is poisoned */
  SPEC_E_NUMERIC = 6    /* NaN logits were seen on the device */
} spec_status;

/* Shape of one decoder stack.  The block is pre-norm: RMSNorm -> q,k,v (no
 * bias) -> rotary -> causal grouped-query attention -> o projection + residual
 * -> RMSNorm -> SwiGLU (silu(gate) * up) -> down projection + residual. */
typedef struct spec_dims {
  int32_t layers;            /* 1..SPEC_MAX_LAYERS */
  int32_t hidden;            /* model width; multiple of 16 */
  int32_t q_heads;           /* query heads; multiple of kv_heads */
  int32_t kv_heads;          /* key/value heads */
  int32_t head_dim;          /* 64 or 128 */
  int32_t ffn;               /* SwiGLU inner width; multiple of 16 */
  int32_t mrope_section[3];  /* (s_T, s_H, s_W) rotary pairs per axis, summing to
                                head_dim/2 (Eq. rope-3d); ignored by the draft unless
                                SPEC_FLAG_DRAFT_MROPE */
  int32_t interleaved;       /* 0: blocked axis assignment, 1: d mod 3 (Eq. axis-assign) */
  float rope_base;           /* theta_d = rope_base^(-2d/head_dim) (Eq. mrope-phase) */
  float rms_eps;             /* RMSNorm epsilon */
} spec_dims;

#define SPEC_FLAG_NO_GRAPHS 1      /* launch kernels one by one instead of replaying HIP graphs */
/* (values 2 and 4 are not used; unknown flag bits are rejected with SPEC_E_INVAL) */
#define SPEC_FLAG_ROWMAJOR 8       /* stream the caller's row-major weights directly.  Without it, passes
                                      on the layered path of at most 16 rows (batch*(K+1) <= 16), or of
                                      rows the batched-row GEMM takes, stream a tile-packed copy of every
                                      weight matrix that spec_init writes into the workspace (its size is
                                      part of spec_workspace_bytes) */
#define SPEC_FLAG_BLOCK_DRAFT 32   /* draft_step proposes all K tokens in one forward of the draft (the
                                      block-diffusion draft family, Sec. 4.1): rows [pending, MASK x K],
                                      the pending row attending causally and every MASK row attending to
                                      the prefix and the whole block; MASK row i proposes d_i.  Accepted
                                      proposals of the previous round are first re-encoded causally.
                                      Needs a draft. */
#define SPEC_FLAG_COND 64          /* the draft is conditioned on target hidden states (Sec. 4.1; fused
                                      EAGLE-3 style, Sec. 5): every verify keeps the target's residual
                                      stream after layers cond_layers[0..2]; for the rows whose inputs get
                                      committed, f = w_fuse [h0; h1; h2] (3*hidden -> hidden) becomes the
                                      slot's feature, and a draft row at slot t takes the layer-0 input
                                      e + w_in [e; f(t-1)] (2*hidden -> hidden; f = 0 where no verified
                                      feature exists: prompt slots and the draft's proposal rows).
                                      Needs a draft with w_fuse and w_in. */
#define SPEC_FLAG_COND_CROSS 256   /* with SPEC_FLAG_COND: the fused features f are the draft's layer-0
                                      cross-attention context (Sec. 4.1: target hidden states fed to the
                                      draft as cross-attention K/V) instead of the input term.  After each
                                      commit, every committed slot s gets k = rot_s(W_k RMSNorm(f_s)) and
                                      v = W_v RMSNorm(f_s) (the draft's layer-0 norm and projections) in
                                      the draft's layer-0 cache; the prompt slots keep the given draft
                                      prompt K/V.  A draft row at slot t attends in layer 0 to the context
                                      slots s < min(t, seq_len) only, and takes the plain embedding as
                                      input (w_in may be null).  Not with SPEC_FLAG_BLOCK_DRAFT. */
#define SPEC_FLAG_FULL_DRAFT_ROWS 128  /* every draft step runs the pass of batch*(K+1) rows.  Without it,
                                      a chained draft step after the first of a round (each live sequence
                                      then consumes exactly one token, its previous proposal) runs as a
                                      pass of one row per sequence on the tile-packed GEMV, when the
                                      batch is at most 32, a packed weight copy exists and neither
                                      SPEC_FLAG_BLOCK_DRAFT nor SPEC_FLAG_COND is set */
#define SPEC_FLAG_DRAFT_MROPE 16   /* the draft rotates with 3D M-RoPE (its own mrope_section and
                                      interleaved, validated as the target's) instead of FlatRoPE: the
                                      comparison arm of the attention-budget readout (Sec. 4.2) */

typedef struct spec_config {
  spec_dims target;          /* deliberative reasoner (3D M-RoPE) */
  spec_dims draft;           /* routine reasoner (FlatRoPE); draft.layers = 0 means no draft.
                                hidden, head_dim and rope_base must equal the target's: the draft
                                shares the embedding and the theta table (Sec. 4.2). */
  int32_t vocab;             /* tied embedding / LM head rows; multiple of 16 */
  int32_t K;                 /* draft block size, 0..SPEC_MAX_K (0: plain greedy decoding) */
  int32_t batch;             /* independent sequences, 1..SPEC_MAX_BATCH; batch*(K+1) <= SPEC_MAX_ROWS */
  int32_t max_new_tokens;    /* committed-token budget per sequence, >= 1 */
  int32_t stop_token;        /* committing this token ends a sequence; -1: none */
  int32_t flags;             /* SPEC_FLAG_* */
  int32_t mask_token;        /* SPEC_FLAG_BLOCK_DRAFT: input token of the MASK rows, in [0, vocab) */
  int32_t cond_layers[3];    /* SPEC_FLAG_COND: target layers (0-based) whose output is fused */
} spec_config;

/* Borrowed device pointers (bf16).  They must stay valid until spec_destroy. */
typedef struct spec_layer_weights {
  const void* attn_norm;     /* [hidden]                        */
  const void* wq;            /* [q_heads*head_dim][hidden]      */
  const void* wk;            /* [kv_heads*head_dim][hidden]     */
  const void* wv;            /* [kv_heads*head_dim][hidden]     */
  const void* wo;            /* [hidden][q_heads*head_dim]      */
  const void* ffn_norm;      /* [hidden]                        */
  const void* w_gate;        /* [ffn][hidden]                   */
  const void* w_up;          /* [ffn][hidden]                   */
  const void* w_down;        /* [hidden][ffn]                   */
} spec_layer_weights;

typedef struct spec_model_weights {
  const spec_layer_weights* layers;  /* host array of dims.layers entries */
  const void* final_norm;            /* [hidden] bf16, device */
  const void* w_fuse;                /* draft, SPEC_FLAG_COND: [hidden][3*hidden] bf16; else ignored */
  const void* w_in;                  /* draft, SPEC_FLAG_COND: [hidden][2*hidden] bf16; else ignored */
} spec_model_weights;

/* A (t, h, w) grid of vision patches occupying sequence indices
 * [start, start + t*h*w), stored t-major, then h, then w.  Its patch (t, h, w)
 * gets the 3D position (start+t, start+h, start+w); every index outside the
 * blocks is text and gets (i, i, i) (Sec. 3.3, Sec. 4.2). */
typedef struct spec_vision_block {
  int32_t start, t, h, w;
} spec_vision_block;

/* One sequence's prompt.  Its first prefix_len KV slots are filled from the
 * given pre-rotation keys and values; index prefix_len holds pending_token,
 * the first row of the first verify. */
typedef struct spec_seq_init {
  int32_t prefix_len;                 /* >= 1 */
  int32_t n_blocks;
  const spec_vision_block* blocks;    /* host; inside [0, prefix_len), non-overlapping */
  int32_t pending_token;              /* in [0, vocab) */
  const void* const* tgt_k;           /* host array [target.layers] of device pointers to
                                         [prefix_len][kv_heads][head_dim] bf16 keys before rotation */
  const void* const* tgt_v;           /* same shape, values */
  const void* const* drf_k;           /* host array [draft.layers]; NULL without a draft */
  const void* const* drf_v;
  const int32_t* page_table;          /* host; NULL, or the physical cache page of each of this
                                         sequence's spec_seq_pages() pages of SPEC_KV_PAGE slots
                                         (slot s lives in page page_table[s / SPEC_KV_PAGE]) */
} spec_seq_init;

/* KV pages one sequence owns: ceil((prefix_len + max_new_tokens + K + 2) /
 * SPEC_KV_PAGE).  Each model's caches are one pool of the sum of these over
 * the batch; a page holds SPEC_KV_PAGE slots of every kv head of one layer.
 * Either every sequence gives a page_table or none does.  Given tables must
 * together name every pool page exactly once (a permutation of
 * [0, pool pages)); without them sequence b owns the pages after those of
 * sequences 0..b-1, in order.  Both models use the same table. */
int32_t spec_seq_pages(const spec_config* cfg, const spec_seq_init* seq);

/* Bytes of device workspace spec_init needs (KV caches, positions, rotary
 * table, activations, partial sums, per-sequence state). */
spec_status spec_workspace_bytes(const spec_config* cfg, const spec_seq_init* seqs /* [batch] */,
                                 size_t* bytes);

/* Creates a context.  embed: [vocab][hidden] bf16 device, the tied token
 * embedding and LM head shared by target and draft.  draft must be NULL
 * exactly when cfg->draft.layers == 0 (then draft_step is unavailable and
 * spec_verify needs explicit draft tokens).
 * The workspace (device, 256-byte aligned, at least spec_workspace_bytes) is
 * owned by the caller and must outlive the context; the library allocates no
 * device memory of its own.  Prefix K/V may be freed once the stream has
 * passed this call.  Builds the 3D position table and the cos/sin table,
 * rotates the prefix keys of every layer into the caches, and leaves the
 * context READY. */
spec_status spec_init(const spec_config* cfg, const void* embed,
                      const spec_model_weights* target, const spec_model_weights* draft,
                      const spec_seq_init* seqs, void* workspace, size_t workspace_bytes,
                      hipStream_t stream, spec_ctx** out);

/* One draft step (Eq. propose as a chain of single-token steps; with
 * SPEC_FLAG_BLOCK_DRAFT the single-forward block proposal, which writes all K
 * columns of d_draft_tokens and counts as the round's K steps).  The draft
 * first consumes the committed tokens it has not yet seen (one row normally,
 * up to K+1 after the verifier overrode its proposals), then proposes a token
 * from its last row with a greedy argmax.  Call j (0-based) of a round writes
 * column j of d_draft_tokens [batch][K] (device int32; may be NULL).
 * State: READY or DRAFTING with fewer than K steps taken -> DRAFTING. */
spec_status draft_step(spec_ctx* ctx, int32_t* d_draft_tokens);

/* n draft steps in one call: the same as n calls of draft_step (columns j..j+n-1
 * of d_draft_tokens), issued as one launch sequence so that the steps follow
 * each other on the device without a gap between them.  1 <= n <= K minus the
 * steps already taken this round; the state rules are those of draft_step. */
spec_status draft_steps(spec_ctx* ctx, int32_t n, int32_t* d_draft_tokens);
/* (With SPEC_FLAG_BLOCK_DRAFT, draft_steps(ctx, K, out) is the block proposal
 * and n must be K.) */

/* One verify pass (Eq. verify, Eq. accept).  Rows [pending, d_1..d_K] of every
 * sequence go through the target in one forward pass; row j's greedy token is
 * r*_{j+1} (argmax over fp32 logits, lowest index on ties, NaN as -inf).
 * d_draft_tokens: [batch][K] device int32 proposals, or NULL to use the
 * draft's own K proposals of this round.  d_logits: [batch][K+1][vocab] bf16
 * device output, or NULL.  Finished sequences are skipped.
 * State: READY (with d_draft_tokens, or K == 0) or DRAFTING after K steps -> VERIFIED. */
spec_status spec_verify(spec_ctx* ctx, const int32_t* d_draft_tokens, void* d_logits);

/* ---- verify without allocation ------------------------------------------- */

#define SPEC_SCRATCH_BYTES (32u << 20)   /* size of the library's static scratch array per GPU */

/* For callers that cannot allocate or instantiate anything while they run:
 * code under HIP stream capture (this call can be captured into the caller's
 * own graph), tight serving loops, harnesses that forbid allocation.
 * Same arguments, state rules, device outputs and results as spec_verify, with
 * two differences:
 *   - the pass's scratch (split-KV attention partials, partial tiles and
 *     k-split sums of the projections, the per-workgroup argmax pairs of the LM
 *     head, their arrival counters and the bf16 logits staging) lives in one
 *     static device array of SPEC_SCRATCH_BYTES bytes that the library holds
 *     on each GPU it runs on until the process ends (its address is looked up
 *     in spec_init), not in the context's workspace;
 *   - every kernel is launched directly on the context's stream: no HIP graph
 *     is captured, instantiated or launched.
 * It calls no hipMalloc, hipFree or other allocating routine.  The counters
 * that must start at zero are cleared by a fill kernel at the start of the
 * call.  Every call on one GPU, from any context, shares that GPU's array,
 * which keeps the last call's contents: calls on one GPU that overlap in time
 * (other streams or threads) race and give wrong results, so serialise them.
 * Returns SPEC_E_CAPACITY, with nothing enqueued and the context unchanged,
 * when the context's verify needs more than SPEC_SCRATCH_BYTES of scratch (the
 * error text gives the need; it grows with batch*(K+1) rows, query heads,
 * sequence capacity and vocabulary).  Any other error is spec_verify's. */
spec_status spec_verify_scratch(spec_ctx* ctx, const int32_t* d_draft_tokens, void* d_logits);

/* Commit (Eq. commit): appends (d_1..d_l, r*_{l+1}), cut after a stop token
 * or at the token budget, to each unfinished sequence; the target keeps KV
 * slots up to the new length and the draft keeps the slots whose inputs still
 * match the committed tokens (the rest are rolled back and later
 * overwritten).  Optional device outputs (int32): d_accept_len [batch] = l,
 * d_committed [batch][K+1] (first d_n_committed[b] entries valid),
 * d_n_committed [batch], d_finished [batch].
 * State: VERIFIED -> READY. */
spec_status spec_commit(spec_ctx* ctx, int32_t* d_accept_len, int32_t* d_committed,
                        int32_t* d_n_committed, int32_t* d_finished);

/* Attention-budget readout (Sec. 4.2, Table attn-budget): arms the next pass
 * of `model` (0: the target, i.e. the next spec_verify; 1: the draft, i.e. the
 * next draft step) to also report where attention layer `layer` (0-based) puts
 * its softmax mass.  Cache slots are classed as visual (inside a vision
 * block), trajectory/text (any other prompt slot) or generated (index >=
 * prefix_len).  For every row j < the pass's row count of sequence b and
 * every query head h of that model, the pass writes d_out[((b*(K+1) + j) *
 * q_heads + h)*4 + c] (device float32, 16-byte aligned):
 *   c = 0, 1, 2  attention mass on visual / trajectory-text / generated slots
 *                (the three sum to 1 up to rounding);
 *   c = 3        entropy of the attention restricted to trajectory/text slots
 *                and renormalised, divided by ln(number of those slots)
 *                (0 when the prompt has at most one such slot).
 * Rows a pass does not run (finished sequences, rows past a draft pass's
 * count) are left unchanged.  The armed pass is launched kernel by kernel
 * (no graph replay); the readout then disarms.  d_out = NULL disarms.
 * Any state. */
spec_status spec_attn_readout(spec_ctx* ctx, int32_t model, int32_t layer, float* d_out);

/* Synchronising: waits for the stream, then reports how many sequences have
 * finished (*n_finished, may be NULL) and returns SPEC_E_INVAL / SPEC_E_NUMERIC
 * if a device-side check failed since spec_init (an out-of-range draft token,
 * which was replaced by token 0, or NaN logits). */
spec_status spec_sync(spec_ctx* ctx, int32_t* n_finished);

void spec_destroy(spec_ctx* ctx);

/* Text of the last error of this context (or of the last failed spec_init if
 * ctx is NULL).  Valid until the next call on the context. */
const char* spec_last_error(const spec_ctx* ctx);

/* ---- inspection (synchronising; for tests and tools) --------------------- */

/* 3D positions (p_T, p_H, p_W) of sequence b's slots 0..len-1 into
 * host_out [3][len] int32.  len <= capacity. */
spec_status spec_debug_positions(spec_ctx* ctx, int32_t b, int32_t* host_out, int32_t len);

/* Sequence b's state into host_out [8] int32: seq_len (slots with target KV =
 * index of the pending token), draft_len, pending token, committed-token
 * count, finished, accept length of the last verify, tokens committed by the
 * last commit, device error bits. */
spec_status spec_debug_state(spec_ctx* ctx, int32_t b, int32_t* host_out);

/* Cached keys (which = 0, after rotation) or values (which = 1) of sequence
 * b, model 0 = target / 1 = draft, layer, slots [pos0, pos0+npos) into
 * host_out [npos][kv_heads][head_dim] bf16. */
spec_status spec_debug_kv(spec_ctx* ctx, int32_t b, int32_t model, int32_t layer, int32_t which,
                          int32_t pos0, int32_t npos, void* host_out);

/* SPEC_FLAG_COND: the fused target features of sequence b's slots [slot0,
 * slot0+n) into host_out [n][hidden] bf16 (zero for slots never verified). */
spec_status spec_debug_feature(spec_ctx* ctx, int32_t b, int32_t slot0, int32_t n, void* host_out);

/* Execution path of the context's passes into *path:
 * SPEC_PATH_ROWMAJOR (one kernel per layer step over the caller's row-major weights),
 * SPEC_PATH_PACKED (one kernel per layer step over the tile-packed weight copy). */
#define SPEC_PATH_ROWMAJOR 0
#define SPEC_PATH_PACKED 1
spec_status spec_debug_path(const spec_ctx* ctx, int32_t* path);

/* Per-kernel timing with HIP events on the context's stream.  While enabled,
 * calls launch kernels one by one (no graph replay), each through
 * hipExtLaunchKernelGGL with a start/stop event pair, and every pass begins
 * with a bounded device-side wait (a few ms) so that the host has enqueued the
 * whole pass before its first kernel runs.  spec_timing_read (synchronising) returns, for kernel class
 * `kind`, the number of launches, their summed duration in milliseconds and
 * the summed algorithmic bytes (weights and activations each launch must
 * move, cached keys and values excluded; 0 for kinds without a byte model)
 * since timing was last enabled. */
enum spec_kernel_kind {
  SPEC_KERNEL_QKV = 0,       /* fused Q/K/V projection with rotary and KV append */
  SPEC_KERNEL_O = 1,         /* attention output projection with the residual add */
  SPEC_KERNEL_GATEUP = 2,    /* fused gate/up projection with SwiGLU */
  SPEC_KERNEL_DOWN = 3,      /* down projection partial sums (split over the FFN width) */
  SPEC_KERNEL_LMHEAD = 4,    /* tied LM head with the fused per-tile argmax */
  SPEC_KERNEL_ATTN = 5,      /* split-KV attention */
  SPEC_KERNEL_OTHER = 6,     /* embed, attention combine, down reduction, accept, commit */
  SPEC_KERNEL_KINDS = 7
};
spec_status spec_timing(spec_ctx* ctx, int32_t enable);

/* Read-only streaming reference (no context): reads `bytes` (a multiple of
 * 16) of device memory at d_buf (16-byte aligned) once with non-temporal
 * 16-byte loads, each wave taking 8 KB chunks (eight 1 KB loads in flight),
 * in sink_words / 4 workgroups of 256 threads, and writes one checksum word
 * per wave to d_sink [sink_words]
 * (device; sink_words a positive multiple of 4).  Enqueued on `stream`.  Used
 * to measure the HBM read rate a kernel reaches on this device and to
 * calibrate byte counters against a known read volume. */
spec_status spec_stream_read(const void* d_buf, size_t bytes, uint32_t* d_sink, int32_t sink_words,
                             hipStream_t stream);
spec_status spec_timing_read(spec_ctx* ctx, int32_t kind, int64_t* launches, double* ms, double* bytes);

#ifdef __cplusplus
}
#endif
#endif /* SPECDEC_SPEC_H */
