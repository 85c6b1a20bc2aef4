// Balanced weight-streaming GEMV over tile-packed weights (sgemv.hip) for
// passes of at most 32 rows (one or two MFMA row blocks): one kernel per projection, with the consumer's
// elementwise step and, for the down projection, the k-slice reduction,
// residual and next-norm input fused in.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "ctx.h"

namespace specdec {

constexpr int kSgWorkers = 15;                // weight-streaming waves per workgroup
constexpr int kSgWaves = kSgWorkers + 1;      // + the control wave
constexpr int kSgDepth = 8;                   // k-steps each worker keeps in flight (one tile's share)
constexpr int kSgDepthMax = 9;                // ... for inputs of up to 15 * 9 steps (4096 wide)
#ifndef SG_DEPTH_XS
#define SG_DEPTH_XS 8
#endif
constexpr int kSgDepthXs = SG_DEPTH_XS;       // k-steps in flight per worker when x is streamed
constexpr int kSgMaxRows = 32;                // rows of a pass: two MFMA row blocks
constexpr int kSgMaxSpan = kSgWorkers * kSgDepth;   // k-steps of one tile slice
constexpr int kSgPendMax = 64;                // units one workgroup may have to finish

enum { SG_ROPE = 0, SG_RESID = 1, SG_SWIGLU = 2, SG_DOWN = 3, SG_ARGMAX = 4 };

// Packed weight layout: output rows in tiles of 16, input columns in steps of
// 32 (zero-padded to a whole step).  Block (tile t, step s) is 1 KB: lane l
// (0..63) of a wave reads its 16 bytes at byte ((t*T + s)*64 + l)*16, which
// hold W[16t + (l & 15)][32s + 8(l >> 4) .. +8], the A operand of one
// 16x16x32 bf16 MFMA.  A tile's T blocks are contiguous.
struct PackSrc {
  const bf16_t* seg[3];   // row-major source segments [rows][Kd]
  int row0[3];            // first packed row of each segment
  int nseg;
  int pair;               // gate/up: packed tile 2c = tile c of seg[0], 2c+1 = tile c of seg[1]
  int Kd;                 // source row length (multiple of 8)
  int ntiles, T;          // packed tiles and steps
};

// One projection of one layer (built on the host at set-up, passed to the
// kernel by value).
struct SgJob {
  const bf16_t* w;        // packed weights [ntiles][T] blocks
  int ntiles, T;
  int S, G;               // k-slices of T; workgroups per slice (grid = S*G)
  int xs;                 // x streamed with the weights (long k-ranges) instead of held in registers
  int dep9;               // x in registers, 9 steps per worker (inputs of 121..135 steps)
  int kmax;               // partial slots per workgroup
  int units;              // fixup units (tiles, or gate/up tile pairs)
  const bf16_t* x;        // input rows [M][ldx], Kd valid columns; or step-major (xpk)
  int xpk;                // x step-major: [ceil(Kd/32)][M][32], so a step's rows are one contiguous run
  int ldx, Kd, M, rps;    // rows; rows per sequence
  const float* ss_in;     // normalised input: [Hn/16][mpad] sums of squares, else null
  int Hn, mpad;
  float eps;
  const SeqState* st;
  float* part;            // partial tiles [S*G][kmax][row blocks][2][64] x float4
  unsigned* cnt;          // [units] arrival counters, zero between launches
  // SG_ROPE: rotation at each row's position, queries, K and V^T cache append
  bf16_t* q;
  bf16_t *kc, *vt;
  const int32_t* pt;
  int pps;
  const float2* rcs;      // [mpad][D/2] per-row (cos, sin)
  int nq, nkv, D;
  // SG_RESID / SG_DOWN: x += y, next norm's input
  float* x32;             // [M][H]
  int H;
  const bf16_t* gain;
  bf16_t* xg;             // [*][H]
  float* ss_out;          // [H/16][mpad]
  int select_last;        // SG_DOWN of a draft pass's last layer: each sequence's last live row as row b
  // SG_SWIGLU
  bf16_t* u;              // [M][ntiles*8], or step-major [ntiles/4][M][32] (upk)
  int upk;
  // SG_ARGMAX
  float* amax_v;          // [amax_n][mpad] (max, index) of each row per workgroup (per tile when k-sliced)
  int32_t* amax_i;
  int amax_n;
  bf16_t* logits;         // [M][ntiles*16]
  int allow_logits;
  // SG_ARGMAX without k-slices: the workgroup that finishes last reduces the
  // per-workgroup pairs of every row to its argmax (no separate launch).
  // tail 1: r* of each row (verify and block passes); 2: a draft step's
  // proposal, recorded in the sequence state and the caller's [B][tail_K]
  // array tail_out; 0: pairs only
  int tail;
  int tail_K;
  int32_t* tail_out;
  unsigned* tail_cnt;     // arrival counter, zero between launches
};

// Fills the geometry of a job (S, G, kmax, units) for ncu compute units;
// false if the shape does not fit the kernel (LDS, step span, offsets).
bool sg_plan(SgJob& j, int epi, int ncu, int lds_limit);
size_t sg_lds_bytes(const SgJob& j);
size_t sg_part_floats(const SgJob& j);
size_t sg_packed_elems(int ntiles, int T);
hipError_t sg_launch(int epi, const SgJob& job, hipStream_t s, hipEvent_t e0, hipEvent_t e1);
hipError_t sg_pack(bf16_t* dst, const PackSrc& src, hipStream_t s);
void sg_set_attributes(int lds_limit);

}  // namespace specdec
