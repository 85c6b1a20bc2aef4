// Arguments of the weight-streaming GEMV kernels (kernels.hip) and of the
// batched-row GEMM (gemm.hip), and the consumer steps their epilogues fuse.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "ctx.h"

namespace specdec {

enum {
  EPI_STORE = 0,   // out[split][m][n]: k-split partial sums (down projection)
  EPI_ROPE = 1,    // y/rms; rotation of q/k at the row's position, q store, K / V^T cache append (QKV)
  EPI_RESID = 2,   // x += y; xg = bf16(x * g); sums of x^2 (O projection)
  EPI_SWIGLU = 3,  // y/rms; half-tiles (8 gate rows, 8 up rows): u = silu(gate) * up (gate/up)
  EPI_ARGMAX = 4   // y/rms; per-tile (max, index) of the logits, optional bf16 logits (LM head)
};

struct GemvArgs {
  const bf16_t* w[3];
  int row0[3];           // first output row of each weight segment (multiples of 16)
  int nseg;
  const bf16_t* pw;      // GEMM only: the tile-packed copy of these weights ([N/16][steps] blocks of
                         // 1 KB, sgemv.h; gate/up as gate, up tile pairs), or null to read w
  int N, Kd;
  const bf16_t* x;       // [M][ldx], or step-major [Kd/32][M][32] (xpk)
  int ldx, M, splits;
  int xpk;               // x is step-major: a 32-wide step's rows are one contiguous run (wide-unit GEMM only)
  const SeqState* st;
  int rps;               // rows per sequence
  int mpad;              // row stride of ss / amax
  const float* ss_in;    // [H/16][mpad] sums of x^2 of the input rows (ROPE, SWIGLU, ARGMAX)
  int H;                 // row length those sums cover
  float eps;
  float* out;            // EPI_STORE: [splits][M][N]
  // EPI_ROPE
  bf16_t* q;             // [M][nq*D]
  bf16_t *kc, *vt;       // layer bases of the paged key / value pools
  const int32_t* pt;     // [B][pps] page tables
  const float2* rcs;     // [Mpad][D/2] (cos, sin) per row
  int nq, nkv, D, pps;
  // EPI_RESID
  float* x32;            // [M][N] residual stream
  const bf16_t* gain;    // [N] gain of the next RMSNorm
  bf16_t* xg;            // [M][N] bf16(x * gain)
  float* ss_out;         // [N/16][mpad] sums of x^2
  // EPI_SWIGLU
  bf16_t* u;             // [M][N/2], or step-major [N/64][M][32] (upk, wide-unit GEMM only)
  int upk;
  // EPI_ARGMAX
  float* amax_v;         // [N/16][mpad]
  int32_t* amax_i;
  bf16_t* logits;        // [M][N]
  int allow_logits;
};

// Passes of up to kThinRows rows use the thin GEMV kernels (kernels.hip);
// larger passes (up to SPEC_MAX_ROWS) the batched-row GEMM (gemm.hip).
constexpr int kThinRows = 64;
constexpr int kSgMaxRowsGemm = 16;   // the GEMM takes passes of more rows than one MFMA block
constexpr int kGemmTiles = 4;   // 16-column output tiles per GEMM workgroup

// Dynamic LDS bytes of a GEMM launch over M rows.
size_t gemm_lds_bytes(int M);
// Raises the dynamic LDS limit of every GEMM instantiation that fits `limit` bytes.
void gemm_set_attributes(int limit);
// y = x W^T over g.M rows (kSgMaxRowsGemm < M <= SPEC_MAX_ROWS) with epilogue
// `epi`.  Over the tile-packed copy (g.pw) with more than 32 rows: the
// wide-unit kernel, one workgroup per CU for SwiGLU and the LM head, grid
// (ceil(N / 256), g.splits) for EPI_STORE; otherwise k_gemm, grid
// (ceil(N / 64), g.splits).  Only EPI_STORE may use k-splits.
hipError_t gemm_launch(int epi, const GemvArgs& g, hipStream_t s, hipEvent_t e0, hipEvent_t e1);
// k-splits of an EPI_STORE GEMM (the down projection) over N outputs and Kd inputs.
int gemm_down_splits(int N, int Kd, int ncu);
// k-splits of an EPI_STORE launch of the wide-unit kernel (passes of more
// than kSgMaxRows rows over the tile-packed copy; 256-column workgroups, one
// per CU): as many as fill one round of the CUs, at least 16 k-steps each.
int gemm_wide_splits(int N, int Kd, int ncu);
// Workgroups of the k-split GEMM over M rows resident per CU: the runtime's
// occupancy for the shapes of up to three row blocks (at most 2), else 1;
// the o and down projections split to fill every resident slot once.
int gemm_wgs_per_cu(int M);
// k-splits of the q/k/v GEMM over M rows: 1 (one launch with the fused rotary
// epilogue) unless its workgroups cover under half the CUs and the fp32
// partials it writes and reads back stay under a tenth of its weight bytes;
// a split launch is finished by k_qkv_finish (kernels.hip).
int gemm_qkv_splits(int N, int Kd, int M, int ncu);
// The q/k/v k-splits of a pass of M rows: gemm_wide_splits on a context whose
// passes run on the wide-unit kernel (wide), else gemm_qkv_splits.
int gemm_qkv_splits_for(int N, int Kd, int M, int ncu, bool wide);

}  // namespace specdec
