// Arguments and host entry points of the persistent forward-pass kernel
// (pass.hip).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "ctx.h"

namespace specdec {

constexpr int kPassWaves = 8;    // waves per workgroup: 1 control + 7 weight-streaming
constexpr int kPassSteps = 16;   // max 32-wide k-steps per worker wave and tile

// One GEMV phase of one layer (built on the host at init, read by the kernel
// from device memory).
struct GemvJob {
  const bf16_t* w[3];        // weight segments, [rows][Kd] bf16
  int row0[3];               // first output row of each segment
  int nseg;
  int N, Kd, splits;
  const bf16_t* x;           // [M][Kd] input rows (per-layer buffer)
  const float* ss_in;        // [Kd/16][mpad] sums of x^2 of a normalised input, or null
  const bf16_t* gain;        // gain of the norm whose input the epilogue writes
  bf16_t* q;                 // QKV: rotated queries
  bf16_t *kc, *vt;           // QKV: this layer's caches
  bf16_t* xg_out;            // O / down: bf16(x * gain)
  float* ss_out;             // O / down: sums of x^2
  bf16_t* u;                 // gate/up: SwiGLU output
  int select_last;           // down, last layer of a draft pass
};
constexpr int kPassJobs = 4;   // QKV, O, gate/up, down
enum { kJobQkv = 0, kJobO = 1, kJobGateUp = 2, kJobDown = 3 };

struct PassArgs {
  SeqState* st;
  int layers, H, nq, nkv, D, F;
  int M, R, B, rps, mpad, pps;
  float eps, scale_log2;
  const LayerW* lw;          // [layers] device copy of the layer weight pointers
  const GemvJob* jobs;       // [layers][kPassJobs]
  const bf16_t* final_norm;
  int select_last;           // draft pass: the last layer keeps each sequence's last row only
  // paged caches (layer 0 bases; kv_layer elements per layer) and page tables
  bf16_t *kc, *vt;
  const int32_t* pt;         // [B][pps]
  size_t kv_layer;
  const float2* rcs;         // [Mpad][D/2] per-row (cos, sin)
  // activations: x is shared; the others are per layer (stride in elements)
  float* x;                  // [Mpad][H] residual stream
  bf16_t* xa;                // [layers + 1][Mpad][H] bf16(x * g_attn) per layer
  bf16_t* xf;                // [layers][Mpad][H] bf16(x * g_ffn)
  float* ssa;                // [layers + 1][H/16][mpad]
  float* ssf;                // [layers][H/16][mpad]
  bf16_t* q;                 // [layers][Mpad][nq*D]
  bf16_t* o;                 // [layers][Mpad][nq*D]
  bf16_t* u;                 // [layers][Mpad][F]
  size_t x_layer, ss_layer, q_layer, u_layer;
  bf16_t* xg_final;          // LM-head input and its sums of squares
  float* ss_final;
  // attention partials
  float *op, *mp, *lp;
  int attn_chunk, attn_splits;
  // down projection
  int down_splits;
  float* part;               // [down_splits][M][H]
  unsigned* bar;             // barrier words (kPassBarWords), zero between launches
  unsigned long long* timeline;  // optional [events][workgroups] wall-clock stamps, or null
};

// Timeline events of one launch: 0 = start, then for each layer and phase
// (QKV, attention, combine, O, gate/up, down) 2 events: the workgroup's work
// done, the following barrier passed (after down: the barrier before the
// down projection's finish).
constexpr int kPassPhases = 6;
inline int pass_timeline_events(int layers) { return 1 + layers * kPassPhases * 2; }

constexpr int kPassBarWords = 1024;

size_t pass_lds_bytes(const PassArgs& a);
size_t pass_gemv_lds_bytes(const PassArgs& a);   // the GEMV phases only
// Fills jobs[layers][kPassJobs] from the (host) arguments and layer weights.
void pass_build_jobs(const PassArgs& a, const LayerW* lw, const bf16_t* final_norm, GemvJob* jobs);
int pass_steps(const PassArgs& a);
void pass_set_attributes(int lds_limit);
// One GEMV job (kind kJob*) as a kernel of its own; d_args supplies rows,
// norms and buffers, d_job the weights and input/output of the phase.
// steps: k-steps per worker wave (gemv_job_steps), at most kPassSteps.
hipError_t gemv_job_launch(int kind, int steps, const PassArgs* d_args, const GemvJob* d_job, int workgroups,
                           size_t lds, hipStream_t s, hipEvent_t e0, hipEvent_t e1);
int gemv_job_steps(int Kd, int splits);
// d_args: device copy of the arguments (constant between launches).
hipError_t pass_launch(const PassArgs* d_args, int head_dim, bool draft, int workgroups, size_t lds, hipStream_t s,
                       hipEvent_t e0, hipEvent_t e1);

}  // namespace specdec
