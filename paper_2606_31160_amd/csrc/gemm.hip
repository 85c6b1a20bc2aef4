// Batched-row GEMMs on MFMA: y[m][n] = sum_k x[m][k] W[n][k] for up to
// SPEC_MAX_ROWS rows, with the same fused epilogues as the thin GEMV kernels
// (1/rms row scale, rotary + paged KV append, residual + next-norm input,
// SwiGLU, per-tile argmax, or k-split partial sums).  Two kernels:
//   * k_gemm_wide (below k_gemm): passes of more than 32 rows over the
//     tile-packed weights (several sequences verified together);
//   * k_gemm: row-major weights (SPEC_FLAG_ROWMAJOR) for passes of more than
//     16 rows, and 17..32-row passes whose width the thin GEMV cannot stage.
//
// k_gemm: a workgroup owns kGemmTiles = 4 output tiles of 16 columns and the k-range
// of split blockIdx.y, walked in chunks of 32 * kSteps columns (kSteps
// 32-wide MFMA steps; kSteps = 4 or 2 by the row count).  It has two kinds
// of waves:
//   * 2 * kSteps MFMA waves.  Wave w = 2q + p multiplies tile pair p (tiles
//     2p, 2p+1) by step q of every chunk: each x operand it reads from LDS
//     feeds two MFMAs, and the step groups split the k-range (their partial
//     tiles are summed through LDS at the end).  They stream only weights,
//     kStages chunks ahead.
//   * 4 loader waves.  They stage every chunk's x rows (all rows) into one of
//     two LDS buffers, loading kStages chunks ahead.
// Loads complete in issue order per wave, so a wave that waited for x would
// also wait for every weight load issued before it; with x in waves of its
// own, the weight loads stay kStages chunks deep.  One workgroup barrier per
// chunk hands a staged buffer to the MFMA waves; barriers wait for LDS
// traffic only, never for loads in flight.  Both loops run a whole number of
// kStages-chunk rounds with no early exit (chunks past the k-range load
// nothing and add zeros): an exit inside the unrolled round would make the
// compiler drain every load in flight at the loop head.
//
// v_mfma_f32_16x16x32_bf16 takes the weight fragment as A (lane l: row l&15,
// k 8*(l>>4)..+8) and x^T as B (lane l: x row l&15, same k); lane l then
// holds y[n0 + 4*(l>>4) + i][row l&15 of the block] for each 16-row block.
#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>

#include <algorithm>
#include <cmath>

#include "ctx.h"
#include "device.h"
#include "gemv.h"
#include "sgemv.h"

namespace specdec {

namespace {

constexpr int kLoadWaves = 4;                 // waves that stage x
constexpr int kOut = 0x7FFFFF00;              // buffer offset past every operand: the load returns zeros
constexpr int kRsrcWord3 = 0x00020000;        // raw buffer resource, 32-bit data
constexpr int kNt = 2;                        // non-temporal hint of the weight loads
constexpr int NL = kLoadWaves * 64;           // loader threads
constexpr int kYStride = 17;                  // floats per row of an output tile in LDS

// Step groups (32-wide k-steps per chunk, one MFMA wave pair each) and chunks
// of loads in flight, by 16-row blocks: up to 3 blocks 2 groups and 8 chunks
// (8 waves of at most 128 registers: two workgroups per CU); 4-5 blocks 4
// groups and 5 chunks (12 waves, 168 registers each); from 6 blocks, whose
// accumulators need more registers, 2 groups and 8 chunks (8 waves of 256).
// The compiler waits for all of a wave's loads once per round of kStages
// chunks, so a deep round is what keeps enough bytes in flight per CU.
constexpr int steps_for(int mb) { return (mb >= 6 || mb <= 3) ? 2 : 4; }
constexpr int stages_for(int mb) { return (mb >= 6 || mb <= 3) ? 8 : 5; }
constexpr int threads_for(int mb) { return (2 * steps_for(mb) + kLoadWaves) * 64; }
constexpr int xstride_for(int mb) { return 32 * steps_for(mb) + 8; }   // bf16 per LDS x row (16-byte pad)
static_assert(kGemmTiles == 4, "MFMA wave w = 2q + p: tile pair p, step group q");
// Sums of squares each thread of the 1/rms prologue loads, with `parts`
// threads per row: enough for hidden 8192 (512 sums) where registers allow.
constexpr int lpt_for(int parts) { return (512 + parts - 1) / parts < 96 ? (512 + parts - 1) / parts : 96; }

// two x buffers of 16 mb rows plus a spare row each (the target of loader
// stores past the last row, so that no branch skips a store)
size_t x_lds_bytes(int mb) { return (size_t)2 * (16 * mb + 1) * xstride_for(mb) * sizeof(bf16_t); }
// output tiles, plus (4 step groups) the partial tiles of groups 2 and 3 while they are summed
size_t y_lds_bytes(int mb) {
  return (size_t)(steps_for(mb) == 4 ? 2 : 1) * kGemmTiles * (16 * mb) * kYStride * sizeof(float);
}

template <int MB, int EPI>
__global__ __launch_bounds__(threads_for(MB)) void k_gemm(GemvArgs a) {
  constexpr int ROWS = MB * 16;
  constexpr int kSteps = steps_for(MB), kStages = stages_for(MB), NT = threads_for(MB);
  constexpr int kMfmaWaves = 2 * kSteps;
  constexpr int kChunk = 32 * kSteps;                         // k columns per stage
  constexpr int kXStride = xstride_for(MB);
  constexpr int CV = kChunk / 8;                              // x vectors per row and chunk
  constexpr int XV = (ROWS * CV + NL - 1) / NL;               // x vectors per loader thread and chunk
  constexpr bool kNorm = EPI == EPI_ROPE || EPI == EPI_SWIGLU || EPI == EPI_ARGMAX;
  extern __shared__ __align__(16) unsigned char lds[];
  __shared__ float inv_rms[ROWS];
  __shared__ int live_s[ROWS];
  __shared__ float rms_part[kNorm ? NT : 1];

  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const bool loader = wave >= kMfmaWaves;                    // wave-uniform role
  const int pair = wave & 1, q = (wave >> 1) & (kSteps - 1);
  const int lt = threadIdx.x - kMfmaWaves * 64;               // loader thread index
  const int split = blockIdx.y;
  const int Kd = a.Kd, M = a.M, N = a.N;
  const int T = (Kd + 31) >> 5;
  const int s0 = (int)((long long)split * T / a.splits);
  const int s1 = (int)((long long)(split + 1) * T / a.splits);
  const int nch = (s1 - s0 + kSteps - 1) / kSteps;
  const int kq = 8 * (lane >> 4);
  const int kend = min(s1 * 32, Kd);

  // Weights are read through buffer resources, x through one over its rows:
  // every load is issued unconditionally, and one that a lane does not need
  // (past the split, a dead row, a tile past N) gets offset kOut and returns
  // zeros without a memory access.  With no branch around a load, the
  // compiler's wait counts stay exact and loads stay kStages chunks deep.
  //
  // MFMA waves, tile t of the pair: on the tile-packed copy, block (tile,
  // step) is 1 KB at (tile * T + step) * 1 KB with lane l at 16 l; on
  // row-major weights, lane l reads row l & 15 of the tile.  SwiGLU tiles
  // come in pairs on both (tile 2c: gate rows 16c..16c+16, tile 2c+1: the up
  // rows of the same features), so every tile is one load per step.
  const bool packed = a.pw != nullptr;
  __amdgpu_buffer_rsrc_t rw[2];
  int wbase[2];          // byte offset of this lane's fragment at step 0 (kOut: tile unused)
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const int tile = blockIdx.x * kGemmTiles + 2 * pair + t;
    const int n0 = tile * kTile;
    const bool on = !loader && n0 < N;
    const int r = lane & 15;
    if (packed) {
      rw[t] = __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16_t*>(a.pw), 0, (N / kTile) * T * 1024, kRsrcWord3);
      wbase[t] = on ? tile * T * 1024 + 16 * lane : kOut;
    } else if constexpr (EPI == EPI_SWIGLU) {
      const int F = N / 2;
      rw[t] = __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16_t*>(a.w[tile & 1]), 0, F * Kd * 2, kRsrcWord3);
      wbase[t] = on ? (((tile >> 1) * kTile + r) * Kd + kq) * 2 : kOut;
    } else {
      int sg = 0;
#pragma unroll
      for (int i = 1; i < 3; ++i)
        if (i < a.nseg && n0 >= a.row0[i]) sg = i;
      const int rows = (sg + 1 < a.nseg ? a.row0[sg + 1] : N) - a.row0[sg];
      rw[t] = __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16_t*>(a.w[sg]), 0, rows * Kd * 2, kRsrcWord3);
      wbase[t] = on ? ((n0 - a.row0[sg] + r) * Kd + kq) * 2 : kOut;
    }
  }
  const __amdgpu_buffer_rsrc_t rx =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16_t*>(a.x), 0, M * a.ldx * 2, kRsrcWord3);

  // live rows: row m is row m % rps of sequence m / rps, live while below
  // that sequence's row count
  for (int m = threadIdx.x; m < ROWS; m += NT) {
    int lv = 0;
    if (m < M) {
      const int b = m / a.rps;
      lv = (m - b * a.rps) < a.st[b].count ? 1 : 0;
    }
    live_s[m] = lv;
  }
  __syncthreads();

  // 1/rms of each live row from the per-16-column sums of squares, at the
  // start.  ss_in is [H/16][mpad]: for one column group the rows are
  // contiguous, so thread (part p, row m) sums groups p*per .. (p+1)*per - 1
  // of row m with loads that are coalesced across the rows, all issued before
  // the first add (one memory round trip per workgroup); the parts are then
  // added in order.  inv_rms is read after the K loop's barriers.
  if constexpr (kNorm) {
    constexpr int P = NT / ROWS;              // parts per row (>= 3)
    constexpr int LPT = lpt_for(P);           // loads per thread (H/16 <= LPT * P, checked on the host)
    const int nt = a.H / kTile, per = (nt + P - 1) / P;
    const int m = threadIdx.x % ROWS, p = threadIdx.x / ROWS;
    float v[LPT];
#pragma unroll
    for (int j = 0; j < LPT; ++j) v[j] = a.ss_in[(size_t)min(p * per + j, nt - 1) * a.mpad + m];
    float sum = 0.f;
#pragma unroll
    for (int j = 0; j < LPT; ++j) sum += (p < P && j < per && p * per + j < nt) ? v[j] : 0.f;
    rms_part[threadIdx.x] = sum;
    __syncthreads();
    if (threadIdx.x < ROWS) {
      float t = 0.f;
      for (int q2 = 0; q2 < P; ++q2) t += rms_part[q2 * ROWS + threadIdx.x];
      inv_rms[threadIdx.x] = live_s[threadIdx.x] ? rsqrtf(t / a.H + a.eps) : 0.f;
    }
  }

  // Loader waves, chunk c: x vector v (v < ROWS*CV) is row v / CV, columns
  // 8*(v % CV) .. +8 of the chunk.  MFMA waves, chunk c: step q of the chunk
  // for both tiles.  Dead rows, columns past the split or past Kd read as
  // zeros (Kd % 8 == 0, so a vector starting below the end lies inside).
  auto issue_x = [&](int c, u32x4 (&xr)[XV]) {
    const int kc = (s0 + kSteps * c) * 32;
#pragma unroll
    for (int i = 0; i < XV; ++i) {
      const int v = lt + NL * i;
      const int m = v / CV, k = kc + 8 * (v % CV);
      const int mm = m < ROWS ? m : ROWS - 1;   // (no branch around the LDS read)
      const bool ok = (v < ROWS * CV) & (m < M) & (live_s[mm] != 0) & (k < kend);
      xr[i] = __builtin_amdgcn_raw_buffer_load_b128(rx, ok ? (m * a.ldx + k) * 2 : kOut, 0, 0);
    }
  };
  auto issue_w = [&](int c, u32x4 (&wr)[2]) {
    const int st = s0 + kSteps * c + q;
    const bool ok = packed ? st < s1 : st * 32 + kq < kend;
    const int step_bytes = packed ? 1024 : 64;
#pragma unroll
    for (int t = 0; t < 2; ++t)
      wr[t] = __builtin_amdgcn_raw_buffer_load_b128(rw[t], (ok && wbase[t] != kOut) ? wbase[t] + st * step_bytes : kOut,
                                                    0, kNt);
  };

  bf16_t* xs = reinterpret_cast<bf16_t*>(lds);
  float* y = reinterpret_cast<float*>(lds);   // output tiles once the x buffers are free
  // Both roles pass the same barriers: one per chunk, then the sums' (five
  // with four step groups, three with two).
  if (loader) {
    u32x4 xr[kStages][XV];
#pragma unroll
    for (int u = 0; u < kStages; ++u) issue_x(u, xr[u]);
    for (int c0 = 0; c0 < nch; c0 += kStages) {   // workgroup-uniform
#pragma unroll
      for (int u = 0; u < kStages; ++u) {
        const int c = c0 + u;   // chunks past the last one load nothing and stage zeros
        // buffer c&1 was last read in chunk c-2, before every wave passed
        // chunk c-1's barrier
        bf16_t* xb = xs + (size_t)(c & 1) * (ROWS + 1) * kXStride;
#pragma unroll
        for (int i = 0; i < XV; ++i) {
          const int v = lt + NL * i;
          const int row = v < ROWS * CV ? v / CV : ROWS;
          *reinterpret_cast<u32x4*>(xb + row * kXStride + 8 * (v % CV)) = xr[u][i];
        }
        issue_x(c + kStages, xr[u]);   // past the last chunk: zeros, no memory access
        __syncthreads();   // chunk c's x rows are visible to every wave
      }
    }
    for (int i = 0; i < (kSteps == 4 ? 5 : 3); ++i) __syncthreads();
  } else {
    u32x4 wr[kStages][2];
#pragma unroll
    for (int u = 0; u < kStages; ++u) issue_w(u, wr[u]);
    f32x4 acc[2][MB];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) acc[t][mb] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int c0 = 0; c0 < nch; c0 += kStages) {   // workgroup-uniform
#pragma unroll
      for (int u = 0; u < kStages; ++u) {
        const int c = c0 + u;   // chunks past the last one multiply zeros
        const bf16_t* xb = xs + (size_t)(c & 1) * (ROWS + 1) * kXStride;
        __syncthreads();   // chunk c's x rows are visible to every wave
        const u32x4 w0 = wr[u][0], w1 = wr[u][1];
        issue_w(c + kStages, wr[u]);   // past the last chunk: zeros, no memory access
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
          const u32x4 xv = *reinterpret_cast<const u32x4*>(xb + (mb * 16 + (lane & 15)) * kXStride + 32 * q + kq);
          acc[0][mb] = mfma16x16x32(w0, xv, acc[0][mb]);
          acc[1][mb] = mfma16x16x32(w1, xv, acc[1][mb]);
        }
      }
    }
    __syncthreads();   // 1: x buffers are free

    // Sum the step groups' partial tiles in a fixed order, ((q0 + q2) + (q1 + q3))
    // with four groups (2 and 3 store, 0 and 1 add; 1 stores, 0 adds) or
    // q0 + q1 with two; group 0 scales by 1/rms and leaves the result in
    // y[tile][m][c].
    auto tile_at = [&](float* base, int t, int mb, int i) -> float& {
      const int m = mb * 16 + (lane & 15);
      return base[((2 * pair + t) * ROWS + m) * kYStride + 4 * (lane >> 4) + i];
    };
    auto store = [&](float* dst) {
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
#pragma unroll
          for (int i = 0; i < 4; ++i) tile_at(dst, t, mb, i) = acc[t][mb][i];
    };
    if constexpr (kSteps == 4) {
      float* yp = y + (size_t)kGemmTiles * ROWS * kYStride;   // the upper partial tiles
      if (q >= 2) store(q == 2 ? y : yp);
      __syncthreads();   // 2
      if (q < 2) {
        float* src = q == 0 ? y : yp;
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
          for (int mb = 0; mb < MB; ++mb)
#pragma unroll
            for (int i = 0; i < 4; ++i) acc[t][mb][i] += tile_at(src, t, mb, i);
      }
      __syncthreads();   // 3
    }
    if (q == 1) store(y);
    __syncthreads();   // 4 (two groups: 2)
    if (q == 0) {
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
          const float sc = kNorm ? inv_rms[mb * 16 + (lane & 15)] : 1.f;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            float& d = tile_at(y, t, mb, i);
            d = (acc[t][mb][i] + d) * sc;
          }
        }
    }
    __syncthreads();   // 5 (two groups: 3)
  }

  // epilogues: items of (tile w, row m, column or pair)
  if constexpr (EPI == EPI_STORE) {
    for (int idx = threadIdx.x; idx < kGemmTiles * ROWS * 16; idx += NT) {
      const int w = idx / (ROWS * 16), r = idx % (ROWS * 16), m = r >> 4, cc = r & 15;
      const int nw = (blockIdx.x * kGemmTiles + w) * kTile;
      if (nw < N && m < M) a.out[((size_t)split * M + m) * N + nw + cc] = y[(w * ROWS + m) * kYStride + cc];
    }
  } else if constexpr (EPI == EPI_ROPE) {
    for (int idx = threadIdx.x; idx < kGemmTiles * ROWS * 8; idx += NT) {
      const int w = idx / (ROWS * 8), r = idx % (ROWS * 8), m = r >> 3, pr = r & 7;
      const int nw = (blockIdx.x * kGemmTiles + w) * kTile;
      if (nw >= N || m >= M || !live_s[m]) continue;
      const int b = m / a.rps, j = m - b * a.rps;
      const int slot = a.st[b].base + j;
      const int head = nw / a.D, d = ((nw % a.D) >> 1) + pr;
      const float e = y[(w * ROWS + m) * kYStride + 2 * pr], o = y[(w * ROWS + m) * kYStride + 2 * pr + 1];
      if (head < a.nq + a.nkv) {
        const float2 cs = a.rcs[(size_t)m * (a.D / 2) + d];
        const float re = e * cs.x - o * cs.y, ro = e * cs.y + o * cs.x;
        if (head < a.nq) {
          *reinterpret_cast<uint32_t*>(a.q + ((size_t)m * a.nq + head) * a.D + 2 * d) = pack2(re, ro);
        } else {
          const size_t pg = (size_t)a.pt[b * a.pps + slot / kAttnChunk] * a.nkv + (head - a.nq);
          *reinterpret_cast<uint32_t*>(a.kc + (pg * kAttnChunk + slot % kAttnChunk) * a.D + 2 * d) =
              pack2(re, ro);
        }
      } else {
        const size_t pg = (size_t)a.pt[b * a.pps + slot / kAttnChunk] * a.nkv + (head - a.nq - a.nkv);
        bf16_t* vp = a.vt + (pg * a.D + 2 * d) * kAttnChunk + slot % kAttnChunk;
        vp[0] = f2bf(e);
        vp[kAttnChunk] = f2bf(o);
      }
    }
  } else if constexpr (EPI == EPI_RESID) {
    // 16 consecutive threads share (w, m): the row's sum of squares over the
    // tile is a 16-lane reduction
    for (int idx = threadIdx.x; idx < kGemmTiles * ROWS * 16; idx += NT) {
      const int w = idx / (ROWS * 16), r = idx % (ROWS * 16), m = r >> 4, cc = r & 15;
      const int nw = (blockIdx.x * kGemmTiles + w) * kTile;
      const bool ok = nw < N && m < M;
      float xn = 0.f;
      if (ok) {
        const int n = nw + cc;
        xn = a.x32[(size_t)m * N + n];
        if (live_s[m]) {                      // rows of idle sequences keep their stream
          xn += y[(w * ROWS + m) * kYStride + cc];
          a.x32[(size_t)m * N + n] = xn;
        }
        a.xg[(size_t)m * N + n] = f2bf(xn * bf2f(a.gain[n]));
      }
      float sq = xn * xn;
      for (int o = 1; o < 16; o <<= 1) sq += __shfl_xor(sq, o);
      if (ok && cc == 0) a.ss_out[(size_t)(nw / kTile) * a.mpad + m] = sq;
    }
  } else if constexpr (EPI == EPI_SWIGLU) {
    // tiles 2j, 2j+1: gate and up rows of features 16 j' .. +16, j' = 2 blockIdx.x + j
    const int F = N / 2;
    for (int idx = threadIdx.x; idx < 2 * ROWS * 16; idx += NT) {
      const int j = idx / (ROWS * 16), r = idx % (ROWS * 16), m = r >> 4, cc = r & 15;
      const int f = (2 * blockIdx.x + j) * kTile + cc;
      if (f >= F || m >= M) continue;
      const float g = y[(2 * j * ROWS + m) * kYStride + cc];
      const float up = y[((2 * j + 1) * ROWS + m) * kYStride + cc];
      a.u[(size_t)m * F + f] = f2bf(g / (1.f + expf(-g)) * up);
    }
  } else {   // EPI_ARGMAX
    if (a.allow_logits) {
      for (int idx = threadIdx.x; idx < kGemmTiles * ROWS * 16; idx += NT) {
        const int w = idx / (ROWS * 16), r = idx % (ROWS * 16), m = r >> 4, cc = r & 15;
        const int nw = (blockIdx.x * kGemmTiles + w) * kTile;
        if (nw < N && m < M && a.st[m / a.rps].want_logits)
          a.logits[(size_t)m * N + nw + cc] = f2bf(y[(w * ROWS + m) * kYStride + cc]);
      }
    }
    for (int idx = threadIdx.x; idx < kGemmTiles * ROWS; idx += NT) {
      const int w = idx / ROWS, m = idx % ROWS;
      const int nw = (blockIdx.x * kGemmTiles + w) * kTile;
      if (nw >= N || m >= M) continue;
      float best = -INFINITY;
      int bi = nw;
      bool nan = false;
      for (int cc = 0; cc < 16; ++cc) {
        float v = y[(w * ROWS + m) * kYStride + cc];
        if (v != v) {
          nan = true;
          v = -INFINITY;
        }
        if (v > best) {
          best = v;
          bi = nw + cc;
        }
      }
      a.amax_v[(size_t)(nw / kTile) * a.mpad + m] = best;
      a.amax_i[(size_t)(nw / kTile) * a.mpad + m] = bi;
      if (nan && live_s[m]) atomicOr(const_cast<int32_t*>(&a.st[m / a.rps].err), ERR_NUMERIC);
    }
  }
}

// ---------------------------------------------------------------------------
// Wide-unit GEMM over the tile-packed weights for passes of 33 to 160 rows
// (3 to 10 row blocks): the gate/up and LM-head projections in one launch, and
// the q/k/v, o and down projections as k-split partial sums.  Gate/up and the
// LM head run one workgroup per CU, each over an even, contiguous share of the
// tile pairs walked in chunks of at most kWideTiles = 16 tiles (256 columns);
// a k-split launch gives each workgroup 16 tiles and the k-range of split
// blockIdx.y.  The 8 waves are 4 column groups x 2 k-groups: wave (cg, kg)
// multiplies tiles 4 cg .. 4 cg + 3 over the kg-th half of the k-range, so
// each x operand it reads from LDS feeds 4 MFMAs and each weight block MB of
// them, and the two k-groups keep two independent streams of loads in flight.
// Per 32-wide k-step each k-group stages the x operands of all rows by
// buffer-to-LDS loads straight in MFMA operand order (block rb of a step: 16
// rows x 32 columns, lane l's 16 bytes at 16 l) into its own ring of D + 1
// slots, D steps ahead; weights go to registers the same depth ahead.  x is
// read from a step-major copy where the producer wrote one (each block then
// one contiguous 1 KB run), else from row-major rows.  One
// barrier per step; its wait count is set by hand (every wave issues the same
// loads per step: its share of its k-group's x blocks, then its 4 weight
// blocks), so that every step in flight stays in flight.  A load past its
// k-group's range or past the last tile gets an offset past the operand and
// returns zeros without a memory access; rows past M read past the end of x
// and are never stored.  At the end the second k-group's partial tiles are
// added to the first's through LDS (first half + second half of the k-range),
// and the first k-group runs the epilogue.
// ---------------------------------------------------------------------------
constexpr int kWideTiles = 16;
constexpr int kWideWaves = 8;
constexpr int kWideCg = 4;                          // column groups
constexpr int kWideTpw = kWideTiles / kWideCg;      // tiles per wave
constexpr int kWideSlice = 8;                       // sums of squares per partial of the 1/rms prologue
// steps in flight per k-group: 4, or 3 for 9 and 10 row blocks (whose
// accumulators take 144 and 160 of a wave's 256 registers)
constexpr int wide_depth(int mb) { return mb >= 9 ? 3 : 4; }

__device__ __forceinline__ void lds_load16(__amdgpu_buffer_rsrc_t r, unsigned char* dst, int voff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)(dst), 16, voff, 0, 0, 0);
}

// the two x rings, the dummy block (target of the spare x loads) and the
// 1/rms partials; the final k-group sum reuses the rings (8 MB blocks)
size_t wide_lds_bytes(int mb, int H) {
  const int nsl = (H / kTile + kWideSlice - 1) / kWideSlice;
  return (size_t)2 * (wide_depth(mb) + 1) * mb * 1024 + 1024 + (size_t)nsl * 16 * mb * sizeof(float);
}

template <int MB, int EPI>
__global__ __launch_bounds__(kWideWaves * 64, 1) void k_gemm_wide(GemvArgs a) {
  static_assert(EPI == EPI_SWIGLU || EPI == EPI_ARGMAX || EPI == EPI_STORE, "wide-unit epilogues");
  constexpr bool kNorm = EPI != EPI_STORE;
  constexpr int ROWS = 16 * MB, TPW = kWideTpw, D = wide_depth(MB), NB = D + 1, NT = kWideWaves * 64;
  constexpr int XPW = (MB + kWideCg - 1) / kWideCg;   // x blocks each wave stages per step
  // loads issued after step c's x loads while they are awaited: that step's
  // weights, then D - 1 steps of both
  constexpr int WAITN = TPW + (D - 1) * (XPW + TPW);
  static_assert(2 * NB >= 2 * kWideCg, "the k-group sum reuses the x rings");
  static_assert(TPW == 4, "the weight wait names four register tuples");
  extern __shared__ __align__(16) unsigned char lds[];
  __shared__ float inv_rms[ROWS];
  __shared__ int live_s[ROWS];
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6)), lane = threadIdx.x & 63;
  const int cg = wave % kWideCg, kg = wave / kWideCg;
  const int M = a.M, N = a.N, ntiles = N / kTile;
  const int T = (a.Kd + 31) >> 5;
  const int split = blockIdx.y;
  const int s0 = (int)((long long)split * T / a.splits), s1 = (int)((long long)(split + 1) * T / a.splits);
  const int half = (s1 - s0 + 1) >> 1;
  const int kb = kg ? s0 + half : s0, ke = kg ? s1 : s0 + half;   // this k-group's steps [kb, ke)
  // Units of two tiles (a gate/up pair).  SwiGLU and argmax: contiguous
  // ranges of units dealt evenly to the gridDim.x workgroups (one per CU), so
  // that every CU streams the same share of the weights, each range walked in
  // chunks of at most 8 units (16 tiles); k-split partial sums: 8 units per
  // workgroup.
  const int nunits = ntiles >> 1;
  int u0, u1;
  if constexpr (EPI == EPI_STORE) {
    u0 = blockIdx.x * (kWideTiles / 2);
    u1 = min(u0 + kWideTiles / 2, nunits);
  } else {
    u0 = (int)((long long)blockIdx.x * nunits / gridDim.x);
    u1 = (int)((long long)(blockIdx.x + 1) * nunits / gridDim.x);
  }
  const int nch = (u1 - u0 + kWideTiles / 2 - 1) / (kWideTiles / 2);
  const int cu = nch > 0 ? (u1 - u0 + nch - 1) / nch : 1;   // units per chunk
  int tile0 = 0, tend = 0;   // this wave's first tile, the chunk's end tile
  // step-major x spans whole 32-wide steps (its buffer is padded to them:
  // columns past Kd meet zero weight columns)
  const __amdgpu_buffer_rsrc_t rx = __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16_t*>(a.x), 0,
                                                                      a.xpk ? T * M * 64 : M * a.ldx * 2, kRsrcWord3);
  unsigned char* ring = lds + (size_t)kg * NB * MB * 1024;           // [NB][MB] blocks of 1 KB
  unsigned char* dummy = lds + (size_t)2 * NB * MB * 1024;           // target of the spare x loads
  float* rms_part = reinterpret_cast<float*>(dummy + 1024);          // [slices][ROWS]
  const int nt16 = kNorm ? a.H / kTile : 0, nsl = (nt16 + kWideSlice - 1) / kWideSlice;

  for (int m = threadIdx.x; m < ROWS; m += NT) {
    int lv = 0;
    if (m < M) {
      const int b = m / a.rps;
      lv = (m - b * a.rps) < a.st[b].count ? 1 : 0;
    }
    live_s[m] = lv;
  }

  // x operand of block b at step st: byte offset xbase[j] + st * xstride;
  // lane l reads row 16 b + (l & 15), 16 bytes at column 32 st + 8 (l >> 4)
  // (MFMA operand order).  Row-major x: 16 rows of 64 bytes ldx apart.
  // Step-major x (xpk, [Kd/32][M][32]): the block is one contiguous 1 KB run.
  const int xstride = a.xpk ? M * 64 : 64;
  int xbase[XPW];
#pragma unroll
  for (int j = 0; j < XPW; ++j) {
    const int b = cg + kWideCg * j;
    const int r = 16 * b + (lane & 15);
    xbase[j] = a.xpk ? r * 64 + 16 * (lane >> 4) : (r * a.ldx + 8 * (lane >> 4)) * 2;
  }
  const int lane_w = 16 * lane;
  // Offsets past a k-group's range or the last tile are ORed with kOut (a
  // wave-uniform scalar select): every offset stays below 2^31, so the result
  // lies past the operand, and no branch splits the loads (a branch would
  // make the compiler drain every load in flight where the paths join).
  auto issue_x = [&](int c) {
    const int st = kb + c;
    const int oob = st < ke ? 0 : kOut;
    unsigned char* slot = ring + (c % NB) * (MB * 1024);
#pragma unroll
    for (int j = 0; j < XPW; ++j) {
      const int b = cg + kWideCg * j;
      const int ob = b < MB ? oob : kOut;
      lds_load16(rx, b < MB ? slot + b * 1024 : dummy, (xbase[j] + st * xstride) | ob);
    }
  };
  // The weight loads are written as inline assembly, and waited for by hand
  // below.  The compiler's own wait counts leave out the buffer-to-LDS loads
  // it issues between them, so they would wait for several steps' loads at
  // once where one step's are due.
  const uint64_t wbase = reinterpret_cast<uint64_t>(a.pw);
  const u32x4 wdesc = u32x4{(uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)wbase),
                            (uint32_t)__builtin_amdgcn_readfirstlane((int)((wbase >> 32) & 0xffffu)),
                            (uint32_t)(ntiles * T * 1024), (uint32_t)kRsrcWord3};
  auto issue_w = [&](int c, u32x4 (&wr)[TPW]) {
    const int st = kb + c;
    const int oob = st < ke ? 0 : kOut;
#pragma unroll
    for (int t = 0; t < TPW; ++t) {
      const int ot = tile0 + t < tend ? oob : kOut;
      const int off = (lane_w + ((tile0 + t) * T + st) * 1024) | ot;
      asm volatile("buffer_load_dwordx4 %0, %1, %2, 0 offen nt" : "=v"(wr[t]) : "v"(off), "s"(wdesc) : "memory");
    }
  };

  // 1/rms, first half: partial sums of kWideSlice consecutive per-16-column
  // sums of squares per (slice, row)
  if constexpr (kNorm) {
    for (int it = threadIdx.x; it < nsl * ROWS; it += 4 * NT) {   // up to 4 items per thread and round
      float v[4][kWideSlice];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int item = it + r * NT, sl = item / ROWS, m = item % ROWS;
#pragma unroll
        for (int k = 0; k < kWideSlice; ++k) {
          const int g = sl * kWideSlice + k;
          v[r][k] = (item < nsl * ROWS && g < nt16) ? a.ss_in[(size_t)g * a.mpad + m] : 0.f;
        }
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int item = it + r * NT;
        float sum = 0.f;
#pragma unroll
        for (int k = 0; k < kWideSlice; ++k) sum += v[r][k];
        if (item < nsl * ROWS) rms_part[item] = sum;
      }
    }
    __syncthreads();
    // 1/rms, second half: the slices of each row in order
    for (int m = threadIdx.x; m < ROWS; m += NT) {
      float t = 0.f;
      for (int sl = 0; sl < nsl; ++sl) t += rms_part[sl * ROWS + m];
      inv_rms[m] = live_s[m] ? rsqrtf(t / a.H + a.eps) : 0.f;
    }
  }
  __syncthreads();

  for (int cs = u0; cs < u1; cs += cu) {   // workgroup-uniform
  tile0 = 2 * cs + cg * TPW;
  tend = 2 * min(cs + cu, u1);
  u32x4 wr[D][TPW];
#pragma unroll
  for (int i = 0; i < D; ++i) {
    issue_x(i);
    issue_w(i, wr[i]);
  }
  f32x4 acc[TPW][MB];
#pragma unroll
  for (int t = 0; t < TPW; ++t)
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) acc[t][mb] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int c0 = 0; c0 < half; c0 += D) {   // workgroup-uniform
#pragma unroll
    for (int uu = 0; uu < D; ++uu) {
      const int c = c0 + uu;
      // step c's x (every wave's share) has landed and is visible; the
      // memory clobbers keep LDS accesses on their side of the barrier
      asm volatile("s_waitcnt vmcnt(%0)" ::"n"(WAITN) : "memory");
      __builtin_amdgcn_s_barrier();
      asm volatile("" ::: "memory");
      const unsigned char* xb = ring + (c % NB) * (MB * 1024) + 16 * lane;
      // step c's weights: the loads issued after them are D - 1 steps of x
      // and weights; the registers are operands of the wait, so nothing reads
      // them before it
      asm volatile("s_waitcnt vmcnt(%4)"
                   : "+v"(wr[uu][0]), "+v"(wr[uu][1]), "+v"(wr[uu][2]), "+v"(wr[uu][3])
                   : "n"((D - 1) * (XPW + TPW))
                   : "memory");
      u32x4 w[TPW];
#pragma unroll
      for (int t = 0; t < TPW; ++t) w[t] = wr[uu][t];
      if (kb + c < ke) {   // wave-uniform
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
          const u32x4 xv = *reinterpret_cast<const u32x4*>(xb + mb * 1024);
#pragma unroll
          for (int t = 0; t < TPW; ++t) acc[t][mb] = mfma16x16x32(w[t], xv, acc[t][mb]);
        }
      }
      asm volatile("" ::: "memory");
      // slot (c + D) % NB was last read at step c - 1, before this step's barrier
      issue_x(c + D);
      issue_w(c + D, wr[uu]);
    }
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // the spare loads past the end
  __syncthreads();

  // the second k-group's partial tiles onto the first's, two tiles at a time
  f32x4* red = reinterpret_cast<f32x4*>(lds);   // [2][kWideCg][MB][64]
#pragma unroll
  for (int h = 0; h < TPW / 2; ++h) {
    if (kg == 1) {
#pragma unroll
      for (int tt = 0; tt < 2; ++tt)
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) red[((tt * kWideCg + cg) * MB + mb) * 64 + lane] = acc[2 * h + tt][mb];
    }
    __syncthreads();
    if (kg == 0) {
#pragma unroll
      for (int tt = 0; tt < 2; ++tt)
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) acc[2 * h + tt][mb] += red[((tt * kWideCg + cg) * MB + mb) * 64 + lane];
    }
    __syncthreads();
  }
  if (kg == 0) {
  const int grp = lane >> 4;
  if constexpr (EPI == EPI_STORE) {
    // fp32 partial sums of this split: out[split][m][n]
#pragma unroll
    for (int t = 0; t < TPW; ++t) {
      const int tile = tile0 + t;
      if (tile >= tend) continue;
      const int n = tile * kTile + 4 * grp;
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        const int m = mb * 16 + (lane & 15);
        if (m < M) *reinterpret_cast<f32x4*>(a.out + ((size_t)split * M + m) * N + n) = acc[t][mb];
      }
    }
  } else if constexpr (EPI == EPI_SWIGLU) {
    // tiles tile0 + 2j, tile0 + 2j + 1: the gate and up rows of features
    // 16 (tile0 / 2 + j) .. +16
    const int F = N / 2;
#pragma unroll
    for (int j = 0; j < TPW / 2; ++j) {
      const int f = ((tile0 >> 1) + j) * kTile + 4 * grp;
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        const int m = mb * 16 + (lane & 15);
        if (m >= M || f >= F || tile0 + 2 * j >= tend) continue;
        const float r = inv_rms[m];
        float o[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float g = acc[2 * j][mb][i] * r, up = acc[2 * j + 1][mb][i] * r;
          o[i] = live_s[m] ? g / (1.f + expf(-g)) * up : 0.f;
        }
        const size_t at = a.upk ? ((size_t)(f >> 5) * M + m) * 32 + (f & 31) : (size_t)m * F + f;
        *reinterpret_cast<u32x2*>(a.u + at) = u32x2{pack2(o[0], o[1]), pack2(o[2], o[3])};
      }
    }
  } else {   // EPI_ARGMAX: per tile and row, the (max, index) of its 16 logits
#pragma unroll
    for (int t = 0; t < TPW; ++t) {
      const int tile = tile0 + t;
      if (tile >= tend) continue;
      const int n = tile * kTile + 4 * grp;
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        const int m = mb * 16 + (lane & 15);
        const int mm = m < ROWS ? m : ROWS - 1;
        const bool live = m < M && live_s[mm];
        const float r = inv_rms[mm];
        float y[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) y[i] = live ? acc[t][mb][i] * r : 0.f;
        if (a.allow_logits && m < M && a.st[m / a.rps].want_logits)
          *reinterpret_cast<u32x2*>(a.logits + (size_t)m * N + n) = u32x2{pack2(y[0], y[1]), pack2(y[2], y[3])};
        float best = -INFINITY;
        int bi = n;
        int nan = 0;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float v = y[i];
          if (v != v) {
            nan = 1;
            v = -INFINITY;
          }
          if (v > best) {
            best = v;
            bi = n + i;
          }
        }
#pragma unroll
        for (int o = 16; o <= 32; o <<= 1) {
          const float v2 = __shfl_xor(best, o);
          const int i2 = __shfl_xor(bi, o);
          nan |= __shfl_xor(nan, o);
          amax_merge(best, bi, v2, i2);
        }
        if (grp == 0 && m < M) {
          a.amax_v[(size_t)tile * a.mpad + m] = best;
          a.amax_i[(size_t)tile * a.mpad + m] = bi;
          if (nan && live) atomicOr(const_cast<int32_t*>(&a.st[m / a.rps].err), ERR_NUMERIC);
        }
      }
    }
  }
  }   // kg == 0
  __syncthreads();   // the chunk's LDS reads are done before the next chunk's loads land
  }   // chunks
}

// CUs of the current device (the wide kernel's grid for SwiGLU and argmax)
int wide_cus() {
  int dev = 0, n = 0;
  if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      n < 1) {
    (void)hipGetLastError();
    return 256;
  }
  return n;
}

template <int EPI>
hipError_t launch_wide(const GemvArgs& g, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  const int mb = (g.M + 15) / 16;
  const int groups = (g.N / kTile + kWideTiles - 1) / kWideTiles;
  const dim3 grid(EPI == EPI_STORE ? groups : std::min(wide_cus(), g.N / kTile / 2), g.splits), block(kWideWaves * 64);
  const size_t lds = wide_lds_bytes(mb, EPI == EPI_STORE ? 0 : g.H);
  switch (mb) {
    case 3: hipExtLaunchKernelGGL((k_gemm_wide<3, EPI>), grid, block, lds, s, e0, e1, 0, g); break;
    case 4: hipExtLaunchKernelGGL((k_gemm_wide<4, EPI>), grid, block, lds, s, e0, e1, 0, g); break;
    case 5: hipExtLaunchKernelGGL((k_gemm_wide<5, EPI>), grid, block, lds, s, e0, e1, 0, g); break;
    case 6: hipExtLaunchKernelGGL((k_gemm_wide<6, EPI>), grid, block, lds, s, e0, e1, 0, g); break;
    case 7: hipExtLaunchKernelGGL((k_gemm_wide<7, EPI>), grid, block, lds, s, e0, e1, 0, g); break;
    case 8: hipExtLaunchKernelGGL((k_gemm_wide<8, EPI>), grid, block, lds, s, e0, e1, 0, g); break;
    case 9: hipExtLaunchKernelGGL((k_gemm_wide<9, EPI>), grid, block, lds, s, e0, e1, 0, g); break;
    case 10: hipExtLaunchKernelGGL((k_gemm_wide<10, EPI>), grid, block, lds, s, e0, e1, 0, g); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <int MB>
void set_wide_attributes(int limit) {
  const int lds = (int)std::min((size_t)limit, wide_lds_bytes(MB, 8192));
  const void* f[3] = {reinterpret_cast<const void*>(&k_gemm_wide<MB, EPI_SWIGLU>),
                      reinterpret_cast<const void*>(&k_gemm_wide<MB, EPI_ARGMAX>),
                      reinterpret_cast<const void*>(&k_gemm_wide<MB, EPI_STORE>)};
  for (const void* p : f) (void)hipFuncSetAttribute(p, hipFuncAttributeMaxDynamicSharedMemorySize, lds);
}

template <int EPI>
hipError_t launch_mb(const GemvArgs& g, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  const int mb = (g.M + 15) / 16;
  const dim3 grid((g.N + kGemmTiles * kTile - 1) / (kGemmTiles * kTile), g.splits), block(threads_for(mb));
  const size_t lds = gemm_lds_bytes(g.M);
  switch (mb) {
    case 2: hipExtLaunchKernelGGL((k_gemm<2, EPI>), grid, block, lds, s, e0, e1, 0, g); break;
    case 3: hipExtLaunchKernelGGL((k_gemm<3, EPI>), grid, block, lds, s, e0, e1, 0, g); break;
    case 4: hipExtLaunchKernelGGL((k_gemm<4, EPI>), grid, block, lds, s, e0, e1, 0, g); break;
    case 5: hipExtLaunchKernelGGL((k_gemm<5, EPI>), grid, block, lds, s, e0, e1, 0, g); break;
    case 6: hipExtLaunchKernelGGL((k_gemm<6, EPI>), grid, block, lds, s, e0, e1, 0, g); break;
    case 7: hipExtLaunchKernelGGL((k_gemm<7, EPI>), grid, block, lds, s, e0, e1, 0, g); break;
    case 8: hipExtLaunchKernelGGL((k_gemm<8, EPI>), grid, block, lds, s, e0, e1, 0, g); break;
    case 9: hipExtLaunchKernelGGL((k_gemm<9, EPI>), grid, block, lds, s, e0, e1, 0, g); break;
    case 10: hipExtLaunchKernelGGL((k_gemm<10, EPI>), grid, block, lds, s, e0, e1, 0, g); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <int MB>
void set_mb_attributes(int limit) {
  const int lds = (int)std::max(x_lds_bytes(MB), y_lds_bytes(MB));
  if (lds > limit) return;   // such a launch is rejected by the host-side LDS check
  const void* f[5] = {reinterpret_cast<const void*>(&k_gemm<MB, EPI_STORE>),
                      reinterpret_cast<const void*>(&k_gemm<MB, EPI_ROPE>),
                      reinterpret_cast<const void*>(&k_gemm<MB, EPI_RESID>),
                      reinterpret_cast<const void*>(&k_gemm<MB, EPI_SWIGLU>),
                      reinterpret_cast<const void*>(&k_gemm<MB, EPI_ARGMAX>)};
  for (const void* p : f) (void)hipFuncSetAttribute(p, hipFuncAttributeMaxDynamicSharedMemorySize, lds);
}

}  // namespace

size_t gemm_lds_bytes(int M) {
  const int mb = (M + 15) / 16;
  return std::max(x_lds_bytes(mb), y_lds_bytes(mb));
}

void gemm_set_attributes(int limit) {
  set_mb_attributes<2>(limit);
  set_mb_attributes<3>(limit);
  set_mb_attributes<4>(limit);
  set_mb_attributes<5>(limit);
  set_mb_attributes<6>(limit);
  set_mb_attributes<7>(limit);
  set_mb_attributes<8>(limit);
  set_mb_attributes<9>(limit);
  set_mb_attributes<10>(limit);
  set_wide_attributes<3>(limit);
  set_wide_attributes<4>(limit);
  set_wide_attributes<5>(limit);
  set_wide_attributes<6>(limit);
  set_wide_attributes<7>(limit);
  set_wide_attributes<8>(limit);
  set_wide_attributes<9>(limit);
  set_wide_attributes<10>(limit);
}

hipError_t gemm_launch(int epi, const GemvArgs& g, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  if (g.M <= kSgMaxRowsGemm || g.M > SPEC_MAX_ROWS || g.splits < 1 || (epi != EPI_STORE && g.splits != 1) ||
      g.N % kTile != 0 || g.Kd % 8 != 0)
    return hipErrorInvalidValue;
  // the 1/rms prologue reads at most lpt_for(parts) sums of squares per
  // thread, in threads_for / rows parts per row
  {
    const int mb = (g.M + 15) / 16, parts = threads_for(mb) / (16 * mb);
    if ((epi == EPI_ROPE || epi == EPI_SWIGLU || epi == EPI_ARGMAX) &&
        (g.H < kTile || g.H / kTile > lpt_for(parts) * parts))
      return hipErrorInvalidValue;
  }
  // every operand is addressed with 32-bit byte offsets below kOut
  if ((long long)g.N * ((g.Kd + 31) / 32) * 64 >= kOut || (long long)g.M * g.ldx * 2 >= kOut) return hipErrorInvalidValue;
  // passes of more than kSgMaxRows rows over the tile-packed copy: the
  // wide-unit kernel for gate/up (tile pairs) and the LM head in one launch,
  // and for the k-split partial sums of the other projections
  {
    const int mb = (g.M + 15) / 16;
    const bool wide = g.pw && g.M > kSgMaxRows && mb <= 10 && (g.N / kTile) % 2 == 0 &&
                      (epi == EPI_STORE || ((epi == EPI_SWIGLU || epi == EPI_ARGMAX) && g.splits == 1)) &&
                      wide_lds_bytes(mb, epi == EPI_STORE ? 0 : g.H) <= (size_t)gemv_lds_limit();
    if (g.xpk && !wide) return hipErrorInvalidValue;   // only the wide kernel reads step-major x
    if (wide) {
      if (epi == EPI_STORE) return launch_wide<EPI_STORE>(g, s, e0, e1);
      return epi == EPI_SWIGLU ? launch_wide<EPI_SWIGLU>(g, s, e0, e1) : launch_wide<EPI_ARGMAX>(g, s, e0, e1);
    }
  }
  switch (epi) {
    case EPI_STORE: return launch_mb<EPI_STORE>(g, s, e0, e1);
    case EPI_ROPE: return launch_mb<EPI_ROPE>(g, s, e0, e1);
    case EPI_RESID: return launch_mb<EPI_RESID>(g, s, e0, e1);
    case EPI_SWIGLU: return launch_mb<EPI_SWIGLU>(g, s, e0, e1);
    case EPI_ARGMAX: return launch_mb<EPI_ARGMAX>(g, s, e0, e1);
    default: return hipErrorInvalidValue;
  }
}

// k-splits of the down projection over M > kThinRows rows: as many as fit
// the resident workgroup slots in one round (a count that overflows them
// leaves a second round for the few workgroups left over, which doubles the
// projection's time: 56 groups x 5 splits = 280 workgroups on 256 slots),
// at least 8 k-steps per split.
int gemm_down_splits(int N, int Kd, int ncu) {
  const int groups = (N + kGemmTiles * kTile - 1) / (kGemmTiles * kTile);
  const int T = (Kd + 31) / 32;
  int s = std::max(1, ncu / groups);
  return std::max(1, std::min(s, T / 8));
}

int gemm_wide_splits(int N, int Kd, int ncu) {
  // one round of resident workgroups (one per CU), at least 16 k-steps per
  // split (8 per k-group)
  const int groups = (N / kTile + kWideTiles - 1) / kWideTiles;
  const int T = (Kd + 31) / 32;
  return std::max(1, std::min(ncu / groups, T / 16));
}

int gemm_wgs_per_cu(int M) {
  // only the 8-wave shape of up to three row blocks is sized for two
  // workgroups per CU; the wider ones keep one, so that their (larger) k-split
  // partials do not double
  const int mb = (M + 15) / 16;
  const void* f = nullptr;
  switch (mb) {
    case 2: f = reinterpret_cast<const void*>(&k_gemm<2, EPI_STORE>); break;
    case 3: f = reinterpret_cast<const void*>(&k_gemm<3, EPI_STORE>); break;
    default: return 1;
  }
  int n = 0;
  const size_t lds = gemm_lds_bytes(M);
  if (hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) != hipSuccess ||
      hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, f, threads_for(mb), lds) != hipSuccess) {
    (void)hipGetLastError();
    return 1;
  }
  return std::max(1, std::min(n, 2));
}

int gemm_qkv_splits(int N, int Kd, int M, int ncu) {
  const int groups = (N + kGemmTiles * kTile - 1) / (kGemmTiles * kTile);
  if (2 * groups >= ncu) return 1;
  // one workgroup per CU: measured faster here than filling both slots, as
  // the doubled partials outweigh the extra streams
  const int s = gemm_down_splits(N, Kd, ncu);
  // Passes of more than 32 rows always split: such a GEMM is far from
  // streaming its weights at full rate (the time goes into each workgroup's
  // MFMA and x-operand work), so spreading it over s times the workgroups
  // pays for the partials (144 rows: 72 workgroups -> 3 x 72).  Fewer rows
  // split only while 2 * s * M * N fp32 partial bytes <= (N * Kd bf16 weight
  // bytes) / 10.
  return (M > kSgMaxRows || (long long)40 * s * M <= Kd) ? s : 1;
}

int gemm_qkv_splits_for(int N, int Kd, int M, int ncu, bool wide) {
  return (wide && M > kSgMaxRows) ? gemm_wide_splits(N, Kd, ncu) : gemm_qkv_splits(N, Kd, M, ncu);
}

}  // namespace specdec
