// Batched-row GEMM on MFMA for passes of more than kThinRows rows (several
// sequences verified together), and of 17..kThinRows rows whose width the
// thin GEMV cannot stage (one sequence with K = 16 at hidden 4096): y[m][n] = sum_k x[m][k] W[n][k] for up to
// SPEC_MAX_ROWS rows, with the same fused epilogues as the thin GEMV kernels
// (1/rms row scale, rotary + paged KV append, residual + next-norm input,
// SwiGLU, per-tile argmax, or k-split partial sums).
//
// A workgroup of 4 waves owns 64 output columns (wave w: the 16-column tile
// 4*blockIdx.x + w) and the k-range of split blockIdx.y.  The k-range is
// walked in chunks of 64 columns (two 32-wide MFMA steps).  Every chunk's x
// rows are staged once in LDS and shared by the 4 waves; each wave streams
// its own 16 weight rows.  Loads run kStages chunks ahead: chunk c's x
// vectors and weight fragments sit in registers while chunks c-1.. are
// multiplied, then x goes to one of two LDS buffers.  Workgroup barriers wait
// for LDS traffic only, never for the loads in flight.
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

namespace specdec {

namespace {

constexpr int kChunk = 64;                    // k columns per stage
constexpr int kStages = 3;                    // chunks of loads in flight
constexpr int kXStride = kChunk + 8;          // bf16 per LDS x row (16-byte pad against bank conflicts)
constexpr int kYStride = 17;                  // floats per row of a wave's output tile in LDS

size_t x_lds_bytes(int rows) { return (size_t)2 * rows * kXStride * sizeof(bf16_t); }
size_t y_lds_bytes(int rows) { return (size_t)kGemmWaves * rows * kYStride * sizeof(float); }

template <int MB, int EPI>
__global__ __launch_bounds__(kGemmWaves * 64) void k_gemm(GemvArgs a) {
  constexpr int ROWS = MB * 16;
  constexpr int XV = (ROWS * (kChunk / 8) + kGemmWaves * 64 - 1) / (kGemmWaves * 64);   // x vectors per thread
  constexpr bool kNorm = EPI == EPI_ROPE || EPI == EPI_SWIGLU || EPI == EPI_ARGMAX;
  constexpr int NT = kGemmWaves * 64;
  extern __shared__ __align__(16) unsigned char lds[];
  __shared__ float inv_rms[ROWS];
  __shared__ int live_s[ROWS];

  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int split = blockIdx.y;
  const int Kd = a.Kd, M = a.M, N = a.N;
  const int T = (Kd + 31) >> 5;
  const int s0 = (int)((long long)split * T / a.splits);
  const int s1 = (int)((long long)(split + 1) * T / a.splits);
  const int nch = (s1 - s0 + 1) >> 1;
  const int kq = 8 * (lane >> 4);
  const int n0 = (blockIdx.x * kGemmWaves + wave) * kTile;   // this wave's output columns
  const bool wtile = n0 < N;

  // this lane's weight row
  const bf16_t* wp = a.w[0];
  if (wtile) {
    const int r = lane & 15;
    if constexpr (EPI == EPI_SWIGLU) {
      // half-tile: rows 0-7 are gate rows n0/2 .. +8, rows 8-15 the matching up rows
      wp = r < 8 ? a.w[0] + (size_t)(n0 / 2 + r) * Kd : a.w[1] + (size_t)(n0 / 2 + r - 8) * Kd;
    } else {
      int sg = 0;
#pragma unroll
      for (int i = 1; i < 3; ++i)
        if (i < a.nseg && n0 >= a.row0[i]) sg = i;
      wp = a.w[sg] + (size_t)(n0 - a.row0[sg] + r) * Kd;
    }
  }

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

  // stage c: x vector v (v < ROWS*8) is row v >> 3, columns 8*(v & 7) .. +8 of
  // the chunk; dead rows, columns past the split or past Kd read as zeros
  auto issue = [&](int c, u32x4 (&xr)[XV], u32x4 (&wr)[2]) {
    const int kc = (s0 + 2 * c) * 32;
    const int kend = min(s1 * 32, Kd);
#pragma unroll
    for (int i = 0; i < XV; ++i) {
      const int v = threadIdx.x + NT * i;
      const int m = v >> 3, k = kc + 8 * (v & 7);
      const bool ok = v < ROWS * 8 && m < M && live_s[m] && k < kend;
      xr[i] = ok ? ld16(a.x + (size_t)m * a.ldx + k) : u32x4{0, 0, 0, 0};
    }
#pragma unroll
    for (int st = 0; st < 2; ++st) {
      const int k = kc + 32 * st + kq;
      wr[st] = (wtile && k < kend) ? ld16_nt(wp + k) : u32x4{0, 0, 0, 0};
    }
  };

  u32x4 xr[kStages][XV];
  u32x4 wr[kStages][2];
#pragma unroll
  for (int u = 0; u < kStages; ++u)
    if (u < nch) issue(u, xr[u], wr[u]);

  f32x4 acc[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) acc[mb] = f32x4{0.f, 0.f, 0.f, 0.f};
  bf16_t* xs = reinterpret_cast<bf16_t*>(lds);

  for (int c0 = 0; c0 < nch; c0 += kStages) {   // workgroup-uniform
#pragma unroll
    for (int u = 0; u < kStages; ++u) {
      const int c = c0 + u;
      if (c >= nch) break;
      bf16_t* xb = xs + (size_t)(c & 1) * ROWS * kXStride;
#pragma unroll
      for (int i = 0; i < XV; ++i) {
        const int v = threadIdx.x + NT * i;
        if (v < ROWS * 8) *reinterpret_cast<u32x4*>(xb + (v >> 3) * kXStride + 8 * (v & 7)) = xr[u][i];
      }
      // LDS stores visible to all waves; buffer c&1 was last read in chunk
      // c-2, before every wave passed chunk c-1's barrier
      __syncthreads();
      const u32x4 w0 = wr[u][0], w1 = wr[u][1];
      if (c + kStages < nch) issue(c + kStages, xr[u], wr[u]);
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        const bf16_t* xp = xb + (mb * 16 + (lane & 15)) * kXStride + kq;
        acc[mb] = mfma16x16x32(w0, *reinterpret_cast<const u32x4*>(xp), acc[mb]);
        acc[mb] = mfma16x16x32(w1, *reinterpret_cast<const u32x4*>(xp + 32), acc[mb]);
      }
    }
  }

  // 1/rms of each live row from the per-16-column sums of squares (fixed order)
  if constexpr (kNorm) {
    for (int m = wave; m < ROWS; m += kGemmWaves) {
      float v = 0.f;
      if (live_s[m])
        for (int t = lane; t < a.H / kTile; t += 64) v += a.ss_in[(size_t)t * a.mpad + m];
      for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
      if (lane == 0) inv_rms[m] = live_s[m] ? rsqrtf(v / a.H + a.eps) : 0.f;
    }
  }
  __syncthreads();   // x buffers are free; inv_rms is complete

  // wave tiles -> LDS: yw[wave][m][c]
  float* y = reinterpret_cast<float*>(lds);
  {
    float* yw = y + (size_t)wave * ROWS * kYStride;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      const int m = mb * 16 + (lane & 15);
      const float sc = kNorm ? inv_rms[m] : 1.f;
#pragma unroll
      for (int i = 0; i < 4; ++i) yw[m * kYStride + 4 * (lane >> 4) + i] = acc[mb][i] * sc;
    }
  }
  __syncthreads();

  // epilogues: items of (wave tile w, row m, column or pair)
  if constexpr (EPI == EPI_STORE) {
    for (int idx = threadIdx.x; idx < kGemmWaves * ROWS * 16; idx += NT) {
      const int w = idx / (ROWS * 16), r = idx % (ROWS * 16), m = r >> 4, cc = r & 15;
      const int nw = (blockIdx.x * kGemmWaves + w) * kTile;
      if (nw < N && m < M) a.out[((size_t)split * M + m) * N + nw + cc] = y[(w * ROWS + m) * kYStride + cc];
    }
  } else if constexpr (EPI == EPI_ROPE) {
    for (int idx = threadIdx.x; idx < kGemmWaves * ROWS * 8; idx += NT) {
      const int w = idx / (ROWS * 8), r = idx % (ROWS * 8), m = r >> 3, pr = r & 7;
      const int nw = (blockIdx.x * kGemmWaves + w) * kTile;
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
    for (int idx = threadIdx.x; idx < kGemmWaves * ROWS * 16; idx += NT) {
      const int w = idx / (ROWS * 16), r = idx % (ROWS * 16), m = r >> 4, cc = r & 15;
      const int nw = (blockIdx.x * kGemmWaves + w) * kTile;
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
    // columns 0-7 gate, 8-15 up of output features nw/2 .. nw/2 + 8
    const int F = N / 2;
    for (int idx = threadIdx.x; idx < kGemmWaves * ROWS * 8; idx += NT) {
      const int w = idx / (ROWS * 8), r = idx % (ROWS * 8), m = r >> 3, cc = r & 7;
      const int nw = (blockIdx.x * kGemmWaves + w) * kTile;
      if (nw >= N || m >= M) continue;
      const float g = y[(w * ROWS + m) * kYStride + cc];
      const float up = y[(w * ROWS + m) * kYStride + 8 + cc];
      a.u[(size_t)m * F + nw / 2 + cc] = f2bf(g / (1.f + expf(-g)) * up);
    }
  } else {   // EPI_ARGMAX
    if (a.allow_logits) {
      for (int idx = threadIdx.x; idx < kGemmWaves * ROWS * 16; idx += NT) {
        const int w = idx / (ROWS * 16), r = idx % (ROWS * 16), m = r >> 4, cc = r & 15;
        const int nw = (blockIdx.x * kGemmWaves + w) * kTile;
        if (nw < N && m < M && a.st[m / a.rps].want_logits)
          a.logits[(size_t)m * N + nw + cc] = f2bf(y[(w * ROWS + m) * kYStride + cc]);
      }
    }
    for (int idx = threadIdx.x; idx < kGemmWaves * ROWS; idx += NT) {
      const int w = idx / ROWS, m = idx % ROWS;
      const int nw = (blockIdx.x * kGemmWaves + w) * kTile;
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

template <int EPI>
hipError_t launch_mb(const GemvArgs& g, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  const int mb = (g.M + 15) / 16;
  const dim3 grid((g.N + kGemmWaves * kTile - 1) / (kGemmWaves * kTile), g.splits), block(kGemmWaves * 64);
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

}  // namespace

size_t gemm_lds_bytes(int M) {
  const int rows = 16 * ((M + 15) / 16);
  return std::max(x_lds_bytes(rows), y_lds_bytes(rows));
}

hipError_t gemm_launch(int epi, const GemvArgs& g, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  if (g.M <= kSgMaxRowsGemm || g.M > SPEC_MAX_ROWS || g.splits < 1 || (epi != EPI_STORE && g.splits != 1) ||
      g.N % kTile != 0 || g.Kd % 8 != 0)
    return hipErrorInvalidValue;
  switch (epi) {
    case EPI_STORE: return launch_mb<EPI_STORE>(g, s, e0, e1);
    case EPI_ROPE: return launch_mb<EPI_ROPE>(g, s, e0, e1);
    case EPI_RESID: return launch_mb<EPI_RESID>(g, s, e0, e1);
    case EPI_SWIGLU: return launch_mb<EPI_SWIGLU>(g, s, e0, e1);
    case EPI_ARGMAX: return launch_mb<EPI_ARGMAX>(g, s, e0, e1);
    default: return hipErrorInvalidValue;
  }
}

// k-splits of the down projection over M > kThinRows rows: enough
// workgroups to cover every CU once, at least two chunks per split.
int gemm_down_splits(int N, int Kd, int ncu) {
  const int groups = (N + kGemmWaves * kTile - 1) / (kGemmWaves * kTile);
  const int T = (Kd + 31) / 32;
  int s = std::max(1, (ncu + groups - 1) / groups);
  return std::max(1, std::min(s, T / (2 * 2)));
}

}  // namespace specdec
