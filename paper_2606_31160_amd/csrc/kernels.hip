// gfx950 kernels of the speculative verify-and-commit path.
//
// One pass (a verify of K+1 rows per sequence, or one draft step) is
//   embed+norm -> per layer { QKV GEMV -> reduce + rotary + KV append ->
//   split-KV attention -> combine -> O GEMV -> reduce + residual + norm ->
//   gate/up GEMV -> reduce + SwiGLU -> down GEMV -> reduce + residual + norm }
//   -> LM-head GEMV with per-tile argmax -> accept (verify) / pick (draft).
//
// Every length the kernels need (row base slot, row count, pending token,
// proposals) lives in device memory (SeqState), so one captured graph serves
// every round.
#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>

#include <algorithm>
#include <vector>
#include <cmath>

#include "ctx.h"
#include "device.h"
#include "gemv.h"
#include "sgemv.h"

namespace specdec {

// ---------------------------------------------------------------------------
// utility
// ---------------------------------------------------------------------------

// One thread waits `ticks` of the constant-rate wall clock, then exits.  The
// timing mode launches it ahead of a pass so that the host has enqueued the
// whole pass before its first kernel starts: the kernels then run back to back
// as in a graph replay instead of each starting on an idle device.
__global__ void k_hold(long long ticks) {
  const long long t0 = wall_clock64();
  while (wall_clock64() - t0 < ticks) __builtin_amdgcn_s_sleep(16);
}

// Read-only streaming: every 16-byte element of p once, non-temporal.  Each
// wave reads 8 KB chunks (eight consecutive 1 KB loads, all in flight), the
// chunks dealt round-robin over the waves of the grid; each wave writes the
// xor of what it read.
__global__ __launch_bounds__(256) void k_stream_read(const u32x4* p, size_t n, uint32_t* sink) {
  const size_t nw = (size_t)gridDim.x * (blockDim.x / 64);
  const size_t wid = (size_t)blockIdx.x * (blockDim.x / 64) + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  constexpr int kChunk = 8 * 64;   // 16-byte elements per chunk
  u32x4 acc = u32x4{0, 0, 0, 0};
  const size_t nchunks = n / kChunk;
  for (size_t c = wid; c < nchunks; c += nw) {
    const u32x4* q = p + c * kChunk + lane;
    u32x4 v[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) v[k] = __builtin_nontemporal_load(q + 64 * k);
#pragma unroll
    for (int k = 0; k < 8; ++k) acc ^= v[k];
  }
  for (size_t i = nchunks * kChunk + wid * 64 + lane; i < n; i += nw * 64) acc ^= __builtin_nontemporal_load(p + i);
  uint32_t x = acc.x ^ acc.y ^ acc.z ^ acc.w;
  for (int o = 32; o > 0; o >>= 1) x ^= __shfl_xor(x, o);
  if (lane == 0) sink[wid] = x;
}

__global__ void k_zero(u32x4* p, size_t n) {
  size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  for (; i < n; i += stride) p[i] = u32x4{0, 0, 0, 0};
}

// ---------------------------------------------------------------------------
// Prompt keys/values -> caches.  One thread per rotary pair of one slot of one
// kv head.  Keys are rotated with the model's positions (Eq. rope-3d with the
// axis assignment of Eq. axis-assign for the target; the slot index for the
// draft, Eq. flatrope-proj); values are stored transposed.  Slot s lives in
// page pt[s / kAttnChunk] at offset s % kAttnChunk; a page holds keys
// [nkv][kAttnChunk][D] and values [nkv][D][kAttnChunk].
// ---------------------------------------------------------------------------
struct PrefixArgs {
  const bf16_t* k_pre;   // [P][nkv][D]
  const bf16_t* v;       // [P][nkv][D]
  bf16_t* kc;            // this layer's key pool
  bf16_t* vt;            // this layer's value pool
  const int32_t* pt;     // this sequence's page table
  const int32_t* pos3;   // this sequence: [3][cap]
  const float2* cs;      // [cap][D/2]
  const int8_t* axis;    // [D/2]
  int P, nkv, D, cap, flat;
};

__global__ void k_prefix_kv(PrefixArgs a) {
  const int half = a.D / 2;
  const size_t total = (size_t)a.P * a.nkv * half;
  for (size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
       idx += (size_t)gridDim.x * blockDim.x) {
    const int d = (int)(idx % half);
    const int h = (int)((idx / half) % a.nkv);
    const int s = (int)(idx / ((size_t)half * a.nkv));
    const size_t src = ((size_t)s * a.nkv + h) * a.D + 2 * d;
    const float e = bf2f(a.k_pre[src]), o = bf2f(a.k_pre[src + 1]);
    const int p = a.flat ? s : a.pos3[a.axis[d] * a.cap + s];
    const float2 c = a.cs[(size_t)p * half + d];
    const float re = e * c.x - o * c.y, ro = e * c.y + o * c.x;
    const size_t pg = (size_t)a.pt[s / kAttnChunk] * a.nkv + h;
    const int off = s % kAttnChunk;
    *reinterpret_cast<uint32_t*>(a.kc + (pg * kAttnChunk + off) * a.D + 2 * d) = pack2(re, ro);
    a.vt[(pg * a.D + 2 * d) * kAttnChunk + off] = a.v[src];
    a.vt[(pg * a.D + 2 * d + 1) * kAttnChunk + off] = a.v[src + 1];
  }
}

// ---------------------------------------------------------------------------
// Verify staging: rows [pending, d_1..d_K].  Out-of-range ids are replaced by
// token 0 and flagged (reported by spec_sync).
// ---------------------------------------------------------------------------
__global__ void k_stage_verify(SeqState* st, const int32_t* over, int K, int V, int want_logits) {
  SeqState& s = st[blockIdx.x];
  const int j = threadIdx.x;
  if (j < K) {
    int t = over ? over[blockIdx.x * K + j] : s.props[j];
    if (t < 0 || t >= V) {
      atomicOr(&s.err, ERR_TOKEN);
      t = 0;
    }
    s.vtok[j + 1] = t;
  }
  if (j == 0) {
    s.vtok[0] = s.pending;
    s.want_logits = want_logits;
  }
}

// ---------------------------------------------------------------------------
// Row plan + embedding gather.  grid (R, B), 1024 threads.
// Verify: rows at slots seq_len .. seq_len+K, tokens vtok.
// Context (cross-attention conditioning, after a commit): rows at the
// verify's committed slots, taking the slots' fused features instead of
// embeddings.
// Draft: rows at slots draft_len .. seq_len+dstep (catch-up), tokens from the
// committed history up to seq_len and the draft's own proposals after it.
// Writes the residual stream x, xg = bf16(x * g) with the first layer's
// attention-norm gain, per-16-column sums of x^2 (the next GEMV applies 1/rms;
// see k_gemv), and each row's (cos, sin) of every rotary pair at its slot:
// target angle theta_d * p_{a(d)}(slot) (Eq. mrope-phase), draft theta_d * slot
// (Eq. flatrope-proj), gathered from the host-built table.
// ---------------------------------------------------------------------------
struct EmbedArgs {
  SeqState* st;
  const int32_t* hist;   // [B][cap]
  const bf16_t* E;       // [V][H]
  const bf16_t* g;       // first layer's attention-norm gain
  float* x;              // [Mpad][H]
  bf16_t* xg;            // [Mpad][H]
  float* ss;             // [H/16][Mpad]
  float2* rcs;           // [Mpad][D/2] (cos, sin) of each row's rotary pairs
  const int32_t* pos3;   // [B][3][cap]
  const float2* cs;      // [cap][D/2]
  const int8_t* axis;    // [D/2]
  int H, R, cap, mode, mpad, D, flat;
  int V;                 // vocabulary size: a token outside [0, V) is reported and read as 0
  int mask;              // block pass: input token of the MASK rows
  bf16_t* cat2;          // conditioned draft: [Mpad][2H] rows [embedding; feature of the previous slot], or null
  const bf16_t* feat;    // [B][cap][H] fused target features
};

__global__ __launch_bounds__(1024) void k_embed(EmbedArgs p) {
  extern __shared__ float sq[];   // [H]
  const int j = blockIdx.x, b = blockIdx.y;
  const SeqState& s = p.st[b];
  int base, count, tok = 0, causal = -1;
  if (p.mode == PASS_VERIFY) {
    base = s.seq_len;
    count = s.finished ? 0 : p.R;
    tok = s.vtok[j];
  } else if (p.mode == PASS_CATCHUP) {
    // committed tokens the draft has not consumed with their own inputs
    base = s.draft_len;
    count = s.finished ? 0 : s.seq_len - base;
    if (count < 0 || count > p.R) {
      if (!s.finished && j == 0 && threadIdx.x == 0) atomicOr(&p.st[b].err, ERR_STATE);
      count = 0;
    }
    if (j < count) tok = p.hist[(size_t)b * p.cap + base + j];
  } else if (p.mode == PASS_BLOCK) {
    // [pending, MASK x (R-1)] at slots seq_len .. seq_len + R - 1
    base = s.seq_len;
    count = s.finished ? 0 : p.R;
    causal = 1;
    tok = j == 0 ? p.hist[(size_t)b * p.cap + base] : p.mask;
  } else if (p.mode == PASS_CTX) {
    // cross-attention context rows: the fused features of the slots whose
    // inputs the last commit took from its verify (rows 0 .. n_commit-1 at
    // the verify's slots)
    base = s.base;
    count = s.count > 0 ? s.n_commit : 0;
  } else {
    base = s.draft_len;
    const int last = s.seq_len + s.dstep;
    count = s.finished ? 0 : last - base + 1;
    if (count < 1 || count > p.R) {
      if (!s.finished && j == 0 && threadIdx.x == 0) atomicOr(&p.st[b].err, ERR_STATE);
      count = 0;
    }
    const int slot = base + j;
    if (j < count) tok = slot <= s.seq_len ? p.hist[(size_t)b * p.cap + slot] : s.props[slot - s.seq_len - 1];
  }
  __syncthreads();
  if (j == 0 && threadIdx.x == 0) {
    p.st[b].base = base;
    p.st[b].count = count;
    p.st[b].causal = causal < 0 ? count : causal;
  }
  const size_t r = (size_t)b * p.R + j;
  const bool live = j < count;
  if (tok < 0 || tok >= p.V) {   // never from a valid pass; guards the gather below
    if (live && threadIdx.x == 0) atomicOr(&p.st[b].err, ERR_TOKEN);
    tok = 0;
  }
  const bf16_t* er = p.mode == PASS_CTX ? p.feat + ((size_t)b * p.cap + (live ? base + j : 0)) * p.H
                                        : p.E + (size_t)tok * p.H;
  for (int n = threadIdx.x; n < p.H; n += blockDim.x) {
    const float v = live ? bf2f(er[n]) : 0.f;
    p.x[r * p.H + n] = v;
    p.xg[r * p.H + n] = f2bf(v * bf2f(p.g[n]));
    sq[n] = v * v;
  }
  if (p.cat2) {
    // the input projection's operand: [embedding; feature of slot - 1], the
    // feature zero where the target has not verified that slot
    const int prev = base + j - 1;
    const bool hasf = live && prev >= s.prefix_len && prev < s.seq_len;
    const bf16_t* fr = p.feat + ((size_t)b * p.cap + (hasf ? prev : 0)) * p.H;
    bf16_t* cr = p.cat2 + r * 2 * p.H;
    for (int n = threadIdx.x; n < p.H; n += blockDim.x) {
      cr[n] = live ? er[n] : (bf16_t)0;
      cr[p.H + n] = hasf ? fr[n] : (bf16_t)0;
    }
  }
  if (live && threadIdx.x < p.D / 2) {
    const int slot = base + j, d = threadIdx.x;
    const int pos = p.flat ? slot : p.pos3[((size_t)b * 3 + p.axis[d]) * p.cap + slot];
    p.rcs[r * (p.D / 2) + d] = p.cs[(size_t)pos * (p.D / 2) + d];
  }
  __syncthreads();
  for (int t = threadIdx.x; t < p.H / kTile; t += blockDim.x) {
    float v = 0.f;
    for (int c = 0; c < kTile; ++c) v += sq[t * kTile + c];
    p.ss[(size_t)t * p.mpad + r] = v;
  }
}

// ---------------------------------------------------------------------------
// Thin-M weight-streaming GEMV on MFMA:  y[m][n] = sum_k x[m][k] * W[n][k],
// with the consumer's step fused into the epilogue.
//
// A workgroup of NW waves owns TT tiles of 16 weight rows and a k-range of
// 32-wide steps; wave w streams a contiguous chunk of at most SMAX steps of
// every tile.  Row-major weights: for one step, lane l reads
// W[row (l&15)][8*(l>>4) .. +8] (16 bytes).  All of a wave's weight loads are
// issued first; the workgroup then stages its live x rows for the k-range in
// LDS with coalesced loads, so each x fragment is fetched from L2 once per
// workgroup and feeds TT MFMAs.  v_mfma_f32_16x16x32_bf16 takes the weight
// fragment as A and x^T as B (lane l: x[m = l&15][same 8 k]); lane l ends with
// y[m = l&15][n0 + 4*(l>>4) + i].  The NW per-wave partial tiles are summed
// through LDS in a fixed order (deterministic), then the epilogue runs on
// complete outputs.  Which rows are live (row m is row m % rps of sequence
// m / rps, live while below that sequence's row count) is read through the
// scalar cache, which does not wait behind the weight stream.
//
// RMSNorm: producers store xg = bf16(x * g) and per-16-column sums of x^2;
// consumers of a normalised input scale y by 1/rms(x), a per-row scalar
// (RMSNorm(x) g W^T = (x g) W^T / rms(x)).
// ---------------------------------------------------------------------------
template <int MB, int NW, int SMAX, int TT, int EPI>
__global__ __launch_bounds__(NW * 64) void k_gemv(GemvArgs a) {
  extern __shared__ __align__(16) unsigned char lds[];
  __shared__ float inv_rms[MB * 16];
  const int tg = blockIdx.x, split = blockIdx.y;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int Kd = a.Kd;
  const int kq = 8 * (lane >> 4);
  const int T = (Kd + 31) >> 5;
  const int s0 = (int)((long long)split * T / a.splits);
  const int s1 = (int)((long long)(split + 1) * T / a.splits);
  const int chunk = (s1 - s0 + NW - 1) / NW;
  const int w0 = s0 + wave * chunk;
  const int w1 = min(w0 + chunk, s1);
  constexpr bool kNorm = EPI == EPI_ROPE || EPI == EPI_SWIGLU || EPI == EPI_ARGMAX;

  int tile[TT];
#pragma unroll
  for (int tt = 0; tt < TT; ++tt) tile[tt] = tg * TT + tt;

  // 1. weight fragments -> registers
  u32x4 wv[TT][SMAX];
#pragma unroll
  for (int tt = 0; tt < TT; ++tt) {
    const int n0 = tile[tt] * kTile;
    int sg = 0;
#pragma unroll
    for (int i = 1; i < 3; ++i)
      if (i < a.nseg && n0 >= a.row0[i]) sg = i;
    const bf16_t* wp = a.w[sg] + (size_t)(n0 - a.row0[sg] + (lane & 15)) * Kd + kq;
    if constexpr (EPI == EPI_SWIGLU) {
      // half-tile: rows 0-7 are gate rows n0/2 .. +8, rows 8-15 the matching up rows
      const int r = lane & 15;
      wp = (r < 8 ? a.w[0] + (size_t)(n0 / 2 + r) * Kd : a.w[1] + (size_t)(n0 / 2 + r - 8) * Kd) + kq;
    }
#pragma unroll
    for (int i = 0; i < SMAX; ++i) {
      const int k = (w0 + i) << 5;
      wv[tt][i] = (w0 + i < w1 && k + kq < Kd) ? ld16_nt(wp + k) : u32x4{0, 0, 0, 0};
    }
  }

  // 2. live rows (scalar cache)
  uint64_t live = 0;
  {
    const int nseq = (a.M + a.rps - 1) / a.rps;
    for (int b = 0; b < nseq; ++b) {
      const int n = min(a.st[b].count, a.rps);
      if (n > 0) live |= ((1ull << n) - 1ull) << (b * a.rps);
    }
  }

  // 3. live x rows, steps [s0, s1) -> LDS.  Rows are padded by one 16-byte
  // chunk so that the 16 rows one MFMA reads at the same k fall in different
  // LDS banks.
  const int per_row = (s1 - s0) * 4;              // 16-byte chunks per row
  const int xstride = per_row + 1;
  u32x4* xs = reinterpret_cast<u32x4*>(lds);
  for (int c = threadIdx.x; per_row > 0 && c < a.M * per_row; c += NW * 64) {
    const int m = c / per_row, q = c - m * per_row;
    if (!((live >> m) & 1)) continue;
    const int k = s0 * 32 + q * 8;
    xs[m * xstride + q] = k < Kd ? ld16(a.x + (size_t)m * a.ldx + k) : u32x4{0, 0, 0, 0};
  }
  if constexpr (kNorm) {
    // 1 / rms of each row from the per-16-column sums of squares (fixed order)
    for (int m = wave; m < MB * 16; m += NW) {
      float v = 0.f;
      if ((live >> m) & 1)
        for (int t = lane; t < a.H / kTile; t += 64) v += a.ss_in[(size_t)t * a.mpad + m];
      for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
      if (lane == 0) inv_rms[m] = rsqrtf(v / a.H + a.eps);
    }
  }
  __syncthreads();

  // 4. MFMAs
  f32x4 acc[TT][MB];
#pragma unroll
  for (int tt = 0; tt < TT; ++tt)
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) acc[tt][mb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int i = 0; i < SMAX; ++i) {
    if (w0 + i < w1) {
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        const int m = mb * 16 + (lane & 15);
        const u32x4 xv = ((live >> m) & 1) ? xs[m * xstride + (w0 + i - s0) * 4 + (lane >> 4)] : u32x4{0, 0, 0, 0};
#pragma unroll
        for (int tt = 0; tt < TT; ++tt) acc[tt][mb] = mfma16x16x32(wv[tt][i], xv, acc[tt][mb]);
      }
    }
  }
  __syncthreads();   // x no longer needed: reuse LDS

  // 5. sum the NW wave partials: y[tt][m][c] (c = column inside the tile)
  f32x4* red = reinterpret_cast<f32x4*>(lds);                                        // [NW][TT][MB][64]
  float* y = reinterpret_cast<float*>(lds + (size_t)NW * TT * MB * 64 * 16);         // [TT][MB*16][17]
#pragma unroll
  for (int tt = 0; tt < TT; ++tt)
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) red[((wave * TT + tt) * MB + mb) * 64 + lane] = acc[tt][mb];
  __syncthreads();
  for (int t = threadIdx.x; t < TT * MB * 256; t += NW * 64) {
    const int tt = t / (MB * 256), r = t % (MB * 256);
    const int mb = r >> 8, L = (r & 255) >> 2, i = r & 3;
    float v = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) v += red[((w * TT + tt) * MB + mb) * 64 + L][i];
    const int m = mb * 16 + (L & 15);
    y[(tt * MB * 16 + m) * 17 + 4 * (L >> 4) + i] = kNorm ? v * inv_rms[m] : v;
  }
  __syncthreads();

  // 6. epilogue on complete 16-column tiles
  const int nrow = MB * 16;
  if constexpr (EPI == EPI_STORE) {
    for (int t = threadIdx.x; t < TT * nrow * 16; t += NW * 64) {
      const int tt = t / (nrow * 16), m = (t / 16) % nrow, c = t & 15;
      if (m < a.M) a.out[((size_t)split * a.M + m) * a.N + tile[tt] * 16 + c] = y[(tt * nrow + m) * 17 + c];
    }
  } else if constexpr (EPI == EPI_ROPE) {
    // one thread per (row, rotary pair); TT == 1
    const int t = threadIdx.x, m = t >> 3, pr = t & 7;
    if (t < nrow * 8 && m < a.M && ((live >> m) & 1)) {
      const int b = m / a.rps, j = m - b * a.rps;
      const int slot = a.st[b].base + j;
      const int n0 = tile[0] * kTile;
      const int head = n0 / a.D, d = ((n0 % a.D) >> 1) + pr;
      const float e = y[m * 17 + 2 * pr], o = y[m * 17 + 2 * pr + 1];
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
    // TT == 1; rows whose sequence is idle keep their stream untouched
    const int t = threadIdx.x, m = t >> 4, c = t & 15;
    const int n = tile[0] * kTile + c;
    float xn = 0.f;
    if (t < nrow * 16 && m < a.M) {
      xn = a.x32[(size_t)m * a.N + n];
      if ((live >> m) & 1) {
        xn += y[m * 17 + c];
        a.x32[(size_t)m * a.N + n] = xn;
      }
      a.xg[(size_t)m * a.N + n] = f2bf(xn * bf2f(a.gain[n]));
    }
    __syncthreads();
    if (t < nrow * 16) y[m * 17 + c] = xn * xn;
    __syncthreads();
    if (threadIdx.x < nrow) {
      float v = 0.f;
      for (int c2 = 0; c2 < 16; ++c2) v += y[threadIdx.x * 17 + c2];
      a.ss_out[(size_t)tile[0] * a.mpad + threadIdx.x] = v;
    }
  } else if constexpr (EPI == EPI_SWIGLU) {
    // TT == 1: columns 0-7 gate, 8-15 up of output features n0/2 .. n0/2 + 8
    const int F = a.N / 2;
    const int n0 = tile[0] * kTile;
    const int t = threadIdx.x, m = t >> 3, c = t & 7;
    if (t < nrow * 8 && m < a.M) {
      const float g = y[m * 17 + c];
      const float up = y[m * 17 + 8 + c];
      a.u[(size_t)m * F + n0 / 2 + c] = f2bf(g / (1.f + expf(-g)) * up);
    }
  } else {   // EPI_ARGMAX, TT tiles of the vocabulary
    for (int t = threadIdx.x; t < TT * nrow * 16; t += NW * 64) {
      const int tt = t / (nrow * 16), m = (t / 16) % nrow, c = t & 15;
      if (a.allow_logits && m < a.M && a.st[m / a.rps].want_logits)
        a.logits[(size_t)m * a.N + tile[tt] * 16 + c] = f2bf(y[(tt * nrow + m) * 17 + c]);
    }
    for (int t = threadIdx.x; t < TT * nrow; t += NW * 64) {
      const int tt = t / nrow, m = t % nrow;
      if (m >= a.M) continue;
      float best = -INFINITY;
      int bi = tile[tt] * 16;
      bool nan = false;
      for (int c = 0; c < 16; ++c) {
        float v = y[(tt * nrow + m) * 17 + c];
        if (v != v) {
          nan = true;
          v = -INFINITY;
        }
        if (v > best) {
          best = v;
          bi = tile[tt] * 16 + c;
        }
      }
      a.amax_v[(size_t)tile[tt] * a.mpad + m] = best;
      a.amax_i[(size_t)tile[tt] * a.mpad + m] = bi;
      if (nan) atomicOr(const_cast<int32_t*>(&a.st[m / a.rps].err), ERR_NUMERIC);
    }
  }
}

// ---------------------------------------------------------------------------
// Persistent variant for the large projections (gate/up, down, LM head).
// gridDim.x workgroups are split into S groups, one per k-split; workgroup g
// of group s stages x for split s's k-range in LDS once and then streams
// tiles g, g + G_s, g + 2 G_s, ... (G_s workgroups per group), keeping the
// next tile's weight fragments in flight while the current tile is reduced
// and written.  Staging x once per workgroup instead of once per tile removes
// most of the activation traffic at several rows per pass.
// ---------------------------------------------------------------------------
template <int MB, int NW, int SMAX, int EPI>
__global__ __launch_bounds__(NW * 64) void k_gemv_p(GemvArgs a) {
  static_assert(EPI == EPI_STORE || EPI == EPI_SWIGLU || EPI == EPI_ARGMAX, "persistent epilogues");
  extern __shared__ __align__(16) unsigned char lds[];
  __shared__ float inv_rms[MB * 16];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int groups = a.splits;
  const int gsize = gridDim.x / groups;
  const int split = blockIdx.x / gsize, g = blockIdx.x % gsize;
  const int ntiles = a.N / kTile;
  const int Kd = a.Kd;
  const int kq = 8 * (lane >> 4);
  const int T = (Kd + 31) >> 5;
  const int s0 = (int)((long long)split * T / a.splits);
  const int s1 = (int)((long long)(split + 1) * T / a.splits);
  const int chunk = (s1 - s0 + NW - 1) / NW;
  const int w0 = s0 + wave * chunk;
  const int w1 = min(w0 + chunk, s1);
  constexpr bool kNorm = EPI == EPI_SWIGLU || EPI == EPI_ARGMAX;
  const int per_row = (s1 - s0) * 4, xstride = per_row + 1;
  u32x4* xs = reinterpret_cast<u32x4*>(lds);
  f32x4* red = reinterpret_cast<f32x4*>(lds + (size_t)a.M * xstride * 16);                 // [NW][MB][64]
  float* y = reinterpret_cast<float*>(lds + (size_t)a.M * xstride * 16 + (size_t)NW * MB * 64 * 16);   // [MB*16][17]

  auto load_tile = [&](int tile, u32x4 (&wv)[SMAX]) {
    const int n0 = tile * kTile;
    const bf16_t* wp;
    if constexpr (EPI == EPI_SWIGLU) {
      const int r = lane & 15;
      wp = (r < 8 ? a.w[0] + (size_t)(n0 / 2 + r) * Kd : a.w[1] + (size_t)(n0 / 2 + r - 8) * Kd) + kq;
    } else {
      wp = a.w[0] + (size_t)(n0 + (lane & 15)) * Kd + kq;
    }
#pragma unroll
    for (int i = 0; i < SMAX; ++i) {
      const int k = (w0 + i) << 5;
      wv[i] = (w0 + i < w1 && k + kq < Kd) ? ld16_nt(wp + k) : u32x4{0, 0, 0, 0};
    }
  };

  u32x4 wa[SMAX], wb[SMAX];
  int t = g;
  if (t < ntiles) load_tile(t, wa);

  uint64_t live = 0;
  {
    const int nseq = (a.M + a.rps - 1) / a.rps;
    for (int b = 0; b < nseq; ++b) {
      const int n = min(a.st[b].count, a.rps);
      if (n > 0) live |= ((1ull << n) - 1ull) << (b * a.rps);
    }
  }
  for (int c = threadIdx.x; per_row > 0 && c < a.M * per_row; c += NW * 64) {
    const int m = c / per_row, q = c - m * per_row;
    if (!((live >> m) & 1)) continue;
    const int k = s0 * 32 + q * 8;
    xs[m * xstride + q] = k < Kd ? ld16(a.x + (size_t)m * a.ldx + k) : u32x4{0, 0, 0, 0};
  }
  if constexpr (kNorm) {
    for (int m = wave; m < MB * 16; m += NW) {
      float v = 0.f;
      if ((live >> m) & 1)
        for (int tt = lane; tt < a.H / kTile; tt += 64) v += a.ss_in[(size_t)tt * a.mpad + m];
      for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
      if (lane == 0) inv_rms[m] = rsqrtf(v / a.H + a.eps);
    }
  }
  __syncthreads();

  const int nrow = MB * 16;
  auto do_tile = [&](int tile, const u32x4 (&wv)[SMAX]) {
    f32x4 acc[MB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) acc[mb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < SMAX; ++i) {
      if (w0 + i < w1) {
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
          const int m = mb * 16 + (lane & 15);
          const u32x4 xv = ((live >> m) & 1) ? xs[m * xstride + (w0 + i - s0) * 4 + (lane >> 4)] : u32x4{0, 0, 0, 0};
          acc[mb] = mfma16x16x32(wv[i], xv, acc[mb]);
        }
      }
    }
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) red[(wave * MB + mb) * 64 + lane] = acc[mb];
    __syncthreads();
    for (int q = threadIdx.x; q < MB * 256; q += NW * 64) {
      const int mb = q >> 8, L = (q & 255) >> 2, i = q & 3;
      float v = 0.f;
#pragma unroll
      for (int w = 0; w < NW; ++w) v += red[(w * MB + mb) * 64 + L][i];
      const int m = mb * 16 + (L & 15);
      y[m * 17 + 4 * (L >> 4) + i] = kNorm ? v * inv_rms[m] : v;
    }
    __syncthreads();
    const int n0 = tile * kTile;
    if constexpr (EPI == EPI_STORE) {
      for (int q = threadIdx.x; q < nrow * 16; q += NW * 64) {
        const int m = q >> 4, c = q & 15;
        if (m < a.M) a.out[((size_t)split * a.M + m) * a.N + n0 + c] = y[m * 17 + c];
      }
    } else if constexpr (EPI == EPI_SWIGLU) {
      const int F = a.N / 2;
      const int q = threadIdx.x, m = q >> 3, c = q & 7;
      if (q < nrow * 8 && m < a.M) {
        const float gt = y[m * 17 + c], up = y[m * 17 + 8 + c];
        a.u[(size_t)m * F + n0 / 2 + c] = f2bf(gt / (1.f + expf(-gt)) * up);
      }
    } else {
      for (int q = threadIdx.x; q < nrow * 16; q += NW * 64) {
        const int m = q >> 4, c = q & 15;
        if (a.allow_logits && m < a.M && a.st[m / a.rps].want_logits)
          a.logits[(size_t)m * a.N + n0 + c] = f2bf(y[m * 17 + c]);
      }
      if (threadIdx.x < nrow && threadIdx.x < a.M) {
        const int m = threadIdx.x;
        float best = -INFINITY;
        int bi = n0;
        bool nan = false;
        for (int c = 0; c < 16; ++c) {
          float v = y[m * 17 + c];
          if (v != v) {
            nan = true;
            v = -INFINITY;
          }
          if (v > best) {
            best = v;
            bi = n0 + c;
          }
        }
        a.amax_v[(size_t)tile * a.mpad + m] = best;
        a.amax_i[(size_t)tile * a.mpad + m] = bi;
        if (nan) atomicOr(const_cast<int32_t*>(&a.st[m / a.rps].err), ERR_NUMERIC);
      }
    }
  };
  // workgroup-uniform loop: every thread reaches every barrier; ends after
  // the last tile of this workgroup's stride
  while (t < ntiles) {
    const int t2 = t + gsize;
    if (t2 < ntiles) load_tile(t2, wb);
    do_tile(t, wa);
    if (t2 >= ntiles) break;
    const int t3 = t2 + gsize;
    if (t3 < ntiles) load_tile(t3, wa);
    do_tile(t2, wb);
    t = t3;
  }
}

// Dynamic LDS of a persistent launch: x rows + per-wave tiles + the summed tile.
size_t gemv_p_lds_bytes(int M, int span_steps) {
  const int MB = (M + 15) / 16;
  return (size_t)M * (span_steps * 64 + 16) + (size_t)kGemvWaves * MB * 64 * 16 + (size_t)MB * 16 * 17 * 4;
}

size_t gemv_lds_bytes(int TT, int M, int span_steps) {
  const int MB = (M + 15) / 16;
  const size_t x = (size_t)M * (span_steps * 64 + 16);
  const size_t red = (size_t)kGemvWaves * TT * MB * 64 * 16 + (size_t)TT * MB * 16 * 17 * 4;
  return std::max(x, red);
}

// ---------------------------------------------------------------------------
// Down-projection finish: x += sum of the k-split partials (residual), then
// xg = bf16(x * g_next) and per-16-column sums of x^2 for the next norm.
// select_last: only each sequence's last live row, stored as row b (the
// draft proposes from it).  grid (H/256, M), one column of one row per thread.
// ---------------------------------------------------------------------------
struct FinishArgs {
  const SeqState* st;
  const float* part;     // [S][M][H]
  int S, M, rps, H, mpad, select_last;
  float* x;              // [M][H]
  const bf16_t* gain;
  bf16_t* xg;
  float* ss;             // [H/16][mpad]
  bf16_t* xgp;           // null, or a step-major copy of xg: [H/32][M][32] (all rows; not with select_last)
};

__global__ __launch_bounds__(256) void k_down_finish(FinishArgs p) {
  const int m = blockIdx.y, n = blockIdx.x * 256 + threadIdx.x;
  if (n >= p.H) return;                            // H % 16 == 0: whole 16-lane groups exit together
  const int b = m / p.rps, j = m - b * p.rps;
  const int count = p.st[b].count;
  float* xp = p.x + (size_t)m * p.H + n;
  float x = *xp;
  if (j < count) {
    float v = 0.f;
    for (int sp = 0; sp < p.S; ++sp) v += p.part[((size_t)sp * p.M + m) * p.H + n];
    x += v;
    *xp = x;
  }
  float sq = x * x;
  for (int o = 1; o < 16; o <<= 1) sq += __shfl_xor(sq, o);
  const int out = p.select_last ? b : m;
  if (p.select_last && j != count - 1) return;
  const bf16_t xb = f2bf(x * bf2f(p.gain[n]));
  p.xg[(size_t)out * p.H + n] = xb;
  if (p.xgp && !p.select_last) p.xgp[((size_t)(n >> 5) * p.M + m) * 32 + (n & 31)] = xb;
  if ((n & 15) == 0) p.ss[(size_t)(n >> 4) * p.mpad + out] = sq;
}

// Finish of a k-split q/k/v GEMM: per live row m and column pair (2i, 2i+1),
// the split partials are added, scaled by the row's 1/rms (the attention
// RMSNorm, whose gain is already in the bf16 input), rotated by the row's
// (cos, sin) when the pair belongs to a q or k head (Sec. 3.3, Eq. rope-3d),
// and stored as the fused rotary epilogue stores them: q rows, key pages and
// transposed value pages.  grid (ceil(N/2 / 256), M), 256 threads.
struct QkvFinishArgs {
  const SeqState* st;
  const float* part;     // [S][M][N]
  int S, M, N, rps, mpad, H;
  float eps;
  const float* ss;       // [H/16][mpad] sums of x^2 of the input rows
  const float2* rcs;     // [Mpad][D/2]
  const int32_t* pt;     // [B][pps]
  int nq, nkv, D, pps;
  bf16_t* q;             // [M][nq*D]
  bf16_t *kc, *vt;       // layer bases of the paged key / value pools
};

__global__ __launch_bounds__(256) void k_qkv_finish(QkvFinishArgs a) {
  __shared__ float inv_rms;
  const int m = blockIdx.y;
  const int b = m / a.rps, j = m - b * a.rps;
  if (j >= a.st[b].count) return;                 // uniform over the workgroup
  if (threadIdx.x < 64) {
    float v = 0.f;
    for (int t = threadIdx.x; t < a.H / kTile; t += 64) v += a.ss[(size_t)t * a.mpad + m];
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
    if (threadIdx.x == 0) inv_rms = rsqrtf(v / a.H + a.eps);
  }
  __syncthreads();
  const int pr = blockIdx.x * 256 + threadIdx.x;
  if (pr >= a.N / 2) return;
  float e = 0.f, o = 0.f;
  for (int sp = 0; sp < a.S; ++sp) {
    const float2 v = *reinterpret_cast<const float2*>(a.part + ((size_t)sp * a.M + m) * a.N + 2 * pr);
    e += v.x;
    o += v.y;
  }
  e *= inv_rms;
  o *= inv_rms;
  const int n = 2 * pr, head = n / a.D, d = (n % a.D) >> 1;
  const int slot = a.st[b].base + j;
  if (head < a.nq + a.nkv) {
    const float2 cs = a.rcs[(size_t)m * (a.D / 2) + d];
    const float re = e * cs.x - o * cs.y, ro = e * cs.y + o * cs.x;
    if (head < a.nq) {
      *reinterpret_cast<uint32_t*>(a.q + ((size_t)m * a.nq + head) * a.D + 2 * d) = pack2(re, ro);
    } else {
      const size_t pg = (size_t)a.pt[b * a.pps + slot / kAttnChunk] * a.nkv + (head - a.nq);
      *reinterpret_cast<uint32_t*>(a.kc + (pg * kAttnChunk + slot % kAttnChunk) * a.D + 2 * d) = pack2(re, ro);
    }
  } else {
    const size_t pg = (size_t)a.pt[b * a.pps + slot / kAttnChunk] * a.nkv + (head - a.nq - a.nkv);
    bf16_t* vp = a.vt + (pg * a.D + 2 * d) * kAttnChunk + slot % kAttnChunk;
    vp[0] = f2bf(e);
    vp[kAttnChunk] = f2bf(o);
  }
}

// ---------------------------------------------------------------------------
// Split-KV causal grouped-query attention on MFMA.
//
// grid (splits, kv_heads * row_blocks, B); a workgroup owns one kv head, up to
// 64 query rows (row = j*G + g: new row j, q head kvh*G + g) and the key range
// [split*chunk, (split+1)*chunk) clipped to the keys that exist: one cache
// page (chunk = kAttnChunk).  Wave w owns query rows 16w..16w+15.
//
// Scores are computed transposed, S^T = K Q^T, so that lane l owns query row
// l&15: A = K tile (lane: key kb + (l&15), 8 dims), B = Q^T (lane: row l&15,
// same 8 dims) -> lane l holds scores of keys kb + 4*(l>>4) + i, i = 0..3.
// Two 16-key tiles give lane l the 8 keys {4g..4g+3, 16+4g..16+4g+3}
// (g = l>>4) of its row, which is exactly a B operand P^T for O^T = V^T P^T
// when the 32 k-slots are mapped to keys in that order; the A operand V^T is
// read from the transposed value cache as two 8-byte loads per lane.  The
// softmax statistics of the chunk are per lane (its row); the row max crosses
// the four lane groups with two xor-shuffles.  Partial outputs are stored
// unnormalised in bf16, with the chunk's max and sum in fp32, for the combine.
//
// The readout variant (RO) also writes, per (row, q head, split), the sums of
// 2^(s - m) over the split's visible keys of each token class (visual,
// trajectory/text, generated; s = score in log2 units, m = the split's max)
// and E = sum over trajectory/text keys of 2^(s - m) (s - m): the terms from
// which the combine forms the attention mass per class and the entropy within
// trajectory/text (Sec. 4.2, Table attn-budget).
// ---------------------------------------------------------------------------

struct AttnArgs {
  const SeqState* st;
  const bf16_t* q;       // [Mpad][nq][D]
  const bf16_t* kc;      // layer base of the key pool [pages][nkv][kAttnChunk][D]
  const bf16_t* vt;      // layer base of the value pool [pages][nkv][D][kAttnChunk]
  const int32_t* pt;     // [B][pps] page tables
  bf16_t* op;            // [splits][B][nq][R][D] unnormalised partial outputs (bf16)
  float* mp;             // [splits][B][nq][R]
  float* lp;
  int nq, nkv, G, R, B, pps, chunk, row_blocks;
  float scale_log2;      // log2(e) / sqrt(D)
  const int8_t* cls;     // readout: [B][cap] class of every slot (0 visual, 1 trajectory/text, 2 generated)
  float* rp;             // readout: [splits][B][nq][R][4] class sums and trajectory E term
  int cap;
  int cross;             // cross-attention context: row j sees the slots below min(base + j, seq_len)
  int ppw;               // k_attn_pages: pages per split (workgroup)
};

// LDS tiles of a page: keys [chunk][D + kAttnPadK] and values transposed
// [D][chunk + kAttnPadV].  A 16-byte LDS read is served eight lanes at a
// time, in the groups lanes 0-3 with 20-23, 4-7 with 16-19, 8-11 with 28-31
// and 12-15 with 24-27 (the same in the upper half).  An MFMA operand read
// takes row (lane & 15) and 16-byte column group (lane >> 4); with rows 32
// bytes past a multiple of 128 bytes, each group's eight reads fall in
// distinct banks.  (Rows 16 bytes past: four times the bank-conflict cycles
// in the multi-page kernel.)
constexpr int kAttnPadK = 16, kAttnPadV = 16;

// Store the 8 values (keys slot .. slot + 7 of value row d, as loaded from the
// page; keys at or past k1 as zeros) into the value tile.  Within each 32-key
// half of a row, key 16 hi + 4 g + e sits at 8 g + 4 hi + e: the eight keys a
// lane of group g contracts in that half (4 g + e and 16 + 4 g + e) are then
// one 16-byte read.  v8 = (slot - k0) / 8.
__device__ __forceinline__ void attn_stage_values(bf16_t* vrow, int v8, int slot, int k1, u32x4 v) {
  if (slot >= k1) {
    v = u32x4{0, 0, 0, 0};
  } else if (slot + 8 > k1) {                       // ragged end of the valid keys
    uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int e = 0; e < 8; ++e)
      if (slot + e >= k1) w[e >> 1] &= (e & 1) ? 0x0000FFFFu : 0xFFFF0000u;
    v = u32x4{w[0], w[1], w[2], w[3]};
  }
  // keys 8 v8 .. 8 v8 + 3 are group 2 (v8 & 1) of half-row (v8 >> 1) & 1, the
  // next four group 2 (v8 & 1) + 1
  bf16_t* vd = vrow + 32 * (v8 >> 2) + 16 * (v8 & 1) + 4 * ((v8 >> 1) & 1);
  *reinterpret_cast<u32x2*>(vd) = u32x2{v.x, v.y};
  *reinterpret_cast<u32x2*>(vd + 8) = u32x2{v.z, v.w};
}

template <int D, bool RO, int NW>
__device__ __forceinline__ void attn_partials(const AttnArgs& a, unsigned char* lds) {
  constexpr int NT = NW * 64;   // threads: NW waves of 16 query rows each
  const int split = blockIdx.x;
  const int kvh = blockIdx.y / a.row_blocks, rb = blockIdx.y % a.row_blocks;
  const int b = blockIdx.z;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int g4 = lane >> 4;
  // The page of this split is read together with the sequence state (it
  // depends on the split only; table entries past a sequence's pages name
  // page 0), so the key and value loads wait for one round trip, not two.
  const int page = a.pt[b * a.pps + split];
  const SeqState& s = a.st[b];
  const int count = s.count, base = s.base, causal = s.causal, seq_len = s.seq_len;
  asm volatile("" ::"s"(page), "s"(count), "s"(base), "s"(causal), "s"(seq_len));   // all loads issued before any is awaited
  const int rows = count * a.G;
  const int wrow0 = rb * (16 * NW) + wave * 16;
  const int qr = wrow0 + (lane & 15);
  const bool rvalid = qr < rows;
  const int j = rvalid ? qr / a.G : 0;
  const int hq = kvh * a.G + (rvalid ? qr % a.G : 0);
  // keys [0, vis_end) of row j: causal (rows past `causal` see the whole
  // pass), or, for a cross-attention context, the context slots before the
  // row's own slot that exist (below seq_len)
  const int kv_end = a.cross ? min(base + count - 1, seq_len) : base + count;
  const int k0 = split * a.chunk;
  const int k1 = min(k0 + a.chunk, kv_end);
  const int vis_end = a.cross ? min(base + j, seq_len) : base + (j < causal ? j + 1 : count);
  const size_t oi = (((size_t)split * a.B + b) * a.nq + hq) * a.R + j;

  if (k0 >= k1) {                                   // no keys in this split (workgroup-uniform)
    if (wrow0 >= rows) return;
    if (rvalid && g4 == 0) {
      a.mp[oi] = -INFINITY;
      a.lp[oi] = 0.f;
    }
    if (rvalid) {
      bf16_t* op = a.op + oi * D;
      for (int d = g4 * 4; d < D; d += 16) *reinterpret_cast<u32x2*>(op + d) = u32x2{0u, 0u};
      if (RO && g4 == 0) *reinterpret_cast<f32x4*>(a.rp + oi * 4) = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    return;
  }

  // This wave's query rows; issued first so their latency overlaps the
  // staging.  Loads are unconditional (an invalid lane reads row 0 of its
  // head): a lane's scores only reach its own row, and those of invalid rows
  // are masked below.
  u32x4 qf[D / 32];
  {
    const bf16_t* qp = a.q + ((size_t)(b * a.R + j) * a.nq + hq) * D + 8 * g4;
#pragma unroll
    for (int t = 0; t < D / 32; ++t) qf[t] = ld16(qp + 32 * t);
  }
  // readout: classes of this lane's 16 keys, 4 consecutive slots per word
  // (byte i of word h: slot k0 + 16 h + 4 g4 + i; k0 + 63 < cap)
  uint32_t cw[4] = {0u, 0u, 0u, 0u};
  if (RO) {
    const int8_t* cp = a.cls + (size_t)b * a.cap + k0 + 4 * g4;
#pragma unroll
    for (int h = 0; h < 4; ++h) cw[h] = *reinterpret_cast<const uint32_t*>(cp + 16 * h);
  }

  // Stage the chunk once for all waves.  The whole page is loaded (its slots
  // past k1 hold stale data): keys there only meet masked scores, values there
  // are stored as zeros.  Every load of the thread is issued before the first
  // LDS store so that their latencies overlap, and unconditionally so that no
  // branch splits them.
  const int kst = D + kAttnPadK, vst = a.chunk + kAttnPadV;
  bf16_t* Ks = reinterpret_cast<bf16_t*>(lds);
  bf16_t* Vs = Ks + (size_t)a.chunk * kst;
  {
    constexpr int PER_T = kAttnChunk * D / 8 / NT;    // 16-byte vectors per thread and operand
    static_assert(PER_T * NT * 8 == kAttnChunk * D, "the threads cover the page exactly");
    const size_t pg = (size_t)page * a.nkv + kvh;
    const bf16_t* Kb = a.kc + pg * kAttnChunk * D;
    const bf16_t* Vb = a.vt + pg * D * kAttnChunk;
    constexpr int per_row = kAttnChunk / 8;
    u32x4 kr[PER_T], vr[PER_T];
#pragma unroll
    for (int u = 0; u < PER_T; ++u) {
      const int i = threadIdx.x + NT * u;
      const int key = i / (D / 8), c8 = i % (D / 8);
      kr[u] = ld16(Kb + (size_t)key * D + 8 * c8);
      const int d = i / per_row, v8 = i % per_row;
      vr[u] = ld16(Vb + (size_t)d * kAttnChunk + 8 * v8);
    }
#pragma unroll
    for (int u = 0; u < PER_T; ++u) {
      const int i = threadIdx.x + NT * u;
      const int key = i / (D / 8), c8 = i % (D / 8);
      *reinterpret_cast<u32x4*>(Ks + (size_t)key * kst + 8 * c8) = kr[u];
      const int d = i / per_row, v8 = i % per_row;
      attn_stage_values(Vs + (size_t)d * vst, v8, k0 + 8 * v8, k1, vr[u]);
    }
  }
  __syncthreads();
  if (wrow0 >= rows) return;                        // wave-uniform; no barrier follows

  // The whole chunk (kAttnChunk = 64 keys) in one step: S^T = K Q^T for the
  // four 16-key groups (lanes own query rows; lane group g4 holds keys
  // 16h + 4 g4 + i), one softmax over the chunk in log2 units, then
  // O^T = V^T P^T over the two 32-key halves.  Within a half the key order of
  // the P^T operand (keys 4 g4 + i and 16 + 4 g4 + i) is the one the V^T
  // operand is read in, so the contraction is exact.
  static_assert(kAttnChunk == 4 * 16, "one step covers four 16-key groups");
  f32x4 sc[4];
#pragma unroll
  for (int h = 0; h < 4; ++h) {
    const bf16_t* kp = Ks + (size_t)(16 * h + (lane & 15)) * kst + 8 * g4;
    f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int t = 0; t < D / 32; ++t) acc = mfma16x16x32(*reinterpret_cast<const u32x4*>(kp + 32 * t), qf[t], acc);
    sc[h] = acc;
  }
  // V^T operands of both halves, read while the softmax runs
  u32x4 va[2][D / 16];
#pragma unroll
  for (int hb = 0; hb < 2; ++hb)
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt) {
      va[hb][dt] = *reinterpret_cast<const u32x4*>(Vs + (size_t)(16 * dt + (lane & 15)) * vst + 32 * hb + 8 * g4);
    }
  float p[16];
  float m_run = -INFINITY;
#pragma unroll
  for (int h = 0; h < 4; ++h)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int key = k0 + 16 * h + 4 * g4 + i;
      const bool ok = rvalid && key < k1 && key < vis_end;
      const float v = ok ? sc[h][i] * a.scale_log2 : -INFINITY;
      p[h * 4 + i] = v;
      m_run = fmaxf(m_run, v);
    }
  m_run = fmaxf(m_run, __shfl_xor(m_run, 16));
  m_run = fmaxf(m_run, __shfl_xor(m_run, 32));
  float l_run = 0.f;
  float rs[4] = {0.f, 0.f, 0.f, 0.f};   // readout: class sums, then the trajectory E term
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const float v = p[i];
    p[i] = (v == -INFINITY) ? 0.f : exp2f(v - m_run);
    l_run += p[i];
    if (RO) {
      const uint32_t cl = (cw[i >> 2] >> (8 * (i & 3))) & 0xffu;
      rs[0] += cl == 0 ? p[i] : 0.f;
      rs[1] += cl == 1 ? p[i] : 0.f;
      rs[2] += cl == 2 ? p[i] : 0.f;
      rs[3] += (cl == 1 && v != -INFINITY) ? p[i] * (v - m_run) : 0.f;
    }
  }
  f32x4 o[D / 16];
#pragma unroll
  for (int dt = 0; dt < D / 16; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int hb = 0; hb < 2; ++hb) {
    const float* ph = p + 8 * hb;
    const u32x4 pb = u32x4{pack2(ph[0], ph[1]), pack2(ph[2], ph[3]), pack2(ph[4], ph[5]), pack2(ph[6], ph[7])};
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt) o[dt] = mfma16x16x32(va[hb][dt], pb, o[dt]);
  }
  l_run += __shfl_xor(l_run, 16);
  l_run += __shfl_xor(l_run, 32);
  if (RO) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      rs[r] += __shfl_xor(rs[r], 16);
      rs[r] += __shfl_xor(rs[r], 32);
    }
    if (rvalid && g4 == 0) *reinterpret_cast<f32x4*>(a.rp + oi * 4) = f32x4{rs[0], rs[1], rs[2], rs[3]};
  }
  if (rvalid) {
    bf16_t* op = a.op + oi * D;
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt)
      *reinterpret_cast<u32x2*>(op + 16 * dt + 4 * g4) =
          u32x2{pack2(o[dt].x, o[dt].y), pack2(o[dt].z, o[dt].w)};
    if (g4 == 0) {
      a.mp[oi] = m_run;
      a.lp[oi] = l_run;
    }
  }
}

// The 8-wave form is held to 6 waves per SIMD (80 registers), three
// workgroups per CU, so that up to 768 of them run at once (at two per CU a
// pass of 65 pages x 8 kv heads left 8 workgroups for a second round).
template <int D, bool RO, int NW>
__global__ __launch_bounds__(NW * 64, (NW == 8 && !RO) ? 6 : 1) void k_attn(AttnArgs a) {
  extern __shared__ __align__(16) unsigned char lds[];
  attn_partials<D, RO, NW>(a, lds);
}

// The same split-KV attention with a.ppw consecutive pages per workgroup,
// for passes over many sequences (there are workgroups enough without one
// per page, and fewer splits mean fewer partial outputs written and merged).
// Pages are taken one at a time through the same LDS tile: the next page's
// keys and values are loaded while this one's scores and products run, and
// the running (max, sum, output) of each row is rescaled when the max grows.
// grid (groups of ppw pages, kv heads x row blocks, B), 256 threads.

template <int D>
__global__ __launch_bounds__(256, 3) void k_attn_pages(AttnArgs a) {
  extern __shared__ __align__(16) unsigned char lds[];
  const int grp = blockIdx.x;
  const int kvh = blockIdx.y / a.row_blocks, rb = blockIdx.y % a.row_blocks;
  const int b = blockIdx.z;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int g4 = lane >> 4;
  const SeqState& s = a.st[b];
  const int count = s.count, base = s.base, causal = s.causal, seq_len = s.seq_len;
  const int rows = count * a.G;
  const int wrow0 = rb * 64 + wave * 16;
  const int qr = wrow0 + (lane & 15);
  const bool rvalid = qr < rows;
  const int j = rvalid ? qr / a.G : 0;
  const int hq = kvh * a.G + (rvalid ? qr % a.G : 0);
  const int kv_end = a.cross ? min(base + count - 1, seq_len) : base + count;
  const int vis_end = a.cross ? min(base + j, seq_len) : base + (j < causal ? j + 1 : count);
  const int gk0 = grp * a.ppw * kAttnChunk;
  const int gk1 = min(gk0 + a.ppw * kAttnChunk, kv_end);
  const size_t oi = (((size_t)grp * a.B + b) * a.nq + hq) * a.R + j;

  if (gk0 >= gk1) {                                 // no keys in this split (workgroup-uniform)
    if (wrow0 >= rows) return;
    if (rvalid && g4 == 0) {
      a.mp[oi] = -INFINITY;
      a.lp[oi] = 0.f;
    }
    if (rvalid) {
      bf16_t* op = a.op + oi * D;
      for (int d = g4 * 4; d < D; d += 16) *reinterpret_cast<u32x2*>(op + d) = u32x2{0u, 0u};
    }
    return;
  }
  const bool active = wrow0 < rows;                 // wave-uniform; inactive waves still pass the barriers
  const int np = (gk1 - gk0 + kAttnChunk - 1) / kAttnChunk;

  u32x4 qf[D / 32];
  {
    const bf16_t* qp = a.q + ((size_t)(b * a.R + j) * a.nq + hq) * D + 8 * g4;
#pragma unroll
    for (int t = 0; t < D / 32; ++t) qf[t] = ld16(qp + 32 * t);
  }
  const int kst = D + kAttnPadK, vst = kAttnChunk + kAttnPadV;
  bf16_t* Ks = reinterpret_cast<bf16_t*>(lds);
  bf16_t* Vs = Ks + (size_t)kAttnChunk * kst;
  constexpr int PER_T = kAttnChunk * D / 8 / 256;   // 16-byte vectors per thread and operand
  static_assert(PER_T * 256 * 8 == kAttnChunk * D, "the threads cover the page exactly");
  constexpr int per_row = kAttnChunk / 8;
  u32x4 kr[PER_T], vr[PER_T];
  auto issue = [&](int pi) {   // page pi of the group: loads into registers
    const int page = a.pt[b * a.pps + grp * a.ppw + pi];
    const size_t pg = (size_t)page * a.nkv + kvh;
    const bf16_t* Kb = a.kc + pg * kAttnChunk * D;
    const bf16_t* Vb = a.vt + pg * D * kAttnChunk;
#pragma unroll
    for (int u = 0; u < PER_T; ++u) {
      const int i = threadIdx.x + 256 * u;
      // non-temporal: the 16 scenes' keys and values (~170 MB a layer) are
      // read once per pass and do not fit the last-level cache
      kr[u] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(Kb + (size_t)(i / (D / 8)) * D + 8 * (i % (D / 8))));
      vr[u] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(Vb + (size_t)(i / per_row) * kAttnChunk + 8 * (i % per_row)));
    }
  };
  auto stage = [&](int k0, int k1) {   // registers -> LDS; values past the valid keys as zeros
#pragma unroll
    for (int u = 0; u < PER_T; ++u) {
      const int i = threadIdx.x + 256 * u;
      *reinterpret_cast<u32x4*>(Ks + (size_t)(i / (D / 8)) * kst + 8 * (i % (D / 8))) = kr[u];
      const int d = i / per_row, v8 = i % per_row;
      attn_stage_values(Vs + (size_t)d * vst, v8, k0 + 8 * v8, k1, vr[u]);
    }
  };

  float m_run = -INFINITY, l_run = 0.f;
  f32x4 o[D / 16];
#pragma unroll
  for (int dt = 0; dt < D / 16; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  issue(0);
  for (int pi = 0; pi < np; ++pi) {   // workgroup-uniform
    const int k0 = gk0 + pi * kAttnChunk, k1 = min(k0 + kAttnChunk, kv_end);
    if (pi > 0) __syncthreads();      // every wave has read the previous page
    stage(k0, k1);
    __syncthreads();
    if (pi + 1 < np) issue(pi + 1);   // in flight while this page is used
    if (!active) continue;
    f32x4 sc[4];
#pragma unroll
    for (int h = 0; h < 4; ++h) {
      const bf16_t* kp = Ks + (size_t)(16 * h + (lane & 15)) * kst + 8 * g4;
      f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int t = 0; t < D / 32; ++t) acc = mfma16x16x32(*reinterpret_cast<const u32x4*>(kp + 32 * t), qf[t], acc);
      sc[h] = acc;
    }
    float p[16];
    float pm = -INFINITY;
#pragma unroll
    for (int h = 0; h < 4; ++h)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int key = k0 + 16 * h + 4 * g4 + i;
        const bool ok = rvalid && key < k1 && key < vis_end;
        const float v = ok ? sc[h][i] * a.scale_log2 : -INFINITY;
        p[h * 4 + i] = v;
        pm = fmaxf(pm, v);
      }
    pm = fmaxf(pm, __shfl_xor(pm, 16));
    pm = fmaxf(pm, __shfl_xor(pm, 32));
    const float m_new = fmaxf(m_run, pm);
    const float alpha = m_run == -INFINITY ? 0.f : exp2f(m_run - m_new);
    float ls = 0.f;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const float v = p[i];
      p[i] = (v == -INFINITY) ? 0.f : exp2f(v - m_new);
      ls += p[i];
    }
    l_run = l_run * alpha + ls;
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt) o[dt] *= alpha;
#pragma unroll
    for (int hb = 0; hb < 2; ++hb) {
      const float* ph = p + 8 * hb;
      const u32x4 pb = u32x4{pack2(ph[0], ph[1]), pack2(ph[2], ph[3]), pack2(ph[4], ph[5]), pack2(ph[6], ph[7])};
      // V^T operands read here, not ahead of the softmax: fewer registers, so
      // that three workgroups fit a CU and more pages are in flight
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt) {
        const bf16_t* vp = Vs + (size_t)(16 * dt + (lane & 15)) * vst + 32 * hb + 8 * g4;
        o[dt] = mfma16x16x32(*reinterpret_cast<const u32x4*>(vp), pb, o[dt]);
      }
    }
    m_run = m_new;
  }
  if (!active) return;
  l_run += __shfl_xor(l_run, 16);
  l_run += __shfl_xor(l_run, 32);
  if (rvalid) {
    bf16_t* op = a.op + oi * D;
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt)
      *reinterpret_cast<u32x2*>(op + 16 * dt + 4 * g4) =
          u32x2{pack2(o[dt].x, o[dt].y), pack2(o[dt].z, o[dt].w)};
    if (g4 == 0) {
      a.mp[oi] = m_run;
      a.lp[oi] = l_run;
    }
  }
}


size_t attn_lds_bytes(int chunk, int D) {
  return ((size_t)chunk * (D + kAttnPadK) + (size_t)D * (chunk + kAttnPadV)) * sizeof(bf16_t);
}

// Merge the splits of each (row, q head): o = sum_s 2^(m_s - M) O_s / sum_s
// 2^(m_s - M) l_s.  grid (R, q_heads, B), 256 threads: 8 groups of splits x 32 groups of 4 columns.
//
// Readout (RO): with w_s = 2^(m_s - M), L = sum_s w_s l_s, the mass of class c
// is sum_s w_s C_c,s / L, and E = sum_s w_s (E_s + (m_s - M) C_1,s) is the
// trajectory term relative to M, so that for q_k = 2^(s_k - M) / C_1 over the
// trajectory/text keys, H(q) = ln C_1 - ln 2 * E / C_1 (C_1 = sum_s w_s C_1,s).
struct CombineArgs {
  const SeqState* st;
  const bf16_t* op;      // bf16 partial outputs
  const float *mp, *lp;
  bf16_t* o;             // [Mpad][nq*D]
  int nq, D, R, B, chunk;
  const float* rp;       // readout: [splits][B][nq][R][4] partial class sums and E terms
  float* ro;             // readout: [B][R][nq][4] masses (visual, trajectory/text, generated), entropy
  float inv_ln[SPEC_MAX_BATCH];   // readout: 1 / ln(trajectory/text slots) of each sequence, 0 if <= 1
  int cross;             // cross-attention context (as AttnArgs::cross)
};

// One (row j, q head h, sequence b) of the combine; coef is LDS of at least
// ((splits + 3) & ~3) + 8 * D floats.  Called by all threads of a workgroup.
constexpr float kLn2 = 0.6931471805599453f;

template <bool RO>
__device__ __forceinline__ void combine_unit(const CombineArgs& a, int j, int h, int b, float* coef) {
  const SeqState& s = a.st[b];
  if (j >= s.count) return;
  const int vis_end = a.cross ? min(s.base + j, s.seq_len) : s.base + (j < s.causal ? j + 1 : s.count);
  const int ns = (vis_end + a.chunk - 1) / a.chunk;   // splits holding keys this row sees
  const size_t row = ((size_t)b * a.nq + h) * a.R + j;
  const size_t sstride = (size_t)a.B * a.nq * a.R;
  if (threadIdx.x < 64) {
    const int l = threadIdx.x;
    float M = -INFINITY;
    for (int sp = l; sp < ns; sp += 64) M = fmaxf(M, a.mp[sp * sstride + row]);
    for (int o = 32; o > 0; o >>= 1) M = fmaxf(M, __shfl_xor(M, o));
    float L = 0.f;
    float r[4] = {0.f, 0.f, 0.f, 0.f};
    for (int sp = l; sp < ns; sp += 64) {
      const float ms = a.mp[sp * sstride + row];   // finite: split sp holds a key the row sees
      const float w = exp2f(ms - M);
      coef[sp] = w;
      L += w * a.lp[sp * sstride + row];
      if (RO) {
        const f32x4 c = *reinterpret_cast<const f32x4*>(a.rp + (sp * sstride + row) * 4);
        r[0] += w * c.x;
        r[1] += w * c.y;
        r[2] += w * c.z;
        r[3] += w * (c.w + (ms - M) * c.y);
      }
    }
    for (int o = 32; o > 0; o >>= 1) L += __shfl_xor(L, o);
    const float inv = 1.f / L;
    for (int sp = l; sp < ns; sp += 64) coef[sp] *= inv;
    if (RO) {
#pragma unroll
      for (int k = 0; k < 4; ++k)
        for (int o = 32; o > 0; o >>= 1) r[k] += __shfl_xor(r[k], o);
      if (l == 0) {
        const float il = a.inv_ln[b];
        const float hn = (il > 0.f && r[1] > 0.f) ? (logf(r[1]) - kLn2 * r[3] / r[1]) * il : 0.f;
        *reinterpret_cast<f32x4*>(a.ro + (((size_t)b * a.R + j) * a.nq + h) * 4) =
            f32x4{r[0] * inv, r[1] * inv, r[2] * inv, hn};
      }
    }
  }
  __syncthreads();
  // thread = (split group sg of 8, 4-wide column group c4); D / 4 <= 32 groups
  float* part = coef + ((ns + 3) & ~3);
  const int c4 = threadIdx.x & 31, sg = threadIdx.x >> 5;
  f32x4 v = f32x4{0.f, 0.f, 0.f, 0.f};
  if (4 * c4 < a.D) {
    const bf16_t* src = a.op + row * a.D + 4 * c4;
    const size_t ostride = sstride * a.D;
#pragma unroll 4
    for (int sp = sg; sp < ns; sp += 8) {
      const u32x2 w = *reinterpret_cast<const u32x2*>(src + sp * ostride);
      const f32x4 ov = f32x4{__uint_as_float(w.x << 16), __uint_as_float(w.x & 0xffff0000u),
                             __uint_as_float(w.y << 16), __uint_as_float(w.y & 0xffff0000u)};
      v += coef[sp] * ov;
    }
    *reinterpret_cast<f32x4*>(part + sg * a.D + 4 * c4) = v;
  }
  __syncthreads();
  const int d = threadIdx.x;
  if (d < a.D) {
    float t = 0.f;
#pragma unroll
    for (int g = 0; g < 8; ++g) t += part[g * a.D + d];
    a.o[(size_t)(b * a.R + j) * a.nq * a.D + h * a.D + d] = f2bf(t);
  }
}

template <bool RO>
__global__ __launch_bounds__(256) void k_attn_combine(CombineArgs a) {
  extern __shared__ float coef[];   // [ns] weights, then [8][D] partial sums
  combine_unit<RO>(a, blockIdx.x, blockIdx.y, blockIdx.z, coef);
}

// ---------------------------------------------------------------------------
// Greedy token of each row (Eq. verify): reduce the LM head's per-tile
// (max, index) pairs; larger logit wins, ties go to the lower index.
// grid (rows per sequence, B), 1024 threads.  Verify: r*_{j+1} of row j goes
// to rstar[j].  Draft: the proposal of the step's last row is appended to the
// sequence's proposals and the draft length advances.
// ---------------------------------------------------------------------------
struct AmaxArgs {
  SeqState* st;
  const float* amax_v;
  const int32_t* amax_i;
  int ntiles, mpad, rps, draft;
  int32_t* out;          // draft: [B][K] proposals, column = draft calls so far (-1 when none); or null
  int K;
};

__global__ __launch_bounds__(1024) void k_argmax_rows(AmaxArgs p) {
  __shared__ float shv[1024];
  __shared__ int shi[1024];
  const int j = blockIdx.x, b = blockIdx.y;
  SeqState& s = p.st[b];
  if (s.count == 0) {
    if (p.draft && threadIdx.x == 0) {   // nothing proposed this call
      if (p.out && s.dcall < p.K) p.out[b * p.K + s.dcall] = -1;
      s.dcall += 1;
    }
    return;
  }
  const int row = b * p.rps + j;
  float v = -INFINITY;
  int i = 0x7fffffff;
  for (int t0 = threadIdx.x; t0 < p.ntiles; t0 += 1024 * 8) {
    float vv[8];
    int ii[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int t = t0 + 1024 * u;
      vv[u] = t < p.ntiles ? p.amax_v[(size_t)t * p.mpad + row] : -INFINITY;
      ii[u] = t < p.ntiles ? p.amax_i[(size_t)t * p.mpad + row] : 0x7fffffff;
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) amax_merge(v, i, vv[u], ii[u]);
  }
  shv[threadIdx.x] = v;
  shi[threadIdx.x] = i;
  __syncthreads();
  for (int o = 512; o > 0; o >>= 1) {
    if (threadIdx.x < o) {
      float v1 = shv[threadIdx.x];
      int i1 = shi[threadIdx.x];
      amax_merge(v1, i1, shv[threadIdx.x + o], shi[threadIdx.x + o]);
      shv[threadIdx.x] = v1;
      shi[threadIdx.x] = i1;
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    if (!p.draft) {
      s.rstar[j] = shi[0];
    } else {
      s.props[s.dstep] = shi[0];
      s.draft_len = s.base + s.count;
      s.dstep += 1;
      if (p.out && s.dcall < p.K) p.out[b * p.K + s.dcall] = shi[0];
      s.dcall += 1;
    }
  }
}

// Accept + commit (Eq. accept, Eq. commit): l = longest prefix of the verify's
// draft tokens equal to the target's greedy tokens; commit (d_1..d_l, r*_{l+1})
// cut after a stop token and at the token budget; append the tokens, advance
// the lengths and roll the draft back to the first slot whose input differs
// from the committed sequence (never past the new pending token).
// grid B, 1 thread.
__global__ void k_commit(SeqState* st, int32_t* hist, int cap, int K, int stop, int max_new, int32_t* o_acc,
                         int32_t* o_com, int32_t* o_n, int32_t* o_fin) {
  const int b = blockIdx.x;
  SeqState& s = st[b];
  int c = 0, l = 0;
  if (!s.finished) {
    while (l < K && s.vtok[l + 1] == s.rstar[l]) ++l;
    c = l + 1;
    for (int i = 0; i < l; ++i) s.committed[i] = s.vtok[i + 1];
    s.committed[l] = s.rstar[l];
    int fin = 0;
    if (stop >= 0)
      for (int i = 0; i < c; ++i)
        if (s.committed[i] == stop) {
          c = i + 1;
          fin = 1;
          break;
        }
    if (c >= max_new - s.n_gen) {
      c = max_new - s.n_gen;
      fin = 1;
    }
    const int n = s.seq_len;
    for (int i = 0; i < c; ++i) hist[(size_t)b * cap + n + 1 + i] = s.committed[i];
    int x = n + 1;
    while (x < s.draft_len && (x - n - 1) < c && s.props[x - n - 1] == s.committed[x - n - 1]) ++x;
    s.draft_len = min(min(s.draft_len, x), n + c);
    s.seq_len = n + c;
    s.pending = s.committed[c - 1];
    s.n_gen += c;
    s.finished = fin;
    s.accept_len = l;
    s.n_commit = c;
  }
  s.dstep = 0;
  s.dcall = 0;
  if (o_acc) o_acc[b] = l;
  if (o_n) o_n[b] = c;
  if (o_fin) o_fin[b] = s.finished;
  if (o_com)
    for (int i = 0; i <= K; ++i) o_com[b * (K + 1) + i] = i < c ? s.committed[i] : -1;
}

// Block proposal (Eq. propose in one forward): MASK row i of the pass (row
// i + 1) proposes d_i; the proposals go to the sequence's state and to the
// caller's [B][K] array.  Only the pending row's slot now holds the draft K/V
// of a real input.  grid B.
__global__ void k_block_props(SeqState* st, int K, int32_t* out) {
  const int b = blockIdx.x;
  SeqState& s = st[b];
  const bool live = s.count > 0;
  for (int i = threadIdx.x; i < K; i += blockDim.x) {
    const int d = live ? s.rstar[i + 1] : -1;
    if (live) s.props[i] = d;
    if (out) out[b * K + i] = d;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    if (live) {
      s.draft_len = s.base + 1;
      s.dstep = K;
    }
    s.dcall = K;
  }
}

// Conditioning: keep the verify rows' residual stream after a chosen target
// layer as column block `part` of cat3 (bf16).  grid (H/256, M).
__global__ void k_capture(const float* x, bf16_t* cat3, int H, int part) {
  const int m = blockIdx.y, n = blockIdx.x * 256 + threadIdx.x;
  if (n < H) cat3[(size_t)m * 3 * H + (size_t)part * H + n] = f2bf(x[(size_t)m * H + n]);
}

// After a commit: the fused features (sum of the k-split partials) of the
// rows whose inputs were committed become the features of their slots.
// grid (rows per sequence, B), 256 threads.
__global__ void k_feat_commit(const SeqState* st, const float* part, int S, int M, int rps, int H, bf16_t* feat,
                              int cap) {
  const int j = blockIdx.x, b = blockIdx.y;
  const SeqState& s = st[b];
  if (s.count == 0 || j >= s.n_commit) return;   // no verify rows, or row j not committed
  const int slot = s.seq_len - s.n_commit + j;
  const size_t m = (size_t)b * rps + j;
  for (int n = threadIdx.x; n < H; n += blockDim.x) {
    float v = 0.f;
    for (int sp = 0; sp < S; ++sp) v += part[((size_t)sp * M + m) * H + n];
    feat[((size_t)b * cap + slot) * H + n] = f2bf(v);
  }
}

// ---------------------------------------------------------------------------
// host-side launch helpers
// ---------------------------------------------------------------------------

int num_cus() {
  static int n = -1;
  if (n < 0) {
    int dev = 0, v = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0)
      v = 256;
    n = v;
  }
  return n;
}

int gemv_lds_limit() {
  static int lim = -1;
  if (lim < 0) {
    int dev = 0, v = 0;
    // without a device to ask (host-side validation), gfx950's 160 KB: the
    // library is built for that target only
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess || v <= 0)
      v = 160 * 1024;
    lim = std::min(v, 160 * 1024) - 256;   // room for the small static arrays
  }
  return lim;
}

int down_splits(int M, int Kd, int ncu) {
  const int T = (Kd + 31) / 32;
  int s = (T + kGemvWaves * kGemvSteps - 1) / (kGemvWaves * kGemvSteps);
  while (s < T && gemv_p_lds_bytes(M, (T + s - 1) / s) > (size_t)gemv_lds_limit()) ++s;
  // prefer a split count that divides the workgroups evenly (one group per split)
  for (int t = s; t <= 2 * s && t <= T; ++t)
    if (ncu % t == 0) return t;
  return s;
}

namespace {

// Per-launch timing: when enabled, the launch inside the scope passes e0/e1 to
// hipExtLaunchKernelGGL, which stamps them with the dispatch's own start and
// end times (no marker packets between kernels).
struct Timed {
  hipEvent_t e0 = nullptr, e1 = nullptr;
  Timed(Ctx& c, int kind, double bytes) {
    if (!c.timing) return;
    if (c.ev_used + 2 > c.ev_pool.size()) {
      for (int i = 0; i < 256; ++i) {
        hipEvent_t e;
        if (hipEventCreate(&e) == hipSuccess) c.ev_pool.push_back(e);
      }
    }
    if (c.ev_used + 2 > c.ev_pool.size()) return;
    e0 = c.ev_pool[c.ev_used++];
    e1 = c.ev_pool[c.ev_used++];
    c.trec.push_back(TimingRec{kind, bytes, e0, e1});
  }
};

hipStream_t S(Ctx& c) { return c.stream; }

template <int EPI, int TT, int MB>
void set_lds_limit() {
  (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&k_gemv<MB, kGemvWaves, kGemvSteps, TT, EPI>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, gemv_lds_limit());
}

template <int EPI, int TT>
hipError_t gemv_launch(Ctx& c, const GemvArgs& g, int kind, double bytes) {
  const int mb = (g.M + 15) / 16;
  const int T = (g.Kd + 31) / 32;
  const int span = (T + g.splits - 1) / g.splits;
  const size_t lds = gemv_lds_bytes(TT, g.M, span);
  if (lds > (size_t)gemv_lds_limit() || (span + kGemvWaves - 1) / kGemvWaves > kGemvSteps) return hipErrorInvalidValue;
  const int groups = g.N / (kTile * TT);
  const dim3 grid(groups, g.splits), block(kGemvWaves * 64);
  Timed t(c, kind, bytes);
  switch (mb) {
    case 1: hipExtLaunchKernelGGL((k_gemv<1, kGemvWaves, kGemvSteps, TT, EPI>), grid, block, lds, S(c), t.e0, t.e1, 0, g); break;
    case 2: hipExtLaunchKernelGGL((k_gemv<2, kGemvWaves, kGemvSteps, TT, EPI>), grid, block, lds, S(c), t.e0, t.e1, 0, g); break;
    case 3: hipExtLaunchKernelGGL((k_gemv<3, kGemvWaves, kGemvSteps, TT, EPI>), grid, block, lds, S(c), t.e0, t.e1, 0, g); break;
    case 4: hipExtLaunchKernelGGL((k_gemv<4, kGemvWaves, kGemvSteps, TT, EPI>), grid, block, lds, S(c), t.e0, t.e1, 0, g); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <int EPI, int MB>
void set_lds_limit_p() {
  (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&k_gemv_p<MB, kGemvWaves, kGemvSteps, EPI>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, gemv_lds_limit());
}

// Persistent launch: `workgroups` is a multiple of g.splits (one group per k-split).
template <int EPI>
hipError_t gemv_launch_p(Ctx& c, const GemvArgs& g, int workgroups, int kind, double bytes) {
  const int mb = (g.M + 15) / 16;
  const int T = (g.Kd + 31) / 32;
  const int span = (T + g.splits - 1) / g.splits;
  const size_t lds = gemv_p_lds_bytes(g.M, span);
  if (lds > (size_t)gemv_lds_limit() || (span + kGemvWaves - 1) / kGemvWaves > kGemvSteps ||
      workgroups % g.splits != 0)
    return hipErrorInvalidValue;
  const dim3 grid(workgroups), block(kGemvWaves * 64);
  Timed t(c, kind, bytes);
  switch (mb) {
    case 1: hipExtLaunchKernelGGL((k_gemv_p<1, kGemvWaves, kGemvSteps, EPI>), grid, block, lds, S(c), t.e0, t.e1, 0, g); break;
    case 2: hipExtLaunchKernelGGL((k_gemv_p<2, kGemvWaves, kGemvSteps, EPI>), grid, block, lds, S(c), t.e0, t.e1, 0, g); break;
    case 3: hipExtLaunchKernelGGL((k_gemv_p<3, kGemvWaves, kGemvSteps, EPI>), grid, block, lds, S(c), t.e0, t.e1, 0, g); break;
    case 4: hipExtLaunchKernelGGL((k_gemv_p<4, kGemvWaves, kGemvSteps, EPI>), grid, block, lds, S(c), t.e0, t.e1, 0, g); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// Algorithmic bytes of a GEMV launch: weights once, activations in, results out.
double gemv_bytes(int N, int Kd, int M, double out_bytes_per_elem) {
  return 2.0 * N * Kd + 2.0 * M * Kd + out_bytes_per_elem * (double)M * N;
}

GemvArgs gemv_base(Ctx& c, int M, int rps) {
  GemvArgs g{};
  g.st = c.st;
  g.M = M;
  g.rps = rps;
  g.splits = 1;
  g.mpad = c.Mpad;
  return g;
}

// Passes of more than kThinRows rows: the batched-row GEMM (gemm.hip).
hipError_t gemm_run(Ctx& c, int epi, const GemvArgs& g, int kind, double bytes) {
  Timed t(c, kind, bytes);
  return gemm_launch(epi, g, S(c), t.e0, t.e1);
}

#define CK(x)                               \
  do {                                      \
    hipError_t e_ = (x);                    \
    if (e_ != hipSuccess) return e_;        \
  } while (0)

// Split-KV attention of one layer + the combine of its splits; on the layer
// an armed readout names, the readout variants of both kernels.
hipError_t launch_attention(Ctx& c, Model& m, int li) {
  const spec_dims& d = m.d;
  const int D = d.head_dim, nq = d.q_heads, nkv = d.kv_heads;
  bf16_t* kc = m.kc + m.kv_layer * li;
  bf16_t* vt = m.vt + m.kv_layer * li;
  const int G = nq / nkv;
  const bool ro = c.ro_out && c.ro_m == &m && c.ro_layer == li;
  const int cross = (c.cross && &m == &c.drf && li == 0) ? 1 : 0;
  // several pages per workgroup where the context asks for it (many
  // sequences); a readout pass keeps one page per workgroup
  const int ppw = ro ? 1 : c.attn_ppw;
  // query rows of one kv head (rows per sequence x q heads per kv head): up
  // to 64 in one workgroup of 4 waves; more (e.g. 17 rows x 4 heads) in
  // workgroups of 8 waves, so that each page is staged once for all of them
  const int nw = (ppw == 1 && c.R * G > 64) ? 8 : 4;
  const int rb = (c.R * G + 16 * nw - 1) / (16 * nw);
  AttnArgs p{c.st, c.q, kc, vt, c.pt, c.op, c.mp, c.lp, nq, nkv, G, c.R, c.B, c.pps, c.attn_chunk, rb,
             kLog2e / sqrtf((float)D), c.cls, c.rp, c.cap, cross, ppw};
  dim3 grid((c.attn_splits + ppw - 1) / ppw, nkv * rb, c.B);
  CombineArgs cb{c.st, c.op, c.mp, c.lp, c.o, nq, D, c.R, c.B, c.attn_chunk * ppw, c.rp,
                 ro ? c.ro_out : nullptr, {}, cross};
  for (int b = 0; b < c.B && b < SPEC_MAX_BATCH; ++b) cb.inv_ln[b] = c.ro_inv_ln[b];
  const size_t comb_lds = (size_t)(((c.attn_splits + 3) & ~3) + 8 * D) * sizeof(float);
  const size_t lds = attn_lds_bytes(c.attn_chunk, D);
  {
    Timed t(c, SPEC_KERNEL_ATTN, 0);
    if (ppw > 1) {
      if (D == 128)
        hipExtLaunchKernelGGL(k_attn_pages<128>, grid, dim3(256), lds, S(c), t.e0, t.e1, 0, p);
      else
        hipExtLaunchKernelGGL(k_attn_pages<64>, grid, dim3(256), lds, S(c), t.e0, t.e1, 0, p);
    } else if (nw == 8) {
      if (D == 128)
        hipExtLaunchKernelGGL(ro ? k_attn<128, true, 8> : k_attn<128, false, 8>, grid, dim3(512), lds, S(c), t.e0, t.e1,
                              0, p);
      else
        hipExtLaunchKernelGGL(ro ? k_attn<64, true, 8> : k_attn<64, false, 8>, grid, dim3(512), lds, S(c), t.e0, t.e1, 0,
                              p);
    } else if (D == 128)
      hipExtLaunchKernelGGL(ro ? k_attn<128, true, 4> : k_attn<128, false, 4>, grid, dim3(256), lds, S(c), t.e0, t.e1, 0,
                            p);
    else
      hipExtLaunchKernelGGL(ro ? k_attn<64, true, 4> : k_attn<64, false, 4>, grid, dim3(256), lds, S(c), t.e0, t.e1, 0, p);
    CK(hipGetLastError());
  }
  Timed t2(c, SPEC_KERNEL_OTHER, 0);
  hipExtLaunchKernelGGL(ro ? k_attn_combine<true> : k_attn_combine<false>, dim3(c.R, nq, c.B), dim3(256), comb_lds,
                        S(c), t2.e0, t2.e1, 0, cb);
  return hipGetLastError();
}

// A packed-GEMV job with the context's current partial-tile, counter,
// argmax and logits buffers: the planned jobs keep the workspace's, and a
// call that moves those buffers elsewhere (spec_verify_scratch) swaps the
// context's pointers for its duration.
SgJob sg_job(const Ctx& c, const SgJob& j) {
  SgJob r = j;
  r.part = c.sg_part;
  r.cnt = c.sg_cnt;
  if (r.amax_v) {
    r.amax_v = c.amax_v;
    r.amax_i = c.amax_i;
    r.logits = c.logits;
  }
  return r;
}

// One layer on the packed-weight path: q/k/v (+rotary, KV append),
// attention, o (+residual), gate/up (+SwiGLU), down (+residual, next norm).
hipError_t run_layer_sg(Ctx& c, Model& m, int li, bool block) {
  const spec_dims& d = m.d;
  const int H = d.hidden, D = d.head_dim, nq = d.q_heads, nkv = d.kv_heads, F = d.ffn;
  const int M = c.M;
  const SgJob* hj = m.sg_host.data() + (size_t)li * 4;
  // a block proposal's last layer writes the LM head input of every row
  const SgJob& down = (block && li + 1 == d.layers) ? m.sg_block[0] : hj[3];
  {
    Timed t(c, SPEC_KERNEL_QKV, gemv_bytes((nq + 2 * nkv) * D, H, M, 2.0));
    CK(sg_launch(SG_ROPE, sg_job(c, hj[0]), S(c), t.e0, t.e1));
  }
  CK(launch_attention(c, m, li));
  {
    Timed t(c, SPEC_KERNEL_O, gemv_bytes(H, nq * D, M, 10.0));
    CK(sg_launch(SG_RESID, sg_job(c, hj[1]), S(c), t.e0, t.e1));
  }
  {
    Timed t(c, SPEC_KERNEL_GATEUP, gemv_bytes(2 * F, H, M, 1.0));
    CK(sg_launch(SG_SWIGLU, sg_job(c, hj[2]), S(c), t.e0, t.e1));
  }
  {
    Timed t(c, SPEC_KERNEL_DOWN, gemv_bytes(H, F, M, 10.0));
    CK(sg_launch(SG_DOWN, sg_job(c, down), S(c), t.e0, t.e1));
  }
  return hipSuccess;
}

// q, k, v (+ 1/rms of the attention norm) + rotary + cache append of one
// layer on the row-major path (thin GEMV or batched GEMM), appending K and
// V^T to the given layer pools.
hipError_t launch_qkv_rm(Ctx& c, Model& m, int li, bf16_t* kc, bf16_t* vt) {
  const spec_dims& d = m.d;
  const int H = d.hidden, D = d.head_dim, nq = d.q_heads, nkv = d.kv_heads;
  const int M = c.M;
  const LayerW& w = m.L[li];
  const bf16_t* pk = (c.gemm_rows && c.gemm_pk) ? m.pk + m.pk_layer * li : nullptr;
  GemvArgs g = gemv_base(c, M, c.R);
  g.w[0] = w.wq;
  g.w[1] = w.wk;
  g.w[2] = w.wv;
  g.row0[0] = 0;
  g.row0[1] = nq * D;
  g.row0[2] = (nq + nkv) * D;
  g.nseg = 3;
  g.N = (nq + 2 * nkv) * D;
  g.Kd = H;
  g.x = c.xg;
  g.ldx = H;
  g.ss_in = c.ss;
  g.H = H;
  g.eps = d.rms_eps;
  g.q = c.q;
  g.kc = kc;
  g.vt = vt;
  g.rcs = c.rcs;
  g.nq = nq;
  g.nkv = nkv;
  g.D = D;
  g.pt = c.pt;
  g.pps = c.pps;
  g.pw = pk;
  const int sq = c.gemm_rows ? gemm_qkv_splits_for(g.N, H, M, c.ncu, c.gemm_wide) : 1;
  if (sq > 1) {
    // too few 64-column workgroups to stream the matrix at full rate: k-split
    // partial sums, then the norm, rotation and cache append in k_qkv_finish
    g.splits = sq;
    g.out = c.part;
    if (pk && c.xgp && li > 0) {   // the step-major copy the previous layer's down finish wrote
      g.x = c.xgp;
      g.xpk = 1;
    }
    CK(gemm_run(c, EPI_STORE, g, SPEC_KERNEL_QKV, gemv_bytes(g.N, H, M, 4.0 * sq)));
    QkvFinishArgs p{c.st, c.part, sq, M, g.N, c.R, c.Mpad, H, d.rms_eps, c.ss, c.rcs, c.pt,
                    nq, nkv, D, c.pps, c.q, kc, vt};
    Timed t(c, SPEC_KERNEL_OTHER, 0);
    hipExtLaunchKernelGGL(k_qkv_finish, dim3((g.N / 2 + 255) / 256, M), dim3(256), 0, S(c), t.e0, t.e1, 0, p);
    CK(hipGetLastError());
  } else if (c.gemm_rows)
    CK(gemm_run(c, EPI_ROPE, g, SPEC_KERNEL_QKV, gemv_bytes(g.N, H, M, 2.0)));
  else
    CK((gemv_launch<EPI_ROPE, 1>(c, g, SPEC_KERNEL_QKV, gemv_bytes(g.N, H, M, 2.0))));
  return hipSuccess;
}

hipError_t run_layer(Ctx& c, Model& m, int li, const bf16_t* next_gain, bool select_last) {
  const spec_dims& d = m.d;
  const int H = d.hidden, D = d.head_dim, nq = d.q_heads, F = d.ffn;
  const int M = c.M;
  const LayerW& w = m.L[li];
  bf16_t* kc = m.kc + m.kv_layer * li;
  bf16_t* vt = m.vt + m.kv_layer * li;
  // the GEMM streams this layer's tile-packed copy when there is one
  const bf16_t* pk = (c.gemm_rows && c.gemm_pk) ? m.pk + m.pk_layer * li : nullptr;

  // q, k, v (+ 1/rms of the attention norm) + rotary + cache append; the
  // draft's layer 0 under cross-attention conditioning appends nowhere
  // visible (its cache holds the target context)
  if (c.cross && &m == &c.drf && li == 0)
    CK(launch_qkv_rm(c, m, li, c.junk_kc, c.junk_vt));
  else
    CK(launch_qkv_rm(c, m, li, kc, vt));
  CK(launch_attention(c, m, li));
  // o projection + residual; bf16(x * g_ffn) and sums of x^2 for the FFN norm
  {
    GemvArgs g = gemv_base(c, M, c.R);
    g.w[0] = w.wo;
    g.nseg = 1;
    g.N = H;
    g.Kd = nq * D;
    g.x = c.o;
    g.ldx = nq * D;
    g.x32 = c.x;
    g.gain = w.ffn_norm;
    g.xg = c.xg;
    g.ss_out = c.ss;
    g.pw = pk ? pk + m.pk_o : nullptr;
    if (c.gemm_rows) {
      // k-split partial sums, so that enough workgroups stream the narrow
      // matrix; the finishing kernel adds them to the residual stream and
      // writes the FFN norm's input, as after the down projection
      g.splits = m.s_o;
      g.out = c.part;
      CK(gemm_run(c, EPI_STORE, g, SPEC_KERNEL_O, gemv_bytes(H, nq * D, M, 4.0 * m.s_o)));
      FinishArgs p{c.st, c.part, m.s_o, M, c.R, H, c.Mpad, 0, c.x, w.ffn_norm, c.xg, c.ss, c.xgp};
      Timed t(c, SPEC_KERNEL_OTHER, 0);
      hipExtLaunchKernelGGL(k_down_finish, dim3((H + 255) / 256, M), dim3(256), 0, S(c), t.e0, t.e1, 0, p);
      CK(hipGetLastError());
    } else {
      CK((gemv_launch<EPI_RESID, 1>(c, g, SPEC_KERNEL_O, gemv_bytes(H, nq * D, M, 10.0))));
    }
  }
  // gate/up (+ 1/rms of the FFN norm) + SwiGLU
  {
    GemvArgs g = gemv_base(c, M, c.R);
    g.w[0] = w.wg;
    g.w[1] = w.wu;
    g.row0[1] = F;
    g.nseg = 2;
    g.N = 2 * F;
    g.Kd = H;
    g.x = c.xg;
    g.ldx = H;
    g.ss_in = c.ss;
    g.H = H;
    g.eps = d.rms_eps;
    g.u = c.u;
    g.pw = pk ? pk + m.pk_gu : nullptr;
    if (pk && c.xgp) {   // the wide-unit GEMM reads the step-major copy the o finish wrote
      g.x = c.xgp;
      g.xpk = 1;
      g.upk = 1;         // and writes u step-major for the down projection
    }
    if (c.gemm_rows)
      CK(gemm_run(c, EPI_SWIGLU, g, SPEC_KERNEL_GATEUP, gemv_bytes(2 * F, H, M, 1.0)));
    else
      CK(gemv_launch_p<EPI_SWIGLU>(c, g, std::min(c.ncu, 2 * F / kTile), SPEC_KERNEL_GATEUP,
                                   gemv_bytes(2 * F, H, M, 1.0)));
  }
  // down projection (k-split partials) -> residual + the next norm's input
  {
    const int S_down = m.s_down;
    {
      GemvArgs g = gemv_base(c, M, c.R);
      g.w[0] = w.wd;
      g.nseg = 1;
      g.N = H;
      g.Kd = F;
      g.x = c.u;
      g.ldx = F;
      g.splits = m.s_down;
      g.out = c.part;
      g.pw = pk ? pk + m.pk_dn : nullptr;
      g.xpk = (pk && c.xgp) ? 1 : 0;   // u as the wide-unit gate/up GEMM wrote it
      if (c.gemm_rows) {
        CK(gemm_run(c, EPI_STORE, g, SPEC_KERNEL_DOWN, gemv_bytes(H, F, M, 4.0 * m.s_down)));
      } else {
        const int per_split = std::max(1, std::min(c.ncu / m.s_down, H / kTile));
        CK(gemv_launch_p<EPI_STORE>(c, g, per_split * m.s_down, SPEC_KERNEL_DOWN, gemv_bytes(H, F, M, 4.0 * m.s_down)));
      }
    }
    FinishArgs p{c.st, c.part, S_down, M, c.R, H, c.Mpad, select_last ? 1 : 0, c.x, next_gain, c.xg, c.ss, c.xgp};
    Timed t(c, SPEC_KERNEL_OTHER, 0);
    hipExtLaunchKernelGGL(k_down_finish, dim3((H + 255) / 256, M), dim3(256), 0, S(c), t.e0, t.e1, 0, p);
    CK(hipGetLastError());
  }
  return hipSuccess;
}

}  // namespace

void init_kernel_attributes() {
  static bool done = false;
  if (done) return;
  done = true;
  sg_set_attributes(gemv_lds_limit());
  gemm_set_attributes(gemv_lds_limit());
  const void* attn[8] = {
      reinterpret_cast<const void*>(&k_attn<128, false, 4>), reinterpret_cast<const void*>(&k_attn<128, true, 4>),
      reinterpret_cast<const void*>(&k_attn<128, false, 8>), reinterpret_cast<const void*>(&k_attn<128, true, 8>),
      reinterpret_cast<const void*>(&k_attn<64, false, 4>),  reinterpret_cast<const void*>(&k_attn<64, true, 4>),
      reinterpret_cast<const void*>(&k_attn<64, false, 8>),  reinterpret_cast<const void*>(&k_attn<64, true, 8>)};
  for (int i = 0; i < 8; ++i)
    (void)hipFuncSetAttribute(attn[i], hipFuncAttributeMaxDynamicSharedMemorySize,
                              (int)attn_lds_bytes(kAttnChunk, i < 4 ? 128 : 64));
  (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&k_attn_pages<128>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)attn_lds_bytes(kAttnChunk, 128));
  (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&k_attn_pages<64>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)attn_lds_bytes(kAttnChunk, 64));
  set_lds_limit_p<EPI_STORE, 1>();
  set_lds_limit_p<EPI_STORE, 2>();
  set_lds_limit_p<EPI_STORE, 3>();
  set_lds_limit_p<EPI_STORE, 4>();
  set_lds_limit_p<EPI_SWIGLU, 1>();
  set_lds_limit_p<EPI_SWIGLU, 2>();
  set_lds_limit_p<EPI_SWIGLU, 3>();
  set_lds_limit_p<EPI_SWIGLU, 4>();
  set_lds_limit_p<EPI_ARGMAX, 1>();
  set_lds_limit_p<EPI_ARGMAX, 2>();
  set_lds_limit_p<EPI_ARGMAX, 3>();
  set_lds_limit_p<EPI_ARGMAX, 4>();
  set_lds_limit<EPI_STORE, 1, 1>();
  set_lds_limit<EPI_STORE, 1, 2>();
  set_lds_limit<EPI_STORE, 1, 3>();
  set_lds_limit<EPI_STORE, 1, 4>();
  set_lds_limit<EPI_ROPE, 1, 1>();
  set_lds_limit<EPI_SWIGLU, 1, 1>();
  set_lds_limit<EPI_ROPE, 1, 2>();
  set_lds_limit<EPI_SWIGLU, 1, 2>();
  set_lds_limit<EPI_ROPE, 1, 3>();
  set_lds_limit<EPI_SWIGLU, 1, 3>();
  set_lds_limit<EPI_ROPE, 1, 4>();
  set_lds_limit<EPI_SWIGLU, 1, 4>();
  set_lds_limit<EPI_RESID, 1, 1>();
  set_lds_limit<EPI_RESID, 1, 2>();
  set_lds_limit<EPI_RESID, 1, 3>();
  set_lds_limit<EPI_RESID, 1, 4>();
  set_lds_limit<EPI_ARGMAX, 1, 1>();
  set_lds_limit<EPI_ARGMAX, 1, 2>();
  set_lds_limit<EPI_ARGMAX, 1, 3>();
  set_lds_limit<EPI_ARGMAX, 1, 4>();
}

hipError_t launch_hold(Ctx& c, double ms) {
  int khz = 0;
  if (hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, c.device) != hipSuccess || khz <= 0)
    khz = 100000;
  ms = std::min(std::max(ms, 0.0), 100.0);
  hipLaunchKernelGGL(k_hold, dim3(1), dim3(1), 0, c.stream, (long long)(ms * khz));
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Packed-weight path: job tables and weight packing
// ---------------------------------------------------------------------------
namespace {
int steps_of(int Kd) { return (Kd + 31) / 32; }
}  // namespace

void pk_offsets(Model& m) {
  const spec_dims& d = m.d;
  const int H = d.hidden, D = d.head_dim, nq = d.q_heads, nkv = d.kv_heads, F = d.ffn;
  const int nqkv = (nq + 2 * nkv) * D;
  m.pk_o = sg_packed_elems(nqkv / kTile, steps_of(H));
  m.pk_gu = m.pk_o + sg_packed_elems(H / kTile, steps_of(nq * D));
  m.pk_dn = m.pk_gu + sg_packed_elems(2 * F / kTile, steps_of(H));
  m.pk_layer = m.pk_dn + sg_packed_elems(H / kTile, steps_of(F));
}

bool sg_build_jobs(Ctx& c, Model& m, bool draft, bool fill) {
  const spec_dims& d = m.d;
  const int H = d.hidden, D = d.head_dim, nq = d.q_heads, nkv = d.kv_heads, F = d.ffn;
  const int ncu = c.ncu, lim = gemv_lds_limit();
  const int nqkv = (nq + 2 * nkv) * D;
  pk_offsets(m);
  m.sg_host.assign((size_t)d.layers * 4 + 1, SgJob{});
  auto base = [&](SgJob& j, int ntiles, int Kd, const bf16_t* x) {
    j.ntiles = ntiles;
    j.T = steps_of(Kd);
    j.Kd = Kd;
    j.ldx = Kd;
    j.x = x;
    j.M = c.M;
    j.rps = c.R;
    j.mpad = c.Mpad;
    j.eps = d.rms_eps;
    j.st = c.st;
    j.part = c.sg_part;
    j.cnt = c.sg_cnt;
  };
  for (int li = 0; li < d.layers; ++li) {
    SgJob* j = m.sg_host.data() + (size_t)li * 4;
    bf16_t* pk = m.pk ? m.pk + m.pk_layer * li : nullptr;
    const bool last = li + 1 == d.layers;
    base(j[0], nqkv / kTile, H, c.xg);
    j[0].w = pk;
    j[0].ss_in = c.ss;
    j[0].Hn = H;
    j[0].q = c.q;
    // the draft's layer 0 under cross-attention conditioning: its rows'
    // own K/V go to the unread pools (that layer's cache is the context)
    const bool junk = c.cross && draft && li == 0;
    j[0].kc = junk ? c.junk_kc : (m.kc ? m.kc + m.kv_layer * li : nullptr);
    j[0].vt = junk ? c.junk_vt : (m.vt ? m.vt + m.kv_layer * li : nullptr);
    j[0].pt = c.pt;
    j[0].pps = c.pps;
    j[0].rcs = c.rcs;
    j[0].nq = nq;
    j[0].nkv = nkv;
    j[0].D = D;
    base(j[1], H / kTile, nq * D, c.o);
    j[1].w = pk ? pk + m.pk_o : nullptr;
    j[1].x32 = c.x;
    j[1].H = H;
    j[1].gain = fill ? m.L[li].ffn_norm : nullptr;
    j[1].xg = c.xg;
    j[1].ss_out = c.ss;
    base(j[2], 2 * F / kTile, H, c.xg);
    j[2].w = pk ? pk + m.pk_gu : nullptr;
    j[2].ss_in = c.ss;
    j[2].Hn = H;
    j[2].u = c.u;
    base(j[3], H / kTile, F, c.u);
    // the down projection streams x; its input is written step-major so that
    // the rows of one k-step are a single contiguous run
    j[2].upk = j[3].xpk = F > 32 * kSgMaxSpan ? 1 : 0;
    j[3].w = pk ? pk + m.pk_dn : nullptr;
    j[3].x32 = c.x;
    j[3].H = H;
    j[3].gain = fill ? (last ? m.final_norm : m.L[li + 1].attn_norm) : nullptr;
    j[3].xg = c.xg;
    j[3].ss_out = c.ss;
    j[3].select_last = (draft && last) ? 1 : 0;
    const int epis[4] = {SG_ROPE, SG_RESID, SG_SWIGLU, SG_DOWN};
    for (int k = 0; k < 4; ++k)
      if (!sg_plan(j[k], epis[k], ncu, lim)) return false;
  }
  SgJob& h = m.sg_host[(size_t)d.layers * 4];
  base(h, c.V / kTile, H, c.xg);
  h.w = c.pk_head;
  h.M = draft ? c.B : c.M;
  h.rps = draft ? 1 : c.R;
  h.ss_in = c.ss;
  h.Hn = H;
  h.amax_v = c.amax_v;
  h.amax_i = c.amax_i;
  h.logits = c.logits;
  h.allow_logits = draft ? 0 : 1;
  if (!sg_plan(h, SG_ARGMAX, ncu, lim)) return false;
  // block proposal: the last layer's down writes every row's LM head input,
  // and the LM head runs over all rows
  m.sg_block.clear();
  if (draft && c.block_draft) {
    SgJob dn = m.sg_host[(size_t)(d.layers - 1) * 4 + 3];
    dn.select_last = 0;
    SgJob hd = h;
    hd.M = c.M;
    hd.rps = c.R;
    hd.allow_logits = 0;
    if (!sg_plan(dn, SG_DOWN, ncu, lim) || !sg_plan(hd, SG_ARGMAX, ncu, lim)) return false;
    m.sg_block = {dn, hd};
  }
  return true;
}

hipError_t sg_pack_model(Ctx& c, Model& m) {
  const spec_dims& d = m.d;
  const int H = d.hidden, D = d.head_dim, nq = d.q_heads, nkv = d.kv_heads, F = d.ffn;
  for (int li = 0; li < d.layers; ++li) {
    const LayerW& w = m.L[li];
    bf16_t* pk = m.pk + m.pk_layer * li;
    PackSrc a{};
    a.seg[0] = w.wq;
    a.seg[1] = w.wk;
    a.seg[2] = w.wv;
    a.row0[1] = nq * D;
    a.row0[2] = (nq + nkv) * D;
    a.nseg = 3;
    a.Kd = H;
    a.ntiles = (nq + 2 * nkv) * D / kTile;
    a.T = steps_of(H);
    CK(sg_pack(pk, a, c.stream));
    PackSrc o{};
    o.seg[0] = w.wo;
    o.nseg = 1;
    o.Kd = nq * D;
    o.ntiles = H / kTile;
    o.T = steps_of(nq * D);
    CK(sg_pack(pk + m.pk_o, o, c.stream));
    PackSrc g{};
    g.seg[0] = w.wg;
    g.seg[1] = w.wu;
    g.nseg = 2;
    g.pair = 1;
    g.Kd = H;
    g.ntiles = 2 * F / kTile;
    g.T = steps_of(H);
    CK(sg_pack(pk + m.pk_gu, g, c.stream));
    PackSrc dn{};
    dn.seg[0] = w.wd;
    dn.nseg = 1;
    dn.Kd = F;
    dn.ntiles = H / kTile;
    dn.T = steps_of(F);
    CK(sg_pack(pk + m.pk_dn, dn, c.stream));
  }
  return hipSuccess;
}

hipError_t sg_pack_head(Ctx& c) {
  PackSrc e{};
  e.seg[0] = c.embed;
  e.nseg = 1;
  e.Kd = c.tgt.d.hidden;
  e.ntiles = c.V / kTile;
  e.T = steps_of(e.Kd);
  return sg_pack(c.pk_head, e, c.stream);
}

hipError_t launch_stream_read(const void* p, size_t bytes, uint32_t* sink, int sink_words, hipStream_t s) {
  hipLaunchKernelGGL(k_stream_read, dim3(sink_words / 4), dim3(256), 0, s, reinterpret_cast<const u32x4*>(p), bytes / 16,
                     sink);
  return hipGetLastError();
}

hipError_t launch_zero(Ctx& c, void* p, size_t bytes) {
  const size_t n = bytes / 16;
  if (n == 0) return hipSuccess;
  const int blocks = (int)std::min<size_t>((n + 255) / 256, 4096);
  hipLaunchKernelGGL(k_zero, dim3(blocks), dim3(256), 0, c.stream, reinterpret_cast<u32x4*>(p), n);
  return hipGetLastError();
}

hipError_t launch_prefix_kv(Ctx& c, Model& m, int layer, int b, int prefix_len, const bf16_t* k_pre,
                            const bf16_t* v) {
  const spec_dims& d = m.d;
  const size_t kvl = m.kv_layer;
  PrefixArgs p{k_pre,
               v,
               m.kc + kvl * layer,
               m.vt + kvl * layer,
               c.pt + (size_t)b * c.pps,
               c.pos3 + (size_t)b * 3 * c.cap,
               c.cs,
               m.axis,
               prefix_len,
               d.kv_heads,
               d.head_dim,
               c.cap,
               m.flat ? 1 : 0};
  const size_t total = (size_t)prefix_len * d.kv_heads * (d.head_dim / 2);
  const int blocks = (int)std::min<size_t>((total + 255) / 256, 8192);
  hipLaunchKernelGGL(k_prefix_kv, dim3(blocks), dim3(256), 0, c.stream, p);
  return hipGetLastError();
}

hipError_t launch_stage_verify(Ctx& c, const int32_t* d_override, int want_logits) {
  Timed t(c, SPEC_KERNEL_OTHER, 0);
  hipExtLaunchKernelGGL(k_stage_verify, dim3(c.B), dim3(64), 0, c.stream, t.e0, t.e1, 0, c.st, d_override, c.K, c.V, want_logits);
  return hipGetLastError();
}

// A k-split GEMV y = W x over the pass's rows (partial sums into `out`),
// on the thin kernels or, for the GEMM's row counts, on the batched GEMM.
hipError_t cond_gemv(Ctx& c, const bf16_t* w, const bf16_t* x, int N, int Kd, int S, float* out) {
  GemvArgs g = gemv_base(c, c.M, c.R);
  g.w[0] = w;
  g.nseg = 1;
  g.N = N;
  g.Kd = Kd;
  g.x = x;
  g.ldx = Kd;
  g.splits = S;
  g.out = out;
  const double bytes = gemv_bytes(N, Kd, c.M, 4.0 * S);
  if (c.gemm_rows) return gemm_run(c, EPI_STORE, g, SPEC_KERNEL_OTHER, bytes);
  const int per_split = std::max(1, std::min(c.ncu / S, N / kTile));
  return gemv_launch_p<EPI_STORE>(c, g, per_split * S, SPEC_KERNEL_OTHER, bytes);
}

// Conditioned draft pass: x = e + W_in [e; f] before layer 0, the layer-0
// norm input rewritten by the finishing kernel of the down projection.
hipError_t launch_cond_input(Ctx& c, Model& m) {
  const int H = m.d.hidden;
  CK(cond_gemv(c, c.w_in, c.cat2, H, 2 * H, kCondSplits, c.part));
  FinishArgs p{c.st, c.part, kCondSplits, c.M, c.R, H, c.Mpad, 0, c.x, m.L[0].attn_norm, c.xg, c.ss};
  Timed t(c, SPEC_KERNEL_OTHER, 0);
  hipExtLaunchKernelGGL(k_down_finish, dim3((H + 255) / 256, c.M), dim3(256), 0, S(c), t.e0, t.e1, 0, p);
  return hipGetLastError();
}

// Verify pass: w_fuse [h0; h1; h2] of every row, as k-split partials (the
// commit keeps the committed rows').
hipError_t launch_cond_fuse(Ctx& c) {
  const int H = c.tgt.d.hidden;
  return cond_gemv(c, c.w_fuse, c.cat3, H, 3 * H, kCondSplits, c.fusedp);
}

hipError_t launch_forward(Ctx& c, PassMode mode) {
  Model& m = mode == PASS_VERIFY ? c.tgt : c.drf;
  const spec_dims& d = m.d;
  const int M = c.M;
  {
    EmbedArgs p{c.st,    c.hist, c.embed,      m.L[0].attn_norm, c.x, c.xg,
                c.ss,  c.rcs,
                c.pos3,  c.cs,   m.axis,       d.hidden,         c.R, c.cap,    (int)mode, c.Mpad,
                d.head_dim, m.flat ? 1 : 0, c.V, c.mask_token,
                (c.cond && !c.cross && mode != PASS_VERIFY) ? c.cat2 : nullptr, c.feat};
    Timed t(c, SPEC_KERNEL_OTHER, 0);
    hipExtLaunchKernelGGL(k_embed, dim3(c.R, c.B), dim3(1024), (size_t)d.hidden * sizeof(float), c.stream, t.e0, t.e1, 0, p);
    CK(hipGetLastError());
  }
  // draft: a draft step, which proposes from each sequence's last row (stored
  // as row b); a block pass runs the LM head over every row, as a verify does
  const bool draft = mode == PASS_DRAFT, block = mode == PASS_BLOCK;
  if (c.cond && !c.cross && mode != PASS_VERIFY) CK(launch_cond_input(c, m));
  auto capture = [&](int li) -> hipError_t {   // conditioning: the verify keeps chosen layers' output
    if (!c.cond || mode != PASS_VERIFY) return hipSuccess;
    for (int i = 0; i < 3; ++i)
      if (c.cond_layers[i] == li) {
        Timed t(c, SPEC_KERNEL_OTHER, 0);
        hipExtLaunchKernelGGL(k_capture, dim3((d.hidden + 255) / 256, M), dim3(256), 0, S(c), t.e0, t.e1, 0, c.x,
                              c.cat3, d.hidden, i);
        CK(hipGetLastError());
      }
    return hipSuccess;
  };
  if (c.sg) {
    for (int li = 0; li < d.layers; ++li) {
      CK(run_layer_sg(c, m, li, block));
      CK(capture(li));
    }
  } else {
    for (int li = 0; li < d.layers; ++li) {
      const bool last = li + 1 == d.layers;
      CK(run_layer(c, m, li, last ? m.final_norm : m.L[li + 1].attn_norm, last && draft));
      CK(capture(li));
    }
  }
  if (c.cond && mode == PASS_VERIFY) CK(launch_cond_fuse(c));
  if (mode == PASS_CATCHUP) return hipSuccess;   // consumes tokens only: no LM head
  // LM head (+ 1/rms of the final norm) with the fused per-tile argmax; the
  // draft proposes from each sequence's last row only (stored as row b)
  bool reduced = false;   // the LM head's last workgroup already reduced the rows (fused tail)
  if (c.sg) {
    const int rows = draft ? c.B : M;
    const double bytes = gemv_bytes(c.V, d.hidden, rows, 0.0) + 8.0 * (c.V / kTile) * rows;
    Timed t(c, SPEC_KERNEL_LMHEAD, bytes);
    const size_t hi = (size_t)d.layers * 4;
    SgJob h = sg_job(c, block ? m.sg_block[1] : m.sg_host[hi]);
    if (h.S == 1) {
      h.tail = draft ? 2 : 1;
      h.tail_K = c.K;
      h.tail_out = draft ? c.draft_out : nullptr;
      h.tail_cnt = c.sg_cnt + c.sg_units;
      reduced = true;
    }
    CK(sg_launch(SG_ARGMAX, h, S(c), t.e0, t.e1));
  } else {
    GemvArgs g = gemv_base(c, draft ? c.B : M, draft ? 1 : c.R);
    g.w[0] = c.embed;
    g.nseg = 1;
    g.N = c.V;
    g.Kd = d.hidden;
    g.x = c.xg;
    g.ldx = d.hidden;
    g.ss_in = c.ss;
    g.H = d.hidden;
    g.eps = d.rms_eps;
    g.amax_v = c.amax_v;
    g.amax_i = c.amax_i;
    g.logits = c.logits;
    g.allow_logits = mode == PASS_VERIFY ? 1 : 0;
    const double bytes = gemv_bytes(c.V, d.hidden, g.M, 0.0) + 8.0 * (c.V / kTile) * g.M;
    if (g.M > kThinRows || (!draft && c.gemm_rows)) {
      g.pw = c.gemm_pk ? c.pk_head : nullptr;
      if (!draft && g.pw && c.xgp) {   // the step-major copy the last down finish wrote
        g.x = c.xgp;
        g.xpk = 1;
      }
      CK(gemm_run(c, EPI_ARGMAX, g, SPEC_KERNEL_LMHEAD, bytes));
    }
    else
      CK(gemv_launch_p<EPI_ARGMAX>(c, g, std::min(c.ncu, c.V / kTile), SPEC_KERNEL_LMHEAD, bytes));
  }
  // (max, index) entries per row the LM head left: one per tile, or one per
  // workgroup on the packed path
  const int ntiles = c.sg ? (block ? m.sg_block[1] : m.sg_host[(size_t)d.layers * 4]).amax_n : c.V / kTile;
  if (!reduced) {
    Timed t(c, SPEC_KERNEL_OTHER, 0);
    AmaxArgs p{c.st, c.amax_v, c.amax_i, ntiles, c.Mpad, draft ? 1 : c.R, draft ? 1 : 0, draft ? c.draft_out : nullptr, c.K};
    hipExtLaunchKernelGGL(k_argmax_rows, dim3(draft ? 1 : c.R, c.B), dim3(1024), 0, c.stream, t.e0, t.e1, 0, p);
    CK(hipGetLastError());
  }
  if (block) {
    Timed t(c, SPEC_KERNEL_OTHER, 0);
    hipExtLaunchKernelGGL(k_block_props, dim3(c.B), dim3(64), 0, c.stream, t.e0, t.e1, 0, c.st, c.K, c.draft_out);
    CK(hipGetLastError());
  }
  return hipSuccess;
}

// Cross-attention conditioning, after a commit (Sec. 4.1): the committed
// slots' fused features become the draft's layer-0 context.  They take the
// draft's layer-0 norm and q/k/v projection as a pass of their own: rows at
// the verify's committed slots, keys rotated at those slots and appended with
// the values to the layer's cache (the query output is not used).
hipError_t launch_ctx_kv(Ctx& c) {
  Model& m = c.drf;
  const spec_dims& d = m.d;
  {
    EmbedArgs p{c.st,   c.hist, c.embed, m.L[0].attn_norm, c.x, c.xg, c.ss, c.rcs, c.pos3, c.cs, m.axis,
                d.hidden, c.R, c.cap, (int)PASS_CTX, c.Mpad, d.head_dim, m.flat ? 1 : 0, c.V, c.mask_token,
                nullptr, c.feat};
    Timed t(c, SPEC_KERNEL_OTHER, 0);
    hipExtLaunchKernelGGL(k_embed, dim3(c.R, c.B), dim3(1024), (size_t)d.hidden * sizeof(float), c.stream, t.e0,
                          t.e1, 0, p);
    CK(hipGetLastError());
  }
  if (c.sg) {
    SgJob j = sg_job(c, m.sg_host[0]);
    j.kc = m.kc;
    j.vt = m.vt;
    Timed t(c, SPEC_KERNEL_OTHER, 0);
    return sg_launch(SG_ROPE, j, S(c), t.e0, t.e1);
  }
  return launch_qkv_rm(c, m, 0, m.kc, m.vt);
}

hipError_t launch_commit(Ctx& c, int32_t* acc, int32_t* committed, int32_t* ncommit, int32_t* fin) {
  {
    Timed t(c, SPEC_KERNEL_OTHER, 0);
    hipExtLaunchKernelGGL(k_commit, dim3(c.B), dim3(1), 0, c.stream, t.e0, t.e1, 0, c.st, c.hist, c.cap, c.K,
                          c.cfg.stop_token, c.cfg.max_new_tokens, acc, committed, ncommit, fin);
    CK(hipGetLastError());
  }
  if (c.cond) {
    Timed t(c, SPEC_KERNEL_OTHER, 0);
    hipExtLaunchKernelGGL(k_feat_commit, dim3(c.R, c.B), dim3(256), 0, c.stream, t.e0, t.e1, 0, c.st, c.fusedp,
                          kCondSplits, c.M, c.R, c.tgt.d.hidden, c.feat, c.cap);
    CK(hipGetLastError());
  }
  if (c.cross) CK(launch_ctx_kv(c));
  return hipSuccess;
}

hipError_t launch_logits_out(Ctx& c, void* d_logits) {
  if (!d_logits) return hipSuccess;
  return hipMemcpyAsync(d_logits, c.logits, (size_t)c.M * c.V * sizeof(bf16_t), hipMemcpyDeviceToDevice, c.stream);
}

}  // namespace specdec
