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

#include <algorithm>
#include <cmath>

#include "ctx.h"

namespace specdec {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr float kLog2e = 1.4426950408889634f;

__device__ __forceinline__ float bf2f(bf16_t h) { return __uint_as_float(((uint32_t)h) << 16); }

// float -> bfloat16, round to nearest even; NaN stays NaN.
__device__ __forceinline__ uint32_t f2bf_bits(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;
  u += 0x7fffu + ((u >> 16) & 1u);
  return u >> 16;
}
__device__ __forceinline__ bf16_t f2bf(float f) { return (bf16_t)f2bf_bits(f); }
__device__ __forceinline__ uint32_t pack2(float lo, float hi) { return f2bf_bits(lo) | (f2bf_bits(hi) << 16); }

__device__ __forceinline__ u32x4 ld16(const bf16_t* p) { return *reinterpret_cast<const u32x4*>(p); }
__device__ __forceinline__ u32x2 ld8(const bf16_t* p) { return *reinterpret_cast<const u32x2*>(p); }

__device__ __forceinline__ f32x4 mfma16x16x32(u32x4 a, u32x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c,
                                                 0, 0, 0);
}

// Block-wide sum of one float per thread (blockDim.x == 256).
__device__ float block_sum256(float v, float* sh) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  if (l == 0) sh[w] = v;
  __syncthreads();
  float t = sh[0] + sh[1] + sh[2] + sh[3];
  __syncthreads();
  return t;
}

// Argmax pair reduction: larger value wins, equal values go to the lower index.
__device__ __forceinline__ void amax_merge(float& v, int& i, float v2, int i2) {
  if (v2 > v || (v2 == v && i2 < i)) {
    v = v2;
    i = i2;
  }
}

// ---------------------------------------------------------------------------
// utility
// ---------------------------------------------------------------------------

__global__ void k_zero(u32x4* p, size_t n) {
  size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  for (; i < n; i += stride) p[i] = u32x4{0, 0, 0, 0};
}

// ---------------------------------------------------------------------------
// Prompt keys/values -> caches.  One thread per rotary pair of one slot of one
// kv head.  Keys are rotated with the model's positions (Eq. rope-3d with the
// axis assignment of Eq. axis-assign for the target; the slot index for the
// draft, Eq. flatrope-proj); values are stored transposed ([head_dim][cap]).
// ---------------------------------------------------------------------------
struct PrefixArgs {
  const bf16_t* k_pre;   // [P][nkv][D]
  const bf16_t* v;       // [P][nkv][D]
  bf16_t* kc;            // this layer & sequence: [nkv][cap][D]
  bf16_t* vt;            // [nkv][D][cap]
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
    *reinterpret_cast<uint32_t*>(a.kc + ((size_t)h * a.cap + s) * a.D + 2 * d) = pack2(re, ro);
    a.vt[((size_t)h * a.D + 2 * d) * a.cap + s] = a.v[src];
    a.vt[((size_t)h * a.D + 2 * d + 1) * a.cap + s] = a.v[src + 1];
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
// Row plan + embedding gather + first RMSNorm.  grid (R, B), 256 threads.
// Verify: rows at slots seq_len .. seq_len+K, tokens vtok.
// Draft: rows at slots draft_len .. seq_len+dstep (catch-up), tokens from the
// committed history up to seq_len and the draft's own proposals after it.
// ---------------------------------------------------------------------------
struct EmbedArgs {
  SeqState* st;
  const int32_t* hist;   // [B][cap]
  const bf16_t* E;       // [V][H]
  const bf16_t* g;       // first layer's attention-norm gain
  float* x;              // [Mpad][H]
  bf16_t* a;             // [Mpad][H]
  int H, R, cap, mode;
  float eps;
};

__global__ __launch_bounds__(256) void k_embed(EmbedArgs p) {
  __shared__ float sh[4];
  const int j = blockIdx.x, b = blockIdx.y;
  const SeqState& s = p.st[b];
  int base, count, tok = 0;
  if (p.mode == PASS_VERIFY) {
    base = s.seq_len;
    count = s.finished ? 0 : p.R;
    tok = s.vtok[j];
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
  }
  const size_t r = (size_t)b * p.R + j;
  float* xr = p.x + r * p.H;
  bf16_t* ar = p.a + r * p.H;
  if (j >= count) {
    for (int n = threadIdx.x; n < p.H; n += 256) {
      xr[n] = 0.f;
      ar[n] = 0;
    }
    return;
  }
  const bf16_t* er = p.E + (size_t)tok * p.H;
  float ss = 0.f;
  for (int n = threadIdx.x; n < p.H; n += 256) {
    const float v = bf2f(er[n]);
    xr[n] = v;
    ss += v * v;
  }
  const float inv = rsqrtf(block_sum256(ss, sh) / p.H + p.eps);
  for (int n = threadIdx.x; n < p.H; n += 256) ar[n] = f2bf(xr[n] * inv * bf2f(p.g[n]));
}

// ---------------------------------------------------------------------------
// Thin-M weight-streaming GEMV on MFMA:  y[m][n] = sum_k x[m][k] * W[n][k].
//
// A workgroup (4 waves) owns 16 consecutive weight rows and a k-range; each
// wave takes every 4th 32-wide k-step of that range.  With
// v_mfma_f32_16x16x32_bf16 the A operand is the weight tile: lane l holds
// W[n0 + (l&15)][k0 + 8*(l>>4) .. +8] (one 16-byte load), the B operand is
// x^T: lane l holds x[m = l&15][same 8 k] (rows beyond M are zero padding in
// the activation buffer), and the result lane l holds y[m = l&15][n0 +
// 4*(l>>4) + i], i = 0..3.  The four waves' results are summed through LDS in
// a fixed order (deterministic).  M up to 16*MB rows reuse each weight
// fragment MB times.
// ---------------------------------------------------------------------------
enum { EPI_PARTIAL = 0, EPI_ARGMAX = 1 };

struct GemvArgs {
  const bf16_t* w[3];
  int row0[3];           // first output row of each segment
  int nseg;
  int N, Kd;
  const bf16_t* x;       // [Mpad][ldx]
  int ldx, M, splits;
  float* part;           // EPI_PARTIAL: [splits][M][N]
  float* amax_v;         // EPI_ARGMAX: [N/16][Mpad]
  int32_t* amax_i;
  bf16_t* logits;        // EPI_ARGMAX: [Mpad][N] when the row's sequence wants logits
  SeqState* st;          // EPI_ARGMAX: flags
  int rps;               // rows per sequence (row m belongs to sequence m / rps)
  int mpad;
  int allow_logits;
};

template <int MB, int EPI, int U>
__global__ __launch_bounds__(256) void k_gemv(GemvArgs a) {
  __shared__ f32x4 red[4][MB][64];
  const int tile = blockIdx.x, split = blockIdx.y;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int n0 = tile * kTile;
  int sg = 0;
#pragma unroll
  for (int i = 1; i < 3; ++i)
    if (i < a.nseg && n0 >= a.row0[i]) sg = i;
  const int Kd = a.Kd;
  const int kq = 8 * (lane >> 4);
  const bf16_t* wp = a.w[sg] + (size_t)(n0 - a.row0[sg] + (lane & 15)) * Kd + kq;
  const bf16_t* xp[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) xp[mb] = a.x + (size_t)(mb * 16 + (lane & 15)) * a.ldx + kq;

  const int T = (Kd + 31) >> 5;       // 32-wide k-steps
  const int Tfull = Kd >> 5;          // steps with no tail
  const int s0 = (int)((long long)split * T / a.splits);
  const int s1 = (int)((long long)(split + 1) * T / a.splits);
  const int s1f = s1 < Tfull ? s1 : Tfull;

  f32x4 acc[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) acc[mb] = f32x4{0.f, 0.f, 0.f, 0.f};

  int st = s0 + wave;
  for (; st + 4 * (U - 1) < s1f; st += 4 * U) {
    u32x4 wv[U], xv[U][MB];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int k = (st + 4 * u) << 5;
      wv[u] = ld16(wp + k);
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) xv[u][mb] = ld16(xp[mb] + k);
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) acc[mb] = mfma16x16x32(wv[u], xv[u][mb], acc[mb]);
  }
  for (; st < s1; st += 4) {
    const int k = st << 5;
    const bool ok = k + kq < Kd;      // Kd % 8 == 0: a lane's 8 elements are all in or all out
    u32x4 wv = ok ? ld16(wp + k) : u32x4{0, 0, 0, 0};
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      u32x4 xv = ok ? ld16(xp[mb] + k) : u32x4{0, 0, 0, 0};
      acc[mb] = mfma16x16x32(wv, xv, acc[mb]);
    }
  }
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) red[wave][mb][lane] = acc[mb];
  __syncthreads();

  const int t = threadIdx.x;
  const int L = t >> 2, i = t & 3;
  if constexpr (EPI == EPI_PARTIAL) {
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      const float v = red[0][mb][L][i] + red[1][mb][L][i] + red[2][mb][L][i] + red[3][mb][L][i];
      const int m = mb * 16 + (L & 15);
      const int n = n0 + 4 * (L >> 4) + i;
      if (m < a.M) a.part[((size_t)split * a.M + m) * a.N + n] = v;
    }
  } else {
    __shared__ float lg[MB * 16][17];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      const float v = red[0][mb][L][i] + red[1][mb][L][i] + red[2][mb][L][i] + red[3][mb][L][i];
      const int m = mb * 16 + (L & 15);
      const int nn = 4 * (L >> 4) + i;
      lg[m][nn] = v;
      if (a.allow_logits && m < a.M && a.st[m / a.rps].want_logits) a.logits[(size_t)m * a.N + n0 + nn] = f2bf(v);
    }
    __syncthreads();
    if (t < MB * 16 && t < a.M) {
      float best = -INFINITY;
      int bi = n0;
      bool nan = false;
      for (int c = 0; c < 16; ++c) {
        float v = lg[t][c];
        if (v != v) {
          nan = true;
          v = -INFINITY;
        }
        if (v > best) {
          best = v;
          bi = n0 + c;
        }
      }
      a.amax_v[(size_t)tile * a.mpad + t] = best;
      a.amax_i[(size_t)tile * a.mpad + t] = bi;
      if (nan) atomicOr(&a.st[t / a.rps].err, ERR_NUMERIC);
    }
  }
}

// ---------------------------------------------------------------------------
// QKV finish: sum k-split partials, rotate q and k at the row's position,
// store q (bf16), append k to the key cache and v to the transposed value
// cache.  grid (R, B), 256 threads, one thread per (head, rotary pair).
// Target: angle theta_d * p_{a(d)}(slot) (Eq. mrope-phase); draft: theta_d *
// slot (Eq. flatrope-proj).  (cos, sin) come from the host-built table.
// ---------------------------------------------------------------------------
struct QkvArgs {
  const SeqState* st;
  const float* part;     // [S][M][N], N = (nq + 2 nkv) D
  int S, M, R;
  bf16_t* q;             // [Mpad][nq][D]
  bf16_t* kc;            // layer base [B][nkv][cap][D]
  bf16_t* vt;            // layer base [B][nkv][D][cap]
  const int32_t* pos3;   // [B][3][cap]
  const float2* cs;
  const int8_t* axis;
  int nq, nkv, D, cap, flat;
};

__global__ __launch_bounds__(256) void k_qkv_rope(QkvArgs p) {
  const int j = blockIdx.x, b = blockIdx.y;
  const SeqState& s = p.st[b];
  if (j >= s.count) return;
  const int slot = s.base + j;
  const int r = b * p.R + j;
  const int half = p.D / 2;
  const int N = (p.nq + 2 * p.nkv) * p.D;
  for (int pr = threadIdx.x; pr < N / 2; pr += 256) {
    const int col = 2 * pr;
    const int head = col / p.D;
    const int d = (col % p.D) >> 1;
    float e = 0.f, o = 0.f;
    for (int sp = 0; sp < p.S; ++sp) {
      const float* pp = p.part + ((size_t)sp * p.M + r) * N + col;
      e += pp[0];
      o += pp[1];
    }
    if (head < p.nq + p.nkv) {
      const int pos = p.flat ? slot : p.pos3[((size_t)b * 3 + p.axis[d]) * p.cap + slot];
      const float2 c = p.cs[(size_t)pos * half + d];
      const float re = e * c.x - o * c.y, ro = e * c.y + o * c.x;
      if (head < p.nq) {
        *reinterpret_cast<uint32_t*>(p.q + ((size_t)r * p.nq + head) * p.D + 2 * d) = pack2(re, ro);
      } else {
        const int h = head - p.nq;
        *reinterpret_cast<uint32_t*>(p.kc + (((size_t)b * p.nkv + h) * p.cap + slot) * p.D + 2 * d) =
            pack2(re, ro);
      }
    } else {
      const int h = head - p.nq - p.nkv;
      bf16_t* vp = p.vt + (((size_t)b * p.nkv + h) * p.D + 2 * d) * p.cap + slot;
      vp[0] = f2bf(e);
      vp[p.cap] = f2bf(o);
    }
  }
}

// ---------------------------------------------------------------------------
// Split-KV causal grouped-query attention on MFMA.
//
// grid (splits, kv_heads * row_blocks, B); a workgroup owns one kv head, up to
// 64 query rows (row = j*G + g: new row j, q head kvh*G + g) and the key range
// [split*chunk, (split+1)*chunk) clipped to the keys that exist.  Wave w owns
// query rows 16w..16w+15.
//
// Scores are computed transposed, S^T = K Q^T, so that lane l owns query row
// l&15: A = K tile (lane: key kb + (l&15), 8 dims), B = Q^T (lane: row l&15,
// same 8 dims) -> lane l holds scores of keys kb + 4*(l>>4) + i, i = 0..3.
// Two 16-key tiles give lane l the 8 keys {4g..4g+3, 16+4g..16+4g+3}
// (g = l>>4) of its row, which is exactly a B operand P^T for O^T = V^T P^T
// when the 32 k-slots are mapped to keys in that order; the A operand V^T is
// read from the transposed value cache as two 8-byte loads per lane.  Online
// softmax statistics are per lane (its row); the row max crosses the four lane
// groups with two xor-shuffles.
// ---------------------------------------------------------------------------
struct AttnArgs {
  const SeqState* st;
  const bf16_t* q;       // [Mpad][nq][D]
  const bf16_t* kc;      // layer base [B][nkv][cap][D]
  const bf16_t* vt;      // layer base [B][nkv][D][cap]
  float* op;             // [splits][B][nq][R][D]
  float* mp;             // [splits][B][nq][R]
  float* lp;
  int nq, nkv, G, R, B, cap, chunk, row_blocks;
  float scale_log2;      // log2(e) / sqrt(D)
};

template <int D>
__global__ __launch_bounds__(256) void k_attn(AttnArgs a) {
  const int split = blockIdx.x;
  const int kvh = blockIdx.y / a.row_blocks, rb = blockIdx.y % a.row_blocks;
  const int b = blockIdx.z;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int g4 = lane >> 4;
  const SeqState& s = a.st[b];
  const int count = s.count, base = s.base;
  const int rows = count * a.G;
  const int wrow0 = rb * 64 + wave * 16;
  if (wrow0 >= rows) return;                        // wave-uniform
  const int qr = wrow0 + (lane & 15);
  const bool rvalid = qr < rows;
  const int j = rvalid ? qr / a.G : 0;
  const int hq = kvh * a.G + (rvalid ? qr % a.G : 0);
  const int kv_end = base + count;
  const int k0 = split * a.chunk;
  const int k1 = min(k0 + a.chunk, kv_end);
  const int vis_end = base + j + 1;
  const size_t oi = (((size_t)split * a.B + b) * a.nq + hq) * a.R + j;

  if (k0 >= k1) {                                   // no keys in this split
    if (rvalid && g4 == 0) {
      a.mp[oi] = -INFINITY;
      a.lp[oi] = 0.f;
    }
    if (rvalid) {
      float* op = a.op + oi * D;
      for (int d = g4 * 4; d < D; d += 16) *reinterpret_cast<f32x4*>(op + d) = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    return;
  }

  u32x4 qf[D / 32];
  {
    const bf16_t* qp = a.q + ((size_t)(b * a.R + j) * a.nq + hq) * D + 8 * g4;
#pragma unroll
    for (int t = 0; t < D / 32; ++t) qf[t] = rvalid ? ld16(qp + 32 * t) : u32x4{0, 0, 0, 0};
  }
  const bf16_t* Kb = a.kc + ((size_t)b * a.nkv + kvh) * a.cap * D;
  const bf16_t* Vb = a.vt + ((size_t)b * a.nkv + kvh) * D * a.cap;

  float m_run = -INFINITY, l_run = 0.f;
  f32x4 o[D / 16];
#pragma unroll
  for (int dt = 0; dt < D / 16; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int kb = k0; kb < k1; kb += kKeyBlock) {
    f32x4 sc[2];
#pragma unroll
    for (int h2 = 0; h2 < 2; ++h2) {
      const bf16_t* kp = Kb + (size_t)(kb + 16 * h2 + (lane & 15)) * D + 8 * g4;
      f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int t = 0; t < D / 32; ++t) acc = mfma16x16x32(ld16(kp + 32 * t), qf[t], acc);
      sc[h2] = acc;
    }
    float p[8];
    float bm = -INFINITY;
#pragma unroll
    for (int h2 = 0; h2 < 2; ++h2)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int key = kb + 16 * h2 + 4 * g4 + i;
        const bool ok = rvalid && key < k1 && key < vis_end;
        const float v = ok ? sc[h2][i] * a.scale_log2 : -INFINITY;
        p[h2 * 4 + i] = v;
        bm = fmaxf(bm, v);
      }
    bm = fmaxf(bm, __shfl_xor(bm, 16));
    bm = fmaxf(bm, __shfl_xor(bm, 32));
    const float m_new = fmaxf(m_run, bm);
    const float alpha = (m_run == -INFINITY) ? 0.f : exp2f(m_run - m_new);
    float ps = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      p[i] = (p[i] == -INFINITY) ? 0.f : exp2f(p[i] - m_new);
      ps += p[i];
    }
    l_run = l_run * alpha + ps;
    m_run = m_new;
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt) o[dt] *= alpha;
    const u32x4 pb = u32x4{pack2(p[0], p[1]), pack2(p[2], p[3]), pack2(p[4], p[5]), pack2(p[6], p[7])};
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt) {
      const bf16_t* vp = Vb + (size_t)(16 * dt + (lane & 15)) * a.cap + kb + 4 * g4;
      const u32x2 lo = ld8(vp), hi = ld8(vp + 16);
      o[dt] = mfma16x16x32(u32x4{lo.x, lo.y, hi.x, hi.y}, pb, o[dt]);
    }
  }
  l_run += __shfl_xor(l_run, 16);
  l_run += __shfl_xor(l_run, 32);
  if (rvalid) {
    float* op = a.op + oi * D;
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt) *reinterpret_cast<f32x4*>(op + 16 * dt + 4 * g4) = o[dt];
    if (g4 == 0) {
      a.mp[oi] = m_run;
      a.lp[oi] = l_run;
    }
  }
}

// Merge the splits of each (row, q head): o = sum_s 2^(m_s - M) O_s / sum_s
// 2^(m_s - M) l_s.  grid (R, B), 256 threads.
struct CombineArgs {
  const SeqState* st;
  const float *op, *mp, *lp;
  bf16_t* o;             // [Mpad][nq*D]
  int nq, D, R, B, chunk;
};

__global__ __launch_bounds__(256) void k_attn_combine(CombineArgs a) {
  extern __shared__ float coef[];   // [nq][ns]
  const int j = blockIdx.x, b = blockIdx.y;
  const SeqState& s = a.st[b];
  if (j >= s.count) return;
  const int vis_end = s.base + j + 1;
  const int ns = (vis_end + a.chunk - 1) / a.chunk;   // splits holding keys this row sees
  for (int h = threadIdx.x; h < a.nq; h += 256) {
    float M = -INFINITY;
    for (int sp = 0; sp < ns; ++sp) M = fmaxf(M, a.mp[(((size_t)sp * a.B + b) * a.nq + h) * a.R + j]);
    float L = 0.f;
    for (int sp = 0; sp < ns; ++sp) {
      const size_t i = (((size_t)sp * a.B + b) * a.nq + h) * a.R + j;
      const float w = exp2f(a.mp[i] - M);
      coef[h * ns + sp] = w;
      L += w * a.lp[i];
    }
    const float inv = 1.f / L;
    for (int sp = 0; sp < ns; ++sp) coef[h * ns + sp] *= inv;
  }
  __syncthreads();
  const int r = b * a.R + j;
  for (int e = threadIdx.x; e < a.nq * a.D; e += 256) {
    const int h = e / a.D, d = e % a.D;
    float v = 0.f;
    for (int sp = 0; sp < ns; ++sp)
      v += coef[h * ns + sp] * a.op[((((size_t)sp * a.B + b) * a.nq + h) * a.R + j) * a.D + d];
    a.o[(size_t)r * a.nq * a.D + e] = f2bf(v);
  }
}

// ---------------------------------------------------------------------------
// Residual add of k-split partials + RMSNorm into the next GEMV input.
// select_last: write only the row count-1 of each sequence, to out row b
// (the draft proposes from its last row only).  grid (R, B), 256 threads.
// ---------------------------------------------------------------------------
struct NormArgs {
  const SeqState* st;
  const float* part;     // [S][M][H] or null
  int S, M, R, H;
  float* x;
  const bf16_t* g;
  bf16_t* out;
  int select_last;
  float eps;
};

__global__ __launch_bounds__(256) void k_resid_norm(NormArgs p) {
  __shared__ float sh[4];
  const int j = blockIdx.x, b = blockIdx.y;
  const int count = p.st[b].count;
  if (j >= count) return;
  if (p.select_last && j != count - 1) return;
  const int r = b * p.R + j;
  float* xr = p.x + (size_t)r * p.H;
  float ss = 0.f;
  for (int n = threadIdx.x; n < p.H; n += 256) {
    float v = xr[n];
    if (p.part)
      for (int sp = 0; sp < p.S; ++sp) v += p.part[((size_t)sp * p.M + r) * p.H + n];
    xr[n] = v;
    ss += v * v;
  }
  const float inv = rsqrtf(block_sum256(ss, sh) / p.H + p.eps);
  bf16_t* orow = p.out + (size_t)(p.select_last ? b : r) * p.H;
  for (int n = threadIdx.x; n < p.H; n += 256) orow[n] = f2bf(xr[n] * inv * bf2f(p.g[n]));
}

// SwiGLU finish: u = silu(gate) * up from the k-split partials of the fused
// [gate; up] GEMV.  grid (R, B).
struct SwigluArgs {
  const SeqState* st;
  const float* part;     // [S][M][2F]
  int S, M, R, F;
  bf16_t* u;             // [Mpad][F]
};

__global__ __launch_bounds__(256) void k_swiglu(SwigluArgs p) {
  const int j = blockIdx.x, b = blockIdx.y;
  if (j >= p.st[b].count) return;
  const int r = b * p.R + j;
  const size_t N = 2 * (size_t)p.F;
  for (int n = threadIdx.x; n < p.F; n += 256) {
    float gt = 0.f, up = 0.f;
    for (int sp = 0; sp < p.S; ++sp) {
      const float* pp = p.part + ((size_t)sp * p.M + r) * N;
      gt += pp[n];
      up += pp[p.F + n];
    }
    const float silu = gt / (1.f + expf(-gt));
    p.u[(size_t)r * p.F + n] = f2bf(silu * up);
  }
}

// ---------------------------------------------------------------------------
// Greedy tokens of the verify rows and the accept length (Eq. verify,
// Eq. accept), plus the commit list cut at a stop token or the budget.
// grid B, 256 threads.
// ---------------------------------------------------------------------------
__device__ void reduce_amax_row(const float* av, const int32_t* ai, int ntiles, int mpad, int row, float* shv,
                                int* shi, float& bv, int& bi) {
  float v = -INFINITY;
  int i = 0x7fffffff;
  for (int t = threadIdx.x; t < ntiles; t += 256) amax_merge(v, i, av[(size_t)t * mpad + row], ai[(size_t)t * mpad + row]);
  shv[threadIdx.x] = v;
  shi[threadIdx.x] = i;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if (threadIdx.x < o) {
      float v2 = shv[threadIdx.x + o];
      int i2 = shi[threadIdx.x + o];
      float v1 = shv[threadIdx.x];
      int i1 = shi[threadIdx.x];
      amax_merge(v1, i1, v2, i2);
      shv[threadIdx.x] = v1;
      shi[threadIdx.x] = i1;
    }
    __syncthreads();
  }
  bv = shv[0];
  bi = shi[0];
  __syncthreads();
}

struct AcceptArgs {
  SeqState* st;
  const float* amax_v;
  const int32_t* amax_i;
  int ntiles, mpad, R, K, stop, max_new;
};

__global__ __launch_bounds__(256) void k_accept(AcceptArgs p) {
  __shared__ float shv[256];
  __shared__ int shi[256];
  const int b = blockIdx.x;
  SeqState& s = p.st[b];
  if (s.finished) {
    if (threadIdx.x == 0) {
      s.n_commit = 0;
      s.fin_pending = 1;
    }
    return;
  }
  for (int j = 0; j < p.R; ++j) {
    float bv;
    int bi;
    reduce_amax_row(p.amax_v, p.amax_i, p.ntiles, p.mpad, b * p.R + j, shv, shi, bv, bi);
    if (threadIdx.x == 0) s.rstar[j] = bi;
  }
  if (threadIdx.x == 0) {
    int l = 0;
    while (l < p.K && s.vtok[l + 1] == s.rstar[l]) ++l;
    int c = l + 1;
    for (int i = 0; i < l; ++i) s.committed[i] = s.vtok[i + 1];
    s.committed[l] = s.rstar[l];
    int fin = 0;
    if (p.stop >= 0)
      for (int i = 0; i < c; ++i)
        if (s.committed[i] == p.stop) {
          c = i + 1;
          fin = 1;
          break;
        }
    const int rem = p.max_new - s.n_gen;
    if (c >= rem) {
      c = rem;
      fin = 1;
    }
    s.accept_len = l;
    s.n_commit = c;
    s.fin_pending = fin;
  }
}

// Draft proposal: argmax of the last row of the draft step.  grid B.
struct PickArgs {
  SeqState* st;
  const float* amax_v;
  const int32_t* amax_i;
  int ntiles, mpad;
};

__global__ __launch_bounds__(256) void k_draft_pick(PickArgs p) {
  __shared__ float shv[256];
  __shared__ int shi[256];
  const int b = blockIdx.x;
  SeqState& s = p.st[b];
  if (s.count == 0) return;
  float bv;
  int bi;
  reduce_amax_row(p.amax_v, p.amax_i, p.ntiles, p.mpad, b, shv, shi, bv, bi);
  if (threadIdx.x == 0) {
    s.props[s.dstep] = bi;
    s.draft_len = s.base + s.count;
    s.dstep += 1;
  }
}

__global__ void k_draft_out(const SeqState* st, int32_t* out, int K, int col) {
  const SeqState& s = st[blockIdx.x];
  out[blockIdx.x * K + col] = (s.count > 0 && s.dstep == col + 1) ? s.props[col] : -1;
}

// Commit (Eq. commit): append the committed tokens, advance the lengths, roll
// the draft back to the first slot whose input differs from the committed
// sequence (never past the new pending token).  grid B, 1 thread.
__global__ void k_commit(SeqState* st, int32_t* hist, int cap, int K, int32_t* o_acc, int32_t* o_com,
                         int32_t* o_n, int32_t* o_fin) {
  const int b = blockIdx.x;
  SeqState& s = st[b];
  int c = 0, acc = 0;
  if (!s.finished) {
    c = s.n_commit;
    acc = s.accept_len;
    const int n = s.seq_len;
    for (int i = 0; i < c; ++i) hist[(size_t)b * cap + n + 1 + i] = s.committed[i];
    int x = n + 1;
    while (x < s.draft_len && (x - n - 1) < c && s.props[x - n - 1] == s.committed[x - n - 1]) ++x;
    s.draft_len = min(min(s.draft_len, x), n + c);
    s.seq_len = n + c;
    s.pending = s.committed[c - 1];
    s.n_gen += c;
    s.finished = s.fin_pending;
  }
  s.dstep = 0;
  if (o_acc) o_acc[b] = acc;
  if (o_n) o_n[b] = c;
  if (o_fin) o_fin[b] = s.finished;
  if (o_com)
    for (int i = 0; i <= K; ++i) o_com[b * (K + 1) + i] = i < c ? s.committed[i] : -1;
}

// ---------------------------------------------------------------------------
// host-side launch helpers
// ---------------------------------------------------------------------------

int pick_splits(int N, int Kd) {
  const int tiles = (N + kTile - 1) / kTile;
  const int steps = (Kd + 31) / 32;
  int s = (1024 + tiles - 1) / tiles;
  const int smax = std::max(1, steps / 8);
  return std::max(1, std::min(s, smax));
}

namespace {

struct Timed {
  Ctx& c;
  int kind;
  double bytes;
  hipEvent_t e1 = nullptr;
  Timed(Ctx& c_, int kind_, double bytes_) : c(c_), kind(kind_), bytes(bytes_) {
    if (!c.timing) return;
    if (c.ev_used + 2 > c.ev_pool.size()) {
      for (int i = 0; i < 256; ++i) {
        hipEvent_t e;
        if (hipEventCreate(&e) == hipSuccess) c.ev_pool.push_back(e);
      }
    }
    if (c.ev_used + 2 > c.ev_pool.size()) return;
    hipEvent_t e0 = c.ev_pool[c.ev_used++];
    e1 = c.ev_pool[c.ev_used++];
    (void)hipEventRecord(e0, c.stream);
    c.trec.push_back(TimingRec{kind, bytes, e0, e1});
  }
  ~Timed() {
    if (e1) (void)hipEventRecord(e1, c.stream);
  }
};

hipStream_t S(Ctx& c) { return c.stream; }

template <int EPI>
hipError_t gemv_dispatch(Ctx& c, const GemvArgs& g, int mb, int kind, double bytes) {
  dim3 grid((g.N + kTile - 1) / kTile, g.splits);
  Timed t(c, kind, bytes);
  switch (mb) {
    case 1: hipLaunchKernelGGL((k_gemv<1, EPI, 4>), grid, dim3(256), 0, S(c), g); break;
    case 2: hipLaunchKernelGGL((k_gemv<2, EPI, 4>), grid, dim3(256), 0, S(c), g); break;
    case 3: hipLaunchKernelGGL((k_gemv<3, EPI, 2>), grid, dim3(256), 0, S(c), g); break;
    case 4: hipLaunchKernelGGL((k_gemv<4, EPI, 2>), grid, dim3(256), 0, S(c), g); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// Algorithmic bytes of a GEMV launch: weights once, activations in, fp32 out.
double gemv_bytes(int N, int Kd, int M, int S) {
  return 2.0 * N * Kd + 2.0 * M * Kd + 4.0 * S * M * N;
}

hipError_t gemv(Ctx& c, const bf16_t* w0, int n0, const bf16_t* w1, int n1, const bf16_t* w2, int n2, int Kd,
                const bf16_t* x, int M, int S) {
  GemvArgs g{};
  g.w[0] = w0;
  g.w[1] = w1;
  g.w[2] = w2;
  g.row0[0] = 0;
  g.row0[1] = n0;
  g.row0[2] = n0 + n1;
  g.nseg = w2 ? 3 : (w1 ? 2 : 1);
  g.N = n0 + n1 + n2;
  g.Kd = Kd;
  g.x = x;
  g.ldx = Kd;
  g.M = M;
  g.splits = S;
  g.part = c.part;
  return gemv_dispatch<EPI_PARTIAL>(c, g, (M + 15) / 16, SPEC_KERNEL_GEMV, gemv_bytes(g.N, Kd, M, S));
}

#define CK(x)                               \
  do {                                      \
    hipError_t e_ = (x);                    \
    if (e_ != hipSuccess) return e_;        \
  } while (0)

hipError_t run_layer(Ctx& c, Model& m, int li, int M, bool last_layer, const bf16_t* next_gain,
                     bf16_t* next_out, bool select_last) {
  const spec_dims& d = m.d;
  const int H = d.hidden, D = d.head_dim, nq = d.q_heads, nkv = d.kv_heads, F = d.ffn;
  const LayerW& w = m.L[li];
  const size_t kvl = m.kv_layer;
  bf16_t* kc = m.kc + kvl * li;
  bf16_t* vt = m.vt + kvl * li;
  const dim3 rows(c.R, c.B);

  // q, k, v
  CK(gemv(c, w.wq, nq * D, w.wk, nkv * D, w.wv, nkv * D, H, c.a, M, m.s_qkv));
  {
    QkvArgs p{c.st, c.part, m.s_qkv, M, c.R, c.q, kc, vt, c.pos3, c.cs, m.axis, nq, nkv, D, c.cap, m.flat ? 1 : 0};
    Timed t(c, SPEC_KERNEL_OTHER, 0);
    hipLaunchKernelGGL(k_qkv_rope, rows, dim3(256), 0, S(c), p);
    CK(hipGetLastError());
  }
  // attention
  {
    const int G = nq / nkv;
    const int rb = (c.R * G + 63) / 64;
    AttnArgs p{c.st, c.q, kc, vt, c.op, c.mp, c.lp, nq, nkv, G, c.R, c.B, c.cap, c.attn_chunk, rb,
               kLog2e / sqrtf((float)D)};
    dim3 grid(c.attn_splits, nkv * rb, c.B);
    // KV bytes of the cached prefix read by every sequence (upper bound: capacity is not read)
    Timed t(c, SPEC_KERNEL_ATTN, 0);
    if (D == 128)
      hipLaunchKernelGGL(k_attn<128>, grid, dim3(256), 0, S(c), p);
    else
      hipLaunchKernelGGL(k_attn<64>, grid, dim3(256), 0, S(c), p);
    CK(hipGetLastError());
    CombineArgs cb{c.st, c.op, c.mp, c.lp, c.o, nq, D, c.R, c.B, c.attn_chunk};
    Timed t2(c, SPEC_KERNEL_OTHER, 0);
    hipLaunchKernelGGL(k_attn_combine, rows, dim3(256), (size_t)nq * c.attn_splits * sizeof(float), S(c), cb);
    CK(hipGetLastError());
  }
  // o projection + residual + ffn norm
  CK(gemv(c, w.wo, H, nullptr, 0, nullptr, 0, nq * D, c.o, M, m.s_o));
  {
    NormArgs p{c.st, c.part, m.s_o, M, c.R, H, c.x, w.ffn_norm, c.a, 0, d.rms_eps};
    Timed t(c, SPEC_KERNEL_OTHER, 0);
    hipLaunchKernelGGL(k_resid_norm, rows, dim3(256), 0, S(c), p);
    CK(hipGetLastError());
  }
  // SwiGLU
  CK(gemv(c, w.wg, F, w.wu, F, nullptr, 0, H, c.a, M, m.s_gu));
  {
    SwigluArgs p{c.st, c.part, m.s_gu, M, c.R, F, c.u};
    Timed t(c, SPEC_KERNEL_OTHER, 0);
    hipLaunchKernelGGL(k_swiglu, rows, dim3(256), 0, S(c), p);
    CK(hipGetLastError());
  }
  // down projection + residual + next norm
  CK(gemv(c, w.wd, H, nullptr, 0, nullptr, 0, F, c.u, M, m.s_down));
  {
    NormArgs p{c.st, c.part, m.s_down, M, c.R, H, c.x, next_gain, next_out, select_last ? 1 : 0, d.rms_eps};
    Timed t(c, SPEC_KERNEL_OTHER, 0);
    hipLaunchKernelGGL(k_resid_norm, rows, dim3(256), 0, S(c), p);
    CK(hipGetLastError());
  }
  (void)last_layer;
  return hipSuccess;
}

}  // namespace

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
  const size_t per_seq = (size_t)d.kv_heads * c.cap * d.head_dim;
  PrefixArgs p{k_pre,
               v,
               m.kc + kvl * layer + per_seq * b,
               m.vt + kvl * layer + per_seq * b,
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
  hipLaunchKernelGGL(k_stage_verify, dim3(c.B), dim3(64), 0, c.stream, c.st, d_override, c.K, c.V, want_logits);
  return hipGetLastError();
}

hipError_t launch_forward(Ctx& c, PassMode mode) {
  Model& m = mode == PASS_VERIFY ? c.tgt : c.drf;
  const spec_dims& d = m.d;
  const int M = c.M;
  {
    EmbedArgs p{c.st, c.hist, c.embed, m.L[0].attn_norm, c.x, c.a, d.hidden, c.R, c.cap, (int)mode, d.rms_eps};
    Timed t(c, SPEC_KERNEL_OTHER, 0);
    hipLaunchKernelGGL(k_embed, dim3(c.R, c.B), dim3(256), 0, c.stream, p);
    CK(hipGetLastError());
  }
  const bool draft = mode == PASS_DRAFT;
  for (int li = 0; li < d.layers; ++li) {
    const bool last = li + 1 == d.layers;
    const bf16_t* g = last ? m.final_norm : m.L[li + 1].attn_norm;
    bf16_t* out = (last && draft) ? c.a_last : c.a;
    CK(run_layer(c, m, li, M, last, g, out, last && draft));
  }
  // LM head with the fused per-tile argmax
  GemvArgs g{};
  g.w[0] = c.embed;
  g.row0[0] = 0;
  g.nseg = 1;
  g.N = c.V;
  g.Kd = d.hidden;
  g.x = draft ? c.a_last : c.a;
  g.ldx = d.hidden;
  g.M = draft ? c.B : M;
  g.splits = 1;
  g.amax_v = c.amax_v;
  g.amax_i = c.amax_i;
  g.logits = c.logits;
  g.st = c.st;
  g.rps = draft ? 1 : c.R;
  g.mpad = c.Mpad;
  g.allow_logits = draft ? 0 : 1;
  CK(gemv_dispatch<EPI_ARGMAX>(c, g, (g.M + 15) / 16, SPEC_KERNEL_LMHEAD,
                               2.0 * c.V * d.hidden + 2.0 * g.M * d.hidden + 8.0 * (c.V / 16) * g.M));
  const int ntiles = c.V / kTile;
  Timed t(c, SPEC_KERNEL_OTHER, 0);
  if (!draft) {
    AcceptArgs p{c.st, c.amax_v, c.amax_i, ntiles, c.Mpad, c.R, c.K, c.cfg.stop_token, c.cfg.max_new_tokens};
    hipLaunchKernelGGL(k_accept, dim3(c.B), dim3(256), 0, c.stream, p);
  } else {
    PickArgs p{c.st, c.amax_v, c.amax_i, ntiles, c.Mpad};
    hipLaunchKernelGGL(k_draft_pick, dim3(c.B), dim3(256), 0, c.stream, p);
  }
  return hipGetLastError();
}

hipError_t launch_draft_out(Ctx& c, int32_t* d_tokens) {
  if (!d_tokens) return hipSuccess;
  hipLaunchKernelGGL(k_draft_out, dim3(c.B), dim3(1), 0, c.stream, c.st, d_tokens, c.K, c.dsteps);
  return hipGetLastError();
}

hipError_t launch_commit(Ctx& c, int32_t* acc, int32_t* committed, int32_t* ncommit, int32_t* fin) {
  Timed t(c, SPEC_KERNEL_OTHER, 0);
  hipLaunchKernelGGL(k_commit, dim3(c.B), dim3(1), 0, c.stream, c.st, c.hist, c.cap, c.K, acc, committed, ncommit,
                     fin);
  return hipGetLastError();
}

hipError_t launch_logits_out(Ctx& c, void* d_logits) {
  if (!d_logits) return hipSuccess;
  return hipMemcpyAsync(d_logits, c.logits, (size_t)c.M * c.V * sizeof(bf16_t), hipMemcpyDeviceToDevice, c.stream);
}

}  // namespace specdec
