// Persistent forward pass on gfx950: every decoder layer of one pass (a verify
// of K+1 rows per sequence, or one draft step) in a single launch.
//
// One workgroup per compute unit, 8 waves (two per SIMD, so each may hold 256
// registers).  Wave 0 is the control wave: it never streams weights, runs the
// device-wide barriers between phases and finishes the down projection's
// tiles; waves 1..7 stream weights, 16 loads of 16 bytes per lane in flight.  Because
// the control wave has no weight loads outstanding, its barrier round trips
// do not queue behind them (vector memory counters complete in order).
//
// Per layer:  QKV (+1/rms, rotary, KV append)  | attention partials (split-KV)
//           | combine                          | O (+ residual, FFN-norm input)
//           | gate/up (+ SwiGLU)               | down partials, and the last
//             k-split of every output tile adds the residual and writes the
//             next norm's input
// with a device-wide barrier after each phase.
//
// Memory coherence across the XCDs inside one launch (each XCD has its own
// L2): everything another workgroup reads later in the launch is stored with
// agent-scope relaxed atomic stores, which write through to memory; buffers
// that are read at an address whose older contents may still sit in this
// XCD's L2 (the residual stream, split partials) are read with agent-scope
// relaxed atomic loads; the activation inputs of the GEMV phases and the
// queries live in per-layer buffers that are read once per launch, so plain
// loads are safe and share each XCD's L2.  Every barrier wait is bounded: a
// timeout sets ERR_SYNC and later waits of the launch are skipped, so the
// launch always ends.
#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>

#include <algorithm>
#include <cmath>

#include "ctx.h"
#include "device.h"
#include "pass.h"

namespace specdec {

namespace {

constexpr int kWorkers = kPassWaves - 1;   // weight-streaming waves 1..7
constexpr int kSpinLimit = 1 << 16;        // polls per barrier before giving up

// ---- global-address-space accesses ---------------------------------------------
// Pointers read from device memory are generic; flat instructions would also
// count on the LDS counter, so a wait for an LDS read would wait for every
// weight load in flight.  These casts keep global accesses global.
#define GLOBAL_AS __attribute__((address_space(1)))
__device__ __forceinline__ u32x4 ldg16(const bf16_t* p) {
  return *(const GLOBAL_AS u32x4*)(p);
}
template <class T>
__device__ __forceinline__ T ldg(const T* p) {
  return *(const GLOBAL_AS T*)(p);
}

// ---- agent-coherent accesses ------------------------------------------------
__device__ __forceinline__ void st_u32(void* p, uint32_t v) {
  __hip_atomic_store((GLOBAL_AS uint32_t*)(p), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_u16(void* p, uint16_t v) {
  __hip_atomic_store((GLOBAL_AS uint16_t*)(p), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_f32(float* p, float v) { st_u32(p, __float_as_uint(v)); }
__device__ __forceinline__ uint32_t ld_u32(const void* p) {
  return __hip_atomic_load((const GLOBAL_AS uint32_t*)(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float ld_f32(const float* p) { return __uint_as_float(ld_u32(p)); }
__device__ __forceinline__ void st_f32x4(float* p, f32x4 v) {
  GLOBAL_AS uint64_t* q = (GLOBAL_AS uint64_t*)(p);
  __hip_atomic_store(q, (uint64_t)__float_as_uint(v.x) | ((uint64_t)__float_as_uint(v.y) << 32), __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
  __hip_atomic_store(q + 1, (uint64_t)__float_as_uint(v.z) | ((uint64_t)__float_as_uint(v.w) << 32), __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
}

// A value the compiler must treat as unknown at this point: keeps per-tile
// scalars inside the tile loop instead of hoisting them for the whole launch.
// (v must be wave-uniform.)
__device__ __forceinline__ int opaque_s(int v) {
  v = __builtin_amdgcn_readfirstlane(v);
  asm volatile("" : "+s"(v));
  return v;
}

// (p must be wave-uniform.)
__device__ __forceinline__ const bf16_t* opaque_p(const bf16_t* p) {
  const uint64_t u = reinterpret_cast<uint64_t>(p);
  int lo = __builtin_amdgcn_readfirstlane((int)(uint32_t)u), hi = __builtin_amdgcn_readfirstlane((int)(u >> 32));
  asm volatile("" : "+s"(lo), "+s"(hi));
  return reinterpret_cast<const bf16_t*>(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}

constexpr int kBufWord3 = 0x00020000;   // raw buffer resource, 32-bit data (gfx9 family)
__device__ __forceinline__ f32x4 ld_f32x4(const float* p) {
  const GLOBAL_AS uint64_t* q = (const GLOBAL_AS uint64_t*)(p);
  const uint64_t a = __hip_atomic_load(q, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  const uint64_t b = __hip_atomic_load(q + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return f32x4{__uint_as_float((uint32_t)a), __uint_as_float((uint32_t)(a >> 32)), __uint_as_float((uint32_t)b),
               __uint_as_float((uint32_t)(b >> 32))};
}

// ---- device-wide barrier ----------------------------------------------------
// Layout of PassArgs::bar (unsigned words): [0] top counter, group g's counter
// at 64 * (1 + g) and its release flag 32 words later (8 groups, one 256-byte
// block each), [kBarDone] workgroups finished (the last one resets all).
constexpr int kBarGroups = 8;
constexpr int kBarDone = 64 * (1 + kBarGroups);

__device__ __forceinline__ bool spin_until(const unsigned* p, unsigned target) {
  for (int i = 0; i < kSpinLimit; ++i) {
    if (__hip_atomic_load((const GLOBAL_AS unsigned*)(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >= target)
      return true;
    __builtin_amdgcn_s_sleep(1);
  }
  return false;
}

// Called by all threads.  Every thread first waits for its own stores (no
// loads are outstanding then); `prefetch` may then issue the next phase's
// weight loads, which stay in flight: the rest uses raw workgroup barriers,
// which do not wait for memory.  Wave 0 (no weight loads) runs the
// device-wide part.
template <class Prefetch>
__device__ __forceinline__ void grid_sync(const PassArgs& a, unsigned gen, bool& failed, Prefetch&& prefetch) {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  prefetch();
  __builtin_amdgcn_s_barrier();
  if (threadIdx.x == 0 && !failed) {
    const unsigned G = gridDim.x;
    const unsigned grp = blockIdx.x % kBarGroups;
    const unsigned gsize = (G - grp + kBarGroups - 1) / kBarGroups;
    unsigned* gc = a.bar + 64 * (1 + grp);
    unsigned* gf = gc + 32;
    const unsigned old = __hip_atomic_fetch_add((GLOBAL_AS unsigned*)(gc), 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    bool ok;
    if (old + 1 == gen * gsize) {
      __hip_atomic_fetch_add((GLOBAL_AS unsigned*)(a.bar), 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      ok = spin_until(a.bar, gen * (unsigned)min((int)G, kBarGroups));
      __hip_atomic_store((GLOBAL_AS unsigned*)(gf), gen, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    } else {
      ok = spin_until(gf, gen);
    }
    if (!ok) {
      failed = true;
      atomicOr(&a.st[0].err, ERR_SYNC);
    }
  }
  __builtin_amdgcn_s_barrier();
}

__device__ __forceinline__ void grid_sync(const PassArgs& a, unsigned gen, bool& failed) {
  grid_sync(a, gen, failed, [] {});
}

// The last workgroup to finish clears every barrier word for the next launch.
__device__ __forceinline__ void grid_done(const PassArgs& a) {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __syncthreads();
  if (threadIdx.x == 0) {
    const unsigned old =
        __hip_atomic_fetch_add((GLOBAL_AS unsigned*)(a.bar + kBarDone), 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (old + 1 == gridDim.x) {
      for (int i = 0; i <= kBarDone; ++i) st_u32(a.bar + i, 0u);
    }
  }
}

// ---- rows -------------------------------------------------------------------
__device__ __forceinline__ uint64_t live_rows(const PassArgs& a) {
  uint64_t live = 0;
  const int nseq = (a.M + a.rps - 1) / a.rps;
  for (int b = 0; b < nseq; ++b) {
    const int n = min(a.st[b].count, a.rps);
    if (n > 0) live |= ((1ull << n) - 1ull) << (b * a.rps);
  }
  return live;
}

// ---- persistent GEMV phase --------------------------------------------------
// y[m][n] = sum_k x[m][k] W[n][k] over 16-row tiles.  The grid is split into
// `splits` groups, one per k-range; workgroup g of its group streams tiles
// g, g + gsize, ... with the next tile's weights in flight.  Worker wave w
// (1..7) owns k-steps [s0 + (w-1) chunk, ...).  x rows of the k-range are
// staged in LDS once.  After the 7 partial tiles are summed the epilogue runs
// on the complete 16-column tile.
enum { PE_ROPE = 0, PE_RESID = 1, PE_SWIGLU = 2, PE_DOWN = 3 };


// Work split of one GEMV phase for this thread's workgroup and wave.
struct Geom {
  int gsize, split, g, Kd, kq, s0, s1, w0, nw_all, ncol, nwork;
};

template <int EPI>
__device__ __forceinline__ Geom gemv_geom(const GemvJob& j) {
  constexpr bool kPair = EPI == PE_SWIGLU;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  Geom q;
  q.gsize = gridDim.x / j.splits;
  q.split = blockIdx.x / q.gsize;
  q.g = blockIdx.x % q.gsize;
  q.Kd = j.Kd;
  q.kq = 8 * (lane >> 4);
  const int T = (j.Kd + 31) >> 5;
  q.s0 = q.split * T / j.splits;                   // T <= 2^16 and splits <= 2^10: 32-bit exact
  q.s1 = (q.split + 1) * T / j.splits;
  const int chunk = (q.s1 - q.s0 + kWorkers - 1) / kWorkers;
  const bool worker = wave > 0;
  q.w0 = q.s0 + (worker ? wave - 1 : 0) * chunk;
  q.nw_all = worker ? max(0, min(chunk, q.s1 - q.w0)) : 0;   // steps of this wave (control: none)
  // gate/up: each 16-column output tile is a gate tile followed by the up
  // tile of the same rows, so every weight tile reads one matrix
  q.ncol = (kPair ? j.N / 2 : j.N) / kTile;
  const int mine = q.g < q.ncol ? (q.ncol - 1 - q.g) / q.gsize + 1 : 0;
  q.nwork = kPair ? 2 * mine : mine;
  return q;
}

constexpr int kOutside = 0x7FFFFF00;   // buffer offset past any segment (segments are below 2 GiB)

// Weight tile k of this workgroup: a buffer resource over its matrix segment
// and this lane's byte offset; step i is at +64 i.  Steps a wave does not own,
// and the prefetch after the last tile, use an offset past the segment, which
// reads zeros without touching memory (no branches in the step loop, so no
// waits for the weights in flight are forced).
template <int EPI>
__device__ __forceinline__ __amdgpu_buffer_rsrc_t gemv_source(const GemvJob& j, const Geom& q, int k, int& voff) {
  constexpr bool kPair = EPI == PE_SWIGLU;
  const int lane = threadIdx.x & 63;
  const int c = q.g + (kPair ? (k >> 1) : k) * q.gsize;
  const int N = j.N;
  int rows, r;
  const bf16_t* base;
  if constexpr (kPair) {
    base = (k & 1) ? j.w[1] : j.w[0];
    rows = N / 2;
    r = c * kTile;
  } else {
    const int n0 = c * kTile, rw1 = j.row0[1], rw2 = j.row0[2], nseg = j.nseg;
    const bool g2 = nseg > 2 && n0 >= rw2, g1 = !g2 && nseg > 1 && n0 >= rw1;
    const int r0 = g2 ? rw2 : (g1 ? rw1 : 0);
    const int r1 = g2 ? N : (g1 ? (nseg > 2 ? rw2 : N) : (nseg > 1 ? rw1 : N));
    base = g2 ? j.w[2] : (g1 ? j.w[1] : j.w[0]);
    rows = r1 - r0;
    r = n0 - r0;
  }
  voff = ((r + (lane & 15)) * q.Kd + q.kq + q.w0 * 32) * 2;
  // built from scalar registers (else every load becomes a loop over the
  // lanes' distinct resources)
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16_t*>(opaque_p(base)), 0, opaque_s(rows * q.Kd * 2),
                                           kBufWord3);
}

// Issues the loads of this workgroup's first weight tile of job j into wv
// (the control wave and workgroups without tiles load zeros).
template <int EPI, int STEPS = kPassSteps>
__device__ __forceinline__ void gemv_prefetch(const GemvJob& j, u32x4 (&wv)[STEPS]) {
  const Geom q = gemv_geom<EPI>(j);
  int voff;
  const __amdgpu_buffer_rsrc_t rs = gemv_source<EPI>(j, q, 0, voff);
  const int nw = q.nwork > 0 ? q.nw_all : 0;
#pragma unroll
  for (int i = 0; i < STEPS; ++i)
    wv[i] = __builtin_amdgcn_raw_buffer_load_b128(rs, i < nw ? voff + 64 * i : kOutside, 0, 0);
}

// The GEMV phase; wv holds the first tile's weights (gemv_prefetch).
template <int EPI, int STEPS = kPassSteps>
__device__ __forceinline__ void gemv_phase(const PassArgs& a, const GemvJob& j, unsigned char* lds, uint64_t live,
                                           u32x4 (&wv)[STEPS]) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const Geom q = gemv_geom<EPI>(j);
  const int split = q.split, g = q.g, gsize = q.gsize, Kd = q.Kd, s0 = q.s0, s1 = q.s1, w0 = q.w0;
  const int nw_all = q.nw_all, nwork = q.nwork;
  const bool worker = wave > 0;
  constexpr bool kNorm = EPI == PE_ROPE || EPI == PE_SWIGLU;
  constexpr bool kPair = EPI == PE_SWIGLU;
  const int N = j.N;
  const int per_row = (s1 - s0) * 4, xstride = per_row + 1;
  u32x4* xs = reinterpret_cast<u32x4*>(lds);
  f32x4* red = reinterpret_cast<f32x4*>(lds + (size_t)a.M * xstride * 16);                 // [7][64]
  float* y = reinterpret_cast<float*>(lds + (size_t)a.M * xstride * 16 + kWorkers * 64 * 16);   // [16][17]
  float* inv_rms = y + 16 * 17;                                                             // [16]
  float* ygate = inv_rms + 16;                                                              // [16][17]

  for (int c = threadIdx.x; per_row > 0 && c < a.M * per_row; c += kPassWaves * 64) {
    const int m = c / per_row, qq = c - m * per_row;
    if (!((live >> m) & 1)) continue;
    const int k = s0 * 32 + qq * 8;
    xs[m * xstride + qq] = k < Kd ? ldg16(j.x + (size_t)m * Kd + k) : u32x4{0, 0, 0, 0};
  }
  if constexpr (kNorm) {
    for (int m = wave; m < 16; m += kPassWaves) {
      float v = 0.f;
      if ((live >> m) & 1)
        for (int tt = lane; tt < Kd / kTile; tt += 64) v += ldg(j.ss_in + (size_t)tt * a.mpad + m);
      for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
      if (lane == 0) inv_rms[m] = rsqrtf(v / Kd + a.eps);
    }
  }
  __syncthreads();

  for (int k = 0; k < nwork; ++k) {                  // workgroup-uniform
    const int tile = g + (kPair ? (k >> 1) : k) * gsize;   // output column tile
    const int sub = kPair ? (k & 1) : 0;
    if (worker) {
      f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
      const int m = lane & 15;
      const bool mok = (live >> m) & 1;
      const int nw = opaque_s(nw_all);
      const int nxt = opaque_s(k + 1 < nwork ? 1 : 0);
      int voff;
      const __amdgpu_buffer_rsrc_t rs = gemv_source<EPI>(j, q, nxt ? k + 1 : k, voff);
      const u32x4* xrow = xs + m * xstride + (w0 - s0) * 4 + (lane >> 4);
#pragma unroll
      for (int i = 0; i < STEPS; ++i) {
        const bool on = i < nw;
        const u32x4 xr = xrow[4 * (on ? i : 0)];
        const u32x4 xv = (on && mok) ? xr : u32x4{0, 0, 0, 0};
        acc = mfma16x16x32(wv[i], xv, acc);
        wv[i] = __builtin_amdgcn_raw_buffer_load_b128(rs, (on && nxt) ? voff + 64 * i : kOutside, 0, 0);
      }
      red[(wave - 1) * 64 + lane] = acc;
    }
    __syncthreads();
    if (threadIdx.x < 256) {
      const int L = threadIdx.x >> 2, i = threadIdx.x & 3;
      float v = 0.f;
#pragma unroll
      for (int w = 0; w < kWorkers; ++w) v += red[w * 64 + L][i];
      const int m = L & 15;
      y[m * 17 + 4 * (L >> 4) + i] = kNorm ? v * inv_rms[m] : v;
    }
    __syncthreads();
    const int n0 = tile * kTile;
    if constexpr (EPI == PE_ROPE) {
      const int q = threadIdx.x, m = q >> 3, pr = q & 7;
      if (q < 128 && m < a.M && ((live >> m) & 1)) {
        const int b = m / a.rps, jj = m - b * a.rps;
        const int slot = a.st[b].base + jj;
        const int D = a.D;
        const int head = n0 / D, d = ((n0 % D) >> 1) + pr;
        const float e = y[m * 17 + 2 * pr], o = y[m * 17 + 2 * pr + 1];
        if (head < a.nq + a.nkv) {
          const float* csp = reinterpret_cast<const float*>(a.rcs + (size_t)m * (D / 2) + d);
          const float cs_c = ldg(csp), cs_s = ldg(csp + 1);
          const float re = e * cs_c - o * cs_s, ro = e * cs_s + o * cs_c;
          if (head < a.nq) {
            st_u32(j.q + ((size_t)m * a.nq + head) * D + 2 * d, pack2(re, ro));
          } else {
            const size_t pg = (size_t)ldg(a.pt + b * a.pps + slot / kAttnChunk) * a.nkv + (head - a.nq);
            st_u32(j.kc + (pg * kAttnChunk + slot % kAttnChunk) * D + 2 * d, pack2(re, ro));
          }
        } else {
          const size_t pg = (size_t)ldg(a.pt + b * a.pps + slot / kAttnChunk) * a.nkv + (head - a.nq - a.nkv);
          bf16_t* vp = j.vt + (pg * D + 2 * d) * kAttnChunk + slot % kAttnChunk;
          st_u16(vp, f2bf(e));
          st_u16(vp + kAttnChunk, f2bf(o));
        }
      }
    } else if constexpr (EPI == PE_RESID) {
      const int q = threadIdx.x, m = q >> 4, c = q & 15;
      const int n = n0 + c;
      float xn = 0.f;
      if (q < 256 && m < a.M) {
        xn = ld_f32(a.x + (size_t)m * a.H + n);
        if ((live >> m) & 1) {
          xn += y[m * 17 + c];
          st_f32(a.x + (size_t)m * a.H + n, xn);
        }
        st_u16(j.xg_out + (size_t)m * a.H + n, f2bf(xn * bf2f(ldg(j.gain + n))));
      }
      float sq = xn * xn;
      for (int o = 1; o < 16; o <<= 1) sq += __shfl_xor(sq, o);
      if (q < 256 && c == 0) st_f32(j.ss_out + (size_t)tile * a.mpad + m, sq);
    } else if constexpr (EPI == PE_SWIGLU) {
      const int q = threadIdx.x, m = q >> 4, c = q & 15;
      if (q < 256) {
        if (sub == 0) {
          ygate[m * 17 + c] = y[m * 17 + c];       // gate tile: keep for the up tile
        } else if (m < a.M) {
          const float gt = ygate[m * 17 + c], up = y[m * 17 + c];
          st_u16(j.u + (size_t)m * (N / 2) + n0 + c, f2bf(gt / (1.f + expf(-gt)) * up));
        }
      }
    } else {
      // k-split partial sums; the finish phase adds them after a barrier
      const int qd = threadIdx.x, m = qd >> 4, c = qd & 15;
      if (qd < 256 && m < a.M) st_f32(a.part + ((size_t)split * a.M + m) * a.H + n0 + c, y[m * 17 + c]);
    }
  }
}

// Down projection finish: x += sum of the k-split partials (live rows), then
// the next norm's input bf16(x * gain) and per-16-column sums of x^2; for the
// last layer of a draft pass only each sequence's last live row, stored as
// row b.  16-column tiles are dealt to the workgroups; 256 threads per tile.
__device__ __forceinline__ void finish_phase(const PassArgs& a, const GemvJob& j) {
  const int ntiles = a.H / kTile;
  const int qd = threadIdx.x, m = qd >> 4, c = qd & 15;
  const int S = j.splits;
  for (int tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {   // workgroup-uniform
    if (qd >= 256) continue;
    const int n = tile * kTile + c;
    const bool row = m < a.M;
    const int b = row ? m / a.rps : 0, jj = row ? m - b * a.rps : 0;
    const int count = row ? a.st[b].count : 0;
    float xn = 0.f;
    if (row) {
      xn = ld_f32(a.x + (size_t)m * a.H + n);
      if (jj < count) {
        float v = 0.f;
        for (int sp = 0; sp < S; ++sp) v += ld_f32(a.part + ((size_t)sp * a.M + m) * a.H + n);
        xn += v;
        st_f32(a.x + (size_t)m * a.H + n, xn);
      }
    }
    float sq = xn * xn;
    for (int o = 1; o < 16; o <<= 1) sq += __shfl_xor(sq, o);
    if (row && (!j.select_last || jj == count - 1)) {
      const int out = j.select_last ? b : m;
      st_u16(j.xg_out + (size_t)out * a.H + n, f2bf(xn * bf2f(ldg(j.gain + n))));
      if (c == 0) st_f32(j.ss_out + (size_t)tile * a.mpad + out, sq);
    }
  }
}

// ---- attention partials ----------------------------------------------------
// Items (b, kv head, row block, split) are dealt to workgroups round-robin,
// two per workgroup at a time; item i of a round goes to workgroup i % G,
// wave group i / G (waves 0-3, 4-7).  Each wave group stages its
// key chunk and transposed value chunk in its own LDS region, then each of its
// waves owns 16 query rows: S^T = K Q^T, online softmax in log2 units, O^T +=
// V^T P^T, partial (o, max, sum) stored for the combine.
template <int D>
__device__ __forceinline__ void attn_phase(const PassArgs& a, const bf16_t* q, const bf16_t* kc, const bf16_t* vt,
                           unsigned char* lds) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int g4 = lane >> 4;
  const int G = gridDim.x;
  const int grp = wave >> 2;                               // 0 or 1
  const int gw = wave & 3;                                 // wave inside its group
  const int gt = gw * 64 + lane;                           // thread inside its group
  const int Gq = a.nq / a.nkv;
  const int rblocks = (a.rps * Gq + 63) / 64;
  const int nitems = a.B * a.nkv * rblocks * a.attn_splits;
  const int chunk = kAttnChunk;   // the pass is only used with this chunk size
  const int kst = D + 8, vst = chunk + 8;
  const size_t region = ((size_t)chunk * kst + (size_t)D * vst) * sizeof(bf16_t);

  for (int base_i = 0; base_i < nitems; base_i += 2 * G) {
    const int item = base_i + grp * G + blockIdx.x;
    const bool have = item < nitems;
    int split = 0, rb = 0, kvh = 0, b = 0;
    if (have) {
      int r = item;
      split = r % a.attn_splits;
      r /= a.attn_splits;
      rb = r % rblocks;
      r /= rblocks;
      kvh = r % a.nkv;
      b = r / a.nkv;
    }
    const SeqState& s = a.st[b];
    const int count = have ? s.count : 0, sbase = s.base;
    const int rows = count * Gq;
    const int wrow0 = rb * 64 + gw * 16;
    const int qr = wrow0 + (lane & 15);
    const bool rvalid = have && qr < rows;
    const int jrow = rvalid ? qr / Gq : 0;
    const int hq = kvh * Gq + (rvalid ? qr % Gq : 0);
    const int kv_end = sbase + count;
    const int k0 = split * chunk;
    const int k1 = min(k0 + chunk, kv_end);
    const int vis_end = sbase + jrow + 1;
    const size_t oi = (((size_t)split * a.B + b) * a.nq + hq) * a.R + jrow;
    bf16_t* Ks = reinterpret_cast<bf16_t*>(lds + grp * region);
    bf16_t* Vs = Ks + (size_t)chunk * kst;
    const bool work = have && k0 < k1 && wrow0 < rows;

    u32x4 qf[D / 32];
    {
      const bf16_t* qp = q + ((size_t)(b * a.R + jrow) * a.nq + hq) * D + 8 * g4;
#pragma unroll
      for (int t = 0; t < D / 32; ++t) qf[t] = (work && rvalid) ? ldg16(qp + 32 * t) : u32x4{0, 0, 0, 0};
    }
    if (have && k0 < k1) {
      // all of the thread's key and value loads are issued before its first
      // LDS store, so their latencies overlap
      constexpr int PER_T = kAttnChunk * D / 8 / 256;
      const size_t pg = (size_t)ldg(a.pt + b * a.pps + split) * a.nkv + kvh;
      const bf16_t* Kb = kc + pg * kAttnChunk * D;
      const bf16_t* Vb = vt + pg * D * kAttnChunk;
      const int per_row = kAttnChunk / 8;
      u32x4 rk[PER_T], rv[PER_T];
#pragma unroll
      for (int u = 0; u < PER_T; ++u) {
        const int i = gt + 256 * u;
        const int key = i / (D / 8), c8 = i % (D / 8);
        rk[u] = k0 + key < k1 ? ldg16(Kb + (size_t)key * D + 8 * c8) : u32x4{0, 0, 0, 0};
        const int d = i / per_row, v8 = i % per_row;
        const int slot = k0 + 8 * v8;
        rv[u] = slot < k1 ? ldg16(Vb + (size_t)d * kAttnChunk + 8 * v8) : u32x4{0, 0, 0, 0};
      }
#pragma unroll
      for (int u = 0; u < PER_T; ++u) {
        const int i = gt + 256 * u;
        const int key = i / (D / 8), c8 = i % (D / 8);
        *reinterpret_cast<u32x4*>(Ks + (size_t)key * kst + 8 * c8) = rk[u];
        const int d = i / per_row, v8 = i % per_row;
        const int slot = k0 + 8 * v8;
        u32x4 v = rv[u];
        if (slot < k1 && slot + 8 > k1) {
          uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
          for (int e = 0; e < 8; ++e)
            if (slot + e >= k1) w[e >> 1] &= (e & 1) ? 0x0000FFFFu : 0xFFFF0000u;
          v = u32x4{w[0], w[1], w[2], w[3]};
        }
        *reinterpret_cast<u32x4*>(Vs + (size_t)d * vst + 8 * v8) = v;
      }
    }
    __syncthreads();
    if (have && wrow0 < rows) {
      if (k0 >= k1) {                          // no keys in this split
        if (rvalid && g4 == 0) {
          st_f32(a.mp + oi, -INFINITY);
          st_f32(a.lp + oi, 0.f);
        }
        if (rvalid) {
          float* op = a.op + oi * D;
          for (int d = g4 * 4; d < D; d += 16) st_f32x4(op + d, f32x4{0.f, 0.f, 0.f, 0.f});
        }
      } else {
        float m_run = -INFINITY, l_run = 0.f;
        f32x4 o[D / 16];
#pragma unroll
        for (int dt = 0; dt < D / 16; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
        for (int kb = 0; kb < k1 - k0; kb += kKeyBlock) {
          f32x4 sc[2];
#pragma unroll
          for (int h2 = 0; h2 < 2; ++h2) {
            const bf16_t* kp = Ks + (size_t)(kb + 16 * h2 + (lane & 15)) * kst + 8 * g4;
            f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int t = 0; t < D / 32; ++t)
              acc = mfma16x16x32(*reinterpret_cast<const u32x4*>(kp + 32 * t), qf[t], acc);
            sc[h2] = acc;
          }
          float p[8];
          float bm = -INFINITY;
#pragma unroll
          for (int h2 = 0; h2 < 2; ++h2)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int key = k0 + kb + 16 * h2 + 4 * g4 + i;
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
          const u32x4 pb = u32x4{pack2(p[0], p[1]), pack2(p[2], p[3]), pack2(p[4], p[5]), pack2(p[6], p[7])};
#pragma unroll
          for (int dt = 0; dt < D / 16; ++dt) {
            const bf16_t* vp = Vs + (size_t)(16 * dt + (lane & 15)) * vst + kb + 4 * g4;
            const u32x2 lo = *reinterpret_cast<const u32x2*>(vp), hi = *reinterpret_cast<const u32x2*>(vp + 16);
            o[dt] = mfma16x16x32(u32x4{lo.x, lo.y, hi.x, hi.y}, pb, o[dt] * alpha);
          }
        }
        l_run += __shfl_xor(l_run, 16);
        l_run += __shfl_xor(l_run, 32);
        if (rvalid) {
          float* op = a.op + oi * D;
#pragma unroll
          for (int dt = 0; dt < D / 16; ++dt) st_f32x4(op + 16 * dt + 4 * g4, o[dt]);
          if (g4 == 0) {
            st_f32(a.mp + oi, m_run);
            st_f32(a.lp + oi, l_run);
          }
        }
      }
    }
    __syncthreads();   // LDS regions are reused by the next round
  }
}

// ---- combine ----------------------------------------------------------------
// Item (b, j, q head): o = sum_s 2^(m_s - M) O_s / sum_s 2^(m_s - M) l_s over
// the splits holding keys row j sees.  Waves 1..7: 4-column groups x split
// groups; the per-group sums are added in a fixed order.
template <int D>
__device__ __forceinline__ void combine_phase(const PassArgs& a, bf16_t* o_out, unsigned char* lds) {
  float* coef = reinterpret_cast<float*>(lds);                          // [splits]
  float* part = coef + ((a.attn_splits + 3) & ~3);                      // [SG][D]
  constexpr int CG = D / 4;                                             // column groups
  constexpr int SG = kWorkers * 64 / CG;                                // split groups
  const int nitems = a.B * a.R * a.nq;
  for (int item = blockIdx.x; item < nitems; item += gridDim.x) {
    const int h = item % a.nq, r = item / a.nq;
    const int jrow = r % a.R, b = r / a.R;
    const SeqState& s = a.st[b];
    if (jrow >= s.count) continue;                                       // workgroup-uniform
    const int vis_end = s.base + jrow + 1;
    const int ns = (vis_end + a.attn_chunk - 1) / a.attn_chunk;
    const size_t row = ((size_t)b * a.nq + h) * a.R + jrow;
    const size_t sstride = (size_t)a.B * a.nq * a.R;
    if (threadIdx.x < 64) {
      const int l = threadIdx.x;
      float M = -INFINITY;
      for (int sp = l; sp < ns; sp += 64) M = fmaxf(M, ld_f32(a.mp + sp * sstride + row));
      for (int o = 32; o > 0; o >>= 1) M = fmaxf(M, __shfl_xor(M, o));
      float L = 0.f;
      for (int sp = l; sp < ns; sp += 64) {
        const float w = exp2f(ld_f32(a.mp + sp * sstride + row) - M);
        coef[sp] = w;
        L += w * ld_f32(a.lp + sp * sstride + row);
      }
      for (int o = 32; o > 0; o >>= 1) L += __shfl_xor(L, o);
      const float inv = 1.f / L;
      for (int sp = l; sp < ns; sp += 64) coef[sp] *= inv;
    }
    __syncthreads();
    if (threadIdx.x >= 64) {
      const int t = threadIdx.x - 64;
      const int c4 = t % CG, sg = t / CG;
      f32x4 v = f32x4{0.f, 0.f, 0.f, 0.f};
      const float* src = a.op + row * D + 4 * c4;
      const size_t ostride = sstride * D;
      for (int sp = sg; sp < ns; sp += SG) v += coef[sp] * ld_f32x4(src + sp * ostride);
      *reinterpret_cast<f32x4*>(part + sg * D + 4 * c4) = v;
    }
    __syncthreads();
    if (threadIdx.x < D / 2) {
      const int d = 2 * threadIdx.x;
      float t0 = 0.f, t1 = 0.f;
      for (int gi = 0; gi < SG; ++gi) {
        t0 += part[gi * D + d];
        t1 += part[gi * D + d + 1];
      }
      st_u32(o_out + (size_t)(b * a.R + jrow) * a.nq * D + h * D + d, pack2(t0, t1));
    }
    __syncthreads();
  }
}

// The arguments live in device memory: read through a plain pointer, the
// loads cannot move above the stores of earlier phases, so each phase reads
// the fields it needs instead of the whole block staying in scalar registers
// for the entire launch.
// ROLE 0: target (verify) passes, 1: draft passes.  Same code; separate
// symbols so that profiles report the two kinds of launch apart.
template <int D, int ROLE>
__global__ __launch_bounds__(kPassWaves * 64) void k_pass(const PassArgs* pa) {
  extern __shared__ __align__(16) unsigned char lds[];
  const PassArgs& a = *pa;
  const uint64_t live = live_rows(a);
  bool failed = false;
  unsigned gen = 0;
  unsigned long long* tl = a.timeline;
  auto stamp = [&](int ev) {
    if (tl && threadIdx.x == 0) tl[(size_t)ev * gridDim.x + blockIdx.x] = wall_clock64();
  };
  stamp(0);
  // Weights of the next GEMV phase's first tile, issued before the barrier
  // that precedes it (they do not depend on the activations): the barrier,
  // and attention and combine for the O projection, overlap their fetch.
  u32x4 wv[kPassSteps];
  const bool worker = (threadIdx.x >> 6) > 0;
  auto prefetch = [&](int li, int job) {
    if (!worker || li >= a.layers) return;
    const GemvJob& j = a.jobs[(size_t)li * kPassJobs + job];
    switch (job) {
      case 0: gemv_prefetch<PE_ROPE>(j, wv); break;
      case 1: gemv_prefetch<PE_RESID>(j, wv); break;
      case 2: gemv_prefetch<PE_SWIGLU>(j, wv); break;
      default: gemv_prefetch<PE_DOWN>(j, wv); break;
    }
  };
  prefetch(0, 0);
  for (int li = 0; li < a.layers; ++li) {
    const GemvJob* jl = a.jobs + (size_t)li * kPassJobs;
    const int ev = 1 + li * kPassPhases * 2;
    gemv_phase<PE_ROPE>(a, jl[0], lds, live, wv);
    stamp(ev + 0);
    grid_sync(a, ++gen, failed, [&] { prefetch(li, 1); });
    stamp(ev + 1);
    attn_phase<D>(a, a.q + a.q_layer * li, a.kc + a.kv_layer * li, a.vt + a.kv_layer * li, lds);
    stamp(ev + 2);
    grid_sync(a, ++gen, failed);
    stamp(ev + 3);
    combine_phase<D>(a, a.o + a.q_layer * li, lds);
    stamp(ev + 4);
    grid_sync(a, ++gen, failed);
    stamp(ev + 5);
    gemv_phase<PE_RESID>(a, jl[1], lds, live, wv);
    stamp(ev + 6);
    grid_sync(a, ++gen, failed, [&] { prefetch(li, 2); });
    stamp(ev + 7);
    gemv_phase<PE_SWIGLU>(a, jl[2], lds, live, wv);
    stamp(ev + 8);
    grid_sync(a, ++gen, failed, [&] { prefetch(li, 3); });
    stamp(ev + 9);
    gemv_phase<PE_DOWN>(a, jl[3], lds, live, wv);
    stamp(ev + 10);
    grid_sync(a, ++gen, failed, [&] { prefetch(li + 1, 0); });
    stamp(ev + 11);
    finish_phase(a, jl[3]);
    if (li + 1 < a.layers) grid_sync(a, ++gen, failed);
  }
  grid_done(a);
}

// One GEMV phase as a kernel of its own (the layered path's large
// projections): the first tile's weights are requested before x is staged.
template <int EPI, int STEPS>
__global__ __launch_bounds__(kPassWaves * 64) void k_gemv_job(const PassArgs* pa, const GemvJob* job) {
  extern __shared__ __align__(16) unsigned char lds[];
  const PassArgs& a = *pa;
  const uint64_t live = live_rows(a);
  u32x4 wv[STEPS];
  if ((threadIdx.x >> 6) > 0) gemv_prefetch<EPI, STEPS>(*job, wv);
  gemv_phase<EPI, STEPS>(a, *job, lds, live, wv);
}

}  // namespace

// Step-count variants of the one-phase kernels: the smallest that covers a
// worker wave's k-steps (fewer idle slots in the step loop).
#define SPECDEC_JOB_KERNELS(X) X(PE_ROPE) X(PE_RESID) X(PE_SWIGLU) X(PE_DOWN)

template <int EPI>
hipError_t job_launch_steps(int steps, const PassArgs* d_args, const GemvJob* d_job, dim3 grid, size_t lds,
                            hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  const dim3 block(kPassWaves * 64);
  if (steps <= 8)
    hipExtLaunchKernelGGL((k_gemv_job<EPI, 8>), grid, block, (uint32_t)lds, s, e0, e1, 0, d_args, d_job);
  else if (steps <= 12)
    hipExtLaunchKernelGGL((k_gemv_job<EPI, 12>), grid, block, (uint32_t)lds, s, e0, e1, 0, d_args, d_job);
  else if (steps <= 16)
    hipExtLaunchKernelGGL((k_gemv_job<EPI, 16>), grid, block, (uint32_t)lds, s, e0, e1, 0, d_args, d_job);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t gemv_job_launch(int kind, int steps, const PassArgs* d_args, const GemvJob* d_job, int workgroups,
                           size_t lds, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  const dim3 grid(workgroups);
  switch (kind) {
    case kJobQkv: return job_launch_steps<PE_ROPE>(steps, d_args, d_job, grid, lds, s, e0, e1);
    case kJobO: return job_launch_steps<PE_RESID>(steps, d_args, d_job, grid, lds, s, e0, e1);
    case kJobGateUp: return job_launch_steps<PE_SWIGLU>(steps, d_args, d_job, grid, lds, s, e0, e1);
    case kJobDown: return job_launch_steps<PE_DOWN>(steps, d_args, d_job, grid, lds, s, e0, e1);
    default: return hipErrorInvalidValue;
  }
}

int gemv_job_steps(int Kd, int splits) {
  const int T = (Kd + 31) / 32;
  const int span = (T + splits - 1) / splits;
  return (span + kWorkers - 1) / kWorkers;
}

void pass_build_jobs(const PassArgs& a, const LayerW* lw, const bf16_t* final_norm, GemvJob* jobs) {
  const int D = a.D;
  for (int li = 0; li < a.layers; ++li) {
    const LayerW& w = lw[li];
    const bool last = li + 1 == a.layers;
    GemvJob* j = jobs + (size_t)li * kPassJobs;
    j[0] = GemvJob{};
    j[0].w[0] = w.wq;
    j[0].w[1] = w.wk;
    j[0].w[2] = w.wv;
    j[0].row0[1] = a.nq * D;
    j[0].row0[2] = (a.nq + a.nkv) * D;
    j[0].nseg = 3;
    j[0].N = (a.nq + 2 * a.nkv) * D;
    j[0].Kd = a.H;
    j[0].splits = 1;
    j[0].x = a.xa + a.x_layer * li;
    j[0].ss_in = a.ssa + a.ss_layer * li;
    j[0].q = a.q + a.q_layer * li;
    j[0].kc = a.kc + a.kv_layer * li;
    j[0].vt = a.vt + a.kv_layer * li;
    j[1] = GemvJob{};
    j[1].w[0] = j[1].w[1] = j[1].w[2] = w.wo;
    j[1].nseg = 1;
    j[1].N = a.H;
    j[1].Kd = a.nq * D;
    j[1].splits = 1;
    j[1].x = a.o + a.q_layer * li;
    j[1].gain = w.ffn_norm;
    j[1].xg_out = a.xf + a.x_layer * li;
    j[1].ss_out = a.ssf + a.ss_layer * li;
    j[2] = GemvJob{};
    j[2].w[0] = w.wg;
    j[2].w[1] = j[2].w[2] = w.wu;
    j[2].nseg = 2;
    j[2].N = 2 * a.F;
    j[2].Kd = a.H;
    j[2].splits = 1;
    j[2].x = a.xf + a.x_layer * li;
    j[2].ss_in = a.ssf + a.ss_layer * li;
    j[2].u = a.u + a.u_layer * li;
    j[3] = GemvJob{};
    j[3].w[0] = j[3].w[1] = j[3].w[2] = w.wd;
    j[3].nseg = 1;
    j[3].N = a.H;
    j[3].Kd = a.F;
    j[3].splits = a.down_splits;
    j[3].x = a.u + a.u_layer * li;
    j[3].gain = last ? final_norm : lw[li + 1].attn_norm;
    j[3].xg_out = last ? a.xg_final : a.xa + a.x_layer * (li + 1);
    j[3].ss_out = last ? a.ss_final : a.ssa + a.ss_layer * (li + 1);
    j[3].select_last = last && a.select_last;
  }
}

size_t pass_gemv_lds_bytes(const PassArgs& a) {
  auto gemv = [&](int Kd, int splits) {
    const int T = (Kd + 31) / 32;
    const int span = (T + splits - 1) / splits;
    return (size_t)a.M * (span * 4 + 1) * 16 + (size_t)kWorkers * 64 * 16 + (2 * 16 * 17 + 16) * sizeof(float);
  };
  return std::max({gemv(a.H, 1), gemv(a.nq * a.D, 1), gemv(a.F, a.down_splits)});
}

size_t pass_lds_bytes(const PassArgs& a) {
  auto gemv = [&](int Kd, int splits) {
    const int T = (Kd + 31) / 32;
    const int span = (T + splits - 1) / splits;
    return (size_t)a.M * (span * 4 + 1) * 16 + (size_t)kWorkers * 64 * 16 + (2 * 16 * 17 + 16) * sizeof(float);
  };
  size_t m = std::max({gemv(a.H, 1), gemv(a.nq * a.D, 1), gemv(a.F, a.down_splits)});
  const size_t attn = 2 * ((size_t)a.attn_chunk * (a.D + 8) + (size_t)a.D * (a.attn_chunk + 8)) * sizeof(bf16_t);
  const size_t comb = (size_t)(((a.attn_splits + 3) & ~3) + (kWorkers * 64 / (a.D / 4)) * a.D) * sizeof(float);
  return std::max({m, attn, comb});
}

// Steps per worker wave of the largest GEMV of the pass; must be <= kPassSteps.
int pass_steps(const PassArgs& a) {
  auto steps = [](int Kd, int splits) {
    const int T = (Kd + 31) / 32;
    const int span = (T + splits - 1) / splits;
    return (span + kWorkers - 1) / kWorkers;
  };
  return std::max({steps(a.H, 1), steps(a.nq * a.D, 1), steps(a.F, a.down_splits)});
}

void pass_set_attributes(int lds_limit) {
  const void* fns[] = {reinterpret_cast<const void*>(&k_pass<128, 0>), reinterpret_cast<const void*>(&k_pass<128, 1>),
                       reinterpret_cast<const void*>(&k_pass<64, 0>), reinterpret_cast<const void*>(&k_pass<64, 1>)};
  for (const void* f : fns) (void)hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, lds_limit);
#define SPECDEC_SET_JOB_ATTR(E)                                                                                  \
  (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&k_gemv_job<E, 8>),                                    \
                            hipFuncAttributeMaxDynamicSharedMemorySize, lds_limit);                             \
  (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&k_gemv_job<E, 12>),                                   \
                            hipFuncAttributeMaxDynamicSharedMemorySize, lds_limit);                             \
  (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&k_gemv_job<E, 16>),                                   \
                            hipFuncAttributeMaxDynamicSharedMemorySize, lds_limit);
  SPECDEC_JOB_KERNELS(SPECDEC_SET_JOB_ATTR)
#undef SPECDEC_SET_JOB_ATTR
}

hipError_t pass_launch(const PassArgs* d_args, int head_dim, bool draft, int workgroups, size_t lds, hipStream_t s,
                       hipEvent_t e0, hipEvent_t e1) {
  const dim3 grid(workgroups), block(kPassWaves * 64);
  if (head_dim == 128 && !draft)
    hipExtLaunchKernelGGL((k_pass<128, 0>), grid, block, (uint32_t)lds, s, e0, e1, 0, d_args);
  else if (head_dim == 128)
    hipExtLaunchKernelGGL((k_pass<128, 1>), grid, block, (uint32_t)lds, s, e0, e1, 0, d_args);
  else if (head_dim == 64 && !draft)
    hipExtLaunchKernelGGL((k_pass<64, 0>), grid, block, (uint32_t)lds, s, e0, e1, 0, d_args);
  else if (head_dim == 64)
    hipExtLaunchKernelGGL((k_pass<64, 1>), grid, block, (uint32_t)lds, s, e0, e1, 0, d_args);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace specdec
