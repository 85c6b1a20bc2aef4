// Balanced weight-streaming GEMV on gfx950 for passes of at most 32 rows.
//
// y[m][n] = sum_k x[m][k] W[n][k] over tile-packed weights (sgemv.h): each
// 16-row x 32-column MFMA operand block is 1 KB contiguous, so every wave
// load reads 1 KB of consecutive memory and a tile is one contiguous run.
//
// Work split.  Whole units (a 16-row tile, or a gate/up tile pair) are dealt
// round-robin to the G workgroups of a k-slice (unit r*G + g in round r, the
// last round ragged), so at any moment the workgroups stream neighbouring
// tiles.  A tile's k-steps (of its slice) are cut into 15 chunks, one per
// worker wave.
//
// Waves.  Waves 1..15 stream weights: each keeps its share of one tile (up to
// 8 loads of 16 bytes per lane) in flight through a rolling register buffer
// and multiplies it against the x operands of its k-steps, which it loads
// once into registers (the same for every tile); a step a wave does not own
// reads a buffer offset past the matrix, which returns zeros without touching
// memory, so the step loop has no branches and the workers issue no other
// memory operation.  Wave 0 (control) sums the 15 partial tiles in a fixed
// order through double-buffered LDS, one workgroup barrier per tile, and runs
// the epilogue while the workers already stream the next tile.
//
// Long k-ranges (the down projection: its input rows are 18944 wide) stream
// x with the weights: a worker's k-steps are taken eight at a time, each slot
// of the rolling buffer holding one weight block and the matching x operand
// (read from L2), so a tile is never cut across workgroups.
//
// k-sliced reductions (S > 1, kept for shapes that ask for them) are finished
// by the workgroup that arrives last at a tile: each slice's
// workgroup stores its partial tile, makes it visible with a release fence and
// counts itself in; the last one reads the partials back in slice order, adds
// them and runs the epilogue, and resets the counter for the next launch.
// Sums are therefore deterministic.
//
// Epilogues (RMSNorm is applied as a per-row 1/rms from the producer's
// per-16-column sums of squares):
//   SG_ROPE    q/k/v: rotation of q and k pairs at each row's position
//              (Eq. rope-3d / Eq. flatrope-proj via the per-row (cos, sin)),
//              query store, K and V^T cache append
//   SG_RESID   o: residual add, bf16(x * g) and sums of x^2 for the next norm
//   SG_SWIGLU  gate/up tile pairs: silu(gate) * up
//   SG_DOWN    down: as SG_RESID; on a draft pass's last layer only each
//              sequence's last live row, stored as row b
//   SG_ARGMAX  LM head: optional bf16 logits, and the (max, index) of each row
//              over the workgroup's tiles (per tile when k-sliced)
#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>

#include <algorithm>
#include <cmath>

#include "ctx.h"
#include "device.h"
#include "sgemv.h"

namespace specdec {

namespace {

constexpr int kOut = 0x7FFFFF00;          // buffer offset past every packed matrix (they are < kOut bytes)
constexpr int kRsrcWord3 = 0x00020000;    // raw buffer resource, 32-bit data
// Cache policy of the weight loads: non-temporal.  Each weight byte is read
// once per pass, and streaming it with the nt hint measured 6.4-6.8 TB/s on
// the large projections against 5.7-6.1 TB/s for default-policy loads.
constexpr int kNt = 2;


// Workgroup barrier that waits for this wave's LDS operations only (global
// loads and stores stay in flight).  The memory clobber keeps the compiler
// from moving LDS accesses across it.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// Per-lane row facts the control wave needs (lane's row m = lane % 16 + 16 rb
// in row block rb).
struct RowInfo {
  bool live;       // row m < M and inside its sequence's current row count
  int b, jr;       // sequence and row within it
  int count;       // that sequence's row count
  int slot, page;  // SG_ROPE: cache slot and its page
  int want_logits;
  float inv_rms;
  // SG_ARGMAX without k-slices: running (max, index) of the row over this
  // workgroup's tiles, and whether a NaN was seen
  float best;
  int bi, nan;
};

template <int EPI>
__device__ __forceinline__ void epilogue(const SgJob& j, RowInfo& ri, int rb, int u, f32x4 ya, f32x4 yb, f32x4 pa,
                                         u32x2 pb) {
  const int lane = threadIdx.x & 63, m = (lane & 15) + 16 * rb, grp = lane >> 4;
  const int M = j.M;
  if constexpr (EPI == SG_ROPE) {
    if (ri.live) {
      const int D = j.D, n0 = 16 * u, head = n0 / D, d0 = (n0 % D) / 2 + 2 * grp;
      const float s = ri.inv_rms;
      const float e0 = ya.x * s, o0 = ya.y * s, e1 = ya.z * s, o1 = ya.w * s;
      const int off = ri.slot % kAttnChunk;
      if (head < j.nq + j.nkv) {
        const uint32_t w0 = pack2(e0 * pa.x - o0 * pa.y, e0 * pa.y + o0 * pa.x);
        const uint32_t w1 = pack2(e1 * pa.z - o1 * pa.w, e1 * pa.w + o1 * pa.z);
        if (head < j.nq) {
          *reinterpret_cast<u32x2*>(j.q + ((size_t)m * j.nq + head) * D + 2 * d0) = u32x2{w0, w1};
        } else {
          const size_t pg = (size_t)ri.page * j.nkv + (head - j.nq);
          *reinterpret_cast<u32x2*>(j.kc + (pg * kAttnChunk + off) * D + 2 * d0) = u32x2{w0, w1};
        }
      } else {
        const size_t pg = (size_t)ri.page * j.nkv + (head - j.nq - j.nkv);
        bf16_t* vp = j.vt + (pg * D + 2 * d0) * kAttnChunk + off;
        vp[0] = f2bf(e0);
        vp[kAttnChunk] = f2bf(o0);
        vp[2 * kAttnChunk] = f2bf(e1);
        vp[3 * kAttnChunk] = f2bf(o1);
      }
    }
  } else if constexpr (EPI == SG_RESID || EPI == SG_DOWN) {
    const int n = 16 * u + 4 * grp;
    f32x4 xn = pa;
    if (ri.live) {
      xn += ya;
      *reinterpret_cast<f32x4*>(j.x32 + (size_t)m * j.H + n) = xn;
    }
    float sq = xn.x * xn.x + xn.y * xn.y + xn.z * xn.z + xn.w * xn.w;
    sq += __shfl_xor(sq, 16);
    sq += __shfl_xor(sq, 32);
    bool write = m < M;
    int out = m;
    if (EPI == SG_DOWN && j.select_last) {
      write = ri.live && ri.jr == ri.count - 1;
      out = ri.b;
    }
    if (write) {
      const float g0 = __uint_as_float(pb.x << 16), g1 = __uint_as_float(pb.x & 0xffff0000u);
      const float g2 = __uint_as_float(pb.y << 16), g3 = __uint_as_float(pb.y & 0xffff0000u);
      *reinterpret_cast<u32x2*>(j.xg + (size_t)out * j.H + n) =
          u32x2{pack2(xn.x * g0, xn.y * g1), pack2(xn.z * g2, xn.w * g3)};
      if (grp == 0) j.ss_out[(size_t)u * j.mpad + out] = sq;
    }
  } else if constexpr (EPI == SG_SWIGLU) {
    if (m < M) {
      const float s = ri.inv_rms;
      const f32x4 g = ya * s, up = yb * s;
      float r[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) r[i] = g[i] / (1.f + expf(-g[i])) * up[i];
      const int F = j.ntiles * 8, n = 16 * u + 4 * grp;
      const size_t at = j.upk ? ((size_t)(n >> 5) * M + m) * 32 + (n & 31) : (size_t)m * F + n;
      *reinterpret_cast<u32x2*>(j.u + at) = u32x2{pack2(r[0], r[1]), pack2(r[2], r[3])};
    }
  } else {   // SG_ARGMAX
    const f32x4 y = ya * ri.inv_rms;
    const int N = j.ntiles * 16, n = 16 * u + 4 * grp;
    if (j.allow_logits && m < M && ri.want_logits)
      *reinterpret_cast<u32x2*>(j.logits + (size_t)m * N + n) = u32x2{pack2(y.x, y.y), pack2(y.z, y.w)};
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
    if (j.S == 1) {
      // one workgroup finishes all of its tiles: keep the row's running best
      // (ties to the lower index, so the order of tiles does not matter)
      amax_merge(ri.best, ri.bi, best, bi);
      ri.nan |= nan;
    } else if (grp == 0 && m < M) {
      j.amax_v[(size_t)u * j.mpad + m] = best;
      j.amax_i[(size_t)u * j.mpad + m] = bi;
      if (nan) atomicOr(const_cast<int32_t*>(&j.st[ri.b].err), ERR_NUMERIC);
    }
  }
}

// Epilogue inputs of unit u that come from memory: the (cos, sin) of the
// lane's two rotary pairs, or the residual and the norm gain of its 4 columns.
template <int EPI>
__device__ __forceinline__ void epilogue_inputs(const SgJob& j, const RowInfo& ri, int rb, int u, f32x4& pa,
                                                u32x2& pb) {
  const int lane = threadIdx.x & 63, m = (lane & 15) + 16 * rb, grp = lane >> 4;
  pa = f32x4{0.f, 0.f, 0.f, 0.f};
  pb = u32x2{0u, 0u};
  if constexpr (EPI == SG_ROPE) {
    const int D = j.D, n0 = 16 * u, head = n0 / D, d0 = (n0 % D) / 2 + 2 * grp;
    if (ri.live && head < j.nq + j.nkv)
      pa = *reinterpret_cast<const f32x4*>(reinterpret_cast<const float*>(j.rcs + (size_t)m * (D / 2) + d0));
  } else if constexpr (EPI == SG_RESID || EPI == SG_DOWN) {
    const int n = 16 * u + 4 * grp;
    if (m < j.M) {
      pa = *reinterpret_cast<const f32x4*>(j.x32 + (size_t)m * j.H + n);
      pb = *reinterpret_cast<const u32x2*>(j.gain + n);
    }
  }
}

// The job is a kernel argument (not a pointer to it) so that its fields
// arrive with the launch: the weight and activation loads do not wait for a
// memory round trip to fetch their addresses first.
//
// MB row blocks of 16 rows (passes of up to 16 * MB rows): every weight block
// a worker loads feeds one MFMA per row block, and each output's sum is formed
// exactly as with one row block (the same k-step chunks per worker, the same
// order of the partial tiles), so a row's result does not depend on MB.
template <int EPI, bool XS, int MB, int DEPN>
__global__ __launch_bounds__(kSgWaves * 64) void k_sgemv(const SgJob j) {
  constexpr int DEP = XS ? kSgDepthXs : DEPN;   // rolling-buffer slots per worker (x in registers: steps per worker)
  extern __shared__ __align__(16) unsigned char lds[];
  constexpr bool kPair = EPI == SG_SWIGLU;
  constexpr int TPU = kPair ? 2 : 1;   // tiles per unit
  constexpr bool kNorm = EPI == SG_ROPE || EPI == SG_SWIGLU || EPI == SG_ARGMAX;
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int lane = threadIdx.x & 63;
  const int S = j.S, G = j.G, T = j.T, M = j.M;
  const int sl = blockIdx.x / G, gi = blockIdx.x - sl * G;
  const int k0 = sl * T / S, k1 = (sl + 1) * T / S, span = k1 - k0;
  // Units (a tile, or a gate/up tile pair) are dealt round-robin: this
  // workgroup takes units gi, gi + G, gi + 2G, ... (the last round ragged), so
  // at any moment the workgroups stream neighbouring tiles.
  const int units = j.ntiles / TPU;
  const int n_it = (units / G + (gi < units % G ? 1 : 0)) * TPU;   // tiles of this workgroup
  auto tile_of = [&](int it) { return ((it / TPU) * G + gi) * TPU + it % TPU; };
  f32x4* red = reinterpret_cast<f32x4*>(lds);                                   // [2][MB][workers][64]
  int* pend = reinterpret_cast<int*>(lds + 2 * MB * kSgWorkers * 64 * 16);      // [kSgPendMax + 4]
  float* rms_sh = reinterpret_cast<float*>(pend + kSgPendMax + 4);              // [16 MB] 1/rms per row

  // Worker w owns k-steps [ws0, ws0 + nst) of every tile of this slice.
  const int wi = wave - 1;
  int ws0 = 0, nst = 0;
  if (wave > 0) {
    ws0 = k0 + span * wi / kSgWorkers;
    nst = k0 + span * (wi + 1) / kSgWorkers - ws0;
  }
  const int m0 = lane & 15, grp = lane >> 4;

  // Issue order (vector memory returns in order per wave): a worker first
  // loads its x operands (the same for every tile, so they stay in registers:
  // lane (m, g) holds x[m][32 s + 8 g .. +8] of its step s), then the first
  // tile's weights, so that the MFMAs can start as soon as weights arrive.
  // Rows of dead sequences are zeroed once the live mask is known.
  u32x4 xv[MB][DEP];
  const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16_t*>(j.w), 0,
                                                                      j.ntiles * T * 1024, kRsrcWord3);
  // x rows as a buffer (streamed x): an offset past it reads zeros
  const __amdgpu_buffer_rsrc_t rsx = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<bf16_t*>(j.x), 0, j.xpk ? T * M * 64 : M * j.ldx * 2, kRsrcWord3);
  bool xrow[MB];                 // lane's x row of each block is loaded (narrowed to live rows once known)
#pragma unroll
  for (int rb = 0; rb < MB; ++rb) xrow[rb] = m0 + 16 * rb < M;
  auto x_off = [&](int rb, int step) {   // byte offset of lane (m, grp)'s x operand of a k-step, or kOut
    const int k = step * 32 + 8 * grp, m = m0 + 16 * rb;
    return (xrow[rb] && k < j.Kd) ? (j.xpk ? ((step * M + m) * 32 + 8 * grp) * 2 : (m * j.ldx + k) * 2) : kOut;
  };
  const int lane_off = lane * 16;
  u32x4 wv[DEP];
  if (wave > 0) {
#pragma unroll
    for (int rb = 0; rb < MB; ++rb)
#pragma unroll
      for (int i = 0; i < DEP; ++i) {
        xv[rb][i] = __builtin_amdgcn_raw_buffer_load_b128(rsx, i < nst ? x_off(rb, ws0 + i) : kOut, 0, 0);
      }
    if (n_it > 0) {
      const int v = (tile_of(0) * T + ws0) * 1024 + lane_off;
#pragma unroll
      for (int i = 0; i < DEP; ++i)
        wv[i] = __builtin_amdgcn_raw_buffer_load_b128(rs, i < nst ? v + 1024 * i : kOut, 0, kNt);
    }
  }

  // live rows: sequence b's rows are live below its row count (scalar loads)
  uint32_t live = 0;
  {
    const int nseq = (M + j.rps - 1) / j.rps;
    for (int b = 0; b < nseq; ++b) {
      const int n = min(j.st[b].count, j.rps);
      if (n > 0) live |= ((1u << n) - 1u) << (b * j.rps);
    }
    if (M < 32) live &= (1u << M) - 1u;
  }
  bool xok[MB];
#pragma unroll
  for (int rb = 0; rb < MB; ++rb) {
    xok[rb] = (live >> (m0 + 16 * rb)) & 1;
    xrow[rb] = xrow[rb] && xok[rb];   // streamed x: rows of dead sequences are not read at all
  }
  if (!XS && wave > 0) {
#pragma unroll
    for (int rb = 0; rb < MB; ++rb)
      if (!xok[rb]) {
#pragma unroll
        for (int i = 0; i < DEP; ++i) xv[rb][i] = u32x4{0, 0, 0, 0};
      }
  }

  // per-row facts of the lane's rows (the control wave before its tile loop;
  // every wave before finishing split units)
  auto row_info = [&](RowInfo* ri) {
#pragma unroll
    for (int rb = 0; rb < MB; ++rb) {
      RowInfo& r = ri[rb];
      const int m = m0 + 16 * rb;
      const bool mok = m < M;
      r.live = mok && ((live >> m) & 1);
      r.b = mok ? m / j.rps : 0;
      r.jr = m - r.b * j.rps;
      r.count = j.st[r.b].count;
      r.want_logits = j.st[r.b].want_logits;
      r.inv_rms = 1.f;
      r.best = -INFINITY;
      r.bi = 0x7fffffff;
      r.nan = 0;
      if constexpr (EPI == SG_ROPE) {
        if (r.live) {
          r.slot = j.st[r.b].base + r.jr;
          r.page = j.pt[r.b * j.pps + r.slot / kAttnChunk];
        }
      }
    }
  };
  int npend = 0;
  // The workers and the control wave run separate loops (the branch is on a
  // wave-uniform value) with one workgroup barrier per tile each, so that
  // the workers' code holds nothing but weight loads and MFMAs.  The barrier
  // waits for LDS traffic only: the control wave's stores stay in flight.
  if (wave > 0 && XS) {
    // streamed x: a tile's steps are taken DEP at a time; slot i holds
    // step g * DEP + i of the worker's range, and is refilled (weights and
    // x) with the same slot of the next group, or of the next tile's first
    const int NG = (nst + DEP - 1) / DEP;
    for (int it = 0; it < n_it; ++it) {
      f32x4 acc[MB];
#pragma unroll
      for (int rb = 0; rb < MB; ++rb) acc[rb] = f32x4{0.f, 0.f, 0.f, 0.f};
      for (int g = 0; g < NG; ++g) {
        const bool lastg = g + 1 == NG;
        const int nit = lastg ? it + 1 : it, ng = lastg ? 0 : g + 1;
        const bool nv = nit < n_it;
        const int vn = (tile_of(nv ? nit : it) * T + ws0 + ng * DEP) * 1024 + lane_off;
#pragma unroll
        for (int i = 0; i < DEP; ++i) {
#pragma unroll
          for (int rb = 0; rb < MB; ++rb) acc[rb] = mfma16x16x32(wv[i], xok[rb] ? xv[rb][i] : u32x4{0, 0, 0, 0}, acc[rb]);
          const int sn = ng * DEP + i;
          const bool on = nv && sn < nst;
          wv[i] = __builtin_amdgcn_raw_buffer_load_b128(rs, on ? vn + 1024 * i : kOut, 0, kNt);
#pragma unroll
          for (int rb = 0; rb < MB; ++rb)
            xv[rb][i] = __builtin_amdgcn_raw_buffer_load_b128(rsx, on ? x_off(rb, ws0 + sn) : kOut, 0, 0);
        }
      }
#pragma unroll
      for (int rb = 0; rb < MB; ++rb) red[(((it & 1) * MB + rb) * kSgWorkers + wi) * 64 + lane] = acc[rb];
      lds_barrier();
    }
  } else if (wave > 0) {
    for (int it = 0; it < n_it; ++it) {
      const bool na = it + 1 < n_it;
      const int vn = (tile_of(it + 1) * T + ws0) * 1024 + lane_off;
      f32x4 acc[MB];
#pragma unroll
      for (int rb = 0; rb < MB; ++rb) acc[rb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int i = 0; i < DEP; ++i) {
        const bool on = i < nst;
#pragma unroll
        for (int rb = 0; rb < MB; ++rb) acc[rb] = mfma16x16x32(wv[i], xv[rb][i], acc[rb]);
        wv[i] = __builtin_amdgcn_raw_buffer_load_b128(rs, (na && on) ? vn + 1024 * i : kOut, 0, kNt);
      }
#pragma unroll
      for (int rb = 0; rb < MB; ++rb) red[(((it & 1) * MB + rb) * kSgWorkers + wi) * 64 + lane] = acc[rb];
      lds_barrier();
    }
  } else {
    RowInfo ri[MB];
    row_info(ri);
    // normalised inputs: 1/rms of each row from the producer's per-16-column
    // sums of squares: lane (t, q) reads rows 16 rb + 4q .. +3 of sum t =
    // lane / 4, 16 sums per load; the 16 lanes of each q are then added by an
    // xor butterfly, which gives every lane bit-identical totals
    if constexpr (kNorm) {
      const int ntt = j.Hn / kTile;
      const int q = lane & 3;
#pragma unroll
      for (int rb = 0; rb < MB; ++rb) {
        f32x4 acc4 = f32x4{0.f, 0.f, 0.f, 0.f};
        for (int t0 = lane >> 2; t0 < ntt; t0 += 16 * 8) {
          f32x4 tmp[8];
#pragma unroll
          for (int b = 0; b < 8; ++b) {
            const int tt = t0 + 16 * b;
            tmp[b] = tt < ntt ? *reinterpret_cast<const f32x4*>(j.ss_in + (size_t)tt * j.mpad + 16 * rb + 4 * q)
                              : f32x4{0.f, 0.f, 0.f, 0.f};
          }
#pragma unroll
          for (int b = 0; b < 8; ++b) acc4 += tmp[b];
        }
#pragma unroll
        for (int o = 4; o < 64; o <<= 1) {
          acc4.x += __shfl_xor(acc4.x, o);
          acc4.y += __shfl_xor(acc4.y, o);
          acc4.z += __shfl_xor(acc4.z, o);
          acc4.w += __shfl_xor(acc4.w, o);
        }
        const int src = m0 >> 2;
        const float c0 = __shfl(acc4.x, src), c1 = __shfl(acc4.y, src), c2 = __shfl(acc4.z, src),
                    c3 = __shfl(acc4.w, src);
        const int c = m0 & 3;
        const float sum = c == 0 ? c0 : c == 1 ? c1 : c == 2 ? c2 : c3;
        ri[rb].inv_rms = rsqrtf(sum / j.Hn + j.eps);
        if (lane < 16) rms_sh[16 * rb + lane] = ri[rb].inv_rms;
      }
    }
    f32x4 ya[MB], yb[MB];
#pragma unroll
    for (int rb = 0; rb < MB; ++rb) ya[rb] = yb[rb] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int it = 0; it < n_it; ++it) {
      const int t = tile_of(it);
      f32x4 pa[MB];
      u32x2 pb[MB];
#pragma unroll
      for (int rb = 0; rb < MB; ++rb)
        epilogue_inputs<EPI>(j, ri[rb], rb, t / TPU, pa[rb], pb[rb]);   // in flight while the workers stream tile t
      lds_barrier();
      const int u = t / TPU, half = t - u * TPU;
#pragma unroll
      for (int rb = 0; rb < MB; ++rb) {
        const f32x4* rr = red + ((it & 1) * MB + rb) * kSgWorkers * 64 + lane;
        f32x4 y = rr[0];
#pragma unroll
        for (int w = 1; w < kSgWorkers; ++w) y += rr[w * 64];
        if (half == 0) {
          ya[rb] = y;
          yb[rb] = f32x4{0.f, 0.f, 0.f, 0.f};
        } else {
          yb[rb] = y;
        }
      }
      if (half == TPU - 1 || it == n_it - 1) {
        if (S == 1) {
#pragma unroll
          for (int rb = 0; rb < MB; ++rb) epilogue<EPI>(j, ri[rb], rb, u, ya[rb], yb[rb], pa[rb], pb[rb]);
        } else {
          const int k = it / TPU;   // partial slot: this workgroup's k-th unit
#pragma unroll
          for (int rb = 0; rb < MB; ++rb) {
            float* pp = j.part + ((((size_t)blockIdx.x * j.kmax + k) * MB + rb) * 2) * 256;
            *reinterpret_cast<f32x4*>(pp + lane * 4) = ya[rb];
            if (kPair) *reinterpret_cast<f32x4*>(pp + 256 + lane * 4) = yb[rb];
          }
          if (lane == 0) pend[npend] = u;
          ++npend;
        }
#pragma unroll
        for (int rb = 0; rb < MB; ++rb) ya[rb] = f32x4{0.f, 0.f, 0.f, 0.f};
      }
    }
    if constexpr (EPI == SG_ARGMAX) {
      if (S == 1 && lane < 16) {   // lanes 0..15 hold rows 16 rb .. 16 rb + 15
#pragma unroll
        for (int rb = 0; rb < MB; ++rb) {
          const int m = lane + 16 * rb;
          if (m < M) {
            float* pv = j.amax_v + (size_t)gi * j.mpad + m;
            int32_t* pi = j.amax_i + (size_t)gi * j.mpad + m;
            if (j.tail) {   // read by the last workgroup, possibly on another XCD
              st_coh_u32(pv, __float_as_uint(ri[rb].best));
              st_coh_u32(pi, (uint32_t)ri[rb].bi);
            } else {
              *pv = ri[rb].best;
              *pi = ri[rb].bi;
            }
            if (ri[rb].nan) atomicOr(const_cast<int32_t*>(&j.st[ri[rb].b].err), ERR_NUMERIC);
          }
        }
      }
    }
  }


  // k-sliced reductions: unit u's partials come from workgroup u % G of every
  // slice, slot u / G.  The control wave counts this workgroup in on all of
  // its units at once (one atomic per lane); the units it completes last are
  // then finished by all waves in parallel, each adding the partials of its
  // unit in slice order.
  if (wave == 0 && lane == 0) pend[kSgPendMax] = npend;
  __syncthreads();
  const int np = pend[kSgPendMax];
  if (np > 0) {
    constexpr int kMine = 1 << 30;
    if (wave == 0) {
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");   // partial stores reach memory first
      for (int p = lane; p < np; p += 64) {
        const int u = pend[p];
        const unsigned old = __hip_atomic_fetch_add(j.cnt + u, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (old + 1 == (unsigned)S) pend[p] = u | kMine;
      }
    }
    __syncthreads();
    RowInfo ri[MB];
    row_info(ri);
    if constexpr (kNorm) {
#pragma unroll
      for (int rb = 0; rb < MB; ++rb) ri[rb].inv_rms = rms_sh[16 * rb + m0];
    }
    for (int p = wave; p < np; p += kSgWaves) {
      const int e = pend[p];
      if (!(e & kMine)) continue;
      const int u = e & ~kMine;
#pragma unroll
      for (int rb = 0; rb < MB; ++rb) {
        f32x4 pa;
        u32x2 pb;
        epilogue_inputs<EPI>(j, ri[rb], rb, u, pa, pb);
        // The partials of up to kBatch slices are loaded together, then added
        // in slice order: one memory round trip per batch, not per slice.
        constexpr int kBatch = kPair ? 4 : 8;
        f32x4 sa = f32x4{0.f, 0.f, 0.f, 0.f}, sb = sa;
        for (int s0 = 0; s0 < S; s0 += kBatch) {
          f32x4 va[kBatch], vb[kBatch];
#pragma unroll
          for (int i = 0; i < kBatch; ++i) {
            const int s2 = min(s0 + i, S - 1);
            const float* pp = j.part + ((((size_t)(s2 * G + u % G) * j.kmax + u / G) * MB + rb) * 2) * 256;
            va[i] = ld_coh4(pp + lane * 4);
            if (kPair) vb[i] = ld_coh4(pp + 256 + lane * 4);
          }
#pragma unroll
          for (int i = 0; i < kBatch; ++i)
            if (s0 + i < S) {
              sa += va[i];
              if (kPair) sb += vb[i];
            }
        }
        epilogue<EPI>(j, ri[rb], rb, u, sa, sb, pa, pb);
      }
      if (lane == 0) __hip_atomic_store(j.cnt + u, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }

  if constexpr (EPI == SG_ARGMAX) {
    if (S == 1 && j.tail) {
      // The pairs of this workgroup are stored (coherently, awaited); the
      // workgroup that arrives last reduces every row over all G pairs.
      if (wave == 0) {
        wait_vmem();
        if (lane == 0) {
          const unsigned t = __hip_atomic_fetch_add(j.tail_cnt, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          pend[kSgPendMax + 1] = t + 1 == (unsigned)G ? 1 : 0;
        }
      }
      __syncthreads();
      if (pend[kSgPendMax + 1]) {
        for (int m = wave; m < M; m += kSgWaves) {   // one row per wave
          float best = -INFINITY;
          int bi = 0x7fffffff;
          for (int g = lane; g < G; g += 64)
            amax_merge(best, bi, __uint_as_float(ld_coh_u32(j.amax_v + (size_t)g * j.mpad + m)),
                       (int)ld_coh_u32(j.amax_i + (size_t)g * j.mpad + m));
#pragma unroll
          for (int o = 32; o > 0; o >>= 1) {
            const float v2 = __shfl_xor(best, o);
            const int i2 = __shfl_xor(bi, o);
            amax_merge(best, bi, v2, i2);
          }
          if (lane == 0) {
            SeqState& s = const_cast<SeqState*>(j.st)[m / j.rps];
            const int jr = m % j.rps;
            if (j.tail == 1) {
              if (jr < s.count) s.rstar[jr] = bi;
            } else if (s.count == 0) {   // a draft step that proposed nothing for this sequence
              if (j.tail_out && s.dcall < j.tail_K) j.tail_out[(m / j.rps) * j.tail_K + s.dcall] = -1;
              s.dcall += 1;
            } else {
              s.props[s.dstep] = bi;
              s.draft_len = s.base + s.count;
              s.dstep += 1;
              if (j.tail_out && s.dcall < j.tail_K) j.tail_out[(m / j.rps) * j.tail_K + s.dcall] = bi;
              s.dcall += 1;
            }
          }
        }
        if (threadIdx.x == 0) __hip_atomic_store(j.tail_cnt, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
  }
}

// Packs row-major weights into the tile layout; one thread per 16-byte block.
__global__ void k_pack(bf16_t* dst, PackSrc p) {
  const size_t nvec = (size_t)p.ntiles * p.T * 64;
  for (size_t v = (size_t)blockIdx.x * blockDim.x + threadIdx.x; v < nvec; v += (size_t)gridDim.x * blockDim.x) {
    const int lane = (int)(v & 63);
    const size_t ts = v >> 6;
    const int step = (int)(ts % p.T), tile = (int)(ts / p.T);
    const int r = lane & 15, k = step * 32 + 8 * (lane >> 4);
    const bf16_t* row;
    if (p.pair) {
      row = p.seg[tile & 1] + (size_t)((tile >> 1) * 16 + r) * p.Kd;
    } else {
      const int n = tile * 16 + r;
      int sg = 0;
      for (int i = 1; i < 3; ++i)
        if (i < p.nseg && n >= p.row0[i]) sg = i;
      row = p.seg[sg] + (size_t)(n - p.row0[sg]) * p.Kd;
    }
    u32x4 val = u32x4{0, 0, 0, 0};
    if (k < p.Kd) val = *reinterpret_cast<const u32x4*>(row + k);
    *reinterpret_cast<u32x4*>(dst + v * 8) = val;
  }
}

}  // namespace

size_t sg_packed_elems(int ntiles, int T) { return (size_t)ntiles * T * 64 * 8; }

// Row blocks of 16 rows of a job.
int sg_row_blocks(const SgJob& j) { return (j.M + 15) / 16; }

size_t sg_lds_bytes(const SgJob& j) {
  const int MB = sg_row_blocks(j);
  return 2 * (size_t)MB * kSgWorkers * 64 * 16 + (kSgPendMax + 4) * sizeof(int) + 16 * MB * sizeof(float);
}

size_t sg_part_floats(const SgJob& j) { return (size_t)j.S * j.G * j.kmax * sg_row_blocks(j) * 2 * 256; }

bool sg_plan(SgJob& j, int epi, int ncu, int lds_limit) {
  const int tpu = epi == SG_SWIGLU ? 2 : 1;
  if (j.ntiles < 1 || j.ntiles % tpu || j.M < 1 || j.M > kSgMaxRows || j.T < 1 || j.rps < 1 || ncu < 1) return false;
  if ((long long)j.ntiles * j.T * 1024 >= kOut || (long long)j.M * j.ldx * 2 >= kOut) return false;
  // A k-range longer than the workers can hold x for is streamed (x loaded
  // with the weights, step by step), which needs no partial tiles and no
  // cross-workgroup fixup, unless k-slices share the work evenly (below).
  // x is held in registers while every worker's share of a tile's steps fits
  // its buffer (8 steps, or 9 for the 4096-wide inputs of the paper's
  // backbone); a row's sum is formed the same way in every variant
  j.xs = j.T > kSgWorkers * kSgDepthMax ? 1 : 0;
  int smin = 1;
  if (j.xs) {
    // k-slices short enough for x in registers (at most kSgDepth steps per
    // worker) instead of streamed x, where the slices' workgroups then share
    // the units evenly: no x re-read from L2 with every weight block, at the
    // price of partial tiles (the paper backbone's down projection: 4 slices
    // of 96 steps, 64 workgroups of 4 tiles each).  The choice depends on the
    // shape only, so every pass of a context sums a row the same way.
    const int sx = (j.T + kSgMaxSpan - 1) / kSgMaxSpan;
    const int gx = ncu / sx;
    const int units = j.ntiles / tpu;
    if (ncu % sx == 0 && gx > 0 && gx <= units && units % gx == 0 && (units / gx) <= kSgPendMax) {
      j.xs = 0;
      smin = sx;
    }
  }
  j.dep9 = (!j.xs && (j.T + smin - 1) / smin > kSgMaxSpan) ? 1 : 0;
  int S = smin;
  for (int s = smin; s <= 2 * smin; ++s)
    if (ncu % s == 0) {
      S = s;
      break;
    }
  for (;; ++S) {
    if (S > j.T) return false;
    j.S = S;
    if (sg_lds_bytes(j) <= (size_t)lds_limit) break;
  }
  j.units = j.ntiles / tpu;
  j.G = std::max(1, std::min(ncu / S, j.units));
  // partial slots (k-sliced reductions): one per unit of a workgroup
  const int kmax = S > 1 ? (j.units + j.G - 1) / j.G : 1;
  if (kmax > kSgPendMax) return false;
  j.kmax = kmax;
  j.amax_n = S == 1 ? j.G : j.ntiles;
  return true;
}

hipError_t sg_launch(int epi, const SgJob& h, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  const dim3 grid(h.S * h.G), block(kSgWaves * 64);
  const uint32_t lds = (uint32_t)sg_lds_bytes(h);
  const bool two = sg_row_blocks(h) == 2;
#define SG_PICK(E, XS_, D)                                                                              \
  hipExtLaunchKernelGGL(two ? k_sgemv<E, XS_, 2, D> : k_sgemv<E, XS_, 1, D>, grid, block, lds, s, e0, e1, 0, h)
#define SG_CASE(E)                                  \
  case E:                                           \
    if (h.xs)                                       \
      SG_PICK(E, true, kSgDepth);                   \
    else if (h.dep9)                                \
      SG_PICK(E, false, kSgDepthMax);               \
    else                                            \
      SG_PICK(E, false, kSgDepth);                  \
    break;
  switch (epi) {
    SG_CASE(SG_ROPE)
    SG_CASE(SG_RESID)
    SG_CASE(SG_SWIGLU)
    SG_CASE(SG_DOWN)
    SG_CASE(SG_ARGMAX)
    default: return hipErrorInvalidValue;
  }
#undef SG_CASE
#undef SG_PICK
  return hipGetLastError();
}

hipError_t sg_pack(bf16_t* dst, const PackSrc& src, hipStream_t s) {
  const size_t nvec = (size_t)src.ntiles * src.T * 64;
  const int blocks = (int)std::min<size_t>((nvec + 255) / 256, 16384);
  hipLaunchKernelGGL(k_pack, dim3(blocks), dim3(256), 0, s, dst, src);
  return hipGetLastError();
}

template <int E>
void sg_set_attr(int lds_limit) {
  const void* fns[] = {reinterpret_cast<const void*>(&k_sgemv<E, false, 1, kSgDepth>),
                       reinterpret_cast<const void*>(&k_sgemv<E, true, 1, kSgDepth>),
                       reinterpret_cast<const void*>(&k_sgemv<E, false, 2, kSgDepth>),
                       reinterpret_cast<const void*>(&k_sgemv<E, true, 2, kSgDepth>),
                       reinterpret_cast<const void*>(&k_sgemv<E, false, 1, kSgDepthMax>),
                       reinterpret_cast<const void*>(&k_sgemv<E, false, 2, kSgDepthMax>)};
  for (const void* f : fns) (void)hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, lds_limit);
}

void sg_set_attributes(int lds_limit) {
  sg_set_attr<SG_ROPE>(lds_limit);
  sg_set_attr<SG_RESID>(lds_limit);
  sg_set_attr<SG_SWIGLU>(lds_limit);
  sg_set_attr<SG_DOWN>(lds_limit);
  sg_set_attr<SG_ARGMAX>(lds_limit);
}

}  // namespace specdec
