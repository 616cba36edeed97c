// The SGD step for models whose W1 does not fit in a workgroup's LDS (hidden
// layer wider than 64 units, e.g. d 128, window 11, H 256): three MFMA
// contractions (16x16x4 f32) with the embedding rows gathered on the fly.
//
//   k_large_fwd   Z = X W1^T and, for the corrupted copy, the centre-block
//                 difference D = (e~ - e_c) W1_c^T (so z~ = z + D; §1 model,
//                 x~); then tanh, both scores, hinge and the per-window
//                 vectors V = (dz + dz~, dz, dz~), written to global memory,
//                 and this workgroup's db1 / dw2 / loss partial.  32 windows
//                 per workgroup, one wave per 64 hidden units.  In score-only
//                 mode it writes s(x) instead.
//   k_large_dw1   dW1 partials: dW1[h][k] = sum_b V_b[h] x_b[k] (centre block:
//                 dz e_c + dz~ e~) over 1024-window slices; a workgroup owns a
//                 64 x KT block of dW1 (KT = 128 when d allows, else 64) and
//                 one slice, its operands staged through LDS.
//   k_large_g     G[e][:] = W1_j^T V for entry e = b(win+1) + j (context
//                 positions dz + dz~, the true centre dz, the corrupt entry dz~
//                 through block c); a workgroup owns 64 windows of one entry
//                 position.
// Rows b >= B read row 0 and are masked out of every result.
#pragma once
#include "common.h"
#include "launch.h"

namespace pg {

__device__ __forceinline__ f4 lg_mfma(float a, float b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// HW waves, wave w owns hidden units [64w, 64w + 64) (4 column blocks of 16);
// both 16-row blocks of the workgroup's 32 windows.
template <int HW>
__global__ __launch_bounds__(HW * kWave) void k_large_fwd(LargeArgs a, int score_only) {
  __shared__ int32_t ids[kLgRows][kMaxWin + 1];
  __shared__ float sred[2][HW][kLgRows];
  __shared__ float gsh[kLgRows];
  __shared__ int badrow[kLgRows];
  const int t = threadIdx.x, lane = t & (kWave - 1);
  const int w = __builtin_amdgcn_readfirstlane(t / kWave);
  const int i = lane & 15, g = lane >> 4;
  const int r0 = blockIdx.x * kLgRows;
  const int W1p = a.win + 1, d = a.d, K = a.K;
  if (t < kLgRows) badrow[t] = 0;
  __syncthreads();
  for (int k = t; k < kLgRows * W1p; k += HW * kWave) {
    const int r = k / W1p, j = k - r * W1p;
    const int b = r0 + r;
    int32_t id = 0;  // score-only mode has no corrupt ids
    if (b < a.B && (j < a.win || !score_only))
      id = j < a.win ? a.windows[(size_t)b * a.win + j] : a.corrupt[b];
    const bool bad = (uint32_t)id >= (uint32_t)a.V_rows;
    if (bad) {
      atomicOr(a.flag, kFlagBadId);
      badrow[r] = 1;
    }
    ids[r][j] = ((uint32_t)id < (uint32_t)a.V_rows) ? id : 0;
  }
  __syncthreads();

  f4 Z[2][4], D[2][4];
#pragma unroll
  for (int rb = 0; rb < 2; ++rb)
#pragma unroll
    for (int cb = 0; cb < 4; ++cb) Z[rb][cb] = D[rb][cb] = kZero4;
  const int cpb = d / 16;  // 16-column chunks per embedding row
  const int nch = K / 16;
  // Chunk kc (16 columns of x) goes through LDS, row-major with 16-byte
  // rows padded to 20 floats: Xs (the 32 windows' rows), Ts (the corrupt
  // rows, centre block only) and Ws (W1 rows of all H units).  Lane (i, g)
  // reads Xs[16rb+i][4g] and Ws[64w+16cb+i][4g] as float4: its operands of
  // the four MFMAs (q) of the chunk.  The 256 float4 of Xs and Ts (item x:
  // Xs for x < 128, else Ts; row (x&127)/4, column 4(x&3)) and the 64*HW*4
  // float4 of Ws are spread over the workgroup's threads.
  constexpr int NT = HW * kWave, XP = 20;
  constexpr int XPT = (256 + NT - 1) / NT;  // float4 of Xs / Ts per thread
  constexpr int WPT = (64 * HW * 4) / NT;   // float4 of W1 rows per thread (= 4)
  __shared__ __align__(16) float Xs[2][kLgRows][XP];
  __shared__ __align__(16) float Ts[2][kLgRows][XP];
  __shared__ __align__(16) float Ws[2][64 * HW][XP];
  auto load = [&](int kc, f4 (&Xv)[XPT], f4 (&Wv)[WPT]) {
    const int jb = kc / cpb, off = (kc - jb * cpb) * 16;
    const bool ctr = jb == a.c && !score_only;
#pragma unroll
    for (int u = 0; u < XPT; ++u) {
      const int x = t + u * NT;
      const int xr = (x & 127) / 4, xc = 4 * (x & 3);
      if (x < 128) Xv[u] = ld4(a.E + (size_t)ids[xr][jb] * d + off + xc);
      else if (x < 256 && ctr) Xv[u] = ld4(a.E + (size_t)ids[xr][a.win] * d + off + xc);
    }
#pragma unroll
    for (int u = 0; u < WPT; ++u) {
      const int x = t + u * NT;
      Wv[u] = ld4(a.W1 + (size_t)(x / 4) * K + 16 * kc + 4 * (x & 3));
    }
  };
  auto store = [&](int buf, int kc, const f4 (&Xv)[XPT], const f4 (&Wv)[WPT]) {
    const bool ctr = kc / cpb == a.c && !score_only;
#pragma unroll
    for (int u = 0; u < XPT; ++u) {
      const int x = t + u * NT;
      const int xr = (x & 127) / 4, xc = 4 * (x & 3);
      if (x < 128) st4(&Xs[buf][xr][xc], Xv[u]);
      else if (x < 256 && ctr) st4(&Ts[buf][xr][xc], Xv[u]);
    }
#pragma unroll
    for (int u = 0; u < WPT; ++u) {
      const int x = t + u * NT;
      st4(&Ws[buf][x / 4][4 * (x & 3)], Wv[u]);
    }
  };
  auto compute = [&](int buf, int kc) {
    f4 A[2], Bv[4];
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) A[rb] = ld4(&Xs[buf][16 * rb + i][4 * g]);
#pragma unroll
    for (int cb = 0; cb < 4; ++cb) Bv[cb] = ld4(&Ws[buf][64 * w + 16 * cb + i][4 * g]);
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
      for (int rb = 0; rb < 2; ++rb)
#pragma unroll
        for (int cb = 0; cb < 4; ++cb) Z[rb][cb] = lg_mfma(A[rb][q], Bv[cb][q], Z[rb][cb]);
    if (kc / cpb == a.c && !score_only) {  // D = (e~ - e_c) W1_c^T
      f4 At[2];
#pragma unroll
      for (int rb = 0; rb < 2; ++rb) At[rb] = ld4(&Ts[buf][16 * rb + i][4 * g]);
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int rb = 0; rb < 2; ++rb) {
          const float dx = At[rb][q] - A[rb][q];
#pragma unroll
          for (int cb = 0; cb < 4; ++cb) D[rb][cb] = lg_mfma(dx, Bv[cb][q], D[rb][cb]);
        }
    }
  };
  // two register sets: chunk kc+2 is loaded while chunks kc and kc+1 are
  // contracted; one barrier per chunk (the buffer written at chunk kc was
  // last read at chunk kc-2, before chunk kc-1's barrier)
  f4 XA[XPT], WA[WPT], XB[XPT], WB[WPT];
#pragma unroll
  for (int u = 0; u < XPT; ++u) XA[u] = XB[u] = kZero4;
  load(0, XA, WA);
  if (nch > 1) load(1, XB, WB);
  for (int kc = 0; kc < nch; kc += 2) {
    store(0, kc, XA, WA);
    if (kc + 2 < nch) load(kc + 2, XA, WA);
    __syncthreads();
    compute(0, kc);
    if (kc + 1 >= nch) break;
    store(1, kc + 1, XB, WB);
    if (kc + 3 < nch) load(kc + 3, XB, WB);
    __syncthreads();
    compute(1, kc + 1);
  }

  // ---- epilogue.  Lane (i, g), component q of Z[rb][cb]: row 16rb + 4g + q,
  // hidden 64w + 16cb + i.
  float b1v[4], w2v[4];
#pragma unroll
  for (int cb = 0; cb < 4; ++cb) {
    const int h = 64 * w + 16 * cb + i;
    b1v[cb] = h < a.H ? a.b1[h] : 0.f;
    w2v[cb] = h < a.H ? a.w2[h] : 0.f;
  }
  float ps[2][4], pst[2][4];
#pragma unroll
  for (int rb = 0; rb < 2; ++rb)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      float s = 0.f, st = 0.f;
#pragma unroll
      for (int cb = 0; cb < 4; ++cb) {
        const float z = Z[rb][cb][q] + b1v[cb];
        s += w2v[cb] * tanh_fast(z);
        if (!score_only) st += w2v[cb] * tanh_fast(z + D[rb][cb][q]);
      }
#pragma unroll
      for (int o = 1; o < 16; o <<= 1) {
        s += __shfl_xor(s, o);
        st += __shfl_xor(st, o);
      }
      ps[rb][q] = s;
      pst[rb][q] = st;
    }
  if (i == 0) {
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        sred[0][w][16 * rb + 4 * g + q] = ps[rb][q];
        sred[1][w][16 * rb + 4 * g + q] = pst[rb][q];
      }
  }
  __syncthreads();
  float lossr = 0.f;
  if (t < kLgRows) {
    float s = 0.f, st = 0.f;
#pragma unroll
    for (int v = 0; v < HW; ++v) {
      s += sred[0][v][t];
      st += sred[1][v][t];
    }
    const int b = r0 + t;
    const float b2v = a.b2[0];
    if (score_only) {
      if (b < a.B) a.scores[b] = badrow[t] ? __builtin_nanf("") : b2v + s;
    } else {
      const float mg = 1.f - (b2v + s) + (b2v + st);
      const bool on = b < a.B && mg > 0.f;  // hinge active (derivative 0 at margin 0)
      gsh[t] = on ? a.invB : 0.f;           // d loss/d s~ = m/B, d loss/d s = -m/B
      lossr = on ? mg : 0.f;
    }
  }
  if (score_only) return;
  __syncthreads();

  // V and the db1 / dw2 sums of this lane's hidden units over its 8 rows
  float db1[4] = {0.f, 0.f, 0.f, 0.f}, dw2[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int rb = 0; rb < 2; ++rb)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int r = 16 * rb + 4 * g + q, b = r0 + r;
      const float gst = gsh[r];
#pragma unroll
      for (int cb = 0; cb < 4; ++cb) {
        const int h = 64 * w + 16 * cb + i;
        const float z = Z[rb][cb][q] + b1v[cb];
        const float hh = tanh_fast(z), ht = tanh_fast(z + D[rb][cb][q]);
        // h - h~ = tanh(z - z~) (1 - h h~) with z - z~ = -D
        const float hmh = tanh_fast(-D[rb][cb][q]) * (1.f - hh * ht);
        const float gw = gst * w2v[cb];
        const float dz = -gw * (1.f - hh * hh);
        const float dzt = gw * (1.f - ht * ht);
        const float dsum = gw * hmh * (hh + ht);
        if (b < a.B && h < a.H) {
          float* vr = a.V + (size_t)b * 3 * a.H + h;
          vr[0] = dsum;
          vr[a.H] = dz;
          vr[2 * a.H] = dzt;
        }
        db1[cb] += dsum;
        dw2[cb] -= gst * hmh;  // -(m/B) h + (m/B) h~
      }
    }
  float* vp = a.vpart + (size_t)blockIdx.x * (2 * a.H + 2);
#pragma unroll
  for (int cb = 0; cb < 4; ++cb) {
    float x = db1[cb], y = dw2[cb];
    x += __shfl_xor(x, 16);
    x += __shfl_xor(x, 32);
    y += __shfl_xor(y, 16);
    y += __shfl_xor(y, 32);
    const int h = 64 * w + 16 * cb + i;
    if (g == 0 && h < a.H) {
      vp[h] = x;
      vp[a.H + h] = y;
    }
  }
  if (w == 0) {  // the workgroup's hinge sum (rows in order), db2 = 0
    for (int o = 1; o < kWave; o <<= 1) lossr += __shfl_xor(lossr, o);
    if (lane == 0) {
      vp[2 * a.H] = lossr;
      vp[2 * a.H + 1] = 0.f;
    }
  }
}

// dW1 partial of a 64 x KT block (hidden h0.., columns k0.. inside one
// window position j) over one 1024-window slice.  The operands go through
// LDS in 16-window blocks, row-major (one window per row):
//   Vs[w][h]   = the window's vector for this position (dz + dz~ for a
//                context position; dz, then dz~ in a second phase, for the
//                centre, whose rows are the true centre and the corrupt word)
//   Xs[w][col] = E[id(w, j)][off0 + col]
// MFMA q of a block contracts windows {q, 4+q, 8+q, 12+q}: lane (i, g)
// supplies Vs[4g+q][16rt+i] and Xs[4g+q][16ct+i].  Row strides are 4 mod 8
// floats, so the two row groups a half-wave reads sit on disjoint banks,
// and a row is stored with float4 writes.  Wave w owns columns
// [w*KT/4, (w+1)*KT/4) and all 64 hidden rows.  The slice's row ids are
// staged in LDS first; rows two blocks ahead are in flight in registers.
template <int KT>
__global__ __launch_bounds__(kBlock) void k_large_dw1(LargeArgs a) {
  constexpr int CT = KT / 64;          // 16-column tiles per wave
  constexpr int XF = 16 * KT / 4;      // float4 of one block's rows
  constexpr int XPT = XF / kBlock;     // ... per thread
  constexpr int XS = KT + 4, VS = 64 + 4;
  __shared__ __align__(16) float Vs[2][16][VS];
  __shared__ __align__(16) float Xs[2][16][XS];
  __shared__ int32_t ids_s[2][kLgSlice];  // row ids of the slice, per phase
  const int t = threadIdx.x, lane = t & (kWave - 1);
  const int w = __builtin_amdgcn_readfirstlane(t / kWave);
  const int i = lane & 15, g = lane >> 4;
  const int h0 = blockIdx.x * 64, k0 = blockIdx.y * KT, sl = blockIdx.z;
  const int d = a.d, j = k0 / d, off0 = k0 - j * d;
  const int phases = (j == a.c) ? 2 : 1;
  const int b_lo = sl * kLgSlice, b_hi = min(a.B, b_lo + kLgSlice), nb = b_hi - b_lo;
  const int nblk = (nb + 15) / 16, total = phases * nblk;

  // every row id of the slice up front, so a block's row loads depend on LDS only
  for (int x = t; x < nb; x += kBlock) {
    const int32_t id0 = a.windows[(size_t)(b_lo + x) * a.win + j];
    ids_s[0][x] = (uint32_t)id0 < (uint32_t)a.V_rows ? id0 : 0;
    if (phases == 2) {
      const int32_t id1 = a.corrupt[b_lo + x];
      ids_s[1][x] = (uint32_t)id1 < (uint32_t)a.V_rows ? id1 : 0;
    }
  }
  __syncthreads();

  // this thread's share of a block: XPT float4 of rows (window xw[u], float4
  // column xc), one float4 of vectors (window t/16, hidden 4*(t%16))
  const int xc = t % (KT / 4);
  int xw[XPT];
#pragma unroll
  for (int u = 0; u < XPT; ++u) xw[u] = (t + u * kBlock) / (KT / 4);
  const int vw = t / 16, vh = 4 * (t % 16);
  auto load = [&](int bi, f4 (&X)[XPT], f4& Vv) {
    const int ph = bi / nblk, r0 = (bi - ph * nblk) * 16;
    const int slot = (phases == 1) ? 0 : 1 + ph;
#pragma unroll
    for (int u = 0; u < XPT; ++u) {
      const int r = r0 + xw[u];
      const int32_t id = r < nb ? ids_s[ph][r] : 0;
      X[u] = ld4(a.E + (size_t)id * d + off0 + 4 * xc);
    }
    const int r = r0 + vw;
    Vv = r < nb ? ld4(a.V + (size_t)(b_lo + r) * 3 * a.H + (size_t)slot * a.H + h0 + vh) : kZero4;
  };
  auto store = [&](int buf, const f4 (&X)[XPT], const f4& Vv) {
#pragma unroll
    for (int u = 0; u < XPT; ++u) st4(&Xs[buf][xw[u]][4 * xc], X[u]);
    st4(&Vs[buf][vw][vh], Vv);
  };
  f4 acc[4][CT];
#pragma unroll
  for (int rt = 0; rt < 4; ++rt)
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) acc[rt][ct] = kZero4;
  auto compute = [&](int buf) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      float A[4], Bm[CT];
#pragma unroll
      for (int rt = 0; rt < 4; ++rt) A[rt] = Vs[buf][4 * g + q][16 * rt + i];
#pragma unroll
      for (int ct = 0; ct < CT; ++ct) Bm[ct] = Xs[buf][4 * g + q][16 * (w * CT + ct) + i];
#pragma unroll
      for (int rt = 0; rt < 4; ++rt)
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) acc[rt][ct] = lg_mfma(A[rt], Bm[ct], acc[rt][ct]);
    }
  };

  // two register sets: the rows of block bi+2 are loaded while blocks bi and
  // bi+1 are contracted.  One barrier per block: the LDS buffer written at
  // block bi was last read at block bi-2, before block bi-1's barrier.
  f4 XA[XPT], VA, XB[XPT], VB;
  if (total > 0) load(0, XA, VA);
  if (total > 1) load(1, XB, VB);
  for (int bi = 0; bi < total; bi += 2) {
    store(0, XA, VA);
    if (bi + 2 < total) load(bi + 2, XA, VA);
    __syncthreads();
    compute(0);
    if (bi + 1 >= total) break;
    store(1, XB, VB);
    if (bi + 3 < total) load(bi + 3, XB, VB);
    __syncthreads();
    compute(1);
  }
  // lane (i, g), component r: hidden h0 + 16rt + 4g + r, column k0 + 16(w*CT + ct) + i
  float* P = a.part + (size_t)sl * a.H * a.K;
#pragma unroll
  for (int rt = 0; rt < 4; ++rt)
#pragma unroll
    for (int ct = 0; ct < CT; ++ct)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        P[(size_t)(h0 + 16 * rt + 4 * g + r) * a.K + k0 + 16 * (w * CT + ct) + i] = acc[rt][ct][r];
}

// G rows of 64 windows at entry position j = blockIdx.y:
// G[b(win+1)+j][:] = W1_jj^T v_b (jj = c for the corrupt entry).  The
// contraction over hidden units goes in 16-unit steps through LDS,
// row-major: Vs[w][h] (the window's vector for this position) and
// Ws[h][col] (W1 rows hc.. of column block jj).  MFMA q of a step contracts
// units {q, 4+q, 8+q, 12+q}: lane (i, g) supplies Vs[16w'+i][4g+q] (one
// 128-bit read for all four) and Ws[4g+q][16ct+i]; Ws rows are 4 mod 8
// floats long, so a half-wave's two rows sit on disjoint banks.  Wave w'
// owns windows 16w'.. and all DQ column blocks; the rows of step s+2 are in
// flight in registers while steps s and s+1 are contracted.
template <int DQ>
__global__ __launch_bounds__(kBlock) void k_large_g(LargeArgs a) {
  constexpr int D = 16 * DQ, WS = D + 4, VS = 16 + 4;
  constexpr int WF = 16 * D / 4;                     // float4 of a step's W1 rows
  constexpr int WPT = (WF + kBlock - 1) / kBlock;    // ... per thread
  __shared__ __align__(16) float Vs[2][kLgGRows][VS];
  __shared__ __align__(16) float Ws[2][16][WS];
  const int t = threadIdx.x, lane = t & (kWave - 1);
  const int w = __builtin_amdgcn_readfirstlane(t / kWave);
  const int i = lane & 15, g = lane >> 4;
  const int j = blockIdx.y, b0 = blockIdx.x * kLgGRows;
  const int ty = (j == a.win) ? 2 : (j == a.c ? 1 : 0);
  const int jj = (j == a.win) ? a.c : j;
  const int nsteps = a.H / 16;
  // this thread's share of a step: one float4 of vectors (window t/4, units
  // 4*(t%4)), WPT float4 of W1 rows (row x / (D/4), float4 column x % (D/4))
  const int vw = t / 4, vh = 4 * (t % 4);
  const bool vok = b0 + vw < a.B;
  const float* vsrc = a.V + (size_t)(vok ? b0 + vw : 0) * 3 * a.H + (size_t)ty * a.H + vh;
  auto load = [&](int st, f4& Vv, f4 (&Wv)[WPT]) {
    const int hc = st * 16;
    Vv = vok ? ld4(vsrc + hc) : kZero4;
#pragma unroll
    for (int u = 0; u < WPT; ++u) {
      const int x = t + u * kBlock;
      if (x < WF) {
        const int r = x / (D / 4), c4 = x % (D / 4);
        Wv[u] = ld4(a.W1 + (size_t)(hc + r) * a.K + (size_t)jj * D + 4 * c4);
      }
    }
  };
  auto store = [&](int buf, const f4& Vv, const f4 (&Wv)[WPT]) {
    st4(&Vs[buf][vw][vh], Vv);
#pragma unroll
    for (int u = 0; u < WPT; ++u) {
      const int x = t + u * kBlock;
      if (x < WF) st4(&Ws[buf][x / (D / 4)][4 * (x % (D / 4))], Wv[u]);
    }
  };
  f4 acc[DQ];
#pragma unroll
  for (int ct = 0; ct < DQ; ++ct) acc[ct] = kZero4;
  auto compute = [&](int buf) {
    const f4 av = ld4(&Vs[buf][16 * w + i][4 * g]);
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
      for (int ct = 0; ct < DQ; ++ct) acc[ct] = lg_mfma(av[q], Ws[buf][4 * g + q][16 * ct + i], acc[ct]);
  };
  f4 VA, WA[WPT], VB, WB[WPT];
  load(0, VA, WA);
  if (nsteps > 1) load(1, VB, WB);
  for (int st = 0; st < nsteps; st += 2) {
    store(0, VA, WA);
    if (st + 2 < nsteps) load(st + 2, VA, WA);
    __syncthreads();
    compute(0);
    if (st + 1 >= nsteps) break;
    store(1, VB, WB);
    if (st + 3 < nsteps) load(st + 3, VB, WB);
    __syncthreads();
    compute(1);
  }
  // lane (i, g), component q: window b0 + 16w + 4g + q, column 16ct + i
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int b = b0 + 16 * w + 4 * g + q;
    if (b < a.B) {
      float* gr = a.G + ((size_t)b * (a.win + 1) + j) * a.d + i;
#pragma unroll
      for (int ct = 0; ct < DQ; ++ct) gr[16 * ct] = acc[ct][q];
    }
  }
}

}  // namespace pg
