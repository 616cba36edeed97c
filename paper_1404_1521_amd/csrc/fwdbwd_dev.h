// Fused gather + forward + hinge + backward of 16-window tiles (16x16x4 f32
// MFMA), ending in the per-entry embedding gradient rows G.
//
// Per tile of 16 windows (rows r), with V = dz + dz~, dz or dz~ (per
// window, H values each):
//   forward   Z = X W1^T split over the K-chunks of the four waves; the
//             corrupted copy only differs in block c, so z~ = z - zctr + zcor
//             comes from one extra 16 x d contraction (§1 model, x~);
//   epilogue  tanh, both scores, hinge mask, dz, dz~ and their sum; wave w
//             takes the rows 4g + w of lane group g (a quarter of the tile)
//             and writes its V values to LDS;
//   dW1       dW1 += V^T X per K-chunk (block c: dz^T e_c + dz~^T e~), held
//             in registers across the workgroup's tiles, written once as
//             this workgroup's partial;
//   G         G[e][:] = W1_j^T V for entry e = b(win+1) + j: context
//             positions take dz + dz~, the true centre dz, the corrupt entry
//             (j = win) dz~ through block c -- one 16 x 16 output tile per
//             (entry position, 16 columns), reduction over the hidden units.
// W1 is staged once per workgroup in LDS (row stride K + 4 floats) and read
// from there as the B operand of the forward and of G.  The row ids of a
// tile sit in one of two LDS tables: tile k+1's ids are loaded (and checked)
// at the start of tile k and stored before its second barrier, so a tile
// needs two workgroup barriers and no exposed id round trip.
#pragma once
#include "common.h"
#include "launch.h"

namespace pg {

__device__ __forceinline__ f4 mfma16(float a, float b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// G output tiles accumulated together per wave: 6 covers the (win+1) * d/16
// = 24 tiles of window 5, d 64 in one pass of the four waves.
constexpr int kGTiles = 6;

// D_ and WIN_ fix the embedding width and the window at compile time for
// the common shapes (0: taken from the arguments).
template <int NT, int CPW, int D_, int WIN_>
__device__ void fwdbwd_wg(const FwdArgs& a, int wg, float* lds) {
  constexpr int HP = NT * 16;
  const int t = threadIdx.x, lane = t & (kWave - 1);
  const int w = __builtin_amdgcn_readfirstlane(t / kWave);  // wave-uniform: scalar branches
  const int n16 = lane & 15, g = lane >> 4;
  const int d = D_ ? D_ : a.d;
  const int win = WIN_ ? WIN_ : a.win;
  const int K = d * win;
  const int cc = win / 2;
  const int W1p = win + 1;
  const int dq = d / 16;
  const int nchunk = K / 16;
  const int S = K + 4;
  float* w1s = lds;                                        // [HP][K+4]
  float* zp = w1s + (size_t)HP * S;                        // [4][3][NT][4][64]
  float* vt = zp + kWavesPerBlock * 3 * NT * kWave * 4;    // [3][16][HP+1]
  float* red = vt + 3 * kTileRows * (HP + 1);              // [4][2*HP+2]
  int32_t* idt = reinterpret_cast<int32_t*>(red + kWavesPerBlock * (2 * HP + 2));  // [2][16][32]

  // ids of a tile, slots t and t + 256 of [16][win+1] (j == win: the corrupt
  // id); rows >= B read as row 0; an id outside [0, V) raises the flag and
  // reads as row 0
  auto load_ids = [&](int tile, int32_t (&v)[2]) {
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      const int i = t + k * kBlock;
      const int r = i / W1p, j = i - r * W1p;
      const int b = tile * kTileRows + r;
      v[k] = 0;
      if (i < kTileRows * W1p && b < a.B)
        v[k] = (j < win) ? a.windows[(size_t)b * win + j] : a.corrupt[b];
    }
    bool bad = false;
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      const bool bk = (uint32_t)v[k] >= (uint32_t)a.V;
      bad |= bk;
      v[k] = bk ? 0 : v[k];
    }
    if (bad) atomicOr(a.flag, kFlagBadId);
  };
  auto store_ids = [&](int buf, const int32_t (&v)[2]) {
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      const int i = t + k * kBlock;
      const int r = i / W1p, j = i - r * W1p;
      if (i < kTileRows * W1p) idt[(buf * kTileRows + r) * (kMaxWin + 1) + j] = v[k];
    }
  };
  // Forward A operand: lane (r=n16, g) holds X[r][16kc + 4g .. +3] (xa), and
  // in the centre block the corrupt row instead (xt); ids first, then loads.
  auto load_fwd = [&](int buf, f4 (&xa)[CPW], f4 (&xt)[CPW]) {
    const int32_t* rid = idt + (buf * kTileRows + n16) * (kMaxWin + 1);
    int32_t idr[CPW];
    const int32_t idc = rid[win];
#pragma unroll
    for (int ci = 0; ci < CPW; ++ci) {
      const int kc = w + kWavesPerBlock * ci;
      idr[ci] = rid[kc < nchunk ? kc / dq : 0];
    }
#pragma unroll
    for (int ci = 0; ci < CPW; ++ci) {
      const int kc = w + kWavesPerBlock * ci;
      const bool ok = kc < nchunk;
      const int j = ok ? kc / dq : 0;
      const bool ctr = ok && j == cc;
      const int q16 = (kc - j * dq) * 16;
      xa[ci] = ok ? ld4(a.E + (size_t)idr[ci] * d + q16 + 4 * g) : kZero4;
      xt[ci] = ctr ? ld4(a.E + (size_t)idc * d + q16 + 4 * g) : kZero4;
    }
  };

  int32_t idv[2];
  load_ids(wg * a.tiles_per_wg, idv);  // in flight with the W1 loads
  {  // W1 into LDS, rows >= H zero; loads batched before the stores
    constexpr int U = 16;  // one batch up to Hp*K = 16384 floats
    const int k4 = K / 4, n4 = HP * k4;
    for (int i0 = 0; i0 < n4; i0 += kBlock * U) {
      f4 v[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int i = i0 + u * kBlock + t;
        const int n = i / k4;
        v[u] = (i < n4 && n < a.H) ? ld4(a.W1 + (size_t)n * K + 4 * (i - n * k4)) : kZero4;
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int i = i0 + u * kBlock + t;
        const int n = i / k4;
        if (i < n4) st4(w1s + (size_t)n * S + 4 * (i - n * k4), v[u]);
      }
    }
  }
  float b1v[NT], w2v[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const int n = nt * 16 + n16;
    b1v[nt] = n < a.H ? a.b1[n] : 0.f;
    w2v[nt] = n < a.H ? a.w2[n] : 0.f;
  }
  const float b2v = a.b2[0];
  store_ids(0, idv);
  __syncthreads();                            // W1 and the first tile's ids staged

  f4 accW[CPW][NT];
#pragma unroll
  for (int ci = 0; ci < CPW; ++ci)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) accW[ci][nt] = kZero4;
  float db1a[NT], dw2a[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) db1a[nt] = dw2a[nt] = 0.f;
  float lossa = 0.f, db2a = 0.f;
  const int ngt = W1p * dq;  // G output tiles per 16-window tile

  for (int tt = 0; tt < a.tiles_per_wg; ++tt) {
    const int tile = wg * a.tiles_per_wg + tt;
    if (tile >= a.ntiles) break;
    const int row0 = tile * kTileRows;
    const int buf = tt & 1;
    // (LDS hazards: zp of the previous tile was last read before its vt
    // barrier, vt before this tile's zp barrier, so no barrier is needed here)
    f4 xa[CPW], xt[CPW];
    load_fwd(buf, xa, xt);
    const bool more = tt + 1 < a.tiles_per_wg && tile + 1 < a.ntiles;
    if (more) load_ids(tile + 1, idv);  // stored before this tile's vt barrier

    // ---- forward, split-K over the waves: common blocks, true centre and
    // corrupt centre accumulate separately (z = b1 + zc + zctr, z~ = b1 + zc + zcor)
    f4 zc[NT], zctr[NT], zcor[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) zc[nt] = zctr[nt] = zcor[nt] = kZero4;
#pragma unroll
    for (int ci = 0; ci < CPW; ++ci) {
      const int kc = w + kWavesPerBlock * ci;
      if (kc < nchunk) {
        // B operand: lane (n16, g) holds W1[nt*16 + n16][16kc + 4g .. +3]
        f4 wb[NT];
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
          wb[nt] = ld4(w1s + (size_t)(nt * 16 + n16) * S + kc * 16 + 4 * g);
        if (kc / dq != cc) {
#pragma unroll
          for (int q = 0; q < 4; ++q)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) zc[nt] = mfma16(xa[ci][q], wb[nt][q], zc[nt]);
        } else {
#pragma unroll
          for (int q = 0; q < 4; ++q)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) {
              zctr[nt] = mfma16(xa[ci][q], wb[nt][q], zctr[nt]);
              zcor[nt] = mfma16(xt[ci][q], wb[nt][q], zcor[nt]);
            }
        }
      }
    }
    // split-K partials, component-major so that a wave reading one
    // component of every lane touches consecutive words
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        zp[(((w * 3 + 0) * NT + nt) * 4 + i) * kWave + lane] = zc[nt][i];
        zp[(((w * 3 + 1) * NT + nt) * 4 + i) * kWave + lane] = zctr[nt][i];
        zp[(((w * 3 + 2) * NT + nt) * 4 + i) * kWave + lane] = zcor[nt][i];
      }

    // ---- dW1 B operands (lane (col=n16, g) holds X[4g+i][16kc + n16]),
    // in flight during the epilogue
    float xb[CPW][4], xr[CPW][4];
    {
      int32_t idb[CPW][4], idq[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int32_t* ri = idt + (buf * kTileRows + 4 * g + i) * (kMaxWin + 1);
        idq[i] = ri[win];
#pragma unroll
        for (int ci = 0; ci < CPW; ++ci) {
          const int kc = w + kWavesPerBlock * ci;
          idb[ci][i] = ri[kc < nchunk ? kc / dq : 0];
        }
      }
#pragma unroll
      for (int ci = 0; ci < CPW; ++ci) {
        const int kc = w + kWavesPerBlock * ci;
        const bool ok = kc < nchunk;
        const int j = ok ? kc / dq : 0;
        const bool ctr = ok && j == cc;
        const int q16 = (kc - j * dq) * 16;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          xb[ci][i] = ok ? a.E[(size_t)idb[ci][i] * d + q16 + n16] : 0.f;
          xr[ci][i] = ctr ? a.E[(size_t)idq[i] * d + q16 + n16] : 0.f;
        }
      }
    }
    __syncthreads();  // zp written

    // ---- epilogue of rows 4g + w: lane (n16, g) takes hidden units nt*16+n16;
    // the four split-K partials are added in wave order
    {
      const int r = 4 * g + w;
      const int row = row0 + r;
      float h[NT], ht[NT], hmh[NT];
      float ps = 0.f, pst = 0.f;
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        float Zc = 0.f, Zctr = 0.f, Zcor = 0.f;
#pragma unroll
        for (int v = 0; v < kWavesPerBlock; ++v) {
          Zc += zp[(((v * 3 + 0) * NT + nt) * 4 + w) * kWave + lane];
          Zctr += zp[(((v * 3 + 1) * NT + nt) * 4 + w) * kWave + lane];
          Zcor += zp[(((v * 3 + 2) * NT + nt) * 4 + w) * kWave + lane];
        }
        const float z = b1v[nt] + (Zc + Zctr);
        const float zt = b1v[nt] + (Zc + Zcor);
        h[nt] = tanh_fast(z);
        ht[nt] = tanh_fast(zt);
        // h - h~ = tanh(z - z~) (1 - h h~), with z - z~ = zctr - zcor taken
        // without cancellation against the common part
        hmh[nt] = tanh_fast(Zctr - Zcor) * (1.f - h[nt] * ht[nt]);
        ps += w2v[nt] * h[nt];
        pst += w2v[nt] * ht[nt];
      }
#pragma unroll
      for (int o = 1; o < 16; o <<= 1) {
        ps += __shfl_xor(ps, o);
        pst += __shfl_xor(pst, o);
      }
      const float mg = 1.f - (b2v + ps) + (b2v + pst);
      const bool on = row < a.B && mg > 0.f;  // hinge active (derivative 0 at margin 0)
      const float gst = on ? a.invB : 0.f;    // d loss/d s~ = m/B, d loss/d s = -m/B
      // dz = -g w2 (1-h^2), dz~ = g w2 (1-h~^2), dz + dz~ = g w2 (h-h~)(h+h~)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const float gw = gst * w2v[nt];
        const float dz = -gw * (1.f - h[nt] * h[nt]);
        const float dzt = gw * (1.f - ht[nt] * ht[nt]);
        const float dsum = gw * hmh[nt] * (h[nt] + ht[nt]);
        // V for the G contraction and dW1: vt[type][r][n], type 0 dz+dz~
        // (context), 1 dz (true centre), 2 dz~ (corrupt)
        vt[(0 * kTileRows + r) * (HP + 1) + nt * 16 + n16] = dsum;
        vt[(1 * kTileRows + r) * (HP + 1) + nt * 16 + n16] = dz;
        vt[(2 * kTileRows + r) * (HP + 1) + nt * 16 + n16] = dzt;
        db1a[nt] += dsum;
        dw2a[nt] -= gst * hmh[nt];  // -(m/B) h + (m/B) h~
      }
      if (n16 == 0) {
        lossa += on ? mg : 0.f;
        db2a += -gst + gst;  // both scores share b2: its gradient is 0
      }
    }
    // next tile's ids: the other table was last read before this tile's zp barrier
    if (more) store_ids(buf ^ 1, idv);
    __syncthreads();  // vt and the next tile's ids written

    // ---- dW1 += dsum^T X (+ centre block: dz^T e_c + dz~^T e~), this wave's
    // chunks.  A operand: lane (n16, g) holds V[4g+i][nt*16 + n16].
    {
      float vc[3][NT][4];
#pragma unroll
      for (int ty = 0; ty < 3; ++ty)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
#pragma unroll
          for (int i = 0; i < 4; ++i)
            vc[ty][nt][i] = vt[(ty * kTileRows + 4 * g + i) * (HP + 1) + nt * 16 + n16];
#pragma unroll
      for (int ci = 0; ci < CPW; ++ci) {
        const int kc = w + kWavesPerBlock * ci;
        if (kc < nchunk) {
          if (kc / dq != cc) {
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
              for (int nt = 0; nt < NT; ++nt)
                accW[ci][nt] = mfma16(vc[0][nt][i], xb[ci][i], accW[ci][nt]);
          } else {
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
              for (int nt = 0; nt < NT; ++nt) {
                accW[ci][nt] = mfma16(vc[1][nt][i], xb[ci][i], accW[ci][nt]);
                accW[ci][nt] = mfma16(vc[2][nt][i], xr[ci][i], accW[ci][nt]);
              }
          }
        }
      }
    }

    // ---- G: output tiles (entry position j, 16 columns cb) go round-robin
    // to the waves, kGTiles accumulated together.  A operand: lane (r=n16,
    // g) holds V[r][4q+g], read once per tile for the three vector types;
    // B operand: lane (col=n16, g) holds W1[4q+g][col].
    float av[3][HP / 4];
#pragma unroll
    for (int ty = 0; ty < 3; ++ty)
#pragma unroll
      for (int q = 0; q < HP / 4; ++q) av[ty][q] = vt[(ty * kTileRows + n16) * (HP + 1) + 4 * q + g];
    for (int t0 = w; t0 < ngt; t0 += kWavesPerBlock * kGTiles) {
      int off[kGTiles], typ[kGTiles];
      f4 acc[kGTiles];
#pragma unroll
      for (int u = 0; u < kGTiles; ++u) {
        const int ot = min(t0 + u * kWavesPerBlock, ngt - 1);
        const int j = ot / dq, cb = ot - j * dq;
        typ[u] = (j == win) ? 2 : (j == cc ? 1 : 0);
        off[u] = ((j == win) ? cc : j) * d + cb * 16 + n16;
        acc[u] = kZero4;
      }
      const int nu = min(kGTiles, (ngt - t0 + kWavesPerBlock - 1) / kWavesPerBlock);
      // A operands of each output tile, chosen by its vector type with exact
      // 0/1 weights (uniform), so no branch sits between the MFMAs
      float aa[kGTiles][HP / 4], bv[kGTiles][HP / 4];
#pragma unroll
      for (int u = 0; u < kGTiles; ++u) {
        const float c0 = typ[u] == 0 ? 1.f : 0.f, c1 = typ[u] == 1 ? 1.f : 0.f;
        const float c2 = typ[u] == 2 ? 1.f : 0.f;
#pragma unroll
        for (int q = 0; q < HP / 4; ++q) {
          aa[u][q] = av[0][q] * c0 + av[1][q] * c1 + av[2][q] * c2;
          bv[u][q] = w1s[(size_t)(4 * q + g) * S + off[u]];
        }
      }
      if (nu == kGTiles) {
#pragma unroll
        for (int q = 0; q < HP / 4; ++q)
#pragma unroll
          for (int u = 0; u < kGTiles; ++u) acc[u] = mfma16(aa[u][q], bv[u][q], acc[u]);
      } else {
#pragma unroll
        for (int q = 0; q < HP / 4; ++q)
#pragma unroll
          for (int u = 0; u < kGTiles; ++u)
            if (u < nu) acc[u] = mfma16(aa[u][q], bv[u][q], acc[u]);
      }
#pragma unroll
      for (int u = 0; u < kGTiles; ++u) {
        const int ot = t0 + u * kWavesPerBlock;
        if (ot < ngt) {
          const int j = ot / dq, cb = ot - j * dq;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int row = row0 + 4 * g + i;
            if (row < a.B) a.G[((size_t)row * W1p + j) * d + cb * 16 + n16] = acc[u][i];
          }
        }
      }
    }
  }

  // ---- this workgroup's partial of the dense gradients
  float* P = a.part + (size_t)wg * a.part_stride;
#pragma unroll
  for (int ci = 0; ci < CPW; ++ci) {
    const int kc = w + kWavesPerBlock * ci;
    if (kc < nchunk) {
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          P[(size_t)(nt * 16 + 4 * g + i) * K + kc * 16 + n16] = accW[ci][nt][i];
    }
  }
  // db1, dw2, loss, db2: per-wave sums (fixed butterflies), then the four
  // waves added in order by wave 0
  float* rw = red + w * (2 * HP + 2);
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    float x = db1a[nt], y = dw2a[nt];
    x += __shfl_xor(x, 16);
    x += __shfl_xor(x, 32);
    y += __shfl_xor(y, 16);
    y += __shfl_xor(y, 32);
    if (g == 0) {
      rw[nt * 16 + n16] = x;
      rw[HP + nt * 16 + n16] = y;
    }
  }
  for (int o = 1; o < kWave; o <<= 1) {
    lossa += __shfl_xor(lossa, o);
    db2a += __shfl_xor(db2a, o);
  }
  if (lane == 0) {
    rw[2 * HP] = lossa;
    rw[2 * HP + 1] = db2a;
  }
  __syncthreads();
  if (w == 0) {
    for (int e = lane; e < 2 * HP + 2; e += kWave) {
      float s = red[e];
#pragma unroll
      for (int v = 1; v < kWavesPerBlock; ++v) s += red[v * (2 * HP + 2) + e];
      // slot layout: dW1 [Hp][K], db1 [Hp], dw2 [Hp], loss, db2
      P[(size_t)a.Hp * K + e] = s;
    }
  }
}

}  // namespace pg
