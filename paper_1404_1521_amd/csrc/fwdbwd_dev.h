// Fused gather + forward + hinge + backward of 16-window tiles (16x16x4 f32
// MFMA), ending in the per-entry embedding gradient rows G.
//
// Per tile of 16 windows (rows r), with V = dz + dz~, dz or dz~ (per
// window, H values each):
//   forward   Z = X W1^T split over the K-chunks of the four waves; the
//             corrupted copy only differs in block c, so z~ = z - zctr + zcor
//             comes from one extra 16 x d contraction (§1 model, x~);
//   epilogue  tanh, both scores, hinge mask, dz, dz~ and their sum;
//   G         G[e][:] = W1_j^T V for entry e = b(win+1) + j: context
//             positions take dz + dz~, the true centre dz, the corrupt entry
//             (j = win) dz~ through block c -- one 16 x 16 output tile per
//             (entry position, 16 columns), reduction over the hidden units;
//   dW1       dW1 += V^T X per K-chunk (block c: dz^T e_c + dz~^T e~), held
//             in registers across the workgroup's tiles, written once as
//             this workgroup's partial, with db1, dw2 and the loss.
// W1 is staged once per workgroup in LDS (row stride K + 4 floats) and read
// from there as the B operand of the forward and of G.
#pragma once
#include "common.h"
#include "launch.h"

namespace pg {

__device__ __forceinline__ f4 mfma16(float a, float b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

constexpr int kGTiles = 2;  // G output tiles accumulated together per wave

template <int NT, int CPW>
__device__ void fwdbwd_wg(const FwdArgs& a, int wg, float* lds) {
  constexpr int HP = NT * 16;
  const int t = threadIdx.x, lane = t & (kWave - 1), w = t / kWave;
  const int n16 = lane & 15, g = lane >> 4;
  const int W1p = a.win + 1;
  const int dq = a.d / 16;
  const int nchunk = a.K / 16;
  const int S = a.K + 4;
  float* w1s = lds;
  f4* zp = reinterpret_cast<f4*>(w1s + (size_t)HP * S);
  float* vt = reinterpret_cast<float*>(zp + kWavesPerBlock * 3 * NT * kWave);
  int32_t* ids = reinterpret_cast<int32_t*>(vt + 3 * kTileRows * (HP + 1));

  {  // W1 into LDS, rows >= H zero; loads batched before the stores
    constexpr int U = 8;
    const int k4 = a.K / 4, n4 = HP * k4;
    for (int i0 = 0; i0 < n4; i0 += kBlock * U) {
      f4 v[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int i = i0 + u * kBlock + t;
        const int n = i / k4;
        v[u] = (i < n4 && n < a.H) ? ld4(a.W1 + (size_t)n * a.K + 4 * (i - n * k4)) : kZero4;
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
    __syncthreads();  // W1 staged; LDS of the previous tile no longer read
    for (int i = t; i < kTileRows * W1p; i += kBlock) {
      const int r = i / W1p, j = i - r * W1p;
      const int b = row0 + r;
      int32_t id = 0;
      if (b < a.B) id = (j < a.win) ? a.windows[(size_t)b * a.win + j] : a.corrupt[b];
      const bool bad = (uint32_t)id >= (uint32_t)a.V;
      if (bad) atomicOr(a.flag, kFlagBadId);
      ids[r * (kMaxWin + 1) + j] = bad ? 0 : id;
    }
    __syncthreads();

    // ---- the forward's embedding values for this wave, in one batch.
    // Forward A operand: lane (r=n16, g) holds X[r][16kc + 4g .. +3].
    const int32_t* rid = ids + n16 * (kMaxWin + 1);
    f4 xa[CPW], xt[CPW];
#pragma unroll
    for (int ci = 0; ci < CPW; ++ci) {
      const int kc = w + kWavesPerBlock * ci;
      const bool ok = kc < nchunk;
      const int j = ok ? kc / dq : 0;
      const bool ctr = ok && j == a.c;
      const int q16 = (kc - j * dq) * 16;
      xa[ci] = ok ? ld4(a.E + (size_t)rid[j] * a.d + q16 + 4 * g) : kZero4;
      xt[ci] = ctr ? ld4(a.E + (size_t)rid[a.win] * a.d + q16 + 4 * g) : kZero4;
    }

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
        if (kc / dq != a.c) {
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
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      zp[((w * 3 + 0) * NT + nt) * kWave + lane] = zc[nt];
      zp[((w * 3 + 1) * NT + nt) * kWave + lane] = zctr[nt];
      zp[((w * 3 + 2) * NT + nt) * kWave + lane] = zcor[nt];
    }
    __syncthreads();
    // ---- the same rows again as dW1 B operands, in flight during the
    // epilogue: lane (col=n16, g) holds X[4g+i][16kc + n16]
    float xb[CPW][4], xr[CPW][4];
#pragma unroll
    for (int ci = 0; ci < CPW; ++ci) {
      const int kc = w + kWavesPerBlock * ci;
      const bool ok = kc < nchunk;
      const int j = ok ? kc / dq : 0;
      const bool ctr = ok && j == a.c;
      const int q16 = (kc - j * dq) * 16;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int32_t* ri = ids + (4 * g + i) * (kMaxWin + 1);
        xb[ci][i] = ok ? a.E[(size_t)ri[j] * a.d + q16 + n16] : 0.f;
        xr[ci][i] = ctr ? a.E[(size_t)ri[a.win] * a.d + q16 + n16] : 0.f;
      }
    }
    // every wave sums the four split-K partials in the same order
    f4 Zc[NT], Zctr[NT], Zcor[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      Zc[nt] = zp[((0 * 3 + 0) * NT + nt) * kWave + lane];
      Zctr[nt] = zp[((0 * 3 + 1) * NT + nt) * kWave + lane];
      Zcor[nt] = zp[((0 * 3 + 2) * NT + nt) * kWave + lane];
#pragma unroll
      for (int v = 1; v < kWavesPerBlock; ++v) {
        Zc[nt] += zp[((v * 3 + 0) * NT + nt) * kWave + lane];
        Zctr[nt] += zp[((v * 3 + 1) * NT + nt) * kWave + lane];
        Zcor[nt] += zp[((v * 3 + 2) * NT + nt) * kWave + lane];
      }
    }

    // ---- epilogue: lane (n16, g) owns rows 4g+i, hidden unit nt*16+n16
    float h[NT][4], ht[NT][4], hmh[NT][4], ps[4], pst[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) ps[i] = pst[i] = 0.f;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float z = b1v[nt] + (Zc[nt][i] + Zctr[nt][i]);
        const float zt = b1v[nt] + (Zc[nt][i] + Zcor[nt][i]);
        h[nt][i] = tanhf(z);
        ht[nt][i] = tanhf(zt);
        // h - h~ = tanh(z - z~) (1 - h h~), with z - z~ = zctr - zcor taken
        // without cancellation against the common part
        hmh[nt][i] = tanhf(Zctr[nt][i] - Zcor[nt][i]) * (1.f - h[nt][i] * ht[nt][i]);
        ps[i] += w2v[nt] * h[nt][i];
        pst[i] += w2v[nt] * ht[nt][i];
      }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int o = 1; o < 16; o <<= 1) {
        ps[i] += __shfl_xor(ps[i], o);
        pst[i] += __shfl_xor(pst[i], o);
      }
    float gst[4], mg[4];
    bool on[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = row0 + 4 * g + i;
      const float s = b2v + ps[i];
      const float st = b2v + pst[i];
      mg[i] = 1.f - s + st;
      on[i] = row < a.B && mg[i] > 0.f;  // hinge active (derivative 0 at margin 0)
      gst[i] = on[i] ? a.invB : 0.f;     // d loss/d s~ = m/B, d loss/d s = -m/B
    }
    // dz = -g w2 (1-h^2), dz~ = g w2 (1-h~^2), dz + dz~ = g w2 (h-h~)(h+h~)
    float dz[NT][4], dzt[NT][4], dsum[NT][4];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float gw = gst[i] * w2v[nt];
        dz[nt][i] = -gw * (1.f - h[nt][i] * h[nt][i]);
        dzt[nt][i] = gw * (1.f - ht[nt][i] * ht[nt][i]);
        dsum[nt][i] = gw * hmh[nt][i] * (h[nt][i] + ht[nt][i]);
      }
    // V transposed through LDS for the G contraction: vt[type][r][n],
    // type 0 dz+dz~ (context), 1 dz (true centre), 2 dz~ (corrupt)
    if (w < 3) {
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float v = (w == 0) ? dsum[nt][i] : (w == 1 ? dz[nt][i] : dzt[nt][i]);
          vt[(w * kTileRows + 4 * g + i) * (HP + 1) + nt * 16 + n16] = v;
        }
    }
    if (w == 0) {
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          db1a[nt] += dsum[nt][i];
          dw2a[nt] -= gst[i] * hmh[nt][i];  // -(m/B) h + (m/B) h~
        }
      if (n16 == 0) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          lossa += on[i] ? mg[i] : 0.f;
          db2a += -gst[i] + gst[i];  // both scores share b2: its gradient is 0
        }
      }
    }

    // ---- dW1 += dsum^T X (+ centre block: dz^T e_c + dz~^T e~), this wave's chunks
#pragma unroll
    for (int ci = 0; ci < CPW; ++ci) {
      const int kc = w + kWavesPerBlock * ci;
      if (kc < nchunk) {
        if (kc / dq != a.c) {
#pragma unroll
          for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt)
              accW[ci][nt] = mfma16(dsum[nt][i], xb[ci][i], accW[ci][nt]);
        } else {
#pragma unroll
          for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) {
              accW[ci][nt] = mfma16(dz[nt][i], xb[ci][i], accW[ci][nt]);
              accW[ci][nt] = mfma16(dzt[nt][i], xr[ci][i], accW[ci][nt]);
            }
        }
      }
    }
    __syncthreads();  // vt written

    // ---- G: output tiles (entry position j, 16 columns cb) go round-robin
    // to the waves, kGTiles accumulated together.  A operand: lane (r=n16,
    // g) holds V[r][4q+g]; B operand: lane (col=n16, g) holds W1[4q+g][col].
    for (int t0 = w; t0 < ngt; t0 += kWavesPerBlock * kGTiles) {
      int off[kGTiles], typ[kGTiles];
      f4 acc[kGTiles];
#pragma unroll
      for (int u = 0; u < kGTiles; ++u) {
        const int ot = min(t0 + u * kWavesPerBlock, ngt - 1);
        const int j = ot / dq, cb = ot - j * dq;
        typ[u] = (j == a.win) ? 2 : (j == a.c ? 1 : 0);
        off[u] = ((j == a.win) ? a.c : j) * a.d + cb * 16 + n16;
        acc[u] = kZero4;
      }
#pragma unroll
      for (int q = 0; q < HP / 4; ++q) {
#pragma unroll
        for (int u = 0; u < kGTiles; ++u) {
          const float av = vt[(typ[u] * kTileRows + n16) * (HP + 1) + 4 * q + g];
          const float bv = w1s[(size_t)(4 * q + g) * S + off[u]];
          acc[u] = mfma16(av, bv, acc[u]);
        }
      }
#pragma unroll
      for (int u = 0; u < kGTiles; ++u) {
        const int ot = t0 + u * kWavesPerBlock;
        if (ot < ngt) {
          const int j = ot / dq, cb = ot - j * dq;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int row = row0 + 4 * g + i;
            if (row < a.B) a.G[((size_t)row * W1p + j) * a.d + cb * 16 + n16] = acc[u][i];
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
          P[(size_t)(nt * 16 + 4 * g + i) * a.K + kc * 16 + n16] = accW[ci][nt][i];
    }
  }
  if (w == 0) {
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      float x = db1a[nt], y = dw2a[nt];
      x += __shfl_xor(x, 16);
      x += __shfl_xor(x, 32);
      y += __shfl_xor(y, 16);
      y += __shfl_xor(y, 32);
      if (g == 0) {
        P[(size_t)a.Hp * a.K + nt * 16 + n16] = x;
        P[(size_t)a.Hp * a.K + a.Hp + nt * 16 + n16] = y;
      }
    }
    for (int o = 1; o < kWave; o <<= 1) {
      lossa += __shfl_xor(lossa, o);
      db2a += __shfl_xor(db2a, o);
    }
    if (lane == 0) {
      P[(size_t)a.Hp * a.K + 2 * a.Hp] = lossa;
      P[(size_t)a.Hp * a.K + 2 * a.Hp + 1] = db2a;
    }
  }
}

}  // namespace pg
