// Fused gather + forward + hinge + backward of 16-window tiles (16x16x4 f32 MFMA).
#pragma once
#include "common.h"
#include "launch.h"
#include "seg_dev.h"
#include "sort_dev.h"

namespace pg {

__device__ __forceinline__ f4 mfma16(float a, float b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

template <int NT, int CPW>
__device__ void fwdbwd_wg(const FwdArgs& a, int wg, uint32_t* lds) {
  const int t = threadIdx.x, lane = t & (kWave - 1), w = t / kWave;
  const int n16 = lane & 15, g = lane >> 4;
  const int W1p = a.win + 1;
  const int dq = a.d / 16;
  const int nchunk = a.K / 16;
  int32_t* ids = reinterpret_cast<int32_t*>(lds);                  // [16][win+1]
  f4* zp = reinterpret_cast<f4*>(lds + kTileRows * (kMaxWin + 1));  // [4][3][NT][64]

  // W1 B-operands of this wave's k-chunks, kept in registers for all tiles:
  // lane (n16, g) holds W1[nt*16 + n16][16*kc + 4g .. +3].
  f4 wreg[CPW][NT];
#pragma unroll
  for (int ci = 0; ci < CPW; ++ci) {
    const int kc = w + kWavesPerBlock * ci;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const int n = nt * 16 + n16;
      wreg[ci][nt] = (kc < nchunk && n < a.H) ? ld4(a.W1 + (size_t)n * a.K + kc * 16 + 4 * g)
                                                : kZero4;
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

  if (wg == 0) {  // copy of W1 taken before any update (rows >= H are zero)
    if (t == 0) *a.long_count = 0u;
    constexpr int U = 8;
    const int n4 = a.Hp * a.K / 4, h4 = a.H * a.K / 4;
    for (int i0 = 0; i0 < n4; i0 += kBlock * U) {
      f4 v[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int i = i0 + u * kBlock + t;
        v[u] = i < h4 ? ld4(a.W1 + 4 * i) : kZero4;
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int i = i0 + u * kBlock + t;
        if (i < n4) st4(a.w1snap + 4 * i, v[u]);
      }
    }
  }

  f4 accW[CPW][NT];
#pragma unroll
  for (int ci = 0; ci < CPW; ++ci)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) accW[ci][nt] = kZero4;
  float db1a[NT], dw2a[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) db1a[nt] = dw2a[nt] = 0.f;
  float lossa = 0.f, db2a = 0.f;

  for (int tt = 0; tt < a.tiles_per_wg; ++tt) {
    const int tile = wg * a.tiles_per_wg + tt;
    if (tile >= a.ntiles) break;
    const int row0 = tile * kTileRows;
    __syncthreads();  // LDS of the previous tile is no longer read
    for (int i = t; i < kTileRows * W1p; i += kBlock) {
      const int r = i / W1p, j = i - r * W1p;
      const int b = row0 + r;
      int32_t id = 0;
      if (b < a.B) id = (j < a.win) ? a.windows[(size_t)b * a.win + j] : a.corrupt[b];
      const bool bad = (uint32_t)id >= (uint32_t)a.V;
      if (bad) atomicOr(a.flag, kFlagBadId);
      ids[i] = bad ? 0 : id;
    }
    __syncthreads();

    // ---- every embedding value this wave needs for the tile, in one batch.
    // Forward A operand: lane (r=n16, g) holds X[r][16kc + 4g .. +3].
    // dW1 B operand:     lane (col=n16, g) holds X[4g+i][16kc + n16].
    const int32_t* rid = ids + n16 * W1p;
    f4 xa[CPW], xt[CPW];
    float xb[CPW][4], xr[CPW][4];
#pragma unroll
    for (int ci = 0; ci < CPW; ++ci) {
      const int kc = w + kWavesPerBlock * ci;
      const bool ok = kc < nchunk;
      const int j = ok ? kc / dq : 0;
      const bool ctr = ok && j == a.c;
      const int q16 = (kc - j * dq) * 16;
      xa[ci] = ok ? ld4(a.E + (size_t)rid[j] * a.d + q16 + 4 * g) : kZero4;
      xt[ci] = ctr ? ld4(a.E + (size_t)rid[a.win] * a.d + q16 + 4 * g) : kZero4;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int32_t* ri = ids + (4 * g + i) * W1p;
        xb[ci][i] = ok ? a.E[(size_t)ri[j] * a.d + q16 + n16] : 0.f;
        xr[ci][i] = ctr ? a.E[(size_t)ri[a.win] * a.d + q16 + n16] : 0.f;
      }
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
        if (kc / dq != a.c) {
#pragma unroll
          for (int q = 0; q < 4; ++q)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) zc[nt] = mfma16(xa[ci][q], wreg[ci][nt][q], zc[nt]);
        } else {
#pragma unroll
          for (int q = 0; q < 4; ++q)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) {
              zctr[nt] = mfma16(xa[ci][q], wreg[ci][nt][q], zctr[nt]);
              zcor[nt] = mfma16(xt[ci][q], wreg[ci][nt][q], zcor[nt]);
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
    // per-window vectors for the embedding update: [0] dz+dz~ (context
    // positions), [1] dz (true centre), [2] dz~ (corrupt row)
    if (w < 3) {
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int row = row0 + 4 * g + i;
          if (row < a.B) {
            const float v = (w == 0) ? dsum[nt][i] : (w == 1 ? dz[nt][i] : dzt[nt][i]);
            a.dzz[((size_t)row * 3 + w) * a.Hp + nt * 16 + n16] = v;
          }
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
