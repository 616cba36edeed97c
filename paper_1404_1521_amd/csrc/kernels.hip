// HIP kernels (gfx950) of the Polyglot window-ranking SGD step.
//
// One step on the device (sorted mode):
//
//   k_step_fwdbwd   workgroups [0, n_sort): the entry sort (whole sort in one
//                   workgroup for small batches, else pass-0 digit counts);
//                   workgroups [n_sort, ...): per 16-window tile, gather the
//                   embedding rows straight into MFMA operands, hidden layer
//                   z = W1 x + b1 and the corrupted-centre z~ (16x16x4 f32
//                   MFMA, split-K over 4 waves), tanh, scores, hinge, dz and
//                   dz~, and this workgroup's share of dW1/db1/dw2/loss;
//   k_sort_down     one launch per radix pass for large batches;
//   k_step_update   workgroups [0, n_e): embedding rows -- per sorted row id,
//                   the dz-space vectors of its entries are summed per window
//                   position and multiplied once by W1^T, E[row] -= lr * grad
//                   (or the atomic variant); workgroups [n_e, ...): reduce the
//                   dense partials in slot order, SGD on W1/b1/w2/b2, write
//                   the mean loss, clear the sort counters for the next call;
//   k_step_segfix   rows whose entries span several chunks (Zipf heavy rows).
//
// Model (§1 Introduction; SENNA-style window ranker):
//   s(x) = w2 . tanh(W1 x + b1) + b2,  loss = mean max(0, 1 - s(x) + s(x~)).
// The embedding update is the advanced-indexing increment of §4.2 (Table 1)
// that §4.3 parallelises.
//
// Global loads are always issued in batches whose values are used only after
// the whole batch is in flight: a use right after each load would serialise
// one memory round trip per element.
#include "common.h"
#include "launch.h"
#include "seg_dev.h"
#include "sort_dev.h"

namespace pg {

__device__ __forceinline__ f4 mfma16(float a, float b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ f4 ld4(const float* p) { return *reinterpret_cast<const f4*>(p); }
__device__ __forceinline__ void st4(float* p, f4 v) { *reinterpret_cast<f4*>(p) = v; }

constexpr f4 kZero4 = {0.f, 0.f, 0.f, 0.f};

// =============================================================== step: fwd/bwd

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
    for (int i = t; i < a.Hp * a.K; i += kBlock) {
      const int n = i / a.K;
      a.w1snap[i] = n < a.H ? a.W1[i] : 0.f;
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

template <int NT, int CPW>
__global__ __launch_bounds__(kBlock) void k_step_fwdbwd(FwdArgs a) {
  extern __shared__ uint32_t lds[];
  if ((int)blockIdx.x < a.n_sort) {
    const StepKeys kf{a.windows, a.corrupt, a.win, a.V};
    if (a.sort_small)
      small_sort(kf, a.N, a.plan, a.sb.keys[a.plan.passes & 1], a.sb.vals[a.plan.passes & 1],
                 a.flag, lds);
    else
      sort_up0_tile(kf, a.N, a.plan, a.sb, blockIdx.x, lds);
    return;
  }
  fwdbwd_wg<NT, CPW>(a, blockIdx.x - a.n_sort, lds);
}

// =============================================================== sort passes

template <class KeyFn>
__global__ __launch_bounds__(kBlock) void k_sort_down(KeyFn kf, int N, SortPlan plan, SortBufs sb,
                                                      int p) {
  extern __shared__ uint32_t lds[];
  sort_down_tile(kf, N, plan, sb, p, blockIdx.x, lds);
}

template <class KeyFn>
__global__ __launch_bounds__(kBlock) void k_sort_first(KeyFn kf, int N, SortPlan plan, SortBufs sb,
                                                       uint32_t* long_count) {
  extern __shared__ uint32_t lds[];
  if (blockIdx.x == 0 && threadIdx.x == 0) *long_count = 0u;
  if (plan.small)
    small_sort(kf, N, plan, sb.keys[plan.passes & 1], sb.vals[plan.passes & 1], sb.flag, lds);
  else
    sort_up0_tile(kf, N, plan, sb, blockIdx.x, lds);
}

// =============================================================== row updates

// Writes rows[s] += scale * gbuf[s] for the nslot buffered rows of this wave,
// every row load of the group in flight at once.
__device__ __forceinline__ void flush_rows(float* T, int d, float scale, const float* gbuf,
                                           const int32_t* pk, int nslot) {
  wave_lds_sync();
  const int lane = lane_id();
  const int q4 = d / 4;
  const int total = nslot * q4;
  constexpr int MAXPER = kFlushGroup * kMaxD / 4 / kWave;
  f4 ev[MAXPER];
#pragma unroll
  for (int u = 0; u < MAXPER; ++u) {
    const int i = lane + u * kWave;
    if (i < total) {
      const int s = i / q4, q = i - s * q4;
      ev[u] = ld4(T + (size_t)pk[s] * d + 4 * q);
    }
  }
#pragma unroll
  for (int u = 0; u < MAXPER; ++u) {
    const int i = lane + u * kWave;
    if (i < total) {
      const int s = i / q4, q = i - s * q4;
      const f4 gv = *reinterpret_cast<const f4*>(gbuf + s * d + 4 * q);
      st4(T + (size_t)pk[s] * d + 4 * q, ev[u] + scale * gv);
    }
  }
  wave_lds_sync();
}

// Loads the dz-space vector of this lane's entry into LDS row `lane` of vec
// (stride Hp+4) and returns its window position block (c for a corrupt id).
__device__ __forceinline__ int stage_step_vectors(const UpdArgs& a, int ent, bool act,
                                                  float* vec) {
  const int lane = lane_id();
  const int b = ent / (a.win + 1);
  const int jj = ent - b * (a.win + 1);
  const int v = (jj < a.win) ? (jj == a.c ? 1 : 0) : 2;
  const float* src = a.dzz + ((size_t)b * 3 + v) * a.Hp;
  f4 buf[kMaxHp / 4];
#pragma unroll
  for (int k = 0; k < kMaxHp / 4; ++k) buf[k] = (act && 4 * k < a.Hp) ? ld4(src + 4 * k) : kZero4;
  const int stride = a.Hp + 4;
#pragma unroll
  for (int k = 0; k < kMaxHp / 4; ++k)
    if (4 * k < a.Hp) st4(vec + lane * stride + 4 * k, buf[k]);
  return (jj < a.win) ? jj : a.c;
}

// grad[col] = sum over touched positions j of sum_n W1[n][j*d + col] * S_j[n],
// S_j[n] held by lane n; lane-strided columns.
template <int WMAX>
__device__ __forceinline__ void row_grad(const float* w1s, const float (&S)[WMAX], uint32_t mask,
                                         int H, int K, int d, float (&gacc)[kMaxD / kWave]) {
  const int lane = lane_id();
#pragma unroll
  for (int u = 0; u < kMaxD / kWave; ++u) gacc[u] = 0.f;
#pragma unroll
  for (int j = 0; j < WMAX; ++j) {
    if (!((mask >> j) & 1u)) continue;
#pragma unroll 4
    for (int n = 0; n < H; ++n) {
      const float s = readlane_f(S[j], n);
      const float* wr = w1s + (size_t)n * K + j * d;
#pragma unroll
      for (int u = 0; u < kMaxD / kWave; ++u) {
        const int col = lane + u * kWave;
        if (col < d) gacc[u] += wr[col] * s;
      }
    }
  }
}

template <int WMAX>
__device__ void step_rows_chunk(const UpdArgs& a, int chunk, const float* w1s, float* vec,
                                float* gbuf, int32_t* pk) {
  const int lane = lane_id();
  const ChunkInfo ci = chunk_info(a.sk, a.sv, a.N, chunk);
  const int stride = a.Hp + 4;
  const int blk_l = stage_step_vectors(a, ci.ent, lane < ci.nact, vec);
  wave_lds_sync();
  int nslot = 0;
  for (int p0 = 0; p0 < ci.nact;) {
    const int p1 = piece_end(ci, p0);
    const int32_t pkey = __builtin_amdgcn_readlane(ci.key, p0);
    float S[WMAX];
#pragma unroll
    for (int j = 0; j < WMAX; ++j) S[j] = 0.f;
    uint32_t mask = 0;
    for (int q = p0; q < p1; ++q) {
      const int blk = __builtin_amdgcn_readlane(blk_l, q);
      const float val = lane < a.Hp ? vec[q * stride + lane] : 0.f;
#pragma unroll
      for (int j = 0; j < WMAX; ++j)
        if (j == blk) S[j] += val;
      mask |= 1u << blk;
    }
    const bool is_cont = p0 == 0 && ci.cont_first;
    const bool is_open = p1 == ci.nact && ci.open_last;
    if (!is_cont && !is_open) {
      float gacc[kMaxD / kWave];
      row_grad<WMAX>(w1s, S, mask, a.H, a.K, a.d, gacc);
#pragma unroll
      for (int u = 0; u < kMaxD / kWave; ++u) {
        const int col = lane + u * kWave;
        if (col < a.d) gbuf[nslot * a.d + col] = gacc[u];
      }
      if (lane == 0) pk[nslot] = pkey;
      if (++nslot == kFlushGroup) {
        flush_rows(a.E, a.d, -a.lr, gbuf, pk, nslot);
        nslot = 0;
      }
    } else {
      float* dst = a.seg_part + ((size_t)chunk * 2 + (is_cont ? 0 : 1)) * a.seg_stride;
#pragma unroll
      for (int j = 0; j < WMAX; ++j)
        if (j < a.win && lane < a.Hp) dst[j * a.Hp + lane] = S[j];
      if (is_open && !is_cont && lane == 0) a.long_list[atomicAdd(a.long_count, 1u)] = chunk;
    }
    p0 = p1;
  }
  if (nslot) flush_rows(a.E, a.d, -a.lr, gbuf, pk, nslot);
}

// Atomic variant (the per-(entry, column) increment of §4.3's kernel, in
// entry order): one float atomic add per element, rounding in arrival order.
__device__ void step_rows_atomic(const UpdArgs& a, int chunk, const float* w1s, float* vec) {
  const int lane = lane_id();
  const int i0 = chunk * kSegChunk;
  const int nact = min(kSegChunk, a.N - i0);
  const int ent = i0 + lane;
  const bool act = lane < nact;
  int32_t key_l = 0;
  if (act) {
    const int b = ent / (a.win + 1);
    const int jj = ent - b * (a.win + 1);
    key_l = (jj < a.win) ? a.windows[(size_t)b * a.win + jj] : a.corrupt[b];
  }
  const int stride = a.Hp + 4;
  const int blk_l = stage_step_vectors(a, ent, act, vec);
  wave_lds_sync();
  for (int q = 0; q < nact; ++q) {
    const int blk = __builtin_amdgcn_readlane(blk_l, q);
    const int32_t key = __builtin_amdgcn_readlane(key_l, q);
    float gacc[kMaxD / kWave];
#pragma unroll
    for (int u = 0; u < kMaxD / kWave; ++u) gacc[u] = 0.f;
#pragma unroll 4
    for (int n = 0; n < a.H; ++n) {
      const float s = vec[q * stride + n];
      const float* wr = w1s + (size_t)n * a.K + blk * a.d;
#pragma unroll
      for (int u = 0; u < kMaxD / kWave; ++u) {
        const int col = lane + u * kWave;
        if (col < a.d) gacc[u] += wr[col] * s;
      }
    }
#pragma unroll
    for (int u = 0; u < kMaxD / kWave; ++u) {
      const int col = lane + u * kWave;
      if (col < a.d) atomicAdd(a.E + (size_t)key * a.d + col, -a.lr * gacc[u]);
    }
  }
}

__device__ __forceinline__ void zero_ranges(const ZeroRanges& z, size_t gid, size_t nthreads) {
#pragma unroll
  for (int r = 0; r < 3; ++r)
    for (size_t i = gid; i < z.n[r]; i += nthreads) z.p[r][i] = 0u;
}

// LDS floats of the embedding role: W1 copy + per wave (vectors, gradient
// rows, row keys).
__host__ __device__ inline size_t update_lds_floats(int Hp, int K, int d) {
  return (size_t)Hp * K + (size_t)kWavesPerBlock * (kSegChunk * (Hp + 4) + kFlushGroup * d + 16);
}

template <int WMAX>
__global__ __launch_bounds__(kBlock) void k_step_update(UpdArgs a) {
  extern __shared__ uint32_t lds[];
  const int t = threadIdx.x, w = t / kWave;
  const bool bad = (*reinterpret_cast<volatile uint32_t*>(a.flag)) != 0u;

  if ((int)blockIdx.x < a.n_e) {
    if (bad) return;  // all-or-nothing: an out-of-range id voids the step
    float* w1s = reinterpret_cast<float*>(lds);
    float* wv = w1s + (size_t)a.Hp * a.K + (size_t)w * (kSegChunk * (a.Hp + 4) + kFlushGroup * a.d + 16);
    float* vec = wv;
    float* gbuf = vec + kSegChunk * (a.Hp + 4);
    int32_t* pk = reinterpret_cast<int32_t*>(gbuf + kFlushGroup * a.d);
    for (int i = 4 * t; i < a.Hp * a.K; i += 4 * kBlock) st4(w1s + i, ld4(a.w1snap + i));
    __syncthreads();
    const int nchunks = ceil_div(a.N, kSegChunk);
    for (int ch = blockIdx.x * kWavesPerBlock + w; ch < nchunks; ch += a.n_e * kWavesPerBlock) {
      if (a.mode == 0)
        step_rows_chunk<WMAX>(a, ch, w1s, vec, gbuf, pk);
      else
        step_rows_atomic(a, ch, w1s, vec);
    }
    return;
  }

  // ---- dense role: reduce the fwd/bwd partials in slot order, apply SGD
  const int gid = (blockIdx.x - a.n_e) * kBlock + t;
  const int nthreads = a.n_d * kBlock;
  const int HK = a.Hp * a.K;
  const int nel = HK + 2 * a.Hp + 2;
  for (int e = gid; e < nel; e += nthreads) {
    float s = 0.f;
    int p = 0;
    for (; p + 8 <= a.n_parts; p += 8) {
      float v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = a.part[(size_t)(p + u) * a.part_stride + e];
#pragma unroll
      for (int u = 0; u < 8; ++u) s += v[u];
    }
    for (; p < a.n_parts; ++p) s += a.part[(size_t)p * a.part_stride + e];
    if (e < HK) {
      if (!bad && e / a.K < a.H) a.W1[e] = a.W1[e] - a.lr * s;
    } else if (e < HK + a.Hp) {
      const int n = e - HK;
      if (!bad && n < a.H) a.b1[n] = a.b1[n] - a.lr * s;
    } else if (e < HK + 2 * a.Hp) {
      const int n = e - HK - a.Hp;
      if (!bad && n < a.H) a.w2[n] = a.w2[n] - a.lr * s;
    } else if (e == HK + 2 * a.Hp) {
      a.loss_out[0] = bad ? __builtin_nanf("") : s * a.invB;
    } else {
      if (!bad) a.b2[0] = a.b2[0] - a.lr * s;
    }
  }
  zero_ranges(a.zero, gid, nthreads);
}

// Rows whose sorted entries span several chunks: add the chunk partials in
// chunk order, one W1^T product per window position, update the row.
template <int WMAX>
__global__ __launch_bounds__(kBlock) void k_step_segfix(UpdArgs a) {
  extern __shared__ uint32_t lds[];
  const int t = threadIdx.x, lane = t & (kWave - 1), w = t / kWave;
  const uint32_t cnt = *a.long_count;
  if (blockIdx.x * kWavesPerBlock >= cnt || *reinterpret_cast<volatile uint32_t*>(a.flag)) return;
  float* w1s = reinterpret_cast<float*>(lds);
  for (int i = 4 * t; i < a.Hp * a.K; i += 4 * kBlock) st4(w1s + i, ld4(a.w1snap + i));
  __syncthreads();
  for (uint32_t li = blockIdx.x * kWavesPerBlock + w; li < cnt; li += gridDim.x * kWavesPerBlock) {
    const int cs = a.long_list[li];
    const int32_t key = a.sk[(size_t)cs * kSegChunk + kSegChunk - 1];
    const int ce = cs + seg_count_fwd(a.sk, a.N, cs, key);
    float S[WMAX];
#pragma unroll
    for (int j = 0; j < WMAX; ++j) {
      const float* src = a.seg_part + ((size_t)cs * 2 + 1) * a.seg_stride;
      S[j] = (j < a.win && lane < a.Hp) ? src[j * a.Hp + lane] : 0.f;
    }
    for (int y0 = cs + 1; y0 <= ce; y0 += 4) {
      float v[4][WMAX];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const float* src = a.seg_part + ((size_t)(y0 + u) * 2) * a.seg_stride;
#pragma unroll
        for (int j = 0; j < WMAX; ++j)
          v[u][j] = (y0 + u <= ce && j < a.win && lane < a.Hp) ? src[j * a.Hp + lane] : 0.f;
      }
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int j = 0; j < WMAX; ++j) S[j] += v[u][j];
    }
    float gacc[kMaxD / kWave];
    const uint32_t mask = (a.win >= 32) ? 0xffffffffu : ((1u << a.win) - 1u);
    row_grad<WMAX>(w1s, S, mask, a.H, a.K, a.d, gacc);
    float* er = a.E + (size_t)key * a.d;
#pragma unroll
    for (int u = 0; u < kMaxD / kWave; ++u) {
      const int col = lane + u * kWave;
      if (col < a.d) er[col] = er[col] - a.lr * gacc[u];
    }
  }
}

// =============================================================== score

template <int NT, int CPW>
__global__ __launch_bounds__(kBlock) void k_score(ScoreArgs a) {
  extern __shared__ uint32_t lds[];
  const int t = threadIdx.x, lane = t & (kWave - 1), w = t / kWave;
  const int n16 = lane & 15, g = lane >> 4;
  const int dq = a.d / 16, nchunk = a.K / 16;
  int32_t* ids = reinterpret_cast<int32_t*>(lds);                  // [16][win]
  int32_t* badrow = ids + kTileRows * kMaxWin;                      // [16]
  f4* zp = reinterpret_cast<f4*>(lds + kTileRows * (kMaxWin + 1));  // [4][NT][64]
  const int row0 = blockIdx.x * kTileRows;
  if (t < kTileRows) badrow[t] = 0;
  __syncthreads();
  for (int i = t; i < kTileRows * a.win; i += kBlock) {
    const int r = i / a.win, j = i - r * a.win;
    const int b = row0 + r;
    const int32_t id = b < a.B ? a.windows[(size_t)b * a.win + j] : 0;
    const bool bad = (uint32_t)id >= (uint32_t)a.V;
    if (bad) {
      atomicOr(a.flag, kFlagBadId);
      badrow[r] = 1;
    }
    ids[i] = bad ? 0 : id;
  }
  __syncthreads();
  f4 x[CPW], wv[CPW][NT];
#pragma unroll
  for (int ci = 0; ci < CPW; ++ci) {
    const int kc = w + kWavesPerBlock * ci;
    const bool ok = kc < nchunk;
    const int j = ok ? kc / dq : 0;
    const int off = (kc - j * dq) * 16 + 4 * g;
    x[ci] = ok ? ld4(a.E + (size_t)ids[n16 * a.win + j] * a.d + off) : kZero4;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const int n = nt * 16 + n16;
      wv[ci][nt] = (ok && n < a.H) ? ld4(a.W1 + (size_t)n * a.K + kc * 16 + 4 * g) : kZero4;
    }
  }
  f4 z[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) z[nt] = kZero4;
#pragma unroll
  for (int ci = 0; ci < CPW; ++ci)
    if (w + kWavesPerBlock * ci < nchunk)
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) z[nt] = mfma16(x[ci][q], wv[ci][nt][q], z[nt]);
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) zp[(w * NT + nt) * kWave + lane] = z[nt];
  __syncthreads();
  if (w != 0) return;
  float ps[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    f4 Z = zp[(0 * NT + nt) * kWave + lane];
#pragma unroll
    for (int v = 1; v < kWavesPerBlock; ++v) Z += zp[(v * NT + nt) * kWave + lane];
    const int n = nt * 16 + n16;
    const float b1v = n < a.H ? a.b1[n] : 0.f, w2v = n < a.H ? a.w2[n] : 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) ps[i] += w2v * tanhf(b1v + Z[i]);
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) ps[i] += __shfl_xor(ps[i], o);
  if (n16 == 0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = 4 * g + i, b = row0 + r;
      if (b < a.B) a.scores[b] = badrow[r] ? __builtin_nanf("") : a.b2[0] + ps[i];
    }
  }
}

// =============================================================== gather

__global__ __launch_bounds__(kBlock) void k_gather(GatherArgs a) {
  // one thread per float4 of output; position j == win is the corrupt row
  const int q4 = a.d / 4;
  const size_t total = (size_t)a.B * (a.win + 1) * q4;
  for (size_t i = (size_t)blockIdx.x * kBlock + threadIdx.x; i < total;
       i += (size_t)gridDim.x * kBlock) {
    const size_t rowi = i / q4;
    const int q = (int)(i - rowi * q4);
    const int b = (int)(rowi / (a.win + 1));
    const int j = (int)(rowi - (size_t)b * (a.win + 1));
    const int32_t id = (j < a.win) ? a.windows[(size_t)b * a.win + j] : a.corrupt[b];
    f4 v;
    if ((uint32_t)id < (uint32_t)a.V) {
      v = ld4(a.E + (size_t)id * a.d + 4 * q);
    } else {
      if (q == 0) atomicOr(a.flag, kFlagBadId);
      const float nan = __builtin_nanf("");
      v = f4{nan, nan, nan, nan};
    }
    float* dst = (j < a.win) ? a.X + ((size_t)b * a.win + j) * a.d + 4 * q
                             : a.Xc + (size_t)b * a.d + 4 * q;
    st4(dst, v);
  }
}

// =============================================================== scatter-add

// LDS floats of the scatter segment role (per wave: gradient rows + keys).
__host__ __device__ inline size_t scatter_lds_floats(int d) {
  return (size_t)kWavesPerBlock * (kFlushGroup * d + 16);
}

__device__ void scatter_chunk(const ScatArgs& a, int chunk, float* gbuf, int32_t* pk) {
  const int lane = lane_id();
  const ChunkInfo ci = chunk_info(a.sk, a.sv, a.N, chunk);
  constexpr int U = kMaxD / kWave;
  int nslot = 0;
  for (int p0 = 0; p0 < ci.nact;) {
    const int p1 = piece_end(ci, p0);
    const int32_t pkey = __builtin_amdgcn_readlane(ci.key, p0);
    float acc[U];
#pragma unroll
    for (int u = 0; u < U; ++u) acc[u] = 0.f;
    for (int q = p0; q < p1; q += 8) {  // 8 rows of Y in flight, added in entry order
      float v[8][U];
#pragma unroll
      for (int r = 0; r < 8; ++r) {
        const int k = __builtin_amdgcn_readlane(ci.ent, min(q + r, kSegChunk - 1));
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int col = lane + u * kWave;
          v[r][u] = (q + r < p1 && col < a.d) ? a.Y[(size_t)k * a.d + col] : 0.f;
        }
      }
#pragma unroll
      for (int r = 0; r < 8; ++r)
#pragma unroll
        for (int u = 0; u < U; ++u) acc[u] += a.alpha * v[r][u];
    }
    const bool is_cont = p0 == 0 && ci.cont_first;
    const bool is_open = p1 == ci.nact && ci.open_last;
    if (!is_cont && !is_open) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int col = lane + u * kWave;
        if (col < a.d) gbuf[nslot * a.d + col] = acc[u];
      }
      if (lane == 0) pk[nslot] = pkey;
      if (++nslot == kFlushGroup) {
        flush_rows(a.table, a.d, 1.f, gbuf, pk, nslot);
        nslot = 0;
      }
    } else {
      float* dst = a.seg_part + ((size_t)chunk * 2 + (is_cont ? 0 : 1)) * a.seg_stride;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int col = lane + u * kWave;
        if (col < a.d) dst[col] = acc[u];
      }
      if (is_open && !is_cont && lane == 0) a.long_list[atomicAdd(a.long_count, 1u)] = chunk;
    }
    p0 = p1;
  }
  if (nslot) flush_rows(a.table, a.d, 1.f, gbuf, pk, nslot);
}

__global__ __launch_bounds__(kBlock) void k_scatter_segments(ScatArgs a) {
  extern __shared__ uint32_t lds[];
  const int t = threadIdx.x, w = t / kWave;
  const bool bad = (*reinterpret_cast<volatile uint32_t*>(a.flag)) != 0u;
  if ((int)blockIdx.x < a.n_e) {
    if (bad) return;
    float* gbuf = reinterpret_cast<float*>(lds) + (size_t)w * (kFlushGroup * a.d + 16);
    int32_t* pk = reinterpret_cast<int32_t*>(gbuf + kFlushGroup * a.d);
    const int nchunks = ceil_div(a.N, kSegChunk);
    for (int ch = blockIdx.x * kWavesPerBlock + w; ch < nchunks; ch += a.n_e * kWavesPerBlock)
      scatter_chunk(a, ch, gbuf, pk);
    return;
  }
  const size_t gid = (size_t)(blockIdx.x - a.n_e) * kBlock + t;
  zero_ranges(a.zero, gid, (size_t)a.n_z * kBlock);
}

__global__ __launch_bounds__(kBlock) void k_scatter_segfix(ScatArgs a) {
  const int t = threadIdx.x, lane = t & (kWave - 1), w = t / kWave;
  const uint32_t cnt = *a.long_count;
  if (blockIdx.x * kWavesPerBlock >= cnt || *reinterpret_cast<volatile uint32_t*>(a.flag)) return;
  constexpr int U = kMaxD / kWave;
  for (uint32_t li = blockIdx.x * kWavesPerBlock + w; li < cnt; li += gridDim.x * kWavesPerBlock) {
    const int cs = a.long_list[li];
    const int32_t key = a.sk[(size_t)cs * kSegChunk + kSegChunk - 1];
    const int ce = cs + seg_count_fwd(a.sk, a.N, cs, key);
    float acc[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int col = lane + u * kWave;
      acc[u] = col < a.d ? a.seg_part[((size_t)cs * 2 + 1) * a.seg_stride + col] : 0.f;
    }
    for (int y0 = cs + 1; y0 <= ce; y0 += 8) {
      float v[8][U];
#pragma unroll
      for (int r = 0; r < 8; ++r)
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int col = lane + u * kWave;
          v[r][u] = (y0 + r <= ce && col < a.d)
                        ? a.seg_part[((size_t)(y0 + r) * 2) * a.seg_stride + col] : 0.f;
        }
#pragma unroll
      for (int r = 0; r < 8; ++r)
#pragma unroll
        for (int u = 0; u < U; ++u) acc[u] += v[r][u];
    }
    float* tr = a.table + (size_t)key * a.d;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int col = lane + u * kWave;
      if (col < a.d) tr[col] = tr[col] + acc[u];
    }
  }
}

__global__ __launch_bounds__(kBlock) void k_check_idx(const int32_t* idx, int N, int rows,
                                                      uint32_t* flag) {
  bool bad = false;
  for (int i = blockIdx.x * kBlock + threadIdx.x; i < N; i += gridDim.x * kBlock)
    bad |= (uint32_t)idx[i] >= (uint32_t)rows;
  if (bad) atomicOr(flag, kFlagBadId);
}

__global__ __launch_bounds__(kBlock) void k_scatter_atomic(ScatArgs a) {
  if (*reinterpret_cast<volatile uint32_t*>(a.flag)) return;
  const size_t total = (size_t)a.N * a.d;
  for (size_t i = (size_t)blockIdx.x * kBlock + threadIdx.x; i < total;
       i += (size_t)gridDim.x * kBlock) {
    const size_t k = i / a.d;
    const int col = (int)(i - k * a.d);
    atomicAdd(a.table + (size_t)a.idx[k] * a.d + col, a.alpha * a.Y[i]);
  }
}

// =============================================================== launchers

static hipError_t launch_err() { return hipGetLastError(); }

template <int NT, int CPW>
static void launch_fwdbwd_t(const FwdArgs& a, int grid, size_t lds, hipStream_t s) {
  hipLaunchKernelGGL((k_step_fwdbwd<NT, CPW>), dim3(grid), dim3(kBlock), lds, s, a);
}

template <int NT>
static void launch_fwdbwd_nt(const FwdArgs& a, int cpw, int grid, size_t lds, hipStream_t s) {
  if (cpw <= 2)
    launch_fwdbwd_t<NT, 2>(a, grid, lds, s);
  else if (cpw <= 5)
    launch_fwdbwd_t<NT, 5>(a, grid, lds, s);
  else
    launch_fwdbwd_t<NT, 8>(a, grid, lds, s);
}

hipError_t launch_step_fwdbwd(const FwdArgs& a, int NT, int cpw, int grid, size_t lds,
                              hipStream_t s) {
  if (NT == 1)
    launch_fwdbwd_nt<1>(a, cpw, grid, lds, s);
  else if (NT == 2)
    launch_fwdbwd_nt<2>(a, cpw, grid, lds, s);
  else
    launch_fwdbwd_nt<4>(a, cpw, grid, lds, s);
  return launch_err();
}

hipError_t launch_sort_down_step(const StepKeys& kf, int N, const SortPlan& plan,
                                 const SortBufs& sb, int p, hipStream_t s) {
  hipLaunchKernelGGL((k_sort_down<StepKeys>), dim3(plan.ntiles), dim3(kBlock),
                     kDownLdsWords * 4, s, kf, N, plan, sb, p);
  return launch_err();
}

hipError_t launch_step_update(const UpdArgs& a, int grid, size_t lds, hipStream_t s) {
  if (a.win <= 8)
    hipLaunchKernelGGL((k_step_update<8>), dim3(grid), dim3(kBlock), lds, s, a);
  else if (a.win <= 16)
    hipLaunchKernelGGL((k_step_update<16>), dim3(grid), dim3(kBlock), lds, s, a);
  else
    hipLaunchKernelGGL((k_step_update<32>), dim3(grid), dim3(kBlock), lds, s, a);
  return launch_err();
}

hipError_t launch_step_segfix(const UpdArgs& a, size_t lds, hipStream_t s) {
  if (a.win <= 8)
    hipLaunchKernelGGL((k_step_segfix<8>), dim3(kSegfixBlocks), dim3(kBlock), lds, s, a);
  else if (a.win <= 16)
    hipLaunchKernelGGL((k_step_segfix<16>), dim3(kSegfixBlocks), dim3(kBlock), lds, s, a);
  else
    hipLaunchKernelGGL((k_step_segfix<32>), dim3(kSegfixBlocks), dim3(kBlock), lds, s, a);
  return launch_err();
}

hipError_t launch_score(const ScoreArgs& a, int NT, int cpw, hipStream_t s) {
  const int grid = ceil_div(a.B, kTileRows);
  const size_t lds = (kTileRows * (kMaxWin + 1)) * 4 + kWavesPerBlock * kMaxNT * kWave * 16;
#define PG_SCORE(NTV, CPWV) \
  hipLaunchKernelGGL((k_score<NTV, CPWV>), dim3(grid), dim3(kBlock), lds, s, a)
  if (NT == 1) {
    if (cpw <= 2) PG_SCORE(1, 2); else if (cpw <= 5) PG_SCORE(1, 5); else PG_SCORE(1, 8);
  } else if (NT == 2) {
    if (cpw <= 2) PG_SCORE(2, 2); else if (cpw <= 5) PG_SCORE(2, 5); else PG_SCORE(2, 8);
  } else {
    if (cpw <= 2) PG_SCORE(4, 2); else if (cpw <= 5) PG_SCORE(4, 5); else PG_SCORE(4, 8);
  }
#undef PG_SCORE
  return launch_err();
}

hipError_t launch_gather(const GatherArgs& a, hipStream_t s) {
  const size_t total = (size_t)a.B * (a.win + 1) * (a.d / 4);
  const size_t want = (total + kBlock - 1) / kBlock;
  const int grid = (int)(want < 8192 ? (want > 0 ? want : 1) : 8192);
  hipLaunchKernelGGL(k_gather, dim3(grid), dim3(kBlock), 0, s, a);
  return launch_err();
}

hipError_t launch_scatter_sorted(const ScatArgs& a, const SortPlan& plan, const SortBufs& sb,
                                 hipStream_t s) {
  const IdxKeys kf{a.idx, a.rows};
  const size_t lds0 = plan.small ? kSmallSortLdsWords * 4 : kUp0LdsWords * 4;
  hipLaunchKernelGGL((k_sort_first<IdxKeys>), dim3(plan.small ? 1 : plan.ntiles), dim3(kBlock),
                     lds0, s, kf, a.N, plan, sb, a.long_count);
  if (!plan.small)
    for (int p = 0; p < plan.passes; ++p)
      hipLaunchKernelGGL((k_sort_down<IdxKeys>), dim3(plan.ntiles), dim3(kBlock),
                         kDownLdsWords * 4, s, kf, a.N, plan, sb, p);
  hipLaunchKernelGGL(k_scatter_segments, dim3(a.n_e + a.n_z), dim3(kBlock),
                     scatter_lds_floats(a.d) * 4, s, a);
  hipLaunchKernelGGL(k_scatter_segfix, dim3(kSegfixBlocks), dim3(kBlock), 0, s, a);
  return launch_err();
}

hipError_t launch_scatter_atomic(const ScatArgs& a, hipStream_t s) {
  const int g1 = ceil_div(a.N, kBlock) < 1024 ? ceil_div(a.N, kBlock) : 1024;
  hipLaunchKernelGGL(k_check_idx, dim3(g1 > 0 ? g1 : 1), dim3(kBlock), 0, s, a.idx, a.N, a.rows,
                     a.flag);
  const size_t total = (size_t)a.N * a.d;
  const size_t g2 = (total + kBlock - 1) / kBlock;
  hipLaunchKernelGGL(k_scatter_atomic, dim3(g2 < 65536 ? (int)g2 : 65536), dim3(kBlock), 0, s,
                     a);
  return launch_err();
}

size_t step_update_lds_bytes(int Hp, int K, int d) { return update_lds_floats(Hp, K, d) * 4; }

}  // namespace pg
