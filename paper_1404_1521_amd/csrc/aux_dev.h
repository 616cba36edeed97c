// Score, gather and index-check kernels.
#pragma once
#include "common.h"
#include "fwdbwd_dev.h"
#include "launch.h"

namespace pg {

// =============================================================== score

template <int NT, int CPW>
__global__ __launch_bounds__(kBlock) void k_score(ScoreArgs a) {
  extern __shared__ uint32_t lds[];
  const int t = threadIdx.x, lane = t & (kWave - 1);
  const int w = __builtin_amdgcn_readfirstlane(t / kWave);
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
    for (int i = 0; i < 4; ++i) ps[i] += w2v * tanh_fast(b1v + Z[i]);
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

// =============================================================== index check

__global__ __launch_bounds__(kBlock) void k_check_idx(const int32_t* idx, int N, int rows,
                                                      uint32_t* flag) {
  bool bad = false;
  for (int i = blockIdx.x * kBlock + threadIdx.x; i < N; i += gridDim.x * kBlock)
    bad |= (uint32_t)idx[i] >= (uint32_t)rows;
  if (bad) atomicOr(flag, kFlagBadId);
}


}  // namespace pg
