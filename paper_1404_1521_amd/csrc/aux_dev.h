// Score, gather and standalone scatter-add kernels.
#pragma once
#include "common.h"
#include "launch.h"
#include "seg_dev.h"
#include "sort_dev.h"

namespace pg {

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
  const ChunkInfo ci = chunk_info(a.sk, a.sv, a.N, chunk, a.ch);
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
        const int k = __builtin_amdgcn_readlane(ci.ent, min(q + r, kWave - 1));
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
    const int nchunks = ceil_div(a.N, a.ch);
    for (int c = blockIdx.x * kWavesPerBlock + w; c < nchunks; c += a.n_e * kWavesPerBlock)
      scatter_chunk(a, c, gbuf, pk);
    return;
  }
  const size_t gid = (size_t)(blockIdx.x - a.n_e) * kBlock + t;
  zero_ranges(a.zero, gid, (size_t)a.n_z * kBlock);
}

__global__ __launch_bounds__(kBlock) void k_scatter_segfix(ScatArgs a) {
  // one workgroup per row; wave w adds chunks cs+1+w, cs+5+w, ... (wave 0
  // also the open piece of the start chunk); wave sums are added in order
  __shared__ float red[kWavesPerBlock][kMaxD];
  const int t = threadIdx.x, lane = t & (kWave - 1), w = t / kWave;
  const uint32_t cnt = *a.long_count;
  if (blockIdx.x >= cnt || *reinterpret_cast<volatile uint32_t*>(a.flag)) return;
  constexpr int U = kMaxD / kWave;
  constexpr int R = 8;
  for (uint32_t li = blockIdx.x; li < cnt; li += gridDim.x) {
    const int cs = a.long_list[li];
    const int32_t key = a.sk[(size_t)cs * a.ch + a.ch - 1];
    const int ce = cs + seg_count_fwd(a.sk, a.N, cs, key, a.ch);
    float acc[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int col = lane + u * kWave;
      acc[u] = (w == 0 && col < a.d) ? a.seg_part[((size_t)cs * 2 + 1) * a.seg_stride + col] : 0.f;
    }
    for (int y0 = cs + 1 + w; y0 <= ce; y0 += R * kWavesPerBlock) {
      float v[R][U];
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const int y = y0 + r * kWavesPerBlock;
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int col = lane + u * kWave;
          v[r][u] = (y <= ce && col < a.d) ? a.seg_part[((size_t)y * 2) * a.seg_stride + col] : 0.f;
        }
      }
#pragma unroll
      for (int r = 0; r < R; ++r)
#pragma unroll
        for (int u = 0; u < U; ++u) acc[u] += v[r][u];
    }
    __syncthreads();  // previous row's reduction buffer is no longer read
#pragma unroll
    for (int u = 0; u < U; ++u) red[w][lane + u * kWave] = acc[u];
    __syncthreads();
    if (w == 0) {
      float* tr = a.table + (size_t)key * a.d;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int col = lane + u * kWave;
        float s = red[0][col];
#pragma unroll
        for (int v = 1; v < kWavesPerBlock; ++v) s += red[v][col];
        if (col < a.d) tr[col] = tr[col] + s;
      }
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
    unsafeAtomicAdd(a.table + (size_t)a.idx[k] * a.d + col, a.alpha * a.Y[i]);
  }
}


}  // namespace pg
