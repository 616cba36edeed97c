// Embedding-row updates (sorted segments or atomics) and the dense SGD
// reduction of one training step.
//
// Per sorted row id, the dz-space vectors of its entries are summed per
// window position j (S_j, H values), and the row gradient is
// sum_j W1_j^T S_j: one W1^T product per (row, position) instead of one per
// entry, which for Zipf data is several times less work than forming every
// entry's d-wide gradient row.  H-wide loops (compile-time HP) issue their
// loads as one batch before any use.
#pragma once
#include "common.h"
#include "launch.h"
#include "seg_dev.h"

namespace pg {

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

// Window position block of entry `ent` (the corrupt id uses the centre block)
// and which per-window vector it takes: 0 dz+dz~ (context), 1 dz (true
// centre), 2 dz~ (corrupt).
__device__ __forceinline__ void entry_role(const UpdArgs& a, int ent, int& b, int& vsel,
                                           int& blk) {
  b = ent / (a.win + 1);
  const int jj = ent - b * (a.win + 1);
  vsel = (jj < a.win) ? (jj == a.c ? 1 : 0) : 2;
  blk = (jj < a.win) ? jj : a.c;
}

// Loads the dz-space vector of this lane's entry into LDS row `lane` of vec
// (stride HP+4); returns the entry's position block.
template <int HP>
__device__ __forceinline__ int stage_step_vectors(const UpdArgs& a, int ent, bool act,
                                                  float* vec) {
  const int lane = lane_id();
  int b, vsel, blk;
  entry_role(a, ent, b, vsel, blk);
  const float* src = a.dzz + ((size_t)b * 3 + vsel) * HP;
  f4 buf[HP / 4];
#pragma unroll
  for (int k = 0; k < HP / 4; ++k) buf[k] = act ? ld4(src + 4 * k) : kZero4;
#pragma unroll
  for (int k = 0; k < HP / 4; ++k) st4(vec + lane * (HP + 4) + 4 * k, buf[k]);
  return blk;
}

// Gradient of one row, column `col` (clamped into [0, d)):
// sum over positions j in mask of sum_n W1[n][j*d + col] * S_j[n], with the
// S_j in LDS (sb[j*HP + n], read as broadcasts).
template <int HP>
__device__ __forceinline__ float row_grad_col(const float* w1s, const float* sb, uint32_t mask,
                                              int K, int d, int col) {
  float g = 0.f;
  for (uint32_t m = mask; m; m &= m - 1) {
    const int j = __ffs(m) - 1;
    float sv[HP], wv[HP];
#pragma unroll
    for (int n = 0; n < HP; ++n) {
      sv[n] = sb[j * HP + n];
      wv[n] = w1s[n * K + j * d + col];
    }
#pragma unroll
    for (int n = 0; n < HP; ++n) g += wv[n] * sv[n];
  }
  return g;
}

template <int WMAX, int HP>
__device__ void step_rows_chunk(const UpdArgs& a, int chunk, const float* w1s, float* vec,
                                float* gbuf, int32_t* pk, float* sb) {
  constexpr int stride = HP + 4;
  const int lane = lane_id();
  const ChunkInfo ci = chunk_info(a.sk, a.sv, a.N, chunk, a.ch);
  const int blk_l = stage_step_vectors<HP>(a, ci.ent, lane < ci.nact, vec);
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
      const float val = lane < HP ? vec[q * stride + lane] : 0.f;
#pragma unroll
      for (int j = 0; j < WMAX; ++j)
        if (j == blk) S[j] += val;
      mask |= 1u << blk;
    }
    const bool is_cont = p0 == 0 && ci.cont_first;
    const bool is_open = p1 == ci.nact && ci.open_last;
    if (!is_cont && !is_open) {
#pragma unroll
      for (int j = 0; j < WMAX; ++j)
        if (((mask >> j) & 1u) && lane < HP) sb[j * HP + lane] = S[j];
      wave_lds_sync();
      for (int c0 = 0; c0 < a.d; c0 += kWave) {
        const int col = c0 + lane;
        const float g = row_grad_col<HP>(w1s, sb, mask, a.K, a.d, min(col, a.d - 1));
        if (col < a.d) gbuf[nslot * a.d + col] = g;
      }
      if (lane == 0) pk[nslot] = pkey;
      wave_lds_sync();
      if (++nslot == kFlushGroup) {
        flush_rows(a.E, a.d, -a.lr, gbuf, pk, nslot);
        nslot = 0;
      }
    } else {
      float* dst = a.seg_part + ((size_t)chunk * 2 + (is_cont ? 0 : 1)) * a.seg_stride;
#pragma unroll
      for (int j = 0; j < WMAX; ++j)
        if (j < a.win && lane < HP) dst[j * HP + lane] = S[j];
      if (is_open && !is_cont && lane == 0) a.long_list[atomicAdd(a.long_count, 1u)] = chunk;
    }
    p0 = p1;
  }
  if (nslot) flush_rows(a.E, a.d, -a.lr, gbuf, pk, nslot);
}

// Atomic variant: the per-(entry, column) increment of the paper's parallel
// kernel (§4.3), in arrival order, one float atomic per element.  Entries go
// kAtomicChunk to a wave.
template <int HP>
__device__ void step_rows_atomic(const UpdArgs& a, int chunk, const float* w1s, float* vec) {
  constexpr int stride = HP + 4;
  const int lane = lane_id();
  const int i0 = chunk * kAtomicChunk;
  const int nact = min(kAtomicChunk, a.N - i0);
  const int ent = i0 + min(lane, nact - 1);
  const bool act = lane < nact;
  int b, vsel, blk0;
  entry_role(a, ent, b, vsel, blk0);
  const int32_t key_l =
      (vsel == 2) ? a.corrupt[b] : a.windows[(size_t)b * a.win + (ent - b * (a.win + 1))];
  const int blk_l = stage_step_vectors<HP>(a, ent, act, vec);
  wave_lds_sync();
  for (int q = 0; q < nact; ++q) {
    const int blk = __builtin_amdgcn_readlane(blk_l, q);
    const int32_t key = __builtin_amdgcn_readlane(key_l, q);
    for (int c0 = 0; c0 < a.d; c0 += kWave) {
      const int col = c0 + lane;
      const float g =
          row_grad_col<HP>(w1s, vec + q * stride - blk * HP, 1u << blk, a.K, a.d, min(col, a.d - 1));
      if (col < a.d) unsafeAtomicAdd(a.E + (size_t)key * a.d + col, -a.lr * g);
    }
  }
}

__device__ __forceinline__ void zero_ranges(const ZeroRanges& z, size_t gid, size_t nthreads) {
#pragma unroll
  for (int r = 0; r < 3; ++r)
    for (size_t i = gid; i < z.n[r]; i += nthreads) z.p[r][i] = 0u;
}

// LDS floats of the embedding role: W1 copy + per wave (vectors, gradient
// rows, row keys, per-position sums of one row).
__host__ __device__ inline size_t update_wave_floats(int Hp, int d, int wmax) {
  return (size_t)kSegChunk * (Hp + 4) + (size_t)kFlushGroup * d + 16 + (size_t)wmax * Hp;
}
__host__ __device__ inline size_t update_lds_floats(int Hp, int K, int d, int wmax) {
  return (size_t)Hp * K + (size_t)kWavesPerBlock * update_wave_floats(Hp, d, wmax);
}

template <int HP>
__device__ __forceinline__ void stage_w1(const UpdArgs& a, float* w1s) {
  const int t = threadIdx.x;
  constexpr int U = 8;
  const int n4 = HP * a.K / 4;
  for (int i0 = 0; i0 < n4; i0 += kBlock * U) {
    f4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i = i0 + u * kBlock + t;
      v[u] = i < n4 ? ld4(a.w1snap + 4 * i) : kZero4;
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i = i0 + u * kBlock + t;
      if (i < n4) st4(w1s + 4 * i, v[u]);
    }
  }
}

template <int WMAX, int HP>
__global__ __launch_bounds__(kBlock) void k_step_update(UpdArgs a) {
  extern __shared__ uint32_t lds[];
  const int t = threadIdx.x, w = t / kWave;
  const bool bad = (*reinterpret_cast<volatile uint32_t*>(a.flag)) != 0u;

  if ((int)blockIdx.x < a.n_e) {
    if (bad) return;  // all-or-nothing: an out-of-range id voids the step
    float* w1s = reinterpret_cast<float*>(lds);
    float* vec = w1s + (size_t)HP * a.K + (size_t)w * update_wave_floats(HP, a.d, WMAX);
    float* gbuf = vec + kSegChunk * (HP + 4);
    int32_t* pk = reinterpret_cast<int32_t*>(gbuf + kFlushGroup * a.d);
    float* sb = gbuf + kFlushGroup * a.d + 16;
    stage_w1<HP>(a, w1s);
    __syncthreads();
    if (a.mode == 0) {
      const int nchunks = ceil_div(a.N, a.ch);
      for (int ch = blockIdx.x * kWavesPerBlock + w; ch < nchunks; ch += a.n_e * kWavesPerBlock)
        step_rows_chunk<WMAX, HP>(a, ch, w1s, vec, gbuf, pk, sb);
    } else {
      const int nchunks = ceil_div(a.N, kAtomicChunk);
      for (int ch = blockIdx.x * kWavesPerBlock + w; ch < nchunks; ch += a.n_e * kWavesPerBlock)
        step_rows_atomic<HP>(a, ch, w1s, vec);
    }
    return;
  }

  // ---- dense role: reduce the fwd/bwd partials, apply SGD.  Eight adjacent
  // lanes share an element: lane s sums slots s, s+8, ... in order, then a
  // fixed butterfly adds the eight sums (deterministic).
  const int gid = (blockIdx.x - a.n_e) * kBlock + t;
  const int nthreads = a.n_d * kBlock;
  const int HK = HP * a.K;
  const int nel = HK + 2 * HP + 2;
  constexpr int SL = kDenseSlices;
  const int sl = gid % SL;
  for (int e0 = gid / SL; e0 < ceil_div(nel, 1); e0 += nthreads / SL) {
    const int e = min(e0, nel - 1);
    float s = 0.f;
    for (int p0 = sl; p0 < a.n_parts; p0 += 8 * SL) {
      float v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int p = p0 + u * SL;
        v[u] = p < a.n_parts ? a.part[(size_t)p * a.part_stride + e] : 0.f;
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) s += v[u];
    }
#pragma unroll
    for (int o = 1; o < SL; o <<= 1) s += __shfl_xor(s, o);
    if (sl != 0 || e0 >= nel) continue;
    if (e < HK) {
      if (!bad && e / a.K < a.H) a.W1[e] = a.W1[e] - a.lr * s;
    } else if (e < HK + HP) {
      const int n = e - HK;
      if (!bad && n < a.H) a.b1[n] = a.b1[n] - a.lr * s;
    } else if (e < HK + 2 * HP) {
      const int n = e - HK - HP;
      if (!bad && n < a.H) a.w2[n] = a.w2[n] - a.lr * s;
    } else if (e == HK + 2 * HP) {
      a.loss_out[0] = bad ? __builtin_nanf("") : s * a.invB;
    } else {
      if (!bad) a.b2[0] = a.b2[0] - a.lr * s;
    }
  }
  zero_ranges(a.zero, gid, nthreads);
}

// Rows whose sorted entries span several chunks: one workgroup per row.
// Wave w adds the partials of chunks cs+1+w, cs+5+w, ... (wave 0 also the
// open piece of the start chunk cs); the four wave sums are then added in
// wave order, so the result never depends on scheduling.
__host__ __device__ inline size_t segfix_lds_floats(int Hp, int K, int wmax) {
  return (size_t)Hp * K + (size_t)(kWavesPerBlock + 1) * wmax * Hp;
}

template <int WMAX, int HP>
__global__ __launch_bounds__(kBlock) void k_step_segfix(UpdArgs a) {
  extern __shared__ uint32_t lds[];
  const int t = threadIdx.x, lane = t & (kWave - 1), w = t / kWave;
  const uint32_t cnt = *a.long_count;
  if (blockIdx.x >= cnt || *reinterpret_cast<volatile uint32_t*>(a.flag)) return;
  float* w1s = reinterpret_cast<float*>(lds);
  float* red = w1s + (size_t)HP * a.K;  // [waves][WMAX][HP]
  float* sb = red + kWavesPerBlock * WMAX * HP;
  stage_w1<HP>(a, w1s);
  constexpr int U = 32 / WMAX;
  for (uint32_t li = blockIdx.x; li < cnt; li += gridDim.x) {
    const int cs = a.long_list[li];
    const int32_t key = a.sk[(size_t)cs * a.ch + a.ch - 1];
    const int ce = cs + seg_count_fwd(a.sk, a.N, cs, key, a.ch);
    float S[WMAX];
#pragma unroll
    for (int j = 0; j < WMAX; ++j) {
      const float* src = a.seg_part + ((size_t)cs * 2 + 1) * a.seg_stride;
      S[j] = (w == 0 && j < a.win && lane < HP) ? src[j * HP + lane] : 0.f;
    }
    for (int y0 = cs + 1 + w; y0 <= ce; y0 += U * kWavesPerBlock) {
      float v[U][WMAX];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int y = y0 + u * kWavesPerBlock;
        const float* src = a.seg_part + ((size_t)y * 2) * a.seg_stride;
#pragma unroll
        for (int j = 0; j < WMAX; ++j)
          v[u][j] = (y <= ce && j < a.win && lane < HP) ? src[j * HP + lane] : 0.f;
      }
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int j = 0; j < WMAX; ++j) S[j] += v[u][j];
    }
    __syncthreads();  // previous row done; w1s staged
#pragma unroll
    for (int j = 0; j < WMAX; ++j)
      if (lane < HP) red[(w * WMAX + j) * HP + lane] = S[j];
    __syncthreads();
    if (w == 0) {
      for (int j = 0; j < a.win; ++j) {
        if (lane < HP) {
          float s = red[(0 * WMAX + j) * HP + lane];
#pragma unroll
          for (int v = 1; v < kWavesPerBlock; ++v) s += red[(v * WMAX + j) * HP + lane];
          sb[j * HP + lane] = s;
        }
      }
      wave_lds_sync();
      const uint32_t mask = (a.win >= 32) ? 0xffffffffu : ((1u << a.win) - 1u);
      float* er = a.E + (size_t)key * a.d;
      for (int c0 = 0; c0 < a.d; c0 += kWave) {
        const int col = c0 + lane;
        const float g = row_grad_col<HP>(w1s, sb, mask, a.K, a.d, min(col, a.d - 1));
        if (col < a.d) er[col] = er[col] - a.lr * g;
      }
    }
  }
}

}  // namespace pg
