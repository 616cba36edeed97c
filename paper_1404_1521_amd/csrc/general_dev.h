// The general advanced-indexing op (§4.3: the increment the paper rewrites
// as a GPU kernel; the library form takes any table, any index vector, and
// either an increment or an assignment):
//   inc  table[idx[k]] += alpha * Y[k]  for every k,
//   set  table[idx[k]]  = Y[k]          for every k (the last k of a row wins),
// with float32, bfloat16 or binary16 tables (Y in the table's format), any
// row width up to kMaxD, int32 or int64 indices.  Both ops run on the sorted
// order of the entries (the radix sort of the step, stable by entry): inc
// accumulates each row's entries in float32 in entry order and rounds the
// row to the storage format once, so a row never loses small increments to
// per-entry rounding; set copies, for each row, the entry that ends its
// sorted segment.  Results do not depend on scheduling.
#pragma once
#include "common.h"
#include "launch.h"
#include "seg_dev.h"
#include "update_dev.h"

namespace pg {

// Storage formats.  bfloat16 is the upper half of a binary32; rounding a
// float to it keeps the upper half after adding half an ulp minus one plus
// the parity of the kept part (round to nearest, ties to even), and a NaN
// keeps a quiet NaN.  binary16 uses the hardware conversion, which rounds to
// nearest even.
struct BF16 {
  uint16_t bits;
};
struct F16 {
  uint16_t bits;
};

template <class T>
struct Elem;
template <>
struct Elem<float> {
  static __device__ __forceinline__ float get(float v) { return v; }
  static __device__ __forceinline__ float put(float v) { return v; }
};
template <>
struct Elem<BF16> {
  static __device__ __forceinline__ float get(BF16 v) {
    return __uint_as_float((uint32_t)v.bits << 16);
  }
  static __device__ __forceinline__ BF16 put(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return BF16{(uint16_t)((u >> 16) | 0x40u)};
    u += 0x7fffu + ((u >> 16) & 1u);
    return BF16{(uint16_t)(u >> 16)};
  }
};
template <>
struct Elem<F16> {
  static __device__ __forceinline__ float get(F16 v) {
    return (float)__builtin_bit_cast(_Float16, v.bits);
  }
  static __device__ __forceinline__ F16 put(float f) {
    return F16{__builtin_bit_cast(uint16_t, (_Float16)f)};
  }
};

// Same fields as SegArgs, with the table and Y in storage format T.
template <class T>
struct GenArgs {
  T* table;                 // [rows][d]
  const T* Y;               // [N][d]
  const int32_t* sk;        // sorted keys [N]
  const int32_t* sv;        // entry ids in sorted order [N]
  float* seg_part;          // [chunks][2][seg_stride] float32 partials
  int2* long_list;          // by chunk, as in SegArgs
  int32_t* seg_end;         // [rows]
  const uint32_t* flag;     // sticky error bits: nonzero voids the update
  int N, d, ch, seg_stride;
  float alpha;
  ZeroRanges zero;          // sort counters cleared by the apply launch
};

template <class T>
__device__ __forceinline__ float seg_load(const GenArgs<T>& a, size_t i) {
  return Elem<T>::get(a.Y[i]);
}
// a completed piece: the chunk's wave is the row's only writer in this launch
template <class T>
__device__ __forceinline__ void seg_add(const GenArgs<T>& a, size_t i, bool cok, float v) {
  if (cok) a.table[i] = Elem<T>::put(Elem<T>::get(a.table[i]) + v);
}

// Increment: one wave per chunk of CH sorted entries (seg_apply_rows), the
// extra workgroups clear the sort counters.
template <int CH, class T>
__global__ __launch_bounds__(kBlock) void k_gen_apply(GenArgs<T> a, int n_e) {
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  if ((int)blockIdx.x < n_e) {
    const int nchunks = ceil_div(a.N, CH);
    for (int c = blockIdx.x * kWavesPerBlock + w; c < nchunks; c += n_e * kWavesPerBlock)
      seg_apply_rows<CH, false>(a, c * CH, a.N, c, ChunkSink{});
    return;
  }
  zero_ranges(a.zero, (size_t)(blockIdx.x - n_e) * kBlock + threadIdx.x,
              (size_t)(gridDim.x - n_e) * kBlock);
}

// Fix-up of crossing segments (as k_segfix): light segments (at most
// kSegfixLight partials) by one wave, lane = column, partials added in
// chunk order; heavy ones by the whole workgroup, wave v adding a contiguous
// run of the partials in order and wave 0 adding the eight run sums in order.
template <class T>
__device__ int gen_fix_row_wave(const GenArgs<T>& a, int cs, int32_t key, int nchunks) {
  const int lane = lane_id();
  const int m = __builtin_amdgcn_readfirstlane(a.seg_end[key]) - cs + 1;
  if (m > kSegfixLight) return m;
  for (int c0 = 0; c0 < a.d; c0 += kWave) {
    const int col = c0 + lane;
    const bool cok = col < a.d;
    float x[kSegfixLight];
#pragma unroll
    for (int i = 0; i < kSegfixLight; ++i) {
      const size_t slot = i == 0 ? (size_t)cs * 2 + 1 : (size_t)(cs + i) * 2;
      x[i] = (i < m && cs + i < nchunks && cok) ? a.seg_part[slot * a.seg_stride + col] : 0.f;
    }
    float acc = 0.f;
#pragma unroll
    for (int i = 0; i < kSegfixLight; ++i) acc += x[i];
    seg_add(a, (size_t)key * a.d + col, cok, a.alpha * acc);
  }
  return m;
}

template <class T>
__device__ void gen_fix_row(const GenArgs<T>& a, int cs, int32_t key, int m, float* red) {
  const int t = threadIdx.x, lane = t & (kWave - 1);
  const int w = __builtin_amdgcn_readfirstlane(t / kWave);
  const int per = ceil_div(m, kSegfixWaves);
  const int i0 = w * per, i1 = min(m, i0 + per);
  constexpr int U = 8;
  for (int c0 = 0; c0 < a.d; c0 += kWave) {
    const int col = c0 + lane;
    const bool cok = col < a.d;
    float acc = 0.f;
    for (int i = i0; i < i1; i += U) {
      float x[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int j = i + u;
        const size_t slot = j == 0 ? (size_t)cs * 2 + 1 : (size_t)(cs + j) * 2;
        x[u] = (j < i1 && cok) ? a.seg_part[slot * a.seg_stride + col] : 0.f;
      }
#pragma unroll
      for (int u = 0; u < U; ++u) acc += x[u];
    }
    __syncthreads();  // red of the previous column block is no longer read
    red[w * kWave + lane] = acc;
    __syncthreads();
    if (w == 0) {
      float s = 0.f;
      for (int v = 0; v < kSegfixWaves; ++v) s += red[v * kWave + lane];
      seg_add(a, (size_t)key * a.d + col, cok, a.alpha * s);
    }
  }
}

template <class T>
__global__ __launch_bounds__(kSegfixThreads) void k_gen_segfix(GenArgs<T> a) {
  __shared__ float red[kSegfixWaves * kWave];
  __shared__ int heavy[kSegfixWaves][3];
  __shared__ int nheavy;
  if (*a.flag) return;
  const uint32_t cnt = (uint32_t)((a.N + a.ch - 1) / a.ch);
  const int t = threadIdx.x, lane = t & (kWave - 1);
  const int w = __builtin_amdgcn_readfirstlane(t / kWave);
  for (uint32_t base = 0; base + blockIdx.x < cnt; base += gridDim.x * kSegfixWaves) {
    if (t == 0) nheavy = 0;
    __syncthreads();
    const uint32_t li = base + (uint32_t)w * gridDim.x + blockIdx.x;
    if (li < cnt) {
      const int2 rec = a.long_list[li];
      if (rec.x >= 0) {
        const int m = gen_fix_row_wave(a, rec.x, rec.y, (int)cnt);
        if (m > kSegfixLight && lane == 0) {
          const int h = atomicAdd(&nheavy, 1);
          heavy[h][0] = rec.x;
          heavy[h][1] = rec.y;
          heavy[h][2] = m;
        }
      }
    }
    __syncthreads();
    const int nh = nheavy;
    for (int h = 0; h < nh; ++h) gen_fix_row(a, heavy[h][0], heavy[h][1], heavy[h][2], red);
    __syncthreads();
  }
}

// Assignment: one wave per 64 sorted entries; an entry whose successor has
// another key (or that is the last) ends its row's segment, so it is the
// row's last entry in index order, and its Y row is copied (lane = column).
// The extra workgroups clear the sort counters.
template <class T>
__global__ __launch_bounds__(kBlock) void k_gen_set(GenArgs<T> a, int n_e) {
  const int lane = lane_id();
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  if ((int)blockIdx.x >= n_e) {
    zero_ranges(a.zero, (size_t)(blockIdx.x - n_e) * kBlock + threadIdx.x,
                (size_t)(gridDim.x - n_e) * kBlock);
    return;
  }
  if (__builtin_amdgcn_readfirstlane(*a.flag) != 0u) return;
  const int ngroups = ceil_div(a.N, kWave);
  for (int gi = blockIdx.x * kWavesPerBlock + w; gi < ngroups; gi += n_e * kWavesPerBlock) {
    const int i = gi * kWave + lane;
    const bool act = i < a.N;
    const int32_t key = act ? a.sk[i] : -1;
    const int32_t nxt = (i + 1 < a.N) ? a.sk[i + 1] : -2;
    const int32_t ent = act ? a.sv[i] : 0;
    uint64_t tails = __ballot(act && key != nxt);
    while (tails) {
      const int src = __ffsll((unsigned long long)tails) - 1;
      tails &= tails - 1;
      const int32_t k = __builtin_amdgcn_readlane(key, src);
      const int32_t e = __builtin_amdgcn_readlane(ent, src);
      for (int c0 = 0; c0 < a.d; c0 += kWave) {
        const int col = c0 + lane;
        if (col < a.d) a.table[(size_t)k * a.d + col] = a.Y[(size_t)e * a.d + col];
      }
    }
  }
}

// int64 indices narrowed to int32 keys; an index outside [0, rows) raises
// kFlagBadId (the whole call is then void) and becomes key 0.
__global__ __launch_bounds__(kBlock) void k_keys_from_i64(const int64_t* __restrict__ idx, int N,
                                                          int rows, int32_t* __restrict__ keys,
                                                          uint32_t* flag) {
  bool bad = false;
  for (int i = blockIdx.x * kBlock + threadIdx.x; i < N; i += gridDim.x * kBlock) {
    const int64_t v = idx[i];
    const bool b = v < 0 || v >= (int64_t)rows;
    bad |= b;
    keys[i] = b ? 0 : (int32_t)v;
  }
  if (__ballot(bad) && lane_id() == 0) atomicOr(flag, kFlagBadId);
}

}  // namespace pg
