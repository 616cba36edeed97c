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
// per-entry rounding (a segment that crosses chunks is finished by the
// float32 fix-up, k_segfix, through this format's row access); set copies,
// for each row, the entry that ends its sorted segment.  Results do not
// depend on scheduling.
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
  float* seg_part;          // [ranges][2][seg_stride] float32 partials
  int2* long_list;          // by range, as in SegArgs
  int32_t* seg_end;         // [rows]
  const uint32_t* flag;     // sticky error bits: nonzero voids the update
  const uint32_t* flag2;    // same word as flag (the general op has one sort of its own)
  int N, d, ch, seg_stride;
  int rg;                   // entries per range of the apply (the fix-up's slots)
  float alpha;
  ZeroRanges zero;          // sort counters cleared by the apply launch
  const int32_t* part_off;  // partition starts of a partitioned sort
  // a row update is a load and a store: deferred past the walk (seg_add_rows)
  static constexpr bool kDeferred = true;
  static constexpr int kPre = 16;  // old rows loaded before the walk (the first block)
  struct Pre {
    T old[kPre];
  };
  static constexpr bool kPacked = false;
  using elem = T;
};

// The same arguments for a 16-bit format whose rows are whole 32-bit words
// (d even, table and Y 4-byte aligned): the walk reads and writes two rows
// per word (seg_walk_packed).
template <class T>
struct GenArgsP : GenArgs<T> {
  static_assert(sizeof(T) == 2, "two elements per word");
  static constexpr bool kPacked = true;
};

template <class T>
__device__ __forceinline__ float seg_load(const GenArgs<T>& a, size_t i) {
  return Elem<T>::get(a.Y[i]);
}
// A segment's sum v (alpha applied) added to element i by the row's only
// writer: one rounding to the storage format.
template <class T>
__device__ __forceinline__ void seg_close(const GenArgs<T>& a, size_t i, float v) {
  a.table[i] = Elem<T>::put(Elem<T>::get(a.table[i]) + v);
}

// The completed pieces of a chunk, after its walk: v[r] holds the sum of the
// piece ending at row r for every bit r of `complete`.  The chunk's wave is
// the only writer of these rows in this launch.  The old values of the first
// kPre rows are loaded before the walk, beside the entries' rows
// (seg_prefetch_rows), so that round trip overlaps the entries'; rows past
// kPre are updated kPre at a time with their loads in flight together, so a
// chunk of many short pieces (the Zipf tail) never waits one round trip per
// piece.  (bfloat16, 327,680 entries in 32-entry chunks: apply 21.8 -> 19.5
// us with the first 16 old rows loaded early.)
__host__ __device__ constexpr uint32_t low_bits(int n) { return n >= 32 ? ~0u : (1u << n) - 1u; }
// Rows per block: kPre, or the whole chunk when it is shorter (blocks of 32
// measured slower: apply 19.5 -> 20.6 us at 32-entry chunks, for the
// occupancy they cost).
__host__ __device__ constexpr int pre_rows(int ch) { return ch < 16 ? ch : 16; }
static_assert(pre_rows(64) <= 16, "a block's mask fits 32 bits");
template <int CH, class T>
__device__ __forceinline__ void seg_prefetch_rows(const GenArgs<T>& a, const ChunkInfo& ci,
                                                  uint64_t complete, int colc,
                                                  typename GenArgs<T>::Pre& pre) {
  constexpr int RB = pre_rows(CH);
  uint32_t cw = (uint32_t)complete & low_bits(RB);
  asm volatile("" : "+s"(cw));
#pragma unroll
  for (int u = 0; u < RB; ++u)
    if ((cw >> u) & 1u)
      pre.old[u] = a.table[(size_t)__builtin_amdgcn_readlane(ci.key, u) * a.d + colc];
}

template <int CH, class T>
__device__ void seg_add_rows(const GenArgs<T>& a, const ChunkInfo& ci, uint64_t complete,
                             const float (&v)[CH], int colc, bool cok,
                             const typename GenArgs<T>::Pre& pre) {
  constexpr int RB = pre_rows(CH);
#pragma unroll
  for (int r0 = 0; r0 < CH; r0 += RB) {
    uint32_t cw = (uint32_t)(complete >> r0) & low_bits(RB);
    asm volatile("" : "+s"(cw));
    if (cw == 0u) continue;
    T old[RB];
#pragma unroll
    for (int u = 0; u < RB; ++u)
      if ((cw >> u) & 1u)
        old[u] = r0 == 0 ? pre.old[u]
                         : a.table[(size_t)__builtin_amdgcn_readlane(ci.key, r0 + u) * a.d + colc];
#pragma unroll
    for (int u = 0; u < RB; ++u)
      if (((cw >> u) & 1u) && cok)
        a.table[(size_t)__builtin_amdgcn_readlane(ci.key, r0 + u) * a.d + colc] =
            Elem<T>::put(Elem<T>::get(old[u]) + v[r0 + u]);
  }
}

// Packed walk.  For pair i of a chunk (rows 2i, 2i + 1), lanes < 32 read
// row 2i and lanes >= 32 row 2i + 1, one 32-bit word (two columns) per lane:
// lane l holds columns 2w, 2w + 1 of its row, w = c0 / 2 + l % 32.  Swapping
// the upper half-wave of the first-column values with the lower half-wave of
// the second-column values (v_permlane32_swap) leaves row 2i in one register
// and row 2i + 1 in the other, lane l on column 2w + l / 32 of both; the same
// swap turns two such rows back into words.  The old values of every row the
// chunk completes are loaded beside the entries' rows, one word per lane per
// pair, so a chunk takes one round of loads and writes each row as its piece
// closes: half the registers per row in flight of the one-row walk, and half
// the load and store instructions.  Same sums, same order, same rounding
// (once per row) as seg_apply_rows.  (bfloat16, 327,680 entries into
// 100000 x 64 in 32-entry chunks: apply 19.6 -> 18.1 us; 16- and 64-entry
// chunks measured 21.2 and 23.4 us.)
__device__ __forceinline__ void swap_halves(float& x, float& y) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(y), false,
                                                  false);
  x = __uint_as_float(r[0]);
  y = __uint_as_float(r[1]);
}
template <class T>
__device__ __forceinline__ void unpack2(uint32_t w, float& x, float& y) {
  x = Elem<T>::get(T{(uint16_t)(w & 0xffffu)});
  y = Elem<T>::get(T{(uint16_t)(w >> 16)});
}
template <class T>
__device__ __forceinline__ uint32_t pack2(float x, float y) {
  return (uint32_t)Elem<T>::put(x).bits | ((uint32_t)Elem<T>::put(y).bits << 16);
}

template <int CH, class A>
__device__ void seg_walk_packed(const A& a, const ChunkInfo& ci, uint64_t tails, uint64_t complete,
                                int first_tail, bool starts_long, const ChunkSink& sink) {
  using T = typename A::elem;
  constexpr int NP = CH / 2;
  const int lane = lane_id(), h = lane >> 5;
  const int nact = ci.nact;
  const uint32_t* Yw = reinterpret_cast<const uint32_t*>(a.Y);
  uint32_t* Tw = reinterpret_cast<uint32_t*>(a.table);
  const int dw = a.d >> 1;  // words per row
  for (int c0 = 0; c0 < a.d; c0 += kWave) {
    const int w = (c0 >> 1) + (lane & 31);
    const bool wok = w < dw;
    const int wc = wok ? w : dw - 1;  // lanes past the row end read its last word
    // every pair's entries (rows past the chunk's end read entry 0's row,
    // which no piece uses) and the old words of its complete rows
    uint32_t y[NP], o[NP];
#pragma unroll
    for (int i = 0; i < NP; ++i) {
      const int e0 = __builtin_amdgcn_readlane(ci.ent, 2 * i);
      const int e1 = __builtin_amdgcn_readlane(ci.ent, 2 * i + 1);
      y[i] = Yw[(size_t)(h ? e1 : e0) * dw + wc];
    }
#pragma unroll
    for (int i = 0; i < NP; ++i) {
      uint32_t c2 = (uint32_t)(complete >> (2 * i)) & 3u;
      asm volatile("" : "+s"(c2));
      o[i] = 0u;
      if (c2 != 0u) {
        const int k0 = __builtin_amdgcn_readlane(ci.key, 2 * i);
        const int k1 = __builtin_amdgcn_readlane(ci.key, 2 * i + 1);
        if ((c2 >> h) & 1u) o[i] = Tw[(size_t)(h ? k1 : k0) * dw + wc];
      }
    }
    float acc = 0.f, first_sum = 0.f, last_sum = 0.f;
#pragma unroll
    for (int r0 = 0; r0 < CH; r0 += 8) {
      uint32_t tw = (uint32_t)(tails >> r0) & 0xffu, cw = (uint32_t)(complete >> r0) & 0xffu;
      int ft = first_tail - r0, lt = nact - 1 - r0;
      asm volatile("" : "+s"(tw), "+s"(cw), "+s"(ft), "+s"(lt));
      float v[8];
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        unpack2<T>(y[r0 / 2 + p], v[2 * p], v[2 * p + 1]);
        swap_halves(v[2 * p], v[2 * p + 1]);
      }
      if (tw == 0u) {  // no piece ends in these rows
#pragma unroll
        for (int u = 0; u < 8; ++u) acc += v[u];
        continue;
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        acc += v[u];
        if ((tw >> u) & 1u) {
          if (u == ft) first_sum = acc;
          if (u == lt) last_sum = acc;
          if ((cw >> u) & 1u) v[u] = a.alpha * acc;
          acc = 0.f;
        }
      }
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        const uint32_t c2 = (cw >> (2 * p)) & 3u;
        if (c2 == 0u) continue;
        float x, z;
        unpack2<T>(o[r0 / 2 + p], x, z);
        swap_halves(x, z);  // old values of rows r0 + 2p (x) and r0 + 2p + 1 (z)
        x += v[2 * p];
        z += v[2 * p + 1];
        swap_halves(x, z);  // back to words: columns 2w, 2w + 1 of this lane's row
        const int k0 = __builtin_amdgcn_readlane(ci.key, r0 + 2 * p);
        const int k1 = __builtin_amdgcn_readlane(ci.key, r0 + 2 * p + 1);
        if (((c2 >> h) & 1u) && wok) Tw[(size_t)(h ? k1 : k0) * dw + w] = pack2<T>(x, z);
      }
    }
    if (wok) {
      const int col = 2 * w + h;
      if (ci.cont_first) sink.first[col] = first_sum;
      if (starts_long) sink.last[col] = last_sum;
    }
  }
}

// Increment: one wave per chunk of CH sorted entries (seg_apply_rows), the
// extra workgroups clear the sort counters.  A: GenArgs<T> or GenArgsP<T>.
// The packed walk fits 7 waves per SIMD without spilling (72 registers; the
// compiler alone picks 76 and 6 waves): 10,240 chunk waves of the 327,680-
// entry bfloat16 list then take about 1.4 rounds instead of 1.7 (apply 18.5
// -> 17.7 us, means of four alternating pairs; 8 waves spill and take 22.5
// us).
template <int CH, class A>
__global__ __launch_bounds__(kBlock, A::kPacked ? 7 : 1) void k_gen_apply(A a, int n_e) {
  __shared__ float F[kWavesPerBlock][kMaxD];
  __shared__ float Lp[kWavesPerBlock][kMaxD];
  __shared__ int meta[kWavesPerBlock][5];
  if ((int)blockIdx.x < n_e) {
    // (the error words are tested beside each chunk's keys)
    const int nranges = ceil_div(a.N, CH * kWavesPerBlock);
    for (int r = blockIdx.x; r < nranges; r += n_e)
      seg_apply_range<CH, kWavesPerBlock>(a, r, F, Lp, meta);
    return;
  }
  zero_ranges(a.zero, (size_t)(blockIdx.x - n_e) * kBlock + threadIdx.x,
              (size_t)(gridDim.x - n_e) * kBlock);
}

// Increment after a partitioned sort (N <= kSmallSortN): workgroup p applies
// partition p, whose segments never leave it, so no fix-up follows; the
// extra workgroups clear nothing (the small sort keeps no counters).
template <class A>
__global__ __launch_bounds__(kPartApplyThreads) void k_gen_apply_part(A a) {
  __shared__ float F[kPartApplyWaves][kMaxD];
  __shared__ float Lp[kPartApplyWaves][kMaxD];
  __shared__ int meta[kPartApplyWaves][5];
  // (the error words are tested beside each chunk's keys)
  const int p = blockIdx.x;
  seg_apply_partition<kPartApplyWaves>(a, a.part_off[p], a.part_off[p + 1], F, Lp, meta);
}

// Row access of the fix-up (seg_fix_slot_wave / seg_fix_row, launched as
// k_segfix<GenArgs<T>>): four consecutive columns at element i, n of them
// inside the row, converted to and from float.  The fix-up is the row's only
// writer.
template <class T>
__device__ __forceinline__ f4 seg_row4(const GenArgs<T>& a, size_t i, int n) {
  f4 r = kZero4;
#pragma unroll
  for (int k = 0; k < 4; ++k)
    if (k < n) r[k] = Elem<T>::get(a.table[i + k]);
  return r;
}
template <class T>
__device__ __forceinline__ void seg_put4(const GenArgs<T>& a, size_t i, int n, f4 v) {
#pragma unroll
  for (int k = 0; k < 4; ++k)
    if (k < n) a.table[i + k] = Elem<T>::put(v[k]);
}
template <class T>
__device__ __forceinline__ void seg_add4(const GenArgs<T>& a, size_t i, int n, f4 v) {
  seg_put4(a, i, n, seg_row4(a, i, n) + v);
}

// Assignment: one wave per 64 sorted entries; an entry whose successor has
// another key (or that is the last) ends its row's segment, so it is the
// row's last entry in index order, and its Y row is copied.  The error words
// are read beside the keys.  Each such entry's (entry, row) goes to the
// wave's LDS slots by its rank among them, and the rows are copied as words
// of W bytes (the widest that divides a row and the pointers' alignment):
// word f of the group's copy is word f % dw of the (f / dw)-th row, dw words
// per row, 8 or 16 words per lane in flight at once, so a group of short
// rows takes one round of loads however many rows it ends (binary16, d 64:
// four rows per load).  The extra workgroups clear the sort counters.
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));  // a 16-byte word
template <class W>
constexpr int set_words() { return sizeof(W) >= 16 ? 8 : 16; }  // per lane, in flight
template <class T, class W>
__global__ __launch_bounds__(kBlock) void k_gen_set(GenArgs<T> a, int n_e) {
  constexpr int kSetWords = set_words<W>();
  __shared__ int2 tl[kWavesPerBlock][kWave];  // (entry, row) of the group's row ends, by rank
  const int lane = lane_id();
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  if ((int)blockIdx.x >= n_e) {
    zero_ranges(a.zero, (size_t)(blockIdx.x - n_e) * kBlock + threadIdx.x,
                (size_t)(gridDim.x - n_e) * kBlock);
    return;
  }
  const W* Yw = reinterpret_cast<const W*>(a.Y);
  W* Tw = reinterpret_cast<W*>(a.table);
  const int dw = (int)((size_t)a.d * sizeof(T) / sizeof(W));
  const int ngroups = ceil_div(a.N, kWave);
  for (int gi = blockIdx.x * kWavesPerBlock + w; gi < ngroups; gi += n_e * kWavesPerBlock) {
    const int i = gi * kWave + lane;
    const bool act = i < a.N;
    const uint32_t flag = *a.flag | *a.flag2;
    const int32_t key = act ? a.sk[i] : -1;
    const int32_t nxt = (i + 1 < a.N) ? a.sk[i + 1] : -2;
    const int32_t ent = act ? a.sv[i] : 0;
    const bool tail = act && key != nxt;
    const uint64_t tails = __ballot(tail);
    if (__builtin_amdgcn_readfirstlane(flag) != 0u) return;  // a bad id voids the call
    const int rank = __builtin_amdgcn_mbcnt_hi((uint32_t)(tails >> 32),
                                               __builtin_amdgcn_mbcnt_lo((uint32_t)tails, 0u));
    if (tail) tl[w][rank] = make_int2(ent, key);
    __builtin_amdgcn_wave_barrier();
    const int total = __popcll((unsigned long long)tails) * dw;  // words to copy
    for (int f0 = 0; f0 < total; f0 += kSetWords * kWave) {
      W v[kSetWords];
      size_t dst[kSetWords];
#pragma unroll
      for (int u = 0; u < kSetWords; ++u) {
        const int f = f0 + u * kWave + lane;
        dst[u] = ~(size_t)0;
        if (f < total) {
          const int j = f / dw, x = f - j * dw;
          const int2 r = tl[w][j];
          v[u] = Yw[(size_t)r.x * dw + x];
          dst[u] = (size_t)r.y * dw + x;
        }
      }
#pragma unroll
      for (int u = 0; u < kSetWords; ++u)
        if (dst[u] != ~(size_t)0) Tw[dst[u]] = v[u];
    }
    __builtin_amdgcn_wave_barrier();  // the slots are rewritten by the next group
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
