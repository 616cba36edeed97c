// Shared definitions of the HIP library: limits, workspace layout, launch
// argument blocks and small wave64 helpers.  gfx950 (CDNA4) only.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pg {

typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;
constexpr int kBlock = 256;             // threads per workgroup of every kernel
constexpr int kWavesPerBlock = kBlock / kWave;
constexpr int kTileRows = 16;           // windows per MFMA tile (16x16x4 f32)
constexpr int kMaxK = 512;              // win*d handled by the fused step kernel
constexpr int kMaxHp = 64;              // hidden units, padded to a multiple of 16
constexpr int kMaxNT = kMaxHp / 16;
constexpr int kMaxWin = 31;
constexpr int kMaxD = 256;
constexpr int kMaxLdsBytes = 160 * 1024;  // LDS per workgroup on gfx950

// Radix sort of (row id, entry) pairs.
constexpr int kSortIPT = 16;                       // keys per thread in a tile
constexpr int kSortTile = kBlock * kSortIPT;       // 4096 keys per tile
constexpr int kMaxDigitBits = 9;
constexpr int kMaxBins = 1 << kMaxDigitBits;
constexpr int kMaxPasses = 4;                      // 31-bit keys at most
constexpr int kSmallSortN = 8192;                  // single-workgroup LDS sort up to this N

// Sticky device error bits.
constexpr uint32_t kFlagBadId = 1u;
constexpr uint32_t kFlagInternal = 2u;  // a sort position fell outside [0, N): a library bug

struct SortPlan {
  int passes;               // 0 when N <= 1 (nothing to order)
  int shift[kMaxPasses];
  int bits[kMaxPasses];
  int ntiles;               // multi-tile path: tiles of kSortTile keys
  int small;                // 1: single-workgroup LDS sort
  int val_bits;             // small path packs (key << val_bits) | entry in 32 bits
};

// Device workspace owned by a context (all sizes fixed at init).
struct Workspace {
  // sort
  int32_t* keys[2];         // ping-pong sorted keys [max_entries]
  int32_t* vals[2];         // ping-pong entry ids   [max_entries]
  uint32_t* totals;         // [kMaxPasses][kMaxBins] global digit counts
  uint32_t* counts;         // [kMaxPasses][kMaxBins][max_tiles] per-tile digit counts
  uint32_t* gcounts;        // [kMaxPasses][kMaxBins][max_groups] per-16-tile digit counts
  // step
  float* G;                 // [max_batch*(win+1)][d] per-entry embedding gradients
  float* part;              // [max_parts][part_stride] dense-gradient partials
  // segmented update
  float* seg_part;          // [max_chunks][2][seg_stride] partial sums of long segments
  int32_t* long_list;       // [max_chunks] start chunks of segments spanning chunks
  uint32_t* long_count;     // number of entries in long_list
  int32_t* seg_end;         // [max(V, max_rows)] end chunk of a long segment, by row id
  uint32_t* flag;           // sticky error bits
  float* scratch_loss;      // loss slot used when the caller passes no loss pointer
};

__host__ __device__ inline int ceil_div(int a, int b) { return (a + b - 1) / b; }

// ---------------------------------------------------------------- wave helpers
__device__ inline int lane_id() { return __lane_id(); }

__device__ inline uint64_t lanemask_lt() {
  const int l = __lane_id();
  return l == 0 ? 0ull : (~0ull >> (64 - l));
}

// Lanes of the wave whose `digit` (low `bits` bits significant) equals this
// lane's, restricted to `active`.
__device__ inline uint64_t match_digit(uint32_t digit, int bits, uint64_t active) {
  uint64_t m = active;
  for (int b = 0; b < bits; ++b) {
    const bool set = (digit >> b) & 1u;
    const uint64_t bal = __ballot(set);
    m &= set ? bal : ~bal;
  }
  return m;
}

__device__ inline float readlane_f(float v, int lane) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), lane));
}

__device__ __forceinline__ f4 ld4(const float* p) { return *reinterpret_cast<const f4*>(p); }
__device__ __forceinline__ void st4(float* p, f4 v) { *reinterpret_cast<f4*>(p) = v; }
constexpr f4 kZero4 = {0.f, 0.f, 0.f, 0.f};

// Orders this wave's LDS writes before its later LDS reads by other lanes.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

}  // namespace pg
