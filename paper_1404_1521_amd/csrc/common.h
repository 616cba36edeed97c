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
constexpr int kMaxHp = 64;              // hidden units of the fused step kernel, padded to 16
constexpr int kMaxLargeH = 256;         // hidden units of the three-contraction path (multiple of 64)
constexpr int kMaxNT = kMaxHp / 16;
constexpr int kMaxWin = 31;
constexpr int kMaxD = 256;
constexpr int kMaxLdsBytes = 160 * 1024;  // LDS per workgroup on gfx950

// Radix sort of (row id, entry) pairs.
constexpr int kSortTileKeys = 4096;                // multi-tile sort: keys per tile (long lists)
constexpr int kSortTileKeysShort = 1024;           // ... and for lists up to kShortTileLimit
constexpr int kShortTileLimit = 131072;
constexpr int kMaxDigitBits = 9;
constexpr int kMaxBins = 1 << kMaxDigitBits;
constexpr int kMaxPasses = 4;                      // 31-bit keys at most
constexpr int kSmallSortN = 8192;                  // partitioned LDS sort up to this N
constexpr int kSmallDigitBits = 7;                 // widest digit of the partitioned sort's passes
constexpr int kSmallBins = 1 << kSmallDigitBits;

// Sticky device error bits.
constexpr uint32_t kFlagBadId = 1u;
constexpr uint32_t kFlagInternal = 2u;  // a sort position fell outside [0, N): a library bug
// Status words written on the device (the values of POLYGLOT_OK and POLYGLOT_EID).
constexpr int32_t kStatusOk = 0;
constexpr int32_t kStatusBadId = -5;

struct SortPlan {
  int passes;               // 0 when N <= 1 (nothing to order)
  int shift[kMaxPasses];
  int bits[kMaxPasses];
  int ntiles;               // multi-tile path: tiles of tile_keys keys
  int tile_keys;            // kSortTileKeysShort or kSortTileKeys
  int small;                // 1: partitioned sort (one launch, 2^part_bits workgroups)
  int val_bits;             // small path packs (key >> part_bits) << val_bits | entry
  int part_bits;            // small path: partitions by the low key bits
  int bucket;               // 1: bucketed sort (mid-size lists; two launches, passes = 1)
  int key_bits;             // bits of the key range
};

// Device workspace owned by a context (all sizes fixed at init).
struct Workspace {
  // sort
  // Two sort sets, so that the sort of the next step can run while the
  // current step reads its own: set q uses keys/vals[2q] and [2q+1] as
  // ping-pong buffers and its own accumulated digit counters.
  int32_t* keys[4];         // sorted keys [max_entries]
  int32_t* vals[4];         // entry ids   [max_entries]
  uint32_t* totals[2];      // [kMaxPasses][kMaxBins] global digit counts
  uint32_t* status[2];      // [kMaxPasses][max_tiles][kMaxBins] look-back words
  uint32_t* tile_ctr[2];    // [kMaxPasses] tile id counters
  int32_t* part_off[2];     // [2^kPartBits + 1] partitioned sort: where each partition starts
  // step
  float* G;                 // [max_batch*(win+1)][d] per-entry embedding gradients
  float* part;              // dense-gradient partials: [max_parts][part_stride], or
                            // [slices][H][K] dW1 partials of the three-contraction path
  float* vpart;             // three-contraction path: [forward workgroups][2H + 2]
  float* vbuf;              // three-contraction path: [max_batch][3][H] dz + dz~, dz, dz~
  // segmented update
  float* seg_part;          // [ranges][2][seg_stride] partial sums of long segments (sized
                            // by chunks: at least the ranges of any call)
  int2* long_list;          // [ranges] by range: (range, row) if a segment crossing
                            // ranges starts there, else (-1, 0)
  int32_t* seg_end;         // [max(V, max_rows)] end range of a long segment, by row id
  uint32_t* flag;           // sticky error bits [3]: word 0 raised by every launch except a
                            // training step's side-stream sort, word 1 + q by the side-stream
                            // sort of sort set q (read only by that set's update)
  float* scratch_loss;      // loss slot used when the caller passes no loss pointer
  uint32_t* pf_sink;        // [1] written only by an unlikely prefetch sum (see Prefetch)
  int32_t* idx32;           // [max_scatter] int64 indices narrowed to int32 keys
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

// Inclusive prefix sum over the 64 lanes of a wave with DPP moves: shifts by
// 1, 2, 4, 8 inside each row of 16 lanes, then the last lane of row 0 (2) is
// broadcast into row 1 (3), and lane 31 into rows 2 and 3.  Out-of-row
// sources and masked rows contribute 0.
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t v) {
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x111, 0xf, 0xf, false);  // row_shr:1
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x112, 0xf, 0xf, false);  // row_shr:2
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x114, 0xf, 0xf, false);  // row_shr:4
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x118, 0xf, 0xf, false);  // row_shr:8
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x142, 0xa, 0xf, false);  // row_bcast:15
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x143, 0xc, 0xf, false);  // row_bcast:31
  return v;
}

__device__ inline float readlane_f(float v, int lane) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), lane));
}

// tanh of the hidden layer, from two identities of the function:
//  |x| < 0.4   the Maclaurin series of tanh, odd terms through x^13 (the
//              coefficients are 2^2n (2^2n - 1) B_2n / (2n)!, B the Bernoulli
//              numbers); the first omitted term is below 2^-27 of tanh(x);
//  |x| >= 0.4  tanh|x| = 1 - 2 / (1 + e^(2|x|)) with the hardware base-2
//              exponential and reciprocal (a few ulp; e^(2|x|) overflowing
//              to infinity gives exactly 1), sign restored.
// Pre-activations of this model are mostly far below 0.4, where the series
// has no cancellation.
__device__ __forceinline__ float tanh_fast(float x) {
  const float ax = __builtin_fabsf(x);
  const float x2 = x * x;
  float p = 21844.f / 6081075.f;
  p = p * x2 - 1382.f / 155925.f;
  p = p * x2 + 62.f / 2835.f;
  p = p * x2 - 17.f / 315.f;
  p = p * x2 + 2.f / 15.f;
  p = p * x2 - 1.f / 3.f;
  const float small = x + x * x2 * p;
  const float e = __builtin_amdgcn_exp2f(2.8853900817779268f * ax);  // e^(2|x|) = 2^(2|x| log2 e)
  const float big = 1.f - 2.f * __builtin_amdgcn_rcpf(1.f + e);
  return ax < 0.4f ? small : __builtin_copysignf(big, x);
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
