// Argument blocks and launchers shared by kernels.hip and the host API.
#pragma once
#include <tuple>
#include <utility>

#include "common.h"
#include "seg_dev.h"
#include "sort_dev.h"
#include "bsort_dev.h"

namespace pg {

// Where a kernel is launched: the stream and, when launches are being
// measured, a source of start/stop events that the runtime binds to the
// kernel's own dispatch (so they time the kernel, not the host enqueue).
struct Launch {
  hipStream_t s = nullptr;
  void* owner = nullptr;
  bool (*take)(void* owner, hipEvent_t* start, hipEvent_t* stop) = nullptr;
};

// Launches kernel k with the given arguments (converted to its parameter
// types); timed through hipExtLaunchKernel when L supplies events.
template <typename... KArgs, typename... Args>
inline hipError_t pg_launch(void (*k)(KArgs...), dim3 grid, dim3 block, uint32_t lds,
                            const Launch& L, Args&&... args) {
  std::tuple<KArgs...> tup{std::forward<Args>(args)...};
  void* argv[sizeof...(KArgs) > 0 ? sizeof...(KArgs) : 1];
  std::apply([&](auto&... x) {
    int i = 0;
    ((argv[i++] = static_cast<void*>(&x)), ...);
  }, tup);
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (L.take && L.take(L.owner, &e0, &e1))
    return hipExtLaunchKernel(reinterpret_cast<const void*>(k), grid, block, argv, lds, L.s, e0,
                              e1, 0);
  return hipLaunchKernel(reinterpret_cast<const void*>(k), grid, block, argv, lds, L.s);
}

struct FwdArgs {
  const float* E;
  const float* W1;
  const float* b1;
  const float* w2;
  const float* b2;
  const int32_t* windows;
  const int32_t* corrupt;
  float* G;          // [B*(win+1)][d] per-entry embedding gradients
  float* part;       // [workgroups][part_stride] dense partials
  uint32_t* flag;
  int V, d, win, H, Hp, K, c, B, N;
  // sort role: workgroups [0, n_sort) run the partitioned small sort
  int n_sort;
  SortPlan plan;
  SortBufs sb;
  int ntiles;        // ceil(B / 16)
  int tiles_per_wg;  // consecutive tiles per workgroup (pair of workgroups when split)
  int split;         // 16-wave kernel: 2 = two workgroups per tile group, each taking
                     // half of the backward; 1 = one
  int part_stride;   // floats per dense partial slot: Hp*K + 2*Hp + 2
  float invB;
};

// Three-contraction path (hidden layer above 64 units).
constexpr int kLgRows = 32;        // windows per forward workgroup
constexpr int kLgSlice = 1024;     // windows per dW1 slice
constexpr int kLgGRows = 64;       // windows per G workgroup

struct LargeArgs {
  const float* E;
  const float* W1;
  const float* b1;
  const float* w2;
  const float* b2;
  const int32_t* windows;
  const int32_t* corrupt;
  float* V;          // [B][3][H]
  float* vpart;      // [forward workgroups][2H + 2]: db1, dw2, loss, db2
  float* part;       // [slices][H][K] dW1 partials
  float* G;          // [B*(win+1)][d]
  float* scores;     // score-only mode: s(x) [B]
  uint32_t* flag;
  int V_rows, d, win, H, K, c, B;
  float invB;
};

// Zero ranges of the sort counters, cleared after their last use in a call.
struct ZeroRanges {
  uint32_t* p[3];
  size_t n[3];
};

// Dense SGD of a step: reduce the fused kernel's partials in slot order.
struct DenseArgs {
  float* W1;
  float* b1;
  float* w2;
  float* b2;
  float* loss_out;
  const float* part;   // dW1 partials: slot p at part + p * part_stride
  const float* vpart;  // db1, dw2, loss, db2 partials: slot p at vpart + p * vstride
  int n_parts, part_stride, n_vparts, vstride, H, Hp, K;
  // 2: the partial slots come in pairs (2q, 2q+1) that each hold half of the
  // dW1 output tiles (tile L = (k / 16) (Hp / 16) + n / 16 in slot 2q + L % 2)
  int split;
  float lr, invB;
};

// The next training step's bucketed sort, run as extra workgroups of this
// step's update (its tiles) and fix-up (its buckets) launches.  n_wg = 0:
// none.
struct NextSort {
  StepKeys kf;
  SortBufs sb;
  int N, ntiles, key_bits;
  int n_wg;
};

// One launch with roles: workgroups [0, n_e) update the table (sorted
// segments or atomics); the next ones run the dense SGD (if n_d > 0) and
// clear the sort counters; the last nx.n_wg rank the next step's sort tiles.
// The next step's ids in a multi-step call (or null): the dense workgroups
// of this step's update read one word per 64-byte line of them, so that the
// next fused kernel's first dependent loads find them in the memory-side
// cache shared by every XCD.  The values are not used (sink: a word written
// only if their sum takes one particular value, which keeps the loads).
struct Prefetch {
  const int32_t* p[2];
  int n[2];
  uint32_t* sink;
};

struct ApplyArgs {
  SegArgs s;
  int mode;  // 0 sorted segments, 1 atomic
  int n_e;
  int n_d;
  const int32_t* part_off;  // partition-wise update: partition starts (n_part + 1)
  int n_part;
  DenseArgs dn;
  ZeroRanges zero;
  NextSort nx;
  Prefetch pf;
};

struct ScoreArgs {
  const float* E;
  const float* W1;
  const float* b1;
  const float* w2;
  const float* b2;
  const int32_t* windows;
  float* scores;
  uint32_t* flag;
  int V, d, win, H, K, B;
};

struct GatherArgs {
  const float* E;
  const int32_t* windows;
  const int32_t* corrupt;
  float* X;
  float* Xc;
  uint32_t* flag;
  int V, d, win, B;
};

hipError_t launch_step_fwdbwd(const FwdArgs& a, int NT, int cpw, int grid, size_t lds,
                              const Launch& L);
// 16-wave fused kernel for the compile-time shapes: fwdbwd8_shape() gives the
// shape id (0: not covered), fwdbwd8_lds_bytes() its LDS.  Workgroups with
// more than one tile take form kF8MultiForm (2: tile pairs, tiles_per_wg
// even; 1: software-pipelined single tiles).
int fwdbwd8_shape(int d, int win, int NT);
size_t fwdbwd8_lds_bytes(int shape, int tiles_per_wg);
constexpr int kF8MultiForm = 2;
// From this many tiles per workgroup the d 64 shape takes the role-specialised
// form (form 3), whose three-stage pipeline fills and drains over two phases.
constexpr int kF8WsMinTiles = 8;  // at 4 (B = 16,384) tile pairs were 1 us faster
constexpr int kF8WsThreads = 12 * kWave;  // its workgroup: 12 waves
constexpr int kF8Waves = 16;
constexpr int kF8Threads = kF8Waves * kWave;  // 1024
constexpr int kF8MaxWorkgroups = 256;         // one workgroup per CU
hipError_t launch_step_fwdbwd8(const FwdArgs& a, int shape, int grid, size_t lds,
                               const Launch& L);
// First sort launch (whole small sort, or pass-0 tile counts) and, for
// multi-tile plans, every later pass.
hipError_t launch_sort_step(const StepKeys& kf, int N, const SortPlan& plan, const SortBufs& sb,
                            const Launch& L);
hipError_t launch_sort_idx(const IdxKeys& kf, int N, const SortPlan& plan, const SortBufs& sb,
                           const Launch& L);
hipError_t launch_sort_i64(const I64Keys& kf, int N, const SortPlan& plan, const SortBufs& sb,
                           const Launch& L);
hipError_t launch_apply_step(const ApplyArgs& a, const StepKeys& kf, int grid, const Launch& L);
hipError_t launch_apply_idx(const ApplyArgs& a, const IdxKeys& kf, int grid, const Launch& L);
hipError_t launch_segfix(const SegArgs& a, int grid, const Launch& L);
// the update of a training step with nx.n_wg extra workgroups for the next
// step's sort tiles, and its fix-up with the buckets of that sort
hipError_t launch_apply_step_next(const ApplyArgs& a, const StepKeys& kf, int grid,
                                  const Launch& L);
hipError_t launch_segfix_step(const SegArgs& a, const NextSort& nx, int n_fix, const Launch& L);

// The general advanced-indexing op (any storage format, increment or
// assignment) over a sorted entry list; pointers as in SegArgs, the table
// and Y in format `dtype` (0 float32, 1 bfloat16, 2 binary16).
struct GenCall {
  void* table;
  const void* Y;
  const int32_t* sk;
  const int32_t* sv;
  float* seg_part;
  int2* long_list;
  int32_t* seg_end;
  const uint32_t* flag;
  int N, d, ch, seg_stride;
  int rg;  // entries per range of the apply (the fix-up's slots)
  float alpha;
  ZeroRanges zero;
  int dtype;  // 0 float32, 1 bfloat16, 2 binary16
  int op;     // 0 increment, 1 assignment
  int n_e;    // workgroups of the apply / assignment role
  int n_z;    // workgroups clearing the sort counters
  // a partitioned (small) list: partition starts; its increments take one
  // launch, one workgroup per partition, and no fix-up
  const int32_t* part_off;
  bool partitioned;
  int n_part;
  // a 16-bit increment whose rows are whole 32-bit words (d even, table and
  // Y 4-byte aligned): the packed walk, two rows per load and store
  bool packed;
  // bytes per word of the assignment's row copies (2, 4, 8 or 16): the
  // widest that divides a row and both pointers' alignment
  int set_word;
};
hipError_t launch_gen_update(const GenCall& c, const Launch& L);
hipError_t launch_gen_fix(const GenCall& c, int grid, const Launch& L);
hipError_t launch_keys_from_i64(const int64_t* idx, int N, int rows, int32_t* keys,
                                uint32_t* flag, const Launch& L);
hipError_t launch_apply_part(const ApplyArgs& a, int grid, const Launch& L);

hipError_t launch_check_idx(const int32_t* idx, int N, int rows, uint32_t* flag, const Launch& L);
hipError_t launch_score(const ScoreArgs& a, int NT, int cpw, const Launch& L);
hipError_t launch_gather(const GatherArgs& a, const Launch& L);
// three-contraction path: forward (or score only), dW1 partials, G rows
hipError_t launch_large_fwd(const LargeArgs& a, int score_only, const Launch& L);
hipError_t launch_large_dw1(const LargeArgs& a, const Launch& L);
hipError_t launch_large_g(const LargeArgs& a, const Launch& L);

// LDS of the fused kernel, in floats: W1 [Hp][K+4], split-K partials
// [4 waves][3][NT][64] f4, V [3][16][Hp+1], per-wave dense sums [4][2Hp+2],
// two tile id tables [2][16][32].
__host__ __device__ inline size_t fwdbwd_lds_floats(int Hp, int K) {
  return (size_t)Hp * (K + 4) + (size_t)kWavesPerBlock * 3 * (Hp / 16) * kWave * 4 +
         (size_t)3 * kTileRows * (Hp + 1) + (size_t)kWavesPerBlock * (2 * Hp + 2) +
         (size_t)2 * kTileRows * (kMaxWin + 1);
}

// Launch-shape constants shared with the host.
constexpr int kDenseSlices = 8;  // slot groups of the dense reduction

}  // namespace pg
