// Argument blocks and launchers shared by kernels.hip and the host API.
#pragma once
#include "common.h"
#include "sort_dev.h"

namespace pg {

struct FwdArgs {
  const float* E;
  const float* W1;
  const float* b1;
  const float* w2;
  const float* b2;
  const int32_t* windows;
  const int32_t* corrupt;
  float* dzz;
  float* part;
  float* w1snap;
  uint32_t* long_count;  // cleared here for the update launch of the same step
  uint32_t* flag;
  int V, d, win, H, Hp, K, c, B, N;
  int ntiles;        // ceil(B / 16)
  int tiles_per_wg;  // consecutive tiles per fwd/bwd workgroup
  int part_stride;   // floats per dense partial slot: Hp*K + 2*Hp + 2
  float invB;
  // sort role (workgroups [0, n_sort))
  int n_sort;
  int sort_small;
  SortPlan plan;
  SortBufs sb;
};

// Zero ranges of the sort counters, cleared after their last use in a call.
struct ZeroRanges {
  uint32_t* p[3];
  size_t n[3];
};

struct UpdArgs {
  float* E;
  float* W1;
  float* b1;
  float* w2;
  float* b2;
  float* loss_out;
  const float* dzz;
  const float* part;
  const float* w1snap;
  const int32_t* sk;  // sorted keys (sorted mode)
  const int32_t* sv;  // sorted entry ids
  const int32_t* windows;
  const int32_t* corrupt;
  float* seg_part;
  int32_t* long_list;
  uint32_t* long_count;
  uint32_t* flag;
  ZeroRanges zero;
  int V, d, win, H, Hp, K, c, B, N;
  int mode;  // 0 sorted, 1 atomic
  int ch;    // sorted entries per chunk (one wave)
  int n_e;   // embedding-role workgroups
  int n_d;   // dense-role workgroups
  int n_parts;
  int part_stride;
  int seg_stride;
  float lr, invB;
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

struct ScatArgs {
  float* table;
  const int32_t* idx;
  const float* Y;
  const int32_t* sk;
  const int32_t* sv;
  float* seg_part;
  int32_t* long_list;
  uint32_t* long_count;
  uint32_t* flag;
  ZeroRanges zero;
  int rows, d, N;
  int ch;  // sorted entries per chunk (one wave)
  int n_e, n_z;
  int seg_stride;
  float alpha;
};

hipError_t launch_step_fwdbwd(const FwdArgs& a, int NT, int cpw, int grid, size_t lds,
                              hipStream_t s);
hipError_t launch_sort_passes_step(const StepKeys& kf, int N, const SortPlan& plan,
                                   const SortBufs& sb, hipStream_t s);
hipError_t launch_step_update(const UpdArgs& a, int grid, hipStream_t s);
hipError_t launch_step_segfix(const UpdArgs& a, hipStream_t s);
hipError_t launch_score(const ScoreArgs& a, int NT, int cpw, hipStream_t s);
hipError_t launch_gather(const GatherArgs& a, hipStream_t s);
hipError_t launch_scatter_sorted(const ScatArgs& a, const SortPlan& plan, const SortBufs& sb,
                                 hipStream_t s);
hipError_t launch_scatter_atomic(const ScatArgs& a, hipStream_t s);

// Launch-shape constants shared with the host.
constexpr int kSegfixBlocks = 64;
constexpr int kFlushGroup = 16;  // completed pieces buffered before their rows are written
constexpr int kAtomicChunk = 8;  // entries per wave in the atomic embedding update
constexpr int kDenseSlices = 8;  // lanes that share one element of the dense reduction

}  // namespace pg
