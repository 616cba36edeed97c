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
#include "fwdbwd_dev.h"
#include "update_dev.h"
#include "aux_dev.h"

namespace pg {

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

__global__ __launch_bounds__(kBlock) void k_sort_up(int N, SortPlan plan, SortBufs sb, int p) {
  extern __shared__ uint32_t lds[];
  sort_up_tile(N, plan, sb, p, blockIdx.x, lds);
}

// All radix passes after the first-pass counts: up(p) for p >= 1, down(p).
template <class KeyFn>
static void launch_sort_passes(const KeyFn& kf, int N, const SortPlan& plan, const SortBufs& sb,
                               hipStream_t s) {
  for (int p = 0; p < plan.passes; ++p) {
    if (p > 0)
      hipLaunchKernelGGL(k_sort_up, dim3(plan.ntiles), dim3(kBlock), kMaxBins * 4, s, N, plan, sb,
                         p);
    hipLaunchKernelGGL((k_sort_down<KeyFn>), dim3(plan.ntiles), dim3(kBlock), kDownLdsWords * 4,
                       s, kf, N, plan, sb, p);
  }
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

hipError_t launch_sort_passes_step(const StepKeys& kf, int N, const SortPlan& plan,
                                   const SortBufs& sb, hipStream_t s) {
  launch_sort_passes(kf, N, plan, sb, s);
  return launch_err();
}

template <int WMAX, int HP>
static void launch_update_t(const UpdArgs& a, int grid, hipStream_t s) {
  hipLaunchKernelGGL((k_step_update<WMAX, HP>), dim3(grid), dim3(kBlock),
                     update_lds_floats(HP, a.K, a.d, WMAX) * 4, s, a);
}

template <int WMAX, int HP>
static void launch_segfix_t(const UpdArgs& a, hipStream_t s) {
  hipLaunchKernelGGL((k_step_segfix<WMAX, HP>), dim3(kSegfixBlocks), dim3(kBlock),
                     segfix_lds_floats(HP, a.K, WMAX) * 4, s, a);
}

#define PG_BY_SHAPE(FN, ...)                                      \
  do {                                                            \
    if (a.win <= 8) {                                             \
      if (a.Hp == 16) FN<8, 16>(__VA_ARGS__);                     \
      else if (a.Hp == 32) FN<8, 32>(__VA_ARGS__);                \
      else FN<8, 64>(__VA_ARGS__);                                \
    } else if (a.win <= 16) {                                     \
      if (a.Hp == 16) FN<16, 16>(__VA_ARGS__);                    \
      else if (a.Hp == 32) FN<16, 32>(__VA_ARGS__);               \
      else FN<16, 64>(__VA_ARGS__);                               \
    } else {                                                      \
      if (a.Hp == 16) FN<32, 16>(__VA_ARGS__);                    \
      else if (a.Hp == 32) FN<32, 32>(__VA_ARGS__);               \
      else FN<32, 64>(__VA_ARGS__);                               \
    }                                                             \
  } while (0)

hipError_t launch_step_update(const UpdArgs& a, int grid, hipStream_t s) {
  PG_BY_SHAPE(launch_update_t, a, grid, s);
  return launch_err();
}

hipError_t launch_step_segfix(const UpdArgs& a, hipStream_t s) {
  PG_BY_SHAPE(launch_segfix_t, a, s);
  return launch_err();
}
#undef PG_BY_SHAPE

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
  if (!plan.small) launch_sort_passes(kf, a.N, plan, sb, s);
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


}  // namespace pg
