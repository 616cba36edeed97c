// HIP kernels (gfx950) of the Polyglot window-ranking SGD step.
//
// One step on the device (sorted mode):
//
//   sort            the step's (row id, entry) pairs, grouped by row id in
//                   entry order.  Small batches: a partitioned sort run by
//                   extra workgroups of the fused kernel below.  Large
//                   batches: k_sort_first + k_sort_up / k_sort_down radix
//                   passes on a side stream (they depend only on the ids; in
//                   a multi-step call the next step's sort runs while the
//                   current step computes);
//   k_step_fwdbwd   per 16-window tile: gather the embedding rows straight
//                   into MFMA operands, z = W1 x + b1 and the corrupted-centre
//                   z~ (16x16x4 f32 MFMA, split-K over 4 waves), tanh, scores,
//                   hinge, dz and dz~, the per-entry gradient rows G of the
//                   embedding and this workgroup's share of dW1/db1/dw2/loss;
//   k_apply         workgroups [0, n_e): for every sorted row id, the sum of
//                   its G rows is subtracted (times lr) from its E row
//                   (or one float atomic per element in the atomic variant);
//                   the other workgroups reduce the dense partials in slot
//                   order, apply SGD to W1/b1/w2/b2, write the mean loss and
//                   clear the sort counters for the next call;
//   k_segfix        rows whose sorted entries span several chunks (Zipf
//                   heavy rows): their chunk partials in a fixed order.
//
// Model (§1 Introduction; SENNA-style window ranker):
//   s(x) = w2 . tanh(W1 x + b1) + b2,  loss = mean max(0, 1 - s(x) + s(x~)).
// The embedding update is the advanced-indexing increment of §4.2 (Table 1)
// that §4.3 parallelises; polyglot_scatter_add runs the same sort, k_apply
// and k_segfix on the caller's table, indices and rows.
//
// Global loads are issued in batches whose values are used only after the
// whole batch is in flight: a use right after each load would serialise one
// memory round trip per element.
#include "common.h"
#include "launch.h"
#include "seg_dev.h"
#include "sort_dev.h"
#include "fwdbwd_dev.h"
#include "fwdbwd8_dev.h"
#include "large_dev.h"
#include "update_dev.h"
#include "aux_dev.h"
#include "general_dev.h"

namespace pg {

// Two workgroups per CU when the shape's registers allow it without spills.
// D and WIN (0: runtime) fix the embedding width and window of the common
// shapes at compile time.
template <int NT, int CPW, int D, int WIN>
__global__ __launch_bounds__(kBlock, (NT == 1 || (NT == 2 && CPW <= 5)) ? 2 : 1) void k_step_fwdbwd(FwdArgs a) {
  extern __shared__ float lds_f[];
  if ((int)blockIdx.x < a.n_sort) {  // small batches: the step's sort, partition blockIdx.x
    const StepKeys kf = step_keys(a.windows, a.corrupt, a.win, a.V);
    part_sort<kBlock>(kf, a.N, a.plan, blockIdx.x, a.sb.keys[a.plan.passes & 1],
                      a.sb.vals[a.plan.passes & 1], a.sb.part_off, a.flag,
                      reinterpret_cast<uint32_t*>(lds_f));
    return;
  }
  fwdbwd_wg<NT, CPW, D, WIN>(a, blockIdx.x - a.n_sort, lds_f);
}

// The same step for the compile-time shapes, 16 waves per workgroup (the
// sort role of small batches too); FORM: 0 single tile, 1 pipelined tiles, 2
// tile pairs; NH = 2: two workgroups per tile, each taking half of the
// backward.
template <int D, int WIN, int NT, int FORM, int NH>
__global__ __launch_bounds__(kF8Threads, 1) void k_step_fwdbwd8(FwdArgs a) {
  extern __shared__ float lds_f[];
  if ((int)blockIdx.x < a.n_sort) {
    const StepKeys kf = step_keys(a.windows, a.corrupt, a.win, a.V);
    part_sort<kF8Threads>(kf, a.N, a.plan, blockIdx.x, a.sb.keys[a.plan.passes & 1],
                          a.sb.vals[a.plan.passes & 1], a.sb.part_off, a.flag,
                          reinterpret_cast<uint32_t*>(lds_f));
    return;
  }
  fwdbwd8_wg<D, WIN, NT, FORM, NH>(a, blockIdx.x - a.n_sort, lds_f);
}

// Role-specialised form for workgroups with many tiles (12 waves; never
// with the sort role, which only small batches take).
template <int D, int WIN>
__global__ __launch_bounds__(kF8WsThreads, 1) void k_step_fwdbwd8_ws(FwdArgs a) {
  extern __shared__ float lds_f[];
  fwdbwd8_ws<D, WIN>(a, blockIdx.x, lds_f);
}

// =============================================================== sort

// Partitioned sort of a small list, partition blockIdx.x.
template <class KeyFn>
__global__ __launch_bounds__(kPartSortThreads) void k_sort_part(KeyFn kf, int N, SortPlan plan,
                                                                SortBufs sb) {
  extern __shared__ uint32_t lds[];
  part_sort<kPartSortThreads>(kf, N, plan, blockIdx.x, sb.keys[plan.passes & 1],
                              sb.vals[plan.passes & 1], sb.part_off, sb.flag, lds,
                              sb.fresh_status);
}

// Digit totals of a large list.
template <class KeyFn>
__global__ __launch_bounds__(kBlock) void k_os_hist(KeyFn kf, int N, SortPlan plan, SortBufs sb) {
  extern __shared__ uint32_t lds[];
  os_hist(kf, N, plan, sb, blockIdx.x, lds);
}

// One radix pass over the tiles of a large list.
template <int R, class KeyFn>
__global__ __launch_bounds__(kOsThreads) void k_os_pass(KeyFn kf, int N, SortPlan plan,
                                                        SortBufs sb, int p) {
  extern __shared__ uint32_t lds[];
  os_pass<R>(kf, N, plan, sb, p, lds);
}

template <class KeyFn>
static hipError_t launch_tiled_sort(const KeyFn& kf, int N, const SortPlan& plan,
                                    const SortBufs& sb, const Launch& L) {
  hipError_t e = pg_launch(k_os_hist<KeyFn>, dim3(ceil_div(N, kBlock * kOsHistIpt)), dim3(kBlock),
                           kOsHistLdsWords * 4, L, kf, N, plan, sb);
  for (int p = 0; p < plan.passes && e == hipSuccess; ++p) {
    if (plan.tile_keys == kSortTileKeysShort)
      e = pg_launch(k_os_pass<kSortTileKeysShort / kOsThreads, KeyFn>, dim3(plan.ntiles),
                    dim3(kOsThreads), kOsPassLdsWords * 4, L, kf, N, plan, sb, p);
    else
      e = pg_launch(k_os_pass<kSortTileKeys / kOsThreads, KeyFn>, dim3(plan.ntiles),
                    dim3(kOsThreads), kOsPassLdsWords * 4, L, kf, N, plan, sb, p);
  }
  return e;
}

// Bucketed sort of a mid-size list: tiles by bucket, then buckets.
template <class KeyFn>
__global__ __launch_bounds__(kBkThreads) void k_bk_tiles(KeyFn kf, int N, int ntiles, SortBufs sb) {
  extern __shared__ uint32_t lds[];
  bk_tiles<kBkThreads>(kf, N, ntiles, sb, blockIdx.x, lds);
}

__global__ __launch_bounds__(kBkSortThreads) void k_bk_buckets(int N, int ntiles, int key_bits,
                                                               SortBufs sb) {
  extern __shared__ uint32_t lds[];
  bk_buckets(N, ntiles, key_bits, sb, blockIdx.x, lds);
}


template <class KeyFn>
static hipError_t launch_sort(const KeyFn& kf, int N, const SortPlan& plan, const SortBufs& sb,
                              const Launch& L) {
  if (plan.small)
    return pg_launch(k_sort_part<KeyFn>, dim3(1 << plan.part_bits), dim3(kPartSortThreads),
                     part_sort_lds_words(kPartSortThreads) * 4, L, kf, N, plan, sb);
  if (plan.bucket) {
    hipError_t e = pg_launch(k_bk_tiles<KeyFn>, dim3(plan.ntiles), dim3(kBkThreads),
                             bk_tiles_lds_words(kBkThreads) * 4, L, kf, N, plan.ntiles, sb);
    if (e == hipSuccess)
      e = pg_launch(k_bk_buckets, dim3(bk_grid(N)), dim3(kBkSortThreads), kBkLdsWords * 4, L, N,
                    plan.ntiles, plan.key_bits, sb);
    return e;
  }
  return launch_tiled_sort(kf, N, plan, sb, L);
}

// =============================================================== launchers

template <int NT>
static hipError_t launch_fwdbwd_nt(const FwdArgs& a, int cpw, int grid, size_t lds,
                                   const Launch& L) {
  if (cpw <= 2) return pg_launch(k_step_fwdbwd<NT, 2, 0, 0>, dim3(grid), dim3(kBlock), lds, L, a);
  if (cpw <= 5) return pg_launch(k_step_fwdbwd<NT, 5, 0, 0>, dim3(grid), dim3(kBlock), lds, L, a);
  return pg_launch(k_step_fwdbwd<NT, 8, 0, 0>, dim3(grid), dim3(kBlock), lds, L, a);
}

int fwdbwd8_shape(int d, int win, int NT) {
  if (d == 64 && win == 5 && NT == 2) return 1;  // the Polyglot-scale model, H <= 32
  if (d == 16 && win == 5 && NT == 1) return 2;  // the small model, H <= 16
  return 0;
}

size_t fwdbwd8_lds_bytes(int shape, int tiles_per_wg) {
  if (shape == 1 && tiles_per_wg >= kF8WsMinTiles) return F8WsShape<64, 5>::kLds * sizeof(float);  // n_sort is 0 there
  constexpr int TP = kF8MultiForm == 2 ? 2 : 1;  // tiles per phase of the multi-tile form
  if (tiles_per_wg > 1)
    return (shape == 1 ? F8Shape<64, 5, 2, TP>::kLds : F8Shape<16, 5, 1, TP>::kLds) * sizeof(float);
  return (shape == 1 ? F8Shape<64, 5, 2, 1>::kLds : F8Shape<16, 5, 1, 1>::kLds) * sizeof(float);
}

hipError_t launch_step_fwdbwd8(const FwdArgs& a, int shape, int grid, size_t lds,
                               const Launch& L) {
  const dim3 g(grid), b(kF8Threads);
  constexpr int MF = kF8MultiForm;
  if (shape == 1)
    return a.tiles_per_wg >= kF8WsMinTiles && a.n_sort == 0
               ? pg_launch(k_step_fwdbwd8_ws<64, 5>, g, dim3(kF8WsThreads), lds, L, a)
           : a.tiles_per_wg > 1 ? pg_launch(k_step_fwdbwd8<64, 5, 2, MF, 1>, g, b, lds, L, a)
           : a.split == 2     ? pg_launch(k_step_fwdbwd8<64, 5, 2, 0, 2>, g, b, lds, L, a)
                              : pg_launch(k_step_fwdbwd8<64, 5, 2, 0, 1>, g, b, lds, L, a);
  return a.tiles_per_wg > 1 ? pg_launch(k_step_fwdbwd8<16, 5, 1, MF, 1>, g, b, lds, L, a)
                            : pg_launch(k_step_fwdbwd8<16, 5, 1, 0, 1>, g, b, lds, L, a);
}

hipError_t launch_step_fwdbwd(const FwdArgs& a, int NT, int cpw, int grid, size_t lds,
                              const Launch& L) {
  if (NT == 1) return launch_fwdbwd_nt<1>(a, cpw, grid, lds, L);
  if (NT == 2) return launch_fwdbwd_nt<2>(a, cpw, grid, lds, L);
  return launch_fwdbwd_nt<4>(a, cpw, grid, lds, L);
}

hipError_t launch_sort_step(const StepKeys& kf, int N, const SortPlan& plan, const SortBufs& sb,
                            const Launch& L) {
  return launch_sort(kf, N, plan, sb, L);
}

hipError_t launch_sort_idx(const IdxKeys& kf, int N, const SortPlan& plan, const SortBufs& sb,
                           const Launch& L) {
  return launch_sort(kf, N, plan, sb, L);
}

hipError_t launch_sort_i64(const I64Keys& kf, int N, const SortPlan& plan, const SortBufs& sb,
                           const Launch& L) {
  return launch_sort(kf, N, plan, sb, L);
}

template <class KeyFn>
static hipError_t launch_apply(const ApplyArgs& a, const KeyFn& kf, int grid, const Launch& L) {
  if (a.s.ch == 16) return pg_launch(k_apply<16, KeyFn>, dim3(grid), dim3(kBlock), 0, L, a, kf);
  return pg_launch(k_apply<32, KeyFn>, dim3(grid), dim3(kBlock), 0, L, a, kf);
}

hipError_t launch_apply_step(const ApplyArgs& a, const StepKeys& kf, int grid, const Launch& L) {
  return launch_apply(a, kf, grid, L);
}

hipError_t launch_apply_step_next(const ApplyArgs& a, const StepKeys& kf, int grid,
                                  const Launch& L) {
  const uint32_t lds = a.nx.n_wg ? bk_tiles_lds_words(kBlock) * 4 : 0;
  const int g = grid + a.nx.n_wg;
  if (a.s.ch == 16) return pg_launch(k_apply<16, StepKeys>, dim3(g), dim3(kBlock), lds, L, a, kf);
  return pg_launch(k_apply<32, StepKeys>, dim3(g), dim3(kBlock), lds, L, a, kf);
}

hipError_t launch_segfix_step(const SegArgs& a, const NextSort& nx, int n_fix, const Launch& L) {
  const uint32_t lds = nx.n_wg ? kBkLdsWords * 4 : 0;
  return pg_launch(k_segfix_step, dim3(n_fix + nx.n_wg), dim3(kSegfixThreads), lds, L, a, nx,
                   n_fix);
}

hipError_t launch_apply_idx(const ApplyArgs& a, const IdxKeys& kf, int grid, const Launch& L) {
  return launch_apply(a, kf, grid, L);
}

hipError_t launch_apply_part(const ApplyArgs& a, int grid, const Launch& L) {
  static_assert(kPartTinyN <= kPartShortN, "the 8-wave form takes 32-entry chunks");
  if (part_apply_threads(a.s.N) == kPartShortThreads)
    return pg_launch(k_apply_part<32, kPartShortThreads>, dim3(grid), dim3(kPartShortThreads), 0, L,
                     a);
  if (a.s.N <= kPartShortN)
    return pg_launch(k_apply_part<32, kPartApplyThreads>, dim3(grid), dim3(kPartApplyThreads), 0, L,
                     a);
  return pg_launch(k_apply_part<kPartApplyChunk, kPartApplyThreads>, dim3(grid),
                   dim3(kPartApplyThreads), 0, L, a);
}

hipError_t launch_segfix(const SegArgs& a, int grid, const Launch& L) {
  return pg_launch(k_segfix<SegArgs>, dim3(grid), dim3(kSegfixThreads), 0, L, a);
}

template <class T>
static GenArgs<T> gen_args(const GenCall& c) {
  GenArgs<T> a{};
  a.table = static_cast<T*>(c.table);
  a.Y = static_cast<const T*>(c.Y);
  a.sk = c.sk;
  a.sv = c.sv;
  a.seg_part = c.seg_part;
  a.long_list = c.long_list;
  a.seg_end = c.seg_end;
  a.flag = c.flag;
  a.flag2 = c.flag;
  a.N = c.N;
  a.d = c.d;
  a.ch = c.ch;
  a.rg = c.rg;
  a.seg_stride = c.seg_stride;
  a.alpha = c.alpha;
  a.zero = c.zero;
  a.part_off = c.part_off;
  return a;
}

template <class A>
static hipError_t launch_gen_inc(const GenCall& c, const A& a, const Launch& L) {
  if (c.partitioned)
    return pg_launch(k_gen_apply_part<A>, dim3(c.n_part), dim3(kPartApplyThreads), 0, L, a);
  const dim3 grid(c.n_e + c.n_z), block(kBlock);
  if (c.ch == 16) return pg_launch(k_gen_apply<16, A>, grid, block, 0, L, a, c.n_e);
  return pg_launch(k_gen_apply<32, A>, grid, block, 0, L, a, c.n_e);
}

template <class T>
static hipError_t launch_gen_update_t(const GenCall& c, const Launch& L) {
  const dim3 grid(c.n_e + c.n_z), block(kBlock);
  if (c.op == 1) {  // copies in the widest words the rows and pointers allow
    const GenArgs<T> a = gen_args<T>(c);
    if (c.set_word == 16) return pg_launch(k_gen_set<T, u32x4>, grid, block, 0, L, a, c.n_e);
    if (c.set_word == 8) return pg_launch(k_gen_set<T, uint64_t>, grid, block, 0, L, a, c.n_e);
    if (c.set_word == 4) return pg_launch(k_gen_set<T, uint32_t>, grid, block, 0, L, a, c.n_e);
    if constexpr (sizeof(T) == 2) return pg_launch(k_gen_set<T, uint16_t>, grid, block, 0, L, a, c.n_e);
    return hipErrorInvalidValue;  // a float32 row is whole 4-byte words
  }
  if constexpr (sizeof(T) == 2)
    if (c.packed) return launch_gen_inc(c, GenArgsP<T>{gen_args<T>(c)}, L);
  return launch_gen_inc(c, gen_args<T>(c), L);
}

hipError_t launch_gen_update(const GenCall& c, const Launch& L) {
  if (c.dtype == 1) return launch_gen_update_t<BF16>(c, L);
  if (c.dtype == 2) return launch_gen_update_t<F16>(c, L);
  return launch_gen_update_t<float>(c, L);
}

template <class T>
static hipError_t launch_gen_fix_t(const GenCall& c, int grid, const Launch& L) {
  if (c.partitioned) return hipSuccess;  // the partitions completed every segment
  return pg_launch(k_segfix<GenArgs<T>>, dim3(grid), dim3(kSegfixThreads), 0, L, gen_args<T>(c));
}

hipError_t launch_gen_fix(const GenCall& c, int grid, const Launch& L) {
  if (c.dtype == 1) return launch_gen_fix_t<BF16>(c, grid, L);
  if (c.dtype == 2) return launch_gen_fix_t<F16>(c, grid, L);
  return launch_gen_fix_t<float>(c, grid, L);
}

hipError_t launch_keys_from_i64(const int64_t* idx, int N, int rows, int32_t* keys,
                                uint32_t* flag, const Launch& L) {
  const int g = std::min(std::max(ceil_div(N, kBlock), 1), 1024);
  return pg_launch(k_keys_from_i64, dim3(g), dim3(kBlock), 0, L, idx, N, rows, keys, flag);
}

hipError_t launch_check_idx(const int32_t* idx, int N, int rows, uint32_t* flag, const Launch& L) {
  const int g = std::min(std::max(ceil_div(N, kBlock), 1), 1024);
  return pg_launch(k_check_idx, dim3(g), dim3(kBlock), 0, L, idx, N, rows, flag);
}

template <int NT>
static hipError_t launch_score_nt(const ScoreArgs& a, int cpw, int grid, size_t lds,
                                  const Launch& L) {
  if (cpw <= 2) return pg_launch(k_score<NT, 2>, dim3(grid), dim3(kBlock), lds, L, a);
  if (cpw <= 5) return pg_launch(k_score<NT, 5>, dim3(grid), dim3(kBlock), lds, L, a);
  return pg_launch(k_score<NT, 8>, dim3(grid), dim3(kBlock), lds, L, a);
}

hipError_t launch_score(const ScoreArgs& a, int NT, int cpw, const Launch& L) {
  const int grid = ceil_div(a.B, kTileRows);
  const size_t lds = (kTileRows * (kMaxWin + 1)) * 4 + kWavesPerBlock * kMaxNT * kWave * 16;
  if (NT == 1) return launch_score_nt<1>(a, cpw, grid, lds, L);
  if (NT == 2) return launch_score_nt<2>(a, cpw, grid, lds, L);
  return launch_score_nt<4>(a, cpw, grid, lds, L);
}

hipError_t launch_large_fwd(const LargeArgs& a, int score_only, const Launch& L) {
  const dim3 grid(ceil_div(a.B, kLgRows));
  switch (a.H / 64) {
    case 2: return pg_launch(k_large_fwd<2>, grid, dim3(2 * kWave), 0, L, a, score_only);
    case 3: return pg_launch(k_large_fwd<3>, grid, dim3(3 * kWave), 0, L, a, score_only);
    default: return pg_launch(k_large_fwd<4>, grid, dim3(4 * kWave), 0, L, a, score_only);
  }
}

hipError_t launch_large_dw1(const LargeArgs& a, const Launch& L) {
  // 128-column blocks when they stay inside one window position
  if (a.d % 128 == 0)
    return pg_launch(k_large_dw1<128>, dim3(a.H / 64, a.K / 128, ceil_div(a.B, kLgSlice)),
                     dim3(kBlock), 0, L, a);
  return pg_launch(k_large_dw1<64>, dim3(a.H / 64, a.K / 64, ceil_div(a.B, kLgSlice)), dim3(kBlock),
                   0, L, a);
}

hipError_t launch_large_g(const LargeArgs& a, const Launch& L) {
  const dim3 grid(ceil_div(a.B, kLgGRows), a.win + 1);
  switch (a.d / 16) {
    case 4: return pg_launch(k_large_g<4>, grid, dim3(kBlock), 0, L, a);
    case 8: return pg_launch(k_large_g<8>, grid, dim3(kBlock), 0, L, a);
    case 12: return pg_launch(k_large_g<12>, grid, dim3(kBlock), 0, L, a);
    default: return pg_launch(k_large_g<16>, grid, dim3(kBlock), 0, L, a);
  }
}

hipError_t launch_gather(const GatherArgs& a, const Launch& L) {
  const size_t total = (size_t)a.B * (a.win + 1) * (a.d / 4);
  const size_t want = (total + kBlock - 1) / kBlock;
  const int grid = (int)(want < 8192 ? (want > 0 ? want : 1) : 8192);
  return pg_launch(k_gather, dim3(grid), dim3(kBlock), 0, L, a);
}

}  // namespace pg
