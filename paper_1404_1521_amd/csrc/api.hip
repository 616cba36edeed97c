// Host side of the C ABI declared in include/polyglot.h: argument checks,
// workspace, launch sequencing, graph replay of multi-step calls, per-kernel
// event timing.
#include "polyglot.h"

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <mutex>
#include <string>
#include <utility>
#include <vector>

#include "launch.h"
#include "seg_dev.h"

using namespace pg;

namespace {

struct GraphKey {
  const void* p[7];
  const void* losses;
  int S, B;
  float lr;
  hipStream_t stream;
  bool operator==(const GraphKey& o) const {
    return std::memcmp(p, o.p, sizeof(p)) == 0 && losses == o.losses && S == o.S && B == o.B &&
           std::memcmp(&lr, &o.lr, sizeof(float)) == 0 && stream == o.stream;
  }
};

}  // namespace

struct polyglot_ctx {
  polyglot_config cfg{};
  hipStream_t stream = nullptr;
  // a step's sort depends only on its ids: it runs on a second stream,
  // forked from `stream` and joined back before the table update.  In a
  // multi-step call the sort of step s+1 (sort set (s+1)&1) runs while step s
  // computes.
  hipStream_t side = nullptr;
  hipEvent_t ev_fork = nullptr, ev_sorted[2] = {nullptr, nullptr},
             ev_done[2] = {nullptr, nullptr};
  int device = 0;
  int Hp = 0, NT = 0, K = 0, c = 0, cpw = 0;
  bool large = false;  // hidden layer above 64 units: the three-contraction path
  int max_entries = 0, max_tiles = 0, max_parts = 0, max_chunks = 0;
  int seg_stride = 0, part_stride = 0;
  Workspace ws{};
  std::vector<void*> allocs;
  std::string err;
  bool have_sorted = false;
  int last_N = 0, last_passes = 0, last_set = 0;
  hipGraphExec_t gexec = nullptr;
  GraphKey gkey{};
  bool gvalid = false;
  // per-kernel timing
  bool timing = false;
  bool capturing = false;
  std::vector<hipEvent_t> ev_pool;
  std::vector<std::pair<int, std::pair<hipEvent_t, hipEvent_t>>> ev_marks;
};

namespace {

int fail(polyglot_ctx* ctx, int code, const std::string& msg) {
  if (ctx) ctx->err = msg;
  return code;
}

int hip_fail(polyglot_ctx* ctx, hipError_t e, const char* what) {
  return fail(ctx, POLYGLOT_EHIP, std::string(what) + ": " + hipGetErrorString(e));
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int bits_for(uint32_t n) {  // smallest b >= 1 with n <= 2^b
  int b = 1;
  while (b < 31 && (1u << b) < n) ++b;
  return b;
}

// Radix plan: the small (partitioned) sort ranks the key bits above the
// partition bits; the multi-tile sort ranks all key bits.
SortPlan make_plan(int key_range, int N) {
  SortPlan pl{};
  const int kb = bits_for((uint32_t)key_range);
  pl.val_bits = bits_for((uint32_t)std::max(N, 2));
  pl.part_bits = std::min(kPartBits, kb);
  pl.small = (N <= kSmallSortN && (kb - pl.part_bits) + pl.val_bits <= 32) ? 1 : 0;
  if (!pl.small) pl.part_bits = 0;
  pl.key_bits = kb;
  pl.bucket = (!pl.small && N <= kBkMaxN && kb <= kBkMaxKeyBits) ? 1 : 0;
  if (pl.bucket) {  // grouped into a second buffer by two launches
    pl.passes = 1;
    pl.tile_keys = kBkTileKeys;
    pl.ntiles = bk_tiles(N);
    return pl;
  }
  const int rb = kb - pl.part_bits;  // bits the radix passes rank
  const int digit = pl.small ? kSmallDigitBits : kMaxDigitBits;
  pl.passes = (rb + digit - 1) / digit;
  if (pl.passes > 0) {
    const int base = rb / pl.passes, rem = rb % pl.passes;
    int sh = 0;
    for (int p = 0; p < pl.passes; ++p) {
      pl.bits[p] = base + (p < rem ? 1 : 0);
      pl.shift[p] = sh;
      sh += pl.bits[p];
    }
  }
  // short lists: smaller tiles, so a pass has more, shorter workgroups
  pl.tile_keys = N <= kShortTileLimit ? kSortTileKeysShort : kSortTileKeys;
  pl.ntiles = ceil_div(N, pl.tile_keys);
  return pl;
}

SortBufs sort_bufs(polyglot_ctx* ctx, int set) {
  SortBufs sb{};
  sb.keys[0] = ctx->ws.keys[2 * set];
  sb.keys[1] = ctx->ws.keys[2 * set + 1];
  sb.vals[0] = ctx->ws.vals[2 * set];
  sb.vals[1] = ctx->ws.vals[2 * set + 1];
  sb.totals = ctx->ws.totals[set];
  sb.status = ctx->ws.status[set];
  sb.tile_ctr = ctx->ws.tile_ctr[set];
  sb.part_off = ctx->ws.part_off[set];
  sb.max_tiles = ctx->max_tiles;
  sb.flag = ctx->ws.flag;
  return sb;
}

// The error word of a training step's side-stream sort into set `set`.  The
// sort of step s+1 runs while step s updates its parameters, so it raises a
// word of its own: step s's update reads word 0 and its own set's word, never
// the other set's.  polyglot_status reports all three words.
uint32_t* set_flag(polyglot_ctx* ctx, int set) { return ctx->ws.flag + 1 + set; }

// Counters a multi-tile sort accumulates atomically (the look-back words are
// cleared by the sort's histogram launch).
ZeroRanges sort_zero_ranges(polyglot_ctx* ctx, const SortPlan& plan, int set) {
  ZeroRanges z{};
  if (plan.small) return z;
  z.p[0] = ctx->ws.totals[set];
  z.n[0] = (size_t)kMaxPasses * kMaxBins;
  return z;
}

template <class T>
hipError_t alloc(polyglot_ctx* ctx, T** p, size_t count) {
  void* q = nullptr;
  hipError_t e = hipMalloc(&q, std::max<size_t>(count, 1) * sizeof(T));
  if (e == hipSuccess) {
    ctx->allocs.push_back(q);
    *p = static_cast<T*>(q);
  }
  return e;
}

void free_all(polyglot_ctx* ctx) {
  for (auto& m : ctx->ev_marks) {
    ctx->ev_pool.push_back(m.second.first);
    ctx->ev_pool.push_back(m.second.second);
  }
  ctx->ev_marks.clear();
  for (hipEvent_t ev : ctx->ev_pool) hipEventDestroy(ev);
  ctx->ev_pool.clear();
  if (ctx->gexec) hipGraphExecDestroy(ctx->gexec);
  ctx->gexec = nullptr;
  for (hipEvent_t* ev : {&ctx->ev_fork, &ctx->ev_sorted[0], &ctx->ev_sorted[1], &ctx->ev_done[0],
                         &ctx->ev_done[1]}) {
    if (*ev) hipEventDestroy(*ev);
    *ev = nullptr;
  }
  if (ctx->side) hipStreamDestroy(ctx->side);
  ctx->side = nullptr;
  for (void* q : ctx->allocs) hipFree(q);
  ctx->allocs.clear();
}

hipEvent_t take_event(polyglot_ctx* ctx) {
  if (!ctx->ev_pool.empty()) {
    hipEvent_t ev = ctx->ev_pool.back();
    ctx->ev_pool.pop_back();
    return ev;
  }
  hipEvent_t ev = nullptr;
  if (hipEventCreate(&ev) != hipSuccess) return nullptr;
  return ev;
}

// Launch parameters for kernel id `kid` on stream `st`.  When timing is on
// (and no graph is being captured) every launch made with it gets its own
// start/stop event pair, bound to the kernel's dispatch.
struct Timed {
  polyglot_ctx* ctx;
  int kid;
  Launch L;
  Timed(polyglot_ctx* c, int k, hipStream_t st) : ctx(c), kid(k) {
    L.s = st;
    if (ctx->timing && !ctx->capturing) {
      L.owner = this;
      L.take = &Timed::take;
    }
  }
  Timed(polyglot_ctx* c, int k) : Timed(c, k, c->stream) {}
  Timed(const Timed&) = delete;
  Timed& operator=(const Timed&) = delete;
  static bool take(void* owner, hipEvent_t* start, hipEvent_t* stop) {
    Timed* t = static_cast<Timed*>(owner);
    hipEvent_t a = take_event(t->ctx), b = take_event(t->ctx);
    if (!a || !b) {
      if (a) t->ctx->ev_pool.push_back(a);
      if (b) t->ctx->ev_pool.push_back(b);
      return false;
    }
    t->ctx->ev_marks.push_back({t->kid, {a, b}});
    *start = a;
    *stop = b;
    return true;
  }
};

SegArgs seg_args(polyglot_ctx* ctx, float* table, const float* Y, const SortPlan& plan, int set,
                 int N, int d, float alpha, bool step) {
  SegArgs a{};
  a.table = table;
  a.Y = Y;
  a.sk = ctx->ws.keys[2 * set + (plan.passes & 1)];
  a.sv = ctx->ws.vals[2 * set + (plan.passes & 1)];
  a.seg_part = ctx->ws.seg_part;
  a.long_list = ctx->ws.long_list;
  a.seg_end = ctx->ws.seg_end;
  a.flag = ctx->ws.flag;
  a.flag2 = step ? set_flag(ctx, set) : ctx->ws.flag;
  a.N = N;
  a.d = d;
  a.ch = seg_chunk_size(N);
  a.rg = a.ch * kWavesPerBlock;
  a.seg_stride = ctx->seg_stride;
  a.alpha = alpha;
  return a;
}

// Workgroups of the table role of k_apply.
int table_workgroups(const SegArgs& s, int mode) {
  const int units = mode == 0 ? ceil_div(ceil_div(s.N, s.ch), kWavesPerBlock)
                              : (int)std::min<int64_t>((int64_t)s.N * s.d / kBlock + 1, 1 << 20);
  return std::max(1, std::min(units, mode == 0 ? 2048 : 8192));
}

int segfix_workgroups(const SegArgs& s) {  // kSegfixWaves tasks per workgroup and round
  return std::max(1, std::min(ceil_div(ceil_div(s.N, s.rg), kSegfixWaves), 2048));
}

// The sort of one step's entries into sort set `set`, on stream `st` (the
// side stream, or the main stream for the first step of a folded call).
hipError_t enqueue_sort(polyglot_ctx* ctx, const int32_t* windows, const int32_t* corrupt, int B,
                        int set, hipStream_t st) {
  const polyglot_config& cf = ctx->cfg;
  const int N = B * (cf.win + 1);
  const StepKeys kf = step_keys(windows, corrupt, cf.win, cf.V);
  Timed tm(ctx, POLYGLOT_K_SORT, st);
  SortBufs sb = sort_bufs(ctx, set);
  sb.flag = set_flag(ctx, set);
  return launch_sort_step(kf, N, make_plan(cf.V, N), sb, tm.L);
}

// A step's bucketed sort into set `set`, as the extra workgroups of the
// previous step's update (tiles) and fix-up (buckets).
NextSort next_sort(polyglot_ctx* ctx, const int32_t* windows, const int32_t* corrupt, int B,
                   int set) {
  const polyglot_config& cf = ctx->cfg;
  NextSort nx{};
  nx.N = B * (cf.win + 1);
  const SortPlan plan = make_plan(cf.V, nx.N);
  nx.kf = step_keys(windows, corrupt, cf.win, cf.V);
  nx.sb = sort_bufs(ctx, set);
  nx.sb.flag = set_flag(ctx, set);
  nx.ntiles = plan.ntiles;
  nx.key_bits = plan.key_bits;
  nx.n_wg = plan.ntiles;
  return nx;
}

// The forward/backward launch(es), then (after `sorted_ev`, if any) the
// table update and, for a list sorted as a whole, the long-segment fix-up of
// one step, on the main stream; sorted mode reads sort set `set`.
int enqueue_compute(polyglot_ctx* ctx, float* E, float* W1, float* b1, float* w2, float* b2,
                    const int32_t* windows, const int32_t* corrupt, int B, float lr,
                    float* loss_dev, int set, hipEvent_t sorted_ev, const NextSort& nx,
                    const int32_t* next_windows, const int32_t* next_corrupt) {
  const polyglot_config& cf = ctx->cfg;
  const int N = B * (cf.win + 1);
  const bool sorted = cf.scatter_mode == POLYGLOT_SCATTER_SORTED;
  const SortPlan plan = make_plan(cf.V, N);
  const StepKeys kf = step_keys(windows, corrupt, cf.win, cf.V);
  hipError_t e = hipSuccess;

  LargeArgs la{};
  int n_fb = 0, split = 1;
  if (ctx->large) {
    la.E = E;
    la.W1 = W1;
    la.b1 = b1;
    la.w2 = w2;
    la.b2 = b2;
    la.windows = windows;
    la.corrupt = corrupt;
    la.V = ctx->ws.vbuf;
    la.vpart = ctx->ws.vpart;
    la.part = ctx->ws.part;
    la.G = ctx->ws.G;
    la.flag = ctx->ws.flag;
    la.V_rows = cf.V;
    la.d = cf.d;
    la.win = cf.win;
    la.H = cf.H;
    la.K = ctx->K;
    la.c = ctx->c;
    la.B = B;
    la.invB = 1.0f / (float)B;
    {
      Timed tm(ctx, POLYGLOT_K_FWDBWD);
      e = launch_large_fwd(la, 0, tm.L);
    }
    if (e == hipSuccess) {
      Timed tm(ctx, POLYGLOT_K_WIDE_DW1);
      e = launch_large_dw1(la, tm.L);
    }
    if (e == hipSuccess) {
      Timed tm(ctx, POLYGLOT_K_WIDE_G);
      e = launch_large_g(la, tm.L);
    }
  } else {
    FwdArgs fa{};
    fa.E = E;
    fa.W1 = W1;
    fa.b1 = b1;
    fa.w2 = w2;
    fa.b2 = b2;
    fa.windows = windows;
    fa.corrupt = corrupt;
    fa.G = ctx->ws.G;
    fa.part = ctx->ws.part;
    fa.flag = ctx->ws.flag;
    fa.V = cf.V;
    fa.d = cf.d;
    fa.win = cf.win;
    fa.H = cf.H;
    fa.Hp = ctx->Hp;
    fa.K = ctx->K;
    fa.c = ctx->c;
    fa.B = B;
    fa.N = N;
    fa.n_sort = (sorted && plan.small) ? (1 << plan.part_bits) : 0;  // the sort as extra workgroups
    fa.plan = plan;
    fa.sb = sort_bufs(ctx, set);
    fa.ntiles = ceil_div(B, kTileRows);
    const int shape8 = fwdbwd8_shape(cf.d, cf.win, ctx->NT);
    fa.tiles_per_wg = ceil_div(fa.ntiles, shape8 ? std::min(ctx->max_parts, kF8MaxWorkgroups)
                                                 : ctx->max_parts);
    // the pair form takes an even number of tiles per workgroup
    if (shape8 && kF8MultiForm == 2 && fa.tiles_per_wg > 1) fa.tiles_per_wg += fa.tiles_per_wg & 1;
    n_fb = ceil_div(fa.ntiles, fa.tiles_per_wg);
    // one tile per workgroup and CUs to spare: two workgroups per tile, each
    // taking half of its backward (the forward runs in both).  Only the
    // d 64 shape: the small one's backward is too short to pay for the
    // second copy of the forward (B = 32 step 11.6 -> 11.8 us split).
    fa.split = (shape8 == 1 && fa.tiles_per_wg == 1 && fa.n_sort + 2 * n_fb <= kF8MaxWorkgroups)
                   ? 2 : 1;
    n_fb *= fa.split;
    split = fa.split;
    fa.part_stride = ctx->part_stride;
    fa.invB = 1.0f / (float)B;
    {
      Timed tm(ctx, POLYGLOT_K_FWDBWD);
      if (shape8) {
        size_t lds = fwdbwd8_lds_bytes(shape8, fa.tiles_per_wg);
        if (fa.n_sort) lds = std::max(lds, part_sort_lds_words(kF8Threads) * 4);
        e = launch_step_fwdbwd8(fa, shape8, fa.n_sort + n_fb, lds, tm.L);
      } else {
        size_t lds = fwdbwd_lds_floats(ctx->Hp, ctx->K) * 4;
        if (fa.n_sort) lds = std::max(lds, part_sort_lds_words(kBlock) * 4);
        e = launch_step_fwdbwd(fa, ctx->NT, ctx->cpw, fa.n_sort + n_fb, lds, tm.L);
      }
    }
  }
  if (e != hipSuccess) return hip_fail(ctx, e, "fwd/bwd launch");
  if (sorted_ev) {
    e = hipStreamWaitEvent(ctx->stream, sorted_ev, 0);
    if (e != hipSuccess) return hip_fail(ctx, e, "sort join");
  }

  ApplyArgs aa{};
  aa.s = seg_args(ctx, E, ctx->ws.G, plan, set, N, cf.d, -lr, true);
  if (next_windows) {  // warm the memory-side cache with the next step's ids
    aa.pf.p[0] = next_windows;
    aa.pf.n[0] = B * cf.win;
    aa.pf.p[1] = next_corrupt;
    aa.pf.n[1] = B;
    aa.pf.sink = ctx->ws.pf_sink;
  }
  aa.mode = sorted ? 0 : 1;
  aa.n_e = table_workgroups(aa.s, aa.mode);
  aa.n_d = ceil_div(ctx->part_stride * kDenseSlices, kBlock);
  aa.dn.W1 = W1;
  aa.dn.b1 = b1;
  aa.dn.w2 = w2;
  aa.dn.b2 = b2;
  aa.dn.loss_out = loss_dev ? loss_dev : ctx->ws.scratch_loss;
  aa.dn.part = ctx->ws.part;
  if (ctx->large) {  // dW1 slices; db1 / dw2 / loss partials of the forward workgroups
    aa.dn.n_parts = ceil_div(B, kLgSlice);
    aa.dn.part_stride = cf.H * ctx->K;
    aa.dn.vpart = ctx->ws.vpart;
    aa.dn.n_vparts = ceil_div(B, kLgRows);
    aa.dn.vstride = 2 * cf.H + 2;
  } else {
    aa.dn.n_parts = n_fb;
    aa.dn.part_stride = ctx->part_stride;
    aa.dn.split = split;
    // the vector partials: every slot, or the first of each pair when split
    aa.dn.vpart = ctx->ws.part + (size_t)ctx->Hp * ctx->K;
    aa.dn.n_vparts = n_fb / split;
    aa.dn.vstride = ctx->part_stride * split;
  }
  aa.dn.H = cf.H;
  aa.dn.Hp = ctx->Hp;
  aa.dn.K = ctx->K;
  aa.dn.lr = lr;
  aa.dn.invB = 1.0f / (float)B;
  if (sorted) aa.zero = sort_zero_ranges(ctx, plan, set);  // counters of this set, now read
  if (sorted && plan.small) {
    // partition-sorted: one workgroup per partition completes every segment,
    // so no fix-up launch follows
    aa.part_off = ctx->ws.part_off[set];
    aa.n_part = 1 << plan.part_bits;
    aa.n_d = ceil_div(aa.n_d * kBlock, part_apply_threads(N));
    Timed tm(ctx, POLYGLOT_K_UPDATE);
    e = launch_apply_part(aa, aa.n_part + aa.n_d, tm.L);
  } else {
    {
      Timed tm(ctx, POLYGLOT_K_UPDATE);
      aa.nx = nx;
      e = nx.n_wg ? launch_apply_step_next(aa, kf, aa.n_e + aa.n_d, tm.L)
                  : launch_apply_step(aa, kf, aa.n_e + aa.n_d, tm.L);
    }
    if (e == hipSuccess && sorted) {
      Timed tm(ctx, POLYGLOT_K_SEGFIX);
      if (nx.n_wg) {
        NextSort nb = nx;
        nb.n_wg = bk_grid(nx.N);
        e = launch_segfix_step(aa.s, nb, segfix_workgroups(aa.s), tm.L);
      } else {
        e = launch_segfix(aa.s, segfix_workgroups(aa.s), tm.L);
      }
    }
  }
  if (e != hipSuccess) return hip_fail(ctx, e, "update launch");

  ctx->have_sorted = sorted;
  ctx->last_N = N;
  ctx->last_passes = plan.passes;
  ctx->last_set = set;
  return POLYGLOT_OK;
}

// Enqueues S consecutive steps (arguments already validated), step s using
// windows + s*B*win and corrupt + s*B.  Sorted mode, small batches: the sort
// is a role of the fused kernel (extra workgroups, no cross-stream join).
// Bucketed sorts (mid-size lists): the first step's sort runs on the main
// stream, and the sort of step s+1 runs as extra workgroups of step s's
// update and fix-up launches, beside their work, with no second stream (the
// fused kernel holds every CU, so a side-stream sort could not overlap it,
// and the cross-queue joins cost time of their own).  Other lists (above
// 786,432 entries, or the small sort of wide layers): the sort of step s+1
// runs on the side stream while step s computes; it waits for step s-1, the
// last reader of the same sort set.
int enqueue_steps(polyglot_ctx* ctx, float* E, float* W1, float* b1, float* w2, float* b2,
                  const int32_t* windows, const int32_t* corrupt, int S, int B, float lr,
                  float* losses_dev) {
  const bool sorted = ctx->cfg.scatter_mode == POLYGLOT_SCATTER_SORTED;
  const SortPlan plan = make_plan(ctx->cfg.V, B * (ctx->cfg.win + 1));
  const bool fold = sorted && plan.bucket;
  const bool side_sort = sorted && !fold && (ctx->large || !plan.small);
  const size_t wstride = (size_t)B * ctx->cfg.win;
  hipError_t e = hipSuccess;
  if (fold) {
    e = enqueue_sort(ctx, windows, corrupt, B, 0, ctx->stream);
    if (e != hipSuccess) return hip_fail(ctx, e, "sort launch");
  }
  if (side_sort) {
    e = hipEventRecord(ctx->ev_fork, ctx->stream);
    if (e == hipSuccess) e = hipStreamWaitEvent(ctx->side, ctx->ev_fork, 0);
    if (e == hipSuccess) e = enqueue_sort(ctx, windows, corrupt, B, 0, ctx->side);
    if (e == hipSuccess) e = hipEventRecord(ctx->ev_sorted[0], ctx->side);
    if (e != hipSuccess) return hip_fail(ctx, e, "sort launch");
  }
  for (int s = 0; s < S; ++s) {
    const int q = s & 1;
    if (side_sort && s + 1 < S) {
      if (s >= 1) e = hipStreamWaitEvent(ctx->side, ctx->ev_done[1 - q], 0);
      if (e == hipSuccess)
        e = enqueue_sort(ctx, windows + (s + 1) * wstride, corrupt + (size_t)(s + 1) * B, B,
                         1 - q, ctx->side);
      if (e == hipSuccess) e = hipEventRecord(ctx->ev_sorted[1 - q], ctx->side);
      if (e != hipSuccess) return hip_fail(ctx, e, "sort launch");
    }
    const NextSort nx =
        (fold && s + 1 < S)
            ? next_sort(ctx, windows + (s + 1) * wstride, corrupt + (size_t)(s + 1) * B, B, 1 - q)
            : NextSort{};
    const bool more = s + 1 < S;
    const int r = enqueue_compute(ctx, E, W1, b1, w2, b2, windows + s * wstride,
                                  corrupt + (size_t)s * B, B, lr,
                                  losses_dev ? losses_dev + s : nullptr, q,
                                  side_sort ? ctx->ev_sorted[q] : nullptr, nx,
                                  more ? windows + (s + 1) * wstride : nullptr,
                                  more ? corrupt + (size_t)(s + 1) * B : nullptr);
    if (r) return r;
    if (side_sort) {
      e = hipEventRecord(ctx->ev_done[q], ctx->stream);
      if (e != hipSuccess) return hip_fail(ctx, e, "step event");
    }
  }
  return POLYGLOT_OK;
}

int check_step_args(polyglot_ctx* ctx, float* E, float* W1, float* b1, float* w2, float* b2,
                    const int32_t* windows, const int32_t* corrupt, int B, float lr) {
  if (!E || !W1 || !b1 || !w2 || !b2 || !windows || !corrupt)
    return fail(ctx, POLYGLOT_ENULL, "train_step: NULL tensor pointer");
  if (B <= 0 || B > ctx->cfg.max_batch)
    return fail(ctx, POLYGLOT_EBATCH, "train_step: B must be in [1, max_batch]");
  if (!std::isfinite(lr)) return fail(ctx, POLYGLOT_EINVAL, "train_step: lr is not finite");
  if (!aligned16(E) || !aligned16(W1))
    return fail(ctx, POLYGLOT_EINVAL, "train_step: E and W1 must be 16-byte aligned");
  return POLYGLOT_OK;
}

// The float32 scatter-add once the arguments are valid: sorted segments
// (partition-wise for short lists) or one atomic per element.
int scatter_add_f32(polyglot_ctx* ctx, float* table, int32_t rows, int32_t d, const int32_t* idx,
                    const float* Y, int32_t N, float alpha, int32_t mode);

}  // namespace

extern "C" {

int polyglot_init(const polyglot_config* cfg, void* stream, polyglot_ctx** out) {
  if (!cfg || !out) return POLYGLOT_ENULL;
  *out = nullptr;
  const polyglot_config& c = *cfg;
  if (c.V < 1 || c.d < 16 || c.d > kMaxD || c.d % 16 != 0 || c.win < 1 || c.win > kMaxWin ||
      c.win % 2 == 0 || c.H < 1 || c.H > kMaxLargeH)
    return POLYGLOT_EINVAL;
  const bool large = c.H > kMaxHp;
  if (large && (c.H % 64 != 0 || c.d % 64 != 0)) return POLYGLOT_EINVAL;
  if (!large && c.win * c.d > kMaxK) return POLYGLOT_EINVAL;
  if (c.scatter_mode != POLYGLOT_SCATTER_SORTED && c.scatter_mode != POLYGLOT_SCATTER_ATOMIC)
    return POLYGLOT_EINVAL;
  if (c.max_batch < 1 || (int64_t)c.max_batch * (c.win + 1) > (1 << 26)) return POLYGLOT_EBATCH;
  if (c.max_scatter < 0 || c.max_scatter > (1 << 26) || c.max_rows < 0 ||
      (c.max_scatter > 0 && c.max_rows < 1))
    return POLYGLOT_EINVAL;
  if (!large) {  // the fused kernel keeps W1 and its tile buffers in one workgroup's LDS
    const int hp = c.H <= 16 ? 16 : (c.H <= 32 ? 32 : 64);
    if (fwdbwd_lds_floats(hp, c.win * c.d) * 4 > (size_t)kMaxLdsBytes) return POLYGLOT_EINVAL;
  }

  polyglot_ctx* ctx = new (std::nothrow) polyglot_ctx();
  if (!ctx) return POLYGLOT_EHIP;
  ctx->cfg = c;
  ctx->stream = static_cast<hipStream_t>(stream);
  ctx->K = c.win * c.d;
  ctx->c = c.win / 2;
  ctx->large = large;
  ctx->NT = large ? c.H / 16 : (c.H <= 16 ? 1 : (c.H <= 32 ? 2 : 4));
  ctx->Hp = 16 * ctx->NT;
  ctx->cpw = ceil_div(ctx->K / 16, kWavesPerBlock);
  ctx->max_entries = std::max({c.max_batch * (c.win + 1), c.max_scatter, 1});
  ctx->max_tiles = std::max(ceil_div(std::min(ctx->max_entries, kShortTileLimit), kSortTileKeysShort),
                            ceil_div(ctx->max_entries, kSortTileKeys));
  ctx->max_parts = std::min(ceil_div(c.max_batch, kTileRows), 512);
  // most chunks any call can cut (short chunks apply up to 131072 entries;
  // the general op cuts longer lists into gen_chunk_size chunks)
  ctx->max_chunks = std::max({ceil_div(std::min(ctx->max_entries, 131072), 16),
                              ceil_div(ctx->max_entries, seg_chunk_size(ctx->max_entries)),
                              ceil_div(c.max_scatter, gen_chunk_size(c.max_scatter))});
  ctx->seg_stride = std::max(c.d, c.max_scatter > 0 ? kMaxD : 0);
  ctx->part_stride = ctx->Hp * ctx->K + 2 * ctx->Hp + 2;

  hipError_t e = hipGetDevice(&ctx->device);
  Workspace& ws = ctx->ws;
  const size_t me = (size_t)ctx->max_entries;
  // passes of the largest key range this context sorts
  const int key_bits = bits_for((uint32_t)std::max({c.V, c.max_rows, 2}));
  const int max_passes = (key_bits + kMaxDigitBits - 1) / kMaxDigitBits;
  // look-back words of the multi-tile sort, or the (bucket, tile) words of the bucketed sort
  const size_t nstatus =
      std::max((size_t)max_passes * kMaxBins * ctx->max_tiles,
               (size_t)kBkBuckets * bk_tiles(std::min(ctx->max_entries, kBkMaxN)));
  for (int k = 0; k < 4; ++k) {
    if (e == hipSuccess) e = alloc(ctx, &ws.keys[k], me);
    if (e == hipSuccess) e = alloc(ctx, &ws.vals[k], me);
  }
  for (int k = 0; k < 2; ++k) {
    if (e == hipSuccess) e = alloc(ctx, &ws.totals[k], (size_t)kMaxPasses * kMaxBins);
    if (e == hipSuccess) e = alloc(ctx, &ws.status[k], nstatus);
    if (e == hipSuccess) e = alloc(ctx, &ws.tile_ctr[k], (size_t)kMaxPasses);
    if (e == hipSuccess) e = alloc(ctx, &ws.part_off[k], (size_t)(1 << kPartBits) + 1);
  }
  if (e == hipSuccess) e = alloc(ctx, &ws.G, (size_t)c.max_batch * (c.win + 1) * c.d);
  if (large) {
    const int slices = ceil_div(c.max_batch, kLgSlice);
    if (e == hipSuccess) e = alloc(ctx, &ws.part, (size_t)slices * c.H * ctx->K);
    if (e == hipSuccess)
      e = alloc(ctx, &ws.vpart, (size_t)ceil_div(c.max_batch, kLgRows) * (2 * c.H + 2));
    if (e == hipSuccess) e = alloc(ctx, &ws.vbuf, (size_t)c.max_batch * 3 * c.H);
  } else if (e == hipSuccess) {
    // two slots per tile group: the split backward gives each workgroup of a
    // pair its own
    e = alloc(ctx, &ws.part, (size_t)2 * ctx->max_parts * ctx->part_stride);
  }
  if (e == hipSuccess) e = alloc(ctx, &ws.seg_end, (size_t)std::max(c.V, c.max_rows));
  if (e == hipSuccess) e = alloc(ctx, &ws.seg_part, (size_t)ctx->max_chunks * 2 * ctx->seg_stride);
  if (e == hipSuccess) e = alloc(ctx, &ws.long_list, (size_t)ctx->max_chunks);
  if (e == hipSuccess) e = alloc(ctx, &ws.idx32, (size_t)c.max_scatter);
  if (e == hipSuccess) e = alloc(ctx, &ws.flag, 3);
  if (e == hipSuccess) e = alloc(ctx, &ws.scratch_loss, 1);
  if (e == hipSuccess) e = alloc(ctx, &ws.pf_sink, 1);
  for (int k = 0; k < 2; ++k) {
    if (e == hipSuccess)
      e = hipMemset(ws.totals[k], 0, sizeof(uint32_t) * kMaxPasses * kMaxBins);
    if (e == hipSuccess) e = hipMemset(ws.status[k], 0, sizeof(uint32_t) * nstatus);
    if (e == hipSuccess) e = hipMemset(ws.tile_ctr[k], 0, sizeof(uint32_t) * kMaxPasses);
  }
  if (e == hipSuccess) e = hipMemset(ws.flag, 0, 3 * sizeof(uint32_t));
  if (e == hipSuccess) e = hipStreamCreateWithFlags(&ctx->side, hipStreamNonBlocking);
  for (hipEvent_t* ev : {&ctx->ev_fork, &ctx->ev_sorted[0], &ctx->ev_sorted[1], &ctx->ev_done[0],
                         &ctx->ev_done[1]})
    if (e == hipSuccess) e = hipEventCreateWithFlags(ev, hipEventDisableTiming);
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (e != hipSuccess) {
    free_all(ctx);
    delete ctx;
    return POLYGLOT_EHIP;
  }
  *out = ctx;
  return POLYGLOT_OK;
}

int polyglot_destroy(polyglot_ctx* ctx) {
  if (!ctx) return POLYGLOT_ENULL;
  hipStreamSynchronize(ctx->stream);
  if (ctx->side) hipStreamSynchronize(ctx->side);
  free_all(ctx);
  delete ctx;
  return POLYGLOT_OK;
}

int polyglot_set_stream(polyglot_ctx* ctx, void* stream) {
  if (!ctx) return POLYGLOT_ENULL;
  ctx->stream = static_cast<hipStream_t>(stream);
  return POLYGLOT_OK;
}

int polyglot_train_step(polyglot_ctx* ctx, float* E, float* W1, float* b1, float* w2, float* b2,
                        const int32_t* windows, const int32_t* corrupt, int32_t B, float lr,
                        float* loss_dev) {
  if (!ctx) return POLYGLOT_ENULL;
  const int rc = check_step_args(ctx, E, W1, b1, w2, b2, windows, corrupt, B, lr);
  if (rc) return rc;
  return enqueue_steps(ctx, E, W1, b1, w2, b2, windows, corrupt, 1, B, lr, loss_dev);
}

int polyglot_train_step_sync(polyglot_ctx* ctx, float* E, float* W1, float* b1, float* w2,
                             float* b2, const int32_t* windows, const int32_t* corrupt,
                             int32_t B, float lr, float* loss_host) {
  if (!ctx) return POLYGLOT_ENULL;
  if (!loss_host) return fail(ctx, POLYGLOT_ENULL, "train_step_sync: NULL loss_host");
  int rc = check_step_args(ctx, E, W1, b1, w2, b2, windows, corrupt, B, lr);
  if (rc) return rc;
  rc = enqueue_steps(ctx, E, W1, b1, w2, b2, windows, corrupt, 1, B, lr, ctx->ws.scratch_loss);
  if (rc) return rc;
  float loss = 0.f;
  uint32_t w[3] = {0, 0, 0};
  hipError_t e = hipMemcpyAsync(&loss, ctx->ws.scratch_loss, sizeof(loss), hipMemcpyDeviceToHost,
                                ctx->stream);
  if (e == hipSuccess)
    e = hipMemcpyAsync(w, ctx->ws.flag, sizeof(w), hipMemcpyDeviceToHost, ctx->stream);
  if (e == hipSuccess) e = hipStreamSynchronize(ctx->stream);
  if (e != hipSuccess) return hip_fail(ctx, e, "train_step_sync: loss copy");
  *loss_host = loss;
  if (w[0] | w[1] | w[2])
    return fail(ctx, (w[0] | w[1] | w[2]) & kFlagBadId ? POLYGLOT_EID : POLYGLOT_EHIP,
                "train_step_sync: a device error word is raised; the step changed nothing");
  return POLYGLOT_OK;
}

int polyglot_train_steps(polyglot_ctx* ctx, float* E, float* W1, float* b1, float* w2,
                         float* b2, const int32_t* windows, const int32_t* corrupt, int32_t S,
                         int32_t B, float lr, float* losses_dev) {
  if (!ctx) return POLYGLOT_ENULL;
  if (S <= 0) return fail(ctx, POLYGLOT_EBATCH, "train_steps: S must be >= 1");
  const int rc = check_step_args(ctx, E, W1, b1, w2, b2, windows, corrupt, B, lr);
  if (rc) return rc;
  auto enqueue_all = [&]() -> int {
    return enqueue_steps(ctx, E, W1, b1, w2, b2, windows, corrupt, S, B, lr, losses_dev);
  };
  if (ctx->stream == nullptr) return enqueue_all();  // the legacy stream cannot be captured

  GraphKey key{{E, W1, b1, w2, b2, windows, corrupt}, losses_dev, S, B, lr, ctx->stream};
  if (!(ctx->gvalid && ctx->gkey == key)) {
    if (ctx->gexec) hipGraphExecDestroy(ctx->gexec);
    ctx->gexec = nullptr;
    ctx->gvalid = false;
    hipError_t e = hipStreamBeginCapture(ctx->stream, hipStreamCaptureModeThreadLocal);
    if (e != hipSuccess) return hip_fail(ctx, e, "train_steps: begin capture");
    ctx->capturing = true;
    const int r = enqueue_all();
    ctx->capturing = false;
    hipGraph_t graph = nullptr;
    e = hipStreamEndCapture(ctx->stream, &graph);
    if (r) {
      if (graph) hipGraphDestroy(graph);
      return r;
    }
    if (e != hipSuccess) return hip_fail(ctx, e, "train_steps: end capture");
    e = hipGraphInstantiate(&ctx->gexec, graph, nullptr, nullptr, 0);
    hipGraphDestroy(graph);
    if (e != hipSuccess) return hip_fail(ctx, e, "train_steps: instantiate");
    ctx->gkey = key;
    ctx->gvalid = true;
  }
  hipError_t e = hipGraphLaunch(ctx->gexec, ctx->stream);
  if (e != hipSuccess) return hip_fail(ctx, e, "train_steps: graph launch");
  const int N = B * (ctx->cfg.win + 1);
  ctx->have_sorted = ctx->cfg.scatter_mode == POLYGLOT_SCATTER_SORTED;
  ctx->last_N = N;
  ctx->last_passes = make_plan(ctx->cfg.V, N).passes;
  ctx->last_set = (S - 1) & 1;
  return POLYGLOT_OK;
}

int polyglot_score(polyglot_ctx* ctx, const float* E, const float* W1, const float* b1,
                   const float* w2, const float* b2, const int32_t* windows, int32_t B,
                   float* scores_dev) {
  if (!ctx) return POLYGLOT_ENULL;
  if (!E || !W1 || !b1 || !w2 || !b2 || !windows || !scores_dev)
    return fail(ctx, POLYGLOT_ENULL, "score: NULL pointer");
  if (B <= 0 || B > ctx->cfg.max_batch) return fail(ctx, POLYGLOT_EBATCH, "score: bad B");
  if (!aligned16(E) || !aligned16(W1))
    return fail(ctx, POLYGLOT_EINVAL, "score: E and W1 must be 16-byte aligned");
  hipError_t e;
  if (ctx->large) {
    LargeArgs la{};
    la.E = E;
    la.W1 = W1;
    la.b1 = b1;
    la.w2 = w2;
    la.b2 = b2;
    la.windows = windows;
    la.scores = scores_dev;
    la.flag = ctx->ws.flag;
    la.V_rows = ctx->cfg.V;
    la.d = ctx->cfg.d;
    la.win = ctx->cfg.win;
    la.H = ctx->cfg.H;
    la.K = ctx->K;
    la.c = ctx->c;
    la.B = B;
    Timed tm(ctx, POLYGLOT_K_SCORE);
    e = launch_large_fwd(la, 1, tm.L);
  } else {
    ScoreArgs a{E, W1, b1, w2, b2, windows, scores_dev, ctx->ws.flag, ctx->cfg.V, ctx->cfg.d,
                ctx->cfg.win, ctx->cfg.H, ctx->K, B};
    Timed tm(ctx, POLYGLOT_K_SCORE);
    e = launch_score(a, ctx->NT, ctx->cpw, tm.L);
  }
  return e == hipSuccess ? POLYGLOT_OK : hip_fail(ctx, e, "score launch");
}

int polyglot_gather(polyglot_ctx* ctx, const float* E, const int32_t* windows,
                    const int32_t* corrupt, int32_t B, float* X, float* Xc) {
  if (!ctx) return POLYGLOT_ENULL;
  if (!E || !windows || !corrupt || !X || !Xc) return fail(ctx, POLYGLOT_ENULL, "gather: NULL");
  if (B <= 0 || B > ctx->cfg.max_batch) return fail(ctx, POLYGLOT_EBATCH, "gather: bad B");
  if (!aligned16(E) || !aligned16(X) || !aligned16(Xc))
    return fail(ctx, POLYGLOT_EINVAL, "gather: E, X, Xc must be 16-byte aligned");
  GatherArgs a{E, windows, corrupt, X, Xc, ctx->ws.flag, ctx->cfg.V, ctx->cfg.d, ctx->cfg.win, B};
  hipError_t e;
  {
    Timed tm(ctx, POLYGLOT_K_GATHER);
    e = launch_gather(a, tm.L);
  }
  return e == hipSuccess ? POLYGLOT_OK : hip_fail(ctx, e, "gather launch");
}

int polyglot_scatter_add(polyglot_ctx* ctx, float* table, int32_t rows, int32_t d,
                         const int32_t* idx, const float* Y, int32_t N, float alpha,
                         int32_t mode) {
  if (!ctx) return POLYGLOT_ENULL;
  if (!table || !idx || !Y) return fail(ctx, POLYGLOT_ENULL, "scatter_add: NULL pointer");
  if (N <= 0 || N > ctx->cfg.max_scatter)
    return fail(ctx, POLYGLOT_EBATCH, "scatter_add: N must be in [1, max_scatter]");
  if (rows <= 0 || rows > ctx->cfg.max_rows || d <= 0 || d > kMaxD || d % 4 != 0)
    return fail(ctx, POLYGLOT_EINVAL, "scatter_add: bad rows or d");
  if (!aligned16(table) || !aligned16(Y))
    return fail(ctx, POLYGLOT_EINVAL, "scatter_add: table and Y must be 16-byte aligned");
  if (!std::isfinite(alpha)) return fail(ctx, POLYGLOT_EINVAL, "scatter_add: alpha not finite");
  if (mode != POLYGLOT_SCATTER_SORTED && mode != POLYGLOT_SCATTER_ATOMIC)
    return fail(ctx, POLYGLOT_EINVAL, "scatter_add: bad mode");
  return scatter_add_f32(ctx, table, rows, d, idx, Y, N, alpha, mode);
}

int polyglot_scatter_update(polyglot_ctx* ctx, void* table, int32_t dtype, int32_t rows,
                            int32_t d, const void* idx, int32_t idx_bytes, const void* Y,
                            int32_t N, float alpha, int32_t op, int32_t mode) {
  if (!ctx) return POLYGLOT_ENULL;
  if (!table || !idx || !Y) return fail(ctx, POLYGLOT_ENULL, "scatter_update: NULL pointer");
  if (N <= 0 || N > ctx->cfg.max_scatter)
    return fail(ctx, POLYGLOT_EBATCH, "scatter_update: N must be in [1, max_scatter]");
  if (rows <= 0 || rows > ctx->cfg.max_rows || d <= 0 || d > kMaxD)
    return fail(ctx, POLYGLOT_EINVAL, "scatter_update: bad rows or d");
  if (dtype != POLYGLOT_F32 && dtype != POLYGLOT_BF16 && dtype != POLYGLOT_F16)
    return fail(ctx, POLYGLOT_EINVAL, "scatter_update: bad storage format");
  if (idx_bytes != 4 && idx_bytes != 8)
    return fail(ctx, POLYGLOT_EINVAL, "scatter_update: indices must be 4 or 8 bytes");
  if (op != POLYGLOT_OP_INC && op != POLYGLOT_OP_SET)
    return fail(ctx, POLYGLOT_EINVAL, "scatter_update: bad op");
  if (mode != POLYGLOT_SCATTER_SORTED && mode != POLYGLOT_SCATTER_ATOMIC)
    return fail(ctx, POLYGLOT_EINVAL, "scatter_update: bad mode");
  if (op == POLYGLOT_OP_INC && !std::isfinite(alpha))
    return fail(ctx, POLYGLOT_EINVAL, "scatter_update: alpha not finite");
  const size_t es = dtype == POLYGLOT_F32 ? 4 : 2;
  if (reinterpret_cast<uintptr_t>(table) % es || reinterpret_cast<uintptr_t>(Y) % es ||
      reinterpret_cast<uintptr_t>(idx) % idx_bytes)
    return fail(ctx, POLYGLOT_EINVAL, "scatter_update: misaligned pointer");
  if (mode == POLYGLOT_SCATTER_ATOMIC && (dtype != POLYGLOT_F32 || op != POLYGLOT_OP_INC))
    return fail(ctx, POLYGLOT_EINVAL, "scatter_update: the atomic mode takes float32 increments only");
  hipError_t e = hipSuccess;
  // float32 increments take the scatter-add kernels (their fix-up reads rows
  // as 16-byte vectors, so the sorted mode wants d % 4 == 0 and aligned rows)
  if (dtype == POLYGLOT_F32 && op == POLYGLOT_OP_INC &&
      (mode == POLYGLOT_SCATTER_ATOMIC || (d % 4 == 0 && aligned16(table) && aligned16(Y)))) {
    const int32_t* keys = static_cast<const int32_t*>(idx);
    if (idx_bytes == 8) {  // narrowed (and range-checked) into the context's key buffer
      Timed tm(ctx, POLYGLOT_K_SORT);
      e = launch_keys_from_i64(static_cast<const int64_t*>(idx), N, rows, ctx->ws.idx32,
                               ctx->ws.flag, tm.L);
      if (e != hipSuccess) return hip_fail(ctx, e, "scatter_update: key launch");
      keys = ctx->ws.idx32;
    }
    return scatter_add_f32(ctx, static_cast<float*>(table), rows, d, keys,
                           static_cast<const float*>(Y), N, alpha, mode);
  }
  // the other calls sort the ids as they are (int64 ids narrowed and
  // range-checked by the sort's own key loads)
  const SortPlan plan = make_plan(rows, N);
  {
    Timed tm(ctx, POLYGLOT_K_SORT);
    e = idx_bytes == 8
            ? launch_sort_i64(I64Keys{static_cast<const int64_t*>(idx), rows}, N, plan,
                              sort_bufs(ctx, 0), tm.L)
            : launch_sort_idx(IdxKeys{static_cast<const int32_t*>(idx), rows}, N, plan,
                              sort_bufs(ctx, 0), tm.L);
  }
  GenCall c{};
  c.table = table;
  c.Y = Y;
  c.sk = ctx->ws.keys[plan.passes & 1];
  c.sv = ctx->ws.vals[plan.passes & 1];
  c.seg_part = ctx->ws.seg_part;
  c.long_list = ctx->ws.long_list;
  c.seg_end = ctx->ws.seg_end;
  c.flag = ctx->ws.flag;
  c.N = N;
  c.d = d;
  c.ch = gen_chunk_size(N);
  c.rg = c.ch * kWavesPerBlock;
  c.seg_stride = ctx->seg_stride;
  c.alpha = alpha;
  c.zero = sort_zero_ranges(ctx, plan, 0);
  c.dtype = dtype;
  c.op = op;
  c.n_e = std::max(1, std::min(ceil_div(ceil_div(N, op == POLYGLOT_OP_SET ? kWave : c.ch),
                                        kWavesPerBlock), 2048));
  c.n_z = plan.small ? 0 : 16;
  // a partitioned (small) list is applied partition-wise, in one launch
  c.part_off = ctx->ws.part_off[0];
  c.partitioned = plan.small;
  c.n_part = 1 << plan.part_bits;  // the partitions this sort wrote
  c.packed = dtype != POLYGLOT_F32 && d % 2 == 0 && reinterpret_cast<uintptr_t>(table) % 4 == 0 &&
             reinterpret_cast<uintptr_t>(Y) % 4 == 0;
  c.set_word = (int)es;
  for (int wb = 16; wb > (int)es; wb /= 2)
    if (((size_t)d * es) % wb == 0 && reinterpret_cast<uintptr_t>(table) % wb == 0 &&
        reinterpret_cast<uintptr_t>(Y) % wb == 0) {
      c.set_word = wb;
      break;
    }
  if (e == hipSuccess) {
    Timed tm(ctx, POLYGLOT_K_SCATTER);
    e = launch_gen_update(c, tm.L);
  }
  if (e == hipSuccess && op == POLYGLOT_OP_INC) {
    Timed tm(ctx, POLYGLOT_K_SEGFIX);
    e = launch_gen_fix(c, std::max(1, std::min(ceil_div(ceil_div(N, c.rg), kSegfixWaves), 2048)),
                       tm.L);
  }
  ctx->have_sorted = false;  // the sort buffers now hold this call's order
  return e == hipSuccess ? POLYGLOT_OK : hip_fail(ctx, e, "scatter_update launch");
}

}  // extern "C"

namespace {

int scatter_add_f32(polyglot_ctx* ctx, float* table, int32_t rows, int32_t d, const int32_t* idx,
                    const float* Y, int32_t N, float alpha, int32_t mode) {
  const SortPlan plan = make_plan(rows, N);
  const IdxKeys kf{idx, rows};
  ApplyArgs aa{};
  aa.s = seg_args(ctx, table, Y, plan, 0, N, d, alpha, false);
  aa.mode = mode == POLYGLOT_SCATTER_SORTED ? 0 : 1;
  aa.n_e = table_workgroups(aa.s, aa.mode);
  aa.n_d = 0;
  hipError_t e;
  if (aa.mode == 0) {
    // the sort validates the indices (sticky flag)
    aa.zero = sort_zero_ranges(ctx, plan, 0);
    const int n_z = plan.small ? 0 : 16;
    {
      Timed tm(ctx, POLYGLOT_K_SORT);
      e = launch_sort_idx(kf, N, plan, sort_bufs(ctx, 0), tm.L);
    }
    if (e == hipSuccess && plan.small) {  // partition-wise: no fix-up launch
      aa.part_off = ctx->ws.part_off[0];
      aa.n_part = 1 << plan.part_bits;
      Timed tm(ctx, POLYGLOT_K_SCATTER);
      e = launch_apply_part(aa, aa.n_part, tm.L);
    } else if (e == hipSuccess) {
      {
        Timed tm(ctx, POLYGLOT_K_SCATTER);
        e = launch_apply_idx(aa, kf, aa.n_e + n_z, tm.L);
      }
      if (e == hipSuccess) {
        Timed tm(ctx, POLYGLOT_K_SEGFIX);
        e = launch_segfix(aa.s, segfix_workgroups(aa.s), tm.L);
      }
    }
  } else {
    Timed tm(ctx, POLYGLOT_K_SCATTER);
    e = launch_check_idx(idx, N, rows, ctx->ws.flag, tm.L);
    if (e == hipSuccess) e = launch_apply_idx(aa, kf, aa.n_e, tm.L);
  }
  ctx->have_sorted = false;  // the sort buffers now hold this call's order
  return e == hipSuccess ? POLYGLOT_OK : hip_fail(ctx, e, "scatter_add launch");
}

}  // namespace

extern "C" {

int polyglot_touched_rows(polyglot_ctx* ctx, int32_t* ids_host, int32_t cap, int32_t* count) {
  if (!ctx || !count) return POLYGLOT_ENULL;
  if (!ctx->have_sorted) return fail(ctx, POLYGLOT_ESTATE, "touched_rows: no sorted step yet");
  hipError_t e = hipStreamSynchronize(ctx->stream);
  if (e != hipSuccess) return hip_fail(ctx, e, "touched_rows: sync");
  std::vector<int32_t> keys(ctx->last_N);
  e = hipMemcpy(keys.data(), ctx->ws.keys[2 * ctx->last_set + (ctx->last_passes & 1)],
                sizeof(int32_t) * ctx->last_N,
                hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_fail(ctx, e, "touched_rows: copy");
  // equal ids are contiguous (grouped) in the sorted order; report them ascending
  std::vector<int32_t> uniq;
  for (int i = 0; i < ctx->last_N; ++i)
    if (i == 0 || keys[i] != keys[i - 1]) uniq.push_back(keys[i]);
  std::sort(uniq.begin(), uniq.end());
  const int32_t n = (int32_t)uniq.size();
  for (int32_t i = 0; ids_host && i < n && i < cap; ++i) ids_host[i] = uniq[i];
  *count = n;
  return POLYGLOT_OK;
}

int polyglot_status(polyglot_ctx* ctx) {
  if (!ctx) return POLYGLOT_ENULL;
  hipError_t e = hipStreamSynchronize(ctx->stream);
  if (e != hipSuccess) return hip_fail(ctx, e, "status: sync");
  uint32_t w[3] = {0, 0, 0};
  e = hipMemcpy(w, ctx->ws.flag, sizeof(w), hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_fail(ctx, e, "status: read flag");
  const uint32_t f = w[0] | w[1] | w[2];
  if (f) {
    e = hipMemset(ctx->ws.flag, 0, sizeof(w));
    if (e != hipSuccess) return hip_fail(ctx, e, "status: clear flag");
    if (f & kFlagBadId) return fail(ctx, POLYGLOT_EID, "an id was outside its table");
    return fail(ctx, POLYGLOT_EHIP, "internal: sort position outside the entry range");
  }
  return POLYGLOT_OK;
}

int polyglot_set_timing(polyglot_ctx* ctx, int enable) {
  if (!ctx) return POLYGLOT_ENULL;
  ctx->timing = enable != 0;
  return POLYGLOT_OK;
}

int polyglot_kernel_times(polyglot_ctx* ctx, double* ms, int32_t* launches) {
  if (!ctx || !ms || !launches) return POLYGLOT_ENULL;
  hipError_t e = hipStreamSynchronize(ctx->stream);
  if (e == hipSuccess) e = hipStreamSynchronize(ctx->side);
  if (e != hipSuccess) return hip_fail(ctx, e, "kernel_times: sync");
  for (int k = 0; k < POLYGLOT_NKERNELS; ++k) {
    ms[k] = 0.0;
    launches[k] = 0;
  }
  for (auto& m : ctx->ev_marks) {
    float t = 0.f;
    if (hipEventElapsedTime(&t, m.second.first, m.second.second) == hipSuccess) {
      ms[m.first] += t;
      launches[m.first] += 1;
    }
    ctx->ev_pool.push_back(m.second.first);
    ctx->ev_pool.push_back(m.second.second);
  }
  ctx->ev_marks.clear();
  return POLYGLOT_OK;
}

const char* polyglot_last_error(const polyglot_ctx* ctx) { return ctx ? ctx->err.c_str() : ""; }

}  // extern "C"

// ------------------------------------------------------------ no-alloc scatter-add
// polyglot_scatter_add_noalloc keeps its sort buffers in `scratch`, a
// file-scope device array that every GPU the library runs on holds for the
// life of the process.  Host code never passes the array's name to a kernel
// (on the host it is only a stand-in for the symbol): the device address comes
// from hipGetSymbolAddress, once per device, with that device current.
namespace {

static_assert(pg::kStatusOk == POLYGLOT_OK && pg::kStatusBadId == POLYGLOT_EID,
              "device status words must equal the ABI codes");
constexpr int kNoAllocMaxN = POLYGLOT_NOALLOC_MAX_N;
constexpr int kNoAllocPartWords = 256;  // partition starts (129 used), one 1 KiB block
constexpr int kNoAllocFlagWords = 64;   // error flag, then the status word used when the
                                        // caller passes none, one 256-byte block
constexpr size_t kNoAllocWords = 2 * (size_t)kNoAllocMaxN + kNoAllocPartWords + kNoAllocFlagWords;
static_assert(kNoAllocWords * 4 == POLYGLOT_NOALLOC_SCRATCH_BYTES, "scratch size");
constexpr int kNoAllocMaxDevices = 64;

std::mutex g_noalloc_mu;
uint32_t* g_noalloc_ptr[kNoAllocMaxDevices];

}  // namespace

// Layout (32-bit words): sorted keys [kNoAllocMaxN], entry ids [kNoAllocMaxN],
// partition starts [kNoAllocPartWords], error flag and spare status word.
static __device__ __align__(256) uint32_t scratch[kNoAllocWords];

namespace {

// Device address of this device's copy of `scratch` (null on a HIP error).
uint32_t* noalloc_scratch() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kNoAllocMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_noalloc_mu);
  if (!g_noalloc_ptr[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return nullptr;
    g_noalloc_ptr[dev] = static_cast<uint32_t*>(ptr);
  }
  return g_noalloc_ptr[dev];
}

}  // namespace

extern "C" int polyglot_scatter_add_noalloc(float* table, int32_t rows, int32_t d,
                                            const int32_t* idx, const float* Y, int32_t N,
                                            float alpha, int32_t* status_dev, void* stream) {
  if (!table || !idx || !Y) return POLYGLOT_ENULL;
  if (N <= 0 || N > kNoAllocMaxN) return POLYGLOT_EBATCH;
  if (rows <= 0 || rows > POLYGLOT_NOALLOC_MAX_ROWS || d <= 0 || d > kMaxD || d % 4 != 0)
    return POLYGLOT_EINVAL;
  if (!aligned16(table) || !aligned16(Y) || !std::isfinite(alpha)) return POLYGLOT_EINVAL;
  const SortPlan plan = make_plan(rows, N);
  if (!plan.small) return POLYGLOT_EINVAL;  // not reached within the limits above
  uint32_t* base = noalloc_scratch();
  if (!base) return POLYGLOT_EHIP;
  int32_t* keys = reinterpret_cast<int32_t*>(base);
  int32_t* vals = reinterpret_cast<int32_t*>(base + kNoAllocMaxN);
  int32_t* part_off = reinterpret_cast<int32_t*>(base + 2 * kNoAllocMaxN);
  uint32_t* flag = base + 2 * kNoAllocMaxN + kNoAllocPartWords;
  SortBufs sb{};
  sb.keys[0] = sb.keys[1] = keys;
  sb.vals[0] = sb.vals[1] = vals;
  sb.part_off = part_off;
  sb.flag = flag;
  // the sort rewrites the flag (no clearing launch) and the status word
  sb.fresh_status = status_dev ? status_dev : reinterpret_cast<int32_t*>(flag + 1);
  ApplyArgs aa{};
  aa.s.table = table;
  aa.s.Y = Y;
  aa.s.sk = keys;
  aa.s.sv = vals;
  aa.s.flag = flag;
  aa.s.flag2 = flag;
  aa.s.N = N;
  aa.s.d = d;
  aa.s.ch = seg_chunk_size(N);
  aa.s.seg_stride = d;
  aa.s.alpha = alpha;
  aa.mode = 0;
  aa.part_off = part_off;
  aa.n_part = 1 << plan.part_bits;
  Launch L;
  L.s = static_cast<hipStream_t>(stream);
  hipError_t e = launch_sort_idx(IdxKeys{idx, rows}, N, plan, sb, L);
  if (e == hipSuccess) e = launch_apply_part(aa, aa.n_part, L);
  return e == hipSuccess ? POLYGLOT_OK : POLYGLOT_EHIP;
}
