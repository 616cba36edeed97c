// Table update of the embedding gradients (the advanced-indexing increment
// of §4.2/§4.3) and the dense SGD of one training step, in one launch with
// roles: k_apply (chunks of the whole sorted list, or the atomic variant)
// and k_apply_part (one workgroup per partition of a partitioned sort).  The
// standalone scatter-add uses the same launches without the dense role.
#pragma once
#include "common.h"
#include "launch.h"
#include "seg_dev.h"
#include "sort_dev.h"

namespace pg {

// Atomic variant: the per-(entry, column) increment of the paper's parallel
// kernel (§4.3), one float atomic add per element in arrival order.  One
// thread per element, so a wave's atomics cover consecutive columns of a row
// (few cache lines per instruction at the L2 atomic units).
template <class KeyFn>
__device__ void atomic_rows(const SegArgs& s, const KeyFn& kf, int wg, int n_e) {
  const size_t total = (size_t)s.N * s.d;
  for (size_t i = (size_t)wg * kBlock + threadIdx.x; i < total; i += (size_t)n_e * kBlock) {
    const int e = (int)(i / s.d);
    const int col = (int)(i - (size_t)e * s.d);
    const int32_t key = kf.load(e);
    unsafeAtomicAdd(s.table + (size_t)key * s.d + col, s.alpha * s.Y[i]);
  }
}

__device__ __forceinline__ uint32_t prefetch_lines(const Prefetch& pf, int gid, int nthreads) {
  uint32_t acc = 0u;
#pragma unroll
  for (int k = 0; k < 2; ++k)
    for (int i = gid * 16; i < pf.n[k]; i += nthreads * 16) acc += (uint32_t)pf.p[k][i];
  return acc;
}
__device__ __forceinline__ void prefetch_keep(const Prefetch& pf, uint32_t acc) {
  if (acc == 0x9E3779B9u && pf.sink != nullptr) *pf.sink = acc;
}

__device__ __forceinline__ void zero_ranges(const ZeroRanges& z, size_t gid, size_t nthreads) {
#pragma unroll
  for (int r = 0; r < 3; ++r)
    for (size_t i = gid; i < z.n[r]; i += nthreads) z.p[r][i] = 0u;
}

// Dense SGD.  A workgroup of T threads takes T / 8 consecutive elements at a
// time; its threads form kDenseSlices = 8 slot groups, group g summing the
// partial slots g, g + 8, g + 16, ... in order, with adjacent threads on
// adjacent elements of one slot (whole cache lines per load).  The eight
// group sums meet in LDS in the fixed tree ((0 + 1) + (2 + 3)) + ((4 + 5) +
// (6 + 7)), so the reduction is deterministic.  Elements: dW1 [Hp][K] from
// the dW1 partials, then db1 [Hp], dw2 [Hp], loss, db2 from the vector
// partials.  wg of nwg: this workgroup among the dense ones; red: T floats of
// LDS.  Every thread of the workgroup takes part (it synchronises).
template <int T>
__device__ void dense_sgd(const DenseArgs& a, int wg, int nwg, bool bad, float* red) {
  constexpr int SL = kDenseSlices;
  constexpr int EW = T / SL;
  static_assert(SL == 8 && T % SL == 0, "the combining tree adds eight group sums");
  const int HK = a.Hp * a.K;
  const int nel = HK + 2 * a.Hp + 2;
  const int t = threadIdx.x;
  const int g = t / EW, j = t - g * EW;
  for (int base = wg * EW; base < nel; base += nwg * EW) {
    const int e = base + j;
    float s = 0.f;
    if (e < nel) {
      const bool mat = e < HK;
      const float* src = mat ? a.part + e : a.vpart + (e - HK);
      int np = mat ? a.n_parts : a.n_vparts;
      size_t stride = mat ? (size_t)a.part_stride : (size_t)a.vstride;
      if (mat && a.split == 2) {  // the slot of the pair that holds this element's tile
        const int n = e / a.K, k = e - n * a.K;
        src += (size_t)((((k >> 4) * (a.Hp >> 4)) + (n >> 4)) & 1) * a.part_stride;
        np >>= 1;
        stride *= 2;
      }
      for (int p0 = g; p0 < np; p0 += 8 * SL) {
        float v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int p = p0 + u * SL;
          v[u] = p < np ? src[(size_t)p * stride] : 0.f;
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) s += v[u];
      }
    }
    red[t] = s;
    __syncthreads();
    if (g == 0 && e < nel) {
      const float* r = red + j;
      s = ((r[0] + r[EW]) + (r[2 * EW] + r[3 * EW])) +
          ((r[4 * EW] + r[5 * EW]) + (r[6 * EW] + r[7 * EW]));
      if (e < HK) {
        if (!bad && e / a.K < a.H) a.W1[e] = a.W1[e] - a.lr * s;
      } else if (e < HK + a.Hp) {
        const int n = e - HK;
        if (!bad && n < a.H) a.b1[n] = a.b1[n] - a.lr * s;
      } else if (e < HK + 2 * a.Hp) {
        const int n = e - HK - a.Hp;
        if (!bad && n < a.H) a.w2[n] = a.w2[n] - a.lr * s;
      } else if (e == HK + 2 * a.Hp) {
        a.loss_out[0] = bad ? __builtin_nanf("") : s * a.invB;
      } else {
        if (!bad) a.b2[0] = a.b2[0] - a.lr * s;
      }
    }
    __syncthreads();  // red is rewritten by the next pass
  }
}

// Workgroups [0, nx.n_wg) rank the tiles of the next training step's
// bucketed sort (its ids only; first in the grid, so that they are dispatched
// beside the table role, not after it); the next n_e update the table; the
// rest run the dense SGD and clearing roles.
template <int CH, class KeyFn>
__global__ __launch_bounds__(kBlock, 5) void k_apply(ApplyArgs a, KeyFn kf) {
  __shared__ float F[kWavesPerBlock][kMaxD];
  __shared__ float Lp[kWavesPerBlock][kMaxD];
  __shared__ int meta[kWavesPerBlock][5];
  const int t = threadIdx.x;
  if ((int)blockIdx.x < a.nx.n_wg) {
    extern __shared__ uint32_t lds_u[];
    bk_tiles<kBlock>(a.nx.kf, a.nx.N, a.nx.ntiles, a.nx.sb, blockIdx.x, lds_u);
    return;
  }
  const int wg = (int)blockIdx.x - a.nx.n_wg;  // index among the update's workgroups
  const int n_dz = (int)gridDim.x - a.nx.n_wg - a.n_e;
  if (wg < a.n_e) {
    // all-or-nothing: an out-of-range id voids the update.  The error words
    // were set (or not) by earlier launches, so every wave reads the same
    // value (the sorted mode tests it beside each chunk's keys)
    if (a.mode == 0) {
      const int nranges = ceil_div(a.s.N, CH * kWavesPerBlock);
      for (int r = wg; r < nranges; r += a.n_e)
        seg_apply_range<CH, kWavesPerBlock>(a.s, r, F, Lp, meta);
    } else {
      if (void_bits(a.s)) return;
      atomic_rows(a.s, kf, wg, a.n_e);
    }
    return;
  }
  const int gid = (wg - a.n_e) * kBlock + t;
  const int nthreads = n_dz * kBlock;
  const uint32_t pfa = prefetch_lines(a.pf, gid, nthreads);
  const bool bad = void_bits(a.s) != 0u;
  if (a.n_d > 0) dense_sgd<kBlock>(a.dn, wg - a.n_e, n_dz, bad, &F[0][0]);
  zero_ranges(a.zero, gid, nthreads);
  prefetch_keep(a.pf, pfa);
}

// Sorted update of a partition-sorted list: workgroup p < n_part applies
// partition p, whose segments never leave it, so no fix-up launch follows;
// the remaining workgroups run the dense SGD and clearing roles.  PC:
// entries per chunk (32 for lists of at most kPartShortN entries, else 64),
// NTH: threads per workgroup (part_apply_threads).
template <int PC, int NTH>
__global__ __launch_bounds__(NTH) void k_apply_part(ApplyArgs a) {
  constexpr int NW = NTH / kWave;
  __shared__ float F[NW][kMaxD];
  __shared__ float Lp[NW][kMaxD];
  __shared__ int meta[NW][5];
  const int t = threadIdx.x;
  if ((int)blockIdx.x < a.n_part) {
    // (the error words are tested beside each chunk's keys)
    const int p = blockIdx.x;
    seg_apply_partition<NW, SegArgs, PC>(a.s, a.part_off[p], a.part_off[p + 1], F, Lp, meta);
    return;
  }
  const int gid = (blockIdx.x - a.n_part) * NTH + t;
  const int nthreads = (gridDim.x - a.n_part) * NTH;
  const uint32_t pfa = prefetch_lines(a.pf, gid, nthreads);
  const bool bad = void_bits(a.s) != 0u;
  if (a.n_d > 0) dense_sgd<NTH>(a.dn, blockIdx.x - a.n_part, gridDim.x - a.n_part, bad, &F[0][0]);
  zero_ranges(a.zero, gid, nthreads);
  prefetch_keep(a.pf, pfa);
}

// Rows whose sorted entries cross chunks.  Task li is chunk li's slot of the
// segment list (empty unless a crossing segment starts in that chunk).  A
// workgroup takes kSegfixWaves slots at a time: a light segment is finished
// by its wave, a heavy one is listed and then summed by the whole workgroup.
// Every row is a different segment's, so the order in which heavy ones are
// taken does not matter.
// Workgroup wg of nwg: crossing segments listed in the range slots (see
// k_segfix).  red, heavy and nheavy are the workgroup's LDS.
template <class A>
__device__ void segfix_wg(const A& a, int wg, int nwg, float* red, int (*heavy)[3],
                          int* nheavy_p) {
  int& nheavy = *nheavy_p;
  // (the error words are tested beside each slot's loads)
  const uint32_t cnt = (uint32_t)((a.N + a.rg - 1) / a.rg);  // ranges of the apply
  const int t = threadIdx.x, lane = t & (kWave - 1);
  const int w = __builtin_amdgcn_readfirstlane(t / kWave);
  // slot li of a round goes to workgroup li % nwg, so the segments of heavy
  // rows that start in nearby ranges land in different workgroups
  for (uint32_t base = 0; base + wg < cnt; base += nwg * kSegfixWaves) {
    if (t == 0) nheavy = 0;
    __syncthreads();
    const uint32_t li = base + (uint32_t)w * nwg + wg;
    if (li < cnt) {
      int32_t key = 0;
      const int m = seg_fix_slot_wave(a, (int)li, (int)cnt, &key);
      if (m > kSegfixLight && lane == 0) {  // a heavy row: its partials run to seg_end[key]
        const int h = atomicAdd(&nheavy, 1);
        heavy[h][0] = (int)li;
        heavy[h][1] = key;
        heavy[h][2] = a.seg_end[key] - (int)li + 1;
      }
    }
    __syncthreads();
    const int nh = nheavy;
    for (int h = 0; h < nh; ++h) seg_fix_row(a, heavy[h][0], heavy[h][1], heavy[h][2], red);
    __syncthreads();  // the heavy list is rewritten by the next round
  }
}

template <class A>
__global__ __launch_bounds__(kSegfixThreads) void k_segfix(A a) {
  __shared__ float red[kSegfixWaves * kMaxD];
  __shared__ int heavy[kSegfixWaves][3];  // (start range, row, partials)
  __shared__ int nheavy;
  segfix_wg(a, blockIdx.x, gridDim.x, red, heavy, &nheavy);
}

// The fix-up of a training step and, in workgroups [0, nx.n_wg) (first, so
// that they are dispatched beside it), the bucket launch of the next step's
// bucketed sort (its tiles ran in the update launch), which only reads that
// step's ids: no stream join needed.
__global__ __launch_bounds__(kSegfixThreads) void k_segfix_step(SegArgs a, NextSort nx, int n_fix) {
  __shared__ float red[kSegfixWaves * kMaxD];
  __shared__ int heavy[kSegfixWaves][3];
  __shared__ int nheavy;
  extern __shared__ uint32_t lds_u[];
  static_assert(kSegfixThreads == kBkSortThreads, "one workgroup size for both roles");
  if ((int)blockIdx.x < nx.n_wg) {
    bk_buckets(nx.N, nx.ntiles, nx.key_bits, nx.sb, blockIdx.x, lds_u);
    return;
  }
  segfix_wg(a, (int)blockIdx.x - nx.n_wg, n_fix, red, heavy, &nheavy);
}

}  // namespace pg
