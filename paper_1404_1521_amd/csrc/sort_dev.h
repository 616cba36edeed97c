// Stable LSD radix sort of (row id, entry index) pairs.
//
// The embedding update of §4.2/§4.3 adds many rows into few distinct table
// rows (Zipf-distributed word ids repeat heavily).  Sorting the entries by row
// id turns that into a segmented sum with one writer per table row, so the
// update is deterministic and free of atomics.  Entries with equal row ids
// keep their entry order (stable LSD), which fixes the summation order.
//
// Two variants:
//  * small (up to kSmallSortN entries): a partitioned sort, one launch of
//    2^part_bits workgroups (see part_sort below);
//  * multi-tile: a histogram launch, then one launch per radix pass over
//    4096-key tiles with a decoupled look-back over earlier tiles' digit
//    counts (see the multi-tile section below).
//
// Ranking inside a wave: keys are held in registers, R rounds of 64; the
// lanes of a round that share a digit are found with ballots, and the lowest
// of them adds the group size to the wave's LDS counter with an atomic that
// returns the old count.  The atomics of all rounds are issued back to back
// (LDS executes one wave's operations in order, so round r sees rounds < r),
// and the returned counts are broadcast to the group afterwards.
#pragma once
#include "common.h"

namespace pg {

// Key sources -------------------------------------------------------------

// Entries of a training step: entry e = b*(win+1) + j is windows[b][j] for
// j < win and corrupt[b] for j = win.  b = e / (win+1) is taken as the high
// word of e * inv with inv = ceil(2^32 / (win+1)), which is exact for
// e < 2^26 and win + 1 <= 32 (the error term e * (inv*(win+1) - 2^32) / 2^32
// stays below 1/(win+1)).
struct StepKeys {
  const int32_t* windows;
  const int32_t* corrupt;
  int win, range;   // range = V
  uint32_t inv;
  __device__ int32_t load(int e) const {
    const int b = (int)__umulhi((uint32_t)e, inv);
    const int j = e - b * (win + 1);
    return (j < win) ? windows[(size_t)b * win + j] : corrupt[b];
  }
};

__host__ __device__ inline StepKeys step_keys(const int32_t* windows, const int32_t* corrupt,
                                              int win, int V) {
  return StepKeys{windows, corrupt, win, V, (uint32_t)(0xffffffffu / (uint32_t)(win + 1)) + 1u};
}

struct IdxKeys {  // entries of the standalone scatter-add
  const int32_t* idx;
  int range;        // table rows
  __device__ int32_t load(int e) const { return idx[e]; }
};
// int64 entries of the general op, narrowed as they are loaded: an id
// outside [0, range) loads as 0xffffffff, which the sort's range check turns
// into key 0 and the sticky error flag (no narrowing launch of its own).
struct I64Keys {
  const int64_t* idx;
  int range;        // table rows
  __device__ int32_t load(int e) const {
    const int64_t v = idx[e];
    return (v < 0 || v >= (int64_t)range) ? -1 : (int32_t)v;
  }
};

// Loads U keys per thread with all loads in flight before any check; ids
// outside [0, range) become 0 and raise the sticky flag once.
template <int U, class KeyFn>
__device__ __forceinline__ void load_keys(const KeyFn& kf, int N, int e0, int stride,
                                          uint32_t* key, uint32_t* flag) {
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int e = e0 + u * stride;
    key[u] = e < N ? (uint32_t)kf.load(e) : 0u;
  }
  bool bad = false;
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const bool b = key[u] >= (uint32_t)kf.range;
    bad |= b;
    key[u] = b ? 0u : key[u];
  }
  if (bad) atomicOr(flag, kFlagBadId);
}

// Exclusive scan over `n` (<= 2*NTH) values in LDS `v`, in place, by one
// workgroup of NTH threads.
template <int NTH = kBlock>
__device__ inline void block_exclusive_scan(uint32_t* v, int n, uint32_t* wave_sums) {
  const int t = threadIdx.x, lane = t & (kWave - 1);
  const int w = __builtin_amdgcn_readfirstlane(t / kWave);
  const uint32_t a = (2 * t < n) ? v[2 * t] : 0u;
  const uint32_t b = (2 * t + 1 < n) ? v[2 * t + 1] : 0u;
  const uint32_t s = a + b;
  const uint32_t inc = wave_incl_scan(s);
  if (lane == kWave - 1) wave_sums[w] = inc;
  __syncthreads();
  uint32_t base = 0;
#pragma unroll
  for (int i = 0; i < NTH / kWave; ++i) base += i < w ? wave_sums[i] : 0u;  // loads in parallel
  const uint32_t ex = base + inc - s;
  if (2 * t < n) v[2 * t] = ex;
  if (2 * t + 1 < n) v[2 * t + 1] = ex + a;
  __syncthreads();
}

// Exclusive scan over `n` (<= 16*NTH) values in LDS `v`, in place, by one
// workgroup of NTH threads: thread t takes a run of ceil(n/NTH) values.
template <int NTH>
__device__ inline void block_exclusive_scan_runs(uint32_t* v, int n, uint32_t* wave_sums) {
  const int t = threadIdx.x, lane = t & (kWave - 1);
  const int w = __builtin_amdgcn_readfirstlane(t / kWave);
  const int E = ceil_div(n, NTH), b0 = t * E;
  uint32_t s = 0;
  for (int i = 0; i < E; ++i)
    if (b0 + i < n) s += v[b0 + i];
  const uint32_t inc = wave_incl_scan(s);
  if (lane == kWave - 1) wave_sums[w] = inc;
  __syncthreads();
  uint32_t run = inc - s;
#pragma unroll
  for (int i = 0; i < NTH / kWave; ++i) run += i < w ? wave_sums[i] : 0u;  // loads in parallel
  for (int i = 0; i < E; ++i) {
    if (b0 + i < n) {
      const uint32_t c = v[b0 + i];
      v[b0 + i] = run;
      run += c;
    }
  }
  __syncthreads();
}

// Stable ranks of up to R rounds of 64 keys held by this wave (round-major
// order); rounds r >= nr and lanes with act[r] false are skipped.  The
// wave's zeroed LDS counter of digit d is hist[d * stride].  On return
// rank[r] is the number of earlier keys of the wave with the same digit, and
// the counters hold the wave's digit counts.
template <int R>
__device__ __forceinline__ void wave_rank(const uint32_t (&dg)[R], const uint64_t (&act)[R],
                                          int nr, int bits, uint32_t* hist, uint32_t (&rank)[R],
                                          int stride = 1) {
  uint32_t old[R], below_leader[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    old[r] = 0u;
    below_leader[r] = 0u;
    if (r < nr) {
      const uint64_t peers = match_digit(dg[r], bits, act[r]);
      const uint32_t below = __popcll(peers & lanemask_lt());
      const uint32_t leader = peers ? (uint32_t)(__ffsll((unsigned long long)peers) - 1) : 0u;
      below_leader[r] = below | (leader << 16);
      if (((act[r] >> lane_id()) & 1ull) && below == 0)
        old[r] = atomicAdd(&hist[dg[r] * stride], (uint32_t)__popcll(peers));
    }
  }
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const uint32_t base = __shfl(old[r], (int)(below_leader[r] >> 16));
    rank[r] = base + (below_leader[r] & 0xffffu);
  }
}

// ------------------------------------------------------- LDS radix passes
constexpr int kRankBatch = 8;  // rounds ranked per batch (registers bounded)

// Stable LSD radix passes of one workgroup (NTH threads) over M <= kSmallSortN
// packed words in LDS, ping-pong between src and dst.  The digit of pass p
// is (word >> (shift0 + plan.shift[p])) & (2^plan.bits[p] - 1).  Wave w
// ranks a contiguous run of the words (wave_rank) into its column of the
// counter table hist[digit][wave]; one exclusive scan of that table in
// (digit, wave) order gives every wave the output offset of every digit, and
// the words are scattered.  Returns the buffer holding the sorted words.
template <int NTH>
__device__ uint32_t* lds_lsd_passes(uint32_t* src, uint32_t* dst, int M, const SortPlan& plan,
                                    int shift0, uint16_t* rank16, uint32_t* hist,
                                    uint32_t* misc) {
  constexpr int R = kRankBatch, NW = NTH / kWave;
  const int lane = threadIdx.x & (kWave - 1);
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  // counter of digit d for wave w at hist[d * (NW + 1) + w]; the extra
  // column (always 0) spreads the digits of one wave over the LDS banks
  constexpr int CS = NW + 1;
  uint32_t* mycol = hist + w;
  // wave w owns words [w*per, (w+1)*per), per a multiple of 64
  const int per = ceil_div(ceil_div(M, NW), kWave) * kWave;
  const int beg = w * per;
  const int nr = max(0, min(per, M - beg) + kWave - 1) / kWave;
  for (int p = 0; p < plan.passes; ++p) {
    const int bits = plan.bits[p], shift = plan.shift[p] + shift0, bins = 1 << bits;
    for (int d = lane; d < bins; d += kWave) {
      mycol[d * CS] = 0;
      if (w == 0) hist[d * CS + NW] = 0;  // the padding column
    }
    wave_lds_sync();
    for (int r0 = 0; r0 < nr; r0 += R) {  // the wave's counters carry over batches
      uint32_t dg[R], rank[R];
      uint64_t act[R];
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const int i = beg + (r0 + r) * kWave + lane;
        const bool ok = r0 + r < nr && i < M;
        act[r] = __ballot(ok);
        dg[r] = ((ok ? src[i] : 0u) >> shift) & (uint32_t)(bins - 1);
      }
      wave_rank<R>(dg, act, min(R, nr - r0), bits, mycol, rank, CS);
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const int i = beg + (r0 + r) * kWave + lane;
        if ((act[r] >> lane) & 1ull) rank16[i] = (uint16_t)rank[r];
      }
    }
    __syncthreads();
    block_exclusive_scan_runs<NTH>(hist, bins * CS, misc);  // offsets by (digit, wave)
    for (int r0 = 0; r0 < nr; r0 += R) {
      uint32_t word[R], rk[R];
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const int i = beg + (r0 + r) * kWave + lane;
        const bool ok = r0 + r < nr && i < M;
        word[r] = ok ? src[i] : 0u;
        rk[r] = ok ? (uint32_t)rank16[i] : 0u;
      }
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const int i = beg + (r0 + r) * kWave + lane;
        if (r0 + r < nr && i < M) {
          const uint32_t pos = mycol[((word[r] >> shift) & (uint32_t)(bins - 1)) * CS] + rk[r];
          if (pos < (uint32_t)M) dst[pos] = word[r];
        }
      }
    }
    __syncthreads();
    uint32_t* tmp = src;
    src = dst;
    dst = tmp;
  }
  return src;
}

// ------------------------------------------------------- partitioned small sort
// Up to kSmallSortN entries are sorted by 2^part_bits workgroups with no
// communication between them.  Workgroup p takes the entries whose key has
// low bits equal to p (a hash partition: the heavy Zipf rows, which are the
// small ids, spread over all workgroups), compacts them in entry order,
// radix-sorts them in LDS by the remaining key bits (stable: entry order is
// kept within a key) and writes them after the entries of the partitions
// below p, which it counts itself while reading the keys.  Equal keys end up
// contiguous and in entry order -- what the segmented sum needs; the order
// between distinct keys is fixed by the keys alone.
constexpr int kPartBits = 7;
// Partitions of at most this many entries are ranked by counting smaller
// words (quadratic in the partition: measured faster than the two LDS radix
// passes up to about 540 entries, slower at 720).
constexpr int kRankSortMax = 512;
constexpr int kRankSplitMin = 128;  // partitions above this place their smallest key first
constexpr int kPartSortThreads = 1024;  // one workgroup of 16 waves per partition
constexpr int kPartSortMisc = 32;       // scan scratch: wave sums, then the partition total
__host__ __device__ constexpr size_t part_sort_lds_words(int nth) {
  return 2 * kSmallSortN + kSmallSortN / 2 + (size_t)(nth / kWave + 1) * kSmallBins + kPartSortMisc;
}

// fresh_status: null for a sort whose error flag is sticky (bad ids OR
// kFlagBadId into *flag).  Otherwise the flag is rewritten by this sort: every
// workgroup reads every key, so workgroup 0 alone stores *flag (kFlagBadId or
// 0) and *fresh_status (kStatusBadId or kStatusOk), and nothing needs
// clearing between calls.
template <int NTH, class KeyFn>
__device__ void part_sort(const KeyFn& kf, int N, const SortPlan& plan, int part,
                          int32_t* out_keys, int32_t* out_vals, int32_t* part_off, uint32_t* flag,
                          uint32_t* lds, int32_t* fresh_status = nullptr) {
  constexpr int NW = NTH / kWave, UMAX = kSmallSortN / NTH;
  static_assert(NW + 1 <= kPartSortMisc, "scan scratch too small");
  uint32_t* bufA = lds;
  uint32_t* bufB = bufA + kSmallSortN;
  uint16_t* rank16 = reinterpret_cast<uint16_t*>(bufB + kSmallSortN);
  uint32_t* hist = bufB + kSmallSortN + kSmallSortN / 2;  // [kSmallBins][waves + 1]
  uint32_t* misc = hist + (NW + 1) * kSmallBins;          // kPartSortMisc words
  const int t = threadIdx.x;
  const int vb = plan.val_bits, pb = plan.part_bits;
  const uint32_t pmask = (1u << pb) - 1u;
  const int U = ceil_div(N, NTH);  // contiguous entries per thread (<= UMAX)

  // keys of entries t*U .. t*U+U-1, every load in flight before any use
  uint32_t key[UMAX];
#pragma unroll
  for (int u = 0; u < UMAX; ++u) {
    const int e = t * U + u;
    key[u] = (u < U && e < N) ? (uint32_t)kf.load(e) : 0u;
  }
  bool bad = false;
  uint32_t mine = 0, below = 0;
#pragma unroll
  for (int u = 0; u < UMAX; ++u) {
    const int e = t * U + u;
    const bool act = u < U && e < N;
    const bool b = act && key[u] >= (uint32_t)kf.range;
    bad |= b;
    key[u] = b ? 0u : key[u];
    const uint32_t pk = key[u] & pmask;
    mine += (act && pk == (uint32_t)part) ? 1u : 0u;
    below += (act && pk < (uint32_t)part) ? 1u : 0u;
  }
  if (fresh_status) {
    const int any = __syncthreads_or(bad ? 1 : 0);
    if (part == 0 && t == 0) {
      *flag = any ? kFlagBadId : 0u;
      *fresh_status = any ? kStatusBadId : kStatusOk;
    }
  } else if (bad) {
    atomicOr(flag, kFlagBadId);
  }

  // exclusive prefix over threads of (below << 16 | mine): each thread's
  // first slot in the partition, and at the end the partition's size and
  // output offset (sums stay below 2^16)
  const uint32_t packed = (below << 16) | mine;
  hist[t] = packed;
  __syncthreads();
  block_exclusive_scan<NTH>(hist, NTH, misc);
  const uint32_t ex = hist[t];
  if (t == NTH - 1) misc[NW] = ex + packed;  // after the NW wave sums
  uint32_t pos = ex & 0xffffu;
#pragma unroll
  for (int u = 0; u < UMAX; ++u) {
    const int e = t * U + u;
    if (u < U && e < N && (key[u] & pmask) == (uint32_t)part)
      bufA[pos++] = ((key[u] >> pb) << vb) | (uint32_t)e;
  }
  __syncthreads();
  const uint32_t tot = misc[NW];
  const int M = (int)(tot & 0xffffu), off = (int)(tot >> 16);
  if (t == 0) {  // the partition's place in the output (for the partition-wise update)
    part_off[part] = off;
    if (part == (int)pmask) part_off[part + 1] = off + M;
  }
  __syncthreads();  // misc and hist are reused by the passes

  // The words (key bits above the partition bits, then the entry id) are
  // distinct, so a word's place in the sorted partition is the number of
  // smaller words: up to kRankSortMax words are ranked by broadcast LDS
  // reads (the same order as the stable radix passes, which larger
  // partitions take).  Word i is counted by G threads, thread group g
  // scanning its own share of the words, so the pass over a partition of
  // M words costs about M / G compares per thread; the G counts meet in LDS.
  // In a frequency-ranked vocabulary the smallest key of a partition (key
  // bits above the partition bits all zero) is by far its most frequent: in
  // a partition of more than kRankSplitMin words those words, already in
  // entry order in bufA, take the first places by a prefix count, and only
  // the others are ranked by comparison.
  uint32_t* res;
  if (M <= kRankSortMax && M <= NTH) {
    uint32_t* cnt = reinterpret_cast<uint32_t*>(rank16);  // [G][S] partial counts
    uint32_t* rest = cnt + NTH;                           // the other words, compacted
    const uint32_t* src = bufA;
    int Mr = M, Z = 0;
    if (M > kRankSplitMin) {
      const int lane = t & (kWave - 1), w = t / kWave;
      const uint32_t wv0 = t < M ? bufA[t] : 0u;
      const bool z = t < M && (wv0 >> vb) == 0u;
      const uint64_t zm = __ballot(z);
      if (lane == 0) misc[w] = (uint32_t)__popcll(zm);
      __syncthreads();
      uint32_t zb = 0u, zt = 0u;
#pragma unroll
      for (int k = 0; k < NW; ++k) {
        const uint32_t c = misc[k];
        zb += k < w ? c : 0u;
        zt += c;
      }
      zb += (uint32_t)__popcll(zm & lanemask_lt());  // zero-key words before word t
      if (t < M) {
        if (z) bufB[zb] = wv0;
        else rest[t - zb] = wv0;
      }
      __syncthreads();
      Z = (int)zt;
      Mr = M - Z;
      src = rest;
    }
    int S = 16;  // words padded to a power of two: thread t counts for word t % S
    while (S < Mr) S <<= 1;
    const int G = min(NTH / S, 16);
    const int i = t & (S - 1), g = t / S;
    uint32_t wv = 0u;
    if (g < G && i < Mr) {
      wv = src[i];
      // this group's share [lo, hi): whole 4-word steps except the last share
      const int lo = ((g * Mr) / G) & ~3;
      const int hi = g == G - 1 ? Mr : (((g + 1) * Mr) / G) & ~3;
      uint32_t r = 0u;
      int j = lo;
      for (; j + 16 <= hi; j += 16) {  // four reads in flight per step
        uint4 q[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) q[u] = *reinterpret_cast<const uint4*>(src + j + 4 * u);
#pragma unroll
        for (int u = 0; u < 4; ++u)
          r += (q[u].x < wv ? 1u : 0u) + (q[u].y < wv ? 1u : 0u) + (q[u].z < wv ? 1u : 0u) +
               (q[u].w < wv ? 1u : 0u);
      }
      for (; j + 4 <= hi; j += 4) {
        const uint4 q = *reinterpret_cast<const uint4*>(src + j);
        r += (q.x < wv ? 1u : 0u) + (q.y < wv ? 1u : 0u) + (q.z < wv ? 1u : 0u) +
             (q.w < wv ? 1u : 0u);
      }
      for (; j < hi; ++j) r += src[j] < wv ? 1u : 0u;
      cnt[g * S + i] = r;
    }
    __syncthreads();
    if (g == 0 && i < Mr) {
      uint32_t r = (uint32_t)Z;
      for (int gg = 0; gg < G; ++gg) r += cnt[gg * S + i];
      bufB[r] = wv;
    }
    __syncthreads();
    res = bufB;
  } else {
    res = lds_lsd_passes<NTH>(bufA, bufB, M, plan, vb, rank16, hist, misc);
  }
  const uint32_t vmask = (1u << vb) - 1u;
  for (int i = t; i < M; i += NTH) {
    const uint32_t word = res[i];
    out_keys[off + i] = (int32_t)(((word >> vb) << pb) | (uint32_t)part);
    out_vals[off + i] = (int32_t)(word & vmask);
  }
}

// ------------------------------------------------------------ multi-tile sort
// Lists above kSmallSortN keys: LSD passes of at most 9 bits over tiles of
// 256 * IPT keys, one launch per pass plus one histogram launch.
//   histogram   every workgroup counts the digits of all passes for a share
//               of the keys (LDS) and adds them into the digit totals; it
//               also resets the per-pass tile counters and clears the
//               status words of this call's tiles;
//   pass p      a workgroup takes the next tile id from an atomic counter
//               (so every tile it waits for below is already running),
//               ranks its keys stably in LDS, publishes the tile's digit
//               counts, and finds the keys of each digit in all earlier
//               tiles by looking back over their published counts: a tile
//               publishes its count first and, once its own prefix is
//               known, its inclusive prefix, so a look-back stops at the
//               first prefix it meets.  Two threads per digit read
//               2 * kOsHalf earlier tiles per step, so at these list sizes
//               one round of loads usually finds the prefix.  Keys and entry
//               ids are then scattered to digit start + earlier tiles + rank.
// A look-back that waits implausibly long raises kFlagInternal and stops
// (the update is then voided), so a library bug cannot hang the device.
constexpr uint32_t kOsAgg = 1u;     // status: the tile's own digit count
constexpr uint32_t kOsPrefix = 2u;  // status: inclusive count over tiles 0..tile
constexpr int kOsHistIpt = 16;      // keys per thread of a histogram workgroup
constexpr uint32_t kOsSpinLimit = 1u << 22;
constexpr int kOsHalf = 64;         // earlier tiles read by each thread of a digit per step

struct SortBufs {
  int32_t* keys[2];
  int32_t* vals[2];
  uint32_t* totals;                 // [kMaxPasses][kMaxBins] digit totals
  uint32_t* status;                 // [kMaxPasses][max_tiles][kMaxBins] look-back words:
                                    // flag (2 bits: 0 none, kOsAgg, kOsPrefix) | count (30)
  uint32_t* tile_ctr;               // [kMaxPasses] next tile id of each pass
  int32_t* part_off;                // [partitions + 1] partitioned sort: where each partition starts
  int max_tiles;
  uint32_t* flag;                   // sticky error bits
  int32_t* fresh_status;            // partitioned sort only: see part_sort (null: sticky flag)
};

__device__ __forceinline__ uint32_t os_word(uint32_t fl, uint32_t v) { return (fl << 30) | v; }

constexpr int kOsHistLdsWords = kMaxPasses * kMaxBins;

// Digit totals of every pass over keys [blk*256*kOsHistIpt, ...).
template <class KeyFn>
__device__ void os_hist(const KeyFn& kf, int N, const SortPlan& plan, const SortBufs& sb, int blk,
                        uint32_t* lds) {
  const int t = threadIdx.x;
  if (blk == 0 && t < kMaxPasses) sb.tile_ctr[t] = 0u;
  // the status words of this call's tiles start unpublished
  const size_t rows = (size_t)plan.ntiles * kMaxBins;
  for (int p = 0; p < plan.passes; ++p)
    for (size_t i = (size_t)blk * kBlock + t; i < rows; i += (size_t)gridDim.x * kBlock)
      sb.status[(size_t)p * sb.max_tiles * kMaxBins + i] = 0u;
  for (int i = t; i < plan.passes * kMaxBins; i += kBlock) lds[i] = 0;
  const int base = blk * kBlock * kOsHistIpt;
  uint32_t key[kOsHistIpt];
  load_keys<kOsHistIpt>(kf, N, base + t, kBlock, key, sb.flag);
  __syncthreads();
#pragma unroll
  for (int q = 0; q < kOsHistIpt; ++q) {
    if (base + q * kBlock + t < N) {
      for (int p = 0; p < plan.passes; ++p) {
        const uint32_t dg = (key[q] >> plan.shift[p]) & ((1u << plan.bits[p]) - 1u);
        atomicAdd(&lds[p * kMaxBins + dg], 1u);
      }
    }
  }
  __syncthreads();
  for (int p = 0; p < plan.passes; ++p) {
    const int bins = 1 << plan.bits[p];
    for (int dg = t; dg < bins; dg += kBlock) {
      const uint32_t c = lds[p * kMaxBins + dg];
      if (c) atomicAdd(&sb.totals[p * kMaxBins + dg], c);
    }
  }
}

// One radix pass: a workgroup of kOsThreads threads per tile of R * 1024 keys.
constexpr int kOsThreads = 1024;
constexpr int kOsWaves = kOsThreads / kWave;
// LDS of a pass: counters [kMaxBins][waves + 1], digit bases (the look-back's
// next tile per digit before that), scan scratch, the tile id, and the
// look-back's exchange between the two threads of a digit [2][kMaxBins].
constexpr int kOsPassLdsWords = kMaxBins * (kOsWaves + 1) + kMaxBins + 2 * kOsWaves + 1 + 2 * kMaxBins;
static_assert(kOsThreads == 2 * kMaxBins, "the look-back takes two threads per digit");

template <int R, class KeyFn>
__device__ void os_pass(const KeyFn& kf, int N, const SortPlan& plan, const SortBufs& sb, int p,
                        uint32_t* lds) {
  constexpr int NW = kOsWaves, CS = NW + 1, TK = R * kOsThreads;
  const int t = threadIdx.x, lane = t & (kWave - 1);
  const int w = __builtin_amdgcn_readfirstlane(t / kWave);
  uint32_t* hist = lds;                      // [kMaxBins][CS]: counts, then wave offsets
  uint32_t* base = hist + kMaxBins * CS;     // [kMaxBins] start of the digit's keys of this tile
  uint32_t* misc = base + kMaxBins;          // scan scratch
  uint32_t* tid_s = misc + 2 * NW;
  uint32_t* lb_sum = tid_s + 1;              // [kMaxBins] look-back: upper half's sum
  uint32_t* lb_res = lb_sum + kMaxBins;      // [kMaxBins] ... its outcome and stop tile
  const int bits = plan.bits[p], shift = plan.shift[p], bins = 1 << bits;
  if (t == 0) tid_s[0] = atomicAdd(&sb.tile_ctr[p], 1u);
  // digit total of digit t (complete: written by the histogram launch)
  const uint32_t tot = t < bins ? sb.totals[p * kMaxBins + t] : 0u;
  uint32_t* mycol = hist + w;
  for (int d = lane; d < bins; d += kWave) {
    mycol[d * CS] = 0;
    if (w == 0) hist[d * CS + NW] = 0;
  }
  __syncthreads();
  const int tile = (int)tid_s[0];
  const int32_t* sk = sb.keys[p & 1];
  const int32_t* sv = sb.vals[p & 1];
  int32_t* dk = sb.keys[(p + 1) & 1];
  int32_t* dv = sb.vals[(p + 1) & 1];

  // keys of the tile: wave w owns R rounds of 64 consecutive keys
  uint32_t key[R], dg[R], loc[R];
  int32_t val[R];
  uint64_t act[R];
  const int wbase = tile * TK + w * (R * kWave);
  if (p == 0) {
    load_keys<R>(kf, N, wbase + lane, kWave, key, sb.flag);
#pragma unroll
    for (int r = 0; r < R; ++r) val[r] = wbase + r * kWave + lane;
  } else {
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int i = wbase + r * kWave + lane;
      key[r] = i < N ? (uint32_t)sk[i] : 0u;
      val[r] = i < N ? sv[i] : 0;
    }
  }
#pragma unroll
  for (int r = 0; r < R; ++r) {
    act[r] = __ballot(wbase + r * kWave + lane < N);
    dg[r] = (key[r] >> shift) & (uint32_t)(bins - 1);
  }
  wave_rank<R>(dg, act, R, bits, mycol, loc, CS);
  __syncthreads();
  // thread t < bins: digit t's count in every wave -> the tile's count of the
  // digit, and each wave's offset inside the digit (written back in place)
  const bool mine = t < bins;
  uint32_t cnt = 0u;
  if (mine) {
    uint32_t c[NW];
#pragma unroll
    for (int v = 0; v < NW; ++v) c[v] = hist[t * CS + v];
#pragma unroll
    for (int v = 0; v < NW; ++v) {
      hist[t * CS + v] = cnt;
      cnt += c[v];
    }
  }

  // publish this tile's digit counts, look back over earlier tiles, publish
  // the inclusive prefix.  Digit bd has two threads, h = 0 (thread bd, which
  // holds the count) and h = 1 (thread bd + kMaxBins).  From the digit's next
  // unread tile c, thread h reads tiles c - h*kOsHalf - i, i < kOsHalf, all at
  // once, and adds them nearest first until it meets an inclusive prefix (or
  // the first tile), an unpublished tile, or the end of its range.  Thread
  // h = 0 then combines: its own sum, and the upper half's only if its range
  // held aggregates alone.  An unpublished tile is read again next step.
  uint32_t* st = sb.status + (size_t)p * sb.max_tiles * kMaxBins;
  const int bd = t & (kMaxBins - 1), h = t / kMaxBins;
  int32_t* lb_cur = reinterpret_cast<int32_t*>(base);  // next unread tile per digit, -1: done
  uint32_t excl = 0u;
  if (mine)
    __hip_atomic_store(&st[(size_t)tile * kMaxBins + t], os_word(tile == 0 ? kOsPrefix : kOsAgg, cnt),
                       __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if (h == 0) lb_cur[bd] = (mine && tile > 0) ? tile - 1 : -1;
  __syncthreads();
  for (uint32_t spins = 0;; ++spins) {
    if (spins > kOsSpinLimit) {  // never expected: give up, void the update
      if (t == 0) atomicOr(sb.flag, kFlagInternal);
      break;
    }
    const int c = lb_cur[bd];
    const int top = c - h * kOsHalf;
    uint32_t sw[kOsHalf];
#pragma unroll
    for (int i = 0; i < kOsHalf; ++i)
      sw[i] = (c >= 0 && top - i >= 0)
                  ? __hip_atomic_load(&st[(size_t)(top - i) * kMaxBins + bd], __ATOMIC_RELAXED,
                                      __HIP_MEMORY_SCOPE_AGENT)
                  : 0u;
    // outcome: 0 all aggregates (continue below the range), 1 unpublished
    // tile `stop`, 2 complete (a prefix or the first tile reached)
    uint32_t ps = 0u;
    int res = 0, stop = top - kOsHalf;
#pragma unroll
    for (int i = 0; i < kOsHalf; ++i) {
      if (res != 0) continue;
      if (top - i < 0) {
        res = 2;
        continue;
      }
      const uint32_t fl = sw[i] >> 30;
      if (fl == 0u) {
        res = 1;
        stop = top - i;
        continue;
      }
      ps += sw[i] & 0x3fffffffu;
      if (fl == kOsPrefix) res = 2;
    }
    if (h == 1) {
      lb_sum[bd] = ps;
      lb_res[bd] = (uint32_t)res | ((uint32_t)(stop + 1) << 2);
    }
    __syncthreads();
    bool more = false;
    if (h == 0 && c >= 0) {
      excl += ps;
      int next = res == 2 ? -1 : stop;
      if (res == 0) {  // this range held aggregates only: the upper half counts
        const uint32_t r1 = lb_res[bd];
        excl += lb_sum[bd];
        next = (r1 & 3u) == 2u ? -1 : (int)(r1 >> 2) - 1;
      }
      lb_cur[bd] = next;
      more = next >= 0;
    }
    if (!__syncthreads_or(more)) break;
  }
  if (mine) {
    if (tile > 0)
      __hip_atomic_store(&st[(size_t)tile * kMaxBins + t], os_word(kOsPrefix, excl + cnt),
                         __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  // digit starts of the pass: exclusive scan of the totals over digits
  {
    const uint32_t inc = wave_incl_scan(tot);
    if (lane == kWave - 1) misc[w] = inc;
    __syncthreads();
    uint32_t b = 0;
#pragma unroll
    for (int v = 0; v < NW; ++v) b += v < w ? misc[v] : 0u;
    if (mine) base[t] = b + inc - tot + excl;
  }
  __syncthreads();
#pragma unroll
  for (int r = 0; r < R; ++r) {
    if ((act[r] >> lane) & 1ull) {
      const uint32_t pos = base[dg[r]] + mycol[dg[r] * CS] + loc[r];
      if (pos >= (uint32_t)N) {  // inconsistent counters: never write out of bounds
        atomicOr(sb.flag, kFlagInternal);
        continue;
      }
      dk[pos] = (int32_t)key[r];
      dv[pos] = val[r];
    }
  }
}

}  // namespace pg
