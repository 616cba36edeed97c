// Bucketed sort of mid-size entry lists (kSmallSortN < N <= kBkMaxN): the
// grouping of (row id, entry) pairs by row id that the segmented form of the
// §4.2/§4.3 increment needs, in two launches with no look-back between
// workgroups.
//
// What the consumers need is weaker than a sorted list: entries with equal
// keys contiguous and in entry order (the order of the increments, which fixes
// the float summation order); the order between distinct keys is free.  So
// the keys are cut into buckets:
//   * a dedicated bucket for each key below kBkDedicated.  Word ids are ranked
//     by frequency (Zipf), so these are the heavy rows: one bucket holds one
//     key and needs no ordering, only copying;
//   * kBkHashed buckets for the other keys, by their low 9 bits above
//     kBkDedicated; such a bucket holds many light keys (a few hundred entries
//     at the batch sizes of the step) and is ordered by the rest of the key.
//
//   k_bk_tiles    tile t (kBkTileKeys consecutive entries) ranks its keys by
//                 bucket in LDS (stable: entry order within a bucket), writes
//                 them grouped by bucket into the tile's slice of the staging
//                 buffers, writes one word per (bucket, tile) -- the bucket's
//                 offset inside the tile and its count -- and adds its counts
//                 into the bucket totals;
//   k_bk_buckets  every workgroup scans the totals (bucket starts) and the
//                 per-bucket work units; a unit is kBkUnit entries of a
//                 dedicated bucket (copied: the tile runs are already in
//                 entry order) or a whole hashed bucket, whose runs are
//                 gathered into LDS and ranked by the rest of the key
//                 (stable), then written at the bucket's start.
// A hashed bucket above kBkCap entries (heavy keys that are not small ids)
// is ordered by its own workgroup in stable 8-bit passes through global
// memory, ping-ponging between its output slice and its own runs in the
// staging buffers (nobody else reads them).
#pragma once
#include "common.h"
#include "sort_dev.h"

namespace pg {

constexpr int kBkDedicated = 64;                    // keys with a bucket of their own
constexpr int kBkHashBits = 9;
constexpr int kBkHashed = 1 << kBkHashBits;         // buckets of the other keys
constexpr int kBkBuckets = kBkDedicated + kBkHashed;
constexpr int kBkDigitBits = 10;                    // bucket ids fit 10 bits
static_assert(kBkBuckets <= (1 << kBkDigitBits), "bucket ids");
constexpr int kBkScanN = 1024;                      // padded length of the per-bucket scans
constexpr int kBkThreads = 512;                     // k_bk_tiles workgroup
// keys per tile: 1536 (214 tiles of the 327,680-entry list, more CUs than
// 160 of 2048) measured faster than 2048 from B = 4096 up (B = 16,384 step
// 59.9 -> 58.4-59.4 us, B = 32,768 85.8 -> 84.0 us) and the same on the
// 327,680-entry scatter-add; 1024 slowed the bucket launch, which reads one
// word per tile for each bucket
constexpr int kBkTileKeys = 1536;
constexpr int kBkMaxTiles = 512;
constexpr int kBkMaxN = kBkTileKeys * kBkMaxTiles;  // 786,432
constexpr int kBkMaxKeyBits = 30;                   // hashed words pack (key >> 9) and 11 index bits
constexpr int kBkSortThreads = 512;                 // k_bk_buckets workgroup
constexpr int kBkUnit = 2048;                       // entries per unit of a dedicated bucket
constexpr int kBkCap = 2048;                        // largest hashed bucket ordered in LDS
constexpr int kBkIdxBits = 11;                      // bits of an index below kBkCap
static_assert((1 << kBkIdxBits) == kBkCap, "index bits");
static_assert(kBkMaxTiles <= kBkSortThreads && 2 * kBkSortThreads >= kBkScanN, "scan sizes");

__host__ __device__ inline int bk_tiles(int N) { return ceil_div(N, kBkTileKeys); }
// Workgroups of k_bk_buckets: every hashed bucket, every dedicated bucket, and
// one more per kBkUnit entries (units beyond the real count leave at once).
__host__ __device__ inline int bk_grid(int N) { return kBkBuckets + ceil_div(N, kBkUnit); }

__device__ __forceinline__ uint32_t bk_bucket(uint32_t key) {
  return key < (uint32_t)kBkDedicated
             ? key
             : (uint32_t)kBkDedicated + ((key - kBkDedicated) & (uint32_t)(kBkHashed - 1));
}
// the order of a key inside its hashed bucket
__device__ __forceinline__ uint32_t bk_high(uint32_t key) {
  return (key - kBkDedicated) >> kBkHashBits;
}

// ------------------------------------------------------------------ tiles
// LDS of bk_tiles for NTH threads, in words.
__host__ __device__ constexpr int bk_tiles_lds_words(int nth) {
  return kBkBuckets * (nth / kWave + 1) + kBkScanN + 32;
}

// Tile `tile` of the list, by a workgroup of NTH threads (R = 2048 / NTH
// rounds of 64 keys per wave).
template <int NTH, class KeyFn>
__device__ void bk_tiles(const KeyFn& kf, int N, int ntiles, const SortBufs& sb, int tile,
                         uint32_t* lds) {
  constexpr int NW = NTH / kWave, CS = NW + 1, R = kBkTileKeys / NTH, P = kBkBuckets;
  static_assert(R * NTH == kBkTileKeys && NW + 1 <= 32, "tile shape");
  uint32_t* hist = lds;                 // [P][CS]: per-wave counts, then wave offsets
  uint32_t* loff = hist + P * CS;       // [kBkScanN]: counts, then offsets inside the tile
  uint32_t* misc = loff + kBkScanN;     // scan scratch
  const int t = threadIdx.x, lane = t & (kWave - 1);
  const int w = __builtin_amdgcn_readfirstlane(t / kWave);
  for (int i = t; i < P * CS; i += NTH) hist[i] = 0u;
  const int wbase = tile * kBkTileKeys + w * (R * kWave);
  uint32_t key[R], dg[R], loc[R];
  uint64_t act[R];
  load_keys<R>(kf, N, wbase + lane, kWave, key, sb.flag);
#pragma unroll
  for (int r = 0; r < R; ++r) {
    act[r] = __ballot(wbase + r * kWave + lane < N);
    dg[r] = bk_bucket(key[r]);
  }
  __syncthreads();
  wave_rank<R>(dg, act, R, kBkDigitBits, hist + w, loc, CS);
  __syncthreads();
  // bucket d: the tile's count and each wave's offset inside the bucket
  constexpr int DPT = kBkScanN / NTH;  // buckets per thread
  uint32_t cnt[DPT];
#pragma unroll
  for (int k = 0; k < DPT; ++k) {
    cnt[k] = 0u;
    const int d = t + k * NTH;
    if (d < P) {
      uint32_t c[NW];
#pragma unroll
      for (int v = 0; v < NW; ++v) c[v] = hist[d * CS + v];
#pragma unroll
      for (int v = 0; v < NW; ++v) {
        hist[d * CS + v] = cnt[k];
        cnt[k] += c[v];
      }
    }
    if (d < kBkScanN) loff[d] = cnt[k];
  }
  __syncthreads();
  block_exclusive_scan_runs<NTH>(loff, kBkScanN, misc);
  uint32_t* col = sb.status;  // [P][ntiles]: (offset inside the tile << 16) | count
#pragma unroll
  for (int k = 0; k < DPT; ++k) {
    const int d = t + k * NTH;
    if (d < P) {
      col[(size_t)d * ntiles + tile] = (loff[d] << 16) | cnt[k];
      if (cnt[k]) atomicAdd(&sb.totals[d], cnt[k]);
    }
  }
  int32_t* tk = sb.keys[0] + (size_t)tile * kBkTileKeys;
  int32_t* tv = sb.vals[0] + (size_t)tile * kBkTileKeys;
#pragma unroll
  for (int r = 0; r < R; ++r) {
    if ((act[r] >> lane) & 1ull) {
      const uint32_t pos = loff[dg[r]] + hist[dg[r] * CS + w] + loc[r];
      tk[pos] = (int32_t)key[r];
      tv[pos] = wbase + r * kWave + lane;
    }
  }
}

// ---------------------------------------------------------------- buckets
// LDS of k_bk_buckets, in words.
constexpr int kBkLdsTot = 0;                              // [kBkScanN] bucket starts
constexpr int kBkLdsUni = kBkLdsTot + kBkScanN;           // [kBkScanN] unit starts
constexpr int kBkLdsRun = kBkLdsUni + kBkScanN;           // [kBkScanN] run starts in the bucket
constexpr int kBkLdsOff = kBkLdsRun + kBkScanN;           // [kBkMaxTiles] run offsets in the tiles
constexpr int kBkLdsMisc = kBkLdsOff + kBkMaxTiles;       // [kPartSortMisc] scan scratch
constexpr int kBkLdsSort = kBkLdsMisc + kPartSortMisc;    // sort area
constexpr int kBkSortNW = kBkSortThreads / kWave;
constexpr int kBkLdsDigit = 8;   // digit of the LDS counting passes
constexpr int kBkRankMax = 192;  // hashed buckets up to this size are ranked by counting
// sort area: bufA, bufB [kBkCap], rank16 [kBkCap / 2], ent [kBkCap], hist [256][NW+1]
constexpr int kBkLdsSortWords =
    3 * kBkCap + kBkCap / 2 + (1 << kBkLdsDigit) * (kBkSortNW + 1);
static_assert(kBkRankMax <= kBkSortThreads, "one thread per word");
// the oversize path's counters [256][NW+1] and digit bases [256] alias the sort area
static_assert(256 * (kBkSortNW + 1) + 256 <= kBkLdsSortWords, "oversize counters");
constexpr int kBkLdsWords = kBkLdsSort + kBkLdsSortWords;

// Largest i in [0, n) with a[i] <= x (a non-decreasing, a[0] <= x).
__device__ __forceinline__ int bk_floor(const uint32_t* a, int n, uint32_t x) {
  int lo = 0, hi = n;  // answer in [lo, hi)
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (a[mid] <= x) lo = mid; else hi = mid;
  }
  return lo;
}

// One stable 8-bit pass of the oversize path over the M entries of a hashed
// bucket: position i of the source is src_out ? out[i] : the i-th entry of the
// bucket's tile runs, and likewise for the destination.
template <class Loc>
__device__ void bk_stream_pass(const Loc& loc, int M, int shift, bool src_out, uint32_t* cnt,
                               uint32_t* base, uint32_t* misc) {
  constexpr int NW = kBkSortNW, CS = NW + 1, RR = 4, RW = RR * kWave;
  const int t = threadIdx.x, lane = t & (kWave - 1);
  const int w = __builtin_amdgcn_readfirstlane(t / kWave);
  // digit totals, one LDS add per distinct digit of a wave's 64 keys
  if (t < 256) base[t] = 0u;
  __syncthreads();
  for (int i0 = w * kWave; i0 < M; i0 += kBkSortThreads) {
    const int i = i0 + lane;
    const bool ok = i < M;
    const uint32_t dg = ok ? (bk_high((uint32_t)loc.key(i, src_out)) >> shift) & 255u : 0u;
    const uint64_t peers = match_digit(dg, 8, __ballot(ok));
    if (ok && __popcll(peers & lanemask_lt()) == 0) atomicAdd(&base[dg], (uint32_t)__popcll(peers));
  }
  __syncthreads();
  {  // exclusive scan of the 256 totals (threads 0..127 take two each)
    uint32_t* v = base;
    block_exclusive_scan<kBkSortThreads>(v, 256, misc);
  }
  for (int r0 = 0; r0 < M; r0 += NW * RW) {
    for (int d = lane; d < 256; d += kWave) cnt[d * CS + w] = 0u;
    __syncthreads();
    uint32_t key[RR], dg[RR], rk[RR];
    int32_t val[RR];
    uint64_t act[RR];
    const int wb = r0 + w * RW;
#pragma unroll
    for (int r = 0; r < RR; ++r) {
      const int i = wb + r * kWave + lane;
      const bool ok = i < M;
      key[r] = ok ? (uint32_t)loc.key(i, src_out) : 0u;
      val[r] = ok ? loc.val(i, src_out) : 0;
      act[r] = __ballot(ok);
      dg[r] = (bk_high(key[r]) >> shift) & 255u;
    }
    wave_rank<RR>(dg, act, RR, 8, cnt + w, rk, CS);
    __syncthreads();
    if (t < 256) {  // offsets of each wave's keys of digit t in this round
      uint32_t run = base[t];
#pragma unroll
      for (int v = 0; v < NW; ++v) {
        const uint32_t c = cnt[t * CS + v];
        cnt[t * CS + v] = run;
        run += c;
      }
      base[t] = run;
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < RR; ++r) {
      if ((act[r] >> lane) & 1ull) {
        const uint32_t pos = cnt[dg[r] * CS + w] + rk[r];
        if (pos < (uint32_t)M) loc.put(pos, !src_out, key[r], val[r]);  // always, by the counts
      }
    }
    __syncthreads();  // the counters are cleared by the next round
  }
}

// Positions of one bucket: i < M is out[start + i] or the i-th entry of the
// bucket's runs in the staging buffers.
struct BkLoc {
  int32_t* ok;          // output keys + start
  int32_t* ov;
  int32_t* tk;          // staging keys / entry ids
  int32_t* tv;
  const uint32_t* run;  // [ntiles] run starts inside the bucket
  const uint32_t* off;  // [ntiles] run offsets inside the tiles
  int ntiles;
  __device__ size_t stage(int i) const {
    const int tt = bk_floor(run, ntiles, (uint32_t)i);
    return (size_t)tt * kBkTileKeys + off[tt] + ((uint32_t)i - run[tt]);
  }
  __device__ int32_t key(int i, bool out) const { return out ? ok[i] : tk[stage(i)]; }
  __device__ int32_t val(int i, bool out) const { return out ? ov[i] : tv[stage(i)]; }
  __device__ void put(uint32_t i, bool out, uint32_t k, int32_t v) const {
    if (out) {
      ok[i] = (int32_t)k;
      ov[i] = v;
    } else {
      const size_t s = stage((int)i);
      tk[s] = (int32_t)k;
      tv[s] = v;
    }
  }
};

// Workgroup j < kBkHashed orders hashed bucket kBkDedicated + j (known before
// any load, so its column of (offset, count) words is read beside the
// totals); the others copy the units of the dedicated buckets in order.
__device__ void bk_buckets(int N, int ntiles, int key_bits, const SortBufs& sb, uint32_t j,
                           uint32_t* lds) {
  constexpr int NTH = kBkSortThreads, P = kBkBuckets;
  uint32_t* tot = lds + kBkLdsTot;
  uint32_t* uni = lds + kBkLdsUni;
  uint32_t* run = lds + kBkLdsRun;
  uint32_t* off = lds + kBkLdsOff;
  uint32_t* misc = lds + kBkLdsMisc;
  uint32_t* sa = lds + kBkLdsSort;
  const int t = threadIdx.x;
  const bool hashed = j < (uint32_t)kBkHashed;
  int b = kBkDedicated + (int)j;
  // bucket totals (and a hashed bucket's column), every load in flight at once
  {
    const uint32_t* col = sb.status + (size_t)b * ntiles;
    uint32_t m[2], cw = 0u;
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      const int d = t + k * NTH;
      m[k] = d < P ? sb.totals[d] : 0u;
    }
    if (hashed && t < ntiles) cw = col[t];
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      const int d = t + k * NTH;
      tot[d] = m[k];
      uni[d] = (d < kBkDedicated && m[k]) ? (m[k] + kBkUnit - 1) / kBkUnit : 0u;
      run[d] = (hashed && d == t && t < ntiles) ? (cw & 0xffffu) : 0u;
    }
    if (hashed && t < ntiles) off[t] = cw >> 16;
  }
  __syncthreads();
  block_exclusive_scan<NTH>(tot, kBkScanN, misc);
  uint32_t sub = 0u;
  if (hashed) {
    block_exclusive_scan<NTH>(run, kBkScanN, misc);
  } else {
    block_exclusive_scan<NTH>(uni, kBkScanN, misc);
    const uint32_t u = j - (uint32_t)kBkHashed;
    if (u >= uni[kBkDedicated]) return;  // past the last unit (uniform over the workgroup)
    b = bk_floor(uni, kBkDedicated, u);
    sub = u - uni[b];
  }
  const uint32_t start = tot[b], M = tot[b + 1] - start;
  if (start + M > (uint32_t)N || tot[P] != (uint32_t)N) {  // inconsistent counters: a library bug
    if (t == 0) atomicOr(sb.flag, kFlagInternal);
    return;
  }
  if (M == 0u) return;
  if (!hashed) {  // the dedicated bucket's run in every tile
    const uint32_t* col = sb.status + (size_t)b * ntiles;
    for (int tt = t; tt < kBkScanN; tt += NTH) {
      const uint32_t wv = tt < ntiles ? col[tt] : 0u;
      run[tt] = wv & 0xffffu;
      if (tt < ntiles) off[tt] = wv >> 16;
    }
    __syncthreads();
    block_exclusive_scan<NTH>(run, kBkScanN, misc);
  }
  const BkLoc loc{sb.keys[1] + start, sb.vals[1] + start, sb.keys[0], sb.vals[0], run, off, ntiles};

  if (!hashed) {  // one key: copy this unit's entries, already in entry order
    const uint32_t lo = sub * kBkUnit, hi = min(M, lo + (uint32_t)kBkUnit);
    constexpr int U = kBkUnit / NTH;
    int32_t v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint32_t i = lo + t + u * NTH;
      v[u] = i < hi ? loc.tv[loc.stage((int)i)] : 0;
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint32_t i = lo + t + u * NTH;
      if (i < hi) {
        loc.ok[i] = b;
        loc.ov[i] = v[u];
      }
    }
    return;
  }

  if (M > (uint32_t)kBkCap) {
    const int hb = max(0, key_bits - kBkHashBits);  // bits of bk_high  // oversize: stable 8-bit passes through global memory
    uint32_t* cnt = sa;                               // [256][NW + 1]
    uint32_t* base = sa + 256 * (kBkSortNW + 1);      // [256]
    const int np = (hb + 7) / 8;
    // the result must end in the output slice: an even number of passes
    // starts there (after a copy), an odd number starts in the runs
    bool in_out = false;
    if (np % 2 == 0) {
      for (int i = t; i < (int)M; i += NTH) loc.put((uint32_t)i, true, loc.key(i, false), loc.val(i, false));
      __syncthreads();
      in_out = true;
    }
    for (int p = 0; p < np; ++p) {
      bk_stream_pass(loc, (int)M, 8 * p, in_out, cnt, base, misc);
      in_out = !in_out;
    }
    return;
  }

  // hashed bucket in LDS: words (order, index in the bucket), distinct
  uint32_t* bufA = sa;
  uint32_t* bufB = bufA + kBkCap;
  uint16_t* rank16 = reinterpret_cast<uint16_t*>(bufB + kBkCap);
  uint32_t* ent = bufB + kBkCap + kBkCap / 2;
  uint32_t* hist = ent + kBkCap;
  for (int i = t; i < (int)M; i += NTH) {
    const size_t s = loc.stage(i);
    const uint32_t k = (uint32_t)loc.tk[s];
    ent[i] = (uint32_t)loc.tv[s];
    bufA[i] = (bk_high(k) << kBkIdxBits) | (uint32_t)i;
  }
  for (int i = (int)M + t; i < ((int)M + 15) / 16 * 16; i += NTH) bufA[i] = 0xffffffffu;  // pad
  __syncthreads();
  const uint32_t* res;
  if (M <= (uint32_t)kBkRankMax) {
    // a word's place is the number of smaller words: one thread per word,
    // broadcast reads of sixteen words per step (the order of the stable
    // radix passes, without their scans)
    if (t < (int)M) {
      const uint32_t wv = bufA[t];
      uint32_t r = 0u;
      for (int q = 0; q < (int)M; q += 16) {
        uint4 x[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) x[u] = *reinterpret_cast<const uint4*>(bufA + q + 4 * u);
#pragma unroll
        for (int u = 0; u < 4; ++u)
          r += (x[u].x < wv ? 1u : 0u) + (x[u].y < wv ? 1u : 0u) + (x[u].z < wv ? 1u : 0u) +
               (x[u].w < wv ? 1u : 0u);
      }
      bufB[r] = wv;
    }
    __syncthreads();
    res = bufB;
  } else {  // stable LDS counting passes of up to 8 bits (one pass below 2^17 rows)
    const int hb = max(0, key_bits - kBkHashBits);  // bits of bk_high
    SortPlan lp{};
    lp.passes = (hb + kBkLdsDigit - 1) / kBkLdsDigit;
    int sh = 0;
    for (int p = 0; p < lp.passes; ++p) {
      lp.bits[p] = hb / lp.passes + (p < hb % lp.passes ? 1 : 0);
      lp.shift[p] = sh;
      sh += lp.bits[p];
    }
    res = lds_lsd_passes<NTH>(bufA, bufB, (int)M, lp, kBkIdxBits, rank16, hist, misc);
  }
  const uint32_t low = (uint32_t)(b - kBkDedicated);
  for (int i = t; i < (int)M; i += NTH) {
    const uint32_t wv = res[i];
    loc.ok[i] = (int32_t)((uint32_t)kBkDedicated + (((wv >> kBkIdxBits) << kBkHashBits) | low));
    loc.ov[i] = (int32_t)ent[wv & (uint32_t)(kBkCap - 1)];
  }
}

}  // namespace pg
