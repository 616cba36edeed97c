// Segmented row sums over entries sorted by table row: the deterministic
// form of the advanced-indexing increment of §4.2/§4.3,
//   table[key(e)] += alpha * sum of Y[e] over the entries e of that key.
// The training step uses it with Y = the per-entry embedding gradients and
// alpha = -lr; polyglot_scatter_add with the caller's Y and alpha.
//
// The sorted entry list is cut into chunks of CH entries (16 or 32; 64 in the
// partition-wise apply), one per wave.  A wave loads the Y rows of its whole chunk at once (lane = column)
// and walks them with a running sum that closes at each piece end (a
// "piece" is a maximal run of equal keys inside the chunk).  Pieces whose
// segment lies wholly inside the chunk are added to their table rows by that
// wave, the rows' only writer, with one float add per element performed at
// the L2 (no read round trip; one add per element, so the result does not
// depend on scheduling).  Few registers per wave keep every wave of a large
// launch resident at once.
// A segment that crosses chunk boundaries leaves the chunks' open pieces in
// LDS, and one wave of the workgroup closes every segment that stays inside
// the workgroup's chunks.  On the whole list a workgroup takes a range of
// consecutive chunks (seg_apply_range); a segment that crosses ranges (a
// heavy Zipf row) leaves one partial per spanned range (slot 1: the open
// last piece of the range where it starts; slot 0: the first piece of every
// later spanned range); the range where it starts records it in its own slot
// of the segment list (no shared counter), every range it runs through marks
// its slot, and its end range is recorded by key; the fix-up launch adds the
// partials in a fixed order and applies the row.  After a partitioned sort, where no key spans two partitions, one
// workgroup per partition completes every segment itself
// (seg_apply_partition).
// Sums never depend on scheduling, no row is written twice and no wave
// waits on another workgroup.
#pragma once
#include "common.h"

namespace pg {

struct SegArgs {
  float* table;             // [rows][d]
  const float* Y;           // [N][d], row e = entry e
  const int32_t* sk;        // sorted keys [N]
  const int32_t* sv;        // entry ids in sorted order [N]
  float* seg_part;          // [chunks][2][seg_stride]
  int2* long_list;          // [ranges] by range: (range, row) if a segment that crosses
                            // ranges starts in it, (-2, 0) if one segment runs through the
                            // whole range, else (-1, 0); every range writes its slot
  int32_t* seg_end;         // [rows]: end range of a crossing segment, by key
  const uint32_t* flag;     // sticky error bits: nonzero voids the update
  const uint32_t* flag2;    // the error word of this list's sort (a training step's sort
                            // set raises its own word; otherwise the same as flag)
  int N, d, ch, seg_stride;
  int rg;                   // entries per range (NW chunks of one workgroup): the fix-up's slots
  float alpha;
  // completed pieces are added as they close (float atomics), not deferred
  static constexpr bool kDeferred = false;
  static constexpr bool kPacked = false;  // one row per load, not the packed walk
  struct Pre {};
};

// Piece structure of one chunk, computed by the whole wave (lanes < ch).
struct ChunkInfo {
  int i0, nact;
  int32_t key;      // this lane's sorted key (-1 beyond the chunk)
  int32_t ent;      // this lane's entry id (0 beyond the chunk)
  uint64_t heads;   // lanes that start a piece
  int32_t last_key; // key of the chunk's last row
  bool cont_first;  // the first piece continues a segment from the previous chunk
  bool open_last;   // the last piece continues into the next chunk
};

// Entries [i0, min(i0 + ch, end)) of a sorted list that ends at `end`.
__device__ __forceinline__ ChunkInfo chunk_info(const int32_t* __restrict__ sk,
                                                const int32_t* __restrict__ sv, int end, int i0,
                                                int ch) {
  ChunkInfo ci;
  const int lane = lane_id();
  ci.i0 = __builtin_amdgcn_readfirstlane(i0);
  ci.nact = __builtin_amdgcn_readfirstlane(min(ch, end - ci.i0));
  const bool act = lane < ci.nact;
  ci.key = act ? sk[ci.i0 + lane] : -1;
  ci.ent = act ? sv[ci.i0 + lane] : 0;
  // the chunk's structure is wave-uniform: held in scalar registers, so the
  // per-row tests built from it compile to scalar branches
  const int32_t before =
      __builtin_amdgcn_readfirstlane((ci.i0 > 0) ? sk[ci.i0 - 1] : -1);
  const int32_t after =
      __builtin_amdgcn_readfirstlane((ci.i0 + ch < end) ? sk[ci.i0 + ch] : -2);
  int32_t prev = __shfl_up(ci.key, 1);
  if (lane == 0) prev = before;
  const uint64_t hb = __ballot(act && ci.key != prev);
  // (readfirstlane returns int: go through uint32_t so bit 31 does not
  // sign-extend into the high word)
  const uint32_t hlo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)hb);
  const uint32_t hhi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(hb >> 32));
  ci.heads = ((uint64_t)hhi << 32) | (uint64_t)hlo;
  ci.last_key = __builtin_amdgcn_readlane(ci.key, ci.nact - 1);
  ci.cont_first = !(ci.heads & 1ull);
  ci.open_last = (after == ci.last_key);
  return ci;
}

// Nonzero when an earlier launch raised an error that voids this update.
template <class A>
__device__ __forceinline__ uint32_t void_bits(const A& a) {
  return *reinterpret_cast<const volatile uint32_t*>(a.flag) |
         *reinterpret_cast<const volatile uint32_t*>(a.flag2);
}

// Chunk size of a sorted list of N entries: short chunks spread small
// batches over more waves; long chunks keep partials few for large ones.
// Measured on training steps (same box, alternating, 16 -> 32 entries):
// B = 2048 26.5 -> 27.7 us, B = 4096 35.7 -> 35.3, B = 8192 43.6 -> 42.2,
// B = 16,384 58.6 -> 58.9; and 64 -> 32 above 131,072 entries: B = 32,768
// 84.4 -> 83.8 us, B = 65,536 126.9 -> 126.2, stress and the 327,680-entry
// scatter-add unchanged.
__host__ __device__ inline int seg_chunk_size(int N) {
  return (N <= 16384 || (N > 65536 && N <= 131072)) ? 16 : 32;
}
// The general op's typed increments defer their row updates past the walk
// (a load and a store per row, 16 rows per round of loads), so shorter
// chunks on long lists pay off there: fewer rounds and more resident waves
// (bfloat16, 327,680 entries: apply 27 -> 16 us, fix-up 8.6 -> 11.5 us).
__host__ __device__ inline int gen_chunk_size(int N) { return N <= 131072 ? 16 : 32; }

// Where a chunk's open pieces go: the wave's slots in LDS (first piece, last
// piece, and the chunk's flags and keys) for the workgroup to combine.
struct ChunkSink {
  float* first;  // [d] sum of the chunk's first piece when it continues a segment
  float* last;   // [d] sum of the chunk's last piece when it opens one
  int* meta;     // cont_first, open_last, single, first key, last key
};

// Element access of the float32 table: a row's entries are read as floats;
// a completed piece is added with one float atomic per element at the L2
// (lanes past the row end add -0.0, which changes nothing).
__device__ __forceinline__ float seg_load(const SegArgs& a, size_t i) { return a.Y[i]; }
__device__ __forceinline__ void seg_add(const SegArgs& a, size_t i, bool cok, float v) {
  unsafeAtomicAdd(a.table + i, cok ? v : -0.f);
}
// A segment's sum v (alpha applied) added to table element i by the row's
// only writer.
__device__ __forceinline__ void seg_close(const SegArgs& a, size_t i, float v) {
  unsafeAtomicAdd(a.table + i, v);
}

// The walk of argument sets whose rows are 16-bit elements read and written
// two rows per 32-bit word (kPacked; defined with those formats).
template <int CH, class A>
__device__ void seg_walk_packed(const A& a, const ChunkInfo& ci, uint64_t tails, uint64_t complete,
                                int first_tail, bool starts_long, const ChunkSink& sink);

// One wave applies entries [i0, min(i0 + CH, end)) of the sorted list (see
// the file comment).  A is SegArgs or another argument set with the same
// fields and its own seg_load / seg_add.  Returns false, having written
// nothing, when an earlier launch raised an error that voids the update (the
// error words are loaded beside the chunk's keys, so the callers need no
// round trip of their own to test them: every wave of the launch reads the
// same value).
template <int CH, class A>
__device__ bool seg_apply_rows(const A& a, int i0, int end, const ChunkSink& sink) {
  static_assert(CH % 8 == 0 && CH <= kWave, "rows are walked in blocks of 8");
  const int lane = lane_id();
  // the error words (set by earlier launches) are read beside the chunk's
  // keys, and tested before any write
  const uint32_t flag = *a.flag | *a.flag2;
  const ChunkInfo ci = chunk_info(a.sk, a.sv, end, i0, CH);
  if (__builtin_amdgcn_readfirstlane(flag) != 0u) return false;  // a bad id voids the update
  const int nact = ci.nact;
  const uint64_t act = nact >= 64 ? ~0ull : ((1ull << nact) - 1ull);
  // piece ends: the lane before every later head, and the last active lane
  const uint64_t tails = ((ci.heads >> 1) | (1ull << (nact - 1))) & act;
  const int first_tail = __ffsll((unsigned long long)tails) - 1;
  const bool single = first_tail == nact - 1;  // the chunk is one piece
  uint64_t complete = tails;
  if (ci.cont_first) complete &= ~(1ull << first_tail);
  if (ci.open_last) complete &= ~(1ull << (nact - 1));
  const bool starts_long = ci.open_last && !(ci.cont_first && single);
  if (lane == 0) {
    sink.meta[0] = ci.cont_first;
    sink.meta[1] = ci.open_last;
    sink.meta[2] = single;
    sink.meta[3] = ci.key;  // lane 0 holds the first piece's key
    sink.meta[4] = ci.last_key;
  }
  if constexpr (A::kPacked) {
    seg_walk_packed<CH>(a, ci, tails, complete, first_tail, starts_long, sink);
    return true;
  }
  for (int c0 = 0; c0 < a.d; c0 += kWave) {
    const int col = c0 + lane;
    const bool cok = col < a.d;
    // Every lane stays active so that every test below is a wave-uniform
    // scalar branch.  Lanes past the row end (d not a multiple of 64) work on
    // the row's last column and add -0.0 there, which leaves any float
    // unchanged.
    const int colc = cok ? col : a.d - 1;
    // every row of the chunk in flight at once (lane = column), issued
    // without branches: rows past the chunk's end read entry 0's row (lanes
    // beyond nact hold entry 0), whose values no piece uses
    float v[CH];
#pragma unroll
    for (int r = 0; r < CH; ++r) {
      const int ent = __builtin_amdgcn_readlane(ci.ent, r);
      v[r] = seg_load(a, (size_t)ent * a.d + colc);
    }
    // (argument sets whose row update is a load and a store: the first
    // block of old rows in flight beside the entries' rows)
    typename A::Pre pre;
    if constexpr (A::kDeferred) seg_prefetch_rows<CH>(a, ci, complete, colc, pre);
    // running sum in entry order, closed at every piece end (tail);
    // completed pieces go straight to their rows, or (argument sets whose
    // row update is a load and a store) replace their tail row's value and
    // are applied after the walk
    const float alpha = cok ? a.alpha : 0.f;
    float acc = 0.f, first_sum = 0.f, last_sum = 0.f;
#pragma unroll
    for (int r0 = 0; r0 < CH; r0 += 8) {
      // this block's bits, taken from the masks here in scalar registers:
      // the empty asm keeps the compiler from computing every row's
      // condition ahead of the loads and parking them in vector lanes
      uint32_t tw = (uint32_t)(tails >> r0) & 0xffu, cw = (uint32_t)(complete >> r0) & 0xffu;
      int ft = first_tail - r0, lt = nact - 1 - r0;
      asm volatile("" : "+s"(tw), "+s"(cw), "+s"(ft), "+s"(lt));
      if (tw == 0u) {  // no piece ends in these rows
#pragma unroll
        for (int u = 0; u < 8; ++u) acc += v[r0 + u];
      } else {
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          acc += v[r0 + u];
          if ((tw >> u) & 1u) {
            if (u == ft) first_sum = acc;
            if (u == lt) last_sum = acc;
            if ((cw >> u) & 1u) {
              if constexpr (A::kDeferred) {
                v[r0 + u] = alpha * acc;
              } else {
                const int32_t key = __builtin_amdgcn_readlane(ci.key, r0 + u);
                seg_add(a, (size_t)key * a.d + colc, cok, alpha * acc);
              }
            }
            acc = 0.f;
          }
        }
      }
    }
    if constexpr (A::kDeferred) seg_add_rows<CH>(a, ci, complete, v, colc, cok, pre);
    if (cok) {
      if (ci.cont_first) sink.first[col] = first_sum;
      if (starts_long) sink.last[col] = last_sum;
    }
  }
  return true;
}

// Threads of a partition workgroup: 16 waves, so one round covers 1024
// entries in 64-entry chunks.  Lists of at most kPartShortN entries take
// 32-entry chunks instead: more waves share a partition's rows.  Training
// steps, 64 -> 32 (same box, alternating): tiny (192 entries) 11.09 -> 10.59
// us, poly256 (1,536) 13.21 -> 12.82, B = 512 14.85 -> 14.66, B = 768
// (4,608) 16.02 -> 15.82; B = 1024 (6,144) 17.05 -> 17.25 us.
constexpr int kPartApplyThreads = 1024;
constexpr int kPartApplyWaves = kPartApplyThreads / kWave;
constexpr int kPartApplyChunk = 64;
constexpr int kPartShortN = 5120;
// Lists of at most kPartTinyN entries take workgroups of 8 waves instead
// of 16 (poly256 step, 1,536 entries: 12.83 -> 12.65 us, tiny 10.52 ->
// 10.39 us); from B = 768 (4,608 entries) a heavy partition then needs a
// second round of chunks (15.8 -> 17.3 us).
constexpr int kPartTinyN = 2048;
constexpr int kPartShortThreads = 512;
__host__ __device__ constexpr int part_apply_threads(int N) {
  return N <= kPartTinyN ? kPartShortThreads : kPartApplyThreads;
}

// Segmented apply of one partition of a partitioned sort (NW waves per
// workgroup), entries [s, e):
// no key has entries in two partitions, so every segment that crosses a
// chunk is completed inside the workgroup.  Each round, wave w applies
// chunk r0 + w and leaves its open pieces in LDS; after a barrier wave 0
// walks the round's chunks in order, adding the pieces of every crossing
// segment (carried over from earlier rounds when it started there) and
// applying the row once the segment closes.  The order of every sum is
// fixed, so the result does not depend on scheduling.
template <int NW, class A, int PC = kPartApplyChunk>
__device__ void seg_apply_partition(const A& a, int s, int e,
                                    float (*F)[kMaxD], float (*Lp)[kMaxD], int (*meta)[5]) {
  const int t = threadIdx.x, lane = t & (kWave - 1);
  const int w = __builtin_amdgcn_readfirstlane(t / kWave);
  constexpr int CB = kMaxD / kWave;  // column blocks of the widest row
  const int nch = (e - s + PC - 1) / PC;
  float open[CB];                    // wave 0: the segment still open, by column block
  int open_key = 0, open_key_next = 0;
#pragma unroll
  for (int cb = 0; cb < CB; ++cb) open[cb] = 0.f;
  for (int r0 = 0; r0 < nch; r0 += NW) {
    const int c = r0 + w;
    bool ok = true;  // (wave 0 always has a chunk: its own test covers the combine)
    if (c < nch)
      ok = seg_apply_rows<PC>(a, s + c * PC, e,
                                           ChunkSink{F[w], Lp[w], meta[w]});
    __syncthreads();  // the round's open pieces are in LDS
    if (w == 0 && ok) {
      const int nc = min(NW, nch - r0);
      // every chunk's flags and keys at once (lane k reads chunk k), then
      // taken as wave-uniform values
      int mk[5];
#pragma unroll
      for (int x = 0; x < 5; ++x) mk[x] = lane < nc ? meta[lane][x] : 0;
      const uint64_t cfm = __ballot(mk[0] != 0), olm = __ballot(mk[1] != 0),
                     sgm = __ballot(mk[2] != 0);
#pragma unroll
      for (int cb = 0; cb < CB; ++cb) {
        const int col = cb * kWave + lane;
        if (cb * kWave >= a.d) break;
        const bool cok = col < a.d;
        // the round's open pieces of this column block, all reads in flight
        float fv[NW], lv[NW];
#pragma unroll
        for (int k = 0; k < NW; ++k) {
          fv[k] = (k < nc && cok) ? F[k][col] : 0.f;
          lv[k] = (k < nc && cok) ? Lp[k][col] : 0.f;
        }
        float o = open[cb];
        int okey = open_key;
#pragma unroll
        for (int k = 0; k < NW; ++k) {
          if (k >= nc) break;
          const bool cf = (cfm >> k) & 1ull, ol = (olm >> k) & 1ull, sg = (sgm >> k) & 1ull;
          if (cf) {  // the chunk's first piece continues the open segment
            o += fv[k];
            if (!(sg && ol) && cok)  // ... and closes it: apply the row
              seg_close(a, (size_t)okey * a.d + col, a.alpha * o);
          }
          if (ol && !(sg && cf)) {  // the chunk's last piece opens a segment
            o = lv[k];
            okey = __builtin_amdgcn_readlane(mk[4], k);
          }
        }
        open[cb] = o;
        if (cb == 0) open_key_next = okey;
      }
      open_key = open_key_next;
    }
    __syncthreads();  // the slots are reused by the next round
  }
}

// One range of the whole sorted list: NW consecutive chunks of CH entries,
// range r = entries [r*NW*CH, (r+1)*NW*CH), one chunk per wave of the
// workgroup.  The chunks leave their open pieces in LDS; wave 0 walks them in
// order, completing every segment that crosses a chunk boundary inside the
// range, and exports at most two partials, by range, with the meaning a
// chunk's have for the fix-up (seg_fix_row): slot 0 the first piece when it
// continues a segment from an earlier range, slot 1 the last piece when a
// segment starts here and continues into the next range (recorded in the
// range's long_list slot; seg_end[key] = the range where such a segment
// ends).  So segments crossing chunks inside a workgroup never reach the
// fix-up, and a heavy row leaves one partial per range instead of one per
// chunk.  Every sum has a fixed order.  The caller has tested the error flag.
template <int CH, int NW, class A>
__device__ void seg_apply_range(const A& a, int r, float (*F)[kMaxD], float (*Lp)[kMaxD],
                                int (*meta)[5]) {
  const int t = threadIdx.x, lane = t & (kWave - 1);
  const int w = __builtin_amdgcn_readfirstlane(t / kWave);
  const int s = r * NW * CH;
  const int nch = min(NW, (a.N - s + CH - 1) / CH);
  bool ok = true;  // (wave 0 always has a chunk: its own test covers the combine)
  if (w < nch) ok = seg_apply_rows<CH>(a, s + w * CH, a.N, ChunkSink{F[w], Lp[w], meta[w]});
  __syncthreads();  // the chunks' open pieces are in LDS
  if (w == 0 && ok) {
    int mk[5];
#pragma unroll
    for (int x = 0; x < 5; ++x) mk[x] = lane < nch ? meta[lane][x] : 0;
    const uint64_t cfm = __ballot(mk[0] != 0), olm = __ballot(mk[1] != 0),
                   sgm = __ballot(mk[2] != 0);
    const bool cf0 = cfm & 1ull;                      // continues from an earlier range
    const bool olL = (olm >> (nch - 1)) & 1ull;       // continues into the next range
    const int32_t key0 = __builtin_amdgcn_readlane(mk[3], 0);
    bool front_open = cf0;                            // (wave-uniform)
    int32_t okey = 0;
    for (int c0 = 0; c0 < a.d; c0 += kWave) {
      const int col = c0 + lane;
      const bool cok = col < a.d;
      float fv[NW], lv[NW];
#pragma unroll
      for (int k = 0; k < NW; ++k) {
        fv[k] = (k < nch && cok) ? F[k][col] : 0.f;
        lv[k] = (k < nch && cok) ? Lp[k][col] : 0.f;
      }
      float o = 0.f, first = 0.f;
      bool front = cf0;
      int32_t ok = 0;
#pragma unroll
      for (int k = 0; k < NW; ++k) {
        if (k >= nch) break;
        const bool cf = (cfm >> k) & 1ull, ol = (olm >> k) & 1ull, sg = (sgm >> k) & 1ull;
        if (cf) {  // the chunk's first piece continues the open segment
          o += fv[k];
          if (!(sg && ol)) {  // ... and closes it
            if (front) {
              first = o;  // the segment from an earlier range ends here
              front = false;
            } else if (cok) {
              seg_close(a, (size_t)ok * a.d + col, a.alpha * o);
            }
          }
        }
        if (ol && !(sg && cf)) {  // the chunk's last piece opens a segment
          o = lv[k];
          ok = __builtin_amdgcn_readlane(mk[4], k);
          front = false;
        }
      }
      // the range's exports (front: the segment from an earlier range spans
      // the whole range; it is then slot 0 and the range records nothing)
      if (cok) {
        if (cf0) a.seg_part[((size_t)r * 2 + 0) * a.seg_stride + col] = front ? o : first;
        if (olL && !front) a.seg_part[((size_t)r * 2 + 1) * a.seg_stride + col] = o;
      }
      front_open = front;
      okey = ok;
    }
    if (lane == 0) {
      const bool starts_long = olL && !front_open;
      const bool middle = cf0 && olL && front_open;  // one segment runs through the range
      a.long_list[r] = starts_long ? make_int2(r, okey) : make_int2(middle ? -2 : -1, 0);
      if (cf0 && !(olL && front_open)) a.seg_end[key0] = r;
    }
  }
  __syncthreads();  // the slots are reused by the workgroup's next range
}

// Fix-up workgroups: each takes kSegfixWaves crossing segments at a time,
// one per wave; a segment with more than kSegfixLight partials (a heavy Zipf
// row) is summed by the whole workgroup instead.
constexpr int kSegfixThreads = 512;
constexpr int kSegfixWaves = kSegfixThreads / kWave;
constexpr int kSegfixUnroll = 16;
constexpr int kSegfixLight = 16;

// Row access of the fix-up, four consecutive columns at element i of the
// table (n of them inside the row; the float32 table has d % 4 == 0 and
// aligned rows, so n is 4 or 0): read as floats, written back.
__device__ __forceinline__ f4 seg_row4(const SegArgs& a, size_t i, int n) {
  return n > 0 ? ld4(a.table + i) : kZero4;
}
__device__ __forceinline__ void seg_put4(const SegArgs& a, size_t i, int n, f4 v) {
  if (n > 0) st4(a.table + i, v);
}
// A crossing segment's sum v (alpha applied) added to the row by its only
// writer: float adds at the L2 (no read round trip; the same rounding as the
// row's load, add and store).
__device__ __forceinline__ void seg_add4(const SegArgs& a, size_t i, int n, f4 v) {
  if (n > 0) {
#pragma unroll
    for (int k = 0; k < 4; ++k) unsafeAtomicAdd(a.table + i + k, v[k]);
  }
}

// One wave takes range slot li of nchunks, the number of ranges (the
// partial slots).  Lane k reads slot li + k
// (k < kSegfixLight) and lane group gq = lane/16 the candidate partials gq,
// gq+4, ... of a segment starting at li, all in one round of loads together
// with the error words; the slots after li say where such a segment ends (a
// run of middle ranges, then its end range), so m, its number of partials,
// needs no second round.  A segment of at most kSegfixLight partials is
// finished here: each lane sums four consecutive columns of its group's
// partials in order, the four group sums meet by a fixed butterfly, and the
// row takes the sum (seg_add4: float32 adds at the L2, else a load and a
// store).  Returns 0 (no segment starts at li, or the update is void), m, or
// kSegfixLight + 1 for a heavier segment, which the caller hands to the
// whole workgroup with *key_out set.  Partial rows are read four columns at a
// time up to the next multiple of 4 (inside the partial slot's stride); the
// row access masks the columns past d.
template <class A>
__device__ int seg_fix_slot_wave(const A& a, int li, int nchunks, int32_t* key_out) {
  const int lane = lane_id(), q = lane & 15, gq = lane >> 4;
  const int2 rec = (lane < kSegfixLight && li + lane < nchunks) ? a.long_list[li + lane]
                                                                 : make_int2(-1, 0);
  const uint32_t flag = *a.flag | *a.flag2;
  f4 x[kSegfixLight / 4];
  {
    const int col = 4 * q;
    const bool cok = col < a.d;
#pragma unroll
    for (int u = 0; u < kSegfixLight / 4; ++u) {
      const int i = 4 * u + gq;
      const size_t slot = i == 0 ? (size_t)li * 2 + 1 : (size_t)(li + i) * 2;
      x[u] = (li + i < nchunks && cok) ? ld4(a.seg_part + slot * a.seg_stride + col) : kZero4;
    }
  }
  const int cs = __builtin_amdgcn_readlane(rec.x, 0);
  if (cs < 0 || __builtin_amdgcn_readfirstlane(flag) != 0u) return 0;
  const int32_t key = __builtin_amdgcn_readlane(rec.y, 0);
  // the end range: the first slot after li that is not a middle range
  const uint64_t ends = __ballot(lane >= 1 && lane < kSegfixLight && rec.x != -2);
  if (ends == 0ull) {
    *key_out = key;
    return kSegfixLight + 1;
  }
  const int m = __ffsll((unsigned long long)ends);  // end slot j = m - 1
  for (int c0 = 0; c0 < a.d; c0 += 64) {
    const int col = c0 + 4 * q;
    const bool cok = col < a.d;
    const size_t tr = (size_t)key * a.d + col;
    const int nrow = (gq == 0 && cok) ? min(4, a.d - col) : 0;
    if (c0 > 0) {
#pragma unroll
      for (int u = 0; u < kSegfixLight / 4; ++u) {
        const int i = 4 * u + gq;
        const size_t slot = i == 0 ? (size_t)cs * 2 + 1 : (size_t)(cs + i) * 2;
        x[u] = (i < m && cok) ? ld4(a.seg_part + slot * a.seg_stride + col) : kZero4;
      }
    }
    f4 acc = kZero4;
#pragma unroll
    for (int u = 0; u < kSegfixLight / 4; ++u)
      if (4 * u + gq < m) acc += x[u];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      acc[k] += __shfl_xor(acc[k], 16);
      acc[k] += __shfl_xor(acc[k], 32);
    }
    seg_add4(a, tr, nrow, a.alpha * acc);
  }
  return m;
}

// The whole workgroup adds the m partials of crossing segment (cs, key) and
// applies its row.  Lane group gq = lane/16 of wave w takes partials
// i = G*u + 4*w + gq, G = 4 * waves (i = 0 is the open piece of the start
// chunk, i >= 1 the first piece of chunk cs+i), each lane four consecutive
// columns; group sums are combined by a fixed butterfly and the wave sums in
// wave order, so the result is independent of scheduling.
template <class A>
__device__ void seg_fix_row(const A& a, int cs, int32_t key, int m,
                            float* red /* [waves][kMaxD] */) {
  const int t = threadIdx.x, lane = t & (kWave - 1);
  const int w = __builtin_amdgcn_readfirstlane(t / kWave);
  const int q = lane & 15, gq = lane >> 4;
  constexpr int G = kSegfixWaves * 4;     // lane groups per workgroup
  for (int c0 = 0; c0 < a.d; c0 += 64) {
    const int col = c0 + 4 * q;
    const bool cok = col < a.d;
    const size_t tr = (size_t)key * a.d + col;
    const bool owner = w == 0 && gq == 0 && cok;
    const int nrow = owner ? min(4, a.d - col) : 0;
    // a table whose row update is a load and a store: the row in flight
    // beside the partials (float32 rows take the sum at the L2 instead)
    f4 row = kZero4;
    if constexpr (A::kDeferred) row = seg_row4(a, tr, nrow);
    f4 acc = kZero4;
    for (int base = 0; base < m; base += G * kSegfixUnroll) {
      f4 x[kSegfixUnroll];
#pragma unroll
      for (int u = 0; u < kSegfixUnroll; ++u) {
        const int i = base + u * G + w * 4 + gq;
        const size_t slot = i == 0 ? (size_t)cs * 2 + 1 : (size_t)(cs + i) * 2;
        x[u] = (i < m && cok) ? ld4(a.seg_part + slot * a.seg_stride + col) : kZero4;
      }
#pragma unroll
      for (int u = 0; u < kSegfixUnroll; ++u) acc += x[u];
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      acc[k] += __shfl_xor(acc[k], 16);
      acc[k] += __shfl_xor(acc[k], 32);
    }
    __syncthreads();  // red of the previous column block is no longer read
    if (gq == 0) st4(red + w * kMaxD + 4 * q, acc);
    __syncthreads();
    if (owner) {
      f4 s = ld4(red + 4 * q);
#pragma unroll
      for (int v = 1; v < kSegfixWaves; ++v) s += ld4(red + v * kMaxD + 4 * q);
      if constexpr (A::kDeferred) seg_put4(a, tr, nrow, row + a.alpha * s);
      else seg_add4(a, tr, nrow, a.alpha * s);
    }
  }
}

}  // namespace pg
