// Segmented sums over entries sorted by table row (the deterministic form of
// the advanced-indexing increment of §4.2/§4.3).
//
// The sorted entry list is cut into chunks of `ch` entries (16 or 64), one
// per wave.  Inside a chunk every maximal run of equal keys ("piece") is
// summed in entry order.  A piece whose segment lies wholly inside the chunk
// is applied to its table row by that wave, the row's only writer.  A
// segment that crosses chunk boundaries (a heavy Zipf row) leaves one partial
// sum per spanned chunk (slot 1: the open last piece of the chunk where the
// segment starts; slot 0: the first piece of every later spanned chunk) and
// its start chunk is appended to a task list; a second launch adds the
// partials in a fixed order and applies the row.  Sums never depend on
// scheduling and no row is written twice, without any inter-workgroup wait.
#pragma once
#include "common.h"

namespace pg {

// Number of consecutive chunks after `chunk` whose first entry has `key`.
__device__ __forceinline__ int seg_count_fwd(const int32_t* sk, int N, int chunk, int32_t key,
                                             int ch) {
  const int lane = lane_id();
  int m = 0;
  for (int base = chunk + 1;; base += kWave) {
    const int y = base + lane;
    const bool eq = ((size_t)y * ch < (size_t)N) && sk[(size_t)y * ch] == key;
    const uint64_t b = __ballot(eq);
    const int run = (~b) ? (__ffsll((unsigned long long)~b) - 1) : kWave;
    m += run;
    if (run < kWave) break;
  }
  return m;
}

// Piece structure of one chunk, computed by the whole wave (lanes < ch).
struct ChunkInfo {
  int i0, nact;
  int32_t key;      // this lane's sorted key (-1 beyond the chunk)
  int32_t ent;      // this lane's entry id
  uint64_t heads;   // lanes that start a piece
  bool cont_first;  // the first piece continues a segment from the previous chunk
  bool open_last;   // the last piece continues into the next chunk
};

__device__ __forceinline__ ChunkInfo chunk_info(const int32_t* __restrict__ sk,
                                                const int32_t* __restrict__ sv, int N, int chunk,
                                                int ch) {
  ChunkInfo ci;
  const int lane = lane_id();
  ci.i0 = chunk * ch;
  ci.nact = min(ch, N - ci.i0);
  const bool act = lane < ci.nact;
  ci.key = act ? sk[ci.i0 + lane] : -1;
  ci.ent = act ? sv[ci.i0 + lane] : 0;
  const int32_t before = (ci.i0 > 0) ? sk[ci.i0 - 1] : -1;
  const int32_t after = (ci.i0 + ch < N) ? sk[ci.i0 + ch] : -2;
  int32_t prev = __shfl_up(ci.key, 1);
  if (lane == 0) prev = before;
  ci.heads = __ballot(act && ci.key != prev);
  const int32_t last_key = __shfl(ci.key, ci.nact - 1);
  ci.cont_first = !(ci.heads & 1ull);
  ci.open_last = (after == last_key);
  return ci;
}

// End (exclusive) of the piece starting at p0.
__device__ __forceinline__ int piece_end(const ChunkInfo& ci, int p0) {
  const uint64_t rest = ci.heads & ~((2ull << p0) - 1ull);
  const int p1 = rest ? (__ffsll((unsigned long long)rest) - 1) : ci.nact;
  return p1 > ci.nact ? ci.nact : p1;
}

// Chunk size of a sorted list of N entries: short chunks spread small
// batches over more waves; long chunks keep partials few for large ones.
__host__ __device__ inline int seg_chunk_size(int N) { return N <= 131072 ? 16 : 64; }

}  // namespace pg
