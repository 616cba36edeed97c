// Fused gather + forward + hinge + backward for compile-time shapes, one
// workgroup of 16 waves per group of consecutive 16-window tiles (16x16x4 f32
// MFMA), ending in the per-entry embedding gradient rows G.
//
// Per tile of 16 windows (rows r), with V = dz + dz~, dz or dz~ (per window,
// H values each):
//   X         the tile's embedding rows -- positions 0..win-1 and the
//             corrupt row as position win -- staged in LDS once, laid out
//             [position][column quad][window] so that both MFMA operand
//             layouts read it without bank conflicts; the rows of tile k+1
//             are loaded into registers while tile k computes, and the ids
//             of tile k+2 are loaded at the same time;
//   forward   Z = X W1^T: wave w takes hidden block nt = w % NT and the
//             K-chunks kc = w / NT + (16 / NT) i; the corrupted copy only
//             differs in block c, so z~ = z - zctr + zcor (§1 model, x~);
//   epilogue  tanh, both scores, hinge mask, dz, dz~ and their sum; a lane
//             of waves 0-7 takes one hidden unit of one row;
//   dW1       dW1 += V^T X for the wave's (nt, chunks), held in registers
//             across the workgroup's tiles and written once as its partial;
//   G         G[e][:] = W1_j^T V for entry e = b(win+1) + j: context
//             positions take dz + dz~, the true centre dz, the corrupt entry
//             (j = win) dz~ through block c; 16x16 output tiles (position,
//             16 columns) round-robin over the waves.
// W1 is staged once per workgroup in LDS (row stride K + 4 floats, rows
// >= H zero) and read from there as the B operand of the forward and of G.
// Small batches (one tile per workgroup, CUs to spare) split the backward:
// two workgroups take the same tile, both run the forward and the epilogue,
// and each computes half of the dW1 and G output tiles, writing its own
// dense-partial slot.
// Three forms (FORM): 0, tiles one after another, three barriers each (a
// workgroup with one tile); 1, tiles software-pipelined, two barriers each,
// dW1 and G of one tile sharing a phase with the forward of the next; 2,
// tiles in pairs, four barriers per pair: each phase holds the work of both
// tiles (two independent MFMA chains per wave, and every wave busy in the
// epilogue), at the price of a single X buffer.
#pragma once
#include <type_traits>

#include "common.h"
#include "launch.h"

namespace pg {

__device__ __forceinline__ f4 mfma16x4(float a, float b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

template <int D, int WIN, int NT, int TP>
struct F8Shape {
  static constexpr int HP = NT * 16;         // hidden units, padded
  static constexpr int K = D * WIN;          // window vector length
  static constexpr int C = WIN / 2;          // centre position
  static constexpr int W1P = WIN + 1;        // positions incl. the corrupt row
  static constexpr int DQ = D / 16;          // 16-column chunks per row
  static constexpr int QD = D / 4;           // column quads per row
  static constexpr int NCH = K / 16;         // K-chunks
  static constexpr int KW = kF8Waves / NT;   // dW1: waves per hidden block
  static constexpr int CPW = (NCH + KW - 1) / KW;  // dW1: chunks per wave
  static constexpr int KWF = kF8Waves / (TP * NT);  // forward: waves per output tile
  static constexpr int CPWF = (NCH + KWF - 1) / KWF;  // forward: chunks per wave
  static constexpr int NGT = W1P * DQ;       // G output tiles per 16-window tile
  static constexpr int GPW = (TP * NGT + kF8Waves - 1) / kF8Waves;  // G tiles per wave
  static constexpr int XF1 = W1P * QD * kTileRows;  // float4 pieces of X per tile
  static constexpr int XF4 = TP * XF1;              // ... per group of TP tiles
  static constexpr int XPT = (XF4 + kF8Threads - 1) / kF8Threads;  // pieces per thread
  static constexpr int S = K + 4;            // W1 row stride in LDS
  static constexpr int NXB = TP == 1 ? 2 : 1;  // X buffers
  // LDS, in floats
  static constexpr int kW1 = HP * S;
  static constexpr int kX = XF4 * 4;                       // one X buffer
  static constexpr int kZp = kF8Waves * 3 * 4 * kWave;     // forward split-K partials
  static constexpr int kVt = TP * 3 * kTileRows * (HP + 1);
  static constexpr int kRed = kF8Waves * (2 * HP + 2);
  static constexpr int kLds = kW1 + NXB * kX + kZp + kVt + kRed;
  static_assert(D % 16 == 0 && WIN % 2 == 1 && kF8Waves % (TP * NT) == 0, "shape");
  static_assert(kLds * 4 <= 160 * 1024, "LDS of one workgroup");
  static_assert(HP <= 32, "one hidden unit per lane of each 32-lane row half");
};

template <int D, int WIN, int NT, int FORM, int NH>
__device__ void fwdbwd8_wg(const FwdArgs& a, int wg, float* lds) {
  constexpr int TP = FORM == 2 ? 2 : 1;  // tiles per phase
  using Sh = F8Shape<D, WIN, NT, TP>;
  constexpr int HP = Sh::HP, K = Sh::K, C = Sh::C, W1P = Sh::W1P, DQ = Sh::DQ, QD = Sh::QD;
  constexpr int NCH = Sh::NCH, CPW = Sh::CPW, NGT = Sh::NGT, GPW = Sh::GPW;
  constexpr int KWF = Sh::KWF, CPWF = Sh::CPWF;
  constexpr int XF1 = Sh::XF1, XF4 = Sh::XF4, XPT = Sh::XPT, S = Sh::S;
  const int t = threadIdx.x, lane = t & (kWave - 1);
  const int w = __builtin_amdgcn_readfirstlane(t / kWave);  // wave-uniform
  const int n16 = lane & 15, g = lane >> 4;
  // forward: this wave's output tile otf (tile otf / NT of the group, hidden
  // block otf % NT) and chunk set kqf
  const int otf = w % (TP * NT), kqf = w / (TP * NT);
  const int tpf = otf / NT, ntf = otf % NT;

  float* w1s = lds;                       // [HP][K+4]
  float* xl = w1s + Sh::kW1;              // [NXB][TP][W1P][QD][16] float4
  float* zp = xl + Sh::NXB * Sh::kX;      // [kqf][3][otf][4][64]
  float* vt = zp + Sh::kZp;               // [TP][3][16][HP+1]
  float* red = vt + Sh::kVt;              // [waves][2*HP+2]

  // Split backward (NH == 2): workgroups 2q and 2q+1 take the same
  // tiles, both run the forward and the epilogue, and half h = wg & 1 takes
  // every second dW1 output tile and every second G output tile (linear
  // indices L = 2 (w + 16 i) + h); each writes its own partial slot, and the
  // db1 / dw2 / loss sums come from half 0 only.
  static_assert(NH == 1 || (NH == 2 && FORM == 0), "the split takes single-tile workgroups");
  constexpr int nh = NH;
  const int h = wg & (nh - 1);
  const int tile0 = (wg / nh) * a.tiles_per_wg;
  // dW1 output tiles L = kc NT + nt of this wave: L = nh (w + 16 i) + h, all
  // in hidden block ntd
  constexpr int NLT = NCH * NT;
  const int ntd = (nh * w + h) % NT;
  const int ntl = min(a.tiles_per_wg, a.ntiles - tile0);  // tiles of this workgroup (>= 1)

  // ids of the X pieces of this thread in the group of TP tiles starting at
  // `tile`: piece pi = t + 1024 p covers tile pi / XF1 of the group and,
  // with q = pi % XF1, window r = q % 16, column quad (q / 16) % QD,
  // position q / (16 QD) (position win: the corrupt id).  Rows >= B read
  // row 0.  The loads are only issued here: the range check waits for them,
  // so it sits in load_x, where the rows' addresses need the ids anyway.
  auto load_ids = [&](int tile, int32_t (&id)[XPT]) {
#pragma unroll
    for (int p = 0; p < XPT; ++p) {
      const int pi = t + kF8Threads * p;
      const int tp = pi / XF1, q = pi - tp * XF1;
      const int r = q % kTileRows, j = q / (kTileRows * QD);
      const int b = (tile + tp) * kTileRows + r;
      id[p] = 0;
      if (pi < XF4 && b < a.B) id[p] = (j < WIN) ? a.windows[(size_t)b * WIN + j] : a.corrupt[b];
    }
  };
  // the rows of one tile into registers; an id outside [0, V) reads row 0
  // and raises the flag (after every load is issued)
  auto load_x = [&](const int32_t (&id)[XPT], f4 (&xr)[XPT]) {
    bool bad = false;
#pragma unroll
    for (int p = 0; p < XPT; ++p) {
      const int pi = t + kF8Threads * p;
      const int qq = ((pi % XF1) / kTileRows) % QD;
      const bool bk = (uint32_t)id[p] >= (uint32_t)a.V;
      bad |= bk;
      xr[p] = pi < XF4 ? ld4(a.E + (size_t)(bk ? 0 : id[p]) * D + 4 * qq) : kZero4;
    }
    if (bad) atomicOr(a.flag, kFlagBadId);
  };
  auto store_x = [&](int buf, const f4 (&xr)[XPT]) {
#pragma unroll
    for (int p = 0; p < XPT; ++p) {
      const int pi = t + kF8Threads * p;
      if (pi < XF4) st4(xl + buf * Sh::kX + 4 * pi, xr[p]);
    }
  };
  // ---- prologue: ids of the first tile, W1 and the first tile's rows in
  // flight together (the rows wait only for the ids), then the ids of the
  // second tile
  int32_t ids[2][XPT];
  f4 xr[XPT];
  load_ids(tile0, ids[0]);
  {  // W1 into LDS (rows >= H zero); loads batched before the stores
    constexpr int N4 = HP * (K / 4);
    constexpr int U = (N4 + kF8Threads - 1) / kF8Threads;
    f4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i = u * kF8Threads + t;
      const int n = i / (K / 4), k4 = i - n * (K / 4);
      v[u] = (i < N4 && n < a.H) ? ld4(a.W1 + (size_t)n * K + 4 * k4) : kZero4;
    }
    load_x(ids[0], xr);
    if (ntl > TP) load_ids(tile0 + TP, ids[1]);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i = u * kF8Threads + t;
      const int n = i / (K / 4), k4 = i - n * (K / 4);
      if (i < N4) st4(w1s + n * S + 4 * k4, v[u]);
    }
  }
  // epilogue lane map: hidden unit hn = lane % 32 of row 2w + lane / 32
  const int hn = lane & 31, rsel = lane >> 5;
  const float b1v = hn < a.H ? a.b1[hn] : 0.f;
  const float w2v = hn < a.H ? a.w2[hn] : 0.f;
  const float b2v = a.b2[0];

  f4 accW[CPW];
#pragma unroll
  for (int ci = 0; ci < CPW; ++ci) accW[ci] = kZero4;
  float db1a = 0.f, dw2a = 0.f, lossa = 0.f;

  // ---- forward of the tiles in X: split-K partials into zp
  auto forward = [&](const float* Xg) {
    // ---- forward: wave (otf, kqf) over chunks kc = kqf + KWF ci; common
    // blocks, true centre and corrupt centre accumulate separately
    const float* X = Xg + 4 * XF1 * tpf;
    f4 zc = kZero4, zctr = kZero4, zcor = kZero4;
#pragma unroll
    for (int ci = 0; ci < CPWF; ++ci) {
      const int kc = kqf + KWF * ci;
      if (kc < NCH) {
        const int j = kc / DQ, qq = 4 * (kc % DQ) + g;
        const f4 xa = ld4(X + 4 * ((j * QD + qq) * kTileRows + n16));
        const f4 wb = ld4(w1s + (ntf * 16 + n16) * S + kc * 16 + 4 * g);
        if (j != C) {
#pragma unroll
          for (int q = 0; q < 4; ++q) zc = mfma16x4(xa[q], wb[q], zc);
        } else {
          const f4 xt = ld4(X + 4 * ((WIN * QD + qq) * kTileRows + n16));
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            zctr = mfma16x4(xa[q], wb[q], zctr);
            zcor = mfma16x4(xt[q], wb[q], zcor);
          }
        }
      }
    }
    // partials [kqf][type][otf][component][lane] (component-major: a
    // reader of one component of every lane touches consecutive words)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      zp[(((kqf * 3 + 0) * (TP * NT) + otf) * 4 + i) * kWave + lane] = zc[i];
      zp[(((kqf * 3 + 1) * (TP * NT) + otf) * 4 + i) * kWave + lane] = zctr[i];
      zp[(((kqf * 3 + 2) * (TP * NT) + otf) * 4 + i) * kWave + lane] = zcor[i];
    }
  };
  // ---- epilogue of the tiles starting at row0: zp -> V (vt) and the
  // accumulators
  auto epilogue = [&](int row0) {
    // ---- epilogue: lane (hn, rsel) of wave w < 8 TP takes hidden unit hn of
    // row 2w + rsel of the group (tile tp = r / 16, row rr = r % 16 in it)
    if (w < TP * kTileRows / 2) {
      const int r = 2 * w + rsel;
      const int row = row0 + r;
      const int tp = r / kTileRows, rr = r % kTileRows;
      const int ot = tp * NT + (hn >> 4), src = (hn & 15) + 16 * (rr >> 2), comp = rr & 3;
      float Zc = 0.f, Zctr = 0.f, Zcor = 0.f;
      if (hn < HP) {
#pragma unroll
        for (int v = 0; v < KWF; ++v) {
          Zc += zp[(((v * 3 + 0) * (TP * NT) + ot) * 4 + comp) * kWave + src];
          Zctr += zp[(((v * 3 + 1) * (TP * NT) + ot) * 4 + comp) * kWave + src];
          Zcor += zp[(((v * 3 + 2) * (TP * NT) + ot) * 4 + comp) * kWave + src];
        }
      }
      const float z = b1v + (Zc + Zctr);
      const float zt = b1v + (Zc + Zcor);
      const float h = tanh_fast(z), ht = tanh_fast(zt);
      // h - h~ = tanh(z - z~) (1 - h h~), z - z~ = zctr - zcor without
      // cancellation against the common part
      const float hmh = tanh_fast(Zctr - Zcor) * (1.f - h * ht);
      float ps = w2v * h, pst = w2v * ht;
#pragma unroll
      for (int o = 1; o < 32; o <<= 1) {
        ps += __shfl_xor(ps, o);
        pst += __shfl_xor(pst, o);
      }
      const float mg = 1.f - (b2v + ps) + (b2v + pst);
      const bool on = row < a.B && mg > 0.f;  // hinge active (derivative 0 at margin 0)
      const float gst = on ? a.invB : 0.f;    // d loss/d s~ = m/B, d loss/d s = -m/B
      const float gw = gst * w2v;
      const float dz = -gw * (1.f - h * h);
      const float dzt = gw * (1.f - ht * ht);
      const float dsum = gw * hmh * (h + ht);  // dz + dz~ = g w2 (h - h~)(h + h~)
      if (hn < HP) {
        vt[((tp * 3 + 0) * kTileRows + rr) * (HP + 1) + hn] = dsum;
        vt[((tp * 3 + 1) * kTileRows + rr) * (HP + 1) + hn] = dz;
        vt[((tp * 3 + 2) * kTileRows + rr) * (HP + 1) + hn] = dzt;
      }
      db1a += dsum;
      dw2a -= gst * hmh;  // -(m/B) h + (m/B) h~
      if (hn == 0) lossa += on ? mg : 0.f;
    }
  };
  // ---- dW1 and G of the tiles in X starting at row0 (reads vt)
  auto backward = [&](const float* Xg, int row0) {
    // ---- dW1 += V^T X for this wave's output tiles (block ntd, chunks kc),
    // the group's tiles in order.  A operand: lane (n16, g) holds
    // V[4ii+g][ntd*16 + n16]; B operand: X[4ii+g][16kc + n16].
#pragma unroll
    for (int tp = 0; tp < TP; ++tp) {
      const float* X = Xg + 4 * XF1 * tp;
      float vc[3][4];
#pragma unroll
      for (int ty = 0; ty < 3; ++ty)
#pragma unroll
        for (int ii = 0; ii < 4; ++ii)
          vc[ty][ii] = vt[((tp * 3 + ty) * kTileRows + 4 * ii + g) * (HP + 1) + ntd * 16 + n16];
#pragma unroll
      for (int ci = 0; ci < CPW; ++ci) {
        const int L = nh * (w + kF8Waves * ci) + h;
        if (L < NLT) {
          const int kc = L / NT;
          const int j = kc / DQ, qq = 4 * (kc % DQ) + (n16 >> 2);
#pragma unroll
          for (int ii = 0; ii < 4; ++ii) {
            const float xb = X[4 * ((j * QD + qq) * kTileRows + 4 * ii + g) + (n16 & 3)];
            if (j != C) {
              accW[ci] = mfma16x4(vc[0][ii], xb, accW[ci]);
            } else {
              const float xc = X[4 * ((WIN * QD + qq) * kTileRows + 4 * ii + g) + (n16 & 3)];
              accW[ci] = mfma16x4(vc[1][ii], xb, accW[ci]);
              accW[ci] = mfma16x4(vc[2][ii], xc, accW[ci]);
            }
          }
        }
      }
    }

    // ---- G: output tiles ot = nh (w + 16u) + h of the group (tile
    // ot / NGT, position j = (ot % NGT) / DQ, columns cb*16).
    // A operand: lane (r = n16, g) holds V_ty[r][4q + g]; B operand: lane
    // (col = n16, g) holds W1[4q + g][jj*D + cb*16 + col].
#pragma unroll
    for (int u = 0; u < GPW; ++u) {
      const int ot = nh * (w + kF8Waves * u) + h;
      if (ot < TP * NGT) {
        const int tp = ot / NGT, o = ot - tp * NGT;
        const int j = o / DQ, cb = o - (o / DQ) * DQ;
        const int ty = (j == WIN) ? 2 : (j == C ? 1 : 0);
        const int jj = (j == WIN) ? C : j;
        f4 acc = kZero4;
#pragma unroll
        for (int q = 0; q < HP / 4; ++q) {
          const float av = vt[((tp * 3 + ty) * kTileRows + n16) * (HP + 1) + 4 * q + g];
          const float bv = w1s[(4 * q + g) * S + jj * D + cb * 16 + n16];
          acc = mfma16x4(av, bv, acc);
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int row = row0 + tp * kTileRows + 4 * g + i;
          if (row < a.B) __builtin_nontemporal_store(acc[i], &a.G[((size_t)row * W1P + j) * D + cb * 16 + n16]);
        }
      }
    }
  };

  if constexpr (FORM == 0) {
    // Tiles one after another, three barriers each (X staged, forward
    // partials, V).  Used when a workgroup has a single tile: the pipelined
    // form measured 0.3 us slower there.
    for (int tt = 0; tt < ntl; ++tt) {
      const int tile = tile0 + tt;
      const int buf = tt & 1;
      const float* X = xl + buf * Sh::kX;
      store_x(buf, xr);
      __syncthreads();  // X of this tile (and W1) staged
      if (tt + 1 < ntl) {
        load_x(ids[(tt + 1) & 1], xr);                      // rows of the next tile
        if (tt + 2 < ntl) load_ids(tile + 2, ids[tt & 1]);  // ids two tiles ahead
      }
      forward(X);
      __syncthreads();  // forward partials written
      epilogue(tile * kTileRows);
      __syncthreads();  // V written
      backward(X, tile * kTileRows);
    }
  } else if constexpr (FORM == 2) {
    // Pairs of tiles, four barriers per pair (X staged, forward partials, V,
    // and the end of the pair's dW1 before the next pair's rows overwrite
    // the single X buffer).  tiles_per_wg is even, so the second tile of a
    // pair is this workgroup's, or past the last tile (rows >= B).
    const int ng = (ntl + 1) / 2;
    for (int gi = 0; gi < ng; ++gi) {
      const int row0 = (tile0 + 2 * gi) * kTileRows;
      store_x(0, xr);
      __syncthreads();  // X of this pair (and W1) staged
      if (gi + 1 < ng) {
        load_x(ids[(gi + 1) & 1], xr);                                // rows of the next pair
        if (gi + 2 < ng) load_ids(tile0 + 2 * (gi + 2), ids[gi & 1]);  // ids two pairs ahead
      }
      forward(xl);
      __syncthreads();  // forward partials written
      epilogue(row0);
      __syncthreads();  // V written
      backward(xl, row0);
      if (gi + 1 < ng) __syncthreads();  // X and vt free (uniform branch)
    }
  } else {
    // Software pipeline, two barriers per tile: the epilogue of tile t runs
    // beside the staging of tile t+1's rows (into the other X buffer), then
    // dW1 and G of tile t run in one phase with the forward of tile t+1.
    // Between a buffer's last reader and its next writer there is always a
    // barrier: zp (forward t+1 after the epilogue of t), vt (epilogue t+1
    // after dW1/G of t), X[t&1] (rows of t+2 after dW1 of t).
    store_x(0, xr);
    if (ntl > 1) {
      load_x(ids[1], xr);                                  // rows of tile 1
      if (ntl > 2) load_ids(tile0 + 2, ids[0]);            // ids of tile 2
    }
    __syncthreads();  // X of tile 0 and W1 staged
    forward(xl);
    __syncthreads();  // forward partials of tile 0 written
    for (int tt = 0; tt < ntl; ++tt) {
      const int row0 = (tile0 + tt) * kTileRows;
      epilogue(row0);
      if (tt + 1 < ntl) {
        store_x((tt + 1) & 1, xr);                         // rows of tile tt+1
        if (tt + 2 < ntl) {
          load_x(ids[tt & 1], xr);                         // rows of tile tt+2
          if (tt + 3 < ntl) load_ids(tile0 + tt + 3, ids[(tt + 1) & 1]);
        }
      }
      __syncthreads();  // V of tile tt and X of tile tt+1 written
      backward(xl + (tt & 1) * Sh::kX, row0);
      if (tt + 1 < ntl) {  // (uniform: every wave takes the same branch)
        forward(xl + ((tt + 1) & 1) * Sh::kX);
        __syncthreads();  // forward partials of tile tt+1 written; vt, X[tt&1] free
      }
    }
  }

  // ---- this workgroup's partial of the dense gradients (streaming stores,
  // like the G rows above: the next kernel reads them once).  Slot layout:
  // dW1 [Hp][K], db1 [Hp], dw2 [Hp], loss, db2.
  float* P = a.part + (size_t)wg * a.part_stride;
#pragma unroll
  for (int ci = 0; ci < CPW; ++ci) {
    const int L = nh * (w + kF8Waves * ci) + h;
    if (L < NLT) {
      const int kc = L / NT;
#pragma unroll
      for (int i = 0; i < 4; ++i) __builtin_nontemporal_store(accW[ci][i], &P[(ntd * 16 + 4 * g + i) * K + kc * 16 + n16]);
    }
  }
  // db1, dw2 (per hidden unit: the two row halves of the wave, then the
  // waves in order), loss (one value per wave); db2 is identically 0 (both
  // scores share b2)
  db1a += __shfl_xor(db1a, 32);
  dw2a += __shfl_xor(dw2a, 32);
  for (int o = 1; o < kWave; o <<= 1) lossa += __shfl_xor(lossa, o);
  float* rw = red + w * (2 * HP + 2);
  if (rsel == 0 && hn < HP) {
    rw[hn] = db1a;
    rw[HP + hn] = dw2a;
  }
  if (lane == 0) {
    rw[2 * HP] = lossa;
    rw[2 * HP + 1] = 0.f;
  }
  __syncthreads();
  if (w == 0 && h == 0) {
    for (int e = lane; e < 2 * HP + 2; e += kWave) {
      float s = red[e];
#pragma unroll
      for (int v = 1; v < kF8Waves; ++v) s += red[v * (2 * HP + 2) + e];
      P[HP * K + e] = s;
    }
  }
}

// ---------------------------------------------------------------------------
// Role-specialised form for workgroups with many tiles (hidden layer of 32
// units, NT = 2), 12 waves per workgroup.  The other forms keep all 16 waves
// in step, so the epilogue (tanh, scores, shuffles: vector-ALU work) never
// overlaps the matrix work.  Here the waves take roles:
//   waves 0-3    staging and epilogue: the ids and rows of later tiles, the
//                X tile into LDS, and the epilogue of tile k-1 (a lane per
//                hidden unit of two rows);
//   waves 4-7    forward of tile k: output block nt = (w-4) / 2, the K-half
//                kh = (w-4) % 2 of the chunks, W1 operands held in
//                registers for the whole launch;
//   waves 8-11   dW1 of tile k-2: output block nt = (w-8) / 2, chunk half
//                (w-8) % 2, accumulated in registers across the tiles;
//   waves 4-11   G of tile k-2, 16x16 output tiles (four per forward wave,
//                two per dW1 wave), their W1 operands held in registers too.
// Each SIMD thus runs a staging/epilogue wave beside two matrix waves, with
// the registers of three waves per SIMD (the register-resident operands do
// not fit four).
// One barrier per phase: phase p runs forward(p), epilogue(p-1) and
// dW1/G(p-2), with four X buffers (a tile's rows are written in phase k-1,
// read by the forward in phase k and by dW1 in phase k+2) and two buffers
// each of the split-K partials and of V.  W1 is not in LDS at all.  The X
// tile is stored by column, [position][column][window] with the 16 windows
// of a column padded to XS = 20 floats: a dW1 lane reads the four windows
// its MFMA steps need in one 128-bit read (the contraction runs over the
// windows in the order 4g + step, on both operands), and the forward's
// operand reads (four columns of one window) and the staging stores are
// 32-bit accesses on 64 distinct banks.
template <int D, int WIN>
struct F8WsShape {
  static constexpr int NT = 2, HP = 32, K = D * WIN, C = WIN / 2, W1P = WIN + 1;
  static constexpr int DQ = D / 16, QD = D / 4, NCH = K / 16;
  static constexpr int NE = 4;                       // staging / epilogue waves
  static constexpr int NW = 12;                      // waves per workgroup
  static constexpr int NTH = NW * kWave;
  static_assert(NTH == kF8WsThreads, "launch shape");
  static constexpr int CF = NCH / 2;                 // chunks per forward or dW1 wave
  static constexpr int NGT = W1P * DQ;               // G output tiles per tile
  static constexpr int XF1 = W1P * QD * kTileRows;   // float4 pieces of X per tile
  static constexpr int XPE = (XF1 + NE * kWave - 1) / (NE * kWave);  // per staging lane
  static constexpr int XS = kTileRows + 4;           // floats per column of an X tile
  static constexpr int kX = W1P * D * XS;            // one X buffer, floats
  static constexpr int kZp = 2 * 3 * NT * 4 * kWave; // one partial buffer: [kh][type][nt][4][64]
  static constexpr int kVt = 3 * kTileRows * (HP + 1);
  static constexpr int kRed = NE * (2 * HP + 2);
  static constexpr int kLds = 4 * kX + 2 * kZp + 2 * kVt + kRed;
  static_assert(NCH % 2 == 0 && D % 16 == 0 && WIN % 2 == 1, "shape");
  static_assert(kLds * 4 <= 160 * 1024, "LDS of one workgroup");
};

template <int D, int WIN>
__device__ void fwdbwd8_ws(const FwdArgs& a, int wg, float* lds) {
  using Sh = F8WsShape<D, WIN>;
  constexpr int NT = Sh::NT, HP = Sh::HP, K = Sh::K, C = Sh::C, W1P = Sh::W1P, DQ = Sh::DQ;
  constexpr int QD = Sh::QD, NE = Sh::NE, CF = Sh::CF, NGT = Sh::NGT;
  constexpr int XF1 = Sh::XF1, XPE = Sh::XPE, XS = Sh::XS;
  const int t = threadIdx.x, lane = t & (kWave - 1);
  const int w = __builtin_amdgcn_readfirstlane(t / kWave);  // wave-uniform
  const bool stager = w < NE;
  float* xl = lds;                                 // [4][W1P][D][XS]
  float* zp = xl + 4 * Sh::kX;                     // [2][kh][3][nt][4][64]
  float* vt = zp + 2 * Sh::kZp;                    // [2][3][16][HP+1]
  float* red = vt + 2 * Sh::kVt;                   // [NE][2*HP+2]
  const int tile0 = wg * a.tiles_per_wg;
  const int ntl = min(a.tiles_per_wg, a.ntiles - tile0);

  // staging lanes: piece pi = t + 256 p of a tile covers window pi % 16,
  // column quad (pi / 16) % QD, position pi / (16 QD); rows >= B read row 0
  auto load_ids = [&](int tile, int32_t (&id)[XPE]) {
#pragma unroll
    for (int p = 0; p < XPE; ++p) {
      const int pi = t + NE * kWave * p;
      const int r = pi % kTileRows, j = pi / (kTileRows * QD);
      const int b = tile * kTileRows + r;
      id[p] = 0;
      if (pi < XF1 && b < a.B) id[p] = (j < WIN) ? a.windows[(size_t)b * WIN + j] : a.corrupt[b];
    }
  };
  auto load_x = [&](const int32_t (&id)[XPE], f4 (&xr)[XPE]) {
    bool bad = false;
#pragma unroll
    for (int p = 0; p < XPE; ++p) {
      const int pi = t + NE * kWave * p;
      const int qq = (pi / kTileRows) % QD;
      const bool bk = (uint32_t)id[p] >= (uint32_t)a.V;
      bad |= bk;
      xr[p] = pi < XF1 ? ld4(a.E + (size_t)(bk ? 0 : id[p]) * D + 4 * qq) : kZero4;
    }
    if (bad) atomicOr(a.flag, kFlagBadId);
  };
  // piece pi (window r, column quad qq, position j) to its four columns
  auto store_x = [&](int buf, const f4 (&xr)[XPE]) {
#pragma unroll
    for (int p = 0; p < XPE; ++p) {
      const int pi = t + NE * kWave * p;
      const int r = pi % kTileRows, qq = (pi / kTileRows) % QD, j = pi / (kTileRows * QD);
      float* dst = xl + buf * Sh::kX + (j * D + 4 * qq) * XS + r;
      if (pi < XF1) {
#pragma unroll
        for (int c = 0; c < 4; ++c) dst[c * XS] = xr[p][c];
      }
    }
  };

  // Registers of the matrix waves.  rr: the forward waves' W1 operands (lane
  // (n16, g) holds W1[nt*16 + n16][16kc + 4g .. +3] for its chunks kc =
  // kh*CF + c), the dW1 waves' accumulators.  wg1: the G operands of the
  // wave's G output tiles (lane (n16, g) holds W1[4q + g][jj*D + cb*16 + n16]
  // at step q).
  f4 rr[CF];
  // G tiles: four per forward wave, two per dW1 wave (the dW1 waves carry
  // more of the rest: measured 0.4 us per step faster than three each)
  constexpr int GF = (NGT * 2 / 3 + 3) / 4, GD = (NGT - 4 * GF + 3) / 4;
  constexpr int GM = GF > GD ? GF : GD;
  float wg1[GM][HP / 4];
#pragma unroll
  for (int c = 0; c < CF; ++c) rr[c] = kZero4;
#pragma unroll
  for (int u = 0; u < GM; ++u)
#pragma unroll
    for (int q = 0; q < HP / 4; ++q) wg1[u][q] = 0.f;

  // The work of matrix wave MI = w - NE (a compile-time constant, so that
  // every operand offset is an immediate): stage 0 loads its W1 operands;
  // stage 1 runs phase p (forward of tile p for MI < 4; dW1 of tile p-2 for
  // MI >= 4; G of tile p-2 for all).
  auto matrix = [&](auto mic, int stage, int p, int n16, int g) {
    constexpr int MI = decltype(mic)::value;
    constexpr int nt = (MI & 3) >> 1, kh = MI & 1;
    constexpr bool FWD = MI < 4;
    if (stage == 0) {
      if constexpr (FWD) {
        const int n = nt * 16 + n16;
#pragma unroll
        for (int c = 0; c < CF; ++c)
          rr[c] = n < a.H ? ld4(a.W1 + (size_t)n * K + (kh * CF + c) * 16 + 4 * g) : kZero4;
      }
#pragma unroll
      for (int u = 0; u < (FWD ? GF : GD); ++u) {
        const int ot = FWD ? MI + 4 * u : 4 * GF + (MI - 4) + 4 * u;
        if (ot < NGT) {
          const int j = ot / DQ, cb = ot % DQ, jj = (j == WIN) ? C : j;
#pragma unroll
          for (int q = 0; q < HP / 4; ++q) {
            const int k = 4 * q + g;
            wg1[u][q] = k < a.H ? a.W1[(size_t)k * K + jj * D + cb * 16 + n16] : 0.f;
          }
        }
      }
      return;
    }
    if constexpr (FWD) {
      if (p < ntl) {
        // ---- forward of tile p: split-K partials of half kh into zp[p % 2]
        const float* X = xl + (p & 3) * Sh::kX;
        f4 zc = kZero4, zctr = kZero4, zcor = kZero4;
#pragma unroll
        for (int c = 0; c < CF; ++c) {
          __builtin_amdgcn_sched_barrier(0);  // one chunk's operands in flight at a time
          const int kc = kh * CF + c;
          const int j = kc / DQ, col = 16 * (kc % DQ) + 4 * g;
          // A operand: X[window n16][col + q], four columns of one window
          float xa[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) xa[q] = X[(j * D + col + q) * XS + n16];
          if (j != C) {
#pragma unroll
            for (int q = 0; q < 4; ++q) zc = mfma16x4(xa[q], rr[c][q], zc);
          } else {
            float xt[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) xt[q] = X[(WIN * D + col + q) * XS + n16];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              zctr = mfma16x4(xa[q], rr[c][q], zctr);
              zcor = mfma16x4(xt[q], rr[c][q], zcor);
            }
          }
        }
        float* Z = zp + (p & 1) * Sh::kZp;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          Z[(((kh * 3 + 0) * NT + nt) * 4 + i) * kWave + lane] = zc[i];
          Z[(((kh * 3 + 1) * NT + nt) * 4 + i) * kWave + lane] = zctr[i];
          Z[(((kh * 3 + 2) * NT + nt) * 4 + i) * kWave + lane] = zcor[i];
        }
      }
    }
    if (p >= 2) {
      const int q2 = p - 2;  // the tile whose backward runs now
      const float* X = xl + (q2 & 3) * Sh::kX;
      const float* V = vt + (q2 & 1) * Sh::kVt;
      const int row0 = (tile0 + q2) * kTileRows;
      if constexpr (!FWD) {
        // ---- dW1 += V^T X for block nt, chunks kc = kh*CF + c, over the
        // windows in the order 4g + ii.  A operand: lane (n16, g) holds
        // V[4g+ii][nt*16 + n16]; B operand: X[4g+ii][16kc + n16], the four
        // of a lane from one 128-bit read.
        float vc[3][4];
#pragma unroll
        for (int ty = 0; ty < 3; ++ty)
#pragma unroll
          for (int ii = 0; ii < 4; ++ii)
            vc[ty][ii] = V[(ty * kTileRows + 4 * g + ii) * (HP + 1) + nt * 16 + n16];
#pragma unroll
        for (int c = 0; c < CF; ++c) {
          __builtin_amdgcn_sched_barrier(0);
          const int kc = kh * CF + c;
          const int j = kc / DQ, col = 16 * (kc % DQ) + n16;
          const f4 xb = ld4(X + (j * D + col) * XS + 4 * g);
          if (j != C) {
#pragma unroll
            for (int ii = 0; ii < 4; ++ii) rr[c] = mfma16x4(vc[0][ii], xb[ii], rr[c]);
          } else {
            const f4 xc = ld4(X + (WIN * D + col) * XS + 4 * g);
#pragma unroll
            for (int ii = 0; ii < 4; ++ii) {
              rr[c] = mfma16x4(vc[1][ii], xb[ii], rr[c]);
              rr[c] = mfma16x4(vc[2][ii], xc[ii], rr[c]);
            }
          }
        }
      }
      // ---- G: this wave's output tiles ot (position j = ot / DQ, columns
      // cb*16).  A operand: lane (r = n16, g) holds V_ty[r][4q + g].
#pragma unroll
      for (int u = 0; u < (FWD ? GF : GD); ++u) {
        const int ot = FWD ? MI + 4 * u : 4 * GF + (MI - 4) + 4 * u;
        if (ot < NGT) {
          const int j = ot / DQ, cb = ot % DQ;
          const int ty = (j == WIN) ? 2 : (j == C ? 1 : 0);
          f4 acc = kZero4;
#pragma unroll
          for (int q = 0; q < HP / 4; ++q)
            acc = mfma16x4(V[(ty * kTileRows + n16) * (HP + 1) + 4 * q + g], wg1[u][q], acc);
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int row = row0 + 4 * g + i;
            if (row < a.B) __builtin_nontemporal_store(acc[i], &a.G[((size_t)row * W1P + j) * D + cb * 16 + n16]);
          }
        }
      }
    }
  };
  auto run_matrix = [&](int stage, int p) {
    // the lane's coordinates through an opaque copy, so that the compiler
    // recomputes each role's operand offsets in the phase instead of
    // hoisting all eight roles' offsets out of the loop into registers
    int ln = lane;
    asm volatile("" : "+v"(ln));
    const int n16 = ln & 15, g = ln >> 4;
    switch (w - NE) {
      case 0: matrix(std::integral_constant<int, 0>{}, stage, p, n16, g); break;
      case 1: matrix(std::integral_constant<int, 1>{}, stage, p, n16, g); break;
      case 2: matrix(std::integral_constant<int, 2>{}, stage, p, n16, g); break;
      case 3: matrix(std::integral_constant<int, 3>{}, stage, p, n16, g); break;
      case 4: matrix(std::integral_constant<int, 4>{}, stage, p, n16, g); break;
      case 5: matrix(std::integral_constant<int, 5>{}, stage, p, n16, g); break;
      case 6: matrix(std::integral_constant<int, 6>{}, stage, p, n16, g); break;
      default: matrix(std::integral_constant<int, 7>{}, stage, p, n16, g); break;
    }
  };

  // epilogue lane map (staging waves): hidden unit hn = lane % 32 of rows
  // 2w + lane / 32 and 2w + lane / 32 + 8
  const int hn = lane & 31, rsel = lane >> 5;
  float b1v = 0.f, w2v = 0.f, b2v = 0.f;
  float db1a = 0.f, dw2a = 0.f, lossa = 0.f;
  // The staging waves' rows in flight live in rr, which they do not use
  // otherwise, so that the union of the roles' registers stays small.  (Ids
  // loaded a phase ahead and held there too measured 1 us slower per step.)
  static_assert(XPE <= CF, "staging rows fit the matrix registers");
  f4 (&xr)[XPE] = *reinterpret_cast<f4 (*)[XPE]>(&rr[0]);
  if (stager) {
    b1v = hn < a.H ? a.b1[hn] : 0.f;
    w2v = hn < a.H ? a.w2[hn] : 0.f;
    b2v = a.b2[0];
    int32_t ids[XPE];
    load_ids(tile0, ids);
    load_x(ids, xr);
    store_x(0, xr);
    if (ntl > 1) {
      load_ids(tile0 + 1, ids);
      load_x(ids, xr);
    }
  } else {
    run_matrix(0, 0);
  }
  __syncthreads();  // X of tile 0 staged

  for (int p = 0; p < ntl + 2; ++p) {
    if (stager) {
      if (p >= 1 && p <= ntl) {
        // ---- epilogue of tile p-1: zp[(p-1) % 2] -> vt[(p-1) % 2]
        const float* Z = zp + ((p - 1) & 1) * Sh::kZp;
        float* V = vt + ((p - 1) & 1) * Sh::kVt;
#pragma unroll
        for (int s8 = 0; s8 < 2; ++s8) {
          const int r = 2 * w + rsel + 8 * s8;
          const int row = (tile0 + p - 1) * kTileRows + r;
          const int ntr = hn >> 4, src = (hn & 15) + 16 * (r >> 2), comp = r & 3;
          float Zc = 0.f, Zctr = 0.f, Zcor = 0.f;
#pragma unroll
          for (int v = 0; v < 2; ++v) {
            Zc += Z[(((v * 3 + 0) * NT + ntr) * 4 + comp) * kWave + src];
            Zctr += Z[(((v * 3 + 1) * NT + ntr) * 4 + comp) * kWave + src];
            Zcor += Z[(((v * 3 + 2) * NT + ntr) * 4 + comp) * kWave + src];
          }
          const float z = b1v + (Zc + Zctr);
          const float zt = b1v + (Zc + Zcor);
          const float h = tanh_fast(z), ht = tanh_fast(zt);
          // h - h~ = tanh(z - z~) (1 - h h~), z - z~ = zctr - zcor without
          // cancellation against the common part
          const float hmh = tanh_fast(Zctr - Zcor) * (1.f - h * ht);
          float ps = w2v * h, pst = w2v * ht;
#pragma unroll
          for (int o = 1; o < 32; o <<= 1) {
            ps += __shfl_xor(ps, o);
            pst += __shfl_xor(pst, o);
          }
          const float mg = 1.f - (b2v + ps) + (b2v + pst);
          const bool on = row < a.B && mg > 0.f;  // hinge active (derivative 0 at margin 0)
          const float gst = on ? a.invB : 0.f;    // d loss/d s~ = m/B, d loss/d s = -m/B
          const float gw = gst * w2v;
          const float dz = -gw * (1.f - h * h);
          const float dzt = gw * (1.f - ht * ht);
          const float dsum = gw * hmh * (h + ht);  // dz + dz~ = g w2 (h - h~)(h + h~)
          V[(0 * kTileRows + r) * (HP + 1) + hn] = dsum;
          V[(1 * kTileRows + r) * (HP + 1) + hn] = dz;
          V[(2 * kTileRows + r) * (HP + 1) + hn] = dzt;
          db1a += dsum;
          dw2a -= gst * hmh;  // -(m/B) h + (m/B) h~
          if (hn == 0) lossa += on ? mg : 0.f;
        }
      }
      if (p + 1 < ntl) {
        store_x((p + 1) & 3, xr);  // rows of tile p+1
        if (p + 2 < ntl) {         // rows of tile p+2 (their ids first: the wait
          int32_t ids[XPE];        // overlaps the matrix waves' work)
          load_ids(tile0 + p + 2, ids);
          load_x(ids, xr);
        }
      }
    } else {
      run_matrix(1, p);
    }
    __syncthreads();  // this phase's X, zp and vt writes visible; its reads done
  }

  // ---- this workgroup's partial slot: dW1 [Hp][K] from the dW1 waves, then
  // db1 [Hp], dw2 [Hp], loss, db2 from the staging waves
  float* P = a.part + (size_t)wg * a.part_stride;
  if (w >= NE + 4) {
    const int mi = w - NE, nt = (mi & 3) >> 1, kh = mi & 1;
    const int n16 = lane & 15, g = lane >> 4;
#pragma unroll
    for (int c = 0; c < CF; ++c) {
      const int kc = kh * CF + c;
#pragma unroll
      for (int i = 0; i < 4; ++i) __builtin_nontemporal_store(rr[c][i], &P[(nt * 16 + 4 * g + i) * K + kc * 16 + n16]);
    }
  }
  if (stager) {
    db1a += __shfl_xor(db1a, 32);
    dw2a += __shfl_xor(dw2a, 32);
    for (int o = 1; o < kWave; o <<= 1) lossa += __shfl_xor(lossa, o);
    float* rw = red + w * (2 * HP + 2);
    if (rsel == 0) {
      rw[hn] = db1a;
      rw[HP + hn] = dw2a;
    }
    if (lane == 0) {
      rw[2 * HP] = lossa;
      rw[2 * HP + 1] = 0.f;
    }
  }
  __syncthreads();
  if (w == 0) {
    for (int e = lane; e < 2 * HP + 2; e += kWave) {
      float s = red[e];
#pragma unroll
      for (int v = 1; v < NE; ++v) s += red[v * (2 * HP + 2) + e];
      P[HP * K + e] = s;
    }
  }
}

}  // namespace pg
