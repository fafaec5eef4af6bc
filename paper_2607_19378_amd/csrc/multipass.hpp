// Geometry and strided-axis tiles shared by the multi-pass 2D/3D forward
// and backward plans.
//
// Per (b, c) line each half spectrum of shape [L0][P1][H] (3D; 2D is the same
// with P1 = L1 = 1) lives in the workspace, H = Plast/2 + 1 valid bins per row
// stored with a row stride HS = H rounded up to 16 complex values (128 B), so
// every row starts on a cache line.
#pragma once

#include "kernels.hpp"

namespace hyenand {
namespace {

constexpr int kMaxP = 1024;

struct MpGeom {
  int L0, P0, L1, P1, LL, PL, H, HS;  // L1 = P1 = 1 in 2D
  int rows;                           // nonzero rows per line: L0 * L1
  int64_t half;                       // complex entries of U (and of K) per line: L0 * P1 * HS
  bool kc;                            // centered kernel: K holds P0 * P1 rows
  int krows0;                         // planes n0 of K: L0, or P0 centered
  int64_t halfK;                      // complex entries of K per line: krows0 * P1 * HS
};

MpGeom mp_geom(const FftConvArgs& a) {
  MpGeom g;
  g.L0 = (int)a.L[0];
  g.P0 = (int)a.P[0];
  if (a.ndim == 3) {
    g.L1 = (int)a.L[1];
    g.P1 = (int)a.P[1];
  } else {
    g.L1 = g.P1 = 1;
  }
  g.LL = (int)a.L[a.ndim - 1];
  g.PL = (int)a.P[a.ndim - 1];
  g.H = g.PL / 2 + 1;
  g.HS = (g.H + 15) & ~15;
  g.rows = g.L0 * g.L1;
  g.half = (int64_t)g.L0 * g.P1 * g.HS;
  g.kc = a.centered;
  g.krows0 = g.kc ? g.P0 : g.L0;
  g.halfK = (int64_t)g.krows0 * g.P1 * g.HS;
  return g;
}

// workspace offset of flat nonzero row r: (n0 * P1 + n1) * HS
__device__ __forceinline__ int64_t ws_row(int r, int L1, int P1, int HS) {
  return ((int64_t)(r / L1) * P1 + (r % L1)) * HS;
}

// Workspace offsets (complex entries from ws) of the NR consecutive chunk
// rows grow0 .. grow0 + NR - 1 that one workgroup moves, written to off[] by
// its NT lanes (NR may exceed NT: short rows pack many per workgroup): the
// divisions by the run-time row counts happen once per row here instead of
// once per element in the copy loops.  Rows at or beyond nrow get offset 0
// (never used).  The caller synchronises before reading off[].
template <int NR, int NT>
__device__ __forceinline__ void ws_row_offsets(int64_t* off, int64_t grow0, int nrow, int rows, int L1, int P1,
                                               int HS, int64_t per_line, int tid) {
  for (int r = tid; r < NR; r += NT) {
    int64_t o = 0;
    if (r < nrow) {
      const int64_t gr = grow0 + r;
      const int64_t line = gr / rows;
      const int rr = (int)(gr - line * rows);
      o = line * per_line + ws_row(rr, L1, P1, HS);
    }
    off[r] = o;
  }
}

// ---------------------------------------------------------------------------
// strided tiles: TL adjacent columns of a [rows][stride] complex matrix,
// transformed along the rows index.  LDS tile [P][TLP].  Columns whose index
// modulo HS is >= H (row padding) are neither loaded nor stored.
// ---------------------------------------------------------------------------
// Tiles: the widest power of two <= 32 whose NS signal tiles fit in KB
// kilobytes of LDS, and E points per lane so that a tile keeps NT lanes busy.
// The axis-1 passes use two 512-lane workgroups per CU (76 KB each); the core
// pass, which holds one signal, uses four 256-lane workgroups (38 KB) where
// that still leaves tiles 16 columns wide, since more resident workgroups
// overlap the load, transform and store phases better.
constexpr int mp_tl(int P, int NS, int KB) {
  int tl = 32;
  while (tl > 1 && NS * P * (tl + 1) * 8 > KB * 1024) tl /= 2;
  return tl;
}
constexpr int mp_pow2_floor(int n) { return n <= 1 ? 1 : 2 * mp_pow2_floor(n / 2); }
constexpr int mp_e(int P, int lines, int NT) { return imin(P, imax(2, mp_pow2_floor(imin(16, P * lines / NT)))); }
constexpr int kTileNT = 512;
constexpr int kTileKB = 76;
constexpr bool mp_core_small(int P0) { return mp_tl(P0, 1, kTileKB / 2) >= 16; }
constexpr int mp_core_nt(int P0) { return mp_core_small(P0) ? kTileNT / 2 : kTileNT; }

template <int P, int NS>
struct TileCfg {  // NS signal tiles, each column of each signal is one line
  static constexpr int TL = mp_tl(P, NS, kTileKB);
  static constexpr int E = mp_e(P, NS * TL, kTileNT);
  static constexpr int T = P / E;
  static constexpr int TLP = TL + 1;
};

__device__ __forceinline__ bool col_valid(int col, int ncols, int HS, int H) {
  return col < ncols && (col % HS) < H;
}

// Each lane always handles the same column cc = tid % TL (NT is a multiple
// of TL), so the column test runs once per lane; rows are copied in batches
// with all loads of a batch in flight together.
template <int NROWS, int TL, int TLP, int NT>
__device__ __forceinline__ void tile_load(float2* tile, const float2* __restrict__ src, int64_t stride, int col0,
                                          int ncols, int HS, int H, int tid) {
  static_assert(NT % TL == 0, "lanes keep their column");
  const int cc = tid % TL;
  const bool ok = col_valid(col0 + cc, ncols, HS, H);
  const float2* s = src + col0 + cc;
  batched_copy<NROWS * TL, NT, 8>(
      tid, [&](int i) { return ok ? s[(int64_t)(i / TL) * stride] : czero(); },
      [&](int i, float2 z) { tile[(i / TL) * TLP + cc] = z; });
}

template <int NROWS, int TL, int TLP, int NT>
__device__ __forceinline__ void tile_store(const float2* tile, float2* __restrict__ dst, int64_t stride, int col0,
                                           int ncols, int HS, int H, int tid) {
  static_assert(NT % TL == 0, "lanes keep their column");
  const int cc = tid % TL;
  const bool ok = col_valid(col0 + cc, ncols, HS, H);
  float2* d = dst + col0 + cc;
  batched_copy<NROWS * TL, NT, 8>(
      tid, [&](int i) { return tile[(i / TL) * TLP + cc]; },
      [&](int i, float2 z) {
        if (ok) d[(int64_t)(i / TL) * stride] = z;
      });
}

// ---------------------------------------------------------------------------
// axis-1 transforms (3D): forward on NS signals (nload nonzero rows in: L1,
// or P1 for a centered kernel; P1 out), inverse on NS signals (P1 in, L1
// cropped rows out).  Signal s of a line starts at sig_off + s * half and
// has `planes` planes n0.  One workgroup per (line, n0, tile).
// ---------------------------------------------------------------------------
template <int P1, bool CIRC, bool INV, int NS>
__global__ void __launch_bounds__(kTileNT)
    mp_axis1(float2* __restrict__ ws, int H, int HS, int planes, int64_t half, int64_t per_line, int nload,
             int64_t sig_off) {
  using Cf = TileCfg<P1, NS>;
  constexpr int TL = Cf::TL, TLP = Cf::TLP, E = Cf::E, T = Cf::T;
  constexpr int L1 = CIRC ? P1 : P1 / 2;
  constexpr int NT = kTileNT;
  __shared__ float2 tile[NS][P1 * TLP];
  __shared__ float2 twl[imax(1, PassTw<P1, E>::kCount)];
  PassTw<P1, E>::fill(twl, threadIdx.x, NT);
  const int ntile = (H + TL - 1) / TL;
  const int64_t bid = blockIdx.x;
  const int tl = (int)(bid % ntile);
  const int64_t rest = bid / ntile;
  const int n0 = (int)(rest % planes);
  const int64_t line = rest / planes;
  const int col0 = tl * TL;
  const int tid = threadIdx.x;
  float2* base = ws + line * per_line + sig_off + (int64_t)n0 * P1 * HS;

  // Lines are (signal, column) pairs; lane (line, t) moves rows t + T e of
  // its column straight between global memory and registers (consecutive
  // lanes, consecutive columns), in place: the forward reads the nload
  // nonzero rows and writes all P1, the inverse reads P1 rows and keeps L1.
  // The LDS tile is only the exchange scratch.
  constexpr int NL = NS * TL;
  const int NLOAD = INV ? P1 : nload;
  constexpr int NSTORE = INV ? L1 : P1;
  for (int l0 = 0; l0 < NL; l0 += NT / T) {
    const int l = l0 + tid % (NT / T), t = tid / (NT / T);
    const int s = l / TL, cc = l % TL;
    const bool act = l < NL;
    const bool cv = act && col0 + cc < H;
    float2* const g = base + (act ? s : 0) * half + col0 + cc;
    float2 w[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int n = t + T * e;
      w[e] = (cv && n < NLOAD) ? g[(int64_t)n * HS] : czero();
    }
    BlockFFT<P1, E, INV>::run(w, t, ScrS<TLP>{tile[act ? s : 0] + cc}, act, twl);
    if (cv) {
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const int n = t + T * e;
        if (n < NSTORE) g[(int64_t)n * HS] = w[e];
      }
    }
  }
}

}  // namespace
}  // namespace hyenand
