// Multi-pass 2D/3D plan for grids whose half spectra do not fit in LDS.
//
// Per (b, c) line the half spectra U, K of shape [L0][P1][H] (3D; 2D is the
// same with P1 = L1 = 1) live in the workspace, H = Plast/2 + 1:
//
//   rows_fwd   read x1, v, k rows; u = x1 v; real-to-complex transform of every
//              nonzero row of u and of k along the last axis (length Plast).
//   axis1_fwd  (3D) transform along axis 1 of the L1 nonzero rows, all P1 out.
//   core       along axis 0: forward transforms of the U and K lines, gated
//              product U (K + D) with the shortcut folded in, inverse
//              transform, keep the L0 cropped rows; Y overwrites U.
//   axis1_inv  (3D) inverse along axis 1, keep the L1 cropped rows.
//   rows_inv   inverse along the last axis from the half spectrum, two real
//              rows per complex transform; crop, outer gate x2, store y.
//
// Inputs are read once and y is written once; only the spectra round-trip
// through the workspace, which is sized per chunk of lines so that a chunk's
// spectra can stay in the Infinity Cache.  Strided axes are transformed in
// tiles of TL adjacent columns, so every global access is a contiguous run of
// TL complex values and no explicit transpose is ever stored.
#include "kernels.hpp"

namespace hyenand {

namespace {

constexpr int kMaxP = 1024;

struct MpGeom {
  int L0, P0, L1, P1, LL, PL, H;  // L1 = P1 = 1 in 2D
  int rows;                       // nonzero rows per line: L0 * L1
  int64_t half;                   // complex entries of U (or K) per line: L0 * P1 * H
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
  g.rows = g.L0 * g.L1;
  g.half = (int64_t)g.L0 * g.P1 * g.H;
  return g;
}

// workspace row of flat nonzero row r: (n0 * P1 + n1) * H
__device__ __forceinline__ int64_t ws_row(int r, int L1, int P1, int H) {
  return ((int64_t)(r / L1) * P1 + (r % L1)) * H;
}

// ---------------------------------------------------------------------------
// rows_fwd: real-to-complex along the last axis for u = x1 v and k
// ---------------------------------------------------------------------------
template <int PL>
struct RowsCfg {
  static constexpr int ML = PL / 2;
  static constexpr int HP = ML + 1;  // row pitch in LDS
  static constexpr int E = imin(16, ML);
  static constexpr int T = ML / E;
  static constexpr int NT = 256;
  static constexpr int RPW = imax(1, imin(NT / (2 * T), (32 * 1024) / (2 * HP * 8)));  // rows per workgroup
};

template <int PL, bool CIRC, typename TS>
__global__ void __launch_bounds__(256)
    mp_rows_fwd(const TS* __restrict__ x1, const TS* __restrict__ v, const TS* __restrict__ k,
                float2* __restrict__ ws, int64_t line0, int nlines, int rows, int L1, int P1,
                int64_t half, int64_t per_line) {
  using Cf = RowsCfg<PL>;
  constexpr int ML = Cf::ML, HP = Cf::HP, E = Cf::E, T = Cf::T, NT = Cf::NT, RPW = Cf::RPW;
  constexpr int LL = CIRC ? PL : PL / 2;
  constexpr int H = ML + 1;
  constexpr int MNZ = (LL + 1) / 2;
  __shared__ float2 Ur[RPW * HP];
  __shared__ float2 Kr[RPW * HP];
  const int64_t total_rows = (int64_t)nlines * rows;
  const int64_t row0 = (int64_t)blockIdx.x * RPW;
  const int nrow = (int)((total_rows - row0) < RPW ? (total_rows - row0) : RPW);
  const int tid = threadIdx.x;

  // stage real rows (the input rows of the chunk are contiguous)
  {
    float* uf = reinterpret_cast<float*>(Ur);
    float* kf = reinterpret_cast<float*>(Kr);
    const size_t gbase = (size_t)(line0 * rows + row0) * LL;
    for (int i = tid; i < nrow * LL; i += NT) {
      const int r = i / LL, col = i - r * LL;
      uf[r * 2 * HP + col] = ld1(x1 + gbase + i) * ld1(v + gbase + i);
      kf[r * 2 * HP + col] = ld1(k + gbase + i);
    }
  }
  __syncthreads();

  // packed half-length transforms (lanes run across lines)
  constexpr int NLINE = 2 * RPW;
  for (int l0 = 0; l0 < NLINE; l0 += NT / T) {
    const int l = l0 + tid % (NT / T), t = tid / (NT / T);
    const int r = l >> 1;
    const bool act = l < NLINE && r < nrow;
    float2* row = ((l & 1) ? Kr : Ur) + r * HP;
    float2 w[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int m = t + T * e;
      w[e] = (act && (CIRC || m < MNZ)) ? row[m] : czero();
    }
    BlockFFT<ML, E, false>::run(w, t, ScrStrided{row, 1}, act);
    if (act) {
#pragma unroll
      for (int e = 0; e < E; ++e) row[t + T * e] = w[e];
    }
  }
  __syncthreads();

  // untangle: items (line, g), g in [0, ML/2]
  constexpr int NPOST = NLINE * (ML / 2 + 1);
  constexpr int IPT = (NPOST + NT - 1) / NT;
  float2 xa[IPT], xb[IPT];
#pragma unroll
  for (int j = 0; j < IPT; ++j) {
    const int it = tid + NT * j;
    const int l = it % NLINE, g = it / NLINE;
    if (it < NPOST && (l >> 1) < nrow) {
      const float2* row = ((l & 1) ? Kr : Ur) + (l >> 1) * HP;
      r2c_pair(row[g], row[(ML - g) & (ML - 1)], twiddle<ilog2(PL), false>(g), xa[j], xb[j]);
    }
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < IPT; ++j) {
    const int it = tid + NT * j;
    const int l = it % NLINE, g = it / NLINE;
    if (it < NPOST && (l >> 1) < nrow) {
      float2* row = ((l & 1) ? Kr : Ur) + (l >> 1) * HP;
      row[g] = xa[j];
      row[ML - g] = xb[j];
    }
  }
  __syncthreads();

  // store the H bins of every row to U and K (contiguous runs per row)
  for (int i = tid; i < nrow * H; i += NT) {
    const int r = i / H, f = i - r * H;
    const int64_t gr = row0 + r;
    const int64_t line = gr / rows;
    const int rr = (int)(gr - line * rows);
    float2* U = ws + line * per_line;
    const int64_t off = ws_row(rr, L1, P1, H) + f;
    U[off] = Ur[r * HP + f];
    U[half + off] = Kr[r * HP + f];
  }
}

// ---------------------------------------------------------------------------
// strided tiles: TL adjacent columns of a [rows][ncols] complex matrix,
// transformed along the rows index.  LDS tile [P][TLP].
// ---------------------------------------------------------------------------
template <int P, int NS>
struct TileCfg {
  static constexpr int E = imin(16, P);
  static constexpr int T = P / E;
  // enough columns for 512 lanes, at most 32, within ~150 KB of LDS
  static constexpr int TL0 = imin(32, imax(4, 512 / (NS * T)));
  static constexpr int TL = (NS * P * (TL0 + 1) * 8 <= 150 * 1024) ? TL0 : imax(1, TL0 / 2);
  static constexpr int TLP = TL + 1;  // LDS pitch
};

// core tiles: each lane carries one column of both U and K
template <int P>
struct CoreCfg {
  static constexpr int E = imin(16, P);
  static constexpr int T = P / E;
  static constexpr int TL0 = imin(32, imax(4, 512 / T));
  static constexpr int TL = (2 * P * (TL0 + 1) * 8 <= 150 * 1024) ? TL0 : imax(1, TL0 / 2);
  static constexpr int TLP = TL + 1;
};

template <int P, int TLP>
__device__ __forceinline__ void tile_load(float2* tile, const float2* __restrict__ src, int64_t stride, int col0,
                                          int ncols, int nrows_load, int TL, int tid, int nt) {
  for (int i = tid; i < nrows_load * TL; i += nt) {
    const int p = i / TL, cc = i - p * TL;
    if (col0 + cc < ncols) tile[p * TLP + cc] = src[p * stride + col0 + cc];
  }
}

template <int P, int TLP>
__device__ __forceinline__ void tile_store(const float2* tile, float2* __restrict__ dst, int64_t stride, int col0,
                                           int ncols, int nrows_store, int TL, int tid, int nt) {
  for (int i = tid; i < nrows_store * TL; i += nt) {
    const int p = i / TL, cc = i - p * TL;
    if (col0 + cc < ncols) dst[p * stride + col0 + cc] = tile[p * TLP + cc];
  }
}

// ---------------------------------------------------------------------------
// axis-1 transforms (3D): forward on U and K (L1 nonzero rows in, P1 out),
// inverse on Y (P1 in, L1 cropped rows out).  One workgroup per (line, n0, tile).
// ---------------------------------------------------------------------------
template <int P1, bool CIRC, bool INV>
__global__ void __launch_bounds__(512)
    mp_axis1(float2* __restrict__ ws, int H, int L0, int64_t half, int64_t per_line) {
  constexpr int NS = INV ? 1 : 2;  // signals
  using Cf = TileCfg<P1, NS>;
  constexpr int TL = Cf::TL, TLP = Cf::TLP, E = Cf::E, T = Cf::T;
  constexpr int L1 = CIRC ? P1 : P1 / 2;
  constexpr int NT = 512;
  __shared__ float2 tile[NS][P1 * TLP];
  const int ntile = (H + TL - 1) / TL;
  const int64_t bid = blockIdx.x;
  const int tl = (int)(bid % ntile);
  const int64_t rest = bid / ntile;
  const int n0 = (int)(rest % L0);
  const int64_t line = rest / L0;
  const int col0 = tl * TL;
  const int tid = threadIdx.x;
  float2* base = ws + line * per_line + (int64_t)n0 * P1 * H;

  const int nload = INV ? P1 : L1;
#pragma unroll
  for (int s = 0; s < NS; ++s) tile_load<P1, TLP>(tile[s], base + s * half, H, col0, H, nload, TL, tid, NT);
  __syncthreads();

  constexpr int NL = NS * TL;
  for (int l0 = 0; l0 < NL; l0 += NT / T) {
    const int l = l0 + tid % (NT / T), t = tid / (NT / T);
    const int s = l / TL, cc = l % TL;
    const bool act = l < NL && col0 + cc < H;
    float2* col = tile[s < NS ? s : 0] + cc;
    float2 w[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int n = t + T * e;
      w[e] = (act && (INV || CIRC || n < L1)) ? col[n * TLP] : czero();
    }
    BlockFFT<P1, E, INV>::run(w, t, ScrStrided{col, TLP}, act);
    if (act) {
#pragma unroll
      for (int e = 0; e < E; ++e) col[(t + T * e) * TLP] = w[e];
    }
  }
  __syncthreads();
  const int nstore = INV ? L1 : P1;
#pragma unroll
  for (int s = 0; s < NS; ++s) tile_store<P1, TLP>(tile[s], base + s * half, H, col0, H, nstore, TL, tid, NT);
}

// ---------------------------------------------------------------------------
// core: along axis 0, forward U and K, gated product, inverse, crop.
// One workgroup per (line, tile of TL adjacent columns of the [L0][ncols] view).
// ---------------------------------------------------------------------------
template <int P0, bool CIRC>
__global__ void __launch_bounds__(512)
    mp_core(float2* __restrict__ ws, const void* __restrict__ Dp, int dbf16, int64_t line0, int C,
            int ncols, int64_t half, int64_t per_line, float scale) {
  using Cf = CoreCfg<P0>;
  constexpr int TL = Cf::TL, TLP = Cf::TLP, E = Cf::E, T = Cf::T;
  constexpr int L0 = CIRC ? P0 : P0 / 2;
  constexpr int NT = 512;
  __shared__ float2 tile[2][P0 * TLP];
  const int ntile = (ncols + TL - 1) / TL;
  const int tl = (int)(blockIdx.x % ntile);
  const int64_t line = blockIdx.x / ntile;
  const int col0 = tl * TL;
  const int tid = threadIdx.x;
  const int c = (int)((line0 + line) % C);
  const float Dv = dbf16 ? ld1((const uint16_t*)Dp + c) : ld1((const float*)Dp + c);
  const float twoD = 2.f * Dv;
  float2* U = ws + line * per_line;

  tile_load<P0, TLP>(tile[0], U, ncols, col0, ncols, L0, TL, tid, NT);
  tile_load<P0, TLP>(tile[1], U + half, ncols, col0, ncols, L0, TL, tid, NT);
  __syncthreads();

  for (int l0 = 0; l0 < TL; l0 += NT / T) {
    const int cc = l0 + tid % (NT / T), t = tid / (NT / T);
    const bool act = cc < TL && col0 + cc < ncols;
    float2* cu = tile[0] + (cc < TL ? cc : 0);
    float2* ck = tile[1] + (cc < TL ? cc : 0);
    float2 wu[E], wk[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int n = t + T * e;
      const bool nz = act && (CIRC || n < L0);
      wu[e] = nz ? cu[n * TLP] : czero();
      wk[e] = nz ? ck[n * TLP] : czero();
    }
    BlockFFT<P0, E, false>::run(wu, t, ScrStrided{cu, TLP}, act);
    BlockFFT<P0, E, false>::run(wk, t, ScrStrided{ck, TLP}, act);
#pragma unroll
    for (int e = 0; e < E; ++e) wu[e] = c_scale(gated_product(wu[e], wk[e], twoD), scale);
    BlockFFT<P0, E, true>::run(wu, t, ScrStrided{cu, TLP}, act);
    if (act) {
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const int n = t + T * e;
        if (CIRC || n < L0) cu[n * TLP] = wu[e];
      }
    }
  }
  __syncthreads();
  tile_store<P0, TLP>(tile[0], U, ncols, col0, ncols, L0, TL, tid, NT);
}

// ---------------------------------------------------------------------------
// rows_inv: complex-to-real along the last axis, two rows per transform,
// crop, outer gate.  Pair regions of PRP >= PL entries.
// ---------------------------------------------------------------------------
template <int PL>
struct RowsInvCfg {
  static constexpr int H = PL / 2 + 1;
  static constexpr int PRP = PL + 17;  // pair region pitch (holds 2H and the scratch)
  static constexpr int E = imin(16, PL);
  static constexpr int T = PL / E;
  static constexpr int NT = 256;
  static constexpr int PPW = imax(1, imin(NT / T, (48 * 1024) / (PRP * 8)));  // pairs per workgroup
};

template <int PL, bool CIRC, typename TS>
__global__ void __launch_bounds__(256)
    mp_rows_inv(const float2* __restrict__ ws, const TS* __restrict__ x2, TS* __restrict__ y, int64_t line0,
                int nlines, int rows, int L1, int P1, int64_t per_line) {
  using Cf = RowsInvCfg<PL>;
  constexpr int H = Cf::H, PRP = Cf::PRP, E = Cf::E, T = Cf::T, NT = Cf::NT, PPW = Cf::PPW;
  constexpr int LL = CIRC ? PL : PL / 2;
  constexpr int ML = PL / 2;
  __shared__ float2 reg[PPW * PRP];
  const int64_t total_pairs = (int64_t)nlines * rows / 2;
  const int64_t pair0 = (int64_t)blockIdx.x * PPW;
  const int npair = (int)((total_pairs - pair0) < PPW ? (total_pairs - pair0) : PPW);
  const int tid = threadIdx.x;

  // load the half-spectrum rows of each pair: row a at [0, H), row b at [H, 2H)
  for (int i = tid; i < npair * 2 * H; i += NT) {
    const int q = i / (2 * H), rem = i - q * 2 * H;
    const int ab = rem / H, f = rem - ab * H;
    const int64_t gr = 2 * (pair0 + q) + ab;
    const int64_t line = gr / rows;
    const int rr = (int)(gr - line * rows);
    reg[q * PRP + rem] = ws[line * per_line + ws_row(rr, L1, P1, H) + f];
  }
  __syncthreads();

  for (int q0 = 0; q0 < PPW; q0 += NT / T) {
    const int q = q0 + tid % (NT / T), t = tid / (NT / T);
    const bool act = q < npair;
    float2* R = reg + (q < PPW ? q : 0) * PRP;
    float2 w[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int f = t + T * e;
      float2 ya = czero(), yb = czero();
      if (act) {
        if (f <= ML) {
          ya = R[f];
          yb = R[H + f];
        } else {
          ya = c_conj(R[PL - f]);
          yb = c_conj(R[H + PL - f]);
        }
      }
      w[e] = make_float2(ya.x - yb.y, ya.y + yb.x);  // ya + i yb
    }
    if constexpr (T == 1) __syncthreads();
    BlockFFT<PL, E, true>::run(w, t, ScrStrided{R, 1}, act);
    if (act) {
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const int n = t + T * e;
        if (CIRC || n < LL) R[n] = w[e];
      }
    }
  }
  __syncthreads();

  const size_t gbase = (size_t)(line0 * rows + 2 * pair0) * LL;
  for (int i = tid; i < npair * 2 * LL; i += NT) {
    const int row = i / LL, n = i - row * LL;
    const float2 qv = reg[(row >> 1) * PRP + n];
    st1(y + gbase + i, ld1(x2 + gbase + i) * ((row & 1) ? qv.y : qv.x));
  }
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
struct MpLaunch {
  const FftConvArgs* a;
  MpGeom g;
  float2* ws;
  int64_t line0;
  int nl;
  int64_t per;  // complex entries per line (U and K)
  float scale;
  hipStream_t s;
};

template <int PL>
hipError_t rows_fwd(const MpLaunch& L) {
  const int64_t total = (int64_t)L.nl * L.g.rows;
  const dim3 grid((unsigned)((total + RowsCfg<PL>::RPW - 1) / RowsCfg<PL>::RPW));
  const FftConvArgs& a = *L.a;
#define HY_ARGS(TS) (const TS*)a.x1, (const TS*)a.v, (const TS*)a.k, L.ws, L.line0, L.nl, L.g.rows, L.g.L1, L.g.P1, \
                    L.g.half, L.per
  if (a.bf16) {
    if (a.circular) hipLaunchKernelGGL((mp_rows_fwd<PL, true, uint16_t>), grid, dim3(256), 0, L.s, HY_ARGS(uint16_t));
    else hipLaunchKernelGGL((mp_rows_fwd<PL, false, uint16_t>), grid, dim3(256), 0, L.s, HY_ARGS(uint16_t));
  } else {
    if (a.circular) hipLaunchKernelGGL((mp_rows_fwd<PL, true, float>), grid, dim3(256), 0, L.s, HY_ARGS(float));
    else hipLaunchKernelGGL((mp_rows_fwd<PL, false, float>), grid, dim3(256), 0, L.s, HY_ARGS(float));
  }
#undef HY_ARGS
  return hipGetLastError();
}

template <int P1, bool INV>
hipError_t axis1(const MpLaunch& L) {
  constexpr int TL = TileCfg<P1, INV ? 1 : 2>::TL;
  const int ntile = (L.g.H + TL - 1) / TL;
  const dim3 grid((unsigned)((int64_t)L.nl * L.g.L0 * ntile));
  if (L.a->circular)
    hipLaunchKernelGGL((mp_axis1<P1, true, INV>), grid, dim3(512), 0, L.s, L.ws, L.g.H, L.g.L0, L.g.half, L.per);
  else
    hipLaunchKernelGGL((mp_axis1<P1, false, INV>), grid, dim3(512), 0, L.s, L.ws, L.g.H, L.g.L0, L.g.half, L.per);
  return hipGetLastError();
}
template <int P1>
hipError_t axis1_fwd(const MpLaunch& L) { return axis1<P1, false>(L); }
template <int P1>
hipError_t axis1_inv(const MpLaunch& L) { return axis1<P1, true>(L); }

template <int P0>
hipError_t core(const MpLaunch& L) {
  constexpr int TL = CoreCfg<P0>::TL;
  const int ncols = L.g.P1 * L.g.H;
  const int ntile = (ncols + TL - 1) / TL;
  const dim3 grid((unsigned)((int64_t)L.nl * ntile));
  const FftConvArgs& a = *L.a;
  if (a.circular)
    hipLaunchKernelGGL((mp_core<P0, true>), grid, dim3(512), 0, L.s, L.ws, a.D, (int)a.bf16, L.line0, (int)a.C,
                       ncols, L.g.half, L.per, L.scale);
  else
    hipLaunchKernelGGL((mp_core<P0, false>), grid, dim3(512), 0, L.s, L.ws, a.D, (int)a.bf16, L.line0, (int)a.C,
                       ncols, L.g.half, L.per, L.scale);
  return hipGetLastError();
}

template <int PL>
hipError_t rows_inv(const MpLaunch& L) {
  const int64_t pairs = (int64_t)L.nl * L.g.rows / 2;
  const dim3 grid((unsigned)((pairs + RowsInvCfg<PL>::PPW - 1) / RowsInvCfg<PL>::PPW));
  const FftConvArgs& a = *L.a;
#define HY_ARGS(TS) L.ws, (const TS*)a.x2, (TS*)a.y, L.line0, L.nl, L.g.rows, L.g.L1, L.g.P1, L.per
  if (a.bf16) {
    if (a.circular) hipLaunchKernelGGL((mp_rows_inv<PL, true, uint16_t>), grid, dim3(256), 0, L.s, HY_ARGS(uint16_t));
    else hipLaunchKernelGGL((mp_rows_inv<PL, false, uint16_t>), grid, dim3(256), 0, L.s, HY_ARGS(uint16_t));
  } else {
    if (a.circular) hipLaunchKernelGGL((mp_rows_inv<PL, true, float>), grid, dim3(256), 0, L.s, HY_ARGS(float));
    else hipLaunchKernelGGL((mp_rows_inv<PL, false, float>), grid, dim3(256), 0, L.s, HY_ARGS(float));
  }
#undef HY_ARGS
  return hipGetLastError();
}

#define HY_SIZE_SWITCH(P, FN, ARG)            \
  switch (P) {                                \
    case 2: return FN<2>(ARG);                \
    case 4: return FN<4>(ARG);                \
    case 8: return FN<8>(ARG);                \
    case 16: return FN<16>(ARG);              \
    case 32: return FN<32>(ARG);              \
    case 64: return FN<64>(ARG);              \
    case 128: return FN<128>(ARG);            \
    case 256: return FN<256>(ARG);            \
    case 512: return FN<512>(ARG);            \
    case 1024: return FN<1024>(ARG);          \
    default: return hipErrorInvalidValue;     \
  }

hipError_t d_rows_fwd(int P, const MpLaunch& L) { HY_SIZE_SWITCH(P, rows_fwd, L) }
hipError_t d_axis1_fwd(int P, const MpLaunch& L) { HY_SIZE_SWITCH(P, axis1_fwd, L) }
hipError_t d_core(int P, const MpLaunch& L) { HY_SIZE_SWITCH(P, core, L) }
hipError_t d_axis1_inv(int P, const MpLaunch& L) { HY_SIZE_SWITCH(P, axis1_inv, L) }
hipError_t d_rows_inv(int P, const MpLaunch& L) { HY_SIZE_SWITCH(P, rows_inv, L) }

}  // namespace

bool multipass_supported(const FftConvArgs& a) {
  if (a.ndim != 2 && a.ndim != 3) return false;
  for (int d = 0; d < a.ndim; ++d)
    if (a.P[d] < 2 || a.P[d] > kMaxP || a.L[d] < 2) return false;
  return true;
}

size_t multipass_bytes_per_line(const FftConvArgs& a) {
  const MpGeom g = mp_geom(a);
  return (size_t)(2 * g.half) * sizeof(float2);
}

hipError_t launch_multipass(const FftConvArgs& a, int64_t chunk, hipStream_t s) {
  if (!multipass_supported(a) || chunk < 1) return hipErrorInvalidValue;
  MpLaunch L;
  L.a = &a;
  L.g = mp_geom(a);
  L.ws = (float2*)a.ws;
  L.per = 2 * L.g.half;
  L.scale = (float)(1.0 / (4.0 * (double)L.g.P0 * (double)L.g.P1 * (double)L.g.PL));
  L.s = s;
  const bool three = a.ndim == 3;
  for (int64_t line0 = 0; line0 < a.lines; line0 += chunk) {
    L.line0 = line0;
    L.nl = (int)((a.lines - line0) < chunk ? (a.lines - line0) : chunk);
    hipError_t e;
    if ((e = d_rows_fwd(L.g.PL, L)) != hipSuccess) return e;
    if (three && (e = d_axis1_fwd(L.g.P1, L)) != hipSuccess) return e;
    if ((e = d_core(L.g.P0, L)) != hipSuccess) return e;
    if (three && (e = d_axis1_inv(L.g.P1, L)) != hipSuccess) return e;
    if ((e = d_rows_inv(L.g.PL, L)) != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace hyenand
