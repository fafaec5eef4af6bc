// Multi-pass 2D/3D plan for grids whose half spectra do not fit in LDS.
//
// Per (b, c) line the half spectra U, K of shape [L0][P1][H] (3D; 2D is the
// same with P1 = L1 = 1) live in the workspace, H = Plast/2 + 1 valid bins
// per row stored with a row stride HS = H rounded up to 16 complex values
// (128 B), so every row starts on a cache line:
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
// through the workspace, which is sized per chunk of lines.  Strided axes are
// transformed in tiles of TL adjacent columns, so every global access is a
// contiguous run of TL complex values and no explicit transpose is stored.
// Tiles are sized so that two 512-lane (core pass: up to four 256-lane)
// workgroups share a CU.
#include <type_traits>

#include "multipass.hpp"

namespace hyenand {

namespace {

// ---------------------------------------------------------------------------
// rows_fwd: real-to-complex along the last axis for u = x1 v and k
// ---------------------------------------------------------------------------
template <int PL>
struct RowsCfg {
  static constexpr int ML = PL / 2;
  static constexpr int HP = ML + 1;  // row pitch in LDS (odd for ML >= 2)
  static constexpr int E = imin(16, ML);
  static constexpr int T = ML / E;
  static constexpr int NT = 256;
  static constexpr int RPW = imax(1, imin(NT / (2 * T), (36 * 1024) / (2 * HP * 8)));  // rows per workgroup
};

template <int PL, bool CIRC, typename TS, bool ACT = false>
__global__ void __launch_bounds__(256)
    mp_rows_fwd(const TS* __restrict__ x1, const TS* __restrict__ v, const TS* __restrict__ k,
                float2* __restrict__ ws, int64_t line0, int nlines, int rows, int L1, int P1, int HS,
                int64_t half, int64_t per_line, int kC, int nsig, ActIn ain, int C) {
  using Cf = RowsCfg<PL>;
  constexpr int ML = Cf::ML, HP = Cf::HP, E = Cf::E, T = Cf::T, NT = Cf::NT, RPW = Cf::RPW;
  constexpr int LL = CIRC ? PL : PL / 2;
  constexpr int H = ML + 1;
  constexpr int MNZ = (LL + 1) / 2;
  __shared__ float2 Ur[RPW * HP];
  __shared__ float2 Kr[RPW * HP];
  __shared__ float2 twl[imax(1, PassTw<ML, E>::kCount)];
  __shared__ int64_t roff[RPW];
  const int64_t total_rows = (int64_t)nlines * rows;
  const int64_t row0 = (int64_t)blockIdx.x * RPW;
  const int nrow = (int)((total_rows - row0) < RPW ? (total_rows - row0) : RPW);
  const int tid = threadIdx.x;
  PassTw<ML, E>::fill(twl, tid, NT);
  ws_row_offsets<RPW, NT>(roff, row0, nrow, rows, L1, P1, HS, per_line, tid);

  // stage real rows (the input rows of the chunk are contiguous), four
  // samples per global load, written to LDS as two 8-byte pairs
  {
    const size_t gbase = (size_t)(line0 * rows + row0) * LL;
    // element e of the chunk's input reads k at kidx(e): the same element
    // of line k_line(e / (rows LL)) (rows and LL are powers of two)
    const size_t per = (size_t)rows * LL;
    auto kidx = [&](size_t e) -> size_t {
      return kC ? (size_t)k_line((int64_t)(e / per), kC) * per + (e & (per - 1)) : e;
    };
    if constexpr (LL % 4 == 0) {
      struct In3 {
        float4 a, b, k;
      };
      batched_copy<RPW * (LL / 4), NT, 4>(
          tid,
          [&](int i4) {
            In3 z;
            const int i = 4 * i4;
            if (i / LL < nrow) {
              z.a = ld4(x1 + gbase + i);
              z.b = ld4(v + gbase + i);
              z.k = nsig > 1 ? ld4(k + kidx(gbase + i)) : make_float4(0.f, 0.f, 0.f, 0.f);
              if constexpr (ACT) {  // the operator's inner gate; a line's points are contiguous
                const size_t e = gbase + i;
                const int64_t line = (int64_t)(e / per);
                z.a = line_gates<true, TS>(ain, line, C).u4(z.a, z.b, (int64_t)(e - (size_t)line * per));
                z.b = make_float4(1.f, 1.f, 1.f, 1.f);
              }
            }
            return z;
          },
          [&](int i4, const In3& z) {
            const int i = 4 * i4;
            const int r = i / LL, col = i - r * LL;
            if (r < nrow) {
              float2* du = Ur + r * HP + col / 2;
              float2* dk = Kr + r * HP + col / 2;
              du[0] = make_float2(z.a.x * z.b.x, z.a.y * z.b.y);
              du[1] = make_float2(z.a.z * z.b.z, z.a.w * z.b.w);
              dk[0] = make_float2(z.k.x, z.k.y);
              dk[1] = make_float2(z.k.z, z.k.w);
            }
          });
    } else {
      float* uf = reinterpret_cast<float*>(Ur);
      float* kf = reinterpret_cast<float*>(Kr);
      batched_copy<RPW * LL, NT, 8>(
          tid,
          [&](int i) {
            float2 z = czero();
            if (i / LL < nrow) {
              const size_t e = gbase + i;
              const int64_t line = (int64_t)(e / per);
              const float u = line_gates<ACT, TS>(ain, line, C).u1(ld1(x1 + e), ld1(v + e), (int64_t)(e - (size_t)line * per));
              z = make_float2(u, nsig > 1 ? ld1(k + kidx(e)) : 0.f);
            }
            return z;
          },
          [&](int i, float2 z) {
            const int r = i / LL, col = i - r * LL;
            if (r < nrow) {
              uf[r * 2 * HP + col] = z.x;
              kf[r * 2 * HP + col] = z.y;
            }
          });
    }
  }
  __syncthreads();

  // packed half-length transforms (lanes run across lines)
  constexpr int NLINE = 2 * RPW;
  for (int l0 = 0; l0 < NLINE; l0 += NT / T) {
    const int l = l0 + tid % (NT / T), t = tid / (NT / T);
    const int r = l >> 1;
    const bool act = l < NLINE && r < nrow && (l & 1) < nsig;
    float2* row = ((l & 1) ? Kr : Ur) + (act ? r : 0) * HP;
    float2 w[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int m = t + T * e;
      w[e] = (act && (CIRC || m < MNZ)) ? row[m] : czero();
    }
    BlockFFT<ML, E, false>::run(w, t, ScrS<1>{row}, act, twl);
    if (act) {
#pragma unroll
      for (int e = 0; e < E; ++e) row[t + T * e] = w[e];
    }
  }
  __syncthreads();

  // untangle in place: item (line, g) owns bins g and ML - g (g = 0 also
  // writes the Nyquist slot ML)
  constexpr int NPOST = NLINE * (ML / 2 + 1);
  for (int it = tid; it < NPOST; it += NT) {
    const int l = it % NLINE, g = it / NLINE;
    if ((l >> 1) < nrow && (l & 1) < nsig) {
      float2* row = ((l & 1) ? Kr : Ur) + (l >> 1) * HP;
      float2 xa, xb;
      r2c_pair(row[g], row[(ML - g) & (ML - 1)], twiddle<ilog2(PL), false>(g), xa, xb);
      row[g] = xa;
      row[ML - g] = xb;
    }
  }
  __syncthreads();

  // store the H bins of every row to U and K (rows start on cache lines)
  batched_copy<RPW * H, NT, 8>(
      tid,
      [&](int i) {
        const int r = i / H, f = i - r * H;
        return make_float4(Ur[r * HP + f].x, Ur[r * HP + f].y, Kr[r * HP + f].x, Kr[r * HP + f].y);
      },
      [&](int i, float4 z) {
        const int r = i / H, f = i - r * H;
        if (r < nrow) {
          float2* U = ws + roff[r] + f;
          U[0] = make_float2(z.x, z.y);
          if (nsig > 1) U[half] = make_float2(z.z, z.w);
        }
      });
}

// ---------------------------------------------------------------------------
// rows of a centered kernel: K holds all P0 x P1 grid rows, each a full real
// row of PL points gathered from the (2 L0 - 1) x (2 L1 - 1) x (2 LL - 1)
// centered points (grid index g of an axis holds displacement g or g - 2L);
// real-to-complex along the last axis, stored at koff + row * HS.
// ---------------------------------------------------------------------------
template <int PL, typename TS>
__global__ void __launch_bounds__(256)
    mp_rows_kc(const TS* __restrict__ k, float2* __restrict__ ws, int64_t line0, int nlines, int krows, int L0,
               int L1, int P1, int HS, int64_t koff, int64_t per_line, int kC) {
  using Cf = RowsCfg<PL>;
  constexpr int ML = Cf::ML, HP = Cf::HP, E = Cf::E, T = Cf::T, NT = Cf::NT;
  constexpr int RPW = 2 * Cf::RPW;  // one signal: the two-signal pass's LDS holds twice the rows
  constexpr int LL = PL / 2;
  constexpr int H = ML + 1;
  __shared__ float2 Kr[RPW * HP];
  __shared__ float2 twl[imax(1, PassTw<ML, E>::kCount)];
  const int64_t total_rows = (int64_t)nlines * krows;
  const int64_t row0 = (int64_t)blockIdx.x * RPW;
  const int nrow = (int)((total_rows - row0) < RPW ? (total_rows - row0) : RPW);
  const int tid = threadIdx.x;
  PassTw<ML, E>::fill(twl, tid, NT);
  const int K1 = 2 * L1 - 1;
  constexpr int K2 = 2 * LL - 1;
  const int64_t kpts = (int64_t)(2 * L0 - 1) * K1 * K2;

  // gather the grid points 2m, 2m + 1 of every row
  batched_copy<RPW * ML, NT, 8>(
      tid,
      [&](int i) {
        const int r = i / ML, m = i - r * ML;
        float2 z = czero();
        if (r < nrow) {
          const int64_t gr = row0 + r;
          const int64_t line = gr / krows;
          const int rr = (int)(gr - line * krows);
          const int j0 = centered_index(rr / P1, L0, 2 * L0), j1 = centered_index(rr % P1, L1, 2 * L1);
          if (j0 >= 0 && j1 >= 0) {
            const TS* kr = k + (size_t)k_line(line0 + line, kC) * kpts + ((size_t)j0 * K1 + j1) * K2;
            const int ja = centered_index(2 * m, LL, PL), jb = centered_index(2 * m + 1, LL, PL);
            z = make_float2(ja >= 0 ? ld1(kr + ja) : 0.f, jb >= 0 ? ld1(kr + jb) : 0.f);
          }
        }
        return z;
      },
      [&](int i, float2 z) {
        const int r = i / ML, m = i - r * ML;
        Kr[r * HP + m] = z;
      });
  __syncthreads();

  for (int l0 = 0; l0 < RPW; l0 += NT / T) {
    const int l = l0 + tid % (NT / T), t = tid / (NT / T);
    const bool act = l < RPW && l < nrow;
    float2* row = Kr + (act ? l : 0) * HP;
    float2 w[E];
#pragma unroll
    for (int e = 0; e < E; ++e) w[e] = act ? row[t + T * e] : czero();
    BlockFFT<ML, E, false>::run(w, t, ScrS<1>{row}, act, twl);
    if (act) {
#pragma unroll
      for (int e = 0; e < E; ++e) row[t + T * e] = w[e];
    }
  }
  __syncthreads();

  constexpr int NPOST = RPW * (ML / 2 + 1);
  for (int it = tid; it < NPOST; it += NT) {
    const int l = it % RPW, g = it / RPW;
    if (l < nrow) {
      float2* row = Kr + l * HP;
      float2 xa, xb;
      r2c_pair(row[g], row[(ML - g) & (ML - 1)], twiddle<ilog2(PL), false>(g), xa, xb);
      row[g] = xa;
      row[ML - g] = xb;
    }
  }
  __syncthreads();

  batched_copy<RPW * H, NT, 8>(
      tid, [&](int i) { return Kr[(i / H) * HP + (i % H)]; },
      [&](int i, float2 z) {
        const int r = i / H, f = i - r * H;
        if (r < nrow) {
          const int64_t gr = row0 + r;
          const int64_t line = gr / krows;
          const int rr = (int)(gr - line * krows);
          ws[line * per_line + koff + (int64_t)rr * HS + f] = z;
        }
      });
}

// ---------------------------------------------------------------------------
// core: along axis 0, forward U and K, gated product, inverse, crop.
// One workgroup per (line, tile of TL adjacent columns of the [L0][ncols]
// view).  Only one signal tile lives in LDS: K's tile is prefetched into
// registers while U's tile loads and transforms, then takes its place.
// The view has ncols / HS rows of HS slots, of which bins 0 .. H - 1 are
// valid.  With nyq set ((H - 1) a multiple of TL, several rows), a row's
// first H - 1 bins make whole aligned tiles and the last bin of every row
// (the Nyquist bin) goes into tiles of its own, TL rows each, so that no
// lane transforms the padding slots; else tiles run over every slot and the
// padding lanes idle.
// ---------------------------------------------------------------------------
template <int P0, bool CIRC>
struct CoreCfg {
  static constexpr int NT = mp_core_nt(P0);
  static constexpr int TL = mp_tl(P0, 1, mp_core_small(P0) ? kTileKB / 2 : kTileKB);
  static constexpr int E = mp_e(P0, TL, NT);
  static constexpr int T = P0 / E;
  static constexpr int TLP = TL + 1;
  static constexpr int L0 = CIRC ? P0 : P0 / 2;
};

template <int P0, bool CIRC>
__global__ void __launch_bounds__(mp_core_nt(P0))
    mp_core(float2* __restrict__ ws, const void* __restrict__ Dp, int dbf16, int64_t line0, int C,
            int ncols, int HS, int H, int64_t half, int64_t per_line, float scale, int krows, int nyq) {
  using Cf = CoreCfg<P0, CIRC>;
  constexpr int TL = Cf::TL, TLP = Cf::TLP, E = Cf::E, T = Cf::T, NT = Cf::NT, L0 = Cf::L0;
  __shared__ float2 tile[P0 * TLP];
  __shared__ float2 twl[imax(1, PassTw<P0, E>::kCount)];
  const int vrows = ncols / HS;
  const int rtiles = (H - 1) / TL;  // aligned tiles per row (nyq)
  const int ntile = nyq ? vrows * rtiles + (vrows + TL - 1) / TL : (ncols + TL - 1) / TL;
  const int tl = (int)(blockIdx.x % ntile);
  const int64_t line = blockIdx.x / ntile;
  const int tid = threadIdx.x;
  PassTw<P0, E>::fill(twl, tid, NT);
  const int c = (int)((line0 + line) % C);
  const float Dv = dbf16 ? ld1((const uint16_t*)Dp + c) : ld1((const float*)Dp + c);
  const float twoD = 2.f * Dv;
  float2* U = ws + line * per_line;
  const float2* K = U + half;

  // Column points of U and K straight from global memory into registers
  // (lane (cc, t) holds rows n = t + T e of column col; consecutive lanes
  // read consecutive columns, except in Nyquist tiles).  K's loads are issued right after U's
  // and arrive while U is transformed.  The LDS tile is only the exchange
  // scratch; the result goes back to U's rows straight from registers.
  static_assert(NT / T >= TL, "one round of columns");
  const int cc = tid % TL, t = tid / TL;
  const bool act = t < T;
  int col;
  bool cv;
  if (!nyq) {
    col = tl * TL + cc;
    cv = act && col_valid(col, ncols, HS, H);
  } else if (tl < vrows * rtiles) {  // aligned bins of one row
    col = (tl / rtiles) * HS + (tl % rtiles) * TL + cc;
    cv = act;
  } else {  // the Nyquist bins of TL rows
    const int r = (tl - vrows * rtiles) * TL + cc;
    cv = act && r < vrows;
    col = cv ? r * HS + (H - 1) : 0;
  }
  float2* const uc = U + col;
  const float2* const kc = K + col;
  const ScrS<TLP> sc{tile + cc};
  float2 wu[E], wk[E];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int n = t + T * e;
    wu[e] = (cv && (CIRC || n < L0)) ? uc[(int64_t)n * ncols] : czero();
  }
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int n = t + T * e;
    wk[e] = (cv && (CIRC || n < krows)) ? kc[(int64_t)n * ncols] : czero();
  }
  BlockFFT<P0, E, false>::run(wu, t, sc, act, twl);
  BlockFFT<P0, E, false>::run(wk, t, sc, act, twl);
#pragma unroll
  for (int e = 0; e < E; ++e) wu[e] = c_scale(gated_product(wu[e], wk[e], twoD), scale);
  BlockFFT<P0, E, true>::run(wu, t, sc, act, twl);
  if (cv) {
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int n = t + T * e;
      if (CIRC || n < L0) uc[(int64_t)n * ncols] = wu[e];
    }
  }
}

// ---------------------------------------------------------------------------
// rows_inv: complex-to-real along the last axis, two rows per transform,
// crop, outer gate.  Pair regions of PRP >= PL entries.
// ---------------------------------------------------------------------------
template <int PL>
struct RowsInvCfg {
  static constexpr int H = PL / 2 + 1;
  // pair region pitch: the two half spectra (2H entries), then the exchange
  // scratch and the outputs with one pad slot per 16 entries
  static constexpr int PRP = imax(2 * H, pad16_size(PL));
  static constexpr int E = imin(16, PL);
  static constexpr int T = PL / E;
  static constexpr int NT = 256;
  static constexpr int PPW = imax(1, imin(NT / T, (48 * 1024) / (PRP * 8)));  // pairs per workgroup
};

template <int PL, bool CIRC, typename TS, bool ACT = false>
__global__ void __launch_bounds__(256)
    mp_rows_inv(const float2* __restrict__ ws, const TS* __restrict__ x2, TS* __restrict__ y, int64_t line0,
                int nlines, int rows, int L1, int P1, int HS, int64_t per_line) {
  using Cf = RowsInvCfg<PL>;
  constexpr int H = Cf::H, PRP = Cf::PRP, E = Cf::E, T = Cf::T, NT = Cf::NT, PPW = Cf::PPW;
  constexpr int LL = CIRC ? PL : PL / 2;
  constexpr int ML = PL / 2;
  __shared__ float2 reg[PPW * PRP];
  __shared__ float2 twl[imax(1, PassTw<PL, E>::kCount)];
  __shared__ int64_t roff[2 * PPW];
  const int64_t total_pairs = (int64_t)nlines * rows / 2;
  const int64_t pair0 = (int64_t)blockIdx.x * PPW;
  const int npair = (int)((total_pairs - pair0) < PPW ? (total_pairs - pair0) : PPW);
  const int tid = threadIdx.x;
  PassTw<PL, E>::fill(twl, tid, NT);
  ws_row_offsets<2 * PPW, NT>(roff, 2 * pair0, 2 * npair, rows, L1, P1, HS, per_line, tid);
  __syncthreads();

  // load the half-spectrum rows of each pair: row a at [0, H), row b at [H, 2H)
  batched_copy<PPW * 2 * H, NT, 8>(
      tid,
      [&](int i) {
        const int q = i / (2 * H), rem = i - q * 2 * H;
        const int ab = rem / H, f = rem - ab * H;
        float2 z = czero();
        if (q < npair) z = ws[roff[2 * q + ab] + f];
        return z;
      },
      [&](int i, float2 z) {
        const int q = i / (2 * H);
        reg[q * PRP + (i - q * 2 * H)] = z;
      });
  __syncthreads();

  // the T lanes of a pair are consecutive (a wavefront holds 64 / T pairs):
  // with the padded scratch every exchange of the 512-point transform reaches
  // 32 distinct bank pairs
  for (int q0 = 0; q0 < PPW; q0 += NT / T) {
    const int q = q0 + tid / T, t = tid % T;
    const bool act = q < npair;
    float2* R = reg + (act ? q : 0) * PRP;
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
    const ScrPad16 sc{R};
    BlockFFT<PL, E, true>::run(w, t, sc, act, twl);
    if (act) {
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const int n = t + T * e;
        if (CIRC || n < LL) *sc(n) = w[e];
      }
    }
  }
  __syncthreads();

  // gate and store; the rows of a pair are consecutive in y, 4 values per access
  const size_t gbase = (size_t)(line0 * rows + 2 * pair0) * LL;
  if constexpr (LL % 4 == 0) {
    batched_copy<PPW * 2 * (LL / 4), NT, 8>(
        tid,
        [&](int i4) {
          const int i = 4 * i4;
          return (i / LL) < 2 * npair ? Gates<ACT>{}.g4(ld4(x2 + gbase + i)) : make_float4(0.f, 0.f, 0.f, 0.f);
        },
        [&](int i4, float4 g) {
          const int i = 4 * i4;
          const int row = i / LL, n = i - row * LL;
          if (row < 2 * npair) {
            // n is a multiple of 4, so n .. n + 3 share one 16-entry block
            const float2* R = reg + (row >> 1) * PRP + n + (n >> 4);
            float4 o;
            if (row & 1)
              o = make_float4(g.x * R[0].y, g.y * R[1].y, g.z * R[2].y, g.w * R[3].y);
            else
              o = make_float4(g.x * R[0].x, g.y * R[1].x, g.z * R[2].x, g.w * R[3].x);
            st4(y + gbase + i, o);
          }
        });
  } else {
    for (int i = tid; i < npair * 2 * LL; i += NT) {
      const int row = i / LL, n = i - row * LL;
      const float2 qv = reg[(row >> 1) * PRP + n + (n >> 4)];
      st1(y + gbase + i, Gates<ACT>{}.g1(ld1(x2 + gbase + i)) * ((row & 1) ? qv.y : qv.x));
    }
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
  const int nsig = L.g.kc ? 1 : 2;  // a centered K has rows of its own (rows_kc)
#define HY_ARGS(TS) (const TS*)a.x1, (const TS*)a.v, (const TS*)a.k, L.ws, L.line0, L.nl, L.g.rows, L.g.L1, L.g.P1, \
                    L.g.HS, L.g.half, L.per, a.kC, nsig, a.act_in, (int)a.C
#define HY_LAUNCH(CI, TS)                                                                                     \
  if (a.act) hipLaunchKernelGGL((mp_rows_fwd<PL, CI, TS, true>), grid, dim3(256), 0, L.s, HY_ARGS(TS)); \
  else hipLaunchKernelGGL((mp_rows_fwd<PL, CI, TS, false>), grid, dim3(256), 0, L.s, HY_ARGS(TS));
  if (a.bf16) {
    if (a.circular) { HY_LAUNCH(true, uint16_t) } else { HY_LAUNCH(false, uint16_t) }
  } else {
    if (a.circular) { HY_LAUNCH(true, float) } else { HY_LAUNCH(false, float) }
  }
#undef HY_LAUNCH
#undef HY_ARGS
  return hipGetLastError();
}

template <int PL>
hipError_t rows_kc(const MpLaunch& L) {
  const FftConvArgs& a = *L.a;
  constexpr int RPW = 2 * RowsCfg<PL>::RPW;
  const int krows = L.g.P0 * L.g.P1;
  const int64_t total = (int64_t)L.nl * krows;
  const dim3 grid((unsigned)((total + RPW - 1) / RPW));
  if (a.bf16)
    hipLaunchKernelGGL((mp_rows_kc<PL, uint16_t>), grid, dim3(256), 0, L.s, (const uint16_t*)a.k, L.ws, L.line0, L.nl,
                       krows, L.g.L0, L.g.L1, L.g.P1, L.g.HS, L.g.half, L.per, a.kC);
  else
    hipLaunchKernelGGL((mp_rows_kc<PL, float>), grid, dim3(256), 0, L.s, (const float*)a.k, L.ws, L.line0, L.nl,
                       krows, L.g.L0, L.g.L1, L.g.P1, L.g.HS, L.g.half, L.per, a.kC);
  return hipGetLastError();
}

template <int P1, bool INV, int NS>
hipError_t axis1_sig(const MpLaunch& L, int planes, int nload, int64_t sig_off) {
  constexpr int TL = TileCfg<P1, NS>::TL;
  const int ntile = (L.g.H + TL - 1) / TL;
  const dim3 grid((unsigned)((int64_t)L.nl * planes * ntile));
  if (L.a->circular)
    hipLaunchKernelGGL((mp_axis1<P1, true, INV, NS>), grid, dim3(kTileNT), 0, L.s, L.ws, L.g.H, L.g.HS, planes,
                       L.g.half, L.per, nload, sig_off);
  else
    hipLaunchKernelGGL((mp_axis1<P1, false, INV, NS>), grid, dim3(kTileNT), 0, L.s, L.ws, L.g.H, L.g.HS, planes,
                       L.g.half, L.per, nload, sig_off);
  return hipGetLastError();
}

// forward: U and K in one pass (a centered K, with P0 planes of P1 nonzero
// rows, in a pass of its own); inverse: Y
template <int P1, bool INV>
hipError_t axis1(const MpLaunch& L) {
  if (INV) return axis1_sig<P1, true, 1>(L, L.g.L0, P1, 0);
  if (!L.g.kc) return axis1_sig<P1, false, 2>(L, L.g.L0, L.g.L1, 0);
  hipError_t e = axis1_sig<P1, false, 1>(L, L.g.L0, L.g.L1, 0);
  if (e != hipSuccess) return e;
  return axis1_sig<P1, false, 1>(L, L.g.P0, P1, L.g.half);
}
template <int P1>
hipError_t axis1_fwd(const MpLaunch& L) { return axis1<P1, false>(L); }
template <int P1>
hipError_t axis1_inv(const MpLaunch& L) { return axis1<P1, true>(L); }

template <int P0>
hipError_t core(const MpLaunch& L) {
  const FftConvArgs& a = *L.a;
  const int ncols = L.g.P1 * L.g.HS;
  auto launch = [&](auto circ) {
    constexpr bool CI = decltype(circ)::value;
    constexpr int TL = CoreCfg<P0, CI>::TL;
    const int rows = ncols / L.g.HS;
    const int nyq = rows > 1 && (L.g.H - 1) % TL == 0 && L.g.H - 1 >= TL;
    const int64_t ntile = nyq ? (int64_t)rows * ((L.g.H - 1) / TL) + (rows + TL - 1) / TL : (ncols + TL - 1) / TL;
    hipLaunchKernelGGL((mp_core<P0, CI>), dim3((unsigned)(L.nl * ntile)), dim3(CoreCfg<P0, CI>::NT), 0, L.s, L.ws,
                       a.D, (int)a.bf16, L.line0, (int)a.C, ncols, L.g.HS, L.g.H, L.g.half, L.per, L.scale,
                       L.g.krows0, nyq);
  };
  if (a.circular) launch(std::true_type{});
  else launch(std::false_type{});
  return hipGetLastError();
}

template <int PL>
hipError_t rows_inv(const MpLaunch& L) {
  const int64_t pairs = (int64_t)L.nl * L.g.rows / 2;
  const dim3 grid((unsigned)((pairs + RowsInvCfg<PL>::PPW - 1) / RowsInvCfg<PL>::PPW));
  const FftConvArgs& a = *L.a;
#define HY_ARGS(TS) L.ws, (const TS*)a.x2, (TS*)a.y, L.line0, L.nl, L.g.rows, L.g.L1, L.g.P1, L.g.HS, L.per
#define HY_LAUNCH(CI, TS)                                                                                     \
  if (a.act) hipLaunchKernelGGL((mp_rows_inv<PL, CI, TS, true>), grid, dim3(256), 0, L.s, HY_ARGS(TS)); \
  else hipLaunchKernelGGL((mp_rows_inv<PL, CI, TS, false>), grid, dim3(256), 0, L.s, HY_ARGS(TS));
  if (a.bf16) {
    if (a.circular) { HY_LAUNCH(true, uint16_t) } else { HY_LAUNCH(false, uint16_t) }
  } else {
    if (a.circular) { HY_LAUNCH(true, float) } else { HY_LAUNCH(false, float) }
  }
#undef HY_LAUNCH
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
hipError_t d_rows_kc(int P, const MpLaunch& L) { HY_SIZE_SWITCH(P, rows_kc, L) }
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
  return (size_t)(g.half + g.halfK) * sizeof(float2);
}

hipError_t launch_multipass(const FftConvArgs& a, int64_t line0, int64_t nl, void* ws, hipStream_t s) {
  if (!multipass_supported(a) || nl < 1 || line0 < 0 || line0 + nl > a.lines) return hipErrorInvalidValue;
  MpLaunch L;
  L.a = &a;
  L.g = mp_geom(a);
  L.ws = (float2*)ws;
  L.per = L.g.half + L.g.halfK;
  L.scale = (float)(1.0 / (4.0 * (double)L.g.P0 * (double)L.g.P1 * (double)L.g.PL));
  L.s = s;
  L.line0 = line0;
  L.nl = (int)nl;
  const bool three = a.ndim == 3;
  hipError_t e;
  if (three && slab3d_supported(a)) {  // slab, line, slab
    if ((e = launch_slab3d(a, line0, nl, ws, false, s)) != hipSuccess) return e;
    if ((e = d_core(L.g.P0, L)) != hipSuccess) return e;
    return launch_slab3d(a, line0, nl, ws, true, s);
  }
  if ((e = d_rows_fwd(L.g.PL, L)) != hipSuccess) return e;
  if (L.g.kc && (e = d_rows_kc(L.g.PL, L)) != hipSuccess) return e;
  if (three && (e = d_axis1_fwd(L.g.P1, L)) != hipSuccess) return e;
  if ((e = d_core(L.g.P0, L)) != hipSuccess) return e;
  if (three && (e = d_axis1_inv(L.g.P1, L)) != hipSuccess) return e;
  return d_rows_inv(L.g.PL, L);
}

}  // namespace hyenand
