// Backward of the gated long convolution, single pass per (b, c) line.
//
// With gy = dLoss/dy, u = x1 v, h = gy x2 and z = k * u + D u (the pre-gate
// output), the gradients are
//
//   gx2 = gy z,   gu = k (*)^T h + D h,   gk[m] = sum_n h[n] u[n - m],
//   gx1 = gu v,   gv = gu x1,             gD[c] = sum_{b, n} h u,
//
// where (*)^T is the adjoint of the convolution (a correlation).  On the
// transform grid of the forward pass this is three products of the spectra
// U, K, H of u, k, h:
//
//   Z = U (K + D),   GU = conj(K + D) H,   GK = conj(U) H,
//
// inverse-transformed and cropped exactly like the forward output (zero
// padding to 2 L per axis makes the cyclic correlations equal the linear ones
// on the kept range).  Each kernel stages u, k, h, runs three forward real
// transforms, the three products and three inverse real transforms, and
// writes gx1, gx2, gv and gk once; the per-line sums of h u for gD go to the
// workspace and a second small kernel adds them over the samples in order.
#include "kernels.hpp"

namespace hyenand {

namespace {

// Sum of one float over a workgroup of NT lanes (NT a multiple of 64);
// red holds NT / 64 floats.  Every lane calls it; lane 0 gets the total.
template <int NT>
__device__ __forceinline__ float block_sum(float x, float* red, int tid) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o, 64);
  if ((tid & 63) == 0) red[tid >> 6] = x;
  __syncthreads();
  float s = 0.f;
  if (tid == 0) {
#pragma unroll
    for (int w = 0; w < NT / 64; ++w) s += red[w];
  }
  return s;
}

// The three spectral products for one bin (inputs are the doubled R2C
// outputs 2U, 2K s, 2H with s the inverse-transform normalisation; twoD =
// 2 D s): Z = U (K + D), GU = conj(K + D) H, GK = conj(U) H, all scaled by
// 4 s so that the unnormalised inverses return the cropped gradients.
struct Prod3 {
  float2 z, gu, gk;
};
__device__ __forceinline__ Prod3 products(float2 U2, float2 K2s, float2 H2, float twoDs, float s) {
  const float2 kd = make_float2(K2s.x + twoDs, K2s.y);
  Prod3 p;
  p.z = c_mul(U2, kd);
  p.gu = c_mulc(H2, kd);                // H conj(K + D)
  p.gk = c_scale(c_mulc(H2, U2), s);    // H conj(U)
  return p;
}

// ---------------------------------------------------------------------------
// 1D: one workgroup per line, three packed lines of M = P/2 in LDS.
// ---------------------------------------------------------------------------
template <int P, bool CIRC>
struct Bwd1D {
  static constexpr int L = CIRC ? P : P / 2;
  static constexpr int M = P / 2;
  static constexpr int MNZ = (L + 1) / 2;
  static constexpr int E = imin(16, M);
  static constexpr int T = M / E;
  static constexpr int NT = imax(64, ((3 * T + 63) / 64) * 64);
  static constexpr int LDSN = pad16_size(M);
};

constexpr int bwd1d_nt(int P) { return imax(64, ((3 * ((P / 2) / imin(16, P / 2)) + 63) / 64) * 64); }

template <int P, bool CIRC, typename TS>
__global__ void __launch_bounds__(bwd1d_nt(P))
    bwd1d_fused(const TS* __restrict__ x1, const TS* __restrict__ x2, const TS* __restrict__ v,
                const TS* __restrict__ k, const TS* __restrict__ Dp, const TS* __restrict__ gy,
                TS* __restrict__ gx1, TS* __restrict__ gx2, TS* __restrict__ gv, TS* __restrict__ gk,
                float* __restrict__ partial, int C) {
  using F = Bwd1D<P, CIRC>;
  constexpr int L = F::L, M = F::M, MNZ = F::MNZ, E = F::E, T = F::T, NT = F::NT;
  static_assert(NT == bwd1d_nt(P), "threads");
  __shared__ float2 buf[3][F::LDSN];  // u, k, h packed lines (then z, gu, gk)
  __shared__ float red[NT / 64];
  const int line = blockIdx.x;
  const int c = line % C;
  const size_t base = (size_t)line * L;
  const int tid = threadIdx.x;
  constexpr float s = 1.f / (4.f * (float)P);  // normalisation, a power of two

  // stage u = x1 v, k s and h = gy x2 as even/odd packed lines; sum h u
  float hu = 0.f;
  if constexpr (L >= 2) {
    for (int m = tid; m < MNZ; m += NT) {
      const float2 a = ld2(x1 + base + 2 * m), b = ld2(v + base + 2 * m), kk = ld2(k + base + 2 * m);
      const float2 g = ld2(gy + base + 2 * m), e2 = ld2(x2 + base + 2 * m);
      const float2 u = make_float2(a.x * b.x, a.y * b.y), h = make_float2(g.x * e2.x, g.y * e2.y);
      buf[0][m + (m >> 4)] = u;
      buf[1][m + (m >> 4)] = make_float2(kk.x * s, kk.y * s);
      buf[2][m + (m >> 4)] = h;
      hu += u.x * h.x + u.y * h.y;
    }
  } else if (tid == 0) {  // a single sample
    const float u = ld1(x1 + base) * ld1(v + base), h = ld1(gy + base) * ld1(x2 + base);
    buf[0][0] = make_float2(u, 0.f);
    buf[1][0] = make_float2(ld1(k + base) * s, 0.f);
    buf[2][0] = make_float2(h, 0.f);
    hu = u * h;
  }
  const float tot = block_sum<NT>(hu, red, tid);  // its barrier also publishes the staging
  if (tid == 0) partial[line] = tot;

  // forward half-length transforms of the three packed lines
  const int which = tid / T, t = tid % T;
  const bool act = which < 3;
  {
    const ScrPad16 scr{buf[act ? which : 0]};
    float2 w[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int m = t + T * e;
      w[e] = (act && m < MNZ) ? *scr(m) : czero();
    }
    BlockFFT<M, E, false>::run(w, t, scr, act);
    if (act) {
#pragma unroll
      for (int e = 0; e < E; ++e) *scr(t + T * e) = w[e];
    }
  }
  __syncthreads();

  // line `which` of the output (0: z, 1: gu, 2: gk): untangle the two spectra
  // it needs at bins g and M - g, form the product, pack it for the
  // half-length inverse
  {
    const float twoDs = 2.f * s * ld1(Dp + c);
    const ScrPad16 su{buf[0]}, sk{buf[1]}, sh{buf[2]};
    float2 w[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int g = t + T * e;
      w[e] = czero();
      if (act) {
        const int gm = (M - g) & (M - 1);
        const float2 tw = twiddle<ilog2(P), false>(g);
        float2 Ug = czero(), Umg = czero(), Kg = czero(), Kmg = czero(), Hg = czero(), Hmg = czero();
        if (which != 2) r2c_pair(*sk(g), *sk(gm), tw, Kg, Kmg);
        if (which != 1) r2c_pair(*su(g), *su(gm), tw, Ug, Umg);
        if (which != 0) r2c_pair(*sh(g), *sh(gm), tw, Hg, Hmg);
        const Prod3 a = products(Ug, Kg, Hg, twoDs, s), b = products(Umg, Kmg, Hmg, twoDs, s);
        const float2 yg = which == 0 ? a.z : (which == 1 ? a.gu : a.gk);
        const float2 ymg = which == 0 ? b.z : (which == 1 ? b.gu : b.gk);
        w[e] = c2r_pair(yg, ymg, tw);
      }
    }
    const ScrPad16 so{buf[act ? which : 0]};
    BlockFFT<M, E, true>::run(w, t, so, act);  // starts with a barrier: every read above is done
    if (act) {
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const int n = 2 * (t + T * e);
        if (n >= L) continue;
        const float2 o = w[e];
        if (which == 0) {
          const float2 g = ld2(gy + base + n);
          st2(gx2 + base + n, make_float2(g.x * o.x, g.y * o.y));
        } else if (which == 1) {
          const float2 a = ld2(x1 + base + n), b = ld2(v + base + n);
          st2(gx1 + base + n, make_float2(o.x * b.x, o.y * b.y));
          st2(gv + base + n, make_float2(o.x * a.x, o.y * a.y));
        } else {
          st2(gk + base + n, o);
        }
      }
    }
  }
}

// L = 1 (a single sample per line) stores one value per tensor
template <bool CIRC, typename TS>
__global__ void __launch_bounds__(64)
    bwd1d_point(const TS* __restrict__ x1, const TS* __restrict__ x2, const TS* __restrict__ v,
                const TS* __restrict__ k, const TS* __restrict__ Dp, const TS* __restrict__ gy,
                TS* __restrict__ gx1, TS* __restrict__ gx2, TS* __restrict__ gv, TS* __restrict__ gk,
                float* __restrict__ partial, int lines, int C) {
  const int line = blockIdx.x * 64 + threadIdx.x;
  if (line >= lines) return;
  const float a = ld1(x1 + line), b = ld1(v + line), kk = ld1(k + line), g = ld1(gy + line), e2 = ld1(x2 + line);
  const float D = ld1(Dp + line % C);
  const float u = a * b, h = g * e2;
  st1(gx2 + line, g * (kk * u + D * u));
  const float gu = (kk + D) * h;
  st1(gx1 + line, gu * b);
  st1(gv + line, gu * a);
  st1(gk + line, h * u);
  partial[line] = h * u;
}

// ---------------------------------------------------------------------------
// 2D: one workgroup per image; the half spectra of u, k and h (nonzero rows
// only) stay in LDS, 3 L0 rows of pitch RP.
// ---------------------------------------------------------------------------
template <int P0, int P1, bool CIRC>
struct Bwd2D {
  static constexpr int L0 = CIRC ? P0 : P0 / 2;
  static constexpr int L1 = CIRC ? P1 : P1 / 2;
  static constexpr int M1 = P1 / 2;
  static constexpr int MNZ = (L1 + 1) / 2;
  static constexpr int RP = M1 + 1;
  static constexpr int NT = 512;
  static constexpr int ER = imin(16, M1), TR = M1 / ER, LR = NT / TR;
  static constexpr int EC = imin(16, P0), TC = P0 / EC, CR = NT / TC;
  static constexpr int EI = imin(8, M1), TI = M1 / EI, RI = NT / TI;
  static constexpr int NROWS = 3 * L0;
  static constexpr size_t kLds = (size_t)(NROWS * RP + 3 * P0) * 8 + 64;
  static_assert(3 * L0 >= P0, "column scratch");
};

template <int P0, int P1, bool CIRC>
constexpr bool bwd2d_fits() {
  return Bwd2D<P0, P1, CIRC>::kLds <= 160 * 1024;
}

template <int P0, int P1, bool CIRC, typename TS>
__global__ void __launch_bounds__(512)
    bwd2d_fused(const TS* __restrict__ x1, const TS* __restrict__ x2, const TS* __restrict__ v,
                const TS* __restrict__ k, const TS* __restrict__ Dp, const TS* __restrict__ gy,
                TS* __restrict__ gx1, TS* __restrict__ gx2, TS* __restrict__ gv, TS* __restrict__ gk,
                float* __restrict__ partial, int C) {
  using F = Bwd2D<P0, P1, CIRC>;
  constexpr int L0 = F::L0, L1 = F::L1, M1 = F::M1, RP = F::RP, NT = F::NT, NROWS = F::NROWS;
  __shared__ float2 SP[NROWS * RP];  // rows of U, then K, then H
  __shared__ float2 NQ[3][P0];       // DC + i Nyquist column of U, K, H
  __shared__ float red[NT / 64];
  float2* const Uh = SP;
  float2* const Kh = SP + L0 * RP;
  float2* const Hh = SP + 2 * L0 * RP;
  const int img = blockIdx.x;
  const int c = img % C;
  const size_t base = (size_t)img * L0 * L1;
  const int tid = threadIdx.x;
  constexpr float s = 1.f / (4.f * (float)P0 * (float)P1);  // a power of two

  // 0. stage u = x1 v, k s, h = gy x2 as packed row pairs; x1, v and gy stay
  //    in registers for the epilogue
  constexpr int NPAIRS = L0 * L1 / 2, JP = (NPAIRS + NT - 1) / NT;
  using R2 = typename Raw2<TS>::type;
  R2 ra[JP], rb[JP], rg[JP];
  float hu = 0.f;
  {
    R2 rk[JP], re[JP];
#pragma unroll
    for (int j = 0; j < JP; ++j) {
      const int i = tid + NT * j;
      if (NPAIRS % NT == 0 || i < NPAIRS) {
        ra[j] = ld2_raw(x1 + base + 2 * i);
        rb[j] = ld2_raw(v + base + 2 * i);
        rk[j] = ld2_raw(k + base + 2 * i);
        rg[j] = ld2_raw(gy + base + 2 * i);
        re[j] = ld2_raw(x2 + base + 2 * i);
      }
    }
#pragma unroll
    for (int j = 0; j < JP; ++j) {
      const int i = tid + NT * j;
      if (NPAIRS % NT == 0 || i < NPAIRS) {
        const int r = i / (L1 / 2), m = i - r * (L1 / 2);
        const float2 a = widen2(ra[j]), b = widen2(rb[j]), kk = widen2(rk[j]);
        const float2 g = widen2(rg[j]), e2 = widen2(re[j]);
        const float2 u = make_float2(a.x * b.x, a.y * b.y), h = make_float2(g.x * e2.x, g.y * e2.y);
        Uh[r * RP + m] = u;
        Kh[r * RP + m] = make_float2(kk.x * s, kk.y * s);
        Hh[r * RP + m] = h;
        hu += u.x * h.x + u.y * h.y;
      }
    }
  }
  const float tot = block_sum<NT>(hu, red, tid);  // its barrier also publishes the staging
  if (tid == 0) partial[img] = tot;

  // 1. forward row transforms of the 3 L0 rows, then untangling (slot 0
  //    keeps DC + i Nyquist of each real row)
  {
    constexpr int E = F::ER, T = F::TR, LR = F::LR;
    using Map = LaneMap<T, NT>;
    static_assert(Map::kLines == LR, "lines per round");
    for (int l0 = 0; l0 < NROWS; l0 += LR) {
      const int l = l0 + Map::line(tid), t = Map::t(tid);
      const bool act = NROWS % LR == 0 || l < NROWS;
      float2* row = SP + (act ? l : 0) * RP;
      float2 w[E];
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const int m = t + T * e;
        w[e] = (act && (CIRC || m < F::MNZ)) ? row[m] : czero();
      }
      BlockFFT<M1, E, false>::run(w, t, ScrS<1>{row}, act);
      if (act) {
#pragma unroll
        for (int e = 0; e < E; ++e) row[t + T * e] = w[e];
      }
    }
    __syncthreads();
    constexpr int NG = imax(1, M1 / 2);
    for (int it = tid; it < NROWS * NG; it += NT) {
      const int l = it % NROWS;
      const int g = it / NROWS;
      float2* row = SP + l * RP;
      float2 xa, xb;
      if (g == 0) {
        r2c_pair(row[0], row[0], make_float2(1.f, 0.f), xa, xb);
        row[0] = make_float2(xa.x, xb.x);
        if constexpr (M1 >= 2) {
          constexpr int h = M1 / 2;
          r2c_pair(row[h], row[h], twiddle<ilog2(P1), false>(h), xa, xb);
          row[h] = xa;
        }
      } else {
        r2c_pair(row[g], row[M1 - g], twiddle<ilog2(P1), false>(g), xa, xb);
        row[g] = xa;
        row[M1 - g] = xb;
      }
    }
  }
  __syncthreads();

  // 2. column groups: forward U, K, H; the three products; inverse of each;
  //    keep rows < L0 (z over U's rows, gu over H's, gk over K's).  Group 0
  //    (DC + i Nyquist) multiplies through LDS on the first wavefronts.
  {
    constexpr int E = F::EC, T = F::TC, CR = F::CR;
    const float twoDs = 2.f * s * ld1(Dp + c);
    for (int c0 = 0; c0 < M1; c0 += CR) {
      using Map = LaneMap<T, NT>;
      static_assert(Map::kLines == CR, "groups per round");
      const int grp = c0 + Map::line(tid), t = Map::t(tid);
      const bool act = M1 % CR == 0 || grp < M1;
      const bool nyq = act && grp == 0;
      const int col = act ? grp : 0;
      const ScrS<RP> sc{SP + col};
      float2 wu[E], wk[E], wh[E];
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const int n = t + T * e;
        const bool nz = act && (CIRC || n < L0);
        wu[e] = nz ? Uh[n * RP + col] : czero();
        wk[e] = nz ? Kh[n * RP + col] : czero();
        wh[e] = nz ? Hh[n * RP + col] : czero();
      }
      BlockFFT<P0, E, false>::run(wu, t, sc, act);
      BlockFFT<P0, E, false>::run(wk, t, sc, act);
      BlockFFT<P0, E, false>::run(wh, t, sc, act);
      // NQ lies outside every group's exchange scratch: no barrier before
      // group 0 writes it
      if (nyq) {
#pragma unroll
        for (int e = 0; e < E; ++e) {
          NQ[0][t + T * e] = wu[e];
          NQ[1][t + T * e] = wk[e];
          NQ[2][t + T * e] = wh[e];
        }
      }
      __syncthreads();
      if (c0 == 0 && tid <= P0 / 2) {
        // item f: bins f and P0 - f of the real columns' spectra A (column 0)
        // and B (column M1), from Z = A + i B: A = (Z[f] + conj Z[-f]) / 2,
        // B = -i (Z[f] - conj Z[-f]) / 2; each product is Hermitian, so at
        // -f it is conj(Ya) + i conj(Yb)
        const int f = tid, fm = (P0 - f) & (P0 - 1);
        float2 pa[3], pb[3];
#pragma unroll
        for (int q = 0; q < 3; ++q) {
          const float2 z = NQ[q][f], zm = NQ[q][fm];
          pa[q] = c_scale(make_float2(z.x + zm.x, z.y - zm.y), 0.5f);
          pb[q] = c_scale(make_float2(z.y + zm.y, zm.x - z.x), 0.5f);
        }
        const Prod3 A = products(pa[0], pa[1], pa[2], twoDs, s), B = products(pb[0], pb[1], pb[2], twoDs, s);
        const float2 ya[3] = {A.z, A.gk, A.gu}, yb[3] = {B.z, B.gk, B.gu};  // slots: z, gk, gu
#pragma unroll
        for (int q = 0; q < 3; ++q) {
          NQ[q][f] = make_float2(ya[q].x - yb[q].y, ya[q].y + yb[q].x);
          if (fm != f) NQ[q][fm] = make_float2(ya[q].x + yb[q].y, yb[q].x - ya[q].y);
        }
      }
      __syncthreads();
      if (nyq) {
#pragma unroll
        for (int e = 0; e < E; ++e) {
          wu[e] = NQ[0][t + T * e];
          wk[e] = NQ[1][t + T * e];
          wh[e] = NQ[2][t + T * e];
        }
      } else {
#pragma unroll
        for (int e = 0; e < E; ++e) {
          const Prod3 p = products(wu[e], wk[e], wh[e], twoDs, s);
          wu[e] = p.z;
          wk[e] = p.gk;
          wh[e] = p.gu;
        }
      }
      BlockFFT<P0, E, true>::run(wu, t, sc, act);
      BlockFFT<P0, E, true>::run(wk, t, sc, act);
      BlockFFT<P0, E, true>::run(wh, t, sc, act);
      __syncthreads();  // scratch reads of the last exchange are done
      if (act) {
#pragma unroll
        for (int e = 0; e < E; ++e) {
          const int n = t + T * e;
          if (CIRC || n < L0) {
            Uh[n * RP + col] = wu[e];
            Kh[n * RP + col] = wk[e];
            Hh[n * RP + col] = wh[e];
          }
        }
      }
    }
  }
  __syncthreads();

  // 3. inverse rows of z, gk, gu: c2r_pair and the half-length inverse leave
  //    out[r][2m] + i out[r][2m+1] in slot m
  {
    constexpr int E = F::EI, T = F::TI, RI = F::RI;
    using Map = LaneMap<T, NT>;
    static_assert(Map::kLines == RI, "rows per round");
    for (int r0 = 0; r0 < NROWS; r0 += RI) {
      const int r = r0 + Map::line(tid), t = Map::t(tid);
      const bool act = NROWS % RI == 0 || r < NROWS;
      float2* row = SP + (act ? r : 0) * RP;
      float2 w[E];
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const int g = t + T * e;
        float2 Yg, Ym;
        if (g == 0) {
          const float2 s0 = row[0];
          Yg = make_float2(s0.x, 0.f);
          Ym = make_float2(s0.y, 0.f);
        } else {
          Yg = row[g];
          Ym = row[M1 - g];
        }
        w[e] = act ? c2r_pair(Yg, Ym, twiddle<ilog2(P1), false>(g)) : czero();
      }
      BlockFFT<M1, E, true>::run(w, t, ScrS<1>{row}, act);
      if (act) {
#pragma unroll
        for (int e = 0; e < E; ++e) {
          const int m = t + T * e;
          if (CIRC || 2 * m < L1) row[m] = w[e];
        }
      }
    }
  }
  __syncthreads();

  // 4. epilogue: gx2 = gy z, gx1 = gu v, gv = gu x1, gk (row pairs)
#pragma unroll
  for (int j = 0; j < JP; ++j) {
    const int i = tid + NT * j;
    if (NPAIRS % NT == 0 || i < NPAIRS) {
      const int r = i / (L1 / 2), m = i - r * (L1 / 2);
      const float2 z = Uh[r * RP + m], gkv = Kh[r * RP + m], guv = Hh[r * RP + m];
      const float2 a = widen2(ra[j]), b = widen2(rb[j]), g = widen2(rg[j]);
      st2(gx2 + base + 2 * i, make_float2(g.x * z.x, g.y * z.y));
      st2(gx1 + base + 2 * i, make_float2(guv.x * b.x, guv.y * b.y));
      st2(gv + base + 2 * i, make_float2(guv.x * a.x, guv.y * a.y));
      st2(gk + base + 2 * i, gkv);
    }
  }
}

// gD[c] = sum over samples b (in order) of the per-line sums
template <typename TS>
__global__ void __launch_bounds__(256) bwd_reduce_D(const float* __restrict__ partial, TS* __restrict__ gD, int B,
                                                    int C) {
  const int c = blockIdx.x * 256 + threadIdx.x;
  if (c >= C) return;
  float acc = 0.f;
  for (int b = 0; b < B; ++b) acc += partial[(size_t)b * C + c];
  st1(gD + c, acc);
}

#define HY_BWD1D_SIZES(X) X(2) X(4) X(8) X(16) X(32) X(64) X(128) X(256) X(512) X(1024) X(2048) X(4096) X(8192)
#define HY_BWD2D_SIZES(X) \
  X(4, 4) X(8, 8) X(16, 16) X(32, 32) X(64, 64) X(128, 128) X(64, 128) X(128, 64) X(32, 64) X(64, 32)

template <int P, bool CIRC, typename TS>
hipError_t launch_bwd1d_t(const FftConvBwdArgs& b, hipStream_t s) {
  const FftConvArgs& a = b.f;
  hipLaunchKernelGGL((bwd1d_fused<P, CIRC, TS>), dim3((unsigned)a.lines), dim3(bwd1d_nt(P)), 0, s, (const TS*)a.x1,
                     (const TS*)a.x2, (const TS*)a.v, (const TS*)a.k, (const TS*)a.D, (const TS*)b.gy, (TS*)b.gx1,
                     (TS*)b.gx2, (TS*)b.gv, (TS*)b.gk, b.partial, (int)a.C);
  return hipGetLastError();
}

template <int P0, int P1, bool CIRC, typename TS>
hipError_t launch_bwd2d_t(const FftConvBwdArgs& b, hipStream_t s) {
  const FftConvArgs& a = b.f;
  if constexpr (bwd2d_fits<P0, P1, CIRC>()) {
    hipLaunchKernelGGL((bwd2d_fused<P0, P1, CIRC, TS>), dim3((unsigned)a.lines), dim3(512), 0, s,
                       (const TS*)a.x1, (const TS*)a.x2, (const TS*)a.v, (const TS*)a.k, (const TS*)a.D,
                       (const TS*)b.gy, (TS*)b.gx1, (TS*)b.gx2, (TS*)b.gv, (TS*)b.gk, b.partial, (int)a.C);
    return hipGetLastError();
  } else {
    return hipErrorInvalidValue;
  }
}

template <typename TS>
hipError_t launch_typed(const FftConvBwdArgs& b, hipStream_t s) {
  const FftConvArgs& a = b.f;
  hipError_t e = hipErrorInvalidValue;
  if (a.ndim == 1 && a.L[0] == 1) {
    const int lines = (int)a.lines;
    hipLaunchKernelGGL((bwd1d_point<false, TS>), dim3((unsigned)((lines + 63) / 64)), dim3(64), 0, s,
                       (const TS*)a.x1, (const TS*)a.x2, (const TS*)a.v, (const TS*)a.k, (const TS*)a.D,
                       (const TS*)b.gy, (TS*)b.gx1, (TS*)b.gx2, (TS*)b.gv, (TS*)b.gk, b.partial, lines, (int)a.C);
    e = hipGetLastError();
  } else if (a.ndim == 1) {
#define HY_CASE(p) \
  if (a.P[0] == p) e = a.circular ? launch_bwd1d_t<p, true, TS>(b, s) : launch_bwd1d_t<p, false, TS>(b, s);
    HY_BWD1D_SIZES(HY_CASE)
#undef HY_CASE
  } else if (a.ndim == 2) {
#define HY_CASE(p0, p1)                                                                                          \
  if (a.P[0] == p0 && a.P[1] == p1)                                                                              \
    e = a.circular ? launch_bwd2d_t<p0, p1, true, TS>(b, s) : launch_bwd2d_t<p0, p1, false, TS>(b, s);
    HY_BWD2D_SIZES(HY_CASE)
#undef HY_CASE
  }
  if (e != hipSuccess) return e;
  const int C = (int)a.C, B = (int)(a.lines / a.C);
  hipLaunchKernelGGL((bwd_reduce_D<TS>), dim3((unsigned)((C + 255) / 256)), dim3(256), 0, s, b.partial, (TS*)b.gD,
                     B, C);
  return hipGetLastError();
}

}  // namespace

bool fused_backward_supported(const FftConvArgs& a) {
  if (a.ndim == 1) {
    if (a.L[0] == 1) return true;
#define HY_CASE(p) \
  if (a.P[0] == p) return true;
    HY_BWD1D_SIZES(HY_CASE)
#undef HY_CASE
    return false;
  }
  if (a.ndim == 2) {
#define HY_CASE(p0, p1) \
  if (a.P[0] == p0 && a.P[1] == p1) return a.circular ? bwd2d_fits<p0, p1, true>() : bwd2d_fits<p0, p1, false>();
    HY_BWD2D_SIZES(HY_CASE)
#undef HY_CASE
  }
  return false;
}

hipError_t launch_backward(const FftConvBwdArgs& b, hipStream_t s) {
  return b.f.bf16 ? launch_typed<uint16_t>(b, s) : launch_typed<float>(b, s);
}

}  // namespace hyenand
