// Single-pass kernels for grid extents that are not powers of two (linear and
// centered modes).  A non-circular convolution of L points is exact on any
// transform length P >= 2L - 1 (every displacement between two grid points
// then has its own bin, with no wrap-around), so these kernels run the
// power-of-two transforms of the single-pass plans, P = the smallest power of
// two >= 2L - 1 per axis, on grids of L points known at run time: inputs are
// gathered point by point (rows of odd length are not pair-aligned), the zero
// padding is never stored, and the crop keeps the first L points.
//
//  * conv1d_rl<P>: 1D lines, P <= 16384.
//  * conv2d_rl<P0, P1>: 2D images whose U and K half spectra fit in LDS side
//    by side (linear: L0 + L0 rows; centered: L0 + P0 rows).
//
// The circular mode takes these kernels too: a circular convolution of L
// points equals the centred one whose kernel holds k[d mod L] at every
// displacement d = -(L-1) .. L-1 (n - m covers exactly that range), so KC
// with per = true gathers k periodically onto the grid.
#include "kernels.hpp"

namespace hyenand {

namespace {

// index of the kernel value at grid point g of a line of L points on a
// transform of P: centred kernel (per = false) or circular kernel repeated
// periodically (per = true); -1 where no displacement lands
__device__ __forceinline__ int kmap(int g, int L, int P, bool per) {
  return per ? periodic_index(g, L, P) : centered_index(g, L, P);
}

// value of that kernel at grid point g (0 where no displacement lands)
template <typename TS>
__device__ __forceinline__ float kc_at(const TS* kl, int g, int L, int P, bool per) {
  const int j = kmap(g, L, P, per);
  return j >= 0 ? ld1(kl + j) : 0.f;
}

constexpr int rl1d_nt(int P) { return imax(64, imax(2 * ((P / 2) / imin(16, P / 2)), (P / 2) / imin(8, P / 2))); }

template <int P, bool KC, typename TS, bool ACT>
__global__ void __launch_bounds__(rl1d_nt(P))
    conv1d_rl(const TS* __restrict__ x1, const TS* __restrict__ x2, const TS* __restrict__ v,
              const TS* __restrict__ k, const TS* __restrict__ Dp, TS* __restrict__ y, int C, int kC, int L,
              ActIn ain, bool per) {
  constexpr int M = P / 2;
  constexpr int EF = imin(16, M), TF = M / EF;
  constexpr int EI = imin(8, M), TI = M / EI;
  constexpr int NT = rl1d_nt(P);
  constexpr int LDSN = pad16_size(M);
  __shared__ float2 Ub[LDSN];
  __shared__ float2 Kb[LDSN];
  const int line = blockIdx.x;
  const int c = line % C;
  const size_t base = (size_t)line * L;
  const int tid = threadIdx.x;
  const Gates<ACT> G = line_gates<ACT, TS>(ain, line, C);
  const int MNZ = (L + 1) / 2;
  const int KNZ = KC ? M : MNZ;  // packed points of k that can be nonzero
  const TS* kl = k + (size_t)k_line(line, kC) * (KC && !per ? 2 * L - 1 : L);

  // stage u = x1 v and k as even/odd packed lines, point by point
  for (int m = tid; m < M; m += NT) {
    float2 u = czero(), kk = czero();
    if (m < MNZ) {
      const int n = 2 * m;
      u.x = G.u1(ld1(x1 + base + n), ld1(v + base + n), n);
      if (n + 1 < L) u.y = G.u1(ld1(x1 + base + n + 1), ld1(v + base + n + 1), n + 1);
    }
    if (KC) {
      kk = make_float2(kc_at(kl, 2 * m, L, P, per), kc_at(kl, 2 * m + 1, L, P, per));
    } else if (m < MNZ) {
      kk.x = ld1(kl + 2 * m);
      if (2 * m + 1 < L) kk.y = ld1(kl + 2 * m + 1);
    }
    Ub[m + (m >> 4)] = u;
    Kb[m + (m >> 4)] = kk;
  }
  __syncthreads();

  {
    const int which = tid / TF, t = tid % TF;
    const bool act = which < 2;
    const ScrPad16 scr{which == 0 ? Ub : Kb};
    const int nz = which == 0 ? MNZ : KNZ;
    float2 w[EF];
#pragma unroll
    for (int e = 0; e < EF; ++e) {
      const int m = t + TF * e;
      w[e] = (act && m < nz) ? *scr(m) : czero();
    }
    BlockFFT<M, EF, false>::run(w, t, scr, act);
    if (act) {
#pragma unroll
      for (int e = 0; e < EF; ++e) *scr(t + TF * e) = w[e];
    }
  }
  __syncthreads();

  {
    const float twoD = 2.f * ld1(Dp + c);
    const float scale = 1.f / (4.f * (float)P);
    const ScrPad16 su{Ub}, sk{Kb};
    const int t = tid;
    const bool act = t < TI;
    float2 w[EI];
#pragma unroll
    for (int e = 0; e < EI; ++e) {
      const int g = t + TI * e;
      w[e] = czero();
      if (act) {
        const int gm = (M - g) & (M - 1);
        const float2 tw = twiddle<ilog2(P), false>(g);
        float2 Ug, Umg, Kg, Kmg;
        r2c_pair(*su(g), *su(gm), tw, Ug, Umg);
        r2c_pair(*sk(g), *sk(gm), tw, Kg, Kmg);
        w[e] = c_scale(c2r_pair(gated_product(Ug, Kg, twoD), gated_product(Umg, Kmg, twoD), tw), scale);
      }
    }
    if constexpr (TI == 1) __syncthreads();
    BlockFFT<M, EI, true>::run(w, t, su, act);
    if (act) {
#pragma unroll
      for (int e = 0; e < EI; ++e) {
        const int n = 2 * (t + TI * e);
        if (n < L) st1(y + base + n, G.g1(ld1(x2 + base + n)) * w[e].x);
        if (n + 1 < L) st1(y + base + n + 1, G.g1(ld1(x2 + base + n + 1)) * w[e].y);
      }
    }
  }
}

// 2D: U rows [0, P0/2) then K rows [0, KR) of the half spectrum in LDS (KR =
// P0/2 linear, P0 centered); column c of the whole array is the exchange
// scratch of that column's transforms (>= P0 slots).  Group 0 carries the DC
// and Nyquist columns as one complex column, split with the mirror bin.
template <int P0, int P1, bool KC, typename TS, bool ACT>
__global__ void __launch_bounds__(512)
    conv2d_rl(const TS* __restrict__ x1, const TS* __restrict__ x2, const TS* __restrict__ v,
              const TS* __restrict__ k, const TS* __restrict__ Dp, TS* __restrict__ y, int C, int kC, int L0,
              int L1, ActIn ain, bool per) {
  constexpr int M1 = P1 / 2, RP = M1 + 1, NT = 512;
  constexpr int L0M = P0 / 2;
  constexpr int KRM = KC ? P0 : L0M;
  constexpr int ER = imin(16, M1), TR = M1 / ER, LR = NT / TR;
  constexpr int EC = imin(16, P0), TC = P0 / EC, CR = NT / TC;
  constexpr int EI = imin(8, M1), TI = M1 / EI, RI = NT / TI;
  static_assert(L0M + KRM >= P0, "column scratch");
  __shared__ float2 UK[(L0M + KRM) * RP];
  float2* const Uh = UK;
  float2* const Kh = UK + L0M * RP;
  const int img = blockIdx.x;
  const int c = img % C;
  const size_t base = (size_t)img * L0 * L1;
  const int tid = threadIdx.x;
  const Gates<ACT> G = line_gates<ACT, TS>(ain, img, C);
  const int MNZ = (L1 + 1) / 2;        // packed points per nonzero row
  const int KR = KC ? P0 : L0;         // K rows that can be nonzero
  const int KNZ = KC ? M1 : MNZ;
  const int KL1 = KC && !per ? 2 * L1 - 1 : L1;  // kernel row length
  const TS* kl = k + (size_t)k_line(img, kC) * (KC && !per ? (2 * L0 - 1) * (2 * L1 - 1) : L0 * L1);
  constexpr float scale = 1.f / (4.f * (float)P0 * (float)P1);

  // 0. stage u and k rows as packed pairs (k scaled by the normalisation)
  for (int i = tid; i < L0 * MNZ; i += NT) {
    const int r = i / MNZ, m = i - r * MNZ;
    const int n = 2 * m;
    const size_t o = base + (size_t)r * L1 + n;
    float2 u;
    u.x = G.u1(ld1(x1 + o), ld1(v + o), (int64_t)r * L1 + n);
    u.y = n + 1 < L1 ? G.u1(ld1(x1 + o + 1), ld1(v + o + 1), (int64_t)r * L1 + n + 1) : 0.f;
    Uh[r * RP + m] = u;
    if constexpr (!KC) {
      const TS* kr = kl + (size_t)r * L1 + n;
      Kh[r * RP + m] = make_float2(ld1(kr) * scale, n + 1 < L1 ? ld1(kr + 1) * scale : 0.f);
    }
  }
  if constexpr (KC) {
    for (int i = tid; i < P0 * M1; i += NT) {
      const int g0 = i / M1, m = i - g0 * M1;
      const int j0 = kmap(g0, L0, P0, per);
      float2 z = czero();
      if (j0 >= 0) {
        const TS* kr = kl + (size_t)j0 * KL1;
        z = make_float2(kc_at(kr, 2 * m, L1, P1, per) * scale, kc_at(kr, 2 * m + 1, L1, P1, per) * scale);
      }
      Kh[g0 * RP + m] = z;
    }
  }
  __syncthreads();

  // 1. row transforms (u rows, then k rows), untangled with DC + i Nyquist in slot 0
  const int NR = L0 + KR;
  for (int l0 = 0; l0 < NR; l0 += LR) {
    const int l = l0 + tid / TR, t = tid % TR;
    const bool act = l < NR;
    float2* row = act ? (l < L0 ? Uh + l * RP : Kh + (l - L0) * RP) : Uh;
    const int nz = l < L0 ? MNZ : KNZ;
    float2 w[ER];
#pragma unroll
    for (int e = 0; e < ER; ++e) {
      const int m = t + TR * e;
      w[e] = (act && m < nz) ? row[m] : czero();
    }
    BlockFFT<M1, ER, false>::run(w, t, ScrS<1>{row}, act);
    if (act) {
#pragma unroll
      for (int e = 0; e < ER; ++e) row[t + TR * e] = w[e];
    }
  }
  __syncthreads();
  {
    constexpr int NG = imax(1, M1 / 2);
    for (int it = tid; it < NR * NG; it += NT) {
      const int l = it % NR, g = it / NR;
      float2* row = l < L0 ? Uh + l * RP : Kh + (l - L0) * RP;
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

  // 2. column groups: forward U and K, product, inverse, keep rows < L0
  {
    const float twoD = 2.f * scale * ld1(Dp + c);
    for (int c0 = 0; c0 < M1; c0 += CR) {
      const int grp = c0 + tid / TC, t = tid % TC;
      const bool act = grp < M1;
      const bool nyq = act && grp == 0;
      const int col = act ? grp : 0;
      float2 wu[EC], wk[EC];
#pragma unroll
      for (int e = 0; e < EC; ++e) {
        const int n = t + TC * e;
        wu[e] = (act && n < L0) ? Uh[n * RP + col] : czero();
        wk[e] = (act && n < KR) ? Kh[n * RP + col] : czero();
      }
      const ScrS<RP> su{UK + col};
      BlockFFT<P0, EC, false>::run(wu, t, su, act);
      BlockFFT<P0, EC, false>::run(wk, t, su, act);
      const ScrS<RP> u0{UK};
      const ScrS<RP> k0{UK + M1};
      __syncthreads();
      if (nyq) {
#pragma unroll
        for (int e = 0; e < EC; ++e) {
          *u0(t + TC * e) = wu[e];
          *k0(t + TC * e) = wk[e];
        }
      }
      __syncthreads();
      if (c0 == 0 && tid <= P0 / 2) {
        const int f = tid, fm = (P0 - f) & (P0 - 1);
        const float2 zu = *u0(f), zum = *u0(fm), zk = *k0(f), zkm = *k0(fm);
        const float2 ua = c_scale(make_float2(zu.x + zum.x, zu.y - zum.y), 0.5f);
        const float2 ub = c_scale(make_float2(zu.y + zum.y, zum.x - zu.x), 0.5f);
        const float2 ka = c_scale(make_float2(zk.x + zkm.x, zk.y - zkm.y), 0.5f);
        const float2 kb = c_scale(make_float2(zk.y + zkm.y, zkm.x - zk.x), 0.5f);
        const float2 ya = gated_product(ua, ka, twoD);
        const float2 yb = gated_product(ub, kb, twoD);
        *u0(f) = make_float2(ya.x - yb.y, ya.y + yb.x);
        if (fm != f) *u0(fm) = make_float2(ya.x + yb.y, yb.x - ya.y);
      }
      __syncthreads();
      if (nyq) {
#pragma unroll
        for (int e = 0; e < EC; ++e) wu[e] = *u0(t + TC * e);
      } else {
#pragma unroll
        for (int e = 0; e < EC; ++e) wu[e] = gated_product(wu[e], wk[e], twoD);
      }
      BlockFFT<P0, EC, true>::run(wu, t, su, act);
      __syncthreads();
      if (act) {
#pragma unroll
        for (int e = 0; e < EC; ++e) {
          const int n = t + TC * e;
          if (n < L0) Uh[n * RP + col] = wu[e];
        }
      }
    }
  }
  __syncthreads();

  // 3. inverse row transforms, two output values per complex point
  for (int r0 = 0; r0 < L0; r0 += RI) {
    const int r = r0 + tid / TI, t = tid % TI;
    const bool act = r < L0;
    float2* row = Uh + (act ? r : 0) * RP;
    float2 w[EI];
#pragma unroll
    for (int e = 0; e < EI; ++e) {
      const int g = t + TI * e;
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
    BlockFFT<M1, EI, true>::run(w, t, ScrS<1>{row}, act);
    if (act) {
#pragma unroll
      for (int e = 0; e < EI; ++e) {
        const int m = t + TI * e;
        if (2 * m < L1) row[m] = w[e];
      }
    }
  }
  __syncthreads();

  // 4. outer gate and store, point by point
  for (int i = tid; i < L0 * L1; i += NT) {
    const int r = i / L1, n = i - r * L1;
    const float2 q = Uh[r * RP + n / 2];
    st1(y + base + i, G.g1(ld1(x2 + base + i)) * ((n & 1) ? q.y : q.x));
  }
}

template <int P, bool KC, typename TS>
hipError_t launch_1d_t(const FftConvArgs& a, hipStream_t s) {
  const int L = (int)a.L[0];
  if (a.act)
    hipLaunchKernelGGL((conv1d_rl<P, KC, TS, true>), dim3((unsigned)a.lines), dim3(rl1d_nt(P)), 0, s,
                       (const TS*)a.x1, (const TS*)a.x2, (const TS*)a.v, (const TS*)a.k, (const TS*)a.D, (TS*)a.y,
                       (int)a.C, a.kC, L, a.act_in, a.periodic);
  else
    hipLaunchKernelGGL((conv1d_rl<P, KC, TS, false>), dim3((unsigned)a.lines), dim3(rl1d_nt(P)), 0, s,
                       (const TS*)a.x1, (const TS*)a.x2, (const TS*)a.v, (const TS*)a.k, (const TS*)a.D, (TS*)a.y,
                       (int)a.C, a.kC, L, a.act_in, a.periodic);
  return hipGetLastError();
}

template <int P>
hipError_t launch_1d_p(const FftConvArgs& a, hipStream_t s) {
  if (a.centered || a.periodic)
    return a.bf16 ? launch_1d_t<P, true, uint16_t>(a, s) : launch_1d_t<P, true, float>(a, s);
  return a.bf16 ? launch_1d_t<P, false, uint16_t>(a, s) : launch_1d_t<P, false, float>(a, s);
}

template <int P0, int P1, bool KC, typename TS>
hipError_t launch_2d_t(const FftConvArgs& a, hipStream_t s) {
  const int L0 = (int)a.L[0], L1 = (int)a.L[1];
  if (a.act)
    hipLaunchKernelGGL((conv2d_rl<P0, P1, KC, TS, true>), dim3((unsigned)a.lines), dim3(512), 0, s, (const TS*)a.x1,
                       (const TS*)a.x2, (const TS*)a.v, (const TS*)a.k, (const TS*)a.D, (TS*)a.y, (int)a.C, a.kC, L0,
                       L1, a.act_in, a.periodic);
  else
    hipLaunchKernelGGL((conv2d_rl<P0, P1, KC, TS, false>), dim3((unsigned)a.lines), dim3(512), 0, s,
                       (const TS*)a.x1, (const TS*)a.x2, (const TS*)a.v, (const TS*)a.k, (const TS*)a.D, (TS*)a.y,
                       (int)a.C, a.kC, L0, L1, a.act_in, a.periodic);
  return hipGetLastError();
}

template <int P0, int P1>
hipError_t launch_2d_p(const FftConvArgs& a, hipStream_t s) {
  if (a.centered || a.periodic)
    return a.bf16 ? launch_2d_t<P0, P1, true, uint16_t>(a, s) : launch_2d_t<P0, P1, true, float>(a, s);
  return a.bf16 ? launch_2d_t<P0, P1, false, uint16_t>(a, s) : launch_2d_t<P0, P1, false, float>(a, s);
}

// every pair of power-of-two transform sizes from 4 to 128 (U and K side by side
// in LDS: at most 100 KB, for a centered 128 x 128)
#define HY_RL2D_SIZES(X) \
  X(4, 4) X(4, 8) X(4, 16) X(4, 32) X(4, 64) X(4, 128) X(8, 4) X(8, 8) X(8, 16) X(8, 32) X(8, 64) \
  X(8, 128) X(16, 4) X(16, 8) X(16, 16) X(16, 32) X(16, 64) X(16, 128) X(32, 4) X(32, 8) X(32, 16) \
  X(32, 32) X(32, 64) X(32, 128) X(64, 4) X(64, 8) X(64, 16) X(64, 32) X(64, 64) X(64, 128) X(128, 4) \
  X(128, 8) X(128, 16) X(128, 32) X(128, 64) X(128, 128)

}  // namespace

bool fused_rl_supported(const FftConvArgs& a) {
  if (a.circular) return false;
  if (a.ndim == 1) return a.P[0] >= 4 && a.P[0] <= 16384;
  if (a.ndim == 2) {
#define HY_CASE(p0, p1) \
  if (a.P[0] == p0 && a.P[1] == p1) return true;
    HY_RL2D_SIZES(HY_CASE)
#undef HY_CASE
  }
  return false;
}

hipError_t launch_fused_rl(const FftConvArgs& a, hipStream_t s) {
  if (!fused_rl_supported(a)) return hipErrorInvalidValue;
  if (a.ndim == 1) {
    switch (a.P[0]) {
      case 4: return launch_1d_p<4>(a, s);
      case 8: return launch_1d_p<8>(a, s);
      case 16: return launch_1d_p<16>(a, s);
      case 32: return launch_1d_p<32>(a, s);
      case 64: return launch_1d_p<64>(a, s);
      case 128: return launch_1d_p<128>(a, s);
      case 256: return launch_1d_p<256>(a, s);
      case 512: return launch_1d_p<512>(a, s);
      case 1024: return launch_1d_p<1024>(a, s);
      case 2048: return launch_1d_p<2048>(a, s);
      case 4096: return launch_1d_p<4096>(a, s);
      case 8192: return launch_1d_p<8192>(a, s);
      case 16384: return launch_1d_p<16384>(a, s);
      default: return hipErrorInvalidValue;
    }
  }
#define HY_CASE(p0, p1) \
  if (a.P[0] == p0 && a.P[1] == p1) return launch_2d_p<p0, p1>(a, s);
  HY_RL2D_SIZES(HY_CASE)
#undef HY_CASE
  return hipErrorInvalidValue;
}

}  // namespace hyenand
