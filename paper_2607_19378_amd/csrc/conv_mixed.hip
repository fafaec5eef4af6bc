// Single-pass kernels on mixed-radix transform grids (extents whose prime
// factors are 2, 3, 5 and 7, known at run time), for grids whose extents are
// not powers of two (section 3.2.2: register rows and patch grids such as
// 14 x 14).
//
// Transform grid, per axis d:
//  * exact: a circular axis whose extent L factors into 2, 3, 5 and 7 is
//    transformed on its own L points (no padding at all);
//  * otherwise the smallest such P >= 2L - 1 (a non-circular convolution is
//    exact on any P >= 2L - 1, every displacement having a bin of its own), k
//    placed at its displacements: linear (k of L points), centered (k of
//    2L - 1 points, displacement -(L-1) .. L-1) or periodic (a circular axis
//    of other extents: k[d mod L] at displacement d).
//
// Arithmetic: two real signals per complex transform, always two of the same
// kind: the u of the two images a, b of a pair in one complex grid
// zu = ua + i ub, their k in zk = ka + i kb.  After the forward transforms
// the mirror bin separates them, Ua(f) = (Zu(f) + conj Zu(-f)) / 2 and
// Ub(f) = (Zu(f) - conj Zu(-f)) / 2i, and so for K.  (Packing u + i k of one
// image instead would give K the rounding error of U, eps |U|, which exceeds
// the fp32 tolerance where |u| >> |k|.)  Each of the two real signals of a
// grid is scaled, exactly, by the power of two that brings its largest
// magnitude into [1/2, 1) before the transforms, and each product by the
// power of two of u's scale times the larger of k's and D's (about the scale
// of y), undone at the store, so that lines of different scales in one pair
// do not pass their rounding error to each other either.  The products Ya
// and Yb (with the shortcut folded in as U (K + D)) go into one grid
// Ya + i Yb, and one more transform of its conjugate gives conj(ya + i yb):
// the inverse of both.  Odd extents need no half-length packing this way, and
// each image costs one and a half complex transforms of the grid.
//
// Each axis runs Stockham passes between two LDS buffers (one barrier per
// pass), each of the largest radix of the kernel's family that divides what
// is left of the axis (every family has 8, 7, 5, 4, 3, 2, and one pair of
// 14 + 12, 16 + 10 or 15 + 9: one pass for a 14-point axis, three for 1000
// points), each butterfly an in-register DFT.  A pass of radix r over an axis
// of P points with stride S, after passes whose radices multiply to Ns:
// butterfly j of a line reads the r points j + t P/r, multiplies point t by
// the twiddle exp(-2 pi i t (j mod Ns) / (Ns r)), takes the r-point DFT and
// writes output t to (j div Ns) Ns r + (j mod Ns) + t Ns; after the last pass
// the axis is in natural order.  Every pass sees the images of the workgroup
// as one list of butterflies, so the lanes stay busy whatever the grid.
//
// The backward (conv_mixed_bwd, further down) runs on the same grids.
#include <stdlib.h>
#include <string.h>

#include <mutex>

#include "kernels.hpp"

namespace hyenand {

namespace {

constexpr int kMrMaxPass = 24;  // passes over all axes
constexpr int kMrMaxN = 4096;   // transform points per image
constexpr size_t kMrMaxLds = 150 * 1024;

// n div d for a run-time d, n < 2^31: (mulhi(n, m) + n) >> l with
// l = ceil(log2 d) and m = floor(2^32 (2^l - d) / d) + 1.
struct FastDiv {
  uint32_t m, l;
};
inline FastDiv make_fastdiv(uint32_t d) {
  uint32_t l = 0;
  while ((uint64_t(1) << l) < d) ++l;
  const uint64_t m = ((uint64_t(1) << 32) * ((uint64_t(1) << l) - d)) / d + 1;
  return FastDiv{(uint32_t)m, l};
}
__device__ __forceinline__ uint32_t fdiv(uint32_t n, FastDiv f) { return (__umulhi(n, f.m) + n) >> f.l; }

enum MrKind : int { MR_EXACT = 0, MR_LINEAR = 1, MR_CENTERED = 2, MR_PERIODIC = 3 };

struct MrPass {
  int r;       // radix
  int q;       // P / r: butterflies per line
  int ns;      // product of the earlier radices of this axis
  int sa;      // stride of the axis in the grid
  int pasa;    // P * sa
  int twoff;   // this axis' twiddles in the table
  int twstep;  // P / (ns r): twiddle index per unit of t (j mod ns)
  FastDiv dsa, dq, dns;
};

// Unit axes lead: a 1D grid is 1 x 1 x P, a 2D grid 1 x P0 x P1.
struct MrPlan {
  int P[3], L[3], KL[3], kind[3];
  int N, Ld, Kd;  // transform, data and kernel points per image
  int Q;          // image pairs per workgroup
  int twoff[3], ntw;
  int nt;         // lanes per workgroup
  int fam;        // radix family of the passes
  int npass;      // forward passes; the inverse runs the same list
  FastDiv dN, dP1, dP2, dL1, dL2, dLd, dC, dKC, dKL1, dKL2, dKd;
  MrPass pass[kMrMaxPass];
};

// ---------------------------------------------------------------------------
// register DFTs of odd radix (3, 5, 7): the points t and R - t in pairs, so
// that each output takes (R - 1) / 2 real cosines and sines
// ---------------------------------------------------------------------------
__host__ __device__ constexpr float odd_cos(int R, int m) {
  return R == 3 ? -0.5f
                : R == 5 ? (m == 1 ? 0.309016994f : -0.809016994f)
                         : (m == 1 ? 0.623489802f : m == 2 ? -0.222520934f : -0.900968868f);
}
__host__ __device__ constexpr float odd_sin(int R, int m) {
  return R == 3 ? 0.866025404f
                : R == 5 ? (m == 1 ? 0.951056516f : 0.587785252f)
                         : (m == 1 ? 0.781831482f : m == 2 ? 0.974927912f : 0.433883739f);
}

template <int R>
__device__ __forceinline__ void dft_odd(float2 (&x)[R]) {
  constexpr int H = (R - 1) / 2;
  float2 a[H], b[H];
#pragma unroll
  for (int t = 1; t <= H; ++t) {
    a[t - 1] = c_add(x[t], x[R - t]);
    b[t - 1] = c_sub(x[t], x[R - t]);
  }
  float2 x0 = x[0];
#pragma unroll
  for (int t = 0; t < H; ++t) x0 = c_add(x0, a[t]);
#pragma unroll
  for (int q = 1; q <= H; ++q) {
    float re = x[0].x, im = x[0].y, sr = 0.f, si = 0.f;
#pragma unroll
    for (int t = 1; t <= H; ++t) {
      const int m = (t * q) % R;
      const int mm = m <= H ? m : R - m;
      const float c = odd_cos(R, mm);
      const float s = m <= H ? odd_sin(R, mm) : -odd_sin(R, mm);
      re = fmaf(a[t - 1].x, c, re);
      im = fmaf(a[t - 1].y, c, im);
      sr = fmaf(b[t - 1].y, s, sr);
      si = fmaf(b[t - 1].x, s, si);
    }
    x[q] = make_float2(re + sr, im - si);
    x[R - q] = make_float2(re - sr, im + si);
  }
  x[0] = x0;
}

// exp(-2 pi i m / R) for m < R, R <= 16, evaluated at compile time (Taylor
// series in double on the angle reduced to [-pi, pi]).
constexpr double kPiD = 3.141592653589793238462643;
constexpr double cx_sin(double x) {
  double term = x, sum = x;
  for (int n = 1; n < 24; ++n) {
    term *= -x * x / ((2.0 * n) * (2.0 * n + 1.0));
    sum += term;
  }
  return sum;
}
constexpr double cx_cos(double x) {
  double term = 1.0, sum = 1.0;
  for (int n = 1; n < 24; ++n) {
    term *= -x * x / ((2.0 * n - 1.0) * (2.0 * n));
    sum += term;
  }
  return sum;
}
template <int R>
struct RootTab {
  float c[R], s[R];
  constexpr RootTab() : c(), s() {
    for (int m = 0; m < R; ++m) {
      const int mm = 2 * m > R ? m - R : m;
      const double th = 2.0 * kPiD * mm / R;
      c[m] = (float)cx_cos(th);
      s[m] = (float)(-cx_sin(th));
    }
  }
};
template <int R>
constexpr RootTab<R> kRoots{};

// a * exp(-2 pi i m / R), m a compile-time constant after unrolling; exact
// for the quarter turns
template <int R>
__device__ __forceinline__ float2 mul_root_c(float2 a, int m) {
  m %= R;
  if (m == 0) return a;
  if (4 * m == R) return make_float2(a.y, -a.x);
  if (2 * m == R) return make_float2(-a.x, -a.y);
  if (4 * m == 3 * R) return make_float2(-a.y, a.x);
  const float c = kRoots<R>.c[m], s = kRoots<R>.s[m];
  return make_float2(fmaf(a.x, c, -a.y * s), fmaf(a.x, s, a.y * c));
}

// largest base radix (8, 7, 5, 4, 3, 2) that divides R and is below it
constexpr int split_radix(int R) {
  for (int a : {8, 7, 5, 4, 3, 2})
    if (a < R && R % a == 0) return a;
  return R;
}
constexpr bool base_radix(int R) { return R == 2 || R == 3 || R == 4 || R == 5 || R == 7 || R == 8; }

// In-register DFT of R points (R <= 16, prime factors <= 7), natural order in
// and out.  Composite R = A B by decimation in time: n = n1 + A n2,
// k = k1 + B k2; B-point DFTs of the A decimated sequences, the twiddles
// exp(-2 pi i n1 k1 / R), then A-point DFTs across them.
template <int R>
__device__ __forceinline__ void dft_reg(float2 (&x)[R]) {
  if constexpr (base_radix(R)) {
    if constexpr (R == 3 || R == 5 || R == 7) dft_odd<R>(x);
    else dft<R, false>(x);
  } else {
    constexpr int A = split_radix(R), B = R / A;
    float2 t[A][B];
#pragma unroll
    for (int n1 = 0; n1 < A; ++n1) {
#pragma unroll
      for (int n2 = 0; n2 < B; ++n2) t[n1][n2] = x[n1 + A * n2];
      dft_reg<B>(t[n1]);
#pragma unroll
      for (int k1 = 0; k1 < B; ++k1) t[n1][k1] = mul_root_c<R>(t[n1][k1], n1 * k1);
    }
#pragma unroll
    for (int k1 = 0; k1 < B; ++k1) {
      float2 u[A];
#pragma unroll
      for (int n1 = 0; n1 < A; ++n1) u[n1] = t[n1][k1];
      dft_reg<A>(u);
#pragma unroll
      for (int k2 = 0; k2 < A; ++k2) x[k1 + B * k2] = u[k2];
    }
  }
}

__device__ __forceinline__ uint32_t umax(uint32_t a, uint32_t b) { return a > b ? a : b; }

// e with |x| 2^-e in [1/2, 1) (0 for 0), for x and for the magnitude whose
// bits are b
__device__ __forceinline__ int mr_fexp(float x) { return __builtin_amdgcn_frexp_expf(x); }
__device__ __forceinline__ int mr_exp(uint32_t b) { return mr_fexp(__uint_as_float(b)); }

// One Stockham pass of radix R over `items` butterflies (all images); TW:
// the pass has twiddles (not the first pass of its axis, where all are 1).
template <int R, int NT, bool TW, bool SC>
__device__ __forceinline__ void mr_pass_t(const float2* src, float2* dst, const float2* tw, const MrPass& ps,
                                          uint32_t items, uint32_t tid, const uint32_t* smx, FastDiv dN) {
  const uint32_t qs = (uint32_t)(ps.q * ps.sa), nss = (uint32_t)(ps.ns * ps.sa);
  for (uint32_t it = tid; it < items; it += NT) {
    const uint32_t t1 = fdiv(it, ps.dsa), s = it - t1 * (uint32_t)ps.sa;
    const uint32_t t2 = fdiv(t1, ps.dq), j = t1 - t2 * (uint32_t)ps.q;
    const uint32_t jn = TW ? fdiv(j, ps.dns) : j, kk = TW ? j - jn * (uint32_t)ps.ns : 0;
    const uint32_t base = t2 * (uint32_t)ps.pasa + s;
    const float2* sp = src + base + j * (uint32_t)ps.sa;
    float2 x[R];
#pragma unroll
    for (int t = 0; t < R; ++t) x[t] = sp[t * qs];
    if constexpr (SC) {  // the staging scales of this grid's two parts
      const uint32_t g = fdiv(base, dN);
      const int ex = -mr_exp(smx[2 * g]), ey = -mr_exp(smx[2 * g + 1]);
#pragma unroll
      for (int t = 0; t < R; ++t) x[t] = make_float2(ldexpf(x[t].x, ex), ldexpf(x[t].y, ey));
    }
    if constexpr (TW) {
      const uint32_t tws = kk * (uint32_t)ps.twstep;
      const float2* tp = tw + ps.twoff;
#pragma unroll
      for (int t = 1; t < R; ++t) x[t] = c_mul(x[t], tp[t * tws]);
    }
    dft_reg<R>(x);
    float2* dp = dst + base + (jn * (uint32_t)(ps.ns * R) + kk) * (uint32_t)ps.sa;
#pragma unroll
    for (int t = 0; t < R; ++t) dp[t * nss] = x[t];
  }
}

// sc: the first pass of the forward transforms, which applies the staging
// scales (it is the first pass of its axis: no twiddles)
template <int R, int NT>
__device__ __forceinline__ void mr_pass(const float2* src, float2* dst, const float2* tw, const MrPass& ps,
                                        uint32_t items, uint32_t tid, bool sc, const uint32_t* smx, FastDiv dN) {
  if (sc) mr_pass_t<R, NT, false, true>(src, dst, tw, ps, items, tid, smx, dN);
  else if (ps.ns == 1) mr_pass_t<R, NT, false, false>(src, dst, tw, ps, items, tid, smx, dN);
  else mr_pass_t<R, NT, true, false>(src, dst, tw, ps, items, tid, smx, dN);
}

// Radix families: every kernel takes 8, 7, 5, 4, 3 and 2, and family f adds
// kFamRadix[f] (more composite radices in one kernel and the compiler keeps
// their arrays in scratch memory instead of registers).
constexpr int kNumFam = 4;
constexpr int kFamRadix[kNumFam][2] = {{0, 0}, {14, 12}, {16, 10}, {15, 9}};
constexpr bool fam_has(int f, int r) {
  return r == 8 || r == 7 || r == 5 || r == 4 || r == 3 || r == 2 || kFamRadix[f][0] == r || kFamRadix[f][1] == r;
}

// every pass of the plan over n points (whole images), ping-ponging src/dst;
// returns with the result in src
// scale: the forward transforms (the first pass applies the staging scales)
template <int NT, int FAM>
__device__ __forceinline__ void mr_transform(float2*& src, float2*& dst, const float2* tw, const MrPass* passes,
                                             int npass, uint32_t n, uint32_t tid, bool scale, const uint32_t* smx,
                                             FastDiv dN) {
  for (int i = 0; i < npass; ++i) {
    const MrPass ps = passes[i];
    const bool sc = scale && i == 0;
    switch (ps.r) {
      case 16: if constexpr (fam_has(FAM, 16)) mr_pass<16, NT>(src, dst, tw, ps, n / 16, tid, sc, smx, dN); break;
      case 15: if constexpr (fam_has(FAM, 15)) mr_pass<15, NT>(src, dst, tw, ps, n / 15, tid, sc, smx, dN); break;
      case 14: if constexpr (fam_has(FAM, 14)) mr_pass<14, NT>(src, dst, tw, ps, n / 14, tid, sc, smx, dN); break;
      case 12: if constexpr (fam_has(FAM, 12)) mr_pass<12, NT>(src, dst, tw, ps, n / 12, tid, sc, smx, dN); break;
      case 10: if constexpr (fam_has(FAM, 10)) mr_pass<10, NT>(src, dst, tw, ps, n / 10, tid, sc, smx, dN); break;
      case 9: if constexpr (fam_has(FAM, 9)) mr_pass<9, NT>(src, dst, tw, ps, n / 9, tid, sc, smx, dN); break;
      case 8: mr_pass<8, NT>(src, dst, tw, ps, n / 8, tid, sc, smx, dN); break;
      case 7: mr_pass<7, NT>(src, dst, tw, ps, n / 7, tid, sc, smx, dN); break;
      case 5: mr_pass<5, NT>(src, dst, tw, ps, n / 5, tid, sc, smx, dN); break;
      case 4: mr_pass<4, NT>(src, dst, tw, ps, n / 4, tid, sc, smx, dN); break;
      case 3: mr_pass<3, NT>(src, dst, tw, ps, n / 3, tid, sc, smx, dN); break;
      default: mr_pass<2, NT>(src, dst, tw, ps, n / 2, tid, sc, smx, dN); break;
    }
    __syncthreads();
    float2* t = src;
    src = dst;
    dst = t;
  }
}

// exp(-2 pi i m / P), 0 <= m < P: the nearest quarter turn q = round(4m / P)
// is taken exactly in integers, and the remainder angle
// 2 pi m / P - q pi / 2 = pi (4m - qP) / (2P), at most pi / 4, goes to sinpif
// and cospif, so the only rounding before them is that of (4m - qP) / 2P
// (|x| <= 1/4).
__device__ __forceinline__ float2 mr_root(int m, int P) {
  const int q = (8 * m + P) / (2 * P);  // round(4m / P), half up
  const float x = (float)(4 * m - q * P) / (float)(2 * P);
  const float s = sinpif(x), c = cospif(x);
  // exp(-i (q pi / 2 + pi x)) = (-i)^q (c - i s)
  switch (q & 3) {
    case 0: return make_float2(c, -s);
    case 1: return make_float2(-s, -c);
    case 2: return make_float2(-c, s);
    default: return make_float2(s, c);
  }
}

// index of the kernel value at transform point g of one axis (-1: none lands)
__device__ __forceinline__ int mr_kidx(int g, int kind, int L, int P) {
  switch (kind) {
    case MR_EXACT: return g;
    case MR_LINEAR: return g < L ? g : -1;
    case MR_CENTERED: return centered_index(g, L, P);
    default: return periodic_index(g, L, P);
  }
}

// The spectra A, B of the two real signals of z = a + i b at bin f, from Z(f)
// and Z(-f): A = (Z(f) + conj Z(-f)) / 2, B = (Z(f) - conj Z(-f)) / 2i.
__device__ __forceinline__ void mr_split(float2 z, float2 zm, float2& A, float2& B) {
  const float2 c = c_conj(zm);
  A = c_scale(c_add(z, c), 0.5f);
  const float2 d = c_sub(z, c);
  B = make_float2(0.5f * d.y, -0.5f * d.x);
}

// Gates of image img (the operator's s row and w_in[c]), without 64-bit division.
template <bool ACT, typename TS>
__device__ __forceinline__ Gates<ACT> mr_gates(const ActIn& ain, uint32_t img, uint32_t C, FastDiv dC) {
  Gates<ACT> g;
  if constexpr (ACT) {
    const uint32_t b = fdiv(img, dC);
    g.s = ain.s + (size_t)b * ain.npos;
    g.w = ld1(reinterpret_cast<const TS*>(ain.w_in) + (img - b * C));
  } else {
    g.s = nullptr;
    g.w = 1.f;
  }
  return g;
}

// One workgroup per group of 2Q images (img0 = 2Q blockIdx.x).
template <typename TS, bool ACT, int NT, int FAM>
__global__ void __launch_bounds__(NT)
    conv_mixed(const TS* __restrict__ x1, const TS* __restrict__ x2, const TS* __restrict__ v,
               const TS* __restrict__ k, const TS* __restrict__ Dp, TS* __restrict__ y, int lines, int C, int kC,
               ActIn ain, MrPlan pl) {
  extern __shared__ float2 mr_lds[];
  const uint32_t tid = threadIdx.x;
  const uint32_t N = (uint32_t)pl.N, Ld = (uint32_t)pl.Ld;
  const uint32_t G2 = 2 * (uint32_t)pl.Q;  // images per group
  const uint32_t i0 = blockIdx.x * G2;
  const uint32_t nimg = imin((int)G2, lines - (int)i0);
  const uint32_t np = (nimg + 1) / 2;  // pairs in this group
  float2* const tw = mr_lds;
  float2* src = mr_lds + pl.ntw;
  float2* dst = src + (size_t)G2 * N;
  float* const Dl = reinterpret_cast<float*>(dst + (size_t)G2 * N);  // D of the group's images
  uint32_t* const smx = reinterpret_cast<uint32_t*>(Dl + G2);           // max |.| of each grid's parts
  const bool exact = pl.N == pl.Ld;  // every axis exact: transform point = data point

  // the pass descriptors, copied with compile-time indices (a run-time index
  // into the plan argument would make the compiler copy all of it to scratch)
  __shared__ MrPass spass[kMrMaxPass];
#pragma unroll
  for (int i = 0; i < kMrMaxPass; ++i)
    if (tid == (uint32_t)i && i < pl.npass) spass[i] = pl.pass[i];

  // twiddles exp(-2 pi i m / P) of each transformed axis
#pragma unroll
  for (int d = 0; d < 3; ++d) {
    if (pl.P[d] < 2) continue;
    for (int m = tid; m < pl.P[d]; m += NT) tw[pl.twoff[d] + m] = mr_root(m, pl.P[d]);
  }
  for (uint32_t i = tid; i < G2; i += NT) {
    const uint32_t img = i0 + i;
    Dl[i] = i < nimg ? ld1(Dp + (img - fdiv(img, pl.dC) * (uint32_t)C)) : 0.f;
  }
  for (uint32_t i = tid; i < 2 * G2; i += NT) smx[i] = 0u;  // (the staging barrier orders it)

  // stage zu = ua + i ub and zk = ka + i kb of every pair on the transform
  // grid: grid i = 2q + r of the group holds pair q's u (r = 0) or k (r = 1)
  for (uint32_t f = tid; f < 2 * np * N; f += NT) {
    const uint32_t i = fdiv(f, pl.dN), p = f - i * N;
    const uint32_t ia = i & ~1u;  // image a of the pair, in the group
    const bool isk = i & 1u, hasb = ia + 1 < nimg;
    float2 z = czero();
    if (exact && kC == 0 && !ACT) {  // the group's x1, v, k: one run from i0 N
      const size_t o = (size_t)(i0 + ia) * N + p;
      if (isk) {
        z.x = ld1(k + o);
        if (hasb) z.y = ld1(k + o + N);
      } else {
        z.x = ld1(x1 + o) * ld1(v + o);
        if (hasb) z.y = ld1(x1 + o + N) * ld1(v + o + N);
      }
    } else {
      // grid point p: the data point n (u; n < 0 outside the image) and the
      // kernel point j (k; j < 0 where no displacement lands)
      int n = (int)p, j = (int)p;
      if (!exact) {
        const uint32_t t = fdiv(p, pl.dP2), g2 = p - t * pl.P[2];
        const uint32_t g0 = fdiv(t, pl.dP1), g1 = t - g0 * pl.P[1];
        n = ((int)g0 < pl.L[0] && (int)g1 < pl.L[1] && (int)g2 < pl.L[2])
                ? (int)((g0 * pl.L[1] + g1) * pl.L[2] + g2) : -1;
        const int j0 = mr_kidx(g0, pl.kind[0], pl.L[0], pl.P[0]);
        const int j1 = mr_kidx(g1, pl.kind[1], pl.L[1], pl.P[1]);
        const int j2 = mr_kidx(g2, pl.kind[2], pl.L[2], pl.P[2]);
        j = (j0 >= 0 && j1 >= 0 && j2 >= 0) ? (j0 * pl.KL[1] + j1) * pl.KL[2] + j2 : -1;
      }
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        if (h == 1 && !hasb) break;
        const uint32_t img = i0 + ia + h;
        float val = 0.f;
        if (isk) {
          if (j >= 0) {
            const uint32_t kl = kC ? img - fdiv(img, pl.dKC) * (uint32_t)kC : img;
            val = ld1(k + (size_t)kl * (uint32_t)pl.Kd + j);
          }
        } else if (n >= 0) {
          const Gates<ACT> G = mr_gates<ACT, TS>(ain, img, (uint32_t)C, pl.dC);
          const size_t o = (size_t)img * Ld + n;
          val = G.u1(ld1(x1 + o), ld1(v + o), n);
        }
        if (h == 0) z.x = val;
        else z.y = val;
      }
    }
    src[f] = z;
  }
  __syncthreads();

  // largest magnitude of each grid's two parts: whole grids per wavefront, or
  // S wavefronts per grid where there are fewer grids than wavefronts; one
  // atomic per wavefront and part (magnitudes as bit patterns, ordered like
  // the values for x >= 0)
  {
    constexpr uint32_t NW = NT / 64;
    const uint32_t w = tid / 64, lane = tid % 64, G = 2 * np;
    const uint32_t S = G >= NW ? 1 : NW / G;
    for (uint32_t gw = w; gw < G * S; gw += NW) {
      const uint32_t g = gw / S, part = gw % S;
      uint32_t mx = 0, my = 0;
      for (uint32_t p = part * 64 + lane; p < N; p += 64 * S) {
        const float2 z = src[g * N + p];
        mx = umax(mx, __float_as_uint(fabsf(z.x)));
        my = umax(my, __float_as_uint(fabsf(z.y)));
      }
#pragma unroll
      for (int o = 32; o >= 1; o /= 2) {
        mx = umax(mx, (uint32_t)__shfl_xor((int)mx, o));
        my = umax(my, (uint32_t)__shfl_xor((int)my, o));
      }
      if (lane == 0) {
        atomicMax(smx + 2 * g, mx);
        atomicMax(smx + 2 * g + 1, my);
      }
    }
  }
  __syncthreads();

  // forward transforms of the 2 np grids
  mr_transform<NT, FAM>(src, dst, tw, spass, pl.npass, 2 * np * N, tid, true, smx, pl.dN);

  // products of each pair, conjugated: conj(Ya + i Yb)
  {
    const float scale = 1.f / (float)pl.N;
    for (uint32_t f = tid; f < np * N; f += NT) {
      const uint32_t q = fdiv(f, pl.dN), p = f - q * N;
      const uint32_t t = fdiv(p, pl.dP2), g2 = p - t * pl.P[2];
      const uint32_t g0 = fdiv(t, pl.dP1), g1 = t - g0 * pl.P[1];
      const uint32_t m0 = g0 ? pl.P[0] - g0 : 0, m1 = g1 ? pl.P[1] - g1 : 0, m2 = g2 ? pl.P[2] - g2 : 0;
      const uint32_t pm = (m0 * pl.P[1] + m1) * pl.P[2] + m2;
      const float2* zu = src + 2 * q * N;
      const float2* zk = zu + N;
      float2 Ua, Ub, Ka, Kb;
      mr_split(zu[p], zu[pm], Ua, Ub);
      mr_split(zk[p], zk[pm], Ka, Kb);
      // grid 2q holds (ua, ub) and grid 2q + 1 (ka, kb), each part scaled
      // by 2^-e; Y = U (K + D) / N comes out scaled by 2^-(eu + ey), ey the
      // larger of ek and D's exponent
      const uint32_t* sm = smx + 4 * q;
      const float Da = Dl[2 * q], Db = Dl[2 * q + 1];
      const int eka = mr_exp(sm[2]), ekb = mr_exp(sm[3]);
      const int eya = imax(eka, mr_fexp(Da)), eyb = imax(ekb, mr_fexp(Db));
      Ua = c_scale(Ua, scale);
      Ub = c_scale(Ub, scale);
      Ka = c_scale(Ka, ldexpf(1.f, eka - eya));
      Kb = c_scale(Kb, ldexpf(1.f, ekb - eyb));
      const float2 ya = c_mul(Ua, make_float2(Ka.x + ldexpf(Da, -eya), Ka.y));
      const float2 yb = c_mul(Ub, make_float2(Kb.x + ldexpf(Db, -eyb), Kb.y));
      dst[f] = make_float2(ya.x - yb.y, -(ya.y + yb.x));
    }
    __syncthreads();
    float2* t = src;
    src = dst;
    dst = t;
  }

  // one transform per pair: the conjugate of both inverses
  mr_transform<NT, FAM>(src, dst, tw, spass, pl.npass, np * N, tid, false, smx, pl.dN);

  // crop, outer gate, store: ya = Re, yb = -Im
  const Gates<ACT> G{};  // the outer gate depends on x2 only
  for (uint32_t f = tid; f < nimg * Ld; f += NT) {
    const uint32_t i = fdiv(f, pl.dLd), n = f - i * Ld;
    uint32_t p = n;
    if (!exact) {
      const uint32_t t = fdiv(n, pl.dL2), n2 = n - t * pl.L[2];
      const uint32_t n0 = fdiv(t, pl.dL1), n1 = t - n0 * pl.L[1];
      p = (n0 * pl.P[1] + n1) * pl.P[2] + n2;
    }
    const float2 r = src[(i >> 1) * N + p];
    const uint32_t* sm = smx + 4 * (i >> 1) + (i & 1);  // u's and k's magnitudes of image i
    const int e = mr_exp(sm[0]) + imax(mr_exp(sm[2]), mr_fexp(Dl[i]));
    const size_t o = (size_t)i0 * Ld + f;
    st1(y + o, G.g1(ld1(x2 + o)) * ldexpf((i & 1) ? -r.y : r.x, e));
  }
}

// ---------------------------------------------------------------------------
// Backward (hyenand_fftconv_backward) on the same transform grid.  With
// u = x1 v and h = gy x2, zero outside the image, and k at its
// displacements, the convolution is circular on the grid, so per bin
//   Z = U (K + D)           z = k conv u + D u       -> gx2 = gy z
//   Gu = H (conj K + D)     gu, the adjoint applied  -> gx1 = gu v, gv = gu x1
//   Gk = H conj U           gk at the displacements of k's points (both
//                           displacements of a periodic axis' point summed)
// and gD[c] = sum over the samples and points of h u (one fp32 sum per line,
// added over the samples in order afterwards).  A pair of images has three
// staged grids, u, k and h (grid 3q + 0, 1, 2: a's part real, b's
// imaginary), and three products, each scaled as in the forward (Z by
// 2^-(eu + ey), Gu by 2^-(eh + ey), Gk by 2^-(eh + eu)).
// ---------------------------------------------------------------------------

// grid coordinate(s) on one axis of kernel index j: one, or two for a
// periodic axis (displacements j and j - L); returns how many
__device__ __forceinline__ int mr_kpos(int j, int kind, int L, int P, int (&g)[2]) {
  switch (kind) {
    case MR_EXACT:
    case MR_LINEAR: g[0] = j; return 1;
    case MR_CENTERED: {
      const int d = j - (L - 1);
      g[0] = d >= 0 ? d : d + P;
      return 1;
    }
    default:
      g[0] = j;
      g[1] = P - L + j;
      return j >= 1 ? 2 : 1;
  }
}

template <typename TS, int NT, int FAM>
__global__ void __launch_bounds__(NT)
    conv_mixed_bwd(const TS* __restrict__ x1, const TS* __restrict__ x2, const TS* __restrict__ v,
                   const TS* __restrict__ k, const TS* __restrict__ Dp, const TS* __restrict__ gy,
                   TS* __restrict__ gx1, TS* __restrict__ gx2, TS* __restrict__ gv, TS* __restrict__ gk,
                   float* __restrict__ partial, int lines, int C, MrPlan pl) {
  extern __shared__ float2 mr_lds[];
  constexpr uint32_t NW = NT / 64;
  const uint32_t tid = threadIdx.x;
  const uint32_t N = (uint32_t)pl.N, Ld = (uint32_t)pl.Ld, Kd = (uint32_t)pl.Kd;
  const uint32_t G2 = 2 * (uint32_t)pl.Q;  // images per group
  const uint32_t i0 = blockIdx.x * G2;
  const uint32_t nimg = imin((int)G2, lines - (int)i0);
  const uint32_t np = (nimg + 1) / 2;
  float2* const tw = mr_lds;
  float2* src = mr_lds + pl.ntw;
  float2* dst = src + (size_t)3 * pl.Q * N;
  float* const Dl = reinterpret_cast<float*>(dst + (size_t)3 * pl.Q * N);
  uint32_t* const smx = reinterpret_cast<uint32_t*>(Dl + G2);         // 6 per pair
  float2* const wsum = reinterpret_cast<float2*>(smx + 6 * pl.Q);    // 16 per pair
  const bool exact = pl.N == pl.Ld;

  __shared__ MrPass spass[kMrMaxPass];
#pragma unroll
  for (int i = 0; i < kMrMaxPass; ++i)
    if (tid == (uint32_t)i && i < pl.npass) spass[i] = pl.pass[i];
#pragma unroll
  for (int d = 0; d < 3; ++d) {
    if (pl.P[d] < 2) continue;
    for (int m = tid; m < pl.P[d]; m += NT) tw[pl.twoff[d] + m] = mr_root(m, pl.P[d]);
  }
  for (uint32_t i = tid; i < G2; i += NT) {
    const uint32_t img = i0 + i;
    Dl[i] = i < nimg ? ld1(Dp + (img - fdiv(img, pl.dC) * (uint32_t)C)) : 0.f;
  }
  for (uint32_t i = tid; i < 6 * (uint32_t)pl.Q; i += NT) smx[i] = 0u;  // (the staging barrier orders it)

  // stage the pairs' u, k and h grids
  for (uint32_t f = tid; f < 3 * np * N; f += NT) {
    const uint32_t gi = fdiv(f, pl.dN), p = f - gi * N;
    const uint32_t q = gi / 3, role = gi - 3 * q;  // 0 u, 1 k, 2 h
    const uint32_t ia = 2 * q;
    const bool hasb = ia + 1 < nimg;
    int n = (int)p, j = (int)p;
    if (!exact) {
      const uint32_t t = fdiv(p, pl.dP2), g2 = p - t * pl.P[2];
      const uint32_t g0 = fdiv(t, pl.dP1), g1 = t - g0 * pl.P[1];
      n = ((int)g0 < pl.L[0] && (int)g1 < pl.L[1] && (int)g2 < pl.L[2]) ? (int)((g0 * pl.L[1] + g1) * pl.L[2] + g2)
                                                                          : -1;
      const int j0 = mr_kidx(g0, pl.kind[0], pl.L[0], pl.P[0]);
      const int j1 = mr_kidx(g1, pl.kind[1], pl.L[1], pl.P[1]);
      const int j2 = mr_kidx(g2, pl.kind[2], pl.L[2], pl.P[2]);
      j = (j0 >= 0 && j1 >= 0 && j2 >= 0) ? (j0 * pl.KL[1] + j1) * pl.KL[2] + j2 : -1;
    }
    float2 z = czero();
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      if (h == 1 && !hasb) break;
      const size_t img = i0 + ia + h;
      float val = 0.f;
      if (role == 1) {
        if (j >= 0) val = ld1(k + img * Kd + j);
      } else if (n >= 0) {
        const size_t o = img * Ld + n;
        val = role == 0 ? ld1(x1 + o) * ld1(v + o) : ld1(gy + o) * ld1(x2 + o);
      }
      if (h == 0) z.x = val;
      else z.y = val;
    }
    src[f] = z;
  }
  __syncthreads();

  // per pair: the largest magnitude of each grid part (scales) and the sums
  // of h u of its two lines (gD), whole pairs per wavefront or S wavefronts
  // per pair; the sums are combined in a fixed order
  const uint32_t S = np >= NW ? 1 : NW / np;
  {
    const uint32_t w = tid / 64, lane = tid % 64;
    for (uint32_t gw = w; gw < np * S; gw += NW) {
      const uint32_t q = gw / S, part = gw % S;
      uint32_t mx[6] = {0, 0, 0, 0, 0, 0};
      float sa = 0.f, sb = 0.f;
      for (uint32_t p = part * 64 + lane; p < N; p += 64 * S) {
        const float2 zu = src[(3 * q) * N + p], zk = src[(3 * q + 1) * N + p], zh = src[(3 * q + 2) * N + p];
        mx[0] = umax(mx[0], __float_as_uint(fabsf(zu.x)));
        mx[1] = umax(mx[1], __float_as_uint(fabsf(zu.y)));
        mx[2] = umax(mx[2], __float_as_uint(fabsf(zk.x)));
        mx[3] = umax(mx[3], __float_as_uint(fabsf(zk.y)));
        mx[4] = umax(mx[4], __float_as_uint(fabsf(zh.x)));
        mx[5] = umax(mx[5], __float_as_uint(fabsf(zh.y)));
        sa = fmaf(zh.x, zu.x, sa);
        sb = fmaf(zh.y, zu.y, sb);
      }
#pragma unroll
      for (int o = 32; o >= 1; o /= 2) {
#pragma unroll
        for (int e = 0; e < 6; ++e) mx[e] = umax(mx[e], (uint32_t)__shfl_xor((int)mx[e], o));
        sa += __shfl_xor(sa, o);
        sb += __shfl_xor(sb, o);
      }
      if (lane == 0) {
#pragma unroll
        for (int e = 0; e < 6; ++e) atomicMax(smx + 6 * q + e, mx[e]);
        wsum[16 * q + part] = make_float2(sa, sb);
      }
    }
  }
  __syncthreads();
  for (uint32_t i = tid; i < nimg; i += NT) {
    float acc = 0.f;
    for (uint32_t part = 0; part < S; ++part) {
      const float2 w2 = wsum[16 * (i >> 1) + part];
      acc += (i & 1) ? w2.y : w2.x;
    }
    partial[i0 + i] = acc;
  }

  // forward transforms of the 3 np grids (the first pass applies the scales)
  mr_transform<NT, FAM>(src, dst, tw, spass, pl.npass, 3 * np * N, tid, true, smx, pl.dN);

  // the three products of each pair, conjugated
  {
    const float scale = 1.f / (float)pl.N;
    for (uint32_t f = tid; f < np * N; f += NT) {
      const uint32_t q = fdiv(f, pl.dN), p = f - q * N;
      const uint32_t t = fdiv(p, pl.dP2), g2 = p - t * pl.P[2];
      const uint32_t g0 = fdiv(t, pl.dP1), g1 = t - g0 * pl.P[1];
      const uint32_t m0 = g0 ? pl.P[0] - g0 : 0, m1 = g1 ? pl.P[1] - g1 : 0, m2 = g2 ? pl.P[2] - g2 : 0;
      const uint32_t pm = (m0 * pl.P[1] + m1) * pl.P[2] + m2;
      const float2* zu = src + 3 * q * N;
      const float2* zk = zu + N;
      const float2* zh = zk + N;
      float2 U[2], K[2], H[2];
      mr_split(zu[p], zu[pm], U[0], U[1]);
      mr_split(zk[p], zk[pm], K[0], K[1]);
      mr_split(zh[p], zh[pm], H[0], H[1]);
      const uint32_t* sm = smx + 6 * q;
      float2 Z[2], Gu[2], Gk[2];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const float D = Dl[2 * q + h];
        const int ek = mr_exp(sm[2 + h]), ey = imax(ek, mr_fexp(D));
        const float2 Kn = c_scale(K[h], ldexpf(1.f, ek - ey));  // K 2^-ey
        const float Dn = ldexpf(D, -ey);
        const float2 Us = c_scale(U[h], scale), Hs = c_scale(H[h], scale);
        Z[h] = c_mul(Us, make_float2(Kn.x + Dn, Kn.y));
        Gu[h] = c_mul(Hs, make_float2(Kn.x + Dn, -Kn.y));
        Gk[h] = c_mul(Hs, c_conj(U[h]));
      }
      float2* out = dst + 3 * q * N;
      out[p] = make_float2(Z[0].x - Z[1].y, -(Z[0].y + Z[1].x));
      out[N + p] = make_float2(Gu[0].x - Gu[1].y, -(Gu[0].y + Gu[1].x));
      out[2 * N + p] = make_float2(Gk[0].x - Gk[1].y, -(Gk[0].y + Gk[1].x));
    }
    __syncthreads();
    float2* t = src;
    src = dst;
    dst = t;
  }

  // inverse transforms of the 3 np grids
  mr_transform<NT, FAM>(src, dst, tw, spass, pl.npass, 3 * np * N, tid, false, smx, pl.dN);

  // data points: gx2 = gy z, gx1 = gu v, gv = gu x1
  for (uint32_t f = tid; f < nimg * Ld; f += NT) {
    const uint32_t i = fdiv(f, pl.dLd), n = f - i * Ld;
    uint32_t p = n;
    if (!exact) {
      const uint32_t t = fdiv(n, pl.dL2), n2 = n - t * pl.L[2];
      const uint32_t n0 = fdiv(t, pl.dL1), n1 = t - n0 * pl.L[1];
      p = (n0 * pl.P[1] + n1) * pl.P[2] + n2;
    }
    const uint32_t q = i >> 1, h = i & 1;
    const uint32_t* sm = smx + 6 * q + h;  // u, k, h parts of image i: sm[0], sm[2], sm[4]
    const int ey = imax(mr_exp(sm[2]), mr_fexp(Dl[i]));
    const float2 rz = src[3 * q * N + p], ru = src[(3 * q + 1) * N + p];
    const float z = ldexpf(h ? -rz.y : rz.x, mr_exp(sm[0]) + ey);
    const float gu = ldexpf(h ? -ru.y : ru.x, mr_exp(sm[4]) + ey);
    const size_t o = (size_t)i0 * Ld + f;
    st1(gx2 + o, ld1(gy + o) * z);
    st1(gx1 + o, gu * ld1(v + o));
    st1(gv + o, gu * ld1(x1 + o));
  }
  // kernel points: gk at the displacement(s) of each
  for (uint32_t f = tid; f < nimg * Kd; f += NT) {
    const uint32_t i = fdiv(f, pl.dKd), j = f - i * Kd;
    const uint32_t q = i >> 1, h = i & 1;
    const float2* rg = src + (3 * q + 2) * N;
    float acc = 0.f;
    if (exact) {
      const float2 r = rg[j];
      acc = h ? -r.y : r.x;
    } else {
      const uint32_t t = fdiv(j, pl.dKL2), j2 = j - t * pl.KL[2];
      const uint32_t j0 = fdiv(t, pl.dKL1), j1 = t - j0 * pl.KL[1];
      int a0[2], a1[2], a2[2];
      const int c0 = mr_kpos(j0, pl.kind[0], pl.L[0], pl.P[0], a0);
      const int c1 = mr_kpos(j1, pl.kind[1], pl.L[1], pl.P[1], a1);
      const int c2 = mr_kpos(j2, pl.kind[2], pl.L[2], pl.P[2], a2);
      for (int e0 = 0; e0 < c0; ++e0)
        for (int e1 = 0; e1 < c1; ++e1)
          for (int e2 = 0; e2 < c2; ++e2) {
            const float2 r = rg[(a0[e0] * pl.P[1] + a1[e1]) * pl.P[2] + a2[e2]];
            acc += h ? -r.y : r.x;
          }
    }
    const uint32_t* sm = smx + 6 * q + h;
    st1(gk + (size_t)i0 * Kd + f, ldexpf(acc, mr_exp(sm[4]) + mr_exp(sm[0])));
  }
}

bool smooth7(int64_t n) {
  if (n < 1) return false;
  for (int r : {2, 3, 5, 7})
    while (n % r == 0) n /= r;
  return n == 1;
}

int64_t smooth7_ceil(int64_t n) {
  while (!smooth7(n)) ++n;
  return n;
}

// twiddles, the two buffers of 2Q images' grids, D of the 2Q images, the
// magnitudes of the 2Q grids' two parts
size_t mr_lds_bytes(const MrPlan& pl, int Q) {
  return ((size_t)pl.ntw + (size_t)4 * Q * pl.N) * sizeof(float2) + (size_t)2 * Q * sizeof(float) +
         (size_t)4 * Q * sizeof(uint32_t);
}

// the backward's: twiddles, two buffers of 3 grids per pair, D, 6 scales and
// 16 partial sums per pair
size_t mr_lds_bytes_bwd(const MrPlan& pl, int Q) {
  return ((size_t)pl.ntw + (size_t)6 * Q * pl.N) * sizeof(float2) + (size_t)2 * Q * sizeof(float) +
         (size_t)6 * Q * sizeof(uint32_t) + (size_t)16 * Q * sizeof(float2);
}

int env_int(const char* name) {
  const char* e = getenv(name);
  return e ? (int)strtol(e, nullptr, 10) : 0;
}

// Passes of every axis with the radices of family f, the twiddle table layout.
bool mr_passes(MrPlan* pl, int f) {
  if (f < 0 || f >= kNumFam) return false;
  int np = 0, tw = 0;
  for (int d = 0; d < 3; ++d) {
    const int P = pl->P[d];
    if (P < 2) continue;
    int S = 1;
    for (int e = d + 1; e < 3; ++e) S *= pl->P[e];
    pl->twoff[d] = tw;
    tw += P;
    int rest = P, ns = 1;
    while (rest > 1) {
      int r = 0;
      for (int c : {16, 15, 14, 12, 10, 9, 8, 7, 5, 4, 3, 2})
        if (fam_has(f, c) && rest % c == 0) {
          r = c;
          break;
        }
      if (r == 0 || np == kMrMaxPass) return false;
      MrPass& ps = pl->pass[np++];
      ps.r = r;
      ps.q = P / r;
      ps.ns = ns;
      ps.sa = S;
      ps.pasa = P * S;
      ps.twoff = pl->twoff[d];
      ps.twstep = P / (ns * r);
      ps.dsa = make_fastdiv((uint32_t)S);
      ps.dq = make_fastdiv((uint32_t)ps.q);
      ps.dns = make_fastdiv((uint32_t)ns);
      ns *= r;
      rest /= r;
    }
  }
  pl->npass = np;
  pl->ntw = tw;
  pl->fam = f;
  return true;
}

// The plan of a call, or false where these kernels do not take it.
bool mixed_plan(const FftConvArgs& a, MrPlan* pl) {
  if (!a.rl || a.circular || a.ndim < 1 || a.ndim > 3) return false;
  memset(pl, 0, sizeof *pl);
  const int lead = 3 - a.ndim;
  int64_t N = 1, Ld = 1, Kd = 1;
  for (int d = 0; d < 3; ++d) {
    if (d < lead) {
      pl->P[d] = pl->L[d] = pl->KL[d] = 1;
      pl->kind[d] = MR_EXACT;
      continue;
    }
    const int64_t L = a.L[d - lead];
    int64_t P;
    int kind;
    if (a.periodic && smooth7(L)) {
      P = L;
      kind = MR_EXACT;
    } else {
      P = smooth7_ceil(2 * L - 1);
      kind = a.centered ? MR_CENTERED : (a.periodic ? MR_PERIODIC : MR_LINEAR);
    }
    if (P > kMrMaxN) return false;
    pl->P[d] = (int)P;
    pl->L[d] = (int)L;
    pl->KL[d] = (int)(kind == MR_CENTERED ? 2 * L - 1 : L);
    pl->kind[d] = kind;
    N *= P;
    Ld *= L;
    Kd *= pl->KL[d];
    if (N > kMrMaxN) return false;
  }
  pl->N = (int)N;
  pl->Ld = (int)Ld;
  pl->Kd = (int)Kd;
  // passes: each axis, the largest radix of the family that divides what is
  // left; the family with the fewest passes (ties: the lower family)
  int best = -1;
  for (int f = 0; f < kNumFam; ++f) {
    MrPlan t = *pl;
    if (!mr_passes(&t, f)) continue;
    if (best < 0 || t.npass < pl->npass) {
      *pl = t;
      best = f;
    }
  }
  if (best < 0) return false;
  if (const char* e = getenv("HYENAND_MIXED_FAMILY")) {  // force a family (sweeps)
    MrPlan t = *pl;
    if (mr_passes(&t, (int)strtol(e, nullptr, 10))) *pl = t;
  }
  // Lanes and image pairs per workgroup, from sweeps of 256 .. 1024 lanes and
  // 1 .. 8 pairs on 12- to 1000-point lines, 14^2 to 48 x 64 grids and 12^3
  // (MI355X): about 3 points of the images' grids per lane below 256
  // transform points and 6 from there, at least 512 workgroups where the
  // lines allow, 256 lanes for groups of at most 768 points, one pair from
  // 1536 points on 1024 lanes (512 for lines below 2560 points: 87 us against
  // 120 for 64 x 64 lines of 2000).
  int nt = 512, Q = 1;
  if (pl->N < 1536) {
    const int target = pl->N >= 256 ? 3072 : 1536;  // grid points per workgroup
    Q = imax(1, (target + pl->N) / (2 * pl->N));
    Q = imax(1, imin(Q, (int)(a.lines / 1024)));
    if (2 * Q * pl->N <= 768) nt = 256;
  } else {
    nt = (a.ndim == 1 && pl->N < 2560) ? 512 : 1024;
  }
  if (const int o = env_int("HYENAND_MIXED_PAIRS"); o > 0) Q = o;
  if (const int o = env_int("HYENAND_MIXED_LANES"); o == 256 || o == 512 || o == 1024) nt = o;
  const int64_t pairs = (a.lines + 1) / 2;
  if (Q > pairs) Q = (int)pairs;
  while (Q > 1 && mr_lds_bytes(*pl, Q) > kMrMaxLds) --Q;
  if (mr_lds_bytes(*pl, Q) > kMrMaxLds) return false;
  pl->Q = Q;
  pl->nt = nt;
  pl->dN = make_fastdiv((uint32_t)pl->N);
  pl->dP1 = make_fastdiv((uint32_t)pl->P[1]);
  pl->dP2 = make_fastdiv((uint32_t)pl->P[2]);
  pl->dL1 = make_fastdiv((uint32_t)pl->L[1]);
  pl->dL2 = make_fastdiv((uint32_t)pl->L[2]);
  pl->dLd = make_fastdiv((uint32_t)pl->Ld);
  pl->dC = make_fastdiv((uint32_t)a.C);
  pl->dKC = make_fastdiv((uint32_t)(a.kC ? a.kC : 1));
  pl->dKL1 = make_fastdiv((uint32_t)pl->KL[1]);
  pl->dKL2 = make_fastdiv((uint32_t)pl->KL[2]);
  pl->dKd = make_fastdiv((uint32_t)pl->Kd);
  return true;
}

template <typename TS, bool ACT, int NT, int FAM>
hipError_t launch_mixed_t(const FftConvArgs& a, const MrPlan& pl, hipStream_t s) {
  const size_t lds = mr_lds_bytes(pl, pl.Q);
  const unsigned nblk = (unsigned)((a.lines + 2 * pl.Q - 1) / (2 * pl.Q));
  // the kernel may take more than the default 64 KB of dynamic LDS
  static std::once_flag once;
  static hipError_t attr = hipSuccess;
  std::call_once(once, [] {
    attr = hipFuncSetAttribute(reinterpret_cast<const void*>(conv_mixed<TS, ACT, NT, FAM>),
                               hipFuncAttributeMaxDynamicSharedMemorySize, (int)kMrMaxLds);
  });
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL((conv_mixed<TS, ACT, NT, FAM>), dim3(nblk), dim3(NT), lds, s, (const TS*)a.x1, (const TS*)a.x2,
                     (const TS*)a.v, (const TS*)a.k, (const TS*)a.D, (TS*)a.y, (int)a.lines, (int)a.C, a.kC,
                     a.act_in, pl);
  return hipGetLastError();
}

template <int NT, int FAM>
hipError_t launch_mixed_f(const FftConvArgs& a, const MrPlan& pl, hipStream_t s) {
  if (a.bf16)
    return a.act ? launch_mixed_t<uint16_t, true, NT, FAM>(a, pl, s)
                 : launch_mixed_t<uint16_t, false, NT, FAM>(a, pl, s);
  return a.act ? launch_mixed_t<float, true, NT, FAM>(a, pl, s) : launch_mixed_t<float, false, NT, FAM>(a, pl, s);
}

template <int NT>
hipError_t launch_mixed_nt(const FftConvArgs& a, const MrPlan& pl, hipStream_t s) {
  switch (pl.fam) {
    case 1: return launch_mixed_f<NT, 1>(a, pl, s);
    case 2: return launch_mixed_f<NT, 2>(a, pl, s);
    case 3: return launch_mixed_f<NT, 3>(a, pl, s);
    default: return launch_mixed_f<NT, 0>(a, pl, s);
  }
}

// The backward's plan: the forward's grid and passes, its own workgroup
// shape, from a sweep of 256 .. 1024 lanes and 1 .. 4 pairs (three grids per
// pair): about 2304 grid points per workgroup below 512 transform points, at
// least 512 workgroups where the lines allow, 256 lanes for groups of at most
// 1152 points; one pair from 512 points (64 x 64 lines of 1000: 101 us
// against 127 with two), on 256 lanes for 2D and 3D grids below 1024 points
// (16 x 384 centred 14 x 14: 88 us against 93 on 512); from 1536 points on
// 1024 lanes, 512 for lines below 2560.
bool mixed_bwd_plan(const FftConvArgs& a, MrPlan* pl) {
  if (a.act || a.kC || !mixed_plan(a, pl)) return false;
  int nt = 512, Q = 1;
  if (pl->N < 512) {
    Q = imax(1, (2 * 2304 + 3 * pl->N) / (6 * pl->N));
    Q = imax(1, imin(Q, (int)(a.lines / 1024)));
    if (6 * Q * pl->N <= 1152) nt = 256;
  } else if (pl->N < 1536) {
    nt = (a.ndim >= 2 && pl->N < 1024) ? 256 : 512;
  } else {
    nt = (a.ndim == 1 && pl->N < 2560) ? 512 : 1024;
  }
  if (const int o = env_int("HYENAND_MIXED_PAIRS"); o > 0) Q = o;
  if (const int o = env_int("HYENAND_MIXED_LANES"); o == 256 || o == 512 || o == 1024) nt = o;
  const int64_t pairs = (a.lines + 1) / 2;
  if (Q > pairs) Q = (int)pairs;
  while (Q > 1 && mr_lds_bytes_bwd(*pl, Q) > kMrMaxLds) --Q;
  if (mr_lds_bytes_bwd(*pl, Q) > kMrMaxLds) return false;
  pl->Q = Q;
  pl->nt = nt;
  return true;
}

template <typename TS, int NT, int FAM>
hipError_t launch_mixed_bwd_t(const FftConvBwdArgs& b, const MrPlan& pl, hipStream_t s) {
  const FftConvArgs& a = b.f;
  const size_t lds = mr_lds_bytes_bwd(pl, pl.Q);
  const unsigned nblk = (unsigned)((a.lines + 2 * pl.Q - 1) / (2 * pl.Q));
  static std::once_flag once;
  static hipError_t attr = hipSuccess;
  std::call_once(once, [] {
    attr = hipFuncSetAttribute(reinterpret_cast<const void*>(conv_mixed_bwd<TS, NT, FAM>),
                               hipFuncAttributeMaxDynamicSharedMemorySize, (int)kMrMaxLds);
  });
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL((conv_mixed_bwd<TS, NT, FAM>), dim3(nblk), dim3(NT), lds, s, (const TS*)a.x1, (const TS*)a.x2,
                     (const TS*)a.v, (const TS*)a.k, (const TS*)a.D, (const TS*)b.gy, (TS*)b.gx1, (TS*)b.gx2,
                     (TS*)b.gv, (TS*)b.gk, b.partial, (int)a.lines, (int)a.C, pl);
  return hipGetLastError();
}

template <int NT, int FAM>
hipError_t launch_mixed_bwd_f(const FftConvBwdArgs& b, const MrPlan& pl, hipStream_t s) {
  return b.f.bf16 ? launch_mixed_bwd_t<uint16_t, NT, FAM>(b, pl, s) : launch_mixed_bwd_t<float, NT, FAM>(b, pl, s);
}

template <int NT>
hipError_t launch_mixed_bwd_nt(const FftConvBwdArgs& b, const MrPlan& pl, hipStream_t s) {
  switch (pl.fam) {
    case 1: return launch_mixed_bwd_f<NT, 1>(b, pl, s);
    case 2: return launch_mixed_bwd_f<NT, 2>(b, pl, s);
    case 3: return launch_mixed_bwd_f<NT, 3>(b, pl, s);
    default: return launch_mixed_bwd_f<NT, 0>(b, pl, s);
  }
}

}  // namespace

bool mixed_supported(const FftConvArgs& a) {
  MrPlan pl;
  return mixed_plan(a, &pl);
}

// Where these kernels beat the power-of-two ones (measured on the MI355X):
// 3D grids (which those do not take; 4 x 64 x 12^3: 13.9 us against 207 us
// embedded), 2D grids up to 2048 transform points (16 x 384 images of 14 x 14:
// 15.1 us against 105 us; 27 x 27 centred: 44 us against 111 us) and larger
// ones with at most a quarter of the power-of-two points (48 x 64: 20.2 us
// against 59 us; 48 x 80 at half: 97 us against 62 us), lines of at most 128
// points (64 x 256 lines of 12: 9.9 us against 20.2 us) or with at most 5/12
// of the power-of-two points (64 x 64 lines of 300 and 3000: 15.4 and 152 us
// against 17.0 and 157 us; of 500, 1000 and 2000 at about half: 22.5, 41.5
// and 99 us against 20.6, 40.0 and 78 us).
bool mixed_preferred(const FftConvArgs& a) {
  MrPlan pl;
  if (!mixed_plan(a, &pl)) return false;
  int64_t pow2_points = 1;
  for (int d = 0; d < a.ndim; ++d) pow2_points *= a.P[d];
  if (a.ndim == 3) return true;
  if (a.ndim == 2) return pl.N <= 2048 || 4 * (int64_t)pl.N <= pow2_points;
  return pl.N <= 128 || 12 * (int64_t)pl.N <= 5 * pow2_points;
}

hipError_t launch_mixed(const FftConvArgs& a, hipStream_t s) {
  MrPlan pl;
  if (!mixed_plan(a, &pl)) return hipErrorInvalidValue;
  switch (pl.nt) {
    case 512: return launch_mixed_nt<512>(a, pl, s);
    case 1024: return launch_mixed_nt<1024>(a, pl, s);
    default: return launch_mixed_nt<256>(a, pl, s);
  }
}

bool mixed_backward_supported(const FftConvArgs& a) {
  MrPlan pl;
  return mixed_bwd_plan(a, &pl);
}

hipError_t launch_mixed_backward(const FftConvBwdArgs& b, hipStream_t s) {
  MrPlan pl;
  if (!mixed_bwd_plan(b.f, &pl)) return hipErrorInvalidValue;
  switch (pl.nt) {
    case 512: return launch_mixed_bwd_nt<512>(b, pl, s);
    case 1024: return launch_mixed_bwd_nt<1024>(b, pl, s);
    default: return launch_mixed_bwd_nt<256>(b, pl, s);
  }
}

}  // namespace hyenand
