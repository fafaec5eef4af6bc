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
// Arithmetic: two real signals per complex transform.  An image's u and k go
// into one complex grid z = u + i k; after the forward transform the mirror
// bin separates them, U(f) = (Z(f) + conj Z(-f)) / 2 and
// K(f) = (Z(f) - conj Z(-f)) / 2i.  The products of two images, Ya and Yb
// (with the shortcut folded in as U (K + D)), go into one grid Ya + i Yb, and
// one more transform of its conjugate gives conj(ya + i yb): the inverse of
// both.  Odd extents need no half-length packing this way, and each image
// costs one and a half complex transforms of the grid.
//
// Each axis runs Stockham passes of radix 8, 4, 2, 7, 5 or 3 between two LDS
// buffers (one barrier per pass).  A pass of radix r over an axis of P points
// with stride S, after passes whose radices multiply to Ns: butterfly j of a
// line reads the r points j + t P/r, multiplies point t by the twiddle
// exp(-2 pi i t (j mod Ns) / (Ns r)), takes the r-point DFT and writes output
// t to (j div Ns) Ns r + (j mod Ns) + t Ns; after the last pass the axis is in
// natural order.  Every pass sees the images of the workgroup as one list of
// butterflies, so the lanes stay busy whatever the grid.
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
  int npass;      // forward passes; the inverse runs the same list
  FastDiv dN, dP1, dP2, dL1, dL2, dLd;
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

template <int R>
__device__ __forceinline__ void dft_any(float2 (&x)[R]) {
  if constexpr (R == 3 || R == 5 || R == 7) dft_odd<R>(x);
  else dft<R, false>(x);
}

// One Stockham pass of radix R over `items` butterflies (all images); TW:
// the pass has twiddles (not the first pass of its axis, where all are 1).
template <int R, int NT, bool TW>
__device__ __forceinline__ void mr_pass_t(const float2* src, float2* dst, const float2* tw, const MrPass& ps,
                                          uint32_t items, uint32_t tid) {
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
    if constexpr (TW) {
      const uint32_t tws = kk * (uint32_t)ps.twstep;
      const float2* tp = tw + ps.twoff;
#pragma unroll
      for (int t = 1; t < R; ++t) x[t] = c_mul(x[t], tp[t * tws]);
    }
    dft_any<R>(x);
    float2* dp = dst + base + (jn * (uint32_t)(ps.ns * R) + kk) * (uint32_t)ps.sa;
#pragma unroll
    for (int t = 0; t < R; ++t) dp[t * nss] = x[t];
  }
}

template <int R, int NT>
__device__ __forceinline__ void mr_pass(const float2* src, float2* dst, const float2* tw, const MrPass& ps,
                                        uint32_t items, uint32_t tid) {
  if (ps.ns == 1) mr_pass_t<R, NT, false>(src, dst, tw, ps, items, tid);
  else mr_pass_t<R, NT, true>(src, dst, tw, ps, items, tid);
}

// every pass of the plan over n points (whole images), ping-ponging src/dst;
// returns with the result in src
template <int NT>
__device__ __forceinline__ void mr_transform(float2*& src, float2*& dst, const float2* tw, const MrPlan& pl,
                                             uint32_t n, uint32_t tid) {
  for (int i = 0; i < pl.npass; ++i) {
    const MrPass& ps = pl.pass[i];
    switch (ps.r) {
      case 8: mr_pass<8, NT>(src, dst, tw, ps, n / 8, tid); break;
      case 4: mr_pass<4, NT>(src, dst, tw, ps, n / 4, tid); break;
      case 2: mr_pass<2, NT>(src, dst, tw, ps, n / 2, tid); break;
      case 7: mr_pass<7, NT>(src, dst, tw, ps, n / 7, tid); break;
      case 5: mr_pass<5, NT>(src, dst, tw, ps, n / 5, tid); break;
      default: mr_pass<3, NT>(src, dst, tw, ps, n / 3, tid); break;
    }
    __syncthreads();
    float2* t = src;
    src = dst;
    dst = t;
  }
}

// exp(-2 pi i m / P), 0 <= m < P: the nearest quarter turn q = round(4m / P)
// is taken exactly in integers, and the remainder angle
// 2 pi m / P - q pi / 2 = pi (4m - qP) / (2P), at most pi / 4, goes to sincospif,
// so the only rounding before it is that of (4m - qP) / 2P (|x| <= 1/4).
__device__ __forceinline__ float2 mr_root(int m, int P) {
  const int q = (8 * m + P) / (2 * P);  // round(4m / P), half up
  const float x = (float)(4 * m - q * P) / (float)(2 * P);
  float s, c;
  sincospif(x, &s, &c);
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

// U (K + D) / N of one image from its transform Z at bin f and the mirror bin
__device__ __forceinline__ float2 mr_product(float2 z, float2 zm, float D, float scale) {
  const float2 a = z, b = c_conj(zm);
  const float2 u = c_scale(c_add(a, b), 0.5f * scale);
  const float2 d = c_sub(a, b);
  return c_mul(u, make_float2(fmaf(0.5f, d.y, D), -0.5f * d.x));
}

template <typename TS, bool ACT, int NT>
__global__ void __launch_bounds__(NT)
    conv_mixed(const TS* __restrict__ x1, const TS* __restrict__ x2, const TS* __restrict__ v,
               const TS* __restrict__ k, const TS* __restrict__ Dp, TS* __restrict__ y, int64_t lines, int C,
               int kC, ActIn ain, MrPlan pl) {
  extern __shared__ float2 mr_lds[];
  const uint32_t tid = threadIdx.x;
  const uint32_t N = (uint32_t)pl.N;
  const int64_t img0 = (int64_t)blockIdx.x * 2 * pl.Q;
  const int nimg = (int)(lines - img0 < 2 * pl.Q ? lines - img0 : 2 * pl.Q);
  const uint32_t np = (uint32_t)(nimg + 1) / 2;  // pairs in this workgroup
  float2* const tw = mr_lds;
  float2* src = mr_lds + pl.ntw;
  float2* dst = src + (size_t)2 * pl.Q * N;
  const bool exact = pl.N == pl.Ld;  // every axis exact: transform point = data point

  // twiddles exp(-2 pi i m / P) of each transformed axis
#pragma unroll
  for (int d = 0; d < 3; ++d) {
    if (pl.P[d] < 2) continue;
    for (int m = tid; m < pl.P[d]; m += NT) tw[pl.twoff[d] + m] = mr_root(m, pl.P[d]);
  }

  // stage z = u + i k of every image on the transform grid
  for (uint32_t f = tid; f < 2 * np * N; f += NT) {
    const uint32_t i = fdiv(f, pl.dN), p = f - i * N;
    float2 z = czero();
    if ((int)i < nimg) {
      const int64_t img = img0 + i;
      const Gates<ACT> G = line_gates<ACT, TS>(ain, img, C);
      const TS* kl = k + (size_t)k_line(img, kC) * pl.Kd;
      const size_t base = (size_t)img * pl.Ld;
      if (exact) {
        z.x = G.u1(ld1(x1 + base + p), ld1(v + base + p), p);
        z.y = ld1(kl + p);
      } else {
        const uint32_t t = fdiv(p, pl.dP2), g2 = p - t * pl.P[2];
        const uint32_t g0 = fdiv(t, pl.dP1), g1 = t - g0 * pl.P[1];
        if ((int)g0 < pl.L[0] && (int)g1 < pl.L[1] && (int)g2 < pl.L[2]) {
          const uint32_t n = (g0 * pl.L[1] + g1) * pl.L[2] + g2;
          z.x = G.u1(ld1(x1 + base + n), ld1(v + base + n), n);
        }
        const int j0 = mr_kidx(g0, pl.kind[0], pl.L[0], pl.P[0]);
        const int j1 = mr_kidx(g1, pl.kind[1], pl.L[1], pl.P[1]);
        const int j2 = mr_kidx(g2, pl.kind[2], pl.L[2], pl.P[2]);
        if (j0 >= 0 && j1 >= 0 && j2 >= 0) z.y = ld1(kl + (j0 * pl.KL[1] + j1) * pl.KL[2] + j2);
      }
    }
    src[f] = z;
  }
  __syncthreads();

  // forward transforms of the 2 np images
  mr_transform<NT>(src, dst, tw, pl, 2 * np * N, tid);

  // products of each pair, conjugated: conj(Ya + i Yb)
  {
    const float scale = 1.f / (float)pl.N;
    for (uint32_t f = tid; f < np * N; f += NT) {
      const uint32_t q = fdiv(f, pl.dN), p = f - q * N;
      const uint32_t t = fdiv(p, pl.dP2), g2 = p - t * pl.P[2];
      const uint32_t g0 = fdiv(t, pl.dP1), g1 = t - g0 * pl.P[1];
      const uint32_t m0 = g0 ? pl.P[0] - g0 : 0, m1 = g1 ? pl.P[1] - g1 : 0, m2 = g2 ? pl.P[2] - g2 : 0;
      const uint32_t pm = (m0 * pl.P[1] + m1) * pl.P[2] + m2;
      const float2* za = src + 2 * q * N;
      const float2* zb = za + N;
      const int64_t ia = img0 + 2 * q, ib = ia + 1;
      const float Da = ld1(Dp + ia % C);
      const float Db = ib < lines ? ld1(Dp + ib % C) : 0.f;
      const float2 ya = mr_product(za[p], za[pm], Da, scale);
      const float2 yb = mr_product(zb[p], zb[pm], Db, scale);
      dst[f] = make_float2(ya.x - yb.y, -(ya.y + yb.x));
    }
    __syncthreads();
    float2* t = src;
    src = dst;
    dst = t;
  }

  // one transform per pair: the conjugate of both inverses
  mr_transform<NT>(src, dst, tw, pl, np * N, tid);

  // crop, outer gate, store: ya = Re, yb = -Im
  for (uint32_t f = tid; f < (uint32_t)nimg * (uint32_t)pl.Ld; f += NT) {
    const uint32_t i = fdiv(f, pl.dLd), n = f - i * (uint32_t)pl.Ld;
    uint32_t p = n;
    if (!exact) {
      const uint32_t t = fdiv(n, pl.dL2), n2 = n - t * pl.L[2];
      const uint32_t n0 = fdiv(t, pl.dL1), n1 = t - n0 * pl.L[1];
      p = (n0 * pl.P[1] + n1) * pl.P[2] + n2;
    }
    const float2 r = src[(i >> 1) * N + p];
    const int64_t img = img0 + i;
    const Gates<ACT> G = line_gates<ACT, TS>(ain, img, C);
    const size_t o = (size_t)img * pl.Ld + n;
    st1(y + o, G.g1(ld1(x2 + o)) * ((i & 1) ? -r.y : r.x));
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

int env_int(const char* name) {
  const char* e = getenv(name);
  return e ? (int)strtol(e, nullptr, 10) : 0;
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
  // passes: each axis, radices 8, 4, 2, 7, 5, 3 in that order
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
      for (int c : {8, 4, 2, 7, 5, 3})
        if (rest % c == 0) {
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
  // Lanes and image pairs per workgroup, from a sweep of 64 .. 1024 lanes and
  // 1 .. 12 pairs on 14^2 to 48 x 64 grids and 300- and 1000-point lines
  // (MI355X): about 3 points of the images' grids per lane below 512
  // transform points, 6 from there, 1024 lanes on one pair from 1536 points.
  int nt = 512, Q = 1;
  if (pl->N < 1536) {
    const int target = pl->N >= 512 ? 3072 : 1536;  // grid points per workgroup
    Q = imax(1, (target + pl->N) / (2 * pl->N));
  } else {
    nt = 1024;
  }
  if (const int o = env_int("HYENAND_MIXED_PAIRS"); o > 0) Q = o;
  if (const int o = env_int("HYENAND_MIXED_LANES"); o == 64 || o == 128 || o == 256 || o == 512 || o == 1024) nt = o;
  const int64_t pairs = (a.lines + 1) / 2;
  if (Q > pairs) Q = (int)pairs;
  while (Q > 1 && ((size_t)pl->ntw + (size_t)4 * Q * pl->N) * sizeof(float2) > kMrMaxLds) --Q;
  if (((size_t)pl->ntw + (size_t)4 * Q * pl->N) * sizeof(float2) > kMrMaxLds) return false;
  pl->Q = Q;
  pl->nt = nt;
  pl->dN = make_fastdiv((uint32_t)pl->N);
  pl->dP1 = make_fastdiv((uint32_t)pl->P[1]);
  pl->dP2 = make_fastdiv((uint32_t)pl->P[2]);
  pl->dL1 = make_fastdiv((uint32_t)pl->L[1]);
  pl->dL2 = make_fastdiv((uint32_t)pl->L[2]);
  pl->dLd = make_fastdiv((uint32_t)pl->Ld);
  return true;
}

template <typename TS, bool ACT, int NT>
hipError_t launch_mixed_t(const FftConvArgs& a, const MrPlan& pl, hipStream_t s) {
  const size_t lds = ((size_t)pl.ntw + (size_t)4 * pl.Q * pl.N) * sizeof(float2);
  const unsigned nblk = (unsigned)((a.lines + 2 * pl.Q - 1) / (2 * pl.Q));
  // the kernel may take more than the default 64 KB of dynamic LDS
  static std::once_flag once;
  static hipError_t attr = hipSuccess;
  std::call_once(once, [] {
    attr = hipFuncSetAttribute(reinterpret_cast<const void*>(conv_mixed<TS, ACT, NT>),
                               hipFuncAttributeMaxDynamicSharedMemorySize, (int)kMrMaxLds);
  });
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL((conv_mixed<TS, ACT, NT>), dim3(nblk), dim3(NT), lds, s, (const TS*)a.x1, (const TS*)a.x2,
                     (const TS*)a.v, (const TS*)a.k, (const TS*)a.D, (TS*)a.y, (int64_t)a.lines, (int)a.C, a.kC,
                     a.act_in, pl);
  return hipGetLastError();
}

template <int NT>
hipError_t launch_mixed_nt(const FftConvArgs& a, const MrPlan& pl, hipStream_t s) {
  if (a.bf16)
    return a.act ? launch_mixed_t<uint16_t, true, NT>(a, pl, s) : launch_mixed_t<uint16_t, false, NT>(a, pl, s);
  return a.act ? launch_mixed_t<float, true, NT>(a, pl, s) : launch_mixed_t<float, false, NT>(a, pl, s);
}

}  // namespace

bool mixed_supported(const FftConvArgs& a) {
  MrPlan pl;
  return mixed_plan(a, &pl);
}

// Where these kernels beat the power-of-two ones (measured on the MI355X):
// 3D grids (which those do not take), 2D grids up to 2048 transform points
// (14 x 14: 14.7 us against 105 us for 16 x 384 images; 27 x 27 centred:
// 44 us against 111 us) and larger ones with at most a quarter of the
// power-of-two points (48 x 64: 21 us against 60 us; 48 x 80 at half: 91 us
// against 62 us), lines of at most 128 points (64 x 256 lines of 12: 6.7 us
// against 20.6 us; 64 x 64 of 100: 8.6 against 11.0) or a third of the
// power-of-two points (300: 15.5 us against 17.9 us; 500 and 1000 at half:
// 23.6 and 44 us against 20.5 and 40 us).
bool mixed_preferred(const FftConvArgs& a) {
  MrPlan pl;
  if (!mixed_plan(a, &pl)) return false;
  int64_t pow2_points = 1;
  for (int d = 0; d < a.ndim; ++d) pow2_points *= a.P[d];
  if (a.ndim == 3) return true;
  if (a.ndim == 2) return pl.N <= 2048 || 4 * (int64_t)pl.N <= pow2_points;
  return pl.N <= 128 || 3 * (int64_t)pl.N <= pow2_points;
}

hipError_t launch_mixed(const FftConvArgs& a, hipStream_t s) {
  MrPlan pl;
  if (!mixed_plan(a, &pl)) return hipErrorInvalidValue;
  switch (pl.nt) {
    case 64: return launch_mixed_nt<64>(a, pl, s);
    case 128: return launch_mixed_nt<128>(a, pl, s);
    case 512: return launch_mixed_nt<512>(a, pl, s);
    case 1024: return launch_mixed_nt<1024>(a, pl, s);
    default: return launch_mixed_nt<256>(a, pl, s);
  }
}

}  // namespace hyenand
