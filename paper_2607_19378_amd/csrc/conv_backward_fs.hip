// Backward of the gated long convolution for 1D lines beyond the single-pass
// limit (2^14 to 2^22 transform points): the four-step structure of the
// forward plan (M = P/2 = N1 x N2, m = m1 N2 + m2, f = f1 + N1 f2) carried
// over to three signals.
//
// With u = x1 v and h = gy x2 the gradients come from the spectral products
// Z = U (K + D), GU = conj(K + D) H and GK = conj(U) H (gx2 = gy z,
// gx1 = gu v, gv = gu x1, gk, and gD[c] = sum_{b, n} h u), cropped like y:
//
//   cols_fwd  per column m2 and signal (u, k or h): transform over m1,
//             twiddle exp(-2 pi i m2 f1 / M), store A[f1][m2].
//   core      per row pair (f1, N1 - f1): transforms over m2 of the three
//             signals; bins g and M - g sit in the pair, so the real spectra
//             are untangled, the three products formed and packed again for
//             half-length inverses; inverse transforms over f2, twiddle
//             exp(+2 pi i f1 m2 / M); Z, GU, GK overwrite A_u, A_k, A_h.
//   cols_inv  per column m2: inverse transforms over f1 of Z, GU and GK
//             (one exchange tile in turn), keep m1 < N1/2 (linear), unpack,
//             write gx2, gx1, gv, gk; per-workgroup sums of h u for gD.
#include "fourstep.hpp"

namespace hyenand {

namespace {

template <int NT>
__device__ __forceinline__ float fs_wg_sum(float x, float* red, int tid) {
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

template <int N1, bool CIRC, typename TS>
__global__ void __launch_bounds__(ColCfgFwd<N1>::NT) __attribute__((amdgpu_waves_per_eu(ColCfgFwd<N1>::kWaves)))
    fsb_cols_fwd(const TS* __restrict__ x1, const TS* __restrict__ v, const TS* __restrict__ k,
                 const TS* __restrict__ gy, const TS* __restrict__ x2, float2* __restrict__ ws, int64_t line0,
                 int N2, int log2M, int64_t per_line) {
  using Cf = ColCfgFwd<N1>;
  constexpr int E = Cf::E, T = Cf::T, NT = Cf::NT, TL = Cf::TL, TLP = Cf::TLP;
  constexpr int NZ = CIRC ? N1 : N1 / 2;  // nonzero rows m1
  static_assert(NT / T >= TL, "one round covers the tile");
  __shared__ float2 tile[N1 * TLP];
  __shared__ float2 twl[imax(1, PassTw<N1, E>::kCount)];
  PassTw<N1, E>::fill(twl, threadIdx.x, NT);
  const int ntile = N2 / TL;
  const int sig = (int)(blockIdx.x % 3);  // 0: u = x1 v, 1: k, 2: h = gy x2
  const int64_t rest = blockIdx.x / 3;
  const int64_t line = rest / ntile;
  const int c0 = (int)(rest % ntile) * TL;
  const int64_t M = (int64_t)N1 * N2;
  const int64_t L = CIRC ? 2 * M : M;
  const size_t gbase = (size_t)(line0 + line) * L;
  const int tid = threadIdx.x;
  const int cc = tid % (NT / T), t = tid / (NT / T);
  const bool act = cc < TL;

  float2 w[E];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int m1 = t + T * e;
    w[e] = czero();
    if (act && (CIRC || m1 < NZ)) {
      const size_t n = gbase + 2 * ((size_t)m1 * N2 + c0 + cc);
      if (sig == 0) {
        const float2 a = ld2(x1 + n), b = ld2(v + n);
        w[e] = make_float2(a.x * b.x, a.y * b.y);
      } else if (sig == 1) {
        w[e] = ld2(k + n);
      } else {
        const float2 a = ld2(gy + n), b = ld2(x2 + n);
        w[e] = make_float2(a.x * b.x, a.y * b.y);
      }
    }
  }
  BlockFFT<N1, E, false>::run(w, t, ScrS<TLP>{tile + (act ? cc : 0)}, act, twl);
  if (act) {
    const uint32_t m2 = (uint32_t)(c0 + cc);
    twiddle_run<E>(w, twiddle_rt<false>(m2 * (uint32_t)t, log2M), twiddle_rt<false>(m2 * (uint32_t)T, log2M));
    float2* A = ws + line * per_line + sig * M + c0 + cc;
#pragma unroll
    for (int e = 0; e < E; ++e) A[(size_t)(t + T * e) * N2] = w[e];
  }
}

// 1024 lanes: six rows of 2048 points (u, k, h at f1 = fa and fb) on 768 of
// them during the transforms, all of them during the products.
template <bool CIRC>
__global__ void __launch_bounds__(1024)
    fsb_core(float2* __restrict__ ws, const void* __restrict__ Dp, int dbf16, int64_t line0, int C, int N1,
             int log2M, int64_t per_line, float scale) {
  constexpr int N2 = kN2;
  constexpr int E = 16, T = N2 / E, NT = 1024;
  constexpr int RS = pad16_size(N2);
  constexpr int IPT = N2 / NT;
  __shared__ float2 R[6][RS];  // u fa, u fb, k fa, k fb, h fa, h fb
  __shared__ float2 twl[PassTw<N2, E>::kCount];
  PassTw<N2, E>::fill(twl, threadIdx.x, NT);
  const int npair = N1 / 2 + 1;
  const int64_t line = blockIdx.x / npair;
  const int fa = (int)(blockIdx.x % npair);
  const int fb = (N1 - fa) & (N1 - 1);
  const bool single = fa == fb;  // rows 0 and N1/2 are their own mirrors
  const int64_t M = (int64_t)N1 * N2;
  const int c = (int)((line0 + line) % C);
  const float twoD = 2.f * (dbf16 ? ld1((const uint16_t*)Dp + c) : ld1((const float*)Dp + c));
  float2* A = ws + line * per_line;
  const int tid = threadIdx.x;
  const float2 om_a = twiddle_rt<false>((uint32_t)fa, log2M + 1);

  // forward transforms over m2: slot sl = 2 signal + (row fb ? 1 : 0)
  {
    const int sl = tid / T, t = tid % T;
    const bool act = sl < 6 && (!single || (sl & 1) == 0);
    const ScrPad16 sc{R[act ? sl : 0]};
    const float2* src = A + (act ? sl >> 1 : 0) * M + (int64_t)((sl & 1) ? fb : fa) * N2 + t;
    float2 w[E];
#pragma unroll
    for (int e = 0; e < E; ++e) w[e] = act ? src[T * e] : czero();
    BlockFFT<N2, E, false>::run(w, t, sc, act, twl);
    if (act) {
#pragma unroll
      for (int e = 0; e < E; ++e) *sc(t + T * e) = w[e];
    }
  }
  __syncthreads();

  // untangle, the three products, pack each for a half-length inverse
  const int ob = single ? 0 : 1;
  float2 zg[IPT], zm[IPT], ug[IPT], um[IPT], kg[IPT], km[IPT];
  int mcol[IPT];
#pragma unroll
  for (int j = 0; j < IPT; ++j) {
    const int f2 = tid + NT * j;
    const int mc = fa == 0 ? ((N2 - f2) & (N2 - 1)) : (N2 - 1 - f2);
    mcol[j] = mc;
    static_assert(2 * N2 == 4096, "the untangling twiddle uses the 4096-point table");
    const float2 om = c_mul(om_a, kTwCoarse[f2]);  // exp(-2 pi i g / P)
    const float2 omm = make_float2(-om.x, om.y);   // exp(-2 pi i (M - g) / P)
    float2 Ug, Umg, Kg, Kmg, Hg, Hmg;
    r2c_pair(*ScrPad16{R[0]}(f2), *ScrPad16{R[ob]}(mc), om, Ug, Umg);
    r2c_pair(*ScrPad16{R[2]}(f2), *ScrPad16{R[2 + ob]}(mc), om, Kg, Kmg);
    r2c_pair(*ScrPad16{R[4]}(f2), *ScrPad16{R[4 + ob]}(mc), om, Hg, Hmg);
    const float2 kdg = make_float2(Kg.x + twoD, Kg.y), kdm = make_float2(Kmg.x + twoD, Kmg.y);
    const float2 Zg = c_mul(Ug, kdg), Zm = c_mul(Umg, kdm);
    const float2 Gg = c_mulc(Hg, kdg), Gm = c_mulc(Hmg, kdm);
    const float2 Qg = c_mulc(Hg, Ug), Qm = c_mulc(Hmg, Umg);
    zg[j] = c_scale(c2r_pair(Zg, Zm, om), scale);
    zm[j] = c_scale(c2r_pair(Zm, Zg, omm), scale);
    ug[j] = c_scale(c2r_pair(Gg, Gm, om), scale);
    um[j] = c_scale(c2r_pair(Gm, Gg, omm), scale);
    kg[j] = c_scale(c2r_pair(Qg, Qm, om), scale);
    km[j] = c_scale(c2r_pair(Qm, Qg, omm), scale);
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < IPT; ++j) {
    const int f2 = tid + NT * j;
    *ScrPad16{R[0]}(f2) = zg[j];
    *ScrPad16{R[2]}(f2) = ug[j];
    *ScrPad16{R[4]}(f2) = kg[j];
    if (!single) {
      *ScrPad16{R[1]}(mcol[j]) = zm[j];
      *ScrPad16{R[3]}(mcol[j]) = um[j];
      *ScrPad16{R[5]}(mcol[j]) = km[j];
    }
  }
  __syncthreads();

  // inverse transforms over f2, twiddle exp(+2 pi i f1 m2 / M), store over A
  {
    const int sl = tid / T, t = tid % T;
    const bool act = sl < 6 && (!single || (sl & 1) == 0);
    const ScrPad16 sc{R[act ? sl : 0]};
    const uint32_t f1 = (uint32_t)((sl & 1) ? fb : fa);
    float2 w[E];
#pragma unroll
    for (int e = 0; e < E; ++e) w[e] = act ? *sc(t + T * e) : czero();
    BlockFFT<N2, E, true>::run(w, t, sc, act, twl);
    if (act) {
      twiddle_run<E>(w, twiddle_rt<true>(f1 * (uint32_t)t, log2M), twiddle_rt<true>(f1 * (uint32_t)T, log2M));
      float2* dst = A + (sl >> 1) * M + (int64_t)f1 * N2 + t;
#pragma unroll
      for (int e = 0; e < E; ++e) dst[T * e] = w[e];
    }
  }
}

template <int N1, bool CIRC, typename TS>
__global__ void __launch_bounds__(512)
    fsb_cols_inv(const float2* __restrict__ ws, const TS* __restrict__ x1, const TS* __restrict__ v,
                 const TS* __restrict__ gy, const TS* __restrict__ x2, TS* __restrict__ gx1, TS* __restrict__ gx2,
                 TS* __restrict__ gv, TS* __restrict__ gk, float* __restrict__ partial, int64_t line0, int N2,
                 int64_t per_line) {
  using Cf = ColCfg<N1>;
  constexpr int E = Cf::E, T = Cf::T, NT = Cf::NT, TL = Cf::TL, TLP = Cf::TLP;
  constexpr int NOUT = CIRC ? N1 : N1 / 2;  // cropped rows m1
  static_assert(NT / T >= TL, "one round covers the tile");
  __shared__ float2 tile[N1 * TLP];
  __shared__ float2 twl[imax(1, PassTw<N1, E>::kCount)];
  __shared__ float red[NT / 64];
  PassTw<N1, E>::fill(twl, threadIdx.x, NT);
  const int ntile = N2 / TL;
  const uint32_t bid = fs_pair_tiles<1>(blockIdx.x);
  const int64_t line = bid / ntile;
  const int c0 = (int)(bid % ntile) * TL;
  const int64_t M = (int64_t)N1 * N2;
  const int64_t L = CIRC ? 2 * M : M;
  const int tid = threadIdx.x;
  const int cc = tid % (NT / T), t = tid / (NT / T);
  const bool act = cc < TL;

  const float2* B = ws + line * per_line + c0 + cc;
  float2 wz[E], wu[E], wk[E];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const size_t o = (size_t)(t + T * e) * N2;
    wz[e] = act ? B[o] : czero();
    wu[e] = act ? B[M + o] : czero();
    wk[e] = act ? B[2 * M + o] : czero();
  }
  const ScrS<TLP> sc{tile + (act ? cc : 0)};
  BlockFFT<N1, E, true>::run(wz, t, sc, act, twl);
  BlockFFT<N1, E, true>::run(wu, t, sc, act, twl);
  BlockFFT<N1, E, true>::run(wk, t, sc, act, twl);
  float hu = 0.f;
  if (act) {
    const size_t gbase = (size_t)(line0 + line) * L + 2 * (size_t)(c0 + cc);
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int m1 = t + T * e;
      if (CIRC || m1 < NOUT) {
        const size_t n = gbase + 2 * (size_t)m1 * N2;
        const float2 a = ld2(x1 + n), b = ld2(v + n), g = ld2(gy + n), q = ld2(x2 + n);
        st2(gx2 + n, make_float2(g.x * wz[e].x, g.y * wz[e].y));
        st2(gx1 + n, make_float2(b.x * wu[e].x, b.y * wu[e].y));
        st2(gv + n, make_float2(a.x * wu[e].x, a.y * wu[e].y));
        st2(gk + n, wk[e]);
        hu += (a.x * b.x) * (g.x * q.x) + (a.y * b.y) * (g.y * q.y);
      }
    }
  }
  const float tot = fs_wg_sum<NT>(hu, red, tid);
  if (tid == 0) partial[(line0 + line) * ntile + (bid % ntile)] = tot;
}

struct FsbLaunch {
  const FftConvBwdArgs* b;
  float2* ws;
  int64_t line0;
  int nl;
  int N1, log2M;
  int64_t per;
  float scale;
  hipStream_t s;
};

template <int N1>
hipError_t b_cols_fwd(const FsbLaunch& L) {
  constexpr int TL = ColCfgFwd<N1>::TL;
  const dim3 grid((unsigned)((int64_t)L.nl * (kN2 / TL) * 3));
  const FftConvArgs& a = L.b->f;
#define HY_ARGS(TS) \
  (const TS*)a.x1, (const TS*)a.v, (const TS*)a.k, (const TS*)L.b->gy, (const TS*)a.x2, L.ws, L.line0, kN2, L.log2M, L.per
  if (a.bf16) {
    if (a.circular) hipLaunchKernelGGL((fsb_cols_fwd<N1, true, uint16_t>), grid, dim3(ColCfgFwd<N1>::NT), 0, L.s, HY_ARGS(uint16_t));
    else hipLaunchKernelGGL((fsb_cols_fwd<N1, false, uint16_t>), grid, dim3(ColCfgFwd<N1>::NT), 0, L.s, HY_ARGS(uint16_t));
  } else {
    if (a.circular) hipLaunchKernelGGL((fsb_cols_fwd<N1, true, float>), grid, dim3(ColCfgFwd<N1>::NT), 0, L.s, HY_ARGS(float));
    else hipLaunchKernelGGL((fsb_cols_fwd<N1, false, float>), grid, dim3(ColCfgFwd<N1>::NT), 0, L.s, HY_ARGS(float));
  }
#undef HY_ARGS
  return hipGetLastError();
}

template <int N1>
hipError_t b_cols_inv(const FsbLaunch& L) {
  constexpr int TL = ColCfg<N1>::TL;
  const dim3 grid((unsigned)((int64_t)L.nl * (kN2 / TL)));
  const FftConvArgs& a = L.b->f;
  const FftConvBwdArgs& b = *L.b;
#define HY_ARGS(TS)                                                                                            \
  L.ws, (const TS*)a.x1, (const TS*)a.v, (const TS*)b.gy, (const TS*)a.x2, (TS*)b.gx1, (TS*)b.gx2, (TS*)b.gv, \
      (TS*)b.gk, b.partial, L.line0, kN2, L.per
  if (a.bf16) {
    if (a.circular) hipLaunchKernelGGL((fsb_cols_inv<N1, true, uint16_t>), grid, dim3(512), 0, L.s, HY_ARGS(uint16_t));
    else hipLaunchKernelGGL((fsb_cols_inv<N1, false, uint16_t>), grid, dim3(512), 0, L.s, HY_ARGS(uint16_t));
  } else {
    if (a.circular) hipLaunchKernelGGL((fsb_cols_inv<N1, true, float>), grid, dim3(512), 0, L.s, HY_ARGS(float));
    else hipLaunchKernelGGL((fsb_cols_inv<N1, false, float>), grid, dim3(512), 0, L.s, HY_ARGS(float));
  }
#undef HY_ARGS
  return hipGetLastError();
}

#define HY_BN1_SWITCH(N, FN, ARG)          \
  switch (N) {                             \
    case 4: return FN<4>(ARG);             \
    case 8: return FN<8>(ARG);             \
    case 16: return FN<16>(ARG);           \
    case 32: return FN<32>(ARG);           \
    case 64: return FN<64>(ARG);           \
    case 128: return FN<128>(ARG);         \
    case 256: return FN<256>(ARG);         \
    case 512: return FN<512>(ARG);         \
    case 1024: return FN<1024>(ARG);       \
    default: return hipErrorInvalidValue;  \
  }

hipError_t d_b_cols_fwd(const FsbLaunch& L) { HY_BN1_SWITCH(L.N1, b_cols_fwd, L) }
hipError_t d_b_cols_inv(const FsbLaunch& L) { HY_BN1_SWITCH(L.N1, b_cols_inv, L) }

int cols_tile(int N1) {
  switch (N1) {
#define HY_CASE(n) \
  case n: return ColCfg<n>::TL;
    HY_CASE(4) HY_CASE(8) HY_CASE(16) HY_CASE(32) HY_CASE(64) HY_CASE(128) HY_CASE(256) HY_CASE(512)
    HY_CASE(1024)
#undef HY_CASE
    default: return 1;
  }
}

}  // namespace

// the forward's four-step shapes and one more: N1 = 4 (16384-point lines,
// which the forward runs in a single pass)
bool backward_fs_supported(const FftConvArgs& a) {
  if (a.ndim != 1) return false;
  const int64_t M = a.P[0] / 2;
  if (M % kN2 != 0) return false;
  const int64_t N1 = M / kN2;
  return N1 >= 4 && N1 <= kMaxN1;
}

size_t backward_fs_bytes_per_line(const FftConvArgs& a) {
  return (size_t)(a.P[0] / 2) * 3 * sizeof(float2);  // A_u, A_k, A_h
}

int64_t backward_fs_partials_per_line(const FftConvArgs& a) {
  const int N1 = (int)(a.P[0] / 2 / kN2);
  return kN2 / cols_tile(N1);
}

hipError_t launch_backward_fs(const FftConvBwdArgs& b, int64_t line0, int64_t nl, void* ws, hipStream_t s) {
  const FftConvArgs& a = b.f;
  if (!backward_fs_supported(a) || nl < 1 || line0 < 0 || line0 + nl > a.lines) return hipErrorInvalidValue;
  FsbLaunch L;
  L.b = &b;
  L.ws = (float2*)ws;
  const int64_t M = a.P[0] / 2;
  L.N1 = (int)(M / kN2);
  L.log2M = ilog2_rt(M);
  L.per = 3 * M;
  L.scale = (float)(1.0 / (4.0 * (double)a.P[0]));
  L.s = s;
  L.line0 = line0;
  L.nl = (int)nl;
  hipError_t e;
  if ((e = d_b_cols_fwd(L)) != hipSuccess) return e;
  const dim3 grid((unsigned)((int64_t)L.nl * (L.N1 / 2 + 1)));
  if (a.circular)
    hipLaunchKernelGGL((fsb_core<true>), grid, dim3(1024), 0, s, L.ws, a.D, (int)a.bf16, line0, (int)a.C, L.N1,
                       L.log2M, L.per, L.scale);
  else
    hipLaunchKernelGGL((fsb_core<false>), grid, dim3(1024), 0, s, L.ws, a.D, (int)a.bf16, line0, (int)a.C, L.N1,
                       L.log2M, L.per, L.scale);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  return d_b_cols_inv(L);
}

}  // namespace hyenand
