// Multi-pass 1D plan for lines longer than the single-pass limit.
//
// The real line of transform length P is read as its even/odd packed complex
// line z[m] = x[2m] + i x[2m+1] of length M = P/2, and the length-M transform
// is split four-step style as M = N1 x N2 with m = m1 N2 + m2 and
// f = f1 + N1 f2 (the paper's three-kernel Cooley-Tukey treatment of long
// lines, appendix "1D FFT Convolution"):
//
//   cols_fwd  per column m2: transform over m1 (length N1; zero half skipped
//             in linear mode) for u = x1 v and for k, twiddle
//             exp(-2 pi i m2 f1 / M); store A[f1][m2] (both signals).
//   core      per row pair (f1, N1 - f1): transforms over m2 (length N2) give
//             the packed spectra of u and k; bins g and M - g sit in this row
//             pair, so the real spectra are untangled (r2c_pair), multiplied
//             (gated product, shortcut folded in), and packed again for a
//             half-length inverse (c2r_pair); inverse transforms over f2,
//             twiddle exp(+2 pi i f1 m2 / M); store in place of A_u.
//   cols_inv  per column m2: inverse transform over f1 (length N1), keep the
//             cropped m1 < N1/2, unpack y[2m], y[2m+1], outer gate, store.
//
// Inputs are read once, y written once; the two complex spectra (16 B per
// packed sample) round-trip through the workspace, chunked by lines.
#include "fourstep.hpp"

namespace hyenand {

namespace {

// KC: k is the centered kernel of 2L - 1 points (linear transform grid); its
// column lines have no zero half.
template <int N1, bool CIRC, typename TS, bool KC = false, bool ACT = false>
__global__ void __launch_bounds__(ColCfgFwd<N1>::NT) __attribute__((amdgpu_waves_per_eu(ColCfgFwd<N1>::kWaves)))
    fs_cols_fwd(const TS* __restrict__ x1, const TS* __restrict__ v, const TS* __restrict__ k,
                float2* __restrict__ ws, int64_t line0, int N2, int log2M, int64_t per_line, int kC, ActIn ain,
                int C, int u_only) {
  static_assert(!(KC && CIRC), "centered kernels use the linear transform grid");
  using Cf = ColCfgFwd<N1>;
  constexpr int E = Cf::E, T = Cf::T, NT = Cf::NT, TL = Cf::TL, TLP = Cf::TLP;
  constexpr int NZ = CIRC ? N1 : N1 / 2;  // nonzero rows m1 of u (and of k unless centered)
  static_assert(NT / T >= TL, "one round covers the tile");
  __shared__ float2 tile[N1 * TLP];  // exchange scratch, one column per line
  __shared__ float2 twl[imax(1, PassTw<N1, E>::kCount)];
  PassTw<N1, E>::fill(twl, threadIdx.x, NT);
  const int ntile = N2 / TL;
  // 0: u = x1 v, 1: k (u_only: every workgroup takes u; k comes from
  // fs_cols_modal)
  const uint32_t bid = u_only ? blockIdx.x : fs_pair_tiles<2>(blockIdx.x);
  const int sig = u_only ? 0 : (int)(bid & 1);
  const int64_t rest = u_only ? (int64_t)bid : (int64_t)(bid >> 1);
  const int64_t line = rest / ntile;
  const int c0 = (int)(rest % ntile) * TL;
  const int64_t M = (int64_t)N1 * N2;
  const int64_t L = CIRC ? 2 * M : M;  // real samples per line
  const size_t gbase = (size_t)(line0 + line) * L;
  const size_t kbase = (size_t)k_line(line0 + line, kC) * L;
  const int tid = threadIdx.x;
  // lanes with consecutive ids take consecutive columns of one row, so every
  // global access below is a contiguous run of TL values per row
  const int cc = tid % (NT / T), t = tid / (NT / T);
  const bool act = cc < TL;

  // column points straight from global memory into registers (lane t holds
  // m1 = t + T e); rows at or beyond NZ are the zero padding
  float2 w[E];
  if (KC && sig == 1) {
    // grid points 2m, 2m + 1 (m = m1 N2 + m2) from the 2L - 1 centered points
    const TS* kl = k + (size_t)k_line(line0 + line, kC) * (size_t)(2 * L - 1);
    const int Li = (int)L;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int m1 = t + T * e;
      w[e] = czero();
      if (act) {
        const int g = 2 * (m1 * N2 + c0 + cc);
        const int ja = centered_index(g, Li, 2 * Li), jb = centered_index(g + 1, Li, 2 * Li);
        w[e] = make_float2(ja >= 0 ? ld1(kl + ja) : 0.f, jb >= 0 ? ld1(kl + jb) : 0.f);
      }
    }
  } else {
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int m1 = t + T * e;
      w[e] = czero();
      if (act && (CIRC || m1 < NZ)) {
        const size_t n = gbase + 2 * ((size_t)m1 * N2 + c0 + cc);
        if (sig == 0) {
          w[e] = line_gates<ACT, TS>(ain, line0 + line, C).u2(ld2(x1 + n), ld2(v + n), (int64_t)(n - gbase));
        } else {
          w[e] = ld2(k + n - gbase + kbase);
        }
      }
    }
  }
  BlockFFT<N1, E, false>::run(w, t, ScrS<TLP>{tile + (act ? cc : 0)}, act, twl);
  if (act) {
    // exp(-2 pi i m2 f1 / M) for f1 = t + T e, then A[f1][m2]
    const uint32_t m2 = (uint32_t)(c0 + cc);
    twiddle_run<E>(w, twiddle_rt<false>(m2 * (uint32_t)t, log2M), twiddle_rt<false>(m2 * (uint32_t)T, log2M));
    float2* A = ws + line * per_line + (sig ? M : 0) + c0 + cc;
#pragma unroll
    for (int e = 0; e < E; ++e) A[(size_t)(t + T * e) * N2] = w[e];
  }
}

// Columns of the packed kernel line for a modal filter generated in place of
// the k read (section 3.2.1's kernel evaluated inside the FFT kernel, here the
// implicit modal filter of the appendix "Filter Generation"): for line
// (b, c) the lane holding rows m1 = t + T e of column m2 needs
// k[2m] + i k[2m + 1], m = m1 N2 + m2, with k[s] = Re sum_j R_j lambda_j^s.
// The workgroup first tabulates, exactly (polar: double phase), A_j[cc] =
// R_j lambda_j^(2 m2) for its TL columns, B_j[t] = lambda_j^(2 N2 t) for the
// T lane rows, the step lambda_j^(2 N2 T) and lambda_j; a lane's first point
// is A_j[cc] B_j[t] and each further row one fp32 step on, at most
// N1 / T - 1 steps from an exact anchor.  Then the same column transform,
// twiddle and store as the k columns of fs_cols_fwd.
template <int N1, bool CIRC>
__global__ void __launch_bounds__(512)
    fs_cols_modal(ModalIn md, float2* __restrict__ ws, int64_t line0, int N2, int log2M, int64_t per_line, int C) {
  using Cf = ColCfg<N1>;
  constexpr int E = Cf::E, T = Cf::T, NT = Cf::NT, TL = Cf::TL, TLP = Cf::TLP;
  constexpr int NZ = CIRC ? N1 : N1 / 2;  // nonzero rows m1 of the kernel
  static_assert(NT / T >= TL, "one round covers the tile");
  __shared__ float2 tile[N1 * TLP];
  __shared__ float2 twl[imax(1, PassTw<N1, E>::kCount)];
  // the mode tables, sized by the order at launch (modal_lds_bytes): two
  // workgroups share a CU up to order 16 with 512-point columns
  extern __shared__ float2 mtab[];
  const int nm = md.M;
  float2* const tA = mtab;            // [nm][TL]
  float2* const tB = tA + nm * TL;    // [nm][T]
  float2* const tS = tB + nm * T;     // [nm]
  float2* const tL = tS + nm;         // [nm]
  const int tid = threadIdx.x;
  PassTw<N1, E>::fill(twl, tid, NT);
  const int ntile = N2 / TL;
  const int64_t line = blockIdx.x / ntile;
  const int c0 = (int)(blockIdx.x % ntile) * TL;
  const int64_t M = (int64_t)N1 * N2;
  const int64_t ch = (line0 + line) % C;
  const float* pa = md.a + ch * nm;
  const float* pt = md.th + ch * nm;
  for (int i = tid; i < nm * (TL + T + 2); i += NT) {
    int j, kind, idx;
    if (i < nm * TL) {
      j = i / TL, idx = i - j * TL, kind = 0;
    } else if (i < nm * (TL + T)) {
      j = (i - nm * TL) / T, idx = i - nm * TL - j * T, kind = 1;
    } else {
      j = (i - nm * (TL + T)) >> 1, idx = 0, kind = 2 + ((i - nm * (TL + T)) & 1);
    }
    const double s = kind == 0 ? 2.0 * (double)(c0 + idx)
                               : (kind == 1 ? 2.0 * (double)N2 * idx : (kind == 2 ? 2.0 * (double)N2 * T : 1.0));
    float cs, sn, mg;
    polar(s * (double)pa[j], s * (double)pt[j], cs, sn, mg);
    float2 z = make_float2(mg * cs, mg * sn);
    if (kind == 0) z = c_mul(make_float2(md.re[ch * nm + j], md.im[ch * nm + j]), z);
    if (kind == 0) tA[j * TL + idx] = z;
    else if (kind == 1) tB[j * T + idx] = z;
    else if (kind == 2) tS[j] = z;
    else tL[j] = z;
  }
  __syncthreads();
  const int cc = tid % (NT / T), t = tid / (NT / T);
  const bool act = cc < TL;
  float2 w[E];
#pragma unroll
  for (int e = 0; e < E; ++e) w[e] = czero();
  if (act) {
    for (int j = 0; j < nm; ++j) {
      float2 z = c_mul(tA[j * TL + cc], tB[j * T + t]);
      const float2 st = tS[j], l1 = tL[j];
#pragma unroll
      for (int e = 0; e < E; ++e) {
        if (CIRC || t + T * e < NZ) {
          w[e].x += z.x;                                  // k[2m]
          w[e].y = fmaf(z.x, l1.x, fmaf(-z.y, l1.y, w[e].y));  // k[2m + 1] = Re(z lambda)
          z = c_mul(z, st);
        }
      }
    }
  }
  BlockFFT<N1, E, false>::run(w, t, ScrS<TLP>{tile + (act ? cc : 0)}, act, twl);
  if (act) {
    const uint32_t m2 = (uint32_t)(c0 + cc);
    twiddle_run<E>(w, twiddle_rt<false>(m2 * (uint32_t)t, log2M), twiddle_rt<false>(m2 * (uint32_t)T, log2M));
    float2* A = ws + line * per_line + M + c0 + cc;
#pragma unroll
    for (int e = 0; e < E; ++e) A[(size_t)(t + T * e) * N2] = w[e];
  }
}

template <bool CIRC>
__global__ void __launch_bounds__(512)
    fs_core(float2* __restrict__ ws, const void* __restrict__ Dp, int dbf16, int64_t line0, int C, int N1,
            int log2M, int64_t per_line, float scale) {
  constexpr int N2 = kN2;
  constexpr int E = 16, T = N2 / E, NT = 512;
  constexpr int RS = pad16_size(N2);
  constexpr int IPT = N2 / NT;
  __shared__ float2 R[4][RS];  // u row a, u row b, k row a, k row b
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
  // exp(-2 pi i g / P) for g = fa + N1 f2 is exp(-2 pi i fa / P) exp(-2 pi i f2 / (2 N2))
  const float2 om_a = twiddle_rt<false>((uint32_t)fa, log2M + 1);
  // slots: 0 = u row fa, 1 = u row fb, 2 = k row fa, 3 = k row fb (a single
  // self-mirrored row uses slots 0 and 2 only).  Forward transforms over m2,
  // lanes along each row; lane t holds f2 = t + T e straight from global
  // memory (consecutive lanes, consecutive addresses).
  {
    const int sl = tid / T, t = tid % T;
    const bool act = sl < 4 && (!single || (sl & 1) == 0);
    const ScrPad16 sc{R[sl & 3]};
    const float2* src = A + ((sl >> 1) ? M : 0) + (int64_t)((sl & 1) ? fb : fa) * N2 + t;
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

  // untangle, gated product, pack for the half-length inverse
  const ScrPad16 ua{R[0]}, ub{R[single ? 0 : 1]}, ka{R[2]}, kb{R[single ? 2 : 3]};
  float2 wg[IPT], wm[IPT];
  int mcol[IPT];
#pragma unroll
  for (int j = 0; j < IPT; ++j) {
    const int f2 = tid + NT * j;
    const int mc = fa == 0 ? ((N2 - f2) & (N2 - 1)) : (N2 - 1 - f2);
    mcol[j] = mc;
    static_assert(2 * N2 == 4096, "the untangling twiddle uses the 4096-point table");
    const float2 om = c_mul(om_a, kTwCoarse[f2]);  // exp(-2 pi i g / P)
    float2 Ug, Umg, Kg, Kmg;
    r2c_pair(*ua(f2), *ub(mc), om, Ug, Umg);
    r2c_pair(*ka(f2), *kb(mc), om, Kg, Kmg);
    const float2 Yg = gated_product(Ug, Kg, twoD);
    const float2 Ymg = gated_product(Umg, Kmg, twoD);
    wg[j] = c_scale(c2r_pair(Yg, Ymg, om), scale);
    const float2 omm = make_float2(-om.x, om.y);  // exp(-2 pi i (M - g) / P) = -conj(om)
    wm[j] = c_scale(c2r_pair(Ymg, Yg, omm), scale);
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < IPT; ++j) {
    const int f2 = tid + NT * j;
    *ua(f2) = wg[j];
    if (!single) *ub(mcol[j]) = wm[j];
  }
  __syncthreads();

  // inverse transforms over f2, twiddle exp(+2 pi i f1 m2 / M), store over A_u
  {
    const int sl = tid / T, t = tid % T;
    const bool act = sl < (single ? 1 : 2);
    const ScrPad16 sc{R[sl & 1]};
    const uint32_t f1 = (uint32_t)(sl == 0 ? fa : fb);
    float2 w[E];
#pragma unroll
    for (int e = 0; e < E; ++e) w[e] = act ? *sc(t + T * e) : czero();
    BlockFFT<N2, E, true>::run(w, t, sc, act, twl);
    if (act) {
      // exp(+2 pi i f1 m2 / M) for m2 = t + T e
      twiddle_run<E>(w, twiddle_rt<true>(f1 * (uint32_t)t, log2M), twiddle_rt<true>(f1 * (uint32_t)T, log2M));
#pragma unroll
      for (int e = 0; e < E; ++e) A[(int64_t)f1 * N2 + t + T * e] = w[e];
    }
  }
}

template <int N1, bool CIRC, typename TS, bool ACT = false>
__global__ void __launch_bounds__(ColCfgFwd<N1>::NT) __attribute__((amdgpu_waves_per_eu(ColCfgFwd<N1>::kWaves)))
    fs_cols_inv(const float2* __restrict__ ws, const TS* __restrict__ x2, TS* __restrict__ y, int64_t line0, int N2,
                int64_t per_line) {
  using Cf = ColCfgFwd<N1>;
  constexpr int E = Cf::E, T = Cf::T, NT = Cf::NT, TL = Cf::TL, TLP = Cf::TLP;
  constexpr int NOUT = CIRC ? N1 : N1 / 2;  // cropped rows m1
  static_assert(NT / T >= TL, "one round covers the tile");
  __shared__ float2 tile[N1 * TLP];  // exchange scratch, one column per line
  __shared__ float2 twl[imax(1, PassTw<N1, E>::kCount)];
  PassTw<N1, E>::fill(twl, threadIdx.x, NT);
  const int ntile = N2 / TL;
  // the x2/y runs of neighbouring tiles share cache lines: keep them on one XCD
  const uint32_t bid = xcd_order(blockIdx.x, gridDim.x);
  const int64_t line = bid / ntile;
  const int c0 = (int)(bid % ntile) * TL;
  const int64_t M = (int64_t)N1 * N2;
  const int64_t L = CIRC ? 2 * M : M;
  const int tid = threadIdx.x;
  const int cc = tid % (NT / T), t = tid / (NT / T);
  const bool act = cc < TL;

  const float2* B = ws + line * per_line + c0 + cc;
  float2 w[E];
#pragma unroll
  for (int e = 0; e < E; ++e) w[e] = act ? B[(size_t)(t + T * e) * N2] : czero();
  // outer gate values for the kept rows m1 = t + T e < NOUT, fetched before
  // the transform so their latency hides behind it
  const size_t gbase = (size_t)(line0 + line) * L + 2 * (size_t)(c0 + cc);
  float2 g[E];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int m1 = t + T * e;
    g[e] = (act && (CIRC || m1 < NOUT)) ? Gates<ACT>{}.g2(ld2(x2 + gbase + 2 * (size_t)m1 * N2)) : czero();
  }
  BlockFFT<N1, E, true>::run(w, t, ScrS<TLP>{tile + (act ? cc : 0)}, act, twl);
  if (act) {
    // unpack y[2m], y[2m+1] and gate
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int m1 = t + T * e;
      if (CIRC || m1 < NOUT)
        st2(y + gbase + 2 * (size_t)m1 * N2, make_float2(g[e].x * w[e].x, g[e].y * w[e].y));
    }
  }
}

struct FsLaunch {
  const FftConvArgs* a;
  float2* ws;
  int64_t line0;
  int nl;
  int N1, log2M;
  int64_t per;
  float scale;
  hipStream_t s;
};

template <int N1>
hipError_t cols_fwd(const FsLaunch& L) {
  constexpr int TL = ColCfg<N1>::TL;
  static_assert(ColCfgFwd<N1>::TL == TL, "the modal and forward column passes share the tiling");
  const FftConvArgs& a = *L.a;
  const int u_only = a.modal.M > 0;  // the kernel's columns come from fs_cols_modal
  const dim3 grid((unsigned)((int64_t)L.nl * (kN2 / TL) * (u_only ? 1 : 2)));
  if (u_only) {
    const dim3 kgrid((unsigned)((int64_t)L.nl * (kN2 / TL)));
    const size_t mbytes = (size_t)a.modal.M * (TL + ColCfg<N1>::T + 2) * sizeof(float2);
    if (a.circular)
      hipLaunchKernelGGL((fs_cols_modal<N1, true>), kgrid, dim3(512), mbytes, L.s, a.modal, L.ws, L.line0, kN2,
                         L.log2M, L.per, (int)a.C);
    else
      hipLaunchKernelGGL((fs_cols_modal<N1, false>), kgrid, dim3(512), mbytes, L.s, a.modal, L.ws, L.line0, kN2,
                         L.log2M, L.per, (int)a.C);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
#define HY_ARGS(TS) \
  (const TS*)a.x1, (const TS*)a.v, (const TS*)a.k, L.ws, L.line0, kN2, L.log2M, L.per, a.kC, a.act_in, (int)a.C, u_only
#define HY_LAUNCH(CI, TS, KC)                                                                                     \
  if (a.act) hipLaunchKernelGGL((fs_cols_fwd<N1, CI, TS, KC, true>), grid, dim3(ColCfgFwd<N1>::NT), 0, L.s, HY_ARGS(TS)); \
  else hipLaunchKernelGGL((fs_cols_fwd<N1, CI, TS, KC, false>), grid, dim3(ColCfgFwd<N1>::NT), 0, L.s, HY_ARGS(TS));
  if (a.centered) {
    if (a.bf16) { HY_LAUNCH(false, uint16_t, true) } else { HY_LAUNCH(false, float, true) }
  } else if (a.bf16) {
    if (a.circular) { HY_LAUNCH(true, uint16_t, false) } else { HY_LAUNCH(false, uint16_t, false) }
  } else {
    if (a.circular) { HY_LAUNCH(true, float, false) } else { HY_LAUNCH(false, float, false) }
  }
#undef HY_LAUNCH
#undef HY_ARGS
  return hipGetLastError();
}

template <int N1>
hipError_t cols_inv(const FsLaunch& L) {
  constexpr int TL = ColCfgFwd<N1>::TL;
  const dim3 grid((unsigned)((int64_t)L.nl * (kN2 / TL)));
  const FftConvArgs& a = *L.a;
#define HY_ARGS(TS) L.ws, (const TS*)a.x2, (TS*)a.y, L.line0, kN2, L.per
#define HY_LAUNCH(CI, TS)                                                                                  \
  if (a.act) hipLaunchKernelGGL((fs_cols_inv<N1, CI, TS, true>), grid, dim3(ColCfgFwd<N1>::NT), 0, L.s, HY_ARGS(TS)); \
  else hipLaunchKernelGGL((fs_cols_inv<N1, CI, TS, false>), grid, dim3(ColCfgFwd<N1>::NT), 0, L.s, HY_ARGS(TS));
  if (a.bf16) {
    if (a.circular) { HY_LAUNCH(true, uint16_t) } else { HY_LAUNCH(false, uint16_t) }
  } else {
    if (a.circular) { HY_LAUNCH(true, float) } else { HY_LAUNCH(false, float) }
  }
#undef HY_LAUNCH
#undef HY_ARGS
  return hipGetLastError();
}

#define HY_N1_SWITCH(N, FN, ARG)           \
  switch (N) {                             \
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

hipError_t d_cols_fwd(const FsLaunch& L) { HY_N1_SWITCH(L.N1, cols_fwd, L) }
hipError_t d_cols_inv(const FsLaunch& L) { HY_N1_SWITCH(L.N1, cols_inv, L) }

}  // namespace

bool fourstep_supported(const FftConvArgs& a) {
  if (a.ndim != 1) return false;
  const int64_t M = a.P[0] / 2;
  if (M % kN2 != 0) return false;
  const int64_t N1 = M / kN2;
  return N1 >= kMinN1 && N1 <= kMaxN1;
}

size_t fourstep_bytes_per_line(const FftConvArgs& a) {
  return (size_t)(a.P[0] / 2) * 2 * sizeof(float2);  // A_u and A_k
}

hipError_t launch_fourstep(const FftConvArgs& a, int64_t line0, int64_t nl, void* ws, hipStream_t s) {
  if (!fourstep_supported(a) || nl < 1 || line0 < 0 || line0 + nl > a.lines) return hipErrorInvalidValue;
  FsLaunch L;
  L.a = &a;
  L.ws = (float2*)ws;
  const int64_t M = a.P[0] / 2;
  L.N1 = (int)(M / kN2);
  L.log2M = ilog2_rt(M);
  L.per = 2 * M;
  L.scale = (float)(1.0 / (4.0 * (double)a.P[0]));
  L.s = s;
  L.line0 = line0;
  L.nl = (int)nl;
  hipError_t e;
  if ((e = d_cols_fwd(L)) != hipSuccess) return e;
  const dim3 grid((unsigned)((int64_t)L.nl * (L.N1 / 2 + 1)));
  if (a.circular)
    hipLaunchKernelGGL((fs_core<true>), grid, dim3(512), 0, s, L.ws, a.D, (int)a.bf16, line0, (int)a.C, L.N1,
                       L.log2M, L.per, L.scale);
  else
    hipLaunchKernelGGL((fs_core<false>), grid, dim3(512), 0, s, L.ws, a.D, (int)a.bf16, line0, (int)a.C, L.N1,
                       L.log2M, L.per, L.scale);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  return d_cols_inv(L);
}

}  // namespace hyenand
