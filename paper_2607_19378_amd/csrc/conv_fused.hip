// Single-pass kernels: the whole padded problem of one (b, c) line stays in
// LDS, so HBM sees only the five tensors (x1, v, k read; x2 read; y written).
//
//  * conv1d_fused<P>: 1D line, transform length P <= 16384.
//  * conv2d_fused<P0, P1>: 2D image whose half spectra fit in LDS.
//
// Real-to-complex transforms: a real line of length P is read as the complex
// line of its even/odd sample pairs (length P/2), transformed, and untangled
// with the mirror bin (r2c_pair).  u = x1 v and k are transformed separately,
// so each spectrum keeps its own relative accuracy.  The product
// U (K + D) is Hermitian; the inverse runs on the half spectrum: in 1D as a
// length-P/2 complex transform of the even/odd packed output (c2r_pair), in
// 2D as column transforms of the P1/2+1 half-spectrum columns followed by row
// transforms that carry two real output rows each (row a in the real part,
// row b in the imaginary part).  Zero padding is never stored: inputs beyond L
// are compile-time zeros of the first pass, and outputs beyond the crop are
// never written.
#include <type_traits>

#include "kernels.hpp"

namespace hyenand {

// ---------------------------------------------------------------------------
// 1D
// ---------------------------------------------------------------------------
constexpr int fused1d_nt(int P) {
  return imax(64, imax(2 * ((P / 2) / imin(16, P / 2)), (P / 2) / imin(8, P / 2)));
}

template <int P, bool CIRC, typename TS>
struct Fused1D {
  static constexpr int L = CIRC ? P : P / 2;
  static constexpr int M = P / 2;          // complex length of the packed real line
  static constexpr int MNZ = (L + 1) / 2;  // nonzero packed samples
  static constexpr int EF = imin(16, M);   // forward: two lines (u, k)
  static constexpr int TF = M / EF;
  static constexpr int EI = imin(8, M);    // inverse: one line
  static constexpr int TI = M / EI;
  static constexpr int NT = fused1d_nt(P);
  static_assert(NT >= 2 * TF && NT >= TI, "threads");
  static constexpr int LDSN = pad16_size(M);
};

// KC: k is the centered kernel of 2L - 1 points (linear transform grid); its
// packed line has no zero half.
// ACT: the HyenaND operator's gates (Gates).
template <int P, bool CIRC, typename TS, bool KC = false, bool ACT = false>
__global__ void __launch_bounds__(fused1d_nt(P))
    conv1d_fused(const TS* __restrict__ x1, const TS* __restrict__ x2, const TS* __restrict__ v,
                 const TS* __restrict__ k, const TS* __restrict__ Dp, TS* __restrict__ y, int C, int kC,
                 ActIn ain) {
  static_assert(!(KC && CIRC), "centered kernels use the linear transform grid");
  using F = Fused1D<P, CIRC, TS>;
  constexpr int L = F::L, M = F::M, MNZ = F::MNZ, NT = F::NT;
  __shared__ float2 Ub[F::LDSN];
  __shared__ float2 Kb[F::LDSN];
  // pass twiddles in LDS where they fit beside the two lines
  using TwF = PassTw<M, F::EF>;
  using TwI = PassTw<M, F::EI>;
  constexpr bool kTwl = (2 * F::LDSN + TwF::kCount + TwI::kCount) * 8 <= 150 * 1024;
  __shared__ float2 twf[kTwl ? imax(1, TwF::kCount) : 1];
  __shared__ float2 twi[kTwl ? imax(1, TwI::kCount) : 1];
  const int line = blockIdx.x;
  const int c = line % C;
  const size_t base = (size_t)line * L;
  const size_t kbase = (size_t)k_line(line, kC) * L;
  const int tid = threadIdx.x;
  const Gates<ACT> G = line_gates<ACT, TS>(ain, line, C);
  if constexpr (kTwl) {
    TwF::fill(twf, tid, NT);
    TwI::fill(twi, tid, NT);
  }

  // stage the even/odd packed real lines u = x1 v and k
  if constexpr (KC) {
    static_assert(L >= 2, "centered lines have two or more points");
    batched_copy<MNZ, NT, 8>(
        tid,
        [&](int m) { return G.u2(ld2(x1 + base + 2 * m), ld2(v + base + 2 * m), 2 * m); },
        [&](int m, float2 z) { Ub[m + (m >> 4)] = z; });
    // grid points 2m, 2m + 1 of k from the 2L - 1 centered points
    const TS* kl = k + (size_t)k_line(line, kC) * (2 * L - 1);
    batched_copy<M, NT, 8>(
        tid,
        [&](int m) {
          const int j0 = centered_index(2 * m, L, P), j1 = centered_index(2 * m + 1, L, P);
          return make_float2(j0 >= 0 ? ld1(kl + j0) : 0.f, j1 >= 0 ? ld1(kl + j1) : 0.f);
        },
        [&](int m, float2 z) { Kb[m + (m >> 4)] = z; });
  } else if constexpr (L >= 2) {
    batched_copy<MNZ, NT, 8>(
        tid,
        [&](int m) {
          const float2 u = G.u2(ld2(x1 + base + 2 * m), ld2(v + base + 2 * m), 2 * m);
          const float2 kk = ld2(k + kbase + 2 * m);
          return make_float4(u.x, u.y, kk.x, kk.y);
        },
        [&](int m, float4 z) {
          Ub[m + (m >> 4)] = make_float2(z.x, z.y);
          Kb[m + (m >> 4)] = make_float2(z.z, z.w);
        });
  } else if (tid == 0) {  // a single sample
    Ub[0] = make_float2(G.u1(ld1(x1 + base), ld1(v + base), 0), 0.f);
    Kb[0] = make_float2(ld1(k + kbase), 0.f);
  }
  // outer gate values of the output pairs this lane stores at the end, as
  // raw storage words, fetched now so that their latency hides behind the
  // transforms (a short line is one launch latency, nothing to hide it in)
  constexpr bool kGpre = L >= 2;
  typename Raw2<TS>::type gpre[kGpre ? F::EI : 1];
  if constexpr (kGpre) {
    if (tid < F::TI) {
#pragma unroll
      for (int e = 0; e < F::EI; ++e) {
        const int n = 2 * (tid + F::TI * e);
        if (n < L) gpre[e] = ld2_raw(x2 + base + n);
      }
    }
  }
  __syncthreads();

  // forward half-length transforms of both packed lines
  {
    constexpr int E = F::EF, T = F::TF;
    const int which = tid / T, t = tid % T;
    const bool act = which < 2;
    float2* buf = which == 0 ? Ub : Kb;
    const ScrPad16 scr{buf};
    const int nz = (KC && which == 1) ? M : MNZ;  // a centered k line is full
    float2 w[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int m = t + T * e;
      w[e] = (act && m < nz) ? *scr(m) : czero();
    }
    if constexpr (kTwl) BlockFFT<M, E, false>::run(w, t, scr, act, twf);
    else BlockFFT<M, E, false>::run(w, t, scr, act);
    if (act) {
#pragma unroll
      for (int e = 0; e < E; ++e) *scr(t + T * e) = w[e];
    }
  }
  __syncthreads();

  // untangle both spectra, gated product with the folded shortcut, and pack
  // the Hermitian product for a half-length inverse:
  //   bin g needs U, K at g and M-g, which come from packed bins g and M-g.
  {
    constexpr int E = F::EI, T = F::TI;
    const float twoD = 2.f * ld1(Dp + c);
    const float scale = 1.f / (4.f * (float)P);
    const ScrPad16 su{Ub}, sk{Kb};
    const int t = tid;
    const bool act = t < T;
    float2 w[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int g = t + T * e;
      w[e] = czero();
      if (act) {
        const int gm = (M - g) & (M - 1);
        const float2 tw = twiddle<ilog2(P), false>(g);
        float2 Ug, Umg, Kg, Kmg;
        r2c_pair(*su(g), *su(gm), tw, Ug, Umg);
        r2c_pair(*sk(g), *sk(gm), tw, Kg, Kmg);
        const float2 Yg = gated_product(Ug, Kg, twoD);
        const float2 Ymg = gated_product(Umg, Kmg, twoD);
        w[e] = c_scale(c2r_pair(Yg, Ymg, tw), scale);
      }
    }
    if constexpr (T == 1) __syncthreads();
    if constexpr (kTwl) BlockFFT<M, E, true>::run(w, t, su, act, twi);
    else BlockFFT<M, E, true>::run(w, t, su, act);
    if (act) {
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const int n = 2 * (t + T * e);
        if constexpr (kGpre) {  // L even: n < L holds both outputs of the pair
          if (n < L) {
            const float2 g = G.g2(widen2(gpre[e]));
            st2(y + base + n, make_float2(g.x * w[e].x, g.y * w[e].y));
          }
        } else {
          if (n < L) st1(y + base + n, G.g1(ld1(x2 + base + n)) * w[e].x);
          if (n + 1 < L) st1(y + base + n + 1, G.g1(ld1(x2 + base + n + 1)) * w[e].y);
        }
      }
    }
  }
}

template <int P, bool CIRC, typename TS, bool KC = false>
static hipError_t launch_1d_fused_t(const FftConvArgs& a, hipStream_t s) {
  using F = Fused1D<P, CIRC, TS>;
  if (a.act)
    hipLaunchKernelGGL((conv1d_fused<P, CIRC, TS, KC, true>), dim3((unsigned)a.lines), dim3(F::NT), 0, s,
                       (const TS*)a.x1, (const TS*)a.x2, (const TS*)a.v, (const TS*)a.k, (const TS*)a.D, (TS*)a.y,
                       (int)a.C, a.kC, a.act_in);
  else
    hipLaunchKernelGGL((conv1d_fused<P, CIRC, TS, KC, false>), dim3((unsigned)a.lines), dim3(F::NT), 0, s,
                       (const TS*)a.x1, (const TS*)a.x2, (const TS*)a.v, (const TS*)a.k, (const TS*)a.D, (TS*)a.y,
                       (int)a.C, a.kC, a.act_in);
  return hipGetLastError();
}

template <int P>
static hipError_t launch_1d_fused_p(const FftConvArgs& a, hipStream_t s) {
  if constexpr (P >= 4) {
    if (a.centered)
      return a.bf16 ? launch_1d_fused_t<P, false, uint16_t, true>(a, s) : launch_1d_fused_t<P, false, float, true>(a, s);
  } else {
    if (a.centered) return hipErrorInvalidValue;
  }
  if (a.circular) {
    return a.bf16 ? launch_1d_fused_t<P, true, uint16_t>(a, s) : launch_1d_fused_t<P, true, float>(a, s);
  }
  return a.bf16 ? launch_1d_fused_t<P, false, uint16_t>(a, s) : launch_1d_fused_t<P, false, float>(a, s);
}

bool fused1d_supported(int64_t P) { return P >= 2 && P <= 16384 && (P & (P - 1)) == 0; }

hipError_t launch_fused1d(const FftConvArgs& a, hipStream_t s) {
  switch (a.P[0]) {
    case 2: return launch_1d_fused_p<2>(a, s);
    case 4: return launch_1d_fused_p<4>(a, s);
    case 8: return launch_1d_fused_p<8>(a, s);
    case 16: return launch_1d_fused_p<16>(a, s);
    case 32: return launch_1d_fused_p<32>(a, s);
    case 64: return launch_1d_fused_p<64>(a, s);
    case 128: return launch_1d_fused_p<128>(a, s);
    case 256: return launch_1d_fused_p<256>(a, s);
    case 512: return launch_1d_fused_p<512>(a, s);
    case 1024: return launch_1d_fused_p<1024>(a, s);
    case 2048: return launch_1d_fused_p<2048>(a, s);
    case 4096: return launch_1d_fused_p<4096>(a, s);
    case 8192: return launch_1d_fused_p<8192>(a, s);
    case 16384: return launch_1d_fused_p<16384>(a, s);
    default: return hipErrorInvalidValue;
  }
}

// ---------------------------------------------------------------------------
// 2D
// ---------------------------------------------------------------------------
// LDS holds the half spectra of the L0 nonzero rows only (linear mode: half
// the padded rows), so two workgroups fit on a CU for the 128 x 128
// transform.  Column transforms exchange through the column's own U and K
// slots (2 L0 >= P0 entries).  Columns 0 and P1/2 of a real row transform are
// real, so they travel together as one complex column (a + i b) and are
// separated with the mirror bin; M1 = P1/2 column groups cover all M1 + 1
// columns.
template <int P0, int P1, bool CIRC, typename TS>
struct Fused2D {
  static constexpr int L0 = CIRC ? P0 : P0 / 2;
  static constexpr int L1 = CIRC ? P1 : P1 / 2;
  static constexpr int M1 = P1 / 2;          // packed complex row length
  static constexpr int MNZ = (L1 + 1) / 2;   // nonzero packed samples per row
  static constexpr int RP = M1 + 1;          // LDS row pitch (half spectrum + Nyquist)
  static constexpr int NT = 512;
  // forward row transforms: 2 L0 lines (u rows, k rows) of M1 points
  static constexpr int ER = imin(16, M1);
  static constexpr int TR = M1 / ER;
  static constexpr int LR = NT / TR;         // lines per round
  // column transforms (length P0): M1 groups
  static constexpr int EC = imin(16, P0);
  static constexpr int TC = P0 / EC;
  static constexpr int CR = NT / TC;         // column groups per round
  // inverse row transforms: one real row each, as the length-M1 transform
  // of its even/odd output pairs
  static constexpr int EI = imin(8, M1);
  static constexpr int TI = M1 / EI;
  static constexpr int RI = NT / TI;         // rows per round
  static_assert(2 * L0 >= P0, "column scratch");
};

// KH selects how the kernel's spectrum is obtained when one kernel serves a
// channel in every sample (kC = C):
//   0: each image transforms its own k (every call shape);
//   1: one workgroup per channel transforms k[c] and writes its column-pass
//      spectrum, khat[c][n][g] (n < P0 along axis 0, g < P1/2 the column
//      group, group 0 the DC + i Nyquist column), and stops there;
//   2: each image reads that spectrum instead of transforming k.
// Modes 1 and 2 together run the same arithmetic on k as mode 0, once per
// channel instead of once per image.
template <int P0, int P1, bool CIRC, typename TS, bool ACT = false, int KH = 0>
__global__ void __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(4)))
    conv2d_fused(const TS* __restrict__ x1, const TS* __restrict__ x2, const TS* __restrict__ v,
                 const TS* __restrict__ k, const TS* __restrict__ Dp, TS* __restrict__ y, int C, int kC,
                 ActIn ain, float2* __restrict__ khat) {
  static_assert(KH >= 0 && KH <= 2 && !(ACT && KH), "kernel spectrum mode");
  using F = Fused2D<P0, P1, CIRC, TS>;
  constexpr int L0 = F::L0, L1 = F::L1, M1 = F::M1, MNZ = F::MNZ, RP = F::RP, NT = F::NT;
  // U half spectrum rows [0, L0), then K's: column c of both is one stride-RP
  // line of 2 L0 >= P0 slots, the exchange scratch of that column's transforms
  __shared__ float2 UK[2 * L0 * RP];
  __shared__ float2 NQ[2][P0];  // column group 0's U and K spectra (DC + i Nyquist)
  float2* const Uh = UK;
  float2* const Kh = UK + L0 * RP;
  int img = blockIdx.x;
  if constexpr (KH == 2) {
    // Workgroup j runs on XCD j mod 8.  Renumber so that the B images of a
    // channel take consecutive slots j, j + 8, ... of one XCD: its spectrum
    // then comes into that XCD's L2 once for all of them.
    if ((C & 7) == 0) {
      const int nb = (int)gridDim.x / C, x = img & 7, q = img >> 3;
      img = (q % nb) * C + (q / nb) * 8 + x;
    }
  }
  const int c = img % C;
  const size_t base = (size_t)img * L0 * L1;
  const size_t kbase = (size_t)k_line(img, kC) * L0 * L1;
  const int tid = threadIdx.x;
  const Gates<ACT> G = line_gates<ACT, TS>(ain, img, C);

  // The normalisation 1 / (4 P0 P1) of the two unnormalised inverses and of
  // the doubled R2C outputs is a power of two: it is applied, exactly, to k
  // and D on the way in.
  constexpr float scale = 1.f / (4.f * (float)P0 * (float)P1);

  // 0. stage the real rows of u = x1 v and k (coalesced along rows); row r of
  //    Uh holds the even/odd packed line u[r][2m] + i u[r][2m+1].
  // 1. forward row transforms (lanes run across rows), then untangle each row
  constexpr int NPS = L0 * L1 / 2, JS = (NPS + NT - 1) / NT;
  constexpr int ES = imin(8, M1), TRS = M1 / ES;
  // split staging: all loads issued at once, k's rows transformed while x1
  // and v are still arriving (where the loads fit in a few registers and one
  // round of 8-point lanes covers the L0 rows of a signal)
  constexpr bool kSplit = JS <= 4 && TRS * L0 == NT;
  if constexpr (kSplit) {
    float2 kr[JS], ar[JS], br[JS];
    if constexpr (KH != 2) {
#pragma unroll
      for (int j = 0; j < JS; ++j) {
        const int i = tid + NT * j;
        if (NPS % NT == 0 || i < NPS) kr[j] = ld2(k + kbase + 2 * i);
      }
    }
    if constexpr (KH != 1) {
#pragma unroll
      for (int j = 0; j < JS; ++j) {
        const int i = tid + NT * j;
        if (NPS % NT == 0 || i < NPS) {
          ar[j] = ld2(x1 + base + 2 * i);
          br[j] = ld2(v + base + 2 * i);
        }
      }
    }
    if constexpr (KH != 2) {
#pragma unroll
      for (int j = 0; j < JS; ++j) {
        const int i = tid + NT * j;
        if (NPS % NT == 0 || i < NPS) {
          const int r = i / (L1 / 2), m = i - r * (L1 / 2);
          Kh[r * RP + m] = make_float2(kr[j].x * scale, kr[j].y * scale);
        }
      }
      __syncthreads();
    }
    using Map = LaneMap<TRS, NT>;
    static_assert(Map::kLines == L0, "one round per signal");
    const int l = Map::line(tid), t = Map::t(tid);
    auto rows = [&](float2* rowp) {
      float2 w[ES];
#pragma unroll
      for (int e = 0; e < ES; ++e) {
        const int m = t + TRS * e;
        w[e] = (CIRC || m < MNZ) ? rowp[m] : czero();
      }
      BlockFFT<M1, ES, false>::run(w, t, ScrS<1>{rowp}, true);
#pragma unroll
      for (int e = 0; e < ES; ++e) rowp[t + TRS * e] = w[e];
    };
    if constexpr (KH != 2) rows(Kh + l * RP);
    if constexpr (KH != 1) {
#pragma unroll
      for (int j = 0; j < JS; ++j) {
        const int i = tid + NT * j;
        if (NPS % NT == 0 || i < NPS) {
          const int r = i / (L1 / 2), m = i - r * (L1 / 2);
          Uh[r * RP + m] = G.u2(ar[j], br[j], 2 * i);
        }
      }
      __syncthreads();
      rows(Uh + l * RP);
    }
  } else {
    if constexpr (KH == 0) {
      batched_copy<L0 * L1 / 2, NT, 8>(
          tid,
          [&](int i) {
            const float2 u = G.u2(ld2(x1 + base + 2 * i), ld2(v + base + 2 * i), 2 * i);
            const float2 kk = ld2(k + kbase + 2 * i);
            return make_float4(u.x, u.y, kk.x * scale, kk.y * scale);
          },
          [&](int i, float4 z) {
            const int r = i / (L1 / 2), m = i - r * (L1 / 2);
            Uh[r * RP + m] = make_float2(z.x, z.y);
            Kh[r * RP + m] = make_float2(z.z, z.w);
          });
    } else {
      batched_copy<L0 * L1 / 2, NT, 8>(
          tid,
          [&](int i) {
            if constexpr (KH == 1) {
              const float2 kk = ld2(k + kbase + 2 * i);
              return make_float2(kk.x * scale, kk.y * scale);
            } else {
              return G.u2(ld2(x1 + base + 2 * i), ld2(v + base + 2 * i), 2 * i);
            }
          },
          [&](int i, float2 z) {
            const int r = i / (L1 / 2), m = i - r * (L1 / 2);
            (KH == 1 ? Kh : Uh)[r * RP + m] = z;
          });
    }
    __syncthreads();
    {
      // rows of U then K (KH = 0), or of the one signal this mode transforms
      constexpr int NL = KH == 0 ? 2 * L0 : L0;
      float2* const R0 = KH == 1 ? Kh : Uh;
      constexpr int E = F::ER, T = F::TR, LR = F::LR;
      for (int l0 = 0; l0 < NL; l0 += LR) {
        using Map = LaneMap<T, NT>;
        static_assert(Map::kLines == LR, "lines per round");
        const int l = l0 + Map::line(tid), t = Map::t(tid);
        const bool act = NL % LR == 0 || l < NL;  // all lanes busy when rounds are full
        float2* row = R0 + (act ? l : 0) * RP;
        float2 w[E];
#pragma unroll
        for (int e = 0; e < E; ++e) {
          const int m = t + T * e;
          w[e] = (act && (CIRC || m < MNZ)) ? row[m] : czero();
        }
        BlockFFT<M1, E, false>::run(w, t, ScrS<1>{row}, act);
        if (act) {
#pragma unroll
          for (int e = 0; e < E; ++e) row[t + T * e] = w[e];
        }
      }
    }
  }
  __syncthreads();
  // The real rows' spectra come out of the packed row transforms Z by
  // untangling (r2c_pair: bin g from Z[g] and Z[M1 - g]).  When one round of
  // column groups covers every column, each column lane untangles the bins it
  // loads (the bin and its mirror are both read before the first exchange
  // barrier of the column transforms, which is the first write to either
  // slot), so no pass rewrites the rows; in linear mode it then untangles
  // only the L0 nonzero rows.  Otherwise a pass over the rows does it first.
  constexpr bool kColUntangle = M1 <= F::CR;
  if constexpr (!kColUntangle) {
    // Untangling, in place: item (row l, g) for 0 < g < M1/2 owns bins g and
    // M1 - g; bins 0 and M1/2 are their own mirrors and share the item g = 0
    // of their row.  The DC and Nyquist bins of a real row are real: slot 0
    // keeps both, as DC + i Nyquist (column group 0 below).  Rows of U and K
    // are contiguous (Kh = Uh + L0 RP); with 2 L0 a multiple of 64 every
    // wavefront shares one g, so its twiddle is a scalar.
    constexpr int NR = KH == 0 ? 2 * L0 : L0, NG = imax(1, M1 / 2);
    float2* const R0 = KH == 1 ? Kh : Uh;
    for (int it = tid; it < NR * NG; it += NT) {
      const int l = it % NR;
      const int g = NR % 64 == 0 ? __builtin_amdgcn_readfirstlane(it / NR) : it / NR;
      float2* row = R0 + l * RP;
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
    __syncthreads();
  }

  // 2. column groups: forward transforms of U and K, gated product with the
  //    folded shortcut, inverse transform; keep rows < L0.  Group 0 is the
  //    complex column DC + i Nyquist of the two real columns 0 and M1.
  {
    constexpr int E = F::EC, T = F::TC, CR = F::CR;
    const float twoD = KH == 1 ? 0.f : 2.f * scale * ld1(Dp + c);
    const float2* const kh = khat + (size_t)c * P0 * M1;  // modes 1 and 2
    for (int c0 = 0; c0 < M1; c0 += CR) {
      using Map = LaneMap<T, NT>;
      static_assert(Map::kLines == CR, "groups per round");
      const int grp = c0 + Map::line(tid), t = Map::t(tid);
      const bool act = M1 % CR == 0 || grp < M1;
      const bool nyq = act && grp == 0;
      const int col = act ? grp : 0;
      const int mcol = (M1 - col) & (M1 - 1);          // mirror bin (0 for 0)
      const float2 twc = twiddle<ilog2(P1), false>(col);  // (1, 0) for column 0
      // bin col of row n: untangled from the packed row spectrum, or as stored
      auto bin = [&](const float2* R, int n) -> float2 {
        if constexpr (kColUntangle) return untangle_bin(R + n * RP, col, mcol, twc);
        else return R[n * RP + col];
      };
      float2 wu[E], wk[E];
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const int n = t + T * e;
        const bool nz = act && (CIRC || n < L0);
        if constexpr (KH != 1) wu[e] = nz ? bin(Uh, n) : czero();
        if constexpr (KH == 2) wk[e] = act ? kh[n * M1 + col] : czero();
        else wk[e] = nz ? bin(Kh, n) : czero();
      }
      const ScrS<RP> su{UK + col};
      if constexpr (KH != 1) BlockFFT<P0, E, false>::run(wu, t, su, act);
      if constexpr (KH != 2) BlockFFT<P0, E, false>::run(wk, t, su, act);
      if constexpr (KH == 1) {
        if (act) {
#pragma unroll
          for (int e = 0; e < E; ++e) khat[(size_t)c * P0 * M1 + (t + T * e) * M1 + col] = wk[e];
        }
        continue;
      }
      // Group 0 holds A + i B with A, B the spectra of the real columns 0
      // and M1: A = (Z[f] + conj Z[-f]) / 2, B = -i (Z[f] - conj Z[-f]) / 2
      // need the mirror bin, so its spectra go through LDS (slots of their
      // own, outside every group's exchange scratch, so no barrier precedes
      // the writes) and the bin pairs (f, P0 - f) are multiplied by lanes of
      // the first two wavefronts; the other groups multiply in registers.
      const ScrS<1> u0{NQ[0]};
      const ScrS<1> k0{NQ[1]};
      if (nyq) {
#pragma unroll
        for (int e = 0; e < E; ++e) {
          *u0(t + T * e) = wu[e];
          *k0(t + T * e) = wk[e];
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
        // Y = Ya + i Yb; both products are Hermitian, so at -f it is conj Ya + i conj Yb
        *u0(f) = make_float2(ya.x - yb.y, ya.y + yb.x);
        if (fm != f) *u0(fm) = make_float2(ya.x + yb.y, yb.x - ya.y);
      }
      __syncthreads();
      if (nyq) {
#pragma unroll
        for (int e = 0; e < E; ++e) wu[e] = *u0(t + T * e);
      } else {
#pragma unroll
        for (int e = 0; e < E; ++e) wu[e] = gated_product(wu[e], wk[e], twoD);
      }
      BlockFFT<P0, E, true>::run(wu, t, su, act);
      __syncthreads();  // scratch reads of the last exchange are done
      if (act) {
#pragma unroll
        for (int e = 0; e < E; ++e) {
          const int n = t + T * e;
          if (CIRC || n < L0) Uh[n * RP + col] = wu[e];
        }
      }
    }
  }
  if constexpr (KH == 1) return;
  __syncthreads();

  // outer gate values of the row pairs this lane stores, fetched before the
  // inverse rows so that their latency hides behind them (when they take
  // few registers)
  constexpr int NP = L0 * L1 / 2, JX = (NP + NT - 1) / NT;
  constexpr bool kPre = JX <= 4;
  float2 gpre[kPre ? JX : 1];
  if constexpr (kPre) {
#pragma unroll
    for (int j = 0; j < JX; ++j) {
      const int i = tid + NT * j;
      if (NP % NT == 0 || i < NP) gpre[j] = G.g2(ld2(x2 + base + 2 * i));
    }
  }

  // 3. inverse row transforms: c2r_pair turns row r's half spectrum (slot 0
  //    holding DC + i Nyquist) into the length-M1 transform of its even/odd
  //    output pairs; the inverse leaves y[r][2m] + i y[r][2m+1] in slot m.
  {
    constexpr int E = F::EI, T = F::TI, RI = F::RI;
    for (int r0 = 0; r0 < L0; r0 += RI) {
      using Map = LaneMap<T, NT>;
      static_assert(Map::kLines == RI, "rows per round");
      const int r = r0 + Map::line(tid), t = Map::t(tid);
      const bool act = L0 % RI == 0 || r < L0;
      float2* row = Uh + (act ? r : 0) * RP;
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

  // 4. outer gate and store (coalesced along rows)
  if constexpr (kPre) {
#pragma unroll
    for (int j = 0; j < JX; ++j) {
      const int i = tid + NT * j;
      if (NP % NT == 0 || i < NP) {
        const int r = i / (L1 / 2), m = i - r * (L1 / 2);
        const float2 q = Uh[r * RP + m], g = gpre[j];
        st2(y + base + 2 * i, make_float2(g.x * q.x, g.y * q.y));
      }
    }
  } else {
    batched_copy<L0 * L1 / 2, NT, 8>(
        tid, [&](int i) { return G.g2(ld2(x2 + base + 2 * i)); },
        [&](int i, float2 g) {
          const int r = i / (L1 / 2), m = i - r * (L1 / 2);
          const float2 q = Uh[r * RP + m];
          st2(y + base + 2 * i, make_float2(g.x * q.x, g.y * q.y));
        });
  }
}

// Centered kernel, single pass: the K half spectrum fills all P0 rows, so U
// does not sit beside it in LDS.  U's rows are transformed first in the same
// region, and each lane keeps the U values of its column group (the nonzero
// rows n < L0 of its column transform) in registers while K's rows take the
// region: one P0 x (P1/2 + 1) region per image, as in the linear kernel, and
// two workgroups per CU for the 128 x 128 grid.
template <int P0, int P1, typename TS, bool ACT = false>
__global__ void __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(4)))
    conv2d_fused_kc(const TS* __restrict__ x1, const TS* __restrict__ x2, const TS* __restrict__ v,
                    const TS* __restrict__ k, const TS* __restrict__ Dp, TS* __restrict__ y, int C, int kC,
                    ActIn ain) {
  using F = Fused2D<P0, P1, false, TS>;
  constexpr int L0 = F::L0, L1 = F::L1, M1 = F::M1, MNZ = F::MNZ, RP = F::RP, NT = F::NT;
  __shared__ float2 S[P0 * RP];  // U rows [0, L0), then K rows [0, P0); column exchange scratch
  __shared__ float2 NQ[2][P0];   // column group 0's U and K spectra (DC + i Nyquist)
  const int img = blockIdx.x;
  const int c = img % C;
  const size_t base = (size_t)img * L0 * L1;
  const TS* kl = k + (size_t)k_line(img, kC) * (2 * L0 - 1) * (2 * L1 - 1);
  const int tid = threadIdx.x;
  const Gates<ACT> G = line_gates<ACT, TS>(ain, img, C);
  constexpr float scale = 1.f / (4.f * (float)P0 * (float)P1);

  // row transforms of NR rows in place (the first nz packed samples of each
  // row nonzero), then untangling with DC + i Nyquist in slot 0
  auto rows_r2c = [&](auto nr_c, int nz) {
    constexpr int NR = decltype(nr_c)::value;
    constexpr int E = F::ER, T = F::TR, LR = F::LR;
    for (int l0 = 0; l0 < NR; l0 += LR) {
      using Map = LaneMap<T, NT>;
      const int l = l0 + Map::line(tid), t = Map::t(tid);
      const bool act = NR % LR == 0 || l < NR;
      float2* row = S + (act ? l : 0) * RP;
      float2 w[E];
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const int m = t + T * e;
        w[e] = (act && m < nz) ? row[m] : czero();
      }
      BlockFFT<M1, E, false>::run(w, t, ScrS<1>{row}, act);
      if (act) {
#pragma unroll
        for (int e = 0; e < E; ++e) row[t + T * e] = w[e];
      }
    }
    __syncthreads();
    constexpr int NG = imax(1, M1 / 2);
    for (int it = tid; it < NR * NG; it += NT) {
      const int l = it % NR;
      const int g = NR % 64 == 0 ? __builtin_amdgcn_readfirstlane(it / NR) : it / NR;
      float2* row = S + l * RP;
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
    __syncthreads();
  };

  // 0-1. u = x1 v rows, their transforms
  batched_copy<L0 * L1 / 2, NT, 8>(
      tid, [&](int i) { return G.u2(ld2(x1 + base + 2 * i), ld2(v + base + 2 * i), 2 * i); },
      [&](int i, float2 z) {
        const int r = i / (L1 / 2), m = i - r * (L1 / 2);
        S[r * RP + m] = z;
      });
  __syncthreads();
  rows_r2c(std::integral_constant<int, L0>{}, MNZ);

  // 2. each lane keeps the U values of its column transform (rows n < L0)
  constexpr int E = F::EC, T = F::TC, CR = F::CR;
  static_assert(M1 <= CR, "one round of column groups");
  static_assert(L0 % T == 0, "the nonzero rows are the first points of every lane");
  constexpr int EU = L0 / T;  // nonzero points per lane
  using Map = LaneMap<T, NT>;
  const int grp = Map::line(tid), t = Map::t(tid);
  const bool act = M1 % CR == 0 || grp < M1;
  const bool nyq = act && grp == 0;
  const int col = act ? grp : 0;
  float2 uh[EU];
#pragma unroll
  for (int e = 0; e < EU; ++e) uh[e] = act ? S[(t + T * e) * RP + col] : czero();
  __syncthreads();

  // 3. K grid rows from the centered points, their transforms (full rows)
  batched_copy<P0 * M1, NT, 8>(
      tid,
      [&](int i) {
        const int g0 = i / M1, m = i - g0 * M1;
        const int j0 = centered_index(g0, L0, P0);
        const int ja = centered_index(2 * m, L1, P1), jb = centered_index(2 * m + 1, L1, P1);
        const TS* kr = kl + (size_t)(j0 >= 0 ? j0 : 0) * (2 * L1 - 1);
        return make_float2((j0 >= 0 && ja >= 0) ? ld1(kr + ja) * scale : 0.f,
                           (j0 >= 0 && jb >= 0) ? ld1(kr + jb) * scale : 0.f);
      },
      [&](int i, float2 z) {
        const int g0 = i / M1, m = i - g0 * M1;
        S[g0 * RP + m] = z;
      });
  __syncthreads();
  rows_r2c(std::integral_constant<int, P0>{}, M1);

  // 4. column groups: forward U (from registers) and K, product with the
  //    folded shortcut, inverse; keep rows < L0.  Group 0 is the complex
  //    column DC + i Nyquist, multiplied through LDS as in the linear kernel.
  {
    const float twoD = 2.f * scale * ld1(Dp + c);
    float2 wu[E], wk[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
      wu[e] = e < EU ? uh[e] : czero();
      wk[e] = act ? S[(t + T * e) * RP + col] : czero();
    }
    const ScrS<RP> su{S + col};
    BlockFFT<P0, E, false>::run(wu, t, su, act);
    BlockFFT<P0, E, false>::run(wk, t, su, act);
    // group 0's spectra go through slots of their own, outside every
    // group's exchange scratch: no barrier precedes the writes
    const ScrS<1> u0{NQ[0]};
    const ScrS<1> k0{NQ[1]};
    if (nyq) {
#pragma unroll
      for (int e = 0; e < E; ++e) {
        *u0(t + T * e) = wu[e];
        *k0(t + T * e) = wk[e];
      }
    }
    __syncthreads();
    if (tid <= P0 / 2) {
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
      for (int e = 0; e < E; ++e) wu[e] = *u0(t + T * e);
    } else {
#pragma unroll
      for (int e = 0; e < E; ++e) wu[e] = gated_product(wu[e], wk[e], twoD);
    }
    BlockFFT<P0, E, true>::run(wu, t, su, act);
    __syncthreads();  // scratch reads of the last exchange are done
    if (act) {
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const int n = t + T * e;
        if (n < L0) S[n * RP + col] = wu[e];
      }
    }
  }
  __syncthreads();

  // outer gate values of the row pairs this lane stores, fetched before the
  // inverse rows so that their latency hides behind them (when they take
  // few registers)
  constexpr int NP = L0 * L1 / 2, JX = (NP + NT - 1) / NT;
  constexpr bool kPre = JX <= 4;
  float2 gpre[kPre ? JX : 1];
  if constexpr (kPre) {
#pragma unroll
    for (int j = 0; j < JX; ++j) {
      const int i = tid + NT * j;
      if (NP % NT == 0 || i < NP) gpre[j] = G.g2(ld2(x2 + base + 2 * i));
    }
  }

  // 5. inverse row transforms (two real output values per complex point)
  {
    constexpr int EI = F::EI, TI = F::TI, RI = F::RI;
    for (int r0 = 0; r0 < L0; r0 += RI) {
      using MapI = LaneMap<TI, NT>;
      const int r = r0 + MapI::line(tid), ti = MapI::t(tid);
      const bool acti = L0 % RI == 0 || r < L0;
      float2* row = S + (acti ? r : 0) * RP;
      float2 w[EI];
#pragma unroll
      for (int e = 0; e < EI; ++e) {
        const int g = ti + TI * e;
        float2 Yg, Ym;
        if (g == 0) {
          const float2 s0 = row[0];
          Yg = make_float2(s0.x, 0.f);
          Ym = make_float2(s0.y, 0.f);
        } else {
          Yg = row[g];
          Ym = row[M1 - g];
        }
        w[e] = acti ? c2r_pair(Yg, Ym, twiddle<ilog2(P1), false>(g)) : czero();
      }
      BlockFFT<M1, EI, true>::run(w, ti, ScrS<1>{row}, acti);
      if (acti) {
#pragma unroll
        for (int e = 0; e < EI; ++e) {
          const int m = ti + TI * e;
          if (2 * m < L1) row[m] = w[e];
        }
      }
    }
  }
  __syncthreads();

  // 6. outer gate and store
  if constexpr (kPre) {
#pragma unroll
    for (int j = 0; j < JX; ++j) {
      const int i = tid + NT * j;
      if (NP % NT == 0 || i < NP) {
        const int r = i / (L1 / 2), m = i - r * (L1 / 2);
        const float2 q = S[r * RP + m], g = gpre[j];
        st2(y + base + 2 * i, make_float2(g.x * q.x, g.y * q.y));
      }
    }
  } else {
    batched_copy<L0 * L1 / 2, NT, 8>(
        tid, [&](int i) { return G.g2(ld2(x2 + base + 2 * i)); },
        [&](int i, float2 g) {
          const int r = i / (L1 / 2), m = i - r * (L1 / 2);
          const float2 q = S[r * RP + m];
          st2(y + base + 2 * i, make_float2(g.x * q.x, g.y * q.y));
        });
  }
}

template <int P0, int P1, typename TS>
static hipError_t launch_2d_fused_kc_t(const FftConvArgs& a, hipStream_t s) {
  if (a.act)
    hipLaunchKernelGGL((conv2d_fused_kc<P0, P1, TS, true>), dim3((unsigned)a.lines), dim3(512), 0, s, (const TS*)a.x1,
                       (const TS*)a.x2, (const TS*)a.v, (const TS*)a.k, (const TS*)a.D, (TS*)a.y, (int)a.C, a.kC,
                       a.act_in);
  else
    hipLaunchKernelGGL((conv2d_fused_kc<P0, P1, TS, false>), dim3((unsigned)a.lines), dim3(512), 0, s, (const TS*)a.x1,
                       (const TS*)a.x2, (const TS*)a.v, (const TS*)a.k, (const TS*)a.D, (TS*)a.y, (int)a.C, a.kC,
                       a.act_in);
  return hipGetLastError();
}

template <int P0, int P1, bool CIRC, typename TS>
static hipError_t launch_2d_fused_t(const FftConvArgs& a, hipStream_t s) {
  if (a.act) {
    hipLaunchKernelGGL((conv2d_fused<P0, P1, CIRC, TS, true>), dim3((unsigned)a.lines), dim3(512), 0, s,
                       (const TS*)a.x1, (const TS*)a.x2, (const TS*)a.v, (const TS*)a.k, (const TS*)a.D, (TS*)a.y,
                       (int)a.C, a.kC, a.act_in, nullptr);
  } else if (a.khat) {
    // each channel's spectrum once, then the images read it
    if (a.khat_pass != 2)
      hipLaunchKernelGGL((conv2d_fused<P0, P1, CIRC, TS, false, 1>), dim3((unsigned)a.C), dim3(512), 0, s,
                         (const TS*)a.x1, (const TS*)a.x2, (const TS*)a.v, (const TS*)a.k, (const TS*)a.D, (TS*)a.y,
                         (int)a.C, a.kC, a.act_in, a.khat);
    if (a.khat_pass != 1)
      hipLaunchKernelGGL((conv2d_fused<P0, P1, CIRC, TS, false, 2>), dim3((unsigned)a.lines), dim3(512), 0, s,
                         (const TS*)a.x1, (const TS*)a.x2, (const TS*)a.v, (const TS*)a.k, (const TS*)a.D, (TS*)a.y,
                         (int)a.C, a.kC, a.act_in, a.khat);
  } else {
    hipLaunchKernelGGL((conv2d_fused<P0, P1, CIRC, TS, false>), dim3((unsigned)a.lines), dim3(512), 0, s,
                       (const TS*)a.x1, (const TS*)a.x2, (const TS*)a.v, (const TS*)a.k, (const TS*)a.D, (TS*)a.y,
                       (int)a.C, a.kC, a.act_in, nullptr);
  }
  return hipGetLastError();
}

template <int P0, int P1>
static hipError_t launch_2d_fused_p(const FftConvArgs& a, hipStream_t s) {
  if (a.centered)
    return a.bf16 ? launch_2d_fused_kc_t<P0, P1, uint16_t>(a, s) : launch_2d_fused_kc_t<P0, P1, float>(a, s);
  if (a.circular) {
    return a.bf16 ? launch_2d_fused_t<P0, P1, true, uint16_t>(a, s) : launch_2d_fused_t<P0, P1, true, float>(a, s);
  }
  return a.bf16 ? launch_2d_fused_t<P0, P1, false, uint16_t>(a, s) : launch_2d_fused_t<P0, P1, false, float>(a, s);
}

// Instantiated sizes: squares 4..128 and the 2:1 shapes next to 64 and 128.
#define HY_FUSED2D_SIZES(X) \
  X(4, 4) X(8, 8) X(16, 16) X(32, 32) X(64, 64) X(128, 128) X(64, 128) X(128, 64) X(32, 64) X(64, 32)

bool fused2d_supported(int64_t P0, int64_t P1) {
#define HY_CASE(a, b) if (P0 == a && P1 == b) return true;
  HY_FUSED2D_SIZES(HY_CASE)
#undef HY_CASE
  return false;
}

size_t fused2d_khat_bytes(const FftConvArgs& a) {
  if (a.ndim != 2 || a.centered || a.rl || a.act || !fused2d_supported(a.P[0], a.P[1])) return 0;
  return ((size_t)a.C * (size_t)a.P[0] * (size_t)(a.P[1] / 2) * sizeof(float2) + 255) / 256 * 256;
}

hipError_t launch_fused2d(const FftConvArgs& a, hipStream_t s) {
#define HY_CASE(p0, p1) if (a.P[0] == p0 && a.P[1] == p1) return launch_2d_fused_p<p0, p1>(a, s);
  HY_FUSED2D_SIZES(HY_CASE)
#undef HY_CASE
  return hipErrorInvalidValue;
}

}  // namespace hyenand
