// Three-pass plan for 3D grids whose planes fit in LDS (plan "slab3d"):
//
//   slab_fwd   one workgroup per (line, plane n0 < L0, signal u or k): stage
//              the plane's L1 real rows, real-to-complex transform of every
//              row along the last axis, then the axis-1 transform of every
//              bin column, written straight to the half spectrum
//              [L0][P1][HS] of the workspace;
//   core       along axis 0 (the multi-pass core, conv_multipass.hip):
//              forward U and K, gated product with the folded shortcut,
//              inverse, keep the L0 cropped planes; Y overwrites U;
//   slab_inv   one workgroup per (line, plane n0 < L0): axis-1 inverse of
//              every bin column with the crop to n1 < L1, complex-to-real
//              rows, crop, outer gate x2, store y.
//
// The two transforms of a plane stay on chip, so the spectra make one round
// trip through the workspace per pass pair (the five-pass plan writes and
// reads them twice more, between the row and the axis-1 passes).  The plane
// [L1][PL/2 + 1] of half spectra is the LDS working set; the DC and Nyquist
// bins of every row, both real, share column 0 as DC + i Nyquist, so the
// bin columns are P/2 complex columns.
//
// In linear mode the axis-1 transform of length P1 = 2 L1 has L1 nonzero
// inputs: its even outputs are the length-L1 transform of the column and its
// odd outputs the length-L1 transform of the column times exp(-2 pi i n /
// P1) (the first radix-2 step of a zero-padded input), so both run in place
// in the column's own L1 slots.  The inverse keeps the outputs n1 < L1 = P1/2
// only: x[n] = E[n] + exp(2 pi i n / P1) O[n] with E, O the length-L1
// inverses of the even and odd bins.  The axis-0 (core) transform is the
// paper's middle kernel of its three-kernel 2D structure (appendix "2D FFT
// Convolution"), carried to the third axis.
#include <stdlib.h>
#include <string.h>

#include "multipass.hpp"

namespace hyenand {

namespace {

template <int P, bool CIRC>
struct SlabCfg {
  static constexpr int ML = P / 2;             // packed row length (complex)
  static constexpr int HP = ML + 1;            // LDS row pitch (odd)
  static constexpr int L1 = CIRC ? P : P / 2;  // nonzero rows of a plane
  static constexpr int LL = L1;                // nonzero reals of a row
  static constexpr int MNZ = (LL + 1) / 2;     // nonzero packed points of a row
  static constexpr int ER = imin(16, ML), TR = ML / ER;  // row transforms
  static constexpr int NC = CIRC ? P : P / 2;            // column transform length
  static constexpr int EC = imin(16, NC), TC = NC / EC;  // column transforms
  static constexpr int NT = imin(1024, imax(64, imax(L1 * TR, ML * TC)));
  static constexpr int kLdsBytes = L1 * HP * 8 + P * 8;
};

template <int P, bool CIRC>
constexpr bool slab_fits() {
  return SlabCfg<P, CIRC>::kLdsBytes <= 150 * 1024;
}

// the packed DC + i Nyquist bin pair of a row from its two bins
__device__ __forceinline__ float2 pack_dc_nyq(float2 dc, float2 nyq) { return make_float2(dc.x - nyq.y, dc.y + nyq.x); }

// ACT: the HyenaND operator's gates (x1, v, x2 hold q, kin, vin; see Gates)
template <int P, bool CIRC, typename TS, bool ACT>
__global__ void __launch_bounds__((SlabCfg<P, CIRC>::NT))
    mp_slab_fwd(const TS* __restrict__ x1, const TS* __restrict__ v, const TS* __restrict__ k,
                float2* __restrict__ ws, int64_t line0, int L0, int HS, int64_t half, int64_t per_line, int kC,
                ActIn ain, int C) {
  using Cf = SlabCfg<P, CIRC>;
  constexpr int ML = Cf::ML, HP = Cf::HP, L1 = Cf::L1, LL = Cf::LL, MNZ = Cf::MNZ, NT = Cf::NT;
  __shared__ float2 pl[L1 * HP];
  __shared__ float2 nq[P];  // column 0's spectrum (DC + i Nyquist)
  const int tid = threadIdx.x;
  const int64_t bid = blockIdx.x;
  const int sig = (int)(bid & 1);
  const int64_t rest = bid >> 1;
  const int n0 = (int)(rest % L0);
  const int64_t line = rest / L0;
  const int64_t gline = line0 + line;
  const int64_t pts = (int64_t)L0 * L1 * LL;  // points of one (b, c) line
  const int64_t pbase = (int64_t)n0 * L1 * LL;

  // 0. the plane's rows, as packed pairs z[m] = s[2m] + i s[2m + 1]
  {
    const TS* a = sig ? k + k_line(gline, kC) * pts + pbase : x1 + gline * pts + pbase;
    const TS* b = v + gline * pts + pbase;
    const Gates<ACT> G = line_gates<ACT, TS>(ain, gline, C);
    batched_copy<L1 * LL / 2, NT, 4>(
        tid,
        [&](int i) {
          const float2 p = ld2(a + 2 * i);
          if (sig) return p;
          return G.u2(p, ld2(b + 2 * i), pbase + 2 * i);
        },
        [&](int i, float2 z) {
          const int r = i / (LL / 2), m = i - r * (LL / 2);
          pl[r * HP + m] = z;
        });
  }
  __syncthreads();

  // 1. row transforms (length ML, the packed half of a real row of P)
  {
    constexpr int E = Cf::ER, T = Cf::TR, LR = NT / T;
    using Map = LaneMap<T, NT>;
    for (int l0 = 0; l0 < L1; l0 += LR) {
      const int l = l0 + Map::line(tid), t = Map::t(tid);
      const bool act = L1 % LR == 0 || l < L1;
      float2* row = pl + (act ? l : 0) * HP;
      float2 w[E];
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const int m = t + T * e;
        w[e] = (act && (CIRC || m < MNZ)) ? row[m] : czero();
      }
      BlockFFT<ML, E, false>::run(w, t, ScrS<1>{row}, act);
      if (act) {
#pragma unroll
        for (int e = 0; e < E; ++e) row[t + T * e] = w[e];
      }
    }
  }
  __syncthreads();
  // The rows' real spectra come out of their packed transforms by untangling
  // (bin g from packed bins g and ML - g).  When one round of column lanes
  // covers the ML bin columns, each lane untangles the bins it loads (the
  // bin and its mirror are read before the first exchange barrier of the
  // axis-1 transforms, the first write to either slot); otherwise a pass
  // over the rows does it in place first.
  constexpr bool kColUntangle = ML <= NT / Cf::TC;
  if constexpr (!kColUntangle) {
    // untangle in place: item (row, g) owns bins g and ML - g; slot 0 of a
    // row keeps its DC and Nyquist bins (both real) as DC + i Nyquist
    constexpr int NG = imax(1, ML / 2);
    for (int it = tid; it < L1 * NG; it += NT) {
      const int l = it % L1, g = it / L1;
      float2* row = pl + l * HP;
      float2 xa, xb;
      if (g == 0) {
        r2c_pair(row[0], row[0], make_float2(1.f, 0.f), xa, xb);
        row[0] = make_float2(xa.x, xb.x);
        if constexpr (ML >= 2) {
          constexpr int h = ML / 2;
          r2c_pair(row[h], row[h], twiddle<ilog2(P), false>(h), xa, xb);
          row[h] = xa;
        }
      } else {
        r2c_pair(row[g], row[ML - g], twiddle<ilog2(P), false>(g), xa, xb);
        row[g] = xa;
        row[ML - g] = xb;
      }
    }
    __syncthreads();
  }

  // 2. axis-1 transforms of the ML bin columns, straight to the workspace:
  //    bin row f1 of plane n0 at ((n0 P + f1) HS) of this signal's half
  //    spectrum; column 0 goes through nq
  float2* const S = ws + line * per_line + (int64_t)sig * half + (int64_t)n0 * P * HS;
  {
    constexpr int E = Cf::EC, T = Cf::TC, NC = Cf::NC, CR = NT / T;
    using Map = LaneMap<T, NT>;
    for (int c0 = 0; c0 < ML; c0 += CR) {
      const int col = c0 + Map::line(tid), t = Map::t(tid);
      const bool act = ML % CR == 0 || col < ML;
      const int cc = act ? col : 0;
      const ScrS<HP> sc{pl + cc};
      const int mc = (ML - cc) & (ML - 1);                // mirror bin (0 for 0)
      const float2 twc = twiddle<ilog2(P), false>(cc);   // (1, 0) for column 0
      float2 x[E];
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const float2* row = pl + (t + T * e) * HP;
        if constexpr (kColUntangle) x[e] = act ? untangle_bin(row, cc, mc, twc) : czero();
        else x[e] = act ? row[cc] : czero();
      }
      if constexpr (CIRC) {
        BlockFFT<NC, E, false>::run(x, t, sc, act);
        if (act) {
#pragma unroll
          for (int e = 0; e < E; ++e) {
            const int f1 = t + T * e;
            if (cc == 0) nq[f1] = x[e];
            else S[(int64_t)f1 * HS + cc] = x[e];
          }
        }
      } else {
        float2 xs[E];
#pragma unroll
        for (int e = 0; e < E; ++e) xs[e] = x[e];
        BlockFFT<NC, E, false>::run(x, t, sc, act);  // even bins f1 = 2j
        if (act) {
#pragma unroll
          for (int e = 0; e < E; ++e) {
            const int f1 = 2 * (t + T * e);
            if (cc == 0) nq[f1] = x[e];
            else S[(int64_t)f1 * HS + cc] = x[e];
          }
        }
#pragma unroll
        for (int e = 0; e < E; ++e) x[e] = c_mul(xs[e], twiddle<ilog2(P), false>(t + T * e));
        BlockFFT<NC, E, false>::run(x, t, sc, act);  // odd bins f1 = 2j + 1
        if (act) {
#pragma unroll
          for (int e = 0; e < E; ++e) {
            const int f1 = 2 * (t + T * e) + 1;
            if (cc == 0) nq[f1] = x[e];
            else S[(int64_t)f1 * HS + cc] = x[e];
          }
        }
      }
    }
  }
  __syncthreads();
  // column 0 holds A + i B with A, B the axis-1 spectra of the DC and the
  // Nyquist column: A = (Z[f] + conj Z[-f]) / 2, B = -i (Z[f] - conj Z[-f]) / 2
  for (int f = tid; f < P; f += NT) {
    const float2 z = nq[f], zm = nq[(P - f) & (P - 1)];
    S[(int64_t)f * HS] = make_float2(0.5f * (z.x + zm.x), 0.5f * (z.y - zm.y));
    S[(int64_t)f * HS + ML] = make_float2(0.5f * (z.y + zm.y), 0.5f * (zm.x - z.x));
  }
}

template <int P, bool CIRC, typename TS, bool ACT>
__global__ void __launch_bounds__((SlabCfg<P, CIRC>::NT))
    mp_slab_inv(const float2* __restrict__ ws, const TS* __restrict__ x2, TS* __restrict__ y, int64_t line0,
                int L0, int HS, int64_t per_line) {
  using Cf = SlabCfg<P, CIRC>;
  constexpr int ML = Cf::ML, HP = Cf::HP, L1 = Cf::L1, LL = Cf::LL, NT = Cf::NT;
  __shared__ float2 pl[L1 * HP];
  const int tid = threadIdx.x;
  const int64_t bid = blockIdx.x;
  const int n0 = (int)(bid % L0);
  const int64_t line = bid / L0;
  const int64_t gline = line0 + line;
  const float2* const Y = ws + line * per_line + (int64_t)n0 * P * HS;

  // 1. axis-1 inverse of the ML bin columns (column 0 as DC + i Nyquist),
  //    rows n1 < L1 kept, into the plane
  {
    constexpr int E = Cf::EC, T = Cf::TC, NC = Cf::NC, CR = NT / T;
    using Map = LaneMap<T, NT>;
    for (int c0 = 0; c0 < ML; c0 += CR) {
      const int col = c0 + Map::line(tid), t = Map::t(tid);
      const bool act = ML % CR == 0 || col < ML;
      const int cc = act ? col : 0;
      const ScrS<HP> sc{pl + cc};
      auto bin = [&](int f1) -> float2 {
        const float2* r = Y + (int64_t)f1 * HS;
        return cc == 0 ? pack_dc_nyq(r[0], r[ML]) : r[cc];
      };
      if constexpr (CIRC) {
        float2 x[E];
#pragma unroll
        for (int e = 0; e < E; ++e) x[e] = act ? bin(t + T * e) : czero();
        BlockFFT<NC, E, true>::run(x, t, sc, act);
        __syncthreads();  // every lane's last exchange read is done
        if (act) {
#pragma unroll
          for (int e = 0; e < E; ++e) pl[(t + T * e) * HP + cc] = x[e];
        }
      } else {
        float2 ev[E], od[E];
#pragma unroll
        for (int e = 0; e < E; ++e) {
          ev[e] = act ? bin(2 * (t + T * e)) : czero();
          od[e] = act ? bin(2 * (t + T * e) + 1) : czero();
        }
        BlockFFT<NC, E, true>::run(ev, t, sc, act);
        BlockFFT<NC, E, true>::run(od, t, sc, act);
        __syncthreads();  // every lane's last exchange read is done
        if (act) {
#pragma unroll
          for (int e = 0; e < E; ++e) {
            const int n = t + T * e;
            pl[n * HP + cc] = c_add(ev[e], c_mul(od[e], twiddle<ilog2(P), true>(n)));
          }
        }
      }
    }
  }
  __syncthreads();

  // outer gate values of the items this lane stores in step 3, as raw storage
  // words, fetched now so that their latency hides behind the row transforms
  const int64_t gbase = (gline * L0 + n0) * (int64_t)L1 * LL;
  constexpr int NI = L1 * LL / 2, IT = (NI + NT - 1) / NT;
  constexpr bool kPre = IT <= 8;
  typename Raw2<TS>::type g2r[kPre ? IT : 1];
  if constexpr (kPre) {
#pragma unroll
    for (int j = 0; j < IT; ++j) {
      const int i = tid + NT * j;
      if (NI % NT == 0 || i < NI) g2r[j] = ld2_raw(x2 + gbase + 2 * i);
    }
  }

  // 2. complex-to-real rows: c2r_pair turns row n1's half spectrum (slot 0
  //    holding DC + i Nyquist) into the length-ML transform of its even/odd
  //    output pairs; the inverse leaves y[2m] + i y[2m + 1] in slot m
  {
    constexpr int E = Cf::ER, T = Cf::TR, LR = NT / T;
    using Map = LaneMap<T, NT>;
    for (int r0 = 0; r0 < L1; r0 += LR) {
      const int r = r0 + Map::line(tid), t = Map::t(tid);
      const bool act = L1 % LR == 0 || r < L1;
      float2* row = pl + (act ? r : 0) * HP;
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
          Ym = row[ML - g];
        }
        w[e] = act ? c2r_pair(Yg, Ym, twiddle<ilog2(P), false>(g)) : czero();
      }
      BlockFFT<ML, E, true>::run(w, t, ScrS<1>{row}, act);
      if (act) {
#pragma unroll
        for (int e = 0; e < E; ++e) {
          const int m = t + T * e;
          if (CIRC || 2 * m < LL) row[m] = w[e];
        }
      }
    }
  }
  __syncthreads();

  // 3. outer gate and store, coalesced along rows
  if constexpr (kPre) {
#pragma unroll
    for (int j = 0; j < IT; ++j) {
      const int i = tid + NT * j;
      if (NI % NT == 0 || i < NI) {
        const float2 g = Gates<ACT>{}.g2(widen2(g2r[j]));
        const int r = i / (LL / 2), m = i - r * (LL / 2);
        const float2 q = pl[r * HP + m];
        st2(y + gbase + 2 * i, make_float2(g.x * q.x, g.y * q.y));
      }
    }
  } else {
    batched_copy<L1 * LL / 2, NT, 4>(
        tid, [&](int i) { return Gates<ACT>{}.g2(ld2(x2 + gbase + 2 * i)); },
        [&](int i, float2 g) {
          const int r = i / (LL / 2), m = i - r * (LL / 2);
          const float2 q = pl[r * HP + m];
          st2(y + gbase + 2 * i, make_float2(g.x * q.x, g.y * q.y));
        });
  }
}

template <int P, bool CIRC>
hipError_t slab_launch(const FftConvArgs& a, const MpGeom& g, float2* ws, int64_t line0, int nl, int64_t per,
                       bool inverse, hipStream_t s) {
  if constexpr (!slab_fits<P, CIRC>()) {
    return hipErrorInvalidValue;
  } else {
    constexpr int NT = SlabCfg<P, CIRC>::NT;
    if (!inverse) {
      const dim3 grid((unsigned)((int64_t)nl * g.L0 * 2));
#define HY_FWD(TS, ACT)                                                                                        \
  hipLaunchKernelGGL((mp_slab_fwd<P, CIRC, TS, ACT>), grid, dim3(NT), 0, s, (const TS*)a.x1, (const TS*)a.v, \
                     (const TS*)a.k, ws, line0, g.L0, g.HS, g.half, per, a.kC, a.act_in, (int)a.C)
      if (a.bf16) {
        if (a.act) HY_FWD(uint16_t, true); else HY_FWD(uint16_t, false);
      } else {
        if (a.act) HY_FWD(float, true); else HY_FWD(float, false);
      }
#undef HY_FWD
    } else {
      const dim3 grid((unsigned)((int64_t)nl * g.L0));
#define HY_INV(TS, ACT)                                                                                   \
  hipLaunchKernelGGL((mp_slab_inv<P, CIRC, TS, ACT>), grid, dim3(NT), 0, s, ws, (const TS*)a.x2, (TS*)a.y, \
                     line0, g.L0, g.HS, per)
      if (a.bf16) {
        if (a.act) HY_INV(uint16_t, true); else HY_INV(uint16_t, false);
      } else {
        if (a.act) HY_INV(float, true); else HY_INV(float, false);
      }
#undef HY_INV
    }
    return hipGetLastError();
  }
}

}  // namespace

bool slab3d_supported(const FftConvArgs& a) {
  if (a.ndim != 3 || a.centered || a.rl || a.periodic) return false;
  if (getenv("HYENAND_SLAB") && strcmp(getenv("HYENAND_SLAB"), "0") == 0) return false;
  const int64_t P = a.P[2];
  if (a.P[1] != P || a.L[1] != a.L[2]) return false;
  if (a.circular) return P == 64 || P == 128;
  return P == 64 || P == 128 || P == 256;
}

hipError_t launch_slab3d(const FftConvArgs& a, int64_t line0, int64_t nl, void* ws, bool inverse, hipStream_t s) {
  if (!slab3d_supported(a) || nl < 1 || line0 < 0 || line0 + nl > a.lines) return hipErrorInvalidValue;
  const MpGeom g = mp_geom(a);
  const int64_t per = g.half + g.halfK;
  float2* w = (float2*)ws;
  const int P = (int)a.P[2];
  if (a.circular) {
    if (P == 64) return slab_launch<64, true>(a, g, w, line0, (int)nl, per, inverse, s);
    if (P == 128) return slab_launch<128, true>(a, g, w, line0, (int)nl, per, inverse, s);
  } else {
    if (P == 64) return slab_launch<64, false>(a, g, w, line0, (int)nl, per, inverse, s);
    if (P == 128) return slab_launch<128, false>(a, g, w, line0, (int)nl, per, inverse, s);
    if (P == 256) return slab_launch<256, false>(a, g, w, line0, (int)nl, per, inverse, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace hyenand
