// Backward of the gated long convolution for 2D/3D grids whose spectra do
// not fit in LDS: the multi-pass structure of the forward plan carried over
// to three signals.
//
// With gy = dLoss/dy, u = x1 v and h = gy x2, the gradients are gx2 = gy z,
// gu = k (*)^T h + D h, gk[m] = sum_n h[n] u[n - m], gx1 = gu v, gv = gu x1
// and gD[c] = sum_{b, n} h u (z = k * u + D u is the pre-gate output), i.e.
// the spectral products Z = U (K + D), GU = conj(K + D) H, GK = conj(U) H on
// the forward's transform grid, inverse-transformed and cropped like y.
//
//   rows_fwd   read x1, v, k, gy, x2 rows; u = x1 v, h = gy x2; real-to-
//              complex transforms of the nonzero rows of u, k and h along the
//              last axis; per-workgroup sums of h u for gD.
//   axis1_fwd  (3D) forward along axis 1 for the three signals.
//   core       along axis 0: forward transforms of U, K, H, the three
//              products, inverse transforms, keep the L0 cropped rows; Z, GU,
//              GK overwrite U, K, H.
//   axis1_inv  (3D) inverse along axis 1 for the three signals.
//   rows_inv   inverse along the last axis, two real rows per complex
//              transform; crop; gx2 = gy z, gx1 = gu v, gv = gu x1, gk.
//   reduce     gD[c]: the workgroup sums of every sample, added in order.
//
// The three spectra of a line (3 x the forward's U) go through the workspace,
// a chunk of lines at a time; the gD sums sit in front of them.
#include "multipass.hpp"

namespace hyenand {

namespace {

constexpr int pow2_floor(int n) { return n <= 1 ? 1 : 2 * pow2_floor(n / 2); }

// Sum over a workgroup of NT lanes (a multiple of 64); red holds NT / 64
// floats; lane 0 gets the total.  Fixed order, so the result is the same on
// every run.
template <int NT>
__device__ __forceinline__ float wg_sum(float x, float* red, int tid) {
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

// ---------------------------------------------------------------------------
// rows_fwd: u = x1 v, k and h = gy x2, real-to-complex along the last axis
// ---------------------------------------------------------------------------
template <int PL>
struct BRowsCfg {
  static constexpr int ML = PL / 2;
  static constexpr int HP = ML + 1;  // row pitch in LDS
  static constexpr int E = imin(16, ML);
  static constexpr int T = ML / E;
  static constexpr int NT = 256;
  // rows per workgroup (a power of two): three signal rows each, ~64 KB
  static constexpr int RPW = pow2_floor(imax(1, imin(NT / T, (64 * 1024) / (3 * HP * 8))));
};

struct In5 {
  float4 a, b, k, g, e;
};

template <int PL, bool CIRC, typename TS>
__global__ void __launch_bounds__(256)
    mpb_rows_fwd(const TS* __restrict__ x1, const TS* __restrict__ v, const TS* __restrict__ k,
                 const TS* __restrict__ gy, const TS* __restrict__ x2, float2* __restrict__ ws,
                 float* __restrict__ partial, int64_t line0, int rows, int rpw, int L1, int P1, int HS,
                 int64_t half, int64_t per_line) {
  using Cf = BRowsCfg<PL>;
  constexpr int ML = Cf::ML, HP = Cf::HP, E = Cf::E, T = Cf::T, NT = Cf::NT, RPW = Cf::RPW;
  constexpr int LL = CIRC ? PL : PL / 2;
  constexpr int H = ML + 1;
  constexpr int MNZ = (LL + 1) / 2;
  __shared__ float2 S[3][RPW * HP];  // u, k, h rows
  __shared__ float2 twl[imax(1, PassTw<ML, E>::kCount)];
  __shared__ float red[NT / 64];
  __shared__ int64_t roff[RPW];
  const int64_t row0 = (int64_t)blockIdx.x * rpw;  // rows of one line (rpw divides rows)
  const int tid = threadIdx.x;
  PassTw<ML, E>::fill(twl, tid, NT);
  ws_row_offsets<RPW, NT>(roff, row0, rpw, rows, L1, P1, HS, per_line, tid);

  // stage the real rows as packed pairs; every lane adds h u over the
  // elements it stages
  float hu = 0.f;
  {
    const size_t gbase = (size_t)(line0 * rows + row0) * LL;
    if constexpr (LL % 4 == 0) {
      batched_copy<RPW * (LL / 4), NT, 2>(
          tid,
          [&](int i4) {
            In5 z;
            const int i = 4 * i4;
            if (i / LL < rpw) {
              z.a = ld4(x1 + gbase + i);
              z.b = ld4(v + gbase + i);
              z.k = ld4(k + gbase + i);
              z.g = ld4(gy + gbase + i);
              z.e = ld4(x2 + gbase + i);
            }
            return z;
          },
          [&](int i4, const In5& z) {
            const int i = 4 * i4;
            const int r = i / LL, col = i - r * LL;
            if (r < rpw) {
              const float4 u = make_float4(z.a.x * z.b.x, z.a.y * z.b.y, z.a.z * z.b.z, z.a.w * z.b.w);
              const float4 h = make_float4(z.g.x * z.e.x, z.g.y * z.e.y, z.g.z * z.e.z, z.g.w * z.e.w);
              float2* du = S[0] + r * HP + col / 2;
              float2* dk = S[1] + r * HP + col / 2;
              float2* dh = S[2] + r * HP + col / 2;
              du[0] = make_float2(u.x, u.y);
              du[1] = make_float2(u.z, u.w);
              dk[0] = make_float2(z.k.x, z.k.y);
              dk[1] = make_float2(z.k.z, z.k.w);
              dh[0] = make_float2(h.x, h.y);
              dh[1] = make_float2(h.z, h.w);
              hu += (u.x * h.x + u.y * h.y) + (u.z * h.z + u.w * h.w);
            }
          });
    } else {
      float* uf = reinterpret_cast<float*>(S[0]);
      float* kf = reinterpret_cast<float*>(S[1]);
      float* hf = reinterpret_cast<float*>(S[2]);
      for (int i = tid; i < RPW * LL; i += NT) {
        const int r = i / LL, col = i - r * LL;
        if (r < rpw) {
          const float u = ld1(x1 + gbase + i) * ld1(v + gbase + i);
          const float h = ld1(gy + gbase + i) * ld1(x2 + gbase + i);
          uf[r * 2 * HP + col] = u;
          kf[r * 2 * HP + col] = ld1(k + gbase + i);
          hf[r * 2 * HP + col] = h;
          hu += u * h;
        }
      }
    }
  }
  const float tot = wg_sum<NT>(hu, red, tid);  // its barrier also publishes the staging
  if (tid == 0) partial[(line0 * rows) / rpw + blockIdx.x] = tot;

  // packed half-length transforms, lanes across the 3 rpw lines
  constexpr int NLINE = 3 * RPW;
  for (int l0 = 0; l0 < NLINE; l0 += NT / T) {
    const int l = l0 + tid % (NT / T), t = tid / (NT / T);
    const int r = l / 3, sg = l - 3 * r;
    const bool act = l < NLINE && r < rpw;
    float2* row = S[act ? sg : 0] + (act ? r : 0) * HP;
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
    const int r = l / 3, sg = l - 3 * r;
    if (r < rpw) {
      float2* row = S[sg] + r * HP;
      float2 xa, xb;
      r2c_pair(row[g], row[(ML - g) & (ML - 1)], twiddle<ilog2(PL), false>(g), xa, xb);
      row[g] = xa;
      row[ML - g] = xb;
    }
  }
  __syncthreads();

  // store the H bins of every row of U, K, H (rows start on cache lines)
  struct Bin3 {
    float2 u, k, h;
  };
  batched_copy<RPW * H, NT, 4>(
      tid,
      [&](int i) {
        const int r = i / H, f = i - r * H;
        Bin3 z;
        z.u = S[0][r * HP + f];
        z.k = S[1][r * HP + f];
        z.h = S[2][r * HP + f];
        return z;
      },
      [&](int i, const Bin3& z) {
        const int r = i / H, f = i - r * H;
        if (r < rpw) {
          float2* U = ws + roff[r] + f;
          U[0] = z.u;
          U[half] = z.k;
          U[2 * half] = z.h;
        }
      });
}

// ---------------------------------------------------------------------------
// core: along axis 0, forward U, K, H; Z = U (K + D), GU = conj(K + D) H,
// GK = conj(U) H (all scaled by the normalisation); inverse; crop.  The
// three column lines of a lane stay in registers; the LDS tile is only the
// exchange scratch.
// ---------------------------------------------------------------------------
template <int P0, bool CIRC>
struct BCoreCfg {
  static constexpr int NT = kTileNT;
  static constexpr int TL = mp_tl(P0, 1, kTileKB);
  static constexpr int E = mp_e(P0, TL, NT);
  static constexpr int T = P0 / E;
  static constexpr int TLP = TL + 1;
  static constexpr int L0 = CIRC ? P0 : P0 / 2;
};

template <int P0, bool CIRC>
__global__ void __launch_bounds__(kTileNT)
    mpb_core(float2* __restrict__ ws, const void* __restrict__ Dp, int dbf16, int64_t line0, int C, int ncols,
             int HS, int H, int64_t half, int64_t per_line, float scale) {
  using Cf = BCoreCfg<P0, CIRC>;
  constexpr int TL = Cf::TL, TLP = Cf::TLP, E = Cf::E, T = Cf::T, NT = Cf::NT, L0 = Cf::L0;
  __shared__ float2 tile[P0 * TLP];
  __shared__ float2 twl[imax(1, PassTw<P0, E>::kCount)];
  const int ntile = (ncols + TL - 1) / TL;
  const int tl = (int)(blockIdx.x % ntile);
  const int64_t line = blockIdx.x / ntile;
  const int col0 = tl * TL;
  const int tid = threadIdx.x;
  PassTw<P0, E>::fill(twl, tid, NT);
  const int c = (int)((line0 + line) % C);
  const float Dv = dbf16 ? ld1((const uint16_t*)Dp + c) : ld1((const float*)Dp + c);
  const float twoD = 2.f * Dv;  // the stored spectra are the doubled R2C outputs
  static_assert(NT / T >= TL, "one round of columns");
  const int cc = tid % TL, t = tid / TL;
  const bool act = t < T;
  const bool cv = act && col_valid(col0 + cc, ncols, HS, H);
  float2* const uc = ws + line * per_line + col0 + cc;  // U; K at + half, H at + 2 half
  const ScrS<TLP> sc{tile + cc};
  float2 wu[E], wk[E], wh[E];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int n = t + T * e;
    const bool ld = cv && (CIRC || n < L0);
    wu[e] = ld ? uc[(int64_t)n * ncols] : czero();
    wk[e] = ld ? uc[half + (int64_t)n * ncols] : czero();
    wh[e] = ld ? uc[2 * half + (int64_t)n * ncols] : czero();
  }
  BlockFFT<P0, E, false>::run(wu, t, sc, act, twl);
  BlockFFT<P0, E, false>::run(wk, t, sc, act, twl);
  BlockFFT<P0, E, false>::run(wh, t, sc, act, twl);
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const float2 kd = make_float2(wk[e].x + twoD, wk[e].y);
    const float2 U2 = wu[e], H2 = wh[e];
    wu[e] = c_scale(c_mul(U2, kd), scale);   // Z
    wk[e] = c_scale(c_mulc(H2, kd), scale);  // GU = H conj(K + D)
    wh[e] = c_scale(c_mulc(H2, U2), scale);  // GK = H conj(U)
  }
  BlockFFT<P0, E, true>::run(wu, t, sc, act, twl);
  BlockFFT<P0, E, true>::run(wk, t, sc, act, twl);
  BlockFFT<P0, E, true>::run(wh, t, sc, act, twl);
  if (cv) {
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int n = t + T * e;
      if (CIRC || n < L0) {
        uc[(int64_t)n * ncols] = wu[e];
        uc[half + (int64_t)n * ncols] = wk[e];
        uc[2 * half + (int64_t)n * ncols] = wh[e];
      }
    }
  }
}

// ---------------------------------------------------------------------------
// rows_inv: complex-to-real along the last axis for Z, GU, GK, two rows per
// transform; crop; the four gradient tensors.
// ---------------------------------------------------------------------------
template <int PL>
struct BRowsInvCfg {
  static constexpr int H = PL / 2 + 1;
  static constexpr int PRP = PL + 18;  // pair region pitch (holds 2H and the scratch)
  static constexpr int E = imin(16, PL);
  static constexpr int T = PL / E;
  static constexpr int NT = 256;
  static constexpr int PPW = imax(1, imin(NT / T, (48 * 1024) / (3 * PRP * 8)));  // pairs per workgroup
};

template <int PL, bool CIRC, typename TS>
__global__ void __launch_bounds__(256)
    mpb_rows_inv(const float2* __restrict__ ws, const TS* __restrict__ x1, const TS* __restrict__ v,
                 const TS* __restrict__ gy, TS* __restrict__ gx1, TS* __restrict__ gx2, TS* __restrict__ gv,
                 TS* __restrict__ gk, int64_t line0, int nlines, int rows, int L1, int P1, int HS, int64_t half,
                 int64_t per_line) {
  using Cf = BRowsInvCfg<PL>;
  constexpr int H = Cf::H, PRP = Cf::PRP, E = Cf::E, T = Cf::T, NT = Cf::NT, PPW = Cf::PPW;
  constexpr int LL = CIRC ? PL : PL / 2;
  constexpr int ML = PL / 2;
  __shared__ float2 reg[3][PPW * PRP];  // z, gu, gk pair regions
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
  struct Bin3 {
    float2 z, gu, gk;
  };
  batched_copy<PPW * 2 * H, NT, 4>(
      tid,
      [&](int i) {
        const int q = i / (2 * H), rem = i - q * 2 * H;
        const int ab = rem / H, f = rem - ab * H;
        Bin3 z;
        z.z = z.gu = z.gk = czero();
        if (q < npair) {
          const float2* src = ws + roff[2 * q + ab] + f;
          z.z = src[0];
          z.gu = src[half];
          z.gk = src[2 * half];
        }
        return z;
      },
      [&](int i, const Bin3& z) {
        const int q = i / (2 * H);
        const int o = q * PRP + (i - q * 2 * H);
        reg[0][o] = z.z;
        reg[1][o] = z.gu;
        reg[2][o] = z.gk;
      });
  __syncthreads();

  constexpr int NLINE = 3 * PPW;
  for (int l0 = 0; l0 < NLINE; l0 += NT / T) {
    const int l = l0 + tid % (NT / T), t = tid / (NT / T);
    const int q = l / 3, sg = l - 3 * q;
    const bool act = l < NLINE && q < npair;
    float2* R = reg[act ? sg : 0] + (act ? q : 0) * PRP;
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
    BlockFFT<PL, E, true>::run(w, t, ScrS<1>{R}, act, twl);
    if (act) {
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const int n = t + T * e;
        if (CIRC || n < LL) R[n] = w[e];
      }
    }
  }
  __syncthreads();

  // gradients; the rows of a pair are consecutive in every tensor
  const size_t gbase = (size_t)(line0 * rows + 2 * pair0) * LL;
  if constexpr (LL % 4 == 0) {
    struct In3 {
      float4 a, b, g;
    };
    batched_copy<PPW * 2 * (LL / 4), NT, 4>(
        tid,
        [&](int i4) {
          const int i = 4 * i4;
          In3 z;
          if ((i / LL) < 2 * npair) {
            z.a = ld4(x1 + gbase + i);
            z.b = ld4(v + gbase + i);
            z.g = ld4(gy + gbase + i);
          }
          return z;
        },
        [&](int i4, const In3& z) {
          const int i = 4 * i4;
          const int row = i / LL, n = i - row * LL;
          if (row < 2 * npair) {
            const int o = (row >> 1) * PRP + n;
            const bool odd = row & 1;
            float zz[4], gu[4], gkk[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              zz[j] = odd ? reg[0][o + j].y : reg[0][o + j].x;
              gu[j] = odd ? reg[1][o + j].y : reg[1][o + j].x;
              gkk[j] = odd ? reg[2][o + j].y : reg[2][o + j].x;
            }
            st4(gx2 + gbase + i, make_float4(z.g.x * zz[0], z.g.y * zz[1], z.g.z * zz[2], z.g.w * zz[3]));
            st4(gx1 + gbase + i, make_float4(z.b.x * gu[0], z.b.y * gu[1], z.b.z * gu[2], z.b.w * gu[3]));
            st4(gv + gbase + i, make_float4(z.a.x * gu[0], z.a.y * gu[1], z.a.z * gu[2], z.a.w * gu[3]));
            st4(gk + gbase + i, make_float4(gkk[0], gkk[1], gkk[2], gkk[3]));
          }
        });
  } else {
    for (int i = tid; i < npair * 2 * LL; i += NT) {
      const int row = i / LL, n = i - row * LL;
      const int o = (row >> 1) * PRP + n;
      const bool odd = row & 1;
      const float zz = odd ? reg[0][o].y : reg[0][o].x;
      const float gu = odd ? reg[1][o].y : reg[1][o].x;
      const float gkk = odd ? reg[2][o].y : reg[2][o].x;
      st1(gx2 + gbase + i, ld1(gy + gbase + i) * zz);
      st1(gx1 + gbase + i, ld1(v + gbase + i) * gu);
      st1(gv + gbase + i, ld1(x1 + gbase + i) * gu);
      st1(gk + gbase + i, gkk);
    }
  }
}

// gD[c] = sum over samples b (in order) of the nper workgroup sums of line (b, c)
template <typename TS>
__global__ void __launch_bounds__(256) mpb_reduce_D(const float* __restrict__ partial, TS* __restrict__ gD, int B,
                                                    int C, int nper) {
  const int c = blockIdx.x * 256 + threadIdx.x;
  if (c >= C) return;
  float acc = 0.f;
  for (int b = 0; b < B; ++b) {
    const float* p = partial + ((size_t)b * C + c) * nper;
    float s = 0.f;
    for (int j = 0; j < nper; ++j) s += p[j];
    acc += s;
  }
  st1(gD + c, acc);
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
struct MpbLaunch {
  const FftConvBwdArgs* b;
  MpGeom g;
  float2* ws;
  int64_t line0;
  int nl;
  int64_t per;  // complex entries per line (U, K and H)
  float scale;
  hipStream_t s;
};

template <int PL>
int rows_per_wg(int rows) {
  return BRowsCfg<PL>::RPW < rows ? BRowsCfg<PL>::RPW : rows;
}

template <int PL>
hipError_t b_rows_fwd(const MpbLaunch& L) {
  const FftConvArgs& a = L.b->f;
  const int rpw = rows_per_wg<PL>(L.g.rows);
  const dim3 grid((unsigned)((int64_t)L.nl * L.g.rows / rpw));
#define HY_ARGS(TS)                                                                                           \
  (const TS*)a.x1, (const TS*)a.v, (const TS*)a.k, (const TS*)L.b->gy, (const TS*)a.x2, L.ws, L.b->partial, \
      L.line0, L.g.rows, rpw, L.g.L1, L.g.P1, L.g.HS, L.g.half, L.per
  if (a.bf16) {
    if (a.circular) hipLaunchKernelGGL((mpb_rows_fwd<PL, true, uint16_t>), grid, dim3(256), 0, L.s, HY_ARGS(uint16_t));
    else hipLaunchKernelGGL((mpb_rows_fwd<PL, false, uint16_t>), grid, dim3(256), 0, L.s, HY_ARGS(uint16_t));
  } else {
    if (a.circular) hipLaunchKernelGGL((mpb_rows_fwd<PL, true, float>), grid, dim3(256), 0, L.s, HY_ARGS(float));
    else hipLaunchKernelGGL((mpb_rows_fwd<PL, false, float>), grid, dim3(256), 0, L.s, HY_ARGS(float));
  }
#undef HY_ARGS
  return hipGetLastError();
}

template <int P1, bool INV>
hipError_t b_axis1(const MpbLaunch& L) {
  constexpr int TL = TileCfg<P1, 3>::TL;
  const int ntile = (L.g.H + TL - 1) / TL;
  const dim3 grid((unsigned)((int64_t)L.nl * L.g.L0 * ntile));
  const int nload = INV ? P1 : L.g.L1;
  if (L.b->f.circular)
    hipLaunchKernelGGL((mp_axis1<P1, true, INV, 3>), grid, dim3(kTileNT), 0, L.s, L.ws, L.g.H, L.g.HS, L.g.L0,
                       L.g.half, L.per, nload, (int64_t)0);
  else
    hipLaunchKernelGGL((mp_axis1<P1, false, INV, 3>), grid, dim3(kTileNT), 0, L.s, L.ws, L.g.H, L.g.HS, L.g.L0,
                       L.g.half, L.per, nload, (int64_t)0);
  return hipGetLastError();
}
template <int P1>
hipError_t b_axis1_fwd(const MpbLaunch& L) { return b_axis1<P1, false>(L); }
template <int P1>
hipError_t b_axis1_inv(const MpbLaunch& L) { return b_axis1<P1, true>(L); }

template <int P0>
hipError_t b_core(const MpbLaunch& L) {
  const FftConvArgs& a = L.b->f;
  const int ncols = L.g.P1 * L.g.HS;
  if (a.circular) {
    constexpr int TL = BCoreCfg<P0, true>::TL;
    const dim3 grid((unsigned)((int64_t)L.nl * ((ncols + TL - 1) / TL)));
    hipLaunchKernelGGL((mpb_core<P0, true>), grid, dim3(kTileNT), 0, L.s, L.ws, a.D, (int)a.bf16, L.line0,
                       (int)a.C, ncols, L.g.HS, L.g.H, L.g.half, L.per, L.scale);
  } else {
    constexpr int TL = BCoreCfg<P0, false>::TL;
    const dim3 grid((unsigned)((int64_t)L.nl * ((ncols + TL - 1) / TL)));
    hipLaunchKernelGGL((mpb_core<P0, false>), grid, dim3(kTileNT), 0, L.s, L.ws, a.D, (int)a.bf16, L.line0,
                       (int)a.C, ncols, L.g.HS, L.g.H, L.g.half, L.per, L.scale);
  }
  return hipGetLastError();
}

template <int PL>
hipError_t b_rows_inv(const MpbLaunch& L) {
  const FftConvArgs& a = L.b->f;
  const int64_t pairs = (int64_t)L.nl * L.g.rows / 2;
  const dim3 grid((unsigned)((pairs + BRowsInvCfg<PL>::PPW - 1) / BRowsInvCfg<PL>::PPW));
#define HY_ARGS(TS)                                                                                        \
  L.ws, (const TS*)a.x1, (const TS*)a.v, (const TS*)L.b->gy, (TS*)L.b->gx1, (TS*)L.b->gx2, (TS*)L.b->gv, \
      (TS*)L.b->gk, L.line0, L.nl, L.g.rows, L.g.L1, L.g.P1, L.g.HS, L.g.half, L.per
  if (a.bf16) {
    if (a.circular) hipLaunchKernelGGL((mpb_rows_inv<PL, true, uint16_t>), grid, dim3(256), 0, L.s, HY_ARGS(uint16_t));
    else hipLaunchKernelGGL((mpb_rows_inv<PL, false, uint16_t>), grid, dim3(256), 0, L.s, HY_ARGS(uint16_t));
  } else {
    if (a.circular) hipLaunchKernelGGL((mpb_rows_inv<PL, true, float>), grid, dim3(256), 0, L.s, HY_ARGS(float));
    else hipLaunchKernelGGL((mpb_rows_inv<PL, false, float>), grid, dim3(256), 0, L.s, HY_ARGS(float));
  }
#undef HY_ARGS
  return hipGetLastError();
}

#define HY_BSIZE_SWITCH(P, FN, ARG)           \
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

hipError_t d_b_rows_fwd(int P, const MpbLaunch& L) { HY_BSIZE_SWITCH(P, b_rows_fwd, L) }
hipError_t d_b_axis1_fwd(int P, const MpbLaunch& L) { HY_BSIZE_SWITCH(P, b_axis1_fwd, L) }
hipError_t d_b_core(int P, const MpbLaunch& L) { HY_BSIZE_SWITCH(P, b_core, L) }
hipError_t d_b_axis1_inv(int P, const MpbLaunch& L) { HY_BSIZE_SWITCH(P, b_axis1_inv, L) }
hipError_t d_b_rows_inv(int P, const MpbLaunch& L) { HY_BSIZE_SWITCH(P, b_rows_inv, L) }

int b_rows_per_wg(int PL, int rows) {
  switch (PL) {
#define HY_CASE(p) \
  case p: return rows_per_wg<p>(rows);
    HY_CASE(2) HY_CASE(4) HY_CASE(8) HY_CASE(16) HY_CASE(32) HY_CASE(64) HY_CASE(128) HY_CASE(256) HY_CASE(512)
    HY_CASE(1024)
#undef HY_CASE
    default: return 1;
  }
}

}  // namespace

size_t backward_mp_bytes_per_line(const FftConvArgs& a) {
  return (size_t)(3 * mp_geom(a).half) * sizeof(float2);
}

int64_t backward_mp_partials_per_line(const FftConvArgs& a) {
  const MpGeom g = mp_geom(a);
  return g.rows / b_rows_per_wg(g.PL, g.rows);
}

hipError_t launch_backward_mp(const FftConvBwdArgs& b, int64_t line0, int64_t nl, void* ws, hipStream_t s) {
  const FftConvArgs& a = b.f;
  if (!multipass_supported(a) || nl < 1 || line0 < 0 || line0 + nl > a.lines) return hipErrorInvalidValue;
  MpbLaunch L;
  L.b = &b;
  L.g = mp_geom(a);
  L.ws = (float2*)ws;
  L.per = 3 * L.g.half;
  L.scale = (float)(1.0 / (4.0 * (double)L.g.P0 * (double)L.g.P1 * (double)L.g.PL));
  L.s = s;
  L.line0 = line0;
  L.nl = (int)nl;
  const bool three = a.ndim == 3;
  hipError_t e;
  if ((e = d_b_rows_fwd(L.g.PL, L)) != hipSuccess) return e;
  if (three && (e = d_b_axis1_fwd(L.g.P1, L)) != hipSuccess) return e;
  if ((e = d_b_core(L.g.P0, L)) != hipSuccess) return e;
  if (three && (e = d_b_axis1_inv(L.g.P1, L)) != hipSuccess) return e;
  return d_b_rows_inv(L.g.PL, L);
}

hipError_t launch_backward_reduce(const FftConvBwdArgs& b, int64_t nper, hipStream_t s) {
  const FftConvArgs& a = b.f;
  const int C = (int)a.C, B = (int)(a.lines / a.C);
  if (b.f.bf16)
    hipLaunchKernelGGL((mpb_reduce_D<uint16_t>), dim3((unsigned)((C + 255) / 256)), dim3(256), 0, s, b.partial,
                       (uint16_t*)b.gD, B, C, (int)nper);
  else
    hipLaunchKernelGGL((mpb_reduce_D<float>), dim3((unsigned)((C + 255) / 256)), dim3(256), 0, s, b.partial,
                       (float*)b.gD, B, C, (int)nper);
  return hipGetLastError();
}

}  // namespace hyenand
