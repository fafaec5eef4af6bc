// Modal filter generation: the implicit long filter of order M (the appendix
// "Filter Generation"), per channel c a sum of M damped complex exponentials,
//
//   k[c, t] = Re sum_m R[c, m] lambda[c, m]^t,  lambda = exp(a + i theta),
//
// written straight to the [C, L] kernel a one-kernel-per-channel convolution
// reads; the [M, L] complex terms are never materialised.  A lane owns the
// points t0 + 64 j (j < kModalT) of one channel, so every store instruction
// writes 64 consecutive points.  For each mode it forms z = R lambda^t0 once
// (the phase t0 theta and the log-magnitude t0 a in double, the phase reduced
// to [-pi, pi] before the fp32 sine and cosine), then advances
// z <- z lambda^64 in fp32, adding Re z into the point's sum: five VALU
// operations per mode and point.  The step drifts by about one fp32 rounding
// per advance, so kModalT bounds the drift.
//
// Up to order 32 the sum runs on the fp32 matrix cores instead.  A tile of
// 1024 points t = t0 + 32 r + n (r, n < 32) is the real part of a product
// of a [32 x M] and an [M x 32] complex matrix,
//
//   k[t0 + 32 r + n] = Re sum_m (R_m lambda_m^(t0 + 32 r)) (lambda_m^n),
//
// i.e. one real [32 x 2M] x [2M x 32] product (Re z Re w - Im z Im w
// summed over the modes), M v_mfma_f32_32x32x2f32 per tile with M rounded
// up to 16 or 32 (for a bf16 kernel tensor, M / 8 bf16 products instead).  The right factor lambda^n is fixed per channel; the left
// one advances by lambda^1024 from tile to tile (four VALU operations per
// mode and row) and is recomputed exactly, as above, every kTilesPerWave
// tiles.
#include "kernels.hpp"

namespace hyenand {

namespace {

constexpr int kModalWaves = 4;
constexpr int kModalT = 32;  // points per lane (advances of lambda^64)


template <typename TS>
__global__ void __launch_bounds__(64 * kModalWaves)
    modal_filter_kernel(const float* __restrict__ a, const float* __restrict__ th, const float* __restrict__ re,
                        const float* __restrict__ im, TS* __restrict__ k, int M, int64_t L) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t c = blockIdx.y;
  const int64_t tw = ((int64_t)blockIdx.x * kModalWaves + wave) * 64 * kModalT;  // the wave's first point
  if (tw >= L) return;  // uniform across the wave
  const int64_t t0 = tw + lane;
  float acc[kModalT];
#pragma unroll
  for (int j = 0; j < kModalT; ++j) acc[j] = 0.f;
  for (int m = 0; m < M; ++m) {
    const int64_t i = c * M + m;
    const float am = a[i], tm = th[i], rr = re[i], ri = im[i];
    float c0, s0, m0, cs, ss, ms;
    polar((double)t0 * am, (double)t0 * tm, c0, s0, m0);
    polar(64.0 * am, 64.0 * tm, cs, ss, ms);
    float zr = m0 * (rr * c0 - ri * s0), zi = m0 * (rr * s0 + ri * c0);
    const float sr = ms * cs, si = ms * ss;  // lambda^64
#pragma unroll
    for (int j = 0; j < kModalT; ++j) {
      acc[j] += zr;
      const float nr = fmaf(zr, sr, -zi * si);
      zi = fmaf(zr, si, zi * sr);
      zr = nr;
    }
  }
  TS* out = k + c * L;
#pragma unroll
  for (int j = 0; j < kModalT; ++j)
    if (t0 + 64 * j < L) st1(out + t0 + 64 * j, acc[j]);
}

// ---------------------------------------------------------------------------
// matrix-core form (order <= 16 MG)
// ---------------------------------------------------------------------------
typedef float v16f __attribute__((ext_vector_type(16)));

constexpr int kMfmaWaves = 4;
constexpr int kTile = 1024;         // points per product: 32 rows of 32
constexpr int kTilesPerWave = 32;   // tiles between exact anchors: at most 31 advances of lambda^1024

// Lane l of a wave takes row r = l % 32 of the left factor and column
// n = l % 32 of the right one; half h = l / 32 supplies inner index 2 s + h of
// product step s.  The halves own disjoint modes, h MH + i (i < MH = MM / 2),
// and step s takes mode i = s % MH of the lane's half, its real part for
// s < MH (A = Re z, B = Re w) and its imaginary part after (A = -Im z,
// B = Im w), so the inner sum is Re z Re w - Im z Im w over every mode and
// each lane advances only its own MH factors.  The stores of a tile's result
// (straight from the matrix-core layout: 32 consecutive points per half-wave
// and register) are issued with the next tile's products, which hide them.
template <int MH>
__device__ __forceinline__ v16f tile_product(const float (&zr)[MH], const float (&zn)[MH], const float (&br)[MH],
                                             const float (&bi)[MH]) {
  v16f acc;
#pragma unroll
  for (int e = 0; e < 16; ++e) acc[e] = 0.f;
#pragma unroll
  for (int s = 0; s < 2 * MH; ++s)
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(s < MH ? zr[s % MH] : zn[s % MH], s < MH ? br[s % MH] : bi[s % MH],
                                               acc, 0, 0, 0);
  return acc;
}

// For a bf16 kernel tensor the same product runs on
// v_mfma_f32_32x32x16_bf16 with both factors rounded to bf16 (the factors
// still advance in fp32; the rounding is of the order of the output's own).
// Lane half h supplies inner indices 16 s + 8 h + t (t < 8) of product s:
// the real parts of its modes 8 s + t for s < NS / 2, then the imaginary
// parts, NS = MH / 4 products per tile.
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));

template <int MH>
__device__ __forceinline__ v16f tile_product_bf(const float (&zr)[MH], const float (&zn)[MH],
                                                const v8bf (&bq)[MH / 4]) {
  constexpr int NS = MH / 4, NH = NS / 2;
  v16f acc;
#pragma unroll
  for (int e = 0; e < 16; ++e) acc[e] = 0.f;
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    v8bf av;
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      const int i = 8 * (s % NH) + t;
      av[t] = (__bf16)(s < NH ? zr[i] : zn[i]);
    }
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, bq[s], acc, 0, 0, 0);
  }
  return acc;
}

// register e of a tile's result: row 8 (e / 4) + 4 h + e % 4, column r
__device__ __forceinline__ int tile_pos(int e, int h, int r) { return 32 * (8 * (e >> 2) + 4 * h + (e & 3)) + r; }

template <typename TS>
__device__ __forceinline__ void store_tile(TS* p, const v16f& acc, int h, int r) {
#pragma unroll
  for (int e = 0; e < 16; ++e) st1(p + tile_pos(e, h, r), acc[e]);
}

template <typename TS, int MG>
__global__ void __launch_bounds__(64 * kMfmaWaves) __attribute__((amdgpu_waves_per_eu(MG == 1 ? 4 : 2)))
    modal_mfma_kernel(const float* __restrict__ a, const float* __restrict__ th, const float* __restrict__ re,
                      const float* __restrict__ im, TS* __restrict__ k, int M, int64_t L, int ntile) {
  constexpr int MM = 16 * MG, MH = MM / 2;
  // factors, computed once per workgroup by all its lanes (modes m >= M are zero)
  __shared__ float2 zs[kMfmaWaves][MM][32];  // R lambda^(tw + 32 r) per wave, mode, row
  __shared__ float2 bs[MM][32];              // lambda^n
  __shared__ float2 ws[MM];                  // lambda^1024
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r = lane & 31, h = lane >> 5;
  const int64_t c = blockIdx.y;
  const int64_t span = (int64_t)ntile * kTile;
  const int64_t tblk = (int64_t)blockIdx.x * kMfmaWaves * span;
  const float* const ac = a + c * M;
  const float* const tc = th + c * M;
  for (int i = tid; i < MM * 32; i += 64 * kMfmaWaves) {
    const int m = i >> 5, n = i & 31;
    float2 v = make_float2(0.f, 0.f);
    if (m < M) {
      float cs, sn, mg;
      polar((double)n * ac[m], (double)n * tc[m], cs, sn, mg);
      v = make_float2(mg * cs, mg * sn);
    }
    bs[m][n] = v;
  }
  for (int m = tid; m < MM; m += 64 * kMfmaWaves) {
    float2 v = make_float2(0.f, 0.f);
    if (m < M) {
      float cs, sn, mg;
      polar((double)kTile * ac[m], (double)kTile * tc[m], cs, sn, mg);
      v = make_float2(mg * cs, mg * sn);
    }
    ws[m] = v;
  }
  {
    // lane (r, h) of each wave forms the factors of its own modes of row r
    const double t = (double)(tblk + (int64_t)wave * span + 32 * r);
    for (int i = 0; i < MH; ++i) {
      const int m = h * MH + i;
      float2 v = make_float2(0.f, 0.f);
      if (m < M) {
        const float rr = re[c * M + m], ri = im[c * M + m];
        float cs, sn, mg;
        polar(t * ac[m], t * tc[m], cs, sn, mg);
        v = make_float2(mg * (rr * cs - ri * sn), mg * (rr * sn + ri * cs));
      }
      zs[wave][m][r] = v;
    }
  }
  __syncthreads();
  const int64_t tw = tblk + (int64_t)wave * span;  // the wave's first point
  if (tw >= L) return;  // uniform across the wave; no barrier follows
  float zr[MH], zn[MH], br[MH], bi[MH], wr[MH], wi[MH];  // zn = -Im z
#pragma unroll
  for (int i = 0; i < MH; ++i) {
    const int m = h * MH + i;
    const float2 z = zs[wave][m][r], w = bs[m][r], st = ws[m];
    zr[i] = z.x;
    zn[i] = -z.y;
    br[i] = w.x;
    bi[i] = w.y;
    wr[i] = st.x;
    wi[i] = st.y;
  }
  constexpr bool BF = sizeof(TS) == 2;
  v8bf bq[MH / 4];
  if constexpr (BF) {
    constexpr int NH = MH / 8;
#pragma unroll
    for (int q = 0; q < MH / 4; ++q)
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const int i = 8 * (q % NH) + t;
        bq[q][t] = (__bf16)(q < NH ? br[i] : bi[i]);
      }
  }
  auto product = [&]() {
    if constexpr (BF) return tile_product_bf<MH>(zr, zn, bq);
    else return tile_product<MH>(zr, zn, br, bi);
  };
  TS* out = k + c * L + tw;
  int64_t nfull = (L - tw) / kTile;  // whole tiles of the wave
  if (nfull > ntile) nfull = ntile;
  // whole tiles, each one's stores issued with the next one's products
  v16f prev;
  for (int64_t j = 0; j < nfull; ++j) {
    const v16f acc = product();
    if (j > 0) store_tile(out + (j - 1) * kTile, prev, h, r);
#pragma unroll
    for (int i = 0; i < MH; ++i) {
      const float nr = fmaf(zr[i], wr[i], zn[i] * wi[i]);
      zn[i] = fmaf(zn[i], wr[i], -zr[i] * wi[i]);
      zr[i] = nr;
    }
    prev = acc;
  }
  if (nfull > 0) store_tile(out + (nfull - 1) * kTile, prev, h, r);
  // the part of a tile before the end of the line
  if (nfull < ntile && tw + nfull * kTile < L) {
    const v16f acc = product();
    const int64_t t0 = tw + nfull * kTile;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int p = tile_pos(e, h, r);
      if (t0 + p < L) st1(out + nfull * kTile + p, acc[e]);
    }
  }
}

template <typename TS, int MG>
void launch_mfma(const float* a, const float* th, const float* re, const float* im, TS* k, int64_t C, int M,
                 int64_t L, hipStream_t s) {
  // tiles per wave: up to kTilesPerWave, fewer for short filters so that a
  // channel still spreads over several waves
  const int64_t tiles = (L + kTile - 1) / kTile;
  int ntile = (int)(tiles / 16);
  ntile = ntile < 1 ? 1 : (ntile > kTilesPerWave ? kTilesPerWave : ntile);
  const int64_t per_block = (int64_t)kMfmaWaves * ntile * kTile;
  const dim3 grid((unsigned)((L + per_block - 1) / per_block), (unsigned)C), block(64 * kMfmaWaves);
  hipLaunchKernelGGL((modal_mfma_kernel<TS, MG>), grid, block, 0, s, a, th, re, im, k, M, L, ntile);
}

template <typename TS>
void launch_typed(const float* a, const float* th, const float* re, const float* im, TS* k, int64_t C, int M,
                  int64_t L, hipStream_t s) {
  if (M <= 16) {
    launch_mfma<TS, 1>(a, th, re, im, k, C, M, L, s);
  } else if (M <= 32) {
    launch_mfma<TS, 2>(a, th, re, im, k, C, M, L, s);
  } else {
    const int64_t per_block = (int64_t)kModalWaves * 64 * kModalT;
    const dim3 grid((unsigned)((L + per_block - 1) / per_block), (unsigned)C), block(64 * kModalWaves);
    hipLaunchKernelGGL(modal_filter_kernel<TS>, grid, block, 0, s, a, th, re, im, k, M, L);
  }
}

}  // namespace

hipError_t launch_modal(const float* a, const float* th, const float* re, const float* im, void* k, int64_t C,
                        int M, int64_t L, bool bf16, hipStream_t s) {
  if (bf16) launch_typed(a, th, re, im, (uint16_t*)k, C, M, L, s);
  else launch_typed(a, th, re, im, (float*)k, C, M, L, s);
  return hipGetLastError();
}

}  // namespace hyenand
