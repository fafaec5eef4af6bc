// The two normalisations around the long convolution in the HyenaND operator
// (Eq. (HyenaND), section 3.2), both across the C channels of every (sample,
// grid point) -- the reduction that the per-(b, c) transform kernels cannot do
// on their own, since a line holds one channel:
//
//   op_prologue_scale  s[b, p] = 1 / (max(||q[b, :, p]||, eps_l2) *
//                      sqrt(mean_c a^2 + eps_rms)),  a = q / max(||q||, eps_l2)
//                      * SiLU(kin); the transform kernels then stage
//                      u = q SiLU(kin) s w_in[c] with no second pass over q.
//   op_rmsnorm         y = z / sqrt(mean_c z^2 + eps_rms) * w_out[c], in place
//                      over the gated convolution output z (one read, one
//                      write: a tile of grid points x all channels in LDS).
//
// Both reduce in double precision and in a fixed order.
#include "kernels.hpp"

namespace hyenand {

namespace {

constexpr int kNormNT = 256;
constexpr int kNormLds = 16384;  // floats of the rmsnorm tile

// A workgroup takes kPro grid points; lane (j, pp) adds channels j, j + G, ...
// of point pp (G = kNormNT / kPro channel groups), eight loads in flight.
constexpr int kPro = 64;

template <typename TS>
__global__ void __launch_bounds__(kNormNT)
    op_prologue_scale(const TS* __restrict__ q, const TS* __restrict__ kin, float* __restrict__ s, int C,
                      int64_t npos, float eps_l2, float eps_rms) {
  constexpr int G = kNormNT / kPro;
  __shared__ double part[2][kNormNT];
  const int tid = threadIdx.x;
  const int pp = tid % kPro, j = tid / kPro;
  const int64_t b = blockIdx.y;
  const int64_t p = (int64_t)blockIdx.x * kPro + pp;
  const bool ok = p < npos;
  const TS* qb = q + b * C * npos + p;
  const TS* kb = kin + b * C * npos + p;
  double sq = 0.0, sa = 0.0;
  if (ok) {
    int c = j;
    for (; c + 7 * G < C; c += 8 * G) {
      float x[8], g[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        x[u] = ld1(qb + (int64_t)(c + u * G) * npos);
        g[u] = ld1(kb + (int64_t)(c + u * G) * npos);
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const double xd = x[u], a = xd * (double)silu_f(g[u]);
        sq += xd * xd;
        sa += a * a;
      }
    }
    for (; c < C; c += G) {
      const double xd = ld1(qb + (int64_t)c * npos), a = xd * (double)silu_f(ld1(kb + (int64_t)c * npos));
      sq += xd * xd;
      sa += a * a;
    }
  }
  part[0][tid] = sq;
  part[1][tid] = sa;
  __syncthreads();
  if (j == 0 && ok) {
    double tq = 0.0, ta = 0.0;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      tq += part[0][g * kPro + pp];
      ta += part[1][g * kPro + pp];
    }
    const double qn = fmax(sqrt(tq), (double)eps_l2);
    const double den = qn > 0.0 ? qn * sqrt(ta / (qn * qn) / C + (double)eps_rms) : 0.0;
    s[b * npos + p] = den > 0.0 ? (float)(1.0 / den) : 0.f;
  }
}

// PT grid points per workgroup (a power of two dividing npos, PT * C <=
// kNormLds).  Lanes move V = min(4, PT) consecutive points of one channel per
// access; the channel sums run over G = 256 / PT lanes per point.
template <typename TS, int PT>
__global__ void __launch_bounds__(kNormNT)
    op_rmsnorm(TS* __restrict__ y, const TS* __restrict__ w_out, int C, int64_t npos, float eps_rms) {
  constexpr int V = PT < 4 ? 1 : 4;
  constexpr int NV = PT / V;  // accesses per channel row of the tile
  __shared__ float tile[kNormLds];
  __shared__ double part[kNormNT];
  __shared__ float rinv[PT];
  const int tid = threadIdx.x;
  const int64_t b = blockIdx.y;
  const int64_t p0 = (int64_t)blockIdx.x * PT;
  TS* yb = y + b * C * npos + p0;
  const int n = C * NV;  // accesses of the tile
  {
    int i0 = tid;
    for (; i0 + 7 * kNormNT < n; i0 += 8 * kNormNT) {
      float4 z[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int i = i0 + u * kNormNT, c = i / NV, pv = (i % NV) * V;
        if constexpr (V == 4) z[u] = ld4(yb + (int64_t)c * npos + pv);
        else z[u].x = ld1(yb + (int64_t)c * npos + pv);
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int i = i0 + u * kNormNT;
        if constexpr (V == 4) *reinterpret_cast<float4*>(tile + 4 * i) = z[u];
        else tile[i] = z[u].x;
      }
    }
    for (; i0 < n; i0 += kNormNT) {
      const int c = i0 / NV, pv = (i0 % NV) * V;
      if constexpr (V == 4) *reinterpret_cast<float4*>(tile + 4 * i0) = ld4(yb + (int64_t)c * npos + pv);
      else tile[i0] = ld1(yb + (int64_t)c * npos + pv);
    }
  }
  __syncthreads();
  // tile[c * PT + pp]; lane (j, pp) adds channels j, j + G, ... of point pp
  constexpr int G = kNormNT / PT;
  {
    const int pp = tid % PT, j = tid / PT;
    double acc = 0.0;
    for (int c = j; c < C; c += G) {
      const double z = tile[c * PT + pp];
      acc += z * z;
    }
    part[tid] = acc;
  }
  __syncthreads();
  if (tid < PT) {
    double tot = 0.0;
#pragma unroll
    for (int j = 0; j < G; ++j) tot += part[j * PT + tid];
    const double r = sqrt(tot / C + (double)eps_rms);
    rinv[tid] = r > 0.0 ? (float)(1.0 / r) : 0.f;
  }
  __syncthreads();
  for (int i = tid; i < n; i += kNormNT) {
    const int c = i / NV, pv = (i % NV) * V;
    const float w = ld1(w_out + c);
    if constexpr (V == 4) {
      const float4 z = *reinterpret_cast<const float4*>(tile + 4 * i);
      st4(yb + (int64_t)c * npos + pv,
          make_float4(z.x * rinv[pv] * w, z.y * rinv[pv + 1] * w, z.z * rinv[pv + 2] * w, z.w * rinv[pv + 3] * w));
    } else {
      st1(yb + (int64_t)c * npos + pv, tile[i] * rinv[pv] * w);
    }
  }
}

template <typename TS>
hipError_t rmsnorm_pt(int PT, TS* y, const TS* w_out, int64_t B, int C, int64_t npos, float eps_rms,
                      hipStream_t st) {
  const dim3 grid((unsigned)(npos / PT), (unsigned)B);
  switch (PT) {
#define HY_CASE(pt) \
  case pt: hipLaunchKernelGGL((op_rmsnorm<TS, pt>), grid, dim3(kNormNT), 0, st, y, w_out, C, npos, eps_rms); break;
    HY_CASE(64) HY_CASE(32) HY_CASE(16) HY_CASE(8) HY_CASE(4) HY_CASE(2) HY_CASE(1)
#undef HY_CASE
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

int op_rmsnorm_points(int C) {
  int pt = 64;
  while (pt > 1 && pt * C > kNormLds) pt /= 2;
  return pt * C <= kNormLds ? pt : 0;
}

hipError_t launch_op_prologue(const void* q, const void* kin, float* s, int64_t B, int C, int64_t npos, bool bf16,
                              float eps_l2, float eps_rms, hipStream_t st) {
  const dim3 grid((unsigned)((npos + kPro - 1) / kPro), (unsigned)B);
  if (bf16)
    hipLaunchKernelGGL((op_prologue_scale<uint16_t>), grid, dim3(kNormNT), 0, st, (const uint16_t*)q,
                       (const uint16_t*)kin, s, C, npos, eps_l2, eps_rms);
  else
    hipLaunchKernelGGL((op_prologue_scale<float>), grid, dim3(kNormNT), 0, st, (const float*)q, (const float*)kin, s,
                       C, npos, eps_l2, eps_rms);
  return hipGetLastError();
}

hipError_t launch_op_rmsnorm(void* y, const void* w_out, int64_t B, int C, int64_t npos, bool bf16, float eps_rms,
                             hipStream_t st) {
  int PT = op_rmsnorm_points(C);
  if (PT < 1) return hipErrorInvalidValue;
  while (PT > 1 && npos % PT != 0) PT /= 2;  // npos is a power of two: PT divides it
  if (bf16) return rmsnorm_pt<uint16_t>(PT, (uint16_t*)y, (const uint16_t*)w_out, B, C, npos, eps_rms, st);
  return rmsnorm_pt<float>(PT, (float*)y, (const float*)w_out, B, C, npos, eps_rms, st);
}

}  // namespace hyenand
