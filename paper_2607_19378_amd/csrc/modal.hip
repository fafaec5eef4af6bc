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
#include "kernels.hpp"

namespace hyenand {

namespace {

constexpr int kModalWaves = 4;
constexpr int kModalT = 32;  // points per lane (advances of lambda^64)

__device__ __forceinline__ void polar(double mag_log, double phase, float& c, float& s, float& m) {
  const double two_pi = 6.283185307179586;
  const float r = (float)(phase - two_pi * rint(phase * (1.0 / two_pi)));  // in [-pi, pi]
  __sincosf(r, &s, &c);
  m = __expf((float)mag_log);
}

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

}  // namespace

hipError_t launch_modal(const float* a, const float* th, const float* re, const float* im, void* k, int64_t C,
                        int M, int64_t L, bool bf16, hipStream_t s) {
  const int64_t per_block = (int64_t)kModalWaves * 64 * kModalT;
  const dim3 grid((unsigned)((L + per_block - 1) / per_block), (unsigned)C), block(64 * kModalWaves);
  if (bf16)
    hipLaunchKernelGGL(modal_filter_kernel<uint16_t>, grid, block, 0, s, a, th, re, im, (uint16_t*)k, M, L);
  else
    hipLaunchKernelGGL(modal_filter_kernel<float>, grid, block, 0, s, a, th, re, im, (float*)k, M, L);
  return hipGetLastError();
}

}  // namespace hyenand
