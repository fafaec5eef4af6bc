// Kernel synthesis on the matrix cores: the HyenaND kernel K(x) = w(r) *
// f_theta(r; z(x)) evaluated on the kernel grid of a convolution
// (section 3.2.1, Eq. (kernel): a SIREN over the normalised grid coordinates;
// section 3.2.2, Eq. (film): per-sample scales and shifts after every hidden
// sine; the masking appendix, Eq. (mask): the per-axis Gaussian window, or
// the exponential decay of the original Hyena).
//
// The hidden layers and the output projection are dense contractions over the
// hidden width Hf, so they run on v_mfma_f32_32x32x2_f32 (fp32 in, fp32
// accumulate).  One wave owns 32 grid points of one sample and carries them
// through every layer without leaving registers: the matrix product is taken
// transposed, out[unit, point] = sum_k W[k, unit] h[point, k], so the points
// are the 32 columns (lane % 32) and the units the 32 rows of each tile.  The
// accumulator layout of one tile (lane l, register e: row 8 (e / 4) +
// 4 (l / 32) + e % 4, column l % 32) then already is the operand layout of
// the next layer, because a contraction may visit its k index in any order:
// at the step of register e the two lane halves contribute units
// 8 (e / 4) + e % 4 and that + 4, and the weight operand is read for exactly
// those units.  Only weights are loaded (from L1/L2, shared by every wave);
// the points' coordinates are generated from their index; K is written once.
#include "kernels.hpp"

namespace hyenand {

namespace {

typedef float v16f __attribute__((ext_vector_type(16)));

constexpr int kSynthWaves = 4;  // independent waves per workgroup

// the hidden unit (within a 32-unit tile) a lane of half g holds in register e
__device__ __forceinline__ int tile_unit(int e, int g) { return 8 * (e >> 2) + 4 * g + (e & 3); }

// sin(x): two-constant Cody-Waite reduction to [-pi, pi], then the hardware
// sine (which takes its argument in turns)
__device__ __forceinline__ float sin_reduced(float x) {
  const float n = rintf(x * 0.15915494309189535f);
  float r = fmaf(-n, 6.28318548202514648f, x);  // float(2 pi)
  r = fmaf(-n, -1.7484555314695172e-7f, r);      // 2 pi - float(2 pi)
  return __builtin_amdgcn_sinf(r * 0.15915494309189535f);
}

template <int HF, typename TS>
__global__ void __launch_bounds__(64 * kSynthWaves) siren_synth(SynthArgs a) {
  constexpr int OT = HF / 32;  // 32-unit tiles of the hidden width
  const int lane = threadIdx.x & 63, g = lane >> 5, pl = lane & 31;
  const int64_t tiles = (a.npos + 31) / 32;
  const int64_t tile = (int64_t)blockIdx.x * kSynthWaves + (threadIdx.x >> 6);
  if (tile >= tiles * a.nb) return;  // uniform across the wave
  const int64_t b = tile / tiles;
  const int64_t p = (tile - b * tiles) * 32 + pl;
  const bool valid = p < a.npos;

  // coordinates of grid point p (last axis fastest)
  float r[3] = {0.f, 0.f, 0.f};
  {
    int64_t q = valid ? p : 0;
    for (int d = a.nd - 1; d >= 0; --d) {
      const int64_t i = q % a.KL[d];
      q /= a.KL[d];
      const int64_t L = a.Lc[d];
      int64_t disp = i;
      if (a.mode == 2) disp = i - (L - 1);
      else if (a.mode == 1 && i > L / 2) disp = i - L;
      r[d] = L > 1 ? (float)disp / (float)(L - 1) : 0.f;
    }
  }
  const float* gam = a.gamma ? a.gamma + b * a.J * HF : nullptr;
  const float* bet = a.beta ? a.beta + b * a.J * HF : nullptr;

  // layer 1 straight into the operand layout
  float h[OT][16];
#pragma unroll
  for (int t = 0; t < OT; ++t)
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int o = t * 32 + tile_unit(e, g);
      float s = 0.f;
      for (int d = 0; d < a.nd; ++d) s = fmaf(r[d], a.W1[d * HF + o], s);
      s = fmaf(a.omega0[o], s, a.bias ? a.bias[o] : 0.f);
      float v = sin_reduced(s);
      if (gam) v = fmaf(gam[o], v, bet[o]);
      h[t][e] = v;
    }

  // hidden layers 2 .. J on the matrix cores
  for (int j = 1; j < a.J; ++j) {
    const float* W = a.Wh + (int64_t)(j - 1) * HF * HF;
    v16f acc[OT];
#pragma unroll
    for (int t = 0; t < OT; ++t) acc[t] = v16f{};
#pragma unroll
    for (int kt = 0; kt < OT; ++kt)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const float* Wk = W + (kt * 32 + tile_unit(e, g)) * HF + pl;
#pragma unroll
        for (int t = 0; t < OT; ++t)
          acc[t] = __builtin_amdgcn_mfma_f32_32x32x2f32(Wk[t * 32], h[kt][e], acc[t], 0, 0, 0);
      }
#pragma unroll
    for (int t = 0; t < OT; ++t)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int o = t * 32 + tile_unit(e, g);
        float v = sin_reduced(acc[t][e] + (a.bias ? a.bias[j * HF + o] : 0.f));
        if (gam) v = fmaf(gam[j * HF + o], v, bet[j * HF + o]);
        h[t][e] = v;
      }
  }

  // output projection, window, store: 32 channels per step
  const int C = a.C;
  TS* out = reinterpret_cast<TS*>(a.k) + b * C * a.npos;
  float rr[3], ra = 0.f;
  for (int d = 0; d < 3; ++d) {
    rr[d] = r[d] * r[d];
    ra += fabsf(r[d]);
  }
  for (int c0 = 0; c0 < C; c0 += 32) {
    const bool cok = c0 + pl < C;
    const float* Wc = a.Wout + c0 + pl;
    v16f acc = v16f{};
#pragma unroll
    for (int kt = 0; kt < OT; ++kt)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const float w = cok ? Wc[(int64_t)(kt * 32 + tile_unit(e, g)) * C] : 0.f;
        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(w, h[kt][e], acc, 0, 0, 0);
      }
    if (valid) {
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int c = c0 + tile_unit(e, g);
        if (c < C) {
          float ex;
          if (a.wkind == 0) {
            ex = 0.f;
            for (int d = 0; d < a.nd; ++d) {
              const float s = a.win[d * C + c];
              ex = fmaf(rr[d], __fdividef(-0.5f, s * s), ex);
            }
          } else {
            ex = -a.win[c] * ra;
          }
          st1(out + (int64_t)c * a.npos + p, __expf(ex) * acc[e]);
        }
      }
    }
  }
}

template <typename TS>
hipError_t launch_typed(const SynthArgs& a, hipStream_t s) {
  const int64_t waves = (a.npos + 31) / 32 * a.nb;
  const dim3 grid((unsigned)((waves + kSynthWaves - 1) / kSynthWaves)), block(64 * kSynthWaves);
  switch (a.hidden) {
    case 32: hipLaunchKernelGGL((siren_synth<32, TS>), grid, block, 0, s, a); break;
    case 64: hipLaunchKernelGGL((siren_synth<64, TS>), grid, block, 0, s, a); break;
    case 128: hipLaunchKernelGGL((siren_synth<128, TS>), grid, block, 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

bool synth_hidden_supported(int hidden) { return hidden == 32 || hidden == 64 || hidden == 128; }

hipError_t launch_synth(const SynthArgs& a, bool bf16, hipStream_t s) {
  return bf16 ? launch_typed<uint16_t>(a, s) : launch_typed<float>(a, s);
}

}  // namespace hyenand
