// Kernel synthesis on the matrix cores: the HyenaND kernel K(x) = w(r) *
// f_theta(r; z(x)) evaluated on the kernel grid of a convolution
// (section 3.2.1, Eq. (kernel): a SIREN over the normalised grid coordinates;
// section 3.2.2, Eq. (film): per-sample scales and shifts after every hidden
// sine; the masking appendix, Eq. (mask): the per-axis Gaussian window, or
// the exponential decay of the original Hyena).
//
// The hidden layers and the output projection are dense contractions over the
// hidden width Hf, so they run on v_mfma_f32_16x16x4_f32 (fp32 in, fp32
// accumulate).  One wave owns 16 grid points of one sample and carries them
// through every layer without leaving registers: the product is taken
// transposed, out[unit, point] = sum_k W[k, unit] h[point, k], so the points
// are the 16 columns (lane % 16) and the units the 16 rows of each tile.  The
// accumulator layout of a tile (lane l, register r: row 4 (l / 16) + r,
// column l % 16) already is the operand layout of the next layer, because a
// contraction may visit its k index in any order: at step r of a 16-unit
// block the four lane groups contribute units 4 g + r (g = l / 16), and the
// weight operand is read for exactly those units.  The weights sit in LDS,
// transposed (row = output unit or channel), so that the four steps of a
// block take one 16-byte read per lane.  Points' coordinates are generated
// from their index; K is written once.
//
// For a bf16 kernel tensor the products run on v_mfma_f32_16x16x32_bf16
// instead (weights and activations rounded to bf16, fp32 accumulate; the
// sines, FiLM and window stay fp32): step s of the contraction takes units
// (2 s + hi) * 16 + 4 g + r (hi, r < 2, 4) from lane group g, i.e. two of the
// lane's own register quads, and the weights sit in LDS as bf16 in that
// order, eight per 16-byte read.
#include <algorithm>
#include <mutex>

#include "kernels.hpp"

namespace hyenand {

namespace {

typedef float v4f __attribute__((ext_vector_type(4)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));

constexpr int kSynthWaves = 8;  // waves per workgroup, one 16-point tile each
constexpr int kThreads = 64 * kSynthWaves;
constexpr float kLog2e = 1.4426950408889634f;

// sin(x): two-constant Cody-Waite reduction to [-pi, pi], then the hardware
// sine (which takes its argument in turns)
__device__ __forceinline__ float sin_reduced(float x) {
  const float n = rintf(x * 0.15915494309189535f);
  float r = fmaf(-n, 6.28318548202514648f, x);  // float(2 pi)
  r = fmaf(-n, -1.7484555314695172e-7f, r);      // 2 pi - float(2 pi)
  return __builtin_amdgcn_sinf(r * 0.15915494309189535f);
}

// LDS layout (floats).  A parameter block at 0: omega0 [HF], W1 [3][HF] (rows
// past N zero), bias [J][HF] (zero without biases).  Then the matrices,
// transposed (row = output unit or channel, row stride HF + 4 floats: the pad
// spreads consecutive rows over the banks).  With every weight resident:
// W_2 .. W_J back to back (HF rows each), then Wout (ldo rows, zero past the
// last channel) and the window exponents q [3][ldo]; streamed, one region
// that holds one hidden matrix or a chunk of ldo = cc output channels at a
// time.  The window exponent of channel c on axis d is q[d][c] s_d, with
// s_d = r_d^2 and q = -log2(e) / (2 sigma^2) for the Gaussian, s_d = |r_d|
// and q = -log2(e) alpha for the exponential, so that
// w = 2^(sum_d q[d][c] s_d).
__device__ __forceinline__ int par_floats(int HF, int J) { return (4 + J) * HF; }

__device__ void stage_params(const SynthArgs& a, float* lds, int HF) {
  for (int i = threadIdx.x; i < par_floats(HF, a.J); i += kThreads) {
    float v = 0.f;
    if (i < HF) v = a.omega0[i];
    else if (i < 4 * HF) {
      const int d = i / HF - 1;
      if (d < a.nd) v = a.W1[d * HF + i % HF];
    } else if (a.bias) {
      v = a.bias[i - 4 * HF];
    }
    lds[i] = v;
  }
}

// Staging: wave w copies rows w, w + 8, ... of a matrix for 64 consecutive
// output columns at a time, one column per lane: global reads coalesced, no
// division, HF / 8 loads in flight per lane before its LDS stores.
// Row stride (in floats) of a staged matrix: HF fp32 values + 4, or HF bf16
// values + 8 (16 bytes of pad either way).
template <int HF, bool BF>
constexpr int row_floats() {
  return BF ? HF / 2 + 4 : HF + 4;
}

// Position of input unit k within a bf16 row: step s = k / 32 of the
// contraction, lane group g = (k % 16) / 4, then the unit's quad (hi = which
// 16-unit block of the step) and r = k % 4.
__device__ __forceinline__ int bf_pos(int k) { return (k >> 5) * 32 + ((k >> 2) & 3) * 8 + ((k >> 4) & 1) * 4 + (k & 3); }

// value v of input unit k in row o of a staged matrix
template <int HF, bool BF>
__device__ __forceinline__ void stage_put(float* dst, int o, int k, float v) {
  if constexpr (BF) {
    reinterpret_cast<__bf16*>(dst)[o * 2 * row_floats<HF, BF>() + bf_pos(k)] = (__bf16)v;
  } else {
    dst[o * row_floats<HF, BF>() + k] = v;
  }
}

// W_j [k][o] -> dst[o][k]
template <int HF, bool BF>
__device__ void stage_hidden(const SynthArgs& a, float* dst, int j) {
  const float* W = a.Wh + (int64_t)(j - 1) * HF * HF;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
  for (int o0 = 0; o0 < HF; o0 += 64) {
    const int o = o0 + lane;
    if (o < HF) {
      float v[HF / kSynthWaves];
#pragma unroll
      for (int kk = 0; kk < HF / kSynthWaves; ++kk) v[kk] = W[(w + kSynthWaves * kk) * HF + o];
#pragma unroll
      for (int kk = 0; kk < HF / kSynthWaves; ++kk) stage_put<HF, BF>(dst, o, w + kSynthWaves * kk, v[kk]);
    }
  }
}

// window exponents of channels c0 .. c0 + n - 1 -> q[3][ld] (zero past n)
__device__ void stage_q(const SynthArgs& a, float* q, int c0, int n, int ld) {
  const int C = a.C;
  for (int i = threadIdx.x; i < 3 * ld; i += kThreads) {
    const int d = i / ld, c = i - d * ld;
    float v = 0.f;
    if (c < n && d < a.nd) {
      if (a.wkind == 0) {
        const float sg = a.win[d * C + c0 + c];
        v = -0.5f * kLog2e / (sg * sg);
      } else {
        v = -kLog2e * a.win[c0 + c];
      }
    }
    q[i] = v;
  }
}

// Wout[:, c0 : c0 + n] -> dst[c][k] for c < ld (ld a multiple of 64; rows
// past n zero), then q[3][ld]
template <int HF, bool BF>
__device__ void stage_out(const SynthArgs& a, float* dst, int c0, int n, int ld) {
  const int C = a.C;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  for (int cb = 0; cb < ld; cb += 64) {
    const int c = cb + lane;
    const bool in = c < n;
    const float* src = a.Wout + c0 + (in ? c : 0);
    float v[HF / kSynthWaves];
#pragma unroll
    for (int kk = 0; kk < HF / kSynthWaves; ++kk) v[kk] = in ? src[(int64_t)(w + kSynthWaves * kk) * C] : 0.f;
#pragma unroll
    for (int kk = 0; kk < HF / kSynthWaves; ++kk) stage_put<HF, BF>(dst, c, w + kSynthWaves * kk, v[kk]);
  }
  stage_q(a, dst + ld * row_floats<HF, BF>(), c0, n, ld);
}

// FiLM scale and shift of layer j for this lane's units t * 16 + 4 g + r,
// from src = gamma and beta of every sample, interleaved per (b, j) as
// [gamma row, beta row] (LDS copy) or from the caller's arrays
template <int HF, bool FILM>
__device__ __forceinline__ void film_load(const SynthArgs& a, const float* film_lds, int64_t b, int j, int g,
                                          v4f (&gm)[HF / 16], v4f (&bt)[HF / 16]) {
  if constexpr (FILM) {
    const float *G, *Bt;
    if (film_lds) {
      G = film_lds + (b * a.J + j) * 2 * HF + 4 * g;
      Bt = G + HF;
    } else {
      G = a.gamma + (b * a.J + j) * HF + 4 * g;
      Bt = a.beta + (b * a.J + j) * HF + 4 * g;
    }
#pragma unroll
    for (int t = 0; t < HF / 16; ++t) {
      gm[t] = *reinterpret_cast<const v4f*>(G + t * 16);
      bt[t] = *reinterpret_cast<const v4f*>(Bt + t * 16);
    }
  }
}

// NT output tiles of 16 rows (weights in LDS at rows[i] = this lane's row of
// tile i): acc[i] = sum over the hidden width of weight x activation; the
// products of the NT tiles alternate, the operands of one 16-unit block are
// read one block ahead
template <int HF, int NT>
__device__ __forceinline__ void chains(const float* const (&rows)[NT], const v4f (&h)[HF / 16], int g, v4f (&acc)[NT]) {
  v4f w[2][NT];
#pragma unroll
  for (int i = 0; i < NT; ++i) {
    acc[i] = v4f{};
    w[0][i] = *reinterpret_cast<const v4f*>(rows[i] + 4 * g);
  }
#pragma unroll
  for (int kt = 0; kt < HF / 16; ++kt) {
    if (kt + 1 < HF / 16)
#pragma unroll
      for (int i = 0; i < NT; ++i) w[(kt + 1) & 1][i] = *reinterpret_cast<const v4f*>(rows[i] + (kt + 1) * 16 + 4 * g);
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
      for (int i = 0; i < NT; ++i) acc[i] = __builtin_amdgcn_mfma_f32_16x16x4f32(w[kt & 1][i][r], h[kt][r], acc[i], 0, 0, 0);
  }
}

// the same on the bf16 matrix cores: hb[s] holds the lane's units of step s
// (register quads 2 s and 2 s + 1) in bf16; rows[i] points at this lane's
// bf16 row of tile i
template <int HF, int NT>
__device__ __forceinline__ void chains_bf(const float* const (&rows)[NT], const v8bf (&hb)[HF / 32], int g,
                                          v4f (&acc)[NT]) {
  v8bf w[2][NT];
#pragma unroll
  for (int i = 0; i < NT; ++i) {
    acc[i] = v4f{};
    w[0][i] = *reinterpret_cast<const v8bf*>(reinterpret_cast<const __bf16*>(rows[i]) + 8 * g);
  }
#pragma unroll
  for (int st = 0; st < HF / 32; ++st) {
    if (st + 1 < HF / 32)
#pragma unroll
      for (int i = 0; i < NT; ++i)
        w[(st + 1) & 1][i] = *reinterpret_cast<const v8bf*>(reinterpret_cast<const __bf16*>(rows[i]) + (st + 1) * 32 + 8 * g);
#pragma unroll
    for (int i = 0; i < NT; ++i) acc[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w[st & 1][i], hb[st], acc[i], 0, 0, 0);
  }
}

template <int HF>
__device__ __forceinline__ void to_bf(const v4f (&h)[HF / 16], v8bf (&hb)[HF / 32]) {
#pragma unroll
  for (int st = 0; st < HF / 32; ++st)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      hb[st][r] = (__bf16)h[2 * st][r];
      hb[st][4 + r] = (__bf16)h[2 * st + 1][r];
    }
}

// NT output tiles through the fp32 or the bf16 products
template <int HF, int NT, bool BF>
__device__ __forceinline__ void tile_products(const float* const (&rows)[NT], const v4f (&h)[HF / 16], const v8bf (&hb)[HF / 32],
                                      int g, v4f (&acc)[NT]) {
  if constexpr (BF) chains_bf<HF, NT>(rows, hb, g, acc);
  else chains<HF, NT>(rows, h, g, acc);
}

// window and store of one 16-channel tile: channels cb + 4 g + r of point p
// (CHECK: skip channels at or past n; tbase points at channel c0)
template <typename TS, bool CHECK>
__device__ __forceinline__ void store_tile(const v4f& acc, TS* tbase, int64_t npos, int64_t p, const float* q, int ld,
                                           int cb, int n, int g, const float (&sd)[3]) {
  const int cr = cb + 4 * g;
  const v4f q0 = *reinterpret_cast<const v4f*>(q + cr);
  const v4f q1 = *reinterpret_cast<const v4f*>(q + ld + cr);
  const v4f q2 = *reinterpret_cast<const v4f*>(q + 2 * ld + cr);
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    if (!CHECK || cr + r < n) {
      const float ex = fmaf(q2[r], sd[2], fmaf(q1[r], sd[1], q0[r] * sd[0]));
      st1(tbase + (int64_t)(cr + r) * npos + p, __builtin_amdgcn_exp2f(ex) * acc[r]);
    }
  }
}

template <int HF, bool FILM, typename TS, bool BF>
__global__ void __launch_bounds__(kThreads) siren_synth(SynthArgs a) {
  constexpr int OT = HF / 16;  // 16-unit blocks of the hidden width
  constexpr int LDW = row_floats<HF, BF>();  // row stride of a staged matrix
  constexpr int NT = HF >= 128 ? 2 : 4;  // output tiles per group
  extern __shared__ float lds[];
  const int lane = threadIdx.x & 63, g = lane >> 4, pl = lane & 15;
  const int wave = threadIdx.x >> 6;
  const int J = a.J, C = a.C;
  const int64_t tiles = (a.npos + 15) / 16;
  const int64_t total = tiles * a.nb;
  const int M0 = (par_floats(HF, J) + 3) & ~3;
  const bool resident = a.resident;
  const int ldo = resident ? (C + 63) & ~63 : a.cc;  // staged output channels
  const int out_off = M0 + (resident ? (J - 1) * HF * LDW : 0);

  // FiLM of every sample in LDS when the launch reserved room for it
  const float* film_lds = nullptr;
  if (FILM && a.film_lds) {
    float* f = lds + out_off + (resident ? ldo * (LDW + 3) : a.stream_floats);
    for (int i = threadIdx.x; i < (int)(a.nb * J * HF); i += kThreads) {
      const int row = i / HF, u = i - row * HF;  // row = b * J + j
      f[row * 2 * HF + u] = a.gamma[i];
      f[row * 2 * HF + HF + u] = a.beta[i];
    }
    film_lds = f;
  }
  stage_params(a, lds, HF);
  if (resident) {
    for (int j = 1; j < J; ++j) stage_hidden<HF, BF>(a, lds + M0 + (j - 1) * HF * LDW, j);
    stage_out<HF, BF>(a, lds + out_off, 0, C, ldo);
  }
  __syncthreads();

  for (int64_t base = (int64_t)blockIdx.x * kSynthWaves; base < total; base += (int64_t)gridDim.x * kSynthWaves) {
    const int64_t tile = base + wave;
    const bool live = tile < total;  // uniform across the wave
    const int64_t b = live ? tile / tiles : 0;
    const int64_t p0 = (tile - b * tiles) * 16;  // first point of the tile
    const int64_t p = p0 + pl;
    const bool valid = live && p < a.npos;

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

    // layer 1 straight into the operand layout: h[t][r] is unit t * 16 +
    // 4 g + r of point p
    v4f h[OT];
    if (live) {
      v4f gm[OT], bt[OT];
      film_load<HF, FILM>(a, film_lds, b, 0, g, gm, bt);
#pragma unroll
      for (int t = 0; t < OT; ++t)
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const int o = t * 16 + 4 * g + k;
          float s = r[0] * lds[HF + o];
          s = fmaf(r[1], lds[2 * HF + o], s);
          s = fmaf(r[2], lds[3 * HF + o], s);
          float v = sin_reduced(fmaf(lds[o], s, lds[4 * HF + o]));
          if constexpr (FILM) v = fmaf(gm[t][k], v, bt[t][k]);
          h[t][k] = v;
        }
    }

    // hidden layers 2 .. J on the matrix cores, weights from LDS
    for (int j = 1; j < J; ++j) {
      const float* W = lds + M0 + (resident ? (j - 1) * HF * LDW : 0);
      if (!resident) {
        __syncthreads();
        stage_hidden<HF, BF>(a, lds + M0, j);
        __syncthreads();
      }
      if (live) {
        v4f gm[OT], bt[OT];
        film_load<HF, FILM>(a, film_lds, b, j, g, gm, bt);
        constexpr int NH = OT < NT ? OT : NT;  // hidden tiles per group
        v4f acc[OT];
        v8bf hb[HF / 32];
        if constexpr (BF) to_bf<HF>(h, hb);
#pragma unroll
        for (int t0 = 0; t0 < OT; t0 += NH) {
          const float* rows[NH];
          v4f part[NH];
#pragma unroll
          for (int i = 0; i < NH; ++i) rows[i] = W + ((t0 + i) * 16 + pl) * LDW;
          tile_products<HF, NH, BF>(rows, h, hb, g, part);
#pragma unroll
          for (int i = 0; i < NH; ++i) acc[t0 + i] = part[i];
        }
        const float* bias = lds + (4 + j) * HF;
#pragma unroll
        for (int t = 0; t < OT; ++t)
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            float v = sin_reduced(acc[t][k] + bias[t * 16 + 4 * g + k]);
            if constexpr (FILM) v = fmaf(gm[t][k], v, bt[t][k]);
            h[t][k] = v;
          }
      }
    }

    // output projection, window, store: chunks of staged channels, NT
    // 16-channel tiles per group (rows past the last channel are zero, so
    // every tile of a group exists)
    TS* out = reinterpret_cast<TS*>(a.k) + b * C * a.npos;
    float sd[3];
#pragma unroll
    for (int d = 0; d < 3; ++d) sd[d] = a.wkind == 0 ? r[d] * r[d] : fabsf(r[d]);
    for (int c0 = 0; c0 < C; c0 += ldo) {
      const int n = min(ldo, C - c0);
      if (!resident) {
        __syncthreads();
        stage_out<HF, BF>(a, lds + M0, c0, n, ldo);
        __syncthreads();
      }
      if (!live) continue;
      const float* Wo = lds + out_off;
      const float* q = Wo + ldo * LDW;
      TS* cbase = out + (int64_t)c0 * a.npos;
      const bool full = p0 + 16 <= a.npos && n % (16 * NT) == 0;  // uniform
      v8bf hb[HF / 32];
      if constexpr (BF) to_bf<HF>(h, hb);
      for (int ct = 0; ct < n; ct += 16 * NT) {
        const float* rows[NT];
#pragma unroll
        for (int i = 0; i < NT; ++i) rows[i] = Wo + (ct + 16 * i + pl) * LDW;
        v4f acc[NT];
        tile_products<HF, NT, BF>(rows, h, hb, g, acc);
        if (full) {
#pragma unroll
          for (int i = 0; i < NT; ++i) store_tile<TS, false>(acc[i], cbase, a.npos, p, q, ldo, ct + 16 * i, n, g, sd);
        } else if (valid) {
#pragma unroll
          for (int i = 0; i < NT; ++i) store_tile<TS, true>(acc[i], cbase, a.npos, p, q, ldo, ct + 16 * i, n, g, sd);
        }
      }
    }
  }
}

// LDS floats of a launch: the parameter block plus either every weight
// (resident) or one streamed region, plus the FiLM block when kept in LDS
size_t lds_floats(const SynthArgs& a, bool resident, bool bf) {
  const size_t H = a.hidden, J = a.J, C = ((size_t)a.C + 63) & ~size_t(63), LDW = bf ? H / 2 + 4 : H + 4;
  const size_t par = ((4 + J) * H + 3) & ~size_t(3);
  const size_t film = a.film_lds ? 2 * (size_t)a.nb * J * H : 0;
  if (resident) return par + (J - 1) * H * LDW + (LDW + 3) * C + film;
  return par + (size_t)a.stream_floats + film;
}

constexpr size_t kLdsLimit = 160 * 1024;

// one launch; the kernel's dynamic LDS limit is raised to the CU's 160 KB
// once per kernel
template <typename K>
hipError_t launch_one(K kernel, int64_t grid, dim3 block, size_t bytes, hipStream_t s, const SynthArgs& a) {
  static std::once_flag once;
  static hipError_t attr = hipSuccess;
  std::call_once(once, [&] {
    attr = hipFuncSetAttribute(reinterpret_cast<const void*>(kernel), hipFuncAttributeMaxDynamicSharedMemorySize,
                               (int)kLdsLimit);
  });
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL(kernel, dim3((unsigned)grid), block, bytes, s, a);
  return hipGetLastError();
}

template <typename TS, bool FILM>
hipError_t launch_film(SynthArgs a, hipStream_t s) {
  constexpr bool BF = sizeof(TS) == 2;  // bf16 output: bf16 products
  // stream the weights when they do not all fit next to each other
  a.cc = 64 * std::max(1, (int)(16384 / a.hidden / 64));  // output channels per streamed chunk
  const int LDW = BF ? a.hidden / 2 + 4 : a.hidden + 4;
  a.stream_floats = (int)std::max(a.hidden * LDW, (LDW + 3) * a.cc);
  // FiLM rows of every sample in LDS when they take at most 32 KiB
  a.film_lds = FILM && 2 * a.nb * a.J * a.hidden * 4 <= 32 * 1024;
  const size_t res_bytes = lds_floats(a, true, BF) * 4;
  a.resident = res_bytes <= kLdsLimit - 8 * 1024;
  const size_t bytes = lds_floats(a, a.resident, BF) * 4;
  static int ncu = 0;
  if (ncu == 0) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) !=
                                                  hipSuccess || ncu <= 0)
      ncu = 256;
  }
  const int per_cu = std::max<int>(1, (int)(kLdsLimit / bytes));
  const int64_t groups = ((a.npos + 15) / 16 * a.nb + kSynthWaves - 1) / kSynthWaves;
  const int64_t grid = std::min<int64_t>(groups, (int64_t)ncu * std::min(per_cu, 2));
  const dim3 block(64 * kSynthWaves);
  switch (a.hidden) {
    case 32: return launch_one(siren_synth<32, FILM, TS, BF>, grid, block, bytes, s, a);
    case 64: return launch_one(siren_synth<64, FILM, TS, BF>, grid, block, bytes, s, a);
    case 128: return launch_one(siren_synth<128, FILM, TS, BF>, grid, block, bytes, s, a);
    default: return hipErrorInvalidValue;
  }
}

template <typename TS>
hipError_t launch_typed(const SynthArgs& a, hipStream_t s) {
  return a.gamma ? launch_film<TS, true>(a, s) : launch_film<TS, false>(a, s);
}

}  // namespace

bool synth_hidden_supported(int hidden) { return hidden == 32 || hidden == 64 || hidden == 128; }

hipError_t launch_synth(const SynthArgs& a, bool bf16, hipStream_t s) {
  return bf16 ? launch_typed<uint16_t>(a, s) : launch_typed<float>(a, s);
}

}  // namespace hyenand
