// Shapes shared by the four-step 1D forward and backward plans: the packed
// complex line of M = P/2 points is split as M = N1 x N2 with N2 = 2048 and
// 8 <= N1 <= 1024; column passes move tiles of TL adjacent columns.
#pragma once

#include "kernels.hpp"

namespace hyenand {
namespace {

constexpr int kN2 = 2048;
constexpr int kMinN1 = 8;
constexpr int kMaxN1 = 1024;

// column tiles: TL adjacent columns of one signal, N1 points each; TL is the
// widest power of two (<= 32) whose tile fits in ~75 KB of LDS, E is chosen
// so the tile keeps 512 lanes busy when it can.
constexpr int fs_tl(int N1) {
  int tl = 32;
  while (tl > 1 && N1 * (tl + 1) * 8 > 76 * 1024) tl /= 2;
  return tl;
}
template <int N1>
struct ColCfg {
  static constexpr int NT = 512;
  static constexpr int TL = fs_tl(N1);
  static constexpr int E = imax(imin(16, N1), imin(N1, imax(2, (N1 * TL) / NT)));
  static constexpr int T = N1 / E;
  static constexpr int TLP = TL + 1;
};

// The forward and inverse column passes with 512-point columns (and the
// backward's forward column pass): 1024 lanes of 8 points on the same
// 16-column tiles, so that two workgroups per CU (the LDS limit) keep 32
// wavefronts, and twice the memory requests, in flight.  Same TL as ColCfg.
template <int N1>
struct ColCfgFwd : ColCfg<N1> {
  static constexpr int kWaves = 4;  // per SIMD, for amdgpu_waves_per_eu
};
template <>
struct ColCfgFwd<512> {
  static constexpr int NT = 1024;
  static constexpr int TL = 16;
  static constexpr int E = 8;
  static constexpr int T = 512 / E;
  static constexpr int TLP = TL + 1;
  static constexpr int kWaves = 8;
  static_assert(TL * T == NT, "every lane busy");
};

// w, w s, w s^2, ... (E values): twiddles of one lane by recurrence
template <int E>
__device__ __forceinline__ void twiddle_run(float2 (&v)[E], float2 w, float2 s) {
#pragma unroll
  for (int e = 0; e < E; ++e) {
    v[e] = c_mul(v[e], w);
    w = c_mul(w, s);
  }
}

// Workgroup numbering of the column passes over NSIG signals: the logical
// index b' = NSIG rest + sig (rest = line * ntile + tile) would put the tiles
// 2q and 2q + 1 of one signal, which share every 128-byte row run of a
// 16-column bf16 tile (64 bytes each), on different XCDs.  Workgroup b runs
// on XCD b mod 8, so pairing b and b + 8 (one XCD, consecutive slots) on those
// two tiles fetches each run once, while workgroups near in b stay near in
// rest.  A bijection of [0, n) when n is a multiple of 16 NSIG and ntile is
// even.  Used by fs_cols_fwd (u, k) and fsb_cols_inv; in the three-signal
// fsb_cols_fwd the same numbering measured slower than the plain one.
template <uint32_t NSIG>
__device__ __forceinline__ uint32_t fs_pair_tiles(uint32_t b) {
  const uint32_t s = b >> 3, x = b & 7u, h = s & 1u;
  const uint32_t g = (s >> 1) * 8u + x;
  return ((g / NSIG) * 2u + h) * NSIG + g % NSIG;
}

inline int ilog2_rt(int64_t n) {
  int r = 0;
  while ((int64_t(1) << r) < n) ++r;
  return r;
}

}  // namespace
}  // namespace hyenand
