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

// w, w s, w s^2, ... (E values): twiddles of one lane by recurrence
template <int E>
__device__ __forceinline__ void twiddle_run(float2 (&v)[E], float2 w, float2 s) {
#pragma unroll
  for (int e = 0; e < E; ++e) {
    v[e] = c_mul(v[e], w);
    w = c_mul(w, s);
  }
}

inline int ilog2_rt(int64_t n) {
  int r = 0;
  while ((int64_t(1) << r) < n) ++r;
  return r;
}

}  // namespace
}  // namespace hyenand
