// Backward of the centred mode and of extents that are not powers of two
// through the circular backward on their transform grid.
//
// These calls are a non-circular convolution computed on a grid of P_d >=
// 2 L_d - 1 points per axis (a power of two): u is zero beyond its L_d
// points, the kernel sits at its displacements taken modulo P_d (index m of a
// linear kernel at m; index i of a centred kernel, displacement
// i - (L_d - 1), at that displacement mod P_d; a circular kernel of other
// extents, repeated periodically, at displacements -(L_d - 1) .. L_d - 1).
// On that grid the operation is exactly the circular one of the embedded
// tensors, and so is its backward: the correlations gu and gk of the circular
// backward never wrap onto a nonzero value because P_d >= 2 L_d - 1.  The
// periodic kernel's gradient gathers the two displacements m and m - L_d that
// hold k[m] (m >= 1) on every axis.  So
//
//   embed     x1, x2, v, gy into the first L_d points of every axis of a
//             P-grid (zeros elsewhere), k at its displacements;
//   circular backward on the P-grid (every plan of the circular mode);
//   (the forward of shapes without a single-pass plan takes the same route:
//   x1, x2, v and k embedded, the circular forward, y extracted)
//   extract   gx1, gx2, gv from the first L_d points, gk from the kernel's
//             displacements; gD comes straight from the circular backward
//             (the zeros add nothing).
//
// Grid extents are powers of two, so indices split with shifts.
#include "kernels.hpp"

namespace hyenand {

namespace {

struct EmbedGeom {
  int nd;
  int lp[3];      // log2 P_d
  int64_t L[3];   // data extents
  int64_t KL[3];  // kernel extents: L_d, or 2 L_d - 1 centred
  int64_t grid;   // prod P_d
  int64_t box;    // prod L_d
  int64_t kbox;   // prod KL_d
  bool centered;
  bool periodic;  // circular kernel repeated over the displacements -(L-1) .. L-1
};

EmbedGeom embed_geom(const FftConvArgs& a) {
  EmbedGeom g;
  g.nd = a.ndim;
  g.grid = g.box = g.kbox = 1;
  g.centered = a.centered;
  g.periodic = a.periodic;
  for (int d = 0; d < 3; ++d) {
    g.lp[d] = 0;
    g.L[d] = g.KL[d] = 1;
  }
  for (int d = 0; d < a.ndim; ++d) {
    int lp = 0;
    while ((int64_t(1) << lp) < a.P[d]) ++lp;
    g.lp[d] = lp;
    g.L[d] = a.L[d];
    g.KL[d] = a.centered ? 2 * a.L[d] - 1 : a.L[d];
    g.grid *= a.P[d];
    g.box *= a.L[d];
    g.kbox *= g.KL[d];
  }
  return g;
}

// kernel index of grid position q along one axis, or -1 where the kernel has
// no point (linear: q < L; centred and periodic: displacement q or q - P)
__device__ __forceinline__ int64_t kernel_pos(int64_t q, int64_t L, int64_t P, bool centered, bool periodic) {
  if (periodic) return q < L ? q : (q > P - L ? q - P + L : -1);
  if (!centered) return q < L ? q : -1;
  return q < L ? q + L - 1 : (q > P - L ? q - P + L - 1 : -1);
}

template <typename TS>
__global__ void __launch_bounds__(256)
    embed_inputs(const TS* __restrict__ x1, const TS* __restrict__ x2, const TS* __restrict__ v,
                 const TS* __restrict__ gy, const TS* __restrict__ k, TS* __restrict__ ex1, TS* __restrict__ ex2,
                 TS* __restrict__ ev, TS* __restrict__ egy, TS* __restrict__ ek, EmbedGeom g, int64_t total,
                 bool shared_k, int64_t C) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= total) return;
  const int64_t line = i >> (g.lp[0] + g.lp[1] + g.lp[2]);
  int64_t r = i & (g.grid - 1);
  int64_t src = 0, ksrc = 0;
  bool in = true, kin = true;
  for (int d = 0; d < g.nd; ++d) {
    const int sh = (d + 1 < g.nd ? g.lp[d + 1] : 0) + (d + 2 < g.nd ? g.lp[d + 2] : 0);
    const int64_t q = r >> sh;
    r &= (int64_t(1) << sh) - 1;
    const int64_t P = int64_t(1) << g.lp[d];
    in = in && q < g.L[d];
    src = src * g.L[d] + (q < g.L[d] ? q : 0);
    const int64_t kp = kernel_pos(q, g.L[d], P, g.centered, g.periodic);
    kin = kin && kp >= 0;
    ksrc = ksrc * g.KL[d] + (kp >= 0 ? kp : 0);
  }
  const int64_t s = line * g.box + src;
  const TS zero{};
  ex1[i] = in ? x1[s] : zero;
  ex2[i] = in ? x2[s] : zero;
  ev[i] = in ? v[s] : zero;
  if (egy) egy[i] = in ? gy[s] : zero;  // the backward's gy (none for the forward)
  ek[i] = kin ? k[(shared_k ? line % C : line) * g.kbox + ksrc] : zero;
}

// gx1, gx2, gv (or the forward's y alone) back from the first L_d points of
// every axis
template <typename TS>
__global__ void __launch_bounds__(256)
    extract_data(const TS* __restrict__ e1, const TS* __restrict__ e2, const TS* __restrict__ e3,
                 TS* __restrict__ o1, TS* __restrict__ o2, TS* __restrict__ o3, EmbedGeom g, int64_t total) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= total) return;
  const int64_t line = i / g.box;
  int64_t r = i - line * g.box, q[3] = {0, 0, 0};
  for (int d = g.nd - 1; d >= 0; --d) {
    q[d] = r % g.L[d];
    r /= g.L[d];
  }
  int64_t e = line;
  for (int d = 0; d < g.nd; ++d) e = (e << g.lp[d]) + q[d];
  o1[i] = e1[e];
  if (o2) o2[i] = e2[e];
  if (o3) o3[i] = e3[e];
}

// gk back from the kernel's displacements (periodic: the sum over the one or
// two displacements of every axis that hold the point, in a fixed order)
template <typename TS>
__global__ void __launch_bounds__(256)
    extract_kernel(const TS* __restrict__ ek, TS* __restrict__ gk, EmbedGeom g, int64_t total) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= total) return;
  const int64_t line = i / g.kbox;
  int64_t r = i - line * g.kbox, q[3] = {0, 0, 0}, q2[3] = {-1, -1, -1};
  for (int d = g.nd - 1; d >= 0; --d) {
    const int64_t m = r % g.KL[d];
    r /= g.KL[d];
    const int64_t P = int64_t(1) << g.lp[d];
    q[d] = g.centered ? (m - (g.L[d] - 1) + P) & (P - 1) : m;
    if (g.periodic && m >= 1) q2[d] = m - g.L[d] + P;  // displacement m - L
  }
  float acc = 0.f;
  const int nc = g.periodic ? 1 << g.nd : 1;
  for (int cmb = 0; cmb < nc; ++cmb) {
    int64_t e = line;
    bool ok = true;
    for (int d = 0; d < g.nd; ++d) {
      const int64_t qd = (cmb >> d) & 1 ? q2[d] : q[d];
      ok = ok && qd >= 0;
      e = (e << g.lp[d]) + (qd >= 0 ? qd : 0);
    }
    if (ok) acc += ld1(ek + e);
  }
  st1(gk + i, acc);
}

unsigned blocks(int64_t n) { return (unsigned)((n + 255) / 256); }

}  // namespace

int64_t embed_grid_elems(const FftConvArgs& a) { return a.lines * embed_geom(a).grid; }

hipError_t launch_embed(const FftConvArgs& a, const void* gy, void* const (&e)[5], hipStream_t s) {
  const EmbedGeom g = embed_geom(a);
  const int64_t total = a.lines * g.grid;
  const bool shared = a.kC != 0;
  if (a.bf16) {
    using T = uint16_t;
    hipLaunchKernelGGL(embed_inputs<T>, dim3(blocks(total)), dim3(256), 0, s, (const T*)a.x1, (const T*)a.x2,
                       (const T*)a.v, (const T*)gy, (const T*)a.k, (T*)e[0], (T*)e[1], (T*)e[2], (T*)e[3], (T*)e[4],
                       g, total, shared, a.C);
  } else {
    using T = float;
    hipLaunchKernelGGL(embed_inputs<T>, dim3(blocks(total)), dim3(256), 0, s, (const T*)a.x1, (const T*)a.x2,
                       (const T*)a.v, (const T*)gy, (const T*)a.k, (T*)e[0], (T*)e[1], (T*)e[2], (T*)e[3], (T*)e[4],
                       g, total, shared, a.C);
  }
  return hipGetLastError();
}

hipError_t launch_embed_fwd(const FftConvArgs& a, void* const (&e)[4], hipStream_t s) {
  const EmbedGeom g = embed_geom(a);
  const int64_t total = a.lines * g.grid;
  const bool shared = a.kC != 0;
  if (a.bf16) {
    using T = uint16_t;
    hipLaunchKernelGGL(embed_inputs<T>, dim3(blocks(total)), dim3(256), 0, s, (const T*)a.x1, (const T*)a.x2,
                       (const T*)a.v, (const T*)nullptr, (const T*)a.k, (T*)e[0], (T*)e[1], (T*)e[2], (T*)nullptr,
                       (T*)e[3], g, total, shared, a.C);
  } else {
    using T = float;
    hipLaunchKernelGGL(embed_inputs<T>, dim3(blocks(total)), dim3(256), 0, s, (const T*)a.x1, (const T*)a.x2,
                       (const T*)a.v, (const T*)nullptr, (const T*)a.k, (T*)e[0], (T*)e[1], (T*)e[2], (T*)nullptr,
                       (T*)e[3], g, total, shared, a.C);
  }
  return hipGetLastError();
}

hipError_t launch_extract_y(const FftConvArgs& a, const void* ey, void* y, hipStream_t s) {
  const EmbedGeom g = embed_geom(a);
  const int64_t nd = a.lines * g.box;
  if (a.bf16) {
    using T = uint16_t;
    hipLaunchKernelGGL(extract_data<T>, dim3(blocks(nd)), dim3(256), 0, s, (const T*)ey, (const T*)nullptr,
                       (const T*)nullptr, (T*)y, (T*)nullptr, (T*)nullptr, g, nd);
  } else {
    using T = float;
    hipLaunchKernelGGL(extract_data<T>, dim3(blocks(nd)), dim3(256), 0, s, (const T*)ey, (const T*)nullptr,
                       (const T*)nullptr, (T*)y, (T*)nullptr, (T*)nullptr, g, nd);
  }
  return hipGetLastError();
}

hipError_t launch_extract(const FftConvArgs& a, void* const (&e)[4], void* gx1, void* gx2, void* gv, void* gk,
                          hipStream_t s) {
  const EmbedGeom g = embed_geom(a);
  const int64_t nd = a.lines * g.box, nk = a.lines * g.kbox;
  if (a.bf16) {
    using T = uint16_t;
    hipLaunchKernelGGL(extract_data<T>, dim3(blocks(nd)), dim3(256), 0, s, (const T*)e[0], (const T*)e[1],
                       (const T*)e[2], (T*)gx1, (T*)gx2, (T*)gv, g, nd);
    hipLaunchKernelGGL(extract_kernel<T>, dim3(blocks(nk)), dim3(256), 0, s, (const T*)e[3], (T*)gk, g, nk);
  } else {
    using T = float;
    hipLaunchKernelGGL(extract_data<T>, dim3(blocks(nd)), dim3(256), 0, s, (const T*)e[0], (const T*)e[1],
                       (const T*)e[2], (T*)gx1, (T*)gx2, (T*)gv, g, nd);
    hipLaunchKernelGGL(extract_kernel<T>, dim3(blocks(nk)), dim3(256), 0, s, (const T*)e[3], (T*)gk, g, nk);
  }
  return hipGetLastError();
}

}  // namespace hyenand
