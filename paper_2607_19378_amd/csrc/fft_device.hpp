// Device building blocks for the gated N-D FFT long convolution on gfx950.
//
// * complex fp32 helpers (float2 = re, im);
// * twiddles exp(-2 pi i m / 2^s) from fp32 tables that were computed in fp64
//   (coarse 2^12 table, and coarse x fine for s up to 24);
// * radix-R DFTs held entirely in registers (R <= 32), natural order in and out;
// * BlockFFT<N, E>: a length-N transform carried by T = N/E lanes that each hold
//   E points in registers (lane t holds x[t + T e]).  Passes are Stockham
//   autosort steps of radix min(E, remaining): each pass applies twiddles, a
//   register DFT, and exchanges through LDS; the last pass leaves the output in
//   registers in the same stride-T distribution, so no bit reversal is needed
//   and a transform can feed the next step directly from registers.
//
// Transforms are unnormalised: forward X[f] = sum_n x[n] exp(-2 pi i f n / N),
// inverse uses exp(+2 pi i f n / N).  The scaling by 1/prod(P) of the inverse
// N-D transform is folded into the spectral product by the callers.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hyenand {

#include "twiddles.inc"

constexpr int ilog2(int n) { return n <= 1 ? 0 : 1 + ilog2(n >> 1); }
constexpr int imin(int a, int b) { return a < b ? a : b; }
constexpr int imax(int a, int b) { return a > b ? a : b; }
constexpr bool is_pow2(int n) { return n >= 1 && (n & (n - 1)) == 0; }
constexpr int bitrev(int k, int nbits) {
  int r = 0;
  for (int i = 0; i < nbits; ++i) r |= ((k >> i) & 1) << (nbits - 1 - i);
  return r;
}

// ---------------------------------------------------------------------------
// complex arithmetic
// ---------------------------------------------------------------------------
__device__ __forceinline__ float2 c_add(float2 a, float2 b) { return make_float2(a.x + b.x, a.y + b.y); }
__device__ __forceinline__ float2 c_sub(float2 a, float2 b) { return make_float2(a.x - b.x, a.y - b.y); }
__device__ __forceinline__ float2 c_conj(float2 a) { return make_float2(a.x, -a.y); }
__device__ __forceinline__ float2 c_scale(float2 a, float s) { return make_float2(a.x * s, a.y * s); }
__device__ __forceinline__ float2 c_mul(float2 a, float2 b) {
  return make_float2(fmaf(a.x, b.x, -a.y * b.y), fmaf(a.x, b.y, a.y * b.x));
}
// a * conj(b)
__device__ __forceinline__ float2 c_mulc(float2 a, float2 b) {
  return make_float2(fmaf(a.x, b.x, a.y * b.y), fmaf(a.y, b.x, -a.x * b.y));
}
// quarter turn: * (-i) for the forward direction, * (+i) for the inverse
template <bool INV>
__device__ __forceinline__ float2 c_quarter(float2 a) {
  return INV ? make_float2(-a.y, a.x) : make_float2(a.y, -a.x);
}
__device__ __forceinline__ float2 czero() { return make_float2(0.f, 0.f); }

// ---------------------------------------------------------------------------
// twiddles
// ---------------------------------------------------------------------------
// exp(-2 pi i m / 2^LOG) for 0 <= m < 2^LOG (conjugated when INV), LOG <= 24.
template <int LOG, bool INV>
__device__ __forceinline__ float2 twiddle(uint32_t m) {
  static_assert(LOG >= 0 && LOG <= 24, "twiddle range");
  float2 w;
  if constexpr (LOG <= 12) {
    w = kTwCoarse[m << (12 - LOG)];
  } else {
    const uint32_t b = m << (24 - LOG);
    w = c_mul(kTwCoarse[b >> 12], kTwFine[b & 4095u]);
  }
  return INV ? c_conj(w) : w;
}

// Same with the size known at run time only (log2n <= 24).
template <bool INV>
__device__ __forceinline__ float2 twiddle_rt(uint32_t m, int log2n) {
  float2 w;
  if (log2n <= 12) {
    w = kTwCoarse[m << (12 - log2n)];
  } else {
    const uint32_t b = m << (24 - log2n);
    w = c_mul(kTwCoarse[b >> 12], kTwFine[b & 4095u]);
  }
  return INV ? c_conj(w) : w;
}

// Stockham pass twiddle exp(-+2 pi i jm r / (NS R)) from the [r-1][jm] table
// of that pass shape: lanes with consecutive jm read consecutive entries.
template <int NS, int R, bool INV>
__device__ __forceinline__ float2 pass_twiddle(uint32_t jm, int r) {
  static_assert(NS >= 2 && R >= 2 && R <= 16 && NS * R <= 8192, "pass table range");
  const float2 w = pass_table<ilog2(NS), ilog2(R)>()[(uint32_t)(r - 1) * NS + jm];
  return INV ? c_conj(w) : w;
}

// a * exp(-+2 pi i n / R) with n a compile-time constant after unrolling.
template <int R, bool INV>
__device__ __forceinline__ float2 mul_root(float2 a, int n) {
  n &= (R - 1);
  if (n == 0) return a;
  if (4 * n == R) return c_quarter<INV>(a);
  if (2 * n == R) return make_float2(-a.x, -a.y);
  if (4 * n == 3 * R) return c_quarter<!INV>(a);
  const int j = (n * (32 / R)) & 31;
  const float c = kCos32[j];
  const float s = INV ? kSin32[j] : -kSin32[j];
  return make_float2(fmaf(a.x, c, -a.y * s), fmaf(a.x, s, a.y * c));
}

// ---------------------------------------------------------------------------
// register DFTs
// ---------------------------------------------------------------------------
// Radix-2 decimation in frequency over v[0], v[S], ..., v[(R-1)S]; leaves the
// outputs in bit-reversed slot order.
template <int R, bool INV, int S>
struct DifStages {
  static __device__ __forceinline__ void run(float2* v) {
    if constexpr (R >= 2) {
#pragma unroll
      for (int n = 0; n < R / 2; ++n) {
        const float2 a = v[n * S], b = v[(n + R / 2) * S];
        v[n * S] = c_add(a, b);
        v[(n + R / 2) * S] = mul_root<R, INV>(c_sub(a, b), n);
      }
      if constexpr (R > 2) {
        DifStages<R / 2, INV, S>::run(v);
        DifStages<R / 2, INV, S>::run(v + (R / 2) * S);
      }
    }
  }
};

// In-register DFT of R points, natural order in and out.
template <int R, bool INV>
__device__ __forceinline__ void dft(float2 (&v)[R]) {
  static_assert(is_pow2(R) && R <= 32, "radix");
  if constexpr (R > 1) {
    DifStages<R, INV, 1>::run(v);
    float2 t[R];
#pragma unroll
    for (int k = 0; k < R; ++k) t[k] = v[bitrev(k, ilog2(R))];
#pragma unroll
    for (int k = 0; k < R; ++k) v[k] = t[k];
  }
}

// ---------------------------------------------------------------------------
// LDS scratch addressing for one line of a block transform.
// kKind 1: element p at base[p * S] with S known at compile time;
// kKind 2: element p at base[p + p/16] (one pad slot per 16 entries);
// kKind 0: anything else (address computed per access).
// For kinds 1 and 2 the block transform computes one address per lane and
// reaches the other elements through compile-time offsets.
// ---------------------------------------------------------------------------
template <int S>
struct ScrS {
  static constexpr int kKind = 1;
  float2* base;
  __device__ __forceinline__ float2* operator()(int p) const { return base + p * S; }
};
struct ScrPad16 {
  static constexpr int kKind = 2;
  float2* base;
  __device__ __forceinline__ float2* operator()(int p) const { return base + p + (p >> 4); }
};
struct ScrStrided {  // element p at base[p * stride], stride known at run time
  static constexpr int kKind = 0;
  float2* base;
  int stride;
  __device__ __forceinline__ float2* operator()(int p) const { return base + p * stride; }
};
__host__ __device__ constexpr int pad16_size(int n) { return n + (n >> 4) + 1; }

// Offset, in float2 slots, between position p0 and p0 + d for the layouts
// above; valid only where the caller has checked pad16_step_ok.
template <class Scr, int S_UNUSED = 0>
struct ScrOff;
template <int S>
struct ScrOff<ScrS<S>> {
  static constexpr int off(int d) { return d * S; }
};
template <>
struct ScrOff<ScrPad16> {
  static constexpr int off(int d) { return d + d / 16; }
};

// ---------------------------------------------------------------------------
// Pass twiddles of BlockFFT<N, E> staged in LDS.  When the lanes of a
// wavefront need different twiddles, reading them from the global pass table
// costs a vector-memory round trip per pass; a workgroup instead copies the
// tables of all its passes into LDS once.  Pass (NS, R) keeps rows r = 1..R-1
// ([r-1][jm], as in the global table) when that is at most kFullMax entries,
// else only rows r = 1, 2, 4, 8 ([log2 r][jm]); the other rows are then formed
// as products of those (at most three roundings more).
// ---------------------------------------------------------------------------
template <int N, int E>
struct PassTw {
  static constexpr int kFullMax = 512;
  static constexpr int radix(int ns) { return (N / ns >= E) ? E : N / ns; }
  static constexpr bool full(int ns) { return (radix(ns) - 1) * ns <= kFullMax; }
  static constexpr int rows(int ns) { return full(ns) ? radix(ns) - 1 : ilog2(radix(ns)); }
  static constexpr int offset(int ns) {  // entries before the pass of stride ns
    int off = 0;
    for (int s = 1; s < ns; s *= radix(s))
      if (s > 1) off += rows(s) * s;
    return off;
  }
  static constexpr int kCount = offset(N);

  // Copy from the global tables; every lane of the workgroup calls it with
  // its id and the workgroup size, and the caller synchronises afterwards.
  template <int NS = 1>
  static __device__ __forceinline__ void fill(float2* lds, int tid, int nt) {
    if constexpr (NS < N) {
      constexpr int R = radix(NS);
      if constexpr (NS > 1) {
        constexpr int off = offset(NS), cnt = rows(NS) * NS;
        const float2* tab = pass_table<ilog2(NS), ilog2(R)>();
        for (int i = tid; i < cnt; i += nt) {
          const int q = i / NS, jm = i - q * NS;
          const int r = full(NS) ? q + 1 : (1 << q);
          lds[off + i] = tab[(uint32_t)(r - 1) * NS + jm];
        }
      }
      fill<NS * R>(lds, tid, nt);
    }
  }

  // x[r] *= W^(jm r), r = 1..R-1, W = exp(-+2 pi i / (NS R))
  template <int NS, int R, bool INV>
  static __device__ __forceinline__ void apply(const float2* lds, uint32_t jm, float2 (&x)[R]) {
    constexpr int off = offset(NS);
    if constexpr (full(NS)) {
#pragma unroll
      for (int r = 1; r < R; ++r) {
        const float2 w = lds[off + (r - 1) * NS + jm];
        x[r] = c_mul(x[r], INV ? c_conj(w) : w);
      }
    } else {
      float2 p[R];
#pragma unroll
      for (int q = 0; (1 << q) < R; ++q) {
        const float2 w = lds[off + q * NS + jm];
        p[1 << q] = INV ? c_conj(w) : w;
      }
#pragma unroll
      for (int r = 3; r < R; ++r) {
        if ((r & (r - 1)) != 0) {
          const int hi = 1 << ilog2(r);
          p[r] = c_mul(p[hi], p[r - hi]);
        }
      }
#pragma unroll
      for (int r = 1; r < R; ++r) x[r] = c_mul(x[r], p[r]);
    }
  }
};

// ---------------------------------------------------------------------------
// Block transform: N points over T = N/E lanes, E points per lane.
// All lanes of the workgroup must call run() the same number of times (it
// contains workgroup barriers when N > E).  Inactive lanes pass active=false:
// they take the barriers but touch no LDS.  The first exchange starts with a
// barrier, so callers may read the scratch line right before calling run().
// ---------------------------------------------------------------------------
template <int N, int E, bool INV>
struct BlockFFT {
  static_assert(is_pow2(N) && is_pow2(E) && E <= N && E <= 32, "block fft shape");
  static constexpr int T = N / E;

  template <class Scr>
  static __device__ __forceinline__ void run(float2 (&v)[E], int t, const Scr& scr, bool active) {
    pass<1>(v, t, scr, active, nullptr);
  }
  // Same, with the pass twiddles read from PassTw<N, E> tables in LDS.
  template <class Scr>
  static __device__ __forceinline__ void run(float2 (&v)[E], int t, const Scr& scr, bool active,
                                             const float2* lds_tw) {
    pass<1, Scr, true>(v, t, scr, active, lds_tw);
  }

  // Pass-16 layout: positions dst + r*NS (r < R) reachable by constant offsets
  // when NS is a multiple of 16, or when the R positions sit inside one
  // 16-entry block (NS * R <= 16; dst is then aligned to NS * R).
  static constexpr bool pad_write_ok(int NS, int R) { return NS % 16 == 0 || NS * R <= 16; }
  // reads t + T e: constant offsets when T is a multiple of 16 or divides 16
  static constexpr bool pad_read_ok() { return T % 16 == 0 || 16 % T == 0; }
  static constexpr int pad_read_off(int e) {
    return T % 16 == 0 ? (T * e) + (T * e) / 16 : T * (e % (16 / T)) + 17 * (e / (16 / T));
  }

  template <int NS, class Scr, bool LTW = false>
  static __device__ __forceinline__ void pass(float2 (&v)[E], int t, const Scr& scr, bool active,
                                              const float2* lds_tw) {
    constexpr int R = (N / NS >= E) ? E : N / NS;
    constexpr int NB = E / R;  // butterflies per lane in this pass
    if (active) {  // waves with no active lane skip the arithmetic
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        float2 x[R];
#pragma unroll
        for (int r = 0; r < R; ++r) x[r] = v[b + NB * r];
        if constexpr (NS > 1) {
          const uint32_t jm = (uint32_t)(t + T * b) & (NS - 1);
          if constexpr (LTW) {
            PassTw<N, E>::template apply<NS, R, INV>(lds_tw, jm, x);
          } else {
#pragma unroll
            for (int r = 1; r < R; ++r) x[r] = c_mul(x[r], pass_twiddle<NS, R, INV>(jm, r));
          }
        }
        dft<R, INV>(x);
#pragma unroll
        for (int r = 0; r < R; ++r) v[b + NB * r] = x[r];
      }
    }
    if constexpr (NS * R < N) {
      __syncthreads();
      if (active) {
#pragma unroll
        for (int b = 0; b < NB; ++b) {
          const int j = t + T * b;
          const int jm = j & (NS - 1);
          const int dst = (j - jm) * R + jm;
          if constexpr (Scr::kKind == 1 || (Scr::kKind == 2 && pad_write_ok(NS, R))) {
            float2* pw = scr(dst);
#pragma unroll
            for (int r = 0; r < R; ++r) pw[ScrOff<Scr>::off(r * NS)] = v[b + NB * r];
          } else {
#pragma unroll
            for (int r = 0; r < R; ++r) *scr(dst + r * NS) = v[b + NB * r];
          }
        }
      }
      __syncthreads();
      if (active) {
        if constexpr (Scr::kKind == 1) {
          const float2* pr = scr(t);
#pragma unroll
          for (int e = 0; e < E; ++e) v[e] = pr[ScrOff<Scr>::off(T * e)];
        } else if constexpr (Scr::kKind == 2 && pad_read_ok()) {
          const float2* pr = scr(t);
#pragma unroll
          for (int e = 0; e < E; ++e) v[e] = pr[pad_read_off(e)];
        } else {
#pragma unroll
          for (int e = 0; e < E; ++e) v[e] = *scr(t + T * e);
        }
      }
      pass<NS * R, Scr, LTW>(v, t, scr, active, lds_tw);
    }
  }
};

// ---------------------------------------------------------------------------
// Lanes of an NT-lane workgroup assigned to (line, t) for block transforms of
// T lanes per line, NT / T lines per round.  When T * 64 <= NT every
// wavefront holds a single t, made wave-uniform, and 64 consecutive lines:
// pass twiddle indices and exchange offsets are then scalar, and the lanes of
// a wavefront touch 64 consecutive lines at one position.  Otherwise
// consecutive lanes take consecutive lines and t = tid / (NT / T).
// ---------------------------------------------------------------------------
template <int T, int NT>
struct LaneMap {
  static constexpr bool kUniform = T * 64 <= NT;
  static constexpr int kLines = NT / T;
  // the final mask tells the compiler that t < T (tid < NT), so positions
  // t + T e known to be padding or outside the crop are compile-time facts
  static __device__ __forceinline__ int t(int tid) {
    if constexpr (kUniform) return __builtin_amdgcn_readfirstlane((tid >> 6) % T) & (T - 1);
    else return (tid / kLines) & (T - 1);
  }
  static __device__ __forceinline__ int line(int tid) {
    if constexpr (kUniform) return ((tid >> 6) / T) * 64 + (tid & 63);
    else return tid % kLines;
  }
};

// ---------------------------------------------------------------------------
// Workgroup renumbering.  The dispatcher hands workgroup b to XCD b % 8 (each
// XCD has its own L2).  xcd_order(b, n) numbers the n workgroups so that each
// XCD receives a contiguous range of logical ids in dispatch order: tiles with
// consecutive logical ids then run together on one XCD and share the cache
// lines they both touch (a bijection of [0, n)).
// ---------------------------------------------------------------------------
constexpr uint32_t kNumXcd = 8;
__host__ __device__ __forceinline__ uint32_t xcd_order(uint32_t b, uint32_t n) {
  const uint32_t x = b % kNumXcd, j = b / kNumXcd, per = n / kNumXcd, rem = n % kNumXcd;
  return x * per + (x < rem ? x : rem) + j;
}

// ---------------------------------------------------------------------------
// Staging copies.  Item i = tid + NT * j for j < ceil(COUNT / NT); a batch of
// BATCH items is loaded (all loads issued) before any of them is stored, so
// global-memory latency overlaps instead of serialising per item.  ld(i)
// returns the value (it may return zero for skipped items); st(i, value)
// stores it (it may ignore skipped items).
// ---------------------------------------------------------------------------
template <int COUNT, int NT, int BATCH, class Ld, class St>
__device__ __forceinline__ void batched_copy(int tid, const Ld& ld, const St& st) {
  constexpr int ITER = (COUNT + NT - 1) / NT;
  using V = decltype(ld(0));
#pragma unroll
  for (int j0 = 0; j0 < ITER; j0 += BATCH) {
    V tmp[BATCH];
#pragma unroll
    for (int b = 0; b < BATCH; ++b) {
      const int i = tid + NT * (j0 + b);
      if (j0 + b < ITER && (COUNT % NT == 0 || i < COUNT)) tmp[b] = ld(i);
    }
#pragma unroll
    for (int b = 0; b < BATCH; ++b) {
      const int i = tid + NT * (j0 + b);
      if (j0 + b < ITER && (COUNT % NT == 0 || i < COUNT)) st(i, tmp[b]);
    }
  }
}

// ---------------------------------------------------------------------------
// storage types: float (fp32) or uint16_t (bf16 bits); compute is fp32
// ---------------------------------------------------------------------------
__device__ __forceinline__ float ld1(const float* p) { return *p; }
__device__ __forceinline__ float ld1(const uint16_t* p) { return __uint_as_float(((uint32_t)*p) << 16); }
// fp32 -> bf16 with round to nearest even (NaN stays NaN): gfx950 converts a
// pair in one instruction (v_cvt_pk_bf16_f32)
typedef __bf16 bf16x2_v __attribute__((ext_vector_type(2)));
typedef float f32x2_v __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t bf16_pack(float lo, float hi) {
  const f32x2_v v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_v));
}
__device__ __forceinline__ uint16_t f32_to_bf16_rne(float x) { return __builtin_bit_cast(uint16_t, (__bf16)x); }
__device__ __forceinline__ void st1(float* p, float x) { *p = x; }
__device__ __forceinline__ void st1(uint16_t* p, float x) { *p = f32_to_bf16_rne(x); }
// four consecutive values (p aligned to four elements)
__device__ __forceinline__ float4 ld4(const float* p) { return *reinterpret_cast<const float4*>(p); }
__device__ __forceinline__ float4 ld4(const uint16_t* p) {
  const uint2 u = *reinterpret_cast<const uint2*>(p);
  return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u), __uint_as_float(u.y << 16),
                     __uint_as_float(u.y & 0xffff0000u));
}
__device__ __forceinline__ void st4(float* p, float4 x) { *reinterpret_cast<float4*>(p) = x; }
__device__ __forceinline__ void st4(uint16_t* p, float4 x) {
  uint2 u;
  u.x = bf16_pack(x.x, x.y);
  u.y = bf16_pack(x.z, x.w);
  *reinterpret_cast<uint2*>(p) = u;
}
// two consecutive values (p must be aligned to two elements)
__device__ __forceinline__ float2 ld2(const float* p) { return *reinterpret_cast<const float2*>(p); }
__device__ __forceinline__ float2 ld2(const uint16_t* p) {
  const uint32_t u = *reinterpret_cast<const uint32_t*>(p);
  return make_float2(__uint_as_float(u << 16), __uint_as_float(u & 0xffff0000u));
}
__device__ __forceinline__ void st2(float* p, float2 x) { *reinterpret_cast<float2*>(p) = x; }
__device__ __forceinline__ void st2(uint16_t* p, float2 x) {
  *reinterpret_cast<uint32_t*>(p) = bf16_pack(x.x, x.y);
}

// Line of k that line `line` (= b C + c) uses: its own, or with one kernel
// per channel (kC = C) the kernel of channel c.
__device__ __forceinline__ int64_t k_line(int64_t line, int kC) { return kC ? line % kC : line; }

// Raw pairs: the storage bits of two consecutive values, widened to fp32 only
// where they are used, so that a load issued early is waited for late.
template <typename TS>
struct Raw2;
template <>
struct Raw2<float> {
  using type = float2;
};
template <>
struct Raw2<uint16_t> {
  using type = uint32_t;
};
__device__ __forceinline__ float2 ld2_raw(const float* p) { return *reinterpret_cast<const float2*>(p); }
__device__ __forceinline__ uint32_t ld2_raw(const uint16_t* p) { return *reinterpret_cast<const uint32_t*>(p); }
__device__ __forceinline__ float2 widen2(float2 r) { return r; }
__device__ __forceinline__ float2 widen2(uint32_t u) {
  return make_float2(__uint_as_float(u << 16), __uint_as_float(u & 0xffff0000u));
}

// Real-to-complex post-pass.  A real line x[0..P) is read as the complex
// line z[m] = x[2m] + i x[2m+1] of length M = P/2 and transformed; with
// A = Z[g], B = Z[(M-g) mod M] and w = exp(-2 pi i g / P) this returns
// Xg = 2 X[g] and Xmg = 2 X[M-g] of the length-P real transform
// (X[f] = Xe[f] + w^f Xo[f], Xe/Xo the transforms of the even/odd samples).
__device__ __forceinline__ void r2c_pair(float2 A, float2 B, float2 w, float2& Xg, float2& Xmg) {
  const float2 e = make_float2(A.x + B.x, A.y - B.y);  // A + conj B      = 2 Xe[g]
  const float2 o = make_float2(A.y + B.y, B.x - A.x);  // -i (A - conj B) = 2 Xo[g]
  const float2 t = c_mul(w, o);
  Xg = c_add(e, t);
  Xmg = make_float2(e.x - t.x, t.y - e.y);  // conj(e - t)
}

// Bin g of a real row's doubled R2C spectrum from its packed transform Z
// (r2c_pair's first output, w = exp(-2 pi i g / P)); for g = 0 the DC and
// Nyquist bins, both real, packed as DC + i Nyquist (w = 1).  gm = (M - g) mod M.
__device__ __forceinline__ float2 untangle_bin(const float2* row, int g, int gm, float2 w) {
  float2 xa, xb;
  r2c_pair(row[g], row[gm], w, xa, xb);
  return g == 0 ? make_float2(xa.x, xb.x) : xa;
}

// Complex-to-real pre-pass, the inverse of r2c_pair: from the Hermitian
// spectrum values Yg = Y[g], Ymg = Y[M-g] of a real length-P signal y and
// w = exp(-2 pi i g / P), returns  Yg + conj Ymg + i w^-1 (Yg - conj Ymg)
// = 2 (E[g] + i O[g]), with E/O the length-M transforms of the even/odd
// samples; the length-M inverse of these bins is 2M (y[2m] + i y[2m+1]).
__device__ __forceinline__ float2 c2r_pair(float2 Yg, float2 Ymg, float2 w) {
  const float2 s = make_float2(Yg.x + Ymg.x, Yg.y - Ymg.y);  // Yg + conj Ymg
  const float2 d = make_float2(Yg.x - Ymg.x, Yg.y + Ymg.y);  // Yg - conj Ymg
  const float2 rd = c_mulc(d, w);                            // d exp(+2 pi i g / P)
  return make_float2(s.x - rd.y, s.y + rd.x);                // s + i rd
}

// Centered kernels (pad mode "centered"): 2L - 1 points per axis, index
// L - 1 the zero displacement, transformed on a grid of P >= 2L points.  Grid
// index g holds displacement g (g < L) or g - P (g > P - L); the indices in
// between hold no displacement of the L grid and stay zero (-1).
__device__ __forceinline__ int centered_index(int g, int L, int P) {
  return g < L ? g + L - 1 : (g > P - L ? g - P + L - 1 : -1);
}

// Same for a circular kernel of L points repeated periodically over the
// displacements -(L-1) .. L-1: displacement d takes k[d mod L].
__device__ __forceinline__ int periodic_index(int g, int L, int P) {
  return g < L ? g : (g > P - L ? g - P + L : -1);
}

// ---------------------------------------------------------------------------
// Inner and outer gates of one (b, c) line.  Plain call: u = x1 v and the
// gate is x2.  HyenaND operator (ACT): x1, v and x2 hold the projections q,
// kin and vin, u = q SiLU(kin) s[p] w_in[c] -- s[p] the l2 normalisation of
// q and the RMSNorm across channels at grid point p, precomputed per sample
// -- and the gate is Sigmoid(vin) (Eq. (HyenaND), section 3.2).
// ---------------------------------------------------------------------------
struct ActIn {
  const float* s;    // [B, npos] normalisation scale per (sample, grid point)
  const void* w_in;  // [C] RMSNorm weights, storage type
  int64_t npos;      // grid points per line
};

// exp through the hardware exp2 (__expf): a few ulp, well inside fp32 parity
__device__ __forceinline__ float silu_f(float x) { return x / (1.f + __expf(-x)); }
__device__ __forceinline__ float sigmoid_f(float x) { return 1.f / (1.f + __expf(-x)); }

template <bool ACT>
struct Gates {
  const float* s;  // this sample's row of s (ACT)
  float w;         // w_in[c] (ACT)
  // u at grid points p, p + 1 (p even) / p .. p + 3 (p a multiple of 4) / p
  __device__ __forceinline__ float2 u2(float2 a, float2 b, int64_t p) const {
    if constexpr (ACT) {
      const float2 sc = *reinterpret_cast<const float2*>(s + p);
      return make_float2(a.x * silu_f(b.x) * (sc.x * w), a.y * silu_f(b.y) * (sc.y * w));
    } else {
      return make_float2(a.x * b.x, a.y * b.y);
    }
  }
  __device__ __forceinline__ float4 u4(float4 a, float4 b, int64_t p) const {
    if constexpr (ACT) {
      const float4 sc = *reinterpret_cast<const float4*>(s + p);
      return make_float4(a.x * silu_f(b.x) * (sc.x * w), a.y * silu_f(b.y) * (sc.y * w),
                         a.z * silu_f(b.z) * (sc.z * w), a.w * silu_f(b.w) * (sc.w * w));
    } else {
      return make_float4(a.x * b.x, a.y * b.y, a.z * b.z, a.w * b.w);
    }
  }
  __device__ __forceinline__ float u1(float a, float b, int64_t p) const {
    if constexpr (ACT) return a * silu_f(b) * (s[p] * w);
    else return a * b;
  }
  __device__ __forceinline__ float2 g2(float2 x) const {
    if constexpr (ACT) return make_float2(sigmoid_f(x.x), sigmoid_f(x.y));
    else return x;
  }
  __device__ __forceinline__ float4 g4(float4 x) const {
    if constexpr (ACT) return make_float4(sigmoid_f(x.x), sigmoid_f(x.y), sigmoid_f(x.z), sigmoid_f(x.w));
    else return x;
  }
  __device__ __forceinline__ float g1(float x) const {
    if constexpr (ACT) return sigmoid_f(x);
    else return x;
  }
};

template <bool ACT, typename TS>
__device__ __forceinline__ Gates<ACT> line_gates(const ActIn& act, int64_t line, int C) {
  Gates<ACT> g;
  if constexpr (ACT) {
    g.s = act.s + (line / C) * act.npos;
    g.w = ld1(reinterpret_cast<const TS*>(act.w_in) + line % C);
  } else {
    g.s = nullptr;
    g.w = 1.f;
  }
  return g;
}

// exp(mag_log) (cos phase, sin phase) from a phase and log-magnitude formed
// in double: the phase is reduced to [-pi, pi] in double before the fp32
// sine and cosine, so a mode's factor at a large power t stays exact to a
// few fp32 roundings (modal filters).
__device__ __forceinline__ void polar(double mag_log, double phase, float& c, float& s, float& m) {
  const double two_pi = 6.283185307179586;
  const float r = (float)(phase - two_pi * rint(phase * (1.0 / two_pi)));  // in [-pi, pi]
  __sincosf(r, &s, &c);
  m = __expf((float)mag_log);
}

// Spectral product with the shortcut folded in: U (K + D), D times the
// transform of a unit impulse (1 at every bin).  Inputs are 2U and 2K.
__device__ __forceinline__ float2 gated_product(float2 U2, float2 K2, float twoD) {
  return c_mul(U2, make_float2(K2.x + twoD, K2.y));
}

}  // namespace hyenand
