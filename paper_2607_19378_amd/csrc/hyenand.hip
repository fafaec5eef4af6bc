// C-ABI front end: argument validation, plan choice, workspace sizing and
// launches.  Validation and sizing are pure host code; nothing here touches
// the GPU before every check has passed.
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <cmath>
#include <string>

#include "../../include/hyenand.h"
#include "kernels.hpp"

using namespace hyenand;

namespace {

thread_local std::string g_last_error;

hyenand_status fail(hyenand_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return s;
}

enum Plan { PLAN_NONE = 0, PLAN_FUSED1D, PLAN_FUSED2D, PLAN_MULTIPASS, PLAN_FOURSTEP, PLAN_FUSED_RL, PLAN_MIXED, PLAN_EMBED };

const char* plan_name(Plan p, const FftConvArgs& a) {
  const int ndim = a.ndim;
  switch (p) {
    case PLAN_FUSED1D: return "fused1d";
    case PLAN_FUSED2D: return "fused2d";
    case PLAN_MULTIPASS: return ndim == 3 ? (slab3d_supported(a) ? "slab3d" : "multipass3d") : "multipass2d";
    case PLAN_FOURSTEP: return "fourstep1d";
    case PLAN_FUSED_RL: return ndim == 1 ? "fused1d_any" : "fused2d_any";
    case PLAN_MIXED: return ndim == 1 ? "mixed1d" : (ndim == 2 ? "mixed2d" : "mixed3d");
    case PLAN_EMBED: return ndim == 1 ? "embedded1d" : (ndim == 2 ? "embedded2d" : "embedded3d");
    default: return "none";
  }
}

bool pow2(int64_t n) { return n >= 1 && (n & (n - 1)) == 0; }

constexpr int64_t kMaxLines = (int64_t(1) << 22) - 1;
// elementwise kernels of the embedded plans: 256 lanes per element block,
// fewer than 2^32 work-items per launch
constexpr int64_t kMaxEmbedElems = (int64_t(1) << 31);

// Shape checks shared by every entry point.  Fills a (pointers left null).
hyenand_status parse_shape(int ndim, const int64_t* dims, int pad_mode, int dtype, FftConvArgs* a) {
  memset(a, 0, sizeof *a);
  if (ndim < 1 || ndim > 3) return fail(HYENAND_ERR_INVALID_ARGUMENT, "ndim must be 1, 2 or 3 (got %d)", ndim);
  if (!dims) return fail(HYENAND_ERR_INVALID_ARGUMENT, "dims is NULL");
  if (pad_mode != HYENAND_PAD_LINEAR && pad_mode != HYENAND_PAD_CIRCULAR && pad_mode != HYENAND_PAD_CENTERED)
    return fail(HYENAND_ERR_INVALID_ARGUMENT, "pad_mode must be 0 (linear), 1 (circular) or 2 (centered), got %d",
                pad_mode);
  if (dtype != HYENAND_DTYPE_F32 && dtype != HYENAND_DTYPE_BF16)
    return fail(HYENAND_ERR_INVALID_ARGUMENT, "dtype must be 0 (f32) or 1 (bf16), got %d", dtype);
  int64_t total = 1;
  for (int i = 0; i < ndim + 2; ++i) {
    if (dims[i] < 1) return fail(HYENAND_ERR_INVALID_ARGUMENT, "dims[%d] = %lld must be >= 1", i, (long long)dims[i]);
    if (dims[i] > (int64_t(1) << 40) || total > (int64_t(1) << 46) / dims[i])
      return fail(HYENAND_ERR_UNSUPPORTED, "tensor too large");
    total *= dims[i];
  }
  a->lines = dims[0] * dims[1];
  a->C = dims[1];
  // one workgroup per (b, c) line in the single-pass kernels, up to 1024
  // lanes each, and a launch holds fewer than 2^32 work-items
  if (a->lines > kMaxLines)
    return fail(HYENAND_ERR_UNSUPPORTED, "B * C = %lld (b, c) lines exceed the %lld one call takes",
                (long long)a->lines, (long long)kMaxLines);
  a->circular = pad_mode == HYENAND_PAD_CIRCULAR;
  a->centered = pad_mode == HYENAND_PAD_CENTERED;
  a->bf16 = dtype == HYENAND_DTYPE_BF16;
  // squeeze unit axes: along an axis of extent 1 every mode reduces to the
  // zero-displacement term (the centered kernel has 2 * 1 - 1 = 1 point there)
  int nd = 0;
  for (int d = 0; d < ndim; ++d) {
    const int64_t L = dims[2 + d];
    if (!pow2(L)) {
      if (L > (int64_t(1) << 24)) return fail(HYENAND_ERR_UNSUPPORTED, "grid extent too large");
      a->rl = true;
    }
    if (L > 1) a->L[nd++] = L;
  }
  if (nd == 0) {  // a single point: the linear transform of length 2 covers it
    nd = 1;
    a->L[0] = 1;
    a->circular = false;
    a->centered = false;
  }
  a->ndim = nd;
  if (a->rl && a->circular) {
    // a circular convolution of L points is the centred one whose kernel
    // repeats k periodically over the displacements -(L-1) .. L-1, so it runs
    // on the non-circular transform grid with that kernel
    a->circular = false;
    a->periodic = true;
  }
  for (int d = 0; d < nd; ++d) {
    // non-circular: the smallest power of two >= 2L - 1 (2L for a power of two)
    int64_t p = 2;
    while (p < 2 * a->L[d] - 1) p *= 2;
    a->P[d] = a->circular ? a->L[d] : p;
  }
  return HYENAND_OK;
}

// A shape whose extents are not powers of two and that neither the
// power-of-two single-pass kernels nor the mixed-radix ones take runs
// embedded in its transform grid (P_d >= 2 L_d - 1, a power of two): on that
// grid the call is the circular convolution of the zero-padded
// inputs and of k placed at its displacements (conv_embed.hip), so x1, x2, v
// and k are embedded, the circular plan of the grid runs, and y is extracted.
// The workspace holds the five embedded tensors (x1, x2, v, k, y; each
// 256-byte aligned) and then the circular plan's own.
struct GridProblem {
  FftConvArgs e;  // the circular problem on the transform grid
  int nd;
  int64_t dims[5];
  size_t tensor;  // bytes of one embedded tensor
};

bool grid_problem(const FftConvArgs& a, GridProblem* m) {
  m->nd = a.ndim;
  m->dims[0] = a.lines / a.C;
  m->dims[1] = a.C;
  for (int d = 0; d < a.ndim; ++d) m->dims[2 + d] = a.P[d];
  const std::string keep = g_last_error;
  const hyenand_status st = parse_shape(m->nd, m->dims, HYENAND_PAD_CIRCULAR,
                                        a.bf16 ? HYENAND_DTYPE_BF16 : HYENAND_DTYPE_F32, &m->e);
  g_last_error = keep;
  m->tensor = ((size_t)embed_grid_elems(a) * (a.bf16 ? 2 : 4) + 255) / 256 * 256;
  return st == HYENAND_OK && embed_grid_elems(a) <= kMaxEmbedElems;
}

Plan choose_plan(const FftConvArgs& a);

// the circular plan of the grid problem of an embedded forward
Plan embedded_inner_plan(const FftConvArgs& a, GridProblem* m) {
  if (!grid_problem(a, m)) return PLAN_NONE;
  const Plan p = choose_plan(m->e);
  return p == PLAN_EMBED ? PLAN_NONE : p;
}

// Extents that are not powers of two: the mixed-radix kernels where they are
// the faster (mixed_preferred), the power-of-two single-pass kernels, then the
// mixed-radix ones for the shapes those do not take, then the embedded plans.
// HYENAND_PLAN=mixed prefers, =nomixed avoids, the mixed-radix kernels.
Plan choose_plan(const FftConvArgs& a) {
  const char* force = getenv("HYENAND_PLAN");
  if (a.rl) {
    const bool want = force && strcmp(force, "mixed") == 0;
    const bool avoid = force && strcmp(force, "nomixed") == 0;
    if (!avoid && (want ? mixed_supported(a) : mixed_preferred(a))) return PLAN_MIXED;
    if (fused_rl_supported(a)) return PLAN_FUSED_RL;
    if (!avoid && mixed_supported(a)) return PLAN_MIXED;
    GridProblem m;
    return embedded_inner_plan(a, &m) != PLAN_NONE ? PLAN_EMBED : PLAN_NONE;
  }
  const bool no_fused = force && (strcmp(force, "multipass") == 0 || strcmp(force, "fourstep") == 0);
  if (a.ndim == 1) {
    if (!no_fused && fused1d_supported(a.P[0])) return PLAN_FUSED1D;
    if (fourstep_supported(a)) return PLAN_FOURSTEP;
    return PLAN_NONE;
  }
  if (a.ndim == 2 && !no_fused && fused2d_supported(a.P[0], a.P[1])) return PLAN_FUSED2D;
  if (multipass_supported(a)) return PLAN_MULTIPASS;
  return PLAN_NONE;
}

size_t bytes_per_line(const FftConvArgs& a, Plan p);

// workspace of an embedded forward: the five tensors, then the inner plan's
// least (or recommended) workspace
size_t embed_fwd_ws(const FftConvArgs& a, bool recommended);

size_t bytes_per_line(const FftConvArgs& a, Plan p) {
  if (p == PLAN_MULTIPASS) return multipass_bytes_per_line(a);
  if (p == PLAN_FOURSTEP) return fourstep_bytes_per_line(a);
  if (p == PLAN_EMBED) return embed_fwd_ws(a, false);  // the least workspace of the whole call
  return 0;
}

// Chunking of the multi-pass plans.  Their spectra go through the caller's
// workspace a chunk of lines at a time.  Consecutive chunks rotate over S
// side streams, each with its own part of the workspace, so that the passes
// of one chunk run in the launch tails of the others'; a chunk's spectra are
// kept near 1/S of a 160 MiB budget so that the next pass over them still
// finds most of them in the 256 MiB Infinity Cache.  S is 2 (measured best
// or equal on the MI355X for 512^2, 2^20 and 128^3 lines against 1, 3 and 4,
// at 160 to 640 MiB budgets).  The recommended workspace is S such chunks;
// HYENAND_WS_TARGET_MB sets the budget and HYENAND_CHUNK_STREAMS fixes S.
size_t ws_target_bytes() {
  size_t target = (size_t)160 << 20;
  if (const char* e = getenv("HYENAND_WS_TARGET_MB")) {
    long mb = strtol(e, nullptr, 10);
    if (mb > 0) target = (size_t)mb << 20;
  }
  return target;
}

// side streams of a chunked call: 1 (the caller's stream only) up to
// kMaxSide, 2 unless HYENAND_CHUNK_STREAMS says otherwise
constexpr int kMaxSide = 4;
int chunk_streams() {
  if (const char* e = getenv("HYENAND_CHUNK_STREAMS")) {
    const long n = strtol(e, nullptr, 10);
    if (n >= 1 && n <= kMaxSide) return (int)n;
  }
  return 2;
}

struct ChunkPlan {
  int64_t chunk;    // lines per chunk (the last one may hold fewer)
  int64_t nchunks;
  int streams;      // 1: everything on the caller's stream
};

ChunkPlan plan_chunks(int64_t lines, size_t per, size_t ws_bytes) {
  ChunkPlan c;
  const int64_t fit = (int64_t)(ws_bytes / per);  // >= 1, checked by the caller
  const int want = chunk_streams();
  c.streams = want;
  if (c.streams > fit) c.streams = (int)fit;
  if (c.streams > lines) c.streams = (int)lines;
  int64_t target = (int64_t)(ws_target_bytes() / (size_t)want / per);
  if (target < 1) target = 1;
  int64_t chunk = fit / c.streams;
  if (chunk > target) chunk = target;
  if (chunk > lines) chunk = lines;
  c.nchunks = (lines + chunk - 1) / chunk;
  c.chunk = (lines + c.nchunks - 1) / c.nchunks;  // balanced
  if (c.nchunks < c.streams) c.streams = (int)c.nchunks;
  return c;
}

size_t recommended_ws(const FftConvArgs& a, Plan p) {
  if (p == PLAN_EMBED) return embed_fwd_ws(a, true);
  const size_t per = bytes_per_line(a, p);
  if (per == 0) return 0;
  const int ns = chunk_streams();
  int64_t n = (int64_t)(ws_target_bytes() / (size_t)ns / per);
  if (n < 1) n = 1;
  n *= ns;
  if (n > a.lines) n = a.lines;
  return (size_t)n * per;
}

size_t embed_fwd_ws(const FftConvArgs& a, bool recommended) {
  GridProblem m;
  const Plan pi = embedded_inner_plan(a, &m);
  if (pi == PLAN_NONE) return 0;
  return 5 * m.tensor + (recommended ? recommended_ws(m.e, pi) : bytes_per_line(m.e, pi));
}

// Side streams of the multi-pass plans, and the events that fork them off
// the caller's stream and join them back: one set per (host thread, device),
// created on that thread's first multi-pass call on the device (default
// priority, non-blocking) and kept until the process ends.  Later calls
// create nothing.  Each host thread has its own set, so calls from several
// threads neither serialise on shared streams nor enter another thread's
// graph capture.
constexpr int kMaxDevices = 64;
struct SideSet {
  bool ready = false;
  hipStream_t s[kMaxSide] = {};
  hipEvent_t fork = nullptr;
  hipEvent_t join[kMaxSide] = {};
};
thread_local SideSet t_side[kMaxDevices];

hipError_t create_side_set(SideSet& st, int dev) {
  int prev = 0;
  hipError_t e = hipGetDevice(&prev);
  if (e == hipSuccess && prev != dev) e = hipSetDevice(dev);
  for (int i = 0; i < kMaxSide && e == hipSuccess; ++i) e = hipStreamCreateWithFlags(&st.s[i], hipStreamNonBlocking);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&st.fork, hipEventDisableTiming);
  for (int i = 0; i < kMaxSide && e == hipSuccess; ++i) e = hipEventCreateWithFlags(&st.join[i], hipEventDisableTiming);
  if (e != hipSuccess) {  // leave nothing half made: the next call tries again
    for (int i = 0; i < kMaxSide; ++i) {
      if (st.s[i]) (void)hipStreamDestroy(st.s[i]);
      if (st.join[i]) (void)hipEventDestroy(st.join[i]);
      st.s[i] = nullptr;
      st.join[i] = nullptr;
    }
    if (st.fork) (void)hipEventDestroy(st.fork);
    st.fork = nullptr;
  }
  if (prev != dev) {
    const hipError_t r = hipSetDevice(prev);
    if (e == hipSuccess) e = r;
  }
  st.ready = e == hipSuccess;
  return e;
}

hipError_t side_set(hipStream_t caller, SideSet** out) {
  int dev = 0;
  hipError_t e = caller ? hipStreamGetDevice(caller, &dev) : hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  SideSet& st = t_side[dev];
  if (!st.ready) {
    e = create_side_set(st, dev);
    if (e != hipSuccess) return e;
  }
  *out = &st;
  return hipSuccess;
}

// Run a multi-pass plan chunk by chunk.  With side streams: they wait for
// the caller's stream, chunk j runs on side stream j % S with workspace part
// j % S, and the caller's stream waits for all S before any later work.
template <class Launch>
hipError_t run_chunked(const FftConvArgs& a, size_t per, hipStream_t caller, Launch launch) {
  const ChunkPlan c = plan_chunks(a.lines, per, a.ws_bytes);
  if (c.streams == 1) {
    for (int64_t j = 0; j < c.nchunks; ++j) {
      const int64_t line0 = j * c.chunk;
      const int64_t nl = a.lines - line0 < c.chunk ? a.lines - line0 : c.chunk;
      if (nl <= 0) break;
      const hipError_t e = launch(line0, nl, a.ws, caller);
      if (e != hipSuccess) return e;
    }
    return hipSuccess;
  }
  const int S = c.streams;
  SideSet* side = nullptr;
  hipError_t e = side_set(caller, &side);
  if (e != hipSuccess) return e;
  e = hipEventRecord(side->fork, caller);
  for (int i = 0; i < S && e == hipSuccess; ++i) e = hipStreamWaitEvent(side->s[i], side->fork, 0);
  if (e != hipSuccess) return e;
  for (int64_t j = 0; j < c.nchunks; ++j) {
    const int64_t line0 = j * c.chunk;
    const int64_t nl = a.lines - line0 < c.chunk ? a.lines - line0 : c.chunk;
    if (nl <= 0) break;
    const int q = (int)(j % S);
    void* ws = (char*)a.ws + (size_t)q * (size_t)c.chunk * per;
    e = launch(line0, nl, ws, side->s[q]);
    if (e != hipSuccess) break;
  }
  // join even after a failed launch, so that no work is left unordered with
  // the caller's stream
  for (int i = 0; i < S; ++i) {
    hipError_t r = hipEventRecord(side->join[i], side->s[i]);
    if (r == hipSuccess) r = hipStreamWaitEvent(caller, side->join[i], 0);
    if (e == hipSuccess) e = r;
  }
  return e;
}

// Backward plans: single pass per line where the three spectra fit in LDS,
// else the multi-pass (2D/3D) or four-step (1D) structure of the forward
// with three signals.  The workspace holds the gD sums (256-byte aligned
// block) and then the spectra of a chunk of lines per side stream.
//
// Extents that are not powers of two run the mixed-radix single pass
// (BWD_MIXED, conv_mixed.hip) where their grid fits; those beyond it and the
// centred mode on power-of-two extents (BWD_EMBED) run the circular backward
// on their transform grid (P_d >= 2 L_d - 1, a power of two): the five
// inputs are embedded in that grid and the four gradient
// tensors extracted from it (conv_embed.hip); gD comes out directly.  Their
// workspace holds the nine embedded tensors (each 256-byte aligned) and then
// the circular backward's own.
enum BwdPlan { BWD_NONE = 0, BWD_FUSED, BWD_MULTIPASS, BWD_FOURSTEP, BWD_MIXED, BWD_EMBED };

BwdPlan choose_bwd_plan(const FftConvArgs& a);

struct Embedded {
  FftConvArgs e;  // the circular problem on the transform grid
  BwdPlan p;      // its plan
  int nd;
  int64_t dims[5];
  size_t tensor;  // bytes of one embedded tensor
};

bool embedded_problem(const FftConvArgs& a, Embedded* m) {
  m->nd = a.ndim;
  m->dims[0] = a.lines / a.C;
  m->dims[1] = a.C;
  for (int d = 0; d < a.ndim; ++d) m->dims[2 + d] = a.P[d];
  const std::string keep = g_last_error;
  const hyenand_status st = parse_shape(m->nd, m->dims, HYENAND_PAD_CIRCULAR,
                                        a.bf16 ? HYENAND_DTYPE_BF16 : HYENAND_DTYPE_F32, &m->e);
  g_last_error = keep;
  if (st != HYENAND_OK) return false;
  m->p = choose_bwd_plan(m->e);
  m->tensor = ((size_t)embed_grid_elems(a) * (a.bf16 ? 2 : 4) + 255) / 256 * 256;
  return m->p != BWD_NONE && m->p != BWD_EMBED && embed_grid_elems(a) <= kMaxEmbedElems;
}

BwdPlan choose_bwd_plan(const FftConvArgs& a) {
  if (a.centered || a.rl) {
    // extents that are not powers of two: the mixed-radix single pass on the
    // forward's grid where it fits (HYENAND_PLAN=nomixed avoids it)
    const char* force = getenv("HYENAND_PLAN");
    if (a.rl && !(force && strcmp(force, "nomixed") == 0) && mixed_backward_supported(a)) return BWD_MIXED;
    Embedded m;
    return embedded_problem(a, &m) ? BWD_EMBED : BWD_NONE;
  }
  if (fused_backward_supported(a)) return BWD_FUSED;
  if ((a.ndim == 2 || a.ndim == 3) && multipass_supported(a)) return BWD_MULTIPASS;
  if (a.ndim == 1 && backward_fs_supported(a)) return BWD_FOURSTEP;
  return BWD_NONE;
}

int64_t bwd_partials_per_line(const FftConvArgs& a, BwdPlan p) {
  switch (p) {
    case BWD_FUSED: return 1;
    case BWD_MIXED: return 1;
    case BWD_MULTIPASS: return backward_mp_partials_per_line(a);
    case BWD_FOURSTEP: return backward_fs_partials_per_line(a);
    default: return 0;
  }
}

size_t bwd_partial_bytes(const FftConvArgs& a, BwdPlan p) {
  const size_t n = (size_t)a.lines * (size_t)bwd_partials_per_line(a, p) * sizeof(float);
  return (n + 255) / 256 * 256;
}

size_t bwd_bytes_per_line(const FftConvArgs& a, BwdPlan p) {
  if (p == BWD_MULTIPASS) return backward_mp_bytes_per_line(a);
  if (p == BWD_FOURSTEP) return backward_fs_bytes_per_line(a);
  return 0;
}

size_t bwd_recommended_spectra(const FftConvArgs& a, BwdPlan p) {
  const size_t per = bwd_bytes_per_line(a, p);
  if (per == 0) return 0;
  const int ns = chunk_streams();
  int64_t n = (int64_t)(ws_target_bytes() / (size_t)ns / per);
  if (n < 1) n = 1;
  n *= ns;
  if (n > a.lines) n = a.lines;
  return (size_t)n * per;
}

bool overlaps(const void* a, size_t na, const void* b, size_t nb) {
  const uintptr_t a0 = (uintptr_t)a, b0 = (uintptr_t)b;
  return a0 < b0 + nb && b0 < a0 + na;
}

// Shape of a call that keeps kernel spectra (one kernel per channel, the
// single-pass 2D plan): parsed, with the plan checked.
hyenand_status spectrum_shape(int ndim, const int64_t* dims, int pad_mode, int dtype, FftConvArgs* a) {
  const hyenand_status st = parse_shape(ndim, dims, pad_mode, dtype, a);
  if (st != HYENAND_OK) return st;
  a->kC = (int)a->C;
  if (choose_plan(*a) != PLAN_FUSED2D || fused2d_khat_bytes(*a) == 0)
    return fail(HYENAND_ERR_UNSUPPORTED,
                "kernel spectra are kept for the single-pass 2D plan only (power-of-two transform grids up to "
                "128 x 128, linear or circular)");
  return HYENAND_OK;
}

}  // namespace

namespace hyenand {
// the calling thread's last-error text, for entry points in other
// translation units
hyenand_status set_last_error(hyenand_status s, const char* msg) { return fail(s, "%s", msg); }
}  // namespace hyenand

extern "C" {

hyenand_status hyenand_fftconv_workspace_size(int ndim, const int64_t* dims, hyenand_pad_mode pad_mode, hyenand_dtype dtype,
                                              size_t* bytes_out) {
  if (!bytes_out) return fail(HYENAND_ERR_INVALID_ARGUMENT, "bytes_out is NULL");
  FftConvArgs a;
  hyenand_status st = parse_shape(ndim, dims, pad_mode, dtype, &a);
  if (st != HYENAND_OK) return st;
  const Plan p = choose_plan(a);
  if (p == PLAN_NONE) return fail(HYENAND_ERR_UNSUPPORTED, "no plan for this shape");
  *bytes_out = recommended_ws(a, p);
  return HYENAND_OK;
}

hyenand_status hyenand_fftconv_shared_k_workspace_size(int ndim, const int64_t* dims, hyenand_pad_mode pad_mode,
                                                       hyenand_dtype dtype, size_t* bytes_out) {
  if (!bytes_out) return fail(HYENAND_ERR_INVALID_ARGUMENT, "bytes_out is NULL");
  FftConvArgs a;
  hyenand_status st = parse_shape(ndim, dims, pad_mode, dtype, &a);
  if (st != HYENAND_OK) return st;
  a.kC = (int)a.C;
  const Plan p = choose_plan(a);
  if (p == PLAN_NONE) return fail(HYENAND_ERR_UNSUPPORTED, "no plan for this shape");
  const size_t khb = (p == PLAN_FUSED2D && a.lines / a.C >= 2) ? fused2d_khat_bytes(a) : 0;
  *bytes_out = std::max(recommended_ws(a, p), khb);
  return HYENAND_OK;
}

hyenand_status hyenand_fftconv_workspace_min(int ndim, const int64_t* dims, hyenand_pad_mode pad_mode, hyenand_dtype dtype,
                                             size_t* bytes_out) {
  if (!bytes_out) return fail(HYENAND_ERR_INVALID_ARGUMENT, "bytes_out is NULL");
  FftConvArgs a;
  hyenand_status st = parse_shape(ndim, dims, pad_mode, dtype, &a);
  if (st != HYENAND_OK) return st;
  const Plan p = choose_plan(a);
  if (p == PLAN_NONE) return fail(HYENAND_ERR_UNSUPPORTED, "no plan for this shape");
  *bytes_out = bytes_per_line(a, p);
  return HYENAND_OK;
}

hyenand_status hyenand_fftconv_plan_name(int ndim, const int64_t* dims, hyenand_pad_mode pad_mode, hyenand_dtype dtype, char* buf,
                                         size_t n) {
  if (!buf || n == 0) return fail(HYENAND_ERR_INVALID_ARGUMENT, "buf is NULL or empty");
  FftConvArgs a;
  hyenand_status st = parse_shape(ndim, dims, pad_mode, dtype, &a);
  if (st != HYENAND_OK) return st;
  const Plan p = choose_plan(a);
  if (p == PLAN_NONE) return fail(HYENAND_ERR_UNSUPPORTED, "no plan for this shape");
  snprintf(buf, n, "%s", plan_name(p, a));
  return HYENAND_OK;
}

}  // extern "C"

namespace {

// Every step of the path for a validated call: the plan's kernels, chunked
// over side streams for the multi-pass plans.
hipError_t launch_plan(const FftConvArgs& a, Plan p, size_t per, hipStream_t s) {
  switch (p) {
    case PLAN_FUSED1D: return launch_fused1d(a, s);
    case PLAN_FUSED2D: return launch_fused2d(a, s);
    case PLAN_MULTIPASS:
      return run_chunked(a, per, s, [&a](int64_t l0, int64_t nl, void* ws, hipStream_t st) {
        return launch_multipass(a, l0, nl, ws, st);
      });
    case PLAN_FOURSTEP:
      return run_chunked(a, per, s, [&a](int64_t l0, int64_t nl, void* ws, hipStream_t st) {
        return launch_fourstep(a, l0, nl, ws, st);
      });
    case PLAN_FUSED_RL: return launch_fused_rl(a, s);
    case PLAN_MIXED: return launch_mixed(a, s);
    default: return hipErrorInvalidValue;
  }
}

// modal: the kernel is generated from these modal-filter parameters instead
// of read (k is NULL; one filter per channel).
hyenand_status forward(const void* x1, const void* x2, const void* v, const void* k, const void* D, void* y,
                       int ndim, const int64_t* dims, int pad_mode, int dtype, void* workspace,
                       size_t workspace_bytes, void* stream, bool shared_k, const ModalIn* modal = nullptr) {
  g_last_error.clear();
  FftConvArgs a;
  hyenand_status st = parse_shape(ndim, dims, pad_mode, dtype, &a);
  if (st != HYENAND_OK) return st;
  a.kC = shared_k ? (int)a.C : 0;
  if (!x1 || !x2 || !v || (!k && !modal) || !D || !y)
    return fail(HYENAND_ERR_INVALID_ARGUMENT, "a tensor pointer is NULL");
  if (modal) {
    const float* mp[4] = {modal->a, modal->th, modal->re, modal->im};
    const char* mn[4] = {"log_mag", "angle", "res_re", "res_im"};
    if (modal->M < 1 || modal->M > kMaxFusedModalOrder)
      return fail(HYENAND_ERR_UNSUPPORTED, "order must be 1..%d for the fused modal filter (got %d)",
                  kMaxFusedModalOrder, modal->M);
    const size_t pb = (size_t)a.C * (size_t)modal->M * sizeof(float);
    size_t nyb = (size_t)a.lines * (a.bf16 ? 2 : 4);
    for (int d = 0; d < a.ndim; ++d) nyb *= (size_t)a.L[d];
    for (int i = 0; i < 4; ++i) {
      if (!mp[i]) return fail(HYENAND_ERR_INVALID_ARGUMENT, "%s is NULL", mn[i]);
      if ((uintptr_t)mp[i] % 4 != 0) return fail(HYENAND_ERR_INVALID_ARGUMENT, "%s is not 4-byte aligned", mn[i]);
      if (overlaps(y, nyb, mp[i], pb)) return fail(HYENAND_ERR_INVALID_ARGUMENT, "y overlaps %s", mn[i]);
      if (workspace && overlaps(workspace, workspace_bytes, mp[i], pb))
        return fail(HYENAND_ERR_INVALID_ARGUMENT, "workspace overlaps %s", mn[i]);
    }
    if (a.centered || a.rl || a.periodic || choose_plan(a) != PLAN_FOURSTEP)
      return fail(HYENAND_ERR_UNSUPPORTED,
                  "the fused modal filter runs on the four-step plan only (1D lines, transform of 2^15 .. 2^22 "
                  "points, linear or circular)");
    a.modal = *modal;
    a.kC = (int)a.C;
  }
  {
    const void* tens[5] = {x1, x2, v, modal ? x1 : k, y};
    const char* tn[5] = {"x1", "x2", "v", "k", "y"};
    for (int i = 0; i < 5; ++i)
      if ((uintptr_t)tens[i] % 16 != 0)
        return fail(HYENAND_ERR_INVALID_ARGUMENT, "%s is not 16-byte aligned", tn[i]);
    if ((uintptr_t)D % (dtype == HYENAND_DTYPE_BF16 ? 2 : 4) != 0)
      return fail(HYENAND_ERR_INVALID_ARGUMENT, "D is not aligned to its element size");
    if (workspace && (uintptr_t)workspace % 16 != 0)
      return fail(HYENAND_ERR_INVALID_ARGUMENT, "workspace is not 16-byte aligned");
  }
  const size_t es = a.bf16 ? 2 : 4;
  size_t n = (size_t)a.lines;
  for (int d = 0; d < a.ndim; ++d) n *= (size_t)a.L[d];
  const size_t nb = n * es;
  size_t kpts = 1;  // kernel points per line: prod L_d, or prod (2 L_d - 1) centered
  for (int d = 0; d < a.ndim; ++d) kpts *= (size_t)(a.centered ? 2 * a.L[d] - 1 : a.L[d]);
  const size_t kb = (size_t)(shared_k ? a.C : a.lines) * kpts * es;  // [C, K...] or [B, C, K...]
  const void* ins[4] = {x1, x2, v, k};
  const size_t in_bytes[4] = {nb, nb, nb, modal ? (size_t)0 : kb};
  const char* names[4] = {"x1", "x2", "v", "k"};
  for (int i = 0; i < 4; ++i)
    if (overlaps(y, nb, ins[i], in_bytes[i])) return fail(HYENAND_ERR_INVALID_ARGUMENT, "y overlaps %s", names[i]);
  if (overlaps(y, nb, D, (size_t)a.C * es)) return fail(HYENAND_ERR_INVALID_ARGUMENT, "y overlaps D");
  const Plan p = choose_plan(a);
  if (p == PLAN_NONE) return fail(HYENAND_ERR_UNSUPPORTED, "no plan for this shape");
  const size_t per = bytes_per_line(a, p);
  // one kernel per channel on the fused 2D plan: with room in the workspace,
  // each channel's spectrum is computed once and read by all its images
  const size_t khb = (shared_k && !modal && p == PLAN_FUSED2D && a.lines / a.C >= 2) ? fused2d_khat_bytes(a) : 0;
  const bool use_khat = khb > 0 && workspace && workspace_bytes >= khb;
  if (per > 0 || use_khat) {
    if (!workspace || workspace_bytes < per)
      return fail(HYENAND_ERR_WORKSPACE_TOO_SMALL, "plan %s needs at least %zu workspace bytes, got %zu",
                  plan_name(p, a), per, workspace ? workspace_bytes : (size_t)0);
    if (overlaps(workspace, workspace_bytes, y, nb)) return fail(HYENAND_ERR_INVALID_ARGUMENT, "workspace overlaps y");
    for (int i = 0; i < 4; ++i)
      if (overlaps(workspace, workspace_bytes, ins[i], in_bytes[i]))
        return fail(HYENAND_ERR_INVALID_ARGUMENT, "workspace overlaps %s", names[i]);
  }
  a.x1 = x1; a.x2 = x2; a.v = v; a.k = k; a.D = D; a.y = y;
  a.ws = workspace;
  a.ws_bytes = workspace_bytes;
  a.khat = use_khat ? (float2*)workspace : nullptr;
  clear_pending_error();
  if (p == PLAN_EMBED) {
    // x1, x2, v, k into the transform grid, the circular plan there, y back
    GridProblem m;
    embedded_inner_plan(a, &m);
    char* w = (char*)workspace;
    void* const e[4] = {w, w + m.tensor, w + 2 * m.tensor, w + 3 * m.tensor};
    void* const ey = w + 4 * m.tensor;
    hipError_t err = launch_embed_fwd(a, e, (hipStream_t)stream);
    if (err != hipSuccess) return fail(HYENAND_ERR_HIP, "HIP error %d: %s", (int)err, hipGetErrorString(err));
    const hyenand_status inner = forward(e[0], e[1], e[2], e[3], D, ey, m.nd, m.dims, HYENAND_PAD_CIRCULAR, dtype,
                                         w + 5 * m.tensor, workspace_bytes - 5 * m.tensor, stream, false);
    if (inner != HYENAND_OK) return inner;
    err = launch_extract_y(a, ey, y, (hipStream_t)stream);
    if (err != hipSuccess) return fail(HYENAND_ERR_HIP, "HIP error %d: %s", (int)err, hipGetErrorString(err));
    return HYENAND_OK;
  }
  const hipError_t err = launch_plan(a, p, per, (hipStream_t)stream);
  if (err != hipSuccess) return fail(HYENAND_ERR_HIP, "HIP error %d: %s", (int)err, hipGetErrorString(err));
  return HYENAND_OK;
}

// HyenaND operator: prologue scale s (B * npos floats, first in the
// workspace, 256-byte block), the plan's kernels with the operator's gates,
// the output RMSNorm in place.
size_t op_scale_bytes(const FftConvArgs& a) {
  int64_t npos = 1;
  for (int d = 0; d < a.ndim; ++d) npos *= a.L[d];
  return ((size_t)(a.lines / a.C) * (size_t)npos * sizeof(float) + 255) / 256 * 256;
}

hyenand_status operator_fwd(const void* q, const void* kin, const void* vin, const void* k, const void* D,
                            const void* w_in, const void* w_out, float eps_l2, float eps_rms, void* y, int ndim,
                            const int64_t* dims, int pad_mode, int dtype, void* workspace, size_t workspace_bytes,
                            void* stream) {
  g_last_error.clear();
  FftConvArgs a;
  hyenand_status st = parse_shape(ndim, dims, pad_mode, dtype, &a);
  if (st != HYENAND_OK) return st;
  const void* ptrs[8] = {q, kin, vin, k, D, w_in, w_out, y};
  const char* pn[8] = {"q", "kin", "vin", "k", "D", "w_in", "w_out", "y"};
  for (int i = 0; i < 8; ++i)
    if (!ptrs[i]) return fail(HYENAND_ERR_INVALID_ARGUMENT, "%s is NULL", pn[i]);
  const size_t es = a.bf16 ? 2 : 4;
  for (int i = 0; i < 8; ++i) {
    const bool vec = i < 4 || i == 7;
    if ((uintptr_t)ptrs[i] % (vec ? 16 : es) != 0) return fail(HYENAND_ERR_INVALID_ARGUMENT, "%s is not aligned", pn[i]);
  }
  if (!(eps_l2 >= 0.f) || !(eps_rms >= 0.f) || !std::isfinite(eps_l2) || !std::isfinite(eps_rms))
    return fail(HYENAND_ERR_INVALID_ARGUMENT, "eps_l2 and eps_rms must be finite and >= 0");
  if (a.C > (int64_t(1) << 30) || op_rmsnorm_points((int)a.C) < 1)
    return fail(HYENAND_ERR_UNSUPPORTED, "C = %lld channels exceed the output norm's tile", (long long)a.C);
  size_t n = (size_t)a.lines;
  for (int d = 0; d < a.ndim; ++d) n *= (size_t)a.L[d];
  const size_t nb = n * es;
  size_t kpts = 1;
  for (int d = 0; d < a.ndim; ++d) kpts *= (size_t)(a.centered ? 2 * a.L[d] - 1 : a.L[d]);
  const size_t bytes[8] = {nb, nb, nb, (size_t)a.lines * kpts * es, (size_t)a.C * es, (size_t)a.C * es,
                           (size_t)a.C * es, nb};
  for (int i = 0; i < 7; ++i)
    if (overlaps(y, nb, ptrs[i], bytes[i])) return fail(HYENAND_ERR_INVALID_ARGUMENT, "y overlaps %s", pn[i]);
  const Plan p = choose_plan(a);
  if (p == PLAN_NONE || p == PLAN_EMBED)
    return fail(HYENAND_ERR_UNSUPPORTED, "no plan for this shape in the operator");
  const size_t sb = op_scale_bytes(a);
  const size_t per = bytes_per_line(a, p);
  if (!workspace || workspace_bytes < sb + per)
    return fail(HYENAND_ERR_WORKSPACE_TOO_SMALL, "the operator needs at least %zu workspace bytes, got %zu", sb + per,
                workspace ? workspace_bytes : (size_t)0);
  if ((uintptr_t)workspace % 16 != 0) return fail(HYENAND_ERR_INVALID_ARGUMENT, "workspace is not 16-byte aligned");
  for (int i = 0; i < 8; ++i)
    if (overlaps(workspace, workspace_bytes, ptrs[i], bytes[i]))
      return fail(HYENAND_ERR_INVALID_ARGUMENT, "workspace overlaps %s", pn[i]);
  const int64_t npos = (int64_t)(n / (size_t)a.lines);
  const int64_t B = a.lines / a.C;
  float* sc = (float*)workspace;
  a.x1 = q; a.v = kin; a.x2 = vin; a.k = k; a.D = D; a.y = y;
  a.ws = (char*)workspace + sb;
  a.ws_bytes = workspace_bytes - sb;
  a.act = true;
  a.act_in.s = sc;
  a.act_in.w_in = w_in;
  a.act_in.npos = npos;
  const hipStream_t s = (hipStream_t)stream;
  clear_pending_error();
  hipError_t err = launch_op_prologue(q, kin, sc, B, (int)a.C, npos, a.bf16, eps_l2, eps_rms, s);
  if (err == hipSuccess) err = launch_plan(a, p, per, s);
  if (err == hipSuccess) err = launch_op_rmsnorm(y, w_out, B, (int)a.C, npos, a.bf16, eps_rms, s);
  if (err != hipSuccess) return fail(HYENAND_ERR_HIP, "HIP error %d: %s", (int)err, hipGetErrorString(err));
  return HYENAND_OK;
}

}  // namespace

extern "C" {

hyenand_status hyenand_fftconv(const void* x1, const void* x2, const void* v, const void* k, const void* D,
                               void* y, int ndim, const int64_t* dims, hyenand_pad_mode pad_mode, hyenand_dtype dtype,
                               void* workspace, size_t workspace_bytes, void* stream) {
  return forward(x1, x2, v, k, D, y, ndim, dims, pad_mode, dtype, workspace, workspace_bytes, stream, false);
}

hyenand_status hyenand_fftconv_shared_k(const void* x1, const void* x2, const void* v, const void* k,
                                        const void* D, void* y, int ndim, const int64_t* dims, hyenand_pad_mode pad_mode,
                                        hyenand_dtype dtype, void* workspace, size_t workspace_bytes, void* stream) {
  return forward(x1, x2, v, k, D, y, ndim, dims, pad_mode, dtype, workspace, workspace_bytes, stream, true);
}

hyenand_status hyenand_fftconv_modal(const void* x1, const void* x2, const void* v, const float* log_mag,
                                     const float* angle, const float* res_re, const float* res_im, int order,
                                     const void* D, void* y, int ndim, const int64_t* dims,
                                     hyenand_pad_mode pad_mode, hyenand_dtype dtype, void* workspace,
                                     size_t workspace_bytes, void* stream) {
  const ModalIn md{log_mag, angle, res_re, res_im, order};
  return forward(x1, x2, v, nullptr, D, y, ndim, dims, pad_mode, dtype, workspace, workspace_bytes, stream, true,
                 &md);
}

hyenand_status hyenand_kernel_spectrum_size(int ndim, const int64_t* dims, hyenand_pad_mode pad_mode,
                                            hyenand_dtype dtype, size_t* bytes_out) {
  if (!bytes_out) return fail(HYENAND_ERR_INVALID_ARGUMENT, "bytes_out is NULL");
  FftConvArgs a;
  const hyenand_status st = spectrum_shape(ndim, dims, pad_mode, dtype, &a);
  if (st != HYENAND_OK) return st;
  *bytes_out = fused2d_khat_bytes(a);
  return HYENAND_OK;
}

hyenand_status hyenand_kernel_spectrum(const void* k, void* khat, size_t khat_bytes, int ndim, const int64_t* dims,
                                       hyenand_pad_mode pad_mode, hyenand_dtype dtype, void* stream) {
  g_last_error.clear();
  FftConvArgs a;
  const hyenand_status st = spectrum_shape(ndim, dims, pad_mode, dtype, &a);
  if (st != HYENAND_OK) return st;
  if (!k || !khat) return fail(HYENAND_ERR_INVALID_ARGUMENT, "k or khat is NULL");
  if ((uintptr_t)k % 16 != 0 || (uintptr_t)khat % 16 != 0)
    return fail(HYENAND_ERR_INVALID_ARGUMENT, "k and khat must be 16-byte aligned");
  const size_t need = fused2d_khat_bytes(a);
  if (khat_bytes < need)
    return fail(HYENAND_ERR_WORKSPACE_TOO_SMALL, "khat needs %zu bytes, got %zu", need, khat_bytes);
  const size_t kb = (size_t)a.C * (size_t)a.L[0] * (size_t)a.L[1] * (a.bf16 ? 2 : 4);
  if (overlaps(k, kb, khat, need)) return fail(HYENAND_ERR_INVALID_ARGUMENT, "khat overlaps k");
  a.k = k;
  a.khat = (float2*)khat;
  a.khat_pass = 1;
  clear_pending_error();
  const hipError_t err = launch_fused2d(a, (hipStream_t)stream);
  if (err != hipSuccess) return fail(HYENAND_ERR_HIP, "HIP error %d: %s", (int)err, hipGetErrorString(err));
  return HYENAND_OK;
}

hyenand_status hyenand_fftconv_spectrum(const void* x1, const void* x2, const void* v, const void* khat,
                                        size_t khat_bytes, const void* D, void* y, int ndim, const int64_t* dims,
                                        hyenand_pad_mode pad_mode, hyenand_dtype dtype, void* stream) {
  g_last_error.clear();
  FftConvArgs a;
  const hyenand_status st = spectrum_shape(ndim, dims, pad_mode, dtype, &a);
  if (st != HYENAND_OK) return st;
  const void* ptrs[6] = {x1, x2, v, khat, D, y};
  const char* pn[6] = {"x1", "x2", "v", "khat", "D", "y"};
  const size_t es = a.bf16 ? 2 : 4;
  for (int i = 0; i < 6; ++i) {
    if (!ptrs[i]) return fail(HYENAND_ERR_INVALID_ARGUMENT, "%s is NULL", pn[i]);
    if ((uintptr_t)ptrs[i] % (i == 4 ? es : 16) != 0)
      return fail(HYENAND_ERR_INVALID_ARGUMENT, "%s is not aligned", pn[i]);
  }
  const size_t need = fused2d_khat_bytes(a);
  if (khat_bytes < need)
    return fail(HYENAND_ERR_WORKSPACE_TOO_SMALL, "khat needs %zu bytes, got %zu", need, khat_bytes);
  const size_t nb = (size_t)a.lines * (size_t)a.L[0] * (size_t)a.L[1] * es;
  const size_t bytes[5] = {nb, nb, nb, need, (size_t)a.C * es};
  for (int i = 0; i < 5; ++i)
    if (overlaps(y, nb, ptrs[i], bytes[i])) return fail(HYENAND_ERR_INVALID_ARGUMENT, "y overlaps %s", pn[i]);
  a.x1 = x1; a.x2 = x2; a.v = v; a.D = D; a.y = y;
  a.khat = (float2*)const_cast<void*>(khat);
  a.khat_pass = 2;
  clear_pending_error();
  const hipError_t err = launch_fused2d(a, (hipStream_t)stream);
  if (err != hipSuccess) return fail(HYENAND_ERR_HIP, "HIP error %d: %s", (int)err, hipGetErrorString(err));
  return HYENAND_OK;
}

hyenand_status hyenand_fftconv_backward_workspace_size(int ndim, const int64_t* dims, hyenand_pad_mode pad_mode, hyenand_dtype dtype,
                                                       size_t* bytes_out) {
  if (!bytes_out) return fail(HYENAND_ERR_INVALID_ARGUMENT, "bytes_out is NULL");
  FftConvArgs a;
  hyenand_status st = parse_shape(ndim, dims, pad_mode, dtype, &a);
  if (st != HYENAND_OK) return st;
  const BwdPlan p = choose_bwd_plan(a);
  if (p == BWD_NONE) return fail(HYENAND_ERR_UNSUPPORTED, "no backward plan for this shape");
  if (p == BWD_EMBED) {
    Embedded m;
    embedded_problem(a, &m);
    *bytes_out = 9 * m.tensor + bwd_partial_bytes(m.e, m.p) + bwd_recommended_spectra(m.e, m.p);
    return HYENAND_OK;
  }
  *bytes_out = bwd_partial_bytes(a, p) + bwd_recommended_spectra(a, p);
  return HYENAND_OK;
}

hyenand_status hyenand_fftconv_backward_workspace_min(int ndim, const int64_t* dims, hyenand_pad_mode pad_mode, hyenand_dtype dtype,
                                                      size_t* bytes_out) {
  if (!bytes_out) return fail(HYENAND_ERR_INVALID_ARGUMENT, "bytes_out is NULL");
  FftConvArgs a;
  hyenand_status st = parse_shape(ndim, dims, pad_mode, dtype, &a);
  if (st != HYENAND_OK) return st;
  const BwdPlan p = choose_bwd_plan(a);
  if (p == BWD_NONE) return fail(HYENAND_ERR_UNSUPPORTED, "no backward plan for this shape");
  if (p == BWD_EMBED) {
    Embedded m;
    embedded_problem(a, &m);
    *bytes_out = 9 * m.tensor + bwd_partial_bytes(m.e, m.p) + bwd_bytes_per_line(m.e, m.p);
    return HYENAND_OK;
  }
  *bytes_out = bwd_partial_bytes(a, p) + bwd_bytes_per_line(a, p);
  return HYENAND_OK;
}

hyenand_status hyenand_fftconv_backward(const void* x1, const void* x2, const void* v, const void* k,
                                        const void* D, const void* gy, void* gx1, void* gx2, void* gv, void* gk,
                                        void* gD, int ndim, const int64_t* dims, hyenand_pad_mode pad_mode, hyenand_dtype dtype,
                                        void* workspace, size_t workspace_bytes, void* stream) {
  g_last_error.clear();
  FftConvArgs a;
  hyenand_status st = parse_shape(ndim, dims, pad_mode, dtype, &a);
  if (st != HYENAND_OK) return st;
  const void* ins[6] = {x1, x2, v, k, gy, D};
  const char* in_names[6] = {"x1", "x2", "v", "k", "gy", "D"};
  void* outs[5] = {gx1, gx2, gv, gk, gD};
  const char* out_names[5] = {"gx1", "gx2", "gv", "gk", "gD"};
  for (int i = 0; i < 6; ++i)
    if (!ins[i]) return fail(HYENAND_ERR_INVALID_ARGUMENT, "%s is NULL", in_names[i]);
  for (int i = 0; i < 5; ++i)
    if (!outs[i]) return fail(HYENAND_ERR_INVALID_ARGUMENT, "%s is NULL", out_names[i]);
  const size_t es = a.bf16 ? 2 : 4;
  size_t n = (size_t)a.lines, kn = (size_t)a.lines;  // elements of the data and of the kernel
  for (int d = 0; d < a.ndim; ++d) {
    n *= (size_t)a.L[d];
    kn *= (size_t)(a.centered ? 2 * a.L[d] - 1 : a.L[d]);
  }
  size_t in_bytes[6], out_bytes[5];
  for (int i = 0; i < 6; ++i) in_bytes[i] = i == 5 ? (size_t)a.C * es : (i == 3 ? kn : n) * es;
  for (int i = 0; i < 5; ++i) out_bytes[i] = i == 4 ? (size_t)a.C * es : (i == 3 ? kn : n) * es;
  for (int i = 0; i < 6; ++i)
    if ((uintptr_t)ins[i] % (i == 5 ? es : 16) != 0)
      return fail(HYENAND_ERR_INVALID_ARGUMENT, "%s is not aligned", in_names[i]);
  for (int i = 0; i < 5; ++i)
    if ((uintptr_t)outs[i] % (i == 4 ? es : 16) != 0)
      return fail(HYENAND_ERR_INVALID_ARGUMENT, "%s is not aligned", out_names[i]);
  for (int i = 0; i < 5; ++i) {
    for (int j = 0; j < 6; ++j)
      if (overlaps(outs[i], out_bytes[i], ins[j], in_bytes[j]))
        return fail(HYENAND_ERR_INVALID_ARGUMENT, "%s overlaps %s", out_names[i], in_names[j]);
    for (int j = 0; j < i; ++j)
      if (overlaps(outs[i], out_bytes[i], outs[j], out_bytes[j]))
        return fail(HYENAND_ERR_INVALID_ARGUMENT, "%s overlaps %s", out_names[i], out_names[j]);
  }
  const BwdPlan p = choose_bwd_plan(a);
  if (p == BWD_NONE) return fail(HYENAND_ERR_UNSUPPORTED, "no backward plan for this shape");
  Embedded m;
  if (p == BWD_EMBED) embedded_problem(a, &m);
  const size_t pbytes = p == BWD_EMBED ? 0 : bwd_partial_bytes(a, p);
  const size_t need = p == BWD_EMBED ? 9 * m.tensor + bwd_partial_bytes(m.e, m.p) + bwd_bytes_per_line(m.e, m.p)
                                     : pbytes + bwd_bytes_per_line(a, p);
  if (!workspace || workspace_bytes < need)
    return fail(HYENAND_ERR_WORKSPACE_TOO_SMALL, "backward needs at least %zu workspace bytes, got %zu", need,
                workspace ? workspace_bytes : (size_t)0);
  if ((uintptr_t)workspace % 16 != 0) return fail(HYENAND_ERR_INVALID_ARGUMENT, "workspace is not 16-byte aligned");
  for (int j = 0; j < 6; ++j)
    if (overlaps(workspace, workspace_bytes, ins[j], in_bytes[j]))
      return fail(HYENAND_ERR_INVALID_ARGUMENT, "workspace overlaps %s", in_names[j]);
  for (int j = 0; j < 5; ++j)
    if (overlaps(workspace, workspace_bytes, outs[j], out_bytes[j]))
      return fail(HYENAND_ERR_INVALID_ARGUMENT, "workspace overlaps %s", out_names[j]);
  FftConvBwdArgs b;
  b.f = a;
  b.f.x1 = x1; b.f.x2 = x2; b.f.v = v; b.f.k = k; b.f.D = D;
  b.gy = gy;
  b.gx1 = gx1; b.gx2 = gx2; b.gv = gv; b.gk = gk; b.gD = gD;
  b.partial = (float*)workspace;
  const hipStream_t s = (hipStream_t)stream;
  hipError_t err = hipSuccess;
  clear_pending_error();
  if (p == BWD_EMBED) {
    char* w = (char*)workspace;
    void* e[9];
    for (int i = 0; i < 9; ++i) e[i] = w + i * m.tensor;
    void* const ein[5] = {e[0], e[1], e[2], e[3], e[4]};  // x1, x2, v, gy, k
    void* const eout[4] = {e[5], e[6], e[7], e[8]};       // gx1, gx2, gv, gk
    err = launch_embed(b.f, gy, ein, s);
    if (err != hipSuccess) return fail(HYENAND_ERR_HIP, "HIP error %d: %s", (int)err, hipGetErrorString(err));
    const hyenand_status inner =
        hyenand_fftconv_backward(e[0], e[1], e[2], e[4], D, e[3], e[5], e[6], e[7], e[8], gD, m.nd, m.dims,
                                 HYENAND_PAD_CIRCULAR, dtype, w + 9 * m.tensor, workspace_bytes - 9 * m.tensor, stream);
    if (inner != HYENAND_OK) return inner;
    err = launch_extract(b.f, eout, gx1, gx2, gv, gk, s);
  } else if (p == BWD_FUSED) {
    err = launch_backward(b, s);
  } else if (p == BWD_MIXED) {
    err = launch_mixed_backward(b, s);
    if (err == hipSuccess) err = launch_backward_reduce(b, 1, s);
  } else {
    // the spectra of each chunk follow the gD sums in the workspace
    FftConvArgs sa = b.f;
    sa.ws = (char*)workspace + pbytes;
    sa.ws_bytes = workspace_bytes - pbytes;
    const size_t per = bwd_bytes_per_line(a, p);
    if (p == BWD_MULTIPASS)
      err = run_chunked(sa, per, s, [&b](int64_t l0, int64_t nl, void* ws, hipStream_t st) {
        return launch_backward_mp(b, l0, nl, ws, st);
      });
    else
      err = run_chunked(sa, per, s, [&b](int64_t l0, int64_t nl, void* ws, hipStream_t st) {
        return launch_backward_fs(b, l0, nl, ws, st);
      });
    if (err == hipSuccess) err = launch_backward_reduce(b, bwd_partials_per_line(a, p), s);
  }
  if (err != hipSuccess) return fail(HYENAND_ERR_HIP, "HIP error %d: %s", (int)err, hipGetErrorString(err));
  return HYENAND_OK;
}

const char* hyenand_status_string(hyenand_status status) {
  switch (status) {
    case HYENAND_OK: return "ok";
    case HYENAND_ERR_INVALID_ARGUMENT: return "invalid argument";
    case HYENAND_ERR_UNSUPPORTED: return "unsupported shape";
    case HYENAND_ERR_WORKSPACE_TOO_SMALL: return "workspace too small";
    case HYENAND_ERR_HIP: return "HIP error";
    default: return "unknown status";
  }
}

const char* hyenand_last_error(void) { return g_last_error.c_str(); }

hyenand_status hyenand_operator(const void* q, const void* kin, const void* vin, const void* k, const void* D,
                                const void* w_in, const void* w_out, float eps_l2, float eps_rms, void* y, int ndim,
                                const int64_t* dims, hyenand_pad_mode pad_mode, hyenand_dtype dtype, void* workspace, size_t workspace_bytes,
                                void* stream) {
  return operator_fwd(q, kin, vin, k, D, w_in, w_out, eps_l2, eps_rms, y, ndim, dims, pad_mode, dtype, workspace,
                      workspace_bytes, stream);
}

hyenand_status hyenand_operator_workspace_size(int ndim, const int64_t* dims, hyenand_pad_mode pad_mode, hyenand_dtype dtype,
                                               size_t* bytes_out) {
  if (!bytes_out) return fail(HYENAND_ERR_INVALID_ARGUMENT, "bytes_out is NULL");
  FftConvArgs a;
  hyenand_status st = parse_shape(ndim, dims, pad_mode, dtype, &a);
  if (st != HYENAND_OK) return st;
  const Plan p = choose_plan(a);
  if (p == PLAN_NONE || p == PLAN_EMBED)
    return fail(HYENAND_ERR_UNSUPPORTED, "no plan for this shape in the operator");
  *bytes_out = op_scale_bytes(a) + recommended_ws(a, p);
  return HYENAND_OK;
}

hyenand_status hyenand_kernel_synth(const float* omega0, const float* W1, const float* Wh, const float* bias,
                                    const float* gamma, const float* beta, const float* Wout, const float* window,
                                    int window_kind, int hidden, int layers, void* k, int ndim, const int64_t* dims,
                                    hyenand_pad_mode pad_mode, hyenand_dtype dtype, void* stream) {
  if (ndim < 1 || ndim > 3) return fail(HYENAND_ERR_INVALID_ARGUMENT, "ndim must be 1, 2 or 3 (got %d)", ndim);
  if (!dims) return fail(HYENAND_ERR_INVALID_ARGUMENT, "dims is NULL");
  if (pad_mode != HYENAND_PAD_LINEAR && pad_mode != HYENAND_PAD_CIRCULAR && pad_mode != HYENAND_PAD_CENTERED)
    return fail(HYENAND_ERR_INVALID_ARGUMENT, "pad_mode must be 0, 1 or 2, got %d", pad_mode);
  if (dtype != HYENAND_DTYPE_F32 && dtype != HYENAND_DTYPE_BF16)
    return fail(HYENAND_ERR_INVALID_ARGUMENT, "dtype must be 0 (f32) or 1 (bf16), got %d", dtype);
  if (window_kind != 0 && window_kind != 1)
    return fail(HYENAND_ERR_INVALID_ARGUMENT, "window_kind must be 0 (gaussian) or 1 (exponential), got %d",
                window_kind);
  if (!synth_hidden_supported(hidden))
    return fail(HYENAND_ERR_UNSUPPORTED, "hidden width must be 32, 64 or 128 (got %d)", hidden);
  if (layers < 1 || layers > 16) return fail(HYENAND_ERR_UNSUPPORTED, "layers must be 1..16 (got %d)", layers);
  if (!omega0 || !W1 || !Wout || !window || !k || (layers > 1 && !Wh))
    return fail(HYENAND_ERR_INVALID_ARGUMENT, "a required pointer is NULL");
  if ((gamma == nullptr) != (beta == nullptr))
    return fail(HYENAND_ERR_INVALID_ARGUMENT, "gamma and beta must both be given or both be NULL");
  SynthArgs a;
  memset(&a, 0, sizeof a);
  int64_t total = 1;
  for (int i = 0; i < ndim + 2; ++i) {
    if (dims[i] < 1) return fail(HYENAND_ERR_INVALID_ARGUMENT, "dims[%d] = %lld must be >= 1", i, (long long)dims[i]);
    if (dims[i] > (int64_t(1) << 30)) return fail(HYENAND_ERR_UNSUPPORTED, "extent too large");
  }
  if (dims[1] > (1 << 20)) return fail(HYENAND_ERR_UNSUPPORTED, "C = %lld is too large", (long long)dims[1]);
  a.nd = ndim;
  a.npos = 1;
  for (int d = 0; d < ndim; ++d) {
    a.Lc[d] = dims[2 + d];
    a.KL[d] = pad_mode == HYENAND_PAD_CENTERED ? 2 * dims[2 + d] - 1 : dims[2 + d];
    if (a.npos > (int64_t(1) << 40) / a.KL[d]) return fail(HYENAND_ERR_UNSUPPORTED, "kernel grid too large");
    a.npos *= a.KL[d];
  }
  a.C = (int)dims[1];
  a.nb = gamma ? dims[0] : 1;
  total = a.nb * a.C;
  if (total > (int64_t(1) << 46) / a.npos) return fail(HYENAND_ERR_UNSUPPORTED, "kernel tensor too large");
  total *= a.npos;
  if ((a.npos + 15) / 16 * a.nb / 8 >= (int64_t(1) << 31)) return fail(HYENAND_ERR_UNSUPPORTED, "grid too large");
  const size_t es = dtype == HYENAND_DTYPE_BF16 ? 2 : 4;
  const float* ptrs[] = {omega0, W1, Wh, bias, gamma, beta, Wout, window};
  const char* names[] = {"omega0", "W1", "Wh", "bias", "gamma", "beta", "Wout", "window"};
  const size_t H = (size_t)hidden, J = (size_t)layers, C = (size_t)a.C;
  const size_t counts[] = {H, (size_t)ndim * H, (J - 1) * H * H, J * H, (size_t)a.nb * J * H,
                           (size_t)a.nb * J * H, H * C, window_kind == 0 ? (size_t)ndim * C : C};
  if ((uintptr_t)k % es != 0) return fail(HYENAND_ERR_INVALID_ARGUMENT, "k is not aligned to its element size");
  for (int i = 0; i < 8; ++i) {
    if (!ptrs[i] || counts[i] == 0) continue;
    // Wh, gamma and beta are read four floats at a time
    const size_t align = (i == 2 || i == 4 || i == 5) ? 16 : 4;
    if ((uintptr_t)ptrs[i] % align != 0)
      return fail(HYENAND_ERR_INVALID_ARGUMENT, "%s is not %zu-byte aligned", names[i], align);
    if (overlaps(k, (size_t)total * es, ptrs[i], counts[i] * 4))
      return fail(HYENAND_ERR_INVALID_ARGUMENT, "k overlaps %s", names[i]);
  }
  a.omega0 = omega0;
  a.W1 = W1;
  a.Wh = layers > 1 ? Wh : nullptr;
  a.bias = bias;
  a.gamma = gamma;
  a.beta = beta;
  a.Wout = Wout;
  a.win = window;
  a.k = k;
  a.mode = pad_mode;
  a.J = layers;
  a.wkind = window_kind;
  a.hidden = hidden;
  clear_pending_error();
  hipError_t err = launch_synth(a, dtype == HYENAND_DTYPE_BF16, (hipStream_t)stream);
  if (err != hipSuccess) return fail(HYENAND_ERR_HIP, "HIP error %d: %s", (int)err, hipGetErrorString(err));
  return HYENAND_OK;
}

hyenand_status hyenand_modal_filter(const float* log_mag, const float* angle, const float* res_re,
                                    const float* res_im, int order, void* k, int64_t C, int64_t L, hyenand_dtype dtype,
                                    void* stream) {
  if (dtype != HYENAND_DTYPE_F32 && dtype != HYENAND_DTYPE_BF16)
    return fail(HYENAND_ERR_INVALID_ARGUMENT, "dtype must be 0 (f32) or 1 (bf16), got %d", dtype);
  if (C < 1 || L < 1 || order < 1)
    return fail(HYENAND_ERR_INVALID_ARGUMENT, "C, L and order must be >= 1 (got %lld, %lld, %d)", (long long)C,
                (long long)L, order);
  if (order > 256 || C > 65535 || L > (int64_t(1) << 29))
    return fail(HYENAND_ERR_UNSUPPORTED, "order <= 256, C <= 65535 and L <= 2^29 are supported");
  const float* ptrs[] = {log_mag, angle, res_re, res_im};
  const char* names[] = {"log_mag", "angle", "res_re", "res_im"};
  const size_t es = dtype == HYENAND_DTYPE_BF16 ? 2 : 4;
  if (!k) return fail(HYENAND_ERR_INVALID_ARGUMENT, "k is NULL");
  if ((uintptr_t)k % es != 0) return fail(HYENAND_ERR_INVALID_ARGUMENT, "k is not aligned to its element size");
  for (int i = 0; i < 4; ++i) {
    if (!ptrs[i]) return fail(HYENAND_ERR_INVALID_ARGUMENT, "%s is NULL", names[i]);
    if ((uintptr_t)ptrs[i] % 4 != 0) return fail(HYENAND_ERR_INVALID_ARGUMENT, "%s is not 4-byte aligned", names[i]);
    if (overlaps(k, (size_t)C * L * es, ptrs[i], (size_t)C * order * 4))
      return fail(HYENAND_ERR_INVALID_ARGUMENT, "k overlaps %s", names[i]);
  }
  clear_pending_error();
  hipError_t err = launch_modal(log_mag, angle, res_re, res_im, k, C, order, L, dtype == HYENAND_DTYPE_BF16,
                                (hipStream_t)stream);
  if (err != hipSuccess) return fail(HYENAND_ERR_HIP, "HIP error %d: %s", (int)err, hipGetErrorString(err));
  return HYENAND_OK;
}

int hyenand_version(void) { return 400; }

}  // extern "C"
