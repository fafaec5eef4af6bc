// Internal interface between the C-ABI front end (hyenand.cpp) and the
// kernel translation units.  Not part of the public header.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "fft_device.hpp"

namespace hyenand {

// A modal filter generated inside the transform kernels instead of read:
// k[c, t] = Re sum_{m < M} (re + i im)[c, m] exp((a + i th)[c, m] t), the
// parameters [C, M] fp32 (hyenand_fftconv_modal).  M = 0: k is read.
struct ModalIn {
  const float *a, *th, *re, *im;
  int M;
};
constexpr int kMaxFusedModalOrder = 32;

// One validated call, after unit axes have been squeezed out.
struct FftConvArgs {
  const void *x1, *x2, *v, *k, *D;
  void* y;
  int64_t lines;  // B * C
  int64_t C;
  int ndim;       // 1..3, every remaining axis has L >= 2 (or the 1D L = 1 case)
  int64_t L[3];   // grid extents of the squeezed problem
  int64_t P[3];   // transform extents: 2L (linear) or L (circular)
  bool circular;
  bool centered;  // linear transform grid, k on the double grid of 2 L_d - 1 points per axis
  bool rl;        // some L_d is not a power of two (P_d = pow2 >= 2 L_d - 1)
  bool periodic;  // circular mode with rl: k repeated periodically on the non-circular grid
  bool bf16;
  int kC;         // 0: k is [B, C, L...]; C: one kernel per channel, k is [C, L...]
  void* ws;       // device workspace (multi-pass plans)
  size_t ws_bytes;
  bool act;       // HyenaND operator: x1, v, x2 are q, kin, vin (see Gates)
  ActIn act_in;
  ModalIn modal;  // modal.M > 0: k generated per channel (four-step plan only)
  float2* khat;   // non-null: the fused 2D plan transforms each channel's k
                  // once into this region (kC = C; fused2d_khat_bytes)
  int khat_pass;  // with khat: 0 spectra then images, 1 spectra only,
                  // 2 images only (spectra written by an earlier call)
};

// Drop the calling thread's pending (non-sticky) HIP error, left by work
// before a call, so that the hipGetLastError after each of the call's
// launches reports that launch only.
inline void clear_pending_error() { (void)hipGetLastError(); }

// single pass (the padded problem of one line fits in LDS)
bool fused1d_supported(int64_t P);
hipError_t launch_fused1d(const FftConvArgs& a, hipStream_t s);
bool fused2d_supported(int64_t P0, int64_t P1);
hipError_t launch_fused2d(const FftConvArgs& a, hipStream_t s);
// bytes of the per-channel kernel spectra of a fused 2D call with one kernel
// per channel (C x P0 x P1/2 complex fp32); 0 where that path does not apply
// (centered or non-power-of-two grids, the operator)
size_t fused2d_khat_bytes(const FftConvArgs& a);

// single pass for grid extents that are not powers of two on power-of-two
// transforms (P_d = the smallest power of two >= 2 L_d - 1; a circular axis
// as the centred convolution of the periodically repeated kernel)
bool fused_rl_supported(const FftConvArgs& a);
hipError_t launch_fused_rl(const FftConvArgs& a, hipStream_t s);

// single pass on mixed-radix transform grids (extents with prime factors 2,
// 3, 5, 7 up to 4096 points per image): circular axes of such extents on
// their own points, the others on the smallest such P_d >= 2 L_d - 1
bool mixed_supported(const FftConvArgs& a);
bool mixed_preferred(const FftConvArgs& a);  // faster than the power-of-two kernels
hipError_t launch_mixed(const FftConvArgs& a, hipStream_t s);

// multi-pass 2D/3D (lines along each axis; spectra staged in the workspace).
// One call runs every pass over lines [line0, line0 + nl) with their spectra
// in ws (nl times the bytes per line), all on stream s.
bool multipass_supported(const FftConvArgs& a);
size_t multipass_bytes_per_line(const FftConvArgs& a);
hipError_t launch_multipass(const FftConvArgs& a, int64_t line0, int64_t nl, void* ws, hipStream_t s);
// three-pass 3D plan (conv_slab.hip) for grids whose planes fit in LDS: the
// slab passes before (inverse = false) and after (inverse = true) the
// multi-pass core, on the same workspace layout; launch_multipass takes it
// where slab3d_supported (HYENAND_SLAB=0 turns it off)
bool slab3d_supported(const FftConvArgs& a);
hipError_t launch_slab3d(const FftConvArgs& a, int64_t line0, int64_t nl, void* ws, bool inverse, hipStream_t s);

// backward
struct FftConvBwdArgs {
  FftConvArgs f;  // shapes and the forward inputs (f.y unused)
  const void* gy;
  void *gx1, *gx2, *gv, *gk, *gD;
  float* partial;  // workspace: the sums of h u for gD
};
// single pass per line (1D up to P = 8192, 2D where the half spectra of u, k
// and h fit in LDS); one float of partial per line; launches the gD reduction
bool fused_backward_supported(const FftConvArgs& a);
hipError_t launch_backward(const FftConvBwdArgs& b, hipStream_t s);
// multi-pass 2D/3D and four-step 1D: one call per chunk of lines [line0,
// line0 + nl) with their three spectra in ws; partial holds the given number
// of sums per line; launch_backward_reduce adds them into gD afterwards
size_t backward_mp_bytes_per_line(const FftConvArgs& a);
int64_t backward_mp_partials_per_line(const FftConvArgs& a);
hipError_t launch_backward_mp(const FftConvBwdArgs& b, int64_t line0, int64_t nl, void* ws, hipStream_t s);
bool backward_fs_supported(const FftConvArgs& a);
size_t backward_fs_bytes_per_line(const FftConvArgs& a);
int64_t backward_fs_partials_per_line(const FftConvArgs& a);
hipError_t launch_backward_fs(const FftConvBwdArgs& b, int64_t line0, int64_t nl, void* ws, hipStream_t s);
hipError_t launch_backward_reduce(const FftConvBwdArgs& b, int64_t partials_per_line, hipStream_t s);
// mixed-radix single pass (conv_mixed.hip) on the forward's transform grid,
// grids of up to about 3000 points; one float of partial per line
bool mixed_backward_supported(const FftConvArgs& a);
hipError_t launch_mixed_backward(const FftConvBwdArgs& b, hipStream_t s);
// centred and non-power-of-two extents (conv_embed.hip): embed x1, x2, v, gy
// and k in the transform grid (e[0..4], lines * prod P elements each), run
// the circular backward there, extract gx1, gx2, gv, gk (from e[0..3])
int64_t embed_grid_elems(const FftConvArgs& a);
hipError_t launch_embed(const FftConvArgs& a, const void* gy, void* const (&e)[5], hipStream_t s);
hipError_t launch_extract(const FftConvArgs& a, void* const (&e)[4], void* gx1, void* gx2, void* gv, void* gk,
                          hipStream_t s);
// forward of the same shapes: x1, x2, v, k embedded (e[0..3]), y extracted
hipError_t launch_embed_fwd(const FftConvArgs& a, void* const (&e)[4], hipStream_t s);
hipError_t launch_extract_y(const FftConvArgs& a, const void* ey, void* y, hipStream_t s);

// multi-pass 1D (four-step split of the long line); one call per chunk of
// lines, as for launch_multipass
bool fourstep_supported(const FftConvArgs& a);
size_t fourstep_bytes_per_line(const FftConvArgs& a);
hipError_t launch_fourstep(const FftConvArgs& a, int64_t line0, int64_t nl, void* ws, hipStream_t s);

// HyenaND operator: the normalisations across channels (op_norm.hip).
// op_rmsnorm_points: grid points per rmsnorm workgroup for C channels (0 if C
// is too large for the LDS tile).
int op_rmsnorm_points(int C);
hipError_t launch_op_prologue(const void* q, const void* kin, float* s, int64_t B, int C, int64_t npos, bool bf16,
                              float eps_l2, float eps_rms, hipStream_t st);
hipError_t launch_op_rmsnorm(void* y, const void* w_out, int64_t B, int C, int64_t npos, bool bf16, float eps_rms,
                             hipStream_t st);

// Kernel synthesis (synth.hip): the SIREN + FiLM + window kernel on the kernel
// grid of a convolution, k [nb, C, KL...] in the storage type.
struct SynthArgs {
  const float *omega0, *W1, *Wh, *bias, *gamma, *beta, *Wout, *win;
  void* k;
  int nd;         // axes of the grid, 1..3 (unit axes kept)
  int64_t KL[3];  // kernel-grid extents: L (linear, circular) or 2L - 1 (centered)
  int64_t Lc[3];  // convolution grid extents, which fix the coordinates
  int mode;       // 0 linear, 1 circular, 2 centered
  int C, J, wkind, hidden;
  int64_t npos;   // prod KL
  int64_t nb;     // kernels written: B (FiLM given) or 1
  int resident;   // set by launch_synth: every weight staged in LDS at once
  int cc;         // set by launch_synth: output channels per streamed chunk
  int stream_floats;  // set by launch_synth: LDS floats of the streamed region
  int film_lds;   // set by launch_synth: FiLM rows of every sample kept in LDS
};
bool synth_hidden_supported(int hidden);

// Modal filter generation (modal.hip): k[c, t] = Re sum_m R lambda^t,
// parameters [C, M], k [C, L] in the storage type.
hipError_t launch_modal(const float* a, const float* th, const float* re, const float* im, void* k, int64_t C,
                        int M, int64_t L, bool bf16, hipStream_t s);
hipError_t launch_synth(const SynthArgs& a, bool bf16, hipStream_t s);

}  // namespace hyenand
