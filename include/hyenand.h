/*
 * hyenand.h -- C ABI of the MI355X (gfx950) gated N-D FFT long convolution.
 *
 * The operation is the long convolution at the heart of the HyenaND operator
 * (Eq. (HyenaND), section 3.2 "The HyenaND Operator") together with its two
 * gates and the per-channel shortcut of the gated Hyena mixer (Def. A.2
 * "Hyena mixer" and Def. A.3 "Gated Hyena mixer" in the appendix "Gated Hyena
 * Computes Separable Attention").  For every sample b, channel c and output
 * index n of an L1 x ... x LN grid (N = 1, 2 or 3):
 *
 *     u = x1 * v                                            (inner gate)
 *     linear:   conv[n] = sum_{m: 0 <= m_d <= n_d} k[b,c,m] u[b,c,n-m]
 *     circular: conv[n] = sum_{m}   k[b,c,m] u[b,c,(n-m) mod L]
 *     y[b,c,n] = x2[b,c,n] * (conv[n] + D[c] * u[b,c,n])    (shortcut, outer gate)
 *
 * Each sample carries its own kernel k[b, c] (section 3.2.2, "FFT path
 * preservation": B kernels, one N-D FFT convolution per input).  "linear" is
 * the non-circular convolution of section 3.2.1 ("Support for circular and
 * non-circular convolutions"): zero-padding to a transform of 2 L_d per axis
 * (at least 2L-1, as the appendix "Hardware Context and IO Profile" requires)
 * and cropping the first L_d outputs of every axis; index 0 of k is the zero
 * displacement.  "circular" treats the grid as a torus (transform L_d).
 * "centered" is the paper's own non-circular form (section 3.2.1): k is
 * evaluated on the double grid of 2 L_d - 1 points per axis, index L_d - 1 is
 * the zero displacement, and
 *     conv[n] = sum_m k[n - m + (L - 1)] u[m]      (every m of the grid),
 * so every displacement between two grid points has its own weight; the
 * transform is 2 L_d per axis and the output is cropped as in "linear".
 *
 * The library computes this with fused FFT kernels on the GPU (fp32 compute).
 * It allocates no memory on the call path and keeps no pointer after a call;
 * the only driver objects it creates are the side streams and events of the
 * multi-pass plans, once per (host thread, device), on that thread's first
 * multi-pass call (see hyenand_fftconv).
 */
#ifndef HYENAND_H
#define HYENAND_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  HYENAND_OK = 0,
  HYENAND_ERR_INVALID_ARGUMENT = 1,  /* null pointer, bad enum, dims <= 0, y aliasing an input */
  HYENAND_ERR_UNSUPPORTED = 2,       /* a shape or size beyond the implemented plans */
  HYENAND_ERR_WORKSPACE_TOO_SMALL = 3,
  HYENAND_ERR_HIP = 4,               /* a HIP launch failed; see hyenand_last_error().  A call
                                        clears the calling thread's pending HIP error (one that
                                        earlier work left to be read by hipGetLastError) before
                                        it launches, so only its own launches are reported. */
  HYENAND_STATUS_MAX_ENUM = 0x7fffffff
} hyenand_status;

/* Each enum ends with a 0x7fffffff member so that it spans every int: the
 * library validates the values it receives, whatever int a caller passes. */
typedef enum {
  HYENAND_PAD_LINEAR = 0,
  HYENAND_PAD_CIRCULAR = 1,
  HYENAND_PAD_CENTERED = 2,
  HYENAND_PAD_MAX_ENUM = 0x7fffffff
} hyenand_pad_mode;

/* Storage type of x1, x2, v, k, D and y.  Compute is fp32 in both cases;
 * bf16 values are widened on load and rounded to nearest-even on store. */
typedef enum { HYENAND_DTYPE_F32 = 0, HYENAND_DTYPE_BF16 = 1, HYENAND_DTYPE_MAX_ENUM = 0x7fffffff } hyenand_dtype;

/*
 * hyenand_fftconv -- y = x2 * (k conv (x1*v) + D*(x1*v)) on the GPU.
 *
 * x1, x2, v, k, y : device pointers, contiguous row-major [B, C, L1, ..., LN]
 *                   of `dtype` (fp32, or bf16 bits), 16-byte aligned (fresh
 *                   allocations are); with pad_mode centered k is
 *                   [B, C, 2 L1 - 1, ..., 2 LN - 1].  y must not overlap any
 *                   input.
 * D               : device pointer, [C] of `dtype`.
 * ndim            : N in {1, 2, 3}.
 * dims            : host pointer to ndim + 2 int64 values {B, C, L1, ..., LN},
 *                   all >= 1, with B * C < 2^22 (one workgroup per (b, c)
 *                   line; a launch holds fewer than 2^32 work-items).
 *                   Transform extents: L_d circular, 2 L_d
 *                   linear and centered; supported up to 2^22 points in 1D
 *                   and 1024 per axis in 2D/3D.  Other extents (section
 *                   3.2.2: patch grids such as 14 x 14, register rows):
 *                   grids of up to 4096 transform points in one pass on
 *                   mixed-radix transforms (radix 2, 3, 4, 5, 7, 8), a
 *                   circular axis whose extent has no prime factor above 7
 *                   on its own L_d points, every other axis on the smallest
 *                   such P_d >= 2 L_d - 1; or on the smallest power of two
 *                   >= 2 L_d - 1, whichever is the faster for the shape (a
 *                   non-circular convolution is exact on any such P_d; a
 *                   circular axis of another extent repeats the kernel
 *                   periodically over the displacements -(L_d - 1) ..
 *                   L_d - 1, which makes it a non-circular one): in one pass
 *                   per line for 1D up to L = 8192 and 2D up to 128-point
 *                   transforms per axis; beyond that embedded in the
 *                   transform grid, where the call is the circular
 *                   convolution of the zero-padded inputs and of k placed at
 *                   its displacements: x1, x2, v and k are copied into the
 *                   workspace on that grid, the circular plan runs there and
 *                   y is copied back (the workspace queries include the five
 *                   embedded tensors; at most 2^31 elements per embedded
 *                   tensor).  The operator takes the single-pass shapes only.
 * pad_mode        : hyenand_pad_mode.
 * dtype           : hyenand_dtype.
 * workspace       : device scratch of workspace_bytes (16-byte aligned), owned
 *                   by the caller; may be NULL when
 *                   hyenand_fftconv_workspace_size() reports 0.
 *                   A workspace smaller than the reported size but at least
 *                   the minimum one is accepted (the work is then split into
 *                   more passes).
 * stream          : hipStream_t to enqueue on (NULL = default stream).
 *
 * Validation is synchronous and launches nothing on error.  On HYENAND_OK the
 * work has been enqueued on `stream` and the call returns without waiting;
 * every buffer must stay alive until the stream reaches that point.  Calls on
 * distinct streams from distinct host threads are safe; two in-flight calls
 * must not share a workspace.  Results are deterministic (no atomics) and do
 * not depend on the workspace size.
 *
 * The multi-pass plans (the ones with a nonzero workspace) fork onto two or
 * three side streams of the library that wait for `stream` and that `stream`
 * waits for before anything enqueued after the call; a graph captured on
 * `stream` therefore takes them in.  Each host thread has its own side
 * streams and fork/join events per device (default priority, created on the
 * thread's first multi-pass call there, kept until the process ends), so
 * calls from several threads run concurrently and a capture on one thread
 * never takes in another thread's work.
 */
hyenand_status hyenand_fftconv(const void* x1, const void* x2, const void* v, const void* k,
                               const void* D, void* y, int ndim, const int64_t* dims,
                               hyenand_pad_mode pad_mode, hyenand_dtype dtype, void* workspace, size_t workspace_bytes,
                               void* stream);

/*
 * hyenand_fftconv_shared_k -- as hyenand_fftconv, with one kernel per channel
 * shared by every sample: the Hyena operator's global kernel K of one row per
 * channel (Eq. (hyena), section "Background: Hyena and CKConv"), before
 * HyenaND makes the kernel input-dependent.  k is [C, L1, ..., LN] (centered:
 * [C, 2 L1 - 1, ...]) and sample b, channel c uses k[c].  Everything else is
 * as for hyenand_fftconv; its workspace sizes are enough.
 * Since the kernel does not depend on the sample, its spectrum is the same
 * for all B samples: on the single-pass 2D plan (power-of-two transform
 * grids, linear or circular, B >= 2) a workspace of at least
 * hyenand_fftconv_shared_k_workspace_size() bytes lets the call transform
 * each channel's kernel once (C x P0 x P1/2 complex fp32 spectra at the
 * start of the workspace) and every image read that spectrum, instead of
 * transforming it once per image.  With a smaller or NULL workspace it
 * does the latter.  The two give the same results up to rounding order.
 */
hyenand_status hyenand_fftconv_shared_k(const void* x1, const void* x2, const void* v, const void* k,
                                        const void* D, void* y, int ndim, const int64_t* dims,
                                        hyenand_pad_mode pad_mode, hyenand_dtype dtype, void* workspace, size_t workspace_bytes,
                                        void* stream);

/* Recommended workspace size (bytes) for hyenand_fftconv_shared_k: that of
 * hyenand_fftconv, or the per-channel spectra where the call can use them
 * (see above).  Pure host function. */
hyenand_status hyenand_fftconv_shared_k_workspace_size(int ndim, const int64_t* dims, hyenand_pad_mode pad_mode,
                                                       hyenand_dtype dtype, size_t* bytes_out);

/*
 * Kernel spectra kept across calls.  A static kernel (the Hyena operator's
 * global kernel K, one row per channel: Eq. (hyena), section "Background:
 * Hyena and CKConv"; at inference it does not change between calls) has the
 * same spectrum in every call, so it can be transformed once:
 *
 *   hyenand_kernel_spectrum_size(ndim, dims, ...)  bytes of the spectra
 *   hyenand_kernel_spectrum(k, khat, ...)          k [C, L1, L2] -> khat
 *   hyenand_fftconv_spectrum(x1, x2, v, khat, ...) y as hyenand_fftconv_shared_k
 *                                                  gives for that k
 *
 * dims, pad_mode, dtype: those of the convolution calls ([B, C, L1, L2];
 * only C, the grid and the mode fix the spectra, so one khat serves every B).
 * Runs on the single-pass 2D plan only: linear or circular mode with a
 * power-of-two transform grid of up to 128 x 128 (hyenand_fftconv_plan_name
 * "fused2d"); other shapes return HYENAND_ERR_UNSUPPORTED.
 * khat: device buffer of at least the reported size (C x P0 x P1/2 complex
 * fp32 values), 16-byte aligned, owned by the caller; its layout is private
 * to the library and valid only for calls with the same C, grid, pad mode
 * and library version.  k, x1, x2, v, y: 16-byte aligned, as for
 * hyenand_fftconv; D element-aligned.  hyenand_kernel_spectrum reads k and
 * writes khat (which must not overlap); hyenand_fftconv_spectrum reads khat
 * and must not write it through y.  Validation, stream and error
 * conventions as for hyenand_fftconv; the results are bitwise those of
 * hyenand_fftconv_shared_k with the same k.
 */
hyenand_status hyenand_kernel_spectrum_size(int ndim, const int64_t* dims, hyenand_pad_mode pad_mode,
                                            hyenand_dtype dtype, size_t* bytes_out);
hyenand_status hyenand_kernel_spectrum(const void* k, void* khat, size_t khat_bytes, int ndim, const int64_t* dims,
                                       hyenand_pad_mode pad_mode, hyenand_dtype dtype, void* stream);
hyenand_status hyenand_fftconv_spectrum(const void* x1, const void* x2, const void* v, const void* khat,
                                        size_t khat_bytes, const void* D, void* y, int ndim, const int64_t* dims,
                                        hyenand_pad_mode pad_mode, hyenand_dtype dtype, void* stream);

/*
 * hyenand_fftconv_noalloc -- hyenand_fftconv for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc.  Arguments, layouts, validation, stream
 * semantics and results are those of hyenand_fftconv, with no workspace
 * argument: the multi-pass plans use the library's own device scratch of
 * 128 MiB (128 << 20 bytes) per GPU instead, a static array reserved when the
 * library's code is loaded on that GPU and held until the process ends.
 * Shapes whose least workspace (hyenand_fftconv_workspace_min) exceeds it
 * return HYENAND_ERR_UNSUPPORTED before anything runs.  The call allocates
 * no memory; the first call on a device looks the array up there once.
 * Every call on one GPU shares that GPU's scratch: two calls whose work may
 * overlap in time on the same GPU (on different streams, or from different
 * host threads without ordering) race on it and give wrong results; order
 * them on one stream or use hyenand_fftconv with a workspace each.  The
 * scratch keeps the last call's contents, which no call reads before writing.
 */
hyenand_status hyenand_fftconv_noalloc(const void* x1, const void* x2, const void* v, const void* k,
                                       const void* D, void* y, int ndim, const int64_t* dims,
                                       hyenand_pad_mode pad_mode, hyenand_dtype dtype, void* stream);

/*
 * hyenand_fftconv_modal -- hyenand_fftconv_shared_k with the kernel of every
 * channel generated inside the transform kernels instead of read: the
 * implicit long filter of order M of the appendix "Filter Generation",
 *
 *     k[c, t] = Re sum_{m < M} R[c, m] lambda[c, m]^t,  t = 0 .. L - 1,
 *     lambda = exp(log_mag + i angle),  R = res_re + i res_im
 *
 * (the filter hyenand_modal_filter writes), evaluated where the FFT kernel
 * would load k -- the paper fuses kernel evaluation into its FFT kernel
 * (section 3.2.1, "Support for circular and non-circular convolutions";
 * section 4, "CUDA Implementation: nSubQ") -- so no k tensor exists.  Every
 * sample of channel c uses filter c.
 * log_mag, angle, res_re, res_im : device pointers, [C, M] fp32, 4-byte
 *   aligned; order = M in 1..32.
 * Other arguments, layouts, workspace (the sizes hyenand_fftconv_workspace_*
 * report for the same dims), stream and error conventions as for
 * hyenand_fftconv.  Runs on the four-step plan only: 1D lines with a
 * transform of 2^15 .. 2^22 points (linear: L = 2^14 .. 2^21; circular:
 * L = 2^15 .. 2^22), pad_mode linear or circular; other shapes return
 * HYENAND_ERR_UNSUPPORTED (hyenand_modal_filter and
 * hyenand_fftconv_shared_k cover them).  Each point of the filter is at most
 * N1 / T - 1 fp32 steps (7 for 2^20-point lines) from terms formed exactly
 * from a double phase, and stays in fp32 (it is not rounded to the storage
 * type).
 */
hyenand_status hyenand_fftconv_modal(const void* x1, const void* x2, const void* v, const float* log_mag,
                                     const float* angle, const float* res_re, const float* res_im, int order,
                                     const void* D, void* y, int ndim, const int64_t* dims,
                                     hyenand_pad_mode pad_mode, hyenand_dtype dtype, void* workspace,
                                     size_t workspace_bytes, void* stream);

/* Recommended workspace size (bytes) for a call with these arguments; 0 for
 * plans that keep everything on chip.  Pure host function. */
hyenand_status hyenand_fftconv_workspace_size(int ndim, const int64_t* dims, hyenand_pad_mode pad_mode,
                                              hyenand_dtype dtype, size_t* bytes_out);

/* Smallest workspace (bytes) hyenand_fftconv accepts for these arguments. */
hyenand_status hyenand_fftconv_workspace_min(int ndim, const int64_t* dims, hyenand_pad_mode pad_mode,
                                             hyenand_dtype dtype, size_t* bytes_out);

/* Name of the plan the call would use ("fused1d", "fused2d", "multipass2d",
 * "multipass3d", "fourstep1d"; for extents that are not powers of two
 * "mixed1d/2d/3d", "fused1d_any", "fused2d_any" or "embedded1d/2d/3d"), written
 * NUL-terminated into buf (at most n bytes).  Pure host function. */
hyenand_status hyenand_fftconv_plan_name(int ndim, const int64_t* dims, hyenand_pad_mode pad_mode, hyenand_dtype dtype,
                                         char* buf, size_t n);

/*
 * hyenand_fftconv_backward -- gradients of a scalar loss through
 * y = x2 * (k conv (x1*v) + D*(x1*v)), given gy = dLoss/dy.
 *
 * With u = x1*v, h = gy*x2 and z = k conv u + D*u (the pre-gate output):
 *
 *     gx2 = gy*z,    gu[j] = sum_n k[n-j] h[n] + D[c]*h[j]   (adjoint of the
 *                    convolution: linear n_d >= j_d, circular (n-j) mod L),
 *     gk[m] = sum_n h[n] u[n-m]  (linear n_d >= m_d, circular mod L),
 *     gx1 = gu*v,    gv = gu*x1,    gD[c] = sum over b and n of h*u.
 *
 * These are the derivatives of the operator of Eq. (HyenaND), section 3.2,
 * with the gates and shortcut of Def. A.2 / A.3 (the paper trains through
 * it).  Same layouts, dtype, pad_mode and stream semantics as
 * hyenand_fftconv; gy and the outputs gx1, gx2, gv, gk are [B, C, L...]
 * (16-byte aligned), gD is [C].  No output may overlap an input or another
 * output.  workspace: device scratch of at least
 * hyenand_fftconv_backward_workspace_min() bytes, 16-byte aligned, contents
 * overwritten: per-line sums of h*u for gD, then (for the multi-pass plans)
 * the three half spectra of u, k and h of a chunk of lines, as in the
 * forward; hyenand_fftconv_backward_workspace_size() is the recommended
 * size.  gD is reduced in a fixed order, so results are deterministic and do
 * not depend on the workspace size.  Supported: every shape the forward
 * supports (1D transforms up to 2^22 points, 2D/3D up to 1024 per axis);
 * other shapes return HYENAND_ERR_UNSUPPORTED.  The multi-pass plans use the
 * library's side streams as hyenand_fftconv does.
 *
 * Centred mode (k and gk [B, C, 2 L1 - 1, ...], gu[j] = sum_n k[n - j +
 * (L - 1)] h[n] + D h[j], gk[i] = sum_n h[n] u[n - i + (L - 1)]) and
 * extents that are not powers of two: both are circular convolutions on
 * their transform grid once u is zero-padded and k placed at its
 * displacements.  Extents that are not powers of two run in one pass on the
 * forward's mixed-radix grid where it fits (about 3000 transform points per
 * image; the workspace holds the gD sums only).  The other shapes, and the
 * centred mode on power-of-two extents, are embedded: the library copies x1,
 * x2, v, gy and k into the transform grid (a power of two >= 2 L_d - 1 per
 * axis), runs the circular backward there and extracts the gradients.  The
 * workspace then starts with the nine embedded tensors (each B * C * prod P
 * elements of dtype, 256-byte aligned); the workspace queries include them.
 * Extents that are not powers of two may also be 3D here.
 */
hyenand_status hyenand_fftconv_backward(const void* x1, const void* x2, const void* v, const void* k,
                                        const void* D, const void* gy, void* gx1, void* gx2, void* gv,
                                        void* gk, void* gD, int ndim, const int64_t* dims, hyenand_pad_mode pad_mode,
                                        hyenand_dtype dtype, void* workspace, size_t workspace_bytes, void* stream);

/* Recommended workspace bytes for hyenand_fftconv_backward with these
 * arguments. */
hyenand_status hyenand_fftconv_backward_workspace_size(int ndim, const int64_t* dims, hyenand_pad_mode pad_mode,
                                                       hyenand_dtype dtype, size_t* bytes_out);

/* Smallest workspace (bytes) hyenand_fftconv_backward accepts for these
 * arguments. */
hyenand_status hyenand_fftconv_backward_workspace_min(int ndim, const int64_t* dims, hyenand_pad_mode pad_mode,
                                                      hyenand_dtype dtype, size_t* bytes_out);

/*
 * hyenand_operator -- the whole HyenaND operator of Eq. (HyenaND), section
 * 3.2, around the same long convolution:
 *
 *     a   = l2(q) * SiLU(kin),  l2(q) = q / max(||q[b, :, p]||_2, eps_l2)
 *     u   = a / sqrt(mean_c a^2 + eps_rms) * w_in[c]            (RMSNorm)
 *     z   = Sigmoid(vin) * (k conv u + D[c] * u)                 (as y above)
 *     y   = z / sqrt(mean_c z^2 + eps_rms) * w_out[c]            (RMSNorm)
 *
 * with SiLU(x) = x / (1 + exp(-x)) and Sigmoid(x) = 1 / (1 + exp(-x)); the
 * norms and means run across the C channels of every sample b and grid point
 * p.  The paper writes the operator without the shortcut: pass D = 0.
 * q, kin, vin, y : [B, C, L...] of dtype (16-byte aligned); k as for
 * hyenand_fftconv (its shape follows pad_mode); D, w_in, w_out : [C] of dtype.
 * eps_l2, eps_rms: finite, >= 0.  C is at most 16384.  y must not overlap an
 * input.  workspace: at least the normalisation scales (B * prod L floats, in
 * a 256-byte block) plus hyenand_fftconv_workspace_min() bytes;
 * hyenand_operator_workspace_size() is the recommended size.  Three stages
 * on `stream`: a pass over q and kin for the per-point scale, the transform
 * kernels with the gates applied as they stage and store, and an in-place
 * RMSNorm of y (one read, one write).  Stream, determinism and error
 * conventions as for hyenand_fftconv.
 */
hyenand_status hyenand_operator(const void* q, const void* kin, const void* vin, const void* k, const void* D,
                                const void* w_in, const void* w_out, float eps_l2, float eps_rms, void* y,
                                int ndim, const int64_t* dims, hyenand_pad_mode pad_mode, hyenand_dtype dtype, void* workspace,
                                size_t workspace_bytes, void* stream);

/* Recommended workspace bytes for hyenand_operator. */
hyenand_status hyenand_operator_workspace_size(int ndim, const int64_t* dims, hyenand_pad_mode pad_mode, hyenand_dtype dtype,
                                               size_t* bytes_out);

/*
 * hyenand_kernel_synth -- the HyenaND kernel K(x) = w(r) * f_theta(r; z(x))
 * written on the kernel grid of a convolution, ready for hyenand_fftconv
 * (section 3.2.1 "Multi-Dimensional Continuous Convolutional Kernels",
 * Eq. (kernel); section 3.2.2 "Input-Dependent Kernels via Registers and
 * FiLM", Eq. (film); the appendix "HyenaND Design Details: Masking and
 * Initialization", Eq. (mask)).  For every sample b, channel c and grid point
 * with normalised coordinates r in [-1, 1]^N:
 *
 *     h_1 = sin(omega0 * (r W1) + bias_1)          then FiLM
 *     h_j = sin(h_{j-1} W_j + bias_j), j = 2..J    then FiLM
 *     FiLM: h_j <- gamma[b, j] * h_j + beta[b, j]  (after the sine)
 *     k[b, c, point] = w_c(r) * (h_J Wout)[c]
 *
 * Window: window_kind 0 is the Gaussian exp(-1/2 sum_d (r_d / sigma[d, c])^2)
 * with window = sigma [N, C] (every sigma > 0); window_kind 1 is the
 * exponential exp(-alpha[c] sum_d |r_d|) with window = alpha [C].
 *
 * The grid is the kernel layout that hyenand_fftconv takes for the same dims
 * and pad_mode: L_d points per axis (linear, circular) or 2 L_d - 1
 * (centered).  A point's displacement along axis d is its index i (linear),
 * i - (L_d - 1) (centered), or the signed periodic one, i for i <= L_d / 2
 * and i - L_d above (circular); r_d = displacement / (L_d - 1), and 0 when
 * L_d = 1.  The centered double grid thus spans [-1, 1] exactly.
 *
 * Parameters (device pointers, fp32, row-major; Wh, gamma and beta 16-byte
 * aligned, the others 4-byte aligned):
 *   omega0 [Hf], W1 [N, Hf], Wh [J - 1, Hf, Hf] (layer j + 1's matrix, rows =
 *   input units; NULL allowed when J = 1), bias [J, Hf] or NULL (no biases),
 *   gamma, beta [B, J, Hf] (the sample's FiLM scales and shifts) or both NULL
 *   (the unmodulated kernel), Wout [Hf, C].
 * hidden = Hf in {32, 64, 128}; layers = J in 1..16.
 * k (output, device, `dtype`, aligned to its element size): [B, C, grid...]
 *   with FiLM, [C, grid...] without (the kernel hyenand_fftconv_shared_k
 *   takes); must not overlap a parameter.
 * dims = {B, C, L1, ..., LN} of the convolution (host pointer), ndim = N.
 * The hidden layers and the output projection run as fp32 matrix-core
 * products; the sine and exponential use the hardware approximations after
 * an exact-to-fp32 argument reduction.  Validation, stream and error
 * conventions as for hyenand_fftconv; no workspace.
 */
hyenand_status hyenand_kernel_synth(const float* omega0, const float* W1, const float* Wh, const float* bias,
                                    const float* gamma, const float* beta, const float* Wout, const float* window,
                                    int window_kind, int hidden, int layers, void* k, int ndim,
                                    const int64_t* dims, hyenand_pad_mode pad_mode, hyenand_dtype dtype, void* stream);

/*
 * hyenand_modal_filter -- the implicit long filter of order M of the appendix
 * "Filter Generation", written as the [C, L] kernel that
 * hyenand_fftconv_shared_k takes (one filter per channel):
 *
 *     k[c, t] = Re sum_{m < M} R[c, m] lambda[c, m]^t,   t = 0 .. L - 1,
 *     lambda = exp(log_mag + i angle),  R = res_re + i res_im,
 *
 * i.e. sum_m exp(t log_mag) (res_re cos(t angle) - res_im sin(t angle)).
 * The M complex terms per point are never stored.  log_mag <= 0 keeps every
 * term bounded; a positive one grows and may overflow as the formula does.
 * log_mag, angle, res_re, res_im : device pointers, [C, M] fp32, 4-byte
 *   aligned; order = M in 1..256.
 * k (output, device, `dtype`, aligned to its element size) : [C, L]; must not
 *   overlap a parameter.  C in 1..65535, L in 1..2^29.
 * Accuracy: up to order 32 the sum runs as fp32 matrix-core products over
 * tiles of 1024 points, each term formed from an exact (double) phase and
 * magnitude at most 31 fp32 advances of lambda^1024 back; above order 32 each
 * point's terms are at most 31 fp32 steps of lambda^64 from such a phase.
 * Errors stay at a few fp32 roundings per mode.  Validation, stream and error
 * conventions as for hyenand_fftconv; no workspace.
 */
hyenand_status hyenand_modal_filter(const float* log_mag, const float* angle, const float* res_re,
                                    const float* res_im, int order, void* k, int64_t C, int64_t L, hyenand_dtype dtype,
                                    void* stream);

/* Static text for a status code. */
const char* hyenand_status_string(hyenand_status status);

/* Detail of the last non-OK return on the calling host thread ("" if none). */
const char* hyenand_last_error(void);

/* Library version, major*10000 + minor*100 + patch. */
int hyenand_version(void);

#ifdef __cplusplus
}
#endif

#endif /* HYENAND_H */
