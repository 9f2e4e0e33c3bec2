/*
 * fdc.h -- C ABI of libfdc, the gfx950 (MI355X) implementation of the
 * Frequency Domain Convolution (FDC) and Frequency Domain Pooling (FDP) layers
 * of Goh, Chen and Lim, "Frequency Domain Convolutional Neural Network:
 * Accelerated CNN for Large Diabetic Retinopathy Image Classification"
 * (arXiv 2106.12736), forward and backward.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Memory.    Every tensor argument is a DEVICE pointer owned by the caller
 *            (the library never frees or keeps it).  Tensors are dense,
 *            contiguous and row-major.  Real tensors are float32; spectra
 *            are complex64 stored as interleaved {float re, im} pairs
 *            (fdc_c64), the layout of torch.complex64.
 * Spectra.   A real H x W image has the half spectrum [H][W/2+1] of the
 *            real-to-complex DFT (section 2.4.1.1):
 *              X[k][l] = sum_{h<H, w<W} x[h][w] exp(-2 pi i (hk/H + wl/W)),
 *            k < H, l <= W/2, unnormalised, rows in natural (unshifted)
 *            order.  The inverse is scaled by 1/(H W) and takes the real
 *            part: for ANY complex half spectrum Y,
 *              irfft2(Y)[h][w] = 1/(HW) sum_{k, l<=W/2} c_l Re(Y[k][l] exp(+2 pi i (hk/H + wl/W)))
 *            with c_0 = c_{W/2} = 1 and c_l = 2 otherwise.
 * Gradients. For a real loss L, the gradient of a complex tensor Z is
 *            dL/dRe(Z) + i dL/dIm(Z).  Gradient outputs are overwritten,
 *            never accumulated.  A NULL gradient output skips that output.
 * Streams.   Every compute call validates its arguments on the host and then
 *            enqueues kernels asynchronously on `stream` (NULL = the null
 *            stream) and returns.  When a call returns an error nothing has
 *            been enqueued.  Device faults surface at the caller's next
 *            synchronisation.  Calls allocate no device memory; workspaces
 *            are supplied by the caller and must not be shared by calls that
 *            may run concurrently.
 * Sizes.     Transform lengths must be in the supported set: a power of two
 *            from 2 to 1024, or 224 (= 7 * 32, the 224 x 224 image size of the
 *            Full FDC workloads).  Other lengths return FDC_EUNSUPPORTED.
 *            The kernels index the rows of a batch with 32-bit integers: a
 *            plan whose images times rows (or times stored bins) reach 2^31
 *            is refused with FDC_EUNSUPPORTED when it is created, so a call
 *            on a valid plan never fails part-way through its launches.
 * Plans.     Plan handles are checked against the library's registry of live
 *            plans before they are read: a destroyed or never-created handle,
 *            or a plan of another kind, returns FDC_EINVAL.  Destroying NULL is
 *            a no-op; destroying a handle twice returns FDC_EINVAL.  (A new
 *            plan may be created at the address of a destroyed one, after
 *            which the old handle names the new plan.)  Plans are immutable
 *            after creation and may be used from several host threads.
 * Errors.    Calls return an fdc_status.  fdc_last_error() gives a
 *            thread-local text for the last non-OK status of this thread.
 *            No C++ exception crosses this interface.
 */
#ifndef FDC_H
#define FDC_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct { float re, im; } fdc_c64;

typedef enum {
  FDC_OK = 0,
  FDC_EINVAL = 1,          /* bad argument: NULL pointer, size <= 0, odd size, S mod C != 0, M > N ... */
  FDC_EUNSUPPORTED = 2,    /* valid but not implemented: transform length outside the supported set,
                              sizes beyond the kernels' 32-bit indexing */
  FDC_EWORKSPACE = 3,      /* workspace pointer NULL or smaller than the queried size */
  FDC_EHIP = 4             /* a HIP runtime call or kernel launch failed (text in fdc_last_error) */
} fdc_status;

/* Convolution artifact handling (section 2.4.1.3).  A frequency-domain product is a
 * circular convolution, whose wrap-around pollutes the top n-1 rows and left n-1
 * columns for an n x n kernel.
 *   NONE: keep the circular result (M x M).
 *   CROP: cut n-1 rows at the top and n-1 columns at the left -> (M-n+1) x (M-n+1),
 *         the size of a spatial convolution without padding.
 *   ROLL: keep M x M but shift by s = (n-1)/2 (integer division) so the artifact is
 *         spread over all edges: out[i][j] = y[(i+s) mod M][(j+s) mod M]. */
typedef enum { FDC_ARTIFACT_NONE = 0, FDC_ARTIFACT_CROP = 1, FDC_ARTIFACT_ROLL = 2 } fdc_artifact;

const char *fdc_status_string(int status);
const char *fdc_last_error(void);
/* Library version as 10000*major + 100*minor + patch. */
int fdc_version(void);

/* ------------------------------------------------------------------------ */
/* 2-D real FFT plans (section 2.4.1.1: RFFT of real images, width N/2+1)    */
/* ------------------------------------------------------------------------ */
typedef struct fdc_fft_plan fdc_fft_plan;

/* A plan for `count` independent h x w real images (h, w in the supported set).
 * The plan is an immutable host object (no device memory); it may be used
 * concurrently on several streams.  Returns FDC_EINVAL for count < 1 or NULL. */
fdc_status fdc_fft_plan_create(fdc_fft_plan **plan, int64_t count, int h, int w);
fdc_status fdc_fft_plan_destroy(fdc_fft_plan *plan);
/* Bytes of workspace the four transforms below need (0 for fdc_rfft2 and
 * fdc_irfft2_backward, which work in their output buffer). */
fdc_status fdc_fft_workspace_size(const fdc_fft_plan *plan, size_t *bytes);

/* x [count][h][w] float32 -> X [count][h][w/2+1] complex, forward, unnormalised. */
fdc_status fdc_rfft2(const fdc_fft_plan *plan, const float *x, fdc_c64 *X,
                     void *ws, size_t ws_bytes, hipStream_t stream);
/* X [count][h][w/2+1] -> x [count][h][w]: the inverse defined above (1/(hw), real part
 * of columns 0 and w/2 after the column inverse, for any complex X). */
fdc_status fdc_irfft2(const fdc_fft_plan *plan, const fdc_c64 *X, float *x,
                      void *ws, size_t ws_bytes, hipStream_t stream);
/* Adjoint of fdc_rfft2: gx[h][w] = sum_{k, l<=w/2} Re(gX[k][l] exp(+2 pi i (hk/H + wl/W))). */
fdc_status fdc_rfft2_backward(const fdc_fft_plan *plan, const fdc_c64 *gX, float *gx,
                              void *ws, size_t ws_bytes, hipStream_t stream);
/* Adjoint of fdc_irfft2: gX[k][l] = (c_l / (h w)) * rfft2(gx)[k][l]. */
fdc_status fdc_irfft2_backward(const fdc_fft_plan *plan, const float *gx, fdc_c64 *gX,
                               void *ws, size_t ws_bytes, hipStream_t stream);
/* fdc_rfft2 restricted to the bins that Frequency Domain Pooling to mh x mw keeps
 * (section 2.4.2): X[i][k][l] for l <= mw/2 and k < mh/2 or k >= h - mh/2, each with
 * the value fdc_rfft2 gives it.  The other bins of X are undefined on return (left as
 * they were or written).  mh and mw even, 2 <= mh <= h, 2 <= mw <= w (FDC_EINVAL
 * otherwise); mh = h, mw = w is fdc_rfft2.  The first FDC + FDP layer of an FDCNN
 * (section 2.5.1) reads only these bins of its input spectrum (fdc_cic_fdp_forward and
 * fdc_cic_fdp_backward with N = h = w, M = mh = mw), so its input transform needs no
 * others: the row pass forms mw/2 + 1 bins of every row, the column pass transforms
 * those columns and stores the mh kept rows.  No workspace. */
fdc_status fdc_rfft2_pooled(const fdc_fft_plan *plan, const float *x, fdc_c64 *X, int mh,
                            int mw, hipStream_t stream);
/* The same bins, with a workspace of count * h * (mw/2 + 1) complex values (at least
 * that many bytes times 8; unused for planes of 16^2 to 64^2): the row pass writes the
 * mw/2 + 1 bins in runs of 8 per row into the workspace, so that the column pass reads
 * whole runs instead of one value per row of X.  Same results bit for bit as
 * fdc_rfft2_pooled.  FDC_EWORKSPACE when ws is NULL or smaller. */
fdc_status fdc_rfft2_pooled_ws(const fdc_fft_plan *plan, const float *x, fdc_c64 *X, int mh,
                               int mw, void *ws, size_t ws_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* Channel Independent Convolution on spectra (Eq. 5, Algorithm 1)          */
/* ------------------------------------------------------------------------ */
/* Y[b][o] = X[b][o / J] o K[o] for o = c*J + j < S, J = S / C (S mod C must be 0),
 * elementwise over the [H][Wf] bins.  X [B][C][H][Wf], K [S][H][Wf], Y [B][S][H][Wf]. */
fdc_status fdc_cic_forward(const fdc_c64 *X, const fdc_c64 *K, fdc_c64 *Y,
                           int B, int C, int S, int H, int Wf, hipStream_t stream);
/* gX[b][c] = sum_j gY[b][cJ+j] conj(K[cJ+j]);  gK[o] = sum_b gY[b][o] conj(X[b][o/J]).
 * The sum over b is done in a fixed order (bitwise reproducible). */
fdc_status fdc_cic_backward(const fdc_c64 *gY, const fdc_c64 *X, const fdc_c64 *K,
                            fdc_c64 *gX, fdc_c64 *gK,
                            int B, int C, int S, int H, int Wf, hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* Frequency Domain Pooling (section 2.4.2)                                 */
/* ------------------------------------------------------------------------ */
/* One FDC layer of the FDCNN on spectra (section 2.5.1: the network transforms once,
 * before its first layer, and inverts once after its last): CIC (Eq. 5) followed by
 * FDP to M x M, forming only the bins FDP keeps.  X [B][C][N][N/2+1], K [S][N][N/2+1]
 * -> Y [B][S][M][M/2+1]; S mod C == 0, N and M even, M <= N.  Y must be 16-byte
 * aligned (torch allocations are): each thread stores two bins at once. */
fdc_status fdc_cic_fdp_forward(const fdc_c64 *X, const fdc_c64 *K, fdc_c64 *Y, int B, int C, int S, int N, int M,
                               hipStream_t stream);
/* gY [B][S][M][M/2+1] -> gX [B][C][N][N/2+1] (NULL: skipped) and gK [S][N][N/2+1]
 * (NULL: skipped; summed over the batch in order), both with exact zeros at the bins
 * FDP drops.  gX must be 16-byte aligned. */
fdc_status fdc_cic_fdp_backward(const fdc_c64 *gY, const fdc_c64 *X, const fdc_c64 *K, fdc_c64 *gX, fdc_c64 *gK,
                                int B, int C, int S, int N, int M, hipStream_t stream);

/* Pi_H in place: Y [count][H][W/2+1] -> rfft2(irfft2(Y)) (section 2.4.1.1, the inverse
 * with real-part semantics).  Columns 0 and W/2 become (Y[k][l] + conj(Y[-k mod H][l]))/2;
 * every other bin is unchanged.  H, W even.  The map is a real-linear orthogonal
 * projection, so it is also its own adjoint (apply it to a gradient to back-propagate).
 * Between two layers of a CIC + FDP stack (artifact NONE) the irfft2 of one layer and
 * the rfft2 of the next reduce to this projection: the FDCNN chain of
 * fdc_cic_fdp_forward with Pi_H after every layer but the last computes the stack. */
fdc_status fdc_hermitian_project(fdc_c64 *Y, int64_t count, int H, int W, hipStream_t stream);
/* The chain of the previous two entries in one call each: fdc_cic_fdp_forward with Y
 * written as Pi_H(Y), and fdc_cic_fdp_backward with gX written as Pi_H(gX) (gK as
 * fdc_cic_fdp_backward writes it).  The results equal the separate calls followed by
 * fdc_hermitian_project (same arithmetic, bit for bit).  Between two layers of a
 * CIC + FDP stack (artifact NONE) the forward of every layer but the last and the
 * backward of every layer but the first take these forms. */
fdc_status fdc_cic_fdp_forward_projected(const fdc_c64 *X, const fdc_c64 *K, fdc_c64 *Y, int B, int C, int S,
                                         int N, int M, hipStream_t stream);
fdc_status fdc_cic_fdp_backward_projected(const fdc_c64 *gY, const fdc_c64 *X, const fdc_c64 *K, fdc_c64 *gX,
                                          fdc_c64 *gK, int B, int C, int S, int N, int M, hipStream_t stream);
/* fdc_cic_fdp_backward and fdc_cic_fdp_backward_projected writing only the bins the
 * FDP keeps (rows k < M/2 and k >= N - M/2, columns l <= M/2) of gX and gK, and, in the
 * projected form, columns 0 and N/2 of gX over every row (Pi_H gives dropped row M/2 half
 * of row N - M/2).  The other bins are not written: a caller whose gX and gK hold zeros
 * there (allocated zeroed and written only by these calls) gets the results of the full
 * calls, bit for bit, without their stores of zeros (three quarters of gX and gK when
 * M = N/2).  Arguments and errors as fdc_cic_fdp_backward. */
fdc_status fdc_cic_fdp_backward_kept(const fdc_c64 *gY, const fdc_c64 *X, const fdc_c64 *K, fdc_c64 *gX,
                                     fdc_c64 *gK, int B, int C, int S, int N, int M, hipStream_t stream);
fdc_status fdc_cic_fdp_backward_projected_kept(const fdc_c64 *gY, const fdc_c64 *X, const fdc_c64 *K,
                                               fdc_c64 *gX, fdc_c64 *gK, int B, int C, int S, int N, int M,
                                               hipStream_t stream);

/* FDP crops the RFFT-shifted half spectrum: (H-Mh)/2 rows off the top and the
 * bottom, (W-Mw)/2 columns off the right, then shifts back.  In unshifted
 * order it keeps rows [0, Mh/2) and [H-Mh/2, H) and columns [0, Mw/2]; no
 * rescaling.  X [count][H][W/2+1] -> Y [count][Mh][Mw/2+1].  H, W, Mh, Mw even,
 * Mh <= H, Mw <= W (any reduction, not only halving). */
fdc_status fdp_forward(const fdc_c64 *X, fdc_c64 *Y, int64_t count,
                       int H, int W, int Mh, int Mw, hipStream_t stream);
/* Adjoint: gX = gY scattered back to the kept positions, zeros elsewhere. */
fdc_status fdp_backward(const fdc_c64 *gY, fdc_c64 *gX, int64_t count,
                        int H, int W, int Mh, int Mw, hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* Fused CIC + FDP layer on spatial activations                             */
/*   x -> rfft2 -> CIC (Eq. 5) -> FDP -> irfft2 -> artifact handling -> y     */
/* (Algorithm 1 inside Algorithm 2's spatial wrapper, with FDP of section    */
/*  2.4.2 applied before the inverse; per-layer transforms)                 */
/* ------------------------------------------------------------------------ */
typedef struct fdc_layer_plan fdc_layer_plan;

/* B images of C channels, N x N (N in the supported set) -> S = J*C channels of
 * M x M (M even, M <= N, N/M a power of two), kernels K [S][N][N/2+1] complex
 * (full-size spectra).  `artifact` with `kernel_n` (the spatial support the
 * kernels stand for, 1 <= kernel_n <= M) sets the output size:
 * NONE/ROLL -> M x M, CROP -> (M-kernel_n+1)^2.  Plans are immutable host objects. */
fdc_status fdc_cic_layer_plan_create(fdc_layer_plan **plan, int B, int C, int S, int N, int M,
                                     int artifact, int kernel_n);
/* Full FDC layer (Algorithm 2 with the per-bin sum over input channels of Eq. 2):
 * x [B][Cin][P][P], weights w [Cout][Cin][n][n] spatial (padded to P x P at the
 * top-left and transformed on every call, section 2.4.1.2), y [B][Cout][O][O] with
 * O = P - n + 1 for CROP and P for NONE/ROLL.  P a multiple of 8 in the supported
 * FFT set, 1 <= n <= 5 (FDC_EUNSUPPORTED otherwise).  No FDP: the layer keeps its
 * spatial size.  The plan owns a P-entry device table of twiddle factors, so it
 * is created on (and must be used with) the device current at creation;
 * FDC_EHIP if that allocation fails. */
fdc_status fdc_full_layer_plan_create(fdc_layer_plan **plan, int B, int Cin, int Cout, int P,
                                      int kernel_n, int artifact);
fdc_status fdc_layer_plan_destroy(fdc_layer_plan *plan);
/* Workspace sizes in bytes: forward scratch, the `saved` buffer forward writes
 * and backward reads, and backward scratch. */
fdc_status fdc_layer_workspace_size(const fdc_layer_plan *plan, size_t *fwd_ws, size_t *saved,
                                    size_t *bwd_ws);
/* Output spatial size (rows = cols) of the layer. */
fdc_status fdc_layer_output_size(const fdc_layer_plan *plan, int *out_size);

/* x [B][C][N][N] float32, K [S][N][N/2+1] complex -> y [B][S][O][O] float32.
 * `saved` (may be NULL when no backward will follow; fdc_layer_workspace_size
 * gives its size) receives the pooled input spectrum the backward pass needs:
 * the M x (M/2+1) bins FDP keeps, complex: columns 0..M/2-1 in a block
 * [B][C][M/16][M][8] of 8-column tiles stored down the rows when M/2 is a multiple
 * of 8 (else a block [B][C][M][M/2]), followed by column M/2 in a block [B][C][M]. */
fdc_status fdc_cic_layer_forward(const fdc_layer_plan *plan, const float *x, const fdc_c64 *K,
                                 float *y, void *saved, void *ws, size_t ws_bytes,
                                 hipStream_t stream);
/* gy [B][S][O][O] -> gx [B][C][N][N] (NULL: skipped) and gK [S][N][N/2+1] (NULL: skipped).
 * gK is summed over the batch in a fixed order and holds exact zeros at the bins
 * FDP drops (they do not reach the output). */
fdc_status fdc_cic_layer_backward(const fdc_layer_plan *plan, const float *gy, const void *saved,
                                  const fdc_c64 *K, float *gx, fdc_c64 *gK,
                                  void *ws, size_t ws_bytes, hipStream_t stream);

/* Strides, in complex elements, of a Full FDC spectrum (the `saved` buffer below).
 * Columns 0..P/2-1 form the main block: row k of every plane side by side, each
 * FDC_FULL_ROW(P) elements (P/2 bins and 16 unused).  Column P/2 forms the side
 * block: FDC_FULL_SIDE_PLANE(P) elements per plane (P bins and 8 unused). */
#define FDC_FULL_ROW(P) ((int64_t)(P) / 2 + 16)
#define FDC_FULL_SIDE_PLANE(P) ((int64_t)(P) + 8)

/* The CIC + FDP layer with spatial kernels (section 2.4.1.2, Algorithm 1): w [S][n][n]
 * fp32, n = the plan's kernel_n (1..8), placed at the top-left of the N x N grid and
 * transformed on every call at the bins FDP keeps; otherwise fdc_cic_layer_forward /
 * backward, with the plan's artifact mode.  The backward gives gw [S][n][n] (NULL:
 * skipped; summed over the batch and bins in a fixed order) and gx (NULL: skipped).
 * Workspaces: fdc_cic_spatial_workspace_size (they hold the kernel spectra and dK). */
fdc_status fdc_cic_spatial_workspace_size(const fdc_layer_plan *plan, size_t *fwd_ws, size_t *bwd_ws);
fdc_status fdc_cic_spatial_layer_forward(const fdc_layer_plan *plan, const float *x, const float *w, float *y,
                                         void *saved, void *ws, size_t ws_bytes, hipStream_t stream);
fdc_status fdc_cic_spatial_layer_backward(const fdc_layer_plan *plan, const float *gy, const void *saved,
                                          const float *w, float *gx, float *gw, void *ws, size_t ws_bytes,
                                          hipStream_t stream);

/* Full FDC forward: y = artifact(irfft2(sum_c rfft2(x[b][c]) o K[s][c])) with
 * K[s][c] = rfft2(pad(w[s][c])).  K is generated per bin inside the contraction
 * and never stored.  `saved` (may be NULL) receives rfft2(x), complex: with
 * planes i = b * Cin + c (n = B * Cin of them), bin (k, l < P/2) of plane i at element
 * (k * n + i) * FDC_FULL_ROW(P) + l and bin (k, P/2) at element
 * P * n * FDC_FULL_ROW(P) + i * FDC_FULL_SIDE_PLANE(P) + k.  The backward pass
 * reads it for dL/dw. */
fdc_status fdc_full_forward(const fdc_layer_plan *plan, const float *x, const float *w, float *y,
                            void *saved, void *ws, size_t ws_bytes, hipStream_t stream);
/* Full FDC backward: gy [B][Cout][O][O] -> gx [B][Cin][P][P] (NULL: skipped) and
 * gw [Cout][Cin][n][n] (NULL: skipped; needs `saved`).  w is needed only for gx.
 * gw is summed over bins in fixed-size chunks and then over chunks in order, so
 * repeated calls give identical results. */
fdc_status fdc_full_backward(const fdc_layer_plan *plan, const float *gy, const void *saved,
                             const float *w, float *gx, float *gw, void *ws, size_t ws_bytes,
                             hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* Stack of CIC + FDP layers executed as one unit                            */
/* ------------------------------------------------------------------------ */
/* Layer i (0 <= i < layers) is the layer of fdc_cic_layer_plan_create with B
 * images, C = channels[i], S = channels[i+1], N = sizes[i], M = sizes[i+1] and
 * artifact NONE (sizes and channels: host arrays of layers + 1 entries, copied).
 * The stack runs the same transforms as the layer calls in sequence (results agree
 * to fp32 rounding), but the activations and activation gradients between layers
 * are not written to memory: the inverse row transform of one layer and the
 * forward row transform of the next run in one kernel on the same rows.  When the
 * last two layers take inputs of at most 128 x 128 (the instantiated shape is
 * 128 -> 64 -> 32 with two output channels per input channel in both), one
 * workgroup per input plane of the first of them runs every step of both layers
 * with all intermediates in LDS (one forward launch; one backward launch plus the
 * in-order sum of the per-image dK products); fdc_cic_stack_tail reports it.
 * FDC_STACK_TAIL=0 in the environment when the plan is created keeps every layer
 * on the per-layer kernels (for comparisons).  Plans are immutable host objects. */
typedef struct fdc_stack_plan fdc_stack_plan;
fdc_status fdc_cic_stack_plan_create(fdc_stack_plan **plan, int B, int layers, const int *sizes,
                                     const int *channels);
fdc_status fdc_cic_stack_plan_destroy(fdc_stack_plan *plan);
/* Workspace bytes of one forward and one backward call. */
fdc_status fdc_cic_stack_workspace_size(const fdc_stack_plan *plan, size_t *fwd_ws, size_t *bwd_ws);
/* Bytes of layer `layer`'s saved buffer (as fdc_layer_workspace_size gives for that layer). */
fdc_status fdc_cic_stack_saved_size(const fdc_stack_plan *plan, int layer, size_t *bytes);
/* x [B][C_0][N_0][N_0] -> y [B][C_L][N_L][N_L] (L = layers).  K and saved are host
 * arrays of `layers` device pointers: K[i] layer i's kernels [S][N][N/2+1]; saved[i]
 * receives layer i's pooled input spectrum (layout of fdc_cic_layer_forward).
 * `saved` may be NULL when no backward follows. */
fdc_status fdc_cic_stack_forward(const fdc_stack_plan *plan, const float *x, const fdc_c64 *const *K, float *y,
                                 void *const *saved, void *ws, size_t ws_bytes, hipStream_t stream);
/* gy [B][C_L][N_L][N_L] -> gK[i] (host array of `layers` device pointers, each
 * overwritten as fdc_cic_layer_backward writes it) and gx [B][C_0][N_0][N_0]
 * (NULL: skipped). */
fdc_status fdc_cic_stack_backward(const fdc_stack_plan *plan, const float *gy, const void *const *saved,
                                  const fdc_c64 *const *K, float *gx, fdc_c64 *const *gK, void *ws,
                                  size_t ws_bytes, hipStream_t stream);
/* The same backward writing only the kept bins of every gK[i] (rows [0, M/2) and
 * [N-M/2, N), columns [0, M/2] of each plane, N = sizes[i], M = sizes[i+1]): the
 * dropped bins, where the gradient is exactly zero because FDP discards them
 * (section 2.4.2), are neither read nor written.  For callers that keep gK buffers
 * across steps with zeros at those bins (zeroed once at allocation): the result then
 * equals fdc_cic_stack_backward's bit for bit, without its stores of zeros (three
 * quarters of every gK when M = N/2).  Arguments, workspace and errors as
 * fdc_cic_stack_backward. */
fdc_status fdc_cic_stack_backward_kept(const fdc_stack_plan *plan, const float *gy, const void *const *saved,
                                       const fdc_c64 *const *K, float *gx, fdc_c64 *const *gK, void *ws,
                                       size_t ws_bytes, hipStream_t stream);

/* The same stack with n x n spatial kernels (section 2.4.1.2) and ROLL artifact
 * handling in every layer: the result of fdc_cic_spatial_layer_forward / backward
 * with artifact ROLL and kernel_n = n, layer after layer (to fp32 rounding).  w is a
 * host array of `layers` device pointers, w[i] [S_i][n][n] fp32 (S_i = channels[i+1]);
 * n in [1, 8] and n <= every layer's output size.  Each call forms every layer's
 * kernel spectra at the kept bins in one launch, with the ROLL shift s = (n-1)/2 of
 * the layer's M x M output folded in as the phase exp(+2 pi i s (k + l) / M) of output
 * bin (k, l), then runs the stack executor on them (saved buffers as
 * fdc_cic_stack_forward).  The backward gives gw[i] [S_i][n][n] (host array of device
 * pointers, all required; each summed over the batch and bins in a fixed order) and
 * gx (NULL: skipped); dK of every layer goes through the workspace and is projected
 * onto the taps in one launch.  Workspaces: fdc_cic_spatial_stack_workspace_size. */
fdc_status fdc_cic_spatial_stack_workspace_size(const fdc_stack_plan *plan, int kernel_n, size_t *fwd_ws,
                                                size_t *bwd_ws);
fdc_status fdc_cic_spatial_stack_forward(const fdc_stack_plan *plan, int kernel_n, const float *x,
                                         const float *const *w, float *y, void *const *saved, void *ws,
                                         size_t ws_bytes, hipStream_t stream);
fdc_status fdc_cic_spatial_stack_backward(const fdc_stack_plan *plan, int kernel_n, const float *gy,
                                          const void *const *saved, const float *const *w, float *gx,
                                          float *const *gw, void *ws, size_t ws_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* FDCNN classifier head and optimiser                                      */
/* ------------------------------------------------------------------------ */
/* The FDCNN of section 2.5.1 (Fig. 3) applies a ReLU to the spatial output of its final
 * inverse transform and feeds it to fully connected layers; section 3.1 trains it with
 * the cross-entropy loss and Adam with weight decay.  The head here is ReLU, one fully
 * connected layer to `classes` outputs (1..16) and the softmax cross-entropy averaged
 * over the batch.
 *   y [B][F] fp32 (the chain output, F = C * M * M), W [classes][F], bias [classes],
 *   labels [B] int32 in [0, classes) (device memory), logits [B][classes], loss [1].
 * Every sum runs in a fixed order.  B * classes <= 15872.  An out-of-range label is
 * not detected on the host: it gives a NaN loss and NaN gradients. */
fdc_status fdc_head_workspace_size(int B, int64_t F, int classes, size_t *bytes);
/* logits = relu(y) W^T + bias; loss = mean_b (logsumexp(logits[b]) - logits[b][labels[b]]).
 * ws: fdc_head_workspace_size bytes of scratch (partial logits). */
fdc_status fdc_head_forward(const float *y, const float *W, const float *bias, const int32_t *labels, float *logits,
                            float *loss, int B, int64_t F, int classes, void *ws, size_t ws_bytes,
                            hipStream_t stream);
/* fdc_head_forward without a workspace argument, for callers that cannot allocate
 * device memory (code under HIP graph capture, serving loops, harnesses that forbid
 * allocation).  It allocates nothing: the partial logits go to a static device array
 * of 2^18 floats (1 MiB) that the library holds on each device it runs on until the
 * process ends.  Same kernels and results as fdc_head_forward.
 * Limit: ceil(F / 1024) * B * classes <= 262144, else FDC_EUNSUPPORTED (nothing
 * enqueued).  The array is looked up on the first call on each device (the current
 * device; `stream` must belong to it).  Every call on a device shares that device's
 * array, so calls that may overlap on one device (different streams, host threads)
 * race and must be ordered by the caller; the array keeps the last call's partial
 * logits, and no part of it needs to start at zero. */
fdc_status fdc_head_forward_noalloc(const float *y, const float *W, const float *bias, const int32_t *labels,
                                    float *logits, float *loss, int B, int64_t F, int classes, hipStream_t stream);
/* From the forward's logits: dlogits = (softmax(logits) - onehot(labels)) / B;
 * gW = dlogits^T relu(y), gbias = sum_b dlogits, gy = [y > 0] (dlogits W) (gy NULL:
 * skipped).  All outputs are overwritten. */
fdc_status fdc_head_backward(const float *y, const float *W, const float *logits, const int32_t *labels, float *gy,
                             float *gW, float *gbias, int B, int64_t F, int classes, hipStream_t stream);
/* One Adam step (Kingma and Ba, with weight decay added to the gradient as PyTorch's
 * Adam does) over n floats, in place on p, m and v (m, v start at zero).  A complex
 * parameter is updated as its (re, im) float pairs.  step_count is a device int32
 * holding the steps taken so far (start it at 0); the call updates with t = count + 1
 * and then stores t, so a captured graph advances on every replay.
 *   g' = g + wd p;  m = b1 m + (1 - b1) g';  v = b2 v + (1 - b2) g'^2;
 *   p -= lr / (1 - b1^t) * m / (sqrt(v) / sqrt(1 - b2^t) + eps). */
fdc_status fdc_adam_step(float *p, const float *g, float *m, float *v, int64_t n, int32_t *step_count, float lr,
                         float beta1, float beta2, float eps, float weight_decay, hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* Kernel timing (measurement support, off by default)                      */
/* ------------------------------------------------------------------------ */
/* While enabled, every kernel the library launches (only those named
 * `only_kernel` when it is not NULL) is bracketed by a pair of HIP events on
 * its stream; fdc_kernel_timing_report() synchronises on those events and
 * writes one line per kernel name: "<name> <launches> <total_ms>\n".
 * Enabling clears earlier records.  At most `max_launches` launches are
 * recorded; events are created when timing is enabled, never during a call.
 * Timing is process-wide and not meant for use under stream capture. */
fdc_status fdc_kernel_timing_enable(int max_launches, const char *only_kernel);
fdc_status fdc_kernel_timing_disable(void);
fdc_status fdc_kernel_timing_report(char *buf, size_t buf_bytes);
/* The same records one line per launch, in launch order: "<name> <ms>\n".
 * FDC_EINVAL when the text (with its terminating NUL) exceeds buf_bytes. */
fdc_status fdc_kernel_timing_launches(char *buf, size_t buf_bytes);

/* How a backward call forms dK (measurement support: which kernels it launches).
 * *ranges = 1: one dK launch ("col_bwd_gk_<M>") writes all of gK.  *ranges = R > 1:
 * the dK launch sums each of R contiguous image ranges into scratch inside the
 * backward workspace (R [S][M][M/2+1] arrays), and a second launch ("gk_reduce")
 * adds the ranges in range order and writes gK, so results stay repeatable.  R
 * depends only on the plan: larger batches are cut into ranges so that enough
 * workgroups run at once.  Layer plans of the spectral-kernel CIC layer (the
 * plan's layer for the stack call); FDC_EINVAL for other plans or layers. */
fdc_status fdc_cic_layer_dk_ranges(const fdc_layer_plan *plan, int *ranges);
fdc_status fdc_cic_stack_dk_ranges(const fdc_stack_plan *plan, int layer, int *ranges);
/* The first layer of the stack's LDS-resident tail (the last two layers run by
 * "tail_fwd_<N>_<M1>_<M2>", "tail_bwd_<N>_<M1>_<M2>" and one "gk_reduce" launch),
 * or -1 when every layer runs on the per-layer kernels.  The dK ranges query does
 * not apply to the tail's two layers. */
fdc_status fdc_cic_stack_tail(const fdc_stack_plan *plan, int *first_layer);

#ifdef __cplusplus
}
#endif
#endif /* FDC_H */
