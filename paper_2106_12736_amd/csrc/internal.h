// Internal interface between the C ABI (api.cpp) and the kernel launchers
// (kernels.hip, full_fdc.hip).  Not installed; not part of the ABI.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <cstdint>

#include "fdc.h"

namespace fdc {

// How a logical rows x cols image maps onto a stored image (row stride `cols_stored`).
//   mode 0: identity.
//   mode 1: artifact crop -- logical (r, w) is stored at (r - shift, w - shift) when
//           both are >= 0, and is absent (zero on load, dropped on store) otherwise.
//   mode 2: artifact roll -- logical (r, w) is stored at ((r - shift) mod rows,
//           (w - shift) mod cols).
struct ImgView {
  int mode;
  int shift;
  int rows;         // logical rows
  int cols_stored;  // row stride of the stored image
};

bool size_supported(int n);

// The kernels index rows (and columns) of a batch of images with 32-bit integers.
// The C ABI checks these limits on the host, at plan creation or at the top of a
// call without a plan, so that a call that fails enqueues nothing.
// index_fits(planes, n): planes * n < 2^31.
inline bool index_fits(long long planes, long long n) {
  return planes > 0 && n > 0 && planes <= ((1LL << 31) - 1) / n;
}

// Storage of a half spectrum of `planes` images with `rows` rows and L stored bins
// per row.  Bins l < L-1 of row r of plane p are at
// main[p*ps + r*rs + (l/8)*ts + l%8] (the 8-bin tiles of a row are ts apart; ts = 8
// is row-major); the last bin, l = L-1, is at side[p*sps + r*srs].
//   plain: the row-major [planes][rows][L] array (side = main + L - 1).
//   split: a row-major main block [planes][rows][L-1] followed by the last column
//          as a [planes][rows] block.  With L - 1 = n/2 a power of two every main
//          row starts on an aligned boundary, and the odd last column is contiguous
//          along the rows.
//   tiled: the split layout with the main block of each plane stored as column
//          tiles [planes][(L-1)/8][rows][8]: a column transform's tile of 8
//          columns is one contiguous run down the rows (64-byte row pieces read
//          from a row-major block run at half the HBM rate), and two adjacent rows
//          of a tile share a 128-byte line, as a row transform's pair of rows
//          reads them.  Used for every intermediate of the CIC layer path.
struct SpecLayout {
  float2 *main;
  long long ps;
  long long rs;
  long long ts;
  float2 *side;
  long long sps;
  long long srs;
};
// Offset of bin l (< L-1) inside its row of the main block.
__host__ __device__ __forceinline__ long long bin_off(const SpecLayout &s, int l) {
  return (long long)(l >> 3) * s.ts + (l & 7);
}
inline SpecLayout plain_layout(const float2 *p, int rows, int L) {
  float2 *q = const_cast<float2 *>(p);
  return SpecLayout{q, (long long)rows * L, L, 8, q + (L - 1), (long long)rows * L, L};
}
inline SpecLayout split_layout(const float2 *p, long long planes, int rows, int L) {
  float2 *q = const_cast<float2 *>(p);
  return SpecLayout{q, (long long)rows * (L - 1), L - 1, 8, q + planes * rows * (L - 1), rows, 1};
}
// Tiles of 8 bins when L - 1 is a multiple of 8; narrower rows are one tile (the
// split layout).
inline SpecLayout tiled_layout(const float2 *p, long long planes, int rows, int L) {
  if ((L - 1) % 8 != 0) return split_layout(p, planes, rows, L);
  float2 *q = const_cast<float2 *>(p);
  return SpecLayout{q, (long long)rows * (L - 1), 8, (long long)rows * 8, q + planes * rows * (L - 1), rows, 1};
}
// Layout of `planes` P x (P/2+1) Full FDC spectra.  Main block: row k of every plane
// side by side, plane i's bins l < P/2 of row k at main[(k * planes + i) * R + l] with
// R = FDC_FULL_ROW(P) (P/2 plus padding), so that one bin of all planes -- what the
// per-bin channel contractions read -- lies within planes * R elements.  Side block
// (column P/2): plane i's P bins at side[i * FDC_FULL_SIDE_PLANE(P) + k].
inline SpecLayout full_spec_layout(const float2 *p, long long planes, int P) {
  float2 *q = const_cast<float2 *>(p);
  const long long R = FDC_FULL_ROW(P);
  return SpecLayout{q, R, planes * R, 8, q + (long long)P * planes * R, FDC_FULL_SIDE_PLANE(P), 1};
}
inline long long full_spec_elems(long long planes, int P) {
  return planes * ((long long)P * FDC_FULL_ROW(P) + FDC_FULL_SIDE_PLANE(P));
}

// Kernel timing (enabled through the ABI): the start and stop events of the next slot
// when launches of `name` are being timed, else false.
bool timing_slot(const char *name, hipEvent_t *start, hipEvent_t *stop);

// Launch kern; while its launches are timed, through hipExtLaunchKernelGGL with a slot's
// events, which the dispatch itself records at the kernel's start and end (so the
// interval is the kernel's execution, without event records of their own around it).
template <class Kern, class... Args>
inline hipError_t timed_launch(const char *name, Kern kern, dim3 grid, dim3 block, size_t lds, hipStream_t s,
                               Args... args) {
  hipEvent_t e0, e1;
  if (timing_slot(name, &e0, &e1))
    hipExtLaunchKernelGGL(kern, grid, block, (std::uint32_t)lds, s, e0, e1, 0u, args...);
  else
    hipLaunchKernelGGL(kern, grid, block, lds, s, args...);
  return hipGetLastError();
}

// The bins of a kernel gradient gK [S][N][N/2+1] that an FDP N -> M drops (rows
// M/2 <= k < N - M/2, and the columns l > M/2 of the other rows): p == NULL for none.
struct ZeroBins {
  float2 *p;
  int S, N, M;
};

// Row transforms of real rows of length n (n in the supported set), processed in pairs.
// rows_per_plane must be even.  Output/input bins beyond L are not written / read as zero;
// the L stored bins are laid out as `spec` says.
//   r2c: out[plane][row][l] = w_l * sum_w x[plane][row][w] e^{-2 pi i w l / n},  l < L
//   c2r: y[plane][row][w] = sum_{l<=n/2} c_l Re(w_l in[plane][row][l] e^{+2 pi i w l / n}),
//        with the imaginary part of bins 0 and n/2 discarded (real-part semantics)
// where w_l = alpha at l = 0 and l = n/2 and alpha * beta otherwise.
hipError_t launch_row_r2c(int n, const float *x, SpecLayout out, long long planes, int rows_per_plane,
                          ImgView in_view, long long in_plane_stride, int L, float alpha, float beta, hipStream_t s);
hipError_t launch_row_c2r(int n, SpecLayout in, float *y, long long planes, int rows_per_plane, int L, float alpha,
                          float beta, ImgView out_view, long long out_plane_stride, hipStream_t s);
// Inverse then forward real row transforms of the same rows (a boundary between two
// stacked layers): launch_row_c2r(in, Lin, a1, b1) followed by launch_row_r2c(out,
// Lout, a2, b2) with the real rows kept in registers.  The same launch also writes the
// zeros of `zeros` (a kernel gradient the next dK launch then leaves to it).
hipError_t launch_row_c2r_r2c(int n, SpecLayout in, int Lin, float a1, float b1, SpecLayout out, int Lout, float a2,
                              float b2, long long planes, int rows_per_plane, hipStream_t s,
                              ZeroBins zeros = ZeroBins{nullptr, 0, 0, 0});

// Column DFTs of length n over the first `L` columns of row-major [planes][n][ld] complex
// data (in place allowed).
hipError_t launch_col_fft(int n, int dir, const float2 *in, float2 *out, long long planes, int L, int ld,
                          long long in_plane_stride, long long out_plane_stride, hipStream_t s,
                          int keep = 0);  // keep > 0: store only the rows an FDP to keep rows keeps
// Column DFTs of `planes` split-layout n x (n/2+1) half spectra with the strides of
// `in` and `out` (in place allowed).
hipError_t launch_col_fft_split(int n, int dir, SpecLayout in, SpecLayout out, long long planes, hipStream_t s);
// Forward column DFTs of length n over the L columns of `planes` row spectra in the
// layout `in` (the tiled layout of a row pass), storing the rows an FDP to `keep` rows
// keeps into the row-major out [planes][n][ld] at their own row indices.
hipError_t launch_col_fft_keep(int n, SpecLayout in, float2 *out, long long planes, int L, int ld, int keep,
                               hipStream_t s);

// Fused CIC + FDP column kernels (square n x n images pooled to m x m; L = m/2 + 1).
// T, Xh, U, Tg and V are split-layout spectra (SpecLayout) with L bins per row.
//   fwd:   T [B*C][n rows] -> Xh [B*C][m rows] and U [B*S][m rows] (one kernel, or two
//          with Xh written and read back)
//   bwd_gk: Tg [B*S][m rows], Xh -> gK [S][n][n/2+1]: every bin (zeros where FDP drops)
//   bwd_gx: Tg, K -> V [B*C][n rows]
bool cic_pair_supported(int n, int m);
// Output channels per workgroup when the forward's two column kernels run as one
// (k_col_fwd_cic) for J = S / C and n-point columns, else 0.
int fwd_cic_jw(int J, int n);
hipError_t launch_col_fwd_cic(int n, int m, const float2 *T, const float2 *K, float2 *U, float2 *Xh, int B,
                              int C, int S, hipStream_t s);
// dK: with scratch `part` (part_elems complex values; may be NULL) the batch is cut
// into gk_batch_ranges(...) ranges whose sums are added in order by a second kernel.
// zeros = false: the dropped bins of gK are left as they are (an earlier launch of the
// same call wrote their zeros, or the caller's buffer holds them).
int gk_batch_ranges(int n, int m, int B, int S, long long part_elems);
hipError_t launch_col_bwd_gk(int n, int m, const float2 *Tg, const float2 *Xh, float2 *gK, int B, int C,
                             int S, float2 *part, long long part_elems, hipStream_t s, bool zeros = true);
hipError_t launch_col_bwd_gx(int n, int m, const float2 *Tg, const float2 *K, float2 *V, int B, int C, int S,
                             hipStream_t s);
// gK [S][N][N/2+1] from BG partial sums part [BG][S][M][M/2+1] (plain layout): at the
// kept bins the partial sums added in order, exact zeros elsewhere (zeros = false: the
// kept bins only); one launch for one reduction (part1 NULL) or two.
hipError_t launch_gk_reduce2(const float2 *part0, float2 *gK0, int S0, int M0, int N0, const float2 *part1,
                             float2 *gK1, int S1, int M1, int N1, int BG, hipStream_t s, bool zeros = true);
// dK (one batch range) and dX of one layer in a single launch, where the dX tiles pack
// the dK workgroup (col_bwd_dk_dx_supported); zeros as for launch_col_bwd_gk.
bool col_bwd_dk_dx_supported(int n, int m);
hipError_t launch_col_bwd_dk_dx(int n, int m, const float2 *Tg, const float2 *Xh, const float2 *K, float2 *gK,
                                float2 *V, int B, int C, int S, hipStream_t s, bool zeros = true);

// The last two layers of a stack with all intermediates in LDS (tail.hip): layer a
// (na -> ma, fan-out ja) and layer b (ma -> mb, fan-out jb), one workgroup per input
// plane (b, c) of layer a, B * C workgroups.
//   fwd: in = previous layer's column-inverted spectra (split [B C][na][na/2+1]) with
//        inverse weight a_in, or x = input images [B][C][na][na] (x non-NULL);
//        saved_a split [B C][ma][ma/2+1], saved_b split [B C ja][mb][mb/2+1]; y.
//   bwd: part_a plain [B][C ja][ma][ma/2+1], part_b plain [B][C ja jb][mb][mb/2+1]
//        (per-image dK products; launch_gk_reduce sums them); out_mode 0: Tg split
//        [B C][na][na/2+1] with weights (c_l a_out); 1: gx [B][C][na][na]; 2: none.
bool tail_supported(int na, int ma, int mb, int ja, int jb);
// Whole 2-D transforms of small square planes in one launch (tail.hip): forward
// x [count][n][n] -> X [count][n][n/2+1] with row weights (alpha, beta), or inverse
// Xi -> xo with c-weights (alpha, beta) and real-part semantics.
bool fft2_small_supported(int h, int w);
hipError_t launch_fft2_small(int n, bool inverse, const float *x, float2 *X, float *xo, const float2 *Xi,
                             long long count, float alpha, float beta, hipStream_t s);
hipError_t launch_tail_fwd(int na, int ma, int mb, int ja, int jb, SpecLayout in, const float *x, float a_in,
                           const float2 *Ka, const float2 *Kb, SpecLayout saved_a, SpecLayout saved_b, float *y,
                           int B, int C, hipStream_t s);
hipError_t launch_tail_bwd(int na, int ma, int mb, int ja, int jb, const float *gy, SpecLayout saved_a,
                           SpecLayout saved_b, const float2 *Ka, const float2 *Kb, float2 *part_a, float2 *part_b,
                           int out_mode, SpecLayout Tg, float a_out, float *gx, int B, int C, hipStream_t s);

// Full FDC (full_fdc.hip).  Spectra in the padded split layout full_spec_layout,
// P a multiple of 8; tw is the device table
// W^j = exp(-2 pi i j / P), j < P.  Rearranged weights take full_weight_floats(KD, ND, nk)
// floats: KD = Cin, ND = Cout forward (gx = false); KD = Cout, ND = Cin for dL/dX.
bool full_kernel_size_supported(int nk);
size_t full_weight_floats(int KD, int ND, int nk);
int full_gw_chunks(int B, int S, int C, int P, int nk);
// Whether every Full FDC launch of a layer (both contractions, dL/dw and its reduction)
// fits its grid limits.
bool full_launch_fits(int B, int Cin, int Cout, int P, int nk);
hipError_t launch_full_weights(const float *w, float *wt, bool gx, int S, int C, int nk, hipStream_t s);
hipError_t launch_full_contract(bool gx, int nk, SpecLayout in, const float *wt, const float2 *tw, SpecLayout out,
                                int B, int KD, int ND, int P, hipStream_t s);
hipError_t launch_full_gw(int nk, SpecLayout G, SpecLayout X, const float2 *tw, float *part, float *gw, int B, int S,
                          int C, int P, hipStream_t s);

// Spectral CIC and FDP.
hipError_t launch_cic_fwd(const float2 *X, const float2 *K, float2 *Y, int B, int C, int S, long long P,
                          hipStream_t s);
hipError_t launch_cic_bwd_gx(const float2 *gY, const float2 *K, float2 *gX, int B, int C, int S, long long P,
                             hipStream_t s);
hipError_t launch_cic_bwd_gk(const float2 *gY, const float2 *X, float2 *gK, int B, int C, int S, long long P,
                             hipStream_t s);
// Spatial-kernel CIC: kernel spectra of n x n kernels at the kept bins of an n_img -> M
// layer (into K [S][n_img][n_img/2+1]), and dL/dw from dK (part: S * cic_wgrad_blocks(M)
// * n * n floats of scratch).
bool spatial_kernel_size_supported(int n);
// Output channels the spatial-kernel weight-gradient launch accepts.
bool spatial_channels_supported(int S);
int cic_wgrad_blocks(int M);
// One layer of a batched spatial-kernel call (k_cic_kspec_stack, k_cic_wgrad_stack):
// the caller fills w, K (kspec) or gK, part, gw (wgrad), N, M, S, n and roll (the ROLL
// shift s, 0 for none); the launchers fill the grid fields.
struct SpatialLayer {
  const float *w;
  float2 *K;
  const float2 *gK;
  float *part, *gw;
  int N, M, S, n, roll;
  int ncb, rowb, block0, elem0;
};
constexpr int kSpatialBatch = 8;
struct SpatialBatch {
  SpatialLayer layer[kSpatialBatch];
  int count;
};
// partial sums per output channel of launch_cic_wgrad_stack for an M-point layer
int cic_wgrad_stack_blocks(int M);
hipError_t launch_cic_kspec_stack(SpatialBatch sb, hipStream_t s);
// Pi_H of half spectra [count][H][Wf] in place (columns 0 and Wf-1 only).
hipError_t launch_hermitian_columns(float2 *Y, long long count, int H, int Wf, hipStream_t s);
hipError_t launch_cic_wgrad_stack(SpatialBatch sb, hipStream_t s);
hipError_t launch_cic_kspec(int n_img, const float *w, float2 *K, int S, int n, int M, hipStream_t s);
hipError_t launch_cic_wgrad(int n_img, const float2 *gK, float *part, float *gw, int S, int n, int M,
                            hipStream_t s);
// FDC layer of the FDCNN on spectra followed by FDP (only the kept bins are formed), and
// its backward (gX and gK with exact zeros at the dropped bins).
// Largest spectrum the spectral FDC + FDP kernels index: N (N/2 + 1) bins below 2^24.
bool cic_fdp_size_supported(int N);
// project: Y written as Pi_H(Y).
hipError_t launch_cic_fdp_fwd(const float2 *X, const float2 *K, float2 *Y, int B, int C, int S, int N, int M,
                              bool project, hipStream_t s);
// gX (NULL: skipped; needs K) and gK (NULL: skipped; needs X) in one launch; project:
// gX written as Pi_H(gX); kept: the bins the FDP drops are not written (with project,
// columns 0 and N/2 of gX are still written over every row).
hipError_t launch_cic_fdp_bwd(const float2 *gY, const float2 *K, float2 *gX, const float2 *X, float2 *gK, int B,
                              int C, int S, int N, int M, bool project, bool kept, hipStream_t s);
hipError_t launch_fdp_gather(const float2 *X, float2 *Y, long long count, int H, int Wf, int Mh, int Mwf,
                             hipStream_t s);
hipError_t launch_fdp_scatter(const float2 *gY, float2 *gX, long long count, int H, int Wf, int Mh, int Mwf,
                              hipStream_t s);

// FDCNN classifier head and Adam (head.hip).  At most kHeadMaxClasses classes; the
// forward takes head_chunks(F) * B * classes floats of scratch (partial logits).
constexpr int kHeadMaxClasses = 16;
constexpr int kHeadMaxPairs = 15872;  // B * classes: the logits in LDS next to a 1 KB reduction buffer
long long head_chunks(long long F);
hipError_t launch_head_forward(const float *y, const float *W, const float *bias, const int *labels, float *logits,
                               float *loss, float *part, int B, long long F, int classes, hipStream_t s);
// The forward without a caller workspace: the partial logits go to a file-scope
// device array of kHeadScratchFloats floats (one per device, shared by all calls on
// it).  Requires head_chunks(F) * B * classes <= kHeadScratchFloats.
constexpr long long kHeadScratchFloats = 1LL << 18;
hipError_t head_scratch_address(float **out);
hipError_t launch_head_forward_noalloc(const float *y, const float *W, const float *bias, const int *labels,
                                       float *logits, float *loss, int B, long long F, int classes, hipStream_t s);
hipError_t launch_head_backward(const float *y, const float *W, const float *logits, const int *labels, float *gy,
                                float *gW, float *gbias, int B, long long F, int classes, hipStream_t s);
hipError_t launch_adam(float *p, const float *g, float *m, float *v, long long n, int *count, float lr, float beta1,
                       float beta2, float eps, float wd, hipStream_t s);

}  // namespace fdc
