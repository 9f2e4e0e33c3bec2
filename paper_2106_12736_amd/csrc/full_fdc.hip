// Full FDC (Algorithm 2 with the per-bin sum over input channels of Eq. 2) on the
// fp32 matrix cores of gfx950, and its backward.
//
// At every frequency bin (k, l) of the P x (P/2+1) half spectrum the layer is a
// small complex matrix product over the batch:
//   forward  Y[b][s] = sum_c X[b][c] K[s][c]            (M = b, N = s, K-dim = c)
//   dL/dX    gX[b][c] = sum_s G[b][s] conj(K[s][c])      (M = b, N = c, K-dim = s)
//   dL/dK    gK[s][c] = sum_b G[b][s] conj(X[b][c])      (M = s, N = c, K-dim = b)
// with K[s][c](k, l) = sum_{a,b < n} w[s][c][a][b] W^(k a) W^(l b), W = e^{-2 pi i / P}:
// the n x n spatial kernel padded at the top-left corner to P x P and transformed
// (section 2.4.1.2).  K is never stored: each lane forms the element it feeds to the
// matrix core from the n*n weights and the bin's phases, so the contraction reads
// only X (or G) and the weights.  dL/dw is the adjoint of that map restricted to the
// n x n support, dL/dw[s][c][a][b] = Re sum_bins gK[s][c] conj(W^(k a) W^(l b)),
// accumulated per bin chunk and reduced in a fixed order.
//
// Spectra use the split layout of a P x (P/2+1) half spectrum: a main block of
// P x P/2 planes (columns 0..P/2-1) followed by a side block of P-element planes (the
// Nyquist column l = P/2), so that runs of 4 bins are 32-byte aligned.  In the main
// block row k of every plane lies side by side (full_spec_layout), so the planes a
// run's contraction reads are a few MB apart rather than a plane apart.
//
// Complex products use four real v_mfma_f32_16x16x4f32 per 4-deep K step:
//   re += Ar Br - Ai Bi,  im += Ar Bi + Ai Br.
// Lane layout of v_mfma_f32_16x16x4f32 (A 16x4, B 4x16, D 16x16): lane l holds
// A[l % 16][l / 16], B[l / 16][l % 16] and D[4 (l / 16) + j][l % 16] in register j.
#include "device.h"
#include "internal.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <string>

namespace fdc {

typedef float v4f __attribute__((ext_vector_type(4)));

__device__ __forceinline__ v4f mfma4(float a, float b, v4f c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// Taps of an n x n kernel, padded to a multiple of 4 for whole 16-byte loads.
template <int NK>
__host__ __device__ constexpr int tap_pad() {
  return (NK * NK + 3) & ~3;
}

// ---------------------------------------------------------------------------
// Forward (GX = false) and dL/dX (GX = true) contraction on split-layout spectra.
//   in  [B][KD] spectra: X (KD = Cin) or G (KD = Cout)
//   wt  weights rearranged as [KDp][NDp][TP], zero-padded (forward: [c][s][tap];
//       dL/dX: [s][c][tap]); KDp = KD rounded up to 4, NDp = ND rounded up to 64
//   out [B][ND] spectra: Y (ND = Cout) or gX (ND = Cin)
// The bins of a spectrum are cut into runs of 4: along a row of the main block
// (same k, four consecutive l) or down the Nyquist column (four consecutive k,
// l = P/2).  A wave owns one run, 16 batch rows and 64 outputs (four 16 x 16 D
// tiles per bin); a workgroup is 4 waves on 4 consecutive runs and the same
// outputs, so their weight loads coincide in L1.  Inside a run the kernel
// spectrum factorises: for a row run K(k, l) = sum_b W^(l b) C_b with
// C_b = sum_a w_ab W^(k a) shared by the 4 bins; for a Nyquist run W^(l b) = (-1)^b
// and K(k, P/2) = sum_a W^(k a) R_a with R_a = sum_b (-1)^b w_ab.
// Every load is unconditional: batch rows and channels past the end are clamped
// to the last valid ones (their weights are zero, their outputs are not stored).
// ---------------------------------------------------------------------------
constexpr int kCtOut = 64;  // outputs per workgroup

template <int NK, bool GX, bool SIDE>
__device__ __forceinline__ void contract_run(const float2 *__restrict__ in, const float *__restrict__ wt,
                                             float2 *__restrict__ out, const float2 (&zs)[NK],
                                             const float2 (&zq)[4][NK], long long pst, long long opst, int B,
                                             int KD, int KDp, int ND, int NDp, int b0, int n0) {
  constexpr int TP = tap_pad<NK>();
  const int lane = threadIdx.x & 63, mrow = lane & 15, kk = lane >> 4;
  v4f accr[4][4], acci[4][4];  // [bin q][tile t]
#pragma unroll
  for (int q = 0; q < 4; ++q)
#pragma unroll
    for (int t = 0; t < 4; ++t) accr[q][t] = acci[q][t] = v4f{0.f, 0.f, 0.f, 0.f};

  const int ba = min(b0 + mrow, B - 1);  // A operand row (batch)
  const float2 *arow = in + (long long)ba * KD * pst;
  // the inputs and the weights of all four tiles are loaded one k-step ahead
  auto load_a = [&](int k0, float4 (&a)[2]) {
    const float4 *a4 = reinterpret_cast<const float4 *>(arow + (long long)min(k0 + kk, KD - 1) * pst);
    a[0] = a4[0], a[1] = a4[1];
  };
  auto load_w = [&](int k0, int t, float4 (&w)[TP / 4]) {
    const float4 *w4 = reinterpret_cast<const float4 *>(wt + ((long long)(k0 + kk) * NDp + n0 + 16 * t + mrow) * TP);
#pragma unroll
    for (int i = 0; i < TP / 4; ++i) w[i] = w4[i];
  };
  float4 an[2], wn[4][TP / 4];
  load_a(0, an);
#pragma unroll
  for (int t = 0; t < 4; ++t) load_w(0, t, wn[t]);
  for (int k0 = 0; k0 < KDp; k0 += 4) {
    const float4 lo = an[0], hi = an[1];
    float4 wc[4][TP / 4];
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int i = 0; i < TP / 4; ++i) wc[t][i] = wn[t][i];
    if (k0 + 4 < KDp) {
      load_a(k0 + 4, an);
#pragma unroll
      for (int t = 0; t < 4; ++t) load_w(k0 + 4, t, wn[t]);
    }
    const float ar[4] = {lo.x, lo.z, hi.x, hi.z}, ai[4] = {lo.y, lo.w, hi.y, hi.w};
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      float w[TP];
#pragma unroll
      for (int i = 0; i < TP / 4; ++i)
        w[4 * i] = wc[t][i].x, w[4 * i + 1] = wc[t][i].y, w[4 * i + 2] = wc[t][i].z, w[4 * i + 3] = wc[t][i].w;
      // the run-invariant half of the kernel spectrum
      float2 y[NK];
      if constexpr (!SIDE) {
#pragma unroll
        for (int b = 0; b < NK; ++b) {  // C_b = w_0b + sum_{a>=1} w_ab u_a
          float cx = w[b], cy = 0.f;
#pragma unroll
          for (int a = 1; a < NK; ++a) {
            cx = fmaf(w[a * NK + b], zs[a].x, cx);
            cy = fmaf(w[a * NK + b], zs[a].y, cy);
          }
          y[b] = make_float2(cx, cy);
        }
      } else {
#pragma unroll
        for (int a = 0; a < NK; ++a) {  // R_a = sum_b (-1)^b w_ab
          float r = w[a * NK];
#pragma unroll
          for (int b = 1; b < NK; ++b) r += (b & 1) ? -w[a * NK + b] : w[a * NK + b];
          y[a] = make_float2(r, 0.f);
        }
      }
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        // K = y_0 + sum_{i>=1} z_qi y_i  (z_q0 = 1)
        float kr = y[0].x, ki = y[0].y;
#pragma unroll
        for (int i = 1; i < NK; ++i) {
          if constexpr (!SIDE) {
            kr = fmaf(zq[q][i].x, y[i].x, kr);
            kr = fmaf(-zq[q][i].y, y[i].y, kr);
            ki = fmaf(zq[q][i].x, y[i].y, ki);
            ki = fmaf(zq[q][i].y, y[i].x, ki);
          } else {
            kr = fmaf(zq[q][i].x, y[i].x, kr);
            ki = fmaf(zq[q][i].y, y[i].x, ki);
          }
        }
        // forward: re += Ar Kr - Ai Ki, im += Ar Ki + Ai Kr
        // dL/dX (conj K): re += Ar Kr + Ai Ki, im += Ai Kr - Ar Ki
        accr[q][t] = mfma4(ar[q], kr, accr[q][t]);
        accr[q][t] = mfma4(GX ? ai[q] : -ai[q], ki, accr[q][t]);
        acci[q][t] = mfma4(GX ? -ar[q] : ar[q], ki, acci[q][t]);
        acci[q][t] = mfma4(ai[q], kr, acci[q][t]);
      }
    }
  }
  // D[m][n]: lane holds rows 4 (lane / 16) + j, column lane % 16 of each tile
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const int n = n0 + 16 * t + mrow;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int b = b0 + 4 * kk + j;
      if (b >= B || n >= ND) continue;
      float4 *o = reinterpret_cast<float4 *>(out + ((long long)b * ND + n) * opst);
      o[0] = make_float4(accr[0][t][j], acci[0][t][j], accr[1][t][j], acci[1][t][j]);
      o[1] = make_float4(accr[2][t][j], acci[2][t][j], accr[3][t][j], acci[3][t][j]);
    }
  }
}

template <int NK, bool GX>
__global__ __launch_bounds__(256) void k_full_contract(SpecLayout in, const float *__restrict__ wt,
                                                       const float2 *__restrict__ tw, SpecLayout out, int B, int KD,
                                                       int KDp, int ND, int NDp, int P, int nwg_run, int nsb) {
  const int H = P / 2;
  const int nmain = P * H / 4, nrun = nmain + P / 4;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int blk = xcd_remap(blockIdx.x, gridDim.x);
  const int sb = blk % nsb, rest = blk / nsb;
  const int g = (rest % nwg_run) * 4 + wave, bt = rest / nwg_run;
  if (g >= nrun) return;  // no barriers in this kernel
  if (g < nmain) {
    const int k = (4 * g) / H, l0 = 4 * g - k * H;
    float2 u[NK], v[4][NK];
#pragma unroll
    for (int a = 0; a < NK; ++a) u[a] = tw[(k * a) % P];
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
      for (int b = 0; b < NK; ++b) v[q][b] = tw[((l0 + q) * b) % P];
    contract_run<NK, GX, false>(in.main + k * in.rs + l0, wt, out.main + k * out.rs + l0, u, v, in.ps, out.ps, B, KD,
                                KDp, ND, NDp, bt * 16, sb * kCtOut);
  } else {
    const int k0 = 4 * (g - nmain);
    float2 z[NK], u[4][NK];
#pragma unroll
    for (int b = 0; b < NK; ++b) z[b] = make_float2((b & 1) ? -1.f : 1.f, 0.f);
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
      for (int a = 0; a < NK; ++a) u[q][a] = tw[((k0 + q) * a) % P];
    contract_run<NK, GX, true>(in.side + k0, wt, out.side + k0, z, u, in.sps, out.sps, B, KD, KDp, ND, NDp, bt * 16,
                               sb * kCtOut);
  }
}

// ---------------------------------------------------------------------------
// dL/dw partial sums over one chunk of runs (runs as in the contraction).
//   G [B][S], X [B][C] split-layout spectra; part [chunk][S][C][NK*NK] float
// Per bin gK[s][c] = sum_b G[b][s] conj(X[b][c]) on the matrix cores (M = s, N = c,
// K-dim = b, 4 batch rows per step), then
//   dL/dw[s][c][a][b] = Re sum_bins gK conj(W^(k a) W^(l b)),
// done per run: a row run sums E_b = sum_q gK_q conj(W^(l_q b)) and adds
// Re(E_b conj(W^(k a))); a Nyquist run sums F_a = sum_q gK_q conj(W^(k_q a)) and adds
// (-1)^b Re(F_a).  A workgroup (4 waves) owns a 32 x 32 (s, c) block, each wave a
// 16 x 16 tile, and walks its chunk one run (4 bins) at a time, 4 batch rows per step.
// A step's G and X rows are loaded once per workgroup and staged in LDS, and the
// loads of step t + 2 are in flight while step t computes.  Loads are unconditional:
// batch rows past the end are clamped and staged as zeros, channels and runs past the
// end are clamped and their results dropped.
// ---------------------------------------------------------------------------
// Twiddles W^i for i < n P in LDS: every phase index the projection forms (k a,
// (l + q) b with k < P, l + q < P/2, a, b < n) is then a plain table index.
template <int NK>
__host__ __device__ constexpr int gw_tw_elems(int P) {
  return (NK * P + 31) & ~31;
}

// Adds one run's gK (4 bins: dr/di[q], lane rows j) projected onto the taps to gw.
// Row run (k, l0..l0+3); Nyquist run (k0..k0+3, P/2) when SIDE.  The phases of tap
// row / column 0 are exactly 1, so their products are plain sums.
template <int NK, bool SIDE>
__device__ __forceinline__ void gw_project_run(float (&gw)[4][NK * NK], const v4f (&dr)[4], const v4f (&di)[4], int k,
                                               int l0, const float2 *tw) {
  if constexpr (!SIDE) {
    float2 u[NK], v[4][NK];
#pragma unroll
    for (int a = 1; a < NK; ++a) u[a] = tw[k * a];
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
      for (int b = 1; b < NK; ++b) v[q][b] = tw[(l0 + q) * b];
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int b = 0; b < NK; ++b) {
        float ex, ey;  // E_b = sum_q D_q conj(v_qb)
        if (b == 0) {
          ex = (dr[0][j] + dr[1][j]) + (dr[2][j] + dr[3][j]);
          ey = (di[0][j] + di[1][j]) + (di[2][j] + di[3][j]);
        } else {
          ex = ey = 0.f;
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            ex = fmaf(dr[q][j], v[q][b].x, ex);
            ex = fmaf(di[q][j], v[q][b].y, ex);
            ey = fmaf(di[q][j], v[q][b].x, ey);
            ey = fmaf(-dr[q][j], v[q][b].y, ey);
          }
        }
        gw[j][b] += ex;
#pragma unroll
        for (int a = 1; a < NK; ++a) gw[j][a * NK + b] = fmaf(ey, u[a].y, fmaf(ex, u[a].x, gw[j][a * NK + b]));
      }
  } else {
    float2 u[4][NK];
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
      for (int a = 1; a < NK; ++a) u[q][a] = tw[(k + q) * a];
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int a = 0; a < NK; ++a) {
        float f;  // Re F_a = Re sum_q D_q conj(u_qa)
        if (a == 0) {
          f = (dr[0][j] + dr[1][j]) + (dr[2][j] + dr[3][j]);
        } else {
          f = 0.f;
#pragma unroll
          for (int q = 0; q < 4; ++q) f = fmaf(di[q][j], u[q][a].y, fmaf(dr[q][j], u[q][a].x, f));
        }
#pragma unroll
        for (int b = 0; b < NK; ++b) gw[j][a * NK + b] += (b & 1) ? -f : f;
      }
  }
}

// Position of a run of 4 bins, advanced one run at a time (no divisions on the way).
struct GwRun {
  int g, k, l0;  // run index; row k and first column l0 (row runs) or first row k (Nyquist runs)
  __device__ void start(int g0, int nmain, int H) {
    g = g0;
    if (g < nmain) {
      k = (4 * g) / H, l0 = 4 * g - k * H;
    } else {
      k = 4 * (g - nmain), l0 = 0;
    }
  }
  __device__ void next(int nmain, int H) {
    ++g;
    if (g == nmain) {
      k = 0, l0 = 0;
    } else if (g > nmain) {
      k += 4;
    } else if ((l0 += 4) == H) {
      l0 = 0, ++k;
    }
  }
};

// LDS staging of one step (4 batch rows, one run of 4 bins) for a 32 x 32 (s, c)
// block: G rows [4][32][5] and X rows [4][32][5] complex, each (b, s) row holding the
// run's 4 bins and one of padding.  Every element is loaded from memory once per
// workgroup (the four waves read each operand row twice: waves 0/1 share s rows, 0/2
// share c rows).
constexpr int kGwStageRow = 5;
// X rows start 8 elements (16 banks of 4 bytes) after the G rows: the staging writes of
// a 16-lane group (8 rows of G and the same 8 rows of X) then fall on distinct banks
// (with the two blocks a multiple of 32 banks apart every write was a 2-way conflict)
constexpr int kGwStageUnit = 4 * 32 * kGwStageRow + 8;
constexpr int kGwStageElems = 2 * kGwStageUnit;

// EVEN: the batch takes an even number of 4-row steps (B rounded up to 4 is a multiple
// of 8), which allows the run-by-run loop.
template <int NK, bool EVEN>
__global__ __launch_bounds__(256, 2) void k_full_gw(SpecLayout G, SpecLayout X, const float2 *__restrict__ twg,
                                                 float *__restrict__ part, int B, int S, int C, int P,
                                                 int runs_per_chunk) {
  constexpr int T = NK * NK, SR = kGwStageRow, SE = kGwStageElems;
  extern __shared__ float smem[];
  float2 *tw = reinterpret_cast<float2 *>(smem);
  float2 *stage = tw + gw_tw_elems<NK>(P);  // two buffers of SE
  for (int i = threadIdx.x; i < NK * P; i += 256) tw[i] = twg[i % P];
  __syncthreads();

  const int H = P / 2, nmain = P * H / 4, nrun = nmain + P / 4;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int mrow = lane & 15, kq = lane >> 4;
  const int sblocks = (S + 31) / 32, cblocks = (C + 31) / 32;
  const int blk = xcd_remap(blockIdx.x, gridDim.x);
  const int tile = blk % (sblocks * cblocks), chunk = blk / (sblocks * cblocks);
  const int sbase = (tile / cblocks) * 32, cbase = (tile % cblocks) * 32;
  const int s0 = sbase + (wave >> 1) * 16, c0 = cbase + (wave & 1) * 16;
  const int r_begin = chunk * runs_per_chunk, r_end = min(nrun, r_begin + runs_per_chunk);

  // Cooperative loads: wave lb takes batch row b0 + lb of the step; lane (lr, unit)
  // loads the run's 4 bins of G row sbase + lr (unit 0) or X row cbase + lr (unit 1).
  // Per-lane bases and batch strides of both blocks, so that a step's address is one
  // multiply-add.
  const int lb = wave, unit = lane & 1, lr = lane >> 1;
  const SpecLayout &L = unit ? X : G;
  const long long row = unit ? min(cbase + lr, C - 1) : min(sbase + lr, S - 1);
  const long long nch = unit ? C : S;
  const float2 *mbase = L.main + row * L.ps, *sbase_p = L.side + row * L.sps;
  const long long mbst = nch * L.ps, sbst = nch * L.sps, mrs = L.rs;

  float gw[4][T];  // rows s0 + 4 (lane / 16) + j, column c0 + lane % 16
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int t = 0; t < T; ++t) gw[j][t] = 0.f;

  // Two register sets hold the loads of the next two steps, so that the loads of step
  // t + 2 are in flight while step t computes.  Past the chunk's last step the run is
  // clamped and the load is not used: an unconditional load keeps the wait counts
  // exact, so step t waits for its own loads only.
  GwRun lrun;
  lrun.start(r_begin, nmain, H);
  int lb0 = 0;  // load cursor: run lrun, batch rows lb0..lb0+3
  auto load_next = [&](float4(&r)[2]) {
    const long long bc = min(lb0 + lb, B - 1);
    const bool side = lrun.g >= nmain;
    const int gk = min(lrun.k, side ? P - 4 : P - 1);  // in range past the last run
    const float2 *a = side ? sbase_p + bc * sbst + gk : mbase + bc * mbst + gk * mrs + lrun.l0;
    const float4 *a4 = reinterpret_cast<const float4 *>(a);
    r[0] = a4[0], r[1] = a4[1];
    lb0 += 4;
    if (lb0 >= B) lb0 = 0, lrun.next(nmain, H);
  };
  float4 ra[2], rb[2];
  load_next(ra);
  load_next(rb);
  // Up to 3 x 3 taps and with the run-by-run loop, Gauss's form of the complex
  // product: t1 = sum Gr Xr, t2 = sum Gi Xi and t3 = sum (Gr + Gi)(Xr - Xi) over the
  // batch, three matrix products per bin instead of four; the run's D = G conj(X) is
  // then re = t1 + t2, im = t3 - t1 + t2.  (Elsewhere the third accumulator would
  // cost occupancy or spill, and four products are kept.)
  constexpr bool kGauss = EVEN && NK <= 3;
  v4f t1[4], t2[4], t3[4], dr[4], di[4];
  GwRun crun;
  crun.start(r_begin, nmain, H);
  int b0 = 0;  // compute cursor
  // Stage the registers r (loaded two steps ago) into LDS buffer buf, then this step's
  // products (4 batch rows of the run crun).
  auto stage_and_multiply = [&](float4(&r)[2], int buf) __attribute__((always_inline)) {
    // (the barrier below also ends every wave's reads of this buffer two steps ago)
    {
      float2 *d = stage + buf * SE + unit * kGwStageUnit + (lb * 32 + lr) * SR;
      if (b0 + lb < B) {
        d[0] = make_float2(r[0].x, r[0].y), d[1] = make_float2(r[0].z, r[0].w);
        d[2] = make_float2(r[1].x, r[1].y), d[3] = make_float2(r[1].z, r[1].w);
      } else {  // batch rows past the end add nothing
        d[0] = d[1] = d[2] = d[3] = make_float2(0.f, 0.f);
      }
    }
    __syncthreads();
    load_next(r);
    const float2 *ag = stage + buf * SE + (kq * 32 + (s0 - sbase) + mrow) * SR;
    const float2 *ax = stage + buf * SE + kGwStageUnit + (kq * 32 + (c0 - cbase) + mrow) * SR;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float2 g2 = ag[q], x2 = ax[q];
      if constexpr (kGauss) {
        t1[q] = mfma4(g2.x, x2.x, t1[q]);
        t2[q] = mfma4(g2.y, x2.y, t2[q]);
        t3[q] = mfma4(g2.x + g2.y, x2.x - x2.y, t3[q]);
      } else {  // D = G conj(X):  re = Gr Xr + Gi Xi,  im = Gi Xr - Gr Xi
        dr[q] = mfma4(g2.x, x2.x, dr[q]);
        dr[q] = mfma4(g2.y, x2.y, dr[q]);
        di[q] = mfma4(g2.y, x2.x, di[q]);
        di[q] = mfma4(-g2.x, x2.y, di[q]);
      }
    }
    b0 += 4;
  };
  auto clear_sums = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if constexpr (kGauss)
        t1[q] = t2[q] = t3[q] = v4f{0.f, 0.f, 0.f, 0.f};
      else
        dr[q] = di[q] = v4f{0.f, 0.f, 0.f, 0.f};
    }
  };
  auto finish_run = [&]() __attribute__((always_inline)) {  // project the run onto the taps
    if constexpr (kGauss) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        dr[q] = t1[q] + t2[q];
        di[q] = (t3[q] - t1[q]) + t2[q];
      }
    }
    if (crun.g >= nmain)
      gw_project_run<NK, true>(gw, dr, di, crun.k, crun.l0, tw);
    else
      gw_project_run<NK, false>(gw, dr, di, crun.k, crun.l0, tw);
    b0 = 0;
    crun.next(nmain, H);
  };
  const int spr = (B + 3) / 4;  // steps per run
  if constexpr (EVEN) {
    // An even step count per run (the launcher checks): a run is whole pairs of steps,
    // so the register sets alternate inside it, and the sums are cleared before and
    // projected after it, with no branch on them inside the step loop.
    for (int g = r_begin; g < r_end; ++g) {
      clear_sums();
      for (int t = 0; t < spr; t += 2) {  // one path round the loop keeps the wait counts exact
        stage_and_multiply(ra, 0);
        stage_and_multiply(rb, 1);
      }
      finish_run();
    }
  } else {
    auto step = [&](float4(&r)[2], int buf) __attribute__((always_inline)) {
      if (b0 == 0) clear_sums();
      stage_and_multiply(r, buf);
      if (b0 >= B) finish_run();
    };
    const int nsteps = max(0, r_end - r_begin) * spr;
    int t = 0;
    for (; t + 1 < nsteps; t += 2) {  // one path round the loop keeps the wait counts exact
      step(ra, 0);
      step(rb, 1);
    }
    if (t < nsteps) step(ra, 0);
  }
  // this chunk's partial sums
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int os = s0 + 4 * kq + j, oc = c0 + mrow;
    if (os >= S || oc >= C) continue;
    float *p = part + (((long long)chunk * S + os) * C + oc) * T;
#pragma unroll
    for (int t = 0; t < T; ++t) p[t] = gw[j][t];
  }
}

// dL/dw = sum over chunks in a fixed order: a workgroup owns 64 outputs; its four
// waves sum the chunks congruent to 0, 1, 2, 3 mod 4 (four accumulators each, chunk
// c into accumulator (c / 4) mod 4), and the 16 partial sums are added in order.
__global__ __launch_bounds__(256) void k_full_gw_reduce(const float *__restrict__ part, float *__restrict__ gw,
                                                        long long n, int chunks) {
  __shared__ float red[4][64];
  const int o = threadIdx.x & 63, w = threadIdx.x >> 6;
  const long long i = (long long)blockIdx.x * 64 + o;
  const long long ii = i < n ? i : n - 1;
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
  int c = w;
  for (; c + 12 < chunks; c += 16) {
#pragma unroll
    for (int u = 0; u < 4; ++u) acc[u] += part[(long long)(c + 4 * u) * n + ii];
  }
  for (int u = 0; c < chunks; c += 4, ++u) acc[u] += part[(long long)c * n + ii];
  red[w][o] = (acc[0] + acc[1]) + (acc[2] + acc[3]);
  __syncthreads();
  if (w == 0 && i < n) gw[i] = (red[0][o] + red[1][o]) + (red[2][o] + red[3][o]);
}

// Weights rearranged for the contraction, zero-padded: wt[kd][nd][tap] of
// [KDp][NDp][TP] with w[s][c][tap] at (kd, nd) = (c, s) forward, (s, c) for dL/dX.
__global__ void k_full_weights(const float *__restrict__ w, float *__restrict__ wt, int S, int C, int T, int TP,
                               int gx, int KDp, int NDp) {
  const int KD = gx ? S : C, ND = gx ? C : S;
  const long long n = (long long)KDp * NDp * TP;
  for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (long long)gridDim.x * blockDim.x) {
    const int tap = (int)(i % TP);
    const long long r = i / TP;
    const int nd = (int)(r % NDp), kd = (int)(r / NDp);
    float v = 0.f;
    if (kd < KD && nd < ND && tap < T) {
      const int s_ = gx ? kd : nd, c_ = gx ? nd : kd;
      v = w[((long long)s_ * C + c_) * T + tap];
    }
    wt[i] = v;
  }
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
template <class F>
static bool dispatch_nk(int nk, F &&f) {
  switch (nk) {
    case 1: f(std::integral_constant<int, 1>{}); return true;
    case 2: f(std::integral_constant<int, 2>{}); return true;
    case 3: f(std::integral_constant<int, 3>{}); return true;
    case 4: f(std::integral_constant<int, 4>{}); return true;
    case 5: f(std::integral_constant<int, 5>{}); return true;
    default: return false;
  }
}

bool full_kernel_size_supported(int nk) { return nk >= 1 && nk <= 5; }

bool full_launch_fits(int B, int Cin, int Cout, int P, int nk) {
  if (P % 8 != 0 || B < 1 || B > 65535 * 16) return false;
  const long long nrun = (long long)P * (P / 2) / 4 + P / 4;
  const long long nwg_run = (nrun + 3) / 4, nbt = (B + 15) / 16;
  const long long lim = 1LL << 31;
  // the two contractions
  if (nwg_run * ((Cout + kCtOut - 1) / kCtOut) * nbt >= lim) return false;
  if (nwg_run * ((Cin + kCtOut - 1) / kCtOut) * nbt >= lim) return false;
  // dL/dw: tiles of 32 x 32 (s, c) times bin chunks, and the fixed-order reduction
  const long long tiles = (long long)((Cout + 31) / 32) * ((Cin + 31) / 32);
  if (tiles * full_gw_chunks(B, Cout, Cin, P, nk) >= lim) return false;
  if (((long long)Cout * Cin * nk * nk + 63) / 64 >= lim) return false;
  return true;
}

static int round_up(int v, int m) { return (v + m - 1) / m * m; }
static int tap_pad_rt(int nk) { return (nk * nk + 3) & ~3; }

size_t full_weight_floats(int KD, int ND, int nk) {
  return (size_t)round_up(KD, 4) * round_up(ND, kCtOut) * tap_pad_rt(nk);
}

hipError_t launch_full_weights(const float *w, float *wt, bool gx, int S, int C, int nk, hipStream_t s) {
  const int KDp = round_up(gx ? S : C, 4), NDp = round_up(gx ? C : S, kCtOut), TP = tap_pad_rt(nk);
  const long long n = (long long)KDp * NDp * TP;
  long long g = (n + 255) / 256;
  if (g > 65536) g = 65536;
  return timed_launch("full_weights", k_full_weights, dim3((unsigned)g), dim3(256), 0, s, w, wt, S, C, nk * nk, TP,
                      gx ? 1 : 0, KDp, NDp);
}

hipError_t launch_full_contract(bool gx, int nk, SpecLayout in, const float *wt, const float2 *tw, SpecLayout out,
                                int B, int KD, int ND, int P, hipStream_t s) {
  const int nrun = P * (P / 2) / 4 + P / 4;
  const int nwg_run = (nrun + 3) / 4, nsb = (ND + kCtOut - 1) / kCtOut, nbt = (B + 15) / 16;
  const long long blocks = (long long)nwg_run * nsb * nbt;
  if (blocks >= (1LL << 31) || P % 8 != 0) return hipErrorInvalidValue;
  const int KDp = round_up(KD, 4), NDp = round_up(ND, kCtOut);
  hipError_t err = hipErrorInvalidValue;
  dispatch_nk(nk, [&](auto nc) {
    constexpr int NK = decltype(nc)::value;
    const char *nm = gx ? "full_contract_gx" : "full_contract_fwd";
    if (gx)
      err = timed_launch(nm, k_full_contract<NK, true>, dim3((unsigned)blocks), dim3(256), 0, s, in, wt, tw, out, B,
                         KD, KDp, ND, NDp, P, nwg_run, nsb);
    else
      err = timed_launch(nm, k_full_contract<NK, false>, dim3((unsigned)blocks), dim3(256), 0, s, in, wt, tw, out, B,
                         KD, KDp, ND, NDp, P, nwg_run, nsb);
  });
  return err;
}

// Bin chunks of the dL/dw pass: about 8192 workgroups, so that the workgroups running
// at one time on an XCD are the tiles of one or two short chunks and share the spectra
// they read through L2, and at most 97 runs (388 bins) per chunk; at most 512 chunks of
// partial sums.  At 512 pixels and 256 channels (64 tiles) the pass took 13.3-13.8 ms
// with 97 or 129 runs per chunk, 15.1 ms with 65, 17-22 ms with 128 (two whole rows:
// every chunk starts at the same column), 22-24 ms with 161 or 193, and 15-19 ms, uneven
// from run to run and with 2.3 times the HBM reads, with the 257 that 8192 workgroups
// alone give.
constexpr int kGwMaxRunsPerChunk = 97;
int full_gw_chunks(int B, int S, int C, int P, int nk) {
  (void)B, (void)nk;
  const int nrun = P * (P / 2) / 4 + P / 4;
  const int tiles = ((S + 31) / 32) * ((C + 31) / 32);
  int chunks = std::max((8192 + tiles - 1) / tiles, (nrun + kGwMaxRunsPerChunk - 1) / kGwMaxRunsPerChunk);
  if (chunks > 512) chunks = 512;
  if (chunks > nrun) chunks = nrun;
  if (chunks < 1) chunks = 1;
  return chunks;
}

hipError_t launch_full_gw(int nk, SpecLayout G, SpecLayout X, const float2 *tw, float *part, float *gw, int B, int S,
                          int C, int P, hipStream_t s) {
  if (P % 8 != 0) return hipErrorInvalidValue;
  const int nrun = P * (P / 2) / 4 + P / 4;
  const int chunks = full_gw_chunks(B, S, C, P, nk);
  const int runs_per_chunk = (nrun + chunks - 1) / chunks;
  const int tiles = ((S + 31) / 32) * ((C + 31) / 32);
  hipError_t err = hipErrorInvalidValue;
  dispatch_nk(nk, [&](auto nc) {
    constexpr int NK = decltype(nc)::value;
    const size_t lds = ((size_t)gw_tw_elems<NK>(P) + 2 * kGwStageElems) * sizeof(float2);
    if (lds > 65536) return;  // (P <= 1024, n <= 5 stays within 60 KB)
    if (((B + 3) / 4) % 2 == 0)
      err = timed_launch("full_gw", k_full_gw<NK, true>, dim3((unsigned)(tiles * chunks)), dim3(256), lds, s, G, X, tw,
                         part, B, S, C, P, runs_per_chunk);
    else
      err = timed_launch("full_gw", k_full_gw<NK, false>, dim3((unsigned)(tiles * chunks)), dim3(256), lds, s, G, X,
                         tw, part, B, S, C, P, runs_per_chunk);
  });
  if (err != hipSuccess) return err;
  const long long n = (long long)S * C * nk * nk;
  const long long g = (n + 63) / 64;
  if (g >= (1LL << 31)) return hipErrorInvalidValue;
  return timed_launch("full_gw_reduce", k_full_gw_reduce, dim3((unsigned)g), dim3(256), 0, s, part, gw, n, chunks);
}

}  // namespace fdc
