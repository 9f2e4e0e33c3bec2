// The last two layers of a CIC + FDP stack with every intermediate in LDS.
//
// Once a layer's input is at most 128 x 128, one input plane's pruned row spectrum
// (N x (M/2+1) complex values) and everything derived from it down to the stack's
// output fit in the 160 KB of LDS of one compute unit.  k_tail_fwd then runs, for
// one input plane (b, c) of layer a (N_a -> M_a) and the J_a * J_b output planes of
// layer b (M_a -> M_b) that depend on it, every step of both layers (section 2.4.1,
// Eq. 5 and the FDP of section 2.4.2) in one workgroup:
//
//   A  rows:    layer a's input rows: the inverse row transform of the previous
//               layer's column-inverted spectrum and the forward row transform of the
//               same rows, keeping M_a/2+1 bins (or, for the stack's first layer, the
//               forward row transform of the input image)
//   B  columns: column DFT (N_a), keep the M_a rows FDP keeps: the saved spectrum
//   C  columns: for each of the J_a output channels o: CIC product with K_a[o] at the
//               kept bins (Eq. 5), inverse column DFT (M_a)
//   D  rows:    inverse row transform of layer a's output (M_a) and the forward row
//               transform of layer b's input, keeping M_b/2+1 bins
//   E, F        layer b's columns, as B and C
//   G  rows:    inverse row transform (M_b) with real-part semantics: the output
//
// k_tail_bwd runs the backward of both layers for one input plane (b, c) of layer a:
// the irfft2 adjoint of the J_a * J_b upstream gradients, their column DFTs, the dK
// products of this image (written to a partial-sum buffer; k_gk_reduce adds the
// images in order), the dX products summed over each layer's fan-out, the FDP
// adjoint and inverse column DFTs, and the row transforms between the layers; its
// output is layer a's upstream-gradient row spectrum for the previous layer's
// column kernels (or the gradient of the stack's input image).
//
// Only HBM traffic left: the input row spectrum (or image), the kernels at the kept
// bins, the saved spectra, the output (and, backward, the per-image dK products).
// Column transforms run in place in their LDS plane; a sequence never spans two
// wavefronts, so every exchange needs only wave-level ordering, and stages are
// separated by workgroup barriers.
#include "device.h"
#include "fft.h"
#include "internal.h"

#include <hip/hip_runtime.h>

#include <string>

namespace fdc {

extern __shared__ float2 t_lds[];

namespace tail {

// Every transform of the tail uses the column plans: E = 8 elements per thread.
template <int N>
using Plan = ColCfg<N>;

// LDS planes: `rows` rows of ld complex values, ld > L (spare columns give idle
// lanes somewhere harmless to exchange through) and odd (a column walked by
// consecutive rows spreads over the banks).
__host__ __device__ constexpr int plane_ld(int L) { return (L % 2 == 1) ? L + 2 : L + 1; }

template <int N, int M>
__device__ __forceinline__ int kept(int mrow) {
  return mrow < M / 2 ? mrow : mrow + (N - M);
}

__device__ __forceinline__ float weight(int l, int n, float alpha, float beta) {
  return (l == 0 || 2 * l == n) ? alpha : alpha * beta;
}

// Bin (plane, row, l) of a spectrum (SpecLayout) in HBM.
__device__ __forceinline__ float2 *spec_at(const SpecLayout &s, long long plane, int row, int l, int L) {
  return l < L - 1 ? s.main + plane * s.ps + (long long)row * s.rs + bin_off(s, l)
                   : s.side + plane * s.sps + (long long)row * s.srs;
}

// Lane roles.  Row passes: t fastest (a wave reads whole rows).  Column passes:
// the W = 64 / TPS columns of a wave fastest (a wave's global accesses are runs of
// W consecutive bins of a row).
template <int N>
struct RowLanes {
  static constexpr int TPS = Plan<N>::TPS, W = 64 / TPS;
  int t, s, first;
  __device__ RowLanes() {
    const int lane = threadIdx.x & 63;
    t = lane % TPS;
    s = lane / TPS;
    first = (threadIdx.x >> 6) * W;
  }
};
template <int N>
struct ColLanes {
  static constexpr int TPS = Plan<N>::TPS, W = 64 / TPS;
  int t, s, first;
  __device__ ColLanes() {
    const int lane = threadIdx.x & 63;
    s = lane % W;
    t = lane / W;
    first = (threadIdx.x >> 6) * W;
  }
};

// ----------------------------------------------------------------------------
// row passes (pairs of real rows packed as one complex sequence z = a + i b)
// ----------------------------------------------------------------------------
// Packed inverse input of rows (r, r + 1): v[m] = A_k + i B_k at k = t + TPS m, the
// Hermitian extensions of the two rows' first LIN bins weighted by c-weights (a1 at
// l = 0 and N/2, a1 b1 elsewhere), with real-part semantics at l = 0 and N/2.
template <int N, int LIN, class Bin>
__device__ __forceinline__ void c2r_in(float2 (&v)[Plan<N>::E], Bin bin, int t, float a1, float b1) {
  constexpr int TPS = Plan<N>::TPS, E = Plan<N>::E;
#pragma unroll
  for (int m = 0; m < E; ++m) {
    const int k = t + TPS * m;
    const bool upper = 2 * k > N;
    const int kk = upper ? N - k : k;
    const bool in = kk < LIN;
    float2 a = bin(0, in ? kk : 0), b = bin(1, in ? kk : 0);
    const bool edge = kk == 0 || 2 * kk == N;
    const float w = in ? (edge ? a1 : a1 * b1) : 0.f;
    a = cscale(a, w);
    b = cscale(b, w);
    if (edge) a.y = b.y = 0.f;
    if (upper) a.y = -a.y, b.y = -b.y;
    v[m] = make_float2(a.x - b.y, a.y + b.x);
  }
}

// Forward transform output of a packed pair (held in registers, comb order) ->
// the two rows' weighted bins k < LOUT: emit(row 0 or 1, k, value).
template <int N, int LOUT, class Emit>
__device__ __forceinline__ void r2c_out(const float2 (&v)[Plan<N>::E], float2 *scr, int sq, int t, float a2,
                                        float b2, Emit emit) {
  constexpr int TPS = Plan<N>::TPS, E = Plan<N>::E;
  lds_barrier<true>();
#pragma unroll
  for (int m = 0; m < E; ++m) scr[lds_phys<kLdsPad>(sq * N + t + TPS * m)] = v[m];
  lds_barrier<true>();
  for (int k = t; k < LOUT; k += TPS) {
    const float2 zk = scr[lds_phys<kLdsPad>(sq * N + k)];
    const float2 zn = scr[lds_phys<kLdsPad>(sq * N + (k == 0 ? 0 : N - k))];
    const float w = 0.5f * weight(k, N, a2, b2);
    emit(0, k, make_float2((zk.x + zn.x) * w, (zk.y - zn.y) * w));
    emit(1, k, make_float2((zk.y + zn.y) * w, (zn.x - zk.x) * w));
  }
}

// ----------------------------------------------------------------------------
// column passes (in place in an LDS plane)
// ----------------------------------------------------------------------------
// For every item (plane q < nq, column l < L): load(v, q, l, t, act) fills the
// column, the N-point transform (direction DIR) runs through column l of plane(q),
// store(v, q, l, t, act) takes the result.  Idle lanes (act = false) work on the
// spare column L of plane 0 and must not store.
template <int N, int DIR, int NT, class Load, class PlaneOf, class Store>
__device__ __forceinline__ void col_pass(int nq, int L, const float2 *tw, int tws, Load load, PlaneOf plane,
                                         Store store) {
  using C = Plan<N>;
  constexpr int SEQ = NT / C::TPS;
  const ColLanes<N> ln;
  const int items = nq * L;
  for (int r0 = 0; r0 + ln.first < items; r0 += SEQ) {
    const int it = r0 + ln.first + ln.s;
    const bool act = it < items;
    const int q = act ? it / L : 0, l = act ? it - (it / L) * L : L;
    float2 v[C::E];
    load(v, q, l, ln.t, act);
    fft_seq<N, DIR, true, true, kLdsPlain, C>(v, ln.t, plane(q), l, plane_ld(L), tw, tws);
    store(v, q, l, ln.t, act);
  }
}

}  // namespace tail

using namespace tail;

// Sizes of the LDS layout of the two tail kernels (complex values).
template <int NA, int MA, int MB, int JA, int JB>
struct TailGeom {
  static constexpr int LP = NA / 2 + 1;  // bins of the previous layer's output rows
  static constexpr int LA = MA / 2 + 1, LB = MB / 2 + 1;
  static constexpr int ldA = plane_ld(LA), ldB = plane_ld(LB);
  static constexpr int TW = twiddle_lds_elems<NA>();
  // forward: TA [NA][ldA], XA [MA][ldA], UA[JA] [MA][ldA], TB[JA] [MA][ldB],
  // XB[JA] [MB][ldB], UB[JA JB] [MB][ldB]
  static constexpr int fTA = TW, fXA = fTA + NA * ldA, fUA = fXA + MA * ldA, fTB = fUA + JA * MA * ldA,
                       fXB = fTB + JA * MA * ldB, fUB = fXB + JA * MB * ldB, fEnd = fUB + JA * JB * MB * ldB;
  // backward: GB[JA JB] [MB][ldB], VB[JA] [MA][ldB], GA[JA] [MA][ldA], VA [NA][ldA]
  static constexpr int bGB = TW, bVB = bGB + JA * JB * MB * ldB, bGA = bVB + JA * MA * ldB,
                       bVA = bGA + JA * MA * ldA, bEnd = bVA + NA * ldA;
};

// Scratch of a row pass of `items` pairs of N-point rows with NT threads (padded
// layout): one N-point sequence per slot, slots of whole waves up to NT / TPS.
template <int N, int NT>
__host__ __device__ constexpr int row_scratch(int items) {
  constexpr int TPS = Plan<N>::TPS, W = 64 / TPS, SEQ = NT / TPS;
  const int used = (items + W - 1) / W * W;
  return lds_size<kLdsPad>((used < SEQ ? used : SEQ) * N);
}

// ----------------------------------------------------------------------------
// forward
// ----------------------------------------------------------------------------
// One workgroup per input plane (b, c) of layer a and group of JL of its JA output
// channels (JL = JA, or fewer when the input planes alone would leave compute units
// idle: each group then repeats stages A and B, and group 0 stores saved_a); workgroup
// w after the XCD remap takes b = w % B, then the group, then c (the B images of one
// channel group read the same kernels).
//   FIRST = false: in = previous layer's column-inverted spectra, split layout
//                  [B * C][NA rows][NA/2+1], inverse row weights a_in (= 1 / NA^2).
//   FIRST = true:  x = input images [B][C][NA][NA].
//   saved_a: split [B * C][MA][LA]; saved_b: split [B * S_a][MB][LB];
//   Ka [S_a][NA][NA/2+1], Kb [S_b][MA][MA/2+1]; y [B][S_b][MB][MB].
template <int NA, int MA, int MB, int JA, int JB, int NT, bool FIRST, int JL>
__global__ __launch_bounds__(NT) void k_tail_fwd(SpecLayout in, const float *__restrict__ x, float a_in,
                                                 const float2 *__restrict__ Ka, const float2 *__restrict__ Kb,
                                                 SpecLayout saved_a, SpecLayout saved_b, float *__restrict__ y, int B,
                                                 int C) {
  static_assert(JA % JL == 0, "channel groups of equal size");
  using G = TailGeom<NA, MA, MB, JL, JB>;
  constexpr int LA = G::LA, LB = G::LB, ldA = G::ldA, ldB = G::ldB;
  constexpr int NFA = NA / 2 + 1, NFB = MA / 2 + 1, JG = JA / JL;
  float2 *tw = t_lds;
  stage_twiddles<NA>(tw, threadIdx.x, NT);
  const int wg = xcd_remap(blockIdx.x, gridDim.x);
  const int b = wg % B, cg = wg / B;
  const int c = cg / JG, j0 = (cg - c * JG) * JL;  // this group's first layer-a output of channel c
  const int Sa = C * JA, Sb = Sa * JB;
  float2 *TA = t_lds + G::fTA, *XA = t_lds + G::fXA, *UA = t_lds + G::fUA, *TB = t_lds + G::fTB,
         *XB = t_lds + G::fXB, *UB = t_lds + G::fUB;

  // The kernel bins of stages C and F, loaded now (when each stage is one round of its
  // column pass, so that this thread's item is known): their loads complete with
  // stage A's, instead of each stage waiting for its own.
  constexpr bool PC = JL * LA <= NT / Plan<MA>::TPS, PF = JL * JB * LB <= NT / Plan<MB>::TPS;
  float2 kpa[Plan<MA>::E], kpb[Plan<MB>::E];
  if constexpr (PC) {
    const ColLanes<MA> ln;
    const int it = ln.first + ln.s;
    const bool act = it < JL * LA;
    const int j = act ? it / LA : 0, lc = act ? it - (it / LA) * LA : 0;
    const float2 *kc = Ka + (long long)(c * JA + j0 + j) * NA * NFA + lc;
#pragma unroll
    for (int m = 0; m < Plan<MA>::E; ++m) kpa[m] = kc[(long long)kept<NA, MA>(ln.t + Plan<MA>::TPS * m) * NFA];
  }
  if constexpr (PF) {
    const ColLanes<MB> ln;
    const int it = ln.first + ln.s;
    const bool act = it < JL * JB * LB;
    const int q = act ? it / LB : 0, lc = act ? it - (it / LB) * LB : 0;
    const float2 *kc = Kb + (long long)((c * JA + j0) * JB + q) * MA * NFB + lc;
#pragma unroll
    for (int m = 0; m < Plan<MB>::E; ++m) kpb[m] = kc[(long long)kept<MA, MB>(ln.t + Plan<MB>::TPS * m) * NFB];
  }

  // A: layer a's input rows -> TA [NA][LA]
  {
    float2 *scr = UA;  // UA and the planes after it are not in use yet (tail_fwd_lds covers the scratch)
    constexpr int TPS = Plan<NA>::TPS, SEQ = NT / TPS;
    const RowLanes<NA> ln;
    const long long plane = (long long)b * C + c;
    for (int r0 = 0; r0 + ln.first < NA / 2; r0 += SEQ) {
      const int p = r0 + ln.first + ln.s;
      const bool act = p < NA / 2;
      const int r = 2 * (act ? p : 0);
      float2 v[Plan<NA>::E];
      if constexpr (FIRST) {
        const float *xr = x + plane * NA * NA + (long long)r * NA;
#pragma unroll
        for (int m = 0; m < Plan<NA>::E; ++m) v[m] = make_float2(xr[ln.t + TPS * m], xr[NA + ln.t + TPS * m]);
      } else {
        c2r_in<NA, NFA>(v, [&](int rr, int k) { return *spec_at(in, plane, r + rr, k, NFA); }, ln.t, a_in, 1.f);
        fft_seq<NA, +1, true, true, kLdsPad, Plan<NA>>(v, ln.t, scr, (ln.first + ln.s) * NA, 1, tw, 1);
      }
      fft_seq<NA, -1, true, true, kLdsPad, Plan<NA>>(v, ln.t, scr, (ln.first + ln.s) * NA, 1, tw, 1);
      r2c_out<NA, LA>(v, scr, ln.first + ln.s, ln.t, 1.f, 1.f, [&](int rr, int k, float2 val) {
        if (act) TA[(r + rr) * ldA + k] = val;
      });
    }
  }
  __syncthreads();
  // B: column DFT (NA) of TA, keep MA rows -> XA and saved_a
  {
    const long long plane = (long long)b * C + c;
    col_pass<NA, -1, NT>(
        1, LA, tw, 1,
        [&](float2 (&v)[Plan<NA>::E], int, int l, int t, bool) {
#pragma unroll
          for (int m = 0; m < Plan<NA>::E; ++m) v[m] = TA[(t + Plan<NA>::TPS * m) * ldA + l];
        },
        [&](int) { return TA; },
        [&](const float2 (&v)[Plan<NA>::E], int, int l, int t, bool act) {
          if (!act) return;
#pragma unroll
          for (int m = 0; m < Plan<NA>::E; ++m) {
            const int k = t + Plan<NA>::TPS * m;
            if (k < MA / 2 || k >= NA - MA / 2) {
              const int mrow = k < MA / 2 ? k : k - (NA - MA);
              XA[mrow * ldA + l] = v[m];
              if (JG == 1 || j0 == 0) *spec_at(saved_a, plane, mrow, l, LA) = v[m];
            }
          }
        });
  }
  __syncthreads();
  // C: CIC product with K_a[c JA + j0 + j] (Eq. 5) and inverse column DFT (MA) -> UA[j]
  col_pass<MA, +1, NT>(
      JL, LA, tw, NA / MA,
      [&](float2 (&v)[Plan<MA>::E], int j, int l, int t, bool act) {
        const int lc = act ? l : 0;
        const float2 *kc = Ka + (long long)(c * JA + j0 + j) * NA * NFA + lc;
#pragma unroll
        for (int m = 0; m < Plan<MA>::E; ++m) {
          const int mrow = t + Plan<MA>::TPS * m;
          v[m] = cmul(XA[mrow * ldA + l], PC ? kpa[m] : kc[(long long)kept<NA, MA>(mrow) * NFA]);
        }
      },
      [&](int j) { return UA + j * MA * ldA; },
      [&](const float2 (&v)[Plan<MA>::E], int j, int l, int t, bool act) {
        if (!act) return;
#pragma unroll
        for (int m = 0; m < Plan<MA>::E; ++m) UA[j * MA * ldA + (t + Plan<MA>::TPS * m) * ldA + l] = v[m];
      });
  __syncthreads();
  // D: inverse rows of UA[j] (1/MA^2) and forward rows of layer b's input -> TB[j] [MA][LB]
  {
    float2 *scr = TA;  // TA is no longer needed
    constexpr int TPS = Plan<MA>::TPS, SEQ = NT / TPS, P = MA / 2;
    const RowLanes<MA> ln;
    const float inv = 1.f / ((float)MA * (float)MA);
    for (int r0 = 0; r0 + ln.first < JL * P; r0 += SEQ) {
      const int it = r0 + ln.first + ln.s;
      const bool act = it < JL * P;
      const int j = act ? it / P : 0, r = 2 * (act ? it % P : 0);
      const float2 *u = UA + j * MA * ldA + r * ldA;
      float2 v[Plan<MA>::E];
      c2r_in<MA, LA>(v, [&](int rr, int k) { return u[rr * ldA + k]; }, ln.t, inv, 1.f);
      fft_seq<MA, +1, true, true, kLdsPad, Plan<MA>>(v, ln.t, scr, (ln.first + ln.s) * MA, 1, tw, NA / MA);
      fft_seq<MA, -1, true, true, kLdsPad, Plan<MA>>(v, ln.t, scr, (ln.first + ln.s) * MA, 1, tw, NA / MA);
      float2 *tb = TB + j * MA * ldB + r * ldB;
      r2c_out<MA, LB>(v, scr, ln.first + ln.s, ln.t, 1.f, 1.f, [&](int rr, int k, float2 val) {
        if (act) tb[rr * ldB + k] = val;
      });
    }
  }
  __syncthreads();
  // E: column DFT (MA) of TB[j], keep MB rows -> XB[j] and saved_b
  col_pass<MA, -1, NT>(
      JL, LB, tw, NA / MA,
      [&](float2 (&v)[Plan<MA>::E], int j, int l, int t, bool) {
#pragma unroll
        for (int m = 0; m < Plan<MA>::E; ++m) v[m] = TB[j * MA * ldB + (t + Plan<MA>::TPS * m) * ldB + l];
      },
      [&](int j) { return TB + j * MA * ldB; },
      [&](const float2 (&v)[Plan<MA>::E], int j, int l, int t, bool act) {
        if (!act) return;
        const long long plane = (long long)b * Sa + c * JA + j0 + j;
#pragma unroll
        for (int m = 0; m < Plan<MA>::E; ++m) {
          const int k = t + Plan<MA>::TPS * m;
          if (k < MB / 2 || k >= MA - MB / 2) {
            const int mrow = k < MB / 2 ? k : k - (MA - MB);
            XB[j * MB * ldB + mrow * ldB + l] = v[m];
            *spec_at(saved_b, plane, mrow, l, LB) = v[m];
          }
        }
      });
  __syncthreads();
  // F: CIC product with K_b[(c JA + j0 + j) JB + i] and inverse column DFT (MB) -> UB[j JB + i]
  col_pass<MB, +1, NT>(
      JL * JB, LB, tw, NA / MB,
      [&](float2 (&v)[Plan<MB>::E], int q, int l, int t, bool act) {
        const int j = q / JB, lc = act ? l : 0;
        const float2 *kc = Kb + (long long)((c * JA + j0) * JB + q) * MA * NFB + lc;
#pragma unroll
        for (int m = 0; m < Plan<MB>::E; ++m) {
          const int mrow = t + Plan<MB>::TPS * m;
          v[m] = cmul(XB[j * MB * ldB + mrow * ldB + l], PF ? kpb[m] : kc[(long long)kept<MA, MB>(mrow) * NFB]);
        }
      },
      [&](int q) { return UB + q * MB * ldB; },
      [&](const float2 (&v)[Plan<MB>::E], int q, int l, int t, bool act) {
        if (!act) return;
#pragma unroll
        for (int m = 0; m < Plan<MB>::E; ++m) UB[q * MB * ldB + (t + Plan<MB>::TPS * m) * ldB + l] = v[m];
      });
  __syncthreads();
  // G: inverse rows of UB[q] (1/MB^2) -> y [b][(c JA + j0) JB + q]
  {
    float2 *scr = TA;
    constexpr int TPS = Plan<MB>::TPS, SEQ = NT / TPS, P = MB / 2;
    const RowLanes<MB> ln;
    const float inv = 1.f / ((float)MB * (float)MB);
    for (int r0 = 0; r0 + ln.first < JL * JB * P; r0 += SEQ) {
      const int it = r0 + ln.first + ln.s;
      const bool act = it < JL * JB * P;
      const int q = act ? it / P : 0, r = 2 * (act ? it % P : 0);
      const float2 *u = UB + q * MB * ldB + r * ldB;
      float2 v[Plan<MB>::E];
      c2r_in<MB, LB>(v, [&](int rr, int k) { return u[rr * ldB + k]; }, ln.t, inv, 1.f);
      fft_seq<MB, +1, true, true, kLdsPad, Plan<MB>>(v, ln.t, scr, (ln.first + ln.s) * MB, 1, tw, NA / MB);
      if (act) {
        float *yr = y + ((long long)b * Sb + (c * JA + j0) * JB + q) * MB * MB + (long long)r * MB;
#pragma unroll
        for (int m = 0; m < Plan<MB>::E; ++m) {
          yr[ln.t + TPS * m] = v[m].x;
          yr[MB + ln.t + TPS * m] = v[m].y;
        }
      }
    }
  }
}

// ----------------------------------------------------------------------------
// backward
// ----------------------------------------------------------------------------
// One workgroup per input plane (b, c) of layer a, numbered as the forward.
//   gy [B][S_b][MB][MB]; saved_a, saved_b, Ka, Kb as the forward.
//   part_a plain [B][S_a][MA][LA], part_b plain [B][S_b][MB][LB]: this image's dK
//   products at the kept bins (k_gk_reduce sums them over the images in order).
//   OUT = 0: Tg = layer a's upstream-gradient row spectrum for the previous layer,
//            split [B * C][NA rows][NA/2+1], weights (c_l / NA^2) (a_out = 1/NA^2);
//   OUT = 1: gx [B][C][NA][NA], the gradient of the stack's input;
//   OUT = 2: no input-side output (the stack's first layer without input gradient).
template <int NA, int MA, int MB, int JA, int JB, int NT, int OUT>
__global__ __launch_bounds__(NT) void k_tail_bwd(const float *__restrict__ gy, SpecLayout saved_a, SpecLayout saved_b,
                                                 const float2 *__restrict__ Ka, const float2 *__restrict__ Kb,
                                                 float2 *__restrict__ part_a, float2 *__restrict__ part_b,
                                                 SpecLayout Tg, float a_out, float *__restrict__ gx, int B, int C) {
  using G = TailGeom<NA, MA, MB, JA, JB>;
  constexpr int LA = G::LA, LB = G::LB, ldA = G::ldA, ldB = G::ldB;
  constexpr int NFA = NA / 2 + 1, NFB = MA / 2 + 1;
  float2 *tw = t_lds;
  stage_twiddles<NA>(tw, threadIdx.x, NT);
  const int wg = xcd_remap(blockIdx.x, gridDim.x);
  const int c = wg / B, b = wg - (wg / B) * B;
  const int Sa = C * JA, Sb = Sa * JB;
  float2 *GB = t_lds + G::bGB, *VB = t_lds + G::bVB, *GA = t_lds + G::bGA, *VA = t_lds + G::bVA;

  // The saved-spectrum and kernel bins of stage S5, loaded now (when the stage is one
  // round of its column pass, so that this thread's item is known): their loads complete
  // with stage S1's, instead of the stage waiting for them after its transform.  (The
  // same for stage S2 as well takes 128 VGPRs and spills: no faster.)
  constexpr bool P5 = JA * LA <= NT / Plan<MA>::TPS;
  float2 xp5[Plan<MA>::E], kp5[Plan<MA>::E];
  if constexpr (P5) {
    const ColLanes<MA> ln;
    const int it = ln.first + ln.s;
    const bool act = it < JA * LA;
    const int j = act ? it / LA : 0, lc = act ? it - (it / LA) * LA : 0;
    const long long xplane = (long long)b * C + c;
    const float2 *kc = Ka + (long long)(c * JA + j) * NA * NFA + lc;
#pragma unroll
    for (int m = 0; m < Plan<MA>::E; ++m) {
      const int row = ln.t + Plan<MA>::TPS * m;
      xp5[m] = *spec_at(saved_a, xplane, row, lc, LA);
      kp5[m] = kc[(long long)kept<NA, MA>(row) * NFA];
    }
  }

  // S1: rows of the JA JB upstream gradients: (c_l / MB^2) rfft -> GB[q] [MB][LB]
  {
    float2 *scr = VB;  // VB, GA are not in use yet
    constexpr int TPS = Plan<MB>::TPS, SEQ = NT / TPS, P = MB / 2;
    const RowLanes<MB> ln;
    const float inv = 1.f / ((float)MB * (float)MB);
    for (int r0 = 0; r0 + ln.first < JA * JB * P; r0 += SEQ) {
      const int it = r0 + ln.first + ln.s;
      const bool act = it < JA * JB * P;
      const int q = act ? it / P : 0, r = 2 * (act ? it % P : 0);
      const float *gr = gy + ((long long)b * Sb + c * JA * JB + q) * MB * MB + (long long)r * MB;
      float2 v[Plan<MB>::E];
#pragma unroll
      for (int m = 0; m < Plan<MB>::E; ++m) v[m] = make_float2(gr[ln.t + TPS * m], gr[MB + ln.t + TPS * m]);
      fft_seq<MB, -1, true, true, kLdsPad, Plan<MB>>(v, ln.t, scr, (ln.first + ln.s) * MB, 1, tw, NA / MB);
      float2 *g = GB + q * MB * ldB + r * ldB;
      r2c_out<MB, LB>(v, scr, ln.first + ln.s, ln.t, inv, 2.f, [&](int rr, int k, float2 val) {
        if (act) g[rr * ldB + k] = val;
      });
    }
  }
  __syncthreads();
  // S2: column DFT (MB) of GB[q]; dK_b product with saved_b -> part_b; GB[q] <- G conj(K_b)
  col_pass<MB, -1, NT>(
      JA * JB, LB, tw, NA / MB,
      [&](float2 (&v)[Plan<MB>::E], int q, int l, int t, bool) {
#pragma unroll
        for (int m = 0; m < Plan<MB>::E; ++m) v[m] = GB[q * MB * ldB + (t + Plan<MB>::TPS * m) * ldB + l];
      },
      [&](int q) { return GB + q * MB * ldB; },
      [&](const float2 (&v)[Plan<MB>::E], int q, int l, int t, bool act) {
        const int lc = act ? l : 0;
        const int oa = c * JA + q / JB, ob = c * JA * JB + q;
        const long long xplane = (long long)b * Sa + oa;
        const float2 *kc = Kb + (long long)ob * MA * NFB + lc;
        float2 *pp = part_b + (((long long)b * Sb + ob) * MB) * LB + lc;
#pragma unroll
        for (int m = 0; m < Plan<MB>::E; ++m) {
          const int row = t + Plan<MB>::TPS * m;
          const float2 xv = *spec_at(saved_b, xplane, row, lc, LB);
          const float2 kv = kc[(long long)kept<MA, MB>(row) * NFB];
          if (act) {
            pp[(long long)row * LB] = cmulc(v[m], xv);
            GB[q * MB * ldB + row * ldB + l] = cmulc(v[m], kv);
          }
        }
      });
  __syncthreads();
  // S3: sum over layer b's fan-out, FDP adjoint (zero rows), inverse column DFT (MA) -> VB[j]
  col_pass<MA, +1, NT>(
      JA, LB, tw, NA / MA,
      [&](float2 (&v)[Plan<MA>::E], int j, int l, int t, bool) {
#pragma unroll
        for (int m = 0; m < Plan<MA>::E; ++m) {
          const int k = t + Plan<MA>::TPS * m;
          float2 s = make_float2(0.f, 0.f);
          if (k < MB / 2 || k >= MA - MB / 2) {
            const int mrow = k < MB / 2 ? k : k - (MA - MB);
#pragma unroll
            for (int i = 0; i < JB; ++i) s = cadd(s, GB[(j * JB + i) * MB * ldB + mrow * ldB + l]);
          }
          v[m] = s;
        }
      },
      [&](int j) { return VB + j * MA * ldB; },
      [&](const float2 (&v)[Plan<MA>::E], int j, int l, int t, bool act) {
        if (!act) return;
#pragma unroll
        for (int m = 0; m < Plan<MA>::E; ++m) VB[j * MA * ldB + (t + Plan<MA>::TPS * m) * ldB + l] = v[m];
      });
  __syncthreads();
  // S4: rfft2-adjoint rows of VB[j] (weights 1, 1/2) and (c_l / MA^2) forward rows -> GA[j] [MA][LA]
  {
    float2 *scr = VA;  // VA is not in use yet
    constexpr int TPS = Plan<MA>::TPS, SEQ = NT / TPS, P = MA / 2;
    const RowLanes<MA> ln;
    const float inv = 1.f / ((float)MA * (float)MA);
    for (int r0 = 0; r0 + ln.first < JA * P; r0 += SEQ) {
      const int it = r0 + ln.first + ln.s;
      const bool act = it < JA * P;
      const int j = act ? it / P : 0, r = 2 * (act ? it % P : 0);
      const float2 *u = VB + j * MA * ldB + r * ldB;
      float2 v[Plan<MA>::E];
      c2r_in<MA, LB>(v, [&](int rr, int k) { return u[rr * ldB + k]; }, ln.t, 1.f, 0.5f);
      fft_seq<MA, +1, true, true, kLdsPad, Plan<MA>>(v, ln.t, scr, (ln.first + ln.s) * MA, 1, tw, NA / MA);
      fft_seq<MA, -1, true, true, kLdsPad, Plan<MA>>(v, ln.t, scr, (ln.first + ln.s) * MA, 1, tw, NA / MA);
      float2 *g = GA + j * MA * ldA + r * ldA;
      r2c_out<MA, LA>(v, scr, ln.first + ln.s, ln.t, inv, 2.f, [&](int rr, int k, float2 val) {
        if (act) g[rr * ldA + k] = val;
      });
    }
  }
  __syncthreads();
  // S5: column DFT (MA) of GA[j]; dK_a product with saved_a -> part_a; GA[j] <- G conj(K_a)
  col_pass<MA, -1, NT>(
      JA, LA, tw, NA / MA,
      [&](float2 (&v)[Plan<MA>::E], int j, int l, int t, bool) {
#pragma unroll
        for (int m = 0; m < Plan<MA>::E; ++m) v[m] = GA[j * MA * ldA + (t + Plan<MA>::TPS * m) * ldA + l];
      },
      [&](int j) { return GA + j * MA * ldA; },
      [&](const float2 (&v)[Plan<MA>::E], int j, int l, int t, bool act) {
        const int lc = act ? l : 0;
        const int oa = c * JA + j;
        const long long xplane = (long long)b * C + c;
        const float2 *kc = Ka + (long long)oa * NA * NFA + lc;
        float2 *pp = part_a + (((long long)b * Sa + oa) * MA) * LA + lc;
#pragma unroll
        for (int m = 0; m < Plan<MA>::E; ++m) {
          const int row = t + Plan<MA>::TPS * m;
          const float2 xv = P5 ? xp5[m] : *spec_at(saved_a, xplane, row, lc, LA);
          const float2 kv = P5 ? kp5[m] : kc[(long long)kept<NA, MA>(row) * NFA];
          if (act) {
            pp[(long long)row * LA] = cmulc(v[m], xv);
            GA[j * MA * ldA + row * ldA + l] = cmulc(v[m], kv);
          }
        }
      });
  if constexpr (OUT == 2) return;
  __syncthreads();
  // S6: sum over layer a's fan-out, FDP adjoint, inverse column DFT (NA) -> VA
  col_pass<NA, +1, NT>(
      1, LA, tw, 1,
      [&](float2 (&v)[Plan<NA>::E], int, int l, int t, bool) {
#pragma unroll
        for (int m = 0; m < Plan<NA>::E; ++m) {
          const int k = t + Plan<NA>::TPS * m;
          float2 s = make_float2(0.f, 0.f);
          if (k < MA / 2 || k >= NA - MA / 2) {
            const int mrow = k < MA / 2 ? k : k - (NA - MA);
#pragma unroll
            for (int j = 0; j < JA; ++j) s = cadd(s, GA[j * MA * ldA + mrow * ldA + l]);
          }
          v[m] = s;
        }
      },
      [&](int) { return VA; },
      [&](const float2 (&v)[Plan<NA>::E], int, int l, int t, bool act) {
        if (!act) return;
#pragma unroll
        for (int m = 0; m < Plan<NA>::E; ++m) VA[(t + Plan<NA>::TPS * m) * ldA + l] = v[m];
      });
  __syncthreads();
  // S7: rfft2-adjoint rows of VA (weights 1, 1/2), then either the previous layer's
  // (c_l / NA^2) forward rows -> Tg, or the input gradient rows -> gx
  {
    float2 *scr = GB;  // GB, VB, GA are no longer needed
    constexpr int TPS = Plan<NA>::TPS, SEQ = NT / TPS;
    const RowLanes<NA> ln;
    const long long plane = (long long)b * C + c;
    for (int r0 = 0; r0 + ln.first < NA / 2; r0 += SEQ) {
      const int p = r0 + ln.first + ln.s;
      const bool act = p < NA / 2;
      const int r = 2 * (act ? p : 0);
      const float2 *u = VA + r * ldA;
      float2 v[Plan<NA>::E];
      c2r_in<NA, LA>(v, [&](int rr, int k) { return u[rr * ldA + k]; }, ln.t, 1.f, 0.5f);
      fft_seq<NA, +1, true, true, kLdsPad, Plan<NA>>(v, ln.t, scr, (ln.first + ln.s) * NA, 1, tw, 1);
      if constexpr (OUT == 1) {
        if (act) {
          float *gr = gx + plane * NA * NA + (long long)r * NA;
#pragma unroll
          for (int m = 0; m < Plan<NA>::E; ++m) {
            gr[ln.t + TPS * m] = v[m].x;
            gr[NA + ln.t + TPS * m] = v[m].y;
          }
        }
      } else {
        fft_seq<NA, -1, true, true, kLdsPad, Plan<NA>>(v, ln.t, scr, (ln.first + ln.s) * NA, 1, tw, 1);
        r2c_out<NA, NFA>(v, scr, ln.first + ln.s, ln.t, a_out, 2.f, [&](int rr, int k, float2 val) {
          if (act) *spec_at(Tg, plane, r + rr, k, NFA) = val;
        });
      }
    }
  }
}

// ----------------------------------------------------------------------------
// Whole 2-D transforms of small square planes (N <= 64), P planes per workgroup:
// the row pass and the column pass of section 2.4.1.1 meet in LDS, so a transform
// is one launch.  Spectra use the plain layout [planes][N][N/2+1].
//   forward: X = rows (weights a2 at l = 0 and N/2, a2 b2 elsewhere) then columns;
//   inverse: columns, then rows with the c-weights a1 (l = 0, N/2) and a1 b1 and
//            real-part semantics, the layout and weights of the row kernels.
// ----------------------------------------------------------------------------
template <int N, int P>
struct Small2d {
  static constexpr int L = N / 2 + 1, ld = plane_ld(L), NT = 256;
  static constexpr int TW = twiddle_lds_elems<N>(), PL = TW, SCR = PL + P * N * ld;
  static constexpr int END = SCR + row_scratch<N, NT>(P * N / 2);
};

template <int N, int P>
__global__ __launch_bounds__(256) void k_fft2_small_fwd(const float *__restrict__ x, float2 *__restrict__ X,
                                                        long long count, float a2, float b2) {
  using G = Small2d<N, P>;
  constexpr int L = G::L, ld = G::ld, NT = G::NT, TPS = Plan<N>::TPS, E = Plan<N>::E;
  float2 *tw = t_lds, *pl = t_lds + G::PL, *scr = t_lds + G::SCR;
  stage_twiddles<N>(tw, threadIdx.x, NT);
  const long long q0 = (long long)xcd_remap(blockIdx.x, gridDim.x) * P;
  const int np = (int)(count - q0 < P ? count - q0 : P);
  {  // rows: pairs of real rows packed as one complex sequence -> planes [N][ld]
    constexpr int SEQ = NT / TPS, H = N / 2;
    const RowLanes<N> ln;
    for (int r0 = 0; r0 + ln.first < np * H; r0 += SEQ) {
      const int it = r0 + ln.first + ln.s;
      const bool act = it < np * H;
      const int q = act ? it / H : 0, r = 2 * (act ? it % H : 0);
      const float *xr = x + ((q0 + q) * N + r) * N;
      float2 v[E];
#pragma unroll
      for (int m = 0; m < E; ++m) v[m] = make_float2(xr[ln.t + TPS * m], xr[N + ln.t + TPS * m]);
      fft_seq<N, -1, true, true, kLdsPad, Plan<N>>(v, ln.t, scr, (ln.first + ln.s) * N, 1, tw, 1);
      float2 *dst = pl + (q * N + r) * ld;
      r2c_out<N, L>(v, scr, ln.first + ln.s, ln.t, a2, b2, [&](int rr, int k, float2 val) {
        if (act) dst[rr * ld + k] = val;
      });
    }
  }
  __syncthreads();
  col_pass<N, -1, NT>(
      np, L, tw, 1,
      [&](float2 (&v)[E], int q, int l, int t, bool) {
#pragma unroll
        for (int m = 0; m < E; ++m) v[m] = pl[(q * N + t + TPS * m) * ld + l];
      },
      [&](int q) { return pl + q * N * ld; },
      [&](const float2 (&v)[E], int q, int l, int t, bool act) {
        if (!act) return;
        float2 *o = X + (q0 + q) * N * L + l;
#pragma unroll
        for (int m = 0; m < E; ++m) o[(t + TPS * m) * L] = v[m];
      });
}

template <int N, int P>
__global__ __launch_bounds__(256) void k_fft2_small_inv(const float2 *__restrict__ X, float *__restrict__ x,
                                                        long long count, float a1, float b1) {
  using G = Small2d<N, P>;
  constexpr int L = G::L, ld = G::ld, NT = G::NT, TPS = Plan<N>::TPS, E = Plan<N>::E;
  float2 *tw = t_lds, *pl = t_lds + G::PL, *scr = t_lds + G::SCR;
  stage_twiddles<N>(tw, threadIdx.x, NT);
  const long long q0 = (long long)xcd_remap(blockIdx.x, gridDim.x) * P;
  const int np = (int)(count - q0 < P ? count - q0 : P);
  col_pass<N, +1, NT>(
      np, L, tw, 1,
      [&](float2 (&v)[E], int q, int l, int t, bool act) {
        const float2 *c = X + (q0 + q) * N * L + (act ? l : 0);  // idle lanes read a valid column
#pragma unroll
        for (int m = 0; m < E; ++m) v[m] = c[(t + TPS * m) * L];
      },
      [&](int q) { return pl + q * N * ld; },
      [&](const float2 (&v)[E], int q, int l, int t, bool act) {
        if (!act) return;
#pragma unroll
        for (int m = 0; m < E; ++m) pl[(q * N + t + TPS * m) * ld + l] = v[m];
      });
  __syncthreads();
  {  // rows: inverse of pairs of rows packed as one complex sequence -> real rows
    constexpr int SEQ = NT / TPS, H = N / 2;
    const RowLanes<N> ln;
    for (int r0 = 0; r0 + ln.first < np * H; r0 += SEQ) {
      const int it = r0 + ln.first + ln.s;
      const bool act = it < np * H;
      const int q = act ? it / H : 0, r = 2 * (act ? it % H : 0);
      const float2 *src = pl + (q * N + r) * ld;
      float2 v[E];
      c2r_in<N, L>(v, [&](int rr, int k) { return src[rr * ld + k]; }, ln.t, a1, b1);
      fft_seq<N, +1, true, true, kLdsPad, Plan<N>>(v, ln.t, scr, (ln.first + ln.s) * N, 1, tw, 1);
      if (act) {
        float *xr = x + ((q0 + q) * N + r) * N;
#pragma unroll
        for (int m = 0; m < E; ++m) xr[ln.t + TPS * m] = v[m].x, xr[N + ln.t + TPS * m] = v[m].y;
      }
    }
  }
}

// ----------------------------------------------------------------------------
// host side
// ----------------------------------------------------------------------------
#ifndef FDC_TAIL_THREADS
#define FDC_TAIL_THREADS 1024
#endif
constexpr int kTailThreads = FDC_TAIL_THREADS;

// LDS of the forward with JL layer-a output channels per workgroup.
template <int NA, int MA, int MB, int JL, int JB>
constexpr size_t tail_fwd_lds() {
  using G = TailGeom<NA, MA, MB, JL, JB>;
  constexpr int T = kTailThreads;
  // row scratch aliases: A from UA on (past the planes when they are smaller), D and G in TA
  constexpr int endA = G::fUA + row_scratch<NA, T>(NA / 2);
  static_assert(G::fTA + row_scratch<MA, T>(JL * MA / 2) <= G::fXA, "tail forward: row scratch D");
  static_assert(G::fTA + row_scratch<MB, T>(JL * JB * MB / 2) <= G::fXA, "tail forward: row scratch G");
  return (size_t)(endA > G::fEnd ? endA : G::fEnd) * sizeof(float2);
}

// Input planes below which the forward tail splits each plane's layer-a output channels
// over two workgroups, so that the launch covers the compute units (at 256^2, 16 images
// of 8 channels: 128 planes).
constexpr long long kTailSplitPlanes = 256;

template <int NA, int MA, int MB, int JA, int JB>
constexpr size_t tail_bwd_lds() {
  using G = TailGeom<NA, MA, MB, JA, JB>;
  constexpr int T = kTailThreads;
  static_assert(G::bVB + row_scratch<MB, T>(JA * JB * MB / 2) <= G::bEnd, "tail backward: row scratch S1");
  static_assert(G::bVA + row_scratch<MA, T>(JA * MA / 2) <= G::bEnd, "tail backward: row scratch S4");
  static_assert(G::bGB + row_scratch<NA, T>(NA / 2) <= G::bVA, "tail backward: row scratch S7");
  return (size_t)G::bEnd * sizeof(float2);
}

// The instantiated tails: (N_a, M_a, M_b, J_a, J_b).
template <class F>
static bool dispatch_tail(int na, int ma, int mb, int ja, int jb, F &&f) {
  if (na == 128 && ma == 64 && mb == 32 && ja == 2 && jb == 2) {
    f(std::integral_constant<int, 128>{}, std::integral_constant<int, 64>{}, std::integral_constant<int, 32>{},
      std::integral_constant<int, 2>{}, std::integral_constant<int, 2>{});
    return true;
  }
  return false;
}

bool tail_supported(int na, int ma, int mb, int ja, int jb) {
  return dispatch_tail(na, ma, mb, ja, jb, [](auto, auto, auto, auto, auto) {});
}

// Raise a kernel's dynamic LDS limit to `bytes` (once per kernel).
template <auto Kern>
static hipError_t allow_lds(size_t bytes) {
  static const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(Kern),
                                                  hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
  return e;
}

template <auto Kern, class... Args>
static hipError_t tail_launch(const char *name, unsigned grid, size_t lds, hipStream_t s, Args... args) {
  hipError_t e = allow_lds<Kern>(lds);
  if (e != hipSuccess) return e;
  const auto kern = Kern;
  return timed_launch(name, kern, dim3(grid), dim3(kTailThreads), lds, s, args...);
}

hipError_t launch_tail_fwd(int na, int ma, int mb, int ja, int jb, SpecLayout in, const float *x, float a_in,
                           const float2 *Ka, const float2 *Kb, SpecLayout saved_a, SpecLayout saved_b, float *y,
                           int B, int C, hipStream_t s) {
  hipError_t err = hipErrorInvalidValue;
  dispatch_tail(na, ma, mb, ja, jb, [&](auto nac, auto mac, auto mbc, auto jac, auto jbc) {
    constexpr int NA = decltype(nac)::value, MA = decltype(mac)::value, MB = decltype(mbc)::value;
    constexpr int JA = decltype(jac)::value, JB = decltype(jbc)::value;
    static const std::string nm =
        "tail_fwd_" + std::to_string(NA) + "_" + std::to_string(MA) + "_" + std::to_string(MB);
    const long long planes = (long long)B * C;
    auto go = [&](auto jlc) {
      constexpr int JL = decltype(jlc)::value;
      constexpr size_t lds = tail_fwd_lds<NA, MA, MB, JL, JB>();
      const unsigned grid = (unsigned)(planes * (JA / JL));
      if (x != nullptr)
        err = tail_launch<k_tail_fwd<NA, MA, MB, JA, JB, kTailThreads, true, JL>>(
            nm.c_str(), grid, lds, s, in, x, a_in, Ka, Kb, saved_a, saved_b, y, B, C);
      else
        err = tail_launch<k_tail_fwd<NA, MA, MB, JA, JB, kTailThreads, false, JL>>(
            nm.c_str(), grid, lds, s, in, x, a_in, Ka, Kb, saved_a, saved_b, y, B, C);
    };
    if constexpr (JA % 2 == 0) {
      if (planes < kTailSplitPlanes) {
        go(std::integral_constant<int, JA / 2>{});
        return;
      }
    }
    go(std::integral_constant<int, JA>{});
  });
  return err;
}

hipError_t launch_tail_bwd(int na, int ma, int mb, int ja, int jb, const float *gy, SpecLayout saved_a,
                           SpecLayout saved_b, const float2 *Ka, const float2 *Kb, float2 *part_a, float2 *part_b,
                           int out_mode, SpecLayout Tg, float a_out, float *gx, int B, int C, hipStream_t s) {
  hipError_t err = hipErrorInvalidValue;
  dispatch_tail(na, ma, mb, ja, jb, [&](auto nac, auto mac, auto mbc, auto jac, auto jbc) {
    constexpr int NA = decltype(nac)::value, MA = decltype(mac)::value, MB = decltype(mbc)::value;
    constexpr int JA = decltype(jac)::value, JB = decltype(jbc)::value;
    constexpr size_t lds = tail_bwd_lds<NA, MA, MB, JA, JB>();
    static const std::string nm =
        "tail_bwd_" + std::to_string(NA) + "_" + std::to_string(MA) + "_" + std::to_string(MB);
    const unsigned grid = (unsigned)((long long)B * C);
    auto go = [&](auto oc) {
      constexpr int OUT = decltype(oc)::value;
      err = tail_launch<k_tail_bwd<NA, MA, MB, JA, JB, kTailThreads, OUT>>(
          nm.c_str(), grid, lds, s, gy, saved_a, saved_b, Ka, Kb, part_a, part_b, Tg, a_out, gx, B, C);
    };
    switch (out_mode) {
      case 0: go(std::integral_constant<int, 0>{}); break;
      case 1: go(std::integral_constant<int, 1>{}); break;
      default: go(std::integral_constant<int, 2>{});
    }
  });
  return err;
}

// Small square 2-D transforms: N in {16, 32, 64}; P planes per workgroup, chosen so
// that a launch has at least about 512 workgroups when the batch allows it.
template <class F>
static bool dispatch_small2d(int n, long long count, F &&f) {
  auto with_p = [&](auto nc) {
    if (count >= 2048)
      f(nc, std::integral_constant<int, 4>{});
    else if (count >= 1024)
      f(nc, std::integral_constant<int, 2>{});
    else
      f(nc, std::integral_constant<int, 1>{});
  };
  switch (n) {
    case 16: with_p(std::integral_constant<int, 16>{}); return true;
    case 32: with_p(std::integral_constant<int, 32>{}); return true;
    case 64: with_p(std::integral_constant<int, 64>{}); return true;
    default: return false;
  }
}

bool fft2_small_supported(int h, int w) { return h == w && (h == 16 || h == 32 || h == 64); }

template <auto Kern, class... Args>
static hipError_t small2d_launch(const char *name, unsigned grid, size_t lds, hipStream_t s, Args... args) {
  hipError_t e = allow_lds<Kern>(lds);
  if (e != hipSuccess) return e;
  const auto kern = Kern;
  return timed_launch(name, kern, dim3(grid), dim3(256), lds, s, args...);
}

hipError_t launch_fft2_small(int n, bool inverse, const float *x, float2 *X, float *xo, const float2 *Xi,
                             long long count, float alpha, float beta, hipStream_t s) {
  hipError_t err = hipErrorInvalidValue;
  dispatch_small2d(n, count, [&](auto nc, auto pc) {
    constexpr int N = decltype(nc)::value, P = decltype(pc)::value;
    constexpr size_t lds = (size_t)Small2d<N, P>::END * sizeof(float2);
    static_assert(lds <= 160 * 1024, "small 2-D transform: LDS");
    const long long grid = (count + P - 1) / P;
    if (count < 1 || grid >= (1LL << 31)) return;
    static const std::string fw = "fft2_small_fwd_" + std::to_string(N);
    static const std::string iv = "fft2_small_inv_" + std::to_string(N);
    if (inverse)
      err = small2d_launch<k_fft2_small_inv<N, P>>(iv.c_str(), (unsigned)grid, lds, s, Xi, xo, count, alpha, beta);
    else
      err = small2d_launch<k_fft2_small_fwd<N, P>>(fw.c_str(), (unsigned)grid, lds, s, x, X, count, alpha, beta);
  });
  return err;
}

}  // namespace fdc
