// HIP kernels of the CIC + FDP layer path for gfx950, and their launchers.
//
// Layer forward (section 2.4.1, Algorithm 1 inside Algorithm 2, FDP of 2.4.2):
//   k_row_r2c      real rows of x -> half-spectrum rows, only the m/2+1 columns FDP keeps
//   k_col_fwd_crop column DFT (n) -> keep the m rows FDP keeps (the saved spectrum)
//   k_col_cic_inv  for each output channel: CIC product (Eq. 5) -> inverse column DFT (m)
//   k_row_c2r      inverse real row DFT (m) with real-part semantics and 1/m^2
// Layer backward:
//   k_row_r2c     upstream gradient -> (c_l/m^2) weighted half spectrum
//   k_col_bwd_gk  column DFT (m), dL/dK = sum_b G conj(Xhat); the batch is split over
//                 wave groups of one workgroup (and, for large batches, over image
//                 ranges added by k_gk_reduce) and summed in a fixed order
//   k_col_bwd_gx  column DFTs (m) of the J gradients, sum_j G conj(K), zero-padded
//                 inverse column DFT (n)
//   k_col_bwd_dk_dx  the two above in one launch (stack executor)
//   k_row_c2r     adjoint row transform (n)
// Stack executor: k_row_c2r_r2c runs a layer's inverse rows and the next layer's
// forward rows (backward: the adjoint pair) on the same rows in one kernel.
// Intermediates stay row-major [plane][row][column]; column kernels own CT adjacent
// columns (numbered across planes) with the column index fastest across lanes, so
// every global access is a run of up to CT consecutive complex values.
#include "device.h"
#include "fft.h"
#include "internal.h"

#include <algorithm>
#include <string>
#include <type_traits>

namespace fdc {

// Element offset of logical pixel (r, w) of an image seen through `v`, or -1 when
// the pixel is not stored (cropped away).  MODE is v.mode, fixed at compile time.
template <int MODE>
__device__ __forceinline__ int view_index(const ImgView &v, int ncols, int r, int w) {
  if constexpr (MODE == 0) {
    return r * v.cols_stored + w;
  } else if constexpr (MODE == 1) {
    const int rr = r - v.shift, ww = w - v.shift;
    return (rr < 0 || ww < 0) ? -1 : rr * v.cols_stored + ww;
  } else {
    int rr = r - v.shift, ww = w - v.shift;
    rr += rr < 0 ? v.rows : 0;
    ww += ww < 0 ? ncols : 0;
    return rr * v.cols_stored + ww;
  }
}

__device__ __forceinline__ float bin_weight(int l, int n, float alpha, float beta) {
  return (l == 0 || 2 * l == n) ? alpha : alpha * beta;
}

extern __shared__ float2 g_lds[];

// LDS layouts (see lds_phys): padded for the row transforms, plain for the column
// transforms.
constexpr int kRowLds = kLdsPad;
constexpr int kColLds = kLdsPlain;

// ---------------------------------------------------------------------------
// row transforms
// ---------------------------------------------------------------------------
// Row pairs per workgroup: 256 threads, at most 64 pairs.
template <int N>
constexpr int row_spw() {
  constexpr int s = 256 / RowCfg<N>::TPS;
  return s > 64 ? 64 : s;
}

// Sequence (row pair) index of this thread in its workgroup.  With one sequence per
// wavefront it is read from the first lane, so that the compiler sees it as uniform
// and keeps the row addresses derived from it in scalar registers.
template <int TPS>
__device__ __forceinline__ int row_seq() {
  const int s = (int)threadIdx.x / TPS;
  if constexpr (TPS == 64) return __builtin_amdgcn_readfirstlane(s);
  else return s;
}

// Element i of p addressed by a 32-bit byte offset (i * sizeof(T) < 2^32): on a base
// uniform across the wavefront the access is one instruction with a scalar base and a
// 32-bit lane offset, instead of 64-bit address arithmetic per lane.
template <class T>
__device__ __forceinline__ T &at32(T *p, unsigned i) {
  using B = typename std::conditional<std::is_const<T>::value, const char, char>::type;
  return *reinterpret_cast<T *>(reinterpret_cast<B *>(p) + i * (unsigned)sizeof(T));
}

// Offset of bin l (< L-1) in its row of the main block, 32-bit: a row's bins lie within
// one plane, (L-1) * rows complex values.
__device__ __forceinline__ unsigned bin_off32(const SpecLayout &sl, int l) {
  return (unsigned)(l >> 3) * (unsigned)sl.ts + (unsigned)(l & 7);
}

// Sequence s's natural-order elements into the padded LDS rows (element e at
// lds_phys(s N + e)), thread t holding elements t + TPS m.
template <int N>
__device__ __forceinline__ void row_to_lds(const float2 (&v)[RowCfg<N>::E], float2 *lds, int s, int t) {
  constexpr int TPS = RowCfg<N>::TPS, E = RowCfg<N>::E;
  if constexpr (N % 32 == 0 && TPS % 32 == 0) {
    const int i0 = lds_phys<kRowLds>(s * N + t);
#pragma unroll
    for (int m = 0; m < E; ++m) lds[i0 + pad_offset(TPS * m)] = v[m];
  } else {
#pragma unroll
    for (int m = 0; m < E; ++m) lds[lds_phys<kRowLds>(s * N + t + TPS * m)] = v[m];
  }
}

// Real rows are transformed in pairs packed as one complex sequence z = a + i b.
// A sequence uses TPS <= 64 threads, so a wavefront holds whole sequences and
// the LDS exchanges need only wave-level ordering.
template <int N, int SPW, int MODE>
__global__ __launch_bounds__(SPW *RowCfg<N>::TPS) void k_row_r2c(const float *__restrict__ x, SpecLayout out,
                                                                long long npairs, int rows_per_plane, ImgView view,
                                                                long long in_plane_stride, int L, float alpha,
                                                                float beta) {
  using Cfg = RowCfg<N>;
  constexpr int TPS = Cfg::TPS, E = Cfg::E;
  static_assert(TPS <= 64, "a row sequence must fit in one wavefront");
  float2 *tw = g_lds, *lds = g_lds + twiddle_lds_elems<N>();
  TwiddleStage<N, SPW * TPS> tws;
  tws.fetch(threadIdx.x);
  const int t = threadIdx.x % TPS, s = row_seq<TPS>();
  // 32-bit row arithmetic: the launchers keep planes * rows_per_plane below 2^31
  int pair = xcd_remap(blockIdx.x, gridDim.x) * SPW + s;
  const bool active = pair < npairs;
  if (!active) pair = (int)npairs - 1;
  const unsigned row0 = 2u * (unsigned)pair;
  const long long plane = row0 / (unsigned)rows_per_plane;
  const int r0 = (int)(row0 - (unsigned)plane * (unsigned)rows_per_plane);
  const float *xp = x + plane * in_plane_stride;

  float2 v[E];
#pragma unroll
  for (int m = 0; m < E; ++m) {
    const int w = t + TPS * m;
    const int ia = view_index<MODE>(view, N, r0, w);
    const int ib = view_index<MODE>(view, N, r0 + 1, w);
    // unconditional loads (a cropped-away pixel reads element 0), zeroed afterwards: a load
    // under a lane condition would be issued in its own branch and wait for its data alone
    const float xa = at32(xp, (unsigned)(ia < 0 ? 0 : ia)), xb = at32(xp, (unsigned)(ib < 0 ? 0 : ib));
    v[m] = make_float2(ia >= 0 ? xa : 0.f, ib >= 0 ? xb : 0.f);
  }
  tws.commit(tw, threadIdx.x);  // the twiddle table and the rows load together
  fft_seq<N, -1, true, true, kRowLds, RowCfg<N>>(v, t, lds, s * N, 1, tw, 1);
  lds_barrier<true>();
  row_to_lds<N>(v, lds, s, t);
  lds_barrier<true>();
  if (!active) return;
  float2 *oa = out.main + plane * out.ps + (long long)r0 * out.rs;
  float2 *ob = oa + out.rs;
  for (int k = t; k < L; k += TPS) {
    const float2 zk = lds[lds_phys<kRowLds>(s * N + k)];
    const float2 zn = lds[lds_phys<kRowLds>(s * N + (k == 0 ? 0 : N - k))];
    const float wgt = 0.5f * bin_weight(k, N, alpha, beta);
    // two real rows packed as z = a + i b:  A = (Z[k] + conj Z[-k]) / 2,  B = (Z[k] - conj Z[-k]) / (2i)
    const float2 A = make_float2((zk.x + zn.x) * wgt, (zk.y - zn.y) * wgt);
    const float2 Bv = make_float2((zk.y + zn.y) * wgt, (zn.x - zk.x) * wgt);
    if (k < L - 1) {
      const unsigned o = bin_off32(out, k);
      at32(oa, o) = A;
      at32(ob, o) = Bv;
    } else {
      float2 *sa = out.side + plane * out.sps + (long long)r0 * out.srs;
      sa[0] = A;
      sa[out.srs] = Bv;
    }
  }
}

// Input of the inverse real row transform of the pair (r0, r0 + 1) for thread t:
// v[m] = A_k + i B_k at k = t + TPS m, where A and B are the Hermitian extensions of
// the two rows' half spectra weighted by c_l (a1 at l = 0 and N/2, a1 b1 elsewhere,
// 0 at l >= Lin), with real-part semantics at l = 0 and N/2.
// Input-bin modes: LIN = 0 any Lin; LIN = 1 Lin = N/2 + 1; LIN = 2 Lin = N/4 + 1.  The
// last two know at compile time which elements are zero, main-block bins or the
// last (side-block) bin, and leave out the common factor a1 b1, which the caller
// applies after the transform (b1 must be nonzero).
template <int N, int LIN>
__device__ __forceinline__ void c2r_gather(float2 (&v)[RowCfg<N>::E], const SpecLayout &in, long long plane, int r0,
                                           int t, int Lin, float a1, float b1) {
  using Cfg = RowCfg<N>;
  constexpr int TPS = Cfg::TPS, E = Cfg::E;
  const float2 *ia = in.main + plane * in.ps + (long long)r0 * in.rs;
  const float2 *ib = ia + in.rs;
  const float2 *sa = in.side + plane * in.sps + (long long)r0 * in.srs;
  if constexpr (LIN == 0) {
#pragma unroll
    for (int m = 0; m < E; ++m) {
      const int k = t + TPS * m;
      const bool upper = 2 * k > N;
      const int kk = upper ? N - k : k;
      // unconditional loads from valid addresses; bins beyond Lin get weight 0 (the loaded
      // value is always used, so the load is not sunk into a per-lane branch)
      const bool in_main = kk < Lin - 1;
      const unsigned o = bin_off32(in, kk);
      const float2 *pa = in_main ? ia + o : sa;
      const float2 *pb = in_main ? ib + o : sa + in.srs;
      float2 a = *pa, b = *pb;
      const bool edge = (kk == 0 || 2 * kk == N);
      const float wgt = kk < Lin ? (edge ? a1 : a1 * b1) : 0.f;
      a = cscale(a, wgt);
      b = cscale(b, wgt);
      if (edge) {  // real-part semantics of the inverse at l = 0 and l = n/2
        a.y = 0.f;
        b.y = 0.f;
      }
      if (upper) {  // Hermitian extension of each real row's half spectrum
        a.y = -a.y;
        b.y = -b.y;
      }
      v[m] = make_float2(a.x - b.y, a.y + b.x);  // A + i B
    }
  } else {
    static_assert(E % (LIN == 1 ? 2 : 4) == 0, "input-bin mode needs E divisible by 2 (LIN 1) or 4 (LIN 2)");
    (void)Lin;
    (void)a1;
    constexpr int KS = LIN == 1 ? N / 2 : N / 4;  // the side-block bin, Lin - 1
    const float2 *sb = sa + in.srs;
    const float e1 = 1.f / b1;  // edge weight a1 relative to the common a1 b1
    const bool t0 = t == 0;
    // Lane conditions act through pointer selects and multipliers, never through a
    // branch around a load (which would make the load wait for its data alone).
    const float ex = t0 ? e1 : 1.f, ey = t0 ? 0.f : 1.f;
    static_for<0, E>([&](auto mc) {
      constexpr int m = decltype(mc)::value;
      constexpr bool low = m < E / 2;  // k < N/2: bin k; otherwise bin N - k, conjugated
      // LIN 2: bins above N/4 are dropped, which empties m in (E/4, 3E/4) and, at
      // m = E/4, every lane but t = 0 (bin N/4)
      if constexpr (LIN == 2 && m > E / 4 && m < 3 * E / 4) {
        v[m] = make_float2(0.f, 0.f);
        return;
      }
      float2 a, b;
      if constexpr (LIN == 2 && m == E / 4) {
        const float keep = t0 ? 1.f : 0.f;
        a = cscale(*sa, keep);
        b = cscale(*sb, keep);
      } else {
        // m whose lane t = 0 holds the side bin KS (bin KS - t on the other lanes)
        constexpr bool side_m = (LIN == 1 && m == E / 2) || (LIN == 2 && m == 3 * E / 4);
        if constexpr (side_m) {
          const unsigned o = bin_off32(in, KS - t);
          const float2 *pa = t0 ? sa : ia + o;
          const float2 *pb = t0 ? sb : ib + o;
          a = *pa;
          b = *pb;
        } else {
          const int kk = low ? t + TPS * m : N - t - TPS * m;
          const unsigned o = bin_off32(in, kk);
          a = at32(ia, o);
          b = at32(ib, o);
        }
        // l = 0 (m = 0, t = 0) and, with LIN 1, l = N/2 (m = E/2, t = 0): weight a1 and
        // real-part semantics
        if constexpr (m == 0 || (LIN == 1 && m == E / 2)) {
          a = make_float2(a.x * ex, a.y * ey);
          b = make_float2(b.x * ex, b.y * ey);
        }
      }
      if constexpr (!low) {
        a.y = -a.y;
        b.y = -b.y;
      }
      v[m] = make_float2(a.x - b.y, a.y + b.x);
    });
  }
}

// Input-bin mode of c2r_gather for Lin bins of an N-point row (and weight b1).
template <int N>
int c2r_lin_mode(int Lin, float b1) {
  if (b1 == 0.f) return 0;
  if (Lin == N / 2 + 1 && RowCfg<N>::E % 2 == 0) return 1;
  if (Lin == N / 4 + 1 && N % 4 == 0 && RowCfg<N>::E % 4 == 0) return 2;
  return 0;
}

template <int N, int SPW, int MODE, int LIN>
__global__ __launch_bounds__(SPW *RowCfg<N>::TPS) void k_row_c2r(SpecLayout in, float *__restrict__ y,
                                                                long long npairs, int rows_per_plane, int L,
                                                                float alpha, float beta, ImgView view,
                                                                long long out_plane_stride) {
  using Cfg = RowCfg<N>;
  constexpr int TPS = Cfg::TPS, E = Cfg::E;
  static_assert(TPS <= 64, "a row sequence must fit in one wavefront");
  float2 *tw = g_lds, *lds = g_lds + twiddle_lds_elems<N>();
  TwiddleStage<N, SPW * TPS> tws;
  tws.fetch(threadIdx.x);
  const int t = threadIdx.x % TPS, s = row_seq<TPS>();
  // 32-bit row arithmetic: the launchers keep planes * rows_per_plane below 2^31
  int pair = xcd_remap(blockIdx.x, gridDim.x) * SPW + s;
  const bool active = pair < npairs;
  if (!active) pair = (int)npairs - 1;
  const unsigned row0 = 2u * (unsigned)pair;
  const long long plane = row0 / (unsigned)rows_per_plane;
  const int r0 = (int)(row0 - (unsigned)plane * (unsigned)rows_per_plane);
  float2 v[E];
  c2r_gather<N, LIN>(v, in, plane, r0, t, L, alpha, beta);
  tws.commit(tw, threadIdx.x);  // the twiddle table and the rows load together
  fft_seq<N, +1, true, true, kRowLds, RowCfg<N>>(v, t, lds, s * N, 1, tw, 1);
  if (!active) return;
  const float sc = LIN == 0 ? 1.f : alpha * beta;  // the factor c2r_gather left out
  float *yp = y + plane * out_plane_stride;
#pragma unroll
  for (int m = 0; m < E; ++m) {
    const int w = t + TPS * m;
    const int oa = view_index<MODE>(view, N, r0, w);
    const int ob = view_index<MODE>(view, N, r0 + 1, w);
    if (oa >= 0) at32(yp, (unsigned)oa) = LIN == 0 ? v[m].x : v[m].x * sc;
    if (ob >= 0) at32(yp, (unsigned)ob) = LIN == 0 ? v[m].y : v[m].y * sc;
  }
}

// Zeros of z.p at the bins the FDP drops, in jobs of one wavefront: jobs [0, S * CA)
// are 512-value chunks of the S contiguous dropped-row blocks ((N - M) (N/2+1) values
// each, CA chunks per block), jobs [S * CA, S * CA + S * M) the dropped columns of one
// kept row.  Wavefront w of nw takes jobs w, w + nw, ...; w is wave-uniform, so the job
// arithmetic is scalar and each store instruction writes 64 consecutive values.
__device__ __forceinline__ void zero_dropped_bins(const ZeroBins &z, unsigned w, unsigned nw, int lane) {
  const int nf = z.N / 2 + 1, L = z.M / 2 + 1;
  const unsigned ra = (unsigned)(z.N - z.M) * (unsigned)nf, ca = (ra + 511) / 512;
  const unsigned ja = (unsigned)z.S * ca, jobs = ja + (unsigned)z.S * (unsigned)z.M;
  const float2 zero = make_float2(0.f, 0.f);
  for (unsigned j = w; j < jobs; j += nw) {
    if (j < ja) {
      const unsigned o = j / ca, c0 = (j - o * ca) * 512;
      float2 *blk = z.p + ((long long)o * z.N + z.M / 2) * nf;
      for (unsigned e = c0 + lane; e < c0 + 512 && e < ra; e += 64) blk[e] = zero;
    } else {
      const unsigned r = j - ja, o = r / (unsigned)z.M;
      const int kr = (int)(r - o * (unsigned)z.M), k = kr < z.M / 2 ? kr : kr + (z.N - z.M);
      float2 *row = z.p + ((long long)o * z.N + k) * nf;
      for (int l = L + lane; l < nf; l += 64) row[l] = zero;
    }
  }
}

// Inverse real row transform followed by the forward real row transform of the same
// rows, for a boundary between two layers of a stack: in (Lin bins per row, weights
// a1 at l = 0 and N/2, a1 * b1 elsewhere, real-part semantics as k_row_c2r) ->
// the two real rows of each pair, kept in registers -> out (Lout bins, weights as
// k_row_r2c with a2, b2).  The same rows, pairing and arithmetic as k_row_c2r
// followed by k_row_r2c, without writing the real rows to memory.
template <int N, int SPW, int LIN>
__global__ __launch_bounds__(SPW *RowCfg<N>::TPS) void k_row_c2r_r2c(SpecLayout in, int Lin, float a1, float b1,
                                                                    SpecLayout out, int Lout, float a2, float b2,
                                                                    long long npairs, int rows_per_plane,
                                                                    ZeroBins zeros) {
  using Cfg = RowCfg<N>;
  constexpr int TPS = Cfg::TPS, E = Cfg::E;
  static_assert(TPS <= 64, "a row sequence must fit in one wavefront");
  float2 *tw = g_lds, *lds = g_lds + twiddle_lds_elems<N>();
  TwiddleStage<N, SPW * TPS> tws;
  tws.fetch(threadIdx.x);
  const int t = threadIdx.x % TPS, s = row_seq<TPS>();
  // 32-bit row arithmetic: the launchers keep planes * rows_per_plane below 2^31
  int pair = xcd_remap(blockIdx.x, gridDim.x) * SPW + s;
  const bool active = pair < npairs;
  if (!active) pair = (int)npairs - 1;
  const unsigned row0 = 2u * (unsigned)pair;
  const long long plane = row0 / (unsigned)rows_per_plane;
  const int r0 = (int)(row0 - (unsigned)plane * (unsigned)rows_per_plane);
  float2 v[E];
  c2r_gather<N, LIN>(v, in, plane, r0, t, Lin, a1, b1);
  tws.commit(tw, threadIdx.x);  // the twiddle table and the rows load together
  fft_seq<N, +1, true, true, kRowLds, RowCfg<N>>(v, t, lds, s * N, 1, tw, 1);
  // v[m] = (row r0, row r0 + 1) at column t + TPS m: the packed input of the forward transform
  fft_seq<N, -1, true, true, kRowLds, RowCfg<N>>(v, t, lds, s * N, 1, tw, 1);
  lds_barrier<true>();
  row_to_lds<N>(v, lds, s, t);
  lds_barrier<true>();
  if (active) {
    const float a2s = LIN == 0 ? a2 : a2 * (a1 * b1);  // with the factor c2r_gather left out
    float2 *oa = out.main + plane * out.ps + (long long)r0 * out.rs;
    float2 *ob = oa + out.rs;
    for (int k = t; k < Lout; k += TPS) {
      const float2 zk = lds[lds_phys<kRowLds>(s * N + k)];
      const float2 zn = lds[lds_phys<kRowLds>(s * N + (k == 0 ? 0 : N - k))];
      const float wgt = 0.5f * bin_weight(k, N, a2s, b2);
      const float2 A = make_float2((zk.x + zn.x) * wgt, (zk.y - zn.y) * wgt);
      const float2 Bv = make_float2((zk.y + zn.y) * wgt, (zn.x - zk.x) * wgt);
      if (k < Lout - 1) {
        const unsigned o = bin_off32(out, k);
        at32(oa, o) = A;
        at32(ob, o) = Bv;
      } else {
        float2 *so = out.side + plane * out.sps + (long long)r0 * out.srs;
        so[0] = A;
        so[out.srs] = Bv;
      }
    }
  }
  // the zeros of a kernel gradient, in wavefront jobs (the rows above are this launch's own work)
  if (zeros.p != nullptr) {
    const unsigned wpb = (SPW * RowCfg<N>::TPS) / 64;
    zero_dropped_bins(zeros, blockIdx.x * wpb + __builtin_amdgcn_readfirstlane(threadIdx.x / 64), gridDim.x * wpb,
                      threadIdx.x % 64);
  }
}

// ---------------------------------------------------------------------------
// column transforms
//
// Column kernels see their input as `planes` row-major [rows][L] complex images.
// A workgroup owns CT columns, with lanes running fastest along the columns so
// that each global access is a run of CT consecutive complex values of one row.
// Tiling: the first MAIN = ((L-1)/CT)*CT columns of every plane form aligned
// tiles (run starts on a multiple of CT, never straddling planes); the remaining
// L - MAIN columns of all planes -- for L = 2^k + 1 only the last, Nyquist,
// column -- are packed CT at a time into tail tiles numbered after the main
// tiles.  Tiles that start off the CT grid split every row access into two
// transactions and run at about half the bandwidth.
// ---------------------------------------------------------------------------
template <int N>
constexpr int col_ct() {
  return ColCfg<N>::TPS >= 64 ? 8 : (ColCfg<N>::TPS >= 32 ? 16 : 32);
}
// Narrower tiles (twice the workgroups) where measurement favoured them: the dX
// kernel (three transforms per tile), the forward crop at 128, 256 and 1024 points (at
// 1024 points 8 images of one channel give 257 workgroups of eight waves; with 4-column
// tiles 10.3 -> 9.0 us) and the CIC inverse at 64 points.
template <int N>
constexpr int col_ct_gx() {
  return col_ct<N>() / 2;
}
template <int N>
constexpr int col_ct_crop() {
  return (N == 128 || N == 256 || N == 1024) ? col_ct<N>() / 2 : col_ct<N>();
}
template <int M>
constexpr int col_ct_cic() {
  return M == 64 ? col_ct<M>() / 2 : col_ct<M>();
}
// Full FDC column passes at 512 points: 16-column tiles, so that each row access of a
// tile is one whole 128-byte line of the row-interleaved spectra (whose rows lie
// megabytes apart); 4.0 -> 3.75 ms per pass at 16 images of 256 channels.
template <int N>
constexpr int col_ct_split() {
  return N == 512 ? 16 : col_ct<N>();
}

// CT for columns [0, L): at most `ct` and a divisor of L - 1 when L - 1 > 0.
__host__ __device__ constexpr int col_ct_for(int ct, int L) {
  const int lm1 = L - 1;
  const int low = lm1 > 0 ? (lm1 & -lm1) : ct;
  return low < ct ? low : ct;
}

__host__ __device__ constexpr long long col_tile_count(long long planes, int L, int ct) {
  return planes * ((L - 1) / ct) + (planes * (L - (L - 1) / ct * ct) + ct - 1) / ct;
}

struct ColRef {
  int plane;
  int l;
  bool ok;
};

// Column `s` of tile w.  Out-of-range lanes of the last tail tile get ok = false
// and a valid (repeated) column, so their loads stay in bounds.
// Main tiles run through G consecutive planes (G divides `planes`) at one column
// position before moving on: kernels number their planes so that such a group
// reads the same columns of a shared operand, which the group's workgroups -- on
// one XCD after xcd_remap, at about the same time -- then fetch once into its L2.
template <int CT>
__device__ __forceinline__ ColRef column_ref(int w, int s, int L, int planes, int G = 1) {
  const int mpp = (L - 1) / CT, rt = L - mpp * CT;
  const int main_tiles = planes * mpp;
  ColRef r;
  if (w < main_tiles) {
    const int blk = G * mpp;
    const int gi = w / blk, rr = w - gi * blk;
    const int tile = rr / G;
    r.plane = gi * G + (rr - tile * G);
    r.l = tile * CT + s;
    r.ok = true;
  } else {
    int q = (w - main_tiles) * CT + s;
    const int total = planes * rt;
    r.ok = q < total;
    if (!r.ok) q = total - 1;
    r.plane = q / rt;
    r.l = mpp * CT + (q - r.plane * rt);
  }
  return r;
}

template <int N, int CT, int DIR>
__global__ __launch_bounds__(CT *ColCfg<N>::TPS) void k_col_fft(const float2 *in, float2 *out, int L, int ld,
                                                               int planes, long long in_plane_stride,
                                                               long long out_plane_stride, int keep) {
  using Cfg = ColCfg<N>;
  constexpr int TPS = Cfg::TPS, E = Cfg::E;
  float2 *tw = g_lds, *lds = g_lds + twiddle_lds_elems<N>();
  stage_twiddles<N>(tw, threadIdx.x, CT * TPS);
  const int s = threadIdx.x % CT, t = threadIdx.x / CT;
  const ColRef c = column_ref<CT>(xcd_remap(blockIdx.x, gridDim.x), s, L, planes);
  const float2 *ip = in + c.plane * in_plane_stride + c.l;
  float2 v[E];
#pragma unroll
  for (int m = 0; m < E; ++m) v[m] = ip[(long long)(t + TPS * m) * ld];  // lanes past the end read a valid column
  fft_seq<N, DIR, true, false, kLdsPlain, ColCfg<N>>(v, t, lds, s, CT, tw, 1);
  if (!c.ok) return;
  float2 *op = out + c.plane * out_plane_stride + c.l;
#pragma unroll
  for (int m = 0; m < E; ++m) {
    const int k = t + TPS * m;  // only the rows an FDP to `keep` rows keeps (keep = N: all)
    if (k < keep / 2 || k >= N - keep / 2) op[(long long)k * ld] = v[m];
  }
}

// Row of the n-point spectrum that pooled row `mrow` (of m) comes from.
template <int N, int M>
__device__ __forceinline__ int kept_row(int mrow) {
  return mrow < M / 2 ? mrow : mrow + (N - M);
}

// Column (plane, l) of a tiled spectrum (tiled_layout) of `planes` images with ROWS
// rows and L bins per row: row r is at p[r * stride].  Bins l < L-1 sit in tiles of
// 8 columns stored down the rows (stride 8); narrower rows (L - 1 < 8) are
// row-major; the last bin is in the side block (stride 1).
struct ColPtr {
  float2 *p;
  int stride;
};
template <int ROWS, int L>
__device__ __forceinline__ ColPtr tiled_col(const float2 *base, int planes, int plane, int l) {
  constexpr int H = L - 1;
  float2 *b = const_cast<float2 *>(base);
  if (l < H) {
    if constexpr (H % 8 == 0)
      return ColPtr{b + (long long)plane * ROWS * H + (long long)(l >> 3) * ROWS * 8 + (l & 7), 8};
    else
      return ColPtr{b + (long long)plane * ROWS * H + l, H};
  }
  return ColPtr{b + (long long)planes * ROWS * H + (long long)plane * ROWS, 1};
}

// Column DFTs (N, direction DIR) of `planes` split-layout N x (N/2+1) half spectra
// with any plane strides (SpecLayout), in place or out of place (each workgroup
// reads its columns whole before writing).
struct ColPtr64 {
  float2 *p;
  long long stride;
};
__device__ __forceinline__ ColPtr64 layout_col(const SpecLayout &sl, int H, int plane, int l) {
  if (l < H) return ColPtr64{sl.main + (long long)plane * sl.ps + bin_off(sl, l), sl.rs};
  return ColPtr64{sl.side + (long long)plane * sl.sps, sl.srs};
}

template <int N, int CT, int DIR>
__global__ __launch_bounds__(CT *ColCfg<N>::TPS) void k_col_fft_split(SpecLayout in, SpecLayout out, int planes) {
  using Cfg = ColCfg<N>;
  constexpr int L = N / 2 + 1, TPS = Cfg::TPS, E = Cfg::E;
  float2 *tw = g_lds, *lds = g_lds + twiddle_lds_elems<N>();
  stage_twiddles<N>(tw, threadIdx.x, CT * TPS);
  const int s = threadIdx.x % CT, t = threadIdx.x / CT;
  const ColRef c = column_ref<CT>(xcd_remap(blockIdx.x, gridDim.x), s, L, planes);
  const ColPtr64 ic = layout_col(in, L - 1, c.plane, c.l);
  float2 v[E];
#pragma unroll
  for (int m = 0; m < E; ++m) v[m] = ic.p[(t + TPS * m) * ic.stride];  // lanes past the end read a valid column
  fft_seq<N, DIR, true, false, kLdsPlain, ColCfg<N>>(v, t, lds, s, CT, tw, 1);
  if (!c.ok) return;
  const ColPtr64 oc = layout_col(out, L - 1, c.plane, c.l);
#pragma unroll
  for (int m = 0; m < E; ++m) oc.p[(t + TPS * m) * oc.stride] = v[m];
}

// Forward column DFT (N) of the L columns of row spectra in the layout `in`; the rows
// an FDP to `keep` rows keeps go to the row-major out (row stride ld) at their own rows.
template <int N, int CT>
__global__ __launch_bounds__(CT *ColCfg<N>::TPS) void k_col_fft_keep(SpecLayout in, float2 *out, int L, int ld,
                                                                    int planes, long long out_plane_stride, int keep) {
  using Cfg = ColCfg<N>;
  constexpr int TPS = Cfg::TPS, E = Cfg::E;
  float2 *tw = g_lds, *lds = g_lds + twiddle_lds_elems<N>();
  TwiddleStage<N, CT * TPS> tws;
  tws.fetch(threadIdx.x);
  const int s = threadIdx.x % CT, t = threadIdx.x / CT;
  const ColRef c = column_ref<CT>(xcd_remap(blockIdx.x, gridDim.x), s, L, planes);
  const ColPtr64 ic = layout_col(in, L - 1, c.plane, c.l);
  float2 v[E];
#pragma unroll
  for (int m = 0; m < E; ++m) v[m] = ic.p[(t + TPS * m) * ic.stride];  // lanes past the end read a valid column
  tws.commit(tw, threadIdx.x);
  fft_seq<N, -1, true, false, kLdsPlain, ColCfg<N>>(v, t, lds, s, CT, tw, 1);
  if (!c.ok) return;
  float2 *op = out + c.plane * out_plane_stride + c.l;
#pragma unroll
  for (int m = 0; m < E; ++m) {
    const int k = t + TPS * m;
    if (k < keep / 2 || k >= N - keep / 2) op[(long long)k * ld] = v[m];
  }
}

// Forward, first half: column DFT (N) of the pruned row spectra, keep the M rows
// FDP keeps.  T [planes][N rows] -> Xh [planes][M rows], both split layout with
// L = M/2 + 1 bins per row (Xh is the pooled input spectrum the backward reads).
template <int N, int M, int CT>
__global__ __launch_bounds__(CT *ColCfg<N>::TPS) void k_col_fwd_crop(const float2 *__restrict__ T,
                                                                    float2 *__restrict__ Xh, int planes) {
  using CN = ColCfg<N>;
  constexpr int L = M / 2 + 1, TPS = CN::TPS, E = CN::E;
  float2 *tw = g_lds, *lds = g_lds + twiddle_lds_elems<N>();
  TwiddleStage<N, CT * TPS> tws;
  tws.fetch(threadIdx.x);
  const int s = threadIdx.x % CT, t = threadIdx.x / CT;
  const ColRef c = column_ref<CT>(xcd_remap(blockIdx.x, gridDim.x), s, L, planes);
  const ColPtr tc = tiled_col<N, L>(T, planes, c.plane, c.l);
  float2 v[E];
#pragma unroll
  for (int m = 0; m < E; ++m) v[m] = tc.p[(t + TPS * m) * tc.stride];  // lanes past the end read a valid column
  tws.commit(tw, threadIdx.x);
  fft_seq<N, -1, true, false, kLdsPlain, ColCfg<N>>(v, t, lds, s, CT, tw, 1);
  if (!c.ok) return;
  const ColPtr xc = tiled_col<M, L>(Xh, planes, c.plane, c.l);
#pragma unroll
  for (int m = 0; m < E; ++m) {
    const int k = t + TPS * m;
    if (k < M / 2) xc.p[k * xc.stride] = v[m];
    else if (k >= N - M / 2) xc.p[(k - (N - M)) * xc.stride] = v[m];
  }
}

// Forward, second half: for every output channel o = c*J + j, the CIC product
// (Eq. 5) of the pooled spectrum with kernel o at the kept bins, then the inverse
// column DFT (M).  Xh [B*C][M rows], K [S][N][N/2+1] -> U [B*S][M rows].
// A workgroup takes JW consecutive output channels of one input channel (groups =
// B * C * J / JW of them): it loads the pooled column once, and the next kernel
// column while the current one is transformed.
// Output channels of one input channel handled by one workgroup of the CIC inverse
// kernel (a divisor of J): the pooled input column is loaded once for all of them.
constexpr int kCicJW = 4;
// CIC inverse grids below this many workgroups switch to 8-column tiles.
constexpr unsigned kCicNarrowGrid = 256;

template <int N, int M, int CT, int JW>
__global__ __launch_bounds__(CT *ColCfg<M>::TPS) void k_col_cic_inv(const float2 *__restrict__ Xh,
                                                                   const float2 *__restrict__ K,
                                                                   float2 *__restrict__ U, int B, int C, int J,
                                                                   int groups) {
  using CM = ColCfg<M>;
  constexpr int L = M / 2 + 1, NF = N / 2 + 1, TPS = CM::TPS, E = CM::E;
  float2 *tw = g_lds, *lds = g_lds + twiddle_lds_elems<M>();
  TwiddleStage<M, CT * TPS> tws;
  tws.fetch(threadIdx.x);
  const int s = threadIdx.x % CT, t = threadIdx.x / CT;
  // group index (ci * JB + jb) * B + b: the B images read the same kernel columns
  const ColRef c = column_ref<CT>(xcd_remap(blockIdx.x, gridDim.x), s, L, groups, B);
  const int S = C * J, JB = J / JW;
  const int b = c.plane % B, cj = c.plane / B;
  const int ci = cj / JB;
  const int o0 = ci * J + (cj - ci * JB) * JW;
  const int bc = b * C + ci;
  const ColPtr xc = tiled_col<M, L>(Xh, groups / JB, bc, c.l);
  float2 x[E], kn[E];
  auto load_k = [&](int o) {
    const float2 *kcol = K + (long long)o * N * NF + c.l;
#pragma unroll
    for (int m = 0; m < E; ++m) kn[m] = kcol[kept_row<N, M>(t + TPS * m) * NF];  // valid column on every lane
  };
#pragma unroll
  for (int m = 0; m < E; ++m) x[m] = xc.p[(t + TPS * m) * xc.stride];
  load_k(o0);
  tws.commit(tw, threadIdx.x);
  for (int jj = 0; jj < JW; ++jj) {
    float2 z[E];
#pragma unroll
    for (int m = 0; m < E; ++m) z[m] = cmul(x[m], kn[m]);
    if (jj + 1 < JW) load_k(o0 + jj + 1);  // the next kernel column loads while this one transforms
    fft_seq<M, +1, true, false, kLdsPlain, ColCfg<M>>(z, t, lds, s, CT, tw, 1);
    if (c.ok) {
      const ColPtr uc = tiled_col<M, L>(U, groups * JW, b * S + o0 + jj, c.l);  // B * S planes
#pragma unroll
      for (int m = 0; m < E; ++m) uc.p[(t + TPS * m) * uc.stride] = z[m];
    }
  }
}

// Forward, both halves in one kernel: column DFT (N) of T, the kept rows to Xh and to
// an LDS tile, then the CIC product (Eq. 5) and inverse column DFT (M) for JW output
// channels.  The J = JW * JB output channels of an input channel are split over JB
// workgroup groups, each of which transforms the input column itself (group 0 stores
// Xh).  The N-point thread layout holds JP = TPS_N / TPS_M groups of the M-point
// layout, which take the output channels in turns.  Planes and tile order as
// k_col_cic_inv: group index (ci * JB + jb) * B + b, the B images of one input
// channel and channel group in a row.
template <int N, int M, int CT, int JW>
__global__ __launch_bounds__(CT *ColCfg<N>::TPS) void k_col_fwd_cic(const float2 *__restrict__ T,
                                                                   const float2 *__restrict__ K,
                                                                   float2 *__restrict__ U, float2 *__restrict__ Xh,
                                                                   int B, int C, int JB) {
  using CN = ColCfg<N>;
  using CM = ColCfg<M>;
  constexpr int L = M / 2 + 1, NF = N / 2 + 1, TPSN = CN::TPS, TPSM = CM::TPS, EN = CN::E, EM = CM::E;
  constexpr int JP = TPSN / TPSM;
  static_assert(JP * TPSM == TPSN, "thread layouts of the two transforms must nest");
  float2 *tw = g_lds, *lds = g_lds + twiddle_lds_elems<N>();
  TwiddleStage<N, CT * TPSN> tws;
  tws.fetch(threadIdx.x);
  const int s = threadIdx.x % CT, t = threadIdx.x / CT;
  const int tp = t % TPSM, js = t / TPSM;
  const ColRef c = column_ref<CT>(xcd_remap(blockIdx.x, gridDim.x), s, L, B * C * JB, B);
  const int b = c.plane % B, cj = c.plane / B;
  const int ci = cj / JB, jb = cj - ci * JB;
  const int bc = b * C + ci, J = JW * JB, S = C * J;
  const ColPtr tc = tiled_col<N, L>(T, B * C, bc, c.l);
  float2 v[EN];
#pragma unroll
  for (int m = 0; m < EN; ++m) v[m] = tc.p[(t + TPSN * m) * tc.stride];  // lanes past the end read a valid column
  tws.commit(tw, threadIdx.x);
  fft_seq<N, -1, true, false, kLdsPlain, CN>(v, t, lds, s, CT, tw, 1);
  const ColPtr xc = tiled_col<M, L>(Xh, B * C, bc, c.l);
  __syncthreads();  // every lane is done with the transform's LDS
#pragma unroll
  for (int m = 0; m < EN; ++m) {
    const int k = t + TPSN * m;
    if (k < M / 2 || k >= N - M / 2) {
      const int mrow = k < M / 2 ? k : k - (N - M);
      if (c.ok && jb == 0) xc.p[mrow * xc.stride] = v[m];
      lds[s + mrow * CT] = v[m];
    }
  }
  __syncthreads();
  float2 x[EM];
#pragma unroll
  for (int m = 0; m < EM; ++m) x[m] = lds[s + (tp + TPSM * m) * CT];
  for (int j0 = 0; j0 < JW; j0 += JP) {
    const int jj = j0 + js;
    const bool act = c.ok && jj < JW;
    const int o = ci * J + jb * JW + (jj < JW ? jj : 0);
    const float2 *kcol = K + (long long)o * N * NF + c.l;
    float2 z[EM];
#pragma unroll
    for (int m = 0; m < EM; ++m) z[m] = cmul(x[m], kcol[kept_row<N, M>(tp + TPSM * m) * NF]);
    // the first exchange write waits for every lane's reads of the tile above
    fft_seq<M, +1, true, false, kLdsPlain, CM>(z, tp, lds, js * M * CT + s, CT, tw, N / M);
    if (act) {
      const ColPtr uc = tiled_col<M, L>(U, B * S, b * S + o, c.l);
#pragma unroll
      for (int m = 0; m < EM; ++m) uc.p[(tp + TPSM * m) * uc.stride] = z[m];
    }
  }
}

template <int N, int M, int CT>
constexpr int fwd_cic_lds_elems() {
  constexpr int a = N * CT, b = (ColCfg<N>::TPS / ColCfg<M>::TPS) * M * CT;
  return lds_size<kColLds>(a > b ? a : b);
}

// Geometry of the dK kernel: tiles of 8 columns (there are only S * L columns,
// so narrow tiles keep the grid at hundreds of workgroups) and BP batch groups
// per workgroup, up to 512 threads and at most 8 groups.
constexpr int kGkCT = 8;
// Workgroups the dK launch aims for before it cuts the batch into ranges.
constexpr long long kGkTargetWgs = 512;
// At 512 points the tiles are 4 columns wide, one 256-thread workgroup each (two or more
// per CU instead of one 512-thread workgroup): 2% faster at 8 images of 1024^2 (41.0
// against 41.9 us; 2-column tiles took 45.1).
template <int M>
constexpr int gk_ct() {
  return M == 512 ? 4 : kGkCT;
}
// batch groups per workgroup for CT-column tiles
template <int M, int CT>
constexpr int gk_bp_ct() {
  constexpr int bp = (M == 512 ? 256 : 512) / (CT * ColCfg<M>::TPS);
  return bp < 1 ? 1 : (bp > 8 ? 8 : bp);
}
template <int M>
constexpr int gk_bp() {
  return gk_bp_ct<M, gk_ct<M>()>();
}
// The standalone dK launch at 128 points takes 4-column tiles (eight batch groups) when
// the grid of 8-column tiles, with its batch ranges, would be below this many
// workgroups: at 256^2, 16 images and 8 output channels give 130, and the launch ran
// 9.1 -> 7.0 us with 4 columns.  On the larger grids (32 images at 512^2) and in the
// merged dK/dX launch the 8-column tiles measured faster.
constexpr long long kGkNarrowWgs = 256;

// Backward, dL/dK: for the kernel-gradient columns (o, l), column DFT (M) of each
// upstream-gradient column Tg[b][o] and dK += G conj(Xh[b][o/J]).
// The batch is cut into BG contiguous ranges, one per workgroup of a tile (grid =
// tiles * BG, range index slowest); inside a workgroup, group g of the BP wave
// groups sums b = lo + g, lo + g + BP, ... of its range, and the BP partial sums
// are added in group order, so the result does not depend on scheduling.
// BG = 1: writes all of gK [S][N][N/2+1], the kept bins and exact zeros at the
// rows and columns FDP drops (rows of the tile's own columns; the columns l >= L
// of every row are shared out over the whole grid); with zeros = false the kept bins
// only (the zeros come from an earlier launch).
// BG > 1: writes range r's sums at the kept bins to part [BG][S][M][M/2+1];
// k_gk_reduce then adds the ranges in order and writes gK.
// One workgroup of the dK launch: workgroup `lin` (after the XCD remap) of `nwg`,
// thread `tid`; tw: the twiddle table of an (M * tws)-point transform in LDS.
template <int M, int CT, int BP>
__device__ __forceinline__ void col_bwd_gk_tile(int lin, int nwg, int tid, const float2 *tw, int tws, float2 *lds,
                                                const float2 *__restrict__ Tg, const float2 *__restrict__ Xh,
                                                float2 *__restrict__ gK, float2 *__restrict__ part, int B, int C,
                                                int J, int N, int S, int BG, bool zeros) {
  using CM = ColCfg<M>;
  constexpr int L = M / 2 + 1, TPS = CM::TPS, E = CM::E;
  constexpr int NT = CT * TPS * BP;
  const int s = tid % CT, t = (tid / CT) % TPS, g = tid / (CT * TPS);
  const int tiles = nwg / BG;
  const int range = lin / tiles, wg = lin - range * tiles;
  const int b_lo = range * B / BG, b_hi = (range + 1) * B / BG;
  // the J output channels of one input channel read the same pooled-input columns
  const ColRef c = column_ref<CT>(wg, s, L, S, J);
  const int o = c.plane, ci = o / J;
  const int nf = N / 2 + 1;

  // zeros of the columns l >= L: groups of LW lanes take the S * N rows in turn
  if (BG == 1 && zeros) {
    static_assert((NT & (NT - 1)) == 0, "NT must be a power of two");
    constexpr int LW = NT < 64 ? NT : 64;
    const int lane = tid % LW;
    const long long ngrp = (long long)nwg * (NT / LW);
    for (long long row = ((long long)wg * NT + tid) / LW; row < (long long)S * N; row += ngrp)
      for (int l = L + lane; l < nf; l += LW) gK[row * nf + l] = make_float2(0.f, 0.f);
  }

  float2 acc[E];
#pragma unroll
  for (int m = 0; m < E; ++m) acc[m] = make_float2(0.f, 0.f);
  for (int b0 = b_lo; b0 < b_hi; b0 += BP) {
    const int b = b0 + g;
    const bool act = c.ok && b < b_hi;
    const ColPtr gc = tiled_col<M, L>(Tg, B * S, (act ? b : 0) * S + o, c.l);
    const ColPtr xc = tiled_col<M, L>(Xh, B * C, (act ? b : 0) * C + ci, c.l);
    // loads are unconditional (inactive lanes read a valid column); inactive lanes add nothing
    float2 v[E], xv[E];
#pragma unroll
    for (int m = 0; m < E; ++m) v[m] = gc.p[(t + TPS * m) * gc.stride];
    // the pooled-input column is loaded before the transform so that its loads are
    // all in flight together (up to 8 values per lane: registers allow it)
    if constexpr (E <= 8) {
#pragma unroll
      for (int m = 0; m < E; ++m) xv[m] = xc.p[(t + TPS * m) * xc.stride];
    }
    fft_seq<M, -1, true, false, kLdsPlain, ColCfg<M>>(v, t, lds, g * M * CT + s, CT, tw, tws);
    if constexpr (E > 8) {
#pragma unroll
      for (int m = 0; m < E; ++m) xv[m] = xc.p[(t + TPS * m) * xc.stride];
    }
#pragma unroll
    for (int m = 0; m < E; ++m) {
      const float2 sum = cfmac(acc[m], v[m], xv[m]);
      acc[m] = act ? sum : acc[m];
    }
  }
  if constexpr (BP > 1) {
    __syncthreads();
#pragma unroll
    for (int m = 0; m < E; ++m) lds[lds_phys<kColLds>(g * M * CT + s + (t + TPS * m) * CT)] = acc[m];
    __syncthreads();
    if (g != 0) return;
#pragma unroll
    for (int m = 0; m < E; ++m) {
      float2 sum = lds[lds_phys<kColLds>(s + (t + TPS * m) * CT)];
#pragma unroll
      for (int q = 1; q < BP; ++q) sum = cadd(sum, lds[lds_phys<kColLds>(q * M * CT + s + (t + TPS * m) * CT)]);
      acc[m] = sum;
    }
  }
  if (!c.ok) return;
  if (BG > 1) {
    float2 *pcol = part + ((long long)range * S + o) * M * L + c.l;
#pragma unroll
    for (int m = 0; m < E; ++m) pcol[(long long)(t + TPS * m) * L] = acc[m];
    return;
  }
  float2 *kcol = gK + (long long)o * N * nf + c.l;
#pragma unroll
  for (int m = 0; m < E; ++m) {
    const int mrow = t + TPS * m;
    const int krow = mrow < M / 2 ? mrow : mrow + (N - M);
    kcol[(long long)krow * nf] = acc[m];
  }
  // dropped rows [M/2, N - M/2) of this column; N - M is a multiple of TPS
  if (zeros)
    for (int k = M / 2 + t; k < N - M / 2; k += TPS) kcol[(long long)k * nf] = make_float2(0.f, 0.f);
}

template <int M, int CT, int BP>
__global__ __launch_bounds__(CT *ColCfg<M>::TPS *BP) void k_col_bwd_gk(const float2 *__restrict__ Tg,
                                                                      const float2 *__restrict__ Xh,
                                                                      float2 *__restrict__ gK,
                                                                      float2 *__restrict__ part, int B, int C,
                                                                      int J, int N, int S, int BG, int zeros) {
  float2 *tw = g_lds, *lds = g_lds + twiddle_lds_elems<M>();
  stage_twiddles<M>(tw, threadIdx.x, CT * ColCfg<M>::TPS * BP);
  col_bwd_gk_tile<M, CT, BP>(xcd_remap(blockIdx.x, gridDim.x), gridDim.x, threadIdx.x, tw, 1, lds, Tg, Xh, gK, part,
                             B, C, J, N, S, BG, zeros != 0);
}

// gK [S][N][N/2+1] from BG partial sums part [BG][S][M][M/2+1] (plain layout), for
// one or two reductions (grid.y selects the GkSum): a thread per gK element, its BG
// partial sums loaded together (16 at a time) and added in order at the kept bins,
// exact zeros elsewhere.  Consecutive threads take consecutive bins of a row.
// kept != 0: a thread per kept bin only, the other bins of gK left as they are.
struct GkSum {
  const float2 *part;
  float2 *gK;
  int BG, S, M, N, kept;
};

constexpr int kGkReduceThreads = 256;

__global__ __launch_bounds__(kGkReduceThreads) void k_gk_reduce(GkSum d0, GkSum d1) {
  const GkSum d = blockIdx.y == 0 ? d0 : d1;
  const int L = d.M / 2 + 1, nf = d.N / 2 + 1;
  // 32-bit element arithmetic: the launchers keep S * N * (N/2+1) below 2^31
  const unsigned total = (unsigned)(d.kept ? d.S * d.M * L : d.S * d.N * nf);
  const long long range_stride = (long long)d.S * d.M * L;
  for (unsigned i = blockIdx.x * kGkReduceThreads + threadIdx.x; i < total; i += gridDim.x * kGkReduceThreads) {
    int o, mrow, l, krow;
    if (d.kept) {
      const int r = (int)(i / (unsigned)L);
      l = (int)i - r * L;
      o = r / d.M;
      mrow = r - o * d.M;
      krow = mrow < d.M / 2 ? mrow : mrow + (d.N - d.M);
    } else {
      const int r = (int)(i / (unsigned)nf);
      l = (int)i - r * nf;
      o = r / d.N;
      krow = r - o * d.N;
      mrow = krow < d.M / 2 ? krow : (krow >= d.N - d.M / 2 ? krow - (d.N - d.M) : -1);
    }
    float2 v = make_float2(0.f, 0.f);
    if (mrow >= 0 && l < L) {
      const float2 *src = d.part + ((long long)o * d.M + mrow) * L + l;
      int q = 0;
      for (; q + 16 <= d.BG; q += 16) {
        float2 a[16];
#pragma unroll
        for (int u = 0; u < 16; ++u) a[u] = src[(q + u) * range_stride];
#pragma unroll
        for (int u = 0; u < 16; ++u) v = cadd(v, a[u]);
      }
      for (; q + 4 <= d.BG; q += 4) {
        float2 a[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) a[u] = src[(q + u) * range_stride];
#pragma unroll
        for (int u = 0; u < 4; ++u) v = cadd(v, a[u]);
      }
      for (; q < d.BG; ++q) v = cadd(v, src[q * range_stride]);
    }
    d.gK[((long long)o * d.N + krow) * nf + l] = v;
  }
}

static long long gk_reduce_items(const GkSum &d) {
  return d.kept ? (long long)d.S * d.M * (d.M / 2 + 1) : (long long)d.S * d.N * (d.N / 2 + 1);
}

static hipError_t gk_reduce(const GkSum &d0, const GkSum *d1, hipStream_t s) {
  long long total = gk_reduce_items(d0);
  if (d1) total = std::max(total, gk_reduce_items(*d1));
  const unsigned gx = (unsigned)std::min<long long>((total + kGkReduceThreads - 1) / kGkReduceThreads, 1 << 16);
  const char *nm = "gk_reduce";
  return timed_launch(nm, k_gk_reduce, dim3(gx, d1 ? 2 : 1), dim3(kGkReduceThreads), 0, s, d0, d1 ? *d1 : d0);
}

template <int N, int M>
constexpr int cic_jp() {
  return ColCfg<N>::TPS / ColCfg<M>::TPS;
}

template <int N, int M, int CT>
constexpr int cic_lds_elems() {
  constexpr int a = N * CT, b = cic_jp<N, M>() * M * CT;
  return lds_size<kColLds>(a > b ? a : b);
}

// Backward, dL/dx: for the columns (b, c, l), column DFTs (M) of the J
// upstream-gradient columns Tg[b][cJ+j], dXh = sum_j G conj(K[cJ+j]) at the kept
// bins, FDP adjoint (zero rows at the dropped frequencies), inverse column DFT (N).
// The thread layout of the N-point transform holds JP = TPS_N / TPS_M groups of
// the M-point layout, which take the J products in turns.
// One tile of the dX launch: tile `lin` (after the XCD remap), thread `tid`; tw: the
// N-point twiddle table in LDS.  With valid = false the tile runs (every barrier is
// reached) but stores nothing.
template <int N, int M, int CT>
__device__ __forceinline__ void col_bwd_gx_tile(int lin, bool valid, int tid, const float2 *tw, float2 *lds,
                                                const float2 *__restrict__ Tg, const float2 *__restrict__ K,
                                                float2 *__restrict__ V, int C, int J, int planes) {
  using CN = ColCfg<N>;
  using CM = ColCfg<M>;
  constexpr int L = M / 2 + 1, NF = N / 2 + 1;
  constexpr int TPSN = CN::TPS, TPSM = CM::TPS, JP = cic_jp<N, M>();
  static_assert(JP * TPSM == TPSN, "thread layouts of the two transforms must nest");
  const int s = tid % CT, t = tid / CT;
  const int tp = t % TPSM, js = t / TPSM;
  // plane index ci * B + b: the B images read the same kernel columns
  ColRef c = column_ref<CT>(lin, s, L, planes, planes / C);
  c.ok = c.ok && valid;
  const int B = planes / C;
  const int ci = c.plane / B;
  const int b = c.plane - ci * B;
  const int S = C * J;

  float2 acc[CM::E];
#pragma unroll
  for (int m = 0; m < CM::E; ++m) acc[m] = make_float2(0.f, 0.f);
  for (int j0 = 0; j0 < J; j0 += JP) {
    const int j = j0 + js;
    const bool act = c.ok && j < J;
    const int o = ci * J + (act ? j : 0);
    const ColPtr gc = tiled_col<M, L>(Tg, planes * J, b * S + o, c.l);
    const float2 *kcol = K + (long long)o * N * NF + c.l;
    // loads are unconditional (inactive lanes read a valid column); inactive lanes add nothing
    float2 g[CM::E], kv[CM::E];
#pragma unroll
    for (int m = 0; m < CM::E; ++m) g[m] = gc.p[(tp + TPSM * m) * gc.stride];
    // the kernel column is loaded before the transform (up to 8 values per lane)
    if constexpr (CM::E <= 8) {
#pragma unroll
      for (int m = 0; m < CM::E; ++m) kv[m] = kcol[(long long)kept_row<N, M>(tp + TPSM * m) * NF];
    }
    fft_seq<M, -1, true, false, kLdsPlain, ColCfg<M>>(g, tp, lds, js * M * CT + s, CT, tw, N / M);
    if constexpr (CM::E > 8) {
#pragma unroll
      for (int m = 0; m < CM::E; ++m) kv[m] = kcol[(long long)kept_row<N, M>(tp + TPSM * m) * NF];
    }
#pragma unroll
    for (int m = 0; m < CM::E; ++m) {
      const float2 sum = cfmac(acc[m], g[m], kv[m]);
      acc[m] = act ? sum : acc[m];
    }
  }
  // sum the JP partial sums and scatter the pooled rows into the n-row column (FDP adjoint)
  __syncthreads();
#pragma unroll
  for (int m = 0; m < CM::E; ++m) lds[lds_phys<kColLds>(js * M * CT + s + (tp + TPSM * m) * CT)] = acc[m];
  __syncthreads();
  float2 w[CN::E];
#pragma unroll
  for (int m = 0; m < CN::E; ++m) {
    const int k = t + TPSN * m;
    float2 sum = make_float2(0.f, 0.f);
    if (k < M / 2 || k >= N - M / 2) {
      const int mrow = k < M / 2 ? k : k - (N - M);
#pragma unroll
      for (int q = 0; q < JP; ++q) sum = cadd(sum, lds[lds_phys<kColLds>(q * M * CT + s + mrow * CT)]);
    }
    w[m] = sum;
  }
  fft_seq<N, +1, true, false, kLdsPlain, ColCfg<N>>(w, t, lds, s, CT, tw, 1);
  if (!c.ok) return;
  const ColPtr vc = tiled_col<N, L>(V, planes, b * C + ci, c.l);
#pragma unroll
  for (int m = 0; m < CN::E; ++m) vc.p[(t + TPSN * m) * vc.stride] = w[m];
}

template <int N, int M, int CT>
__global__ __launch_bounds__(CT *ColCfg<N>::TPS) void k_col_bwd_gx(const float2 *__restrict__ Tg,
                                                                  const float2 *__restrict__ K,
                                                                  float2 *__restrict__ V, int C, int J,
                                                                  int planes) {
  float2 *tw = g_lds, *lds = g_lds + twiddle_lds_elems<N>();
  stage_twiddles<N>(tw, threadIdx.x, CT * ColCfg<N>::TPS);
  col_bwd_gx_tile<N, M, CT>(xcd_remap(blockIdx.x, gridDim.x), true, threadIdx.x, tw, lds, Tg, K, V, C, J, planes);
}

// dK and dX of one layer in one launch (they are independent; both read Tg): the
// first nk workgroups (nk_used of them real, nk a multiple of 8 so the XCD numbering
// of the rest stays aligned) run dK tiles of CTK columns; the others each run PACK
// dX tiles of CTX columns side by side, PACK = dK threads / dX threads.
template <int N, int M, int CTK, int BP, int CTX>
__global__ __launch_bounds__(CTK *ColCfg<M>::TPS *BP) void k_col_bwd_dk_dx(
    const float2 *__restrict__ Tg, const float2 *__restrict__ Xh, const float2 *__restrict__ K,
    float2 *__restrict__ gK, float2 *__restrict__ V, int B, int C, int J, int S, int nk, int nk_used, int nx_tiles,
    int zeros) {
  constexpr int NT = CTK * ColCfg<M>::TPS * BP, NX = CTX * ColCfg<N>::TPS, PACK = NT / NX;
  static_assert(PACK >= 1 && PACK * NX == NT, "dX tiles must pack the dK workgroup exactly");
  float2 *tw = g_lds, *lds = g_lds + twiddle_lds_elems<N>();
  stage_twiddles<N>(tw, threadIdx.x, NT);
  const int bid = blockIdx.x;
  if (bid < nk) {
    if (bid >= nk_used) return;  // padding: no barrier follows
    col_bwd_gk_tile<M, CTK, BP>(xcd_remap(bid, nk_used), nk_used, threadIdx.x, tw, N / M, lds, Tg, Xh, gK,
                                nullptr, B, C, J, N, S, 1, zeros != 0);
    return;
  }
  const int xb = bid - nk, nxb = gridDim.x - nk;
  const int sub = threadIdx.x / NX;
  const int tile = xcd_remap(xb, nxb) * PACK + sub;
  const bool valid = tile < nx_tiles;
  col_bwd_gx_tile<N, M, CTX>(valid ? tile : nx_tiles - 1, valid, threadIdx.x - sub * NX, tw,
                             lds + sub * cic_lds_elems<N, M, CTX>(), Tg, K, V, C, J, B * C);
}

// ---------------------------------------------------------------------------
// spectral CIC and FDP (standalone ops)
// ---------------------------------------------------------------------------
__global__ void k_cic_fwd(const float2 *__restrict__ X, const float2 *__restrict__ K, float2 *__restrict__ Y,
                          int C, int J, long long P, long long total) {
  const int S = C * J;
  for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (long long)gridDim.x * blockDim.x) {
    const long long p = i % P, bo = i / P;
    const int o = (int)(bo % S);
    const long long b = bo / S;
    Y[i] = cmul(X[(b * C + o / J) * P + p], K[(long long)o * P + p]);
  }
}

__global__ void k_cic_bwd_gx(const float2 *__restrict__ gY, const float2 *__restrict__ K, float2 *__restrict__ gX,
                             int C, int J, long long P, long long total) {
  const int S = C * J;
  for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (long long)gridDim.x * blockDim.x) {
    const long long p = i % P, bc = i / P;
    const int c = (int)(bc % C);
    const long long b = bc / C;
    float2 acc = make_float2(0.f, 0.f);
    for (int j = 0; j < J; ++j) {
      const int o = c * J + j;
      acc = cfmac(acc, gY[(b * S + o) * P + p], K[(long long)o * P + p]);
    }
    gX[i] = acc;
  }
}

__global__ void k_cic_bwd_gk(const float2 *__restrict__ gY, const float2 *__restrict__ X, float2 *__restrict__ gK,
                             int B, int C, int J, long long P, long long total) {
  const int S = C * J;
  for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (long long)gridDim.x * blockDim.x) {
    const long long p = i % P;
    const int o = (int)(i / P);
    const int c = o / J;
    float2 acc = make_float2(0.f, 0.f);
    for (int b = 0; b < B; ++b) acc = cfmac(acc, gY[((long long)b * S + o) * P + p], X[((long long)b * C + c) * P + p]);
    gK[i] = acc;
  }
}

__global__ void k_fdp_gather(const float2 *__restrict__ X, float2 *__restrict__ Y, long long total, int H, int Wf,
                             int Mh, int Mwf) {
  for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (long long)gridDim.x * blockDim.x) {
    const int l = (int)(i % Mwf);
    const long long pm = i / Mwf;
    const int m = (int)(pm % Mh);
    const long long p = pm / Mh;
    const int k = m < Mh / 2 ? m : m + (H - Mh);
    Y[i] = X[(p * H + k) * Wf + l];
  }
}

__global__ void k_fdp_scatter(const float2 *__restrict__ gY, float2 *__restrict__ gX, long long total, int H,
                              int Wf, int Mh, int Mwf) {
  for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (long long)gridDim.x * blockDim.x) {
    const int l = (int)(i % Wf);
    const long long pk = i / Wf;
    const int k = (int)(pk % H);
    const long long p = pk / H;
    const bool kept = l < Mwf && (k < Mh / 2 || k >= H - Mh / 2);
    const int m = k < Mh / 2 ? k : k - (H - Mh);
    gX[i] = kept ? gY[(p * Mh + m) * Mwf + l] : make_float2(0.f, 0.f);
  }
}

// ---------------------------------------------------------------------------
// host side: size dispatch and launchers
// ---------------------------------------------------------------------------
template <class F>
static bool dispatch_n(int n, F &&f) {
  switch (n) {
#define FDC_CASE(V)                          \
  case V:                                    \
    f(std::integral_constant<int, V>{});     \
    return true;
    FDC_CASE(2) FDC_CASE(4) FDC_CASE(8) FDC_CASE(16) FDC_CASE(32) FDC_CASE(64) FDC_CASE(128) FDC_CASE(256)
    FDC_CASE(512) FDC_CASE(1024) FDC_CASE(224)
#undef FDC_CASE
    default:
      return false;
  }
}

// (n, m) pairs of the fused CIC kernels: m = n, n/2 or n/4 (powers of two), or 224 -> 224.
template <class F>
static bool dispatch_nm(int n, int m, F &&f) {
  bool found = false;
  dispatch_n(n, [&](auto nc) {
    constexpr int N = decltype(nc)::value;
    if (m == N) {
      found = true;
      f(nc, nc);
      return;
    }
    if constexpr (N != 224 && N >= 4) {
      if (m == N / 2) {
        found = true;
        f(nc, std::integral_constant<int, N / 2>{});
        return;
      }
    }
    if constexpr (N != 224 && N >= 8) {
      if (m == N / 4) {
        found = true;
        f(nc, std::integral_constant<int, N / 4>{});
        return;
      }
    }
  });
  return found;
}

bool size_supported(int n) {
  return dispatch_n(n, [](auto) {});
}

bool cic_pair_supported(int n, int m) {
  return dispatch_nm(n, m, [](auto, auto) {});
}

template <class Kern, class... Args>
static hipError_t launch(const char *name, Kern kern, unsigned grid, unsigned block, size_t lds, hipStream_t s,
                         Args... args) {
  if (grid == 0) return hipSuccess;
  return timed_launch(name, kern, dim3(grid), dim3(block), lds, s, args...);
}

static unsigned grid_stride_blocks(long long total, int block) {
  long long g = (total + block - 1) / block;
  if (g > 1048576) g = 1048576;
  return (unsigned)(g > 0 ? g : 0);
}

hipError_t launch_row_r2c(int n, const float *x, SpecLayout out, long long planes, int rows_per_plane,
                          ImgView in_view, long long in_plane_stride, int L, float alpha, float beta, hipStream_t s) {
  hipError_t err = hipErrorInvalidValue;
  if (planes * rows_per_plane >= (1LL << 31)) return err;
  dispatch_n(n, [&](auto nc) {
    constexpr int N = decltype(nc)::value;
    constexpr int SPW = row_spw<N>();
    const long long npairs = planes * rows_per_plane / 2;
    const unsigned grid = (unsigned)((npairs + SPW - 1) / SPW);
    const size_t lds = (twiddle_lds_elems<N>() + lds_size<kRowLds>(SPW * N)) * sizeof(float2);
    static const std::string nm = "row_r2c_" + std::to_string(N);
    switch (in_view.mode) {
      case 0:
        err = launch(nm.c_str(), k_row_r2c<N, SPW, 0>, grid, SPW * RowCfg<N>::TPS, lds, s, x, out, npairs,
                     rows_per_plane, in_view, in_plane_stride, L, alpha, beta);
        break;
      case 1:
        err = launch(nm.c_str(), k_row_r2c<N, SPW, 1>, grid, SPW * RowCfg<N>::TPS, lds, s, x, out, npairs,
                     rows_per_plane, in_view, in_plane_stride, L, alpha, beta);
        break;
      default:
        err = launch(nm.c_str(), k_row_r2c<N, SPW, 2>, grid, SPW * RowCfg<N>::TPS, lds, s, x, out, npairs,
                     rows_per_plane, in_view, in_plane_stride, L, alpha, beta);
    }
  });
  return err;
}

hipError_t launch_row_c2r(int n, SpecLayout in, float *y, long long planes, int rows_per_plane, int L, float alpha,
                          float beta, ImgView out_view, long long out_plane_stride, hipStream_t s) {
  hipError_t err = hipErrorInvalidValue;
  if (planes * rows_per_plane >= (1LL << 31)) return err;
  dispatch_n(n, [&](auto nc) {
    constexpr int N = decltype(nc)::value;
    constexpr int SPW = row_spw<N>();
    const long long npairs = planes * rows_per_plane / 2;
    const unsigned grid = (unsigned)((npairs + SPW - 1) / SPW);
    const size_t lds = (twiddle_lds_elems<N>() + lds_size<kRowLds>(SPW * N)) * sizeof(float2);
    static const std::string nm = "row_c2r_" + std::to_string(N);
    auto go = [&](auto kern) {
      err = launch(nm.c_str(), kern, grid, SPW * RowCfg<N>::TPS, lds, s, in, y, npairs, rows_per_plane, L, alpha,
                   beta, out_view, out_plane_stride);
    };
    switch (out_view.mode) {
      case 0:
        switch (c2r_lin_mode<N>(L, beta)) {
          case 1:
            if constexpr (RowCfg<N>::E % 2 == 0) go(k_row_c2r<N, SPW, 0, 1>);
            break;
          case 2:
            if constexpr (RowCfg<N>::E % 4 == 0) go(k_row_c2r<N, SPW, 0, 2>);
            break;
          default: go(k_row_c2r<N, SPW, 0, 0>);
        }
        break;
      case 1: go(k_row_c2r<N, SPW, 1, 0>); break;
      default: go(k_row_c2r<N, SPW, 2, 0>);
    }
  });
  return err;
}

hipError_t launch_row_c2r_r2c(int n, SpecLayout in, int Lin, float a1, float b1, SpecLayout out, int Lout, float a2,
                              float b2, long long planes, int rows_per_plane, hipStream_t s, ZeroBins zeros) {
  hipError_t err = hipErrorInvalidValue;
  if (planes * rows_per_plane >= (1LL << 31)) return err;
  dispatch_n(n, [&](auto nc) {
    constexpr int N = decltype(nc)::value;
    constexpr int SPW = row_spw<N>();
    const long long npairs = planes * rows_per_plane / 2;
    const unsigned grid = (unsigned)((npairs + SPW - 1) / SPW);
    const size_t lds = (twiddle_lds_elems<N>() + lds_size<kRowLds>(SPW * N)) * sizeof(float2);
    static const std::string nm = "row_c2r_r2c_" + std::to_string(N);
    auto go = [&](auto kern) {
      err = launch(nm.c_str(), kern, grid, SPW * RowCfg<N>::TPS, lds, s, in, Lin, a1, b1, out, Lout, a2, b2, npairs,
                   rows_per_plane, zeros);
    };
    switch (c2r_lin_mode<N>(Lin, b1)) {
      case 1:
        if constexpr (RowCfg<N>::E % 2 == 0) go(k_row_c2r_r2c<N, SPW, 1>);
        break;
      case 2:
        if constexpr (RowCfg<N>::E % 4 == 0) go(k_row_c2r_r2c<N, SPW, 2>);
        break;
      default: go(k_row_c2r_r2c<N, SPW, 0>);
    }
  });
  return err;
}

// Grid of a column launch; 0 (nothing launched, error reported) when the tile or
// column count does not fit the kernels' 32-bit tile arithmetic.
static unsigned col_grid(long long planes, int L, int ct) {
  const long long t = col_tile_count(planes, L, ct);
  return (planes * L >= (1LL << 31) || t >= (1LL << 31)) ? 0u : (unsigned)t;
}

hipError_t launch_col_fft(int n, int dir, const float2 *in, float2 *out, long long planes, int L, int ld,
                          long long in_plane_stride, long long out_plane_stride, hipStream_t s, int keep) {
  hipError_t err = hipErrorInvalidValue;
  dispatch_n(n, [&](auto nc) {
    constexpr int N = decltype(nc)::value;
    constexpr int CT = col_ct<N>();
    const size_t lds = (twiddle_lds_elems<N>() + lds_size<kColLds>(N * CT)) * sizeof(float2);
    const unsigned grid = col_grid(planes, L, CT);
    if (grid == 0) return;
    static const std::string nf = "col_fft_fwd_" + std::to_string(N);
    static const std::string ni = "col_fft_inv_" + std::to_string(N);
    if (dir < 0)
      err = launch(nf.c_str(), k_col_fft<N, CT, -1>, grid, CT * ColCfg<N>::TPS, lds, s, in, out, L, ld, (int)planes,
                   in_plane_stride, out_plane_stride, keep > 0 ? keep : N);
    else
      err = launch(ni.c_str(), k_col_fft<N, CT, +1>, grid, CT * ColCfg<N>::TPS, lds, s, in, out, L, ld, (int)planes,
                   in_plane_stride, out_plane_stride, keep > 0 ? keep : N);
  });
  return err;
}

hipError_t launch_col_fft_keep(int n, SpecLayout in, float2 *out, long long planes, int L, int ld, int keep,
                               hipStream_t s) {
  hipError_t err = hipErrorInvalidValue;
  dispatch_n(n, [&](auto nc) {
    constexpr int N = decltype(nc)::value;
    constexpr int CT = col_ct_crop<N>();
    const size_t lds = (twiddle_lds_elems<N>() + lds_size<kColLds>(N * CT)) * sizeof(float2);
    const unsigned grid = col_grid(planes, L, CT);
    if (grid == 0) return;
    static const std::string nm = "col_fft_keep_" + std::to_string(N);
    err = launch(nm.c_str(), k_col_fft_keep<N, CT>, grid, CT * ColCfg<N>::TPS, lds, s, in, out, L, ld, (int)planes,
                 (long long)N * ld, keep);
  });
  return err;
}

hipError_t launch_col_fft_split(int n, int dir, SpecLayout in, SpecLayout out, long long planes, hipStream_t s) {
  hipError_t err = hipErrorInvalidValue;
  dispatch_n(n, [&](auto nc) {
    constexpr int N = decltype(nc)::value;
    constexpr int L = N / 2 + 1;
    constexpr int CT = col_ct_for(col_ct_split<N>(), L);
    const size_t lds = (twiddle_lds_elems<N>() + lds_size<kColLds>(N * CT)) * sizeof(float2);
    const unsigned grid = col_grid(planes, L, CT);
    if (grid == 0) return;
    static const std::string nf = "col_fft_fwd_" + std::to_string(N);
    static const std::string ni = "col_fft_inv_" + std::to_string(N);
    if (dir < 0)
      err = launch(nf.c_str(), k_col_fft_split<N, CT, -1>, grid, CT * ColCfg<N>::TPS, lds, s, in, out, (int)planes);
    else
      err = launch(ni.c_str(), k_col_fft_split<N, CT, +1>, grid, CT * ColCfg<N>::TPS, lds, s, in, out, (int)planes);
  });
  return err;
}

// Output channels per workgroup of the fused forward column kernel for J output
// channels per input channel and n-point columns (0: not fused, the crop and CIC
// inverse kernels run instead).  J = 8 at n <= 256 is split into two groups of four,
// each of which transforms the input column itself: at 256 points that costs less than
// storing the pooled spectrum and reading it back (the 256^2 stack 0.0797 -> 0.0771 ms);
// at 512 and 1024 points it measured slower (0.3051 -> 0.3087 ms) or the same.
int fwd_cic_jw(int J, int n) { return (J == 1 || J == 2 || J == 4) ? J : ((J == 8 && n <= 256) ? 4 : 0); }

hipError_t launch_col_fwd_cic(int n, int m, const float2 *T, const float2 *K, float2 *U, float2 *Xh, int B,
                              int C, int S, hipStream_t s) {
  hipError_t err = hipErrorInvalidValue;
  dispatch_nm(n, m, [&](auto nc, auto mc) {
    constexpr int N = decltype(nc)::value, M = decltype(mc)::value;
    constexpr int L = M / 2 + 1;
    constexpr int CTN = col_ct_for(col_ct_crop<N>(), L), CTM = col_ct_for(col_ct_cic<M>(), L);
    static const std::string n1 = "col_fwd_crop_" + std::to_string(N) + "_" + std::to_string(M);
    static const std::string n2 = "col_cic_inv_" + std::to_string(N) + "_" + std::to_string(M);
    static const std::string n3 = "col_fwd_cic_" + std::to_string(N) + "_" + std::to_string(M);
    const int J = S / C, jwf = fwd_cic_jw(J, N);
    if (jwf > 0) {
      // both halves in one kernel: jwf output channels per workgroup
      const int jb = J / jwf;
      const unsigned g = col_grid((long long)B * C * jb, L, CTN);
      if (g == 0) return;
      const size_t lds = (twiddle_lds_elems<N>() + fwd_cic_lds_elems<N, M, CTN>()) * sizeof(float2);
      auto go = [&](auto kern) {
        err = launch(n3.c_str(), kern, g, CTN * ColCfg<N>::TPS, lds, s, T, K, U, Xh, B, C, jb);
      };
      switch (jwf) {
        case 4: go(k_col_fwd_cic<N, M, CTN, 4>); break;
        case 2: go(k_col_fwd_cic<N, M, CTN, 2>); break;
        default: go(k_col_fwd_cic<N, M, CTN, 1>);
      }
      return;
    }
    const unsigned g1 = col_grid((long long)B * C, L, CTN);
    if (g1 == 0) return;
    err = launch(n1.c_str(), k_col_fwd_crop<N, M, CTN>, g1, CTN * ColCfg<N>::TPS, (twiddle_lds_elems<N>() + lds_size<kColLds>(N * CTN)) * sizeof(float2),
                 s, T, Xh, B * C);
    if (err != hipSuccess) return;
    const int jw = J % kCicJW == 0 ? kCicJW : (J % 4 == 0 && kCicJW >= 4 ? 4 : (J % 2 == 0 && kCicJW >= 2 ? 2 : 1));
    const long long groups = (long long)B * C * (J / jw);
    const unsigned g2 = col_grid(groups, L, CTM);
    if (g2 == 0) {
      err = hipErrorInvalidValue;
      return;
    }
    const size_t lds2 = (twiddle_lds_elems<M>() + lds_size<kColLds>(M * CTM)) * sizeof(float2);
    auto go = [&](auto kern) {
      err = launch(n2.c_str(), kern, g2, CTM * ColCfg<M>::TPS, lds2, s, Xh, K, U, B, C, J, (int)groups);
    };
    // Few planes (a small batch at the first layer): 8-column tiles, up to four times the
    // workgroups, when the default tiles would leave most compute units idle.
    constexpr int CTS = 8;
    if (CTS < CTM && jw == kCicJW && g2 < kCicNarrowGrid) {
      const unsigned g3 = col_grid(groups, L, CTS);
      const size_t lds3 = (twiddle_lds_elems<M>() + lds_size<kColLds>(M * CTS)) * sizeof(float2);
      err = launch(n2.c_str(), k_col_cic_inv<N, M, CTS, kCicJW>, g3, CTS * ColCfg<M>::TPS, lds3, s, Xh, K, U, B, C, J,
                   (int)groups);
      return;
    }
    switch (jw) {
      case 8: go(k_col_cic_inv<N, M, CTM, 8>); break;
      case 4: go(k_col_cic_inv<N, M, CTM, 4>); break;
      case 2: go(k_col_cic_inv<N, M, CTM, 2>); break;
      default: go(k_col_cic_inv<N, M, CTM, 1>);
    }
  });
  return err;
}

// Batch ranges of the dK launch at M points with CT-column tiles.
template <int M, int CT>
static int gk_ranges_ct(int B, int S, long long part_elems) {
  constexpr int L = M / 2 + 1, BP = gk_bp_ct<M, CT>();
  const long long tiles = col_tile_count(S, L, CT);
  // enough workgroups to fill the chip (kGkTargetWgs), at least BP batch entries per
  // range, and range sums (written and read once more) of at most a quarter of Tg
  // (at 8 images, two ranges measured slower than one)
  long long want = (kGkTargetWgs + tiles - 1) / tiles;
  want = std::min<long long>(want, std::max(1, B / 8));
  want = std::min<long long>(want, std::max(1, B / BP));
  const long long per = (long long)S * M * L;
  want = std::min<long long>(want, per > 0 ? part_elems / per : 1);
  if (tiles * want >= (1LL << 31)) want = 1;
  return (int)std::max<long long>(1, want);
}

// Whether the standalone dK launch at M points takes 4-column tiles (kGkNarrowWgs).
template <int M>
static bool gk_narrow(int B, int S, long long part_elems) {
  if constexpr (M != 128) {
    return false;
  } else {
    constexpr int L = M / 2 + 1, CT = col_ct_for(gk_ct<M>(), L);
    return col_tile_count(S, L, CT) * gk_ranges_ct<M, CT>(B, S, part_elems) < kGkNarrowWgs;
  }
}

int gk_batch_ranges(int n, int m, int B, int S, long long part_elems) {
  int bg = 1;
  dispatch_n(m, [&](auto mc) {
    constexpr int M = decltype(mc)::value;
    constexpr int L = M / 2 + 1;
    constexpr int CT = col_ct_for(gk_ct<M>(), L), CT4 = col_ct_for(4, L);
    bg = gk_narrow<M>(B, S, part_elems) ? gk_ranges_ct<M, CT4>(B, S, part_elems)
                                        : gk_ranges_ct<M, CT>(B, S, part_elems);
  });
  (void)n;
  return bg;
}

hipError_t launch_col_bwd_gk(int n, int m, const float2 *Tg, const float2 *Xh, float2 *gK, int B, int C, int S,
                             float2 *part, long long part_elems, hipStream_t s, bool zeros) {
  hipError_t err = hipErrorInvalidValue;
  if (!cic_pair_supported(n, m)) return err;
  const long long pe = part ? part_elems : 0;
  const int BG = part ? gk_batch_ranges(n, m, B, S, part_elems) : 1;
  dispatch_n(m, [&](auto mc) {
    constexpr int M = decltype(mc)::value;
    constexpr int L = M / 2 + 1;
    static const std::string nm = "col_bwd_gk_" + std::to_string(M);
    auto go = [&](auto ctc) {
      constexpr int CT = decltype(ctc)::value, BP = gk_bp_ct<M, CT>();
      const size_t lds = (twiddle_lds_elems<M>() + lds_size<kColLds>(BP * M * CT)) * sizeof(float2);
      const unsigned tiles = col_grid(S, L, CT);
      if (tiles == 0) return;
      err = launch(nm.c_str(), k_col_bwd_gk<M, CT, BP>, tiles * (unsigned)BG, CT * ColCfg<M>::TPS * BP, lds, s, Tg,
                   Xh, gK, part, B, C, S / C, n, S, BG, zeros ? 1 : 0);
    };
    if (gk_narrow<M>(B, S, pe))
      go(std::integral_constant<int, col_ct_for(4, L)>{});
    else
      go(std::integral_constant<int, col_ct_for(gk_ct<M>(), L)>{});
    if (err != hipSuccess || BG == 1) return;
    err = gk_reduce(GkSum{part, gK, BG, S, M, n, zeros ? 0 : 1}, nullptr, s);
  });
  return err;
}

hipError_t launch_gk_reduce2(const float2 *part0, float2 *gK0, int S0, int M0, int N0, const float2 *part1,
                             float2 *gK1, int S1, int M1, int N1, int BG, hipStream_t s, bool zeros) {
  const int kept = zeros ? 0 : 1;
  const GkSum d1{part1, gK1, BG, S1, M1, N1, kept};
  return gk_reduce(GkSum{part0, gK0, BG, S0, M0, N0, kept}, part1 ? &d1 : nullptr, s);
}

hipError_t launch_col_bwd_dk_dx(int n, int m, const float2 *Tg, const float2 *Xh, const float2 *K, float2 *gK,
                                float2 *V, int B, int C, int S, hipStream_t s, bool zeros) {
  hipError_t err = hipErrorInvalidValue;
  if (!cic_pair_supported(n, m)) return err;
  dispatch_nm(n, m, [&](auto nc, auto mc) {
    constexpr int N = decltype(nc)::value, M = decltype(mc)::value;
    constexpr int L = M / 2 + 1;
    constexpr int CTK = col_ct_for(gk_ct<M>(), L), BP = gk_bp<M>(), CTX = col_ct_for(col_ct_gx<N>(), L);
    constexpr int NT = CTK * ColCfg<M>::TPS * BP, NX = CTX * ColCfg<N>::TPS;
    if constexpr (NX <= NT && NT % NX == 0) {
      constexpr int PACK = NT / NX;
      const unsigned nk_used = col_grid(S, L, CTK), nx_tiles = col_grid((long long)B * C, L, CTX);
      if (nk_used == 0 || nx_tiles == 0) return;
      const unsigned nk = (nk_used + 7) & ~7u, nxb = (nx_tiles + PACK - 1) / PACK;
      const long long gk_lds = lds_size<kColLds>(BP * M * CTK), gx_lds = (long long)PACK * cic_lds_elems<N, M, CTX>();
      const size_t lds = (twiddle_lds_elems<N>() + (gk_lds > gx_lds ? gk_lds : gx_lds)) * sizeof(float2);
      static const std::string nm = "col_bwd_dk_dx_" + std::to_string(N) + "_" + std::to_string(M);
      err = launch(nm.c_str(), k_col_bwd_dk_dx<N, M, CTK, BP, CTX>, nk + nxb, NT, lds, s, Tg, Xh, K, gK, V, B, C,
                   S / C, S, (int)nk, (int)nk_used, (int)nx_tiles, zeros ? 1 : 0);
    }
  });
  return err;
}

bool col_bwd_dk_dx_supported(int n, int m) {
  // measured: one launch helps the small layers (64 -> 32: 13 -> 9 us) and costs at
  // 512 -> 256 (49 -> 53 us), where both kernels already fill the chip
  if (n > 256) return false;
  bool ok = false;
  dispatch_nm(n, m, [&](auto nc, auto mc) {
    constexpr int N = decltype(nc)::value, M = decltype(mc)::value;
    constexpr int L = M / 2 + 1;
    constexpr int CTK = col_ct_for(gk_ct<M>(), L), BP = gk_bp<M>(), CTX = col_ct_for(col_ct_gx<N>(), L);
    constexpr int NT = CTK * ColCfg<M>::TPS * BP, NX = CTX * ColCfg<N>::TPS;
    ok = NX <= NT && NT % NX == 0;
  });
  return ok;
}

hipError_t launch_col_bwd_gx(int n, int m, const float2 *Tg, const float2 *K, float2 *V, int B, int C, int S,
                             hipStream_t s) {
  hipError_t err = hipErrorInvalidValue;
  dispatch_nm(n, m, [&](auto nc, auto mc) {
    constexpr int N = decltype(nc)::value, M = decltype(mc)::value;
    constexpr int L = M / 2 + 1;
    constexpr int CT = col_ct_for(col_ct_gx<N>(), L);
    const size_t lds = (twiddle_lds_elems<N>() + cic_lds_elems<N, M, CT>()) * sizeof(float2);
    const unsigned grid = col_grid((long long)B * C, L, CT);
    if (grid == 0) return;
    static const std::string nm = "col_bwd_gx_" + std::to_string(N) + "_" + std::to_string(M);
    err = launch(nm.c_str(), k_col_bwd_gx<N, M, CT>, grid, CT * ColCfg<N>::TPS, lds, s, Tg, K, V, C, S / C,
                 B * C);
  });
  return err;
}

// e / d and e mod d for 0 <= e < 2^24, d >= 1: a float estimate corrected by one step.
__device__ __forceinline__ int div_small(int e, int d, float rd, int &rem) {
  int q = (int)((float)e * rd);
  int r = e - q * d;
  if (r < 0) q -= 1, r += d;
  if (r >= d) q += 1, r -= d;
  rem = r;
  return q;
}

// k_cic_fdp_fwd and the dX blocks of k_cic_fdp_bwd give each thread two consecutive bins (e0,
// e0 + 1), e0 even, of the plane they write: a plane holds an even number of bins (its
// row count is even), so the pair is one 16-byte store (the launchers check that the
// output is 16-byte aligned); the pair may straddle two rows, and inputs are read bin
// by bin.  (Two bins per lane also for the loads, as 8-byte-aligned 16-byte loads, is
// slower on gfx950; so is this layout for the dK blocks, whose main stream is their
// loads.)
struct BinPair {
  int k[2], l[2];  // row and column of the two bins in a plane of rows x cols
  __device__ BinPair(int e0, int cols, float rcols) {
    k[0] = div_small(e0, cols, rcols, l[0]);
    k[1] = k[0], l[1] = l[0] + 1;
    if (l[1] == cols) k[1] += 1, l[1] = 0;
  }
};

__device__ __forceinline__ float4 pack2(float2 a, float2 b) { return make_float4(a.x, a.y, b.x, b.y); }

// images whose loads a thread has in flight at once
constexpr int kChainImages = 8;

// FDC layer of the FDCNN on spectra (Eq. 5, Algorithm 1) followed by FDP, forming only
// the bins FDP keeps: Y [B][S][M][M/2+1] from X [B][C][N][N/2+1], K [S][N][N/2+1].
// Kept rows of the N-point spectrum: k < M/2 and k >= N - M/2 (output row k or
// k - (N - M)); kept columns l <= M/2.  Grid: x over an output plane's bin pairs in
// order (contiguous stores) times groups of JB output channels of one input channel
// (o = c J + j): a thread loads its two bins of X[b][c] once for the group's JB
// outputs, and each output's two kernel bins once for every image.
// Pi_H of one bin of column 0 or the last column from its value y and the value yp of
// row -k of the same column: (y + conj(yp)) / 2, the real part alone where row -k is
// row k (k = 0 and H/2); the arithmetic of k_hermitian_columns.
__device__ __forceinline__ float2 hermitian_bin(float2 y, float2 yp, bool self) {
  return self ? make_float2(y.x, 0.f) : make_float2(0.5f * (y.x + yp.x), 0.5f * (y.y - yp.y));
}

// PROJ: Y is written as Pi_H(Y) (columns 0 and M/2 Hermitian-projected along the rows),
// which equals k_cic_fdp_fwd followed by k_hermitian_columns on Y: the main workgroups
// (the first nmain) store every bin but those of the two columns, and the workgroups
// after them form those columns, a thread per bin (b, o, row, column), from the bin and
// its partner in row -k.  The products use cmul_f, so both paths round alike.
template <int JB, bool PROJ>
__global__ __launch_bounds__(256) void k_cic_fdp_fwd(const float2 *__restrict__ X, const float2 *__restrict__ K,
                                                     float2 *__restrict__ Y, int B, int C, int J, int N, int M,
                                                     int nmain) {
  const int S = C * J, Lm = M / 2 + 1, NF = N / 2 + 1, pe = M * Lm, JG = J / JB;
  if constexpr (PROJ) {
    if ((int)blockIdx.x >= nmain) {
      const long long id = (long long)(blockIdx.x - nmain) * 256 + threadIdx.x;
      if (id >= (long long)B * S * M * 2) return;
      const int l = (id & 1) ? Lm - 1 : 0;
      const long long r = id >> 1;
      const int k = (int)(r % M);
      const long long bo = r / M;  // b * S + o
      const int o = (int)(bo % S), b = (int)(bo / S), c = o / J, kp = (M - k) % M;
      const float2 *xo = X + ((long long)b * C + c) * N * NF + l, *ko = K + (long long)o * N * NF + l;
      const int kr = k < M / 2 ? k : k + (N - M), krp = kp < M / 2 ? kp : kp + (N - M);
      const float2 y = cmul_f(xo[(long long)kr * NF], ko[(long long)kr * NF]);
      const float2 yp = cmul_f(xo[(long long)krp * NF], ko[(long long)krp * NF]);
      Y[(bo * M + k) * Lm + l] = hermitian_bin(y, yp, k == 0 || 2 * k == M);
      return;
    }
  }
  // one group of one block of bin pairs per workgroup, the groups of a block consecutive
  // after the XCD remap, so that the J / JB groups reading the same input bins run
  // together on one XCD and share them through its L2
  const int lin = xcd_remap(blockIdx.x, nmain), gi = lin % (C * JG);
  const int e0 = 2 * ((lin / (C * JG)) * 256 + threadIdx.x);
  if (e0 >= pe) return;
  const BinPair q(e0, Lm, 1.f / (float)Lm);
  int off[2];  // bin offsets in an N-plane
#pragma unroll
  for (int h = 0; h < 2; ++h) off[h] = (q.k[h] < M / 2 ? q.k[h] : q.k[h] + (N - M)) * NF + q.l[h];
  // bins the edge workgroups store (PROJ)
  const bool skip0 = PROJ && (q.l[0] == 0 || q.l[0] == Lm - 1), skip1 = PROJ && (q.l[1] == 0 || q.l[1] == Lm - 1);
  auto store = [&](float4 *dst, float2 v0, float2 v1) {
    if (!skip0 && !skip1) {
      *dst = pack2(v0, v1);
    } else {
      float2 *d2 = reinterpret_cast<float2 *>(dst);
      if (!skip0) d2[0] = v0;
      if (!skip1) d2[1] = v1;
    }
  };
  const long long xs = (long long)C * N * NF, ys = (long long)S * (pe / 2);  // image strides (float2, float4)
  {
    const int c = gi / JG, o0 = c * J + (gi - c * JG) * JB;
    const float2 *xo = X + (long long)c * N * NF;
    float2 kv[JB][2];
#pragma unroll
    for (int jj = 0; jj < JB; ++jj) {
      const float2 *ko = K + (long long)(o0 + jj) * N * NF;
      kv[jj][0] = ko[off[0]], kv[jj][1] = ko[off[1]];
    }
    float4 *yo = reinterpret_cast<float4 *>(Y + (long long)o0 * pe + e0);
    int b = 0;
    for (; b + kChainImages <= B; b += kChainImages) {
      float2 a0[kChainImages], a1[kChainImages];
#pragma unroll
      for (int u = 0; u < kChainImages; ++u) {
        a0[u] = xo[(b + u) * xs + off[0]];
        a1[u] = xo[(b + u) * xs + off[1]];
      }
#pragma unroll
      for (int jj = 0; jj < JB; ++jj)
#pragma unroll
        for (int u = 0; u < kChainImages; ++u)
          store(yo + (b + u) * ys + jj * (pe / 2), cmul_f(a0[u], kv[jj][0]), cmul_f(a1[u], kv[jj][1]));
    }
    for (; b < B; ++b) {
      const float2 a0 = xo[b * xs + off[0]], a1 = xo[b * xs + off[1]];
#pragma unroll
      for (int jj = 0; jj < JB; ++jj) store(yo + b * ys + jj * (pe / 2), cmul_f(a0, kv[jj][0]), cmul_f(a1, kv[jj][1]));
    }
  }
}

// Backward of k_cic_fdp_fwd, dX and dK of one layer in one launch (both read gY; on
// the small layers of a chain neither fills the chip alone).
//
// dX block (bx, by): gX [B][C][N][N/2+1] = sum_j gY conj(K) at the kept bins (j in
// order), exact zeros at the bins FDP drops.  bx runs over a plane's bin pairs, by (step
// ny) over the input channels; a thread forms its two bins for every image, four
// images at a time.
// PROJ: the bins of columns 0 and N/2 are left to fdp_bwd_gx_edge.
template <bool PROJ>
__device__ __forceinline__ void fdp_bwd_gx_block(const float2 *__restrict__ gY, const float2 *__restrict__ K,
                                                 float2 *__restrict__ gX, int B, int C, int J, int N, int M, int bx,
                                                 int by, int ny) {
  constexpr int BI = 4;
  const int S = C * J, Lm = M / 2 + 1, NF = N / 2 + 1, pe = N * NF;
  const int e0 = 2 * (bx * 256 + threadIdx.x);
  if (e0 >= pe) return;
  const BinPair q(e0, NF, 1.f / (float)NF);
  bool kept[2];
  int koff[2], yoff[2];  // bin offsets in an N-plane (K) and in an M-plane (gY)
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int kr = q.k[h], l = q.l[h];
    kept[h] = l < Lm && (kr < M / 2 || kr >= N - M / 2);
    const int k = kr < M / 2 ? kr : kr - (N - M);
    koff[h] = kept[h] ? kr * NF + l : 0;  // a dropped bin reads bin 0 and is not used
    yoff[h] = kept[h] ? k * Lm + l : 0;
  }
  const long long mpe = (long long)M * Lm, ys = (long long)S * mpe, xs = (long long)C * (pe / 2);
  const long long kps = (long long)N * NF;
  const bool skip0 = PROJ && (q.l[0] == 0 || q.l[0] == NF - 1), skip1 = PROJ && (q.l[1] == 0 || q.l[1] == NF - 1);
  auto store = [&](float4 *dst, float2 v0, float2 v1) {
    if (!skip0 && !skip1) {
      *dst = pack2(v0, v1);
    } else {
      float2 *d2 = reinterpret_cast<float2 *>(dst);
      if (!skip0) d2[0] = v0;
      if (!skip1) d2[1] = v1;
    }
  };
  for (int c = by; c < C; c += ny) {
    float4 *gp = reinterpret_cast<float4 *>(gX + (long long)c * pe + e0);
    if (!kept[0] && !kept[1]) {
      for (int b = 0; b < B; ++b) store(gp + b * xs, make_float2(0.f, 0.f), make_float2(0.f, 0.f));
      continue;
    }
    const float2 *kp = K + (long long)c * J * kps;   // K[cJ + j] at j * N * NF
    const float2 *yp = gY + (long long)c * J * mpe;  // gY[b][cJ + j] at b * S * mpe + j * mpe
    for (int b0 = 0; b0 < B; b0 += BI) {
      float2 a0[BI], a1[BI];
#pragma unroll
      for (int u = 0; u < BI; ++u) a0[u] = a1[u] = make_float2(0.f, 0.f);
      for (int j = 0; j < J; ++j) {
        const float2 k0 = kp[j * kps + koff[0]], k1 = kp[j * kps + koff[1]];
        float2 g0[BI], g1[BI];
#pragma unroll
        for (int u = 0; u < BI; ++u) {
          const long long bo = (long long)min(b0 + u, B - 1) * ys + j * mpe;  // images past the end: not stored
          g0[u] = yp[bo + yoff[0]];
          g1[u] = yp[bo + yoff[1]];
        }
#pragma unroll
        for (int u = 0; u < BI; ++u) {
          a0[u] = cfmac_f(a0[u], g0[u], k0);
          a1[u] = cfmac_f(a1[u], g1[u], k1);
        }
      }
#pragma unroll
      for (int u = 0; u < BI; ++u)
        if (b0 + u < B)
          store(gp + (b0 + u) * xs, kept[0] ? a0[u] : make_float2(0.f, 0.f), kept[1] ? a1[u] : make_float2(0.f, 0.f));
    }
  }
}

// Pi_H of dX at columns 0 and N/2, thread id over (b, c, row, column): the bin and its
// partner in row -k formed as fdp_bwd_gx_block forms them (zero at bins FDP drops; Pi_H
// acts on the whole N-plane, so the dropped row M/2 receives half of row N - M/2).
__device__ __forceinline__ void fdp_bwd_gx_edge(const float2 *__restrict__ gY, const float2 *__restrict__ K,
                                                float2 *__restrict__ gX, int B, int C, int J, int N, int M,
                                                long long id) {
  const int S = C * J, Lm = M / 2 + 1, NF = N / 2 + 1;
  if (id >= (long long)B * C * N * 2) return;
  const int l = (id & 1) ? NF - 1 : 0;
  const long long r = id >> 1;
  const int kr = (int)(r % N);
  const long long bc = r / N;  // b * C + c
  const int c = (int)(bc % C), b = (int)(bc / C), krp = (N - kr) % N;
  const long long mpe = (long long)M * Lm, kps = (long long)N * NF;
  auto dsum = [&](int row) {  // sum_j gY conj(K) at (row, l), zero where FDP drops it
    float2 a = make_float2(0.f, 0.f);
    if (l < Lm && (row < M / 2 || row >= N - M / 2)) {
      const int k = row < M / 2 ? row : row - (N - M);
      const float2 *yp = gY + ((long long)b * S + (long long)c * J) * mpe + (long long)k * Lm + l;
      const float2 *kp = K + (long long)c * J * kps + (long long)row * NF + l;
      for (int j = 0; j < J; ++j) a = cfmac_f(a, yp[j * mpe], kp[j * kps]);
    }
    return a;
  };
  gX[(bc * N + kr) * NF + l] = hermitian_bin(dsum(kr), dsum(krp), kr == 0 || 2 * kr == N);
}

// dK block (bx, by): dK [S][N][N/2+1] = sum_b gY conj(X) at the kept bins (batch summed
// in order), exact zeros at the bins FDP drops.  bx runs over the bins of a plane, by
// (step ny) over the output channels, so that each channel's planes are streamed in
// order.  (The J channels of one input channel side by side on one XCD, sharing its
// bins through L2, or one thread for several of them: 76-79 -> 97-101 and 83-97 us at
// 1024^2.)
__device__ __forceinline__ void fdp_bwd_gk_block(const float2 *__restrict__ gY, const float2 *__restrict__ X,
                                                 float2 *__restrict__ gK, int B, int C, int J, int N, int M, int bx,
                                                 int by, int ny) {
  const int S = C * J, Lm = M / 2 + 1, NF = N / 2 + 1, pe = N * NF;
  const float rn = 1.f / (float)NF;
  const int e = bx * 256 + threadIdx.x;
  if (e >= pe) return;
  int l;
  const int kr = div_small(e, NF, rn, l);
  const bool kept = l < Lm && (kr < M / 2 || kr >= N - M / 2);
  const int k = kr < M / 2 ? kr : kr - (N - M);
  for (long long o = by; o < S; o += ny) {
    float2 acc = make_float2(0.f, 0.f);
    if (kept) {
      const long long c = o / J;
#pragma unroll 4
      for (int b = 0; b < B; ++b)
        acc = cfmac(acc, gY[(((long long)b * S + o) * M + k) * Lm + l], X[(((long long)b * C + c) * N + kr) * NF + l]);
    }
    gK[o * pe + e] = acc;
  }
}

// Kept-bins forms of the two blocks (fdc_cic_fdp_backward_kept): a thread per bin the
// FDP keeps, bx over those M (M/2+1) bins of a plane in order (row k of the kept rows,
// then column l); the bins FDP drops are not written.  The arithmetic of each kept bin
// is that of fdp_bwd_gx_block and fdp_bwd_gk_block.  PROJ: columns 0 and N/2 of dX are
// left to fdp_bwd_gx_edge, which writes them over every row.
template <bool PROJ>
__device__ __forceinline__ void fdp_bwd_gx_kept(const float2 *__restrict__ gY, const float2 *__restrict__ K,
                                                float2 *__restrict__ gX, int B, int C, int J, int N, int M, int bx,
                                                int by, int ny) {
  constexpr int BI = 4;
  const int S = C * J, Lm = M / 2 + 1, NF = N / 2 + 1;
  const int e = bx * 256 + threadIdx.x;
  if (e >= M * Lm) return;
  int l;
  const int k = div_small(e, Lm, 1.f / (float)Lm, l);
  if (PROJ && (l == 0 || l == NF - 1)) return;
  const int kr = k < M / 2 ? k : k + (N - M);
  const long long mpe = (long long)M * Lm, ys = (long long)S * mpe, pe = (long long)N * NF;
  const long long kps = (long long)N * NF;
  const int koff = kr * NF + l, yoff = e;
  for (int c = by; c < C; c += ny) {
    float2 *gp = gX + (long long)c * pe + koff;
    const float2 *kp = K + (long long)c * J * kps;
    const float2 *yp = gY + (long long)c * J * mpe;
    for (int b0 = 0; b0 < B; b0 += BI) {
      float2 a[BI];
#pragma unroll
      for (int u = 0; u < BI; ++u) a[u] = make_float2(0.f, 0.f);
      for (int j = 0; j < J; ++j) {
        const float2 kv = kp[j * kps + koff];
        float2 g[BI];
#pragma unroll
        for (int u = 0; u < BI; ++u) g[u] = yp[(long long)min(b0 + u, B - 1) * ys + j * mpe + yoff];
#pragma unroll
        for (int u = 0; u < BI; ++u) a[u] = cfmac_f(a[u], g[u], kv);
      }
#pragma unroll
      for (int u = 0; u < BI; ++u)
        if (b0 + u < B) gp[(long long)(b0 + u) * C * pe] = a[u];
    }
  }
}
__device__ __forceinline__ void fdp_bwd_gk_kept(const float2 *__restrict__ gY, const float2 *__restrict__ X,
                                                float2 *__restrict__ gK, int B, int C, int J, int N, int M, int bx,
                                                int by, int ny) {
  const int S = C * J, Lm = M / 2 + 1, NF = N / 2 + 1, pe = N * NF;
  const int e = bx * 256 + threadIdx.x;
  if (e >= M * Lm) return;
  int l;
  const int k = div_small(e, Lm, 1.f / (float)Lm, l);
  const int kr = k < M / 2 ? k : k + (N - M);
  for (long long o = by; o < S; o += ny) {
    float2 acc = make_float2(0.f, 0.f);
    const long long c = o / J;
#pragma unroll 4
    for (int b = 0; b < B; ++b)
      acc = cfmac(acc, gY[(((long long)b * S + o) * M + k) * Lm + l], X[(((long long)b * C + c) * N + kr) * NF + l]);
    gK[o * pe + (long long)kr * NF + l] = acc;
  }
}

// Kept bins, dX and dK in one pass (B <= kChainImages): a thread per (kept bin, input
// channel c) reads the upstream gradient of its bin for the J output channels of c and
// the B images once, for both products.  Per output channel o = c J + j it adds
// gY[b][o] conj(X[b][c]) over b in order and writes dK; per image it adds gY[b][o] K[o]
// over j in order.  The operations and their order are those of fdp_bwd_gk_kept and
// fdp_bwd_gx_kept, so the results are the same bit for bit; the separate blocks read gY
// twice, and dK there reads X once per output channel.  PROJ: columns 0 and N/2 of dX
// are left to fdp_bwd_gx_edge.  Without dX the J output channels may be split over js
// threads (channel group jg of js), each of which loads X of its bin itself.
template <bool PROJ>
__device__ __forceinline__ void fdp_bwd_kept_fused(const float2 *__restrict__ gY, const float2 *__restrict__ K,
                                                   float2 *__restrict__ gX, const float2 *__restrict__ X,
                                                   float2 *__restrict__ gK, int B, int C, int J, int N, int M,
                                                   int bx, int c, int jg, int js) {
  constexpr int BI = kChainImages;
  const int S = C * J, Lm = M / 2 + 1, NF = N / 2 + 1;
  const int e = bx * 256 + threadIdx.x;
  if (e >= M * Lm) return;
  int l;
  const int k = div_small(e, Lm, 1.f / (float)Lm, l);
  const int kr = k < M / 2 ? k : k + (N - M);
  const long long mpe = (long long)M * Lm, ys = (long long)S * mpe, pe = (long long)N * NF;
  const int koff = kr * NF + l;
  const bool dx = gX && !(PROJ && (l == 0 || l == NF - 1));
  float2 xv[BI], a[BI];
#pragma unroll
  for (int u = 0; u < BI; ++u) {
    a[u] = make_float2(0.f, 0.f);
    xv[u] = gK ? X[((long long)min(u, B - 1) * C + c) * pe + koff] : make_float2(0.f, 0.f);
  }
  const float2 *yp = gY + (long long)c * J * mpe + e;
  const float2 *kp = K + (long long)c * J * pe + koff;
  const int jn = J / js;
  for (int j = jg * jn; j < (jg + 1) * jn; ++j) {
    float2 g[BI];
#pragma unroll
    for (int u = 0; u < BI; ++u) g[u] = yp[(long long)min(u, B - 1) * ys + j * mpe];
    if (gK) {
      float2 acc = make_float2(0.f, 0.f);
#pragma unroll
      for (int u = 0; u < BI; ++u)
        if (u < B) acc = cfmac(acc, g[u], xv[u]);
      gK[((long long)c * J + j) * pe + koff] = acc;
    }
    if (dx) {
      const float2 kv = kp[(long long)j * pe];
#pragma unroll
      for (int u = 0; u < BI; ++u) a[u] = cfmac_f(a[u], g[u], kv);
    }
  }
  if (dx) {
    float2 *gp = gX + (long long)c * pe + koff;
#pragma unroll
    for (int u = 0; u < BI; ++u)
      if (u < B) gp[(long long)u * C * pe] = a[u];
  }
}

// Workgroups [0, xbx * xby) run dX blocks, the next kbx * kby dK blocks, and with PROJ
// the rest the Pi_H bins of dX (fdp_bwd_gx_edge).
// KEPT: the kept-bins blocks (fdp_bwd_gx_kept, fdp_bwd_gk_kept); with FUSED (KEPT only)
// the first nk workgroups run fdp_bwd_kept_fused instead, on kbx * kby tiles (kby = C,
// xbx = xby = 0).  js > 1 (no dX): each tile's J channels in js groups, nk = js times the
// tile count rounded up to a multiple of 8; workgroup id runs tile
// ((id / 8) / js) * 8 + id % 8 and group (id / 8) % js, so the js groups of a tile share
// an XCD (workgroups go to the XCDs in turn) and are dispatched close together: the
// input bins they all read come through that XCD's L2.
template <bool PROJ, bool KEPT, bool FUSED>
__global__ __launch_bounds__(256) void k_cic_fdp_bwd(const float2 *__restrict__ gY, const float2 *__restrict__ K,
                                                     float2 *__restrict__ gX, const float2 *__restrict__ X,
                                                     float2 *__restrict__ gK, int B, int C, int J, int N, int M,
                                                     int xbx, int xby, int kbx, int kby, int nk, int js) {
  const int id = blockIdx.x, nx = xbx * xby;
  if constexpr (FUSED) {
    static_assert(KEPT, "the one-pass form writes the kept bins only");
    if (id < nk) {
      if (js == 1) {
        fdp_bwd_kept_fused<PROJ>(gY, K, gX, X, gK, B, C, J, N, M, id % kbx, id / kbx, 0, 1);
      } else {
        const int r = id >> 3, t = (r / js) * 8 + (id & 7);
        if (t < kbx * kby) fdp_bwd_kept_fused<PROJ>(gY, K, gX, X, gK, B, C, J, N, M, t % kbx, t / kbx, r % js, js);
      }
    } else if constexpr (PROJ)
      fdp_bwd_gx_edge(gY, K, gX, B, C, J, N, M, (long long)(id - nk) * 256 + threadIdx.x);
    return;
  }
  if (id < nx) {
    if constexpr (KEPT)
      fdp_bwd_gx_kept<PROJ>(gY, K, gX, B, C, J, N, M, id % xbx, id / xbx, xby);
    else
      fdp_bwd_gx_block<PROJ>(gY, K, gX, B, C, J, N, M, id % xbx, id / xbx, xby);
  } else if (!PROJ || id < nx + nk) {
    const int i = id - nx;
    if constexpr (KEPT)
      fdp_bwd_gk_kept(gY, X, gK, B, C, J, N, M, i % kbx, i / kbx, kby);
    else
      fdp_bwd_gk_block(gY, X, gK, B, C, J, N, M, i % kbx, i / kbx, kby);
  } else {
    fdp_bwd_gx_edge(gY, K, gX, B, C, J, N, M, (long long)(id - nx - nk) * 256 + threadIdx.x);
  }
}

// Pi_H in place (the round trip rfft2(irfft2(Y)) of section 2.4.1.1 with the real-part
// semantics of the inverse): half spectra Y [count][H][Wf], H even; columns 0 and Wf-1
// become (Y[k][l] + conj(Y[-k mod H][l])) / 2, the others are unchanged.  A thread
// owns one row pair (k, H - k) of one of the two columns, so the update is in place.
__global__ __launch_bounds__(256) void k_hermitian_columns(float2 *__restrict__ Y, long long count, int H, int Wf) {
  const int pairs = H / 2 + 1;
  const long long total = count * 2 * pairs;
  for (long long i = (long long)blockIdx.x * 256 + threadIdx.x; i < total; i += (long long)gridDim.x * 256) {
    const int k = (int)(i % pairs);
    const long long rest = i / pairs;
    const int l = (rest & 1) ? Wf - 1 : 0;
    float2 *col = Y + (rest >> 1) * H * (long long)Wf + l;
    if (k == 0 || 2 * k == H) {
      col[(long long)k * Wf].y = 0.f;
    } else {
      const float2 a = col[(long long)k * Wf], b = col[(long long)(H - k) * Wf];
      const float2 p = make_float2(0.5f * (a.x + b.x), 0.5f * (a.y - b.y));
      col[(long long)k * Wf] = p;
      col[(long long)(H - k) * Wf] = cconj(p);
    }
  }
}

hipError_t launch_hermitian_columns(float2 *Y, long long count, int H, int Wf, hipStream_t s) {
  const long long total = count * 2 * (H / 2 + 1);
  return launch("hermitian_columns", k_hermitian_columns, grid_stride_blocks(total, 256), 256, 0, s, Y, count, H,
                Wf);
}

static dim3 plane_grid(long long plane_elems, long long planes) {
  return dim3((unsigned)((plane_elems + 255) / 256), (unsigned)(planes < 65535 ? planes : 65535));
}

// Output channels per thread of the chain's forward: the largest of 8, 4, 2 dividing J
// that leaves at least 512 workgroups (the input bins are loaded J / JB times), else 1.
// (Minimum 256 or 1024 workgroups instead: 0.2202 and 0.2235 ms per chain step
// against 0.2197.)
static int fdp_fwd_jb(long long gx, int C, int J) {
  for (int jb = 8; jb > 1; jb /= 2)
    if (J % jb == 0 && gx * C * (J / jb) >= 512) return jb;
  return 1;
}
template <typename F>
static void dispatch_jb(int jb, F &&f) {
  switch (jb) {
    case 8: f(std::integral_constant<int, 8>{}); break;
    case 4: f(std::integral_constant<int, 4>{}); break;
    case 2: f(std::integral_constant<int, 2>{}); break;
    default: f(std::integral_constant<int, 1>{});
  }
}

hipError_t launch_cic_fdp_fwd(const float2 *X, const float2 *K, float2 *Y, int B, int C, int S, int N, int M,
                              bool project, hipStream_t s) {
  if ((long long)N * (N / 2 + 1) >= (1 << 24)) return hipErrorInvalidValue;
  const int J = S / C;
  const dim3 g0 = plane_grid((long long)M * (M / 2 + 1) / 2, 1);
  if ((long long)g0.x * S >= (1LL << 31)) return hipErrorInvalidValue;
  const int jb = fdp_fwd_jb(g0.x, C, J);
  hipError_t e = hipSuccess;
  dispatch_jb(jb, [&](auto jc) {
    constexpr int JB = decltype(jc)::value;
    const long long nmain = g0.x * (long long)C * (J / JB);
    if (project) {
      const long long nedge = ((long long)B * S * M * 2 + 255) / 256;
      e = timed_launch("cic_fdp_fwd", k_cic_fdp_fwd<JB, true>, dim3((unsigned)(nmain + nedge)), dim3(256), 0, s, X,
                       K, Y, B, C, J, N, M, (int)nmain);
    } else {
      e = timed_launch("cic_fdp_fwd", k_cic_fdp_fwd<JB, false>, dim3((unsigned)nmain), dim3(256), 0, s, X, K, Y, B,
                       C, J, N, M, (int)nmain);
    }
  });
  return e;
}

// Workgroups below which the one-pass backward without dX splits the output channels.
constexpr long long kFdpBwdMinWgs = 2048;

hipError_t launch_cic_fdp_bwd(const float2 *gY, const float2 *K, float2 *gX, const float2 *X, float2 *gK, int B,
                              int C, int S, int N, int M, bool project, bool kept, hipStream_t s) {
  const long long pe = (long long)N * (N / 2 + 1), pk = (long long)M * (M / 2 + 1);
  if (pe >= (1 << 24)) return hipErrorInvalidValue;
  // kept bins of at most kChainImages images: dX and dK in one pass over gY
  const bool fused = kept && B <= kChainImages && (gX || gK);
  long long xbx = gX ? ((kept ? pk : pe / 2) + 255) / 256 : 0, xby = gX ? C : 0;
  long long kbx = gK ? ((kept ? pk : pe) + 255) / 256 : 0, kby = gK ? S : 0;
  if (fused) xbx = xby = 0, kbx = (pk + 255) / 256, kby = C;
  // without dX: the output channels in js groups when the tiles alone give fewer than
  // kFdpBwdMinWgs workgroups
  const int J = S / C;
  int js = 1;
  if (fused && !gX)
    while (js < J && kbx * kby * js < kFdpBwdMinWgs && J % (2 * js) == 0) js *= 2;
  const long long nfused = js == 1 ? kbx * kby : ((kbx * kby + 7) / 8 * 8) * js;
  const long long nedge = (gX && project) ? ((long long)B * C * N * 2 + 255) / 256 : 0;
  const long long total = xbx * xby + (fused ? nfused : kbx * kby) + nedge;
  if (total == 0) return hipSuccess;
  if (total >= (1LL << 31)) return hipErrorInvalidValue;
  const int kbx1 = (int)(kbx > 0 ? kbx : 1), kby1 = (int)(kby > 0 ? kby : 1);
  const int nk = (int)(fused ? nfused : kbx * kby);
  auto go = [&](auto kern) {
    return timed_launch("cic_fdp_bwd", kern, dim3((unsigned)total), dim3(256), 0, s, gY, K, gX, X, gK, B, C, J, N,
                        M, (int)xbx, (int)xby, kbx1, kby1, nk, js);
  };
  if (project && gX) {
    if (fused) return go(k_cic_fdp_bwd<true, true, true>);
    return kept ? go(k_cic_fdp_bwd<true, true, false>) : go(k_cic_fdp_bwd<true, false, false>);
  }
  if (fused) return go(k_cic_fdp_bwd<false, true, true>);
  return kept ? go(k_cic_fdp_bwd<false, true, false>) : go(k_cic_fdp_bwd<false, false, false>);
}

// Largest spatial kernel of the spatial-kernel CIC calls.
constexpr int kSpatialMaxN = 8;

// Kernel spectra of n x n spatial kernels placed at the top-left of the N x N grid
// (section 2.4.1.2), formed on every call at the bins the FDP of an N -> M layer keeps:
// K[o](k, l) = sum_a W^(k a) R_a(l) with R_a(l) = sum_b w[o][a][b] W^(l b),
// W = exp(-2 pi i / N), into K [S][N][N/2+1] (the other bins are not written).  A
// thread owns one column (o, l) of one block of kKspecRows kept rows: it forms R_a(l)
// once and walks the rows, so each row of K is written by consecutive lanes.
// Twiddles come from an LDS copy.
constexpr int kKspecRows = 16;
template <int N>
__global__ __launch_bounds__(256) void k_cic_kspec(const float *__restrict__ w, float2 *__restrict__ K, int n, int M,
                                                   int ncol_blocks) {
  constexpr int NF = N / 2 + 1;
  __shared__ float2 tw[N];
  for (int i = threadIdx.x; i < N; i += 256) tw[i] = twiddle_load<N>(i);
  __syncthreads();
  const int L = M / 2 + 1;
  const int o = blockIdx.x / ncol_blocks;
  const int l = (blockIdx.x - o * ncol_blocks) * 64 + (threadIdx.x & 63);
  if (l >= L) return;
  const float *wo = w + (long long)o * n * n;
  float2 R[kSpatialMaxN];
#pragma unroll
  for (int a = 0; a < kSpatialMaxN; ++a) {
    float rx = 0.f, ry = 0.f;
    if (a < n) {
      for (int b = 0; b < n; ++b) {
        const float2 v = tw[(l * b) % N];
        rx = fmaf(wo[a * n + b], v.x, rx);
        ry = fmaf(wo[a * n + b], v.y, ry);
      }
    }
    R[a] = make_float2(rx, ry);
  }
  float2 *ko = K + (long long)o * N * NF + l;
  const int k_end = min(M, (int)(blockIdx.y + 1) * kKspecRows);
  for (int k = blockIdx.y * kKspecRows + (threadIdx.x >> 6); k < k_end; k += 4) {
    const int kr = k < M / 2 ? k : k + (N - M);
    float2 acc = make_float2(0.f, 0.f);
#pragma unroll
    for (int a = 0; a < kSpatialMaxN; ++a) {
      if (a < n) {
        const float2 u = tw[(kr * a) % N];
        acc.x = fmaf(u.x, R[a].x, fmaf(-u.y, R[a].y, acc.x));
        acc.y = fmaf(u.x, R[a].y, fmaf(u.y, R[a].x, acc.y));
      }
    }
    ko[(long long)kr * NF] = acc;
  }
}

// dL/dw of those kernels from dK [S][N][N/2+1] at the kept bins (the rfft2 adjoint
// restricted to the n x n support): dL/dw[o][a][b] = Re sum dK(k, l) conj(W^(k a + l b)).
// Workgroup (rb, o) takes rows rb, rb + RB, ... of the M kept rows; a wave sums one
// row at a time, E_b = sum_l dK(k, l) conj(W^(l b)) reduced across its lanes, and
// adds Re(E_b conj(W^(k a))).  Partial sums part [S][RB][n n] are added in order by
// k_cic_wgrad_reduce.  n <= kSpatialMaxN.
template <int N>
__global__ __launch_bounds__(256) void k_cic_wgrad_part(const float2 *__restrict__ gK, float *__restrict__ part,
                                                        int n, int M, int RB) {
  constexpr int NF = N / 2 + 1;
  __shared__ float2 tw[N];
  for (int i = threadIdx.x; i < N; i += 256) tw[i] = twiddle_load<N>(i);
  __syncthreads();
  const int L = M / 2 + 1;
  const int rb = blockIdx.x, o = blockIdx.y;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  float acc[kSpatialMaxN * kSpatialMaxN];
#pragma unroll
  for (int i = 0; i < kSpatialMaxN * kSpatialMaxN; ++i) acc[i] = 0.f;
  for (int k = rb + RB * wave; k < M; k += 4 * RB) {
    const int kr = k < M / 2 ? k : k + (N - M);
    const float2 *row = gK + ((long long)o * N + kr) * NF;
    float ex[kSpatialMaxN], ey[kSpatialMaxN];
#pragma unroll
    for (int b = 0; b < kSpatialMaxN; ++b) ex[b] = ey[b] = 0.f;
    for (int l = lane; l < L; l += 64) {
      const float2 g = row[l];
#pragma unroll
      for (int b = 0; b < kSpatialMaxN; ++b) {
        if (b < n) {
          const float2 v = tw[(l * b) % N];  // g conj(v)
          ex[b] = fmaf(g.x, v.x, fmaf(g.y, v.y, ex[b]));
          ey[b] = fmaf(g.y, v.x, fmaf(-g.x, v.y, ey[b]));
        }
      }
    }
#pragma unroll
    for (int b = 0; b < kSpatialMaxN; ++b) {
      if (b < n) {
        for (int off = 32; off > 0; off >>= 1) {
          ex[b] += __shfl_xor(ex[b], off);
          ey[b] += __shfl_xor(ey[b], off);
        }
      }
    }
#pragma unroll
    for (int a = 0; a < kSpatialMaxN; ++a) {
      if (a < n) {
        const float2 u = tw[(kr * a) % N];
#pragma unroll
        for (int b = 0; b < kSpatialMaxN; ++b)
          if (b < n) acc[a * kSpatialMaxN + b] = fmaf(ex[b], u.x, fmaf(ey[b], u.y, acc[a * kSpatialMaxN + b]));
      }
    }
  }
  // every lane of a wave holds the wave's sums; add the four waves in order
  __shared__ float red[4][kSpatialMaxN * kSpatialMaxN];
  if (lane == 0) {
#pragma unroll
    for (int i = 0; i < kSpatialMaxN * kSpatialMaxN; ++i) red[wave][i] = acc[i];
  }
  __syncthreads();
  const int t = threadIdx.x;
  if (t < n * n) {
    const int a = t / n, b = t - (t / n) * n;
    const int i = a * kSpatialMaxN + b;
    part[((long long)o * RB + rb) * n * n + t] = (red[0][i] + red[1][i]) + (red[2][i] + red[3][i]);
  }
}

__global__ void k_cic_wgrad_reduce(const float *__restrict__ part, float *__restrict__ gw, int nn, int RB,
                                   int total) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= total) return;
  const int o = i / nn, t = i - (i / nn) * nn;
  float acc = 0.f;
  for (int rb = 0; rb < RB; ++rb) acc += part[((long long)o * RB + rb) * nn + t];
  gw[i] = acc;
}

// ---------------------------------------------------------------------------
// The same two steps for every layer of a stack in one launch each (the spatial-kernel
// stack): layer sizes are runtime values, each workgroup stages its layer's twiddle
// table.  ROLL artifact handling (out[i][j] = y[(i + s) mod M][(j + s) mod M]) of a
// layer's M x M output is a phase at each output bin, exp(+2 pi i s (k' + l) / M) with
// k' the output row, so it is folded into the kernel spectra here (and its conjugate
// into dK before the projection); the stack executor then runs without artifact
// handling.
// ---------------------------------------------------------------------------
__device__ const float2 *twiddle_table(int n) {
  switch (n) {
#define FDC_TW(V) \
  case V:         \
    return reinterpret_cast<const float2 *>(g_twiddle<V>.v);
    FDC_TW(2) FDC_TW(4) FDC_TW(8) FDC_TW(16) FDC_TW(32) FDC_TW(64) FDC_TW(128) FDC_TW(256) FDC_TW(512) FDC_TW(1024)
    FDC_TW(224)
#undef FDC_TW
    default:
      return nullptr;
  }
}

constexpr int kSpatialTwMax = 1024;
// rows of one workgroup of k_cic_kspec_stack
constexpr int kKspecStackRows = 64;

__device__ __forceinline__ const SpatialLayer &spatial_layer_of(const SpatialBatch &sb, int blk) {
  int i = 0;
  while (i + 1 < sb.count && blk >= sb.layer[i + 1].block0) ++i;
  return sb.layer[i];
}

// a + b mod n for 0 <= a, b < n
__device__ __forceinline__ int add_mod(int a, int b, int n) {
  const int t = a + b;
  return t >= n ? t - n : t;
}

// Table index of exp(+2 pi i s (k + l) / M) = conj(W_N^(s (k + l) N / M)) for output
// bin (k < M, l <= M/2), 0 <= s <= 3 (n <= 8)
__device__ __forceinline__ int roll_index(int s, int k, int l, int M, int N) {
  const int t = add_mod(k, l < M ? l : l - M, M);
  int u = 0;
  for (int r = 0; r < s; ++r) u = add_mod(u, t, M);
  return u * (N / M);
}

template <int NK>
__global__ __launch_bounds__(256) void k_cic_kspec_stack(SpatialBatch sb) {
  __shared__ float2 tw[kSpatialTwMax];
  const SpatialLayer &d = spatial_layer_of(sb, blockIdx.x);
  const int N = d.N, M = d.M, NF = N / 2 + 1, L = M / 2 + 1;
  const float2 *tab = twiddle_table(N);
  for (int i = threadIdx.x; i < N; i += 256) tw[i] = tab[i];
  __syncthreads();
  const int local = blockIdx.x - d.block0;
  const int rb = local % d.rowb, rest = local / d.rowb;
  const int cb = rest % d.ncb, o = rest / d.ncb;
  const int l = cb * 64 + (threadIdx.x & 63);
  if (l >= L) return;
  const float *wo = d.w + (long long)o * NK * NK;
  float2 R[NK];  // R_a(l) = sum_b w[o][a][b] W^(l b)
#pragma unroll
  for (int a = 0; a < NK; ++a) {
    float rx = 0.f, ry = 0.f;
    int idx = 0;  // l b mod N
#pragma unroll
    for (int b = 0; b < NK; ++b) {
      const float2 v = tw[idx];
      rx = fmaf(wo[a * NK + b], v.x, rx);
      ry = fmaf(wo[a * NK + b], v.y, ry);
      idx = add_mod(idx, l, N);
    }
    R[a] = make_float2(rx, ry);
  }
  float2 *ko = d.K + (long long)o * N * NF + l;
  const int k_end = min(M, (rb + 1) * kKspecStackRows);
  for (int k = rb * kKspecStackRows + (threadIdx.x >> 6); k < k_end; k += 4) {
    const int kr = k < M / 2 ? k : k + (N - M);
    float2 acc = make_float2(0.f, 0.f);
    int idx = 0;  // kr a mod N
#pragma unroll
    for (int a = 0; a < NK; ++a) {
      const float2 u = tw[idx];
      acc.x = fmaf(u.x, R[a].x, fmaf(-u.y, R[a].y, acc.x));
      acc.y = fmaf(u.x, R[a].y, fmaf(u.y, R[a].x, acc.y));
      idx = add_mod(idx, kr, N);
    }
    if (d.roll) acc = cmul(acc, cconj(tw[roll_index(d.roll, k, l, M, N)]));
    ko[(long long)kr * NF] = acc;
  }
}

// Rows of one workgroup of k_cic_wgrad_stack (a quarter per wave).
constexpr int kWgradStackRows = 64;

// Partial sums of dL/dw for every layer of the batch.  dL/dw[o][a][b] =
// Re sum_l conj(W^(l b)) F_a(l) with F_a(l) = sum_k dK(k, l) conj(W^(k a)) (k the
// N-grid row of a kept row): a lane owns one column l and sums F_a(l) down the
// workgroup's rows (a wave reads a row segment of 64 bins with one load), projects it
// onto the taps at the end, and the workgroup adds its 256 lanes in a fixed order.
// Workgroup (layer, o, column block cb, row block rb) writes
// part[(o * ncb * rowb + cb * rowb + rb) * NK^2 + tap] of its layer.
template <int NK>
__global__ __launch_bounds__(256) void k_cic_wgrad_stack(SpatialBatch sb) {
  constexpr int T = NK * NK;
  __shared__ float2 tw[kSpatialTwMax];
  __shared__ float red[4][T];
  const SpatialLayer &d = spatial_layer_of(sb, blockIdx.x);
  const int N = d.N, M = d.M, NF = N / 2 + 1, L = M / 2 + 1;
  const float2 *tab = twiddle_table(N);
  for (int i = threadIdx.x; i < N; i += 256) tw[i] = tab[i];
  __syncthreads();
  const int local = blockIdx.x - d.block0;
  const int rb = local % d.rowb, rest = local / d.rowb;
  const int cb = rest % d.ncb, o = rest / d.ncb;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int l = cb * 64 + lane;
  const bool on = l < L;
  const float2 *col = d.gK + (long long)o * N * NF + (on ? l : 0);
  float2 F[NK];
#pragma unroll
  for (int a = 0; a < NK; ++a) F[a] = make_float2(0.f, 0.f);
  const int k_end = min(M, (rb + 1) * kWgradStackRows);
  constexpr int U = 4;  // rows whose loads are in flight together
  for (int k0 = rb * kWgradStackRows + wave; k0 < k_end; k0 += 4 * U) {
    float2 g[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int k = k0 + 4 * u;
      const int kr = k < M / 2 ? k : k + (N - M);
      g[u] = (on && k < k_end) ? col[(long long)kr * NF] : make_float2(0.f, 0.f);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int k = k0 + 4 * u;
      if (k >= k_end) break;
      const int kr = k < M / 2 ? k : k + (N - M);
      float2 gv = g[u];
      if (d.roll) gv = cmul(gv, tw[roll_index(d.roll, k, on ? l : 0, M, N)]);  // dK = dK' conj(phase)
      int idx = 0;  // kr a mod N
#pragma unroll
      for (int a = 0; a < NK; ++a) {
        F[a] = cfmac(F[a], gv, tw[idx]);
        idx = add_mod(idx, kr, N);
      }
    }
  }
  // project onto the taps: Re(F_a conj(W^(l b)))
  float acc[T];
  {
    int idx = 0;  // l b mod N
#pragma unroll
    for (int b = 0; b < NK; ++b) {
      const float2 v = tw[idx];
#pragma unroll
      for (int a = 0; a < NK; ++a) acc[a * NK + b] = fmaf(F[a].x, v.x, F[a].y * v.y);
      idx = add_mod(idx, on ? l : 0, N);
    }
  }
#pragma unroll
  for (int t = 0; t < T; ++t)
    for (int off = 32; off > 0; off >>= 1) acc[t] += __shfl_xor(acc[t], off);
  if (lane == 0) {
#pragma unroll
    for (int t = 0; t < T; ++t) red[wave][t] = acc[t];
  }
  __syncthreads();
  if (threadIdx.x < T) {
    const int t = threadIdx.x;
    d.part[((long long)o * d.ncb * d.rowb + cb * d.rowb + rb) * T + t] =
        (red[0][t] + red[1][t]) + (red[2][t] + red[3][t]);
  }
}

// gw of every layer of the batch from its partial sums (nb = ncb * rowb per output
// channel), added in order (eight partials' loads in flight at a time).
__global__ __launch_bounds__(256) void k_cic_wgrad_stack_reduce(SpatialBatch sb, int total) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= total) return;
  int li = 0;
  while (li + 1 < sb.count && i >= sb.layer[li + 1].elem0) ++li;
  const SpatialLayer &d = sb.layer[li];
  const int nn = d.n * d.n, e = i - d.elem0, nb = d.ncb * d.rowb;
  const int o = e / nn, t = e - (e / nn) * nn;
  const float *src = d.part + (long long)o * nb * nn + t;
  float acc = 0.f;
  int q = 0;
  for (; q + 8 <= nb; q += 8) {
    float v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = src[(q + u) * nn];
#pragma unroll
    for (int u = 0; u < 8; ++u) acc += v[u];
  }
  for (; q < nb; ++q) acc += src[q * nn];
  d.gw[e] = acc;
}

template <class F>
static bool dispatch_spatial_n(int n, F &&f) {
  switch (n) {
#define FDC_CASE(V)                      \
  case V:                                \
    f(std::integral_constant<int, V>{}); \
    return true;
    FDC_CASE(1) FDC_CASE(2) FDC_CASE(3) FDC_CASE(4) FDC_CASE(5) FDC_CASE(6) FDC_CASE(7) FDC_CASE(8)
#undef FDC_CASE
    default:
      return false;
  }
}

int cic_wgrad_stack_blocks(int M) { return ((M / 2 + 1 + 63) / 64) * ((M + kWgradStackRows - 1) / kWgradStackRows); }

hipError_t launch_cic_kspec_stack(SpatialBatch sb, hipStream_t s) {
  int blocks = 0;
  for (int i = 0; i < sb.count; ++i) {
    SpatialLayer &d = sb.layer[i];
    if (d.n != sb.layer[0].n || d.N > kSpatialTwMax || d.N % d.M) return hipErrorInvalidValue;
    d.ncb = (d.M / 2 + 1 + 63) / 64;
    d.rowb = (d.M + kKspecStackRows - 1) / kKspecStackRows;
    d.block0 = blocks;
    const long long nb = (long long)d.S * d.ncb * d.rowb;
    if (blocks + nb >= (1LL << 31)) return hipErrorInvalidValue;
    blocks += (int)nb;
  }
  hipError_t err = hipErrorInvalidValue;
  dispatch_spatial_n(sb.layer[0].n, [&](auto nc) {
    err = launch("cic_kspec_stack", k_cic_kspec_stack<decltype(nc)::value>, (unsigned)blocks, 256, 0, s, sb);
  });
  return err;
}

hipError_t launch_cic_wgrad_stack(SpatialBatch sb, hipStream_t s) {
  int blocks = 0, elems = 0;
  for (int i = 0; i < sb.count; ++i) {
    SpatialLayer &d = sb.layer[i];
    if (d.n != sb.layer[0].n || d.N > kSpatialTwMax || d.N % d.M) return hipErrorInvalidValue;
    d.ncb = (d.M / 2 + 1 + 63) / 64;
    d.rowb = (d.M + kWgradStackRows - 1) / kWgradStackRows;
    d.block0 = blocks;
    d.elem0 = elems;
    const long long nb = (long long)d.S * d.ncb * d.rowb, ne = (long long)d.S * d.n * d.n;
    if (blocks + nb >= (1LL << 31) || elems + ne >= (1LL << 31)) return hipErrorInvalidValue;
    blocks += (int)nb;
    elems += (int)ne;
  }
  hipError_t e = hipErrorInvalidValue;
  dispatch_spatial_n(sb.layer[0].n, [&](auto nc) {
    e = launch("cic_wgrad_stack", k_cic_wgrad_stack<decltype(nc)::value>, (unsigned)blocks, 256, 0, s, sb);
  });
  if (e != hipSuccess) return e;
  return launch("cic_wgrad_stack_reduce", k_cic_wgrad_stack_reduce, (unsigned)((elems + 255) / 256), 256, 0, s, sb,
                elems);
}

bool spatial_kernel_size_supported(int n) { return n >= 1 && n <= kSpatialMaxN; }

bool spatial_channels_supported(int S) { return S >= 1 && S <= 65535; }

bool cic_fdp_size_supported(int N) { return (long long)N * (N / 2 + 1) < (1 << 24); }

int cic_wgrad_blocks(int M) { return M >= 256 ? 32 : (M >= 64 ? 16 : 4); }

hipError_t launch_cic_kspec(int n_img, const float *w, float2 *K, int S, int n, int M, hipStream_t s) {
  if (!spatial_kernel_size_supported(n)) return hipErrorInvalidValue;
  hipError_t err = hipErrorInvalidValue;
  dispatch_n(n_img, [&](auto nc) {
    constexpr int N = decltype(nc)::value;
    const int ncb = (M / 2 + 1 + 63) / 64;
    const long long blocks = (long long)S * ncb;
    if (blocks >= (1LL << 31)) return;
    const int rowb = (M + kKspecRows - 1) / kKspecRows;
    err = timed_launch("cic_kspec", k_cic_kspec<N>, dim3((unsigned)blocks, rowb), dim3(256), 0, s, w, K, n, M, ncb);
  });
  return err;
}

hipError_t launch_cic_wgrad(int n_img, const float2 *gK, float *part, float *gw, int S, int n, int M,
                            hipStream_t s) {
  if (!spatial_kernel_size_supported(n)) return hipErrorInvalidValue;
  const int RB = cic_wgrad_blocks(M);
  hipError_t err = hipErrorInvalidValue;
  dispatch_n(n_img, [&](auto nc) {
    constexpr int N = decltype(nc)::value;
    if (S > 65535) return;
    err = timed_launch("cic_wgrad", k_cic_wgrad_part<N>, dim3(RB, S), dim3(256), 0, s, gK, part, n, M, RB);
  });
  if (err != hipSuccess) return err;
  const int total = S * n * n;
  return launch("cic_wgrad_reduce", k_cic_wgrad_reduce, (unsigned)((total + 255) / 256), 256, 0, s, part, gw, n * n,
                RB, total);
}

hipError_t launch_cic_fwd(const float2 *X, const float2 *K, float2 *Y, int B, int C, int S, long long P,
                          hipStream_t s) {
  const long long total = (long long)B * S * P;
  return launch("cic_fwd", k_cic_fwd, grid_stride_blocks(total, 256), 256, 0, s, X, K, Y, C, S / C, P, total);
}

hipError_t launch_cic_bwd_gx(const float2 *gY, const float2 *K, float2 *gX, int B, int C, int S, long long P,
                             hipStream_t s) {
  const long long total = (long long)B * C * P;
  return launch("cic_bwd_gx", k_cic_bwd_gx, grid_stride_blocks(total, 256), 256, 0, s, gY, K, gX, C, S / C, P,
                total);
}

hipError_t launch_cic_bwd_gk(const float2 *gY, const float2 *X, float2 *gK, int B, int C, int S, long long P,
                             hipStream_t s) {
  const long long total = (long long)S * P;
  return launch("cic_bwd_gk", k_cic_bwd_gk, grid_stride_blocks(total, 256), 256, 0, s, gY, X, gK, B, C, S / C, P,
                total);
}

hipError_t launch_fdp_gather(const float2 *X, float2 *Y, long long count, int H, int Wf, int Mh, int Mwf,
                             hipStream_t s) {
  const long long total = count * Mh * Mwf;
  return launch("fdp_gather", k_fdp_gather, grid_stride_blocks(total, 256), 256, 0, s, X, Y, total, H, Wf, Mh,
                Mwf);
}

hipError_t launch_fdp_scatter(const float2 *gY, float2 *gX, long long count, int H, int Wf, int Mh, int Mwf,
                              hipStream_t s) {
  const long long total = count * H * Wf;
  return launch("fdp_scatter", k_fdp_scatter, grid_stride_blocks(total, 256), 256, 0, s, gY, gX, total, H, Wf, Mh,
                Mwf);
}

}  // namespace fdc
