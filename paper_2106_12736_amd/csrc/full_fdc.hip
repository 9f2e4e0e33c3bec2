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
// Complex products use four real v_mfma_f32_16x16x4f32 per 4-deep K step:
//   re += Ar Br - Ai Bi,  im += Ar Bi + Ai Br.
// Lane layout of v_mfma_f32_16x16x4f32 (A 16x4, B 4x16, D 16x16): lane l holds
// A[l % 16][l / 16], B[l / 16][l % 16] and D[4 (l / 16) + j][l % 16] in register j.
#include "internal.h"

#include <hip/hip_runtime.h>

#include <string>

namespace fdc {

typedef float v4f __attribute__((ext_vector_type(4)));

__device__ __forceinline__ v4f mfma4(float a, float b, v4f c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// Phases of bin `bin` (flat index k * Pf + l): u[a] = W^(k a), v[b] = W^(l b), a, b < NK,
// from the twiddle table tw[j] = W^j, j < P (exponents reduced mod P exactly).
template <int NK>
__device__ __forceinline__ void bin_phases(const float2 *tw, int P, int Pf, int bin, float2 (&u)[NK],
                                           float2 (&v)[NK]) {
  const int k = bin / Pf, l = bin - (bin / Pf) * Pf;
#pragma unroll
  for (int a = 0; a < NK; ++a) {
    u[a] = tw[(k * a) % P];
    v[a] = tw[(l * a) % P];
  }
}

// K = sum_a u[a] sum_b w[a][b] v[b] for one (s, c) pair.
template <int NK>
__device__ __forceinline__ float2 kernel_value(const float (&w)[NK * NK], const float2 (&u)[NK],
                                               const float2 (&v)[NK]) {
  float2 acc = make_float2(0.f, 0.f);
#pragma unroll
  for (int a = 0; a < NK; ++a) {
    float rx = 0.f, ry = 0.f;
#pragma unroll
    for (int b = 0; b < NK; ++b) {
      rx += w[a * NK + b] * v[b].x;
      ry += w[a * NK + b] * v[b].y;
    }
    acc.x += u[a].x * rx - u[a].y * ry;
    acc.y += u[a].x * ry + u[a].y * rx;
  }
  return acc;
}

// ---------------------------------------------------------------------------
// Forward (GX = false) and dL/dX (GX = true) contraction.
//   in  [B][KD][NB] complex: X (KD = Cin) or G (KD = Cout)
//   wt  weights rearranged as [KD][NK*NK][ND] (forward: [c][tap][s]; dL/dX: [s][tap][c])
//   out [B][ND][NB] complex: Y (ND = Cout) or gX (ND = Cin)
// A workgroup (4 waves) computes 16 batch rows x 4 consecutive bins x 256 outputs; wave
// w owns outputs [64 w, 64 w + 64) as four 16-wide tiles.  The K dimension is staged
// in LDS 4 at a time: the 16 x 4 x 4 input values and the 4 x NK*NK x 256 weights.
// ---------------------------------------------------------------------------
constexpr int kFcBins = 4;     // bins per workgroup
constexpr int kFcOut = 256;    // outputs per workgroup
constexpr int kFcThreads = 256;

template <int NK, bool GX>
__global__ __launch_bounds__(kFcThreads) void k_full_contract(const float2 *__restrict__ in,
                                                              const float *__restrict__ wt,
                                                              const float2 *__restrict__ twg,
                                                              float2 *__restrict__ out, int B, int KD, int ND,
                                                              int P, int Pf, int NB) {
  constexpr int T = NK * NK;
  extern __shared__ float smem[];
  float2 *tw = reinterpret_cast<float2 *>(smem);            // P
  float2 *sA = tw + ((P + 31) & ~31);                       // [16 b][4 kk][4 bins]
  float *sW = reinterpret_cast<float *>(sA + 16 * 4 * kFcBins);  // [4 kk][T][256 n]
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nbg = (NB + kFcBins - 1) / kFcBins;
  const int bg = blockIdx.x % nbg;
  const int n0 = (blockIdx.x / nbg) * kFcOut;
  const int b0 = blockIdx.y * 16;
  const int bin0 = bg * kFcBins;
  for (int i = tid; i < P; i += kFcThreads) tw[i] = twg[i];
  __syncthreads();

  // phases of this workgroup's bins (the same for every lane)
  float2 u[kFcBins][NK], v[kFcBins][NK];
#pragma unroll
  for (int q = 0; q < kFcBins; ++q) {
    const int bin = bin0 + q < NB ? bin0 + q : NB - 1;
    bin_phases<NK>(tw, P, Pf, bin, u[q], v[q]);
  }

  v4f accr[kFcBins][4], acci[kFcBins][4];
#pragma unroll
  for (int q = 0; q < kFcBins; ++q)
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      accr[q][t] = v4f{0.f, 0.f, 0.f, 0.f};
      acci[q][t] = v4f{0.f, 0.f, 0.f, 0.f};
    }

  const int mrow = lane % 16, kk = lane / 16;  // A operand: row b0 + mrow, k = k0 + kk
  for (int k0 = 0; k0 < KD; k0 += 4) {
    // stage the inputs: thread -> (b, kk, bin q); out-of-range entries are zero
    {
      const int b = tid / 16, kq = (tid / 4) % 4, q = tid % 4;
      const int gb = b0 + b, gk = k0 + kq, gbin = bin0 + q;
      float2 val = make_float2(0.f, 0.f);
      if (gb < B && gk < KD && gbin < NB) val = in[((long long)gb * KD + gk) * NB + gbin];
      sA[(b * 4 + kq) * kFcBins + q] = val;
    }
    // stage the weights [kq][tap][n] for n in [n0, n0 + 256)
    for (int i = tid; i < 4 * T * kFcOut; i += kFcThreads) {
      const int n = i % kFcOut, r = i / kFcOut;  // r = kq * T + tap
      const int kq = r / T, tap = r - kq * T;
      const int gk = k0 + kq, gn = n0 + n;
      sW[i] = (gk < KD && gn < ND) ? wt[((long long)gk * T + tap) * ND + gn] : 0.f;
    }
    __syncthreads();

    float2 a[kFcBins];
#pragma unroll
    for (int q = 0; q < kFcBins; ++q) a[q] = sA[(mrow * 4 + kk) * kFcBins + q];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int nl = wave * 64 + t * 16 + mrow;  // B operand column n0 + nl, row k0 + kk
      float w[T];
#pragma unroll
      for (int tap = 0; tap < T; ++tap) w[tap] = sW[(kk * T + tap) * kFcOut + nl];
#pragma unroll
      for (int q = 0; q < kFcBins; ++q) {
        const float2 kv = kernel_value<NK>(w, u[q], v[q]);
        const float br = kv.x, bi = GX ? -kv.y : kv.y;  // dL/dX uses conj(K)
        accr[q][t] = mfma4(a[q].x, br, accr[q][t]);
        accr[q][t] = mfma4(-a[q].y, bi, accr[q][t]);
        acci[q][t] = mfma4(a[q].x, bi, acci[q][t]);
        acci[q][t] = mfma4(a[q].y, br, acci[q][t]);
      }
    }
    __syncthreads();
  }

  // D[m][n]: lane holds rows 4 (lane / 16) + j, column lane % 16 of each 16 x 16 tile
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const int gn = n0 + wave * 64 + t * 16 + mrow;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int gb = b0 + 4 * kk + j;
      if (gb >= B || gn >= ND) continue;
      float2 *o = out + ((long long)gb * ND + gn) * NB + bin0;
#pragma unroll
      for (int q = 0; q < kFcBins; ++q)
        if (bin0 + q < NB) o[q] = make_float2(accr[q][t][j], acci[q][t][j]);
    }
  }
}

// ---------------------------------------------------------------------------
// dL/dw partial sums over one chunk of bins.
//   G [B][S][NB], X [B][C][NB] complex; part [chunk][S][C][NK*NK] float
// gK[s][c] = sum_b G[b][s] conj(X[b][c]) on the matrix cores (M = s, N = c, K-dim = b,
// 4 batch rows per step), then dL/dw[s][c][a][b] += Re(gK conj(W^(k a) W^(l b))).
// A workgroup (4 waves) owns a 32 x 32 (s, c) block, each wave a 16 x 16 tile, and
// walks the chunk's bins 8 at a time; for each group of 8 bins the batch is staged in
// LDS 16 rows at a time, so the LDS footprint does not depend on B.
// ---------------------------------------------------------------------------
constexpr int kGwBins = 8;
constexpr int kGwBatch = 16;

template <int NK>
__global__ __launch_bounds__(256) void k_full_gw(const float2 *__restrict__ G, const float2 *__restrict__ X,
                                                 const float2 *__restrict__ twg, float *__restrict__ part, int B,
                                                 int S, int C, int P, int Pf, int NB, int chunk_bins) {
  constexpr int T = NK * NK;
  extern __shared__ float smem[];
  float2 *tw = reinterpret_cast<float2 *>(smem);
  float2 *sG = tw + ((P + 31) & ~31);          // [16 b][32 s][8 bins]
  float2 *sX = sG + kGwBatch * 32 * kGwBins;   // [16 b][32 c][8 bins]
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int sblocks = (S + 31) / 32, cblocks = (C + 31) / 32;
  const int blk = blockIdx.x % (sblocks * cblocks);
  const int chunk = blockIdx.x / (sblocks * cblocks);
  const int s0 = (blk / cblocks) * 32, c0 = (blk % cblocks) * 32;
  const int ws = (wave >> 1) * 16, wc = (wave & 1) * 16;  // wave tile inside the block
  const int bin_begin = chunk * chunk_bins;
  const int bin_end = min(NB, bin_begin + chunk_bins);
  for (int i = tid; i < P; i += 256) tw[i] = twg[i];

  float gw[4][T];  // rows s0 + ws + 4 (lane / 16) + j, column c0 + wc + lane % 16
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int t = 0; t < T; ++t) gw[j][t] = 0.f;
  const int mrow = lane % 16, kq = lane / 16;

  for (int bb = bin_begin; bb < bin_end; bb += kGwBins) {
    v4f dr[kGwBins], di[kGwBins];
#pragma unroll
    for (int q = 0; q < kGwBins; ++q) dr[q] = di[q] = v4f{0.f, 0.f, 0.f, 0.f};
    for (int b0 = 0; b0 < B; b0 += kGwBatch) {
      __syncthreads();
      // stage G[b0..b0+16][s0..s0+32][bins] and X[b0..b0+16][c0..c0+32][bins]; zero outside
      for (int i = tid; i < kGwBatch * 32 * kGwBins; i += 256) {
        const int q = i % kGwBins, r = i / kGwBins;  // r = b * 32 + x
        const int b = b0 + r / 32, x = r % 32;
        const int gbin = bb + q;
        const bool ok = gbin < bin_end && b < B;
        const int gs = s0 + x, gc = c0 + x;
        sG[i] = (ok && gs < S) ? G[((long long)b * S + gs) * NB + gbin] : make_float2(0.f, 0.f);
        sX[i] = (ok && gc < C) ? X[((long long)b * C + gc) * NB + gbin] : make_float2(0.f, 0.f);
      }
      __syncthreads();
#pragma unroll
      for (int q = 0; q < kGwBins; ++q)
#pragma unroll
        for (int b4 = 0; b4 < kGwBatch; b4 += 4) {
          const int b = b4 + kq;
          const float2 g = sG[(b * 32 + ws + mrow) * kGwBins + q];  // A[m = s][k = b]
          const float2 x = sX[(b * 32 + wc + mrow) * kGwBins + q];  // B[k = b][n = c]
          // D = G conj(X):  re = Gr Xr + Gi Xi,  im = Gi Xr - Gr Xi
          dr[q] = mfma4(g.x, x.x, dr[q]);
          dr[q] = mfma4(g.y, x.y, dr[q]);
          di[q] = mfma4(g.y, x.x, di[q]);
          di[q] = mfma4(-g.x, x.y, di[q]);
        }
    }
#pragma unroll
    for (int q = 0; q < kGwBins; ++q) {
      const int gbin = bb + q;
      if (gbin >= bin_end) break;
      float2 u[NK], v[NK];
      bin_phases<NK>(tw, P, Pf, gbin, u, v);
#pragma unroll
      for (int a = 0; a < NK; ++a)
#pragma unroll
        for (int b = 0; b < NK; ++b) {
          // phase W^(k a) W^(l b); Re(D conj(phase)) = Dr pr + Di pi
          const float pr = u[a].x * v[b].x - u[a].y * v[b].y;
          const float pi = u[a].x * v[b].y + u[a].y * v[b].x;
#pragma unroll
          for (int j = 0; j < 4; ++j) gw[j][a * NK + b] += dr[q][j] * pr + di[q][j] * pi;
        }
    }
  }
  // write this chunk's partial sums
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int gs = s0 + ws + 4 * kq + j, gc = c0 + wc + mrow;
    if (gs >= S || gc >= C) continue;
    float *p = part + (((long long)chunk * S + gs) * C + gc) * T;
#pragma unroll
    for (int t = 0; t < T; ++t) p[t] = gw[j][t];
  }
}

// dL/dw = sum over chunks, in chunk order.
__global__ void k_full_gw_reduce(const float *__restrict__ part, float *__restrict__ gw, long long n, int chunks) {
  for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (long long)gridDim.x * blockDim.x) {
    float acc = 0.f;
    for (int c = 0; c < chunks; ++c) acc += part[(long long)c * n + i];
    gw[i] = acc;
  }
}

// Weights rearranged for the contraction: forward [c][tap][s], dL/dX [s][tap][c].
__global__ void k_full_weights(const float *__restrict__ w, float *__restrict__ wf, float *__restrict__ wg, int S,
                               int C, int T) {
  const long long n = (long long)S * C * T;
  for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (long long)gridDim.x * blockDim.x) {
    const int tap = (int)(i % T);
    const long long sc = i / T;
    const int c = (int)(sc % C), s = (int)(sc / C);
    if (wf) wf[((long long)c * T + tap) * S + s] = w[i];
    if (wg) wg[((long long)s * T + tap) * C + c] = w[i];
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

static size_t contract_lds(int P, int nk) {
  return ((size_t)((P + 31) & ~31) + 16 * 4 * kFcBins) * sizeof(float2) + (size_t)4 * nk * nk * kFcOut * sizeof(float);
}

hipError_t launch_full_weights(const float *w, float *wf, float *wg, int S, int C, int nk, hipStream_t s) {
  const long long n = (long long)S * C * nk * nk;
  long long g = (n + 255) / 256;
  if (g > 65536) g = 65536;
  timing_before("full_weights", s);
  hipLaunchKernelGGL(k_full_weights, dim3((unsigned)g), dim3(256), 0, s, w, wf, wg, S, C, nk * nk);
  const hipError_t e = hipGetLastError();
  timing_after("full_weights", s);
  return e;
}

hipError_t launch_full_contract(bool gx, int nk, const float2 *in, const float *wt, const float2 *tw, float2 *out,
                                int B, int KD, int ND, int P, hipStream_t s) {
  const int Pf = P / 2 + 1, NB = P * Pf;
  const long long nbg = (NB + kFcBins - 1) / kFcBins;
  const long long gx_ = nbg * ((ND + kFcOut - 1) / kFcOut);
  const int gy = (B + 15) / 16;
  if (gx_ >= (1LL << 31)) return hipErrorInvalidValue;
  hipError_t err = hipErrorInvalidValue;
  dispatch_nk(nk, [&](auto nc) {
    constexpr int NK = decltype(nc)::value;
    const char *nm = gx ? "full_contract_gx" : "full_contract_fwd";
    timing_before(nm, s);
    if (gx)
      hipLaunchKernelGGL((k_full_contract<NK, true>), dim3((unsigned)gx_, gy), dim3(kFcThreads), contract_lds(P, NK),
                         s, in, wt, tw, out, B, KD, ND, P, Pf, NB);
    else
      hipLaunchKernelGGL((k_full_contract<NK, false>), dim3((unsigned)gx_, gy), dim3(kFcThreads),
                         contract_lds(P, NK), s, in, wt, tw, out, B, KD, ND, P, Pf, NB);
    err = hipGetLastError();
    timing_after(nm, s);
  });
  return err;
}

int full_gw_chunks(int B, int S, int C, int P) {
  const int NB = P * (P / 2 + 1);
  const int blocks = ((S + 31) / 32) * ((C + 31) / 32);
  int chunks = (2048 + blocks - 1) / blocks;  // about 2048 workgroups
  const int maxc = (NB + kGwBins - 1) / kGwBins;
  if (chunks > maxc) chunks = maxc;
  if (chunks < 1) chunks = 1;
  (void)B;
  return chunks;
}

hipError_t launch_full_gw(int nk, const float2 *G, const float2 *X, const float2 *tw, float *part, float *gw, int B,
                          int S, int C, int P, hipStream_t s) {
  const int Pf = P / 2 + 1, NB = P * Pf;
  const int chunks = full_gw_chunks(B, S, C, P);
  int chunk_bins = (NB + chunks - 1) / chunks;
  chunk_bins = (chunk_bins + kGwBins - 1) / kGwBins * kGwBins;
  const int blocks = ((S + 31) / 32) * ((C + 31) / 32);
  const size_t lds = ((size_t)((P + 31) & ~31) + 2 * (size_t)kGwBatch * 32 * kGwBins) * sizeof(float2);
  hipError_t err = hipErrorInvalidValue;
  dispatch_nk(nk, [&](auto nc) {
    constexpr int NK = decltype(nc)::value;
    timing_before("full_gw", s);
    hipLaunchKernelGGL((k_full_gw<NK>), dim3((unsigned)(blocks * chunks)), dim3(256), lds, s, G, X, tw, part, B, S, C,
                       P, Pf, NB, chunk_bins);
    err = hipGetLastError();
    timing_after("full_gw", s);
  });
  if (err != hipSuccess) return err;
  const long long n = (long long)S * C * nk * nk;
  long long g = (n + 255) / 256;
  if (g > 65536) g = 65536;
  timing_before("full_gw_reduce", s);
  hipLaunchKernelGGL(k_full_gw_reduce, dim3((unsigned)g), dim3(256), 0, s, part, gw, n, chunks);
  err = hipGetLastError();
  timing_after("full_gw_reduce", s);
  return err;
}

}  // namespace fdc
