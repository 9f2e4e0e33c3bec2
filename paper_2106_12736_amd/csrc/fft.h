// Device FFT building blocks for gfx950 (wave64, 160 KB LDS per CU).
//
// The transforms of section 2.4.1.1 (RFFT / IRFFT) are computed as batched
// Stockham FFTs.  One sequence of length N is owned by TPS threads; thread t
// holds the E = N / TPS elements t, t + TPS, t + 2 TPS, ... in registers on
// entry and on exit ("comb" layout), so a kernel can load the input with
// coalesced global reads, run the transform, and apply its epilogue (pooling
// crop, CIC product, weights, stores) straight from registers.  Between
// Stockham passes the data goes through LDS once per pass; radices are large
// (up to 32, computed in registers) so that N <= 1024 needs at most two
// passes, i.e. a single LDS exchange.
//
// Twiddle factors are evaluated at compile time in double precision with the
// exponent reduced as an exact integer (k mod n) and rounded to float once.
#pragma once

#include <hip/hip_runtime.h>

#include <type_traits>

namespace fdc {

// ---------------------------------------------------------------------------
// complex helpers (float2 = {re, im})
// ---------------------------------------------------------------------------
__device__ __forceinline__ float2 cadd(float2 a, float2 b) { return make_float2(a.x + b.x, a.y + b.y); }
__device__ __forceinline__ float2 csub(float2 a, float2 b) { return make_float2(a.x - b.x, a.y - b.y); }
__device__ __forceinline__ float2 cmul(float2 a, float2 b) {
  return make_float2(a.x * b.x - a.y * b.y, a.x * b.y + a.y * b.x);
}
// a * conj(b)
__device__ __forceinline__ float2 cmulc(float2 a, float2 b) {
  return make_float2(a.x * b.x + a.y * b.y, a.y * b.x - a.x * b.y);
}
// cmul and cfmac with the fused multiply-adds written out, so that every call site rounds
// alike (the compiler may fuse the plain forms differently in different code paths)
__device__ __forceinline__ float2 cmul_f(float2 a, float2 b) {
  return make_float2(fmaf(a.x, b.x, -(a.y * b.y)), fmaf(a.x, b.y, a.y * b.x));
}
__device__ __forceinline__ float2 cfmac_f(float2 a, float2 b, float2 c) {
  return make_float2(fmaf(b.y, c.y, fmaf(b.x, c.x, a.x)), fmaf(-b.x, c.y, fmaf(b.y, c.x, a.y)));
}
__device__ __forceinline__ float2 cscale(float2 a, float s) { return make_float2(a.x * s, a.y * s); }
__device__ __forceinline__ float2 cconj(float2 a) { return make_float2(a.x, -a.y); }
// a + b * conj(c)
__device__ __forceinline__ float2 cfmac(float2 a, float2 b, float2 c) {
  return make_float2(a.x + b.x * c.x + b.y * c.y, a.y + b.y * c.x - b.x * c.y);
}

// ---------------------------------------------------------------------------
// compile-time trigonometry: cos / sin of 2 pi k / n in double precision
// ---------------------------------------------------------------------------
constexpr double kPi = 3.14159265358979323846264338327950288;

constexpr double ct_reduce(long long k, long long n) {
  long long r = k % n;
  if (r < 0) r += n;
  if (2 * r > n) r -= n;  // angle in (-pi, pi]
  return 2.0 * kPi * static_cast<double>(r) / static_cast<double>(n);
}
constexpr double ct_sin_x(double x) {
  double term = x, sum = x;
  for (int i = 1; i < 24; ++i) {
    term *= -x * x / static_cast<double>((2 * i) * (2 * i + 1));
    sum += term;
  }
  return sum;
}
constexpr double ct_cos_x(double x) {
  double term = 1.0, sum = 1.0;
  for (int i = 1; i < 24; ++i) {
    term *= -x * x / static_cast<double>((2 * i - 1) * (2 * i));
    sum += term;
  }
  return sum;
}
constexpr double ct_cos2pi(long long k, long long n) { return ct_cos_x(ct_reduce(k, n)); }
constexpr double ct_sin2pi(long long k, long long n) { return ct_sin_x(ct_reduce(k, n)); }

// Table of exp(-2 pi i t / N), t < N, as interleaved floats.
template <int N>
struct TwiddleTable {
  float v[2 * N];
  constexpr TwiddleTable() : v() {
    for (int t = 0; t < N; ++t) {
      v[2 * t] = static_cast<float>(ct_cos2pi(t, N));
      v[2 * t + 1] = static_cast<float>(-ct_sin2pi(t, N));
    }
  }
};

template <int N>
__device__ const TwiddleTable<N> g_twiddle = TwiddleTable<N>();

template <int N>
__device__ __forceinline__ float2 twiddle_load(int idx) {
  return *reinterpret_cast<const float2 *>(&g_twiddle<N>.v[2 * idx]);
}

// Kernels copy the twiddle table of their longest transform into LDS once and
// read every twiddle from there: a table read from global memory costs a vector
// memory instruction per twiddle, and the address unit, not DRAM, is what limits
// these kernels.  A transform of length N / tws reads entry i * tws.
template <int N>
__host__ __device__ constexpr int twiddle_lds_elems() {
  return (N + 31) & ~31;
}
template <int N>
__device__ __forceinline__ void stage_twiddles(float2 *tw, int tid, int nthreads) {
  for (int i = tid; i < N; i += nthreads) tw[i] = twiddle_load<N>(i);
  __syncthreads();
}

// The same staging in two halves, so that a kernel can issue its own global loads
// between them and wait for both together: fetch() loads this thread's share of the
// table into registers, commit() writes it to LDS and synchronises the workgroup
// (every thread of the workgroup must call it).
template <int N, int NT>
struct TwiddleStage {
  static constexpr int PER = (N + NT - 1) / NT;
  float2 v[PER];
  __device__ __forceinline__ void fetch(int tid) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int j = tid + i * NT;
      v[i] = twiddle_load<N>(j < N ? j : 0);
    }
  }
  __device__ __forceinline__ void commit(float2 *tw, int tid) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int j = tid + i * NT;
      if (j < N) tw[j] = v[i];
    }
    __syncthreads();
  }
};

// ---------------------------------------------------------------------------
// compile-time loops
// ---------------------------------------------------------------------------
template <int I, int END, class F>
__device__ __forceinline__ void static_for(F &&f) {
  if constexpr (I < END) {
    f(std::integral_constant<int, I>{});
    static_for<I + 1, END>(f);
  }
}

// Multiply by the constant exp(DIR * 2 pi i K / N); DIR = -1 forward, +1 inverse.
template <int DIR, int N, int K>
__device__ __forceinline__ float2 rot_const(float2 v) {
  constexpr int k = ((K % N) + N) % N;
  if constexpr (k == 0) {
    return v;
  } else if constexpr (2 * k == N) {
    return make_float2(-v.x, -v.y);
  } else if constexpr (4 * k == N) {
    return DIR < 0 ? make_float2(v.y, -v.x) : make_float2(-v.y, v.x);
  } else if constexpr (4 * k == 3 * N) {
    return DIR < 0 ? make_float2(-v.y, v.x) : make_float2(v.y, -v.x);
  } else {
    constexpr float c = static_cast<float>(ct_cos2pi(k, N));
    constexpr float s = static_cast<float>(DIR * ct_sin2pi(k, N));
    return make_float2(v.x * c - v.y * s, v.x * s + v.y * c);
  }
}

// ---------------------------------------------------------------------------
// in-register DFTs of small radix, natural order in and out
// ---------------------------------------------------------------------------
template <int R, int DIR>
struct Dft;

template <int DIR>
struct Dft<1, DIR> {
  __device__ __forceinline__ static void run(float2 *) {}
};

template <int DIR>
struct Dft<2, DIR> {
  __device__ __forceinline__ static void run(float2 *v) {
    float2 a = v[0];
    v[0] = cadd(a, v[1]);
    v[1] = csub(a, v[1]);
  }
};

template <int DIR>
struct Dft<4, DIR> {
  __device__ __forceinline__ static void run(float2 *v) {
    float2 s02 = cadd(v[0], v[2]), d02 = csub(v[0], v[2]);
    float2 s13 = cadd(v[1], v[3]), d13 = rot_const<DIR, 4, 1>(csub(v[1], v[3]));
    v[0] = cadd(s02, s13);
    v[2] = csub(s02, s13);
    v[1] = cadd(d02, d13);
    v[3] = csub(d02, d13);
  }
};

// Seven-point DFT by conjugate-symmetric pairs (n, 7-n).
template <int DIR>
struct Dft<7, DIR> {
  __device__ __forceinline__ static void run(float2 *v) {
    const float2 x0 = v[0];
    float2 s[4], d[4];
    s[1] = cadd(v[1], v[6]); d[1] = csub(v[1], v[6]);
    s[2] = cadd(v[2], v[5]); d[2] = csub(v[2], v[5]);
    s[3] = cadd(v[3], v[4]); d[3] = csub(v[3], v[4]);
    v[0] = cadd(x0, cadd(s[1], cadd(s[2], s[3])));
    static_for<1, 4>([&](auto kk) {
      constexpr int k = decltype(kk)::value;
      float2 a = x0, b = make_float2(0.f, 0.f);
      static_for<1, 4>([&](auto nn) {
        constexpr int n = decltype(nn)::value;
        constexpr float c = static_cast<float>(ct_cos2pi(n * k, 7));
        constexpr float sn = static_cast<float>(ct_sin2pi(n * k, 7));
        a = make_float2(a.x + c * s[n].x, a.y + c * s[n].y);
        b = make_float2(b.x + sn * d[n].x, b.y + sn * d[n].y);
      });
      // X[k] = a + DIR i b, X[7-k] = a - DIR i b
      float2 ib = DIR < 0 ? make_float2(b.y, -b.x) : make_float2(-b.y, b.x);
      v[k] = cadd(a, ib);
      v[7 - k] = csub(a, ib);
    });
  }
};

// Composite radix R = R1 * R2 by one decimation-in-time split:
// X[k1 + R1 k2] = sum_{n2} W_{R2}^{n2 k2} W_R^{n2 k1} sum_{n1} x[R2 n1 + n2] W_{R1}^{n1 k1}.
template <int R>
struct SplitOf {
  static constexpr int R1 = (R % 4 == 0 && R != 8) ? 4 : 2;
  static constexpr int R2 = R / R1;
};

template <int R, int DIR>
struct Dft {
  static_assert(R == 8 || R == 16 || R == 32 || R == 64, "unsupported in-register radix");
  __device__ __forceinline__ static void run(float2 *v) {
    constexpr int R1 = SplitOf<R>::R1, R2 = SplitOf<R>::R2;
    float2 t[R];
    static_for<0, R2>([&](auto n2c) {
      constexpr int n2 = decltype(n2c)::value;
      float2 a[R1];
      static_for<0, R1>([&](auto n1c) { a[decltype(n1c)::value] = v[R2 * decltype(n1c)::value + n2]; });
      Dft<R1, DIR>::run(a);
      static_for<0, R1>([&](auto k1c) {
        constexpr int k1 = decltype(k1c)::value;
        t[n2 * R1 + k1] = rot_const<DIR, R, n2 * k1>(a[k1]);
      });
    });
    static_for<0, R1>([&](auto k1c) {
      constexpr int k1 = decltype(k1c)::value;
      float2 b[R2];
      static_for<0, R2>([&](auto n2c) { b[decltype(n2c)::value] = t[decltype(n2c)::value * R1 + k1]; });
      Dft<R2, DIR>::run(b);
      static_for<0, R2>([&](auto k2c) { v[k1 + R1 * decltype(k2c)::value] = b[decltype(k2c)::value]; });
    });
  }
};

// ---------------------------------------------------------------------------
// per-length Stockham plans: radix of each pass, threads per sequence
// ---------------------------------------------------------------------------
template <int N>
struct FftCfg;
// TPS threads per sequence, E = N / TPS elements per thread, radices of the
// Stockham passes in order (1 = unused).  Every radix must divide E so that
// each thread runs whole butterflies in every pass.  E is kept at 8..16 (16..32
// VGPRs of data) so that kernels stay at 4 or more waves per SIMD; TPS grows
// with N, which lets the thread layouts of an N- and an M-point transform
// (M < N) nest inside one workgroup.
template <int N_, int TPS_, int R0_, int R1_, int R2_, int R3_>
struct FftPlan {
  static constexpr int N = N_;
  static constexpr int TPS = TPS_;
  static constexpr int E = N_ / TPS_;
  static constexpr int R[4] = {R0_, R1_, R2_, R3_};
  static constexpr int P = (R1_ == 1) ? 1 : (R2_ == 1 ? 2 : (R3_ == 1 ? 3 : 4));
};
#define FDC_FFT_CFG(N_, TPS_, R0_, R1_, R2_, R3_) \
  template <>                                     \
  struct FftCfg<N_> : FftPlan<N_, TPS_, R0_, R1_, R2_, R3_> {};
//            N   TPS  radices
FDC_FFT_CFG(2, 1, 2, 1, 1, 1)
FDC_FFT_CFG(4, 1, 4, 1, 1, 1)
FDC_FFT_CFG(8, 1, 8, 1, 1, 1)
FDC_FFT_CFG(16, 2, 8, 2, 1, 1)
FDC_FFT_CFG(32, 4, 8, 4, 1, 1)
FDC_FFT_CFG(64, 8, 8, 8, 1, 1)
FDC_FFT_CFG(128, 8, 16, 8, 1, 1)
FDC_FFT_CFG(256, 32, 8, 8, 4, 1)
FDC_FFT_CFG(512, 64, 8, 8, 8, 1)
FDC_FFT_CFG(1024, 64, 16, 8, 8, 1)
FDC_FFT_CFG(224, 8, 7, 4, 4, 2)
#undef FDC_FFT_CFG

// Plans of the row transforms (one sequence per TPS <= 64 lanes, LDS exchanges
// ordered per wave); the same as FftCfg unless specialised.
template <int N>
struct RowCfg : FftCfg<N> {};
// Plans of the column transforms (a sequence spread over the waves of a workgroup);
// the same as FftCfg unless specialised.  128 points: 16 threads of 8 elements in
// three passes instead of 8 threads of 16 in two, which halves the registers of the
// column kernels' data (the dK kernel went from 159 to 110 VGPRs, two workgroups per
// CU instead of one, and a layer's dK + dX from 37 to 24 us).
template <int N>
struct ColCfg : FftCfg<N> {};
template <>
struct ColCfg<128> : FftPlan<128, 16, 8, 8, 2, 1> {};

template <class Cfg>
constexpr int stockham_ns(int p) {  // product of the radices before pass p
  int ns = 1;
  for (int i = 0; i < p; ++i) ns *= Cfg::R[i];
  return ns;
}

// LDS addressing of the Stockham exchanges, chosen per kernel family:
//   kLdsPlain: plain index.  With CT columns interleaved (element stride CT) the
//              exchanges of the column kernels spread over the banks already, and
//              constant offsets fold into the LDS instructions;
//   kLdsXor:   XOR swizzle inside each aligned block of 32 complex values (bits 5..9
//              of the index flip bits 0..4);
//   kLdsPad:   one complex value of padding after every 32, which breaks up the
//              power-of-two strides of the row kernels' exchanges (element stride 1).
// lds_size<LAYOUT>(n) complex values hold indices [0, n).
enum { kLdsPlain = 0, kLdsXor = 1, kLdsPad = 2 };
template <int LAYOUT>
__device__ __forceinline__ int lds_phys(int i) {
  if constexpr (LAYOUT == kLdsPlain) return i;
  else if constexpr (LAYOUT == kLdsXor) return i ^ ((i >> 5) & 31);
  else return i + (i >> 5);
}
template <int LAYOUT>
__host__ __device__ constexpr int lds_size(int n) {
  return LAYOUT == kLdsPad ? n + (n >> 5) + 1 : (n + 31) & ~31;
}

// Barrier between the LDS writes and reads of an exchange.  WAVE: every
// sequence lives inside one wavefront (TPS <= 64 threads and no column
// interleaving across waves), so ordering the wave's own LDS accesses is enough;
// LDS operations of one wavefront are performed in program order.
template <bool WAVE>
__device__ __forceinline__ void lds_barrier() {
  if constexpr (WAVE) {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  } else {
    __syncthreads();
  }
}

// Padded-layout index arithmetic with compile-time offsets.  For a base that is a
// multiple of 32, i0 >= 0 and a power-of-two stride S (a divisor or a multiple
// of 32), lds_phys(i0 + r S) = lds_phys(i0) + r S + floor(r S / 32) whenever the
// run i0, i0 + S, ... stays in one aligned block of max(32, S * count) -- true for
// the Stockham exchanges below -- so only lds_phys(i0) is computed at run time.
constexpr bool pad_pow2_fit(int s) { return s > 0 && (s & (s - 1)) == 0; }
constexpr int pad_offset(int c) { return c + c / 32; }

// Transform one sequence.  Thread t (0 <= t < TPS) holds v[m] = element t + TPS*m
// on entry and exit.  Element e of the sequence lives in LDS at
// lds[lds_phys(base + e * es)].  Every thread of the workgroup (of the wave with
// WAVE) must call this: it contains barriers.  With LEAD_SYNC the first LDS write
// waits for every thread's earlier use of the LDS.  LAYOUT: lds_phys layout; with
// kLdsPad, es must be 1 and, when N is a multiple of 32, base a multiple of 32.
// tw: twiddle table in LDS (stage_twiddles) of length N * tws.
template <int N, int DIR, bool LEAD_SYNC = true, bool WAVE = false, int LAYOUT = kLdsPlain, class Cfg = FftCfg<N>>
__device__ __forceinline__ void fft_seq(float2 (&v)[Cfg::E], int t, float2 *lds, int base, int es, const float2 *tw,
                                        int tws) {
  using C = Cfg;
  static_assert(C::N == N, "plan length");
  constexpr int E = C::E;
  constexpr int TPS = C::TPS;
  constexpr bool PAD = LAYOUT == kLdsPad && N % 32 == 0;
  static_for<0, C::P>([&](auto pc) {
    constexpr int p = decltype(pc)::value;
    constexpr int R = C::R[p];
    constexpr int BPT = E / R;       // butterflies per thread in this pass
    constexpr int NS = stockham_ns<C>(p);
    constexpr int NR = N / R;
    static_assert(BPT * R == E && BPT * TPS == NR, "radix plan does not fit the thread layout");
    // folded padded addressing of this pass's reads (j + r NR, and j = t + TPS q)
    // and writes (jo + r NS, jo inside an aligned block of NS R)
    constexpr bool FOLD_RD = PAD && NR % 32 == 0;
    constexpr bool FOLD_RQ = FOLD_RD && TPS % 32 == 0;
    constexpr bool FOLD_WR = PAD && pad_pow2_fit(NS) && pad_pow2_fit(NS * R);
    float2 a[E];
    if constexpr (p == 0) {
#pragma unroll
      for (int m = 0; m < E; ++m) a[m] = v[m];
    } else {
      const int rd0 = FOLD_RQ ? lds_phys<LAYOUT>(base + t) : 0;
#pragma unroll
      for (int q = 0; q < BPT; ++q) {
        const int j = t + TPS * q;
        const int k = j % NS;
        const int rdq = FOLD_RQ ? rd0 + pad_offset(TPS * q) : (FOLD_RD ? lds_phys<LAYOUT>(base + j) : 0);
#pragma unroll
        for (int r = 0; r < R; ++r) {
          float2 x = FOLD_RD ? lds[rdq + pad_offset(r * NR)] : lds[lds_phys<LAYOUT>(base + (j + r * NR) * es)];
          if (r > 0) {
            float2 w = tw[r * k * (N / (NS * R)) * tws];
            if (DIR > 0) w.y = -w.y;
            x = cmul(x, w);
          }
          a[q + BPT * r] = x;
        }
      }
    }
    // butterflies: a[q + BPT r], r < R, belong to butterfly q
#pragma unroll
    for (int q = 0; q < BPT; ++q) {
      float2 b[R];
#pragma unroll
      for (int r = 0; r < R; ++r) b[r] = a[q + BPT * r];
      Dft<R, DIR>::run(b);
#pragma unroll
      for (int r = 0; r < R; ++r) a[q + BPT * r] = b[r];
    }
    if constexpr (p == C::P - 1) {
#pragma unroll
      for (int m = 0; m < E; ++m) v[m] = a[m];
    } else {
      if (p > 0 || LEAD_SYNC) lds_barrier<WAVE>();
#pragma unroll
      for (int q = 0; q < BPT; ++q) {
        const int j = t + TPS * q;
        const int jo = (j / NS) * NS * R + (j % NS);
        if constexpr (FOLD_WR) {
          const int w0 = lds_phys<LAYOUT>(base + jo);
#pragma unroll
          for (int r = 0; r < R; ++r) lds[w0 + pad_offset(r * NS)] = a[q + BPT * r];
        } else {
#pragma unroll
          for (int r = 0; r < R; ++r) lds[lds_phys<LAYOUT>(base + (jo + r * NS) * es)] = a[q + BPT * r];
        }
      }
      lds_barrier<WAVE>();
    }
  });
}

}  // namespace fdc
