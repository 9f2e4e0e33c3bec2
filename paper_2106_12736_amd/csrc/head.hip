// The FDCNN classifier head and optimiser (section 2.5.1 and Fig. 3: a ReLU between
// the final inverse transform and the fully connected layer; section 3.1: softmax
// cross-entropy loss, Adam with weight decay).
//
//   k_head_fwd   partial logits over a chunk of features: relu(y[b][f]) W[o][f]
//   k_head_loss  logits (chunk sums in a fixed order, plus bias), mean cross-entropy
//   k_head_bwd   dlogits = (softmax - onehot) / B; gW, gbias, and gy through the ReLU
//   k_adam       one Adam step over a flat parameter array (k_adam_count: step count)
//
// Every sum runs in a fixed order, so results repeat bit for bit.  The head is a
// streaming pass over y and W (HBM-bound): one fully connected layer to a handful of
// classes reads each feature once per image.
#include "device.h"
#include "internal.h"

#include <hip/hip_runtime.h>

#include <mutex>

namespace fdc {

constexpr int kHeadThreads = 256;
constexpr int kHeadChunk = kHeadThreads * 4;  // features per forward workgroup

long long head_chunks(long long F) { return (F + kHeadChunk - 1) / kHeadChunk; }

// Fixed-order tree sum of red[0..255] into red[0] (all threads take part).
__device__ __forceinline__ void block_sum(float *red) {
  for (int w = kHeadThreads / 2; w > 0; w >>= 1) {
    __syncthreads();
    if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
  }
  __syncthreads();
}

// grid (chunks, B): part[b][chunk][o] = sum over the chunk's features of relu(y) W[o].
__global__ __launch_bounds__(kHeadThreads) void k_head_fwd(const float *__restrict__ y, const float *__restrict__ W,
                                                           float *__restrict__ part, long long F, int classes,
                                                           int chunks) {
  __shared__ float red[kHeadThreads];
  const int chunk = blockIdx.x, b = blockIdx.y;
  const long long f0 = (long long)chunk * kHeadChunk;
  const float *yb = y + (long long)b * F;
  float acc[kHeadMaxClasses];
#pragma unroll
  for (int o = 0; o < kHeadMaxClasses; ++o) acc[o] = 0.f;
  for (int i = threadIdx.x; i < kHeadChunk; i += kHeadThreads) {
    const long long f = f0 + i;
    if (f >= F) break;
    const float r = fmaxf(yb[f], 0.f);
#pragma unroll
    for (int o = 0; o < kHeadMaxClasses; ++o)
      if (o < classes) acc[o] = fmaf(r, W[(long long)o * F + f], acc[o]);
  }
  for (int o = 0; o < classes; ++o) {
    red[threadIdx.x] = acc[o];
    block_sum(red);
    if (threadIdx.x == 0) part[((long long)b * chunks + chunk) * classes + o] = red[0];
  }
}

// One workgroup: logits[b][o] = sum_chunk part[b][chunk][o] + bias[o] (one wave per
// (b, o): lane l sums chunks l, l + 64, ... in order, then a fixed butterfly across the
// lanes); loss = mean_b of logsumexp(logits[b]) - logits[b][label[b]] (NaN for a
// label outside [0, classes)).
__global__ __launch_bounds__(kHeadThreads) void k_head_loss(const float *__restrict__ part,
                                                            const float *__restrict__ bias,
                                                            const int *__restrict__ labels, float *__restrict__ logits,
                                                            float *__restrict__ loss, int B, int classes, int chunks) {
  extern __shared__ float lg[];  // [B][classes]
  __shared__ float red[kHeadThreads];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  for (int idx = wave; idx < B * classes; idx += kHeadThreads / 64) {
    const int b = idx / classes, o = idx - b * classes;
    const float *pb = part + (long long)b * chunks * classes + o;
    float s = 0.f;
    for (int c = lane; c < chunks; c += 64) s += pb[(long long)c * classes];
    for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off, 64);
    if (lane == 0) {
      s += bias[o];
      lg[idx] = s;
      logits[idx] = s;
    }
  }
  __syncthreads();
  float mine = 0.f;  // this thread's images, in order
  for (int b = threadIdx.x; b < B; b += kHeadThreads) {
    const float *l = lg + b * classes;
    float mx = -INFINITY;
    for (int o = 0; o < classes; ++o) mx = fmaxf(mx, l[o]);
    float se = 0.f;
    for (int o = 0; o < classes; ++o) se += expf(l[o] - mx);
    const int lab = labels[b];
    const float lb = (lab >= 0 && lab < classes) ? l[lab] : NAN;
    mine += (mx + logf(se)) - lb;
  }
  red[threadIdx.x] = mine;
  block_sum(red);
  if (threadIdx.x == 0) loss[0] = red[0] / (float)B;
}

// grid over features: dl = (softmax(logits) - onehot) / B (every workgroup forms it in
// LDS), then per feature f: gW[o][f] = sum_b dl[b][o] relu(y[b][f]),
// gy[b][f] = [y[b][f] > 0] sum_o dl[b][o] W[o][f] (gy NULL: skipped); workgroup 0 also
// writes gbias[o] = sum_b dl[b][o].
__global__ __launch_bounds__(kHeadThreads) void k_head_bwd(const float *__restrict__ y, const float *__restrict__ W,
                                                           const float *__restrict__ logits,
                                                           const int *__restrict__ labels, float *__restrict__ gy,
                                                           float *__restrict__ gW, float *__restrict__ gbias,
                                                           long long F, int B, int classes) {
  extern __shared__ float dl[];  // [B][classes]
  for (int b = threadIdx.x; b < B; b += kHeadThreads) {
    float mx = -INFINITY;
    for (int o = 0; o < classes; ++o) mx = fmaxf(mx, logits[b * classes + o]);
    float se = 0.f;
    for (int o = 0; o < classes; ++o) se += expf(logits[b * classes + o] - mx);
    const int lab = labels[b];
    const bool ok = lab >= 0 && lab < classes;
    for (int o = 0; o < classes; ++o) {
      const float p = expf(logits[b * classes + o] - mx) / se;
      dl[b * classes + o] = ok ? (p - (o == lab ? 1.f : 0.f)) / (float)B : NAN;
    }
  }
  __syncthreads();
  if (blockIdx.x == 0 && (int)threadIdx.x < classes) {
    float s = 0.f;
    for (int b = 0; b < B; ++b) s += dl[b * classes + threadIdx.x];
    gbias[threadIdx.x] = s;
  }
  const long long f = (long long)blockIdx.x * kHeadThreads + threadIdx.x;
  if (f >= F) return;
  float w[kHeadMaxClasses], g[kHeadMaxClasses];
#pragma unroll
  for (int o = 0; o < kHeadMaxClasses; ++o) {
    w[o] = o < classes ? W[(long long)o * F + f] : 0.f;
    g[o] = 0.f;
  }
  for (int b = 0; b < B; ++b) {
    const float v = y[(long long)b * F + f];
    const float r = fmaxf(v, 0.f);
    float d = 0.f;
#pragma unroll
    for (int o = 0; o < kHeadMaxClasses; ++o)
      if (o < classes) {
        g[o] = fmaf(dl[b * classes + o], r, g[o]);
        d = fmaf(dl[b * classes + o], w[o], d);
      }
    if (gy) gy[(long long)b * F + f] = v > 0.f ? d : 0.f;
  }
#pragma unroll
  for (int o = 0; o < kHeadMaxClasses; ++o)
    if (o < classes) gW[(long long)o * F + f] = g[o];
}

// Adam (Kingma and Ba) as PyTorch states it, weight decay added to the gradient:
//   g' = g + wd p;  m = b1 m + (1 - b1) g';  v = b2 v + (1 - b2) g'^2;
//   p -= lr / (1 - b1^t) * m / (sqrt(v) / sqrt(1 - b2^t) + eps),
// t = *count + 1 (the steps taken so far are read from device memory, so that a
// captured graph advances on every replay; k_adam_count stores t afterwards).
__device__ __forceinline__ void adam_one(float &p, float g, float &m, float &v, float step_size, float sqrt_bc2,
                                         float beta1, float beta2, float eps, float wd) {
  const float gi = fmaf(wd, p, g);
  m = fmaf(beta1, m, (1.f - beta1) * gi);
  v = fmaf(beta2, v, (1.f - beta2) * gi * gi);
  p = p - step_size * (m / (sqrtf(v) / sqrt_bc2 + eps));
}

// VEC: the arrays are 16-byte aligned and each thread takes float4 runs (the last
// n mod 4 elements one by one); otherwise one float at a time.
template <bool VEC>
__global__ __launch_bounds__(256) void k_adam(float *__restrict__ p, const float *__restrict__ g,
                                              float *__restrict__ m, float *__restrict__ v, long long n,
                                              const int *__restrict__ count, float lr, float beta1, float beta2,
                                              float eps, float wd) {
  const float t = (float)(count[0] + 1);
  const float step_size = lr / (1.f - powf(beta1, t)), sqrt_bc2 = sqrtf(1.f - powf(beta2, t));
  const long long stride = (long long)gridDim.x * blockDim.x;
  long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if constexpr (VEC) {
    const long long n4 = n / 4;
    float4 *p4 = reinterpret_cast<float4 *>(p), *m4 = reinterpret_cast<float4 *>(m), *v4 = reinterpret_cast<float4 *>(v);
    const float4 *g4 = reinterpret_cast<const float4 *>(g);
    for (long long j = i; j < n4; j += stride) {
      float4 pp = p4[j], mm = m4[j], vv = v4[j];
      const float4 gg = g4[j];
      adam_one(pp.x, gg.x, mm.x, vv.x, step_size, sqrt_bc2, beta1, beta2, eps, wd);
      adam_one(pp.y, gg.y, mm.y, vv.y, step_size, sqrt_bc2, beta1, beta2, eps, wd);
      adam_one(pp.z, gg.z, mm.z, vv.z, step_size, sqrt_bc2, beta1, beta2, eps, wd);
      adam_one(pp.w, gg.w, mm.w, vv.w, step_size, sqrt_bc2, beta1, beta2, eps, wd);
      p4[j] = pp, m4[j] = mm, v4[j] = vv;
    }
    i += 4 * n4;  // the tail, one element per thread
  }
  for (; i < n; i += stride) {
    float pp = p[i], mm = m[i], vv = v[i];
    adam_one(pp, g[i], mm, vv, step_size, sqrt_bc2, beta1, beta2, eps, wd);
    p[i] = pp, m[i] = mm, v[i] = vv;
  }
}

__global__ void k_adam_count(int *count) {
  if (threadIdx.x == 0) count[0] += 1;
}

hipError_t launch_head_forward(const float *y, const float *W, const float *bias, const int *labels, float *logits,
                               float *loss, float *part, int B, long long F, int classes, hipStream_t s) {
  const long long chunks = head_chunks(F);
  if (chunks >= (1LL << 31) || B > 65535) return hipErrorInvalidValue;
  const hipError_t e = timed_launch("head_fwd", k_head_fwd, dim3((unsigned)chunks, (unsigned)B), dim3(kHeadThreads), 0,
                                    s, y, W, part, F, classes, (int)chunks);
  if (e != hipSuccess) return e;
  return timed_launch("head_loss", k_head_loss, dim3(1), dim3(kHeadThreads), (size_t)B * classes * sizeof(float), s,
                      part, bias, labels, logits, loss, B, classes, (int)chunks);
}

// Partial logits of the allocation-free forward (fdc_head_forward_noalloc): one array
// per device, resident while the library is loaded, shared by every call on that
// device.  In host code `scratch` names a host-side stand-in; kernels get the device
// address that hipGetSymbolAddress returns for the current device.
static __device__ __align__(256) float scratch[kHeadScratchFloats];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
float *g_scratch_ptr[kMaxDevices];  // device address of `scratch`, per device (nullptr: not yet looked up)
}  // namespace

hipError_t head_scratch_address(float **out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> g(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void *ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (ptr == nullptr) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = static_cast<float *>(ptr);
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

hipError_t launch_head_forward_noalloc(const float *y, const float *W, const float *bias, const int *labels,
                                       float *logits, float *loss, int B, long long F, int classes, hipStream_t s) {
  if (head_chunks(F) * B * classes > kHeadScratchFloats) return hipErrorInvalidValue;
  float *part = nullptr;
  const hipError_t e = head_scratch_address(&part);
  if (e != hipSuccess) return e;
  // every partial-logit slot the loss kernel reads is written first by k_head_fwd, so
  // nothing needs clearing between calls
  return launch_head_forward(y, W, bias, labels, logits, loss, part, B, F, classes, s);
}

hipError_t launch_head_backward(const float *y, const float *W, const float *logits, const int *labels, float *gy,
                                float *gW, float *gbias, int B, long long F, int classes, hipStream_t s) {
  const long long blocks = (F + kHeadThreads - 1) / kHeadThreads;
  if (blocks >= (1LL << 31)) return hipErrorInvalidValue;
  const size_t lds = (size_t)B * classes * sizeof(float);
  return timed_launch("head_bwd", k_head_bwd, dim3((unsigned)blocks), dim3(kHeadThreads), lds, s, y, W, logits, labels,
                      gy, gW, gbias, F, B, classes);
}

hipError_t launch_adam(float *p, const float *g, float *m, float *v, long long n, int *count, float lr, float beta1,
                       float beta2, float eps, float wd, hipStream_t s) {
  const auto aligned = [](const void *q) { return (reinterpret_cast<uintptr_t>(q) & 15) == 0; };
  const bool vec = aligned(p) && aligned(g) && aligned(m) && aligned(v);
  long long blocks = ((vec ? (n + 3) / 4 : n) + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  hipError_t e = hipSuccess;
  if (blocks > 0) {
    if (vec)
      e = timed_launch("adam", k_adam<true>, dim3((unsigned)blocks), dim3(256), 0, s, p, g, m, v, n, count, lr, beta1,
                       beta2, eps, wd);
    else
      e = timed_launch("adam", k_adam<false>, dim3((unsigned)blocks), dim3(256), 0, s, p, g, m, v, n, count, lr, beta1,
                       beta2, eps, wd);
    if (e != hipSuccess) return e;
  }
  return timed_launch("adam_count", k_adam_count, dim3(1), dim3(64), 0, s, count);
}

}  // namespace fdc
