// Exact fp32 causal softmax-prior FEM read on the vector units.
//
// For fp32 inputs the read must be accurate to ~1e-4, which bf16 matrix-core
// operands cannot give; this path evaluates, per (b, h, t, j),
//   F = [ LSE_{i<=t}(s_{t,i} + beta_j v_{i,j}) - LSE_{i<=t}(s_{t,i}) ] / beta_j
// with s_{t,i} = q_t . k_i / sqrt(d) in fp32 (free-energy read, Sec. 2.3, with
// the softmax prior of Sec. 1 written as log sum alpha e^{beta v} =
// log sum e^{s + beta v} - log sum e^{s}).  Each log-sum-exp is streamed with
// its own joint running maximum per (t, j), so there is no shared shift and no
// underflow path.  Work is O(T^2 d) with one exponential per (t, i, j): this is
// the accuracy path for fp32 inputs, not the throughput path.
//
// One workgroup per (b, h, t); its threads first compute a chunk of scores
// into LDS (one key per thread), then stream them, one channel per thread.

#include "fem_device.h"
#include "fem_internal.h"

namespace fem {
namespace {

constexpr int kThreads = 256;  // also the maximum d

__global__ __launch_bounds__(kThreads) void softmax_f32_kernel(
    const float* __restrict__ Q, const float* __restrict__ K, const float* __restrict__ V,
    const float* __restrict__ beta, float* __restrict__ out, int H, int T, int d) {
  __shared__ float sq[kThreads];
  __shared__ float ss[kThreads];

  const int tid = threadIdx.x;
  const int t = T - 1 - (int)blockIdx.x;  // longest rows first
  const int bh = blockIdx.y;
  const int h = bh % H;
  const size_t base = (size_t)bh * T * d;
  const float scale2 = kLog2e / sqrtf((float)d);

  if (tid < d) sq[tid] = Q[base + (size_t)t * d + tid];
  const bool own = tid < d;
  const float bl = own ? beta[h * d + tid] * kLog2e : 1.f;

  Lse2 num, den;
  for (int i0 = 0; i0 <= t; i0 += kThreads) {
    __syncthreads();  // sq ready / previous chunk consumed
    const int i = i0 + tid;
    float s = -INFINITY;
    if (i <= t) {
      const float* kr = K + base + (size_t)i * d;
      float dot = 0.f;
      for (int c = 0; c < d; ++c) dot = fmaf(sq[c], kr[c], dot);
      s = dot * scale2;
    }
    ss[tid] = s;
    __syncthreads();
    const int cnt = min(kThreads, t - i0 + 1);
    if (own) {
      const float* vc = V + base + (size_t)i0 * d + tid;
      for (int r = 0; r < cnt; ++r) {
        const float sr = ss[r];
        den.add(sr);
        num.add(fmaf(vc[(size_t)r * d], bl, sr));
      }
    }
  }
  if (own) out[base + (size_t)t * d + tid] = ((num.m + log2_hw(num.s)) - (den.m + log2_hw(den.s))) / bl;
}

}  // namespace

hipError_t launch_softmax_f32(const float* Q, const float* K, const float* V, const float* beta,
                              float* out, int B, int H, int T, int d, hipStream_t stream) {
  if (d < 1 || d > kThreads) return hipErrorInvalidValue;
  dim3 grid((unsigned)T, (unsigned)(B * H)), block(kThreads);
  hipLaunchKernelGGL(softmax_f32_kernel, grid, block, 0, stream, Q, K, V, beta, out, H, T, d);
  return hipGetLastError();
}

}  // namespace fem
