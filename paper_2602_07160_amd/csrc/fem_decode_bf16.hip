// One decoding step of the softmax-prior FEM read against a KV cache.
//
// For every (b, h) a single new query q reads the first n = lens[b] cached
// keys and values (the new token's own k and v included):
//
//   F_j = (1/beta_j) log sum_{i<n} p(i) exp(beta_j v_{i,j}),
//   p(i) = softmax_{i<n}(q . k_i / sqrt d_qk)
//
// (free-energy read, Sec. 2.3; the autoregressive KV-cache setting of the
// softmax prior, Appendix "Parameterizations of the Prior Selection").
//
// The step reads every cached key and value once, so it is bound by HBM
// bandwidth; with one query there is no matrix product to feed the MFMA
// units.  The arithmetic is fp32 on the vector units and exact in form: each
// channel keeps its own joint log-sum-exp of x_{i,j} = s_i + beta_j log2(e)
// v_{i,j} (log2 units) with its own running maximum, and the read is
// LSE_j(x) - LSE(s), so there is no shared shift and no underflow case.
//
// Split-K: workgroup (split, b*H + h) covers keys [split*SL, (split+1)*SL)
// in blocks of 64, with the next block's K and V already loading while the
// current one is reduced.  Per block, four lanes form each of the 64 scores
// (a quarter of the dot product each, then two lane swaps); then each lane
// takes 8 consecutive channels of a few keys (16-byte V loads) and folds them
// into its running (max, sum) pairs.  The split's pairs are merged through
// LDS and written to a workspace; a second kernel merges the splits and
// forms the read.

#include "fem_device.h"
#include "fem_internal.h"

#include <atomic>
#include <math.h>

namespace fem {
namespace {

constexpr int kThreads = 256;
constexpr int kBlk = 64;  // keys per block

template <int DK, int DV>
struct Dec {
  static constexpr int KDIM = DK / 4;        // dims of one score lane
  static constexpr int KVEC = KDIM / 8;      // 16-byte K loads per lane and key
  static constexpr int NOCT = DV / 8;        // 8-channel groups
  static constexpr int NGRP = kThreads / NOCT;  // key groups
  static constexpr int KPG = kBlk / NGRP;    // keys per lane in the channel phase
  static_assert(KVEC >= 1 && KPG >= 1 && NGRP * NOCT == kThreads, "decode mapping");
};

// (max, sum) of 2^x over a set, combined with another such pair.
__device__ __forceinline__ void lse_merge(float& M, float& S, float m2, float s2) {
  const float mn = fmaxf(M, m2);
  if (mn == -INFINITY) return;
  S = S * exp2_hw(M - mn) + s2 * exp2_hw(m2 - mn);
  M = mn;
}

template <int DK, int DV>
__global__ __launch_bounds__(kThreads) void decode_partial_kernel(
    const bf16* __restrict__ q, const bf16* __restrict__ Kc, const bf16* __restrict__ Vc,
    const int* __restrict__ lens, const float* __restrict__ beta, float2* __restrict__ ws, int H,
    int L, int nsplit, int bps) {
  using C = Dec<DK, DV>;
  __shared__ float sc[2][kBlk];                 // block scores (log2 units)
  __shared__ float2 part[C::NGRP][DV + 1];      // per key group: channels, then the scores

  const int tid = threadIdx.x;
  const int split = blockIdx.x, bh = blockIdx.y;
  const int b = bh / H, h = bh % H;
  const int n0 = lens ? lens[b] : L;
  const int n = (n0 >= 1 && n0 <= L) ? n0 : 0;  // an invalid length reads nothing
  const int kbeg = split * bps * kBlk;
  const int kend = min(n, kbeg + bps * kBlk);
  const int nblk = kend > kbeg ? (kend - kbeg + kBlk - 1) / kBlk : 0;

  // score phase: key kk of the block, quarter qp of the dot product
  const int kk = tid >> 2, qp = tid & 3;
  // channel phase: channels 8*oc .. 8*oc+7 of keys grp*KPG ..
  const int oc = tid % C::NOCT, grp = tid / C::NOCT;

  const float qscale = kLog2e / sqrtf((float)DK);
  float qr[C::KDIM];
  {
    const bf16x8* qv = reinterpret_cast<const bf16x8*>(q + (size_t)bh * DK + qp * C::KDIM);
#pragma unroll
    for (int u = 0; u < C::KVEC; ++u) {
      const bf16x8 x = qv[u];
#pragma unroll
      for (int e = 0; e < 8; ++e) qr[u * 8 + e] = (float)x[e] * qscale;
    }
  }
  float bl[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) bl[e] = beta[h * DV + oc * 8 + e] * kLog2e;

  const bf16* Kh = Kc + (size_t)bh * L * DK;
  const bf16* Vh = Vc + (size_t)bh * L * DV;
  bf16x8 kr[C::KVEC], vr[C::KPG];
  auto load = [&](int blk) {
    const int k0 = kbeg + blk * kBlk;
    const int ik = min(k0 + kk, kend - 1);  // rows past the end re-read a valid row
#pragma unroll
    for (int u = 0; u < C::KVEC; ++u)
      kr[u] = *reinterpret_cast<const bf16x8*>(Kh + (size_t)ik * DK + qp * C::KDIM + u * 8);
#pragma unroll
    for (int r = 0; r < C::KPG; ++r) {
      const int iv = min(k0 + grp * C::KPG + r, kend - 1);
      vr[r] = *reinterpret_cast<const bf16x8*>(Vh + (size_t)iv * DV + oc * 8);
    }
  };

  float M[8], S[8], md = -INFINITY, sd = 0.f;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    M[e] = -INFINITY;
    S[e] = 0.f;
  }
  if (nblk > 0) load(0);
  for (int blk = 0; blk < nblk; ++blk) {
    const int k0 = kbeg + blk * kBlk;
    bf16x8 kc[C::KVEC], vc[C::KPG];
#pragma unroll
    for (int u = 0; u < C::KVEC; ++u) kc[u] = kr[u];
#pragma unroll
    for (int r = 0; r < C::KPG; ++r) vc[r] = vr[r];
    if (blk + 1 < nblk) load(blk + 1);

    float dot = 0.f;
#pragma unroll
    for (int u = 0; u < C::KVEC; ++u) {
#pragma unroll
      for (int e = 0; e < 8; ++e) dot = fmaf(qr[u * 8 + e], (float)kc[u][e], dot);
    }
    dot += __shfl_xor(dot, 1);
    dot += __shfl_xor(dot, 2);
    if (qp == 0) sc[blk & 1][kk] = (k0 + kk < kend) ? dot : -INFINITY;
    __syncthreads();

    float x[C::KPG][8];
    float bm[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) bm[e] = -INFINITY;
#pragma unroll
    for (int r = 0; r < C::KPG; ++r) {
      const float s = sc[blk & 1][grp * C::KPG + r];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        x[r][e] = fmaf(bl[e], (float)vc[r][e], s);
        bm[e] = fmaxf(bm[e], x[r][e]);
      }
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float mn = fmaxf(M[e], bm[e]);
      if (mn == -INFINITY) continue;  // every key of this lane is masked
      float acc = S[e] * exp2_hw(M[e] - mn);
#pragma unroll
      for (int r = 0; r < C::KPG; ++r) acc += exp2_hw(x[r][e] - mn);
      S[e] = acc;
      M[e] = mn;
    }
    if (oc == 0) {  // the prior's normaliser, once per key
      float sm = -INFINITY;
#pragma unroll
      for (int r = 0; r < C::KPG; ++r) sm = fmaxf(sm, sc[blk & 1][grp * C::KPG + r]);
      const float mn = fmaxf(md, sm);
      if (mn != -INFINITY) {
        float acc = sd * exp2_hw(md - mn);
#pragma unroll
        for (int r = 0; r < C::KPG; ++r) acc += exp2_hw(sc[blk & 1][grp * C::KPG + r] - mn);
        sd = acc;
        md = mn;
      }
    }
  }

  // merge the key groups of this split
#pragma unroll
  for (int e = 0; e < 8; ++e) part[grp][oc * 8 + e] = make_float2(M[e], S[e]);
  if (oc == 0) part[grp][DV] = make_float2(md, sd);
  __syncthreads();
  for (int j = tid; j <= DV; j += kThreads) {
    float Mj = -INFINITY, Sj = 0.f;
    for (int g = 0; g < C::NGRP; ++g) lse_merge(Mj, Sj, part[g][j].x, part[g][j].y);
    ws[((size_t)bh * nsplit + split) * (DV + 1) + j] = make_float2(Mj, Sj);
  }
}

template <int DV>
__global__ __launch_bounds__(kThreads) void decode_merge_kernel(
    const float2* __restrict__ ws, const int* __restrict__ lens, const float* __restrict__ beta,
    float* __restrict__ out, int H, int L, int nsplit) {
  const int bh = blockIdx.x;
  const int b = bh / H, h = bh % H;
  const int n0 = lens ? lens[b] : L;
  const bool valid = n0 >= 1 && n0 <= L;
  const float2* w = ws + (size_t)bh * nsplit * (DV + 1);
  float md = -INFINITY, sd = 0.f;
  for (int s = 0; s < nsplit; ++s) lse_merge(md, sd, w[s * (DV + 1) + DV].x, w[s * (DV + 1) + DV].y);
  for (int j = threadIdx.x; j < DV; j += kThreads) {
    float Mj = -INFINITY, Sj = 0.f;
    for (int s = 0; s < nsplit; ++s) lse_merge(Mj, Sj, w[s * (DV + 1) + j].x, w[s * (DV + 1) + j].y);
    const float bl = beta[h * DV + j] * kLog2e;
    const float o = ((Mj - md) + (log2_hw(Sj) - log2_hw(sd))) / bl;
    out[(size_t)bh * DV + j] = valid ? o : NAN;
  }
}

// Split count of a step: enough (b, h, split) workgroups for about one per
// compute unit of a 256-CU device, each split a whole number of key blocks.
// (At B8 H16 L4096 d128: one per CU 45.8 us, two 47.7, three 48.3, four
// 51.3; fewer, longer splits also shrink the merge.)
// A function of the sizes only, so that the workspace query needs no device.
constexpr int kTargetWorkgroups = 256;

void decode_splits(int B, int H, int L, int* nsplit_out, int* bps_out) {
  const int nbh = B * H;
  const int blocks = (L + kBlk - 1) / kBlk;
  int nsplit = (kTargetWorkgroups + nbh - 1) / nbh;
  nsplit = max(1, min(nsplit, blocks));
  const int bps = (blocks + nsplit - 1) / nsplit;
  *nsplit_out = (blocks + bps - 1) / bps;
  *bps_out = bps;
}

template <int DK, int DV>
hipError_t launch_decode(const void* q, const void* Kc, const void* Vc, const int* lens,
                         const float* beta, float* out, int B, int H, int L, void* wsv,
                         hipStream_t stream) {
  const int nbh = B * H;
  int nsplit, bps;
  decode_splits(B, H, L, &nsplit, &bps);
  if (nsplit > 65535 || nbh > 65535) return hipErrorInvalidValue;
  float2* ws = static_cast<float2*>(wsv);  // partials [nbh][nsplit][DV + 1]
  hipLaunchKernelGGL((decode_partial_kernel<DK, DV>), dim3((unsigned)nsplit, (unsigned)nbh),
                     dim3(kThreads), 0, stream, reinterpret_cast<const bf16*>(q),
                     reinterpret_cast<const bf16*>(Kc), reinterpret_cast<const bf16*>(Vc), lens,
                     beta, ws, H, L, nsplit, bps);
  hipError_t e = hipGetLastError();
  if (e == hipSuccess) {
    hipLaunchKernelGGL((decode_merge_kernel<DV>), dim3((unsigned)nbh), dim3(kThreads), 0, stream,
                       ws, lens, beta, out, H, L, nsplit);
    e = hipGetLastError();
  }
  return e;
}

}  // namespace

// Scratch of the entry point that allocates nothing (decode_noalloc): one
// array per device, held until the process ends.  Host code never passes the
// array's name to a kernel (on the host it is a stand-in, not the device
// address): the device address comes from hipGetSymbolAddress, once per
// device, and is kept below.
static __device__ __align__(256) unsigned char scratch[kNoallocScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch_addr[kMaxDevices];

// Device address of `scratch` on the current device (resolved on the first
// call on that device).
hipError_t scratch_address(void** p) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  void* a = g_scratch_addr[dev].load(std::memory_order_acquire);
  if (!a) {
    e = hipGetSymbolAddress(&a, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!a) return hipErrorInvalidSymbol;
    g_scratch_addr[dev].store(a, std::memory_order_release);
  }
  *p = a;
  return hipSuccess;
}
}  // namespace

hipError_t launch_decode_noalloc_bf16(const void* q, const void* Kc, const void* Vc,
                                      const int* lens, const float* beta, float* out, int B,
                                      int H, int L, int dk, int dv, hipStream_t stream) {
  if (decode_ws_bytes(B, H, L, dv) > kNoallocScratchBytes) return hipErrorInvalidValue;
  void* ws = nullptr;
  const hipError_t e = scratch_address(&ws);
  if (e != hipSuccess) return e;
  return launch_decode_bf16(q, Kc, Vc, lens, beta, out, B, H, L, dk, dv, ws, stream);
}

size_t decode_ws_bytes(int B, int H, int L, int dv) {
  int nsplit, bps;
  decode_splits(B, H, L, &nsplit, &bps);
  return (size_t)B * H * nsplit * (dv + 1) * sizeof(float2);
}

hipError_t launch_decode_bf16(const void* q, const void* Kc, const void* Vc, const int* lens,
                              const float* beta, float* out, int B, int H, int L, int dk, int dv,
                              void* ws, hipStream_t stream) {
  if (dk == 32 && dv == 32)
    return launch_decode<32, 32>(q, Kc, Vc, lens, beta, out, B, H, L, ws, stream);
  if (dk == 64 && dv == 64)
    return launch_decode<64, 64>(q, Kc, Vc, lens, beta, out, B, H, L, ws, stream);
  if (dk == 128 && dv == 128)
    return launch_decode<128, 128>(q, Kc, Vc, lens, beta, out, B, H, L, ws, stream);
  if (dk == 64 && dv == 32)
    return launch_decode<64, 32>(q, Kc, Vc, lens, beta, out, B, H, L, ws, stream);
  if (dk == 128 && dv == 64)
    return launch_decode<128, 64>(q, Kc, Vc, lens, beta, out, B, H, L, ws, stream);
  return hipErrorInvalidValue;
}

}  // namespace fem
