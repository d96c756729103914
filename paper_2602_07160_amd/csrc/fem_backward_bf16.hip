// Backward pass of the causal softmax-prior FEM read (bf16 inputs, fp32
// gradients).
//
// With s_ti = q_t.k_i / sqrt d, prior p_t(i) = softmax_{i<=t}(s_ti), read
// F_tj = (1/beta_j) log sum_i p_t(i) e^{beta_j v_ij} and upstream gradient
// G_tj, the paper's closed forms give
//   dL/dv_ij   = sum_t G_tj q_tj(i)                          (posterior as the
//                value gradient, Proposition "Local geometry", eq.
//                app-grad-hess)
//   dL/ds_ti   = sum_j (G_tj/beta_j) (q_tj(i) - p_t(i))      (normalized-logit
//                gradient, prior sensitivity (iv))
//   dL/dbeta_j = sum_t G_tj KL(q_tj || p_t) / beta_j^2       (eq. app-beta-deriv)
//              = sum_t G_tj (E_{q_tj}[v_j] - F_tj) / beta_j
// with the posterior q_tj(i) = p_t(i) e^{beta_j (v_ij - F_tj)}.
//
// The posterior is evaluated element by element in the exponent domain,
//   q_tj(i) = 2^{(s_ti log2e - lse_t log2e) + (beta_j log2e)(v_ij - F_tj)},
// from the forward's log-normaliser lse and output F: the exponent is at
// most 0 up to rounding, so nothing overflows, and no shared shift can
// underflow an in-support term.  That is T^2 d / 2 exponentials, on the
// vector units; the contractions around it run on the matrix cores:
//   kv kernel: one workgroup per (b, h, 64-key tile), over the query tiles
//              at or after its diagonal: S = Q K^T (MFMA), the posterior loop
//              (thread = key, channel quarter) accumulates dV and forms dS,
//              then dK += dS^T Q (MFMA);
//   q kernel:  one workgroup per (b, h, 64-query tile), over the key tiles up
//              to its diagonal: S = Q K^T, the posterior loop (thread = query,
//              channel quarter) forms dS, then dQ += dS K (MFMA).  It also
//              sums, per (t, j), Z = sum_i q^_tj(i) and X = sum_i q^_tj(i)
//              (v_ij - F^_tj) over the unnormalised posterior q^ built from
//              the forward's F^ and lse, and P = sum_i p^_t(i): since
//              F = F^ + ln(Z/P)/beta exactly, E_q[v] - F = X/Z - ln(Z/P)/beta,
//              in which the forward's rounding of F^ and lse cancels (it would
//              otherwise swamp the small difference E_q[v] - F ~ beta Var/2
//              at small beta);
//   dbeta:     per (h, j), the q kernel's per-tile sums of
//              G (E_q[v] - F) / beta, added in double precision.
// No atomics: every output is written by exactly one workgroup.

#include "fem_device.h"
#include "fem_internal.h"

#include <mutex>

namespace fem {
namespace {

constexpr int kTile = 64;   // queries and keys per tile
constexpr int kThreads = 256;
constexpr int kJG = 4;      // channel quarters per key (kv) or query (q)

template <int D>
struct Bw {
  static constexpr int JPT = D / kJG;     // channels per thread in the posterior loop
  static constexpr int ROW = D + 8;       // bf16 row stride of a [64][D] tile (16 B pad)
  static constexpr int TROW = kTile + 8;  // bf16 row stride of a [D][64] or [64][64] tile
  static constexpr int SROW = kTile + 1;  // fp32 row stride of the score tile
  static constexpr int NKS = D / 16;      // k-steps of Q K^T
  static constexpr int NCB = D / 32;      // 32-column output blocks of dK / dQ
  static_assert(JPT % 4 == 0, "float4 channel groups");
};

// ---- shared tile helpers -------------------------------------------------

// Copy rows [r0, r0 + 64) of a [T, D] bf16 matrix into LDS, row-major (row
// stride ROW) and, if tr, also transposed ([D][64], stride TROW).  Rows at or
// past T are zero.
template <int D>
__device__ __forceinline__ void stage_tile(const bf16* __restrict__ src, int r0, int T,
                                           bf16* rowm, bf16* trn) {
  using C = Bw<D>;
  constexpr int CPR = D / 8;  // 16-byte chunks per row
  for (int e = threadIdx.x; e < kTile * CPR; e += kThreads) {
    const int r = e / CPR, c8 = (e % CPR) * 8;
    bf16x8 x = {};
    if (r0 + r < T) x = *reinterpret_cast<const bf16x8*>(src + (size_t)(r0 + r) * D + c8);
    *reinterpret_cast<bf16x8*>(rowm + r * C::ROW + c8) = x;
    if (trn) {
#pragma unroll
      for (int u = 0; u < 8; ++u) trn[(c8 + u) * C::TROW + r] = x[u];
    }
  }
}

// S block (32 x 32) of wave-tile (qh, kh): rows qh*32.. of qt against rows
// kh*32.. of kt, contraction over D.  Lane (n, hl) gets key kh*32 + n and the
// query rows qh*32 + 8*(r/4) + 4*hl + r%4, r = 0..15.
template <int D>
__device__ __forceinline__ f32x16 score_block(const bf16* qt, const bf16* kt, int qh, int kh) {
  using C = Bw<D>;
  const int lane = threadIdx.x & 63, n = lane & 31, hl = lane >> 5;
  f32x16 acc = {};
#pragma unroll
  for (int ks = 0; ks < C::NKS; ++ks) {
    const bf16x8 a = *reinterpret_cast<const bf16x8*>(qt + (qh * 32 + n) * C::ROW + ks * 16 + hl * 8);
    const bf16x8 b = *reinterpret_cast<const bf16x8*>(kt + (kh * 32 + n) * C::ROW + ks * 16 + hl * 8);
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc, 0, 0, 0);
  }
  return acc;
}

// LDS of the kv kernel
template <int D>
struct KvSmem {
  using C = Bw<D>;
  bf16 kt[kTile * C::ROW];    // K tile [key][d]
  bf16 qt[kTile * C::ROW];    // Q tile [query][d]
  bf16 qT[D * C::TROW];       // Q tile transposed [d][query]
  bf16 dsT[kTile * C::TROW];  // dS^T [key][query]
  float sc[kTile * C::SROW];  // log2 p: s log2e - lse log2e, -inf off the support [query][key]
  float gq[kTile * D];        // G [query][j]
  float fb[kTile * D];        // beta log2e F [query][j]
  float dsum[kTile];          // sum_j G_tj / beta_j
};

// LDS of the q kernel
template <int D>
struct QSmem {
  using C = Bw<D>;
  bf16 qt[kTile * C::ROW];    // Q tile [query][d]
  bf16 kt[kTile * C::ROW];    // K tile [key][d]
  bf16 kT[D * C::TROW];       // K tile transposed [d][key]
  bf16 ds[kTile * C::TROW];   // dS [query][key]
  float sc[kTile * C::SROW];  // [query][key]
  float bv[kTile * D];        // beta log2e v [key][j]
};

// Scores of the (query tile q0, key tile k0) block into sm.sc as log2 p.
template <int D, class S>
__device__ __forceinline__ void block_logp(S& sm, const float* lse2, int q0, int k0, int T) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, n = lane & 31, hl = lane >> 5;
  const int qh = wave >> 1, kh = wave & 1;
  const f32x16 acc = score_block<D>(sm.qt, sm.kt, qh, kh);
  const float scale2 = kLog2e / sqrtf((float)D);
  const int i = kh * 32 + n;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int t = qh * 32 + 8 * (r >> 2) + 4 * hl + (r & 3);
    const bool ok = k0 + i <= q0 + t && q0 + t < T && k0 + i < T;
    sm.sc[t * Bw<D>::SROW + i] = ok ? fmaf(acc[r], scale2, -lse2[t]) : -INFINITY;
  }
}

// ---- kv kernel: dK, dV -----------------------------------------------------

template <int D>
__global__ __launch_bounds__(kThreads) void bwd_kv_kernel(
    const bf16* __restrict__ Q, const bf16* __restrict__ K, const bf16* __restrict__ V,
    const float* __restrict__ beta, const float* __restrict__ F, const float* __restrict__ lse,
    const float* __restrict__ G, float* __restrict__ dK, float* __restrict__ dV, int H, int T,
    int ntile) {
  using C = Bw<D>;
  __shared__ __align__(16) KvSmem<D> sm;
  __shared__ float lse2[kTile];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, n = lane & 31, hl = lane >> 5;
  const int kb = blockIdx.x % ntile, bh = blockIdx.x / ntile, h = bh % H;
  const int k0 = kb * kTile;
  const size_t base = (size_t)bh * T * D;

  // posterior-loop mapping: key ki, channels jg*JPT ..
  const int ki = tid >> 2, jg = tid & 3, j0 = jg * C::JPT;
  float bv[C::JPT], ib[C::JPT], dv[C::JPT];
#pragma unroll
  for (int u = 0; u < C::JPT; ++u) {
    const float b = beta[h * D + j0 + u];
    const float vv = k0 + ki < T ? (float)V[base + (size_t)(k0 + ki) * D + j0 + u] : 0.f;
    bv[u] = b * kLog2e * vv;
    ib[u] = 1.f / b;
    dv[u] = 0.f;
  }
  stage_tile<D>(K + base, k0, T, sm.kt, nullptr);

  // dK accumulators: wave (kh = wave & 1, dh = wave >> 1) owns keys kh*32..,
  // output blocks cb = dh, dh + 2, ... of the d columns
  const int kh = wave & 1, dh = wave >> 1;
  f32x16 dk[(C::NCB + 1) / 2];
#pragma unroll
  for (int c = 0; c < (C::NCB + 1) / 2; ++c) dk[c] = f32x16{};

  const int qlast = (T - 1) / kTile;
  for (int qb = kb; qb <= qlast; ++qb) {
    const int q0 = qb * kTile;
    __syncthreads();  // the previous block's readers are done with the tiles
    stage_tile<D>(Q + base, q0, T, sm.qt, sm.qT);
    for (int e = tid; e < kTile * D / 4; e += kThreads) {
      const int t = e / (D / 4), c4 = (e % (D / 4)) * 4;
      f32x4 g = {}, f = {};
      if (q0 + t < T) {
        g = *reinterpret_cast<const f32x4*>(G + base + (size_t)(q0 + t) * D + c4);
        f = *reinterpret_cast<const f32x4*>(F + base + (size_t)(q0 + t) * D + c4);
      }
      f32x4 fbv;
#pragma unroll
      for (int u = 0; u < 4; ++u) fbv[u] = beta[h * D + c4 + u] * kLog2e * f[u];
      *reinterpret_cast<f32x4*>(sm.gq + t * D + c4) = g;
      *reinterpret_cast<f32x4*>(sm.fb + t * D + c4) = fbv;
    }
    if (tid < kTile) lse2[tid] = q0 + tid < T ? lse[(size_t)bh * T + q0 + tid] * kLog2e : 0.f;
    __syncthreads();
    // sum_j G_tj / beta_j: thread (row tid >> 2, quarter tid & 3), four lanes combined
    {
      const int t = tid >> 2;
      float s = 0.f;
      for (int u = 0; u < C::JPT; ++u) s += sm.gq[t * D + j0 + u] / beta[h * D + j0 + u];
      s += __shfl_xor(s, 1);
      s += __shfl_xor(s, 2);
      if (jg == 0) sm.dsum[t] = s;
    }
    block_logp<D>(sm, lse2, q0, k0, T);
    __syncthreads();

    // posterior loop: dV_ij += G_tj q_tj(i);  dS_ti = sum_j (G_tj/beta_j) q - p D_t
    for (int t = 0; t < kTile; ++t) {
      const float lp = sm.sc[t * C::SROW + ki];
      float ds = 0.f;
      if (lp != -INFINITY) {
        float part = 0.f;
#pragma unroll
        for (int u4 = 0; u4 < C::JPT; u4 += 4) {
          const f32x4 fb4 = *reinterpret_cast<const f32x4*>(sm.fb + t * D + j0 + u4);
          const f32x4 g4 = *reinterpret_cast<const f32x4*>(sm.gq + t * D + j0 + u4);
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const float gqv = g4[u] * exp2_hw(lp + (bv[u4 + u] - fb4[u]));
            dv[u4 + u] += gqv;
            part = fmaf(gqv, ib[u4 + u], part);
          }
        }
        ds = part;
      }
      ds += __shfl_xor(ds, 1);
      ds += __shfl_xor(ds, 2);
      if (jg == 0) {
        const float p = lp != -INFINITY ? exp2_hw(lp) : 0.f;
        sm.dsT[ki * C::TROW + t] = (bf16)(ds - p * sm.dsum[t]);
      }
    }
    __syncthreads();

    // dK(keys kh*32.., d block cb) += dS^T Q : contraction over the 64 queries
#pragma unroll
    for (int c = 0; c < (C::NCB + 1) / 2; ++c) {
      const int cb = dh + 2 * c;
      if (cb >= C::NCB) break;
#pragma unroll
      for (int ks = 0; ks < kTile / 16; ++ks) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(sm.dsT + (kh * 32 + n) * C::TROW + ks * 16 + hl * 8);
        const bf16x8 b = *reinterpret_cast<const bf16x8*>(sm.qT + (cb * 32 + n) * C::TROW + ks * 16 + hl * 8);
        dk[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, dk[c], 0, 0, 0);
      }
    }
  }

  // dV: thread (key ki, channels j0..)
  if (k0 + ki < T) {
#pragma unroll
    for (int u4 = 0; u4 < C::JPT; u4 += 4) {
      const f32x4 o = {dv[u4], dv[u4 + 1], dv[u4 + 2], dv[u4 + 3]};
      *reinterpret_cast<f32x4*>(dV + base + (size_t)(k0 + ki) * D + j0 + u4) = o;
    }
  }
  // dK = dS^T Q / sqrt d: lane (n, hl) holds d column cb*32 + n, keys kh*32 + 8(r/4) + 4hl + r%4
  const float rs = 1.f / sqrtf((float)D);
#pragma unroll
  for (int c = 0; c < (C::NCB + 1) / 2; ++c) {
    const int cb = dh + 2 * c;
    if (cb >= C::NCB) break;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int key = k0 + kh * 32 + 8 * (r >> 2) + 4 * hl + (r & 3);
      if (key < T) dK[base + (size_t)key * D + cb * 32 + n] = dk[c][r] * rs;
    }
  }
}

// ---- q kernel: dQ ----------------------------------------------------------

template <int D>
__global__ __launch_bounds__(kThreads) void bwd_q_kernel(
    const bf16* __restrict__ Q, const bf16* __restrict__ K, const bf16* __restrict__ V,
    const float* __restrict__ beta, const float* __restrict__ F, const float* __restrict__ lse,
    const float* __restrict__ G, float* __restrict__ dQ, float* __restrict__ dbp, int H, int T,
    int ntile) {
  using C = Bw<D>;
  __shared__ __align__(16) QSmem<D> sm;
  __shared__ float lse2[kTile];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, n = lane & 31, hl = lane >> 5;
  const int qb = ntile - 1 - blockIdx.x % ntile;  // longest causal extent first
  const int bh = blockIdx.x / ntile, h = bh % H;
  const int q0 = qb * kTile;
  const size_t base = (size_t)bh * T * D;

  // posterior-loop mapping: query qi, channels j0..
  const int qi = tid >> 2, jg = tid & 3, j0 = jg * C::JPT;
  float fb[C::JPT], w[C::JPT], dsum = 0.f;
  float zs[C::JPT], xs[C::JPT];  // sum_i q^, sum_i q^ (beta log2e)(v - F^)
  float ps = 0.f;                // sum_i p^
#pragma unroll
  for (int u = 0; u < C::JPT; ++u) {
    const float b = beta[h * D + j0 + u];
    const bool ok = q0 + qi < T;
    const float g = ok ? G[base + (size_t)(q0 + qi) * D + j0 + u] : 0.f;
    const float f = ok ? F[base + (size_t)(q0 + qi) * D + j0 + u] : 0.f;
    fb[u] = b * kLog2e * f;
    w[u] = g / b;
    dsum += w[u];
    zs[u] = 0.f;
    xs[u] = 0.f;
  }
  dsum += __shfl_xor(dsum, 1);
  dsum += __shfl_xor(dsum, 2);
  if (tid < kTile) lse2[tid] = q0 + tid < T ? lse[(size_t)bh * T + q0 + tid] * kLog2e : 0.f;
  stage_tile<D>(Q + base, q0, T, sm.qt, nullptr);

  const int th = wave >> 1, dh = wave & 1;
  f32x16 dq[(C::NCB + 1) / 2];
#pragma unroll
  for (int c = 0; c < (C::NCB + 1) / 2; ++c) dq[c] = f32x16{};

  for (int kb = 0; kb <= qb; ++kb) {
    const int k0 = kb * kTile;
    __syncthreads();
    stage_tile<D>(K + base, k0, T, sm.kt, sm.kT);
    for (int e = tid; e < kTile * D / 8; e += kThreads) {
      const int i = e / (D / 8), c8 = (e % (D / 8)) * 8;
      bf16x8 x = {};
      if (k0 + i < T) x = *reinterpret_cast<const bf16x8*>(V + base + (size_t)(k0 + i) * D + c8);
#pragma unroll
      for (int u = 0; u < 8; ++u) sm.bv[i * D + c8 + u] = beta[h * D + c8 + u] * kLog2e * (float)x[u];
    }
    __syncthreads();
    block_logp<D>(sm, lse2, q0, k0, T);
    __syncthreads();

    for (int i = 0; i < kTile; ++i) {
      const float lp = sm.sc[qi * C::SROW + i];
      float ds = 0.f;
      if (lp != -INFINITY) {
        float part = 0.f;
        ps += exp2_hw(lp);
#pragma unroll
        for (int u4 = 0; u4 < C::JPT; u4 += 4) {
          const f32x4 bv4 = *reinterpret_cast<const f32x4*>(sm.bv + i * D + j0 + u4);
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const float x = bv4[u] - fb[u4 + u];
            const float e = exp2_hw(lp + x);
            part = fmaf(w[u4 + u], e, part);
            zs[u4 + u] += e;
            xs[u4 + u] = fmaf(e, x, xs[u4 + u]);
          }
        }
        ds = part;
      }
      ds += __shfl_xor(ds, 1);
      ds += __shfl_xor(ds, 2);
      if (jg == 0) {
        const float p = lp != -INFINITY ? exp2_hw(lp) : 0.f;
        sm.ds[qi * C::TROW + i] = (bf16)(ds - p * dsum);
      }
    }
    __syncthreads();

    // dQ(queries th*32.., d block cb) += dS K : contraction over the 64 keys
#pragma unroll
    for (int c = 0; c < (C::NCB + 1) / 2; ++c) {
      const int cb = dh + 2 * c;
      if (cb >= C::NCB) break;
#pragma unroll
      for (int ks = 0; ks < kTile / 16; ++ks) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(sm.ds + (th * 32 + n) * C::TROW + ks * 16 + hl * 8);
        const bf16x8 b = *reinterpret_cast<const bf16x8*>(sm.kT + (cb * 32 + n) * C::TROW + ks * 16 + hl * 8);
        dq[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, dq[c], 0, 0, 0);
      }
    }
  }

  const float rs = 1.f / sqrtf((float)D);
#pragma unroll
  for (int c = 0; c < (C::NCB + 1) / 2; ++c) {
    const int cb = dh + 2 * c;
    if (cb >= C::NCB) break;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int t = q0 + th * 32 + 8 * (r >> 2) + 4 * hl + (r & 3);
      if (t < T) dQ[base + (size_t)t * D + cb * 32 + n] = dq[c][r] * rs;
    }
  }

  // dbeta partial of this tile: sum_t G (X/Z - ln(Z/P)/beta)/beta, with
  // X/Z = sum_i q (v - F^) = xs / (Z beta log2e)
  __syncthreads();  // sm.bv is free: reuse it for the per-row terms
  float* contrib = sm.bv;
  const bool live = q0 + qi < T;
#pragma unroll
  for (int u = 0; u < C::JPT; ++u) {
    const float b = beta[h * D + j0 + u];
    float term = 0.f;
    if (live && zs[u] > 0.f) {
      const float eqv = xs[u] / (zs[u] * b * kLog2e) - (log2_hw(zs[u]) - log2_hw(ps)) * kLn2 / b;
      term = w[u] * eqv;  // G/beta * (E_q[v] - F)
    }
    contrib[qi * D + j0 + u] = term;
  }
  __syncthreads();
  for (int j = tid; j < D; j += kThreads) {
    float s = 0.f;
    for (int t = 0; t < kTile; ++t) s += contrib[t * D + j];
    dbp[((size_t)bh * ntile + qb) * D + j] = s;
  }
}

// ---- dbeta -----------------------------------------------------------------

// dbeta[h][j] = sum over (b, query tile) of the q kernel's partial sums.
template <int D>
__global__ void dbeta_final_kernel(const float* __restrict__ part, float* __restrict__ dbeta,
                                   int B, int H, int ntile) {
  const int h = blockIdx.x;
  for (int j = threadIdx.x; j < D; j += blockDim.x) {
    double s = 0.0;
    for (int b = 0; b < B; ++b)
      for (int c = 0; c < ntile; ++c) s += part[(((size_t)b * H + h) * ntile + c) * D + j];
    dbeta[h * D + j] = (float)s;
  }
}

template <int D>
hipError_t launch_bwd(const void* Q, const void* K, const void* V, const float* beta,
                      const float* out, const float* lse, const float* dout, float* dQ, float* dK,
                      float* dV, float* dbeta, int B, int H, int T, hipStream_t stream) {
  const int nbh = B * H;
  const int ntile = (T + kTile - 1) / kTile;
  const bf16* q = reinterpret_cast<const bf16*>(Q);
  const bf16* k = reinterpret_cast<const bf16*>(K);
  const bf16* v = reinterpret_cast<const bf16*>(V);
  hipLaunchKernelGGL(bwd_kv_kernel<D>, dim3((unsigned)(nbh * ntile)), dim3(kThreads), 0, stream, q,
                     k, v, beta, out, lse, dout, dK, dV, H, T, ntile);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  float* part = nullptr;
  e = workspace_alloc(reinterpret_cast<void**>(&part), (size_t)nbh * ntile * D * sizeof(float),
                      stream);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(bwd_q_kernel<D>, dim3((unsigned)(nbh * ntile)), dim3(kThreads), 0, stream, q,
                     k, v, beta, out, lse, dout, dQ, part, H, T, ntile);
  e = hipGetLastError();
  if (e == hipSuccess) {
    hipLaunchKernelGGL(dbeta_final_kernel<D>, dim3((unsigned)H), dim3(128), 0, stream, part, dbeta,
                       B, H, ntile);
    e = hipGetLastError();
  }
  const hipError_t f = workspace_free(part, stream);
  return e != hipSuccess ? e : f;
}

}  // namespace

hipError_t launch_softmax_bwd_bf16(const void* Q, const void* K, const void* V,
                                   const float* beta, const float* out, const float* lse,
                                   const float* dout, float* dQ, float* dK, float* dV,
                                   float* dbeta, int B, int H, int T, int d, hipStream_t stream) {
  switch (d) {
    case 32: return launch_bwd<32>(Q, K, V, beta, out, lse, dout, dQ, dK, dV, dbeta, B, H, T, stream);
    case 64: return launch_bwd<64>(Q, K, V, beta, out, lse, dout, dQ, dK, dV, dbeta, B, H, T, stream);
    case 128:
      return launch_bwd<128>(Q, K, V, beta, out, lse, dout, dQ, dK, dV, dbeta, B, H, T, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace fem
