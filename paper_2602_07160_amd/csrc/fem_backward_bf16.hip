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
// Two evaluations of these sums live here.  The default one (the matrix-core
// path, below the element-wise kernels) factors the posterior ratio so that
// every sum over keys or channels is an MFMA product; it covers every channel
// whose beta-scaled value range fits fp32's exponent range.  Otherwise the
// element-wise kernels, exact in form for every beta > 0, redo the call:
//
// The posterior is evaluated element by element in the exponent domain,
//   q_tj(i) = 2^{(s_ti log2e - lse_t log2e) + (beta_j log2e)(v_ij - F_tj)},
// from the forward's log-normaliser lse and output F: the exponent is at
// most 0 up to rounding, so nothing overflows, and no shared shift can
// underflow an in-support term.  That is T^2 d / 2 exponentials, on the
// vector units; the contractions around it run on the matrix cores:
//   q kernel:  one workgroup per (b, h, 64-query tile), over the key tiles up
//              to its diagonal: S = Q K^T, the posterior loop (thread = query,
//              channel quarter) forms dS, then dQ += dS K (MFMA).  It also
//              sums, per (t, j), Z = sum_i q^_tj(i) and X = sum_i q^_tj(i)
//              (v_ij - F^_tj) over the unnormalised posterior q^ built from
//              the forward's F^ and lse, and P = sum_i p^_t(i): since
//              F = F^ + ln(Z/P)/beta exactly, E_q[v] - F = X/Z - ln(Z/P)/beta,
//              in which the forward's rounding of F^ and lse cancels (it would
//              otherwise swamp the small difference E_q[v] - F ~ beta Var/2
//              at small beta).  It writes beta log2e F for the kv kernel;
//   kv kernel: one workgroup per (b, h, 64-key tile), over the query tiles
//              at or after its diagonal: S = Q K^T (MFMA), the posterior loop
//              (thread = key, channel quarter) accumulates dV and forms dS
//              from the posterior at the q kernel's F, which sums to one over
//              the keys, then dK += dS^T Q (MFMA);
//   dbeta:     per (h, j), the q kernel's per-tile sums of
//              G (E_q[v] - F) / beta, added in double precision.
// No atomics: every output is written by exactly one workgroup.

#include "fem_device.h"
#include "fem_internal.h"

#include <cstddef>
#include <type_traits>

namespace fem {
namespace {

constexpr int kTile = 64;   // queries and keys per tile
constexpr int kThreads = 256;
constexpr int kJG = 4;      // channel quarters per key (kv) or query (q)

// Form of a channel (b, h, j), set from the range of beta log2e v over the
// sequence: the matrix-core pass uses R - 1 = E U - 1 (plain) or A U + (U - 1)
// with A = E - 1 (split, small ranges); a wide channel's factors leave fp32's
// range, so the element-wise kernels take that channel instead.
constexpr float kPlainForm = 0.f;
constexpr float kSplitForm = 1.f;
constexpr float kWide = 2.f;

// What the element-wise kernels do, from the flags the matrix-core pass set:
// nothing; the wide channels only, added to the matrix-core gradients
// (flag[1]); or every channel, replacing them (flag[0]: a factor of some
// other channel left fp32's range).
constexpr int kExactNone = 0, kExactWide = 1, kExactAll = 2;
__device__ __forceinline__ int exact_mode(const int* flag) {
  return flag[0] ? kExactAll : flag[1] ? kExactWide : kExactNone;
}

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
  constexpr int N = kTile * CPR / kThreads;
  static_assert(N * kThreads == kTile * CPR, "whole rounds");
  // every load of the tile is in flight before the first store
  bf16x8 x[N];
#pragma unroll
  for (int it = 0; it < N; ++it) {
    const int e = threadIdx.x + it * kThreads, r = e / CPR, c8 = (e % CPR) * 8;
    x[it] = bf16x8{};
    if (r0 + r < T) x[it] = *reinterpret_cast<const bf16x8*>(src + (size_t)(r0 + r) * D + c8);
  }
#pragma unroll
  for (int it = 0; it < N; ++it) {
    const int e = threadIdx.x + it * kThreads, r = e / CPR, c8 = (e % CPR) * 8;
    *reinterpret_cast<bf16x8*>(rowm + r * C::ROW + c8) = x[it];
    if (trn) {
#pragma unroll
      for (int u = 0; u < 8; ++u) trn[(c8 + u) * C::TROW + r] = x[it][u];
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

// FB: beta log2e F per (t, j) of the channels it takes, the read with the
// forward's rounding removed (written by bwd_q_kernel, which runs first).
template <int D>
__global__ __launch_bounds__(kThreads) void bwd_kv_kernel(
    const bf16* __restrict__ Q, const bf16* __restrict__ K, const bf16* __restrict__ V,
    const float* __restrict__ beta, const float* __restrict__ FB, const float* __restrict__ lse,
    const float* __restrict__ G, float* __restrict__ dK, float* __restrict__ dV, int H, int T,
    int ntile, const int* __restrict__ flag, const float* __restrict__ splitf) {
  using C = Bw<D>;
  static_assert(D <= kThreads && C::JPT <= 32, "channel masks");
  const int mode = exact_mode(flag);
  if (mode == kExactNone) return;  // the matrix-core pass took every channel
  const bool all = mode == kExactAll;
  const int tid = threadIdx.x;
  const int kb = blockIdx.x % ntile, bh = blockIdx.x / ntile, h = bh % H;
  // wide channels only: nothing to do for a (b, h) without one
  if (!all && !__syncthreads_or(tid < D && splitf[bh * D + tid] == kWide)) return;
  __shared__ __align__(16) KvSmem<D> sm;
  __shared__ float lse2[kTile];
  const int wave = tid >> 6, lane = tid & 63, n = lane & 31, hl = lane >> 5;
  const int k0 = kb * kTile;
  const size_t base = (size_t)bh * T * D;

  // posterior-loop mapping: key ki, channels jg*JPT ..; bit u of act: channel
  // j0 + u is taken here
  const int ki = tid >> 2, jg = tid & 3, j0 = jg * C::JPT;
  unsigned act = 0;
#pragma unroll
  for (int u = 0; u < C::JPT; ++u)
    if (all || splitf[bh * D + j0 + u] == kWide) act |= 1u << u;
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
    {
      // thread tid handles channels c4.. of rows tid / (D/4) + it * (kThreads / (D/4));
      // the G and F loads of a round are all in flight before its stores
      constexpr int N = kTile * D / 4 / kThreads, RPI = kThreads / (D / 4), NB = N >= 4 ? 4 : N;
      static_assert(N * kThreads == kTile * D / 4 && N % NB == 0, "whole rounds");
      const int c4 = (tid % (D / 4)) * 4, t0 = tid / (D / 4);
#pragma unroll
      for (int i0 = 0; i0 < N; i0 += NB) {
        f32x4 g[NB], f[NB];
#pragma unroll
        for (int i = 0; i < NB; ++i) {
          const int t = t0 + (i0 + i) * RPI;
          g[i] = f32x4{};
          f[i] = f32x4{};
          if (q0 + t < T) {
            g[i] = *reinterpret_cast<const f32x4*>(G + base + (size_t)(q0 + t) * D + c4);
            f[i] = *reinterpret_cast<const f32x4*>(FB + base + (size_t)(q0 + t) * D + c4);
          }
        }
#pragma unroll
        for (int i = 0; i < NB; ++i) {
          const int t = t0 + (i0 + i) * RPI;
          *reinterpret_cast<f32x4*>(sm.gq + t * D + c4) = g[i];
          // (channels not taken here hold stale values, never read)
          *reinterpret_cast<f32x4*>(sm.fb + t * D + c4) = f[i];
        }
      }
    }
    if (tid < kTile) lse2[tid] = q0 + tid < T ? lse[(size_t)bh * T + q0 + tid] * kLog2e : 0.f;
    __syncthreads();
    // sum_j G_tj / beta_j: thread (row tid >> 2, quarter tid & 3), four lanes combined
    {
      const int t = tid >> 2;
      float s = 0.f;
      // (t, j0..) is also this thread's posterior channel range: ib holds 1/beta
#pragma unroll
      for (int u4 = 0; u4 < C::JPT; u4 += 4) {
        const f32x4 g4 = *reinterpret_cast<const f32x4*>(sm.gq + t * D + j0 + u4);
#pragma unroll
        for (int u = 0; u < 4; ++u)
          s += ((act >> (u4 + u)) & 1) ? g4[u] * ib[u4 + u] : 0.f;
      }
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
          if (!((act >> u4) & 0xfu)) continue;
          const f32x4 fb4 = *reinterpret_cast<const f32x4*>(sm.fb + t * D + j0 + u4);
          const f32x4 g4 = *reinterpret_cast<const f32x4*>(sm.gq + t * D + j0 + u4);
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const float gqv =
                ((act >> (u4 + u)) & 1) ? g4[u] * exp2_hw(lp + (bv[u4 + u] - fb4[u])) : 0.f;
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

  // dV: thread (key ki, channels j0..); the columns taken here only
  if (k0 + ki < T) {
#pragma unroll
    for (int u4 = 0; u4 < C::JPT; u4 += 4) {
      float* at = dV + base + (size_t)(k0 + ki) * D + j0 + u4;
      if (all) {
        *reinterpret_cast<f32x4*>(at) = f32x4{dv[u4], dv[u4 + 1], dv[u4 + 2], dv[u4 + 3]};
      } else {
#pragma unroll
        for (int u = 0; u < 4; ++u)
          if ((act >> (u4 + u)) & 1) at[u] = dv[u4 + u];
      }
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
      if (key >= T) continue;
      float* at = dK + base + (size_t)key * D + cb * 32 + n;
      *at = all ? dk[c][r] * rs : *at + dk[c][r] * rs;  // wide only: add to the matrix-core dK
    }
  }
}

// ---- q kernel: dQ ----------------------------------------------------------

template <int D>
__global__ __launch_bounds__(kThreads) void bwd_q_kernel(
    const bf16* __restrict__ Q, const bf16* __restrict__ K, const bf16* __restrict__ V,
    const float* __restrict__ beta, const float* __restrict__ F, const float* __restrict__ lse,
    const float* __restrict__ G, float* __restrict__ dQ, float* __restrict__ dbp,
    float* __restrict__ FB, int H, int T, int ntile, const int* __restrict__ flag,
    const float* __restrict__ splitf) {
  using C = Bw<D>;
  static_assert(D <= kThreads && C::JPT <= 32, "channel masks");
  const int mode = exact_mode(flag);
  if (mode == kExactNone) return;
  const bool all = mode == kExactAll;
  if (!all && !__syncthreads_or(threadIdx.x < D &&
                                splitf[(blockIdx.x / ntile) * D + threadIdx.x] == kWide))
    return;
  __shared__ __align__(16) QSmem<D> sm;
  __shared__ float lse2[kTile];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, n = lane & 31, hl = lane >> 5;
  const int qb = ntile - 1 - blockIdx.x % ntile;  // longest causal extent first
  const int bh = blockIdx.x / ntile, h = bh % H;
  const int q0 = qb * kTile;
  const size_t base = (size_t)bh * T * D;

  // posterior-loop mapping: query qi, channels j0..; bit u of act: channel
  // j0 + u is taken here (a channel not taken has W = 0 and no posterior)
  const int qi = tid >> 2, jg = tid & 3, j0 = jg * C::JPT;
  unsigned act = 0;
#pragma unroll
  for (int u = 0; u < C::JPT; ++u)
    if (all || splitf[bh * D + j0 + u] == kWide) act |= 1u << u;
  float fb[C::JPT], w[C::JPT], dsum = 0.f;
  float zs[C::JPT], xs[C::JPT];  // sum_i q^, sum_i q^ (beta log2e)(v - F^)
  float ps = 0.f;                // sum_i p^
#pragma unroll
  for (int u = 0; u < C::JPT; ++u) {
    const float b = beta[h * D + j0 + u];
    const bool ok = q0 + qi < T && ((act >> u) & 1);
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
    {
      // thread tid handles channels c8.. of rows tid / (D/8) + it * (kThreads / (D/8))
      constexpr int N = kTile * D / 8 / kThreads, RPI = kThreads / (D / 8);
      static_assert(N * kThreads == kTile * D / 8, "whole rounds");
      const int c8 = (tid % (D / 8)) * 8, i0 = tid / (D / 8);
      bf16x8 x[N];
#pragma unroll
      for (int it = 0; it < N; ++it) {
        const int i = i0 + it * RPI;
        x[it] = bf16x8{};
        if (k0 + i < T) x[it] = *reinterpret_cast<const bf16x8*>(V + base + (size_t)(k0 + i) * D + c8);
      }
#pragma unroll
      for (int it = 0; it < N; ++it) {
        const int i = i0 + it * RPI;
#pragma unroll
        for (int u = 0; u < 8; ++u)
          sm.bv[i * D + c8 + u] = beta[h * D + c8 + u] * kLog2e * (float)x[it][u];
      }
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
          if (!((act >> u4) & 0xfu)) continue;
          const f32x4 bv4 = *reinterpret_cast<const f32x4*>(sm.bv + i * D + j0 + u4);
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const float x = bv4[u] - fb[u4 + u];
            const float e = ((act >> (u4 + u)) & 1) ? exp2_hw(lp + x) : 0.f;
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
      if (t >= T) continue;
      float* at = dQ + base + (size_t)t * D + cb * 32 + n;
      *at = all ? dq[c][r] * rs : *at + dq[c][r] * rs;  // wide only: add to the matrix-core dQ
    }
  }

  // The read with the forward's rounding removed, beta log2e F = beta log2e
  // F^ + log2(Z/P), for the kv kernel: its posterior then sums to one over
  // the keys, and so do the dV and dS it forms.
  if (q0 + qi < T) {
#pragma unroll
    for (int u = 0; u < C::JPT; ++u)
      if ((act >> u) & 1)
        FB[base + (size_t)(q0 + qi) * D + j0 + u] =
            zs[u] > 0.f ? fb[u] + (log2_hw(zs[u]) - log2_hw(ps)) : fb[u];
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

// ---- matrix-core path ------------------------------------------------------
//
// With c_j a per-channel constant, q_tj(i) = p_ti E_ij U_tj, E_ij =
// 2^{bl_j v_ij - c_j}, U_tj = 2^{c_j - bl_j F^_tj} (bl = beta log2 e), so
//   dS_ti = p_ti sum_j W_tj (R_tij - 1),   R = E U,   W = G / beta,
//   dV_ij = E_ij sum_t p_ti G_tj U_tj
// are products over j and over t.  c_j = bl_j max v_.j over the (b, h)'s
// whole sequence, so E depends on the key alone and U on the query alone:
// both are formed once, in the layouts the matrix cores read, and the passes
// over tile pairs only stream them.  Two forms per channel:
//   split (bl_j times the range of v_.j <= 4): R - 1 = A U + (U - 1) with
//     A = E - 1 (expm1): the product sum_j (W U) A and the row constant
//     sum_j W (U - 1) carry no cancellation when beta is small (|A|, |U - 1|
//     are small, U in [1, 2^4]);
//   plain (otherwise): R - 1 = E U - 1, row constant -sum_j W.
// Both factors enter as bf16 hi + lo parts (three MFMAs, ~2^-16 relative).
// Since out lies between the smallest and the largest v it averages,
// E >= 2^-L and U <= 2^L with L = bl (max v - min v); with L <= 110 every
// factor, product and sum stays inside fp32's normal range (the dV sums
// sum_t p G U are at most T max|G| 2^L).  A channel with a wider range, or a
// row whose W U would leave that range, sets a device flag; the element-wise
// kernels then redo the whole pass, and otherwise return at once.
// p comes from the forward's lse, which sums bf16-rounded probabilities and
// so may be off by a few 2^-9: the q pass sums P = sum_i p per row exactly,
// divides its products by P and hands lse + ln P to the kv pass, so both use
// rows of p that sum to one to fp32 accuracy.
//
// Normalisation: R^ built from the forward's F^ gives sum_i p R^ = Z/P =
// e^{beta (F - F^)} != 1 (the forward rounds p to bf16).  The q kernel, which
// sees every key of its rows, forms ln(Z/P) per (t, j) from SA = sum_i p Y
// (Y = A or E): split, Z/P - 1 = (U - 1) + U SA / P; plain, Z/P = U SA / P.
// The kv pass then uses the normalised posterior, U' = U / (Z/P).  So
// dbeta = sum_t G (E_q[v] - F) / beta = (sum_i v dV - sum_t G F) / beta with
// F = F^ + ln(Z/P)/beta is formed from normalised quantities; its terms are
// small next to their parts (~ beta Var/2 at small beta, ~ KL/beta at large).
//
// Kernels, in stream order:
//   vstats: per 64-row tile, each channel's max and min v;
//   prepk: c_j and the channel form; Y row-major (hi and lo);
//   q:     per 64-query tile over its key tiles: S^T, p, dP^T = Y (W U)^T,
//          dS, dQ^T += K^T dS^T and SA^T += Y^T P^T; ln(Z/P), lse + ln P and
//          the G F^ terms of dbeta;
//   prepq: W U' row-major (hi and lo) and the row constants;
//   kv:    per 64-key tile over its query tiles: S, p, dP = (W U') Y^T, dS,
//          dV^T += (W U')^T P (dV = beta E times it) and dK^T += Q^T dS; the
//          v dV terms of dbeta;
//   dbeta: per (h, j), the partial sums in double precision.
// The streamed side of a pass (K, Y in the q pass; Q, W U' in the kv pass)
// goes global -> LDS by direct loads into a double buffer, one tile pair
// ahead, so the loads cost no registers and no waiting; the transposed
// operands (K^T, Y^T; Q^T, (W U')^T) are read from the same row-major tiles
// by transposing LDS reads (ds_read_b64_tr_b16).

__device__ __forceinline__ void split_bf16(float x, bf16& hi, bf16& lo) {
  hi = (bf16)x;
  lo = (bf16)(x - (float)hi);
}

// p and dS of a 32 x 32 block as MFMA B operands (k = the accumulator's
// rows): hi / lo parts of p and bf16 dS, two values per conversion.
// pc(r) gives accumulator row r's p and row constant c_r; dS = p (dP + c_r).
template <class PC>
__device__ __forceinline__ void pack_p_ds(PC&& pc, const f32x16& dp, bf16x8 (&ph)[2],
                                          bf16x8 (&pl)[2], bf16x8 (&ds)[2]) {
  typedef __attribute__((ext_vector_type(4))) unsigned u32x4;
  u32x4 h[2], l[2], d[2];
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    const f32x2 x = pc(2 * k), y = pc(2 * k + 1);  // (p, c)
    const float a = x[0], b = y[0];
    const unsigned hu = __builtin_bit_cast(unsigned, to_bf16x2(a, b));
    const float ha = __uint_as_float(hu << 16), hb = __uint_as_float(hu & 0xffff0000u);
    h[k >> 2][k & 3] = hu;
    l[k >> 2][k & 3] = __builtin_bit_cast(unsigned, to_bf16x2(a - ha, b - hb));
    d[k >> 2][k & 3] = __builtin_bit_cast(
        unsigned, to_bf16x2(a * (dp[2 * k] + x[1]), b * (dp[2 * k + 1] + y[1])));
  }
#pragma unroll
  for (int g = 0; g < 2; ++g) {
    ph[g] = __builtin_bit_cast(bf16x8, h[g]);
    pl[g] = __builtin_bit_cast(bf16x8, l[g]);
    ds[g] = __builtin_bit_cast(bf16x8, d[g]);
  }
}

__device__ __forceinline__ f32x16 mfma(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

constexpr float kRange = 110.f;  // largest bl (max v - min v) of a channel
constexpr float kSplit = 4.f;    // largest bl (max v - min v) of a split channel
constexpr float kGuardU = 120.f; // largest log2 U of a row
constexpr float kGuardW = 0x1p124f;

// Consecutive workgroups go to the eight XCDs in turn; this order hands each
// XCD a contiguous range of tiles (one (b, h) at a time), so the key or query
// tiles its workgroups stream stay in its own L2.
__device__ __forceinline__ int xcd_order(int b, int nblk) {
  if (nblk & 7) return b;
  return (b & 7) * (nblk >> 3) + (b >> 3);
}


// Direct global -> LDS copy of rows [0, 64) of a row-major [., D] bf16 source
// into a swizzled tile; rows past lim re-read row lim (their keys or queries
// are masked).  Wave w fills the 1 KiB blocks w, w + 4, ...: lane l of block
// b fills slot 64 b + l, i.e. row (64 b + l) / (D / 8), chunk position
// (64 b + l) % (D / 8), from the chunk that position holds.
template <int D>
__device__ __forceinline__ void load_swz(const bf16* __restrict__ src, bf16* dst, int lim) {
  constexpr int CPR = D / 8;
  static_assert(CPR % 4 == 0, "whole blocks per wave");
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const char* s8 = reinterpret_cast<const char*>(src);
#pragma unroll
  for (int u = 0; u < CPR / 4; ++u) {
    const int blk = wave + 4 * u;
    const int s = blk * 64 + lane, row = s / CPR, pos = s % CPR;
    const unsigned off = (unsigned)(min(row, lim) * D * 2 + ((pos ^ swz<D>(row)) << 4));
    dma16(s8 + off, dst + blk * 512);
  }
}

__device__ __forceinline__ void wait_vmem() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// Make the compiler complete the loads of x here: a use before the main loop
// keeps its wait for them out of the loop, where it would also wait for the
// direct loads in flight.
__device__ __forceinline__ void settle(const bf16x8& x) { asm volatile("" ::"v"(x)); }
__device__ __forceinline__ void settle(float x) { asm volatile("" ::"v"(x)); }


// Per 64-row tile of V, the max and min of each channel (for the channel
// shifts and forms); the first workgroup clears the fallback flags.
template <int D>
__global__ __launch_bounds__(kThreads) void bwd_vstats_kernel(const bf16* __restrict__ V,
                                                              float* __restrict__ vmx,
                                                              float* __restrict__ vmn,
                                                              int* __restrict__ flag, int T,
                                                              int ntile) {
  // thread: 8 consecutive channels (16-byte loads) of every RG-th row
  constexpr int CPR = D / 8, RG = kThreads / CPR;
  static_assert(kThreads % CPR == 0 && kTile % RG == 0, "vstats mapping");
  __shared__ float sx[RG][D], sn[RG][D];
  const int tid = threadIdx.x, c8 = (tid % CPR) * 8, rg = tid / CPR;
  const int tb = blockIdx.x % ntile, bh = blockIdx.x / ntile;
  const int r0 = tb * kTile;
  if (blockIdx.x == 0 && tid < 2) flag[tid] = 0;
  const bf16* Vh = V + (size_t)bh * T * D;
  float a[8], b[8];
#pragma unroll
  for (int u = 0; u < 8; ++u) {
    a[u] = -INFINITY;
    b[u] = INFINITY;
  }
  bf16x8 x[kTile / RG];
#pragma unroll
  for (int i = 0; i < kTile / RG; ++i) {  // every load first
    const int r = min(r0 + rg + RG * i, T - 1);  // rows past T repeat row T - 1
    x[i] = *reinterpret_cast<const bf16x8*>(Vh + (size_t)r * D + c8);
  }
#pragma unroll
  for (int i = 0; i < kTile / RG; ++i)
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      a[u] = fmaxf(a[u], (float)x[i][u]);
      b[u] = fminf(b[u], (float)x[i][u]);
    }
#pragma unroll
  for (int u = 0; u < 8; ++u) {
    sx[rg][c8 + u] = a[u];
    sn[rg][c8 + u] = b[u];
  }
  __syncthreads();
  for (int j = tid; j < D; j += kThreads) {
    float mx = sx[0][j], mn = sn[0][j];
    for (int g = 1; g < RG; ++g) {
      mx = fmaxf(mx, sx[g][j]);
      mn = fminf(mn, sn[g][j]);
    }
    vmx[((size_t)bh * ntile + tb) * D + j] = mx;
    vmn[((size_t)bh * ntile + tb) * D + j] = mn;
  }
}

// Channel constants of a (b, h) from the per-tile max / min of V: c_j, the
// form (kSplitForm, kPlainForm, or kWide for a channel whose range is beyond
// the matrix-core form: the element-wise pass takes it), and bl_j, into LDS;
// with publish, also to global memory, and a wide channel raises flag[1].
template <int D>
__device__ __forceinline__ void channel_consts(const float* __restrict__ beta,
                                               const float* __restrict__ vmx,
                                               const float* __restrict__ vmn, int bh, int h,
                                               int ntile, float* c, float* split, float* bl,
                                               bool publish, float* __restrict__ cg,
                                               float* __restrict__ splitf, int* __restrict__ flag) {
  for (int j = threadIdx.x; j < D; j += kThreads) {
    float a = -INFINITY, b = INFINITY;
    for (int k = 0; k < ntile; ++k) {
      a = fmaxf(a, vmx[((size_t)bh * ntile + k) * D + j]);
      b = fminf(b, vmn[((size_t)bh * ntile + k) * D + j]);
    }
    const float l = beta[h * D + j] * kLog2e, range = l * (a - b);
    const float sp = !(range <= kRange) ? kWide : range <= kSplit ? kSplitForm : kPlainForm;
    c[j] = l * a;
    split[j] = sp;
    bl[j] = l;
    if (publish) {
      cg[bh * D + j] = l * a;
      splitf[bh * D + j] = sp;
      if (sp == kWide) flag[1] = 1;
    }
  }
}

// Per 64-row tile of a (b, h): the channel constants (the first tile publishes
// them); for the rows as keys, Y = A (split) or E (plain), E = 2^{bl v - c};
// for the rows as queries of the q pass, W U with U = 2^{c - bl F} and the
// row constants sum_j (split ? W (U - 1) : -W).  Y and W U row-major, hi and
// lo parts, zero past T.  Thread e handles 8 channels of one row; the D/8
// threads of a row are adjacent lanes.
template <int D>
__global__ __launch_bounds__(kThreads) void bwd_prepk_kernel(
    const bf16* __restrict__ V, const float* __restrict__ beta, const float* __restrict__ F,
    const float* __restrict__ G, const float* __restrict__ vmx, const float* __restrict__ vmn,
    float* __restrict__ cg, float* __restrict__ splitf, bf16* __restrict__ yh,
    bf16* __restrict__ yl, bf16* __restrict__ wh, bf16* __restrict__ wl,
    float* __restrict__ cst, int* __restrict__ flag, int H, int T, int ntile) {
  __shared__ float c[D], split[D], bl[D], ib[D];
  constexpr int CPR = D / 8;
  static_assert(kThreads % CPR == 0 && CPR <= 64, "a row's threads share a wave");
  const int kb = blockIdx.x % ntile, bh = blockIdx.x / ntile, h = bh % H;
  const int k0 = kb * kTile;
  channel_consts<D>(beta, vmx, vmn, bh, h, ntile, c, split, bl, kb == 0, cg, splitf, flag);
  for (int j = threadIdx.x; j < D; j += kThreads) ib[j] = 1.f / beta[h * D + j];
  __syncthreads();
  const size_t base = (size_t)bh * T * D;
  const size_t rows = ((size_t)bh * ntile + kb) * kTile;  // first row in the padded [., D] arrays
  bool bad = false;
  for (int e = threadIdx.x; e < kTile * CPR; e += kThreads) {
    const int i = e / CPR, c8 = (e % CPR) * 8;
    const bool live = k0 + i < T;
    const size_t at = base + (size_t)(k0 + i) * D + c8;
    bf16x8 vx = {}, hi, lo, whi, wlo;
    f32x4 g4[2] = {}, f4[2] = {};
    if (live) {
      vx = *reinterpret_cast<const bf16x8*>(V + at);
#pragma unroll
      for (int k = 0; k < 2; ++k) {
        g4[k] = *reinterpret_cast<const f32x4*>(G + at + 4 * k);
        f4[k] = *reinterpret_cast<const f32x4*>(F + at + 4 * k);
      }
    }
    float cs = 0.f;
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int j = c8 + u;
      // a wide channel contributes nothing here: Y = 0, W U = 0
      const bool sp = split[j] == kSplitForm, on = live && split[j] != kWide;
      float y = 0.f;
      if (on) {
        const float xv = fmaf(bl[j], (float)vx[u], -c[j]);
        y = sp ? expm1f(xv * kLn2) : exp2_hw(xv);
      }
      bf16 a, b;
      split_bf16(y, a, b);
      hi[u] = a;
      lo[u] = b;
      const float w = on ? g4[u >> 2][u & 3] * ib[j] : 0.f;
      const float x = on ? c[j] - bl[j] * f4[u >> 2][u & 3] : 0.f;  // log2 U
      const float wu = w * exp2_hw(fminf(x, kGuardU));
      if (!(x <= kGuardU && fabsf(wu) < kGuardW)) bad = true;
      cs += sp ? w * expm1f(x * kLn2) : -w;
      split_bf16(wu, a, b);
      whi[u] = a;
      wlo[u] = b;
    }
    const size_t o = (rows + i) * D + c8;
    *reinterpret_cast<bf16x8*>(yh + o) = hi;
    *reinterpret_cast<bf16x8*>(yl + o) = lo;
    *reinterpret_cast<bf16x8*>(wh + o) = whi;
    *reinterpret_cast<bf16x8*>(wl + o) = wlo;
#pragma unroll
    for (int m = 1; m < CPR; m <<= 1) cs += __shfl_xor(cs, m);
    if (e % CPR == 0) cst[rows + i] = cs;
  }
  if (bad) flag[0] = 1;
}

// q kernel, matrix-core form.  Wave (kh = w >> 1, qh = w & 1) owns the
// S^T block (keys kh*32.., queries qh*32..) of each tile pair; its query
// rows' operands (Q and W U hi / lo as MFMA B fragments), row constant and
// log-normaliser stay in registers.
template <int D>
struct QFast {
  bf16 key[3][3][kTile * D];  // [buffer][K, Y hi, Y lo], swizzled [key][d or j]
  float pt[2][kTile];         // row sums of p from the two key halves
};

template <int D>
__global__ __launch_bounds__(kThreads) void bwd_q_fast_kernel(
    const bf16* __restrict__ Q, const bf16* __restrict__ K, const float* __restrict__ lse,
    const bf16* __restrict__ yh, const bf16* __restrict__ yl, const bf16* __restrict__ wh,
    const bf16* __restrict__ wl, const float* __restrict__ cst, float* __restrict__ dQ,
    float* __restrict__ sap, float* __restrict__ lse_p, int T, int ntile) {
  using C = Bw<D>;
  constexpr int NB = C::NCB;
  __shared__ __align__(16) QFast<D> sm;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, n = lane & 31, hl = lane >> 5;
  const int lb = xcd_order(blockIdx.x, gridDim.x);
  const int qb = ntile - 1 - lb % ntile, bh = lb / ntile;
  const int q0 = qb * kTile;
  const size_t base = (size_t)bh * T * D;
  const size_t rows0 = (size_t)bh * ntile * kTile;
  const int kh = wave >> 1, qh = wave & 1;
  auto fetch = [&](int kb) {
    const int k0 = kb * kTile;
    bf16* dst = &sm.key[kb % 3][0][0];
    load_swz<D>(K + base + (size_t)k0 * D, dst, T - 1 - k0);
    load_swz<D>(yh + (rows0 + k0) * D, dst + kTile * D, kTile - 1);
    load_swz<D>(yl + (rows0 + k0) * D, dst + 2 * kTile * D, kTile - 1);
  };
  fetch(0);

  const int t = qh * 32 + n;
  // this wave's query rows as MFMA B fragments: Q (for S^T; rows past T
  // re-read row T - 1, their p is masked) and W U hi / lo (for dP^T, zero
  // past T), loop-invariant
  bf16x8 qf[C::NKS], wf[C::NKS][2];
  {
    const size_t qr = base + (size_t)min(q0 + t, T - 1) * D, wr = (rows0 + q0 + t) * D;
#pragma unroll
    for (int ks = 0; ks < C::NKS; ++ks) {
      qf[ks] = *reinterpret_cast<const bf16x8*>(Q + qr + ks * 16 + hl * 8);
      wf[ks][0] = *reinterpret_cast<const bf16x8*>(wh + wr + ks * 16 + hl * 8);
      wf[ks][1] = *reinterpret_cast<const bf16x8*>(wl + wr + ks * 16 + hl * 8);
    }
  }
  const float ct = cst[rows0 + q0 + t];
  const float l2 = q0 + t < T ? lse[(size_t)bh * T + q0 + t] * kLog2e : 0.f;
#pragma unroll
  for (int ks = 0; ks < C::NKS; ++ks) {
    settle(qf[ks]);
    settle(wf[ks][0]);
    settle(wf[ks][1]);
  }
  settle(ct);
  settle(l2);

  f32x16 dqt[NB], sat[NB];  // (d or j block) x queries qh*32.., partial over this wave's keys
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    dqt[b] = f32x16{};
    sat[b] = f32x16{};
  }
  float psum = 0.f;
  const float scale2 = kLog2e / sqrtf((float)D);
  // Software pipeline over the key tiles, three LDS buffers.  Iteration kb
  // runs the row-major products of tile kb (S^T = K Q^T, dP^T = Y (W U)^T)
  // and the transposed products of tile kb - 1 (dQ^T += K^T dS^T,
  // SA^T += Y^T P^T, with that tile's p and dS) in one basic block of
  // independent MFMA chains, then forms p and dS of tile kb: the scheduler
  // interleaves the chains, so the matrix pipe stays busy while operands
  // arrive and while the vector units form p and dS.
  constexpr int NG = 2 * NB;  // groups (d or j block, k-step) of the transposed products
  bf16x8 ph[2] = {}, pl[2] = {}, dsb[2] = {};  // p hi / lo and dS of the tile before
  auto tr_products = [&](int kb, int g0, int g1) {
    const bf16* kt = &sm.key[kb % 3][0][0];
    const bf16* ty = kt + kTile * D;
    const bf16* tyl = ty + kTile * D;
#pragma unroll
    for (int g = g0; g < g1; ++g) {
      const int b = g >> 1, k2 = g & 1, p0 = kh * 32 + k2 * 16;
      const bf16x8 fk = frag_tr<D>(kt, b * 32, p0);
      const bf16x8 fh = frag_tr<D>(ty, b * 32, p0);
      const bf16x8 fl = frag_tr<D>(tyl, b * 32, p0);
      dqt[b] = mfma(fk, dsb[k2], dqt[b]);
      sat[b] = mfma(fh, ph[k2], sat[b]);
      sat[b] = mfma(fl, ph[k2], sat[b]);
      sat[b] = mfma(fh, pl[k2], sat[b]);
    }
  };
  // one iteration; prev: whether tile kb - 1's transposed products run in
  // it; masked: whether the tile pair needs the causal and length masks (only
  // the diagonal tile, or a query tile that runs past T)
  auto iteration = [&](int kb, auto prev, auto masked) {
    const int k0 = kb * kTile;
    wait_vmem();
    __syncthreads();  // tile kb is in; every wave is done with tile kb - 2
    if (kb < qb) fetch(kb + 1);
    const bf16* kt = &sm.key[kb % 3][0][0];
    const bf16* ty = kt + kTile * D;   // Y hi
    const bf16* tyl = ty + kTile * D;  // Y lo
    f32x16 s = {}, dp = {};
#pragma unroll
    for (int k = 0; k < C::NKS; ++k) s = mfma(frag_rows<D>(kt, kh * 32 + n, 2 * k + hl), qf[k], s);
    if constexpr (decltype(prev)::value) tr_products(kb - 1, 0, NG / 2);
#pragma unroll
    for (int ks = 0; ks < C::NKS; ++ks) {
      const bf16x8 ah = frag_rows<D>(ty, kh * 32 + n, 2 * ks + hl);
      const bf16x8 al = frag_rows<D>(tyl, kh * 32 + n, 2 * ks + hl);
      dp = mfma(ah, wf[ks][0], dp);
      dp = mfma(al, wf[ks][0], dp);
      dp = mfma(ah, wf[ks][1], dp);
    }
    if constexpr (decltype(prev)::value) tr_products(kb - 1, NG / 2, NG);
    const bool tlive = q0 + t < T;
    pack_p_ds(
        [&](int r) {
          const float x = fmaf(s[r], scale2, -l2);
          float pr;
          if constexpr (decltype(masked)::value) {
            const int i = kh * 32 + 8 * (r >> 2) + 4 * hl + (r & 3);
            const bool ok = k0 + i <= q0 + t && tlive && k0 + i < T;
            pr = exp2_hw(ok ? x : -INFINITY);
          } else {
            pr = exp2_hw(x);
          }
          psum += pr;
          return f32x2{pr, ct};
        },
        dp, ph, pl, dsb);
  };
  const std::true_type yes;
  const std::false_type no;
  if (qb == 0) {
    iteration(0, no, yes);
  } else if (q0 + kTile <= T) {
    iteration(0, no, no);
    for (int kb = 1; kb < qb; ++kb) iteration(kb, yes, no);
    iteration(qb, yes, yes);
  } else {  // the query tile runs past T: every tile pair masks its rows
    iteration(0, no, yes);
    for (int kb = 1; kb <= qb; ++kb) iteration(kb, yes, yes);
  }
  tr_products(qb, 0, NG);

  // ---- epilogue.  The key halves (waves kh = 0, 1 of the same qh) meet in
  // LDS as [64 queries][D + 1] totals of dQ^T and SA^T; then every thread
  // takes (query, channel) elements with the channel fastest (coalesced
  // global writes): dQ and SA / P.
  __syncthreads();
  constexpr int SR = D + 1;
  float* dqs = reinterpret_cast<float*>(&sm.key[0][0][0]);  // [64][SR]
  float* sas = dqs + kTile * SR;                             // [64][SR]
  static_assert(2 * kTile * (D + 1) * 4 <= sizeof(sm.key), "epilogue area");
  psum += __shfl_xor(psum, 32);
  if (kh == 1) {
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = b * 32 + 8 * (r >> 2) + 4 * hl + (r & 3);
        dqs[t * SR + row] = dqt[b][r];
        sas[t * SR + row] = sat[b][r];
      }
    if (hl == 0) sm.pt[1][t] = psum;
  } else if (hl == 0) {
    sm.pt[0][t] = psum;
  }
  __syncthreads();
  if (kh == 0) {
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = b * 32 + 8 * (r >> 2) + 4 * hl + (r & 3);
        dqs[t * SR + row] += dqt[b][r];
        sas[t * SR + row] += sat[b][r];
      }
  }
  __syncthreads();
  {
    // p was formed from the forward's lse, whose sum of bf16-rounded terms
    // may differ from the exact one by a few 2^-9: P = sum_i p rescales it
    const int j = tid % D;
    const float rs = 1.f / sqrtf((float)D);
    for (int r = tid / D; r < kTile && q0 + r < T; r += kThreads / D) {
      const float rP = 1.f / (sm.pt[0][r] + sm.pt[1][r]);
      const size_t at = base + (size_t)(q0 + r) * D + j;
      dQ[at] = dqs[r * SR + j] * rs * rP;
      sap[at] = sas[r * SR + j] * rP;
    }
    if (tid < kTile && q0 + tid < T)
      lse_p[(size_t)bh * T + q0 + tid] =
          lse[(size_t)bh * T + q0 + tid] + logf(sm.pt[0][tid] + sm.pt[1][tid]);
  }
}

// For the kv pass, per 64-query tile: ln(Z/P) per (t, j) from the q pass's
// SA / P (split: log1p((U - 1) + U SA / P); plain: log2 U + log2(SA / P),
// in nats), the normalised posterior's U' = U / (Z/P), W U' row-major (hi
// and lo) and the row constants sum_j (split ? W (U' - 1) : -W), zero past T;
// and the tile's partial sums of G (F^ + ln(Z/P) / beta) per channel, the
// G F terms of dbeta.  Thread e handles 8 channels of one row; the D/8
// threads of a row are adjacent lanes and keep their channels throughout.
template <int D>
__global__ __launch_bounds__(kThreads) void bwd_prepq_kernel(
    const float* __restrict__ beta, const float* __restrict__ F, const float* __restrict__ G,
    const float* __restrict__ sap, const float* __restrict__ cg, const float* __restrict__ splitf,
    bf16* __restrict__ wh, bf16* __restrict__ wl, float* __restrict__ cst, float* __restrict__ gf,
    int* __restrict__ flag, int H, int T, int ntile) {
  constexpr int CPR = D / 8, RG = kThreads / CPR;
  static_assert(kThreads % CPR == 0 && CPR <= 64, "a row's threads share a wave");
  __shared__ float c[D], split[D], bl[D], ib[D], part[RG][D];
  const int qb = blockIdx.x % ntile, bh = blockIdx.x / ntile, h = bh % H;
  const int q0 = qb * kTile;
  for (int j = threadIdx.x; j < D; j += kThreads) {
    bl[j] = beta[h * D + j] * kLog2e;
    ib[j] = 1.f / beta[h * D + j];
    split[j] = splitf[bh * D + j];
    c[j] = cg[bh * D + j];
  }
  __syncthreads();
  const size_t base = (size_t)bh * T * D;
  const size_t rows = ((size_t)bh * ntile + qb) * kTile;
  const int c8 = (threadIdx.x % CPR) * 8;
  float gacc[8] = {};
  bool bad = false, under = false;
  for (int e = threadIdx.x; e < kTile * CPR; e += kThreads) {
    const int t = e / CPR;
    const bool live = q0 + t < T;
    const size_t at = base + (size_t)(q0 + t) * D + c8;
    bf16x8 hi, lo;
    f32x4 g4[2] = {}, f4[2] = {}, z4[2] = {};
    if (live) {
#pragma unroll
      for (int k = 0; k < 2; ++k) {
        g4[k] = *reinterpret_cast<const f32x4*>(G + at + 4 * k);
        f4[k] = *reinterpret_cast<const f32x4*>(F + at + 4 * k);
        z4[k] = *reinterpret_cast<const f32x4*>(sap + at + 4 * k);
      }
    }
    float cs = 0.f;
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int j = c8 + u;
      // a wide channel contributes nothing here (W U' = 0, no G F term)
      const bool sp = split[j] == kSplitForm, on = live && split[j] != kWide;
      const float g = on ? g4[u >> 2][u & 3] : 0.f, f = f4[u >> 2][u & 3], sa = z4[u >> 2][u & 3];
      const float rb = ib[j], w = g * rb;
      const float x = on ? c[j] - bl[j] * f : 0.f;  // log2 U
      float lz = 0.f;                               // ln(Z/P): F = F^ + ln(Z/P)/beta
      if (on) {
        if (sp) {
          const float um1 = expm1f(x * kLn2);
          lz = log1pf(um1 + (um1 + 1.f) * sa);
        } else {
          if (!(sa > 0x1p-120f)) under = true;
          lz = (x + log2_hw(sa)) * kLn2;
        }
      }
      gacc[u] += g * (f + lz * rb);
      const float xu = fminf(x, kGuardU) - lz * kLog2e;  // log2 U'
      const float wu = w * exp2_hw(xu);
      if (!(x <= kGuardU && fabsf(wu) < kGuardW)) bad = true;
      cs += sp ? w * expm1f(xu * kLn2) : -w;
      bf16 a, b;
      split_bf16(wu, a, b);
      hi[u] = a;
      lo[u] = b;
    }
    *reinterpret_cast<bf16x8*>(wh + (rows + t) * D + c8) = hi;
    *reinterpret_cast<bf16x8*>(wl + (rows + t) * D + c8) = lo;
#pragma unroll
    for (int m = 1; m < CPR; m <<= 1) cs += __shfl_xor(cs, m);
    if (e % CPR == 0) cst[rows + t] = cs;
  }
  if (bad || under) flag[0] = 1;  // a factor or a plain channel's sum left fp32's range
#pragma unroll
  for (int u = 0; u < 8; ++u) part[threadIdx.x / CPR][c8 + u] = gacc[u];
  __syncthreads();
  for (int j = threadIdx.x; j < D; j += kThreads) {
    float acc = 0.f;
    for (int g = 0; g < RG; ++g) acc += part[g][j];
    gf[((size_t)bh * ntile + qb) * D + j] = acc;
  }
}

// kv kernel, matrix-core form.  Wave (qh = w >> 1, kh = w & 1) owns the
// 32 x 32 block (queries qh*32.., keys kh*32..) of each tile pair; its key
// rows' operands (K and Y hi / lo as MFMA B fragments) stay in registers.
template <int D>
struct KvFast {
  bf16 qry[3][3][kTile * D];  // [buffer][Q, W U' hi, W U' lo], swizzled [query][d or j]
  float cst[3][kTile], lse[3][kTile], c[D], bl[D];
};

template <int D>
__global__ __launch_bounds__(kThreads) void bwd_kv_fast_kernel(
    const bf16* __restrict__ Q, const bf16* __restrict__ K, const bf16* __restrict__ V,
    const float* __restrict__ beta, const float* __restrict__ lse, const float* __restrict__ cg,
    const bf16* __restrict__ yh, const bf16* __restrict__ yl, const bf16* __restrict__ wh,
    const bf16* __restrict__ wl, const float* __restrict__ cst, float* __restrict__ dK,
    float* __restrict__ dV, float* __restrict__ vdv, int H, int T, int ntile) {
  using C = Bw<D>;
  constexpr int NB = C::NCB;  // 32-row blocks of d (and of j)
  __shared__ __align__(16) KvFast<D> sm;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, n = lane & 31, hl = lane >> 5;
  const int lb = xcd_order(blockIdx.x, gridDim.x);
  const int kb = lb % ntile, bh = lb / ntile, h = bh % H;
  const int k0 = kb * kTile;
  const size_t base = (size_t)bh * T * D;
  const size_t rows0 = (size_t)bh * ntile * kTile;
  const int qh = wave >> 1, kh = wave & 1;
  auto fetch = [&](int qb) {
    const int q0 = qb * kTile;
    bf16* dst = &sm.qry[qb % 3][0][0];
    load_swz<D>(Q + base + (size_t)q0 * D, dst, T - 1 - q0);
    load_swz<D>(wh + (rows0 + q0) * D, dst + kTile * D, kTile - 1);
    load_swz<D>(wl + (rows0 + q0) * D, dst + 2 * kTile * D, kTile - 1);
    // row constants and log-normalisers: one dword per lane (rows past T re-read row T - 1)
    if (wave == 0) dma4(cst + rows0 + q0 + lane, &sm.cst[qb % 3][0]);
    if (wave == 1) dma4(lse + (size_t)bh * T + min(q0 + lane, T - 1), &sm.lse[qb % 3][0]);
  };
  fetch(kb);

  for (int j = tid; j < D; j += kThreads) {
    sm.bl[j] = beta[h * D + j] * kLog2e;
    sm.c[j] = cg[bh * D + j];
  }
  const int i = kh * 32 + n;
  // this wave's key rows as MFMA B fragments: K (for S; rows past T re-read
  // row T - 1, their p is masked) and Y hi / lo (for dP, zero past T),
  // loop-invariant
  bf16x8 kf[C::NKS], yf[C::NKS][2];
  {
    const size_t kr = base + (size_t)min(k0 + i, T - 1) * D, yr = (rows0 + k0 + i) * D;
#pragma unroll
    for (int ks = 0; ks < C::NKS; ++ks) {
      kf[ks] = *reinterpret_cast<const bf16x8*>(K + kr + ks * 16 + hl * 8);
      yf[ks][0] = *reinterpret_cast<const bf16x8*>(yh + yr + ks * 16 + hl * 8);
      yf[ks][1] = *reinterpret_cast<const bf16x8*>(yl + yr + ks * 16 + hl * 8);
    }
#pragma unroll
    for (int ks = 0; ks < C::NKS; ++ks) {
      settle(kf[ks]);
      settle(yf[ks][0]);
      settle(yf[ks][1]);
    }
  }

  f32x16 dvt[NB], dkt[NB];  // (j or d block) x keys kh*32.., partial over this wave's queries
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    dvt[b] = f32x16{};
    dkt[b] = f32x16{};
  }
  const float scale2 = kLog2e / sqrtf((float)D);
  const int qlast = (T - 1) / kTile;
  // Software pipeline over the query tiles, three LDS buffers, as in the q
  // pass: iteration qb runs S = Q K^T and dP = (W U') Y^T of tile qb and the
  // transposed products of tile qb - 1 (dV^T += (W U')^T P, dK^T += Q^T dS)
  // in one basic block, then forms p and dS of tile qb.
  constexpr int NG = 2 * NB;
  bf16x8 ph[2] = {}, pl[2] = {}, dsb[2] = {};  // p hi / lo and dS of the tile before
  auto tr_products = [&](int qb, int g0, int g1) {
    const bf16* tq = &sm.qry[qb % 3][0][0];
    const bf16* tw = tq + kTile * D;
    const bf16* twl = tw + kTile * D;
#pragma unroll
    for (int g = g0; g < g1; ++g) {
      const int b = g >> 1, k2 = g & 1, p0 = qh * 32 + k2 * 16;
      const bf16x8 gh = frag_tr<D>(tw, b * 32, p0);
      const bf16x8 gl = frag_tr<D>(twl, b * 32, p0);
      const bf16x8 fq = frag_tr<D>(tq, b * 32, p0);
      dvt[b] = mfma(gh, ph[k2], dvt[b]);
      dvt[b] = mfma(gl, ph[k2], dvt[b]);
      dvt[b] = mfma(gh, pl[k2], dvt[b]);
      dkt[b] = mfma(fq, dsb[k2], dkt[b]);
    }
  };
  // one iteration; prev: whether tile qb - 1's transposed products run in
  // it; masked: whether the tile pair needs the causal and length masks (the
  // diagonal tile, or a tile that runs past T)
  auto iteration = [&](int qb, auto prev, auto masked) {
    const int q0 = qb * kTile;
    wait_vmem();
    __syncthreads();  // tile qb is in; every wave is done with tile qb - 2
    if (qb < qlast) fetch(qb + 1);
    const bf16* tq = &sm.qry[qb % 3][0][0];
    const bf16* tw = tq + kTile * D;   // W U' hi
    const bf16* twl = tw + kTile * D;  // W U' lo
    const float* lq = sm.lse[qb % 3];
    const float* cq = sm.cst[qb % 3];
    f32x16 s = {}, dp = {};
#pragma unroll
    for (int k = 0; k < C::NKS; ++k) s = mfma(frag_rows<D>(tq, qh * 32 + n, 2 * k + hl), kf[k], s);
    if constexpr (decltype(prev)::value) tr_products(qb - 1, 0, NG / 2);
#pragma unroll
    for (int ks = 0; ks < C::NKS; ++ks) {
      const bf16x8 ah = frag_rows<D>(tw, qh * 32 + n, 2 * ks + hl);
      const bf16x8 al = frag_rows<D>(twl, qh * 32 + n, 2 * ks + hl);
      dp = mfma(ah, yf[ks][0], dp);
      dp = mfma(al, yf[ks][0], dp);
      dp = mfma(ah, yf[ks][1], dp);
    }
    if constexpr (decltype(prev)::value) tr_products(qb - 1, NG / 2, NG);
    pack_p_ds(
        [&](int r) {
          const int t = qh * 32 + 8 * (r >> 2) + 4 * hl + (r & 3);
          const float x = fmaf(s[r], scale2, -lq[t] * kLog2e);
          float pr;
          if constexpr (decltype(masked)::value) {
            const bool ok = k0 + i <= q0 + t && q0 + t < T && k0 + i < T;
            pr = exp2_hw(ok ? x : -INFINITY);
          } else {
            pr = exp2_hw(x);
          }
          return f32x2{pr, cq[t]};
        },
        dp, ph, pl, dsb);
  };
  const std::true_type yes;
  const std::false_type no;
  const bool ragged = qlast * kTile + kTile > T;  // the last query tile runs past T
  iteration(kb, no, yes);
  for (int qb = kb + 1; qb < qlast; ++qb) iteration(qb, yes, no);
  if (qlast > kb) {
    if (ragged) iteration(qlast, yes, yes);
    else iteration(qlast, yes, no);
  }
  tr_products(qlast, 0, NG);

  // ---- epilogue.  The query halves (waves qh = 0, 1 of the same kh) meet
  // in LDS as [64 keys][D + 1] totals of dV^T and dK^T; then every thread
  // takes (key, channel) elements with the channel fastest (coalesced global
  // access).  Thread tid keeps channel tid % D throughout.
  __syncthreads();
  constexpr int SR = D + 1;
  float* dvs = reinterpret_cast<float*>(&sm.qry[0][0][0]);  // [64][SR]
  float* dks = dvs + kTile * SR;                             // [64][SR]
  float* vpart = dks + kTile * SR;                           // [kThreads]
  static_assert((2 * kTile * (D + 1) + kThreads) * 4 <= sizeof(sm.qry), "epilogue area");
  if (qh == 1) {
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = b * 32 + 8 * (r >> 2) + 4 * hl + (r & 3);
        dvs[i * SR + row] = dvt[b][r];
        dks[i * SR + row] = dkt[b][r];
      }
  }
  __syncthreads();
  if (qh == 0) {
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = b * 32 + 8 * (r >> 2) + 4 * hl + (r & 3);
        dvs[i * SR + row] += dvt[b][r];
        dks[i * SR + row] += dkt[b][r];
      }
  }
  __syncthreads();
  {
    const int j = tid % D;
    const float cj = sm.c[j], blj = sm.bl[j], bj = beta[h * D + j];
    const float rs = 1.f / sqrtf((float)D);
    float vacc = 0.f;
    for (int r = tid / D; r < kTile && k0 + r < T; r += kThreads / D) {
      const size_t at = base + (size_t)(k0 + r) * D + j;
      const float vv = (float)V[at];
      // dV = beta E sum_t p (W U'), E = 2^{bl v - c}
      const float dvv = exp2_hw(fmaf(blj, vv, -cj)) * bj * dvs[r * SR + j];
      dV[at] = dvv;
      dK[at] = dks[r * SR + j] * rs;
      vacc += dvv * vv;
    }
    vpart[tid] = vacc;
  }
  __syncthreads();
  if (tid < D) {
    float acc = 0.f;
    for (int g = 0; g < kThreads / D; ++g) acc += vpart[g * D + tid];
    vdv[((size_t)bh * ntile + kb) * D + tid] = acc;
  }
}

// dbeta from the per-tile partial sums: the element-wise pass's for the
// channels it took (every channel, or the wide ones of a (b, h)), else
// (sum v dV - sum G F) / beta from the matrix-core pass.  One workgroup per
// (h, 32 channels); its 8 thread rows split the (b, tile) partials and meet
// in LDS.
template <int D>
__global__ __launch_bounds__(256) void dbeta_kernel(const float* __restrict__ exact,
                                                    const float* __restrict__ vdv,
                                                    const float* __restrict__ gf,
                                                    const float* __restrict__ beta,
                                                    const int* __restrict__ flag,
                                                    const float* __restrict__ splitf,
                                                    float* __restrict__ dbeta, int B, int H,
                                                    int ntile) {
  __shared__ double part[8][32];
  const int h = blockIdx.x, j = blockIdx.y * 32 + (threadIdx.x & 31), row = threadIdx.x >> 5;
  const bool all = flag[0] != 0;
  double se = 0.0, sm = 0.0;  // element-wise partials; matrix-core partials (times beta)
  for (int u = row; u < B * ntile; u += 8) {
    const int b = u / ntile, c = u % ntile;
    const size_t at = (((size_t)b * H + h) * ntile + c) * D + j;
    if (all || splitf[((size_t)b * H + h) * D + j] == kWide)
      se += (double)exact[at];
    else
      sm += (double)vdv[at] - (double)gf[at];
  }
  double s = se + sm / (double)beta[h * D + j];
  part[row][threadIdx.x & 31] = s;
  __syncthreads();
  if (row == 0) {
    for (int r = 1; r < 8; ++r) s += part[r][threadIdx.x & 31];
    dbeta[h * D + j] = (float)s;
  }
}

// Workspace layout (fp32 unless noted): flag | lse renormalised by the q
// pass [nbh T] | c, split [nbh D] | V max, V min, vdv, gf, exact partials
// [nbh ntile D] | SA / P [nbh T D] | row constants [nbh Tp] | four bf16
// operand arrays [nbh Tp D], Tp = 64 ntile: Y hi, Y lo, and W U hi, lo (the
// q pass's, then the kv pass's W U').  Offsets in bytes from the base.
struct BwdLayout {
  size_t nl, nc, np, nz, nr, no, fbytes, total;
  BwdLayout(int B, int H, int T, int D) {
    const size_t nbh = (size_t)B * H;
    const size_t ntile = ((size_t)T + kTile - 1) / kTile;
    const size_t tp = ntile * kTile;
    nl = nbh * T;
    nc = nbh * D;
    np = nbh * ntile * D;
    nz = nbh * T * D;
    nr = nbh * tp;
    no = nbh * tp * D;
    const size_t fl = nl + 2 * nc + 5 * np + nz + nr;
    fbytes = (fl * sizeof(float) + 255) & ~(size_t)255;
    total = 256 + fbytes + 4 * no * sizeof(bf16);
  }
};

template <int D>
hipError_t launch_bwd(const void* Q, const void* K, const void* V, const float* beta,
                      const float* out, const float* lse_fwd, const float* dout, float* dQ,
                      float* dK, float* dV, float* dbeta, int B, int H, int T, void* wsv,
                      hipStream_t stream) {
  const int nbh = B * H;
  const int ntile = (T + kTile - 1) / kTile;
  const bf16* q = reinterpret_cast<const bf16*>(Q);
  const bf16* k = reinterpret_cast<const bf16*>(K);
  const bf16* v = reinterpret_cast<const bf16*>(V);
  const BwdLayout lay(B, H, T, D);
  const size_t nl = lay.nl, nc = lay.nc, np = lay.np, nz = lay.nz, no = lay.no;
  const size_t fbytes = lay.fbytes;
  char* ws = static_cast<char*>(wsv);
  int* flag = reinterpret_cast<int*>(ws);
  float* lse = reinterpret_cast<float*>(ws + 256);
  float* cg = lse + nl;
  float* splitf = cg + nc;
  float* vmx = splitf + nc;
  float* vmn = vmx + np;
  float* vdv = vmn + np;
  float* gfp = vdv + np;
  float* exact = gfp + np;
  float* sap = exact + np;
  float* cst = sap + nz;
  bf16* yh = reinterpret_cast<bf16*>(ws + 256 + fbytes);
  bf16* yl = yh + no;
  bf16* wh = yl + no;
  bf16* wl = wh + no;
  hipError_t e = hipSuccess;
  const dim3 grid((unsigned)(nbh * ntile)), blk(kThreads);
  hipLaunchKernelGGL(bwd_vstats_kernel<D>, grid, blk, 0, stream, v, vmx, vmn, flag, T, ntile);
  e = hipGetLastError();
  if (e == hipSuccess) {  // channel constants; Y (key side) and the q pass's W U
    hipLaunchKernelGGL(bwd_prepk_kernel<D>, grid, blk, 0, stream, v, beta, out, dout, vmx, vmn, cg,
                       splitf, yh, yl, wh, wl, cst, flag, H, T, ntile);
    e = hipGetLastError();
  }
  if (e == hipSuccess) {  // the q pass first: its SA / P give ln(Z/P), which the kv pass uses
    hipLaunchKernelGGL(bwd_q_fast_kernel<D>, grid, blk, 0, stream, q, k, lse_fwd, yh, yl, wh, wl,
                       cst, dQ, sap, lse, T, ntile);
    e = hipGetLastError();
  }
  if (e == hipSuccess) {  // ln(Z/P), the kv pass's W U' and row constants, the G F sums
    hipLaunchKernelGGL(bwd_prepq_kernel<D>, grid, blk, 0, stream, beta, out, dout, sap, cg, splitf,
                       wh, wl, cst, gfp, flag, H, T, ntile);
    e = hipGetLastError();
  }
  if (e == hipSuccess) {
    hipLaunchKernelGGL(bwd_kv_fast_kernel<D>, grid, blk, 0, stream, q, k, v, beta, lse, cg, yh, yl,
                       wh, wl, cst, dK, dV, vdv, H, T, ntile);
    e = hipGetLastError();
  }
  // element-wise passes: they return at once unless a wide channel or a
  // failed guard raised a flag; wide channels only add to dQ / dK and write
  // their own dV columns, a failed guard replaces every gradient.  The q
  // pass runs first: it leaves the normalised beta log2e F of the channels
  // it takes in the SA / P buffer (free once the fast kv pass has run),
  // which the kv pass's posterior uses.
  float* fbn = sap;
  if (e == hipSuccess) {
    hipLaunchKernelGGL(bwd_q_kernel<D>, grid, blk, 0, stream, q, k, v, beta, out, lse, dout, dQ,
                       exact, fbn, H, T, ntile, flag, splitf);
    e = hipGetLastError();
  }
  if (e == hipSuccess) {
    hipLaunchKernelGGL(bwd_kv_kernel<D>, grid, blk, 0, stream, q, k, v, beta, fbn, lse, dout, dK, dV,
                       H, T, ntile, flag, splitf);
    e = hipGetLastError();
  }
  if (e == hipSuccess) {
    hipLaunchKernelGGL(dbeta_kernel<D>, dim3((unsigned)H, D / 32), dim3(256), 0, stream, exact, vdv,
                       gfp, beta, flag, splitf, dbeta, B, H, ntile);
    e = hipGetLastError();
  }
  return e;
}

}  // namespace

size_t softmax_bwd_ws_bytes(int B, int H, int T, int d) { return BwdLayout(B, H, T, d).total; }

hipError_t launch_softmax_bwd_bf16(const void* Q, const void* K, const void* V,
                                   const float* beta, const float* out, const float* lse,
                                   const float* dout, float* dQ, float* dK, float* dV,
                                   float* dbeta, int B, int H, int T, int d, void* ws,
                                   hipStream_t stream) {
  switch (d) {
    case 32:
      return launch_bwd<32>(Q, K, V, beta, out, lse, dout, dQ, dK, dV, dbeta, B, H, T, ws, stream);
    case 64:
      return launch_bwd<64>(Q, K, V, beta, out, lse, dout, dQ, dK, dV, dbeta, B, H, T, ws, stream);
    case 128:
      return launch_bwd<128>(Q, K, V, beta, out, lse, dout, dQ, dK, dV, dbeta, B, H, T, ws, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace fem
