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

#include <cstddef>
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
    int ntile, const int* __restrict__ run_if) {
  using C = Bw<D>;
  if (run_if && *run_if == 0) return;  // the matrix-core pass needed no fallback
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
    int ntile, const int* __restrict__ run_if) {
  using C = Bw<D>;
  if (run_if && *run_if == 0) return;
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

// ---- matrix-core path ------------------------------------------------------
//
// With c_j a per-channel constant, q_tj(i) = p_ti E_ij U_tj, E_ij =
// 2^{bl_j v_ij - c_j}, U_tj = 2^{c_j - bl_j F^_tj} (bl = beta log2 e), so
//   dS_ti = p_ti sum_j W_tj (R_tij - 1),   R = E U,   W = G / beta,
//   dV_ij = E_ij sum_t p_ti G_tj U_tj
// are products over j and over t.  Two forms per channel:
//   split (bl_j times the range of v_.j over the sequence <= 4): c_j = bl_j max
//     v_.j of the (b, h), R - 1 = A U + (U - 1) with A = E - 1 (expm1): the
//     product sum_j (W U) A and the row constant sum_j W (U - 1) carry no
//     cancellation when beta is small (|A|, |U - 1| are small, U in
//     [2^-4, 2^4]);
//   plain (otherwise): c_j = the key tile's max of bl v, R - 1 = E U - 1, row
//     constant -sum_j W.
// Both factors enter as bf16 hi + lo parts (three MFMAs, ~2^-16 relative).
// p comes from an fp32 log-normaliser recomputed here (the forward's lse sums
// bf16-rounded probabilities), so the rows of p sum to one to fp32 accuracy.
// A block whose U would exceed 2^100 (a row's F far below the key tile's
// largest beta v) sets a device flag; the exact kernels then redo the whole
// pass, and otherwise return at once.  Below that bound every product stays
// inside fp32's range (W U <= 2^100 |G| / beta), and an E that flushes to
// zero (< 2^-126) drops a posterior ratio R = E U < 2^-26.
//
// Normalisation: R^ built from the forward's F^ gives sum_i p R^ = Z/P =
// e^{beta (F - F^)} != 1 (the forward rounds p to bf16).  The q kernel, which
// sees every key of its rows, forms ln(Z/P) per (t, j) exactly -- from the
// split form (D = (U - 1) P + U sum_i p A) for split channels, from a running
// per-channel log-sum of the tiles' sum_i p E for plain ones -- and writes
// it; the kv kernel then uses the normalised posterior R^ / (Z/P).  So
// dbeta = sum_t G (E_q[v] - F) / beta = (sum_i v dV - sum_t G F) / beta with
// F = F^ + ln(Z/P)/beta is formed from normalised quantities; its terms are
// small next to their parts (~ beta Var/2 at small beta, ~ KL/beta at large).

__host__ __device__ constexpr int epos32(int r) {
  return (r & 16) + (((r >> 2) & 1) << 3) + (((r >> 3) & 1) << 2) + (r & 3);
}
// Storage position of contraction index x (0..63) in a row whose 32-blocks
// feed MFMA A operands against B operands taken from an accumulator's rows.
__host__ __device__ constexpr int ppos(int x) { return (x & 32) + epos32(x & 31); }

__device__ __forceinline__ void split_bf16(float x, bf16& hi, bf16& lo) {
  hi = (bf16)x;
  lo = (bf16)(x - (float)hi);
}

__device__ __forceinline__ f32x16 mfma(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// The prior's log-normaliser in fp32 from unrounded probabilities:
// lse_t = ln sum_{i<=t} exp(q_t.k_i / sqrt d).  One workgroup per (b, h,
// 64-query tile); wave (kh, qh) takes the S^T block of keys kh*32.. and
// queries qh*32..; lane (query n, half hl) keeps a running (max, sum).
template <int D>
__global__ __launch_bounds__(kThreads) void bwd_lse_kernel(const bf16* __restrict__ Q,
                                                           const bf16* __restrict__ K,
                                                           float* __restrict__ lse, int T,
                                                           int ntile) {
  using C = Bw<D>;
  __shared__ __align__(16) bf16 qt[kTile * C::ROW];
  __shared__ __align__(16) bf16 kt[kTile * C::ROW];
  __shared__ float rm[4][64], rs[4][64];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, n = lane & 31, hl = lane >> 5;
  const int qb = blockIdx.x % ntile, bh = blockIdx.x / ntile;
  const int q0 = qb * kTile;
  const size_t base = (size_t)bh * T * D;
  const int kh = wave >> 1, qh = wave & 1;
  const int t = qh * 32 + n;
  stage_tile<D>(Q + base, q0, T, qt, nullptr);
  const float scale2 = kLog2e / sqrtf((float)D);
  float m = -INFINITY, sum = 0.f;
  for (int kb = 0; kb <= qb; ++kb) {
    const int k0 = kb * kTile;
    __syncthreads();
    stage_tile<D>(K + base, k0, T, kt, nullptr);
    __syncthreads();
    const f32x16 acc = score_block<D>(kt, qt, kh, qh);  // M = keys, N = queries
    float x[16], bm = -INFINITY;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int i = kh * 32 + 8 * (r >> 2) + 4 * hl + (r & 3);
      const bool ok = k0 + i <= q0 + t && k0 + i < T;
      x[r] = ok ? acc[r] * scale2 : -INFINITY;
      bm = fmaxf(bm, x[r]);
    }
    const float mn = fmaxf(m, bm);
    if (mn != -INFINITY) {
      float a = sum * exp2_hw(m - mn);
#pragma unroll
      for (int r = 0; r < 16; ++r) a += exp2_hw(x[r] - mn);
      sum = a;
      m = mn;
    }
  }
  rm[wave][lane] = m;
  rs[wave][lane] = sum;
  __syncthreads();
  if (tid < kTile) {
    const int qq = tid >> 5, nn = tid & 31;  // query qq*32 + nn: waves (0, qq), (1, qq), both halves
    float M = -INFINITY, S = 0.f;
    for (int k2 = 0; k2 < 2; ++k2)
      for (int h2 = 0; h2 < 2; ++h2) {
        const float mm = rm[k2 * 2 + qq][h2 * 32 + nn], ss = rs[k2 * 2 + qq][h2 * 32 + nn];
        const float mx = fmaxf(M, mm);
        if (mx != -INFINITY) {
          S = S * exp2_hw(M - mx) + ss * exp2_hw(mm - mx);
          M = mx;
        }
      }
    if (q0 + tid < T) lse[(size_t)bh * T + q0 + tid] = (M + log2_hw(S)) * kLn2;
  }
}

// Per (b, h, j): whether channel j takes the split form, and its sequence-wide
// shift c_j = bl_j max v.  Also clears the fallback flag.
template <int D>
__global__ __launch_bounds__(kThreads) void bwd_prep_kernel(const bf16* __restrict__ V,
                                                            const float* __restrict__ beta,
                                                            float* __restrict__ cg,
                                                            float* __restrict__ splitf,
                                                            int* __restrict__ flag, int H,
                                                            int T) {
  constexpr int RG = kThreads / D;
  __shared__ float mx[kThreads], mn[kThreads];
  const int bh = blockIdx.x, h = bh % H, tid = threadIdx.x, j = tid % D, rg = tid / D;
  if (bh == 0 && tid == 0) flag[0] = 0;
  const bf16* Vh = V + (size_t)bh * T * D;
  float a = -INFINITY, b = INFINITY;
  for (int t = rg; t < T; t += RG) {
    const float v = (float)Vh[(size_t)t * D + j];
    a = fmaxf(a, v);
    b = fminf(b, v);
  }
  mx[tid] = a;
  mn[tid] = b;
  __syncthreads();
  if (rg == 0) {
    for (int g = 1; g < RG; ++g) {
      a = fmaxf(a, mx[g * D + j]);
      b = fminf(b, mn[g * D + j]);
    }
    const float bl = beta[h * D + j] * kLog2e;
    cg[bh * D + j] = bl * a;
    splitf[bh * D + j] = bl * (a - b) <= 4.f ? 1.f : 0.f;
  }
}

constexpr float kGuard = 100.f;  // largest log2 U of the plain form

// kv kernel, matrix-core form.  Wave (qh = w >> 1, kh = w & 1) owns the
// 32 x 32 block (queries qh*32.., keys kh*32..) of each tile pair.
template <int D>
struct KvFast {
  using C = Bw<D>;
  bf16 kt[kTile * C::ROW];                  // K [key][d]
  bf16 qt[kTile * C::ROW];                  // Q [query][d]
  bf16 qTp[D * C::TROW];                    // Q^T [d][query, permuted]
  bf16 yh[kTile * C::ROW], yl[kTile * C::ROW];    // Y [key][j]
  bf16 wuh[kTile * C::ROW], wul[kTile * C::ROW];  // W U [query][j]
  bf16 guh[D * C::TROW], gul[D * C::TROW];        // (G U)^T [j][query, permuted]
  float cst[kTile], lse2[kTile], c[D], split[D], bl[D];
};

template <int D>
__global__ __launch_bounds__(kThreads) void bwd_kv_fast_kernel(
    const bf16* __restrict__ Q, const bf16* __restrict__ K, const bf16* __restrict__ V,
    const float* __restrict__ beta, const float* __restrict__ F, const float* __restrict__ lse,
    const float* __restrict__ G, const float* __restrict__ cg, const float* __restrict__ splitf,
    const float* __restrict__ lnz, float* __restrict__ dK, float* __restrict__ dV,
    float* __restrict__ vdv,
    int* __restrict__ flag, int H, int T, int ntile) {
  using C = Bw<D>;
  constexpr int NB = C::NCB;  // 32-row blocks of d (and of j)
  __shared__ __align__(16) KvFast<D> sm;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, n = lane & 31, hl = lane >> 5;
  const int kb = blockIdx.x % ntile, bh = blockIdx.x / ntile, h = bh % H;
  const int k0 = kb * kTile;
  const size_t base = (size_t)bh * T * D;
  const int qh = wave >> 1, kh = wave & 1;

  // ---- the key tile: shifts c_j and Y = A (split) or E (plain)
  float* scratch = reinterpret_cast<float*>(sm.guh);  // [64][D] fp32 bl v (fits in guh + gul)
  for (int j = tid; j < D; j += kThreads) {
    sm.bl[j] = beta[h * D + j] * kLog2e;
    sm.split[j] = splitf[bh * D + j];
  }
  stage_tile<D>(K + base, k0, T, sm.kt, nullptr);
  __syncthreads();
  for (int e = tid; e < kTile * D; e += kThreads) {
    const int i = e / D, j = e % D;
    scratch[e] = k0 + i < T ? sm.bl[j] * (float)V[base + (size_t)(k0 + i) * D + j] : -INFINITY;
  }
  __syncthreads();
  for (int j = tid; j < D; j += kThreads) {
    float mxv = -INFINITY;
    for (int i = 0; i < kTile; ++i) mxv = fmaxf(mxv, scratch[i * D + j]);
    sm.c[j] = sm.split[j] != 0.f ? cg[bh * D + j] : mxv;
  }
  __syncthreads();
  for (int e = tid; e < kTile * D; e += kThreads) {
    const int i = e / D, j = e % D;
    const float x = scratch[e] - sm.c[j];
    float y = 0.f;
    if (k0 + i < T) y = sm.split[j] != 0.f ? expm1f(x * kLn2) : exp2_hw(x);
    split_bf16(y, sm.yh[i * C::ROW + j], sm.yl[i * C::ROW + j]);
  }

  f32x16 dvt[NB], dkt[NB];  // (j or d block) x keys kh*32.., partial over this wave's queries
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    dvt[b] = f32x16{};
    dkt[b] = f32x16{};
  }
  const float scale2 = kLog2e / sqrtf((float)D);
  const int qlast = (T - 1) / kTile;
  bool bad = false;
  for (int qb = kb; qb <= qlast; ++qb) {
    const int q0 = qb * kTile;
    __syncthreads();
    // Q tile, row-major and transposed in permuted query order
    {
      constexpr int CPR = D / 8;
      for (int e = tid; e < kTile * CPR; e += kThreads) {
        const int r = e / CPR, c8 = (e % CPR) * 8;
        bf16x8 x = {};
        if (q0 + r < T) x = *reinterpret_cast<const bf16x8*>(Q + base + (size_t)(q0 + r) * D + c8);
        *reinterpret_cast<bf16x8*>(sm.qt + r * C::ROW + c8) = x;
#pragma unroll
        for (int u = 0; u < 8; ++u) sm.qTp[(c8 + u) * C::TROW + ppos(r)] = x[u];
      }
    }
    // W U', (G U')^T and the row constants, U' = U / (Z/P) normalising the
    // posterior; thread (row tid >> 2, quarter tid & 3)
    {
      const int t = tid >> 2, j0 = (tid & 3) * (D / 4);
      const bool live = q0 + t < T;
      float cs = 0.f;
      for (int u = 0; u < D / 4; ++u) {
        const int j = j0 + u;
        float w = 0.f, g = 0.f, x = 0.f, lz = 0.f;
        if (live) {
          const size_t at = base + (size_t)(q0 + t) * D + j;
          g = G[at];
          x = sm.c[j] - sm.bl[j] * F[at];
          lz = lnz[at] * kLog2e;
          w = g / beta[h * D + j];
          if (x > kGuard) bad = true;
        }
        const float xu = fminf(x, kGuard) - lz;  // log2 U'
        const float U = exp2_hw(xu);
        cs += sm.split[j] != 0.f ? w * expm1f(xu * kLn2) : -w;
        split_bf16(w * U, sm.wuh[t * C::ROW + j], sm.wul[t * C::ROW + j]);
        split_bf16(g * U, sm.guh[j * C::TROW + ppos(t)], sm.gul[j * C::TROW + ppos(t)]);
      }
      cs += __shfl_xor(cs, 1);
      cs += __shfl_xor(cs, 2);
      if ((tid & 3) == 0) sm.cst[t] = cs;
      if (tid < kTile) sm.lse2[tid] = q0 + tid < T ? lse[(size_t)bh * T + q0 + tid] * kLog2e : 0.f;
    }
    __syncthreads();

    // S (queries x keys), p in fp32
    const f32x16 s = score_block<D>(sm.qt, sm.kt, qh, kh);
    const int i = kh * 32 + n;
    float p[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int t = qh * 32 + 8 * (r >> 2) + 4 * hl + (r & 3);
      const bool ok = k0 + i <= q0 + t && q0 + t < T && k0 + i < T;
      p[r] = ok ? exp2_hw(fmaf(s[r], scale2, -sm.lse2[t])) : 0.f;
    }
    // dP = (W U) Y^T over j
    f32x16 dp = {};
#pragma unroll
    for (int ks = 0; ks < C::NKS; ++ks) {
      const int ao = (qh * 32 + n) * C::ROW + ks * 16 + hl * 8, bo = (kh * 32 + n) * C::ROW + ks * 16 + hl * 8;
      const bf16x8 ah = *reinterpret_cast<const bf16x8*>(sm.wuh + ao);
      const bf16x8 al = *reinterpret_cast<const bf16x8*>(sm.wul + ao);
      const bf16x8 bh8 = *reinterpret_cast<const bf16x8*>(sm.yh + bo);
      const bf16x8 bl8 = *reinterpret_cast<const bf16x8*>(sm.yl + bo);
      dp = mfma(ah, bh8, dp);
      dp = mfma(al, bh8, dp);
      dp = mfma(ah, bl8, dp);
    }
    // dS = p (dP + const); p and dS as B operands (k = this wave's queries, accumulator order)
    bf16x8 ph[2], pl[2], dsb[2];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int t = qh * 32 + 8 * (r >> 2) + 4 * hl + (r & 3);
      const float ds = p[r] * (dp[r] + sm.cst[t]);
      bf16 a, b;
      split_bf16(p[r], a, b);
      ph[r >> 3][r & 7] = a;
      pl[r >> 3][r & 7] = b;
      dsb[r >> 3][r & 7] = (bf16)ds;
    }
    // dV^T(j block, keys) += (G U)^T P ;  dK^T(d block, keys) += Q^T dS
#pragma unroll
    for (int b = 0; b < NB; ++b) {
#pragma unroll
      for (int k2 = 0; k2 < 2; ++k2) {
        const int ao = (b * 32 + n) * C::TROW + qh * 32 + k2 * 16 + hl * 8;
        const bf16x8 gh = *reinterpret_cast<const bf16x8*>(sm.guh + ao);
        const bf16x8 gl = *reinterpret_cast<const bf16x8*>(sm.gul + ao);
        dvt[b] = mfma(gh, ph[k2], dvt[b]);
        dvt[b] = mfma(gl, ph[k2], dvt[b]);
        dvt[b] = mfma(gh, pl[k2], dvt[b]);
        const bf16x8 qa = *reinterpret_cast<const bf16x8*>(sm.qTp + ao);
        dkt[b] = mfma(qa, dsb[k2], dkt[b]);
      }
    }
  }
  if (bad) flag[0] = 1;

  // ---- combine the two query halves (waves qh = 0, 1 of the same kh)
  __syncthreads();
  // [2 kh][2 sets][NB][16][64] fp32 (64 KiB at d = 128) over kt, qt, qTp, yh;
  // the v dV products go to wuh onwards
  float* red = reinterpret_cast<float*>(sm.kt);
  static_assert(4 * C::NCB * 16 * 64 * 4 <= offsetof(KvFast<D>, wuh), "reduction area");
  static_assert(offsetof(KvFast<D>, wuh) + kTile * D * 4 <= offsetof(KvFast<D>, cst), "v dV area");
  auto slot = [&](int set, int b, int r) { return (((kh * 2 + set) * NB + b) * 16 + r) * 64 + lane; };
  if (qh == 1) {
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        red[slot(0, b, r)] = dvt[b][r];
        red[slot(1, b, r)] = dkt[b][r];
      }
  }
  __syncthreads();
  float* vdvs = reinterpret_cast<float*>(sm.wuh);  // [64 keys][D] v dV products
  if (qh == 0) {
    const float rs = 1.f / sqrtf((float)D);
    const int key = k0 + kh * 32 + n;
#pragma unroll
    for (int b = 0; b < NB; ++b) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = b * 32 + 8 * (r >> 2) + 4 * hl + (r & 3);  // j or d
        const float sv = dvt[b][r] + red[slot(0, b, r)];
        const float sk = dkt[b][r] + red[slot(1, b, r)];
        float dvv = 0.f;
        if (key < T) {
          const float vv = (float)V[base + (size_t)key * D + row];
          const float E = exp2_hw(fmaf(sm.bl[row], vv, -sm.c[row]));
          dvv = E * sv;
          dV[base + (size_t)key * D + row] = dvv;
          dK[base + (size_t)key * D + row] = sk * rs;
          dvv *= vv;
        }
        vdvs[(kh * 32 + n) * D + row] = dvv;
      }
    }
  }
  __syncthreads();
  for (int j = tid; j < D; j += kThreads) {
    float acc = 0.f;
    for (int i = 0; i < kTile; ++i) acc += vdvs[i * D + j];
    vdv[((size_t)bh * ntile + kb) * D + j] = acc;
  }
}

// q kernel, matrix-core form.  Wave (kh = w >> 1, qh = w & 1) owns the
// S^T block (keys kh*32.., queries qh*32..) of each tile pair.
template <int D>
struct QFast {
  using C = Bw<D>;
  bf16 qt[kTile * C::ROW];                        // Q [query][d]
  bf16 kt[kTile * C::ROW];                        // K [key][d]
  bf16 kTp[D * C::TROW];                          // K^T [d][key, permuted]
  bf16 yh[kTile * C::ROW], yl[kTile * C::ROW];    // Y [key][j]
  bf16 wuh[kTile * C::ROW], wul[kTile * C::ROW];  // W U [query][j]
  bf16 yTh[D * C::TROW], yTl[D * C::TROW];        // Y^T [j][key, permuted]
  float cst[kTile], lse2[kTile], c[D], split[D], bl[D], pt[2][kTile];
  float cref[D], resc[D];  // running reference shift of the plain channels' sums, rescale
};

template <int D>
__global__ __launch_bounds__(kThreads) void bwd_q_fast_kernel(
    const bf16* __restrict__ Q, const bf16* __restrict__ K, const bf16* __restrict__ V,
    const float* __restrict__ beta, const float* __restrict__ F, const float* __restrict__ lse,
    const float* __restrict__ G, const float* __restrict__ cg, const float* __restrict__ splitf,
    float* __restrict__ dQ, float* __restrict__ gf, float* __restrict__ lnz,
    int* __restrict__ flag, int H, int T, int ntile) {
  using C = Bw<D>;
  constexpr int NB = C::NCB;
  __shared__ __align__(16) QFast<D> sm;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, n = lane & 31, hl = lane >> 5;
  const int qb = ntile - 1 - blockIdx.x % ntile, bh = blockIdx.x / ntile, h = bh % H;
  const int q0 = qb * kTile;
  const size_t base = (size_t)bh * T * D;
  const int kh = wave >> 1, qh = wave & 1;

  for (int j = tid; j < D; j += kThreads) {
    sm.bl[j] = beta[h * D + j] * kLog2e;
    sm.split[j] = splitf[bh * D + j];
    sm.cref[j] = sm.split[j] != 0.f ? cg[bh * D + j] : -INFINITY;
  }
  if (tid < kTile) sm.lse2[tid] = q0 + tid < T ? lse[(size_t)bh * T + q0 + tid] * kLog2e : 0.f;
  stage_tile<D>(Q + base, q0, T, sm.qt, nullptr);
  __syncthreads();
  // row constants: sum_j (split ? W (U - 1) : -W), with U from the sequence-wide shift
  {
    const int t = tid >> 2, j0 = (tid & 3) * (D / 4);
    float cs = 0.f;
    if (q0 + t < T) {
      for (int u = 0; u < D / 4; ++u) {
        const int j = j0 + u;
        const float w = G[base + (size_t)(q0 + t) * D + j] / beta[h * D + j];
        if (sm.split[j] != 0.f) {
          const float x = cg[bh * D + j] - sm.bl[j] * F[base + (size_t)(q0 + t) * D + j];
          cs += w * expm1f(x * kLn2);
        } else {
          cs -= w;
        }
      }
    }
    cs += __shfl_xor(cs, 1);
    cs += __shfl_xor(cs, 2);
    if ((tid & 3) == 0) sm.cst[t] = cs;
  }

  f32x16 dqt[NB], sat[NB];  // (d or j block) x queries qh*32.., partial over this wave's keys
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    dqt[b] = f32x16{};
    sat[b] = f32x16{};
  }
  float psum = 0.f;
  const float scale2 = kLog2e / sqrtf((float)D);
  bool bad = false;
  float* scratch = reinterpret_cast<float*>(sm.yTh);  // [64][D] fp32 bl v (fits in yTh + yTl)
  for (int kb = 0; kb <= qb; ++kb) {
    const int k0 = kb * kTile;
    __syncthreads();
    {
      constexpr int CPR = D / 8;
      for (int e = tid; e < kTile * CPR; e += kThreads) {
        const int r = e / CPR, c8 = (e % CPR) * 8;
        bf16x8 x = {};
        if (k0 + r < T) x = *reinterpret_cast<const bf16x8*>(K + base + (size_t)(k0 + r) * D + c8);
        *reinterpret_cast<bf16x8*>(sm.kt + r * C::ROW + c8) = x;
#pragma unroll
        for (int u = 0; u < 8; ++u) sm.kTp[(c8 + u) * C::TROW + ppos(r)] = x[u];
      }
    }
    for (int e = tid; e < kTile * D; e += kThreads) {
      const int i = e / D, j = e % D;
      scratch[e] = k0 + i < T ? sm.bl[j] * (float)V[base + (size_t)(k0 + i) * D + j] : -INFINITY;
    }
    __syncthreads();
    for (int j = tid; j < D; j += kThreads) {
      float mxv = -INFINITY;
      for (int i = 0; i < kTile; ++i) mxv = fmaxf(mxv, scratch[i * D + j]);
      const bool sp = sm.split[j] != 0.f;
      sm.c[j] = sp ? cg[bh * D + j] : mxv;
      // plain channels: the running reference of their sums rises with the tiles
      const float cold = sm.cref[j], cnew = sp ? cold : fmaxf(cold, mxv);
      sm.resc[j] = cnew == cold ? 1.f : exp2_hw(cold - cnew);
      sm.cref[j] = cnew;
    }
    __syncthreads();
    // the plain channels' sums move to the new reference
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) sat[b][r] *= sm.resc[b * 32 + 8 * (r >> 2) + 4 * hl + (r & 3)];
    // Y (row-major) into yh / yl for dP; for the sums (transposed copy, written
    // once scratch is read) the plain channels take E 2^{c - cref} <= 1
    float yv[kTile * D / kThreads];
    for (int e = tid, u = 0; e < kTile * D; e += kThreads, ++u) {
      const int i = e / D, j = e % D;
      const float x = scratch[e] - sm.c[j];
      float y = 0.f, ys = 0.f;
      if (k0 + i < T) {
        if (sm.split[j] != 0.f) {
          y = ys = expm1f(x * kLn2);
        } else {
          y = exp2_hw(x);
          ys = exp2_hw(scratch[e] - sm.cref[j]);
        }
      }
      yv[u] = ys;
      split_bf16(y, sm.yh[i * C::ROW + j], sm.yl[i * C::ROW + j]);
    }
    // W U for this key tile's shifts
    {
      const int t = tid >> 2, j0 = (tid & 3) * (D / 4);
      const bool live = q0 + t < T;
      for (int u = 0; u < D / 4; ++u) {
        const int j = j0 + u;
        float w = 0.f, x = 0.f;
        if (live) {
          w = G[base + (size_t)(q0 + t) * D + j] / beta[h * D + j];
          x = sm.c[j] - sm.bl[j] * F[base + (size_t)(q0 + t) * D + j];
          if (x > kGuard) bad = true;
        }
        split_bf16(w * exp2_hw(fminf(x, kGuard)), sm.wuh[t * C::ROW + j], sm.wul[t * C::ROW + j]);
      }
    }
    __syncthreads();  // scratch fully read
    for (int e = tid, u = 0; e < kTile * D; e += kThreads, ++u) {
      const int i = e / D, j = e % D;
      split_bf16(yv[u], sm.yTh[j * C::TROW + ppos(i)], sm.yTl[j * C::TROW + ppos(i)]);
    }
    __syncthreads();

    // S^T (keys x queries), p in fp32
    const f32x16 s = score_block<D>(sm.kt, sm.qt, kh, qh);
    const int t = qh * 32 + n;
    float p[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int i = kh * 32 + 8 * (r >> 2) + 4 * hl + (r & 3);
      const bool ok = k0 + i <= q0 + t && q0 + t < T && k0 + i < T;
      p[r] = ok ? exp2_hw(fmaf(s[r], scale2, -sm.lse2[t])) : 0.f;
      psum += p[r];
    }
    // dP^T = Y (W U)^T over j
    f32x16 dp = {};
#pragma unroll
    for (int ks = 0; ks < C::NKS; ++ks) {
      const int ao = (kh * 32 + n) * C::ROW + ks * 16 + hl * 8, bo = (qh * 32 + n) * C::ROW + ks * 16 + hl * 8;
      const bf16x8 ah = *reinterpret_cast<const bf16x8*>(sm.yh + ao);
      const bf16x8 al = *reinterpret_cast<const bf16x8*>(sm.yl + ao);
      const bf16x8 bh8 = *reinterpret_cast<const bf16x8*>(sm.wuh + bo);
      const bf16x8 bl8 = *reinterpret_cast<const bf16x8*>(sm.wul + bo);
      dp = mfma(ah, bh8, dp);
      dp = mfma(al, bh8, dp);
      dp = mfma(ah, bl8, dp);
    }
    bf16x8 ph[2], pl[2], dsb[2];
    const float ct = sm.cst[t];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      bf16 a, b;
      split_bf16(p[r], a, b);
      ph[r >> 3][r & 7] = a;
      pl[r >> 3][r & 7] = b;
      dsb[r >> 3][r & 7] = (bf16)(p[r] * (dp[r] + ct));
    }
    // dQ^T(d block, queries) += K^T dS^T ;  SA^T(j block, queries) += Y^T P^T
#pragma unroll
    for (int b = 0; b < NB; ++b) {
#pragma unroll
      for (int k2 = 0; k2 < 2; ++k2) {
        const int ao = (b * 32 + n) * C::TROW + kh * 32 + k2 * 16 + hl * 8;
        const bf16x8 ka = *reinterpret_cast<const bf16x8*>(sm.kTp + ao);
        dqt[b] = mfma(ka, dsb[k2], dqt[b]);
        const bf16x8 yh8 = *reinterpret_cast<const bf16x8*>(sm.yTh + ao);
        const bf16x8 yl8 = *reinterpret_cast<const bf16x8*>(sm.yTl + ao);
        sat[b] = mfma(yh8, ph[k2], sat[b]);
        sat[b] = mfma(yl8, ph[k2], sat[b]);
        sat[b] = mfma(yh8, pl[k2], sat[b]);
      }
    }
  }
  if (bad) flag[0] = 1;

  // ---- combine the key halves (waves kh = 0, 1 of the same qh) and both lane halves of P
  __syncthreads();
  // [2 qh][2 sets][NB][16][64] fp32 over qt, kt, kTp, yh; the G F terms go to wuh onwards
  float* red = reinterpret_cast<float*>(sm.qt);
  static_assert(4 * C::NCB * 16 * 64 * 4 <= offsetof(QFast<D>, wuh), "reduction area");
  static_assert(offsetof(QFast<D>, wuh) + kTile * D * 4 <= offsetof(QFast<D>, cst), "G F area");
  auto slot = [&](int set, int b, int r) { return (((qh * 2 + set) * NB + b) * 16 + r) * 64 + lane; };
  psum += __shfl_xor(psum, 32);
  if (kh == 1) {
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        red[slot(0, b, r)] = dqt[b][r];
        red[slot(1, b, r)] = sat[b][r];
      }
    if (hl == 0) sm.pt[1][qh * 32 + n] = psum;
  } else if (hl == 0) {
    sm.pt[0][qh * 32 + n] = psum;
  }
  __syncthreads();
  float* gfs = reinterpret_cast<float*>(sm.wuh);  // [64 queries][D] G F terms
  if (kh == 0) {
    const float rs = 1.f / sqrtf((float)D);
    const int tq = q0 + qh * 32 + n;
    const float P = sm.pt[0][qh * 32 + n] + sm.pt[1][qh * 32 + n];
#pragma unroll
    for (int b = 0; b < NB; ++b) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = b * 32 + 8 * (r >> 2) + 4 * hl + (r & 3);  // d or j
        const float sq = dqt[b][r] + red[slot(0, b, r)];
        const float sa = sat[b][r] + red[slot(1, b, r)];
        float term = 0.f;
        if (tq < T) {
          dQ[base + (size_t)tq * D + row] = sq * rs;
          const float g = G[base + (size_t)tq * D + row], f = F[base + (size_t)tq * D + row];
          float lz;  // ln(Z/P): F = F^ + ln(Z/P)/beta
          if (sm.split[row] != 0.f) {
            // Z/P - 1 = (U - 1) + U SA / P, U = 2^{c - bl F^}
            const float um1 = expm1f((cg[bh * D + row] - sm.bl[row] * f) * kLn2);
            lz = log1pf(um1 + (um1 + 1.f) * sa / P);
          } else {
            // Z = 2^{cref - bl F^} sum_tiles 2^{c_k - cref} sum_i p E_k
            if (!(sa > 0x1p-100f * P)) flag[0] = 1;  // sums underflowed: exact pass
            lz = (sm.cref[row] - sm.bl[row] * f) * kLn2 + logf(sa / P);
          }
          lnz[base + (size_t)tq * D + row] = lz;
          term = g * (f + lz / beta[h * D + row]);
        }
        gfs[(qh * 32 + n) * D + row] = term;
      }
    }
  }
  __syncthreads();
  for (int j = tid; j < D; j += kThreads) {
    float acc = 0.f;
    for (int i = 0; i < kTile; ++i) acc += gfs[i * D + j];
    gf[((size_t)bh * ntile + qb) * D + j] = acc;
  }
}

// dbeta from the per-tile partial sums: the exact pass's when it ran, else
// (sum v dV - sum G F) / beta from the matrix-core pass.
template <int D>
__global__ void dbeta_kernel(const float* __restrict__ exact, const float* __restrict__ vdv,
                             const float* __restrict__ gf, const float* __restrict__ beta,
                             const int* __restrict__ flag, float* __restrict__ dbeta, int B, int H,
                             int ntile) {
  const int h = blockIdx.x;
  const bool ex = flag[0] != 0;
  for (int j = threadIdx.x; j < D; j += blockDim.x) {
    double s = 0.0;
    for (int b = 0; b < B; ++b)
      for (int c = 0; c < ntile; ++c) {
        const size_t at = (((size_t)b * H + h) * ntile + c) * D + j;
        s += ex ? (double)exact[at] : (double)vdv[at] - (double)gf[at];
      }
    dbeta[h * D + j] = (float)(ex ? s : s / (double)beta[h * D + j]);
  }
}

template <int D>
hipError_t launch_bwd(const void* Q, const void* K, const void* V, const float* beta,
                      const float* out, const float* lse_fwd, const float* dout, float* dQ,
                      float* dK, float* dV, float* dbeta, int B, int H, int T, hipStream_t stream) {
  (void)lse_fwd;  // the passes use the fp32 log-normaliser recomputed below
  const int nbh = B * H;
  const int ntile = (T + kTile - 1) / kTile;
  const bf16* q = reinterpret_cast<const bf16*>(Q);
  const bf16* k = reinterpret_cast<const bf16*>(K);
  const bf16* v = reinterpret_cast<const bf16*>(V);
  // workspace: flag | lse [nbh T] | c, split [nbh D] | vdv, gf, exact partials
  // [nbh ntile D] | ln(Z/P) [nbh T D]
  const size_t nl = (size_t)nbh * T, nc = (size_t)nbh * D, np = (size_t)nbh * ntile * D;
  const size_t nz = (size_t)nbh * T * D;
  const size_t bytes = 256 + (nl + 2 * nc + 3 * np + nz) * sizeof(float);
  char* ws = nullptr;
  hipError_t e = workspace_alloc(reinterpret_cast<void**>(&ws), bytes, stream);
  if (e != hipSuccess) return e;
  int* flag = reinterpret_cast<int*>(ws);
  float* lse = reinterpret_cast<float*>(ws + 256);
  float* cg = lse + nl;
  float* splitf = cg + nc;
  float* vdv = splitf + nc;
  float* gfp = vdv + np;
  float* exact = gfp + np;
  float* lnz = exact + np;
  const dim3 grid((unsigned)(nbh * ntile)), blk(kThreads);
  hipLaunchKernelGGL(bwd_lse_kernel<D>, grid, blk, 0, stream, q, k, lse, T, ntile);
  e = hipGetLastError();
  if (e == hipSuccess) {
    hipLaunchKernelGGL(bwd_prep_kernel<D>, dim3((unsigned)nbh), blk, 0, stream, v, beta, cg, splitf,
                       flag, H, T);
    e = hipGetLastError();
  }
  // the q pass first: it forms ln(Z/P), which the kv pass uses
  if (e == hipSuccess) {
    hipLaunchKernelGGL(bwd_q_fast_kernel<D>, grid, blk, 0, stream, q, k, v, beta, out, lse, dout, cg,
                       splitf, dQ, gfp, lnz, flag, H, T, ntile);
    e = hipGetLastError();
  }
  if (e == hipSuccess) {
    hipLaunchKernelGGL(bwd_kv_fast_kernel<D>, grid, blk, 0, stream, q, k, v, beta, out, lse, dout,
                       cg, splitf, lnz, dK, dV, vdv, flag, H, T, ntile);
    e = hipGetLastError();
  }
  // exact element-wise passes: they return at once unless a block raised the flag
  if (e == hipSuccess) {
    hipLaunchKernelGGL(bwd_kv_kernel<D>, grid, blk, 0, stream, q, k, v, beta, out, lse, dout, dK, dV,
                       H, T, ntile, flag);
    e = hipGetLastError();
  }
  if (e == hipSuccess) {
    hipLaunchKernelGGL(bwd_q_kernel<D>, grid, blk, 0, stream, q, k, v, beta, out, lse, dout, dQ,
                       exact, H, T, ntile, flag);
    e = hipGetLastError();
  }
  if (e == hipSuccess) {
    hipLaunchKernelGGL(dbeta_kernel<D>, dim3((unsigned)H), dim3(128), 0, stream, exact, vdv, gfp,
                       beta, flag, dbeta, B, H, ntile);
    e = hipGetLastError();
  }
  const hipError_t f = workspace_free(ws, stream);
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
