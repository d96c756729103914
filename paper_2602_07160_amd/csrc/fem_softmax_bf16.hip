// Fused causal softmax-prior FEM read on the gfx950 matrix cores (bf16 inputs).
//
// Computes, per (b, h, t, j),
//   F = (1/beta_j) log sum_{i<=t} alpha_{t,i} exp(beta_j v_{i,j}),
//   alpha_{t,.} = softmax_{i<=t}(q_t . k_i / sqrt d)
// (free-energy read, Sec. 2.3; softmax prior, Sec. 1) in one flash-style pass:
//
//   * log2 domain throughout: scores are scaled by log2(e)/sqrt(d) and the
//     tilt exponent is x_{i,j} = beta_j log2(e) v_{i,j}.
//   * S^T = K Q^T per 64-key tile on MFMA (v_mfma_f32_32x32x16_bf16); the
//     transposed product leaves one query per lane pair, so row max / row sum
//     need one v_permlane32_swap and no LDS traffic.
//   * Online row softmax with a running row max m_t (raised lazily, only when
//     a tile beats it by kRowLag) and a row sum l_t accumulated from the SAME
//     bf16-rounded probabilities that feed the product (v_dot2 with ones), so
//     that rounding P cancels between numerator and normaliser.
//   * Tilted values E_{i,j} = 2^(x_{i,j} - c_j + kBias), formed once per K/V
//     tile per workgroup and shared by all its waves through LDS.  c_j is a
//     running per-channel maximum of x over the tiles seen so far (raised
//     lazily, only when a tile beats it by kColLag); when it rises the
//     accumulator columns are rescaled by 2^(c_old - c_new).  This is the
//     paper's per-channel LSE shift ("Numerical stability" paragraph of the
//     two-level gated FEM appendix) made streaming.
//   * O^T += E^T P^T on MFMA with E split into bf16 hi + lo parts (two
//     products): bf16 alone would cost up to 2^-8/beta in the output, which
//     exceeds a 2e-2 budget for beta < 0.2.
//   * Epilogue o = (log2 acc - log2 l + c_j - kBias) / (beta_j log2 e).  An
//     accumulator below kUnderflow (its in-support terms sat too far below the
//     shared column shift) is recomputed exactly by the wave with a joint
//     per-(t, j) log-sum-exp in fp32.
//
// Work decomposition: one workgroup of NW waves owns BQ = 32*NW query rows of
// one (b, h); each wave owns 32 rows.  Workgroups are launched longest-first
// (largest causal extent first); consecutive heads land on consecutive XCDs.

#include "fem_device.h"
#include "fem_internal.h"

#include <mutex>

namespace fem {
namespace {

constexpr float kBias = 64.f;        // E = 2^(x - c + kBias) <= 2^(kBias + kColLag)
constexpr float kColLag = 16.f;      // column shift raised only past this lag
constexpr float kRowLag = 8.f;       // row max raised only past this lag (P <= 2^8)
constexpr float kUnderflow = 0x1p-64f;

template <int D, int NW>
struct Cfg {
  static constexpr int BQ = NW * 32;      // query rows per workgroup
  static constexpr int BK = 64;           // keys per tile
  static constexpr int NT = NW * 64;      // threads
  static constexpr int NCB = D / 32;      // 32-channel output blocks
  static constexpr int NKS = D / 16;      // 16-wide k-steps of Q K^T
  static constexpr int KROW = D + 8;      // K tile row stride (bf16), +16 B pad
  static constexpr int EROW = BK + 8;     // E^T row stride (bf16), +16 B pad
  static constexpr int NPART = NT / D;    // tilt threads per channel
  static constexpr int KPP = BK / NPART;  // keys per tilt thread
  static constexpr size_t LDS =
      sizeof(bf16) * (BK * KROW + BK * D + 2 * D * EROW) +
      sizeof(float) * (4 * D + NPART * D + NW * D) + 16;
  static_assert(NT % D == 0 && BK % NPART == 0, "tilt mapping");
};

// Position of key r (0..63 within a tile) inside an E^T row.  Within each
// 16-key group the keys are stored in the order the MFMA B operand (P^T,
// taken straight from the S^T accumulator layout) consumes them: lane half h
// holds keys {4h..4h+3, 8+4h..8+4h+3} as its 8 consecutive k-slots.
__device__ __forceinline__ int e_pos(int r) {
  const int g = r & 15;
  return (r & ~15) + (((g >> 2) & 1) << 3) + (((g >> 3) & 1) << 2) + (g & 3);
}

// Exact fp32 read of one (t, j) by the whole wave: joint log-sum-exp of
// (score + tilt) over i <= t, minus the log-sum-exp of the scores.
template <int D>
__device__ float exact_read(const bf16* __restrict__ Qh, const bf16* __restrict__ Kh,
                            const bf16* __restrict__ Vh, int t, int j, float scale2,
                            float bl) {
  const int lane = threadIdx.x & 63;
  Lse2 num, den;
  const bf16x8* qrow = reinterpret_cast<const bf16x8*>(Qh + (size_t)t * D);
  for (int i = lane; i <= t; i += 64) {
    const bf16x8* krow = reinterpret_cast<const bf16x8*>(Kh + (size_t)i * D);
    float dot = 0.f;
#pragma unroll 4
    for (int c = 0; c < D / 8; ++c) {
      bf16x8 a = qrow[c], b = krow[c];
#pragma unroll
      for (int e = 0; e < 8; ++e) dot += (float)a[e] * (float)b[e];
    }
    const float s = dot * scale2;
    den.add(s);
    num.add(s + (float)Vh[(size_t)i * D + j] * bl);
  }
  return (num.wave_total() - den.wave_total()) / bl;
}

template <int D, int NW>
__global__ __launch_bounds__(NW * 64) void softmax_bf16_kernel(
    const bf16* __restrict__ Q, const bf16* __restrict__ K, const bf16* __restrict__ V,
    const float* __restrict__ beta, float* __restrict__ out, int H, int T, int nqb,
    int nbh) {
  using C = Cfg<D, NW>;
  extern __shared__ __align__(16) unsigned char smem[];
  bf16* sK = reinterpret_cast<bf16*>(smem);
  bf16* sV = sK + C::BK * C::KROW;
  bf16* sEh = sV + C::BK * D;
  bf16* sEl = sEh + D * C::EROW;
  float* sC = reinterpret_cast<float*>(sEl + D * C::EROW);  // running column shift
  float* sBl = sC + D;                                      // beta * log2(e)
  float* sInv = sBl + D;                                    // 1 / (beta * log2(e))
  float* sG = sInv + D;                                     // column rescale, this tile
  float* sPart = sG + D;                                    // partial column maxima
  float* sCw = sPart + C::NPART * D;  // column shift each wave's accumulator ends on
  int* sRose = reinterpret_cast<int*>(sCw + NW * D);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int n = lane & 31;   // query column of this lane in the 32x32 blocks
  const int hl = lane >> 5;  // lane half

  const int bid = blockIdx.x;
  const int qb = nqb - 1 - bid / nbh;  // longest causal extent first
  const int bh = bid % nbh;
  const int h = bh % H;
  const int q0 = qb * C::BQ;
  const size_t base = (size_t)bh * T * D;
  const bf16* Qh = Q + base;
  const bf16* Kh = K + base;
  const bf16* Vh = V + base;
  float* Oh = out + base;

  for (int j = tid; j < D; j += C::NT) {
    const float bl = beta[h * D + j] * kLog2e;
    sBl[j] = bl;
    sInv[j] = 1.f / bl;
    sC[j] = -INFINITY;
  }

  const int wq0 = q0 + wave * 32;  // first query row of this wave
  const int tq = wq0 + n;          // this lane's query row
  const bool wave_live = wq0 < T;

  bf16x8 qf[C::NKS];
#pragma unroll
  for (int ks = 0; ks < C::NKS; ++ks) {
    bf16x8 z = {};
    qf[ks] = (tq < T) ? *reinterpret_cast<const bf16x8*>(Qh + (size_t)tq * D + ks * 16 + hl * 8)
                      : z;
  }

  f32x16 acc[C::NCB];
#pragma unroll
  for (int cb = 0; cb < C::NCB; ++cb) acc[cb] = f32x16{};
  float m = -INFINITY;  // running row max (log2 units), shared by the lane pair
  float l = 0.f;        // this lane's half of the row sum
  const float scale2 = kLog2e / sqrtf((float)D);

  const int qlast = min(q0 + C::BQ, T) - 1;
  const int ntiles = qlast / C::BK + 1;
  // Last tile this wave multiplies into its accumulator.  Later tiles may still
  // raise the shared column shift; the wave keeps the shift its accumulator
  // was last rescaled to (sCw) instead of rescaling for tiles it skips.
  const int wlast = min((wq0 + 31) / C::BK, ntiles - 1);

  for (int kt = 0; kt < ntiles; ++kt) {
    const int k0 = kt * C::BK;

    // ---- K and V tile: HBM -> LDS (16-byte vectors; rows past T are zero)
    constexpr int CH = D / 8;
    for (int c = tid; c < C::BK * CH; c += C::NT) {
      const int r = c / CH, cc = c % CH;
      bf16x8 kv = {}, vv = {};
      if (k0 + r < T) {
        kv = *reinterpret_cast<const bf16x8*>(Kh + (size_t)(k0 + r) * D + cc * 8);
        vv = *reinterpret_cast<const bf16x8*>(Vh + (size_t)(k0 + r) * D + cc * 8);
      }
      *reinterpret_cast<bf16x8*>(sK + r * C::KROW + cc * 8) = kv;
      *reinterpret_cast<bf16x8*>(sV + r * D + cc * 8) = vv;
    }
    if (tid == 0) *sRose = 0;
    __syncthreads();

    // ---- tilt: column max, running shift, E = 2^(x - c + bias) as bf16 hi/lo
    {
      const int j = tid % D, part = tid / D;
      const float bl = sBl[j];
      const float cold = sC[j];
      float xs[C::KPP];
      float mx = -INFINITY;
#pragma unroll
      for (int r = 0; r < C::KPP; ++r) {
        const int key = part * C::KPP + r;
        xs[r] = (float)sV[key * D + j] * bl;
        if (k0 + key < T) mx = fmaxf(mx, xs[r]);
      }
      sPart[part * D + j] = mx;
      __syncthreads();
      float tmx = sPart[j];
#pragma unroll
      for (int p = 1; p < C::NPART; ++p) tmx = fmaxf(tmx, sPart[p * D + j]);
      const float cnew = (tmx > cold + kColLag) ? tmx : cold;
      const float sh = kBias - cnew;
#pragma unroll
      for (int r = 0; r < C::KPP; ++r) {
        const int key = part * C::KPP + r;
        const float e = (k0 + key < T) ? exp2_hw(xs[r] + sh) : 0.f;
        const bf16 hi = (bf16)e;
        const bf16 lo = (bf16)(e - (float)hi);
        sEh[j * C::EROW + e_pos(key)] = hi;
        sEl[j * C::EROW + e_pos(key)] = lo;
      }
      if (part == 0) {
        sG[j] = exp2_hw(cold - cnew);
        if (cnew != cold) *sRose = 1;
        sC[j] = cnew;
      }
    }
    __syncthreads();

    // ---- per wave: scores, online softmax, tilted product
    if (wave_live && k0 <= wq0 + 31) {
      f32x16 sacc[2] = {f32x16{}, f32x16{}};
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
        for (int ks = 0; ks < C::NKS; ++ks) {
          const bf16x8 a =
              *reinterpret_cast<const bf16x8*>(sK + (kb * 32 + n) * C::KROW + ks * 16 + hl * 8);
          sacc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[ks], sacc[kb], 0, 0, 0);
        }
      }
      const bool need_mask = (k0 + C::BK - 1 > wq0) || (k0 + C::BK > T);
      float mx = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          float s = sacc[kb][i] * scale2;
          if (need_mask) {
            const int key = k0 + kb * 32 + (i >> 2) * 8 + hl * 4 + (i & 3);
            if (key > tq || key >= T) s = -INFINITY;
          }
          sacc[kb][i] = s;
          mx = fmaxf(mx, s);
        }
      }
      mx = fmaxf(mx, other_half(mx));
      const float mnew = (mx > m + kRowLag) ? mx : m;
      if (__any(mnew != m)) {
        const float alpha = exp2_hw(m - mnew);
        l *= alpha;
#pragma unroll
        for (int cb = 0; cb < C::NCB; ++cb) acc[cb] *= alpha;
        m = mnew;
      }

      bf16x8 pf[4];
      const bf16x2 ones = to_bf16x2(1.f, 1.f);
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const int kb = ks >> 1, s0 = (ks & 1) * 8;
#pragma unroll
        for (int u = 0; u < 8; u += 2) {
          const bf16x2 p2 = to_bf16x2(exp2_hw(sacc[kb][s0 + u] - m),
                                      exp2_hw(sacc[kb][s0 + u + 1] - m));
          pf[ks][u] = p2[0];
          pf[ks][u + 1] = p2[1];
          l = dot2_bf16(p2, ones, l);
        }
      }

      if (*sRose) {
#pragma unroll
        for (int cb = 0; cb < C::NCB; ++cb) {
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            const f32x4 gg = *reinterpret_cast<const f32x4*>(sG + cb * 32 + g * 8 + hl * 4);
#pragma unroll
            for (int e = 0; e < 4; ++e) acc[cb][g * 4 + e] *= gg[e];
          }
        }
      }

#pragma unroll
      for (int cb = 0; cb < C::NCB; ++cb) {
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
          const int off = (cb * 32 + n) * C::EROW + ks * 16 + hl * 8;
          const bf16x8 ah = *reinterpret_cast<const bf16x8*>(sEh + off);
          const bf16x8 al = *reinterpret_cast<const bf16x8*>(sEl + off);
          acc[cb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, pf[ks], acc[cb], 0, 0, 0);
          acc[cb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(al, pf[ks], acc[cb], 0, 0, 0);
        }
      }
      if (kt == wlast) {
        for (int j = lane; j < D; j += 64) sCw[wave * D + j] = sC[j];
      }
    }
    __syncthreads();
  }

  if (!wave_live) return;

  // ---- epilogue: o = (log2 acc - log2 l + c - bias) / (beta log2 e)
  const float ll = log2_hw(l + other_half(l));
  uint64_t flags = 0;
#pragma unroll
  for (int cb = 0; cb < C::NCB; ++cb) {
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int ch0 = cb * 32 + g * 8 + hl * 4;
      f32x4 o;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float a = acc[cb][g * 4 + e];
        o[e] = ((log2_hw(a) - kBias) - ll + sCw[wave * D + ch0 + e]) * sInv[ch0 + e];
        if (!(a >= kUnderflow) && tq < T) flags |= 1ull << (cb * 16 + g * 4 + e);
      }
      if (tq < T) *reinterpret_cast<f32x4*>(Oh + (size_t)tq * D + ch0) = o;
    }
  }

  // ---- rare path: exact recompute of accumulators that underflowed
  while (true) {
    const uint64_t who = __ballot(flags != 0);
    if (who == 0) break;
    const int src = __builtin_ctzll(who);
    const uint32_t flo = __builtin_amdgcn_readlane((uint32_t)flags, src);
    const uint32_t fhi = __builtin_amdgcn_readlane((uint32_t)(flags >> 32), src);
    const uint64_t fl = ((uint64_t)fhi << 32) | flo;
    const int e = __builtin_ctzll(fl);
    const int t = __builtin_amdgcn_readlane(tq, src);
    const int cb = e >> 4, i = e & 15;
    const int ch = cb * 32 + (i >> 2) * 8 + (src >> 5) * 4 + (i & 3);
    const float o = exact_read<D>(Qh, Kh, Vh, t, ch, scale2, sBl[ch]);
    if (lane == src) {
      flags &= ~(1ull << e);
      Oh[(size_t)t * D + ch] = o;
    }
  }
}

template <int D, int NW>
hipError_t launch(const void* Q, const void* K, const void* V, const float* beta, float* out,
                  int B, int H, int T, hipStream_t stream) {
  using C = Cfg<D, NW>;
  static std::once_flag once;
  static hipError_t attr_err = hipSuccess;
  std::call_once(once, [] {
    attr_err = hipFuncSetAttribute(reinterpret_cast<const void*>(&softmax_bf16_kernel<D, NW>),
                                   hipFuncAttributeMaxDynamicSharedMemorySize, (int)C::LDS);
  });
  if (attr_err != hipSuccess) return attr_err;
  const int nqb = (T + C::BQ - 1) / C::BQ;
  const int nbh = B * H;
  dim3 grid((unsigned)(nqb * nbh)), block(C::NT);
  hipLaunchKernelGGL((softmax_bf16_kernel<D, NW>), grid, block, C::LDS, stream,
                     reinterpret_cast<const bf16*>(Q), reinterpret_cast<const bf16*>(K),
                     reinterpret_cast<const bf16*>(V), beta, out, H, T, nqb, nbh);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_softmax_bf16(const void* Q, const void* K, const void* V, const float* beta,
                               float* out, int B, int H, int T, int d, hipStream_t stream) {
  switch (d) {
    case 32: return launch<32, 8>(Q, K, V, beta, out, B, H, T, stream);
    case 64: return launch<64, 8>(Q, K, V, beta, out, B, H, T, stream);
    case 128: return launch<128, 8>(Q, K, V, beta, out, B, H, T, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace fem
