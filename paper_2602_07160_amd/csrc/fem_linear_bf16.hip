// Linear-attention-prior FEM read as an O(T) chunked scan on the gfx950 matrix
// cores (bf16 inputs, fp32 state).
//
// Prior p_t(i) = <phi q_t, phi k_i> / sum_{r<=t} <phi q_t, phi k_r>, phi = elu+1
// (linear attention, Appendix "Selection distributions, support, and
// normalization"), read F_{t,j} = (1/beta_j) log sum_{i<=t} p_t(i) e^{beta_j v_ij}
// (Sec. 2.3).  Streaming form (Appendix "Parameterizations of the Prior
// Selection", associative scan with a constant channel for the normaliser):
//
//   num_t = phi(q_t)^T S_t,  den_t = phi(q_t)^T z_t,
//   S_t = sum_{i<=t} phi(k_i) E_i^T,  z_t = sum_{i<=t} phi(k_i),
//   E_{ij} = 2^(x_ij - c_j + kBias),  x = beta v log2(e),
//   F = (log2 num - log2 den + c_j - kBias) / (beta_j log2 e).
//
// c_j is a running per-channel maximum of x, raised lazily (only when a chunk
// beats it by kColLag); when it rises the state S is rescaled by
// 2^(c_old - c_new) (the paper's per-channel LSE shift, made streaming).
//
// Chunking: 64-token chunks inside 512-token segments.
//   kernel 1 (state):  one workgroup per (b, h, segment): the segment's own
//                      state [S | z] and shift c, starting from zero.
//   kernel 2 (read):   one workgroup per (b, h, segment): combines the states
//                      of all earlier segments into its entering state, then
//                      scans its chunks: intra-chunk (phi Q phi K^T masked) E,
//                      inter-chunk phi Q S, and the state update phi K^T E.
// All products run on v_mfma_f32_32x32x16_bf16 in transposed form (outputs
// are [channel][token]); E and S enter as bf16 hi + lo pairs, the masked
// intra-chunk scores A enter as bf16 and the normaliser is summed from the
// same rounded A.  An output whose numerator underflowed is recomputed exactly
// by the wave.

#include "fem_device.h"
#include "fem_internal.h"

#include <mutex>

namespace fem {
namespace {

constexpr int DK = 64, DV = 64;  // supported widths
constexpr int CH = 64;           // tokens per chunk
constexpr int SEGC = 8;          // chunks per segment
constexpr int SEG = CH * SEGC;   // tokens per segment
constexpr int NTH = 256;         // 4 waves
constexpr int ROW = 64 + 8;      // padded bf16 row (64 values + 16 B)
constexpr int SROW = DK + 8;     // padded S^T row (bf16)
constexpr int STATE = DV * DK + DK + DV;  // floats per saved segment state

constexpr float kBias = 64.f;
constexpr float kColLag = 16.f;
constexpr float kUnderflow = 0x1p-64f;

typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4;

struct LinSmem {
  bf16 fq[CH * ROW];    // phi(Q) [token][d_k]
  bf16 fk[CH * ROW];    // phi(K) [token][d_k]
  bf16 fkt[DK * ROW];   // phi(K)^T [d_k][key, MFMA order]
  bf16 v[CH * ROW];     // V [token][d_v]
  bf16 eh[DV * ROW];    // E^T hi [d_v][key, MFMA order]
  bf16 el[DV * ROW];    // E^T lo
  bf16 sh[DV * SROW];   // S^T hi [d_v][d_k]
  bf16 sl[DV * SROW];   // S^T lo
  float c[DV];          // running shift
  float g[DV];          // shift change of this chunk, 2^(c_old - c_new)
  float bl[DV];         // beta log2 e
  float inv[DV];
  float z[DK];          // sum of phi(k) over earlier chunks
  float zc[DK];         // sum of phi(k) over this chunk
  int rose;
};

// Key r of a chunk -> position inside an MFMA-ordered row (see the softmax
// kernel: the B operand taken from a transposed accumulator holds keys
// {4h..4h+3, 8+4h..8+4h+3} of each 16-key group in lane half h).
__device__ __forceinline__ int e_pos(int r) {
  const int g = r & 15;
  return (r & ~15) + (((g >> 2) & 1) << 3) + (((g >> 3) & 1) << 2) + (g & 3);
}

__device__ __forceinline__ float phi(float x) { return x > 0.f ? x + 1.f : exp2_hw(x * kLog2e); }

// Exact fp32 read of one (t, j) of the linear prior by the whole wave.
__device__ float exact_read_linear(const bf16* __restrict__ Qh, const bf16* __restrict__ Kh,
                                   const bf16* __restrict__ Vh, int t, int j, float bl) {
  const int lane = threadIdx.x & 63;
  Lse2 num, den;
  const bf16* qrow = Qh + (size_t)t * DK;
  for (int i = lane; i <= t; i += 64) {
    const bf16* krow = Kh + (size_t)i * DK;
    float a = 0.f;
    for (int c = 0; c < DK; ++c) a = fmaf(phi((float)qrow[c]), phi((float)krow[c]), a);
    const float w = log2_hw(a);
    den.add(w);
    num.add(w + (float)Vh[(size_t)i * DV + j] * bl);
  }
  return (num.wave_total() - den.wave_total()) / bl;
}

// One chunk of the scan.  Loads tokens [t0, t0 + CH) (rows past T are zero and
// masked), tilts V, rescales the state, produces outputs (OUT) and updates S.
// Wave w owns S^T block (dvb = w >> 1, dkb = w & 1) and output block
// (dvb = w >> 1, qb = w & 1).
template <bool OUT>
__device__ __forceinline__ void scan_chunk(LinSmem& sm, f32x16& st, const bf16* Qh,
                                           const bf16* Kh, const bf16* Vh, float* Oh, int t0,
                                           int T) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n = lane & 31, hl = lane >> 5;
  const int dvb = wave >> 1, sub = wave & 1;

  // ---- stage Q, K, V of the chunk; phi in fp32, rounded to bf16
  for (int e = tid; e < CH * 8; e += NTH) {
    const int r = e >> 3, c8 = (e & 7) * 8;
    const bool ok = t0 + r < T;
    bf16x8 kq = {}, kk = {}, kv = {};
    if (ok) {
      kk = *reinterpret_cast<const bf16x8*>(Kh + (size_t)(t0 + r) * DK + c8);
      kv = *reinterpret_cast<const bf16x8*>(Vh + (size_t)(t0 + r) * DV + c8);
      if (OUT) kq = *reinterpret_cast<const bf16x8*>(Qh + (size_t)(t0 + r) * DK + c8);
    }
    bf16x8 pk, pq;
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      pk[u] = ok ? (bf16)phi((float)kk[u]) : (bf16)0.f;
      pq[u] = ok ? (bf16)phi((float)kq[u]) : (bf16)0.f;
      sm.fkt[(c8 + u) * ROW + e_pos(r)] = pk[u];
    }
    *reinterpret_cast<bf16x8*>(sm.fk + r * ROW + c8) = pk;
    *reinterpret_cast<bf16x8*>(sm.v + r * ROW + c8) = kv;
    if (OUT) *reinterpret_cast<bf16x8*>(sm.fq + r * ROW + c8) = pq;
  }
  if (tid == 0) sm.rose = 0;
  __syncthreads();

  // ---- tilt: wave w owns channels 16w .. 16w+15; lane = channel + 16 * key group
  {
    const int jj = lane & 15, g = lane >> 4;
    const int j = wave * 16 + jj;
    const float bl = sm.bl[j];
    float vv[16];
    float vmax = -INFINITY;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        const int key = 4 * (g + 4 * u) + b;
        vv[u * 4 + b] = (float)sm.v[key * ROW + j];
        if (t0 + key < T) vmax = fmaxf(vmax, vv[u * 4 + b]);
      }
    }
    vmax = fmaxf(vmax, __shfl_xor(vmax, 16));
    vmax = fmaxf(vmax, __shfl_xor(vmax, 32));
    const float mx = vmax * bl;
    const float cold = sm.c[j];
    const float cnew = (mx > cold + kColLag) ? mx : cold;
    const float sh = kBias - cnew;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int key0 = 4 * (g + 4 * u);
      bf16x4 hi, lo;
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        const float e = (t0 + key0 + b < T) ? exp2_hw(fmaf(vv[u * 4 + b], bl, sh)) : 0.f;
        hi[b] = (bf16)e;
        lo[b] = (bf16)(e - (float)hi[b]);
      }
      *reinterpret_cast<bf16x4*>(sm.eh + j * ROW + e_pos(key0)) = hi;
      *reinterpret_cast<bf16x4*>(sm.el + j * ROW + e_pos(key0)) = lo;
    }
    __syncthreads();  // every lane has read sm.c before it changes
    if (g == 0) {
      sm.g[j] = exp2_hw(cold - cnew);
      sm.c[j] = cnew;
      if (cnew != cold) sm.rose = 1;
    }
    // chunk sum of phi(k): wave 0..3 each sum 16 d_k columns
    if (g == 0) {
      const int dkc = wave * 16 + jj;
      float s = 0.f;
      for (int r = 0; r < CH; ++r) s += (float)sm.fk[r * ROW + dkc];
      sm.zc[dkc] = s;
    }
  }
  __syncthreads();

  // ---- rescale the state rows (d_v) when the shift rose, publish S^T hi/lo
  if (sm.rose) {
#pragma unroll
    for (int i = 0; i < 16; ++i) st[i] *= sm.g[dvb * 32 + (i >> 2) * 8 + hl * 4 + (i & 3)];
  }
  if (OUT) {
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int row = dvb * 32 + (i >> 2) * 8 + hl * 4 + (i & 3);
      const int col = sub * 32 + n;
      const bf16 hi = (bf16)st[i];
      sm.sh[row * SROW + col] = hi;
      sm.sl[row * SROW + col] = (bf16)(st[i] - (float)hi);
    }
    __syncthreads();

    // ---- outputs of query block qb = sub, channel block dvb
    const int qb = sub;
    const int tq = t0 + qb * 32 + n;
    // A^T blocks (keys kb x queries qb), kb <= qb
    f32x16 at[2] = {f32x16{}, f32x16{}};
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      if (kb > qb) continue;
#pragma unroll
      for (int ks = 0; ks < DK / 16; ++ks) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(sm.fk + (kb * 32 + n) * ROW + ks * 16 + hl * 8);
        const bf16x8 b = *reinterpret_cast<const bf16x8*>(sm.fq + (qb * 32 + n) * ROW + ks * 16 + hl * 8);
        at[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, at[kb], 0, 0, 0);
      }
    }
    // mask (key > query), round to bf16, normaliser from the rounded values
    bf16x8 pf[4] = {};
    float den = 0.f;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const int kb = ks >> 1, s0 = (ks & 1) * 8;
      if (kb > qb) continue;
#pragma unroll
      for (int u = 0; u < 8; u += 2) {
        const int i0 = s0 + u, i1 = s0 + u + 1;
        const int key0 = kb * 32 + (i0 >> 2) * 8 + hl * 4 + (i0 & 3);
        const int key1 = kb * 32 + (i1 >> 2) * 8 + hl * 4 + (i1 & 3);
        const float a0 = (key0 <= qb * 32 + n) ? at[kb][i0] : 0.f;
        const float a1 = (key1 <= qb * 32 + n) ? at[kb][i1] : 0.f;
        const bf16x2 p2 = to_bf16x2(a0, a1);
        pf[ks][u] = p2[0];
        pf[ks][u + 1] = p2[1];
        den = add_bf16x2(p2, den);
      }
    }
    // inter-chunk normaliser phi(q)^T z, this lane's half of d_k
    {
      const bf16* fqr = sm.fq + (qb * 32 + n) * ROW;
#pragma unroll
      for (int ks = 0; ks < DK / 16; ++ks) {
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int dk = ks * 16 + hl * 8 + u;
          den = fmaf((float)fqr[dk], sm.z[dk], den);
        }
      }
    }
    den += other_half(den);
    // numerator: E^T A^T (intra) + S^T phi(Q)^T (inter)
    f32x16 num = f32x16{};
    const int eoff = (dvb * 32 + n) * ROW + hl * 8;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      if ((ks >> 1) > qb) continue;
      const bf16x8 ah = *reinterpret_cast<const bf16x8*>(sm.eh + eoff + ks * 16);
      const bf16x8 al = *reinterpret_cast<const bf16x8*>(sm.el + eoff + ks * 16);
      num = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, pf[ks], num, 0, 0, 0);
      num = __builtin_amdgcn_mfma_f32_32x32x16_bf16(al, pf[ks], num, 0, 0, 0);
    }
    const int soff = (dvb * 32 + n) * SROW + hl * 8;
#pragma unroll
    for (int ks = 0; ks < DK / 16; ++ks) {
      const bf16x8 ah = *reinterpret_cast<const bf16x8*>(sm.sh + soff + ks * 16);
      const bf16x8 al = *reinterpret_cast<const bf16x8*>(sm.sl + soff + ks * 16);
      const bf16x8 b = *reinterpret_cast<const bf16x8*>(sm.fq + (qb * 32 + n) * ROW + ks * 16 + hl * 8);
      num = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, b, num, 0, 0, 0);
      num = __builtin_amdgcn_mfma_f32_32x32x16_bf16(al, b, num, 0, 0, 0);
    }
    // epilogue
    int ed;
    const float fd = log2_hw(frexpf(den, &ed));
    uint32_t flags = 0;
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) {
      const int ch0 = dvb * 32 + g4 * 8 + hl * 4;
      f32x4 o;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float a = num[g4 * 4 + e];
        int ea;
        const float fa = log2_hw(frexpf(a, &ea));
        o[e] = ((float)(ea - ed - (int)kBias) + (fa - fd) + sm.c[ch0 + e]) * sm.inv[ch0 + e];
        if (!(a >= kUnderflow) && tq < T) flags |= 1u << (g4 * 4 + e);
      }
      if (tq < T) *reinterpret_cast<f32x4*>(Oh + (size_t)tq * DV + ch0) = o;
    }
    while (true) {
      const uint64_t who = __ballot(flags != 0);
      if (who == 0) break;
      const int src = __builtin_ctzll(who);
      const uint32_t fl = __builtin_amdgcn_readlane(flags, src);
      const int e = __builtin_ctz(fl);
      const int t = __builtin_amdgcn_readlane(tq, src);
      const int ch = dvb * 32 + (e >> 2) * 8 + (src >> 5) * 4 + (e & 3);
      const float o = exact_read_linear(Qh, Kh, Vh, t, ch, sm.bl[ch]);
      if (lane == src) {
        flags &= ~(1u << e);
        Oh[(size_t)t * DV + ch] = o;
      }
    }
  }

  // ---- state update S^T(dvb, dkb = sub) += E^T phi(K)   (keys of this chunk)
  {
    const int eoff = (dvb * 32 + n) * ROW + hl * 8;
    const int koff = (sub * 32 + n) * ROW + hl * 8;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const bf16x8 ah = *reinterpret_cast<const bf16x8*>(sm.eh + eoff + ks * 16);
      const bf16x8 al = *reinterpret_cast<const bf16x8*>(sm.el + eoff + ks * 16);
      const bf16x8 b = *reinterpret_cast<const bf16x8*>(sm.fkt + koff + ks * 16);
      st = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, b, st, 0, 0, 0);
      st = __builtin_amdgcn_mfma_f32_32x32x16_bf16(al, b, st, 0, 0, 0);
    }
  }
  __syncthreads();
  if (tid < DK) sm.z[tid] += sm.zc[tid];
  __syncthreads();
}

template <bool OUT>
__global__ __launch_bounds__(NTH) void linear_kernel(const bf16* __restrict__ Q,
                                                     const bf16* __restrict__ K,
                                                     const bf16* __restrict__ V,
                                                     const float* __restrict__ beta,
                                                     float* __restrict__ out,
                                                     float* __restrict__ ws, int H, int T,
                                                     int nseg) {
  __shared__ __align__(16) LinSmem sm;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int hl = lane >> 5;
  const int seg = blockIdx.x % nseg;
  const int bh = blockIdx.x / nseg;
  const int h = bh % H;
  const bf16* Qh = Q + (size_t)bh * T * DK;
  const bf16* Kh = K + (size_t)bh * T * DK;
  const bf16* Vh = V + (size_t)bh * T * DV;
  float* Oh = out + (size_t)bh * T * DV;
  float* wsh = ws + (size_t)bh * nseg * STATE;
  const int dvb = wave >> 1, sub = wave & 1;

  if (tid < DV) {
    const float bl = beta[h * DV + tid] * kLog2e;
    sm.bl[tid] = bl;
    sm.inv[tid] = 1.f / bl;
    sm.c[tid] = -INFINITY;
  }
  if (tid < DK) sm.z[tid] = 0.f;
  f32x16 st = f32x16{};
  __syncthreads();

  if (OUT && seg > 0) {
    // entering state: all earlier segments, each relative to its own shift
    if (tid < DV) {
      float C = -INFINITY;
      for (int s = 0; s < seg; ++s) C = fmaxf(C, wsh[(size_t)s * STATE + DV * DK + DK + tid]);
      sm.c[tid] = C;
    }
    if (tid < DK) {
      float z = 0.f;
      for (int s = 0; s < seg; ++s) z += wsh[(size_t)s * STATE + DV * DK + tid];
      sm.z[tid] = z;
    }
    __syncthreads();
    for (int s = 0; s < seg; ++s) {
      const float* S = wsh + (size_t)s * STATE;
      const float* cs = S + DV * DK + DK;
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int row = dvb * 32 + (i >> 2) * 8 + hl * 4 + (i & 3);
        const int col = sub * 32 + (lane & 31);
        st[i] = fmaf(S[row * DK + col], exp2_hw(cs[row] - sm.c[row]), st[i]);
      }
    }
  }

  const int tbeg = seg * SEG;
  const int tend = min(tbeg + SEG, T);
  for (int t0 = tbeg; t0 < tend; t0 += CH) scan_chunk<OUT>(sm, st, Qh, Kh, Vh, Oh, t0, T);

  if (!OUT) {
    float* S = wsh + (size_t)seg * STATE;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int row = dvb * 32 + (i >> 2) * 8 + hl * 4 + (i & 3);
      const int col = sub * 32 + (lane & 31);
      S[row * DK + col] = st[i];
    }
    if (tid < DK) S[DV * DK + tid] = sm.z[tid];
    if (tid < DV) S[DV * DK + DK + tid] = sm.c[tid];
  }
}

}  // namespace

hipError_t launch_linear_bf16(const void* Q, const void* K, const void* V, const float* beta,
                              float* out, int B, int H, int T, int dk, int dv, int chunk,
                              hipStream_t stream) {
  if (dk != DK || dv != DV || chunk != CH) return hipErrorNotSupported;
  const int nseg = (T + SEG - 1) / SEG;
  const int nbh = B * H;
  float* ws = nullptr;
  const size_t bytes = (size_t)nbh * nseg * STATE * sizeof(float);
  hipError_t e = workspace_alloc(reinterpret_cast<void**>(&ws), bytes, stream);
  if (e != hipSuccess) return e;
  if (nseg > 1) {
    hipLaunchKernelGGL(linear_kernel<false>, dim3((unsigned)(nbh * nseg)), dim3(NTH), 0, stream,
                       reinterpret_cast<const bf16*>(Q), reinterpret_cast<const bf16*>(K),
                       reinterpret_cast<const bf16*>(V), beta, out, ws, H, T, nseg);
    e = hipGetLastError();
  }
  if (e == hipSuccess) {
    hipLaunchKernelGGL(linear_kernel<true>, dim3((unsigned)(nbh * nseg)), dim3(NTH), 0, stream,
                       reinterpret_cast<const bf16*>(Q), reinterpret_cast<const bf16*>(K),
                       reinterpret_cast<const bf16*>(V), beta, out, ws, H, T, nseg);
    e = hipGetLastError();
  }
  const hipError_t f = workspace_free(ws, stream);
  return e != hipSuccess ? e : f;
}

}  // namespace fem
