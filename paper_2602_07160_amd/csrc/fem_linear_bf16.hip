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
//   kernel 2 (prefix): per (b, h), the exclusive prefix of the segment states
//                      (the state entering each segment), one thread per
//                      state entry, in place.
//   kernel 3 (read):   one workgroup per (b, h, segment): loads its entering
//                      state, then scans its chunks: intra-chunk (phi Q phi
//                      K^T masked) E, inter-chunk phi Q S, and the state update
//                      phi K^T E.  The next chunk's Q, K, V are fetched into
//                      registers while the current one is processed.
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
  float zc[4 * DK];     // partial sums of phi(k) over this chunk (four row quarters)
  int rose;
};

// Key r of a chunk -> position inside an MFMA-ordered row (see the softmax
// kernel: the B operand taken from a transposed accumulator holds keys
// {4h..4h+3, 8+4h..8+4h+3} of each 16-key group in lane half h).
__device__ __forceinline__ int e_pos(int r) {
  const int g = r & 15;
  return (r & ~15) + (((g >> 2) & 1) << 3) + (((g >> 3) & 1) << 2) + (g & 3);
}

// Workgroup barrier that orders LDS only: every wave's LDS accesses complete
// before it, while global loads in flight (the next chunk's prefetch) keep
// running.  (__syncthreads() would also wait for those.)
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// elu(x) + 1, without a branch: the exponential is evaluated for every x (at
// min(x, 0), so it stays finite) and selected.
__device__ __forceinline__ float phi(float x) {
  const float e = exp2_hw(fminf(x, 0.f) * kLog2e);
  return x > 0.f ? x + 1.f : e;
}

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

// Raw Q, K, V of one chunk held in registers: thread tid covers the 16-byte
// slots e = tid + NTH*i (row e >> 3, columns (e & 7)*8 ..).
constexpr int SLOTS = CH * 8 / NTH;
struct ChunkRegs {
  bf16x8 q[SLOTS], k[SLOTS], v[SLOTS];
};

template <bool OUT>
__device__ __forceinline__ void fetch_chunk(ChunkRegs& cr, const bf16* Qh, const bf16* Kh,
                                            const bf16* Vh, int t0, int T) {
  const int tid = threadIdx.x;
#pragma unroll
  for (int i = 0; i < SLOTS; ++i) {
    const int e = tid + NTH * i, r = e >> 3, c8 = (e & 7) * 8;
    bf16x8 z = {};
    const bool ok = t0 + r < T;
    cr.k[i] = ok ? *reinterpret_cast<const bf16x8*>(Kh + (size_t)(t0 + r) * DK + c8) : z;
    cr.v[i] = ok ? *reinterpret_cast<const bf16x8*>(Vh + (size_t)(t0 + r) * DV + c8) : z;
    if (OUT) cr.q[i] = ok ? *reinterpret_cast<const bf16x8*>(Qh + (size_t)(t0 + r) * DK + c8) : z;
  }
}

// One chunk of the scan.  Stages tokens [t0, t0 + CH) from cr (rows past T
// are zero and masked), starts fetching the next chunk into cr, tilts V,
// rescales the state, produces outputs (OUT) and updates S.
// Wave w owns S^T block (dvb = w >> 1, dkb = w & 1) and output block
// (dvb = w >> 1, qb = w & 1).
template <bool OUT>
__device__ __forceinline__ void scan_chunk(LinSmem& sm, f32x16& st, ChunkRegs& cr,
                                           const bf16* Qh, const bf16* Kh, const bf16* Vh,
                                           float* Oh, int t0, int tnext, int T) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n = lane & 31, hl = lane >> 5;
  const int dvb = wave >> 1, sub = wave & 1;

  // ---- stage Q, K, V of the chunk; phi in fp32, rounded to bf16
#pragma unroll
  for (int i = 0; i < SLOTS; ++i) {
    const int e = tid + NTH * i, r = e >> 3, c8 = (e & 7) * 8;
    // rows past T: phi of the zeros fetched there, times 0 (no branch)
    const float okf = t0 + r < T ? 1.f : 0.f;
    bf16x8 pk, pq;
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      pk[u] = (bf16)(phi((float)cr.k[i][u]) * okf);
      if (OUT) pq[u] = (bf16)(phi((float)cr.q[i][u]) * okf);
      sm.fkt[(c8 + u) * ROW + e_pos(r)] = pk[u];
    }
    *reinterpret_cast<bf16x8*>(sm.fk + r * ROW + c8) = pk;
    *reinterpret_cast<bf16x8*>(sm.v + r * ROW + c8) = cr.v[i];
    if (OUT) *reinterpret_cast<bf16x8*>(sm.fq + r * ROW + c8) = pq;
  }
  if (tid == 0) sm.rose = 0;
  // the next chunk's loads run while this one is processed
  if (tnext < T) fetch_chunk<OUT>(cr, Qh, Kh, Vh, tnext, T);
  lds_barrier();

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
    lds_barrier();  // every lane has read sm.c before it changes
    if (g == 0) {
      sm.g[j] = exp2_hw(cold - cnew);
      sm.c[j] = cnew;
      if (cnew != cold) sm.rose = 1;
    }
    // chunk sum of phi(k): thread (column tid & 63, quarter tid >> 6) sums 16
    // rows; the four partial sums meet in LDS
    {
      const int dkc = tid & 63, q4 = tid >> 6;
      float s = 0.f;
#pragma unroll
      for (int r = 0; r < CH / 4; ++r) s += (float)sm.fk[(q4 * (CH / 4) + r) * ROW + dkc];
      sm.zc[q4 * DK + dkc] = s;
    }
  }
  lds_barrier();

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
    lds_barrier();

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
    // numerator: E^T A^T (intra) + S^T phi(Q)^T (inter), in independent
    // accumulators so the MFMAs do not wait on each other; the inter-chunk
    // normaliser phi(q)^T z (this lane's half of d_k) reuses the phi(Q)
    // fragments, with four partial sums
    f32x16 nacc[4] = {f32x16{}, f32x16{}, f32x16{}, f32x16{}};
    const int eoff = (dvb * 32 + n) * ROW + hl * 8;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      if ((ks >> 1) > qb) continue;
      const bf16x8 ah = *reinterpret_cast<const bf16x8*>(sm.eh + eoff + ks * 16);
      const bf16x8 al = *reinterpret_cast<const bf16x8*>(sm.el + eoff + ks * 16);
      nacc[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, pf[ks], nacc[0], 0, 0, 0);
      nacc[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(al, pf[ks], nacc[1], 0, 0, 0);
    }
    const int soff = (dvb * 32 + n) * SROW + hl * 8;
    float dz[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < DK / 16; ++ks) {
      const bf16x8 ah = *reinterpret_cast<const bf16x8*>(sm.sh + soff + ks * 16);
      const bf16x8 al = *reinterpret_cast<const bf16x8*>(sm.sl + soff + ks * 16);
      const bf16x8 b = *reinterpret_cast<const bf16x8*>(sm.fq + (qb * 32 + n) * ROW + ks * 16 + hl * 8);
      nacc[2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, b, nacc[2], 0, 0, 0);
      nacc[3] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(al, b, nacc[3], 0, 0, 0);
      const f32x4 z0 = *reinterpret_cast<const f32x4*>(sm.z + ks * 16 + hl * 8);
      const f32x4 z1 = *reinterpret_cast<const f32x4*>(sm.z + ks * 16 + hl * 8 + 4);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        dz[u] = fmaf((float)b[u], z0[u], dz[u]);
        dz[u] = fmaf((float)b[u + 4], z1[u], dz[u]);
      }
    }
    den += (dz[0] + dz[1]) + (dz[2] + dz[3]);
    den += other_half(den);
    const f32x16 num = (nacc[0] + nacc[1]) + (nacc[2] + nacc[3]);
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
  lds_barrier();
  if (tid < DK) sm.z[tid] += (sm.zc[tid] + sm.zc[DK + tid]) + (sm.zc[2 * DK + tid] + sm.zc[3 * DK + tid]);
  lds_barrier();
}

// Exclusive prefix of the segment states of one (b, h) (blockIdx.y): slot s
// of `pre` receives the state entering segment s, combined from the own states
// of segments 0 .. s-1 in `own`, each relative to its own shift.  One thread
// per state entry: S[j][*] carries row shift c_j, z needs none, c is the max.
__global__ __launch_bounds__(NTH) void prefix_kernel(const float* __restrict__ own,
                                                     float* __restrict__ pre, int nseg) {
  const int e = blockIdx.x * NTH + threadIdx.x;
  if (e >= STATE) return;
  const size_t base = (size_t)blockIdx.y * nseg * STATE;
  const float* ob = own + base;
  float* pb = pre + base;
  const int j = e < DV * DK ? e / DK : (e >= DV * DK + DK ? e - DV * DK - DK : -1);
  float acc = 0.f, C = -INFINITY;
  for (int sg = 0; sg + 1 < nseg; ++sg) {
    const float val = ob[(size_t)sg * STATE + e];
    if (e < DV * DK) {
      const float cs = ob[(size_t)sg * STATE + DV * DK + DK + j];
      const float Cn = fmaxf(C, cs);
      acc = acc * exp2_hw(C - Cn) + val * exp2_hw(cs - Cn);
      C = Cn;
    } else if (e < DV * DK + DK) {
      acc += val;
    } else {
      acc = fmaxf(C, val);
      C = acc;
    }
    pb[(size_t)(sg + 1) * STATE + e] = acc;
  }
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
  float* wsh = ws + (size_t)bh * nseg * STATE;  // own states; entering states follow gridDim.x slots on
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

  const int tbeg = seg * SEG;
  const int tend = min(tbeg + SEG, T);
  ChunkRegs cr;
  fetch_chunk<OUT>(cr, Qh, Kh, Vh, tbeg, T);

  if (OUT && seg > 0) {
    // entering state, left by the prefix kernel in the second half of ws
    const float* S = wsh + (size_t)gridDim.x * STATE + (size_t)seg * STATE;
    if (tid < DK) sm.z[tid] = S[DV * DK + tid];
    if (tid < DV) sm.c[tid] = S[DV * DK + DK + tid];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int row = dvb * 32 + (i >> 2) * 8 + hl * 4 + (i & 3);
      const int col = sub * 32 + (lane & 31);
      st[i] = S[row * DK + col];
    }
    __syncthreads();
  }

  for (int t0 = tbeg; t0 < tend; t0 += CH)
    scan_chunk<OUT>(sm, st, cr, Qh, Kh, Vh, Oh, t0, t0 + CH < tend ? t0 + CH : T, T);

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
  // own segment states, then the entering (prefix) states
  const size_t bytes = 2 * (size_t)nbh * nseg * STATE * sizeof(float);
  hipError_t e = workspace_alloc(reinterpret_cast<void**>(&ws), bytes, stream);
  if (e != hipSuccess) return e;
  if (nseg > 1) {
    hipLaunchKernelGGL(linear_kernel<false>, dim3((unsigned)(nbh * nseg)), dim3(NTH), 0, stream,
                       reinterpret_cast<const bf16*>(Q), reinterpret_cast<const bf16*>(K),
                       reinterpret_cast<const bf16*>(V), beta, out, ws, H, T, nseg);
    e = hipGetLastError();
    if (e == hipSuccess) {
      hipLaunchKernelGGL(prefix_kernel, dim3((unsigned)((STATE + NTH - 1) / NTH), (unsigned)nbh),
                         dim3(NTH), 0, stream, ws, ws + (size_t)nbh * nseg * STATE, nseg);
      e = hipGetLastError();
    }
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
