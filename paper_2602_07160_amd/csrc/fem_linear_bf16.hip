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
// Chunking: 64-token chunks inside segments of segc chunks, segc chosen at
// launch so that the (b, h, segment) workgroups fill the device once.
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
// same rounded A.  E is formed in registers by the waves that use it (no LDS
// round trip).  An output whose numerator underflowed is recomputed exactly
// by the wave.

#include "fem_device.h"
#include "fem_internal.h"

#include <mutex>

namespace fem {
namespace {

constexpr int DK = 64, DV = 64;  // supported widths
constexpr int CH = 64;           // tokens per chunk
constexpr int WG_PER_CU = 2;     // resident workgroups per CU (VGPR budget)
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
  // V^T [d_v][key, MFMA order] while the waves form E; then S^T hi [d_v][d_k]
  bf16 vt_sh[DV * ROW];
  bf16 sl[DV * SROW];   // S^T lo
  float c[DV];          // running shift (published for the epilogue)
  float bl[DV];         // beta log2 e
  float inv[DV];
  float z[DK];          // sum of phi(k) over earlier chunks
  float zc[4 * DK];     // partial sums of phi(k) over this chunk (four row quarters)
};
static_assert(ROW == SROW, "S^T hi shares the V^T rows");

// Key r of a chunk -> position inside an MFMA-ordered row (see the softmax
// kernel: the B operand taken from a transposed accumulator holds keys
// {4h..4h+3, 8+4h..8+4h+3} of each 16-key group in lane half h).
__device__ __forceinline__ int e_pos(int r) {
  const int g = r & 15;
  return (r & ~15) + (((g >> 2) & 1) << 3) + (((g >> 3) & 1) << 2) + (g & 3);
}

// phi(K)^T and V^T rows are written one bf16 at a time down a column of
// eight rows per lane group; the 16-byte chunk of a row is XORed with the
// row's group of eight so that those writes spread over the banks.  Readers
// of 16-byte MFMA fragments apply the same map.
__device__ __forceinline__ int tpos(int row, int pos) {
  return row * ROW + ((((pos >> 3) ^ (row >> 3)) & 7) << 3) + (pos & 7);
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

// Buffer resource over `bytes` bytes from `base` (raw, untyped): a load at
// or past the end returns zero.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* base, unsigned bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                           0x00020000);
}

__device__ __forceinline__ bf16x8 load16(__amdgpu_buffer_rsrc_t r, unsigned off) {
  return __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0));
}

// Rows past T come back as zeros (the resource ends at row T).
template <bool OUT>
__device__ __forceinline__ void fetch_chunk(ChunkRegs& cr, const bf16* Qh, const bf16* Kh,
                                            const bf16* Vh, int t0, int T) {
  const int tid = threadIdx.x;
  const unsigned rows = (unsigned)min(CH, T - t0);
  const __amdgpu_buffer_rsrc_t rk = rsrc(Kh + (size_t)t0 * DK, rows * DK * 2u);
  const __amdgpu_buffer_rsrc_t rv = rsrc(Vh + (size_t)t0 * DV, rows * DV * 2u);
  const __amdgpu_buffer_rsrc_t rq = rsrc(Qh + (size_t)t0 * DK, rows * DK * 2u);
#pragma unroll
  for (int i = 0; i < SLOTS; ++i) {
    const int e = tid + NTH * i, r = e >> 3, c8 = (e & 7) * 8;
    cr.k[i] = load16(rk, (unsigned)(r * DK + c8) * 2u);
    cr.v[i] = load16(rv, (unsigned)(r * DV + c8) * 2u);
    if (OUT) cr.q[i] = load16(rq, (unsigned)(r * DK + c8) * 2u);
  }
}

// One chunk of the scan.  Stages tokens [t0, t0 + CH) from cr (rows past T
// are zero and masked), starts fetching the next chunk into cr, forms the
// tilt, rescales the state, produces outputs (OUT) and updates S.
// Wave w owns channel block dvb = w >> 1 and sub = w & 1: S^T block
// (dvb, d_k block sub) and output block (dvb, query block sub).
//
// The tilt E^T (32 channels x 64 keys of the wave's block) is formed in
// registers as the MFMA A operand: lane (n, hl) holds channel dvb*32 + n and
// the keys at MFMA positions ks*16 + hl*8 .. +8 of each k-step ks, read from
// V^T staged in the same key order.  The two waves of a channel block form
// the same E; each lane keeps the running shift cj of its channel.
template <bool OUT>
__device__ __forceinline__ void scan_chunk(LinSmem& sm, f32x16& st, float& cj, float blj,
                                           ChunkRegs& cr, const bf16* Qh, const bf16* Kh,
                                           const bf16* Vh, float* Oh, int t0, int tnext, int T) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n = lane & 31, hl = lane >> 5;
  const int dvb = wave >> 1, sub = wave & 1;
  const int ch = dvb * 32 + n;

  // ---- stage phi(Q), phi(K), phi(K)^T and V^T; phi in fp32, rounded to bf16
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
      sm.fkt[tpos(c8 + u, e_pos(r))] = pk[u];
      sm.vt_sh[tpos(c8 + u, e_pos(r))] = cr.v[i][u];
    }
    *reinterpret_cast<bf16x8*>(sm.fk + r * ROW + c8) = pk;
    if (OUT) *reinterpret_cast<bf16x8*>(sm.fq + r * ROW + c8) = pq;
  }
  // the next chunk's loads run while this one is processed
  if (tnext < T) fetch_chunk<OUT>(cr, Qh, Kh, Vh, tnext, T);
  lds_barrier();

  // ---- tilt of the wave's channel block, in registers
  bf16x8 eh[4], el[4];
  float gj;
  bool rose;
  {
    bf16x8 vr[4];
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
      vr[ks] = *reinterpret_cast<const bf16x8*>(sm.vt_sh + tpos(ch, ks * 16 + hl * 8));
    // keys at or past T (last chunk only) stay out of the max and give E = 0
    const bool full = t0 + CH <= T;
    float vmax = -INFINITY;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (full || t0 + e_pos(ks * 16 + hl * 8 + u) < T) vmax = fmaxf(vmax, (float)vr[ks][u]);
    }
    vmax = fmaxf(vmax, other_half(vmax));  // lanes n and n + 32 hold the same channel
    const float mx = vmax * blj;
    const float cnew = (mx > cj + kColLag) ? mx : cj;
    const float sh = kBias - cnew;
    gj = exp2_hw(cj - cnew);
    rose = __any(cnew != cj);
    cj = cnew;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
#pragma unroll
      for (int u = 0; u < 8; u += 2) {
        float ev[2];
#pragma unroll
        for (int b = 0; b < 2; ++b) {
          const int key = e_pos(ks * 16 + hl * 8 + u + b);
          const float x = exp2_hw(fmaf((float)vr[ks][u + b], blj, sh));
          ev[b] = (full || t0 + key < T) ? x : 0.f;
        }
        const bf16x2 h2 = to_bf16x2(ev[0], ev[1]);
        const bf16x2 l2 = to_bf16x2(ev[0] - (float)h2[0], ev[1] - (float)h2[1]);
        eh[ks][u] = h2[0];
        eh[ks][u + 1] = h2[1];
        el[ks][u] = l2[0];
        el[ks][u + 1] = l2[1];
      }
    }
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

  // ---- rescale the state rows (d_v) when a shift of the block rose
  if (rose) {
#pragma unroll
    for (int i = 0; i < 16; ++i) st[i] *= __shfl(gj, (i >> 2) * 8 + hl * 4 + (i & 3));
  }
  if (OUT) {
    lds_barrier();  // every wave has read V^T before S^T hi replaces it
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int row = dvb * 32 + (i >> 2) * 8 + hl * 4 + (i & 3);
      const int col = sub * 32 + n;
      const bf16 hi = (bf16)st[i];
      sm.vt_sh[row * SROW + col] = hi;
      sm.sl[row * SROW + col] = (bf16)(st[i] - (float)hi);
    }
    if (sub == 0 && hl == 0) sm.c[ch] = cj;
    lds_barrier();

    // ---- outputs of query block qb = sub, channel block dvb
    const int qb = sub;
    const int tq = t0 + qb * 32 + n;
    // A^T blocks (keys kb x queries qb), kb <= qb; masked (key > query),
    // rounded to bf16, normaliser from the rounded values
    bf16x8 pf[4] = {};
    float den = 0.f;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      if (kb > qb) continue;
      f32x16 at = f32x16{};
#pragma unroll
      for (int ks = 0; ks < DK / 16; ++ks) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(sm.fk + (kb * 32 + n) * ROW + ks * 16 + hl * 8);
        const bf16x8 b = *reinterpret_cast<const bf16x8*>(sm.fq + (qb * 32 + n) * ROW + ks * 16 + hl * 8);
        at = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, at, 0, 0, 0);
      }
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        const int ks = kb * 2 + half, s0 = half * 8;
#pragma unroll
        for (int u = 0; u < 8; u += 2) {
          const int i0 = s0 + u, i1 = s0 + u + 1;
          const int key0 = kb * 32 + (i0 >> 2) * 8 + hl * 4 + (i0 & 3);
          const int key1 = kb * 32 + (i1 >> 2) * 8 + hl * 4 + (i1 & 3);
          const float a0 = (key0 <= qb * 32 + n) ? at[i0] : 0.f;
          const float a1 = (key1 <= qb * 32 + n) ? at[i1] : 0.f;
          const bf16x2 p2 = to_bf16x2(a0, a1);
          pf[ks][u] = p2[0];
          pf[ks][u + 1] = p2[1];
          den = add_bf16x2(p2, den);
        }
      }
    }
    // numerator: E^T A^T (intra) + S^T phi(Q)^T (inter); the inter-chunk
    // normaliser phi(q)^T z (this lane's half of d_k) reuses the phi(Q)
    // fragments, with four partial sums
    f32x16 num = f32x16{};
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      if ((ks >> 1) > qb) continue;
      num = __builtin_amdgcn_mfma_f32_32x32x16_bf16(eh[ks], pf[ks], num, 0, 0, 0);
      num = __builtin_amdgcn_mfma_f32_32x32x16_bf16(el[ks], pf[ks], num, 0, 0, 0);
    }
    const int soff = (dvb * 32 + n) * SROW + hl * 8;
    float dz[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < DK / 16; ++ks) {
      const bf16x8 ah = *reinterpret_cast<const bf16x8*>(sm.vt_sh + soff + ks * 16);
      const bf16x8 al = *reinterpret_cast<const bf16x8*>(sm.sl + soff + ks * 16);
      const bf16x8 b = *reinterpret_cast<const bf16x8*>(sm.fq + (qb * 32 + n) * ROW + ks * 16 + hl * 8);
      num = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, b, num, 0, 0, 0);
      num = __builtin_amdgcn_mfma_f32_32x32x16_bf16(al, b, num, 0, 0, 0);
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
    // epilogue
    int ed;
    const float fd = log2_hw(frexpf(den, &ed));
    uint32_t flags = 0;
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) {
      const int ch0 = dvb * 32 + g4 * 8 + hl * 4;
      const f32x4 cc = *reinterpret_cast<const f32x4*>(sm.c + ch0);
      const f32x4 iv = *reinterpret_cast<const f32x4*>(sm.inv + ch0);
      f32x4 o;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float a = num[g4 * 4 + e];
        int ea;
        const float fa = log2_hw(frexpf(a, &ea));
        o[e] = ((float)(ea - ed - (int)kBias) + (fa - fd) + cc[e]) * iv[e];
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
      const int ch2 = dvb * 32 + (e >> 2) * 8 + (src >> 5) * 4 + (e & 3);
      const float o = exact_read_linear(Qh, Kh, Vh, t, ch2, sm.bl[ch2]);
      if (lane == src) {
        flags &= ~(1u << e);
        Oh[(size_t)t * DV + ch2] = o;
      }
    }
  }

  // ---- state update S^T(dvb, dkb = sub) += E^T phi(K)   (keys of this chunk)
  {
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const bf16x8 b =
          *reinterpret_cast<const bf16x8*>(sm.fkt + tpos(sub * 32 + n, ks * 16 + hl * 8));
      st = __builtin_amdgcn_mfma_f32_32x32x16_bf16(eh[ks], b, st, 0, 0, 0);
      st = __builtin_amdgcn_mfma_f32_32x32x16_bf16(el[ks], b, st, 0, 0, 0);
    }
  }
  // every read of this chunk's LDS tiles and of z is done before the next
  // chunk stages and before z moves on
  lds_barrier();
  if (tid < DK) sm.z[tid] += (sm.zc[tid] + sm.zc[DK + tid]) + (sm.zc[2 * DK + tid] + sm.zc[3 * DK + tid]);
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
                                                     int nseg, int segc) {
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
  const int ch = dvb * 32 + (lane & 31);  // this lane's tilt channel

  if (tid < DV) {
    const float bl = beta[h * DV + tid] * kLog2e;
    sm.bl[tid] = bl;
    sm.inv[tid] = 1.f / bl;
  }
  if (tid < DK) sm.z[tid] = 0.f;
  f32x16 st = f32x16{};
  const float blj = beta[h * DV + ch] * kLog2e;
  float cj = -INFINITY;  // running shift of channel ch
  __syncthreads();

  const int tbeg = seg * segc * CH;
  const int tend = min(tbeg + segc * CH, T);
  ChunkRegs cr;
  fetch_chunk<OUT>(cr, Qh, Kh, Vh, tbeg, T);

  if (OUT && seg > 0) {
    // entering state, left by the prefix kernel in the second half of ws
    const float* S = wsh + (size_t)gridDim.x * STATE + (size_t)seg * STATE;
    if (tid < DK) sm.z[tid] = S[DV * DK + tid];
    cj = S[DV * DK + DK + ch];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int row = dvb * 32 + (i >> 2) * 8 + hl * 4 + (i & 3);
      const int col = sub * 32 + (lane & 31);
      st[i] = S[row * DK + col];
    }
    __syncthreads();
  }

  for (int t0 = tbeg; t0 < tend; t0 += CH)
    scan_chunk<OUT>(sm, st, cj, blj, cr, Qh, Kh, Vh, Oh, t0, t0 + CH < tend ? t0 + CH : T, T);

  if (!OUT) {
    float* S = wsh + (size_t)seg * STATE;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int row = dvb * 32 + (i >> 2) * 8 + hl * 4 + (i & 3);
      const int col = sub * 32 + (lane & 31);
      S[row * DK + col] = st[i];
    }
    __syncthreads();  // the last z update
    if (tid < DK) S[DV * DK + tid] = sm.z[tid];
    if (sub == 0 && hl == 0) S[DV * DK + DK + ch] = cj;
  }
}

}  // namespace

hipError_t launch_linear_bf16(const void* Q, const void* K, const void* V, const float* beta,
                              float* out, int B, int H, int T, int dk, int dv, int chunk,
                              hipStream_t stream) {
  if (dk != DK || dv != DV || chunk != CH) return hipErrorNotSupported;
  const int nbh = B * H;
  // Segments: the scan is sequential inside one, so the fewest chunks per
  // segment that still let every workgroup be resident at once.
  const int nchunk = (T + CH - 1) / CH;
  const int slots = device_cus() * WG_PER_CU;
  const int want = max(1, slots / nbh);
  const int segc = (nchunk + want - 1) / want;
  const int nseg = (nchunk + segc - 1) / segc;
  float* ws = nullptr;
  // own segment states, then the entering (prefix) states
  const size_t bytes = 2 * (size_t)nbh * nseg * STATE * sizeof(float);
  hipError_t e = workspace_alloc(reinterpret_cast<void**>(&ws), bytes, stream);
  if (e != hipSuccess) return e;
  if (nseg > 1) {
    hipLaunchKernelGGL(linear_kernel<false>, dim3((unsigned)(nbh * nseg)), dim3(NTH), 0, stream,
                       reinterpret_cast<const bf16*>(Q), reinterpret_cast<const bf16*>(K),
                       reinterpret_cast<const bf16*>(V), beta, out, ws, H, T, nseg, segc);
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
                       reinterpret_cast<const bf16*>(V), beta, out, ws, H, T, nseg, segc);
    e = hipGetLastError();
  }
  const hipError_t f = workspace_free(ws, stream);
  return e != hipSuccess ? e : f;
}

}  // namespace fem
