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
// GLA prior (Appendix "Gated Linear Attention (GLA) Prior"): the same scan
// with features q~ = ReLU(RoPE(q)) + eps, k~ likewise, and a decay envelope
// per key channel c: p_t(i) propto sum_c q~_tc k~_ic exp(G_tc - G_ic), G the
// running sum of the log-decays g, which must lie in [-2, 0].  Inside a chunk, with
// B the chunk-local running sum and R = B at its middle row:
//   intra:  A_ti = sum_c (q~_tc e^{B_tc - R_c}) (k~_ic e^{R_c - B_ic})
//   inter:  num_t += sum_c (q~_tc e^{B_tc - R_c}) (e^{R_c} S_c)
//   update: S_c <- e^{B_last,c} S_c + sum_i k~_ic e^{B_last,c - B_ic} [E_i | 1]
// Every factor stays within e^{+-64} because a chunk has 64 rows and g >= -2.
// The segment prefix carries each segment's total log-decay.
//
// All products run on v_mfma_f32_32x32x16_bf16 in transposed form (outputs
// are [channel][token]); E and S enter as bf16 hi + lo pairs, the masked
// intra-chunk scores A enter as bf16 and the normaliser is summed from the
// same rounded A.  E is formed in registers by the waves that use it (no LDS
// round trip).  An output whose numerator underflowed is recomputed exactly
// by the wave.

#include "fem_device.h"
#include "fem_internal.h"


namespace fem {
namespace {

constexpr int DK = 64, DV = 64;  // supported widths
constexpr int GCH = 64;          // tokens per chunk of the GLA prior
constexpr int NTH = 256;         // 4 waves
constexpr int ROW = 64 + 8;      // padded bf16 row (64 values + 16 B)
// State snapshot S [d_k][d_v] in LDS (bf16): a row is 16 eight-byte chunks of
// 4 channels, chunk k of row r stored at position k ^ snap_swz(r), so that
// 16 consecutive rows written at one chunk, and 4 consecutive rows read at 4
// consecutive chunks, each meet every bank once.
constexpr int SROW = DV;
static_assert(DV == 64, "16 chunks per snapshot row");
__host__ __device__ constexpr int snap_swz(int r) { return ((r & 3) << 2) | ((r >> 2) & 3); }
__device__ __forceinline__ int snap_off(int r, int j) {  // j a multiple of 4
  return r * SROW + ((((j >> 2) ^ snap_swz(r))) << 2);
}
constexpr int OBR = 32 + 4;      // padded row of a staged output block (floats)
constexpr int STATE = DV * DK + DK + DV;  // floats per saved segment state
constexpr int kElu = 0, kGla = 1;         // the prior
// GLA adds the segment's total log-decay per key channel
template <int PRIOR>
constexpr int state_floats() { return PRIOR == kGla ? STATE + DK : STATE; }

constexpr float kGlaEps = 1e-6f;   // the feature map's positive constant
// The log-decays' domain is [kGlaGMin, 0] (a precondition of the entry
// point: the paper's decays have g <= 0, and the floor keeps every factor of
// the 64-token chunk form within e^+-64).  Values outside it are clamped into
// it, which only keeps the arithmetic finite: the read is then not the
// paper's for those inputs.
constexpr float kGlaGMin = -2.f;

// RoPE frequencies in revolutions per position, f_m = 10000^(-2m/DK) / (2 pi),
// as float hi + lo pairs of the double value (m = 0 .. DK/2 - 1), so that the
// angle of position t reduces modulo one revolution almost exactly.
constexpr double cexp_neg(double x) {  // e^x for -10 <= x <= 0
  double y = x / 1024.0, term = 1.0, sum = 1.0;
  for (int n = 1; n < 24; ++n) {
    term *= y / n;
    sum += term;
  }
  for (int i = 0; i < 10; ++i) sum *= sum;
  return sum;
}
struct RopeTab {
  float hi[DK / 2], lo[DK / 2];
};
constexpr RopeTab make_rope_tab() {
  RopeTab t{};
  for (int m = 0; m < DK / 2; ++m) {
    const double f = cexp_neg(-2.0 * m / DK * 9.210340371976184) / 6.283185307179586;
    t.hi[m] = (float)f;
    t.lo[m] = (float)(f - (double)t.hi[m]);
  }
  return t;
}
__constant__ RopeTab kRope = make_rope_tab();

constexpr float kBias = 64.f;
constexpr float kColLag = 16.f;
constexpr float kUnderflow = 0x1p-64f;

typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4;

// One tile of CH tokens; NSUB sub-chunks of CH / NSUB tokens per tile.  The
// state enters the outputs of sub-chunk s as it stood at the start of s.
template <int CH, int NSUB>
struct LinSmem {
  bf16 fq[CH * ROW];          // phi(Q) [token][d_k]
  bf16 fk[CH * DK];           // phi(K) [key][d_k], swizzled; phi(K)^T comes from transposing reads
  bf16 vs[CH * DV];           // V [key][d_v], swizzled; V^T comes from transposing reads
  bf16 sh[NSUB][DK * SROW];   // S hi [d_k][d_v] at the start of each sub-chunk
  bf16 sl[NSUB][DK * SROW];   // S lo
  float ci[DV];               // (c - kBias) / (beta log2 e): the running shift as the epilogue adds it
  float bl[DV];               // beta log2 e
  float inv[DV];
  float z[DK];                // sum of phi(k) over earlier tiles
  // the vector whose product with phi(q) is the inter-chunk normaliser (z,
  // or e^R z for GLA) as bf16 hi + lo: the A operand (all rows equal) of
  // the matrix-core row sums that form the normaliser
  bf16 zh[DK], zl[DK];
  float zc[4 * DK];           // partial sums of phi(k) over this tile (four row quarters)
};

// GLA: chunk-local running log-decay B[token][d_k] (fp32), its quarter
// totals, and e^{R} z for the inter-chunk normaliser.
struct GlaSmem {
  float b[GCH * DK];
  float bq[4 * DK];
  float zr[DK];
  bf16 fk2[GCH * DK];  // k~ e^{B_last - B} [key][d_k], swizzled (the state update's operand)
};
template <int PRIOR, int CH, int NSUB>
struct ScanSmem : LinSmem<CH, NSUB> {
  // E fragments passed between the two waves of a channel block (linear
  // prior, one chunk per tile of at most 64 tokens): [block][k-step][hi, lo][lane]
  static constexpr bool SPLIT_E = NSUB == 1 && CH <= 64;
  bf16x8 ex[SPLIT_E ? (DV / 32) * (CH / 16) * 2 * 64 : 1];
  // tiles of at most 64 tokens: each wave's 32 x 32 block of outputs, rows
  // padded to OBR floats, so that the stores leave in whole 128-byte rows
  static constexpr bool STAGE_OUT = CH <= 64;
  __align__(16) float ob[STAGE_OUT ? 4 * 32 * OBR : 1];
  __device__ float* gb() { return nullptr; }
  __device__ float* gbq() { return nullptr; }
  __device__ float* gzr() { return nullptr; }
  __device__ bf16* fku() { return this->fk; }  // the state update's key features
};
template <>
struct ScanSmem<kGla, GCH, 1> : LinSmem<GCH, 1> {
  // (with the exchange buffer the state pass would lose its second
  // workgroup per CU; splitting the read's tilt alone measured slower)
  static constexpr bool SPLIT_E = false;
  bf16x8 ex[1];
  static constexpr bool STAGE_OUT = false;
  GlaSmem gla;
  __device__ float* gb() { return gla.b; }
  __device__ float* gbq() { return gla.bq; }
  __device__ float* gzr() { return gla.zr; }
  __device__ bf16* fku() { return gla.fk2; }
};

// Entry i of the inter-chunk normaliser vector, as bf16 hi + lo.
template <int CH, int NSUB>
__device__ __forceinline__ void put_zn(LinSmem<CH, NSUB>& sm, int i, float v) {
  const bf16 hi = (bf16)v;
  sm.zh[i] = hi;
  sm.zl[i] = (bf16)(v - (float)hi);
}

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

// MFMA A fragments A[m][k] = S[k0 + k][j0 + m] (m < 32, k < 16) of a state
// snapshot S [d_k][d_v] (layout at snap_off): two transposing reads, rows in
// natural order.  In each 16-lane group g, lane i gives the address of 4
// columns (j0 + 16 (g & 1) + 4 (i & 3) ...) of row k0 + 8 (g >> 1) + i / 4
// (then 4 rows further down) and receives column j0 + 16 (g & 1) + i of the
// 4 rows: lane m + 32 hl holds A[m][8 hl + u], the A layout of
// v_mfma_f32_32x32x16_bf16.  With k0 a multiple of 16 the swizzle does not
// depend on k0, so the lane's two offsets are formed once (SnapFrag) and k0
// is a constant displacement.
struct SnapFrag {
  int lo, hi;  // element offsets of the lane's two reads at k0 = 0
  __device__ __forceinline__ explicit SnapFrag(int j0) {
    const int lane = threadIdx.x & 63, g = lane >> 4, i = lane & 15;
    const int row = 8 * (g >> 1) + (i >> 2);
    const int col = j0 + 16 * (g & 1) + 4 * (i & 3);
    lo = snap_off(row, col);
    hi = snap_off(row + 4, col);
  }
  // k0: a multiple of 16 (the swizzle repeats every 16 rows)
  __device__ __forceinline__ bf16x8 read(const bf16* t, int k0) const {
    typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
    const bf16* b = t + k0 * SROW;
    const s16x4 l = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(b + lo));
    const s16x4 h = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(b + hi));
    typedef short s16x8 __attribute__((ext_vector_type(8)));
    const s16x8 x = {l[0], l[1], l[2], l[3], h[0], h[1], h[2], h[3]};
    return __builtin_bit_cast(bf16x8, x);
  }
};

// elu(x) + 1 = max(e^min(x, 0), x + 1), without a select: 2^y is increasing
// with 2^0 = 1, so e^min(x, 0) is 2^(x log2 e) clamped to [0, 1] (the clamp
// bit of the exponential instruction), and e^x >= x + 1 for every x.
__device__ __forceinline__ float phi(float x) {
  const float e = __builtin_amdgcn_fmed3f(exp2_hw(x * kLog2e), 0.f, 1.f);
  return fmaxf(e, x + 1.f);
}

// RoPE of the pair (x0, x1) = dims (2m, 2m+1) at position t, then ReLU + eps.
__device__ __forceinline__ void gla_pair(float& x0, float& x1, int m, int t) {
  const float tf = (float)t;
  const float p = tf * kRope.hi[m];
  const float e = fmaf(tf, kRope.hi[m], -p);  // exact rounding error of p
  float r = (p - floorf(p)) + (e + tf * kRope.lo[m]);
  r -= floorf(r);
  const float c = __builtin_amdgcn_cosf(r), s = __builtin_amdgcn_sinf(r);  // revolutions
  const float y0 = x0 * c - x1 * s, y1 = x0 * s + x1 * c;
  x0 = fmaxf(y0, 0.f) + kGlaEps;
  x1 = fmaxf(y1, 0.f) + kGlaEps;
}

__device__ __forceinline__ float clip_g(float g) { return fminf(fmaxf(g, kGlaGMin), 0.f); }

// Exact fp32 read of one (t, j) of the GLA prior by the whole wave: lane c
// holds key channel c (d_k = 64), the keys are walked from t down to 0 with
// each lane's decay exp(sum_{tau=i+1}^{t} g_tau,c) kept as a running product.
__device__ float exact_read_gla(const bf16* __restrict__ Qh, const bf16* __restrict__ Kh,
                                const bf16* __restrict__ Vh, const float* __restrict__ Gh,
                                int t, int j, float bl) {
  static_assert(DK == 64, "one lane per key channel");
  constexpr int U = 8;  // keys whose loads are in flight together
  const int c = threadIdx.x & 63;
  float q0 = (float)Qh[(size_t)t * DK + (c & ~1)], q1 = (float)Qh[(size_t)t * DK + (c | 1)];
  gla_pair(q0, q1, c >> 1, t);
  const float qc = (c & 1) ? q1 : q0;
  Lse2 num, den;
  float dec = 1.f;
  for (int i0 = t; i0 >= 0; i0 -= U) {
    float k0[U], k1[U], gg[U], vv[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i = max(i0 - u, 0);
      k0[u] = (float)Kh[(size_t)i * DK + (c & ~1)];
      k1[u] = (float)Kh[(size_t)i * DK + (c | 1)];
      gg[u] = Gh[(size_t)i * DK + c];
      vv[u] = (float)Vh[(size_t)i * DV + j];
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i = i0 - u;
      if (i < 0) break;
      gla_pair(k0[u], k1[u], c >> 1, i);
      const float a = wave_sum(qc * ((c & 1) ? k1[u] : k0[u]) * dec);
      if (a > 0.f) {
        const float w = log2_hw(a);
        den.add(w);
        num.add(w + vv[u] * bl);
      }
      dec *= exp2_hw(clip_g(gg[u]) * kLog2e);
    }
  }
  // every lane holds the same (num, den)
  return (num.m + log2_hw(num.s) - (den.m + log2_hw(den.s))) / bl;
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

// Raw Q, K, V of one tile held in registers: thread tid covers the 16-byte
// slots e = tid + NTH*i (row e >> 3, columns (e & 7)*8 ..).
template <int CH>
struct ChunkRegs {
  static constexpr int SLOTS = CH * 8 / NTH;
  bf16x8 q[SLOTS], k[SLOTS], v[SLOTS];
  f32x4 g[SLOTS][2];  // GLA log-decays of the slot's 8 channels
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
__device__ __forceinline__ f32x4 load16f(__amdgpu_buffer_rsrc_t r, unsigned off) {
  return __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0));
}

template <int PRIOR, bool OUT, int CH>
__device__ __forceinline__ void fetch_chunk(ChunkRegs<CH>& cr, const bf16* Qh, const bf16* Kh,
                                            const bf16* Vh, const float* Gh, int t0, int T) {
  constexpr int SLOTS = ChunkRegs<CH>::SLOTS;
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
  if (PRIOR == kGla) {
    const __amdgpu_buffer_rsrc_t rg = rsrc(Gh + (size_t)t0 * DK, rows * DK * 4u);
#pragma unroll
    for (int i = 0; i < SLOTS; ++i) {
      const int e = tid + NTH * i, r = e >> 3, c8 = (e & 7) * 8;
      cr.g[i][0] = load16f(rg, (unsigned)(r * DK + c8) * 4u);
      cr.g[i][1] = load16f(rg, (unsigned)(r * DK + c8 + 4) * 4u);
    }
  }
}

// One tile of the scan.  Stages tokens [t0, t0 + CH) from cr (rows past T
// are zero and masked), starts fetching the next tile into cr, forms the
// tilt, rescales the state, produces outputs (OUT) and updates S.
// Wave w owns channel block dvb = w >> 1 and sub = w & 1: S^T block
// (dvb, d_k block sub) and the outputs of channel block dvb for the query
// blocks qb = sub, sub + 2, ... of the tile.
//
// The chunk of the scan is CH / NSUB tokens: a query sees the keys of its
// own chunk through the masked intra-chunk product A and every earlier key
// through the state.  With NSUB = 2 (16-token chunks in a 32-token tile) the
// state also advances by the first chunk's keys before the second chunk's
// outputs, which read it as a second snapshot.
//
// The tilt E^T (32 channels x CH keys of the wave's block) is formed in
// registers as the MFMA A operand: lane (n, hl) holds channel dvb*32 + n and
// the keys at MFMA positions ks*16 + hl*8 .. +8 of each k-step ks, read from
// V^T staged in the same key order.  Each lane keeps the running shift cj
// of its channel; the two waves of a channel block compute the same shift
// and, for the linear prior with one chunk per tile of at most 64 tokens,
// form the E of half the k-steps each (the halves meet in LDS); otherwise
// both form all of it.  FIXED: the shift is the segment's own, set before
// the first tile (every value of the segment lies at most kColLag above it),
// so no tile raises it and only the wave's own k-steps of V^T are read.
template <int PRIOR, bool OUT, int CH, int NSUB, bool FIXED>
__device__ __forceinline__ void scan_chunk(ScanSmem<PRIOR, CH, NSUB>& sm, f32x16& st, float& cj,
                                           float blj, float& ldc, ChunkRegs<CH>& cr,
                                           const bf16* Qh, const bf16* Kh, const bf16* Vh,
                                           const float* Gh, float* Oh, int t0, int tnext, int T) {
  constexpr int SLOTS = ChunkRegs<CH>::SLOTS;
  constexpr int NKS = CH / 16;    // 16-key k-steps of the tile
  constexpr int NQB = CH / 32;    // 32-row query blocks of the tile
  constexpr int SUB = CH / NSUB;  // tokens per chunk
  static_assert(CH == 32 || CH == 64 || CH == 128, "tile length");
  static_assert(NSUB == 1 || (CH == 32 && NSUB == 2), "two 16-token chunks per 32-token tile");
  static_assert(PRIOR != kGla || (CH == GCH && NSUB == 1), "GLA: 64-token chunks");
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n = lane & 31, hl = lane >> 5;
  const int dvb = wave >> 1, sub = wave & 1;
  const int ch = dvb * 32 + n;

  if constexpr (PRIOR == kGla) {
    // ---- chunk-local running log-decay B down each key channel: clipped g
    // into LDS, prefix of each quarter of 16 rows, then the lower quarters'
    // totals added (rows past T hold g = 0 from the fetch)
#pragma unroll
    for (int i = 0; i < SLOTS; ++i) {
      const int e = tid + NTH * i, r = e >> 3, c8 = (e & 7) * 8;
      f32x4 g0, g1;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        g0[u] = clip_g(cr.g[i][0][u]);
        g1[u] = clip_g(cr.g[i][1][u]);
      }
      *reinterpret_cast<f32x4*>(sm.gb() + r * DK + c8) = g0;
      *reinterpret_cast<f32x4*>(sm.gb() + r * DK + c8 + 4) = g1;
    }
    lds_barrier();
    {
      const int c = tid & 63, q4 = tid >> 6;
      float run = 0.f;
#pragma unroll
      for (int r = 0; r < CH / 4; ++r) {
        run += sm.gb()[(q4 * (CH / 4) + r) * DK + c];
        sm.gb()[(q4 * (CH / 4) + r) * DK + c] = run;
      }
      sm.gbq()[q4 * DK + c] = run;
    }
    lds_barrier();
    {
      const int c = tid & 63, q4 = tid >> 6;
      float off = 0.f;
      for (int w = 0; w < q4; ++w) off += sm.gbq()[w * DK + c];
      if (q4 > 0) {
#pragma unroll
        for (int r = 0; r < CH / 4; ++r) sm.gb()[(q4 * (CH / 4) + r) * DK + c] += off;
      }
    }
    lds_barrier();
  }

  // ---- stage phi(Q), phi(K) and V, row-major; phi in fp32, rounded to bf16.
  // GLA: phi(Q) = q~ e^{B - R}, phi(K) = k~ e^{R - B}, and for the state
  // update k~ e^{B_last - B}.
  const auto stage = [&](auto partial) __attribute__((always_inline)) {
#pragma unroll
  for (int i = 0; i < SLOTS; ++i) {
    const int e = tid + NTH * i, r = e >> 3, c8 = (e & 7) * 8;
    // rows past T (a partial tile only): phi of the zeros fetched there,
    // times 0
    const float okf = !decltype(partial)::value || t0 + r < T ? 1.f : 0.f;
    bf16x8 pk, pq;
    if constexpr (PRIOR == kGla) {
      float kx[8], qx[8];
      bf16x8 pu;
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        kx[u] = (float)cr.k[i][u];
        qx[u] = OUT ? (float)cr.q[i][u] : 0.f;
      }
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        gla_pair(kx[2 * m], kx[2 * m + 1], c8 / 2 + m, t0 + r);
        if (OUT) gla_pair(qx[2 * m], qx[2 * m + 1], c8 / 2 + m, t0 + r);
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const float b = sm.gb()[r * DK + c8 + u];
        const float R = sm.gb()[(CH / 2 - 1) * DK + c8 + u];
        const float bl = sm.gb()[(CH - 1) * DK + c8 + u];
        if (OUT) {
          // k~ e^{B_last - B} = (k~ e^{R - B}) e^{B_last - R}, the second
          // factor per channel (the same for every slot of the thread)
          const float kr = kx[u] * exp2_hw((R - b) * kLog2e) * okf;
          pk[u] = (bf16)kr;
          pq[u] = (bf16)(qx[u] * exp2_hw((b - R) * kLog2e) * okf);
          pu[u] = (bf16)(kr * exp2_hw((bl - R) * kLog2e));
        } else {
          pu[u] = (bf16)(kx[u] * exp2_hw((bl - b) * kLog2e) * okf);
        }
      }
      *reinterpret_cast<bf16x8*>(reinterpret_cast<char*>(sm.fku()) + swz_off<DK>(r, c8 >> 3)) = pu;
    } else {
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        if constexpr (decltype(partial)::value) {
          pk[u] = (bf16)(phi((float)cr.k[i][u]) * okf);
          if (OUT) pq[u] = (bf16)(phi((float)cr.q[i][u]) * okf);
        } else {
          pk[u] = (bf16)phi((float)cr.k[i][u]);
          if (OUT) pq[u] = (bf16)phi((float)cr.q[i][u]);
        }
      }
    }
    // (the state pass of the GLA prior reads only k~ e^{B_last - B}, above)
    if (OUT || PRIOR != kGla)
      *reinterpret_cast<bf16x8*>(reinterpret_cast<char*>(sm.fk) + swz_off<DK>(r, c8 >> 3)) = pk;
    *reinterpret_cast<bf16x8*>(reinterpret_cast<char*>(sm.vs) + swz_off<DV>(r, c8 >> 3)) = cr.v[i];
    if (OUT) *reinterpret_cast<bf16x8*>(sm.fq + r * ROW + c8) = pq;
  }
  };
  if (t0 + CH <= T) stage(std::false_type());
  else stage(std::true_type());
  // the next tile's loads run while this one is processed
  if (tnext < T) fetch_chunk<PRIOR, OUT, CH>(cr, Qh, Kh, Vh, Gh, tnext, T);
  lds_barrier();

  // ---- tilt of the wave's channel block, in registers.  With one chunk per
  // tile of at most 64 tokens the two waves of a block split the k-steps:
  // each forms the E of its half and passes it to the other through LDS
  // (read back after the next barrier, see take_e).
  constexpr bool SPLIT_E = ScanSmem<PRIOR, CH, NSUB>::SPLIT_E;
  constexpr int KSH = SPLIT_E ? NKS / 2 : NKS;  // k-steps whose E this wave forms
  bf16x8 eh[NKS], el[NKS];
  float gj;
  bool rose;
  {
    // V^T fragments, this wave's half of the k-steps first (split: the
    // k-step of fragment f is ksof(f))
    const auto ksof = [&](int f) { return SPLIT_E ? (f + sub * KSH) % NKS : f; };
    constexpr int NVR = FIXED ? KSH : NKS;  // fragments read: FIXED needs no tile max
    bf16x8 vr[NVR];
#pragma unroll
    for (int f = 0; f < NVR; ++f) vr[f] = frag_tr<DV>(sm.vs, dvb * 32, ksof(f) * 16);
    // keys at or past T (a partial last tile only) stay out of the max and
    // give E = 0
    const auto tilt = [&](auto partial) __attribute__((always_inline)) {
    constexpr bool PART = decltype(partial)::value;
    if constexpr (FIXED) {
      gj = 1.f;
      rose = false;
    } else {
      float vmax = -INFINITY;
#pragma unroll
      for (int f = 0; f < NKS; ++f) {
#pragma unroll
        for (int u = 0; u < 8; ++u)
          if (!PART || t0 + e_pos(ksof(f) * 16 + hl * 8 + u) < T) vmax = fmaxf(vmax, (float)vr[f][u]);
      }
      vmax = fmaxf(vmax, other_half(vmax));  // lanes n and n + 32 hold the same channel
      const float mx = vmax * blj;
      const float cnew = (mx > cj + kColLag) ? mx : cj;
      gj = exp2_hw(cj - cnew);
      rose = __any(cnew != cj);
      cj = cnew;
    }
    const float sh = kBias - cj;
#pragma unroll
    for (int kk = 0; kk < KSH; ++kk) {
      const int ks = ksof(kk);
      const bf16x8 v = vr[kk];
#pragma unroll
      for (int u = 0; u < 8; u += 2) {
        float ev[2];
#pragma unroll
        for (int b = 0; b < 2; ++b) {
          const int key = e_pos(ks * 16 + hl * 8 + u + b);
          const float x = exp2_hw(fmaf((float)v[u + b], blj, sh));
          ev[b] = (!PART || t0 + key < T) ? x : 0.f;
        }
        const bf16x2 h2 = to_bf16x2(ev[0], ev[1]);
        const bf16x2 l2 = to_bf16x2(ev[0] - (float)h2[0], ev[1] - (float)h2[1]);
        eh[kk][u] = h2[0];
        eh[kk][u + 1] = h2[1];
        el[kk][u] = l2[0];
        el[kk][u + 1] = l2[1];
      }
      if constexpr (SPLIT_E) {
        sm.ex[((dvb * NKS + ks) * 2 + 0) * 64 + lane] = eh[kk];
        sm.ex[((dvb * NKS + ks) * 2 + 1) * 64 + lane] = el[kk];
      }
    }
    };
    if (t0 + CH <= T) tilt(std::false_type());
    else tilt(std::true_type());
  }
  // every k-step's E of the block, after a barrier that follows the stores
  auto take_e = [&]() {
    if constexpr (SPLIT_E) {
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) {
        eh[ks] = sm.ex[((dvb * NKS + ks) * 2 + 0) * 64 + lane];
        el[ks] = sm.ex[((dvb * NKS + ks) * 2 + 1) * 64 + lane];
      }
    }
  };
  // tile sum of phi(k): wave q4 takes a quarter of the rows, lane (pair cp,
  // half h) sums columns 2cp and 2cp + 1 over CH/8 of them with 4-byte reads;
  // the two halves meet by a lane swap, the four quarters in LDS
  {
    const int q4 = tid >> 6, cp = lane & 31, h = lane >> 5;
    float s0 = 0.f, s1 = 0.f;
#pragma unroll
    for (int r = 0; r < CH / 8; ++r) {
      const int row = q4 * (CH / 4) + h * (CH / 8) + r;
      const bf16x2 p = *reinterpret_cast<const bf16x2*>(
          reinterpret_cast<const char*>(sm.fku()) + swz_off<DK>(row, cp >> 2) + (cp & 3) * 4);
      s0 += (float)p[0];
      s1 += (float)p[1];
    }
    s0 += other_half(s0);
    s1 += other_half(s1);
    if (h == 0) {
      sm.zc[q4 * DK + 2 * cp] = s0;
      sm.zc[q4 * DK + 2 * cp + 1] = s1;
    }
    // GLA: the inter-chunk normaliser reads e^{R} z
    if (PRIOR == kGla && q4 == 0)
    {
      const int dkc = lane;
      const float zr = sm.z[dkc] * exp2_hw(sm.gb()[(CH / 2 - 1) * DK + dkc] * kLog2e);
      sm.gzr()[dkc] = zr;
      put_zn(sm, dkc, zr);
    }
  }

  // ---- rescale the state rows (d_v) when a shift of the block rose
  if (rose) {
#pragma unroll
    for (int i = 0; i < 16; ++i) st[i] *= __shfl(gj, (i >> 2) * 8 + hl * 4 + (i & 3));
  }
  // S^T(dvb, dkb = sub) += E^T phi(K) over the keys of k-steps [k0, k1)
  auto update = [&](int k0, int k1) {
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      if (ks < k0 || ks >= k1) continue;
      const bf16x8 b = frag_tr<DK>(sm.fku(), sub * 32, ks * 16);
      st = __builtin_amdgcn_mfma_f32_32x32x16_bf16(eh[ks], b, st, 0, 0, 0);
      st = __builtin_amdgcn_mfma_f32_32x32x16_bf16(el[ks], b, st, 0, 0, 0);
    }
  };
  // the state update of the first chunk's keys comes before the second
  // chunk's snapshot (NSUB = 2); the rest after the outputs
  constexpr int KS_EARLY = NSUB == 2 ? NKS / 2 : 0;
  if (OUT) {
    const float eR =
        PRIOR == kGla ? exp2_hw(sm.gb()[(CH / 2 - 1) * DK + sub * 32 + n] * kLog2e) : 1.f;
    // S^T (dvb, sub) into LDS as S [d_k][d_v] in bf16 hi + lo: entries
    // 4q..4q+3 of this lane are channels dvb*32 + 8q + 4hl + 0..3 of key dim
    // sub*32 + n, 8 contiguous bytes of a row
    auto snapshot = [&](int sn) {
      typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float sv[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) sv[r] = st[4 * q + r] * eR;
        const bf16x2 h01 = to_bf16x2(sv[0], sv[1]), h23 = to_bf16x2(sv[2], sv[3]);
        const bf16x2 l01 = to_bf16x2(sv[0] - (float)h01[0], sv[1] - (float)h01[1]);
        const bf16x2 l23 = to_bf16x2(sv[2] - (float)h23[0], sv[3] - (float)h23[1]);
        const int off = snap_off(sub * 32 + n, dvb * 32 + q * 8 + hl * 4);
        *reinterpret_cast<u32x2*>(sm.sh[sn] + off) =
            u32x2{__builtin_bit_cast(unsigned, h01), __builtin_bit_cast(unsigned, h23)};
        *reinterpret_cast<u32x2*>(sm.sl[sn] + off) =
            u32x2{__builtin_bit_cast(unsigned, l01), __builtin_bit_cast(unsigned, l23)};
      }
    };
    snapshot(0);
    if (NSUB == 2) {
      update(0, KS_EARLY);
      snapshot(1);
    }
    if (sub == 0 && hl == 0) sm.ci[ch] = (cj - kBias) * sm.inv[ch];
    lds_barrier();
    take_e();

    // ---- outputs of channel block dvb for the query blocks of this wave
#pragma unroll
    for (int qb = sub; qb < NQB; qb += 2) {
      const int qrow = qb * 32 + n;  // query row within the tile
      const int tq = t0 + qrow;
      const int qs = qrow / SUB;     // its chunk within the tile
      // A^T blocks (keys kb x queries qb), kb <= qb; masked to keys of the
      // query's own chunk at or before it, rounded to bf16, normaliser from
      // the rounded values
      bf16x8 pf[NKS];
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) pf[ks] = bf16x8{};
      // the normaliser: with one chunk per tile, on the matrix cores (every
      // row of dacc sums the rounded A^T over keys plus zn^T phi(q)); with
      // two, in the vector units (below)
      constexpr bool MDEN = NSUB == 1;
      float den = 0.f;
#pragma unroll
      for (int kb = 0; kb < NQB; ++kb) {
        if (kb > qb) continue;
        f32x16 at = f32x16{};
#pragma unroll
        for (int ks = 0; ks < DK / 16; ++ks) {
          const bf16x8 a = frag_rows<DK>(sm.fk, kb * 32 + n, 2 * ks + hl);
          const bf16x8 b = *reinterpret_cast<const bf16x8*>(sm.fq + qrow * ROW + ks * 16 + hl * 8);
          at = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, at, 0, 0, 0);
        }
        // only the diagonal block needs the mask (NSUB = 1: a block below
        // it holds earlier keys only)
        const auto round_block = [&](auto masked) __attribute__((always_inline)) {
#pragma unroll
          for (int half = 0; half < 2; ++half) {
            const int ks = kb * 2 + half, s0 = half * 8;
#pragma unroll
            for (int u = 0; u < 8; u += 2) {
              const int i0 = s0 + u, i1 = s0 + u + 1;
              const int key0 = kb * 32 + (i0 >> 2) * 8 + hl * 4 + (i0 & 3);
              const int key1 = kb * 32 + (i1 >> 2) * 8 + hl * 4 + (i1 & 3);
              bool in0 = true, in1 = true;
              if constexpr (decltype(masked)::value) {
                in0 = key0 <= qrow && (NSUB == 1 || key0 / SUB == qs);
                in1 = key1 <= qrow && (NSUB == 1 || key1 / SUB == qs);
              }
              const bf16x2 p2 = to_bf16x2(in0 ? at[i0] : 0.f, in1 ? at[i1] : 0.f);
              pf[ks][u] = p2[0];
              pf[ks][u + 1] = p2[1];
              if (!MDEN) den = add_bf16x2(p2, den);
            }
          }
        };
        if (NSUB == 1 && kb < qb) round_block(std::false_type());
        else round_block(std::true_type());
      }
      // numerator: E^T A^T (intra) + S^T phi(Q)^T (inter, the state at the
      // start of the query's chunk); the inter-chunk normaliser phi(q)^T z
      // (this lane's half of d_k) reuses the phi(Q) fragments, with four
      // partial sums
      f32x16 num = f32x16{}, dacc = f32x16{};
      bf16x8 ones;
#pragma unroll
      for (int u = 0; u < 8; ++u) ones[u] = (bf16)1.f;
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) {
        if ((ks >> 1) > qb) continue;
        num = __builtin_amdgcn_mfma_f32_32x32x16_bf16(eh[ks], pf[ks], num, 0, 0, 0);
        num = __builtin_amdgcn_mfma_f32_32x32x16_bf16(el[ks], pf[ks], num, 0, 0, 0);
        if (MDEN) dacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ones, pf[ks], dacc, 0, 0, 0);
      }
      float dz[4] = {0.f, 0.f, 0.f, 0.f};
      const SnapFrag sf(dvb * 32);
#pragma unroll
      for (int sn = 0; sn < NSUB; ++sn) {
        // NSUB = 2: snapshot sn feeds only the query columns of chunk sn
        const bool mine = NSUB == 1 || qs == sn;
#pragma unroll
        for (int ks = 0; ks < DK / 16; ++ks) {
          const bf16x8 ah = sf.read(sm.sh[sn], ks * 16);
          const bf16x8 al = sf.read(sm.sl[sn], ks * 16);
          bf16x8 b = *reinterpret_cast<const bf16x8*>(sm.fq + qrow * ROW + ks * 16 + hl * 8);
          if (!mine) b = bf16x8{};
          num = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, b, num, 0, 0, 0);
          num = __builtin_amdgcn_mfma_f32_32x32x16_bf16(al, b, num, 0, 0, 0);
          if (MDEN) {
            const bf16x8 zh = *reinterpret_cast<const bf16x8*>(sm.zh + ks * 16 + hl * 8);
            const bf16x8 zl = *reinterpret_cast<const bf16x8*>(sm.zl + ks * 16 + hl * 8);
            dacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(zh, b, dacc, 0, 0, 0);
            dacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(zl, b, dacc, 0, 0, 0);
            continue;
          }
          const float* zz = PRIOR == kGla ? sm.gzr() : sm.z;
          f32x4 z0 = *reinterpret_cast<const f32x4*>(zz + ks * 16 + hl * 8);
          f32x4 z1 = *reinterpret_cast<const f32x4*>(zz + ks * 16 + hl * 8 + 4);
          if (NSUB == 2 && sn == 1) {  // plus the first chunk's phi(k) (quarters 0, 1)
            z0 += *reinterpret_cast<const f32x4*>(sm.zc + ks * 16 + hl * 8) +
                  *reinterpret_cast<const f32x4*>(sm.zc + DK + ks * 16 + hl * 8);
            z1 += *reinterpret_cast<const f32x4*>(sm.zc + ks * 16 + hl * 8 + 4) +
                  *reinterpret_cast<const f32x4*>(sm.zc + DK + ks * 16 + hl * 8 + 4);
          }
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            dz[u] = fmaf((float)b[u], z0[u], dz[u]);
            dz[u] = fmaf((float)b[u + 4], z1[u], dz[u]);
          }
        }
      }
      if (MDEN) {
        den = dacc[0];
      } else {
        den += (dz[0] + dz[1]) + (dz[2] + dz[3]);
        den += other_half(den);
      }
      // epilogue: F = (log2(num / den) + c - kBias) / (beta log2 e), one
      // logarithm per output.  num / den is a weighted mean of E (at most
      // 2^(kColLag + kBias)); it is flagged below when it or num could have
      // lost precision (num < 2^-64, or num / den < 2^-100)
      const float rd = __builtin_amdgcn_rcpf(den);
      float amin = INFINITY;
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        const int ch0 = dvb * 32 + g4 * 8 + hl * 4;
        const f32x4 ci = *reinterpret_cast<const f32x4*>(sm.ci + ch0);
        const f32x4 iv = *reinterpret_cast<const f32x4*>(sm.inv + ch0);
        f32x4 o;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float a = num[g4 * 4 + e];
          o[e] = fmaf(log2_hw(a * rd), iv[e], ci[e]);
          amin = fminf(amin, a);
        }
        if constexpr (ScanSmem<PRIOR, CH, NSUB>::STAGE_OUT)
          *reinterpret_cast<f32x4*>(sm.ob + (wave * 32 + n) * OBR + g4 * 8 + hl * 4) = o;
        else if (tq < T)
          *reinterpret_cast<f32x4*>(Oh + (size_t)tq * DV + ch0) = o;
      }
      if constexpr (ScanSmem<PRIOR, CH, NSUB>::STAGE_OUT) {
        // the wave's block back by rows: 8 lanes cover the 32 channels of a row
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int r = i * 8 + (lane >> 3), c4 = (lane & 7) * 4;
          const f32x4 x = *reinterpret_cast<const f32x4*>(sm.ob + (wave * 32 + r) * OBR + c4);
          const int t = t0 + qb * 32 + r;
          if (t < T) *reinterpret_cast<f32x4*>(Oh + (size_t)t * DV + dvb * 32 + c4) = x;
        }
      }
      // outputs whose numerator underflowed (rare): recomputed exactly below
      uint32_t flags = 0;
      const auto low = [&](float a) { return !(a >= kUnderflow && a * rd >= 0x1p-100f); };
      if (__ballot(low(amin) && tq < T) != 0) {
#pragma unroll
        for (int i = 0; i < 16; ++i)
          if (low(num[i]) && tq < T) flags |= 1u << i;
        // the repaired values overwrite the stores above
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      }
      while (true) {
        const uint64_t who = __ballot(flags != 0);
        if (who == 0) break;
        const int src = __builtin_ctzll(who);
        const uint32_t fl = __builtin_amdgcn_readlane(flags, src);
        const int e = __builtin_ctz(fl);
        const int t = __builtin_amdgcn_readlane(tq, src);
        const int ch2 = dvb * 32 + (e >> 2) * 8 + (src >> 5) * 4 + (e & 3);
        const float o = PRIOR == kGla ? exact_read_gla(Qh, Kh, Vh, Gh, t, ch2, sm.bl[ch2])
                                      : exact_read_linear(Qh, Kh, Vh, t, ch2, sm.bl[ch2]);
        if (lane == src) {
          flags &= ~(1u << e);
          Oh[(size_t)t * DV + ch2] = o;
        }
      }
    }
  }

  // ---- state update S^T(dvb, dkb = sub) += E^T phi(K)   (keys of this tile);
  // GLA: the state first decays by e^{B_last} along its key channel (column)
  {
    if constexpr (PRIOR == kGla) {
      const float dcy = exp2_hw(sm.gb()[(CH - 1) * DK + sub * 32 + n] * kLog2e);
#pragma unroll
      for (int i = 0; i < 16; ++i) st[i] *= dcy;
    }
    if (!OUT && SPLIT_E) {
      lds_barrier();
      take_e();
    }
    update(OUT ? KS_EARLY : 0, NKS);
  }
  // every read of this tile's LDS tiles and of z is done before the next
  // tile stages and before z moves on
  // (B_last is read before the barrier: the next chunk overwrites B after it)
  const float blast = (PRIOR == kGla && tid < DK) ? sm.gb()[(CH - 1) * DK + tid] : 0.f;
  lds_barrier();
  if (tid < DK) {
    const float add = (sm.zc[tid] + sm.zc[DK + tid]) + (sm.zc[2 * DK + tid] + sm.zc[3 * DK + tid]);
    if (PRIOR == kGla) {
      sm.z[tid] = sm.z[tid] * exp2_hw(blast * kLog2e) + add;
      ldc += blast;  // the segment's total log-decay of channel tid
    } else {
      sm.z[tid] += add;
      put_zn(sm, tid, sm.z[tid]);
    }
  }
}

// Exclusive prefix of the segment states of one (b, h) (blockIdx.y): slot s
// of `pre` receives the state entering segment s, combined from the own states
// of segments 0 .. s-1 in `own`, each relative to its own shift.  One thread
// per state entry: S[j][*] carries row shift c_j, z needs none, c is the max.
// GLA: the state entering segment s+1 is the one entering s, decayed by the
// total log-decay of segment s along its key channel, plus the own state of s.
template <int PRIOR>
__global__ __launch_bounds__(NTH) void prefix_kernel(const float* __restrict__ own,
                                                     float* __restrict__ pre, int nseg) {
  constexpr int SF = state_floats<PRIOR>();
  const int e = blockIdx.x * NTH + threadIdx.x;
  if (e >= STATE) return;  // (the GLA log-decays need no prefix)
  const size_t base = (size_t)blockIdx.y * nseg * SF;
  const float* ob = own + base;
  float* pb = pre + base;
  const int j = e < DV * DK ? e / DK : (e >= DV * DK + DK ? e - DV * DK - DK : -1);
  // key channel of an S or z entry (decay), -1 for a shift entry
  const int kc = e < DV * DK ? e % DK : (e < DV * DK + DK ? e - DV * DK : -1);
  // segments in batches of PB: every load of a batch is issued before the
  // batch's (sequential) combination
  constexpr int PB = 8;
  float acc = 0.f, C = -INFINITY;
  for (int s0 = 0; s0 + 1 < nseg; s0 += PB) {
    float val[PB], cs[PB], lg[PB];
#pragma unroll
    for (int u = 0; u < PB; ++u) {
      const size_t o = (size_t)min(s0 + u, nseg - 2) * SF;  // (past the end: unused)
      val[u] = ob[o + e];
      cs[u] = j >= 0 ? ob[o + DV * DK + DK + j] : 0.f;
      lg[u] = (PRIOR == kGla && kc >= 0) ? ob[o + STATE + kc] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < PB; ++u) {
      const int sg = s0 + u;
      if (sg + 1 >= nseg) break;
      const float dcy = (PRIOR == kGla && kc >= 0) ? exp2_hw(lg[u] * kLog2e) : 1.f;
      if (e < DV * DK) {
        const float Cn = fmaxf(C, cs[u]);
        acc = acc * dcy * exp2_hw(C - Cn) + val[u] * exp2_hw(cs[u] - Cn);
        C = Cn;
      } else if (e < DV * DK + DK) {
        acc = acc * dcy + val[u];
      } else {
        acc = fmaxf(C, val[u]);
        C = acc;
      }
      pb[(size_t)(sg + 1) * SF + e] = acc;
    }
  }
}

// Own state [S | z | c] of one segment, linear prior, with the four waves of
// the workgroup independent of each other: wave w takes the segment's 32-key
// tiles w, w + 4, w + 8, ..., streams each into a double-buffered tile pair of
// its own in LDS by direct buffer loads (no workgroup barrier inside the
// loop), and accumulates its own S^T (64 x 64 fp32), its own sum of phi(k)
// (a matrix-core product with rows of ones, from the same rounded phi(k) as
// S: rows 0-15 of one accumulator sum d_k 0-31, rows 16-31 sum d_k 32-63)
// and its own lazily raised per-channel shift.  The four partial states
// meet in LDS at the end, each rescaled to the largest of the four shifts.
// The sum over a segment does not depend on the order of its keys, so the
// result is the state the sequential scan leaves, up to rounding.
constexpr int SKT = 32;  // keys per wave tile
struct StateTiles {      // one buffer of one wave
  bf16 k[SKT * DK];      // K [key][d_k], swizzled (see swz_off)
  bf16 v[SKT * DV];      // V [key][d_v], swizzled
};
struct StatePart {       // one wave's state after its tiles
  float s[DV * DK];      // S [d_v][d_k]
  float z[DK];
  float c[DV];
};
union StateSmem {
  StateTiles t[4][2];
  StatePart p[4];
};

__global__ __launch_bounds__(NTH, 2) void linear_state_kernel(const bf16* __restrict__ K,
                                                           const bf16* __restrict__ V,
                                                           const float* __restrict__ beta,
                                                           float* __restrict__ ws, int H, int T,
                                                           int nseg, int segt) {
  static_assert(DK == 64 && DV == 64, "two 32-wide blocks of each");
  __shared__ __align__(16) StateSmem sm;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n = lane & 31, hl = lane >> 5;
  const int wave_s = __builtin_amdgcn_readfirstlane(wave);
  const int seg = blockIdx.x % nseg;
  const int bh = blockIdx.x / nseg;
  const int h = bh % H;
  const bf16* Kh = K + (size_t)bh * T * DK;
  const bf16* Vh = V + (size_t)bh * T * DV;
  const int tbeg = seg * segt, tend = min(tbeg + segt, T);

  // lane offsets of the direct loads: LDS slot i * 64 + lane of a tile is
  // row i * 8 + lane / 8, position lane % 8, which holds 16-byte chunk
  // (lane % 8) ^ swz(row) of that row
  unsigned goff[SKT / 8];
#pragma unroll
  for (int i = 0; i < SKT / 8; ++i) {
    const int r = i * 8 + (lane >> 3);
    goff[i] = (unsigned)(r * DK * 2 + (((lane & 7) ^ swz<DK>(r)) << 4));
  }
  const unsigned lds0 = lds_addr(&sm) + (unsigned)wave_s * 2u * (unsigned)sizeof(StateTiles);
  const auto issue = [&](int t0, int b) {
    // rows at or past the segment's end load as zeros
    const unsigned bytes = (unsigned)(min(tend, t0 + SKT) - t0) * DK * 2u;
    const rsrc_t rk = buffer_rsrc(Kh + (size_t)t0 * DK, bytes);
    const rsrc_t rv = buffer_rsrc(Vh + (size_t)t0 * DV, bytes);
    const unsigned lk = lds0 + (unsigned)b * (unsigned)sizeof(StateTiles);
    const unsigned lv = lk + (unsigned)(SKT * DK * 2);
#pragma unroll
    for (int i = 0; i < SKT / 8; ++i) {
      dma16b(rk, goff[i], lk + i * 1024u);
      dma16b(rv, goff[i], lv + i * 1024u);
    }
  };

  float blj[2], cj[2] = {-INFINITY, -INFINITY};
#pragma unroll
  for (int cb = 0; cb < 2; ++cb) blj[cb] = beta[h * DV + cb * 32 + n] * kLog2e;
  f32x16 st[2][2], zacc = f32x16{};
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) st[a][b] = f32x16{};
  // A operand rows 0-15 (kb = 0) or 16-31 (kb = 1) all ones, the rest zero
  bf16x8 ones[2];
#pragma unroll
  for (int u = 0; u < 8; ++u) {
    ones[0][u] = (bf16)(n < 16 ? 1.f : 0.f);
    ones[1][u] = (bf16)(n < 16 ? 0.f : 1.f);
  }

  // (t0 is held wave-uniform, so the partial last tile is a branch of its own)
  if (tbeg + wave_s * SKT < tend) issue(tbeg + wave_s * SKT, 0);
  int it = 0;
  for (int t0 = tbeg + wave_s * SKT; t0 < tend; t0 += 4 * SKT, ++it) {
    const int b = it & 1;
    // the other buffer was read (and its reads waited for) last iteration
    if (t0 + 4 * SKT < tend) {
      issue(t0 + 4 * SKT, b ^ 1);
      static_assert(2 * (SKT / 8) == 8, "loads per tile");
      asm volatile("s_waitcnt vmcnt(8)" ::: "memory");  // this tile's loads done, the next one's in flight
    } else {
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    }
    const StateTiles& tl = sm.t[wave][b];
    const auto tile = [&](auto partial) __attribute__((always_inline)) {
    constexpr bool part = decltype(partial)::value;
    // key of element u of a fragment at k-step ks (frag_tr's order)
    const auto valid = [&](int ks, int u) { return t0 + ppos(ks * 16 + hl * 8 + u) < tend; };

    // phi(K)^T fragments (B operand: column d_k, keys), rounded to bf16;
    // keys past the segment give 0
    bf16x8 kf[2][2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        const bf16x8 raw = frag_tr<DK>(tl.k, kb * 32, ks * 16);
#pragma unroll
        for (int u = 0; u < 8; u += 2) {
          float f0 = phi((float)raw[u]), f1 = phi((float)raw[u + 1]);
          if (part) {
            f0 = valid(ks, u) ? f0 : 0.f;
            f1 = valid(ks, u + 1) ? f1 : 0.f;
          }
          const bf16x2 p2 = to_bf16x2(f0, f1);
          kf[kb][ks][u] = p2[0];
          kf[kb][ks][u + 1] = p2[1];
        }
      }
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int ks = 0; ks < 2; ++ks)
        zacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ones[kb], kf[kb][ks], zacc, 0, 0, 0);

    // per channel block: the tile's column max, the lazy shift, the tilt as
    // E^T fragments (A operand: channel, keys) in bf16 hi + lo, and the update
#pragma unroll
    for (int cb = 0; cb < 2; ++cb) {
      float x[2][8];
      float vmax = -INFINITY;
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        const bf16x8 raw = frag_tr<DV>(tl.v, cb * 32, ks * 16);
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          x[ks][u] = (float)raw[u];
          if (part && !valid(ks, u)) x[ks][u] = -INFINITY;
          vmax = fmaxf(vmax, x[ks][u]);
        }
      }
      vmax = fmaxf(vmax, other_half(vmax));
      const float mx = vmax * blj[cb];
      const float cnew = (mx > cj[cb] + kColLag) ? mx : cj[cb];
      if (__any(cnew != cj[cb])) {
        // S^T rows of this block are channels: lane (i, hl) holds row
        // 8 (i / 4) + 4 hl + i % 4, whose factor sits in lane of that index
        const float g = exp2_hw(cj[cb] - cnew);
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const float gi = __shfl(g, (i >> 2) * 8 + hl * 4 + (i & 3));
          st[cb][0][i] *= gi;
          st[cb][1][i] *= gi;
        }
      }
      cj[cb] = cnew;
      const float sh = kBias - cnew;
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        bf16x8 eh, el;
#pragma unroll
        for (int u = 0; u < 8; u += 2) {
          const float e0 = exp2_hw(fmaf(x[ks][u], blj[cb], sh));
          const float e1 = exp2_hw(fmaf(x[ks][u + 1], blj[cb], sh));
          const bf16x2 h2 = to_bf16x2(e0, e1);
          const bf16x2 l2 = to_bf16x2(e0 - (float)h2[0], e1 - (float)h2[1]);
          eh[u] = h2[0];
          eh[u + 1] = h2[1];
          el[u] = l2[0];
          el[u + 1] = l2[1];
        }
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
          st[cb][kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(eh, kf[kb][ks], st[cb][kb], 0, 0, 0);
          st[cb][kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(el, kf[kb][ks], st[cb][kb], 0, 0, 0);
        }
      }
    }
    };
    if (t0 + SKT <= tend) tile(std::false_type());
    else tile(std::true_type());
  }

  // ---- the four partial states meet in LDS (over the tiles: every wave's
  // reads of them are done after the barrier)
  __syncthreads();
  StatePart& P = sm.p[wave];
#pragma unroll
  for (int cb = 0; cb < 2; ++cb)
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int i = 0; i < 16; ++i)
        P.s[(cb * 32 + (i >> 2) * 8 + hl * 4 + (i & 3)) * DK + kb * 32 + n] = st[cb][kb][i];
  if (hl == 0) {
    P.z[n] = zacc[0];        // row 4 hl, below 16
    P.z[32 + n] = zacc[8];   // row 16 + 4 hl
    P.c[n] = cj[0];
    P.c[32 + n] = cj[1];
  }
  __syncthreads();
  float* S = ws + ((size_t)bh * nseg + seg) * STATE;
  for (int e = tid; e < DV * DK; e += NTH) {
    const int j = e / DK;
    const float C = fmaxf(fmaxf(sm.p[0].c[j], sm.p[1].c[j]), fmaxf(sm.p[2].c[j], sm.p[3].c[j]));
    float acc = 0.f;
#pragma unroll
    for (int w = 0; w < 4; ++w) acc += sm.p[w].s[e] * exp2_hw(sm.p[w].c[j] - C);
    S[e] = acc;
  }
  if (tid < DK) S[DV * DK + tid] = (sm.p[0].z[tid] + sm.p[1].z[tid]) + (sm.p[2].z[tid] + sm.p[3].z[tid]);
  if (tid < DV)
    S[DV * DK + DK + tid] =
        fmaxf(fmaxf(sm.p[0].c[tid], sm.p[1].c[tid]), fmaxf(sm.p[2].c[tid], sm.p[3].c[tid]));
}

template <int PRIOR, bool OUT, int CH, int NSUB, bool FIXED>
__global__ __launch_bounds__(NTH, (PRIOR == kElu || FIXED) && CH <= 64 ? 2 : 1) void linear_kernel(const bf16* __restrict__ Q,
                                                     const bf16* __restrict__ K,
                                                     const bf16* __restrict__ V,
                                                     const float* __restrict__ G,
                                                     const float* __restrict__ beta,
                                                     float* __restrict__ out,
                                                     float* __restrict__ ws, int H, int T,
                                                     int nseg, int segc) {
  constexpr int SF = state_floats<PRIOR>();
  __shared__ __align__(16) ScanSmem<PRIOR, CH, NSUB> sm;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int hl = lane >> 5;
  const int seg = blockIdx.x % nseg;
  const int bh = blockIdx.x / nseg;
  const int h = bh % H;
  const bf16* Qh = Q + (size_t)bh * T * DK;
  const bf16* Kh = K + (size_t)bh * T * DK;
  const bf16* Vh = V + (size_t)bh * T * DV;
  const float* Gh = PRIOR == kGla ? G + (size_t)bh * T * DK : nullptr;
  float* Oh = out + (size_t)bh * T * DV;
  float* wsh = ws + (size_t)bh * nseg * SF;  // own states; entering states follow gridDim.x slots on
  const int dvb = wave >> 1, sub = wave & 1;
  const int ch = dvb * 32 + (lane & 31);  // this lane's tilt channel

  if (tid < DV) {
    const float bl = beta[h * DV + tid] * kLog2e;
    sm.bl[tid] = bl;
    sm.inv[tid] = 1.f / bl;
  }
  if (tid < DK) {
    sm.z[tid] = 0.f;
    put_zn(sm, tid, 0.f);
  }
  f32x16 st = f32x16{};
  const float blj = beta[h * DV + ch] * kLog2e;
  float cj = -INFINITY;  // running shift of channel ch
  float ldc = 0.f;       // GLA: this segment's total log-decay of key channel tid (tid < DK)
  __syncthreads();

  const int tbeg = seg * segc * CH;
  const int tend = min(tbeg + segc * CH, T);
  ChunkRegs<CH> cr;
  fetch_chunk<PRIOR, OUT, CH>(cr, Qh, Kh, Vh, Gh, tbeg, T);

  // FIXED: the shift is the segment's own (left by the state pass with its
  // own state), raised to the entering state's where that one is larger
  const float* cown = wsh + (size_t)seg * SF + DV * DK + DK;
  if (FIXED) cj = cown[ch];
  if (OUT && seg > 0) {
    // entering state, left by the prefix kernel in the second half of ws
    const float* S = wsh + (size_t)gridDim.x * SF + (size_t)seg * SF;
    if (tid < DK) {
      sm.z[tid] = S[DV * DK + tid];
      put_zn(sm, tid, sm.z[tid]);
    }
    cj = FIXED ? fmaxf(cj, S[DV * DK + DK + ch]) : S[DV * DK + DK + ch];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int row = dvb * 32 + (i >> 2) * 8 + hl * 4 + (i & 3);
      const int col = sub * 32 + (lane & 31);
      float v = S[row * DK + col];
      if (FIXED) {
        const float ce = S[DV * DK + DK + row];
        v *= exp2_hw(ce - fmaxf(ce, cown[row]));
      }
      st[i] = v;
    }
    __syncthreads();
  }

  for (int t0 = tbeg; t0 < tend; t0 += CH)
    scan_chunk<PRIOR, OUT, CH, NSUB, FIXED>(sm, st, cj, blj, ldc, cr, Qh, Kh, Vh, Gh, Oh, t0,
                                     t0 + CH < tend ? t0 + CH : T, T);

  if (!OUT) {
    float* S = wsh + (size_t)seg * SF;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int row = dvb * 32 + (i >> 2) * 8 + hl * 4 + (i & 3);
      const int col = sub * 32 + (lane & 31);
      S[row * DK + col] = st[i];
    }
    __syncthreads();  // the last z update
    if (tid < DK) S[DV * DK + tid] = sm.z[tid];
    if (sub == 0 && hl == 0) S[DV * DK + DK + ch] = cj;
    if (PRIOR == kGla && tid < DK) S[STATE + tid] = ldc;
  }
}

// Segments of one call: the scan is sequential inside a segment, so the
// fewest tiles per segment that still give about kScanSlots (b, h, segment)
// workgroups (two per compute unit of a 256-CU device, all resident at
// once).  A function of the sizes only, so the workspace query needs no
// device.  Tiles are max(chunk, 32) tokens.
constexpr int kScanSlots = 512;

int tile_of_chunk(int chunk) { return chunk < 32 ? 32 : chunk; }

struct ScanPlan {
  int nseg, segc;
  ScanPlan(int B, int H, int T, int tile) {
    const int nbh = B * H;
    const int ntile = (T + tile - 1) / tile;
    const int want = max(1, kScanSlots / nbh);
    segc = (ntile + want - 1) / want;
    nseg = (ntile + segc - 1) / segc;
  }
  // own segment states, then the entering (prefix) states; nothing when the
  // whole sequence is one segment
  size_t bytes(int B, int H, bool gla) const {
    if (nseg <= 1) return 0;
    const size_t sf = gla ? state_floats<kGla>() : state_floats<kElu>();
    return 2 * (size_t)B * H * nseg * sf * sizeof(float);
  }
};

template <int PRIOR, int CH, int NSUB>
hipError_t launch_scan(const void* Q, const void* K, const void* V, const float* G,
                       const float* beta, float* out, int B, int H, int T, void* wsv,
                       hipStream_t stream) {
  constexpr int SF = state_floats<PRIOR>();
  const int nbh = B * H;
  const ScanPlan plan(B, H, T, CH);
  const int nseg = plan.nseg, segc = plan.segc;
  float* ws = static_cast<float*>(wsv);
  const bf16* q = reinterpret_cast<const bf16*>(Q);
  const bf16* k = reinterpret_cast<const bf16*>(K);
  const bf16* v = reinterpret_cast<const bf16*>(V);
  hipError_t e = hipSuccess;
  if (nseg > 1) {
    if constexpr (PRIOR == kElu)
      hipLaunchKernelGGL(linear_state_kernel, dim3((unsigned)(nbh * nseg)), dim3(NTH), 0, stream,
                         k, v, beta, ws, H, T, nseg, segc * CH);
    else
      hipLaunchKernelGGL((linear_kernel<PRIOR, false, CH, NSUB, false>), dim3((unsigned)(nbh * nseg)),
                         dim3(NTH), 0, stream, q, k, v, G, beta, out, ws, H, T, nseg, segc);
    e = hipGetLastError();
    if (e == hipSuccess) {
      hipLaunchKernelGGL(prefix_kernel<PRIOR>,
                         dim3((unsigned)((STATE + NTH - 1) / NTH), (unsigned)nbh), dim3(NTH), 0,
                         stream, ws, ws + (size_t)nbh * nseg * SF, nseg);
      e = hipGetLastError();
    }
  }
  if (e == hipSuccess) {
    // with segment states, each segment reads at its own final shift
    if (nseg > 1)
      hipLaunchKernelGGL((linear_kernel<PRIOR, true, CH, NSUB, true>), dim3((unsigned)(nbh * nseg)),
                         dim3(NTH), 0, stream, q, k, v, G, beta, out, ws, H, T, nseg, segc);
    else
      hipLaunchKernelGGL((linear_kernel<PRIOR, true, CH, NSUB, false>), dim3((unsigned)(nbh * nseg)),
                         dim3(NTH), 0, stream, q, k, v, G, beta, out, ws, H, T, nseg, segc);
    e = hipGetLastError();
  }
  return e;
}

}  // namespace

size_t scan_ws_bytes(int B, int H, int T, int chunk, bool gla) {
  return ScanPlan(B, H, T, tile_of_chunk(chunk)).bytes(B, H, gla);
}

hipError_t launch_linear_bf16(const void* Q, const void* K, const void* V, const float* beta,
                              float* out, int B, int H, int T, int dk, int dv, int chunk,
                              void* ws, hipStream_t stream) {
  if (dk != DK || dv != DV) return hipErrorNotSupported;
  switch (chunk) {
    case 16: return launch_scan<kElu, 32, 2>(Q, K, V, nullptr, beta, out, B, H, T, ws, stream);
    case 32: return launch_scan<kElu, 32, 1>(Q, K, V, nullptr, beta, out, B, H, T, ws, stream);
    case 64: return launch_scan<kElu, 64, 1>(Q, K, V, nullptr, beta, out, B, H, T, ws, stream);
    case 128: return launch_scan<kElu, 128, 1>(Q, K, V, nullptr, beta, out, B, H, T, ws, stream);
    default: return hipErrorNotSupported;
  }
}

hipError_t launch_gla_bf16(const void* Q, const void* K, const void* V, const float* G,
                           const float* beta, float* out, int B, int H, int T, int dk, int dv,
                           int chunk, void* ws, hipStream_t stream) {
  if (dk != DK || dv != DV || chunk != GCH) return hipErrorNotSupported;
  return launch_scan<kGla, GCH, 1>(Q, K, V, G, beta, out, B, H, T, ws, stream);
}

}  // namespace fem
