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
//     bf16-rounded probabilities that feed the product (a small MFMA against
//     a 0/1 selector), so that rounding P cancels between numerator and
//     normaliser.
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
// one (b, h); each wave owns 32 rows for the products and D/NW channels for
// the tilt (so the running column maximum needs no cross-wave reduction).
//
// Schedule.  A wave cannot issue vector instructions while its own MFMAs run,
// but the two waves sharing a SIMD can overlap each other's.  So every wave
// alternates a matrix-only block M(k) = {PV(k-1), QK(k)} with a vector-only
// block {softmax(k) -> P(k), tilt of its channels of tile k}, and the two
// waves of a SIMD run them in opposite halves of each iteration (two barriers
// per 64-key tile).  K(k+1) and V(k+1) stream straight into the free LDS
// buffers (global_load_lds_dwordx4) during iteration k; K, V and E are double
// buffered.  Workgroups run longest causal extent first; workgroup i of a
// causal level covers head i, so a head's workgroups share an XCD.

#include "fem_device.h"
#include "fem_internal.h"

#include <mutex>

namespace fem {
namespace {

constexpr float kBias = 64.f;        // E = 2^(x - c + kBias) <= 2^(kBias + kColLag)
constexpr float kColLag = 16.f;      // column shift raised only past this lag
constexpr float kRowLag = 8.f;       // row max raised only past this lag (P <= 2^8)
constexpr float kUnderflow = 0x1p-64f;

typedef __attribute__((ext_vector_type(4))) int i32x4;
typedef __attribute__((ext_vector_type(2))) unsigned u32x2;

template <int D, int NW>
struct Cfg {
  static constexpr int BQ = NW * 32;      // query rows per workgroup
  static constexpr int BK = 64;           // keys per tile
  static constexpr int NT = NW * 64;      // threads
  static constexpr int NCB = D / 32;      // 32-channel output blocks
  static constexpr int NKS = D / 16;      // 16-wide k-steps of Q K^T
  static constexpr int KROW = D + 8;      // K / V tile row stride (bf16): one 16-byte pad slot
  static constexpr int EROW = BK + 8;     // E^T row stride (bf16), +16 B pad
  static constexpr int CPW = D / NW;      // channels tilted per wave
  static constexpr int G = 64 / CPW;      // lanes per channel in the tilt
  static constexpr int RPL = 16 / G;      // 4-key runs per tilt lane
  // K / V tiles are filled by direct global->LDS loads: each wave instruction
  // writes 64 consecutive 16-byte slots (1 KiB); a padded row is SPR slots.
  static constexpr int SPR = KROW / 8;               // slots per padded row
  static constexpr int BLOCKS = BK * SPR / 64;       // 1 KiB blocks per tile
  static constexpr int BPW = (BLOCKS + NW - 1) / NW; // blocks per wave
  // LDS layout (bytes)
  static constexpr int KB = BK * KROW * 2;
  static constexpr int EB = D * EROW * 2;
  static constexpr int OFF_K = 0;                 // 2 buffers
  static constexpr int OFF_V = OFF_K + 2 * KB;    // 2 buffers
  static constexpr int OFF_EH = OFF_V + 2 * KB;   // 2 buffers
  static constexpr int OFF_EL = OFF_EH + 2 * EB;  // 2 buffers
  static constexpr int OFF_F = OFF_EL + 2 * EB;   // floats
  static constexpr int NF = D /*bl*/ + D /*inv*/ + 2 * D /*c*/ + 2 * D /*g*/ + NW * D /*cw*/;
  static constexpr int OFF_R = OFF_F + NF * 4;    // rose flags [2][NW]
  static constexpr size_t LDS = OFF_R + 2 * NW * 4;
  static_assert(CPW * NW == D && G * CPW == 64 && RPL * G == 16, "tilt mapping");
  static_assert(BK * SPR % 64 == 0, "tile = whole 1 KiB blocks");
  static_assert(LDS <= 160 * 1024, "LDS budget");
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
struct Smem {
  using C = Cfg<D, NW>;
  unsigned char* base;
  __device__ unsigned char* k(int b) const { return base + C::OFF_K + b * C::KB; }
  __device__ unsigned char* v(int b) const { return base + C::OFF_V + b * C::KB; }
  __device__ unsigned char* eh(int b) const { return base + C::OFF_EH + b * C::EB; }
  __device__ unsigned char* el(int b) const { return base + C::OFF_EL + b * C::EB; }
  __device__ float* bl() const { return reinterpret_cast<float*>(base + C::OFF_F); }
  __device__ float* inv() const { return bl() + D; }
  __device__ float* c(int b) const { return bl() + 2 * D + b * D; }
  __device__ float* g(int b) const { return bl() + 4 * D + b * D; }
  __device__ float* cw(int w) const { return bl() + 6 * D + w * D; }
  __device__ int* rose(int b) const { return reinterpret_cast<int*>(base + C::OFF_R) + b * NW; }
};

// Bits of two floats' upper halves packed into one dword (bf16 truncation).
__device__ __forceinline__ unsigned pack_hi16(float lo_elem, float hi_elem) {
  return __builtin_amdgcn_perm(__float_as_uint(hi_elem), __float_as_uint(lo_elem), 0x07060302u);
}

// max(x, x of lane ^ o) without going through LDS where the hardware has a
// lane swap for that distance (v_permlane16_swap / v_permlane32_swap).
__device__ __forceinline__ float max_xor(float x, int o) {
  const unsigned u = __float_as_uint(x);
  if (o == 32) {
    const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
  }
  if (o == 16) {
    const auto r = __builtin_amdgcn_permlane16_swap(u, u, false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
  }
  return fmaxf(x, __shfl_xor(x, o));
}

// Tilt of tile tt (first key k0) for this wave's CPW channels, in two steps so
// that the LDS reads of V can be issued before unrelated vector work:
//   tilt_read   : this lane's V values (channel jj, 4-key runs g + G*u);
//   tilt_finish : column max over the tile (in-lane, then across the G lanes
//                 of a channel), lazily raised running shift, E = 2^(x - c +
//                 bias) split into bf16 hi (truncated) and lo (the rounded
//                 remainder) -> E^T buffers.  FULL: every key of the tile < T.
template <int D, int NW>
__device__ __forceinline__ void tilt_read(const Smem<D, NW>& sm, int tt, int wave, int lane,
                                          float (&v)[Cfg<D, NW>::RPL][4]) {
  using C = Cfg<D, NW>;
  const int jj = lane % C::CPW, g = lane / C::CPW;
  const int j = wave * C::CPW + jj;
  const unsigned char* sv = sm.v(tt & 1) + j * 2;
#pragma unroll
  for (int u = 0; u < C::RPL; ++u) {
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const int key = 4 * (g + C::G * u) + b;
      v[u][b] = (float)*reinterpret_cast<const bf16*>(sv + key * C::KROW * 2);
    }
  }
}

template <int D, int NW, bool FULL>
__device__ __forceinline__ void tilt_finish(const Smem<D, NW>& sm, int tt, int k0, int T,
                                            int wave, int lane,
                                            const float (&v)[Cfg<D, NW>::RPL][4]) {
  using C = Cfg<D, NW>;
  const int jj = lane % C::CPW, g = lane / C::CPW;
  const int j = wave * C::CPW + jj;
  const float bl = sm.bl()[j];
  float vmax = -INFINITY;
#pragma unroll
  for (int u = 0; u < C::RPL; ++u) {
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const int key = 4 * (g + C::G * u) + b;
      if (FULL || k0 + key < T) vmax = fmaxf(vmax, v[u][b]);
    }
  }
#pragma unroll
  for (int o = C::CPW; o < 64; o <<= 1) vmax = max_xor(vmax, o);
  const float mx = vmax * bl;  // bl > 0: max of beta*v*log2e
  const float cold = (tt == 0) ? -INFINITY : sm.c((tt - 1) & 1)[j];
  const float cnew = (mx > cold + kColLag) ? mx : cold;
  const float sh = kBias - cnew;
  unsigned char* eh = sm.eh(tt & 1) + j * C::EROW * 2;
  unsigned char* el = sm.el(tt & 1) + j * C::EROW * 2;
#pragma unroll
  for (int u = 0; u < C::RPL; ++u) {
    const int key0 = 4 * (g + C::G * u);
    float e[4], lo[4];
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      e[b] = exp2_hw(fmaf(v[u][b], bl, sh));
      if (!FULL && k0 + key0 + b >= T) e[b] = 0.f;
      lo[b] = e[b] - __uint_as_float(__float_as_uint(e[b]) & 0xffff0000u);
    }
    const u32x2 hi2 = {pack_hi16(e[0], e[1]), pack_hi16(e[2], e[3])};
    const bf16x2 l01 = to_bf16x2(lo[0], lo[1]), l23 = to_bf16x2(lo[2], lo[3]);
    const u32x2 lo2 = {__builtin_bit_cast(unsigned, l01), __builtin_bit_cast(unsigned, l23)};
    *reinterpret_cast<u32x2*>(eh + e_pos(key0) * 2) = hi2;
    *reinterpret_cast<u32x2*>(el + e_pos(key0) * 2) = lo2;
  }
  if (g == 0) {
    sm.c(tt & 1)[j] = cnew;
    sm.g(tt & 1)[j] = exp2_hw(cold - cnew);
  }
  const bool rose = __any(cnew != cold);
  if (lane == 0) sm.rose(tt & 1)[wave] = rose ? 1 : 0;
}

// Whole tilt of tile tt (prologue).
template <int D, int NW, bool FULL>
__device__ __forceinline__ void tilt_tile(const Smem<D, NW>& sm, int tt, int k0, int T, int wave,
                                          int lane) {
  float v[Cfg<D, NW>::RPL][4];
  tilt_read<D, NW>(sm, tt, wave, lane, v);
  tilt_finish<D, NW, FULL>(sm, tt, k0, T, wave, lane, v);
}

// Direct global -> LDS copy of one K or V tile (rows k0 .. k0+63, padded rows).
// Wave w writes 1 KiB blocks w, w+NW, ...; lane l of a block fills slot
// 64*blk + l, i.e. row slot/SPR, chunk slot%SPR (the pad chunk re-reads chunk
// 0).  Rows at or past T are clamped to T-1: their keys are masked anyway.
// The address is a uniform tile base plus a 32-bit lane offset, so the loads
// use scalar-base addressing and no 64-bit lane addresses stay live.
template <int D, int NW>
__device__ __forceinline__ void load_tile(const bf16* __restrict__ src, unsigned char* dst, int k0,
                                          int T, int wave, int lane) {
  using C = Cfg<D, NW>;
  const char* base = reinterpret_cast<const char*>(src + (size_t)k0 * D);
  const int rmax = T - 1 - k0;
#pragma unroll
  for (int u = 0; u < C::BPW; ++u) {
    const int blk = wave + NW * u;
    if (C::BLOCKS % NW == 0 || blk < C::BLOCKS) {
      const int slot = blk * 64 + lane;
      const int row = min(slot / C::SPR, rmax), chunk = slot % C::SPR;
      const unsigned off = (unsigned)(row * D + (chunk < D / 8 ? chunk * 8 : 0)) * 2u;
      __builtin_amdgcn_global_load_lds(base + off, dst + blk * 1024, 16, 0, 0);
    }
  }
}

__device__ __forceinline__ void wait_vmem() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// Matrix-only block: PV of the previous tile (if PV) then QK^T of this tile
// (if QK), as one straight run of MFMAs.  Every MFMA takes its A operand
// (E^T hi/lo or K) from LDS; the fragments are prefetched RING steps ahead so
// that LDS latency hides behind the MFMAs already issued.  PV steps alternate
// the output blocks (independent accumulators) within each hi/lo half.
//
// With PV the block also adds this tile's row sums of P into lacc: a 16x16x32
// product of a constant 0/1 selector (lsel) with the same P^T fragments.
// Lane l supplies selector row l%16 over k-block l/16; the B operand's k-block
// b holds query (l%16) + 16*(b%2), so a one in row m = 4r for the k-blocks
// with b%2 == r%2 sums query (l%16) + 16*(r%2) into output row 4r, which the
// 16x16 output layout places in register 0 of lane 16r + l%16.  Hence
// lacc[0] of every lane is the full row sum of its query l%32.
template <int D, int NW, bool PV, bool QK>
__device__ __forceinline__ void mfma_block(f32x16 (&acc)[D / 32], f32x4& lacc, f32x16& s0,
                                           f32x16& s1, const bf16x8 (&pf)[4],
                                           const bf16x8 (&qf)[D / 16], const bf16x8& lsel,
                                           const unsigned char* eh, const unsigned char* el,
                                           const unsigned char* kt) {
  using C = Cfg<D, NW>;
  constexpr int NPV = PV ? 4 * 2 * C::NCB : 0;
  constexpr int NQK = QK ? 2 * C::NKS : 0;
  constexpr int NS = NPV + NQK;
  constexpr int RING = 6;
  auto frag = [&](int s) -> bf16x8 {
    if (s < NPV) {
      const int ks = s / (2 * C::NCB), rem = s % (2 * C::NCB);
      const int lo = rem / C::NCB, cb = rem % C::NCB;
      const unsigned char* b = lo ? el : eh;
      return *reinterpret_cast<const bf16x8*>(b + cb * 32 * C::EROW * 2 + ks * 32);
    }
    const int t = s - NPV, ks = t >> 1, kb = t & 1;
    return *reinterpret_cast<const bf16x8*>(kt + kb * 32 * C::KROW * 2 + ks * 32);
  };
  bf16x8 ring[RING];
#pragma unroll
  for (int s = 0; s < RING; ++s)
    if (s < NS) ring[s] = frag(s);
  // Row sums of P on the matrix pipe while the first fragments are in flight.
  if (PV) {
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
      lacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(lsel, pf[ks], lacc, 0, 0, 0);
  }
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    const bf16x8 a = ring[s % RING];
    if (s + RING < NS) ring[s % RING] = frag(s + RING);
    if (s < NPV) {
      const int ks = s / (2 * C::NCB), cb = (s % (2 * C::NCB)) % C::NCB;
      acc[cb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pf[ks], acc[cb], 0, 0, 0);
    } else {
      const int t = s - NPV, ks = t >> 1;
      if (t & 1) s1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[ks], s1, 0, 0, 0);
      else s0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[ks], s0, 0, 0, 0);
    }
  }
  // Pin the order: RING fragment reads up front, the row-sum MFMAs, then one
  // read ahead per MFMA.
#pragma unroll
  for (int s = 0; s < RING; ++s) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
  if (PV) __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    if (s + RING < NS) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
  }
}

template <int D, int NW>
__global__ __launch_bounds__(NW * 64) void softmax_bf16_kernel(
    const bf16* __restrict__ Q, const bf16* __restrict__ K, const bf16* __restrict__ V,
    const float* __restrict__ beta, float* __restrict__ out, int H, int T, int nqb,
    int nbh) {
  using C = Cfg<D, NW>;
  extern __shared__ __align__(16) unsigned char smem[];
  const Smem<D, NW> sm{smem};

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int n = lane & 31;   // query column of this lane in the 32x32 blocks
  const int hl = lane >> 5;  // lane half
  // Waves w and w + NW/2 share a SIMD.  Group A (w < NW/2) runs its matrix
  // block in the first half of every iteration and its vector block in the
  // second; group B the other way round, so one wave's vector work overlaps
  // the other's MFMAs.
  const bool grpB = wave >= NW / 2;

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
    sm.bl()[j] = bl;
    sm.inv()[j] = 1.f / bl;
  }

  const int wq0 = q0 + wave * 32;  // first query row of this wave
  const int tq = wq0 + n;          // this lane's query row
  const bool wave_live = wq0 < T;
  const int qlast = min(q0 + C::BQ, T) - 1;
  const int ntiles = qlast / C::BK + 1;
  // Last tile this wave multiplies into its accumulator.  Later tiles may still
  // raise the shared column shift; the wave keeps the shift its accumulator
  // was last rescaled to (cw) instead of rescaling for tiles it skips.
  const int wlast = wave_live ? min((wq0 + 31) / C::BK, ntiles - 1) : -1;

  load_tile<D, NW>(Kh, sm.k(0), 0, T, wave, lane);
  load_tile<D, NW>(Vh, sm.v(0), 0, T, wave, lane);
  bf16x8 qf[C::NKS];
#pragma unroll
  for (int ks = 0; ks < C::NKS; ++ks) {
    bf16x8 z = {};
    qf[ks] = (tq < T) ? *reinterpret_cast<const bf16x8*>(Qh + (size_t)tq * D + ks * 16 + hl * 8)
                      : z;
  }
  wait_vmem();
  __syncthreads();

  f32x16 acc[C::NCB];
#pragma unroll
  for (int cb = 0; cb < C::NCB; ++cb) acc[cb] = f32x16{};
  f32x16 sacc[2] = {f32x16{}, f32x16{}};  // scores: QK(k) -> softmax(k)
  bf16x8 pf[4] = {};                      // probabilities: softmax(k) -> PV(k)
  float m = -INFINITY;  // running row max (log2 units), shared by the lane pair
  f32x4 lacc = {};      // lacc[0]: row sum of the rounded P (see mfma_block)
  bf16x8 lsel;
  {
    const int r = lane & 15, b = lane >> 4;
    const __bf16 one = ((r & 3) == 0 && ((r >> 2) & 1) == (b & 1)) ? (__bf16)1.f : (__bf16)0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) lsel[e] = one;
  }
  const float scale2 = kLog2e / sqrtf((float)D);
  const int kofs = n * C::KROW * 2 + hl * 16;  // lane part of K fragment addresses
  const int eofs = n * C::EROW * 2 + hl * 16;  // lane part of E fragment addresses

  // ---- matrix block of iteration k: PV(k-1) then QK(k)
  auto mblock = [&](int k) {
    const int j = k - 1;
    const bool do_pv = j >= 0 && j <= wlast;
    const bool do_qk = k <= wlast;
    if (!do_pv && !do_qk) return;
    const int pb = j & 1;
    if (do_pv && j > 0) {  // tile 0 always raises the shift, but the accumulator is still zero
      const i32x4* rf = reinterpret_cast<const i32x4*>(sm.rose(pb));
      i32x4 any4 = rf[0];
#pragma unroll
      for (int w = 1; w < NW / 4; ++w) any4 |= rf[w];
      if (any4[0] | any4[1] | any4[2] | any4[3]) {
        const float* gcol = sm.g(pb);
#pragma unroll
        for (int cb = 0; cb < C::NCB; ++cb) {
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            const f32x4 gg = *reinterpret_cast<const f32x4*>(gcol + cb * 32 + g * 8 + hl * 4);
#pragma unroll
            for (int e = 0; e < 4; ++e) acc[cb][g * 4 + e] *= gg[e];
          }
        }
      }
    }
    const unsigned char* seh = sm.eh(pb & 1) + eofs;
    const unsigned char* sel = sm.el(pb & 1) + eofs;
    const unsigned char* sk = sm.k(k & 1) + kofs;
    f32x16 s0 = f32x16{}, s1 = f32x16{};
    if (do_pv && do_qk)
      mfma_block<D, NW, true, true>(acc, lacc, s0, s1, pf, qf, lsel, seh, sel, sk);
    else if (do_pv)
      mfma_block<D, NW, true, false>(acc, lacc, s0, s1, pf, qf, lsel, seh, sel, sk);
    else
      mfma_block<D, NW, false, true>(acc, lacc, s0, s1, pf, qf, lsel, seh, sel, sk);
    if (do_qk) {
      sacc[0] = s0;
      sacc[1] = s1;
    }
    if (do_pv && j == wlast) {
      const float* cc = sm.c(pb);
      for (int c = lane; c < D; c += 64) sm.cw(wave)[c] = cc[c];
    }
  };

  // ---- vector block: softmax of tile js (-> P, row rescale), tilt of tile jt
  auto vblock = [&](int js, int jt) {
    float tv[C::RPL][4];
    const bool do_tilt = jt < ntiles;
    if (do_tilt) tilt_read<D, NW>(sm, jt, wave, lane, tv);
    if (js >= 0 && js <= wlast) {
      const int k0 = js * C::BK;
      // scores stay raw (q.k); scale2 > 0 so the row max commutes with it
      if ((k0 + C::BK - 1 > wq0) || (k0 + C::BK > T)) {
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            const int key = k0 + kb * 32 + (i >> 2) * 8 + hl * 4 + (i & 3);
            if (key > tq || key >= T) sacc[kb][i] = -INFINITY;
          }
        }
      }
      float mx = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
        for (int i = 0; i < 16; ++i) mx = fmaxf(mx, sacc[kb][i]);
      }
      mx = fmaxf(mx, other_half(mx)) * scale2;
      const float mnew = (mx > m + kRowLag) ? mx : m;
      if (__any(mnew != m)) {
        const float alpha = exp2_hw(m - mnew);
        lacc[0] *= alpha;
#pragma unroll
        for (int cb = 0; cb < C::NCB; ++cb) acc[cb] *= alpha;
        m = mnew;
      }
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const int kb = ks >> 1, s0i = (ks & 1) * 8;
#pragma unroll
        for (int u = 0; u < 8; u += 2) {
          const bf16x2 p2 = to_bf16x2(exp2_hw(fmaf(sacc[kb][s0i + u], scale2, -m)),
                                      exp2_hw(fmaf(sacc[kb][s0i + u + 1], scale2, -m)));
          pf[ks][u] = p2[0];
          pf[ks][u + 1] = p2[1];
        }
      }
    }
    if (do_tilt) {
      if ((jt + 1) * C::BK <= T) tilt_finish<D, NW, true>(sm, jt, jt * C::BK, T, wave, lane, tv);
      else tilt_finish<D, NW, false>(sm, jt, jt * C::BK, T, wave, lane, tv);
    }
  };

  for (int k = 0; k <= ntiles; ++k) {
    if (k + 1 < ntiles) {
      load_tile<D, NW>(Kh, sm.k((k + 1) & 1), (k + 1) * C::BK, T, wave, lane);
      load_tile<D, NW>(Vh, sm.v((k + 1) & 1), (k + 1) * C::BK, T, wave, lane);
    }
    if (!grpB) {
      mblock(k);
      vblock(k, k);
    } else {
      vblock(k - 1, k);
      mblock(k);
    }
    wait_vmem();
    __syncthreads();
  }

  if (!wave_live) return;

  // ---- epilogue: o = (log2 acc - log2 l + c - bias) / (beta log2 e).  The
  // logarithms are split into exponent and mantissa so the bias and the
  // integer parts cancel exactly (tiny beta amplifies any error here).
  const float lt = lacc[0];
  int el;
  const float fl = log2_hw(frexpf(lt, &el));
  const float* cw = sm.cw(wave);
  const float* inv = sm.inv();
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
        int ea;
        const float fa = log2_hw(frexpf(a, &ea));
        o[e] = ((float)(ea - el - (int)kBias) + (fa - fl) + cw[ch0 + e]) * inv[ch0 + e];
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
    const uint64_t fl64 = ((uint64_t)fhi << 32) | flo;
    const int e = __builtin_ctzll(fl64);
    const int t = __builtin_amdgcn_readlane(tq, src);
    const int cb = e >> 4, i = e & 15;
    const int ch = cb * 32 + (i >> 2) * 8 + (src >> 5) * 4 + (i & 3);
    const float o = exact_read<D>(Qh, Kh, Vh, t, ch, scale2, sm.bl()[ch]);
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
