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
//     transposed product leaves one query per lane pair, so the row max needs
//     one v_permlane32_swap and no LDS traffic.
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
// Work decomposition: one workgroup of NW = 8 waves (two per SIMD) owns
// BQ = 32*NW query rows of one (b, h); each wave owns 32 rows for the
// products (two 32-key blocks per tile, so every Q fragment feeds two MFMAs)
// and D/NW channels for the tilt (so the running column maximum needs no
// cross-wave reduction).
//
// The same kernel serves the two-level gated read (Sec. "Two-Level Gated
// FEM", eqs. inner-gate-main and fem-two-gates-main) in two launches:
//   kMean : the prior's expectation mu = sum_i p_t(i) v_i.  The "tilt" stores
//           V itself (exact in bf16, so no lo part and no shift), the
//           accumulator needs only the row rescale, and the epilogue writes
//           mu = acc / l.
//   kGated: the free-energy pass at beta_max whose epilogue reads mu back
//           from the output and writes o = g * ((1 - lam) mu + lam F).
// Both launches reuse one P per tile and row sum per launch; a single pass
// with both accumulators would need 64 more registers per lane at d = 128
// than two waves per SIMD leave, and a third double-buffered E^T tile in LDS.
//
// Schedule.  A wave keeps issuing independent vector instructions while its
// own MFMAs run (about four per 32x32x16 MFMA come for free), so each
// iteration k (one barrier) is two interleaved phases per wave:
//   phase 1: QK^T(k), the row sums and k-step 0 of PV(k-1) on the matrix
//            pipe  ||  tilt of the wave's channels of tile k and the direct
//            loads of tile k+1;
//   phase 2: PV(k-1) k-steps 1..3 (hi and lo)  ||  softmax of tile k (the
//            scores phase 1 just produced).
// The instruction order of each phase is pinned with scheduling barriers, and
// each chain of vector work (exponent, 2^, rounding) is spread over
// consecutive slots so that no instruction waits on its own slot.  Row and
// column rescales of the accumulator are rare; they are deferred to the start
// of the next iteration, before any MFMA reads the accumulator.  P is double
// buffered (softmax(k) writes one buffer while PV(k-1) reads the other); the
// loop is unrolled by two so that the buffer index is a compile-time
// constant.  K(k+1) and V(k+1) stream straight into the free LDS buffers
// (global_load_lds_dwordx4) during iteration k; K, V and E are double
// buffered.  Workgroups run longest causal extent first; workgroup i of a
// causal level covers head i, so a head's workgroups share an XCD.

#include "fem_device.h"
#include "fem_internal.h"

#include <type_traits>


namespace fem {
namespace {

constexpr float kBias = 64.f;        // E = 2^(x - c + kBias) <= 2^(kBias + kColLag)
constexpr float kColLag = 16.f;      // column shift raised only past this lag
constexpr float kRowLag = 8.f;       // row max raised only past this lag (P <= 2^8)
constexpr float kUnderflow = 0x1p-64f;
// Channels with beta at or above this take E rounded to bf16 (relative error
// at most 2^-8, which moves F by at most 2^-8 / beta <= 2^-7) and no lo
// product; smaller beta amplifies that rounding, so those keep hi + lo.
constexpr float kLoBeta = 0.5f;

// What a launch computes (see the header comment).
constexpr int kFem = 0;    // F at beta
constexpr int kMean = 1;   // mu
constexpr int kGated = 2;  // g * ((1 - lam) mu + lam F), mu read from out

typedef __attribute__((ext_vector_type(4))) int i32x4;
typedef __attribute__((ext_vector_type(2))) unsigned u32x2;

// Compile-time shape and variant of a launch: the width of Q and K (DK) and
// of V and the output (DV), the waves per workgroup, what the launch computes
// (MODE), causal or encoder (all keys) read, and fp32 or bf16 output.
template <int DK_, int DV_, int NW_, int MODE_, bool CAUSAL_ = true, bool OBF16_ = false>
struct Cfg {
  static constexpr int DK = DK_, DV = DV_, NW = NW_, MODE = MODE_;
  static constexpr bool CAUSAL = CAUSAL_, OBF16 = OBF16_;
  static constexpr int BQ = NW * 32;      // query rows per workgroup
  static constexpr int BK = 64;           // keys per tile
  static constexpr int NT = NW * 64;      // threads
  static constexpr int NCB = DV / 32;     // 32-channel output blocks
  static constexpr int NKS = DK / 16;     // 16-wide k-steps of Q K^T
  static constexpr int KROW = DK + 8;     // K tile row stride (bf16): one 16-byte pad slot
  static constexpr int VROW = DV + 8;     // V tile row stride (bf16)
  static constexpr int EROW = BK + 8;     // E^T row stride (bf16), +16 B pad
  static constexpr int CPW = DV / NW;     // channels tilted per wave
  static constexpr int G = 64 / CPW;      // lanes per channel in the tilt
  static constexpr int RPL = 16 / G;      // 4-key runs per tilt lane
  // K / V tiles are filled by direct global->LDS loads: each wave instruction
  // writes 64 consecutive 16-byte slots (1 KiB); a padded row is (W+8)/8 slots.
  static constexpr int BLOCKSK = BK * (KROW / 8) / 64;  // 1 KiB blocks per K tile
  static constexpr int BLOCKSV = BK * (VROW / 8) / 64;  // ... per V tile
  static constexpr int BPWK = (BLOCKSK + NW - 1) / NW;  // blocks per wave
  static constexpr int BPWV = (BLOCKSV + NW - 1) / NW;
  static constexpr bool SAME = DK == DV;  // K and V tiles share their load offsets
  // LDS layout (bytes)
  static constexpr int KB = BK * KROW * 2;
  static constexpr int VB = BK * VROW * 2;
  static constexpr int EB = DV * EROW * 2;
  static constexpr int OFF_K = 0;                 // 2 buffers
  static constexpr int OFF_V = OFF_K + 2 * KB;    // 2 buffers
  static constexpr int OFF_EH = OFF_V + 2 * VB;   // 2 buffers
  static constexpr int OFF_EL = OFF_EH + 2 * EB;  // 2 buffers
  static constexpr int OFF_F = OFF_EL + 2 * EB;   // floats
  static constexpr int NF =
      DV /*bl*/ + DV /*inv*/ + 2 * DV /*c*/ + 2 * DV /*g*/ + 64 /*sink*/ + DV /*channel order*/;
  static constexpr int OFF_R = OFF_F + NF * 4;    // column-update flags [2][NW]
  static constexpr size_t LDS = OFF_R + 2 * NW * 4;
  static_assert(CPW * NW == DV && G * CPW == 64 && RPL * G == 16, "tilt mapping");
  static_assert(DK % 32 == 0 && DV % 32 == 0, "widths");
  static_assert(NW % 4 == 0, "flags are read as int4");
  static_assert(LDS <= 160 * 1024, "LDS budget");
  static_assert(OFF_EL - OFF_EH + EB < 65536, "hi and lo share a base register");
  static_assert(!OBF16 || MODE == kFem, "bf16 output only for the plain read");
};

// Position of key r (0..63 within a tile) inside an E^T row.  Within each
// 16-key group the keys are stored in the order the MFMA B operand (P^T,
// taken straight from the S^T accumulator layout) consumes them: lane half h
// holds keys {4h..4h+3, 8+4h..8+4h+3} as its 8 consecutive k-slots.
__host__ __device__ constexpr int e_pos(int r) {
  return (r & ~15) + ((((r & 15) >> 2) & 1) << 3) + ((((r & 15) >> 3) & 1) << 2) + (r & 3);
}

// The tilt lane with group index g writes keys 4(g + G u): their positions
// split into a lane part and a part that is a compile-time constant.
constexpr bool e_pos_splits(int G) {
  for (int g = 0; g < G; ++g)
    for (int u = 0; u < 16 / G; ++u)
      if (e_pos(4 * (g + G * u)) != e_pos(4 * g) + e_pos(4 * G * u)) return false;
  return true;
}

// An LDS byte offset kept in one register exactly as computed at this point:
// the compiler neither folds parts of it into per-access immediates (the
// 16-bit DS offset field cannot hold buffer bases past 64 KiB, which costs a
// register per access) nor hoists it out of the loop.  Accesses then take
// the form base + small immediate.
__device__ __forceinline__ unsigned pin(unsigned x) {
  asm volatile("" : "+v"(x));
  return x;
}

// Channels of one row recomputed per pass over its keys by the exact path.
constexpr int kRepairBatch = 16;

// Exact fp32 read of channels ch[0..nb) (nb <= NB) of row t by the whole
// wave: per channel the joint log-sum-exp of (score + tilt) over the keys
// i < n, minus the log-sum-exp of the scores; each key's score is formed
// once for the whole batch.  Lane c < nb returns channel ch[c]'s value.
template <class C, int NB>
__device__ float exact_row(const bf16* __restrict__ Qh, const bf16* __restrict__ Kh,
                           const bf16* __restrict__ Vh, int t, int n, const int (&ch)[NB],
                           const float (&bl)[NB], int nb, float scale2) {
  const int lane = threadIdx.x & 63;
  Lse2 den, num[NB];
  const bf16x8* qrow = reinterpret_cast<const bf16x8*>(Qh + (size_t)t * C::DK);
  for (int i = lane; i < n; i += 64) {
    const bf16x8* krow = reinterpret_cast<const bf16x8*>(Kh + (size_t)i * C::DK);
    float dot = 0.f;
#pragma unroll 4
    for (int c = 0; c < C::DK / 8; ++c) {
      bf16x8 a = qrow[c], b = krow[c];
#pragma unroll
      for (int e = 0; e < 8; ++e) dot += (float)a[e] * (float)b[e];
    }
    const float s = dot * scale2;
    den.add(s);
#pragma unroll
    for (int c = 0; c < NB; ++c)
      if (c < nb) num[c].add(s + (float)Vh[(size_t)i * C::DV + ch[c]] * bl[c]);
  }
  const float d = den.wave_total();
  float mine = 0.f;
#pragma unroll
  for (int c = 0; c < NB; ++c) {
    if (c < nb) {
      const float o = (num[c].wave_total() - d) / bl[c];
      if (lane == c) mine = o;
    }
  }
  return mine;
}

template <class C>
struct Smem {
  static constexpr int DV = C::DV;
  unsigned char* base;
  __device__ unsigned char* k(int b) const { return base + C::OFF_K + b * C::KB; }
  __device__ unsigned char* v(int b) const { return base + C::OFF_V + b * C::VB; }
  __device__ unsigned char* eh(int b) const { return base + C::OFF_EH + b * C::EB; }
  __device__ unsigned char* el(int b) const { return base + C::OFF_EL + b * C::EB; }
  __device__ float* bl() const { return reinterpret_cast<float*>(base + C::OFF_F); }
  __device__ float* inv() const { return bl() + DV; }
  __device__ float* c(int b) const { return bl() + 2 * DV + b * DV; }
  __device__ float* g(int b) const { return bl() + 4 * DV + b * DV; }
  // Write-only slots for lanes whose store would otherwise need a branch.
  __device__ float* sink() const { return bl() + 6 * DV; }
  // Input channel held by accumulator column j (channel split, see kLoBeta).
  __device__ int* chan() const { return reinterpret_cast<int*>(bl() + 6 * DV + 64); }
  __device__ int* upd(int b) const { return reinterpret_cast<int*>(base + C::OFF_R) + b * C::NW; }
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

// Tilt of tile tt for this wave's CPW channels, as separately placeable steps
// (the phases interleave them with MFMAs):
//   read    : this lane's V values (accumulator column jj, which holds input
//             channel vcol; 4-key runs g + G*u), beta and the previous column
//             shift, all from LDS;
//   colmax  : column max over the tile (a tree in-lane, then across the G
//             lanes of a channel);
//   shift   : lazily raised running shift c_j; stores c, the rescale factor
//             g = 2^(c_old - c_new) and the wave's "some c rose" flag;
//   value(u, b), store(u) : E = 2^(x - c + bias) of key 4(g + G u) + b split
//             into bf16 hi (truncated) and lo (the rounded remainder), or for
//             a column without lo product E rounded to bf16, and the store of
//             run u into the E^T buffers.
// Keys at or past T (last tile only) were loaded as zeros (see load_block);
// read() turns them into -inf, so they leave the column max unchanged and
// give E = 0, which meets P = 0 (the causal mask).
// Stores that only one lane of a group should make go to a sink slot from the
// other lanes, so the code has no branches.
template <class C>
struct Tilt {
  static constexpr int MODE = C::MODE;
  float v[C::RPL][4];
  float e[C::RPL][4];
  float bl, cold, cnew, sh;
  unsigned char* eh;

  // nvalid: the tile's keys before T.  Rows past it were loaded as zeros;
  // the read and gated modes take them as -inf, which stays out of the
  // column max and gives E = 0 (P = 0 there anyway); the mean mode keeps
  // the zeros as values.
  __device__ __forceinline__ void read(const Smem<C>& sm, int tt, int nvalid, int wave, int lane,
                                       int vcol) {
    const int jj = lane % C::CPW, g = lane / C::CPW;
    const int j = wave * C::CPW + jj;
    const unsigned char* sv =
        sm.base + pin(C::OFF_V + (tt & 1) * C::VB + vcol * 2 + 4 * g * C::VROW * 2);
#pragma unroll
    for (int u = 0; u < C::RPL; ++u) {
#pragma unroll
      for (int b = 0; b < 4; ++b)
        v[u][b] = (float)*reinterpret_cast<const bf16*>(sv + (4 * C::G * u + b) * C::VROW * 2);
    }
    if (MODE != kMean && nvalid < C::BK) {
#pragma unroll
      for (int u = 0; u < C::RPL; ++u) {
#pragma unroll
        for (int b = 0; b < 4; ++b)
          if (4 * (g + C::G * u) + b >= nvalid) v[u][b] = -INFINITY;
      }
    }
    if (MODE == kMean) {
      eh = sm.base + pin(C::OFF_EH + (tt & 1) * C::EB + j * C::EROW * 2 + e_pos(4 * g) * 2);
      return;
    }
    bl = sm.bl()[j];
    cold = (tt == 0) ? -INFINITY : sm.c((tt - 1) & 1)[j];
  }

  __device__ __forceinline__ float colmax() const {
    float t[C::RPL];
#pragma unroll
    for (int u = 0; u < C::RPL; ++u)
      t[u] = fmaxf(fmaxf(v[u][0], v[u][1]), fmaxf(v[u][2], v[u][3]));
#pragma unroll
    for (int w = 1; w < C::RPL; w <<= 1) {
#pragma unroll
      for (int u = 0; u + w < C::RPL; u += 2 * w) t[u] = fmaxf(t[u], t[u + w]);
    }
    float x = t[0];
#pragma unroll
    for (int o = C::CPW; o < 64; o <<= 1) x = max_xor(x, o);
    return x;
  }

  __device__ __forceinline__ void shift(const Smem<C>& sm, int tt, int wave, int lane,
                                        float vmax) {
    const int jj = lane % C::CPW, g = lane / C::CPW;
    const int j = wave * C::CPW + jj;
    const float mx = vmax * bl;  // bl > 0: max of beta*v*log2e
    cnew = (mx > cold + kColLag) ? mx : cold;
    sh = kBias - cnew;
    eh = sm.base + pin(C::OFF_EH + (tt & 1) * C::EB + j * C::EROW * 2 + e_pos(4 * g) * 2);
    float* sink = sm.sink() + lane;
    *(g == 0 ? sm.c(tt & 1) + j : sink) = cnew;
    *(g == 0 ? sm.g(tt & 1) + j : sink) = exp2_hw(cold - cnew);
    const int rose = __any(cnew != cold) ? 1 : 0;
    *(lane == 0 ? sm.upd(tt & 1) + wave : reinterpret_cast<int*>(sink)) = rose;
  }

  // E of key 4(g + G u) + b in two stages, placed one slot apart: the exponent,
  // then 2^exponent.
  __device__ __forceinline__ void value_arg(int u, int b) {
    e[u][b] = MODE == kMean ? v[u][b] : fmaf(v[u][b], bl, sh);
  }
  __device__ __forceinline__ void value_exp(int u, int b) {
    if (MODE != kMean) e[u][b] = exp2_hw(e[u][b]);
  }

  // with_lo: this wave's columns take the lo product (wave-uniform)
  __device__ __forceinline__ void store(int u, bool with_lo) {
    static_assert(e_pos_splits(C::G), "tilt write positions");
    if (MODE == kMean) {  // bf16 values: the truncation is exact
      const u32x2 v2 = {pack_hi16(e[u][0], e[u][1]), pack_hi16(e[u][2], e[u][3])};
      *reinterpret_cast<u32x2*>(eh + e_pos(4 * C::G * u) * 2) = v2;
      return;
    }
    if (!with_lo) {
      const bf16x2 h01 = to_bf16x2(e[u][0], e[u][1]), h23 = to_bf16x2(e[u][2], e[u][3]);
      const u32x2 h2 = {__builtin_bit_cast(unsigned, h01), __builtin_bit_cast(unsigned, h23)};
      *reinterpret_cast<u32x2*>(eh + e_pos(4 * C::G * u) * 2) = h2;
      return;
    }
    float lo[4];
#pragma unroll
    for (int b = 0; b < 4; ++b)
      lo[b] = e[u][b] - __uint_as_float(__float_as_uint(e[u][b]) & 0xffff0000u);
    const u32x2 hi2 = {pack_hi16(e[u][0], e[u][1]), pack_hi16(e[u][2], e[u][3])};
    const bf16x2 l01 = to_bf16x2(lo[0], lo[1]), l23 = to_bf16x2(lo[2], lo[3]);
    const u32x2 lo2 = {__builtin_bit_cast(unsigned, l01), __builtin_bit_cast(unsigned, l23)};
    *reinterpret_cast<u32x2*>(eh + e_pos(4 * C::G * u) * 2) = hi2;
    *reinterpret_cast<u32x2*>(eh + (C::OFF_EL - C::OFF_EH) + e_pos(4 * C::G * u) * 2) = lo2;
  }
};

// Online softmax of one tile's scores (entry (kb, i) of sc holds key
// k0 + kb*32 + (i>>2)*8 + hl*4 + (i&3) of this lane's row), as placeable
// steps: mask (diagonal tile only), a three-level max tree, the lazy row-max
// update, and the probabilities of one pair of entries of k-step ks into the
// MFMA B-operand registers.
struct Softmax {
  float t1[11], t2[4], mx;

  template <bool MASK>
  __device__ __forceinline__ void mask(f32x16 (&sc)[2], int k0, int tq, int hl) {
    if (MASK) {
      // entry (kb, i) holds key k0 + hl*4 + r(kb, i); it is in the past of
      // row tq iff r <= lim.  Keys at or past T are past every row below T.
      const int lim = tq - k0 - hl * 4;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int r = kb * 32 + (i >> 2) * 8 + (i & 3);
          if (r > lim) sc[kb][i] = -INFINITY;
        }
      }
    }
  }
  __device__ __forceinline__ static float at(const f32x16 (&sc)[2], int e) {
    return sc[e >> 4][e & 15];
  }
  // level 1, entries [0, 15) or [15, 32) of the 32
  __device__ __forceinline__ void max1(const f32x16 (&sc)[2], int half) {
    if (half == 0) {
#pragma unroll
      for (int q = 0; q < 5; ++q)
        t1[q] = fmaxf(fmaxf(at(sc, 3 * q), at(sc, 3 * q + 1)), at(sc, 3 * q + 2));
    } else {
#pragma unroll
      for (int q = 5; q < 10; ++q)
        t1[q] = fmaxf(fmaxf(at(sc, 3 * q), at(sc, 3 * q + 1)), at(sc, 3 * q + 2));
      t1[10] = fmaxf(at(sc, 30), at(sc, 31));
    }
  }
  __device__ __forceinline__ void max2() {
    t2[0] = fmaxf(fmaxf(t1[0], t1[1]), t1[2]);
    t2[1] = fmaxf(fmaxf(t1[3], t1[4]), t1[5]);
    t2[2] = fmaxf(fmaxf(t1[6], t1[7]), t1[8]);
    t2[3] = fmaxf(t1[9], t1[10]);
    mx = fmaxf(fmaxf(t2[0], t2[1]), fmaxf(t2[2], t2[3]));
  }
  // scores stay raw (q.k) up to here; scale2 > 0 so the max commutes with it
  __device__ __forceinline__ void update(float& m, float& apend, float scale2) {
    const float x = fmaxf(mx, other_half(mx)) * scale2;
    const float mnew = (x > m + kRowLag) ? x : m;
    apend = (mnew == m) ? 1.f : exp2_hw(m - mnew);
    m = mnew;
  }
  // The probabilities of pair q (k-step q / 4, entries 2 (q % 4), +1) in three
  // stages, placed one slot apart so that no stage waits on the one before:
  // the exponents, 2^exponent, and the rounding into the MFMA B operand.
  __device__ __forceinline__ static void prob_arg(const f32x16 (&sc)[2], f32x2& x, int q, float m,
                                                  float scale2) {
    const int ks = q >> 2, u = 2 * (q & 3), kb = ks >> 1, s0 = (ks & 1) * 8;
    x[0] = fmaf(sc[kb][s0 + u], scale2, -m);
    x[1] = fmaf(sc[kb][s0 + u + 1], scale2, -m);
  }
  __device__ __forceinline__ static void prob_exp(f32x2& x) {
    x[0] = exp2_hw(x[0]);
    x[1] = exp2_hw(x[1]);
  }
  __device__ __forceinline__ static void prob_round(const f32x2& x, bf16x8 (&p)[4], int q) {
    const int ks = q >> 2, u = 2 * (q & 3);
    const bf16x2 p2 = to_bf16x2(x[0], x[1]);
    p[ks][u] = p2[0];
    p[ks][u + 1] = p2[1];
  }
};

// Direct global -> LDS copy of one K or V tile (rows k0 .. k0+63, padded rows).
// Wave w writes 1 KiB blocks w, w+NW, ...; lane l of a block fills slot
// 64*blk + l, i.e. row slot/SPR, chunk slot%SPR (the pad chunk re-reads chunk
// 0).  The lane offset inside the tile is the same for every tile and is
// computed once.
template <int W, int NW>
__device__ __forceinline__ unsigned tile_offset(int u, int wave, int lane) {
  constexpr int SPR = (W + 8) / 8;  // 16-byte slots per padded row
  const int slot = (wave + NW * u) * 64 + lane;
  const int row = slot / SPR, chunk = slot % SPR;
  return (unsigned)(row * W + (chunk < W / 8 ? chunk * 8 : 0)) * 2u;
}

// Block u of this wave's share of a tile: the direct load, if the tile has it.
// rsrc covers the rows k0 .. T-1 of the head, so rows at or past T load as
// zeros (their keys are masked; the tilt leaves them out of the column max).
// wave_s is the wave index held as a scalar and dst the LDS byte address of
// the tile buffer, so the block's LDS address and the test are scalar work;
// off is the lane offset inside the tile, the same for every tile.
template <int W, int NW>
__device__ __forceinline__ void load_block(rsrc_t rsrc, unsigned dst, int wave_s, int u,
                                           unsigned off) {
  constexpr int BLOCKS = 64 * ((W + 8) / 8) / 64;
  const int blk = wave_s + NW * u;
  if (BLOCKS % NW == 0 || blk < BLOCKS) dma16b(rsrc, off, dst + (unsigned)blk * 1024u);
}

__device__ __forceinline__ void wait_vmem() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// Phase 1 of an iteration, interleaved by hand with the tilt of tile k (QKT):
// on the matrix pipe, S^T = K Q^T of tile k into s (QKT), then the row-sum
// products and k-step 0 of PV(k-1) (PVA; the lo product for the first NLO
// column blocks only).  Slot st issues MFMA st, the LDS
// read of the operand fragment RING steps ahead, one stage of the tilt and
// whatever side(st) adds (the next tile's direct loads); a scheduling
// barrier after every slot keeps this order.  The tilt's stages sit one
// slot apart (exponent, 2^, rounding and store), so no vector instruction
// waits on a result from its own slot.
//
// Row sums: a 16x16x32 product of a constant 0/1 selector (lsel) with the
// same P^T fragments.  Lane l supplies selector row l%16 over k-block l/16;
// the B operand's k-block b holds query (l%16) + 16*(b%2), so a one in row
// m = 4r for the k-blocks with b%2 == r%2 sums query (l%16) + 16*(r%2) into
// output row 4r, which the 16x16 output layout places in register 0 of lane
// 16r + l%16.  Hence lacc[0] of every lane is the row sum of its query l%32.
template <class C, int NLO, bool PVA, bool QKT, class Side>
__device__ __forceinline__ void phase1(const Smem<C>& sm, Tilt<C>& tl, int k, int nvalid, int wave, int lane,
                                       int kofs, int eofs, int vcol, const bf16x8 (&qf)[C::NKS],
                                       f32x16 (&s)[2], f32x16 (&acc)[C::NCB], f32x4& lacc,
                                       const bf16x8 (&pp)[4], const bf16x8& lsel, Side&& side) {
  constexpr int MODE = C::MODE;
  static_assert(NLO >= 0 && NLO <= C::NCB && (MODE != kMean || NLO == 0), "lo blocks");
  constexpr int NQ = QKT ? 2 * C::NKS : 0;    // QK MFMAs
  constexpr int NL = PVA ? 4 : 0;             // row-sum MFMAs
  constexpr int NE = PVA ? C::NCB + NLO : 0;  // PV k-step 0: hi blocks, then lo blocks
  constexpr int NF = NQ + NE;                 // LDS operand fragments, in issue order
  constexpr int NS = NQ + NL + NE;
  constexpr int RING = 4;
  constexpr int NV = QKT ? C::RPL * 4 : 0;    // tilt values of the lane
  // Tilt stages: column max at CM (late enough for the V reads issued at the
  // start of the phase to have landed), shift at CM + 1, then value x's
  // exponent at V0 + x, its 2^ one slot later, and run u's store one slot
  // after its last 2^.
  constexpr int CM = 4;
  constexpr int V0 = CM + 2;
  constexpr int NVS = NV > 0 ? V0 + NV + 2 : 0;
  constexpr int NSLOT = NS > NVS ? NS : NVS;
  if (QKT) tl.read(sm, k, nvalid, wave, lane, vcol);
  const bool lo = wave * C::CPW < 32 * NLO;  // this wave's columns take the lo product
  const unsigned char* kt = sm.base + pin(C::OFF_K + (k & 1) * C::KB + kofs);
  const unsigned char* eb = sm.base + (PVA ? pin(C::OFF_EH + ((k - 1) & 1) * C::EB + eofs) : 0u);
  auto frag = [&](int f) -> bf16x8 {
    if (f < NQ)
      return *reinterpret_cast<const bf16x8*>(kt + (f & 1) * 32 * C::KROW * 2 + (f >> 1) * 32);
    const int e = f - NQ;
    const int lo = e >= C::NCB ? 1 : 0, cb = lo ? e - C::NCB : e;
    return *reinterpret_cast<const bf16x8*>(eb + lo * (C::OFF_EL - C::OFF_EH) +
                                            cb * 32 * C::EROW * 2);
  };
  bf16x8 ring[RING];
#pragma unroll
  for (int f = 0; f < RING; ++f)
    if (f < NF) ring[f] = frag(f);
  if (QKT) {
    s[0] = f32x16{};
    s[1] = f32x16{};
  }
  __builtin_amdgcn_sched_barrier(0);
  float vmax = 0.f;
#pragma unroll
  for (int st = 0; st < NSLOT; ++st) {
    if (st < NQ || (st >= NQ + NL && st < NS)) {
      const int f = st < NQ ? st : st - NL;
      const bf16x8 a = ring[f % RING];
      if (f + RING < NF) ring[f % RING] = frag(f + RING);
      if (f < NQ) {
        s[f & 1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[f >> 1], s[f & 1], 0, 0, 0);
      } else {
        const int e = f - NQ, cb = e >= C::NCB ? e - C::NCB : e;
        acc[cb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pp[0], acc[cb], 0, 0, 0);
      }
    } else if (st >= NQ && st < NQ + NL) {
      lacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(lsel, pp[st - NQ], lacc, 0, 0, 0);
    }
    side(st);
    if (QKT) {
      if (MODE != kMean && st == CM) vmax = tl.colmax();
      if (MODE != kMean && st == CM + 1) tl.shift(sm, k, wave, lane, vmax);
      const int xa = st - V0, xe = xa - 1, xs = xa - 5;  // values at each stage
      if (xa >= 0 && xa < NV) tl.value_arg(xa >> 2, xa & 3);
      if (xe >= 0 && xe < NV) tl.value_exp(xe >> 2, xe & 3);
      if (xs >= 0 && (xs & 3) == 0 && (xs >> 2) < C::RPL) tl.store(xs >> 2, lo);
    }
    __builtin_amdgcn_sched_barrier(0);
  }
}

// Phase 2 of an iteration: k-steps 1..3 of PV(k-1) (PVB; hi blocks, then the
// NLO lo blocks of each k-step), reading P(k-1)
// from pp, interleaved by hand with the softmax of this tile (SM; MASK on the
// wave's diagonal tile and the tiles after it), which writes P(k) into the
// other buffer pn.  The softmax's stages sit one slot apart as in phase 1.
template <class C, int NLO, bool PVB, bool SM, bool MASK>
__device__ __forceinline__ void phase2(const Smem<C>& sm, f32x16 (&acc)[C::NCB],
                                       const bf16x8 (&pp)[4], bf16x8 (&pn)[4], f32x16 (&sc)[2],
                                       float& m, float& apend, int j, int eofs, int k0, int tq,
                                       int hl, float scale2) {
  static_assert(NLO >= 0 && NLO <= C::NCB && (C::MODE != kMean || NLO == 0), "lo blocks");
  constexpr int NPK = C::NCB + NLO;                   // fragments per k-step
  constexpr int NF = PVB ? 3 * NPK : 0;               // k-steps 1..3
  constexpr int RING = 4;
  // Softmax stages: the max tree in slots 0..2, the row-max update in 3, then
  // pair q's exponents at P0 + q, its 2^ one slot later and its rounding into
  // the next P buffer one slot after that.
  constexpr int P0 = 4;
  constexpr int NSS = SM ? P0 + 16 + 2 : 0;
  constexpr int NSLOT = NF > NSS ? NF : NSS;
  const unsigned char* eb = sm.base + (PVB ? pin(C::OFF_EH + (j & 1) * C::EB + eofs) : 0u);
  auto frag = [&](int f) -> bf16x8 {
    const int ks = 1 + f / NPK, rem = f % NPK;
    const int lo = rem >= C::NCB ? 1 : 0, cb = lo ? rem - C::NCB : rem;
    return *reinterpret_cast<const bf16x8*>(eb + lo * (C::OFF_EL - C::OFF_EH) +
                                            cb * 32 * C::EROW * 2 + ks * 32);
  };
  bf16x8 ring[RING];
#pragma unroll
  for (int f = 0; f < RING; ++f)
    if (f < NF) ring[f] = frag(f);
  Softmax smx;
  f32x2 px[16];
  if (SM) smx.mask<MASK>(sc, k0, tq, hl);
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int st = 0; st < NSLOT; ++st) {
    if (st < NF) {
      const bf16x8 a = ring[st % RING];
      if (st + RING < NF) ring[st % RING] = frag(st + RING);
      const int ks = 1 + st / NPK, rem = st % NPK, cb = rem >= C::NCB ? rem - C::NCB : rem;
      acc[cb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pp[ks], acc[cb], 0, 0, 0);
    }
    if (SM) {
      if (st == 0) smx.max1(sc, 0);
      if (st == 1) smx.max1(sc, 1);
      if (st == 2) smx.max2();
      if (st == 3) smx.update(m, apend, scale2);
      const int qa = st - P0, qe = qa - 1, qr = qa - 2;  // pairs at each stage
      if (qa >= 0 && qa < 16) Softmax::prob_arg(sc, px[qa], qa, m, scale2);
      if (qe >= 0 && qe < 16) Softmax::prob_exp(px[qe]);
      if (qr >= 0 && qr < 16) Softmax::prob_round(px[qr], pn, qr);
    }
    __builtin_amdgcn_sched_barrier(0);
  }
}

// Number of channels of one head whose beta needs the lo product (the same
// value in every lane).
template <class C>
__device__ __forceinline__ int lo_channels(const float* hbeta, int lane) {
  int n = 0;
#pragma unroll
  for (int c0 = 0; c0 < C::DV; c0 += 64) {
    const int j = c0 + lane;
    n += __popcll(__ballot(j < C::DV && !(hbeta[j] >= kLoBeta)));
  }
  return n;
}

// Number of set bits of m below this lane.
__device__ __forceinline__ int bits_below(uint64_t m) {
  return (int)__builtin_amdgcn_mbcnt_hi((unsigned)(m >> 32),
                                        __builtin_amdgcn_mbcnt_lo((unsigned)m, 0u));
}

// The read of one workgroup (a block of BQ query rows of one head) whose
// first NLO accumulator column blocks take the lo product.  With 0 < NLO <
// NCB the columns hold the head's channels reordered: the nlo channels with
// beta below kLoBeta first, then the others, each group in input order.
template <class C, int NLO>
__device__ __forceinline__ void read_body(
    const bf16* __restrict__ Q, const bf16* __restrict__ K, const bf16* __restrict__ V,
    const float* __restrict__ beta, const float* lam, const float* gate, float* out,
    float* __restrict__ lse, int H, int T, int nqb, int nbh, unsigned char* smem, int nneed) {
  constexpr int MODE = C::MODE;
  constexpr bool SPLIT = NLO > 0 && NLO < C::NCB;  // columns hold reordered channels
  const Smem<C> sm{smem};

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int n = lane & 31;   // query column of this lane in the 32x32 blocks
  const int hl = lane >> 5;  // lane half

  const int bid = blockIdx.x;
  const int qblk = nqb - 1 - bid / nbh;  // longest causal extent first
  const int bh = bid % nbh;
  const int h = bh % H;
  const int q0 = qblk * C::BQ;
  const size_t baseq = (size_t)bh * T * C::DK;  // Q, K
  const size_t base = (size_t)bh * T * C::DV;   // V, out, lam, gate
  const bf16* Qh = Q + baseq;
  const bf16* Kh = K + baseq;
  const bf16* Vh = V + base;
  float* Oh = out + base;
  bf16* Ob = reinterpret_cast<bf16*>(out) + base;

  if (!SPLIT) {
    for (int j = tid; j < C::DV; j += C::NT) {
      const float bl = beta[h * C::DV + j] * kLog2e;
      sm.bl()[j] = bl;
      sm.inv()[j] = 1.f / bl;
    }
  } else if (wave == 0) {
    // column of channel j: its rank among the channels of its group, after
    // the nlo channels that need the lo product if it does not
    int below_lo = 0, below_hi = 0;
#pragma unroll
    for (int c0 = 0; c0 < C::DV; c0 += 64) {
      const int j = c0 + lane;
      const bool valid = j < C::DV;
      const float b = valid ? beta[h * C::DV + j] : 1.f;
      const bool need = valid && !(b >= kLoBeta);
      const uint64_t mlo = __ballot(need), mhi = __ballot(valid && !need);
      const int col = need ? below_lo + bits_below(mlo) : nneed + below_hi + bits_below(mhi);
      if (valid) {
        sm.chan()[col] = j;
        sm.bl()[col] = b * kLog2e;
        sm.inv()[col] = 1.f / (b * kLog2e);
      }
      below_lo += __popcll(mlo);
      below_hi += __popcll(mhi);
    }
  }

  const int wq0 = q0 + wave * 32;  // first query row of this wave
  const int tq = wq0 + n;          // this lane's query row
  const bool wave_live = wq0 < T;
  const int qlast = min(q0 + C::BQ, T) - 1;
  // last key a lane's row may see: its own row (causal) or the last key
  const int tm = C::CAUSAL ? tq : T - 1;
  const int ntiles = (C::CAUSAL ? qlast : T - 1) / C::BK + 1;
  // The first masked tile.  Causal: the tile holding the wave's diagonal (the
  // wave's first row is a multiple of 32, which divides the tile size, so
  // earlier tiles lie wholly below the wave's rows); encoder read: the last
  // tile, whose keys at or past T are masked.
  const int wlast = !wave_live ? -1
                    : C::CAUSAL ? min((wq0 + 31) / C::BK, ntiles - 1)
                                : ntiles - 1;

  // the wave index as a scalar and the LDS byte address of the tile
  // buffers, for the direct loads' addresses
  const int wave_s = __builtin_amdgcn_readfirstlane(wave);
  const unsigned lds0 = lds_addr(smem);
  // lane offsets of a full K / V tile (the same for every tile)
  unsigned koff[C::BPWK], voff[C::BPWV];
#pragma unroll
  for (int u = 0; u < C::BPWK; ++u) koff[u] = tile_offset<C::DK, C::NW>(u, wave, lane);
#pragma unroll
  for (int u = 0; u < C::BPWV; ++u)
    voff[u] = C::SAME ? koff[u] : tile_offset<C::DV, C::NW>(u, wave, lane);
  // rows k0 .. T-1 of the head's K and V
  auto krsrc = [&](int k0) { return buffer_rsrc(Kh + (size_t)k0 * C::DK, (unsigned)(T - k0) * C::DK * 2u); };
  auto vrsrc = [&](int k0) { return buffer_rsrc(Vh + (size_t)k0 * C::DV, (unsigned)(T - k0) * C::DV * 2u); };
  auto kload = [&](int u, const rsrc_t& r, int buf) {
    load_block<C::DK, C::NW>(r, lds0 + C::OFF_K + buf * C::KB, wave_s, u, koff[u]);
  };
  auto vload = [&](int u, const rsrc_t& r, int buf) {
    load_block<C::DV, C::NW>(r, lds0 + C::OFF_V + buf * C::VB, wave_s, u, voff[u]);
  };
  {
    const rsrc_t rk = krsrc(0), rv = vrsrc(0);
#pragma unroll
    for (int u = 0; u < C::BPWK; ++u) kload(u, rk, 0);
#pragma unroll
    for (int u = 0; u < C::BPWV; ++u) vload(u, rv, 0);
  }
  bf16x8 qf[C::NKS];
#pragma unroll
  for (int ks = 0; ks < C::NKS; ++ks) {
    bf16x8 z = {};
    qf[ks] = (tq < T)
                 ? *reinterpret_cast<const bf16x8*>(Qh + (size_t)tq * C::DK + ks * 16 + hl * 8)
                 : z;
  }
  wait_vmem();
  __syncthreads();
  // input channel of this lane's tilt column
  const int vcol = SPLIT ? sm.chan()[wave * C::CPW + lane % C::CPW] : wave * C::CPW + lane % C::CPW;

  f32x16 acc[C::NCB];
#pragma unroll
  for (int cb = 0; cb < C::NCB; ++cb) acc[cb] = f32x16{};
  f32x16 sacc[2] = {f32x16{}, f32x16{}};  // scores of the current tile
  // probabilities, double-buffered: softmax(k) writes tile k's into buffer
  // k & 1 while PV(k-1) reads buffer (k-1) & 1
  bf16x8 pbuf[2][4] = {};
  float m = -INFINITY;  // running row max (log2 units), shared by the lane pair
  float apend = 1.f;    // row rescale owed to the accumulator before the next PV
  f32x4 lacc = {};      // lacc[0]: row sum of the rounded P (see phase2)
  bf16x8 lsel;
  {
    const int r = lane & 15, b = lane >> 4;
    const __bf16 one = ((r & 3) == 0 && ((r >> 2) & 1) == (b & 1)) ? (__bf16)1.f : (__bf16)0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) lsel[e] = one;
  }
  const float scale2 = kLog2e / sqrtf((float)C::DK);
  const int kofs = n * C::KROW * 2 + hl * 16;  // lane part of K fragment addresses
  const int eofs = n * C::EROW * 2 + hl * 16;  // lane part of E fragment addresses

  // Direct loads of tile k+1 into the free K and V buffers.
  auto load_next = [&](int k) {
    const int kn = (k + 1) * C::BK;
    const rsrc_t rk = krsrc(kn), rv = vrsrc(kn);
#pragma unroll
    for (int u = 0; u < C::BPWK; ++u) kload(u, rk, (k + 1) & 1);
#pragma unroll
    for (int u = 0; u < C::BPWV; ++u) vload(u, rv, (k + 1) & 1);
  };
  // The same loads spread over the MFMA slots of phase 1, one per slot from
  // slot LD0 on (K blocks, then V blocks), so that the waves of a workgroup
  // do not all wait on the memory pipeline at once.
  constexpr int LD0 = 2;
  auto loads_in_slots = [&](int k) {
    const bool more = k + 1 < ntiles;
    const int kn = (k + 1) * C::BK;
    const rsrc_t rk = krsrc(kn), rv = vrsrc(kn);
    return [=](int st) __attribute__((always_inline)) {
      if (!more) return;
      const int u = st - LD0, w = u - C::BPWK;
      if (u >= 0 && u < C::BPWK) kload(u, rk, (k + 1) & 1);
      if (w >= 0 && w < C::BPWV) vload(w, rv, (k + 1) & 1);
    };
  };
  // Deferred rescales owed before PV(j): the row factor of softmax(j) and the
  // column factors of tilt(j) (flag word from upd(j)).
  auto rescale = [&](int j, const i32x4& any4) {
    const bool col = MODE != kMean && (any4[0] | any4[1] | any4[2] | any4[3]) != 0;
    if (col || __any(apend != 1.f)) {
      const float* gcol = sm.g(j & 1);
#pragma unroll
      for (int cb = 0; cb < C::NCB; ++cb) {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          f32x4 gg = {apend, apend, apend, apend};
          if (col) gg *= *reinterpret_cast<const f32x4*>(gcol + cb * 32 + g * 8 + hl * 4);
#pragma unroll
          for (int e = 0; e < 4; ++e) acc[cb][g * 4 + e] *= gg[e];
          // one group of factors at a time: this runs where the scores and
          // the tilt's values are live
          __builtin_amdgcn_sched_barrier(0);
        }
      }
      lacc[0] *= apend;
    }
  };
  auto flags_of = [&](int j) {
    if (MODE == kMean) return i32x4{};  // no column shift
    const i32x4* uf = reinterpret_cast<const i32x4*>(sm.upd(j & 1));
    i32x4 any4 = uf[0];
#pragma unroll
    for (int w = 1; w < C::NW / 4; ++w) any4 |= uf[w];
    return any4;
  };
#define FEM_PHASE1(PVA, QKT, PPREV, SIDE)                                                   \
  phase1<C, NLO, PVA, QKT>(sm, tl, k, T - k * C::BK, wave, lane, kofs, eofs, vcol, qf, sacc, acc, lacc, PPREV, \
                           lsel, SIDE)
  const auto none = [](auto...) __attribute__((always_inline)) {};
#define FEM_PHASE2(PVB, SM, MK, PPREV, PNEXT)                                                    \
  phase2<C, NLO, PVB, SM, MK>(sm, acc, PPREV, PNEXT, sacc, m, apend, k - 1, eofs, k * C::BK, tm, \
                              hl, scale2)

  // Every wave runs the same steps on every tile: past its diagonal tile the
  // softmax masks every key, so P = 0 and PV adds nothing, while the
  // accumulator keeps following the shared column shift to the last tile.
  // Iteration k: loads of tile k+1; rescales owed before PV(k-1); phase 1:
  // row sums + PV(k-1) k-step 0 + QK(k) || tilt(k); phase 2: PV(k-1) k-steps
  // 1..3 || softmax(k); one barrier.
  {
    const int k = 0;
    if (k + 1 < ntiles) load_next(k);
    Tilt<C> tl;
    FEM_PHASE1(false, true, pbuf[1], none);
    if (wlast <= 0) FEM_PHASE2(false, true, true, pbuf[1], pbuf[0]);
    else FEM_PHASE2(false, true, false, pbuf[1], pbuf[0]);
    wait_vmem();
    __syncthreads();
  }
  // iteration k; PAR = k & 1 is a compile-time constant so that the P
  // buffers stay in registers
  auto body = [&](const int k, auto par) __attribute__((always_inline)) {
    constexpr int PAR = decltype(par)::value;
    // the flag words' LDS reads go out first; their latency hides behind
    // the load issue
    if (k > 1) rescale(k - 1, flags_of(k - 1));
    Tilt<C> tl;
    // A wave in phase 1 issues ahead of the other wave of its SIMD in phase
    // 2: the QK products then run while the other wave does its softmax on
    // the vector unit, and the two waves reach the barrier closer together.
    __builtin_amdgcn_s_setprio(1);
    FEM_PHASE1(true, true, pbuf[PAR ^ 1], loads_in_slots(k));
    __builtin_amdgcn_s_setprio(0);
    if (k >= wlast) FEM_PHASE2(true, true, true, pbuf[PAR ^ 1], pbuf[PAR]);
    else FEM_PHASE2(true, true, false, pbuf[PAR ^ 1], pbuf[PAR]);
    wait_vmem();
    __syncthreads();
  };
  int kk = 1;
  for (; kk + 1 < ntiles; kk += 2) {
    body(kk, std::integral_constant<int, 1>());
    body(kk + 1, std::integral_constant<int, 0>());
  }
  if (kk < ntiles) body(kk, std::integral_constant<int, 1>());
  auto tail = [&](auto par) __attribute__((always_inline)) {
    constexpr int PAR = decltype(par)::value;  // parity of the last tile
    const int k = ntiles;
    if (k > 1) rescale(k - 1, flags_of(k - 1));
    Tilt<C> tl;
    FEM_PHASE1(true, false, pbuf[PAR], none);
    FEM_PHASE2(true, false, false, pbuf[PAR], pbuf[PAR]);
  };
  if ((ntiles - 1) & 1) tail(std::integral_constant<int, 1>());
  else tail(std::integral_constant<int, 0>());
#undef FEM_PHASE1
#undef FEM_PHASE2

  // With reordered channels the outputs go through LDS (the tile buffers are
  // free once every wave is done with the last tile) so that the rows reach
  // memory in channel order with whole-row stores.
  constexpr bool STAGE = SPLIT;
  constexpr int SROW = C::DV + 4;  // staged row stride (floats)
  static_assert(!STAGE || C::NW * 32 * SROW * 4 <= C::OFF_F, "staging must not reach the tables");
  if (STAGE) __syncthreads();
  float* stage = reinterpret_cast<float*>(smem) + wave * 32 * SROW;

  if (!wave_live) return;

  if (MODE == kMean) {  // ---- mu = acc / l
    if (tq >= T) return;
    const float rl = 1.f / lacc[0];
#pragma unroll
    for (int cb = 0; cb < C::NCB; ++cb) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int ch0 = cb * 32 + g * 8 + hl * 4;
        f32x4 o;
#pragma unroll
        for (int e = 0; e < 4; ++e) o[e] = acc[cb][g * 4 + e] * rl;
        *reinterpret_cast<f32x4*>(Oh + (size_t)tq * C::DV + ch0) = o;
      }
    }
    return;
  }

  // ---- epilogue: o = (log2(acc / l) - bias + c) / (beta log2 e) with one
  // logarithm per output.  acc / l is a weighted mean of E = 2^(x - c +
  // bias); it is scaled by 2^-bias (exactly) before the logarithm, so that
  // the argument lies near 1 and the logarithm keeps its absolute precision
  // (tiny beta amplifies any error here).  Outputs whose acc fell below
  // 2^-64, or whose scaled mean is not a normal float, are flagged for the
  // exact repair below.
  static_assert(kBias == 64.f, "the scale below is 2^-bias");
  const float lt = lacc[0];
  // the prior's log-normaliser ln sum_i exp(q.k_i / sqrt d), for a backward pass
  if (MODE == kFem && lse && hl == 0 && tq < T) lse[(size_t)bh * T + tq] = (m + log2_hw(lt)) * kLn2;
  const float rl = 0x1p-64f / lt;
  const float* cw = sm.c((ntiles - 1) & 1);  // the accumulator's final column frame
  const float* inv = sm.inv();
  const float* Lh = MODE == kGated ? lam + base : nullptr;
  const float* Gh = MODE == kGated && gate ? gate + base : nullptr;
  const auto low = [&](float a) { return !(a >= kUnderflow && a * rl >= 0x1p-120f); };
  uint64_t flags = 0;
  {
    float amin = INFINITY;
#pragma unroll
    for (int cb = 0; cb < C::NCB; ++cb)
#pragma unroll
      for (int i = 0; i < 16; ++i) amin = fminf(amin, acc[cb][i]);
    if (__ballot(low(amin) && tq < T) != 0) {  // rare: find the flagged outputs
#pragma unroll
      for (int cb = 0; cb < C::NCB; ++cb)
#pragma unroll
        for (int i = 0; i < 16; ++i)
          if (low(acc[cb][i]) && tq < T) flags |= 1ull << (cb * 16 + i);
    }
  }
#pragma unroll
  for (int cb = 0; cb < C::NCB; ++cb) {
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int ch0 = cb * 32 + g * 8 + hl * 4;
      f32x4 o;
#pragma unroll
      for (int e = 0; e < 4; ++e)
        o[e] = (log2_hw(acc[cb][g * 4 + e] * rl) + cw[ch0 + e]) * inv[ch0 + e];
      if (STAGE) {  // into the staged row at the channel's own column
        const i32x4 oc = SPLIT ? *reinterpret_cast<const i32x4*>(sm.chan() + ch0)
                               : i32x4{ch0, ch0 + 1, ch0 + 2, ch0 + 3};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          // the gated mix keeps mu where F underflowed (NaN marks those)
          const bool flagged = (flags >> (cb * 16 + g * 4 + e)) & 1ull;
          stage[n * SROW + oc[e]] = MODE == kGated && flagged ? __builtin_nanf("") : o[e];
        }
        continue;
      }
      if (tq >= T) continue;
      const size_t at = (size_t)tq * C::DV + ch0;
      if (MODE == kGated) {
        // mu from the kMean launch; an underflowed F keeps mu in place for
        // the exact path below
        const f32x4 mu = *reinterpret_cast<const f32x4*>(Oh + at);
        const f32x4 lm = *reinterpret_cast<const f32x4*>(Lh + at);
        const f32x4 gg = Gh ? *reinterpret_cast<const f32x4*>(Gh + at) : f32x4{1.f, 1.f, 1.f, 1.f};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const bool flagged = (flags >> (cb * 16 + g * 4 + e)) & 1ull;
          o[e] = flagged ? mu[e] : gg[e] * fmaf(lm[e], o[e] - mu[e], mu[e]);
        }
      }
      if (C::OBF16) {
        const bf16x2 o01 = to_bf16x2(o[0], o[1]), o23 = to_bf16x2(o[2], o[3]);
        const u32x2 ob = {__builtin_bit_cast(unsigned, o01), __builtin_bit_cast(unsigned, o23)};
        *reinterpret_cast<u32x2*>(Ob + at) = ob;
      } else {
        *reinterpret_cast<f32x4*>(Oh + at) = o;
      }
    }
  }

  if (STAGE) {
    // whole rows: lane l stores channels 4 (l % LPR) .. +3 of row l / LPR of
    // each group of RPI rows
    constexpr int LPR = C::DV / 4, RPI = 64 / LPR;
    const int c4 = (lane % LPR) * 4;
#pragma unroll
    for (int r0 = 0; r0 < 32; r0 += RPI) {
      const int r = r0 + lane / LPR, t = wq0 + r;
      f32x4 o = *reinterpret_cast<const f32x4*>(stage + r * SROW + c4);
      if (t >= T) continue;
      const size_t at = (size_t)t * C::DV + c4;
      if (MODE == kGated) {
        const f32x4 mu = *reinterpret_cast<const f32x4*>(Oh + at);
        const f32x4 lm = *reinterpret_cast<const f32x4*>(Lh + at);
        const f32x4 gg = Gh ? *reinterpret_cast<const f32x4*>(Gh + at) : f32x4{1.f, 1.f, 1.f, 1.f};
#pragma unroll
        for (int e = 0; e < 4; ++e)
          o[e] = o[e] != o[e] ? mu[e] : gg[e] * fmaf(lm[e], o[e] - mu[e], mu[e]);
      }
      if (C::OBF16) {
        const bf16x2 o01 = to_bf16x2(o[0], o[1]), o23 = to_bf16x2(o[2], o[3]);
        const u32x2 ob = {__builtin_bit_cast(unsigned, o01), __builtin_bit_cast(unsigned, o23)};
        *reinterpret_cast<u32x2*>(Ob + at) = ob;
      } else {
        *reinterpret_cast<f32x4*>(Oh + at) = o;
      }
    }
  }

  // ---- rare path: exact recompute of accumulators that underflowed, one
  // row at a time (its flags sit in lanes n and n + 32), up to kRepairBatch
  // of its channels per pass over the keys, so that a row's scores are
  // formed once per batch rather than once per channel
  if (__ballot(flags != 0) == 0) return;
  wait_vmem();  // the epilogue's stores above (the gated mix reads mu back)
  while (true) {
    const uint64_t who = __ballot(flags != 0);
    if (who == 0) break;
    const int r = __builtin_ctzll(who) & 31;
    const int t = __builtin_amdgcn_readlane(tq, r);
    uint64_t fw[2];  // the row's flag words: channels of lane half 0 and 1
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const uint32_t flo = __builtin_amdgcn_readlane((uint32_t)flags, r + 32 * h);
      const uint32_t fhi = __builtin_amdgcn_readlane((uint32_t)(flags >> 32), r + 32 * h);
      fw[h] = ((uint64_t)fhi << 32) | flo;
    }
    while ((fw[0] | fw[1]) != 0) {
      int chs[kRepairBatch];
      float bls[kRepairBatch];
      int nb = 0, mych = 0;
#pragma unroll
      for (int c = 0; c < kRepairBatch; ++c) {
        chs[c] = 0;
        bls[c] = 1.f;
        if ((fw[0] | fw[1]) == 0) continue;
        const int h = fw[0] != 0 ? 0 : 1;
        const int e = __builtin_ctzll(fw[h]);
        fw[h] &= fw[h] - 1;
        const int cb = e >> 4, i = e & 15;
        const int col = cb * 32 + (i >> 2) * 8 + h * 4 + (i & 3);
        chs[c] = SPLIT ? sm.chan()[col] : col;  // input channel
        bls[c] = sm.bl()[col];
        nb = c + 1;
        if (lane == c) mych = chs[c];
      }
      const float o = exact_row<C, kRepairBatch>(Qh, Kh, Vh, t, C::CAUSAL ? t + 1 : T, chs, bls, nb,
                                                 scale2);
      if (lane < nb) {
        const size_t at = (size_t)t * C::DV + mych;
        if (MODE == kGated) {
          const float mu = Oh[at];
          Oh[at] = (Gh ? Gh[at] : 1.f) * fmaf(Lh[at], o - mu, mu);
        } else if (C::OBF16) {
          Ob[at] = (bf16)o;
        } else {
          Oh[at] = o;
        }
      }
    }
    if ((lane & 31) == r) flags = 0;
  }
}

// Dispatch on the number of column blocks that take the lo product.
template <class C, int N, class... A>
__device__ __forceinline__ void read_nlo(int nlo, A... a) {
  if constexpr (N == C::NCB) {
    read_body<C, N>(a...);
  } else {
    if (nlo == N) read_body<C, N>(a...);
    else read_nlo<C, N + 1>(nlo, a...);
  }
}

template <class C>
__global__ __launch_bounds__(C::NT) void softmax_bf16_kernel(
    const bf16* __restrict__ Q, const bf16* __restrict__ K, const bf16* __restrict__ V,
    const float* __restrict__ beta, const float* lam, const float* gate, float* out,
    float* __restrict__ lse, int H, int T, int nqb, int nbh) {
  __shared__ __align__(16) unsigned char smem[C::LDS];
  if constexpr (C::MODE == kMean) {
    read_body<C, 0>(Q, K, V, beta, lam, gate, out, lse, H, T, nqb, nbh, smem, 0);
  } else {
    const int h = (int)(blockIdx.x % (unsigned)nbh) % H;
    const int nneed = lo_channels<C>(beta + h * C::DV, threadIdx.x & 63);
    read_nlo<C, 0>((nneed + 31) >> 5, Q, K, V, beta, lam, gate, out, lse, H, T, nqb, nbh, smem,
                   nneed);
  }
}

template <class C>
hipError_t launch(const void* Q, const void* K, const void* V, const float* beta,
                  const float* lam, const float* gate, void* out, int B, int H, int T,
                  hipStream_t stream, float* lse = nullptr) {
  const int nqb = (T + C::BQ - 1) / C::BQ;
  const int nbh = B * H;
  dim3 grid((unsigned)(nqb * nbh)), block(C::NT);
  hipLaunchKernelGGL((softmax_bf16_kernel<C>), grid, block, 0, stream,
                     reinterpret_cast<const bf16*>(Q), reinterpret_cast<const bf16*>(K),
                     reinterpret_cast<const bf16*>(V), beta, lam, gate,
                     reinterpret_cast<float*>(out), lse, H, T, nqb, nbh);
  return hipGetLastError();
}

template <int D>
hipError_t launch_gated(const void* Q, const void* K, const void* V, const float* beta_max,
                        const float* lam, const float* gate, float* out, int B, int H, int T,
                        hipStream_t stream) {
  hipError_t e =
      launch<Cfg<D, D, 8, kMean>>(Q, K, V, beta_max, nullptr, nullptr, out, B, H, T, stream);
  if (e != hipSuccess) return e;
  return launch<Cfg<D, D, 8, kGated>>(Q, K, V, beta_max, lam, gate, out, B, H, T, stream);
}

// The variants of the plain read: widths (d_qk, d_v), causal or encoder
// read, fp32 or bf16 output.
template <int DK, int DV>
hipError_t launch_ex(const void* Q, const void* K, const void* V, const float* beta, void* out,
                     int B, int H, int T, bool causal, bool obf16, hipStream_t stream) {
  if (causal && !obf16)
    return launch<Cfg<DK, DV, 8, kFem, true, false>>(Q, K, V, beta, nullptr, nullptr, out, B, H,
                                                     T, stream);
  if (causal)
    return launch<Cfg<DK, DV, 8, kFem, true, true>>(Q, K, V, beta, nullptr, nullptr, out, B, H,
                                                    T, stream);
  if (!obf16)
    return launch<Cfg<DK, DV, 8, kFem, false, false>>(Q, K, V, beta, nullptr, nullptr, out, B, H,
                                                      T, stream);
  return launch<Cfg<DK, DV, 8, kFem, false, true>>(Q, K, V, beta, nullptr, nullptr, out, B, H, T,
                                                   stream);
}

}  // namespace

hipError_t launch_softmax_bf16(const void* Q, const void* K, const void* V, const float* beta,
                               float* out, int B, int H, int T, int d, hipStream_t stream) {
  return launch_softmax_ex_bf16(Q, K, V, beta, out, B, H, T, d, d, true, false, stream);
}

hipError_t launch_softmax_ex_bf16(const void* Q, const void* K, const void* V, const float* beta,
                                  void* out, int B, int H, int T, int dk, int dv, bool causal,
                                  bool obf16, hipStream_t stream) {
  const auto go = [&](auto f) { return f(Q, K, V, beta, out, B, H, T, causal, obf16, stream); };
  if (dk == 32 && dv == 32) return go(launch_ex<32, 32>);
  if (dk == 64 && dv == 64) return go(launch_ex<64, 64>);
  if (dk == 128 && dv == 128) return go(launch_ex<128, 128>);
  if (dk == 64 && dv == 32) return go(launch_ex<64, 32>);
  if (dk == 128 && dv == 64) return go(launch_ex<128, 64>);
  return hipErrorInvalidValue;
}

hipError_t launch_softmax_train_bf16(const void* Q, const void* K, const void* V,
                                     const float* beta, float* out, float* lse, int B, int H,
                                     int T, int d, hipStream_t stream) {
  switch (d) {
    case 32:
      return launch<Cfg<32, 32, 8, kFem>>(Q, K, V, beta, nullptr, nullptr, out, B, H, T, stream, lse);
    case 64:
      return launch<Cfg<64, 64, 8, kFem>>(Q, K, V, beta, nullptr, nullptr, out, B, H, T, stream, lse);
    case 128:
      return launch<Cfg<128, 128, 8, kFem>>(Q, K, V, beta, nullptr, nullptr, out, B, H, T, stream,
                                            lse);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_softmax_gated_bf16(const void* Q, const void* K, const void* V,
                                     const float* beta_max, const float* lam, const float* gate,
                                     float* out, int B, int H, int T, int d, hipStream_t stream) {
  switch (d) {
    case 32: return launch_gated<32>(Q, K, V, beta_max, lam, gate, out, B, H, T, stream);
    case 64: return launch_gated<64>(Q, K, V, beta_max, lam, gate, out, B, H, T, stream);
    case 128: return launch_gated<128>(Q, K, V, beta_max, lam, gate, out, B, H, T, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace fem
