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
//   phase 1: QK^T(k) on the matrix pipe  ||  tilt of the wave's channels of
//            tile k on the vector pipe;
//   phase 2: PV(k-1) (hi, lo and the row-sum product)  ||  softmax of tile k
//            (the scores phase 1 just produced).
// The instruction order of each phase is pinned with scheduling barriers.  Row
// and column rescales of the accumulator are rare; they are deferred to just
// before the next PV so that neither phase needs a branch.  softmax(k)
// overwrites the P registers behind PV(k-1) as it issues.  K(k+1) and
// V(k+1) stream straight into the free LDS buffers (global_load_lds_dwordx4)
// during iteration k; K, V and E are double buffered.  Workgroups run longest
// causal extent first; workgroup i of a causal level covers head i, so a
// head's workgroups share an XCD.

#include "fem_device.h"
#include "fem_internal.h"


namespace fem {
namespace {

constexpr float kBias = 64.f;        // E = 2^(x - c + kBias) <= 2^(kBias + kColLag)
constexpr float kColLag = 16.f;      // column shift raised only past this lag
constexpr float kRowLag = 8.f;       // row max raised only past this lag (P <= 2^8)
constexpr float kUnderflow = 0x1p-64f;

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
  static constexpr int NF = DV /*bl*/ + DV /*inv*/ + 2 * DV /*c*/ + 2 * DV /*g*/ + 64 /*sink*/;
  static constexpr int OFF_R = OFF_F + NF * 4;    // column-update flags [2][NW]
  // tile-load lane offsets [NW][64][TW]: K tile, then V tile unless SAME
  static constexpr int OFF_T = OFF_R + 2 * NW * 4;
  static constexpr int TWK = (BPWK + 3) / 4 * 4;
  static constexpr int TW = TWK + (SAME ? 0 : (BPWV + 3) / 4 * 4);
  static constexpr size_t LDS = OFF_T + NW * 64 * TW * 4;
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

// Exact fp32 read of one (t, j) by the whole wave: joint log-sum-exp of
// (score + tilt) over the keys i < n, minus the log-sum-exp of the scores.
template <class C>
__device__ float exact_read(const bf16* __restrict__ Qh, const bf16* __restrict__ Kh,
                            const bf16* __restrict__ Vh, int t, int n, int j, float scale2,
                            float bl) {
  const int lane = threadIdx.x & 63;
  Lse2 num, den;
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
    num.add(s + (float)Vh[(size_t)i * C::DV + j] * bl);
  }
  return (num.wave_total() - den.wave_total()) / bl;
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
  __device__ int* upd(int b) const { return reinterpret_cast<int*>(base + C::OFF_R) + b * C::NW; }
  // this lane's offsets of a whole K tile; those of a V tile follow unless SAME
  __device__ unsigned* ltab(int w, int l) const {
    return reinterpret_cast<unsigned*>(base + C::OFF_T) + (w * 64 + l) * C::TW;
  }
  __device__ unsigned* ltabv(int w, int l) const { return ltab(w, l) + (C::SAME ? 0 : C::TWK); }
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
//   read    : this lane's V values (channel jj, 4-key runs g + G*u), beta and
//             the previous column shift, all from LDS;
//   colmax  : column max over the tile (a tree in-lane, then across the G
//             lanes of a channel);
//   shift   : lazily raised running shift c_j; stores c, the rescale factor
//             g = 2^(c_old - c_new) and the wave's "some c rose" flag;
//   value(u, b), store(u) : E = 2^(x - c + bias) of key 4(g + G u) + b split
//             into bf16 hi (truncated) and lo (the rounded remainder), and the
//             store of run u into the E^T buffers.
// Keys at or past T (last tile only) hold copies of row T-1 (see load_tile):
// they leave the column max unchanged and give finite E, which meet P = 0
// (the causal mask), so the tilt treats every tile as full.
// Stores that only one lane of a group should make go to a sink slot from the
// other lanes, so the code has no branches.
template <class C>
struct Tilt {
  static constexpr int MODE = C::MODE;
  float v[C::RPL][4];
  float e[C::RPL][4];
  float bl, cold, cnew, sh;
  unsigned char* eh;

  __device__ __forceinline__ void read(const Smem<C>& sm, int tt, int wave, int lane) {
    const int jj = lane % C::CPW, g = lane / C::CPW;
    const int j = wave * C::CPW + jj;
    const unsigned char* sv =
        sm.base + pin(C::OFF_V + (tt & 1) * C::VB + j * 2 + 4 * g * C::VROW * 2);
#pragma unroll
    for (int u = 0; u < C::RPL; ++u) {
#pragma unroll
      for (int b = 0; b < 4; ++b)
        v[u][b] = (float)*reinterpret_cast<const bf16*>(sv + (4 * C::G * u + b) * C::VROW * 2);
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

  __device__ __forceinline__ void value(int u, int b) {
    e[u][b] = MODE == kMean ? v[u][b] : exp2_hw(fmaf(v[u][b], bl, sh));
  }

  __device__ __forceinline__ void store(int u) {
    static_assert(e_pos_splits(C::G), "tilt write positions");
    if (MODE == kMean) {  // bf16 values: the truncation is exact
      const u32x2 v2 = {pack_hi16(e[u][0], e[u][1]), pack_hi16(e[u][2], e[u][3])};
      *reinterpret_cast<u32x2*>(eh + e_pos(4 * C::G * u) * 2) = v2;
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
  __device__ __forceinline__ static void probs(const f32x16 (&sc)[2], bf16x8& p, int ks, int u,
                                               float m, float scale2) {
    const int kb = ks >> 1, s0 = (ks & 1) * 8;
    const bf16x2 p2 = to_bf16x2(exp2_hw(fmaf(sc[kb][s0 + u], scale2, -m)),
                                exp2_hw(fmaf(sc[kb][s0 + u + 1], scale2, -m)));
    p[u] = p2[0];
    p[u + 1] = p2[1];
  }
};

// Direct global -> LDS copy of one K or V tile (rows k0 .. k0+63, padded rows).
// Wave w writes 1 KiB blocks w, w+NW, ...; lane l of a block fills slot
// 64*blk + l, i.e. row slot/SPR, chunk slot%SPR (the pad chunk re-reads chunk
// 0).  Rows at or past T are clamped to T-1: their keys are masked anyway.
// The address is a uniform tile base plus a 32-bit lane offset, so the loads
// use scalar-base addressing.  The lane offsets of a whole tile (no clamping)
// are computed once into an LDS table (tile_offsets) and read back per tile,
// rather than held in registers across the loop.
template <int W, int NW>
__device__ __forceinline__ unsigned tile_offset(int u, int k0, int T, int wave, int lane) {
  constexpr int SPR = (W + 8) / 8;  // 16-byte slots per padded row
  const int slot = (wave + NW * u) * 64 + lane;
  const int row = min(slot / SPR, T - 1 - k0), chunk = slot % SPR;
  return (unsigned)(row * W + (chunk < W / 8 ? chunk * 8 : 0)) * 2u;
}

template <int BPW>
__device__ __forceinline__ void tile_offsets(const unsigned* t, unsigned* off) {
#pragma unroll
  for (int u = 0; u < BPW; ++u) off[u] = t[u];
}

template <int W, int NW, int BPW>
__device__ __forceinline__ void load_tile(const bf16* __restrict__ src, unsigned char* dst, int k0,
                                          int wave, const unsigned* off) {
  constexpr int BLOCKS = 64 * ((W + 8) / 8) / 64;
  const char* base = reinterpret_cast<const char*>(src + (size_t)k0 * W);
#pragma unroll
  for (int u = 0; u < BPW; ++u) {
    const int blk = wave + NW * u;
    if (BLOCKS % NW == 0 || blk < BLOCKS)
      dma16(base + off[u], dst + blk * 1024);
  }
}

__device__ __forceinline__ void wait_vmem() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// Phase 1 of an iteration, interleaved by hand with the tilt of tile k (QKT):
// on the matrix pipe, the row-sum products and k-step 0 of PV(k-1) (PVA),
// then S^T = K Q^T of tile k into s (QKT).  Slot st issues MFMA st, the LDS
// read of the operand fragment RING steps ahead and a fixed slice of the
// tilt; a scheduling barrier after every slot keeps this order.
//
// Row sums: a 16x16x32 product of a constant 0/1 selector (lsel) with the
// same P^T fragments.  Lane l supplies selector row l%16 over k-block l/16;
// the B operand's k-block b holds query (l%16) + 16*(b%2), so a one in row
// m = 4r for the k-blocks with b%2 == r%2 sums query (l%16) + 16*(r%2) into
// output row 4r, which the 16x16 output layout places in register 0 of lane
// 16r + l%16.  Hence lacc[0] of every lane is the row sum of its query l%32.
template <class C, bool PVA, bool QKT>
__device__ __forceinline__ void phase1(const Smem<C>& sm, Tilt<C>& tl, int k, int wave, int lane,
                                       int kofs, int eofs, const bf16x8 (&qf)[C::NKS],
                                       f32x16 (&s)[2], f32x16 (&acc)[C::NCB], f32x4& lacc,
                                       const bf16x8 (&pp)[4], const bf16x8& lsel) {
  constexpr int MODE = C::MODE;
  constexpr int NL = PVA ? 4 : 0;             // row-sum MFMAs
  constexpr int NLO = MODE == kMean ? 0 : C::NCB;  // lo blocks
  constexpr int NE = PVA ? C::NCB + NLO : 0;  // PV k-step 0: hi blocks, then lo blocks
  constexpr int NQ = QKT ? 2 * C::NKS : 0;    // QK MFMAs
  constexpr int NF = NE + NQ;                 // LDS operand fragments
  constexpr int NS = NL + NF;
  constexpr int RING = 4;
  constexpr int NV = QKT ? C::RPL * 4 : 0;    // tilt values of the lane
  constexpr int C0 = PVA ? 2 : 0;             // slot of the column max
  constexpr int NSLOT = NS > C0 + 2 + NV ? NS : C0 + 2 + NV;
  auto vslot = [&](int x) { return C0 + 2 + (x * (NSLOT - C0 - 2)) / (NV > 0 ? NV : 1); };
  if (QKT) tl.read(sm, k, wave, lane);
  const unsigned char* kt = sm.base + pin(C::OFF_K + (k & 1) * C::KB + kofs);
  const unsigned char* eb = sm.base + (PVA ? pin(C::OFF_EH + ((k - 1) & 1) * C::EB + eofs) : 0u);
  auto frag = [&](int f) -> bf16x8 {
    if (f < NE) {
      const int lo = f >= C::NCB ? 1 : 0, cb = lo ? f - C::NCB : f;
      return *reinterpret_cast<const bf16x8*>(eb + lo * (C::OFF_EL - C::OFF_EH) +
                                              cb * 32 * C::EROW * 2);
    }
    const int st = f - NE;
    return *reinterpret_cast<const bf16x8*>(kt + (st & 1) * 32 * C::KROW * 2 + (st >> 1) * 32);
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
    if (st < NL) {
      lacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(lsel, pp[st], lacc, 0, 0, 0);
    } else if (st < NS) {
      const int f = st - NL;
      const bf16x8 a = ring[f % RING];
      if (f + RING < NF) ring[f % RING] = frag(f + RING);
      if (f < NE) {
        const int cb = f >= C::NCB ? f - C::NCB : f;
        acc[cb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pp[0], acc[cb], 0, 0, 0);
      } else {
        const int q = f - NE;
        s[q & 1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[q >> 1], s[q & 1], 0, 0, 0);
      }
    }
    if (QKT) {
      if (MODE != kMean && st == C0) vmax = tl.colmax();
      if (MODE != kMean && st == C0 + 1) tl.shift(sm, k, wave, lane, vmax);
#pragma unroll
      for (int x = 0; x < NV; ++x) {
        if (vslot(x) == st) {
          tl.value(x >> 2, x & 3);
          if ((x & 3) == 3) tl.store(x >> 2);
        }
      }
    }
    __builtin_amdgcn_sched_barrier(0);
  }
}

// Phase 2 of an iteration: k-steps 1..3 of PV(k-1) (PVB), interleaved by hand
// with the softmax of this tile (SM; MASK on the wave's diagonal tile and the
// tiles after it).  One P buffer serves both products: an MFMA reads its
// operands when it issues, so the softmax writes the new P of k-step ks only
// in slots after the last MFMA that reads ks (k-step 0 was read in phase 1).
template <class C, bool PVB, bool SM, bool MASK>
__device__ __forceinline__ void phase2(const Smem<C>& sm, f32x16 (&acc)[C::NCB],
                                       bf16x8 (&pp)[4], f32x16 (&sc)[2], float& m, float& apend,
                                       int j, int eofs, int k0, int tq, int hl, float scale2) {
  constexpr int MODE = C::MODE;
  constexpr int NPK = MODE == kMean ? C::NCB : 2 * C::NCB;  // fragments per k-step
  constexpr int NF = PVB ? 3 * NPK : 0;               // k-steps 1..3
  constexpr int RING = 4;
  constexpr int NSLOT = NF > 8 ? NF : 8;
  // first slot free of reads of P k-step ks, then spread the 4 pairs
  auto pslot = [&](int ks, int u) {
    const int first = PVB ? NPK * ks : 0;
    const int sl = first + (u / 2) * (NPK >= 4 ? NPK / 4 : 1);
    return sl < 4 ? 4 + sl : sl;
  };
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
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
#pragma unroll
        for (int u = 0; u < 8; u += 2)
          if (pslot(ks, u) == st) Softmax::probs(sc, pp[ks], ks, u, m, scale2);
      }
    }
    __builtin_amdgcn_sched_barrier(0);
  }
  if (SM) {
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
#pragma unroll
      for (int u = 0; u < 8; u += 2)
        if (pslot(ks, u) >= NSLOT) Softmax::probs(sc, pp[ks], ks, u, m, scale2);
    }
  }
}

template <class C>
__global__ __launch_bounds__(C::NT) void softmax_bf16_kernel(
    const bf16* __restrict__ Q, const bf16* __restrict__ K, const bf16* __restrict__ V,
    const float* __restrict__ beta, const float* lam, const float* gate, float* out,
    float* __restrict__ lse, int H, int T, int nqb, int nbh) {
  constexpr int MODE = C::MODE;
  __shared__ __align__(16) unsigned char smem[C::LDS];
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

  for (int j = tid; j < C::DV; j += C::NT) {
    const float bl = beta[h * C::DV + j] * kLog2e;
    sm.bl()[j] = bl;
    sm.inv()[j] = 1.f / bl;
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

  {
    unsigned offk[C::BPWK], offv[C::BPWV];
#pragma unroll
    for (int u = 0; u < C::BPWK; ++u) {
      offk[u] = tile_offset<C::DK, C::NW>(u, 0, T, wave, lane);
      sm.ltab(wave, lane)[u] = tile_offset<C::DK, C::NW>(u, 0, 1 << 30, wave, lane);
    }
    if (!C::SAME) {
#pragma unroll
      for (int u = 0; u < C::BPWV; ++u) {
        offv[u] = tile_offset<C::DV, C::NW>(u, 0, T, wave, lane);
        sm.ltabv(wave, lane)[u] = tile_offset<C::DV, C::NW>(u, 0, 1 << 30, wave, lane);
      }
    }
    load_tile<C::DK, C::NW, C::BPWK>(Kh, sm.k(0), 0, wave, offk);
    load_tile<C::DV, C::NW, C::BPWV>(Vh, sm.v(0), 0, wave, C::SAME ? offk : offv);
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

  f32x16 acc[C::NCB];
#pragma unroll
  for (int cb = 0; cb < C::NCB; ++cb) acc[cb] = f32x16{};
  f32x16 sacc[2] = {f32x16{}, f32x16{}};  // scores of the current tile
  bf16x8 pp[4] = {};                      // probabilities: softmax(k) -> PV(k)
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

  // The lane offsets of the next tile's loads: the table, or clamped rows for
  // the last tile.
  auto next_offsets = [&](int k, unsigned* offk, unsigned* offv) {
    const int kn = (k + 1) * C::BK;
    if (kn + C::BK <= T) {
      tile_offsets<C::BPWK>(sm.ltab(wave, lane), offk);
      if (!C::SAME) tile_offsets<C::BPWV>(sm.ltabv(wave, lane), offv);
    } else {  // last tile: rows at or past T read row T-1
#pragma unroll
      for (int u = 0; u < C::BPWK; ++u) offk[u] = tile_offset<C::DK, C::NW>(u, kn, T, wave, lane);
      if (!C::SAME) {
#pragma unroll
        for (int u = 0; u < C::BPWV; ++u)
          offv[u] = tile_offset<C::DV, C::NW>(u, kn, T, wave, lane);
      }
    }
  };
  auto load_next = [&](int k, const unsigned* offk, const unsigned* offv) {
    const int kn = (k + 1) * C::BK;
    load_tile<C::DK, C::NW, C::BPWK>(Kh, sm.k((k + 1) & 1), kn, wave, offk);
    load_tile<C::DV, C::NW, C::BPWV>(Vh, sm.v((k + 1) & 1), kn, wave, C::SAME ? offk : offv);
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
#define FEM_PHASE1(PVA, QKT) \
  phase1<C, PVA, QKT>(sm, tl, k, wave, lane, kofs, eofs, qf, sacc, acc, lacc, pp, lsel)
#define FEM_PHASE2(PVB, SM, MK) \
  phase2<C, PVB, SM, MK>(sm, acc, pp, sacc, m, apend, k - 1, eofs, k * C::BK, tm, hl, scale2)

  // Every wave runs the same steps on every tile: past its diagonal tile the
  // softmax masks every key, so P = 0 and PV adds nothing, while the
  // accumulator keeps following the shared column shift to the last tile.
  // Iteration k: loads of tile k+1; rescales owed before PV(k-1); phase 1:
  // row sums + PV(k-1) k-step 0 + QK(k) || tilt(k); phase 2: PV(k-1) k-steps
  // 1..3 || softmax(k); one barrier.
  {
    const int k = 0;
    if (k + 1 < ntiles) {
      unsigned offk[C::BPWK], offv[C::BPWV];
      next_offsets(k, offk, offv);
      load_next(k, offk, offv);
    }
    Tilt<C> tl;
    FEM_PHASE1(false, true);
    if (wlast <= 0) FEM_PHASE2(false, true, true);
    else FEM_PHASE2(false, true, false);
    wait_vmem();
    __syncthreads();
  }
  for (int k = 1; k < ntiles; ++k) {
    // LDS reads of the flag words and the load offsets go out together
    const i32x4 any4 = flags_of(k - 1);
    if (k + 1 < ntiles) {
      unsigned offk[C::BPWK], offv[C::BPWV];
      next_offsets(k, offk, offv);
      load_next(k, offk, offv);
    }
    if (k > 1) rescale(k - 1, any4);
    Tilt<C> tl;
    FEM_PHASE1(true, true);
    if (k >= wlast) FEM_PHASE2(true, true, true);
    else FEM_PHASE2(true, true, false);
    wait_vmem();
    __syncthreads();
  }
  {
    const int k = ntiles;
    if (k > 1) rescale(k - 1, flags_of(k - 1));
    Tilt<C> tl;
    FEM_PHASE1(true, false);
    FEM_PHASE2(true, false, false);
  }
#undef FEM_PHASE1
#undef FEM_PHASE2

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

  // ---- epilogue: o = (log2 acc - log2 l + c - bias) / (beta log2 e).  The
  // logarithms are split into exponent and mantissa so the bias and the
  // integer parts cancel exactly (tiny beta amplifies any error here).
  const float lt = lacc[0];
  // the prior's log-normaliser ln sum_i exp(q.k_i / sqrt d), for a backward pass
  if (MODE == kFem && lse && hl == 0 && tq < T) lse[(size_t)bh * T + tq] = (m + log2_hw(lt)) * kLn2;
  int el;
  const float fl = log2_hw(frexpf(lt, &el));
  const float* cw = sm.c((ntiles - 1) & 1);  // the accumulator's final column frame
  const float* inv = sm.inv();
  const float* Lh = MODE == kGated ? lam + base : nullptr;
  const float* Gh = MODE == kGated && gate ? gate + base : nullptr;
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
    const float o = exact_read<C>(Qh, Kh, Vh, t, C::CAUSAL ? t + 1 : T, ch, scale2, sm.bl()[ch]);
    if (lane == src) {
      flags &= ~(1ull << e);
      const size_t at = (size_t)t * C::DV + ch;
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
