/*
 * fem.h -- C ABI of the MI355X Free Energy Mixer (FEM) read library (libfem.so).
 *
 * The library computes the FEM free-energy read of "Free Energy Mixer"
 * (Lu & Yang, ICLR 2026): for every batch b, head h, step t and channel j,
 *
 *     F[b,h,t,j] = (1 / beta[h,j]) * log  sum_{i <= t}  p_t(i) * exp(beta[h,j] * v[b,h,i,j])
 *
 * (Sec. 2.3, free-energy read, eq. fem-free-energy-main), over a causal prior
 * p_t on the support {0, ..., t} (0-based, diagonal included):
 *
 *   fem_softmax_fwd:  p_t(i) = softmax_{i <= t}( q_t . k_i / sqrt(d) )
 *                     (Sec. 1, masked scores; Appendix "Parameterizations of
 *                      the Prior Selection", softmax prior, with no bias term)
 *   fem_linear_fwd:   p_t(i) = <phi(q_t), phi(k_i)> / sum_{r <= t} <phi(q_t), phi(k_r)>,
 *                     phi = elu + 1  (Appendix "Selection distributions,
 *                      support, and normalization", linear attention)
 *   fem_gla_fwd:      the decay-gated linear (GLA) prior of the appendix
 *                     "Gated Linear Attention (GLA) Prior"
 *
 * and the two-level gated read of the paper's models, which mixes F at a
 * per-channel beta_max with the prior's expectation (fem_softmax_gated_fwd).
 *
 * Conventions shared by every entry point:
 *   - Every tensor argument is a DEVICE pointer (HIP device memory, e.g.
 *     torch tensors' data_ptr()).  The caller owns every buffer; the library
 *     keeps no pointer after the call returns.
 *   - The library allocates no memory and holds no global state, so calls
 *     are thread-safe and re-entrant.  An entry point that needs scratch
 *     memory takes a caller-provided workspace `ws` of `ws_bytes` bytes
 *     (device memory, 256-byte aligned) and has a query,
 *     fem_*_workspace_bytes(...), that returns the exact size it needs for
 *     the given sizes (0: none, and `ws` may be NULL).  The workspace holds
 *     intermediate results only until the call's kernels have run on
 *     `stream`; it needs no initialisation, and calls that run at the same
 *     time need workspaces of their own.
 *   - Layout: contiguous row-major [B, H, T, width] (width fastest); Q, K, V
 *     16-byte aligned.  beta is [H, width_v] float32, shared over B and T.
 *   - out is always float32 [B, H, T, width_v] and must not alias an input.
 *   - Calls are asynchronous on `stream` (a hipStream_t; 0 is the null
 *     stream): they return after enqueueing the kernels.  Launch errors are
 *     reported as FEM_ERR_HIP; errors of the kernels themselves surface at the
 *     caller's next synchronisation.
 *   - Every argument check is made on the host before anything is launched;
 *     on error nothing is launched and `out` is untouched.  The library never
 *     aborts, throws or prints.
 *   - Preconditions that are NOT checked (they would need a device read):
 *     beta finite and > 0 (the read is defined for beta > 0 only, Sec. 2.3)
 *     and all inputs finite.  Violations give unspecified values; NaN inputs
 *     propagate.
 */
#ifndef FEM_H
#define FEM_H

#include <stddef.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Element type of Q, K and V.  beta and out are always float32. */
typedef enum {
  FEM_DTYPE_F32 = 0,
  FEM_DTYPE_BF16 = 1
} fem_dtype;

typedef enum {
  FEM_OK = 0,
  FEM_ERR_NULLPTR = 1,      /* a required pointer is NULL                      */
  FEM_ERR_SHAPE = 2,        /* B, H or T <= 0, or a size overflows             */
  FEM_ERR_UNSUPPORTED = 3,  /* width, chunk or dtype outside the supported set */
  FEM_ERR_ALIGN = 4,        /* a tensor argument is not 16-byte aligned, or ws
                               is not 256-byte aligned                         */
  FEM_ERR_HIP = 5,          /* a HIP call or kernel launch failed              */
  FEM_ERR_WORKSPACE = 6     /* ws is NULL or ws_bytes is below the workspace
                               query's value                                   */
} fem_status;

/*
 * Causal softmax-prior FEM read (Sec. 2.3 with the softmax prior of Sec. 1).
 *
 *   Q, K, V : [B, H, T, d], element type `dtype`
 *   beta    : [H, d] float32, > 0
 *   out     : [B, H, T, d] float32
 *   d       : 32, 64 or 128 for FEM_DTYPE_BF16 (matrix-core path);
 *             any 1 <= d <= 256 for FEM_DTYPE_F32 (exact vector path)
 *
 * Score scale is fixed at 1/sqrt(d).  Returns a fem_status.
 */
int fem_softmax_fwd(const void* Q, const void* K, const void* V,
                    const float* beta, float* out,
                    int B, int H, int T, int d, int dtype, hipStream_t stream);

/* Option bits of fem_softmax_fwd_ex. */
typedef enum {
  FEM_FLAG_ENCODER = 1,  /* no causal mask: every query sees all T keys       */
  FEM_FLAG_OUT_BF16 = 2  /* out is bfloat16 (round to nearest even), not fp32 */
} fem_flags;

/*
 * Variants of the softmax-prior read (same definition as fem_softmax_fwd):
 *
 *   - FEM_FLAG_ENCODER: the encoder read, p_t(i) = softmax over every i < T
 *     (encoder-only use removes the mask; Sec. "Empirical Evaluation").
 *   - d_v != d_qk: budget (i) of Sec. "Free Energy Mixer" gives the values
 *     half the key width.  The score scale stays 1/sqrt(d_qk).
 *   - FEM_FLAG_OUT_BF16: bf16 output.  Its rounding adds up to 2^-9 |o| to
 *     the read's own error.
 *
 *   Q, K     : [B, H, T, d_qk] bfloat16
 *   V        : [B, H, T, d_v] bfloat16
 *   beta     : [H, d_v] float32, > 0
 *   out      : [B, H, T, d_v], float32 or (FEM_FLAG_OUT_BF16) bfloat16
 *   (d_qk, d_v): (32, 32), (64, 64), (128, 128), (64, 32) or (128, 64)
 *   flags    : an OR of fem_flags; other bits return FEM_ERR_UNSUPPORTED
 *   dtype    : FEM_DTYPE_BF16
 *
 * With flags = 0 and d_qk = d_v this is fem_softmax_fwd's bf16 path.
 * Returns a fem_status.
 */
int fem_softmax_fwd_ex(const void* Q, const void* K, const void* V,
                       const float* beta, void* out,
                       int B, int H, int T, int d_qk, int d_v, int flags,
                       int dtype, hipStream_t stream);

/*
 * One decoding step of the softmax-prior read against a KV cache: for every
 * (b, h) the new query q[b,h] reads the first lens[b] cached keys and values,
 * which include the new token's own k and v (the autoregressive KV-cache
 * setting, Appendix "Parameterizations of the Prior Selection"):
 *
 *   out[b,h,j] = (1/beta[h,j]) log sum_{i < lens[b]} p(i) exp(beta[h,j] v[b,h,i,j]),
 *   p(i) = softmax_{i < lens[b]}( q[b,h] . k[b,h,i] / sqrt(d_qk) )
 *
 * i.e. row lens[b]-1 of fem_softmax_fwd when q is that row's query.
 *
 *   q      : [B, H, d_qk] bfloat16
 *   Kc     : [B, H, L, d_qk] bfloat16 key cache (rows >= lens[b] are not read)
 *   Vc     : [B, H, L, d_v] bfloat16 value cache
 *   lens   : [B] int32 DEVICE array, each in [1, L]; NULL means L for every b.
 *            A length outside [1, L] is not an error on the host (it would
 *            need a device read): that sequence's outputs are NaN.
 *   beta   : [H, d_v] float32, > 0
 *   out    : [B, H, d_v] float32
 *   (d_qk, d_v): as fem_softmax_fwd_ex
 *   dtype  : FEM_DTYPE_BF16
 *
 * fp32 arithmetic with a per-channel joint log-sum-exp (no shared shift).
 * The keys are split over workgroups: S = ceil(L / (64 n)) splits of n =
 * ceil(ceil(L / 64) / s0) key blocks of 64 each, s0 = min(ceil(256 / (B H)),
 * ceil(L / 64)).  Their partial results need a workspace of
 *
 *   fem_softmax_decode_workspace_bytes(B, H, L, d_qk, d_v) = 8 * B * H * S * (d_v + 1)
 *
 * bytes (0 for arguments outside the supported set).  Returns a fem_status.
 */
size_t fem_softmax_decode_workspace_bytes(int B, int H, int L, int d_qk, int d_v);

int fem_softmax_decode(const void* q, const void* Kc, const void* Vc,
                       const int* lens, const float* beta, float* out,
                       int B, int H, int L, int d_qk, int d_v, int dtype,
                       void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * fem_softmax_decode for callers that cannot allocate device memory at all:
 * code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc.  Same arguments, result and kernels as fem_softmax_decode,
 * without ws / ws_bytes: the partial results live in a fixed array of 8 MiB
 * in the library's device code, one per device, kept until the process
 * ends.  The call allocates nothing; its first call on a device looks the
 * array's address up (hipGetSymbolAddress) with that device current.
 *
 * Limit: sizes whose fem_softmax_decode_workspace_bytes(...) exceeds
 * 8 MiB (8388608 bytes) return FEM_ERR_WORKSPACE; e.g. d_v = 128 allows
 * B * H up to 8128 at any L.  Every call on one device shares that device's
 * array: calls that overlap in time on one device (different streams, or
 * different host threads) race and give undefined results.  Returns a
 * fem_status.
 */
int fem_softmax_decode_noalloc(const void* q, const void* Kc, const void* Vc,
                               const int* lens, const float* beta, float* out,
                               int B, int H, int L, int d_qk, int d_v, int dtype,
                               hipStream_t stream);

/*
 * Training pair of the causal softmax-prior read (bf16 inputs, d = 32, 64 or
 * 128).
 *
 * fem_softmax_fwd_train: fem_softmax_fwd that also writes
 *   lse[b,h,t] = ln sum_{i <= t} exp(q_t . k_i / sqrt d)      [B, H, T] float32,
 * the prior's log-normaliser, which the backward pass reads.
 *
 * fem_softmax_bwd: gradients of L = sum dout * out from the paper's closed
 * forms (posterior as the value gradient, Proposition "Local geometry" /
 * eq. app-grad-hess; (q - p)/beta as the normalized-logit gradient, prior
 * sensitivity (iv); KL(q || p)/beta^2 as the temperature derivative, eq.
 * app-beta-deriv):
 *   Q, K, V, beta  : the forward's inputs
 *   out, lse       : the forward's outputs (fem_softmax_fwd_train)
 *   dout           : [B, H, T, d] float32, dL/dout
 *   dQ, dK, dV     : [B, H, T, d] float32, overwritten
 *   dbeta          : [H, d] float32, overwritten (summed over batch and time)
 * The posterior ratio R = exp(beta (v_i - out_t)) is factorised as
 * E_i U_t per channel (one shift per channel over the sequence), so the sums
 * over keys and channels run on the matrix cores (bf16 hi + lo parts,
 * ~2^-16 relative); channels whose beta-scaled value range is at most
 * 4 / log2(e) use the cancellation-free form R - 1 = (E - 1) U + (U - 1).
 * A channel (b, h, j) whose range beta (max v - min v) over the sequence
 * exceeds 110 / log2(e) would leave fp32's exponent range: an element-wise
 * pass, exact in form for every beta > 0, takes that channel and adds its
 * part of dQ and dK (at B8 H16 T4096 d128, one such channel in every batch
 * of one head costs ~8 ms on top of ~6.4 ms).  Should a factor of another
 * channel still leave fp32's range (an output gradient near 2^100), the
 * element-wise pass redoes the whole call (~34x slower).  dbeta is
 * formed from the normalised posterior sums, so the forward's rounding of
 * out cancels from it.  The passes exchange intermediate results through a
 * workspace of
 *
 *   fem_softmax_bwd_workspace_bytes(B, H, T, d) =
 *       256 + round_up_256(4 * (B H T + 2 B H d + 5 B H n d + B H T d + B H Tp))
 *           + 8 * B H Tp d,        n = ceil(T / 64), Tp = 64 n
 *
 * bytes (about 12 B H T d: at B8 H16 T4096 d128, 829 MB; 0 for arguments
 * outside the supported set).  All pointers 16-byte aligned; outputs must not
 * alias inputs.  Returns a fem_status.
 */
int fem_softmax_fwd_train(const void* Q, const void* K, const void* V,
                          const float* beta, float* out, float* lse,
                          int B, int H, int T, int d, int dtype, hipStream_t stream);

size_t fem_softmax_bwd_workspace_bytes(int B, int H, int T, int d);

int fem_softmax_bwd(const void* Q, const void* K, const void* V,
                    const float* beta, const float* out, const float* lse,
                    const float* dout, float* dQ, float* dK, float* dV, float* dbeta,
                    int B, int H, int T, int d, int dtype,
                    void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * Two-level gated FEM read with the causal softmax prior (Sec. "Two-Level
 * Gated FEM", eqs. inner-gate-main and fem-two-gates-main; the inner gate is
 * the linearized temperature learning of eqs. ltl and ltl-final):
 *
 *   o[b,h,t,j]  = g[b,h,t,j] * ( (1 - lam[b,h,t,j]) * mu[b,h,t,j]
 *                                + lam[b,h,t,j] * F[b,h,t,j] )
 *   mu[b,h,t,j] = sum_{i <= t} p_t(i) * v[b,h,i,j]      (expectation baseline)
 *   F[b,h,t,j]  = the read of fem_softmax_fwd at beta = beta_max[h,j]
 *
 *   Q, K, V  : [B, H, T, d] bfloat16, d = 32, 64 or 128
 *   beta_max : [H, d] float32, > 0
 *   lam      : [B, H, T, d] float32, the inner (temperature) gate; meant to
 *              lie in [0, 1] (not checked: other values extrapolate linearly)
 *   gate     : [B, H, T, d] float32, the outer gate (> 0 in the paper's
 *              parameterization; any finite value is applied as given), or
 *              NULL for g = 1
 *   out      : [B, H, T, d] float32; must alias none of the inputs
 *   dtype    : FEM_DTYPE_BF16
 *
 * lam, gate (when given) and out must be 16-byte aligned.  Two kernels run
 * in order on `stream`; the first leaves mu in `out` for the second, so out
 * holds partial results until the second has run.  Returns a fem_status.
 */
int fem_softmax_gated_fwd(const void* Q, const void* K, const void* V,
                          const float* beta_max, const float* lam, const float* gate,
                          float* out, int B, int H, int T, int d, int dtype,
                          hipStream_t stream);

/*
 * Causal linear-prior FEM read, phi = elu + 1, as an O(T) chunked scan
 * (Appendix "Parameterizations of the Prior Selection": associative-scan
 * form with a constant channel appended to the values for the normaliser;
 * no decay and no feature scaling).
 *
 *   Q, K    : [B, H, T, d_k], element type `dtype`
 *   V       : [B, H, T, d_v], element type `dtype`
 *   beta    : [H, d_v] float32, > 0
 *   out     : [B, H, T, d_v] float32
 *   d_k, d_v: 64 (both)
 *   chunk   : length of the intra-chunk (quadratic) block of the scan: 16, 32,
 *             64 or 128.  A query sees the keys of its own chunk through the
 *             masked product phi(Q_c) phi(K_c)^T and every earlier key
 *             through the carried state.  The chunk only schedules the work:
 *             the result does not depend on it beyond rounding.  Other
 *             values return FEM_ERR_UNSUPPORTED.
 *   dtype   : FEM_DTYPE_BF16
 *
 * The scan runs over tiles of L = max(chunk, 32) tokens (chunk 16: two
 * chunks per tile) in segments of c = ceil(n / w) tiles, n = ceil(T / L),
 * w = max(1, floor(512 / (B H))), S = ceil(n / c) segments per (b, h).
 * With S > 1 the segments' own states and the states entering them need a
 * workspace of
 *
 *   fem_linear_workspace_bytes(B, H, T, d_k, d_v, chunk) = 2 * 4 * B * H * S * 4224
 *
 * bytes (a state is the 64 x 64 matrix, the 64-entry normaliser and the 64
 * channel shifts, 4224 floats); with S = 1 it is 0 and ws may be NULL.  0 is
 * also returned for arguments outside the supported set.
 *
 * Returns a fem_status.
 */
size_t fem_linear_workspace_bytes(int B, int H, int T, int d_k, int d_v, int chunk);

int fem_linear_fwd(const void* Q, const void* K, const void* V,
                   const float* beta, float* out,
                   int B, int H, int T, int d_k, int d_v, int chunk,
                   int dtype, void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * Causal GLA-prior FEM read as an O(T) chunked scan (Appendix "Gated Linear
 * Attention (GLA) Prior", eqs. gla-score-appendix and gla-assoc):
 *
 *   p_t(i) = sum_c q~[t,c] k~[i,c] exp(sum_{tau=i+1}^{t} g[tau,c]) / Z_t,  i <= t,
 *   q~ = ReLU(RoPE(q)) + 1e-6, k~ likewise,
 *
 * with the read of fem_linear_fwd on top.  RoPE rotates the pair of
 * dimensions (2m, 2m+1) of position t by t * 10000^(-2m/d_k); the decay is
 * per key channel c (a scalar or per-head decay is the same value repeated).
 *
 *   Q, K    : [B, H, T, d_k] bfloat16
 *   V       : [B, H, T, d_v] bfloat16
 *   G       : [B, H, T, d_k] float32 log-decays, each in [-2, 0]
 *             (precondition, not checked: it would need a device read).
 *             g <= 0 is the paper's decay; the floor, a decay factor of at
 *             least e^-2 per step, keeps every factor of the 64-token chunk
 *             form inside float range.  Values outside the domain are
 *             clamped into it, so the result is then not the read of the
 *             given decays
 *   beta    : [H, d_v] float32, > 0
 *   out     : [B, H, T, d_v] float32
 *   d_k, d_v: 64 (both);  chunk: 64 (the decay factors of a chunk stay
 *             inside float range for 64 tokens);  dtype: FEM_DTYPE_BF16
 *
 * Workspace as fem_linear_fwd at chunk 64, each state carrying also its
 * segment's total log-decay per key channel (4288 floats):
 *
 *   fem_gla_workspace_bytes(B, H, T, d_k, d_v, chunk) = 2 * 4 * B * H * S * 4288
 *
 * for S > 1, else 0.  Returns a fem_status.
 */
size_t fem_gla_workspace_bytes(int B, int H, int T, int d_k, int d_v, int chunk);

int fem_gla_fwd(const void* Q, const void* K, const void* V, const float* G,
                const float* beta, float* out,
                int B, int H, int T, int d_k, int d_v, int chunk,
                int dtype, void* ws, size_t ws_bytes, hipStream_t stream);

/* Static, NUL-terminated name of a status code (never NULL). */
const char* fem_status_str(int status);

#ifdef __cplusplus
}
#endif

#endif /* FEM_H */
