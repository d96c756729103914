// C ABI of libfem.so: argument validation and dispatch (declared in fem.h).

#include "fem.h"
#include "fem_internal.h"

#include <stdint.h>

namespace {

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Every [B, H, T, w] tensor must be indexable with 64-bit offsets and every
// grid dimension must fit the launch limits.
bool sizes_ok(int B, int H, int T, int w) {
  if (B <= 0 || H <= 0 || T <= 0 || w <= 0) return false;
  const unsigned long long n = (unsigned long long)B * H * T * w;
  if (n > (1ull << 46)) return false;
  if ((unsigned long long)B * H > 65535ull * 1024ull) return false;
  return true;
}

int from_hip(hipError_t e) { return e == hipSuccess ? FEM_OK : FEM_ERR_HIP; }

// A caller workspace of `need` bytes: present, large enough, 256-byte aligned.
int check_ws(const void* ws, size_t ws_bytes, size_t need) {
  if (need == 0) return FEM_OK;
  if (!ws || ws_bytes < need) return FEM_ERR_WORKSPACE;
  if ((reinterpret_cast<uintptr_t>(ws) & 255u) != 0) return FEM_ERR_ALIGN;
  return FEM_OK;
}

bool decode_pair_ok(int d_qk, int d_v) {
  return (d_qk == d_v && (d_v == 32 || d_v == 64 || d_v == 128)) ||
         (d_qk == 2 * d_v && (d_v == 32 || d_v == 64));
}

bool decode_sizes_ok(int B, int H, int L, int d_qk, int d_v) {
  return sizes_ok(B, H, L, d_qk) && sizes_ok(B, H, L, d_v) && (unsigned long long)B * H <= 65535ull;
}

// The linear scan takes chunks of 16, 32, 64 or 128 tokens; the GLA scan 64.
bool scan_args_ok(int B, int H, int T, int d_k, int d_v, int chunk, bool gla) {
  const bool chunk_ok = gla ? chunk == 64 : (chunk == 16 || chunk == 32 || chunk == 64 || chunk == 128);
  return sizes_ok(B, H, T, d_k) && sizes_ok(B, H, T, d_v) && d_k == 64 && d_v == 64 && chunk_ok;
}

bool bwd_args_ok(int B, int H, int T, int d) {
  return sizes_ok(B, H, T, d) && (unsigned long long)H <= 65535ull &&
         (d == 32 || d == 64 || d == 128);
}

}  // namespace

extern "C" int fem_softmax_fwd(const void* Q, const void* K, const void* V, const float* beta,
                               float* out, int B, int H, int T, int d, int dtype,
                               hipStream_t stream) {
  if (!Q || !K || !V || !beta || !out) return FEM_ERR_NULLPTR;
  if (!sizes_ok(B, H, T, d)) return FEM_ERR_SHAPE;
  if (dtype == FEM_DTYPE_BF16) {
    if (d != 32 && d != 64 && d != 128) return FEM_ERR_UNSUPPORTED;
    if (!aligned16(Q) || !aligned16(K) || !aligned16(V) || !aligned16(out)) return FEM_ERR_ALIGN;
    return from_hip(fem::launch_softmax_bf16(Q, K, V, beta, out, B, H, T, d, stream));
  }
  if (dtype == FEM_DTYPE_F32) {
    if (d > 256) return FEM_ERR_UNSUPPORTED;
    if ((unsigned long long)B * H > 65535ull) return FEM_ERR_SHAPE;
    if (!aligned16(Q) || !aligned16(K) || !aligned16(V) || !aligned16(out)) return FEM_ERR_ALIGN;
    return from_hip(fem::launch_softmax_f32(static_cast<const float*>(Q),
                                            static_cast<const float*>(K),
                                            static_cast<const float*>(V), beta, out, B, H, T,
                                            d, stream));
  }
  return FEM_ERR_UNSUPPORTED;
}

extern "C" int fem_softmax_fwd_ex(const void* Q, const void* K, const void* V, const float* beta,
                                  void* out, int B, int H, int T, int d_qk, int d_v, int flags,
                                  int dtype, hipStream_t stream) {
  if (!Q || !K || !V || !beta || !out) return FEM_ERR_NULLPTR;
  if (!sizes_ok(B, H, T, d_qk) || !sizes_ok(B, H, T, d_v)) return FEM_ERR_SHAPE;
  if (dtype != FEM_DTYPE_BF16) return FEM_ERR_UNSUPPORTED;
  if (flags & ~(FEM_FLAG_ENCODER | FEM_FLAG_OUT_BF16)) return FEM_ERR_UNSUPPORTED;
  const bool pair_ok = (d_qk == d_v && (d_v == 32 || d_v == 64 || d_v == 128)) ||
                       (d_qk == 2 * d_v && (d_v == 32 || d_v == 64));
  if (!pair_ok) return FEM_ERR_UNSUPPORTED;
  if (!aligned16(Q) || !aligned16(K) || !aligned16(V) || !aligned16(out)) return FEM_ERR_ALIGN;
  return from_hip(fem::launch_softmax_ex_bf16(Q, K, V, beta, out, B, H, T, d_qk, d_v,
                                              !(flags & FEM_FLAG_ENCODER),
                                              (flags & FEM_FLAG_OUT_BF16) != 0, stream));
}

extern "C" size_t fem_softmax_decode_workspace_bytes(int B, int H, int L, int d_qk, int d_v) {
  if (!decode_sizes_ok(B, H, L, d_qk, d_v) || !decode_pair_ok(d_qk, d_v)) return 0;
  return fem::decode_ws_bytes(B, H, L, d_v);
}

extern "C" int fem_softmax_decode(const void* q, const void* Kc, const void* Vc, const int* lens,
                                  const float* beta, float* out, int B, int H, int L, int d_qk,
                                  int d_v, int dtype, void* ws, size_t ws_bytes,
                                  hipStream_t stream) {
  if (!q || !Kc || !Vc || !beta || !out) return FEM_ERR_NULLPTR;
  if (!decode_sizes_ok(B, H, L, d_qk, d_v)) return FEM_ERR_SHAPE;
  if (dtype != FEM_DTYPE_BF16) return FEM_ERR_UNSUPPORTED;
  if (!decode_pair_ok(d_qk, d_v)) return FEM_ERR_UNSUPPORTED;
  if (!aligned16(q) || !aligned16(Kc) || !aligned16(Vc)) return FEM_ERR_ALIGN;
  const int w = check_ws(ws, ws_bytes, fem::decode_ws_bytes(B, H, L, d_v));
  if (w != FEM_OK) return w;
  return from_hip(
      fem::launch_decode_bf16(q, Kc, Vc, lens, beta, out, B, H, L, d_qk, d_v, ws, stream));
}

extern "C" int fem_softmax_decode_noalloc(const void* q, const void* Kc, const void* Vc,
                                          const int* lens, const float* beta, float* out, int B,
                                          int H, int L, int d_qk, int d_v, int dtype,
                                          hipStream_t stream) {
  if (!q || !Kc || !Vc || !beta || !out) return FEM_ERR_NULLPTR;
  if (!decode_sizes_ok(B, H, L, d_qk, d_v)) return FEM_ERR_SHAPE;
  if (dtype != FEM_DTYPE_BF16) return FEM_ERR_UNSUPPORTED;
  if (!decode_pair_ok(d_qk, d_v)) return FEM_ERR_UNSUPPORTED;
  if (!aligned16(q) || !aligned16(Kc) || !aligned16(Vc)) return FEM_ERR_ALIGN;
  if (fem::decode_ws_bytes(B, H, L, d_v) > fem::kNoallocScratchBytes) return FEM_ERR_WORKSPACE;
  return from_hip(fem::launch_decode_noalloc_bf16(q, Kc, Vc, lens, beta, out, B, H, L, d_qk,
                                                  d_v, stream));
}

extern "C" int fem_softmax_fwd_train(const void* Q, const void* K, const void* V,
                                     const float* beta, float* out, float* lse, int B, int H,
                                     int T, int d, int dtype, hipStream_t stream) {
  if (!Q || !K || !V || !beta || !out || !lse) return FEM_ERR_NULLPTR;
  if (!sizes_ok(B, H, T, d)) return FEM_ERR_SHAPE;
  if (dtype != FEM_DTYPE_BF16) return FEM_ERR_UNSUPPORTED;
  if (d != 32 && d != 64 && d != 128) return FEM_ERR_UNSUPPORTED;
  if (!aligned16(Q) || !aligned16(K) || !aligned16(V) || !aligned16(out)) return FEM_ERR_ALIGN;
  return from_hip(fem::launch_softmax_train_bf16(Q, K, V, beta, out, lse, B, H, T, d, stream));
}

extern "C" size_t fem_softmax_bwd_workspace_bytes(int B, int H, int T, int d) {
  if (!bwd_args_ok(B, H, T, d)) return 0;
  return fem::softmax_bwd_ws_bytes(B, H, T, d);
}

extern "C" int fem_softmax_bwd(const void* Q, const void* K, const void* V, const float* beta,
                               const float* out, const float* lse, const float* dout, float* dQ,
                               float* dK, float* dV, float* dbeta, int B, int H, int T, int d,
                               int dtype, void* ws, size_t ws_bytes, hipStream_t stream) {
  if (!Q || !K || !V || !beta || !out || !lse || !dout || !dQ || !dK || !dV || !dbeta)
    return FEM_ERR_NULLPTR;
  if (!sizes_ok(B, H, T, d)) return FEM_ERR_SHAPE;
  if ((unsigned long long)H > 65535ull) return FEM_ERR_SHAPE;
  if (dtype != FEM_DTYPE_BF16) return FEM_ERR_UNSUPPORTED;
  if (d != 32 && d != 64 && d != 128) return FEM_ERR_UNSUPPORTED;
  const void* ptrs[] = {Q, K, V, out, dout, dQ, dK, dV};
  for (const void* p : ptrs)
    if (!aligned16(p)) return FEM_ERR_ALIGN;
  const int w = check_ws(ws, ws_bytes, fem::softmax_bwd_ws_bytes(B, H, T, d));
  if (w != FEM_OK) return w;
  return from_hip(fem::launch_softmax_bwd_bf16(Q, K, V, beta, out, lse, dout, dQ, dK, dV, dbeta,
                                               B, H, T, d, ws, stream));
}

extern "C" int fem_softmax_gated_fwd(const void* Q, const void* K, const void* V,
                                     const float* beta_max, const float* lam, const float* gate,
                                     float* out, int B, int H, int T, int d, int dtype,
                                     hipStream_t stream) {
  if (!Q || !K || !V || !beta_max || !lam || !out) return FEM_ERR_NULLPTR;
  if (!sizes_ok(B, H, T, d)) return FEM_ERR_SHAPE;
  if (dtype != FEM_DTYPE_BF16) return FEM_ERR_UNSUPPORTED;
  if (d != 32 && d != 64 && d != 128) return FEM_ERR_UNSUPPORTED;
  if (!aligned16(Q) || !aligned16(K) || !aligned16(V) || !aligned16(lam) || !aligned16(out) ||
      (gate && !aligned16(gate)))
    return FEM_ERR_ALIGN;
  return from_hip(
      fem::launch_softmax_gated_bf16(Q, K, V, beta_max, lam, gate, out, B, H, T, d, stream));
}

extern "C" size_t fem_linear_workspace_bytes(int B, int H, int T, int d_k, int d_v, int chunk) {
  if (!scan_args_ok(B, H, T, d_k, d_v, chunk, false)) return 0;
  return fem::scan_ws_bytes(B, H, T, chunk, false);
}

extern "C" size_t fem_gla_workspace_bytes(int B, int H, int T, int d_k, int d_v, int chunk) {
  if (!scan_args_ok(B, H, T, d_k, d_v, chunk, true)) return 0;
  return fem::scan_ws_bytes(B, H, T, chunk, true);
}

extern "C" int fem_linear_fwd(const void* Q, const void* K, const void* V, const float* beta,
                              float* out, int B, int H, int T, int d_k, int d_v, int chunk,
                              int dtype, void* ws, size_t ws_bytes, hipStream_t stream) {
  if (!Q || !K || !V || !beta || !out) return FEM_ERR_NULLPTR;
  if (!sizes_ok(B, H, T, d_k) || !sizes_ok(B, H, T, d_v)) return FEM_ERR_SHAPE;
  if (dtype != FEM_DTYPE_BF16) return FEM_ERR_UNSUPPORTED;
  if (!scan_args_ok(B, H, T, d_k, d_v, chunk, false)) return FEM_ERR_UNSUPPORTED;
  if (!aligned16(Q) || !aligned16(K) || !aligned16(V) || !aligned16(out)) return FEM_ERR_ALIGN;
  const int w = check_ws(ws, ws_bytes, fem::scan_ws_bytes(B, H, T, chunk, false));
  if (w != FEM_OK) return w;
  const hipError_t e =
      fem::launch_linear_bf16(Q, K, V, beta, out, B, H, T, d_k, d_v, chunk, ws, stream);
  if (e == hipErrorNotSupported) return FEM_ERR_UNSUPPORTED;
  return from_hip(e);
}

extern "C" int fem_gla_fwd(const void* Q, const void* K, const void* V, const float* G,
                           const float* beta, float* out, int B, int H, int T, int d_k, int d_v,
                           int chunk, int dtype, void* ws, size_t ws_bytes, hipStream_t stream) {
  if (!Q || !K || !V || !G || !beta || !out) return FEM_ERR_NULLPTR;
  if (!sizes_ok(B, H, T, d_k) || !sizes_ok(B, H, T, d_v)) return FEM_ERR_SHAPE;
  if (dtype != FEM_DTYPE_BF16) return FEM_ERR_UNSUPPORTED;
  if (!scan_args_ok(B, H, T, d_k, d_v, chunk, true)) return FEM_ERR_UNSUPPORTED;
  if (!aligned16(Q) || !aligned16(K) || !aligned16(V) || !aligned16(G) || !aligned16(out))
    return FEM_ERR_ALIGN;
  const int w = check_ws(ws, ws_bytes, fem::scan_ws_bytes(B, H, T, chunk, true));
  if (w != FEM_OK) return w;
  const hipError_t e =
      fem::launch_gla_bf16(Q, K, V, G, beta, out, B, H, T, d_k, d_v, chunk, ws, stream);
  if (e == hipErrorNotSupported) return FEM_ERR_UNSUPPORTED;
  return from_hip(e);
}

extern "C" const char* fem_status_str(int status) {
  switch (status) {
    case FEM_OK: return "FEM_OK";
    case FEM_ERR_NULLPTR: return "FEM_ERR_NULLPTR: a required pointer is NULL";
    case FEM_ERR_SHAPE: return "FEM_ERR_SHAPE: B, H, T or a width is not positive, or a size overflows";
    case FEM_ERR_UNSUPPORTED: return "FEM_ERR_UNSUPPORTED: width, chunk or dtype outside the supported set";
    case FEM_ERR_ALIGN: return "FEM_ERR_ALIGN: an input or out is not 16-byte aligned, or ws is not 256-byte aligned";
    case FEM_ERR_HIP: return "FEM_ERR_HIP: a HIP call or kernel launch failed";
    case FEM_ERR_WORKSPACE:
      return "FEM_ERR_WORKSPACE: ws is NULL or smaller than the entry point's workspace query";
    default: return "FEM_ERR_UNKNOWN: not a fem_status value";
  }
}
