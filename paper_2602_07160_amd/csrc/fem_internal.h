// Host-side launchers behind the C ABI (internal; not exported).
#pragma once

#include <hip/hip_runtime.h>

namespace fem {

// Fused bf16 matrix-core softmax-prior read, d in {32, 64, 128}.
hipError_t launch_softmax_bf16(const void* Q, const void* K, const void* V,
                               const float* beta, float* out,
                               int B, int H, int T, int d, hipStream_t stream);

// The plain read's variants: (dk, dv) in {(32,32), (64,64), (128,128),
// (64,32), (128,64)}, causal or encoder (all keys), fp32 or bf16 output.
hipError_t launch_softmax_ex_bf16(const void* Q, const void* K, const void* V, const float* beta,
                                  void* out, int B, int H, int T, int dk, int dv, bool causal,
                                  bool obf16, hipStream_t stream);

// The plain causal read (bf16, d in {32, 64, 128}) that also writes the
// prior's log-normaliser lse [B, H, T] (natural log) for the backward pass.
hipError_t launch_softmax_train_bf16(const void* Q, const void* K, const void* V,
                                     const float* beta, float* out, float* lse, int B, int H,
                                     int T, int d, hipStream_t stream);

// Backward of the causal softmax-prior read (bf16 inputs, d in {32, 64, 128}).
// ws holds at least softmax_bwd_ws_bytes(B, H, T, d) bytes, 256-byte aligned.
size_t softmax_bwd_ws_bytes(int B, int H, int T, int d);
hipError_t launch_softmax_bwd_bf16(const void* Q, const void* K, const void* V,
                                   const float* beta, const float* out, const float* lse,
                                   const float* dout, float* dQ, float* dK, float* dV,
                                   float* dbeta, int B, int H, int T, int d, void* ws,
                                   hipStream_t stream);

// Two-level gated read g * ((1 - lam) mu + lam F(beta_max)) with the softmax
// prior, bf16, d in {32, 64, 128}; gate may be null (g = 1).
hipError_t launch_softmax_gated_bf16(const void* Q, const void* K, const void* V,
                                     const float* beta_max, const float* lam, const float* gate,
                                     float* out, int B, int H, int T, int d, hipStream_t stream);

// One decoding step against a KV cache (single query per (b, h)), bf16,
// (dk, dv) as launch_softmax_ex_bf16.  lens may be null (every row has L keys).
// ws holds at least decode_ws_bytes(B, H, L, dv) bytes, 256-byte aligned.
size_t decode_ws_bytes(int B, int H, int L, int dv);
hipError_t launch_decode_bf16(const void* q, const void* Kc, const void* Vc, const int* lens,
                              const float* beta, float* out, int B, int H, int L, int dk, int dv,
                              void* ws, hipStream_t stream);

// The same step with its partials in a fixed per-device array of
// kNoallocScratchBytes (no allocation, no workspace argument).  Sizes whose
// decode_ws_bytes exceed it return hipErrorInvalidValue.
constexpr size_t kNoallocScratchBytes = (size_t)8 << 20;
hipError_t launch_decode_noalloc_bf16(const void* q, const void* Kc, const void* Vc,
                                      const int* lens, const float* beta, float* out, int B,
                                      int H, int L, int dk, int dv, hipStream_t stream);

// Exact fp32 vector-unit softmax-prior read, 1 <= d <= 256.
hipError_t launch_softmax_f32(const float* Q, const float* K, const float* V,
                              const float* beta, float* out,
                              int B, int H, int T, int d, hipStream_t stream);

// Chunked-scan linear-prior read (phi = elu + 1), bf16, d_k = d_v = 64.
// ws holds at least scan_ws_bytes(B, H, T, chunk, false) bytes, 256-byte
// aligned (it may be null when that is 0).
size_t scan_ws_bytes(int B, int H, int T, int chunk, bool gla);
hipError_t launch_linear_bf16(const void* Q, const void* K, const void* V,
                              const float* beta, float* out,
                              int B, int H, int T, int dk, int dv, int chunk, void* ws,
                              hipStream_t stream);

// Chunked-scan GLA-prior read (RoPE, ReLU + eps features, per-channel
// log-decays G [B, H, T, d_k] clipped to [-2, 0]), bf16, d_k = d_v = 64.
// ws as launch_linear_bf16 with gla = true.
hipError_t launch_gla_bf16(const void* Q, const void* K, const void* V, const float* G,
                           const float* beta, float* out, int B, int H, int T, int dk, int dv,
                           int chunk, void* ws, hipStream_t stream);

}  // namespace fem
