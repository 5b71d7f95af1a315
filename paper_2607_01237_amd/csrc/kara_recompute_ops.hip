// Element-wise and per-token steps of the window recompute pass (App. C.2):
// RMSNorm of the fp32 residual stream into bf16, the rotary embedding of
// the projected queries into the scoring-query layout, and the SwiGLU gate.
// The matrix products are rocBLAS calls on the host side; attention is
// kara_attn.hip.
#include <hip/hip_bf16.h>

#include "kara_internal.h"

namespace kara {
namespace {

constexpr int kNormThreads = 256;

__device__ inline float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// One workgroup per token: x = h / sqrt(mean(h^2) + eps) * g, stored bf16.
__global__ __launch_bounds__(kNormThreads) void rmsnorm_kernel(const float* __restrict__ h,
                                                               const uint16_t* __restrict__ gamma,
                                                               __hip_bfloat16* __restrict__ x, int D, float eps) {
  const int64_t tok = blockIdx.x;
  const float* row = h + tok * D;
  float ss = 0.f;
  for (int i = threadIdx.x; i < D; i += kNormThreads) ss += row[i] * row[i];
  __shared__ float red[kNormThreads / 64];
  for (int o = 32; o > 0; o >>= 1) ss += __shfl_xor(ss, o, 64);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  float tot = 0.f;
#pragma unroll
  for (int w = 0; w < kNormThreads / 64; ++w) tot += red[w];
  const float r = 1.f / sqrtf(tot / (float)D + eps);
  __hip_bfloat16* out = x + tok * D;
  for (int i = threadIdx.x; i < D; i += kNormThreads) out[i] = __float2bfloat16(row[i] * r * bf16_to_f32(gamma[i]));
}

// Rotate-half rotary embedding: for i < d/2 the pair (x_i, x_{i+d/2}) of
// every query head turns by pos * theta^(-2i/d), pos = rope_pos0[s] + w.
// The angle and its sine and cosine are formed in fp64 (positions reach
// tens of thousands of radians).  Rows of flagged sequences are skipped.
__global__ void rope_kernel(const uint16_t* __restrict__ qraw, __hip_bfloat16* __restrict__ q_out, int W, int Hq,
                            int d, double log2_theta, const int32_t* __restrict__ trig,
                            const int32_t* __restrict__ rope_pos0, const int32_t* __restrict__ status,
                            int64_t n_pairs) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n_pairs) return;
  const int half = d / 2;
  const int j = (int)(i % half);
  const int64_t row = i / half;                 // (token, head)
  const int64_t tok = row / Hq;
  const int t = (int)(tok / W);
  if (status[t] != 0) return;
  const int w = (int)(tok - (int64_t)t * W);
  const double pos = (double)rope_pos0[trig[t]] + w;
  const double ang = pos * exp2(-(2.0 * j / d) * log2_theta);
  double sn, cs;
  sincos(ang, &sn, &cs);
  const uint16_t* src = qraw + row * d;
  const float a = bf16_to_f32(src[j]), b = bf16_to_f32(src[j + half]);
  const float c = (float)cs, s = (float)sn;
  __hip_bfloat16* dst = q_out + row * d;
  dst[j] = __float2bfloat16(a * c - b * s);
  dst[j + half] = __float2bfloat16(b * c + a * s);
}

// gate <- silu(gate) * up, in fp32, stored bf16.
__global__ void swiglu_kernel(uint16_t* __restrict__ gate, const uint16_t* __restrict__ up, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const float g = bf16_to_f32(gate[i]);
  const float u = bf16_to_f32(up[i]);
  const float v = g / (1.f + expf(-g)) * u;
  const __hip_bfloat16 r = __float2bfloat16(v);
  gate[i] = *(const uint16_t*)&r;
}

}  // namespace

hipError_t launch_rmsnorm(const float* h, const void* gamma, void* x, int64_t n_tok, int D, float eps,
                          hipStream_t stream) {
  if (n_tok == 0) return hipSuccess;
  hipLaunchKernelGGL(rmsnorm_kernel, dim3((unsigned)n_tok), dim3(kNormThreads), 0, stream, h,
                     (const uint16_t*)gamma, (__hip_bfloat16*)x, D, eps);
  return hipGetLastError();
}

hipError_t launch_rope(const void* qraw, void* q_out, int n_trig, int W, int Hq, int d, float theta,
                       const int32_t* trig, const int32_t* rope_pos0, const int32_t* status, hipStream_t stream) {
  const int64_t n = (int64_t)n_trig * W * Hq * (d / 2);
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(rope_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream, (const uint16_t*)qraw,
                     (__hip_bfloat16*)q_out, W, Hq, d, std::log2((double)theta), trig, rope_pos0, status, n);
  return hipGetLastError();
}

hipError_t launch_swiglu(void* gate, const void* up, int64_t n, hipStream_t stream) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(swiglu_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream, (uint16_t*)gate,
                     (const uint16_t*)up, n);
  return hipGetLastError();
}

}  // namespace kara
