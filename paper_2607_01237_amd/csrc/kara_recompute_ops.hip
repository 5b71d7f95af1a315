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

// two floats to a pair of bf16 (round to nearest even), low half first
__device__ inline uint32_t pack2(float a, float b) {
  const __hip_bfloat16 x = __float2bfloat16(a), y = __float2bfloat16(b);
  return (uint32_t)(*(const uint16_t*)&x) | ((uint32_t)(*(const uint16_t*)&y) << 16);
}

// One workgroup per token: x = h / sqrt(mean(h^2) + eps) * g, stored bf16;
// four elements per thread and access (D a multiple of 4).
__global__ __launch_bounds__(kNormThreads) void rmsnorm_kernel(const float* __restrict__ h,
                                                               const uint16_t* __restrict__ gamma,
                                                               uint16_t* __restrict__ x, int D, float eps) {
  const int64_t tok = blockIdx.x;
  const float4* row = (const float4*)(h + tok * D);
  const int n4 = D / 4;
  float ss = 0.f;
  for (int i = threadIdx.x; i < n4; i += kNormThreads) {
    const float4 v = row[i];
    ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
  }
  __shared__ float red[kNormThreads / 64];
  for (int o = 32; o > 0; o >>= 1) ss += __shfl_xor(ss, o, 64);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  float tot = 0.f;
#pragma unroll
  for (int w = 0; w < kNormThreads / 64; ++w) tot += red[w];
  const float r = 1.f / sqrtf(tot / (float)D + eps);
  const uint2* g4 = (const uint2*)gamma;
  uint2* out = (uint2*)(x + tok * D);
  for (int i = threadIdx.x; i < n4; i += kNormThreads) {
    const float4 v = row[i];
    const uint2 g = g4[i];
    const float y0 = v.x * r * bf16_to_f32((uint16_t)(g.x & 0xffff));
    const float y1 = v.y * r * bf16_to_f32((uint16_t)(g.x >> 16));
    const float y2 = v.z * r * bf16_to_f32((uint16_t)(g.y & 0xffff));
    const float y3 = v.w * r * bf16_to_f32((uint16_t)(g.y >> 16));
    out[i] = uint2{pack2(y0, y1), pack2(y2, y3)};
  }
}

// Rotate-half rotary embedding: for i < d/2 the pair (x_i, x_{i+d/2}) of
// every query head turns by pos * theta^(-2i/d), pos = rope_pos0[s] + w.
// One workgroup per window token (all its heads): the inverse frequencies
// are formed once per workgroup in fp64, each angle is formed and reduced
// modulo 2 pi in fp64 (positions reach tens of thousands of radians) and
// its sine and cosine taken in fp32.  Rows of flagged sequences are skipped.
__global__ __launch_bounds__(256) void rope_kernel(const uint16_t* __restrict__ qraw, uint16_t* __restrict__ q_out,
                                                   int W, int Hq, int d, double log2_theta,
                                                   const int32_t* __restrict__ trig,
                                                   const int32_t* __restrict__ rope_pos0,
                                                   const int32_t* __restrict__ status) {
  __shared__ double inv_freq[64];
  const int64_t tok = blockIdx.x;
  const int t = (int)(tok / W);
  if (status[t] != 0) return;
  const int half = d / 2;
  for (int j = threadIdx.x; j < half; j += blockDim.x) inv_freq[j] = exp2(-(2.0 * j / d) * log2_theta);
  __syncthreads();
  const int w = (int)(tok - (int64_t)t * W);
  const double pos = (double)rope_pos0[trig[t]] + w;
  constexpr double kTwoPi = 6.283185307179586476925286766559;
  const uint16_t* src = qraw + tok * (int64_t)Hq * d;
  uint16_t* dst = q_out + tok * (int64_t)Hq * d;
  for (int i = threadIdx.x; i < Hq * half; i += blockDim.x) {
    const int hh = i / half, j = i - hh * half;
    double ang = pos * inv_freq[j];
    ang -= floor(ang * (1.0 / kTwoPi)) * kTwoPi;
    float sn, cs;
    sincosf((float)ang, &sn, &cs);
    const uint16_t* sr = src + hh * d;
    const float a = bf16_to_f32(sr[j]), b = bf16_to_f32(sr[j + half]);
    const __hip_bfloat16 ra = __float2bfloat16(a * cs - b * sn), rb = __float2bfloat16(b * cs + a * sn);
    dst[hh * d + j] = *(const uint16_t*)&ra;
    dst[hh * d + j + half] = *(const uint16_t*)&rb;
  }
}

// gate <- silu(gate) * up, in fp32, stored bf16; eight elements per thread
// and access (n a multiple of 8).
__global__ void swiglu_kernel(uint4* __restrict__ gate, const uint4* __restrict__ up, int64_t n8) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n8) return;
  const uint4 g = gate[i], u = up[i];
  const uint32_t gw[4] = {g.x, g.y, g.z, g.w}, uw[4] = {u.x, u.y, u.z, u.w};
  uint32_t o[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const float g0 = bf16_to_f32((uint16_t)(gw[k] & 0xffff)), g1 = bf16_to_f32((uint16_t)(gw[k] >> 16));
    const float u0 = bf16_to_f32((uint16_t)(uw[k] & 0xffff)), u1 = bf16_to_f32((uint16_t)(uw[k] >> 16));
    o[k] = pack2(g0 / (1.f + expf(-g0)) * u0, g1 / (1.f + expf(-g1)) * u1);
  }
  gate[i] = uint4{o[0], o[1], o[2], o[3]};
}

}  // namespace

hipError_t launch_rmsnorm(const float* h, const void* gamma, void* x, int64_t n_tok, int D, float eps,
                          hipStream_t stream) {
  if (n_tok == 0) return hipSuccess;
  hipLaunchKernelGGL(rmsnorm_kernel, dim3((unsigned)n_tok), dim3(kNormThreads), 0, stream, h,
                     (const uint16_t*)gamma, (uint16_t*)x, D, eps);
  return hipGetLastError();
}

hipError_t launch_rope(const void* qraw, void* q_out, int n_trig, int W, int Hq, int d, float theta,
                       const int32_t* trig, const int32_t* rope_pos0, const int32_t* status, hipStream_t stream) {
  const int64_t n_tok = (int64_t)n_trig * W;
  if (n_tok == 0) return hipSuccess;
  hipLaunchKernelGGL(rope_kernel, dim3((unsigned)n_tok), dim3(256), 0, stream, (const uint16_t*)qraw,
                     (uint16_t*)q_out, W, Hq, d, std::log2((double)theta), trig, rope_pos0, status);
  return hipGetLastError();
}

hipError_t launch_swiglu(void* gate, const void* up, int64_t n, hipStream_t stream) {
  const int64_t n8 = n / 8;
  if (n8 == 0) return hipSuccess;
  hipLaunchKernelGGL(swiglu_kernel, dim3((unsigned)((n8 + 255) / 256)), dim3(256), 0, stream, (uint4*)gate,
                     (const uint4*)up, n8);
  return hipGetLastError();
}

}  // namespace kara
