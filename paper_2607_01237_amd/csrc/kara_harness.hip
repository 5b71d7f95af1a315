// Decoding-side helpers for long-running workloads (kara_harness.h): token
// append into the paged cache, and split-key decode attention of one query
// per (layer, sequence, query head) over the compressed cache.  Not part of
// the compression step; same paged layout.
#include <cmath>

#include "kara_harness.h"
#include "kara_internal.h"

namespace kara {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kNegInf = -__builtin_huge_valf();
constexpr int kSplitKeys = KARA_HARNESS_SPLIT_KEYS;

// ---------------------------------------------------------------- append

__global__ void append_check_kernel(Geom g, int n, const int32_t* __restrict__ seqs, int n_new,
                                    const int32_t* __restrict__ bt, const int32_t* __restrict__ seq_lens,
                                    int32_t* __restrict__ status) {
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= n) return;
  const int s = seqs[j];
  if (s < 0 || s >= g.n_seqs) {
    status[j] = KARA_SEQ_BAD_INDEX;
    return;
  }
  int st = 0;
  for (int o = 0; o < n; ++o)
    if (o != j && seqs[o] == s) st |= KARA_SEQ_DUP_TRIGGER;
  const int64_t len = seq_lens[s];
  const int64_t new_len = len + n_new;
  if (len < 0 || new_len > (int64_t)g.max_blocks * g.bs) {
    status[j] = st | KARA_SEQ_BAD_WINDOW;
    return;
  }
  const int32_t* row = bt + (int64_t)s * g.max_blocks;
  for (int64_t b = len / g.bs; b < (new_len + g.bs - 1) / g.bs; ++b) {
    const int pg = row[b];
    if (pg < 0 || pg >= g.num_pages) {
      st |= KARA_SEQ_BAD_PAGE;
      break;
    }
  }
  status[j] = st;
}

// One thread per 16 bytes of new rows: grid (chunks of n * n_new * Hkv rows, layer, K|V).
__global__ __launch_bounds__(256) void append_kernel(Geom g, int n, const int32_t* __restrict__ seqs, int n_new,
                                                     const char* __restrict__ k_new, const char* __restrict__ v_new,
                                                     PoolPtrs kp, PoolPtrs vp, const int32_t* __restrict__ bt,
                                                     const int32_t* __restrict__ seq_lens,
                                                     const int32_t* __restrict__ status) {
  const int l = blockIdx.y;
  const int kv = blockIdx.z;
  const int row_bytes = g.d * g.esize;
  const int cpr = row_bytes / 16;
  const int64_t per_layer = (int64_t)n * n_new * g.Hkv * cpr;   // 16-byte pieces of one layer
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= per_layer) return;
  const int c = (int)(i % cpr);
  const int64_t row = i / cpr;                 // [n][n_new][Hkv]
  const int h = (int)(row % g.Hkv);
  const int tok = (int)((row / g.Hkv) % n_new);
  const int j = (int)(row / ((int64_t)g.Hkv * n_new));
  if (status[j] != 0) return;
  const int s = seqs[j];
  const int pos = seq_lens[s] + tok;
  const int64_t page = bt[(int64_t)s * g.max_blocks + pos / g.bs];
  const char* src = (kv ? v_new : k_new) + ((int64_t)l * per_layer + i) * 16;
  char* dst = (char*)(kv ? vp.p[l] : kp.p[l]) + ((page * g.Hkv + h) * g.bs + pos % g.bs) * (int64_t)row_bytes + c * 16;
  *(uint4*)dst = *(const uint4*)src;
}

__global__ void append_commit_kernel(int n, const int32_t* __restrict__ seqs, int n_new,
                                     int32_t* __restrict__ seq_lens, const int32_t* __restrict__ status) {
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j < n && status[j] == 0) seq_lens[seqs[j]] += n_new;
}

// ---------------------------------------------------------------- decode

// A lane's MFMA operand for 16-row tiles: lane group gq = lane/16 supplies
// head-dim elements [gq*d/4, (gq+1)*d/4) of row lane%16.
template <int DT, int D>
struct Op16 {
  static constexpr int kChunks = (D * (DT == KARA_BF16 ? 2 : 4) / 16) / 4;
  uint4 v[kChunks];
};

template <int DT, int D>
__device__ inline floatx4 dot16(const Op16<DT, D>& a, const Op16<DT, D>& b) {
  floatx4 acc = {0.f, 0.f, 0.f, 0.f};
  if constexpr (DT == KARA_BF16) {
#pragma unroll
    for (int s = 0; s < Op16<DT, D>::kChunks; ++s) {
      bf16x8 x, y;
      __builtin_memcpy(&x, &a.v[s], 16);
      __builtin_memcpy(&y, &b.v[s], 16);
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(x, y, acc, 0, 0, 0);
    }
  } else {
    const float* x = (const float*)a.v;
    const float* y = (const float*)b.v;
#pragma unroll
    for (int s = 0; s < Op16<DT, D>::kChunks * 4; ++s) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(x[s], y[s], acc, 0, 0, 0);
  }
  return acc;
}

__device__ inline float to_f32(const char* p, int dtype) {
  if (dtype == KARA_BF16) {
    const uint32_t b = *(const uint16_t*)p;
    return __uint_as_float(b << 16);
  }
  return *(const float*)p;
}

// One wave per (layer, sequence, KV head, split of kSplitKeys keys): for the
// G query heads of the KV head, the split's running maximum m, exponential
// sum l and unnormalised output o (log2 units; partial softmax of the split).
// Workspace record per (layer, j, query head, split): m, l, o[d].
template <int DT, int D>
__global__ __launch_bounds__(64) void decode_split_kernel(Geom g, int n, const int32_t* __restrict__ seqs,
                                                          const char* __restrict__ q, PoolPtrs kp, PoolPtrs vp,
                                                          const int32_t* __restrict__ bt,
                                                          const int32_t* __restrict__ seq_lens, int max_len,
                                                          int n_splits, float* __restrict__ ws) {
  constexpr int ES = DT == KARA_BF16 ? 2 : 4;
  constexpr int kRowBytes = D * ES;
  constexpr int KC = Op16<DT, D>::kChunks;
  constexpr int kDPerLane = D / 64;
  __shared__ float p_tile[16][16];   // probabilities of the tile: [query head][key]

  const int lane = threadIdx.x;
  const int gq = lane >> 4, li = lane & 15;
  const int split = blockIdx.x % n_splits;
  const int64_t rest = blockIdx.x / n_splits;
  const int h = (int)(rest % g.Hkv);
  const int j = (int)((rest / g.Hkv) % n);
  const int l = (int)(rest / ((int64_t)g.Hkv * n));
  const int s = seqs[j];
  if (s < 0 || s >= g.n_seqs) return;   // the combine kernel writes its zero rows
  const int len = seq_lens[s];
  const int k0 = split * kSplitKeys;
  if (len <= 0 || len > max_len || k0 >= len) return;
  const int k1 = min(len, k0 + kSplitKeys);
  const int G = g.G;
  const float c = g.scale * kLog2e;

  // query rows (row r < G is query head h*G + r; others zero)
  Op16<DT, D> qa;
  {
    const int r = li;
    const uint4* src = (const uint4*)(q + (((int64_t)l * n + j) * g.Hq + h * G + (r < G ? r : 0)) * kRowBytes) + gq * KC;
#pragma unroll
    for (int x = 0; x < KC; ++x) qa.v[x] = r < G ? src[x] : uint4{0, 0, 0, 0};
  }
  const int32_t* row_pages = bt + (int64_t)s * g.max_blocks;
  const char* kbase = (const char*)kp.p[l];
  const char* vbase = (const char*)vp.p[l];

  // per-row state, held in lanes gq = r/4 (element r%4) for the softmax and
  // replicated into every lane for the output
  float m[4] = {kNegInf, kNegInf, kNegInf, kNegInf}, lsum[4] = {0.f, 0.f, 0.f, 0.f};
  float o[16][kDPerLane];
  float mo[16];   // each row's running maximum, as every lane sees it
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    mo[r] = kNegInf;
#pragma unroll
    for (int e = 0; e < kDPerLane; ++e) o[r][e] = 0.f;
  }

  for (int t0 = k0; t0 < k1; t0 += 16) {
    const int key = t0 + li;
    Op16<DT, D> kb;
    if (key < k1) {
      const int64_t pg = row_pages[key / g.bs];
      const uint4* src = (const uint4*)(kbase + ((pg * g.Hkv + h) * g.bs + key % g.bs) * kRowBytes) + gq * KC;
#pragma unroll
      for (int x = 0; x < KC; ++x) kb.v[x] = src[x];
    } else {
#pragma unroll
      for (int x = 0; x < KC; ++x) kb.v[x] = uint4{0, 0, 0, 0};
    }
    const floatx4 sc = dot16<DT, D>(qa, kb);   // rows 4*gq+e, key li
    // running maximum and sum per row (lanes of one lane group share rows)
    float pv[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float x = key < k1 ? sc[e] * c : kNegInf;
      float tm = x;
#pragma unroll
      for (int off = 1; off < 16; off <<= 1) tm = fmaxf(tm, __shfl_xor(tm, off, 64));
      const float mn = fmaxf(m[e], tm);
      const float p = key < k1 ? __builtin_amdgcn_exp2f(x - mn) : 0.f;
      float ps = p;
#pragma unroll
      for (int off = 1; off < 16; off <<= 1) ps += __shfl_xor(ps, off, 64);
      lsum[e] = lsum[e] * (m[e] == kNegInf ? 0.f : __builtin_amdgcn_exp2f(m[e] - mn)) + ps;
      m[e] = mn;
      pv[e] = p;
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) p_tile[4 * gq + e][li] = pv[e];
    __syncthreads();
    // o[r] = o[r] * 2^(m_old - m_new) + sum_k p[r][k] v_k; lane owns head-dim
    // elements lane*kDPerLane..
    float vrow[16][kDPerLane];
#pragma unroll
    for (int kk = 0; kk < 16; ++kk) {
      const int kx = t0 + kk;
      if (kx < k1) {
        const int64_t pg = row_pages[kx / g.bs];
        const char* vr = vbase + ((pg * g.Hkv + h) * g.bs + kx % g.bs) * kRowBytes + lane * kDPerLane * ES;
#pragma unroll
        for (int e = 0; e < kDPerLane; ++e) vrow[kk][e] = to_f32(vr + e * ES, DT);
      } else {
#pragma unroll
        for (int e = 0; e < kDPerLane; ++e) vrow[kk][e] = 0.f;
      }
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      if (r >= G) break;
      const float mn = __shfl(m[r & 3], (r >> 2) * 16, 64);
      const float f = mo[r] == kNegInf ? 0.f : __builtin_amdgcn_exp2f(mo[r] - mn);
      mo[r] = mn;
#pragma unroll
      for (int e = 0; e < kDPerLane; ++e) {
        float acc = o[r][e] * f;
#pragma unroll
        for (int kk = 0; kk < 16; ++kk) acc = fmaf(p_tile[r][kk], vrow[kk][e], acc);
        o[r][e] = acc;
      }
    }
    __syncthreads();
  }
  // records: m, l, o[d]
  const int rec = D + 2;
  for (int r = 0; r < G; ++r) {
    float* w = ws + ((((int64_t)l * n + j) * g.Hq + h * G + r) * n_splits + split) * rec;
    const float mr = __shfl(m[r & 3], (r >> 2) * 16, 64);
    const float lr = __shfl(lsum[r & 3], (r >> 2) * 16, 64);
    if (lane == 0) {
      w[0] = mr;
      w[1] = lr;
    }
#pragma unroll
    for (int e = 0; e < kDPerLane; ++e) w[2 + lane * kDPerLane + e] = o[r][e];
  }
}

// One wave per (layer, sequence, query head): combine the splits.
template <int D>
__global__ __launch_bounds__(64) void decode_combine_kernel(Geom g, int n, const int32_t* __restrict__ seqs,
                                                            const int32_t* __restrict__ seq_lens, int max_len,
                                                            int n_splits, const float* __restrict__ ws,
                                                            float* __restrict__ out) {
  constexpr int kDPerLane = D / 64;
  const int lane = threadIdx.x;
  const int64_t row = blockIdx.x;                 // (l, j, hq)
  const int j = (int)((row / g.Hq) % n);
  const int s = seqs[j];
  const int len = s >= 0 && s < g.n_seqs ? seq_lens[s] : 0;
  float* dst = out + row * D + lane * kDPerLane;
  if (len <= 0 || len > max_len) {
#pragma unroll
    for (int e = 0; e < kDPerLane; ++e) dst[e] = 0.f;
    return;
  }
  const int ns = (len + kSplitKeys - 1) / kSplitKeys;
  const int rec = D + 2;
  const float* w = ws + row * n_splits * rec;
  float M = kNegInf;
  for (int sp = 0; sp < ns; ++sp) M = fmaxf(M, w[sp * rec]);
  float L = 0.f, acc[kDPerLane] = {};
  for (int sp = 0; sp < ns; ++sp) {
    const float f = __builtin_amdgcn_exp2f(w[sp * rec] - M);
    L += w[sp * rec + 1] * f;
#pragma unroll
    for (int e = 0; e < kDPerLane; ++e) acc[e] += w[sp * rec + 2 + lane * kDPerLane + e] * f;
  }
#pragma unroll
  for (int e = 0; e < kDPerLane; ++e) dst[e] = acc[e] / L;
}

template <int DT, int D>
hipError_t launch_decode(const Geom& g, int n, const int32_t* seqs, int n_layers, const void* q, const PoolPtrs& kp,
                         const PoolPtrs& vp, const int32_t* bt, const int32_t* seq_lens, int max_len, float* out,
                         float* ws, int n_splits, hipStream_t stream) {
  const int64_t blocks = (int64_t)n_layers * n * g.Hkv * n_splits;
  hipLaunchKernelGGL((decode_split_kernel<DT, D>), dim3((unsigned)blocks), dim3(64), 0, stream, g, n, seqs,
                     (const char*)q, kp, vp, bt, seq_lens, max_len, n_splits, ws);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((decode_combine_kernel<D>), dim3((unsigned)((int64_t)n_layers * n * g.Hq)), dim3(64), 0,
                     stream, g, n, seqs, seq_lens, max_len, n_splits, (const float*)ws, out);
  return hipGetLastError();
}

// the step's window fields are irrelevant here; validate the rest
kara_status_t harness_geom(const kara_params_t* p, int32_t n, Geom* g) {
  kara_status_t st = make_geom(p, n, g);
  if (st != KARA_OK) return st;
  return KARA_OK;
}

}  // namespace
}  // namespace kara

using namespace kara;

extern "C" {

kara_status_t kara_harness_kv_append(const kara_params_t* p, int32_t n, const int32_t* seqs, int32_t n_new,
                                     int32_t n_layers, const void* k_new, const void* v_new, void* const* k_pools,
                                     void* const* v_pools, const int32_t* block_table, int32_t* seq_lens,
                                     int32_t* status, void* stream) {
  Geom g;
  kara_status_t st = harness_geom(p, n, &g);
  if (st != KARA_OK) return st;
  if (n < 0 || n_new < 0 || n_layers < 1 || n_layers > kMaxLayersPerLaunch) return KARA_ERR_INVALID_ARG;
  if (n == 0 || n_new == 0) return KARA_OK;
  if (!seqs || !k_new || !v_new || !block_table || !seq_lens || !status ||
      !pools_ok((const void* const*)k_pools, n_layers) || !pools_ok((const void* const*)v_pools, n_layers))
    return KARA_ERR_INVALID_ARG;
  hipStream_t s = (hipStream_t)stream;
  hipLaunchKernelGGL(append_check_kernel, dim3((n + 255) / 256), dim3(256), 0, s, g, n, seqs, n_new, block_table,
                     seq_lens, status);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_status(e);
  PoolPtrs kp{}, vp{};
  for (int i = 0; i < n_layers; ++i) {
    kp.p[i] = k_pools[i];
    vp.p[i] = v_pools[i];
  }
  const int64_t pieces = (int64_t)n * n_new * g.Hkv * (g.d * g.esize / 16);
  hipLaunchKernelGGL(append_kernel, dim3((unsigned)((pieces + 255) / 256), (unsigned)n_layers, 2), dim3(256), 0, s,
                     g, n, seqs, n_new, (const char*)k_new, (const char*)v_new, kp, vp, block_table, seq_lens,
                     status);
  e = hipGetLastError();
  if (e != hipSuccess) return hip_status(e);
  hipLaunchKernelGGL(append_commit_kernel, dim3((n + 255) / 256), dim3(256), 0, s, n, seqs, n_new, seq_lens, status);
  return hip_status(hipGetLastError());
}

kara_status_t kara_harness_decode_workspace_size(const kara_params_t* p, int32_t n, int32_t n_layers,
                                                 int32_t max_len, size_t* bytes) {
  Geom g;
  kara_status_t st = harness_geom(p, n, &g);
  if (st != KARA_OK) return st;
  if (!bytes || n_layers < 1 || max_len < 1 || (int64_t)max_len > (int64_t)g.max_blocks * g.bs)
    return KARA_ERR_INVALID_ARG;
  const int64_t n_splits = (max_len + kSplitKeys - 1) / kSplitKeys;
  *bytes = (size_t)n_layers * n * g.Hq * n_splits * (g.d + 2) * sizeof(float);
  return KARA_OK;
}

kara_status_t kara_harness_decode_attention(const kara_params_t* p, int32_t n, const int32_t* seqs,
                                            int32_t n_layers, const void* q, const void* const* k_pools,
                                            const void* const* v_pools, const int32_t* block_table,
                                            const int32_t* seq_lens, int32_t max_len, float* out,
                                            void* workspace, size_t workspace_bytes, void* stream) {
  Geom g;
  kara_status_t st = harness_geom(p, n, &g);
  if (st != KARA_OK) return st;
  if (g.G > KARA_HARNESS_MAX_GROUP) return KARA_ERR_UNSUPPORTED;
  size_t need = 0;
  st = kara_harness_decode_workspace_size(p, n, n_layers, max_len, &need);
  if (st != KARA_OK) return st;
  if (n_layers > kMaxLayersPerLaunch) return KARA_ERR_INVALID_ARG;
  if (n == 0) return KARA_OK;
  if (!seqs || !q || !block_table || !seq_lens || !out || !pools_ok(k_pools, n_layers) ||
      !pools_ok(v_pools, n_layers))
    return KARA_ERR_INVALID_ARG;
  if (!workspace || workspace_bytes < need) return KARA_ERR_WORKSPACE;
  PoolPtrs kp{}, vp{};
  for (int i = 0; i < n_layers; ++i) {
    kp.p[i] = const_cast<void*>(k_pools[i]);
    vp.p[i] = const_cast<void*>(v_pools[i]);
  }
  const int n_splits = (max_len + kSplitKeys - 1) / kSplitKeys;
  hipStream_t s = (hipStream_t)stream;
  float* ws = (float*)workspace;
  hipError_t e;
  if (g.dtype == KARA_BF16)
    e = g.d == 128 ? launch_decode<KARA_BF16, 128>(g, n, seqs, n_layers, q, kp, vp, block_table, seq_lens, max_len,
                                                  out, ws, n_splits, s)
                   : launch_decode<KARA_BF16, 64>(g, n, seqs, n_layers, q, kp, vp, block_table, seq_lens, max_len,
                                                 out, ws, n_splits, s);
  else
    e = g.d == 128 ? launch_decode<KARA_F32, 128>(g, n, seqs, n_layers, q, kp, vp, block_table, seq_lens, max_len,
                                                 out, ws, n_splits, s)
                   : launch_decode<KARA_F32, 64>(g, n, seqs, n_layers, q, kp, vp, block_table, seq_lens, max_len,
                                                out, ws, n_splits, s);
  return hip_status(e);
}

}  // extern "C"
