// Host side of the window recompute pass (include/kara_recompute.h): the
// layer loop, its workspace, and the matrix products on rocBLAS (bf16
// operands, fp32 accumulation; the two products that feed the residual
// stream accumulate into it in fp32).
#include <rocblas/rocblas.h>

#include <cmath>
#include <mutex>

#include "kara_internal.h"
#include "kara_recompute.h"

using namespace kara;

namespace {

kara_status_t recompute_geom(const kara_params_t* p, int32_t n_trig, Geom* g) {
  const kara_status_t st = make_geom(p, n_trig, g);
  if (st != KARA_OK) return st;
  if (g->dtype != KARA_BF16) return KARA_ERR_UNSUPPORTED;
  return KARA_OK;
}

// vectorised element-wise kernels: hidden a multiple of 4, ffn of 8
bool model_ok(const kara_model_t* m) {
  return m && m->hidden >= 4 && m->hidden % 4 == 0 && m->ffn >= 8 && m->ffn % 8 == 0 && m->rope_theta > 1.f && std::isfinite(m->rope_theta) &&
         m->rms_eps >= 0.f && std::isfinite(m->rms_eps);
}

struct RecomputeWs {
  size_t x, qraw, attn, gate, up, blas, total;
};

// Scratch handed to rocBLAS for the products (rocblas_set_workspace), so it
// allocates none of its own; each call checks with a size query that its
// products fit.
constexpr size_t kBlasWorkspace = (size_t)32 << 20;

size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

RecomputeWs recompute_ws(const Geom& g, const kara_model_t& m, int32_t n_trig) {
  const size_t T = (size_t)n_trig * g.W;
  RecomputeWs w{};
  size_t off = 0;
  w.x = off;
  off += align256(T * m.hidden * 2);
  w.qraw = off;
  off += align256(T * g.Hq * g.d * 2);
  w.attn = off;
  off += align256(T * g.Hq * g.d * 2);
  w.gate = off;
  off += align256(T * m.ffn * 2);
  w.up = off;
  off += align256(T * m.ffn * 2);
  w.blas = off;
  off += kBlasWorkspace;
  w.total = off;
  return w;
}

// One rocBLAS handle per device, created on first use; each call then points
// it at the caller's workspace slice.
constexpr int kMaxDevices = 64;
rocblas_handle g_handles[kMaxDevices];
std::mutex g_handle_mutex;

rocblas_handle handle_for_current_device() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_handle_mutex);
  if (!g_handles[dev] && rocblas_create_handle(&g_handles[dev]) != rocblas_status_success) g_handles[dev] = nullptr;
  return g_handles[dev];
}

// Row-major C[rows][n] (= or +=) A[rows][k] B[k][n]: the column-major product
// C^T = B^T A^T with the row-major arrays read as their transposes.
bool gemm(rocblas_handle h, int64_t rows, int n, int k, const void* A, const void* B, void* C, bool f32_accum_out) {
  const float alpha = 1.f, beta = f32_accum_out ? 1.f : 0.f;
  const rocblas_datatype out_t = f32_accum_out ? rocblas_datatype_f32_r : rocblas_datatype_bf16_r;
  const rocblas_status st = rocblas_gemm_ex(
      h, rocblas_operation_none, rocblas_operation_none, n, (rocblas_int)rows, k, &alpha, B, rocblas_datatype_bf16_r,
      n, A, rocblas_datatype_bf16_r, k, &beta, C, out_t, n, C, out_t, n, rocblas_datatype_f32_r,
      rocblas_gemm_algo_standard, 0, 0);
  return st == rocblas_status_success;
}

}  // namespace

extern "C" {

kara_status_t kara_recompute_attention(const kara_params_t* p, int32_t n_trig, const int32_t* trig,
                                       const void* q, const void* k_pool, const void* v_pool,
                                       const int32_t* block_table, const int32_t* seq_lens,
                                       const int32_t* win_start, void* out, int32_t* status, void* stream) {
  Geom g;
  kara_status_t st = recompute_geom(p, n_trig, &g);
  if (st != KARA_OK) return st;
  if (n_trig == 0) return KARA_OK;
  if (!trig || !q || !k_pool || !v_pool || !block_table || !seq_lens || !win_start || !out || !status)
    return KARA_ERR_INVALID_ARG;
  if ((int64_t)n_trig * g.Hkv * ((int64_t)g.G * g.W + 127) / 128 > INT32_MAX) return KARA_ERR_INVALID_ARG;
  hipError_t e = launch_recompute_validate(g, trig, block_table, seq_lens, win_start, status, (hipStream_t)stream);
  if (e == hipSuccess)
    e = launch_recompute_attention(g, q, k_pool, v_pool, trig, block_table, win_start, out, status,
                                   (hipStream_t)stream);
  return hip_status(e);
}

kara_status_t kara_recompute_workspace_size(const kara_params_t* p, const kara_model_t* m, int32_t n_trig,
                                            size_t* bytes) {
  Geom g;
  kara_status_t st = recompute_geom(p, n_trig, &g);
  if (st != KARA_OK) return st;
  if (!model_ok(m) || !bytes) return KARA_ERR_INVALID_ARG;
  *bytes = recompute_ws(g, *m, n_trig).total;
  return KARA_OK;
}

kara_status_t kara_recompute_queries(const kara_params_t* p, const kara_model_t* m, int32_t n_trig,
                                     const int32_t* trig, int32_t n_layers, const kara_layer_weights_t* weights,
                                     const float* hidden_in, float* hidden_out, const void* const* k_pools,
                                     const void* const* v_pools, const int32_t* block_table,
                                     const int32_t* seq_lens, const int32_t* win_start, const int32_t* rope_pos0,
                                     void* q_out, int32_t* status, void* workspace, size_t workspace_bytes,
                                     void* stream) {
  Geom g;
  kara_status_t st = recompute_geom(p, n_trig, &g);
  if (st != KARA_OK) return st;
  if (!model_ok(m) || n_layers < 1) return KARA_ERR_INVALID_ARG;
  if (n_trig == 0) return KARA_OK;
  if (!trig || !weights || !hidden_in || !hidden_out || !k_pools || !v_pools || !block_table || !seq_lens ||
      !win_start || !rope_pos0 || !q_out || !status)
    return KARA_ERR_INVALID_ARG;
  for (int l = 0; l < n_layers; ++l) {
    const kara_layer_weights_t& w = weights[l];
    if (!w.w_q || !w.w_o || !w.w_gate || !w.w_up || !w.w_down || !w.g_attn || !w.g_ffn || !k_pools[l] ||
        !v_pools[l])
      return KARA_ERR_INVALID_ARG;
  }
  const int64_t T = (int64_t)n_trig * g.W;
  const int HD = g.Hq * g.d;
  if (T > INT32_MAX / 4 || (int64_t)n_trig * g.Hkv * ((int64_t)g.G * g.W + 127) / 128 > INT32_MAX)
    return KARA_ERR_INVALID_ARG;
  const RecomputeWs wl = recompute_ws(g, *m, n_trig);
  if (!workspace || workspace_bytes < wl.total) return KARA_ERR_WORKSPACE;
  rocblas_handle h = handle_for_current_device();
  if (!h) return KARA_ERR_HIP;
  hipStream_t s = (hipStream_t)stream;
  if (rocblas_set_stream(h, s) != rocblas_status_success) return KARA_ERR_HIP;
  char* ws = (char*)workspace;
  void* x = ws + wl.x;
  void* qraw = ws + wl.qraw;
  void* attn = ws + wl.attn;
  void* gate = ws + wl.gate;
  void* up = ws + wl.up;
  // the products' scratch is the caller's: size the products (a size query
  // launches nothing), then hand rocBLAS the slice
  {
    const kara_layer_weights_t& w = weights[0];
    if (rocblas_start_device_memory_size_query(h) != rocblas_status_success) return KARA_ERR_HIP;
    (void)gemm(h, T, HD, m->hidden, x, w.w_q, qraw, false);
    (void)gemm(h, T, m->hidden, HD, attn, w.w_o, hidden_out, true);
    (void)gemm(h, T, m->ffn, m->hidden, x, w.w_gate, gate, false);
    (void)gemm(h, T, m->hidden, m->ffn, gate, w.w_down, hidden_out, true);
    size_t need = 0;
    if (rocblas_stop_device_memory_size_query(h, &need) != rocblas_status_success) return KARA_ERR_HIP;
    if (need > kBlasWorkspace) return KARA_ERR_WORKSPACE;
    if (rocblas_set_workspace(h, ws + wl.blas, kBlasWorkspace) != rocblas_status_success) return KARA_ERR_HIP;
  }
  const size_t q_layer = (size_t)T * HD * 2;

  hipError_t e = launch_recompute_validate(g, trig, block_table, seq_lens, win_start, status, s);
  if (e == hipSuccess && hidden_out != hidden_in)
    e = hipMemcpyAsync(hidden_out, hidden_in, (size_t)T * m->hidden * sizeof(float), hipMemcpyDeviceToDevice, s);
  float* hs = hidden_out;
  for (int l = 0; l < n_layers && e == hipSuccess; ++l) {
    const kara_layer_weights_t& w = weights[l];
    void* ql = (char*)q_out + l * q_layer;
    e = launch_rmsnorm(hs, w.g_attn, x, T, m->hidden, m->rms_eps, s);
    if (e != hipSuccess) break;
    if (!gemm(h, T, HD, m->hidden, x, w.w_q, qraw, false)) return KARA_ERR_HIP;
    e = launch_rope(qraw, ql, n_trig, g.W, g.Hq, g.d, m->rope_theta, trig, rope_pos0, status, s);
    if (e == hipSuccess)
      e = launch_recompute_attention(g, ql, k_pools[l], v_pools[l], trig, block_table, win_start, attn, status, s);
    if (e != hipSuccess) break;
    if (!gemm(h, T, m->hidden, HD, attn, w.w_o, hs, true)) return KARA_ERR_HIP;
    e = launch_rmsnorm(hs, w.g_ffn, x, T, m->hidden, m->rms_eps, s);
    if (e != hipSuccess) break;
    if (!gemm(h, T, m->ffn, m->hidden, x, w.w_gate, gate, false)) return KARA_ERR_HIP;
    if (!gemm(h, T, m->ffn, m->hidden, x, w.w_up, up, false)) return KARA_ERR_HIP;
    e = launch_swiglu(gate, up, T * m->ffn, s);
    if (e != hipSuccess) break;
    if (!gemm(h, T, m->hidden, m->ffn, gate, w.w_down, hs, true)) return KARA_ERR_HIP;
  }
  return hip_status(e);
}

}  // extern "C"
