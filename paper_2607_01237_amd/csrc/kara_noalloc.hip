// Allocation-free variant of kara_compress_window: the step's scratch (split
// partial column sums, and the scores and index sets the caller does not
// request) lives in a static device array of fixed size instead of a caller
// workspace.  For callers that cannot allocate device memory.
#include <mutex>

#include "kara_internal.h"

namespace {

// One copy per device, resident from module load until the process ends.
// In host code `scratch` names a host-side stand-in, not device memory: the
// device address comes from hipGetSymbolAddress, per device.
__device__ __align__(256) char scratch[KARA_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The array's address on the current device, resolved on first use with
// that device current; nullptr if it cannot be resolved.
void* scratch_on_current_device() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return nullptr;
    g_scratch_ptr[dev] = ptr;
  }
  return g_scratch_ptr[dev];
}

}  // namespace

extern "C" kara_status_t kara_compress_window_noalloc(
    const kara_params_t* p, int32_t n_trig, const int32_t* trig, int32_t n_layers, const void* q,
    void* const* k_pools, void* const* v_pools, int32_t* block_table, int32_t* seq_lens, const int32_t* win_start,
    int32_t commit, float* scores, int32_t* discrete, int32_t* kept, int32_t* freed, int32_t* n_freed,
    int32_t* status, void* stream) {
  kara::Geom g;
  kara_status_t st = kara::make_geom(p, n_trig, &g);
  if (st != KARA_OK) return st;
  if (n_layers < 1) return KARA_ERR_INVALID_ARG;
  if (n_trig == 0) return KARA_OK;
  const size_t need = kara::compress_workspace_bytes(g, n_layers);
  if (need > KARA_NOALLOC_SCRATCH_BYTES) return KARA_ERR_SCRATCH_LIMIT;
  void* ws = scratch_on_current_device();
  if (!ws) return KARA_ERR_SCRATCH_LIMIT;
  return kara::compress(p, n_trig, trig, 1, n_layers, q, k_pools, v_pools, block_table, seq_lens, win_start, commit,
                        scores, discrete, kept, freed, n_freed, status, ws, KARA_NOALLOC_SCRATCH_BYTES, stream);
}
