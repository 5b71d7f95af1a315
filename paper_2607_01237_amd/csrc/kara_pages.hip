// Paged-cache side of the step: window validation, the in-place window gather
// of Eq. (9) (Algorithm 1's MemoryCompaction) and the metadata update
// (UpdateMetadata: trailing blocks released, table and length rewritten).
#include "kara_internal.h"

namespace kara {
namespace {

// One workgroup per listed sequence.  Besides the window and page-range
// checks, no page of the blocks compaction writes ([p0/bs, ceil(len/bs)))
// may appear twice among the sequence's blocks [0, ceil(len/bs)): compaction
// moves rows in place, and a page mapped twice would be read and written by
// two workgroups at once.  keep_kept: a KARA_SEQ_BAD_KEPT bit already in
// status[t] survives (the staged per-layer calls of one event).
constexpr int kValidateThreads = 256;
constexpr int kValidateRowLds = 8192;   // table entries staged in LDS (32 KB)

__global__ __launch_bounds__(kValidateThreads) void validate_kernel(
    Geom g, const int32_t* __restrict__ trig, const int32_t* __restrict__ bt,
    const int32_t* __restrict__ seq_lens, const int32_t* __restrict__ win_start,
    int32_t* __restrict__ status, int keep_kept) {
  const int t = blockIdx.x;
  const int tid = threadIdx.x;
  const int kept_bit = keep_kept ? (status[t] & KARA_SEQ_BAD_KEPT) : 0;
  // every thread has read status[t] before thread 0 rewrites it
  __syncthreads();
  const int s = trig[t];
  if (s < 0 || s >= g.n_seqs) {
    if (tid == 0) status[t] = KARA_SEQ_BAD_INDEX | kept_bit;
    return;
  }
  int dup = 0;
  for (int o = tid; o < g.n_trig; o += kValidateThreads)
    if (o != t && trig[o] == s) dup = 1;
  const int st0 = (__syncthreads_or(dup) ? KARA_SEQ_DUP_TRIGGER : 0) | kept_bit;
  const int p0 = win_start[s];
  const int len = seq_lens[s];
  // the windows cover [p0, p0 + (n_win-1)*N + W)
  if (p0 < 0 || (int64_t)p0 + (int64_t)(g.n_win - 1) * g.N + g.W > (int64_t)len ||
      (int64_t)len > (int64_t)g.max_blocks * g.bs) {
    if (tid == 0) status[t] = st0 | KARA_SEQ_BAD_WINDOW;
    return;
  }
  const int32_t* row = bt + (int64_t)s * g.max_blocks;
  const int b0 = p0 / g.bs;
  const int b1 = (len + g.bs - 1) / g.bs;
  // the table row in LDS when it fits (the pairwise scan reads it often)
  __shared__ int32_t row_lds[kValidateRowLds];
  const bool in_lds = b1 <= kValidateRowLds;
  if (in_lds)
    for (int b = tid; b < b1; b += kValidateThreads) row_lds[b] = row[b];
  __syncthreads();
  int bad = 0, twice = 0;
  for (int b = b0 + tid; b < b1; b += kValidateThreads) {
    const int pg = in_lds ? row_lds[b] : row[b];
    if (pg < 0 || pg >= g.num_pages) {
      bad = 1;
      continue;
    }
    if (in_lds) {
      for (int c = 0; c < b; ++c) twice |= row_lds[c] == pg;
    } else {
      for (int c = 0; c < b; ++c) twice |= row[c] == pg;
    }
  }
  const int st = st0 | (__syncthreads_or(bad) ? KARA_SEQ_BAD_PAGE : 0) |
                 (__syncthreads_or(twice) ? KARA_SEQ_DUP_PAGE : 0);
  if (tid == 0) status[t] = st;
}

// Flags triggered sequences whose kept rows (caller-supplied) are not a
// strictly ascending subset of [0, N); one workgroup per unit
// ((layer, trigger, window, head)).
__global__ void check_kept_kernel(Geom g, int n_layers, const int32_t* __restrict__ kept,
                                  int32_t* __restrict__ status) {
  const int64_t u = blockIdx.x;
  const int t = (int)((u / ((int64_t)g.Hkv * g.n_win)) % g.n_trig);
  const int32_t* kr = kept + u * g.budget;
  int bad = 0;
  for (int j = threadIdx.x; j < g.budget; j += blockDim.x) {
    const int v = kr[j];
    if (v < 0 || v >= g.N || (j > 0 && kr[j - 1] >= v)) bad = 1;
  }
  if (__syncthreads_or(bad) && threadIdx.x == 0) atomicOr(&status[t], KARA_SEQ_BAD_KEPT);
}

constexpr int kCompactThreads = 256;
constexpr int kCompactUnroll = 8;

// Compaction touches each row once and nothing reads it back in the same
// step, so its loads and stores are nontemporal (streamed past the caches).
// On 64 x 40 x 8 units of W = 2048 (8.75 GB of moved rows, read and write)
// back to back: 2.12 -> 1.89 ms; after the step's scoring: 1.97 -> 1.95 ms.
// Staging a unit's row sources and block-table slice in LDS, so that a
// tile's row addresses need no dependent global reads, and 128-row tiles:
// 2.0-2.1 -> 1.52-1.55 ms after scoring.
constexpr int kCompactStageBytes = 32768;   // LDS limit of the staged instance
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// One workgroup per ((layer, trigger, head), K|V).  Destination row j
// (relative to the first window's start p0) takes source row m(j): for the
// n_win windows in turn (window w's compressible rows start at w*N) its kept
// rows w*N + kept_w[.], then everything after the last window's compressible
// region -- its buffer and the tail -- in order.  (One window: kept, buffer,
// tail.)  m is strictly increasing with m(j) >= j, so processing destination
// tiles in ascending order -- every source of a tile loaded before any row of
// it is stored -- never overwrites a row still to be read.
//
// STAGED: the workgroup first copies the kept rows' sources m(j), j <
// kept_rows, and the block-table entries of the blocks holding rows p0 ..
// seq_len - 1 into LDS (dynamic, (n_win * budget + max_blocks) words at
// most); without it every tile reads the kept indices and then the table
// from global memory before its row loads can issue.
template <bool STAGED>
__global__ __launch_bounds__(kCompactThreads) void compact_kernel(
    Geom g, const int32_t* __restrict__ trig, const int32_t* __restrict__ kept, PoolPtrs kp,
    PoolPtrs vp, const int32_t* __restrict__ bt, const int32_t* __restrict__ seq_lens,
    const int32_t* __restrict__ win_start, const int32_t* __restrict__ status) {
  const int64_t bid = blockIdx.x;
  const int kv = (int)(bid & 1);
  const int64_t u = bid >> 1;
  const int h = (int)(u % g.Hkv);
  const int t = (int)((u / g.Hkv) % g.n_trig);
  const int l = (int)(u / ((int64_t)g.Hkv * g.n_trig));
  if (status[t] != 0) return;
  const int s = trig[t];
  const int p0 = win_start[s];
  const int kept_rows = g.n_win * g.budget;
  const int comp_rows = g.n_win * g.N;
  const int n_dst = seq_lens[s] - p0 - (comp_rows - kept_rows);
  // kept rows of window w: kr + w * Hkv * budget ([l][t][w][h][budget])
  const int32_t* __restrict__ kr = kept + (((int64_t)l * g.n_trig + t) * g.n_win * g.Hkv + h) * g.budget;
  const int64_t kr_win = (int64_t)g.Hkv * g.budget;
  char* base = (char*)(kv ? vp.p[l] : kp.p[l]);
  const int32_t* __restrict__ row_pages = bt + (int64_t)s * g.max_blocks;
  const int row_bytes = g.d * g.esize;
  const int cpr = row_bytes >> 4;          // 16-byte chunks per row
  const int rpp = kCompactThreads / cpr;   // rows per pass
  const int tile = rpp * kCompactUnroll;
  const int c = threadIdx.x % cpr;
  const int r = threadIdx.x / cpr;

  extern __shared__ int32_t cstage[];
  const int pb0 = p0 / g.bs;
  if constexpr (STAGED) {
    // the kept rows' sources and the block-table slice the rows live in, in
    // LDS: the tile loop's addresses then need no global reads
    for (int j = threadIdx.x; j < kept_rows; j += blockDim.x) {
      const int w = g.n_win == 1 ? 0 : j / g.budget;
      cstage[j] = w * g.N + kr[w * kr_win + (j - w * g.budget)];
    }
    const int nb = (seq_lens[s] - 1) / g.bs - pb0 + 1;
    for (int b = threadIdx.x; b < nb; b += blockDim.x) cstage[kept_rows + b] = row_pages[pb0 + b];
    __syncthreads();
  }
  auto row_addr = [&](int x) -> char* {
    const int pos = p0 + x;
    const int64_t page = STAGED ? cstage[kept_rows + pos / g.bs - pb0] : row_pages[pos / g.bs];
    return base + ((page * g.Hkv + h) * g.bs + pos % g.bs) * (int64_t)row_bytes + c * 16;
  };

  for (int x0 = 0; x0 < n_dst; x0 += tile) {
    u32x4 v[kCompactUnroll];
    int dst[kCompactUnroll];
#pragma unroll
    for (int k = 0; k < kCompactUnroll; ++k) {
      const int j = x0 + k * rpp + r;
      dst[k] = -1;
      if (j < n_dst) {
        int src;
        if (j < kept_rows) {
          if constexpr (STAGED) {
            src = cstage[j];
          } else {
            const int w = g.n_win == 1 ? 0 : j / g.budget;
            src = w * g.N + kr[w * kr_win + (j - w * g.budget)];
          }
        } else {
          src = comp_rows + (j - kept_rows);
        }
        if (src != j) {
          dst[k] = j;
          v[k] = __builtin_nontemporal_load((const u32x4*)row_addr(src));
        }
      }
    }
    // all of this tile's loads have landed before any thread stores
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
#pragma unroll
    for (int k = 0; k < kCompactUnroll; ++k)
      if (dst[k] >= 0) __builtin_nontemporal_store(v[k], (u32x4*)row_addr(dst[k]));
  }
}

__global__ void commit_kernel(Geom g, const int32_t* __restrict__ trig, int32_t* __restrict__ bt,
                              int32_t* __restrict__ seq_lens, int32_t* __restrict__ freed,
                              int32_t* __restrict__ n_freed, const int32_t* __restrict__ status) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= g.n_trig) return;
  int32_t* fr = freed + (int64_t)t * g.max_blocks;
  if (status[t] != 0) {
    n_freed[t] = 0;
    for (int b = 0; b < g.max_blocks; ++b) fr[b] = -1;
    return;
  }
  const int s = trig[t];
  const int len = seq_lens[s];
  const int new_len = len - g.n_win * (g.N - g.budget);
  const int old_b = (len + g.bs - 1) / g.bs;
  const int new_b = (new_len + g.bs - 1) / g.bs;
  int32_t* row = bt + (int64_t)s * g.max_blocks;
  int c = 0;
  for (int b = new_b; b < old_b; ++b) {
    fr[c++] = row[b];
    row[b] = -1;
  }
  for (; c < g.max_blocks; ++c) fr[c] = -1;
  n_freed[t] = old_b - new_b;
  seq_lens[s] = new_len;
}

}  // namespace

hipError_t launch_validate(const Geom& g, const int32_t* trig, const int32_t* block_table,
                           const int32_t* seq_lens, const int32_t* win_start, int32_t* status,
                           bool keep_kept, hipStream_t stream) {
  if (g.n_trig == 0) return hipSuccess;
  hipLaunchKernelGGL(validate_kernel, dim3((unsigned)g.n_trig), dim3(kValidateThreads), 0, stream, g, trig,
                     block_table, seq_lens, win_start, status, keep_kept ? 1 : 0);
  return hipGetLastError();
}

hipError_t launch_check_kept(const Geom& g, int n_layers, const int32_t* kept, int32_t* status,
                             hipStream_t stream) {
  const int64_t units = (int64_t)n_layers * g.n_trig * g.n_win * g.Hkv;
  hipLaunchKernelGGL(check_kept_kernel, dim3((unsigned)units), dim3(256), 0, stream, g, n_layers,
                     kept, status);
  return hipGetLastError();
}

hipError_t launch_compact(const Geom& g, int n_layers, const int32_t* trig, const int32_t* kept,
                          const PoolPtrs& k_pools, const PoolPtrs& v_pools,
                          const int32_t* block_table, const int32_t* seq_lens,
                          const int32_t* win_start, const int32_t* status, hipStream_t stream) {
  const int64_t units = (int64_t)n_layers * g.n_trig * g.Hkv;
  const size_t lds = (size_t)(g.n_win * g.budget + g.max_blocks) * sizeof(int32_t);
  if (lds <= (size_t)kCompactStageBytes)
    hipLaunchKernelGGL(compact_kernel<true>, dim3((unsigned)(units * 2)), dim3(kCompactThreads), lds, stream, g,
                       trig, kept, k_pools, v_pools, block_table, seq_lens, win_start, status);
  else
    hipLaunchKernelGGL(compact_kernel<false>, dim3((unsigned)(units * 2)), dim3(kCompactThreads), 0, stream, g,
                       trig, kept, k_pools, v_pools, block_table, seq_lens, win_start, status);
  return hipGetLastError();
}

hipError_t launch_commit(const Geom& g, const int32_t* trig, int32_t* block_table,
                         int32_t* seq_lens, const int32_t* win_start, int32_t* freed,
                         int32_t* n_freed, const int32_t* status, hipStream_t stream) {
  (void)win_start;
  const int threads = 256;
  const int blocks = (g.n_trig + threads - 1) / threads;
  hipLaunchKernelGGL(commit_kernel, dim3(blocks), dim3(threads), 0, stream, g, trig, block_table,
                     seq_lens, freed, n_freed, status);
  return hipGetLastError();
}

}  // namespace kara
