// Per-unit selection on chip: discrete TopK (Eq. (5)), Token2Chunk
// (Eq. (6)-(8)) and the fill rule of App. C.3.  One workgroup per
// (sequence, layer, KV head); the unit's scores live in LDS.  Every ranking
// is exact and deterministic -- larger key first, lower position first among
// equal keys -- on order-preserving integer keys: a block-wide radix select
// for large counts, argmax rounds for the few chunks and fill positions
// usually asked for.
#include "kara_internal.h"

namespace kara {
namespace {

constexpr int kSelThreads = 256;
constexpr int kSelEptMax = KARA_MAX_COMPRESSIBLE / kSelThreads;  // positions per thread, at most
// Kernel instances: EPT positions per thread, 8 (windows of up to 2048
// compressible positions) or EPTMax; the smaller arrays keep more
// units in flight.
constexpr int kSelWaves = kSelThreads / 64;
constexpr uint32_t kArgmaxMax = 8;   // selections of at most this many items use argmax rounds

// Fixed part of the LDS; the unit's arrays follow it, sized by N and by the
// discrete set's size.
struct SelFixed {
  // radix histograms, one per wave (less atomic contention), in three
  // buffers: pass p counts into buffer p % 3 while the buffer of pass p + 2
  // is cleared, so a pass needs one barrier
  uint32_t hist[3][kSelWaves][256];
  uint32_t wsum[kSelWaves];
  uint64_t best_key[2][kSelWaves];   // argmax rounds: per-wave best, double-buffered
  int32_t best_pos[2][kSelWaves];
};

struct SelSmem {
  SelFixed* f;
  float* a;          // [N] scores
  int32_t* disc;     // [k] discrete positions, ascending
  uint8_t* mark;     // [N] bit0 discrete, bit1 chunk interior, bit2 fill
};

__host__ __device__ constexpr size_t align16(size_t x) { return (x + 15) & ~(size_t)15; }
__host__ __device__ inline size_t sel_lds_bytes(int N, int k) {
  return align16(sizeof(SelFixed)) + align16((size_t)N * 4) + align16((size_t)k * 4) + align16((size_t)N);
}

// Order-preserving maps to unsigned keys (larger value -> larger key); -0
// ranks equal to +0, as in a floating-point comparison.
__device__ inline uint32_t ord32(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) == 0) u = 0;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ inline uint64_t ord64(double x) {
  uint64_t u = (uint64_t)__double_as_longlong(x);
  if ((u & 0x7fffffffffffffffull) == 0) u = 0;
  return (u >> 63) ? ~u : (u | 0x8000000000000000ull);
}

// Eq. (6): chunk score from the fp32 endpoint scores, in fp64 (the sum of two
// fp32 values and its product with a small integer round the same way on
// every IEEE implementation; no contraction).
__device__ inline double chunk_score(float a_lo, float a_hi, int gap) {
#pragma clang fp contract(off)
  const double s = (double)a_lo + (double)a_hi;
  return s * (double)(gap - 1);
}

// Cross-lane steps use DPP row operations (16-lane rows, a few cycles each)
// and readlane, not LDS-routed shuffles.
constexpr int kDppRowShr1 = 0x111, kDppRowShr2 = 0x112, kDppRowShr4 = 0x114, kDppRowShr8 = 0x118;
constexpr int kDppQuadXor1 = 0xB1, kDppQuadXor2 = 0x4E, kDppRowHalfMirror = 0x141, kDppRowMirror = 0x140;

__device__ inline uint32_t dpp_u32(uint32_t v, int ctrl) {
  switch (ctrl) {
    case kDppRowShr1: return __builtin_amdgcn_update_dpp(0u, v, kDppRowShr1, 0xf, 0xf, true);
    case kDppRowShr2: return __builtin_amdgcn_update_dpp(0u, v, kDppRowShr2, 0xf, 0xf, true);
    case kDppRowShr4: return __builtin_amdgcn_update_dpp(0u, v, kDppRowShr4, 0xf, 0xf, true);
    case kDppRowShr8: return __builtin_amdgcn_update_dpp(0u, v, kDppRowShr8, 0xf, 0xf, true);
    case kDppQuadXor1: return __builtin_amdgcn_update_dpp(0u, v, kDppQuadXor1, 0xf, 0xf, true);
    case kDppQuadXor2: return __builtin_amdgcn_update_dpp(0u, v, kDppQuadXor2, 0xf, 0xf, true);
    case kDppRowHalfMirror: return __builtin_amdgcn_update_dpp(0u, v, kDppRowHalfMirror, 0xf, 0xf, true);
    default: return __builtin_amdgcn_update_dpp(0u, v, kDppRowMirror, 0xf, 0xf, true);
  }
}

// Inclusive prefix sum over the 64 lanes: within each 16-lane row by
// shifted adds (lanes shifted in from outside the row read 0), then each
// row adds the totals of the rows before it.
__device__ inline uint32_t wave_incl_scan(uint32_t v) {
  v += dpp_u32(v, kDppRowShr1);
  v += dpp_u32(v, kDppRowShr2);
  v += dpp_u32(v, kDppRowShr4);
  v += dpp_u32(v, kDppRowShr8);
  const uint32_t r0 = __builtin_amdgcn_readlane(v, 15), r1 = __builtin_amdgcn_readlane(v, 31),
                 r2 = __builtin_amdgcn_readlane(v, 47);
  const int row = (threadIdx.x & 63) >> 4;
  return v + (row >= 1 ? r0 : 0u) + (row >= 2 ? r1 : 0u) + (row >= 3 ? r2 : 0u);
}

// Maximum over the 64 lanes, the same in every lane: a butterfly within
// each row (neighbours, pairs, the row's mirror halves), then the four rows.
__device__ inline uint32_t umax32(uint32_t a, uint32_t b) { return a > b ? a : b; }

__device__ inline uint32_t wave_max_u32(uint32_t v) {
  v = umax32(v, dpp_u32(v, kDppQuadXor1));
  v = umax32(v, dpp_u32(v, kDppQuadXor2));
  v = umax32(v, dpp_u32(v, kDppRowHalfMirror));
  v = umax32(v, dpp_u32(v, kDppRowMirror));
  return umax32(umax32((uint32_t)__builtin_amdgcn_readlane(v, 0), (uint32_t)__builtin_amdgcn_readlane(v, 16)),
                umax32((uint32_t)__builtin_amdgcn_readlane(v, 32), (uint32_t)__builtin_amdgcn_readlane(v, 48)));
}

// Exclusive prefix sum over threads in index order; *total = block sum.
__device__ uint32_t block_excl_scan(uint32_t v, SelFixed& f, uint32_t* total) {
  const uint32_t inc = wave_incl_scan(v);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 63) f.wsum[w] = inc;
  __syncthreads();
  uint32_t off = 0, tot = 0;
#pragma unroll
  for (int i = 0; i < kSelWaves; ++i) {
    const uint32_t x = f.wsum[i];
    off += (i < w) ? x : 0u;
    tot += x;
  }
  __syncthreads();
  *total = tot;
  return off + inc - v;
}

// Marks in sel[] the K best eligible items -- larger key first, lower
// position first among equal keys -- where thread i owns positions
// [i*ept, i*ept+ept).  MSB-first radix select over 8-bit digits finds the
// K-th key; items equal to it are then taken in position order.  When the
// K-th key's bin holds exactly the items still needed, every item of the
// bin is selected and the lower digits need no pass.
template <int EPT, typename KeyT>
__device__ void radix_top(const KeyT (&key)[EPT], const bool (&elig)[EPT], bool (&sel)[EPT],
                          uint32_t K, SelFixed& f) {
  constexpr int kBits = sizeof(KeyT) * 8;
  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  // the first two passes' histograms start cleared
  *(uint4*)&f.hist[0][tid >> 6][(tid & 63) * 4] = uint4{0u, 0u, 0u, 0u};
  *(uint4*)&f.hist[1][tid >> 6][(tid & 63) * 4] = uint4{0u, 0u, 0u, 0u};
  __syncthreads();
  KeyT prefix = 0;
  uint32_t remaining = K;
  int whole_bin = -1;   // the digit shift of a bin taken whole, if any
  int pass = 0;
  for (int shift = kBits - 8; shift >= 0; shift -= 8, ++pass) {
    uint32_t(&hist)[kSelWaves][256] = f.hist[pass % 3];
    // a thread's positions often share a digit (the top digits of nearby
    // scores): add runs of equal digits with one atomic
    uint32_t run_bin = 0, run = 0;
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
      if (!elig[e]) continue;
      const bool match = (shift == kBits - 8) || (((key[e] ^ prefix) >> (shift + 8)) == 0);
      if (!match) continue;
      const uint32_t b = (uint32_t)(key[e] >> shift) & 255u;
      if (run && b == run_bin) {
        ++run;
      } else {
        if (run) atomicAdd(&hist[wave][run_bin], run);
        run_bin = b;
        run = 1;
      }
    }
    if (run) atomicAdd(&hist[wave][run_bin], run);
    __syncthreads();
    // Every wave scans all 256 bins, largest first (lane l holds bins
    // 255 - 4l down to 252 - 4l), and finds the bin of the remaining-th
    // item itself: the same result in every wave, with no exchange.
    const int b0 = 252 - 4 * lane;
    uint4 c = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int w = 0; w < kSelWaves; ++w) {
      const uint4 v = *(const uint4*)&hist[w][b0];
      c.x += v.x;
      c.y += v.y;
      c.z += v.z;
      c.w += v.w;
    }
    // the buffer of pass + 2 was last read by pass - 1, before this pass's barrier
    *(uint4*)&f.hist[(pass + 2) % 3][tid >> 6][(tid & 63) * 4] = uint4{0u, 0u, 0u, 0u};
    const uint32_t tot = c.x + c.y + c.z + c.w;
    const uint32_t incl = wave_incl_scan(tot);
    const uint32_t above = incl - tot;   // items in the bins above this lane's
    const bool holder = above < remaining && remaining <= incl;
    uint32_t bin = 0, need = 0, in_bin = 0;
    if (holder) {
      uint32_t a = above;
      if (remaining <= a + c.w) {
        bin = b0 + 3, need = remaining - a, in_bin = c.w;
      } else if (a += c.w, remaining <= a + c.z) {
        bin = b0 + 2, need = remaining - a, in_bin = c.z;
      } else if (a += c.z, remaining <= a + c.y) {
        bin = b0 + 1, need = remaining - a, in_bin = c.y;
      } else {
        a += c.y;
        bin = b0, need = remaining - a, in_bin = c.x;
      }
    }
    const int src = (int)__builtin_ctzll(__ballot(holder));
    bin = (uint32_t)__builtin_amdgcn_readlane((int)bin, src);
    need = (uint32_t)__builtin_amdgcn_readlane((int)need, src);
    in_bin = (uint32_t)__builtin_amdgcn_readlane((int)in_bin, src);
    prefix |= (KeyT)bin << shift;
    remaining = need;
    if (in_bin == need) {   // (uniform)
      whole_bin = shift;
      break;
    }
  }
  if (whole_bin >= 0) {
    // the items above the bin and the whole bin: top digits >= the prefix's
#pragma unroll
    for (int e = 0; e < EPT; ++e) sel[e] = elig[e] && (key[e] >> whole_bin) >= (prefix >> whole_bin);
    return;
  }
  uint32_t eq = 0;
#pragma unroll
  for (int e = 0; e < EPT; ++e) eq += (elig[e] && key[e] == prefix) ? 1u : 0u;
  uint32_t tot;
  uint32_t rank = block_excl_scan(eq, f, &tot);
#pragma unroll
  for (int e = 0; e < EPT; ++e) {
    const bool is_eq = elig[e] && key[e] == prefix;
    sel[e] = (elig[e] && key[e] > prefix) || (is_eq && rank < remaining);
    rank += is_eq ? 1u : 0u;
  }
}

// (key, pos) ordering of the rankings: a beats b
__device__ inline bool beats(uint64_t ka, int pa, uint64_t kb, int pb) {
  return ka > kb || (ka == kb && pa < pb);
}

// The same selection as radix_top for small K: K rounds, each taking the best
// remaining item (a block argmax over (key desc, position asc)).
template <int EPT, typename KeyT>
__device__ void argmax_top(const KeyT (&key)[EPT], const bool (&elig)[EPT], bool (&sel)[EPT],
                           uint32_t K, int base, SelFixed& f) {
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
#pragma unroll
  for (int e = 0; e < EPT; ++e) sel[e] = false;
  for (uint32_t r = 0; r < K; ++r) {
    // this thread's best: positions ascend with e, so the first maximum wins ties
    uint64_t bk = 0;
    int bp = 0x7fffffff;
#pragma unroll
    for (int e = 0; e < EPT; ++e)
      if (elig[e] && !sel[e] && beats((uint64_t)key[e], base + e, bk, bp)) {
        bk = (uint64_t)key[e];
        bp = base + e;
      }
    // the wave's best: the largest key (high word, then low word among the
    // lanes holding the largest high word), then the lowest lane holding it;
    // lanes own ascending blocks of positions, so that lane's position is
    // the lowest among equal keys
    {
      const uint32_t hi = wave_max_u32((uint32_t)(bk >> 32));
      const uint32_t lo = wave_max_u32((uint32_t)(bk >> 32) == hi ? (uint32_t)bk : 0u);
      const uint64_t wk = ((uint64_t)hi << 32) | lo;
      const uint64_t owners = __ballot(bk == wk);
      const int src = (int)__builtin_ctzll(owners);
      bk = wk;
      bp = __builtin_amdgcn_readlane(bp, src);
    }
    const int slot = r & 1;
    if (lane == 0) {
      f.best_key[slot][wave] = bk;
      f.best_pos[slot][wave] = bp;
    }
    __syncthreads();   // the other slot is rewritten only after the next round's barrier
    uint64_t gk = f.best_key[slot][0];
    int gp = f.best_pos[slot][0];
#pragma unroll
    for (int w = 1; w < kSelWaves; ++w)
      if (beats(f.best_key[slot][w], f.best_pos[slot][w], gk, gp)) {
        gk = f.best_key[slot][w];
        gp = f.best_pos[slot][w];
      }
    if (gp == 0x7fffffff) break;   // nothing eligible is left
    // only the owner marks it (other threads' slots past their own positions
    // are never eligible)
    const int e = gp - base;
#pragma unroll
    for (int i = 0; i < EPT; ++i)
      if (i == e && elig[i]) sel[i] = true;
  }
}

template <int EPT, typename KeyT>
__device__ void select_top(const KeyT (&key)[EPT], const bool (&elig)[EPT], bool (&sel)[EPT],
                           uint32_t K, int base, SelFixed& f) {
  uint32_t cnt = 0;
#pragma unroll
  for (int e = 0; e < EPT; ++e) cnt += elig[e] ? 1u : 0u;
  uint32_t n_el;
  block_excl_scan(cnt, f, &n_el);
  if (K >= n_el || K == 0) {
#pragma unroll
    for (int e = 0; e < EPT; ++e) sel[e] = K != 0 && elig[e];
    return;
  }
  if (K <= kArgmaxMax) argmax_top<EPT>(key, elig, sel, K, base, f);
  else radix_top<EPT>(key, elig, sel, K, f);
}

template <int EPT>
__global__ __launch_bounds__(kSelThreads) void select_kernel(
    Geom g, int mode, const float* __restrict__ scores, const int32_t* __restrict__ disc_in,
    int32_t* __restrict__ disc_out, int32_t* __restrict__ kept_out) {
  extern __shared__ __attribute__((aligned(16))) char sel_lds[];
  const int N = g.N;
  SelSmem sm;
  sm.f = (SelFixed*)sel_lds;
  sm.a = (float*)(sel_lds + align16(sizeof(SelFixed)));
  sm.disc = (int32_t*)((char*)sm.a + align16((size_t)N * 4));
  sm.mark = (uint8_t*)((char*)sm.disc + align16((size_t)g.k_disc * 4));
  SelFixed& f = *sm.f;

  const int64_t u = blockIdx.x;
  const int tid = threadIdx.x;
  const int k = g.k_disc;

  for (int j = tid; j < N; j += kSelThreads) {
    sm.a[j] = scores[u * N + j];
    sm.mark[j] = 0;
  }
  __syncthreads();

  const int ept = (N + kSelThreads - 1) / kSelThreads;
  const int base = tid * ept;
  uint32_t key[EPT];
  bool elig[EPT], sel[EPT];

  if (mode & kSelectDiscrete) {
    // Eq. (5): the budget - alpha best positions, kept ascending
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
      const int j = base + e;
      elig[e] = e < ept && j < N;
      key[e] = elig[e] ? ord32(sm.a[j]) : 0u;
    }
    select_top<EPT>(key, elig, sel, (uint32_t)k, base, f);
    uint32_t c = 0;
#pragma unroll
    for (int e = 0; e < EPT; ++e) c += sel[e] ? 1u : 0u;
    uint32_t tot;
    uint32_t r = block_excl_scan(c, f, &tot);
#pragma unroll
    for (int e = 0; e < EPT; ++e)
      if (sel[e]) {
        const int j = base + e;
        sm.disc[r] = j;
        sm.mark[j] = 1;
        if (disc_out) disc_out[u * k + r] = j;
        ++r;
      }
  } else {
    int bad = 0;
    for (int i = tid; i < k; i += kSelThreads) {
      const int v = disc_in[u * k + i];
      sm.disc[i] = v;
      if (v < 0 || v >= N) bad = 1;
    }
    __syncthreads();
    for (int i = tid; i + 1 < k; i += kSelThreads)
      if (sm.disc[i] >= sm.disc[i + 1]) bad = 1;
    if (__syncthreads_or(bad)) {
      for (int i = tid; i < g.budget; i += kSelThreads) kept_out[u * g.budget + i] = -1;
      return;
    }
    for (int i = tid; i < k; i += kSelThreads) sm.mark[sm.disc[i]] = 1;
  }
  __syncthreads();
  if (!(mode & kSelectKept)) return;

  // Eq. (6)-(8): candidate chunk i spans (disc[i], disc[i+1]) when its length
  // with both endpoints is at most gamma and its interior is not empty; the
  // n_chunks best (R desc, i asc) add their interiors.
  uint32_t added_here = 0;
  if (g.n_chunks > 0 && k >= 2) {
    const int nc = k - 1;
    const int ept2 = (nc + kSelThreads - 1) / kSelThreads;
    const int base2 = tid * ept2;
    uint64_t key2[EPT];
    bool el2[EPT], s2[EPT];
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
      const int i = base2 + e;
      el2[e] = false;
      key2[e] = 0;
      if (e < ept2 && i < nc) {
        const int lo = sm.disc[i], hi = sm.disc[i + 1];
        const int gap = hi - lo;
        if (gap >= 2 && gap <= g.gamma - 1) {
          key2[e] = ord64(chunk_score(sm.a[lo], sm.a[hi], gap));
          el2[e] = true;
        }
      }
    }
    select_top<EPT>(key2, el2, s2, (uint32_t)g.n_chunks, base2, f);
#pragma unroll
    for (int e = 0; e < EPT; ++e)
      if (s2[e]) {
        const int i = base2 + e;
        const int lo = sm.disc[i], hi = sm.disc[i + 1];
        for (int x = lo + 1; x < hi; ++x) sm.mark[x] |= 2;
        added_here += (uint32_t)(hi - lo - 1);
      }
  }
  uint32_t added;
  block_excl_scan(added_here, f, &added);

  // App. C.3: top up to alpha added positions with the best unselected ones
  const int fill = g.alpha - (int)added;
  if (fill > 0) {
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
      const int j = base + e;
      elig[e] = e < ept && j < N && sm.mark[j] == 0;
      key[e] = elig[e] ? ord32(sm.a[j]) : 0u;
    }
    select_top<EPT>(key, elig, sel, (uint32_t)fill, base, f);
#pragma unroll
    for (int e = 0; e < EPT; ++e)
      if (sel[e]) sm.mark[base + e] |= 4;
  }
  __syncthreads();

  // the kept set, ascending
  uint32_t c = 0;
#pragma unroll
  for (int e = 0; e < EPT; ++e) {
    const int j = base + e;
    if (e < ept && j < N && sm.mark[j]) ++c;
  }
  uint32_t tot;
  uint32_t r = block_excl_scan(c, f, &tot);
#pragma unroll
  for (int e = 0; e < EPT; ++e) {
    const int j = base + e;
    if (e < ept && j < N && sm.mark[j]) kept_out[u * g.budget + r++] = j;
  }
}

}  // namespace

hipError_t launch_select(const Geom& g, int64_t n_units, int mode, const float* scores,
                         const int32_t* discrete_in, int32_t* discrete_out, int32_t* kept_out,
                         hipStream_t stream) {
  if (n_units <= 0) return hipSuccess;
  if (g.N <= 8 * kSelThreads)
    hipLaunchKernelGGL(select_kernel<8>, dim3((unsigned)n_units), dim3(kSelThreads), sel_lds_bytes(g.N, g.k_disc), stream,
                       g, mode, scores, discrete_in, discrete_out, kept_out);
  else
    hipLaunchKernelGGL(select_kernel<kSelEptMax>, dim3((unsigned)n_units), dim3(kSelThreads),
                       sel_lds_bytes(g.N, g.k_disc), stream, g, mode, scores, discrete_in, discrete_out, kept_out);
  return hipGetLastError();
}

}  // namespace kara
