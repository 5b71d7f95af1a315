// Window scoring, Eq. (4) of Kara: A = colsum(softmax(Q_W K_{W\U}^T / sqrt(d)))
// per (sequence, layer, KV head), all G query heads of the group acting as
// queries of their KV head.
//
// Single pass over the logits.  A workgroup of 8 waves owns 16*RG query rows
// at a time and all N = W-U keys, split over CG column groups (CG*RG = 8);
// every wave keeps its 16 x (16*NT) logit tile in registers.  The logits come
// from MFMA (bf16: v_mfma_f32_16x16x32_bf16, fp32: v_mfma_f32_16x16x4f32)
// with the keys read through the block table; row max and row sum are
// reduced across lanes with shuffles and across column groups through LDS;
// each lane then adds its rows' normalised probabilities to per-column
// register accumulators.  After its rows the workgroup reduces those
// accumulators in a fixed order and writes one partial column sum per row
// split; the selection kernel adds the splits in order.  No atomics touch
// floating-point data, so the scores are bit-reproducible.
#include "kara_internal.h"

namespace kara {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int kScoreThreads = 512;
constexpr int kScoreWaves = kScoreThreads / 64;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kNegInf = -__builtin_huge_valf();

struct ScoreArgs {
  Geom g;
  const char* q;              // [n_layers][n_trig][W][Hq][d]
  PoolPtrs k;                 // per-layer K pools
  const int32_t* trig;
  const int32_t* bt;
  const int32_t* win_start;
  const int32_t* status;
  float* partials;            // [units][n_splits][N]
  int n_splits, n_rb;
  int64_t n_blocks;
};

// Per-lane operand slice: lane group gq = lane/16 supplies head-dim elements
// [gq*d/4, (gq+1)*d/4) of its row, consumed k-step by k-step.  A (queries)
// and B (keys) use the same assignment, so every product q_c k_c enters the
// dot product exactly once.
template <int DT, int D>
struct Slice;

template <int D>
struct Slice<KARA_BF16, D> {
  static constexpr int kBytes = D / 4 * 2;
  static constexpr int kVec = kBytes / 16;   // 16-byte loads
  static constexpr int kSteps = kVec;        // one 8-element k-step per load
  uint4 v[kVec];
  __device__ void load(const char* p) {
#pragma unroll
    for (int i = 0; i < kVec; ++i) v[i] = ((const uint4*)p)[i];
  }
  __device__ void zero() {
#pragma unroll
    for (int i = 0; i < kVec; ++i) v[i] = make_uint4(0, 0, 0, 0);
  }
};

template <int D>
struct Slice<KARA_F32, D> {
  static constexpr int kBytes = D / 4 * 4;
  static constexpr int kVec = kBytes / 16;
  static constexpr int kSteps = D / 4;       // one element per k-step
  uint4 v[kVec];
  __device__ void load(const char* p) {
#pragma unroll
    for (int i = 0; i < kVec; ++i) v[i] = ((const uint4*)p)[i];
  }
  __device__ void zero() {
#pragma unroll
    for (int i = 0; i < kVec; ++i) v[i] = make_uint4(0, 0, 0, 0);
  }
};

template <int DT, int D>
__device__ inline floatx4 dot_tile(const Slice<DT, D>& qa, const Slice<DT, D>& kb, floatx4 acc) {
  if constexpr (DT == KARA_BF16) {
#pragma unroll
    for (int s = 0; s < Slice<DT, D>::kSteps; ++s) {
      bf16x8 a, b;
      __builtin_memcpy(&a, &qa.v[s], 16);
      __builtin_memcpy(&b, &kb.v[s], 16);
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc, 0, 0, 0);
    }
  } else {
    const float* a = (const float*)qa.v;
    const float* b = (const float*)kb.v;
#pragma unroll
    for (int s = 0; s < Slice<DT, D>::kSteps; ++s)
      acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[s], b[s], acc, 0, 0, 0);
  }
  return acc;
}

__device__ inline float max16(float v) {
#pragma unroll
  for (int o = 1; o < 16; o <<= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ inline float sum16(float v) {
#pragma unroll
  for (int o = 1; o < 16; o <<= 1) v += __shfl_xor(v, o, 64);
  return v;
}

template <int DT, int D, int NT, int CG>
__global__ __launch_bounds__(kScoreThreads) void score_kernel(ScoreArgs a) {
  constexpr int RG = kScoreWaves / CG;
  constexpr int ES = DT == KARA_BF16 ? 2 : 4;
  constexpr int NCOL = CG * NT * 16;       // padded columns of the workgroup
  using S = Slice<DT, D>;

  __shared__ float red_max[RG][CG][16];
  __shared__ float red_sum[RG][CG][16];
  __shared__ float part[4 * RG][NCOL];
  __shared__ int32_t pages[KARA_MAX_COMPRESSIBLE + 2];

  const Geom& g = a.g;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int cg = wave % CG;
  const int rg = wave / CG;
  const int gq = lane >> 4;     // lane group: rows 4*gq..4*gq+3 of the 16-row tile
  const int li = lane & 15;     // column (key) within a 16-key tile / row of the A operand

  // Blocks are dealt round-robin to the 8 XCDs; renumber so that the row
  // splits of one unit share an XCD (and its L2 copy of the unit's keys).
  int64_t bid = blockIdx.x;
  if ((a.n_blocks & 7) == 0) bid = (bid & 7) * (a.n_blocks >> 3) + (bid >> 3);
  const int64_t u = bid / a.n_splits;
  const int split = (int)(bid % a.n_splits);
  const int h = (int)(u % g.Hkv);
  const int t = (int)((u / g.Hkv) % g.n_trig);
  const int l = (int)(u / ((int64_t)g.Hkv * g.n_trig));
  const int N = g.N;
  float* out = a.partials + (u * a.n_splits + split) * (int64_t)N;

  if (a.status[t] != 0) {
    for (int j = tid; j < N; j += kScoreThreads) out[j] = 0.f;
    return;
  }
  const int s = a.trig[t];
  const int p0 = a.win_start[s];
  const int first_blk = p0 / g.bs;
  const int n_blk = (p0 + N - 1) / g.bs - first_blk + 1;
  const int32_t* row_pages = a.bt + (int64_t)s * g.max_blocks + first_blk;
  for (int i = tid; i < n_blk; i += kScoreThreads) pages[i] = row_pages[i];
  __syncthreads();

  const char* kpool = (const char*)a.k.p[l];
  const int64_t row_bytes = (int64_t)D * ES;
  const int slice_off = gq * S::kBytes;
  const int R = g.G * g.W;
  const char* qbase = a.q + ((int64_t)l * g.n_trig + t) * g.W * g.Hq * row_bytes + slice_off;
  const float c = g.scale * kLog2e;

  // this lane's keys: tile i covers keys (cg*NT + i)*16 + 0..15
  float cacc[NT];
#pragma unroll
  for (int i = 0; i < NT; ++i) cacc[i] = 0.f;

  const int rb0 = (int)((int64_t)split * a.n_rb / a.n_splits);
  const int rb1 = (int)((int64_t)(split + 1) * a.n_rb / a.n_splits);
  for (int rb = rb0; rb < rb1; ++rb) {
    const int row0 = (rb * RG + rg) * 16;
    // A operand: query row row0 + li (flattened (w, g), g fastest)
    S qa;
    {
      const int r = row0 + li;
      if (r < R) {
        const int w = r / g.G, gi = r - w * g.G;
        qa.load(qbase + ((int64_t)w * g.Hq + h * g.G + gi) * row_bytes);
      } else {
        qa.zero();
      }
    }
    floatx4 acc[NT];
#pragma unroll
    for (int i = 0; i < NT; ++i) {
      const int j = (cg * NT + i) * 16 + li;
      S kb;
      if (j < N) {
        const int pos = p0 + j;
        const int64_t page = pages[pos / g.bs - first_blk];
        kb.load(kpool + ((page * g.Hkv + h) * g.bs + pos % g.bs) * row_bytes + slice_off);
      } else {
        kb.zero();
      }
      acc[i] = dot_tile<DT, D>(qa, kb, floatx4{0.f, 0.f, 0.f, 0.f});
    }
    // columns past N take no part
#pragma unroll
    for (int i = 0; i < NT; ++i) {
      const int j = (cg * NT + i) * 16 + li;
      if (j >= N) acc[i] = floatx4{kNegInf, kNegInf, kNegInf, kNegInf};
    }
    // row max over this wave's columns, then over the column groups
    float m[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      float v = acc[0][q];
#pragma unroll
      for (int i = 1; i < NT; ++i) v = fmaxf(v, acc[i][q]);
      m[q] = max16(v);
    }
    if constexpr (CG > 1) {
      if (li == 0) {
#pragma unroll
        for (int q = 0; q < 4; ++q) red_max[rg][cg][gq * 4 + q] = m[q];
      }
      __syncthreads();
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float v = red_max[rg][0][gq * 4 + q];
#pragma unroll
        for (int o = 1; o < CG; ++o) v = fmaxf(v, red_max[rg][o][gq * 4 + q]);
        m[q] = v;
      }
    }
    // exp2((s - m) * scale * log2 e) and row sums
    float lsum[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float mc = m[q] * c;
      float sum = 0.f;
#pragma unroll
      for (int i = 0; i < NT; ++i) {
        const float e = __builtin_amdgcn_exp2f(acc[i][q] * c - mc);
        acc[i][q] = e;
        sum += e;
      }
      lsum[q] = sum16(sum);
    }
    if constexpr (CG > 1) {
      if (li == 0) {
#pragma unroll
        for (int q = 0; q < 4; ++q) red_sum[rg][cg][gq * 4 + q] = lsum[q];
      }
      __syncthreads();
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float v = red_sum[rg][0][gq * 4 + q];
#pragma unroll
        for (int o = 1; o < CG; ++o) v += red_sum[rg][o][gq * 4 + q];
        lsum[q] = v;
      }
    }
    // softmax weights of this lane's four rows (rows past R weigh nothing)
    float wr[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) wr[q] = (row0 + gq * 4 + q < R) ? 1.0f / lsum[q] : 0.f;
    // colsum: this lane's four rows of each of its columns
#pragma unroll
    for (int i = 0; i < NT; ++i) {
      float v = acc[i][0] * wr[0];
      v = fmaf(acc[i][1], wr[1], v);
      v = fmaf(acc[i][2], wr[2], v);
      v = fmaf(acc[i][3], wr[3], v);
      cacc[i] += v;
    }
  }

  // fixed-order reduction over the four lane groups and the row groups
#pragma unroll
  for (int i = 0; i < NT; ++i) part[rg * 4 + gq][(cg * NT + i) * 16 + li] = cacc[i];
  __syncthreads();
  for (int j = tid; j < N; j += kScoreThreads) {
    float v = part[0][j];
#pragma unroll
    for (int p = 1; p < 4 * RG; ++p) v += part[p][j];
    out[j] = v;
  }
}

template <int DT, int D, int NT, int CG>
hipError_t launch_cfg(const ScoreArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL((score_kernel<DT, D, NT, CG>), dim3((unsigned)a.n_blocks), dim3(kScoreThreads), 0,
                     stream, a);
  return hipGetLastError();
}

template <int DT, int D>
hipError_t launch_d(const ScoreArgs& a, const ScorePlan& sp, hipStream_t stream) {
  if (sp.nt == 8) return launch_cfg<DT, D, 8, 1>(a, stream);
  if (sp.nt == 16) return launch_cfg<DT, D, 16, 1>(a, stream);
  switch (sp.cg) {
    case 1: return launch_cfg<DT, D, 32, 1>(a, stream);
    case 2: return launch_cfg<DT, D, 32, 2>(a, stream);
    case 4: return launch_cfg<DT, D, 32, 4>(a, stream);
    default: return launch_cfg<DT, D, 32, 8>(a, stream);
  }
}

}  // namespace

ScorePlan plan_score(const Geom& g, int64_t n_units) {
  ScorePlan sp{};
  const int tiles = (g.N + 15) / 16;
  if (tiles <= 8) {
    sp.cg = 1; sp.nt = 8;
  } else if (tiles <= 16) {
    sp.cg = 1; sp.nt = 16;
  } else {
    sp.nt = 32;
    sp.cg = tiles <= 32 ? 1 : tiles <= 64 ? 2 : tiles <= 128 ? 4 : 8;
  }
  sp.rg = kScoreWaves / sp.cg;
  sp.n_cols = sp.cg * sp.nt * 16;
  const int64_t rows = (int64_t)g.G * g.W;
  sp.n_rb = (int)((rows + 16 * sp.rg - 1) / (16 * sp.rg));
  // enough workgroups to fill 256 CUs several times over
  const int64_t target = 2048;
  int64_t splits = (target + n_units - 1) / (n_units > 0 ? n_units : 1);
  if (splits < 1) splits = 1;
  if (splits > sp.n_rb) splits = sp.n_rb;
  sp.n_splits = (int)splits;
  return sp;
}

hipError_t launch_score(const Geom& g, const ScorePlan& sp, int n_layers, const void* q,
                        const PoolPtrs& k_pools, const int32_t* trig, const int32_t* block_table,
                        const int32_t* win_start, const int32_t* status, float* partials,
                        hipStream_t stream) {
  ScoreArgs a;
  a.g = g;
  a.q = (const char*)q;
  a.k = k_pools;
  a.trig = trig;
  a.bt = block_table;
  a.win_start = win_start;
  a.status = status;
  a.partials = partials;
  a.n_splits = sp.n_splits;
  a.n_rb = sp.n_rb;
  a.n_blocks = (int64_t)n_layers * g.n_trig * g.Hkv * sp.n_splits;
  if (a.n_blocks == 0) return hipSuccess;
  if (g.dtype == KARA_BF16) {
    if (g.d == 128) return launch_d<KARA_BF16, 128>(a, sp, stream);
    return launch_d<KARA_BF16, 64>(a, sp, stream);
  }
  if (g.d == 128) return launch_d<KARA_F32, 128>(a, sp, stream);
  return launch_d<KARA_F32, 64>(a, sp, stream);
}

}  // namespace kara
