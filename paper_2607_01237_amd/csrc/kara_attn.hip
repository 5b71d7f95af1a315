// Causal attention of the window queries over the paged cache, the attention
// step of the window recompute pass (App. C.2): window token w of a
// triggered sequence, at cache position p0 + w, attends to cache rows
// [0, p0 + w]; query head hq reads KV head hq / G.
//
// One workgroup of 4 waves owns 16*QT*4 query rows of one (sequence, KV
// head), rows ordered (window position, head in group), and streams the
// cache rows [0, p0 + last row's position] through LDS in 64-key chunks,
// double buffered: K as stored ([key][d], 16-byte chunks XOR-swizzled by
// row) and V transposed ([d][key], 8-byte units XOR-swizzled by row).
//
// Per chunk and 16-query tile a wave forms S^T = K Q^T with
// v_mfma_f32_16x16x32_bf16 (keys as the M dimension), so a lane holds four
// keys of one query: the online softmax needs one cross-lane maximum per
// chunk, and the probabilities, converted to bf16, are already the B
// operand of O^T += V^T P^T (the k index of that product runs over keys in
// the order the S^T tiles left them; V^T is read in the same order).  The
// row sums stay per lane until the end.
#include "kara_internal.h"
#include "kara_recompute.h"

namespace kara {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int kAttnThreads = 256;
constexpr int kAttnWaves = kAttnThreads / 64;
constexpr int kKeys = 64;                   // keys per chunk
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kNegInf = -__builtin_huge_valf();
constexpr float kMaxFloor = -1e30f;         // finite start of a running maximum

template <int D, int QT>
struct ACfg {
  static constexpr int kRowBytes = D * 2;
  static constexpr int kCPR = kRowBytes / 16;          // 16-byte chunks per row
  static constexpr int kKS = kCPR / 4;                 // k-steps of one dot product (per lane group)
  static constexpr int kDT = D / 16;                   // 16-row tiles of O^T
  static constexpr int kRowsWave = 16 * QT;
  static constexpr int kRowsWG = kAttnWaves * kRowsWave;
  static constexpr int kKBytes = kKeys * kRowBytes;    // one K chunk
  static constexpr int kVRow = kKeys * 2;              // one V^T row (d fixed): 128 bytes
  static constexpr int kVBytes = D * kVRow;
  static constexpr int kStage = kKBytes + kVBytes;
  static constexpr int kKLoads = kKeys * kCPR / kAttnThreads;        // 16-byte K loads per thread
  static constexpr int kVItems = (kKeys / 4) * kCPR;                 // (4-key unit, d chunk) items
  static_assert(kKLoads * kAttnThreads == kKeys * kCPR, "uniform K loads");
  static_assert(kVItems <= kAttnThreads, "one V item per thread at most");
};

struct AttnArgs {
  int W, Hq, Hkv, G, bs, max_blocks, n_trig;
  float c;                    // logit scale times log2(e)
  const char* q;              // [n_trig][W][Hq][d]
  const char* kpool;          // [pages][Hkv][bs][d]
  const char* vpool;
  const int32_t* trig;
  const int32_t* bt;
  const int32_t* win_start;
  const int32_t* status;
  char* out;                  // [n_trig][W][Hq][d]
  int n_rb;                   // row blocks per (sequence, KV head)
  int64_t n_blocks;
};

__device__ inline float wave_max4(float v) {
  // maximum over the four lane groups holding the same query
  v = fmaxf(v, __shfl_xor(v, 16, 64));
  v = fmaxf(v, __shfl_xor(v, 32, 64));
  return v;
}

template <int D, int QT>
__global__ __launch_bounds__(kAttnThreads) void attn_kernel(AttnArgs a) {
  using C = ACfg<D, QT>;
  __shared__ __attribute__((aligned(16))) char smem[2 * C::kStage];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int gq = lane >> 4;
  const int li = lane & 15;

  // blocks of one (sequence, KV head) together on one XCD, heaviest first
  int64_t bid = blockIdx.x;
  if ((a.n_blocks & 7) == 0) bid = (bid & 7) * (a.n_blocks >> 3) + (bid >> 3);
  const int64_t unit = bid / a.n_rb;
  const int rb = a.n_rb - 1 - (int)(bid % a.n_rb);
  const int h = (int)(unit % a.Hkv);
  const int t = (int)(unit / a.Hkv);
  if (a.status[t] != 0) return;
  const int s = a.trig[t];
  const int p0 = a.win_start[s];
  const int R = a.G * a.W;
  const int row0 = rb * C::kRowsWG;
  const int last_row = min(row0 + C::kRowsWG, R) - 1;
  const int kend = p0 + last_row / a.G + 1;           // keys this workgroup needs
  const int n_chunks = (kend + kKeys - 1) / kKeys;
  const int32_t* row_pages = a.bt + (int64_t)s * a.max_blocks;
  const int64_t head_stride = (int64_t)a.bs * C::kRowBytes;

  // ---- this wave's queries as B operands (lane: query li of each tile) ----
  const int wrow0 = row0 + wave * C::kRowsWave;
  uint4 qop[QT][C::kKS];
  int qpos[QT];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    const int r = min(wrow0 + qt * 16 + li, R - 1);
    const int w = r / a.G;
    const int hq = h * a.G + (r - w * a.G);
    qpos[qt] = p0 + w;
    const char* qrow = a.q + (((int64_t)t * a.W + w) * a.Hq + hq) * C::kRowBytes;
#pragma unroll
    for (int ks = 0; ks < C::kKS; ++ks) qop[qt][ks] = *(const uint4*)(qrow + (gq * C::kKS + ks) * 16);
  }
  const int wave_first_pos = p0 + min(wrow0, R - 1) / a.G;
  const int wave_last_pos = p0 + min(wrow0 + C::kRowsWave - 1, R - 1) / a.G;

  floatx4 o[QT][C::kDT];
  float m[QT], l[QT];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    m[qt] = kMaxFloor;
    l[qt] = 0.f;
#pragma unroll
    for (int dt = 0; dt < C::kDT; ++dt) o[qt][dt] = floatx4{0.f, 0.f, 0.f, 0.f};
  }

  // ---- staging of one chunk: global -> registers -> LDS ----
  uint4 kst[C::kKLoads];
  uint4 vst[4];
  const bool v_item = tid < C::kVItems;
  const int v_unit = tid / C::kCPR;       // keys 4*v_unit .. +3
  const int v_chunk = tid % C::kCPR;      // d 8*v_chunk .. +7
  auto row_ptr = [&](const char* pool, int pos) -> const char* {
    const int64_t page = row_pages[pos / a.bs];
    return pool + (page * a.Hkv + h) * head_stride + (int64_t)(pos % a.bs) * C::kRowBytes;
  };
  auto load_chunk = [&](int k0) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < C::kKLoads; ++j) {
      const int idx = j * kAttnThreads + tid;
      const int key = idx / C::kCPR, c = idx % C::kCPR;
      const int pos = k0 + key;
      kst[j] = pos < kend ? *(const uint4*)(row_ptr(a.kpool, pos) + c * 16) : uint4{0, 0, 0, 0};
    }
    if (v_item) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int pos = k0 + 4 * v_unit + i;
        vst[i] = pos < kend ? *(const uint4*)(row_ptr(a.vpool, pos) + v_chunk * 16) : uint4{0, 0, 0, 0};
      }
    }
  };
  auto store_chunk = [&](char* st) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < C::kKLoads; ++j) {
      const int idx = j * kAttnThreads + tid;
      const int key = idx / C::kCPR, c = idx % C::kCPR;
      *(uint4*)(st + key * C::kRowBytes + ((c ^ (key & (C::kCPR - 1))) * 16)) = kst[j];
    }
    if (v_item) {
      char* vt = st + C::kKBytes;
      const uint16_t* e0 = (const uint16_t*)&vst[0];
      const uint16_t* e1 = (const uint16_t*)&vst[1];
      const uint16_t* e2 = (const uint16_t*)&vst[2];
      const uint16_t* e3 = (const uint16_t*)&vst[3];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int d = v_chunk * 8 + e;
        uint2 packed;
        packed.x = (uint32_t)e0[e] | ((uint32_t)e1[e] << 16);
        packed.y = (uint32_t)e2[e] | ((uint32_t)e3[e] << 16);
        *(uint2*)(vt + d * C::kVRow + ((v_unit ^ (d & 15)) * 8)) = packed;
      }
    }
  };

  load_chunk(0);
  store_chunk(smem);
  __syncthreads();

  for (int ch = 0; ch < n_chunks; ++ch) {
    const int k0 = ch * kKeys;
    const bool more = ch + 1 < n_chunks;
    if (more) load_chunk(k0 + kKeys);
    const char* st = smem + (ch & 1) * C::kStage;
    if (k0 <= wave_last_pos) {
      const bool diag = k0 + kKeys - 1 > wave_first_pos;
      // S^T tiles: keys kt*16 + (4*gq + r), query li
      floatx4 sv[QT][4];
#pragma unroll
      for (int qt = 0; qt < QT; ++qt)
#pragma unroll
        for (int kt = 0; kt < 4; ++kt) sv[qt][kt] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kt = 0; kt < 4; ++kt) {
        const int key = kt * 16 + li;
#pragma unroll
        for (int ks = 0; ks < C::kKS; ++ks) {
          const int c = gq * C::kKS + ks;
          bf16x8 ka;
          __builtin_memcpy(&ka, st + key * C::kRowBytes + ((c ^ (key & (C::kCPR - 1))) * 16), 16);
#pragma unroll
          for (int qt = 0; qt < QT; ++qt) {
            bf16x8 qb;
            __builtin_memcpy(&qb, &qop[qt][ks], 16);
            sv[qt][kt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka, qb, sv[qt][kt], 0, 0, 0);
          }
        }
      }
      // online softmax per query (lane's query li of each tile)
      bf16x8 pb[QT][2];
#pragma unroll
      for (int qt = 0; qt < QT; ++qt) {
        float x[4][4];
        float cmax = kNegInf;
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            float v = sv[qt][kt][r] * a.c;
            if (diag && k0 + kt * 16 + 4 * gq + r > qpos[qt]) v = kNegInf;
            x[kt][r] = v;
            cmax = fmaxf(cmax, v);
          }
        cmax = wave_max4(cmax);
        const float mn = fmaxf(m[qt], cmax);
        const float alpha = exp2f(m[qt] - mn);
        m[qt] = mn;
        float lsum = 0.f;
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float p = exp2f(x[kt][r] - mn);
            lsum += p;
            pb[qt][kt >> 1][(kt & 1) * 4 + r] = (__bf16)p;
          }
        l[qt] = l[qt] * alpha + lsum;
#pragma unroll
        for (int dt = 0; dt < C::kDT; ++dt) o[qt][dt] *= alpha;
      }
      // O^T += V^T P^T, two 32-key halves
      const char* vt = st + C::kKBytes;
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int u1 = 8 * j + gq, u2 = 8 * j + 4 + gq;
#pragma unroll
        for (int dt = 0; dt < C::kDT; ++dt) {
          const int d = dt * 16 + li;
          const char* vrow = vt + d * C::kVRow;
          uint2 lo = *(const uint2*)(vrow + ((u1 ^ (d & 15)) * 8));
          uint2 hi = *(const uint2*)(vrow + ((u2 ^ (d & 15)) * 8));
          uint4 both{lo.x, lo.y, hi.x, hi.y};
          bf16x8 va;
          __builtin_memcpy(&va, &both, 16);
#pragma unroll
          for (int qt = 0; qt < QT; ++qt)
            o[qt][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, pb[qt][j], o[qt][dt], 0, 0, 0);
        }
      }
    }
    if (more) store_chunk(smem + ((ch + 1) & 1) * C::kStage);
    __syncthreads();
  }

  // ---- normalise and store: lane holds O^T[dt*16 + 4*gq + r][query li] ----
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    float lt = l[qt] + __shfl_xor(l[qt], 16, 64);
    lt += __shfl_xor(lt, 32, 64);
    const float inv = 1.f / lt;
    const int r = wrow0 + qt * 16 + li;
    if (r >= R) continue;
    const int w = r / a.G;
    const int hq = h * a.G + (r - w * a.G);
    char* orow = a.out + (((int64_t)t * a.W + w) * a.Hq + hq) * C::kRowBytes;
#pragma unroll
    for (int dt = 0; dt < C::kDT; ++dt) {
      bf16x4 v;
#pragma unroll
      for (int i = 0; i < 4; ++i) v[i] = (__bf16)(o[qt][dt][i] * inv);
      *(bf16x4*)(orow + (dt * 16 + 4 * gq) * 2) = v;
    }
  }
}

// Per triggered sequence: index in range, not listed twice, the window and
// every cache row before it inside the sequence, and every page of
// [0, p0 + W) inside the pool.
__global__ void attn_validate_kernel(int n_trig, int n_seqs, int W, int bs, int max_blocks, int num_pages,
                                     const int32_t* __restrict__ trig, const int32_t* __restrict__ bt,
                                     const int32_t* __restrict__ seq_lens, const int32_t* __restrict__ win_start,
                                     int32_t* __restrict__ status) {
  const int t = blockIdx.x;
  const int s = trig[t];
  __shared__ int st;
  if (threadIdx.x == 0) {
    st = 0;
    if (s < 0 || s >= n_seqs) {
      st = KARA_SEQ_BAD_INDEX;
    } else {
      for (int o = 0; o < n_trig; ++o)
        if (o != t && trig[o] == s) st |= KARA_SEQ_DUP_TRIGGER;
      const int p0 = win_start[s];
      const int len = seq_lens[s];
      if (p0 < 0 || (int64_t)p0 + W > (int64_t)len || (int64_t)len > (int64_t)max_blocks * bs)
        st |= KARA_SEQ_BAD_WINDOW;
    }
  }
  __syncthreads();
  if (st == 0) {
    const int nb = (win_start[s] + W + bs - 1) / bs;
    const int32_t* row = bt + (int64_t)s * max_blocks;
    int bad = 0;
    for (int b = threadIdx.x; b < nb; b += blockDim.x) {
      const int pg = row[b];
      if (pg < 0 || pg >= num_pages) bad = 1;
    }
    if (__syncthreads_or(bad) && threadIdx.x == 0) st = KARA_SEQ_BAD_PAGE;
  }
  __syncthreads();
  if (threadIdx.x == 0) status[t] = st;
}

template <int D, int QT>
hipError_t launch_attn_t(AttnArgs a, hipStream_t stream) {
  using C = ACfg<D, QT>;
  a.n_rb = (a.G * a.W + C::kRowsWG - 1) / C::kRowsWG;
  a.n_blocks = (int64_t)a.n_trig * a.Hkv * a.n_rb;
  if (a.n_blocks == 0) return hipSuccess;
  hipLaunchKernelGGL((attn_kernel<D, QT>), dim3((unsigned)a.n_blocks), dim3(kAttnThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_recompute_validate(const Geom& g, const int32_t* trig, const int32_t* block_table,
                                     const int32_t* seq_lens, const int32_t* win_start, int32_t* status,
                                     hipStream_t stream) {
  hipLaunchKernelGGL(attn_validate_kernel, dim3(g.n_trig), dim3(256), 0, stream, g.n_trig, g.n_seqs, g.W, g.bs,
                     g.max_blocks, g.num_pages, trig, block_table, seq_lens, win_start, status);
  return hipGetLastError();
}

hipError_t launch_recompute_attention(const Geom& g, const void* q, const void* k_pool, const void* v_pool,
                                      const int32_t* trig, const int32_t* block_table, const int32_t* win_start,
                                      void* out, const int32_t* status, hipStream_t stream) {
  AttnArgs a{};
  a.W = g.W;
  a.Hq = g.Hq;
  a.Hkv = g.Hkv;
  a.G = g.G;
  a.bs = g.bs;
  a.max_blocks = g.max_blocks;
  a.n_trig = g.n_trig;
  a.c = g.scale * kLog2e;
  a.q = (const char*)q;
  a.kpool = (const char*)k_pool;
  a.vpool = (const char*)v_pool;
  a.trig = trig;
  a.bt = block_table;
  a.win_start = win_start;
  a.status = status;
  a.out = (char*)out;
  if (g.d == 128) return launch_attn_t<128, 2>(a, stream);
  return launch_attn_t<64, 2>(a, stream);
}

}  // namespace kara
