// Causal attention of the window queries over the paged cache, the attention
// step of the window recompute pass (App. C.2): window token w of a
// triggered sequence, at cache position p0 + w, attends to cache rows
// [0, p0 + w]; query head hq reads KV head hq / G.
//
// One workgroup of 8 waves owns 16*QT*8 query rows of one (sequence, KV
// head), rows ordered (window position, head in group), and streams the
// cache rows [0, p0 + last row's position] through a four-stage LDS ring in
// 64-key chunks, three chunks ahead of the one being worked on: K and V as
// stored ([key][d], 16-byte chunks XOR-swizzled by row; V is read through
// the transposed LDS load).  The pages of the rows come from a copy of the
// sequence's block-table row in LDS, so inside the chunk loop the only
// global memory operations are the copies, and the wait for a chunk counts
// exactly the copies issued after it.
//
// Per chunk and 16-query tile a wave forms S^T = K Q^T with
// v_mfma_f32_16x16x32_bf16 (keys as the M dimension), so a lane holds four
// keys of one query: the online softmax needs one cross-lane maximum per
// chunk, and the probabilities, converted to bf16, are already the B
// operand of O^T += V^T P^T (the k index of that product runs over keys in
// the order the S^T tiles left them; V^T is read in the same order).  The
// row sums come from the same product with an all-ones A operand, so the
// normalisation uses exactly the bf16 weights the numerator used.  The softmax reference maximum is
// raised lazily (only past a headroom of 2^8), which skips the rescaling of
// the accumulators on almost every chunk.  Exponentials are the bare
// v_exp_f32: arguments below the normal range flush to 0, which is the
// right weight there.
#include <type_traits>

#include "kara_internal.h"
#include "kara_recompute.h"

namespace kara {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int kAttnThreads = 512;
constexpr int kAttnWaves = kAttnThreads / 64;
constexpr int kKeys = 64;                   // keys per chunk
constexpr int kStages = 4;                  // LDS ring: chunks ch .. ch+3 resident or in flight
constexpr int kLookahead = kStages - 1;     // chunks copied ahead of the one being worked on
constexpr int kPageTbl = 2048;              // block-table entries held in LDS at a time
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kNegInf = -__builtin_huge_valf();
constexpr float kMaxFloor = -1e30f;         // finite start of a running maximum
constexpr float kHeadroom = 8.f;            // log2 units a row may exceed its reference maximum

template <int D, int QT>
struct ACfg {
  static constexpr int kRowBytes = D * 2;
  static constexpr int kCPR = kRowBytes / 16;          // 16-byte chunks per row
  static constexpr int kSwz = kCPR - 1;
  // XOR swizzles of a row's 16-byte chunks.  K (read 16 rows x 16 bytes per
  // lane group): by the row with its two low bits moved to the top.  V
  // (read through the transposed load, 32 lanes x 8 bytes at a time over 8
  // rows and two adjacent chunks): by twice the row (twice its half at
  // d = 64, whose rows are half a bank sweep), so the 16 (row, chunk) pairs
  // of such a read land in 16 distinct chunks.  Measured on gfx950 free of
  // bank conflicts (K at d = 64 and 128, V at d = 128); XOR by the row itself
  // costs about four conflict cycles per K read and two per V read.
  static __device__ __forceinline__ int swz_k(int row) {
    if constexpr (D == 128) return ((row & 3) << 2) | ((row >> 2) & 3);
    return ((row & 3) << 1) | ((row >> 2) & 1);
  }
  static __device__ __forceinline__ int swz_v(int row) { return (2 * (D == 128 ? row : row >> 1)) & kSwz; }
  static constexpr int kKS = kCPR / 4;                 // k-steps of one dot product (per lane group)
  static constexpr int kDT = D / 16;                   // 16-row tiles of O^T
  static constexpr int kRowsWave = 16 * QT;
  static constexpr int kRowsWG = kAttnWaves * kRowsWave;
  static constexpr int kKBytes = kKeys * kRowBytes;    // one chunk of K (or V) rows
  static constexpr int kStage = 2 * kKBytes;           // K rows, then V rows
  static constexpr int kCopies = kKBytes / (kAttnThreads * 16);      // 16-byte copies per thread per pool
  static constexpr int kPerChunk = 2 * kCopies;        // copy instructions per thread per chunk
  static_assert(kCopies * kAttnThreads * 16 == kKBytes, "uniform copies");
  static_assert(kStages * kStage + kPageTbl * 4 <= 160 * 1024, "LDS budget");
};

struct AttnArgs {
  int W, Hq, Hkv, G, bs, max_blocks, n_trig;
  int bs_shift;               // log2(bs) when bs is a power of two, else -1
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

// Direct global->LDS copy of 16 bytes per lane; lane i's bytes land at
// lds_wave_base + 16*i (global_load_lds_dwordx4, LDS base in M0).  Issued
// through inline assembly so the compiler adds no wait of its own before
// LDS reads; the kernel waits explicitly.  M0 is restored.
__device__ inline void copy16(const void* g, char* lds_wave_base) {
  const uint32_t lds = __builtin_amdgcn_readfirstlane(
      (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)lds_wave_base);
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %2\n\t"
      "global_load_lds_dwordx4 %1, off\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(g), "s"(lds)
      : "memory");
}

// Barrier for LDS traffic only (the copies it covers are waited for first).
__device__ inline void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

template <int N>
__device__ inline void wait_vm() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Wait for this thread's copies of a chunk when the copies of `newer` later
// chunks (0 .. kStages-2, run-time) were issued after them.
template <int kPerChunk>
__device__ inline void wait_chunk(int newer) {
  static_assert(kLookahead == 3, "wait_chunk covers up to two newer chunks");
  if (newer >= 2) {
    wait_vm<2 * kPerChunk>();
  } else if (newer == 1) {
    wait_vm<kPerChunk>();
  } else {
    wait_vm<0>();
  }
}

typedef short v4i16 __attribute__((ext_vector_type(4)));

// Transposed LDS read (gfx950): within each 16-lane group, lane 4j+e gets
// element e of the 4-element rows addressed by lanes j, j+4, j+8, j+12.
__device__ inline v4i16 read_tr(const char* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) v4i16*)(__attribute__((address_space(3))) char*)p);
}

template <int D, int QT>
__global__ __launch_bounds__(kAttnThreads, 1) void attn_kernel(AttnArgs a) {
  using C = ACfg<D, QT>;
  __shared__ __attribute__((aligned(16))) char smem[kStages * C::kStage];
  // row index (page*Hkv + h)*bs of slot 0 of the sequence's logical blocks
  // [pt_base, pt_base + kPageTbl), for this workgroup's KV head
  __shared__ uint32_t ptbl[kPageTbl];
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
  // consume the query loads before any copy is issued, so the compiler
  // waits for them here and not inside the chunk loop
#pragma unroll
  for (int qt = 0; qt < QT; ++qt)
#pragma unroll
    for (int ks = 0; ks < C::kKS; ++ks)
      asm volatile("" ::"v"(qop[qt][ks].x), "v"(qop[qt][ks].y), "v"(qop[qt][ks].z), "v"(qop[qt][ks].w));
  const int wave_first_pos = p0 + min(wrow0, R - 1) / a.G;
  const int wave_last_pos = p0 + min(wrow0 + C::kRowsWave - 1, R - 1) / a.G;

  // o: O^T tiles; l: the row sums, formed on the matrix cores as one more
  // 16-row tile whose A operand is all ones (every lane then holds its
  // query's sum of the bf16 weights PV used, four times)
  floatx4 o[QT][C::kDT], l[QT];
  float m[QT];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    m[qt] = kMaxFloor;
    l[qt] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int dt = 0; dt < C::kDT; ++dt) o[qt][dt] = floatx4{0.f, 0.f, 0.f, 0.f};
  }
  bf16x8 ones;
#pragma unroll
  for (int i = 0; i < 8; ++i) ones[i] = (__bf16)1.f;

  // ---- block-table segment in LDS, and copies ----
  // Chunk ch's rows are positions ch*64 .. ch*64+63 (past kend: row kend-1,
  // finite and masked for every query).  A chunk never straddles two
  // segments: a segment spans kPageTbl*bs positions, a multiple of 64.
  const int seg_pos = kPageTbl * a.bs;
  const int n_blk = (kend + a.bs - 1) / a.bs;
  int pt_base = -1;                      // first block held in ptbl (uniform)
  auto load_segment = [&](int seg) __attribute__((always_inline)) {
    pt_base = seg * kPageTbl;
    const int n = min(kPageTbl, n_blk - pt_base);
    for (int i = tid; i < n; i += kAttnThreads)
      ptbl[i] = (uint32_t)(((int64_t)row_pages[pt_base + i] * a.Hkv + h) * a.bs);
  };
  // copy r of this thread fills slot r*512 + tid of the K (V) region: row
  // kr = slot / kCPR, stored chunk slot % kCPR, fetched chunk (slot % kCPR)
  // ^ swz(kr)
  int kr_of[C::kCopies], chunk_k[C::kCopies], chunk_v[C::kCopies];
#pragma unroll
  for (int r = 0; r < C::kCopies; ++r) {
    const int slot = r * kAttnThreads + tid;
    kr_of[r] = slot / C::kCPR;
    chunk_k[r] = (slot % C::kCPR) ^ C::swz_k(kr_of[r]);
    chunk_v[r] = (slot % C::kCPR) ^ C::swz_v(kr_of[r]);
  }
  auto issue = [&](int ch) __attribute__((always_inline)) {
    if (ch * kKeys >= (pt_base + kPageTbl) * a.bs) {
      // next segment (rare): every earlier copy lands first, as the table's
      // loads are waited for with the compiler's own count
      wait_vm<0>();
      lds_barrier();
      load_segment(ch * kKeys / seg_pos);
      lds_barrier();
    }
    char* st = smem + (ch % kStages) * C::kStage;
#pragma unroll
    for (int r = 0; r < C::kCopies; ++r) {
      const int pos = min(ch * kKeys + kr_of[r], kend - 1);
      int blk, slot;
      if (a.bs_shift >= 0) {
        blk = pos >> a.bs_shift;
        slot = pos & (a.bs - 1);
      } else {
        blk = pos / a.bs;
        slot = pos - blk * a.bs;
      }
      const uint64_t row = (uint64_t)(ptbl[blk - pt_base] + (uint32_t)slot) * C::kCPR;
      copy16(a.kpool + (row + chunk_k[r]) * 16, st + (r * kAttnWaves + wave) * 1024);
      copy16(a.vpool + (row + chunk_v[r]) * 16, st + C::kKBytes + (r * kAttnWaves + wave) * 1024);
    }
  };

  load_segment(0);
  lds_barrier();
  for (int c = 0; c < kLookahead && c < n_chunks; ++c) issue(c);

  // Per-lane LDS byte offsets of the operand reads.  K operand rows are
  // 16*kt + li, so swz_k(row) = swz_k(li) and the swizzled chunk depends on
  // the lane and ks only; V rows read through the transposed load are
  // 32*j + 16*half + 4*gq + (li >> 2), and swz_v of such a row does not
  // depend on j or half.  The tile and half offsets are then compile-time
  // constants.
  int koff[C::kKS], voff[C::kDT];
#pragma unroll
  for (int ks = 0; ks < C::kKS; ++ks)
    koff[ks] = li * C::kRowBytes + (((gq * C::kKS + ks) ^ C::swz_k(li)) * 16);
  {
    const int vrow = 4 * gq + (li >> 2);
#pragma unroll
    for (int dt = 0; dt < C::kDT; ++dt)
      voff[dt] = C::kKBytes + vrow * C::kRowBytes + (((dt * 2 + ((li & 3) >> 1)) ^ C::swz_v(vrow)) * 16) +
                 (li & 1) * 8;
  }

  // One chunk of this wave's work in two phases: A forms the S^T tiles
  // (`masked`, a compile-time tag, selects the copy with the causal mask,
  // used only where some key of the chunk lies past some row of the wave),
  // B does the online softmax and O^T += V^T P^T.
  // S^T tiles: keys kt*16 + (4*gq + r), query li
  floatx4 sv[QT][4];
  auto phase_a = [&](const char* st, int k0, auto masked) __attribute__((always_inline)) {
#pragma unroll
      for (int kt = 0; kt < 4; ++kt) {
#pragma unroll
        for (int ks = 0; ks < C::kKS; ++ks) {
          bf16x8 ka;
          __builtin_memcpy(&ka, st + koff[ks] + kt * 16 * C::kRowBytes, 16);
#pragma unroll
          for (int qt = 0; qt < QT; ++qt) {
            bf16x8 qb;
            __builtin_memcpy(&qb, &qop[qt][ks], 16);
            sv[qt][kt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                ka, qb, ks == 0 ? floatx4{0.f, 0.f, 0.f, 0.f} : sv[qt][kt], 0, 0, 0);
          }
        }
      }
      // causal mask, only in chunks where some key lies past some row of this wave
      if constexpr (decltype(masked)::value) {
#pragma unroll
        for (int qt = 0; qt < QT; ++qt)
#pragma unroll
          for (int kt = 0; kt < 4; ++kt)
#pragma unroll
            for (int r = 0; r < 4; ++r)
              if (k0 + kt * 16 + 4 * gq + r > qpos[qt]) sv[qt][kt][r] = kNegInf;
      }
  };
  auto phase_b = [&](const char* st) __attribute__((always_inline)) {
      // online softmax per query (lane's query li of each tile), in log2 units
      bf16x8 pb[QT][2];
#pragma unroll
      for (int qt = 0; qt < QT; ++qt) {
        float cmax = kNegInf;
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
#pragma unroll
          for (int r = 0; r < 4; ++r) cmax = fmaxf(cmax, sv[qt][kt][r]);
        cmax = wave_max4(cmax) * a.c;
        // the reference m is raised only when some row's maximum passes it
        // by more than kHeadroom; otherwise weights up to 2^kHeadroom are
        // accumulated as they are (the decision is per wave)
        if (__ballot(cmax > m[qt] + kHeadroom) != 0ull) {
          const float mn = fmaxf(m[qt], cmax);
          const float alpha = __builtin_amdgcn_exp2f(m[qt] - mn);
          m[qt] = mn;
          l[qt] *= alpha;
#pragma unroll
          for (int dt = 0; dt < C::kDT; ++dt) o[qt][dt] *= alpha;
        }
        const float mr = m[qt];
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            pb[qt][kt >> 1][(kt & 1) * 4 + r] = (__bf16)__builtin_amdgcn_exp2f(fmaf(sv[qt][kt][r], a.c, -mr));
      }
      // O^T += V^T P^T over two 32-key halves; lane (gq, li) reads, through
      // the transposed load, keys 32j + 4gq + (li >> 2) (+16) at head-dim
      // columns dt*16 + 4*(li & 3) .. +3 and receives four keys at column
      // dt*16 + li
#pragma unroll
      for (int j = 0; j < 2; ++j) {
#pragma unroll
        for (int dt = 0; dt < C::kDT; ++dt) {
          const v4i16 lo = read_tr(st + voff[dt] + (32 * j) * C::kRowBytes);
          const v4i16 hi = read_tr(st + voff[dt] + (32 * j + 16) * C::kRowBytes);
          bf16x8 va;
          __builtin_memcpy(&va, &lo, 8);
          __builtin_memcpy((char*)&va + 8, &hi, 8);
#pragma unroll
          for (int qt = 0; qt < QT; ++qt)
            o[qt][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, pb[qt][j], o[qt][dt], 0, 0, 0);
        }
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) l[qt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, pb[qt][j], l[qt], 0, 0, 0);
      }
  };

  // Every wave passes the same barriers chunk by chunk; a wave works on the
  // chunks up to its last row's position, with the causal mask from the
  // first chunk in which some key lies past its first row.  Two loops over
  // the same step keep the unmasked code free of the mask.  (Staggering the
  // two waves of each SIMD half a chunk apart, as the scoring kernel does,
  // was measured slower here, also with K and V in rings of their own that
  // keep three chunks of lookahead.)
  auto step = [&](int ch, auto masked) __attribute__((always_inline)) {
    // chunks ch+1 .. ch+kLookahead-1 were issued after chunk ch
    wait_chunk<C::kPerChunk>(min(kLookahead - 1, n_chunks - 1 - ch));
    lds_barrier();
    // the stage of chunk ch-1 is free: every wave has passed this barrier
    if (ch + kLookahead < n_chunks) issue(ch + kLookahead);
    const int k0 = ch * kKeys;
    if (k0 <= wave_last_pos) {
      const char* st = smem + (ch % kStages) * C::kStage;
      phase_a(st, k0, masked);
      phase_b(st);
    }
  };
  // first chunk whose last key passes this wave's first row position
  const int first_masked = min(n_chunks, wave_first_pos >= kKeys - 1 ? (wave_first_pos - (kKeys - 1)) / kKeys + 1 : 0);
  int ch = 0;
  for (; ch < first_masked; ++ch) step(ch, std::false_type{});
  for (; ch < n_chunks; ++ch) step(ch, std::true_type{});

  // ---- normalise and store: lane holds O^T[dt*16 + 4*gq + r][query li] ----
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    const float inv = 1.f / l[qt][0];
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
  a.bs_shift = (g.bs & (g.bs - 1)) == 0 ? __builtin_ctz((unsigned)g.bs) : -1;
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
