// Window scoring, Eq. (4) of Kara: A = colsum(softmax(Q_W K_{W\U}^T / sqrt(d)))
// per (sequence, layer, KV head), all G query heads of the group acting as
// queries of their KV head.
//
// Two kernels.  score1_kernel (bf16, d = 128, 512 < N <= 2048, the shapes
// of the Qwen3-shaped workloads) forms and exponentiates every logit once,
// holding each row block's weights in fp16 until the block's row sums are
// known; it is described where it is defined.  score_kernel serves every
// other shape with two sweeps over the keys:
//
// A workgroup of 8 waves owns 128*RT
// query rows of one unit (16*RT rows per wave, held as MFMA operands in
// registers for the whole kernel) and streams the unit's N keys through an
// LDS ring, 64 keys per chunk, twice:
//   sweep A  logits -> per-row maximum and exponential sum (log-sum-exp),
//   sweep B  logits again -> normalised probabilities -> column sums.
// Every wave sees every key of its own rows, so the row statistics need no
// exchange between waves.  Recomputing the logits doubles the matrix work
// but keeps nothing per logit between the sweeps, so the rows sharing one
// read of the keys (512 for bf16) are limited by the operand registers only.
// Keys reach LDS by direct global->LDS
// copies, so no register is spent on staging and the copies of later chunks
// overlap the matrix and exponential work of the current one.
//
// Column sums of a chunk are reduced within each wave in a fixed lane order,
// then across the 8 waves in wave order into a per-workgroup row in LDS.
// Each workgroup (of either kernel) writes one partial sum per row split and
// a second kernel adds them in split order.  (Handing the sum to the last
// split to finish would need a device-scope release/acquire, which on this
// multi-XCD part writes back and invalidates the whole L2 of the XCD every
// time.)  No floating-point atomics, so the scores are bit-reproducible.
#include <type_traits>

#include "kara_internal.h"

namespace kara {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int kScoreThreads = 512;
constexpr int kScoreWaves = kScoreThreads / 64;
constexpr int kLdsLimit = 160 * 1024;
constexpr int kTps = 4;                   // 16-key tiles per chunk
constexpr int kChunkKeys = kTps * 16;     // keys per chunk
constexpr int kMaxChunks = (KARA_MAX_COMPRESSIBLE + kChunkKeys - 1) / kChunkKeys;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kNegInf = -__builtin_huge_valf();
constexpr float kPosInf = __builtin_huge_valf();
// Lower end of a running row maximum (log2 units): finite, so that
// exp2(m_old - m_new) never sees inf - inf.
constexpr float kMaxFloor = -1e30f;
// Sweep A accumulates exp2(x - m) against a maximum m that is only raised
// when a row sum would pass this bound, so no term or sum can overflow.
constexpr float kSumBound = 18446744073709551616.f;   // 2^64

struct ScoreArgs {
  Geom g;
  const char* q;              // [n_layers][n_trig][W][Hq][d]
  PoolPtrs k;                 // per-layer K pools
  const int32_t* trig;
  const int32_t* bt;
  const int32_t* win_start;
  const int32_t* status;
  float* partials;            // [units][n_splits][N] (unused with one split)
  float* scores;              // [units][N]
  int n_splits;
  int64_t n_blocks;
};

// Static geometry of one kernel instance: element type DT, head dim D, RT
// 16-row tiles per wave.
template <int DT, int D, int RT>
struct Cfg {
  static constexpr int kES = DT == KARA_BF16 ? 2 : 4;
  static constexpr int kRowBytes = D * kES;              // one key or query row
  static constexpr int kCPR = kRowBytes / 16;            // 16-byte chunks per row
  static constexpr int kSwz = kCPR < 16 ? kCPR - 1 : 15; // XOR swizzle mask
  // XOR swizzle of a key row's 16-byte chunks, a function of the row, with
  // the row's two low bits moved to the top: measured on gfx950, a 16-byte
  // read of 16 rows x 4 lane groups then has no bank conflicts, where XOR by
  // the row itself costs about four conflict cycles per read (256-byte rows:
  // bf16 d = 128, fp32 d = 64; 128-byte rows: bf16 d = 64).
  static __device__ __forceinline__ int swz(int row) {
    if constexpr (kCPR == 16) return ((row & 3) << 2) | ((row >> 2) & 3);
    if constexpr (kCPR == 8) return ((row & 3) << 1) | ((row >> 2) & 1);
    return row & kSwz;
  }
  static constexpr int kRowsWG = kScoreWaves * 16 * RT;  // query rows per workgroup
  static constexpr int kStageBytes = kChunkKeys * kRowBytes;
  static constexpr int kL = kStageBytes / (kScoreThreads * 16);   // copies per thread per chunk
  // key offsets and workgroup column sums, plus up to five chunks' per-wave column sums
  static constexpr int kFixedBytes = 2 * kMaxChunks * kChunkKeys * 4 + 5 * kScoreWaves * kChunkKeys * 4;
  static constexpr int fit_stages() {
    int s = 6;
    while (s > 2 && s * kStageBytes + kFixedBytes > kLdsLimit) --s;
    return s;
  }
  static constexpr int kStages = fit_stages();
  static_assert(kL >= 1 && kL * kScoreThreads * 16 == kStageBytes, "chunk copies must be uniform over threads");
  static_assert(kStages * kStageBytes + kFixedBytes <= kLdsLimit, "LDS budget");
};

// A lane's operand: lane group gq = lane/16 supplies head-dim elements
// [gq*d/4, (gq+1)*d/4) of its row -- 16-byte chunks gq*kChunks.. -- one
// k-step per chunk (bf16: 8 elements) or per element (fp32).  Keys and
// queries use the same assignment, so every product q_c k_c enters the dot
// product exactly once.
template <int DT, int D>
struct Operand {
  static constexpr int kChunks = (D * (DT == KARA_BF16 ? 2 : 4) / 16) / 4;
  uint4 v[kChunks];
};

template <int DT, int D>
__device__ inline floatx4 dot_tile(const Operand<DT, D>& qa, const Operand<DT, D>& kb, floatx4 acc) {
  if constexpr (DT == KARA_BF16) {
#pragma unroll
    for (int s = 0; s < Operand<DT, D>::kChunks; ++s) {
      bf16x8 a, b;
      __builtin_memcpy(&a, &qa.v[s], 16);
      __builtin_memcpy(&b, &kb.v[s], 16);
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc, 0, 0, 0);
    }
  } else {
    const float* a = (const float*)qa.v;
    const float* b = (const float*)kb.v;
#pragma unroll
    for (int s = 0; s < Operand<DT, D>::kChunks * 4; ++s)
      acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[s], b[s], acc, 0, 0, 0);
  }
  return acc;
}

// reductions over the 16 lanes of a lane group (the 16 keys of a tile)
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

// Direct global->LDS copy of 16 bytes per lane; lane i's bytes land at
// lds_wave_base + 16*i (global_load_lds_dwordx4 with the LDS base in M0).
// Issued through inline assembly: the compiler then inserts no wait of its
// own before LDS reads (it cannot tell the ring stages apart and would drain
// every copy); the kernel waits explicitly with wait_chunks().  M0 is
// restored.
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

// Workgroup barrier for LDS traffic only.  __syncthreads() would also drain
// every outstanding global->LDS copy (its release fence waits on vmcnt),
// defeating the prefetch ring; the copies this barrier must cover are waited
// for explicitly first.
__device__ inline void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

template <int N>
__device__ inline void wait_vm() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Wait until at most kL*newer of this thread's memory operations are
// outstanding, newer <= P-1 (a run-time count, compile-time wait fields).
template <int kL, int P>
__device__ inline void wait_chunks(int newer) {
  if constexpr (P >= 6) { if (newer >= 5) { wait_vm<5 * kL>(); return; } }
  if constexpr (P >= 5) { if (newer >= 4) { wait_vm<4 * kL>(); return; } }
  if constexpr (P >= 4) { if (newer >= 3) { wait_vm<3 * kL>(); return; } }
  if constexpr (P >= 3) { if (newer >= 2) { wait_vm<2 * kL>(); return; } }
  if constexpr (P >= 2) { if (newer >= 1) { wait_vm<kL>(); return; } }
  wait_vm<0>();
}

template <int DT, int D, int RT>
__global__ __launch_bounds__(kScoreThreads) void score_kernel(ScoreArgs a) {
  using C = Cfg<DT, D, RT>;
  using Op = Operand<DT, D>;
  constexpr int CPR = C::kCPR;
  constexpr int S = C::kStages;
  // The ring is synchronised once per group of GS chunks (two when there
  // are stages enough): one barrier then covers two chunks of work.  Chunks
  // are copied P ahead of the group being worked on.
  constexpr int GS = S >= 5 ? 2 : 1;
  constexpr int P = S - GS;
  // a chunk's per-wave column sums are added at the first group start after
  // both halves wrote them, at most 1 + 2*GS chunks later
  constexpr int kColSlots = 1 + 2 * GS;
  constexpr int kL = C::kL;
  constexpr int KC = Op::kChunks;
  static_assert(P <= 6, "wait_chunks covers at most six chunks in flight");

  __shared__ __attribute__((aligned(16))) char kbuf[S * C::kStageBytes];
  // byte offset / 16 of every compressible key row in the K pool (the block
  // table resolved once per workgroup); padding entries repeat key 0
  __shared__ uint32_t key_off[kMaxChunks * kChunkKeys];
  // this workgroup's column sums; per-wave column sums of the last kColSlots chunks
  __shared__ float col_wg[kMaxChunks * kChunkKeys];
  __shared__ float col_wave[kColSlots][kScoreWaves][kChunkKeys];

  const Geom& g = a.g;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform, kept in an SGPR
  const int gq = lane >> 4;     // lane group: rows 4*gq..4*gq+3 of a 16-row tile
  const int li = lane & 15;     // key of a 16-key tile / row of the query operand

  // Blocks are dealt round-robin to the 8 XCDs; renumber so that the row
  // splits of one unit run together on one XCD and share its L2 copy of the
  // unit's keys.
  int64_t bid = blockIdx.x;
  if ((a.n_blocks & 7) == 0) bid = (bid & 7) * (a.n_blocks >> 3) + (bid >> 3);
  const int64_t u = bid / a.n_splits;
  const int split = (int)(bid % a.n_splits);
  // unit u = ((l * n_trig + t) * n_win + w) * Hkv + h; window w of the
  // trigger starts w*N after win_start
  const int h = (int)(u % g.Hkv);
  const int tw = (int)((u / g.Hkv) % ((int64_t)g.n_trig * g.n_win));
  const int t = tw / g.n_win;
  const int wi = tw - t * g.n_win;
  const int l = (int)(u / ((int64_t)g.Hkv * g.n_trig * g.n_win));
  const int N = g.N;
  const int nch = (N + kChunkKeys - 1) / kChunkKeys;
  float* out = a.n_splits == 1 ? a.scores + u * (int64_t)N : a.partials + (u * a.n_splits + split) * (int64_t)N;

  if (a.status[t] != 0) {
    for (int j = tid; j < N; j += kScoreThreads) out[j] = 0.f;
    return;
  }
  const int s = a.trig[t];
  const int p0 = a.win_start[s] + wi * N;
  const char* kpool = (const char*)a.k.p[l];
  const char* qunit = a.q + (((int64_t)l * g.n_trig + t) * g.n_win + wi) * g.Wq * g.Hq * (int64_t)C::kRowBytes;
  const int R = g.G * g.Wq;
  const float c = g.scale * kLog2e;

  // ---- this wave's query rows, straight into operand registers ----
  // row r = w*G + gi (scoring position w of the Wq in q, query head
  // h*G + gi); rows past R
  // repeat row 0 and are given no weight
  const int row_base = split * C::kRowsWG + wave * 16 * RT;
  Op qa[RT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    int r = row_base + rt * 16 + li;
    if (r >= R) r = 0;
    const int w = r / g.G, gi = r - w * g.G;
    const uint4* src = (const uint4*)(qunit + ((int64_t)w * g.Hq + h * g.G + gi) * C::kRowBytes) + gq * KC;
#pragma unroll
    for (int ks = 0; ks < KC; ++ks) qa[rt].v[ks] = src[ks];
  }
  // Consume the query registers here, before any key copy is issued, so the
  // compiler waits for these loads once.  Otherwise it keeps them pending
  // into the chunk loops and waits on them there with counts that cannot
  // see the copies in flight, draining the key ring every chunk.
#pragma unroll
  for (int rt = 0; rt < RT; ++rt)
#pragma unroll
    for (int ks = 0; ks < KC; ++ks) asm volatile("" ::"v"(qa[rt].v[ks].x), "v"(qa[rt].v[ks].y),
                                                 "v"(qa[rt].v[ks].z), "v"(qa[rt].v[ks].w));

  {
    const int32_t* row_pages = a.bt + (int64_t)s * g.max_blocks;
    for (int j = tid; j < nch * kChunkKeys; j += kScoreThreads) {
      const int pos = p0 + (j < N ? j : 0);        // padding keys: any valid row
      const uint64_t row = ((uint64_t)row_pages[pos / g.bs] * g.Hkv + h) * g.bs + pos % g.bs;
      key_off[j] = (uint32_t)(row * (C::kRowBytes / 16));
    }
  }
  // the key offsets must be in LDS before the copies below compute addresses
  lds_barrier();

  // ---- key copies: every thread issues exactly kL per chunk ----
  // Copy r of this thread fills stage slot r*512 + tid: key row kr = slot /
  // CPR of the chunk, 16-byte chunk (slot % CPR) ^ swz(kr).  The key
  // offsets of a chunk are read from the table one iteration before its
  // copies are issued, so issuing them never waits on LDS.
  const char* kpool_c[kL];
  int kr0[kL];
#pragma unroll
  for (int r = 0; r < kL; ++r) {
    const int slot = r * kScoreThreads + tid;
    const int kr = slot / CPR;
    const int chunk = (slot % CPR) ^ C::swz(kr);
    kpool_c[r] = kpool + chunk * 16;
    kr0[r] = kr;
  }
  const int n_it = 2 * nch;                // sweep A, then sweep B, over the same chunks
  uint32_t coff[GS][kL];   // key offsets of the next group's copies
  auto read_offsets = [&](int it, int x) __attribute__((always_inline)) {
    const int ch = it < nch ? it : it - nch;
#pragma unroll
    for (int r = 0; r < kL; ++r) coff[x][r] = key_off[ch * kChunkKeys + kr0[r]];
  };
  auto issue_copies = [&](int it, int x) __attribute__((always_inline)) {
    char* sbase = kbuf + (it % S) * C::kStageBytes;
#pragma unroll
    for (int r = 0; r < kL; ++r)
      copy16(kpool_c[r] + (uint64_t)coff[x][r] * 16, sbase + (r * kScoreWaves + wave) * 1024);
  };

  // per-lane LDS byte offsets of the key operand chunks (key rows are
  // multiples of 16 plus li, so the swizzle term depends on the lane only)
  int koff[KC];
#pragma unroll
  for (int ks = 0; ks < KC; ++ks) koff[ks] = li * C::kRowBytes + (((gq * KC + ks) ^ C::swz(li)) * 16);

  // logits of this wave's rows x the chunk's 64 keys:
  // acc[rt][ti][q] = row rt*16 + 4*gq + q, key ti*16 + li
  floatx4 acc[RT][kTps];
  auto b_read = [&](const char* sb, int ti, Op& kb) __attribute__((always_inline)) {
#pragma unroll
    for (int ks = 0; ks < KC; ++ks) kb.v[ks] = *(const uint4*)(sb + koff[ks] + ti * 16 * C::kRowBytes);
  };
  auto mfma_tile = [&](const Op& kb, int ti) __attribute__((always_inline)) {
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) acc[rt][ti] = dot_tile<DT, D>(qa[rt], kb, floatx4{0.f, 0.f, 0.f, 0.f});
  };

  // Logits of chunk `it` (its keys are in stage it % S): acc holds this
  // wave's rows x the chunk's 64 keys; keys past N become -inf.
  auto form = [&](int it) __attribute__((always_inline)) {
    const char* sb = kbuf + (it % S) * C::kStageBytes;
    const int ch = it < nch ? it : it - nch;
    // key operands double-buffered: the next tile's LDS reads are in flight
    // while the matrix cores work on this one
    Op kb[2];
    b_read(sb, 0, kb[0]);
#pragma unroll
    for (int ti = 0; ti < kTps; ++ti) {
      if (ti + 1 < kTps) b_read(sb, ti + 1, kb[(ti + 1) & 1]);
      mfma_tile(kb[ti & 1], ti);
      __builtin_amdgcn_sched_barrier(0);
    }
    if ((ch + 1) * kChunkKeys > N) {
#pragma unroll
      for (int ti = 0; ti < kTps; ++ti)
        if (ch * kChunkKeys + ti * 16 + li >= N) {
#pragma unroll
          for (int rt = 0; rt < RT; ++rt) acc[rt][ti] = floatx4{kNegInf, kNegInf, kNegInf, kNegInf};
        }
    }
  };

  // ---- sweep A: per-row reference m and sum l of exp2(x - m), x = logit*c,
  // over this lane's keys.  The first chunk sets m to the lane's maximum so
  // far (an exact running-maximum update); later chunks only add terms, which
  // may then exceed 1.  fp32 holds such sums exactly enough unless a logit
  // lies about 128 log2-units above m, which makes the sum infinite: a wave
  // that sees that redoes the sweep on its own with the running maximum.
  float m[RT][4], lsum[RT][4];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      m[rt][q] = kMaxFloor;
      lsum[rt][q] = 0.f;
    }
  // running-maximum update by one 16-key tile (keys past N are -inf)
  auto valu_exact = [&](int ti) __attribute__((always_inline)) {
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float x = acc[rt][ti][q] * c;
        const float mn = fmaxf(m[rt][q], x);
        lsum[rt][q] = fmaf(lsum[rt][q], __builtin_amdgcn_exp2f(m[rt][q] - mn), __builtin_amdgcn_exp2f(x - mn));
        m[rt][q] = mn;
      }
  };
  auto valu_a = [&](int ti) __attribute__((always_inline)) {
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int q = 0; q < 4; ++q) lsum[rt][q] += __builtin_amdgcn_exp2f(fmaf(acc[rt][ti][q], c, -m[rt][q]));
  };
  // after sweep A, m[][] holds each row's log-sum-exp (log2 units)
  auto finish_sweep_a = [&]() __attribute__((always_inline)) {
    bool bad = false;
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int q = 0; q < 4; ++q) bad |= !(lsum[rt][q] <= 3.4e38f);
    if (__builtin_amdgcn_ballot_w64(bad) != 0) {
      // redo this wave's rows, reading the key operands from global memory
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          m[rt][q] = kMaxFloor;
          lsum[rt][q] = 0.f;
        }
      for (int j0 = 0; j0 < N; j0 += 16) {
        const int j = j0 + li;
        const uint4* src = (const uint4*)(kpool + (uint64_t)key_off[j < N ? j : 0] * 16) + gq * KC;
        Op kb;
#pragma unroll
        for (int ks = 0; ks < KC; ++ks) kb.v[ks] = src[ks];
        mfma_tile(kb, 0);
        if (j >= N) {
#pragma unroll
          for (int rt = 0; rt < RT; ++rt) acc[rt][0] = floatx4{kNegInf, kNegInf, kNegInf, kNegInf};
        }
        valu_exact(0);
      }
    }
    // combine the 16 lanes of each row: lse = M + log2(sum_lanes l*2^(m-M));
    // rows past R get lse = +inf and so zero probabilities
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float M = max16(m[rt][q]);
        const float L = sum16(lsum[rt][q] * __builtin_amdgcn_exp2f(m[rt][q] - M));
        const bool live = row_base + rt * 16 + gq * 4 + q < R;
        m[rt][q] = live ? M + __builtin_amdgcn_logf(L) : kPosInf;
      }
  };

  // ---- sweep B: probabilities exp2(x - lse); per chunk, each wave's column
  // sums go to col_wave[chunk % kColSlots][wave], lane group gq holding tile gq
  auto sweep_b = [&](int ch) __attribute__((always_inline)) {
    float v[kTps];
#pragma unroll
    for (int ti = 0; ti < kTps; ++ti) {
      float sum = 0.f;
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int q = 0; q < 4; ++q) sum += __builtin_amdgcn_exp2f(fmaf(acc[rt][ti][q], c, -m[rt][q]));
      v[ti] = sum;
    }
    // over the four lane groups, leaving lane group gq with tile gq:
    // groups {0,1} keep tiles 0,1 and {2,3} keep tiles 2,3, then pairs split.
    // The exchanges are register swaps between lane halves and between
    // 16-lane rows: after permlane32_swap(a, b), the first result holds a's
    // low half and b's low half, the second a's high half and b's high
    // half, so their sum is tile a's pair sum in lanes 0-31 and tile b's in
    // lanes 32-63; permlane16_swap does the same for even and odd rows.
    static_assert(kTps == 4, "the reduce-scatter covers four key tiles");
    const auto s0 = __builtin_amdgcn_permlane32_swap(__float_as_uint(v[0]), __float_as_uint(v[2]), false, false);
    const auto s1 = __builtin_amdgcn_permlane32_swap(__float_as_uint(v[1]), __float_as_uint(v[3]), false, false);
    const float x0 = __uint_as_float(s0[0]) + __uint_as_float(s0[1]);
    const float x1 = __uint_as_float(s1[0]) + __uint_as_float(s1[1]);
    const auto s2 = __builtin_amdgcn_permlane16_swap(__float_as_uint(x0), __float_as_uint(x1), false, false);
    const float y = __uint_as_float(s2[0]) + __uint_as_float(s2[1]);
    col_wave[ch % kColSlots][wave][gq * 16 + li] = y;
  };
  // the eight waves' sums of one chunk, added in wave order
  auto reduce_chunk = [&](int ch) __attribute__((always_inline)) {
    const float* cw = &col_wave[ch % kColSlots][0][0];
    float sum = cw[lane];
#pragma unroll
    for (int w = 1; w < kScoreWaves; ++w) sum += cw[w * kChunkKeys + lane];
    col_wg[ch * kChunkKeys + lane] = sum;
  };

  // sweep A's vector work on chunk it once its logits are formed
  auto values_a = [&](int it) __attribute__((always_inline)) {
    if (it == 0) {
#pragma unroll
      for (int ti = 0; ti < kTps; ++ti) valu_exact(ti);
    } else {
#pragma unroll
      for (int ti = 0; ti < kTps; ++ti) valu_a(ti);
    }
  };

  // The two halves of the workgroup run the same chunk sequence half a
  // chunk apart (see below); each half is compiled as its own code path.
  auto run = [&](auto lag_tag) __attribute__((always_inline)) {
    constexpr bool kLag = decltype(lag_tag)::value;
    // prologue: the first P chunks, and the offsets of the next group's
    for (int j = 0; j < P && j < n_it; ++j) {
      read_offsets(j, 0);
      issue_copies(j, 0);
    }
#pragma unroll
    for (int x = 0; x < GS; ++x)
      if (P + x < n_it) read_offsets(P + x, x);

    // Iteration it: wait for chunk it and make every wave's copies of it
    // visible (the stage of chunk it-1 is then free and receives chunk it+P).
    // Waves 0-3 form chunk it's logits and then do its vector work; waves 4-7,
    // one per SIMD, first do the vector work of chunk it-1 and then form chunk
    // it, so on every SIMD one wave keeps the matrix cores busy while the other
    // computes exponentials.
    // At the start of each group (it a multiple of GS; n_it is even): wait
    // for the group's chunks and make every wave's copies of them visible;
    // the previous group's stages are then free and receive chunks it+P...
    auto sync = [&](int it) __attribute__((always_inline)) {
      if (it % GS != 0) return;
      wait_chunks<kL, P>(min(P - GS, n_it - GS - it));
      lds_barrier();
#pragma unroll
      for (int x = 0; x < GS; ++x)
        if (it + P + x < n_it) issue_copies(it + P + x, x);
#pragma unroll
      for (int x = 0; x < GS; ++x)
        if (it + GS + P + x < n_it) read_offsets(it + GS + P + x, x);
    };
    // (the scheduling fences keep one chunk's logits live at a time)
    for (int it = 0; it < nch; ++it) {
      sync(it);
      if constexpr (!kLag) {
        form(it);
        __builtin_amdgcn_sched_barrier(0);
        values_a(it);
      } else {
        if (it > 0) values_a(it - 1);
        __builtin_amdgcn_sched_barrier(0);
        form(it);
      }
    }
    if constexpr (!kLag) finish_sweep_a();
    // first chunk of sweep B: the lagging waves finish sweep A first
    sync(nch);
    if constexpr (!kLag) {
      form(nch);
      __builtin_amdgcn_sched_barrier(0);
      sweep_b(0);
    } else {
      values_a(nch - 1);
      finish_sweep_a();
      __builtin_amdgcn_sched_barrier(0);
      form(nch);
    }
    for (int it = nch + 1; it < n_it; ++it) {
      sync(it);
      // at a group start: chunks whose column sums both halves completed
      // before this group's barrier (chunk ch: at iterations nch+ch, nch+ch+1)
      if (it % GS == 0) {
#pragma unroll
        for (int x = 0; x < GS; ++x) {
          const int ch = it - nch - 1 - GS + x;
          if (ch >= 0 && wave == ch % kScoreWaves) reduce_chunk(ch);
        }
      }
      if constexpr (!kLag) {
        form(it);
        __builtin_amdgcn_sched_barrier(0);
        sweep_b(it - nch);
      } else {
        sweep_b(it - 1 - nch);
        __builtin_amdgcn_sched_barrier(0);
        form(it);
      }
    }
    if constexpr (kLag) sweep_b(nch - 1);
  };
  if (wave >= kScoreWaves / 2) run(std::true_type{});
  else run(std::false_type{});
  lds_barrier();
  for (int ch = nch - GS - 1 > 0 ? nch - GS - 1 : 0; ch < nch; ++ch)
    if (wave == ch % kScoreWaves) reduce_chunk(ch);
  lds_barrier();
  for (int j = tid; j < N; j += kScoreThreads) out[j] = col_wg[j];
}

// Scores of a unit: its row splits' partial column sums added in split order
// (a kernel boundary orders them after every split's writes).
__global__ __launch_bounds__(256) void split_sum_kernel(const float* __restrict__ partials,
                                                        float* __restrict__ scores, int N, int n_splits) {
  const int64_t u = blockIdx.x;
  const int j = blockIdx.y * 256 + threadIdx.x;
  if (j >= N) return;
  const float* src = partials + u * n_splits * (int64_t)N + j;
  float v = src[0];
  for (int p = 1; p < n_splits; ++p) v += src[(int64_t)p * N];
  scores[u * (int64_t)N + j] = v;
}

// ---------------------------------------------------------------------------
// Single-sweep scoring (bf16, d = 128, up to 2048 compressible keys).
//
// Every logit is formed and exponentiated once.  A workgroup of 4 waves, one
// per SIMD, takes a unit's query rows 64 at a time (a row block); within a
// block wave w owns the keys of tiles [w*ntw, (w+1)*ntw) (16 keys a tile)
// against all 64 rows, so its tiles' weights e = 2^(x - m) fit in its
// accumulation registers as fp16 (64 rows x 512 keys = 256 registers).  The
// reference m of a row is shared by the four waves: the maximum of their
// first tiles' logits less kS1Headroom, exchanged once per block through
// LDS.  When the row sums are known, the weights 1/L (one per row, the same
// for every wave since m is shared) are applied by fp16 MFMAs of the stored
// values, 32 rows at a time, which sums each key's column; the row sums
// themselves accumulate on the matrix cores too, each tile pair's stored
// values times a constant 0/1 selector.  The keys of a
// wave stream through its own LDS ring by direct global->LDS copies, the
// same keys for every block of the unit, so the ring runs on across blocks
// and no workgroup barrier guards it; the next block's queries are copied
// into LDS during the current block.
//
// Precision.  e is rounded once to fp16 (relative error 2^-11, or 2^-25
// absolute below fp16's normal range); the row weight is carried as an
// fp16 pair (hi + lo) scaled by 2^21, so it loses nothing that matters; all
// sums are fp32.  With m = (first-tile maximum) - 6 the top first-tile term
// is 64, so a term of fp16's subnormal range contributes at most 2^-31 to a
// probability.  A row whose later logits rise more than about 10 log2 units
// above its first tiles' maximum would overflow fp16: any wave's row sum
// reaching 65504 (which every overflowing term would exceed) or NaN (where
// the selector's zeros met an infinity) sends the block
// through once more with m = (exact row maximum) - 6, where no term exceeds
// 64 and no wave sum 64 * 512.
// ---------------------------------------------------------------------------
constexpr int kS1QIt = 2;                  // iteration that copies the next block's queries
constexpr int kS1BlocksPerSplit = 16;      // row blocks per workgroup (consecutive blocks of one unit)
constexpr int kS1RowBytes = 256;           // one bf16 row of 128
constexpr int kS1TileBytes = 16 * kS1RowBytes;
constexpr float kS1Headroom = 6.f;
constexpr float kF16Max = 65504.f;
constexpr float kS1WScale = 2097152.f;     // 2^21: row weights 1/L, L in [64, 2^18], as fp16

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef float float2v __attribute__((ext_vector_type(2)));

struct Score1Args {
  ScoreArgs s;
  int ntw;          // key tiles per wave
};

// the 16-byte chunk swizzle of a 256-byte row in LDS (conflict-free for the
// operand reads: row's two low bits moved to the top)
__device__ __forceinline__ int s1_swz(int row) { return ((row & 3) << 2) | ((row >> 2) & 3); }

// Reductions over the 16 lanes of a row by DPP butterflies (quad swaps,
// then half-row and row mirrors).  Every lane ends with the same value:
// each step combines two equal partial results, in either order.
template <class Op>
__device__ __forceinline__ float dpp_reduce16(float v, Op op) {
  v = op(v, __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0xB1, 0xF, 0xF, false)));
  v = op(v, __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x4E, 0xF, 0xF, false)));
  v = op(v, __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x141, 0xF, 0xF, false)));
  v = op(v, __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x140, 0xF, 0xF, false)));
  return v;
}
__device__ __forceinline__ float dpp_max16(float v) {
  return dpp_reduce16(v, [](float x, float y) { return fmaxf(x, y); });
}
__device__ __forceinline__ float dpp_sum16(float v) {
  return dpp_reduce16(v, [](float x, float y) { return x + y; });
}

// The same butterflies for 8 or 16 values at once, one DPP step over all of
// them before the next (so no step reads a value written fewer than 8
// instructions before; the leading s_nop covers the values' last writes
// before the block).  Written as instructions because the compiler keeps a
// separate DPP move per step, and in IEEE mode adds a quieting max before
// every fmaxf.
#define S1_DPP8(OP, PAT)                                                                               \
  asm volatile("s_nop 1\n\t"                                                                           \
               OP " %0, %0, %0 " PAT "\n\t" OP " %1, %1, %1 " PAT "\n\t" OP " %2, %2, %2 " PAT "\n\t"  \
               OP " %3, %3, %3 " PAT "\n\t" OP " %4, %4, %4 " PAT "\n\t" OP " %5, %5, %5 " PAT "\n\t"  \
               OP " %6, %6, %6 " PAT "\n\t" OP " %7, %7, %7 " PAT                                        \
               : "+v"(v[0]), "+v"(v[1]), "+v"(v[2]), "+v"(v[3]), "+v"(v[4]), "+v"(v[5]), "+v"(v[6]),     \
                 "+v"(v[7]))
#define S1_DPP16(OP, PAT)                                                                              \
  asm volatile("s_nop 1\n\t"                                                                           \
               OP " %0, %0, %0 " PAT "\n\t" OP " %1, %1, %1 " PAT "\n\t" OP " %2, %2, %2 " PAT "\n\t"  \
               OP " %3, %3, %3 " PAT "\n\t" OP " %4, %4, %4 " PAT "\n\t" OP " %5, %5, %5 " PAT "\n\t"  \
               OP " %6, %6, %6 " PAT "\n\t" OP " %7, %7, %7 " PAT "\n\t" OP " %8, %8, %8 " PAT "\n\t"  \
               OP " %9, %9, %9 " PAT "\n\t" OP " %10, %10, %10 " PAT "\n\t" OP " %11, %11, %11 " PAT   \
               "\n\t" OP " %12, %12, %12 " PAT "\n\t" OP " %13, %13, %13 " PAT "\n\t" OP " %14, %14, %14 " \
               PAT "\n\t" OP " %15, %15, %15 " PAT                                                      \
               : "+v"(v[0]), "+v"(v[1]), "+v"(v[2]), "+v"(v[3]), "+v"(v[4]), "+v"(v[5]), "+v"(v[6]),     \
                 "+v"(v[7]), "+v"(v[8]), "+v"(v[9]), "+v"(v[10]), "+v"(v[11]), "+v"(v[12]), "+v"(v[13]), \
                 "+v"(v[14]), "+v"(v[15]))
#define S1_DPP_ALL(M)                                                      \
  if constexpr (MAX) {                                                     \
    M("v_max_f32_dpp", "quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf");  \
    M("v_max_f32_dpp", "quad_perm:[2,3,0,1] row_mask:0xf bank_mask:0xf");  \
    M("v_max_f32_dpp", "row_half_mirror row_mask:0xf bank_mask:0xf");      \
    M("v_max_f32_dpp", "row_mirror row_mask:0xf bank_mask:0xf");           \
  } else {                                                                 \
    M("v_add_f32_dpp", "quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf");  \
    M("v_add_f32_dpp", "quad_perm:[2,3,0,1] row_mask:0xf bank_mask:0xf");  \
    M("v_add_f32_dpp", "row_half_mirror row_mask:0xf bank_mask:0xf");      \
    M("v_add_f32_dpp", "row_mirror row_mask:0xf bank_mask:0xf");           \
  }
template <bool MAX, int N>
__device__ __forceinline__ void dpp_reduce16xn(float (&v)[N]) {
  static_assert(N == 8 || N == 16, "8 or 16 values");
  if constexpr (N == 16) {
    S1_DPP_ALL(S1_DPP16)
  } else {
    S1_DPP_ALL(S1_DPP8)
  }
}
#undef S1_DPP_ALL
#undef S1_DPP16
#undef S1_DPP8
// Reduce-scatter over the 16 lanes of a row: every lane's v[i] combined,
// lane li ending with index li's result.  Four butterfly steps, each
// keeping half of the values: lanes li and li ^ 8 (a rotation by 8), then
// li and 7 - li within each half (the half mirror), then the quad swaps
// li ^ 2 and li ^ 1.  A lane keeps the half its bit names and sends the
// other, so each step combines only the values that stay: 45 instructions
// against 64 for every lane's full result.
// (each step is one asm statement that starts with the wait states a DPP
// read needs after the VALU writes of its sources, which all precede it)
template <bool MAX, int K, int PATTERN>
__device__ __forceinline__ void s1_rs_step(float (&keep)[8], const float (&send)[8]) {
  // PATTERN: 0 row_ror:8, 1 row_half_mirror, 2 quad_perm:[2,3,0,1], 3 quad_perm:[1,0,3,2]
#define S1_OPS(OP, PAT)                                                                                     \
  if constexpr (K == 8)                                                                                     \
    asm volatile("s_nop 1\n\t"                                                                              \
                 OP " %0, %8, %0 " PAT "\n\t" OP " %1, %9, %1 " PAT "\n\t" OP " %2, %10, %2 " PAT "\n\t"    \
                 OP " %3, %11, %3 " PAT "\n\t" OP " %4, %12, %4 " PAT "\n\t" OP " %5, %13, %5 " PAT "\n\t"  \
                 OP " %6, %14, %6 " PAT "\n\t" OP " %7, %15, %7 " PAT                                     \
                 : "+v"(keep[0]), "+v"(keep[1]), "+v"(keep[2]), "+v"(keep[3]), "+v"(keep[4]), "+v"(keep[5]), \
                   "+v"(keep[6]), "+v"(keep[7])                                                             \
                 : "v"(send[0]), "v"(send[1]), "v"(send[2]), "v"(send[3]), "v"(send[4]), "v"(send[5]),     \
                   "v"(send[6]), "v"(send[7]));                                                             \
  else if constexpr (K == 4)                                                                                \
    asm volatile("s_nop 1\n\t"                                                                              \
                 OP " %0, %4, %0 " PAT "\n\t" OP " %1, %5, %1 " PAT "\n\t" OP " %2, %6, %2 " PAT "\n\t"     \
                 OP " %3, %7, %3 " PAT                                                                      \
                 : "+v"(keep[0]), "+v"(keep[1]), "+v"(keep[2]), "+v"(keep[3])                               \
                 : "v"(send[0]), "v"(send[1]), "v"(send[2]), "v"(send[3]));                                 \
  else if constexpr (K == 2)                                                                                \
    asm volatile("s_nop 1\n\t" OP " %0, %2, %0 " PAT "\n\t" OP " %1, %3, %1 " PAT                           \
                 : "+v"(keep[0]), "+v"(keep[1])                                                             \
                 : "v"(send[0]), "v"(send[1]));                                                             \
  else                                                                                                      \
    asm volatile("s_nop 1\n\t" OP " %0, %1, %0 " PAT : "+v"(keep[0]) : "v"(send[0]))
  if constexpr (MAX) {
    if constexpr (PATTERN == 0) S1_OPS("v_max_f32_dpp", "row_ror:8 row_mask:0xf bank_mask:0xf");
    else if constexpr (PATTERN == 1) S1_OPS("v_max_f32_dpp", "row_half_mirror row_mask:0xf bank_mask:0xf");
    else if constexpr (PATTERN == 2) S1_OPS("v_max_f32_dpp", "quad_perm:[2,3,0,1] row_mask:0xf bank_mask:0xf");
    else S1_OPS("v_max_f32_dpp", "quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf");
  } else {
    if constexpr (PATTERN == 0) S1_OPS("v_add_f32_dpp", "row_ror:8 row_mask:0xf bank_mask:0xf");
    else if constexpr (PATTERN == 1) S1_OPS("v_add_f32_dpp", "row_half_mirror row_mask:0xf bank_mask:0xf");
    else if constexpr (PATTERN == 2) S1_OPS("v_add_f32_dpp", "quad_perm:[2,3,0,1] row_mask:0xf bank_mask:0xf");
    else S1_OPS("v_add_f32_dpp", "quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf");
  }
#undef S1_OPS
}
template <bool MAX>
__device__ __forceinline__ float reduce_scatter16(const float (&v)[16], int li) {
  float keep[8], send[8];
  const bool h3 = (li & 8) != 0, h2 = (li & 4) != 0, h1 = (li & 2) != 0, h0 = (li & 1) != 0;
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    keep[k] = h3 ? v[8 + k] : v[k];
    send[k] = h3 ? v[k] : v[8 + k];
  }
  s1_rs_step<MAX, 8, 0>(keep, send);
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const float a = keep[k], b = keep[4 + k];
    keep[k] = h2 ? b : a;
    send[k] = h2 ? a : b;
  }
  s1_rs_step<MAX, 4, 1>(keep, send);
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const float a = keep[k], b = keep[2 + k];
    keep[k] = h1 ? b : a;
    send[k] = h1 ? a : b;
  }
  s1_rs_step<MAX, 2, 2>(keep, send);
  {
    const float a = keep[0], b = keep[1];
    keep[0] = h0 ? b : a;
    send[0] = h0 ? a : b;
  }
  s1_rs_step<MAX, 1, 3>(keep, send);
  return keep[0];
}

// max of three, with no quieting of its operands
__device__ __forceinline__ float s1_max3(float a, float b, float c) {
  float r;
  asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}

// N direct global->LDS copies of 16 bytes per lane under one M0: copy j
// moves lane i's bytes from g[j] + voff[j] + 1024 j to LDS address lbase +
// OFF + 1024 j + 16 i (the instruction offset moves both addresses, so the
// callers fold its 1024 j out of the wave-uniform bases g[j]).  M0 is formed
// by one scalar add and left clobbered.
template <int OFF, int N>
__device__ __forceinline__ void copy_n(const uint64_t (&g)[N], const uint32_t (&voff)[N], uint32_t lbase) {
  static_assert(N == 1 || N == 2 || N == 4, "one, two or four copies");
  if constexpr (N == 4)
    asm volatile(
        "s_add_u32 m0, %4, %5\n\t"
        "global_load_lds_dwordx4 %0, %6\n\t"
        "global_load_lds_dwordx4 %1, %7 offset:1024\n\t"
        "global_load_lds_dwordx4 %2, %8 offset:2048\n\t"
        "global_load_lds_dwordx4 %3, %9 offset:3072"
        :
        : "v"(voff[0]), "v"(voff[1]), "v"(voff[2]), "v"(voff[3]), "s"(lbase), "n"(OFF), "s"(g[0]), "s"(g[1]),
          "s"(g[2]), "s"(g[3])
        : "memory", "scc", "m0");
  else if constexpr (N == 2)
    asm volatile(
        "s_add_u32 m0, %2, %3\n\t"
        "global_load_lds_dwordx4 %0, %4\n\t"
        "global_load_lds_dwordx4 %1, %5 offset:1024"
        :
        : "v"(voff[0]), "v"(voff[1]), "s"(lbase), "n"(OFF), "s"(g[0]), "s"(g[1])
        : "memory", "scc", "m0");
  else
    asm volatile(
        "s_add_u32 m0, %1, %2\n\t"
        "global_load_lds_dwordx4 %0, %3"
        :
        : "v"(voff[0]), "s"(lbase), "n"(OFF), "s"(g[0])
        : "memory", "scc", "m0");
}

// a packed weight pair into an accumulation register (it is only read by MFMAs)
__device__ __forceinline__ uint32_t s1_to_agpr(uint32_t x) {
  uint32_t r;
  asm volatile("v_accvgpr_write_b32 %0, %1" : "=a"(r) : "v"(x));
  return r;
}

__device__ __forceinline__ uint32_t s1_pack(float a, float b) {
  const float2v v = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, f16x2));   // round to nearest
}

// Calls f(std::integral_constant<int, I>) for I = B..E-1: a loop whose
// index is a compile-time constant in every copy of the body.
template <int B, int E, class F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, E>(f);
  }
}

// Geometry of one single-sweep instance: WAVES waves of RT row tiles each.
// The keys are split in four quarters (one per SIMD) and the block's rows in
// WAVES/4 groups; wave w takes key quarter w % 4 and row group w / 4.  Four
// waves (one per SIMD, 512 registers each) hold 64 rows as one group; eight
// (two per SIMD, 256 registers each) hold them as two groups of 32, so that
// two waves share each SIMD's issue slots: a single wave issues a vector
// instruction at most every ~7 cycles, two together every ~3.5.
template <int WAVES, int RT>
struct S1Cfg {
  static constexpr int kWaves = WAVES;
  static constexpr int kThreads = 64 * WAVES;
  static constexpr int kRT = RT;
  static constexpr int kKQ = 4;                            // key quarters
  static constexpr int kRG = WAVES / kKQ;                  // row groups
  static constexpr int kWaveRows = 16 * RT;                // query rows of a wave
  static constexpr int kRows = kWaveRows * kRG;            // query rows per block
  // one LDS ring of key tiles per key quarter, shared by its row groups:
  // each wave copies kCW of a tile's four 1 KB parts, and with more than one
  // group the waves meet at a barrier before every tile's operands are read
  static constexpr int kStages = 8;                        // key tiles in a ring
  static constexpr int kAhead = kStages - 1;               // tiles copied ahead of the one being read
  static constexpr int kCW = 4 / kRG;                      // copies of a tile per wave
  // Logits are double-buffered, so a tile's vector work follows the next
  // tile's MFMAs.  One wave per SIMD also double-buffers the key operands
  // (read before the MFMAs) and keeps the weights in accumulation registers;
  // with two, the operands are read between the MFMAs and the vector work,
  // after the tile's barrier, and the weights fit the ordinary registers.
  static constexpr bool kAgpr = WAVES == 4;
  static constexpr int kKbBuf = WAVES == 4 ? 2 : 1;
  static constexpr int kQCopies = kRows / 4;               // query copies of a block (4 rows each)
  static constexpr int kQMax = (kQCopies + WAVES - 1) / WAVES;   // per wave, at most
  static constexpr int kQMin = kQCopies / WAVES;                   // per wave, at least
  static_assert(kQMin >= 1, "every wave copies part of the queries");
  static_assert(WAVES % kKQ == 0 && kRG >= 1 && 4 % kRG == 0, "whole row groups, whole copies");
};

// FULL: every wave's NT tiles hold keys below N (N = 16 * NT * waves), so
// no tile is skipped or masked.
template <class CF, int NT, bool FULL>
__global__ __launch_bounds__(CF::kThreads) __attribute__((amdgpu_waves_per_eu(CF::kWaves / 4, CF::kWaves / 4)))
void score1_kernel(Score1Args aa) {
  constexpr int D = CF::kAhead;
  constexpr int S = CF::kStages;
  constexpr int RT = CF::kRT;
  constexpr int NW = CF::kWaves;
  constexpr int ROWS = CF::kRows;
  constexpr int NTH = CF::kThreads;
  constexpr int KQ = CF::kKQ;
  constexpr int WROWS = CF::kWaveRows;
  static_assert(NT % S == 0 && NT % 4 == 0, "tiles per wave: a multiple of the ring and of 4");
  const ScoreArgs& a = aa.s;
  __shared__ __attribute__((aligned(16))) char kring[CF::kKQ][S][kS1TileBytes];
  __shared__ __attribute__((aligned(16))) char qbuf[ROWS * kS1RowBytes];
  // byte offset of key j's row in the K pool; entries past N repeat key 0
  __shared__ uint32_t key_off[KQ * NT * 16];
  // per key quarter: row maxima of the first tiles, row sums
  __shared__ __attribute__((aligned(16))) float smax[KQ][ROWS];
  __shared__ __attribute__((aligned(16))) float ssum[KQ][ROWS];
  // per wave: a row sum of the block reached fp16's largest value
  __shared__ __attribute__((aligned(16))) int sbad[NW];
  // byte offset of each of the split's query rows in the unit's queries
  // (rows past R repeat row 0)
  __shared__ uint32_t qrow_off[kS1BlocksPerSplit * ROWS];

  const Geom& g = a.g;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int gq = lane >> 4;
  const int li = lane & 15;
  const int kq = wave % KQ;              // key quarter
  const int rg = wave / KQ;              // row group
  const int rbase = rg * WROWS;          // first block row of this wave
  constexpr int CW = CF::kCW;

  // the row splits of one unit run together on one XCD (its L2 keeps the keys)
  int64_t bid = blockIdx.x;
  if ((a.n_blocks & 7) == 0) bid = (bid & 7) * (a.n_blocks >> 3) + (bid >> 3);
  const int64_t u = bid / a.n_splits;
  const int split = (int)(bid % a.n_splits);
  const int h = (int)(u % g.Hkv);
  const int tw = (int)((u / g.Hkv) % ((int64_t)g.n_trig * g.n_win));
  const int t = tw / g.n_win;
  const int wi = tw - t * g.n_win;
  const int l = (int)(u / ((int64_t)g.Hkv * g.n_trig * g.n_win));
  const int N = g.N;
  float* out = a.n_splits == 1 ? a.scores + u * (int64_t)N : a.partials + (u * a.n_splits + split) * (int64_t)N;
  if (a.status[t] != 0) {
    for (int j = tid; j < N; j += NTH) out[j] = 0.f;
    return;
  }
  const int s = a.trig[t];
  const int p0 = a.win_start[s] + wi * N;
  // (pool and queries in SGPRs: the copies address them as base + 32-bit offset)
  const char* kpool = (const char*)a.k.p[l];
  const char* qunit = a.q + (((int64_t)l * g.n_trig + t) * g.n_win + wi) * g.Wq * g.Hq * (int64_t)kS1RowBytes;
  const int R = g.G * g.Wq;
  const float c = g.scale * kLog2e;
  const int nblk = (R + ROWS - 1) / ROWS;
  const int b0 = split * kS1BlocksPerSplit;
  const int b1 = min(nblk, b0 + kS1BlocksPerSplit);
  const int ntw = aa.ntw;
  const int T = (N + 15) / 16;
  const int wt0 = kq * ntw;                                   // this wave's first tile
  const int nvalid = FULL ? NT : max(0, min(ntw, T - wt0));   // its tiles holding a key < N

  {
    const int32_t* row_pages = a.bt + (int64_t)s * g.max_blocks;
    for (int j = tid; j < KQ * NT * 16; j += NTH) {
      const int pos = p0 + (j < N ? j : 0);
      const uint64_t row = ((uint64_t)row_pages[pos / g.bs] * g.Hkv + h) * g.bs + pos % g.bs;
      key_off[j] = (uint32_t)(row * kS1RowBytes);
    }
    for (int j = tid; j < kS1BlocksPerSplit * ROWS; j += NTH) {
      int gr = b0 * ROWS + j;
      if (gr >= R) gr = 0;
      const int w = gr / g.G, gi = gr - w * g.G;
      qrow_off[j] = (uint32_t)((w * g.Hq + h * g.G + gi) * kS1RowBytes);
    }
  }
  lds_barrier();

  // ---- copies.  Copy r of a tile fills slots r*64 + lane: key row kr =
  // 4r + gq, stored chunk li holding the row's chunk li ^ swz(kr) =
  // li ^ (gq << 2) ^ r; a row's byte offset is a multiple of 256, so the
  // source is row offset ^ chunk byte offset (one three-way XOR).
  const uint32_t cbase = (uint32_t)((li ^ (gq << 2)) << 4);
  // (this wave's copies of a tile: r = rg*CW .. rg*CW + CW-1)
  uint32_t coff[CW];
  auto read_offsets = [&](int tile) __attribute__((always_inline)) {
#pragma unroll
    for (int r = 0; r < CW; ++r) coff[r] = key_off[(wt0 + tile) * 16 + 4 * (rg * CW + r) + gq];
  };
  const uint32_t ring_base = __builtin_amdgcn_readfirstlane(
      (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)&kring[kq][0][0]);
  const uint32_t qbuf_base = __builtin_amdgcn_readfirstlane(
      (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)&qbuf[0]);
  // (one M0 per tile: copy j's base folds out the 1024 j its offset adds)
  uint64_t kbase[CW];
  uint32_t cxor[CW];
#pragma unroll
  for (int j = 0; j < CW; ++j) {
    kbase[j] = (uint64_t)(uintptr_t)kpool - 1024 * j;
    cxor[j] = cbase ^ ((uint32_t)(rg * CW + j) << 4);
  }
  const uint32_t kring_part = ring_base + rg * CW * 1024;
  auto issue_k = [&](auto stage_c) __attribute__((always_inline)) {
    constexpr int stage = decltype(stage_c)::value;
    uint32_t vo[CW];
#pragma unroll
    for (int j = 0; j < CW; ++j) vo[j] = coff[j] ^ cxor[j];
    copy_n<stage * kS1TileBytes>(kbase, vo, kring_part);
  };
  // the query rows of block blk (rows past R repeat row 0), 4 rows a copy:
  // wave w issues copies w, w + NW, ...; copy cq holds rows 4cq + gq
  auto issue_q = [&](int blk) __attribute__((always_inline)) {
    static_for<0, CF::kQMax>([&](auto r_c) __attribute__((always_inline)) {
      constexpr int r = decltype(r_c)::value;
      const int cq = wave + r * NW;
      if (r < CF::kQMin || cq < CF::kQCopies) {
        const int rr = 4 * cq + gq;
        const uint64_t qb[1] = {(uint64_t)(uintptr_t)qunit};
        const uint32_t qoff[1] = {qrow_off[(blk - b0) * ROWS + rr] + (uint32_t)((li ^ s1_swz(rr & 15)) * 16)};
        copy_n<0>(qb, qoff, qbuf_base + cq * 1024);
      }
    });
  };

  // per-lane LDS byte offsets of a tile's key operand (key li, chunk
  // gq*4 + ks; the k step must name the same chunk in every lane)
  int koff[4];
#pragma unroll
  for (int ks = 0; ks < 4; ++ks) koff[ks] = li * kS1RowBytes + (((gq * 4 + ks) ^ s1_swz(li)) * 16);

  // prologue: the first block's queries, then tiles 0..D-1
  issue_q(b0);
  static_for<0, D>([&](auto j_c) __attribute__((always_inline)) {
    read_offsets(decltype(j_c)::value % NT);
    issue_k(std::integral_constant<int, decltype(j_c)::value % S>{});
  });
  read_offsets(D % NT);

  bf16x8 qa[RT][4];                // [row tile][k step]
  bf16x8 kb[CF::kKbBuf][4];        // key operands
  floatx4 acc[2][RT];              // logits: [buffer][row tile], rows 4gq+q, key li
  float m[RT][4], L[RT][4];
  // fp16 weights in pairs of the same row from tiles 2s and 2s+1:
  // es[s][rt][q] = (row (rt, 4gq+q) at key li of tile 2s, of tile 2s+1)
  uint32_t es[NT / 2][RT][4];
  // row-sum selector: A[M][K] = 1 where K holds row M's value (lane (gq, li),
  // word q holds K = 8gq + 2q, +1: row 4gq + q of the pair's two tiles)
  const uint4 rsel = {li == 4 * gq + 0 ? 0x3c003c00u : 0u, li == 4 * gq + 1 ? 0x3c003c00u : 0u,
                      li == 4 * gq + 2 ? 0x3c003c00u : 0u, li == 4 * gq + 3 ? 0x3c003c00u : 0u};
  float ep[RT][4];        // weights of the even tile of the pair in progress
  float colacc[NT / 4];
#pragma unroll
  for (int j = 0; j < NT / 4; ++j) colacc[j] = 0.f;

  auto kread = [&](int stage, int b) __attribute__((always_inline)) {
    const char* sb = &kring[kq][stage][0];
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const uint4 v = *(const uint4*)(sb + koff[ks]);
      __builtin_memcpy(&kb[b][ks], &v, 16);
    }
  };
  // (k step outer: the row tiles' accumulation chains interleave)
  auto form = [&](int b, int kbi) __attribute__((always_inline)) {
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
        acc[b][rt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
            qa[rt][ks], kb[kbi][ks], ks == 0 ? floatx4{0.f, 0.f, 0.f, 0.f} : acc[b][rt], 0, 0, 0);
  };
  // keys of tile `tile` past N: logits -inf
  auto mask = [&](int tile, int b) __attribute__((always_inline)) {
    if (FULL) return;
    if ((wt0 + tile + 1) * 16 > N && (wt0 + tile) * 16 + li >= N) {
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) acc[b][rt] = floatx4{kNegInf, kNegInf, kNegInf, kNegInf};
    }
  };
  // a finished pair: round to fp16, add both to the row sums and store.  The
  // row sums are a matrix product too: with the selector as A, output row M
  // of the pair's operand is the sum of row M's two values in every key
  // column, accumulated over the block in L (the lane's rows and keys of the
  // logits' layout): one MFMA per row tile and tile pair
  auto finish_pair = [&](int sp, const float (&eo)[RT][4]) __attribute__((always_inline)) {
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      uint32_t hp[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) hp[q] = s1_pack(ep[rt][q], eo[rt][q]);
      const uint4 bv = {hp[0], hp[1], hp[2], hp[3]};
      const floatx4 s = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, rsel),
                                                               __builtin_bit_cast(f16x8, bv),
                                                               floatx4{L[rt][0], L[rt][1], L[rt][2], L[rt][3]}, 0, 0, 0);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        L[rt][q] = s[q];
        // one wave per SIMD keeps them in accumulation registers; with two
        // waves (256 registers each) everything fits the ordinary ones
        if constexpr (CF::kAgpr) es[sp][rt][q] = s1_to_agpr(hp[q]);
        else es[sp][rt][q] = hp[q];
      }
    }
  };
  // weights of tile `tile` from x = logit * c - m (given as e's exponent)
  auto weights = [&](int tile, const float (&e)[RT][4]) __attribute__((always_inline)) {
    if (tile & 1) {
      finish_pair(tile >> 1, e);
    } else {
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int q = 0; q < 4; ++q) ep[rt][q] = e[rt][q];
      // the pair's odd tile holds no key below N
      if (!FULL && tile + 1 >= nvalid) {
        const float zero[RT][4] = {};
        finish_pair(tile >> 1, zero);
      }
    }
  };
  auto vexp = [&](int tile, int b) __attribute__((always_inline)) {
    float e[RT][4];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int q = 0; q < 4; ++q) e[rt][q] = __builtin_amdgcn_exp2f(fmaf(acc[b][rt][q], c, -m[rt][q]));
    weights(tile, e);
  };
  // row reference from every wave's maxima mx of the raw logits, per lane
  // (c > 0, so the maximum of x = logit * c is c times theirs)
  auto share_max = [&](float (&mx)[RT][4]) __attribute__((always_inline)) {
    if constexpr (RT == 4) {
      // lane li holds row (li >> 2, 4gq + (li & 3))'s maximum: it forms that
      // row's reference from every wave's, and the wave shares the 64
      // through its own row of ssum (no wave reads ssum between a block's
      // sum exchange and the next one, which this barrier precedes; LDS
      // operations of a wave complete in order)
      const int rrow = rbase + (li >> 2) * 16 + 4 * gq + (li & 3);
      smax[kq][rrow] = reduce_scatter16<true>(reinterpret_cast<float(&)[16]>(mx), li);
      lds_barrier();
      static_assert(KQ == 4, "four key quarters");
      const float v = s1_max3(s1_max3(smax[0][rrow], smax[1][rrow], smax[2][rrow]), smax[3][rrow], smax[3][rrow]);
      ssum[kq][rrow] = fmaf(v, c, -kS1Headroom);
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        const float4 mm = *(const float4*)&ssum[kq][rbase + rt * 16 + 4 * gq];
        m[rt][0] = mm.x;
        m[rt][1] = mm.y;
        m[rt][2] = mm.z;
        m[rt][3] = mm.w;
      }
      return;
    } else {
      if constexpr (RT == 2) {
        dpp_reduce16xn<true, RT * 4>(reinterpret_cast<float(&)[RT * 4]>(mx));
      } else {
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
#pragma unroll
          for (int q = 0; q < 4; ++q) mx[rt][q] = dpp_max16(mx[rt][q]);
      }
      if (li == 0) {
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
          *(float4*)&smax[kq][rbase + rt * 16 + 4 * gq] = float4{mx[rt][0], mx[rt][1], mx[rt][2], mx[rt][3]};
      }
    }
    lds_barrier();
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      float4 v = *(const float4*)&smax[0][rbase + rt * 16 + 4 * gq];
#pragma unroll
      for (int w = 1; w < KQ; w += 2) {
        const float4 o = *(const float4*)&smax[w][rbase + rt * 16 + 4 * gq];
        const float4 p = w + 1 < KQ ? *(const float4*)&smax[w + 1][rbase + rt * 16 + 4 * gq] : o;
        v = float4{s1_max3(v.x, o.x, p.x), s1_max3(v.y, o.y, p.y), s1_max3(v.z, o.z, p.z), s1_max3(v.w, o.w, p.w)};
      }
      m[rt][0] = fmaf(v.x, c, -kS1Headroom);
      m[rt][1] = fmaf(v.y, c, -kS1Headroom);
      m[rt][2] = fmaf(v.z, c, -kS1Headroom);
      m[rt][3] = fmaf(v.w, c, -kS1Headroom);
    }
  };

  // wait for tile 0's copies (the queries are older still) and publish both
  wait_vm<CW * (D - 1)>();
  lds_barrier();
  kread(0, 0);

  // vmcnt for tile t+1's copies at iteration t: tiles t+2..t+D-1 are newer,
  // and the next block's queries when copied in between
  auto wait_next = [&](auto it_c) __attribute__((always_inline)) {
    constexpr int it = decltype(it_c)::value;
    if constexpr (kS1QIt <= it - 1 && it + 1 <= kS1QIt + D) wait_vm<CW * (D - 2) + CF::kQMin>();
    else wait_vm<CW * (D - 2)>();
    // the other row groups' parts of the tile
    if constexpr (CF::kRG > 1) lds_barrier();
  };

  // One pass over the block's key tiles.  Iteration it: logits of tile it,
  // weights of tile it-1, operands of tile it+1 (the next block's tile 0 at
  // the end), copies of tile it+D into the stage tile it-1 left.  With one
  // wave per SIMD the operands are read first, into the other buffer; with
  // two, after the logits' MFMAs are issued (and the tile's barrier), so the
  // weights' vector work overlaps both the MFMAs and the reads.
  auto run_block = [&](bool m_given, int blk) __attribute__((always_inline)) {
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int q = 0; q < 4; ++q) L[rt][q] = 0.f;
    static_for<0, NT>([&](auto it_c) __attribute__((always_inline)) {
      constexpr int it = decltype(it_c)::value;
      constexpr int b = it & 1;                             // logits of tile it
      constexpr int bp = b ^ 1;                             // of tile it-1
      constexpr int kbi = CF::kKbBuf == 2 ? (it & 1) : 0;   // operands of tile it
      if constexpr (CF::kKbBuf == 2) {
        wait_next(it_c);
        kread((it + 1) % S, kbi ^ 1);
      }
      if (it < nvalid) {
        form(b, kbi);
        mask(it, b);
      }
      if constexpr (CF::kKbBuf == 1) {
        wait_next(it_c);
        kread((it + 1) % S, 0);
      }
      if constexpr (it == 1) {
        // the shared reference, from every wave's tile 0
        if (!m_given) {
          float mx[RT][4];   // (share_max reduces its argument in place)
#pragma unroll
          for (int rt = 0; rt < RT; ++rt)
#pragma unroll
            for (int q = 0; q < 4; ++q) mx[rt][q] = nvalid > 0 ? acc[bp][rt][q] : kNegInf;
          share_max(mx);
        }
        if (nvalid > 0) vexp(0, bp);
      } else if constexpr (it > 1) {
        if (it - 1 < nvalid) vexp(it - 1, bp);
      }
      issue_k(std::integral_constant<int, (it + D) % S>{});
      read_offsets((it + D + 1) % NT);
      // (the split's last block copies its own rows again, unused)
      if (it == kS1QIt) issue_q(min(blk + 1, b1 - 1));
    });
    if (NT - 1 < nvalid) vexp(NT - 1, (NT - 1) & 1);
  };

  // exact row maxima over this wave's keys, read straight from the pool
  auto exact_max = [&]() {
    float mx[RT][4];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int q = 0; q < 4; ++q) mx[rt][q] = kNegInf;
    for (int tile = 0; tile < nvalid; ++tile) {
      const char* src = kpool + key_off[(wt0 + tile) * 16 + li] + gq * 64;
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const uint4 v = *(const uint4*)(src + ks * 16);
        __builtin_memcpy(&kb[0][ks], &v, 16);
      }
      form(0, 0);
      mask(tile, 0);
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int q = 0; q < 4; ++q) mx[rt][q] = fmaxf(mx[rt][q], acc[0][rt][q]);
    }
    share_max(mx);
    // kb[0] is the next pass's tile 0 again, from its stage
    kread(0, 0);
  };

  for (int blk = b0; blk < b1; ++blk) {
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const uint4 v =
            *(const uint4*)(qbuf + (rbase + rt * 16 + li) * kS1RowBytes + (((gq * 4 + ks) ^ s1_swz(li)) * 16));
        __builtin_memcpy(&qa[rt][ks], &v, 16);
      }
    float ltot[RT][4];
    float lrow = 0.f;   // (four row tiles) the total of this lane's row of the reduce-scatter
    bool m_given = false;
    for (int pass = 0; pass < 2; ++pass) {
      run_block(m_given, blk);
      // this wave's row sums, then every wave's; a wave's overflow flag:
      // any of its row sums reached fp16's largest value (rows past R repeat
      // row 0, so they overflow only where row 0 did)
      bool over;
      if constexpr (RT == 4) {
        // lane li holds row (li >> 2, 4gq + (li & 3))'s sum (NaN, never
        // below fp16's largest value, where the selector product met an
        // infinity)
        const float r = reduce_scatter16<false>(reinterpret_cast<float(&)[16]>(L), li);
        ssum[kq][rbase + (li >> 2) * 16 + 4 * gq + (li & 3)] = r * (1.f / kS1WScale);
        over = !(r < kF16Max);
      } else {
        if constexpr (RT == 2) {
          dpp_reduce16xn<false, RT * 4>(reinterpret_cast<float(&)[RT * 4]>(L));
        } else {
#pragma unroll
          for (int rt = 0; rt < RT; ++rt)
#pragma unroll
            for (int q = 0; q < 4; ++q) L[rt][q] = dpp_sum16(L[rt][q]);
        }
        if (li == 0) {
          constexpr float s = 1.f / kS1WScale;
#pragma unroll
          for (int rt = 0; rt < RT; ++rt)
            *(float4*)&ssum[kq][rbase + rt * 16 + 4 * gq] =
                float4{L[rt][0] * s, L[rt][1] * s, L[rt][2] * s, L[rt][3] * s};
        }
        // (each sum on its own: a row tile's sums are all NaN where two of
        // its values overflowed, 0 times infinity in the selector product,
        // and a maximum would pass over them)
        over = false;
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
#pragma unroll
          for (int q = 0; q < 4; ++q) over |= !(L[rt][q] < kF16Max);
      }
      {
        const bool wbad = __builtin_amdgcn_ballot_w64(over) != 0;
        if (lane == 0) sbad[wave] = wbad;
      }
      // the next block's queries are in LDS once the copies issued after
      // them are at most the last 4*(D-1)
      wait_vm<CW * (D - 1)>();
      lds_barrier();
      int anybad = 0;
#pragma unroll
      for (int w = 0; w < NW; w += 4) {
        const int4 f = *(const int4*)&sbad[w];
        anybad |= f.x | f.y | f.z | f.w;
      }
      if (__builtin_amdgcn_readfirstlane(anybad) == 0) {
        if constexpr (RT == 4) {
          const int row = rbase + (li >> 2) * 16 + 4 * gq + (li & 3);
          lrow = ssum[0][row];
#pragma unroll
          for (int w = 1; w < KQ; ++w) lrow += ssum[w][row];
          break;
        }
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
          float4 v[KQ];
#pragma unroll
          for (int w = 0; w < KQ; ++w) v[w] = *(const float4*)&ssum[w][rbase + rt * 16 + 4 * gq];
          ltot[rt][0] = v[0].x;
          ltot[rt][1] = v[0].y;
          ltot[rt][2] = v[0].z;
          ltot[rt][3] = v[0].w;
#pragma unroll
          for (int w = 1; w < KQ; ++w) {
            ltot[rt][0] += v[w].x;
            ltot[rt][1] += v[w].y;
            ltot[rt][2] += v[w].z;
            ltot[rt][3] += v[w].w;
          }
        }
        break;
      }
      exact_max();
      m_given = true;
    }

    // ---- weighted column sums: per tile pair, RT fp16 MFMAs over the
    // block's rows, one per row tile.  B operand (pair s, row tile rt):
    // element j = 2q + par of lane (gq, li) holds row (rt, 4gq + q) of tile
    // 2s + par at key li.  A operand of row tile rt: lane (gq, li) -- output
    // row li -- supplies the weight of that row to the elements of tile
    // parity li >> 3 and 0 to the others, the high fp16 part for even li and
    // the low part for odd li.  Output rows 4gq'+i then hold, for key li',
    // the high (i even) or low (i odd) sum of tile 2s + (gq' >> 1), so a lane
    // adds its own first two results.  (A lane's part of a weight goes to
    // the low or high half of its word by a shift; even lanes take the high
    // fp16 part, odd lanes what it leaves.)
    const uint32_t half_shift = (uint32_t)(li >> 3) * 16;
    const bool low_part = (li & 1) != 0;
    const bool last_block = (blk + 1) * ROWS > R;
    // Four row tiles: each lane forms the weight of its one row of the
    // reduce-scatter as an fp16 pair (high | low << 16), and the wave
    // shares the pairs through its own row of smax (free until the next
    // block's exchange; LDS operations of a wave complete in order); a
    // lane's A-operand word is then one byte permutation of a pair.
    uint32_t wrow[RT][4];
    if constexpr (RT == 4) {
      const int rrow = (li >> 2) * 16 + 4 * gq + (li & 3);   // the lane's row within the wave's rows
      float w = __builtin_amdgcn_rcpf(lrow);
      if (last_block && blk * ROWS + rbase + rrow >= R) w = 0.f;   // rows past R weigh nothing
      const _Float16 hi = (_Float16)w;
      const _Float16 lo = (_Float16)(w - (float)hi);
      uint32_t* share = (uint32_t*)&smax[kq][rbase];
      share[rrow] = (uint32_t)__builtin_bit_cast(uint16_t, hi) | ((uint32_t)__builtin_bit_cast(uint16_t, lo) << 16);
      // bytes of the pair into the word: the high part (even li) or the low
      // part (odd li), at the low (li < 8) or high half
      const uint32_t sel = (li & 1) ? ((li >> 3) ? 0x03020c0cu : 0x0c0c0302u) : ((li >> 3) ? 0x01000c0cu : 0x0c0c0100u);
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        const uint4 p = *(const uint4*)&share[rt * 16 + 4 * gq];
        wrow[rt][0] = __builtin_amdgcn_perm(p.x, p.x, sel);
        wrow[rt][1] = __builtin_amdgcn_perm(p.y, p.y, sel);
        wrow[rt][2] = __builtin_amdgcn_perm(p.z, p.z, sel);
        wrow[rt][3] = __builtin_amdgcn_perm(p.w, p.w, sel);
      }
    }
    // (the exchanged sums carry 2^-21, so 1 / sum is the scaled weight)
    auto weights_of = [&](int rt, uint32_t (&wa)[4]) __attribute__((always_inline)) {
      if constexpr (RT == 4) {
#pragma unroll
        for (int q = 0; q < 4; ++q) wa[q] = wrow[rt][q];
        return;
      }
      float wt[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) wt[q] = __builtin_amdgcn_rcpf(ltot[rt][q]);
      if (last_block) {   // (uniform) rows past R weigh nothing
#pragma unroll
        for (int q = 0; q < 4; ++q)
          if (blk * ROWS + rbase + rt * 16 + 4 * gq + q >= R) wt[q] = 0.f;
      }
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float w = wt[q];
        const float hi = (float)(_Float16)w;
        const _Float16 part = (_Float16)(w - (low_part ? hi : 0.f));
        wa[q] = (uint32_t)__builtin_bit_cast(uint16_t, part) << half_shift;
      }
    };
    auto mfma_w = [&](const uint32_t (&wa)[4], int sp, int rt, floatx4 cin) __attribute__((always_inline)) {
      const uint4 av = {wa[0], wa[1], wa[2], wa[3]};
      const uint4 ev = {es[sp][rt][0], es[sp][rt][1], es[sp][rt][2], es[sp][rt][3]};
      return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, av), __builtin_bit_cast(f16x8, ev), cin,
                                                    0, 0, 0);
    };
    auto add_pair = [&](auto s_c, const floatx4& cs) __attribute__((always_inline)) {
      constexpr int sp = decltype(s_c)::value;
      // lane (gq, li): tile 2sp + (gq >> 1), high + low (added by value
      // selection, which keeps colacc in registers)
      const float v = cs[0] + cs[1];
      colacc[sp >> 1] += (gq & 1) == (sp & 1) ? v : 0.f;
    };
    if constexpr (FULL) {
      // row tile by row tile: its weights, then its MFMA for every pair (one
      // accumulator per pair), so a tile's weight arithmetic overlaps the
      // previous tile's MFMAs
      floatx4 cs[NT / 2];
      static_for<0, RT>([&](auto rt_c) __attribute__((always_inline)) {
        constexpr int rt = decltype(rt_c)::value;
        uint32_t wa[4];
        weights_of(rt, wa);
        static_for<0, NT / 2>([&](auto s_c) __attribute__((always_inline)) {
          constexpr int sp = decltype(s_c)::value;
          cs[sp] = mfma_w(wa, sp, rt, rt == 0 ? floatx4{0.f, 0.f, 0.f, 0.f} : cs[sp]);
        });
      });
      static_for<0, NT / 2>([&](auto s_c) __attribute__((always_inline)) { add_pair(s_c, cs[decltype(s_c)::value]); });
    } else {
      uint32_t wa[RT][4];
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) weights_of(rt, wa[rt]);
      static_for<0, NT / 2>([&](auto s_c) __attribute__((always_inline)) {
        constexpr int sp = decltype(s_c)::value;
        if (2 * sp < nvalid) {
          floatx4 cs = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int rt = 0; rt < RT; ++rt) cs = mfma_w(wa[rt], sp, rt, cs);
          add_pair(s_c, cs);
        }
      });
    }
  }
  wait_vm<0>();
  if constexpr (CF::kRG > 1) {
    // the row groups' column sums of one key quarter, added through its
    // ring once every wave's copies have landed
    static_assert((CF::kRG - 1) * NT / 4 * 64 * 4 <= S * kS1TileBytes, "column sums fit a ring");
    lds_barrier();
    float* part = (float*)&kring[kq][0][0];
    if (rg != 0) {
#pragma unroll
      for (int j = 0; j < NT / 4; ++j) part[((rg - 1) * (NT / 4) + j) * 64 + lane] = colacc[j];
    }
    lds_barrier();
    if (rg != 0) return;
#pragma unroll
    for (int r = 1; r < CF::kRG; ++r)
#pragma unroll
      for (int j = 0; j < NT / 4; ++j) colacc[j] += part[((r - 1) * (NT / 4) + j) * 64 + lane];
  }
  // colacc[j] of lane (gq, li): pair 2j + (gq & 1), tile 2(2j + (gq & 1)) + (gq >> 1)
#pragma unroll
  for (int j = 0; j < NT / 4; ++j) {
    const int tile = 2 * (2 * j + (gq & 1)) + (gq >> 1);
    const int key = (wt0 + tile) * 16 + li;
    if (tile < nvalid && key < N) out[key] = colacc[j] * (1.f / kS1WScale);
  }
}

// Row tiles per wave.  At most four (512 rows per workgroup), two for fp32
// with 128-wide heads, whose operands take twice the registers.  Fewer when
// a unit has few query rows (scoring by a buffer or an observation window):
// the count that pads the unit's rows least, the larger one on a tie, since
// each workgroup streams all of the unit's keys.
int row_tiles(const Geom& g) {
  const int max_rt = (g.dtype == KARA_F32 && g.d == 128) ? 2 : 4;
  const int64_t rows = (int64_t)g.G * g.Wq;
  int best = max_rt;
  int64_t best_pad = -1;
  for (int rt = max_rt; rt >= 1; --rt) {
    const int64_t per = (int64_t)kScoreWaves * 16 * rt;
    const int64_t pad = (rows + per - 1) / per * per - rows;
    if (best_pad < 0 || pad < best_pad) {
      best = rt;
      best_pad = pad;
    }
  }
  return best;
}

template <int DT, int D>
hipError_t launch_d(const ScoreArgs& a, int rt, hipStream_t stream) {
  const dim3 grid((unsigned)a.n_blocks), block(kScoreThreads);
  if constexpr (DT == KARA_F32 && D == 128) {
    if (rt == 1) hipLaunchKernelGGL((score_kernel<DT, D, 1>), grid, block, 0, stream, a);
    else hipLaunchKernelGGL((score_kernel<DT, D, 2>), grid, block, 0, stream, a);
  } else {
    switch (rt) {
      case 1: hipLaunchKernelGGL((score_kernel<DT, D, 1>), grid, block, 0, stream, a); break;
      case 2: hipLaunchKernelGGL((score_kernel<DT, D, 2>), grid, block, 0, stream, a); break;
      case 3: hipLaunchKernelGGL((score_kernel<DT, D, 3>), grid, block, 0, stream, a); break;
      default: hipLaunchKernelGGL((score_kernel<DT, D, 4>), grid, block, 0, stream, a); break;
    }
  }
  return hipGetLastError();
}

// The single-sweep instance the launches use.
using S1Use = S1Cfg<4, 4>;

// Tiles per wave of the single-sweep kernel for g, 0 where the two-sweep
// kernel runs: bf16 with d = 128 and 512 < N <= 2048 (its weights of the
// block's rows x N/waves keys fit the waves' accumulation registers).
int single_sweep_tiles(const Geom& g) {
  if (g.dtype != KARA_BF16 || g.d != 128 || g.N <= 512 || g.N > 2048) return 0;
  // its copies address a layer's K pool and a unit's queries by 32-bit offsets
  if ((uint64_t)g.num_pages * g.Hkv * g.bs * kS1RowBytes > 0xffffffffull) return 0;
  if ((uint64_t)g.Wq * g.Hq * kS1RowBytes > 0xffffffffull) return 0;
  constexpr int KQ = S1Use::kKQ;
  const int ntw = ((g.N + 15) / 16 + KQ - 1) / KQ;
  // the smallest multiple of 8 (of the ring, and of 4) holding ntw
  static_assert(8 % S1Use::kStages == 0, "instances come in steps of 8 tiles");
  return (ntw + 7) / 8 * 8;
}

template <int NT>
void launch_s1(const Score1Args& a1, bool full, hipStream_t stream) {
  const dim3 grid((unsigned)a1.s.n_blocks), block(S1Use::kThreads);
  if (full) hipLaunchKernelGGL((score1_kernel<S1Use, NT, true>), grid, block, 0, stream, a1);
  else hipLaunchKernelGGL((score1_kernel<S1Use, NT, false>), grid, block, 0, stream, a1);
}

}  // namespace

ScorePlan plan_score(const Geom& g, int64_t n_units) {
  (void)n_units;
  ScorePlan sp{};
  const int64_t rows = (int64_t)g.G * g.Wq;
  sp.single_nt = single_sweep_tiles(g);
  if (sp.single_nt) {
    sp.rows_wg = S1Use::kRows * kS1BlocksPerSplit;
  } else {
    sp.rows_wg = kScoreWaves * 16 * row_tiles(g);
  }
  sp.n_splits = (int)((rows + sp.rows_wg - 1) / sp.rows_wg);
  return sp;
}

hipError_t launch_score(const Geom& g, const ScorePlan& sp, int n_layers, const void* q,
                        const PoolPtrs& k_pools, const int32_t* trig, const int32_t* block_table,
                        const int32_t* win_start, const int32_t* status, float* partials,
                        float* scores, hipStream_t stream) {
  ScoreArgs a;
  a.g = g;
  a.q = (const char*)q;
  a.k = k_pools;
  a.trig = trig;
  a.bt = block_table;
  a.win_start = win_start;
  a.status = status;
  a.partials = partials;
  a.scores = scores;
  a.n_splits = sp.n_splits;
  a.n_blocks = (int64_t)n_layers * g.n_trig * g.n_win * g.Hkv * sp.n_splits;
  if (a.n_blocks == 0) return hipSuccess;
  const int rt = sp.rows_wg / (kScoreWaves * 16);
  hipError_t e;
  if (sp.single_nt) {
    Score1Args a1;
    a1.s = a;
    a1.ntw = ((g.N + 15) / 16 + S1Use::kKQ - 1) / S1Use::kKQ;
    const bool full = g.N == S1Use::kKQ * 16 * sp.single_nt;
    switch (sp.single_nt / 8) {
      case 2: launch_s1<16>(a1, full, stream); break;
      case 3: launch_s1<24>(a1, full, stream); break;
      default: launch_s1<32>(a1, full, stream); break;
    }
    e = hipGetLastError();
  } else if (g.dtype == KARA_BF16)
    e = g.d == 128 ? launch_d<KARA_BF16, 128>(a, rt, stream) : launch_d<KARA_BF16, 64>(a, rt, stream);
  else
    e = g.d == 128 ? launch_d<KARA_F32, 128>(a, rt, stream) : launch_d<KARA_F32, 64>(a, rt, stream);
  if (e != hipSuccess || sp.n_splits == 1) return e;
  const int64_t units = a.n_blocks / sp.n_splits;
  hipLaunchKernelGGL(split_sum_kernel, dim3((unsigned)units, (unsigned)((g.N + 255) / 256)), dim3(256), 0, stream,
                     partials, scores, g.N, sp.n_splits);
  return hipGetLastError();
}

}  // namespace kara
