// Window scoring, Eq. (4) of Kara: A = colsum(softmax(Q_W K_{W\U}^T / sqrt(d)))
// per (sequence, layer, KV head), all G query heads of the group acting as
// queries of their KV head.
//
// Single pass over the logits.  A workgroup of 8 waves owns 32*RG query rows
// at a time and all N = W-U keys, split over CG column groups (CG*RG = 8).
// Every wave holds the logits of its 32 rows x 16*NT keys in registers; its
// two 16-row MFMA tiles share each key operand read from LDS.  Keys (and the
// next row block's queries) stream into LDS by direct global->LDS copies
// through a three-stage ring, so no register is spent on staging and the
// copies of later chunks overlap the MFMAs and exponentials of the current
// one.  Per chunk each lane updates a running row maximum over its own keys
// (earlier exponentials are rescaled only when a chunk exceeds it by more
// than 2^32), exponentiates and accumulates row sums; once all keys are
// seen, row maximum and sum are combined across lanes (shuffles) and column
// groups (LDS), and each lane adds its rows' normalised probabilities to
// fixed per-(lane group, column) slots in LDS.  The workgroup finally
// reduces those slots in a fixed order and writes one partial column sum per
// row split; the selection kernel adds the splits in order.  No
// floating-point atomics, so the scores are bit-reproducible.
#include "kara_internal.h"

namespace kara {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int kScoreThreads = 512;
constexpr int kScoreWaves = kScoreThreads / 64;
constexpr int kLdsLimit = 160 * 1024;
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
  float* partials;            // [units][n_splits][N] (unused with one split)
  float* scores;              // [units][N]
  uint32_t* done;             // [units] splits finished; zeroed by the validation kernel
  int n_splits, n_rb;
  int64_t n_blocks;
};

// Static geometry of one kernel instance.
template <int DT, int D, int NT, int CG>
struct Cfg {
  static constexpr int kES = DT == KARA_BF16 ? 2 : 4;
  static constexpr int kRowBytes = D * kES;             // one key or query row
  static constexpr int kCPR = kRowBytes / 16;            // 16-byte chunks per row
  static constexpr int kSwz = kCPR < 16 ? kCPR - 1 : 15; // XOR swizzle mask
  static constexpr int kRG = kScoreWaves / CG;
  static constexpr int kRows = 32 * kRG;                 // query rows per row block
  static constexpr int kNCol = CG * NT * 16;
  static constexpr int kPartBytes = kRG * kNCol * 4;
  static constexpr int kSmallBytes = kNCol * 4 + 2 * kRG * CG * 32 * 4;
  // query tile, padded so every thread issues the same number of copies
  static constexpr int kQL = (kRows * kCPR + kScoreThreads - 1) / kScoreThreads;
  static constexpr int kQBytes = kQL * kScoreThreads * 16;
  // key chunks: TPS 16-key tiles per column group, kStages stages in a ring;
  // the stage of a chunk must be a compile-time function of the chunk index,
  // so kStages divides the chunks per row block
  static constexpr int kTpsMin0 = kScoreThreads / (16 * kCPR * CG);
  static constexpr int kTpsMin = kTpsMin0 < 1 ? 1 : kTpsMin0;
  static constexpr int stages_for(int tps) {
    return (NT / tps) % 4 == 0 ? 4 : (NT / tps) % 2 == 0 ? 2 : 1;
  }
  static constexpr int lds_bytes(int tps) {
    return stages_for(tps) * CG * tps * 16 * kRowBytes + kQBytes + kPartBytes + kSmallBytes;
  }
  static constexpr int fit_tps() {
    int tps = (32768 / kRowBytes / 16) / CG;           // ~32 KB stages
    if (tps > NT / 4) tps = NT / 4;                    // at least four chunks per row block
    if (tps < kTpsMin) tps = kTpsMin;
    if (tps > NT) tps = NT;
    while (tps > kTpsMin && lds_bytes(tps) > kLdsLimit) tps /= 2;
    return tps;
  }
  static constexpr int kTPS = fit_tps();
  static constexpr int kStages = stages_for(kTPS);
  static constexpr int kKeys = CG * kTPS * 16;           // keys per stage
  static constexpr int kStageBytes = kKeys * kRowBytes;
  static constexpr int kL = kKeys * kCPR / kScoreThreads; // copies per thread per stage
  static constexpr int kNCH = NT / kTPS;                  // chunks per row block
  static_assert(NT % kTPS == 0, "chunks must tile the wave's keys");
  static_assert(kNCH % kStages == 0, "stage index must be static");
  static_assert((kKeys * kCPR) % kScoreThreads == 0, "stage copies must be uniform over threads");
  static_assert(lds_bytes(kTPS) <= kLdsLimit, "LDS budget");
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
// every copy); the kernel waits explicitly with wait_vm().  M0 is restored.
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
// for explicitly with wait_vm() first.
__device__ inline void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

template <int N>
__device__ inline void wait_vm() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

template <int DT, int D, int NT, int CG>
__global__ __launch_bounds__(kScoreThreads) void score_kernel(ScoreArgs a) {
  using C = Cfg<DT, D, NT, CG>;
  using Op = Operand<DT, D>;
  constexpr int RG = C::kRG;
  constexpr int TPS = C::kTPS;
  constexpr int NCH = C::kNCH;
  constexpr int CPR = C::kCPR;
  constexpr int S = C::kStages;
  constexpr int P = S - 1;                // prefetch distance in chunks
  constexpr int kL = C::kL, kQL = C::kQL;
  constexpr int KC = Op::kChunks;
  constexpr bool kEarlyQ = S == 4;        // next row block's queries fetched at chunk 1

  __shared__ __attribute__((aligned(16))) char kbuf[S * C::kStageBytes];
  __shared__ __attribute__((aligned(16))) char qbuf[C::kQBytes];
  // column sums of this workgroup's rows, per row group; slot (rg, column)
  // is updated by exactly one lane after each row block
  __shared__ float part[RG][C::kNCol];
  __shared__ float red_max[RG][CG][32];
  __shared__ float red_sum[RG][CG][32];
  // byte offset / 16 of every compressible key row in the K pool (the block
  // table resolved once per workgroup); padding entries repeat row 0
  __shared__ uint32_t key_off[C::kNCol];

  const Geom& g = a.g;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform, kept in an SGPR
  const int cg = wave % CG;
  const int rg = wave / CG;
  const int gq = lane >> 4;     // lane group: rows 4*gq..4*gq+3 of a 16-row tile
  const int li = lane & 15;     // key of a 16-key tile / row of the query operand

  // Blocks are dealt round-robin to the 8 XCDs; renumber so that the row
  // splits of one unit run together on one XCD and share its L2 copy of the
  // unit's keys.
  int64_t bid = blockIdx.x;
  if ((a.n_blocks & 7) == 0) bid = (bid & 7) * (a.n_blocks >> 3) + (bid >> 3);
  const int64_t u = bid / a.n_splits;
  const int split = (int)(bid % a.n_splits);
  const int h = (int)(u % g.Hkv);
  const int t = (int)((u / g.Hkv) % g.n_trig);
  const int l = (int)(u / ((int64_t)g.Hkv * g.n_trig));
  const int N = g.N;
  float* out = a.n_splits == 1 ? a.scores + u * (int64_t)N : a.partials + (u * a.n_splits + split) * (int64_t)N;

  if (a.status[t] != 0) {
    float* sc = a.scores + u * (int64_t)N;
    for (int j = tid; j < N; j += kScoreThreads) sc[j] = 0.f;
    return;
  }
  const int s = a.trig[t];
  const int p0 = a.win_start[s];
  {
    const int32_t* row_pages = a.bt + (int64_t)s * g.max_blocks;
    for (int j = tid; j < C::kNCol; j += kScoreThreads) {
      const int pos = p0 + (j < N ? j : 0);        // padding keys: any valid row
      const uint64_t row = ((uint64_t)row_pages[pos / g.bs] * g.Hkv + h) * g.bs + pos % g.bs;
      key_off[j] = (uint32_t)(row * (C::kRowBytes / 16));
    }
    for (int i = tid; i < RG * C::kNCol; i += kScoreThreads) (&part[0][0])[i] = 0.f;
  }
  // the key offsets must be in LDS before the copies below compute addresses
  lds_barrier();

  const char* kpool = (const char*)a.k.p[l];
  const char* qunit = a.q + ((int64_t)l * g.n_trig + t) * g.W * g.Hq * (int64_t)C::kRowBytes;
  const int R = g.G * g.W;
  const float c = g.scale * kLog2e;

  // ---- copies into LDS (every thread issues exactly kL / kQL per call) ----
  // Key copy r of this thread fills stage slot r*512 + tid: key row
  // kr = slot / CPR of the stage, 16-byte chunk (slot % CPR) ^ (kr & kSwz).
  // Only the key index depends on the chunk, by a compile-time step, so per
  // copy the address costs one LDS read of the key table and one shift-add.
  const char* kpool_c[kL];
  int kidx0[kL];
#pragma unroll
  for (int r = 0; r < kL; ++r) {
    const int slot = r * kScoreThreads + tid;
    const int kr = slot / CPR;
    const int chunk = (slot % CPR) ^ (kr & C::kSwz);
    kpool_c[r] = kpool + chunk * 16;
    kidx0[r] = (kr / (TPS * 16)) * NT * 16 + kr % (TPS * 16);
  }
  auto load_keys = [&](int ch, int stage) {
    char* sbase = kbuf + stage * C::kStageBytes;
#pragma unroll
    for (int r = 0; r < kL; ++r) {
      const uint32_t off = key_off[kidx0[r] + ch * TPS * 16];
      copy16(kpool_c[r] + (uint64_t)off * 16, sbase + (r * kScoreWaves + wave) * 1024);
    }
  };
  auto load_queries = [&](int rb) {
#pragma unroll
    for (int r = 0; r < kQL; ++r) {
      const int slot = r * kScoreThreads + tid;
      const int row = slot / CPR;
      const int chunk = (slot % CPR) ^ (row & C::kSwz);
      int rr = rb * C::kRows + row;
      if (row >= C::kRows || rr >= R) rr = 0;      // padding rows: any valid row
      const int w = rr / g.G, gi = rr - w * g.G;
      const char* src = qunit + ((int64_t)w * g.Hq + h * g.G + gi) * C::kRowBytes + chunk * 16;
      copy16(src, qbuf + (r * kScoreWaves + wave) * 1024);
    }
  };

  // per-lane LDS byte offsets of the operand chunks (rows are multiples of 16
  // plus li, so the swizzle term depends on the lane only)
  int koff[KC], qoff[KC];
#pragma unroll
  for (int ks = 0; ks < KC; ++ks) {
    const int sw = ((gq * KC + ks) ^ (li & C::kSwz)) * 16;
    koff[ks] = (cg * TPS * 16 + li) * C::kRowBytes + sw;
    qoff[ks] = (rg * 32 + li) * C::kRowBytes + sw;
  }

  const int rb0 = (int)((int64_t)split * a.n_rb / a.n_splits);
  const int rb1 = (int)((int64_t)(split + 1) * a.n_rb / a.n_splits);
  const int n_it = (rb1 - rb0) * NCH;

  // prologue: queries of the first row block, then the first key chunks
  load_queries(rb0);
#pragma unroll
  for (int j = 0; j < (P > 0 ? P : 1); ++j)
    if (j < n_it) load_keys(j % NCH, j % S);

  Op qa[2];
  floatx4 acc[2][NT];
  int it = 0;
  for (int rb = rb0; rb < rb1; ++rb) {
    // ---- MFMA phase: all keys of the row block, chunk by chunk ----
#pragma unroll
    for (int ch = 0; ch < NCH; ++ch, ++it) {
      // Wait for chunk `it` (and, at a row block start, the queries, issued
      // before it).  Per thread copies are issued in the order Q(rb0),
      // K(0..P-1), then per iteration j: [Q(rb+1) if chunk 1] K(j+P); so the
      // copies still allowed in flight are those of iterations it-P+1..it-1.
      if constexpr (S == 4) {
        const int newer_k = (it + 1 < n_it) + (it + 2 < n_it);
        const bool newer_q = (ch == 2 || ch == 3) && rb + 1 < rb1;
        if (newer_q) {
          if (newer_k == 2) wait_vm<2 * kL + kQL>();
          else if (newer_k == 1) wait_vm<kL + kQL>();
          else wait_vm<kQL>();
        } else {
          if (newer_k == 2) wait_vm<2 * kL>();
          else if (newer_k == 1) wait_vm<kL>();
          else wait_vm<0>();
        }
      } else {
        wait_vm<0>();
      }
      lds_barrier();
      if (ch == 0) {
#pragma unroll
        for (int rt = 0; rt < 2; ++rt)
#pragma unroll
          for (int ks = 0; ks < KC; ++ks) qa[rt].v[ks] = *(const uint4*)(qbuf + qoff[ks] + rt * 16 * C::kRowBytes);
        if constexpr (!kEarlyQ) {
          // every wave holds its queries before the buffer is refilled
          lds_barrier();
          if (rb + 1 < rb1) load_queries(rb + 1);
        }
      }
      if constexpr (kEarlyQ) {
        if (ch == 1 && rb + 1 < rb1) load_queries(rb + 1);
      }
      if constexpr (P > 0) {
        if (it + P < n_it) load_keys((ch + P) % NCH, (ch + P) % S);
      }
      // the two 16-row tiles share each key operand
      const char* sbase = kbuf + (ch % S) * C::kStageBytes;
#pragma unroll
      for (int ti = 0; ti < TPS; ++ti) {
        Op kb;
#pragma unroll
        for (int ks = 0; ks < KC; ++ks) kb.v[ks] = *(const uint4*)(sbase + koff[ks] + ti * 16 * C::kRowBytes);
#pragma unroll
        for (int rt = 0; rt < 2; ++rt)
          acc[rt][ch * TPS + ti] = dot_tile<DT, D>(qa[rt], kb, floatx4{0.f, 0.f, 0.f, 0.f});
      }
      if constexpr (P == 0) {
        // single stage: every wave is done with it before the next copy
        if (it + 1 < n_it) {
          lds_barrier();
          load_keys((ch + 1) % NCH, 0);
        }
      }
    }

    // ---- softmax over all keys of each row, then column sums ----
    // keys past N take no part (only waves whose keys run past N look)
    if ((cg * NT + NT) * 16 > N) {
#pragma unroll
      for (int i = 0; i < NT; ++i)
        if ((cg * NT + i) * 16 + li >= N) {
#pragma unroll
          for (int rt = 0; rt < 2; ++rt) acc[rt][i] = floatx4{kNegInf, kNegInf, kNegInf, kNegInf};
        }
    }
    float M[2][4];
#pragma unroll
    for (int rt = 0; rt < 2; ++rt)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float v = acc[rt][0][q];
#pragma unroll
        for (int i = 1; i < NT; ++i) v = fmaxf(v, acc[rt][i][q]);
        M[rt][q] = max16(v);
      }
    if constexpr (CG > 1) {
      if (li == 0) {
#pragma unroll
        for (int rt = 0; rt < 2; ++rt)
#pragma unroll
          for (int q = 0; q < 4; ++q) red_max[rg][cg][rt * 16 + gq * 4 + q] = M[rt][q];
      }
      lds_barrier();
#pragma unroll
      for (int rt = 0; rt < 2; ++rt)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          float v = red_max[rg][0][rt * 16 + gq * 4 + q];
#pragma unroll
          for (int o = 1; o < CG; ++o) v = fmaxf(v, red_max[rg][o][rt * 16 + gq * 4 + q]);
          M[rt][q] = v;
        }
    }
    float L[2][4];
#pragma unroll
    for (int rt = 0; rt < 2; ++rt)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float mc = M[rt][q] * c;
        float sum = 0.f;
#pragma unroll
        for (int i = 0; i < NT; ++i) {
          const float e = __builtin_amdgcn_exp2f(acc[rt][i][q] * c - mc);
          acc[rt][i][q] = e;
          sum += e;
        }
        L[rt][q] = sum16(sum);
      }
    if constexpr (CG > 1) {
      if (li == 0) {
#pragma unroll
        for (int rt = 0; rt < 2; ++rt)
#pragma unroll
          for (int q = 0; q < 4; ++q) red_sum[rg][cg][rt * 16 + gq * 4 + q] = L[rt][q];
      }
      lds_barrier();
#pragma unroll
      for (int rt = 0; rt < 2; ++rt)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          float v = red_sum[rg][0][rt * 16 + gq * 4 + q];
#pragma unroll
          for (int o = 1; o < CG; ++o) v += red_sum[rg][o][rt * 16 + gq * 4 + q];
          L[rt][q] = v;
        }
    }
    // softmax weight of each of this lane's eight rows (rows past R: none)
    float wr[2][4];
    const int row0 = rb * C::kRows + rg * 32;
#pragma unroll
    for (int rt = 0; rt < 2; ++rt)
#pragma unroll
      for (int q = 0; q < 4; ++q)
        wr[rt][q] = (row0 + rt * 16 + gq * 4 + q < R) ? __builtin_amdgcn_rcpf(L[rt][q]) : 0.f;
    // column sums: this lane's eight rows, then the four lane groups (fixed
    // order: (g0 + g1) + (g2 + g3)); lane group 0 adds the result to LDS
    float* my_part = &part[rg][cg * NT * 16 + li];
#pragma unroll
    for (int i = 0; i < NT; ++i) {
      float v = acc[0][i][0] * wr[0][0];
      v = fmaf(acc[0][i][1], wr[0][1], v);
      v = fmaf(acc[0][i][2], wr[0][2], v);
      v = fmaf(acc[0][i][3], wr[0][3], v);
      v = fmaf(acc[1][i][0], wr[1][0], v);
      v = fmaf(acc[1][i][1], wr[1][1], v);
      v = fmaf(acc[1][i][2], wr[1][2], v);
      v = fmaf(acc[1][i][3], wr[1][3], v);
      v += __shfl_xor(v, 16, 64);
      v += __shfl_xor(v, 32, 64);
      if (gq == 0) my_part[i * 16] += v;
    }
  }

  // fixed-order reduction over the row groups
  lds_barrier();
  for (int j = tid; j < N; j += kScoreThreads) {
    float v = part[0][j];
#pragma unroll
    for (int p = 1; p < RG; ++p) v += part[p][j];
    out[j] = v;
  }
  if (a.n_splits == 1) return;

  // The last split of the unit to finish adds all splits' partial sums in
  // split order (the order does not depend on which split finishes last).
  __shared__ uint32_t ticket;
  __threadfence();
  __syncthreads();
  if (tid == 0) ticket = atomicAdd(&a.done[u], 1u);
  __syncthreads();
  if (ticket != (uint32_t)a.n_splits - 1) return;
  __threadfence();
  const float* slabs = a.partials + u * a.n_splits * (int64_t)N;
  float* sc = a.scores + u * (int64_t)N;
  for (int j = tid; j < N; j += kScoreThreads) {
    float v = slabs[j];
    for (int p = 1; p < a.n_splits; ++p) v += slabs[(int64_t)p * N + j];
    sc[j] = v;
  }
  if (tid == 0) a.done[u] = 0;   // ready for the next call
}

template <int DT, int D, int NT, int CG>
hipError_t launch_cfg(const ScoreArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL((score_kernel<DT, D, NT, CG>), dim3((unsigned)a.n_blocks), dim3(kScoreThreads), 0,
                     stream, a);
  return hipGetLastError();
}

template <int DT, int D>
hipError_t launch_d(const ScoreArgs& a, const ScorePlan& sp, hipStream_t stream) {
  if constexpr (DT == KARA_F32 && D == 128) {
    // fp32 with 512-byte rows: at most 512 keys, at least two column groups
    if (sp.nt == 8) return launch_cfg<DT, D, 8, 2>(a, stream);
    return launch_cfg<DT, D, 16, 2>(a, stream);
  } else {
    if (sp.nt == 8) return launch_cfg<DT, D, 8, 1>(a, stream);
    switch (sp.cg) {
      case 1: return launch_cfg<DT, D, 16, 1>(a, stream);
      case 2: return launch_cfg<DT, D, 16, 2>(a, stream);
      case 4: return launch_cfg<DT, D, 16, 4>(a, stream);
      default:
        if constexpr (DT == KARA_BF16) return launch_cfg<DT, D, 16, 8>(a, stream);
        return hipErrorInvalidValue;
    }
  }
}

}  // namespace

ScorePlan plan_score(const Geom& g, int64_t n_units) {
  (void)n_units;
  ScorePlan sp{};
  const int tiles = (g.N + 15) / 16;
  if (g.dtype == KARA_F32 && g.d == 128) {
    sp.cg = 2;
    sp.nt = tiles <= 16 ? 8 : 16;
  } else if (tiles <= 8) {
    sp.cg = 1;
    sp.nt = 8;
  } else {
    sp.nt = 16;
    sp.cg = tiles <= 16 ? 1 : tiles <= 32 ? 2 : tiles <= 64 ? 4 : 8;
  }
  sp.rg = kScoreWaves / sp.cg;
  sp.n_cols = sp.cg * sp.nt * 16;
  const int64_t rows = (int64_t)g.G * g.W;
  sp.n_rb = (int)((rows + 32 * sp.rg - 1) / (32 * sp.rg));
  // 32 row splits per unit: the 32 CUs of one XCD work on the same unit at
  // once, so its keys are read from that XCD's L2
  sp.n_splits = sp.n_rb < 32 ? sp.n_rb : 32;
  return sp;
}


hipError_t launch_score(const Geom& g, const ScorePlan& sp, int n_layers, const void* q,
                        const PoolPtrs& k_pools, const int32_t* trig, const int32_t* block_table,
                        const int32_t* win_start, const int32_t* status, float* partials,
                        float* scores, uint32_t* done, hipStream_t stream) {
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
  a.done = done;
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
