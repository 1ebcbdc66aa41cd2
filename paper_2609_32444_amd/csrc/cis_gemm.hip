// Dense products of the LM-head form (gfx950 MFMA): C = alpha * A * B^T (+ C), both operands
// bf16 and K-contiguous, float32 accumulation; and a tiled transpose that converts to bf16. Used
// for the logits of a row chunk (hidden * W^T), the gradient with respect to the hidden states
// (G * W) and the gradient of the head weight (G^T * hidden).
//
// Tiling: a workgroup of 8 waves owns a 256 x 256 tile of C; each wave owns 128 x 64 as 8 x 4
// blocks of v_mfma_f32_16x16x32_bf16 (which sustains about 98% of the matrix cores' peak on this
// part against about 86% for the 32x32x16 form). K advances 64 at a time through a ring of two
// LDS slabs that the buffer unit fills directly (buffer loads that write LDS: no registers
// staged, no LDS store instructions): the next slab is requested right after the barrier that
// frees its buffer and is multiplied one slab later. Within a slab the fragments of the second
// 32-step are read while the first is multiplied.
//
// LDS slab: 512 rows (A's 256, then B's) of 64 bf16 = 128 bytes, unpadded because one
// buffer->LDS instruction fills 1 KiB contiguously. The 16-byte chunk c of row r is stored at
// chunk c ^ (r & 7): a fragment read then touches 16 rows at one logical chunk without bank
// conflicts (measured with the LDS counters; without the swizzle every read is a 4-way
// conflict).
//
// MFMA operand layout (16x16x32): lane l supplies X[i = l % 16][k = 8 (l / 16) + j], j = 0..7,
// for both operands, and accumulator register r of lane l is the product's element
// (i = 4 (l / 16) + r, i' = l % 16) (checked on the device against an exact integer product).
// The B fragment is passed as the first operand, so a lane's four registers hold four
// consecutive columns of one row of C and the epilogue stores 16 bytes at a time.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "cis_gemm.h"

namespace cis {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kRsrcWord3 = 0x00020000;  // raw buffer, 32-bit data format

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, (int)bytes, kRsrcWord3);
}

// Bytes of an R x K row-major matrix (row stride ld elements of `es` bytes) from row r0 on,
// clamped to the 32-bit range of a buffer resource (offsets used stay below it).
__device__ __forceinline__ uint32_t span_bytes(int64_t R, int64_t r0, int64_t K, int64_t ld,
                                               int es) {
  if (r0 >= R) return 0;
  const int64_t b = ((R - r0 - 1) * ld + K) * es;
  return b > 0xFFFFFFFFll ? 0xFFFFFFFFu : (uint32_t)b;
}

// Logical work unit -> (split, tile). Logically the smaller operand's tile index runs fastest:
// the larger operand's panel is then shared by consecutive units and streamed from HBM about
// once.
template <int BM, int BN>
__device__ __forceinline__ void unit_tile(const GemmArgs& g, int64_t lin, int64_t& tm,
                                          int64_t& tn, int64_t& split) {
  const int64_t mt = (g.M + BM - 1) / BM, nt = (g.N + BN - 1) / BN;
  split = lin / (mt * nt);
  const int64_t t = lin % (mt * nt);
  if (g.m_fastest) {
    tm = t % mt;
    tn = t / mt;
  } else {
    tn = t % nt;
    tm = t / nt;
  }
}

// Consecutive workgroup ids go to the 8 XCDs in turn and each XCD has an L2 of its own, so XCD
// x is given the contiguous run [xcd_first(x), xcd_first(x) + xcd_count(x)) of the n units.
__device__ __forceinline__ int64_t xcd_count(int64_t n, int x) {
  return n / kGemmQueues + (x < n % kGemmQueues ? 1 : 0);
}
__device__ __forceinline__ int64_t xcd_first(int64_t n, int x) {
  const int64_t per = n / kGemmQueues, rem = n % kGemmQueues;
  return x < rem ? x * (per + 1) : rem * (per + 1) + (x - rem) * per;
}

// One workgroup per unit: workgroup id -> unit.
__device__ __forceinline__ int64_t unit_of_workgroup() {
  const int64_t nwg = (int64_t)gridDim.x, id = blockIdx.x;
  return xcd_first(nwg, (int)(id % kGemmQueues)) + id / kGemmQueues;
}

// Work queues (thread 0 of a persistent workgroup): the next unit of the home XCD's run, then
// of the other XCDs' runs in turn; -1 when all are taken. `tried` counts the runs found empty
// (kept across calls), so a workgroup makes at most kGemmQueues failed attempts in all.
__device__ __forceinline__ int64_t next_unit(const GemmArgs& g, int home, int& tried) {
  while (tried < kGemmQueues) {
    const int x = (home + tried) % kGemmQueues;
    const int i = atomicAdd(&g.queue[x], 1);
    if (i < xcd_count(g.units, x)) return xcd_first(g.units, x) + i;
    ++tried;
  }
  return -1;
}

// Waits until at most N of this wave's buffer operations are outstanding (gfx9 encoding: vmcnt
// in bits 3:0 and 15:14; expcnt and lgkmcnt left at their maxima).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x0F70);
}

// 16-byte buffer load that writes LDS: lane l stores at lds_wave + 16 l bytes (lds_wave is the
// same for the whole wave). Counted by vmcnt. (The builtin sits in a device function of its own:
// inside a lambda it loses its host-side declaration.)
__device__ __forceinline__ void load_lds16(__amdgpu_buffer_rsrc_t r, __bf16* lds_wave,
                                           uint32_t voff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)lds_wave,
                                           16, voff, 0, 0, 0);
}

// Workgroup barrier after this wave's LDS operations. __syncthreads() would also wait for every
// buffer->LDS load still in flight; the slab waits are explicit (wait_vmcnt) instead. The memory
// clobber keeps the compiler from moving LDS accesses across it.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

constexpr int kWaves = (kGemmTile / kGemmWaveM) * (kGemmTile / kGemmWaveN);  // 8
constexpr int kThreads = kWaves * 64;
constexpr int kTm = kGemmWaveM / 16, kTn = kGemmWaveN / 16;                 // 8 x 4 blocks
constexpr int kSlab = 2 * kGemmTile * kGemmBK;       // bf16 per LDS slab (A rows, B rows)
constexpr int kLoads = 2 * kGemmTile * (kGemmBK / 8) / kThreads;  // 16-byte units per lane
constexpr int kALoads = kLoads / 2;                  // the first half fill A's rows
static_assert(kGemmBK == 64 && kThreads * 8 / 64 * kALoads == kGemmTile,
              "a slab row is 8 chunks; each load covers 64 rows");

// One slab of MFMAs for a wave's kTm x kTn blocks: two 32-steps, the fragments of the second
// read from LDS while the first is multiplied. fa(i, s) / fb(j, s) give fragment addresses.
//   SPLIT = false: each step's 12 reads have landed before the next step's are issued (the LDS
//     counter tracks at most 15 reads; with 24 in flight the compiler would wait for all of
//     them before the first MFMA).
//   SPLIT = true: the first step's fragments are read B first, then A row by row, and each row
//     of MFMAs waits only for its own fragments (the compiler's counted LDS waits), so the
//     first MFMAs after the slab barrier start once five reads have landed. The second step's
//     12 reads are issued after row kSplitRow of the first step, which keeps every wait within
//     the counter's 15.
constexpr int kSplitRow = 4;
template <bool SPLIT, class FA, class FB>
__device__ __forceinline__ void mfma_slab(f32x4 (&acc)[kTm][kTn], FA fa, FB fb) {
  static_assert(kGemmBK == 64, "two 32-steps per slab");
  static_assert((kTm - 1 - kSplitRow) + kTm + kTn <= 15, "waits stay within the LDS counter");
  bf16x8 a0[kTm], b0[kTn], a1[kTm], b1[kTn];
  auto row = [&](int i, const bf16x8(&a)[kTm], const bf16x8(&b)[kTn]) {
#pragma unroll
    for (int j = 0; j < kTn; ++j)
      acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(b[j], a[i], acc[i][j], 0, 0, 0);
  };
  // SPLIT reads B first (every row of MFMAs needs all of B); otherwise A first
  auto read = [&](int s, bf16x8(&a)[kTm], bf16x8(&b)[kTn]) {
    if constexpr (SPLIT) {
#pragma unroll
      for (int j = 0; j < kTn; ++j) b[j] = *(const bf16x8*)fb(j, s);
    }
#pragma unroll
    for (int i = 0; i < kTm; ++i) a[i] = *(const bf16x8*)fa(i, s);
    if constexpr (!SPLIT) {
#pragma unroll
      for (int j = 0; j < kTn; ++j) b[j] = *(const bf16x8*)fb(j, s);
    }
  };
  read(0, a0, b0);
  if constexpr (SPLIT) {
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < kSplitRow; ++i) {
      row(i, a0, b0);
      __builtin_amdgcn_sched_barrier(0);
    }
    read(1, a1, b1);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = kSplitRow; i < kTm; ++i) {
      row(i, a0, b0);
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int i = 0; i < kTm; ++i) {
      row(i, a1, b1);
      __builtin_amdgcn_sched_barrier(0);
    }
  } else {
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0); vmcnt and expcnt at their maxima
    __builtin_amdgcn_sched_barrier(0);
    read(1, a1, b1);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < kTm; ++i) row(i, a0, b0);
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_waitcnt(0xC07F);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < kTm; ++i) row(i, a1, b1);
    __builtin_amdgcn_sched_barrier(0);
  }
}

// Epilogue of a tile: lane holds C[m][n .. n + 3] for m = m-block row + lane % 16,
// n = n-block column + 4 (lane / 16); 16-byte stores where the row allows them.
template <bool BETA>
__device__ __forceinline__ void store_tile(const GemmArgs& g, const f32x4 (&acc)[kTm][kTn],
                                           int64_t m0, int64_t n0, int64_t split) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / (kGemmTile / kGemmWaveN), wn = wave % (kGemmTile / kGemmWaveN);
  const int fr = lane & 15, fq = lane >> 4;
  float* Cp = g.C + split * g.c_split_stride;
  const bool vec = g.c_vec;
#pragma unroll
  for (int i = 0; i < kTm; ++i) {
    const int64_t m = m0 + wm * kGemmWaveM + i * 16 + fr;
    if (m >= g.M) continue;
    float* crow = Cp + m * g.ldc;
#pragma unroll
    for (int j = 0; j < kTn; ++j) {
      const int64_t n = n0 + wn * kGemmWaveN + j * 16 + 4 * fq;
      f32x4 v = acc[i][j] * g.alpha;
      if (vec && n + 3 < g.N) {
        if (BETA) v += *(const f32x4*)(crow + n);
        *(f32x4*)(crow + n) = v;
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (n + e < g.N) crow[n + e] = BETA ? v[e] + crow[n + e] : v[e];
      }
    }
  }
}

constexpr float kLog2e = 1.44269504088896340736f;
constexpr float kMinRef = -0x1p127f;  // floor of a running max: keeps max * log2(e) finite

// Row-loss epilogue kEpiLse of a logits tile (rows m0.., vocabulary columns n0.., tile column
// tn): per row and wave, the max over the wave's 64 columns and the sum of exp(z - max) leaving
// out the sampled column, one pair in part[row * ldp + 4 tn + wn] (the four lanes of a row in a
// wave combine by shuffles; the combine kernel folds a row's pairs in this order). The lane
// holding the sampled column stores its logit in zy[row].
template <bool FULL>
__device__ __forceinline__ void lse_tile(const GemmArgs& g, const f32x4 (&acc)[kTm][kTn],
                                         int64_t m0, int64_t n0, int64_t tn,
                                         const int (&ep_y)[kGemmTile]) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / (kGemmTile / kGemmWaveN), wn = wave % (kGemmTile / kGemmWaveN);
  const int fr = lane & 15, fq = lane >> 4;
  const int N = (int)g.N;                                   // V <= 2^22
  const int nb = (int)n0 + wn * kGemmWaveN + 4 * fq;         // this lane's first column
  const int64_t pidx = tn * (kGemmTile / kGemmWaveN) + wn;
#pragma unroll
  for (int i = 0; i < kTm; ++i) {
    const int64_t m = m0 + wm * kGemmWaveM + i * 16 + fr;
    const bool row_ok = m < g.M;
    const int y = ep_y[wm * kGemmWaveM + i * 16 + fr];
    float mx = kMinRef;
#pragma unroll
    for (int j = 0; j < kTn; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (FULL || nb + j * 16 + e < N) mx = fmaxf(mx, acc[i][j][e]);
    mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    const float mb = mx * kLog2e;
    const int dy = y - nb;  // the sampled column in this lane's 4 x 4 columns?
    const bool has_y = dy >= 0 && dy < kTn * 16 && (dy & 15) < 4;
    float sm = 0.f;
    if (has_y) {  // the one lane of the row that holds y leaves it out element by element
#pragma unroll
      for (int j = 0; j < kTn; ++j)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int n = nb + j * 16 + e;
          const float x = __builtin_amdgcn_exp2f(__builtin_fmaf(acc[i][j][e], kLog2e, -mb));
          sm += ((FULL || n < N) && n != y) ? x : 0.f;
        }
    } else {
#pragma unroll
      for (int j = 0; j < kTn; ++j)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float x = __builtin_amdgcn_exp2f(__builtin_fmaf(acc[i][j][e], kLog2e, -mb));
          sm += (FULL || nb + j * 16 + e < N) ? x : 0.f;
        }
    }
    sm += __shfl_xor(sm, 16, 64);
    sm += __shfl_xor(sm, 32, 64);
    if (row_ok && has_y) {
#pragma unroll
      for (int j = 0; j < kTn; ++j)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (dy == j * 16 + e) g.e.zy[m] = acc[i][j][e];
    }
    if (row_ok && fq == 0) g.e.part[m * g.e.ldp + pidx] = float2{mx, sm};
  }
}

// dL/dz of logit z in column n of a row with parameters p: -coef exp(z - lse), evaluated as
// +-exp2(z log2(e) - b2), and coef (1 - p) at the sampled column; 0 for a row without gradient.
__device__ __forceinline__ float grad_value(const GradParams& p, float z, int64_t n) {
  const float x = __builtin_amdgcn_exp2f(__builtin_fmaf(z, kLog2e, -p.b2));
  return p.y < 0 ? 0.f : ((n == p.y) ? p.gy : (p.neg ? -x : x));
}

// Row-loss epilogue kEpiGrad: grad_value of every logit of the tile, rounded to bf16 (nearest
// even) into G.
__device__ __forceinline__ void grad_tile(const GemmArgs& g, const f32x4 (&acc)[kTm][kTn],
                                          int64_t m0, int64_t n0) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / (kGemmTile / kGemmWaveN), wn = wave % (kGemmTile / kGemmWaveN);
  const int fr = lane & 15, fq = lane >> 4;
  GradParams ps[kTm];  // every row's parameters requested before the first is used
#pragma unroll
  for (int i = 0; i < kTm; ++i) {
    const int64_t m = m0 + wm * kGemmWaveM + i * 16 + fr;
    ps[i] = m < g.M ? g.e.gp[m] : GradParams{INFINITY, 0, 0.f, -1};
  }
#pragma unroll
  for (int i = 0; i < kTm; ++i) {
    const int64_t m = m0 + wm * kGemmWaveM + i * 16 + fr;
    if (m >= g.M) continue;
    const GradParams p = ps[i];
    __bf16* grow = g.e.G + m * g.e.ldg;
#pragma unroll
    for (int j = 0; j < kTn; ++j) {
      const int64_t n = n0 + wn * kGemmWaveN + j * 16 + 4 * fq;
      float v[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = grad_value(p, acc[i][j][e], n + e);
      const bf16x4 o = {(__bf16)v[0], (__bf16)v[1], (__bf16)v[2], (__bf16)v[3]};
      if (n + 3 < g.N) {
        *(bf16x4*)(grow + n) = o;
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (n + e < g.N) grow[n + e] = o[e];
      }
    }
  }
}

// The (tm, tn) tile of C over split `split` of the contraction, by the whole workgroup. The
// caller puts a barrier between two tiles of one workgroup (the last slab's reads must end
// before the next tile refills LDS; with an empty K range there is no barrier inside).
// The sampled ids of the tile's rows for kEpiLse, loaded into LDS before the contraction (the
// K loop's barriers make them visible; reading them in the epilogue would put a load latency
// after every tile).
struct EpiRows {
  int y[kGemmTile];            // sampled id, or -1 when outside [0, N)
};

template <bool BETA, int EPI, bool SPLIT>
__device__ __forceinline__ void gemm_tile(const GemmArgs& g, int64_t tm, int64_t tn,
                                          int64_t split, __bf16 (&lds)[2 * kSlab], EpiRows& er) {
  constexpr int BM = kGemmTile, BN = kGemmTile, BK = kGemmBK;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / (BN / kGemmWaveN), wn = wave % (BN / kGemmWaveN);
  const int64_t m0 = tm * BM, n0 = tn * BN;
  const int64_t kbeg = split * g.k_split;
  const int64_t kend = kbeg + g.k_split < g.K ? kbeg + g.k_split : g.K;
  const __bf16* A = static_cast<const __bf16*>(g.A) + m0 * g.lda;
  const __bf16* B = static_cast<const __bf16*>(g.B) + n0 * g.ldb;
  const __amdgpu_buffer_rsrc_t ra = make_rsrc(A, span_bytes(g.M, m0, g.K, g.lda, 2));
  const __amdgpu_buffer_rsrc_t rb = make_rsrc(B, span_bytes(g.N, n0, g.K, g.ldb, 2));

  // Load j of a wave fills the slab's 16-byte units (8 j + wave) 64 + lane: slab row
  // r = 64 j + 8 wave + lane / 8 (A rows, then B rows from j = kALoads on), stored chunk
  // lane % 8, holding logical chunk (lane % 8) ^ (r & 7) = (lane % 8) ^ (lane / 8 % 8).
  // Rows past M or N read as zero through the buffer range check.
  const int lchunk = (lane & 7) ^ ((lane >> 3) & 7);
  const int64_t r0 = wave * 8 + (lane >> 3);
  const uint32_t offa = (uint32_t)((r0 * g.lda + lchunk * 8) * 2);
  const uint32_t offb = (uint32_t)((r0 * g.ldb + lchunk * 8) * 2);
  const uint32_t stepa = (uint32_t)(64 * g.lda * 2), stepb = (uint32_t)(64 * g.ldb * 2);
  auto off = [&](int j) { return j < kALoads ? offa + j * stepa : offb + (j - kALoads) * stepb; };
  const int64_t nk = kend > kbeg ? (kend - kbeg + BK - 1) / BK : 0;
  auto issue = [&](int64_t kt) {
    __bf16* st = lds + (int)(kt & 1) * kSlab;
    const int64_t k0 = kbeg + kt * BK;
    const uint32_t ko = (uint32_t)(k0 * 2);
    if (k0 + BK <= kend) {
#pragma unroll
      for (int j = 0; j < kLoads; ++j)
        load_lds16(j < kALoads ? ra : rb, st + (j * kWaves + wave) * 512, off(j) + ko);
    } else {
      // the last slab of the range goes through registers: zero past kend, and a vector that
      // straddles kend is read element by element (a 16-byte buffer load that is partly
      // outside the resource returns zeros)
#pragma unroll
      for (int j = 0; j < kLoads; ++j) {
        const __amdgpu_buffer_rsrc_t rs = j < kALoads ? ra : rb;
        const uint32_t o = off(j) + ko;
        const int64_t k = k0 + lchunk * 8;
        bf16x8 e{};
        if (k + 8 <= kend) {
          e = __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(rs, o, 0, 0));
        } else if (k < kend) {
          for (int i = 0; i < 8; ++i)
            if (k + i < kend)
              e[i] = __builtin_bit_cast(
                  __bf16, (unsigned short)__builtin_amdgcn_raw_buffer_load_b16(rs, o + 2 * i, 0, 0));
        }
        *(bf16x8*)(st + ((j * kWaves + wave) * 64 + lane) * 8) = e;
      }
    }
  };

  f32x4 acc[kTm][kTn];
#pragma unroll
  for (int i = 0; i < kTm; ++i)
#pragma unroll
    for (int j = 0; j < kTn; ++j) acc[i][j] = f32x4{};

  // the epilogue's per-row inputs: requested now, stored to LDS once the first slab has landed
  const int64_t mrow = m0 + tid;
  constexpr bool kLse = EPI == kEpiLse || EPI == kEpiLseStore;
  const bool erow = kLse && tid < kGemmTile && mrow < g.M;
  int64_t ey = -1;
  if (erow) ey = g.e.ids[mrow];
  // a fragment row is a multiple of 16 plus lane % 16, so its swizzle is lane & 7
  const int fr = lane & 15, fq = lane >> 4, sw = lane & 7;
  if (nk > 0) issue(0);
  // (the ids were requested before the first slab, so this waits for them alone; the first
  // slab's barrier makes them visible, and a loop free of first-iteration code keeps the
  // compiler from peeling it into a copy that spills)
  if (kLse && tid < kGemmTile) er.y[tid] = (ey >= 0 && ey < g.N) ? (int)ey : -1;
  for (int64_t kt = 0; kt < nk; ++kt) {
    wait_vmcnt<0>();  // this wave's part of slab kt is in LDS
    lds_barrier();    // every wave's is, and every wave is done with slab kt - 1's buffer
    if (kt + 1 < nk) issue(kt + 1);
    const __bf16* st = lds + (int)(kt & 1) * kSlab;
    const __bf16* la = st + (wm * kGemmWaveM + fr) * BK;
    const __bf16* lb = st + (BM + wn * kGemmWaveN + fr) * BK;
    mfma_slab<SPLIT>(acc, [&](int i, int s) { return la + i * 16 * BK + ((4 * s + fq) ^ sw) * 8; },
              [&](int j, int s) { return lb + j * 16 * BK + ((4 * s + fq) ^ sw) * 8; });
  }

  if (kLse) {
    if (n0 + kGemmTile <= g.N)
      lse_tile<true>(g, acc, m0, n0, tn, er.y);
    else
      lse_tile<false>(g, acc, m0, n0, tn, er.y);
  }
  if (EPI == kEpiGrad)
    grad_tile(g, acc, m0, n0);
  else if (EPI == kEpiStore || EPI == kEpiLseStore)
    store_tile<BETA>(g, acc, m0, n0, split);
}

template <bool BETA, bool QUEUED, int EPI = kEpiStore>
__global__ __launch_bounds__(kThreads) void gemm_bf16_kernel(const GemmArgs g) {
  __shared__ __attribute__((aligned(16))) __bf16 lds[2 * kSlab];
  __shared__ int64_t unit;
  __shared__ EpiRows er;
  const int home = (int)(blockIdx.x % kGemmQueues);
  int tried = 0;
  // one unit per workgroup, or (queued) units until every queue is empty: all threads read the
  // same `unit` and leave together
  for (int64_t u = QUEUED ? -1 : unit_of_workgroup();;) {
    if (QUEUED) {
      // every wave has read the previous `unit` and is done with the previous tile's LDS (a
      // tile with an empty K range has no barrier of its own)
      __syncthreads();
      if (threadIdx.x == 0) unit = next_unit(g, home, tried);
      __syncthreads();
      u = unit;
    }
    if (u < 0) break;
    int64_t tm, tn, split;
    unit_tile<kGemmTile, kGemmTile>(g, u, tm, tn, split);
    // The split fragment reads where the compiler keeps the K loop free of full vmcnt waits:
    // in the other forms it placed a vmcnt(0) before the first step's A reads, which also
    // waits for the next slab's loads.
    constexpr bool kSplitReads = EPI == kEpiLse || (EPI == kEpiLseStore && QUEUED);
    gemm_tile<BETA, EPI, kSplitReads>(g, tm, tn, split, lds, er);
    if (!QUEUED) break;
  }
}

// C = alpha * sum_s P[s] (+ C): the split-K partials summed in split order.
struct ReduceArgs {
  const float* P;
  float* C;
  int64_t M, N, ldc, split_stride;
  int32_t splits;
  float alpha;
  bool beta;
};

__global__ __launch_bounds__(256) void splitk_reduce_kernel(const ReduceArgs r) {
  const int64_t total = r.M * r.N;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * 256) {
    const int64_t m = i / r.N, n = i % r.N;
    float s = 0.f;
    for (int k = 0; k < r.splits; ++k) s += r.P[k * r.split_stride + m * r.N + n];
    float* c = r.C + m * r.ldc + n;
    *c = r.beta ? s * r.alpha + *c : s * r.alpha;
  }
}

// out[c][r] = bf16(f(in[r][c])) for an R x C matrix (row strides ldi, ldo), and optionally
// out_n[r][c] = bf16(f(in[r][c])) (row stride ldn): 64 x 64 tiles through LDS, every global
// access row-contiguous (four elements per thread). GRAD: f is grad_value with row r's
// GradParams (the loss gradient of stored float32 logits), else the identity.
template <class TI, bool GRAD = false>
__global__ __launch_bounds__(256) void transpose_kernel(const TransposeArgs t) {
  __shared__ float tile[64][65];
  const TI* in = static_cast<const TI*>(t.in);
  __bf16* out = static_cast<__bf16*>(t.out);
  __bf16* outn = static_cast<__bf16*>(t.out_n);
  const int64_t ct = (t.C + 63) / 64;
  const int64_t r0 = (int64_t)(blockIdx.x / ct) * 64, c0 = (int64_t)(blockIdx.x % ct) * 64;
  const int q = threadIdx.x & 15, p = threadIdx.x >> 4;  // 16 quads per row, 16 rows per pass
#pragma unroll
  for (int pass = 0; pass < 4; ++pass) {
    const int lr = p + 16 * pass;
    const int64_t r = r0 + lr, c = c0 + 4 * q;
    float v[4] = {0.f, 0.f, 0.f, 0.f};
    if (r < t.R) {
      const TI* src = in + r * t.ldi + c;
      if (c + 4 <= t.C) {
        if constexpr (sizeof(TI) == 4) {
          const f32x4 x = *(const f32x4*)src;
          v[0] = x[0], v[1] = x[1], v[2] = x[2], v[3] = x[3];
        } else {
          const bf16x4 x = *(const bf16x4*)src;
          v[0] = (float)x[0], v[1] = (float)x[1], v[2] = (float)x[2], v[3] = (float)x[3];
        }
      } else {
        for (int e = 0; e < 4; ++e)
          if (c + e < t.C) v[e] = (float)src[e];
      }
      if constexpr (GRAD) {
        const GradParams gp = t.gp[r];
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = grad_value(gp, v[e], c + e);
      }
      if (outn) {
        __bf16* dst = outn + r * t.ldn + c;
        if (c + 4 <= t.C) {
          *(bf16x4*)dst = bf16x4{(__bf16)v[0], (__bf16)v[1], (__bf16)v[2], (__bf16)v[3]};
        } else {
          for (int e = 0; e < 4; ++e)
            if (c + e < t.C) dst[e] = (__bf16)v[e];
        }
      }
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) tile[lr][4 * q + e] = v[e];
  }
  __syncthreads();
#pragma unroll
  for (int pass = 0; pass < 4; ++pass) {
    const int lc = p + 16 * pass;
    const int64_t c = c0 + lc, r = r0 + 4 * q;
    if (c >= t.C) continue;
    __bf16* dst = out + c * t.ldo + r;
    const bf16x4 x = {(__bf16)tile[4 * q][lc], (__bf16)tile[4 * q + 1][lc],
                      (__bf16)tile[4 * q + 2][lc], (__bf16)tile[4 * q + 3][lc]};
    if (r + 4 <= t.R) {
      *(bf16x4*)dst = x;
    } else {
      for (int e = 0; e < 4; ++e)
        if (r + e < t.R) dst[e] = x[e];
    }
  }
}

// Launch over `splits` splits; with g.queue, one workgroup per CU (the LDS ring allows one)
// works through the queues.
hipError_t launch_tiles(GemmArgs g, bool beta, int splits, int num_cu, hipStream_t stream) {
  const int64_t mt = (g.M + kGemmTile - 1) / kGemmTile, nt = (g.N + kGemmTile - 1) / kGemmTile;
  g.units = mt * nt * splits;
  const int64_t grid = g.queue && num_cu < g.units ? num_cu : g.units;
  const void* fn = g.queue ? (beta ? (const void*)&gemm_bf16_kernel<true, true>
                                   : (const void*)&gemm_bf16_kernel<false, true>)
                           : (beta ? (const void*)&gemm_bf16_kernel<true, false>
                                   : (const void*)&gemm_bf16_kernel<false, false>);
  void* args[] = {&g};
  return hipLaunchKernel(fn, dim3((unsigned)grid), dim3(kThreads), args, 0, stream);
}

__global__ __launch_bounds__(kGemmQueues) void zero_queue_kernel(int* q) { q[threadIdx.x] = 0; }

}  // namespace

hipError_t launch_gemm_epi(GemmArgs g, int* queue, int num_cu, hipStream_t stream) {
  if (g.M <= 0 || g.N <= 0) return hipSuccess;
  g.m_fastest = g.M <= g.N;
  g.k_split = g.K > 0 ? g.K : 1;
  g.c_split_stride = 0;
  g.c_vec = g.epi == kEpiLseStore && ((uintptr_t)g.C % 16 == 0) && g.ldc % 4 == 0;
  const int64_t mt = (g.M + kGemmTile - 1) / kGemmTile, nt = (g.N + kGemmTile - 1) / kGemmTile;
  g.units = mt * nt;
  g.queue = g.units > num_cu ? queue : nullptr;
  if (g.queue) {
    void* zargs[] = {&g.queue};
    if (hipError_t e = hipLaunchKernel((const void*)&zero_queue_kernel, dim3(1),
                                       dim3(kGemmQueues), zargs, 0, stream))
      return e;
  }
  const int64_t grid = g.queue ? num_cu : g.units;
  const void* fn;
  switch (g.epi) {
    case kEpiLse:
      fn = g.queue ? (const void*)&gemm_bf16_kernel<false, true, kEpiLse>
                   : (const void*)&gemm_bf16_kernel<false, false, kEpiLse>;
      break;
    case kEpiGrad:
      fn = g.queue ? (const void*)&gemm_bf16_kernel<false, true, kEpiGrad>
                   : (const void*)&gemm_bf16_kernel<false, false, kEpiGrad>;
      break;
    case kEpiLseStore:
      fn = g.queue ? (const void*)&gemm_bf16_kernel<false, true, kEpiLseStore>
                   : (const void*)&gemm_bf16_kernel<false, false, kEpiLseStore>;
      break;
    default:
      return hipErrorInvalidValue;
  }
  void* args[] = {&g};
  return hipLaunchKernel(fn, dim3((unsigned)grid), dim3(kThreads), args, 0, stream);
}

int64_t gemm_splitk_count(int64_t M, int64_t N, int64_t K, int num_cu) {
  const int64_t tiles = ((M + kGemmTile - 1) / kGemmTile) * ((N + kGemmTile - 1) / kGemmTile);
  int64_t s = 1;
  // split the contraction until every CU has a tile, keeping >= 2048 of K per split
  while (s < kGemmMaxSplits && tiles * s < num_cu && K / (2 * s) >= 2048) s *= 2;
  return s;
}

hipError_t launch_gemm_nt(GemmArgs g, bool beta, float* partial, int* queue, int num_cu,
                          hipStream_t stream) {
  if (g.M <= 0 || g.N <= 0) return hipSuccess;
  // A is M x K, B is N x K: the smaller one's tiles run fastest
  g.m_fastest = g.M <= g.N;
  const int64_t splits = partial ? gemm_splitk_count(g.M, g.N, g.K, num_cu) : 1;
  const int64_t units =
      ((g.M + kGemmTile - 1) / kGemmTile) * ((g.N + kGemmTile - 1) / kGemmTile) * splits;
  // the queues pay off once there is more than one workgroup per CU to place
  g.queue = units > num_cu ? queue : nullptr;
  if (g.queue) {  // a fill kernel rather than a memset node, so the call can be graph-captured
    void* zargs[] = {&g.queue};
    if (hipError_t e = hipLaunchKernel((const void*)&zero_queue_kernel, dim3(1),
                                       dim3(kGemmQueues), zargs, 0, stream))
      return e;
  }
  const bool c_aligned = ((uintptr_t)g.C % 16 == 0) && g.ldc % 4 == 0;
  if (splits <= 1) {
    g.k_split = g.K > 0 ? g.K : 1;
    g.c_split_stride = 0;
    g.c_vec = c_aligned;
    return launch_tiles(g, beta, 1, num_cu, stream);
  }
  // split-K: partial products into `partial` [splits][M][N], then summed in split order
  const int64_t kper = ((g.K + splits - 1) / splits + kGemmBK - 1) / kGemmBK * kGemmBK;
  GemmArgs p = g;
  p.C = partial;
  p.ldc = g.N;
  p.alpha = 1.f;
  p.k_split = kper;
  p.c_split_stride = g.M * g.N;
  p.c_vec = ((uintptr_t)partial % 16 == 0) && g.N % 4 == 0;
  if (hipError_t e = launch_tiles(p, false, (int)splits, num_cu, stream))
    return e;
  ReduceArgs r{partial, g.C, g.M, g.N, g.ldc, g.M * g.N, (int32_t)splits, g.alpha, beta};
  const int64_t blocks = (g.M * g.N + 255) / 256;
  void* args[] = {&r};
  return hipLaunchKernel((const void*)&splitk_reduce_kernel,
                         dim3((unsigned)(blocks < 4096 ? blocks : 4096)), dim3(256), args, 0,
                         stream);
}

hipError_t launch_transpose(TransposeArgs t, bool in_f32, hipStream_t stream) {
  if (t.R <= 0 || t.C <= 0) return hipSuccess;
  if (t.gp && !in_f32) return hipErrorInvalidValue;
  const int64_t tiles = ((t.C + kTransposeTile - 1) / kTransposeTile) *
                        ((t.R + kTransposeTile - 1) / kTransposeTile);
  const void* fn = t.gp    ? (const void*)&transpose_kernel<float, true>
                   : in_f32 ? (const void*)&transpose_kernel<float>
                            : (const void*)&transpose_kernel<__bf16>;
  void* args[] = {&t};
  return hipLaunchKernel(fn, dim3((unsigned)tiles), dim3(256), args, 0, stream);
}

}  // namespace cis
