// Internal interface of the LM-head products (cis_gemm.hip). Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "cis_internal.h"

namespace cis {

// Epilogues of the logits product z = h W^T of a row chunk (A = h, B = W):
//   kEpiLse:      per row and 64-column block (4 per 256-column tile tn), the pair (max, sum
//                 of exp(z - max) leaving out the sampled column) into
//                 part[row * ldp + 4 tn + wn], and the sampled logit into zy[row]; z itself
//                 is not stored;
//   kEpiGrad:     dL/dz of the row from its GradParams, rounded to bf16, into
//                 G[row * ldg + col];
//   kEpiLseStore: kEpiLse, and z into C (float32) as kEpiStore does.
enum { kEpiStore = 0, kEpiLse = 1, kEpiGrad = 2, kEpiLseStore = 3 };
struct GemmEpi {
  const int64_t* ids;       // [M] sampled ids (kEpiLse)
  float2* part;             // [M, ldp] (kEpiLse)
  float* zy;                // [M] (kEpiLse)
  int64_t ldp;
  const GradParams* gp;     // [M] (kEpiGrad)
  __bf16* G;                // [M, ldg] (kEpiGrad; ldg a multiple of 4)
  int64_t ldg;
};

// C[M, N] (float32, row stride ldc) = alpha * A[M, K] * B[N, K]^T (+ C when accumulating), or
// one of the row-loss epilogues above instead of C. A and B are bf16, row-major with K
// contiguous (row strides lda, ldb: multiples of 8 elements, bases 16-byte aligned). Any M, N,
// K >= 0. The fields after alpha are set by launch_gemm_nt.
struct GemmArgs {
  const void* A;
  const void* B;
  float* C;
  int64_t M, N, K, lda, ldb, ldc;
  float alpha;
  bool m_fastest;           // tile order: M tiles fastest
  bool c_vec;               // C rows and base allow 16-byte stores
  int64_t k_split;          // contraction length per split
  int64_t c_split_stride;   // elements between the splits' partial outputs
  int64_t units;            // tiles x splits
  int* queue;               // kGemmQueues work counters (zero at launch), or null
  int epi;                  // kEpiStore, kEpiLse or kEpiGrad
  GemmEpi e;
};

inline GemmArgs gemm_args(const void* A, const void* B, float* C, int64_t M, int64_t N,
                          int64_t K, int64_t lda, int64_t ldb, int64_t ldc) {
  GemmArgs g{};
  g.A = A;
  g.B = B;
  g.C = C;
  g.M = M;
  g.N = N;
  g.K = K;
  g.lda = lda;
  g.ldb = ldb;
  g.ldc = ldc;
  g.alpha = 1.f;
  return g;
}

// out[c][r] = bf16(f(in[r][c])), in R x C (float32 or bf16, row stride ldi), out C x R (ldo);
// out_n (nullable) receives bf16(f(in)) in the input's layout (row stride ldn). f is the
// identity, or with gp (float32 input only) the loss gradient of logit in[r][c] from row r's
// GradParams (the kEpiGrad formula). Row strides are multiples of 4 elements and bases
// 16-byte aligned.
struct TransposeArgs {
  const void* in;
  void* out;
  void* out_n;
  int64_t R, C, ldi, ldo, ldn;
  const GradParams* gp;
};

constexpr int kGemmTile = 256;      // C tile per workgroup (rows and columns)
constexpr int kGemmBK = 64;         // contraction slab
constexpr int kGemmWaveM = 128;     // C tile per wave: 128 rows x 64 columns (8 waves)
constexpr int kGemmWaveN = 64;
constexpr int kGemmMaxSplits = 8;   // split-K partial buffers
constexpr int kTransposeTile = 64;
constexpr int kGemmQueues = 8;      // one work queue per XCD

// Number of K splits launch_gemm_nt uses for an M x N x K product when given a partial buffer
// (enough workgroups for every CU; 1 when the tiles already cover the chip).
int64_t gemm_splitk_count(int64_t M, int64_t N, int64_t K, int num_cu);

// Launch on `stream`; `beta` adds the product to C instead of overwriting it. With `partial`
// (float32, >= gemm_splitk_count(...) * M * N elements, 16-byte aligned) small products are
// split along K and the partials summed in a fixed order. With `queue` (kGemmQueues ints of
// device scratch, cleared on `stream` before the product) and more tiles than CUs, one
// workgroup per CU takes tiles from per-XCD queues until all are taken, so XCDs that run faster
// take over tiles of slower ones. Results do not depend on it: a tile is computed the same way
// by whichever workgroup takes it.
hipError_t launch_gemm_nt(GemmArgs g, bool beta, float* partial, int* queue, int num_cu,
                          hipStream_t stream);
// The logits product of a row chunk with a row-loss epilogue (kEpiLse, kEpiGrad or
// kEpiLseStore; no split-K; C only with kEpiLseStore): M rows of h, N = V columns of W.
hipError_t launch_gemm_epi(GemmArgs g, int* queue, int num_cu, hipStream_t stream);
hipError_t launch_transpose(TransposeArgs t, bool in_f32, hipStream_t stream);

}  // namespace cis
