// Internal interface of the LM-head products (cis_gemm.hip). Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cis {

// C[M, N] (float32, row stride ldc) = alpha * A[M, K] * B[N, K]^T (+ C when accumulating).
// A is float32 or bf16 (converted to bf16 on load, round to nearest even), B is bf16; both
// row-major with K contiguous (row strides lda, ldb, multiples of 8 elements; bases 16-byte
// aligned). Any M, N, K >= 0.
struct GemmArgs {
  const void* A;
  const void* B;
  float* C;
  int64_t M, N, K, lda, ldb, ldc;
  float alpha;
  bool m_fastest;   // set by launch_gemm_nt
};

// out[c][r] = bf16(in[r][c]), in R x C (float32 or bf16, row stride ldi), out C x R (ldo).
struct TransposeArgs {
  const void* in;
  void* out;
  int64_t R, C, ldi, ldo;
};

constexpr int kGemmTile = 128;   // C tile per workgroup (rows and columns)
constexpr int kGemmThreads = 256;
constexpr int kTransposeTile = 64;

// Launch on `stream`; `beta` adds the product to C instead of overwriting it.
hipError_t launch_gemm_nt(GemmArgs g, bool a_f32, bool beta, hipStream_t stream);
hipError_t launch_transpose(TransposeArgs t, bool in_f32, hipStream_t stream);

}  // namespace cis
