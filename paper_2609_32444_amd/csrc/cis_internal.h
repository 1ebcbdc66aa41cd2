// Internal interface between the C-ABI entry points (cis_api.cpp) and the HIP kernels
// (cis_kernels.hip). Not installed; not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/cis.h"

namespace cis {

// Workspace layout (bytes): [0, 256) cis_stats_t; then float terms[T]; then uint8 flags[T].
constexpr size_t kStatsBytes = 256;
inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }
inline size_t ws_terms_offset() { return kStatsBytes; }
inline size_t ws_flags_offset(int64_t T) { return align_up(kStatsBytes + 4 * (size_t)T, 256); }
inline size_t ws_bytes(int64_t T) { return align_up(ws_flags_offset(T) + (size_t)T, 256); }

// Per-row status bits (workspace flags[T]).
enum : uint8_t { kFlagValid = 1, kFlagBadId = 2, kFlagNonFinite = 4, kFlagTrunc = 8 };

// Arguments of the row kernels, passed by value.
struct RowArgs {
  const void* logits;       // [T, ld] elements
  void* dlogits;            // [T, ldg] elements (bwd only)
  int64_t row_bytes;        // ld  * sizeof(elem)
  int64_t grow_bytes;       // ldg * sizeof(elem)
  const int64_t* ids;
  const float* logp_infer;
  const float* adv;
  const uint8_t* mask;      // nullable
  float* logp_train_out;    // nullable
  float* w_out;             // nullable
  uint8_t* trunc_out;       // nullable
  float* terms_user;        // nullable
  float* terms_ws;          // workspace terms[T]
  uint8_t* flags_ws;        // workspace flags[T]
  int64_t T;
  int32_t V;
  int32_t nvec;             // ceil(V / elements per 16-byte vector)
  float lam, kappa, scale;
};

struct FinalizeArgs {
  const float* terms_ws;
  const uint8_t* flags_ws;
  int64_t T;
  cis_stats_t* stats;
  float* loss_out;          // nullable
};

struct WeightsArgs {
  const float* logp_train;
  const float* logp_infer;
  const uint8_t* mask;      // nullable
  float* w_out;
  uint8_t* trunc_out;       // nullable
  int64_t T;
  float lam, kappa;
};

// A compiled row-kernel variant: BLOCK threads per workgroup, NV register-resident 16-byte
// vectors per thread.
struct RowVariant {
  int block;
  int nv;                   // slots held in registers
  int nl;                   // further slots held in LDS (0: the last slot sits in a register)
  const void* fn;           // __global__ function (for hipLaunchKernel / occupancy queries)
};

// Picks the variant for `nvec` 16-byte vectors per row; dtype is CIS_BF16 or CIS_F32.
const RowVariant& select_row_variant(int dtype, bool bwd, int32_t nvec);

const void* finalize_kernel();
const void* weights_kernel();
constexpr int kFinalizeBlock = 1024;
constexpr int kWeightsBlock = 256;

}  // namespace cis
