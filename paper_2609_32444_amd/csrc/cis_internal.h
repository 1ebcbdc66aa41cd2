// Internal interface between the C-ABI entry points (cis_api.cpp) and the HIP kernels
// (cis_kernels.hip, cis_kernels_ext.hip). Not installed; not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/cis.h"

namespace cis {

// Workspace layout (bytes), every array 256-byte aligned:
//   [0, 256)     cis_stats_t
//   [256, 1280)  the fused pass's row-queue counters, one per 128-byte line
//   terms  float[T]   per-row loss term
//   logk   float[T]   per-row log k (diagnostics)
//   excess float[T]   per-row k - w (diagnostics)
//   wpre   float[T]   weight from the pre-pass (decoupled path)
//   flags  uint8[T]   per-row status bits (kFlag*)
//   pflags uint8[T]   pre-pass bits (kFlagTrunc = acted on)
//   logK   double[n_seq]  per-response log K (sequence operators)
//   part   float2[T * kSegMax]  per-segment (max, exp-sum) of the split forward pass
//   zy     float[T]           the sampled logit (split forward pass)
// The last two exist only in the layout of the forward entry points (`seg`); the fused pass and
// the LM-head path do not use them.
constexpr size_t kStatsBytes = 256;
static_assert(sizeof(cis_stats_t) <= kStatsBytes, "the statistics fit their block");
// The row queue: up to kRowQueues counters of 8 bytes, each on a 128-byte line of its own.
// Returning atomics on one line are served one at a time, about 80 M per second on this part,
// which short rows approach (one draw per row); counters on separate lines are served in
// parallel. Short rows use all of them, long rows one (with eight, the long-row workloads ran
// 2-3% slower).
constexpr int kRowQueues = 8;
constexpr size_t kQueueOff = kStatsBytes;
constexpr size_t kQueueStride = 128;
constexpr size_t kHeadBytes = kQueueOff + kRowQueues * kQueueStride;
// Segments per row at most in the split forward pass (the partials per row in the workspace).
constexpr int kSegMax = 32;

// Per-row gradient parameters of the fused LM-head pass (written by the row combine, read by
// the logits product's gradient epilogue): g_j = s exp2(z_j log2(e) - b2) with s = -1 when neg
// (coef > 0), else +1; the sampled column y gets gy; y = -1 for a row without gradient
// (b2 = +inf, gy = 0).
struct GradParams {
  float b2;
  int32_t neg;
  float gy;
  int32_t y;
};

constexpr size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }
struct WsLayout {
  size_t terms, logk, excess, wpre, flags, pflags, logK, part, zy, total;
  bool seg;
};
constexpr WsLayout ws_layout(int64_t T, int64_t n_seq, bool seg = false) {
  const size_t f = align_up(4 * (size_t)T, 256), b = align_up((size_t)T, 256);
  WsLayout L{};
  L.terms = kHeadBytes;
  L.logk = L.terms + f;
  L.excess = L.logk + f;
  L.wpre = L.excess + f;
  L.flags = L.wpre + f;
  L.pflags = L.flags + b;
  L.logK = L.pflags + b;
  L.part = L.logK + align_up(8 * (size_t)n_seq, 256);
  L.zy = L.part + (seg ? align_up(8 * (size_t)kSegMax * (size_t)T, 256) : 0);
  L.total = L.zy + (seg ? f : 0);
  L.seg = seg;
  return L;
}
constexpr size_t ws_bytes(int64_t T) { return ws_layout(T, 0).total; }

// LM-head workspace: the loss workspace above, then (256-byte aligned)
//   Q   int[kGemmQueues]   the products' work queues (256 bytes)
//   Z   float[rows, ldz]   the chunk's logits (the default backward only)
//   then per row and 64-column block the pair (max, exp-sum) (float2[rows, ntv]), the sampled
//   logit (float[rows]) and the gradient parameters (GradParams[rows])
//   Wt  bf16[H, ldv]       W^T (backward)
//   Gt  bf16[V, ldc]       (dL/dz)^T of the rows of a dL/dW group (backward)
//   Ht  bf16[H, ldc]       their hidden states transposed (backward)
//   Gb  bf16[rows, ldv]    dL/dz of the chunk in bf16 (backward)
//   P   float[kLmSplits, rows, H]  split-K partials of dL/dh (backward)
// with rows = min(T, chunk), ldc = min(T, lm_dw_rows(chunk)) and row strides rounded up to 8
// elements.
constexpr int64_t kLmMaxH = int64_t(1) << 16;
constexpr int64_t kLmMaxChunk = int64_t(1) << 16;
// The products address a 256-row operand tile with 32-bit byte offsets, so operand row strides
// stay below 2^23 elements: V (the contracted length of dL/dh) and ld_h, ld_w up to 2^22.
constexpr int64_t kLmMaxV = int64_t(1) << 22;
constexpr int64_t kLmMaxLd = int64_t(1) << 22;
constexpr int64_t kLmSplits = 8;
// dL/dW is one product per group of consecutive chunks, up to kLmDwRows rows: fewer products
// that accumulate into dL/dW. A group holds whole chunks; the chunk's columns of Gt and Ht start
// 16-byte aligned only when chunk is a multiple of 8, otherwise a group is one chunk.
constexpr int64_t kLmDwRows = int64_t(1) << 14;
inline int64_t lm_dw_rows(int64_t chunk) {
  if (chunk % 8 != 0 || chunk >= kLmDwRows) return chunk;
  return chunk * (kLmDwRows / chunk);
}
struct LmLayout {
  WsLayout loss;
  int64_t ldz, ldv, ldc, ntv;
  size_t z, wt, gt, ht, gb, part, queue, total;
  size_t tpart, tzy, tgp;  // the product's (max, exp-sum) pairs, sampled logits, gradient
                           // parameters of the chunk's rows
  bool fused;
};
inline LmLayout lm_layout(int64_t T, int64_t V, int64_t H, int64_t chunk, int64_t n_seq,
                          bool bwd, bool fused) {
  LmLayout M;
  M.fused = fused;
  M.loss = ws_layout(T, n_seq);
  const int64_t rows = T < chunk ? T : chunk;
  M.ldz = (V + 7) / 8 * 8;
  M.ldv = M.ldz;
  M.ntv = (V + 255) / 256 * 4;  // four 64-column blocks per 256-column tile
  const int64_t grows = T < lm_dw_rows(chunk) ? T : lm_dw_rows(chunk);
  M.ldc = ((grows > 0 ? grows : 1) + 7) / 8 * 8;
  M.queue = align_up(M.loss.total, 256);  // the products' work queues
  M.z = M.queue + 256;
  size_t end = M.z;
  if (!fused) end += align_up((size_t)rows * (size_t)M.ldz * 4, 256);  // the chunk's logits
  M.tpart = end;
  end += align_up((size_t)rows * (size_t)M.ntv * 8, 256);
  M.tzy = end;
  end += align_up((size_t)rows * 4, 256);
  M.tgp = end;
  end += align_up((size_t)rows * sizeof(GradParams), 256);
  M.wt = M.gt = M.ht = M.gb = M.part = end;
  if (bwd) {
    end += align_up((size_t)H * (size_t)M.ldv * 2, 256);
    M.gt = end;
    end += align_up((size_t)V * (size_t)M.ldc * 2, 256);
    M.ht = end;
    end += align_up((size_t)H * (size_t)M.ldc * 2, 256);
    M.gb = end;
    end += align_up((size_t)rows * (size_t)M.ldv * 2, 256);
    M.part = end;
    end += align_up((size_t)kLmSplits * (size_t)rows * (size_t)H * 4, 256);
  }
  M.total = end;
  return M;
}

// Per-row status bits (workspace flags[T]; kFlagTrunc = the operator acted on the row).
enum : uint8_t { kFlagValid = 1, kFlagBadId = 2, kFlagNonFinite = 4, kFlagTrunc = 8 };

// Operator parameters as the kernels see them (cis_params_t minus the loss fields).
struct OpArgs {
  int32_t op;
  float lam, kappa, lo, hi;
};

// Arguments of the row kernels, passed by value.
struct RowArgs {
  const void* logits;       // [T, ld] elements
  void* dlogits;            // [T, ldg] gradient elements (bwd only)
  int64_t row_bytes;        // ld  * sizeof(logit element)
  int64_t grow_bytes;       // ldg * sizeof(gradient element)
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
  float* logk_ws;           // workspace logk[T]
  float* excess_ws;         // workspace excess[T]
  int64_t T;
  int32_t V;
  int32_t nvec;             // ceil(V / elements per 16-byte vector)
  float lam, kappa, scale;
  // extended kernels only
  OpArgs ops;               // rate-1 path: the operator applied in the epilogue
  const float* logp_old;    // non-null: decoupled path (weight from the pre-pass)
  const float* wpre_ws;     // pre-pass weight[T]
  const uint8_t* pflags_ws; // pre-pass acted bits[T]
  float* eps_out;           // nullable; rate-1 path only (the pre-pass writes it otherwise)
  float clip_low, clip_high;
  // row queue of the row kernel (up to kRowQueues counters, kQueueStride bytes apart): a
  // workgroup's first two rows are blockIdx.x and blockIdx.x + gridDim.x; with n counters in
  // use (kRowQueues for blocks of up to 512 threads, else 1), counter c hands out the later rows
  // 2*gridDim.x + c + n*q, q = 0, 1, ... Cleared by queue_reset_kernel before every launch.
  unsigned long long* queue;
};

// Rows whose (max, exp-sum) comes in pieces: the split forward pass (cis_seg_kernel) and the
// fused LM-head pass (the logits product's epilogue), folded by cis_combine_kernel.
struct SegArgs {
  float2* part;     // [T * stride] (max, exp-sum without the sampled logit) per piece
  float* zy;        // [T] the sampled logit
  int32_t nseg;     // pieces per row (<= stride)
  int32_t segvec;   // 16-byte vectors per segment (split forward pass)
  int64_t stride;   // pieces per row in `part`
  GradParams* gp;   // [T] nullable: gradient parameters for the fused LM-head pass
};
constexpr int kCombineBlock = 256;
// A compiled segment kernel: `block` threads with K 16-byte vectors each, so block * K vectors
// per segment.
struct SegVariant {
  int block, k;
  const void* fn;
};
// The segment kernel for rows of `nvec` vectors, or nullptr when the row kernel serves them
// better (short rows) or they need more than kSegMax segments of the largest variant.
const SegVariant* select_seg_variant(int dtype, int32_t nvec);
// lane: one lane per row (rows of at most kSegMax pieces), else one wave per row
const void* combine_kernel(bool ext, bool lane);
const void* combine_kernel_ext(bool lane);

struct FinalizeArgs {
  const float* terms_ws;
  const uint8_t* flags_ws;
  const float* logk_ws;
  const float* excess_ws;
  int64_t T;
  cis_stats_t* stats;
  float* loss_out;          // nullable
  cis_stats_t* stats_copy;  // nullable: a second copy of the statistics (caller's memory)
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

// Per-response sum of log k over valid tokens (sequence operators).
struct SeqSumArgs {
  const float* logp_p;
  const float* logp_q;
  const uint8_t* mask;      // nullable
  const int64_t* ids;       // nullable (weights path: validity is the mask alone)
  const int64_t* offsets;   // [n_seq + 1]
  double* logK;             // [n_seq]
  int64_t T, n_seq;
  int32_t V;
};

// Per-token weights of an operator from recorded log-probabilities: the decoupled path's
// pre-pass and cis_weights_ex.
struct PrepassArgs {
  const float* logp_p;
  const float* logp_q;
  const uint8_t* mask;      // nullable
  const int64_t* ids;       // nullable
  const int64_t* offsets;   // sequence operators
  const double* logK;       // sequence operators
  OpArgs ops;
  int64_t T, n_seq;
  int32_t V;
  float* w_out;             // nullable
  uint8_t* acted_out;       // nullable
  float* eps_out;           // nullable
  float* wpre_ws;           // nullable (loss path)
  uint8_t* pflags_ws;       // nullable (loss path)
  float* logk_ws;
  float* excess_ws;
  uint8_t* flags_ws;        // nullable: weights path writes valid/acted bits here
  float* terms_ws;          // nullable: weights path writes zeros here
};

// A compiled row-kernel variant: BLOCK threads per workgroup, NV register-resident 16-byte
// vectors per thread.
struct RowVariant {
  int block;
  int nv;                   // slots held in registers
  int nl;                   // further slots held in LDS (0: the last slot sits in a register)
  const void* fn;           // __global__ function (for hipLaunchKernel / occupancy queries)
};

// Picks the variant for `nvec` 16-byte vectors per row; dtype is CIS_BF16 or CIS_F32. The
// extended variants carry the operator family and the decoupled path in their epilogue.
const RowVariant& select_row_variant(int dtype, bool bwd, int32_t nvec);
const RowVariant& select_row_variant_ext(int dtype, bool bwd, int32_t nvec);

const void* finalize_kernel();
const void* queue_reset_kernel();
const void* weights_kernel();
const void* seq_sum_kernel();
const void* prepass_kernel();
constexpr int kFinalizeBlock = 1024;
constexpr int kWeightsBlock = 256;
constexpr int kSeqBlock = 256;      // four responses per workgroup, one per wave

}  // namespace cis
