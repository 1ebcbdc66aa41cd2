// HIP kernels (gfx950) of the operator family and the decoupled PPO-clip path: the extended
// row-kernel variants (cis_row.h with EXT), the per-response log K of the sequence operators,
// and the per-token weight pass over recorded log-probabilities (cis_weights_ex, and the
// decoupled path's pre-pass).
#define CIS_EXT true
#include "cis_row.h"
#include "cis_seg.h"

namespace cis {

static const RowVariant kBf16BwdExt[] = CIS_BWD_TABLE(Bf16);
static const RowVariant kBf16FwdExt[] = CIS_FWD_TABLE(Bf16, 18);
static const RowVariant kF32BwdExt[] = CIS_BWD_TABLE(F32);
static const RowVariant kF32FwdExt[] = CIS_FWD_TABLE(F32, 15);
const RowVariant& select_row_variant_ext(int dtype, bool bwd, int32_t nvec) {
  constexpr int nb = sizeof(kBf16BwdExt) / sizeof(kBf16BwdExt[0]);
  constexpr int nf = sizeof(kBf16FwdExt) / sizeof(kBf16FwdExt[0]);
  const RowVariant* t = dtype == CIS_BF16 ? (bwd ? kBf16BwdExt : kBf16FwdExt)
                                          : (bwd ? kF32BwdExt : kF32FwdExt);
  return pick_variant(t, bwd ? nb : nf, nvec);
}

__device__ __forceinline__ bool token_valid(const uint8_t* mask, const int64_t* ids, int V,
                                            int64_t t) {
  if (mask && mask[t] == 0) return false;
  if (ids) {
    const int64_t y = ids[t];
    return y >= 0 && y < (int64_t)V;
  }
  return true;
}

// ------------------------------------------------------------------------------------------
// Sequence operators (Table tab:baselines, Seq-TIS / Seq-MIS): log K of every response, the
// float64 sum of log k = l_p - l_q over its valid tokens. One wave per response; lanes take
// the tokens in a fixed stride and the wave reduces in a fixed tree, so K is deterministic.
// ------------------------------------------------------------------------------------------
__global__ __launch_bounds__(kSeqBlock) void cis_seq_sum_kernel(const SeqSumArgs a) {
  const int lane = threadIdx.x & 63;
  const int64_t s = (int64_t)blockIdx.x * (kSeqBlock / 64) + (threadIdx.x >> 6);
  if (s >= a.n_seq) return;  // whole waves leave together; no barrier follows
  int64_t b = a.offsets[s], e = a.offsets[s + 1];
  b = b < 0 ? 0 : (b > a.T ? a.T : b);
  e = e < b ? b : (e > a.T ? a.T : e);
  double acc = 0.0;
  for (int64_t t = b + lane; t < e; t += 64)
    if (token_valid(a.mask, a.ids, a.V, t)) acc += (double)a.logp_p[t] - (double)a.logp_q[t];
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) acc += __shfl_xor(acc, off, 64);
  if (lane == 0) a.logK[s] = acc;
}

// Response holding token t: the largest s with offsets[s] <= t, if t < offsets[s + 1];
// -1 when no response holds t. Stays within [0, n_seq] for any offsets.
__device__ __forceinline__ int64_t find_response(const int64_t* off, int64_t n_seq, int64_t t) {
  int64_t lo = 0, hi = n_seq;  // invariant: the answer is in [lo, hi)
  if (n_seq < 1 || off[0] > t) return -1;
  while (hi - lo > 1) {
    const int64_t mid = lo + (hi - lo) / 2;
    if (off[mid] <= t)
      lo = mid;
    else
      hi = mid;
  }
  return t < off[lo + 1] ? lo : -1;
}

// ------------------------------------------------------------------------------------------
// Per-token weights of an operator from recorded log-probabilities: w, acted, the
// displacement and the diagnostics (log k, k - w). The decoupled path runs it before the row
// kernel with l_p = l_old; cis_weights_ex runs it on its own.
// ------------------------------------------------------------------------------------------
__global__ __launch_bounds__(kWeightsBlock) void cis_prepass_kernel(const PrepassArgs a) {
  const bool seq = a.ops.op == CIS_OP_SEQ_TIS || a.ops.op == CIS_OP_SEQ_MIS;
  for (int64_t t = (int64_t)blockIdx.x * kWeightsBlock + threadIdx.x; t < a.T;
       t += (int64_t)gridDim.x * kWeightsBlock) {
    float w = 0.f, logk = 0.f, excess = 0.f, eps = 0.f;
    bool acted = false;
    const bool valid = token_valid(a.mask, a.ids, a.V, t);
    if (valid) {
      const float lp = a.logp_p[t], lq = a.logp_q[t];
      const float one_m_p = -expm1f(lp);
      logk = lp - lq;
      if (seq) {
        const int64_t s = find_response(a.offsets, a.n_seq, t);
        if (s >= 0) {
          const double lK = a.logK[s];
          if (a.ops.op == CIS_OP_SEQ_TIS) {
            acted = lK > log((double)a.ops.hi);
            w = acted ? a.ops.hi : (float)exp(lK);
          } else {
            const bool keep = lK >= log((double)a.ops.lo) && lK <= log((double)a.ops.hi);
            acted = !keep;
            w = keep ? (float)exp(lK) : 0.f;
          }
        }
      } else {
        w = op_weight(a.ops, lp, lq, one_m_p, acted);
      }
      const float k = expf(logk);
      excess = (k == w) ? 0.f : k - w;
      eps = displacement(lp, lq, one_m_p);
    }
    if (a.w_out) a.w_out[t] = w;
    if (a.acted_out) a.acted_out[t] = acted ? 1 : 0;
    if (a.eps_out) a.eps_out[t] = eps;
    if (a.wpre_ws) a.wpre_ws[t] = w;
    if (a.pflags_ws) a.pflags_ws[t] = acted ? kFlagTrunc : 0;
    a.logk_ws[t] = logk;
    a.excess_ws[t] = excess;
    if (a.flags_ws) a.flags_ws[t] = valid ? (uint8_t)(kFlagValid | (acted ? kFlagTrunc : 0)) : 0;
    if (a.terms_ws) a.terms_ws[t] = 0.f;
  }
}

const void* seq_sum_kernel() { return (const void*)&cis_seq_sum_kernel; }
const void* combine_kernel_ext(bool lane) {
  return lane ? (const void*)&cis_combine_lane_kernel<true> : (const void*)&cis_combine_kernel<true>;
}
const void* prepass_kernel() { return (const void*)&cis_prepass_kernel; }

}  // namespace cis
