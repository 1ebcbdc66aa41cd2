// HIP kernels (gfx950) of the CIS token loss: the base row-kernel variants (CIS weight at
// update ratio 1), the deterministic loss/statistics reduction, and the elementwise weight
// kernel of Algorithm 1. The row kernel itself is in cis_row.h.
#define CIS_EXT false
#include "cis_row.h"
#include "cis_seg.h"

namespace cis {

// ------------------------------------------------------------------------------------------
// Loss and statistics: one workgroup, fixed summation order (independent of the row grid).
// ------------------------------------------------------------------------------------------
__global__ __launch_bounds__(kFinalizeBlock) void cis_finalize_kernel(const FinalizeArgs a) {
  constexpr int NW = kFinalizeBlock / 64;
  __shared__ double sh_loss[NW];
  __shared__ double sh_exc[NW];
  __shared__ float sh_max[NW];
  __shared__ long long sh_cnt[4][NW];
  const int tid = threadIdx.x;
  double acc = 0.0, exc = 0.0;
  float mx = 0.f;
  long long nv = 0, nb = 0, nf = 0, nt = 0;
  auto take = [&](float term, uint8_t f, float lk, float ex) {
    acc += (double)term;
    nv += (f & kFlagValid) ? 1 : 0;
    nb += (f & kFlagBadId) ? 1 : 0;
    nf += (f & kFlagNonFinite) ? 1 : 0;
    nt += (f & kFlagTrunc) ? 1 : 0;
    if (f & kFlagValid) {
      mx = fmaxf(mx, fabsf(lk));  // fmaxf ignores NaN
      exc += (double)ex;
    }
  };
  // four rows per thread and step, with 16-byte (4-byte for the flags) loads of the 256-byte
  // aligned workspace arrays; the loop is unrolled so that several steps' loads are in flight
  typedef float f4 __attribute__((ext_vector_type(4)));
  const int64_t T4 = a.T / 4;
  const f4* terms4 = reinterpret_cast<const f4*>(a.terms_ws);
  const f4* logk4 = reinterpret_cast<const f4*>(a.logk_ws);
  const f4* exc4 = reinterpret_cast<const f4*>(a.excess_ws);
  const uint32_t* flags4 = reinterpret_cast<const uint32_t*>(a.flags_ws);
#pragma unroll 4
  for (int64_t q = tid; q < T4; q += kFinalizeBlock) {
    const f4 tv = terms4[q], lv = logk4[q], ev = exc4[q];
    const uint32_t fv = flags4[q];
#pragma unroll
    for (int e = 0; e < 4; ++e) take(tv[e], (uint8_t)(fv >> (8 * e)), lv[e], ev[e]);
  }
  for (int64_t t = T4 * 4 + tid; t < a.T; t += kFinalizeBlock)
    take(a.terms_ws[t], a.flags_ws[t], a.logk_ws[t], a.excess_ws[t]);
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    acc += __shfl_down(acc, off, 64);
    exc += __shfl_down(exc, off, 64);
    mx = fmaxf(mx, __shfl_down(mx, off, 64));
    nv += __shfl_down(nv, off, 64);
    nb += __shfl_down(nb, off, 64);
    nf += __shfl_down(nf, off, 64);
    nt += __shfl_down(nt, off, 64);
  }
  const int wid = tid >> 6;
  if ((tid & 63) == 0) {
    sh_loss[wid] = acc;
    sh_exc[wid] = exc;
    sh_max[wid] = mx;
    sh_cnt[0][wid] = nv;
    sh_cnt[1][wid] = nb;
    sh_cnt[2][wid] = nf;
    sh_cnt[3][wid] = nt;
  }
  __syncthreads();
  if (tid == 0) {
    double L = 0.0, X = 0.0;
    float Mx = 0.f;
    long long c[4] = {0, 0, 0, 0};
    for (int w = 0; w < NW; ++w) {
      L += sh_loss[w];
      X += sh_exc[w];
      Mx = fmaxf(Mx, sh_max[w]);
      for (int k = 0; k < 4; ++k) c[k] += sh_cnt[k][w];
    }
    a.stats->loss = L;
    a.stats->n_valid = c[0];
    a.stats->n_bad_id = c[1];
    a.stats->n_nonfinite = c[2];
    a.stats->n_trunc = c[3];
    a.stats->max_abs_logk = (double)Mx;
    a.stats->trunc_excess = X;
    a.stats->reserved = 0;
    if (a.stats_copy) *a.stats_copy = *a.stats;
    if (a.loss_out) *a.loss_out = (float)L;
  }
}

// ------------------------------------------------------------------------------------------
// Algorithm 1 as an elementwise pass over recorded log-probabilities.
// ------------------------------------------------------------------------------------------
__global__ __launch_bounds__(kWeightsBlock) void cis_weights_kernel(const WeightsArgs a) {
  for (int64_t t = (int64_t)blockIdx.x * kWeightsBlock + threadIdx.x; t < a.T;
       t += (int64_t)gridDim.x * kWeightsBlock) {
    float w = 0.f;
    bool trunc = false;
    if (!a.mask || a.mask[t]) {
      const float lt = a.logp_train[t];
      const float delta = lt - a.logp_infer[t];
      const float lam_phi = a.lam * fmaxf(-expm1f(lt), a.kappa);
      trunc = delta > log1pf(lam_phi);
      w = trunc ? 1.0f + lam_phi : expf(delta);
    }
    a.w_out[t] = w;
    if (a.trunc_out) a.trunc_out[t] = trunc ? 1 : 0;
  }
}

// ------------------------------------------------------------------------------------------
// Variant tables
// ------------------------------------------------------------------------------------------
static const RowVariant kBf16Bwd[] = CIS_BWD_TABLE(Bf16);
static const RowVariant kBf16Fwd[] = CIS_FWD_TABLE(Bf16, 18);
static const RowVariant kF32Bwd[] = CIS_BWD_TABLE(F32);
static const RowVariant kF32Fwd[] = CIS_FWD_TABLE(F32, 15);

const RowVariant& select_row_variant(int dtype, bool bwd, int32_t nvec) {
  constexpr int nb = sizeof(kBf16Bwd) / sizeof(kBf16Bwd[0]);
  constexpr int nf = sizeof(kBf16Fwd) / sizeof(kBf16Fwd[0]);
  const RowVariant* t = dtype == CIS_BF16 ? (bwd ? kBf16Bwd : kBf16Fwd) : (bwd ? kF32Bwd : kF32Fwd);
  return pick_variant(t, bwd ? nb : nf, nvec);
}

// Split forward pass. Rows shorter than kSegMinVec vectors stay with the row kernel (one short
// row per workgroup is already a small independent read); longer rows take the first variant
// that covers them with at most kSegMax segments.
constexpr int32_t kSegMinVec = 2048;
#define CIS_SEG(E, B, K, RE) SegVariant{B, K, (const void*)&cis_seg_kernel<E, B, K, RE>}
// 128-thread workgroups of 8 vectors each (16 KiB of bf16 logits) measured best at V = 32768,
// 151936 and 262144 among 64-256 threads x 4-16 vectors; longer rows take longer segments.
static const SegVariant kSegBf16[] = {CIS_SEG(Bf16, 128, 8, true), CIS_SEG(Bf16, 128, 16, true),
                                      CIS_SEG(Bf16, 256, 16, true)};
static const SegVariant kSegF32[] = {CIS_SEG(F32, 128, 8, true), CIS_SEG(F32, 128, 16, true),
                                     CIS_SEG(F32, 256, 16, true)};

const SegVariant* select_seg_variant(int dtype, int32_t nvec) {
  if (nvec < kSegMinVec) return nullptr;
  const SegVariant* t = dtype == CIS_BF16 ? kSegBf16 : kSegF32;
  for (int i = 0; i < 3; ++i)
    if ((int64_t)t[i].block * t[i].k * kSegMax >= nvec) return &t[i];
  return nullptr;
}

const void* combine_kernel(bool ext, bool lane) {
  if (ext) return combine_kernel_ext(lane);
  return lane ? (const void*)&cis_combine_lane_kernel<false> : (const void*)&cis_combine_kernel<false>;
}

// Clears the row kernel's queue counters ahead of each launch: a kernel rather than a memset,
// so a captured call holds no memset node.
__global__ __launch_bounds__(64) void cis_queue_reset_kernel(unsigned long long* q) {
  if (threadIdx.x < kRowQueues) q[threadIdx.x * (kQueueStride / sizeof(*q))] = 0ull;
}

const void* finalize_kernel() { return (const void*)&cis_finalize_kernel; }
const void* queue_reset_kernel() { return (const void*)&cis_queue_reset_kernel; }
const void* weights_kernel() { return (const void*)&cis_weights_kernel; }

}  // namespace cis
