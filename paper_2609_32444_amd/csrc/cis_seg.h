// Forward pass over long rows split into segments (the loss without the gradient): short-lived
// workgroups each reduce one segment of one row, a second kernel folds each row's partials.
//
//   * cis_seg_kernel: workgroup b takes segment b % nseg of row b / nseg (consecutive
//     workgroups read consecutive segments of a row). Each thread loads its K 16-byte vectors
//     at once, takes their max, then the exp-sum relative to that max with the sampled logit
//     left out; the workgroup combines its lanes (shuffles, then LDS in a fixed order) into one
//     (max, exp-sum) pair, stored in the workspace. The thread that holds the sampled logit
//     stores it. Invalid rows are not read. The workgroups are short-lived: a persistent grid
//     whose workgroups walk segment after segment, with the next segment's loads in flight,
//     measured 10-30% slower.
//   * cis_combine_kernel: folds each row's partials in a fixed order, so the result does not
//     depend on which segment finished first, and runs the row kernel's epilogue. Rows of at
//     most kSegMax partials (every split row) take one lane each: the max of the partials, then
//     their rescaled sums in segment order, and the epilogue by that lane alone. Rows of more
//     partials (the LM head's 64-column pieces) take one wave each: lane l takes partials
//     l, l + 64, ..., then a fixed xor tree.
//
// A row's logits are read once, like the register-resident row kernel; the difference is the
// traffic pattern: many small independent reads per CU instead of one row-sized working set,
// which is what the read-only stream of this device favours.
#pragma once

#include "cis_row.h"

namespace cis {

// BLOCK threads take a segment of BLOCK * K vectors. RE: re-unpack the vectors for the
// exp-sum instead of keeping K * EPV floats alive from the max pass (fewer registers, one more
// VALU operation per logit).
template <class E, int BLOCK, int K, bool RE>
__global__ __launch_bounds__(BLOCK) void cis_seg_kernel(const RowArgs a, const SegArgs g) {
  constexpr int EPV = E::kPerVec;
  constexpr int NW = BLOCK / 64;
  __shared__ float sh_m[NW];
  __shared__ float sh_s[NW];
  const int V = a.V;
  const int64_t total = a.T * (int64_t)g.nseg;
  for (int64_t b = blockIdx.x; b < total; b += gridDim.x) {
    int tid = threadIdx.x;
    const int64_t row = b / g.nseg;
    const int seg = (int)(b - row * g.nseg);
    const RowScalars rsc = fetch_row_scalars<false>(a, row);
    if (!rsc.valid(V)) continue;  // uniform: the whole workgroup skips the row
    const int y = (int)rsc.y;
    const __amdgpu_buffer_rsrc_t rs =
        make_rsrc((const char*)a.logits + row * a.row_bytes, (uint32_t)a.nvec * 16u);
    const int v0 = seg * g.segvec + tid;
    u32x4 r[K];
    static_for<K>([&](auto I) {
      constexpr int k = I;
      r[k] = bload(rs, (uint32_t)(v0 + k * BLOCK) * 16u, 0u);
    });
    // vectors that reach past the row (the ragged last one, and whole vectors beyond it in
    // the last segment) read as -inf
    const bool tail = (v0 + (K - 1) * BLOCK + 1) * EPV > V;
    float m = kMinRef;
    static_for<K>([&](auto I) {
      constexpr int k = I;
      float f[EPV];
      E::unpack(r[k], f);
      if (tail) mask_past_end<E>(f, v0 + k * BLOCK, V);
#pragma unroll
      for (int e = 0; e < EPV; ++e) m = fmaxf(m, f[e]);
    });
    if (RE) opaque(r);
    const float mb = m * kLog2e;
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
    float zy_mine = 0.f;
    bool y_mine = false;
    const int vy = y / EPV;
    static_for<K>([&](auto I) {
      constexpr int k = I;
      float f[EPV];
      E::unpack(r[k], f);
      const int v = v0 + k * BLOCK;
      if (tail) mask_past_end<E>(f, v, V);
      if (v == vy) {  // one thread of one segment per row
        y_mine = true;
        accum_vec_skip<E>(f, mb, acc, true, y % EPV, zy_mine);
      } else {
        accum_vec<E>(f, mb, acc);
      }
    });
    float s = (acc[0] + acc[1]) + (acc[2] + acc[3]);
    wave_lse_reduce(m, s);
    if (y_mine) g.zy[row] = zy_mine;
    if (NW == 1) {
      if (tid == 0) g.part[row * g.stride + seg] = float2{m, s};
      continue;
    }
    const int wid = tid >> 6;
    if ((tid & 63) == 0) {
      sh_m[wid] = m;
      sh_s[wid] = s;
    }
    __syncthreads();
    if (tid == 0) {
      float M = sh_m[0], S = sh_s[0];
#pragma unroll
      for (int w = 1; w < NW; ++w) lse_combine(M, S, sh_m[w], sh_s[w]);
      g.part[row * g.stride + seg] = float2{M, S};
    }
    __syncthreads();  // sh_m / sh_s are reused by the next segment of this workgroup
  }
}

// GradParams of a row for the fused LM-head pass: the row kernel's gradient
// -coef exp(z - lse) = s exp2(z log2(e) - b2), and coef (1 - p) at y.
__device__ __forceinline__ GradParams grad_params(const RowResult& rr, int64_t y) {
  const float coef = rr.coef;
  const float b2 = coef != 0.f ? (rr.lse - logf(fabsf(coef))) * kLog2e : INFINITY;
  return GradParams{b2, coef > 0.f ? 1 : 0, coef * rr.one_m_p, (int32_t)y};
}

template <bool EXT>
__global__ __launch_bounds__(kCombineBlock) void cis_combine_lane_kernel(const RowArgs a,
                                                                         const SegArgs g) {
  const int64_t row = (int64_t)blockIdx.x * kCombineBlock + threadIdx.x;
  if (row >= a.T) return;  // no barrier follows
  const RowScalars rsc = fetch_row_scalars_lane<EXT>(a, row);
  if (!rsc.valid(a.V)) {
    row_invalid<EXT>(a, rsc, row);
    if (g.gp) g.gp[row] = GradParams{INFINITY, 0, 0.f, -1};
    return;
  }
  const float2* pr = g.part + row * g.stride;
  float M = kMinRef;
  for (int k = 0; k < g.nseg; ++k) M = fmaxf(M, pr[k].x);
  float s = 0.f;
  for (int k = 0; k < g.nseg; ++k) {
    const float2 p = pr[k];
    s += p.y * fast_exp2((p.x - M) * kLog2e);
  }
  const RowResult rr = row_epilogue<EXT>(a, rsc, row, M, s, g.zy[row], true);
  if (g.gp) g.gp[row] = grad_params(rr, rsc.y);
}

template <bool EXT>
__global__ __launch_bounds__(kCombineBlock) void cis_combine_kernel(const RowArgs a,
                                                                    const SegArgs g) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * (kCombineBlock / 64) +
                      (__builtin_amdgcn_readfirstlane(threadIdx.x) >> 6);
  if (row >= a.T) return;  // whole waves leave together; no barrier follows
  const RowScalars rsc = fetch_row_scalars<EXT>(a, row);
  if (!rsc.valid(a.V)) {
    if (lane == 0) {
      row_invalid<EXT>(a, rsc, row);
      if (g.gp) g.gp[row] = GradParams{INFINITY, 0, 0.f, -1};
    }
    return;
  }
  float m = kMinRef, s = 0.f;
  for (int k = lane; k < g.nseg; k += 64) {
    const float2 p = g.part[row * g.stride + k];
    lse_combine(m, s, p.x, p.y);
  }
  wave_lse_reduce(m, s);
  const float zy = g.zy[row];
  const RowResult rr = row_epilogue<EXT>(a, rsc, row, m, s, zy, lane == 0);
  if (g.gp && lane == 0) g.gp[row] = grad_params(rr, rsc.y);
}

}  // namespace cis
