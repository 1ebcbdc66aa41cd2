// Dense products of the LM-head form (gfx950 MFMA): C = alpha * A * B^T (+ C), both operands
// K-contiguous, bf16 multiplies with float32 accumulation, and a tiled transpose that also
// converts to bf16. Used for the logits of a row chunk (hidden * W^T), the gradient with respect
// to the hidden states (G * W) and the gradient of the head weight (G^T * hidden).
//
// Tiling: a 256-thread workgroup owns a 128 x 128 tile of C as 2 x 2 waves of 64 x 64, each
// wave 2 x 2 v_mfma_f32_32x32x16_bf16 blocks. K advances 32 at a time through two LDS buffers
// (the next slab's global loads are in flight while the current one is multiplied). LDS rows
// hold 32 + 8 bf16 (80 bytes): a lane's 16-byte fragment read then hits a bank group of its own
// among the 16 lanes the hardware serves together.
//
// MFMA operand layout (32x32x16): lane l holds A[m = l % 32][k = 8 (l / 32) + i] and
// B[k = 8 (l / 32) + i][n = l % 32] for i = 0..7; accumulator register r of lane l is
// C[m = r % 4 + 8 (r / 4) + 4 (l / 32)][n = l % 32].
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "cis_gemm.h"

namespace cis {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4g __attribute__((ext_vector_type(4)));

constexpr int kGemmBM = 128, kGemmBN = 128, kGemmBK = 32, kGemmLdsW = kGemmBK + 8;

// 8 consecutive K-elements of row `r` starting at column `k` (a multiple of 8), as bf16; zeros
// outside the matrix. Rows start 16-byte aligned (ld a multiple of 8), so a whole vector is one
// aligned load; the vector that straddles K is read element by element.
__device__ __forceinline__ bf16x8 cvt8(const __bf16* q) {
  return __builtin_bit_cast(bf16x8, *(const u32x4g*)q);
}
__device__ __forceinline__ bf16x8 cvt8(const float* q) {
  const f32x4 a = ((const f32x4*)q)[0], b = ((const f32x4*)q)[1];
  bf16x8 o;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    o[i] = (__bf16)a[i];  // round to nearest even
    o[4 + i] = (__bf16)b[i];
  }
  return o;
}
template <class T>
__device__ __forceinline__ bf16x8 load8(const T* p, int64_t r, int64_t k, int64_t R, int64_t K,
                                        int64_t ld) {
  bf16x8 o{};
  if (r >= R || k >= K) return o;
  const T* q = p + r * ld + k;
  if (k + 8 <= K) return cvt8(q);
  for (int i = 0; i < 8; ++i)
    if (k + i < K) o[i] = (__bf16)q[i];
  return o;
}

// Workgroup -> C tile. Consecutive workgroup ids go to the 8 XCDs in turn and each XCD has an
// L2 of its own, so the id is first remapped so that every XCD receives a contiguous run of the
// logical order. Logically the smaller operand's tile index runs fastest: the larger operand's
// panel is then shared by consecutive workgroups and streamed from HBM about once.
__device__ __forceinline__ void tile_of(const GemmArgs& g, int64_t& tm, int64_t& tn) {
  const int64_t nwg = (int64_t)gridDim.x, id = blockIdx.x;
  const int64_t per = nwg / 8, rem = nwg % 8, x = id % 8, loc = id / 8;
  const int64_t lin = (x < rem ? x * (per + 1) : rem * (per + 1) + (x - rem) * per) + loc;
  const int64_t mt = (g.M + kGemmBM - 1) / kGemmBM, nt = (g.N + kGemmBN - 1) / kGemmBN;
  if (g.m_fastest) {
    tm = lin % mt;
    tn = lin / mt;
  } else {
    tn = lin % nt;
    tm = lin / nt;
  }
}

template <class TA, bool BETA>
__global__ __launch_bounds__(256) void gemm_nt_kernel(const GemmArgs g) {
  __shared__ __bf16 sA[2][kGemmBM * kGemmLdsW];
  __shared__ __bf16 sB[2][kGemmBN * kGemmLdsW];
  const TA* A = static_cast<const TA*>(g.A);
  const __bf16* B = static_cast<const __bf16*>(g.B);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  int64_t tm, tn;
  tile_of(g, tm, tn);
  const int64_t m0 = tm * kGemmBM, n0 = tn * kGemmBN;
  // each thread stages rows lr and lr + 64, K-vector lc of both slabs
  const int lr = tid >> 2, lc = (tid & 3) * 8;
  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x16{};
  bf16x8 ra[2], rb[2];
  auto gload = [&](int64_t k0) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      ra[h] = load8(A, m0 + lr + 64 * h, k0 + lc, g.M, g.K, g.lda);
      rb[h] = load8(B, n0 + lr + 64 * h, k0 + lc, g.N, g.K, g.ldb);
    }
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      *(bf16x8*)&sA[buf][(lr + 64 * h) * kGemmLdsW + lc] = ra[h];
      *(bf16x8*)&sB[buf][(lr + 64 * h) * kGemmLdsW + lc] = rb[h];
    }
  };
  const int64_t nk = (g.K + kGemmBK - 1) / kGemmBK;
  gload(0);
  lstore(0);
  __syncthreads();
  for (int64_t kt = 0; kt < nk; ++kt) {
    const int cur = (int)(kt & 1);
    if (kt + 1 < nk) gload((kt + 1) * kGemmBK);
#pragma unroll
    for (int ks = 0; ks < kGemmBK / 16; ++ks) {
      bf16x8 fa[2], fb[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int kk = ks * 16 + 8 * (lane >> 5);
        fa[i] = *(const bf16x8*)&sA[cur][(wm * 64 + i * 32 + (lane & 31)) * kGemmLdsW + kk];
        fb[i] = *(const bf16x8*)&sB[cur][(wn * 64 + i * 32 + (lane & 31)) * kGemmLdsW + kk];
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) lstore(cur ^ 1);
    __syncthreads();
  }
  float* C = g.C;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t m = m0 + wm * 64 + i * 32 + (r % 4) + 8 * (r / 4) + 4 * (lane >> 5);
        const int64_t n = n0 + wn * 64 + j * 32 + (lane & 31);
        if (m < g.M && n < g.N) {
          float v = g.alpha * acc[i][j][r];
          if (BETA) v += C[m * g.ldc + n];
          C[m * g.ldc + n] = v;
        }
      }
}

// out[c][r] = bf16(in[r][c]) for an R x C matrix (row strides ldi, ldo), 64 x 64 tiles through
// LDS so that both the reads and the writes are row-contiguous.
template <class TI>
__global__ __launch_bounds__(256) void transpose_kernel(const TransposeArgs t) {
  __shared__ float tile[64][65];
  const TI* in = static_cast<const TI*>(t.in);
  __bf16* out = static_cast<__bf16*>(t.out);
  const int64_t ct = (t.C + 63) / 64;
  const int64_t r0 = (int64_t)(blockIdx.x / ct) * 64, c0 = (int64_t)(blockIdx.x % ct) * 64;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
#pragma unroll
  for (int i = 0; i < 64; i += 4) {
    const int64_t r = r0 + ty + i, c = c0 + tx;
    tile[ty + i][tx] = (r < t.R && c < t.C) ? (float)in[r * t.ldi + c] : 0.f;
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < 64; i += 4) {
    const int64_t c = c0 + ty + i, r = r0 + tx;
    if (c < t.C && r < t.R) out[c * t.ldo + r] = (__bf16)tile[tx][ty + i];
  }
}

hipError_t launch_gemm_nt(GemmArgs g, bool a_f32, bool beta, hipStream_t stream) {
  if (g.M <= 0 || g.N <= 0) return hipSuccess;
  const int64_t mt = (g.M + kGemmBM - 1) / kGemmBM, nt = (g.N + kGemmBN - 1) / kGemmBN;
  // A is M x K, B is N x K: the smaller one's tiles run fastest
  g.m_fastest = g.M <= g.N;
  const void* fn = a_f32 ? (beta ? (const void*)&gemm_nt_kernel<float, true>
                                 : (const void*)&gemm_nt_kernel<float, false>)
                         : (beta ? (const void*)&gemm_nt_kernel<__bf16, true>
                                 : (const void*)&gemm_nt_kernel<__bf16, false>);
  void* args[] = {&g};
  return hipLaunchKernel(fn, dim3((unsigned)(mt * nt)), dim3(kGemmThreads), args, 0, stream);
}

hipError_t launch_transpose(TransposeArgs t, bool in_f32, hipStream_t stream) {
  if (t.R <= 0 || t.C <= 0) return hipSuccess;
  const int64_t tiles = ((t.C + kTransposeTile - 1) / kTransposeTile) *
                        ((t.R + kTransposeTile - 1) / kTransposeTile);
  const dim3 grid((unsigned)tiles);
  const void* fn =
      in_f32 ? (const void*)&transpose_kernel<float> : (const void*)&transpose_kernel<__bf16>;
  void* args[] = {&t};
  return hipLaunchKernel(fn, grid, dim3(256), args, 0, stream);
}

}  // namespace cis
