// Row kernel of the CIS token loss (gfx950), shared by the base and the extended kernels.
// Row kernel design (one persistent workgroup per row at a time; the fused pass takes its rows
// from a queue):
//   * Each thread owns the 16-byte vectors v = tid, tid + BLOCK, ... of the row. The first
//     NV of them stay in VGPRs from the load to the gradient store, so a row that fits in
//     NV*BLOCK vectors is read from HBM exactly once. Long rows park the next NL slots in
//     LDS (filled by buffer loads that write LDS directly, no register round trip); vectors
//     beyond that are streamed: read once for the exp-sum and, with the gradient, once more.
//   * Sweep 1: an online (max, exp-sum) pass per lane, each vector folded in as its load
//     lands (the LDS variants take the max of the resident vectors first and their exp-sum
//     after); the sampled id is left out of the sum. Lanes combine across the wave with
//     shuffles and across waves through LDS in a fixed order (deterministic).
//   * Epilogue: l_train, 1 - p (complement mass), the weight (Algorithm 1, or an operator of
//     the family, or the pre-pass weight with the clipped update ratio of Eq. (1)) and the
//     loss term, all computed redundantly by every thread from the same LDS values.
//   * Sweep 2 (backward): g_j = -coef * exp(z_j - lse), evaluated as one FMA and one v_exp_f32
//     with |coef| folded into the exponent, rounded to bf16 with the hardware RNE convert; the
//     sampled element gets coef * (1 - p).
#pragma once

#include <hip/hip_runtime.h>
#include <float.h>
#include <math.h>
#include <stdint.h>

#include <utility>

#include "cis_internal.h"

namespace cis {

// Calls f(std::integral_constant<int, 0>) ... f(std::integral_constant<int, N-1>). Every access
// to the register-resident row goes through a compile-time index, so the row array is
// promoted to VGPRs (a runtime index anywhere would move it to scratch memory).
template <class F, int... I>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
template <int N, class F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

constexpr float kLog2e = 1.44269504088896340736f;
// Lowest reference point for a lane's running max. Keeping every max >= -2^127 keeps
// max*log2(e) finite, so exp(z - max) can be evaluated with a single FMA even for lanes that
// only hold -inf (padding) entries. A row whose largest logit is outside [-2^127, 2^127] is
// reported as non-finite.
constexpr float kMinRef = -0x1p127f;
constexpr float kMaxRef = 0x1p127f;

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// ------------------------------------------------------------------------------------------
// Element formats: a 16-byte vector holds 8 bf16 or 4 fp32 logits.
// ------------------------------------------------------------------------------------------
struct Bf16 {
  static constexpr int kPerVec = 8;
  static constexpr int kBytes = 2;
  static constexpr uint32_t kNegInf2 = 0xFF80FF80u;
  static constexpr uint32_t kSignMask = 0x80008000u;

  __device__ static __forceinline__ void unpack(const u32x4 v, float (&f)[8]) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      f[2 * k] = __uint_as_float(v[k] << 16);
      f[2 * k + 1] = __uint_as_float(v[k] & 0xFFFF0000u);
    }
  }
  __device__ static __forceinline__ u32x4 pack(const float (&f)[8]) {  // round to nearest even
    u32x4 out;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      bf16x2 p = {(__bf16)f[2 * k], (__bf16)f[2 * k + 1]};
      out[k] = __builtin_bit_cast(uint32_t, p);
    }
    return out;
  }
  __device__ static __forceinline__ u32x4 neg_inf_vec() {
    return u32x4{kNegInf2, kNegInf2, kNegInf2, kNegInf2};
  }
  __device__ static __forceinline__ uint32_t bits_of(float x) {
    bf16x2 p = {(__bf16)x, (__bf16)0.0f};
    return __builtin_bit_cast(uint32_t, p) & 0xFFFFu;
  }
  // value of element e (runtime index)
  __device__ static __forceinline__ float get(const u32x4 v, int e) {
    const uint32_t d = v[e >> 1];
    return __uint_as_float((e & 1) ? (d & 0xFFFF0000u) : (d << 16));
  }
  // replace element e with the 16-bit pattern `bits`
  __device__ static __forceinline__ u32x4 set(u32x4 v, int e, uint32_t bits) {
    const int k = e >> 1;
    const uint32_t d = v[k];
    const uint32_t nd = (e & 1) ? ((d & 0x0000FFFFu) | (bits << 16)) : ((d & 0xFFFF0000u) | bits);
#pragma unroll
    for (int j = 0; j < 4; ++j)
      if (j == k) v[j] = nd;
    return v;
  }
  // elements with index >= n become -inf
  __device__ static __forceinline__ u32x4 mask_tail(u32x4 v, int n) {
#pragma unroll 1
    for (int e = n; e < 8; ++e) v = set(v, e, 0xFF80u);
    return v;
  }
  __device__ static __forceinline__ void store_elem(void* row, int idx, uint32_t bits) {
    reinterpret_cast<uint16_t*>(row)[idx] = (uint16_t)bits;
  }
  __device__ static __forceinline__ uint32_t elem_bits(const u32x4 v, int e) {
    const uint32_t d = v[e >> 1];
    return (e & 1) ? (d >> 16) : (d & 0xFFFFu);
  }
};

struct F32 {
  static constexpr int kPerVec = 4;
  static constexpr int kBytes = 4;
  static constexpr uint32_t kSignMask = 0x80000000u;

  __device__ static __forceinline__ void unpack(const u32x4 v, float (&f)[4]) {
#pragma unroll
    for (int k = 0; k < 4; ++k) f[k] = __uint_as_float(v[k]);
  }
  __device__ static __forceinline__ u32x4 pack(const float (&f)[4]) {
    u32x4 out;
#pragma unroll
    for (int k = 0; k < 4; ++k) out[k] = __float_as_uint(f[k]);
    return out;
  }
  __device__ static __forceinline__ u32x4 neg_inf_vec() {
    return u32x4{0xFF800000u, 0xFF800000u, 0xFF800000u, 0xFF800000u};
  }
  __device__ static __forceinline__ uint32_t bits_of(float x) { return __float_as_uint(x); }
  __device__ static __forceinline__ float get(const u32x4 v, int e) { return __uint_as_float(v[e]); }
  __device__ static __forceinline__ u32x4 set(u32x4 v, int e, uint32_t bits) {
#pragma unroll
    for (int j = 0; j < 4; ++j)
      if (j == e) v[j] = bits;
    return v;
  }
  __device__ static __forceinline__ u32x4 mask_tail(u32x4 v, int n) {
#pragma unroll 1
    for (int e = n; e < 4; ++e) v = set(v, e, 0xFF800000u);
    return v;
  }
  __device__ static __forceinline__ void store_elem(void* row, int idx, uint32_t bits) {
    reinterpret_cast<uint32_t*>(row)[idx] = bits;
  }
  __device__ static __forceinline__ uint32_t elem_bits(const u32x4 v, int e) { return v[e]; }
};

__device__ __forceinline__ u32x4 ld16(const u32x4* p) { return __builtin_nontemporal_load(p); }

// Buffer addressing for the row sweeps: the row base lives in a scalar resource descriptor, the
// per-thread offset tid*16 in one VGPR, and the per-slot offset i*BLOCK*16 in an SGPR, so the
// register-resident slots need no per-slot address registers. Accesses whose VGPR offset is at
// or beyond num_records are dropped (stores) or return zero (loads).
constexpr int kRsrcWord3 = 0x00020000;  // gfx9 raw buffer: 32-bit data format
constexpr int kAuxNT = 2;                // non-temporal: streamed once
constexpr uint32_t kOutOfRange = 0x80000000u;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, (int)bytes, kRsrcWord3);
}
__device__ __forceinline__ u32x4 bload(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, kAuxNT);
}
__device__ __forceinline__ void bstore(u32x4 v, __amdgpu_buffer_rsrc_t r, uint32_t voff,
                                       uint32_t soff) {
  __builtin_amdgcn_raw_buffer_store_b128(v, r, voff, soff, kAuxNT);
}
// Cache policy of the two reads of a streamed slot (rows longer than registers and LDS hold):
// the exp-sum sweep reads it with the default policy, so that the gradient sweep's read a few
// microseconds later can hit in L2 (5 slots x 16 KiB per CU stay within an XCD's 4 MB), and
// the second read is non-temporal (its last use). At V = 262144 this took the fused pass from
// 6.10 to 5.82 ms against non-temporal loads for both.
constexpr int kAuxStream1 = 0;
constexpr int kAuxStream2 = kAuxNT;
template <int AUX>
__device__ __forceinline__ u32x4 bload_aux(__amdgpu_buffer_rsrc_t r, uint32_t voff) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, voff, 0u, AUX);
}

// 16-byte buffer load that writes LDS directly: lane l of the wave stores its vector at
// lds_wave + 16*l, where lds_wave is the wave's (uniform) base address. The load is counted
// by vmcnt like any other buffer load, and the compiler does not order later LDS reads after
// it: lds_fill_wait() must precede the first read of the data.
__device__ __forceinline__ void bload_lds(__amdgpu_buffer_rsrc_t r, u32x4* lds_wave,
                                          uint32_t voff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(
      r, (__attribute__((address_space(3))) void*)lds_wave, 16, voff, 0, 0, kAuxNT);
}
__device__ __forceinline__ void lds_fill_wait() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// Elements at index >= V become -inf (the last vector of a row and lanes past it).
template <class E>
__device__ __forceinline__ void mask_past_end(float (&f)[E::kPerVec], int v, int V) {
  const int j0 = v * E::kPerVec;
#pragma unroll
  for (int e = 0; e < E::kPerVec; ++e) f[e] = (j0 + e < V) ? f[e] : -INFINITY;
}

// (m, s) pairs represent s * exp(m): combine two of them.
__device__ __forceinline__ void lse_combine(float& m, float& s, float m2, float s2) {
  const float mn = fmaxf(m, m2);
  s = s * fast_exp2((m - mn) * kLog2e) + s2 * fast_exp2((m2 - mn) * kLog2e);
  m = mn;
}

// Lane x of the lane's row of 16 after a DPP permutation within that row (CTRL: quad_perm,
// row_mirror or row_half_mirror; no lane leaves its row).
template <int CTRL>
__device__ __forceinline__ float dpp16(float x) {
  return __builtin_bit_cast(
      float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ float lane_value(float x, int lane) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), lane));
}
constexpr int kDppXor1 = 0xB1, kDppXor2 = 0x4E;              // quad_perm [1,0,3,2], [2,3,0,1]
constexpr int kDppHalfMirror = 0x141, kDppRowMirror = 0x140;  // lane i <-> 7-i, i <-> 15-i
// Max / sum over each row of 16 lanes (butterfly steps within the row); the row's result is
// taken from one of its lanes.
__device__ __forceinline__ float row16_max(float x) {
  x = fmaxf(x, dpp16<kDppXor1>(x));
  x = fmaxf(x, dpp16<kDppXor2>(x));
  x = fmaxf(x, dpp16<kDppHalfMirror>(x));
  return fmaxf(x, dpp16<kDppRowMirror>(x));
}
__device__ __forceinline__ float row16_sum(float x) {
  x += dpp16<kDppXor1>(x);
  x += dpp16<kDppXor2>(x);
  x += dpp16<kDppHalfMirror>(x);
  return x + dpp16<kDppRowMirror>(x);
}

// Wave-wide (m, s): the max first, then each lane's sum rescaled to it once and added up, so
// the exponentials are independent rather than a chain of pairwise combines. Rows of 16 lanes
// reduce through DPP (a few cycles a step, where a cross-lane shuffle through the LDS crossbar
// costs an LDS round trip); the first lanes of the four rows are read as wave-uniform values
// and combined in a fixed order, so every lane returns the same bits. All 64 lanes must be
// active.
__device__ __forceinline__ void wave_lse_reduce(float& m, float& s) {
  const float rm = row16_max(m);
  const float M = fmaxf(fmaxf(lane_value(rm, 0), lane_value(rm, 16)),
                        fmaxf(lane_value(rm, 32), lane_value(rm, 48)));
  const float rs = row16_sum(s * fast_exp2((m - M) * kLog2e));
  s = (lane_value(rs, 0) + lane_value(rs, 16)) + (lane_value(rs, 32) + lane_value(rs, 48));
  m = M;
}

// Optimisation barrier: the register-resident row is "redefined" here, so the compiler cannot
// keep unpacked fp32 copies of it alive from one sweep to the next (it re-unpacks instead,
// which costs one VALU op per element but keeps the row at 16 bytes per vector in VGPRs).
template <int I, int NV>
__device__ __forceinline__ void opaque_one(u32x4 (&r)[NV]) {
  asm volatile("" : "+v"(r[I]));
}
template <int NV>
__device__ __forceinline__ void opaque(u32x4 (&r)[NV]) {
  static_for<NV>([&](auto I) { opaque_one<I>(r); });
}

// Keeps the scheduler from moving instructions across slot boundaries. Without it, once a row
// is resident it unpacks every slot up front (one register per element) or hoists the next
// row's loads above the current sweep (two rows of registers).
__device__ __forceinline__ void slot_fence() { __builtin_amdgcn_sched_barrier(0); }

// Returns 0, computed after all of its inputs are available. Added to a refill load's offset,
// it makes the load wait until the vector it overwrites has been consumed.
__device__ __forceinline__ uint32_t after(u32x4 x) {
  uint32_t z;
  asm volatile("v_mov_b32 %0, 0" : "=v"(z) : "v"(x));
  return z;
}
__device__ __forceinline__ uint32_t after(u32x2 x) {
  uint32_t z;
  asm volatile("v_mov_b32 %0, 0" : "=v"(z) : "v"(x));
  return z;
}
__device__ __forceinline__ uint32_t after(float a, float b, float c, float d) {
  uint32_t z;
  asm volatile("v_mov_b32 %0, 0" : "=v"(z) : "v"(a), "v"(b), "v"(c), "v"(d));
  return z;
}

// Row geometry shared by the sweeps. Vector v = i*BLOCK + tid of the row is "slot i" of thread
// tid; slot L = (nvec-1)/BLOCK holds the last vector. When L <= NV, slots 0..L-1 (all complete)
// live in r[0..L-1] and slot L (possibly partial, possibly ending in padding) in one extra
// register vector rp; otherwise r holds slots 0..NV-1, the next nlds slots sit in LDS and the
// rest up to L are streamed twice.
struct RowGeom {
  int nvec, tail;
  int L;             // slot of the last vector
  int nres;          // complete slots held in r[]
  bool has_rp;       // slot L is held in rp
  bool ragged;       // the last vector ends in padding (V % elements-per-vector != 0)
  bool last_mine;    // this thread holds the last vector
  bool rp_mine;      // this thread holds a vector of slot L
  int nlds;          // slots NV..NV+nlds-1 live in LDS (only when slot L is not in rp)
  int sbeg;          // first streamed slot (streaming covers sbeg..L)
};

__device__ __forceinline__ uint32_t rp_off(int BLOCK, const RowGeom& g, uint32_t voff) {
  return (g.has_rp && g.rp_mine) ? voff + (uint32_t)(g.L * BLOCK * 16) : kOutOfRange;
}

// Gradient of one 16-byte vector of logits: exp2(z*log2e - b2) rounded to the storage format,
// with the sign applied as an xor of the sign bits (sgn = 0 or the format's sign mask).
template <class E>
__device__ __forceinline__ u32x4 grad_vec(u32x4 zv, float b2, uint32_t sgn) {
  float f[E::kPerVec];
  E::unpack(zv, f);
#pragma unroll
  for (int e = 0; e < E::kPerVec; ++e) f[e] = fast_exp2(__builtin_fmaf(f[e], kLog2e, -b2));
  return E::pack(f) ^ u32x4{sgn, sgn, sgn, sgn};
}

// Gradient output of one 16-byte vector of logits, in the logits' format and position.
template <class E>
struct GradOut {
  typedef u32x4 vec;
  static constexpr uint32_t kSign = E::kSignMask;
  __device__ static __forceinline__ vec zero() { return u32x4{0u, 0u, 0u, 0u}; }
  __device__ static __forceinline__ vec make(u32x4 zv, float b2, uint32_t sgn) {
    return grad_vec<E>(zv, b2, sgn);
  }
  __device__ static __forceinline__ void store(vec v, __amdgpu_buffer_rsrc_t r, uint32_t o) {
    bstore(v, r, o, 0u);
  }
  __device__ static __forceinline__ uint32_t elem(vec v, int e) { return E::elem_bits(v, e); }
};

// Exp-sum of one vector relative to mb = max*log2e, optionally leaving out element `skip`.
template <class E>
__device__ __forceinline__ void accum_vec(const float (&f)[E::kPerVec], float mb, float (&acc)[4]) {
#pragma unroll
  for (int e = 0; e < E::kPerVec; ++e) acc[e & 3] += fast_exp2(__builtin_fmaf(f[e], kLog2e, -mb));
}
template <class E>
__device__ __forceinline__ void accum_vec_skip(const float (&f)[E::kPerVec], float mb,
                                               float (&acc)[4], bool mine, int skip,
                                               float& z_skip) {
  // Not speculatable: keeps the caller's uniform branch a branch instead of per-slot selects.
  asm volatile("");
#pragma unroll
  for (int e = 0; e < E::kPerVec; ++e) {
    const bool hit = mine && e == skip;
    z_skip = hit ? f[e] : z_skip;
    acc[e & 3] += hit ? 0.f : fast_exp2(__builtin_fmaf(f[e], kLog2e, -mb));
  }
}

// Streamed part of a long row (slots sbeg..L): folds every logit except the sampled one into the
// lane's running (max m, exp-sum s) online, rescaling s when the max grows; records z_y if this
// thread holds it. Padding after V is skipped. With PIPE the next vector's load is in flight
// while the current one is summed (four more registers).
template <class E, int BLOCK, bool PIPE>
__device__ __forceinline__ void stream_lse(__amdgpu_buffer_rsrc_t rs, const RowGeom& g,
                                           uint32_t voff, int V, int y, float& m, float& s,
                                           float& zy_mine) {
  constexpr int EPV = E::kPerVec;
  // Two-level sum: the exponentials of kFold consecutive slots go into a partial that is then
  // added to the thread's total. With one float32 accumulator, a long row (2^28 logits: 2^18 per
  // thread) would round away every term below half an ulp of the growing total.
  constexpr uint32_t kFold = 64;
  const uint32_t end = (uint32_t)g.nvec * 16u, step = (uint32_t)(BLOCK * 16);
  uint32_t o = voff + (uint32_t)g.sbeg * step;
  u32x4 cur = PIPE ? bload_aux<kAuxStream1>(rs, o < end ? o : kOutOfRange) : u32x4{0u, 0u, 0u, 0u};
  float part = 0.f;  // both relative to the running max m
  for (; o < end; o += step) {
    u32x4 nxt = cur;
    if (PIPE)
      nxt = bload_aux<kAuxStream1>(rs, o + step < end ? o + step : kOutOfRange);
    else
      cur = bload_aux<kAuxStream1>(rs, o);
    float f[EPV];
    E::unpack(cur, f);
    const int j0 = (int)(o >> 4) * EPV;
    if (j0 + EPV > V) {  // ragged last vector
#pragma unroll
      for (int e = 0; e < EPV; ++e) f[e] = (j0 + e < V) ? f[e] : -INFINITY;
    }
    float mv = m;  // the max includes the sampled logit, the sum leaves it out
#pragma unroll
    for (int e = 0; e < EPV; ++e) mv = fmaxf(mv, f[e]);
    if (j0 <= y && y < j0 + EPV) {  // this vector holds the sampled logit
#pragma unroll
      for (int e = 0; e < EPV; ++e) {
        if (j0 + e == y) zy_mine = f[e];
        f[e] = (j0 + e == y) ? -INFINITY : f[e];
      }
    }
    const float mb = mv * kLog2e;
    const float sc = fast_exp2((m - mv) * kLog2e);
    float acc = part * sc;
#pragma unroll
    for (int e = 0; e < EPV; ++e) acc += fast_exp2(__builtin_fmaf(f[e], kLog2e, -mb));
    s *= sc;
    // slot (o - voff) / step ends a group of kFold: move the partial into the total
    const bool fold = (((o - voff) / step) % kFold) == kFold - 1;
    s = fold ? s + acc : s;
    part = fold ? 0.f : acc;
    m = mv;
    cur = nxt;
  }
  s += part;
}

// Per-row inputs other than the logits. Each workgroup fetches them one row ahead, so their
// load latency overlaps the previous row instead of stalling the start (or the epilogue) of
// the row that needs them.
struct RowScalars {
  int64_t y;
  float logp_infer, adv;
  float logp_old, wpre;  // decoupled path (extended kernels): l_old and the pre-pass weight
  bool on;               // mask bit (true when there is no mask)
  bool pacted;           // decoupled path: the pre-pass operator acted on the row
  __device__ bool valid(int V) const { return on && y >= 0 && y < (int64_t)V; }
};
// Scalar (SGPR) load of a kernel input that no thread writes while the kernel runs; the row
// index is uniform, so one load serves the whole wave and the value stays out of VGPRs.
template <class T>
__device__ __forceinline__ T sload(const T* p) {
  return *(const __attribute__((address_space(4))) T*)p;
}
// Byte `i` of a uint8 array through a scalar load of the aligned 4-byte word that holds it.
// Scalar loads read whole dwords, so for the first and last bytes of the array up to 3
// neighbouring bytes outside it are read and ignored; the C ABI states that those bytes must
// be mapped (the word never crosses a page).
__device__ __forceinline__ uint32_t sload_byte(const uint8_t* p, int64_t i) {
  const uintptr_t addr = (uintptr_t)(p + i);
  const uint32_t word = sload((const uint32_t*)(addr & ~(uintptr_t)3));
  return (word >> (8u * (uint32_t)(addr & 3))) & 0xFFu;
}
template <bool EXT>
__device__ __forceinline__ RowScalars fetch_row_scalars(const RowArgs& a, int64_t row) {
  RowScalars s{0, 0.f, 0.f, 0.f, 0.f, false, false};
  if (row < a.T) {
    s.y = sload(a.ids + row);
    s.on = a.mask ? (sload_byte(a.mask, row) != 0) : true;
    s.logp_infer = sload(a.logp_infer + row);
    s.adv = sload(a.adv + row);
    if (EXT && a.logp_old) {
      s.logp_old = sload(a.logp_old + row);
      s.wpre = sload(a.wpre_ws + row);
      s.pacted = (sload_byte(a.pflags_ws, row) & kFlagTrunc) != 0;
    }
  }
  return s;
}

// The same inputs through vector loads, for kernels whose lanes take different rows.
template <bool EXT>
__device__ __forceinline__ RowScalars fetch_row_scalars_lane(const RowArgs& a, int64_t row) {
  RowScalars s{0, 0.f, 0.f, 0.f, 0.f, false, false};
  s.y = a.ids[row];
  s.on = a.mask ? (a.mask[row] != 0) : true;
  s.logp_infer = a.logp_infer[row];
  s.adv = a.adv[row];
  if (EXT && a.logp_old) {
    s.logp_old = a.logp_old[row];
    s.wpre = a.wpre_ws[row];
    s.pacted = (a.pflags_ws[row] & kFlagTrunc) != 0;
  }
  return s;
}

// ------------------------------------------------------------------------------------------
// The operator family (App. C.1 "Operators", Table tab:baselines): the weight on the token
// loss from the training-side log-probability lp (and 1 - p), the inference-side lq, with
// k = exp(lp - lq). Comparisons with bounds are taken on log k so that no k overflows; KPop's
// Bernoulli KL is evaluated in float64 as App. D.5 prescribes.
// ------------------------------------------------------------------------------------------
__device__ __forceinline__ double bernoulli_kl(double a, double b) {
  const double lo = 1e-8, hi = 1.0 - 1e-8;
  a = fmin(fmax(a, lo), hi);
  b = fmin(fmax(b, lo), hi);
  return a * log(a / b) + (1.0 - a) * log((1.0 - a) / (1.0 - b));
}
__device__ __forceinline__ double kpop_metric(float lp, float lq) {
  const double p = exp((double)lp), q = exp((double)lq);
  if (isnan(p) || isnan(q)) return 0.0;
  return fmax(bernoulli_kl(p, q), bernoulli_kl(q, p));
}

// Returns the weight and sets `acted` when the operator changed it. Sequence operators are
// handled by the pre-pass (their weight needs the whole response).
__device__ __forceinline__ float op_weight(const OpArgs& o, float lp, float lq, float one_m_p,
                                           bool& acted) {
  const float logk = lp - lq;
  const float k = expf(logk);
  acted = false;
  switch (o.op) {
    case CIS_OP_CIS:
    case CIS_OP_TWO_SIDED: {
      const float lam_phi = o.lam * fmaxf(one_m_p, o.kappa);
      acted = logk > log1pf(lam_phi);
      float w = acted ? 1.0f + lam_phi : k;
      if (o.op == CIS_OP_TWO_SIDED) {
        const float floor = 1.0f - 0.5f * one_m_p;  // (1 + p)/2: e^eps lifted to 1/2
        if (w < floor) {
          w = floor;
          acted = true;
        }
      }
      return w;
    }
    case CIS_OP_NONE:
      return 1.0f;
    case CIS_OP_EXACT: {
      const bool below = logk < logf(o.lo), above = logk > logf(o.hi);
      acted = below || above;
      return below ? o.lo : (above ? o.hi : k);
    }
    case CIS_OP_TIS:
      acted = logk > logf(o.hi);
      return acted ? o.hi : k;
    case CIS_OP_ICEPOP: {
      const bool keep = logk >= logf(o.lo) && logk <= logf(o.hi);
      acted = !keep;
      return keep ? k : 0.0f;
    }
    case CIS_OP_KPOP: {
      const bool keep = kpop_metric(lp, lq) <= (double)o.hi;
      acted = !keep;
      return keep ? k : 0.0f;
    }
    case CIS_OP_QFIXED: {
      // cap 1/(q + (1 - q) e^{-c}) with c = log(1 + lambda)
      const float den = expf(lq) + (-expm1f(lq)) / (1.0f + o.lam);
      acted = logk > -logf(den);
      return acted ? 1.0f / den : k;
    }
    default:
      return NAN;
  }
}

// Log-odds displacement logit p - logit q (Sec. 3.1) from the two log-probabilities; +inf when
// only p = 1, -inf when only q = 1, log k when both are 1.
__device__ __forceinline__ float displacement(float lp, float lq, float one_m_p) {
  const float one_m_q = -expm1f(lq);
  const float logk = lp - lq;
  if (one_m_p == one_m_q) return logk;
  if (one_m_p <= 0.0f) return INFINITY;
  if (one_m_q <= 0.0f) return -INFINITY;
  return logk - (logf(one_m_p) - logf(one_m_q));
}

// Epilogue of a valid row (every thread of the row's workgroup or wave computes the same values
// from the same inputs; `writer` stores the per-row outputs): from the row's max M (sampled
// element included), its complement exp-sum sr = sum_{j != y} exp(z_j - M) and the sampled
// logit zy, the training log-probability, 1 - p, the weight (Algorithm 1, an operator of the
// family, or the decoupled path's pre-pass weight with the clipped ratio of Eq. (1)) and the
// loss term. Returns the gradient coefficient, the log-sum-exp and 1 - p.
struct RowResult {
  float coef, lse, one_m_p;
};
template <bool EXT>
__device__ __forceinline__ RowResult row_epilogue(const RowArgs& a, const RowScalars& rsc,
                                                  int64_t row, float M, float sr, float zy,
                                                  bool writer) {
  const float s_rest = sr;
  const float e_y = expf(zy - M);
  const float ssum = e_y + s_rest;
  const float lse = M + logf(ssum);
  const float ltr = (e_y >= s_rest) ? -log1pf(s_rest / e_y) : (zy - M) - logf(ssum);
  const float one_m_p = s_rest / ssum;
  float coef = 0.f;
  float w, term, logk = 0.f, excess = 0.f, eps = 0.f;
  bool acted, bad = false;
  const bool decoupled = EXT && a.logp_old != nullptr;
  if (!EXT) {
    // CIS weight (Algorithm 1) at update ratio 1
    const float delta = ltr - rsc.logp_infer;
    const float lam_phi = a.lam * fmaxf(one_m_p, a.kappa);
    acted = delta > log1pf(lam_phi);
    const float k = expf(delta);
    w = acted ? 1.0f + lam_phi : k;
    excess = acted ? k - w : 0.f;
    logk = delta;
    coef = a.scale * w * rsc.adv;
    term = (coef == 0.f) ? 0.f : coef * ltr;
  } else if (decoupled) {
    // Eq. (1): scale * w * min(rho A, clip(rho) A), rho = p(theta) / p_old; the gradient
    // flows where rho*A is the smaller branch
    w = rsc.wpre;
    acted = rsc.pacted;
    const float rho = expf(ltr - rsc.logp_old);
    const float A = rsc.adv;
    const bool gate = (A > 0.f && rho <= 1.f + a.clip_high) || (A < 0.f && rho >= 1.f - a.clip_low);
    const float sw = a.scale * w;
    const float clipped = fminf(fmaxf(rho, 1.f - a.clip_low), 1.f + a.clip_high);
    term = (sw == 0.f || A == 0.f) ? 0.f : sw * fminf(rho * A, clipped * A);
    coef = gate ? sw * A * rho : 0.f;
    bad = isnan(rho);
  } else {
    // any token operator at update ratio 1
    w = op_weight(a.ops, ltr, rsc.logp_infer, one_m_p, acted);
    logk = ltr - rsc.logp_infer;
    const float k = expf(logk);
    excess = (k == w) ? 0.f : k - w;
    eps = displacement(ltr, rsc.logp_infer, one_m_p);
    coef = a.scale * w * rsc.adv;
    term = (coef == 0.f) ? 0.f : coef * ltr;
  }
  const bool nonfinite =
      !(isfinite(lse) && M > kMinRef && M < kMaxRef) || isnan(w) || bad;
  if (writer) {
    if (a.logp_train_out) a.logp_train_out[row] = ltr;
    if (a.terms_user) a.terms_user[row] = term;
    a.terms_ws[row] = term;
    a.flags_ws[row] = kFlagValid | (acted ? kFlagTrunc : 0) | (nonfinite ? kFlagNonFinite : 0);
    if (!decoupled) {  // the decoupled path's pre-pass wrote these
      if (a.w_out) a.w_out[row] = w;
      if (a.trunc_out) a.trunc_out[row] = acted ? 1 : 0;
      a.logk_ws[row] = logk;
      a.excess_ws[row] = excess;
      if (EXT && a.eps_out) a.eps_out[row] = eps;
    }
  }
  return RowResult{coef, lse, one_m_p};
}

// Outputs of an invalid row (masked, or id out of range): zeros, and the bad-id flag for an
// unmasked row.
template <bool EXT>
__device__ __forceinline__ void row_invalid(const RowArgs& a, const RowScalars& rsc, int64_t row) {
  if (a.logp_train_out) a.logp_train_out[row] = 0.f;
  if (a.terms_user) a.terms_user[row] = 0.f;
  a.terms_ws[row] = 0.f;
  a.flags_ws[row] = rsc.on ? kFlagBadId : 0;
  if (!(EXT && a.logp_old)) {
    if (a.w_out) a.w_out[row] = 0.f;
    if (a.trunc_out) a.trunc_out[row] = 0;
    a.logk_ws[row] = 0.f;
    a.excess_ws[row] = 0.f;
    if (EXT && a.eps_out) a.eps_out[row] = 0.f;
  }
}

// One persistent workgroup per row at a time.
//   BWD: write the gradient (sweep 2); otherwise forward only.
//   PF:  refill each register with the next row's vector during the row's last sweep, so the
//        next row's loads overlap this row's arithmetic (the first row is loaded up front).
//        Without PF each row's loads are issued at the top of its iteration.
// An invalid row (masked, or id out of range) runs the same sweeps with its arithmetic skipped:
// its loads have zero records (no data is read) and it stores a zero gradient row.
//   NL:  slots held in LDS for rows longer than NV+1 slots (BWD only: the forward pass reads
//        every vector once anyway).
//   EXT: the epilogue also carries the operator family (rate-1 path, any token operator) and
//        the decoupled PPO-clip path (weight from the pre-pass, clipped update ratio). The base
//        kernels compute the CIS weight only, which keeps their registers for the row.
template <class E, int BLOCK, int NV, int NL, bool BWD, bool PF, bool EXT>
__global__ __launch_bounds__(BLOCK) void cis_row_kernel(const RowArgs a) {
  static_assert(NL == 0 || (BWD && !PF), "LDS slots are for the fused pass");
  using GO = GradOut<E>;
  constexpr int EPV = E::kPerVec;
  constexpr int NW = BLOCK / 64;
  __shared__ float sh_m[2][NW];
  __shared__ float sh_s[2][NW];
  __shared__ float sh_zy[2];
  __shared__ unsigned long long sh_q[2];
  __shared__ float sh_ep[2][3];  // wave 0's epilogue for the other waves: coef, b2, 1 - p
  // slot NV+k of thread tid at lds_row[k*BLOCK + tid]; each wave fills and reads its own part
  __shared__ u32x4 lds_row[NL > 0 ? NL * BLOCK : 1];

  const int V = a.V;
  int buf = 0;
  u32x4 r[NV];
  u32x4 rp;

  // Row geometry. It is loop-invariant, but letting the compiler hoist everything derived from
  // it (one mask or address per slot) out of the row loop exhausts the register file, so it is
  // re-derived from opaque copies each row (a few scalar instructions).
  auto geometry = [&](int tid) {
    int nvec_r = a.nvec;
    asm volatile("" : "+s"(nvec_r));
    RowGeom g;
    g.nvec = nvec_r;
    g.tail = V - (g.nvec - 1) * EPV;  // valid elements in the last vector, 1..EPV
    g.L = (g.nvec - 1) / BLOCK;
    g.has_rp = g.L <= NV;
    g.nres = g.has_rp ? g.L : NV;
    g.ragged = g.tail != EPV;
    g.last_mine = ((g.nvec - 1) % BLOCK) == tid;
    g.rp_mine = g.L * BLOCK + tid < g.nvec;
    g.nlds = g.has_rp ? 0 : min(NL, g.L + 1 - NV);
    g.sbeg = NV + g.nlds;
    return g;
  };
  // Read descriptor of a row: its complete and partial vectors, or nothing for invalid rows.
  auto row_rsrc = [&](int64_t row, bool valid, const RowGeom& g) {
    return make_rsrc((const char*)a.logits + (valid ? row : 0) * a.row_bytes,
                     valid ? (uint32_t)g.nvec * 16u : 0u);
  };
  // The same for the register slots only (slots 0..nres-1, all complete): their accesses need
  // no per-slot test, the range check drops the slots a shorter row does not have.
  auto reg_rsrc = [&](int64_t row, bool valid, const RowGeom& g) {
    return make_rsrc((const char*)a.logits + (valid ? row : 0) * a.row_bytes,
                     valid ? (uint32_t)(g.nres * BLOCK * 16) : 0u);
  };
  auto load_row = [&](__amdgpu_buffer_rsrc_t rs, __amdgpu_buffer_rsrc_t rr, const RowGeom& g,
                      uint32_t voff, int wid) {
    // Issued in slot order (the fences keep the scheduler from sinking slot 0's load, whose
    // address needs no add, below the others): loads return in order, so sweep 1 can fold
    // slot i as soon as the first i+1 loads have landed instead of waiting for the whole row.
    static_for<NV>([&](auto I) {
      r[I] = bload(rr, voff + (uint32_t)(I * BLOCK * 16), 0u);
      slot_fence();
    });
    rp = bload(rs, rp_off(BLOCK, g, voff), 0u);
    // (unused LDS slots get out-of-range offsets rather than a branch, so every row issues
    // the same loads and the compiler's wait counts stay exact)
    static_for<NL>([&](auto K) {
      constexpr int k = K;
      const uint32_t o = k < g.nlds ? voff + (uint32_t)((NV + k) * BLOCK * 16) : kOutOfRange;
      bload_lds(rs, &lds_row[k * BLOCK + wid * 64], o);
    });
  };
  // vector of LDS slot k (unpacked), with elements past the row's end set to -inf when slot
  // k is the row's last
  auto lds_vec = [&](int k, const RowGeom& g, int tid, float (&f)[EPV]) {
    E::unpack(lds_row[k * BLOCK + tid], f);
    if (NV + k == g.L) mask_past_end<E>(f, g.L * BLOCK + tid, V);
  };

  if (PF) {
    int tid = threadIdx.x;
    const RowGeom g = geometry(tid);
    const int64_t row = blockIdx.x;
    const bool v0 = fetch_row_scalars<EXT>(a, row).valid(V);
    load_row(row_rsrc(row, v0, g), reg_rsrc(row, v0, g), g, (uint32_t)tid * 16u, 0);
  }

  RowScalars cur = fetch_row_scalars<EXT>(a, blockIdx.x);
  // The fused pass takes rows from a queue, so that workgroups that meet cheap rows (masked
  // ones) or run on a faster part of the chip take more of them: the first three rows of a
  // workgroup are fixed, every later one is drawn as a ticket at the start of the gradient
  // sweep two rows before its use and turned into a row at the next row's reduction (the next
  // row is needed at the top of a row, for its scalars and, with PF, its loads). gfx9 counts
  // loads, stores and atomics in one in-order vmcnt, so waiting for a ticket also waits for
  // every memory operation issued before it: drawn ahead of the row's stores, it lets a masked
  // row (stores only) proceed while the previous row's stores are still in flight. Short rows
  // (blocks of up to 512 threads, or up to 4 slots per thread) draw at a high rate and use
  // kRowQueues counters on separate cache lines, since one counter serialises every draw;
  // counter c hands out the rows congruent to c modulo kRowQueues in increasing order,
  // workgroup b starts on counter b mod kRowQueues and, once its counter has run dry, moves on
  // to the next. Longer rows draw from one counter (eight measured 0.5-3.5% slower there). The
  // forward pass keeps the fixed stride: its long rows go to the split kernels, whose
  // short-lived workgroups balance by themselves.
  constexpr bool kQueue = BWD;
  int64_t nrow = (int64_t)blockIdx.x + gridDim.x;
  bool first = true;             // the first row publishes the workgroup's third, fixed row
  unsigned long long tk = 0ull;  // thread 0's ticket, drawn in the previous row's gradient sweep
  constexpr uint32_t qshift = (BLOCK <= 512 || NV <= 3) ? 3 : 0;
  static_assert((1 << 3) == kRowQueues, "short rows use every counter");
  constexpr uint64_t qmask = (1ull << qshift) - 1;
  // thread 0's counter, kept 64-bit: with a 32-bit index, the 64-bit ticket arithmetic below
  // was compiled with an uninitialised high half for it
  uint64_t qc = blockIdx.x & qmask;
  auto draw = [&](uint64_t c) -> unsigned long long {
    // The pointer goes through a VGPR so that the compiler's atomic optimizer (which turns a
    // uniform-address atomic into a wave scan and waits for its result on the spot, i.e. for
    // every older load and store of the wave) leaves it alone.
    auto* q = (__attribute__((address_space(1))) unsigned long long*)a.queue +
              c * (kQueueStride / sizeof(unsigned long long));
    asm volatile("" : "+v"(q));
    return __hip_atomic_fetch_add(q, 1ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  };
  auto ticket_row = [&](unsigned long long t, uint64_t c) -> int64_t {
    return (int64_t)(3 * (uint64_t)gridDim.x + c + (t << qshift));
  };
  for (int64_t row = blockIdx.x; row < a.T;) {
    int tid = threadIdx.x;
    asm volatile("" : "+v"(tid));
    const int wid = __builtin_amdgcn_readfirstlane(tid) >> 6;
    const RowGeom g = geometry(tid);
    uint32_t voff = (uint32_t)tid * 16u;

    const RowScalars rsc = cur;
    cur = fetch_row_scalars<EXT>(a, nrow);  // the next row's, for the next iteration
    const bool valid = rsc.valid(V);
    const int y = valid ? (int)rsc.y : 0;
    const int vy = y / EPV, ey = y % EPV;
    const int slot_y = vy / BLOCK;
    const bool y_mine = (vy % BLOCK) == tid;
    const __amdgpu_buffer_rsrc_t rs = row_rsrc(row, valid, g);
    const __amdgpu_buffer_rsrc_t rr = reg_rsrc(row, valid, g);
    void* grow = BWD ? (void*)((char*)a.dlogits + row * a.grow_bytes) : nullptr;
    // write descriptor: complete vectors only
    const __amdgpu_buffer_rsrc_t ws = make_rsrc(
        grow, BWD ? (uint32_t)(g.nvec - (g.ragged ? 1 : 0)) * 16u : 0u);
    const __amdgpu_buffer_rsrc_t wr =
        make_rsrc(grow, BWD ? (uint32_t)(g.nres * BLOCK * 16) : 0u);
    // the next row of this workgroup (prefetched during this row's last sweep)
    const bool nvalid = PF && cur.valid(V);
    const __amdgpu_buffer_rsrc_t nrs = row_rsrc(nrow, nvalid, g);
    const __amdgpu_buffer_rsrc_t nrr = reg_rsrc(nrow, nvalid, g);

    if (!PF) load_row(rs, rr, g, voff, wid);

    // (Forward only with PF: sweep 1 is the row's last sweep, so each register is refilled with
    // the next row's vector right after it has been read.)
    constexpr bool kRefill1 = PF && !BWD;
    float m = kMinRef, s = 0.f, zy_mine = 0.f;
    if constexpr (NL == 0) {
      // ---- sweep 1: max and exp-sum in one online pass -------------------------------------
      // Each vector is folded into the lane's running (max m, exp-sum s) as soon as its load
      // has landed, so little of the sum is left once the row's last load arrives: the max
      // includes the sampled logit, the sum leaves it out, and s is rescaled when the max
      // grows. (The LDS variants below keep two passes: this one's extra registers spill
      // there.)
      auto fold_vec = [&](const float (&f)[EPV], bool has_y) {
        float mv = m;
#pragma unroll
        for (int e = 0; e < EPV; ++e) mv = fmaxf(mv, f[e]);
        const float mb = mv * kLog2e;
        float a0 = s * fast_exp2((m - mv) * kLog2e), a1 = 0.f;
        if (has_y) {
          asm volatile("");  // keeps the caller's uniform branch a branch
#pragma unroll
          for (int e = 0; e < EPV; ++e) {
            const bool hit = y_mine && e == ey;
            zy_mine = hit ? f[e] : zy_mine;
            const float x = hit ? 0.f : fast_exp2(__builtin_fmaf(f[e], kLog2e, -mb));
            if (e & 1) a1 += x; else a0 += x;
          }
        } else {
#pragma unroll
          for (int e = 0; e < EPV; ++e) {
            const float x = fast_exp2(__builtin_fmaf(f[e], kLog2e, -mb));
            if (e & 1) a1 += x; else a0 += x;
          }
        }
        s = a0 + a1;
        m = mv;
      };
      static_for<NV>([&](auto I) {
        constexpr int i = I;
        float f[EPV];
        E::unpack(r[i], f);
        if (kRefill1)
          r[i] = bload(nrr, voff + (uint32_t)(i * BLOCK * 16) + after(f[0], f[EPV / 4], f[EPV / 2], f[EPV - 1]), 0u);
        if (valid && i < g.nres) fold_vec(f, i == slot_y);
        slot_fence();
      });
      if (valid) {
        // Entries of rp that are not logits of this row become -inf: lanes past the last
        // vector and the padding after V in a ragged last vector.
        rp = g.rp_mine ? rp : E::neg_inf_vec();
        if (g.ragged && g.last_mine) rp = E::mask_tail(rp, g.tail);
      }
      {
        float f[EPV];
        E::unpack(rp, f);
        if (kRefill1) rp = bload(nrs, rp_off(BLOCK, g, voff) + after(f[0], f[EPV / 4], f[EPV / 2], f[EPV - 1]), 0u);
        if (valid && g.has_rp) fold_vec(f, slot_y == g.L);
      }
      // streamed slots NV..L (rows longer than the registers hold): the same online pass, the
      // next vector's load in flight while the current one is summed
      if (valid && !g.has_rp) stream_lse<E, BLOCK, !PF>(rs, g, voff, V, y, m, s, zy_mine);
    } else {
      // LDS variants (fused pass, rows beyond the registers): two passes over the resident
      // slots, max first, then the exp-sum relative to it.
      // ---- sweep 1a: max ------------------------------------------------------------------
      if (valid) {
        static_for<NV>([&](auto I) {
          constexpr int i = I;
          if (i < g.nres) {
            float f[EPV];
            E::unpack(r[i], f);
#pragma unroll
            for (int e = 0; e < EPV; ++e) m = fmaxf(m, f[e]);
          }
          slot_fence();
        });
        // Entries of rp that are not logits of this row become -inf: lanes past the last
        // vector and the padding after V in a ragged last vector.
        rp = g.rp_mine ? rp : E::neg_inf_vec();
        if (g.ragged && g.last_mine) rp = E::mask_tail(rp, g.tail);
        if (g.has_rp) {
          float f[EPV];
          E::unpack(rp, f);
#pragma unroll
          for (int e = 0; e < EPV; ++e) m = fmaxf(m, f[e]);
        }
        if (NL > 0 && g.nlds > 0) {
          lds_fill_wait();
          static_for<NL>([&](auto K) {
            constexpr int k = K;
            if (k < g.nlds) {
              float f[EPV];
              lds_vec(k, g, tid, f);
#pragma unroll
              for (int e = 0; e < EPV; ++e) m = fmaxf(m, f[e]);
            }
          });
        }
      }
      opaque(r);

      // ---- streamed slots NV..L: one online pass for max and exp-sum, the next vector's load
      // in flight while the current one is summed -------------------------------------------
      if (valid && !g.has_rp) stream_lse<E, BLOCK, !PF>(rs, g, voff, V, y, m, s, zy_mine);

      // ---- sweep 1b: exp-sum excluding the sampled id -------------------------------------
      {
        const float mb = m * kLog2e;
        float acc[4] = {0.f, 0.f, 0.f, 0.f};
        static_for<NV>([&](auto I) {
          constexpr int i = I;
          float f[EPV];
          E::unpack(r[i], f);
          if (valid && i < g.nres) {
            if (i == slot_y)
              accum_vec_skip<E>(f, mb, acc, y_mine, ey, zy_mine);
            else
              accum_vec<E>(f, mb, acc);
          }
          slot_fence();
        });
        {
          float f[EPV];
          E::unpack(rp, f);
          if (valid && g.has_rp) {
            if (slot_y == g.L)
              accum_vec_skip<E>(f, mb, acc, y_mine, ey, zy_mine);
            else
              accum_vec<E>(f, mb, acc);
          }
        }
        if (NL > 0 && valid) {
          static_for<NL>([&](auto K) {
            constexpr int k = K;
            if (k < g.nlds) {
              float f[EPV];
              lds_vec(k, g, tid, f);
              if (NV + k == slot_y)
                accum_vec_skip<E>(f, mb, acc, y_mine, ey, zy_mine);
              else
                accum_vec<E>(f, mb, acc);
            }
          });
        }
        s += (acc[0] + acc[1]) + (acc[2] + acc[3]);
      }
    }
    if (BWD) opaque(r);
    asm volatile("" : "+v"(voff));

    // ---- block reduction and epilogue: l_train, 1 - p, weight (Algorithm 1), loss term -----
    float coef = 0.f, b2 = INFINITY, one_m_p = 0.f;
    // (at least one barrier per row, valid or not, so that the double-buffered shared values
    // of row n are read before row n + 2 writes them)
    // The row after the next one: the workgroup's third row, or the row of the ticket drawn
    // in the previous row's gradient sweep; a counter that has run dry sends thread 0 to the
    // next one (a draw waited for at once, at the end of the pass only). A row >= T after
    // every counter ends the loop.
    uint64_t nq = 0;
    if (kQueue && tid == 0) {
      int64_t r = (int64_t)blockIdx.x + 2 * (int64_t)gridDim.x;
      if (!first) {
        asm volatile("" : "+v"(tk));  // keeps the arithmetic on the ticket (and its wait) here
        r = ticket_row(tk, qc);
        for (uint64_t k = 1; k <= qmask && r >= a.T; ++k) {
          qc = (qc + 1) & qmask;
          r = ticket_row(draw(qc), qc);
        }
      }
      nq = (uint64_t)r;
      if (NW > 1) sh_q[buf] = nq;
    }
    auto drawn = [&]() -> int64_t {
      if (!kQueue) return nrow + gridDim.x;
      if (NW > 1) return (int64_t)sh_q[buf];
      const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)nq);
      const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(nq >> 32));
      return (int64_t)(((uint64_t)hi << 32) | lo);
    };
    int64_t nn;
    if (valid) {
      wave_lse_reduce(m, s);
      if ((tid & 63) == 0) {
        sh_m[buf][wid] = m;
        sh_s[buf][wid] = s;
      }
      if (y_mine) sh_zy[buf] = zy_mine;
      __syncthreads();
      nn = drawn();
      // Wave 0 alone combines the waves' pairs and runs the epilogue (a few hundred serial
      // instructions); the other waves wait at the next barrier and read its result from LDS.
      // Alone on its SIMD, wave 0 finishes sooner than sixteen waves doing the same work.
      if (NW == 1 || wid == 0) {
        // the waves' pairs: max, then the rescaled sums in wave order (independent exponentials)
        float M = sh_m[buf][0];
#pragma unroll
        for (int w = 1; w < NW; ++w) M = fmaxf(M, sh_m[buf][w]);
        float sr = 0.f;
#pragma unroll
        for (int w = 0; w < NW; ++w) sr += sh_s[buf][w] * fast_exp2((sh_m[buf][w] - M) * kLog2e);
        const float zy = sh_zy[buf];
        // M: max over the row (sampled element included); sr: sum_{j != y} exp(z_j - M).
        const RowResult rr = row_epilogue<EXT>(a, rsc, row, M, sr, zy, tid == 0);
        coef = rr.coef;
        one_m_p = rr.one_m_p;
        // g_j = -coef * exp(z_j - lse) = sign * exp2(z_j*log2e - b2) with sign = -sign(coef)
        // and b2 = (lse - ln|coef|) * log2e; coef = 0 keeps b2 = +inf, which gives an all-zero
        // row. The float32 offset is accurate to a few 1e-6 relative, far inside bf16 rounding.
        if (BWD && coef != 0.f) b2 = (rr.lse - logf(fabsf(coef))) * kLog2e;
        if (NW > 1 && tid == 0) {
          sh_ep[buf][0] = coef;
          sh_ep[buf][1] = b2;
          sh_ep[buf][2] = one_m_p;
        }
      }
      if (NW > 1) {
        __syncthreads();
        coef = sh_ep[buf][0];
        b2 = sh_ep[buf][1];
        one_m_p = sh_ep[buf][2];
      }
      buf ^= 1;
    } else {
      if (kQueue && NW > 1) __syncthreads();
      nn = drawn();
      buf ^= 1;
      if (tid == 0) row_invalid<EXT>(a, rsc, row);
    }

    // ---- sweep 2: gradient ----------------------------------------------------------------
    // Every vector is stored through the write descriptor (which drops the partial last vector
    // and out-of-range lanes); the partial last vector is then written element by element, and
    // finally the sampled element is overwritten with coef*(1-p) by the thread that stored its
    // vector (same-thread program order). Invalid rows store zeros without reading their
    // register slots, so their stores wait for no load (nor, through the in-order vmcnt, for
    // the previous row's stores).
    if (BWD) {
      // the ticket of the row after next, drawn ahead of this row's stores
      if (kQueue && tid == 0) tk = draw(qc);
      slot_fence();
      const uint32_t sgn = coef > 0.f ? GO::kSign : 0u;
      if (valid) {
        static_for<NV>([&](auto I) {
          constexpr int i = I;
          const uint32_t o = voff + (uint32_t)(i * BLOCK * 16);
          const typename GO::vec out = GO::make(r[i], b2, sgn);
          if (PF) r[i] = bload(nrr, o + after(out), 0u);
          GO::store(out, wr, o);
          slot_fence();
        });
        const uint32_t o = rp_off(BLOCK, g, voff);
        const typename GO::vec out = GO::make(rp, b2, sgn);
        if (PF) rp = bload(nrs, o + after(out), 0u);
        GO::store(out, ws, o);
      } else {
        static_for<NV>([&](auto I) {
          constexpr int i = I;
          const uint32_t o = voff + (uint32_t)(i * BLOCK * 16);
          if (PF) r[i] = bload(nrr, o, 0u);
          GO::store(GO::zero(), wr, o);
          slot_fence();
        });
        const uint32_t o = rp_off(BLOCK, g, voff);
        if (PF) rp = bload(nrs, o, 0u);
        GO::store(GO::zero(), ws, o);
      }
      static_for<NL>([&](auto K) {
        constexpr int k = K;
        if (k < g.nlds) {
          typename GO::vec out = GO::zero();
          if (valid) out = GO::make(lds_row[k * BLOCK + tid], b2, sgn);
          GO::store(out, ws, voff + (uint32_t)((NV + k) * BLOCK * 16));
        }
      });
      if (!g.has_rp) {
        // streamed slots: re-read with the next vector's load in flight
        const uint32_t end = (uint32_t)g.nvec * 16u, step = (uint32_t)(BLOCK * 16);
        uint32_t o = voff + (uint32_t)g.sbeg * step;
        u32x4 cur = bload_aux<kAuxStream2>(rs, o < end ? o : kOutOfRange);
        for (; o < end; o += step) {
          const u32x4 nxt = bload_aux<kAuxStream2>(rs, o + step < end ? o + step : kOutOfRange);
          typename GO::vec out = GO::zero();
          if (valid) out = GO::make(cur, b2, sgn);
          GO::store(out, ws, o);
          cur = nxt;
        }
      }
      if (g.ragged && g.last_mine) {
        typename GO::vec out = GO::zero();
        if (valid) out = GO::make(bload(rs, (uint32_t)(g.nvec - 1) * 16u, 0u), b2, sgn);
        for (int e = 0; e < g.tail; ++e)
          E::store_elem(grow, (g.nvec - 1) * EPV + e, GO::elem(out, e));
      }
      if (valid && y_mine) E::store_elem(grow, y, E::bits_of(coef * one_m_p));
    }
    row = nrow;
    nrow = nn;
    first = false;
  }
}

// ------------------------------------------------------------------------------------------
// Variant ladders (instantiated by each translation unit with CIS_EXT defined to the EXT value)
// ------------------------------------------------------------------------------------------
#define CIS_V(E, B, N, L, BWD, PF) \
  RowVariant{B, N, L, (const void*)&cis_row_kernel<E, B, N, L, BWD, PF, CIS_EXT>}

// Row capacity of a variant: block*(nv+1) vectors (block*(nv+nl) with LDS slots); a row goes
// to the first variant that holds it. The ladders were chosen by timing every (block, nv)
// pair over V = 1024 ... 262144: small blocks with many slots per thread win on short rows
// (more rows in flight per CU), 1024-thread blocks on long ones. The fused pass prefers
// fewer slots per thread than the forward pass, prefetches the next row during the gradient
// sweep only on short rows (on long ones it costs more than it hides), and adds 9 LDS slots
// (144 KiB) for rows beyond its registers. The fp32 forward kernel stops at 15 slots (18
// would spill the prefetched row to scratch). For rows of up to 4096 vectors (V = 32768 in
// bf16) 1024 x 3 without the prefetch took over once loads were issued in slot order and the
// queue tickets were drawn ahead of the stores: 0.625 ms against 0.635 for 512 x 7 without and
// 0.657 with the prefetch, 0.658 for 256 x 15 with it and 0.677 without.
#define CIS_BWD_TABLE(E)                                                                    \
  {CIS_V(E, 64, 1, 0, true, true),     CIS_V(E, 64, 3, 0, true, true),                      \
   CIS_V(E, 64, 7, 0, true, true),     CIS_V(E, 64, 15, 0, true, true),                     \
   CIS_V(E, 512, 3, 0, true, false),   CIS_V(E, 1024, 3, 0, true, false),                   \
   CIS_V(E, 1024, 7, 0, true, false),  CIS_V(E, 1024, 11, 0, true, false),                  \
   CIS_V(E, 1024, 15, 0, true, false), CIS_V(E, 1024, 18, 0, true, false),                  \
   CIS_V(E, 1024, 18, 9, true, false)}
#define CIS_FWD_TABLE(E, LAST)                                                              \
  {CIS_V(E, 64, 1, 0, false, true),    CIS_V(E, 64, 3, 0, false, true),                     \
   CIS_V(E, 64, 7, 0, false, true),    CIS_V(E, 64, 15, 0, false, true),                    \
   CIS_V(E, 128, 15, 0, false, true),  CIS_V(E, 256, 15, 0, false, true),                   \
   CIS_V(E, 512, 15, 0, false, true),  CIS_V(E, 1024, 11, 0, false, true),                  \
   CIS_V(E, 1024, LAST, 0, false, true)}


// First variant whose row capacity holds `nvec` vectors, else the last (which streams the rest).
inline const RowVariant& pick_variant(const RowVariant* t, int n, int32_t nvec) {
  for (int i = 0; i < n; ++i)
    if ((int64_t)t[i].block * (t[i].nv + (t[i].nl > 0 ? t[i].nl : 1)) >= nvec) return t[i];
  // longer rows: the last variant streams the vectors beyond its registers (read once for
  // the exp-sum and, with the gradient, once more)
  return t[n - 1];
}

}  // namespace cis
