// C-ABI entry points of libcis: argument validation, launch configuration and launches on the
// caller's stream. No device memory is allocated and nothing synchronises.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>
#include <string.h>

#include <mutex>

#include "cis_gemm.h"
#include "cis_internal.h"

namespace {

constexpr int kMaxDevices = 64;
constexpr int64_t kMaxV = int64_t(1) << 28;

struct DeviceInfo {
  bool ok = false;        // gfx950
  int num_cu = 0;
};

std::mutex g_mu;
DeviceInfo g_dev[kMaxDevices];
bool g_dev_init[kMaxDevices] = {};

// Occupancy cache: (device, kernel) -> resident workgroups per CU.
struct OccEntry {
  const void* fn;
  int dev;
  int per_cu;
};
OccEntry g_occ[256];
int g_nocc = 0;

int current_device(DeviceInfo* info) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return CIS_ERR_DEVICE;
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_dev_init[dev]) {
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, dev) != hipSuccess) return CIS_ERR_DEVICE;
    g_dev[dev].ok = strncmp(prop.gcnArchName, "gfx950", 6) == 0;
    g_dev[dev].num_cu = prop.multiProcessorCount;
    g_dev_init[dev] = true;
  }
  if (!g_dev[dev].ok) return CIS_ERR_DEVICE;
  *info = g_dev[dev];
  return dev;
}

int blocks_per_cu(const void* fn, int block, int dev) {
  std::lock_guard<std::mutex> lk(g_mu);
  for (int i = 0; i < g_nocc; ++i)
    if (g_occ[i].fn == fn && g_occ[i].dev == dev) return g_occ[i].per_cu;
  int n = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, fn, block, 0) != hipSuccess || n < 1) n = 1;
  if (g_nocc < (int)(sizeof(g_occ) / sizeof(g_occ[0]))) g_occ[g_nocc++] = OccEntry{fn, dev, n};
  return n;
}

bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

int launch(const void* fn, int grid, int block, void* arg, hipStream_t stream) {
  void* args[] = {arg};
  return hipLaunchKernel(fn, dim3(grid), dim3(block), args, 0, stream) == hipSuccess
             ? CIS_OK
             : CIS_ERR_LAUNCH;
}

int check_params(float lam, float kappa, float scale) {
  if (!(lam >= 0.f) || !isfinite(lam)) return CIS_ERR_PARAM;
  if (!(kappa >= 0.f && kappa <= 1.f)) return CIS_ERR_PARAM;
  if (!isfinite(scale)) return CIS_ERR_PARAM;
  return CIS_OK;
}

bool is_seq_op(int op) { return op == CIS_OP_SEQ_TIS || op == CIS_OP_SEQ_MIS; }

// Ranges of cis_params_t per operator (cis.h). `decoupled` also checks the PPO clip.
int check_op_params(const cis_params_t* p, bool decoupled) {
  if (!p) return CIS_ERR_NULL;
  if (p->op < CIS_OP_CIS || p->op > CIS_OP_SEQ_MIS) return CIS_ERR_PARAM;
  if (!isfinite(p->scale)) return CIS_ERR_PARAM;
  switch (p->op) {
    case CIS_OP_CIS:
    case CIS_OP_TWO_SIDED:
      if (int rc = check_params(p->lambda, p->kappa, p->scale)) return rc;
      break;
    case CIS_OP_QFIXED:
      if (!(p->lambda >= 0.f) || !isfinite(p->lambda)) return CIS_ERR_PARAM;
      break;
    case CIS_OP_EXACT:
    case CIS_OP_ICEPOP:
    case CIS_OP_SEQ_MIS:
      if (!(p->lo >= 0.f && p->lo <= p->hi)) return CIS_ERR_PARAM;
      break;
    case CIS_OP_TIS:
    case CIS_OP_KPOP:
    case CIS_OP_SEQ_TIS:
      if (!(p->hi >= 0.f)) return CIS_ERR_PARAM;
      break;
    default:
      break;
  }
  if (decoupled) {
    if (!(p->clip_low >= 0.f && p->clip_low <= 1.f)) return CIS_ERR_PARAM;
    if (!(p->clip_high >= 0.f) || !isfinite(p->clip_high)) return CIS_ERR_PARAM;
  }
  return CIS_OK;
}

cis::OpArgs op_args(const cis_params_t& p) {
  return cis::OpArgs{p.op, p.lambda, p.kappa, p.lo, p.hi};
}

struct Ws {
  char* base;
  cis::WsLayout L;
  float* f(size_t off) const { return reinterpret_cast<float*>(base + off); }
  uint8_t* b(size_t off) const { return reinterpret_cast<uint8_t*>(base + off); }
  cis_stats_t* stats() const { return reinterpret_cast<cis_stats_t*>(base); }
};

int launch_grid_stride(const void* fn, int64_t T, int block, const DeviceInfo& info, void* arg,
                       hipStream_t stream) {
  const int64_t need = (T + block - 1) / block;
  const int64_t cap = (int64_t)info.num_cu * 8;
  return launch(fn, (int)(need < cap ? need : cap), block, arg, stream);
}

// Sequence operators: per-response log K into the workspace.
int launch_seq_sum(const float* lp, const float* lq, const uint8_t* mask, const int64_t* ids,
                   int64_t V, const int64_t* offsets, int64_t n_seq, int64_t T, const Ws& ws,
                   hipStream_t stream) {
  cis::SeqSumArgs sa{lp, lq, mask, ids, offsets, reinterpret_cast<double*>(ws.base + ws.L.logK),
                     T, n_seq, (int32_t)V};
  const int64_t per = cis::kSeqBlock / 64;
  return launch(cis::seq_sum_kernel(), (int)((n_seq + per - 1) / per), cis::kSeqBlock, &sa,
                stream);
}

// Everything the loss entry points share. `ext` selects the extended kernels (operator
// family / decoupled path); the base entry points pass the CIS operator with ext = false.
struct LossCall {
  bool bwd, ext;
  const void* logits;
  int dtype;
  int64_t T, V, ld;
  const int64_t* ids;
  const float* logp_infer;
  const float* logp_old;
  const float* adv;
  const uint8_t* mask;
  const int64_t* offsets;
  int64_t n_seq;
  cis_params_t prm;
  void* dlogits;
  int64_t ld_g;
  float *logp_train_out, *w_out;
  uint8_t* acted_out;
  float *terms_out, *eps_out, *loss_out;
  cis_stats_t* stats_out;   // nullable: a copy of the workspace's statistics
  void* workspace;
  size_t workspace_bytes;
};

// Parameter checks shared by every loss entry point.
int check_loss_params(const LossCall& c) {
  const bool decoupled = c.logp_old != nullptr;
  if (c.ext) {
    if (int rc = check_op_params(&c.prm, decoupled)) return rc;
    if (is_seq_op(c.prm.op) && !decoupled) return CIS_ERR_PARAM;
    if (is_seq_op(c.prm.op) && c.T > 0 && c.n_seq < 1) return CIS_ERR_SHAPE;
  } else if (int rc = check_params(c.prm.lambda, c.prm.kappa, c.prm.scale)) {
    return rc;
  }
  return CIS_OK;
}

int64_t seq_count(const LossCall& c) { return c.ext && is_seq_op(c.prm.op) ? c.n_seq : 0; }

// Decoupled path: the weight depends only on (l_old, l_infer), so it is computed for all T rows
// before any logits row is read.
int launch_prepass(const LossCall& c, const Ws& ws, const DeviceInfo& info, hipStream_t stream) {
  const int64_t n_seq = seq_count(c);
  if (n_seq > 0) {
    if (int rc = launch_seq_sum(c.logp_old, c.logp_infer, c.mask, c.ids, c.V, c.offsets, n_seq,
                                c.T, ws, stream))
      return rc;
  }
  cis::PrepassArgs pa{};
  pa.logp_p = c.logp_old;
  pa.logp_q = c.logp_infer;
  pa.mask = c.mask;
  pa.ids = c.ids;
  pa.offsets = c.offsets;
  pa.logK = reinterpret_cast<const double*>(ws.base + ws.L.logK);
  pa.ops = op_args(c.prm);
  pa.T = c.T;
  pa.n_seq = n_seq;
  pa.V = (int32_t)c.V;
  pa.w_out = c.w_out;
  pa.acted_out = c.acted_out;
  pa.eps_out = c.eps_out;
  pa.wpre_ws = ws.f(ws.L.wpre);
  pa.pflags_ws = ws.b(ws.L.pflags);
  pa.logk_ws = ws.f(ws.L.logk);
  pa.excess_ws = ws.f(ws.L.excess);
  return launch_grid_stride(cis::prepass_kernel(), c.T, cis::kWeightsBlock, info, &pa, stream);
}

template <class P>
P* at(P* p, int64_t t0) { return p ? p + t0 : nullptr; }

// Row-kernel arguments for rows [t0, t0 + rows) of the call: `logits` / `dlogits` point at the
// first of those rows (row strides ld, ld_g elements of c.dtype); per-row arrays are indexed
// from t0.
cis::RowArgs row_args(const LossCall& c, const Ws& ws, const void* logits, void* dlogits,
                      int64_t ld, int64_t ld_g, int64_t t0, int64_t rows) {
  const int esize = c.dtype == CIS_BF16 ? 2 : 4;
  const int32_t nvec = (int32_t)((c.V + 16 / esize - 1) / (16 / esize));
  cis::RowArgs ra{};
  ra.logits = logits;
  ra.dlogits = dlogits;
  ra.row_bytes = ld * esize;
  ra.grow_bytes = c.bwd ? ld_g * esize : 0;
  ra.ids = c.ids + t0;
  ra.logp_infer = c.logp_infer + t0;
  ra.adv = c.adv + t0;
  ra.mask = at(c.mask, t0);
  ra.logp_train_out = at(c.logp_train_out, t0);
  ra.w_out = at(c.w_out, t0);
  ra.trunc_out = at(c.acted_out, t0);
  ra.terms_user = at(c.terms_out, t0);
  ra.terms_ws = ws.f(ws.L.terms) + t0;
  ra.flags_ws = ws.b(ws.L.flags) + t0;
  ra.logk_ws = ws.f(ws.L.logk) + t0;
  ra.excess_ws = ws.f(ws.L.excess) + t0;
  ra.T = rows;
  ra.V = (int32_t)c.V;
  ra.nvec = nvec;
  ra.lam = c.prm.lambda;
  ra.kappa = c.prm.kappa;
  ra.scale = c.prm.scale;
  ra.ops = op_args(c.prm);
  ra.logp_old = at(c.logp_old, t0);
  ra.wpre_ws = ws.f(ws.L.wpre) + t0;
  ra.pflags_ws = ws.b(ws.L.pflags) + t0;
  ra.eps_out = at(c.eps_out, t0);
  ra.clip_low = c.prm.clip_low;
  ra.clip_high = c.prm.clip_high;
  ra.queue = reinterpret_cast<unsigned long long*>(ws.base + cis::kQueueOff);
  return ra;
}

// cis_combine_kernel over rows [t0, t0 + rows): their pieces (max, exp-sum) folded and the
// epilogue run.
int launch_combine(const LossCall& c, cis::RowArgs& ra, cis::SegArgs& sa, int64_t rows,
                   hipStream_t stream) {
  void* args[] = {&ra, &sa};
  const bool lane = sa.nseg <= cis::kSegMax;  // one lane per row, else one wave per row
  const int64_t per = lane ? cis::kCombineBlock : cis::kCombineBlock / 64;
  return hipLaunchKernel(cis::combine_kernel(c.ext, lane), dim3((unsigned)((rows + per - 1) / per)),
                         dim3(cis::kCombineBlock), args, 0, stream) == hipSuccess
             ? CIS_OK
             : CIS_ERR_LAUNCH;
}

// The row kernel over rows [t0, t0 + rows) of the call (see row_args).
int launch_rows(const LossCall& c, const Ws& ws, const void* logits, void* dlogits, int64_t ld,
                int64_t ld_g, int64_t t0, int64_t rows, int dev, const DeviceInfo& info,
                hipStream_t stream) {
  if (rows <= 0) return CIS_OK;
  cis::RowArgs ra = row_args(c, ws, logits, dlogits, ld, ld_g, t0, rows);
  const int32_t nvec = ra.nvec;
  const cis::RowVariant& var = c.ext ? cis::select_row_variant_ext(c.dtype, c.bwd, nvec)
                                     : cis::select_row_variant(c.dtype, c.bwd, nvec);
  // forward pass over long rows: segment kernel + combine (when the workspace has the room)
  const cis::SegVariant* sv =
      (!c.bwd && ws.L.seg) ? cis::select_seg_variant(c.dtype, nvec) : nullptr;
  if (sv) {
    cis::SegArgs sa{};
    sa.segvec = sv->block * sv->k;
    sa.nseg = (int32_t)((nvec + sa.segvec - 1) / sa.segvec);
    sa.part = reinterpret_cast<float2*>(ws.base + ws.L.part) + t0 * cis::kSegMax;
    sa.zy = ws.f(ws.L.zy) + t0;
    sa.stride = cis::kSegMax;
    void* args[] = {&ra, &sa};
    // one short-lived workgroup per (row, segment); the kernel loops only past 2^30 of them
    const int64_t total = rows * sa.nseg;
    const int64_t cap = int64_t(1) << 30;
    if (hipLaunchKernel(sv->fn, dim3((unsigned)(total < cap ? total : cap)), dim3(sv->block),
                        args, 0, stream) != hipSuccess)
      return CIS_ERR_LAUNCH;
    return launch_combine(c, ra, sa, rows, stream);
  }
  const int per_cu = blocks_per_cu(var.fn, var.block, dev);
  const int64_t resident = (int64_t)per_cu * info.num_cu;
  const int grid = (int)(rows < resident ? rows : resident);
  if (c.bwd) {  // the fused pass takes its rows from a queue (see cis_row_kernel)
    void* qargs[] = {&ra.queue};
    if (hipLaunchKernel(cis::queue_reset_kernel(), dim3(1), dim3(64), qargs, 0, stream) !=
        hipSuccess)
      return CIS_ERR_LAUNCH;
  }
  return launch(var.fn, grid, var.block, &ra, stream);
}

int launch_finalize(const Ws& ws, int64_t T, float* loss_out, hipStream_t stream,
                    cis_stats_t* stats_out = nullptr) {
  cis::FinalizeArgs fa{ws.f(ws.L.terms), ws.b(ws.L.flags), ws.f(ws.L.logk), ws.f(ws.L.excess), T,
                       ws.stats(), loss_out, stats_out};
  return launch(cis::finalize_kernel(), 1, cis::kFinalizeBlock, &fa, stream);
}

int run_loss(const LossCall& c, hipStream_t stream) {
  const bool bwd = c.bwd;
  const int64_t T = c.T, V = c.V;
  if (c.dtype != CIS_BF16 && c.dtype != CIS_F32) return CIS_ERR_DTYPE;
  if (T < 0 || V < 1 || c.ld < V || (bwd && c.ld_g < V) || c.n_seq < 0) return CIS_ERR_SHAPE;
  const int esize = c.dtype == CIS_BF16 ? 2 : 4;
  if (V > kMaxV) return CIS_ERR_SHAPE;  // row byte offsets stay within 32 bits
  if (c.ld > INT64_MAX / esize || (bwd && c.ld_g > INT64_MAX / esize)) return CIS_ERR_SHAPE;
  if (int rc = check_loss_params(c)) return rc;
  const int64_t n_seq = seq_count(c);
  if (!c.workspace) return CIS_ERR_NULL;
  if (T > 0 && (!c.logits || !c.ids || !c.logp_infer || !c.adv || (bwd && !c.dlogits)))
    return CIS_ERR_NULL;
  if (n_seq > 0 && T > 0 && !c.offsets) return CIS_ERR_NULL;
  if (!aligned(c.workspace, 256)) return CIS_ERR_ALIGN;
  // the forward pass keeps room for the split kernels' partials (cis_workspace_bytes covers it)
  const cis::WsLayout L = cis::ws_layout(T, n_seq, !bwd);
  if (c.workspace_bytes < L.total) return CIS_ERR_WORKSPACE;
  if (T > 0) {
    if (!aligned(c.logits, 16) || (c.ld * esize) % 16 != 0) return CIS_ERR_ALIGN;
    if (bwd) {
      if (!aligned(c.dlogits, 16) || (c.ld_g * esize) % 16 != 0) return CIS_ERR_ALIGN;
      const uintptr_t a0 = (uintptr_t)c.logits, a1 = a0 + (uintptr_t)(T * c.ld * esize);
      const uintptr_t b0 = (uintptr_t)c.dlogits, b1 = b0 + (uintptr_t)(T * c.ld_g * esize);
      if (a0 == b0) {
        if (c.ld_g != c.ld) return CIS_ERR_ALIAS;
      } else if (a0 < b1 && b0 < a1) {
        return CIS_ERR_ALIAS;
      }
    }
  }
  DeviceInfo info;
  const int dev = current_device(&info);
  if (dev < 0) return dev;

  const Ws ws{static_cast<char*>(c.workspace), L};
  if (T > 0) {
    if (c.logp_old) {
      if (int rc = launch_prepass(c, ws, info, stream)) return rc;
    }
    if (int rc = launch_rows(c, ws, c.logits, c.dlogits, c.ld, c.ld_g, 0, T, dev, info, stream))
      return rc;
  }
  return launch_finalize(ws, T, c.loss_out, stream, c.stats_out);
}

// ------------------------------------------------------------------------------------------
// Fixed scratch for cis_loss_bwd_noalloc: the loss workspace of up to CIS_NOALLOC_MAX_T rows
// in a file-scope device array (one copy per device, held until the process ends). In host
// code `scratch` names a host-side stand-in, not device memory: host code uses only the
// address that hipGetSymbolAddress returns for the current device.
// ------------------------------------------------------------------------------------------
constexpr size_t kScratchBytes = cis::ws_bytes(CIS_NOALLOC_MAX_T);
static_assert(kScratchBytes % 256 == 0, "whole 256-byte blocks");
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

void* g_scratch[kMaxDevices] = {};

// Device address of `scratch` on device `dev` (the current device), looked up once per device.
int scratch_on(int dev, void** out) {
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return CIS_ERR_DEVICE;
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return CIS_OK;
}

// Byte range [lo, hi) of a rows x cols matrix with a row stride of ld elements of es bytes
// (empty for a null pointer or no rows); hi saturates at the top of the address space.
struct Span {
  uintptr_t lo, hi;
};

Span span_of(const void* p, int64_t rows, int64_t cols, int64_t ld, int es) {
  if (!p || rows <= 0 || cols <= 0) return Span{0, 0};
  const unsigned __int128 n = ((unsigned __int128)(rows - 1) * (uint64_t)ld + (uint64_t)cols) *
                              (unsigned)es;
  const uintptr_t lo = (uintptr_t)p;
  return Span{lo, n > (unsigned __int128)(UINTPTR_MAX - lo) ? UINTPTR_MAX : lo + (uintptr_t)n};
}

bool overlaps(Span a, Span b) { return a.lo < b.hi && b.lo < a.hi; }

// The loss on the logits hidden * W^T, a chunk of rows at a time (cis_lmhead_loss_fwd/_bwd).
struct LmHeadCall {
  LossCall loss;            // logits / dlogits / ld unused; dtype is the chunk's (float32)
  const void* hidden;       // [T, ld_h] bf16
  const void* weight;       // [V, ld_w] bf16
  int64_t H, ld_h, ld_w, chunk;
  float* dhidden;           // [T, ld_dh] float32
  float* dweight;           // [V, ld_dw] float32
  int64_t ld_dh, ld_dw;
  bool accumulate;
  bool recompute;           // backward: never store the logits (form the product twice)
};

int run_lmhead(const LmHeadCall& m, hipStream_t stream) {
  const LossCall& c = m.loss;
  const bool bwd = c.bwd;
  const int64_t T = c.T, V = c.V, H = m.H;
  if (T < 0 || V < 1 || V > kMaxV || H < 1 || c.n_seq < 0 || m.chunk < 1) return CIS_ERR_SHAPE;
  if (m.ld_h < H || m.ld_w < H || (bwd && (m.ld_dh < H || m.ld_dw < H))) return CIS_ERR_SHAPE;
  if (H > cis::kLmMaxH || m.chunk > cis::kLmMaxChunk || V > cis::kLmMaxV) return CIS_ERR_SHAPE;
  if (m.ld_h > cis::kLmMaxLd || m.ld_w > cis::kLmMaxLd) return CIS_ERR_SHAPE;
  if (int rc = check_loss_params(c)) return rc;
  const int64_t n_seq = seq_count(c);
  if (!c.workspace || !m.weight) return CIS_ERR_NULL;
  if (T > 0 && (!m.hidden || !c.ids || !c.logp_infer || !c.adv)) return CIS_ERR_NULL;
  if (bwd && (!m.dweight || (T > 0 && !m.dhidden))) return CIS_ERR_NULL;
  if (n_seq > 0 && T > 0 && !c.offsets) return CIS_ERR_NULL;
  if (!aligned(c.workspace, 256)) return CIS_ERR_ALIGN;
  if (!aligned(m.weight, 16) || m.ld_w % 8 != 0) return CIS_ERR_ALIGN;
  if (T > 0 && (!aligned(m.hidden, 16) || m.ld_h % 8 != 0)) return CIS_ERR_ALIGN;
  // the forward never stores the logits; the backward keeps one chunk of them unless recompute
  const cis::LmLayout LM = cis::lm_layout(T, V, H, m.chunk, n_seq, bwd, !bwd || m.recompute);
  if (c.workspace_bytes < LM.total) return CIS_ERR_WORKSPACE;
  if (bwd) {  // the gradients may not overlap each other, the operands or the workspace
    const Span dh = span_of(m.dhidden, T, H, m.ld_dh, 4), dw = span_of(m.dweight, V, H, m.ld_dw, 4);
    const Span ins[] = {span_of(m.hidden, T, H, m.ld_h, 2), span_of(m.weight, V, H, m.ld_w, 2),
                        Span{(uintptr_t)c.workspace, (uintptr_t)c.workspace + LM.total}};
    for (const Span& s : ins)
      if (overlaps(dh, s) || overlaps(dw, s)) return CIS_ERR_ALIAS;
    if (overlaps(dh, dw)) return CIS_ERR_ALIAS;
  }
  DeviceInfo info;
  const int dev = current_device(&info);
  if (dev < 0) return dev;

  char* base = static_cast<char*>(c.workspace);
  const Ws ws{base, LM.loss};
  float* Z = reinterpret_cast<float*>(base + LM.z);
  __bf16* Wt = reinterpret_cast<__bf16*>(base + LM.wt);
  __bf16* Gt = reinterpret_cast<__bf16*>(base + LM.gt);
  __bf16* Ht = reinterpret_cast<__bf16*>(base + LM.ht);
  __bf16* Gb = reinterpret_cast<__bf16*>(base + LM.gb);
  float* part = reinterpret_cast<float*>(base + LM.part);
  int* queue = reinterpret_cast<int*>(base + LM.queue);
  auto ok = [](hipError_t e) { return e == hipSuccess ? CIS_OK : CIS_ERR_LAUNCH; };
  const __bf16* hid = static_cast<const __bf16*>(m.hidden);
  const int ncu = info.num_cu;

  if (bwd && T > 0) {  // W^T once: the operand of dL/dh = G W with V as the contracted axis
    if (int rc = ok(cis::launch_transpose(
            cis::TransposeArgs{m.weight, Wt, nullptr, V, H, m.ld_w, LM.ldv, 0, nullptr}, false,
            stream)))
      return rc;
  }
  if (T > 0 && c.logp_old) {
    if (int rc = launch_prepass(c, ws, info, stream)) return rc;
  }
  const int64_t group = cis::lm_dw_rows(m.chunk);  // rows per dL/dW product
  for (int64_t t0 = 0; t0 < T; t0 += m.chunk) {
    const int64_t tc = T - t0 < m.chunk ? T - t0 : m.chunk;
    const int64_t g0 = t0 / group * group;  // first row of this chunk's dL/dW group
    const __bf16* hc = hid + t0 * m.ld_h;
    // The logits product's epilogue leaves per row and 64-column block a (max, exp-sum) pair
    // (and the sampled logit); the combine folds a row's pairs in column order, runs the loss
    // epilogue and, for the backward, writes the row's gradient parameters. The default
    // backward also stores the chunk's logits in float32 and forms G and G^T from them in one
    // tiled pass; the forward, and the backward with `recompute`, never store them (the
    // backward forms the product a second time, with an epilogue that writes G).
    cis::GemmArgs ga = cis::gemm_args(hc, m.weight, LM.fused ? nullptr : Z, tc, V, H, m.ld_h,
                                      m.ld_w, LM.fused ? 0 : LM.ldz);
    ga.epi = LM.fused ? cis::kEpiLse : cis::kEpiLseStore;
    ga.e.ids = c.ids + t0;
    ga.e.part = reinterpret_cast<float2*>(base + LM.tpart);
    ga.e.ldp = LM.ntv;
    ga.e.zy = reinterpret_cast<float*>(base + LM.tzy);
    if (int rc = ok(cis::launch_gemm_epi(ga, queue, ncu, stream))) return rc;
    cis::RowArgs ra = row_args(c, ws, nullptr, nullptr, 0, 0, t0, tc);
    cis::SegArgs sa{};
    sa.part = ga.e.part;
    sa.zy = ga.e.zy;
    sa.nseg = (int32_t)LM.ntv;
    sa.stride = LM.ntv;
    sa.gp = bwd ? reinterpret_cast<cis::GradParams*>(base + LM.tgp) : nullptr;
    if (int rc = launch_combine(c, ra, sa, tc, stream)) return rc;
    if (!bwd) continue;
    if (LM.fused) {
      ga.epi = cis::kEpiGrad;
      ga.e.gp = sa.gp;
      ga.e.G = Gb;
      ga.e.ldg = LM.ldv;
      if (int rc = ok(cis::launch_gemm_epi(ga, queue, ncu, stream))) return rc;
      // G^T (operand of dL/dW) into the group's columns t0 - g0 ..
      if (int rc = ok(cis::launch_transpose(
              cis::TransposeArgs{Gb, Gt + (t0 - g0), nullptr, tc, V, LM.ldv, LM.ldc, 0, nullptr},
              false, stream)))
        return rc;
    } else {
      // G = dL/dz in bf16 (operand of dL/dh) and G^T (operand of dL/dW, the group's columns
      // t0 - g0 ..) from the stored logits
      if (int rc = ok(cis::launch_transpose(
              cis::TransposeArgs{Z, Gt + (t0 - g0), Gb, tc, V, LM.ldz, LM.ldc, LM.ldv, sa.gp},
              true, stream)))
        return rc;
    }
    // h_c^T (operand of dL/dW)
    if (int rc = ok(cis::launch_transpose(
            cis::TransposeArgs{hc, Ht + (t0 - g0), nullptr, tc, H, m.ld_h, LM.ldc, 0, nullptr},
            false, stream)))
      return rc;
    // dL/dh_c = G W = G (W^T)^T
    if (int rc = ok(cis::launch_gemm_nt(
            cis::gemm_args(Gb, Wt, m.dhidden + t0 * m.ld_dh, tc, H, V, LM.ldv, LM.ldv, m.ld_dh),
            false, part, queue, ncu, stream)))
      return rc;
    // dL/dW (+)= G^T h over the group's rows, once its last chunk is in
    const int64_t gend = g0 + group < T ? g0 + group : T;
    if (t0 + tc < gend) continue;
    if (int rc = ok(cis::launch_gemm_nt(
            cis::gemm_args(Gt, Ht, m.dweight, V, H, gend - g0, LM.ldc, LM.ldc, m.ld_dw),
            m.accumulate || g0 > 0, nullptr, queue, ncu, stream)))
      return rc;
  }
  if (bwd && T == 0 && !m.accumulate) {  // no rows: dL/dW = 0 (an empty contraction)
    if (int rc = ok(cis::launch_gemm_nt(
            cis::gemm_args(Wt, Wt, m.dweight, V, H, 0, 8, 8, m.ld_dw), false, nullptr, queue,
            ncu, stream)))
      return rc;
  }
  return launch_finalize(ws, T, c.loss_out, stream);
}

LossCall base_call(bool bwd, const void* logits, int dtype, int64_t T, int64_t V, int64_t ld,
                   const int64_t* ids, const float* logp_infer, const float* adv,
                   const uint8_t* mask, float lam, float kappa, float scale, void* dlogits,
                   int64_t ld_g, float* logp_train_out, float* w_out, uint8_t* trunc_out,
                   float* loss_terms_out, float* loss_out, void* workspace,
                   size_t workspace_bytes) {
  LossCall c{};
  c.bwd = bwd;
  c.ext = false;
  c.logits = logits;
  c.dtype = dtype;
  c.T = T;
  c.V = V;
  c.ld = ld;
  c.ids = ids;
  c.logp_infer = logp_infer;
  c.adv = adv;
  c.mask = mask;
  c.prm = cis_params_t{CIS_OP_CIS, lam, kappa, 0.f, 0.f, 0.f, 0.f, scale};
  c.dlogits = dlogits;
  c.ld_g = ld_g;
  c.logp_train_out = logp_train_out;
  c.w_out = w_out;
  c.acted_out = trunc_out;
  c.terms_out = loss_terms_out;
  c.loss_out = loss_out;
  c.workspace = workspace;
  c.workspace_bytes = workspace_bytes;
  return c;
}

LossCall ext_call(bool bwd, const void* logits, int dtype, int64_t T, int64_t V, int64_t ld,
                  const int64_t* ids, const float* logp_infer, const float* logp_old,
                  const float* adv, const uint8_t* mask, const int64_t* offsets, int64_t n_seq,
                  const cis_params_t* params, void* dlogits, int64_t ld_g,
                  float* logp_train_out, float* w_out, uint8_t* acted_out, float* terms_out,
                  float* eps_out, float* loss_out, void* workspace, size_t workspace_bytes) {
  LossCall c = base_call(bwd, logits, dtype, T, V, ld, ids, logp_infer, adv, mask, 0.f, 0.f,
                         0.f, dlogits, ld_g, logp_train_out, w_out, acted_out, terms_out,
                         loss_out, workspace, workspace_bytes);
  c.ext = true;
  c.logp_old = logp_old;
  c.offsets = offsets;
  c.n_seq = n_seq;
  c.eps_out = eps_out;
  if (params) c.prm = *params;
  return c;
}

LmHeadCall lm_call(bool bwd, const void* hidden, int64_t T, int64_t H, int64_t ld_h,
                   const void* weight, int64_t V, int64_t ld_w, const int64_t* ids,
                   const float* logp_infer, const float* logp_old, const float* adv,
                   const uint8_t* mask, const int64_t* offsets, int64_t n_seq,
                   const cis_params_t* params, int64_t chunk, float* dhidden, int64_t ld_dh,
                   float* dweight, int64_t ld_dw, int accumulate, int recompute,
                   float* logp_train_out,
                   float* w_out, uint8_t* acted_out, float* terms_out, float* eps_out,
                   float* loss_out, void* workspace, size_t workspace_bytes) {
  LmHeadCall m{};
  m.loss = ext_call(bwd, nullptr, CIS_F32, T, V, 0, ids, logp_infer, logp_old, adv, mask, offsets,
                    n_seq, params, nullptr, 0, logp_train_out, w_out, acted_out, terms_out,
                    eps_out, loss_out, workspace, workspace_bytes);
  m.hidden = hidden;
  m.weight = weight;
  m.H = H;
  m.ld_h = ld_h;
  m.ld_w = ld_w;
  m.chunk = chunk;
  m.dhidden = dhidden;
  m.dweight = dweight;
  m.ld_dh = ld_dh;
  m.ld_dw = ld_dw;
  m.accumulate = accumulate != 0;
  m.recompute = recompute != 0;
  return m;
}

}  // namespace

extern "C" {

size_t cis_lmhead_workspace_bytes(int64_t T, int64_t V, int64_t H, int64_t chunk, int64_t n_seq,
                                  int with_grad) {
  if (T < 0 || V < 1 || H < 1 || chunk < 1 || n_seq < 0) return 0;
  if (V > cis::kLmMaxV || H > cis::kLmMaxH || chunk > cis::kLmMaxChunk) return 0;
  if (with_grad < 0 || with_grad > 2) return 0;
  return cis::lm_layout(T, V, H, chunk, n_seq, with_grad != 0, with_grad != 1).total;
}

int cis_lmhead_loss_fwd(const void* hidden, int64_t T, int64_t H, int64_t ld_h,
                        const void* weight, int64_t V, int64_t ld_w, const int64_t* ids,
                        const float* logp_infer, const float* logp_old, const float* adv,
                        const uint8_t* mask, const int64_t* seq_offsets, int64_t n_seq,
                        const cis_params_t* params, int64_t chunk, float* logp_train_out,
                        float* w_out, uint8_t* acted_out, float* loss_terms_out, float* eps_out,
                        float* loss_out, void* workspace, size_t workspace_bytes,
                        hipStream_t stream) {
  if (!params) return CIS_ERR_NULL;
  return run_lmhead(lm_call(false, hidden, T, H, ld_h, weight, V, ld_w, ids, logp_infer,
                            logp_old, adv, mask, seq_offsets, n_seq, params, chunk, nullptr, 0,
                            nullptr, 0, 0, 0, logp_train_out, w_out, acted_out, loss_terms_out,
                            eps_out, loss_out, workspace, workspace_bytes),
                    stream);
}

int cis_lmhead_loss_bwd(const void* hidden, int64_t T, int64_t H, int64_t ld_h,
                        const void* weight, int64_t V, int64_t ld_w, const int64_t* ids,
                        const float* logp_infer, const float* logp_old, const float* adv,
                        const uint8_t* mask, const int64_t* seq_offsets, int64_t n_seq,
                        const cis_params_t* params, int64_t chunk, float* dhidden,
                        int64_t ld_dh, float* dweight, int64_t ld_dw, int accumulate_dweight,
                        int recompute, float* logp_train_out, float* w_out, uint8_t* acted_out,
                        float* loss_terms_out, float* eps_out, float* loss_out, void* workspace,
                        size_t workspace_bytes, hipStream_t stream) {
  if (!params) return CIS_ERR_NULL;
  if (recompute != 0 && recompute != 1) return CIS_ERR_PARAM;
  return run_lmhead(lm_call(true, hidden, T, H, ld_h, weight, V, ld_w, ids, logp_infer,
                            logp_old, adv, mask, seq_offsets, n_seq, params, chunk, dhidden,
                            ld_dh, dweight, ld_dw, accumulate_dweight, recompute, logp_train_out,
                            w_out,
                            acted_out, loss_terms_out, eps_out, loss_out, workspace,
                            workspace_bytes),
                    stream);
}

size_t cis_workspace_bytes(int64_t T) { return T < 0 ? 0 : cis::ws_layout(T, 0, true).total; }

size_t cis_workspace_bytes_ex(int64_t T, int64_t n_seq) {
  return (T < 0 || n_seq < 0) ? 0 : cis::ws_layout(T, n_seq, true).total;
}

const char* cis_status_string(int status) {
  switch (status) {
    case CIS_OK: return "ok";
    case CIS_ERR_NULL: return "a required pointer is NULL";
    case CIS_ERR_SHAPE:
      return "invalid shape (T < 0, V outside [1, 2^28], a row stride < V, n_seq < 0, or a "
             "sequence operator without responses)";
    case CIS_ERR_DTYPE: return "unknown dtype";
    case CIS_ERR_PARAM:
      return "invalid parameter (lambda must be finite and >= 0, kappa in [0,1], scale finite; "
             "operator known, its bounds in range, PPO clip in range; sequence operators need "
             "logp_old)";
    case CIS_ERR_ALIGN:
      return "misaligned buffer (logits/dlogits base and row stride must be 16-byte multiples; "
             "workspace 256-byte aligned)";
    case CIS_ERR_LAUNCH: return "kernel launch failed";
    case CIS_ERR_WORKSPACE: return "workspace too small (see cis_workspace_bytes)";
    case CIS_ERR_ALIAS: return "dlogits overlaps logits other than exactly in place (ld_g == ld)";
    case CIS_ERR_DEVICE: return "current device is not a gfx950 GPU";
    case CIS_ERR_SCRATCH:
      return "T exceeds the fixed scratch of cis_loss_bwd_noalloc (CIS_NOALLOC_MAX_T = 262144 "
             "rows); use cis_loss_bwd with a workspace";
    default: return "unknown status";
  }
}

int cis_weights(const float* logp_train, const float* logp_infer, const uint8_t* mask,
                int64_t T, float lambda, float kappa, float* w_out, uint8_t* trunc_out,
                hipStream_t stream) {
  if (T < 0) return CIS_ERR_SHAPE;
  if (int rc = check_params(lambda, kappa, 1.0f)) return rc;
  if (T == 0) return CIS_OK;
  if (!logp_train || !logp_infer || !w_out) return CIS_ERR_NULL;
  DeviceInfo info;
  const int dev = current_device(&info);
  if (dev < 0) return dev;
  cis::WeightsArgs wa{logp_train, logp_infer, mask, w_out, trunc_out, T, lambda, kappa};
  return launch_grid_stride(cis::weights_kernel(), T, cis::kWeightsBlock, info, &wa, stream);
}

int cis_weights_ex(const float* logp_p, const float* logp_q, const uint8_t* mask, int64_t T,
                   const int64_t* seq_offsets, int64_t n_seq, const cis_params_t* params,
                   float* w_out, uint8_t* acted_out, float* eps_out, void* workspace,
                   size_t workspace_bytes, hipStream_t stream) {
  if (T < 0 || n_seq < 0) return CIS_ERR_SHAPE;
  if (int rc = check_op_params(params, false)) return rc;
  const bool seq = is_seq_op(params->op);
  if (seq && T > 0 && n_seq < 1) return CIS_ERR_SHAPE;
  if (!workspace) return CIS_ERR_NULL;
  if (T > 0 && (!logp_p || !logp_q || !w_out || (seq && !seq_offsets))) return CIS_ERR_NULL;
  if (!aligned(workspace, 256)) return CIS_ERR_ALIGN;
  const cis::WsLayout L = cis::ws_layout(T, seq ? n_seq : 0);
  if (workspace_bytes < L.total) return CIS_ERR_WORKSPACE;
  DeviceInfo info;
  const int dev = current_device(&info);
  if (dev < 0) return dev;
  const Ws ws{static_cast<char*>(workspace), L};
  if (T > 0) {
    if (seq) {
      if (int rc = launch_seq_sum(logp_p, logp_q, mask, nullptr, 1, seq_offsets, n_seq, T, ws,
                                  stream))
        return rc;
    }
    cis::PrepassArgs pa{};
    pa.logp_p = logp_p;
    pa.logp_q = logp_q;
    pa.mask = mask;
    pa.offsets = seq_offsets;
    pa.logK = reinterpret_cast<const double*>(ws.base + L.logK);
    pa.ops = op_args(*params);
    pa.T = T;
    pa.n_seq = seq ? n_seq : 0;
    pa.V = 1;
    pa.w_out = w_out;
    pa.acted_out = acted_out;
    pa.eps_out = eps_out;
    pa.logk_ws = ws.f(L.logk);
    pa.excess_ws = ws.f(L.excess);
    pa.flags_ws = ws.b(L.flags);
    pa.terms_ws = ws.f(L.terms);
    if (int rc = launch_grid_stride(cis::prepass_kernel(), T, cis::kWeightsBlock, info, &pa,
                                    stream))
      return rc;
  }
  cis::FinalizeArgs fa{ws.f(L.terms), ws.b(L.flags), ws.f(L.logk), ws.f(L.excess), T,
                       ws.stats(), nullptr};
  return launch(cis::finalize_kernel(), 1, cis::kFinalizeBlock, &fa, stream);
}

int cis_loss_fwd(const void* logits, int dtype, int64_t T, int64_t V, int64_t ld,
                 const int64_t* ids, const float* logp_infer, const float* adv,
                 const uint8_t* mask, float lambda, float kappa, float scale,
                 float* logp_train_out, float* w_out, uint8_t* trunc_out,
                 float* loss_terms_out, float* loss_out, void* workspace,
                 size_t workspace_bytes, hipStream_t stream) {
  return run_loss(base_call(false, logits, dtype, T, V, ld, ids, logp_infer, adv, mask, lambda,
                            kappa, scale, nullptr, 0, logp_train_out, w_out, trunc_out,
                            loss_terms_out, loss_out, workspace, workspace_bytes),
                  stream);
}

int cis_loss_bwd(const void* logits, int dtype, int64_t T, int64_t V, int64_t ld,
                 const int64_t* ids, const float* logp_infer, const float* adv,
                 const uint8_t* mask, float lambda, float kappa, float scale, void* dlogits,
                 int64_t ld_g, float* logp_train_out, float* w_out, uint8_t* trunc_out,
                 float* loss_terms_out, float* loss_out, void* workspace,
                 size_t workspace_bytes, hipStream_t stream) {
  return run_loss(base_call(true, logits, dtype, T, V, ld, ids, logp_infer, adv, mask, lambda,
                            kappa, scale, dlogits, ld_g, logp_train_out, w_out, trunc_out,
                            loss_terms_out, loss_out, workspace, workspace_bytes),
                  stream);
}

int cis_loss_bwd_noalloc(const void* logits, int dtype, int64_t T, int64_t V, int64_t ld,
                         const int64_t* ids, const float* logp_infer, const float* adv,
                         const uint8_t* mask, float lambda, float kappa, float scale,
                         void* dlogits, int64_t ld_g, float* logp_train_out, float* w_out,
                         uint8_t* trunc_out, float* loss_terms_out, float* loss_out,
                         cis_stats_t* stats_out, hipStream_t stream) {
  if (T > CIS_NOALLOC_MAX_T) return CIS_ERR_SCRATCH;
  if (T < 0) return CIS_ERR_SHAPE;
  // the device check comes before the scratch lookup (the lookup needs a gfx950 device)
  DeviceInfo info;
  const int dev = current_device(&info);
  if (dev < 0) return dev;
  void* ws = nullptr;
  if (int rc = scratch_on(dev, &ws)) return rc;
  LossCall c = base_call(true, logits, dtype, T, V, ld, ids, logp_infer, adv, mask, lambda, kappa,
                         scale, dlogits, ld_g, logp_train_out, w_out, trunc_out, loss_terms_out,
                         loss_out, ws, kScratchBytes);
  c.stats_out = stats_out;
  return run_loss(c, stream);
}

int cis_loss_fwd_ex(const void* logits, int dtype, int64_t T, int64_t V, int64_t ld,
                    const int64_t* ids, const float* logp_infer, const float* logp_old,
                    const float* adv, const uint8_t* mask, const int64_t* seq_offsets,
                    int64_t n_seq, const cis_params_t* params, float* logp_train_out,
                    float* w_out, uint8_t* acted_out, float* loss_terms_out, float* eps_out,
                    float* loss_out, void* workspace, size_t workspace_bytes,
                    hipStream_t stream) {
  if (!params) return CIS_ERR_NULL;
  return run_loss(ext_call(false, logits, dtype, T, V, ld, ids, logp_infer, logp_old, adv, mask,
                           seq_offsets, n_seq, params, nullptr, 0, logp_train_out, w_out,
                           acted_out, loss_terms_out, eps_out, loss_out, workspace,
                           workspace_bytes),
                  stream);
}

int cis_loss_bwd_ex(const void* logits, int dtype, int64_t T, int64_t V, int64_t ld,
                    const int64_t* ids, const float* logp_infer, const float* logp_old,
                    const float* adv, const uint8_t* mask, const int64_t* seq_offsets,
                    int64_t n_seq, const cis_params_t* params, void* dlogits, int64_t ld_g,
                    float* logp_train_out, float* w_out, uint8_t* acted_out,
                    float* loss_terms_out, float* eps_out, float* loss_out, void* workspace,
                    size_t workspace_bytes, hipStream_t stream) {
  if (!params) return CIS_ERR_NULL;
  return run_loss(ext_call(true, logits, dtype, T, V, ld, ids, logp_infer, logp_old, adv, mask,
                           seq_offsets, n_seq, params, dlogits, ld_g, logp_train_out, w_out,
                           acted_out, loss_terms_out, eps_out, loss_out, workspace,
                           workspace_bytes),
                  stream);
}

}  // extern "C"
