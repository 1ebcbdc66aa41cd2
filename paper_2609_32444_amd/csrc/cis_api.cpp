// C-ABI entry points of libcis: argument validation, launch configuration and launches on the
// caller's stream. No device memory is allocated and nothing synchronises.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>
#include <string.h>

#include <mutex>

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

int loss_common(bool bwd, const void* logits, int dtype, int64_t T, int64_t V, int64_t ld,
                const int64_t* ids, const float* logp_infer, const float* adv,
                const uint8_t* mask, float lam, float kappa, float scale, void* dlogits,
                int64_t ld_g, float* logp_train_out, float* w_out, uint8_t* trunc_out,
                float* loss_terms_out, float* loss_out, void* workspace, size_t workspace_bytes,
                hipStream_t stream) {
  if (dtype != CIS_BF16 && dtype != CIS_F32) return CIS_ERR_DTYPE;
  if (T < 0 || V < 1 || ld < V || (bwd && ld_g < V)) return CIS_ERR_SHAPE;
  const int esize = dtype == CIS_BF16 ? 2 : 4;
  const int epv = 16 / esize;
  if (V > kMaxV) return CIS_ERR_SHAPE;  // row byte offsets stay within 32 bits
  if (ld > INT64_MAX / esize || (bwd && ld_g > INT64_MAX / esize)) return CIS_ERR_SHAPE;
  if (int rc = check_params(lam, kappa, scale)) return rc;
  if (!workspace) return CIS_ERR_NULL;
  if (T > 0 && (!logits || !ids || !logp_infer || !adv || (bwd && !dlogits))) return CIS_ERR_NULL;
  if (!aligned(workspace, 256)) return CIS_ERR_ALIGN;
  if (workspace_bytes < cis::ws_bytes(T)) return CIS_ERR_WORKSPACE;
  if (T > 0) {
    if (!aligned(logits, 16) || (ld * esize) % 16 != 0) return CIS_ERR_ALIGN;
    if (bwd) {
      if (!aligned(dlogits, 16) || (ld_g * esize) % 16 != 0) return CIS_ERR_ALIGN;
      const uintptr_t a0 = (uintptr_t)logits, a1 = a0 + (uintptr_t)(T * ld * esize);
      const uintptr_t b0 = (uintptr_t)dlogits, b1 = b0 + (uintptr_t)(T * ld_g * esize);
      if (a0 == b0) {
        if (ld_g != ld) return CIS_ERR_ALIAS;
      } else if (a0 < b1 && b0 < a1) {
        return CIS_ERR_ALIAS;
      }
    }
  }
  DeviceInfo info;
  const int dev = current_device(&info);
  if (dev < 0) return dev;

  char* ws = static_cast<char*>(workspace);
  float* terms_ws = reinterpret_cast<float*>(ws + cis::ws_terms_offset());
  uint8_t* flags_ws = reinterpret_cast<uint8_t*>(ws + cis::ws_flags_offset(T));

  if (T > 0) {
    const int32_t nvec = (int32_t)((V + epv - 1) / epv);
    const cis::RowVariant& var = cis::select_row_variant(dtype, bwd, nvec);
    cis::RowArgs ra;
    ra.logits = logits;
    ra.dlogits = dlogits;
    ra.row_bytes = ld * esize;
    ra.grow_bytes = bwd ? ld_g * esize : 0;
    ra.ids = ids;
    ra.logp_infer = logp_infer;
    ra.adv = adv;
    ra.mask = mask;
    ra.logp_train_out = logp_train_out;
    ra.w_out = w_out;
    ra.trunc_out = trunc_out;
    ra.terms_user = loss_terms_out;
    ra.terms_ws = terms_ws;
    ra.flags_ws = flags_ws;
    ra.T = T;
    ra.V = (int32_t)V;
    ra.nvec = nvec;
    ra.lam = lam;
    ra.kappa = kappa;
    ra.scale = scale;
    const int per_cu = blocks_per_cu(var.fn, var.block, dev);
    const int64_t resident = (int64_t)per_cu * info.num_cu;
    const int grid = (int)(T < resident ? T : resident);
    if (int rc = launch(var.fn, grid, var.block, &ra, stream)) return rc;
  }
  cis::FinalizeArgs fa{terms_ws, flags_ws, T, reinterpret_cast<cis_stats_t*>(ws), loss_out};
  return launch(cis::finalize_kernel(), 1, cis::kFinalizeBlock, &fa, stream);
}

}  // namespace

extern "C" {

size_t cis_workspace_bytes(int64_t T) { return T < 0 ? 0 : cis::ws_bytes(T); }

const char* cis_status_string(int status) {
  switch (status) {
    case CIS_OK: return "ok";
    case CIS_ERR_NULL: return "a required pointer is NULL";
    case CIS_ERR_SHAPE: return "invalid shape (T < 0, V outside [1, 2^28], or a row stride < V)";
    case CIS_ERR_DTYPE: return "unknown dtype";
    case CIS_ERR_PARAM:
      return "invalid parameter (lambda must be finite and >= 0, kappa in [0,1], scale finite)";
    case CIS_ERR_ALIGN:
      return "misaligned buffer (logits/dlogits base and row stride must be 16-byte multiples; "
             "workspace 256-byte aligned)";
    case CIS_ERR_LAUNCH: return "kernel launch failed";
    case CIS_ERR_WORKSPACE: return "workspace too small (see cis_workspace_bytes)";
    case CIS_ERR_ALIAS: return "dlogits overlaps logits other than exactly in place (ld_g == ld)";
    case CIS_ERR_DEVICE: return "current device is not a gfx950 GPU";
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
  const int64_t need = (T + cis::kWeightsBlock - 1) / cis::kWeightsBlock;
  const int64_t cap = (int64_t)info.num_cu * 8;
  return launch(cis::weights_kernel(), (int)(need < cap ? need : cap), cis::kWeightsBlock, &wa,
                stream);
}

int cis_loss_fwd(const void* logits, int dtype, int64_t T, int64_t V, int64_t ld,
                 const int64_t* ids, const float* logp_infer, const float* adv,
                 const uint8_t* mask, float lambda, float kappa, float scale,
                 float* logp_train_out, float* w_out, uint8_t* trunc_out,
                 float* loss_terms_out, float* loss_out, void* workspace,
                 size_t workspace_bytes, hipStream_t stream) {
  return loss_common(false, logits, dtype, T, V, ld, ids, logp_infer, adv, mask, lambda, kappa,
                     scale, nullptr, 0, logp_train_out, w_out, trunc_out, loss_terms_out,
                     loss_out, workspace, workspace_bytes, stream);
}

int cis_loss_bwd(const void* logits, int dtype, int64_t T, int64_t V, int64_t ld,
                 const int64_t* ids, const float* logp_infer, const float* adv,
                 const uint8_t* mask, float lambda, float kappa, float scale, void* dlogits,
                 int64_t ld_g, float* logp_train_out, float* w_out, uint8_t* trunc_out,
                 float* loss_terms_out, float* loss_out, void* workspace,
                 size_t workspace_bytes, hipStream_t stream) {
  return loss_common(true, logits, dtype, T, V, ld, ids, logp_infer, adv, mask, lambda, kappa,
                     scale, dlogits, ld_g, logp_train_out, w_out, trunc_out, loss_terms_out,
                     loss_out, workspace, workspace_bytes, stream);
}

}  // extern "C"
