// C entry points of the attention path: argument validation on the host,
// workspace sizing, then the launchers of attn_fwd.hip / attn_bwd.hip.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <mutex>
#include <vector>

#include "attn_common.h"
#include "errors.h"
#include "libra.h"

using namespace libra;

// Device scratch of libra_attn_fwd_noalloc: the forward's work-item
// workspace, one copy per device (each GPU the library runs on holds it until
// the process ends).  In host code `scratch` names a host-side stand-in: its
// device address comes from hipGetSymbolAddress, per device (scratch_ptr).
constexpr size_t kNoAllocScratchBytes = size_t(16) << 20;
static_assert(kNoAllocScratchBytes == LIBRA_FWD_NOALLOC_MAX_WORKSPACE, "documented limit");
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch[kMaxDevices] = {};

// Device address of `scratch` on the current device, looked up once per device.
int scratch_ptr(void **out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return fail(LIBRA_EHIP, "hipGetDevice failed");
  if (dev < 0 || dev >= kMaxDevices) return fail(LIBRA_EUNSUPPORTED, "device index %d", dev);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void *p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(LIBRA_EHIP, "hipGetSymbolAddress(scratch) failed: %s", hipGetErrorString(e));
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return LIBRA_OK;
}

constexpr int64_t kMaxRows = (int64_t(1) << 31) - 256;

int check_sizes(int64_t n, int64_t n_q, int64_t n_kv, int32_t h_q, int32_t h_kv, int32_t d) {
  if (h_q < 1 || h_kv < 1 || h_q % h_kv)
    return fail(LIBRA_EINVAL, "need h_q >= 1, h_kv >= 1, h_kv | h_q (got %d, %d)", h_q, h_kv);
  if (h_kv > 64) return fail(LIBRA_EUNSUPPORTED, "more than 64 KV heads");
  if (d != 64 && d != 128) return fail(LIBRA_EUNSUPPORTED, "head_dim %d (supported: 64, 128)", d);
  if (n < 1) return fail(LIBRA_EINVAL, "num_samples must be >= 1");
  if (n_q < 0 || n_kv < 1 || n_q > kMaxRows || n_kv > kMaxRows || n > kMaxRows)
    return fail(LIBRA_EINVAL, "row counts out of range");
  return LIBRA_OK;
}

int check_ws(const void *ws, size_t bytes, size_t need) {
  if (!ws) return fail(LIBRA_EINVAL, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(ws) % 256)
    return fail(LIBRA_EINVAL, "workspace must be 256-byte aligned");
  if (bytes < need)
    return fail(LIBRA_ENOSPC, "workspace of %zu bytes, need %zu", bytes, need);
  return LIBRA_OK;
}

// Per-thread event records of the main kernels (libra_timing_*).  The events
// are reused across enables and released with the process (destroying them
// from a thread-exit destructor could run after the HIP runtime is gone).
struct Timing {
  bool on = false;
  std::vector<KernelTimer> ev[3];
  size_t used[3] = {0, 0, 0};
};
Timing &timing() {
  static thread_local Timing t;
  return t;
}

// Next event pair for a main kernel, or nullptr when timing is off.
const KernelTimer *next_timer(int which, int *rc) {
  Timing &t = timing();
  *rc = LIBRA_OK;
  if (!t.on) return nullptr;
  auto &v = t.ev[which];
  if (t.used[which] == v.size()) {
    KernelTimer k;
    if (hipEventCreate(&k.begin) != hipSuccess || hipEventCreate(&k.end) != hipSuccess) {
      *rc = fail(LIBRA_EHIP, "hipEventCreate failed");
      return nullptr;
    }
    v.push_back(k);
  }
  return &v[t.used[which]++];
}

}  // namespace

extern "C" int libra_timing_enable(int enable) {
  Timing &t = timing();
  t.on = enable != 0;
  t.used[0] = t.used[1] = t.used[2] = 0;
  return LIBRA_OK;
}

extern "C" int libra_timing_read(int which, double *total_ms, int64_t *launches) {
  if (which < 0 || which > 2 || !total_ms || !launches)
    return fail(LIBRA_EINVAL, "libra_timing_read: which must be 0, 1 or 2, outputs non-NULL");
  Timing &t = timing();
  double sum = 0.0;
  for (size_t i = 0; i < t.used[which]; ++i) {
    const KernelTimer &k = t.ev[which][i];
    float ms = 0.f;
    if (hipEventSynchronize(k.end) != hipSuccess ||
        hipEventElapsedTime(&ms, k.begin, k.end) != hipSuccess)
      return fail(LIBRA_EHIP, "reading timing events failed");
    sum += ms;
  }
  *total_ms = sum;
  *launches = (int64_t)t.used[which];
  return LIBRA_OK;
}

extern "C" size_t libra_attn_workspace_size(int64_t num_tiles, int64_t num_samples,
                                            int64_t n_q_rows, int64_t n_kv_rows, int32_t h_q,
                                            int32_t h_kv, int32_t head_dim, int32_t backward) {
  if (num_tiles < 0 || check_sizes(num_samples, n_q_rows, n_kv_rows, h_q, h_kv, head_dim))
    return 0;
  if (backward)
    return bwd_layout(num_tiles, num_samples, n_q_rows, n_kv_rows, h_q, h_kv, head_dim).total;
  return fwd_layout(num_tiles, num_samples, n_q_rows, n_kv_rows, h_q, h_kv, head_dim).total;
}

extern "C" int libra_attn_fwd(const void *q, const void *k, const void *v,
                              const int64_t *cu_seqlens, int64_t num_samples,
                              const libra_tile_t *tiles, int64_t num_tiles, int64_t n_q_rows,
                              int64_t n_kv_rows, int32_t h_q, int32_t h_kv, int32_t head_dim,
                              float softmax_scale, void *o, float *lse, void *workspace,
                              size_t workspace_bytes, void *stream) {
  last_error_text().clear();
  if (int rc = check_sizes(num_samples, n_q_rows, n_kv_rows, h_q, h_kv, head_dim)) return rc;
  if (num_tiles < 0) return fail(LIBRA_EINVAL, "num_tiles < 0");
  if (num_tiles == 0) return LIBRA_OK;
  if (!q || !k || !v || !cu_seqlens || !tiles || !o || !lse)
    return fail(LIBRA_EINVAL, "NULL tensor argument");
  const FwdLayout L =
      fwd_layout(num_tiles, num_samples, n_q_rows, n_kv_rows, h_q, h_kv, head_dim);
  if (int rc = check_ws(workspace, workspace_bytes, L.total)) return rc;
  const float scale = softmax_scale > 0.f ? softmax_scale : 1.f / std::sqrt((float)head_dim);
  int rc = LIBRA_OK;
  const KernelTimer *tm = next_timer(0, &rc);
  if (rc) return rc;
  return launch_fwd(q, k, v, cu_seqlens, num_samples, tiles, num_tiles, n_q_rows, n_kv_rows, h_q,
                    h_kv, head_dim, scale, o, lse, workspace, L,
                    static_cast<hipStream_t>(stream), tm);
}

extern "C" int libra_attn_fwd_noalloc(const void *q, const void *k, const void *v,
                                      const int64_t *cu_seqlens, int64_t num_samples,
                                      const libra_tile_t *tiles, int64_t num_tiles,
                                      int64_t n_q_rows, int64_t n_kv_rows, int32_t h_q,
                                      int32_t h_kv, int32_t head_dim, float softmax_scale,
                                      void *o, float *lse, void *stream) {
  last_error_text().clear();
  if (int rc = check_sizes(num_samples, n_q_rows, n_kv_rows, h_q, h_kv, head_dim)) return rc;
  if (num_tiles < 0) return fail(LIBRA_EINVAL, "num_tiles < 0");
  if (num_tiles == 0) return LIBRA_OK;
  if (!q || !k || !v || !cu_seqlens || !tiles || !o || !lse)
    return fail(LIBRA_EINVAL, "NULL tensor argument");
  // no split K here: its partial slots would not fit the scratch
  const FwdLayout L =
      fwd_layout(num_tiles, num_samples, n_q_rows, n_kv_rows, h_q, h_kv, head_dim, false);
  if (L.total > kNoAllocScratchBytes)
    return fail(LIBRA_ENOSPC, "these sizes need %zu bytes of workspace, more than the %zu of "
                "the built-in scratch; use libra_attn_fwd with a workspace",
                L.total, kNoAllocScratchBytes);
  void *ws = nullptr;
  if (int rc = scratch_ptr(&ws)) return rc;
  const float scale = softmax_scale > 0.f ? softmax_scale : 1.f / std::sqrt((float)head_dim);
  int rc = LIBRA_OK;
  const KernelTimer *tm = next_timer(0, &rc);
  if (rc) return rc;
  return launch_fwd(q, k, v, cu_seqlens, num_samples, tiles, num_tiles, n_q_rows, n_kv_rows, h_q,
                    h_kv, head_dim, scale, o, lse, ws, L, static_cast<hipStream_t>(stream), tm);
}

extern "C" int libra_attn_skipped_tiles(const void *workspace, int32_t *count, void *stream) {
  last_error_text().clear();
  if (!workspace || !count) return fail(LIBRA_EINVAL, "NULL workspace or count");
  const hipStream_t st = static_cast<hipStream_t>(stream);
  int32_t v = 0;
  if (hipMemcpyAsync(&v, static_cast<const char *>(workspace) + LIBRA_WS_SKIPPED_OFFSET,
                     sizeof(v), hipMemcpyDeviceToHost, st) != hipSuccess ||
      hipStreamSynchronize(st) != hipSuccess)
    return fail(LIBRA_EHIP, "reading the skipped-tile count failed");
  *count = v;
  return LIBRA_OK;
}

extern "C" int libra_attn_bwd(const void *q, const void *k, const void *v, const void *o,
                              const float *lse, const void *dout, const int64_t *cu_seqlens,
                              int64_t num_samples, const libra_tile_t *tiles, int64_t num_tiles,
                              int64_t n_q_rows, int64_t n_kv_rows, int32_t h_q, int32_t h_kv,
                              int32_t head_dim, float softmax_scale, void *dq, void *dk,
                              void *dv, uint32_t flags, void *workspace, size_t workspace_bytes,
                              void *stream) {
  last_error_text().clear();
  if (int rc = check_sizes(num_samples, n_q_rows, n_kv_rows, h_q, h_kv, head_dim)) return rc;
  if (num_tiles < 0) return fail(LIBRA_EINVAL, "num_tiles < 0");
  if (flags & ~LIBRA_BWD_ACCUMULATE_DKV) return fail(LIBRA_EINVAL, "unknown flags 0x%x", flags);
  if (!dk || !dv) return fail(LIBRA_EINVAL, "NULL dk / dv");
  if (num_tiles > 0 && (!q || !k || !v || !o || !lse || !dout || !cu_seqlens || !tiles || !dq))
    return fail(LIBRA_EINVAL, "NULL tensor argument");
  const BwdLayout L =
      bwd_layout(num_tiles, num_samples, n_q_rows, n_kv_rows, h_q, h_kv, head_dim);
  if (num_tiles > 0)
    if (int rc = check_ws(workspace, workspace_bytes, L.total)) return rc;
  const float scale = softmax_scale > 0.f ? softmax_scale : 1.f / std::sqrt((float)head_dim);
  int rc = LIBRA_OK;
  const KernelTimer *tm_kv = num_tiles > 0 ? next_timer(1, &rc) : nullptr;
  if (rc) return rc;
  const KernelTimer *tm_q = num_tiles > 0 ? next_timer(2, &rc) : nullptr;
  if (rc) return rc;
  return launch_bwd(q, k, v, o, lse, dout, cu_seqlens, num_samples, tiles, num_tiles, n_q_rows,
                    n_kv_rows, h_q, h_kv, head_dim, scale, dq, dk, dv,
                    (flags & LIBRA_BWD_ACCUMULATE_DKV) != 0, workspace, L,
                    static_cast<hipStream_t>(stream), tm_kv, tm_q);
}
