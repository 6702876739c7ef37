// Host-side helpers of the C ABI: status strings, workspace sizes, budgets from
// ratios (Eq. dcut-budget), nearest captured batch (App. C), profiling hook.
#include "dcut_internal.h"

namespace dcut {
size_t layer_ws_bytes(const dcut_layer_cfg *c, int B, int D);
size_t lmhead_ws_bytes(int H, int V, int B, int D);
size_t accept_rs_ws_bytes(int V, int B);

ProfileHook &profile_hook() {
  static thread_local ProfileHook h = {DCUT_KERNEL_NONE, nullptr, nullptr};
  return h;
}
}  // namespace dcut

using namespace dcut;

extern "C" const char *dcut_strerror(int status) {
  switch (status) {
    case DCUT_OK: return "ok";
    case DCUT_EINVAL: return "invalid argument";
    case DCUT_EUNSUPPORTED: return "unsupported shape or configuration";
    case DCUT_EWORKSPACE: return "workspace missing, misaligned or too small";
    case DCUT_EHIP: return "HIP launch or runtime error";
  }
  return "unknown status";
}

extern "C" size_t dcut_workspace_bytes(int which, const dcut_layer_cfg *cfg, int B, int D) {
  if (!batch_ok(B, D)) return (size_t)-1;
  switch (which) {
    case 0: return 0;
    case 1: return layer_ws_bytes(cfg, B, D);
    case 2:
      if (!cfg || cfg->hidden <= 0 || cfg->hidden % 8 || cfg->vocab <= 0) return (size_t)-1;
      return lmhead_ws_bytes(cfg->hidden, cfg->vocab, B, D);
    case 3: return 0;
    case 4:
      if (!cfg || cfg->vocab <= 0) return (size_t)-1;
      return accept_rs_ws_bytes(cfg->vocab, B);
  }
  return (size_t)-1;
}

extern "C" int dcut_budgets_from_ratios(int B, int D, int R, const int32_t *num, const int32_t *den,
                                        int32_t *out) {
  if (!batch_ok(B, D) || R < 1 || R > DCUT_MAX_CANDIDATES || !num || !den || !out) return DCUT_EINVAL;
  const long long total = (long long)B * (D + 1);
  for (int r = 0; r < R; ++r) {
    if (den[r] <= 0 || num[r] < 0 || num[r] > den[r]) return DCUT_EINVAL;
  }
  for (int r = 0; r < R; ++r) {
    long long k = (num[r] * total + den[r] - 1) / den[r];   // exact ceiling, num*total >= 0
    out[r] = (int32_t)(k < B ? B : k);
  }
  return DCUT_OK;
}

extern "C" int dcut_nearest_batch(int B, int n, const int32_t *captured) {
  if (n < 1 || !captured) return -1;
  int best = 0;
  for (int j = 1; j < n; ++j) {
    long long dj = captured[j] > B ? (long long)captured[j] - B : (long long)B - captured[j];
    long long db = captured[best] > B ? (long long)captured[best] - B : (long long)B - captured[best];
    if (dj < db || (dj == db && captured[j] > captured[best])) best = j;
  }
  return best;
}

extern "C" int dcut_profile_arm(int kernel, hipEvent_t start, hipEvent_t stop) {
  if (kernel < DCUT_KERNEL_NONE || kernel > DCUT_KERNEL_ATTN_PLAN) return DCUT_EINVAL;
  if (kernel != DCUT_KERNEL_NONE && (!start || !stop)) return DCUT_EINVAL;
  ProfileHook &h = profile_hook();
  h.kernel = kernel;
  h.start = start;
  h.stop = stop;
  return DCUT_OK;
}
