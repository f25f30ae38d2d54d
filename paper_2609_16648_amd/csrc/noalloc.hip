// gm_spec_accept_noalloc: the accept with no workspace argument and no allocation.  Its
// scratch is a file-scope device array of fixed size; each device the library runs on holds
// its own copy until the process ends.  The array's name is a host-side stand-in, so host code
// uses only the device address that hipGetSymbolAddress returns, looked up once per device on
// the first call there (with that device current).
#include <mutex>

#include "forward.h"

namespace {
constexpr size_t kScratchBytes = 16u << 20;   // 16 MiB: B = 256 rows of k = 7 at V = 151936 with top-p fit
constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_mu;
void *g_scratch[kMaxDevices];   // device address of `scratch` per device (null: not looked up yet)

// the device address of this device's scratch, or null (error message set)
void *scratch_ptr() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    (void)hipGetLastError();
    gm::set_error(GM_ERR_DEVICE, "gm_spec_accept_noalloc: no current device (or device %d beyond %d)", dev,
                  kMaxDevices);
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_scratch[dev]) {
    void *p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      (void)hipGetLastError();
      gm::set_error(GM_ERR_DEVICE, "gm_spec_accept_noalloc: hipGetSymbolAddress of the scratch failed: %s",
                    hipGetErrorString(e));
      return nullptr;
    }
    g_scratch[dev] = p;
  }
  return g_scratch[dev];
}
}  // namespace

extern "C" gm_status gm_spec_accept_noalloc(int B, int k, int V, int mode, float temperature, float top_p,
                                            const float *target_logits, const float *draft_logits,
                                            const gm_row_stats *target_stats, const gm_row_stats *draft_stats,
                                            const gm_nucleus *draft_nucleus, const int32_t *draft_tokens,
                                            const float *u_accept, const float *u_final, int32_t *n_accept,
                                            int32_t *out_tokens, const gm_record *record, void *stream) {
  // sizes are checked on the host before anything touches the device
  if (B < 0 || k < 0 || k > 15 || V < 1)
    return gm::set_error(GM_ERR_INVALID_ARG, "bad B=%d k=%d V=%d", B, k, V);
  if (B == 0) return GM_OK;
  const size_t need = gm::accept_workspace_bytes(B, k, V);
  if (need > kScratchBytes)
    return gm::set_error(GM_ERR_CAPACITY,
                         "gm_spec_accept_noalloc: B=%d k=%d V=%d needs %zu bytes of scratch; the fixed scratch holds %zu",
                         B, k, V, need, kScratchBytes);
  void *ws = scratch_ptr();
  if (!ws) return GM_ERR_DEVICE;
  // Nothing in the scratch has to start at zero: every region is written before it is read
  // within one call (histograms are cleared in LDS, partial sums fully written).
  return gm::spec_accept_impl(B, k, V, mode, temperature, top_p, target_logits, draft_logits, target_stats, draft_stats,
                              draft_nucleus, draft_tokens, u_accept, u_final, n_accept, out_tokens, record, ws,
                              kScratchBytes, stream);
}
