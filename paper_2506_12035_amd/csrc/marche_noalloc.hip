// marche_step_images_noalloc: the decoder step with a library-owned
// workspace, for callers that cannot allocate device memory.  The workspace
// is a file-scope static device array; host code never passes the array's
// own name to a kernel or a copy (on the host it is a stand-in, not a device
// address), only the address hipGetSymbolAddress returns for the current
// device, looked up once per device.
#include <hip/hip_runtime.h>

#include <mutex>

#include "../../include/marche.h"
#include "marche_host.h"

namespace {

static __device__ __align__(256) unsigned char scratch[MARCHE_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void *g_scratch[kMaxDevices];  // device address of `scratch` per device, once looked up

}  // namespace

extern "C" marche_status_t marche_step_images_noalloc(
    const marche_model_t *m, const marche_layer_t *layers, const marche_kv_cache_t *cache,
    int32_t first_image, int32_t layer_begin, int32_t layer_end, int32_t batch, float *x,
    const int32_t *a_idx, const int32_t *a_off, const int32_t *n_gen, int32_t a_total,
    int32_t a_max, int32_t gen_max, float *scores, int32_t score_layer, marche_stream_t stream) {
  // host-only checks first: the size needed, before any HIP call
  const size_t need = marche_step_workspace_bytes(m, batch, a_total);
  if (need > MARCHE_SCRATCH_BYTES)
    return marche::set_error(MARCHE_ERR_WORKSPACE,
                             "step needs %zu bytes of workspace > MARCHE_SCRATCH_BYTES = %zu "
                             "(a_total=%d)",
                             need, MARCHE_SCRATCH_BYTES, a_total);
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess)
    return marche::set_error(MARCHE_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices)
    return marche::set_error(MARCHE_ERR_UNSUPPORTED, "device %d outside [0, %d)", dev, kMaxDevices);
  void *ws = nullptr;
  {
    std::lock_guard<std::mutex> lk(g_mu);
    if (!g_scratch[dev]) {
      void *p = nullptr;
      e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
      if (e != hipSuccess || !p)
        return marche::set_error(MARCHE_ERR_HIP, "hipGetSymbolAddress(scratch) on device %d: %s",
                                 dev, hipGetErrorString(e));
      g_scratch[dev] = p;
    }
    ws = g_scratch[dev];
  }
  return marche::step_impl(m, layers, cache, first_image, layer_begin, layer_end, batch, x, a_idx,
                           a_off, n_gen, a_total, a_max, gen_max, scores, score_layer, ws,
                           MARCHE_SCRATCH_BYTES, stream);
}
