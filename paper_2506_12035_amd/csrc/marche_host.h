// Host-side internals shared by the C-ABI translation units of libmarche.so
// (not part of the public ABI, which is include/marche.h).
#pragma once

#include "../../include/marche.h"

namespace marche {

// Records a formatted message for marche_last_error() and returns s.
marche_status_t set_error(marche_status_t s, const char *fmt, ...)
    __attribute__((format(printf, 2, 3)));

// The decoder step on images [first_image, first_image + batch) of the
// cache, with the caller's workspace: the body of marche_step and
// marche_step_images (validation, then the per-layer launch sequence).
marche_status_t step_impl(const marche_model_t *m, const marche_layer_t *layers,
                          const marche_kv_cache_t *cache, int32_t first_image, int32_t layer_begin,
                          int32_t layer_end, int32_t batch, float *x, const int32_t *a_idx,
                          const int32_t *a_off, const int32_t *n_gen, int32_t a_total,
                          int32_t a_max, int32_t gen_max, float *scores, int32_t score_layer,
                          void *workspace, size_t workspace_bytes, marche_stream_t stream);

}  // namespace marche
