// Library-internal hooks between the step context (maskstep.hip) and the
// static-scratch entry point (noalloc.hip).
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "../../include/maskstep.h"

namespace ms {

// Records the calling thread's error message (mask_last_error) and returns `st`.
ms_status set_error(ms_status st, const char* fmt, ...);

// Bytes of workspace a step over `batch` requests of `desc` needs (*need), after
// the validation mask_workspace_bytes does.
ms_status workspace_need(const ms_model_desc* desc, int32_t batch, size_t* need);

// mask_step_init over the workspace `ws`; `static_dev` >= 0 marks a context that
// holds that device's static scratch (released by mask_step_destroy).
ms_status step_init(ms_step** out, const ms_model_desc* desc, int32_t batch, const uint8_t* d_mask,
                    void* ws, size_t ws_bytes, void* stream, int static_dev);

// Gives device `dev`'s static scratch back (noalloc.hip).
void release_static_scratch(int dev);

}  // namespace ms
