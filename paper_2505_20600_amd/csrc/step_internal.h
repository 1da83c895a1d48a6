// Library-internal hooks between the step context (maskstep.hip), the
// static-scratch entry point (noalloc.hip) and the cache-load planner
// (copyplan.hip).
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <vector>

#include "../../include/maskstep.h"

namespace ms {

// Records the calling thread's error message (mask_last_error) and returns `st`.
ms_status set_error(ms_status st, const char* fmt, ...);
// Clears the calling thread's error message; returns MS_OK.
ms_status clear_error();

// Bytes of workspace a step over `batch` requests of `desc` needs (*need), after
// the validation mask_workspace_bytes does.
ms_status workspace_need(const ms_model_desc* desc, int32_t batch, size_t* need);

// mask_step_init over the workspace `ws`; `static_dev` >= 0 marks a context that
// holds that device's static scratch (released by mask_step_destroy).
ms_status step_init(ms_step** out, const ms_model_desc* desc, int32_t batch, const uint8_t* d_mask,
                    void* ws, size_t ws_bytes, void* stream, int static_dev);

// Gives device `dev`'s static scratch back (noalloc.hip).
void release_static_scratch(int dev);

// One copy of a cache-load plan: image rows n0 + i * grid_w + [0, w) for
// i < h (one strided 2-D copy when h > 1; w < grid_w then).
struct CopyRect {
    int n0, w, h;
};

// The copies that load one request's cached rows (copyplan.hip): mask [H][P]
// (non-zero = masked), C = one copy command's cost in rows of link time;
// `strided` false: contiguous runs merged across short gaps only. Covers every
// unmasked row.
void plan_copies(const uint8_t* mask, int H, int P, double C, bool strided, std::vector<CopyRect>& out);

}  // namespace ms
