// Internal declarations shared by the library's translation units.
#pragma once

#include <stdint.h>

#include <string>

#include "surge.h"

namespace surge {

// Thread-local error message of the last failing call.
surge_status fail(surge_status code, const char* fmt, ...);
void clear_error();

// SuperBatch formation (Alg. 1), host only.  Appends to the output vectors.
struct PlanSB {
  int64_t text_begin, text_end, seg_begin, seg_end;
};
struct PlanSeg {
  int64_t first_text, count, row_offset;
  int32_t partition;
};
surge_status plan_superbatches(const int64_t* part_offsets, int32_t n_parts, int64_t b_min,
                               int64_t n_max, int32_t policy, void (*emit_sb)(void*, const PlanSB&),
                               void (*emit_seg)(void*, const PlanSeg&), void* ctx,
                               int64_t* n_sbs, int64_t* n_segs);

// Host-side check of an encoder description.
surge_status validate_desc(const surge_encoder_desc* desc);

// bf16 bits of a float, nearest value with ties to even (host side).
uint16_t f32_to_bf16_rne(float f);

}  // namespace surge
