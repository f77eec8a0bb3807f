// Internal launchers shared between translation units of the library.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

int ptd_launch_tree_mask(const int32_t* parent, const int32_t* tree_len, int B, int T,
                         uint64_t* mask, int32_t* depth, int32_t* dev_status,
                         hipStream_t stream);
