// Helpers shared by the HIP translation units of the library.
#pragma once

#include <hip/hip_runtime.h>

#include <algorithm>
#include <string>

#include "samd_internal.hpp"

namespace samd {

// Blocks for a grid-stride loop over `items`, capped so huge inputs loop instead.
inline int grid_for(int64_t items, int block) {
    int64_t blocks = (items + block - 1) / block;
    return (int)std::min<int64_t>(std::max<int64_t>(blocks, 1), 65536);
}

// Map a failed launch to SAMD_EHIP with the runtime's message.
inline int check_launch(const char *what) {
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) {
        set_error(std::string(what) + ": " + hipGetErrorString(e));
        return SAMD_EHIP;
    }
    return SAMD_OK;
}

// Expands MACRO(bits, signed) for every operand format.
#define SAMD_FOR_EACH_FMT(MACRO)                                                                    \
    MACRO(1, false) MACRO(2, false) MACRO(3, false) MACRO(4, false) MACRO(5, false) MACRO(6, false) \
    MACRO(7, false) MACRO(8, false) MACRO(1, true) MACRO(2, true) MACRO(3, true) MACRO(4, true)     \
    MACRO(5, true) MACRO(6, true) MACRO(7, true) MACRO(8, true)

}  // namespace samd
