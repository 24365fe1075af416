// Host interface of the online-softmax reducer over an implicit triangular or dense relation.
#pragma once

#include "common.hpp"

namespace tiga {
namespace attention {

// dtype: TIGA_DT_F16 / TIGA_DT_BF16; relation: TIGA_REL_TRIANGULAR / TIGA_REL_DENSE.
// Arguments are validated by the caller; q, k, v, y are 16-byte aligned head-major [heads, n, width].
int forward(int64_t n, int32_t heads, int32_t width, int dtype, const void *q, const void *k, const void *v,
            float scale, int relation, void *y, float *lse, hipStream_t stream);

}  // namespace attention
}  // namespace tiga
