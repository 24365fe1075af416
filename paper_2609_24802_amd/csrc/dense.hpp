// Host interface of the dense all-pairs relation.
#pragma once

#include "common.hpp"

namespace tiga {
namespace dense {

size_t workspace_bytes(int64_t n);
int forward(int64_t n, const float *pos, const float *q, float eps, float *y, void *ws, hipStream_t stream);

}  // namespace dense
}  // namespace tiga
