// Host interface of the generated exact kNN relation.
#pragma once

#include "common.hpp"

namespace tiga {
namespace knn {

constexpr int kMaxK = 32;

size_t workspace_bytes(int64_t n);
// Arguments validated by the caller: 0 <= k <= kMaxK, x/y present when feat > 0.
int forward(int64_t n, int32_t feat, const float *pos, const float *x, int32_t k, float *y, int32_t *nbr, void *ws,
            hipStream_t stream);

}  // namespace knn
}  // namespace tiga
