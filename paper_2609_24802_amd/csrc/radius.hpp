// Host interface of the generated radius relation.
#pragma once

#include "common.hpp"

namespace tiga {
namespace radius {

size_t workspace_bytes(int64_t n, int64_t feat);
int forward(int64_t n, int32_t feat, const float *pos, const float *x, float radius, float sigma, float *y,
            int32_t *count, void *ws, hipStream_t stream);
int backward(int64_t n, int32_t feat, const float *pos, const float *x, float radius, float sigma, const float *dy,
             float *dx, float *dpos, void *ws, hipStream_t stream);
int neighbors(int64_t n, const float *pos, float radius, const int64_t *nbr_ptr, int32_t *nbr_idx, void *ws,
              hipStream_t stream);

}  // namespace radius
}  // namespace tiga
