// Host interface of the edge-local MLP message over the generated radius relation.
#pragma once

#include "common.hpp"

namespace tiga {
namespace edgenn {

constexpr int kMaxFeat = 64;
constexpr int kMaxHidden = 64;
constexpr int kMaxOut = 8;

struct Net {
    int32_t feat, hidden, out;
    const float *W1, *b1, *W2, *b2;   // [hidden][3 + feat], [hidden], [out][hidden], [out]
};

struct Grads {
    float *dx, *dpos, *dW1, *db1, *dW2, *db2;   // each may be null
};

size_t workspace_bytes(int64_t n, const Net &net);
int forward(int64_t n, const float *pos, const float *x, float radius, const Net &net, float *y, void *ws,
            hipStream_t stream);
int backward(int64_t n, const float *pos, const float *x, float radius, const Net &net, const float *dy,
             const Grads &g, void *ws, hipStream_t stream);

}  // namespace edgenn
}  // namespace tiga
