// C entry point of the online-softmax reducer over implicit triangular and dense relations.
#include "attention.hpp"

using namespace tiga;

extern "C" {

int tiga_mp_attention_fwd(int64_t n, int32_t heads, int32_t width, int dtype, const void *q, const void *k,
                          const void *v, float scale, int relation, void *y, float *lse, void *stream) {
    EntryScope scope;
    if (n < 0 || heads < 0) return fail(TIGA_EINVAL, "attention: negative size (n %lld, heads %d)", (long long)n, heads);
    if (dtype != TIGA_DT_F16 && dtype != TIGA_DT_BF16) return fail(TIGA_EINVAL, "attention: unknown dtype %d", dtype);
    if (relation != TIGA_REL_TRIANGULAR && relation != TIGA_REL_DENSE)
        return fail(TIGA_EINVAL, "attention: unknown relation %d", relation);
    if (!(scale > 0.0f) || !(scale < 3.0e38f)) return fail(TIGA_EINVAL, "attention: scale must be finite and > 0");
    if (width != 64 && width != 128) return fail(TIGA_EUNSUPPORTED, "attention: width %d (64 or 128 supported)", width);
    if (n >= (int64_t(1) << 31)) return fail(TIGA_EUNSUPPORTED, "attention: n = %lld needs n < 2^31", (long long)n);
    if (n * static_cast<int64_t>(heads) >= (int64_t(1) << 40))
        return fail(TIGA_EUNSUPPORTED, "attention: heads * n must be < 2^40");
    if (n == 0 || heads == 0) return TIGA_OK;
    if (!q || !k || !v || !y) return fail(TIGA_EINVAL, "attention: q, k, v and y are required");
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(y))
        return fail(TIGA_EINVAL, "attention: q, k, v and y must be 16-byte aligned");
    if (lse && (reinterpret_cast<uintptr_t>(lse) & 3u)) return fail(TIGA_EINVAL, "attention: lse misaligned");
    return attention::forward(n, heads, width, dtype, q, k, v, scale, relation, y, lse,
                              static_cast<hipStream_t>(stream));
}

}  // extern "C"
