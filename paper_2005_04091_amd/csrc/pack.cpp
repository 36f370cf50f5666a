// Host-side CSR packing of a dense-stored sparse filter (spconv_pack_csr).
//
// Paper, "Sparse Convolution with CSR": the (K, C, k, k) filter is flattened to a
// K x (C*k*k) matrix whose rows are compressed. Each entry keeps its flattened
// column and, for the GPU kernel, the column lowered to an offset inside one
// zero-padded C x Hp x Wp input image (the `off` the paper's loop adds to the
// output position).
#include <cstdint>
#include <cstring>
#include <limits>

#include "dense_layout.h"
#include "spconv.h"

namespace {

// Entry rule: with a mask, a nonzero mask byte (explicit 0.0 values are kept);
// without one, a value unequal to 0.0f (-0.0 dropped, NaN kept).
inline bool is_entry(const float *w, const uint8_t *mask, size_t i) {
    return mask ? mask[i] != 0 : w[i] != 0.0f;
}

constexpr int64_t kI32Max = std::numeric_limits<int32_t>::max();

}  // namespace

extern "C" int spconv_pack_csr(const float *w, const uint8_t *mask, int K, int C, int R, int S, int Hp, int Wp,
                               int32_t *rowptr, int32_t *colidx, int32_t *offset, float *vals, int64_t capacity,
                               int64_t *nnz_out) {
    if (!w || !nnz_out) return SPCONV_EINVAL;
    if (K < 1 || C < 1 || R < 1 || S < 1 || Hp < R || Wp < S) return SPCONV_EINVAL;
    const bool any_out = colidx || offset || vals;
    const bool all_out = colidx && offset && vals;
    if (any_out && (!all_out || !rowptr || capacity < 0)) return SPCONV_EINVAL;
    const int64_t taps = (int64_t)C * R * S;
    const int64_t plane = (int64_t)Hp * Wp;
    if (taps > kI32Max || (int64_t)(C - 1) * plane + (int64_t)(R - 1) * Wp + (S - 1) > kI32Max)
        return SPCONV_EINVAL;

    // Count pass (also fills rowptr when given).
    int64_t nnz = 0;
    if (rowptr) rowptr[0] = 0;
    for (int k = 0; k < K; ++k) {
        const size_t row = (size_t)k * (size_t)taps;
        for (int64_t t = 0; t < taps; ++t) nnz += is_entry(w, mask, row + (size_t)t) ? 1 : 0;
        if (nnz > kI32Max) return SPCONV_EINVAL;
        if (rowptr) rowptr[k + 1] = (int32_t)nnz;
    }
    *nnz_out = nnz;
    if (!all_out) return SPCONV_OK;
    if (nnz > capacity) return SPCONV_ECAPACITY;

    // Fill pass: columns in increasing (c, r, s) order within each row.
    int64_t j = 0;
    for (int k = 0; k < K; ++k) {
        const size_t row = (size_t)k * (size_t)taps;
        int32_t col = 0;
        for (int c = 0; c < C; ++c) {
            const int32_t cbase = (int32_t)((int64_t)c * plane);
            for (int r = 0; r < R; ++r) {
                for (int s = 0; s < S; ++s, ++col) {
                    if (!is_entry(w, mask, row + (size_t)col)) continue;
                    colidx[j] = col;
                    offset[j] = cbase + r * Wp + s;
                    std::memcpy(&vals[j], &w[row + (size_t)col], sizeof(float));
                    ++j;
                }
            }
        }
    }
    return SPCONV_OK;
}

extern "C" int spconv_dense_size(int K, int C, int R, int S, int64_t *floats) {
    if (!floats || K < 1 || C < 1 || R < 1 || S < 1) return SPCONV_EINVAL;
    const long long v = (long long)((C + 1) / 2) * R * S * dense_layout::kp(K) * 2;
    if (v >= (1LL << 40)) return SPCONV_EINVAL;
    *floats = v;
    return SPCONV_OK;
}

extern "C" int spconv_pack_dense(const float *w, const uint8_t *mask, int K, int C, int R, int S, float *packed,
                                 int64_t packed_len) {
    if (!w || !packed) return SPCONV_EINVAL;
    int64_t need = 0;
    const int rc = spconv_dense_size(K, C, R, S, &need);
    if (rc != SPCONV_OK) return rc;
    if (packed_len < need) return SPCONV_ECAPACITY;
    const int64_t RS = (int64_t)R * S;
    const int64_t Kp = need / ((int64_t)((C + 1) / 2) * RS * 2);
    std::memset(packed, 0, (size_t)need * sizeof(float));
    for (int k = 0; k < K; ++k)
        for (int c = 0; c < C; ++c)
            for (int64_t t = 0; t < RS; ++t) {
                const size_t i = ((size_t)k * C + c) * (size_t)RS + (size_t)t;
                if (!is_entry(w, mask, i)) continue;
                packed[(((int64_t)(c / 2) * RS + t) * Kp + k) * 2 + (c & 1)] = w[i];
            }
    return SPCONV_OK;
}
