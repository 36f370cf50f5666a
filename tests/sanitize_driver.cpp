// Host-side driver run under AddressSanitizer and UndefinedBehaviorSanitizer
// by tests/test_sanitizers.py: the library's host packers (pack.cpp) and the
// C oracle, built with -fsanitize=address,undefined, on randomized shapes
// including empty rows, explicit zeros under a mask, -0.0, NaN, 1x1 filters,
// one-pixel planes and every error path of the packers. The CSR packer is
// compared bit for bit with the oracle's packer; the dense packer with a
// direct loop over its documented layout. Any sanitizer report aborts the
// process (-fno-sanitize-recover), any mismatch exits with status 1.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <random>
#include <vector>

#include "spconv.h"

extern "C" {
long long oracle_pack_csr(const float *w, const uint8_t *mask, int K, int C, int R, int S, int Hp, int Wp,
                          int32_t *rowptr, int32_t *colidx, int32_t *offset, float *vals);
int oracle_conv_res(const float *x, int N, int C, int H, int W, const float *w, const uint8_t *mask, int K, int R,
                    int S, const float *bias, const float *res, int stride, int pad, int relu, int pool,
                    const int32_t *pairs, int npairs, double *out, double *absacc, int nthreads);
void oracle_resize_bilinear(const float *x, int N, int C, int Hin, int Win, int H, int W, double *out,
                            double *weights_out);
}

static int failures = 0;
#define EXPECT(c)                                                     \
    do {                                                              \
        if (!(c)) {                                                   \
            std::fprintf(stderr, "FAILED %s at line %d\n", #c, __LINE__); \
            ++failures;                                               \
        }                                                             \
    } while (0)

static uint32_t bits(float f) {
    uint32_t u;
    std::memcpy(&u, &f, 4);
    return u;
}

int main() {
    std::mt19937 rng(2005);
    auto uni = [&](int lo, int hi) { return lo + (int)(rng() % (unsigned)(hi - lo + 1)); };
    auto unif = [&]() { return (float)((rng() >> 8) * (1.0 / 16777216.0)) * 2.0f - 1.0f; };
    int packed_cases = 0, conv_cases = 0;
    for (int it = 0; it < 200; ++it) {
        const int K = uni(1, 9), C = uni(1, 9), R = uni(1, 5), S = uni(1, 5);
        const int Hp = R + uni(0, 6), Wp = S + uni(0, 6);
        const double d = (it % 4 == 0) ? 0.0 : (it % 4 == 1 ? 0.05 : (it % 4 == 2 ? 0.4 : 1.0));
        const size_t n = (size_t)K * C * R * S;
        std::vector<float> w(n);
        std::vector<uint8_t> mask(n);
        for (size_t i = 0; i < n; ++i) {
            w[i] = unif();
            const unsigned r = rng() % 100;
            if (r < 8) w[i] = 0.0f;
            else if (r < 12) w[i] = -0.0f;
            else if (r < 14 && it % 3 == 0) w[i] = NAN;
            mask[i] = ((rng() % 1000) < d * 1000) ? 1 : 0;
        }
        if (K > 2)
            for (int j = 0; j < C * R * S; ++j) mask[(size_t)1 * C * R * S + j] = 0;  // an empty row
        for (int use_mask = 0; use_mask < 2; ++use_mask) {
            const uint8_t *m = use_mask ? mask.data() : nullptr;
            std::vector<int32_t> rp(K + 1), rp_o(K + 1), ci(n + 1), ci_o(n + 1), off(n + 1), off_o(n + 1);
            std::vector<float> va(n + 1), va_o(n + 1);
            int64_t nnz = -1;
            EXPECT(spconv_pack_csr(w.data(), m, K, C, R, S, Hp, Wp, rp.data(), nullptr, nullptr, nullptr, 0, &nnz) ==
                   SPCONV_OK);
            const long long nnz_o =
                oracle_pack_csr(w.data(), m, K, C, R, S, Hp, Wp, rp_o.data(), ci_o.data(), off_o.data(), va_o.data());
            EXPECT(nnz == nnz_o);
            if (nnz > 0) {
                std::vector<int32_t> small(nnz - 1 > 0 ? nnz - 1 : 1);
                std::vector<float> smallv(small.size());
                int64_t got = -1;
                EXPECT(spconv_pack_csr(w.data(), m, K, C, R, S, Hp, Wp, rp.data(), small.data(), small.data(),
                                       smallv.data(), nnz - 1, &got) == SPCONV_ECAPACITY);
                EXPECT(got == nnz);
            }
            // exact-capacity arrays, so an overrun is caught by the sanitizer
            std::vector<int32_t> ci_x(nnz > 0 ? nnz : 1), off_x(nnz > 0 ? nnz : 1);
            std::vector<float> va_x(nnz > 0 ? nnz : 1);
            int64_t nnz2 = -1;
            EXPECT(spconv_pack_csr(w.data(), m, K, C, R, S, Hp, Wp, rp.data(), ci_x.data(), off_x.data(), va_x.data(),
                                   nnz, &nnz2) == SPCONV_OK);
            EXPECT(nnz2 == nnz);
            for (int k = 0; k <= K; ++k) EXPECT(rp[k] == rp_o[k]);
            for (int64_t j = 0; j < nnz; ++j) {
                EXPECT(ci_x[j] == ci_o[j]);
                EXPECT(off_x[j] == off_o[j]);
                EXPECT(bits(va_x[j]) == bits(va_o[j]));
            }
            // dense packing against its documented layout
            int64_t fl = 0;
            EXPECT(spconv_dense_size(K, C, R, S, &fl) == SPCONV_OK);
            std::vector<float> pk(fl);
            EXPECT(spconv_pack_dense(w.data(), m, K, C, R, S, pk.data(), fl - 1) == SPCONV_ECAPACITY);
            EXPECT(spconv_pack_dense(w.data(), m, K, C, R, S, pk.data(), fl) == SPCONV_OK);
            const int64_t Kp = fl / ((int64_t)((C + 1) / 2) * R * S * 2);
            for (int64_t i = 0; i < fl; ++i) {
                const int64_t half = i % 2, k = (i / 2) % Kp, t = (i / 2 / Kp) % (R * S), cp = i / 2 / Kp / (R * S);
                const int64_t c = 2 * cp + half;
                float want = 0.0f;
                if (k < K && c < C) {
                    const size_t src = (((size_t)k * C + c) * R + t / S) * S + t % S;
                    const bool entry = m ? m[src] != 0 : w[src] != 0.0f;
                    if (entry) want = w[src];
                }
                EXPECT(bits(pk[i]) == bits(want));
            }
            ++packed_cases;
        }
        // error paths
        int64_t dummy = 0;
        EXPECT(spconv_pack_csr(nullptr, nullptr, K, C, R, S, Hp, Wp, nullptr, nullptr, nullptr, nullptr, 0, &dummy) ==
               SPCONV_EINVAL);
        EXPECT(spconv_pack_csr(w.data(), nullptr, K, C, R, S, R - 1, Wp, nullptr, nullptr, nullptr, nullptr, 0,
                               &dummy) == SPCONV_EINVAL);
        EXPECT(spconv_pack_csr(w.data(), nullptr, K, C, R, S, Hp, Wp, nullptr, nullptr, nullptr, nullptr, 0,
                               nullptr) == SPCONV_EINVAL);
    }
    // the oracle on small layers (any stride, pad, pool, residual), whole and by planes
    for (int it = 0; it < 60; ++it) {
        const int N = uni(1, 3), C = uni(1, 5), K = uni(1, 5), R = uni(1, 4), S = uni(1, 4);
        const int stride = uni(1, 3), pad = uni(0, 2);
        const int H = uni(1, 10), W = uni(1, 10);
        if (H + 2 * pad < R || W + 2 * pad < S) continue;
        const int Ho = (H + 2 * pad - R) / stride + 1, Wo = (W + 2 * pad - S) / stride + 1;
        const int pool = (Ho >= 2 && Wo >= 2) ? it % 2 : 0;
        std::vector<float> x((size_t)N * C * H * W), w((size_t)K * C * R * S), b(K), res((size_t)N * K * Ho * Wo);
        for (auto &v : x) v = unif();
        for (auto &v : w) v = (rng() % 3 == 0) ? unif() : 0.0f;
        for (auto &v : b) v = unif() * 0.1f;
        for (auto &v : res) v = unif();
        const int Hs = pool ? Ho / 2 : Ho, Ws = pool ? Wo / 2 : Wo;
        std::vector<double> out((size_t)N * K * Hs * Ws), ab(out.size());
        EXPECT(oracle_conv_res(x.data(), N, C, H, W, w.data(), nullptr, K, R, S, b.data(), it % 3 ? nullptr : res.data(),
                               stride, pad, 1, pool, nullptr, 0, out.data(), ab.data(), 2) == 0);
        std::vector<int32_t> pairs = {0, 0, N - 1, K - 1};
        std::vector<double> out2((size_t)2 * Hs * Ws), ab2(out2.size());
        EXPECT(oracle_conv_res(x.data(), N, C, H, W, w.data(), nullptr, K, R, S, b.data(), nullptr, stride, pad, 0,
                               pool, pairs.data(), 2, out2.data(), ab2.data(), 1) == 0);
        ++conv_cases;
    }
    for (int it = 0; it < 20; ++it) {
        const int N = uni(1, 2), C = uni(1, 3), Hin = uni(1, 12), Win = uni(1, 12), H = uni(1, 12), W = uni(1, 12);
        std::vector<float> x((size_t)N * C * Hin * Win);
        for (auto &v : x) v = unif();
        std::vector<double> out((size_t)N * C * H * W), wts(out.size());
        oracle_resize_bilinear(x.data(), N, C, Hin, Win, H, W, out.data(), wts.data());
    }
    std::printf("sanitized run: %d packing cases, %d oracle layers, %d failures\n", packed_cases, conv_cases,
                failures);
    return failures ? 1 : 0;
}
