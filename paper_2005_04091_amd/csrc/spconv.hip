// Fused sparse direct convolution for MI355X (gfx950): padded-input kernel,
// sparse gather-accumulate kernel with fused bias / ReLU / 2x2 max-pool, and
// the C-ABI entry points that validate, plan the tiling and launch them.
//
// The method is the CSR direct convolution of the paper's "Sparse Convolution
// with CSR" paragraph: for output channel k and each nonzero (offset, coeff) of
// CSR row k, every output pixel p accumulates coeff * in_padded[p + offset].
// With stride 1 and the padded row pitch Wp as the pixel pitch, pixel
// (y, x) sits at p = y*Wp + x ("virtual" columns x >= Wo are computed and never
// stored), so one nonzero moves a whole contiguous pixel range by one offset.
//
// Mapping to CDNA4:
//  * a workgroup (4 wave64s) owns (image group, output-channel tile of KT rows,
//    spatial tile of TH output rows at full width);
//  * the padded input rows of the tile are staged in LDS one channel chunk at a
//    time; the CSR rows are walked in order, the nonzeros of each row arriving
//    through scalar loads, so every lane sees the same (offset, coeff);
//  * lane l of a wave owns pixels q0 + l + 64*j (j < P): each LDS read of a wave
//    touches 64 consecutive floats (no bank conflicts) and each global store of
//    the epilogue is coalesced;
//  * accumulators for all KT rows stay in VGPRs across the channel chunks; the
//    epilogue adds the bias, applies ReLU and, for the pooled variant, reduces
//    the 2x2 windows through an LDS staging tile before the single store.
// MFMA is not used: at the densities this path serves, the work is a
// gather-accumulate, not a dense contraction.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <cstring>

#include "spconv.h"

namespace {

constexpr int kWave = 64;
constexpr int kWaves = 4;
constexpr int kThreads = kWave * kWaves;
constexpr int kXcds = 8;                  // MI355X: 8 XCDs, workgroups dispatched round-robin
constexpr int kLdsBudgetFloats = 16384;   // 64 KiB of LDS per workgroup (two workgroups per CU)

// ---------------------------------------------------------------------------
// Padded input (spconv_pad_input)
// ---------------------------------------------------------------------------

// One workgroup covers 4*256 consecutive elements of one padded plane; each of
// its four store instructions writes 256 consecutive floats.
constexpr int kPadPerThread = 4;
constexpr int kPadPerBlock = kThreads * kPadPerThread;

struct PadArgs {
    const float *in;
    float *out;
    int H, W, pad, Hp, Wp;
    int plane;            // Hp*Wp
    int blocks_per_plane;
    uint32_t wp_magic;    // x / Wp == (x * wp_magic) >> wp_shift for 0 <= x < 2^31
    int wp_shift;
};

__device__ __forceinline__ uint32_t fast_div(uint32_t x, uint32_t magic, int shift) {
    return (uint32_t)(((uint64_t)x * (uint64_t)magic) >> shift);
}

__global__ __launch_bounds__(kThreads) void pad_nchw_kernel(PadArgs a) {
    const uint32_t plane_id = blockIdx.x / (uint32_t)a.blocks_per_plane;
    const uint32_t blk = blockIdx.x - plane_id * (uint32_t)a.blocks_per_plane;
    const float *src = a.in + (size_t)plane_id * (size_t)a.H * (size_t)a.W;
    float *dst = a.out + (size_t)plane_id * (size_t)a.plane;
#pragma unroll
    for (int u = 0; u < kPadPerThread; ++u) {
        const int e = (int)blk * kPadPerBlock + u * kThreads + (int)threadIdx.x;
        if (e < a.plane) {
            const int yp = (int)fast_div((uint32_t)e, a.wp_magic, a.wp_shift);
            const int xp = e - yp * a.Wp;
            const int y = yp - a.pad, x = xp - a.pad;
            float v = 0.0f;
            if (y >= 0 && y < a.H && x >= 0 && x < a.W) v = src[(size_t)y * a.W + x];
            dst[e] = v;
        }
    }
}

// ---------------------------------------------------------------------------
// Sparse convolution (spconv_forward)
// ---------------------------------------------------------------------------

struct FwdArgs {
    const float *xp;        // [N][C][Hp][Wp]
    const int32_t *rowptr;  // [K+1]
    const int32_t *offset;  // [nnz]
    const float *vals;      // [nnz]
    const float *bias;      // [K] or null
    float *out;
    int N, C, K, Hp, Wp, Ho, Wo, Hq, Wq, stride;
    int relu;
    // tiling
    int TH;            // output rows per spatial tile
    int ntiles_y;      // spatial tiles per image
    int ipw;           // images per workgroup
    int wpi;           // waves per image
    int nktiles;       // ceil(K / KT)
    int Cc;            // channels per LDS chunk
    int nchunks;
    int rows_in;       // padded input rows staged per tile
    int PL;            // LDS floats per staged channel (rows_in * Wp)
    int img_lds;       // LDS floats per image block (Cc * PL)
    int wv;            // pixel pitch of the virtual tile: Wp (stride 1) or Wo
    int total_wgs;
    uint32_t magic;    // c = offset / (Hp*Wp) == (offset * magic) >> shift
    int shift;
    int plane_delta;   // Hp*Wp - PL
};

// Workgroup id -> linear work index such that consecutive work items (the KT
// tiles of one image tile, which read the same staged input) land on the same
// XCD and therefore share its L2.
__device__ __forceinline__ int xcd_linear_id(int b, int G) {
    const int xcd = b % kXcds, i = b / kXcds;
    const int per = G / kXcds, rem = G % kXcds;
    return (xcd < rem) ? xcd * (per + 1) + i : rem * (per + 1) + (xcd - rem) * per + i;
}

template <int P, int KT, bool S1, bool POOL>
__global__ __launch_bounds__(kThreads) void spconv_fwd_kernel(FwdArgs a) {
    extern __shared__ float lds[];

    const int L = xcd_linear_id((int)blockIdx.x, a.total_wgs);
    const int kt = L % a.nktiles;
    const int grp = L / a.nktiles;
    const int ty = grp % a.ntiles_y;
    const int ig = grp / a.ntiles_y;
    const int y0 = ty * a.TH;
    const int k0 = kt * KT;

    const int wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
    const int lane = (int)threadIdx.x & 63;
    const int img = wave / a.wpi;
    const int wseg = wave - img * a.wpi;
    const int n = ig * a.ipw + img;
    const bool active = n < a.N;
    const int plane = a.Hp * a.Wp;

    // CSR cursor per row of the tile (scalar registers).
    int cur[KT], end[KT];
#pragma unroll
    for (int kk = 0; kk < KT; ++kk) {
        const int k = k0 + kk;
        cur[kk] = (k < a.K) ? a.rowptr[k] : 0;
        end[kk] = (k < a.K) ? a.rowptr[k + 1] : 0;
    }

    // Pixels of this lane inside the image tile: q = qw + 64*j.
    const int qw = wseg * kWave * P + lane;
    const int tile_px = a.TH * a.wv;
    int base[S1 ? 1 : P];
    if constexpr (S1) {
        base[0] = qw;
    } else {
#pragma unroll
        for (int j = 0; j < P; ++j) {
            const int q = qw + kWave * j;
            const int yl = q / a.Wo, x = q - yl * a.Wo;
            base[j] = (q < tile_px) ? yl * a.stride * a.Wp + x * a.stride : 0;
        }
    }

    float acc[KT][P];
#pragma unroll
    for (int kk = 0; kk < KT; ++kk)
#pragma unroll
        for (int j = 0; j < P; ++j) acc[kk][j] = 0.0f;

    const int in_row0 = y0 * a.stride;
    const int seg_len = min(a.rows_in, a.Hp - in_row0) * a.Wp;

    for (int ch = 0; ch < a.nchunks; ++ch) {
        const int c0 = ch * a.Cc;
        const int cn = min(a.Cc, a.C - c0);
        __syncthreads();  // every wave is done with the previous chunk
        for (int im = 0; im < a.ipw; ++im) {
            const int nn = ig * a.ipw + im;
            if (nn >= a.N) break;
            for (int cl = 0; cl < cn; ++cl) {
                const float *src = a.xp + ((size_t)(nn * a.C + c0 + cl) * a.Hp + in_row0) * a.Wp;
                float *dst = lds + im * a.img_lds + cl * a.PL;
                for (int e = (int)threadIdx.x; e < seg_len; e += kThreads) dst[e] = src[e];
            }
        }
        __syncthreads();
        if (!active) continue;

        // LDS address of tap `off` for pixel base b: vb + off - c*plane_delta + b,
        // where c = off / plane is the tap's channel.
        const int vb = img * a.img_lds - c0 * a.PL;
        const int bound = (c0 + cn) * plane;
#pragma unroll
        for (int kk = 0; kk < KT; ++kk) {
            int j = cur[kk];
            const int e = end[kk];
            while (j + 8 <= e) {
                int o[8];
#pragma unroll
                for (int u = 0; u < 8; ++u) o[u] = a.offset[j + u];
                if (o[7] >= bound) break;
#pragma unroll
                for (int u = 0; u < 8; ++u) {
                    const float v = a.vals[j + u];
                    const int c = (int)fast_div((uint32_t)o[u], a.magic, a.shift);
                    const int ad = vb + o[u] - c * a.plane_delta;
                    if constexpr (S1) {
#pragma unroll
                        for (int p = 0; p < P; ++p) acc[kk][p] = fmaf(v, lds[ad + base[0] + kWave * p], acc[kk][p]);
                    } else {
#pragma unroll
                        for (int p = 0; p < P; ++p) acc[kk][p] = fmaf(v, lds[ad + base[p]], acc[kk][p]);
                    }
                }
                j += 8;
            }
            while (j < e) {
                const int o = a.offset[j];
                if (o >= bound) break;
                const float v = a.vals[j];
                const int c = (int)fast_div((uint32_t)o, a.magic, a.shift);
                const int ad = vb + o - c * a.plane_delta;
                if constexpr (S1) {
#pragma unroll
                    for (int p = 0; p < P; ++p) acc[kk][p] = fmaf(v, lds[ad + base[0] + kWave * p], acc[kk][p]);
                } else {
#pragma unroll
                    for (int p = 0; p < P; ++p) acc[kk][p] = fmaf(v, lds[ad + base[p]], acc[kk][p]);
                }
                ++j;
            }
            cur[kk] = j;
        }
    }

    if constexpr (!POOL) {
        if (!active) return;
        int pix[P];  // in-plane output index of each of this lane's pixels, or -1
#pragma unroll
        for (int j = 0; j < P; ++j) {
            const int q = qw + kWave * j;
            const int yl = q / a.wv, x = q - yl * a.wv;
            const int y = y0 + yl;
            pix[j] = (q < tile_px && x < a.Wo && y < a.Ho) ? y * a.Wo + x : -1;
        }
#pragma unroll
        for (int kk = 0; kk < KT; ++kk) {
            const int k = k0 + kk;
            if (k >= a.K) break;
            const float bk = a.bias ? a.bias[k] : 0.0f;
            float *op = a.out + ((size_t)n * a.K + k) * (size_t)a.Ho * a.Wo;
#pragma unroll
            for (int j = 0; j < P; ++j) {
                float v = acc[kk][j] + bk;
                if (a.relu) v = v > 0.0f ? v : 0.0f;
                if (pix[j] >= 0) op[pix[j]] = v;
            }
        }
    } else {
        // Stage each row's activated tile in LDS, then reduce 2x2 windows.
        const int img_px = a.wpi * kWave * P;
        const int prow0 = y0 / 2;
        const int prows = a.TH / 2;
        const int per_img = prows * a.Wq;
        const int total = a.ipw * per_img;
#pragma unroll
        for (int kk = 0; kk < KT; ++kk) {
            const int k = k0 + kk;
            if (k >= a.K) break;
            const float bk = a.bias ? a.bias[k] : 0.0f;
            __syncthreads();  // previous readers of the staging area are done
#pragma unroll
            for (int j = 0; j < P; ++j) {
                float v = acc[kk][j] + bk;
                if (a.relu) v = v > 0.0f ? v : 0.0f;
                lds[img * img_px + qw + kWave * j] = v;
            }
            __syncthreads();
            for (int t = (int)threadIdx.x; t < total; t += kThreads) {
                const int im = t / per_img;
                const int rem = t - im * per_img;
                const int i = rem / a.Wq;
                const int jq = rem - i * a.Wq;
                const int nn = ig * a.ipw + im;
                const int pi = prow0 + i;
                if (nn < a.N && pi < a.Hq) {
                    const float *s0 = lds + im * img_px + (2 * i) * a.wv + 2 * jq;
                    const float m = fmaxf(fmaxf(s0[0], s0[1]), fmaxf(s0[a.wv], s0[a.wv + 1]));
                    a.out[((size_t)nn * a.K + k) * (size_t)a.Hq * a.Wq + (size_t)pi * a.Wq + jq] = m;
                }
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Host side
// ---------------------------------------------------------------------------

// x / d == (x * magic) >> shift for all 0 <= x < 2^31 (d >= 1): with
// L = ceil(log2 d), magic = ceil(2^(31+L) / d) < 2^32 and the rounding error
// x * (magic*d - 2^(31+L)) / (d * 2^(31+L)) stays below 1/d.
bool div_magic(uint32_t d, uint32_t *magic, int *shift) {
    if (d == 0) return false;
    if (d == 1) {
        *magic = 1;
        *shift = 0;
        return true;
    }
    int L = 0;
    while ((1ull << L) < d) ++L;
    const int s = 31 + L;
    const uint64_t m = ((1ull << s) + d - 1) / d;
    if (m > 0xffffffffull) return false;
    *magic = (uint32_t)m;
    *shift = s;
    return true;
}

int ceil_div(int a, int b) { return (a + b - 1) / b; }

struct Plan {
    int P = 0, KT = 0;
    bool s1 = true;
    int TH = 0, ntiles_y = 0, ipw = 0, wpi = 0, Cc = 0, nchunks = 0, rows_in = 0, PL = 0, img_lds = 0, wv = 0;
    int nktiles = 0, total_wgs = 0;
    size_t lds_bytes = 0;
};

// Picks the pixels per lane (P), the waves per image and the tile height that
// waste the fewest lanes, then the channel chunk that fits the LDS budget.
bool make_plan(int N, int C, int K, int Hp, int Wp, int Ho, int Wo, int stride, int R, int S, bool pool, Plan *out) {
    const bool s1 = stride == 1;
    const int wv = s1 ? Wp : Wo;
    const int img_pix = Ho * wv;
    static const int kP_s1[] = {8, 7, 6, 5, 4};
    static const int kP_gen[] = {4};
    const int *Ps = s1 ? kP_s1 : kP_gen;
    const int nP = s1 ? 5 : 1;
    Plan best;
    double best_eff = -1.0;
    for (int pi = 0; pi < nP; ++pi) {
        const int P = Ps[pi];
        for (int wpi : {4, 2, 1}) {
            const int ipw = kWaves / wpi;
            const int cap = wpi * kWave * P;  // virtual pixels per image tile
            int TH, nt;
            if (img_pix <= cap) {
                TH = Ho;
                nt = 1;
            } else {
                if (ipw != 1) continue;  // several images per workgroup only when each fits whole
                int th_max = cap / wv;
                if (pool) th_max &= ~1;
                if (th_max < 1) continue;
                nt = ceil_div(Ho, th_max);
                TH = ceil_div(Ho, nt);
                if (pool && (TH & 1)) ++TH;
                nt = ceil_div(Ho, TH);
            }
            const int rows_in = (TH - 1) * stride + R;
            const int PL = rows_in * Wp;
            const int slack = s1 ? (cap - TH * Wp) + S : 0;
            int cc_max = (kLdsBudgetFloats - slack) / (ipw * PL);
            if (cc_max < 1) continue;
            cc_max = std::min(cc_max, C);
            const int nchunks = ceil_div(C, cc_max);
            const int Cc = ceil_div(C, nchunks);
            const double eff = (double)Ho * Wo / ((double)nt * ipw * cap / ipw);
            // Prefer the least waste; on ties, more pixels per lane.
            if (eff > best_eff + 1e-9) {
                best_eff = eff;
                best.P = P;
                best.s1 = s1;
                best.TH = TH;
                best.ntiles_y = nt;
                best.ipw = ipw;
                best.wpi = wpi;
                best.Cc = Cc;
                best.nchunks = nchunks;
                best.rows_in = rows_in;
                best.PL = PL;
                best.img_lds = Cc * PL;
                best.wv = wv;
                size_t floats = (size_t)ipw * Cc * PL + (size_t)slack;
                if (pool) floats = std::max(floats, (size_t)ipw * cap);
                best.lds_bytes = floats * sizeof(float);
            }
        }
    }
    if (best_eff < 0) return false;
    const int groups = ceil_div(N, best.ipw) * best.ntiles_y;
    best.KT = (groups * ceil_div(K, 8) >= 512) ? 8 : 4;
    if (!s1) best.KT = 4;
    best.nktiles = ceil_div(K, best.KT);
    const long long wgs = (long long)groups * best.nktiles;
    if (wgs > 0x7fffffffLL) return false;
    best.total_wgs = (int)wgs;
    *out = best;
    return true;
}

using FwdKernel = void (*)(FwdArgs);

template <int P, int KT, bool S1>
FwdKernel pick_pool(bool pool) {
    return pool ? spconv_fwd_kernel<P, KT, S1, true> : spconv_fwd_kernel<P, KT, S1, false>;
}

template <int P>
FwdKernel pick_kt(int KT, bool pool) {
    return KT == 8 ? pick_pool<P, 8, true>(pool) : pick_pool<P, 4, true>(pool);
}

FwdKernel pick_kernel(const Plan &pl, bool pool) {
    if (!pl.s1) return pick_pool<4, 4, false>(pool);
    switch (pl.P) {
        case 8: return pick_kt<8>(pl.KT, pool);
        case 7: return pick_kt<7>(pl.KT, pool);
        case 6: return pick_kt<6>(pl.KT, pool);
        case 5: return pick_kt<5>(pl.KT, pool);
        case 4: return pick_kt<4>(pl.KT, pool);
        default: return nullptr;
    }
}

bool out_extent(int in, int f, int stride, int pad, int *o) {
    const long long span = (long long)in + 2LL * pad - f;
    if (span < 0) return false;
    *o = (int)(span / stride + 1);
    return true;
}

}  // namespace

extern "C" int spconv_output_shape(int H, int W, int R, int S, int stride, int pad, uint32_t flags, int *Ho, int *Wo) {
    if (!Ho || !Wo || H < 1 || W < 1 || R < 1 || S < 1 || stride < 1 || pad < 0) return SPCONV_EINVAL;
    if (flags & ~(SPCONV_RELU | SPCONV_MAXPOOL2X2)) return SPCONV_EINVAL;
    int ho, wo;
    if (!out_extent(H, R, stride, pad, &ho) || !out_extent(W, S, stride, pad, &wo)) return SPCONV_EINVAL;
    if (flags & SPCONV_MAXPOOL2X2) {
        if (ho < 2 || wo < 2) return SPCONV_EINVAL;
        ho /= 2;
        wo /= 2;
    }
    *Ho = ho;
    *Wo = wo;
    return SPCONV_OK;
}

extern "C" const char *spconv_strerror(int code) {
    switch (code) {
        case SPCONV_OK: return "success";
        case SPCONV_EINVAL: return "invalid argument";
        case SPCONV_ECAPACITY: return "output arrays too small for the number of nonzeros";
        case SPCONV_EHIP: return "HIP runtime error or kernel launch failure";
        default: return "unknown spconv status code";
    }
}

extern "C" int spconv_pad_input(const float *in, int N, int C, int H, int W, int pad, float *out_padded,
                                hipStream_t stream) {
    if (!in || !out_padded || N < 1 || C < 1 || H < 1 || W < 1 || pad < 0) return SPCONV_EINVAL;
    const long long Hp = (long long)H + 2LL * pad, Wp = (long long)W + 2LL * pad;
    const long long plane = Hp * Wp;
    const long long planes = (long long)N * C;
    if (plane >= (1LL << 31) || planes * plane >= (1LL << 40)) return SPCONV_EINVAL;
    PadArgs a;
    a.in = in;
    a.out = out_padded;
    a.H = H;
    a.W = W;
    a.pad = pad;
    a.Hp = (int)Hp;
    a.Wp = (int)Wp;
    a.plane = (int)plane;
    a.blocks_per_plane = (int)((plane + kPadPerBlock - 1) / kPadPerBlock);
    if (!div_magic((uint32_t)Wp, &a.wp_magic, &a.wp_shift)) return SPCONV_EINVAL;
    const long long blocks = planes * a.blocks_per_plane;
    if (blocks > 0x7fffffffLL) return SPCONV_EINVAL;
    hipLaunchKernelGGL(pad_nchw_kernel, dim3((unsigned)blocks), dim3(kThreads), 0, stream, a);
    return hipGetLastError() == hipSuccess ? SPCONV_OK : SPCONV_EHIP;
}

extern "C" int spconv_forward(const float *in_padded, int N, int C, int H, int W, const spconv_csr *csr, int K, int R,
                              int S, int stride, int pad, const float *bias, uint32_t flags, float *out,
                              hipStream_t stream) {
    if (!in_padded || !csr || !out) return SPCONV_EINVAL;
    if (N < 1 || C < 1 || H < 1 || W < 1 || K < 1 || R < 1 || S < 1 || stride < 1 || pad < 0) return SPCONV_EINVAL;
    if (flags & ~(SPCONV_RELU | SPCONV_MAXPOOL2X2)) return SPCONV_EINVAL;
    if (csr->K != K || csr->C != C || csr->R != R || csr->S != S) return SPCONV_EINVAL;
    const long long Hp = (long long)H + 2LL * pad, Wp = (long long)W + 2LL * pad;
    if (csr->Hp != Hp || csr->Wp != Wp) return SPCONV_EINVAL;
    if (csr->nnz < 0 || csr->nnz >= (1LL << 31)) return SPCONV_EINVAL;
    if (!csr->rowptr || (csr->nnz > 0 && (!csr->offset || !csr->vals))) return SPCONV_EINVAL;
    if ((long long)C * Hp * Wp >= (1LL << 31)) return SPCONV_EINVAL;
    const bool pool = (flags & SPCONV_MAXPOOL2X2) != 0;
    int Ho, Wo;
    if (!out_extent(H, R, stride, pad, &Ho) || !out_extent(W, S, stride, pad, &Wo)) return SPCONV_EINVAL;
    if (Ho < 1 || Wo < 1) return SPCONV_EINVAL;
    if (pool && (Ho < 2 || Wo < 2)) return SPCONV_EINVAL;

    Plan pl;
    if (!make_plan(N, C, K, (int)Hp, (int)Wp, Ho, Wo, stride, R, S, pool, &pl)) return SPCONV_EINVAL;
    FwdArgs a;
    a.xp = in_padded;
    a.rowptr = csr->rowptr;
    a.offset = csr->offset;
    a.vals = csr->vals;
    a.bias = bias;
    a.out = out;
    a.N = N;
    a.C = C;
    a.K = K;
    a.Hp = (int)Hp;
    a.Wp = (int)Wp;
    a.Ho = Ho;
    a.Wo = Wo;
    a.Hq = pool ? Ho / 2 : Ho;
    a.Wq = pool ? Wo / 2 : Wo;
    a.stride = stride;
    a.relu = (flags & SPCONV_RELU) ? 1 : 0;
    a.TH = pl.TH;
    a.ntiles_y = pl.ntiles_y;
    a.ipw = pl.ipw;
    a.wpi = pl.wpi;
    a.nktiles = pl.nktiles;
    a.Cc = pl.Cc;
    a.nchunks = pl.nchunks;
    a.rows_in = pl.rows_in;
    a.PL = pl.PL;
    a.img_lds = pl.img_lds;
    a.wv = pl.wv;
    a.total_wgs = pl.total_wgs;
    if (!div_magic((uint32_t)(Hp * Wp), &a.magic, &a.shift)) return SPCONV_EINVAL;
    a.plane_delta = (int)(Hp * Wp) - pl.PL;
    FwdKernel kern = pick_kernel(pl, pool);
    if (!kern) return SPCONV_EINVAL;
    hipLaunchKernelGGL(kern, dim3((unsigned)pl.total_wgs), dim3(kThreads), pl.lds_bytes, stream, a);
    return hipGetLastError() == hipSuccess ? SPCONV_OK : SPCONV_EHIP;
}
