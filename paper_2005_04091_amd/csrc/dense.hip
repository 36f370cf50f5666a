// Dense path of the fused convolution on the matrix cores (gfx950 MFMA), for
// filters dense enough that skipping zeros no longer pays, and the host model
// that chooses between it and the sparse path (spconv_select_path).
//
// The convolution is the implicit GEMM  out[k, p] = sum over (c, r, s) of
// W[k, c, r, s] * Xp[c, p + r*Wp + s]  (stride 1, p = y*Wp + x, the paper's
// offset trick with the padded row pitch as pixel pitch; columns x >= Wo are
// computed and dropped). It runs in fp32 on v_mfma_f32_32x32x2f32, so products
// and sums keep fp32 precision like the sparse path:
//  * a workgroup owns (image, tile of TH output rows, 32*nw output channels);
//    each of its nw*ks waves owns 32 channels, NB blocks of 32 consecutive
//    virtual pixels of the tile (one 32x32 accumulator tile per block) and
//    every ks-th channel pair of the reduction; the ks partial sums of a tile
//    are added through LDS in a fixed order at the end;
//  * the tile's padded input rows are copied to LDS one channel chunk at a
//    time with asynchronous global->LDS loads into two buffers;
//  * the GEMM's reduction runs over channel pairs: one MFMA takes taps (2cp,
//    t) and (2cp+1, t), so B is the staged input shifted by the tap offset —
//    lanes 0-31 read 32 consecutive pixels of channel 2cp, lanes 32-63 of
//    channel 2cp+1 — and A is one 256-byte load from the filter packed by
//    spconv_pack_dense in exactly that fragment order;
//  * the epilogue adds bias (and a residual), applies ReLU, pools 2x2 windows
//    through a per-wave LDS tile when asked, and stores once.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>

#include "common.h"
#include "dense_layout.h"
#include "spconv.h"

__attribute__((visibility("hidden"))) int dense_kernel_variants(int32_t *variants, int32_t capacity, int32_t *count);

namespace {

typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kDnsTile = dense_layout::kTile;  // MFMA tile: 32 channels x 32 pixels
constexpr int kDnsMaxThreads = 512;       // nw * ks waves per workgroup, at most 8
constexpr int kDnsMaxBlocks = 8;          // pixel blocks per wave (16 accumulator VGPRs each)
constexpr int kDnsBlock = 256;            // floats per 16-byte-per-lane LDS DMA instruction
constexpr int kDnsLdsBytes = 64 * 1024;   // per workgroup: two resident per CU
constexpr int kDnsPoolCh = 8;             // channels of one pooled staging round (4 accumulator rows x 2 halves)

struct DenseArgs {
    int N, C, K, Kp, Hp, Wp, Ho, Wo, Hq, Wq;
    int relu;
    int TH;          // output rows per tile
    int ntiles_y;    // tiles per image
    int nw;          // channel tiles of 32 per workgroup
    int ks;          // waves splitting the reduction over channel pairs
    int nkt;         // channel tiles of 32*nw
    int Cc;          // channels per LDS chunk (even)
    int nchunks;
    int PLp;         // LDS floats per staged channel
    // staging units dealt round-robin to the nw*ks waves: (channel, padded
    // row) from an unpadded input, (channel, block of kDnsBlock) otherwise
    UnitStep row_units, blk_units;
    int buf_floats;  // Cc * PLp
    size_t total_floats;  // N*C*Hp*Wp
    int total_wgs;
    int out_pad, opitch;
    size_t oplane;
    int res_pad, rpitch;
    size_t rplane;
    int wpk_bytes;   // bytes of the packed filter (below 2^31)
    // epilogues: x / Wp, x / ((TH/2) * Wq) and x / Wq as multiply-shift
    uint32_t wp_magic, pch_magic, wq_magic;
    int wp_shift, pch_shift, wq_shift;
    int unpadded;    // input is N x C x H x W: the border is formed in LDS
    int H, W, pad, rows_in;
};

// Queue the copy of one channel chunk of the tile: channel cl of the chunk gets
// PLp floats from the tile's first padded row at buf + cl*PLp. A unit (channel,
// block of 256 floats) is one 16-byte-per-lane copy; units are dealt round-
// robin to the waves (the LDS-DMA engine's cost is per instruction, so 1 KiB
// copies move four times the bytes of dword ones for the same cost); the last
// block of a channel masks the lanes past PLp. Copies past the channel's rows
// read the next rows (never used by a stored pixel); the buffer range stops
// them at the end of the input tensor (such lanes read 0).
__device__ __forceinline__ void dense_stage(const DenseArgs &a, const float *__restrict__ xp, float *buf, int ch,
                                            int n, int row0, int wave, int lane) {
    const int c0 = ch * a.Cc;
    const int cn = min(a.Cc, a.C - c0);
    const int plane = a.Hp * a.Wp;
    const int nwaves = a.nw * a.ks;
    if (a.unpadded) {
        // Row by row from the unpadded input: padded row row0 + i is image row
        // row0 + i - pad, written at column pad of the channel's LDS row i, 64
        // floats per instruction (lanes past the row masked off). Border rows
        // and columns keep the zeros stored before the first copy.
        const int segs = (a.W + kWave - 1) / kWave;
        int cl, i;
        unit_first(a.row_units, wave, cl, i);
        while (cl < cn) {
            const int y = row0 + i - a.pad;
            if (y >= 0 && y < a.H) {
                const float *src = xp + (((size_t)n * a.C + c0 + cl) * a.H + y) * a.W;
                float *dst = buf + cl * a.PLp + i * a.Wp + a.pad;
                for (int sg = 0; sg < segs; ++sg) {
                    const int x0 = sg * kWave;
                    if (lane < a.W - x0)
                        __builtin_amdgcn_global_load_lds((global_void_t *)(src + x0 + lane), (lds_void_t *)(dst + x0),
                                                         4, 0, 0);
                }
            }
            unit_next(a.row_units, cl, i);
        }
    }
    if (!a.unpadded) {
        const size_t first = ((size_t)n * a.C + c0) * plane + (size_t)row0 * a.Wp;
        const size_t avail = (a.total_floats - first) * sizeof(float);
        const int nrec = avail > 0xffffffffull ? (int)0xffffffffu : (int)(uint32_t)avail;
        __amdgpu_buffer_rsrc_t rsrc =
            __builtin_amdgcn_make_buffer_rsrc((void *)(xp + first), (short)0, nrec, 0x00020000);
        int cl, b;
        unit_first(a.blk_units, wave, cl, b);
        while (cl < cn) {
            // Byte offsets of a chunk fit 32 bits (the planner checks).
            const uint32_t voff = (uint32_t)(cl * plane + b * kDnsBlock) * (uint32_t)sizeof(float) + lane * 16;
            if (b * kDnsBlock + lane * 4 < a.PLp)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (lds_void_t *)(buf + cl * a.PLp + b * kDnsBlock), 16,
                                                         voff, 0, 0, 0);
            unit_next(a.blk_units, cl, b);
        }
    }
    // An odd last chunk reads one channel slot past the tensor's channels with
    // zero weights; it must hold finite values: zero it.
    if (cn & 1)
        for (int e = (int)threadIdx.x; e < a.PLp; e += nwaves * kWave) buf[cn * a.PLp + e] = 0.0f;
}

__device__ __forceinline__ void dense_wait_copies() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

template <int R, int S, int NB, bool POOL>
__global__ __launch_bounds__(kDnsMaxThreads) void spconv_dense_kernel(DenseArgs a, const float *__restrict__ xp,
                                                                            const float *__restrict__ wpk,
                                                                            const float *__restrict__ bias,
                                                                            const float *__restrict__ res,
                                                                            float *__restrict__ out) {
    extern __shared__ float lds[];
    constexpr int RS = R * S;
    const int lane = (int)threadIdx.x & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x / kWave);
    const int work = xcd_linear_id((int)blockIdx.x, a.total_wgs);
    const int kt = work % a.nkt;
    const int rest = work / a.nkt;
    const int ty = rest % a.ntiles_y;
    const int n = rest / a.ntiles_y;
    const int y0 = ty * a.TH;
    const int wn = wave % a.nw, wk = wave / a.nw;  // channel tile, reduction share
    const int k0 = (kt * a.nw + wn) * kDnsTile;
    const int half = lane >> 5, col = lane & 31;

    // CH independent accumulator chains per pixel block: with one block a
    // wave's MFMAs would form one dependent chain, so its taps alternate
    // between two accumulators, added once after the loop.
    constexpr int CH = NB == 1 ? 2 : 1;
    f32x16_t acc[NB * CH];
#pragma unroll
    for (int b = 0; b < NB * CH; ++b)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[b][r] = 0.0f;

    // A fragment of (pair cp, tap t): wpk[((cp*RS + t)*Kp + k0 + col)*2 + half],
    // read through a buffer descriptor: the lane's part is a fixed VGPR
    // offset, the (pair, tap) part one scalar offset.
    const __amdgpu_buffer_rsrc_t wrs =
        __builtin_amdgcn_make_buffer_rsrc((void *)wpk, (short)0, a.wpk_bytes, 0x00020000);
    const int wvoff = ((k0 + col) * 2 + half) * (int)sizeof(float);
    const int wtap_bytes = a.Kp * 2 * (int)sizeof(float);
    // B fragment: the staged channel 2cp + half, pixel 32*b + col, shifted by r*Wp + s.
    const int lane_b = half * a.PLp + col;

    if (a.unpadded) {
        for (int e = (int)threadIdx.x * 4; e < 2 * a.buf_floats; e += (int)blockDim.x * 4)
            *reinterpret_cast<float4 *>(lds + e) = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
        __syncthreads();
    }
    dense_stage(a, xp, lds, 0, n, y0, wave, lane);
    dense_wait_copies();
    __syncthreads();

    // Two A register sets alternate over this wave's pairs (wk, wk + ks, ...)
    // of each chunk: the loads for the next pair are in flight while the MFMAs
    // of the current one issue. With few blocks a pair's MFMAs are short next
    // to an A load's latency (an L2 hit), and a third set keeps two pairs'
    // loads in flight.
    constexpr bool kA3 = NB <= 4;
    auto mma_pair = [&](const float(&av)[RS], int cp, const float *bb) {
        const float *bp = bb + 2 * cp * a.PLp;
#pragma unroll
        for (int r = 0; r < R; ++r)
#pragma unroll
            for (int s = 0; s < S; ++s) {
                const float *bt = bp + r * a.Wp + s;
                const int chain = CH == 2 ? ((r * S + s) & 1) : 0;
#pragma unroll
                for (int b = 0; b < NB; ++b)
                    acc[b * CH + chain] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[r * S + s], bt[kDnsTile * b],
                                                                             acc[b * CH + chain], 0, 0, 0);
            }
    };
    auto load_a = [&](float(&av)[RS], int gcp) {
        const int base = gcp * RS * wtap_bytes;
#pragma unroll
        for (int t = 0; t < RS; ++t)
            av[t] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(wrs, wvoff, base + t * wtap_bytes, 0));
    };
    for (int ch = 0; ch < a.nchunks; ++ch) {
        if (ch + 1 < a.nchunks) dense_stage(a, xp, lds + ((ch + 1) & 1) * a.buf_floats, ch + 1, n, y0, wave, lane);
        const float *bb = lds + (ch & 1) * a.buf_floats + lane_b;
        const int c0 = ch * a.Cc;
        const int npairs = (min(a.Cc, a.C - c0) + 1) / 2;
        const int gcp0 = c0 / 2;
        if constexpr (kA3) {
            // Three A sets: the loads of the next two pairs are in flight.
            float a0[RS], a1[RS], a2[RS];
            const int st = a.ks;
            if (wk < npairs) load_a(a0, gcp0 + wk);
            if (wk + st < npairs) load_a(a1, gcp0 + wk + st);
            for (int cp = wk; cp < npairs; cp += 3 * st) {
                if (cp + 2 * st < npairs) load_a(a2, gcp0 + cp + 2 * st);
                mma_pair(a0, cp, bb);
                if (cp + st >= npairs) break;
                if (cp + 3 * st < npairs) load_a(a0, gcp0 + cp + 3 * st);
                mma_pair(a1, cp + st, bb);
                if (cp + 2 * st >= npairs) break;
                if (cp + 4 * st < npairs) load_a(a1, gcp0 + cp + 4 * st);
                mma_pair(a2, cp + 2 * st, bb);
            }
        } else {
            float a0[RS], a1[RS];
            if (wk < npairs) load_a(a0, gcp0 + wk);
            for (int cp = wk; cp < npairs; cp += 2 * a.ks) {
                const int cq = cp + a.ks;
                if (cq < npairs) load_a(a1, gcp0 + cq);
                mma_pair(a0, cp, bb);
                if (cq < npairs) {
                    if (cq + a.ks < npairs) load_a(a0, gcp0 + cq + a.ks);
                    mma_pair(a1, cq, bb);
                }
            }
        }
        dense_wait_copies();
        __syncthreads();
    }

    if constexpr (CH == 2)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[0][r] += acc[1][r];

    // Sum the ks partial tiles into the waves with wk == 0, in order wk = 1,
    // 2, ...; the chunk buffers are free after the loop's last barrier.
    if (a.ks > 1) {
        float *red = lds + (size_t)wn * NB * 16 * kWave;
        for (int k = 1; k < a.ks; ++k) {
            if (wk == k)
#pragma unroll
                for (int b = 0; b < NB; ++b)
#pragma unroll
                    for (int j = 0; j < 16; ++j) red[(b * 16 + j) * kWave + lane] = acc[b][j];
            __syncthreads();
            if (wk == 0)
#pragma unroll
                for (int b = 0; b < NB; ++b)
#pragma unroll
                    for (int j = 0; j < 16; ++j) acc[b][j] += red[(b * 16 + j) * kWave + lane];
            __syncthreads();
        }
        if (wk != 0) return;
    }

    // Accumulator (block b, register j) holds channel k0 + 8*(j/4) + 4*half + j%4
    // at virtual pixel 32*b + col of the tile.
    const int tile_px = a.TH * a.Wp;
    const bool stream = a.out_pad == 0;
    if constexpr (!POOL) {
        // Row and column of this lane's pixel in each block (-1: not stored).
        int ys[NB], xs[NB];
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            const int q = kDnsTile * b + col;
            const int yl = (int)fast_div((uint32_t)q, a.wp_magic, a.wp_shift), x = q - yl * a.Wp;
            const bool in = q < tile_px && x < a.Wo && y0 + yl < a.Ho;
            ys[b] = in ? y0 + yl : -1;
            xs[b] = x;
        }
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            const int k = k0 + 8 * (j >> 2) + 4 * half + (j & 3);
            if (k >= a.K) continue;
            const float bk = bias ? bias[k] : 0.0f;
            float *plane = out + ((size_t)n * a.K + k) * a.oplane;
            const float *rplane = res ? res + ((size_t)n * a.K + k) * a.rplane : nullptr;
#pragma unroll
            for (int b = 0; b < NB; ++b) {
                const int y = ys[b], x = xs[b];
                if (y < 0) continue;
                float v = acc[b][j] + bk;
                if (rplane) v += rplane[(size_t)(y + a.res_pad) * a.rpitch + x + a.res_pad];
                if (a.relu) v = v > 0.0f ? v : 0.0f;
                store_out(plane + (size_t)(y + a.out_pad) * a.opitch + x + a.out_pad, v, stream);
            }
        }
        if (a.out_pad) {
            const int r1 = min(y0 + a.TH, a.Ho);
            for (int kk = k0; kk < min(k0 + kDnsTile, a.K); ++kk)
                zero_border(out + ((size_t)n * a.K + kk) * a.oplane, y0, r1, a.Ho, a.Wo, a.out_pad, a.opitch, ty == 0,
                            ty == a.ntiles_y - 1, lane, kWave);
        }
    } else {
        // Pool through a per-wave LDS tile, 8 channels at a time: activated
        // values on the conv grid, then the max of each 2x2 window. Only this
        // wave touches its area, and its LDS operations execute in issue
        // order; the chunk loop's last barrier ordered these writes after
        // every wave's reads of the input buffers.
        constexpr int kPx = NB * kDnsTile;
        float *st = lds + wn * kDnsPoolCh * kPx;
        const int prow0 = y0 / 2;
        const int prows = a.TH / 2;
        const int per_ch = prows * a.Wq;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) {
                const int j = 4 * g + jj;
                const int k = k0 + 8 * g + 4 * half + jj;
                const float bk = (bias && k < a.K) ? bias[k] : 0.0f;
                const float *rplane = (res && k < a.K) ? res + ((size_t)n * a.K + k) * a.rplane : nullptr;
#pragma unroll
                for (int b = 0; b < NB; ++b) {
                    const int q = kDnsTile * b + col;
                    float v = acc[b][j] + bk;
                    if (rplane) {
                        const int yl = (int)fast_div((uint32_t)q, a.wp_magic, a.wp_shift), x = q - yl * a.Wp;
                        if (q < tile_px && x < a.Wo && y0 + yl < a.Ho)
                            v += rplane[(size_t)(y0 + yl + a.res_pad) * a.rpitch + x + a.res_pad];
                    }
                    if (a.relu) v = v > 0.0f ? v : 0.0f;
                    st[(4 * half + jj) * kPx + q] = v;
                }
            }
            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
            for (int t = lane; t < kDnsPoolCh * per_ch; t += kWave) {
                const int cc = (int)fast_div((uint32_t)t, a.pch_magic, a.pch_shift);
                const int rem = t - cc * per_ch;
                const int r = (int)fast_div((uint32_t)rem, a.wq_magic, a.wq_shift), jq = rem - r * a.Wq;
                const int k = k0 + 8 * g + cc;
                const int pr = prow0 + r;
                if (k < a.K && pr < a.Hq) {
                    const float *s0 = st + cc * kPx + 2 * r * a.Wp + 2 * jq;
                    const float m = fmaxf(fmaxf(s0[0], s0[1]), fmaxf(s0[a.Wp], s0[a.Wp + 1]));
                    store_out(out + ((size_t)n * a.K + k) * a.oplane + (size_t)(pr + a.out_pad) * a.opitch + jq +
                                  a.out_pad,
                              m, stream);
                }
            }
        }
        if (a.out_pad) {
            const int r1 = min(prow0 + prows, a.Hq);
            for (int kk = k0; kk < min(k0 + kDnsTile, a.K); ++kk)
                zero_border(out + ((size_t)n * a.K + kk) * a.oplane, prow0, r1, a.Hq, a.Wq, a.out_pad, a.opitch,
                            ty == 0, ty == a.ntiles_y - 1, lane, kWave);
        }
    }
}

using DenseKernel = void (*)(DenseArgs, const float *, const float *, const float *, const float *, float *);

template <int R, int S, int NB>
DenseKernel pick_dense_pool(bool pool) {
    return pool ? spconv_dense_kernel<R, S, NB, true> : spconv_dense_kernel<R, S, NB, false>;
}

template <int R, int S>
DenseKernel pick_dense_nb(int NB, bool pool) {
    switch (NB) {
        case 1: return pick_dense_pool<R, S, 1>(pool);
        case 2: return pick_dense_pool<R, S, 2>(pool);
        case 3: return pick_dense_pool<R, S, 3>(pool);
        case 4: return pick_dense_pool<R, S, 4>(pool);
        case 5: return pick_dense_pool<R, S, 5>(pool);
        case 6: return pick_dense_pool<R, S, 6>(pool);
        case 7: return pick_dense_pool<R, S, 7>(pool);
        case 8: return pick_dense_pool<R, S, kDnsMaxBlocks>(pool);
        default: return nullptr;
    }
}

// Filter shapes the dense kernel is built for.
DenseKernel pick_dense(int R, int S, int NB, bool pool) {
    if (R == 3 && S == 3) return pick_dense_nb<3, 3>(NB, pool);
    if (R == 1 && S == 1) return pick_dense_nb<1, 1>(NB, pool);
    return nullptr;
}

}  // namespace

// (R, S, blocks per wave, pool) of every compiled dense instance (a library-
// internal helper of spconv_kernel_variants, not exported).
__attribute__((visibility("hidden"))) int dense_kernel_variants(int32_t *variants, int32_t capacity, int32_t *count) {
    int n = 0;
    for (int rs : {3, 1})
        for (int nb = 1; nb <= kDnsMaxBlocks; ++nb)
            for (int pool = 0; pool < 2; ++pool)
                if (pick_dense(rs, rs, nb, pool != 0)) {
                    if (n < capacity) {
                        variants[4 * n] = rs;
                        variants[4 * n + 1] = rs;
                        variants[4 * n + 2] = nb;
                        variants[4 * n + 3] = pool;
                    }
                    ++n;
                }
    *count = n;
    return SPCONV_OK;
}

namespace {

struct DensePlan {
    int TH = 0, ntiles_y = 0, NB = 0, nw = 0, ks = 1, nkt = 0, Cc = 0, nchunks = 0, PLp = 0, total_wgs = 0;
    size_t lds_bytes = 0;
};

using dense_layout::round_up;

int dense_waves(int K) { return dense_layout::waves(K); }

// Kp of the packed filter: K rounded up to whole workgroup channel tiles.
int dense_kp(int K) { return dense_layout::kp(K); }

// Waves that split the reduction over channel pairs (1, 2 or 4), each adding
// a 32-channel partial tile that is summed through LDS: 2 where the workgroup
// (8 waves), the LDS area of the partial tiles (64 KiB) and the chunk's pairs
// allow, 4 only when even 2 would leave the grid under 1024 waves (measured:
// 4 splits cost up to 30% more than 2 on grids that have enough waves).
int dense_ks(long long base_waves, int nw, int NB, int Cc) {
    const size_t red_bytes = (size_t)nw * NB * 16 * kWave * sizeof(float);
    int ks = 1;
    auto fits = [&](int k) { return nw * k * kWave <= kDnsMaxThreads && red_bytes <= (size_t)kDnsLdsBytes && k <= Cc / 2; };
    if (fits(2)) ks = 2;
    if (ks == 2 && base_waves * 2 < 1024 && fits(4)) ks = 4;
    return ks;
}

// Tile rows: among the heights whose tile fits 8 pixel blocks (even heights
// when pooling), the least modelled work, tiles x (blocks + 1): a wave's MFMAs
// per channel pair (one per block and tap) plus about one block's worth for
// the pair's A fragments, which each block reuses; provided the grid keeps at
// least 1536 waves (six per SIMD over the run) when any height can, ties going
// to the grid with more waves. Measured on 14x14 (256 channels), 28x28 pooled
// and 56x56 layers: the picks are each layer's fastest tiling of the sweep.
bool plan_dense(int N, int C, int K, int Wp, int Ho, int R, int S, bool pool, DensePlan *pl) {
    DensePlan p;
    p.nw = dense_waves(K);
    p.nkt = (K + kDnsTile * p.nw - 1) / (kDnsTile * p.nw);
    const long long kMinWaves = 1536;
    DensePlan best;
    long long best_cost = 0, best_waves = 0;
    for (int th = pool ? 2 : 1; th <= (pool ? round_up(Ho, 2) : Ho); th += pool ? 2 : 1) {
        DensePlan q = p;
        q.TH = th;
        q.NB = (th * Wp + kDnsTile - 1) / kDnsTile;
        if (q.NB > kDnsMaxBlocks) break;
        q.ntiles_y = (Ho + th - 1) / th;
        // A channel's staged rows must cover every B read: the last block's
        // last pixel shifted by the largest tap offset. Slots are 16-byte
        // aligned for the 16-byte copies.
        q.PLp = round_up(std::max((th + R - 1) * Wp, q.NB * kDnsTile + (R - 1) * Wp + S - 1), 4);
        const int cmax = kDnsLdsBytes / (2 * q.PLp * (int)sizeof(float)) / 2 * 2;
        if (cmax < 2) continue;
        q.Cc = std::min(cmax, round_up(C, 2));
        q.nchunks = (C + q.Cc - 1) / q.Cc;
        // The copy offsets of one chunk are 32-bit byte offsets (and int floats).
        if (((long long)(q.Cc - 1) * (Ho + R - 1) * Wp + q.PLp + kDnsBlock) * 4 >= (1LL << 31)) continue;
        const long long base_waves = (long long)N * q.ntiles_y * q.nkt * q.nw;
        q.ks = dense_ks(base_waves, q.nw, q.NB, q.Cc);
        const long long waves = base_waves * q.ks;
        const long long cost = (long long)q.ntiles_y * (q.NB + 1);
        bool better;
        if (best.TH == 0) {
            better = true;
        } else {
            const bool ok = waves >= kMinWaves, best_ok = best_waves >= kMinWaves;
            if (ok != best_ok)
                better = ok;
            else if (!ok)
                better = waves > best_waves;
            else
                better = cost < best_cost || (cost == best_cost && waves > best_waves);
        }
        if (better) {
            best = q;
            best_cost = cost;
            best_waves = waves;
        }
    }
    if (best.TH == 0) return false;
    p = best;
    size_t lds = (size_t)2 * p.Cc * p.PLp * sizeof(float);
    if (pool) lds = std::max(lds, (size_t)p.nw * kDnsPoolCh * p.NB * kDnsTile * sizeof(float));
    if (p.ks > 1) lds = std::max(lds, (size_t)p.nw * p.NB * 16 * kWave * sizeof(float));
    if (lds > (size_t)kDnsLdsBytes) return false;
    p.lds_bytes = lds;
    const long long wgs = (long long)N * p.ntiles_y * p.nkt;
    if (wgs > 0x7fffffffLL) return false;
    p.total_wgs = (int)wgs;
    *pl = p;
    return true;
}

bool out_extent(int in, int k, int pad, int *o) {
    const long long v = (long long)in + 2LL * pad - k + 1;
    if (v < 1 || v > 0x7fffffffLL) return false;
    *o = (int)v;
    return true;
}

// Checks and plan of a dense forward call (everything but the buffers).
int prepare_dense(int N, int C, int H, int W, int K, int R, int S, int pad, uint32_t flags,
                  const spconv_options *opt, DensePlan *plp, DenseArgs *ap) {
    if (N < 1 || C < 1 || H < 1 || W < 1 || K < 1 || R < 1 || S < 1 || pad < 0) return SPCONV_EINVAL;
    if (flags & ~(SPCONV_RELU | SPCONV_MAXPOOL2X2 | SPCONV_UNPADDED_INPUT)) return SPCONV_EINVAL;
    const long long Hp = (long long)H + 2LL * pad, Wp = (long long)W + 2LL * pad;
    if ((long long)C * Hp * Wp >= (1LL << 31)) return SPCONV_EINVAL;
    const bool pool = (flags & SPCONV_MAXPOOL2X2) != 0;
    int Ho, Wo;
    if (!out_extent(H, R, pad, &Ho) || !out_extent(W, S, pad, &Wo)) return SPCONV_EINVAL;
    if (pool && (Ho < 2 || Wo < 2)) return SPCONV_EINVAL;
    DensePlan pl;
    if (!plan_dense(N, C, K, (int)Wp, Ho, R, S, pool, &pl)) return SPCONV_EINVAL;
    if (!pick_dense(R, S, pl.NB, pool)) return SPCONV_EINVAL;
    DenseArgs a;
    a.N = N;
    a.C = C;
    a.K = K;
    a.Kp = dense_kp(K);
    const long long wbytes = (long long)((C + 1) / 2) * R * S * a.Kp * 2 * (long long)sizeof(float);
    if (wbytes >= (1LL << 31)) return SPCONV_EINVAL;
    a.wpk_bytes = (int)wbytes;
    a.Hp = (int)Hp;
    a.Wp = (int)Wp;
    a.Ho = Ho;
    a.Wo = Wo;
    a.Hq = pool ? Ho / 2 : Ho;
    a.Wq = pool ? Wo / 2 : Wo;
    a.pch_magic = a.wq_magic = 1;
    a.pch_shift = a.wq_shift = 0;
    if (!div_magic((uint32_t)a.Wp, &a.wp_magic, &a.wp_shift) ||
        (pool && (!div_magic((uint32_t)((pl.TH / 2) * a.Wq), &a.pch_magic, &a.pch_shift) ||
                  !div_magic((uint32_t)a.Wq, &a.wq_magic, &a.wq_shift))))
        return SPCONV_EINVAL;
    a.relu = (flags & SPCONV_RELU) ? 1 : 0;
    a.unpadded = (flags & SPCONV_UNPADDED_INPUT) ? 1 : 0;
    a.H = H;
    a.W = W;
    a.pad = pad;
    a.rows_in = pl.TH + R - 1;
    a.TH = pl.TH;
    a.ntiles_y = pl.ntiles_y;
    a.nw = pl.nw;
    a.ks = pl.ks;
    a.nkt = pl.nkt;
    a.Cc = pl.Cc;
    a.nchunks = pl.nchunks;
    a.PLp = pl.PLp;
    if (!unit_step(a.rows_in, pl.nw * pl.ks, &a.row_units) ||
        !unit_step((pl.PLp + kDnsBlock - 1) / kDnsBlock, pl.nw * pl.ks, &a.blk_units))
        return SPCONV_EINVAL;
    a.buf_floats = pl.Cc * pl.PLp;
    a.total_floats = (size_t)N * C * Hp * Wp;
    a.total_wgs = pl.total_wgs;
    const long long op = opt ? opt->out_pad : 0;
    const long long rp = (opt && opt->residual) ? opt->residual_pad : 0;
    if (op < 0 || rp < 0) return SPCONV_EINVAL;
    const long long oh = a.Hq + 2 * op, ow = a.Wq + 2 * op;
    const long long rh = a.Ho + 2 * rp, rw = a.Wo + 2 * rp;
    if (oh * ow >= (1LL << 31) || rh * rw >= (1LL << 31)) return SPCONV_EINVAL;
    a.out_pad = (int)op;
    a.opitch = (int)ow;
    a.oplane = (size_t)(oh * ow);
    a.res_pad = (int)rp;
    a.rpitch = (int)rw;
    a.rplane = (size_t)(rh * rw);
    *plp = pl;
    *ap = a;
    return SPCONV_OK;
}

}  // namespace

extern "C" int spconv_forward_dense(const float *in_padded, int N, int C, int H, int W, const float *packed, int K,
                                    int R, int S, int pad, const float *bias, uint32_t flags,
                                    const spconv_options *opt, float *out, hipStream_t stream) {
    if (!in_padded || !packed || !out) return SPCONV_EINVAL;
    DensePlan pl;
    DenseArgs a;
    const int rc = prepare_dense(N, C, H, W, K, R, S, pad, flags, opt, &pl, &a);
    if (rc != SPCONV_OK) return rc;
    DenseKernel kern = pick_dense(R, S, pl.NB, (flags & SPCONV_MAXPOOL2X2) != 0);
    const float *residual = opt ? opt->residual : nullptr;
    // Raised once per instance to the family's budget (see raise_lds_limit).
    if (!raise_lds_limit((const void *)kern, kDnsLdsBytes)) return SPCONV_EHIP;
    hipLaunchKernelGGL(kern, dim3((unsigned)pl.total_wgs), dim3((unsigned)(pl.nw * pl.ks * kWave)), pl.lds_bytes, stream, a,
                       in_padded, packed, bias, residual, out);
    return hipGetLastError() == hipSuccess ? SPCONV_OK : SPCONV_EHIP;
}

extern "C" int spconv_dense_plan(int N, int C, int H, int W, int K, int R, int S, int pad, uint32_t flags,
                                 spconv_plan_info *info) {
    if (!info) return SPCONV_EINVAL;
    DensePlan pl;
    DenseArgs a;
    const int rc = prepare_dense(N, C, H, W, K, R, S, pad, flags, nullptr, &pl, &a);
    if (rc != SPCONV_OK) return rc;
    info->kernel = SPCONV_KERNEL_DENSE;
    info->pixels_per_lane = pl.NB;
    info->images_per_group = 1;
    info->channels_per_wave = kDnsTile;
    info->tile_rows = pl.TH;
    info->tiles_per_image = pl.ntiles_y;
    info->channels_per_chunk = pl.Cc;
    info->chunks = pl.nchunks;
    info->workgroups = pl.total_wgs;
    info->threads_per_workgroup = pl.nw * pl.ks * kWave;
    info->lds_bytes = (int64_t)pl.lds_bytes;
    info->lds_channel_floats = info->lds_row_pitch = info->lds_col_shift = 0;
    info->launch_workgroups = pl.total_wgs;
    info->tile_pixels = 0;
    return SPCONV_OK;
}

namespace {

// Break-even filter density on MI355X: above it the dense kernel beats the
// sparse ones. Measured with both paths on the same layers (fp32, batch 32,
// back-to-back launches): about 0.245 for 256 channels at 14x14, 0.44 for 128
// channels at 28x28 with the pool, 0.42-0.47 at 56x56 (64 or 128 channels,
// pooled or not) and 0.67 for 64 channels at 224x224. The sparse kernels spread
// each entry's fixed cost over the pixels of an image tile, so their rate,
// and the break-even, grow with the image: the threshold interpolates
// log-linearly in output pixels per image between those measurements and
// stays at the end values beyond them.
double break_even_density(int Ho, int Wo) {
    struct Anchor {
        double px, d;
    };
    static constexpr Anchor kAnchors[] = {{196.0, 0.245}, {784.0, 0.44}, {3136.0, 0.43}, {50176.0, 0.67}};
    constexpr int n = (int)(sizeof(kAnchors) / sizeof(kAnchors[0]));
    const double px = std::max(1.0, (double)Ho * Wo);
    if (px <= kAnchors[0].px) return kAnchors[0].d;
    for (int i = 1; i < n; ++i)
        if (px <= kAnchors[i].px) {
            const double t = std::log2(px / kAnchors[i - 1].px) / std::log2(kAnchors[i].px / kAnchors[i - 1].px);
            return kAnchors[i - 1].d + t * (kAnchors[i].d - kAnchors[i - 1].d);
        }
    return kAnchors[n - 1].d;
}

}  // namespace

extern "C" int spconv_select_path(int N, int C, int H, int W, int K, int R, int S, int stride, int pad, int64_t nnz,
                                  uint32_t flags, int *path) {
    if (!path || N < 1 || C < 1 || H < 1 || W < 1 || K < 1 || R < 1 || S < 1 || stride < 1 || pad < 0 || nnz < 0 ||
        nnz > (int64_t)K * C * R * S || (flags & ~(SPCONV_RELU | SPCONV_MAXPOOL2X2 | SPCONV_UNPADDED_INPUT)))
        return SPCONV_EINVAL;
    *path = SPCONV_PATH_SPARSE;
    if (stride != 1) return SPCONV_OK;
    DensePlan pl;
    DenseArgs a;
    if (prepare_dense(N, C, H, W, K, R, S, pad, flags & ~SPCONV_UNPADDED_INPUT, nullptr, &pl, &a) != SPCONV_OK)
        return SPCONV_OK;
    if ((double)nnz > break_even_density(a.Ho, a.Wo) * (double)K * C * R * S) *path = SPCONV_PATH_DENSE;
    return SPCONV_OK;
}
