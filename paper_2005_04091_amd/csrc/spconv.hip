// Fused sparse direct convolution for MI355X (gfx950): padded-input kernel,
// sparse gather-accumulate kernels with fused bias / ReLU / 2x2 max-pool, and
// the C-ABI entry points that validate, plan the tiling and launch them.
//
// The method is the CSR direct convolution of the paper's "Sparse Convolution
// with CSR" paragraph: for output channel k and each nonzero (offset, coeff) of
// CSR row k, every output pixel p accumulates coeff * in_padded[p + offset].
// With stride 1 and the padded row pitch Wp as the pixel pitch, pixel (y, x)
// sits at p = y*Wp + x ("virtual" columns x >= Wo are computed and never
// stored), so one nonzero shifts a whole contiguous pixel range by one offset.
//
// Stride-1 kernel (the hot path), mapped to CDNA4:
//  * a workgroup (16 wave64s, one per CU) owns (group of IPW images, spatial
//    tile of TH output rows at full padded width, tile of 16*RPW output
//    channels); each wave owns RPW of those channels and every pixel of the
//    tile;
//  * the padded input rows of the tile are copied to LDS one channel chunk at
//    a time with asynchronous global->LDS loads into two buffers, so the copy of
//    chunk c+1 overlaps the arithmetic on chunk c;
//  * each wave walks its CSR rows in order: a window of entries is loaded one
//    per lane, its offsets are decoded to LDS indices, and each entry's (index,
//    weight) is broadcast to all lanes;
//  * lane l owns the pixel pairs (2l + 128j, 2l+1 + 128j), so a tap is one
//    aligned 8-byte LDS read per pair (the fastest LDS read form on gfx950);
//    taps whose LDS index is odd are read as the pairs (2l-1, 2l) into a second
//    accumulator set, merged with one cross-lane shift in the epilogue;
//  * accumulators stay in VGPRs across the chunks; the epilogue adds the bias,
//    applies ReLU and, for the pooled variant, reduces 2x2 windows through an
//    LDS staging tile before the single store.
// MFMA is not used: at the densities this path serves, the work is a
// gather-accumulate, not a dense contraction.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <type_traits>
#include <vector>

#include "common.h"
#include "spconv.h"

// Instances of the dense kernel (dense.hip), for spconv_kernel_variants.
__attribute__((visibility("hidden"))) int dense_kernel_variants(int32_t *variants, int32_t capacity, int32_t *count);

namespace {

constexpr int kWaves = 4;
constexpr int kThreads = kWave * kWaves;
constexpr int kLdsBudgetFloats = 20480;   // generic kernel: 80 KiB of LDS per workgroup (two per CU)
constexpr int kGenericLdsBytes = kLdsBudgetFloats * 4;


// ---------------------------------------------------------------------------
// Padded input (spconv_pad_input)
// ---------------------------------------------------------------------------

// The padded tensor is treated as one flat array of 4-element quads. A
// workgroup covers kPadQuads consecutive quads per thread: in round j thread t
// writes quad (block*kPadQuads + j)*256 + t with one 16-byte store (when the
// output is 16-byte aligned), so each round's stores coalesce; a quad inside
// one input row is fetched with one 16-byte load, border quads element by
// element (0 outside the input). All loads of a thread are issued before its
// stores. The workgroup's first plane takes one 64-bit division; every quad's
// plane, row and column inside the workgroup's span take 32-bit
// multiply-shift divisions.
constexpr int kPadQuads = 2;  // measured on MI355X: 2 beats 1, 4 and 8 (more workgroups in flight)
constexpr int kPadSpan = 4 * kThreads * kPadQuads;  // elements per workgroup
constexpr long long kPadMaxPlane = (1LL << 31) - 4096;  // padded planes must stay below this
static_assert(kPadSpan <= 4096, "a workgroup's span must fit below 2^31 past any plane start");

struct PadArgs {
    const float *in;
    float *out;
    long long total;       // N*C*Hp*Wp
    int H, W, pad, Hp, Wp;
    int plane;             // Hp*Wp, below kPadMaxPlane
    uint32_t plane_magic;  // x / plane == (x * plane_magic) >> plane_shift for 0 <= x < 2^31
    int plane_shift;
    uint32_t wp_magic;     // x / Wp likewise
    int wp_shift;
};

// Quad starting at flat element f0 = pbase*plane + e (0 <= e < plane + kPadSpan).
__device__ __forceinline__ float4 pad_quad(const PadArgs &a, long long f0, long long pbase, int e) {
    const int q = (int)fast_div((uint32_t)e, a.plane_magic, a.plane_shift);
    long long pid = pbase + q;  // plane (n, c) of the first element
    e -= q * a.plane;
    int yp = (int)fast_div((uint32_t)e, a.wp_magic, a.wp_shift);
    int xp = e - yp * a.Wp;
    const int y0 = yp - a.pad, x0 = xp - a.pad;
    if (f0 + 3 < a.total && y0 >= 0 && y0 < a.H && x0 >= 0 && x0 + 3 < a.W) {
        float4 v;  // all four inside one input row: one 16-byte load (4-byte aligned)
        __builtin_memcpy(&v, a.in + pid * a.H * a.W + (long long)y0 * a.W + x0, sizeof(v));
        return v;
    }
    float v[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int y = yp - a.pad, x = xp - a.pad;
        v[j] = 0.0f;
        if (f0 + j < a.total && y >= 0 && y < a.H && x >= 0 && x < a.W)
            v[j] = a.in[pid * a.H * a.W + (long long)y * a.W + x];
        if (++xp == a.Wp) {  // next element of the flat array
            xp = 0;
            if (++yp == a.Hp) {
                yp = 0;
                ++pid;
            }
        }
    }
    return make_float4(v[0], v[1], v[2], v[3]);
}

template <bool VEC>
__global__ __launch_bounds__(kThreads) void pad_nchw_kernel(PadArgs a) {
    const long long fb = (long long)blockIdx.x * kPadSpan;
    const long long pbase = fb / a.plane;
    const int eb = (int)(fb - pbase * a.plane);
    float4 q[kPadQuads];
#pragma unroll
    for (int j = 0; j < kPadQuads; ++j) {
        const int off = (j * kThreads + (int)threadIdx.x) * 4;
        if (fb + off < a.total) q[j] = pad_quad(a, fb + off, pbase, eb + off);
    }
#pragma unroll
    for (int j = 0; j < kPadQuads; ++j) {
        const long long f = fb + (j * kThreads + (int)threadIdx.x) * 4;
        if (f >= a.total) break;
        if (VEC && f + 3 < a.total) {
            stream_store4(a.out + f, q[j]);
        } else {
            const float v[4] = {q[j].x, q[j].y, q[j].z, q[j].w};
#pragma unroll
            for (int u = 0; u < 4; ++u)
                if (f + u < a.total) stream_store(a.out + f + u, v[u]);
        }
    }
}

// ---------------------------------------------------------------------------
// Bilinear resize into the padded layout (spconv_resize_pad_input)
// ---------------------------------------------------------------------------

// Output coordinate o of an axis resized from n_in to n_out samples the input
// at s = (o + 1/2) * n_in / n_out - 1/2 (pixel centres aligned), clamped below
// at 0, between the taps i0 = floor(s) and i1 = min(i0 + 1, n_in - 1), with
// weight t = s - i0 on i1. In integers s = num / (2 n_out) with
// num = (2o + 1) n_in - n_out, so i0 is exact and t is the correctly rounded
// float of an exact fraction. Sides are at most 16384, so num < 2^30.
struct ResizeTap {
    int i0, i1;
    float t;
};

__device__ __forceinline__ ResizeTap resize_tap(int o, int n_in, int n_out) {
    const int num = max((2 * o + 1) * n_in - n_out, 0);
    const int den = 2 * n_out;
    ResizeTap r;
    r.i0 = num / den;
    r.i1 = min(r.i0 + 1, n_in - 1);
    r.t = (float)(num - r.i0 * den) / (float)den;
    return r;
}

// Interpolation in lerp form: with t = 0 (an axis of unchanged size) it
// returns its first operand exactly, so an unchanged plane is copied bitwise.
__device__ __forceinline__ float lerp_f(float a, float b, float t) { return a + t * (b - a); }

struct ResizeArgs {
    int Hin, Win, H, W, pad, Hp, Wp;
    int bands;       // row bands per plane, one workgroup each
    int band_rows;   // padded output rows per band
};

constexpr int kResizeMaxSide = 16384;
constexpr int kResizeTargetWgs = 2048;  // split planes into row bands until the grid has this many workgroups

// Row variant, for planes too large for the flat variant's LDS tables (any
// width): one workgroup writes one band of padded rows of one (n, c) plane;
// waves take the band's rows round-robin and each row is written 64 columns at
// a time (coalesced stores; the two source rows of a row are read by one
// wave). Border rows and columns are written as +0.0.
__global__ __launch_bounds__(kThreads) void resize_pad_rows_kernel(ResizeArgs a, const float *__restrict__ in,
                                                                   float *__restrict__ out) {
    const int lane = (int)threadIdx.x & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x / kWave);
    const int plane = (int)blockIdx.x / a.bands;
    const int band = (int)blockIdx.x - plane * a.bands;
    const float *src = in + (size_t)plane * a.Hin * a.Win;
    float *dst = out + (size_t)plane * a.Hp * a.Wp;
    const int r1 = min(a.Hp, (band + 1) * a.band_rows);
    for (int yp = band * a.band_rows + wave; yp < r1; yp += kWaves) {
        float *drow = dst + (size_t)yp * a.Wp;
        const int y = yp - a.pad;
        if (y < 0 || y >= a.H) {  // a border row (wave-uniform)
            for (int xp = lane; xp < a.Wp; xp += kWave) stream_store(drow + xp, 0.0f);
            continue;
        }
        const ResizeTap ty = resize_tap(y, a.Hin, a.H);
        const float *s0 = src + (size_t)ty.i0 * a.Win;
        const float *s1 = src + (size_t)ty.i1 * a.Win;
        for (int xp = lane; xp < a.Wp; xp += kWave) {
            const int x = xp - a.pad;
            float o = 0.0f;
            if (x >= 0 && x < a.W) {
                const ResizeTap t = resize_tap(x, a.Win, a.W);
                o = lerp_f(lerp_f(s0[t.i0], s0[t.i1], t.t), lerp_f(s1[t.i0], s1[t.i1], t.t), ty.t);
            }
            stream_store(drow + xp, o);
        }
    }
}

// Plane variant, for small planes (source and padded output): a workgroup
// copies ppw consecutive source planes into LDS with coalesced loads (16
// bytes per lane when aligned), then writes their padded output planes as one
// flat range, each wave round one coalesced streaming store, reading each
// element's four taps from LDS. Tap tables and interpolation order are the
// flat variant's, so both give the same bits. Replaces that variant's four
// gathers from global memory per element by one streamed read of the source.
constexpr int kResizePlaneMaxIn = 4096;       // source floats per plane
constexpr int kResizePlaneMaxOut = 16384;     // padded output floats per plane
constexpr int kResizePlaneLds = 48 * 1024;    // bytes of staged source per workgroup
constexpr long long kResizePlaneWgs = 2048;   // planes per workgroup grow while the grid keeps this many

struct ResizePlaneArgs {
    int Hin, Win, H, W, pad, Hp, Wp;
    int ps;               // Hp * Wp
    int in_ps;            // Hin * Win
    int ppw;              // planes per workgroup
    int vec;              // 16-byte source loads (aligned tensor, in_ps % 4 == 0)
    long long planes;
    uint32_t ps_magic, wp_magic;  // x / ps, x / Wp as multiply-shift
    int ps_shift, wp_shift;
};

__global__ __launch_bounds__(kThreads) void resize_pad_plane_kernel(ResizePlaneArgs a, const float *__restrict__ in,
                                                                    float *__restrict__ out) {
    extern __shared__ int tab[];
    const int nt = a.Hp + a.Wp;
    int *tap0 = tab;
    int *tap1 = tab + nt;
    float *tapw = reinterpret_cast<float *>(tab + 2 * nt);
    float *src = reinterpret_cast<float *>(tab + ((3 * nt + 3) & ~3));
    for (int i = (int)threadIdx.x; i < nt; i += kThreads) {
        const bool row = i < a.Hp;
        const int o = (row ? i : i - a.Hp) - a.pad;
        const int n_out = row ? a.H : a.W;
        const int scale = row ? a.Win : 1;
        int t0 = -1, t1 = 0;
        float w = 0.0f;
        if (o >= 0 && o < n_out) {
            const ResizeTap r = resize_tap(o, row ? a.Hin : a.Win, n_out);
            t0 = r.i0 * scale;
            t1 = r.i1 * scale;
            w = r.t;
        }
        tap0[i] = t0;
        tap1[i] = t1;
        tapw[i] = w;
    }
    const long long p0 = (long long)blockIdx.x * a.ppw;
    const int np = (int)min((long long)a.ppw, a.planes - p0);
    const float *sp = in + p0 * a.in_ps;
    const int n = np * a.in_ps;
    if (a.vec) {
        for (int i = (int)threadIdx.x * 4; i < n; i += kThreads * 4)
            *reinterpret_cast<float4 *>(src + i) = *reinterpret_cast<const float4 *>(sp + i);
    } else {
        for (int i = (int)threadIdx.x; i < n; i += kThreads) src[i] = sp[i];
    }
    __syncthreads();
    float *op = out + p0 * a.ps;
    const int m = np * a.ps;
    for (int e = (int)threadIdx.x; e < m; e += kThreads) {
        const int q = (int)fast_div((uint32_t)e, a.ps_magic, a.ps_shift);
        const int ee = e - q * a.ps;
        const int yp = (int)fast_div((uint32_t)ee, a.wp_magic, a.wp_shift);
        const int xp = ee - yp * a.Wp;
        const int r0 = tap0[yp], c0 = tap0[a.Hp + xp];
        float o = 0.0f;
        if ((r0 | c0) >= 0) {
            const int r1 = tap1[yp], c1 = tap1[a.Hp + xp];
            const float tx = tapw[a.Hp + xp];
            const float *pl = src + q * a.in_ps;
            o = lerp_f(lerp_f(pl[r0 + c0], pl[r0 + c1], tx), lerp_f(pl[r1 + c0], pl[r1 + c1], tx), tapw[yp]);
        }
        stream_store(op + e, o);
    }
}

// Flat variant for planes whose two tap tables fit in LDS (Hp + Wp entries):
// the padded output of all planes is one flat array, each thread takes
// kResizeFlatElems elements 256 apart (every lane busy whatever the width, each
// round one coalesced store per wave) and issues the loads of all of them
// before the first store. Per element: (plane, row, column) by multiply-shift
// division, the row and column taps from the tables, four loads at 32-bit
// offsets from the workgroup's first plane, three interpolations.
constexpr int kResizeFlatElems = 8;
constexpr int kResizeFlatMaxTab = 4096;   // Hp + Wp; 12 B of LDS per entry

struct ResizeFlatArgs {
    int Hin, Win, H, W, pad, Hp, Wp;
    int ps;               // Hp * Wp
    uint32_t ps_magic;    // x / ps == (x * ps_magic) >> ps_shift for 0 <= x < 2^31
    int ps_shift;
    uint32_t wp_magic;    // x / Wp likewise
    int wp_shift;
    long long total;      // planes * ps
};

__global__ __launch_bounds__(kThreads) void resize_pad_flat_kernel(ResizeFlatArgs a, const float *__restrict__ in,
                                                                   float *__restrict__ out) {
    // Tables, entry i < Hp for padded row i, Hp + x for padded column x:
    // first and second tap (row taps pre-multiplied by Win; -1 = border) and
    // the weight of the second.
    extern __shared__ int tab[];
    const int nt = a.Hp + a.Wp;
    int *tap0 = tab;
    int *tap1 = tab + nt;
    float *tapw = reinterpret_cast<float *>(tab + 2 * nt);
    for (int i = (int)threadIdx.x; i < nt; i += kThreads) {
        const bool row = i < a.Hp;
        const int o = (row ? i : i - a.Hp) - a.pad;
        const int n_out = row ? a.H : a.W;
        const int scale = row ? a.Win : 1;
        int t0 = -1, t1 = 0;
        float w = 0.0f;
        if (o >= 0 && o < n_out) {
            const ResizeTap r = resize_tap(o, row ? a.Hin : a.Win, n_out);
            t0 = r.i0 * scale;
            t1 = r.i1 * scale;
            w = r.t;
        }
        tap0[i] = t0;
        tap1[i] = t1;
        tapw[i] = w;
    }
    __syncthreads();

    constexpr int E = kResizeFlatElems;
    const long long f0 = (long long)blockIdx.x * (kThreads * E);
    const long long p0 = f0 / a.ps;
    const int e0 = (int)(f0 - p0 * a.ps);
    const float *sblk = in + p0 * a.Hin * a.Win;  // the workgroup's first source plane
    const uint32_t src_plane = (uint32_t)(a.Hin * a.Win);
    float v[E][4];
    float tx[E], ty[E];
    bool inside[E];
#pragma unroll
    for (int j = 0; j < E; ++j) {
        const int e = e0 + j * kThreads + (int)threadIdx.x;
        const uint32_t q = fast_div((uint32_t)e, a.ps_magic, a.ps_shift);
        const int ee = e - (int)q * a.ps;
        const int yp = (int)fast_div((uint32_t)ee, a.wp_magic, a.wp_shift);
        const int xp = ee - yp * a.Wp;
        const int r0 = tap0[yp], c0 = tap0[a.Hp + xp];
        inside[j] = f0 + j * kThreads + threadIdx.x < a.total && (r0 | c0) >= 0;
        ty[j] = tapw[yp];
        tx[j] = tapw[a.Hp + xp];
        if (inside[j]) {
            const int r1 = tap1[yp], c1 = tap1[a.Hp + xp];
            const uint32_t pb = q * src_plane;
            v[j][0] = sblk[pb + (uint32_t)(r0 + c0)];
            v[j][1] = sblk[pb + (uint32_t)(r0 + c1)];
            v[j][2] = sblk[pb + (uint32_t)(r1 + c0)];
            v[j][3] = sblk[pb + (uint32_t)(r1 + c1)];
        }
    }
#pragma unroll
    for (int j = 0; j < E; ++j) {
        const long long f = f0 + j * kThreads + threadIdx.x;
        if (f >= a.total) break;
        float o = 0.0f;
        if (inside[j]) o = lerp_f(lerp_f(v[j][0], v[j][1], tx[j]), lerp_f(v[j][2], v[j][3], tx[j]), ty[j]);
        stream_store(out + f, o);
    }
}

// ---------------------------------------------------------------------------
// Sparse convolution (spconv_forward)
// ---------------------------------------------------------------------------

// Sizes and tiling of one launch. The buffers travel as separate __restrict__
// kernel arguments: that is what lets the compiler fetch the CSR stream with
// scalar loads (it must know no store or asynchronous LDS copy in the kernel
// can modify them).
struct FwdArgs {
    int N, C, K, Hp, Wp, Ho, Wo, Hq, Wq, stride;
    int nnz;
    int relu;
    // tiling
    int TH;            // output rows per spatial tile
    int ntiles_y;      // spatial tiles per image
    int ipw;           // images per workgroup
    int wpi;           // waves per image (generic kernel)
    int nktiles;       // ceil(K / rows per workgroup)
    int Cc;            // channels per LDS chunk
    int nchunks;
    int rows_in;       // padded input rows staged per tile
    int PL;            // LDS floats per staged channel (rows_in * Wp)
    int img_lds;       // LDS floats per image block (Cc * PL)
    int PLp;           // LDS pitch of one staged channel (stride-1 kernel: PL rounded up to 4)
    UnitStep stage_units;  // stride-1 padded staging: (channel, block of kStageBlock) units over 16 waves
    int buf_floats;    // LDS floats per chunk buffer (stride-1 kernel: two buffers)
    size_t total_floats;  // N*C*Hp*Wp, the extent of the padded input
    int wv;            // pixel pitch of the virtual tile: Wp (stride 1) or Wo
    int total_wgs;
    uint32_t magic;    // c = offset / (Hp*Wp) == (offset * magic) >> shift
    int shift;
    int plane_delta;   // Hp*Wp - PL
    // epilogue: stored planes carry a zero border of out_pad (pitch opitch,
    // oplane elements each); the residual planes a border of res_pad (pitch
    // rpitch, rplane elements each)
    int out_pad, opitch;
    size_t oplane;
    int res_pad, rpitch;
    size_t rplane;
    // input layout: 0 = padded (N x C x Hp x Wp); 1 = unpadded (N x C x H x W),
    // the zero border formed in LDS by the stride-1 kernel's staging
    int unpadded;
    int H, W, pad;
    // stride-1 kernel: pitch of the virtual tile and of the staged LDS rows
    // (Wp, or Wp rounded up to 4 when an unpadded input's rows are whole
    // 16-byte groups), the LDS column of padded column 0 (lds_shift), and
    // whether an unpadded input is copied 16 bytes per lane
    int vp, lds_shift, dma16;
    uint32_t wp_magic;  // x / Wp == (x * wp_magic) >> wp_shift
    int wp_shift;
    uint32_t plp_magic;  // x / PLp (stride-1 kernel's unpadded staging)
    int plp_shift;
    // stride-1 epilogues: x / vp, x / ((TH/2) * Wq) and x / Wq as multiply-
    // shift (a runtime integer division is some 30 instructions, several of
    // them quarter rate, per stored pixel)
    uint32_t vp_magic, pimg_magic, wq_magic;
    int vp_shift, pimg_shift, wq_shift;
    // stride-1 unpooled epilogue: a lane's pixel pair (2l, 2l+1) always lies in
    // one stored row or outside the output, so each pair moves with one
    // two-dword access
    int pair_store;
    // lowered entry stream (spconv_pack_lowered): headers {start, n_even,
    // n_odd, k} per (channel tile, wave, row slot, chunk), then n_entries
    // (LDS index, weight) pairs and an over-read pad of kLwPad pairs
    int lw_headers;
    int lw_entries;
    int lds_floats;  // dynamic LDS of the launch, in floats
    int pf_bytes;    // stride-1 lowered walk: bytes of a wave's entry lists prefetched per item
    // pooled epilogue: the pitch vp is even, so pixel pairs are horizontal
    // pool pairs (pair-maxima staging), and that staging fits one chunk buffer
    int pool_pairs, pool_in_buf;
    // stride-1 kernel with a lowered stream: virtual pixels per row-spanning
    // tile (tile t covers [t*span, (t+1)*span) of its image, from the row it
    // starts in), or 0 for tiles of TH whole rows
    int span;
};

// Entries fetched per scalar load in the lowered walk (one s_load_dwordx16),
// and the pad of entries after the stream that such loads may read (a walk
// near the end of the stream loads the batch after its current one).
constexpr int kLwBatch = 8;
constexpr int kLwPad = 2 * kLwBatch;
constexpr int kLwSinkFloats = 64;  // stride-1 kernel: LDS sink of the entry-stream prefetch (never read)

// Queue asynchronous global->LDS copies of one channel chunk: for each image of
// the group and each channel of the chunk, seg_len consecutive floats (the
// tile's padded input rows) land at buf + im*img_lds + cl*PL. Each wave copies
// blocks of 64 floats, one per lane.
__device__ __forceinline__ void stage_chunk(const FwdArgs &a, const float *__restrict__ xp, float *buf, int ch, int ig,
                                            int in_row0, int seg_len, int wave, int lane) {
    const int c0 = ch * a.Cc;
    const int cn = min(a.Cc, a.C - c0);
    const int nblk = (seg_len + kWave - 1) / kWave;
    for (int im = 0; im < a.ipw; ++im) {
        const int nn = ig * a.ipw + im;
        if (nn >= a.N) break;
        for (int cl = 0; cl < cn; ++cl) {
            const float *src = xp + ((size_t)(nn * a.C + c0 + cl) * a.Hp + in_row0) * a.Wp;
            float *dst = buf + im * a.img_lds + cl * a.PL;
            for (int b = wave; b < nblk; b += kWaves) {
                const int e = b * kWave + lane;
                if (e < seg_len)
                    __builtin_amdgcn_global_load_lds((global_void_t *)(src + e), (lds_void_t *)(dst + b * kWave), 4, 0,
                                                     0);
            }
        }
    }
}

__device__ __forceinline__ void wait_async_copies() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// ---- Stride-1 kernel ------------------------------------------------------

constexpr int kS1Waves = 16;
constexpr int kS1Threads = kS1Waves * kWave;
constexpr int kS1LdsFloats = 40960;  // 160 KiB: one workgroup per CU, two chunk buffers
constexpr int kStageBlock = 256;     // floats per 16-byte-per-lane LDS DMA instruction

// Queue the asynchronous copy of one channel chunk: for each image of the group
// and each channel of the chunk, the channel's LDS slot of PLp floats at
// buf + im*img_lds + cl*PLp. The slot starts at column col0 of padded row
// in_row0 (col0 = 0 but for the window of a row-spanning tile).
//
// Padded input: PLp consecutive floats from there, every lane moving 16 bytes
// per instruction (buffer_load_dwordx4 ... lds). Copies may run past the
// tile's rows into the slot's padding; the buffer range stops them at the end
// of the input tensor (such lanes read 0).
//
// Unpadded input: the chunk's slots are rewritten whole, each instruction
// filling one block of consecutive LDS floats (64 lanes of 16 or 4 bytes)
// whatever the row length. A lane maps its LDS position to (slot cl, staged
// row i, column x of the image row y = in_row0 + i - pad) and takes the image
// pixels there; everything else (border columns, rows outside the image, the
// pitch gap, the slot's tail) reads as zeros through an offset past the
// buffer's range. So no border survives from an earlier tile, and no separate
// zero fill is needed. With dma16 (W and the row starts 16-byte aligned,
// pitch and shift + pad multiples of 4) a lane's four floats lie all inside or
// all outside the image row; otherwise each lane moves one.
__device__ __forceinline__ void stage_chunk_s1(const FwdArgs &a, const float *__restrict__ xp, float *buf, int ch,
                                               int ig, int in_row0, int wave, int lane, int col0 = 0) {
    const int c0 = ch * a.Cc;
    const int cn = min(a.Cc, a.C - c0);
    if (a.unpadded) {
        const int per_lane = a.dma16 ? 4 : 1;
        const int blk_floats = kWave * per_lane;
        const int span = cn * a.PLp;
        const int nblk = (span + blk_floats - 1) / blk_floats;
        // Image rows [y_lo, y_lo + y_span) hold every pixel the tile reads.
        const int y_lo = max(in_row0 - a.pad, 0);
        const int y_span = max(min(in_row0 - a.pad + a.rows_in, a.H) - y_lo, 0);
        // Bytes from the chunk's first row to the end of its last: every image
        // pixel a lane reads lies below, and `nrec` itself reads as zeros.
        const uint32_t nrec = (uint32_t)(((size_t)(cn - 1) * a.H + y_span) * a.W * sizeof(float));
        const int lead = a.lds_shift + a.pad;  // slot position of image column 0, staged row 0
        for (int im = 0; im < a.ipw; ++im) {
            const int nn = ig * a.ipw + im;
            if (nn >= a.N) break;
            const float *base = xp + (((size_t)nn * a.C + c0) * a.H + y_lo) * a.W;
            __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc((void *)base, (short)0, (int)nrec, 0x00020000);
            float *dst = buf + im * a.img_lds;
            for (int b = wave; b < nblk; b += kS1Waves) {
                const int P = b * blk_floats + lane * per_lane;
                if (P < span) {
                    const int cl = (int)fast_div((uint32_t)P, a.plp_magic, a.plp_shift);
                    // t = i*vp + x from image column 0 of staged row 0; t + vp >= 0
                    // (positions before it belong to row -1, at x >= W).
                    const int t = P - cl * a.PLp - lead + col0;
                    const int i = (int)fast_div((uint32_t)(t + a.vp), a.vp_magic, a.vp_shift) - 1;
                    const int x = t - i * a.vp;
                    const int y = in_row0 + i - a.pad;
                    const bool in = i < a.rows_in && x < a.W && y >= 0 && y < a.H;  // x >= 0 and i >= 0 follow
                    const uint32_t voff =
                        in ? (uint32_t)((cl * a.H + (y - y_lo)) * a.W + x) * (uint32_t)sizeof(float) : nrec;
                    if (a.dma16)
                        __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (lds_void_t *)(dst + b * blk_floats), 16, voff, 0,
                                                                 0, 0);
                    else
                        __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (lds_void_t *)(dst + b * blk_floats), 4, voff, 0,
                                                                 0, 0);
                }
            }
        }
        return;
    }
    const int plane = a.Hp * a.Wp;
    for (int im = 0; im < a.ipw; ++im) {
        const int nn = ig * a.ipw + im;
        if (nn >= a.N) break;
        const size_t first = ((size_t)(nn * a.C + c0) * a.Hp + in_row0) * a.Wp + col0;
        const size_t avail = (a.total_floats - first) * sizeof(float);
        const int nrec = avail > 0xffffffffull ? (int)0xffffffffu : (int)(uint32_t)avail;
        __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc((void *)(xp + first), (short)0, nrec, 0x00020000);
        float *dst = buf + im * a.img_lds;
        // Work units (channel cl, block b) are dealt round-robin to the waves.
        int cl, b;
        unit_first(a.stage_units, wave, cl, b);
        while (cl < cn) {
            const uint32_t voff = (uint32_t)((cl * plane + b * kStageBlock) * (int)sizeof(float)) + lane * 16;
            if (b * kStageBlock + lane * 4 < a.PLp)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (lds_void_t *)(dst + cl * a.PLp + b * kStageBlock), 16,
                                                         voff, 0, 0, 0);
            unit_next(a.stage_units, cl, b);
        }
    }
}

// Up to 128 consecutive CSR entries of one row as loaded: lane l holds entries
// base+l (slot 0) and base+64+l (slot 1); entries at or past the row's end read
// as offset INT32_MAX, weight 0.
struct RawWindow {
    int o[2];
    float w[2];
    int base;
};

__device__ __forceinline__ RawWindow fetch_window(const int32_t *__restrict__ offset, const float *__restrict__ vals,
                                                  int j, int e, int lane) {
    RawWindow r;
    r.base = j;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int idx = j + h * kWave + lane;
        const bool valid = idx < e;
        r.o[h] = valid ? offset[idx] : 0x7fffffff;
        r.w[h] = valid ? vals[idx] : 0.0f;
    }
    return r;
}

// A window decoded for one channel chunk. Per slot, the entries of the chunk
// (a prefix of the window) are split by the parity of their tap's LDS float
// index for virtual pixel 0; each lane holds that index rounded down to even
// (`lo`) and its weight. Even taps are read as aligned pixel pairs (2l, 2l+1);
// odd taps as the aligned pairs (2l-1, 2l), which accumulate into the
// pixel-shifted accumulator set. Two forms:
//  * masks: the entries stay in their lanes; `even`/`odd` are the lane masks
//    of the two classes, walked with find-first-set;
//  * compacted: lanes 0..ne-1 hold the even taps, ne..ne+no-1 the odd ones
//    (CSR order within each class), walked with a counter: three fewer
//    scalar instructions per entry, which pays where an entry has few FMAs.
// `n` counts the chunk's entries. (Each form holds only its own fields: the
// scalar registers of two channels' windows are a tight budget.)
struct WindowMasks {
    int lo[2];
    float w[2];
    uint64_t even[2], odd[2];
    int n;
};
struct WindowCompact {
    int lo[2];
    float w[2];
    int ne[2], no[2];
    int n;
};
template <bool COMPACT>
using Window = typename std::conditional<COMPACT, WindowCompact, WindowMasks>::type;

// Number of set bits of m in lanes below this one.
__device__ __forceinline__ int lanes_below(uint64_t m) {
    return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

template <bool COMPACT>
__device__ __forceinline__ Window<COMPACT> decode_window(const FwdArgs &a, const RawWindow &r, int e, int bound,
                                                         int vb, int lane) {
    Window<COMPACT> win;
    win.n = 0;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int o = r.o[h];
        const bool in = r.base + h * kWave + lane < e && o < bound;
        const int c = (int)fast_div((uint32_t)o, a.magic, a.shift);
        // LDS index of the tap for virtual pixel 0: channel slot c*PLp, then
        // the tap (r, s) at r*vp + s + lds_shift (o - c*Hp*Wp = r*Wp + s).
        const int tap_row = (int)fast_div((uint32_t)(o - c * a.Hp * a.Wp), a.wp_magic, a.wp_shift);
        const int t = vb + o - c * a.plane_delta + tap_row * (a.vp - a.Wp) + a.lds_shift;
        const int odd = t & 1;
        const uint64_t me = __builtin_amdgcn_ballot_w64(in && !odd);
        const uint64_t mo = __builtin_amdgcn_ballot_w64(in && odd);
        const int ne = __builtin_popcountll(me), no = __builtin_popcountll(mo);
        if constexpr (COMPACT) {
            // Destination lane: even taps first, then odd ones, then the lanes
            // outside the chunk (a permutation of the 64 lanes).
            const int be = lanes_below(me), bo = ne + lanes_below(mo), bx = ne + no + lanes_below(~(me | mo));
            const int dst = in ? (odd ? bo : be) : bx;
            win.lo[h] = __builtin_amdgcn_ds_permute(dst * 4, t - odd);
            win.w[h] = __int_as_float(__builtin_amdgcn_ds_permute(dst * 4, __float_as_int(r.w[h])));
            win.ne[h] = ne;
            win.no[h] = no;
        } else {
            win.lo[h] = t - odd;
            // Touch the loaded weight here, so that the wait for its load is
            // placed at this decode and not deferred into the compute loop,
            // where it would also wait for the chunk copies in flight.
            float w = r.w[h];
            asm volatile("" : "+v"(w));
            win.w[h] = w;
            win.even[h] = me;
            win.odd[h] = mo;
        }
        win.n += ne + no;
    }
    return win;
}

// Pixel pairs of one tap: x[im][j] = the two floats at LDS index ad + 128*j of
// image block im (ad even, so every read is one aligned ds_read_b64).
// The loads are volatile LDS accesses of a clang vector type:
//  * volatile keeps the compiler from fusing two of them into one
//    ds_read2st64_b64, which gfx950 serves at half the bandwidth of two
//    ds_read_b64 (about 127 vs 230-250 bytes per clock per CU);
//  * a vector type rather than HIP's float2 struct, because through the
//    struct the compiler also waits for the chunk copies in flight before
//    each read.
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef const volatile __attribute__((address_space(3))) f32x2 lds_pair_t;

template <int PJ, int IPW>
__device__ __forceinline__ void load_pairs(f32x2 (&x)[IPW][PJ], const float *lds, int ad, int img_lds) {
#pragma unroll
    for (int im = 0; im < IPW; ++im)
#pragma unroll
        for (int p = 0; p < PJ; ++p) x[im][p] = *(lds_pair_t *)(lds + ad + im * img_lds + 2 * kWave * p);
}

template <int PJ, int IPW>
__device__ __forceinline__ void fma_pairs(float2 (&acc)[IPW][PJ], const f32x2 (&x)[IPW][PJ], float v) {
#pragma unroll
    for (int im = 0; im < IPW; ++im)
#pragma unroll
        for (int p = 0; p < PJ; ++p) {
            acc[im][p].x = fmaf(v, x[im][p].x, acc[im][p].x);
            acc[im][p].y = fmaf(v, x[im][p].y, acc[im][p].y);
        }
}

__device__ __forceinline__ int lane_read_i(int v, int l) { return __builtin_amdgcn_readlane(v, l); }
__device__ __forceinline__ float lane_read_f(float v, int l) {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
}

// Accumulate the window entries whose lanes are set in mask m into acc, in
// lane order (scalar find-first-set); the same pipeline as run_range below.
template <int NB, int PJ, int IPW>
__device__ __forceinline__ void run_mask(float2 (&acc)[IPW][PJ], int lo, float w, uint64_t m, const float *lds,
                                         int q, int img_lds) {
    int r = __builtin_popcountll(m);
    if (r == 0) return;
    f32x2 x[NB][IPW][PJ];
    float wt[NB];
    auto next = [&](f32x2 (&xb)[IPW][PJ], float &wb) {
        const int u = __builtin_ctzll(m);
        m &= m - 1;
        wb = lane_read_f(w, u);
        load_pairs(xb, lds, lane_read_i(lo, u) + q, img_lds);
    };
#pragma unroll
    for (int b = 0; b < NB - 1; ++b)
        if (b < r) next(x[b], wt[b]);
    for (; r >= 2 * NB - 1; r -= NB) {
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            next(x[(b + NB - 1) % NB], wt[(b + NB - 1) % NB]);
            fma_pairs(acc, x[b], wt[b]);
            __builtin_amdgcn_sched_barrier(0);
        }
    }
#pragma unroll
    for (int b = 0; b < 2 * NB - 2; ++b) {
        if (b >= r) break;
        if (b + NB - 1 < r) next(x[(b + NB - 1) % NB], wt[(b + NB - 1) % NB]);
        fma_pairs(acc, x[b % NB], wt[b % NB]);
        __builtin_amdgcn_sched_barrier(0);
    }
}

// Accumulate window entries j0..j1-1 (compacted lanes) into acc. Software
// pipeline of NB buffers: the LDS reads of the next NB-1 entries are in
// flight while the FMAs of the current one issue. Each entry's reads then
// have NB-1 entries' worth of this wave's FMAs to arrive; tilings with few
// pixels per lane (few FMAs per entry) need the deeper pipelines. Buffer
// indices are compile-time constants in the unrolled bodies, so the buffers
// stay in registers; the scheduling barriers keep each refill after the FMAs
// that read the buffer it overwrites. The main loop has no exit in the
// middle, so the accumulators stay in place.
template <int NB, int PJ, int IPW>
__device__ __forceinline__ void run_range(float2 (&acc)[IPW][PJ], int lo, float w, int j, int j1, const float *lds,
                                          int q, int img_lds) {
    int r = j1 - j;
    if (r <= 0) return;
    f32x2 x[NB][IPW][PJ];
    float wt[NB];
    auto next = [&](f32x2 (&xb)[IPW][PJ], float &wb) {
        wb = lane_read_f(w, j);
        load_pairs(xb, lds, lane_read_i(lo, j) + q, img_lds);
        ++j;
    };
#pragma unroll
    for (int b = 0; b < NB - 1; ++b)
        if (b < r) next(x[b], wt[b]);
    // Invariant: buffers 0..NB-2 hold the next NB-1 entries; an iteration
    // loads the NB after them, so at least 2*NB - 1 must remain.
    for (; r >= 2 * NB - 1; r -= NB) {
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            next(x[(b + NB - 1) % NB], wt[(b + NB - 1) % NB]);
            fma_pairs(acc, x[b], wt[b]);
            __builtin_amdgcn_sched_barrier(0);
        }
    }
#pragma unroll
    for (int b = 0; b < 2 * NB - 2; ++b) {
        if (b >= r) break;
        if (b + NB - 1 < r) next(x[(b + NB - 1) % NB], wt[(b + NB - 1) % NB]);
        fma_pairs(acc, x[b % NB], wt[b % NB]);
        __builtin_amdgcn_sched_barrier(0);
    }
}

// Walk of one list of a lowered stream: n entries (LDS index of the pixel
// pair read for virtual pixel 0 of the chunk, weight bits) from entry j on,
// accumulated into acc. Entries arrive in batches of kLwBatch with one scalar
// load each, so index and weight are wave-uniform SGPRs: an entry costs one
// address add and its FMAs (the weight is the FMAs' scalar operand), no
// broadcast. Software pipeline of NB pixel-pair buffers as in run_range; the
// next batch is loaded one entry before its first use, so its scalar load
// overlaps one entry's FMAs (scalar loads complete out of order with LDS
// reads, so the first LDS wait after it waits for both). The main loop's body
// has no branch (a branch would let the compiler move every FMA of the batch
// behind its reads, with register copies between); list ends are handled in a
// guarded tail.
// Calls f(integral_constant<int, U>) for U = I, I+1, ... below END while it
// returns true: a loop unrolled at compile time, with a constant index.
template <int I, int END, typename F>
__device__ __forceinline__ void unroll_while(F &&f) {
    if constexpr (I < END) {
        if (f(std::integral_constant<int, I>{})) unroll_while<I + 1, END>(f);
    }
}

template <int B>
struct LwBatch {
    int v[2 * B];
};

template <int NB, int PJ, int IPW>
__device__ __forceinline__ void run_lowered(float2 (&acc)[IPW][PJ], const int32_t *__restrict__ ent, int j, int n,
                                            const float *lds, int qv, int img_lds) {
    if (n <= 0) return;
    constexpr int B = kLwBatch;
    static_assert(B % NB == 0, "buffer rotation must repeat every batch");
    // With few reads per entry (two pixel pairs or fewer), the reads of the
    // entries after the list's end are issued too, in place of a scalar test
    // and branch per entry: they are the next lists' entries (or the stream's
    // zero pad), LDS indices of the same chunk window, and their values are
    // never used.
    constexpr bool kEager = IPW * PJ <= 2;
    // This lane's window base: an entry's address is one shift-add on it.
    const float *lb = lds + qv;
    f32x2 x[NB][IPW][PJ];
    LwBatch<B> b = *reinterpret_cast<const LwBatch<B> *>(ent + 2 * j);
#pragma unroll
    for (int u = 0; u < NB - 1; ++u)
        if (kEager || u < n) load_pairs(x[u], lb, b.v[2 * u], img_lds);
    int r = n;
    // Main loop, branch free: a whole batch, and the NB - 1 entries whose
    // reads issue ahead of it all exist (the first of them come from the
    // next batch), or, eager, are read whether they exist or not.
    for (; r >= (kEager ? B : B + NB - 1); r -= B) {
        LwBatch<B> nb;
#pragma unroll
        for (int u = 0; u < B; ++u) {
            if (u == B - NB) nb = *reinterpret_cast<const LwBatch<B> *>(ent + 2 * (j + B));
            const int f = u + NB - 1;  // entry whose reads issue now
            load_pairs(x[f % NB], lb, f < B ? b.v[2 * f] : nb.v[2 * (f - B)], img_lds);
            fma_pairs(acc, x[u % NB], __int_as_float(b.v[2 * u + 1]));
            __builtin_amdgcn_sched_barrier(0);
        }
        b = nb;
        j += B;
    }
    // Tail: r < B + NB - 1 entries, the first min(r, NB - 1) in flight; past
    // entry B - 1 they come from the next batch. That batch is loaded
    // whether or not the list reaches it (a conditional load would not stay
    // scalar); the stream's pad of two batches keeps it inside the stream.
    const LwBatch<B> nb = *reinterpret_cast<const LwBatch<B> *>(ent + 2 * (j + B));
    // Unrolled at compile time (a loop with this early exit is not), so every
    // batch index is a constant and the batches stay in SGPRs.
    unroll_while<0, B + NB - 1>([&](auto U) {
        constexpr int u = decltype(U)::value;
        constexpr int f = u + NB - 1;
        if (u >= r) return false;
        if (kEager || f < r) {
            if constexpr (f < B)
                load_pairs(x[f % NB], lb, b.v[2 * f], img_lds);
            else
                load_pairs(x[f % NB], lb, nb.v[2 * (f - B)], img_lds);
        }
        float w;
        if constexpr (u < B)
            w = __int_as_float(b.v[2 * u + 1]);
        else
            w = __int_as_float(nb.v[2 * (u - B) + 1]);
        fma_pairs(acc, x[u % NB], w);
        __builtin_amdgcn_sched_barrier(0);
        return true;
    });
}

// Pipeline depth of the stride-1 kernel: deeper for fewer FMAs per entry
// (IPW * PI), where the 128 VGPRs of four waves per SIMD hold the buffers
// (accumulators plus buffers within 98 floats, at most two channels a wave:
// each channel's window state takes registers too).
template <int PI, int IPW, int RPW>
constexpr int pipeline_buffers() {
    const int want = IPW * PI <= 8 ? 3 : 2;
    for (int nb = want; nb > 2; --nb)
        if (RPW <= 2 && 2 * RPW * IPW * PI + nb * IPW * PI <= 98) return nb;
    return 2;
}

// Sums of this lane's virtual pixel pairs (2l + 128j, 2l+1 + 128j) of one
// image: the even-tap pairs plus the odd-tap pairs, which are shifted by one
// pixel (lane l holds pixels 2l-1 and 2l). Pixel 2l+1 takes the odd pair of
// lane l+1; lane 63 takes lane 0 of pair j+1. The last virtual pixel of the
// tile (lane 63, last pair) has no such source: the planner keeps every tile
// below 64*PI pixels, so that pixel is never stored.
template <int PJ>
__device__ __forceinline__ void merge_pairs(const float2 (&e)[PJ], const float2 (&o)[PJ], float2 (&v)[PJ], int lane) {
    const int src = ((lane + 1) & (kWave - 1)) * 4;
    float rot[PJ];
#pragma unroll
    for (int p = 0; p < PJ; ++p) rot[p] = __int_as_float(__builtin_amdgcn_ds_bpermute(src, __float_as_int(o[p].x)));
#pragma unroll
    for (int p = 0; p < PJ; ++p) {
        const float next = p + 1 < PJ ? rot[p + 1] : 0.0f;
        const float right = lane == kWave - 1 ? next : rot[p];
        v[p] = make_float2(e[p].x + o[p].y, e[p].y + right);
    }
}

// Issue priority (0 lowest .. 3 highest) from a wave's progress through its
// entries of the current chunk. Among ready waves of equal priority a SIMD
// issues the oldest first, so left alone the oldest wave of each SIMD runs
// ahead, the youngest finishes every chunk alone at a fraction of the SIMD's
// rate, and the others idle at the chunk barrier. Dropping one level per
// quarter of the chunk done lets the waves that are behind issue first, and
// the four waves of a SIMD reach the barrier nearly together.
__device__ __forceinline__ void set_progress_prio(int done, int total) {
    const int d4 = 4 * done;
    if (d4 >= 3 * total)
        __builtin_amdgcn_s_setprio(0);
    else if (d4 >= 2 * total)
        __builtin_amdgcn_s_setprio(1);
    else if (d4 >= total)
        __builtin_amdgcn_s_setprio(2);
    else
        __builtin_amdgcn_s_setprio(3);
}

// Pipeline depth of the lowered walk: a divisor of its batch, four buffers for
// tilings with few FMAs per entry where the registers hold them.
template <int PI, int IPW, int RPW>
constexpr int lowered_pipeline_buffers() {
    return (IPW * PI <= 8 && 2 * RPW * IPW * PI + 4 * IPW * PI <= 80) ? 4 : 2;
}

// Epilogue of one tile of the stride-1 kernel: bias, residual, ReLU, then the
// stores (or the 2x2 pool through a wave-private LDS staging tile), and the
// zero border of bordered outputs. accE/accO hold the even- and odd-tap sums of
// the wave's RPW channels krow over the tile (images ig*IPW.., rows y0..).
// The pooled form reuses the chunk buffers: every wave must be past its last
// read of them (a barrier) before the call.
//
// Pooled staging: with an even tile pitch (a.pool_pairs) a lane's pixel pair
// (2l, 2l+1) + 128j is one horizontal pool pair, so each wave stages only
// the pair maxima (64 * PI/2 floats per image) at `stage`, and a pooled output
// takes the larger of two staged maxima one pitch apart (the same maxima as
// over the four pixels, same bits). Otherwise whole activated tiles are staged
// from `lds` on, over both chunk buffers.
template <int PI, int IPW, int RPW, bool POOL>
__device__ __forceinline__ void s1_epilogue(const FwdArgs &a, float2 (&accE)[RPW][IPW][PI / 2],
                                            float2 (&accO)[RPW][IPW][PI / 2], const int (&krow)[RPW], int ig, int ty,
                                            int y0, int phi, int wave, int lane, float *lds, float *stage,
                                            const float *__restrict__ bias, const float *__restrict__ res,
                                            float *__restrict__ out) {
    constexpr int PJ = PI / 2;
    const int q = 2 * lane;
    const int tile_px = a.TH * a.vp;
    if constexpr (!POOL) {
        // Tile row of each of this lane's pixels, or -1 when the pixel is not
        // stored (outside the output, or past a row-spanning tile's span). The
        // tile starts at column phi of row y0 (0 for whole-row tiles): tile
        // pixel qq is pixel qa = qq + phi = yl*vp + x counted from row y0, and
        // lands at qa + yl*(pitch - vp) past that row's first element, in the
        // output and the residual alike.
        const int span = a.span ? a.span : tile_px;
        int ylo[PJ][2];
#pragma unroll
        for (int p = 0; p < PJ; ++p)
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int qq = q + 2 * kWave * p + h, qa = qq + phi;
                const int yl = (int)fast_div((uint32_t)qa, a.vp_magic, a.vp_shift), x = qa - yl * a.vp;
                ylo[p][h] = (qq < span && x < a.Wo && y0 + yl < a.Ho) ? yl : -1;
            }
        const int odelta = a.opitch - a.vp, rdelta = a.rpitch - a.vp;
#pragma unroll
        for (int i = 0; i < RPW; ++i) {
            const int k = krow[i];
            if (k >= a.K) continue;
            const float bk = bias ? bias[k] : 0.0f;
#pragma unroll
            for (int im = 0; im < IPW; ++im) {
                const int n = ig * IPW + im;
                if (n >= a.N) break;
                float *plane = out + ((size_t)n * a.K + k) * a.oplane;
                float *op = plane + (size_t)(y0 + a.out_pad) * a.opitch + a.out_pad;
                const float *rp =
                    res ? res + ((size_t)n * a.K + k) * a.rplane + (size_t)(y0 + a.res_pad) * a.rpitch + a.res_pad
                        : nullptr;
                float2 sum[PJ];
                merge_pairs(accE[i][im], accO[i][im], sum, lane);
                if (a.pair_store) {
#pragma unroll
                    for (int p = 0; p < PJ; ++p) {
                        const int yl = ylo[p][0];
                        if (yl < 0) continue;
                        const int qq = q + 2 * kWave * p + phi;
                        float2 v = make_float2(sum[p].x + bk, sum[p].y + bk);
                        if (rp) {
                            const f32x2_a4_t r = *reinterpret_cast<const f32x2_a4_t *>(rp + qq + yl * rdelta);
                            v.x += r.x;
                            v.y += r.y;
                        }
                        if (a.relu) {
                            v.x = v.x > 0.0f ? v.x : 0.0f;
                            v.y = v.y > 0.0f ? v.y : 0.0f;
                        }
                        store_out2(op + qq + yl * odelta, v, a.out_pad == 0);
                    }
                } else {
#pragma unroll
                for (int p = 0; p < PJ; ++p)
#pragma unroll
                    for (int h = 0; h < 2; ++h) {
                        const int yl = ylo[p][h];
                        if (yl < 0) continue;
                        const int qq = q + 2 * kWave * p + h + phi;
                        float v = (h ? sum[p].y : sum[p].x) + bk;
                        if (rp) v += rp[qq + yl * rdelta];
                        if (a.relu) v = v > 0.0f ? v : 0.0f;
                        store_out(op + qq + yl * odelta, v, a.out_pad == 0);
                    }
                }
                if (a.out_pad) {
                    // The side borders of the rows whose column 0 lies in this
                    // tile (its whole rows: rows y0 .. y0 + TH - 1).
                    int r0 = y0, r1 = min(y0 + a.TH, a.Ho);
                    if (a.span) {
                        r0 = y0 + (phi > 0 ? 1 : 0);
                        r1 = min((int)fast_div((uint32_t)(y0 * a.vp + phi + a.span + a.vp - 1), a.vp_magic,
                                               a.vp_shift),
                                 a.Ho);
                    }
                    zero_border(plane, r0, max(r0, r1), a.Ho, a.Wo, a.out_pad, a.opitch, ty == 0,
                                ty == a.ntiles_y - 1, lane, kWave);
                }
            }
        }
    } else if (a.pool_pairs) {
        // Pair maxima, staged per wave (see above); only the wave's own LDS
        // order matters, and the last barrier of the chunk loop ordered these
        // writes after every wave's reads of the staging buffer.
        constexpr int kImgPairs = kWave * PJ;
        float *st = stage + wave * IPW * kImgPairs;
        const int prow0 = y0 / 2;
        const int prows = a.TH / 2;
        const int per_img = prows * a.Wq;
        const int half = a.vp / 2;
#pragma unroll
        for (int i = 0; i < RPW; ++i) {
            const int k = krow[i];
            const float bk = (k < a.K && bias) ? bias[k] : 0.0f;
#pragma unroll
            for (int im = 0; im < IPW; ++im) {
                float2 sum[PJ];
                merge_pairs(accE[i][im], accO[i][im], sum, lane);
                const int n = ig * IPW + im;
                const float *rp = (res && k < a.K && n < a.N)
                                      ? res + ((size_t)n * a.K + k) * a.rplane +
                                            (size_t)(y0 + a.res_pad) * a.rpitch + a.res_pad
                                      : nullptr;
#pragma unroll
                for (int p = 0; p < PJ; ++p) {
                    float v[2] = {sum[p].x + bk, sum[p].y + bk};
                    if (rp) {
#pragma unroll
                        for (int h = 0; h < 2; ++h) {
                            const int qq = q + 2 * kWave * p + h;
                            const int yl = (int)fast_div((uint32_t)qq, a.vp_magic, a.vp_shift), x = qq - yl * a.vp;
                            if (qq < tile_px && x < a.Wo && y0 + yl < a.Ho) v[h] += rp[qq + yl * (a.rpitch - a.vp)];
                        }
                    }
                    if (a.relu) {
                        v[0] = v[0] > 0.0f ? v[0] : 0.0f;
                        v[1] = v[1] > 0.0f ? v[1] : 0.0f;
                    }
                    st[im * kImgPairs + lane + kWave * p] = fmaxf(v[0], v[1]);
                }
            }
            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // the pair maxima are staged
            if (k < a.K) {
                for (int t = lane; t < IPW * per_img; t += kWave) {
                    const int im = (int)fast_div((uint32_t)t, a.pimg_magic, a.pimg_shift);
                    const int rem = t - im * per_img;
                    const int r = (int)fast_div((uint32_t)rem, a.wq_magic, a.wq_shift);
                    const int jq = rem - r * a.Wq;
                    const int n = ig * IPW + im;
                    const int pr = prow0 + r;
                    if (n < a.N && pr < a.Hq) {
                        const float *s0 = st + im * kImgPairs + r * a.vp + jq;
                        const float m = fmaxf(s0[0], s0[half]);
                        store_out(out + ((size_t)n * a.K + k) * a.oplane + (size_t)(pr + a.out_pad) * a.opitch + jq +
                                      a.out_pad,
                                  m, a.out_pad == 0);
                    }
                }
                if (a.out_pad)
                    for (int im = 0; im < IPW; ++im) {
                        const int n = ig * IPW + im;
                        if (n >= a.N) break;
                        zero_border(out + ((size_t)n * a.K + k) * a.oplane, prow0, min(prow0 + prows, a.Hq), a.Hq,
                                    a.Wq, a.out_pad, a.opitch, ty == 0, ty == a.ntiles_y - 1, lane, kWave);
                    }
            }
        }
    } else {
        // Each wave stages its own rows' activated tiles (all images) in LDS,
        // then reduces 2x2 windows; no other wave touches that area, so only
        // the wave's own LDS order matters (its LDS operations execute in
        // issue order). The last barrier of the chunk loop ordered these
        // writes after every read of the input buffers by any wave.
        constexpr int kImgPx = kWave * PI;
        float *st = lds + wave * IPW * kImgPx;
        const int prow0 = y0 / 2;
        const int prows = a.TH / 2;
        const int per_img = prows * a.Wq;
#pragma unroll
        for (int i = 0; i < RPW; ++i) {
            const int k = krow[i];
            const float bk = (k < a.K && bias) ? bias[k] : 0.0f;
#pragma unroll
            for (int im = 0; im < IPW; ++im) {
                float2 sum[PJ];
                merge_pairs(accE[i][im], accO[i][im], sum, lane);
                const int n = ig * IPW + im;
                // The residual is added on the convolution's grid, before the
                // activation and the pool; pixels outside the plane get none.
                const float *rp = (res && k < a.K && n < a.N)
                                      ? res + ((size_t)n * a.K + k) * a.rplane +
                                            (size_t)(y0 + a.res_pad) * a.rpitch + a.res_pad
                                      : nullptr;
#pragma unroll
                for (int p = 0; p < PJ; ++p) {
                    float v[2] = {sum[p].x + bk, sum[p].y + bk};
                    if (rp) {
#pragma unroll
                        for (int h = 0; h < 2; ++h) {
                            const int qq = q + 2 * kWave * p + h;
                            const int yl = (int)fast_div((uint32_t)qq, a.vp_magic, a.vp_shift), x = qq - yl * a.vp;
                            if (qq < tile_px && x < a.Wo && y0 + yl < a.Ho) v[h] += rp[qq + yl * (a.rpitch - a.vp)];
                        }
                    }
                    if (a.relu) {
                        v[0] = v[0] > 0.0f ? v[0] : 0.0f;
                        v[1] = v[1] > 0.0f ? v[1] : 0.0f;
                    }
                    *reinterpret_cast<float2 *>(st + im * kImgPx + q + 2 * kWave * p) = make_float2(v[0], v[1]);
                }
            }
            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // the whole tile is staged
            if (k < a.K) {
                for (int t = lane; t < IPW * per_img; t += kWave) {
                    const int im = (int)fast_div((uint32_t)t, a.pimg_magic, a.pimg_shift);
                    const int rem = t - im * per_img;
                    const int r = (int)fast_div((uint32_t)rem, a.wq_magic, a.wq_shift);
                    const int jq = rem - r * a.Wq;
                    const int n = ig * IPW + im;
                    const int pr = prow0 + r;
                    if (n < a.N && pr < a.Hq) {
                        const float *s0 = st + im * kImgPx + (2 * r) * a.vp + 2 * jq;
                        const float m = fmaxf(fmaxf(s0[0], s0[1]), fmaxf(s0[a.vp], s0[a.vp + 1]));
                        store_out(out + ((size_t)n * a.K + k) * a.oplane + (size_t)(pr + a.out_pad) * a.opitch + jq +
                                      a.out_pad,
                                  m, a.out_pad == 0);
                    }
                }
                if (a.out_pad)
                    for (int im = 0; im < IPW; ++im) {
                        const int n = ig * IPW + im;
                        if (n >= a.N) break;
                        zero_border(out + ((size_t)n * a.K + k) * a.oplane, prow0, min(prow0 + prows, a.Hq), a.Hq,
                                    a.Wq, a.out_pad, a.opitch, ty == 0, ty == a.ntiles_y - 1, lane, kWave);
                    }
            }
        }
    }
}

// Stride-1 kernel with a lowered entry stream (see FwdArgs): the workgroup
// takes work items (channel tile, spatial tile, image group) b, b + G, b + 2G,
// ... of the T = a.total_wgs items in the grid of G workgroups (one per CU
// when T exceeds the CUs), so the copies and stores at a tile's edges overlap
// the arithmetic of its neighbours: the chunk copies run as one stream across
// tiles (chunk buffer = global chunk count & 1), the next tile's first chunk
// is copied during the current tile's last chunk, and the current tile's
// stores drain while the next tile computes. With the pooled epilogue, whose
// staging tile reuses the chunk buffers, the next tile's first copy follows
// the epilogue. At iteration t the workgroup takes item t*G + its XCD-ordered
// index within that round, so the workgroups of one XCD work on neighbouring
// tiles (shared input rows in that XCD's L2), as in a one-tile-per-workgroup
// grid.
template <int PI, int IPW, int RPW, bool POOL, bool PERSIST>
__device__ __forceinline__ void s1_lowered_tiles(const FwdArgs &a, const float *__restrict__ xp,
                                                 const int32_t *__restrict__ lw, const float *__restrict__ bias,
                                                 const float *__restrict__ res, float *__restrict__ out, float *lds) {
    constexpr int PJ = PI / 2;
    constexpr int NBL = lowered_pipeline_buffers<PI, IPW, RPW>();
    const int wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
    const int lane = (int)threadIdx.x & 63;
    const int q = 2 * lane;
    const int G = (int)gridDim.x, T = a.total_wgs, b = (int)blockIdx.x;
    const int32_t *ent = lw + 4 * (size_t)a.lw_headers;
    auto header = [&](int kt, int i, int ch) {
        return *reinterpret_cast<const int4 *>(lw + 4 * (size_t)(((kt * kS1Waves + wave) * RPW + i) * a.nchunks + ch));
    };
    struct Item {
        int kt, ty, ig;
    };
    // First output row of tile ty (= first staged padded input row). A
    // row-spanning tile starts at column phi of that row and stages the window
    // from column phi rounded down to a multiple of 4.
    auto row0_of = [&](int ty) {
        return a.span ? (int)fast_div((uint32_t)(ty * a.span), a.vp_magic, a.vp_shift) : ty * a.TH;
    };
    auto col0_of = [&](int ty, int row0) { return a.span ? (ty * a.span - row0 * a.vp) & ~3 : 0; };
    // Round it holds items it*G .. min((it+1)*G, T) - 1; workgroup b takes
    // the one at its XCD-ordered position among that round's (b is below
    // the round's size whenever the round has an item for it).
    auto item_of = [&](int it) {
        const int L = it * G + xcd_linear_id(b, min(G, T - it * G));
        Item r;
        r.kt = L % a.nktiles;
        const int t = L / a.nktiles;
        r.ty = t % a.ntiles_y;
        r.ig = t / a.ntiles_y;
        return r;
    };
    if (b >= T) return;
    // Pull this wave's entry lists of an item (contiguous in the stream, from
    // its first list on: pf_bytes covers RPW rows with a margin) into the L2
    // ahead of the walk's scalar loads, which otherwise miss to HBM batch by
    // batch on a cold stream (narrow 14x14 layer at density 0.2: 95 -> 72 us
    // after a cache flush). One 4-byte LDS-DMA read per lane at 128-byte steps
    // touches 64 cache lines (8 KiB) per instruction; the data land in a sink
    // at the end of the LDS that nothing reads.
    auto prefetch_stream = [&](int first) {
        const int e0 = min(max(first, 0), a.lw_entries);
        const uint32_t bytes = min((uint32_t)(a.lw_entries - e0) * 8u, (uint32_t)a.pf_bytes);
        __amdgpu_buffer_rsrc_t rsrc =
            __builtin_amdgcn_make_buffer_rsrc((void *)(ent + 2 * (size_t)e0), (short)0, (int)bytes, 0x00020000);
        float *sink = lds + (a.lds_floats - kLwSinkFloats);
        for (uint32_t off = 0; off < bytes && off < 4u * 8192u; off += 8192u)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (lds_void_t *)sink, 4, off + (uint32_t)lane * 128u, 0, 0, 0);
    };
    Item cur = item_of(0);
    {
        const int r0 = row0_of(cur.ty);
        stage_chunk_s1(a, xp, lds, 0, cur.ig, r0, wave, lane, col0_of(cur.ty, r0));
    }
    wait_async_copies();
    __syncthreads();
    int sbuf = 0;  // buffer of the chunk being computed
    for (int it = 0;; ++it) {
        const bool has_next = PERSIST && (it + 1) * G + b < T;
        const Item nxt = has_next ? item_of(it + 1) : cur;
        const int y0 = row0_of(cur.ty);
        const int phi = a.span ? cur.ty * a.span - y0 * a.vp : 0;
        const int col0 = phi & ~3;
        const int nrow0 = row0_of(nxt.ty), ncol0 = col0_of(nxt.ty, nrow0);
        int krow[RPW];
        int4 h[RPW];
#pragma unroll
        for (int i = 0; i < RPW; ++i) {
            h[i] = header(cur.kt, i, 0);
            krow[i] = h[i].w;
        }
        prefetch_stream(h[0].x);
        float2 accE[RPW][IPW][PJ], accO[RPW][IPW][PJ];
#pragma unroll
        for (int i = 0; i < RPW; ++i)
#pragma unroll
            for (int im = 0; im < IPW; ++im)
#pragma unroll
                for (int pp = 0; pp < PJ; ++pp) {
                    accE[i][im][pp] = make_float2(0.0f, 0.0f);
                    accO[i][im][pp] = make_float2(0.0f, 0.0f);
                }
        for (int ch = 0; ch < a.nchunks; ++ch) {
            const bool more = ch + 1 < a.nchunks;
            // The copy of the next chunk (or of the next tile's first). The
            // oldest wave of each SIMD issues its share before its walk, the
            // other three halfway through their lists (after the first row's
            // two lists, or after the even list of a single row): issued all
            // at once, some 80 one-KiB copies queue at the CU's texture path
            // and hold the younger waves up to 2 us at the issue; spread this
            // way the copy still lands well before the chunk ends.
            float *nbuf = lds + (sbuf ^ 1) * a.buf_floats;
            const bool do_stage = more || ((!POOL || a.pool_in_buf) && has_next);
            const int s_ch = more ? ch + 1 : 0, s_ig = more ? cur.ig : nxt.ig;
            const int s_row = more ? y0 : nrow0, s_col = more ? col0 : ncol0;
            constexpr int kLateList = RPW > 1 ? 2 : 1;  // list before which the younger waves issue
            const bool early = wave < 4;  // wave w runs on SIMD w % 4, and waves 0..3 are the oldest
            if (do_stage && early) stage_chunk_s1(a, xp, nbuf, s_ch, s_ig, s_row, wave, lane, s_col);
            // Entry lists of this chunk, clamped to the stream.
            int st[RPW], ne[RPW], no[RPW];
            int total = 0, done = 0;
#pragma unroll
            for (int i = 0; i < RPW; ++i) {
                st[i] = min(max(h[i].x, 0), a.lw_entries);
                ne[i] = min(max(h[i].y, 0), a.lw_entries - st[i]);
                no[i] = min(max(h[i].z, 0), a.lw_entries - st[i] - ne[i]);
                total += ne[i] + no[i];
            }
            // The window starts col0 before the tile's first pixel.
            const int qv = sbuf * a.buf_floats + q + (phi - col0);
            set_progress_prio(0, total);
#pragma unroll
            for (int i = 0; i < RPW; ++i) {
                run_lowered<NBL>(accE[i], ent, st[i], ne[i], lds, qv, a.img_lds);
                done += ne[i];
                if (2 * i + 1 == kLateList && do_stage && !early)
                    stage_chunk_s1(a, xp, nbuf, s_ch, s_ig, s_row, wave, lane, s_col);
                set_progress_prio(done, total);
                run_lowered<NBL>(accO[i], ent, st[i] + ne[i], no[i], lds, qv, a.img_lds);
                done += no[i];
                if (2 * i + 2 == kLateList && do_stage && !early)
                    stage_chunk_s1(a, xp, nbuf, s_ch, s_ig, s_row, wave, lane, s_col);
                set_progress_prio(done, total);
            }
            if (more) {
#pragma unroll
                for (int i = 0; i < RPW; ++i) h[i] = header(cur.kt, i, ch + 1);
            }
            // The next chunk (or the next tile's first) is in LDS and every
            // wave is done with this chunk's buffer (or, before the pooled
            // epilogue, with both).
            if (more || POOL || has_next) {
                wait_async_copies();
                __syncthreads();
            }
            sbuf ^= 1;
        }
        // The pooled staging goes to the buffer of the last chunk (now free)
        // when it fits there, else over both buffers.
        float *stage = (POOL && a.pool_in_buf) ? lds + (sbuf ^ 1) * a.buf_floats : lds;
        // The epilogue at the highest issue priority: a wave leaves its last
        // chunk at the lowest, and the waves that reach their stores last
        // would otherwise queue behind the others' walk of the next item
        // (VGG conv1 -2%, same bits).
        __builtin_amdgcn_s_setprio(3);
        s1_epilogue<PI, IPW, RPW, POOL>(a, accE, accO, krow, cur.ig, cur.ty, y0, phi, wave, lane, lds, stage, bias,
                                        res, out);
        if (!has_next) break;
        if (POOL && a.pool_in_buf) {
            // The next tile's first chunk is in the other buffer; its second
            // chunk's copy into the staging buffer waits for every wave's
            // pooled reads.
            __syncthreads();
        } else if constexpr (POOL) {
            // The staging tile overlaps the buffers: the next tile's first
            // chunk is copied after every wave's pooled stores.
            __syncthreads();
            stage_chunk_s1(a, xp, lds + sbuf * a.buf_floats, 0, nxt.ig, nrow0, wave, lane, ncol0);
            wait_async_copies();
            __syncthreads();
        }
        cur = nxt;
    }
}

// MODE: kModePlain walks the CSR rows (rowptr/offset/vals); kModeLowered and
// kModeTiled read the lowered entry stream (lw, see FwdArgs) instead: rows are
// assigned to waves by the stream's headers and each (row, chunk) is two
// ready lists of (LDS index, weight) per tap parity; kModeTiled runs several
// work items per workgroup (s1_lowered_tiles).
constexpr int kModePlain = 0, kModeLowered = 1, kModeTiled = 2;

template <int PI, int IPW, int RPW, bool POOL, int MODE>
__global__ __launch_bounds__(kS1Threads) __attribute__((amdgpu_waves_per_eu(4, 4))) void spconv_s1_kernel(
    FwdArgs a, const float *__restrict__ xp, const int32_t *__restrict__ rowptr, const int32_t *__restrict__ offset,
    const float *__restrict__ vals, const int32_t *__restrict__ lw, const float *__restrict__ bias,
    const float *__restrict__ res, float *__restrict__ out) {
    extern __shared__ float lds[];
    constexpr int KT = RPW * kS1Waves;  // output channels per workgroup
    constexpr int PJ = PI / 2;          // pixel pairs per lane per image
    static_assert(PI % 2 == 0, "pixels per lane come in pairs");
    constexpr int NB = pipeline_buffers<PI, IPW, RPW>();
    constexpr bool kCompact = NB > 2;  // compacted windows where entries have few FMAs
    if constexpr (MODE != kModePlain) {
        s1_lowered_tiles<PI, IPW, RPW, POOL, MODE == kModeTiled>(a, xp, lw, bias, res, out, lds);
        return;
    }

    const int L = xcd_linear_id((int)blockIdx.x, a.total_wgs);
    const int wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
    const int lane = (int)threadIdx.x & 63;
    const int kt = L % a.nktiles;
    const int tile = L / a.nktiles;
    const int ty = tile % a.ntiles_y;
    const int ig = tile / a.ntiles_y;
    const int y0 = ty * a.TH;
    const int plane = a.Hp * a.Wp;

    // Output channels of this wave. With RPW > 1 the workgroup's KT channels
    // are ranked by nonzero count and dealt to the waves in snake order (ranks
    // w, 2*16-1-w, 2*16+w, ...), so heavy and light channels share a wave and
    // the waves' loads even out.
    int krow[RPW];
    if constexpr (RPW == 1) {
        krow[0] = kt * KT + wave;
    } else {
        const int k0 = kt * KT;
        int nz = -1;
        if (lane < KT && k0 + lane < a.K) nz = rowptr[k0 + lane + 1] - rowptr[k0 + lane];
        int rank = 0;
        for (int j = 0; j < KT; ++j) {
            const int o = __builtin_amdgcn_readlane(nz, j);
            rank += (o > nz || (o == nz && j < lane)) ? 1 : 0;
        }
#pragma unroll
        for (int i = 0; i < RPW; ++i) {
            const int want = i * kS1Waves + ((i & 1) ? kS1Waves - 1 - wave : wave);
            const unsigned long long m = __builtin_amdgcn_ballot_w64(lane < KT && rank == want);
            krow[i] = k0 + (int)__builtin_ctzll(m);
        }
    }
    int cur[RPW], end[RPW];
#pragma unroll
    for (int i = 0; i < RPW; ++i) {
        const int k = krow[i];
        cur[i] = (k < a.K) ? rowptr[k] : 0;
        end[i] = (k < a.K) ? rowptr[k + 1] : 0;
    }

    // accE: pixels (2l + 128j, 2l+1 + 128j) from even taps; accO: pixels
    // (2l-1 + 128j, 2l + 128j) from odd taps.
    float2 accE[RPW][IPW][PJ], accO[RPW][IPW][PJ];
#pragma unroll
    for (int i = 0; i < RPW; ++i)
#pragma unroll
        for (int im = 0; im < IPW; ++im)
#pragma unroll
            for (int p = 0; p < PJ; ++p) {
                accE[i][im][p] = make_float2(0.0f, 0.0f);
                accO[i][im][p] = make_float2(0.0f, 0.0f);
            }

    // LDS float index of tap offset o for chunk ch, pixel q: vb(ch) + o - c*plane_delta + q.
    auto vb_of = [&](int ch) { return (ch & 1) * a.buf_floats - ch * a.Cc * a.PLp; };
    auto bound_of = [&](int ch) { return min((ch + 1) * a.Cc, a.C) * plane; };
    const int q = 2 * lane;

    Window<kCompact> win[RPW];
    RawWindow next[RPW];
    stage_chunk_s1(a, xp, lds, 0, ig, y0, wave, lane);
#pragma unroll
    for (int i = 0; i < RPW; ++i) {
        next[i] = fetch_window(offset, vals, cur[i], end[i], lane);
        win[i] = decode_window<kCompact>(a, next[i], end[i], bound_of(0), vb_of(0), lane);
    }
    wait_async_copies();
    __syncthreads();

    for (int ch = 0; ch < a.nchunks; ++ch) {
        const bool more = ch + 1 < a.nchunks;
        if (more) {
            stage_chunk_s1(a, xp, lds + ((ch + 1) & 1) * a.buf_floats, ch + 1, ig, y0, wave, lane);
            // Fetch the next chunk's windows now, from where this chunk's
            // entries end, so their latency hides behind this chunk's work.
#pragma unroll
            for (int i = 0; i < RPW; ++i) next[i] = fetch_window(offset, vals, cur[i] + win[i].n, end[i], lane);
        }
        const int bound = bound_of(ch);
        const int vb = vb_of(ch);
        int total = 0, done = 0;
#pragma unroll
        for (int i = 0; i < RPW; ++i) total += win[i].n;
        set_progress_prio(0, total);
#pragma unroll
        for (int i = 0; i < RPW; ++i) {
            for (;;) {
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    if constexpr (kCompact) {
                        const int ne = win[i].ne[h], no = win[i].no[h];
                        run_range<NB>(accE[i], win[i].lo[h], win[i].w[h], 0, ne, lds, q, a.img_lds);
                        done += ne;
                        set_progress_prio(done, total);
                        run_range<NB>(accO[i], win[i].lo[h], win[i].w[h], ne, ne + no, lds, q, a.img_lds);
                        done += no;
                    } else {
                        run_mask<NB>(accE[i], win[i].lo[h], win[i].w[h], win[i].even[h], lds, q, a.img_lds);
                        done += __builtin_popcountll(win[i].even[h]);
                        set_progress_prio(done, total);
                        run_mask<NB>(accO[i], win[i].lo[h], win[i].w[h], win[i].odd[h], lds, q, a.img_lds);
                        done += __builtin_popcountll(win[i].odd[h]);
                    }
                    set_progress_prio(done, total);
                }
                const int n = win[i].n;
                cur[i] += n;
                if (n < 2 * kWave || cur[i] >= end[i]) break;
                // The row has more entries in this chunk than one window holds.
                win[i] = decode_window<kCompact>(a, fetch_window(offset, vals, cur[i], end[i], lane), end[i], bound,
                                                 vb, lane);
            }
        }
        if (more) {
#pragma unroll
            for (int i = 0; i < RPW; ++i) {
                // A row that overflowed a window in this chunk ends elsewhere.
                if (next[i].base != cur[i]) next[i] = fetch_window(offset, vals, cur[i], end[i], lane);
                win[i] = decode_window<kCompact>(a, next[i], end[i], bound_of(ch + 1), vb_of(ch + 1), lane);
            }
        }
        // Chunk ch+1 is in LDS and every wave is done with chunk ch's buffer.
        // After the last chunk only the pooled epilogue, which reuses the
        // buffers, needs the barrier.
        if (POOL || more) {
            wait_async_copies();
            __syncthreads();
        }
    }

    s1_epilogue<PI, IPW, RPW, POOL>(a, accE, accO, krow, ig, ty, y0, 0, wave, lane, lds, lds, bias, res, out);
}

// Generic-stride kernel: waves split the pixels of the tile and every wave
// walks all KT rows; each pixel keeps its own LDS base (y*stride*Wp +
// x*stride), so a nonzero costs one address add per pixel. Correct for any
// stride; the stride-1 kernel above is the fast path.
template <int P, int KT, bool POOL>
__global__ __launch_bounds__(kThreads) void spconv_generic_kernel(FwdArgs a, const float *__restrict__ xp,
                                                                  const int32_t *__restrict__ rowptr,
                                                                  const int32_t *__restrict__ offset,
                                                                  const float *__restrict__ vals,
                                                                  const int32_t *__restrict__ lw,
                                                                  const float *__restrict__ bias,
                                                                  const float *__restrict__ res,
                                                                  float *__restrict__ out) {
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

    int cur[KT], end[KT];
#pragma unroll
    for (int kk = 0; kk < KT; ++kk) {
        const int k = k0 + kk;
        cur[kk] = (k < a.K) ? rowptr[k] : 0;
        end[kk] = (k < a.K) ? rowptr[k + 1] : 0;
    }

    const int qw = wseg * kWave * P + lane;
    const int tile_px = a.TH * a.wv;
    int base[P];
#pragma unroll
    for (int j = 0; j < P; ++j) {
        const int q = qw + kWave * j;
        const int yl = q / a.Wo, x = q - yl * a.Wo;
        base[j] = (q < tile_px) ? yl * a.stride * a.Wp + x * a.stride : 0;
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
        stage_chunk(a, xp, lds, ch, ig, in_row0, seg_len, wave, lane);
        wait_async_copies();
        __syncthreads();
        if (!active) continue;

        const int vb = img * a.img_lds - c0 * a.PL;
        const int bound = (c0 + cn) * plane;
#pragma unroll
        for (int kk = 0; kk < KT; ++kk) {
            int j = cur[kk];
            const int e = end[kk];
            while (j < e) {
                const int o = offset[j];
                if (o >= bound) break;
                const float v = vals[j];
                const int c = (int)fast_div((uint32_t)o, a.magic, a.shift);
                const int ad = vb + o - c * a.plane_delta;
#pragma unroll
                for (int p = 0; p < P; ++p) acc[kk][p] = fmaf(v, lds[ad + base[p]], acc[kk][p]);
                ++j;
            }
            cur[kk] = j;
        }
    }

    // Tile row of each of this lane's pixels, or -1 when the pixel is not
    // stored; pixel q = yl*wv + x of the tile lands at q + yl*(pitch - wv) past
    // the tile's first element, in the output and the residual alike.
    int ylo[P];
#pragma unroll
    for (int j = 0; j < P; ++j) {
        const int q = qw + kWave * j;
        const int yl = q / a.wv, x = q - yl * a.wv;
        ylo[j] = (q < tile_px && x < a.Wo && y0 + yl < a.Ho) ? yl : -1;
    }
    const int rdelta = a.rpitch - a.wv;
    if constexpr (!POOL) {
        if (!active) return;
        const int odelta = a.opitch - a.wv;
#pragma unroll
        for (int kk = 0; kk < KT; ++kk) {
            const int k = k0 + kk;
            if (k >= a.K) break;
            const float bk = bias ? bias[k] : 0.0f;
            float *plane = out + ((size_t)n * a.K + k) * a.oplane;
            float *op = plane + (size_t)(y0 + a.out_pad) * a.opitch + a.out_pad;
            const float *rp =
                res ? res + ((size_t)n * a.K + k) * a.rplane + (size_t)(y0 + a.res_pad) * a.rpitch + a.res_pad
                    : nullptr;
#pragma unroll
            for (int j = 0; j < P; ++j) {
                if (ylo[j] < 0) continue;
                const int q = qw + kWave * j;
                float v = acc[kk][j] + bk;
                if (rp) v += rp[q + ylo[j] * rdelta];
                if (a.relu) v = v > 0.0f ? v : 0.0f;
                store_out(op + q + ylo[j] * odelta, v, a.out_pad == 0);
            }
            if (a.out_pad && wseg == 0)
                zero_border(plane, y0, min(y0 + a.TH, a.Ho), a.Ho, a.Wo, a.out_pad, a.opitch, ty == 0,
                            ty == a.ntiles_y - 1, lane, kWave);
        }
    } else {
        const int img_px = a.wpi * kWave * P;
        const int prow0 = y0 / 2;
        const int prows = a.TH / 2;
        const int per_img = prows * a.Wq;
        const int total = a.ipw * per_img;
#pragma unroll
        for (int kk = 0; kk < KT; ++kk) {
            const int k = k0 + kk;
            if (k >= a.K) break;
            const float bk = bias ? bias[k] : 0.0f;
            __syncthreads();  // previous readers of the staging area are done
            // The residual is added on the convolution's grid, before the
            // activation and the pool.
            const float *rp = (res && active) ? res + ((size_t)n * a.K + k) * a.rplane +
                                                    (size_t)(y0 + a.res_pad) * a.rpitch + a.res_pad
                                              : nullptr;
#pragma unroll
            for (int j = 0; j < P; ++j) {
                float v = acc[kk][j] + bk;
                if (rp && ylo[j] >= 0) v += rp[qw + kWave * j + ylo[j] * rdelta];
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
                    store_out(out + ((size_t)nn * a.K + k) * a.oplane + (size_t)(pi + a.out_pad) * a.opitch + jq +
                                  a.out_pad,
                              m, a.out_pad == 0);
                }
            }
            if (a.out_pad)
                for (int im = 0; im < a.ipw; ++im) {
                    const int nn = ig * a.ipw + im;
                    if (nn >= a.N) break;
                    zero_border(out + ((size_t)nn * a.K + k) * a.oplane, prow0, min(prow0 + prows, a.Hq), a.Hq, a.Wq,
                                a.out_pad, a.opitch, ty == 0, ty == a.ntiles_y - 1, (int)threadIdx.x, kThreads);
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
int ceil_div(int a, int b) { return (a + b - 1) / b; }

enum class Kind { kStride1, kGeneric };

struct Plan {
    Kind kind = Kind::kStride1;
    int PI = 0, IPW = 0, RPW = 0;  // stride-1 kernel
    int P = 0, KT = 0;             // generic kernel
    int TH = 0, ntiles_y = 0, ipw = 0, wpi = 0, Cc = 0, nchunks = 0, rows_in = 0, PL = 0, PLp = 0, img_lds = 0;
    int buf_floats = 0, wv = 0, rows_per_wg = 0, nktiles = 0, total_wgs = 0;
    int span = 0;  // stride-1 kernel: virtual pixels per row-spanning tile (0: tiles of TH whole rows)
    size_t lds_bytes = 0;
};

using FwdKernel = void (*)(FwdArgs, const float *, const int32_t *, const int32_t *, const float *, const int32_t *,
                          const float *, const float *, float *);

// Stride-1 kernel instances: (PI, IPW, RPW, pools), pools bit 0 = built
// without the pool epilogue, bit 1 = with it. Four waves per SIMD leave 128
// VGPRs per lane: two accumulator sets of RPW * IPW * PI floats (even and odd
// taps) plus the pipeline buffers, so IPW * PI <= 24 and RPW * IPW * PI <= 32
// (at most 16 pixels with two channels, 8 with four). The list holds the
// instances the planner can pick; the GPU tests run each one against the
// oracle.
struct S1Variant {
    int pi, ipw, rpw, pools;
};

// Tilings also built to run several work items per workgroup with a lowered
// stream: those of large planes (one image per tile, many pixels per lane),
// whose grids run many rounds of workgroups. Other tilings keep one work item
// per workgroup, which holds fewer registers.
constexpr bool tiled_variant(const S1Variant &v) { return v.ipw == 1 && v.pi >= 12; }
constexpr S1Variant kS1Variants[] = {
    // one image per tile
    {24, 1, 1, 3}, {22, 1, 1, 3}, {20, 1, 1, 3}, {18, 1, 1, 3}, {16, 1, 1, 3}, {14, 1, 1, 3}, {12, 1, 1, 3},
    {10, 1, 1, 3}, {8, 1, 1, 3},  {6, 1, 1, 3},  {4, 1, 1, 3},
    {16, 1, 2, 3}, {14, 1, 2, 3}, {12, 1, 2, 3}, {10, 1, 2, 3}, {8, 1, 2, 3}, {6, 1, 2, 3}, {4, 1, 2, 3},
    {8, 1, 4, 3},  {6, 1, 4, 3},  {4, 1, 4, 3},
    // two images per tile
    {8, 2, 1, 3}, {6, 2, 1, 3}, {4, 2, 1, 3}, {2, 2, 1, 3},
    {8, 2, 2, 3}, {6, 2, 2, 3}, {4, 2, 2, 3}, {2, 2, 2, 3},
    {4, 2, 4, 3}, {2, 2, 4, 3},
    // four images per tile
    {6, 4, 1, 3}, {4, 4, 1, 3}, {2, 4, 1, 3},
    {4, 4, 2, 3}, {2, 4, 2, 3},
    {2, 4, 4, 3},
};
constexpr int kNumS1Variants = (int)(sizeof(kS1Variants) / sizeof(kS1Variants[0]));

template <int PI, int IPW, int RPW, bool POOL, bool TILED>
FwdKernel pick_s1_mode(int mode) {
    if (mode == kModePlain) return spconv_s1_kernel<PI, IPW, RPW, POOL, kModePlain>;
    if (mode == kModeLowered) return spconv_s1_kernel<PI, IPW, RPW, POOL, kModeLowered>;
    if constexpr (TILED) return spconv_s1_kernel<PI, IPW, RPW, POOL, kModeTiled>;
    return nullptr;
}

template <int I>
FwdKernel pick_s1_from(int PI, int IPW, int RPW, bool pool, int mode) {
    if constexpr (I == kNumS1Variants) {
        return nullptr;
    } else {
        constexpr S1Variant v = kS1Variants[I];
        static_assert(v.ipw * v.pi <= 24 && v.rpw * v.ipw * v.pi <= 32 && v.pi % 2 == 0,
                      "tiling exceeds the register budget");
        constexpr bool tiled = tiled_variant(v);
        if (v.pi == PI && v.ipw == IPW && v.rpw == RPW) {
            if (pool) {
                if constexpr ((v.pools & 2) != 0) return pick_s1_mode<v.pi, v.ipw, v.rpw, true, tiled>(mode);
                return nullptr;
            }
            if constexpr ((v.pools & 1) != 0) return pick_s1_mode<v.pi, v.ipw, v.rpw, false, tiled>(mode);
            return nullptr;
        }
        return pick_s1_from<I + 1>(PI, IPW, RPW, pool, mode);
    }
}

// Pixels per lane per image (PI) the planner tries with one image per tile
// and with several.
constexpr int kPiSingle[] = {24, 22, 20, 18, 16, 14, 12, 10, 8, 6, 4};
constexpr int kPiMulti[] = {8, 6, 4, 2};

FwdKernel pick_s1(int PI, int IPW, int RPW, bool pool, int mode = kModePlain) {
    return pick_s1_from<0>(PI, IPW, RPW, pool, mode);
}

// Picks the stride-1 tiling with the smallest modelled run time. The model
// counts LDS cycles: every nonzero costs a wave IPW*PI LDS reads (2 cycles
// each, 64 lanes x 4 bytes at 128 bytes per cycle) plus about one read's
// worth of issue overhead (weight and offset broadcast, address add, loop
// control), and the 16 waves of a workgroup share one LDS. Each chunk adds a
// fixed cost (barrier, pipeline refill) and the LDS writes of its copy, halo
// rows included; the pooled epilogue adds a staging round (LDS writes and
// the 2x2 reductions) per channel of a wave, 4000 cycles since it stages pair
// maxima (at 8000 the model picked (22,1,1) for the 224x224 pooled layer,
// 0.5-2.5% slower than (16,1,2)). Workgroups run one per CU, in rounds of 256.
// Uneven nonzero counts between the waves of a workgroup cost little while
// the slowest wave has at most ~1.3x the mean (the others' LDS bandwidth
// passes to it as they finish). Beyond that the workgroup waits for it: with
// one channel per wave that happens for skewed filters (max_row_nnz well
// above the mean); with two or more, heavy and light channels are paired and
// the pair sums stay close to the mean. One channel per wave also pays ~3%
// more for the chunk-to-chunk variation of a single row's counts.
// The constants were fitted to measured run times of 5-7 tilings each of
// ResNet, VGG (with and without pooling), conv+pool and narrow 256-channel
// layers, so that the model orders each layer's tilings as measured.
// vp: pitch of the virtual tile and of the staged LDS rows; shift: LDS column
// of padded column 0 (both Wp and 0 for a padded input).
// span_ok: the chosen tiling's tiles of one image may also be row-spanning:
// tile t covers the virtual pixels [t*span, (t+1)*span) of the image, span =
// 64*PI - 2, whatever rows they fall in, so no lane computes pixels of rows a
// whole-row tile would have to leave out (at 224x224 with PI = 16, 4 rows of
// 228 fill 912 of a tile's 1024 pixels). Unpooled layers with a lowered stream
// only (224x224 layer: 56 -> 50 tiles per image, 636 -> 615 us).
bool plan_stride1(int N, int C, int K, int Hp, int Wp, int vp, int shift, int Ho, int Wo, int R, int S, bool pool,
                  long long nnz, long long max_row_nnz, bool span_ok, Plan *out) {
    const int img_pix = Ho * vp;
    const double row_nnz = std::max(1.0, (double)nnz / K);
    const double skew = max_row_nnz > 0 ? (double)max_row_nnz / row_nnz : 1.0;
    Plan best;
    double best_time = -1.0;
    auto consider = [&](int PI, int IPW, int RPW, bool spanning) {
        if (!pick_s1(PI, IPW, RPW, pool)) return;
        // Virtual pixels per image tile. The last one (64*PI - 1) has no odd-tap
        // partner, so a tile holds at most cap - 1 pixels.
        const int cap = kWave * PI;
        int TH, nt, span = 0;
        if (spanning) {
            // Row-spanning tiles of span (even) pixels up to the last stored
            // one; TH = the most output rows a tile touches.
            // The lanes' pixel pairs stay aligned only if every tile starts at
            // an even column: span and the pitch even.
            if (IPW != 1 || img_pix <= cap - 1 || (vp & 1)) return;
            span = cap - 2;
            const long long last = (long long)(Ho - 1) * vp + Wo;
            nt = (int)((last + span - 1) / span);
            TH = 0;
            for (int t = 0; t < nt; ++t) {
                const long long s0 = (long long)t * span;
                const int r0 = (int)(s0 / vp);
                const int r1 = (int)std::min<long long>((s0 + span - 1) / vp, Ho - 1);
                TH = std::max(TH, r1 - r0 + 1);
            }
        } else if (img_pix <= cap - 1) {
            TH = Ho;
            nt = 1;
        } else {
            if (IPW != 1) return;
            int th_max = (cap - 1) / vp;
            if (pool) th_max &= ~1;
            if (th_max < 1) return;
            nt = ceil_div(Ho, th_max);
            TH = ceil_div(Ho, nt);
            if (pool && (TH & 1)) ++TH;
            nt = ceil_div(Ho, TH);
        }
        int rows_in = TH + R - 1;
        int PL = rows_in * vp + shift;
        if (spanning) {
            // A row-spanning tile stages only the window of virtual pixels it
            // reads: from its first pixel's column rounded down to a multiple
            // of 4 (col0, at most 3 before it) through its last lane's last
            // tap, so the window holds cap + (R-1)*vp + S pixels and a little
            // more, however the tile sits in its rows. rows_in = the most rows
            // such a window touches.
            PL = shift + 3 + cap + (R - 1) * vp + S;
            rows_in = ceil_div(vp + PL, vp);
        }
        // Channel slots 16-byte aligned; a slot's last copy masks the lanes
        // past it (rounding slots up to whole 256-float copies would cost
        // LDS and, at 64 channels of 56x56, a fourth chunk).
        const int PLp = ceil_div(PL, 4) * 4;
        // Lanes past a whole-row tile read up to cap - TH*vp + S - 2 floats
        // beyond the last image block (values that only dropped pixels use).
        // Past the first buffer they land in the second; past the second, in
        // one slack area after it. A row-spanning tile's window holds every
        // read of its lanes.
        const int slack = spanning ? S : cap - TH * vp + S;
        int cc_max = ((kS1LdsFloats - slack - kLwSinkFloats) / 2) / (IPW * PLp);
        if (cc_max < 1) return;
        cc_max = std::min(cc_max, C);
        const int nchunks = ceil_div(C, cc_max);
        const int Cc = ceil_div(C, nchunks);
        // The DMA offsets of one chunk are 32-bit byte offsets.
        if (((long long)(Cc - 1) * Hp * Wp + PLp) * 4 >= (1LL << 32)) return;
        const int KT = kS1Waves * RPW;
        const long long wgs = (long long)ceil_div(N, IPW) * nt * ceil_div(K, KT);
        if (wgs > 0x7fffffffLL) return;
        const double pair_skew = 1.0 + (skew - 1.0) / (2.0 * RPW - 1.0);
        const double imb = std::max(1.0, (RPW == 1 ? skew : pair_skew) / 1.3) * (RPW == 1 ? 1.03 : 1.0);
        // Buffers rounded up to 64 floats may not fit once slack is added.
        const int buf_floats = ceil_div(IPW * Cc * PLp, 64) * 64;
        size_t floats = 2 * (size_t)buf_floats + slack;
        if (pool) floats = std::max(floats, (size_t)kS1Waves * IPW * kWave * PI);
        floats += kLwSinkFloats;  // the stream prefetch's sink, last
        if (floats > (size_t)kS1LdsFloats) return;
        const double compute = kS1Waves * RPW * row_nnz * 2.0 * (IPW * PI + 1.0) * imb;
        const double wg_cycles =
            compute + nchunks * (3000.0 + IPW * (double)Cc * PLp / 32.0) + (pool ? 4000.0 * RPW : 0.0);
        const double time = (double)ceil_div((int)std::min<long long>(wgs, 1 << 30), 256) * wg_cycles;
        if (best_time < 0 || time < best_time * 0.999) {
            best_time = time;
            best.kind = Kind::kStride1;
            best.PI = PI;
            best.IPW = IPW;
            best.RPW = RPW;
            best.TH = TH;
            best.ntiles_y = nt;
            best.ipw = IPW;
            best.Cc = Cc;
            best.nchunks = nchunks;
            best.rows_in = rows_in;
            best.PL = PL;
            best.PLp = PLp;
            best.img_lds = Cc * PLp;
            best.buf_floats = buf_floats;
            best.wv = vp;
            best.rows_per_wg = KT;
            best.nktiles = ceil_div(K, KT);
            best.total_wgs = (int)wgs;
            best.span = span;
            best.lds_bytes = floats * sizeof(float);
        }
    };
    for (int RPW : {1, 2, 4}) {
        for (int PI : kPiSingle) consider(PI, 1, RPW, false);
        for (int IPW : {2, 4})
            if (IPW <= N)
                for (int PI : kPiMulti) consider(PI, IPW, RPW, false);
    }
    if (best_time < 0) return false;
    // Row-spanning tiles are a choice of geometry for the chosen tiling, made
    // when they are modelled faster, so that a layer runs the same kernel
    // instance with or without a lowered stream.
    if (span_ok && !pool && best.IPW == 1) consider(best.PI, 1, best.RPW, true);
    *out = best;
    return true;
}

bool plan_generic(int N, int C, int K, int Hp, int Wp, int Ho, int Wo, int stride, int R, bool pool, Plan *out) {
    constexpr int P = 4, KT = 4;
    const int wv = Wo;
    const int img_pix = Ho * wv;
    Plan best;
    double best_eff = -1.0;
    for (int wpi : {4, 2, 1}) {
        const int ipw = kWaves / wpi;
        const int cap = wpi * kWave * P;
        int TH, nt;
        if (img_pix <= cap) {
            TH = Ho;
            nt = 1;
        } else {
            if (ipw != 1) continue;
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
        int cc_max = kLdsBudgetFloats / (ipw * PL);
        if (cc_max < 1) continue;
        cc_max = std::min(cc_max, C);
        const int nchunks = ceil_div(C, cc_max);
        const int Cc = ceil_div(C, nchunks);
        const double eff = (double)Ho * Wo / ((double)nt * cap);
        if (eff > best_eff + 1e-9) {
            best_eff = eff;
            best.kind = Kind::kGeneric;
            best.P = P;
            best.KT = KT;
            best.TH = TH;
            best.ntiles_y = nt;
            best.ipw = ipw;
            best.wpi = wpi;
            best.Cc = Cc;
            best.nchunks = nchunks;
            best.rows_in = rows_in;
            best.PL = PL;
            best.img_lds = Cc * PL;
            best.buf_floats = ipw * Cc * PL;
            best.wv = wv;
            size_t floats = (size_t)best.buf_floats;
            if (pool) floats = std::max(floats, (size_t)ipw * cap);
            best.lds_bytes = floats * sizeof(float);
        }
    }
    if (best_eff < 0) return false;
    const int groups = ceil_div(N, best.ipw) * best.ntiles_y;
    best.rows_per_wg = KT;
    best.nktiles = ceil_div(K, KT);
    const long long wgs = (long long)groups * best.nktiles;
    if (wgs > 0x7fffffffLL) return false;
    best.total_wgs = (int)wgs;
    *out = best;
    return true;
}

FwdKernel pick_kernel(const Plan &pl, bool pool, int mode = kModePlain) {
    if (pl.kind == Kind::kGeneric)
        return mode != kModePlain ? nullptr
                                  : (pool ? spconv_generic_kernel<4, 4, true> : spconv_generic_kernel<4, 4, false>);
    return pick_s1(pl.PI, pl.IPW, pl.RPW, pool, mode);
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
    if (flags & ~(SPCONV_RELU | SPCONV_MAXPOOL2X2 | SPCONV_UNPADDED_INPUT)) return SPCONV_EINVAL;
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
    if (plane >= kPadMaxPlane || planes * plane >= (1LL << 40)) return SPCONV_EINVAL;
    PadArgs a;
    a.in = in;
    a.out = out_padded;
    a.total = planes * plane;
    a.H = H;
    a.W = W;
    a.pad = pad;
    a.Hp = (int)Hp;
    a.Wp = (int)Wp;
    a.plane = (int)plane;
    if (!div_magic((uint32_t)Wp, &a.wp_magic, &a.wp_shift) ||
        !div_magic((uint32_t)plane, &a.plane_magic, &a.plane_shift))
        return SPCONV_EINVAL;
    const long long per_block = kPadSpan;
    const long long blocks = (a.total + per_block - 1) / per_block;
    if (blocks > 0x7fffffffLL) return SPCONV_EINVAL;
    const bool vec = (reinterpret_cast<uintptr_t>(out_padded) & 15) == 0;
    hipLaunchKernelGGL(vec ? pad_nchw_kernel<true> : pad_nchw_kernel<false>, dim3((unsigned)blocks), dim3(kThreads),
                       0, stream, a);
    return hipGetLastError() == hipSuccess ? SPCONV_OK : SPCONV_EHIP;
}

extern "C" int spconv_resize_pad_input(const float *in, int N, int C, int Hin, int Win, int H, int W, int pad,
                                       float *out_padded, hipStream_t stream) {
    if (!in || !out_padded || N < 1 || C < 1 || Hin < 1 || Win < 1 || H < 1 || W < 1 || pad < 0)
        return SPCONV_EINVAL;
    if (Hin > kResizeMaxSide || Win > kResizeMaxSide || H > kResizeMaxSide || W > kResizeMaxSide)
        return SPCONV_EINVAL;
    const long long Hp = (long long)H + 2LL * pad, Wp = (long long)W + 2LL * pad;
    const long long planes = (long long)N * C;
    if (Hp * Wp >= (1LL << 31) || planes * Hp * Wp >= (1LL << 40) || planes * Hin * Win >= (1LL << 40))
        return SPCONV_EINVAL;
    const long long ps = Hp * Wp;
    const long long in_ps = (long long)Hin * Win;
    // Plane kernel when a source plane and its padded output are small (tap
    // tables of at most 12 KiB plus at most 48 KiB of staged planes).
    if (in_ps <= kResizePlaneMaxIn && ps <= kResizePlaneMaxOut && Hp + Wp <= 1024) {
        ResizePlaneArgs g;
        g.Hin = Hin;
        g.Win = Win;
        g.H = H;
        g.W = W;
        g.pad = pad;
        g.Hp = (int)Hp;
        g.Wp = (int)Wp;
        g.ps = (int)ps;
        g.in_ps = (int)in_ps;
        g.planes = planes;
        const long long by_lds = std::max(1LL, (long long)kResizePlaneLds / (in_ps * (long long)sizeof(float)));
        const long long by_grid = std::max(1LL, planes / kResizePlaneWgs);
        g.ppw = (int)std::min(by_lds, by_grid);
        g.vec = (in_ps % 4 == 0 && (reinterpret_cast<uintptr_t>(in) & 15) == 0) ? 1 : 0;
        if (!div_magic((uint32_t)ps, &g.ps_magic, &g.ps_shift) || !div_magic((uint32_t)Wp, &g.wp_magic, &g.wp_shift))
            return SPCONV_EINVAL;
        const long long blocks = (planes + g.ppw - 1) / g.ppw;
        if (blocks > 0x7fffffffLL) return SPCONV_EINVAL;
        const size_t lds = (size_t)((3 * (Hp + Wp) + 3) & ~3LL) * sizeof(int) + (size_t)g.ppw * in_ps * sizeof(float);
        hipLaunchKernelGGL(resize_pad_plane_kernel, dim3((unsigned)blocks), dim3(kThreads), lds, stream, g, in,
                           out_padded);
        return hipGetLastError() == hipSuccess ? SPCONV_OK : SPCONV_EHIP;
    }
    // Flat kernel when both tap tables fit in LDS and the source planes one
    // workgroup can touch are addressable with 32-bit offsets (in elements).
    const long long span_planes = (long long)kThreads * kResizeFlatElems / ps + 2;
    if (Hp + Wp <= kResizeFlatMaxTab && span_planes * Hin * Win < (1LL << 31)) {
        ResizeFlatArgs f;
        f.Hin = Hin;
        f.Win = Win;
        f.H = H;
        f.W = W;
        f.pad = pad;
        f.Hp = (int)Hp;
        f.Wp = (int)Wp;
        f.ps = (int)ps;
        f.total = planes * ps;
        if (!div_magic((uint32_t)ps, &f.ps_magic, &f.ps_shift) || !div_magic((uint32_t)Wp, &f.wp_magic, &f.wp_shift))
            return SPCONV_EINVAL;
        const long long per_block = (long long)kThreads * kResizeFlatElems;
        const long long blocks = (f.total + per_block - 1) / per_block;
        if (blocks > 0x7fffffffLL) return SPCONV_EINVAL;
        const size_t lds = (size_t)(Hp + Wp) * 3 * sizeof(int);
        hipLaunchKernelGGL(resize_pad_flat_kernel, dim3((unsigned)blocks), dim3(kThreads), lds, stream, f, in,
                           out_padded);
        return hipGetLastError() == hipSuccess ? SPCONV_OK : SPCONV_EHIP;
    }
    ResizeArgs a;
    a.Hin = Hin;
    a.Win = Win;
    a.H = H;
    a.W = W;
    a.pad = pad;
    a.Hp = (int)Hp;
    a.Wp = (int)Wp;
    const long long max_bands = (Hp + kWaves - 1) / kWaves;
    const long long want = (kResizeTargetWgs + planes - 1) / planes;
    const long long bands0 = std::max(1LL, std::min(want, max_bands));
    a.band_rows = (int)((Hp + bands0 - 1) / bands0);
    a.bands = (int)((Hp + a.band_rows - 1) / a.band_rows);
    const long long blocks = planes * a.bands;
    if (blocks > 0x7fffffffLL) return SPCONV_EINVAL;
    hipLaunchKernelGGL(resize_pad_rows_kernel, dim3((unsigned)blocks), dim3(kThreads), 0, stream, a, in,
                       out_padded);
    return hipGetLastError() == hipSuccess ? SPCONV_OK : SPCONV_EHIP;
}

namespace {

// Host-side checks of a forward call (everything but the buffer pointers) and
// its launch plan. Returns SPCONV_OK or SPCONV_EINVAL.
int prepare_forward(int N, int C, int H, int W, const spconv_csr *csr, int K, int R, int S, int stride, int pad,
                    uint32_t flags, long long max_row_nnz, bool lowered, Plan *plp, FwdArgs *ap) {
    if (!csr) return SPCONV_EINVAL;
    if (N < 1 || C < 1 || H < 1 || W < 1 || K < 1 || R < 1 || S < 1 || stride < 1 || pad < 0) return SPCONV_EINVAL;
    if (flags & ~(SPCONV_RELU | SPCONV_MAXPOOL2X2 | SPCONV_UNPADDED_INPUT)) return SPCONV_EINVAL;
    if (csr->K != K || csr->C != C || csr->R != R || csr->S != S) return SPCONV_EINVAL;
    const long long Hp = (long long)H + 2LL * pad, Wp = (long long)W + 2LL * pad;
    if (csr->Hp != Hp || csr->Wp != Wp) return SPCONV_EINVAL;
    if (csr->nnz < 0 || csr->nnz >= (1LL << 31)) return SPCONV_EINVAL;
    if (max_row_nnz < 0 || max_row_nnz > csr->nnz) return SPCONV_EINVAL;
    if (!csr->rowptr || (csr->nnz > 0 && (!csr->offset || !csr->vals))) return SPCONV_EINVAL;
    if ((long long)C * Hp * Wp >= (1LL << 31)) return SPCONV_EINVAL;
    const bool pool = (flags & SPCONV_MAXPOOL2X2) != 0;
    int Ho, Wo;
    if (!out_extent(H, R, stride, pad, &Ho) || !out_extent(W, S, stride, pad, &Wo)) return SPCONV_EINVAL;
    if (Ho < 1 || Wo < 1) return SPCONV_EINVAL;
    if (pool && (Ho < 2 || Wo < 2)) return SPCONV_EINVAL;

    // An unpadded input whose rows are a whole number of 16-byte groups is
    // staged with 16-byte row copies: the LDS rows then take a pitch vp that
    // is a multiple of 4 floats, and padded column 0 sits at LDS column shift,
    // so that every row's first image column is 16-byte aligned.
    const bool unpadded = (flags & SPCONV_UNPADDED_INPUT) != 0;
    bool row16 = unpadded && stride == 1 && W % 4 == 0;
    Plan pl;
    bool ok = false;
    if (stride != 1) {
        ok = plan_generic(N, C, K, (int)Hp, (int)Wp, Ho, Wo, stride, R, pool, &pl);
    } else {
        if (row16)
            ok = plan_stride1(N, C, K, (int)Hp, (int)Wp, ((int)Wp + 3) / 4 * 4, (4 - pad % 4) % 4, Ho, Wo, R, S,
                              pool, csr->nnz, max_row_nnz, lowered, &pl);
        if (!ok) {
            row16 = false;
            ok = plan_stride1(N, C, K, (int)Hp, (int)Wp, (int)Wp, 0, Ho, Wo, R, S, pool, csr->nnz, max_row_nnz,
                              lowered, &pl);
        }
    }
    if (!ok) return SPCONV_EINVAL;
    if (unpadded && pl.kind != Kind::kStride1) return SPCONV_EINVAL;
    FwdArgs a;
    a.unpadded = unpadded ? 1 : 0;
    a.vp = pl.kind == Kind::kStride1 ? pl.wv : (int)Wp;
    a.lds_shift = row16 ? (4 - pad % 4) % 4 : 0;
    a.dma16 = row16 ? 1 : 0;
    a.pair_store = 0;
    a.lw_headers = a.lw_entries = 0;
    a.pf_bytes = 0;
    a.pool_pairs = a.pool_in_buf = 0;
    a.span = pl.kind == Kind::kStride1 ? pl.span : 0;
    if (!div_magic((uint32_t)Wp, &a.wp_magic, &a.wp_shift)) return SPCONV_EINVAL;
    if (!div_magic((uint32_t)a.vp, &a.vp_magic, &a.vp_shift)) return SPCONV_EINVAL;
    a.H = H;
    a.W = W;
    a.pad = pad;
    a.N = N;
    a.C = C;
    a.K = K;
    a.Hp = (int)Hp;
    a.Wp = (int)Wp;
    a.Ho = Ho;
    a.Wo = Wo;
    a.Hq = pool ? Ho / 2 : Ho;
    a.Wq = pool ? Wo / 2 : Wo;
    a.pimg_magic = a.wq_magic = 1;
    a.pimg_shift = a.wq_shift = 0;
    if (pl.kind == Kind::kStride1 && pool &&
        (!div_magic((uint32_t)((pl.TH / 2) * a.Wq), &a.pimg_magic, &a.pimg_shift) ||
         !div_magic((uint32_t)a.Wq, &a.wq_magic, &a.wq_shift)))
        return SPCONV_EINVAL;
    a.stride = stride;
    a.nnz = (int)csr->nnz;
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
    a.buf_floats = pl.buf_floats;
    a.lds_floats = (int)(pl.lds_bytes / sizeof(float));
    if (pl.kind == Kind::kStride1 && pool) {
        // Pair-maxima staging needs an even pitch; it fits the buffer of the
        // last chunk when 16 waves x IPW images x 64 lanes x PI/2 maxima do.
        a.pool_pairs = (a.vp % 2 == 0) ? 1 : 0;
        a.pool_in_buf = (a.pool_pairs &&
                         (long long)kS1Waves * pl.IPW * kWave * (pl.PI / 2) <= (long long)pl.buf_floats)
                            ? 1
                            : 0;
    }
    a.PLp = pl.PLp;
    a.plp_magic = 1;
    a.plp_shift = 0;
    if (pl.kind == Kind::kStride1 && !div_magic((uint32_t)pl.PLp, &a.plp_magic, &a.plp_shift)) return SPCONV_EINVAL;
    a.stage_units = UnitStep{1, kS1Waves, 0, 65536u};
    if (pl.kind == Kind::kStride1 && !unit_step(ceil_div(pl.PLp, kStageBlock), kS1Waves, &a.stage_units))
        return SPCONV_EINVAL;
    a.total_floats = (size_t)N * C * Hp * Wp;
    a.wv = pl.wv;
    a.total_wgs = pl.total_wgs;
    if (!div_magic((uint32_t)(Hp * Wp), &a.magic, &a.shift)) return SPCONV_EINVAL;
    // Both kernels address a staged channel at its LDS pitch: PLp (stride 1) or PL.
    a.plane_delta = (int)(Hp * Wp) - (pl.kind == Kind::kStride1 ? pl.PLp : pl.PL);
    if (!pick_kernel(pl, pool)) return SPCONV_EINVAL;
    // Epilogue defaults: dense output planes, no residual.
    a.out_pad = 0;
    a.opitch = a.Wq;
    a.oplane = (size_t)a.Hq * a.Wq;
    a.res_pad = 0;
    a.rpitch = a.Wo;
    a.rplane = (size_t)a.Ho * a.Wo;
    *plp = pl;
    *ap = a;
    return SPCONV_OK;
}

// Border and residual options of spconv_forward_ex, checked and folded into
// the args.
// Kernel mode of a launch: the plain CSR walk, or with a lowered stream the
// one-item-per-workgroup form, or, where the tiling is built for it and there
// are more work items than one round of workgroups (one per CU of MI355X,
// each holding the CU's whole LDS), the form that runs several items per
// workgroup and overlaps tile edges.
constexpr int kResidentWgs = 256;
int launch_mode(const Plan &pl, bool lowered, bool pool) {
    if (!lowered || pl.kind != Kind::kStride1) return kModePlain;
    if (pl.total_wgs > kResidentWgs && pick_s1(pl.PI, pl.IPW, pl.RPW, pool, kModeTiled)) return kModeTiled;
    return kModeLowered;
}
int launch_grid(const Plan &pl, int mode) {
    return mode == kModeTiled ? std::min(pl.total_wgs, kResidentWgs) : pl.total_wgs;
}

// Lowered stream of a stride-1 plan: headers (4 words each) per (channel
// tile, wave, row slot, chunk), then nnz entries and kLwPad pad entries (2
// words each).
int lowered_headers(const Plan &pl) { return pl.nktiles * kS1Waves * pl.RPW * pl.nchunks; }
long long lowered_words(const Plan &pl, long long nnz) {
    return 4LL * lowered_headers(pl) + 2LL * (nnz + kLwPad);
}

int apply_epilogue(const spconv_options *opt, FwdArgs *a) {
    if (!opt) return SPCONV_OK;
    if (opt->out_pad < 0 || (opt->residual && opt->residual_pad < 0)) return SPCONV_EINVAL;
    const long long op = opt->out_pad, rp = opt->residual ? opt->residual_pad : 0;
    const long long oh = a->Hq + 2 * op, ow = a->Wq + 2 * op;
    const long long rh = a->Ho + 2 * rp, rw = a->Wo + 2 * rp;
    if (oh * ow >= (1LL << 31) || rh * rw >= (1LL << 31)) return SPCONV_EINVAL;
    a->out_pad = (int)op;
    a->opitch = (int)ow;
    a->oplane = (size_t)(oh * ow);
    a->res_pad = (int)rp;
    a->rpitch = (int)rw;
    a->rplane = (size_t)(rh * rw);
    return SPCONV_OK;
}

}  // namespace

extern "C" int spconv_forward_ex(const float *in_padded, int N, int C, int H, int W, const spconv_csr *csr, int K,
                                 int R, int S, int stride, int pad, const float *bias, uint32_t flags,
                                 const spconv_options *opt, float *out, hipStream_t stream) {
    if (!in_padded || !out) return SPCONV_EINVAL;
    Plan pl;
    FwdArgs a;
    int rc = prepare_forward(N, C, H, W, csr, K, R, S, stride, pad, flags, opt ? opt->max_row_nnz : 0,
                             opt && opt->lowered, &pl, &a);
    if (rc != SPCONV_OK) return rc;
    rc = apply_epilogue(opt, &a);
    if (rc != SPCONV_OK) return rc;
    const float *residual = opt ? opt->residual : nullptr;
    // 16-byte row copies need a 16-byte aligned tensor; otherwise the same
    // layout is filled 4 bytes per lane.
    if (a.dma16 && (reinterpret_cast<uintptr_t>(in_padded) & 15) != 0) a.dma16 = 0;
    // Pixel pairs (2l, 2l+1) of the virtual tile share a row when its pitch vp
    // is even, and are both inside or both outside the output when Wo is even
    // too; two-dword accesses need only 4-byte aligned tensors.
    a.pair_store = pl.kind == Kind::kStride1 && (flags & SPCONV_MAXPOOL2X2) == 0 && a.vp % 2 == 0 &&
                   a.Wo % 2 == 0 && (reinterpret_cast<uintptr_t>(out) & 3) == 0 &&
                   (!residual || (reinterpret_cast<uintptr_t>(residual) & 3) == 0);
    const int32_t *lowered = opt ? opt->lowered : nullptr;
    if (lowered) {
        if (pl.kind != Kind::kStride1 || (reinterpret_cast<uintptr_t>(lowered) & 15) != 0) return SPCONV_EINVAL;
        if (opt->lowered_words != lowered_words(pl, csr->nnz)) return SPCONV_EINVAL;
        a.lw_headers = lowered_headers(pl);
        a.lw_entries = (int)csr->nnz;
        // A wave's lists hold RPW rows: 1.5x their mean entries (row skew),
        // in whole 128-byte lines, at most 32 KiB.
        const long long pf = ((long long)pl.RPW * (csr->nnz * 3 / (2LL * K) + 1) * 8 + 127) / 128 * 128;
        a.pf_bytes = (int)std::min<long long>(4LL * 8192, pf);
    }
    const int mode = launch_mode(pl, lowered != nullptr, (flags & SPCONV_MAXPOOL2X2) != 0);
    FwdKernel kern = pick_kernel(pl, (flags & SPCONV_MAXPOOL2X2) != 0, mode);
    if (!kern) return SPCONV_EINVAL;
    const unsigned threads = pl.kind == Kind::kStride1 ? kS1Threads : kThreads;
    // Each kernel instance's dynamic-LDS limit is raised once, to the most any
    // plan of its family uses, so that launches of different shapes from
    // several host threads never lower it under one another.
    if (!raise_lds_limit((const void *)kern, pl.kind == Kind::kStride1 ? kS1LdsFloats * 4 : kGenericLdsBytes))
        return SPCONV_EHIP;
    hipLaunchKernelGGL(kern, dim3((unsigned)launch_grid(pl, mode)), dim3(threads), pl.lds_bytes, stream, a,
                       in_padded, csr->rowptr, csr->offset, csr->vals, lowered, bias, residual, out);
    return hipGetLastError() == hipSuccess ? SPCONV_OK : SPCONV_EHIP;
}

extern "C" int spconv_forward(const float *in_padded, int N, int C, int H, int W, const spconv_csr *csr, int K, int R,
                              int S, int stride, int pad, const float *bias, uint32_t flags, float *out,
                              hipStream_t stream) {
    return spconv_forward_ex(in_padded, N, C, H, W, csr, K, R, S, stride, pad, bias, flags, nullptr, out, stream);
}

extern "C" int spconv_plan(int N, int C, int H, int W, const spconv_csr *csr, int K, int R, int S, int stride,
                           int pad, uint32_t flags, const spconv_options *opt, spconv_plan_info *info) {
    if (!info) return SPCONV_EINVAL;
    Plan pl;
    FwdArgs a;
    int rc = prepare_forward(N, C, H, W, csr, K, R, S, stride, pad, flags, opt ? opt->max_row_nnz : 0,
                             opt && opt->lowered, &pl, &a);
    if (rc != SPCONV_OK) return rc;
    rc = apply_epilogue(opt, &a);
    if (rc != SPCONV_OK) return rc;
    const bool s1 = pl.kind == Kind::kStride1;
    info->kernel = s1 ? SPCONV_KERNEL_STRIDE1 : SPCONV_KERNEL_GENERIC;
    info->pixels_per_lane = s1 ? pl.PI : pl.P;
    info->images_per_group = pl.ipw;
    info->channels_per_wave = s1 ? pl.RPW : pl.KT;
    info->tile_rows = pl.TH;
    info->tiles_per_image = pl.ntiles_y;
    info->channels_per_chunk = pl.Cc;
    info->chunks = pl.nchunks;
    info->workgroups = pl.total_wgs;
    info->threads_per_workgroup = (int32_t)(s1 ? kS1Threads : kThreads);
    info->lds_bytes = (int64_t)pl.lds_bytes;
    info->lds_channel_floats = s1 ? pl.PLp : 0;
    info->lds_row_pitch = s1 ? a.vp : 0;
    info->lds_col_shift = s1 ? a.lds_shift : 0;
    info->launch_workgroups =
        launch_grid(pl, launch_mode(pl, opt && opt->lowered, (flags & SPCONV_MAXPOOL2X2) != 0));
    info->tile_pixels = s1 ? pl.span : 0;
    return SPCONV_OK;
}

extern "C" int spconv_kernel_variants(int32_t kernel, int32_t *variants, int32_t capacity, int32_t *count) {
    if (!count || capacity < 0 || (capacity > 0 && !variants)) return SPCONV_EINVAL;
    if (kernel == SPCONV_KERNEL_DENSE) return dense_kernel_variants(variants, capacity, count);
    if (kernel != SPCONV_KERNEL_STRIDE1 && kernel != SPCONV_KERNEL_GENERIC && kernel != SPCONV_KERNEL_STRIDE1_TILED)
        return SPCONV_EINVAL;
    int n = 0;
    auto put = [&](int a, int b, int c, int d) {
        if (n < capacity) {
            variants[4 * n] = a;
            variants[4 * n + 1] = b;
            variants[4 * n + 2] = c;
            variants[4 * n + 3] = d;
        }
        ++n;
    };
    if (kernel == SPCONV_KERNEL_GENERIC) {
        put(4, 0, 4, 0);
        put(4, 0, 4, 1);
    } else {
        for (const S1Variant &v : kS1Variants)
            for (int pool = 0; pool < 2; ++pool)
                if ((v.pools & (1 << pool)) && (kernel == SPCONV_KERNEL_STRIDE1 || tiled_variant(v)))
                    put(v.pi, v.ipw, v.rpw, pool);
    }
    *count = n;
    return SPCONV_OK;
}

extern "C" int spconv_lowered_size(int N, int C, int H, int W, const spconv_csr *csr, int K, int R, int S, int stride,
                                   int pad, uint32_t flags, const spconv_options *opt, int64_t *words) {
    if (!words) return SPCONV_EINVAL;
    Plan pl;
    FwdArgs a;
    int rc = prepare_forward(N, C, H, W, csr, K, R, S, stride, pad, flags, opt ? opt->max_row_nnz : 0, true, &pl,
                             &a);
    if (rc != SPCONV_OK) return rc;
    rc = apply_epilogue(opt, &a);
    if (rc != SPCONV_OK) return rc;
    if (pl.kind != Kind::kStride1) return SPCONV_EINVAL;
    const long long w = lowered_words(pl, csr->nnz);
    if (w >= (1LL << 31)) return SPCONV_EINVAL;
    *words = w;
    return SPCONV_OK;
}

namespace {

// Issue shares of the four waves of a SIMD by age (waves w, w+4, w+8, w+12
// run on SIMD w % 4, oldest first): the SIMD's arbiter serves the oldest
// ready wave first, so with equal entry counts the four finish a chunk in age
// order, ~0.4 us apart on 8 us chunks, and the SIMD ends each chunk with one
// or two waves that cannot hide the LDS latency. Giving older waves
// proportionally more entries lets the four finish together (measured over
// the workloads' layers: 1-4% faster than equal shares; wider spreads no
// better).
constexpr int kAgeShare[4] = {120, 107, 93, 80};
constexpr int kAgeShareSum = kAgeShare[0] + kAgeShare[1] + kAgeShare[2] + kAgeShare[3];

// Refines the assignment of a channel tile's rows to (wave, slot) so that the
// waves' work is even within every chunk, not only over the whole row: the
// workgroup waits at each chunk's barrier for its busiest SIMD (waves w,
// w+4, w+8, w+12 share one), and a wave given more than its age share of the
// SIMD's issue slots (kAgeShare) finishes late. Cost of a chunk: the largest
// over SIMDs of max(SIMD entries, each wave's entries scaled by its share),
// in units where both equal the SIMD's time; the assignment takes the best
// swap of two rows of different waves while that lowers the sum over chunks
// (deterministic, a bounded number of passes). slot_row[w*RPW + i] is a row
// (k >= K: an empty slot).
void balance_slots(std::vector<int> &slot_row, const int32_t *rp, const int32_t *ci, int K, int RS, int Cc,
                   int nchunks, int RPW) {
    const int KT = (int)slot_row.size();
    constexpr int kSimds = 4;
    // Entries of each slot's row per chunk.
    std::vector<int> cnt((size_t)KT * nchunks, 0);
    for (int q = 0; q < KT; ++q) {
        const int k = slot_row[q];
        if (k >= K) continue;
        for (int j = rp[k]; j < rp[k + 1]; ++j) ++cnt[(size_t)q * nchunks + (ci[j] / RS) / Cc];
    }
    std::vector<int> wl((size_t)kS1Waves * nchunks, 0);  // wave loads
    for (int q = 0; q < KT; ++q)
        for (int c = 0; c < nchunks; ++c) wl[(size_t)(q / RPW) * nchunks + c] += cnt[(size_t)q * nchunks + c];
    auto chunk_cost = [&](int c) {
        long long worst = 0;
        for (int sm = 0; sm < kSimds; ++sm) {
            long long sum = 0, top = 0;
            for (int w = sm; w < kS1Waves; w += kSimds) {
                const long long v = wl[(size_t)w * nchunks + c];
                sum += v;
                top = std::max(top, v * kAgeShareSum * 1000 / kAgeShare[w / kSimds]);
            }
            worst = std::max(worst, std::max(sum * 1000, top));
        }
        return worst;
    };
    auto total = [&]() {
        long long t = 0;
        for (int c = 0; c < nchunks; ++c) t += chunk_cost(c);
        return t;
    };
    auto swap_rows = [&](int a, int b) {
        const int wa = a / RPW, wb = b / RPW;
        for (int c = 0; c < nchunks; ++c) {
            const int da = cnt[(size_t)a * nchunks + c], db = cnt[(size_t)b * nchunks + c];
            wl[(size_t)wa * nchunks + c] += db - da;
            wl[(size_t)wb * nchunks + c] += da - db;
            std::swap(cnt[(size_t)a * nchunks + c], cnt[(size_t)b * nchunks + c]);
        }
        std::swap(slot_row[a], slot_row[b]);
    };
    long long cur = total();
    for (int pass = 0; pass < 64; ++pass) {
        long long best = cur;
        int ba = -1, bb = -1;
        for (int a = 0; a < KT; ++a)
            for (int b = a + 1; b < KT; ++b) {
                if (a / RPW == b / RPW) continue;
                swap_rows(a, b);
                const long long t = total();
                swap_rows(a, b);
                if (t < best) {
                    best = t;
                    ba = a;
                    bb = b;
                }
            }
        if (ba < 0) break;
        swap_rows(ba, bb);
        cur = best;
    }
}

}  // namespace

extern "C" int spconv_pack_lowered(int N, int C, int H, int W, const spconv_csr *csr, int K, int R, int S, int stride,
                                   int pad, uint32_t flags, const spconv_options *opt, int32_t *lowered,
                                   int64_t capacity) {
    if (!lowered) return SPCONV_EINVAL;
    int64_t words = 0;
    int rc = spconv_lowered_size(N, C, H, W, csr, K, R, S, stride, pad, flags, opt, &words);
    if (rc != SPCONV_OK) return rc;
    Plan pl;
    FwdArgs a;
    rc = prepare_forward(N, C, H, W, csr, K, R, S, stride, pad, flags, opt ? opt->max_row_nnz : 0, true, &pl,
                             &a);
    if (rc != SPCONV_OK) return rc;
    // The CSR, read on the host: a valid (K, C*R*S) matrix.
    const long long nnz = csr->nnz, cols = (long long)C * R * S;
    const int32_t *rp = csr->rowptr, *ci = csr->colidx;
    const float *va = csr->vals;
    if (!rp || (nnz > 0 && (!ci || !va)) || rp[0] != 0 || rp[K] != nnz) return SPCONV_EINVAL;
    for (int k = 0; k < K; ++k) {
        if (rp[k + 1] < rp[k]) return SPCONV_EINVAL;
        for (int j = rp[k]; j < rp[k + 1]; ++j)
            if (ci[j] < 0 || ci[j] >= cols || (j > rp[k] && ci[j] <= ci[j - 1])) return SPCONV_EINVAL;
    }
    if (capacity < words) return SPCONV_ECAPACITY;
    const int KT = kS1Waves * pl.RPW;
    const int nh = lowered_headers(pl);
    int32_t *hdr = lowered;
    int32_t *ent = lowered + 4LL * nh;
    long long e = 0;  // entries written
    std::vector<int> slot_row(KT);
    std::vector<int> order(KT);
    for (int kt = 0; kt < pl.nktiles; ++kt) {
        const int k0 = kt * KT;
        // Rows of this channel tile by entry count, most first (ties: lower
        // channel first), dealt to (slot i, wave w) in snake order: ranks
        // i*16 + w for even i, i*16 + 15 - w for odd i (one row per wave
        // needs no ranking); then balanced chunk by chunk (balance_slots).
        for (int j = 0; j < KT; ++j) order[j] = j;
        auto nz = [&](int j) { return k0 + j < K ? rp[k0 + j + 1] - rp[k0 + j] : -1; };
        if (pl.RPW > 1)
            std::stable_sort(order.begin(), order.end(), [&](int x, int y) { return nz(x) > nz(y); });
        for (int r = 0; r < KT; ++r) {
            const int i = r / kS1Waves, w = (i & 1) ? kS1Waves - 1 - r % kS1Waves : r % kS1Waves;
            slot_row[w * pl.RPW + i] = k0 + order[r];
        }
        balance_slots(slot_row, rp, ci, K, R * S, pl.Cc, pl.nchunks, pl.RPW);
        for (int w = 0; w < kS1Waves; ++w)
            for (int i = 0; i < pl.RPW; ++i) {
                const int k = slot_row[w * pl.RPW + i];
                for (int ch = 0; ch < pl.nchunks; ++ch) {
                    int32_t *h = hdr + 4LL * (((long long)(kt * kS1Waves + w) * pl.RPW + i) * pl.nchunks + ch);
                    h[0] = (int32_t)e;
                    h[1] = h[2] = 0;
                    h[3] = k < K ? k : K;
                    if (k >= K) continue;
                    const int c0 = ch * pl.Cc, c1 = std::min(C, c0 + pl.Cc);
                    for (int parity = 0; parity < 2; ++parity)
                        for (int j = rp[k]; j < rp[k + 1]; ++j) {
                            const int c = ci[j] / (R * S), t = ci[j] % (R * S);
                            if (c < c0 || c >= c1) continue;
                            const int idx = (c - c0) * pl.PLp + (t / S) * a.vp + (t % S) + a.lds_shift;
                            if ((idx & 1) != parity) continue;
                            ent[2 * e] = idx - parity;
                            std::memcpy(&ent[2 * e + 1], &va[j], sizeof(float));
                            ++e;
                            ++h[1 + parity];
                        }
                }
            }
    }
    if (e != nnz) return SPCONV_EINVAL;  // every entry lies in one chunk of one slot
    std::memset(ent + 2 * e, 0, sizeof(int32_t) * 2 * kLwPad);
    return SPCONV_OK;
}
