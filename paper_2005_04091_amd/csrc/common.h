// Device helpers shared by the kernels of libspconv (internal header).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <mutex>
#include <set>
#include <utility>

namespace {

constexpr int kWave = 64;
constexpr int kXcds = 8;  // MI355X: 8 XCDs, workgroups dispatched round-robin

typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(1))) void global_void_t;

// Streaming stores (nontemporal): every output tensor of this library is
// written once, by whole cache lines, and read back (if at all) by the next
// kernel; on gfx950 such stores sustain a markedly higher write rate than
// ordinary ones.
typedef float f32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ void stream_store(float *p, float v) { __builtin_nontemporal_store(v, p); }

// Output element store of the conv kernels: streaming when the planes are
// stored without a border (whole lines written by the same kernel's streaming
// stores); ordinary when a border is written around them, where rows start
// mid-line and share lines with the border's scattered ordinary stores (mixing
// the two on one line measured ~10% slower).
__device__ __forceinline__ void store_out(float *p, float v, bool stream) {
    if (stream)
        stream_store(p, v);
    else
        *p = v;
}

// Two adjacent floats at any 4-byte boundary: gfx9 global loads and stores of
// two dwords need only dword alignment.
typedef float f32x2_a4_t __attribute__((ext_vector_type(2), aligned(4)));

// Two adjacent output elements (p 4-byte aligned); streaming as store_out.
__device__ __forceinline__ void store_out2(float *p, float2 v, bool stream) {
    const f32x2_a4_t t = {v.x, v.y};
    if (stream)
        __builtin_nontemporal_store(t, reinterpret_cast<f32x2_a4_t *>(p));
    else
        *reinterpret_cast<f32x2_a4_t *>(p) = t;
}

__device__ __forceinline__ void stream_store4(float *p, float4 v) {
    const f32x4_t t = {v.x, v.y, v.z, v.w};
    __builtin_nontemporal_store(t, reinterpret_cast<f32x4_t *>(p));
}

// x / d for x < 2^31 as one multiply-high and a shift, with (magic, shift)
// from div_magic(d) on the host (round-up reciprocal, shift 31 + ceil(log2 d)).
__device__ __forceinline__ uint32_t fast_div(uint32_t x, uint32_t magic, int shift) {
    return (uint32_t)(((uint64_t)x * (uint64_t)magic) >> shift);
}

inline bool div_magic(uint32_t d, uint32_t *magic, int *shift) {
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

// Work units u = q*n + r (0 <= r < n) dealt round-robin to `step` waves: wave
// w takes u = w, w + step, ... The staging loops walk (q, r) without a
// division per unit (a loop of subtractions cost up to step/n scalar
// iterations per unit, 16 for one-block channel slots). UnitStep holds what
// that takes for one n: step = dq*n + dr, and recip = ceil(2^16 / n), with
// which (w * recip) >> 16 = floor(w / n) whenever w*n < 2^16: w*recip / 2^16
// exceeds w/n by less than w / 2^16 < 1/n, and the fraction of w/n is at
// most (n-1)/n.
struct UnitStep {
    int n, dq, dr;
    uint32_t recip;
};

inline bool unit_step(int n, int step, UnitStep *u) {
    if (n < 1 || step < 1 || (long long)step * n >= 65536) return false;
    u->n = n;
    u->dq = step / n;
    u->dr = step % n;
    u->recip = (65536u + (uint32_t)n - 1u) / (uint32_t)n;
    return true;
}

__device__ __forceinline__ void unit_first(const UnitStep &u, int w, int &q, int &r) {
    q = (int)(((uint32_t)w * u.recip) >> 16);
    r = w - q * u.n;
}

__device__ __forceinline__ void unit_next(const UnitStep &u, int &q, int &r) {
    q += u.dq;
    r += u.dr;
    if (r >= u.n) {
        r -= u.n;
        ++q;
    }
}

// Raise a kernel instance's dynamic-LDS limit to `bytes` on the current
// device, once per (device, instance). Every caller of one instance passes
// the same value (the most any plan of its family uses), so launches of
// different shapes from several host threads never lower the limit under
// one another.
inline bool raise_lds_limit(const void *fn, int bytes) {
    static std::mutex mu;
    static std::set<std::pair<int, const void *>> done;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return false;
    std::lock_guard<std::mutex> lock(mu);
    if (done.count({dev, fn})) return true;
    if (bytes > 65536 && hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, bytes) != hipSuccess)
        return false;
    done.insert({dev, fn});
    return true;
}

// Workgroup id -> linear work index such that consecutive work items (the
// channel tiles of one image tile, which read the same input rows) land on the
// same XCD and therefore share its L2.
__device__ __forceinline__ int xcd_linear_id(int b, int G) {
    const int xcd = b % kXcds, i = b / kXcds;
    const int per = G / kXcds, rem = G % kXcds;
    return (xcd < rem) ? xcd * (per + 1) + i : rem * (per + 1) + (xcd - rem) * per + i;
}

// Zero the border of one stored output plane (Hs x Ws inside a border of pd,
// row pitch `pitch`) for a tile of stored rows [r0, r1): the left and right
// border columns of those rows, and the top border rows when the tile is the
// first of the plane, the bottom ones when it is the last. The tiles of a
// plane partition its rows, so every border element is written exactly once.
__device__ __forceinline__ void zero_border(float *plane, int r0, int r1, int Hs, int Ws, int pd, int pitch,
                                            bool first, bool last, int lane, int nlanes) {
    const int side = (r1 - r0) * 2 * pd;
    const int top = first ? pd * pitch : 0;
    const int bottom = last ? pd * pitch : 0;
    for (int t = lane; t < side + top + bottom; t += nlanes) {
        int idx;
        if (t < side) {
            const int rr = t / (2 * pd), c = t - rr * 2 * pd;
            idx = (r0 + rr + pd) * pitch + (c < pd ? c : Ws + c);
        } else if (t < side + top) {
            idx = t - side;
        } else {
            idx = (pd + Hs) * pitch + (t - side - top);
        }
        plane[idx] = 0.0f;
    }
}

}  // namespace
