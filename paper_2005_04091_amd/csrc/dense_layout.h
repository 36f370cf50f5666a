// Layout of the packed dense filter shared by the host packer (pack.cpp) and
// the dense kernel's host code (dense.hip); internal header, host only.
#pragma once

#include <algorithm>

namespace dense_layout {

constexpr int kTile = 32;      // MFMA tile: 32 output channels x 32 pixels
constexpr int kMaxWaves = 4;   // channel tiles (of 32) per workgroup

inline int round_up(int a, int b) { return (a + b - 1) / b * b; }

// Channel tiles of 32 per workgroup for K output channels.
inline int waves(int K) { return std::min(kMaxWaves, (K + kTile - 1) / kTile); }

// Kp of the packed filter: K rounded up to whole workgroup channel tiles.
inline int kp(int K) { return round_up(K, kTile * waves(K)); }

}  // namespace dense_layout
