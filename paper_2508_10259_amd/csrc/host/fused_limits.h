// Compile-time limits shared by the kernels and the host-side planning (plain
// C++: the host bookkeeping also builds without HIP).
#pragma once

namespace ams {

// Largest K splits of the persistent decode's residual projections and key
// splits of its attention (its merges keep every partial in registers).
constexpr int FUSED_MAX_SPLIT = 8;
constexpr int FUSED_MAX_ATTN_SPLIT = 16;

}  // namespace ams
