// Sizes shared by the host scheduler and the device code.
#pragma once

namespace fm {
// LDS floats a workgroup has for one operator's staged data: the activation slab of a GEMV
// tile, or the split-KV partials of one (lane, KV head) group in the combine.
constexpr int kSlabFloats = 24576;
}  // namespace fm
