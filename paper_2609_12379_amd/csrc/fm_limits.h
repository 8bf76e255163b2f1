// Sizes shared by the host scheduler and the device code.
#pragma once

namespace fm {
// LDS floats for the split-KV partials of one (lane, KV head) group, staged by its merger.
constexpr int kMergeFloats = 24576;
}  // namespace fm
