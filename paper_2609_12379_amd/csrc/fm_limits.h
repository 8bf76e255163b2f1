// Sizes shared by the host scheduler and the device code.
#pragma once

namespace fm {
// LDS floats for the split-KV partials of one (lane, KV head) group, staged by its merger.
constexpr int kMergeFloats = 24576;

// GEMV stages in dynamic chunks (VALU tiles, batch <= 2).
// LDS of a VALU tile: the activation slab (input vector, plus the residual vector when the
// stage adds one) and the row sums of the chunks a workgroup takes.
constexpr int kXslabFloatsVALU = 29184;
constexpr int kRowaccFloatsVALU = 8192;
// Claim pools per stage: workgroup w serves pool w mod kPools (on MI355X, the workgroups of
// one XCD).
constexpr int kPools = 8;
// Chunks one workgroup may take in one stage (LDS list of chunk ids).
constexpr int kDynMaxSlots = 48;
// Target weight bytes per chunk (automatic setting), and the fewest chunks per workgroup
// worth the claims.
#ifndef FM_DYN_CHUNK_KB
#define FM_DYN_CHUNK_KB 128
#endif
constexpr long long kDynChunkBytes = (long long)FM_DYN_CHUNK_KB << 10;
constexpr int kDynMinPerWg = 2;
constexpr int kDynMaxPerWg = 16;
// Each wave streams one item of every chunk: at least this many 16-byte units (128-column
// segments), so that the next chunk can be claimed one ring round ahead.
constexpr int kDynMinSegs = 8;
}  // namespace fm
