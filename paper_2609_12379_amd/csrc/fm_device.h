// Device-side building blocks of the decode step for gfx950 (CDNA4, wave64).
//
// Memory protocol between workgroups:
//   * Activations that cross workgroups (q/k/v, attention output, residual stream, MLP
//     product) are 64-bit words {fp32 value, 32-bit step epoch}, written with device-scope
//     (sc1) stores and read with device-scope (sc1) loads. A consumer waits until every
//     word it needs carries the current epoch. The data word itself is the dependency
//     counter, so a handoff costs one store and one read round trip. There is no separate
//     flag, no grid barrier, and no L2 writeback or invalidate (both cost microseconds on
//     MI355X's eight non-coherent XCD L2s).
//   * Attention partials use plain fp32 sc1 stores, published by an arrival counter that
//     is incremented after the stores complete.
//   * Weights and the KV cache are streamed with non-temporal 128-bit buffer loads.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fm {
namespace dev {

typedef uint32_t u32;
typedef uint64_t u64;
typedef u32 u32x4 __attribute__((ext_vector_type(4)));

constexpr int NT = 512;              // threads per workgroup
constexpr int NWAVE = NT / 64;
constexpr int XSLAB_FLOATS = 24576;  // activation slab (96 KB)
constexpr int ROWACC_FLOATS = 4096;  // per-row partial sums across slabs (16 KB)
constexpr int RESID_FLOATS = 2048;   // residual rows staged for the epilogue (8 KB)
constexpr int MISC_FLOATS = 512;
constexpr int LDS_FLOATS = XSLAB_FLOATS + ROWACC_FLOATS + RESID_FLOATS + MISC_FLOATS;

constexpr u32 CPOL_NT = 2;    // non-temporal (streaming)
constexpr u32 CPOL_SC1 = 16;  // device-scope coherent

struct LayerPtrs {
  const uint16_t *attn_norm, *wq, *wk, *wv, *q_norm, *k_norm, *wo, *mlp_norm, *wg, *wu, *wd;
  uint16_t *kc, *vc;
};

// Everything one launch needs; passed by value.
struct Params {
  // shape
  int32_t L, h, nh, nkv, d, inter, V, b, max_ctx, qk_norm, G;
  int32_t nwg, P, maxc, n_lm_instr;
  float eps, q_scale;            // q_scale = log2(e) / sqrt(d)
  // weights
  const LayerPtrs* layers;
  const uint16_t *embed, *final_norm, *lm_head;
  const float* rope;             // [max_ctx][d/2][2] (cos, sin)
  // schedule
  const int32_t* instrs;         // [n][4]
  const int32_t* qoff;           // [nwg + 1]
  const int32_t* stage_rng;      // [n_stages][nwg][2]
  int32_t stage;                 // -1: whole step in one launch; else one stage
  // scratch: tagged words, word offsets into `act`
  u64* act;
  u32 act_bytes;
  u32 off_x, off_qkv, off_o, off_x1, off_m;      // bases; per-layer strides below
  u32 st_x, st_qkv, st_o, st_x1, st_m;           // words per layer (all lanes)
  float* part;                   // [b][nh][maxc][d + 2]
  u32* arrive;                   // [b][nkv]
  u64* amax;                     // [b]
  u32* lm_arrive;                // [1]
  u32* abort_flag;               // [1]
  u32* err_host;                 // pinned host word
  // per step
  const int32_t *tok, *pos, *kvl;
  float* logits;
  int32_t* next_ids;
  float* taps;
  int64_t tap_block;             // floats per (layer, lane) block
  int32_t tap_a, tap_qkv, tap_qrot, tap_krot, tap_o, tap_x1, tap_a2, tap_mlp, tap_x2;
  u32 epoch;
};

// ---- small helpers ---------------------------------------------------------------------

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* p, u32 bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}

__device__ __forceinline__ void vm_wait0() {
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

__device__ __forceinline__ float bf16lo(u32 w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16hi(u32 w) { return __uint_as_float(w & 0xffff0000u); }

// Round to nearest bf16, ties to even (NaN kept quiet).
__device__ __forceinline__ uint16_t to_bf16(float f) {
  u32 u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

__device__ __forceinline__ u64 tag(float v, u32 epoch) { return ((u64)epoch << 32) | (u64)__float_as_uint(v); }

__device__ __forceinline__ void st_tag(u64* p, float v, u32 epoch) {
  __hip_atomic_store(p, tag(v, epoch), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_dev(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float ld_dev(const float* p) {
  return __hip_atomic_load(const_cast<float*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__device__ __forceinline__ u64 clock_now() { return wall_clock64(); }

// Watchdog bound on any single wait (wall clock runs at 100 MHz on MI355X): 2 s.
constexpr u64 WAIT_TICKS = 200000000ull;

}  // namespace dev
}  // namespace fm
