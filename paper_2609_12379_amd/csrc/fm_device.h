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
//   * Attention partials are tagged words too. The items holding a (lane, KV head) group's
//     last chunks wait for the group's other partials and merge them, a set of heads each.
//   * Weights and the KV cache are streamed with non-temporal 128-bit buffer loads.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fm_limits.h"

namespace fm {
namespace dev {

typedef uint32_t u32;
typedef uint64_t u64;
typedef u32 u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int NT = 512;              // threads per workgroup
constexpr int NWAVE = NT / 64;
// Wave roles inside a GEMV tile: streaming waves only load weights; control waves only poll
// and stage the inputs. A wave's memory operations complete in issue order, so a wave that
// polled its input behind its own weight prefetch would see the input only after the
// prefetch landed.
// Measured on MI355X: splitting roles (2 control + 6 streaming waves) was slower than
// letting all 8 waves do both, so NCTL = 0 (every wave streams and stages).
#ifndef FM_RING
#define FM_RING 4
#endif
#ifndef FM_NCTL
#define FM_NCTL 0
#endif
constexpr int NCTL = FM_NCTL;
constexpr int NSW = NWAVE - NCTL;
// LDS of a workgroup (158 KB of the CU's 160 KB), laid out per operator:
//   GEMV tiles: [activation slab][row sums ROWACC][residual rows RESID][MISC];
//   attention items: [merger's partials, kMergeFloats] ... [item scratch ATT][MISC].
// Matrix-core (batched) tiles need fewer row sums and a larger slab.
constexpr int LDS_FLOATS = 40448;
constexpr int MISC_FLOATS = 1024;   // block reductions, argmax keys, chunk ids; timeline marks in the last 24
// Each lane's token, position and KV length for the step, copied into the misc area at
// kernel start (words LANE_IN .. LANE_IN + 24: tokens, then positions, then KV lengths, 8
// each). Read through an LDS pointer they wait on no memory counter, so reading them never
// waits for loads or stores in flight.
constexpr int LANE_IN = 640;
typedef __attribute__((address_space(3))) int lds_i32;
constexpr int RESID_FLOATS = 2048;  // residual rows staged for the epilogue
constexpr int ATT_FLOATS = 9600;    // q heads, k, v and per-wave partials of one item (G <= 8, d <= 128)
template <int B> constexpr int rowacc_floats() { return B >= 4 ? 4096 : 8192; }
template <int B> constexpr int xslab_floats() {
  return LDS_FLOATS - MISC_FLOATS - RESID_FLOATS - rowacc_floats<B>();
}
static_assert(kMergeFloats + ATT_FLOATS + MISC_FLOATS <= LDS_FLOATS, "attention LDS layout");
static_assert(xslab_floats<1>() == kXslabFloatsVALU && xslab_floats<2>() == kXslabFloatsVALU &&
              rowacc_floats<1>() == kRowaccFloatsVALU, "the scheduler's view of the VALU tile's LDS");

constexpr u32 CPOL_NT = 2;    // non-temporal (streaming)
constexpr u32 CPOL_SC1 = 16;  // device-scope coherent

struct LayerPtrs {
  const uint16_t *attn_norm, *wq, *wk, *wv, *q_norm, *k_norm, *wo, *mlp_norm, *wg, *wu, *wd;
  uint16_t *kc, *vc;
};

// Everything about the model and the handle's scratch; uploaded once to device memory.
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
  // scratch: tagged words, word offsets into `act`
  u64* act;
  u32 act_bytes;
  u32 off_x, off_qkv, off_o, off_x1, off_m;      // bases; per-layer strides below
  u32 st_x, st_qkv, st_o, st_x1, st_m;           // words per layer (all lanes)
  const uint16_t* zero_page;      // 64 KiB of zeros: the target of loads with nothing to load
  u64* part;                     // tagged [L][b][nh][maxc][d + 2]: split-KV partials
  u64* amax;                     // [b]
  u32* lm_arrive;                // [1]
  u32* dyn_ctr;                  // [kPools][dyn_stride]: claim counters of dynamic GEMV stages
  int32_t dyn_stride;            // counters per pool (one per GEMV stage, padded to 128 bytes)
  u32* abort_flag;               // [1]
  u32* err_host;                 // pinned host word
  int64_t tap_block;             // floats per (layer, lane) block
  int32_t tap_a, tap_qkv, tap_qrot, tap_krot, tap_o, tap_x1, tap_a2, tap_mlp, tap_x2;
};

// Params is read through the constant address space: scalar loads that no store can alias,
// so reading a field never stalls on (or is re-issued after) outstanding memory operations.
typedef __attribute__((address_space(4))) const Params CParams;
typedef __attribute__((address_space(4))) const LayerPtrs CLayerPtrs;

// Per-step arguments, passed by value with each launch (Params lives in device memory).
struct Step {
  const int32_t *tok, *pos, *kvl;
  float* logits;
  int32_t* next_ids;
  float* taps;                   // optional mid-state taps
  u64* timeline;                 // optional: per instruction {start, inputs ready, end, wg}
  u32 epoch;
  int32_t stage;                 // -1: whole step in one launch; else one stage
};

// ---- small helpers ---------------------------------------------------------------------

typedef __attribute__((address_space(1))) const u32x4 global_u32x4;

// 16-byte non-temporal load through the global (not flat) address space, so it is tracked
// by vmcnt only and never delays an LDS wait.
__device__ __forceinline__ u32x4 ld_stream16(const void* p) {
  return __builtin_nontemporal_load((const global_u32x4*)p);
}

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

// Value of another lane of the same 16-lane row (DPP control ctl: a lane permutation inside
// each quad, a mirror or a rotation of the row, for which every lane has a source). Written as
// a DPP update with bound_ctrl so that an add of the result folds into one v_add_f32_dpp.
template <int CTL>
__device__ __forceinline__ float dpp_row(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTL, 0xF, 0xF, true));
}
constexpr int DPP_QUAD_1032 = 0xB1, DPP_QUAD_2301 = 0x4E, DPP_HALF_MIRROR = 0x141, DPP_MIRROR = 0x140;
constexpr int DPP_ROR4 = 0x124, DPP_ROR8 = 0x128;

// Sum within each 16-lane row; every lane of the row gets the total (DPP, no LDS).
__device__ __forceinline__ float row16_sum(float s) {
  s += dpp_row<DPP_QUAD_1032>(s);
  s += dpp_row<DPP_QUAD_2301>(s);
  s += dpp_row<DPP_HALF_MIRROR>(s);
  s += dpp_row<DPP_MIRROR>(s);
  return s;
}

// Value of lane (lane xor 16) / (lane xor 32), on the VALU. permlane16_swap(a, a): the first
// result holds row r & ~1 in both rows of a pair, the second row r | 1; permlane32_swap(a, a):
// the first result holds lanes 0-31 in both halves, the second 32-63.
__device__ __forceinline__ u32 xor16_u32(u32 v, int lane) {
  auto p = __builtin_amdgcn_permlane16_swap(v, v, false, false);
  return ((lane >> 4) & 1) ? p[0] : p[1];
}
__device__ __forceinline__ u32 xor32_u32(u32 v, int lane) {
  auto p = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  return (lane >> 5) ? p[0] : p[1];
}

// Sum over the wave; every lane gets the same total. VALU only (DPP within rows, permlane
// swaps across them): cross-lane shuffles through the LDS crossbar cost about 100 cycles per
// dependent step.
__device__ __forceinline__ float wave_sum(float v) {
  const int lane = __lane_id();
  v = row16_sum(v);
  v += __uint_as_float(xor16_u32(__float_as_uint(v), lane));
  v += __uint_as_float(xor32_u32(__float_as_uint(v), lane));
  return v;
}

// Maximum of a 64-bit key over the wave (same exchanges as wave_sum).
__device__ __forceinline__ u64 wave_max_u64(u64 k) {
  const int lane = __lane_id();
  auto take = [&](u32 lo, u32 hi) {
    const u64 o = ((u64)hi << 32) | lo;
    k = o > k ? o : k;
  };
#define FM_DPP_U32(v, ctl) ((u32)__builtin_amdgcn_mov_dpp((int)(v), ctl, 0xF, 0xF, false))
  take(FM_DPP_U32(k, 0xB1), FM_DPP_U32(k >> 32, 0xB1));
  take(FM_DPP_U32(k, 0x4E), FM_DPP_U32(k >> 32, 0x4E));
  take(FM_DPP_U32(k, 0x141), FM_DPP_U32(k >> 32, 0x141));
  take(FM_DPP_U32(k, 0x140), FM_DPP_U32(k >> 32, 0x140));
#undef FM_DPP_U32
  take(xor16_u32((u32)k, lane), xor16_u32((u32)(k >> 32), lane));
  take(xor32_u32((u32)k, lane), xor32_u32((u32)(k >> 32), lane));
  return k;
}

__device__ __forceinline__ u64 clock_now() { return wall_clock64(); }

// Instruction timeline marks are kept in LDS while an instruction runs (and written to memory
// when it ends): a store to memory in the middle of an operator would make its next full wait
// for loads also wait for the store's acknowledgement.
typedef __attribute__((address_space(3))) u64 tl_t;
__device__ __forceinline__ lds_i32* lane_inputs(float* smem) {
  return (lds_i32*)(__attribute__((address_space(3))) float*)(smem + LDS_FLOATS - MISC_FLOATS + LANE_IN);
}

// Watchdog bound on any single wait (wall clock runs at 100 MHz on MI355X): 2 s.
constexpr u64 WAIT_TICKS = 200000000ull;

}  // namespace dev
}  // namespace fm
