// Operator bodies executed by the step interpreter: GEMV row-tiles (with fused RMSNorm
// prologue, residual/SiLU/argmax epilogues) and split-KV attention work items (with fused
// QK-norm, RoPE, KV append, online softmax and the log-sum-exp merge of a group's chunks).
#pragma once
#include <type_traits>

#include "fm_device.h"
#include "../../include/fm.h"

namespace fm {
namespace dev {

// ---- waiting on tagged words ----------------------------------------------------------

__device__ __forceinline__ bool abort_raised(CParams& p) {
  return __hip_atomic_load(p.abort_flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0u;
}

__device__ __forceinline__ void raise_error(CParams& p, u32 code) {
  __hip_atomic_store(p.abort_flag, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __hip_atomic_store(p.err_host, code, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

// Reads the tagged pair at word offset w (even), spinning until both words carry the
// epoch. Returns false if the watchdog fires or another workgroup raised the abort flag.
__device__ __forceinline__ bool wait_pair(CParams& p, const Step& st, __amdgpu_buffer_rsrc_t ra, u32 w,
                                          float& a, float& b) {
  u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(ra, w * 8u, 0, CPOL_SC1);
  if (v.y != st.epoch || v.w != st.epoch) {
    const u64 t0 = clock_now();
    int it = 0;
    while (true) {
      __builtin_amdgcn_s_sleep(1);
      v = __builtin_amdgcn_raw_buffer_load_b128(ra, w * 8u, 0, CPOL_SC1);
      if (v.y == st.epoch && v.w == st.epoch) break;
      if ((++it & 63) == 0) {
        if (clock_now() - t0 > WAIT_TICKS) {
          raise_error(p, FM_DEV_WATCHDOG);
          return false;
        }
        if (abort_raised(p)) return false;
      }
    }
  }
  a = __uint_as_float(v.x);
  b = __uint_as_float(v.z);
  return true;
}

// Wait for n (even) tagged words at word offset w0 and copy their values to dst (LDS);
// accumulates the sum of squares of the values this thread copied into ss. Each thread
// issues up to WB pair loads before checking any of them, so a vector costs one round trip
// when its producers are done. Stale pairs are re-polled together, one round trip per
// retry whatever their number. Values are consumed in index order once all are current, so
// the sum of squares does not depend on which pairs had to wait.
constexpr int WB = 8;
// Pair loads in flight per thread when only the control waves stage a GEMV input.
constexpr int WBC = NCTL ? 16 : WB;
template <int WBT>
__device__ __forceinline__ bool repoll(CParams& p, const Step& st, __amdgpu_buffer_rsrc_t ra, const u32 (&w)[WBT],
                                       u32x4 (&v)[WBT], u32 pend) {
  const u64 t0 = clock_now();
  int it = 0;
  while (pend) {
    __builtin_amdgcn_s_sleep(1);
#pragma unroll
    for (int j = 0; j < WBT; ++j)
      if (pend & (1u << j)) v[j] = __builtin_amdgcn_raw_buffer_load_b128(ra, w[j] * 8u, 0, CPOL_SC1);
#pragma unroll
    for (int j = 0; j < WBT; ++j)
      if ((pend & (1u << j)) && v[j].y == st.epoch && v[j].w == st.epoch) pend &= ~(1u << j);
    if (pend && (++it & 63) == 0) {
      if (clock_now() - t0 > WAIT_TICKS) {
        raise_error(p, FM_DEV_WATCHDOG);
        return false;
      }
      if (abort_raised(p)) return false;
    }
  }
  return true;
}

// Polls n (even) tagged words from word w0 on, pairs k = t*2 + j*nthr*2 as wait_copy_t does,
// and hands each pair, once current, to use(k, a, b, side) in index order. side is the u32
// at side[k / 2] (a pair of bf16 gains), loaded with the poll; 0 when side is null.
// One batch of pair loads per thread (pairs k = k0 + j * nthr * 2, j < WBT), with their side
// words.
template <int WBT>
struct PairBatch {
  u32x4 v[WBT];
  u32 w[WBT], sv[WBT];
};

template <int WBT>
__device__ __forceinline__ void issue_pairs(__amdgpu_buffer_rsrc_t ra, u32 w0, int n, const u32* side, int k0,
                                            int nthr, PairBatch<WBT>& b) {
#pragma unroll
  for (int j = 0; j < WBT; ++j) {
    const int k = k0 + j * nthr * 2;
    b.w[j] = (k < n) ? w0 + (u32)k : 0x1FFFFFFEu;
    b.v[j] = __builtin_amdgcn_raw_buffer_load_b128(ra, (k < n) ? b.w[j] * 8u : 0xFFFFFFF0u, 0, CPOL_SC1);
    b.sv[j] = (side && k < n) ? side[k >> 1] : 0u;
  }
}

template <int WBT, class Use>
__device__ __forceinline__ bool finish_pairs(CParams& p, const Step& st, __amdgpu_buffer_rsrc_t ra, int n, Use use,
                                             int k0, int nthr, PairBatch<WBT>& b) {
  u32 pend = 0;
#pragma unroll
  for (int j = 0; j < WBT; ++j) {
    const int k = k0 + j * nthr * 2;
    if (k < n && (b.v[j].y != st.epoch || b.v[j].w != st.epoch)) pend |= 1u << j;
  }
  if (pend && !repoll<WBT>(p, st, ra, b.w, b.v, pend)) return false;
#pragma unroll
  for (int j = 0; j < WBT; ++j) {
    const int k = k0 + j * nthr * 2;
    if (k < n) use(k, __uint_as_float(b.v[j].x), __uint_as_float(b.v[j].z), b.sv[j]);
  }
  return true;
}

// Pairs per thread of an input's early poll batch, issued ahead of the weight prefetch: with 512
// threads a vector of up to 4096 values, and few registers held across the prefetch. Longer
// inputs are polled after the prefetch in full batches as before (split, they would cost an
// extra round trip).
constexpr int WBF = 4;
// Pairs per thread in one batch for long inputs of the batch-1 dynamic-chunk stages (up to
// 14336 values: the down projection's input on the 7B-13B shapes), which would otherwise take
// two round trips. (At batch 2 the registers are not there.)
constexpr int WBL = 14;

// first: the caller's first WBF pairs (k0 = t * 2), already issued with the same arguments, or
// null.
template <int WBT, class Use>
__device__ __forceinline__ bool wait_pairs(CParams& p, const Step& st, __amdgpu_buffer_rsrc_t ra, u32 w0, int n,
                                           const u32* side, Use use, int t, int nthr,
                                           PairBatch<WBF>* first = nullptr) {
  int k0 = t * 2;
  if (first) {
    if (!finish_pairs<WBF>(p, st, ra, n, use, k0, nthr, *first)) return false;
    k0 += nthr * 2 * WBF;
  }
  for (; k0 < n; k0 += nthr * 2 * WBT) {
    PairBatch<WBT> b;
    issue_pairs<WBT>(ra, w0, n, side, k0, nthr, b);
    if (!finish_pairs<WBT>(p, st, ra, n, use, k0, nthr, b)) return false;
  }
  return true;
}

template <int WBT = WB>
__device__ __forceinline__ bool wait_copy_t(CParams& p, const Step& st, __amdgpu_buffer_rsrc_t ra, u32 w0, int n,
                                            float* dst, float& ss, int t, int nthr) {
  auto use = [&](int k, float a, float b, u32) {
    ss += a * a + b * b;
    if (dst) {
      dst[k] = a;
      dst[k + 1] = b;
    }
  };
  return wait_pairs<WBT>(p, st, ra, w0, n, nullptr, use, t, nthr);
}

__device__ __forceinline__ bool wait_copy(CParams& p, const Step& st, __amdgpu_buffer_rsrc_t ra, u32 w0, int n,
                                          float* dst, float& ss, int tid) {
  return wait_copy_t<WB>(p, st, ra, w0, n, dst, ss, tid, NT);
}

// Waits for n (even) tagged words whose pair k (k even) lives at word where(k) and goes to
// LDS at dst(k): the same batched polling as wait_copy_t over an arbitrary index map.
template <int WBT, class Where>
__device__ __forceinline__ bool wait_copy_map(CParams& p, const Step& st, __amdgpu_buffer_rsrc_t ra, int n,
                                              Where where, int tid) {
  for (int k0 = tid * 2; k0 < n; k0 += NT * 2 * WBT) {
    u32x4 v[WBT];
    u32 w[WBT];
    u32 pend = 0;
#pragma unroll
    for (int j = 0; j < WBT; ++j) {
      const int k = k0 + j * NT * 2;
      float* d = nullptr;
      w[j] = 0x1FFFFFFEu;
      if (k < n) where(k, w[j], d);
      v[j] = __builtin_amdgcn_raw_buffer_load_b128(ra, (k < n) ? w[j] * 8u : 0xFFFFFFF0u, 0, CPOL_SC1);
    }
#pragma unroll
    for (int j = 0; j < WBT; ++j) {
      const int k = k0 + j * NT * 2;
      if (k < n && (v[j].y != st.epoch || v[j].w != st.epoch)) pend |= 1u << j;
    }
    if (pend && !repoll<WBT>(p, st, ra, w, v, pend)) return false;
#pragma unroll
    for (int j = 0; j < WBT; ++j) {
      const int k = k0 + j * NT * 2;
      if (k < n) {
        u32 ww; float* d;
        where(k, ww, d);
        d[0] = __uint_as_float(v[j].x);
        d[1] = __uint_as_float(v[j].z);
      }
    }
  }
  return true;
}

// wait_copy_map in two halves for inputs of at most NT * 2 * WBT words (one batch): the
// polls are issued first, other loads may follow, and the caller finishes later; loads
// return in issue order, so the polls are not held up by what was issued after them.
template <int WBT>
struct MapBatch {
  u32x4 v[WBT];
  u32 w[WBT];
};

template <int WBT, class Where>
__device__ __forceinline__ void issue_map(__amdgpu_buffer_rsrc_t ra, int n, Where where, int tid, MapBatch<WBT>& b) {
#pragma unroll
  for (int j = 0; j < WBT; ++j) {
    const int k = tid * 2 + j * NT * 2;
    float* d = nullptr;
    b.w[j] = 0x1FFFFFFEu;
    if (k < n) where(k, b.w[j], d);
    b.v[j] = __builtin_amdgcn_raw_buffer_load_b128(ra, (k < n) ? b.w[j] * 8u : 0xFFFFFFF0u, 0, CPOL_SC1);
  }
}

template <int WBT, class Where>
__device__ __forceinline__ bool finish_map(CParams& p, const Step& st, __amdgpu_buffer_rsrc_t ra, int n, Where where,
                                           int tid, MapBatch<WBT>& b) {
  u32 pend = 0;
#pragma unroll
  for (int j = 0; j < WBT; ++j) {
    const int k = tid * 2 + j * NT * 2;
    if (k < n && (b.v[j].y != st.epoch || b.v[j].w != st.epoch)) pend |= 1u << j;
  }
  if (pend && !repoll<WBT>(p, st, ra, b.w, b.v, pend)) return false;
#pragma unroll
  for (int j = 0; j < WBT; ++j) {
    const int k = tid * 2 + j * NT * 2;
    if (k < n) {
      u32 ww; float* d;
      where(k, ww, d);
      d[0] = __uint_as_float(b.v[j].x);
      d[1] = __uint_as_float(b.v[j].z);
    }
  }
  return true;
}


// Sum over the workgroup; every thread gets the total. Uses misc[0..NWAVE).
__device__ __forceinline__ float block_sum(float v, float* misc, int lane, int wave) {
  v = wave_sum(v);
  __syncthreads();
  if (lane == 0) misc[wave] = v;
  __syncthreads();
  float t = 0.f;
#pragma unroll
  for (int w = 0; w < NWAVE; ++w) t += misc[w];
  return t;
}

__device__ __forceinline__ float silu(float z) { return z / (1.0f + expf(-z)); }

__device__ __forceinline__ u32 ordered(float f) {
  u32 u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// ---- GEMV row tile ---------------------------------------------------------------------
//
// Output rows [ra, rb) of one operator for B lanes (B = batch rounded up to 1, 2, 4, 8), with
// NW weight rows per output row (2 for gate/up: weight row wr = 2 q + {0: gate, 1: up}).
//
// Lane layout: 16 lanes per weight row, 4 rows per wave load. A load ("unit") is 16 B per lane
// = 128 columns of each of 4 rows ("quad"), so one reduction is a 4-step DPP sum inside each
// 16-lane row and the activation chunk is an LDS broadcast. Quads are split along K into KP
// parts when the tile has fewer quads than waves, so every wave keeps its U ring loads in
// flight whatever the tile's shape. Items (quad, part) are dealt to waves round-robin; a wave's units
// run item by item, SP segments per item. Part sums land in LDS and are added in part order
// by the epilogue, so results do not depend on timing.
//
// Every ring slot issues exactly one global load per round (so the compiler counts loads in
// flight exactly); lanes with nothing to load read a zeroed page instead. The last round
// issues none.
//
// Batch-8 tiles run the products on the matrix cores instead (a skinny GEMM): a unit is
// then 16 weight rows x 32 columns, loaded in the A-operand layout of
// v_mfma_f32_16x16x32_bf16 (lane l: row l % 16, columns 8 (l / 16) .. + 8, still one 16 B
// load per lane). The B operand is the activation slab: each fp32 value x is split into three
// bf16 planes hi = rne(x), mid = rne(x - hi), lo = rne(x - hi - mid), and all three go
// through the matrix core into the same fp32 accumulator, so the product keeps about 24 bits
// of the activation's mantissa. Lanes 16 .. of the B operand's 16 columns (batch lanes past B)
// are zero. (At batch 4 the VALU tiles measured faster on MI355X; at batch 8 the matrix
// cores.)

struct GemvGeom {
  int K, Ks, nslab;           // columns, slab width, slabs
  int nwr, NQ, KP, nitems;    // weight rows, quads, K parts, items
  int nseg, SP, kend, k0;     // current slab: segments, segments per part, column bound/start
  int items_w;                // items of this wave
};

struct GemvCursor {
  int it, sg;                 // wave-local item and segment within it
  int qd, pt;                 // its quad and K part
  bool live;                  // item exists
};

// Wave-uniform integers are passed through readfirstlane so the compiler keeps them (and
// the branches on them) scalar; otherwise the ring's loads end up under divergent control
// flow and the compiler can no longer count them in flight.
__device__ __forceinline__ int uni(int v) { return __builtin_amdgcn_readfirstlane(v); }

__device__ __forceinline__ void cursor_at(GemvCursor& c, const GemvGeom& g, int it, int wave) {
  c.it = uni(it); c.sg = 0;
  const int t = uni(wave + it * NSW);
  c.live = uni(it < g.items_w ? 1 : 0) != 0;
  c.qd = uni(t / g.KP);
  c.pt = uni(t - c.qd * g.KP);
}

__device__ __forceinline__ void cursor_next(GemvCursor& c, const GemvGeom& g, int wave) {
  c.sg = uni(c.sg + 1);
  if (c.sg == g.SP) cursor_at(c, g, c.it + 1, wave);
}

// Issues the load of the cursor's unit into `dst`: exactly one load per call, so the number
// of loads in flight behind any ring slot is a compile-time constant and the wait for a slot
// is a partial one (vmcnt(U - 1)). Lanes with nothing to load (units past the wave's items
// or the slab's segments, rows past the tile, the ragged last segment) read their slot of
// the zero page, which stays in cache.
// Unit shape: 4 rows x 128 columns (VALU tiles) or 16 rows x 32 columns (matrix-core tiles).
// Padding of each matrix-core activation plane row, in bf16 values (16 bytes).
constexpr int XPAD = 8;

template <bool MF> struct UnitShape {
  static constexpr int rows = MF ? 16 : 4, cols = MF ? 32 : 128;
  __device__ static int row(int lane) { return MF ? (lane & 15) : (lane >> 4); }
  __device__ static int col8(int lane) { return MF ? (lane >> 4) : (lane & 15); }
};

template <int NW, bool MF>
__device__ __forceinline__ void load_unit(u32x4& dst, const GemvGeom& g, const GemvCursor& c, int lane, int op,
                                          int ra, const uint16_t* m0, const uint16_t* m1, const uint16_t* m2,
                                          int n0, int n1, const uint16_t* zero_page) {
  using US = UnitShape<MF>;
  const int seg = c.pt * g.SP + c.sg;
  const int wr = c.qd * US::rows + US::row(lane);
  const int k = g.k0 + seg * US::cols + US::col8(lane) * 8;
  const bool valid = c.live && seg < g.nseg && wr < g.nwr && k < g.kend;
  const uint16_t* ptr;
  if (NW == 2) {
    ptr = ((wr & 1) ? m1 : m0) + (size_t)(ra + (wr >> 1)) * g.K + k;
  } else {
    const int r = ra + wr;
    if (op == FM_OP_QKV) {
      ptr = (r >= n0 + n1) ? m2 + (size_t)(r - n0 - n1) * g.K + k
          : (r >= n0 ? m1 + (size_t)(r - n0) * g.K + k : m0 + (size_t)r * g.K + k);
    } else {
      ptr = m0 + (size_t)r * g.K + k;
    }
  }
  dst = ld_stream16(valid ? ptr : zero_page);
}

// Per-lane slot in the 64 KiB zero page (16 B per lane, spread over 4096 slots so idle lanes
// of different waves and workgroups do not all hit one cache line).
__device__ __forceinline__ const uint16_t* zero_slot(CParams& p, int wave, int lane) {
  return p.zero_page + ((((int)blockIdx.x * NWAVE + wave) * 64 + lane) & 4095) * 8;
}

// What a GEMV operator reads and writes: its matrices, input vector, norm and residual.
struct GemvOperand {
  int K = 0, rows = 0;              // columns and output rows of the operator's matrix
  int sidx = 0;                     // claim counter of its stage (dynamic chunks)
  const uint16_t* gain = nullptr;   // RMSNorm gain (norm prologue) or null
  bool from_embed = false;          // input is the embedding row (layer 0 QKV)
  u32 in_w = 0, in_stride = 0;      // tagged input: word offset of lane 0, words per lane
  u32 res_w = 0, res_stride = 0;    // tagged residual (OPROJ, DOWN)
  bool res_embed = false, has_res = false;
  const uint16_t* m0 = nullptr;     // matrices: QKV uses m0..m2 (W_q, W_k, W_v), GU m0, m1
  const uint16_t* m1 = nullptr;
  const uint16_t* m2 = nullptr;
  u64* out = nullptr;               // tagged output of lane 0 (not the LM head)
  u32 out_stride = 0;               // words per batch lane
};

__device__ __forceinline__ GemvOperand gemv_operand(CParams& p, int op, int l) {
  const int nq = p.nh * p.d, nk = p.nkv * p.d;
  CLayerPtrs* Lw = (op == FM_OP_LM) ? nullptr : (CLayerPtrs*)p.layers + l;
  GemvOperand o;
  switch (op) {
    case FM_OP_QKV:
      o.K = p.h; o.rows = nq + 2 * nk; o.sidx = 4 * l; o.gain = Lw->attn_norm;
      if (l == 0) o.from_embed = true; else { o.in_w = p.off_x + (u32)l * p.st_x; o.in_stride = p.h; }
      o.m0 = Lw->wq; o.m1 = Lw->wk; o.m2 = Lw->wv;
      o.out = p.act + p.off_qkv + (u32)l * p.st_qkv; o.out_stride = (u32)(nq + 2 * nk);
      break;
    case FM_OP_OPROJ:
      o.K = nq; o.rows = p.h; o.sidx = 4 * l + 1; o.in_w = p.off_o + (u32)l * p.st_o; o.in_stride = nq;
      o.has_res = true;
      if (l == 0) o.res_embed = true; else { o.res_w = p.off_x + (u32)l * p.st_x; o.res_stride = p.h; }
      o.m0 = Lw->wo;
      o.out = p.act + p.off_x1 + (u32)l * p.st_x1; o.out_stride = (u32)p.h;
      break;
    case FM_OP_GU:
      o.K = p.h; o.rows = p.inter; o.sidx = 4 * l + 2; o.gain = Lw->mlp_norm;
      o.in_w = p.off_x1 + (u32)l * p.st_x1; o.in_stride = p.h;
      o.m0 = Lw->wg; o.m1 = Lw->wu;
      o.out = p.act + p.off_m + (u32)l * p.st_m; o.out_stride = (u32)p.inter;
      break;
    case FM_OP_DOWN:
      o.K = p.inter; o.rows = p.h; o.sidx = 4 * l + 3; o.in_w = p.off_m + (u32)l * p.st_m; o.in_stride = p.inter;
      o.has_res = true; o.res_w = p.off_x1 + (u32)l * p.st_x1; o.res_stride = p.h;
      o.m0 = Lw->wd;
      o.out = p.act + p.off_x + (u32)(l + 1) * p.st_x; o.out_stride = (u32)p.h;
      break;
    default:  // FM_OP_LM
      o.K = p.h; o.rows = p.V; o.sidx = 4 * p.L; o.gain = p.final_norm;
      o.in_w = p.off_x + (u32)p.L * p.st_x; o.in_stride = p.h;
      o.m0 = p.lm_head;
      break;
  }
  return o;
}

// Clears the claim counters of the dynamic GEMV stages for the next step. Called by the
// workgroup that completes the step's LM head: every workgroup has made its last claim by
// then, since each stores its rows only after its last claim of the stage has returned.
__device__ __forceinline__ void reset_claims(CParams& p, int tid) {
  for (int k = tid; k < kPools * p.dyn_stride; k += NT)
    __hip_atomic_store(p.dyn_ctr + k, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// End of an LM-head instruction: the workgroup folds its lanes' packed keys (key[i], one per
// thread) into one per batch lane with an integer max, applies it to the step's maximum with
// an atomic max, and counts itself in. The workgroup that arrives last (all maxima performed)
// writes the greedy tokens and resets the step's counters.
template <int B>
__device__ __forceinline__ void lm_finish(CParams& p, const Step& st, const u64 (&key)[B], float* misc, int tid,
                                          int lane, int wave) {
  u64* wkeys = reinterpret_cast<u64*>(misc + 16);   // [NWAVE][B]
#pragma unroll
  for (int i = 0; i < B; ++i) {
    const u64 k = wave_max_u64(key[i]);
    if (lane == 0) wkeys[wave * B + i] = k;
  }
  __syncthreads();
  // One thread per batch lane folds the waves' keys into the step's maximum (all lanes'
  // atomics in flight together), and waits until its atomic has been performed.
  if (tid < p.b) {
    u64 k = 0;
    for (int w = 0; w < NWAVE; ++w) k = wkeys[w * B + tid] > k ? wkeys[w * B + tid] : k;
    if (k) __hip_atomic_fetch_max(p.amax + tid, k, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    vm_wait0();
  }
  __syncthreads();
  int* last = reinterpret_cast<int*>(misc + 8);
  if (tid == 0) {
    const u32 old = __hip_atomic_fetch_add(p.lm_arrive, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const int is_last = old == (u32)p.n_lm_instr - 1u ? 1 : 0;
    if (is_last) __hip_atomic_store(p.lm_arrive, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    *last = is_last;
  }
  __syncthreads();
  if (*last) {
    if (tid < p.b) {
      const u64 k = __hip_atomic_load(p.amax + tid, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      st.next_ids[tid] = (int32_t)(0xFFFFFFFFu - (u32)(k & 0xFFFFFFFFull));
      __hip_atomic_store(p.amax + tid, (u64)0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    reset_claims(p, tid);
  }
}

template <int B, int NW>
__device__ __forceinline__ bool op_gemv(CParams& p, const Step& st, const int32_t* ins, float* smem, int tid,
                                        int lane, int wave, tl_t* tl) {
  const int op = uni(ins[0]), l = uni(ins[1]), ra = uni(ins[2]), rb = uni(ins[3]);
  const int nr = rb - ra;
  const int nq = p.nh * p.d, nk = p.nkv * p.d;

  // Operator geometry.
  const GemvOperand opd = gemv_operand(p, op, l);
  const int K = opd.K;
  const uint16_t* gain = opd.gain;
  const bool from_embed = opd.from_embed, res_embed = opd.res_embed, has_res = opd.has_res;
  const u32 in_w = opd.in_w, in_stride = opd.in_stride, res_w = opd.res_w, res_stride = opd.res_stride;
  const uint16_t* m0 = opd.m0; const uint16_t* m1 = opd.m1; const uint16_t* m2 = opd.m2;
  const __amdgpu_buffer_rsrc_t ract = rsrc(p.act, p.act_bytes);

  // Geometry (all wave-uniform).
  GemvGeom g;
  g.K = K;
  constexpr bool MF = (B >= 8);           // matrix-core tiles for batch 8
  using US = UnitShape<MF>;
  constexpr int XSF = xslab_floats<B>();
  {
    const int Kpad = (K + 127) & ~127;
    // fp32 slab [B][Ks], or three bf16 planes [3][B][Ks + XPAD] (6 bytes per value) on the
    // matrix cores
    const int ks = (MF ? (XSF * 4) / (6 * B) - XPAD : XSF / B) & ~127;
    g.Ks = ks < Kpad ? ks : Kpad;
  }
  g.K = uni(K);
  g.Ks = uni(g.Ks);
  g.nslab = uni((K + g.Ks - 1) / g.Ks);
  g.nwr = uni(nr * NW);
  g.NQ = uni((g.nwr + US::rows - 1) / US::rows);
  auto set_slab = [&](int s) {
    g.k0 = uni(s * g.Ks);
    const int kn = min(g.Ks, K - g.k0);
    g.kend = uni(g.k0 + kn);
    g.nseg = uni((kn + US::cols - 1) / US::cols);
    if (s == 0) {
      // K parts: the fewest (1, 2, 4 or 8) that deal the (row group, part) items to the waves
      // within 3% of even, as far as the row sums fit in LDS. They are fixed for the whole
      // tile (every slab splits its columns the same way, so each item stays with one wave
      // and its row sums add up across slabs); a shorter last slab leaves some parts empty.
      int kp = 1;
      for (int c = 1; c <= 8; c *= 2) {
        if (c > g.nseg || c * nr * NW * B > rowacc_floats<B>()) break;
        kp = c;
        const int items = g.NQ * c, per = (items + NSW - 1) / NSW;
        if (per * NSW * 100 <= items * 103) break;
      }
      g.KP = uni(kp);
      g.nitems = uni(g.NQ * g.KP);
      g.items_w = uni((wave < NSW && g.nitems > wave) ? (g.nitems - wave + NSW - 1) / NSW : 0);
    }
    g.SP = uni((g.nseg + g.KP - 1) / g.KP);
  };
  set_slab(0);
  const int KP0 = g.KP;

  float* xs = smem;
  float* rowacc = smem + XSF;            // [KP][nr][NW][B]
  float* resid = rowacc + rowacc_floats<B>();
  float* misc = smem + LDS_FLOATS - MISC_FLOATS;
  const lds_i32* lin = lane_inputs(smem);            // this step's tokens at lin[0 .. b)

  // 1. Prefetch this wave's first U units, before waiting for the input.
  const uint16_t* zp = zero_slot(p, wave, lane);
  constexpr int U = FM_RING;
  u32x4 ring[U];
  GemvCursor ci;                          // issue cursor
  auto refill = [&](int sl) {
    load_unit<NW, MF>(ring[sl], g, ci, lane, op, ra, m0, m1, m2, nq, nk, zp);
    cursor_next(ci, g, wave);
  };
  auto prefill = [&]() {
    cursor_at(ci, g, 0, wave);
#pragma unroll
    for (int sl = 0; sl < U; ++sl) refill(sl);
  };
  // The first batch of input polls goes out before the weight prefetch: a wave's loads
  // return in issue order, so a poll issued behind the prefetch could not report a ready
  // input before the prefetch had landed.
  // (Not on the matrix-core tiles: their registers are taken by the planes' staging.)
  PairBatch<WBF> pre;
  const bool early = !MF && !from_embed && p.b > 0 && (NCTL == 0 || wave >= NSW) &&
                     min(g.Ks, K) <= (NCTL ? NCTL * 64 : NT) * 2 * WBF;
  if constexpr (!MF)
    if (early)
      issue_pairs<WBF>(ract, in_w, min(g.Ks, K), gain ? reinterpret_cast<const u32*>(gain) : nullptr,
                       (NCTL ? tid - NSW * 64 : tid) * 2, NCTL ? NCTL * 64 : NT, pre);
  prefill();

  // 2. Input: wait for the producers, then stage x * g (x times its RMSNorm gain, if any) in
  //    LDS: fp32 for VALU tiles; three bf16 planes for matrix-core tiles (hi + mid + lo =
  //    x * g to about 2^-24 relative). The norm's 1/rms is applied to the finished rows in the
  //    epilogue: the sum of squares is gathered while staging, and no pass over the slab is
  //    needed once it is known.
  bool ok = true;
  float rs[B];
#pragma unroll
  for (int i = 0; i < B; ++i) rs[i] = 1.0f;
  // Inputs are polled and staged by the control waves (ct = thread index among them).
  const bool ctl = (NCTL == 0) || wave >= NSW;
  const int ct = NCTL ? tid - NSW * 64 : tid, nct = NCTL ? NCTL * 64 : NT;
  uint16_t* planes = reinterpret_cast<uint16_t*>(xs);   // matrix-core tiles: [3][B][Ks]
  // Matrix-core planes: rows of Ks + XPAD values, so the batch rows that one 8-lane group reads
  // for a B operand (same columns, consecutive rows) start 16 bytes apart and fall in
  // different LDS banks (with rows of Ks values, a multiple of 128, they all shared banks).
  const int RS = MF ? g.Ks + XPAD : g.Ks;                // values per plane row
  const int pst = B * RS;                               // values per plane
  auto put_pair = [&](int i, int k, float a, float b) {
    if constexpr (MF) {
      const uint16_t h0 = to_bf16(a), h1 = to_bf16(b);
      a -= __uint_as_float((u32)h0 << 16);
      b -= __uint_as_float((u32)h1 << 16);
      const uint16_t m0_ = to_bf16(a), m1_ = to_bf16(b);
      a -= __uint_as_float((u32)m0_ << 16);
      b -= __uint_as_float((u32)m1_ << 16);
      const uint16_t l0 = to_bf16(a), l1 = to_bf16(b);
      u32* q = reinterpret_cast<u32*>(planes + i * RS + k);
      q[0] = (u32)h0 | ((u32)h1 << 16);
      q[pst / 2] = (u32)m0_ | ((u32)m1_ << 16);
      q[pst] = (u32)l0 | ((u32)l1 << 16);
    } else {
      xs[i * g.Ks + k] = a;
      xs[i * g.Ks + k + 1] = b;
    }
  };
  float* mss = misc + 512;                              // [NWAVE][B] partial sums of squares
  auto stage = [&](int s) -> bool {
    const int k0 = s * g.Ks, kn = min(g.Ks, K - k0);
    const int kfill = (kn + US::cols - 1) & ~(US::cols - 1);
    // zeros: the padding columns of every lane, every column of absent batch lanes
#pragma unroll
    for (int i = 0; i < B; ++i) {
      for (int k = (i >= p.b ? 0 : kn) + tid * 2; k < kfill; k += NT * 2) put_pair(i, k, 0.f, 0.f);
    }
    if (!ctl) return true;
    const u32* gsl = gain ? reinterpret_cast<const u32*>(gain + k0) : nullptr;
#pragma unroll
    for (int i = 0; i < B; ++i) {
      if (i >= p.b) continue;
      float ss = 0.f;
      auto use = [&](int k, float a, float b, u32 g2) {
        ss += a * a + b * b;
        if (gsl) { a *= bf16lo(g2); b *= bf16hi(g2); }
        put_pair(i, k, a, b);
      };
      if (from_embed) {
        const uint16_t* e = p.embed + (size_t)lin[i] * p.h + k0;
        for (int k = ct * 2; k < kn; k += nct * 2) {
          const u32 w2 = *reinterpret_cast<const u32*>(e + k);
          use(k, bf16lo(w2), bf16hi(w2), gsl ? gsl[k >> 1] : 0u);
        }
      } else {
        if (!wait_pairs<WBC>(p, st, ract, in_w + (u32)i * in_stride + (u32)k0, kn, gsl, use, ct, nct,
                             (!MF && s == 0 && i == 0 && early) ? &pre : nullptr))
          return false;
      }
      if (gain) {
        // Sum of squares so far: one partial per wave and lane in LDS (the stream keeps no
        // registers for it).
        const float wsum = wave_sum(ss);
        if (lane == 0) mss[wave * B + i] = (s == 0 ? 0.f : mss[wave * B + i]) + wsum;
      }
    }
    return true;
  };

  ok = stage(0);
  // Residual rows for the epilogue.
  if (ok && has_res && ctl) {
    for (int i = 0; i < B && ok; ++i) {
      if (i >= p.b) continue;
      if (res_embed) {
        const uint16_t* e = p.embed + (size_t)lin[i] * p.h;
        for (int k = ct; k < nr; k += nct) resid[i * nr + k] = __uint_as_float((u32)e[ra + k] << 16);
      } else {
        const int lo = ra & ~1, hi = (rb + 1) & ~1;
        for (int k = lo + ct * 2; k < hi; k += nct * 2) {
          float a, b;
          if (!wait_pair(p, st, ract, res_w + (u32)i * res_stride + (u32)k, a, b)) { ok = false; break; }
          if (k >= ra && k < rb) resid[i * nr + (k - ra)] = a;
          if (k + 1 >= ra && k + 1 < rb) resid[i * nr + (k + 1 - ra)] = b;
        }
      }
    }
  }
  if (__syncthreads_or(!ok)) return false;
  if (tl && tid == 0) { tl[1] = clock_now(); tl[2] = tl[1]; }

  // 3. Stream the weights: consume the ring in order, refilling each slot as it is used.
  for (int s = 0; s < g.nslab; ++s) {
    if (s > 0) {
      __syncthreads();
      if (!stage(s)) ok = false;
      if (__syncthreads_or(!ok)) return false;
      set_slab(s);
      prefill();
    }
    const int units = uni(g.items_w * g.SP);
    GemvCursor cc;                        // consume cursor
    cursor_at(cc, g, 0, wave);
    float acc[B];
#pragma unroll
    for (int i = 0; i < B; ++i) acc[i] = 0.f;
    f32x4 acc4 = {0.f, 0.f, 0.f, 0.f};     // matrix-core tiles: C rows 4 (lane / 16) + r, column lane % 16
    // Each round consumes the U slots in order and refills each one after its use (the refill
    // then lands in the same registers; issued before the use, it would need other registers
    // and a copy back that waits for it). Refills are unconditional (see load_unit), except
    // that the last round only drains the ring: a refill there would load nothing the tile
    // needs, and the epilogue, which reuses the ring's registers, would wait for it to land.
    // (Refilling only the units that exist in the round before costs more: the compiler then
    // drains the ring at every wait.)
    auto consume = [&](const u32x4 w) {
      const int seg = cc.pt * g.SP + cc.sg;
      // Units past the slab's segments (the last K part may be short) were never loaded
      // and contribute nothing.
      if constexpr (MF) {
        if (seg < g.nseg) {
          const int j = lane & 15;
          const int kk = seg * 32 + (lane >> 4) * 8;      // this lane's 8-column block
          bf16x8 xh = {}, xm = {}, xl = {};
          if (j < B) {
            const uint16_t* pl = planes + j * RS + kk;
            xh = *reinterpret_cast<const bf16x8*>(pl);
            xm = *reinterpret_cast<const bf16x8*>(pl + pst);
            xl = *reinterpret_cast<const bf16x8*>(pl + 2 * pst);
          }
          const bf16x8 wa = __builtin_bit_cast(bf16x8, w);
          acc4 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wa, xl, acc4, 0, 0, 0);
          acc4 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wa, xm, acc4, 0, 0, 0);
          acc4 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wa, xh, acc4, 0, 0, 0);
        }
      } else if (seg < g.nseg) {
        const int kk = seg * 128 + (lane & 15) * 8;   // column within the slab
        const float w0 = bf16lo(w.x), w1 = bf16hi(w.x), w2 = bf16lo(w.y), w3 = bf16hi(w.y);
        const float w4 = bf16lo(w.z), w5 = bf16hi(w.z), w6 = bf16lo(w.w), w7 = bf16hi(w.w);
#pragma unroll
        for (int i = 0; i < B; ++i) {
          const float4 xa = *reinterpret_cast<const float4*>(xs + i * g.Ks + kk);
          const float4 xb = *reinterpret_cast<const float4*>(xs + i * g.Ks + kk + 4);
          float t0 = w0 * xa.x, t1 = w1 * xa.y;
          t0 = fmaf(w2, xa.z, t0); t1 = fmaf(w3, xa.w, t1);
          t0 = fmaf(w4, xb.x, t0); t1 = fmaf(w5, xb.y, t1);
          t0 = fmaf(w6, xb.z, t0); t1 = fmaf(w7, xb.w, t1);
          acc[i] += t0 + t1;
        }
      }
      if (cc.sg == g.SP - 1) {
        // Item finished: store the part sums (added to earlier slabs' sums).
        if constexpr (MF) {
          const int j = lane & 15;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int wr = cc.qd * 16 + 4 * (lane >> 4) + r;
            if (j < B && wr < g.nwr) {
              float* dst = rowacc + ((cc.pt * nr) * NW + wr) * B + j;
              *dst = (s == 0) ? acc4[r] : *dst + acc4[r];
            }
          }
          acc4 = f32x4{0.f, 0.f, 0.f, 0.f};
        } else {
          // Each 16-lane row sums its weight row; its first lane stores the part sum.
          const int wr = cc.qd * 4 + (lane >> 4);
          const bool writer = (lane & 15) == 0 && wr < g.nwr;
#pragma unroll
          for (int i = 0; i < B; ++i) {
            const float v = row16_sum(acc[i]);
            acc[i] = 0.f;
            if (writer) {
              float* dst = rowacc + ((cc.pt * nr) * NW + wr) * B + i;
              *dst = (s == 0) ? v : *dst + v;
            }
          }
        }
      }
      cursor_next(cc, g, wave);
    };
    int base = 0;
    for (; base + U < units; base += U) {
#pragma unroll
      for (int sl = 0; sl < U; ++sl) {
        consume(ring[sl]);
        refill(sl);
      }
    }
#pragma unroll
    for (int sl = 0; sl < U; ++sl)
      if (base + sl < units) consume(ring[sl]);
  }
  __syncthreads();
  if (tl && tid == 0) tl[3] = clock_now();
  if (gain) {
    // The norm's 1/rms, now that every slab has been seen, and the normalised input tap
    // (re-read from the input words, still current this step).
#pragma unroll
    for (int i = 0; i < B; ++i) {
      float t = 0.f;
      // only the waves that staged the input hold partial sums (all waves unless NCTL > 0)
      for (int w = NCTL ? NSW : 0; w < NWAVE; ++w) t += mss[w * B + i];
      rs[i] = 1.0f / sqrtf(t / (float)K + p.eps);
    }
    if (st.taps && ra == 0) {
      const int off = (op == FM_OP_QKV) ? p.tap_a : (op == FM_OP_GU ? p.tap_a2 : 0);
#pragma unroll
      for (int i = 0; i < B; ++i) {
        if (i >= p.b) continue;
        float* t = (op == FM_OP_LM)
                       ? st.taps + (size_t)p.L * p.b * p.tap_block + (size_t)i * p.h
                       : st.taps + ((size_t)l * p.b + i) * p.tap_block + off;
        for (int k = tid; k < K; k += NT) {
          const float x = from_embed
              ? __uint_as_float((u32)p.embed[(size_t)lin[i] * p.h + k] << 16)
              : __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(ract, (in_w + (u32)i * in_stride + (u32)k) * 8u,
                                                                      0, CPOL_SC1));
          t[k] = x * rs[i] * __uint_as_float((u32)gain[k] << 16);
        }
      }
    }
  }

  // 4. Epilogue, one output row per thread: K-part sums in order, residual adds, SiLU * up,
  //    tagged stores, taps, logits; the LM head also folds its rows into one packed argmax
  //    key per lane. The output's address was resolved with the operator, so nothing here
  //    waits on parameter loads.
  u64 key[B];
#pragma unroll
  for (int i = 0; i < B; ++i) key[i] = 0;
  u64* const out = opd.out;
  const u32 ost = opd.out_stride, epoch = st.epoch;
  for (int rl = tid; rl < nr; rl += NT) {
    const int r = ra + rl;
#pragma unroll
    for (int i = 0; i < B; ++i) {
      if (i >= p.b) break;
      float y = 0.f, up = 0.f;
      for (int pt = 0; pt < KP0; ++pt) {
        y += rowacc[((pt * nr + rl) * NW) * B + i];
        if (NW == 2) up += rowacc[((pt * nr + rl) * NW + 1) * B + i];
      }
      if (gain) {
        y *= rs[i];
        up *= rs[i];
      }
      switch (op) {
        case FM_OP_QKV:
          st_tag(out + (u32)i * ost + r, y, epoch);
          if (st.taps) st.taps[((size_t)l * p.b + i) * p.tap_block + p.tap_qkv + r] = y;
          break;
        case FM_OP_OPROJ: {
          const float x1 = y + resid[i * nr + rl];
          st_tag(out + (u32)i * ost + r, x1, epoch);
          if (st.taps) st.taps[((size_t)l * p.b + i) * p.tap_block + p.tap_x1 + r] = x1;
          break;
        }
        case FM_OP_GU:
          st_tag(out + (u32)i * ost + r, silu(y) * up, epoch);
          break;
        case FM_OP_DOWN: {
          const float xr = y + resid[i * nr + rl];
          st_tag(out + (u32)i * ost + r, xr, epoch);
          if (st.taps) {
            st.taps[((size_t)l * p.b + i) * p.tap_block + p.tap_mlp + r] = y;
            st.taps[((size_t)l * p.b + i) * p.tap_block + p.tap_x2 + r] = xr;
          }
          break;
        }
        default: {
          if (st.logits) __builtin_nontemporal_store(y, st.logits + (size_t)i * p.V + r);
          // Packed key: order-preserving float bits, then the complemented row index, so
          // the integer maximum picks the largest logit and, among equal ones, the lowest row.
          const u64 k = ((u64)ordered(y) << 32) | (u64)(0xFFFFFFFFu - (u32)r);
          key[i] = k > key[i] ? k : key[i];
          break;
        }
      }
    }
  }

  // 5. LM head: one packed key per lane per tile via an integer max (order-independent),
  //    then the last LM tile of the step writes the greedy tokens.
  if (op == FM_OP_LM) lm_finish<B>(p, st, key, misc, tid, lane, wave);
  __syncthreads();   // LDS is reused by the next instruction
  return true;
}

// ---- GEMV stage in dynamic chunks (VALU tiles, B <= 2) -----------------------------------
//
// With one fixed tile per workgroup a stage ends when its slowest tile does, and which tiles
// stream slowly changes from stage to stage. Large VALU stages of the QKV, O-projection and
// down operators are therefore cut into chunks of Rc output rows, grouped into pools: workgroup w serves pool w mod 8 (on MI355X, the
// workgroups that share one XCD's L2). Each workgroup takes one chunk of its pool's range as
// its own; the range's other chunks go to the pool's workgroups as they ask for them, through
// one atomic counter per (stage, pool), so a workgroup that runs late takes fewer chunks.
// Every chunk is computed the same way whoever takes it (same K split, same order of sums),
// so the results do not depend on the assignment.
//
// A chunk is Rc = 4 * 8 / KP rows split into KP parts along K: exactly one (row quad,
// K part) item per wave, the same one in every chunk, SP segments of 128 columns long. A wave
// thus streams SP units per chunk through one register ring, with no barrier between chunks:
// the chunk ids sit in an LDS list that wave 0 fills. Wave 0 claims the next chunk during the
// last ring rounds of the current one (at a round start, publishing the answer at the next
// round start, when the claim is older than the ring's U loads in flight and the publication
// does not wait). Row part sums stay in LDS per chunk; the epilogue writes all of the
// workgroup's rows once its last chunk is done, after its last claim has returned.

typedef __attribute__((address_space(3))) volatile int lds_int;

template <int B>
__device__ __forceinline__ bool op_gemv_dyn(CParams& p, const Step& st, const int32_t* ins, float* smem, int tid,
                                            int lane, int wave, tl_t* tl) {
  static_assert(B <= 2 && NCTL == 0, "dynamic chunks run VALU tiles streamed by every wave");
  constexpr int U = FM_RING;
  constexpr int UNKNOWN = -2, END = -1;
  const int op = uni(ins[0]), l = uni(ins[1]);
  const int Rc = uni(-ins[2]), KP = uni(ins[3] & 0xff), nslot = uni(ins[3] >> 8);
  const int nq = p.nh * p.d, nk = p.nkv * p.d;
  const GemvOperand o = gemv_operand(p, op, l);
  const int K = o.K, R = o.rows;
  const int Kpad = uni((K + 127) & ~127), nseg = uni(Kpad / 128);
  const int NQ = uni(NWAVE / KP), nwr = uni(4 * NQ);
  const int SP = uni((nseg + KP - 1) / KP);
  // This wave's item in every chunk: row quad qd, K part pt; sp_ok of its SP segments lie
  // inside the matrix.
  const int qd = uni(wave / KP), pt = uni(wave - (wave / KP) * KP);
  const int sp_ok = uni(max(0, min(SP, nseg - pt * SP)));

  float* xs = smem;                                  // [B][Kpad] input times its gain
  float* rowacc = smem + xslab_floats<B>();          // [nslot][KP][nwr][B] row part sums
  float* misc = smem + LDS_FLOATS - MISC_FLOATS;
  float* mss = misc + 512;                           // [NWAVE][B] partial sums of squares
  const lds_i32* lin = lane_inputs(smem);            // this step's tokens at lin[0 .. b)
  lds_int* chl = (lds_int*)(__attribute__((address_space(3))) int*)(misc + 256);   // [nslot + 1] chunk ids

  // The schedule guarantees these; a violation would overrun LDS, so it stops the step.
  if (!(op == FM_OP_QKV || op == FM_OP_OPROJ || op == FM_OP_DOWN) || nslot < 2 || nslot > 254 ||
      !(KP == 1 || KP == 2 || KP == 4 || KP == 8) || Rc != nwr || SP < U ||
      B * Kpad > xslab_floats<B>() || nslot * KP * nwr * B > rowacc_floats<B>()) {
    if (tid == 0) raise_error(p, FM_DEV_BAD_PLAN);
    return false;
  }

  // This workgroup's pool, its own chunk and the pool's shared range.
  const int nwg = p.nwg, np = min(kPools, nwg), wg = (int)blockIdx.x;
  const int px = wg % np, kx = wg / np;
  const int nwx = (nwg - px + np - 1) / np;
  const int sx = px * (nwg / np) + min(px, nwg % np);
  const int nch = (R + Rc - 1) / Rc;
  const int c0 = (int)((long long)nch * sx / nwg), c1 = (int)((long long)nch * (sx + nwx) / nwg);
  const int own = uni(c0 + kx), dyn0 = uni(c0 + nwx), ndyn = uni(c1 - c0 - nwx);
  u32* ctr = p.dyn_ctr + px * p.dyn_stride + o.sidx;
  if (tid == 0) {
    chl[0] = own;
    for (int j = 1; j <= nslot; ++j) chl[j] = (j == nslot || ndyn == 0) ? END : UNKNOWN;
  }

  // Per lane: weight row wr of the chunk (16 lanes per row), first column kl of its part, and
  // how many of the part's segments hold columns of this lane inside K.
  const int wr = qd * 4 + (lane >> 4);
  const int kl = pt * SP * 128 + (lane & 15) * 8;
  const int seg_ok = max(0, min(sp_ok, (K - kl + 127) / 128));
  const uint16_t* zp = zero_slot(p, wave, lane);
  // Row pointer of chunk c for this lane (at column kl), and its count of loadable segments.
  auto chunk_row = [&](int c, const uint16_t*& rp, int& lim) {
    const int r = c * Rc + wr;
    const uint16_t* m;
    int rr = r;
    if (op == FM_OP_QKV) {
      m = r >= nq + nk ? o.m2 : (r >= nq ? o.m1 : o.m0);
      rr = r >= nq + nk ? r - nq - nk : (r >= nq ? r - nq : r);
    } else {
      m = o.m0;
    }
    const bool live = r < R;
    rp = live ? m + (size_t)rr * K + kl : zp;
    lim = live ? seg_ok : 0;
  };

  // Claims (wave 0; lane 0 holds the counter's answer). The next slot is claimed at a round
  // start once the issue cursor is within 2U units of its chunk's end.
  const int claim_from = uni(max(0, SP - 2 * U));
  int pend_slot = -1, claimed = 0;
  bool exhausted = ndyn == 0;
  u32 pend = 0;
  auto publish = [&]() {
    const u32 v = (u32)uni((int)pend);
    const int ch = v < (u32)ndyn ? dyn0 + (int)v : END;
    if (lane == 0) chl[pend_slot] = ch;
    if (ch < 0) exhausted = true;
    pend_slot = -1;
  };

  // Issue cursor: slot i_j, segment i_sg; the lane's row pointer and loadable segments.
  int i_j = 0, i_sg = 0;
  bool i_live = true;
  const uint16_t* i_rp;
  int i_lim;
  chunk_row(own, i_rp, i_lim);
  auto issue = [&](u32x4& dst) {
    dst = ld_stream16(i_sg < i_lim ? i_rp + i_sg * 128 : zp);
    i_sg = uni(i_sg + 1);
    if (i_sg == SP && i_live) {
      // Next slot: wait (on LDS) until its chunk id is known.
      i_sg = 0;
      i_j = uni(i_j + 1);
      if (wave == 0 && pend_slot == i_j) publish();   // wave 0 caught up with its own claim
      int v = uni(chl[i_j]);
      if (v == UNKNOWN) {
        const u64 t0 = clock_now();
        while (true) {
          __builtin_amdgcn_s_sleep(1);
          v = uni(chl[i_j]);
          if (v != UNKNOWN) break;
          if (clock_now() - t0 > WAIT_TICKS) {
            raise_error(p, FM_DEV_WATCHDOG);
            v = END;
            break;
          }
        }
      }
      if (v < 0) {
        i_live = false;
        i_lim = 0;
      } else {
        chunk_row(v, i_rp, i_lim);
      }
    }
  };

  // 1. The first batch of input polls (before the prefetch: loads return in issue order),
  //    then U units of the own chunk (SP >= U), then the claim of the second chunk (the
  //    ring's first round start comes too late in the own chunk).
  const __amdgpu_buffer_rsrc_t ract = rsrc(p.act, p.act_bytes);
  const u32* gsl = o.gain ? reinterpret_cast<const u32*>(o.gain) : nullptr;
  PairBatch<WBF> pre;
  const bool early = !o.from_embed && p.b > 0 && K <= NT * 2 * WBF;
  if (early) issue_pairs<WBF>(ract, o.in_w, K, gsl, tid * 2, NT, pre);
  u32x4 ring[U];
#pragma unroll
  for (int sl = 0; sl < U; ++sl) issue(ring[sl]);
  if (wave == 0 && !exhausted) {
    if (lane == 0) pend = __hip_atomic_fetch_add(ctr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    pend_slot = 1;
    claimed = 1;
  }

  // 2. Stage the input times its gain (sum of squares on the side).
  bool ok = true;
  float rs[B];
#pragma unroll
  for (int i = 0; i < B; ++i) {
    rs[i] = 1.0f;
    for (int k = (i >= p.b ? 0 : K) + tid; k < Kpad; k += NT) xs[i * Kpad + k] = 0.f;
  }
#pragma unroll
  for (int i = 0; i < B; ++i) {
    if (i >= p.b || !ok) continue;
    float ss = 0.f;
    auto use = [&](int k, float a, float b, u32 g2) {
      ss += a * a + b * b;
      if (gsl) { a *= bf16lo(g2); b *= bf16hi(g2); }
      xs[i * Kpad + k] = a;
      xs[i * Kpad + k + 1] = b;
    };
    if (o.from_embed) {
      const uint16_t* e = p.embed + (size_t)lin[i] * p.h;
      for (int k = tid * 2; k < K; k += NT * 2) {
        const u32 w2 = *reinterpret_cast<const u32*>(e + k);
        use(k, bf16lo(w2), bf16hi(w2), gsl ? gsl[k >> 1] : 0u);
      }
    } else if (B == 1 && K > NT * 2 * WBC && K <= NT * 2 * WBL) {
      if constexpr (B == 1)
        if (!wait_pairs<WBL>(p, st, ract, o.in_w + (u32)i * o.in_stride, K, gsl, use, tid, NT)) ok = false;
    } else if (!wait_pairs<WBC>(p, st, ract, o.in_w + (u32)i * o.in_stride, K, gsl, use, tid, NT,
                                (i == 0 && early) ? &pre : nullptr)) {
      ok = false;
    }
    if (o.gain) {
      const float wsum = wave_sum(ss);
      if (lane == 0) mss[wave * B + i] = wsum;
    }
  }
  // The second chunk's claim was issued before the polls above, which have all returned.
  if (wave == 0 && pend_slot >= 0) publish();
  if (__syncthreads_or(!ok)) return false;
  if (tl && tid == 0) { tl[1] = clock_now(); tl[2] = tl[1]; }

  // 3. Stream every chunk the workgroup takes. Each round consumes the U slots in order and
  //    refills each after its use; past the last chunk the refills read the zero page.
  int c_j = 0, c_sg = 0;
  bool c_live = true;
  float acc[B];
#pragma unroll
  for (int i = 0; i < B; ++i) acc[i] = 0.f;
  const int kx0 = pt * SP * 128 + (lane & 15) * 8;   // LDS column of segment 0
  auto consume = [&](const u32x4 w) {
    if (!c_live) return;
    if (c_sg < sp_ok) {
      const int kk = kx0 + c_sg * 128;
      const float w0 = bf16lo(w.x), w1 = bf16hi(w.x), w2 = bf16lo(w.y), w3 = bf16hi(w.y);
      const float w4 = bf16lo(w.z), w5 = bf16hi(w.z), w6 = bf16lo(w.w), w7 = bf16hi(w.w);
#pragma unroll
      for (int i = 0; i < B; ++i) {
        const float4 xa = *reinterpret_cast<const float4*>(xs + i * Kpad + kk);
        const float4 xb = *reinterpret_cast<const float4*>(xs + i * Kpad + kk + 4);
        float t0 = w0 * xa.x, t1 = w1 * xa.y;
        t0 = fmaf(w2, xa.z, t0); t1 = fmaf(w3, xa.w, t1);
        t0 = fmaf(w4, xb.x, t0); t1 = fmaf(w5, xb.y, t1);
        t0 = fmaf(w6, xb.z, t0); t1 = fmaf(w7, xb.w, t1);
        acc[i] += t0 + t1;
      }
    }
    c_sg = uni(c_sg + 1);
    if (c_sg == SP) {
      // Item done: each 16-lane row sums its weight row; its first lane stores the part.
#pragma unroll
      for (int i = 0; i < B; ++i) {
        const float v = row16_sum(acc[i]);
        acc[i] = 0.f;
        if ((lane & 15) == 0) rowacc[((c_j * KP + pt) * nwr + wr) * B + i] = v;
      }
      c_sg = 0;
      c_j = uni(c_j + 1);
      // the issue cursor passed this boundary U units ago, so the id is published
      if (uni(chl[c_j]) < 0) c_live = false;
    }
  };
  while (c_live) {
    if (wave == 0) {
      if (pend_slot >= 0) publish();
      if (!exhausted && i_live && i_sg >= claim_from && claimed <= i_j && i_j + 1 < nslot) {
        if (lane == 0) pend = __hip_atomic_fetch_add(ctr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        pend_slot = i_j + 1;
        claimed = i_j + 1;
      }
    }
#pragma unroll
    for (int sl = 0; sl < U; ++sl) {
      consume(ring[sl]);
      issue(ring[sl]);
    }
  }
  // The ring's last refills (zero-page reads) are still in flight: let them land here, before
  // the epilogue's stores, so that no load is pending on a register the next instruction
  // writes (the compiler would wait for it there, behind these stores' acknowledgements).
  __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0)
  __syncthreads();
  if (tl && tid == 0) tl[3] = clock_now();
  // Every wave walked the same slots: the consume cursor stopped at the first empty one.
  const int nused = c_j;
  if (tl && tid == 0) tl[6] = (u64)nused;

  if (o.gain) {
#pragma unroll
    for (int i = 0; i < B; ++i) {
      float t = 0.f;
      for (int w = 0; w < NWAVE; ++w) t += mss[w * B + i];
      rs[i] = 1.0f / sqrtf(t / (float)K + p.eps);
    }
    if (st.taps && wg == 0) {
      const int off = (op == FM_OP_QKV) ? p.tap_a : (op == FM_OP_GU ? p.tap_a2 : 0);
#pragma unroll
      for (int i = 0; i < B; ++i) {
        if (i >= p.b) continue;
        float* t = (op == FM_OP_LM)
                       ? st.taps + (size_t)p.L * p.b * p.tap_block + (size_t)i * p.h
                       : st.taps + ((size_t)l * p.b + i) * p.tap_block + off;
        for (int k = tid; k < K; k += NT) {
          const float x = o.from_embed
              ? __uint_as_float((u32)p.embed[(size_t)lin[i] * p.h + k] << 16)
              : __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(ract, (o.in_w + (u32)i * o.in_stride + (u32)k) * 8u,
                                                                      0, CPOL_SC1));
          t[k] = x * rs[i] * __uint_as_float((u32)o.gain[k] << 16);
        }
      }
    }
  }

  // 4. Epilogue over the workgroup's rows (chunk slot j, row rl): K-part sums in order,
  //    residual adds (the residual word is read here, produced two stages ago), tagged
  //    stores and taps.
  u64* const out = o.out;
  const u32 ost = o.out_stride, epoch = st.epoch;
  for (int u = tid; u < nused * Rc && ok; u += NT) {
    const int j = u / Rc, rl = u - j * Rc;
    const int r = chl[j] * Rc + rl;
    if (r >= R) continue;
#pragma unroll
    for (int i = 0; i < B; ++i) {
      if (i >= p.b) break;
      float y = 0.f;
      for (int q = 0; q < KP; ++q) y += rowacc[((j * KP + q) * nwr + rl) * B + i];
      if (o.gain) y *= rs[i];
      float res = 0.f;
      if (o.has_res) {
        if (o.res_embed) {
          res = __uint_as_float((u32)p.embed[(size_t)lin[i] * p.h + r] << 16);
        } else {
          float ra_, rb_;
          if (!wait_pair(p, st, ract, o.res_w + (u32)i * o.res_stride + (u32)(r & ~1), ra_, rb_)) { ok = false; break; }
          res = (r & 1) ? rb_ : ra_;
        }
      }
      switch (op) {
        case FM_OP_QKV:
          st_tag(out + (u32)i * ost + r, y, epoch);
          if (st.taps) st.taps[((size_t)l * p.b + i) * p.tap_block + p.tap_qkv + r] = y;
          break;
        case FM_OP_OPROJ: {
          const float x1 = y + res;
          st_tag(out + (u32)i * ost + r, x1, epoch);
          if (st.taps) st.taps[((size_t)l * p.b + i) * p.tap_block + p.tap_x1 + r] = x1;
          break;
        }
        default: {  // FM_OP_DOWN
          const float xr = y + res;
          st_tag(out + (u32)i * ost + r, xr, epoch);
          if (st.taps) {
            st.taps[((size_t)l * p.b + i) * p.tap_block + p.tap_mlp + r] = y;
            st.taps[((size_t)l * p.b + i) * p.tap_block + p.tap_x2 + r] = xr;
          }
          break;
        }
      }
    }
  }
  if (__syncthreads_or(!ok)) return false;   // also: LDS is reused by the next instruction
  return true;
}

// ---- attention work items ---------------------------------------------------------------
//
// Per layer the step has P work items. At run time item j maps, from kv_lens alone, to a
// lane i, a KV head g and a chunk [t0, t1) of that lane's slots 0..kv_len: every
// (lane, KV head) gets ceil((kv_len+1)/T) chunks of at most T slots. T is the smallest
// multiple of an item's pass width (the slots all waves cover at once) for which the chunks
// fit in P, so ragged lanes are balanced per step and no pass runs mostly empty.
// An item reads its group's raw q (G heads), k and v and applies QK-norm and RoPE. The item
// holding the group's last chunk also rounds the new k/v to bf16 and appends them at slot
// kv_len. Each item runs a softmax over its slots (Eq. 1; base-2 exponent with
// log2(e)/sqrt(d) folded into q) a block of passes at a time: scores first, then a running
// maximum shared by the wave, then exponentials and weighted V sums. It yields one partial
// (max, sum, weighted V) per head. Lanes: LPS = d/8 lanes per slot, 8 dims (16 B of K and
// of V) per lane, so a wave covers 64/LPS slots per pass and the K/V loads are contiguous.
// The group's heads are merged by its last M = min(G, nc, workgroups) chunk items: the item
// of chunk c = nc - 1 - r merges heads r, r + M, r + 2M, ... Every item publishes its partials
// of the heads it does not merge as tagged words; a merger combines the other chunks' partials
// of its heads with its own in chunk order (log-sum-exp), so the result does not depend on M,
// and writes those heads' attention output. A merger waits for items at most M - 1 indices
// after its own, and an item can only be held up by items at least one queue length (the
// workgroup count) before it in its workgroup's queue, so with M at most the workgroup count
// no chain of waits can close on itself.

// Chunk length of this step (see above); spp is the pass width.
// gran (<= spp) is the work granularity of one wave: chunks shorter than half a pass are
// rounded to it instead (short contexts then keep many items, each on a few waves). tmin is
// the shortest chunk worth its share of the merge.
__device__ __forceinline__ int chunk_len(CParams& p, const lds_i32* kvls, int spp, int gran, int tmin) {
  long long total = 0;
  for (int ii = 0; ii < p.b; ++ii) total += kvls[ii] + 1;
  total *= p.nkv;
  const long long denom = p.P - p.nkv * p.b;
  const int T0 = (int)((total + denom - 1) / denom);
  const int q = (2 * T0 <= spp) ? gran : spp;
  return max(((T0 + q - 1) / q) * q, tmin);
}

__device__ __forceinline__ bool item_map(CParams& p, const lds_i32* kvls, int j, int spp, int gran, int tmin, int& i,
                                         int& g, int& c, int& nc, int& t0, int& t1) {
  const int T = chunk_len(p, kvls, spp, gran, tmin);
  int idx = j;
  for (int ii = 0; ii < p.b; ++ii) {
    const int W = kvls[ii] + 1;
    const int n = (W + T - 1) / T;
    const int per = p.nkv * n;
    if (idx < per) {
      i = ii; g = idx / n; c = idx % n; nc = n;
      t0 = c * T; t1 = min(t0 + T, W);
      return true;
    }
    idx -= per;
  }
  return false;
}

// Makes the eight values computed before any later memory access: a ring slot's data are
// converted before its refill is issued, so the refill can reuse the slot's registers (a
// refill hoisted above the conversion would need fresh ones, and copies back, each waiting
// for its load, at the end of every loop iteration).
__device__ __forceinline__ void order_before_load(float (&x)[8]) {
  asm volatile("" : "+v"(x[0]), "+v"(x[1]), "+v"(x[2]), "+v"(x[3]), "+v"(x[4]), "+v"(x[5]), "+v"(x[6]), "+v"(x[7])
               :: "memory");
}

// Sum within each 8-lane half-row; every lane of it gets the total (DPP).
__device__ __forceinline__ float row8_sum(float s) {
  s += dpp_row<DPP_QUAD_1032>(s);
  s += dpp_row<DPP_QUAD_2301>(s);
  s += dpp_row<DPP_HALF_MIRROR>(s);
  return s;
}

// Value of lane (lane xor 8), (lane xor 16), (lane xor 32), in the VALU.
__device__ __forceinline__ float lane_xor8(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x128, 0xF, 0xF, false));  // row rotate 8
}
__device__ __forceinline__ float lane_xor16(float v, int lane) { return __uint_as_float(xor16_u32(__float_as_uint(v), lane)); }
__device__ __forceinline__ float lane_xor32(float v, int lane) { return __uint_as_float(xor32_u32(__float_as_uint(v), lane)); }
template <int O>
__device__ __forceinline__ float lane_xor(float v, int lane) {
  static_assert(O == 8 || O == 16 || O == 32, "exchange distance");
  return O == 8 ? lane_xor8(v) : (O == 16 ? lane_xor16(v, lane) : lane_xor32(v, lane));
}

// Maximum over the slot groups of a wave (lanes lane xor O for O = LPS, 2 LPS, ..., 32): every
// lane gets the wave's maximum.
template <int O>
__device__ __forceinline__ float max_slot_groups(float v, int lane) {
  if constexpr (O <= 32) {
    v = fmaxf(v, lane_xor<O>(v, lane));
    return max_slot_groups<O * 2>(v, lane);
  } else {
    return v;
  }
}

// Value of lane (lane + O) for the lanes whose bit O is clear, within each 2O-lane block
// (other lanes get some other lane's value): one cross-lane move, no select.
template <int O>
__device__ __forceinline__ float lane_up(float v) {
  static_assert(O == 8 || O == 16 || O == 32, "exchange distance");
  if constexpr (O == 8) {
    return lane_xor8(v);
  } else if constexpr (O == 16) {
    return __uint_as_float(__builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false)[1]);
  } else {
    return __uint_as_float(__builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false)[1]);
  }
}

// Sums the softmax denominators and weighted V sums of a wave's slot groups (same lanes as
// above) into the first group (lanes 0 .. LPS-1); other lanes end with partial sums. All
// groups share one running maximum, so this is a plain sum.
template <int O, int GT>
__device__ __forceinline__ void sum_slot_groups(float (&ls)[GT], float (&acc)[GT][8]) {
  if constexpr (O <= 32) {
#pragma unroll
    for (int h = 0; h < GT; ++h) {
      ls[h] += lane_up<O>(ls[h]);
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[h][e] += lane_up<O>(acc[h][e]);
    }
    sum_slot_groups<O * 2, GT>(ls, acc);
  }
}

// A merger of (lane i, KV head g): chunk c = nc - 1 - r of the group, merging heads r, r + M,
// ... below G. Waits for the tagged partials of the other chunks of those heads (staged into cp
// around its own chunk c, already in LDS), combines them in chunk order (log-sum-exp) and
// writes those heads' attention output.
template <int D, int GT>
__device__ __forceinline__ bool merge_group(CParams& p, const Step& st, int l, int i, int g, int c, int nc, int M,
                                            float* cp, int tid) {
  const int G = p.G, nh = p.nh, row = D + 2;
  const int r = nc - 1 - c;
  const int nH = (G - r + M - 1) / M;     // heads merged here
  const __amdgpu_buffer_rsrc_t rpart = rsrc(p.part, (u32)((size_t)p.L * p.b * nh * p.maxc * row * 8));
  const int per_head = nc * row;
  const int others = (nc - 1) * row;      // even: row is even
  const int below = c * row;              // words of the chunks before this item's own
  // The group's heads are contiguous: [G][maxc][row] words, the first nc chunks in use.
  const u32 w0 = (u32)((((size_t)l * p.b + i) * nh + (size_t)g * G) * p.maxc * row);
  const u32 hstride = (u32)(p.maxc * row);
  auto where = [&](int k, u32& w, float*& d) {
    const int hi = k / others, rr = k - hi * others;
    const int o = rr < below ? rr : rr + row;   // skip chunk c (pairs never straddle a row)
    w = w0 + (u32)(r + hi * M) * hstride + (u32)o;
    d = cp + hi * per_head + o;
  };
  const bool ok = wait_copy_map<WB>(p, st, rpart, nH * others, where, tid);
  if (__syncthreads_or(!ok)) return false;
  const u32 obase = p.off_o + (u32)l * p.st_o + (u32)i * (u32)(nh * D);
  for (int u = tid; u < nH * D; u += NT) {
    const int hi = u / D, e = u % D, h = r + hi * M;
    const float* src = cp + hi * per_head;
    // The chunks in batches of 8: a batch's reads are issued together (indices past the last
    // chunk read the last chunk again and are dropped by a select), then used in chunk order.
    float mx = -INFINITY, den = 0.f, num = 0.f;
    for (int c0 = 0; c0 < nc; c0 += 8) {
      float mv[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) mv[k] = src[min(c0 + k, nc - 1) * row + D];
#pragma unroll
      for (int k = 0; k < 8; ++k) mx = fmaxf(mx, c0 + k < nc ? mv[k] : -INFINITY);
    }
    for (int c0 = 0; c0 < nc; c0 += 8) {
      float mv[8], lv[8], ov[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const float* pc = src + min(c0 + k, nc - 1) * row;
        mv[k] = pc[D];
        lv[k] = pc[D + 1];
        ov[k] = pc[e];
      }
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const float f = c0 + k < nc ? exp2f(mv[k] - mx) : 0.f;
        den += f * lv[k];
        num += f * ov[k];
      }
    }
    const float o = num / den;
    st_tag(p.act + obase + (u32)((g * G + h) * D + e), o, st.epoch);
    if (st.taps) st.taps[((size_t)l * p.b + i) * p.tap_block + p.tap_o + (g * G + h) * D + e] = o;
  }
  return true;
}

template <int D, int GT>
__device__ __forceinline__ bool op_attn(CParams& p, const Step& st, const int32_t* ins, float* smem, int tid,
                                        int lane, int wave, tl_t* tl) {
  // Grouped-query kernels with d = 64 (GT >= 2) run the scores and the weighted V sums on the
  // matrix cores in tiles of 16 slots per wave (pass width 128). At d = 128 the matrix-core
  // tiles measured slower on the Qwen3-0.6B shape and barely faster elsewhere, so those
  // kernels, and one-head-per-group kernels, use the VALU.
  constexpr bool MFA = GT >= 2 && D == 64;
  constexpr int VROW = D + 4;               // LDS row of one V slot, in bf16 values
  constexpr int LPS = D / 8, SPW = 64 / LPS, SPP = MFA ? 16 * NWAVE : SPW * NWAVE, NPF = 4;
  constexpr int KB = D / 32, DB = D / 16;   // 32-dim blocks (scores), 16-dim blocks (V sums)
  const int l = uni(ins[1]), j = uni(ins[2]);
  int i, g, c, nc, t0, t1;
  // VALU items cover at least 64 slots (two passes at d = 128): shorter chunks cost the merger
  // more than they save (measured on the Qwen3-0.6B shape at context 512).
  const lds_i32* lin = lane_inputs(smem);
  if (!item_map(p, lin + 16, j, SPP, MFA ? 16 : SPP, MFA ? 16 : 64, i, g, c, nc, t0, t1)) return true;
  i = uni(i); g = uni(g); c = uni(c); nc = uni(nc); t0 = uni(t0); t1 = uni(t1);
  const int G = p.G;
  const int kvl = uni(lin[16 + i]);
  const bool is_last = (t1 == kvl + 1);     // holds the new slot
  const int t_end = min(t1, kvl);            // slots [t0, t_end) come from the arena
  const int ssl = lane / LPS, de = (lane % LPS) * 8;
  CLayerPtrs& Lw = ((CLayerPtrs*)p.layers)[l];
  const u32 arena_bytes = (u32)p.b * (u32)p.nkv * (u32)p.max_ctx * (u32)D * 2u;
  const __amdgpu_buffer_rsrc_t rk = rsrc(Lw.kc, arena_bytes);
  const __amdgpu_buffer_rsrc_t rv = rsrc(Lw.vc, arena_bytes);
  const u32 head_slot0 = ((u32)i * p.nkv + (u32)g) * (u32)p.max_ctx;

  // This lane's rotary row and the QK-norm gains (they depend on no activation of this step),
  // then the q/k/v polls, then the K/V prefetch.
  const int half = D / 2;
  const float* rt = p.rope + (size_t)lin[8 + i] * half * 2;
  float2 rot = make_float2(1.f, 0.f);
  const int pe = tid % half;                  // rotary pair this thread applies
  rot = *reinterpret_cast<const float2*>(rt + pe * 2);
  // QK-norm gains (bf16) for dims lane and lane + 64, converted only once the polls are
  // checked (bf16 1.0 without QK-norm).
  u32 gq_b = 0x3F80u, gk_b = 0x3F80u, gq2_b = 0x3F80u, gk2_b = 0x3F80u;
  if (p.qk_norm) {
    gq_b = Lw.q_norm[lane];
    gk_b = Lw.k_norm[lane];
    if (D > 64) {
      gq2_b = Lw.q_norm[lane + 64];
      gk2_b = Lw.k_norm[lane + 64];
    }
  }

  // The q/k/v polls go out first (loads return in issue order: a poll behind the prefetch
  // could not report ready inputs before the prefetch had landed).
  const __amdgpu_buffer_rsrc_t ract = rsrc(p.act, p.act_bytes);
  const u32 base = p.off_qkv + (u32)l * p.st_qkv + (u32)i * (u32)((p.nh + 2 * p.nkv) * D);
  const int n3 = G * D + 2 * D;
  float* qs = smem + LDS_FLOATS - MISC_FLOATS - ATT_FLOATS;  // [G][D]
  float* ks = qs + GT * D;          // [D]
  float* vs = ks + D;               // [D]
  const u32 wq = base + (u32)(g * G * D), wk = base + (u32)(p.nh * D + g * D), wv = base + (u32)((p.nh + p.nkv) * D + g * D);
  auto where3 = [&](int k, u32& w, float*& d) {
    if (k < G * D) { w = wq + (u32)k; d = qs + k; }
    else if (k < G * D + D) { w = wk + (u32)(k - G * D); d = ks + (k - G * D); }
    else { w = wv + (u32)(k - G * D - D); d = vs + (k - G * D - D); }
  };
  static_assert((GT + 2) * D <= NT * 2 * 2, "q, k and v fit one poll batch of two pairs per thread");
  MapBatch<2> qkv_polls;
  issue_map<2>(ract, n3, where3, tid, qkv_polls);

  // Prefetch, before waiting for q: the first K/V of this wave (NPF passes, or two tiles),
  // this lane's rotary row and the QK-norm gains (none of them depend on this step's
  // activations).
  u32x4 kr[MFA ? 1 : NPF], vr[MFA ? 1 : NPF];
  auto kv_off = [&](int pass) {
    const int t = t0 + pass * SPP + wave * SPW + ssl;
    return (t < t_end) ? ((head_slot0 + (u32)t) * (u32)D + (u32)de) * 2u : 0xFFFFFFF0u;
  };
  auto issue_k = [&](int slot, int pass) { kr[slot] = __builtin_amdgcn_raw_buffer_load_b128(rk, kv_off(pass), 0, CPOL_NT); };
  auto issue_v = [&](int slot, int pass) { vr[slot] = __builtin_amdgcn_raw_buffer_load_b128(rv, kv_off(pass), 0, CPOL_NT); };
  // Matrix-core tiles: 16 slots s0 .. s0 + 15. K in the A-operand layout of the score product
  // (lane l: slot s0 + l % 16, dims 32 kb + 8 (l / 16) .. + 8: one 16-byte load per block); V
  // rows loaded the same way, to be transposed through LDS. Slots past the chunk load zeros
  // (out-of-range offsets).
  u32x4 kA[MFA ? KB : 1], kB2[MFA ? KB : 1];
  u32x4 wA[MFA ? KB : 1], wB2[MFA ? KB : 1];
  auto tile_load = [&](u32x4* kt, u32x4* wt, int s0) {
    const int tk = s0 + (lane & 15);
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      const u32 off = tk < t_end ? ((head_slot0 + (u32)tk) * (u32)D + (u32)(32 * kb + 8 * (lane >> 4))) * 2u : 0xFFFFFFF0u;
      kt[kb] = __builtin_amdgcn_raw_buffer_load_b128(rk, off, 0, CPOL_NT);
      wt[kb] = __builtin_amdgcn_raw_buffer_load_b128(rv, off, 0, CPOL_NT);
    }
  };
  if constexpr (MFA) {
    tile_load(kA, wA, t0 + 16 * wave);
    tile_load(kB2, wB2, t0 + 16 * (wave + NWAVE));
  } else {
#pragma unroll
    for (int s = 0; s < NPF; ++s) { issue_k(s, s); issue_v(s, s); }
  }
  // LDS: the merger's partials at the start, this item's working vectors near the end.
  static_assert(GT * D + 2 * D + NWAVE * GT * (D + 2) <= ATT_FLOATS, "attention LDS");
  static_assert(kMergeFloats + 3 * KB * 64 * 4 <= LDS_FLOATS - MISC_FLOATS - ATT_FLOATS, "q planes in LDS");
  static_assert(NWAVE * 16 * VROW <= 2 * kMergeFloats, "V tiles in the merge region");
  float* cp = smem;                 // [G][nc][D + 2], at most kMergeFloats
  float* wst = vs + D;              // [NWAVE][GT][D + 2]

  // The first uses of the polls, the rotary row and the gains stay behind the prefetch: the
  // compiler would otherwise wait for them between the prefetch's loads (and a wait for any
  // load also waits for the previous instruction's stores).
  asm volatile("" : "+v"(qkv_polls.v[0]), "+v"(qkv_polls.v[1]), "+v"(rot), "+v"(gq_b), "+v"(gk_b), "+v"(gq2_b),
               "+v"(gk2_b) :: "memory");
  const float gq = __uint_as_float(gq_b << 16), gk = __uint_as_float(gk_b << 16);
  const float gq2 = __uint_as_float(gq2_b << 16), gk2 = __uint_as_float(gk2_b << 16);

  // Wait for this group's q heads, k and v (one batched round trip when they are ready).
  bool ok = finish_map<2>(p, st, ract, n3, where3, tid, qkv_polls);
  if (__syncthreads_or(!ok)) return false;
  if (tl && tid == 0) tl[1] = clock_now();

  // Per-head RMSNorm on q and k (Qwen3-shaped models), then RoPE.
  if (p.qk_norm) {
    for (int hh = wave; hh <= G; hh += NWAVE) {
      float* v = (hh < G) ? qs + hh * D : ks;
      float a0 = v[lane], a1 = (D > 64) ? v[lane + 64] : 0.f;
      const float ss = wave_sum(a0 * a0 + a1 * a1);
      const float r = 1.0f / sqrtf(ss / (float)D + p.eps);
      v[lane] = a0 * r * ((hh < G) ? gq : gk);
      if (D > 64) v[lane + 64] = a1 * r * ((hh < G) ? gq2 : gk2);
    }
    __syncthreads();
  }
  for (int u = tid; u < (G + 1) * half; u += NT) {
    const int hh = u / half, e = u % half;     // e == pe since NT is a multiple of half
    float* v = (hh < G) ? qs + hh * D : ks;
    const float a = v[e], b = v[e + half];
    v[e] = a * rot.x - b * rot.y;
    v[e + half] = b * rot.x + a * rot.y;
  }
  __syncthreads();
  if (st.taps) {
    float* tb = st.taps + ((size_t)l * p.b + i) * p.tap_block;
    if (c == 0)
      for (int u = tid; u < G * D; u += NT) tb[p.tap_qrot + g * G * D + u] = qs[u];
    if (is_last)
      for (int u = tid; u < D; u += NT) tb[p.tap_krot + g * D + u] = ks[u];
  }
  if (is_last) {
    // KV append: round to bf16 and write slot kv_len; attention reads the rounded values.
    uint16_t* kd = Lw.kc + ((size_t)head_slot0 + kvl) * D;
    uint16_t* vd = Lw.vc + ((size_t)head_slot0 + kvl) * D;
    for (int e = tid; e < D; e += NT) {
      const uint16_t kb = to_bf16(ks[e]), vb = to_bf16(vs[e]);
      kd[e] = kb; vd[e] = vb;
      ks[e] = __uint_as_float((u32)kb << 16);
      vs[e] = __uint_as_float((u32)vb << 16);
    }
    __syncthreads();
  }

  if constexpr (MFA) {
    // q as the B operand of the score product S^T = K Q^T (v_mfma_f32_16x16x32_bf16): lane l
    // holds head l % 16 (zero past G) at dims 32 kb + 8 (l / 16) .. + 8, split into three bf16
    // planes (hi + mid + lo = q to about 2^-24 relative), so the scores keep fp32 precision.
    // The same for every wave: built once in LDS, [plane][kb][lane] 16 bytes each.
    u32x4* qpl = reinterpret_cast<u32x4*>(smem + kMergeFloats);
    for (int u = tid; u < KB * 64; u += NT) {
      const int kb = u / 64, ln = u % 64, h = ln & 15, d0 = 32 * kb + 8 * (ln >> 4);
      u32 w[3][4];
#pragma unroll
      for (int e2 = 0; e2 < 4; ++e2) {
        u32 hv[2], mv[2], lv[2];
#pragma unroll
        for (int q2 = 0; q2 < 2; ++q2) {
          float x = (h < G) ? qs[h * D + d0 + 2 * e2 + q2] * p.q_scale : 0.f;
          const uint16_t hi = to_bf16(x);
          x -= __uint_as_float((u32)hi << 16);
          const uint16_t mi = to_bf16(x);
          x -= __uint_as_float((u32)mi << 16);
          hv[q2] = hi; mv[q2] = mi; lv[q2] = to_bf16(x);
        }
        w[0][e2] = hv[0] | (hv[1] << 16);
        w[1][e2] = mv[0] | (mv[1] << 16);
        w[2][e2] = lv[0] | (lv[1] << 16);
      }
#pragma unroll
      for (int pl = 0; pl < 3; ++pl) qpl[(pl * KB + kb) * 64 + ln] = u32x4{w[pl][0], w[pl][1], w[pl][2], w[pl][3]};
    }
    __syncthreads();
    // Per lane: head l % 16; running maximum m (the same in the lane's four groups), partial
    // denominator ls over its slots, and O^T blocks (dims 16 db + 4 (l / 16) + r).
    float m = -INFINITY, ls = 0.f;
    f32x4 o[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db) o[db] = f32x4{0.f, 0.f, 0.f, 0.f};
    // One tile: scores S^T (rows = slots 4 (l / 16) + r, columns = heads), a running maximum
    // per head across the wave, then O^T += V^T P^T on v_mfma_f32_16x16x16_bf16, whose B
    // operand (slots 4 (l / 16) .. + 4 of head l % 16) is the score tile's own C layout. P is
    // split into three bf16 planes like q.
    typedef short s16x4 __attribute__((ext_vector_type(4)));
    uint16_t* vbuf = reinterpret_cast<uint16_t*>(smem) + wave * 16 * VROW;   // this wave's V tile
    auto tile = [&](const u32x4* kt, const u32x4* wt, auto live_row) {
      // V rows into LDS ([16 slots][VROW]; rows 8 bytes longer than d so that the four slot
      // rows read together below fall in different banks), read back transposed below.
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) {
        u32* dst = reinterpret_cast<u32*>(vbuf + (lane & 15) * VROW + 32 * kb + 8 * (lane >> 4));
        dst[0] = wt[kb].x; dst[1] = wt[kb].y; dst[2] = wt[kb].z; dst[3] = wt[kb].w;
      }
      // The rows are written as 32-bit words and read back as 16-bit values: keep the compiler
      // from moving the reads above the writes (type-based alias analysis would).
      asm volatile("" ::: "memory");
      f32x4 sc4 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) {
        const bf16x8 a = __builtin_bit_cast(bf16x8, kt[kb]);
#pragma unroll
        for (int pl = 2; pl >= 0; --pl)
          sc4 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, __builtin_bit_cast(bf16x8, qpl[(pl * KB + kb) * 64 + lane]),
                                                        sc4, 0, 0, 0);
      }
      const bool head_live = (lane & 15) < G;
      float sc[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) sc[r] = (head_live && live_row(r)) ? sc4[r] : -INFINITY;
      float mt = fmaxf(fmaxf(sc[0], sc[1]), fmaxf(sc[2], sc[3]));
      mt = fmaxf(mt, lane_xor<16>(mt, lane));
      mt = fmaxf(mt, lane_xor<32>(mt, lane));
      const float mn = fmaxf(m, mt);
      const float a = (m == -INFINITY) ? 0.f : exp2f(m - mn);
      ls *= a;
#pragma unroll
      for (int db = 0; db < DB; ++db) o[db] *= a;
      m = mn;
      s16x4 ph, pm, pl;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float x = (sc[r] == -INFINITY) ? 0.f : exp2f(sc[r] - mn);
        ls += x;
        const uint16_t hi = to_bf16(x);
        x -= __uint_as_float((u32)hi << 16);
        const uint16_t mi = to_bf16(x);
        x -= __uint_as_float((u32)mi << 16);
        const uint16_t lo = to_bf16(x);
        ph[r] = (short)hi; pm[r] = (short)mi; pl[r] = (short)lo;
      }
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        // V^T operand: dim 16 db + l % 16 of slots 4 (l / 16) .. + 4.
        s16x4 va;
#pragma unroll
        for (int r = 0; r < 4; ++r) va[r] = (short)vbuf[(4 * (lane >> 4) + r) * VROW + 16 * db + (lane & 15)];
        o[db] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(va, pl, o[db], 0, 0, 0);
        o[db] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(va, pm, o[db], 0, 0, 0);
        o[db] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(va, ph, o[db], 0, 0, 0);
      }
      asm volatile("" ::: "memory");   // the next tile's rows are written after these reads
    };
    if (tl && tid == 0) tl[2] = clock_now();
    // This wave's tiles: 16-slot tiles wave, wave + 8, ... of the chunk, two in flight.
    const int n_arena = t_end - t0;
    const int ntile = n_arena > 16 * wave ? (n_arena - 16 * wave + SPP - 1) / SPP : 0;
    for (int k = 0; k < ntile; k += 2) {
      {
        const int s0 = t0 + 16 * (wave + NWAVE * k);
        tile(kA, wA, [&](int r) { return s0 + 4 * (lane >> 4) + r < t_end; });
        if (k + 2 < ntile) tile_load(kA, wA, t0 + 16 * (wave + NWAVE * (k + 2)));
      }
      if (k + 1 < ntile) {
        const int s0 = t0 + 16 * (wave + NWAVE * (k + 1));
        tile(kB2, wB2, [&](int r) { return s0 + 4 * (lane >> 4) + r < t_end; });
        if (k + 3 < ntile) tile_load(kB2, wB2, t0 + 16 * (wave + NWAVE * (k + 3)));
      }
    }
    if (is_last && wave == 0) {
      // The new slot, as stored (bf16), folded into wave 0's running state on the VALU: its
      // score for each head (a wave sum over the dims), then the usual update of this lane's
      // head. The denominator counts it once, in the first lane group.
      float s_new = -INFINITY;
#pragma unroll
      for (int hh = 0; hh < GT; ++hh) {   // unrolled: the heads' reductions interleave
        float x = hh < G ? qs[hh * D + lane] * p.q_scale * ks[lane] : 0.f;
        if (D > 64 && hh < G) x = fmaf(qs[hh * D + lane + 64] * p.q_scale, ks[lane + 64], x);
        x = wave_sum(x);
        if ((lane & 15) == hh && hh < G) s_new = x;
      }
      const float mn = fmaxf(m, s_new);
      const float a = (m == -INFINITY) ? 0.f : exp2f(m - mn);
      const float pw = (s_new == -INFINITY) ? 0.f : exp2f(s_new - mn);
      ls = ls * a + (((lane >> 4) == 0) ? pw : 0.f);
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int r = 0; r < 4; ++r) o[db][r] = fmaf(pw, vs[16 * db + 4 * (lane >> 4) + r], o[db][r] * a);
      m = mn;
    }
    if (tl && tid == 0) tl[6] = clock_now();
    // The denominator of each head over the wave's slots: its four lane groups.
    ls += lane_xor<16>(ls, lane);
    ls += lane_xor<32>(ls, lane);
    const int h = lane & 15;
    if (h < G) {
      float* w = wst + (wave * GT + h) * (D + 2);
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int r = 0; r < 4; ++r) w[16 * db + 4 * (lane >> 4) + r] = o[db][r];
      if ((lane >> 4) == 0) { w[D] = m; w[D + 1] = ls; }
    }
  } else {
    // q of the group's heads for this lane's 8 dims: two 16-byte LDS reads per head, all in
    // flight together (heads past G read the buffer's unused rows and are zeroed by the
    // select, not by a branch around the read).
    float qr[GT][8];
  #pragma unroll
    for (int h = 0; h < GT; ++h) {
      const float4 a = *reinterpret_cast<const float4*>(qs + h * D + de);
      const float4 c = *reinterpret_cast<const float4*>(qs + h * D + de + 4);
      const float v[8] = {a.x, a.y, a.z, a.w, c.x, c.y, c.z, c.w};
  #pragma unroll
      for (int e = 0; e < 8; ++e) qr[h][e] = (h < G) ? v[e] * p.q_scale : 0.f;
    }
    // The running maxima start at -FLT_MAX rather than -inf, so that every exponent below is
    // m - m' or s - m with m finite: never inf - inf, and exp2 of -inf (an empty slot) is 0.
    // That lets the hardware exp2 run unguarded; its arguments are never positive.
    float m[GT], ls[GT], acc[GT][8];
  #pragma unroll
    for (int h = 0; h < GT; ++h) {
      m[h] = -3.40282347e38f; ls[h] = 0.f;   // -FLT_MAX
  #pragma unroll
      for (int e = 0; e < 8; ++e) acc[h][e] = 0.f;
    }
    // One block of NB slot passes (all wave-uniform): the scores of every slot in the block
    // first, then one running maximum per head shared by the whole wave, then the exponentials
    // and the weighted V sums. Because the maximum is the same in every lane, the wave's slot
    // groups are combined at the end by plain sums, with no rescaling. ok[s] says the wave holds
    // pass s; val[s] that this lane's slot in it is live. refill_k / refill_v(s) are called once
    // pass s's K (V) registers are no longer needed, for every s: loads under a branch would
    // leave the compiler unsure how many loads follow each slot's, and it would then wait for
    // all of them (the refill just issued included) before every slot. Passes past the chunk
    // load zeros.
    auto block = [&](auto nbc, const u32x4* kw, const u32x4* vw, const bool* ok, const bool* val, auto refill_k,
                     auto refill_v) {
      constexpr int NB = decltype(nbc)::value;
      float sc[NB][GT];
  #pragma unroll
      for (int s = 0; s < NB; ++s) {
  #pragma unroll
        for (int h = 0; h < GT; ++h) sc[s][h] = -INFINITY;
        const u32x4 k = kw[s];
        float kf[8] = {bf16lo(k.x), bf16hi(k.x), bf16lo(k.y), bf16hi(k.y),
                       bf16lo(k.z), bf16hi(k.z), bf16lo(k.w), bf16hi(k.w)};
        order_before_load(kf);
        refill_k(s);
        if (ok[s]) {
  #pragma unroll
          for (int h = 0; h < GT; ++h) {
            if (h < G) {
              float x = 0.f;
  #pragma unroll
              for (int e = 0; e < 8; ++e) x = fmaf(qr[h][e], kf[e], x);
              x = (LPS == 16) ? row16_sum(x) : row8_sum(x);
              sc[s][h] = val[s] ? x : -INFINITY;
            }
          }
        }
      }
  #pragma unroll
      for (int h = 0; h < GT; ++h) {
        float bm = sc[0][h];
  #pragma unroll
        for (int s = 1; s < NB; ++s) bm = fmaxf(bm, sc[s][h]);
        bm = max_slot_groups<LPS>(bm, lane);
        const float mn = fmaxf(m[h], bm);
        const float a = __builtin_amdgcn_exp2f(m[h] - mn);
        ls[h] *= a;
  #pragma unroll
        for (int e = 0; e < 8; ++e) acc[h][e] *= a;
        m[h] = mn;
      }
  #pragma unroll
      for (int s = 0; s < NB; ++s) {
        const u32x4 v = vw[s];
        float vf[8] = {bf16lo(v.x), bf16hi(v.x), bf16lo(v.y), bf16hi(v.y),
                       bf16lo(v.z), bf16hi(v.z), bf16lo(v.w), bf16hi(v.w)};
        order_before_load(vf);
        refill_v(s);
        if (ok[s]) {
  #pragma unroll
          for (int h = 0; h < GT; ++h) {
            const float pw = __builtin_amdgcn_exp2f(sc[s][h] - m[h]);
            ls[h] += pw;
  #pragma unroll
            for (int e = 0; e < 8; ++e) acc[h][e] = fmaf(pw, vf[e], acc[h][e]);
          }
        }
      }
    };
    if (tl && tid == 0) tl[2] = clock_now();
    const int n_arena = t_end - t0;
    const int npass = n_arena > 0 ? (n_arena + SPP - 1) / SPP : 0;
    // Full blocks with more passes after them refill the ring in place (every pass held, no
    // branch); the last block, full or not, only consumes. Within a block the compiler then
    // waits for each slot's own loads only.
    int pb = 0;
    for (; pb + NPF < npass; pb += NPF) {
      bool ok[NPF], val[NPF];
  #pragma unroll
      for (int sl = 0; sl < NPF; ++sl) {
        ok[sl] = true;
        val[sl] = t0 + (pb + sl) * SPP + wave * SPW + ssl < t_end;
      }
      block(std::integral_constant<int, NPF>{}, kr, vr, ok, val,
            [&](int sl) { issue_k(sl, pb + sl + NPF); }, [&](int sl) { issue_v(sl, pb + sl + NPF); });
    }
    if (pb < npass) {
      bool ok[NPF], val[NPF];
  #pragma unroll
      for (int sl = 0; sl < NPF; ++sl) {
        ok[sl] = pb + sl < npass;
        val[sl] = t0 + (pb + sl) * SPP + wave * SPW + ssl < t_end;
      }
      block(std::integral_constant<int, NPF>{}, kr, vr, ok, val, [](int) {}, [](int) {});
    }
    if (is_last && wave == 0) {
      // The new slot, as stored (bf16), in the first slot group of wave 0.
      u32x4 kw1, vw1;
      u32 kp[4], vp[4];
  #pragma unroll
      for (int j = 0; j < 4; ++j) {
        kp[j] = (__float_as_uint(ks[de + 2 * j]) >> 16) | (__float_as_uint(ks[de + 2 * j + 1]) & 0xffff0000u);
        vp[j] = (__float_as_uint(vs[de + 2 * j]) >> 16) | (__float_as_uint(vs[de + 2 * j + 1]) & 0xffff0000u);
      }
      kw1 = u32x4{kp[0], kp[1], kp[2], kp[3]};
      vw1 = u32x4{vp[0], vp[1], vp[2], vp[3]};
      const bool ok1[1] = {true}, val1[1] = {ssl == 0};
      block(std::integral_constant<int, 1>{}, &kw1, &vw1, ok1, val1, [](int) {}, [](int) {});
    }
    if (tl && tid == 0) tl[6] = clock_now();
    sum_slot_groups<LPS, GT>(ls, acc);
    if (ssl == 0) {
  #pragma unroll
      for (int h = 0; h < GT; ++h) {
        if (h < G) {
          float* w = wst + (wave * GT + h) * (D + 2);
  #pragma unroll
          for (int e = 0; e < 8; ++e) w[de + e] = acc[h][e];
          if (de == 0) { w[D] = m[h]; w[D + 1] = ls[h]; }
        }
      }
    }
  }
  __syncthreads();
  if (tl && tid == 0) tl[7] = clock_now();
  // Merge the waves in order: the chunk's partial for each head. A merger keeps its own of the
  // heads it merges in LDS (slot c of cp); the rest are published as tagged words.
  const int nh = p.nh;
  const int row = D + 2;
  const int NM = uni(min(min(G, nc), (int)p.nwg));  // mergers of the group (see above)
  const int mr = nc - 1 - c;                         // merger rank, when below NM
  for (int u = tid; u < G * row; u += NT) {
    const int h = u / row, e = u % row;
    // Every wave's maximum and value first (all reads in flight together), then the sum in
    // wave order; an empty wave (maximum -inf) contributes 0 through a select, not a branch.
    float mw[NWAVE], vw[NWAVE];
#pragma unroll
    for (int w = 0; w < NWAVE; ++w) {
      mw[w] = wst[(w * GT + h) * row + D];
      vw[w] = wst[(w * GT + h) * row + e];
    }
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < NWAVE; ++w) M = fmaxf(M, mw[w]);
    float A = 0.f;
#pragma unroll
    for (int w = 0; w < NWAVE; ++w) {
      const float f = exp2f(mw[w] - M);
      A += vw[w] * (mw[w] == -INFINITY ? 0.f : f);   // e == D + 1 sums the softmax denominators
    }
    const float val = (e == D) ? M : A;
    if (mr < NM && h % NM == mr) {
      cp[((h / NM) * nc + c) * row + e] = val;
    } else {
      u64* dst = p.part + ((((size_t)l * p.b + i) * nh + g * G + h) * p.maxc + c) * row;
      st_tag(dst + e, val, st.epoch);
    }
  }
  if (tl && tid == 0) tl[3] = clock_now();
  if (mr < NM && !merge_group<D, GT>(p, st, l, i, g, c, nc, NM, cp, tid)) return false;
  __syncthreads();   // LDS is reused by the next instruction
  return true;
}

}  // namespace dev
}  // namespace fm
