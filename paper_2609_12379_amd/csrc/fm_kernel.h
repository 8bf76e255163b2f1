// The step interpreter kernel (one persistent launch per step, or one launch per stage).
// Each workgroup walks its own instruction queue, built on the host by fm_plan.cpp, and
// waits only for the data its next instruction consumes (arXiv 2609.12379 Sec. 4.1).
#pragma once
#include "fm_device.h"
#include "fm_ops.h"

namespace fm {
namespace dev {

template <int B, int D, int GT>
__global__ __launch_bounds__(NT, 1) void step_kernel(const Params* __restrict__ pparams, Step st) {
  CParams& p = *(CParams*)pparams;
  __shared__ __attribute__((aligned(16))) float smem[LDS_FLOATS];
  const int tid = threadIdx.x, lane = tid & 63, wg = blockIdx.x;
  // The wave index is uniform across a wave; readfirstlane tells the compiler so, which keeps
  // per-wave loop counters and buffer descriptors in scalar registers.
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);

  // Per-lane inputs live on the device: check them here. A bad step does nothing but record
  // the error (every workgroup reaches the same verdict).
  u32 code = 0;
  if (tid < p.b) {
    const int t = st.tok[tid], ps = st.pos[tid], kl = st.kvl[tid];
    lds_i32* lin = lane_inputs(smem);
    lin[tid] = t;
    lin[8 + tid] = ps;
    lin[16 + tid] = kl;
    if (t < 0 || t >= p.V) code = FM_DEV_BAD_TOKEN;
    else if (ps < 0 || ps >= p.max_ctx) code = FM_DEV_BAD_POSITION;
    else if (kl < 0 || kl >= p.max_ctx) code = FM_DEV_BAD_KV_LEN;
  }
  if (__syncthreads_or(code != 0)) {
    if (code && wg == 0) raise_error(p, code);
    return;
  }
  if (abort_raised(p)) return;

  // Queue bounds and instruction words come in by scalar loads (constant address space, counted
  // by lgkmcnt): a vector load would be waited for with vmcnt, which first waits for every
  // store of the previous instruction to be acknowledged. The tables are written by the host
  // before the launch and never during it. (At batch 4 and 8 it measured slower: the wider
  // tiles need those scalar registers, and the matrix-core tiles would spill.)
  typedef const __attribute__((address_space(4))) int32_t cq_t;
  constexpr bool SCAL = B <= 2;
  int q0, q1;
  if (st.stage < 0) {
    q0 = SCAL ? ((const cq_t*)p.qoff)[wg] : p.qoff[wg];
    q1 = SCAL ? ((const cq_t*)p.qoff)[wg + 1] : p.qoff[wg + 1];
  } else {
    const size_t k = ((size_t)st.stage * p.nwg + wg) * 2;
    q0 = SCAL ? ((const cq_t*)p.stage_rng)[k] : p.stage_rng[k];
    q1 = SCAL ? ((const cq_t*)p.stage_rng)[k + 1] : p.stage_rng[k + 1];
  }
  if constexpr (SCAL) {
    q0 = __builtin_amdgcn_readfirstlane(q0);
    q1 = __builtin_amdgcn_readfirstlane(q1);
  }
  for (int q = q0; q < q1; ++q) {
    // Re-derive the parameter pointer per instruction, opaquely: the compiler then reloads
    // fields from the (scalar-cached) kernel-argument segment inside each operator instead of
    // keeping every field of every operator live in scalar registers for the whole step.
    CParams* pp = (CParams*)pparams;
    asm volatile("" : "+s"(pp));
    CParams& P = *pp;
    const int32_t* insg = P.instrs + 4 * (size_t)q;
    int32_t iw[4];
    if constexpr (SCAL) {
      const cq_t* insc = (const cq_t*)insg;
      iw[0] = insc[0]; iw[1] = insc[1]; iw[2] = insc[2]; iw[3] = insc[3];
    }
    const int32_t* ins = SCAL ? iw : insg;
    const int op = ins[0];
    u64* tg = st.timeline ? st.timeline + 8 * (size_t)q : nullptr;
    tl_t* tl = tg ? (tl_t*)(__attribute__((address_space(3))) float*)(smem + LDS_FLOATS - 24) : nullptr;   // 8 marks
    if (tl && tid == 0) { tl[0] = clock_now(); tl[1] = 0; tl[2] = 0; tl[3] = 0; tl[5] = (u64)wg; tl[6] = 0; tl[7] = 0; }
    bool ok = true;
    if (op == FM_OP_ATTN) {
      ok = op_attn<D, GT>(P, st, ins, smem, tid, lane, wave, tl);
    } else if (ins[2] < 0) {
      // A QKV, O-projection or down stage in dynamic chunks (VALU tiles only).
      if constexpr (B <= 2) {
        ok = op_gemv_dyn<B>(P, st, ins, smem, tid, lane, wave, tl);
      } else {
        if (tid == 0) raise_error(P, FM_DEV_BAD_PLAN);
        ok = false;
      }
    } else if (op == FM_OP_GU) {
      ok = op_gemv<B, 2>(P, st, ins, smem, tid, lane, wave, tl);
    } else {
      ok = op_gemv<B, 1>(P, st, ins, smem, tid, lane, wave, tl);
    }
    if (!ok) return;
    if (tl && tid == 0) {
      tl[4] = clock_now();
#pragma unroll
      for (int k = 0; k < 8; ++k) tg[k] = tl[k];
    }
  }
}

}  // namespace dev
}  // namespace fm


namespace fm {
namespace dev {
// Kernel lookup, one per batch specialisation (defined in fm_kernels.hip, compiled once per B).
const void* kernel_for_b1(int d, int G);
const void* kernel_for_b2(int d, int G);
const void* kernel_for_b4(int d, int G);
const void* kernel_for_b8(int d, int G);
}  // namespace dev
}  // namespace fm
