// Operator bodies executed by the step interpreter: GEMV row-tiles (with fused RMSNorm
// prologue, residual/SiLU/argmax epilogues) and split-KV attention work items (with fused
// QK-norm, RoPE, KV append, online softmax and a last-arriver log-sum-exp combine).
#pragma once
#include "fm_device.h"
#include "../../include/fm.h"

namespace fm {
namespace dev {

// ---- waiting on tagged words ----------------------------------------------------------

__device__ __forceinline__ bool abort_raised(const Params& p) {
  return __hip_atomic_load(p.abort_flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0u;
}

__device__ __forceinline__ void raise_error(const Params& p, u32 code) {
  __hip_atomic_store(p.abort_flag, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __hip_atomic_store(p.err_host, code, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

// Reads the tagged pair at word offset w (even), spinning until both words carry the
// epoch. Returns false if the watchdog fires or another workgroup raised the abort flag.
__device__ __forceinline__ bool wait_pair(const Params& p, __amdgpu_buffer_rsrc_t ra, u32 w,
                                          float& a, float& b) {
  u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(ra, w * 8u, 0, CPOL_SC1);
  if (v.y != p.epoch || v.w != p.epoch) {
    const u64 t0 = clock_now();
    int it = 0;
    while (true) {
      __builtin_amdgcn_s_sleep(1);
      v = __builtin_amdgcn_raw_buffer_load_b128(ra, w * 8u, 0, CPOL_SC1);
      if (v.y == p.epoch && v.w == p.epoch) break;
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
// accumulates the sum of squares of the values this thread copied into ss.
__device__ __forceinline__ bool wait_copy(const Params& p, __amdgpu_buffer_rsrc_t ra, u32 w0, int n,
                                          float* dst, float& ss, int tid) {
  for (int k = tid * 2; k < n; k += NT * 2) {
    float a, b;
    if (!wait_pair(p, ra, w0 + (u32)k, a, b)) return false;
    ss += a * a + b * b;
    if (dst) {
      dst[k] = a;
      dst[k + 1] = b;
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
// Output rows [ra, rb) of one operator, B lanes (B is the batch rounded up to 1, 2, 4 or 8),
// NW weight rows per output row (2 for gate/up, else 1). Rows are dealt to the waves
// round-robin. Inside a wave, each lane streams 16 bytes (8 bf16) per weight-row segment of
// 512 columns. U such loads stay in flight per lane in a register ring. The ring is filled
// BEFORE the input wait, so a tile's weights stream while its producers finish. The input
// vector is staged in LDS (fp32, RMSNorm applied when the operator has one) in slabs of
// at most XSLAB_FLOATS / B columns. Partial sums across slabs accumulate in LDS.

template <int B, int NW>
__device__ bool op_gemv(const Params& p, const int32_t* ins, float* smem, int tid, int lane, int wave) {
  const int op = ins[0], l = ins[1], ra = ins[2], rb = ins[3];
  const int nr = rb - ra;
  const int nq = p.nh * p.d, nk = p.nkv * p.d, nqkv = nq + 2 * nk;
  const LayerPtrs* Lw = (op == FM_OP_LM) ? nullptr : p.layers + l;

  // Operator geometry.
  int K = 0;
  const uint16_t* gain = nullptr;   // RMSNorm gain (norm prologue) or null
  bool from_embed = false;          // input is the embedding row (layer 0 QKV)
  u32 in_w = 0, in_stride = 0;      // tagged input: word offset of lane 0, words per lane
  u32 res_w = 0, res_stride = 0;    // tagged residual (OPROJ, DOWN)
  bool res_embed = false, has_res = false;
  const uint16_t* m0 = nullptr; const uint16_t* m1 = nullptr; const uint16_t* m2 = nullptr;
  u32 n0 = 0, n1 = 0;               // QKV: rows of W_q, W_k
  switch (op) {
    case FM_OP_QKV:
      K = p.h; gain = Lw->attn_norm;
      if (l == 0) from_embed = true; else { in_w = p.off_x + (u32)l * p.st_x; in_stride = p.h; }
      m0 = Lw->wq; m1 = Lw->wk; m2 = Lw->wv; n0 = nq; n1 = nk;
      break;
    case FM_OP_OPROJ:
      K = nq; in_w = p.off_o + (u32)l * p.st_o; in_stride = nq;
      has_res = true;
      if (l == 0) res_embed = true; else { res_w = p.off_x + (u32)l * p.st_x; res_stride = p.h; }
      m0 = Lw->wo;
      break;
    case FM_OP_GU:
      K = p.h; gain = Lw->mlp_norm; in_w = p.off_x1 + (u32)l * p.st_x1; in_stride = p.h;
      m0 = Lw->wg; m1 = Lw->wu;
      break;
    case FM_OP_DOWN:
      K = p.inter; in_w = p.off_m + (u32)l * p.st_m; in_stride = p.inter;
      has_res = true; res_w = p.off_x1 + (u32)l * p.st_x1; res_stride = p.h;
      m0 = Lw->wd;
      break;
    default:  // FM_OP_LM
      K = p.h; gain = p.final_norm; in_w = p.off_x + (u32)p.L * p.st_x; in_stride = p.h;
      m0 = p.lm_head;
      break;
  }
  const u32 rowbytes = (u32)K * 2u;
  __amdgpu_buffer_rsrc_t r0, r1, r2;
  if (op == FM_OP_QKV) {
    r0 = rsrc(m0, n0 * rowbytes); r1 = rsrc(m1, n1 * rowbytes); r2 = rsrc(m2, n1 * rowbytes);
  } else if (op == FM_OP_GU) {
    r0 = rsrc(m0, (u32)p.inter * rowbytes); r1 = rsrc(m1, (u32)p.inter * rowbytes); r2 = r0;
  } else {
    const u32 rows = (op == FM_OP_LM) ? (u32)p.V : (u32)p.h;
    r0 = rsrc(m0, rows * rowbytes); r1 = r0; r2 = r0;
  }
  const __amdgpu_buffer_rsrc_t ract = rsrc(p.act, p.act_bytes);

  // Slab geometry.
  const int Kpad = (K + 511) & ~511;
  int Ks = (XSLAB_FLOATS / B) & ~511;
  if (Ks > Kpad) Ks = Kpad;
  const int nslab = (K + Ks - 1) / Ks;
  const int rows_w = nr > wave ? (nr - wave + NWAVE - 1) / NWAVE : 0;

  float* xs = smem;
  float* rowacc = smem + XSLAB_FLOATS;
  float* resid = rowacc + ROWACC_FLOATS;
  float* misc = resid + RESID_FLOATS;

  // Weight ring: deeper for small batches (fewer accumulators, more registers free).
  constexpr int U = (B <= 2) ? 16 : 8;
  u32x4 ring[U];
  int iq = 0, iw = 0, isg = 0;   // next unit to issue: (row of this wave, weight row, segment)
  int slab_i = 0, nseg_i = 0;    // slab being issued and its segment count
  auto seg_count = [&](int s) { return (min(Ks, K - s * Ks) + 511) >> 9; };
  auto issue = [&](int slot) {
    u32 off = 0xFFFFFFF0u;       // past every resource: the load returns zeros, no traffic
    __amdgpu_buffer_rsrc_t rr = r0;
    if (iq < rows_w) {
      const int r = ra + wave + iq * NWAVE;
      const int k = slab_i * Ks + isg * 512 + lane * 8;
      u32 lrow = (u32)r;
      if (op == FM_OP_QKV) {
        if (r >= (int)(n0 + n1)) { rr = r2; lrow = (u32)r - n0 - n1; }
        else if (r >= (int)n0) { rr = r1; lrow = (u32)r - n0; }
      } else if (NW == 2 && iw == 1) {
        rr = r1;
      }
      if (k < K) off = lrow * rowbytes + (u32)k * 2u;
      if (++isg == nseg_i) { isg = 0; if (++iw == NW) { iw = 0; ++iq; } }
    }
    ring[slot] = __builtin_amdgcn_raw_buffer_load_b128(rr, off, 0, CPOL_NT);
  };
  auto start_slab_issue = [&](int s) {
    slab_i = s; nseg_i = seg_count(s); iq = 0; iw = 0; isg = 0;
#pragma unroll
    for (int sl = 0; sl < U; ++sl) issue(sl);
  };

  // 1. Prefetch the first weights, before waiting for the input.
  start_slab_issue(0);

  // 2. Input: wait for the producers, then stage (normalised) values in LDS.
  bool ok = true;
  float rs[B];
#pragma unroll
  for (int i = 0; i < B; ++i) rs[i] = 1.0f;
  auto stage = [&](int s, bool accumulate_ss, float* ssv) -> bool {
    const int k0 = s * Ks, kn = min(Ks, K - k0);
    const int kfill = (kn + 511) & ~511;
#pragma unroll
    for (int i = 0; i < B; ++i) {
      float* dst = xs + i * Ks;
      float ss = 0.f;
      if (i < p.b) {
        if (from_embed) {
          const uint16_t* e = p.embed + (size_t)p.tok[i] * p.h + k0;
          for (int k = tid * 2; k < kn; k += NT * 2) {
            u32 w2 = *reinterpret_cast<const u32*>(e + k);
            float a = bf16lo(w2), b = bf16hi(w2);
            ss += a * a + b * b;
            dst[k] = a; dst[k + 1] = b;
          }
        } else {
          if (!wait_copy(p, ract, in_w + (u32)i * in_stride + (u32)k0, kn, dst, ss, tid)) return false;
        }
      } else {
        for (int k = tid; k < kn; k += NT) dst[k] = 0.f;
      }
      for (int k = kn + tid; k < kfill; k += NT) dst[k] = 0.f;
      if (accumulate_ss) ssv[i] += ss;
    }
    return true;
  };
  auto scale_slab = [&](int s) {
    if (!gain) return;
    const int k0 = s * Ks, kn = min(Ks, K - k0);
#pragma unroll
    for (int i = 0; i < B; ++i) {
      float* dst = xs + i * Ks;
      for (int k = tid; k < kn; k += NT) dst[k] = dst[k] * rs[i] * __uint_as_float((u32)gain[k0 + k] << 16);
    }
  };

  float ssv[B];
#pragma unroll
  for (int i = 0; i < B; ++i) ssv[i] = 0.f;
  if (nslab == 1) {
    ok = stage(0, gain != nullptr, ssv);
  } else if (gain) {
    // Whole-vector pass for the norm statistics, then stage slab 0.
    for (int i = 0; i < B && ok; ++i) {
      if (i >= p.b) continue;
      float ss = 0.f;
      if (from_embed) {
        const uint16_t* e = p.embed + (size_t)p.tok[i] * p.h;
        for (int k = tid * 2; k < K; k += NT * 2) {
          u32 w2 = *reinterpret_cast<const u32*>(e + k);
          float a = bf16lo(w2), b = bf16hi(w2);
          ss += a * a + b * b;
        }
      } else {
        ok = wait_copy(p, ract, in_w + (u32)i * in_stride, K, nullptr, ss, tid);
      }
      ssv[i] += ss;
    }
    if (ok) ok = stage(0, false, ssv);
  } else {
    ok = stage(0, false, ssv);
  }
  // Residual rows for the epilogue.
  if (ok && has_res) {
    for (int i = 0; i < B && ok; ++i) {
      if (i >= p.b) continue;
      if (res_embed) {
        const uint16_t* e = p.embed + (size_t)p.tok[i] * p.h;
        for (int k = tid; k < nr; k += NT) resid[i * nr + k] = __uint_as_float((u32)e[ra + k] << 16);
      } else {
        // ra is even for every split (rows are split into even-sized... not guaranteed): copy pairwise from an even base
        const int lo = ra & ~1, hi = (rb + 1) & ~1;
        for (int k = lo + tid * 2; k < hi; k += NT * 2) {
          float a, b;
          if (!wait_pair(p, ract, res_w + (u32)i * res_stride + (u32)k, a, b)) { ok = false; break; }
          if (k >= ra && k < rb) resid[i * nr + (k - ra)] = a;
          if (k + 1 >= ra && k + 1 < rb) resid[i * nr + (k + 1 - ra)] = b;
        }
      }
    }
  }
  if (__syncthreads_or(!ok)) return false;
  if (gain) {
#pragma unroll
    for (int i = 0; i < B; ++i) {
      float t = block_sum(ssv[i], misc, lane, wave);
      rs[i] = 1.0f / sqrtf(t / (float)K + p.eps);
    }
    scale_slab(0);
    __syncthreads();
  }
  // Taps of the normed input (first tile of the operator only), one slab at a time.
  auto tap_slab = [&](int s) {
    if (!(p.taps && gain && ra == 0)) return;
    const int k0 = s * Ks, kn = min(Ks, K - k0);
    const int off = (op == FM_OP_QKV) ? p.tap_a : (op == FM_OP_GU ? p.tap_a2 : 0);
    for (int i = 0; i < p.b; ++i) {
      float* t = (op == FM_OP_LM)
                     ? p.taps + (size_t)p.L * p.b * p.tap_block + (size_t)i * p.h
                     : p.taps + ((size_t)l * p.b + i) * p.tap_block + off;
      for (int k = tid; k < kn; k += NT) t[k0 + k] = xs[i * Ks + k];
    }
  };
  tap_slab(0);

  // 3. Stream the weights.
  float best_v[B];
  int best_i[B];
#pragma unroll
  for (int i = 0; i < B; ++i) { best_v[i] = 0.f; best_i[i] = -1; }
  float v0[B];
#pragma unroll
  for (int i = 0; i < B; ++i) v0[i] = 0.f;

  for (int s = 0; s < nslab; ++s) {
    if (s > 0) {
      __syncthreads();
      if (!stage(s, false, ssv)) ok = false;
      if (__syncthreads_or(!ok)) return false;
      scale_slab(s);
      __syncthreads();
      tap_slab(s);
      start_slab_issue(s);
    }
    const int nseg = seg_count(s);
    const int units = rows_w * NW * nseg;
    int cq = 0, cw = 0, csg = 0;
    float acc0[B], acc1[B];
#pragma unroll
    for (int i = 0; i < B; ++i) { acc0[i] = 0.f; acc1[i] = 0.f; }
    for (int base = 0; base < units; base += U) {
#pragma unroll
      for (int sl = 0; sl < U; ++sl) {
        if (base + sl < units) {
          const u32x4 w = ring[sl];
          issue(sl);
          const float wf[8] = {bf16lo(w.x), bf16hi(w.x), bf16lo(w.y), bf16hi(w.y),
                               bf16lo(w.z), bf16hi(w.z), bf16lo(w.w), bf16hi(w.w)};
          const int kk = csg * 512 + lane * 8;
#pragma unroll
          for (int i = 0; i < B; ++i) {
            const float4 xa = *reinterpret_cast<const float4*>(xs + i * Ks + kk);
            const float4 xb = *reinterpret_cast<const float4*>(xs + i * Ks + kk + 4);
            float t0 = wf[0] * xa.x, t1 = wf[1] * xa.y;
            t0 = fmaf(wf[2], xa.z, t0); t1 = fmaf(wf[3], xa.w, t1);
            t0 = fmaf(wf[4], xb.x, t0); t1 = fmaf(wf[5], xb.y, t1);
            t0 = fmaf(wf[6], xb.z, t0); t1 = fmaf(wf[7], xb.w, t1);
            if (NW == 2 && cw == 1) acc1[i] += t0 + t1; else acc0[i] += t0 + t1;
          }
          if (csg == nseg - 1) {
            // One weight row finished for this slab: reduce across the wave.
            float v[B];
#pragma unroll
            for (int i = 0; i < B; ++i) {
              v[i] = wave_sum((NW == 2 && cw == 1) ? acc1[i] : acc0[i]);
              if (NW == 2 && cw == 1) acc1[i] = 0.f; else acc0[i] = 0.f;
            }
            const int rl = wave + cq * NWAVE;   // row within the tile
            if (nslab > 1) {
              float* ra_ = rowacc + (rl * NW + cw) * B;
#pragma unroll
              for (int i = 0; i < B; ++i) {
                const float prev = (s == 0) ? 0.f : ra_[i];
                v[i] += prev;
              }
              if (s < nslab - 1) {
                if (lane == 0) {
#pragma unroll
                  for (int i = 0; i < B; ++i) ra_[i] = v[i];
                }
              }
            }
            if (s == nslab - 1) {
              if (NW == 2 && cw == 0) {
#pragma unroll
                for (int i = 0; i < B; ++i) v0[i] = v[i];
              } else {
                // Epilogue for output row r.
                const int r = ra + rl;
                if (lane == 0) {
#pragma unroll
                  for (int i = 0; i < B; ++i) {
                    if (i >= p.b) break;
                    float y = v[i];
                    switch (op) {
                      case FM_OP_QKV:
                        st_tag(p.act + p.off_qkv + (u32)l * p.st_qkv + (u32)i * nqkv + r, y, p.epoch);
                        if (p.taps) p.taps[((size_t)l * p.b + i) * p.tap_block + p.tap_qkv + r] = y;
                        break;
                      case FM_OP_OPROJ:
                        y += resid[i * nr + rl];
                        st_tag(p.act + p.off_x1 + (u32)l * p.st_x1 + (u32)i * p.h + r, y, p.epoch);
                        if (p.taps) p.taps[((size_t)l * p.b + i) * p.tap_block + p.tap_x1 + r] = y;
                        break;
                      case FM_OP_GU:
                        y = silu(v0[i]) * v[i];
                        st_tag(p.act + p.off_m + (u32)l * p.st_m + (u32)i * p.inter + r, y, p.epoch);
                        break;
                      case FM_OP_DOWN: {
                        const float xr = y + resid[i * nr + rl];
                        st_tag(p.act + p.off_x + (u32)(l + 1) * p.st_x + (u32)i * p.h + r, xr, p.epoch);
                        if (p.taps) {
                          p.taps[((size_t)l * p.b + i) * p.tap_block + p.tap_mlp + r] = y;
                          p.taps[((size_t)l * p.b + i) * p.tap_block + p.tap_x2 + r] = xr;
                        }
                        break;
                      }
                      default:
                        if (p.logits) __builtin_nontemporal_store(y, p.logits + (size_t)i * p.V + r);
                        break;
                    }
                  }
                }
                if (op == FM_OP_LM) {
#pragma unroll
                  for (int i = 0; i < B; ++i) {
                    if (best_i[i] < 0 || v[i] > best_v[i]) { best_v[i] = v[i]; best_i[i] = r; }
                  }
                }
              }
            }
          }
          if (++csg == nseg) { csg = 0; if (++cw == NW) { cw = 0; ++cq; } }
        }
      }
    }
  }

  // 4. LM head: merge the waves' argmax candidates, publish one packed key per lane, and
  //    let the last LM tile of the step write the greedy tokens.
  if (op == FM_OP_LM) {
    float* cand_v = misc + 16;            // [NWAVE][B]
    int* cand_i = reinterpret_cast<int*>(misc + 16 + NWAVE * 8);
    __syncthreads();
    if (lane == 0) {
#pragma unroll
      for (int i = 0; i < B; ++i) { cand_v[wave * B + i] = best_v[i]; cand_i[wave * B + i] = best_i[i]; }
    }
    __syncthreads();
    if (tid == 0) {
      u64 sink = 0;
      for (int i = 0; i < p.b; ++i) {
        float bv = 0.f; int bi = -1;
        for (int w = 0; w < NWAVE; ++w) {
          const int ci = cand_i[w * B + i];
          const float cv = cand_v[w * B + i];
          if (ci < 0) continue;
          if (bi < 0 || cv > bv || (cv == bv && ci < bi)) { bv = cv; bi = ci; }
        }
        if (bi >= 0) {
          const u64 key = ((u64)ordered(bv) << 32) | (u64)(0xFFFFFFFFu - (u32)bi);
          sink += __hip_atomic_fetch_max(p.amax + i, key, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
      }
      vm_wait0();
      const u32 old = __hip_atomic_fetch_add(p.lm_arrive, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (old + (u32)(sink == 1234567ull) == (u32)p.n_lm_instr - 1u) {
        for (int i = 0; i < p.b; ++i) {
          const u64 key = __hip_atomic_load(p.amax + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          p.next_ids[i] = (int32_t)(0xFFFFFFFFu - (u32)(key & 0xFFFFFFFFull));
          __hip_atomic_store(p.amax + i, (u64)0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        __hip_atomic_store(p.lm_arrive, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
  }
  __syncthreads();   // LDS is reused by the next instruction
  return true;
}

// ---- attention work items ---------------------------------------------------------------
//
// Per layer the step has P work items. At run time item j maps, from kv_lens alone, to a
// lane i, a KV head g and a chunk [t0, t1) of that lane's slots 0..kv_len: every
// (lane, KV head) gets ceil((kv_len+1)/T) chunks of at most T slots, with T chosen so the
// total chunk count fits in P. Ragged lanes are thus balanced per step. An item reads its
// group's raw q (G heads), k and v and applies QK-norm and RoPE. The item holding the last
// chunk also rounds the new k/v to bf16 and appends them at slot kv_len. The item then
// runs an online softmax over its slots (base-2 exponent with log2(e)/sqrt(d) folded into
// q) and publishes one partial (max, sum, weighted V) per head. The last item of a
// (lane, KV head) to arrive merges the partials in chunk order and writes the attention
// output.

__device__ __forceinline__ bool item_map(const Params& p, int j, int& i, int& g, int& c, int& nc,
                                         int& t0, int& t1) {
  long long total = 0;
  for (int ii = 0; ii < p.b; ++ii) total += p.kvl[ii] + 1;
  total *= p.nkv;
  const long long denom = p.P - p.nkv * p.b;
  const int T = (int)((total + denom - 1) / denom);
  int idx = j;
  for (int ii = 0; ii < p.b; ++ii) {
    const int W = p.kvl[ii] + 1;
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

__device__ __forceinline__ void sm_merge(float& m, float& l, float* acc, float mo, float lo, const float* acco) {
  const float mn = fmaxf(m, mo);
  const float a = (m == -INFINITY) ? 0.f : exp2f(m - mn);
  const float b = (mo == -INFINITY) ? 0.f : exp2f(mo - mn);
  l = l * a + lo * b;
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] = acc[e] * a + acco[e] * b;
  m = mn;
}

template <int D, int GT>
__device__ bool op_attn(const Params& p, const int32_t* ins, float* smem, int tid, int lane, int wave) {
  const int l = ins[1], j = ins[2];
  int i, g, c, nc, t0, t1;
  if (!item_map(p, j, i, g, c, nc, t0, t1)) return true;
  const int G = p.G;
  const int kvl = p.kvl[i];
  const bool is_last = (t1 == kvl + 1);
  const int t_end = min(t1, kvl);            // slots [t0, t_end) come from the arena
  constexpr int LPS = D / 8, SPW = 64 / LPS, SPP = SPW * NWAVE, NPF = 4;
  const int ssl = lane / LPS, de = (lane % LPS) * 8;
  const LayerPtrs& Lw = p.layers[l];
  const u32 arena_bytes = (u32)p.b * (u32)p.nkv * (u32)p.max_ctx * (u32)D * 2u;
  const __amdgpu_buffer_rsrc_t rk = rsrc(Lw.kc, arena_bytes);
  const __amdgpu_buffer_rsrc_t rv = rsrc(Lw.vc, arena_bytes);
  const u32 head_slot0 = ((u32)i * p.nkv + (u32)g) * (u32)p.max_ctx;

  // Prefetch the first NPF passes of K/V (they do not depend on this step's q).
  u32x4 kr[NPF], vr[NPF];
  auto issue = [&](int slot, int pass) {
    const int t = t0 + pass * SPP + wave * SPW + ssl;
    const u32 off = (t < t_end) ? ((head_slot0 + (u32)t) * (u32)D + (u32)de) * 2u : 0xFFFFFFF0u;
    kr[slot] = __builtin_amdgcn_raw_buffer_load_b128(rk, off, 0, CPOL_NT);
    vr[slot] = __builtin_amdgcn_raw_buffer_load_b128(rv, off, 0, CPOL_NT);
  };
#pragma unroll
  for (int s = 0; s < NPF; ++s) issue(s, s);

  float* qs = smem;                 // [G][D]
  float* ks = qs + GT * D;          // [D]
  float* vs = ks + D;               // [D]
  float* wst = vs + D;              // [NWAVE][GT][D + 2]
  float* misc = wst + NWAVE * GT * (D + 2);

  // Wait for this group's q heads, k and v.
  const __amdgpu_buffer_rsrc_t ract = rsrc(p.act, p.act_bytes);
  const u32 base = p.off_qkv + (u32)l * p.st_qkv + (u32)i * (u32)((p.nh + 2 * p.nkv) * D);
  float dummy = 0.f;
  bool ok = wait_copy(p, ract, base + (u32)(g * G * D), G * D, qs, dummy, tid);
  if (ok) ok = wait_copy(p, ract, base + (u32)(p.nh * D + g * D), D, ks, dummy, tid);
  if (ok) ok = wait_copy(p, ract, base + (u32)((p.nh + p.nkv) * D + g * D), D, vs, dummy, tid);
  if (__syncthreads_or(!ok)) return false;

  // Per-head RMSNorm on q and k (Qwen3-shaped models), then RoPE.
  if (p.qk_norm) {
    for (int hh = wave; hh <= G; hh += NWAVE) {
      float* v = (hh < G) ? qs + hh * D : ks;
      const uint16_t* gn = (hh < G) ? Lw.q_norm : Lw.k_norm;
      float ss = 0.f;
      for (int e = lane; e < D; e += 64) ss += v[e] * v[e];
      ss = wave_sum(ss);
      const float r = 1.0f / sqrtf(ss / (float)D + p.eps);
      for (int e = lane; e < D; e += 64) v[e] = v[e] * r * __uint_as_float((u32)gn[e] << 16);
    }
    __syncthreads();
  }
  {
    const int half = D / 2;
    const float* rt = p.rope + (size_t)p.pos[i] * half * 2;
    for (int u = tid; u < (G + 1) * half; u += NT) {
      const int hh = u / half, e = u % half;
      float* v = (hh < G) ? qs + hh * D : ks;
      const float cs = rt[e * 2], sn = rt[e * 2 + 1];
      const float a = v[e], b = v[e + half];
      v[e] = a * cs - b * sn;
      v[e + half] = b * cs + a * sn;
    }
  }
  __syncthreads();
  if (p.taps) {
    float* tb = p.taps + ((size_t)l * p.b + i) * p.tap_block;
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
  }
  __syncthreads();

  float qr[GT][8];
#pragma unroll
  for (int h = 0; h < GT; ++h)
#pragma unroll
    for (int e = 0; e < 8; ++e) qr[h][e] = (h < G) ? qs[h * D + de + e] * p.q_scale : 0.f;
  float m[GT], ls[GT], acc[GT][8];
#pragma unroll
  for (int h = 0; h < GT; ++h) {
    m[h] = -INFINITY; ls[h] = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[h][e] = 0.f;
  }
  auto update = [&](const float* kf, const float* vf, bool valid) {
#pragma unroll
    for (int h = 0; h < GT; ++h) {
      float s = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) s = fmaf(qr[h][e], kf[e], s);
#pragma unroll
      for (int o = 1; o < LPS; o <<= 1) s += __shfl_xor(s, o, 64);
      if (valid && h < G) {
        const float mn = fmaxf(m[h], s);
        const float a = (m[h] == -INFINITY) ? 0.f : exp2f(m[h] - mn);
        const float pe = exp2f(s - mn);
        ls[h] = ls[h] * a + pe;
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[h][e] = fmaf(pe, vf[e], acc[h][e] * a);
        m[h] = mn;
      }
    }
  };
  const int n_arena = t_end - t0;
  const int npass = n_arena > 0 ? (n_arena + SPP - 1) / SPP : 0;
  for (int pb = 0; pb < npass; pb += NPF) {
#pragma unroll
    for (int sl = 0; sl < NPF; ++sl) {
      const int pass = pb + sl;
      if (pass < npass) {
        const u32x4 kw = kr[sl], vw = vr[sl];
        issue(sl, pass + NPF);
        const int t = t0 + pass * SPP + wave * SPW + ssl;
        const float kf[8] = {bf16lo(kw.x), bf16hi(kw.x), bf16lo(kw.y), bf16hi(kw.y),
                             bf16lo(kw.z), bf16hi(kw.z), bf16lo(kw.w), bf16hi(kw.w)};
        const float vf[8] = {bf16lo(vw.x), bf16hi(vw.x), bf16lo(vw.y), bf16hi(vw.y),
                             bf16lo(vw.z), bf16hi(vw.z), bf16lo(vw.w), bf16hi(vw.w)};
        update(kf, vf, t < t_end);
      }
    }
  }
  if (is_last && wave == 0) {
    float kf[8], vf[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) { kf[e] = ks[de + e]; vf[e] = vs[de + e]; }
    update(kf, vf, ssl == 0);
  }
  // Merge the slot groups of the wave (lanes with equal dims, different slots).
#pragma unroll
  for (int o = LPS; o < 64; o <<= 1) {
#pragma unroll
    for (int h = 0; h < GT; ++h) {
      const float mo = __shfl_xor(m[h], o, 64), lo = __shfl_xor(ls[h], o, 64);
      float ao[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) ao[e] = __shfl_xor(acc[h][e], o, 64);
      sm_merge(m[h], ls[h], acc[h], mo, lo, ao);
    }
  }
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
  __syncthreads();
  // Merge the waves in order and publish this chunk's partial for each head.
  const int nh = p.nh;
  for (int u = tid; u < G * D; u += NT) {
    const int h = u / D, e = u % D;
    float M = -INFINITY;
    for (int w = 0; w < NWAVE; ++w) M = fmaxf(M, wst[(w * GT + h) * (D + 2) + D]);
    float Lsum = 0.f, A = 0.f;
    for (int w = 0; w < NWAVE; ++w) {
      const float* ws = wst + (w * GT + h) * (D + 2);
      const float f = (ws[D] == -INFINITY) ? 0.f : exp2f(ws[D] - M);
      Lsum += ws[D + 1] * f;
      A += ws[e] * f;
    }
    float* dst = p.part + (((size_t)i * nh + g * G + h) * p.maxc + c) * (D + 2);
    st_dev(dst + e, A);
    if (e == 0) { st_dev(dst + D, M); st_dev(dst + D + 1, Lsum); }
  }
  vm_wait0();
  __syncthreads();
  u32* arr = p.arrive + i * p.nkv + g;
  int* flag = reinterpret_cast<int*>(misc);
  if (tid == 0) {
    const u32 old = __hip_atomic_fetch_add(arr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    flag[0] = (old == (u32)nc - 1u);
    if (flag[0]) {
      __hip_atomic_store(arr, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      vm_wait0();
    }
  }
  __syncthreads();
  if (flag[0]) {
    // Last arriver: log-sum-exp merge of the chunks in chunk order.
    const u32 obase = p.off_o + (u32)l * p.st_o + (u32)i * (u32)(nh * D);
    for (int u = tid; u < G * D; u += NT) {
      const int h = u / D, e = u % D;
      const float* src = p.part + ((size_t)i * nh + g * G + h) * p.maxc * (D + 2);
      float M = -INFINITY;
      for (int cc = 0; cc < nc; ++cc) M = fmaxf(M, ld_dev(src + cc * (D + 2) + D));
      float den = 0.f, num = 0.f;
      for (int cc = 0; cc < nc; ++cc) {
        const float* pc = src + cc * (D + 2);
        const float f = exp2f(ld_dev(pc + D) - M);
        den += f * ld_dev(pc + D + 1);
        num += f * ld_dev(pc + e);
      }
      const float o = num / den;
      st_tag(p.act + obase + (u32)((g * G + h) * D + e), o, p.epoch);
      if (p.taps) p.taps[((size_t)l * p.b + i) * p.tap_block + p.tap_o + (g * G + h) * D + e] = o;
    }
  }
  __syncthreads();
  return true;
}

}  // namespace dev
}  // namespace fm
