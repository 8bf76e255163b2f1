// The decode-step library's C ABI: handle creation, the single-launch step, the multi-launch
// ablation (the same kernel launched once per stage = one operator of one layer), taps and
// the instruction timeline. The kernels are in fm_kernel.h / fm_kernels.hip.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/fm.h"
#include "fm_kernel.h"
#include "fm_plan.h"

using namespace fm;
using namespace fm::dev;

// Fixed device scratch of fm_decode_step_noalloc: the step's tagged activation words, split-KV
// partials, argmax words, LM-head arrival counter and chunk claim counters, in place of the
// handle's own. Every GPU
// the library runs on holds one copy until the process ends. Host code never passes `scratch`
// itself to a kernel (in host code the name is a host-side stand-in): it uses the per-device
// address from hipGetSymbolAddress, kept in g_scratch[].
static __device__ __align__(256) unsigned char scratch[FM_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices] = {};    // device address of `scratch`, per device
u32 g_scratch_epoch[kMaxDevices] = {};  // step epoch shared by every handle using that copy

// Looks up this device's copy of `scratch` once (the device must be current). Returns null
// on failure.
void* scratch_address(int dev) {
  if (dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess) return nullptr;
    g_scratch[dev] = ptr;
  }
  return g_scratch[dev];
}

// Clears the arrival counter, argmax words and claim counters of the fixed scratch before a
// step that uses it (another handle's step may have left other data there). A kernel, not a
// memset, so the call stays capturable.
__global__ void clear_words(u32* w, int n) {
  for (int k = threadIdx.x; k < n; k += blockDim.x) w[k] = 0u;
}

}  // namespace

struct fm_handle {
  fm_model_cfg cfg{};
  int device = 0;
  Plan plan;
  const void* kernel = nullptr;
  int B = 1;
  Params base{};
  Params* d_params = nullptr;
  Params* d_params_noalloc = nullptr;   // Params with the fixed scratch's buffers; null if it does not fit
  size_t noalloc_bytes = 0;             // bytes of the fixed scratch this handle's steps use
  int noalloc_clear_words = 0;          // leading words of it cleared before each step
  float* taps = nullptr;
  u64* timeline = nullptr;
  LayerPtrs* d_layers = nullptr;
  float* d_rope = nullptr;
  int32_t *d_instrs = nullptr, *d_qoff = nullptr, *d_stage = nullptr;
  u64* d_act = nullptr;
  u64* d_part = nullptr;
  u64* d_amax = nullptr;
  u32* d_lm_arrive = nullptr;
  u32* d_dyn = nullptr;    // claim counters of the dynamic GEMV stages
  u32* d_abort = nullptr;
  uint16_t* d_zero = nullptr;
  u32* h_err = nullptr;   // pinned, device-visible
  u32* d_err = nullptr;
  u32 epoch = 0;
};

namespace {

const void* kernel_for(int Bt, int d, int G) {
  switch (Bt) {
    case 1: return kernel_for_b1(d, G);
    case 2: return kernel_for_b2(d, G);
    case 4: return kernel_for_b4(d, G);
    default: return kernel_for_b8(d, G);
  }
}

int round_batch(int b) { return b <= 1 ? 1 : b <= 2 ? 2 : b <= 4 ? 4 : 8; }

void free_handle(fm_handle* h) {
  if (!h) return;
  hipFree(h->d_layers); hipFree(h->d_rope); hipFree(h->d_instrs); hipFree(h->d_qoff);
  hipFree(h->d_stage); hipFree(h->d_act); hipFree(h->d_part);
  hipFree(h->d_amax); hipFree(h->d_lm_arrive); hipFree(h->d_dyn); hipFree(h->d_abort); hipFree(h->d_params); hipFree(h->d_zero);
  hipFree(h->d_params_noalloc);
  if (h->h_err) hipHostFree(h->h_err);
  delete h;
}

struct TapOff {
  int64_t a, qkv, qrot, krot, o, x1, a2, mlp, x2, block;
};

TapOff tap_offsets(const fm_model_cfg& c) {
  const int64_t h = c.hidden, qd = (int64_t)c.n_heads * c.head_dim, kd = (int64_t)c.n_kv_heads * c.head_dim;
  TapOff t;
  t.a = 0; t.qkv = h; t.qrot = t.qkv + qd + 2 * kd; t.krot = t.qrot + qd; t.o = t.krot + kd;
  t.x1 = t.o + qd; t.a2 = t.x1 + h; t.mlp = t.a2 + h; t.x2 = t.mlp + h; t.block = t.x2 + h;
  return t;
}

#define HIP_TRY(x)                              \
  do {                                          \
    if ((x) != hipSuccess) {                    \
      free_handle(h);                           \
      return FM_ERR_HIP;                        \
    }                                           \
  } while (0)

template <class T>
hipError_t upload(T** dst, const T* src, size_t n) {
  hipError_t e = hipMalloc((void**)dst, sizeof(T) * (n ? n : 1));
  if (e != hipSuccess) return e;
  return n ? hipMemcpy(*dst, src, sizeof(T) * n, hipMemcpyHostToDevice) : hipSuccess;
}

enum class Mode { Single, PerStage, NoAlloc };

fm_status launch(fm_handle* h, const int32_t* tok, const int32_t* pos, const int32_t* kvl,
                 float* logits, int32_t* next_ids, hipStream_t stream, Mode mode) {
  if (!h) return FM_ERR_INVALID_ARG;
  if (!tok || !pos || !kvl || !next_ids) return FM_ERR_INVALID_ARG;
  if (__atomic_load_n(h->h_err, __ATOMIC_ACQUIRE) != 0) return FM_ERR_DEVICE;
  const bool multi = mode == Mode::PerStage;
  const Params* dp = h->d_params;
  u32 epoch = 0;
  if (mode == Mode::NoAlloc) {
    if (!h->d_params_noalloc) return FM_ERR_CAPACITY;
    u32* words = nullptr;
    {
      std::lock_guard<std::mutex> lk(g_scratch_mu);
      words = (u32*)g_scratch[h->device];
      u32& e = g_scratch_epoch[h->device];
      if (++e == 0) e = 1;
      epoch = e;
    }
    // the arrival counter, the argmax words and the claim counters start at zero in every step
    int n_words = h->noalloc_clear_words;
    void* cargs[] = {&words, &n_words};
    if (hipLaunchKernel((const void*)clear_words, dim3(1), dim3(256), cargs, 0, stream) != hipSuccess)
      return FM_ERR_HIP;
    dp = h->d_params_noalloc;
  } else {
    if (++h->epoch == 0) h->epoch = 1;
    epoch = h->epoch;
  }
  Step st{};
  st.tok = tok; st.pos = pos; st.kvl = kvl; st.logits = logits; st.next_ids = next_ids;
  st.taps = h->taps; st.timeline = h->timeline; st.epoch = epoch;
  if (!multi) {
    st.stage = -1;
    void* args[] = {&dp, &st};
    if (hipLaunchCooperativeKernel(h->kernel, dim3(h->plan.nwg), dim3(NT), args, 0, stream) != hipSuccess)
      return FM_ERR_HIP;
  } else {
    for (int s = 0; s < h->plan.n_stages; ++s) {
      st.stage = s;
      void* args[] = {&dp, &st};
      if (hipLaunchKernel(h->kernel, dim3(h->plan.nwg), dim3(NT), args, 0, stream) != hipSuccess)
        return FM_ERR_HIP;
    }
  }
  return FM_OK;
}

}  // namespace

extern "C" {

const char* fm_status_string(fm_status s) {
  switch (s) {
    case FM_OK: return "ok";
    case FM_ERR_INVALID_ARG: return "invalid argument";
    case FM_ERR_UNSUPPORTED: return "unsupported shape";
    case FM_ERR_CAPACITY: return "capacity exceeded";
    case FM_ERR_HIP: return "HIP runtime error";
    case FM_ERR_DEVICE: return "device-side error recorded";
  }
  return "unknown status";
}

size_t fm_tap_count(const fm_model_cfg* cfg) {
  if (!cfg) return 0;
  TapOff t = tap_offsets(*cfg);
  return (size_t)cfg->n_layers * cfg->batch * t.block + (size_t)cfg->batch * cfg->hidden;
}

fm_status fm_plan_query(const fm_model_cfg* cfg, int32_t n_cu, fm_plan_stats* out) {
  if (!cfg || !out) return FM_ERR_INVALID_ARG;
  Plan p;
  fm_status st = build_plan(*cfg, n_cu, p, nullptr);
  if (st != FM_OK) return st;
  *out = p.stats;
  return FM_OK;
}

fm_status fm_plan_export(const fm_model_cfg* cfg, int32_t n_cu, int32_t* qoff, int32_t qoff_cap,
                         int32_t* instrs, int32_t instr_cap) {
  if (!cfg || !qoff || !instrs) return FM_ERR_INVALID_ARG;
  Plan p;
  fm_status st = build_plan(*cfg, n_cu, p, nullptr);
  if (st != FM_OK) return st;
  if (qoff_cap < (int32_t)p.qoff.size() || instr_cap < (int32_t)p.instrs.size() * 4) return FM_ERR_CAPACITY;
  std::memcpy(qoff, p.qoff.data(), sizeof(int32_t) * p.qoff.size());
  std::memcpy(instrs, p.instrs.data(), sizeof(Instr) * p.instrs.size());
  return FM_OK;
}

fm_status fm_create(const fm_model_cfg* cfg, const fm_weight_ptrs* w, const fm_kv_ptrs* kv, fm_handle** out) {
  if (out) *out = nullptr;
  if (!cfg || !w || !kv || !out || !w->layers || !kv->k || !kv->v || !w->embed || !w->final_norm)
    return FM_ERR_INVALID_ARG;
  const fm_model_cfg& c = *cfg;
  if (!c.tied_embedding && !w->lm_head) return FM_ERR_INVALID_ARG;
  for (int l = 0; l < c.n_layers; ++l) {
    const fm_layer_weights& L = w->layers[l];
    if (!L.attn_norm || !L.w_q || !L.w_k || !L.w_v || !L.w_o || !L.mlp_norm || !L.w_gate || !L.w_up ||
        !L.w_down || !kv->k[l] || !kv->v[l])
      return FM_ERR_INVALID_ARG;
    if (c.qk_norm && (!L.q_norm || !L.k_norm)) return FM_ERR_INVALID_ARG;
  }
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return FM_ERR_HIP;
  hipDeviceProp_t prop;
  if (hipGetDeviceProperties(&prop, dev) != hipSuccess) return FM_ERR_HIP;
  const int nwg = c.n_workgroups > 0 ? c.n_workgroups : prop.multiProcessorCount;

  fm_handle* h = new fm_handle();
  h->cfg = c;
  h->device = dev;
  fm_status st = build_plan(c, nwg, h->plan, nullptr);
  if (st != FM_OK) { free_handle(h); return st; }
  const Plan& P = h->plan;

  // Capacity: 32-bit buffer offsets (matrices, KV arenas, scratch), LDS tiles.
  const int64_t L = c.n_layers, hd = c.hidden, d = c.head_dim, nh = c.n_heads, nkv = c.n_kv_heads;
  const int64_t inter = c.intermediate, V = c.vocab, b = c.batch;
  const int64_t nqkv = (nh + 2 * nkv) * d;
  const int64_t biggest = std::max({V * hd, nqkv * hd, inter * hd, hd * nh * d}) * 2;
  const int64_t arena = b * nkv * (int64_t)c.max_ctx * d * 2;
  const int64_t words = (L + 1) * b * hd + L * b * (nqkv + nh * d + hd + inter);
  h->B = round_batch(c.batch);
  const int Bt = h->B;
  if (biggest >= (1ll << 31) || arena >= (1ll << 31) || words * 8 >= (1ll << 32)) { free_handle(h); return FM_ERR_CAPACITY; }
  {
    // Per-tile LDS needs: residual rows, and per-row partials when K spans several slabs.
    auto rows_max = [&](int64_t n) { return (n + nwg - 1) / nwg; };
    if (rows_max(hd) * Bt > RESID_FLOATS) { free_handle(h); return FM_ERR_CAPACITY; }
    const int64_t rowacc_cap = Bt >= 4 ? rowacc_floats<4>() : rowacc_floats<1>();
    // The row sums of a tile, [KP][rows][nw][B], must fit with one K part at least (the
    // kernel uses more parts only while they fit).
    auto needs = [&](int64_t rows, int nw) { return rows_max(rows) * nw * Bt; };
    if (needs(nqkv, 1) > rowacc_cap || needs(hd, 1) > rowacc_cap || needs(inter, 2) > rowacc_cap ||
        needs(V, 1) > rowacc_cap) {
      free_handle(h);
      return FM_ERR_CAPACITY;
    }
  }
  // The group merge stages one group's partials in LDS: G heads x chunks x (d + 2) floats.
  if ((nh / nkv) * (int64_t)P.attn_max_chunks * (d + 2) > kMergeFloats) { free_handle(h); return FM_ERR_CAPACITY; }
  h->kernel = kernel_for(Bt, (int)d, (int)(nh / nkv));
  if (!h->kernel) { free_handle(h); return FM_ERR_UNSUPPORTED; }
  int occ = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, h->kernel, NT, 0) != hipSuccess) { free_handle(h); return FM_ERR_HIP; }
  if ((int64_t)occ * prop.multiProcessorCount < nwg) { free_handle(h); return FM_ERR_CAPACITY; }

  // Weight pointer table.
  std::vector<LayerPtrs> lp(L);
  for (int l = 0; l < L; ++l) {
    const fm_layer_weights& s = w->layers[l];
    lp[l] = LayerPtrs{(const uint16_t*)s.attn_norm, (const uint16_t*)s.w_q, (const uint16_t*)s.w_k,
                      (const uint16_t*)s.w_v, (const uint16_t*)s.q_norm, (const uint16_t*)s.k_norm,
                      (const uint16_t*)s.w_o, (const uint16_t*)s.mlp_norm, (const uint16_t*)s.w_gate,
                      (const uint16_t*)s.w_up, (const uint16_t*)s.w_down, (uint16_t*)kv->k[l],
                      (uint16_t*)kv->v[l]};
  }
  HIP_TRY(upload(&h->d_layers, lp.data(), lp.size()));
  // Rotary table: angle pos * theta^(-2e/d) in double, cos/sin rounded to fp32.
  {
    const int half = (int)d / 2;
    std::vector<float> rt((size_t)c.max_ctx * half * 2);
    for (int ps = 0; ps < c.max_ctx; ++ps)
      for (int e = 0; e < half; ++e) {
        const double ang = (double)ps * std::pow(c.rope_theta, -2.0 * (double)e / (double)d);
        rt[((size_t)ps * half + e) * 2] = (float)std::cos(ang);
        rt[((size_t)ps * half + e) * 2 + 1] = (float)std::sin(ang);
      }
    HIP_TRY(upload(&h->d_rope, rt.data(), rt.size()));
  }
  HIP_TRY(upload(&h->d_instrs, (const int32_t*)P.instrs.data(), P.instrs.size() * 4));
  HIP_TRY(upload(&h->d_qoff, P.qoff.data(), P.qoff.size()));
  HIP_TRY(upload(&h->d_stage, P.stage_rng.data(), P.stage_rng.size()));
  HIP_TRY(hipMalloc(&h->d_act, words * 8));
  HIP_TRY(hipMemset(h->d_act, 0, words * 8));
  const size_t part_words = (size_t)L * b * nh * P.attn_max_chunks * (d + 2);
  if (part_words * 8 >= (1ull << 32)) { free_handle(h); return FM_ERR_CAPACITY; }
  HIP_TRY(hipMalloc(&h->d_part, part_words * 8));
  HIP_TRY(hipMemset(h->d_part, 0, part_words * 8));
  HIP_TRY(hipMalloc(&h->d_amax, b * 8));
  HIP_TRY(hipMemset(h->d_amax, 0, b * 8));
  HIP_TRY(hipMalloc(&h->d_lm_arrive, 64));
  HIP_TRY(hipMemset(h->d_lm_arrive, 0, 64));
  // One counter per (GEMV stage, pool); each pool's counters on their own 128-byte lines.
  const int32_t dyn_stride = ((4 * (int32_t)L + 1) + 31) / 32 * 32;
  const size_t dyn_bytes = (size_t)kPools * dyn_stride * 4;
  HIP_TRY(hipMalloc(&h->d_dyn, dyn_bytes));
  HIP_TRY(hipMemset(h->d_dyn, 0, dyn_bytes));
  HIP_TRY(hipMalloc(&h->d_zero, 65536));
  HIP_TRY(hipMemset(h->d_zero, 0, 65536));
  HIP_TRY(hipMalloc(&h->d_abort, 64));
  HIP_TRY(hipMemset(h->d_abort, 0, 64));
  HIP_TRY(hipHostMalloc((void**)&h->h_err, 64, hipHostMallocMapped));
  std::memset(h->h_err, 0, 64);
  HIP_TRY(hipHostGetDevicePointer((void**)&h->d_err, h->h_err, 0));

  Params& p = h->base;
  p.L = (int32_t)L; p.h = (int32_t)hd; p.nh = (int32_t)nh; p.nkv = (int32_t)nkv; p.d = (int32_t)d;
  p.inter = (int32_t)inter; p.V = (int32_t)V; p.b = (int32_t)b; p.max_ctx = c.max_ctx;
  p.qk_norm = c.qk_norm; p.G = (int32_t)(nh / nkv);
  p.nwg = nwg; p.P = P.attn_items; p.maxc = P.attn_max_chunks; p.n_lm_instr = P.n_lm_instr;
  p.eps = (float)c.rms_eps;
  p.q_scale = (float)(1.4426950408889634 / std::sqrt((double)d));
  p.layers = h->d_layers;
  p.embed = (const uint16_t*)w->embed;
  p.final_norm = (const uint16_t*)w->final_norm;
  p.lm_head = (const uint16_t*)(c.tied_embedding ? w->embed : w->lm_head);
  p.rope = h->d_rope;
  p.instrs = h->d_instrs; p.qoff = h->d_qoff; p.stage_rng = h->d_stage;
  p.act = h->d_act; p.act_bytes = (u32)(words * 8);
  p.st_x = (u32)(b * hd); p.st_qkv = (u32)(b * nqkv); p.st_o = (u32)(b * nh * d);
  p.st_x1 = (u32)(b * hd); p.st_m = (u32)(b * inter);
  p.off_x = 0;
  p.off_qkv = p.off_x + (u32)(L + 1) * p.st_x;
  p.off_o = p.off_qkv + (u32)L * p.st_qkv;
  p.off_x1 = p.off_o + (u32)L * p.st_o;
  p.off_m = p.off_x1 + (u32)L * p.st_x1;
  p.zero_page = h->d_zero;
  p.part = h->d_part; p.amax = h->d_amax; p.lm_arrive = h->d_lm_arrive;
  p.dyn_ctr = h->d_dyn; p.dyn_stride = dyn_stride;
  p.abort_flag = h->d_abort; p.err_host = h->d_err;
  const TapOff t = tap_offsets(c);
  p.tap_block = t.block;
  p.tap_a = (int32_t)t.a; p.tap_qkv = (int32_t)t.qkv; p.tap_qrot = (int32_t)t.qrot; p.tap_krot = (int32_t)t.krot;
  p.tap_o = (int32_t)t.o; p.tap_x1 = (int32_t)t.x1; p.tap_a2 = (int32_t)t.a2; p.tap_mlp = (int32_t)t.mlp;
  p.tap_x2 = (int32_t)t.x2;
  HIP_TRY(upload(&h->d_params, &h->base, 1));
  {
    // The same parameters over the fixed scratch, for fm_decode_step_noalloc:
    // [arrival counter: 256 B][argmax words: 256 B][claim counters][activation words][split-KV
    // partials]. Everything before the activation words is cleared before each such step.
    const size_t dyn_off = 512, act_off = dyn_off + ((dyn_bytes + 255) & ~(size_t)255);
    const size_t part_off = act_off + (((size_t)words * 8 + 255) & ~(size_t)255);
    h->noalloc_clear_words = (int)(act_off / 4);
    const size_t need = part_off + part_words * 8;
    h->noalloc_bytes = need;
    void* base = scratch_address(dev);
    if (!base) { free_handle(h); return FM_ERR_HIP; }
    if (need <= (size_t)FM_NOALLOC_SCRATCH_BYTES) {
      Params q = h->base;
      unsigned char* b8 = (unsigned char*)base;
      q.lm_arrive = (u32*)b8;
      q.amax = (u64*)(b8 + 256);
      q.dyn_ctr = (u32*)(b8 + dyn_off);
      q.act = (u64*)(b8 + act_off);
      q.part = (u64*)(b8 + part_off);
      HIP_TRY(upload(&h->d_params_noalloc, &q, 1));
    }
  }
  *out = h;
  return FM_OK;
}

fm_status fm_decode_step(fm_handle* h, const int32_t* token_ids, const int32_t* positions,
                         const int32_t* kv_lens, float* logits_out, int32_t* next_ids, hipStream_t stream) {
  return launch(h, token_ids, positions, kv_lens, logits_out, next_ids, stream, Mode::Single);
}

fm_status fm_decode_step_multilaunch(fm_handle* h, const int32_t* token_ids, const int32_t* positions,
                                     const int32_t* kv_lens, float* logits_out, int32_t* next_ids,
                                     hipStream_t stream) {
  return launch(h, token_ids, positions, kv_lens, logits_out, next_ids, stream, Mode::PerStage);
}

fm_status fm_decode_step_noalloc(fm_handle* h, const int32_t* token_ids, const int32_t* positions,
                                 const int32_t* kv_lens, float* logits_out, int32_t* next_ids,
                                 hipStream_t stream) {
  return launch(h, token_ids, positions, kv_lens, logits_out, next_ids, stream, Mode::NoAlloc);
}

size_t fm_noalloc_scratch_bytes(const fm_handle* h) { return h ? h->noalloc_bytes : 0; }

fm_status fm_extend(fm_handle* h, const int32_t* token_ids, const int32_t* positions, const int32_t* kv_lens,
                    int32_t n_tokens, float* logits_out, int32_t* next_ids, hipStream_t stream) {
  if (!h || !token_ids || !positions || !kv_lens || !next_ids || n_tokens < 0) return FM_ERR_INVALID_ARG;
  const size_t b = (size_t)h->base.b;
  for (int32_t t = 0; t < n_tokens; ++t) {
    const size_t r = (size_t)t * b;
    const fm_status s = launch(h, token_ids + r, positions + r, kv_lens + r,
                               t + 1 == n_tokens ? logits_out : nullptr, next_ids, stream, Mode::Single);
    if (s != FM_OK) return s;
  }
  return FM_OK;
}

fm_status fm_destroy(fm_handle* h) {
  if (!h) return FM_ERR_INVALID_ARG;
  hipDeviceSynchronize();
  free_handle(h);
  return FM_OK;
}

fm_status fm_last_error(fm_handle* h, int32_t* device_code) {
  if (!h || !device_code) return FM_ERR_INVALID_ARG;
  if (hipDeviceSynchronize() != hipSuccess) return FM_ERR_HIP;
  *device_code = (int32_t)__atomic_load_n(h->h_err, __ATOMIC_ACQUIRE);
  return *device_code ? FM_ERR_DEVICE : FM_OK;
}

fm_status fm_set_timeline(fm_handle* h, uint64_t* buf) {
  if (!h) return FM_ERR_INVALID_ARG;
  h->timeline = buf;
  return FM_OK;
}

int32_t fm_instruction_count(const fm_handle* h) { return h ? (int32_t)h->plan.instrs.size() : -1; }

fm_status fm_set_taps(fm_handle* h, float* tap_buf) {
  if (!h) return FM_ERR_INVALID_ARG;
  h->taps = tap_buf;
  return FM_OK;
}

}  // extern "C"
