// Reference decoder for one transformer decode step: TEST INFRASTRUCTURE ONLY.
//
// This file is the plain, slow CPU oracle the GPU library is checked against. Only the
// test-suite, the smoke check and the CPU-baseline leg of the benchmark may load it; the
// product path never calls it. It shares no code, header, table or constant generator
// with the GPU library.
//
// What it computes (arXiv 2609.12379, Sec. 2.1 "The decode step", Eq. 1): per lane and
// per layer, RMSNorm -> Q/K/V projections -> (optional per-head QK-RMSNorm) -> RoPE ->
// append the new K/V to the cache -> grouped-query attention over the cache (Eq. 1) ->
// O projection + residual -> RMSNorm -> gate/up -> SiLU * up -> down + residual; then a
// final RMSNorm, the LM head and a greedy argmax.
//
// Precision (the paper's precision contract, Sec. 4.2, keeps accumulators, norm gains and
// the rotary table at fp32 or wider; where it is silent this file takes the following
// reading): weights and the KV cache are bf16 storage, upcast exactly; every other value
// is held in the arithmetic type T; the new token's K/V are rounded to bf16 (round to
// nearest even) when appended, and attention reads them back as stored. T = float is the
// oracle proper; T = double is the float64 instantiation (the paper's golden forward
// pass, Sec. 4.2) used to bound the oracle's own rounding.
//
// Every loop runs in the order the definition states: sequential sums over the
// contraction index, no blocking, no reassociation. OpenMP splits only independent
// output rows and independent heads.
//
// Readings where the paper is silent (each listed in the design notes):
//   * RMSNorm: y = x / sqrt(mean(x^2) + eps) * g, eps inside the square root.
//   * RoPE: rotate-half pairing (j, j + d/2), inv_freq_j = theta^(-2j/d); the angle
//     pos * inv_freq_j is formed in float64 and cos/sin are rounded to T.
//   * QK-norm (Qwen3-shaped models): per-head RMSNorm over head_dim with gains [head_dim]
//     shared by all heads, applied after the projection and before RoPE.
//   * GQA head map g(j) = floor(j / (n_heads / n_kv_heads)).
//   * Attention covers slots 0..kv_len inclusive: the kv_len cached tokens plus the new one.
//   * SiLU(z) = z / (1 + exp(-z)).
//   * Greedy argmax returns the lowest index among equal maxima.

#include <cmath>
#include <cstdint>
#include <cstring>
#include <vector>
#include <limits>

namespace {

struct Cfg {
  int32_t n_layers, hidden, n_heads, n_kv_heads, head_dim, intermediate, vocab;
  int32_t qk_norm, tied_embedding, batch, max_ctx, reserved;
  double rope_theta, rms_eps;
};

struct Layer {
  const uint16_t *attn_norm, *wq, *wk, *wv, *q_norm, *k_norm, *wo, *mlp_norm, *wg, *wu, *wd;
};

struct Weights {
  const uint16_t* embed;
  const uint16_t* final_norm;
  const uint16_t* lm_head;
  const Layer* layers;
};

// ---- bf16 storage ---------------------------------------------------------------------

float bf16_to_float(uint16_t h) {
  uint32_t u = (uint32_t)h << 16;
  float f;
  std::memcpy(&f, &u, 4);
  return f;
}

template <class T> T up(uint16_t h) { return (T)bf16_to_float(h); }

// Round a float to the nearest bf16, ties to even. NaN stays a (quiet) NaN.
uint16_t bf16_from_float(float f) {
  uint32_t u;
  std::memcpy(&u, &f, 4);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x0040u);
  uint32_t lsb = (u >> 16) & 1u;
  u += 0x7fffu + lsb;
  return (uint16_t)(u >> 16);
}

// Round a double to the nearest bf16 directly (no intermediate float rounding), ties to
// even. Within float's normal range bf16 keeps 8 significant bits, so this rounds the
// 53-bit significand at bit 45. Below float's normal range it falls back to the float
// path (values there never occur in the decode step).
uint16_t bf16_from_double(double d) {
  if (std::isnan(d)) return bf16_from_float((float)d);
  double a = std::fabs(d);
  if (a < 1.1754943508222875e-38) return bf16_from_float((float)d);
  uint64_t u;
  std::memcpy(&u, &d, 8);
  const uint64_t half = (1ull << 44);
  uint64_t lsb = (u >> 45) & 1ull;
  u += (half - 1ull) + lsb;
  u &= ~((1ull << 45) - 1ull);
  double r;
  std::memcpy(&r, &u, 8);
  // r is now a bf16 value or beyond bf16's range; the float conversion is exact or
  // overflows to infinity as bf16 would.
  float f = (float)r;
  if (std::fabs(r) > 3.3895313892515355e+38) f = std::copysign(std::numeric_limits<float>::infinity(), (float)d);
  uint32_t fu;
  std::memcpy(&fu, &f, 4);
  return (uint16_t)(fu >> 16);
}

uint16_t to_bf16(float v) { return bf16_from_float(v); }
uint16_t to_bf16(double v) { return bf16_from_double(v); }

// ---- operators ------------------------------------------------------------------------

// RMSNorm: out = x / sqrt(mean(x^2) + eps) * g.
template <class T>
void rmsnorm(const T* x, const uint16_t* g, int n, double eps, T* out) {
  T ss = 0;
  for (int k = 0; k < n; ++k) ss += x[k] * x[k];
  T r = T(1) / std::sqrt(ss / T(n) + T(eps));
  for (int k = 0; k < n; ++k) out[k] = x[k] * r * up<T>(g[k]);
}

// y[n] = sum_k W[n][k] * x[k]; W row-major [N][K] bf16.
template <class T>
void gemv(const uint16_t* W, int N, int K, const T* x, T* y) {
#pragma omp parallel for schedule(static)
  for (int n = 0; n < N; ++n) {
    const uint16_t* w = W + (size_t)n * K;
    T acc = 0;
    for (int k = 0; k < K; ++k) acc += up<T>(w[k]) * x[k];
    y[n] = acc;
  }
}

// Rotary embedding, rotate-half form, applied in place to one head vector of length d.
template <class T>
void rope(T* v, int d, int pos, double theta) {
  int half = d / 2;
  for (int j = 0; j < half; ++j) {
    double inv_freq = std::pow(theta, -2.0 * (double)j / (double)d);
    double ang = (double)pos * inv_freq;
    T c = (T)std::cos(ang), s = (T)std::sin(ang);
    T a = v[j], b = v[j + half];
    v[j] = a * c - b * s;
    v[j + half] = b * c + a * s;
  }
}

// Eq. 1 for one query head: softmax(q K^T / sqrt(d)) V over n_slots cached rows.
// Kc, Vc: [n_slots][d] bf16 rows of this head's KV head.
template <class T>
void attend(const T* q, const uint16_t* Kc, const uint16_t* Vc, int n_slots, int d, T* o) {
  std::vector<T> s(n_slots);
  T scale = T(1) / std::sqrt(T(d));
  for (int t = 0; t < n_slots; ++t) {
    T dot = 0;
    for (int e = 0; e < d; ++e) dot += q[e] * up<T>(Kc[(size_t)t * d + e]);
    s[t] = dot * scale;
  }
  T m = s[0];
  for (int t = 1; t < n_slots; ++t) m = s[t] > m ? s[t] : m;
  T l = 0;
  for (int t = 0; t < n_slots; ++t) {
    s[t] = std::exp(s[t] - m);
    l += s[t];
  }
  for (int e = 0; e < d; ++e) {
    T acc = 0;
    for (int t = 0; t < n_slots; ++t) acc += s[t] * up<T>(Vc[(size_t)t * d + e]);
    o[e] = acc / l;
  }
}

template <class T> T silu(T z) { return z / (T(1) + std::exp(-z)); }

// Lowest index among equal maxima; NaN compares false and is never selected over a number.
template <class T>
int32_t argmax(const T* v, int n) {
  int32_t best = 0;
  for (int k = 1; k < n; ++k)
    if (v[k] > v[best]) best = k;
  return best;
}

// ---- tap layout -----------------------------------------------------------------------
// Per layer l and lane i, a block of: a[h] | qkv[(nh+2nkv)d] | q_rot[nh d] | k_rot[nkv d] |
// o[nh d] | x1[h] | a2[h] | mlp[h] | x2[h]. Blocks are laid out [L][b]; after them the
// final normed vector [b][h].
struct TapLayout {
  size_t a, qkv, qrot, krot, o, x1, a2, mlp, x2, block;
};

TapLayout tap_layout(const Cfg& c) {
  size_t h = c.hidden, qd = (size_t)c.n_heads * c.head_dim, kd = (size_t)c.n_kv_heads * c.head_dim;
  TapLayout t;
  t.a = 0;
  t.qkv = t.a + h;
  t.qrot = t.qkv + qd + 2 * kd;
  t.krot = t.qrot + qd;
  t.o = t.krot + kd;
  t.x1 = t.o + qd;
  t.a2 = t.x1 + h;
  t.mlp = t.a2 + h;
  t.x2 = t.mlp + h;
  t.block = t.x2 + h;
  return t;
}

bool cfg_ok(const Cfg& c) {
  if (c.n_layers < 1 || c.hidden < 1 || c.n_heads < 1 || c.n_kv_heads < 1 || c.head_dim < 2 ||
      c.intermediate < 1 || c.vocab < 1 || c.batch < 1 || c.max_ctx < 1)
    return false;
  if (c.n_heads % c.n_kv_heads != 0 || c.head_dim % 2 != 0) return false;
  return true;
}

// One decode step for all lanes. Returns 0 on success, a negative code on bad input
// (nothing is written then).
template <class T>
int decode_step(const Cfg& c, const Weights& w, uint16_t* const* kcache, uint16_t* const* vcache,
                const int32_t* tok, const int32_t* pos, const int32_t* kv_lens, T* logits,
                int32_t* next_ids, T* taps) {
  if (!cfg_ok(c)) return -1;
  for (int i = 0; i < c.batch; ++i) {
    if (tok[i] < 0 || tok[i] >= c.vocab) return -2;
    if (pos[i] < 0) return -3;
    if (kv_lens[i] < 0 || kv_lens[i] >= c.max_ctx) return -4;
  }
  const int h = c.hidden, d = c.head_dim, nh = c.n_heads, nkv = c.n_kv_heads, G = nh / nkv;
  const int inter = c.intermediate;
  const TapLayout tl = tap_layout(c);
  std::vector<T> x(h), a(h), q((size_t)nh * d), k((size_t)nkv * d), v((size_t)nkv * d),
      o((size_t)nh * d), proj(h), gt(inter), upv(inter), m(inter);

  for (int i = 0; i < c.batch; ++i) {
    // Embedding gather: the residual stream starts as the token's embedding row.
    for (int e = 0; e < h; ++e) x[e] = up<T>(w.embed[(size_t)tok[i] * h + e]);
    for (int l = 0; l < c.n_layers; ++l) {
      const Layer& L = w.layers[l];
      T* tp = taps ? taps + ((size_t)l * c.batch + i) * tl.block : nullptr;
      // Attention block.
      rmsnorm(x.data(), L.attn_norm, h, c.rms_eps, a.data());
      gemv(L.wq, nh * d, h, a.data(), q.data());
      gemv(L.wk, nkv * d, h, a.data(), k.data());
      gemv(L.wv, nkv * d, h, a.data(), v.data());
      if (tp) {
        std::memcpy(tp + tl.a, a.data(), sizeof(T) * h);
        std::memcpy(tp + tl.qkv, q.data(), sizeof(T) * nh * d);
        std::memcpy(tp + tl.qkv + (size_t)nh * d, k.data(), sizeof(T) * nkv * d);
        std::memcpy(tp + tl.qkv + (size_t)(nh + nkv) * d, v.data(), sizeof(T) * nkv * d);
      }
      if (c.qk_norm) {
        std::vector<T> tmp(d);
        for (int j = 0; j < nh; ++j) {
          rmsnorm(q.data() + (size_t)j * d, L.q_norm, d, c.rms_eps, tmp.data());
          std::memcpy(q.data() + (size_t)j * d, tmp.data(), sizeof(T) * d);
        }
        for (int g = 0; g < nkv; ++g) {
          rmsnorm(k.data() + (size_t)g * d, L.k_norm, d, c.rms_eps, tmp.data());
          std::memcpy(k.data() + (size_t)g * d, tmp.data(), sizeof(T) * d);
        }
      }
      for (int j = 0; j < nh; ++j) rope(q.data() + (size_t)j * d, d, pos[i], c.rope_theta);
      for (int g = 0; g < nkv; ++g) rope(k.data() + (size_t)g * d, d, pos[i], c.rope_theta);
      if (tp) {
        std::memcpy(tp + tl.qrot, q.data(), sizeof(T) * nh * d);
        std::memcpy(tp + tl.krot, k.data(), sizeof(T) * nkv * d);
      }
      // KV append: slot kv_lens[i] of lane i, every KV head, stored as bf16.
      const int slot = kv_lens[i];
      for (int g = 0; g < nkv; ++g) {
        size_t base = (((size_t)i * nkv + g) * c.max_ctx + slot) * d;
        for (int e = 0; e < d; ++e) {
          kcache[l][base + e] = to_bf16(k[(size_t)g * d + e]);
          vcache[l][base + e] = to_bf16(v[(size_t)g * d + e]);
        }
      }
      // Grouped-query attention over slots 0..kv_len (Eq. 1).
#pragma omp parallel for schedule(static)
      for (int j = 0; j < nh; ++j) {
        int g = j / G;
        size_t base = ((size_t)i * nkv + g) * c.max_ctx * (size_t)d;
        attend(q.data() + (size_t)j * d, kcache[l] + base, vcache[l] + base, slot + 1, d,
               o.data() + (size_t)j * d);
      }
      gemv(L.wo, h, nh * d, o.data(), proj.data());
      for (int e = 0; e < h; ++e) x[e] = x[e] + proj[e];
      if (tp) {
        std::memcpy(tp + tl.o, o.data(), sizeof(T) * nh * d);
        std::memcpy(tp + tl.x1, x.data(), sizeof(T) * h);
      }
      // MLP block.
      rmsnorm(x.data(), L.mlp_norm, h, c.rms_eps, a.data());
      gemv(L.wg, inter, h, a.data(), gt.data());
      gemv(L.wu, inter, h, a.data(), upv.data());
      for (int r = 0; r < inter; ++r) m[r] = silu(gt[r]) * upv[r];
      gemv(L.wd, h, inter, m.data(), proj.data());
      for (int e = 0; e < h; ++e) x[e] = x[e] + proj[e];
      if (tp) {
        std::memcpy(tp + tl.a2, a.data(), sizeof(T) * h);
        std::memcpy(tp + tl.mlp, proj.data(), sizeof(T) * h);
        std::memcpy(tp + tl.x2, x.data(), sizeof(T) * h);
      }
    }
    // Final norm, LM head, greedy token.
    rmsnorm(x.data(), w.final_norm, h, c.rms_eps, a.data());
    if (taps) std::memcpy(taps + (size_t)c.n_layers * c.batch * tl.block + (size_t)i * h, a.data(), sizeof(T) * h);
    const uint16_t* lm = c.tied_embedding ? w.embed : w.lm_head;
    T* lg = logits + (size_t)i * c.vocab;
    gemv(lm, c.vocab, h, a.data(), lg);
    next_ids[i] = argmax(lg, c.vocab);
  }
  return 0;
}

}  // namespace

// ---- exported C entry points (ctypes) ---------------------------------------------------

extern "C" {

size_t fmo_tap_count(const Cfg* c) {
  TapLayout t = tap_layout(*c);
  return (size_t)c->n_layers * c->batch * t.block + (size_t)c->batch * c->hidden;
}

void fmo_tap_offsets(const Cfg* c, int64_t* out10) {
  TapLayout t = tap_layout(*c);
  int64_t v[10] = {(int64_t)t.a, (int64_t)t.qkv, (int64_t)t.qrot, (int64_t)t.krot, (int64_t)t.o,
                   (int64_t)t.x1, (int64_t)t.a2, (int64_t)t.mlp, (int64_t)t.x2, (int64_t)t.block};
  for (int k = 0; k < 10; ++k) out10[k] = v[k];
}

int fmo_decode_step_f32(const Cfg* c, const Weights* w, uint16_t* const* kc, uint16_t* const* vc,
                        const int32_t* tok, const int32_t* pos, const int32_t* kv_lens, float* logits,
                        int32_t* next_ids, float* taps) {
  return decode_step<float>(*c, *w, kc, vc, tok, pos, kv_lens, logits, next_ids, taps);
}

int fmo_decode_step_f64(const Cfg* c, const Weights* w, uint16_t* const* kc, uint16_t* const* vc,
                        const int32_t* tok, const int32_t* pos, const int32_t* kv_lens, double* logits,
                        int32_t* next_ids, double* taps) {
  return decode_step<double>(*c, *w, kc, vc, tok, pos, kv_lens, logits, next_ids, taps);
}

// Single operators, for pinning each one against closed forms.
void fmo_rmsnorm_f32(const float* x, const uint16_t* g, int n, double eps, float* out) { rmsnorm(x, g, n, eps, out); }
void fmo_rmsnorm_f64(const double* x, const uint16_t* g, int n, double eps, double* out) { rmsnorm(x, g, n, eps, out); }
void fmo_gemv_f32(const uint16_t* W, int N, int K, const float* x, float* y) { gemv(W, N, K, x, y); }
void fmo_gemv_f64(const uint16_t* W, int N, int K, const double* x, double* y) { gemv(W, N, K, x, y); }
void fmo_rope_f32(float* v, int d, int pos, double theta) { rope(v, d, pos, theta); }
void fmo_rope_f64(double* v, int d, int pos, double theta) { rope(v, d, pos, theta); }
void fmo_attend_f32(const float* q, const uint16_t* K, const uint16_t* V, int n, int d, float* o) { attend(q, K, V, n, d, o); }
void fmo_attend_f64(const double* q, const uint16_t* K, const uint16_t* V, int n, int d, double* o) { attend(q, K, V, n, d, o); }
void fmo_silu_mul_f32(const float* g, const float* u, int n, float* out) { for (int k = 0; k < n; ++k) out[k] = silu(g[k]) * u[k]; }
void fmo_silu_mul_f64(const double* g, const double* u, int n, double* out) { for (int k = 0; k < n; ++k) out[k] = silu(g[k]) * u[k]; }
int32_t fmo_argmax_f32(const float* v, int n) { return argmax(v, n); }
int32_t fmo_argmax_f64(const double* v, int n) { return argmax(v, n); }
void fmo_to_bf16_f32(const float* v, int64_t n, uint16_t* out) { for (int64_t k = 0; k < n; ++k) out[k] = bf16_from_float(v[k]); }
void fmo_to_bf16_f64(const double* v, int64_t n, uint16_t* out) { for (int64_t k = 0; k < n; ++k) out[k] = bf16_from_double(v[k]); }

}  // extern "C"
