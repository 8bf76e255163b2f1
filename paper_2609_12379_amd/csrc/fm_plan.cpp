// Host-side schedule compiler (see fm_plan.h).
#include "fm_plan.h"
#include "fm_limits.h"

#include <algorithm>
#include <cstdio>

namespace fm {

namespace {

bool fail(std::string* why, const char* msg) {
  if (why) *why = msg;
  return false;
}

bool check_cfg(const fm_model_cfg& c, std::string* why, fm_status* st) {
  *st = FM_ERR_INVALID_ARG;
  if (c.n_layers < 1 || c.hidden < 1 || c.n_heads < 1 || c.n_kv_heads < 1 || c.head_dim < 1 ||
      c.intermediate < 1 || c.vocab < 1 || c.batch < 1 || c.max_ctx < 1 || c.n_workgroups < 0 ||
      c.attn_items < 0 || c.dyn_chunk_kb < -1)
    return fail(why, "dimensions must be positive (n_workgroups, attn_items >= 0, dyn_chunk_kb >= -1)");
  if (c.n_heads % c.n_kv_heads != 0) return fail(why, "n_heads must be a multiple of n_kv_heads");
  if (!(c.rope_theta > 0.0) || !(c.rms_eps >= 0.0)) return fail(why, "rope_theta > 0 and rms_eps >= 0 required");
  *st = FM_ERR_UNSUPPORTED;
  if (c.head_dim != 64 && c.head_dim != 128) return fail(why, "head_dim must be 64 or 128");
  if (c.n_heads / c.n_kv_heads > 8) return fail(why, "n_heads / n_kv_heads must be <= 8");
  if (c.batch > 8) return fail(why, "batch must be <= 8");
  if (c.hidden % 8 || (c.n_heads * c.head_dim) % 8 || c.intermediate % 8)
    return fail(why, "hidden, n_heads*head_dim and intermediate must be multiples of 8");
  return true;
}

// Balanced contiguous split of [0, n) into nwg parts; part w is [lo, hi).
void split(int64_t n, int32_t nwg, int32_t w, int32_t& lo, int32_t& hi) {
  lo = (int32_t)(n * w / nwg);
  hi = (int32_t)(n * (w + 1) / nwg);
}

// Geometry of a GEMV stage in dynamic chunks, or false when the stage stays static: rows
// output rows of K columns, nw weight rows per output row, B the kernel's batch width.
// A chunk gives each of the 8 waves exactly one item: nq row quads times kp K parts = 8, with
// at least kDynMinSegs 128-column segments per part. nq is the smallest power of two whose
// chunk reaches chunk_bytes with at most kDynMaxPerWg chunks per workgroup (or the largest
// allowed).
struct DynGeom {
  int32_t rc, kp, slots;
};

bool dyn_geometry(int64_t rows, int64_t K, int32_t nw, int32_t B, int32_t nwg, int64_t chunk_bytes, DynGeom& g) {
  if (B > 2 || chunk_bytes <= 0) return false;              // matrix-core tiles stay static
  const int64_t kpad = (K + 127) / 128 * 128;
  if (kpad * B > kXslabFloatsVALU) return false;            // one slab holds the whole input
  const int32_t nseg = (int32_t)(kpad / 128);
  int32_t nq = 0;
  for (int32_t q = 1; q <= 8; q *= 2) {
    const int32_t kp = 8 / q;
    if ((nseg + kp - 1) / kp < kDynMinSegs) continue;        // parts too short
    nq = q;
    const int64_t rcq = 4 * q / nw;
    if ((int64_t)4 * q * K * 2 >= chunk_bytes &&              // 4 q weight rows of K columns
        (rows + rcq - 1) / rcq <= (int64_t)kDynMaxPerWg * nwg)
      break;
  }
  if (nq == 0) return false;
  const int32_t rc = 4 * nq / nw;
  const int64_t nch = (rows + rc - 1) / rc;
  if (nch < (int64_t)kDynMinPerWg * nwg) return false;
  const int32_t kp = 8 / nq;
  const int32_t slots = std::min<int32_t>(kDynMaxSlots, kRowaccFloatsVALU / (kp * rc * nw * B));
  if (slots < 2) return false;
  // Every chunk of a pool must fit in its workgroups' slots, whoever takes it.
  const int32_t np = std::min(kPools, nwg);
  for (int32_t x = 0; x < np; ++x) {
    const int64_t nwx = (nwg - x + np - 1) / np;
    const int64_t sx = (int64_t)x * (nwg / np) + std::min<int64_t>(x, nwg % np);
    const int64_t c0 = nch * sx / nwg, c1 = nch * (sx + nwx) / nwg;
    if (c1 - c0 < nwx || c1 - c0 > nwx * slots) return false;
  }
  g.rc = rc;
  g.kp = kp;
  g.slots = slots;
  return true;
}

}  // namespace

fm_status build_plan(const fm_model_cfg& c, int32_t nwg, Plan& p, std::string* why) {
  fm_status st;
  if (!check_cfg(c, why, &st)) return st;
  if (nwg < 1) {
    if (why) *why = "need at least one workgroup";
    return FM_ERR_INVALID_ARG;
  }
  const int32_t L = c.n_layers, h = c.hidden, d = c.head_dim, nh = c.n_heads, nkv = c.n_kv_heads;
  const int32_t inter = c.intermediate, V = c.vocab, b = c.batch;
  const int64_t qkv_rows = (int64_t)(nh + 2 * nkv) * d;

  // Attention work items per layer. Each (lane, KV head) needs at least one item, and the
  // per-step chunking (see the kernel's item map) needs P > n_kv * b.
  // Automatic count: about one item per workgroup (more when there are many (lane, KV head)
  // groups), capped so that one group's chunk partials fit the merge's LDS staging.
  int32_t P = c.attn_items;
  if (P == 0) {
    int32_t need = nkv * b;
    P = nwg;
    if (need > nwg / 2) P = nwg * ((need + nwg + nwg - 1) / nwg);
    const int32_t cap = kMergeFloats / ((nh / nkv) * (d + 2));   // chunks per group
    if (cap >= 1 && P > need + (cap - 1) * nkv) P = need + (cap - 1) * nkv;
    if (P <= need) P = need + 1;
  }
  if (P <= nkv * b) {
    if (why) *why = "attn_items must exceed n_kv_heads * batch";
    return FM_ERR_INVALID_ARG;
  }
  p = Plan();
  p.nwg = nwg;
  p.attn_items = P;
  p.attn_max_chunks = (P - nkv * b) / nkv + 1;
  p.n_stages = 5 * L + 1;

  std::vector<std::vector<Instr>> q(nwg);
  std::vector<double> bytes(nwg, 0.0);
  // The kernel's batch width (lanes rounded up to 1, 2, 4, 8).
  const int32_t Bk = b <= 1 ? 1 : b <= 2 ? 2 : b <= 4 ? 4 : 8;
  int32_t n_dyn = 0;
  const int64_t chunk_bytes = c.dyn_chunk_kb == 0 ? kDynChunkBytes : (int64_t)c.dyn_chunk_kb << 10;
  auto gemv = [&](int32_t op, int32_t l, int64_t rows, int64_t K, int32_t nw) {
    // Dynamic chunks for the QKV, O-projection and down stages; gate/up and the LM head
    // measured slower in chunks than in fixed tiles on MI355X.
    const bool dyn_op = op == FM_OP_QKV || op == FM_OP_OPROJ || op == FM_OP_DOWN;
    DynGeom g;
    if (dyn_op && dyn_geometry(rows, K, nw, Bk, nwg, chunk_bytes, g)) {
      ++n_dyn;
      for (int32_t w = 0; w < nwg; ++w) {
        q[w].push_back(Instr{op, l, -g.rc, g.kp | (g.slots << 8)});
        bytes[w] += (double)rows * K * 2.0 * nw / nwg;
      }
      return;
    }
    for (int32_t w = 0; w < nwg; ++w) {
      int32_t lo, hi;
      split(rows, nwg, w, lo, hi);
      if (hi > lo) {
        q[w].push_back(Instr{op, l, lo, hi});
        bytes[w] += (double)(hi - lo) * K * 2.0 * nw;
      }
    }
  };
  for (int32_t l = 0; l < L; ++l) {
    gemv(FM_OP_QKV, l, qkv_rows, h, 1);
    for (int32_t j = 0; j < P; ++j) q[j % nwg].push_back(Instr{FM_OP_ATTN, l, j, 0});
    gemv(FM_OP_OPROJ, l, h, (int64_t)nh * d, 1);
    gemv(FM_OP_GU, l, inter, h, 2);
    gemv(FM_OP_DOWN, l, h, inter, 1);
  }
  gemv(FM_OP_LM, L, V, h, 1);

  p.qoff.assign(nwg + 1, 0);
  p.stage_rng.assign((size_t)p.n_stages * nwg * 2, 0);
  int32_t lm = 0;
  for (int32_t w = 0; w < nwg; ++w) {
    p.qoff[w] = (int32_t)p.instrs.size();
    int32_t base = (int32_t)p.instrs.size();
    for (size_t k = 0; k < q[w].size(); ++k) {
      const Instr& in = q[w][k];
      int32_t s = stage_of(in, L);
      int32_t* r = &p.stage_rng[((size_t)s * nwg + w) * 2];
      int32_t idx = base + (int32_t)k;
      if (r[1] == r[0]) r[0] = idx;
      r[1] = idx + 1;
      if (in.op == FM_OP_LM) ++lm;
      p.instrs.push_back(in);
    }
  }
  p.qoff[nwg] = (int32_t)p.instrs.size();
  p.n_lm_instr = lm;

  // Statistics (the paper's interpreter gate: instruction types, instructions per layer,
  // queue imbalance; its dependency gate: distinct counters).
  fm_plan_stats& s = p.stats;
  s.n_cu = nwg;
  s.n_instr = (int32_t)p.instrs.size();
  s.n_types = 6;
  int32_t min_pl = 1 << 30;
  for (int32_t l = 0; l < L; ++l) {
    int32_t cnt = 0;
    for (const Instr& in : p.instrs) cnt += (in.layer == l && in.op != FM_OP_LM);
    min_pl = std::min(min_pl, cnt);
  }
  s.min_instr_per_layer = min_pl;
  // Per layer: tagged qkv, o, x1, m and x vectors (5) plus one tagged partial block per
  // (lane, KV head); per step: the LM arrival counter and b argmax words; per dynamic stage
  // one claim counter per pool.
  s.n_counters = 5 * L + L * nkv * b + 1 + b + n_dyn * std::min(kPools, nwg);
  s.attn_items = P;
  s.attn_max_chunks = p.attn_max_chunks;
  s.n_stages = p.n_stages;
  s.n_dyn_stages = n_dyn;
  double mx = 0, sum = 0;
  for (double v : bytes) {
    mx = std::max(mx, v);
    sum += v;
  }
  s.max_bytes_per_cu = mx;
  s.mean_bytes_per_cu = sum / nwg;
  s.imbalance = sum > 0 ? mx / (sum / nwg) : 1.0;
  return FM_OK;
}

}  // namespace fm
