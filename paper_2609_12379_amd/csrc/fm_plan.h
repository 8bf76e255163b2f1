// Host-side schedule compiler: model config -> per-workgroup instruction queues.
//
// Each decode step is compiled into typed instructions with explicit operand ranges, one
// queue per persistent workgroup (arXiv 2609.12379 Sec. 4.1, first step). Every queue is
// ordered by (layer, stage), which is one global topological order of the step's
// dependency graph. A workgroup waits only for inputs produced earlier in that order, so
// when all workgroups are co-resident the step cannot deadlock.
#pragma once
#include <cstdint>
#include <string>
#include <vector>

#include "../../include/fm.h"

namespace fm {

// One instruction: op (FM_OP_*), layer, and an operand range whose meaning depends on op:
//   GEMV ops  -> output rows [a, b) of that op's matrix (QKV rows index [W_q; W_k; W_v]),
//   FM_OP_ATTN -> attention work item a of the layer (mapped to lane/KV head/slots per step;
//                 a (lane, KV head) group's last items also merge its partials, a head set each).
struct Instr {
  int32_t op, layer, a, b;
};

struct Plan {
  int32_t nwg = 0;
  int32_t attn_items = 0;      // P: items per layer
  int32_t attn_max_chunks = 0; // partials capacity per (lane, KV head)
  int32_t n_lm_instr = 0;      // workgroups holding LM-head rows
  int32_t n_stages = 0;        // 5 per layer + LM head
  std::vector<Instr> instrs;
  std::vector<int32_t> qoff;       // [nwg + 1]
  std::vector<int32_t> stage_rng;  // [n_stages][nwg][2]: each queue's sub-range per stage
  fm_plan_stats stats{};
};

// Validates cfg. Returns FM_OK and fills `plan`, or an error with a message in `why`.
fm_status build_plan(const fm_model_cfg& cfg, int32_t nwg, Plan& plan, std::string* why);

// Stage index of an instruction in the multi-launch order.
// Per layer: QKV, attention items, O projection, gate/up, down; then the LM head.
inline int32_t stage_of(const Instr& in, int32_t n_layers) {
  if (in.op == FM_OP_LM) return 5 * n_layers;
  const int32_t order = in.op == FM_OP_QKV ? 0 : in.op == FM_OP_ATTN ? 1 : in.op == FM_OP_OPROJ ? 2
                      : in.op == FM_OP_GU ? 3 : 4;
  return 5 * in.layer + order;
}

}  // namespace fm
