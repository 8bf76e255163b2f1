/*
 * fm.h -- single-launch transformer decode step for AMD MI355X (gfx950).
 *
 * One call of fm_decode_step runs one decode step for a batch of b lanes inside ONE
 * persistent kernel launch. Per lane it does the following:
 *   - embedding gather;
 *   - per layer: RMSNorm -> QKV projection -> optional per-head QK-RMSNorm -> RoPE ->
 *     KV-cache append -> grouped-query attention over the cache -> O projection + residual ->
 *     RMSNorm -> gate/up -> SiLU*up -> down projection + residual;
 *   - final RMSNorm -> LM head -> greedy argmax.
 * The step is the paper's (arXiv 2609.12379, Sec. 2.1 "The decode step", Eq. 1 for attention).
 * The single persistent launch, the per-CU instruction queues, the dependency tracking that
 * replaces grid-wide barriers, and the on-chip staging pool follow the structure of Sec. 4.1.
 *
 * Arithmetic: weights and the KV cache are bf16 storage, upcast exactly. Every other value
 * stays in fp32: the residual stream, norm outputs, q/k/v, softmax, the SiLU product and
 * the logits. New K/V are rounded to bf16 (round to nearest even) when appended.
 *
 * Memory ownership: the caller allocates every weight, KV, id and logit buffer on the
 * device and keeps it alive until fm_destroy. The library only borrows those pointers: it
 * never copies or repacks weights. The handle owns only its private scratch: instruction
 * queues, activation words, attention partials, counters and the rotary table.
 *
 * Errors come in two kinds.
 *   - Synchronous: host-checkable problems (NULL pointers, bad or unsupported shapes) are
 *     returned at once.
 *   - Asynchronous: per-step arrays live on the device, so bad token ids, positions or
 *     cache lengths are detected there. The kernel then performs no memory access for the
 *     step, records a sticky code, and the next fm_decode_step / fm_last_error returns
 *     FM_ERR_DEVICE. A stalled dependency wait (a scheduling fault) is handled the same way
 *     and is bounded by a watchdog instead of hanging. Once a handle reports FM_ERR_DEVICE
 *     it stays in that state.
 *
 * Concurrency: all calls are stream-ordered. One handle must not be used on two streams at
 * once, because its scratch is per handle. Several handles may coexist.
 *
 * Determinism: identical inputs give bit-identical outputs from run to run. No float
 * atomics are used, every reduction has a fixed order, and the argmax uses an
 * order-independent integer maximum.
 */
#ifndef FM_H
#define FM_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum fm_status {
  FM_OK = 0,
  FM_ERR_INVALID_ARG = 1,   /* NULL pointer, negative or inconsistent dimension */
  FM_ERR_UNSUPPORTED = 2,   /* a shape this build does not implement (see fm_create) */
  FM_ERR_CAPACITY = 3,      /* device resources exceeded (LDS, co-residency, 4 GiB matrices) */
  FM_ERR_HIP = 4,           /* a HIP runtime call failed */
  FM_ERR_DEVICE = 5         /* the device recorded an error in an earlier step (sticky) */
} fm_status;

/* Device-side error codes reported through fm_last_error. */
enum {
  FM_DEV_OK = 0,
  FM_DEV_BAD_TOKEN = 1,     /* token_ids[i] outside [0, vocab) */
  FM_DEV_BAD_POSITION = 2,  /* positions[i] outside [0, max_ctx) */
  FM_DEV_BAD_KV_LEN = 3,    /* kv_lens[i] outside [0, max_ctx - 1] */
  FM_DEV_WATCHDOG = 4,      /* a dependency wait exceeded its time bound */
  FM_DEV_BAD_PLAN = 5       /* an instruction's geometry does not fit the kernel's LDS layout
                               (cannot happen with a schedule built by fm_create) */
};

/* Model shape, batch and context bound (the model configuration the schedule is compiled
 * from, Sec. 4.1). These stay fixed for the handle's lifetime: the paper compiles one kernel
 * per (model, b, S) cell (Sec. 5.3, context bins).
 * Supported: head_dim 64 or 128; hidden, n_heads*head_dim and intermediate multiples of 8;
 * n_heads a multiple of n_kv_heads with n_heads/n_kv_heads <= 8; batch 1..8.
 * The last three integer fields are tuning knobs, not part of the model: leave them 0. */
typedef struct fm_model_cfg {
  int32_t n_layers, hidden, n_heads, n_kv_heads, head_dim, intermediate, vocab;
  int32_t qk_norm;          /* 1: per-head RMSNorm on q and k before RoPE (Qwen3-shaped) */
  int32_t tied_embedding;   /* 1: the LM head is the embedding matrix */
  int32_t batch;            /* b: every step decodes exactly b lanes */
  int32_t max_ctx;          /* S_max: KV slots per lane per layer; also the RoPE table length */
  /* Tuning (0 = automatic; the automatic values are the measured best on MI355X): */
  int32_t n_workgroups;     /* persistent workgroups; 0 = one per compute unit */
  int32_t attn_items;       /* attention work items per layer; 0 = about one per workgroup */
  int32_t dyn_chunk_kb;     /* weight KiB per chunk of a QKV, O-projection or down stage split
                               into chunks that the workgroups claim at run time; 0 = automatic
                               (128), -1 = every GEMV stage in fixed per-workgroup tiles */
  double rope_theta;        /* RoPE base */
  double rms_eps;           /* RMSNorm epsilon, inside the square root */
} fm_model_cfg;

/* Device pointers to bf16 weights, row-major [out][in]. The layer computes
 *   q = W_q a, k = W_k a, v = W_v a   with a = RMSNorm(x) * attn_norm,
 *   x += W_o attn(q, k, v),
 *   x += W_down (silu(W_gate a2) * (W_up a2))   with a2 = RMSNorm(x) * mlp_norm. */
typedef struct fm_layer_weights {
  const void *attn_norm;          /* [hidden] */
  const void *w_q;                /* [n_heads*head_dim][hidden] */
  const void *w_k, *w_v;          /* [n_kv_heads*head_dim][hidden] */
  const void *q_norm, *k_norm;    /* [head_dim], shared by all heads; NULL unless qk_norm */
  const void *w_o;                /* [hidden][n_heads*head_dim] */
  const void *mlp_norm;           /* [hidden] */
  const void *w_gate, *w_up;      /* [intermediate][hidden] */
  const void *w_down;             /* [hidden][intermediate] */
} fm_layer_weights;

typedef struct fm_weight_ptrs {
  const void *embed;              /* [vocab][hidden] */
  const void *final_norm;         /* [hidden] */
  const void *lm_head;            /* [vocab][hidden]; ignored (may be NULL) when tied */
  const fm_layer_weights *layers; /* HOST array [n_layers] of device pointers */
} fm_weight_ptrs;

/* KV arena, owned by the caller (the paper's harness owns it, Sec. 4.2). Per layer one K and
 * one V buffer of bf16 [batch][n_kv_heads][max_ctx][head_dim]. */
typedef struct fm_kv_ptrs {
  void *const *k;                 /* HOST array [n_layers] of device pointers */
  void *const *v;
} fm_kv_ptrs;

typedef struct fm_handle fm_handle;

/* Build the per-CU instruction queues for this model and allocate the handle's scratch on
 * the current HIP device. This is the schedule compiler of Sec. 4.1 (the interpreter step of
 * the milestones: the model configuration becomes typed per-CU instruction streams), fixed
 * for one (model, b, S_max) cell as in Sec. 5.3. Borrows the weight and KV pointers (see
 * "Memory ownership" above). Checks every pointer for NULL. Returns:
 *   FM_ERR_UNSUPPORTED for a shape outside the supported set above;
 *   FM_ERR_CAPACITY if a matrix exceeds 2 GiB or the grid cannot be co-resident;
 *   FM_ERR_HIP if an allocation fails.
 * On failure *out is set to NULL. */
fm_status fm_create(const fm_model_cfg *cfg, const fm_weight_ptrs *w, const fm_kv_ptrs *kv,
                    fm_handle **out);

/* One decode step for all lanes, as one kernel launch on `stream`: the decode step of
 * Sec. 2.1 (embedding, per-layer RMSNorm, projections, RoPE, KV append, attention by Eq. 1,
 * SwiGLU MLP, final norm, LM head, greedy token), generating one token per sequence from the
 * weights and the KV cache. Arguments:
 *   token_ids   device int32[b]: token embedded for lane i.
 *   positions   device int32[b]: RoPE position of lane i's new token.
 *   kv_lens     device int32[b]: number of tokens already cached for lane i. The new K/V
 *               are written to slot kv_lens[i]. Attention covers slots 0..kv_lens[i]
 *               inclusive. No other slot is written, and no slot above kv_lens[i] is read.
 *   logits_out  device fp32 [b][vocab], or NULL to skip writing logits.
 *   next_ids    device int32[b]: greedy argmax of each lane's logits (lowest index on ties).
 * The call is asynchronous and advances neither positions nor kv_lens: that is the caller's
 * job. The buffers may be reused by the next step once it is stream-ordered after this one.
 * For example, next_ids of step t may serve as token_ids of step t+1. */
fm_status fm_decode_step(fm_handle *h, const int32_t *token_ids, const int32_t *positions,
                         const int32_t *kv_lens, float *logits_out, int32_t *next_ids,
                         hipStream_t stream);

/* The same step split into one kernel launch per operator stage: per layer a QKV,
 * attention, O-projection, gate/up and down launch, plus one LM-head launch. Each launch
 * runs the same device code on the same per-CU queues and keeps the fusions inside its
 * stage (RMSNorm in the projection's staging, QK-norm, RoPE and the KV append in the
 * attention items, the split-KV merge in each group's last items). This per-stage ablation
 * measures what the single launch saves in launches and drains between stages (the launch
 * and synchronisation costs of split-step engines, Sec. 1 and Sec. 5.2.3). Arguments and
 * results are as for fm_decode_step. The outputs are bit-identical to it. */
fm_status fm_decode_step_multilaunch(fm_handle *h, const int32_t *token_ids,
                                     const int32_t *positions, const int32_t *kv_lens,
                                     float *logits_out, int32_t *next_ids, hipStream_t stream);

/* Size of the fixed device scratch that fm_decode_step_noalloc uses (each GPU holds one copy
 * for the life of the process). */
#define FM_NOALLOC_SCRATCH_BYTES (64u << 20)

/* For callers that cannot allocate device memory while they run steps (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation). The same step as
 * fm_decode_step, with the same arguments, results and errors, bit-identical outputs, and the
 * same kernels; but its per-step scratch (tagged activation words, split-KV partials, argmax
 * words, LM-head arrival counter) lives in a fixed device array of FM_NOALLOC_SCRATCH_BYTES
 * instead of the handle's own buffers, and the call makes no allocation of any kind.
 * Every handle on one GPU shares that GPU's array, which keeps the last step's contents: each
 * call clears what must start at zero (with a small kernel, so the call can be captured), and
 * steps tell their own words from stale ones by an epoch counter shared by all handles of the
 * device. Calls that overlap on one GPU (on different streams, or from different threads
 * without stream order between them) race on the array and give undefined results.
 * Returns FM_ERR_CAPACITY, without launching anything, when the handle's step needs more than
 * FM_NOALLOC_SCRATCH_BYTES (fm_noalloc_scratch_bytes tells how much it needs; batch-1 shapes
 * up to 13B parameters fit). */
fm_status fm_decode_step_noalloc(fm_handle *h, const int32_t *token_ids, const int32_t *positions,
                                 const int32_t *kv_lens, float *logits_out, int32_t *next_ids,
                                 hipStream_t stream);
size_t fm_noalloc_scratch_bytes(const fm_handle *h);

/* Prompt extension (prefill) as a loop of single-token steps, the way the paper's serving
 * integration runs an extend batch (Sec. 4.3, deployment in a serving engine): n_tokens
 * decode steps of all b lanes, launched back to back on `stream` with no host
 * synchronisation between them. Step t reads row t of each array:
 *   token_ids   device int32[n_tokens][b]: the prompt token of lane i at step t
 *               (teacher-forced: the steps never feed back their own greedy tokens);
 *   positions   device int32[n_tokens][b]: its RoPE position;
 *   kv_lens     device int32[n_tokens][b]: its cache slot, as for fm_decode_step. A lane
 *               normally uses kv_lens = positions = its cached length + t. A lane whose
 *               prompt is shorter than n_tokens repeats its last row, which recomputes
 *               the same slot.
 *   logits_out  device fp32 [b][vocab], written by the last step only (NULL: not written);
 *   next_ids    device int32[b]: the greedy tokens of the last step (the first generated
 *               tokens). Every step writes it, so it must not alias token_ids.
 * Each step is exactly fm_decode_step: the results are bit-identical to n_tokens such calls.
 * n_tokens = 0 does nothing. Errors are those of fm_decode_step. The first failing step's
 * status is returned and later steps are not launched. */
fm_status fm_extend(fm_handle *h, const int32_t *token_ids, const int32_t *positions,
                    const int32_t *kv_lens, int32_t n_tokens, float *logits_out, int32_t *next_ids,
                    hipStream_t stream);

/* Release the handle's scratch. The caller's buffers are untouched. No passage of the paper
 * defines this call; it is resource management of the library. Synchronises the device
 * first, so no step of this handle is still running. Returns FM_ERR_INVALID_ARG for NULL. */
fm_status fm_destroy(fm_handle *h);

/* Synchronise the device, then report the sticky device error code (FM_DEV_*) in
 * *device_code. Returns FM_OK when no error was recorded, FM_ERR_DEVICE when one was, and
 * FM_ERR_HIP if the synchronisation fails. No passage of the paper defines this call: it
 * reports the asynchronous errors described at the top of this file. Debug only. */
fm_status fm_last_error(fm_handle *h, int32_t *device_code);

/* Mid-state taps, for the mid-state test oracle of Sec. 4.2 (per-layer intermediate values
 * compared against a reference decoder, layer by layer). When tap_buf (device fp32,
 * fm_tap_count(cfg) floats, owned by the caller and kept alive while taps are on) is
 * non-NULL, each step also writes per layer and lane the values below, in this order:
 *   a[h] | qkv[(nh + 2 nkv) d] | q_rot[nh d] | k_rot[nkv d] | o[nh d] | x1[h] | a2[h] | mlp[h] | x2[h]
 * Blocks are laid out [n_layers][batch]. After them comes the final normed vector [batch][h].
 * The fields:
 *   a     attention-norm output;
 *   qkv   raw projection output;
 *   q_rot, k_rot   after QK-norm and RoPE, before rounding;
 *   o     attention output;
 *   x1    residual after attention;
 *   a2    MLP-norm output;
 *   mlp   W_down m;
 *   x2    residual after the MLP.
 * Pass NULL to turn taps off. Taps cost extra stores and are meant for verification. */
fm_status fm_set_taps(fm_handle *h, float *tap_buf);
size_t fm_tap_count(const fm_model_cfg *cfg);

/* Instruction timeline: when buf (device uint64, 8 * fm_instruction_count(h) words) is
 * non-NULL, each step records per queued instruction q, at buf[8q..8q+7], the device
 * wall-clock ticks {start, inputs ready, prologue done, stream done, end, workgroup, a, b}.
 * For attention items the middle marks are: q/k/v ready, rotary and KV append done, partials
 * published; the span from there to the end is the merge of the item's heads (only in a
 * group's last min(G, chunks, workgroups) items, each merging every such count-th head);
 * a = the item's slot passes done, b = its waves' partials gathered in LDS. GEMV tiles leave
 * a and b 0, except that a GEMV stage in dynamic chunks records in a the number of chunks the
 * workgroup took (a count, not a time).
 * Marks an instruction does not reach are 0. The ticks are from the 100 MHz constant clock,
 * read with s_memrealtime. These spans give the paper's busy fraction and tail spread
 * (Sec. 4.1, dependency gate). Pass NULL to turn the timeline off. */
fm_status fm_set_timeline(fm_handle *h, uint64_t *buf);
int32_t fm_instruction_count(const fm_handle *h);

/* Host-only schedule inspection (no GPU needed). The queues are the per-CU instruction
 * streams that the host compiles from the model (Sec. 4.1, first step).
 *   fm_plan_query fills the summary statistics. n_cu is the workgroup count to plan for.
 *   fm_plan_export copies the queues: qoff (int32[n_cu + 1]) gives queue w's range in
 *   instrs, and instrs holds int32[4] records {op, layer, a, b} (FM_OP_*):
 *     GEMV, a >= 0: output rows [a, b) of the op's matrix, streamed by this workgroup alone;
 *     GEMV, a < 0 (QKV, O projection, down; batch <= 2): a stage in dynamic chunks of -a
 *       rows. Every workgroup holds one such
 *       record per stage. Workgroup w serves pool w mod P (P = min(8, n_cu)); the stage's
 *       ceil(rows / -a) chunks are split into contiguous pool ranges in proportion to the
 *       pools' workgroup counts. Each workgroup of a pool takes one chunk of the range (its
 *       (w div P)-th), and the range's other chunks go to the pool's workgroups on demand,
 *       through one device counter per (stage, pool). b packs the chunk's K split (b & 255)
 *       and the most chunks one workgroup may take (b >> 8).
 *     FM_OP_ATTN: attention work item a of the layer.
 *   Its return codes: FM_ERR_CAPACITY when the arrays are shorter than fm_plan_query
 *   reports; FM_ERR_INVALID_ARG or FM_ERR_UNSUPPORTED for a bad cfg. */
enum { FM_OP_QKV = 1, FM_OP_ATTN = 2, FM_OP_OPROJ = 3, FM_OP_GU = 4, FM_OP_DOWN = 5, FM_OP_LM = 6 };

typedef struct fm_plan_stats {
  int32_t n_cu;              /* workgroups planned for */
  int32_t n_instr;           /* total instructions */
  int32_t n_types;           /* distinct instruction types */
  int32_t min_instr_per_layer;
  int32_t n_counters;        /* distinct dependency objects (tagged vectors + arrival counters) */
  int32_t attn_items;        /* attention work items per layer */
  int32_t attn_max_chunks;   /* capacity of split-KV partials per (lane, KV head) */
  int32_t n_stages;          /* launches the multi-launch ablation makes per step */
  int32_t n_dyn_stages;      /* GEMV stages run in dynamic chunks */
  double max_bytes_per_cu;   /* weight bytes streamed by the busiest queue (a dynamic stage
                                counts its mean share for every queue) */
  double mean_bytes_per_cu;
  double imbalance;          /* max / mean */
} fm_plan_stats;

fm_status fm_plan_query(const fm_model_cfg *cfg, int32_t n_cu, fm_plan_stats *out);
fm_status fm_plan_export(const fm_model_cfg *cfg, int32_t n_cu, int32_t *qoff, int32_t qoff_cap,
                         int32_t *instrs, int32_t instr_cap);

const char *fm_status_string(fm_status s);

#ifdef __cplusplus
}
#endif
#endif /* FM_H */
