/*
 * atom.h - C ABI of libatom: one swapped GPT training step on one MI355X.
 *
 * The model of Atom (arXiv 2403.10504): a complete GPT-3-style model lives in
 * host memory (Section I; Section III-A, "Design Overview"); it is cut at
 * decoder-block boundaries into contiguous sub-models ("groups") that a
 * static analysis fits into a GPU memory budget (Section III-D, Algorithm 1);
 * the runtime swaps groups into the GPU on one stream while another runs the
 * current group (Section IV), and gradient accumulation over C micro-batches
 * lengthens compute per swap (Section III-C).
 *
 * Layer chain ("nodes", topologically sorted as in Section III-D):
 *   node 0        embedding: wte [V][d], wpe [T][d]
 *   nodes 1..L    decoder blocks (pre-LayerNorm GPT block)
 *   node L+1      final LayerNorm + LM head ("Logits" layer): lnf_g, lnf_b,
 *                 w_head [Vp][d] with Vp = V rounded up to 128 (zero rows)
 * Linear weights are [out][in]: y = x W^T + b.  A block holds, in order:
 *   ln1_g [d], ln1_b [d], w_qkv [3d][d], b_qkv [3d], w_o [d][d], b_o [d],
 *   ln2_g [d], ln2_b [d], w_fc [f][d], b_fc [f], w_pr [d][f], b_pr [d].
 * Each node's tensors are one contiguous host range (tensor offsets aligned
 * to 256 bytes, see atom_node_layout) and consecutive nodes are adjacent, so
 * a group swaps with one copy.
 *
 * Ownership.  The caller owns the device arena (one allocation of exactly
 * atom_plan.arena_bytes, e.g. a torch uint8 tensor) and the compute
 * stream; both must outlive the context.  The library never allocates
 * device memory.  Weight and gradient copies run on the GPU's system DMA
 * engines (one fixed engine per direction), issued by library threads.  The
 * context therefore takes no copy streams: a copy queued on a HIP stream
 * would run on HIP's own engine selection (device-to-host copies as a blit
 * kernel that competes with the training kernels for compute units), so
 * only the compute stream comes from the caller.
 * The library owns the pinned host model (weights in the working dtype), the
 * host gradient buffer (the last step's gradients in the working dtype) and
 * the fp32 gradient accumulators.  Pinned host memory: the weights, one
 * gradient buffer and, with host checkpoints, the evicted block inputs.
 *
 * Errors.  Every call returns an atom_status; nothing throws across the ABI.
 * atom_last_error(ctx) describes the last failure on a context;
 * atom_last_error(NULL) the last failed atom_ctx_create of the calling
 * thread.  Calls that
 * enqueue GPU work report launch errors at once; execution errors surface at
 * the next synchronising call (atom_step, atom_sync, atom_ctx_destroy).
 * Threading: one context per host thread.
 */
#ifndef ATOM_H
#define ATOM_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ATOM_MAX_NODES 256

typedef enum atom_status {
  ATOM_OK = 0,
  ATOM_EINVAL = -1,       /* bad argument or unsupported shape */
  ATOM_ENOPLAN = -2,      /* no partition fits the device budget */
  ATOM_EBUDGET = -3,      /* arena smaller than the plan needs */
  ATOM_EHIP = -4,         /* a HIP runtime call failed */
  ATOM_ESTATE = -5,       /* call-order violation (e.g. compute on a group not swapped in) */
  ATOM_ENOMEM_HOST = -6   /* pinned host allocation failed */
} atom_status;

typedef enum atom_dtype { ATOM_F32 = 0, ATOM_BF16 = 1 } atom_dtype;
typedef enum atom_ckpt_policy { ATOM_CKPT_DEVICE = 0, ATOM_CKPT_HOST = 1 } atom_ckpt_policy;

/* Model and step shape (Table II gives the GPT-3 shapes).  d_model must be
 * a multiple of 64 (at most 8192), d_model / n_head must be 64 or 128, and
 * accum is the gradient-accumulation degree C (micro-batches per step). */
typedef struct atom_config {
  int32_t n_layer, d_model, n_head, d_mlp, vocab, seq_len, batch, accum;
  int32_t dtype; /* atom_dtype: working precision of weights and activations */
  int32_t ckpt;  /* atom_ckpt_policy: where block-input checkpoints live.
                  * ATOM_CKPT_DEVICE keeps all L+1 block inputs (fp32 [N][d]
                  * per micro-batch) in the arena.  ATOM_CKPT_HOST keeps a ring
                  * of 4 per micro-batch: the forward copies inputs 0..L-4 to
                  * pinned host memory (D2H engine) after the kernel that wrote
                  * them, and the backward restores each (H2D engine) before the
                  * block that reads it; results are bitwise unchanged.  The
                  * plan's h2d/d2h/forced byte counts include these copies. */
} atom_config;

/* Cost of one node of the augmented graph (Section III-D: the node's
 * loading time t^u, forward time t^f, backward time t^b; memory is its
 * weight bytes, which sets the slot it needs).  Times in seconds; t_fwd and
 * t_bwd are per micro-batch, t_bwd includes the forward recompute; t_store
 * is the time to copy the node's gradients back to the host. */
typedef struct atom_node_cost {
  uint64_t weight_bytes;
  double t_fwd, t_bwd, t_load, t_store;
} atom_node_cost;

/* A partition of the chain into contiguous groups and its static layout.
 * Group g holds nodes first[g]..last[g] and uses weight slot g % n_slots;
 * the last n_slots groups stay resident from the forward into the backward.
 * Gradients of a group go to one of n_gslots gradient slots (2 to 16, used
 * round-robin in backward order); a copy out to the host must finish before
 * its slot is reused, so more slots let the copies lag further behind the
 * backward.  arena_bytes = reserve_bytes + (n_slots + n_gslots) * slot_bytes
 * (+ 2 * slot_bytes fp32 accumulation slot for bf16 with accum > 1). */
#define ATOM_MAX_GSLOTS 16
typedef struct atom_plan {
  int32_t n_nodes, n_groups, n_slots, overlap_ok, exhaustive, accum, n_gslots;
  int32_t first[ATOM_MAX_NODES], last[ATOM_MAX_NODES];
  uint64_t budget_bytes, reserve_bytes, slot_bytes, arena_bytes;
  uint64_t h2d_bytes, d2h_bytes, forced_h2d_bytes;
  double pred_fwd_s, pred_step_s;
  int64_t n_evaluated;
} atom_plan;

/* One tensor of a node's host range. */
typedef struct atom_tensor_desc {
  char name[16];
  int32_t rows, cols;     /* cols == 1 for vectors */
  uint64_t offset, bytes; /* within the node's range, working dtype */
} atom_tensor_desc;

typedef struct atom_ctx atom_ctx;

/* Library version string. */
const char* atom_version(void);
/* Short text for a status code. */
const char* atom_status_string(int status);

/* Tensor layout of node `node` under cfg.  Writes up to `max` descriptors,
 * the count to *n_out and the node's total bytes to *node_bytes.
 * ATOM_EINVAL for a bad node index or config. */
int atom_node_layout(const atom_config* cfg, int32_t node, atom_tensor_desc* out, int32_t max, int32_t* n_out,
                     uint64_t* node_bytes);

/* Analytic node costs for cfg (n = n_layer + 2 entries): FLOP counts at an
 * assumed MFMA rate and bytes at an assumed host-link rate (the values are
 * half the dense MFMA peak, i.e. 1.25 PFLOP/s bf16 or 78.65 TFLOP/s fp32, 50 GB/s
 * host link each way, 4 TB/s HBM for the embedding); callers may substitute
 * measured costs. */
int atom_node_costs(const atom_config* cfg, atom_node_cost* out, int32_t n);

/* Device bytes the step needs besides weight and gradient slots
 * (checkpoints, activations, workspace, tokens). */
int atom_reserve_bytes(const atom_config* cfg, uint64_t* out);

/* Planner core (Algorithm 1 with the constraints and selection rule of
 * Section III-D: co-resident executing and prefetched groups, overlap as a
 * reported soft constraint, smallest predicted step time then fewest bytes loaded then fewest groups
 * then smallest end-node list): searches contiguous
 * partitions of `n` nodes with the given costs, a device budget and
 * `reserve` bytes of non-slot memory.  Exhaustive for n <= 20 nodes; for
 * longer chains it searches the structured family that identical decoder
 * blocks allow.  The memory model counts two gradient slots (n_gslots = 2).
 * Returns ATOM_ENOPLAN when no partition fits. */
int atom_plan_search(const atom_config* cfg, uint64_t budget_bytes, uint64_t reserve_bytes,
                     const atom_node_cost* costs, int32_t n, atom_plan* out);

/* atom_plan_partition: the static analysis of Section III-D for cfg under
 * a device budget.  costs == NULL uses atom_node_costs; the reserve comes
 * from atom_reserve_bytes.  Budget the search leaves unused becomes extra
 * gradient slots (up to ATOM_MAX_GSLOTS), which changes no transfer and no
 * result, only how far gradient copies may lag the backward.  Errors:
 * ATOM_EINVAL, ATOM_ENOPLAN. */
int atom_plan_partition(const atom_config* cfg, uint64_t device_budget_bytes, const atom_node_cost* costs,
                        int32_t n_costs, atom_plan* out);

/* A plan for a given partition: group g ends at node last[g] (strictly
 * increasing, last[n_groups-1] = n_layer + 1), with n_slots weight slots
 * (1 <= n_slots <= n_groups, at least min(n_groups, 2)) and n_gslots
 * gradient slots (2..ATOM_MAX_GSLOTS).  Fills the slot
 * size, arena size and transfer bytes from the layout; predicted times use
 * the analytic costs.  ATOM_EINVAL for a malformed partition. */
int atom_plan_fixed(const atom_config* cfg, int32_t n_groups, const int32_t* last, int32_t n_slots,
                    int32_t n_gslots, atom_plan* out);

/* Create a context: validates cfg against plan, carves the arena, allocates
 * the pinned host model (zero weights; fill them through atom_host_tensor)
 * and the host gradient buffer, and opens the two DMA engines on the
 * current HIP device.  compute_stream is a hipStream_t handle (e.g.
 * torch.cuda.Stream().cuda_stream) that receives every kernel; the library
 * also runs a few threads of its own (copies, host accumulation).  Errors:
 * ATOM_EINVAL, ATOM_EBUDGET (arena_bytes < plan->arena_bytes),
 * ATOM_ENOMEM_HOST, ATOM_EHIP. */
int atom_ctx_create(const atom_config* cfg, const atom_plan* plan, void* dev_arena, uint64_t arena_bytes,
                    void* compute_stream, atom_ctx** out);
/* Waits for all work, frees host memory and events.  NULL is ignored. */
void atom_ctx_destroy(atom_ctx* ctx);

/* Host buffers of a node: which = 0 weights (working dtype, writable),
 * 1 fp32 gradient accumulators (sum over committed steps), 2 gradients of
 * the last step in the working dtype. */
int atom_host_tensor(atom_ctx* ctx, int32_t node, int32_t which, void** ptr, uint64_t* bytes);

/* Zero the fp32 gradient accumulators. */
int atom_zero_grads(atom_ctx* ctx);

/* Upload tokens for the next step: host int32 [accum][batch][seq_len + 1];
 * inputs are [..., :T], next-token targets [..., 1:]; every id must be in
 * [0, vocab) (ATOM_EINVAL otherwise).  Synchronous. */
int atom_set_tokens(atom_ctx* ctx, const int32_t* tokens);

/* --- the per-group calls atom_step composes (all asynchronous) --- */

/* Swap-in (Section IV: a second stream prefetches the next sub-model as soon
 * as the current one starts; Section III-D: a sub-model is a contiguous group
 * of nodes).  Copies group `group`'s weights from the pinned host model into
 * its weight slot on the host-to-device system DMA engine; the copy is issued
 * by a library worker thread once the slot's previous occupant has finished
 * its last kernel (an event on the compute stream).  The first kernel of the
 * group waits for the copy.  ATOM_ESTATE if the group is already resident. */
int atom_swap_in(atom_ctx* ctx, int32_t group);
/* Forward of one node (Section III-B: the GPT-3 layers; Section III-C:
 * micro-batch `micro` of the C accumulated ones) on the compute stream.  Node
 * 0 embeds the tokens; a block node writes its output checkpoint; node L+1
 * runs the final LayerNorm, the LM head, the cross-entropy and the head's
 * backward (it starts the gradient of the residual stream).  ATOM_ESTATE if
 * the node's group is not swapped in, or its input is not ready. */
int atom_block_fwd(atom_ctx* ctx, int32_t node, int32_t micro);
/* Backward of one node for micro-batch `micro` (Section III-B; the last
 * forward sub-model is reused by the backward, Section IV): a block restores
 * its input checkpoint, recomputes its forward and writes its gradients into
 * the group's gradient slot; node 0 runs the embedding backward.  Node L+1
 * has no separate backward (ATOM_EINVAL). */
int atom_block_bwd(atom_ctx* ctx, int32_t node, int32_t micro);
/* Swap-out of a completed sub-model (Section IV).  Copies group `group`'s
 * gradients to the pinned host gradient buffer on the device-to-host system
 * DMA engine (issued by a library worker thread after the group's last
 * backward kernel), then a host thread adds them to the fp32 accumulators
 * (the gradient of the global batch, Section III-E).  Releases the group's
 * weight slot. */
int atom_swap_out(atom_ctx* ctx, int32_t group);
/* Wait for every stream and host accumulation; *loss_out (may be NULL)
 * receives the mean loss of the step. */
int atom_sync(atom_ctx* ctx, float* loss_out);

/* One whole training step: uploads tokens, runs the plan's schedule (swap-in
 * with prefetch, forward of every group for every micro-batch, head, backward
 * with reloads, gradient swap-out and host accumulation) and waits.  The mean
 * loss goes to *loss_out.  Synchronous. */
int atom_step(atom_ctx* ctx, const int32_t* tokens, float* loss_out);

/* `n_steps` (1..64) training steps of one global batch, pipelined: the host
 * model is not changed between them (the optimizer runs after the global
 * batch, Section III-E), so the next step's first groups are swapped in while
 * the current step's backward runs and its gradients are swapped out (the
 * overlap of Section IV carried across the step boundary).  Every step still
 * loads every weight and copies out every gradient, and the fp32 host
 * accumulators receive the gradients of all steps.  tokens: host int32
 * [n_steps][accum][batch][seq_len + 1]; losses: host float[n_steps] (may be
 * NULL), the mean loss of each step.  The result is bitwise that of n_steps
 * calls of atom_step.  All token ids are validated before anything runs
 * (ATOM_EINVAL; nothing is changed).  Synchronous. */
int atom_steps(atom_ctx* ctx, const int32_t* tokens, int32_t n_steps, float* losses);

/* Weight retention across the steps of one atom_steps call (default off).
 * The host model does not change inside a global batch, and the paper keeps
 * the sub-models that fit on the device from one iteration to the next (the
 * embedding's, Section III-C; the last forward sub-model into the backward,
 * Section IV).  With retention on and a plan that gives every group a weight
 * slot of its own (n_slots >= n_groups), atom_steps loads each group once per
 * call instead of once per step; gradients still leave the GPU every step and
 * reach the host accumulators.  Results are bitwise those with retention off
 * (same kernels, same order, same weights).  No effect when n_slots <
 * n_groups, and none on calls other than atom_steps (atom_step is one step).
 * The next call loads every group again.  ATOM_EINVAL for a NULL ctx. */
int atom_set_retention(atom_ctx* ctx, int32_t on);

/* Host optimizer (Section V-B: AdamW on the host CPUs once a global batch
 * is complete, learning rate 1e-4 after a linear warm-up, betas 0.9 and
 * 0.999).  atom_optimizer_init allocates fp32 master weights (copied from
 * the host model) and the two moments (zero), 12 bytes per parameter of
 * pageable memory.  atom_optimizer_step waits for all work, then for every
 * parameter: g = grad_scale * accumulator (e.g. 1 / steps of the global
 * batch), m = beta1 m + (1 - beta1) g, v = beta2 v + (1 - beta2) g^2,
 * p = p (1 - lr wd) - lr (m / (1 - beta1^step)) / (sqrt(v / (1 - beta2^step))
 * + eps), with weight decay only on the linear layers' weight matrices
 * (w_qkv, w_o, w_fc, w_pr, w_head); it writes the working-dtype weights
 * (bf16 rounded to nearest even) into the host model and zeroes the
 * accumulators.  fp32 arithmetic on the host thread pool.  step >= 1 counts
 * optimizer steps.  ATOM_ESTATE before atom_optimizer_init. */
typedef struct atom_adamw {
  float lr, beta1, beta2, eps, weight_decay;
} atom_adamw;
int atom_optimizer_init(atom_ctx* ctx);
int atom_optimizer_step(atom_ctx* ctx, const atom_adamw* hp, float grad_scale, int32_t step);

/* Measured node costs for the planner (the per-layer profile of Section
 * III-D: loading time t^u, forward time t^f, backward time t^b, plus the
 * time to store a node's gradients): each node's weights copied alone to the
 * device and its gradients back on the step's DMA engines (best of three),
 * and the kernel time of each node's forward and backward (per micro-batch,
 * HIP events on the compute stream) in a step of the context's plan on
 * `tokens` (host int32 [accum][batch][seq_len + 1]) that follows one
 * untimed step on the same tokens.  Both steps' gradients are added to the
 * accumulators like atom_step's.  out: n = n_layer + 2
 * entries; pass them to atom_plan_partition.  Synchronous. */
int atom_profile_nodes(atom_ctx* ctx, const int32_t* tokens, atom_node_cost* out, int32_t n);

/* The configuration and plan a context was created with (either pointer may
 * be NULL).  Bindings use it to check host token arrays against
 * [accum][batch][seq_len + 1] before a call reads them.  ATOM_EINVAL for a
 * NULL ctx. */
int atom_ctx_config(const atom_ctx* ctx, atom_config* cfg, atom_plan* plan);

/* Per-step counters of the last atom_step / atom_steps call (bytes and
 * swap counts summed over its steps; times per step). */
typedef struct atom_stats {
  uint64_t h2d_bytes, d2h_bytes;
  double step_s, host_accum_s;
  int32_t swap_ins, swap_outs;
} atom_stats;
int atom_get_stats(atom_ctx* ctx, atom_stats* out);

/* Kernel probe for measurement.  While enabled, every launch of the GEMM
 * instantiation (a_kcontig, b_kcontig, epilogue as in atom_kernels.h) that
 * the step makes is bracketed by timing events on the compute stream;
 * atom_probe_read returns the number of launches, their summed duration,
 * their summed algorithmic FLOPs (2*M*N*K) and their summed algorithmic HBM
 * bytes (each operand read once, the output written once, plus the tensors
 * the epilogue reads: residual, pre-activation) since the probe was enabled.
 * The LM head's weight gradient runs over the padded vocabulary but is
 * counted at V rows.  epi < 0 disables the probe.  At most 4096 launches are
 * recorded per step call (atom_step or atom_steps); later ones go untimed. */
int atom_probe_gemm(atom_ctx* ctx, int32_t a_kcontig, int32_t b_kcontig, int32_t epi);
int atom_probe_read(atom_ctx* ctx, int64_t* launches, double* seconds, double* flops, double* bytes);

/* Host-link microbenchmark on the context's own pinned buffers and arena
 * (weight-slot region; call between steps): `bytes` per copy (clamped to the
 * slot region), `iters` repetitions.  Rates in GB/s (1e9 bytes/s): pinned
 * host to device alone, device to pinned host alone, and both directions at
 * once (sum of both directions), on the DMA engines a step uses. */
int atom_link_bench(atom_ctx* ctx, uint64_t bytes, int32_t iters, double* h2d_gbs, double* d2h_gbs,
                    double* bidir_gbs);

/* Text of the last error on ctx (never NULL). */
const char* atom_last_error(const atom_ctx* ctx);

#ifdef __cplusplus
}
#endif

#endif /* ATOM_H */
