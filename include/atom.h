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

/* Cost of one node of the augmented graph (Section III-D, problem
 * definition: the node's maximum working memory m_i, forward time t^f,
 * backward time t^b and loading time t^u).  weight_bytes is what a swap moves
 * for the node (its weights; this sets the slot a group needs).  mem_bytes is
 * m_i besides the weights: the device workspace the node's kernels use while
 * it runs (activations, partial sums; every node recomputes its activations
 * from its input checkpoint in the backward, so none of it outlives the node).
 * cut_bytes is the size of the node's output tensor for one micro-batch, the
 * tensor that crosses the cut when a group ends at this node (the fp32
 * [batch][seq_len][d_model] residual stream; Table II lists it per model).
 * Times in seconds; t_fwd and t_bwd are per micro-batch, t_bwd includes the
 * forward recompute; t_store is the time to copy the node's gradients back to
 * the host. */
typedef struct atom_node_cost {
  uint64_t weight_bytes, mem_bytes, cut_bytes;
  double t_fwd, t_bwd, t_load, t_store;
} atom_node_cost;

/* Planner options.  strict = 1 keeps the paper's search result literally:
 * only partitions that meet both the memory and the overlap constraint
 * qualify, and ATOM_ENOPLAN is returned when none does.  strict = 0 falls
 * back to the fastest memory-feasible partition when no partition meets the
 * overlap constraint (atom_plan.rule = ATOM_RULE_TIME).  duplex is the rate
 * of each copy direction while both directions run, relative to its rate
 * alone (both share the host link; 0 selects ATOM_DEFAULT_DUPLEX). */
#define ATOM_DEFAULT_DUPLEX 0.85
typedef struct atom_plan_opts {
  int32_t strict;
  double duplex;
} atom_plan_opts;

/* How a plan was selected. */
enum { ATOM_RULE_PAPER = 0, ATOM_RULE_TIME = 1, ATOM_RULE_FIXED = 2 };

/* A partition of the chain into contiguous groups and its static layout.
 * Group g holds nodes first[g]..last[g] and uses weight slot g % n_slots in
 * even steps (n_slots-1-(g % n_slots) in odd steps of a pipelined call);
 * the last n_slots groups stay resident from the forward into the backward.
 * Gradients of a group go to one of n_gslots gradient slots (2 to 16, used
 * round-robin in claim order); a copy out to the host must finish before
 * its slot is reused, so more slots let the copies lag further behind the
 * backward.  arena_bytes = reserve_bytes + (n_slots + n_gslots) * slot_bytes
 * (+ 2 * slot_bytes fp32 accumulation slot for bf16 with accum > 1), where
 * reserve_bytes holds the largest m_i.  cut_bytes is the total size of the
 * tensors on the cut edges (Section III-D's selection criterion).
 * Predicted times come from an event model of the schedule (the compute
 * stream and the two copy engines, which share the host link at `duplex`):
 * pred_first_step_s is one step alone (atom_step), pred_step_s a step of a
 * pipelined call in steady state (atom_steps), pred_fwd_s the forward part of
 * the first. */
#define ATOM_MAX_GSLOTS 16
typedef struct atom_plan {
  int32_t n_nodes, n_groups, n_slots, overlap_ok, exhaustive, accum, n_gslots, rule;
  int32_t first[ATOM_MAX_NODES], last[ATOM_MAX_NODES];
  uint64_t budget_bytes, reserve_bytes, slot_bytes, arena_bytes, work_bytes;
  uint64_t h2d_bytes, d2h_bytes, forced_h2d_bytes, cut_bytes;
  double pred_fwd_s, pred_first_step_s, pred_step_s, duplex;
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
 * host link each way, 4 TB/s HBM for the embedding); mem_bytes is the
 * workspace the arena carves for the node (blocks: the block workspace;
 * head: the head workspace; embedding: none); callers may substitute
 * measured costs (atom_profile_nodes). */
int atom_node_costs(const atom_config* cfg, atom_node_cost* out, int32_t n);

/* Device bytes the step needs besides weight and gradient slots
 * (checkpoints, activations, workspace, tokens). */
int atom_reserve_bytes(const atom_config* cfg, uint64_t* out);

/* Planner core (Algorithm 1, Section III-D).  Searches the contiguous
 * partitions of the n = cfg->n_layer + 2 nodes (node 0 the embedding, node
 * n-1 the head) under
 *   memory (hard): base_bytes + max_i mem_bytes + K * S + 2 S (+ 2 S fp32
 *     accumulation slot for bf16 with accum > 1) <= budget, with S the
 *     largest group's weight bytes and K = min(G, what fits) >= min(G, 2)
 *     weight slots, so the executing and the prefetched group are
 *     co-resident; budget left over becomes gradient slots (up to 16);
 *   overlap: accum * t^f(g_j) >= t^u(g_{j+1}) for consecutive groups, and
 *     accum * t^b(g_{j+1}) >= t^u(g_j) for every group loaded again in the
 *     backward (j < G - K);
 * and selects, among partitions meeting both, the one with the smallest
 * total cut size, then the smallest predicted step time, then the smallest
 * list of group end nodes (ATOM_RULE_PAPER).  When none meets the overlap
 * constraint: ATOM_ENOPLAN if opts->strict, else the memory-feasible one with
 * the smallest predicted step time, then fewest bytes loaded, then smallest
 * cut, then end list (ATOM_RULE_TIME).  Exhaustive for n <= 16 nodes; longer
 * chains search the structured family identical decoder blocks allow (the
 * embedding alone or with the first block, the head alone or with the last,
 * the remaining blocks in runs of s).  opts may be NULL (non-strict, default
 * duplex).  ATOM_ENOPLAN when no partition fits the budget. */
int atom_plan_search(const atom_config* cfg, uint64_t budget_bytes, uint64_t base_bytes,
                     const atom_node_cost* costs, int32_t n, const atom_plan_opts* opts, atom_plan* out);

/* atom_plan_partition: the static analysis of Section III-D for cfg under
 * a device budget.  costs == NULL uses atom_node_costs.  The arena carves
 * each node's workspace at its analytic size, so a node's m_i counts as at
 * least that.  opts may be NULL.  Errors: ATOM_EINVAL, ATOM_ENOPLAN. */
int atom_plan_partition(const atom_config* cfg, uint64_t device_budget_bytes, const atom_node_cost* costs,
                        int32_t n_costs, const atom_plan_opts* opts, atom_plan* out);

/* A plan for a given partition: group g ends at node last[g] (strictly
 * increasing, last[n_groups-1] = n_layer + 1), with n_slots weight slots
 * (1 <= n_slots <= n_groups, at least min(n_groups, 2)) and n_gslots
 * gradient slots (2..ATOM_MAX_GSLOTS).  Fills the slot
 * size, arena size and transfer bytes from the layout; predicted times use
 * the analytic costs and the default duplex.  ATOM_EINVAL for a malformed
 * partition. */
int atom_plan_fixed(const atom_config* cfg, int32_t n_groups, const int32_t* last, int32_t n_slots,
                    int32_t n_gslots, atom_plan* out);

/* Predicted end time of every step of one call of n_steps (1..64) steps of
 * `plan` (n_steps = 1: atom_step; more: atom_steps) under node costs `costs`
 * (NULL = analytic) and link sharing `duplex` (0 = default), from the event
 * model atom_plan documents: ends[s] for s < n_steps; *fwd_s (may be NULL)
 * the end of step 0's forward.  retain != 0 models atom_set_retention (every
 * group in a slot of its own keeps its weights across the steps of the call,
 * so only step 0 loads; like retention itself, no effect when the plan has
 * fewer slots than groups).  ATOM_EINVAL for a bad plan or count. */
int atom_plan_predict(const atom_config* cfg, const atom_plan* plan, const atom_node_cost* costs, int32_t n_costs,
                      double duplex, int32_t n_steps, int32_t retain, double* ends, double* fwd_s);

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
 * the last step in the working dtype; with the optimizer state allocated
 * (atom_optimizer_init, else ATOM_ESTATE): 3 fp32 master weights, 4 and 5
 * the fp32 first and second AdamW moments. */
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

/* Row-sparse embedding transfers (default off).  A step reads only the rows
 * of wte its input tokens name, and only those rows of the wte gradient are
 * nonzero (the embedding lookup of Section III-B's first layer; its backward
 * adds each token's output gradient into its own row).  With this on, the
 * swap-in of group 0 copies only the step's distinct rows of wte (ascending
 * id, packed at the start of the slot's wte region) and its swap-out only
 * their gradients, which the host accumulation adds to their rows: at most
 * min(V, accum * batch * seq_len) rows each way instead of V.  The kernels
 * address the packed rows through the step's remapped ids.  Losses, the fp32
 * accumulators and the host gradient buffer (atom_host_tensor which = 2 of
 * node 0, spread back to full rows when asked for, after waiting for all
 * work) are bitwise those with it off; atom_stats counts the bytes that
 * actually moved.  Allocates a pinned staging buffer of min(V, accum * batch
 * * seq_len) rows on first use (ATOM_ENOMEM_HOST if refused).  Waits for all
 * work, drops weight residency and requires tokens to be set again (atom_step
 * and atom_steps set them).  ATOM_ESTATE while retention across steps is on
 * (a retained group 0 would hold an earlier step's rows; atom_set_retention
 * refuses the converse in the same way); ATOM_EINVAL for a NULL ctx. */
int atom_set_embedding_rows(atom_ctx* ctx, int32_t on);

/* Host optimizer (Section V-B: AdamW on the host CPUs once a global batch
 * is complete, learning rate 1e-4 after a linear warm-up, betas 0.9 and
 * 0.999).  atom_optimizer_init allocates fp32 master weights (copied from
 * the host model) and the two moments (zero), 12 bytes per parameter of
 * pinned host memory, or pageable memory when the system refuses to pin that
 * much (atom_stats.opt_state_pinned tells which; the GPU never reads this
 * state).  atom_optimizer_step waits for all work, then for every
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
/* The same update, applied during the next atom_step / atom_steps call
 * instead of after it: in that call's last step, as soon as a group's
 * gradients have been added to the accumulators (the group's last gradients
 * of the global batch, Section III-E), the host thread pool updates that
 * group's parameters, so the update of the groups that finish their backward
 * first overlaps the backward of the others on the GPU.  The call returns
 * once every group is updated; the result (host model, master weights,
 * moments, zeroed accumulators) is bitwise that of the call followed by
 * atom_optimizer_step with the same arguments.  One-shot: the call consumes
 * it (also when it fails, in which case the update may cover only some
 * groups).  ATOM_ESTATE before atom_optimizer_init. */
int atom_optimizer_arm(atom_ctx* ctx, const atom_adamw* hp, float grad_scale, int32_t step);

/* Measured node costs for the planner (the per-layer profile of Section
 * III-D: loading time t^u, forward time t^f, backward time t^b and working
 * memory m_i, plus the time to store a node's gradients): each node's weights
 * copied alone to the device and its gradients back on the step's DMA engines
 * (best of three); the kernel time of each node's forward and backward (per
 * micro-batch, HIP events on the compute stream) in a step of the context's
 * plan on `tokens` (host int32 [accum][batch][seq_len + 1]) that follows one
 * untimed step on the same tokens; and mem_bytes, how far into the device
 * workspace the node's kernels wrote (the workspace is filled with a marker
 * word before each node runs and scanned after it; no workspace data outlives
 * a node, so the results are those of an ordinary step).  cut_bytes is the
 * node's output tensor (fp32 [batch][seq_len][d_model]; 4 for the head).
 * Both steps' gradients are added to the accumulators like atom_step's.
 * out: n = n_layer + 2 entries; pass them to atom_plan_partition or
 * atom_plan_predict.  Synchronous. */
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
  double host_update_s;      /* host time of an armed optimizer update (whole call) */
  int32_t updated_groups;    /* groups that update covered */
  int32_t opt_state_pinned;  /* optimizer state allocated in pinned memory (else pageable, or absent) */
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
