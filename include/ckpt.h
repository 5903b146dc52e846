/*
 * ckpt.h -- C ABI of libckpt: the checkpointed (sublinear-memory) training
 * step of Chen, Xu, Zhang and Guestrin, "Training Deep Nets with Sublinear
 * Memory Cost", on AMD Instinct MI355X (gfx950).
 *
 * The paper's problem (section 4.1): train an n-unit chain while keeping only
 * some intermediate results and recomputing the others during back-propagation.
 * Two calls carry it:
 *   plan_checkpoints(n, per-unit sizes, budget)  -> which boundaries to keep
 *   train_step(net, batch, plan)                 -> loss, every gradient, peak
 *                                                   activation bytes
 *
 * Conventions
 *   - Every function returning int returns CKPT_OK (0) or a negative CKPT_E_*
 *     code; ckpt_last_error() then describes the failure (thread-local string,
 *     valid until the next call on the same thread).
 *   - Arguments are validated before anything is launched on the GPU: a call
 *     that returns an error other than CKPT_E_HIP has enqueued no work.
 *   - "device" pointers are GPU memory (hipMalloc or torch tensors) that the
 *     caller owns; "host" pointers are ordinary CPU memory.  The library never
 *     allocates or frees device memory: the caller passes one workspace.
 *   - Unit i of the chain maps x_i to x_{i+1}; a cut at c keeps x_{c+1}.
 *   - Plans and nets are library-owned opaque objects, freed with plan_free /
 *     net_destroy.  They are immutable after creation and may be shared
 *     between threads; calls that use the same workspace must not overlap.
 */
#ifndef CKPT_H
#define CKPT_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- return codes ------------------------------------------------------ */
#define CKPT_OK              0
#define CKPT_E_INVALID     (-1)  /* bad argument (null pointer, size, cut list) */
#define CKPT_E_WORKSPACE   (-2)  /* workspace smaller than net_workspace_bytes  */
#define CKPT_E_MISMATCH    (-3)  /* plan built for a different unit count        */
#define CKPT_E_HIP         (-4)  /* a HIP runtime call failed (message has text) */
#define CKPT_E_UNSUPPORTED (-5)  /* valid request the library does not handle    */

/* ---- plan modes (section 4) --------------------------------------------- */
#define CKPT_NONE      0  /* one segment, activations of the first forward kept     */
#define CKPT_SQRT      1  /* section 4.3, Eq. 1: ceil(sqrt n) equal segments         */
#define CKPT_GREEDY    2  /* Alg. 3: budget-driven greedy segmentation               */
#define CKPT_RECURSIVE 3  /* section 4.4, Eq. 2-3: k splits per level, k log_{k+1} n */
#define CKPT_USER      4  /* explicit cut list: the user-set mirror attribute (4.5)  */

/* plan flags */
#define CKPT_FLAG_KEEP_LAST 1 /* one-level plans: reuse the last segment's first-
                                 forward activations instead of re-running it   */

typedef struct ckpt_plan ckpt_plan;
typedef struct ckpt_net ckpt_net;

/*
 * plan_checkpoints -- choose the boundaries to keep (section 4.3, Alg. 3,
 * section 4.4).
 *   n_layers     number of units n (> 0).
 *   layer_bytes  host [n]: bytes unit i holds while its segment is re-run
 *                (saved internals + output; Alg. 3's size-of-output).
 *   cut_bytes    host [n]: bytes of x_{i+1} when kept; 0 marks a boundary that
 *                is not a candidate split point (Alg. 3's set C).  The last
 *                entry must be 0: the chain's output feeds the loss (Alg. 1).
 *   budget       GREEDY: Alg. 3's per-segment budget B (bytes).  SQRT: the
 *                stride (units per segment) if > 0, else ceil(sqrt n).
 *                RECURSIVE: the fan-out k of section 4.4 (boundaries stored
 *                per level; 0 means 1, at most 2^31 - 1): a range of L > 1
 *                units splits into at most k + 1 parts at
 *                floor(j L / (k+1)), j = 1..k, repeats dropped; the parts
 *                are handled last to first.  Ignored by the other modes.
 *   mode         CKPT_NONE .. CKPT_USER.
 *   user_cuts    host [n_user_cuts], CKPT_USER only: strictly ascending
 *                candidate positions below n-1.
 *   flags        0 or CKPT_FLAG_KEEP_LAST.
 *   out          receives the new plan (free with plan_free).
 * Errors: CKPT_E_INVALID for n <= 0, null pointers, cut_bytes[n-1] != 0, an
 *   unknown mode, or a user cut list that is unsorted, repeated, out of range
 *   or on a non-candidate; CKPT_E_UNSUPPORTED for RECURSIVE on a chain with a
 *   non-candidate boundary; CKPT_E_INVALID for a RECURSIVE fan-out of 2^31
 *   or more.
 */
int plan_checkpoints(int32_t n_layers, const uint64_t *layer_bytes, const uint64_t *cut_bytes,
                     uint64_t budget, int32_t mode, const int32_t *user_cuts,
                     int32_t n_user_cuts, int32_t flags, ckpt_plan **out);

/*
 * plan_info -- summary of a plan.  Any output pointer may be null.
 *   mode, n_layers, n_cuts   as planned (RECURSIVE reports 0 cuts: its split
 *                            tree is implicit, the fan-out splits of every range)
 *   x, y                     Alg. 3's outputs for the plan's cut set: kept
 *                            boundary bytes, and the largest segment total
 *                            among segments ending at a cut (0 for RECURSIVE)
 *   extra_unit_forwards      unit forwards beyond the first pass: n for a
 *                            literal one-level plan (one extra forward pass,
 *                            section 4.3), fewer with KEEP_LAST, 0 for NONE,
 *                            the recursion's count for RECURSIVE.
 */
int plan_info(const ckpt_plan *plan, int32_t *mode, int32_t *n_layers, int32_t *n_cuts,
              uint64_t *x, uint64_t *y, uint64_t *extra_unit_forwards);

/* plan_cuts -- copy the ascending cut list into host cuts[cap]; *n_cuts gets
 * the full count (the copy is truncated to cap). */
int plan_cuts(const ckpt_plan *plan, int32_t *cuts, int32_t cap, int32_t *n_cuts);

/*
 * plan_serialize -- canonical little-endian bytes of the plan:
 *   "CKPL" u32 version=2, u32 mode, u32 keep_last, u32 fanout (RECURSIVE's
 *   k, else 0), u32 n, u32 n_cuts, i32 cuts[n_cuts], u64 x, u64 y,
 *   u64 extra_unit_forwards.
 * buf (host, cap bytes) may be null to query *len.  CKPT_E_INVALID if cap is
 * too small for a non-null buf.
 */
int plan_serialize(const ckpt_plan *plan, uint8_t *buf, uint64_t cap, uint64_t *len);

void plan_free(ckpt_plan *plan);

/*
 * plan_search -- the search over Alg. 3's budget B of the paper's appendix A:
 * run Alg. 3 with B = 0 to get x (kept bytes) and y (largest segment), set
 * B0 = floor(sqrt(x y)), try B0 and six budgets evenly spaced from
 * floor(B0 / sqrt 2) to floor(sqrt(2) B0) (integer steps j (hi - lo) / 5,
 * j = 0..5), and return the GREEDY plan whose exact PEAK under the static
 * layout below is lowest (ties: the smaller budget).  The returned plan is
 * identical to plan_checkpoints(GREEDY, *budget, flags).
 *   layer_bytes, cut_bytes: [n] as for plan_checkpoints (host).
 *   b [n+1], a [n], q [n]: the layout tables of net_unit_sizes (host).
 *   grad_slot: bytes of one gradient slot (0: the largest b_i, i >= 1);
 *   grad_extra: fixed gradient buffers (net_grad_bytes gives both).
 *   flags: CKPT_FLAG_KEEP_LAST or 0.
 *   out: new plan (free with plan_free); budget, peak: nullable outputs.
 * Errors: CKPT_E_INVALID as plan_checkpoints (null arrays, n <= 0,
 *   cut_bytes[n-1] != 0, unknown flags).
 */
int plan_search(int32_t n_layers, const uint64_t *layer_bytes, const uint64_t *cut_bytes,
                const uint64_t *b, const uint64_t *a, const uint64_t *q, uint64_t grad_slot,
                uint64_t grad_extra, int32_t flags, ckpt_plan **out, uint64_t *budget,
                uint64_t *peak);

/* ---- gradient graphs with mirror nodes (Alg. 2) and the static allocator
 *      of section 3 (liveness counters, in-place writes, memory sharing) ---- */
#define CKPT_NODE_INPLACE  1 /* the operator may write its output over its first input */
#define CKPT_NODE_GRAD_OUT 2 /* its backward reads the node's own output               */
#define CKPT_NODE_GRAD_IN  4 /* its backward reads the node's inputs                   */

#define CKPT_ALLOC_NONE    0 /* every output its own memory                           */
#define CKPT_ALLOC_INPLACE 1 /* + in-place writes over a dead first input              */
#define CKPT_ALLOC_SHARE   2 /* + sharing: dead outputs' memory recycled               */

#define CKPT_GNODE_FORWARD 0 /* kinds of the nodes of a planned gradient graph          */
#define CKPT_GNODE_MIRROR  1
#define CKPT_GNODE_GRAD    2

typedef struct ckpt_graph_plan ckpt_graph_plan;

/*
 * graph_plan -- Alg. 2's gradient-graph construction followed by section 3's
 * static memory allocation, for a forward computation graph at any
 * granularity.
 *   n_nodes    forward nodes (> 0), listed in a topological order.
 *   pred_ptr   host [n_nodes + 1]: CSR offsets into pred_idx (pred_ptr[0] = 0,
 *              non-decreasing).
 *   pred_idx   host [pred_ptr[n_nodes]]: the inputs of node v are
 *              pred_idx[pred_ptr[v] .. pred_ptr[v+1]), each < v.
 *   out_bytes  host [n_nodes]: bytes of each node's output.
 *   flags      host [n_nodes]: CKPT_NODE_* bits -- in-place capability and the
 *              minimum dependencies of the node's backward (section 3).
 *   mirror     host [n_nodes] or null (all 0): Alg. 2's m(v) >= 0, how many
 *              times v is recomputed for the backward pass (0: its output is
 *              kept); ignored for nodes without inputs.
 *   strategy   CKPT_ALLOC_*.
 * Construction: round k = 1 .. max m mirrors, in topological order, every v
 * with m(v) >= k on top of the current mirrors of its inputs.  The execution
 * order is the forward graph, then for v from last to first the not yet
 * scheduled ancestors of v's gradient node (in creation order) and the
 * gradient node, which reads the successors' gradient nodes, v's (latest)
 * output if CKPT_NODE_GRAD_OUT and its inputs' if CKPT_NODE_GRAD_IN, and
 * produces the gradients of v's inputs (the sum of their bytes).
 * Allocation: one pass over that order with a liveness counter per output;
 * an in-place node whose first input's counter is 1 reuses that input's
 * memory (strategies INPLACE, SHARE); under SHARE an output whose counter
 * reaches 0 returns its memory to a pool, from which a new output takes the
 * smallest block that fits (lowest id on ties).  The peak is the total of
 * the memory blocks assigned before execution.
 *   out        receives the plan (free with graph_plan_free).
 * Errors: CKPT_E_INVALID for n_nodes <= 0, null arrays, an input that is not
 *   an earlier node, negative mirror counts, unknown flags or strategy.
 */
int graph_plan(int32_t n_nodes, const int32_t *pred_ptr, const int32_t *pred_idx,
               const uint64_t *out_bytes, const int32_t *flags, const int32_t *mirror,
               int32_t strategy, ckpt_graph_plan **out);

/* graph_plan_info -- nodes executed (forward, mirror and gradient), mirror
 * nodes executed, memory blocks and the peak bytes.  Outputs nullable. */
int graph_plan_info(const ckpt_graph_plan *plan, int32_t *n_exec, int32_t *n_mirror,
                    int32_t *n_blocks, uint64_t *peak_bytes);

/* graph_plan_schedule -- the execution order, one entry per executed node:
 * kind (CKPT_GNODE_*), the forward node it derives from, and the memory block
 * its output uses (-1: no output).  Host arrays of cap entries (each may be
 * null); *n_exec gets the full count (the copy is truncated to cap). */
int graph_plan_schedule(const ckpt_graph_plan *plan, int32_t *kind, int32_t *of, int32_t *block,
                        int32_t cap, int32_t *n_exec);

/* graph_plan_blocks -- bytes of each memory block, host [cap]; *n_blocks gets
 * the full count. */
int graph_plan_blocks(const ckpt_graph_plan *plan, uint64_t *bytes, int32_t cap, int32_t *n_blocks);

void graph_plan_free(ckpt_graph_plan *plan);

/* ---- networks --------------------------------------------------------- */
/* (the node-graph calls net_node_graph, graph_workspace_bytes and
 *  train_step_graph follow train_step below) */
#define CKPT_NET_MLP               1 /* y = x + relu(x W + b) blocks, MSE head        */
#define CKPT_NET_RESNET_BASIC      2 /* CIFAR stem + 3 stages of basic blocks + FC-CE */
#define CKPT_NET_LSTM              3 /* LSTM steps, each with a softmax head          */
#define CKPT_NET_RESNET_BOTTLENECK 4 /* 7x7 stem + bottleneck stages + FC-CE, bf16     */

typedef struct ckpt_net_desc {
  int32_t kind;          /* CKPT_NET_*                                             */
  int32_t batch;         /* samples per step                                       */
  int32_t depth;         /* MLP: blocks.  RESNET_BASIC: basic blocks per stage.
                            LSTM: time steps T.  RESNET_BOTTLENECK: stages (1-4)   */
  int32_t width;         /* MLP: width.   RESNET_BASIC: first-stage channels.
                            LSTM: hidden size H.
                            RESNET_BOTTLENECK: first-stage bottleneck width        */
  int32_t image;         /* RESNET_*: input side (square images, 3 channels).
                            LSTM: input size E                                     */
  int32_t n_classes;     /* RESNET_*: classifier outputs.  LSTM: vocabulary V      */
  int32_t grad_chunk;    /* LSTM: time steps per weight-gradient chunk (0 = 32)    */
  int32_t stage_blocks[4]; /* RESNET_BOTTLENECK: blocks per stage (zero past depth) */
  int32_t expansion;     /* RESNET_BOTTLENECK: output channels / bottleneck width  */
  int32_t stem_channels; /* RESNET_BOTTLENECK: channels of the stem's output       */
  int32_t drop_bn_relu;  /* RESNET_BASIC: 1 = keep only convolution outputs and
                            re-form relu(bn(.)) from them and their statistics
                            when read (smaller saved internals, same gradients)  */
  int32_t reserved[2];   /* must be zero                                           */
} ckpt_net_desc;

/*
 * net_create -- build the unit chain described by desc (host only).
 *   MLP:          n = depth units; parameters per unit W [width, width]
 *                 (x W, row-major [in, out]) then b [width]; input x0 f32
 *                 [batch, width]; target f32 [batch, width]; loss = mean
 *                 squared error over all elements.
 *   RESNET_BASIC: n = 1 + 3*depth units: stem conv3x3 3->width + BN + ReLU,
 *                 then basic blocks (conv3x3-BN-ReLU-conv3x3-BN, identity or
 *                 option-A shortcut, ReLU) of width, 2 width, 4 width channels
 *                 with stride-2 transitions; head = global average pool, FC
 *                 [4 width, n_classes] + bias, softmax cross-entropy averaged
 *                 over the batch.  Conv weights [Cout,3,3,Cin]; input f32 NHWC
 *                 [batch, image, image, 3]; target int32 [batch].
 *   LSTM:         n = T units, one per time step: z = x_t W_x + h W_h + b with
 *                 gates i, f, g, o in column blocks of H, c = f c + i g,
 *                 h = o tanh c; per-step head logits = h W_o + b_o, softmax
 *                 cross-entropy averaged over T*batch (section 5.3's long
 *                 unrolled LSTM).  Parameters W_x [E,4H], W_h [H,4H], b [4H],
 *                 W_o [H,V], b_o [V]; input bf16 [T, batch, E]; target int32
 *                 [T, batch].  GEMM operands are bf16 (weights rounded once per
 *                 step), accumulation and the cell state fp32, h bf16.  Sizes
 *                 must be multiples of 8.
 *   RESNET_BOTTLENECK: n = 1 + sum(stage_blocks) units: stem conv7x7/2 (pad 3)
 *                 3 -> stem_channels + BN + ReLU + max pool 3x3/2 (pad 1); then
 *                 per stage t bottleneck blocks conv1x1 (width 2^t) - BN - ReLU
 *                 - conv3x3 (stride 2 in the first block of stages t > 0) - BN
 *                 - ReLU - conv1x1 (expansion x width 2^t) - BN, + shortcut
 *                 (projection conv1x1 with the block's stride + BN in each
 *                 stage's first block, else identity), ReLU; head as
 *                 RESNET_BASIC (section 5.2's deep residual network).  Parameter
 *                 order per block: W1, gamma1, beta1, W2, gamma2, beta2, W3,
 *                 gamma3, beta3 [, Wp, gammap, betap]; conv weights [Cout, R, R,
 *                 Cin].  Input bf16 NHWC [batch, image, image, 3]; target int32
 *                 [batch].  Activations bf16, convolutions accumulate in fp32,
 *                 batch-norm statistics from float64 sums.  Channel counts must
 *                 be powers of two in [8, 2048] (CKPT_E_UNSUPPORTED otherwise)
 *                 and every stride-2 stage input side even.
 * Errors: CKPT_E_INVALID for a null pointer, an unknown kind, a field another
 *   kind uses set to non-zero, or a non-positive or inconsistent size.
 */
int net_create(const ckpt_net_desc *desc, ckpt_net **out);
void net_destroy(ckpt_net *net);

/* net_units -- number of units n in the chain. */
int net_units(const ckpt_net *net, int32_t *n);

/*
 * net_unit_sizes -- the static layout's byte tables (host arrays, any may be
 * null): b[n+1] boundary x_i bytes, a[n] saved internals, q[n] gradient
 * scratch.  Every tensor is rounded up to 256 bytes.
 */
int net_unit_sizes(const ckpt_net *net, uint64_t *b, uint64_t *a, uint64_t *q);

/*
 * net_grad_bytes -- the gradient part of the static layout: one gradient slot
 * (the gradient of a boundary; two are used in turn) and the unit kind's
 * fixed gradient buffers (the LSTM's weight-gradient chunk buffers; 0 for the
 * others).  Either output may be null.
 */
int net_grad_bytes(const ckpt_net *net, uint64_t *slot, uint64_t *extra);

/* net_layer_sizes -- plan_checkpoints inputs: layer_bytes[i] = a_i + b_{i+1},
 * cut_bytes[i] = b_{i+1} (0 for the last unit).  Host arrays of n entries. */
int net_layer_sizes(const ckpt_net *net, uint64_t *layer_bytes, uint64_t *cut_bytes);

/*
 * Parameters and gradients live in two caller-owned device buffers of
 * net_param_bytes bytes each, f32, tensor k at byte offset *offset with
 * *numel elements (256-byte aligned, in chain order, head last).  The name is
 * "u<i>.<tensor>" or "head.<tensor>" (copied into host name[cap], NUL-ended).
 */
int net_param_bytes(const ckpt_net *net, uint64_t *bytes);
int net_param_count(const ckpt_net *net, int32_t *count);
int net_param_info(const ckpt_net *net, int32_t k, char *name, int32_t cap, uint64_t *offset,
                   uint64_t *numel);

/*
 * plan_accounting -- exact feature-map bytes of the plan on this net (the
 * cost a static allocation gives, section 5.1; parameters and operator
 * workspace excluded): kept boundaries (ckpt), the re-run arena (arena) and
 * the gradient buffers (grad); peak = ckpt + arena + grad.  Any output may be
 * null.  CKPT_E_MISMATCH if the plan's n differs from the net's.
 */
int plan_accounting(const ckpt_net *net, const ckpt_plan *plan, uint64_t *ckpt, uint64_t *arena,
                    uint64_t *grad, uint64_t *peak);

/* net_workspace_bytes -- size of the single device workspace train_step needs
 * for this plan: peak plus operator workspace (loss partials, reduction
 * partials, head buffers), each region 256-byte aligned. */
int net_workspace_bytes(const ckpt_net *net, const ckpt_plan *plan, uint64_t *bytes);

typedef struct ckpt_batch {
  const void *input;   /* device: MLP f32 [batch,width]; RESNET_BASIC f32 NHWC images;
                          LSTM bf16 [T,batch,E]                                        */
  const void *target;  /* device: MLP f32 [batch,width]; RESNET_BASIC int32 [batch];
                          LSTM int32 [T,batch]                                         */
} ckpt_batch;

typedef struct ckpt_step_stats {
  uint64_t unit_forwards;   /* unit forward passes run (n + extra)                */
  uint64_t unit_backwards;  /* unit backward passes run (n)                       */
  uint64_t kernel_launches; /* kernels enqueued by this step                      */
  uint64_t ckpt_bytes, arena_bytes, grad_bytes; /* plan_accounting of this step   */
} ckpt_step_stats;

/*
 * train_step -- one checkpointed training step (Alg. 1 for one-level plans,
 * the section 4.4 recursion for RECURSIVE): forward keeping only the plan's
 * boundaries, the loss head, then for each segment in reverse order its
 * forward re-run from the kept boundary followed by its backward.
 *   params     device f32, net_param_bytes (read only)
 *   grads      device f32, net_param_bytes: every gradient is overwritten
 *   batch      device input/target pointers (read only)
 *   workspace  device, >= net_workspace_bytes(net, plan) bytes, 256-aligned;
 *              contents on entry are ignored
 *   stream     hipStream_t to enqueue on (null = the default stream)
 *   loss_dev   nullable device f32 scalar receiving the loss (asynchronous)
 *   loss_host  nullable host float: if given, the stream is synchronised and
 *              the loss copied here
 *   peak       nullable host: the plan's peak activation bytes
 *   stats      nullable host: counters of this step
 * The gradients are bit-identical for every plan of the same net: every
 * kernel reduces in a fixed order and recomputation reproduces the first
 * forward exactly (section 5.1: the same weight gradient).
 * Errors: CKPT_E_INVALID (null net/params/grads/batch/plan/workspace, or an
 *   unaligned workspace), CKPT_E_MISMATCH, CKPT_E_WORKSPACE, CKPT_E_HIP.
 */
int train_step(ckpt_net *net, const void *params, void *grads, const ckpt_batch *batch,
               const ckpt_plan *plan, void *workspace, uint64_t workspace_bytes, void *stream,
               float *loss_dev, float *loss_host, uint64_t *peak, ckpt_step_stats *stats);

/*
 * train_step_static -- train_step for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc): the same step with the same arguments minus the
 * workspace, which is instead a fixed scratch array of
 * CKPT_STATIC_SCRATCH_BYTES the library holds on each GPU it runs on (from
 * the first call on that GPU until the process ends).  It calls no
 * hipMalloc, hipFree or other allocating routine.  The scratch of the calling
 * thread's current device (hipGetDevice) is used; `stream` must belong to
 * that device.  Results equal train_step's bit for bit (same kernels, same
 * layout).  Every call on one GPU shares that GPU's scratch, which keeps the
 * last call's contents (the step ignores them on entry); calls that overlap
 * in time on one GPU race on it.
 * Errors: as train_step; CKPT_E_WORKSPACE when net_workspace_bytes(net, plan)
 *   exceeds CKPT_STATIC_SCRATCH_BYTES; CKPT_E_INVALID with kernel timing on
 *   (timing creates events).
 */
#define CKPT_STATIC_SCRATCH_BYTES (64u << 20)
int train_step_static(ckpt_net *net, const void *params, void *grads, const ckpt_batch *batch,
                      const ckpt_plan *plan, void *stream, float *loss_dev, float *loss_host,
                      uint64_t *peak, ckpt_step_stats *stats);

/*
 * Recorded steps.  A checkpointed step is a fixed sequence of small kernels
 * (the plan fixes every launch and every buffer: section 4's static plan);
 * recording it once as a HIP graph and launching the graph replaces the
 * per-kernel host submissions with one.
 *
 * step_graph_create -- record one train_step with these arguments (loss to
 *   loss_dev only; no host loss, no peak) on `stream` and instantiate it.
 *   Nothing runs while recording.  stream must be a created stream (not the
 *   default one) that is not already being captured; kernel timing must be
 *   off.  *out receives the recorded step; stats (nullable) the step's
 *   counters.  The recorded step keeps the addresses of params, grads, the
 *   batch buffers, workspace and loss_dev: they must stay allocated while it
 *   exists, and each launch reads their contents at that time.
 * step_graph_launch -- enqueue the recorded step on `stream` (null = default);
 *   its results are those of train_step with the same arguments, bit for bit.
 *   Launches on one stream run in order; two launches of one recorded step
 *   that overlap in time (different streams, no ordering) race on its buffers.
 * step_graph_free -- release a recorded step (null is a no-op); launches
 *   already enqueued complete normally.
 * Errors: as train_step; CKPT_E_INVALID for the default stream, a stream
 *   under capture or timing on; CKPT_E_HIP when recording, instantiation or
 *   the launch fails.
 */
typedef struct ckpt_step_graph ckpt_step_graph;
int step_graph_create(ckpt_net *net, const void *params, void *grads, const ckpt_batch *batch,
                      const ckpt_plan *plan, void *workspace, uint64_t workspace_bytes,
                      void *stream, float *loss_dev, ckpt_step_graph **out,
                      ckpt_step_stats *stats);
int step_graph_launch(ckpt_step_graph *graph, void *stream);
void step_graph_free(ckpt_step_graph *graph);

/*
 * net_node_graph -- the net's forward graph at operator granularity, in the
 * form graph_plan takes (section 3's computation graph; Alg. 2 plans mirror
 * counts on it).  Provided for CKPT_NET_MLP: node 0 is the input; block i is
 * 1 + 3i fully connected (x W + b, backward reads its input), 2 + 3i ReLU
 * (in place, backward reads its output), 3 + 3i add (ReLU output + block
 * input, in place); node 3n + 1 is the MSE loss (its output is the loss
 * gradient).  Every node's output is one [batch, width] f32 tensor.
 *   n_nodes: receives the node count; pred_ptr host [n_nodes + 1], pred_idx
 *   host [edges], out_bytes, flags host [n_nodes]: filled when cap_nodes and
 *   cap_edges are large enough (query with null arrays first); *n_edges gets
 *   the edge count.
 * Errors: CKPT_E_UNSUPPORTED for other nets; CKPT_E_INVALID for a null net
 *   or arrays that are too small.
 */
int net_node_graph(const ckpt_net *net, int32_t *n_nodes, int32_t *n_edges, int32_t *pred_ptr,
                   int32_t *pred_idx, uint64_t *out_bytes, int32_t *flags, int32_t cap_nodes,
                   int32_t cap_edges);

/* graph_workspace_bytes -- workspace train_step_graph needs for a graph plan
 * of this net's node graph: the plan's memory blocks (each 256-byte aligned)
 * plus the operator workspace (partial sums, loss, one tensor for adding the
 * gradients of a node with several readers).  CKPT_E_MISMATCH if the plan is
 * not of net_node_graph's graph, CKPT_E_UNSUPPORTED for nets without one. */
int graph_workspace_bytes(const ckpt_net *net, const ckpt_graph_plan *plan, uint64_t *bytes);

/*
 * train_step_graph -- one training step over the node graph in the order and
 * memory blocks of a graph plan (Alg. 2's gradient graph with mirror nodes:
 * the forward graph, then each gradient node preceded by the mirrors it needs;
 * every output in its planned block).  Arguments as for train_step, with a
 * graph plan of net_node_graph's graph and a workspace of
 * graph_workspace_bytes; *peak receives the plan's planned bytes.  stats:
 * unit_forwards = forward and mirror nodes run, unit_backwards = gradient
 * nodes run, arena_bytes = planned bytes.  The gradients equal train_step's
 * bit for bit for every plan.
 * Errors: as train_step; CKPT_E_UNSUPPORTED for nets without a node graph.
 */
int train_step_graph(ckpt_net *net, const void *params, void *grads, const ckpt_batch *batch,
                     const ckpt_graph_plan *plan, void *workspace, uint64_t workspace_bytes,
                     void *stream, float *loss_dev, float *loss_host, uint64_t *peak,
                     ckpt_step_stats *stats);

/*
 * net_set_side_stream -- lets (enable = 1, the default) or stops (0) a net run
 * part of each unit's backward on a second stream of its own.  The
 * RESNET_BOTTLENECK net uses one for its units' weight gradients (Alg. 1's
 * backward of a unit: the weight-gradient products do not feed the input
 * gradient, so they run beside it), ordered with the step's stream by events:
 * each waits for the gradient it reads, and the step's stream waits for them
 * before it next writes what they read (the next unit's gradient scratch, a
 * re-run's activations) and at the step's end; other nets run everything on
 * the step's stream.  The gradients are the same bits either way.  The stream
 * and its events are created by the
 * first train_step or step_graph_create that can use them (not by a step whose
 * stream is being captured, and not by train_step_static, which allocates
 * nothing: those use the second stream only once it exists), on the device
 * of the step's stream when that device is current; they are released by
 * net_destroy.  A step on another device than the one they were created on
 * runs on its own stream alone.
 * Errors: CKPT_E_INVALID for a null net; CKPT_E_HIP when creating them fails
 * (reported by the step that tries).
 */
int net_set_side_stream(ckpt_net *net, int32_t enable);

/*
 * Kernel timing for benchmarks.  net_timing_enable(net, 1) makes every later
 * train_step bracket each launch of the net's dominant kernel family (the
 * conv3x3 forward / data-gradient kernel of RESNET_BASIC, the GEMM of MLP)
 * with a pair of HIP events on the step's stream, and resets the totals;
 * 0 turns it off.  net_timing_read synchronises on the recorded events and
 * returns, since the last enable: the launches timed, their summed duration
 * (ms), their summed algorithmic flops and bytes (each operand read once, each
 * result written once), and the family's kernel-name prefix (host name[cap]).
 * The events add a little time to each step: time throughput separately.
 */
int net_timing_enable(ckpt_net *net, int32_t enable);
int net_timing_read(ckpt_net *net, uint64_t *launches, double *ms, double *flops, double *bytes,
                    char *name, int32_t cap);
/*
 * The same timed launches against their own rooflines: *roofline_ms = the sum
 * over the launches of max(flops / peak_flops, bytes / peak_bytes_per_s) (the
 * time each would take at the bound of its own arithmetic intensity), and
 * *kernel_ms = their summed measured duration, so a family of launches with
 * different bounds gets one fraction of its roofline, roofline_ms / kernel_ms.
 * *busy_ms = the time during which at least one of them ran (the union of
 * their intervals on the device clock): below kernel_ms when launches on the
 * net's side stream overlap launches on the step's stream.  Any output may be
 * null.  Peaks in flop/s and byte/s, both > 0 (CKPT_E_INVALID otherwise).
 */
int net_timing_roofline(ckpt_net *net, double peak_flops, double peak_bytes_per_s,
                        double *roofline_ms, double *kernel_ms, double *busy_ms);

/* ---- operator calls -----------------------------------------------------
 * The single operators the bf16 bottleneck units (section 5.2's deep residual
 * network, built from the conv-BN-activation pipeline of section 4.2) are
 * made of, each one launch (or a fixed short sequence) of exactly the kernels
 * train_step runs, on caller buffers: a caller can check or compose one
 * operator on inputs of its choice.  Tensors are NHWC, channel counts powers
 * of two >= 8; "bf16" buffers hold bfloat16, "f32" float, "f64" double.
 * All buffers are device memory the caller owns and sizes; the library cannot
 * check their extents (a short buffer is a GPU memory fault).  Work is
 * enqueued on `stream` (null = the default stream) and nothing is
 * synchronised.  Arguments are validated before any launch (CKPT_E_INVALID,
 * CKPT_E_UNSUPPORTED); a failed launch returns CKPT_E_HIP.
 */
#define CKPT_EPI_STORE     0 /* C = product                                          */
#define CKPT_EPI_ADD       1 /* C = product + D (D may alias C)                      */
#define CKPT_EPI_BF16STATS 3 /* Cb (bf16) = bf16(product); per row tile of the GEMM,
                                f64 column sums of the rounded values and their
                                squares: stats[row tile][2][n] (batch-norm input)    */
#define CKPT_EPI_ADDMASK   4 /* C = product + (mask > 0 ? D : 0), mask bf16 like D   */
#define CKPT_EPI_BNBWD     6 /* the gradient reaching a batch norm's output through a
                                ReLU: C = ds = (mask > 0 ? product : 0), and per row
                                tile f64 column sums of ds and ds * xhat,
                                xhat = (cv - bst[col]) * bst[n + col], block-major
                                stats[row tile][2][n]                               */

/* op_gemm_bf16_blocks -- row and column tiles the bf16 GEMM uses for an
 * [m, n] product (row tiles = the leading dimension of the per-tile stats of
 * BF16STATS / BNBWD).  Either output may be null. */
int op_gemm_bf16_blocks(int32_t m, int32_t n, int32_t *row_blocks, int32_t *col_blocks);

/*
 * op_gemm_bf16 -- C[m, n] (f32) = epi(op(A) op(B)), products accumulated in
 * fp32 over k in one fixed order (a 1x1 convolution of NHWC tensors is this
 * product with m = pixels).  A bf16 (or f32 rounded to bf16 on load when
 * a_fp32, STORE / ADD only); ak: A[i * lda + k] (k contiguous), else
 * A[k * lda + i]; B bf16, bk: B[j * ldb + k], else B[k * ldb + j]; C / D /
 * mask / cv row stride ldc / ldd.  splits > 1 (STORE only): C receives
 * `splits` partial products [m, ldc] over consecutive k ranges, to be added
 * in order (op_sum_partials).  BF16STATS writes cb (bf16, stride ldc) and
 * stats instead of C; BNBWD needs k-contiguous bf16 A, n-contiguous B,
 * ldc == n, one split, mask, cv, bst and stats.  bias (nullable, STORE):
 * + bias[j].
 */
int op_gemm_bf16(int32_t m, int32_t n, int32_t k, const void *a, int32_t a_fp32, int32_t lda,
                 int32_t ak, const void *b, int32_t ldb, int32_t bk, float *c, int32_t ldc,
                 int32_t epi, const float *d, int32_t ldd, const float *bias, int32_t splits,
                 const void *mask, void *cb, double *stats, const void *cv, const float *bst,
                 void *stream);

/* op_sum_partials -- out[e] = sum over b = 0..nb-1 (in order) of
 * part[b * count + e], f32, 0 < count < 2^31. */
int op_sum_partials(const float *part, int32_t nb, int64_t count, float *out, void *stream);

/* Geometry of an r x r convolution with stride s (1 or 2) and zero padding
 * p: input [n, h, w, ci], output [n, ho, wo, co], weights [co, r, r, ci];
 * ho = (h + 2p - r) / s + 1, wo likewise; n h w below 2^24. */
typedef struct ckpt_conv_geo {
  int32_t n, h, w, ci, ho, wo, co, r, s, p;
} ckpt_conv_geo;

/* op_conv_bf16_fwd -- y (bf16) = bf16(conv(x, w)), x and w bf16, as an
 * implicit GEMM (m = n ho wo output pixels, k = r r ci); stats as for
 * BF16STATS with op_gemm_bf16_blocks(n ho wo, co) row tiles. */
int op_conv_bf16_fwd(const ckpt_conv_geo *geo, const void *x, const void *w, void *y, double *stats,
                     void *stream);

/* op_conv_bf16_dgrad -- dx (f32, [n, h, w, ci]) = the data gradient of the
 * convolution for dy (bf16, [n, ho, wo, co]) through w (bf16), with epilogue
 * STORE, ADD (+ d), ADDMASK (+ d where mask > 0) or BNBWD (mask, cv, bst,
 * stats as for op_gemm_bf16 with op_gemm_bf16_blocks(n h w, ci) row tiles);
 * d, mask and cv shaped like dx (mask, cv bf16). */
int op_conv_bf16_dgrad(const ckpt_conv_geo *geo, const void *dy, const void *w, float *dx, int32_t epi,
                       const float *d, const void *mask, const void *cv, const float *bst,
                       double *stats, void *stream);

/* op_conv_bf16_wgrad -- dw (f32, [co, r, r, ci]) = the weight gradient from x
 * (bf16 input) and dy (bf16 output gradient), summed over the n ho wo output
 * pixels; splits > 1 splits that sum into `splits` partials in part (f32,
 * splits co r r ci) added in a fixed order. */
int op_conv_bf16_wgrad(const ckpt_conv_geo *geo, const void *x, const void *dy, float *part,
                       int32_t splits, float *dw, void *stream);

/* op_bn_finalize -- batch-norm statistics from f64 partial sums of nb blocks
 * over m values per channel, j channels; channel_major: part[2][j][nb], else
 * part[nb][2][j].  Forward (backward = 0): out[0..j) = mean, out[j..2j) =
 * 1/sqrt(biased variance + 1e-5) from the sums of v and v^2.  Backward: from
 * the sums of ds and ds * xhat, out[0..j) = their mean over m, out[j..2j) =
 * the mean of ds * xhat, dbeta = sum ds, dgamma = sum ds * xhat. */
int op_bn_finalize(int32_t backward, const double *part, int32_t nb, int32_t j, int64_t m, float *out,
                   float *dgamma, float *dbeta, int32_t channel_major, void *stream);

/* op_bnb_partial_blocks -- partial-sum blocks op_bnb_backward uses for p
 * pixels of j channels (its part holds nb * 2j doubles). */
int op_bnb_partial_blocks(int64_t p, int32_t j, int32_t *nb);

#define CKPT_BNB_RES_NONE 0 /* y = relu(bn(c))                                     */
#define CKPT_BNB_RES_ID   1 /* y = relu(bn(c) + x), x bf16 like c                   */
#define CKPT_BNB_RES_BN   2 /* y = relu(bn(c) + bn_p(x)), the projection's batch norm
                               with statistics stp, scale gp, shift bp             */
/* op_bnb_apply -- y (bf16, [p, j]) = bf16(relu(gamma (c - mean) rstd + beta
 * [+ shortcut])), c bf16 [p, j], st = mean [j] | rstd [j] (f32). */
int op_bnb_apply(int32_t res, int64_t p, int32_t j, const void *c, const float *st, const float *gamma,
                 const float *beta, const void *x, const float *stp, const float *gp, const float *bp,
                 void *y, void *stream);

/* op_bnb_backward -- the batch-norm backward for ds = (ym > 0 ? g : 0)
 * (ym bf16, nullable: ds = g), g f32 [p, j], c the batch norm's bf16 input
 * with statistics st: dbeta = sum ds, dgamma = sum ds xhat, d (bf16) =
 * bf16(gamma rstd (ds - mean(ds) - xhat mean(ds xhat))); part holds
 * op_bnb_partial_blocks(p, j) * 2j doubles, sums 2j floats (the two means).
 * p < 2^31. */
int op_bnb_backward(int64_t p, int32_t j, const float *g, const void *ym, const void *c, const float *st,
                    const float *gamma, double *part, float *sums, float *dgamma, float *dbeta, void *d,
                    void *stream);

/* op_bnb_backward_apply -- the element pass of op_bnb_backward alone, given
 * sums (2j floats from op_bn_finalize(backward = 1)). */
int op_bnb_backward_apply(int64_t p, int32_t j, const float *g, const void *ym, const void *c,
                          const float *st, const float *gamma, const float *sums, void *d,
                          void *stream);

/* op_im2col7 -- col (bf16, [n ho wo, kp]) = the 7x7 stride-2 pad-3 patches
 * of x (bf16 [n, h, w, 3]) in (kh, kw, c) order in the first 147 columns of
 * each row, zero outside the image and in the columns past 147; kp = 147 or
 * a multiple of 8 above it (the network uses 160, rows a GEMM can load in
 * 16-byte chunks). */
int op_im2col7(int32_t n, int32_t h, int32_t w, int32_t ho, int32_t wo, int32_t kp, const void *x,
               void *col, void *stream);

/* op_maxpool -- 3x3 stride-2 pad-1 max pool of r (bf16 [n, h, w, c]):
 * forward (backward = 0) out = y (bf16 [n, ho, wo, c]); backward out = dr
 * (f32 [n, h, w, c]): each window's g (f32 [n, ho, wo, c]) goes to the first
 * maximum of the window in row-major order (y the forward's output).  arg
 * (backward only, n ho wo c bytes of workspace, or null): two passes (each
 * window's first-maximum tap, then the sum per input pixel, the network's
 * form) instead of one; the same result. */
int op_maxpool(int32_t backward, int32_t n, int32_t h, int32_t w, int32_t c, int32_t ho, int32_t wo,
               const float *g, const void *r, const void *y, void *out, void *arg, void *stream);

/* ckpt_last_error -- message of the last failed call on this thread ("" if
 * none). */
const char *ckpt_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* CKPT_H */
