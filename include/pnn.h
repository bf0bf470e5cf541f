/*
 * libpnn -- the training forward / backward pass of a parareal neural network (Lee, Lee & Park,
 * "Parareal Neural Networks Emulating a Parallel-in-time Algorithm") on one AMD Instinct MI355X
 * (gfx950).
 *
 * The network f-bar (eq. (barf)) is h o [coarse correction] o {g^j o C^j}_{j=1..N}:
 *
 *   x_j = C^j(x),  y_j = g^j(x_j)                    (eq. (xjyj), Alg. para2)      pnn_pre_fwd,
 *                                                                                  parareal_fine_fwd
 *   r_j = y_j - x_{j+1} (j < N), r_N = 0             (eq. (rk))                    parareal_combine_fwd
 *   rt_1 = r_1, rt_{j+1} = r_{j+1} + F^j(rt_j)       (eq. (tilderk))               coarse_fwd,
 *                                                                                  coarse_fwd_all
 *   ytilde = y_N + rt_N                              (eq. (tildey))                coarse_fwd (j = N-1)
 *   logits = h(ytilde), loss, D_N = dL/dytilde       (Alg. para3, first line)      pnn_head_fwd_bwd
 *   D_j = D_{j+1} . dF^j/drt_j, dL/deta_j            (Alg. para3, eq. (etak))      coarse_bwd,
 *                                                                                  coarse_bwd_all
 *   dL/dphi_j = D_j . dg^j/dphi_j, D_j . dg^j/dx_j   (Alg. para3, eq. (phij))      parareal_fine_bwd
 *   (the last two together, overlapped)                                            parareal_bwd
 *   dL/dx_j = D_j . dg^j/dx_j - D_{j-1}              (eq. (deltaj))                parareal_combine_bwd
 *   dL/ddelta_j                                       (eq. (deltaj))                pnn_pre_bwd
 *
 * All N fine sub-networks g^j run in the same kernel launches (grouped convolutions over N
 * independent weight sets).  The coarse network is sequential by definition (Sec. 3.1): one block
 * F^j per call (coarse_fwd / coarse_bwd) or the whole chain in order (coarse_fwd_all /
 * coarse_bwd_all / parareal_bwd).
 *
 * Conventions for every entry point
 *   - Every tensor pointer is a DEVICE pointer owned by the caller.  Activations are NHWC and
 *     dense ([batch][H][W][C]); convolution filters are [c_out][k][k][c_in].
 *   - Storage type: PNN_F32 plans store everything in float; PNN_BF16 plans store activations,
 *     activation gradients and filters as bfloat16 bit patterns (uint16_t) and keep BN
 *     parameters, every parameter gradient, the head and the loss in float.  Arithmetic is fp32
 *     (bf16 MFMA operands with fp32 accumulation).
 *   - Entry points never allocate memory, free or synchronise, and never create streams or
 *     events.  All work is ordered on the given stream.  parareal_fine_fwd / parareal_fine_bwd /
 *     parareal_bwd may run groups of sub-networks on up to pnn_set_streams() streams: the given
 *     one and internal streams of the plan (default priority), which first wait for the work
 *     enqueued on the given stream before the call; the given stream waits for all of them before
 *     the call returns.  pnn_set_streams creates those internal streams and their events (no
 *     device memory) and pnn_plan_destroy releases them; pnn_plan_create allocates host memory
 *     only.  So every compute call can be captured into a HIP graph, the first one included.
 *   - Alignment: every tensor pointer (activations, their gradients, the image) and every
 *     parameter / gradient / momentum buffer must be 16-byte aligned (the kernels move 16-byte
 *     chunks); the workspaces 256-byte aligned; labels, logits and the loss 4-byte aligned.  A
 *     violation returns PNN_ERR_ALIGN before anything is enqueued.
 *   - Workspaces: the caller allocates one "saved" buffer (activations kept from the forward for
 *     the backward; pnn_workspace_size(PNN_WS_SAVED)) and one "scratch" buffer (temporaries;
 *     PNN_WS_SCRATCH), both at least 256-byte aligned, and passes the same ones to every call of a
 *     step.  Calls that share a scratch buffer must not overlap in time.
 *   - Return value: PNN_OK (0) or a negative pnn_status; on error nothing has been enqueued,
 *     except for PNN_ERR_HIP (a launch failed; earlier launches of the same call may have run).
 *     No C++ exception crosses this interface.  Asynchronous kernel faults surface at the
 *     caller's next synchronisation.
 */
#ifndef PNN_H
#define PNN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int pnn_status;
enum {
  PNN_OK = 0,
  PNN_ERR_NULL = -1,        /* a required pointer is NULL */
  PNN_ERR_SHAPE = -2,       /* inconsistent shapes / node list */
  PNN_ERR_DTYPE = -3,       /* unknown storage type */
  PNN_ERR_WORKSPACE = -4,   /* unknown workspace kind */
  PNN_ERR_UNSUPPORTED = -5, /* a valid network this library does not run (e.g. channels not a multiple of 16) */
  PNN_ERR_HIP = -6,         /* a HIP call failed */
  PNN_ERR_INDEX = -7,       /* sub-network / coarse block index out of range */
  PNN_ERR_ALIGN = -8,       /* a pointer violates the alignment rules above */
  PNN_ERR_TOO_LARGE = -9    /* the problem exceeds the fixed scratch of an allocation-free entry point */
};

typedef enum { PNN_F32 = 0, PNN_BF16 = 1 } pnn_dtype;

/* Node kinds of a segment (see pnn_segment_desc). */
enum {
  PNN_OP_CONV = 0,     /* dst = conv_{k,stride,pad}(A) [+ res];  A = ReLU(BN_bn(src)) if bn >= 0 else src */
  PNN_OP_BNACT = 1,    /* dst = pool(ReLU(BN_bn(src))) [+ res];  pool = 2x2/2 max pool when pool == 2 */
  PNN_OP_MAXPOOL3 = 2  /* dst = 3x3 / stride 2 / pad 1 max pool of src (preprocessing only) */
};

/* One node.  Slots are tensors of the segment: slot 0 is its input.  Convolution is
 * cross-correlation with zero padding and no bias.  BN is batch normalisation in training mode
 * (batch statistics over N, H, W; biased variance; eps = 1e-5) with per-channel gamma / beta. */
typedef struct {
  int op;
  int src, dst;        /* slot indices */
  int bn;              /* BN instance applied to src (with ReLU) before the op, or -1 */
  int pool;            /* PNN_OP_BNACT: 0 or 2 */
  int k, stride, pad;  /* PNN_OP_CONV: k in {1, 3} */
  int cout;            /* PNN_OP_CONV: output channels */
  int res;             /* slot added to the result, or -1 */
} pnn_node_desc;

/* A segment: C^j, g^j or F^j as a list of nodes in evaluation order.  bn_slot[b] is the slot
 * that BN instance b normalises; all nodes naming b share its activation. */
typedef struct {
  int in_h, in_w, in_c;
  int n_nodes;
  const pnn_node_desc* nodes;
  int n_bn;
  const int* bn_slot;
  int out_slot;
} pnn_segment_desc;

/* The whole network (eq. (barf)): N preprocessing operators, N sub-networks, N-1 coarse blocks
 * and a head (global average pool + linear layer with bias, softmax cross-entropy). */
typedef struct {
  int dtype;                       /* pnn_dtype */
  int batch;
  int img_h, img_w, img_c;
  int n_sub;                       /* N >= 1 */
  int n_classes;
  const pnn_segment_desc* pre;     /* [N]   C^j : image  -> X_{j-1} */
  const pnn_segment_desc* fine;    /* [N]   g^j : X_{j-1} -> X_j    */
  const pnn_segment_desc* coarse;  /* [N-1] F^j : X_j -> X_{j+1}    */
} pnn_net_desc;

typedef struct pnn_plan pnn_plan;

/* Validate a network description and build a plan (shapes, parameter / workspace layouts, launch
 * schedules).  The description is copied; the caller may free it afterwards.  Allocates host
 * memory only.  Errors: PNN_ERR_NULL, PNN_ERR_DTYPE, PNN_ERR_SHAPE, PNN_ERR_UNSUPPORTED. */
pnn_status pnn_plan_create(const pnn_net_desc* desc, pnn_plan** out);
void pnn_plan_destroy(pnn_plan* plan);

typedef enum { PNN_WS_SAVED = 0, PNN_WS_SCRATCH = 1 } pnn_ws_kind;
pnn_status pnn_workspace_size(const pnn_plan* plan, int kind, size_t* bytes);

/* Parameter layout of one segment (part 0 = C^j, 1 = g^j, 2 = F^j; index j is 0-based).
 * A parameter buffer holds the conv filters of the segment's nodes in node order (storage type),
 * then gamma[C], beta[C] of every BN instance (float).  A gradient buffer has the same order with
 * everything in float.  offsets[i] (i < n_nodes) is the byte offset of node i's filter (or
 * SIZE_MAX for nodes without one); offsets[n_nodes + 2b] / [n_nodes + 2b + 1] are the offsets of
 * gamma / beta of BN b.  `offsets` needs n_nodes + 2 n_bn entries and may be NULL.  grad = 0:
 * parameter buffer, grad = 1: gradient buffer.  *total receives the buffer size in bytes. */
pnn_status pnn_param_layout(const pnn_plan* plan, int part, int j, int grad, size_t* offsets,
                            size_t* total);

/* Shape (H, W, C) of sub-network j's input x_j (which = 0) or output y_j (which = 1). */
pnn_status pnn_tensor_shape(const pnn_plan* plan, int which, int j, int* h, int* w, int* c);

/* ---- forward (Alg. para2) ----------------------------------------------------------------- */

/* x_j = C^j(image) for j = 0..N-1 (eq. (xjyj)).  image: [B][img_h][img_w][img_c]; x[j]: X_{j-1}
 * shaped.  delta[j]: parameter buffer of C^j (may be NULL when C^j has no parameters). */
pnn_status pnn_pre_fwd(pnn_plan* plan, const void* image, void* const* x, const void* const* delta,
                       void* saved, void* scratch, void* stream);

/* y_j = g^j(x_j) for all j in one set of grouped launches (Alg. para2, parallel loop).  Stores
 * the layer inputs and BN statistics needed by parareal_fine_bwd in `saved`. */
pnn_status parareal_fine_fwd(pnn_plan* plan, const void* const* x, const void* const* phi,
                             void* const* y, void* saved, void* scratch, void* stream);

/* r_j = y_j - x_{j+1}, j = 0..N-2 (eq. (rk)), r[j] shaped like y_j.  rnorm2 (nullable, float[N-1])
 * receives ||r_j||^2 (the interface mismatch the coarse network corrects, Sec. 3.1).  With a
 * scratch (nullable when rnorm2 is NULL) a non-finite element of some r_j sets non-finite flag 0
 * (pnn_inspect what = 5). */
pnn_status parareal_combine_fwd(pnn_plan* plan, const void* const* y, const void* const* x,
                                void* const* r, float* rnorm2, void* scratch, void* stream);

/* One coarse block, j = 0..N-2 (eq. (tilderk)): rt_next = add + F^j(rt_j).  Pass add = r_{j+1}
 * for j < N-2 and add = y_N for j = N-2; then rt_next = ytilde (eq. (tildey), r_N = 0).
 * rt_j: X_j shaped (rt_0 = r_0), rt_next and add: X_{j+1} shaped.  rt_next must not alias
 * rt_j. */
pnn_status coarse_fwd(pnn_plan* plan, int j, const void* rt_j, const void* eta_j, const void* add,
                      void* rt_next, void* saved, void* scratch, void* stream);

/* The whole coarse chain, j = 0..N-2 in order (eq. (tilderk), (tildey)): rt[j + 1] = add[j] +
 * F^j(rt[j]).  rt has N entries: rt[0] = r_0 is read, rt[1..N-2] = rt_1..rt_{N-2} and rt[N-1] =
 * ytilde are written; add[j] = r_{j+1} for j < N-2 and add[N-2] = y_N; eta[j] as for coarse_fwd.
 * rt[j + 1] must not alias rt[j].  Same arithmetic as the N-1 coarse_fwd calls, except that a
 * block's input BN statistics are summed by the previous block's last convolution as it writes
 * that input (one pass over rt_j fewer per block), in a different order. */
pnn_status coarse_fwd_all(pnn_plan* plan, void* const* rt, const void* const* eta,
                          const void* const* add, void* saved, void* scratch, void* stream);

/* Postprocessing h and the loss, forward and backward (Alg. para3, first line): logits =
 * mean_{h,w}(ytilde) W^T + b (eps = [W (classes x C) | b (classes)] float), loss = mean softmax
 * cross-entropy over the batch.  Writes logits[B][classes] (float, nullable), *loss (float,
 * device), D_N = dL/dytilde (X_N shaped) and deps = [dW | db] (float). labels: int32[B]; a label
 * outside [0, classes) makes that sample's loss term, and so *loss, NaN.  A non-finite loss or
 * element of deps sets non-finite flag 1 (pnn_inspect what = 5). */
pnn_status pnn_head_fwd_bwd(pnn_plan* plan, const void* ytilde, const float* eps,
                            const int32_t* labels, float* logits, float* loss, void* D_N,
                            float* deps, void* scratch, void* stream);

/* For callers that cannot allocate device memory or hand over a workspace (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): pnn_head_fwd_bwd with the same
 * arguments and results, minus the scratch workspace.  Its temporaries (B * (C + classes + 1)
 * floats for a batch of B and C channels of ytilde) live in a fixed 4 MiB device array of the
 * library, one per GPU, kept until the process ends; a larger problem returns PNN_ERR_TOO_LARGE.
 * Calls nothing that allocates.  The first call on a device (with that device current) looks up
 * the array's address (PNN_ERR_HIP if that fails).  Every call on one GPU shares that array:
 * calls that overlap in time on one GPU race.  It raises no non-finite flag (they live in the
 * scratch workspace). */
pnn_status pnn_head_fwd_bwd_noalloc(pnn_plan* plan, const void* ytilde, const float* eps,
                                    const int32_t* labels, float* logits, float* loss, void* D_N,
                                    float* deps, void* stream);

/* ---- backward (Alg. para3) ---------------------------------------------------------------- */

/* D_j = D_{j+1} . dF^j/drt_j and deta_j = D_{j+1} . dF^j/deta_j (eq. (etak)), j = N-2..0,
 * called in that order.  D_next: X_{j+1} shaped, D_j: X_j shaped (must not alias D_next),
 * deta_j: gradient buffer of F^j (overwritten). */
pnn_status coarse_bwd(pnn_plan* plan, int j, const void* D_next, const void* rt_j,
                      const void* eta_j, const void* saved, void* D_j, float* deta_j,
                      void* scratch, void* stream);

/* The whole coarse chain at once: for j = N-2 .. 0 the data gradients D_j as coarse_bwd computes
 * them, then every deta_j (the weight gradients do not feed the chain, Alg. para3) in grouped
 * launches.  D[N-1] = D_N is read, D[0..N-2] are written (D[j] must not alias D[j+1]); rt[j],
 * eta[j], deta[j] for j = 0..N-2.  Same results as the N-1 coarse_bwd calls. */
pnn_status coarse_bwd_all(pnn_plan* plan, void* const* D, const void* const* rt,
                          const void* const* eta, const void* saved, float* const* deta,
                          void* scratch, void* stream);

/* For all j at once (Alg. para3, parallel loop; dL/dy_j = D_j by eq. (ingredient1)):
 * dphi[j] = D_j . dg^j/dphi_j (gradient buffer, overwritten) and dx[j] = D_j . dg^j/dx_j
 * (X_{j-1} shaped).  dy[j] = D_j. */
pnn_status parareal_fine_bwd(pnn_plan* plan, const void* const* dy, const void* const* x,
                             const void* const* phi, const void* saved, void* const* dx,
                             float* const* dphi, void* scratch, void* stream);

/* coarse_bwd_all followed by parareal_fine_bwd (dy = D) in one call, with the same results: the
 * coarse chain runs on the given stream, and each group of fine sub-networks (as grouped by
 * pnn_set_streams) starts on its own stream as soon as the chain has produced the last D_j it
 * needs (the chain produces D_{N-2} first and D_0 last); the coarse weight gradients follow on a
 * side stream.  The transposed filters of the data gradients (parameters only) are formed first:
 * the coarse blocks' on the given stream ahead of the chain, the fine groups' on the side
 * streams.  Arguments as in those two calls. */
pnn_status parareal_bwd(pnn_plan* plan, void* const* D, const void* const* rt, const void* const* eta,
                        float* const* deta, const void* const* x, const void* const* phi,
                        void* const* dx, float* const* dphi, const void* saved, void* scratch,
                        void* stream);

/* dx[j] -= D_{j-1} in place for j = 1..N-1 (eq. (deltaj), the -D_{j-1} term; D_0 = 0). */
pnn_status parareal_combine_bwd(pnn_plan* plan, void* const* dx, const void* const* D,
                                void* stream);

/* ddelta[j] = dL/ddelta_j from g_j = dL/dx_j (after parareal_combine_bwd), eq. (deltaj).  No
 * gradient with respect to the image is formed.  ddelta[j] may be NULL for a C^j without
 * parameters. */
pnn_status pnn_pre_bwd(pnn_plan* plan, const void* image, const void* const* g,
                       const void* const* delta, const void* saved, float* const* ddelta,
                       void* scratch, void* stream);

/* ---- parameter update ---------------------------------------------------------------------- */

/* One step of stochastic gradient descent with momentum (Nesterov's form when nesterov != 0) and
 * weight decay, the optimiser of the paper's training runs (Sec. 4: SGD, momentum 0.9, weight decay
 * 5e-4 / 1e-4), for every parameter of one part of the network:
 *     d = g + weight_decay * w;   v = mu * v + d;   w = w - lr * (nesterov ? d + mu * v : v)
 * evaluated in fp32 per element; weight decay applies to every parameter.
 *   part 0 / 1 / 2: the segments C^j / g^j / F^j (N, N, N - 1 of them).  params[j]: the segment's
 *                   parameter buffer (filters in the storage type, written back rounded to
 *                   nearest even for PNN_BF16; BN gamma / beta in float); grads[j]: its gradient
 *                   buffer (float, pnn_param_layout(.., 1, ..)); momentum[j]: float buffer laid out
 *                   like the gradient buffer, updated in place (zero before the first step).
 *   part 3:         the head: params[0] = eps, grads[0] = deps, momentum[0]; K * C + K floats.
 * master (nullable; used by PNN_BF16 plans, parts 0 - 2): master[j] is a float buffer laid out
 * like the gradient buffer that holds an fp32 master copy of the segment's bf16 filters.  With it,
 * each filter update reads w from the master (master_init != 0: from the stored bf16 filter, for
 * the first step), writes the updated fp32 w back to the master and its nearest-even bf16 rounding
 * to params, so updates smaller than half a bf16 ulp (weight decay, late-training steps)
 * accumulate instead of being rounded away.  Without it the bf16 filter itself is the state.
 * BN parameters and the head are float and need no master.
 * Buffers may not alias one another.  PNN_ERR_INDEX for another part; PNN_ERR_NULL for a missing
 * buffer of a segment that has parameters. */
pnn_status pnn_sgd_step(pnn_plan* plan, int part, void* const* params, const float* const* grads,
                        float* const* momentum, float* const* master, int master_init, float lr,
                        float mu, float weight_decay, int nesterov, void* stream);

/* ---- misc ----------------------------------------------------------------------------------- */

/* Where the library keeps the internal tensors of one segment (part 0 = C^j, 1 = g^j, 2 = F^j;
 * j 0-based), for tests and inspection after a step:
 *   what = 0: value of slot idx (in the saved workspace, storage type, NHWC)
 *   what = 1: gradient dL/d(slot idx) (in scratch, storage type)
 *   what = 2: dL/d(BN output) of BN instance idx as stored before the BN backward (scratch)
 *   what = 3: statistics of BN instance idx: mean, invstd, scale, shift, float [4][C] (saved)
 *   what = 4: (part, j, idx ignored) the resident kernel's barrier words in scratch: uint32 [0] an
 *             error flag, non-zero when a barrier wait gave up, [1] barriers completed by the last
 *             resident launch (one per batch-normalisation point per unit and sub-network)
 *   what = 5: (part, j, idx ignored) the non-finite flags in scratch, uint32 [2]: [0] set to 1 by
 *             parareal_combine_fwd (given a scratch) when an element of some r_j is not finite,
 *             [1] by pnn_head_fwd_bwd when the loss or an element of deps is not finite; sticky
 *             until pnn_flags_clear
 * *offset receives the byte offset into that workspace.  PNN_ERR_INDEX when the tensor is not held
 * by the library (slot 0 and the segment output are the caller's tensors) or does not exist. */
pnn_status pnn_inspect(const pnn_plan* plan, int part, int j, int what, int idx, size_t* offset);

const char* pnn_status_string(pnn_status s);

/* Number of streams (1 .. 4, default 1) over which parareal_fine_fwd / parareal_fine_bwd /
 * parareal_bwd may run their sub-networks: the sub-networks are grouped by the spatial size of
 * their input (the ResNet stage they start in), the group with the most work is halved while
 * streams are left, and each group's level-by-level launches go to a stream of its own.  1 keeps
 * every launch on the call's stream.  Results do not depend on it (every group's launches are the
 * same; no reduction crosses groups).  Creates the plan's internal streams (default priority,
 * non-blocking) and fork / join events the first time more streams are asked for than exist (a
 * set-up call: needs a HIP device, allocates no device memory); PNN_ERR_HIP if that fails.
 * PNN_ERR_INDEX outside 1 .. 4. */
pnn_status pnn_set_streams(pnn_plan* plan, int streams);

/* Clears the non-finite flags (pnn_inspect what = 5) with a one-workgroup kernel on stream (no
 * memset node, so the call can be captured in a graph).  Scratch content is undefined after
 * allocation: clear before the first step whose flags are read.  PNN_ERR_NULL, PNN_ERR_ALIGN
 * (scratch not 256-byte aligned), PNN_ERR_HIP. */
pnn_status pnn_flags_clear(pnn_plan* plan, void* scratch, void* stream);

/* Resident forward of bottleneck-unit runs (PNN_BF16 plans; default off, 1 turns it on):
 * parareal_fine_fwd then runs each fine sub-network's run of identity pre-activation bottleneck units
 * at 32x32 with 64 channels (ResNet-1001's first stage, Table resnet) in one kernel per wave of
 * sub-networks, the residual stream kept on chip across the units and every BN point a barrier
 * over the sub-network's workgroups (one workgroup per image; sub-networks in waves of as many
 * images as the device holds at once).  Same results as the unit-by-unit kernels up to the
 * summation order of the BN statistics.  Off by default: on gfx950 its barriers and the
 * one-workgroup-per-CU schedule make it slower than the unit-by-unit kernels at these shapes. */
pnn_status pnn_set_resident(pnn_plan* plan, int on);

/* Per-kernel-family GPU time accounting with HIP events recorded on the call's stream around
 * every launch of one family (0 = off).  Families: 1 = grouped conv forward / data-gradient
 * kernel, 2 = weight-gradient kernels, 3 = streaming pointwise kernels (narrow 1x1 forward and
 * data gradients; BN sums of deferred-apply BNs).  pnn_timing_read synchronises on the recorded events and
 * returns the summed milliseconds, the launch count, and the summed multiply-add count
 * (2 x MACs = FLOPs) and minimum HBM bytes of those launches; it resets the accumulators. */
pnn_status pnn_timing_enable(pnn_plan* plan, int family);
pnn_status pnn_timing_read(pnn_plan* plan, double* ms, long long* launches, double* flops,
                           double* bytes);

#ifdef __cplusplus
}
#endif
#endif /* PNN_H */
