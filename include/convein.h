/*
 * convein.h - C ABI of the conv_einsum engine for AMD Instinct MI355X (gfx950).
 *
 * The engine evaluates one tensorial convolution layer written as a
 * conv_einsum string (arXiv 2401.03384, Section 2.2 'From einsum to
 * conv_einsum'; layer strings of Section 2.3 and Appendix A.3), e.g.
 *
 *     "bshw,rs,rt,rh,rw->bthw|hw"          CP layer
 *     "bshw,sp,pqhw,qt->bthw|hw"           Tucker-2 layer
 *
 * as a sequence of pairwise multilinear steps chosen to minimise the number
 * of multiplications under the paper's tnn-cost model (Section 3.2 and
 * Appendix B), and runs the forward pass and the backward pass (gradients of
 * every operand) with HIP kernels.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Grammar: operands separated by ',', then '->', the output, and
 *    optionally '|' followed by the convolved labels ("|hw" or "|h,w").  A
 *    label is one letter or a parenthesised name such as "(s1)".  Blanks are
 *    ignored.  A label occurs at most once per operand and once in the output;
 *    every convolved label must be kept in the output.
 *  - Sizes: a label that is not convolved has one size everywhere.  A
 *    convolved label held by two operands may have two sizes: the larger is
 *    the feature side, the smaller the filter side (Appendix B, 'Convolution
 *    Varieties'); equal sizes go to the designated feature operand when it is
 *    one of the two (operand 0 unless ce_expr_set_feature says otherwise),
 *    else to the lower operand index.
 *  - Convolution: cross-correlation, zero 'same' padding, stride 1 unless
 *    ce_expr_set_stride says otherwise:
 *        out[p] = sum_k feat[s*p + k - floor((K-1)/2)] * filt[k],
 *    p in [0, ceil(I / s)), with feat zero outside [0, I).  With stride 1 the
 *    output keeps the feature size I.
 *  - A label held by one operand only and absent from the output is summed
 *    away (Section 3.1, case (5)) before the pairwise steps.
 *  - A convolved label held by more than two operands (multi-way) is
 *    convolved circularly (see ce_expr_set_conv, CE_PAD_CIRCULAR).
 *  - Tensors are dense, row-major, in the label order written in the string
 *    (operands) or after '->' (output).  Element type is the plan's dtype,
 *    except gradients of operands other than the feature operand, which are
 *    always float32.  bfloat16 is stored as its raw 16-bit pattern.
 *  - Device memory (inputs, output, gradients, workspace) is owned by the
 *    caller.  The library never allocates device memory: all scratch lives in
 *    the caller's workspace, sized by ce_plan_workspace_size and aligned to
 *    256 bytes.
 *  - Host objects (ce_expr, ce_plan) are owned by the library, created by the
 *    *_parse / *_create calls and released by the *_destroy calls.  After
 *    creation they are immutable: one plan may be used from several threads
 *    and streams at once provided each call gets its own workspace.
 *  - Errors: every call returns a ce_status and, on failure, ce_last_error()
 *    returns a message (thread-local, valid until the next call on the same
 *    thread); out-parameters are left unset.  No C++ exception crosses this
 *    interface.  Every argument, size and workspace check of ce_forward /
 *    ce_backward happens before the first launch, so a call that fails with
 *    any status other than CE_ERR_HIP has enqueued nothing and left outputs,
 *    gradients and workspace untouched.  CE_ERR_HIP means the HIP runtime
 *    refused a launch (or an event record) part-way through the call's
 *    sequence: the launches before it stay enqueued on the stream and may
 *    already have written part of the output, of the gradients and of the
 *    workspace, none of the later ones is enqueued, and the contents of all
 *    of them are undefined until a later call succeeds.
 */
#ifndef CONVEIN_H
#define CONVEIN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    CE_OK = 0,
    CE_ERR_PARSE = -1,        /* malformed string */
    CE_ERR_SHAPE = -2,        /* ranks or sizes inconsistent with the string */
    CE_ERR_UNSUPPORTED = -3,  /* valid but not supported (too many operands or loop dimensions) */
    CE_ERR_ARG = -4,          /* null or out-of-range argument */
    CE_ERR_WORKSPACE = -5,    /* workspace too small or misaligned */
    CE_ERR_OVERFLOW = -6,     /* a cost or a size exceeds 64 bits */
    CE_ERR_HIP = -7           /* a HIP runtime call failed */
} ce_status;

typedef enum { CE_F32 = 0, CE_BF16 = 1 } ce_dtype;

/* Cost model of the sequencer.
 * CE_COST_FWD          multiplications of the forward pass (Appendix B cost
 *                      equations: contraction, batch, outer product, convolution).
 * CE_COST_TRAIN_PAPER  cost(f) + cost(g1) + cost(g2) per step (Appendix B,
 *                      'Modification of the cost model for training'). */
typedef enum { CE_COST_FWD = 0, CE_COST_TRAIN_PAPER = 1 } ce_cost_mode;

typedef struct ce_expr ce_expr;
typedef struct ce_plan ce_plan;

/* Opaque HIP stream handle (hipStream_t); NULL is the default stream. */
typedef void* ce_stream;

/* Maximum number of operands and of distinct labels. */
#define CE_MAX_OPERANDS 16
#define CE_MAX_LABELS 64

/* ---- expression ---------------------------------------------------------- */

/* Parse `spec` and bind operand sizes (Section 2.2; Appendix A sizes rule).
 *   n_in     number of operands; must equal the operands in `spec`
 *   ranks    [n_in] rank of each operand (must equal its label count)
 *   dims     [n_in] pointers to [ranks[i]] sizes, each >= 1
 *   out      receives a new ce_expr (release with ce_expr_destroy)
 * Errors: CE_ERR_PARSE, CE_ERR_SHAPE, CE_ERR_ARG, CE_ERR_UNSUPPORTED (more
 * than CE_MAX_OPERANDS operands or CE_MAX_LABELS labels). */
ce_status ce_expr_parse(const char* spec, int n_in, const int* ranks,
                        const int64_t* const* dims, ce_expr** out);

/* Designate the operand whose convolved labels are features when the two
 * sizes are equal (default 0).  Must be called before ce_plan_create. */
ce_status ce_expr_set_feature(ce_expr* e, int operand);

/* Boundary handling of a convolved label (Appendix A: "same" size output;
 * Appendix B: circular convolution, the only kind for a label held by more
 * than two operands). */
typedef enum { CE_PAD_SAME_ZERO = 0, CE_PAD_CIRCULAR = 1 } ce_pad;

/* Set the padding of convolved label `label` (its name in the string, e.g.
 * "h" or "(h1)").
 *   CE_PAD_SAME_ZERO (the default for a label held by two operands): output
 *     size = feature size, the filter centred with floor((K-1)/2) taps
 *     before, zero outside the feature (cross-correlation).
 *   CE_PAD_CIRCULAR (the default, and the only choice, for a label held by
 *     three or more operands): commutative circular convolution; every holder
 *     is zero-padded to N, the largest of its sizes, and positions add modulo
 *     N:  out[p] = sum over i_1 + ... + i_m = p (mod N) of prod_k T_k[i_k],
 *     p in [0, N).  A tensor merging two or more holders has N positions; a
 *     step merging sides of sizes a and b costs a * b for the label.  Steps
 *     with a circular label run on the generic kernel.
 * Must be called before ce_plan_create.
 * Errors: CE_ERR_ARG (NULL, unknown or not convolved label, unknown
 * padding, CE_PAD_CIRCULAR on a label held by one operand),
 * CE_ERR_UNSUPPORTED (CE_PAD_SAME_ZERO on a label held by more than two
 * operands). */
ce_status ce_expr_set_conv(ce_expr* e, const char* label, ce_pad pad);

/* Stride of convolved label `label` (Appendix B, 'Convolution Varieties': a
 * strided convolution is one of the non-commutative kinds, supported for a
 * label held by exactly two operands).  With stride s the output keeps
 * ceil(I / s) positions, output position p reading the feature at
 * s*p + k - floor((K-1)/2) (zero outside [0, I)): for odd K this is
 * PyTorch's conv with stride s and padding (K-1)/2.  A pairwise step that
 * convolves the label costs (output positions) x (filter size) for it.
 * Default 1.  Must be called before ce_plan_create; the fused chains are not
 * used for a plan with a strided label.
 * Errors: CE_ERR_ARG (NULL, unknown or not convolved label, stride < 1),
 * CE_ERR_UNSUPPORTED (the label is not held by exactly two operands). */
ce_status ce_expr_set_stride(ce_expr* e, const char* label, int stride);

/* Output rank and sizes (a convolved output label takes its feature size,
 * ceil(size / stride) when strided).
 *   rank   receives the output rank
 *   dims   if non-NULL, receives [rank] sizes */
ce_status ce_expr_output_shape(const ce_expr* e, int* rank, int64_t* dims);

void ce_expr_destroy(ce_expr* e);

/* ---- plan ----------------------------------------------------------------- */

/* Plan flags. */
#define CE_FLAG_GENERIC_ONLY 0x1u  /* run every step on the generic strided kernel */
#define CE_FLAG_NO_FUSION 0x2u     /* one launch per pairwise step (no fused chains) */
/* Keep every forward intermediate in the workspace for the backward instead of
 * recomputing it (Section 3.3 trades memory for recomputation): ce_backward
 * then skips the recompute launches and must receive the workspace the
 * preceding ce_forward of the same inputs used, unchanged, and of at least
 * ce_plan_workspace_size(p, 1) bytes (which covers the forward's).  A fused
 * chain whose backward is fused too (the CP and reshaped-CP chains) keeps its
 * intermediates on chip and recomputes them there, so for such a plan the
 * flag changes nothing; a fusion of the forward alone (the tensor-train
 * contraction + convolution) is not used with this flag, so the forward
 * writes the intermediate the backward then reads. */
#define CE_FLAG_SAVE_INTERMEDIATES 0x4u
/* Make every launch of the general contraction kernel use 64-bit element
 * offsets and predicated loads, the code path it takes for operands beyond
 * 2 GiB, even where 32-bit offsets would do (results are the same; this lets
 * small inputs exercise the wide-offset path). */
#define CE_FLAG_WIDE_OFFSETS 0x8u

/* Choose the pairwise evaluation order with the fewest multiplications under
 * `mode` (Section 3.2, optimal sequencer; Appendix B tnn-cost), searching
 * every binary tree including outer products.  Among trees of equal cost the
 * one whose first split (the part holding the lowest operand index) has the
 * smallest operand bitmask is taken, recursively.  Then lower each step to
 * kernels and lay out the workspace.  `e` may be destroyed afterwards.
 * Errors: CE_ERR_ARG, CE_ERR_OVERFLOW, CE_ERR_UNSUPPORTED. */
ce_status ce_plan_create(const ce_expr* e, ce_cost_mode mode, ce_dtype dtype,
                         unsigned flags, ce_plan** out);

/* Same, with a memory limit (Section 3.2, Figure 2: the paper's sequencer can
 * trade multiplications for intermediate size): the cheapest order among
 * those whose every intermediate tensor (every merged operand set except the
 * whole expression) holds at most max_elements elements, sizes counted as in
 * the planned layouts (a convolved label at its largest size in the set).
 * Ties are broken as in ce_plan_create.  Errors: as ce_plan_create, and
 * CE_ERR_UNSUPPORTED when no order fits the limit. */
ce_status ce_plan_create_limited(const ce_expr* e, ce_cost_mode mode, ce_dtype dtype,
                                 unsigned flags, uint64_t max_elements, ce_plan** out);

/* Options of ce_plan_create_ex.  A zero cap means no cap. */
typedef struct {
    ce_cost_mode mode;        /* cost model of the search and of max_step_cost */
    ce_dtype dtype;
    unsigned flags;           /* CE_FLAG_* */
    /* Per-node cost cap (Section 3.2, Figure 2, the path meeting a cost cap
     * c at each node): only orders in which every pairwise step costs at most
     * max_step_cost under `mode` compete. */
    uint64_t max_step_cost;
    /* Every intermediate holds at most max_elements elements (as
     * ce_plan_create_limited). */
    uint64_t max_elements;
    /* Checkpointing (Section 3.3): bytes of forward intermediates the
     * backward may read instead of recomputing.  0 recomputes every
     * intermediate (the default of the other entry points); otherwise the
     * planner keeps the set of intermediates the forward writes that avoids
     * the most recompute multiplications with at most save_budget bytes in
     * total (ties: fewer bytes, then the lower step indices).  As with
     * CE_FLAG_SAVE_INTERMEDIATES (which keeps every one, whatever the
     * budget), ce_backward must then receive the workspace of the preceding
     * ce_forward of the same inputs, unchanged; the kept intermediates sit at
     * its start, and ce_plan_workspace_size(p, 1) covers the forward's size. */
    uint64_t save_budget;
} ce_plan_options;

/* The optimal order under the options' caps, with the options'
 * checkpointing choice.  Errors: as ce_plan_create; CE_ERR_UNSUPPORTED when
 * no order meets the caps. */
ce_status ce_plan_create_ex(const ce_expr* e, const ce_plan_options* opt, ce_plan** out);

/* Checkpointing choice of a plan: bit s of saved_steps is set when the
 * result of step s is kept from the forward for the backward; saved_bytes
 * is their total size, recompute_macs the multiplications of the steps the
 * backward recomputes (on chip for a fused chain).  Any out-pointer may be
 * NULL. */
ce_status ce_plan_checkpoint(const ce_plan* p, uint64_t* saved_steps, uint64_t* saved_bytes,
                             uint64_t* recompute_macs);

/* Same, with a caller-given order (e.g. the left-to-right baseline of
 * Section 5): `pairs` holds n_pairs = n_in - 1 pairs (i, j) of positions in
 * the current operand list; the merged tensor is appended to the end of the
 * list (opt_einsum's path format).  Left-to-right is (0,1) followed by
 * (0, len-1) for the current list length len, e.g. (0,1),(0,3),(0,2),(0,1)
 * for five operands.  Costs are reported in CE_COST_FWD. */
ce_status ce_plan_create_with_path(const ce_expr* e, const int* pairs, int n_pairs,
                                   ce_dtype dtype, unsigned flags, ce_plan** out);

/* Number of pairwise steps (n_in - 1). */
ce_status ce_plan_num_steps(const ce_plan* p, int* n);

/* Step i in execution order (post order, first child first): operand bitmasks
 * of its two inputs (lhs holds the lowest operand index of the step) and its
 * multiplications under CE_COST_FWD.  Any out-pointer may be NULL. */
ce_status ce_plan_step(const ce_plan* p, int i, uint64_t* lhs_mask, uint64_t* rhs_mask,
                       uint64_t* macs);

/* Total cost of the plan in the plan's cost mode, and its forward
 * multiplications.  Either pointer may be NULL. */
ce_status ce_plan_cost(const ce_plan* p, uint64_t* total_cost, uint64_t* fwd_macs);

/* Multiplications of the left-to-right order under the plan's cost mode. */
ce_status ce_plan_left_to_right_cost(const ce_plan* p, uint64_t* cost);

/* Workspace bytes needed by ce_forward (for_backward = 0) or ce_backward
 * (for_backward = 1). */
ce_status ce_plan_workspace_size(const ce_plan* p, int for_backward, size_t* bytes);

/* Human-readable description of the steps and kernels (valid while p lives). */
const char* ce_plan_describe(const ce_plan* p);

void ce_plan_destroy(ce_plan* p);

/* ---- execution -------------------------------------------------------------- */

/* Forward pass (Section 3.1 atomic steps in the planned order).
 *   in        [n_in] device pointers to the operands
 *   out       device pointer to the output
 *   ws        device workspace of ws_bytes >= ce_plan_workspace_size(p, 0),
 *             256-byte aligned (may be NULL when the size is 0)
 *   stream    HIP stream; all work is enqueued asynchronously on it
 * Errors: CE_ERR_ARG, CE_ERR_WORKSPACE, CE_ERR_UNSUPPORTED (nothing
 * enqueued); CE_ERR_HIP (a launch failed part-way: the earlier launches stay
 * enqueued, `out` and `ws` are undefined, see the conventions above). */
ce_status ce_forward(const ce_plan* p, const void* const* in, void* out,
                     void* ws, size_t ws_bytes, ce_stream stream);

/* Backward pass: gradients of L = <Y, dout> with respect to the operands
 * (Appendix B: g1 and g2 of every step, in reverse order).  Intermediates are
 * recomputed from the inputs (gradient checkpointing, Section 3.3), so no
 * forward call needs to precede it, unless the plan was created with
 * CE_FLAG_SAVE_INTERMEDIATES (then the forward's workspace is read).
 *   in        [n_in] device pointers to the operands
 *   dout      device pointer to dL/dY (plan dtype, output layout)
 *   din       [n_in] device pointers receiving dL/d operand_i in the operand's
 *             layout (plan dtype for the feature operand, float32 for the
 *             others); a NULL entry means that gradient is not wanted
 *   ws        workspace of ws_bytes >= ce_plan_workspace_size(p, 1)
 * Errors: as ce_forward. */
ce_status ce_backward(const ce_plan* p, const void* const* in, const void* dout,
                      void* const* din, void* ws, size_t ws_bytes, ce_stream stream);

/* Workspace bytes that ce_backward_noalloc provides. */
#define CE_NOALLOC_WORKSPACE_BYTES (64u << 20)

/* ce_backward for callers that cannot allocate device memory: code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc.
 * The same launches as ce_backward, with the workspace taken from a fixed
 * device array of CE_NOALLOC_WORKSPACE_BYTES (64 MiB) that the library holds
 * on every GPU it runs on until the process ends; nothing is allocated.  The
 * array's device address is looked up on the first call on a device.
 *   in, dout, din   as ce_backward
 *   stream          must belong to the current device (NULL: the default
 *                   stream of the current device)
 * Every call on one GPU uses the same array, which keeps the contents the
 * last call left: calls that can overlap on one GPU (other streams, other
 * threads, without ordering between them) race on it; calls ordered on one
 * stream do not.  No part of the array has to start at any value: every
 * launch writes what a later launch of the same call reads.
 * Errors: as ce_backward; CE_ERR_WORKSPACE when ce_plan_workspace_size(p, 1)
 * exceeds CE_NOALLOC_WORKSPACE_BYTES; CE_ERR_UNSUPPORTED for a plan whose
 * backward reads intermediates kept in the forward's workspace
 * (CE_FLAG_SAVE_INTERMEDIATES or a save budget, see ce_plan_checkpoint);
 * CE_ERR_ARG when the stream belongs to another device. */
ce_status ce_backward_noalloc(const ce_plan* p, const void* const* in, const void* dout,
                              void* const* din, ce_stream stream);

/* ---- launch timing (profiling harnesses) ---------------------------------- */

/* Start recording on the calling thread: every kernel that ce_forward /
 * ce_backward enqueue from now on is bracketed by two HIP events recorded on
 * the same stream (events are created by the library and reused; no device
 * memory is allocated).  Adds two event records per launch. */
ce_status ce_timing_begin(void);

/* As ce_timing_begin, but only launches of the kernel labelled `kernel` (the
 * label ce_timing_record reports, e.g. "cp_bwd<float, 3, 3, 2, 2>") are
 * bracketed, so the other launches run without event records in between.
 * NULL or "" records every launch.  The label is copied. */
ce_status ce_timing_begin_kernel(const char* kernel);

/* Stop recording; waits for the recorded events and keeps the records until
 * the next ce_timing_begin on this thread.  n_records receives their count. */
ce_status ce_timing_end(int* n_records);

/* Record i (enqueue order): kernel name, step description (valid until the
 * next ce_timing_begin), elapsed milliseconds, and the launch's algorithmic
 * bytes (each operand read once, the result written once) and flops
 * (2 x multiplications of its pairwise step).  Any out-pointer may be NULL. */
ce_status ce_timing_record(int i, const char** kernel, const char** step, float* ms,
                           double* bytes, double* flops);

/* Message for the last non-OK status returned on this thread. */
const char* ce_last_error(void);

/* Library version string. */
const char* ce_version(void);

#ifdef __cplusplus
}
#endif

#endif /* CONVEIN_H */
