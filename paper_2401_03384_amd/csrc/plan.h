// Host planner: tnn-cost, optimal sequencer, tensor layouts, pairwise step
// lowering for the forward and backward passes, workspace layout.
#pragma once

#include <mutex>
#include <string>
#include <vector>

#include "desc.h"
#include "expr.h"

namespace ce {

enum BufKind : int { BUF_NONE = 0, BUF_IN, BUF_OUT, BUF_DOUT, BUF_DIN, BUF_WS };

struct BufRef {
    BufKind kind = BUF_NONE;
    int index = 0;        // operand index for BUF_IN / BUF_DIN
    size_t offset = 0;    // byte offset for BUF_WS
    int64_t shift = 0;    // further byte offset of a view into the buffer (any kind)
};

struct TensorRef {
    std::vector<int> labels;
    std::vector<int64_t> dims;
    std::vector<int64_t> strides;   // in elements
    DType dtype = DT_F32;
    BufRef buf;
    int64_t numel() const;
    int pos(int label) const;       // -1 if absent
    int64_t stride_of(int label) const { int p = pos(label); return p < 0 ? 0 : strides[p]; }
    int64_t dim_of(int label) const { int p = pos(label); return p < 0 ? 1 : dims[p]; }
    bool has(int label) const { return pos(label) >= 0; }
};

// One convolved label of a pairwise step (see GenericDesc): output index p in
// [0, O), reduction index j in [0, J), operand position a*p + b*j + g (taken
// modulo `mod` for a circular label), valid in [0, lim).
struct ConvMap {
    int label;
    int64_t O, J;
    int aL, bL;
    int64_t gL, limL;
    int aR, bR;
    int64_t gR, limR;
    int64_t modL = 0, modR = 0;   // circular label: position taken modulo N first
};

// C = sum over the reduced labels (and taps) of L * R.
struct PairOp {
    TensorRef L, R, C;
    bool has_r = true;
    std::vector<ConvMap> convs;
    uint32_t need = 0;     // backward: run only if a wanted gradient lies below
    uint64_t macs = 0;     // multiplications of the pairwise step it belongs to
    std::string what;
    bool generic_only = false;   // lower on the generic kernel (an op whose terms are all skipped)
};

struct Launch {
    int32_t kind = 0;
    BufRef a, b, c, d;                // operands (meaning depends on kind)
    std::vector<BufRef> extra;        // further operands of fused kernels
    uint32_t need = 0;
    uint32_t grid[3] = {1, 1, 1}, block[3] = {1, 1, 1};
    uint32_t lds = 0;
    std::vector<unsigned char> desc;  // descriptor bytes passed to the kernel
    std::string what;                 // step description
    std::string kname;                // kernel name
    double alg_bytes = 0, alg_flops = 0;
};

struct Node {
    uint32_t mask = 0;                // operands merged in this node
    int left = -1, right = -1;        // children (internal nodes)
    std::vector<int> labels;          // layout, outermost first
    std::vector<int64_t> dims;
};

struct Step {
    int a, b, c;                      // node ids: inputs (a holds the lowest operand), result
    uint64_t macs;                    // CE_COST_FWD multiplications
    uint64_t cost;                    // in the plan's cost mode
};

}  // namespace ce

struct ce_plan {
    ce_expr e;
    ce_cost_mode mode = CE_COST_FWD;
    ce_dtype dtype = CE_F32;
    unsigned flags = 0;
    std::vector<ce::Node> nodes;      // 0..n-1 leaves, then one per step
    std::vector<ce::Step> steps;      // execution order
    uint64_t total_cost = 0, fwd_macs = 0, ltr_cost = 0;
    std::vector<ce::Launch> fwd, bwd;
    size_t ws_fwd = 0, ws_bwd = 0;
    // intermediates the forward keeps for the backward (bit s: the result of
    // step s), their bytes, and the multiplications of the recompute steps
    // the backward still runs
    uint32_t save_mask = 0;
    uint64_t saved_bytes = 0, recompute_macs = 0;
    bool executable = true;
    std::string why_not;
    // description, built once on first request (plans are shared across threads)
    mutable std::once_flag text_once;
    mutable std::string text;
};

namespace ce {

// Limits of the search and the checkpointing choice of a plan.
struct PlanLimits {
    uint64_t max_elements = ~uint64_t(0);    // every intermediate's elements
    uint64_t max_step_cost = ~uint64_t(0);   // every step's cost in the plan's mode
    uint64_t save_budget = 0;                // bytes of intermediates kept for the backward
};

// Build a plan: the optimal order when use_path is false, else the order
// given by `pairs` (opt_einsum path format, n_pairs = n_in - 1).
ce_plan* make_plan(const ce_expr& e, ce_cost_mode mode, ce_dtype dtype, unsigned flags,
                   bool use_path, const int* pairs, int n_pairs,
                   const PlanLimits& lim = PlanLimits());

// Text description of a plan (steps, costs, workspace, launches).
std::string describe_plan(const ce_plan& p);

// Exposed for tests of the search: cost of merging operand sets A and B.
uint64_t pair_cost(const ce_expr& e, uint32_t A, uint32_t B, ce_cost_mode mode);

// Workspace scratch requested by a lowering (e.g. split-reduction partials);
// lives for the duration of the op's launches.
struct ScratchAlloc {
    virtual BufRef alloc(size_t bytes) = 0;
    virtual ~ScratchAlloc() = default;
};

// Both gradients of one step (gl: grad lhs, gr: grad rhs) as one fused
// launch and its partial sum, or nothing when they do not match.
std::vector<Launch> lower_grad_pair(const PairOp& gl, const PairOp& gr, unsigned flags, ScratchAlloc& scratch);

// The generic strided kernel for any pairwise op.
Launch lower_generic(const PairOp& op);

// Replace runs of launches that form a fused chain (e.g. the CP chain) by one
// fused launch.  Returns the number of fusions done.
int fuse_launches(std::vector<Launch>& v, bool backward);

// Backward of a plan whose whole forward is one fused CP chain launch `f`:
// one fused gradient launch plus ordered reductions of its partial factor
// gradients (scratch from `scratch`).  False when the chain's sizes are not
// covered by the fused backward kernel.
bool fuse_cp_backward(const Launch& f, int feature_operand, ScratchAlloc& scratch,
                      std::vector<Launch>& out);

// The whole forward of a reshaped-CP plan (three mode factors and a spatial
// factor applied one at a time) as one fused launch, when the layout and
// sizes match a compiled instantiation.
bool fuse_rcp_forward(const ce_plan& p, Launch& out);

// Backward of a plan whose forward is one fused reshaped-CP launch `f`: one
// fused gradient launch writing fp32 partials (dX per t1 and t2 chunk, the
// factor gradients per workgroup), then their ordered sums.
bool fuse_rcp_backward(const Launch& f, const ce_plan& p, ScratchAlloc& scratch, std::vector<Launch>& out);

// A contraction step `prod` and the convolution step `cons` that consumes its
// result as one fused launch (K_TT_FWD), when their labels and layouts fit
// the fused kernel; `out` reads the producer's operands and the consumer's
// other operand and writes the consumer's result.
bool fuse_tt_forward(const PairOp& prod, const PairOp& cons, Launch& out);

// Lowering of one pairwise op to launches: a specialised kernel when the
// op's label structure fits one (unless CE_FLAG_GENERIC_ONLY), else generic.
std::vector<Launch> lower_op(const ce_expr& e, const PairOp& op, unsigned flags,
                             ScratchAlloc& scratch);

}  // namespace ce
