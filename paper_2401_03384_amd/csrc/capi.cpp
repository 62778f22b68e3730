// Host-side C entry points (expression, plan, queries).  The execution entry
// points live with the executor.
#include <cstring>
#include <string>

#include "capi_internal.h"
#include "expr.h"
#include "plan.h"

namespace ce {
namespace {
thread_local std::string g_last_error;
}
void set_last_error(const std::string& msg) { g_last_error = msg; }
}  // namespace ce

using namespace ce;

namespace {
// Label id of `label` (its name as written, e.g. "h" or "(h1)", or the name
// inside the parentheses), -1 if unknown.
int find_label(const ce_expr& e, const char* label) {
    int id = -1;
    for (int l = 0; l < e.num_labels(); l++) {
        const std::string& nm = e.names[l];
        if (nm == label || (nm.size() > 2 && nm.front() == '(' && nm.back() == ')' &&
                            nm.compare(1, nm.size() - 2, label) == 0))
            id = l;
    }
    return id;
}
}  // namespace

extern "C" {

const char* ce_last_error(void) { return g_last_error.c_str(); }

const char* ce_version(void) { return "convein 0.1 (gfx950)"; }

ce_status ce_expr_parse(const char* spec, int n_in, const int* ranks, const int64_t* const* dims,
                        ce_expr** out) {
    return guard([&] {
        if (!out) fail(CE_ERR_ARG, "out is NULL");
        if (n_in < 1) fail(CE_ERR_ARG, "n_in must be >= 1");
        *out = parse_expr(spec, n_in, ranks, dims);
    });
}

ce_status ce_expr_set_feature(ce_expr* e, int operand) {
    return guard([&] {
        if (!e) fail(CE_ERR_ARG, "expr is NULL");
        if (operand < 0 || operand >= e->n) fail(CE_ERR_ARG, "operand out of range");
        e->feature_operand = operand;
    });
}

ce_status ce_expr_set_conv(ce_expr* e, const char* label, ce_pad pad) {
    return guard([&] {
        if (!e || !label) fail(CE_ERR_ARG, "NULL argument");
        int id = find_label(*e, label);
        if (id < 0) fail(CE_ERR_ARG, std::string("unknown label ") + label);
        if (!e->is_conv(id)) fail(CE_ERR_ARG, std::string("label ") + label + " is not convolved");
        const int holders = popcount64(e->holders[id]);
        if (pad == CE_PAD_SAME_ZERO) {
            if (holders > 2)
                fail(CE_ERR_UNSUPPORTED, std::string("label ") + label +
                                             " is held by more than two operands: only circular");
            e->circular[id] = 0;
        } else if (pad == CE_PAD_CIRCULAR) {
            if (holders < 2)
                fail(CE_ERR_ARG, std::string("label ") + label + " is held by one operand only");
            e->circular[id] = 1;
        } else {
            fail(CE_ERR_ARG, "unknown padding");
        }
    });
}

ce_status ce_expr_set_stride(ce_expr* e, const char* label, int stride) {
    return guard([&] {
        if (!e || !label) fail(CE_ERR_ARG, "NULL argument");
        int id = find_label(*e, label);
        if (id < 0) fail(CE_ERR_ARG, std::string("unknown label ") + label);
        if (!e->is_conv(id)) fail(CE_ERR_ARG, std::string("label ") + label + " is not convolved");
        if (stride < 1) fail(CE_ERR_ARG, "stride must be >= 1");
        if (popcount64(e->holders[id]) != 2)
            fail(CE_ERR_UNSUPPORTED, std::string("label ") + label +
                                         ": a stride needs a convolved label held by exactly two operands");
        e->stride[id] = stride;
    });
}

ce_status ce_expr_output_shape(const ce_expr* e, int* rank, int64_t* dims) {
    return guard([&] {
        if (!e || !rank) fail(CE_ERR_ARG, "NULL argument");
        auto d = e->out_dims();
        *rank = (int)d.size();
        if (dims)
            for (size_t k = 0; k < d.size(); k++) dims[k] = d[k];
    });
}

void ce_expr_destroy(ce_expr* e) { delete e; }

ce_status ce_plan_create(const ce_expr* e, ce_cost_mode mode, ce_dtype dtype, unsigned flags,
                         ce_plan** out) {
    return guard([&] {
        if (!e || !out) fail(CE_ERR_ARG, "NULL argument");
        *out = make_plan(*e, mode, dtype, flags, false, nullptr, 0);
    });
}

ce_status ce_plan_create_limited(const ce_expr* e, ce_cost_mode mode, ce_dtype dtype, unsigned flags,
                                 uint64_t max_elements, ce_plan** out) {
    return guard([&] {
        if (!e || !out) fail(CE_ERR_ARG, "NULL argument");
        PlanLimits lim;
        lim.max_elements = max_elements;
        *out = make_plan(*e, mode, dtype, flags, false, nullptr, 0, lim);
    });
}

ce_status ce_plan_create_ex(const ce_expr* e, const ce_plan_options* opt, ce_plan** out) {
    return guard([&] {
        if (!e || !opt || !out) fail(CE_ERR_ARG, "NULL argument");
        PlanLimits lim;
        if (opt->max_elements) lim.max_elements = opt->max_elements;
        if (opt->max_step_cost) lim.max_step_cost = opt->max_step_cost;
        lim.save_budget = opt->save_budget;
        *out = make_plan(*e, opt->mode, opt->dtype, opt->flags, false, nullptr, 0, lim);
    });
}

ce_status ce_plan_checkpoint(const ce_plan* p, uint64_t* saved_steps, uint64_t* saved_bytes,
                             uint64_t* recompute_macs) {
    return guard([&] {
        if (!p) fail(CE_ERR_ARG, "plan is NULL");
        if (saved_steps) *saved_steps = p->save_mask;
        if (saved_bytes) *saved_bytes = p->saved_bytes;
        if (recompute_macs) *recompute_macs = p->recompute_macs;
    });
}

ce_status ce_plan_create_with_path(const ce_expr* e, const int* pairs, int n_pairs, ce_dtype dtype,
                                   unsigned flags, ce_plan** out) {
    return guard([&] {
        if (!e || !out) fail(CE_ERR_ARG, "NULL argument");
        if (n_pairs > 0 && !pairs) fail(CE_ERR_ARG, "pairs is NULL");
        *out = make_plan(*e, CE_COST_FWD, dtype, flags, true, pairs, n_pairs);
    });
}

ce_status ce_plan_num_steps(const ce_plan* p, int* n) {
    return guard([&] {
        if (!p || !n) fail(CE_ERR_ARG, "NULL argument");
        *n = (int)p->steps.size();
    });
}

ce_status ce_plan_step(const ce_plan* p, int i, uint64_t* lhs_mask, uint64_t* rhs_mask,
                       uint64_t* macs) {
    return guard([&] {
        if (!p) fail(CE_ERR_ARG, "plan is NULL");
        if (i < 0 || i >= (int)p->steps.size()) fail(CE_ERR_ARG, "step index out of range");
        const Step& st = p->steps[i];
        if (lhs_mask) *lhs_mask = p->nodes[st.a].mask;
        if (rhs_mask) *rhs_mask = p->nodes[st.b].mask;
        if (macs) *macs = st.macs;
    });
}

ce_status ce_plan_cost(const ce_plan* p, uint64_t* total_cost, uint64_t* fwd_macs) {
    return guard([&] {
        if (!p) fail(CE_ERR_ARG, "plan is NULL");
        if (total_cost) *total_cost = p->total_cost;
        if (fwd_macs) *fwd_macs = p->fwd_macs;
    });
}

ce_status ce_plan_left_to_right_cost(const ce_plan* p, uint64_t* cost) {
    return guard([&] {
        if (!p || !cost) fail(CE_ERR_ARG, "NULL argument");
        if (p->ltr_cost == ~uint64_t(0)) fail(CE_ERR_OVERFLOW, "left-to-right cost exceeds 64 bits");
        *cost = p->ltr_cost;
    });
}

ce_status ce_plan_workspace_size(const ce_plan* p, int for_backward, size_t* bytes) {
    return guard([&] {
        if (!p || !bytes) fail(CE_ERR_ARG, "NULL argument");
        *bytes = for_backward ? p->ws_bwd : p->ws_fwd;
    });
}

const char* ce_plan_describe(const ce_plan* p) {
    if (!p) return "";
    std::call_once(p->text_once, [p] { p->text = ce::describe_plan(*p); });
    return p->text.c_str();
}

void ce_plan_destroy(ce_plan* p) { delete p; }

}  // extern "C"
