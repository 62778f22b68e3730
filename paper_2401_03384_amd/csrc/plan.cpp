// Host planner.
//
// Cost model (Appendix B): a pairwise step costs the product, over the union
// of the labels its two operands keep, of the label size; a label shared by
// both operands counts once, except a convolved label held by both, which
// counts (feature size) * (filter size).  Training mode adds the two gradient
// steps (Appendix B, 'Modification of the cost model for training').
//
// Sequencer (Section 3.2): exhaustive dynamic programme over operand subsets,
// every binary tree including outer products; ties go to the split whose part
// holding the lowest operand index has the smallest bitmask.
#include "plan.h"

#include <algorithm>
#include <cstring>
#include <memory>
#include <sstream>

namespace ce {

int64_t TensorRef::numel() const {
    int64_t n = 1;
    for (auto d : dims) n *= d;
    return n;
}

int TensorRef::pos(int label) const {
    for (size_t k = 0; k < labels.size(); k++)
        if (labels[k] == label) return (int)k;
    return -1;
}

namespace {

constexpr uint64_t kSat = ~uint64_t(0);

uint64_t mul_sat(uint64_t a, uint64_t b) {
    unsigned __int128 r = (unsigned __int128)a * b;
    return (r >> 64) ? kSat : (uint64_t)r;
}
uint64_t add_sat(uint64_t a, uint64_t b) {
    uint64_t r = a + b;
    return r < a ? kSat : r;
}

// Labels kept by the intermediate merging operand set S: held in S and either
// in the output or still held outside S.
uint64_t kept_mask(const ce_expr& e, uint32_t S) {
    uint64_t m = 0;
    for (int l = 0; l < e.num_labels(); l++) {
        uint32_t h = e.holders[l];
        if ((h & S) && (e.in_out(l) || (h & ~S))) m |= 1ull << l;
    }
    return m;
}

// Size of label l in the intermediate of S: the largest size among S's
// operands holding it (for a convolved label, the feature size once both
// sides are merged; for a strided one, its ceil(I / s) output positions).
int64_t size_in_set(const ce_expr& e, uint32_t S, int l) {
    if (e.stride_of(l) > 1 && (e.holders[l] & S) == e.holders[l]) return e.out_size(l);
    // a circular label with two or more holders merged: its N positions
    if (e.is_circular(l) && popcount64(e.holders[l] & S) >= 2) return e.out_size(l);
    int64_t m = 0;
    for (int i = 0; i < e.n; i++)
        if (((S >> i) & 1) && ((e.holders[l] >> i) & 1)) m = std::max(m, e.size_in(i, l));
    return m;
}

// Is side A the feature side of convolved label l in the step (A, B)?
bool feature_on_a(const ce_expr& e, uint32_t A, uint32_t B, int l) {
    int f = e.feature_of(l);
    if (f >= 0) return (A >> f) & 1;
    return size_in_set(e, A, l) >= size_in_set(e, B, l);   // multi-way label
}

uint64_t step_cost_sat(const ce_expr& e, uint32_t A, uint32_t B, ce_cost_mode mode) {
    uint64_t ka = kept_mask(e, A), kb = kept_mask(e, B);
    uint64_t plain = 1, conv_f = 1, conv_ga = 1, conv_gb = 1;
    for (int l = 0; l < e.num_labels(); l++) {
        bool ia = (ka >> l) & 1, ib = (kb >> l) & 1;
        if (!ia && !ib) continue;
        if (ia && ib && e.is_circular(l)) {
            // every pair of positions meets once (forward and each gradient)
            plain = mul_sat(plain, mul_sat((uint64_t)size_in_set(e, A, l), (uint64_t)size_in_set(e, B, l)));
        } else if (ia && ib && e.is_conv(l)) {
            uint64_t sa = size_in_set(e, A, l), sb = size_in_set(e, B, l);
            bool fa = feature_on_a(e, A, B, l);
            const uint64_t st = (uint64_t)e.stride_of(l);
            uint64_t feat = fa ? sa : sb, filt = fa ? sb : sa, out = (feat + st - 1) / st;
            // forward: output positions x taps (feature x filter for stride 1)
            conv_f = mul_sat(conv_f, mul_sat(out, filt));
            // gradient of the feature side: output * filter; of the filter side: feature * output
            conv_ga = mul_sat(conv_ga, fa ? mul_sat(out, filt) : mul_sat(feat, out));
            conv_gb = mul_sat(conv_gb, fa ? mul_sat(feat, out) : mul_sat(out, filt));
        } else {
            plain = mul_sat(plain, (uint64_t)size_in_set(e, ia ? A : B, l));
        }
    }
    uint64_t f = mul_sat(plain, conv_f);
    if (mode == CE_COST_FWD) return f;
    return add_sat(f, add_sat(mul_sat(plain, conv_ga), mul_sat(plain, conv_gb)));
}

// Elements of the tensor merging the operands in S (kept labels; a
// convolved label at its largest size in S), saturating.
uint64_t set_numel(const ce_expr& e, uint32_t S) {
    const uint64_t k = kept_mask(e, S);
    uint64_t n = 1;
    for (int l = 0; l < e.num_labels(); l++)
        if ((k >> l) & 1) n = mul_sat(n, (uint64_t)size_in_set(e, S, l));
    return n;
}

std::string mask_str(uint32_t m) {
    std::string s = "{";
    bool first = true;
    for (int i = 0; i < 32; i++)
        if ((m >> i) & 1) {
            if (!first) s += ",";
            s += std::to_string(i);
            first = false;
        }
    return s + "}";
}

// Layout of an intermediate: output labels that are not convolved (output
// order), then labels still to be reduced (order of first appearance), then
// convolved labels (output order), so spatial labels are innermost.
std::vector<int> node_layout(const ce_expr& e, uint64_t kept, bool is_root) {
    std::vector<int> r;
    if (is_root) return e.out;
    for (int l : e.out)
        if (((kept >> l) & 1) && !e.is_conv(l)) r.push_back(l);
    for (int l = 0; l < e.num_labels(); l++)
        if (((kept >> l) & 1) && !e.in_out(l)) r.push_back(l);
    for (int l : e.out)
        if (((kept >> l) & 1) && e.is_conv(l)) r.push_back(l);
    return r;
}

struct Builder {
    const ce_expr& e;
    ce_plan& p;
    int n;
    Builder(const ce_expr& e_, ce_plan& p_) : e(e_), p(p_), n(e_.n) {}

    // ---- search ---------------------------------------------------------
    // Cheapest split of every operand set (subset DP).  With a limit, a set
    // other than the whole expression whose merged tensor exceeds `limit`
    // elements is infeasible, and so is every split that uses one; a split
    // whose own step costs more than `step_cap` is not taken (the per-node
    // cost cap of Section 3.2, Figure 2).  Returns false when the whole
    // expression has no feasible split.
    bool optimal_splits(uint64_t* best_cost, std::vector<uint32_t>& split,
                        uint64_t limit = ~uint64_t(0), uint64_t step_cap = ~uint64_t(0)) {
        uint32_t full = (n >= 32) ? 0xffffffffu : ((1u << n) - 1);
        std::vector<uint64_t> best(size_t(full) + 1, 0);
        std::vector<char> feasible(size_t(full) + 1, 1);
        split.assign(size_t(full) + 1, 0);
        for (uint32_t S = 1; S <= full; S++) {
            if (popcount64(S) == 1) continue;
            if (S != full && limit != ~uint64_t(0) && set_numel(e, S) > limit) {
                feasible[S] = 0;
                continue;
            }
            uint32_t low = S & (~S + 1), rest = S ^ low;
            uint64_t bc = kSat;
            uint32_t bA = 0;
            bool found = false;
            for (uint32_t sub = rest;; sub = (sub - 1) & rest) {
                uint32_t A = sub | low, B = S ^ A;
                if (B && feasible[A] && feasible[B]) {
                    const uint64_t sc = step_cost_sat(e, A, B, p.mode);
                    if (sc > step_cap) {
                        if (!sub) break;
                        continue;
                    }
                    uint64_t c = add_sat(add_sat(best[A], best[B]), sc);
                    if (!found || c < bc || (c == bc && A < bA)) {
                        bc = c;
                        bA = A;
                        found = true;
                    }
                }
                if (!sub) break;
            }
            best[S] = bc;
            split[S] = bA;
            feasible[S] = found;
        }
        *best_cost = best[full];
        return feasible[full] != 0;
    }

    int build_tree(uint32_t S, const std::vector<uint32_t>& split) {
        if (popcount64(S) == 1) return lowest_bit(S);
        uint32_t A = split[S], B = S ^ A;
        int a = build_tree(A, split);
        int b = build_tree(B, split);
        return add_node(a, b);
    }

    int add_node(int a, int b) {
        Node nd;
        nd.mask = p.nodes[a].mask | p.nodes[b].mask;
        nd.left = a;
        nd.right = b;
        p.nodes.push_back(nd);
        int c = (int)p.nodes.size() - 1;
        Step st;
        st.a = a;
        st.b = b;
        st.c = c;
        st.macs = step_cost_sat(e, p.nodes[a].mask, p.nodes[b].mask, CE_COST_FWD);
        st.cost = step_cost_sat(e, p.nodes[a].mask, p.nodes[b].mask, p.mode);
        p.steps.push_back(st);
        return c;
    }

    void make_leaves() {
        for (int i = 0; i < n; i++) {
            Node nd;
            nd.mask = 1u << i;
            nd.labels = e.ops[i];
            nd.dims = e.dims[i];
            p.nodes.push_back(nd);
        }
    }

    void tree_from_pairs(const int* pairs, int n_pairs) {
        if (n_pairs != n - 1) fail(CE_ERR_ARG, "a path needs n_in - 1 pairs");
        std::vector<int> cur;
        for (int i = 0; i < n; i++) cur.push_back(i);
        for (int k = 0; k < n_pairs; k++) {
            int i = pairs[2 * k], j = pairs[2 * k + 1];
            if (i == j || i < 0 || j < 0 || i >= (int)cur.size() || j >= (int)cur.size())
                fail(CE_ERR_ARG, "bad pair in path");
            int a = cur[i], b = cur[j];
            cur.erase(cur.begin() + std::max(i, j));
            cur.erase(cur.begin() + std::min(i, j));
            if (lowest_bit(p.nodes[b].mask) < lowest_bit(p.nodes[a].mask)) std::swap(a, b);
            cur.push_back(add_node(a, b));
        }
    }

    uint64_t left_to_right_cost() {
        uint64_t c = 0;
        uint32_t acc = 1;
        for (int i = 1; i < n; i++) {
            c = add_sat(c, step_cost_sat(e, acc, 1u << i, p.mode));
            acc |= 1u << i;
        }
        return c;
    }

    // ---- layouts ------------------------------------------------------------
    void assign_layouts() {
        for (size_t s = 0; s < p.steps.size(); s++) {
            Node& nd = p.nodes[p.steps[s].c];
            bool root = (s + 1 == p.steps.size());
            uint64_t kept = kept_mask(e, nd.mask);
            nd.labels = node_layout(e, kept, root);
            nd.dims.clear();
            for (int l : nd.labels) {
                int64_t d = root ? e.out_size(l) : size_in_set(e, nd.mask, l);
                nd.dims.push_back(d);
            }
        }
    }

    TensorRef tensor_of(int node, DType dt, BufRef buf) const {
        const Node& nd = p.nodes[node];
        TensorRef t;
        t.labels = nd.labels;
        t.dims = nd.dims;
        t.strides.assign(nd.dims.size(), 1);
        for (int k = (int)nd.dims.size() - 2; k >= 0; k--) t.strides[k] = t.strides[k + 1] * nd.dims[k + 1];
        t.dtype = dt;
        t.buf = buf;
        return t;
    }

    // Conv maps of a step.  mode 0: forward C = f(A, B); 1: dA = g(dC, B); 2: dB = g(A, dC).
    std::vector<ConvMap> conv_maps(const Step& st, int which) const {
        std::vector<ConvMap> v;
        uint32_t A = p.nodes[st.a].mask, B = p.nodes[st.b].mask;
        uint64_t ka = kept_mask(e, A), kb = kept_mask(e, B);
        for (int l = 0; l < e.num_labels(); l++) {
            if (!e.is_conv(l) || !((ka >> l) & 1) || !((kb >> l) & 1)) continue;
            if (e.is_circular(l)) {
                // C[p] = sum_j A[(p - j) mod N] B[j]; dA[i] = sum_j dC[(i + j) mod N] B[j];
                // dB[j] = sum_i A[i] dC[(i + j) mod N]
                const int64_t sa = size_in_set(e, A, l), sb = size_in_set(e, B, l);
                const int64_t N = e.out_size(l);
                ConvMap m{};
                m.label = l;
                if (which == 0) {
                    m.O = N; m.J = sb;
                    m.aL = 1; m.bL = -1; m.gL = 0; m.limL = sa; m.modL = N;
                    m.aR = 0; m.bR = 1; m.gR = 0; m.limR = sb;
                } else if (which == 1) {
                    m.O = sa; m.J = sb;
                    m.aL = 1; m.bL = 1; m.gL = 0; m.limL = N; m.modL = N;
                    m.aR = 0; m.bR = 1; m.gR = 0; m.limR = sb;
                } else {
                    m.O = sb; m.J = sa;
                    m.aL = 0; m.bL = 1; m.gL = 0; m.limL = sa;
                    m.aR = 1; m.bR = 1; m.gR = 0; m.limR = N; m.modR = N;
                }
                v.push_back(m);
                continue;
            }
            bool fa = feature_on_a(e, A, B, l);
            int64_t I = size_in_set(e, fa ? A : B, l);
            int64_t K = size_in_set(e, fa ? B : A, l);
            int64_t c = (K - 1) / 2;
            const int s = e.stride_of(l);
            const int64_t Oq = (I + s - 1) / s;   // output positions
            ConvMap m{};
            m.label = l;
            if (which == 0) {
                // C[p] = sum_j feat[s*p + j - c] * filt[j]
                m.O = Oq;
                m.J = K;
                if (fa) { m.aL = s; m.bL = 1; m.gL = -c; m.limL = I; m.aR = 0; m.bR = 1; m.gR = 0; m.limR = K; }
                else    { m.aL = 0; m.bL = 1; m.gL = 0; m.limL = K; m.aR = s; m.bR = 1; m.gR = -c; m.limR = I; }
            } else if (which == 1) {
                // L = dC, R = B, output dA
                if (fa) {  // dA[q] = sum_j dC[q - j + c] B[j]  (stride 1; see phase_split)
                    m.O = I; m.J = K;
                    m.aL = 1; m.bL = -1; m.gL = c; m.limL = Oq;
                    m.aR = 0; m.bR = 1; m.gR = 0; m.limR = K;
                } else {   // dA[k] = sum_p dC[p] B[s*p + k - c]
                    m.O = K; m.J = Oq;
                    m.aL = 0; m.bL = 1; m.gL = 0; m.limL = Oq;
                    m.aR = 1; m.bR = s; m.gR = -c; m.limR = I;
                }
            } else {
                // L = A, R = dC, output dB
                if (fa) {  // dB[k] = sum_p A[s*p + k - c] dC[p]
                    m.O = K; m.J = Oq;
                    m.aL = 1; m.bL = s; m.gL = -c; m.limL = I;
                    m.aR = 0; m.bR = 1; m.gR = 0; m.limR = Oq;
                } else {   // dB[q] = sum_j A[j] dC[q - j + c]  (stride 1; see phase_split)
                    m.O = I; m.J = K;
                    m.aL = 0; m.bL = 1; m.gL = 0; m.limL = K;
                    m.aR = 1; m.bR = -1; m.gR = c; m.limR = Oq;
                }
            }
            v.push_back(m);
        }
        return v;
    }

    // The gradient of the feature side of a strided convolution (a
    // transposed convolution) as stride-1-shaped ops: for output positions
    // q = s*q' + r of residue r, only taps j = j0 + s*j' with
    // j0 = (r + c) mod s reach them, reading dC at q' - j' + (r + c - j0)/s.
    // Each phase is the op on views of the output (positions r, r + s, ...)
    // and of the filter (taps j0, j0 + s, ...), every phase of every strided
    // label once; labels of stride 1 keep their single map.  `op` is the
    // gradient op of step `st` (which = 1: dA, 2: dB) with maps from
    // conv_maps; returns the phase ops (just `op` when nothing is strided).
    std::vector<PairOp> phase_split(const Step& st, int which, const PairOp& op) const {
        uint32_t A = p.nodes[st.a].mask, B = p.nodes[st.b].mask;
        std::vector<int> idx;   // maps to split: strided, gradient of the feature side
        for (size_t k = 0; k < op.convs.size(); k++) {
            const int l = op.convs[k].label;
            const bool fa = feature_on_a(e, A, B, l);
            if (e.stride_of(l) > 1 && ((which == 1) == fa)) idx.push_back((int)k);
        }
        if (idx.empty()) return {op};
        // the filter operand of the op: R for dA (which 1), L for dB (which 2)
        const bool filt_is_r = which == 1;
        const size_t esC = op.C.dtype == DT_BF16 ? 2 : 4;
        const TensorRef& F0 = filt_is_r ? op.R : op.L;
        const size_t esF = F0.dtype == DT_BF16 ? 2 : 4;
        int64_t nph = 1;
        for (int k : idx) nph *= e.stride_of(op.convs[k].label);
        std::vector<PairOp> out;
        for (int64_t ph = 0; ph < nph; ph++) {
            PairOp q = op;
            TensorRef& F = filt_is_r ? q.R : q.L;
            bool empty = false, none = false;
            int64_t x = ph;
            for (int k : idx) {
                ConvMap& m = q.convs[k];
                const int l = m.label;
                const int64_t s = e.stride_of(l);
                const int64_t r = x % s;
                x /= s;
                const int64_t I = m.O, K = m.J, c = (K - 1) / 2;
                const int64_t j0 = (r + c) % s;
                const int64_t Q = I > r ? (I - r + s - 1) / s : 0;
                const int64_t J = K > j0 ? (K - j0 + s - 1) / s : 0;
                if (Q == 0) none = true;
                const int pc = q.C.pos(l), pf = F.pos(l);
                q.C.buf.shift += (int64_t)(r * q.C.strides[pc] * (int64_t)esC);
                q.C.dims[pc] = Q;
                q.C.strides[pc] *= s;
                m.O = Q;
                if (J == 0) {
                    // no tap reaches these positions: every term is skipped
                    empty = true;
                    F.dims[pf] = 1;
                    m.J = 1;
                } else {
                    F.buf.shift += (int64_t)(j0 * F.strides[pf] * (int64_t)esF);
                    F.dims[pf] = J;
                    F.strides[pf] *= s;
                    m.J = J;
                }
                const int64_t g = (r + c - j0) / s;
                if (filt_is_r) {
                    m.gL = g;
                    m.limR = empty ? 0 : m.J;
                } else {
                    m.gR = g;
                    m.limL = empty ? 0 : m.J;
                }
            }
            if (none) continue;
            q.macs = op.macs / nph;
            q.what = op.what + " phase " + std::to_string(ph);
            q.generic_only = empty;
            out.push_back(q);
        }
        return out;
    }

};

// ---- workspace layout: greedy interval packing ---------------------------
struct WsItem {
    size_t bytes;
    int t0, t1;
    size_t offset = 0;
    int id;
};

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

size_t pack(std::vector<WsItem>& items) {
    std::vector<int> order(items.size());
    for (size_t i = 0; i < items.size(); i++) order[i] = (int)i;
    std::sort(order.begin(), order.end(), [&](int a, int b) {
        if (items[a].bytes != items[b].bytes) return items[a].bytes > items[b].bytes;
        return items[a].t0 < items[b].t0;
    });
    std::vector<int> placed;
    size_t total = 0;
    for (int id : order) {
        WsItem& it = items[id];
        std::vector<std::pair<size_t, size_t>> busy;
        for (int q : placed) {
            const WsItem& o = items[q];
            if (o.t1 < it.t0 || it.t1 < o.t0) continue;
            busy.push_back({o.offset, o.offset + align256(o.bytes)});
        }
        std::sort(busy.begin(), busy.end());
        size_t off = 0;
        for (auto& b : busy) {
            if (off + align256(it.bytes) <= b.first) break;
            off = std::max(off, b.second);
        }
        it.offset = off;
        total = std::max(total, off + align256(it.bytes));
        placed.push_back(id);
    }
    return total;
}

// Workspace items no launch refers to (intermediates a fused launch keeps
// on chip) take no space.
void drop_unused(std::vector<WsItem>& items, const std::vector<Launch>& v) {
    std::vector<int> used;
    for (const Launch& ln : v) {
        for (const BufRef* b : {&ln.a, &ln.b, &ln.c, &ln.d})
            if (b->kind == BUF_WS) used.push_back(b->index);
        for (const BufRef& b : ln.extra)
            if (b.kind == BUF_WS) used.push_back(b.index);
    }
    std::vector<WsItem> kept;
    for (const WsItem& it : items)
        if (std::find(used.begin(), used.end(), it.id) != used.end()) kept.push_back(it);
    items.swap(kept);
}

}  // namespace

// ---- generic lowering ----------------------------------------------------
Launch lower_generic(const PairOp& op) {
    GenericDesc d;
    std::memset(&d, 0, sizeof(d));
    struct Dim { int64_t size, sL, sR, sC; bool conv; };
    std::vector<Dim> od, rd;
    auto conv_of = [&](int l) -> int {
        for (size_t k = 0; k < op.convs.size(); k++)
            if (op.convs[k].label == l) return (int)k;
        return -1;
    };
    std::vector<int> cv_out(op.convs.size(), -1), cv_red(op.convs.size(), -1);
    for (size_t k = 0; k < op.C.labels.size(); k++) {
        int l = op.C.labels[k];
        int ci = conv_of(l);
        if (ci >= 0) {
            cv_out[ci] = (int)od.size();
            od.push_back({op.convs[ci].O, 0, 0, op.C.strides[k], true});
        } else {
            od.push_back({op.C.dims[k], op.L.stride_of(l), op.has_r ? op.R.stride_of(l) : 0,
                          op.C.strides[k], false});
        }
    }
    for (size_t k = 0; k < op.convs.size(); k++) {
        cv_red[k] = (int)rd.size();
        rd.push_back({op.convs[k].J, 0, 0, 0, true});
    }
    for (size_t k = 0; k < op.L.labels.size(); k++) {
        int l = op.L.labels[k];
        if (op.C.has(l) || conv_of(l) >= 0) continue;
        rd.push_back({op.L.dims[k], op.L.strides[k], op.has_r ? op.R.stride_of(l) : 0, 0, false});
    }
    if (op.has_r)
        for (size_t k = 0; k < op.R.labels.size(); k++) {
            int l = op.R.labels[k];
            if (op.C.has(l) || op.L.has(l) || conv_of(l) >= 0) continue;
            rd.push_back({op.R.dims[k], 0, op.R.strides[k], 0, false});
        }
    // merge neighbouring plain dims whose strides chain in every operand
    auto merge = [](std::vector<Dim>& v, std::vector<int>& idx_fix) {
        for (size_t i = 0; i + 1 < v.size();) {
            Dim& a = v[i];
            Dim& b = v[i + 1];
            bool ok = !a.conv && !b.conv && a.sL == b.sL * b.size && a.sR == b.sR * b.size &&
                      a.sC == b.sC * b.size;
            if (ok) {
                a.size *= b.size;
                a.sL = b.sL;
                a.sR = b.sR;
                a.sC = b.sC;
                v.erase(v.begin() + i + 1);
                for (auto& x : idx_fix)
                    if (x > (int)i) x--;
            } else {
                i++;
            }
        }
    };
    merge(od, cv_out);
    merge(rd, cv_red);
    if ((int)od.size() > kMaxDims || (int)rd.size() > kMaxDims || (int)op.convs.size() > kMaxConv)
        fail(CE_ERR_UNSUPPORTED, "step has too many loop dimensions for the generic kernel");
    d.nout = (int)od.size();
    d.nred = (int)rd.size();
    d.nconv = (int)op.convs.size();
    d.has_r = op.has_r ? 1 : 0;
    d.total_out = 1;
    d.total_red = 1;
    for (int i = 0; i < d.nout; i++) {
        d.out_size[i] = od[i].size;
        d.out_sL[i] = od[i].sL;
        d.out_sR[i] = od[i].sR;
        d.out_sC[i] = od[i].sC;
        d.total_out *= od[i].size;
    }
    for (int i = 0; i < d.nred; i++) {
        d.red_size[i] = rd[i].size;
        d.red_sL[i] = rd[i].sL;
        d.red_sR[i] = rd[i].sR;
        d.total_red *= rd[i].size;
    }
    for (int k = 0; k < d.nconv; k++) {
        const ConvMap& m = op.convs[k];
        d.cv_out[k] = cv_out[k];
        d.cv_red[k] = cv_red[k];
        d.cv_aL[k] = m.aL;
        d.cv_bL[k] = m.bL;
        d.cv_gL[k] = m.gL;
        d.cv_limL[k] = m.limL;
        d.cv_sL[k] = op.L.stride_of(m.label);
        d.cv_aR[k] = m.aR;
        d.cv_bR[k] = m.bR;
        d.cv_gR[k] = m.gR;
        d.cv_limR[k] = m.limR;
        d.cv_sR[k] = op.has_r ? op.R.stride_of(m.label) : 0;
        d.cv_modL[k] = m.modL;
        d.cv_modR[k] = m.modR;
    }
    Launch ln;
    ln.a = op.L.buf;
    ln.b = op.R.buf;
    ln.c = op.C.buf;
    ln.need = op.need;
    ln.what = op.what;
    int32_t tL = op.L.dtype, tR = op.has_r ? op.R.dtype : DT_F32, tC = op.C.dtype;
    // kind encodes the variant and the three element types
    int variant;
    if (d.total_red <= 256) {
        variant = K_GENERIC_THREAD;
        ln.block[0] = 256;
        ln.grid[0] = (uint32_t)((d.total_out + 255) / 256);
    } else if (d.total_red <= 65536) {
        variant = K_GENERIC_WAVE;
        ln.block[0] = 256;
        ln.grid[0] = (uint32_t)((d.total_out + 3) / 4);
    } else {
        variant = K_GENERIC_BLOCK;
        ln.block[0] = 256;
        ln.grid[0] = (uint32_t)d.total_out;
    }
    if (d.total_out > (int64_t)0x7fffffff * 4) fail(CE_ERR_UNSUPPORTED, "step too large");
    ln.kind = variant | (tL << 8) | (tR << 9) | (tC << 10);
    ln.desc.resize(sizeof(d));
    std::memcpy(ln.desc.data(), &d, sizeof(d));
    return ln;
}

namespace {

std::string tensor_str(const ce_expr& e, const TensorRef& t) {
    std::string s;
    for (size_t k = 0; k < t.labels.size(); k++) {
        const std::string& nm = e.names[t.labels[k]];
        s += nm.size() == 1 ? nm : "(" + nm + ")";
    }
    return s;
}

}  // namespace

uint64_t pair_cost(const ce_expr& e, uint32_t A, uint32_t B, ce_cost_mode mode) {
    uint64_t c = step_cost_sat(e, A, B, mode);
    if (c == kSat) fail(CE_ERR_OVERFLOW, "step cost exceeds 64 bits");
    return c;
}

ce_plan* make_plan(const ce_expr& e, ce_cost_mode mode, ce_dtype dtype, unsigned flags,
                   bool use_path, const int* pairs, int n_pairs, const PlanLimits& lim) {
    if (!e.bound) fail(CE_ERR_ARG, "expression is not bound");
    for (int l = 0; l < e.num_labels(); l++)
        if (e.stride_of(l) > 1 && e.feature_of(l) < 0)
            fail(CE_ERR_UNSUPPORTED, "label " + e.names[l] +
                                         ": a stride needs a convolved label held by exactly two operands");
    if (mode != CE_COST_FWD && mode != CE_COST_TRAIN_PAPER) fail(CE_ERR_ARG, "bad cost mode");
    if (dtype != CE_F32 && dtype != CE_BF16) fail(CE_ERR_ARG, "bad dtype");
    std::unique_ptr<ce_plan> p(new ce_plan());
    p->e = e;
    p->mode = mode;
    p->dtype = dtype;
    p->flags = flags;
    Builder bld(p->e, *p);
    const ce_expr& E = p->e;
    int n = E.n;
    bld.make_leaves();
    if (use_path && n_pairs != n - 1) fail(CE_ERR_ARG, "a path needs n_in - 1 pairs");
    if (n >= 2) {
        if (use_path) {
            bld.tree_from_pairs(pairs, n_pairs);
        } else {
            uint64_t best;
            std::vector<uint32_t> split;
            if (!bld.optimal_splits(&best, split, lim.max_elements, lim.max_step_cost))
                fail(CE_ERR_UNSUPPORTED, "no pairwise order keeps every intermediate within " +
                                             std::to_string(lim.max_elements) +
                                             " elements and every step within cost " +
                                             std::to_string(lim.max_step_cost));
            bld.build_tree((n >= 32) ? 0xffffffffu : ((1u << n) - 1), split);
        }
    }
    p->total_cost = 0;
    p->fwd_macs = 0;
    for (auto& st : p->steps) {
        if (st.macs == kSat || st.cost == kSat) fail(CE_ERR_OVERFLOW, "plan cost exceeds 64 bits");
        p->total_cost = add_checked(p->total_cost, st.cost);
        p->fwd_macs = add_checked(p->fwd_macs, st.macs);
    }
    p->ltr_cost = bld.left_to_right_cost();
    bld.assign_layouts();

    for (int l = 0; l < E.num_labels(); l++)
        if (E.is_circular(l) && E.stride_of(l) > 1)
            fail(CE_ERR_UNSUPPORTED, "label " + E.names[l] + ": a circular convolution has no stride");
    DType dt = dtype == CE_BF16 ? DT_BF16 : DT_F32;
    int m = (int)p->steps.size();
    // the fused chains are written for stride-1, zero-padded convolutions
    bool special = false;
    for (int l = 0; l < E.num_labels(); l++)
        if (E.stride_of(l) > 1 || E.is_circular(l)) special = true;
    if (special) flags |= CE_FLAG_NO_FUSION;

    if (p->executable) {
        // Workspace items: intermediates (id = node), their gradients
        // (id = GRAD_ID + node) and per-launch scratch (ids from SCRATCH_ID).
        // Launch buffers refer to items by id; offsets are patched after packing.
        const int GRAD_ID = 1 << 20, SCRATCH_ID = 1 << 24;
        auto elem = [&](DType t) { return t == DT_BF16 ? 2 : 4; };
        auto consumer_step = [&](int node) -> int {
            for (int s = 0; s < m; s++)
                if (p->steps[s].a == node || p->steps[s].b == node) return s;
            return m;
        };
        auto patch = [&](std::vector<Launch>& v, const std::vector<WsItem>& items) {
            for (auto& ln : v) {
                std::vector<BufRef*> refs = {&ln.a, &ln.b, &ln.c, &ln.d};
                for (auto& x : ln.extra) refs.push_back(&x);
                for (BufRef* b : refs)
                    if (b->kind == BUF_WS) {
                        bool found = false;
                        for (auto& it : items)
                            if (it.id == b->index) { b->offset = it.offset; found = true; break; }
                        if (!found) fail(CE_ERR_ARG, "internal: workspace item missing");
                    }
            }
        };
        struct ItemScratch : ScratchAlloc {
            std::vector<WsItem>* items = nullptr;
            int t = 0, next = 0;
            BufRef alloc(size_t bytes) override {
                WsItem it;
                it.bytes = bytes;
                it.t0 = it.t1 = t;
                it.id = next++;
                items->push_back(it);
                BufRef b;
                b.kind = BUF_WS;
                b.index = it.id;
                return b;
            }
        };
        auto dense_out = [&](BufKind k) {
            TensorRef out;
            out.labels = E.out;
            out.dims = E.out_dims();
            out.strides.assign(out.dims.size(), 1);
            for (int k2 = (int)out.dims.size() - 2; k2 >= 0; k2--)
                out.strides[k2] = out.strides[k2 + 1] * out.dims[k2 + 1];
            out.dtype = dt;
            out.buf.kind = k;
            return out;
        };

        // ---------------- forward ----------------
        std::vector<WsItem> items;
        for (int s = 0; s + 1 < m; s++) {
            int c = p->steps[s].c;
            WsItem it;
            it.bytes = (size_t)bld.tensor_of(c, dt, {}).numel() * elem(dt);
            it.t0 = s;
            it.t1 = consumer_step(c);
            it.id = c;
            items.push_back(it);
        }
        auto fval = [&](int node) -> TensorRef {
            BufRef b;
            if (node < n) { b.kind = BUF_IN; b.index = node; }
            else if (node == (int)p->nodes.size() - 1) { b.kind = BUF_OUT; }
            else { b.kind = BUF_WS; b.index = node; }
            return bld.tensor_of(node, dt, b);
        };
        ItemScratch fs;
        fs.items = &items;
        fs.next = SCRATCH_ID;
        if (m == 0) {
            PairOp op;
            op.L = fval(0);
            op.has_r = false;
            op.C = dense_out(BUF_OUT);
            op.what = "unary";
            for (auto& l : lower_op(E, op, flags, fs)) p->fwd.push_back(l);
        }
        std::vector<PairOp> fops(m);
        for (int s = 0; s < m; s++) {
            const Step& st = p->steps[s];
            PairOp& op = fops[s];
            op.L = fval(st.a);
            op.R = fval(st.b);
            op.C = fval(st.c);
            op.convs = bld.conv_maps(st, 0);
            op.macs = st.macs;
            op.need = 0x7fffffff;
            op.what = "step " + std::to_string(s) + " fwd " + tensor_str(E, op.L) + "," +
                      tensor_str(E, op.R) + "->" + tensor_str(E, op.C);
        }
        auto node_bytes = [&](int s) {
            return (uint64_t)bld.tensor_of(p->steps[s].c, dt, {}).numel() * elem(dt);
        };
        // a contraction whose result only feeds a convolution of the
        // tensor-train pattern runs fused with it (the result stays on chip);
        // not when the caller asks to keep every intermediate for the
        // backward, nor when the save budget can hold that result (keeping it
        // then spares its recompute, which the fused chain cannot)
        std::vector<int> fused_to(m, -1), fused_from(m, -1);
        std::vector<Launch> fused(m);
        if (!(flags & CE_FLAG_GENERIC_ONLY) && !(flags & CE_FLAG_NO_FUSION) &&
            !(flags & CE_FLAG_SAVE_INTERMEDIATES)) {
            for (int s = 0; s + 1 < m; s++) {
                const int cs = consumer_step(p->steps[s].c);
                if (cs >= m || fused_from[s] >= 0 || fused_to[s] >= 0 || fused_from[cs] >= 0) continue;
                if (lim.save_budget > 0 && node_bytes(s) <= lim.save_budget) continue;
                Launch ln;
                if (!fuse_tt_forward(fops[s], fops[cs], ln)) continue;
                fused_to[s] = cs;
                fused_from[cs] = s;
                ln.need = 0;
                ln.what = "fused tensor-train steps " + std::to_string(s) + "+" + std::to_string(cs) + ": " +
                          fops[s].what.substr(fops[s].what.find("fwd ") + 4) + " then " +
                          fops[cs].what.substr(fops[cs].what.find("fwd ") + 4);
                fused[cs] = ln;
                // the producer's operands are read at the consumer's position now
                for (const TensorRef* t : {&fops[s].L, &fops[s].R})
                    if (t->buf.kind == BUF_WS)
                        for (WsItem& it : items)
                            if (it.id == t->buf.index) it.t1 = std::max(it.t1, cs);
            }
        }
        for (int s = 0; s < m; s++) {
            if (fused_to[s] >= 0) continue;
            if (fused_from[s] >= 0) {
                // the convolution's A operands laid out in load order, then the fused launch
                Launch ln = fused[s];
                TtDesc td;
                std::memcpy(&td, ln.desc.data(), sizeof(td));
                fs.t = s;
                const BufRef a2 = fs.alloc((size_t)td.U * 48 * 64 * 4);
                ln.extra.push_back(a2);
                Launch prep = ln;
                prep.kind = K_TT_PREP;
                prep.grid[0] = (uint32_t)(((int64_t)td.U * 48 * 64 + 255) / 256);
                prep.block[0] = 256;
                prep.lds = 0;
                prep.kname = "tt_prep";
                prep.alg_bytes = (double)td.U * 48 * 64 * 4;
                prep.alg_flops = 0;
                p->fwd.push_back(prep);
                p->fwd.push_back(ln);
                continue;
            }
            fops[s].need = 0;
            fs.t = s;
            for (auto& l : lower_op(E, fops[s], flags, fs)) p->fwd.push_back(l);
        }
        if (!(flags & CE_FLAG_GENERIC_ONLY) && !(flags & CE_FLAG_NO_FUSION)) {
            fuse_launches(p->fwd, false);
            Launch rf;
            if (fuse_rcp_forward(*p, rf)) p->fwd.assign(1, rf);
        }
        drop_unused(items, p->fwd);
        // Checkpointing (Section 3.3): the intermediates the forward writes
        // may be kept for the backward instead of recomputed there; all of
        // them with CE_FLAG_SAVE_INTERMEDIATES, else the set that avoids the
        // most recompute multiplications within the save budget.
        std::vector<int> cand;   // steps whose result the forward writes
        for (int s = 0; s + 1 < m; s++)
            for (const WsItem& it : items)
                if (it.id == p->steps[s].c) cand.push_back(s);
        uint32_t save = 0;
        if (flags & CE_FLAG_SAVE_INTERMEDIATES) {
            for (int s : cand) save |= 1u << s;
        } else if (lim.save_budget > 0) {
            const size_t k = cand.size();
            uint64_t best_v = 0, best_w = 0;
            uint32_t best_m = 0;
            for (uint32_t sub = 0; sub < (1u << k); sub++) {
                uint64_t v = 0, w = 0;
                uint32_t msk = 0;
                for (size_t j = 0; j < k; j++)
                    if ((sub >> j) & 1) {
                        v += p->steps[cand[j]].macs;
                        w += node_bytes(cand[j]);
                        msk |= 1u << cand[j];
                    }
                if (w > lim.save_budget) continue;
                if (v > best_v || (v == best_v && (w < best_w || (w == best_w && msk < best_m)))) {
                    best_v = v;
                    best_w = w;
                    best_m = msk;
                }
            }
            save = best_m;
        }
        p->save_mask = save;
        p->saved_bytes = 0;
        p->recompute_macs = 0;
        for (int s : cand) {
            if ((save >> s) & 1) p->saved_bytes += node_bytes(s);
        }
        auto saved_node = [&](int id) {
            for (int s = 0; s + 1 < m; s++)
                if (((save >> s) & 1) && p->steps[s].c == id) return true;
            return false;
        };
        // kept intermediates first, back to back; the rest of the forward's
        // items (and later the backward's own) packed after them
        std::vector<WsItem> kept, rest;
        for (const WsItem& it : items) (saved_node(it.id) ? kept : rest).push_back(it);
        size_t base = 0;
        for (WsItem& it : kept) {
            it.offset = base;
            base += align256(it.bytes);
        }
        p->ws_fwd = base + pack(rest);
        for (WsItem& it : rest) it.offset += base;
        items = rest;
        items.insert(items.end(), kept.begin(), kept.end());
        patch(p->fwd, items);

        // ---------------- backward ----------------
        // timeline: recompute step t at time t (t < m-1); backward of step s at
        // time (m-1) + (m-1-s).
        std::vector<WsItem> bitems;
        auto T = [&](int s) { return (m - 1) + (m - 1 - s); };
        for (int s = 0; s + 1 < m; s++) {
            int c = p->steps[s].c;
            WsItem it;
            it.bytes = (size_t)bld.tensor_of(c, dt, {}).numel() * elem(dt);
            it.t0 = s;
            it.t1 = T(consumer_step(c));
            it.id = c;
            bitems.push_back(it);
            WsItem g = it;
            g.t0 = T(consumer_step(c));
            g.t1 = T(s);
            g.id = GRAD_ID + c;
            bitems.push_back(g);
        }
        auto bval = [&](int node) -> TensorRef {
            BufRef b;
            if (node < n) { b.kind = BUF_IN; b.index = node; }
            else { b.kind = BUF_WS; b.index = node; }
            return bld.tensor_of(node, dt, b);
        };
        auto bgrad = [&](int node) -> TensorRef {
            BufRef b;
            DType gdt = dt;
            if (node < n) {
                b.kind = BUF_DIN;
                b.index = node;
                gdt = (node == E.feature_operand) ? dt : DT_F32;
            } else if (node == (int)p->nodes.size() - 1) {
                b.kind = BUF_DOUT;
            } else {
                b.kind = BUF_WS;
                b.index = GRAD_ID + node;
            }
            return bld.tensor_of(node, gdt, b);
        };
        // A plan that is exactly one fused CP chain gets the fused backward
        // (and the unfused backward is not lowered at all).
        bool fused_bwd = false;
        if (!(flags & CE_FLAG_GENERIC_ONLY) && !(flags & CE_FLAG_NO_FUSION) && p->fwd.size() == 1 &&
            (p->fwd[0].kind & 0xff) == K_CP_FWD) {
            std::vector<WsItem> fitems;
            ItemScratch fsc;
            fsc.items = &fitems;
            fsc.next = SCRATCH_ID;
            std::vector<Launch> v;
            if (fuse_cp_backward(p->fwd[0], E.feature_operand, fsc, v)) {
                p->bwd.swap(v);
                bitems.swap(fitems);
                fused_bwd = true;
            }
        }
        if (!(flags & CE_FLAG_GENERIC_ONLY) && !(flags & CE_FLAG_NO_FUSION) && p->fwd.size() == 1 &&
            (p->fwd[0].kind & 0xff) == K_RCP_FWD) {
            std::vector<WsItem> fitems;
            ItemScratch fsc;
            fsc.items = &fitems;
            fsc.next = SCRATCH_ID;
            std::vector<Launch> v;
            if (fuse_rcp_backward(p->fwd[0], *p, fsc, v)) {
                p->bwd.swap(v);
                bitems.swap(fitems);
                fused_bwd = true;
            }
        }
        ItemScratch bs;
        bs.items = &bitems;
        bs.next = SCRATCH_ID;
        if (m == 0) {
            // Y = unary(X): dX = dY broadcast back through the same label map
            PairOp op;
            op.L = dense_out(BUF_DOUT);
            op.has_r = false;
            op.C = bgrad(0);
            op.need = 1u;
            op.what = "unary bwd";
            for (auto& l : lower_op(E, op, flags, bs)) p->bwd.push_back(l);
        }
        // intermediates the forward left in the workspace are read there (a
        // fused backward recomputes on chip and reads none)
        if (fused_bwd) {
            p->save_mask = save = 0;
            p->saved_bytes = 0;
            kept.clear();
            base = 0;
            for (int s = 0; s + 1 < m; s++) p->recompute_macs += p->steps[s].macs;
        }
        if (save) {
            std::vector<WsItem> own;
            for (const WsItem& it : bitems)
                if (!saved_node(it.id)) own.push_back(it);
            bitems.swap(own);
        }
        for (int s = 0; !fused_bwd && s + 1 < m; s++) {
            if ((save >> s) & 1) continue;
            p->recompute_macs += p->steps[s].macs;
            const Step& st = p->steps[s];
            PairOp op;
            op.L = bval(st.a);
            op.R = bval(st.b);
            op.C = bval(st.c);
            op.convs = bld.conv_maps(st, 0);
            op.macs = st.macs;
            op.what = "step " + std::to_string(s) + " recompute";
            bs.t = s;
            for (auto& l : lower_op(E, op, flags, bs)) p->bwd.push_back(l);
        }
        for (int s = m - 1; !fused_bwd && s >= 0; s--) {
            const Step& st = p->steps[s];
            TensorRef dC = bgrad(st.c);
            bs.t = T(s);
            PairOp gl, gr;
            gl.L = dC;
            gl.R = bval(st.b);
            gl.C = bgrad(st.a);
            gl.convs = bld.conv_maps(st, 1);
            gl.macs = st.macs;
            gl.need = p->nodes[st.a].mask;
            gl.what = "step " + std::to_string(s) + " grad lhs " + tensor_str(E, gl.L) + "," +
                      tensor_str(E, gl.R) + "->" + tensor_str(E, gl.C);
            gr.L = bval(st.a);
            gr.R = dC;
            gr.C = bgrad(st.b);
            gr.convs = bld.conv_maps(st, 2);
            gr.macs = st.macs;
            gr.need = p->nodes[st.b].mask;
            gr.what = "step " + std::to_string(s) + " grad rhs " + tensor_str(E, gr.L) + "," +
                      tensor_str(E, gr.R) + "->" + tensor_str(E, gr.C);
            // a channel-mixing step: both gradients from one read of dC
            std::vector<Launch> pair;
            if (gl.convs.empty() && gr.convs.empty()) pair = lower_grad_pair(gl, gr, flags, bs);
            if (!pair.empty()) {
                for (auto& l : pair) p->bwd.push_back(l);
                continue;
            }
            for (const PairOp& q : bld.phase_split(st, 1, gl))
                for (auto& l : lower_op(E, q, flags, bs)) p->bwd.push_back(l);
            for (const PairOp& q : bld.phase_split(st, 2, gr))
                for (auto& l : lower_op(E, q, flags, bs)) p->bwd.push_back(l);
        }
        drop_unused(bitems, p->bwd);
        p->ws_bwd = pack(bitems);
        if (save) {
            // the backward's own items after the kept intermediates, which
            // stay at their forward offsets; the backward's size covers the
            // forward's, so one buffer serves both calls
            for (WsItem& it : bitems) it.offset += base;
            p->ws_bwd = std::max(p->ws_bwd + base, p->ws_fwd);
            bitems.insert(bitems.end(), kept.begin(), kept.end());
        }
        patch(p->bwd, bitems);
    }
    return p.release();
}

// The plan's description (built on first request, not on every plan).
std::string describe_plan(const ce_plan& p) {
    const int m = (int)p.steps.size();
    std::ostringstream txt;
    txt << "conv_einsum plan: " << p.e.n << " operands, " << m << " steps, "
        << (p.mode == CE_COST_FWD ? "fwd" : "train_paper") << " cost " << p.total_cost
        << ", forward MACs " << p.fwd_macs << ", left-to-right " << p.ltr_cost << "\n";
    for (int s = 0; s < m; s++) {
        const Step& st = p.steps[s];
        txt << "  step " << s << ": " << mask_str(p.nodes[st.a].mask) << " x "
            << mask_str(p.nodes[st.b].mask) << "  macs " << st.macs << "\n";
    }
    txt << "  workspace fwd " << p.ws_fwd << " B, bwd " << p.ws_bwd << " B\n";
    for (auto& l : p.fwd) txt << "  fwd " << l.kname << ": " << l.what << "\n";
    for (auto& l : p.bwd) txt << "  bwd " << l.kname << ": " << l.what << "\n";
    if (!p.executable) txt << "  not executable: " << p.why_not << "\n";
    return txt.str();
}

}  // namespace ce
