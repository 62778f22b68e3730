// conv_einsum string parser and size binding.
#include "expr.h"

#include <cctype>
#include <memory>

namespace {

using ce::fail;

struct Lexer {
    std::string s;   // blanks removed
    size_t i = 0;
    bool done() const { return i >= s.size(); }
    char peek() const { return s[i]; }
};

// One label at the cursor: a letter, or '(' alnum/_ name ')'.
std::string read_label(Lexer& lx, const char* where) {
    char c = lx.peek();
    if (c == '(') {
        size_t j = lx.s.find(')', lx.i);
        if (j == std::string::npos) fail(CE_ERR_PARSE, std::string("unclosed '(' in ") + where);
        std::string name = lx.s.substr(lx.i + 1, j - lx.i - 1);
        if (name.empty()) fail(CE_ERR_PARSE, std::string("empty label in ") + where);
        for (char ch : name)
            if (!(std::isalnum((unsigned char)ch) || ch == '_'))
                fail(CE_ERR_PARSE, std::string("bad label '(") + name + ")' in " + where);
        lx.i = j + 1;
        return name;
    }
    if (std::isalpha((unsigned char)c)) {
        lx.i++;
        return std::string(1, c);
    }
    fail(CE_ERR_PARSE, std::string("unexpected character '") + c + "' in " + where);
}

}  // namespace

int64_t ce_expr::size_in(int i, int l) const {
    for (size_t k = 0; k < ops[i].size(); k++)
        if (ops[i][k] == l) return dims[i][k];
    return -1;
}

int ce_expr::feature_of(int l) const {
    if (!is_conv(l) || ce::popcount64(holders[l]) != 2 || is_circular(l)) return -1;
    int a = ce::lowest_bit(holders[l]);
    int b = ce::lowest_bit(holders[l] & ~(1u << a));
    int64_t da = size_in(a, l), db = size_in(b, l);
    if (da != db) return da > db ? a : b;
    if (feature_operand == a || feature_operand == b) return feature_operand;
    return a;
}

int64_t ce_expr::out_size(int l) const {
    int f = feature_of(l);
    if (f >= 0) {
        const int64_t s = stride_of(l);
        return (size_in(f, l) + s - 1) / s;   // ceil(I / s) positions (I for stride 1)
    }
    int64_t m = 0;
    for (int i = 0; i < n; i++)
        if ((holders[l] >> i) & 1) m = std::max(m, size_in(i, l));
    return m;
}

std::vector<int64_t> ce_expr::out_dims() const {
    std::vector<int64_t> d;
    for (int l : out) d.push_back(out_size(l));
    return d;
}

namespace ce {

ce_expr* parse_expr(const char* spec, int n_in, const int* ranks, const int64_t* const* dims) {
    if (!spec) fail(CE_ERR_ARG, "spec is NULL");
    std::unique_ptr<ce_expr> e(new ce_expr());
    Lexer lx;
    for (const char* p = spec; *p; p++)
        if (!std::isspace((unsigned char)*p)) lx.s.push_back(*p);

    auto label_id = [&](const std::string& name) -> int {
        for (size_t k = 0; k < e->names.size(); k++)
            if (e->names[k] == name) return (int)k;
        if ((int)e->names.size() >= CE_MAX_LABELS)
            fail(CE_ERR_UNSUPPORTED, "more than 64 distinct labels");
        e->names.push_back(name);
        return (int)e->names.size() - 1;
    };

    size_t arrow = lx.s.find("->");
    if (arrow == std::string::npos || lx.s.find("->", arrow + 2) != std::string::npos)
        fail(CE_ERR_PARSE, "a conv_einsum string needs exactly one '->'");
    // operands
    std::vector<std::vector<int>> ops(1);
    while (lx.i < arrow) {
        char c = lx.peek();
        if (c == ',') {
            ops.emplace_back();
            lx.i++;
            continue;
        }
        if (c == '|') fail(CE_ERR_PARSE, "'|' must follow the output term");
        std::string nm = read_label(lx, "an operand");
        if (lx.i > arrow) fail(CE_ERR_PARSE, "label runs into '->'");
        int id = label_id(nm);
        for (int x : ops.back())
            if (x == id)
                fail(CE_ERR_PARSE, "operand " + std::to_string(ops.size() - 1) + " repeats label " + nm);
        ops.back().push_back(id);
    }
    lx.i = arrow + 2;
    // output
    std::vector<int> out;
    while (!lx.done() && lx.peek() != '|') {
        std::string nm = read_label(lx, "the output");
        int id = -1;
        for (size_t k = 0; k < e->names.size(); k++)
            if (e->names[k] == nm) id = (int)k;
        if (id < 0) fail(CE_ERR_PARSE, "output label " + nm + " is in no operand");
        for (int x : out)
            if (x == id) fail(CE_ERR_PARSE, "output repeats label " + nm);
        out.push_back(id);
    }
    uint64_t conv = 0;
    if (!lx.done()) {
        lx.i++;  // '|'
        while (!lx.done()) {
            if (lx.peek() == ',') {
                lx.i++;
                continue;
            }
            if (lx.peek() == '|') fail(CE_ERR_PARSE, "at most one '|'");
            std::string nm = read_label(lx, "the convolution list");
            int id = -1;
            for (size_t k = 0; k < e->names.size(); k++)
                if (e->names[k] == nm) id = (int)k;
            if (id < 0) fail(CE_ERR_PARSE, "convolved label " + nm + " is in no operand");
            if ((conv >> id) & 1) fail(CE_ERR_PARSE, "convolved label " + nm + " listed twice");
            conv |= 1ull << id;
        }
    }
    uint64_t out_mask = 0;
    for (int l : out) out_mask |= 1ull << l;
    if (conv & ~out_mask) fail(CE_ERR_PARSE, "every convolved label must be kept in the output");
    if ((int)ops.size() > CE_MAX_OPERANDS) fail(CE_ERR_UNSUPPORTED, "more than 16 operands");

    // sizes
    if (n_in != (int)ops.size())
        fail(CE_ERR_SHAPE, "string has " + std::to_string(ops.size()) + " operands, got " +
                               std::to_string(n_in));
    if (!ranks || !dims) fail(CE_ERR_ARG, "ranks/dims is NULL");
    e->n = n_in;
    e->ops = ops;
    e->out = out;
    e->conv = conv;
    e->out_mask = out_mask;
    e->dims.resize(n_in);
    e->holders.assign(e->names.size(), 0);
    e->stride.assign(e->names.size(), 1);
    e->circular.assign(e->names.size(), 0);
    for (int i = 0; i < n_in; i++) {
        if (ranks[i] != (int)ops[i].size())
            fail(CE_ERR_SHAPE, "operand " + std::to_string(i) + ": rank " + std::to_string(ranks[i]) +
                                   " but " + std::to_string(ops[i].size()) + " labels");
        if (ranks[i] > 0 && !dims[i]) fail(CE_ERR_ARG, "dims[i] is NULL");
        for (int k = 0; k < ranks[i]; k++) {
            if (dims[i][k] < 1) fail(CE_ERR_SHAPE, "sizes must be >= 1");
            if (dims[i][k] > (int64_t(1) << 40)) fail(CE_ERR_OVERFLOW, "size too large");
            e->dims[i].push_back(dims[i][k]);
            e->holders[ops[i][k]] |= 1u << i;
        }
    }
    for (int l = 0; l < e->num_labels(); l++) {
        if (e->is_conv(l)) continue;
        int64_t s = -1;
        for (int i = 0; i < n_in; i++) {
            int64_t d = e->size_in(i, l);
            if (d < 0) continue;
            if (s >= 0 && d != s)
                fail(CE_ERR_SHAPE, "label " + e->names[l] + " has sizes " + std::to_string(s) +
                                       " and " + std::to_string(d));
            s = d;
        }
    }
    // a label convolved among three or more operands is circular (the only
    // multi-way kind, Appendix B 'Convolution Varieties')
    for (int l = 0; l < e->num_labels(); l++)
        if (e->is_conv(l) && ce::popcount64(e->holders[l]) > 2) e->circular[l] = 1;
    e->bound = true;
    return e.release();
}

}  // namespace ce
