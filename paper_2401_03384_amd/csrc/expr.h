// Parsed and size-bound conv_einsum expression (host side).
//
// Grammar: Section 2.2 ('From einsum to conv_einsum') and the layer strings of
// Appendix A.3.  Sizes: Appendix A (sizes of a non-convolved label agree) and
// Appendix B, 'Convolution Varieties' (of the two holders of a convolved
// label, the larger size is the feature side).
#pragma once

#include <cstdint>
#include <string>
#include <vector>

#include "common.h"

struct ce_expr {
    int n = 0;                                  // operands
    std::vector<std::string> names;             // label id -> name
    std::vector<std::vector<int>> ops;          // operand -> label ids, string order
    std::vector<std::vector<int64_t>> dims;     // operand -> sizes, string order
    std::vector<int> out;                       // output label ids
    uint64_t conv = 0;                          // bit per convolved label
    uint64_t out_mask = 0;                      // bit per output label
    std::vector<uint32_t> holders;              // label -> bitmask of operands holding it
    std::vector<int> stride;                    // label -> stride of a convolved label (1: none)
    std::vector<uint8_t> circular;              // label -> convolved circularly (commutative)
    int feature_operand = 0;
    bool bound = false;

    int num_labels() const { return (int)names.size(); }
    bool is_conv(int l) const { return (conv >> l) & 1; }
    bool in_out(int l) const { return (out_mask >> l) & 1; }
    // size of label l in operand i (label must be held by i)
    int64_t size_in(int i, int l) const;
    // feature operand of a two-way convolved label (-1 if none)
    int feature_of(int l) const;
    int64_t out_size(int l) const;
    int stride_of(int l) const { return l < (int)stride.size() ? stride[l] : 1; }
    bool is_circular(int l) const { return l < (int)circular.size() && circular[l]; }
    std::vector<int64_t> out_dims() const;
};

namespace ce {
// Parse `spec` and bind sizes; throws ce::Error.
ce_expr* parse_expr(const char* spec, int n_in, const int* ranks, const int64_t* const* dims);
}
