// Internal helpers shared by the host-side sources (no HIP dependency).
#pragma once

#include <cstdint>
#include <stdexcept>
#include <string>

#include "../../include/convein.h"

namespace ce {

// Internal error carrying a ce_status; converted to a status code at the ABI.
struct Error : std::runtime_error {
    ce_status status;
    Error(ce_status s, const std::string& msg) : std::runtime_error(msg), status(s) {}
};

[[noreturn]] inline void fail(ce_status s, const std::string& msg) { throw Error(s, msg); }

inline int popcount64(uint64_t x) { return __builtin_popcountll(x); }
inline int lowest_bit(uint64_t x) { return __builtin_ctzll(x); }

// a * b with overflow detection (exact unsigned 64-bit arithmetic).
inline uint64_t mul_checked(uint64_t a, uint64_t b) {
    unsigned __int128 r = (unsigned __int128)a * b;
    if (r >> 64) fail(CE_ERR_OVERFLOW, "cost or size exceeds 64 bits");
    return (uint64_t)r;
}
inline uint64_t add_checked(uint64_t a, uint64_t b) {
    uint64_t r = a + b;
    if (r < a) fail(CE_ERR_OVERFLOW, "cost exceeds 64 bits");
    return r;
}

}  // namespace ce
