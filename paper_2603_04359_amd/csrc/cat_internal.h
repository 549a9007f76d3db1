// Internal declarations shared by the library's translation units.
#pragma once

#include <cstddef>
#include <cstdint>
#include <string>

#include "../../include/cat.h"

namespace cat {

// Record a message for cat_last_error() and return `code`.
int fail(int code, const std::string& msg);
// Clear the thread's message (called on success paths that want it).
void clear_error();

inline bool is_pow2(int64_t v) { return v > 0 && (v & (v - 1)) == 0; }
inline bool aligned16(const void* p) {
    return (reinterpret_cast<uintptr_t>(p) & 15u) == 0;
}

}  // namespace cat
