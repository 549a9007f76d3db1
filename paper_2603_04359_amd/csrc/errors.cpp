// Thread-local error reporting for the C ABI.
#include <string>

#include "cat_internal.h"

namespace {
thread_local std::string g_last_error;
}

namespace cat {

int fail(int code, const std::string& msg) {
    g_last_error = msg;
    return code;
}

void clear_error() { g_last_error.clear(); }

}  // namespace cat

extern "C" const char* cat_last_error(void) { return g_last_error.c_str(); }

extern "C" const char* cat_version(void) { return "cat-mi355x 0.1"; }
