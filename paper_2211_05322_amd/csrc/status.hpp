// status.hpp -- error reporting shared by the files that implement the C ABI.
#pragma once

#include <exception>
#include <new>
#include <string>

#include "../../include/reshard.h"

namespace rs {

// Record `msg` as the calling thread's last error and return `st`; never
// throws (if the text cannot be stored, the last error becomes "").
reshard_status_t fail(reshard_status_t st, const std::string &msg) noexcept;
reshard_status_t fail(reshard_status_t st, const char *msg) noexcept;

// Run an entry point's body so that no C++ exception crosses the C ABI:
// running out of host memory becomes ENOMEM, anything else an "internal:"
// EINVAL.
template <typename F>
reshard_status_t guarded(F &&body) noexcept {
    try {
        return body();
    } catch (const std::bad_alloc &) {
        return fail(RESHARD_ENOMEM, "out of host memory");
    } catch (...) {
        return fail(RESHARD_EINVAL, "internal: unexpected exception");
    }
}

}  // namespace rs
