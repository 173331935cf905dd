// The exported functions of libhwr run their bodies through c_boundary: a
// host-side exception (a host allocation that fails, a thread that cannot
// start) becomes HWR_ERR_OOM, its message goes to `note` (where the function's
// errors are read), and nothing propagates into the caller's frame.  No HIP
// dependency: the host-only simulator uses it too.
#pragma once

#include <exception>

#include "hwr.h"

namespace hwr {

template <class Body, class Note>
hwr_status c_boundary(Body &&body, Note &&note) noexcept {
    try {
        return body();
    } catch (const std::exception &e) {
        try {
            note(e.what());
        } catch (...) {
        }
    } catch (...) {
        try {
            note("unknown host exception");
        } catch (...) {
        }
    }
    return HWR_ERR_OOM;
}

}  // namespace hwr
