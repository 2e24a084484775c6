// Exception barrier of the C ABI: the host code behind an entry point may
// throw (std::bad_alloc from a container, std::system_error from a thread
// that cannot be started); the entry point returns DTE_ERR_HOST instead of
// letting the exception cross the C interface.
#pragma once

#include "../../include/dte.h"

namespace dte {

template <typename F>
dte_status no_throw(F&& f) noexcept
{
    try {
        return f();
    } catch (...) {
        return DTE_ERR_HOST;
    }
}

}  // namespace dte
