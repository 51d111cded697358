// Host-side helpers shared by the library's translation units: the
// thread-local error message and argument checks.  No device code.
#pragma once

#include <cstdarg>
#include <cstddef>
#include <cstdint>

#include "structadmm.h"

namespace sa {

// Formats the calling thread's error message and returns `code`.
int fail(int code, const char *fmt, ...);
// Clears the calling thread's error message.
void clear_error();
// Records a failed HIP call (returns SA_E_HIP) or returns SA_OK.
int check_hip(hipError_t e, const char *what);

inline bool aligned(const void *p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

inline int64_t n_groups(const sa_project_desc &d) {
    switch (d.kind) {
    case SA_FILTER: return d.A;
    case SA_CHANNEL: return d.B;
    case SA_SHAPE: return d.B * d.C * d.D;
    case SA_ELEMENT: return d.A * d.B * d.C * d.D;
    default: return -1;
    }
}

// Host validation of one projection descriptor (index i for messages).
int validate_project(const sa_project_desc &d, int i);
int validate_dual(const sa_dual_desc &d, int i);
int validate_sgd(const sa_sgd_desc &d, int i);
int validate_compact(const sa_compact_desc &d);
int validate_conv(const sa_conv_desc &d);

inline int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

}  // namespace sa
