// Host-side helpers shared by the C-ABI entry points: argument checks and
// launch status.  Nothing here calls the HIP runtime except launch_status().
#pragma once

#include <hip/hip_runtime.h>
#include <cstring>
#include <stddef.h>
#include <stdint.h>

#include "polestar.h"

namespace ps {

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Whether a caller's dtype argument names a supported type.  Taken by
// reference and read as an int: a C caller may pass any int, and in C++
// loading an enum object that holds a value outside the enumerators' range is
// undefined, so the value is checked before any enum-typed use.
inline bool dtype_ok(const polestar_dtype& dt) {
    int v;
    std::memcpy(&v, &dt, sizeof v);
    return v == POLESTAR_FP32 || v == POLESTAR_BF16;
}

inline size_t elem_bytes(polestar_dtype dt) { return dt == POLESTAR_BF16 ? 2 : 4; }

// Rows of `n` elements must be whole 16-byte chunks.
inline bool row_ok(polestar_dtype dt, long n) {
    return dt == POLESTAR_BF16 ? (n % 8) == 0 : (n % 4) == 0;
}

inline polestar_status launch_status() {
    hipError_t e = hipGetLastError();
    return e == hipSuccess ? POLESTAR_OK : POLESTAR_ERR_LAUNCH;
}

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

inline int ceil_div(long a, long b) { return static_cast<int>((a + b - 1) / b); }

}  // namespace ps
