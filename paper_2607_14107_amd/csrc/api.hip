// Library-wide C-ABI helpers: ABI version and status names.
#include <cstring>

#include "polestar.h"

extern "C" int polestar_version(void) { return 10000; }   // 1.0.0

// A C caller may pass any int as a polestar_status; the value is read as an
// int (in C++, loading an enum object that holds a value outside the
// enumerators' range is undefined).
extern "C" const char* polestar_status_string(polestar_status s) {
    int v;
    std::memcpy(&v, &s, sizeof v);
    switch (v) {
        case POLESTAR_OK: return "ok";
        case POLESTAR_ERR_INVALID_ARGUMENT: return "invalid argument";
        case POLESTAR_ERR_UNSUPPORTED: return "unsupported shape, dtype or alignment";
        case POLESTAR_ERR_LAUNCH: return "kernel launch failed";
        case POLESTAR_ERR_WORKSPACE: return "workspace too small";
    }
    return "unknown status";
}
