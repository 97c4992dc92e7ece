// Library-wide C-ABI helpers: ABI version and status names.
#include "polestar.h"

extern "C" int polestar_version(void) { return 10000; }   // 1.0.0

extern "C" const char* polestar_status_string(polestar_status s) {
    switch (s) {
        case POLESTAR_OK: return "ok";
        case POLESTAR_ERR_INVALID_ARGUMENT: return "invalid argument";
        case POLESTAR_ERR_UNSUPPORTED: return "unsupported shape, dtype or alignment";
        case POLESTAR_ERR_LAUNCH: return "kernel launch failed";
        case POLESTAR_ERR_WORKSPACE: return "workspace too small";
    }
    return "unknown status";
}
