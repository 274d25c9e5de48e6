// Status strings, thread-local error detail and launch checking.
#include <stdio.h>

#include "sg_internal.h"

namespace sg {

static thread_local char g_err[512] = "";

void set_error(const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof(g_err), fmt, ap);
    va_end(ap);
}

void clear_error() { g_err[0] = '\0'; }

int launch_status(const char *what) {
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) {
        set_error("%s: kernel launch failed: %s", what, hipGetErrorString(e));
        return SG_EHIP;
    }
    return SG_OK;
}

bool host_memory(const void *p) {
    hipPointerAttribute_t a;
    if (hipPointerGetAttributes(&a, p) != hipSuccess) {
        (void)hipGetLastError();   // an unknown pointer is not an error of the next launch
        return false;
    }
    return a.type == hipMemoryTypeHost;
}

}  // namespace sg

extern "C" int sg_version(void) { return 100; }

extern "C" const char *sg_status_str(int status) {
    switch (status) {
        case SG_OK: return "ok";
        case SG_EINVAL: return "invalid argument";
        case SG_EUNSUPPORTED: return "unsupported configuration";
        case SG_EWORKSPACE: return "workspace or destination too small";
        case SG_EHIP: return "HIP runtime error";
        case SG_EINTERNAL: return "internal error";
        default: return "unknown status";
    }
}

extern "C" const char *sg_last_error(void) { return sg::g_err; }
