// Specialised kernels: dispatch by launch kind.
#include "desc.h"
#include "hip_util.h"
#include "kernels.h"

namespace ce {

hipError_t launch_fast(const Launch& ln, const void* a, const void* b, void* c, void* d,
                       hipStream_t s) {
    (void)ln; (void)a; (void)b; (void)c; (void)d; (void)s;
    return hipErrorInvalidValue;
}

}  // namespace ce
