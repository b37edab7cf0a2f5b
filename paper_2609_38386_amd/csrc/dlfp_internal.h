// Declarations shared by the translation units of libdlfp (not part of the ABI).
#ifndef DLFP_INTERNAL_H
#define DLFP_INTERNAL_H

#include "dlfp.h"

namespace dlfp {

// DLFP_OK if dims are supported; *group receives Hq / Hkv.
int check_dims(const dlfp_dims* dims, int* group);

}  // namespace dlfp

#endif  // DLFP_INTERNAL_H
