// Argument checks shared by the C-ABI translation units (mfpsn_api.cpp,
// mfpsn_api_ext.cpp).  Not installed; not part of the ABI.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "mfpsn.h"

namespace mfpsn {

// Storage bytes of one element of x (and of the streaming ring)
inline int elem_bytes(int dtype) { return dtype == MFPSN_F32 ? 4 : 2; }
inline bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }
// The descriptor's fields, as every whole-sequence entry point needs them:
// MFPSN_OK or the status the call returns
int validate(const mfpsn_desc* d);

}  // namespace mfpsn
