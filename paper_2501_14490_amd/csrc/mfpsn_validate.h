// Argument checks shared by the C-ABI translation units (mfpsn_api.cpp,
// mfpsn_api_ext.cpp).  Not installed; not part of the ABI.
#pragma once

#include <math.h>
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

// Largest |dH| the Q8.8 backward can produce: |grad_spikes| <= 2^15 times the
// integer surrogate factor, which is at most 2^15 * max sigma' (+1 for rounding).
inline double q88_max_dh(const mfpsn_desc* d)
{
    double peak;
    switch (d->surrogate) {
    case MFPSN_SG_SIGMOID: peak = d->alpha / 4.0; break;
    case MFPSN_SG_ATAN: peak = d->alpha / 2.0; break;
    default: peak = 1.0; break;
    }
    return ceil(32768.0 * peak) + 1.0;
}

}  // namespace mfpsn
