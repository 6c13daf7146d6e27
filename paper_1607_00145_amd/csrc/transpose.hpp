// transpose.hpp -- host entry of the Eq. 4 transposition kernel.
#pragma once
#include <hip/hip_runtime_api.h>
#include <stdint.h>

#include "../../include/gett.h"
#include "desc.hpp"

namespace gett {

// out[Pi(i)] <- alpha * in[i] + beta * out[Pi(i)] over the iteration space
// ext[0..rank) with input strides sin and output strides sout (elements).
// The caller has validated the arguments: offsets below 2^31, output strides
// injective, in and out not overlapping when alpha != 0.  `in` is not read
// when alpha == 0, `out` is not read when beta == 0.
gett_status_t transpose_launch(gett_dtype_t dtype, int rank, const int64_t *ext,
                               const int64_t *sin, const int64_t *sout, double alpha,
                               const void *in, double beta, void *out, hipStream_t stream);

}  // namespace gett
