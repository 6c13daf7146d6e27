// blas.hpp -- the rocBLAS handle shared by the TTGT and LoG paths.
#pragma once
#include <hip/hip_runtime_api.h>
#include <rocblas/rocblas.h>

#include <functional>

#include "../../include/gett.h"

namespace gett {

// Runs `call` with this device's rocBLAS handle bound to `stream`, under a
// process-wide lock (the handle's stream is shared state).  The handle is
// created on first use and kept for the life of the process.
gett_status_t with_blas(hipStream_t stream, const std::function<rocblas_status(rocblas_handle)> &call);

}  // namespace gett
