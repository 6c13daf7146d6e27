// blas.cpp -- one rocBLAS handle per device for the library's GEMM calls.
#include "blas.hpp"

#include <map>
#include <mutex>

namespace gett {
namespace {
std::mutex g_blasMutex;
std::map<int, rocblas_handle> g_handles;
}  // namespace

gett_status_t with_blas(hipStream_t stream, const std::function<rocblas_status(rocblas_handle)> &call)
{
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return GETT_ERROR_HIP;
    std::lock_guard<std::mutex> lock(g_blasMutex);
    rocblas_handle &h = g_handles[dev];
    if (!h && rocblas_create_handle(&h) != rocblas_status_success) {
        h = nullptr;
        return GETT_ERROR_HIP;
    }
    if (rocblas_set_stream(h, stream) != rocblas_status_success) return GETT_ERROR_HIP;
    return call(h) == rocblas_status_success ? GETT_SUCCESS : GETT_ERROR_HIP;
}

}  // namespace gett
