#include "spl_common.h"
namespace spl {
hipError_t launch_sparse_int8(const int8_t*, const float*, int64_t, const spl_matrix&, const float*, void*, int32_t*, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_dense_int8(const int8_t*, const float*, int64_t, const int8_t*, const float*, int64_t, int64_t, void*, int32_t*, hipStream_t) { return hipErrorNotSupported; }
}
