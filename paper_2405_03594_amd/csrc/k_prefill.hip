#include "spl_common.h"
namespace spl {
hipError_t launch_sparse_prefill(const void*, int64_t, const spl_matrix&, void*, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_dense_prefill(const void*, int64_t, const void*, int32_t, int64_t, int64_t, void*, hipStream_t) { return hipErrorNotSupported; }
}
