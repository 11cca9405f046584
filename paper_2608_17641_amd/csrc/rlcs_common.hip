// Entry points that launch nothing: workspace size, status strings, version, and the test-only
// variant override.
#include "rlcs_dispatch.h"
#include "rlcs_testing.h"

using namespace rlcs;
using namespace rlcs::host;

namespace rlcs {
namespace host {
thread_local int g_variant = 0;
}  // namespace host
}  // namespace rlcs

extern "C" {

size_t rlcs_workspace_size(int64_t N, int64_t T) {
    if (N <= 0 || T <= 0) return kWsRecordsOffset;
    if (N > INT64_MAX / T) return 0;
    // N * (tiles per row) records, at most kMinTile steps per tile
    const int64_t per_row = (T + kMinTile - 1) / kMinTile;
    if (N > int64_t((SIZE_MAX - kWsRecordsOffset) / kWsRecordBytes) / per_row) return 0;
    return kWsRecordsOffset + size_t(N * per_row) * kWsRecordBytes;
}

const char* rlcs_status_string(rlcs_status status) {
    switch (status) {
        case RLCS_OK: return "RLCS_OK";
        case RLCS_ERR_INVALID_ARG: return "RLCS_ERR_INVALID_ARG: invalid size, pointer, parameter or enum";
        case RLCS_ERR_DTYPE: return "RLCS_ERR_DTYPE: unsupported dtype";
        case RLCS_ERR_WORKSPACE: return "RLCS_ERR_WORKSPACE: workspace missing or too small";
        case RLCS_ERR_LAUNCH: return "RLCS_ERR_LAUNCH: kernel launch failed";
    }
    return "unknown rlcs_status";
}

int rlcs_version(void) { return 100; }

rlcs_status rlcs_testing_set_variant(int variant) {
    if (variant < 0 || variant > 4) return RLCS_ERR_INVALID_ARG;
    g_variant = variant;
    return RLCS_OK;
}

}  // extern "C"
