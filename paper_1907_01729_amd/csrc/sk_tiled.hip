// sk_tiled.hip -- placeholder until the tiled sweep lands.
#include "sk_internal.h"

namespace sk {
size_t tiled_workspace_bytes(int, int, int, int) { return 0; }
hipError_t launch_tiled(const FwdArgs &, void *, hipStream_t) { return hipErrorNotSupported; }
}  // namespace sk
