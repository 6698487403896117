// Host-only build of the library for the sanitizer test: every device
// launcher fails with hipErrorInvalidValue, so only the host steps (argument
// checks, assignment, clique, simulator, row tables) can run.
#include <hip/hip_runtime_api.h>

#include "../../paper_2108_02416_amd/csrc/aspis_internal.h"

namespace aspis {

size_t workspace_bytes(int64_t f, int r) {
    return (size_t)f * 12 + 256 + 1024 + (size_t)f * r * 4 + 1024 + (size_t)f + kDirtyWords * 4 + 256;
}
Workspace carve_workspace(void *, int64_t, int) { return Workspace{}; }
hipError_t launch_fill_u32(uint32_t *, int64_t, uint32_t, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_fill_u64(uint64_t *, int64_t, uint64_t, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_agree(const float *, const int32_t *, int64_t, int, int64_t, int64_t, uint32_t *,
                        hipStream_t) {
    return hipErrorInvalidValue;
}
hipError_t launch_agree_file(const float *, const int32_t *, int64_t, int, int64_t, const ProbeSet &,
                             uint32_t *, hipStream_t) {
    return hipErrorInvalidValue;
}
hipError_t launch_vote(const uint32_t *, const int32_t *, int64_t, int, int8_t *, uint8_t *,
                       uint64_t *, hipStream_t) {
    return hipErrorInvalidValue;
}
hipError_t launch_vote_rows(const uint32_t *, const int32_t *, int64_t, int, int, int8_t *,
                            uint8_t *, uint64_t *, uint64_t *, hipStream_t) {
    return hipErrorInvalidValue;
}
hipError_t launch_select(const int32_t *, const int8_t *, int64_t, int, int, uint64_t,
                         const int32_t *, const Workspace &, int32_t *, uint32_t *, int64_t,
                         hipStream_t) {
    return hipErrorInvalidValue;
}
bool plan_median(int64_t, bool, KernelPlan *out, bool) {
    *out = KernelPlan{};
    out->kind = kKernelMedianRadix;
    return true;
}
bool plan_fused(int64_t, int, bool, bool, KernelPlan *out, bool) {
    *out = KernelPlan{};
    return false;
}
hipError_t launch_median(const float *, int64_t, const Workspace &, int64_t, float *, hipStream_t,
                         TileUse *, bool, bool) {
    return hipErrorInvalidValue;
}
hipError_t launch_mean(const float *, int64_t, const Workspace &, float *, hipStream_t, bool) {
    return hipErrorInvalidValue;
}
hipError_t launch_fused(const float *, const int32_t *, int64_t, int, int64_t, const Workspace &,
                        uint32_t *, float *, hipStream_t, TileUse *, bool) {
    return hipErrorInvalidValue;
}
bool fused_supported(int64_t, int) { return false; }
hipError_t launch_fused_mean(const float *, const int32_t *, int64_t, int, int64_t,
                             const Workspace &, uint32_t *, float *, hipStream_t) {
    return hipErrorInvalidValue;
}
bool fused_mean_supported(int64_t, int) { return false; }
hipError_t scratch_ptr(void **) { return hipErrorInvalidValue; }
hipError_t launch_tie_probe(const float *, const int32_t *, int64_t, int, int64_t, const ProbeSet &,
                            uint32_t *, hipStream_t) {
    return hipErrorInvalidValue;
}
hipError_t launch_save_sel(const Workspace &, int64_t, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_dirty_tiles(const float *, const int32_t *, int64_t, int, int64_t, const Workspace &,
                              const uint32_t *, int, hipStream_t) {
    return hipErrorInvalidValue;
}
int reduce_tile_cols(const float *, int64_t, int64_t, bool, bool) { return 0; }
size_t read_probe_sink_words() { return 0; }
hipError_t launch_read_probe(const void *, size_t, uint32_t *, hipStream_t) {
    return hipErrorInvalidValue;
}

}  // namespace aspis
