// Host-only stand-ins for the gfx950 launch interface (mtn_kernels.h), linked
// into the sanitizer build of the host library instead of the kernels: that
// build is compiled by g++ with AddressSanitizer and UndefinedBehaviorSanitizer
// and exercises the planner, the block tables and the admission controller on
// host-only pools, which never launch.  Every launch here fails with
// hipErrorNotSupported; the shape queries answer as the kernels do.
#include "mtn_kernels.h"

namespace mtn {

hipError_t launch_plan_apply(const int32_t *, const int32_t *, int32_t, int32_t *, const int32_t *,
                             int32_t, const double *, int32_t, float2 *, hipStream_t) {
    return hipErrorNotSupported;
}
hipError_t launch_append(int, const PoolGeom &, const PlanView &, int32_t, const void *,
                         const void *, const int32_t *, const int32_t *, int32_t, hipStream_t) {
    return hipErrorNotSupported;
}
hipError_t launch_attn_valu(int, const AttnArgs &, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_merge(int, const AttnArgs &, hipStream_t) { return hipErrorNotSupported; }
int prefill_rows_per_pass() { return 256; }
bool prefill_pass_rows_valid(int rows) { return rows == 128 || rows == 256; }
hipError_t launch_prefill_mfma(int, const AttnArgs &, const int32_t *, int32_t, int32_t,
                               const uint8_t *, hipStream_t) {
    return hipErrorNotSupported;
}
hipError_t launch_poison(int, const PoolGeom &, int32_t, int64_t, const uint16_t *, hipStream_t) {
    return hipErrorNotSupported;
}
hipError_t launch_copy(const void *, void *, size_t, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_read(const void *, size_t, uint32_t *, hipStream_t) {
    return hipErrorNotSupported;
}
hipError_t scratch_buffer(float **, size_t *) { return hipErrorNotSupported; }
int fp8_head_stride(int d) { return d == 128 ? 4224 : 0; }
static bool group_ok(int g) { return g == 1 || g == 2 || g == 4 || g == 8; }
bool attn_fp8_supported(int d, int g) { return d == 128 && group_ok(g); }
int attn_fp8_resident_per_cu(int) { return 1; }
hipError_t launch_append_fp8(const PoolGeom &, const PlanView &, int32_t, const void *, const void *,
                             hipStream_t) {
    return hipErrorNotSupported;
}
hipError_t launch_attn_fp8(const AttnArgs &, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_poison_fp8(const PoolGeom &, int32_t, int64_t, const uint16_t *, hipStream_t) {
    return hipErrorNotSupported;
}
bool attn_mfma_bf16_supported(int d, int g) { return attn_fp8_supported(d, g); }
int attn_mfma_bf16_resident_per_cu(int) { return 1; }
hipError_t launch_attn_mfma_bf16(const AttnArgs &, hipStream_t) { return hipErrorNotSupported; }
bool attn_valu_supported(int dtype, int d, int g) {
    return (dtype == 0 || dtype == 1) && (d == 64 || d == 128) && group_ok(g);
}
int attn_valu_resident_per_cu(int, int, int) { return 1; }
bool prefill_mfma_supported(int dtype, int d, int g) {
    return (dtype == 1 || dtype == 2) && d == 128 && group_ok(g);
}

}  // namespace mtn
