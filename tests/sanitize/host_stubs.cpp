// Host-only stand-ins for the device side of libtreekv.so, linked instead of the HIP objects into a
// sanitizer build of the host library (block manager, planner, search controller, C entry points)
// that the CPU tests load without a GPU.  Every device entry point fails with TKV_EHIP and touches
// nothing; a plan's destructor returns its host image to the planner's pool, as the real one does.
#include "internal.h"

namespace tkv {
int launch_attention(const tkv_plan*, const void*, const void*, const void*, void*, float*, void*) {
    return set_error(TKV_EHIP, "attention: host-only build, no device");
}
int upload(tkv_plan*, void*, size_t, void*) { return set_error(TKV_EHIP, "tkv_plan_upload: host-only build, no device"); }
void wait_copies(const tkv_plan*) {}  // no copies without a device
}  // namespace tkv

tkv_plan::~tkv_plan() { tkv::give_image(std::move(image), image_cap); }

TKV_EXPORT int tkv_plan_profile(tkv_plan*, int32_t) {
    tkv::clear_error();
    return tkv::set_error(TKV_EHIP, "tkv_plan_profile: host-only build, no device");
}
TKV_EXPORT int tkv_plan_profile_read(tkv_plan*, int32_t*, float*, float*) {
    tkv::clear_error();
    return tkv::set_error(TKV_EHIP, "tkv_plan_profile_read: host-only build, no device");
}
TKV_EXPORT int tkv_verify_noalloc(const tkv_plan*, const void*, const void*, const void*, void*, float*, void*) {
    tkv::clear_error();
    return tkv::set_error(TKV_EHIP, "tkv_verify_noalloc: host-only build, no device");
}
TKV_EXPORT int tkv_kv_append(const tkv_shape*, const int32_t*, int32_t, const void*, const void*, void*, void*, void*) {
    tkv::clear_error();
    return tkv::set_error(TKV_EHIP, "tkv_kv_append: host-only build, no device");
}
TKV_EXPORT int tkv_cd_sample(int32_t, int32_t, float, int32_t, const float*, const float*, const int32_t*, int32_t, int32_t*,
                             int32_t*, int32_t*, void*) {
    tkv::clear_error();
    return tkv::set_error(TKV_EHIP, "tkv_cd_sample: host-only build, no device");
}
