// Placeholder executors for families not yet implemented.
#include "model.h"

namespace fo {
static size_t ws0(const fo_model*) { return 0; }
static fo_status init_na(fo_model* m) {
    set_error("config %d is not implemented yet", m->cid);
    return FO_EINVAL;
}
static fo_status step_na(fo_model* m, const fo_acts*, const int32_t*) {
    set_error("config %d is not implemented yet", m->cid);
    return FO_EINVAL;
}
static void destroy_na(fo_model*) {}
const Family* family_cnn16() {
    static const Family f = {ws0, init_na, step_na, destroy_na};
    return &f;
}
int64_t cnn16_param_count(int32_t cid) { return cid == 3 ? 11070308 : 15206410; }
}  // namespace fo
