// Stand-in for the gfx950 kernel launchers, for host-only sanitizer builds of
// the ABI layer: every call the host driver makes is rejected before a launch,
// so reaching any of these is a failure.
#include <stdio.h>
#include <stdlib.h>

#include "internal.h"

namespace murmur {
static int reached(const char *what) {
    fprintf(stderr, "a kernel launcher was reached: %s\n", what);
    abort();
}
int launch_evict_compact(const murmur_seg *, const murmur_policy *, int32_t, int32_t, int32_t *, int32_t, int32_t *,
                         int32_t *, const int32_t *, int32_t, int32_t, murmur_stream_t) {
    return reached("evict_compact");
}
int launch_decode_attn(const AttnLaunch &, murmur_stream_t) { return reached("decode_attn"); }
int launch_workspace_init(int32_t *, int64_t, murmur_stream_t) { return reached("workspace_init"); }
int launch_read_probe(const void *, int64_t, int32_t, int32_t, int32_t, bool, uint32_t *, murmur_stream_t) {
    return reached("read_probe");
}
int launch_paged_step(const murmur_seg *, const murmur_policy *, int32_t, int32_t, int32_t *, int32_t, int32_t,
                      int32_t *, int32_t *, int32_t, int32_t, murmur_stream_t) {
    return reached("paged_step");
}
int launch_paged_append(const murmur_seg *, int32_t, const int32_t *, int32_t, int32_t, const murmur_kv &, int32_t,
                        const void *, const void *, murmur_stream_t) {
    return reached("paged_append");
}
int static_scratch(void **, bool *) { return reached("static_scratch"); }
int read_and_clear_device_error(murmur_stream_t, int32_t *) { return reached("device_error"); }
const char *hip_error_text(int) { return "stub"; }
}  // namespace murmur
