// host_stubs.cpp -- stand-ins for the device-code parts of libmsa (the
// kernel launchers, and the no-allocation entry point, whose workspace is a
// device array) in the host-only build that the sanitizer test compiles
// with g++.  Host-only plans never reach them; each returns an error if
// called.
#include "msa.h"
#include "msa_internal.h"
#include "append.h"

namespace msa {
int launch_attn(const AttnParams&, int, int, int, void*) { return 98; }  // hipErrorInvalidDeviceFunction
int launch_merge(const MergeParams&, int, int, void*) { return 98; }
int launch_kv_append(const AppendParams&, int, int, void*) { return 98; }
}  // namespace msa

extern "C" msa_status msa_forward_noalloc(msa_plan_t, const void*, const void*, const void*,
                                          const int32_t*, void*, float*, void*) {
  return MSA_ERR_UNSUPPORTED;
}
