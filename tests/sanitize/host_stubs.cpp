// host_stubs.cpp -- stand-ins for the device-code parts of libmsa (the
// kernel launchers) in the host-only build that the sanitizer test compiles
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
