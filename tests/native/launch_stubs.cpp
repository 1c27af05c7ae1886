// Host-only stand-ins for the kernel launchers and the device-scratch lookup
// (which live in the HIP sources), for building the library's host code on
// the CPU under sanitizers.  The host checks never reach a launch: with no
// device every compute entry point stops at its first HIP call.  If one were
// reached anyway, the program stops here instead of touching a device.
#include <cstdio>
#include <cstdlib>

#include "nsp_internal.hpp"

namespace nsp {

[[noreturn]] static void unreachable(const char *what) {
  std::fprintf(stderr, "host check reached a kernel launch (%s)\n", what);
  std::abort();
}

hipError_t launch_attn_fwd(int, bool, const AttnArgs &, int, hipStream_t) { unreachable("attn_fwd"); }
hipError_t launch_bwd_preprocess(int, bool, const AttnArgs &, int, hipStream_t) { unreachable("preprocess"); }
hipError_t launch_bwd_dq(int, bool, const AttnArgs &, int, hipStream_t) { unreachable("dq"); }
hipError_t launch_bwd_dkdv(int, bool, const AttnArgs &, int, hipStream_t) { unreachable("dkdv"); }
hipError_t launch_relayout(const void *, void *, const CopyTask *, int, int, hipStream_t) { unreachable("relayout"); }
hipError_t noalloc_scratch(char **) { unreachable("scratch"); }

}  // namespace nsp
