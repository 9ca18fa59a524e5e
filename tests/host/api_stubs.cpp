// Host-only stand-ins for the kernel entry points of kernels.hip, so that the
// C-ABI layer (api.cpp) can be built with g++ under the sanitizers.  Launches
// do nothing and succeed: no kernel runs, so nothing ever reads the fake
// buffer addresses the checks use.  The sizes follow kernels.hip's variants;
// they only shape the launch-level steps the host code builds.
#include "kernels.hpp"

namespace pat {

int variant_in_bytes(Variant v) {
  switch (v) {
    case kAgVec: case kRsI32Vec: case kRsF32Vec: case kAgVecU: case kRsI32VecU: case kRsF32VecU: return 16;
    case kRsB16Vec: case kRsB16VecU: return 8;
    case kAgS4: case kRsI32S: case kRsF32S: return 4;
    default: return 2;
  }
}
bool variant_partial(Variant v) { return v == kAgVecU || v == kRsI32VecU || v == kRsF32VecU || v == kRsB16VecU; }
bool variant_partial_items(Variant v) { return v == kRsB16VecU; }
int variant_tile(Variant v) { return v == kAgS4 || v == kAgS2 || v == kRsI32S || v == kRsF32S || v == kRsB16S ? 2048 : v == kRsB16Vec || v == kRsB16VecU ? 1024 : 512; }
int variant_pack_tile(Variant v) { return v == kAgS4 || v == kAgS2 || v == kRsI32S || v == kRsF32S || v == kRsB16S ? 1024 : v == kRsB16Vec || v == kRsB16VecU ? 1024 : 512; }

hipError_t launch_step(Variant, bool, int64_t, const KCtx&, const DevStep&, hipStream_t) { return hipSuccess; }
hipError_t launch_tree(Variant, bool, const KCtx&, const TreeRange&, hipStream_t) { return hipSuccess; }
hipError_t launch_step2(Variant, bool, int64_t, const KCtx&, int, const DevStep&, int, const DevStep&, hipStream_t) {
  return hipSuccess;
}
hipError_t launch_persistent(Variant, bool, const KCtx&, int, hipStream_t) { return hipSuccess; }
hipError_t launch_dataflow(Variant, bool, const KCtx&, bool, int, hipStream_t) { return hipSuccess; }
hipError_t persistent_capacity(Variant, bool, int* blocks) {
  *blocks = 1024;
  return hipSuccess;
}
// The no-allocation entry point's array does not exist in a host build: its
// lookup fails, so a valid call stops with PAT_ERR_HIP before any copy.
size_t scratch_bytes() { return size_t(256) << 20; }
hipError_t scratch_base(int, char**) { return hipErrorNotSupported; }

}  // namespace pat
