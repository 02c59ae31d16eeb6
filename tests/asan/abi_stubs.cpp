// Host-only stand-ins for the kernel launchers and the two HIP runtime calls that the C-ABI
// layer (fs_api.cpp) makes, so that its validation can be built with the address and
// undefined-behaviour sanitizers and run on a machine without a GPU. Every launcher reports
// hipErrorNoDevice, which the ABI must turn into FS_ERR_HIP.
#include <hip/hip_runtime_api.h>

#include "../../paper_2609_32525_amd/csrc/fs_internal.h"

namespace fs {

hipError_t launch_slice(const Geom&, const void*, const void*, const float*, const float*,
                        const float*, float*, float*, float*, char*, hipStream_t) {
  return hipErrorNoDevice;
}
hipError_t launch_deslice(const Geom&, const void*, const float*, const float*, const float*,
                          const float*, const float*, float*, void*, hipStream_t) {
  return hipErrorNoDevice;
}
hipError_t launch_mix(const Geom&, const MixArgs&, const float*, float*, float*, hipStream_t) {
  return hipErrorNoDevice;
}
hipError_t launch_mix_bwd(const Geom&, const MixArgs&, const float*, const float*, const float*,
                          const float*, const float*, float*, float*, float*, float*, float*,
                          float*, float*, bool, hipStream_t) {
  return hipErrorNoDevice;
}
hipError_t launch_bwd(const Geom&, const MixArgs&, const void*, const void*, const float*,
                      const float*, const float*, const float*, const float*, const float*,
                      const float*, const float*, const void*, void*, void*, float*, float*,
                      float*, float*, float*, char*, hipStream_t, const UntiedArgs*,
                      const float*) {
  return hipErrorNoDevice;
}
hipError_t launch_linearno_slice(const Geom&, const void*, const void*, const float*,
                                 const float*, const float*, float*, float*, char*, hipStream_t) {
  return hipErrorNoDevice;
}
hipError_t static_scratch(int, void**) { return hipErrorNoDevice; }
// sizes only enter the workspace totals; any fixed values keep the ABI self-consistent
size_t point_image_bytes(const Geom& g) { return (size_t)g.BH() * g.G * 64; }
size_t stat_image_bytes(const Geom& g) { return g.D == 64 ? (size_t)g.BH() * g.G * 32 : 0; }
bool attn_rows(const Geom& g, int kind) { return kind == 3 && g.G > 256; }

}  // namespace fs

extern "C" {
hipError_t hipGetDevice(int* d) {
  if (d) *d = 0;
  return hipErrorNoDevice;
}
hipError_t hipStreamGetDevice(hipStream_t, hipDevice_t* d) {
  if (d) *d = 0;
  return hipErrorNoDevice;
}
}
