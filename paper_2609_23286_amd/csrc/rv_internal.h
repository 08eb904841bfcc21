// rv_internal.h -- shared between librv's host code and its gfx950 kernels (not installed):
// the argument blocks and plans of rv_plan.h, and the kernel launchers.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "rv_plan.h"

namespace rv {

hipError_t launch_attention(const AttnArgs& a, int grid, bool merge, hipStream_t s);
// The attention launch with the saliency in its epilogue: the forward launch, then one
// merge workgroup per unit that forms the unit's outputs and LSE (when its key range was
// split) and then the unit's row of per-block saliency (SalEpi).
hipError_t launch_attention_saliency(const AttnArgs& a, const SalEpi& e, int grid, hipStream_t s);
// Device address, on the current device, of the library's static partial-slot array
// (kStaticScratchSlots slots of kAttnSlotFloats floats).
hipError_t static_scratch_address(float** ptr);
// Copies a frame's K, V ([n][H][64] bf16) to staged arena rows: row j of head h goes to
// dK / dV + (h * head_stride + j) * 64.
hipError_t launch_stage(uint16_t* dK, uint16_t* dV, int64_t head_stride, const uint16_t* K, const uint16_t* V,
                        int n, int H, hipStream_t s);
// The same for a.n_layers layers' frames in one launch.
hipError_t launch_stage_layers(const StageArgs& a, hipStream_t s);
// Records the hardware XCC id of each of n_blocks workgroups into ids (device memory).
hipError_t launch_xcc_probe(int* ids, int n_blocks, hipStream_t s);
// max_lds: the device's LDS limit per workgroup (bytes), for the kernel attribute.
hipError_t launch_admit(const AdmitArgs& a, int max_lds, hipStream_t s);

}  // namespace rv
