// Launchers of the measurement aids (csrc/ceiling.hip); the optional (e0, e1)
// events are attached to the launch itself.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>

namespace parrot {

// Read-bandwidth probe: every 16-byte piece of src read once (nontemporal),
// `unroll` loads in flight per thread, in grid-stride order or one
// contiguous span per wave (`spans`), XOR-folded into *sink.
hipError_t launch_read_ceiling(const void* src, size_t bytes, unsigned* sink, int workgroups,
                               int unroll, bool spans, hipStream_t s, hipEvent_t e0, hipEvent_t e1);
// Matrix-core issue probe: `iters` iterations of eight 16x16x32 f16 MFMAs per
// wave with vx4 / 4 vector instructions per MFMA (vx4 in {0, 8, 10, 11, 12, 16}).
hipError_t launch_mfma_issue(unsigned* sink, int workgroups, int iters, int vx4, hipStream_t s,
                             hipEvent_t e0, hipEvent_t e1);

}  // namespace parrot
