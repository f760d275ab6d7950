// Tile shape of the prefill kernel, shared by the kernel and the host sizing.
#pragma once

namespace parrot {

// fp16 / bf16 caches: 4 waves, each with kWideSets column sets of 16 query
// rows (fp32 caches use decode's 64-row tile).
constexpr int kWideSets = 2;
constexpr int kWideRows = 4 * 16 * kWideSets;

}  // namespace parrot
