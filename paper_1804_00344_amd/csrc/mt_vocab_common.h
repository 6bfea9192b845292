// Definitions shared by the vocabulary projection kernels (single model and fused ensemble):
// tile and list sizes, the wave shape of a workgroup, and the k-step of each operand type.
#pragma once
#include "mt_internal.h"

namespace mt {

typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;
typedef uint32_t v4u __attribute__((ext_vector_type(4)));

constexpr int kVRows = 64;       // vocabulary rows per wave tile (2 MFMA blocks)
constexpr int kLists = 8;        // candidate buffers per (hypothesis, chunk): 2 lane halves x 4 runs
constexpr int kSampleMax = 2048;  // vocabulary entries of the threshold pass
constexpr float kLog2e = 1.4426950408889634f;

// Hypothesis columns per wave: at most 64 (two 32-column MFMA blocks); a workgroup of HB
// columns runs HB/64 waves per vocabulary run on the same tiles.
template <typename CT, int HB>
struct VShape {
  static constexpr int WH = HB >= 64 ? 64 : HB;  // columns per wave
  static constexpr int HBW = WH / 32;            // 32-column MFMA blocks per wave
  static constexpr int NW = 4 * (HB / WH);       // waves per workgroup
  static constexpr int NT = 64 * NW;             // threads per workgroup
};

template <typename CT>
struct VCfg;
template <>
struct VCfg<bf16> {
  static constexpr int KV = 16;  // k per 16-byte vector step
};
template <>
struct VCfg<float> {
  static constexpr int KV = 8;
};

}  // namespace mt
