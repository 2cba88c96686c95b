// Internal definitions of the gated delta fusion (kernels and host API).
//
// Sec. 3.4.1, Eqs. (delta), (fusion): Delta = o - n,
// g = sigmoid(W_g [n; o; Delta] + b_g), h = n + g * (W_Delta Delta).  The
// reduction runs over four segments of length d: n, o and Delta against the
// three column blocks of W_g (gate), and Delta against W_Delta.
#pragma once

#include "kvshot_common.h"

namespace kvshot {

constexpr int kFusionTokens = 64;     // tokens per fusion workgroup (128 with the large-call tile)
constexpr int kFusionChannels = 128;  // output channels per fusion workgroup
constexpr int kFusionMaxSplits = 16;

struct FusionParams {
  const uint16_t* n;            // [tokens][d] bf16
  const uint16_t* o;            // [tokens][d] bf16
  const uint16_t* w_g;          // [d][3d] bf16, row c = output channel c over [n | o | Delta]
  const float* b_g;             // [d]
  const uint16_t* w_delta;      // [d][d] bf16
  const uint16_t* w_packed;     // both weight matrices in the kernel's operand order (packed path) or null
  void* h;                      // [tokens][d] bf16 or float32
  float* g_out;                 // [tokens][d] or null
  float* part;                  // [splits][2][tokens][d]: per split, a gate plane and a delta-projection plane
  uint32_t part_g_mask;         // bit s: split s contributes to the gate (writes its gate plane)
  uint32_t part_d_mask;         // bit s: split s contributes to the delta projection
  int32_t tokens, d;
  int32_t m_tiles, n_tiles, splits;
  int32_t kparts;               // reduction-index parts of a segment: splits / (segment groups)
  int32_t tile_tokens;          // tokens per workgroup tile: 64 or 128
  int32_t cross_only, out_fp32;
};

hipError_t launch_fusion(const FusionParams& p, hipStream_t s);
hipError_t launch_fusion_combine(const FusionParams& p, hipStream_t s);
hipError_t launch_fusion_pack(const uint16_t* w_g, const uint16_t* w_delta, uint16_t* packed, int d, hipStream_t s);

}  // namespace kvshot
