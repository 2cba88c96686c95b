// Internal definitions of the projected-KV cache builder (kernels and host API).
//
// Sec. 3.2 (linear projection of the L_s sampled layers' KV, optional RoPE on
// the projected key): k' = W_K [k^(1); ...; k^(L_s)], v' = W_V [v^(1); ...],
// one GEMM per tensor with the reduction running over L_s d_kv inputs that are
// gathered from paged caches.
#pragma once

#include "kvshot_common.h"

namespace kvshot {

constexpr int kProjTile = 256;        // output channels and tokens per workgroup
constexpr int kProjMaxLayers = 4;
constexpr int kProjMaxSplits = 16;
constexpr int kProjWorkspaceRows = 8192;   // (split, token) rows of 2 d_kv floats
constexpr int kProjDirectMaxTile16 = 4;  // direct kernel: at most 64 tokens per tile

struct KvProjParams {
  const uint16_t* k_src[kProjMaxLayers];   // source K pools, stacking order
  const uint16_t* v_src[kProjMaxLayers];
  const uint16_t* w_k;                     // [d_kv][L d_kv] bf16
  const uint16_t* w_v;
  uint16_t* k_dst;
  uint16_t* v_dst;
  const int32_t* page_table;               // [batch][max_pages_per_seq]
  const int32_t* dst_page_table;
  const int32_t* token_seq;                // [n_tokens]
  const int32_t* token_pos;
  const float2* rope;                      // [max_position][64] (cos, sin)
  const double* rope_rev;                  // [64]: theta^(-2m/128) / (2 pi), revolutions per position
  float* part;                             // [splits][n_tokens][2 d_kv] (split plans only)
  int64_t page_stride, head_stride, slot_stride;
  int64_t dst_page_stride, dst_head_stride, dst_slot_stride;
  int32_t n_tokens, batch, hkv, layers;
  int32_t page_shift, max_pages_per_seq, num_pages, dst_num_pages, max_position;
  int32_t m_tiles;                         // channel tiles: ceil(Hkv / 2)
  int32_t n_tiles;                         // token tiles: ceil(n_tokens / 256), direct kernel ceil(n_tokens / (16 tile16))
  int32_t splits, work_items, rope_keys;
  int32_t tile16;                          // direct kernel: tokens per tile / 16 (1 .. kProjDirectMaxTile16)
};

hipError_t launch_kvproj(const KvProjParams& p, hipStream_t s);
hipError_t launch_kvproj_combine(const KvProjParams& p, hipStream_t s);
hipError_t launch_kvproj_direct(const KvProjParams& p, hipStream_t s);
hipError_t launch_kvproj_validate(const KvProjParams& p, int32_t* flag, hipStream_t s);

}  // namespace kvshot
