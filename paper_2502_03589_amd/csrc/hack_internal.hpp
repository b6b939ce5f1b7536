// Launchers shared between the C-ABI layer (hack_api.hip) and the kernel files.
#pragma once

#include <hip/hip_runtime.h>
#include <hip/hip_fp16.h>
#include <stdint.h>

#include "../../include/hack.h"
#include "hack_device.hpp"

namespace hack {

// Decode split plan: tokens per workgroup (a multiple of 4*partition) and the
// number of splits of the longest sequence.  Depends only on the sizes, so the
// workspace query and the attend call always agree.
// Workspace layout: the chunk counters first, at offset 0, one int32 per
// (sequence, kv head, head group), padded to 256 bytes; the chunk records after them.
// The counters' place depends only on batch, H_kv and the group size, so a call with a
// different max_len (hence a different split count) never lands its counters on an
// earlier call's records.
struct DecodePlan {
  int chunk;
  int splits;
  int head_groups;          // workgroups per (sequence, kv head, chunk)
  int64_t partial_floats;   // batch * H_kv * splits * G * (4 + head_dim)
  int64_t counter_bytes;    // batch * H_kv * head_groups int32 counters, padded to 256 bytes
  int64_t record_offset;    // byte offset of the chunk records (= counter_bytes)
  int64_t workspace_bytes;
};

// Fills the layout fields of a plan from its chunk/split choice.
inline void finish_plan(DecodePlan& p, int64_t pairs, int64_t group, int64_t head_groups, int64_t head_dim) {
  p.head_groups = (int)head_groups;
  p.partial_floats = pairs * p.splits * group * (4 + head_dim);
  p.counter_bytes = ((pairs * head_groups * 4 + 255) / 256) * 256;
  p.record_offset = p.counter_bytes;
  p.workspace_bytes = p.record_offset + ((p.partial_floats * 4 + 255) / 256) * 256;
}

DecodePlan plan_decode(const hack_kv_layout& lay, int batch, int num_q_heads, int max_len);
DecodePlan plan_decode128(const hack_kv_layout& lay, int batch, int num_q_heads, int max_len);

hipError_t launch_quantize(const hack_kv_layout& lay, const CacheView& c, const __half* k,
                           const __half* v, const int32_t* lens, int batch, int max_len,
                           hipStream_t stream);

hipError_t launch_append(const hack_kv_layout& lay, const CacheView& c, const __half* k_new,
                         const __half* v_new, int32_t* lens, int batch, int capacity,
                         int tail_mode, hipStream_t stream);

enum DecodeMode { MODE_ATTEND = 0, MODE_QK = 1, MODE_PV = 2 };

struct DecodeArgs {
  CacheView c;
  const __half* q;        // [B][H_q][128]
  const int32_t* lens;    // [B]
  float* out;             // [B][H_q][128]
  float* partials;        // [B][H_kv][splits][G][4 + 128]: max, sum, pad, O
  int32_t* counters;      // [B][H_kv] chunks finished (zero between calls)
  int num_q_heads;
  int group;              // H_q / H_kv
  int head_groups;        // workgroups per (sequence, kv head, chunk), each for up to 4*GT heads
  int chunk;
  int splits;
  int tail_requant;       // open V block mode: 0 fp16, 1 / 2 its codes (re-quantized from fp16 / from codes)
  int max_len;
  float qmax;             // 2^b_QP - 1 of the transient Q and P codes (15 or 255)
  float inv_qmax;         // 1 / qmax
  int qoff;               // Q/P codes enter the signed int8 MFMA as code - qoff, qoff = 2^(b_QP - 1)
  float qoff_f;
  // fused append (hack_decode_step): when k_new is set, token lens[s] of every
  // (sequence, kv head) is appended first, the attention covers lens[s] + 1 tokens
  // and lens_out[s] = lens[s] + 1
  const __half* k_new;    // [B][H_kv][128]
  const __half* v_new;    // [B][H_kv][128]
  int32_t* lens_out;      // [B]
  int capacity;
  int stochastic;
  uint64_t key_k, key_v;
  uint64_t key_q, key_p;  // stochastic rounding of the Q and P codes (streams 3 and 4)
  // test exports
  uint8_t* dbg_qcodes;    // [B][H_q][128]
  float* dbg_qmeta;       // [B][H_q][P][2]
  int32_t* dbg_prod;      // QK: [B][H_q][max_len][P]; PV: [B][H_q][NB][128]
  const uint8_t* dbg_pcodes;  // [B][H_q][NB][PI]
  const float* dbg_pmeta;     // [B][H_q][NB][2]
};

hipError_t launch_decode(const hack_kv_layout& lay, const DecodeArgs& a, int batch, int mode,
                         hipStream_t stream);

// Decode attention (MODE_ATTEND) for partition 128: VALU int8-dot kernel.
hipError_t launch_decode128(const hack_kv_layout& lay, const DecodeArgs& a, int batch, hipStream_t stream);

// QKV generation fused with quantize-on-write (kernels_project.hip).
struct ProjectArgs {
  CacheView c;
  const __half* e;    // [batch][len][hidden] embeddings
  const __half* w;    // [(H_q + 2 H_kv) * 128][hidden] weights, one row per output channel
  __half* q;          // [batch][H_q][len][128] query heads out
  int batch, len, hidden, q_heads, kv_heads;
  // filled by launch_project
  int mtiles;         // 256-token tiles per sequence
  int nheads;         // output heads: H_q + 2 H_kv
  int ntiles;         // channel tiles of two heads: ceil(nheads / 2)
  int64_t total;      // batch * mtiles * ntiles
  int stochastic;
  uint64_t key_k, key_v;
};

hipError_t launch_project(const hack_kv_layout& lay, const ProjectArgs& a, hipStream_t stream);

hipError_t launch_prefill(const hack_kv_layout& lay, const CacheView& c, const __half* q,
                          int num_q_heads, int batch, int len, int causal, float* out,
                          hipStream_t stream);

}  // namespace hack
