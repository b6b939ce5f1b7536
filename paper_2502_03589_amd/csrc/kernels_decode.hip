// Decode attention on quantized K/V (Sec. 5.3 with L_Q = 1; Eq. 2-4).
//
// Work split: one workgroup of four 64-lane wavefronts per (sequence, kv head,
// chunk of the context); wave w takes spans w, w+4, ... of the chunk, where a span
// is four V blocks (4*PI tokens).  Every global load of a span is issued before
// any of its arithmetic.  Per span a wave computes, for up to 4 query heads of
// the kv group per row tile:
//   Q'K'  v_mfma_i32_16x16x64_i8: A = 8-bit Q codes (minus 128), rows = (channel
//         quarter q, head h), block-diagonal so that lane group g only carries
//         quarter g; B = 2/4-bit K codes unpacked in registers (lane = token,
//         group = quarter).  Lane (t, g) receives the products of quarter g for the
//         4 heads.
//   Eq. 4 the rank-1 terms (m~_q * s_k sum k' and R_q * m_k) come from two
//         v_mfma_f32_16x16x4_f32 (block-diagonal A of Q constants, B = the lane's
//         own K partition metadata); the product term s_q s_k C~ is on the VALU.
//         A permlane reduce-scatter sums the quarters so that lane (t, g) holds the
//         score of head g (log2 units).
//   softmax online with a lazily raised reference max; P quantized to 8 bits per
//         V block (min, scale, round-to-nearest-even codes), staged through LDS.
//   P'V'  v_mfma_i32_16x16x64_i8: A = P codes, rows = (block, head) block-diagonal
//         over the span's 4 blocks; B = V codes of 16 channels (lane = channel,
//         group = block).  One more MFMA with an all-ones B gives the P code sums.
//         Eq. 4 with the cached V sums: the product term on the VALU, the rank-1
//         terms through two v_mfma_f32_16x16x4_f32 accumulating into O.
//   open block  fp16 values times unquantized probabilities (TAIL_FP16), or its
//         re-quantized codes with n = T (TAIL_REQUANT).
// The four waves merge in LDS; when a sequence spans several chunks, each chunk's
// partial (max, sum, O) goes to the workspace and a second, small kernel merges them.
#include <type_traits>

#include "hack_internal.hpp"

namespace hack {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef float v4f __attribute__((ext_vector_type(4)));

// Operand byte position (4*register + byte) -> element offset within a 16-element
// slice, for the in-register unpack of 16 codes (b = 2: one dword; b = 4: two).
template <int BITS>
__device__ __forceinline__ constexpr int perm_offset(int bp) {
  return BITS == 2 ? 4 * (bp & 3) + (bp >> 2) : 8 * (bp >> 3) + 2 * (bp & 3) + ((bp >> 2) & 1);
}
// Inverse of perm_offset.
template <int BITS>
__device__ __forceinline__ constexpr int perm_position(int e) {
  return BITS == 2 ? 4 * (e & 3) + (e >> 2) : 8 * (e >> 3) + 4 * (e & 1) + ((e & 7) >> 1);
}

// 16 packed codes -> 16 int8 lanes of an MFMA operand (byte order per perm_offset).
template <int BITS>
__device__ __forceinline__ v4i unpack16(const uint32_t* w) {
  if constexpr (BITS == 2) {
    const uint32_t x = w[0];
    return v4i{(int)(x & 0x03030303u), (int)((x >> 2) & 0x03030303u), (int)((x >> 4) & 0x03030303u),
               (int)((x >> 6) & 0x03030303u)};
  } else {
    const uint32_t x = w[0], y = w[1];
    return v4i{(int)(x & 0x0F0F0F0Fu), (int)((x >> 4) & 0x0F0F0F0Fu), (int)(y & 0x0F0F0F0Fu),
               (int)((y >> 4) & 0x0F0F0F0Fu)};
  }
}

// N dwords from a 4*N-byte aligned address, as wide as the count allows.
template <int N>
__device__ __forceinline__ void load_words(const uint8_t* p, uint32_t* w) {
  if constexpr (N % 4 == 0) {
#pragma unroll
    for (int i = 0; i < N / 4; ++i) {
      const uint4 v = reinterpret_cast<const uint4*>(p)[i];
      w[4 * i] = v.x; w[4 * i + 1] = v.y; w[4 * i + 2] = v.z; w[4 * i + 3] = v.w;
    }
  } else if constexpr (N == 2) {
    const uint2 v = *reinterpret_cast<const uint2*>(p);
    w[0] = v.x; w[1] = v.y;
  } else {
#pragma unroll
    for (int i = 0; i < N; ++i) w[i] = reinterpret_cast<const uint32_t*>(p)[i];
  }
}

__device__ __forceinline__ v4i mfma_i8(v4i a, v4i b, v4i c) {
  return __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ v4f mfma_f32(float a, float b, v4f c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ float lo_half(uint32_t w) { return __half2float(__ushort_as_half((uint16_t)(w & 0xFFFFu))); }
__device__ __forceinline__ float hi_half(uint32_t w) { return __half2float(__ushort_as_half((uint16_t)(w >> 16))); }

// Sum four per-quarter partial values over the four lane groups so that lane
// group g ends with the total of value g (permlane swaps across 32 and 16 lanes).
__device__ __forceinline__ float reduce_scatter4(float v0, float v1, float v2, float v3) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(v0), __float_as_uint(v2), false, false);
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v1), __float_as_uint(v3), false, false);
  const float x = __uint_as_float(a[0]) + __uint_as_float(a[1]);  // groups 0,1: value 0; 2,3: value 2
  const float y = __uint_as_float(b[0]) + __uint_as_float(b[1]);  // groups 0,1: value 1; 2,3: value 3
  const auto c = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(y), false, false);
  return __uint_as_float(c[0]) + __uint_as_float(c[1]);
}

__device__ __forceinline__ float pick4(const float (&v)[4], int i) {
  return i == 0 ? v[0] : (i == 1 ? v[1] : (i == 2 ? v[2] : v[3]));
}

// 1/sqrt(128) * log2(e): scores are kept in log2 units so softmax uses exp2.
constexpr float kScoreScale = 0.12751743074941640f;
// The reference max of the online softmax is raised only when a block's max
// exceeds it by more than this (p~ <= 2^8 in between).
constexpr float kMaxSlack = 8.0f;

constexpr int kWaves = 4;

#ifndef HACK_DECODE_PREFETCH
#define HACK_DECODE_PREFETCH 0
#endif
#ifndef HACK_DECODE_WAVES_PER_SIMD
#define HACK_DECODE_WAVES_PER_SIMD 2
#endif
#ifndef HACK_DECODE_TARGET_WGS
#define HACK_DECODE_TARGET_WGS 512
#endif

// Cache addresses of the four V blocks of a span (wave-uniform): the row of each
// block's first token in the K sections and the block's index in the V sections.
struct SpanAddr {
  int64_t krow[4];
  int64_t vblk[4];
};

template <int PI>
__device__ __forceinline__ void span_addresses(const CacheView& c, int s, int hkv, int span0, int L,
                                               SpanAddr& ad) {
  const int bpp = c.page_tokens / PI;  // blocks per page
  const int kb0 = span0 / PI;
  int pidx = 0, slot = kb0;
  if (c.block_table) {
    pidx = kb0 / bpp;
    slot = kb0 - pidx * bpp;
  }
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    int64_t page = 0;
    if (span0 + k * PI < L) {
      if (c.block_table) {
        int64_t pg = c.block_table[(int64_t)s * c.mbps + pidx];
        page = pg < 0 ? 0 : (pg >= c.num_pages ? c.num_pages - 1 : pg);
      } else {
        page = s < c.num_pages ? s : c.num_pages - 1;
      }
    }
    ad.krow[k] = (page * c.kv_heads + hkv) * c.page_tokens + (int64_t)slot * PI;
    ad.vblk[k] = (page * c.kv_heads + hkv) * bpp + slot;
    if (++slot == bpp && c.block_table) {
      slot = 0;
      ++pidx;
    }
  }
}

// Register copy of one span's compressed data for one lane.
template <int BITS, int PI>
struct SpanData {
  static constexpr int NT = PI / 4;              // 16-token tiles per span
  static constexpr int KW = BITS;                // K dwords per (token, quarter)
  static constexpr int VW = PI * BITS / 32;      // V dwords per (channel, block)
  uint32_t kc[NT][KW];  // K codes of the lane's token and channel quarter, per tile
  uint32_t km[NT];      // (m_k, s_k) of the lane's K partition, per tile
  uint32_t kz[NT];      // cached code sum of that partition, per tile
  uint32_t vc[8 * VW];  // V codes of 8 channels of the lane's block
  uint32_t vm[8];       // (m_v, s_v) of those channels
  uint32_t vz[8];       // cached V code sums
};

// LDS of one wave.
template <int PI, int GT>
struct WaveLds {
  int8_t p[GT][4][4][PI];       // P codes - 128: [row tile][block][head][token position]
  float pst[GT][4][2][4];       // [rt][block][s_p | m~_p][head], scaled to the span's reference max
  float alpha[GT][4];           // O rescale of the span, per head
  float tailf[GT][4];           // scale of the fp16 open block's probabilities
  float ptail[GT][4][PI];       // unquantized p~ of the open block
};

template <int BITS, int PI, int GT, int MODE>
__global__ __launch_bounds__(256, HACK_DECODE_WAVES_PER_SIMD) void decode_kernel(DecodeArgs a) {
  constexpr int D = 128;
  constexpr int P = D / PI;          // K partitions per token
  constexpr int QPP = 4 / P;         // channel quarters per partition
  constexpr int TILES = PI / 16;     // 16-token tiles per V block
  constexpr int SPAN = 4 * PI;
  constexpr int NT = 4 * TILES;      // token tiles per span
  constexpr int KW = BITS;           // K code dwords per (token, quarter of 32 channels)
  constexpr int VW = PI * BITS / 32; // V code dwords per (channel, block)
  constexpr int SW = BITS / 2;       // dwords per 16-code slice
  constexpr int HT = GT * 4;

  __shared__ int8_t q_lds[HT][D];
  __shared__ float qm_lds[HT][4][3];
  __shared__ __attribute__((aligned(16))) WaveLds<PI, GT> wl_all[kWaves];
  __shared__ float mrg_o[kWaves][HT][D];
  __shared__ float mrg_ml[kWaves][HT][2];

  const CacheView& c = a.c;
  const int tid = threadIdx.x;
  // wave index made explicitly wave-uniform so span bookkeeping stays in scalar registers
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const int col = lane & 15, grp = lane >> 4;
  const int s = blockIdx.z, hkv = blockIdx.y, split = blockIdx.x;
  const int G = a.group, Hq = a.num_q_heads, H = c.kv_heads;
  // lengths outside [0, max_len] break the caller contract; clamp so that every
  // access stays inside the cache and the workspace
  const int L = max(0, min(a.lens[s], a.max_len));
  const int t0 = split * a.chunk;
  if (t0 >= L) {
    if (MODE == MODE_ATTEND && split == 0) {  // empty sequence: zeros
      for (int i = tid; i < G * D; i += 256) a.out[((int64_t)s * Hq + hkv * G) * D + i] = 0.0f;
    }
    return;
  }
  const int t1 = min(L, t0 + a.chunk);
  const int nsplit = (L + a.chunk - 1) / a.chunk;
  const int F = L / PI, T = L - F * PI;
  const bool requant = a.tail_requant != 0;
  WaveLds<PI, GT>& wl = wl_all[wave];

  // ---- Q: 8-bit codes per partition with float32 metadata (Sec. 5.1, Sec. 5.2) ----
  // wave w quantizes head slots w, w+4, ...; each lane holds two channels
  if constexpr (MODE != MODE_PV) {
    for (int gh = wave; gh < HT; gh += kWaves) {
      const bool real = gh < G;
      const int hq = hkv * G + gh;
      float x0 = 0.0f, x1 = 0.0f;
      if (real) {
        const float2 f = __half22float2(reinterpret_cast<const __half2*>(a.q + ((int64_t)s * Hq + hq) * D)[lane]);
        x0 = f.x;
        x1 = f.y;
      }
      float mn = fminf(x0, x1), mx = fmaxf(x0, x1);
#pragma unroll
      for (int m = 1; m < PI / 2; m <<= 1) {
        mn = fminf(mn, __shfl_xor(mn, m, 64));
        mx = fmaxf(mx, __shfl_xor(mx, m, 64));
      }
      float sq, c0 = 0.0f, c1 = 0.0f;
      {
#pragma clang fp contract(off)
        sq = __fdiv_rn(__fsub_rn(mx, mn), 255.0f);
        if (sq != 0.0f) {
          const float r = __fdiv_rn(1.0f, sq);
          c0 = fminf(rintf(__fmul_rn(__fsub_rn(x0, mn), r)), 255.0f);
          c1 = fminf(rintf(__fmul_rn(__fsub_rn(x1, mn), r)), 255.0f);
        }
      }
      int csum = (int)c0 + (int)c1;
#pragma unroll
      for (int m = 1; m < PI / 2; m <<= 1) csum += __shfl_xor(csum, m, 64);
      q_lds[gh][2 * lane] = real ? (int8_t)((int)c0 - 128) : (int8_t)0;
      q_lds[gh][2 * lane + 1] = real ? (int8_t)((int)c1 - 128) : (int8_t)0;
      const int p = (2 * lane) / PI;
      if ((2 * lane) % PI == 0) {
        // per partition: s_q, m~_q = m_q + 128 s_q, R = s_q sum q' + n m_q (all in log2 units)
        qm_lds[gh][p][0] = real ? kScoreScale * sq : 0.0f;
        qm_lds[gh][p][1] = real ? kScoreScale * (mn + 128.0f * sq) : 0.0f;
        qm_lds[gh][p][2] = real ? kScoreScale * (sq * (float)csum + (float)PI * mn) : 0.0f;
        if (MODE == MODE_QK && real && split == 0) {
          a.dbg_qmeta[(((int64_t)s * Hq + hq) * P + p) * 2 + 0] = mn;
          a.dbg_qmeta[(((int64_t)s * Hq + hq) * P + p) * 2 + 1] = sq;
        }
      }
      if (MODE == MODE_QK && real && split == 0) {
        a.dbg_qcodes[((int64_t)s * Hq + hq) * D + 2 * lane] = (uint8_t)c0;
        a.dbg_qcodes[((int64_t)s * Hq + hq) * D + 2 * lane + 1] = (uint8_t)c1;
      }
    }
  }
  __syncthreads();

  // Q operands.  Rows of the QK tile are (quarter q, head h) = 4q + h; lane (row, group g)
  // is non-zero only for q == g.  qa: int8 codes; ra: the rank-1 coefficients of Eq. 4
  // (m~_q and R, divided among the QPP quarters of a partition); sq_: s_q of the lane's
  // quarter for head i, used by the product term.
  v4i qa[GT][2];
  float ra[GT][2];
  float sq_[GT][4];
  const int pl = grp / QPP;  // partition of this lane's quarter
  if constexpr (MODE != MODE_PV) {
    const int qq = col >> 2, hh = col & 3;
#pragma unroll
    for (int rt = 0; rt < GT; ++rt) {
#pragma unroll
      for (int m = 0; m < 2; ++m) {
        int b4[4] = {0, 0, 0, 0};
        if (qq == grp) {
#pragma unroll
          for (int bp = 0; bp < 16; ++bp) {
            const int v = (int)(uint8_t)q_lds[rt * 4 + hh][32 * grp + 16 * m + perm_offset<BITS>(bp)];
            b4[bp >> 2] |= v << (8 * (bp & 3));
          }
        }
        qa[rt][m] = v4i{b4[0], b4[1], b4[2], b4[3]};
      }
      constexpr float inv_qpp = 1.0f / (float)QPP;
      ra[rt][0] = qq == grp ? qm_lds[rt * 4 + hh][pl][1] * inv_qpp : 0.0f;
      ra[rt][1] = qq == grp ? qm_lds[rt * 4 + hh][pl][2] * inv_qpp : 0.0f;
#pragma unroll
      for (int i = 0; i < 4; ++i) sq_[rt][i] = qm_lds[rt * 4 + i][pl][0];
    }
  }

  float m_ref[GT], l_run[GT];
  v4f o_acc[GT][8];  // PV layout: lane (channel col, group k) rows (k, head i); summed over k at the end
#pragma unroll
  for (int rt = 0; rt < GT; ++rt) {
    m_ref[rt] = -INFINITY;
    l_run[rt] = 0.0f;
#pragma unroll
    for (int j = 0; j < 8; ++j) o_acc[rt][j] = v4f{0.0f, 0.0f, 0.0f, 0.0f};
  }

  const int nspan = (t1 - t0 + SPAN - 1) / SPAN;
  const uint32_t k_lane_off = (uint32_t)(col * (D * BITS / 8) + grp * (32 * BITS / 8));

  // Full spans (every token valid, every block quantized) are software-pipelined:
  // the loads of a wave's next span are in flight while it computes the current one.
  // At most one span per chunk, its last, is partial; it takes the masked path.
  const int nspan_full = max(0, min(nspan, (F * PI - t0) / SPAN));
  auto load_span = [&](SpanData<BITS, PI>& d, int span0, auto masked_tag) __attribute__((always_inline)) {
    constexpr bool MASKED = decltype(masked_tag)::value;
    constexpr bool full = !MASKED;
    SpanAddr ad;
    span_addresses<PI>(c, s, hkv, span0, L, ad);
    // ---------------- global loads of the whole span ----------------
#pragma unroll
    for (int ti = 0; ti < NT; ++ti) {
      const int tb = span0 + 16 * ti;  // first token of the tile (wave-uniform)
      const int64_t row0 = ad.krow[ti / TILES] + 16 * (ti % TILES);
      if (full || tb + col < L) {
        load_words<KW>(c.k_codes + row0 * (D * BITS / 8) + k_lane_off, d.kc[ti]);
        const uint32_t mi = (uint32_t)(col * P + pl);
        d.km[ti] = reinterpret_cast<const uint32_t*>(c.k_meta)[row0 * P + mi];
        d.kz[ti] = load_sum(c.k_sums + row0 * P * c.sum_bytes, mi, c.sum_bytes);
      } else {
#pragma unroll
        for (int w = 0; w < KW; ++w) d.kc[ti][w] = 0u;
        d.km[ti] = 0u;
        d.kz[ti] = 0u;
      }
    }
    // V of this lane's block (group g = block g of the span), channels 8*col .. 8*col+7
    const int vbt0 = span0 + grp * PI;
    const int vkb = vbt0 / PI;
    bool gvalid = full || (vbt0 < L && (vkb < F || (requant && vkb == F && T > 0)));
    if constexpr (MODE == MODE_PV) gvalid = vbt0 < L && vkb < F;
#pragma unroll
    for (int w = 0; w < 8 * VW; ++w) d.vc[w] = 0u;
#pragma unroll
    for (int j = 0; j < 8; ++j) d.vm[j] = d.vz[j] = 0u;
    if (gvalid) {
      const int64_t vb = grp == 0 ? ad.vblk[0] : (grp == 1 ? ad.vblk[1] : (grp == 2 ? ad.vblk[2] : ad.vblk[3]));
      load_words<8 * VW>(c.v_codes + (vb * D + 8 * col) * (PI * BITS / 8), d.vc);
      const uint4* mp = reinterpret_cast<const uint4*>(c.v_meta + vb * D + 8 * col);
      const uint4 m0 = mp[0], m1 = mp[1];
      d.vm[0] = m0.x; d.vm[1] = m0.y; d.vm[2] = m0.z; d.vm[3] = m0.w;
      d.vm[4] = m1.x; d.vm[5] = m1.y; d.vm[6] = m1.z; d.vm[7] = m1.w;
      if (c.sum_bytes == 1) {
        const uint2 z = *reinterpret_cast<const uint2*>(c.v_sums + vb * D + 8 * col);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          d.vz[j] = (z.x >> (8 * j)) & 0xFFu;
          d.vz[4 + j] = (z.y >> (8 * j)) & 0xFFu;
        }
      } else {
        const uint4 z = *reinterpret_cast<const uint4*>(reinterpret_cast<const uint16_t*>(c.v_sums) + vb * D + 8 * col);
        const uint32_t zz[4] = {z.x, z.y, z.z, z.w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          d.vz[2 * j] = zz[j] & 0xFFFFu;
          d.vz[2 * j + 1] = zz[j] >> 16;
        }
      }
    }
  };
  auto compute_span = [&](const SpanData<BITS, PI>& d, int span0, auto masked_tag) __attribute__((always_inline)) {
    constexpr bool MASKED = decltype(masked_tag)::value;
    constexpr bool full = !MASKED;
    // V of this lane's block (group g = block g of the span), channels 8*col .. 8*col+7
    const int vbt0 = span0 + grp * PI;
    const int vkb = vbt0 / PI;
    bool gvalid = full || (vbt0 < L && (vkb < F || (requant && vkb == F && T > 0)));
    if constexpr (MODE == MODE_PV) gvalid = vbt0 < L && vkb < F;
    // ---------------- Q'K', Eq. 4, softmax and P quantization ----------------
    float m_start[GT], m_blk[GT][4], ps_s[GT][4], ps_m[GT][4];
    int kF = -1;  // position of the fp16 open block in this span
#pragma unroll
    for (int rt = 0; rt < GT; ++rt) m_start[rt] = m_ref[rt];

#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int bt0 = span0 + k * PI;
      const int kb = bt0 / PI;
      const bool present = full || bt0 < L;
      const bool quantized = full || (present && (kb < F || requant));
      if (!full && present && kb == F && !requant) kF = k;
#pragma unroll
      for (int rt = 0; rt < GT; ++rt) {
        m_blk[rt][k] = m_ref[rt];
        ps_s[rt][k] = 0.0f;
        ps_m[rt][k] = 0.0f;
      }
      if constexpr (MODE == MODE_PV) {
        // injected P codes and metadata of full blocks
        const int NB = a.max_len / PI;
        for (int i = lane; i < GT * 4 * PI; i += 64) {
          const int rt = i / (4 * PI), hh = (i / PI) & 3, e = i % PI;
          const int gh = rt * 4 + hh;
          int8_t v = 0;
          if (present && kb < F && gh < G)
            v = (int8_t)((int)a.dbg_pcodes[(((int64_t)s * Hq + hkv * G + gh) * NB + kb) * PI + e] ^ 0x80);
          wl.p[rt][k][hh][(e >> 4) * 16 + perm_position<BITS>(e & 15)] = v;
        }
        if (lane < HT) {
          const int rt = lane >> 2, hh = lane & 3, gh = lane;
          float pm = 0.0f, ps = 0.0f;
          if (present && kb < F && gh < G) {
            const int64_t base = ((int64_t)s * Hq + hkv * G + gh) * NB + kb;
            pm = a.dbg_pmeta[base * 2 + 0];
            ps = a.dbg_pmeta[base * 2 + 1];
          }
          wl.pst[rt][k][0][hh] = ps;
          wl.pst[rt][k][1][hh] = pm + 128.0f * ps;
        }
        continue;
      } else {
        if (!present) {
          for (int i = lane; i < GT * PI; i += 64) reinterpret_cast<int*>(&wl.p[i / PI][k][0][0])[i % PI] = 0;
          continue;
        }
        float sv[GT][TILES];
#pragma unroll
        for (int tl = 0; tl < TILES; ++tl) {
          const int ti = k * TILES + tl;
          const v4i b0 = unpack16<BITS>(d.kc[ti]);
          const v4i b1 = unpack16<BITS>(d.kc[ti] + SW);
          // the lane's own K partition: m_k, s_k and the cached code sum
          const float mk = lo_half(d.km[ti]), skv = hi_half(d.km[ti]);
          const float bz = skv * (float)d.kz[ti];
#pragma unroll
          for (int rt = 0; rt < GT; ++rt) {
            v4i acc = v4i{0, 0, 0, 0};
            acc = mfma_i8(qa[rt][0], b0, acc);
            acc = mfma_i8(qa[rt][1], b1, acc);
            v4f rk = v4f{0.0f, 0.0f, 0.0f, 0.0f};
            rk = mfma_f32(ra[rt][0], bz, rk);   // m~_q * s_k * sum k'
            rk = mfma_f32(ra[rt][1], mk, rk);   // R_q * m_k
            float part[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) part[i] = fmaf(sq_[rt][i] * skv, (float)acc[i], rk[i]);
            if constexpr (MODE == MODE_QK) {
              // integer partition products (unsigned codes) for the test export
              int cp[4];
#pragma unroll
              for (int i = 0; i < 4; ++i) {
                int v = acc[i];
                if constexpr (QPP >= 2) v += __shfl_xor(v, 16, 64);
                if constexpr (QPP >= 4) v += __shfl_xor(v, 32, 64);
                cp[i] = v + 128 * (int)d.kz[ti];
              }
              const int tok = bt0 + 16 * tl + col;
              if (tok < L && grp % QPP == 0) {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                  const int gh = rt * 4 + i;
                  if (gh < G)
                    a.dbg_prod[(((int64_t)s * Hq + hkv * G + gh) * a.max_len + tok) * P + pl] = cp[i];
                }
              }
            }
            const float sc = reduce_scatter4(part[0], part[1], part[2], part[3]);
            sv[rt][tl] = (full || bt0 + 16 * tl + col < L) ? sc : -INFINITY;
          }
        }
        if constexpr (MODE == MODE_QK) continue;
#pragma unroll
        for (int rt = 0; rt < GT; ++rt) {
          float bmax = sv[rt][0];
#pragma unroll
          for (int tl = 1; tl < TILES; ++tl) bmax = fmaxf(bmax, sv[rt][tl]);
          bmax = row16_max(bmax);
          if (bmax > m_ref[rt] + kMaxSlack || m_ref[rt] == -INFINITY) {  // raise the reference max
            l_run[rt] *= __builtin_amdgcn_exp2f(m_ref[rt] - bmax);
            m_ref[rt] = bmax;
          }
          const float mr = m_ref[rt];
          m_blk[rt][k] = mr;
          float pt[TILES];
          float lsum = 0.0f;
#pragma unroll
          for (int tl = 0; tl < TILES; ++tl) {
            pt[tl] = __builtin_amdgcn_exp2f(sv[rt][tl] - mr);
            lsum += pt[tl];
          }
          l_run[rt] += lsum;
          if (quantized) {
            float bmin = (full || bt0 + col < L) ? sv[rt][0] : INFINITY;
#pragma unroll
            for (int tl = 1; tl < TILES; ++tl)
              bmin = fminf(bmin, (full || bt0 + 16 * tl + col < L) ? sv[rt][tl] : INFINITY);
            bmin = row16_min(bmin);
            const float pmax = __builtin_amdgcn_exp2f(bmax - mr);
            const float pmin = __builtin_amdgcn_exp2f(bmin - mr);
            const float dp = pmax - pmin;
            const float r = dp > 0.0f ? 255.0f * __builtin_amdgcn_rcpf(dp) : 0.0f;
            const float bias = -pmin * r;
#pragma unroll
            for (int tl = 0; tl < TILES; ++tl) {
              // round-to-nearest-even with saturation to [0, 255]
              const uint32_t code = __builtin_amdgcn_cvt_pk_u8_f32(fmaf(pt[tl], r, bias), 0, 0u);
              const bool valid = full || bt0 + 16 * tl + col < L;
              wl.p[rt][k][grp][tl * 16 + perm_position<BITS>(col)] = valid ? (int8_t)(code ^ 0x80u) : (int8_t)0;
            }
            ps_s[rt][k] = dp * (1.0f / 255.0f);
            ps_m[rt][k] = pmin;
          } else {
#pragma unroll
            for (int tl = 0; tl < TILES; ++tl) {
              wl.p[rt][k][grp][tl * 16 + perm_position<BITS>(col)] = 0;
              wl.ptail[rt][grp][tl * 16 + col] = pt[tl];
            }
          }
        }
      }
    }
    if constexpr (MODE == MODE_QK) return;

    if constexpr (MODE != MODE_PV) {
      if (col == 0) {
#pragma unroll
        for (int rt = 0; rt < GT; ++rt) {
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            const float f = __builtin_amdgcn_exp2f(m_blk[rt][k] - m_ref[rt]);
            wl.pst[rt][k][0][grp] = ps_s[rt][k] * f;
            wl.pst[rt][k][1][grp] = (ps_m[rt][k] + 128.0f * ps_s[rt][k]) * f;
            if (k == kF) wl.tailf[rt][grp] = f;
          }
          wl.alpha[rt][grp] = __builtin_amdgcn_exp2f(m_start[rt] - m_ref[rt]);
        }
      }
    }
    // LDS written above is read below by other lanes of this wave
    __builtin_amdgcn_s_waitcnt(0xC07F);
    __builtin_amdgcn_wave_barrier();

    // ---------------- P'V' and Eq. 4: lane (channel col, group = block k) ----------------
    {
      const float n_g = (float)(vkb < F ? PI : T);
      const int kk = col >> 2, hh = col & 3;
      v4i pa[GT][TILES];
      float sp_[GT][4];
      float pr1[GT], pr2[GT];
#pragma unroll
      for (int rt = 0; rt < GT; ++rt) {
#pragma unroll
        for (int sl = 0; sl < TILES; ++sl) {
          if (kk == grp) {
            const int4 w = *reinterpret_cast<const int4*>(&wl.p[rt][kk][hh][sl * 16]);
            pa[rt][sl] = v4i{w.x, w.y, w.z, w.w};
          } else {
            pa[rt][sl] = v4i{0, 0, 0, 0};
          }
        }
        const float4 f0 = *reinterpret_cast<const float4*>(&wl.pst[rt][grp][0][0]);
        sp_[rt][0] = f0.x; sp_[rt][1] = f0.y; sp_[rt][2] = f0.z; sp_[rt][3] = f0.w;
        if constexpr (MODE != MODE_PV) {
          const float4 al = *reinterpret_cast<const float4*>(&wl.alpha[rt][0]);
          if (al.x != 1.0f || al.y != 1.0f || al.z != 1.0f || al.w != 1.0f) {
#pragma unroll
            for (int j = 0; j < 8; ++j) o_acc[rt][j] *= v4f{al.x, al.y, al.z, al.w};
          }
        }
        // P code sums (signed codes) of (block, head) from an all-ones B operand:
        // lane (channel, group k) receives sum p~' of block k for heads 0..3
        v4i sacc = v4i{0, 0, 0, 0};
#pragma unroll
        for (int sl = 0; sl < TILES; ++sl)
          sacc = mfma_i8(pa[rt][sl], v4i{0x01010101, 0x01010101, 0x01010101, 0x01010101}, sacc);
        const float zp[4] = {(float)sacc[0], (float)sacc[1], (float)sacc[2], (float)sacc[3]};
        // rank-1 coefficients, block-diagonal: lane (row kk*4+hh, group g) non-zero for kk == g
        // (such a lane's own registers hold the sums of block g = kk)
        pr1[rt] = kk == grp ? wl.pst[rt][kk][0][hh] * pick4(zp, hh) : 0.0f;  // s_p * sum p~'
        pr2[rt] = kk == grp ? wl.pst[rt][kk][1][hh] : 0.0f;                 // m~_p = m_p + 128 s_p
      }
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float mv = lo_half(d.vm[j]), svj = hi_half(d.vm[j]);
        const float vbar = fmaf(n_g, mv, svj * (float)d.vz[j]);  // s_v sum v' + n m_v
#pragma unroll
        for (int rt = 0; rt < GT; ++rt) {
          v4i acc = v4i{0, 0, 0, 0};
#pragma unroll
          for (int sl = 0; sl < TILES; ++sl) acc = mfma_i8(pa[rt][sl], unpack16<BITS>(d.vc + j * VW + sl * SW), acc);
          // Eq. 4: s_p s_v D~ + (s_p sum p~') m_v + m~_p (s_v sum v' + n m_v)
          o_acc[rt][j] = mfma_f32(pr1[rt], mv, o_acc[rt][j]);
          o_acc[rt][j] = mfma_f32(pr2[rt], vbar, o_acc[rt][j]);
#pragma unroll
          for (int i = 0; i < 4; ++i) o_acc[rt][j][i] = fmaf(sp_[rt][i] * svj, (float)acc[i], o_acc[rt][j][i]);
          if constexpr (MODE == MODE_PV) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int gh = rt * 4 + i;
              if (gvalid && gh < G)
                a.dbg_prod[(((int64_t)s * Hq + hkv * G + gh) * (a.max_len / PI) + vkb) * D + 8 * col + j] =
                    acc[i] + 128 * (int)d.vz[j];
            }
          }
        }
      }
    }
    // ---------------- fp16 open block: sum_t p_t v_t with unquantized p ----------------
    if constexpr (MODE == MODE_ATTEND) {
      if (kF >= 0) {
        const int tb = span0 + kF * PI;
        const __half* vt = c.v_tail + (((int64_t)s * H + hkv) * PI) * D + 8 * col;
        for (int e = grp; e < L - tb; e += 4) {
          const uint4 raw = *reinterpret_cast<const uint4*>(vt + (int64_t)e * D);
          const __half2* h2 = reinterpret_cast<const __half2*>(&raw);
          float vv[8];
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const float2 f = __half22float2(h2[j]);
            vv[2 * j] = f.x;
            vv[2 * j + 1] = f.y;
          }
#pragma unroll
          for (int rt = 0; rt < GT; ++rt)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const float p = wl.ptail[rt][i][e] * wl.tailf[rt][i];
#pragma unroll
              for (int j = 0; j < 8; ++j) o_acc[rt][j][i] = fmaf(p, vv[j], o_acc[rt][j][i]);
            }
        }
      }
    }
    // the next span rewrites this wave's LDS
    __builtin_amdgcn_s_waitcnt(0xC07F);
    __builtin_amdgcn_wave_barrier();
  };
  int si = wave;
#if HACK_DECODE_PREFETCH
  if (si < nspan_full) {
    SpanData<BITS, PI> cur;
    load_span(cur, t0 + si * SPAN, std::false_type{});
    for (; si < nspan_full; si += kWaves) {
      SpanData<BITS, PI> nxt;
      const bool more = si + kWaves < nspan_full;
      if (more) load_span(nxt, t0 + (si + kWaves) * SPAN, std::false_type{});
      compute_span(cur, t0 + si * SPAN, std::false_type{});
      if (more) cur = nxt;
    }
  }
#else
  for (; si < nspan_full; si += kWaves) {
    SpanData<BITS, PI> cur;
    load_span(cur, t0 + si * SPAN, std::false_type{});
    compute_span(cur, t0 + si * SPAN, std::false_type{});
  }
#endif
  if (nspan - 1 >= nspan_full && (nspan - 1) % kWaves == wave) {
    SpanData<BITS, PI> last;
    load_span(last, t0 + (nspan - 1) * SPAN, std::true_type{});
    compute_span(last, t0 + (nspan - 1) * SPAN, std::true_type{});
  }
  if constexpr (MODE == MODE_QK) return;

  // ---- wave result: O summed over the 4 lane groups (block slots), max and sum per head ----
#pragma unroll
  for (int rt = 0; rt < GT; ++rt) {
    float ov[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      float v4[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float v = o_acc[rt][j][i];
        v += __shfl_xor(v, 16, 64);
        v += __shfl_xor(v, 32, 64);
        v4[i] = v;
      }
      ov[j] = pick4(v4, grp);
    }
    const float lsum = row16_sum(l_run[rt]);
    // lane group g writes head slot 4*rt + g: channels 8*col .. 8*col+7
    float* dst = &mrg_o[wave][rt * 4 + grp][8 * col];
#pragma unroll
    for (int j = 0; j < 8; ++j) dst[j] = ov[j];
    if (col == 0) {
      mrg_ml[wave][rt * 4 + grp][0] = (MODE == MODE_PV) ? 0.0f : m_ref[rt];
      mrg_ml[wave][rt * 4 + grp][1] = (MODE == MODE_PV) ? 1.0f : lsum;
    }
  }
  __syncthreads();

  // ---- merge the four waves: thread (head slot, channel pair) ----
  const int64_t pair = (int64_t)s * H + hkv;
  constexpr int REC = 4 + D;  // max, sum, 2 pad, O
  for (int idx = tid; idx < G * (D / 2); idx += 256) {
    const int gh = idx / (D / 2), ch = 2 * (idx % (D / 2));
    float mmax = -INFINITY;
#pragma unroll
    for (int w = 0; w < kWaves; ++w)
      if (mrg_ml[w][gh][1] > 0.0f) mmax = fmaxf(mmax, mrg_ml[w][gh][0]);
    float lsum = 0.0f, o0 = 0.0f, o1 = 0.0f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      if (mrg_ml[w][gh][1] > 0.0f) {
        const float wt = MODE == MODE_PV ? 1.0f : __builtin_amdgcn_exp2f(mrg_ml[w][gh][0] - mmax);
        lsum = fmaf(mrg_ml[w][gh][1], wt, lsum);
        o0 = fmaf(mrg_o[w][gh][ch], wt, o0);
        o1 = fmaf(mrg_o[w][gh][ch + 1], wt, o1);
      }
    }
    float* o = a.out + ((int64_t)s * Hq + hkv * G + gh) * D + ch;
    if (MODE == MODE_PV) {
      o[0] = o0;
      o[1] = o1;
    } else if (nsplit == 1) {
      const float inv = 1.0f / lsum;
      o[0] = o0 * inv;
      o[1] = o1 * inv;
    } else {
      float* rec = a.partials + ((pair * a.splits + split) * G + gh) * REC;
      if (ch == 0) {
        rec[0] = mmax;
        rec[1] = lsum;
      }
      rec[4 + ch] = o0;
      rec[5 + ch] = o1;
    }
  }
}

// Split-K merge: one workgroup per (sequence, kv head) combines the partial
// (max, sum, O) of its chunks.  Runs as a separate launch so that the partials
// written by other workgroups are visible without device-wide cache flushes.
__global__ __launch_bounds__(256) void decode_merge_kernel(DecodeArgs a) {
  constexpr int D = 128, REC = 4 + D;
  const int s = blockIdx.y, hkv = blockIdx.x;
  const int G = a.group, Hq = a.num_q_heads;
  const int L = max(0, min(a.lens[s], a.max_len));
  const int nsplit = (L + a.chunk - 1) / a.chunk;
  if (nsplit <= 1) return;  // written directly by the attention kernel
  const int64_t pair = (int64_t)s * a.c.kv_heads + hkv;
  // thread (head gh, channels 4*q .. 4*q+3), one pass with a running max
  for (int idx = threadIdx.x; idx < G * (D / 4); idx += blockDim.x) {
    const int gh = idx / (D / 4), ch = 4 * (idx % (D / 4));
    float mrun = -INFINITY, lsum = 0.0f;
    float4 o = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll 4
    for (int sp = 0; sp < nsplit; ++sp) {
      const float* rec = a.partials + ((pair * a.splits + sp) * G + gh) * REC;
      const float ms = rec[0], ls = rec[1];
      const float4 os = *reinterpret_cast<const float4*>(rec + 4 + ch);
      const float mn = fmaxf(mrun, ms);
      const float wa = __builtin_amdgcn_exp2f(mrun - mn), wb = __builtin_amdgcn_exp2f(ms - mn);
      lsum = lsum * wa + ls * wb;
      o.x = o.x * wa + os.x * wb;
      o.y = o.y * wa + os.y * wb;
      o.z = o.z * wa + os.z * wb;
      o.w = o.w * wa + os.w * wb;
      mrun = mn;
    }
    const float inv = 1.0f / lsum;
    *reinterpret_cast<float4*>(a.out + ((int64_t)s * Hq + hkv * G + gh) * D + ch) =
        float4{o.x * inv, o.y * inv, o.z * inv, o.w * inv};
  }
}

DecodePlan plan_decode(const hack_kv_layout& lay, int batch, int num_q_heads, int max_len) {
  DecodePlan p{};
  const int64_t wg_tokens = 4 * lay.partition * kWaves;  // one span per wave
  const int64_t pairs = (int64_t)batch * lay.num_kv_heads;
  const int64_t G = lay.num_kv_heads > 0 ? num_q_heads / lay.num_kv_heads : 0;
  // workgroups to aim for over the whole grid (four waves each, 256 compute units)
  const int64_t target = HACK_DECODE_TARGET_WGS;
  int64_t chunk = pairs > 0 ? ((int64_t)max_len * pairs + target - 1) / target : wg_tokens;
  chunk = ((chunk + wg_tokens - 1) / wg_tokens) * wg_tokens;
  if (chunk < wg_tokens) chunk = wg_tokens;
  p.chunk = (int)chunk;
  p.splits = max_len > 0 ? (int)(((int64_t)max_len + chunk - 1) / chunk) : 1;
  p.partial_floats = pairs * p.splits * G * (4 + lay.head_dim);
  p.workspace_bytes = ((p.partial_floats * 4 + 255) / 256) * 256;
  return p;
}

template <int BITS, int PI, int GT, int MODE>
static hipError_t decode_impl(const DecodeArgs& a, int batch, hipStream_t stream) {
  dim3 grid((unsigned)a.splits, (unsigned)a.c.kv_heads, (unsigned)batch);
  hipLaunchKernelGGL((decode_kernel<BITS, PI, GT, MODE>), grid, dim3(256), 0, stream, a);
  if (MODE == MODE_ATTEND && a.splits > 1)
    hipLaunchKernelGGL(decode_merge_kernel, dim3((unsigned)a.c.kv_heads, (unsigned)batch), dim3(256), 0, stream, a);
  return hipGetLastError();
}

template <int BITS, int PI, int GT>
static hipError_t decode_mode(const DecodeArgs& a, int batch, int mode, hipStream_t stream) {
  switch (mode) {
    case MODE_ATTEND: return decode_impl<BITS, PI, GT, MODE_ATTEND>(a, batch, stream);
    case MODE_QK: return decode_impl<BITS, PI, GT, MODE_QK>(a, batch, stream);
    case MODE_PV: return decode_impl<BITS, PI, GT, MODE_PV>(a, batch, stream);
    default: return hipErrorInvalidValue;
  }
}

template <int BITS, int PI>
static hipError_t decode_gt(const DecodeArgs& a, int batch, int mode, hipStream_t stream) {
  if (a.group <= 4) return decode_mode<BITS, PI, 1>(a, batch, mode, stream);
  if (a.group <= 8) return decode_mode<BITS, PI, 2>(a, batch, mode, stream);
  return hipErrorInvalidValue;
}

hipError_t launch_decode(const hack_kv_layout& lay, const DecodeArgs& a, int batch, int mode,
                         hipStream_t stream) {
  switch (lay.kv_bits * 1000 + lay.partition) {
    case 2032: return decode_gt<2, 32>(a, batch, mode, stream);
    case 2064: return decode_gt<2, 64>(a, batch, mode, stream);
    case 4032: return decode_gt<4, 32>(a, batch, mode, stream);
    case 4064: return decode_gt<4, 64>(a, batch, mode, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace hack
