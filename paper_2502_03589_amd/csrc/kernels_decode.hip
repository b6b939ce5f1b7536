// Decode attention on quantized K/V (Sec. 5.3 with L_Q = 1; Eq. 2-4).
//
// Work split: one workgroup of four 64-lane wavefronts per (sequence, kv head,
// chunk of the context); wave w takes spans w, w+4, ... of the chunk, where a span
// is four V blocks (4*PI tokens) that lie in one page.  Every global load of a span
// is issued before any of its arithmetic, from wave-uniform section bases plus
// fixed per-lane offsets.  Per span a wave computes, for up to 4 query heads of the
// kv group per row tile:
//   Q'K'  rows (head h, channel quarter q), block-diagonal so that each quarter meets
//         only its own K channels; B = the K codes of the lane's token (lane = token,
//         group = quarter).  Lane (t, g) receives the four quarter products of head g.
//         2-bit K, partition 32: v_mfma_f32_16x16x128_f8f6f4 with the codes as e2m1
//         values c/2 (one mask and shift per 8 codes, no conversion of the products)
//         against the Q codes as two e4m3 pieces 16*(q >> 4) and q & 15 (both exact),
//         fp32 sums that are exact.  Otherwise v_mfma_i32_16x16x64_i8 with Q codes minus
//         2^(b-1) (signed) and the codes unpacked to bytes.
//   Eq. 4 matrix-core products with B = the lane's own K partition metadata spread
//         it over the output layout: v_mfma_f32_16x16x16_f16 gives s_q s_k per (head,
//         quarter) from s_q as three fp16 pieces against the stored fp16 s_k (as
//         exact as fp32, half the issue cycles of the fp32 product); the rank-1
//         terms (m~_q s_k sum k' and R_q m_k) arrive already summed over the
//         partitions, at 2 bits from one v_mfma_f32_16x16x32_f16 (the query-side
//         factors in fp16 pieces under a power-of-two scale per head, s_k sum k'
//         split exactly into two fp16 values, m_k as stored), at 4 bits from two
//         v_mfma_f32_16x16x4_f32.  The VALU converts the integer products and takes
//         four fused multiply-adds per score (log2 units).
//   softmax online with a lazily raised reference max; P quantized to 8 bits per
//         V block (min, scale, round-to-nearest-even codes), staged through LDS.
//   P'V'  v_mfma_i32_16x16x64_i8: A = P codes, rows = (block, head) block-diagonal
//         over the span's 4 blocks; B = V codes of 16 channels (lane = channel,
//         group = block).  One more MFMA with an all-ones B gives the P code sums.
//         Eq. 4 with the cached V sums on the VALU: each output of the P'V' layout
//         is (block, head) at the lane's channel, and the lane holds that block's V
//         metadata, so s_p s_v D~ + (s_p sum p~' + n m~_p) m_v + m~_p s_v sum v' is
//         a multiply and three fused multiply-adds per output (a block-diagonal
//         matrix-core product would spend four times the slots it uses).
//   open block  fp16 values times unquantized probabilities (TAIL_FP16), or its
//         re-quantized codes with n = T (TAIL_REQUANT).
// The four waves merge in LDS; when a sequence spans several chunks, each chunk's
// partial (max, sum, O) goes to the workspace and the workgroup that finishes the
// sequence's last chunk merges them in the same launch.
#include <algorithm>
#include <type_traits>

#include "hack_internal.hpp"

namespace hack {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef _Float16 v4h __attribute__((ext_vector_type(4)));

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

// Sum of the b-bit codes packed in N dwords, from population counts of the bit
// planes (the sum a cache without summation elimination does not store).
template <int BITS, int N>
__device__ __forceinline__ uint32_t code_sum(const uint32_t* w) {
  uint32_t s = 0;
#pragma unroll
  for (int i = 0; i < N; ++i) {
    if constexpr (BITS == 2) {
      s += __popc(w[i] & 0x55555555u) + 2u * __popc(w[i] & 0xAAAAAAAAu);
    } else {
      s += __popc(w[i] & 0x11111111u) + 2u * __popc(w[i] & 0x22222222u) + 4u * __popc(w[i] & 0x44444444u) +
           8u * __popc(w[i] & 0x88888888u);
    }
  }
  return s;
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
// fp16 matrix-core product with fp32 accumulation, four fp16 values per lane (element 2i
// in the low half of dword i): k slots 4g .. 4g+3 of lane group g.
__device__ __forceinline__ v4f mfma_f16k16(u32x2 a, u32x2 b, v4f c) {
  return __builtin_amdgcn_mfma_f32_16x16x16f16(__builtin_bit_cast(v4h, a), __builtin_bit_cast(v4h, b), c, 0, 0, 0);
}

typedef int v8i __attribute__((ext_vector_type(8)));
// 16x16x128 matrix-core product of fp8 (e4m3) A and fp4 (e2m1) B with fp32 accumulation.
// Lane (row or column l % 16, group g): the fp4 operand holds k = 32g .. 32g+31 in nibble
// order (its dwords 0-3); the fp8 operand holds k = 16g .. 16g+15 in dwords 0-3 and k =
// 64+16g .. 64+16g+15 in dwords 4-7.  Zero scale arguments select the unscaled instruction
// (no block scaling, measured identical to unit E8M0 scales): the scaled form keeps its
// scales in a VGPR, which the compiler was seen to rematerialize inside divergent code,
// leaving the lanes masked there with stale scales for the whole-wave product.
__device__ __forceinline__ v4f mfma_f8f4(v8i a, v8i b, v4f c) {
  return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, c, 0, 4, 0, 0, 0, 0);
}
// e4m3 encoding of an integer 0 <= v <= 15 (exact).
__device__ __forceinline__ uint32_t e4m3_int(uint32_t v) {
  if (v == 0) return 0u;
  const uint32_t e = 31u - (uint32_t)__builtin_clz(v);
  return ((e + 7u) << 3) | ((v << 3 >> e) & 7u);
}
// A 2-bit code c placed in a nibble is the e2m1 value c / 2.  One dword of 16 codes ->
// two operand dwords: nibble i of the first = code 2i, of the second = code 2i + 1.  Within
// a quarter's 32 k slots, slot f therefore holds channel fp4_channel(f).
__device__ __forceinline__ constexpr int fp4_channel(int f) {
  return (f & 16) | ((f & 7) << 1) | ((f >> 3) & 1);
}
__device__ __forceinline__ constexpr int fp4_slot(int ch) {  // inverse of fp4_channel
  return (ch & 16) | ((ch & 1) << 3) | ((ch >> 1) & 7);
}

// x (0 <= |x| < 65504) as three fp16 values h1 + h2 + h3 (h1 = fp16(x), h2 = fp16(x - h1),
// h3 = fp16(x - h1 - h2); both differences are exact in fp32), packed (h1, h2), (h3, 0).
// |x - h1 - h2 - h3| <= 2^-33 |x| while all three are normal fp16 values and <= 2^-25
// otherwise (half the subnormal spacing).  Against an fp16 value y in three k slots of
// an fp16 product the fp32 accumulator receives x*y to about fp32 accuracy.
__device__ __forceinline__ u32x2 split3(float x) {
  const __half h1 = __float2half_rn(x);
  const float r1 = x - __half2float(h1);
  const __half h2 = __float2half_rn(r1);
  const __half h3 = __float2half_rn(r1 - __half2float(h2));
  return u32x2{(uint32_t)__half_as_ushort(h1) | ((uint32_t)__half_as_ushort(h2) << 16), (uint32_t)__half_as_ushort(h3)};
}
// The fp16 value in the high half of w in three k slots: (y, y, y, 0).
__device__ __forceinline__ u32x2 triple_hi(uint32_t w) {
  const uint32_t y = w >> 16;
  return u32x2{y * 0x10001u, y};
}

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef _Float16 v8h __attribute__((ext_vector_type(8)));
// fp16 matrix-core product with fp32 accumulation, eight fp16 values per lane (element
// 2i in the low half of dword i); A and B pair their elements slot by slot.
__device__ __forceinline__ v4f mfma_f16k32(u32x4 a, u32x4 b, v4f c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(v8h, a), __builtin_bit_cast(v8h, b), c, 0, 0, 0);
}
// x as two fp16 values, each in both halves of a dword: (hi, hi) and (lo, lo), hi = x
// rounded toward zero, lo = x - hi (exact in fp32) rounded toward zero.  For x with at
// most 21 significant bits (an fp16 value times an integer below 2^10, times a power of
// two) and lo in fp16's normal range, hi + lo = x.
__device__ __forceinline__ u32x2 split2_rtz_pairs(float x) {
  const auto h = __builtin_amdgcn_cvt_pkrtz(x, x);
  const float r = x - (float)h[0];
  const auto l = __builtin_amdgcn_cvt_pkrtz(r, r);
  return u32x2{__builtin_bit_cast(uint32_t, h), __builtin_bit_cast(uint32_t, l)};
}
// x as two fp16 values rounded to nearest, (h1, h2) packed: |x - h1 - h2| <= 2^-22 |x|
// while both are normal.
__device__ __forceinline__ uint32_t split2(float x) {
  const __half h1 = __float2half_rn(x);
  const __half h2 = __float2half_rn(x - __half2float(h1));
  return (uint32_t)__half_as_ushort(h1) | ((uint32_t)__half_as_ushort(h2) << 16);
}

// Scores are kept scaled by score_unit<QP>(): a power of two that lifts the small factor
// s_q (log2 units) of the fp16 product above fp16's subnormal range without overflowing
// it: for fp16 inputs s_q <= 2^17 / (2^QP - 1) * 0.128, so score_unit * s_q < 2^14.
template <int QP>
constexpr float score_unit() {
  return QP == 8 ? 256.0f : 16.0f;
}
__device__ __forceinline__ float lo_half(uint32_t w) { return __half2float(__ushort_as_half((uint16_t)(w & 0xFFFFu))); }
__device__ __forceinline__ float hi_half(uint32_t w) { return __half2float(__ushort_as_half((uint16_t)(w >> 16))); }

// Sum four per-lane values over the four lane groups so that lane group g ends
// with the total of value g (permlane swaps across 32 and 16 lanes).
__device__ __forceinline__ float reduce_scatter4(float v0, float v1, float v2, float v3) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(v0), __float_as_uint(v2), false, false);
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v1), __float_as_uint(v3), false, false);
  const float x = __uint_as_float(a[0]) + __uint_as_float(a[1]);  // groups 0,1: value 0; 2,3: value 2
  const float y = __uint_as_float(b[0]) + __uint_as_float(b[1]);  // groups 0,1: value 1; 2,3: value 3
  const auto c = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(y), false, false);
  return __uint_as_float(c[0]) + __uint_as_float(c[1]);
}

// 1/sqrt(128) * log2(e): scores are kept in log2 units so softmax uses exp2.
constexpr float kScoreScale = 0.12751743074941640f;
// The reference max of the online softmax is raised only when a block's max
// exceeds it by more than this (p~ <= 2^8 in between).
constexpr float kMaxSlack = 8.0f;

constexpr int kWaves = 4;
constexpr int kComputeUnits = 256;  // MI355X


// Bytes of one cached code sum: 1 when b + ceil(log2 PI) <= 8, else 2 (Sec. 5.3).
template <int BITS, int PI>
constexpr int sum_width() {
  int need = BITS;
  for (int v = 1; v < PI; v <<= 1) ++need;
  return need <= 8 ? 1 : 2;
}

// Waves per SIMD the register budget is sized for (the launch bound's minimum).
// Measured: compiling for two waves per SIMD leaves the 2-bit, partition-32 kernel
// at about 145 VGPRs, so three are resident; a cap for three (168 VGPRs) or four
// (128 VGPRs, with V staged through LDS by direct loads) forced spills or a full
// wait on every span's loads and was slower.
template <int BITS, int PI, int GT>
constexpr int decode_occupancy() {
  return 2;
}

// Section bases of a span: its four V blocks are consecutive blocks of one page.
struct SpanBase {
  const uint8_t* kc;
  const uint8_t* km;
  const uint8_t* kz;
  const uint8_t* vc;
  const uint8_t* vm;
  const uint8_t* vz;
};

template <int BITS, int PI>
__device__ __forceinline__ SpanBase span_base(const CacheView& c, int s, int hkv, int span0) {
  constexpr int D = 128, P = D / PI, SB = sum_width<BITS, PI>();
  int64_t page;
  int slot0;
  if (c.block_table) {
    const int pidx = span0 / c.page_tokens;
    // the entry is wave-uniform and the kernel never writes the table: a scalar load
    // through the constant address space, which waits on itself alone (a vector load
    // here would be followed by a wait on every outstanding vector load)
    const auto* bt = (const __attribute__((address_space(4))) int32_t*)(uintptr_t)c.block_table;
    const int64_t pg = bt[(int64_t)s * c.mbps + pidx];
    page = pg < 0 ? 0 : (pg >= c.num_pages ? c.num_pages - 1 : pg);
    slot0 = span0 - pidx * c.page_tokens;
  } else {
    page = s < c.num_pages ? s : c.num_pages - 1;
    slot0 = span0;
  }
  const int64_t krow = (page * c.kv_heads + hkv) * c.page_tokens + slot0;
  const int64_t vblk = (page * c.kv_heads + hkv) * (c.page_tokens / PI) + slot0 / PI;
  SpanBase b;
  b.kc = c.k_codes + krow * (D * BITS / 8);
  b.km = reinterpret_cast<const uint8_t*>(c.k_meta) + krow * (P * 4);
  b.kz = c.k_sums + krow * (P * SB);
  b.vc = c.v_codes + vblk * (D * (PI * BITS / 8));
  b.vm = reinterpret_cast<const uint8_t*>(c.v_meta) + vblk * (D * 4);
  b.vz = c.v_sums + vblk * (D * SB);
  return b;
}

// Register copy of one span's compressed data for one lane.
template <int BITS, int PI>
struct SpanData {
  static constexpr int NT = PI / 4;              // 16-token tiles per span
  static constexpr int VW = PI * BITS / 32;      // V dwords per (channel, block)
  static constexpr int SB = sum_width<BITS, PI>();
  uint32_t kc[NT][BITS];  // K codes of the lane's token and channel quarter, per tile
  uint32_t km[NT];        // (m_k, s_k) of the lane's K partition, per tile
  uint32_t kz[NT];        // cached code sum of that partition, per tile
  uint32_t vc[8 * VW];    // V codes of 8 channels of the lane's block
  uint32_t vm[8];         // (m_v, s_v) of those channels
  uint32_t vz[2 * SB];    // cached V code sums of those channels, packed
};

// LDS of one wave.
template <int BITS, int PI, int GT>
struct WaveLds {
  static constexpr int HT = 4 * GT;
  int8_t p[GT][4][4][PI];       // P codes - qoff: [row tile][block][head][token position]
  int8_t pz[PI];                // zeros: the P operand of the lanes off the block diagonal
  float pst[GT][4][2][4];       // [rt][block][s_p | m~_p][head], scaled to the span's reference max
  float alpha[GT][4];           // O rescale of the span, per head
  float tailf[GT][4];           // scale of the fp16 open block's probabilities
  float ptail[GT][4][PI];       // unquantized p~ of the open block
  float mrg_o[HT][128];          // the wave's partial O after its last span
};

// Split-K merge of one (sequence, kv head): combines the partial (max, sum, O) of
// its nsplit chunks with a running max and writes O / sum.  The records of all
// planned chunks are read together (records past the sequence are stale and are
// masked by the length), so the caller waits on memory once per group of U chunks.
__device__ __forceinline__ float ld_rec(const float* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void merge_chunks(const DecodeArgs& a, int s, int hkv, int Lraw, int head0, int Gl) {
  constexpr int D = 128, REC = 4 + D, U = 8;
  const int G = a.group, Hq = a.num_q_heads;
  const int64_t pair = (int64_t)s * a.c.kv_heads + hkv;
  // thread (head gh, channels 4*q .. 4*q+3)
  for (int idx = threadIdx.x; idx < Gl * (D / 4); idx += blockDim.x) {
    const int gh = head0 + idx / (D / 4), ch = 4 * (idx % (D / 4));
    float mrun = -INFINITY, lsum = 0.0f;
    float4 o = {0.0f, 0.0f, 0.0f, 0.0f};
    for (int sp0 = 0; sp0 < a.splits; sp0 += U) {
      float ms[U], ls[U];
      float4 os[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        if (sp0 + u < a.splits) {
          // agent-coherent loads: the records were written by other workgroups
          const float* rec = a.partials + ((pair * a.splits + sp0 + u) * G + gh) * REC;
          ms[u] = ld_rec(rec);
          ls[u] = ld_rec(rec + 1);
          os[u] = float4{ld_rec(rec + 4 + ch), ld_rec(rec + 5 + ch), ld_rec(rec + 6 + ch), ld_rec(rec + 7 + ch)};
        } else {
          ms[u] = -INFINITY;
          ls[u] = 0.0f;
          os[u] = float4{0.0f, 0.0f, 0.0f, 0.0f};
        }
      }
      const int L = max(0, min(Lraw, a.max_len));
      const int nsplit = (L + a.chunk - 1) / a.chunk;
      float mn = mrun;
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (sp0 + u < nsplit && ls[u] > 0.0f) mn = fmaxf(mn, ms[u]);
      const float wa = mrun == -INFINITY ? 0.0f : __builtin_amdgcn_exp2f(mrun - mn);
      lsum *= wa;
      o.x *= wa; o.y *= wa; o.z *= wa; o.w *= wa;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const float wb = (sp0 + u < nsplit && ls[u] > 0.0f) ? __builtin_amdgcn_exp2f(ms[u] - mn) : 0.0f;
        lsum = fmaf(ls[u], wb, lsum);
        o.x = fmaf(os[u].x, wb, o.x);
        o.y = fmaf(os[u].y, wb, o.y);
        o.z = fmaf(os[u].z, wb, o.z);
        o.w = fmaf(os[u].w, wb, o.w);
      }
      mrun = mn;
    }
    const float inv = 1.0f / lsum;
    *reinterpret_cast<float4*>(a.out + ((int64_t)s * Hq + hkv * G + gh) * D + ch) =
        float4{o.x * inv, o.y * inv, o.z * inv, o.w * inv};
  }
}

// SE: the cache stores the partition code sums (summation elimination, Sec. 5.3);
// without them each sum is rebuilt from the packed codes already in registers.
// SR: the Q and P codes are rounded stochastically (the layout's rounding mode).
template <int BITS, int PI, int GT, int MODE, int QP, bool SE, bool SR>
__global__ __launch_bounds__(256, (decode_occupancy<BITS, PI, GT>())) void decode_kernel(DecodeArgs a) {
  constexpr int D = 128;
  // Q and P codes of QP bits: 2^QP - 1 levels; they enter the signed MFMA as code - 2^(QP-1)
  constexpr float kQmax = (float)((1 << QP) - 1);
  constexpr float kInvQmax = 1.0f / kQmax;
  constexpr int kQoff = 1 << (QP - 1);
  constexpr float kQoffF = (float)kQoff;
  constexpr float kSU = score_unit<QP>(), kInvSU = 1.0f / kSU;  // score unit (see score_unit)
  // Q'K' rank-1 terms on one fp16 16x16x32 product (2-bit K) or two fp32 16x16x4 products
  // (4-bit K, whose kernels sit at the register budget of three waves per SIMD: the fp16
  // operands take three more registers).  2^kRankB (2^BITS - 1) PI <= 1 keeps
  // s_k sum k' 2^kRankB below fp16's largest value.
  constexpr bool kRankF16 = BITS == 2;
  constexpr int kRankB = BITS == 2 ? (PI == 32 ? -7 : -8) : (PI == 32 ? -9 : -10);
  constexpr float kRankScale = BITS == 2 ? (PI == 32 ? 0x1p-7f : 0x1p-8f) : (PI == 32 ? 0x1p-9f : 0x1p-10f);
  constexpr int P = D / PI;          // K partitions per token
  constexpr int QPP = 4 / P;         // channel quarters per partition
  constexpr int TILES = PI / 16;     // 16-token tiles per V block
  constexpr int SPAN = 4 * PI;
  constexpr int NT = 4 * TILES;      // token tiles per span
  constexpr int KW = BITS;           // K code dwords per (token, quarter of 32 channels)
  constexpr int VW = PI * BITS / 32; // V code dwords per (channel, block)
  constexpr int SW = BITS / 2;       // dwords per 16-code slice
  constexpr int SB = sum_width<BITS, PI>();
  constexpr int HT = GT * 4;
  constexpr int KROW = D * BITS / 8; // K code bytes per token

  // Q codes - qoff per (head slot, quarter, 16-channel slice), each slice already in
  // the byte order of the K operand's in-register unpack
  // 2-bit K at partition 32: Q'K' runs on fp8 x fp4 products (K codes need only a nibble
  // spread, the products arrive in fp32); Q codes enter as e4m3 pieces 16*(q >> 4) and
  // q & 15.  At partition 64 a span holds twice the tiles and the 32-cycle fp8 products
  // cost more than the unpack they save (measured 22.4 against 19.3 us on the 4K
  // workload), so the int8 path stays there.
  constexpr bool F4 = BITS == 2 && PI == 32;
  __shared__ __attribute__((aligned(16))) int8_t q_lds[F4 ? 1 : HT][4][2][16];
  __shared__ __attribute__((aligned(16))) uint8_t q8_lds[2][F4 ? HT : 1][4][32];
  __shared__ float qm_lds[HT][4][3];
  __shared__ float qu_lds[HT];  // unscale of a head's fp16 rank-1 product
  __shared__ __attribute__((aligned(16))) WaveLds<BITS, PI, GT> wl_all[kWaves];
  __shared__ float mrg_ml[kWaves][HT][2];

  const CacheView& c = a.c;
  const int tid = threadIdx.x;
  // wave index made explicitly wave-uniform so span bookkeeping stays in scalar registers
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const int col = lane & 15, grp = lane >> 4;
  // chunk index slowest: every (sequence, head) pair's first chunks are dispatched
  // before any pair's later ones, so a long sequence's chunks do not queue behind
  // the short sequences of a ragged batch
  const int G = a.group, Hq = a.num_q_heads, H = c.kv_heads;
  // a kv group of more than HT heads is split over workgroups (blockIdx.x = hg * H + hkv,
  // so the workgroups of one chunk are H apart in the grid and share an XCD's L2)
  const bool one_group = a.head_groups == 1;
  const int s = blockIdx.y, split = blockIdx.z;
  const int hkv = one_group ? (int)blockIdx.x : (int)blockIdx.x % H, hg = one_group ? 0 : (int)blockIdx.x / H;
  const int head0 = HT * hg, Gl = min(HT, G - head0);  // this workgroup's heads of the group
  // lengths outside [0, max_len] break the caller contract; clamp so that every
  // access stays inside the cache and the workspace
  // this wave's query values (head slots wave, wave + 4, ...) do not depend on the
  // length: their loads are issued first so the two memory round trips overlap
  uint32_t qraw[GT];
#pragma unroll
  for (int i = 0; i < GT; ++i) {
    const int gh = wave + kWaves * i;
    qraw[i] = (MODE != MODE_PV && gh < Gl)
                  ? reinterpret_cast<const uint32_t*>(a.q + ((int64_t)s * Hq + hkv * G + head0 + gh) * D)[lane]
                  : 0u;
  }
  const int Lin = a.lens[s];
  int Lq = max(0, min(Lin, a.max_len));
  const int t0 = split * a.chunk;
  if (MODE == MODE_ATTEND && a.k_new != nullptr) {
    // decode step: append token Lin first (the workgroup whose chunk holds it), then
    // attend over Lin + 1 tokens.  Other chunks never read the appended slots, and
    // the new length goes to a separate array so no workgroup sees it half-way.
    const bool ok = Lin >= 0 && Lin < a.capacity && Lin + 1 <= a.max_len;
    Lq = ok ? Lin + 1 : Lq;
    if (split == 0 && blockIdx.x == 0 && tid == 0) a.lens_out[s] = Lq;
    if (ok && Lin / a.chunk == split) {
      append_head<BITS, PI>(c, a.k_new + ((int64_t)s * H + hkv) * D, a.v_new + ((int64_t)s * H + hkv) * D, s, hkv,
                            Lin, a.tail_requant, a.stochastic != 0, a.key_k, a.key_v, tid, 256);
      __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): the appended bytes are in L2
      __syncthreads();
    }
  }
  const int L = Lq;
  if (t0 >= L) {
    if (MODE == MODE_ATTEND && split == 0) {  // empty sequence: zeros
      for (int i = tid; i < Gl * D; i += 256) a.out[((int64_t)s * Hq + hkv * G + head0) * D + i] = 0.0f;
    }
    return;
  }
  const int t1 = min(L, t0 + a.chunk);
  const int nsplit = (L + a.chunk - 1) / a.chunk;
  const int F = L / PI, T = L - F * PI;
  const bool requant = a.tail_requant != 0;
  WaveLds<BITS, PI, GT>& wl = wl_all[wave];
  if (lane < PI / 4) reinterpret_cast<int*>(wl.pz)[lane] = 0;  // read by this wave only

  // ---- Q: 8-bit codes per partition with float32 metadata (Sec. 5.1, Sec. 5.2) ----
  // wave w quantizes head slots w, w+4, ...; each lane holds two channels
  if constexpr (MODE != MODE_PV) {
#pragma unroll
    for (int i = 0; i < GT; ++i) {
      const int gh = wave + kWaves * i;
      const bool real = gh < Gl;
      const int hq = hkv * G + head0 + gh;
      float x0 = 0.0f, x1 = 0.0f;
      if (real) {
        const float2 f = __half22float2(*reinterpret_cast<const __half2*>(&qraw[i]));
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
        sq = __fdiv_rn(__fsub_rn(mx, mn), kQmax);
        if (sq != 0.0f) {
          const float r = __fdiv_rn(1.0f, sq);
          const float t0 = __fmul_rn(__fsub_rn(x0, mn), r), t1 = __fmul_rn(__fsub_rn(x1, mn), r);
          if constexpr (SR) {
            c0 = round_stochastic(t0, sr_threshold(a.key_q, qp_index(s, Hq, hq, 0, 2 * lane)), kQmax);
            c1 = round_stochastic(t1, sr_threshold(a.key_q, qp_index(s, Hq, hq, 0, 2 * lane + 1)), kQmax);
          } else {
            c0 = fminf(rintf(t0), kQmax);
            c1 = fminf(rintf(t1), kQmax);
          }
        }
      }
      int csum = (int)c0 + (int)c1;
#pragma unroll
      for (int m = 1; m < PI / 2; m <<= 1) csum += __shfl_xor(csum, m, 64);
      {
        const int ch = 2 * lane;  // channels ch, ch + 1 share quarter and slice
        const int g = ch >> 5, m = (ch >> 4) & 1, e = ch & 15;
        if constexpr (F4) {
          const uint32_t u0 = real ? (uint32_t)c0 : 0u, u1 = real ? (uint32_t)c1 : 0u;
          const int f0 = fp4_slot(ch & 31), f1 = fp4_slot((ch + 1) & 31);
          q8_lds[0][gh][g][f0] = (uint8_t)((u0 >> 4) ? e4m3_int(u0 >> 4) + 0x20u : 0u);  // 16 * (q >> 4)
          q8_lds[0][gh][g][f1] = (uint8_t)((u1 >> 4) ? e4m3_int(u1 >> 4) + 0x20u : 0u);
          q8_lds[1][gh][g][f0] = (uint8_t)e4m3_int(u0 & 15u);
          q8_lds[1][gh][g][f1] = (uint8_t)e4m3_int(u1 & 15u);
        } else {
          q_lds[gh][g][m][perm_position<BITS>(e)] = real ? (int8_t)((int)c0 - kQoff) : (int8_t)0;
          q_lds[gh][g][m][perm_position<BITS>(e + 1)] = real ? (int8_t)((int)c1 - kQoff) : (int8_t)0;
        }
      }
      const int p = (2 * lane) / PI;
      // Rank-1 factors of the partition in score units, divided among its QPP quarters:
      // m~_q = m_q + qoff s_q (the fp8 products take the unsigned codes: m_q) and
      // R = s_q sum q' + n m_q.  For the fp16 product both are scaled by a power of two
      // 2^e per head (R by 2^(e + kRankB) more) that brings the head's largest magnitude
      // into [2^13, 2^14): fp16's range then holds them for any fp16 input.
      constexpr float kRankUnit = kSU / (float)QPP;
      float r1 = real ? kScoreScale * (F4 ? mn : mn + kQoffF * sq) * kRankUnit : 0.0f;
      float r2 = real ? kScoreScale * (sq * (float)csum + (float)PI * mn) * kRankUnit : 0.0f;
      int qe = 0;
      if constexpr (kRankF16) {
        float mx = fmaxf(fabsf(r1), fabsf(r2) * kRankScale);
#pragma unroll
        for (int m = PI / 2; m < 64; m <<= 1) mx = fmaxf(mx, __shfl_xor(mx, m, 64));
        qe = mx > 0.0f ? 14 - __builtin_amdgcn_frexp_expf(mx) : 0;
        r1 = ldexpf(r1, qe);
        r2 = ldexpf(r2, qe + kRankB);
      }
      if ((2 * lane) % PI == 0) {
        // per partition (log2 units): s_q and the rank-1 factors above
        qm_lds[gh][p][0] = real ? kScoreScale * sq : 0.0f;
        qm_lds[gh][p][1] = r1;
        qm_lds[gh][p][2] = r2;
        if (kRankF16 && p == 0) qu_lds[gh] = ldexpf(1.0f, -(qe + kRankB));
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

  // Q operands.  Rows of the QK tile are (head h, quarter q) = 4h + q; the i8
  // operand of lane (row, group g) is non-zero only for q == g.  The Eq. 4 operands
  // take the lane's group as the summed index k: qs = s_q of (h, quarter k) on the
  // diagonal q == k, so s_q s_k lands at (lane group h, register q); the rank-1
  // operands hold m~_q and R of (h, partition of quarter k), divided among the QPP
  // quarters of a partition, so that the rank-1 terms arrive summed over the partitions.
  // With fp8 x fp4 products (2-bit K) the quarter q of row (h, q) occupies k slots 32q ..
  // 32q+31, which the fp8 operand spreads over lane groups 2(q mod 2), 2(q mod 2) + 1 in
  // dwords 0-3 (q < 2) or 4-7 (q >= 2); those products carry K codes as e2m1 values c/2,
  // so s_q is doubled.
  v4i qa[F4 ? 1 : GT][2];
  v8i q8h[F4 ? GT : 1], q8l[F4 ? GT : 1];
  u32x2 qs[GT];
  float ra0[kRankF16 ? 1 : GT], ra1[kRankF16 ? 1 : GT];  // rank-1 A operands (fp32 products)
  u32x4 ra[kRankF16 ? GT : 1];                            // rank-1 A operand (fp16 product)
  float run[kRankF16 ? GT : 1];                           // its unscale for head grp
  const int pl = grp / QPP;  // partition of this lane's quarter
  if constexpr (MODE != MODE_PV) {
    const int hh = col >> 2, qq = col & 3;
#pragma unroll
    for (int rt = 0; rt < GT; ++rt) {
      if constexpr (F4) {
        const bool lo_half = qq == (grp >> 1), hi_half = qq == 2 + (grp >> 1);
        int4 wh = int4{0, 0, 0, 0}, wl = int4{0, 0, 0, 0};
        if (lo_half || hi_half) {
          wh = *reinterpret_cast<const int4*>(&q8_lds[0][rt * 4 + hh][qq][16 * (grp & 1)]);
          wl = *reinterpret_cast<const int4*>(&q8_lds[1][rt * 4 + hh][qq][16 * (grp & 1)]);
        }
        q8h[rt] = lo_half ? v8i{wh.x, wh.y, wh.z, wh.w, 0, 0, 0, 0} : v8i{0, 0, 0, 0, wh.x, wh.y, wh.z, wh.w};
        q8l[rt] = lo_half ? v8i{wl.x, wl.y, wl.z, wl.w, 0, 0, 0, 0} : v8i{0, 0, 0, 0, wl.x, wl.y, wl.z, wl.w};
      } else {
#pragma unroll
        for (int m = 0; m < 2; ++m) {
          const int4 w = *reinterpret_cast<const int4*>(&q_lds[rt * 4 + hh][grp][m][0]);
          qa[rt][m] = qq == grp ? v4i{w.x, w.y, w.z, w.w} : v4i{0, 0, 0, 0};
        }
      }
      qs[rt] = qq == grp ? split3((F4 ? 2.0f * kSU : kSU) * qm_lds[rt * 4 + hh][pl][0]) : u32x2{0u, 0u};
      if constexpr (kRankF16) {
        // per lane group, A slots (m~ hi, m~ lo, m~ hi, m~ lo, R h1, R h2, R h3, 0) of (head,
        // partition of the quarter) against B slots (b hi, b hi, b lo, b lo, m_k, m_k, m_k,
        // s_k) of (token, partition), b = s_k sum k' 2^kRankB split exactly; the last B
        // dword is the stored (m_k, s_k) word itself
        const uint32_t a0 = split2(qm_lds[rt * 4 + hh][pl][1]);
        const u32x2 a1 = split3(qm_lds[rt * 4 + hh][pl][2]);
        ra[rt] = u32x4{a0, a0, a1[0], a1[1]};
        run[rt] = qu_lds[rt * 4 + grp];
      } else {
        ra0[rt] = qm_lds[rt * 4 + hh][pl][1];
        ra1[rt] = qm_lds[rt * 4 + hh][pl][2];
      }
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
  // per-lane byte offsets inside a span's sections (tile ti adds ti * 16 rows)
  const uint32_t kc_off = (uint32_t)(col * KROW + grp * (32 * BITS / 8));
  const uint32_t km_off = (uint32_t)((col * P + pl) * 4);
  const uint32_t kz_off = (uint32_t)((col * P + pl) * SB);
  const uint32_t vc_off = (uint32_t)((grp * D + 8 * col) * (PI * BITS / 8));
  const uint32_t vm_off = (uint32_t)((grp * D + 8 * col) * 4);
  const uint32_t vz_off = (uint32_t)((grp * D + 8 * col) * SB);

  // Spans whose tokens are all valid and whose blocks are all quantized take the
  // unmasked path; at most one span per chunk, its last, is partial.
  const int nspan_full = max(0, min(nspan, (F * PI - t0) / SPAN));
  auto load_span = [&](SpanData<BITS, PI>& d, int span0, auto masked_tag) __attribute__((always_inline)) {
    constexpr bool MASKED = decltype(masked_tag)::value;
    constexpr bool full = !MASKED;
    const SpanBase b = span_base<BITS, PI>(c, s, hkv, span0);
    // the offsets stay 32-bit values next to each load (not hoisted and widened), so
    // every load takes the scalar-base + 32-bit-offset + immediate form
    uint32_t o_kc = kc_off, o_km = km_off, o_kz = kz_off, o_vc = vc_off, o_vm = vm_off, o_vz = vz_off;
    asm volatile("" : "+v"(o_kc), "+v"(o_km), "+v"(o_kz), "+v"(o_vc), "+v"(o_vm), "+v"(o_vz));
#pragma unroll
    for (int ti = 0; ti < NT; ++ti) {
      if (full || span0 + 16 * ti + col < L) {
        load_words<KW>(b.kc + o_kc + ti * 16 * KROW, d.kc[ti]);
        d.km[ti] = *reinterpret_cast<const uint32_t*>(b.km + o_km + ti * 16 * P * 4);
        if constexpr (!SE) d.kz[ti] = 0u;
        else if constexpr (SB == 1) d.kz[ti] = *(b.kz + o_kz + ti * 16 * P);  // offset folds into the load
        else d.kz[ti] = *reinterpret_cast<const uint16_t*>(b.kz + o_kz + ti * 16 * P * 2);
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
    if (gvalid) {
      load_words<8 * VW>(b.vc + o_vc, d.vc);
      load_words<8>(b.vm + o_vm, d.vm);
      if constexpr (SE) {
        load_words<2 * SB>(b.vz + o_vz, d.vz);
      } else {
#pragma unroll
        for (int j = 0; j < 2 * SB; ++j) d.vz[j] = 0u;
      }
    } else {
#pragma unroll
      for (int w = 0; w < 8 * VW; ++w) d.vc[w] = 0u;
#pragma unroll
      for (int j = 0; j < 8; ++j) d.vm[j] = 0u;
#pragma unroll
      for (int j = 0; j < 2 * SB; ++j) d.vz[j] = 0u;
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
          if (present && kb < F && gh < Gl)
            v = (int8_t)((int)a.dbg_pcodes[(((int64_t)s * Hq + hkv * G + head0 + gh) * NB + kb) * PI + e] - kQoff);
          wl.p[rt][k][hh][(e >> 4) * 16 + perm_position<BITS>(e & 15)] = v;
        }
        if (lane < HT) {
          const int rt = lane >> 2, hh = lane & 3, gh = lane;
          float pm = 0.0f, ps = 0.0f;
          if (present && kb < F && gh < Gl) {
            const int64_t base = ((int64_t)s * Hq + hkv * G + head0 + gh) * NB + kb;
            pm = a.dbg_pmeta[base * 2 + 0];
            ps = a.dbg_pmeta[base * 2 + 1];
          }
          wl.pst[rt][k][0][hh] = ps;
          wl.pst[rt][k][1][hh] = pm + kQoffF * ps;
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
          v4i b0, b1;
          v8i b8;
          if constexpr (F4) {
            const uint32_t w0 = d.kc[ti][0], w1 = d.kc[ti][1];
            b8 = v8i{(int)(w0 & 0x33333333u), (int)((w0 >> 2) & 0x33333333u), (int)(w1 & 0x33333333u),
                     (int)((w1 >> 2) & 0x33333333u), 0, 0, 0, 0};
          } else {
            b0 = unpack16<BITS>(d.kc[ti]);
            b1 = unpack16<BITS>(d.kc[ti] + SW);
          }
          // the lane's own K partition: m_k, s_k and the cached code sum
          uint32_t kzv;  // code sum of the lane's K partition
          if constexpr (SE) {
            kzv = d.kz[ti];
          } else {
            kzv = code_sum<BITS, KW>(d.kc[ti]);
            if constexpr (QPP == 2) kzv += (uint32_t)__shfl_xor((int)kzv, 16, 64);  // the partition's other quarter
          }
          [[maybe_unused]] float bz, mk;   // s_k sum k' and m_k for the fp32 products
          [[maybe_unused]] u32x4 rb;       // B operand of the fp16 product
          if constexpr (kRankF16) {
            // s_k sum k' 2^kRankB, exact in fp32 (the fp16 s_k enters the FMA unconverted)
            const u32x2 b = split2_rtz_pairs(fmaf(hi_half(d.km[ti]), (float)kzv * kRankScale, 0.0f));
            rb = u32x4{b[0], b[1], __builtin_amdgcn_perm(d.km[ti], d.km[ti], 0x01000100u), d.km[ti]};
          } else {
            bz = hi_half(d.km[ti]) * (float)kzv;
            mk = lo_half(d.km[ti]);
          }
#pragma unroll
          for (int rt = 0; rt < GT; ++rt) {
            // quarter products: fp32 sum of q' k' / 2 (unsigned codes) or int32 sum of (q' - qoff) k'
            v4f accf;
            v4i acc = v4i{0, 0, 0, 0};
            if constexpr (F4) {
              accf = QP == 8 ? mfma_f8f4(q8h[rt], b8, v4f{0.0f, 0.0f, 0.0f, 0.0f}) : v4f{0.0f, 0.0f, 0.0f, 0.0f};
              accf = mfma_f8f4(q8l[rt], b8, accf);
            } else {
              acc = mfma_i8(qa[rt][0], b0, acc);
              acc = mfma_i8(qa[rt][1], b1, acc);
              accf = v4f{(float)acc[0], (float)acc[1], (float)acc[2], (float)acc[3]};
            }
            // s_q s_k per quarter (in score units)
            const v4f sqk = mfma_f16k16(qs[rt], triple_hi(d.km[ti]), v4f{0.0f, 0.0f, 0.0f, 0.0f});
            // sum over partitions of m~_q s_k sum k' + R_q m_k
            float sc;
            if constexpr (kRankF16) {
              sc = mfma_f16k32(ra[rt], rb, v4f{0.0f, 0.0f, 0.0f, 0.0f})[0] * run[rt];
            } else {
              v4f rk = mfma_f32(ra0[rt], bz, v4f{0.0f, 0.0f, 0.0f, 0.0f});
              sc = mfma_f32(ra1[rt], mk, rk)[0];
            }
#pragma unroll
            for (int q = 0; q < 4; ++q) sc = fmaf(accf[q], sqk[q], sc);
            if constexpr (MODE == MODE_QK) {
              // integer partition products (unsigned codes) for the test export:
              // quarter q's code sum comes from lane (token, q)
              const int tok = bt0 + 16 * tl + col;
              const int gh = rt * 4 + grp;
              int zq[P];
#pragma unroll
              for (int p = 0; p < P; ++p) zq[p] = __shfl((int)d.kz[ti], 16 * (p * QPP) + col, 64);
              if (tok < L && gh < Gl) {
#pragma unroll
                for (int p = 0; p < P; ++p) {
                  int v = F4 ? 0 : kQoff * zq[p];
#pragma unroll
                  for (int q = p * QPP; q < (p + 1) * QPP; ++q) v += F4 ? (int)(2.0f * accf[q]) : acc[q];
                  a.dbg_prod[(((int64_t)s * Hq + hkv * G + head0 + gh) * a.max_len + tok) * P + p] = v;
                }
              }
            }
            sv[rt][tl] = (full || bt0 + 16 * tl + col < L) ? sc : -INFINITY;
          }
        }
        if constexpr (MODE == MODE_QK) continue;
#pragma unroll
        for (int rt = 0; rt < GT; ++rt) {
          float bmax = sv[rt][0];
#pragma unroll
          for (int tl = 1; tl < TILES; ++tl) bmax = fmaxf(bmax, sv[rt][tl]);
          bmax = row16_max(bmax) * kInvSU;  // the scores are in score units
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
            pt[tl] = __builtin_amdgcn_exp2f(fmaf(sv[rt][tl], kInvSU, -mr));
            lsum += pt[tl];
          }
          l_run[rt] += lsum;
          if (quantized) {
            float bmin = (full || bt0 + col < L) ? sv[rt][0] : INFINITY;
#pragma unroll
            for (int tl = 1; tl < TILES; ++tl)
              bmin = fminf(bmin, (full || bt0 + 16 * tl + col < L) ? sv[rt][tl] : INFINITY);
            bmin = row16_min(bmin) * kInvSU;
            const float pmax = __builtin_amdgcn_exp2f(bmax - mr);
            const float pmin = __builtin_amdgcn_exp2f(bmin - mr);
            const float dp = pmax - pmin;
            const float r = dp > 0.0f ? kQmax * __builtin_amdgcn_rcpf(dp) : 0.0f;
            const float bias = -pmin * r;
#pragma unroll
            for (int tl = 0; tl < TILES; ++tl) {
              // round-to-nearest-even with saturation (codes stay within [0, qmax])
              uint32_t code;
              if constexpr (SR) {
                const int tok = bt0 + 16 * tl + col;
                const float u = sr_threshold(a.key_p, qp_index(s, Hq, hkv * G + head0 + rt * 4 + grp, 0, tok));
                code = (uint32_t)round_stochastic(fmaf(pt[tl], r, bias), u, kQmax);
              } else {
                code = __builtin_amdgcn_cvt_pk_u8_f32(fmaf(pt[tl], r, bias), 0, 0u);
              }
              const bool valid = full || bt0 + 16 * tl + col < L;
              wl.p[rt][k][grp][tl * 16 + perm_position<BITS>(col)] = valid ? (int8_t)((int)code - kQoff) : (int8_t)0;
            }
            ps_s[rt][k] = dp * kInvQmax;
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
            wl.pst[rt][k][1][grp] = (ps_m[rt][k] + kQoffF * ps_s[rt][k]) * f;
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
      const uint32_t* vcr = d.vc;
      const uint32_t* vmr = d.vm;
      const uint32_t* vzr = d.vz;
      const float n_g = (float)(vkb < F ? PI : T);
      const int kk = col >> 2, hh = col & 3;
      v4i pa[GT][TILES];
      float psp[GT][4], pc1[GT][4], pmt[GT][4];
#pragma unroll
      for (int rt = 0; rt < GT; ++rt) {
        // block-diagonal P operand.  At 2 bits the lanes off the diagonal read the zero
        // row, so every lane loads unconditionally (no masked loads and operand copies);
        // at 4 bits the kernels sit at the 168-register budget of three waves per SIMD,
        // which that form exceeds by two registers.
        if constexpr (BITS == 2) {
          const int8_t* prow = kk == grp ? &wl.p[rt][kk][hh][0] : &wl.pz[0];
#pragma unroll
          for (int sl = 0; sl < TILES; ++sl) {
            const int4 w = *reinterpret_cast<const int4*>(prow + sl * 16);
            pa[rt][sl] = v4i{w.x, w.y, w.z, w.w};
          }
        } else {
#pragma unroll
          for (int sl = 0; sl < TILES; ++sl) {
            if (kk == grp) {
              const int4 w = *reinterpret_cast<const int4*>(&wl.p[rt][kk][hh][sl * 16]);
              pa[rt][sl] = v4i{w.x, w.y, w.z, w.w};
            } else {
              pa[rt][sl] = v4i{0, 0, 0, 0};
            }
          }
        }
        if constexpr (MODE != MODE_PV) {
          // the rescale is exactly 1 for a head whose reference max stayed put in this
          // span; a wave-wide vote skips the multiplies (and the LDS read) when all did
          if (__builtin_amdgcn_ballot_w64(m_start[rt] != m_ref[rt]) != 0) {
            const float4 al = *reinterpret_cast<const float4*>(&wl.alpha[rt][0]);
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
        // The lane's outputs are (block grp, heads 0..3) at its channel: the P-side factors of
        // its own block.
        const float4 sp4 = *reinterpret_cast<const float4*>(&wl.pst[rt][grp][0][0]);
        const float4 mp4 = *reinterpret_cast<const float4*>(&wl.pst[rt][grp][1][0]);
        const float spa[4] = {sp4.x, sp4.y, sp4.z, sp4.w}, mpa[4] = {mp4.x, mp4.y, mp4.z, mp4.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          psp[rt][i] = spa[i];                                               // s_p
          pmt[rt][i] = mpa[i];                                               // m~_p = m_p + qoff s_p
          pc1[rt][i] = fmaf(n_g, pmt[rt][i], psp[rt][i] * (float)sacc[i]);  // s_p sum p~' + n m~_p
        }
      }
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float mv = lo_half(vmr[j]), svj = hi_half(vmr[j]);
        uint32_t zj;
        if constexpr (!SE) zj = code_sum<BITS, VW>(vcr + j * VW);
        else if constexpr (SB == 1) zj = (vzr[j >> 2] >> (8 * (j & 3))) & 0xFFu;
        else zj = (vzr[j >> 1] >> (16 * (j & 1))) & 0xFFFFu;
        const float svz = svj * (float)zj;  // s_v sum v'
#pragma unroll
        for (int rt = 0; rt < GT; ++rt) {
          v4i acc = v4i{0, 0, 0, 0};
#pragma unroll
          for (int sl = 0; sl < TILES; ++sl) acc = mfma_i8(pa[rt][sl], unpack16<BITS>(vcr + j * VW + sl * SW), acc);
          // Eq. 4: s_p s_v D~ + (s_p sum p~' + n m~_p) m_v + m~_p s_v sum v'
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            float o = fmaf(psp[rt][i] * svj, (float)acc[i], o_acc[rt][j][i]);
            o = fmaf(pc1[rt][i], mv, o);
            o_acc[rt][j][i] = fmaf(pmt[rt][i], svz, o);
          }
          if constexpr (MODE == MODE_PV) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int gh = rt * 4 + i;
              if (gvalid && gh < Gl)
                a.dbg_prod[(((int64_t)s * Hq + hkv * G + head0 + gh) * (a.max_len / PI) + vkb) * D + 8 * col + j] =
                    acc[i] + kQoff * (int)zj;
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
  for (; si < nspan_full; si += kWaves) {
    SpanData<BITS, PI> cur;
    load_span(cur, t0 + si * SPAN, std::false_type{});
    compute_span(cur, t0 + si * SPAN, std::false_type{});
  }
  if (nspan - 1 >= nspan_full && (nspan - 1) % kWaves == wave) {
    SpanData<BITS, PI> last;
    load_span(last, t0 + (nspan - 1) * SPAN, std::true_type{});
    compute_span(last, t0 + (nspan - 1) * SPAN, std::true_type{});
  }
  if constexpr (MODE == MODE_QK) return;

  // this workgroup's heads, recomputed from the grid index instead of being kept live
  // across the span loop (where they would take scalar registers)
  int bx = (int)blockIdx.x;
  asm volatile("" : "+s"(bx));
  const int hg_e = a.head_groups == 1 ? 0 : bx / H, head0_e = HT * hg_e, Gl_e = min(HT, G - head0_e);

  // ---- wave result: O summed over the 4 lane groups (block slots), max and sum per head ----
#pragma unroll
  for (int rt = 0; rt < GT; ++rt) {
    float ov[8];
#pragma unroll
    for (int j = 0; j < 8; ++j)
      ov[j] = reduce_scatter4(o_acc[rt][j][0], o_acc[rt][j][1], o_acc[rt][j][2], o_acc[rt][j][3]);
    const float lsum = row16_sum(l_run[rt]);
    // lane group g writes head slot 4*rt + g: channels 8*col .. 8*col+7
    float* dst = &wl.mrg_o[rt * 4 + grp][8 * col];
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
  for (int idx = tid; idx < Gl_e * (D / 2); idx += 256) {
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
        o0 = fmaf(wl_all[w].mrg_o[gh][ch], wt, o0);
        o1 = fmaf(wl_all[w].mrg_o[gh][ch + 1], wt, o1);
      }
    }
    float* o = a.out + ((int64_t)s * Hq + hkv * G + head0_e + gh) * D + ch;
    if (MODE == MODE_PV) {
      o[0] = o0;
      o[1] = o1;
    } else if (nsplit == 1) {
      const float inv = 1.0f / lsum;
      o[0] = o0 * inv;
      o[1] = o1 * inv;
    } else {
      float* rec = a.partials + ((pair * a.splits + split) * G + head0_e + gh) * REC;
      // agent-coherent (write-through) stores: complete at the device's coherence
      // point once the wave's store counter drains
      if (ch == 0) {
        __hip_atomic_store(rec, mmax, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(rec + 1, lsum, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
      __hip_atomic_store(rec + 4 + ch, o0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(rec + 5 + ch, o1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
  if (MODE == MODE_ATTEND && nsplit > 1) {
    // The workgroup that finishes a sequence's last chunk merges all of them.
    __shared__ int last_chunk;
    __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): this wave's record stores are done
    __syncthreads();
    if (tid == 0) {
      // relaxed: the records are complete at the coherence point (vmcnt drained
      // above), and the merger reads them with agent-coherent loads
      const int done = __hip_atomic_fetch_add(&a.counters[pair * a.head_groups + hg_e], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      last_chunk = done == nsplit - 1;
    }
    __syncthreads();
    if (last_chunk) {
      merge_chunks(a, s, hkv, L, head0_e, Gl_e);
      if (tid == 0) __hip_atomic_store(&a.counters[pair * a.head_groups + hg_e], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

constexpr int64_t kFillWgSpans = 64;
constexpr int64_t kRaggedWgSpans = 48;
constexpr int64_t kMaxGridZ = 65535;

// Workgroups per (sequence, kv head, chunk): one per four query heads of the group.
// (A two-row-tile workgroup for groups of 8 needed about 230 VGPRs, two waves per
// SIMD, and was slower than two one-row-tile workgroups at three.)
static int head_groups_of(int G) { return (G + 3) / 4; }

// Workgroups per compute unit the grid is sized for.  The 2-bit, partition-32 kernel
// uses about 145 VGPRs, so three waves per SIMD are resident even though it is
// compiled for two (measured best on the 4K-context decode workload).
static int occupancy_of(const hack_kv_layout& lay) {
  return (lay.kv_bits == 2 && lay.partition == 32) ? 3 : 2;
}

DecodePlan plan_decode(const hack_kv_layout& lay, int batch, int num_q_heads, int max_len) {
  DecodePlan p{};
  const int64_t span = 4 * lay.partition;
  const int64_t pairs = (int64_t)batch * lay.num_kv_heads;
  const int64_t G = lay.num_kv_heads > 0 ? num_q_heads / lay.num_kv_heads : 0;
  const int64_t nhg = G > 0 ? head_groups_of((int)G) : 1;
  // one workgroup per compute unit and resident wave slot of a SIMD
  const int64_t per_cu = occupancy_of(lay);
  const int64_t target = kComputeUnits * per_cu;
  const int64_t spans_seq = ((int64_t)max_len + span - 1) / span;
  int64_t wg_spans = pairs > 0 ? (spans_seq * pairs * nhg + target - 1) / target : 1;
  if (wg_spans < 1) wg_spans = 1;
  // A chunk of at most kFillWgSpans spans bounds the time one workgroup holds a slot:
  // in a ragged batch the longest sequences then spread over more workgroups than an
  // even share of the mean length would give them.  When the even share at max_len is
  // more than twice that (a batch of many long sequences, several rounds of the
  // resident slots), the chunk is kRaggedWgSpans: on a batch of 1K-32K-token sequences
  // chunks of 40 / 48 / 56 / 64 spans took 289-290 / 287-289 / 288-290 / 293-295 us,
  // while a batch of equal lengths whose share is just above 64 spans loses a round to
  // the smaller chunk.  The grid's z extent (the splits) stays within its 65535 limit.
  if (wg_spans > 2 * kFillWgSpans) wg_spans = kRaggedWgSpans;
  else if (wg_spans > kFillWgSpans) wg_spans = kFillWgSpans;
  wg_spans = std::max<int64_t>(wg_spans, (spans_seq + kMaxGridZ - 1) / kMaxGridZ);
  p.chunk = (int)(wg_spans * span);
  p.splits = max_len > 0 ? (int)(((int64_t)max_len + p.chunk - 1) / p.chunk) : 1;
  finish_plan(p, pairs, G, nhg, lay.head_dim);
  return p;
}

template <int BITS, int PI, int GT, int MODE, int QP, bool SE, bool SR = false>
static hipError_t decode_impl(const DecodeArgs& a, int batch, hipStream_t stream) {
  dim3 grid((unsigned)(a.c.kv_heads * a.head_groups), (unsigned)batch, (unsigned)a.splits);
  hipLaunchKernelGGL((decode_kernel<BITS, PI, GT, MODE, QP, SE, SR>), grid, dim3(256), 0, stream, a);
  return hipGetLastError();
}

template <int BITS, int PI, int GT, int QP>
static hipError_t decode_mode(const DecodeArgs& a, int batch, int mode, hipStream_t stream) {
  if (a.c.sum_bytes == 0) {  // no cached sums: attention only (the exports need them)
    if (mode != MODE_ATTEND) return hipErrorInvalidValue;
    return a.stochastic ? decode_impl<BITS, PI, GT, MODE_ATTEND, QP, false, true>(a, batch, stream)
                        : decode_impl<BITS, PI, GT, MODE_ATTEND, QP, false>(a, batch, stream);
  }
  if (a.stochastic && mode == MODE_ATTEND) return decode_impl<BITS, PI, GT, MODE_ATTEND, QP, true, true>(a, batch, stream);
  if (a.stochastic && mode == MODE_QK) return decode_impl<BITS, PI, GT, MODE_QK, QP, true, true>(a, batch, stream);
  switch (mode) {
    case MODE_ATTEND: return decode_impl<BITS, PI, GT, MODE_ATTEND, QP, true>(a, batch, stream);
    case MODE_QK: return decode_impl<BITS, PI, GT, MODE_QK, QP, true>(a, batch, stream);
    case MODE_PV: return decode_impl<BITS, PI, GT, MODE_PV, QP, true>(a, batch, stream);
    default: return hipErrorInvalidValue;
  }
}

template <int BITS, int PI, int GT>
static hipError_t decode_qp(const DecodeArgs& a, int batch, int mode, hipStream_t stream) {
  if (a.qoff == 128) return decode_mode<BITS, PI, GT, 8>(a, batch, mode, stream);
  if (a.qoff == 8) return decode_mode<BITS, PI, GT, 4>(a, batch, mode, stream);
  return hipErrorInvalidValue;
}

template <int BITS, int PI>
static hipError_t decode_gt(const DecodeArgs& args, int batch, int mode, hipStream_t stream) {
  if (args.group < 1 || args.group > 8) return hipErrorInvalidValue;
  DecodeArgs a = args;
  a.head_groups = head_groups_of(a.group);
  return decode_qp<BITS, PI, 1>(a, batch, mode, stream);
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
