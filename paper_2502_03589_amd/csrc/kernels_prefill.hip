// Prefill attention on quantized Q/K/V/P (Sec. 5.3 with L_Q = L_KV; Eq. 2-4).
//
// One workgroup of eight 64-lane wavefronts per (32 query rows, up to 4 query heads
// of one kv group, sequence); wave w owns query head 4*hg + (w % 4) of the group and
// the 16 rows r0 + 16*(w / 4) ...  The workgroup walks the V blocks (PI tokens each)
// up to the causal diagonal:
//   staging  the 512 threads load block kb+1 (K codes unpacked to int8 in channel
//            order, V codes unpacked to int8 in the token order of the P.V operand,
//            per-token K and per-channel V metadata) into the other LDS buffer while
//            the waves compute block kb.
//   S^T = K'Q'^T  v_mfma_i32_16x16{32,64}_i8, one per (16-token tile, 16-row tile,
//            K partition): A = K codes (lane = token), B = Q codes minus 2^(b-1)
//            quantized in registers (lane = query row).  Lane (row n, group g) gets
//            tokens 4g..4g+3 of the tile for row n.  Eq. 4: the rank-1 terms
//            (m~_q s_k sum k' + R m_k, all partitions) are outer products of a
//            token-side and a row-side vector, so one v_mfma_f32_16x16x4_f32 per
//            tile forms them in the tile's layout (its four k slots: two partitions
//            x two terms); the VALU applies s_q s_k to each converted integer
//            product.  (The scale products as fp16 matrix-core products of exact
//            pieces left the time unchanged: the multiplies they remove came back
//            as operand assembly.)
//   softmax  online per row with a lazily raised reference max; causal mask.
//   P        8-bit per (row, V block) with round-to-nearest-even codes; the masked
//            zeros inside the diagonal block are quantized with it.  The lane's codes
//            are already the B operand of the P.V product (no transpose).
//   O^T = V'^T P'^T  one MFMA per (16-channel tile, row tile); an all-ones A gives
//            the P code sums.  Eq. 4: the VALU applies s_p s_v to each converted
//            integer product; the rank-1 terms of two V blocks share one
//            v_mfma_f32_16x16x4_f32 per 16 channels (k slots: two blocks x two
//            terms, against the cached V sums and minima).
//   open block  (len mod PI tokens) multiplied in fp16 with unquantized p.
#include <type_traits>

#include "hack_internal.hpp"

namespace hack {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef float v4f __attribute__((ext_vector_type(4)));

namespace {

constexpr int kRows = 32;        // query rows per workgroup (two 16-row MFMA tiles)
constexpr float kScale = 0.12751743074941640f;  // log2(e) / sqrt(128)
constexpr float kSlack = 8.0f;   // reference max raised only beyond this (log2 units)

template <int PI>
struct PrefillCfg {
  static constexpr int D = 128;
  static constexpr int P = D / PI;    // K partitions per token
  static constexpr int TL = PI / 16;  // 16-token tiles per block
  static constexpr int KSL = PI / 4;  // operand bytes per lane per MFMA (k-slots of a lane group)
  // LDS row strides of the unpacked K and V codes (bytes); the 32-byte pads were the
  // best of a padding sweep of LDS bank conflicts.  At partition 128 a 16-byte pad keeps
  // two workgroups' double-buffered 128-token stages within a compute unit's LDS.
  static constexpr int PAD = PI == 128 ? 16 : 32;
  static constexpr int KROW = D + PAD;
  static constexpr int VROW = PI + PAD;
};

// int8 MFMA with K = PI: 16x16x64 (16 bytes per lane) or 16x16x32 (8 bytes per lane).
template <int PI>
struct Op;
template <>
struct Op<64> {
  typedef v4i T;
  static __device__ __forceinline__ v4i mfma(v4i a, v4i b, v4i c) {
    return __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, c, 0, 0, 0);
  }
  static __device__ __forceinline__ v4i lds(const int8_t* p) {
    const int4 w = *reinterpret_cast<const int4*>(p);
    return v4i{w.x, w.y, w.z, w.w};
  }
  static __device__ __forceinline__ v4i ones() { return v4i{0x01010101, 0x01010101, 0x01010101, 0x01010101}; }
  static __device__ __forceinline__ v4i from(const uint32_t* w) {
    return v4i{(int)w[0], (int)w[1], (int)w[2], (int)w[3]};
  }
};
// partition 128: one partition is two 16x16x64 products over the lane's 32 bytes (bytes
// 0-15 of each operand against each other, then bytes 16-31), i.e. a 16x16x128 product
template <>
struct Op<128> {
  struct T {
    v4i lo, hi;
  };
  static __device__ __forceinline__ v4i mfma(T a, T b, v4i c) {
    c = __builtin_amdgcn_mfma_i32_16x16x64_i8(a.lo, b.lo, c, 0, 0, 0);
    return __builtin_amdgcn_mfma_i32_16x16x64_i8(a.hi, b.hi, c, 0, 0, 0);
  }
  static __device__ __forceinline__ T lds(const int8_t* p) {
    const int4 w0 = reinterpret_cast<const int4*>(p)[0], w1 = reinterpret_cast<const int4*>(p)[1];
    return T{v4i{w0.x, w0.y, w0.z, w0.w}, v4i{w1.x, w1.y, w1.z, w1.w}};
  }
  static __device__ __forceinline__ T ones() {
    const v4i o = v4i{0x01010101, 0x01010101, 0x01010101, 0x01010101};
    return T{o, o};
  }
  static __device__ __forceinline__ T from(const uint32_t* w) {
    return T{v4i{(int)w[0], (int)w[1], (int)w[2], (int)w[3]}, v4i{(int)w[4], (int)w[5], (int)w[6], (int)w[7]}};
  }
};
template <>
struct Op<32> {
  typedef long T;
  static __device__ __forceinline__ v4i mfma(long a, long b, v4i c) {
    return __builtin_amdgcn_mfma_i32_16x16x32_i8(a, b, c, 0, 0, 0);
  }
  static __device__ __forceinline__ long lds(const int8_t* p) { return *reinterpret_cast<const long*>(p); }
  static __device__ __forceinline__ long ones() { return 0x0101010101010101L; }
  static __device__ __forceinline__ long from(const uint32_t* w) {
    return (long)(((uint64_t)w[1] << 32) | (uint64_t)w[0]);
  }
};

// V metadata of one block, per channel: s_v, m_v, s_v*sum v' + PI*m_v.  Kept in a
// ring of three (block kb in slot kb % 3) apart from the two K/V code stages, so
// that a block's metadata outlives its codes by one block.
typedef float VMeta[3][128];

// LDS of one staged V block.
template <int PI>
struct Stage {
  int8_t k[PI][PrefillCfg<PI>::KROW];          // K codes, [token][channel]
  int8_t v[128][PrefillCfg<PI>::VROW];         // V codes, [channel][operand position]
  float km[PrefillCfg<PI>::P][3][PI];          // per token and partition: s_k, s_k*sum k', m_k
};

__device__ __forceinline__ v4f mfma_f32(float a, float b, v4f c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// Max / min / sum over the four lane groups (lanes l, l^16, l^32, l^48).
__device__ __forceinline__ float xg_max(float x) {
  auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float xg_min(float x) {
  auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = fminf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fminf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float xg_sum(float x) {
  auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}
__device__ __forceinline__ int xg_sum_i(int x) {
  auto a = __builtin_amdgcn_permlane32_swap((uint32_t)x, (uint32_t)x, false, false);
  x = (int)a[0] + (int)a[1];
  auto b = __builtin_amdgcn_permlane16_swap((uint32_t)x, (uint32_t)x, false, false);
  return (int)b[0] + (int)b[1];
}

struct PrefillArgs {
  CacheView c;
  const __half* q;   // [B][H_q][L][128]
  float* out;        // [B][H_q][L][128]
  int num_q_heads;
  int group;
  int head_groups;   // ceil(group / 4)
  int len;
  int causal;
  int nqb;           // query blocks of kRows rows
  float qmax;        // 2^b_QP - 1 of the transient Q and P codes (15 or 255)
  float inv_qmax;    // 1 / qmax
  int qoff;          // Q/P codes enter the signed int8 MFMA as code - qoff, qoff = 2^(b_QP - 1)
  float qoff_f;
  uint64_t key_q, key_p;  // stochastic rounding of the Q and P codes (streams 3 and 4)
};

// Staging of one V block by the 512 threads of the workgroup (threads 0-255: K,
// threads 256-511: V), in two phases so that the global loads of block kb+1 are in
// flight while block kb is computed: stage_load() fills registers, stage_store()
// unpacks them into LDS.
template <int BITS, int PI>
struct StageRegs {
  static constexpr int KW = (PI / 2) * BITS / 32;  // K code dwords per thread
  uint32_t w[KW];     // K codes (threads 0-255) or V codes (threads 256-511)
  uint32_t meta, sum; // K metadata of (token, partition) or V metadata of a channel
};

// Bytes of one cached code sum: 1 when b + log2(PI) <= 8, else 2 (Sec. 5.3).
template <int BITS, int PI>
constexpr int sum_bytes() {
  int need = BITS;
  for (int v = 1; v < PI; v <<= 1) ++need;
  return need <= 8 ? 1 : 2;
}

// Section bases of the block are wave-uniform; each thread adds a 32-bit offset
// that is recomputed from its index (not kept live across the block loop).
template <int BITS, int PI>
__device__ __forceinline__ void stage_load(const PrefillArgs& a, StageRegs<BITS, PI>& r, int s, int hkv, int kb,
                                           bool with_v) {
  constexpr int D = 128, P = PrefillCfg<PI>::P, SB = sum_bytes<BITS, PI>();
  constexpr int CPT = PI / 2, TPR = D / CPT;
  const CacheView& c = a.c;
  const int tid = threadIdx.x;
  const int64_t page = page_of(c, s, kb * PI);
  const int64_t krow0 = (page * c.kv_heads + hkv) * c.page_tokens + (int64_t)(kb * PI) % c.page_tokens;
  r.meta = 0u;
  r.sum = 0u;
#pragma unroll
  for (int i = 0; i < StageRegs<BITS, PI>::KW; ++i) r.w[i] = 0u;
  if (tid < 256) {
    // K codes: thread -> (token tid / TPR, PI/2 channels)
    const uint8_t* kc = c.k_codes + krow0 * (D * BITS / 8);
    uint32_t off = (uint32_t)((tid / TPR) * (D * BITS / 8) + (tid % TPR) * CPT * BITS / 8);
    asm volatile("" : "+v"(off));
    const uint32_t* src = reinterpret_cast<const uint32_t*>(kc + off);
#pragma unroll
    for (int i = 0; i < StageRegs<BITS, PI>::KW; ++i) r.w[i] = src[i];
    if (tid < PI * P) {  // K metadata: thread -> (token, partition); rows of P entries
      uint32_t mi = (uint32_t)tid;
      asm volatile("" : "+v"(mi));
      r.meta = reinterpret_cast<const uint32_t*>(reinterpret_cast<const uint8_t*>(c.k_meta) + krow0 * P * 4)[mi];
      const uint8_t* ks = c.k_sums + krow0 * P * SB;
      r.sum = SB == 1 ? (uint32_t)ks[mi] : (uint32_t)reinterpret_cast<const uint16_t*>(ks)[mi];
    }
  } else if (with_v) {
    const int64_t vb = (page * c.kv_heads + hkv) * (c.page_tokens / PI) + ((int64_t)(kb * PI) % c.page_tokens) / PI;
    const int vt = tid - 256;
    // V codes: two threads per channel, PI/2 tokens each
    const uint8_t* vc = c.v_codes + vb * D * (PI * BITS / 8);
    uint32_t off = (uint32_t)((vt >> 1) * (PI * BITS / 8) + (vt & 1) * (PI / 2) * BITS / 8);
    asm volatile("" : "+v"(off));
    const uint32_t* src = reinterpret_cast<const uint32_t*>(vc + off);
#pragma unroll
    for (int i = 0; i < StageRegs<BITS, PI>::KW; ++i) r.w[i] = src[i];
    if (vt < D) {
      uint32_t mi = (uint32_t)vt;
      asm volatile("" : "+v"(mi));
      r.meta = reinterpret_cast<const uint32_t*>(reinterpret_cast<const uint8_t*>(c.v_meta) + vb * D * 4)[mi];
      const uint8_t* vs = c.v_sums + vb * D * SB;
      r.sum = SB == 1 ? (uint32_t)vs[mi] : (uint32_t)reinterpret_cast<const uint16_t*>(vs)[mi];
    }
  }
}

// One dword of packed codes (element e in bits [BITS*e, BITS*e + BITS)) expanded to
// one byte per element in element order: masks pick every other (4-bit) or every
// fourth (2-bit) element, byte permutes interleave them back.
template <int BITS>
__device__ __forceinline__ void expand_word(uint32_t x, uint32_t* out) {
  if constexpr (BITS == 4) {
    const uint32_t lo = x & 0x0F0F0F0Fu, hi = (x >> 4) & 0x0F0F0F0Fu;  // elements 0,2,4,6 | 1,3,5,7
    out[0] = __builtin_amdgcn_perm(hi, lo, 0x05010400u);
    out[1] = __builtin_amdgcn_perm(hi, lo, 0x07030602u);
  } else {
    uint32_t d[4];  // d[k] byte j = element 4j + k
#pragma unroll
    for (int k = 0; k < 4; ++k) d[k] = (x >> (2 * k)) & 0x03030303u;
    const uint32_t a0 = __builtin_amdgcn_perm(d[1], d[0], 0x05010400u), a1 = __builtin_amdgcn_perm(d[1], d[0], 0x07030602u);
    const uint32_t b0 = __builtin_amdgcn_perm(d[3], d[2], 0x05010400u), b1 = __builtin_amdgcn_perm(d[3], d[2], 0x07030602u);
    out[0] = __builtin_amdgcn_perm(b0, a0, 0x05040100u);
    out[1] = __builtin_amdgcn_perm(b0, a0, 0x07060302u);
    out[2] = __builtin_amdgcn_perm(b1, a1, 0x05040100u);
    out[3] = __builtin_amdgcn_perm(b1, a1, 0x07060302u);
  }
}

template <int BITS, int PI>
__device__ __forceinline__ void stage_store(const StageRegs<BITS, PI>& r, Stage<PI>& st, VMeta& vm, bool with_v) {
  using C = PrefillCfg<PI>;
  constexpr int D = 128, P = C::P, KSL = C::KSL;
  constexpr int CPT = PI / 2, TPR = D / CPT;
  const int tid = threadIdx.x;
  if (tid < 256) {
    // K codes unpacked to int8 in channel order
    const int tt = tid / TPR, cb = (tid % TPR) * CPT;
    uint32_t* dst = reinterpret_cast<uint32_t*>(&st.k[tt][cb]);
    uint32_t bytes[CPT / 4];
#pragma unroll
    for (int i = 0; i < StageRegs<BITS, PI>::KW; ++i) expand_word<BITS>(r.w[i], bytes + i * (32 / BITS) / 4);
#pragma unroll
    for (int e4 = 0; e4 < CPT / 4; ++e4) dst[e4] = bytes[e4];
    if (tid < PI * P) {
      const int tt2 = tid / P, p = tid % P;
      const float mk = __half2float(__ushort_as_half((uint16_t)(r.meta & 0xFFFFu)));
      const float sk = __half2float(__ushort_as_half((uint16_t)(r.meta >> 16)));
      st.km[p][0][tt2] = sk;
      st.km[p][1][tt2] = sk * (float)r.sum;
      st.km[p][2][tt2] = mk;
    }
  } else if (with_v) {
    // V codes: token tau = 16*tl + 4*g + i goes to operand position g*KSL + 4*tl + i
    const int vt = tid - 256;
    const int ch = vt >> 1, half = vt & 1;
    uint32_t bytes[PI / 8];
#pragma unroll
    for (int i = 0; i < StageRegs<BITS, PI>::KW; ++i) expand_word<BITS>(r.w[i], bytes + i * (32 / BITS) / 4);
#pragma unroll
    for (int q4 = 0; q4 < PI / 8; ++q4) {
      const uint32_t v = bytes[q4];
      const int tau0 = half * (PI / 2) + 4 * q4;
      const int tl = tau0 >> 4, g = (tau0 >> 2) & 3;
      *reinterpret_cast<uint32_t*>(&st.v[ch][g * KSL + 4 * tl]) = v;
    }
    if (vt < D) {
      const float mv = __half2float(__ushort_as_half((uint16_t)(r.meta & 0xFFFFu)));
      const float sv = __half2float(__ushort_as_half((uint16_t)(r.meta >> 16)));
      vm[0][vt] = sv;
      vm[1][vt] = mv;
      vm[2][vt] = fmaf((float)PI, mv, sv * (float)r.sum);
    }
  }
}

}  // namespace

// Two workgroups per compute unit (four waves per SIMD, 128 VGPRs each; the two
// workgroups' LDS, about 78 KB each for partition 64, fits the 160 KB of a CU), so
// that one workgroup's block barrier and staging overlap the other's arithmetic
// (measured 1.61 -> 1.36-1.44 ms on the 8K causal prefill).
// SR: the Q and P codes are rounded stochastically (the layout's rounding mode).
// Partition 128 (eight 16-token tiles per V block, twice the scores and P codes per lane)
// needs more than 128 VGPRs: one workgroup per compute unit, two waves per SIMD.
template <int PI>
constexpr int prefill_waves_per_simd() {
  return PI == 128 ? 2 : 4;
}

template <int BITS, int PI, bool SR>
__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(prefill_waves_per_simd<PI>(),
                                                                     prefill_waves_per_simd<PI>()))) void prefill_kernel(PrefillArgs a) {
  using C = PrefillCfg<PI>;
  using OP = Op<PI>;
  typedef typename OP::T opT;
  constexpr int D = 128, P = C::P, TL = C::TL, KSL = C::KSL;

  __shared__ __attribute__((aligned(16))) Stage<PI> stages[2];
  __shared__ __attribute__((aligned(16))) VMeta vm_ring[3];

  const CacheView& c = a.c;
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const int col = lane & 15, grp = lane >> 4;
  const int s = blockIdx.z;
  const int hkv = blockIdx.y / a.head_groups, hg = blockIdx.y % a.head_groups;
  const int qb = a.causal ? (a.nqb - 1 - (int)blockIdx.x) : (int)blockIdx.x;  // heavy blocks first
  const int r0 = qb * kRows;
  const int L = a.len;
  const int gh = 4 * hg + (wave & 3);
  const bool head_ok = gh < a.group;
  const int hq = hkv * a.group + (head_ok ? gh : 0);
  const int row = r0 + 16 * (wave >> 2) + col;  // this lane's query row
  const int F = L / PI, T = L - F * PI;
  const int nblk_q = F + (T > 0 ? 1 : 0);
  const int nblk = a.causal ? min(nblk_q, (min(r0 + kRows, L) - 1) / PI + 1) : nblk_q;

  // ---- Q row: 8-bit codes per partition (float32 metadata), in MFMA operand layout ----
  opT qop[P];
  float sq[P], mq[P], rq[P];
  {
    const bool rv = head_ok && row < L;
    const __half* qrow = a.q + (((int64_t)s * a.num_q_heads + hq) * L + (rv ? row : 0)) * D;
#pragma unroll
    for (int p = 0; p < P; ++p) {
      float x[KSL];
      const int c0 = p * PI + grp * KSL;
#pragma unroll
      for (int e = 0; e < KSL; e += 2) {
        const float2 f = rv ? __half22float2(*reinterpret_cast<const __half2*>(qrow + c0 + e)) : float2{0.0f, 0.0f};
        x[e] = f.x;
        x[e + 1] = f.y;
      }
      float mn = x[0], mx = x[0];
#pragma unroll
      for (int e = 1; e < KSL; ++e) {
        mn = fminf(mn, x[e]);
        mx = fmaxf(mx, x[e]);
      }
      mn = xg_min(mn);
      mx = xg_max(mx);
      uint32_t w[KSL / 4];
      int csum = 0;
      float s32;
      {
#pragma clang fp contract(off)
        s32 = __fdiv_rn(__fsub_rn(mx, mn), a.qmax);
        const float r = s32 != 0.0f ? __fdiv_rn(1.0f, s32) : 0.0f;
#pragma unroll
        for (int e4 = 0; e4 < KSL / 4; ++e4) {
          uint32_t v = 0;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float t = __fmul_rn(__fsub_rn(x[4 * e4 + i], mn), r);
            int code = 0;
            if (s32 != 0.0f) {
              if constexpr (SR) {
                const float u = sr_threshold(a.key_q, qp_index(s, a.num_q_heads, hq, row, c0 + 4 * e4 + i));
                code = (int)round_stochastic(t, u, a.qmax);
              } else {
                code = (int)fminf(rintf(t), a.qmax);
              }
            }
            csum += code;
            v |= (uint32_t)((code - a.qoff) & 0xFF) << (8 * i);
          }
          w[e4] = v;
        }
      }
      csum = xg_sum_i(csum);
      qop[p] = OP::from(w);
      // Eq. 4 coefficients in log2 units: s_q, m~_q = m_q + qoff s_q, R = s_q sum q' + n m_q
      sq[p] = kScale * s32;
      mq[p] = kScale * (mn + a.qoff_f * s32);
      rq[p] = kScale * (s32 * (float)csum + (float)PI * mn);
    }
  }

  // Row-side operands of the outer-product MFMAs (lane (row, group g) supplies slot g):
  // rank terms of partitions 2m, 2m+1 as (m~_q, R, m~_q, R).
  float brank[(P + 1) / 2];
#pragma unroll
  for (int m = 0; m < (P + 1) / 2; ++m) {
    const int p = min(P - 1, 2 * m + (grp >> 1));
    const bool live = 2 * m + (grp >> 1) < P;
    brank[m] = live ? ((grp & 1) ? rq[p] : mq[p]) : 0.0f;
  }

  float m_ref = -INFINITY, l_run = 0.0f;
  v4f o[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) o[j] = v4f{0.0f, 0.0f, 0.0f, 0.0f};
  // P'V' rank-1 terms of two V blocks go into one f32 MFMA per 16 channels (its four
  // k slots: (s_p sum p~', m~_p) of each block against (m_v, s_v sum v' + n m_v)).
  // The row-side pair of the first block waits here; that block's stage stays
  // intact until the end of the next iteration.
  float rk_pz = 0.0f, rk_pm = 0.0f;
  int rk_blk = -1;
  auto rank_pair = [&](const VMeta& vm1, float pz1, float pm1, bool have1) __attribute__((always_inline)) {
    const VMeta& vm0 = vm_ring[rk_blk % 3];
    const float b = grp == 0 ? rk_pz : (grp == 1 ? rk_pm : (grp == 2 ? pz1 : pm1));
    const float* src = grp < 2 ? &vm0[1 + (grp & 1)][col] : &vm1[1 + (grp & 1)][col];
    const bool live = grp < 2 || have1;
#pragma unroll
    for (int j = 0; j < 8; ++j) o[j] = mfma_f32(live ? src[16 * j] : 0.0f, live ? b : 0.0f, o[j]);
    rk_blk = -1;
  };

  StageRegs<BITS, PI> sr;
  if (nblk > 0) {
    stage_load<BITS, PI>(a, sr, s, hkv, 0, 0 < F);
    stage_store<BITS, PI>(sr, stages[0], vm_ring[0], 0 < F);
  }
  __syncthreads();

  // One V block: quantized blocks run in the main loop; the fp16 open block (at most
  // one, the last) runs after it, so the loop body holds no branch on the block kind.
  auto block = [&](const int kb, auto tail_tag) __attribute__((always_inline)) {
    constexpr bool is_tail = decltype(tail_tag)::value;  // the fp16 open block
    Stage<PI>& st = stages[kb & 1];
    const VMeta& vmc = vm_ring[kb % 3];
    const bool next = kb + 1 < nblk;
    if (next) stage_load<BITS, PI>(a, sr, s, hkv, kb + 1, kb + 1 < F);
    const int tb0 = kb * PI;

    // ---------------- S^T tiles and Eq. 4 (lane: row `row`, tokens 16 tl + 4 grp + i) ----------------
    // masking is needed only in the block holding the length or this wave's diagonal
    const bool need_mask = is_tail || tb0 + PI > L || (a.causal && tb0 + PI - 1 > r0 + 16 * (wave >> 2));
    float sv[TL][4];
#pragma unroll
    for (int tl = 0; tl < TL; ++tl) {
      const int tt = 16 * tl + col;  // token of this lane's A-operand row
      // rank-1 terms summed over the partitions: token-side slot g = (partition, term)
      v4f s4 = v4f{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int m = 0; m < (P + 1) / 2; ++m) {
        const int p = min(P - 1, 2 * m + (grp >> 1));
        const bool live = 2 * m + (grp >> 1) < P;
        const float ak = live ? st.km[p][1 + (grp & 1)][tt] : 0.0f;  // s_k sum k' | m_k
        s4 = mfma_f32(ak, brank[m], s4);
      }
#pragma unroll
      for (int p = 0; p < P; ++p) {
        const opT ka = OP::lds(&st.k[tt][p * PI + grp * KSL]);
        const v4i acc = OP::mfma(ka, qop[p], v4i{0, 0, 0, 0});
        const float4 fk = *reinterpret_cast<const float4*>(&st.km[p][0][16 * tl + 4 * grp]);
        const float ksk[4] = {fk.x, fk.y, fk.z, fk.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) s4[i] = fmaf(sq[p] * ksk[i], (float)acc[i], s4[i]);  // s_q s_k C~
      }
      if (need_mask) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int tok = tb0 + 16 * tl + 4 * grp + i;
          const bool masked = tok >= L || (a.causal && tok > row);
          sv[tl][i] = masked ? -INFINITY : s4[i];
        }
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i) sv[tl][i] = s4[i];
      }
    }

    // ---------------- softmax and P codes ----------------
    float bmax = -INFINITY;
#pragma unroll
    for (int tl = 0; tl < TL; ++tl)
#pragma unroll
      for (int i = 0; i < 4; ++i) bmax = fmaxf(bmax, sv[tl][i]);
    bmax = xg_max(bmax);
    if (bmax > m_ref + kSlack || (m_ref == -INFINITY && bmax > -INFINITY)) {  // raise the reference max
      const float alpha = __builtin_amdgcn_exp2f(m_ref - bmax);
      l_run *= alpha;
#pragma unroll
      for (int j = 0; j < 8; ++j) o[j] *= alpha;
      rk_pz *= alpha;
      rk_pm *= alpha;
      m_ref = bmax;
    }
    float pt[TL][4];
    float pmin = INFINITY, lsum = 0.0f;
#pragma unroll
    for (int tl = 0; tl < TL; ++tl)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        pt[tl][i] = __builtin_amdgcn_exp2f(sv[tl][i] - m_ref);  // masked: exp2(-inf) = 0
        lsum += pt[tl][i];
        pmin = fminf(pmin, pt[tl][i]);
      }
    l_run += lsum;

    if constexpr (!is_tail) {
      pmin = xg_min(pmin);
      const float pmax = bmax > -INFINITY ? __builtin_amdgcn_exp2f(bmax - m_ref) : 0.0f;
      const float dp = pmax - pmin;
      const float r = dp > 0.0f ? a.qmax * __builtin_amdgcn_rcpf(dp) : 0.0f;
      // bytes code + 128 - qoff (an integer shift before rounding changes no code),
      // then bit 7 flipped: code - qoff as a signed byte
      const float bias = fmaf(-pmin, r, 128.0f - a.qoff_f);
      uint32_t w[TL];
#pragma unroll
      for (int tl = 0; tl < TL; ++tl) {
        uint32_t v = 0;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          if constexpr (SR) {
            const int tok = tb0 + 16 * tl + 4 * grp + i;
            const float u = sr_threshold(a.key_p, qp_index(s, a.num_q_heads, hq, row, tok));
            const float c = round_stochastic(fmaf(pt[tl][i], r, -pmin * r), u, a.qmax);
            v = __builtin_amdgcn_cvt_pk_u8_f32(c + (128.0f - a.qoff_f), i, v);
          } else {
            v = __builtin_amdgcn_cvt_pk_u8_f32(fmaf(pt[tl][i], r, bias), i, v);
          }
        }
        w[tl] = v ^ 0x80808080u;
      }
      const opT pop = OP::from(w);
      const float ps = dp * a.inv_qmax;        // s_p
      const float pm = pmin + a.qoff_f * ps;   // m~_p
      // sum of the signed codes of this row's block: all-ones A operand
      const v4i z = OP::mfma(OP::ones(), pop, v4i{0, 0, 0, 0});
      const float pz = ps * (float)z[0];       // s_p * sum p~'

      // ---------------- O^T += V'^T P'^T with Eq. 4 (lane: row, channels 16 j + 4 grp + i) ----------------
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int cc = 16 * j + col;  // channel of this lane's A-operand row
        const opT va = OP::lds(&st.v[cc][grp * KSL]);
        const v4i acc = OP::mfma(va, pop, v4i{0, 0, 0, 0});
        // (s_p sum p~') m_v + m~_p (s_v sum v' + n m_v), then s_p s_v D~
        const float4 fs = *reinterpret_cast<const float4*>(&vmc[0][16 * j + 4 * grp]);
        const float vs[4] = {fs.x, fs.y, fs.z, fs.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) o[j][i] = fmaf(ps * vs[i], (float)acc[i], o[j][i]);
      }
      if (rk_blk < 0) {
        rk_pz = pz;
        rk_pm = pm;
        rk_blk = kb;
      } else {
        rank_pair(vmc, pz, pm, true);
      }
    } else {
      if (rk_blk >= 0) rank_pair(vmc, 0.0f, 0.0f, false);
      // fp16 open block: O[row][ch] += sum_{t < T} p[row][t] v_t[ch] with unquantized p;
      // p[row][t] lives in lane (row, group (t mod 16) / 4) and is read by a lane shuffle
      const __half* vt = c.v_tail + (((int64_t)s * c.kv_heads + hkv) * PI) * D;
#pragma unroll
      for (int tl = 0; tl < TL; ++tl)
#pragma unroll
        for (int g = 0; g < 4; ++g)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int t = 16 * tl + 4 * g + i;
            const float pr = __shfl(pt[tl][i], col + 16 * g, 64);
            if (t < T) {
#pragma unroll
              for (int j = 0; j < 8; ++j) {
                const uint2 raw = *reinterpret_cast<const uint2*>(vt + (int64_t)t * D + 16 * j + 4 * grp);
                const float2 v01 = __half22float2(*reinterpret_cast<const __half2*>(&raw.x));
                const float2 v23 = __half22float2(*reinterpret_cast<const __half2*>(&raw.y));
                o[j][0] = fmaf(pr, v01.x, o[j][0]);
                o[j][1] = fmaf(pr, v01.y, o[j][1]);
                o[j][2] = fmaf(pr, v23.x, o[j][2]);
                o[j][3] = fmaf(pr, v23.y, o[j][3]);
              }
            }
          }
    }
    if (next) stage_store<BITS, PI>(sr, stages[(kb + 1) & 1], vm_ring[(kb + 1) % 3], kb + 1 < F);
    __syncthreads();  // stage kb+1 complete; stage kb free for kb+2
  };
  const int nq = min(nblk, F);
  for (int kb = 0; kb < nq; ++kb) block(kb, std::false_type{});
  if (nblk > nq) block(nq, std::true_type{});

  if (rk_blk >= 0) rank_pair(vm_ring[0], 0.0f, 0.0f, false);
  // ---- normalize and write O[row][16 j + 4 grp + i] ----
  const float lsum = xg_sum(l_run);
  if (head_ok && row < L) {
    const float inv = lsum > 0.0f ? 1.0f / lsum : 0.0f;
    float* dst = a.out + (((int64_t)s * a.num_q_heads + hq) * L + row) * D;
#pragma unroll
    for (int j = 0; j < 8; ++j)
      *reinterpret_cast<float4*>(dst + 16 * j + 4 * grp) =
          float4{o[j][0] * inv, o[j][1] * inv, o[j][2] * inv, o[j][3] * inv};
  }
}

template <int BITS, int PI>
static hipError_t prefill_impl(const PrefillArgs& a, int batch, bool stochastic, hipStream_t stream) {
  dim3 grid((unsigned)a.nqb, (unsigned)(a.c.kv_heads * a.head_groups), (unsigned)batch);
  if (stochastic)
    hipLaunchKernelGGL((prefill_kernel<BITS, PI, true>), grid, dim3(512), 0, stream, a);
  else
    hipLaunchKernelGGL((prefill_kernel<BITS, PI, false>), grid, dim3(512), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_prefill(const hack_kv_layout& lay, const CacheView& c, const __half* q, int num_q_heads,
                          int batch, int len, int causal, float* out, hipStream_t stream) {
  PrefillArgs a;
  a.c = c;
  a.q = q;
  a.out = out;
  a.num_q_heads = num_q_heads;
  a.group = num_q_heads / lay.num_kv_heads;
  a.head_groups = (a.group + 3) / 4;
  a.len = len;
  a.causal = causal;
  a.nqb = (len + kRows - 1) / kRows;
  a.key_q = lay.seed ^ (3ull << 56);
  a.key_p = lay.seed ^ (4ull << 56);
  const bool sr = lay.rounding == HACK_ROUND_STOCHASTIC;
  a.qmax = (float)((1 << lay.qp_bits) - 1);
  a.inv_qmax = 1.0f / a.qmax;
  a.qoff = 1 << (lay.qp_bits - 1);
  a.qoff_f = (float)a.qoff;
  switch (lay.kv_bits * 1000 + lay.partition) {
    case 2032: return prefill_impl<2, 32>(a, batch, sr, stream);
    case 2064: return prefill_impl<2, 64>(a, batch, sr, stream);
    case 4032: return prefill_impl<4, 32>(a, batch, sr, stream);
    case 4064: return prefill_impl<4, 64>(a, batch, sr, stream);
    case 2128: return prefill_impl<2, 128>(a, batch, sr, stream);
    case 4128: return prefill_impl<4, 128>(a, batch, sr, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace hack
