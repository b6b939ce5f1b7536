// Decode attention for a partition of 128 channels / tokens (Sec. 5.2, 5.3, Eq. 4).
//
// With Π = d = 128 every K row is one partition and every V block holds 128
// tokens, so Eq. 4's corrections are per (head, token) for Q'K' and per (head,
// channel) for P'V'.  The integer products run on the VALU's 4-way int8 dot
// instruction: the packed codes are split into byte planes with one shift and mask
// each, and the Q (or P) codes sit in LDS in the matching byte order, so no
// operand is transposed in registers.
//
// Attention only: a decode step appends the new token with the append kernel first.
// One workgroup of four waves per (sequence, kv head, up to four query heads,
// chunk).  A wave takes whole V blocks of the chunk: lane l scores tokens l and
// 64 + l of the block and accumulates output channels 2l and 2l + 1.  Chunks of a
// sequence are merged by the workgroup that finishes last, from records written
// with agent-coherent stores (the same protocol and workspace layout as the
// partition-32/64 kernels).
#include <algorithm>

#include "hack_device.hpp"
#include "hack_internal.hpp"

namespace hack {
namespace {

constexpr int kD = 128;       // head dimension
constexpr int kBlk = 128;     // partition: channels per K partition, tokens per V block
constexpr int kWaves128 = 4;  // waves per workgroup
constexpr int kHeads = 4;     // query heads per workgroup
constexpr float kLog2Scale = 0.12751743074941640f;  // log2(e) / sqrt(128): scores in log2 units
constexpr float kRaiseSlack = 8.0f;                 // the reference max is raised lazily
constexpr int kCUs = 256;                           // compute units of an MI355X

// Workgroups per compute unit the register budget allows (the grid is sized for it).
template <int BITS>
constexpr int occupancy128() { return BITS == 2 ? 4 : 2; }

__device__ __forceinline__ float f16_lo(uint32_t w) { return __half2float(__ushort_as_half((uint16_t)(w & 0xFFFFu))); }
__device__ __forceinline__ float f16_hi(uint32_t w) { return __half2float(__ushort_as_half((uint16_t)(w >> 16))); }

// Wave-wide reductions: a row of 16 lanes by DPP rotates, then the four row results
// read into scalar registers (the result is wave-uniform).
__device__ __forceinline__ float lane_f(float x, int l) { return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), l)); }
__device__ __forceinline__ float wave_max(float x) {
  x = row16_max(x);
  return fmaxf(fmaxf(lane_f(x, 0), lane_f(x, 16)), fmaxf(lane_f(x, 32), lane_f(x, 48)));
}
__device__ __forceinline__ float wave_min(float x) {
  x = row16_min(x);
  return fminf(fminf(lane_f(x, 0), lane_f(x, 16)), fminf(lane_f(x, 32), lane_f(x, 48)));
}
__device__ __forceinline__ float wave_sum(float x) {
  x = row16_sum(x);
  return (lane_f(x, 0) + lane_f(x, 16)) + (lane_f(x, 32) + lane_f(x, 48));
}
__device__ __forceinline__ int wave_sum_i(int x) {
  x = row16_sum_i(x);
  return (__builtin_amdgcn_readlane(x, 0) + __builtin_amdgcn_readlane(x, 16)) +
         (__builtin_amdgcn_readlane(x, 32) + __builtin_amdgcn_readlane(x, 48));
}

// Byte position, inside a 128-byte operand, of element e (a channel of Q, a token
// of P) so that operand dword (w * NJ + j) pairs with byte plane j of code dword w:
// plane j of a dword holding PER codes LSB-first has element PER*w + NJ*m + j in
// byte m.
template <int BITS>
__device__ __forceinline__ int operand_pos(int e) {
  constexpr int PER = 32 / BITS, NJ = 8 / BITS;
  const int w = e / PER, i = e % PER;
  return ((w * NJ + (i % NJ)) << 2) + i / NJ;
}

// Integer products of two code rows (two K tokens, or two V channels) with the
// operands of up to four heads: acc[h][r] += sum over the code dwords of row r of
// (byte planes of the dword) . (operand dwords of head h for that dword).  Dword w
// outermost, so only its planes and one operand slice are live at a time.  The codes
// are in [0, 2^b - 1]; the operands hold code - offset as signed bytes.
template <int BITS, int N>
__device__ __forceinline__ void dot_rows(const uint32_t* x0, const uint32_t* x1, const int* op_lds, int op_stride,
                                         int nheads, int (&acc)[4][2]) {
  constexpr int NJ = 8 / BITS;
  constexpr uint32_t MASK = BITS == 2 ? 0x03030303u : 0x0F0F0F0Fu;
#pragma unroll
  for (int w = 0; w < N; ++w) {
    int b0[NJ], b1[NJ];
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      b0[j] = (int)((x0[w] >> (BITS * j)) & MASK);
      b1[j] = (int)((x1[w] >> (BITS * j)) & MASK);
    }
#pragma unroll
    for (int h = 0; h < 4; ++h) {
      if (h >= nheads) break;
      int q[NJ];
      if constexpr (NJ == 4) {
        const int4 v = *reinterpret_cast<const int4*>(op_lds + h * op_stride + w * NJ);
        q[0] = v.x; q[1] = v.y; q[2] = v.z; q[3] = v.w;
      } else {
        const int2 v = *reinterpret_cast<const int2*>(op_lds + h * op_stride + w * NJ);
        q[0] = v.x; q[1] = v.y;
      }
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        acc[h][0] = __builtin_amdgcn_sdot4(b0[j], q[j], acc[h][0], false);
        acc[h][1] = __builtin_amdgcn_sdot4(b1[j], q[j], acc[h][1], false);
      }
    }
  }
}

// sum of the codes packed in x[0..N): population counts of the bit planes (2-bit
// codes) or the 4-bit dot instruction against ones (4-bit codes)
template <int BITS, int N>
__device__ __forceinline__ uint32_t sum_codes(const uint32_t* x) {
  uint32_t s = 0;
#pragma unroll
  for (int w = 0; w < N; ++w) {
    if constexpr (BITS == 2) {
      s += __popc(x[w] & 0x55555555u) + 2u * __popc(x[w] & 0xAAAAAAAAu);
    } else {
      s = __builtin_amdgcn_udot8(x[w], 0x11111111u, s, false);  // eight 4-bit codes times one
    }
  }
  return s;
}

// two floats as one 8-byte word (first in the low half) and back
__device__ __forceinline__ uint64_t pack2(float lo, float hi) {
  return (uint64_t)__float_as_uint(lo) | ((uint64_t)__float_as_uint(hi) << 32);
}
__device__ __forceinline__ void unpack2(uint64_t w, float& lo, float& hi) {
  lo = __uint_as_float((uint32_t)w);
  hi = __uint_as_float((uint32_t)(w >> 32));
}

template <int N>
__device__ __forceinline__ void load_dwords(const uint8_t* p, uint32_t* x) {
#pragma unroll
  for (int i = 0; i < N / 4; ++i) {
    const uint4 v = reinterpret_cast<const uint4*>(p)[i];
    x[4 * i] = v.x; x[4 * i + 1] = v.y; x[4 * i + 2] = v.z; x[4 * i + 3] = v.w;
  }
}

template <int BITS, bool SE, bool SR>
__global__ __launch_bounds__(256, occupancy128<BITS>()) void decode128_kernel(DecodeArgs a) {
  constexpr int KD = 4 * BITS;  // code dwords per K row, and per V channel of a block
  constexpr int REC = 4 + kD;   // chunk record: max, sum, 2 pad, O

  __shared__ __attribute__((aligned(16))) int q_op[kHeads][32];        // Q codes - qoff, operand order
  __shared__ float q_m[kHeads][3];                                       // s_q, m~_q, R (log2 units)
  __shared__ __attribute__((aligned(16))) int p_op[kWaves128][kHeads][32];  // P codes - qoff, operand order
  __shared__ float p_tail[kWaves128][kHeads][kBlk];                      // unquantized p of an fp16 open block
  __shared__ float w_o[kWaves128][kHeads][kD];
  __shared__ float w_ml[kWaves128][kHeads][2];
  __shared__ int last_chunk;

  const CacheView& c = a.c;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int G = a.group, Hq = a.num_q_heads, H = c.kv_heads;
  const bool one_group = a.head_groups == 1;
  const int s = blockIdx.y, split = blockIdx.z;
  const int hkv = one_group ? (int)blockIdx.x : (int)blockIdx.x % H, hg = one_group ? 0 : (int)blockIdx.x / H;
  const int head0 = kHeads * hg, Gl = min(kHeads, G - head0);
  const float qmax = a.qmax;
  const int qoff = a.qoff;

  // wave w quantizes head slot w; its query load is issued before the length's
  const uint32_t qraw =
      wave < Gl ? reinterpret_cast<const uint32_t*>(a.q + ((int64_t)s * Hq + hkv * G + head0 + wave) * kD)[lane] : 0u;
  // lengths outside [0, max_len] break the caller contract; clamp so that every
  // access stays inside the cache and the workspace
  const int L = max(0, min(a.lens[s], a.max_len));
  const int t0 = split * a.chunk;
  if (t0 >= L) {
    if (split == 0)  // empty sequence: zeros
      for (int i = tid; i < Gl * kD; i += 256) a.out[((int64_t)s * Hq + hkv * G + head0) * kD + i] = 0.0f;
    return;
  }
  const int t1 = min(L, t0 + a.chunk);
  const int nsplit = (L + a.chunk - 1) / a.chunk;
  const int F = L / kBlk, T = L - F * kBlk;
  const bool codes_open = a.tail_requant != 0;  // the open V block is read from its codes

  // ---- Q: one partition of 128 channels per head, b_QP-bit codes (Sec. 5.1, 5.2) ----
  {
    const bool real = wave < Gl;
    const int hq = hkv * G + head0 + wave;
    float x0 = 0.0f, x1 = 0.0f;
    if (real) {
      const float2 f = __half22float2(*reinterpret_cast<const __half2*>(&qraw));
      x0 = f.x;
      x1 = f.y;
    }
    const float mn = wave_min(fminf(x0, x1)), mx = wave_max(fmaxf(x0, x1));
    float sq, c0 = 0.0f, c1 = 0.0f;
    {
#pragma clang fp contract(off)
      sq = __fdiv_rn(__fsub_rn(mx, mn), qmax);
      if (sq != 0.0f) {
        const float r = __fdiv_rn(1.0f, sq);
        const float u0 = __fmul_rn(__fsub_rn(x0, mn), r), u1 = __fmul_rn(__fsub_rn(x1, mn), r);
        if constexpr (SR) {
          c0 = round_stochastic(u0, sr_threshold(a.key_q, qp_index(s, Hq, hq, 0, 2 * lane)), qmax);
          c1 = round_stochastic(u1, sr_threshold(a.key_q, qp_index(s, Hq, hq, 0, 2 * lane + 1)), qmax);
        } else {
          c0 = fminf(rintf(u0), qmax);
          c1 = fminf(rintf(u1), qmax);
        }
      }
    }
    const int csum = wave_sum_i((int)c0 + (int)c1);
    int8_t* qb = reinterpret_cast<int8_t*>(&q_op[wave][0]);
    qb[operand_pos<BITS>(2 * lane)] = real ? (int8_t)((int)c0 - qoff) : (int8_t)0;
    qb[operand_pos<BITS>(2 * lane + 1)] = real ? (int8_t)((int)c1 - qoff) : (int8_t)0;
    if (lane == 0) {
      // s_q, m~_q = m_q + qoff s_q and R = s_q sum q' + 128 m_q, scaled to log2 units
      q_m[wave][0] = real ? kLog2Scale * sq : 0.0f;
      q_m[wave][1] = real ? kLog2Scale * (mn + (float)qoff * sq) : 0.0f;
      q_m[wave][2] = real ? kLog2Scale * (sq * (float)csum + (float)kBlk * mn) : 0.0f;
    }
  }
  __syncthreads();

  float m_ref[kHeads], l_run[kHeads], o0[kHeads], o1[kHeads];
#pragma unroll
  for (int h = 0; h < kHeads; ++h) {
    m_ref[h] = -INFINITY;
    l_run[h] = 0.0f;
    o0[h] = 0.0f;
    o1[h] = 0.0f;
  }
  const int nblk = (t1 - t0 + kBlk - 1) / kBlk;
  int8_t* pb = reinterpret_cast<int8_t*>(&p_op[wave][0][0]);

  // K rows of tokens lane and 64 + lane of the block starting at token tbx.  With
  // cached sums a wave requests its next block's rows as soon as the current scores
  // are computed, so they arrive while it runs the softmax and P'V' of the current
  // block (1-3% faster); rebuilding the sums from the codes keeps more registers live
  // there, and the prefetch would spill, so that variant loads each block's rows at
  // its start.
  uint32_t kc[2][KD], km[2], kz[2];
  auto load_k = [&](int tbx) __attribute__((always_inline)) {
    const int64_t krow = k_row(c, s, hkv, tbx);  // a block never crosses a page
#pragma unroll
    for (int r = 0; r < 2; ++r) {
      const int e = 64 * r + lane;
      if (tbx + e < L) {
        load_dwords<KD>(c.k_codes + (krow + e) * (kD * BITS / 8), kc[r]);
        km[r] = reinterpret_cast<const uint32_t*>(c.k_meta)[krow + e];
        kz[r] = SE ? (uint32_t)reinterpret_cast<const uint16_t*>(c.k_sums)[krow + e] : 0u;
      } else {
#pragma unroll
        for (int w = 0; w < KD; ++w) kc[r][w] = 0u;
        km[r] = 0u;
        kz[r] = 0u;
      }
    }
  };
  if constexpr (SE) {
    if (wave < nblk) load_k(t0 + wave * kBlk);
  }

  for (int bi = wave; bi < nblk; bi += kWaves128) {
    const int tb = t0 + bi * kBlk;  // chunks start at multiples of the block
    const int kb = tb / kBlk;
    const bool vq = kb < F || (codes_open && kb == F && T > 0);  // V read from codes
    const bool v16 = !codes_open && kb == F && T > 0;            // fp16 open block
    const int nb = kb < F ? kBlk : T;                            // tokens of the block
    // a block never crosses a page (pages hold whole decode spans of 4 blocks)
    const int64_t vblk = v_block<kBlk>(c, s, hkv, tb);
    if constexpr (!SE) load_k(tb);

    // ---- Q'K' and Eq. 4 per (head, token) ----
    float sc[kHeads][2];
    float mk[2], sk[2], zk[2];
#pragma unroll
    for (int r = 0; r < 2; ++r) {
      mk[r] = f16_lo(km[r]);
      sk[r] = f16_hi(km[r]);
      zk[r] = (float)(SE ? kz[r] : sum_codes<BITS, KD>(kc[r]));
    }
    int dq[kHeads][2] = {{0, 0}, {0, 0}, {0, 0}, {0, 0}};
    dot_rows<BITS, KD>(kc[0], kc[1], &q_op[0][0], 32, Gl, dq);
    if constexpr (SE) {
      if (bi + kWaves128 < nblk) load_k(tb + kWaves128 * kBlk);  // the K registers are free now
    }
#pragma unroll
    for (int h = 0; h < kHeads; ++h) {
      if (h >= Gl) break;
      const float sqs = q_m[h][0], mqs = q_m[h][1], rq = q_m[h][2];
#pragma unroll
      for (int r = 0; r < 2; ++r) {
        // s_q s_k D~ + m~_q s_k sum k' + R m_k
        const float v = fmaf(sk[r], fmaf(sqs, (float)dq[h][r], mqs * zk[r]), rq * mk[r]);
        sc[h][r] = tb + 64 * r + lane < L ? v : -INFINITY;
      }
    }

    // ---- softmax with a lazily raised reference max; P codes per (head, block) ----
    float ps[kHeads], pm[kHeads];
    int pz[kHeads];  // wave-uniform integer sums stay in scalar registers
#pragma unroll
    for (int h = 0; h < kHeads; ++h) {
      if (h >= Gl) break;
      const float bmax = wave_max(fmaxf(sc[h][0], sc[h][1]));
      if (bmax > m_ref[h] + kRaiseSlack || m_ref[h] == -INFINITY) {
        const float f = m_ref[h] == -INFINITY ? 0.0f : __builtin_amdgcn_exp2f(m_ref[h] - bmax);
        l_run[h] *= f;
        o0[h] *= f;
        o1[h] *= f;
        m_ref[h] = bmax;
      }
      const float mr = m_ref[h];
      const float p0 = __builtin_amdgcn_exp2f(sc[h][0] - mr), p1 = __builtin_amdgcn_exp2f(sc[h][1] - mr);
      l_run[h] += p0 + p1;
      ps[h] = 0.0f;
      pm[h] = 0.0f;
      pz[h] = 0;
      if (vq) {
        const bool ok0 = tb + lane < L, ok1 = tb + 64 + lane < L;
        const float bmin = wave_min(fminf(ok0 ? sc[h][0] : INFINITY, ok1 ? sc[h][1] : INFINITY));
        const float pmax = __builtin_amdgcn_exp2f(bmax - mr), pmin = __builtin_amdgcn_exp2f(bmin - mr);
        const float dp = pmax - pmin;
        const float r = dp > 0.0f ? qmax * __builtin_amdgcn_rcpf(dp) : 0.0f;
        const float bias = -pmin * r;
        int cd[2];
#pragma unroll
        for (int k = 0; k < 2; ++k) {
          const float pk = k == 0 ? p0 : p1;
          const bool ok = k == 0 ? ok0 : ok1;
          uint32_t code;
          if constexpr (SR) {
            const float u = sr_threshold(a.key_p, qp_index(s, Hq, hkv * G + head0 + h, 0, tb + 64 * k + lane));
            code = (uint32_t)round_stochastic(fmaf(pk, r, bias), u, qmax);
          } else {
            code = __builtin_amdgcn_cvt_pk_u8_f32(fmaf(pk, r, bias), 0, 0u);
          }
          cd[k] = ok ? (int)code - qoff : 0;
          pb[h * 128 + operand_pos<BITS>(64 * k + lane)] = (int8_t)cd[k];
        }
        ps[h] = dp * a.inv_qmax;
        pm[h] = pmin;
        pz[h] = wave_sum_i(cd[0] + cd[1]);  // sum of p~' = p' - qoff over the block
      } else if (v16) {
        p_tail[wave][h][lane] = p0;
        p_tail[wave][h][64 + lane] = p1;
      }
    }
    // P codes written above by every lane are read back whole by each lane
    __builtin_amdgcn_s_waitcnt(0xC07F);
    __builtin_amdgcn_wave_barrier();

    // ---- P'V' and Eq. 4 per (head, channel) ----
    // V channels 2 lane, 2 lane + 1, loaded only now: their registers are not live
    // during Q'K' and softmax (≈ 20 fewer VGPRs; the other waves of the SIMD cover
    // the load; 6-9% faster than loading them with K)
    uint32_t vc[2 * KD], vm[2] = {0u, 0u}, vz = 0u;
    if (vq) {
      load_dwords<2 * KD>(c.v_codes + (vblk * kD + 2 * lane) * (kBlk * BITS / 8), vc);
      const uint2 m2 = *reinterpret_cast<const uint2*>(reinterpret_cast<const uint32_t*>(c.v_meta) + vblk * kD + 2 * lane);
      vm[0] = m2.x;
      vm[1] = m2.y;
      if constexpr (SE) vz = *reinterpret_cast<const uint32_t*>(c.v_sums + (vblk * kD + 2 * lane) * 2);
    } else {
#pragma unroll
      for (int w = 0; w < 2 * KD; ++w) vc[w] = 0u;
    }
    if (vq) {
      float mv[2], sv[2], vbar[2];
#pragma unroll
      for (int k = 0; k < 2; ++k) {
        mv[k] = f16_lo(vm[k]);
        sv[k] = f16_hi(vm[k]);
        const uint32_t z = SE ? ((vz >> (16 * k)) & 0xFFFFu) : sum_codes<BITS, KD>(vc + k * KD);
        vbar[k] = fmaf((float)nb, mv[k], sv[k] * (float)z);  // s_v sum v' + n m_v
      }
      int dv[kHeads][2] = {{0, 0}, {0, 0}, {0, 0}, {0, 0}};
      dot_rows<BITS, KD>(vc, vc + KD, &p_op[wave][0][0], 32, Gl, dv);
#pragma unroll
      for (int h = 0; h < kHeads; ++h) {
        if (h >= Gl) break;
        // s_p s_v D~ + (s_p sum p~') m_v + m~_p (s_v sum v' + n m_v)
        const float spz = ps[h] * (float)pz[h], mtp = fmaf((float)qoff, ps[h], pm[h]);
        o0[h] += fmaf(ps[h] * sv[0], (float)dv[h][0], fmaf(spz, mv[0], mtp * vbar[0]));
        o1[h] += fmaf(ps[h] * sv[1], (float)dv[h][1], fmaf(spz, mv[1], mtp * vbar[1]));
      }
    } else if (v16) {
      // fp16 open block: sum_t p_t v_t with unquantized p.  The lane's byte offset is
      // opaque to the compiler, so its address is formed here rather than hoisted
      // out of the block loop (where it would stay live, and spill, for every wave).
      uint32_t lo = 4u * (uint32_t)lane;
      asm volatile("" : "+v"(lo));
      const uint8_t* vt = reinterpret_cast<const uint8_t*>(c.v_tail + ((int64_t)s * H + hkv) * kBlk * kD) + lo;
      for (int e = 0; e < T; ++e) {
        const float2 v = __half22float2(*reinterpret_cast<const __half2*>(vt + (uint32_t)e * (kD * 2)));
#pragma unroll
        for (int h = 0; h < kHeads; ++h) {
          if (h >= Gl) break;
          const float p = p_tail[wave][h][e];
          o0[h] = fmaf(p, v.x, o0[h]);
          o1[h] = fmaf(p, v.y, o1[h]);
        }
      }
    }
    // the next block rewrites this wave's LDS
    __builtin_amdgcn_s_waitcnt(0xC07F);
    __builtin_amdgcn_wave_barrier();
  }

  // ---- wave results, then the four waves merged: thread (head, channel pair) ----
#pragma unroll
  for (int h = 0; h < kHeads; ++h) {
    const float ls = wave_sum(l_run[h]);
    w_o[wave][h][2 * lane] = o0[h];
    w_o[wave][h][2 * lane + 1] = o1[h];
    if (lane == 0) {
      w_ml[wave][h][0] = m_ref[h];
      w_ml[wave][h][1] = h < Gl ? ls : 0.0f;
    }
  }
  __syncthreads();
  const int64_t pair = (int64_t)s * H + hkv;
  for (int idx = tid; idx < Gl * (kD / 2); idx += 256) {
    const int gh = idx / (kD / 2), ch = 2 * (idx % (kD / 2));
    float mmax = -INFINITY;
#pragma unroll
    for (int w = 0; w < kWaves128; ++w)
      if (w_ml[w][gh][1] > 0.0f) mmax = fmaxf(mmax, w_ml[w][gh][0]);
    float lsum = 0.0f, x0 = 0.0f, x1 = 0.0f;
#pragma unroll
    for (int w = 0; w < kWaves128; ++w) {
      if (w_ml[w][gh][1] > 0.0f) {
        const float wt = __builtin_amdgcn_exp2f(w_ml[w][gh][0] - mmax);
        lsum = fmaf(w_ml[w][gh][1], wt, lsum);
        x0 = fmaf(w_o[w][gh][ch], wt, x0);
        x1 = fmaf(w_o[w][gh][ch + 1], wt, x1);
      }
    }
    if (nsplit == 1) {
      float* o = a.out + ((int64_t)s * Hq + hkv * G + head0 + gh) * kD + ch;
      const float inv = 1.0f / lsum;
      o[0] = x0 * inv;
      o[1] = x1 * inv;
    } else {
      // agent-coherent (write-through) 8-byte stores, complete once the store counter
      // drains; a record is 8-byte aligned (528 bytes each from a 256-byte base)
      uint64_t* rec = reinterpret_cast<uint64_t*>(a.partials + ((pair * a.splits + split) * G + head0 + gh) * REC);
      if (ch == 0) __hip_atomic_store(rec, pack2(mmax, lsum), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(rec + 2 + ch / 2, pack2(x0, x1), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
  if (nsplit == 1) return;
  // the workgroup that finishes a sequence's last chunk merges all of them
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): this wave's record stores are done
  __syncthreads();
  if (tid == 0) {
    const int done = __hip_atomic_fetch_add(&a.counters[pair * a.head_groups + hg], 1, __ATOMIC_RELAXED,
                                            __HIP_MEMORY_SCOPE_AGENT);
    last_chunk = done == nsplit - 1;
  }
  __syncthreads();
  if (!last_chunk) return;
  // one pass with a running max; the records of eight chunks are requested together
  // so the merge waits on memory once per eight chunks
  for (int idx = tid; idx < Gl * (kD / 2); idx += 256) {
    const int gh = idx / (kD / 2), ch = 2 * (idx % (kD / 2));
    float mrun = -INFINITY, lsum = 0.0f, x0 = 0.0f, x1 = 0.0f;
    for (int sp0 = 0; sp0 < nsplit; sp0 += 8) {
      float ms[8], ls[8], xa[8], xb[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        if (sp0 + u < nsplit) {
          const uint64_t* rec =
              reinterpret_cast<const uint64_t*>(a.partials + ((pair * a.splits + sp0 + u) * G + head0 + gh) * REC);
          unpack2(__hip_atomic_load(rec, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT), ms[u], ls[u]);
          unpack2(__hip_atomic_load(rec + 2 + ch / 2, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT), xa[u], xb[u]);
        } else {
          ms[u] = -INFINITY;
          ls[u] = 0.0f;
          xa[u] = 0.0f;
          xb[u] = 0.0f;
        }
      }
      float mn = mrun;
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (ls[u] > 0.0f) mn = fmaxf(mn, ms[u]);
      const float wa = mrun == -INFINITY ? 0.0f : __builtin_amdgcn_exp2f(mrun - mn);
      lsum *= wa;
      x0 *= wa;
      x1 *= wa;
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const float wb = ls[u] > 0.0f ? __builtin_amdgcn_exp2f(ms[u] - mn) : 0.0f;
        lsum = fmaf(ls[u], wb, lsum);
        x0 = fmaf(xa[u], wb, x0);
        x1 = fmaf(xb[u], wb, x1);
      }
      mrun = mn;
    }
    float* o = a.out + ((int64_t)s * Hq + hkv * G + head0 + gh) * kD + ch;
    const float inv = 1.0f / lsum;
    o[0] = x0 * inv;
    o[1] = x1 * inv;
  }
  if (tid == 0)
    __hip_atomic_store(&a.counters[pair * a.head_groups + hg], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

template <int BITS, bool SE, bool SR>
hipError_t launch128(const DecodeArgs& a, int batch, hipStream_t stream) {
  dim3 grid((unsigned)(a.c.kv_heads * a.head_groups), (unsigned)batch, (unsigned)a.splits);
  hipLaunchKernelGGL((decode128_kernel<BITS, SE, SR>), grid, dim3(256), 0, stream, a);
  return hipGetLastError();
}

template <int BITS>
hipError_t launch128_bits(const DecodeArgs& a, int batch, hipStream_t stream) {
  const bool se = a.c.sum_bytes != 0;
  if (a.stochastic) return se ? launch128<BITS, true, true>(a, batch, stream) : launch128<BITS, false, true>(a, batch, stream);
  return se ? launch128<BITS, true, false>(a, batch, stream) : launch128<BITS, false, false>(a, batch, stream);
}

}  // namespace

// A chunk is a whole number of 4-block spans (one block per wave); chunks per
// sequence are chosen so that the grid fills every compute unit at the kernel's
// occupancy, at most 64 spans per chunk, and the grid's z extent stays <= 65535.
DecodePlan plan_decode128(const hack_kv_layout& lay, int batch, int num_q_heads, int max_len) {
  DecodePlan p{};
  const int64_t span = (int64_t)kWaves128 * kBlk;
  const int64_t pairs = (int64_t)batch * lay.num_kv_heads;
  const int64_t G = lay.num_kv_heads > 0 ? num_q_heads / lay.num_kv_heads : 0;
  const int64_t nhg = G > 0 ? (G + kHeads - 1) / kHeads : 1;
  const int64_t target = (int64_t)kCUs * (lay.kv_bits == 2 ? occupancy128<2>() : occupancy128<4>());
  const int64_t spans_seq = ((int64_t)max_len + span - 1) / span;
  int64_t wg_spans = pairs > 0 ? (spans_seq * pairs * nhg + target - 1) / target : 1;
  wg_spans = std::min<int64_t>(std::max<int64_t>(wg_spans, 1), 64);
  wg_spans = std::max<int64_t>(wg_spans, (spans_seq + 65534) / 65535);
  p.chunk = (int)(wg_spans * span);
  p.splits = max_len > 0 ? (int)(((int64_t)max_len + p.chunk - 1) / p.chunk) : 1;
  finish_plan(p, pairs, G, nhg, kD);
  return p;
}

hipError_t launch_decode128(const hack_kv_layout& lay, const DecodeArgs& args, int batch, hipStream_t stream) {
  if (lay.partition != kBlk || lay.head_dim != kD || args.group < 1 || args.group > 8) return hipErrorInvalidValue;
  DecodeArgs a = args;
  a.head_groups = (a.group + kHeads - 1) / kHeads;
  switch (lay.kv_bits) {
    case 2: return launch128_bits<2>(a, batch, stream);
    case 4: return launch128_bits<4>(a, batch, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace hack
