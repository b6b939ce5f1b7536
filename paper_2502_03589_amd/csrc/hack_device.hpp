// Device-side helpers of the HIP kernels: cache addressing, the partition
// quantizer (Sec. 5.2) in a pinned float32 operation order, and cross-lane
// reductions.  Everything here is compiled for gfx950 only.
#pragma once

#include <hip/hip_runtime.h>
#include <hip/hip_fp16.h>
#include <stdint.h>

namespace hack {

// Geometry and device pointers of one cache (see the section layout in hack.h).
struct CacheView {
  uint8_t* k_codes;
  __half2* k_meta;
  uint8_t* k_sums;
  uint8_t* v_codes;
  __half2* v_meta;
  uint8_t* v_sums;
  __half* v_tail;
  const int32_t* block_table;  // [batch][mbps] or nullptr
  int mbps;                    // max blocks per sequence
  int64_t num_pages;
  int page_tokens;
  int kv_heads;
  int head_dim;
  int sum_bytes;
};

// Page of token t of sequence s (a contiguous cache maps sequence s to page s).
// A page index outside [0, num_pages) is clamped: a bad table gives wrong values,
// never an access outside the cache.
__device__ __forceinline__ int64_t page_of(const CacheView& c, int s, int t) {
  int64_t pg = c.block_table ? (int64_t)c.block_table[(int64_t)s * c.mbps + t / c.page_tokens] : (int64_t)s;
  return pg < 0 ? 0 : (pg >= c.num_pages ? c.num_pages - 1 : pg);
}

// Row index of token t's K data: ((page * H + h) * page_tokens + slot).
__device__ __forceinline__ int64_t k_row(const CacheView& c, int s, int h, int t) {
  return (page_of(c, s, t) * c.kv_heads + h) * c.page_tokens + (t % c.page_tokens);
}

// Index of the V block holding token t: ((page * H + h) * page_tokens/PI + block-in-page).
template <int PI>
__device__ __forceinline__ int64_t v_block(const CacheView& c, int s, int h, int t) {
  return (page_of(c, s, t) * c.kv_heads + h) * (c.page_tokens / PI) + (t % c.page_tokens) / PI;
}

__device__ __forceinline__ uint32_t load_sum(const uint8_t* base, int64_t idx, int sum_bytes) {
  return sum_bytes == 1 ? (uint32_t)base[idx] : (uint32_t)reinterpret_cast<const uint16_t*>(base)[idx];
}

__device__ __forceinline__ void store_sum(uint8_t* base, int64_t idx, int sum_bytes, uint32_t v) {
  if (sum_bytes == 0) return;  // no cached sums (summation elimination off)
  if (sum_bytes == 1) base[idx] = (uint8_t)v;
  else reinterpret_cast<uint16_t*>(base)[idx] = (uint16_t)v;
}

// ---------------------------------------------------------------------------
// Stochastic-rounding thresholds: SplitMix64 (Steele, Lea and Flood, 2014).
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint64_t splitmix64(uint64_t x) {
  uint64_t z = x + 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// u in [0, 1): the top 24 bits of SplitMix64(key ^ idx) scaled by 2^-24.
__device__ __forceinline__ float sr_threshold(uint64_t key, uint64_t idx) {
  return (float)(uint32_t)(splitmix64(key ^ idx) >> 40) * 5.9604644775390625e-08f;
}

// Canonical index of a transient Q or P element: query head `head` of sequence `seq`,
// query row `row` (0 in decode), column `col` (Q channel or P key token):
// ((seq * H_q + head) * 2^20 + row) * 2^24 + col.
__device__ __forceinline__ uint64_t qp_index(int seq, int q_heads, int head, int row, int col) {
  return ((((uint64_t)(seq * q_heads + head)) << 20) + (uint64_t)row) * (1ull << 24) + (uint64_t)col;
}

// Stochastic rounding of t >= 0 to an integer code in [0, qmax]: floor(t) + [u < frac(t)].
__device__ __forceinline__ float round_stochastic(float t, float u, float qmax) {
  const float fl = floorf(t);
  return fminf(fmaxf(fl + (u < t - fl ? 1.0f : 0.0f), 0.0f), qmax);
}

// Smallest fp16 value >= s (s >= 0, finite), as raw bits.
__device__ __forceinline__ uint16_t half_bits_round_up(float s) {
  __half h = __float2half_rn(s);
  uint16_t bits = __half_as_ushort(h);
  if (__half2float(h) < s) bits = (uint16_t)(bits + 1);
  return bits;
}

// Quantize the first `n` of N values as one partition (Sec. 5.2):
//   m = min, s = fp16_round_up(fl(fl(max - m) / (2^b - 1))), r = fl(1/s),
//   t = fl(fl(x - m) * r), code = min(2^b - 1, round(t)) (nearest-even, or stochastic
//   with threshold u: floor(t) + [u < t - floor(t)]); s == 0 gives all-zero codes.
// Codes are packed LSB-first into `words` (element e at bit e*BITS); elements past n
// get code 0.  Returns the code sum; writes (m, s) as raw fp16 bits.
template <int BITS, int N>
__device__ __forceinline__ uint32_t quantize_values(const float (&x)[N], int n, bool stochastic,
                                                    uint64_t key, uint64_t idx0, uint64_t idx_step,
                                                    uint32_t (&words)[(N * BITS + 31) / 32],
                                                    uint16_t& m_bits, uint16_t& s_bits) {
#pragma clang fp contract(off)
  constexpr float QMAX = (float)((1 << BITS) - 1);
  float mn = x[0], mx = x[0];
#pragma unroll
  for (int e = 1; e < N; ++e) {
    if (e < n) {
      mn = fminf(mn, x[e]);
      mx = fmaxf(mx, x[e]);
    }
  }
  const float s32 = __fdiv_rn(__fsub_rn(mx, mn), QMAX);
  s_bits = half_bits_round_up(s32);
  m_bits = __half_as_ushort(__float2half_rn(mn));  // exact: m is an fp16 input value
  const float s = __half2float(__ushort_as_half(s_bits));
#pragma unroll
  for (int w = 0; w < (N * BITS + 31) / 32; ++w) words[w] = 0u;
  uint32_t sum = 0;
  if (s != 0.0f) {
    const float r = __fdiv_rn(1.0f, s);
#pragma unroll
    for (int e = 0; e < N; ++e) {
      if (e < n) {
        const float t = __fmul_rn(__fsub_rn(x[e], mn), r);
        float c;
        if (!stochastic) {
          c = rintf(t);
        } else {
          const float fl = floorf(t);
          const float u = sr_threshold(key, idx0 + (uint64_t)e * idx_step);
          c = fl + ((u < __fsub_rn(t, fl)) ? 1.0f : 0.0f);
        }
        c = fminf(c, QMAX);
        const uint32_t ci = (uint32_t)c;
        words[(e * BITS) / 32] |= ci << ((e * BITS) % 32);
        sum += ci;
      }
    }
  }
  return sum;
}

// Canonical element index used for stochastic thresholds:
// ((seq * H_kv + head) * 2^32 + token) * d + channel.
__device__ __forceinline__ uint64_t element_index(int s, int kv_heads, int h, int t, int d, int ch) {
  return ((((uint64_t)(s * kv_heads + h)) << 32) + (uint64_t)t) * (uint64_t)d + (uint64_t)ch;
}

template <int PI>
__device__ __forceinline__ void load_f16_run(const __half* __restrict__ src, float (&x)[PI]) {
  // PI contiguous fp16 values, 16 bytes at a time (PI is a multiple of 16).
  const uint4* p = reinterpret_cast<const uint4*>(src);
#pragma unroll
  for (int i = 0; i < PI / 8; ++i) {
    uint4 w = p[i];
    const __half2* h = reinterpret_cast<const __half2*>(&w);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      float2 f = __half22float2(h[j]);
      x[8 * i + 2 * j] = f.x;
      x[8 * i + 2 * j + 1] = f.y;
    }
  }
}

template <int BITS, int PI>
__device__ __forceinline__ void store_codes(uint8_t* dst, const uint32_t (&w)[(PI * BITS + 31) / 32]) {
  uint32_t* d = reinterpret_cast<uint32_t*>(dst);
#pragma unroll
  for (int i = 0; i < (PI * BITS + 31) / 32; ++i) d[i] = w[i];
}

// Open V block modes (the library's HACK_TAIL_* values).
constexpr int kTailFp16 = 0, kTailRequant = 1, kTailDequant = 2;

// The new token's V value of channel `ch` (Sec. 5.3): it goes to row T = L mod PI of
// the fp16 open block, and the block (n = T + 1 values) is quantized when it fills or,
// in the re-quantizing modes, on every append.  Requant takes the earlier values from
// the fp16 rows; Dequant recovers them from the block's codes,
// x = fp16(fl(fl(s * code) + min)), so every earlier rounding error is kept.
template <int BITS, int PI>
__device__ __forceinline__ void append_v_channel(const CacheView& c, int s, int h, int L, int ch, __half vn,
                                                 int tail_mode, bool stochastic, uint64_t key_v) {
  const int H = c.kv_heads, d = c.head_dim;
  const int F = L / PI, T = L - F * PI;  // the new token is element T of block F
  __half* tail = c.v_tail + (((int64_t)s * H + h) * PI) * d + ch;  // row 0 of the open block
  tail[(int64_t)T * d] = vn;
  if (!(T + 1 == PI || tail_mode != kTailFp16)) return;
  constexpr int NW = (PI * BITS + 31) / 32;
  const int64_t vbh = v_block<PI>(c, s, h, F * PI);
  uint32_t* cdst = reinterpret_cast<uint32_t*>(c.v_codes + (vbh * d + ch) * (PI * BITS / 8));
  float x[PI];
  if (tail_mode == kTailDequant) {
    uint32_t old[NW];
#pragma unroll
    for (int w = 0; w < NW; ++w) old[w] = T > 0 ? cdst[w] : 0u;
    const uint32_t meta = T > 0 ? reinterpret_cast<const uint32_t*>(c.v_meta)[vbh * d + ch] : 0u;
    const float mn = __half2float(__ushort_as_half((uint16_t)(meta & 0xFFFFu)));
    const float sc = __half2float(__ushort_as_half((uint16_t)(meta >> 16)));
#pragma unroll
    for (int e = 0; e < PI; ++e) {
      const float code = (float)((old[(e * BITS) / 32] >> ((e * BITS) % 32)) & ((1u << BITS) - 1u));
      const float xe = __half2float(__float2half_rn(__fadd_rn(__fmul_rn(sc, code), mn)));
      x[e] = e < T ? xe : (e == T ? __half2float(vn) : 0.0f);
    }
  } else {
    // every row of the open block is read (rows past T are ignored), so the loads
    // are independent of T and issue together
    __half raw[PI];
#pragma unroll
    for (int e = 0; e < PI; ++e) raw[e] = tail[(int64_t)e * d];
#pragma unroll
    for (int e = 0; e < PI; ++e) x[e] = e < T ? __half2float(raw[e]) : (e == T ? __half2float(vn) : 0.0f);
  }
  uint32_t words[NW];
  uint16_t mb, sb;
  const uint32_t sum = quantize_values<BITS, PI>(x, T + 1, stochastic, key_v, element_index(s, H, h, F * PI, d, ch),
                                                 (uint64_t)d, words, mb, sb);
#pragma unroll
  for (int w = 0; w < NW; ++w) cdst[w] = words[w];
  reinterpret_cast<uint32_t*>(c.v_meta)[vbh * d + ch] = (uint32_t)mb | ((uint32_t)sb << 16);
  store_sum(c.v_sums, vbh * d + ch, c.sum_bytes, sum);
}

// Quantize-on-write of one token of one (sequence, kv head) (Sec. 5.3): the new
// token is token L of the sequence.  Its K row is quantized per partition; its V
// values go through append_v_channel.  Threads tid < d/PI take one K partition each,
// threads tid, tid + nthreads, ... one V channel each.  The caller guarantees
// 0 <= L < capacity.
template <int BITS, int PI>
__device__ __forceinline__ void append_head(const CacheView& c, const __half* __restrict__ k_new,
                                            const __half* __restrict__ v_new, int s, int h, int L,
                                            int tail_mode, bool stochastic, uint64_t key_k, uint64_t key_v,
                                            int tid, int nthreads) {
  const int H = c.kv_heads, d = c.head_dim, P = d / PI;
  if (tid < P) {
    float xk[PI];
    load_f16_run<PI>(k_new + tid * PI, xk);
    uint32_t words[(PI * BITS + 31) / 32];
    uint16_t mb, sb;
    const uint32_t sum = quantize_values<BITS, PI>(xk, PI, stochastic, key_k, element_index(s, H, h, L, d, tid * PI),
                                                   1ull, words, mb, sb);
    const int64_t row = k_row(c, s, h, L);
    store_codes<BITS, PI>(c.k_codes + row * (d * BITS / 8) + tid * (PI * BITS / 8), words);
    reinterpret_cast<uint32_t*>(c.k_meta)[row * P + tid] = (uint32_t)mb | ((uint32_t)sb << 16);
    store_sum(c.k_sums, row * P + tid, c.sum_bytes, sum);
  }
  for (int ch = tid; ch < d; ch += nthreads)
    append_v_channel<BITS, PI>(c, s, h, L, ch, v_new[ch], tail_mode, stochastic, key_v);
}

// ---------------------------------------------------------------------------
// Cross-lane reductions inside a row of 16 lanes (DPP row rotates).
// ---------------------------------------------------------------------------
// Every lane of a row rotate has a source in its own row, so the bound-control
// form changes nothing; it lets the compiler fold the move into the ALU op that
// consumes it (v_max_f32_dpp, v_add_f32_dpp, ...).
template <int CTRL>
__device__ __forceinline__ float dpp_f(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, true));
}
template <int CTRL>
__device__ __forceinline__ int dpp_i(int x) {
  return __builtin_amdgcn_update_dpp(0, x, CTRL, 0xF, 0xF, true);
}

// row_ror:n has DPP control 0x120 + n.
__device__ __forceinline__ float row16_max(float x) {
  x = fmaxf(x, dpp_f<0x128>(x));
  x = fmaxf(x, dpp_f<0x124>(x));
  x = fmaxf(x, dpp_f<0x122>(x));
  x = fmaxf(x, dpp_f<0x121>(x));
  return x;
}
__device__ __forceinline__ float row16_min(float x) {
  x = fminf(x, dpp_f<0x128>(x));
  x = fminf(x, dpp_f<0x124>(x));
  x = fminf(x, dpp_f<0x122>(x));
  x = fminf(x, dpp_f<0x121>(x));
  return x;
}
__device__ __forceinline__ float row16_sum(float x) {
  x += dpp_f<0x128>(x);
  x += dpp_f<0x124>(x);
  x += dpp_f<0x122>(x);
  x += dpp_f<0x121>(x);
  return x;
}
__device__ __forceinline__ int row16_sum_i(int x) {
  x += dpp_i<0x128>(x);
  x += dpp_i<0x124>(x);
  x += dpp_i<0x122>(x);
  x += dpp_i<0x121>(x);
  return x;
}

}  // namespace hack
