// Quantize-on-write kernels (Sec. 5.1 steps 2 and 9; Sec. 5.2 quantizer; Sec. 5.3
// partitioning and the fp16 open V block).
//   quantize_kv: one launch for K and V at partitions below 64: its first workgroups
//                take one thread per (sequence, kv head, V block, channel pair), the
//                rest one thread per (sequence, kv head, token, K partition along d),
//                so the V tasks' serial chains overlap the K tasks' streaming
//   quantize_k_split / quantize_v_split: partitions of 64 or more, split over lanes
//   append     : one workgroup per sequence, one new token for every kv head
// All are HBM-bound: they read fp16 values once and write codes, (min, scale) and sums.
#include <type_traits>

#include "hack_internal.hpp"

namespace hack {

// K task gid: (sequence, kv head, token, partition) in row-major order.
template <int BITS, int PI>
__device__ __forceinline__ void quantize_k_task(const CacheView& c, const __half* __restrict__ k,
                                                const int32_t* __restrict__ lens, int batch, int max_len,
                                                int stochastic, uint64_t key, int64_t gid) {
  const int P = c.head_dim / PI;
  const int64_t total = (int64_t)batch * c.kv_heads * max_len * P;
  if (gid >= total) return;
  const int p = (int)(gid % P);
  int64_t r = gid / P;
  const int t = (int)(r % max_len);
  r /= max_len;
  const int h = (int)(r % c.kv_heads);
  const int s = (int)(r / c.kv_heads);
  if (t >= min(lens[s], max_len)) return;
  float x[PI];
  load_f16_run<PI>(k + (((int64_t)s * c.kv_heads + h) * max_len + t) * c.head_dim + p * PI, x);
  uint32_t w[(PI * BITS + 31) / 32];
  uint16_t mb, sb;
  const uint32_t sum = quantize_values<BITS, PI>(
      x, PI, stochastic != 0, key, element_index(s, c.kv_heads, h, t, c.head_dim, p * PI), 1ull, w, mb, sb);
  const int64_t row = k_row(c, s, h, t);
  store_codes<BITS, PI>(c.k_codes + row * (c.head_dim * BITS / 8) + p * (PI * BITS / 8), w);
  reinterpret_cast<uint32_t*>(c.k_meta)[row * P + p] = (uint32_t)mb | ((uint32_t)sb << 16);
  store_sum(c.k_sums, row * P + p, c.sum_bytes, sum);
}

// K for partitions of 64 channels or more: two adjacent lanes per (token,
// partition), each with half of the partition's channels; minima, maxima and code
// sums are exchanged between the two lanes, every value is quantized with the same
// float32 operations as quantize_values.
template <int BITS, int PI>
__global__ __launch_bounds__(256) void quantize_k_split_kernel(CacheView c, const __half* __restrict__ k,
                                                               const int32_t* __restrict__ lens, int batch,
                                                               int max_len, int stochastic, uint64_t key) {
  constexpr int HC = PI / 2;           // channels per lane
  constexpr int HW = HC * BITS / 32;   // code dwords per lane
  constexpr float QMAX = (float)((1 << BITS) - 1);
  const int P = c.head_dim / PI;
  const int64_t total = (int64_t)batch * c.kv_heads * max_len * P * 2;
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  // lanes past the end take part in the exchanges with a copy of the last pair's work
  const int64_t g = gid < total ? gid : total - 1;
  const int hh = (int)(g & 1);
  int64_t r = g >> 1;
  const int p = (int)(r % P);
  r /= P;
  const int t = (int)(r % max_len);
  r /= max_len;
  const int h = (int)(r % c.kv_heads);
  const int s = (int)(r / c.kv_heads);
  const bool live = gid < total && t < min(lens[s], max_len);
  float x[HC];
  load_f16_run<HC>(k + (((int64_t)s * c.kv_heads + h) * max_len + t) * c.head_dim + p * PI + hh * HC, x);
  float mn = x[0], mx = x[0];
#pragma unroll
  for (int e = 1; e < HC; ++e) {
    mn = fminf(mn, x[e]);
    mx = fmaxf(mx, x[e]);
  }
  mn = fminf(mn, __shfl_xor(mn, 1, 64));
  mx = fmaxf(mx, __shfl_xor(mx, 1, 64));
  uint32_t w[HW];
#pragma unroll
  for (int i = 0; i < HW; ++i) w[i] = 0u;
  uint32_t z = 0;
  uint16_t sb, mb;
  {
#pragma clang fp contract(off)
    const float s32 = __fdiv_rn(__fsub_rn(mx, mn), QMAX);
    sb = half_bits_round_up(s32);
    mb = __half_as_ushort(__float2half_rn(mn));  // exact: an input value
    const float sc = __half2float(__ushort_as_half(sb));
    if (sc != 0.0f) {
      const float rr = __fdiv_rn(1.0f, sc);
      const uint64_t idx0 = element_index(s, c.kv_heads, h, t, c.head_dim, p * PI + hh * HC);
#pragma unroll
      for (int e = 0; e < HC; ++e) {
        const float tt = __fmul_rn(__fsub_rn(x[e], mn), rr);
        float cf;
        if (!stochastic) {
          cf = rintf(tt);
        } else {
          const float fl = floorf(tt);
          cf = fl + ((sr_threshold(key, idx0 + (uint64_t)e) < __fsub_rn(tt, fl)) ? 1.0f : 0.0f);
        }
        const uint32_t ci = (uint32_t)fminf(cf, QMAX);
        w[(e * BITS) / 32] |= ci << ((e * BITS) % 32);
        z += ci;
      }
    }
  }
  z += (uint32_t)__shfl_xor((int)z, 1, 64);
  if (!live) return;
  const int64_t row = k_row(c, s, h, t);
  uint8_t* cdst = c.k_codes + row * (c.head_dim * BITS / 8) + p * (PI * BITS / 8) + hh * (HC * BITS / 8);
  if constexpr (HW % 4 == 0) {
#pragma unroll
    for (int i = 0; i < HW / 4; ++i)
      reinterpret_cast<uint4*>(cdst)[i] = uint4{w[4 * i], w[4 * i + 1], w[4 * i + 2], w[4 * i + 3]};
  } else {
#pragma unroll
    for (int i = 0; i < HW / 2; ++i) reinterpret_cast<uint2*>(cdst)[i] = uint2{w[2 * i], w[2 * i + 1]};
  }
  if (hh == 0) {
    reinterpret_cast<uint32_t*>(c.k_meta)[row * P + p] = (uint32_t)mb | ((uint32_t)sb << 16);
    store_sum(c.k_sums, row * P + p, c.sum_bytes, z);
  }
}

// V: one thread per (sequence, kv head, V block, channel pair).  The threads of a
// block's channel pairs are consecutive, so each of the block's PI token rows is
// read as one contiguous run of 4-byte loads (a whole row per 64 pairs), and each
// thread writes the adjacent codes, (min, scale) and sums of its two channels.
// V task gid: (sequence, kv head, V block, channel pair) in row-major order.
template <int BITS, int PI>
__device__ __forceinline__ void quantize_v_task(const CacheView& c, const __half* __restrict__ v,
                                                const int32_t* __restrict__ lens, int batch, int max_len,
                                                int stochastic, uint64_t key, int64_t gid) {
  constexpr int CB = PI * BITS / 8;  // code bytes per (block, channel)
  const int d = c.head_dim, pairs = d / 2;
  const int NB = (max_len + PI - 1) / PI;
  const int64_t total = (int64_t)batch * c.kv_heads * NB * pairs;
  if (gid >= total) return;
  const int ch = 2 * (int)(gid % pairs);
  int64_t r = gid / pairs;
  const int blk = (int)(r % NB);
  r /= NB;
  const int h = (int)(r % c.kv_heads);
  const int s = (int)(r / c.kv_heads);
  const int L = max(0, min(lens[s], max_len));  // lengths past max_len are ignored
  const int F = L / PI, T = L - F * PI;
  if (blk > F || (blk == F && T == 0)) return;
  const int n = blk < F ? PI : T;
  const __half* src = v + (((int64_t)s * c.kv_heads + h) * max_len + (int64_t)blk * PI) * d + ch;
  uint32_t raw[PI];  // (channel ch, channel ch + 1) of each token row
#pragma unroll
  for (int e = 0; e < PI; ++e) raw[e] = e < n ? *reinterpret_cast<const uint32_t*>(src + (int64_t)e * d) : 0u;
  const int64_t vb = v_block<PI>(c, s, h, blk * PI);
  constexpr int NW = (PI * BITS + 31) / 32;
  uint32_t meta[2], sums[2];
  uint32_t w0[NW], w1[NW];
  // channel ch + j of the pair: the half j of every raw word
  auto quantize_channel = [&](auto j_tag, uint32_t (&w)[NW]) __attribute__((always_inline)) {
    constexpr int J = decltype(j_tag)::value;
    float x[PI];
#pragma unroll
    for (int e = 0; e < PI; ++e) x[e] = __half2float(__ushort_as_half((uint16_t)(raw[e] >> (16 * J))));
    uint16_t mb, sb;
    sums[J] = quantize_values<BITS, PI>(x, n, stochastic != 0, key,
                                        element_index(s, c.kv_heads, h, blk * PI, d, ch + J), (uint64_t)d, w, mb,
                                        sb);
    meta[J] = (uint32_t)mb | ((uint32_t)sb << 16);
  };
  quantize_channel(std::integral_constant<int, 0>{}, w0);
  quantize_channel(std::integral_constant<int, 1>{}, w1);
  // the two channels' codes are adjacent: 2 * CB bytes from a 2 * CB-aligned offset
  uint32_t both[2 * NW];
#pragma unroll
  for (int i = 0; i < NW; ++i) {
    both[i] = w0[i];
    both[NW + i] = w1[i];
  }
  uint8_t* cdst = c.v_codes + (vb * d + ch) * CB;
  if constexpr (2 * CB % 16 == 0) {
#pragma unroll
    for (int i = 0; i < 2 * CB / 16; ++i)
      reinterpret_cast<uint4*>(cdst)[i] = uint4{both[4 * i], both[4 * i + 1], both[4 * i + 2], both[4 * i + 3]};
  } else {
    *reinterpret_cast<uint2*>(cdst) = uint2{both[0], both[1]};
  }
  *reinterpret_cast<uint2*>(reinterpret_cast<uint32_t*>(c.v_meta) + vb * d + ch) = uint2{meta[0], meta[1]};
  if (c.sum_bytes == 1) {
    *reinterpret_cast<uint16_t*>(c.v_sums + vb * d + ch) = (uint16_t)(sums[0] | (sums[1] << 8));
  } else if (c.sum_bytes == 2) {
    *reinterpret_cast<uint32_t*>(c.v_sums + 2 * (vb * d + ch)) = sums[0] | (sums[1] << 16);
  }
  if (blk == F) {  // the open block: keep its fp16 originals
    __half* tail = c.v_tail + (((int64_t)s * c.kv_heads + h) * PI) * d + ch;
#pragma unroll
    for (int e = 0; e < PI; ++e)
      if (e < T) *reinterpret_cast<uint32_t*>(tail + (int64_t)e * d) = raw[e];
  }
}

// K and V in one launch: workgroups [0, v_blocks) run V tasks, the rest K tasks.
template <int BITS, int PI>
__global__ __launch_bounds__(256) void quantize_kv_kernel(CacheView c, const __half* __restrict__ k,
                                                          const __half* __restrict__ v,
                                                          const int32_t* __restrict__ lens, int batch, int max_len,
                                                          int stochastic, uint64_t key_k, uint64_t key_v,
                                                          int64_t v_blocks) {
  const int64_t b = blockIdx.x;
  if (b < v_blocks)
    quantize_v_task<BITS, PI>(c, v, lens, batch, max_len, stochastic, key_v, b * 256 + threadIdx.x);
  else
    quantize_k_task<BITS, PI>(c, k, lens, batch, max_len, stochastic, key_k, (b - v_blocks) * 256 + threadIdx.x);
}

// V for partitions of 64 tokens or more: one workgroup per (sequence, kv head, V
// block), each channel pair split over two threads (the two halves of the block's
// tokens, in different waves), so that a small cache still fills the chip.  The
// halves exchange their minima and maxima and their code sums through LDS; every
// value is quantized with the same float32 operations as quantize_values.
template <int BITS, int PI>
__global__ __launch_bounds__(256) void quantize_v_split_kernel(CacheView c, const __half* __restrict__ v,
                                                               const int32_t* __restrict__ lens, int max_len,
                                                               int stochastic, uint64_t key) {
  constexpr int HT = PI / 2;           // tokens per half
  constexpr int CB = PI * BITS / 8;    // code bytes per (block, channel)
  constexpr int HW = HT * BITS / 32;   // code dwords per (half, channel)
  constexpr float QMAX = (float)((1 << BITS) - 1);
  __shared__ float mm[2][128][2][2];   // [half][pair][channel][min, max]
  __shared__ uint32_t zs[2][128][2];   // [half][pair][channel] code sums
  const int d = c.head_dim, pairs = d / 2;
  const int NB = (max_len + PI - 1) / PI;
  const int tid = threadIdx.x;
  const int hh = tid / pairs, cp = tid % pairs, ch = 2 * cp;
  const int blk = (int)(blockIdx.x % NB);
  const int h = (int)((blockIdx.x / NB) % c.kv_heads);
  const int s = (int)(blockIdx.x / NB / c.kv_heads);
  const int L = max(0, min(lens[s], max_len));
  const int F = L / PI, T = L - F * PI;
  if (blk > F || (blk == F && T == 0)) return;  // uniform across the workgroup
  const int n = blk < F ? PI : T;
  const int e0 = hh * HT;                      // first token of this half
  const __half* src = v + (((int64_t)s * c.kv_heads + h) * max_len + (int64_t)blk * PI + e0) * d + ch;
  uint32_t raw[HT];
#pragma unroll
  for (int e = 0; e < HT; ++e) raw[e] = e0 + e < n ? *reinterpret_cast<const uint32_t*>(src + (int64_t)e * d) : 0u;
  float x[2][HT];
  float mn[2] = {INFINITY, INFINITY}, mx[2] = {-INFINITY, -INFINITY};
#pragma unroll
  for (int e = 0; e < HT; ++e) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      x[j][e] = __half2float(__ushort_as_half((uint16_t)(raw[e] >> (16 * j))));
      if (e0 + e < n) {
        mn[j] = fminf(mn[j], x[j][e]);
        mx[j] = fmaxf(mx[j], x[j][e]);
      }
    }
  }
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    mm[hh][cp][j][0] = mn[j];
    mm[hh][cp][j][1] = mx[j];
  }
  __syncthreads();
  uint32_t w[2][HW], meta[2], zloc[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
#pragma clang fp contract(off)
    const float lo = fminf(mm[0][cp][j][0], mm[1][cp][j][0]), hi = fmaxf(mm[0][cp][j][1], mm[1][cp][j][1]);
    const float s32 = __fdiv_rn(__fsub_rn(hi, lo), QMAX);
    const uint16_t sb = half_bits_round_up(s32);
    const uint16_t mb = __half_as_ushort(__float2half_rn(lo));  // exact: an input value
    const float sc = __half2float(__ushort_as_half(sb));
    meta[j] = (uint32_t)mb | ((uint32_t)sb << 16);
#pragma unroll
    for (int i = 0; i < HW; ++i) w[j][i] = 0u;
    uint32_t z = 0;
    if (sc != 0.0f) {
      const float r = __fdiv_rn(1.0f, sc);
      const uint64_t idx0 = element_index(s, c.kv_heads, h, blk * PI + e0, d, ch + j);
#pragma unroll
      for (int e = 0; e < HT; ++e) {
        if (e0 + e < n) {
          const float t = __fmul_rn(__fsub_rn(x[j][e], lo), r);
          float cf;
          if (!stochastic) {
            cf = rintf(t);
          } else {
            const float fl = floorf(t);
            cf = fl + ((sr_threshold(key, idx0 + (uint64_t)e * d) < __fsub_rn(t, fl)) ? 1.0f : 0.0f);
          }
          const uint32_t ci = (uint32_t)fminf(cf, QMAX);
          w[j][(e * BITS) / 32] |= ci << ((e * BITS) % 32);
          z += ci;
        }
      }
    }
    zloc[j] = z;
  }
  const int64_t vb = v_block<PI>(c, s, h, blk * PI);
#pragma unroll
  for (int j = 0; j < 2; ++j) {  // this half of each channel's code row: CB / 2 bytes
    uint8_t* cdst = c.v_codes + (vb * d + ch + j) * CB + hh * (CB / 2);
    if constexpr (HW % 4 == 0) {
#pragma unroll
      for (int i = 0; i < HW / 4; ++i)
        reinterpret_cast<uint4*>(cdst)[i] = uint4{w[j][4 * i], w[j][4 * i + 1], w[j][4 * i + 2], w[j][4 * i + 3]};
    } else {
#pragma unroll
      for (int i = 0; i < HW / 2; ++i) reinterpret_cast<uint2*>(cdst)[i] = uint2{w[j][2 * i], w[j][2 * i + 1]};
    }
  }
  zs[hh][cp][0] = zloc[0];
  zs[hh][cp][1] = zloc[1];
  __syncthreads();
  if (hh == 0) {
    const uint32_t z0 = zs[0][cp][0] + zs[1][cp][0], z1 = zs[0][cp][1] + zs[1][cp][1];
    *reinterpret_cast<uint2*>(reinterpret_cast<uint32_t*>(c.v_meta) + vb * d + ch) = uint2{meta[0], meta[1]};
    if (c.sum_bytes == 1) {
      *reinterpret_cast<uint16_t*>(c.v_sums + vb * d + ch) = (uint16_t)(z0 | (z1 << 8));
    } else if (c.sum_bytes == 2) {
      *reinterpret_cast<uint32_t*>(c.v_sums + 2 * (vb * d + ch)) = z0 | (z1 << 16);
    }
  }
  if (blk == F) {  // the open block: keep its fp16 originals
    __half* tail = c.v_tail + (((int64_t)s * c.kv_heads + h) * PI + e0) * d + ch;
#pragma unroll
    for (int e = 0; e < HT; ++e)
      if (e0 + e < T) *reinterpret_cast<uint32_t*>(tail + (int64_t)e * d) = raw[e];
  }
}

// One new token per sequence: K partitions of the token; V value into the fp16
// open block, which is quantized when it fills (and on every call in the
// re-quantizing modes, see append_v_channel).
// The new token's values are loaded together with the sequence length (they do not
// depend on it) so that the kernel pays one memory round trip before its stores.
template <int BITS, int PI>
__global__ __launch_bounds__(256) void append_kernel(CacheView c, const __half* __restrict__ k_new,
                                                     const __half* __restrict__ v_new, int32_t* lens,
                                                     int capacity, int tail_mode, int stochastic,
                                                     uint64_t key_k, uint64_t key_v) {
  constexpr int MAXV = 8;  // V channels per thread: H * d <= 256 * MAXV
  const int s = blockIdx.x;
  const int H = c.kv_heads, d = c.head_dim, P = d / PI;
  const int nk = H * P, nv = H * d;
  // K partition of this thread (one per thread for H * P <= 256)
  float xk[PI];
  const bool has_k = (int)threadIdx.x < nk;
  if (has_k) {
    const int h = threadIdx.x / P, p = threadIdx.x % P;
    load_f16_run<PI>(k_new + ((int64_t)s * H + h) * d + p * PI, xk);
  }
  __half vn[MAXV];
#pragma unroll
  for (int i = 0; i < MAXV; ++i) {
    const int w = threadIdx.x + i * blockDim.x;
    vn[i] = w < nv ? v_new[(int64_t)s * nv + w] : __float2half(0.0f);
  }
  const int L = lens[s];
  if (L < 0 || L >= capacity) return;  // uniform across the workgroup
  if (has_k) {
    const int h = threadIdx.x / P, p = threadIdx.x % P;
    uint32_t words[(PI * BITS + 31) / 32];
    uint16_t mb, sb;
    const uint32_t sum = quantize_values<BITS, PI>(
        xk, PI, stochastic != 0, key_k, element_index(s, H, h, L, d, p * PI), 1ull, words, mb, sb);
    const int64_t row = k_row(c, s, h, L);
    store_codes<BITS, PI>(c.k_codes + row * (d * BITS / 8) + p * (PI * BITS / 8), words);
    reinterpret_cast<uint32_t*>(c.k_meta)[row * P + p] = (uint32_t)mb | ((uint32_t)sb << 16);
    store_sum(c.k_sums, row * P + p, c.sum_bytes, sum);
  }
#pragma unroll
  for (int i = 0; i < MAXV; ++i) {
    const int w = threadIdx.x + i * blockDim.x;
    if (w >= nv) break;
    append_v_channel<BITS, PI>(c, s, w / d, L, w % d, vn[i], tail_mode, stochastic != 0, key_v);
  }
  __syncthreads();  // every thread has read lens[s]
  if (threadIdx.x == 0) lens[s] = L + 1;
}

static uint64_t stream_key(uint64_t seed, uint64_t stream) { return seed ^ (stream << 56); }

template <int BITS, int PI>
static hipError_t quantize_impl(const hack_kv_layout& lay, const CacheView& c, const __half* k,
                                const __half* v, const int32_t* lens, int batch, int max_len,
                                hipStream_t stream) {
  const int stoch = lay.rounding == HACK_ROUND_STOCHASTIC;
  const int64_t nk = (int64_t)batch * c.kv_heads * max_len * (c.head_dim / PI);
  const int64_t nblk = (int64_t)batch * c.kv_heads * ((max_len + PI - 1) / PI);
  if constexpr (PI >= 64) {
    // K: two lanes per partition; V: one workgroup per V block (head_dim <= 256 threads)
    if (nblk > 0x7FFFFFFF || (2 * nk + 255) / 256 > 0x7FFFFFFF) return hipErrorInvalidValue;
    if (nk > 0)
      hipLaunchKernelGGL((quantize_k_split_kernel<BITS, PI>), dim3((unsigned)((2 * nk + 255) / 256)), dim3(256), 0,
                         stream, c, k, lens, batch, max_len, stoch, stream_key(lay.seed, 1));
    if (nblk > 0)
      hipLaunchKernelGGL((quantize_v_split_kernel<BITS, PI>), dim3((unsigned)nblk), dim3(c.head_dim), 0, stream, c,
                         v, lens, max_len, stoch, stream_key(lay.seed, 2));
  } else {
    const int64_t nv = nblk * (c.head_dim / 2);
    const int64_t vb = (nv + 255) / 256, kb = (nk + 255) / 256;
    if (vb + kb > 0x7FFFFFFF) return hipErrorInvalidValue;
    if (vb + kb > 0)
      hipLaunchKernelGGL((quantize_kv_kernel<BITS, PI>), dim3((unsigned)(vb + kb)), dim3(256), 0, stream, c, k, v,
                         lens, batch, max_len, stoch, stream_key(lay.seed, 1), stream_key(lay.seed, 2), vb);
  }
  return hipGetLastError();
}

template <int BITS, int PI>
static hipError_t append_impl(const hack_kv_layout& lay, const CacheView& c, const __half* k_new,
                              const __half* v_new, int32_t* lens, int batch, int capacity,
                              int tail_mode, hipStream_t stream) {
  const int stoch = lay.rounding == HACK_ROUND_STOCHASTIC;
  hipLaunchKernelGGL((append_kernel<BITS, PI>), dim3(batch), dim3(256), 0, stream, c, k_new, v_new, lens,
                     capacity, tail_mode, stoch, stream_key(lay.seed, 1), stream_key(lay.seed, 2));
  return hipGetLastError();
}

#define HACK_DISPATCH_BITS_PI(BITS_, PI_, CALL)                        \
  switch ((BITS_) * 1000 + (PI_)) {                                    \
    case 2016: return CALL(2, 16);                                     \
    case 2032: return CALL(2, 32);                                     \
    case 2064: return CALL(2, 64);                                     \
    case 2128: return CALL(2, 128);                                    \
    case 4016: return CALL(4, 16);                                     \
    case 4032: return CALL(4, 32);                                     \
    case 4064: return CALL(4, 64);                                     \
    case 4128: return CALL(4, 128);                                    \
    default: return hipErrorInvalidValue;                              \
  }

hipError_t launch_quantize(const hack_kv_layout& lay, const CacheView& c, const __half* k,
                           const __half* v, const int32_t* lens, int batch, int max_len,
                           hipStream_t stream) {
#define CALLQ(B, P) quantize_impl<B, P>(lay, c, k, v, lens, batch, max_len, stream)
  HACK_DISPATCH_BITS_PI(lay.kv_bits, lay.partition, CALLQ)
#undef CALLQ
}

hipError_t launch_append(const hack_kv_layout& lay, const CacheView& c, const __half* k_new,
                         const __half* v_new, int32_t* lens, int batch, int capacity,
                         int tail_mode, hipStream_t stream) {
#define CALLA(B, P) append_impl<B, P>(lay, c, k_new, v_new, lens, batch, capacity, tail_mode, stream)
  HACK_DISPATCH_BITS_PI(lay.kv_bits, lay.partition, CALLA)
#undef CALLA
}

}  // namespace hack
