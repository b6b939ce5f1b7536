// Quantize-on-write kernels (Sec. 5.1 steps 2 and 9; Sec. 5.2 quantizer; Sec. 5.3
// partitioning and the fp16 open V block).
//   quantize_k: one thread per (sequence, kv head, token, K partition along d)
//   quantize_v: one thread per (sequence, kv head, V block, channel pair)
//   append    : one workgroup per sequence, one new token for every kv head
// All are HBM-bound: they read fp16 values once and write codes, (min, scale) and sums.
#include <type_traits>

#include "hack_internal.hpp"

namespace hack {

template <int BITS, int PI>
__global__ __launch_bounds__(256) void quantize_k_kernel(CacheView c, const __half* __restrict__ k,
                                                         const int32_t* __restrict__ lens, int batch,
                                                         int max_len, int stochastic, uint64_t key) {
  const int P = c.head_dim / PI;
  const int64_t total = (int64_t)batch * c.kv_heads * max_len * P;
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
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

// V: one thread per (sequence, kv head, V block, channel pair).  The threads of a
// block's channel pairs are consecutive, so each of the block's PI token rows is
// read as one contiguous run of 4-byte loads (a whole row per 64 pairs), and each
// thread writes the adjacent codes, (min, scale) and sums of its two channels.
template <int BITS, int PI>
__global__ __launch_bounds__(256) void quantize_v_kernel(CacheView c, const __half* __restrict__ v,
                                                         const int32_t* __restrict__ lens, int batch,
                                                         int max_len, int stochastic, uint64_t key) {
  constexpr int CB = PI * BITS / 8;  // code bytes per (block, channel)
  const int d = c.head_dim, pairs = d / 2;
  const int NB = (max_len + PI - 1) / PI;
  const int64_t total = (int64_t)batch * c.kv_heads * NB * pairs;
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
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
  if (nk > 0)
    hipLaunchKernelGGL((quantize_k_kernel<BITS, PI>), dim3((unsigned)((nk + 255) / 256)), dim3(256), 0,
                       stream, c, k, lens, batch, max_len, stoch, stream_key(lay.seed, 1));
  const int64_t nv = (int64_t)batch * c.kv_heads * ((max_len + PI - 1) / PI) * (c.head_dim / 2);
  if (nv > 0)
    hipLaunchKernelGGL((quantize_v_kernel<BITS, PI>), dim3((unsigned)((nv + 255) / 256)), dim3(256), 0,
                       stream, c, v, lens, batch, max_len, stoch, stream_key(lay.seed, 2));
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
