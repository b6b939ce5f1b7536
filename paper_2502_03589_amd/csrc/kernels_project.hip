// QKV generation (Sec. 4, Eq. 1) fused with quantize-on-write (Sec. 5.2 quantizer,
// Sec. 5.3 partitioning), the front half of the paper's prefill kernel (Sec. 6).
//
// The projection is one GEMM: out[token][n] = sum_i E[token][i] W[n][i], where the
// output channels n are the H_q query heads' 128 channels, then the H_kv key heads',
// then the H_kv value heads'.  One workgroup of eight 64-lane waves computes a tile of
// 256 tokens x 256 channels, i.e. two heads of 256 tokens of one sequence:
//   main loop  K steps of 64 input channels; both 256 x 64 fp16 tiles (E rows and W
//              rows) are staged in LDS (two buffers: the next step's global loads are
//              in flight while this step's MFMAs run); wave (wm, wn) computes rows
//              128 wm .. +128 and channels 64 wn .. +64 with v_mfma_f32_32x32x16_f16
//              (4 x 2 tiles of 32 x 32, fp32 accumulators), so each 16-byte LDS read
//              feeds 21 multiply-adds per lane (the 64 x 64 wave tile of a 128 x 128
//              workgroup tile fed 16, the rate at which one compute unit's LDS and its
//              matrix cores are equally busy), and each fetched byte of E and W serves
//              twice as many products.
//   epilogue   the tile is rounded to fp16 into LDS; then, for each of its two heads:
//              a query head is written out in fp16 (the prefill attention quantizes
//              Q itself); a key head is quantized per (token, partition) and a value
//              head per (V block, channel) straight into the cache, with the same
//              quantizer and element indices as hack_quantize, including the fp16
//              open V block.  The fp16 K and V never reach device memory.
// Tiles are numbered so that the workgroups one XCD runs at a time share their E and
// W tiles (groups of four token tiles per channel tile, contiguous ranges per XCD), so
// each 64-channel slab is fetched into that XCD's L2 once for several workgroups.
#include "hack_internal.hpp"

namespace hack {

namespace {

typedef _Float16 v8h __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kBM = 256;          // tokens per tile
constexpr int kBN = 256;          // output channels per tile (two heads)
constexpr int kBK = 64;           // input channels per step
constexpr int kThreads = 512;     // eight waves: 2 (tokens) x 4 (channels)
constexpr int kRowH = kBK + 8;    // LDS row stride of a staged tile (halves): 144 bytes, so that the
                                  // eight lanes of an LDS cycle read distinct banks
constexpr int kTileH = kBN + 8;   // LDS row stride of the fp16 output tile (halves)
constexpr int kGroupM = 4;        // token tiles that share each channel tile in the numbering
constexpr int kXcds = 8;          // workgroups are dealt to the XCDs round-robin
constexpr int kPieces = kBM * kBK / 8 / kThreads;  // 16-byte pieces per thread and operand per step

struct Stages {
  __half a[2][kBM][kRowH];
  __half b[2][kBN][kRowH];
};
union ProjectLds {
  Stages st;
  __half tile[kBM][kTileH];
};

__device__ __forceinline__ v16f mfma_f16(v8h a, v8h b, v16f c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
}

}  // namespace

template <int BITS, int PI>
__global__ __launch_bounds__(kThreads, 1) void project_kernel(ProjectArgs p) {
  __shared__ __attribute__((aligned(16))) ProjectLds lds;
  const CacheView& c = p.c;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 2, wn = wave & 3;

  // ---- tile of this workgroup: contiguous ranges per XCD, then groups of kGroupM
  // token tiles sharing each head tile ----
  const int64_t wg = blockIdx.x;
  const int64_t xcd = wg % kXcds, idx = wg / kXcds;
  const int64_t per = p.total / kXcds, rem = p.total % kXcds;
  const int64_t tl = xcd < rem ? xcd * (per + 1) + idx : rem * (per + 1) + (xcd - rem) * per + idx;
  const int64_t mt_all = p.total / p.ntiles;
  const int64_t group = tl / ((int64_t)kGroupM * p.ntiles);
  const int64_t first_m = group * kGroupM;
  const int64_t gsize = min((int64_t)kGroupM, mt_all - first_m);
  const int64_t local = tl - group * kGroupM * p.ntiles;
  const int64_t mtile = first_m + local % gsize;
  const int ntile = (int)(local / gsize);
  const int s = (int)(mtile / p.mtiles);
  const int t0 = (int)(mtile % p.mtiles) * kBM;
  const __half* e_rows = p.e + ((int64_t)s * p.len + t0) * p.hidden;
  const int nrows = p.nheads * 128;  // output channels
  const __half* w_rows = p.w + (int64_t)ntile * kBN * p.hidden;

  // ---- main loop ----
  v16f acc[4][2];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;
  const int nk = p.hidden / kBK;
  // piece c = tid + 512 i of a 256 x 64 tile: row c / 8, halves 8 (c % 8) .. + 8; the
  // byte offsets are 32-bit per-lane values next to wave-uniform bases
  const int rows_valid = min(kBM, p.len - t0);
  const int wrows_valid = min(kBN, nrows - ntile * kBN);
  uint32_t e_off[kPieces], w_off[kPieces];
  int lds_off[kPieces];
#pragma unroll
  for (int i = 0; i < kPieces; ++i) {
    const int cpc = tid + kThreads * i, row = cpc >> 3, part = cpc & 7;
    // rows of E past the sequence (and of W past the last head) read the last valid row
    // (they are computed, never stored)
    e_off[i] = (uint32_t)((min(row, rows_valid - 1) * p.hidden + 8 * part) * 2);
    w_off[i] = (uint32_t)((min(row, wrows_valid - 1) * p.hidden + 8 * part) * 2);
    lds_off[i] = row * kRowH + 8 * part;
  }
  const uint8_t* e_base = reinterpret_cast<const uint8_t*>(e_rows);
  const uint8_t* w_base = reinterpret_cast<const uint8_t*>(w_rows);
  u32x4 ra[kPieces], rb[kPieces];
#pragma unroll
  for (int i = 0; i < kPieces; ++i) {
    ra[i] = *reinterpret_cast<const u32x4*>(e_base + e_off[i]);
    rb[i] = *reinterpret_cast<const u32x4*>(w_base + w_off[i]);
  }
#pragma unroll
  for (int i = 0; i < kPieces; ++i) {
    *reinterpret_cast<u32x4*>(&lds.st.a[0][0][0] + lds_off[i]) = ra[i];
    *reinterpret_cast<u32x4*>(&lds.st.b[0][0][0] + lds_off[i]) = rb[i];
  }
  __syncthreads();
  const int frow = lane & 31, fk = 8 * (lane >> 5);
  for (int ks = 0; ks < nk; ++ks) {
    const int buf = ks & 1;
    const bool more = ks + 1 < nk;
    if (more) {
      const uint32_t kb = (uint32_t)((ks + 1) * kBK * 2);
#pragma unroll
      for (int i = 0; i < kPieces; ++i) {
        ra[i] = *reinterpret_cast<const u32x4*>(e_base + e_off[i] + kb);
        rb[i] = *reinterpret_cast<const u32x4*>(w_base + w_off[i] + kb);
      }
    }
    const __half* sa = &lds.st.a[buf][0][0];
    const __half* sb = &lds.st.b[buf][0][0];
#pragma unroll
    for (int kk = 0; kk < kBK / 16; ++kk) {
      v8h af[4], bf[2];
#pragma unroll
      for (int i = 0; i < 4; ++i)
        af[i] = *reinterpret_cast<const v8h*>(sa + (128 * wm + 32 * i + frow) * kRowH + 16 * kk + fk);
#pragma unroll
      for (int j = 0; j < 2; ++j)
        bf[j] = *reinterpret_cast<const v8h*>(sb + (64 * wn + 32 * j + frow) * kRowH + 16 * kk + fk);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = mfma_f16(af[i], bf[j], acc[i][j]);
    }
    if (more) {
      __half* da = &lds.st.a[buf ^ 1][0][0];
      __half* db = &lds.st.b[buf ^ 1][0][0];
#pragma unroll
      for (int i = 0; i < kPieces; ++i) {
        *reinterpret_cast<u32x4*>(da + lds_off[i]) = ra[i];
        *reinterpret_cast<u32x4*>(db + lds_off[i]) = rb[i];
      }
    }
    __syncthreads();
  }

  // ---- the tile in fp16 (round to nearest even), [token][channel] ----
  // accumulator register r of lane l: row 8 (r / 4) + 4 (l / 32) + r % 4, column l % 32
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = 128 * wm + 32 * i + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        const int col = 64 * wn + 32 * j + (lane & 31);
        lds.tile[row][col] = __float2half_rn(acc[i][j][r]);
      }
  __syncthreads();

  const int valid = rows_valid;
  const int Hq = p.q_heads, H = p.kv_heads;
  constexpr int D = 128, P = D / PI;
#pragma unroll 1
  for (int hh = 0; hh < 2; ++hh) {
    const int head = 2 * ntile + hh;  // output head: query heads, then key heads, then value heads
    const int cb = D * hh;            // its channels in the tile
    if (head >= p.nheads) break;
    if (head < Hq) {
      // query head: 128-channel fp16 rows, 16 bytes per thread and step
      __half* dst = p.q + (((int64_t)s * Hq + head) * p.len + t0) * D;
      for (int i = tid; i < valid * (D / 8); i += kThreads) {
        const int row = i / (D / 8), part = i % (D / 8);
        *reinterpret_cast<uint4*>(dst + (int64_t)row * D + 8 * part) =
            *reinterpret_cast<const uint4*>(&lds.tile[row][cb + 8 * part]);
      }
    } else if (head < Hq + H) {
      // key head: one thread per (token, partition along the head dimension)
      const int h = head - Hq;
      for (int task = tid; task < valid * P; task += kThreads) {
        const int row = task / P, pp = task % P, t = t0 + row;
        float x[PI];
#pragma unroll
        for (int e = 0; e < PI; e += 8) {
          const uint4 raw = *reinterpret_cast<const uint4*>(&lds.tile[row][cb + pp * PI + e]);
          const __half2* h2 = reinterpret_cast<const __half2*>(&raw);
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const float2 f = __half22float2(h2[q]);
            x[e + 2 * q] = f.x;
            x[e + 2 * q + 1] = f.y;
          }
        }
        uint32_t w[(PI * BITS + 31) / 32];
        uint16_t mb, sb;
        const uint32_t sum = quantize_values<BITS, PI>(x, PI, p.stochastic != 0, p.key_k,
                                                       element_index(s, H, h, t, D, pp * PI), 1ull, w, mb, sb);
        const int64_t kr = k_row(c, s, h, t);
        store_codes<BITS, PI>(c.k_codes + kr * (D * BITS / 8) + pp * (PI * BITS / 8), w);
        reinterpret_cast<uint32_t*>(c.k_meta)[kr * P + pp] = (uint32_t)mb | ((uint32_t)sb << 16);
        store_sum(c.k_sums, kr * P + pp, c.sum_bytes, sum);
      }
    } else {
      // value head: one thread per (V block of PI tokens, channel); the open block is
      // quantized with n = T and its fp16 values kept in the open-block buffer
      const int h = head - Hq - H;
      const int F = p.len / PI, T = p.len - F * PI;
      constexpr int NBT = kBM / PI;  // V blocks per tile
      for (int task = tid; task < NBT * D; task += kThreads) {
        const int bl = task / D, ch = task % D;
        const int blk = t0 / PI + bl;
        if (blk > F || (blk == F && T == 0)) continue;
        const int n = blk < F ? PI : T;
        float x[PI];
#pragma unroll
        for (int e = 0; e < PI; ++e) x[e] = e < n ? __half2float(lds.tile[bl * PI + e][cb + ch]) : 0.0f;
        uint32_t w[(PI * BITS + 31) / 32];
        uint16_t mb, sb;
        const uint32_t sum = quantize_values<BITS, PI>(x, n, p.stochastic != 0, p.key_v,
                                                       element_index(s, H, h, blk * PI, D, ch), (uint64_t)D, w, mb, sb);
        const int64_t vb = v_block<PI>(c, s, h, blk * PI);
        store_codes<BITS, PI>(c.v_codes + (vb * D + ch) * (PI * BITS / 8), w);
        reinterpret_cast<uint32_t*>(c.v_meta)[vb * D + ch] = (uint32_t)mb | ((uint32_t)sb << 16);
        store_sum(c.v_sums, vb * D + ch, c.sum_bytes, sum);
        if (blk == F) {
          __half* tail = c.v_tail + (((int64_t)s * H + h) * PI) * D + ch;
          for (int e = 0; e < T; ++e) tail[(int64_t)e * D] = lds.tile[bl * PI + e][cb + ch];
        }
      }
    }
  }
}

template <int BITS, int PI>
static hipError_t project_impl(const ProjectArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL((project_kernel<BITS, PI>), dim3((unsigned)a.total), dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_project(const hack_kv_layout& lay, const ProjectArgs& args, hipStream_t stream) {
  ProjectArgs a = args;
  a.mtiles = (a.len + kBM - 1) / kBM;
  a.nheads = a.q_heads + 2 * a.kv_heads;
  a.ntiles = (a.nheads + 1) / 2;
  a.total = (int64_t)a.batch * a.mtiles * a.ntiles;
  a.stochastic = lay.rounding == HACK_ROUND_STOCHASTIC;
  a.key_k = lay.seed ^ (1ull << 56);
  a.key_v = lay.seed ^ (2ull << 56);
  if (a.total == 0) return hipSuccess;
  switch (lay.kv_bits * 1000 + lay.partition) {
    case 2016: return project_impl<2, 16>(a, stream);
    case 2032: return project_impl<2, 32>(a, stream);
    case 2064: return project_impl<2, 64>(a, stream);
    case 2128: return project_impl<2, 128>(a, stream);
    case 4016: return project_impl<4, 16>(a, stream);
    case 4032: return project_impl<4, 32>(a, stream);
    case 4064: return project_impl<4, 64>(a, stream);
    case 4128: return project_impl<4, 128>(a, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace hack
