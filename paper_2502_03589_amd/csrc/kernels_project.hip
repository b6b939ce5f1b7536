// QKV generation (Sec. 4, Eq. 1) fused with quantize-on-write (Sec. 5.2 quantizer,
// Sec. 5.3 partitioning), the front half of the paper's prefill kernel (Sec. 6).
//
// The projection is one GEMM: out[token][n] = sum_i E[token][i] W[n][i], where the
// output channels n are the H_q query heads' 128 channels, then the H_kv key heads',
// then the H_kv value heads'.  One workgroup of eight 64-lane waves computes a tile of
// 256 tokens x 256 channels, i.e. two heads of 256 tokens of one sequence:
//   main loop  K steps of 32 input channels through four LDS stages of 32 KB (the 256 E
//              rows and the 256 W rows of the step, 64 bytes each, 16-byte chunks
//              XOR-swizzled so that fragment reads hit distinct banks).  The stages are
//              filled by direct global-to-LDS loads (global_load_lds_dwordx4, 1 KB per
//              wave instruction, no registers) issued three steps ahead, so about three
//              steps of matrix work cover each load's latency; one barrier per step
//              publishes a stage and frees the one computed before it.  Wave (wm, wn)
//              computes rows 128 wm .. +128 and channels 64 wn .. +64 with
//              v_mfma_f32_32x32x16_f16 (4 x 2 tiles of 32 x 32, fp32 accumulators), so
//              each 16-byte LDS read feeds 21 multiply-adds per lane, and each fetched
//              byte of E and W serves twice as many products as with 128 x 128 tiles.
//   epilogue   the tile is rounded to fp16 into the stage buffers; then, for each of its
//              two heads: a query head is written out in fp16 (the prefill attention
//              quantizes Q itself); a key head is quantized per (token, partition) and a
//              value head per (V block, channel) straight into the cache, with the same
//              quantizer and element indices as hack_quantize, including the fp16 open
//              V block.  The fp16 K and V never reach device memory.
// Tiles are numbered so that the workgroups one XCD runs at a time share their E and
// W tiles (groups of four token tiles per channel tile, contiguous ranges per XCD), so
// each slab is fetched into that XCD's L2 once for several workgroups.
#include "hack_internal.hpp"

namespace hack {

namespace {

typedef _Float16 v8h __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));

constexpr int kBM = 256;          // tokens per tile
constexpr int kBN = 256;          // output channels per tile (two heads)
constexpr int kBK = 32;           // input channels per step
constexpr int kThreads = 512;     // eight waves: 2 (tokens) x 4 (channels)
constexpr int kStages = 4;        // LDS stages: loads run three steps ahead of the products
constexpr int kStageH = (kBM + kBN) * kBK;  // halves per stage: 256 E rows, then 256 W rows, of 64 bytes
constexpr int kDma = kStageH * 2 / 1024 / (kThreads / 64);  // 1-KB direct-to-LDS loads per wave and step
constexpr int kGroupM = 4;        // token tiles that share each channel tile in the numbering
constexpr int kXcds = 8;          // workgroups are dealt to the XCDs round-robin
static_assert(2 * kDma < 16, "the stage waits encode vmcnt in four bits");
typedef __attribute__((address_space(3))) void lvoid;

// Position of 16-byte chunk c (0..3) of staged row r: rows are 64 bytes, and chunk c
// sits at c ^ ((r / 2) mod 4), so the eight rows one LDS cycle reads (32-row fragment
// reads, eight lanes per cycle) cover all eight 16-byte slots of 128 bytes.
__device__ __forceinline__ int stage_chunk(int r, int c) { return c ^ ((r >> 1) & 3); }

// 16 bytes per lane from global memory straight into LDS: lane l reads base + off and
// writes LDS bytes lds + 16 l (base and lds wave-uniform, lds via M0).  Issued as inline
// assembly so that the compiler does not add waits for it before LDS reads of other
// stages; the kernel waits for each stage's loads explicitly (vmcnt) before the barrier
// that publishes it.  The per-lane offset is a register that stays live for the whole
// main loop, so no later instruction (in particular no matrix-core result) overwrites
// an address operand while a load is still in flight.
__device__ __forceinline__ void dma16(const void* base, uint32_t off, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(off), "s"(base), "s"(lds)
               : "memory", "m0");
}

// Workgroup barrier that orders LDS accesses without waiting for outstanding
// direct-to-LDS loads (a fence would wait for all of them); each wave waits for its
// own loads of a stage explicitly before it.
__device__ __forceinline__ void stage_barrier() { asm volatile("s_barrier" ::: "memory"); }

__device__ __forceinline__ v16f mfma_f16(v8h a, v8h b, v16f c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
}

}  // namespace

template <int BITS, int PI>
__global__ __launch_bounds__(kThreads, 1) void project_kernel(ProjectArgs p) {
  // one LDS array per stage, so that the compiler tracks each stage's loads on its own
  __shared__ __attribute__((aligned(1024))) __half st0[kStageH];
  __shared__ __attribute__((aligned(1024))) __half st1[kStageH];
  __shared__ __attribute__((aligned(1024))) __half st2[kStageH];
  __shared__ __attribute__((aligned(1024))) __half st3[kStageH];
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
  const int rows_valid = min(kBM, p.len - t0);
  const int wrows_valid = min(kBN, nrows - ntile * kBN);
  // Direct-to-LDS loads: wave w fills 1-KB pieces q = kDma w + i of a stage (16 staged
  // rows each; waves 0-3 the E rows, 4-7 the W rows), lane l row 16 q + l / 4 at chunk
  // slot l % 4.  Rows past the sequence (or the last head) read the last valid row.
  const bool wave_e = wave < kThreads / 128;
  const uint8_t* gbase = wave_e ? reinterpret_cast<const uint8_t*>(e_rows) : reinterpret_cast<const uint8_t*>(w_rows);
  uint32_t goff[kDma];
#pragma unroll
  for (int i = 0; i < kDma; ++i) {
    const int r = 16 * (kDma * wave + i) + (lane >> 2);  // staged row 0 .. 511
    const int row = wave_e ? min(r, rows_valid - 1) : min(r - kBM, wrows_valid - 1);
    goff[i] = (uint32_t)((row * p.hidden + 8 * stage_chunk(r, lane & 3)) * 2);
  }
  auto load_stage = [&](__half* st, int k) __attribute__((always_inline)) {
    const uint8_t* base = gbase + (int64_t)k * kBK * 2;
#pragma unroll
    for (int i = 0; i < kDma; ++i) dma16(base, goff[i], (uint32_t)(uintptr_t)(lvoid*)(st + 512 * (kDma * wave + i)));
  };
  // fragment reads: lane l reads staged row (base + l % 32), chunk 2 kk + l / 32
  const int frow = lane & 31;
  auto compute = [&](const __half* st) __attribute__((always_inline)) {
#pragma unroll
    for (int kk = 0; kk < kBK / 16; ++kk) {
      const int ck = 2 * kk + (lane >> 5);
      v8h af[4], bf[2];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = 128 * wm + 32 * i + frow;
        af[i] = *reinterpret_cast<const v8h*>(st + r * kBK + 8 * stage_chunk(r, ck));
      }
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int r = kBM + 64 * wn + 32 * j + frow;
        bf[j] = *reinterpret_cast<const v8h*>(st + r * kBK + 8 * stage_chunk(r, ck));
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = mfma_f16(af[i], bf[j], acc[i][j]);
    }
  };
  // step k: wait for this wave's loads of stage k (the loads of steps k + 1 and k + 2
  // may stay in flight), barrier (every wave's loads of stage k are in LDS, and every
  // wave is done with step k - 1, whose stage takes step k + 3), then compute
  auto step = [&](int k, const __half* cur, __half* nxt) __attribute__((always_inline)) {
    if (k + 2 < nk) __builtin_amdgcn_s_waitcnt(0x0F70 | (2 * kDma));
    else if (k + 1 < nk) __builtin_amdgcn_s_waitcnt(0x0F70 | kDma);
    else __builtin_amdgcn_s_waitcnt(0x0F70);
    stage_barrier();
    if (k + 3 < nk) load_stage(nxt, k + 3);
    compute(cur);
  };
  load_stage(st0, 0);
  if (nk > 1) load_stage(st1, 1);
  if (nk > 2) load_stage(st2, 2);
  for (int ks = 0; ks < nk; ks += kStages) {
    step(ks, st0, st3);
    if (ks + 1 < nk) step(ks + 1, st1, st0);
    if (ks + 2 < nk) step(ks + 2, st2, st1);
    if (ks + 3 < nk) step(ks + 3, st3, st2);
  }
  stage_barrier();  // every wave is done reading the stages

  // ---- the tile in fp16 (round to nearest even): head hh's rows 0-127 in stage array
  // 2 hh, rows 128-255 in 2 hh + 1, 128 channels per row ----
  // accumulator register r of lane l: row 8 (r / 4) + 4 (l / 32) + r % 4, column l % 32
  {
    const int a = 2 * (wn >> 1) + wm;
    __half* dst = a == 0 ? st0 : (a == 1 ? st1 : (a == 2 ? st2 : st3));
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = 32 * i + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
          const int col = 64 * (wn & 1) + 32 * j + (lane & 31);
          dst[row * 128 + col] = __float2half_rn(acc[i][j][r]);
        }
  }
  __syncthreads();
  const int valid = rows_valid;
  const int Hq = p.q_heads, H = p.kv_heads;
  constexpr int D = 128, P = D / PI;
#pragma unroll 1
  for (int hh = 0; hh < 2; ++hh) {
    const int head = 2 * ntile + hh;  // output head: query heads, then key heads, then value heads
    if (head >= p.nheads) break;
    const __half* t_lo = hh == 0 ? st0 : st2;
    const __half* t_hi = hh == 0 ? st1 : st3;
    auto tile_row = [&](int row) __attribute__((always_inline)) -> const __half* {
      return (row < 128 ? t_lo : t_hi) + (row & 127) * 128;
    };
    if (head < Hq) {
      // query head: 128-channel fp16 rows, 16 bytes per thread and step
      __half* dst = p.q + (((int64_t)s * Hq + head) * p.len + t0) * D;
      for (int i = tid; i < valid * (D / 8); i += kThreads) {
        const int row = i / (D / 8), part = i % (D / 8);
        *reinterpret_cast<uint4*>(dst + (int64_t)row * D + 8 * part) =
            *reinterpret_cast<const uint4*>(tile_row(row) + 8 * part);
      }
    } else if (head < Hq + H) {
      // key head: one thread per (token, partition along the head dimension)
      const int h = head - Hq;
      for (int task = tid; task < valid * P; task += kThreads) {
        const int row = task / P, pp = task % P, t = t0 + row;
        float x[PI];
#pragma unroll
        for (int e = 0; e < PI; e += 8) {
          const uint4 raw = *reinterpret_cast<const uint4*>(tile_row(row) + pp * PI + e);
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
        for (int e = 0; e < PI; ++e) x[e] = e < n ? __half2float(tile_row(bl * PI + e)[ch]) : 0.0f;
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
          for (int e = 0; e < T; ++e) tail[(int64_t)e * D] = tile_row(bl * PI + e)[ch];
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
