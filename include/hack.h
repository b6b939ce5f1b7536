/*
 * hack.h -- C ABI of the MI355X (gfx950) implementation of HACK's hot path:
 * attention computed directly on asymmetrically quantized K/V (and quantized
 * Q and P) without a dequantization pass (arXiv 2502.03589).
 *
 * Method (paper, Sec. 5.2 and Sec. 5.3):
 *   - Every partition of Pi elements along a contraction dimension is stored as
 *     b-bit codes x' = round((x - m) / s) with m = min, s = (max - m)/(2^b - 1).
 *   - A product sum_z a_z b_z over one partition is recovered from the integer
 *     product of the codes by Eq. 4:
 *       s_a s_b sum a'b' + s_a m_b sum a' + m_a s_b sum b' + n m_a m_b,
 *     using code sums cached next to the codes (summation elimination).
 *   - K is partitioned along the head dimension (per token), V along the
 *     sequence (Pi-token blocks per channel).  Q is quantized to 8 bits per
 *     partition, P to 8 bits per V block.  The open, partial V block is kept in
 *     fp16 and multiplied unquantized (requantization elimination).
 *
 * Conventions for every call:
 *   - Pointers named *_dev are device pointers; the caller owns every buffer
 *     (cache sections, inputs, outputs, workspace).  The library allocates no
 *     device memory and keeps no state besides cached device properties.
 *   - Work is enqueued asynchronously on `stream` (0 = the null stream); no call
 *     synchronizes.  Host structs are read only during the call.
 *   - Argument errors are detected on the host and returned before anything is
 *     launched; a launch failure returns HACK_ERR_HIP.  Device-side faults surface
 *     at the caller's next synchronization.  Nothing is printed.
 *   - fp16 means IEEE binary16, little-endian.  All outputs are fp32.
 */
#ifndef HACK_H
#define HACK_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum hack_status {
  HACK_OK = 0,
  HACK_ERR_INVALID_ARGUMENT = 1, /* null pointer, bad size or inconsistent shape   */
  HACK_ERR_UNSUPPORTED = 2,      /* a valid format the kernels do not implement     */
  HACK_ERR_CAPACITY = 3,         /* lengths exceed the cache's per-sequence capacity */
  HACK_ERR_WORKSPACE = 4,        /* workspace missing or smaller than required     */
  HACK_ERR_HIP = 5               /* the HIP runtime rejected a launch              */
} hack_status;

/* Rounding of every code the library produces (Sec. 5.2): the stored K/V codes
 * (hack_quantize, hack_append, hack_decode_step) and the transient Q and P codes inside
 * the attention kernels.  NEAREST_EVEN rounds t = (x - min) / scale to the nearest
 * integer, ties to even.  STOCHASTIC rounds t up with probability frac(t): the code is
 * floor(t) + [u < t - floor(t)] with u = (SplitMix64(seed ^ (stream << 56) ^ idx) >> 40)
 * * 2^-24.  Streams and element indices:
 *   K 1, V 2: idx = ((seq*H_kv + head) * 2^32 + token) * head_dim + channel;
 *   Q 3, P 4: idx = ((seq*H_q + q_head) * 2^20 + row) * 2^24 + column, where row is the
 *             query row (0 in decode) and column the Q channel or the P key token. */
enum { HACK_ROUND_NEAREST_EVEN = 0, HACK_ROUND_STOCHASTIC = 1 };

/* Treatment of the open (last, partial) V block of T = len mod Pi tokens (Sec. 5.3):
 * FP16    - kept in fp16 and multiplied with the unquantized P (requantization
 *           elimination, the paper's default);
 * REQUANT - re-quantized from its fp16 originals (kept in V_TAIL) with n = T on every
 *           append, and multiplied through Eq. 4 with n = T;
 * DEQUANT - re-quantized on every append from its dequantized codes plus the new value
 *           (the alternative that requantization elimination replaces; its rounding
 *           errors accumulate), and multiplied through Eq. 4 with n = T.
 * A cache is attended with the mode it was appended with. */
enum { HACK_TAIL_FP16 = 0, HACK_TAIL_REQUANT = 1, HACK_TAIL_DEQUANT = 2 };

/* Device arrays of a quantized KV cache.  Let P = head_dim/partition,
 * CB = head_dim*kv_bits/8 (code bytes per token), VB = partition*kv_bits/8 (code
 * bytes per channel and block), SB = sum_bytes, NP = page_tokens/partition:
 *   K_CODES [pages][H_kv][page_tokens][CB]         token's codes, partitions in order
 *   K_META  [pages][H_kv][page_tokens][P]  half2   (min, scale) of each K partition
 *   K_SUMS  [pages][H_kv][page_tokens][P]  u8/u16  code sum of each K partition
 *   V_CODES [pages][H_kv][NP][head_dim][VB]        channel's codes over a block
 *   V_META  [pages][H_kv][NP][head_dim]    half2   (min, scale) per block and channel
 *   V_SUMS  [pages][H_kv][NP][head_dim]    u8/u16
 *   V_TAIL  [seqs][H_kv][partition][head_dim] fp16 open block of each sequence
 * Codes are packed LSB-first in element order within a partition.  Token t of
 * sequence s is stored on page block_table[s][t / page_tokens] at slot
 * t % page_tokens; the V block of token t is slot (t % page_tokens)/partition of
 * that page.  The open block's slot holds its re-quantized codes (n = T, zero
 * codes past T).  K_CODES..V_TAIL are the bytes a prefill instance ships to a
 * decode instance (codes, min and scale; the sums may be rebuilt or shipped). */
typedef enum hack_kv_section {
  HACK_K_CODES = 0, HACK_K_META = 1, HACK_K_SUMS = 2,
  HACK_V_CODES = 3, HACK_V_META = 4, HACK_V_SUMS = 5, HACK_V_TAIL = 6
} hack_kv_section;

/* Quantization format; build it with hack_kv_layout_make. */
typedef struct hack_kv_layout {
  int32_t head_dim;      /* d_h                                                    */
  int32_t num_kv_heads;  /* H_kv                                                   */
  int32_t kv_bits;       /* b, bits per stored K/V code: 2 or 4                    */
  int32_t partition;     /* Pi: 16, 32, 64 or 128 (a multiple of 16, Sec. 5.3)     */
  int32_t page_tokens;   /* tokens per page; a multiple of Pi                      */
  int32_t qp_bits;       /* bits of the transient Q and P codes: 8 (Sec. 5.1, the
                            paper's INT8) or 4                                      */
  int32_t rounding;      /* HACK_ROUND_*                                           */
  int32_t sum_bytes;     /* 1 if b + ceil(log2 Pi) <= 8 else 2 (Sec. 5.3, Sec. 6);
                            0 when no sums are cached (hack_kv_layout_set_sums)     */
  uint64_t seed;         /* stochastic-rounding seed                               */
} hack_kv_layout;

/* One cache: device pointers to the seven sections plus the page table.
 * block_table_dev: int32 [batch][max_blocks_per_seq] page indices, or NULL, in which
 * case sequence s uses page s only (a contiguous cache with capacity page_tokens).
 * Per-sequence capacity = page_tokens * (block_table ? max_blocks_per_seq : 1). */
typedef struct hack_kv_cache {
  void* k_codes;
  void* k_meta;
  void* k_sums;
  void* v_codes;
  void* v_meta;
  void* v_sums;
  void* v_tail;
  const int32_t* block_table_dev;
  int32_t max_blocks_per_seq;
  int32_t reserved0;
  int64_t num_pages;
} hack_kv_cache;

/* Fill *out with a validated layout.  Rejects (HACK_ERR_INVALID_ARGUMENT) a null
 * out, head_dim not a positive multiple of partition or above 256, num_kv_heads < 1,
 * kv_bits not in {2,4}, partition not in {16,32,64,128}, page_tokens not a positive
 * multiple of partition, qp_bits not in {4,8}, an unknown rounding mode.  Host only. */
hack_status hack_kv_layout_make(hack_kv_layout* out, int32_t head_dim, int32_t num_kv_heads,
                                int32_t kv_bits, int32_t partition, int32_t page_tokens,
                                int32_t qp_bits, int32_t rounding, uint64_t seed);

/* Summation elimination (Sec. 5.3) on or off for `layout`.  cached = 1 (the
 * default of hack_kv_layout_make): the code sum of every partition is stored with
 * it (K_SUMS, V_SUMS) and read by the kernels.  cached = 0: no sums are stored
 * (their sections have 0 bytes and their pointers may be NULL); decode attention
 * rebuilds each sum from the packed codes it has loaded.  With cached = 0,
 * hack_attend_prefill and the debug exports return HACK_ERR_UNSUPPORTED.  Returns
 * HACK_ERR_INVALID_ARGUMENT for a null or invalid layout or cached not in {0,1}.
 * Host only. */
hack_status hack_kv_layout_set_sums(hack_kv_layout* layout, int32_t cached);

/* Bytes of one cache section: `count` is the number of pages for the K_* and V_*
 * code/meta/sum sections and the number of sequences for V_TAIL.  Returns -1 for a
 * null or invalid layout, a negative count or an unknown section.  Host only. */
int64_t hack_kv_bytes(const hack_kv_layout* layout, int64_t count, int32_t section);

/* Prefill-side quantize-on-write (Sec. 5.1, steps 1-2 and 7; Sec. 5.3 partitioning).
 * k_dev, v_dev: fp16 [batch][H_kv][max_len][head_dim]; seq_lens_dev: int32 [batch],
 * 0 <= seq_lens[s] <= max_len.  Writes, for every sequence, the K codes/meta/sums of
 * tokens [0, len), the V codes/meta/sums of the full blocks, the open block both
 * re-quantized (n = T) at its block slot and in fp16 in V_TAIL.  Nothing outside these
 * slots is written.  HACK_ERR_CAPACITY if max_len exceeds the per-sequence capacity;
 * HACK_ERR_UNSUPPORTED if batch * H_kv * ceil(max_len / partition) exceeds 2^31 - 1. */
hack_status hack_quantize(const hack_kv_layout* layout, const hack_kv_cache* cache,
                          const void* k_dev, const void* v_dev, const int32_t* seq_lens_dev,
                          int32_t batch, int32_t max_len, hipStream_t stream);

/* Decode-side quantize-on-write of one token per sequence (Sec. 5.1, step 9; Sec. 5.3).
 * k_new_dev, v_new_dev: fp16 [batch][H_kv][head_dim].  The new token goes to position
 * seq_lens[s]: its K partitions are quantized (earlier K partitions never change);
 * its V values enter the fp16 open block; when the open block reaches Pi tokens it is
 * quantized as a full block.  In HACK_TAIL_REQUANT mode the open block is also
 * re-quantized from its fp16 values on every call (n = T); in HACK_TAIL_DEQUANT mode
 * its codes are dequantized to fp16, x = fp16(fl(fl(s*code) + min)), the new value is
 * added and the block is quantized again (also when it fills).  A cache must be
 * attended with the tail mode it was appended with.  seq_lens_dev is incremented on
 * the device.  max_len is a host upper bound of seq_lens before the call; returns
 * HACK_ERR_CAPACITY if max_len + 1 exceeds the capacity (the kernel also skips any
 * sequence already at capacity); HACK_ERR_UNSUPPORTED if H_kv * head_dim > 2048. */
hack_status hack_append(const hack_kv_layout* layout, const hack_kv_cache* cache,
                        const void* k_new_dev, const void* v_new_dev, int32_t* seq_lens_dev,
                        int32_t batch, int32_t max_len, int32_t tail_mode, hipStream_t stream);

/* Workspace bytes hack_attend_decode needs for these sizes.  Layout: one int32
 * chunk counter per (sequence, kv head, group of four query heads) at offset 0, padded
 * to 256 bytes, then the split-K chunk records (max, sum and unnormalized O per chunk
 * and query head).  The counters' place and size depend only on batch, H_kv and
 * H_q/H_kv, never on max_len.  -1 on invalid arguments. */
int64_t hack_decode_workspace_bytes(const hack_kv_layout* layout, int32_t batch,
                                    int32_t num_q_heads, int32_t max_len);

/* Decode attention of one query token per sequence over its quantized cache
 * (Sec. 5.3 with L_Q = 1; Eq. 2-4).  q_dev: fp16 [batch][H_q][head_dim]; q head h
 * attends kv head h / (H_q/H_kv).  Per sequence, all seq_lens[s] cached tokens are
 * attended (0 <= seq_lens[s] <= max_len; a sequence of length 0 yields zeros).
 * out_dev: fp32 [batch][H_q][head_dim].  workspace_dev must hold
 * hack_decode_workspace_bytes(...) bytes.  Its counters (the first bytes, see
 * hack_decode_workspace_bytes) must be zero before the first call, and again before
 * a call with a different batch, H_q or layout; every call leaves them zero, so a
 * workspace may be reused by calls that differ only in max_len.  A workspace must not
 * be shared by calls that may run concurrently.  One kernel is launched; when a
 * sequence is split into several chunks, the workgroup that finishes its last chunk
 * merges them.
 * Requires head_dim 128, partition 32, 64 or 128, H_q/H_kv <= 8, batch <= 65535 and,
 * for a paged cache, page_tokens a multiple of 4 * partition (else
 * HACK_ERR_UNSUPPORTED).  Partitions of 32 and 64 run on the matrix cores; a
 * partition of 128 (one K partition per token row, V blocks of 128 tokens) runs on
 * the VALU's int8 dot instruction. */
hack_status hack_attend_decode(const hack_kv_layout* layout, const hack_kv_cache* cache,
                               const void* q_dev, int32_t num_q_heads, const int32_t* seq_lens_dev,
                               int32_t batch, int32_t max_len, int32_t tail_mode, float* out_dev,
                               void* workspace_dev, int64_t workspace_bytes, hipStream_t stream);

/* hack_attend_decode without a caller workspace, for callers that cannot allocate
 * device memory or pass a scratch buffer: code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc.  Arguments and results as hack_attend_decode;
 * the split-K counters and chunk records live in a library-owned static device array
 * instead (one per GPU, 16.25 MiB, held until the process ends).  Limits: at most
 * 65536 chunk counters (batch * H_kv * ceil(H_q/H_kv / 4)) and 16 MiB of chunk records
 * (hack_decode_workspace_bytes(...) minus its counter bytes); larger shapes return
 * HACK_ERR_WORKSPACE before anything is launched.  Nothing is allocated: no hipMalloc,
 * hipFree or allocating library call.  The first call on a device looks the array up
 * and launches a small kernel on `stream` that clears its counters; every call leaves
 * them zero again.  All calls on one GPU share the array, so calls that may overlap
 * on one GPU (several streams or host threads without ordering between them) race and
 * give wrong results.  HACK_ERR_HIP if the array cannot be located. */
hack_status hack_attend_decode_noalloc(const hack_kv_layout* layout, const hack_kv_cache* cache,
                                       const void* q_dev, int32_t num_q_heads,
                                       const int32_t* seq_lens_dev, int32_t batch, int32_t max_len,
                                       int32_t tail_mode, float* out_dev, hipStream_t stream);

/* One decode step (Sec. 5.3 with L_Q = 1, and the decode-side quantize-on-write of
 * §6, fused in one launch): for every sequence s and kv head, the new token
 * (k_new_dev / v_new_dev: fp16 [batch][H_kv][head_dim]) is written as token
 * seq_lens_in[s] exactly as hack_append writes it (tail_mode as there), then the
 * query q_dev attends over the seq_lens_in[s] + 1 cached tokens as in
 * hack_attend_decode, and seq_lens_out[s] = seq_lens_in[s] + 1.  The two length
 * arrays must be distinct (callers swap them between steps).  max_len bounds
 * seq_lens_in; max_len + 1 must not exceed the capacity (HACK_ERR_CAPACITY).  The
 * workspace is the one hack_decode_workspace_bytes(layout, batch, H_q, max_len + 1)
 * sizes, with its counters zeroed as for hack_attend_decode.  The step is one launch,
 * except with partition 128, and in DEQUANT mode when H_q/H_kv > 4 (the kv group then
 * spans several workgroups, and one kernel must requantize the open block before any
 * of them reads it): then it is three operations on the stream (a copy of the
 * lengths, the append kernel, the attention kernel). */
hack_status hack_decode_step(const hack_kv_layout* layout, const hack_kv_cache* cache,
                             const void* k_new_dev, const void* v_new_dev, const void* q_dev,
                             int32_t num_q_heads, const int32_t* seq_lens_in_dev,
                             int32_t* seq_lens_out_dev, int32_t batch, int32_t max_len,
                             int32_t tail_mode, float* out_dev, void* workspace_dev,
                             int64_t workspace_bytes, hipStream_t stream);

/* Prefill attention of `len` query tokens per sequence over the quantized cache of
 * the same `len` tokens (Sec. 5.3 with L_Q = L_KV; Eq. 2-4), as written by
 * hack_quantize with all seq_lens = len.  q_dev: fp16 [batch][H_q][len][head_dim];
 * out_dev: fp32 [batch][H_q][len][head_dim].  causal != 0 masks token j > i for
 * query i; the masked zeros of P inside a block are quantized with the block.  The
 * open V block is used in fp16.  Requires head_dim 128, partition 32, 64 or 128, cached
 * code sums, H_q % H_kv == 0, H_q/H_kv <= 8 and batch <= 65535 (else
 * HACK_ERR_UNSUPPORTED). */
hack_status hack_attend_prefill(const hack_kv_layout* layout, const hack_kv_cache* cache,
                                const void* q_dev, int32_t num_q_heads, int32_t batch, int32_t len,
                                int32_t causal, float* out_dev, hipStream_t stream);

/* QKV generation fused with quantize-on-write: the front of the prefill (Sec. 4, Eq. 1,
 * fused as in the paper's prefill kernel, Sec. 6).  For every sequence s and token t <
 * len: out[n] = sum_i E[s][t][i] W[n][i] over the hidden dimension, accumulated in
 * fp32 and rounded to fp16, for n over the output channels of the H_q query heads,
 * then the H_kv key heads, then the H_kv value heads (head_dim 128 channels each).
 *   e_dev:     fp16 [batch][len][hidden], the prompt's embeddings;
 *   w_dev:     fp16 [(H_q + 2 H_kv) * 128][hidden], one row per output channel (the
 *              transposed W_Q, W_K, W_V stacked, as a fused QKV weight);
 *   q_out_dev: fp16 [batch][H_q][len][128], the query heads, in the layout
 *              hack_attend_prefill takes.
 * The key and value heads are not written out: they are quantized into `cache` exactly
 * as hack_quantize quantizes fp16 K and V of length len (codes, min/scale, sums, the
 * open V block in fp16 and re-quantized with n = T), with the layout's rounding.
 * Requires head_dim 128 and hidden a positive multiple of 64 (else HACK_ERR_UNSUPPORTED);
 * HACK_ERR_CAPACITY if len exceeds the cache's capacity.  One kernel. */
hack_status hack_project_qkv(const hack_kv_layout* layout, const hack_kv_cache* cache, const void* e_dev,
                             const void* w_dev, int32_t num_q_heads, int32_t hidden, int32_t batch,
                             int32_t len, void* q_out_dev, hipStream_t stream);

/* The prefill from embeddings (Sec. 6): hack_project_qkv, then hack_attend_prefill on
 * its query heads over the cache it wrote (two kernels on `stream`).  q_out_dev is the
 * caller's fp16 [batch][H_q][len][128] buffer for the query heads; out_dev fp32
 * [batch][H_q][len][128].  The shape limits of both calls apply and are checked before
 * anything is launched. */
hack_status hack_prefill_from_embeddings(const hack_kv_layout* layout, const hack_kv_cache* cache,
                                         const void* e_dev, const void* w_dev, int32_t num_q_heads,
                                         int32_t hidden, int32_t batch, int32_t len, int32_t causal,
                                         void* q_out_dev, float* out_dev, hipStream_t stream);

/* Static, NUL-terminated description of a status code. */
const char* hack_status_string(hack_status status);

/* ---- test exports: integer products of the decode kernel, for bit-exact checks ----
 * Partitions 32 and 64 only (HACK_ERR_UNSUPPORTED for 128). */

/* Runs the decode kernel's QK^T stage only (Sec. 5.3, Eq. 4 integer part).
 * q_codes_dev: u8 [batch][H_q][head_dim] 8-bit Q codes; q_meta_dev: fp32
 * [batch][H_q][P][2] (min, scale) of each Q partition; products_dev: int32
 * [batch][H_q][max_len][P], products_dev[s][h][t][p] = sum over partition p of
 * q'_z k'_{t,z} (unsigned codes) for t < seq_lens[s]; entries past the length are
 * not written. */
hack_status hack_debug_qk_products(const hack_kv_layout* layout, const hack_kv_cache* cache,
                                   const void* q_dev, int32_t num_q_heads,
                                   const int32_t* seq_lens_dev, int32_t batch, int32_t max_len,
                                   uint8_t* q_codes_dev, float* q_meta_dev, int32_t* products_dev,
                                   hipStream_t stream);

/* Runs the decode kernel's P.V stage on injected 8-bit P codes (Sec. 5.3, Eq. 4).
 * p_codes_dev: u8 [batch][H_q][NB][partition] with NB = max_len / partition;
 * p_meta_dev: fp32 [batch][H_q][NB][2] (min, scale).  For every full block k <
 * seq_lens[s]/partition: products_dev (int32 [batch][H_q][NB][head_dim]) receives
 * D'_{k,c} = sum_e p'_e v'_{e,c} and out_dev (fp32 [batch][H_q][head_dim]) the sum
 * over those blocks of Eq. 4 with n = partition. */
hack_status hack_debug_pv_products(const hack_kv_layout* layout, const hack_kv_cache* cache,
                                   const uint8_t* p_codes_dev, const float* p_meta_dev,
                                   int32_t num_q_heads, const int32_t* seq_lens_dev, int32_t batch,
                                   int32_t max_len, int32_t* products_dev, float* out_dev,
                                   hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* HACK_H */
