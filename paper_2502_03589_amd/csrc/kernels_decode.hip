// Decode attention on quantized K/V (Sec. 5.3 with L_Q = 1; Eq. 2-4).
//
// One 64-lane wavefront per (sequence, kv head, split of the context).  The
// wavefront walks its tokens in spans of four V blocks (4*PI tokens):
//   QK^T  for every 16-token tile: v_mfma_i32_16x16x64_i8 with
//         A = 8-bit Q codes (minus 128) of up to 4 heads x 4 channel quarters,
//             laid out block-diagonally (lane group g carries channel quarter g),
//         B = 2/4-bit K codes unpacked in registers (lane = token, group = quarter),
//         so lane (token t, group h) receives the four quarter products of head h;
//         Eq. 4 with the cached K sums turns them into the score (log2 units).
//   softmax  online per V block (running max), P quantized to 8 bits per block.
//   P.V   v_mfma_i32_16x16x64_i8 with A = P codes (rows = block x head, block-
//         diagonal over the four blocks of the span), B = V codes of 16 channels
//         (lane = channel, group = block): lane (c, group k) receives the integer
//         products of block k for 4 heads, corrected by Eq. 4 with the cached V sums.
//   open block  fp16 values times the unquantized probabilities (TAIL_FP16), or
//         its re-quantized codes with n = T (TAIL_REQUANT).
// Partial (max, sum, O) of each split go to the workspace; the last split to
// arrive for a (sequence, kv head) merges them and writes O (no second launch).
#include "hack_internal.hpp"

namespace hack {

typedef int v4i __attribute__((ext_vector_type(4)));

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
__device__ __forceinline__ void load_words(const uint8_t* p, uint32_t (&w)[N]) {
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

__device__ __forceinline__ float xor_shfl(float x, int m) { return __shfl_xor(x, m, 64); }

// 1/sqrt(128) * log2(e): scores are kept in log2 units so softmax uses exp2.
constexpr float kScoreScale = 0.12751743074941640f;

template <int BITS, int PI, int GT, int MODE>
__global__ __launch_bounds__(64) void decode_kernel(DecodeArgs a) {
  constexpr int D = 128;
  constexpr int P = D / PI;             // K partitions per token (4 or 2)
  constexpr int QPP = 4 / P;            // channel quarters per partition
  constexpr int TILES = PI / 16;        // 16-token tiles per V block
  constexpr int SPAN = 4 * PI;          // tokens per span (four V blocks)
  constexpr int KW = 32 * BITS / 32;    // K code dwords per (token, quarter): 2 or 4
  constexpr int VW = PI * BITS / 32;    // V code dwords per (channel, block)
  constexpr int SW = 16 * BITS / 32;    // code dwords per 16-element slice: 1 or 2
  constexpr int HT = GT * 4;            // head slots

  __shared__ int8_t q_lds[HT][D];
  __shared__ float qm_lds[HT][4][3];
  __shared__ __attribute__((aligned(16))) int8_t p_lds[GT][4][4][PI];   // [rt][block][head][token pos]
  __shared__ __attribute__((aligned(16))) float pst_lds[GT][4][3][4];   // [rt][block][field][head]
  __shared__ __attribute__((aligned(16))) float alpha_lds[GT][4];
  __shared__ __attribute__((aligned(16))) float tailf_lds[GT][4];
  __shared__ float ptail_lds[GT][4][PI];

  const CacheView& c = a.c;
  const int lane = threadIdx.x;
  const int col = lane & 15, grp = lane >> 4;
  const int s = blockIdx.z, hkv = blockIdx.y, split = blockIdx.x;
  const int G = a.group, Hq = a.num_q_heads, H = c.kv_heads;
  // lengths outside [0, max_len] break the caller contract; clamp so that every
  // access stays inside the cache and the workspace
  const int L = max(0, min(a.lens[s], a.max_len));
  const int t0 = split * a.chunk;
  if (t0 >= L) {
    if (MODE == MODE_ATTEND && split == 0) {  // empty sequence: zeros
      for (int gh = 0; gh < G; ++gh) {
        float* o = a.out + ((int64_t)s * Hq + hkv * G + gh) * D;
        o[lane] = 0.0f;
        o[lane + 64] = 0.0f;
      }
    }
    return;
  }
  const int t1 = min(L, t0 + a.chunk);
  const int nsplit = (L + a.chunk - 1) / a.chunk;
  const int F = L / PI, T = L - F * PI;
  const bool requant = a.tail_requant != 0;

  // ---- Q: 8-bit codes per partition with float32 metadata (Sec. 5.1, Sec. 5.2) ----
  v4i qa[GT][2];
  float qc[GT][P][3];
  if constexpr (MODE != MODE_PV) {
    for (int gh = 0; gh < HT; ++gh) {
      const bool real = gh < G;
      const int hq = hkv * G + gh;
      float x0 = 0.0f, x1 = 0.0f;
      if (real) {
        const __half2 v2 = reinterpret_cast<const __half2*>(a.q + ((int64_t)s * Hq + hq) * D)[lane];
        const float2 f = __half22float2(v2);
        x0 = f.x;
        x1 = f.y;
      }
      // partition of this lane's two channels: lanes [p*PI/2, (p+1)*PI/2)
      float mn = fminf(x0, x1), mx = fmaxf(x0, x1);
#pragma unroll
      for (int m = 1; m < PI / 2; m <<= 1) {
        mn = fminf(mn, xor_shfl(mn, m));
        mx = fmaxf(mx, xor_shfl(mx, m));
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
    __syncthreads();
    // A operands: lane (row = 4*head + quarter, group g) is non-zero only when quarter == g.
#pragma unroll
    for (int rt = 0; rt < GT; ++rt) {
      const int hh = col >> 2, qq = col & 3;
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
#pragma unroll
      for (int p = 0; p < P; ++p)
#pragma unroll
        for (int f = 0; f < 3; ++f) qc[rt][p][f] = qm_lds[rt * 4 + grp][p][f];
    }
  }

  float m_run[GT], l_run[GT];
  float o_acc[GT][8][4];
#pragma unroll
  for (int rt = 0; rt < GT; ++rt) {
    m_run[rt] = -INFINITY;
    l_run[rt] = 0.0f;
#pragma unroll
    for (int j = 0; j < 8; ++j)
#pragma unroll
      for (int hh = 0; hh < 4; ++hh) o_acc[rt][j][hh] = 0.0f;
  }

  for (int span0 = t0; span0 < t1; span0 += SPAN) {
    float m_start[GT];
    float m_blk[GT][4], ps_s[GT][4], ps_m[GT][4];
    int ps_sum[GT][4];
    int kF = -1;  // position of the fp16 open block in this span (TAIL_FP16 only)
#pragma unroll
    for (int rt = 0; rt < GT; ++rt) m_start[rt] = m_run[rt];

    // ---------------- QK^T, softmax and P quantization, one V block at a time ------------
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int bt0 = span0 + k * PI;  // first token of the block (wave-uniform)
      const int kb = bt0 / PI;
      const bool present = bt0 < L;
      const bool quantized = present && (kb < F || requant);
      if (present && kb == F && !requant) kF = k;
#pragma unroll
      for (int rt = 0; rt < GT; ++rt) {
        m_blk[rt][k] = m_run[rt];
        ps_s[rt][k] = 0.0f;
        ps_m[rt][k] = 0.0f;
        ps_sum[rt][k] = 0;
      }
      if constexpr (MODE == MODE_PV) {
        // injected P codes of full blocks
        if (lane < 16 * GT) {
          const int rt = lane >> 4, hh = (lane >> 2) & 3, part = lane & 3;
          const int gh = rt * 4 + hh;
          const int NB = a.max_len / PI;
          const bool ok = present && kb < F && gh < G;
          for (int e = part * (PI / 4); e < (part + 1) * (PI / 4); ++e) {
            int8_t v = 0;
            if (ok) v = (int8_t)((int)a.dbg_pcodes[(((int64_t)s * Hq + hkv * G + gh) * NB + kb) * PI + e] - 128);
            p_lds[rt][k][hh][(e >> 4) * 16 + perm_position<BITS>(e & 15)] = v;
          }
        }
        if (lane < 4 * GT) {
          const int rt = lane >> 2, hh = lane & 3, gh = rt * 4 + hh;
          const int NB = a.max_len / PI;
          float pm = 0.0f, ps = 0.0f, sum = 0.0f;
          if (present && kb < F && gh < G) {
            const int64_t base = ((int64_t)s * Hq + hkv * G + gh) * NB + kb;
            pm = a.dbg_pmeta[base * 2 + 0];
            ps = a.dbg_pmeta[base * 2 + 1];
            int tot = 0;
            for (int e = 0; e < PI; ++e) tot += a.dbg_pcodes[base * PI + e];
            sum = (float)tot;
          }
          pst_lds[rt][k][0][hh] = ps;
          pst_lds[rt][k][1][hh] = pm;
          pst_lds[rt][k][2][hh] = sum;
        }
        continue;
      } else {
        float sv[GT][TILES];
        if (present) {
          const int64_t page = page_of(c, s, bt0);
          const int64_t krow0 = (page * H + hkv) * c.page_tokens + (bt0 % c.page_tokens);
#pragma unroll
          for (int ti = 0; ti < TILES; ++ti) {
            const int tok = bt0 + 16 * ti + col;
            const bool valid = tok < L;
            uint32_t kw[KW];
            float km[P], ks[P], kz[P];
            if (valid) {
              const int64_t row = krow0 + 16 * ti + col;
              const uint32_t* src = reinterpret_cast<const uint32_t*>(c.k_codes + row * (D * BITS / 8)) + grp * KW;
              if constexpr (KW == 2) {
                const uint2 w = *reinterpret_cast<const uint2*>(src);
                kw[0] = w.x;
                kw[1] = w.y;
              } else {
                const uint4 w = *reinterpret_cast<const uint4*>(src);
                kw[0] = w.x;
                kw[1] = w.y;
                kw[2] = w.z;
                kw[3] = w.w;
              }
#pragma unroll
              for (int p = 0; p < P; ++p) {
                const float2 f = __half22float2(c.k_meta[row * P + p]);
                km[p] = f.x;
                ks[p] = f.y;
                kz[p] = (float)load_sum(c.k_sums, row * P + p, c.sum_bytes);
              }
            } else {
#pragma unroll
              for (int w = 0; w < KW; ++w) kw[w] = 0u;
#pragma unroll
              for (int p = 0; p < P; ++p) km[p] = ks[p] = kz[p] = 0.0f;
            }
            const v4i b0 = unpack16<BITS>(kw);
            const v4i b1 = unpack16<BITS>(kw + SW);
#pragma unroll
            for (int rt = 0; rt < GT; ++rt) {
              v4i acc = v4i{0, 0, 0, 0};
              acc = mfma_i8(qa[rt][0], b0, acc);
              acc = mfma_i8(qa[rt][1], b1, acc);
              float sc = 0.0f;
#pragma unroll
              for (int p = 0; p < P; ++p) {
                int cp = 0;
#pragma unroll
                for (int qq = 0; qq < QPP; ++qq) cp += acc[p * QPP + qq];
                // Eq. 4 (log2 units): s_k (s_q C~ + m~_q sum k') + m_k (s_q sum q' + n m_q)
                const float z = fmaf(qc[rt][p][0], (float)cp, qc[rt][p][1] * kz[p]);
                sc = fmaf(ks[p], z, sc);
                sc = fmaf(km[p], qc[rt][p][2], sc);
                if constexpr (MODE == MODE_QK) {
                  const int gh = rt * 4 + grp;
                  if (valid && gh < G)
                    a.dbg_prod[(((int64_t)s * Hq + hkv * G + gh) * a.max_len + tok) * P + p] =
                        cp + 128 * (int)kz[p];
                }
              }
              sv[rt][ti] = valid ? sc : -INFINITY;
            }
          }
        }
        if constexpr (MODE == MODE_QK) continue;
        if (!present) {  // block past the end: no P codes, zero statistics
          for (int i = lane; i < GT * PI; i += 64)
            reinterpret_cast<int*>(&p_lds[i / PI][k][0][0])[i % PI] = 0;
          continue;
        }
#pragma unroll
        for (int rt = 0; rt < GT; ++rt) {
          float bmax = sv[rt][0];
#pragma unroll
          for (int ti = 1; ti < TILES; ++ti) bmax = fmaxf(bmax, sv[rt][ti]);
          bmax = row16_max(bmax);
          const float m_new = fmaxf(m_run[rt], bmax);
          const float alpha = __builtin_amdgcn_exp2f(m_run[rt] - m_new);
          float pt[TILES];
          float lsum = 0.0f, pmin = INFINITY, pmax = 0.0f;
#pragma unroll
          for (int ti = 0; ti < TILES; ++ti) {
            pt[ti] = __builtin_amdgcn_exp2f(sv[rt][ti] - m_new);
            lsum += pt[ti];
            const bool valid = bt0 + 16 * ti + col < L;
            if (valid) {
              pmin = fminf(pmin, pt[ti]);
              pmax = fmaxf(pmax, pt[ti]);
            }
          }
          l_run[rt] = fmaf(l_run[rt], alpha, lsum);
          m_run[rt] = m_new;
          m_blk[rt][k] = m_new;
          if (quantized) {
            pmin = row16_min(pmin);
            pmax = row16_max(pmax);
            const float sp = (pmax - pmin) * (1.0f / 255.0f);
            const float r = sp > 0.0f ? __builtin_amdgcn_rcpf(sp) : 0.0f;
            int csum = 0;
#pragma unroll
            for (int ti = 0; ti < TILES; ++ti) {
              const bool valid = bt0 + 16 * ti + col < L;
              const int code = valid ? (int)fminf(rintf((pt[ti] - pmin) * r), 255.0f) : 0;
              csum += code;
              p_lds[rt][k][grp][ti * 16 + perm_position<BITS>(col)] = valid ? (int8_t)(code - 128) : (int8_t)0;
            }
            csum = row16_sum_i(csum);
            ps_s[rt][k] = sp;
            ps_m[rt][k] = pmin;
            ps_sum[rt][k] = csum;
          } else {
#pragma unroll
            for (int ti = 0; ti < TILES; ++ti) {
              p_lds[rt][k][grp][ti * 16 + perm_position<BITS>(col)] = 0;
              ptail_lds[rt][grp][ti * 16 + col] = pt[ti];  // open block: unquantized p
            }
          }
        }
      }
    }
    if constexpr (MODE == MODE_QK) continue;

    if constexpr (MODE != MODE_PV) {
      // scale factors from each block's running max to the span's final max
      if (col == 0) {
#pragma unroll
        for (int rt = 0; rt < GT; ++rt) {
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            const float f = __builtin_amdgcn_exp2f(m_blk[rt][k] - m_run[rt]);
            pst_lds[rt][k][0][grp] = ps_s[rt][k] * f;
            pst_lds[rt][k][1][grp] = ps_m[rt][k] * f;
            pst_lds[rt][k][2][grp] = (float)ps_sum[rt][k];
            if (k == kF) tailf_lds[rt][grp] = f;
          }
          alpha_lds[rt][grp] = __builtin_amdgcn_exp2f(m_start[rt] - m_run[rt]);
        }
      }
    }
    __syncthreads();

    // ---------------- P.V: lane (channel col, group = block k of the span) ----------------
    {
      const int bt0 = span0 + grp * PI;
      const int kb = bt0 / PI;
      bool gvalid = bt0 < L && (kb < F || (requant && kb == F && T > 0));
      if constexpr (MODE == MODE_PV) gvalid = bt0 < L && kb < F;
      const float n_g = (float)(kb < F ? PI : T);
      int64_t vb = 0;
      if (gvalid) vb = v_block<PI>(c, s, hkv, bt0);
      // V metadata of channels 8*col .. 8*col+7 of this lane's block
      float vs_[8], vm_[8], vw_[8], vbar_[8];
      uint32_t zs[8] = {0, 0, 0, 0, 0, 0, 0, 0};
      {
        uint4 mraw[2] = {uint4{0, 0, 0, 0}, uint4{0, 0, 0, 0}};
        if (gvalid) {
          const uint4* mp = reinterpret_cast<const uint4*>(c.v_meta + vb * D + 8 * col);
          mraw[0] = mp[0];
          mraw[1] = mp[1];
          if (c.sum_bytes == 1) {
            const uint2 z = *reinterpret_cast<const uint2*>(c.v_sums + vb * D + 8 * col);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              zs[j] = (z.x >> (8 * j)) & 0xFFu;
              zs[4 + j] = (z.y >> (8 * j)) & 0xFFu;
            }
          } else {
            const uint4 z = *reinterpret_cast<const uint4*>(reinterpret_cast<const uint16_t*>(c.v_sums) + vb * D + 8 * col);
            const uint32_t zz[4] = {z.x, z.y, z.z, z.w};
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              zs[2 * j] = zz[j] & 0xFFFFu;
              zs[2 * j + 1] = zz[j] >> 16;
            }
          }
        }
        const uint32_t mw[8] = {mraw[0].x, mraw[0].y, mraw[0].z, mraw[0].w,
                                mraw[1].x, mraw[1].y, mraw[1].z, mraw[1].w};
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const float mv = __half2float(__ushort_as_half((uint16_t)(mw[j] & 0xFFFFu)));
          const float sv = __half2float(__ushort_as_half((uint16_t)(mw[j] >> 16)));
          const float vsum = sv * (float)zs[j];
          vs_[j] = sv;
          vm_[j] = mv;
          vw_[j] = 128.0f * vsum;
          vbar_[j] = fmaf(n_g, mv, vsum);
        }
      }
      // P codes (A operand): lane (row = 4*block + head, group g) non-zero only when block == g
      v4i pa[GT][TILES];
      float sp_[GT][4], mp_[GT][4], zp_[GT][4];
#pragma unroll
      for (int rt = 0; rt < GT; ++rt) {
        const int kk = col >> 2, hh = col & 3;
#pragma unroll
        for (int sl = 0; sl < TILES; ++sl) {
          if (kk == grp) {
            const int4 w = *reinterpret_cast<const int4*>(&p_lds[rt][kk][hh][sl * 16]);
            pa[rt][sl] = v4i{w.x, w.y, w.z, w.w};
          } else {
            pa[rt][sl] = v4i{0, 0, 0, 0};
          }
        }
        const float4 f0 = *reinterpret_cast<const float4*>(&pst_lds[rt][grp][0][0]);
        const float4 f1 = *reinterpret_cast<const float4*>(&pst_lds[rt][grp][1][0]);
        const float4 f2 = *reinterpret_cast<const float4*>(&pst_lds[rt][grp][2][0]);
        sp_[rt][0] = f0.x; sp_[rt][1] = f0.y; sp_[rt][2] = f0.z; sp_[rt][3] = f0.w;
        mp_[rt][0] = f1.x; mp_[rt][1] = f1.y; mp_[rt][2] = f1.z; mp_[rt][3] = f1.w;
        zp_[rt][0] = f2.x; zp_[rt][1] = f2.y; zp_[rt][2] = f2.z; zp_[rt][3] = f2.w;
        if constexpr (MODE != MODE_PV) {
          const float4 al = *reinterpret_cast<const float4*>(&alpha_lds[rt][0]);
          const float alv[4] = {al.x, al.y, al.z, al.w};
#pragma unroll
          for (int j = 0; j < 8; ++j)
#pragma unroll
            for (int hh2 = 0; hh2 < 4; ++hh2) o_acc[rt][j][hh2] *= alv[hh2];
        }
      }
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int ch = 8 * col + j;
        uint32_t vw[VW];
        if (gvalid) {
          load_words<VW>(c.v_codes + (vb * D + ch) * (PI * BITS / 8), vw);
        } else {
#pragma unroll
          for (int w = 0; w < VW; ++w) vw[w] = 0u;
        }
#pragma unroll
        for (int rt = 0; rt < GT; ++rt) {
          v4i acc = v4i{0, 0, 0, 0};
#pragma unroll
          for (int sl = 0; sl < TILES; ++sl) acc = mfma_i8(pa[rt][sl], unpack16<BITS>(vw + sl * SW), acc);
#pragma unroll
          for (int hh = 0; hh < 4; ++hh) {
            // Eq. 4: s_p (s_v D~ + m_v sum p' + 128 s_v sum v') + m_p (s_v sum v' + n m_v)
            const float y = fmaf(vm_[j], zp_[rt][hh], vw_[j]);
            const float z = fmaf(vs_[j], (float)acc[hh], y);
            float o = fmaf(sp_[rt][hh], z, o_acc[rt][j][hh]);
            o_acc[rt][j][hh] = fmaf(mp_[rt][hh], vbar_[j], o);
            if constexpr (MODE == MODE_PV) {
              const int gh = rt * 4 + hh;
              if (gvalid && gh < G)
                a.dbg_prod[(((int64_t)s * Hq + hkv * G + gh) * (a.max_len / PI) + kb) * D + ch] =
                    acc[hh] + 128 * (int)zs[j];
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
        float tf[GT][4];
#pragma unroll
        for (int rt = 0; rt < GT; ++rt) {
          const float4 f = *reinterpret_cast<const float4*>(&tailf_lds[rt][0]);
          tf[rt][0] = f.x; tf[rt][1] = f.y; tf[rt][2] = f.z; tf[rt][3] = f.w;
        }
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
            for (int hh = 0; hh < 4; ++hh) {
              const float p = ptail_lds[rt][hh][e] * tf[rt][hh];
#pragma unroll
              for (int j = 0; j < 8; ++j) o_acc[rt][j][hh] = fmaf(p, vv[j], o_acc[rt][j][hh]);
            }
        }
      }
    }
    __syncthreads();
  }
  if constexpr (MODE == MODE_QK) return;

  // ---- reduce over the four lane groups: every group then holds O for all heads ----
#pragma unroll
  for (int rt = 0; rt < GT; ++rt)
#pragma unroll
    for (int j = 0; j < 8; ++j)
#pragma unroll
      for (int hh = 0; hh < 4; ++hh) {
        float v = o_acc[rt][j][hh];
        v += xor_shfl(v, 16);
        v += xor_shfl(v, 32);
        o_acc[rt][j][hh] = v;
      }

  if constexpr (MODE == MODE_PV) {
#pragma unroll
    for (int rt = 0; rt < GT; ++rt) {
      const int gh = rt * 4 + grp;
      if (gh < G) {
        float* o = a.out + ((int64_t)s * Hq + hkv * G + gh) * D + 8 * col;
#pragma unroll
        for (int j = 0; j < 8; ++j) o[j] = o_acc[rt][j][grp];
      }
    }
    return;
  } else {
    // lane group grp now writes head rt*4 + grp; its max and sum live in the same lanes
    float l_fin[GT];
#pragma unroll
    for (int rt = 0; rt < GT; ++rt) l_fin[rt] = row16_sum(l_run[rt]);
    if (nsplit == 1) {
#pragma unroll
      for (int rt = 0; rt < GT; ++rt) {
        const int gh = rt * 4 + grp;
        if (gh < G) {
          const float inv = 1.0f / l_fin[rt];
          float* o = a.out + ((int64_t)s * Hq + hkv * G + gh) * D + 8 * col;
          const float4 v0 = {o_acc[rt][0][grp] * inv, o_acc[rt][1][grp] * inv, o_acc[rt][2][grp] * inv,
                             o_acc[rt][3][grp] * inv};
          const float4 v1 = {o_acc[rt][4][grp] * inv, o_acc[rt][5][grp] * inv, o_acc[rt][6][grp] * inv,
                             o_acc[rt][7][grp] * inv};
          reinterpret_cast<float4*>(o)[0] = v0;
          reinterpret_cast<float4*>(o)[1] = v1;
        }
      }
      return;
    }
    const int64_t pair = (int64_t)s * H + hkv;
    constexpr int REC = 2 + D;
#pragma unroll
    for (int rt = 0; rt < GT; ++rt) {
      const int gh = rt * 4 + grp;
      if (gh < G) {
        float* rec = a.partials + ((pair * a.splits + split) * G + gh) * REC;
        if (col == 0) {
          rec[0] = m_run[rt];
          rec[1] = l_fin[rt];
        }
#pragma unroll
        for (int j = 0; j < 8; ++j) rec[2 + 8 * col + j] = o_acc[rt][j][grp];
      }
    }
    __threadfence();
    int prior = 0;
    if (lane == 0) prior = atomicAdd(&a.counters[pair], 1);
    prior = __shfl(prior, 0, 64);
    if (prior != nsplit - 1) return;
    __threadfence();
    // last arrival: merge the nsplit partial results of this (sequence, kv head)
    for (int gh = 0; gh < G; ++gh) {
      float mmax = -INFINITY;
      for (int sp = 0; sp < nsplit; ++sp)
        mmax = fmaxf(mmax, a.partials[((pair * a.splits + sp) * G + gh) * REC]);
      float lsum = 0.0f, o0 = 0.0f, o1 = 0.0f;
      for (int sp = 0; sp < nsplit; ++sp) {
        const float* rec = a.partials + ((pair * a.splits + sp) * G + gh) * REC;
        const float w = __builtin_amdgcn_exp2f(rec[0] - mmax);
        lsum = fmaf(rec[1], w, lsum);
        o0 = fmaf(rec[2 + lane], w, o0);
        o1 = fmaf(rec[2 + 64 + lane], w, o1);
      }
      const float inv = 1.0f / lsum;
      float* o = a.out + ((int64_t)s * Hq + hkv * G + gh) * D;
      o[lane] = o0 * inv;
      o[lane + 64] = o1 * inv;
    }
    if (lane == 0) atomicExch(&a.counters[pair], 0);
  }
}

}  // namespace hack

namespace hack {

DecodePlan plan_decode(const hack_kv_layout& lay, int batch, int num_q_heads, int max_len) {
  DecodePlan p{};
  const int64_t span = 4 * lay.partition;
  const int64_t pairs = (int64_t)batch * lay.num_kv_heads;
  const int64_t G = lay.num_kv_heads > 0 ? num_q_heads / lay.num_kv_heads : 0;
  // about 8 workgroups per compute unit of a 256-CU device, at least one span each
  const int64_t target = 2048;
  int64_t chunk = pairs > 0 ? ((int64_t)max_len * pairs + target - 1) / target : span;
  chunk = ((chunk + span - 1) / span) * span;
  if (chunk < span) chunk = span;
  p.chunk = (int)chunk;
  p.splits = max_len > 0 ? (int)(((int64_t)max_len + chunk - 1) / chunk) : 1;
  p.partial_floats = pairs * p.splits * G * (2 + lay.head_dim);
  p.counter_offset = ((p.partial_floats * 4 + 255) / 256) * 256;
  p.workspace_bytes = p.counter_offset + ((pairs * 4 + 255) / 256) * 256;
  return p;
}

template <int BITS, int PI, int GT, int MODE>
static hipError_t decode_impl(const DecodeArgs& a, int batch, hipStream_t stream) {
  dim3 grid((unsigned)a.splits, (unsigned)a.c.kv_heads, (unsigned)batch);
  hipLaunchKernelGGL((decode_kernel<BITS, PI, GT, MODE>), grid, dim3(64), 0, stream, a);
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
