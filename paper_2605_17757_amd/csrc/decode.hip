// Decode attention over the INT2 paged cache (Alg. 1 DecodeStep; Sec. 4
// "Decoding Attention Kernel"), in three kernels:
//   prepare : q~ = q R_k * (sm_scale * log2 e)                    [B*Hq, 128] fp32
//             (in append.hip, where it can share a launch with the cache update)
//   split   : online softmax over page ranges in the rotated basis, unnormalized
//             o~ and (m, l) per piece (decode_mfma.hip)
//   reduce  : log-sum-exp merge of the pieces, o = o~ R_v^T, bf16/fp32 store
//             (this file)
//
// Rotated-basis identities used (Sec. 2, K^ = Q(K~) R^T with R orthogonal):
//   q k^T = (q R_k) Q(k~)^T,   sum_t p_t v^_t = (sum_t p_t Q(v~_t)) R_v^T,
// and per group g of 32 channels, with Q(x~)_c = s_g (code_c - z_g):
//   q~ . Q(k~) = sum_g s_g (sum_{c in g} q~_c code_c - z_g sum_{c in g} q~_c).
// Scores are kept in log2 units (q~ carries log2 e) so the softmax uses exp2.
#include <hip/hip_fp16.h>

#include "internal.h"

namespace oscar {
namespace {

__device__ inline uint16_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}


// ---------------------------------------------------------------------------
// reduce: RB = 8 or 16 (sequence, head) rows per block (16 for many rows: each
// block reads R_v once).
//   1. thread (row, 128 / (256 / RB) channels): M = max_s m_s, L = sum_s
//      2^(m_s - M) l_s over
//      the row's splits (empty splits have m_s = -inf and only follow live
//      ones), then o~[c] = sum_s 2^(m_s - M) part_o[s][c] / L over the live
//      splits, with independent loads over s; o~ to LDS;
//   2. o = o~ R_v^T on the fp32 matrix cores: wave w computes column tiles 2w,
//      2w + 1 of the rows (a 16-row tile; rows RB.. of it are zero) as 32 chained
//      16x16x4 MFMAs per tile, step s taking
//      channel c = 32k + s in k-slot k (A: lane (row lo, k-slot hi) reads
//      o~[lo][32hi + s] from LDS; B: lane (column lo, k-slot hi) holds
//      R_v[16t + lo][32hi + s], 128 contiguous bytes of a row of R_v read from L2
//      at the start, before the loads of the partial states).  D lane (column
//      lo, hi): rows 4hi + i.
// ---------------------------------------------------------------------------
constexpr int kOmPitch = kD + 4;  // LDS row pitch of o~ (floats)

typedef float red_f4 __attribute__((ext_vector_type(4)));

// MIXED: a row has num_splits + 1 slots; the last holds the bf16 tokens' state
// in the original basis, o = (sum_s e_s o~_s R_v^T + e_b o_b) / L.
// Rows are taken RB per block in the natural order, or (rph: one R_v per KV
// head) RB rows of one KV head per block.
template <bool MIXED, int RB>
__global__ __launch_bounds__(256) void reduce_kernel(int rows, int num_splits,
                                                     const float* __restrict__ part_o,
                                                     const float* __restrict__ part_ml,
                                                     const float* __restrict__ Rv,
                                                     void* __restrict__ out, int out_f32, int rph,
                                                     int Hq, int Hkv) {
  constexpr int kRedRows = RB;
  constexpr int TPR = 256 / RB;          // threads per row in the merge
  constexpr int NC = 32 / TPR;           // float4 columns per thread
  constexpr int SR = RB == 8 ? 16 : 8;   // slots whose loads are issued together
  __shared__ float om[16 * kOmPitch];
  __shared__ float eb_il[16];  // MIXED: e_b / L per row
  const int stride = MIXED ? num_splits + 1 : num_splits;
  const int t = threadIdx.x, w = t >> 6, lo = t & 15, hi = (t >> 4) & 3;
  int kvh;
  query_row(blockIdx.x, 0, kRedRows, rows, Hq, Hkv, rph, kvh);
  if (Rv && rph) Rv += (size_t)kvh * kD * kD;
  auto row_of = [&](int r) {  // the block's r-th row, or rows (past the end)
    int kv_;
    const int x = query_row(blockIdx.x, r, kRedRows, rows, Hq, Hkv, rph, kv_);
    return x < 0 ? rows : x;
  };
  // R_v operands of the wave's two column tiles, issued first (L2)
  float4 rb[2][8];
  if (Rv) {
#pragma unroll
    for (int tt = 0; tt < 2; ++tt) {
      const float4* src = reinterpret_cast<const float4*>(Rv + (size_t)(16 * (2 * w + tt) + lo) * kD + 32 * hi);
#pragma unroll
      for (int k = 0; k < 8; ++k) rb[tt][k] = src[k];
    }
  }
  if (RB < 16)  // rows RB..15 of the MFMA tile
    for (int i = t; i < (16 - RB) * kOmPitch; i += 256) om[RB * kOmPitch + i] = 0.0f;
  {  // RB rows x TPR threads: thread c8 of a row holds float4 columns c8 + TPR h, h < NC
    const int rr = t / TPR, c8 = t % TPR, r = row_of(rr);
    float4 o[NC];
#pragma unroll
    for (int h = 0; h < NC; ++h) o[h] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    const float2* ml = reinterpret_cast<const float2*>(part_ml + (size_t)r * stride * 2);
    // live slots lead (empty ones only follow the end of a sequence): n_live is
    // one past the last live slot.  Slot s is read by thread s % TPR of the row;
    // maximum and last live slot are then reduced over the row's TPR threads.
    float M = -INFINITY;
    int n_live = 0;
    if (r < rows)
      for (int s = c8; s < num_splits; s += TPR) {
        const float m = ml[s].x;
        M = fmaxf(M, m);
        n_live = (m != -INFINITY) ? s + 1 : n_live;
      }
#pragma unroll
    for (int off = TPR / 2; off >= 1; off >>= 1) {
      M = fmaxf(M, __shfl_xor(M, off, TPR));
      n_live = max(n_live, __shfl_xor(n_live, off, TPR));
    }
    float2 mb = make_float2(-INFINITY, 0.0f);
    if (MIXED && r < rows) mb = ml[num_splits];
    if (MIXED) M = fmaxf(M, mb.x);
    float ebl = 0.0f;
    if (r < rows) {
      if (M != -INFINITY) {
        const float4* po = reinterpret_cast<const float4*>(part_o + (size_t)r * stride * kD) + c8;
        float L = 0.0f;
        // up to SR slots per round, loads issued together (indices clamped to the
        // live range, weights of the clamped repeats set to 0)
        for (int s0 = 0; s0 < n_live; s0 += SR) {
          float2 m[SR];
          float4 x[SR][NC];
#pragma unroll
          for (int k = 0; k < SR; ++k) {
            const int s = min(s0 + k, n_live - 1);
            m[k] = ml[s];
#pragma unroll
            for (int h = 0; h < NC; ++h) x[k][h] = po[(size_t)s * (kD / 4) + TPR * h];
          }
#pragma unroll
          for (int k = 0; k < SR; ++k) {
            const bool use = s0 + k < n_live && m[k].x != -INFINITY;  // empty slots add nothing
            const float e = use ? exp2f(m[k].x - M) : 0.0f;
            L = fmaf(e, use ? m[k].y : 0.0f, L);
#pragma unroll
            for (int h = 0; h < NC; ++h) {
              o[h].x = fmaf(e, use ? x[k][h].x : 0.0f, o[h].x);
              o[h].y = fmaf(e, use ? x[k][h].y : 0.0f, o[h].y);
              o[h].z = fmaf(e, use ? x[k][h].z : 0.0f, o[h].z);
              o[h].w = fmaf(e, use ? x[k][h].w : 0.0f, o[h].w);
            }
          }
        }
        float eb = 0.0f;
        if (MIXED && mb.x != -INFINITY) {
          eb = exp2f(mb.x - M);
          L = fmaf(eb, mb.y, L);
        }
        const float il = L > 0.0f ? 1.0f / L : 0.0f;
#pragma unroll
        for (int h = 0; h < NC; ++h) {
          o[h].x *= il; o[h].y *= il; o[h].z *= il; o[h].w *= il;
        }
        ebl = eb * il;
      }
    }
#pragma unroll
    for (int h = 0; h < NC; ++h)
      *reinterpret_cast<float4*>(&om[rr * kOmPitch + 4 * (c8 + TPR * h)]) = o[h];
    if (MIXED && c8 == 0) eb_il[rr] = ebl;
  }
  __syncthreads();
  // lane (column lo, hi), tile tt: out[row 4hi + i][16 (2w + tt) + lo]
  auto store = [&](int tt, int i, float v) {
    const int rr = 4 * hi + i, col = 16 * (2 * w + tt) + lo;
    if (rr >= RB) return;
    const int r = row_of(rr);
    if (r >= rows) return;
    if (MIXED) {  // the bf16 tokens' part, already in the original basis
      const float e = eb_il[rr];
      if (e != 0.0f) v = fmaf(e, part_o[((size_t)r * stride + num_splits) * kD + col], v);
    }
    if (out_f32) static_cast<float*>(out)[(size_t)r * kD + col] = v;
    else static_cast<uint16_t*>(out)[(size_t)r * kD + col] = f32_to_bf16_rne(v);
  };
  if (!Rv) {  // R = I (bf16 baseline)
#pragma unroll
    for (int tt = 0; tt < 2; ++tt)
#pragma unroll
      for (int i = 0; i < 4; ++i) store(tt, i, om[(4 * hi + i) * kOmPitch + 16 * (2 * w + tt) + lo]);
    return;
  }
  // Both tiles' products first, then their stores, on a path no other branch
  // joins: with the identity case as the other arm of an if/else whose join read
  // the MFMA results, the compiler put no wait states between the last MFMA and
  // the first read of its result (wrong values in one result register).
  red_f4 d[2];
#pragma unroll
  for (int tt = 0; tt < 2; ++tt) {
    d[tt] = red_f4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const float4 a = *reinterpret_cast<const float4*>(&om[lo * kOmPitch + 32 * hi + 4 * k]);
      d[tt] = __builtin_amdgcn_mfma_f32_16x16x4f32(a.x, rb[tt][k].x, d[tt], 0, 0, 0);
      d[tt] = __builtin_amdgcn_mfma_f32_16x16x4f32(a.y, rb[tt][k].y, d[tt], 0, 0, 0);
      d[tt] = __builtin_amdgcn_mfma_f32_16x16x4f32(a.z, rb[tt][k].z, d[tt], 0, 0, 0);
      d[tt] = __builtin_amdgcn_mfma_f32_16x16x4f32(a.w, rb[tt][k].w, d[tt], 0, 0, 0);
    }
  }
  float res[2][4];
#pragma unroll
  for (int tt = 0; tt < 2; ++tt)
#pragma unroll
    for (int i = 0; i < 4; ++i) res[tt][i] = d[tt][i];
#pragma unroll
  for (int tt = 0; tt < 2; ++tt)
#pragma unroll
    for (int i = 0; i < 4; ++i) store(tt, i, res[tt][i]);
}

}  // namespace

hipError_t launch_decode_split(const uint8_t* pages, int Hkv, int B, int Hq,
                               const int32_t* block_table, int max_pages,
                               const int32_t* seq_lens, int num_splits, const float* qt,
                               float* part_o, float* part_ml, hipStream_t st, int meta_bf16,
                               int ng, const MixedSpec* mixed) {
  return launch_decode_split_mfma(pages, Hkv, B, Hq, block_table, max_pages, seq_lens,
                                  num_splits, device_cus(), qt, part_o, part_ml, st,
                                  meta_bf16, ng, mixed);
}

hipError_t launch_decode_reduce(int B, int Hq, int num_splits, const float* part_o,
                                const float* part_ml, const float* Rv, void* out, int out_f32,
                                hipStream_t st, const MixedSpec* mixed, int rph, int Hkv) {
  const int rows = B * Hq;
  // 16 rows per block when there are enough rows to keep every CU busy with them
  const bool wide = rows >= 4096;
  auto go = [&](auto kernel, int rb) {
    hipLaunchKernelGGL(kernel, dim3(query_blocks(B, Hq, Hkv, rph, rb)), dim3(256), 0, st, rows,
                       num_splits, part_o, part_ml, Rv, out, out_f32, rph, Hq, Hkv);
  };
  if (mixed) {
    if (wide) go(reduce_kernel<true, 16>, 16);
    else go(reduce_kernel<true, 8>, 8);
  } else {
    if (wide) go(reduce_kernel<false, 16>, 16);
    else go(reduce_kernel<false, 8>, 8);
  }
  return hipGetLastError();
}

}  // namespace oscar
