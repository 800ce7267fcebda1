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
// reduce: 8 (sequence, head) rows per block.
//   1. thread (row, 4 channels): M = max_s m_s, L = sum_s 2^(m_s - M) l_s over
//      the row's splits (empty splits have m_s = -inf and only follow live
//      ones), then o~[c] = sum_s 2^(m_s - M) part_o[s][c] / L over the live
//      splits, with independent loads over s;
//   2. o = o~ R_v^T, R_v copied to LDS with rows padded to 132 floats (16-byte
//      aligned rows; threads of consecutive j read different banks).
// ---------------------------------------------------------------------------
constexpr int kRedRows = 8;
constexpr int kRvPitch4 = kD / 4 + 1;  // row pitch of the LDS copy in float4

// MIXED: a row has num_splits + 1 slots; the last holds the bf16 tokens' state
// in the original basis, o = (sum_s e_s o~_s R_v^T + e_b o_b) / L.
// Rows are taken 8 per block in the natural order, or (rph: one R_v per KV head)
// 8 rows of one KV head per block.
template <bool MIXED>
__global__ __launch_bounds__(256) void reduce_kernel(int rows, int num_splits,
                                                     const float* __restrict__ part_o,
                                                     const float* __restrict__ part_ml,
                                                     const float* __restrict__ Rv,
                                                     void* __restrict__ out, int out_f32, int rph,
                                                     int Hq, int Hkv) {
  __shared__ float4 Rs[kD * kRvPitch4];
  __shared__ float4 om[kRedRows][kD / 4];
  __shared__ float eb_il[kRedRows];  // MIXED: e_b / L per row
  const int stride = MIXED ? num_splits + 1 : num_splits;
  const int t = threadIdx.x;
  int kvh;
  query_row(blockIdx.x, 0, kRedRows, rows, Hq, Hkv, rph, kvh);
  if (Rv && rph) Rv += (size_t)kvh * kD * kD;
  auto row_of = [&](int r) {  // the block's r-th row, or rows (past the end)
    int kv_;
    const int x = query_row(blockIdx.x, r, kRedRows, rows, Hq, Hkv, rph, kv_);
    return x < 0 ? rows : x;
  };
  {  // 8 rows x 32 float4 columns: one (row, float4) per thread
    const int rr = t >> 5, c4 = t & 31, r = row_of(rr);
    float4 o = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    const float2* ml = reinterpret_cast<const float2*>(part_ml + (size_t)r * stride * 2);
    // live slots lead (empty ones only follow the end of a sequence): n_live is
    // one past the last live slot.  Slot s is read by thread s % 32 of the row;
    // maximum and last live slot are then reduced over the row's 32 threads.
    float M = -INFINITY;
    int n_live = 0;
    const float m0 = (r < rows && c4 < num_splits) ? ml[c4].x : -INFINITY;
    float2 mb = make_float2(-INFINITY, 0.0f);
    if (MIXED && r < rows) mb = ml[num_splits];
    // R_v (row-major 128 x 128) to LDS, 16 float4 per thread: loads issued here so
    // that they overlap the slot loads
    float4 v[kD * kD / 4 / 256];
    if (Rv) {
#pragma unroll
      for (int k = 0; k < kD * kD / 4 / 256; ++k) v[k] = reinterpret_cast<const float4*>(Rv)[t + 256 * k];
    }
    if (Rv) {
#pragma unroll
      for (int k = 0; k < kD * kD / 4 / 256; ++k) {
        const int i = t + 256 * k;
        Rs[(i >> 5) * kRvPitch4 + (i & 31)] = v[k];
      }
    }
    M = m0;
    n_live = m0 != -INFINITY ? c4 + 1 : 0;
    if (r < rows)
      for (int s = c4 + 32; s < num_splits; s += 32) {
        const float m = ml[s].x;
        M = fmaxf(M, m);
        n_live = (m != -INFINITY) ? s + 1 : n_live;
      }
#pragma unroll
    for (int off = 16; off >= 1; off >>= 1) {
      M = fmaxf(M, __shfl_xor(M, off, 32));
      n_live = max(n_live, __shfl_xor(n_live, off, 32));
    }
    if (MIXED) M = fmaxf(M, mb.x);
    float ebl = 0.0f;
    if (r < rows) {
      if (M != -INFINITY) {
        const float4* po = reinterpret_cast<const float4*>(part_o + (size_t)r * stride * kD) + c4;
        float L = 0.0f;
        // up to 16 slots per round, loads issued together (indices clamped to the
        // live range, weights of the clamped repeats set to 0)
        for (int s0 = 0; s0 < n_live; s0 += 16) {
          float2 m[16];
          float4 x[16];
#pragma unroll
          for (int k = 0; k < 16; ++k) {
            const int s = min(s0 + k, n_live - 1);
            m[k] = ml[s];
            x[k] = po[(size_t)s * (kD / 4)];
          }
#pragma unroll
          for (int k = 0; k < 16; ++k) {
            const bool use = s0 + k < n_live && m[k].x != -INFINITY;  // empty slots add nothing
            const float e = use ? exp2f(m[k].x - M) : 0.0f;
            L = fmaf(e, use ? m[k].y : 0.0f, L);
            o.x = fmaf(e, use ? x[k].x : 0.0f, o.x); o.y = fmaf(e, use ? x[k].y : 0.0f, o.y);
            o.z = fmaf(e, use ? x[k].z : 0.0f, o.z); o.w = fmaf(e, use ? x[k].w : 0.0f, o.w);
          }
        }
        float eb = 0.0f;
        if (MIXED && mb.x != -INFINITY) {
          eb = exp2f(mb.x - M);
          L = fmaf(eb, mb.y, L);
        }
        const float il = L > 0.0f ? 1.0f / L : 0.0f;
        o.x *= il; o.y *= il; o.z *= il; o.w *= il;
        ebl = eb * il;
      }
    }
    om[rr][c4] = o;
    if (MIXED && c4 == 0) eb_il[rr] = ebl;
  }
  __syncthreads();
  const int j = t & (kD - 1);
  const int rg = (t >> 7) * 4;
  float acc[4];
  if (Rv) {
#pragma unroll
    for (int i = 0; i < 4; ++i) acc[i] = 0.0f;
    const float4* Rj = Rs + j * kRvPitch4;
#pragma unroll 4
    for (int c4 = 0; c4 < kD / 4; ++c4) {
      const float4 rv = Rj[c4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float4 x = om[rg + i][c4];
        acc[i] = fmaf(x.x, rv.x, acc[i]);
        acc[i] = fmaf(x.y, rv.y, acc[i]);
        acc[i] = fmaf(x.z, rv.z, acc[i]);
        acc[i] = fmaf(x.w, rv.w, acc[i]);
      }
    }
  } else {  // R = I (bf16 baseline)
    const float* O = reinterpret_cast<const float*>(om);
#pragma unroll
    for (int i = 0; i < 4; ++i) acc[i] = O[(rg + i) * kD + j];
  }
  if (MIXED) {  // the bf16 tokens' part, already in the original basis
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = row_of(rg + i);
      const float e = eb_il[rg + i];
      if (r < rows && e != 0.0f)
        acc[i] = fmaf(e, part_o[((size_t)r * stride + num_splits) * kD + j], acc[i]);
    }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = row_of(rg + i);
    if (r >= rows) continue;
    if (out_f32) static_cast<float*>(out)[(size_t)r * kD + j] = acc[i];
    else static_cast<uint16_t*>(out)[(size_t)r * kD + j] = f32_to_bf16_rne(acc[i]);
  }
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
  const dim3 grid(query_blocks(B, Hq, Hkv, rph, kRedRows));
  if (mixed)
    hipLaunchKernelGGL(reduce_kernel<true>, grid, dim3(256), 0, st, rows, num_splits, part_o,
                       part_ml, Rv, out, out_f32, rph, Hq, Hkv);
  else
    hipLaunchKernelGGL(reduce_kernel<false>, grid, dim3(256), 0, st, rows, num_splits, part_o,
                       part_ml, Rv, out, out_f32, rph, Hq, Hkv);
  return hipGetLastError();
}

}  // namespace oscar
