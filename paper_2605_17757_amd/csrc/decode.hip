// Decode attention over the INT2 paged cache (Alg. 1 DecodeStep; Sec. 4
// "Decoding Attention Kernel"), in three kernels:
//   prepare : q~ = q R_k * (sm_scale * log2 e)                    [B*Hq, 128] fp32
//             (in append.hip, where it can share a launch with the cache update)
//   split   : per (split, kv-head, sequence) block, online softmax over the
//             split's pages in the rotated basis, unnormalized o~ and (m, l)
//   reduce  : log-sum-exp merge of the splits, o = o~ R_v^T, bf16/fp32 store
//
// Rotated-basis identities used (Sec. 2, K^ = Q(K~) R^T with R orthogonal):
//   q k^T = (q R_k) Q(k~)^T,   sum_t p_t v^_t = (sum_t p_t Q(v~_t)) R_v^T,
// and per group g of 32 channels, with Q(x~)_c = s_g (code_c - z_g):
//   q~ . Q(k~) = sum_g s_g (sum_{c in g} q~_c code_c - z_g sum_{c in g} q~_c).
// Scores are kept in log2 units (q~ carries log2 e) so the softmax uses exp2.
#include <hip/hip_fp16.h>
#include <stdlib.h>

#include "internal.h"

namespace oscar {
namespace {

__device__ inline float f16_lo(uint32_t w) { return __half2float(__ushort_as_half((uint16_t)(w & 0xffffu))); }
__device__ inline float f16_hi(uint32_t w) { return __half2float(__ushort_as_half((uint16_t)(w >> 16))); }
__device__ inline float bf16_to_f32(uint16_t h) { return __uint_as_float(((uint32_t)h) << 16); }
__device__ inline uint16_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

__device__ inline float wave_max(float x) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) x = fmaxf(x, __shfl_xor(x, m, 64));
  return x;
}
__device__ inline float wave_sum(float x) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) x += __shfl_xor(x, m, 64);
  return x;
}

// ---------------------------------------------------------------------------
// split: block (split s, kv-head, sequence b), 4 waves.  Pages of the split are
// dealt round-robin to the waves; each wave keeps its own online-softmax state
// and the four states are merged at the end.
//   phase 1  lane = token slot: scores for all NH heads from the packed codes
//   phase 2  per head: page max, rescale factor, p = exp2(score - m)
//   phase 3  lane = channels (l, l+64): o~ += (p s_v) (code - z_v)
// ---------------------------------------------------------------------------
constexpr int kWaves = 4;
constexpr int kVcStride = 72;  // bytes per quad row of staged V codes (bank spread)

template <int NH>
struct SplitSmem {
  float qs[kD][NH];                  // q~, [channel][head]
  float qsum[kNG][NH];               // per-group sums of q~
  float wz[kWaves][kP][kNG][NH + 1]; // per token/group: z_v, then p*s_v for each head
  uint8_t vc[kWaves][32 * kVcStride];
  float mm[kWaves][NH], ll[kWaves][NH];
};

template <int NH>
__global__ __launch_bounds__(256) void split_kernel(
    const uint8_t* __restrict__ pages, int Hkv, int Hq, const int32_t* __restrict__ block_table,
    int max_pages, const int32_t* __restrict__ seq_lens, int num_splits, int pages_per_split,
    const float* __restrict__ qt, float* __restrict__ part_o, float* __restrict__ part_ml) {
  extern __shared__ __align__(16) uint8_t smem_raw[];
  SplitSmem<NH>& sm = *reinterpret_cast<SplitSmem<NH>*>(smem_raw);

  const int s = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
  const int g = Hq / Hkv;
  const int len = seq_lens[b];
  const int npg = (len + kP - 1) / kP;
  const int p0 = s * pages_per_split;
  const int p1 = min(npg, p0 + pages_per_split);
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;

  for (int i = threadIdx.x; i < kD * NH; i += blockDim.x) {
    const int c = i / NH, h = i % NH;
    sm.qs[c][h] = (h < g) ? qt[((size_t)b * Hq + kvh * g + h) * kD + c] : 0.0f;
  }
  __syncthreads();
  if (threadIdx.x < kNG * NH) {
    const int G = threadIdx.x / NH, h = threadIdx.x % NH;
    float acc = 0.0f;
    for (int c = 0; c < kG; ++c) acc += sm.qs[G * kG + c][h];
    sm.qsum[G][h] = acc;
  }
  __syncthreads();

  float m[NH], lsum[NH], acc0[NH], acc1[NH];
#pragma unroll
  for (int h = 0; h < NH; ++h) { m[h] = -INFINITY; lsum[h] = 0.0f; acc0[h] = acc1[h] = 0.0f; }

  const int32_t* __restrict__ bt = block_table + (size_t)b * max_pages;
  for (int pr = p0; pr < p1; pr += kWaves) {
    const int pg = pr + w;
    const bool active = pg < p1;
    const int tok0 = pg * kP;
    const int ntok = active ? min(kP, len - tok0) : 0;
    const uint8_t* blk = nullptr;
    if (active) blk = pages + ((size_t)bt[pg] * Hkv + kvh) * kBlockBytes;

    // ---- phase 1: scores (lane = token slot) ----
    float p[NH];
    const bool valid = l < ntok;
    uint32_t kc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    uint32_t ksz[kNG] = {0, 0, 0, 0}, vsz[kNG] = {0, 0, 0, 0};
    if (valid) {
      const uint4* src = reinterpret_cast<const uint4*>(blk + kOffKCodes + l * (kD / 4));
      const uint4 a = src[0], c4 = src[1];
      kc[0] = a.x; kc[1] = a.y; kc[2] = a.z; kc[3] = a.w;
      kc[4] = c4.x; kc[5] = c4.y; kc[6] = c4.z; kc[7] = c4.w;
#pragma unroll
      for (int G = 0; G < kNG; ++G) {
        ksz[G] = *reinterpret_cast<const uint32_t*>(blk + kOffKSz + (G * kP + l) * 4);
        vsz[G] = *reinterpret_cast<const uint32_t*>(blk + kOffVSz + (G * kP + l) * 4);
      }
    }
    float score[NH], dot[NH];
#pragma unroll
    for (int h = 0; h < NH; ++h) score[h] = dot[h] = 0.0f;
    // word wd of the token's codes holds channels 16*wd .. 16*wd+15 (2 bits each)
#pragma unroll
    for (int wd = 0; wd < 8; ++wd) {
      const uint32_t word = kc[wd];
#pragma unroll 2
      for (int k = 0; k < 16; ++k) {
        const float cf = (float)((word >> (2 * k)) & 3u);
        const float* qrow = sm.qs[wd * 16 + k];
#pragma unroll
        for (int h = 0; h < NH; ++h) dot[h] = fmaf(qrow[h], cf, dot[h]);
      }
      if (wd & 1) {  // group wd/2 complete: score += s * (dot - z * sum(q~))
        const int G = wd >> 1;
        const float sG = f16_lo(ksz[G]), zG = f16_hi(ksz[G]);
#pragma unroll
        for (int h = 0; h < NH; ++h) {
          score[h] = fmaf(sG, fmaf(-zG, sm.qsum[G][h], dot[h]), score[h]);
          dot[h] = 0.0f;
        }
      }
    }

    // ---- phase 2: online softmax per head (wave-wide) ----
    float alpha[NH];
#pragma unroll
    for (int h = 0; h < NH; ++h) {
      const float sc = valid ? score[h] : -INFINITY;
      const float mx = active ? wave_max(sc) : -INFINITY;
      const float mn = fmaxf(m[h], mx);
      alpha[h] = (mn == -INFINITY) ? 1.0f : exp2f(m[h] - mn);
      p[h] = valid ? exp2f(sc - mn) : 0.0f;
      lsum[h] = lsum[h] * alpha[h] + (active ? wave_sum(p[h]) : 0.0f);
      m[h] = mn;
    }
    if (valid) {
#pragma unroll
      for (int G = 0; G < kNG; ++G) {
        const float sV = f16_lo(vsz[G]);
        float* row = sm.wz[w][l][G];
        row[0] = f16_hi(vsz[G]);
#pragma unroll
        for (int h = 0; h < NH; ++h) row[1 + h] = p[h] * sV;
      }
    }
    if (active) {
      // stage the V code block: lane l copies 32 bytes (quad l/2, tokens (l%2)*32..+31)
      const uint2* src = reinterpret_cast<const uint2*>(blk + kOffVCodes + l * 32);
      uint2* dst = reinterpret_cast<uint2*>(&sm.vc[w][(l >> 1) * kVcStride + (l & 1) * 32]);
#pragma unroll
      for (int i = 0; i < 4; ++i) dst[i] = src[i];
    }
    __syncthreads();

    // ---- phase 3: P.V in the rotated basis (lane = channels l, l+64) ----
#pragma unroll
    for (int h = 0; h < NH; ++h) { acc0[h] *= alpha[h]; acc1[h] *= alpha[h]; }
    const int q0 = l >> 2, q1 = 16 + (l >> 2), sh = 2 * (l & 3);
    const int G0 = l >> 5, G1 = 2 + (l >> 5);
    for (int t4 = 0; t4 < ntok; t4 += 4) {
      const uint32_t d0 = *reinterpret_cast<const uint32_t*>(&sm.vc[w][q0 * kVcStride + t4]);
      const uint32_t d1 = *reinterpret_cast<const uint32_t*>(&sm.vc[w][q1 * kVcStride + t4]);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int t = t4 + i;
        if (t >= ntok) break;
        const float* r0 = sm.wz[w][t][G0];
        const float* r1 = sm.wz[w][t][G1];
        const float dv0 = (float)((d0 >> (8 * i + sh)) & 3u) - r0[0];
        const float dv1 = (float)((d1 >> (8 * i + sh)) & 3u) - r1[0];
#pragma unroll
        for (int h = 0; h < NH; ++h) {
          acc0[h] = fmaf(r0[1 + h], dv0, acc0[h]);
          acc1[h] = fmaf(r1[1 + h], dv1, acc1[h]);
        }
      }
    }
    __syncthreads();
  }

  // ---- merge the four wave states ----
  float* ao = &sm.wz[0][0][0][0];  // reuse: [kWaves][NH][kD]
  if (l == 0) {
#pragma unroll
    for (int h = 0; h < NH; ++h) { sm.mm[w][h] = m[h]; sm.ll[w][h] = lsum[h]; }
  }
#pragma unroll
  for (int h = 0; h < NH; ++h) {
    ao[(w * NH + h) * kD + l] = acc0[h];
    ao[(w * NH + h) * kD + l + 64] = acc1[h];
  }
  __syncthreads();
  for (int i = threadIdx.x; i < g * kD; i += blockDim.x) {
    const int h = i / kD, c = i % kD;
    float M = -INFINITY;
#pragma unroll
    for (int ww = 0; ww < kWaves; ++ww) M = fmaxf(M, sm.mm[ww][h]);
    float o = 0.0f, L = 0.0f;
    if (M != -INFINITY) {
#pragma unroll
      for (int ww = 0; ww < kWaves; ++ww) {
        const float e = exp2f(sm.mm[ww][h] - M);
        o += e * ao[(ww * NH + h) * kD + c];
        L += e * sm.ll[ww][h];
      }
    }
    const size_t row = ((size_t)b * Hq + kvh * g + h) * num_splits + s;
    part_o[row * kD + c] = o;
    if (c == 0) { part_ml[row * 2] = M; part_ml[row * 2 + 1] = L; }
  }
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

__global__ __launch_bounds__(256) void reduce_kernel(int rows, int num_splits,
                                                     const float* __restrict__ part_o,
                                                     const float* __restrict__ part_ml,
                                                     const float* __restrict__ Rv,
                                                     void* __restrict__ out, int out_f32) {
  __shared__ float4 Rs[kD * kRvPitch4];
  __shared__ float4 om[kRedRows][kD / 4];
  const int r0 = blockIdx.x * kRedRows;
  const int t = threadIdx.x;
  if (Rv) {
    float4 v[kD * kD / 4 / 256];  // 16 float4 per thread, loads issued before the stores
#pragma unroll
    for (int k = 0; k < kD * kD / 4 / 256; ++k) v[k] = reinterpret_cast<const float4*>(Rv)[t + 256 * k];
#pragma unroll
    for (int k = 0; k < kD * kD / 4 / 256; ++k) {
      const int i = t + 256 * k;
      Rs[(i >> 5) * kRvPitch4 + (i & 31)] = v[k];
    }
  }
  {  // 8 rows x 32 float4 columns: one (row, float4) per thread
    const int rr = t >> 5, c4 = t & 31, r = r0 + rr;
    float4 o = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    if (r < rows) {
      const float2* ml = reinterpret_cast<const float2*>(part_ml + (size_t)r * num_splits * 2);
      // live slots lead (empty ones only follow the end of a sequence): n_live
      // is one past the last live slot
      float M = -INFINITY;
      int n_live = 0;
#pragma unroll 8
      for (int s = 0; s < num_splits; ++s) {
        const float m = ml[s].x;
        M = fmaxf(M, m);
        n_live = (m != -INFINITY) ? s + 1 : n_live;
      }
      if (M != -INFINITY) {
        const float4* po = reinterpret_cast<const float4*>(part_o + (size_t)r * num_splits * kD) + c4;
        float L = 0.0f;
#pragma unroll 8
        for (int s = 0; s < n_live; ++s) {
          const float2 m = ml[s];
          const float4 x = po[(size_t)s * (kD / 4)];  // loaded unconditionally: no load->branch chain
          const bool live = m.x != -INFINITY;         // an empty split contributes nothing
          const float e = live ? exp2f(m.x - M) : 0.0f;
          L = fmaf(e, live ? m.y : 0.0f, L);
          o.x = fmaf(e, live ? x.x : 0.0f, o.x); o.y = fmaf(e, live ? x.y : 0.0f, o.y);
          o.z = fmaf(e, live ? x.z : 0.0f, o.z); o.w = fmaf(e, live ? x.w : 0.0f, o.w);
        }
        const float il = L > 0.0f ? 1.0f / L : 0.0f;
        o.x *= il; o.y *= il; o.z *= il; o.w *= il;
      }
    }
    om[rr][c4] = o;
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
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = r0 + rg + i;
    if (r >= rows) continue;
    if (out_f32) static_cast<float*>(out)[(size_t)r * kD + j] = acc[i];
    else static_cast<uint16_t*>(out)[(size_t)r * kD + j] = f32_to_bf16_rne(acc[i]);
  }
}

template <int NH>
hipError_t launch_split_nh(const uint8_t* pages, int Hkv, int B, int Hq, const int32_t* bt,
                           int max_pages, const int32_t* seq_lens, int S, const float* qt,
                           float* po, float* pml, hipStream_t st) {
  const int pps = (max_pages + S - 1) / S;
  dim3 grid(S, Hkv, B);
  const size_t smem = sizeof(SplitSmem<NH>);
  hipLaunchKernelGGL(split_kernel<NH>, grid, dim3(256), smem, st, pages, Hkv, Hq, bt, max_pages,
                     seq_lens, S, pps, qt, po, pml);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_decode_split(const uint8_t* pages, int Hkv, int B, int Hq,
                               const int32_t* block_table, int max_pages,
                               const int32_t* seq_lens, int num_splits, const float* qt,
                               float* part_o, float* part_ml, hipStream_t st) {
  static const bool use_v0 = [] {
    const char* e = getenv("OSCAR_SPLIT_KERNEL");
    return e && e[0] == 'v' && e[1] == '0';
  }();
  if (!use_v0)
    return launch_decode_split_mfma(pages, Hkv, B, Hq, block_table, max_pages, seq_lens,
                                    num_splits, 16 * device_cus(), qt, part_o, part_ml, st);
  const int g = Hq / Hkv;
  if (g <= 4)
    return launch_split_nh<4>(pages, Hkv, B, Hq, block_table, max_pages, seq_lens, num_splits,
                              qt, part_o, part_ml, st);
  if (g <= 8)
    return launch_split_nh<8>(pages, Hkv, B, Hq, block_table, max_pages, seq_lens, num_splits,
                              qt, part_o, part_ml, st);
  if (g <= 12)
    return launch_split_nh<12>(pages, Hkv, B, Hq, block_table, max_pages, seq_lens, num_splits,
                               qt, part_o, part_ml, st);
  return launch_split_nh<16>(pages, Hkv, B, Hq, block_table, max_pages, seq_lens, num_splits, qt,
                             part_o, part_ml, st);
}

hipError_t launch_decode_reduce(int B, int Hq, int num_splits, const float* part_o,
                                const float* part_ml, const float* Rv, void* out, int out_f32,
                                hipStream_t st) {
  const int rows = B * Hq;
  hipLaunchKernelGGL(reduce_kernel, dim3((rows + kRedRows - 1) / kRedRows), dim3(256), 0, st,
                     rows, num_splits, part_o, part_ml, Rv, out, out_f32);
  return hipGetLastError();
}

}  // namespace oscar
