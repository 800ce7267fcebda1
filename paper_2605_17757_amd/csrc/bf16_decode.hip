// bf16 paged-decode baseline: the same paging and split-K / log-sum-exp scheme as
// the INT2 path, over an uncompressed bf16 cache (no rotation, no quantization).
// It exists to compare the INT2 path against plain bf16 decode on the same GPU.
// The query is scaled by sm_scale*log2 e by the prepare kernel with R = I.
#include "internal.h"

namespace oscar {
namespace {

constexpr int kWaves = 4;
constexpr int kRowElems = kD;              // bf16 elements per token row
constexpr int kBlockElems = 2 * kP * kD;   // bf16 elements per page-head block

__device__ inline float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ inline float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

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

__global__ __launch_bounds__(256) void bf16_append_kernel(uint16_t* __restrict__ pages, int Hkv,
                                                          const uint16_t* __restrict__ k,
                                                          const uint16_t* __restrict__ v,
                                                          const int64_t* __restrict__ slots,
                                                          int n_rows) {
  // one wave per (token, head) row; lane copies 4 bytes of K and of V
  const int row = blockIdx.x * kWaves + (threadIdx.x >> 6);
  const int l = threadIdx.x & 63;
  if (row >= n_rows) return;
  const int tok = row / Hkv, h = row - tok * Hkv;
  const int64_t slot = slots[tok];
  const int64_t page = slot / kP;
  const int t = (int)(slot - page * kP);
  uint16_t* blk = pages + ((size_t)page * Hkv + h) * kBlockElems;
  reinterpret_cast<uint32_t*>(blk + (size_t)t * kD)[l] =
      reinterpret_cast<const uint32_t*>(k + (size_t)row * kD)[l];
  reinterpret_cast<uint32_t*>(blk + (size_t)(kP + t) * kD)[l] =
      reinterpret_cast<const uint32_t*>(v + (size_t)row * kD)[l];
}

template <int NH>
struct Bf16Smem {
  float qs[kD][NH];
  float pw[kWaves][kD][NH];  // p per token (first kP rows); [kWaves][NH][kD] at merge
  float mm[kWaves][NH], ll[kWaves][NH];
};

template <int NH>
__global__ __launch_bounds__(256) void bf16_split_kernel(
    const uint16_t* __restrict__ pages, int Hkv, int Hq, const int32_t* __restrict__ block_table,
    int max_pages, const int32_t* __restrict__ seq_lens, int num_splits, int pages_per_split,
    const float* __restrict__ qt, float* __restrict__ part_o, float* __restrict__ part_ml) {
  extern __shared__ __align__(16) uint8_t smem_raw[];
  Bf16Smem<NH>& sm = *reinterpret_cast<Bf16Smem<NH>*>(smem_raw);
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

  float m[NH], lsum[NH], acc0[NH], acc1[NH];
#pragma unroll
  for (int h = 0; h < NH; ++h) { m[h] = -INFINITY; lsum[h] = 0.0f; acc0[h] = acc1[h] = 0.0f; }
  const int32_t* __restrict__ bt = block_table + (size_t)b * max_pages;

  for (int pr = p0; pr < p1; pr += kWaves) {
    const int pg = pr + w;
    const bool active = pg < p1;
    const int ntok = active ? min(kP, len - pg * kP) : 0;
    const uint16_t* blk = nullptr;
    if (active) blk = pages + ((size_t)bt[pg] * Hkv + kvh) * kBlockElems;
    const bool valid = l < ntok;

    // phase 1: lane = token, score for every head
    float score[NH];
#pragma unroll
    for (int h = 0; h < NH; ++h) score[h] = 0.0f;
    if (valid) {
      const uint4* kr = reinterpret_cast<const uint4*>(blk + (size_t)l * kRowElems);
#pragma unroll 4
      for (int ch = 0; ch < kD / 8; ++ch) {
        const uint4 u = kr[ch];
        const uint32_t wd[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float k0 = bf16_lo(wd[e]), k1 = bf16_hi(wd[e]);
          const float* q0 = sm.qs[ch * 8 + 2 * e];
          const float* q1 = sm.qs[ch * 8 + 2 * e + 1];
#pragma unroll
          for (int h = 0; h < NH; ++h) score[h] = fmaf(q1[h], k1, fmaf(q0[h], k0, score[h]));
        }
      }
    }
    // phase 2: online softmax
    float alpha[NH];
#pragma unroll
    for (int h = 0; h < NH; ++h) {
      const float sc = valid ? score[h] : -INFINITY;
      const float mx = active ? wave_max(sc) : -INFINITY;
      const float mn = fmaxf(m[h], mx);
      alpha[h] = (mn == -INFINITY) ? 1.0f : exp2f(m[h] - mn);
      const float p = valid ? exp2f(sc - mn) : 0.0f;
      lsum[h] = lsum[h] * alpha[h] + (active ? wave_sum(p) : 0.0f);
      m[h] = mn;
      sm.pw[w][l][h] = p;
    }
    __syncthreads();
    // phase 3: lane = channels (2l, 2l+1)
#pragma unroll
    for (int h = 0; h < NH; ++h) { acc0[h] *= alpha[h]; acc1[h] *= alpha[h]; }
    for (int t = 0; t < ntok; ++t) {
      const uint32_t vv = reinterpret_cast<const uint32_t*>(blk + (size_t)(kP + t) * kRowElems)[l];
      const float v0 = bf16_lo(vv), v1 = bf16_hi(vv);
      const float* pr_ = sm.pw[w][t];
#pragma unroll
      for (int h = 0; h < NH; ++h) {
        acc0[h] = fmaf(pr_[h], v0, acc0[h]);
        acc1[h] = fmaf(pr_[h], v1, acc1[h]);
      }
    }
    __syncthreads();
  }

  // merge the wave states; pw is reused as [kWaves][NH][kD]
  float* ao = &sm.pw[0][0][0];
  if (l == 0) {
#pragma unroll
    for (int h = 0; h < NH; ++h) { sm.mm[w][h] = m[h]; sm.ll[w][h] = lsum[h]; }
  }
#pragma unroll
  for (int h = 0; h < NH; ++h) {
    ao[(w * NH + h) * kD + 2 * l] = acc0[h];
    ao[(w * NH + h) * kD + 2 * l + 1] = acc1[h];
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

template <int NH>
hipError_t launch_bf16_nh(const uint16_t* pages, int Hkv, int B, int Hq, const int32_t* bt,
                          int max_pages, const int32_t* seq_lens, int S, const float* qt,
                          float* po, float* pml, hipStream_t st) {
  const int pps = (max_pages + S - 1) / S;
  const size_t smem = sizeof(Bf16Smem<NH>);
  hipLaunchKernelGGL(bf16_split_kernel<NH>, dim3(S, Hkv, B), dim3(256), smem, st, pages, Hkv, Hq,
                     bt, max_pages, seq_lens, S, pps, qt, po, pml);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_bf16_append(void* pages, int64_t Hkv, const uint16_t* k, const uint16_t* v,
                              const int64_t* slots, int n_tok, hipStream_t st) {
  const int64_t n_rows = (int64_t)n_tok * Hkv;
  hipLaunchKernelGGL(bf16_append_kernel, dim3((unsigned)((n_rows + kWaves - 1) / kWaves)),
                     dim3(256), 0, st, static_cast<uint16_t*>(pages), (int)Hkv, k, v, slots,
                     (int)n_rows);
  return hipGetLastError();
}

hipError_t launch_bf16_split(const uint16_t* pages, int Hkv, int B, int Hq,
                             const int32_t* block_table, int max_pages, const int32_t* seq_lens,
                             int num_splits, const float* qt, float* part_o, float* part_ml,
                             hipStream_t st) {
  const int g = Hq / Hkv;
  if (g <= 4)
    return launch_bf16_nh<4>(pages, Hkv, B, Hq, block_table, max_pages, seq_lens, num_splits, qt,
                             part_o, part_ml, st);
  if (g <= 8)
    return launch_bf16_nh<8>(pages, Hkv, B, Hq, block_table, max_pages, seq_lens, num_splits, qt,
                             part_o, part_ml, st);
  if (g <= 12)
    return launch_bf16_nh<12>(pages, Hkv, B, Hq, block_table, max_pages, seq_lens, num_splits,
                              qt, part_o, part_ml, st);
  return launch_bf16_nh<16>(pages, Hkv, B, Hq, block_table, max_pages, seq_lens, num_splits, qt,
                            part_o, part_ml, st);
}

}  // namespace oscar
