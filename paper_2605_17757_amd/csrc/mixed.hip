// bf16 tokens of the mixed-precision cache (Sec. 4 "KV Cache Layout"; Alg. 1
// DecodeStep): the attention sink [0, S0) and the recent window [n - W, n) of
// every sequence stay in bf16, in a segment store next to the INT2 pool:
//   [B][Hkv][K, V][S0 + W][d] bf16,
// position p at segment slot p (p < S0) or S0 + (p - S0) mod W (window).  At
// length n the valid slots are exactly [0, nb), nb = lo + (n - hi) with
// lo = min(S0, n), hi = max(lo, n - W): the window only holds tokens once the
// sink is full, and it fills its slots from S0 upward before wrapping.  Softmax
// sums do not depend on the order of the tokens, so the kernel walks the slots.
//
// seg_partial: one block per (sequence, kv-head) with one wave per 64-slot chunk
// (nw = ceil((S0 + W) / 64) waves, at most 8; wave w takes the chunks w, w + nw,
// ...); up to 5 waves a block (S0 + W <= 320) and 8 query heads per kv-head,
// two blocks are resident per CU (<= 128 VGPRs, <= 80 KB LDS), so every wave of
// the launch runs at once.
//   loads  : K with 16-byte loads, 8 lanes per 128-byte half row (loads 0-7 of a
//            lane: channel half 0 of rows 8 i + lane / 8; loads 8-15: half 1),
//            issued with the V dwords of the chunk's first 32 tokens (4 heads;
//            16 for 8 heads); the other V dwords once K is staged;
//   scores : lane = token.  K is staged in LDS one channel half (64 channels) at
//            a time at a pitch of 9 16-byte slots (the row reads of a
//            ds_read_b128 pass hit distinct bank groups).  Each lane accumulates
//            q . k with v_dot2_f32_bf16 on packed bf16 channel pairs (q and k are
//            bf16: the products are exact, the sums fp32), then scales by
//            sm_scale log2 e;
//   softmax: running max and sum per head (wave-uniform, scalar registers);
//   P.V    : lane = channels (2l, 2l + 1), fp32 FMAs, weights read back from LDS.
// The wave states are merged in LDS and written, unnormalized, as the state
// (o, m, l) of slot num_splits of the rows (num_splits + 1 slots a row); the
// reduce adds it after the back-rotation of the INT2 part.
#include <algorithm>

#include "internal.h"

namespace oscar {
namespace {

constexpr int kSegWaves = 8;   // at most; blockDim.x / 64 in a launch
constexpr int kPitch = 9;      // 16-byte slots per staged 64-channel half row (one pad)
// V tokens whose loads go out with the K loads (as many as 128 VGPRs allow)
constexpr int v_early(int nh) { return nh <= 4 ? 32 : nh <= 8 ? 16 : 0; }

typedef uint32_t u4v __attribute__((ext_vector_type(4)));
typedef __bf16 bf2 __attribute__((ext_vector_type(2)));

__device__ inline float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ inline float bf_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// a.lo * b.lo + a.hi * b.hi + c for packed bf16 pairs
__device__ inline float dot2(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf2, a), __builtin_bit_cast(bf2, b), c,
                                        false);
}

// max / sum over the wave: quad swaps and row rotations (DPP) inside rows of 16
// lanes, then the row swaps across 32 and 16 lanes
__device__ inline float wave_max(float x) {
  x = fmaxf(x, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0xB1, 0xF, 0xF, false)));
  x = fmaxf(x, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x4E, 0xF, 0xF, false)));
  x = fmaxf(x, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x124, 0xF, 0xF, false)));
  x = fmaxf(x, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x128, 0xF, 0xF, false)));
  uint32_t u = __float_as_uint(x);
  auto a = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  x = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  u = __float_as_uint(x);
  auto c = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  return fmaxf(__uint_as_float(c[0]), __uint_as_float(c[1]));
}
__device__ inline float wave_sum(float x) {
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0xB1, 0xF, 0xF, false));
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x4E, 0xF, 0xF, false));
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x124, 0xF, 0xF, false));
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x128, 0xF, 0xF, false));
  uint32_t u = __float_as_uint(x);
  auto a = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  x = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  u = __float_as_uint(x);
  auto c = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  return __uint_as_float(c[0]) + __uint_as_float(c[1]);
}

__device__ inline float uniform(float x) {
  return __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(x)));
}

// Raw buffer resource over `bytes` bytes at p (gfx9 descriptor: 32-bit data
// format); offsets at or beyond `bytes` load 0.
__device__ inline __amdgpu_buffer_rsrc_t make_rsrc(const void* p, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, bytes, 0x00020000);
}

// small arrays first: every LDS address stays within reach of one base register
// and the 16-bit instruction offset
template <int NH>
struct SegSmem {
  uint32_t qp[kD / 2][NH];                          // q as packed bf16 channel pairs
  float mm[kSegWaves][NH], ll[kSegWaves][NH];
  union {
    u4v kr[kSegWaves][kP * kPitch];                 // staged half rows; then the chunk's p
    float ao[kSegWaves][NH][kD];                    // wave states at the merge
  };
};

template <int NH>
__global__ __launch_bounds__(512)
__attribute__((amdgpu_waves_per_eu(NH > 8 ? 2 : 4, NH > 8 ? 2 : 4))) void seg_partial_kernel(
    const uint16_t* __restrict__ seg, int Hkv, int S0, int W, int Hq,
    const int32_t* __restrict__ seq_lens, int max_pages, const uint16_t* __restrict__ q,
    float qscale, int num_splits, float* __restrict__ part_o, float* __restrict__ part_ml) {
  __shared__ SegSmem<NH> sm;
  const int b = blockIdx.x / Hkv, kvh = blockIdx.x % Hkv;
  const int g = Hq / Hkv;
  const int nw = blockDim.x >> 6;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), l = threadIdx.x & 63;
  const int len = min(max(seq_lens[b], 0), max_pages * kP);
  const int lo = min(S0, len), hi = max(lo, len - W);
  const int nb = lo + (len - hi);

  for (int i = threadIdx.x; i < kD / 2 * NH; i += blockDim.x) {
    const int cp = i / NH, h = i % NH;
    sm.qp[cp][h] = h < g ? reinterpret_cast<const uint32_t*>(q + ((size_t)b * Hq + kvh * g + h) * kD)[cp] : 0u;
  }
  __syncthreads();

  // K and V rows of the block as buffer resources of exactly nb rows: loads past
  // the valid slots return 0 without touching memory
  const size_t rows = (size_t)(S0 + W) * kD;
  const uint16_t* Kb = seg + ((size_t)b * Hkv + kvh) * 2 * rows;
  const __amdgpu_buffer_rsrc_t krs = make_rsrc(Kb, nb * kD * 2);
  const __amdgpu_buffer_rsrc_t vrs = make_rsrc(Kb + rows, nb * kD * 2);
  u4v* kr = sm.kr[w];
  float* pw = reinterpret_cast<float*>(kr);  // [token][head], after the scores
  float m[NH], ls[NH], a0[NH], a1[NH];
#pragma unroll
  for (int h = 0; h < NH; ++h) { m[h] = -INFINITY; ls[h] = 0.0f; a0[h] = a1[h] = 0.0f; }

  for (int c0 = kP * w; c0 < nb; c0 += kP * nw) {
    const int ntok = min(kP, nb - c0);
    u4v kv[16];
    uint32_t vv[kP];
    const int kofs = (c0 + (l >> 3)) * (kD * 2) + 16 * (l & 7);
#pragma unroll
    for (int i = 0; i < 16; ++i)
      kv[i] = __builtin_amdgcn_raw_buffer_load_b128(krs, kofs, (8 * (i & 7)) * kD * 2 + 128 * (i >> 3), 0);
    const int vofs = c0 * (kD * 2) + 4 * l;
#pragma unroll
    for (int t = 0; t < v_early(NH); ++t) vv[t] = __builtin_amdgcn_raw_buffer_load_b32(vrs, vofs, t * kD * 2, 0);
    float sc[NH];
#pragma unroll
    for (int h = 0; h < NH; ++h) sc[h] = 0.0f;
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      __builtin_amdgcn_wave_barrier();
      lane_exchange();
      {  // half rows of this channel half: row 8 i + l / 8, piece l % 8
        u4v* dst = kr + kPitch * (l >> 3) + (l & 7);
#pragma unroll
        for (int i = 0; i < 8; ++i) dst[8 * kPitch * i] = kv[8 * half + i];
      }
      __builtin_amdgcn_wave_barrier();
      lane_exchange();
      if (half == 1) {  // the K registers are free: the remaining V dwords
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int t = v_early(NH); t < kP; ++t) vv[t] = __builtin_amdgcn_raw_buffer_load_b32(vrs, vofs, t * kD * 2, 0);
      }
#pragma unroll 1
      for (int c8 = 0; c8 < 8; ++c8) {  // channel pairs 32 half + 4 c8 + (0..3)
        const u4v u = kr[kPitch * l + c8];
        const uint32_t wd[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int cp = 32 * half + 4 * c8 + e;
#pragma unroll
          for (int h = 0; h < NH; ++h) sc[h] = dot2(sm.qp[cp][h], wd[e], sc[h]);
        }
      }
    }
    __builtin_amdgcn_wave_barrier();
    lane_exchange();
    float alpha[NH];
#pragma unroll
    for (int h = 0; h < NH; ++h) {
      const float sv = l < ntok ? sc[h] * qscale : -INFINITY;
      // the running max and sum are wave-uniform: kept in scalar registers
      const float mn = uniform(fmaxf(m[h], wave_max(sv)));  // finite: the chunk has a token
      alpha[h] = exp2f(m[h] - mn);
      const float p = l < ntok ? exp2f(sv - mn) : 0.0f;
      ls[h] = uniform(fmaf(ls[h], alpha[h], wave_sum(p)));
      m[h] = mn;
      pw[l * NH + h] = p;  // over the staged rows: a wave's LDS accesses run in order
    }
    __builtin_amdgcn_wave_barrier();
    lane_exchange();
#pragma unroll
    for (int h = 0; h < NH; ++h) { a0[h] *= alpha[h]; a1[h] *= alpha[h]; }
#pragma unroll
    for (int t = 0; t < kP; ++t) {  // p = 0 for t >= ntok
      const float v0 = bf_lo(vv[t]), v1 = bf_hi(vv[t]);
#pragma unroll
      for (int h = 0; h < NH; ++h) {
        const float p = pw[t * NH + h];
        a0[h] = fmaf(p, v0, a0[h]);
        a1[h] = fmaf(p, v1, a1[h]);
      }
    }
    __builtin_amdgcn_wave_barrier();
    lane_exchange();
  }

  __syncthreads();  // the staging area becomes the merge area
  if (l == 0) {
#pragma unroll
    for (int h = 0; h < NH; ++h) { sm.mm[w][h] = m[h]; sm.ll[w][h] = ls[h]; }
  }
#pragma unroll
  for (int h = 0; h < NH; ++h) {
    sm.ao[w][h][2 * l] = a0[h];
    sm.ao[w][h][2 * l + 1] = a1[h];
  }
  __syncthreads();
  const int stride = num_splits + 1;
  for (int i = threadIdx.x; i < g * kD; i += blockDim.x) {
    const int h = i / kD, c = i % kD;
    float M = -INFINITY;
    for (int ww = 0; ww < nw; ++ww) M = fmaxf(M, sm.mm[ww][h]);
    float o = 0.0f, L = 0.0f;
    if (M != -INFINITY) {
      for (int ww = 0; ww < nw; ++ww) {
        const float e = sm.mm[ww][h] == -INFINITY ? 0.0f : exp2f(sm.mm[ww][h] - M);
        o = fmaf(e, sm.ao[ww][h][c], o);
        L = fmaf(e, sm.ll[ww][h], L);
      }
    }
    const size_t row = ((size_t)b * Hq + kvh * g + h) * stride + num_splits;
    part_o[row * kD + c] = o;
    if (c == 0) {
      part_ml[row * 2] = M;
      part_ml[row * 2 + 1] = L;
    }
  }
}

template <int NH>
hipError_t launch_seg_nh(const uint16_t* seg, int Hkv, int S0, int W, int B, int Hq,
                         const int32_t* seq_lens, int max_pages, const uint16_t* q, float qscale,
                         int num_splits, float* part_o, float* part_ml, hipStream_t st) {
  const int nw = std::min(kSegWaves, std::max(1, (S0 + W + kP - 1) / kP));
  hipLaunchKernelGGL(seg_partial_kernel<NH>, dim3((unsigned)(B * Hkv)), dim3(64 * nw), 0, st, seg,
                     Hkv, S0, W, Hq, seq_lens, max_pages, q, qscale, num_splits, part_o, part_ml);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_seg_partial(const uint16_t* seg, int Hkv, int S0, int W, int B, int Hq,
                              const int32_t* seq_lens, int max_pages, const uint16_t* q,
                              float qscale, int num_splits, float* part_o, float* part_ml,
                              hipStream_t st) {
  const int g = Hq / Hkv;
  if (g <= 4)
    return launch_seg_nh<4>(seg, Hkv, S0, W, B, Hq, seq_lens, max_pages, q, qscale, num_splits,
                            part_o, part_ml, st);
  if (g <= 8)
    return launch_seg_nh<8>(seg, Hkv, S0, W, B, Hq, seq_lens, max_pages, q, qscale, num_splits,
                            part_o, part_ml, st);
  return launch_seg_nh<16>(seg, Hkv, S0, W, B, Hq, seq_lens, max_pages, q, qscale, num_splits,
                           part_o, part_ml, st);
}

}  // namespace oscar
