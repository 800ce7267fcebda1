// Split kernel of INT2 decode attention on the matrix cores (gfx950
// v_mfma_i32_16x16x64_i8).  One wave per (split, kv-head, sequence, chunk of 4
// query heads); the wave walks its pages (64 tokens each) and keeps the
// online-softmax state of its 4 heads in registers.  Waves of the same (split,
// kv-head, sequence) and different chunks get workgroup ids that are equal
// modulo 8, so under round-robin dispatch over the 8 XCDs they share one XCD's
// L2 for the page data they both read.
//
// Arithmetic (Sec. 2: K^ = Q(K R) R^T; Alg. 1 DecodeStep), per 32-channel group g
// with Q(x~)_c = s_g (code_c - z_g):
//   score(t, h) = sum_g s_g ( sum_{c in g} q~_hc code_tc - z_g sum_{c in g} q~_hc )
//   o~(h, c)    = sum_t w(t,h,g(c)) code_tc - sum_t w(t,h,g(c)) z_tg,  w = p s_v
// The integer parts are int8 matrix products:
//   * q~ of a head is scaled to a 24-bit integer (q_int = rne(q~ * Q / max|q~|),
//     Q = 8355000) and split into three signed int8 digits,
//     q_int = 65536 d2 + 256 d1 + d0; the codes are int8 0..3.  Per 16-token tile
//     the products codes x d_j go to separate accumulators, combined as
//     ((a_2 << 8) + a_1) << 8 + a_0, exact in int32 (|.| <= 32 * 3 * Q < 2^31).
//   * w of a head on one page is scaled to [0, Q] (scale p_max * max s_v of the
//     page) and split the same way; the V codes are the other operand
//     (|.| <= 64 * 3 * Q < 2^31).
// The products are exact, so the approximations are the 24-bit quantization of
// q~ and of w (relative 2^-24 of the head's largest value) and fp32
// accumulation.  (With 16-bit scaling the error reached 1.4e-3 on outputs of
// magnitude ~30; 24 bits keeps it near 1e-5.)
//
// Lane roles (l = lane, lo = l & 15, hi = l >> 4), MFMA 16x16x64 layout: A row =
// lo, B column = lo, k-slots (hi, element), D (row 4*hi + i, column lo):
//   score tile u (u = 0..3): MFMA row r <-> token 16*(r>>2) + 4u + (r&3);
//     A operand lane l = K codes of token 16*(lo>>2) + 4u + (lo&3), dwords hi
//     (instruction X=0, groups 0/1) and 4+hi (X=1, groups 2/3), expanded as
//     M_j = (x >> 2j) & 0x03030303 (element 4j+b <-> channel 16w + 4b + j);
//     B column lo = (head lo>>2, group lo&3), zero outside that group;
//     D lane l holds (head lo>>2, group lo&3) for tokens 16*hi + 4u + i.
//   after a sum over the 4 group lanes, lane l holds the scores of head lo>>2
//   for its 16 tokens 16*hi + (0..15): exactly the k-slots of the P.V A operand
//   row lo = (head, group) -- no data movement between softmax and P.V.
//   P.V tile (set S, f): B column lo = channel 4*(16S + lo) + f, V codes of quad
//     16S + lo, tokens 16*hi + (0..15) (quad-major V layout: one 16-byte load);
//     D lane l, register 2S + (lo>>3) = (head hi, group of the column).
#include <hip/hip_fp16.h>

#include "internal.h"

namespace oscar {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));

constexpr float kQMax = 8355000.0f;       // keeps the top digit of a 3-digit split in int8
constexpr float kMagic = 8388608.0f;       // 2^23: x + 2^23 (0 <= x < 2^23) has x in its mantissa
constexpr int kNDig = 3;                   // int8 digits per scaled value (most significant first)

__device__ inline v4i mfma(v4i a, v4i b, v4i c) {
  return __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, c, 0, 0, 0);
}

__device__ inline v4i expand2(uint32_t x) {  // four int8-dwords of 2-bit fields
  v4i r;
  r.x = (int)(x & 0x03030303u);
  r.y = (int)((x >> 2) & 0x03030303u);
  r.z = (int)((x >> 4) & 0x03030303u);
  r.w = (int)((x >> 6) & 0x03030303u);
  return r;
}

// raw v_exp_f32 (results below 2^-126 flush to 0: negligible softmax weights)
__device__ inline float ex2(float x) { return __builtin_amdgcn_exp2f(x); }

// v_fma_mix_f32 with one binary16 operand taken from the low / high half of a
// packed (scale, zero) word: no separate conversion instructions.
__device__ inline float mix_lo(uint32_t h, float b, float c) {  // lo(h) * b + c
  float r;
  asm("v_fma_mix_f32 %0, %1, %2, %3 op_sel:[0,0,0] op_sel_hi:[1,0,0]" : "=v"(r) : "v"(h), "v"(b), "v"(c));
  return r;
}
__device__ inline float mix_hi(uint32_t h, float b, float c) {  // hi(h) * b + c
  float r;
  asm("v_fma_mix_f32 %0, %1, %2, %3 op_sel:[1,0,0] op_sel_hi:[1,0,0]" : "=v"(r) : "v"(h), "v"(b), "v"(c));
  return r;
}
__device__ inline float mix_nhi(uint32_t h, float b, float c) {  // -hi(h) * b + c
  float r;
  asm("v_fma_mix_f32 %0, -%1, %2, %3 op_sel:[1,0,0] op_sel_hi:[1,0,0]" : "=v"(r) : "v"(h), "v"(b), "v"(c));
  return r;
}

typedef unsigned short us2 __attribute__((ext_vector_type(2)));
__device__ inline uint32_t max_u16x2(uint32_t a, uint32_t b) {
  const us2 r = __builtin_elementwise_max(__builtin_bit_cast(us2, a), __builtin_bit_cast(us2, b));
  return __builtin_bit_cast(uint32_t, r);
}

__device__ inline float h_lo(uint32_t w) { return __half2float(__ushort_as_half((uint16_t)(w & 0xffffu))); }
__device__ inline float h_hi(uint32_t w) { return __half2float(__ushort_as_half((uint16_t)(w >> 16))); }
__device__ inline uint32_t comp(uint4 v, int i) { return i == 0 ? v.x : i == 1 ? v.y : i == 2 ? v.z : v.w; }

// sum over the 4 lanes of a quad (xor 1, xor 2) with DPP
__device__ inline float quad_sum(float x) {
  int v = __float_as_int(x);
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, v, 0xB1, 0xF, 0xF, false));  // [1,0,3,2]
  v = __float_as_int(x);
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, v, 0x4E, 0xF, 0xF, false));  // [2,3,0,1]
  return x;
}
__device__ inline float quad_max(float x) {
  int v = __float_as_int(x);
  x = fmaxf(x, __int_as_float(__builtin_amdgcn_update_dpp(0, v, 0xB1, 0xF, 0xF, false)));
  v = __float_as_int(x);
  x = fmaxf(x, __int_as_float(__builtin_amdgcn_update_dpp(0, v, 0x4E, 0xF, 0xF, false)));
  return x;
}
// Reductions over lanes l, l^16, l^32, l^48 with the gfx950 row-swap permutes
// (VALU only, no LDS round trip): swapping a value with itself across the wave
// halves / odd-even rows leaves x[l] and x[l^32] (then x[l^16]) in the two outputs.
__device__ inline float rows_max(float x) {
  uint32_t u = __float_as_uint(x);
  auto a = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  x = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  u = __float_as_uint(x);
  auto b = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ inline float rows_sum(float x) {
  uint32_t u = __float_as_uint(x);
  auto a = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  x = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  u = __float_as_uint(x);
  auto b = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}
// Pack byte `sel` (0..3) of four words into one dword (bytes in order a, b, c, d).
__device__ inline uint32_t pack4(uint32_t a, uint32_t b, uint32_t c, uint32_t d, uint32_t sel) {
  const uint32_t lo2 = 0x0c0c0400u + sel * 0x00000101u;  // [x.sel, y.sel, 0, 0]
  const uint32_t ab = __builtin_amdgcn_perm(b, a, lo2);
  const uint32_t cd = __builtin_amdgcn_perm(d, c, lo2);
  return __builtin_amdgcn_perm(cd, ab, 0x05040100u);
}

// ((a << 8) + b) << 8 + c for signed digit sums, in unsigned arithmetic (the
// intermediate values may be negative; the result fits in int32).
__device__ inline int combine3(int a, int b, int c) {
  return (int)((((uint32_t)a << 8) + (uint32_t)b) * 256u + (uint32_t)c);
}

struct PageBuf {
  uint32_t kx0[4], kx1[4];  // K code dwords for the score A operands, per tile
  uint4 ksz[4];             // K (s,z) of tokens 16*hi + 4u + (0..3), group lo&3
  uint4 vq[2];              // V codes, quads lo and 16+lo, tokens 16*hi + (0..15)
  uint4 vsz[4];             // V (s,z), same tokens and group as ksz
};

__device__ inline void load_page(PageBuf& pb, const uint8_t* __restrict__ blk, int lo, int hi) {
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int tok = 16 * (lo >> 2) + 4 * u + (lo & 3);
    pb.kx0[u] = *reinterpret_cast<const uint32_t*>(blk + kOffKCodes + tok * 32 + 4 * hi);
    pb.kx1[u] = *reinterpret_cast<const uint32_t*>(blk + kOffKCodes + tok * 32 + 16 + 4 * hi);
  }
  const int G = lo & 3;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    pb.ksz[u] = *reinterpret_cast<const uint4*>(blk + kOffKSz + (G * kP + 16 * hi + 4 * u) * 4);
    pb.vsz[u] = *reinterpret_cast<const uint4*>(blk + kOffVSz + (G * kP + 16 * hi + 4 * u) * 4);
  }
  pb.vq[0] = *reinterpret_cast<const uint4*>(blk + kOffVCodes + lo * kP + 16 * hi);
  pb.vq[1] = *reinterpret_cast<const uint4*>(blk + kOffVCodes + (16 + lo) * kP + 16 * hi);
}

struct WaveState {
  v4i bq[2][kNDig];     // query operands [instruction X][digit, most significant first]
  float sq;             // q scale of head lo>>2
  float qs;             // sum of q_int over group lo&3 of head lo>>2
  float m;              // running max (log2 units), head lo>>2
  float lsum;           // partial sum of p over this lane's tokens, head lo>>2
  float zacc;           // partial sum of w * z_v, (head lo>>2, group lo&3)
  float of[8];          // unnormalized o~ of head hi at this lane's 8 channels
};

// FULL: all 64 token slots of the page are in the sequence (every page but
// possibly the sequence's last); otherwise slots >= ntok are masked.
template <bool FULL>
__device__ inline void compute_page(WaveState& st, const PageBuf& pb, int ntok, int lo, int hi) {
  // ---- scores ----
  // One accumulator per digit of q_int (independent MFMAs), combined as
  // (a_2 << 16) + (a_1 << 8) + a_0 for the most to least significant digit.
  float S[4][4];
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const v4i a0 = expand2(pb.kx0[u]);
    const v4i a1 = expand2(pb.kx1[u]);
    v4i d[kNDig];
#pragma unroll
    for (int dg = 0; dg < kNDig; ++dg) {
      const v4i z4 = {0, 0, 0, 0};
      d[dg] = mfma(a1, st.bq[1][dg], mfma(a0, st.bq[0][dg], z4));
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int t = combine3(d[0][i], d[1][i], d[2][i]);
      const uint32_t sz = comp(pb.ksz[u], i);
      // s * (acc - z * sum q_int) with s, z read from the packed binary16 pair
      const float part = mix_lo(sz, mix_nhi(sz, st.qs, (float)t), 0.0f);
      S[u][i] = quad_sum(part);
    }
  }
  // ---- online softmax (head lo>>2, tokens 16*hi + 4u + i) ----
  const int tbase = 16 * hi;
  auto valid = [&](int u, int i) { return FULL || tbase + 4 * u + i < ntok; };
  float mx = -INFINITY;
#pragma unroll
  for (int u = 0; u < 4; ++u)
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (valid(u, i)) mx = fmaxf(mx, S[u][i]);
  mx = rows_max(mx) * st.sq;  // sq > 0
  const float mn = fmaxf(st.m, mx);
  const float alpha = ex2(st.m - mn);  // m = -inf on the first page -> 0
  const float pmax = ex2(mx - mn);
  float ls = 0.0f;
#pragma unroll
  for (int u = 0; u < 4; ++u)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float p = valid(u, i) ? ex2(fmaf(st.sq, S[u][i], -mn)) : 0.0f;
      S[u][i] = p;
      ls += p;
    }
  st.lsum = fmaf(st.lsum, alpha, ls);
  st.m = mn;
  // ---- P.V weights w = p * s_v, quantized per head to three int8 digits ----
  // largest V scale of the page: scales are positive binary16, so their bit
  // patterns order like their values (packed u16 max; the high halves are ignored)
  uint32_t smax = 0;
#pragma unroll
  for (int u = 0; u < 4; ++u)
#pragma unroll
    for (int i = 0; i < 4; ++i)
      smax = max_u16x2(smax, valid(u, i) ? comp(pb.vsz[u], i) : 0u);
  const float svmax = rows_max(quad_max(h_lo(smax)));  // whole page, all groups
  const float sig = pmax * svmax;  // >= every w of this head on this page
  const float inv = sig > 0.0f ? kQMax / sig : 0.0f;
  const float wscale = sig * (1.0f / kQMax);
  float zp = 0.0f;
  uint32_t wd[kNDig][4];
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    uint32_t b0[4], b1[4], b2[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint32_t sz = valid(u, i) ? comp(pb.vsz[u], i) : 0u;  // (0, 0): w = 0, z = 0
      const float w = mix_lo(sz, S[u][i], 0.0f);
      // mantissa of f = rne(w * inv) = k in [0, Q]; signed digits of k:
      // d0 = byte 0 of k, d1 = byte 1 of k + 128, d2 = byte 2 of k + 32896
      const float f = fmaf(w, inv, kMagic);
      b0[i] = __float_as_uint(f);
      b1[i] = b0[i] + 128u;
      b2[i] = b0[i] + 32896u;
      zp = mix_hi(sz, w, zp);  // unquantized w: differs from the quantized by <= 2^-24 sig
    }
    wd[0][u] = pack4(b2[0], b2[1], b2[2], b2[3], 2);
    wd[1][u] = pack4(b1[0], b1[1], b1[2], b1[3], 1);
    wd[2][u] = pack4(b0[0], b0[1], b0[2], b0[3], 0);
  }
  v4i aw[kNDig];
#pragma unroll
  for (int dg = 0; dg < kNDig; ++dg)
    aw[dg] = v4i{(int)wd[dg][0], (int)wd[dg][1], (int)wd[dg][2], (int)wd[dg][3]};
  st.zacc = fmaf(st.zacc, alpha, zp);
  // ---- P.V on the matrix cores ----
  // per-head factors of head hi for the accumulators of this lane
  const float ascale = __shfl(alpha, 4 * hi, 64);
  const float awsc = __shfl(wscale, 4 * hi, 64);
  const bool upper = (lo >> 3) != 0;
#pragma unroll
  for (int S_ = 0; S_ < 2; ++S_) {
    const uint4 d = pb.vq[S_];
#pragma unroll
    for (int f = 0; f < 4; ++f) {
      const uint32_t msk = 0x03030303u;
      const v4i bv = {(int)((d.x >> (2 * f)) & msk), (int)((d.y >> (2 * f)) & msk),
                      (int)((d.z >> (2 * f)) & msk), (int)((d.w >> (2 * f)) & msk)};
      int e[kNDig];
#pragma unroll
      for (int dg = 0; dg < kNDig; ++dg) {
        const v4i z4 = {0, 0, 0, 0};
        const v4i acc = mfma(aw[dg], bv, z4);
        e[dg] = upper ? acc[2 * S_ + 1] : acc[2 * S_];  // row (head hi, group of column)
      }
      const int useful = combine3(e[0], e[1], e[2]);
      float& o = st.of[S_ * 4 + f];
      o = fmaf((float)useful, awsc, o * ascale);
    }
  }
}

// Grid: 1-D, ceil(S*Hkv*B / 8) * 8 * nch workgroups of one wave.  Workgroup id
// -> (xcd = id % 8, slot = id / 8); chunk = slot % nch; item = (slot / nch) * 8
// + xcd; item -> (split, kv-head, sequence).  Items beyond S*Hkv*B exit.
__global__ __launch_bounds__(64) void split_mfma_kernel(
    const uint8_t* __restrict__ pages, int Hkv, int Hq, const int32_t* __restrict__ block_table,
    int max_pages, const int32_t* __restrict__ seq_lens, int num_splits, int pages_per_split,
    int B, const float* __restrict__ qt, float* __restrict__ part_o,
    float* __restrict__ part_ml) {
  const int g = Hq / Hkv;
  const int nch = (g + 3) >> 2;
  const int xcd = blockIdx.x & 7;
  const int slot = blockIdx.x >> 3;
  const int chunk = slot % nch;
  const int64_t item = (int64_t)(slot / nch) * 8 + xcd;
  if (item >= (int64_t)num_splits * Hkv * B) return;
  const int s = (int)(item % num_splits);
  const int kvh = (int)((item / num_splits) % Hkv);
  const int b = (int)(item / ((int64_t)num_splits * Hkv));
  const int l = threadIdx.x, lo = l & 15, hi = l >> 4;
  const int hq = lo >> 2, G = lo & 3;
  const int len = seq_lens[b];
  const int npg = (len + kP - 1) / kP;
  const int p0 = s * pages_per_split;
  const int p1 = min(npg, p0 + pages_per_split);

  WaveState st;
  // ---- query operands: q_int = rne(q~ * Q / max|q~|), three int8 digits ----
  // Lane (head hq, group G, k-group hi) owns channels 32G + 16(hi&1) + 0..15 when
  // (hi>>1) == (G&1), for instruction X = G>>1; it is zero otherwise.
  {
    const bool owns = (hi >> 1) == (G & 1);
    const int cbase = 32 * G + 16 * (hi & 1);
    const int hloc = 4 * chunk + hq;
    float qv[16];
    float amax = 0.0f;
#pragma unroll
    for (int e = 0; e < 16; ++e) qv[e] = 0.0f;
    if (owns && hloc < g) {
      const float4* src =
          reinterpret_cast<const float4*>(qt + ((size_t)b * Hq + kvh * g + hloc) * kD + cbase);
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const float4 x = src[v];
        qv[4 * v] = x.x; qv[4 * v + 1] = x.y; qv[4 * v + 2] = x.z; qv[4 * v + 3] = x.w;
      }
#pragma unroll
      for (int e = 0; e < 16; ++e) amax = fmaxf(amax, fabsf(qv[e]));
    }
    amax = rows_max(quad_max(amax));  // all 128 channels of the head
    const float inv = amax > 0.0f ? kQMax / amax : 0.0f;
    st.sq = amax > 0.0f ? amax * (1.0f / kQMax) : 1.0f;
    int qi[16];
    int qsum = 0;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      qi[e] = (int)rintf(qv[e] * inv);
      qsum += qi[e];
    }
    // element 4j + b of the operand <-> channel cbase + 4b + j;
    // q = 65536 d2 + 256 d1 + d0 with d0 = q - 256 c1, c1 = (q + 128) >> 8, etc.
    uint32_t dw[kNDig][4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      uint32_t w2 = 0, w1 = 0, w0 = 0;
#pragma unroll
      for (int bb = 0; bb < 4; ++bb) {
        const int v = qi[4 * bb + j];
        const int c1 = (v + 128) >> 8;
        const int d0 = v - 256 * c1;
        const int d2 = (c1 + 128) >> 8;
        const int d1 = c1 - 256 * d2;
        w2 |= ((uint32_t)d2 & 0xffu) << (8 * bb);
        w1 |= ((uint32_t)d1 & 0xffu) << (8 * bb);
        w0 |= ((uint32_t)d0 & 0xffu) << (8 * bb);
      }
      dw[0][j] = w2;
      dw[1][j] = w1;
      dw[2][j] = w0;
    }
    const v4i zero = {0, 0, 0, 0};
    const bool x1 = (G >> 1) != 0;
#pragma unroll
    for (int dg = 0; dg < kNDig; ++dg) {
      const v4i v = {(int)dw[dg][0], (int)dw[dg][1], (int)dw[dg][2], (int)dw[dg][3]};
      st.bq[0][dg] = x1 ? zero : v;
      st.bq[1][dg] = x1 ? v : zero;
    }
    // sum over the group's 32 channels (two owning lanes), exact in int
    qsum += __shfl_xor(qsum, 16, 64);
    qsum += __shfl_xor(qsum, 32, 64);
    st.qs = (float)qsum;
    st.m = -INFINITY;
    st.lsum = 0.0f;
    st.zacc = 0.0f;
#pragma unroll
    for (int k = 0; k < 8; ++k) st.of[k] = 0.0f;
  }

  const int32_t* __restrict__ bt = block_table + (size_t)b * max_pages;
  const uint8_t* __restrict__ base = pages + (size_t)kvh * kBlockBytes;
  const size_t page_stride = (size_t)Hkv * kBlockBytes;
  // pages [p0, pf) are full; page pf (if < p1) is the sequence's partial last page
  const int pf = (p1 == npg && (len & (kP - 1)) != 0) ? p1 - 1 : p1;
  PageBuf pa, pb;
  if (p0 < p1) load_page(pa, base + (size_t)bt[p0] * page_stride, lo, hi);
  int pg = p0;
  for (; pg + 1 < pf; pg += 2) {
    load_page(pb, base + (size_t)bt[pg + 1] * page_stride, lo, hi);
    compute_page<true>(st, pa, kP, lo, hi);
    if (pg + 2 < p1) load_page(pa, base + (size_t)bt[pg + 2] * page_stride, lo, hi);
    compute_page<true>(st, pb, kP, lo, hi);
  }
  if (pg < pf) {  // one full page left; pa holds it
    if (pg + 1 < p1) load_page(pb, base + (size_t)bt[pg + 1] * page_stride, lo, hi);
    compute_page<true>(st, pa, kP, lo, hi);
    ++pg;
    if (pg < p1) compute_page<false>(st, pb, len - pg * kP, lo, hi);
  } else if (pg < p1) {  // only the partial page left; pa holds it
    compute_page<false>(st, pa, len - pg * kP, lo, hi);
  }

  // ---- write the split's partial state ----
  const float ltot = rows_sum(st.lsum);            // head lo>>2
  const float ztot = rows_sum(st.zacc);            // (head lo>>2, group lo&3)
  const int hout = 4 * chunk + hi;                 // accumulator head of this lane
  const float mh = __shfl(st.m, 4 * hi, 64);
  const float lh = __shfl(ltot, 4 * hi, 64);
  float zh2[2];
#pragma unroll
  for (int S_ = 0; S_ < 2; ++S_) zh2[S_] = __shfl(ztot, 4 * hi + 2 * S_ + (lo >> 3), 64);
  if (hout >= g) return;  // padding head (every lane took part in the shuffles above)
  const size_t row = ((size_t)b * Hq + kvh * g + hout) * num_splits + s;
#pragma unroll
  for (int S_ = 0; S_ < 2; ++S_) {
#pragma unroll
    for (int f = 0; f < 4; ++f) {
      const int ch = 4 * (16 * S_ + lo) + f;
      part_o[row * kD + ch] = (mh == -INFINITY) ? 0.0f : st.of[S_ * 4 + f] - zh2[S_];
    }
  }
  if (lo == 0) {
    part_ml[row * 2] = mh;
    part_ml[row * 2 + 1] = lh;
  }
}

}  // namespace

hipError_t launch_decode_split_mfma(const uint8_t* pages, int Hkv, int B, int Hq,
                                    const int32_t* block_table, int max_pages,
                                    const int32_t* seq_lens, int num_splits, const float* qt,
                                    float* part_o, float* part_ml, hipStream_t st) {
  const int g = Hq / Hkv;
  const int nch = (g + 3) / 4;
  const int pps = (max_pages + num_splits - 1) / num_splits;
  const int64_t items = (int64_t)num_splits * Hkv * B;
  const int64_t blocks = (items + 7) / 8 * 8 * nch;
  if (blocks > 0x7fffffffLL) return hipErrorInvalidConfiguration;
  hipLaunchKernelGGL(split_mfma_kernel, dim3((unsigned)blocks), dim3(64), 0, st, pages, Hkv, Hq,
                     block_table, max_pages, seq_lens, num_splits, pps, B, qt, part_o, part_ml);
  return hipGetLastError();
}

}  // namespace oscar
