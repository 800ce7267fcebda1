// Split kernel of INT2 decode attention on the matrix cores (gfx950 MFMA).
// Persistent waves: each wave owns one (page range, kv-head), walks the range's
// pages (64 tokens each) and keeps the online-softmax state of the kv-head's
// query heads in registers; a range that crosses sequence boundaries writes one
// partial state per sequence piece (see split_mfma_kernel).  Up to 4 query heads
// per kv-head: int8 products for the scores and P.V, as below.  5 to 16: the scores
// on fp16 products with one or two rows per head, P.V on int8 in chunks of 4 heads
// (compute_page_wide, further down).
//
// Arithmetic (Sec. 2: K^ = Q(K R) R^T; Alg. 1 DecodeStep), per 32-channel group g
// with Q(x~)_c = s_g (code_c - z_g):
//   score(t, h) = sum_g s_g ( sum_{c in g} q~_hc code_tc - z_g sum_{c in g} q~_hc )
//   o~(h, c)    = sum_t w(t,h,g(c)) code_tc - sum_t w(t,h,g(c)) z_tg,  w = p s_v
// The integer parts are int8 matrix products:
//   * q~ of a head is scaled to a 24-bit integer (q_int = rne(q~ * Q / max|q~|),
//     Q = 8355000) and split into three signed int8 digits,
//     q_int = 65536 d_0 + 256 d_1 + d_2; the codes are int8 0..3.  The three
//     digits are three rows of one MFMA, combined as ((a_0 << 8) + a_1) << 8 + a_2,
//     exact in int32 (|.| <= 32 * 3 * Q < 2^31).
//   * w of a (head, group) row on one page is scaled to [0, 2^21] (scale: the
//     page's p_max of the head times the largest V scale of the group) and split
//     the same way; the V codes are the other operand, taken as code or 4 x code
//     (|.| <= 64 * 12 * 2^21 < 2^31).
// The products are exact, so the approximations are the quantization of q~ (24
// bits) and of w (21 bits), relative to the largest value, and fp32 accumulation.
//
// Data path.  Each page-head block (6144 B) is read with six coalesced 16-byte
// loads per lane into registers (issued one page ahead) and stored to a per-wave
// LDS copy, from which every lane reads the operands of its role.  In the LDS
// copy every 8 16-byte chunks of the K-code region are followed by one chunk of
// padding, which spreads the per-token reads of the score operands over the banks.
//
// Lane roles (l = lane, lo = l & 15, hi = l >> 4).  MFMA 16x16 layout: A row = lo,
// B column = lo, k-slots (hi, element), D (row 4*hi + i, column lo).  MFMA rows
// are (head lo>>2, digit lo&3); digit row 3 is padding whose output is never read.
//   scores, token tile u (u = 0..3), group g: 16x16x32; A = digit of q~ of the head
//     on 8 channels of g per k-group; B = K codes of token 4*lo + u on the same
//     channels (element e of k-group hi <-> channel
//     32g + 16(hi>>1) + 4(e&3) + 2(hi&1) + (e>>2)).  D lane l, register i = digit
//     i of head hi for token 4*lo + u: digits combine inside the lane, and the
//     sum over groups too.
//   p (head hi, tokens 4*lo + u) goes through LDS to the weight layout: lane
//     (head lo>>2, group lo&3) computes w for tokens 16*hi + (0..15) and stores
//     its three digit operands to LDS, where the P.V layout reads them back.
//   P.V, tile (G, F) (G = 0..3, F = 0..1): 16x16x64; A = digit of w of (head,
//     group G), k = tokens 16*hi + (0..15); B column lo = channel
//     32G + 4(lo&7) + 2F + (lo>>3) (all 16 columns in group G).  D lane l,
//     register i = digit i of head hi at that channel.
#include <hip/hip_fp16.h>

#include <algorithm>
#include <type_traits>

#include "internal.h"

namespace oscar {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));

constexpr float kQMax = 8355000.0f;        // q~ scale: the 3-digit split keeps the top digit in int8
constexpr float kWMax = 2097152.0f;        // w scale 2^21: 64 * 12 * 2^21 < 2^31 (P.V columns may be x4)
constexpr float kMagic = 8388608.0f;       // 2^23: x + 2^23 (0 <= x < 2^23) has x in its mantissa
constexpr float kDigitBias = 32896.0f;     // 128 + 128 * 256 (offset of the two low digits)
constexpr int kNDig = 3;                   // int8 digits per scaled value (most significant first)
// A head's reference maximum m moves only on a page whose maximum exceeds it by
// more than kSlack (log2 units): p and the running sums are relative to m, at most
// 2^kSlack times their size relative to the true maximum, and they are rescaled on
// those pages only (a wave-uniform branch).
constexpr float kSlack = 10.0f;
// LDS copy of a page-head block, in 16-byte slots.  The placement keeps every LDS
// instruction of the page loop free of bank conflicts on gfx950, whose ds_read_b128
// serves a wave in four passes of 16 lanes (4-lane blocks {0,3,5,6}, {1,2,4,7} of
// each wave half) over 16 bank groups of 16 bytes, and whose ds_write_b128 serves
// 8 consecutive lanes at a time over 8 bank groups.
//   K codes  chunk c < 128        -> slot c + (c >> 3)          (one pad slot per 8)
//   K scales chunk 256 + i        -> slot 144 + i
//   V codes  chunk 128 + c        -> slot 208 + (c ^ 2 * ((c >> 4) & 1))
//   V scales chunk 320 + 16 g + t -> slot 336 + 17 g + t            (pitch 17)
constexpr int kSlotKSz = 144;
constexpr int kSlotVCodes = 208;
constexpr int kSlotVSz = 336;
constexpr int kSlots = kSlotVSz + 4 * 17;
constexpr int kLdsKCodes = 0;
constexpr int kLdsKSz = kSlotKSz * 16;
constexpr int kLdsVCodes = kSlotVCodes * 16;
constexpr int kLdsVSz = kSlotVSz * 16;
// Weight-digit operands of a page, stored over the page's K codes and K scales (no
// longer needed once the scores are done): group G, row (head, digit), k-group k at
// slot kWBase[G] + 13 k + 3 perm_k(head) + digit, where perm_k is the identity for
// even k and (0, 2, 3, 1) for odd k.
__device__ inline int w_base(int G) { return G == 0 ? 0 : G == 1 ? 51 : G == 2 ? 103 : 156; }
// The same as arithmetic, for a lane-varying G (no branches in the page loop).
__device__ inline int w_base_v(int G) { return 51 * G + ((G * (G - 1)) >> 1); }
__device__ inline int w_slot(int head, int k) {
  return 13 * k + 3 * ((k & 1) ? (0x1320 >> (4 * head)) & 0xf : head);
}

__device__ inline v4i mfma64(v4i a, v4i b) {
  const v4i z = {0, 0, 0, 0};
  return __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, z, 0, 0, 0);
}
__device__ inline v4i mfma32(long a, long b) {
  const v4i z = {0, 0, 0, 0};
  return __builtin_amdgcn_mfma_i32_16x16x32_i8(a, b, z, 0, 0, 0);
}
__device__ inline v4i mfma32acc(long a, long b, v4i c) {
  return __builtin_amdgcn_mfma_i32_16x16x32_i8(a, b, c, 0, 0, 0);
}

// raw v_exp_f32 (results below 2^-126 flush to 0: negligible softmax weights)
__device__ inline float ex2(float x) { return __builtin_amdgcn_exp2f(x); }

// v_fma_mix_f32 with one binary16 operand taken from the low / high half of a
// packed (scale, zero) word (no conversion instructions), in inline asm whose
// result overwrites its own addend or multiplicand register.  The compiler places
// no wait states around inline asm: a result written to a free register could land
// in one that an MFMA still in flight reads (its operands are dead to the compiler
// once the MFMA has issued), so every helper writes only a register that holds one
// of its own live inputs, an LDS or VALU value that is never an MFMA operand or
// result.  Plain C gives the same instructions here but converts the scales of a
// whole page at once and spills at 128 VGPRs.
__device__ inline void mix_lo_acc(uint32_t h, float b, float& acc) {  // acc += lo(h) * b
  asm("v_fma_mix_f32 %0, %1, %2, %0 op_sel:[0,0,0] op_sel_hi:[1,0,0]" : "+v"(acc) : "v"(h), "v"(b));
}
__device__ inline void mix_hi_acc(uint32_t h, float b, float& acc) {  // acc += hi(h) * b
  asm("v_fma_mix_f32 %0, %1, %2, %0 op_sel:[1,0,0] op_sel_hi:[1,0,0]" : "+v"(acc) : "v"(h), "v"(b));
}
__device__ inline void mix_nhi_acc(uint32_t h, float b, float& acc) {  // acc -= hi(h) * b
  asm("v_fma_mix_f32 %0, -%1, %2, %0 op_sel:[1,0,0] op_sel_hi:[1,0,0]" : "+v"(acc) : "v"(h), "v"(b));
}
__device__ inline void mix_lo_mul(uint32_t h, float& b) {  // b = lo(h) * b
  asm("v_fma_mix_f32 %0, %1, %0, 0 op_sel:[0,0,0] op_sel_hi:[1,0,0]" : "+v"(b) : "v"(h));
}

// The same for either metadata format: binary16 as above, bfloat16 as the upper
// bits of a binary32 (a shift or a mask) in plain C.
template <bool BF>
__device__ inline void sz_s_acc(uint32_t h, float b, float& acc) {  // acc += s * b
  if (BF) acc = fmaf(__uint_as_float(h << 16), b, acc);
  else mix_lo_acc(h, b, acc);
}
template <bool BF>
__device__ inline void sz_z_acc(uint32_t h, float b, float& acc) {  // acc += z * b
  if (BF) acc = fmaf(__uint_as_float(h & 0xffff0000u), b, acc);
  else mix_hi_acc(h, b, acc);
}
template <bool BF>
__device__ inline void sz_nz_acc(uint32_t h, float b, float& acc) {  // acc -= z * b
  if (BF) acc = fmaf(-__uint_as_float(h & 0xffff0000u), b, acc);
  else mix_nhi_acc(h, b, acc);
}
template <bool BF>
__device__ inline void sz_s_mul(uint32_t h, float& b) {  // b *= s
  if (BF) b *= __uint_as_float(h << 16);
  else mix_lo_mul(h, b);
}

// s * b + c for a binary16 s as one v_fma_mix_f32 in inline asm, for the P.V
// weights of the wide path: plain C converts a scale once for all chunks and then
// needs an FMA per chunk as well.  The compiler places no wait states around inline
// asm, so this is used only where no MFMA can be in flight: after every score MFMA
// result has been read (the weights depend on the softmax), before the P.V MFMAs
// (a later basic block).
template <bool BF>
__device__ inline float sz_s_fma_asm(uint32_t h, float b, float c) {
  if (BF) return fmaf(__uint_as_float(h << 16), b, c);
  float r;
  asm("v_fma_mix_f32 %0, %1, %2, %3 op_sel:[0,0,0] op_sel_hi:[1,0,0]" : "=v"(r) : "v"(h), "v"(b), "v"(c));
  return r;
}

// s * b + c with s read from a packed (scale, zero) word, in plain C (v_fma_mix_f32
// for binary16): for operands that come straight from an MFMA, whose read-after-
// write wait states the compiler inserts only before instructions it knows.
template <bool BF>
__device__ inline float sz_s_fma_c(uint32_t h, float b, float c) {
  return fmaf(BF ? __uint_as_float(h << 16) : __half2float(__ushort_as_half((uint16_t)(h & 0xffffu))), b, c);
}

// unsigned maximum of the low halves of three words (high half of the result unused)
__device__ inline uint32_t max3_lo16(uint32_t a, uint32_t b, uint32_t c) {
  const uint16_t m = max(max((uint16_t)a, (uint16_t)b), (uint16_t)c);
  return m;
}

__device__ inline float h_lo(uint32_t w) { return __half2float(__ushort_as_half((uint16_t)(w & 0xffffu))); }
__device__ inline uint32_t comp(uint4 v, int i) { return i == 0 ? v.x : i == 1 ? v.y : i == 2 ? v.z : v.w; }
__device__ inline float compf(float4 v, int i) { return i == 0 ? v.x : i == 1 ? v.y : i == 2 ? v.z : v.w; }

// Sum over the 16 lanes of a row (quad swaps, then row rotations by 4 and 8).
__device__ inline float row16_sum(float x) {
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0xB1, 0xF, 0xF, false));
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x4E, 0xF, 0xF, false));
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x124, 0xF, 0xF, false));
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x128, 0xF, 0xF, false));
  return x;
}
// Max over the lanes l and l ^ 2 of a quad, and over all four lanes of a quad,
// of non-negative floats (their bit patterns order like their values, so the
// integer maximum needs no NaN quieting); v_max_u32 with DPP operands.  The asm
// DPP helpers start with s_nop 4: the compiler does not see their DPP reads, and
// an EXEC write by a scalar instruction needs 5 wait states before one (a VALU
// result 2); the later s_nops cover the dependent steps.
__device__ inline float quad_pair_max_pos(float a) {
  asm volatile(
      "s_nop 4\n"
      "v_max_u32_dpp %0, %0, %0 quad_perm:[2,3,0,1] row_mask:0xf bank_mask:0xf\n"
      : "+v"(a));
  return a;
}
__device__ inline float quad_max_pos(float a) {
  asm volatile(
      "s_nop 4\n"
      "v_max_u32_dpp %0, %0, %0 quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf\n"
      "s_nop 1\n"
      "v_max_u32_dpp %0, %0, %0 quad_perm:[2,3,0,1] row_mask:0xf bank_mask:0xf\n"
      : "+v"(a));
  return a;
}
__device__ inline float quad_sum(float x) {
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0xB1, 0xF, 0xF, false));
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x4E, 0xF, 0xF, false));
  return x;
}
// Max over the 16 lanes of a row for four values at once: v_max_f32 with DPP
// operands (quad swaps, then row rotations by 4 and 8), the four chains
// interleaved so that every DPP read is 3 instructions after the write it reads
// (2 wait states required).
__device__ inline void row16_max4(float& a, float& b, float& c, float& d) {
  asm volatile(
      "s_nop 4\n"
      "v_max_f32_dpp %0, %0, %0 quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf\n"
      "v_max_f32_dpp %1, %1, %1 quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf\n"
      "v_max_f32_dpp %2, %2, %2 quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf\n"
      "v_max_f32_dpp %3, %3, %3 quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf\n"
      "v_max_f32_dpp %0, %0, %0 quad_perm:[2,3,0,1] row_mask:0xf bank_mask:0xf\n"
      "v_max_f32_dpp %1, %1, %1 quad_perm:[2,3,0,1] row_mask:0xf bank_mask:0xf\n"
      "v_max_f32_dpp %2, %2, %2 quad_perm:[2,3,0,1] row_mask:0xf bank_mask:0xf\n"
      "v_max_f32_dpp %3, %3, %3 quad_perm:[2,3,0,1] row_mask:0xf bank_mask:0xf\n"
      "v_max_f32_dpp %0, %0, %0 row_ror:4 row_mask:0xf bank_mask:0xf\n"
      "v_max_f32_dpp %1, %1, %1 row_ror:4 row_mask:0xf bank_mask:0xf\n"
      "v_max_f32_dpp %2, %2, %2 row_ror:4 row_mask:0xf bank_mask:0xf\n"
      "v_max_f32_dpp %3, %3, %3 row_ror:4 row_mask:0xf bank_mask:0xf\n"
      "v_max_f32_dpp %0, %0, %0 row_ror:8 row_mask:0xf bank_mask:0xf\n"
      "v_max_f32_dpp %1, %1, %1 row_ror:8 row_mask:0xf bank_mask:0xf\n"
      "v_max_f32_dpp %2, %2, %2 row_ror:8 row_mask:0xf bank_mask:0xf\n"
      "v_max_f32_dpp %3, %3, %3 row_ror:8 row_mask:0xf bank_mask:0xf\n"
      : "+v"(a), "+v"(b), "+v"(c), "+v"(d));
}
// The same for three values (three interleaved chains: every read is 2
// instructions after its write).
__device__ inline void row16_max3(float& a, float& b, float& c) {
  asm volatile(
      "s_nop 4\n"
      "v_max_f32_dpp %0, %0, %0 quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf\n"
      "v_max_f32_dpp %1, %1, %1 quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf\n"
      "v_max_f32_dpp %2, %2, %2 quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf\n"
      "v_max_f32_dpp %0, %0, %0 quad_perm:[2,3,0,1] row_mask:0xf bank_mask:0xf\n"
      "v_max_f32_dpp %1, %1, %1 quad_perm:[2,3,0,1] row_mask:0xf bank_mask:0xf\n"
      "v_max_f32_dpp %2, %2, %2 quad_perm:[2,3,0,1] row_mask:0xf bank_mask:0xf\n"
      "v_max_f32_dpp %0, %0, %0 row_ror:4 row_mask:0xf bank_mask:0xf\n"
      "v_max_f32_dpp %1, %1, %1 row_ror:4 row_mask:0xf bank_mask:0xf\n"
      "v_max_f32_dpp %2, %2, %2 row_ror:4 row_mask:0xf bank_mask:0xf\n"
      "v_max_f32_dpp %0, %0, %0 row_ror:8 row_mask:0xf bank_mask:0xf\n"
      "v_max_f32_dpp %1, %1, %1 row_ror:8 row_mask:0xf bank_mask:0xf\n"
      "v_max_f32_dpp %2, %2, %2 row_ror:8 row_mask:0xf bank_mask:0xf\n"
      : "+v"(a), "+v"(b), "+v"(c));
}
// The same for two values (s_nop between the dependent pairs).
__device__ inline void row16_max2(float& a, float& b) {
  asm volatile(
      "s_nop 4\n"
      "v_max_f32_dpp %0, %0, %0 quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf\n"
      "v_max_f32_dpp %1, %1, %1 quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf\n"
      "s_nop 0\n"
      "v_max_f32_dpp %0, %0, %0 quad_perm:[2,3,0,1] row_mask:0xf bank_mask:0xf\n"
      "v_max_f32_dpp %1, %1, %1 quad_perm:[2,3,0,1] row_mask:0xf bank_mask:0xf\n"
      "s_nop 0\n"
      "v_max_f32_dpp %0, %0, %0 row_ror:4 row_mask:0xf bank_mask:0xf\n"
      "v_max_f32_dpp %1, %1, %1 row_ror:4 row_mask:0xf bank_mask:0xf\n"
      "s_nop 0\n"
      "v_max_f32_dpp %0, %0, %0 row_ror:8 row_mask:0xf bank_mask:0xf\n"
      "v_max_f32_dpp %1, %1, %1 row_ror:8 row_mask:0xf bank_mask:0xf\n"
      : "+v"(a), "+v"(b));
}
// The same for one value (s_nop between the dependent steps).
__device__ inline float row16_max1(float a) {
  asm volatile(
      "s_nop 4\n"
      "v_max_f32_dpp %0, %0, %0 quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf\n"
      "s_nop 1\n"
      "v_max_f32_dpp %0, %0, %0 quad_perm:[2,3,0,1] row_mask:0xf bank_mask:0xf\n"
      "s_nop 1\n"
      "v_max_f32_dpp %0, %0, %0 row_ror:4 row_mask:0xf bank_mask:0xf\n"
      "s_nop 1\n"
      "v_max_f32_dpp %0, %0, %0 row_ror:8 row_mask:0xf bank_mask:0xf\n"
      : "+v"(a));
  return a;
}
// Reductions over lanes l, l^16, l^32, l^48 with the gfx950 row-swap permutes:
// swapping a value with itself across the wave halves / odd-even rows leaves
// x[l] and x[l^32] (then x[l^16]) in the two outputs.
__device__ inline float rows_max(float x) {
  uint32_t u = __float_as_uint(x);
  auto a = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  x = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  u = __float_as_uint(x);
  auto b = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
// The same maximum for non-negative floats, on their bit patterns.
__device__ inline float rows_max_pos(float x) {
  uint32_t u = __float_as_uint(x);
  auto a = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  u = max(a[0], a[1]);
  auto b = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  return __uint_as_float(max(b[0], b[1]));
}
__device__ inline float rows_sum(float x) {
  uint32_t u = __float_as_uint(x);
  auto a = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  x = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  u = __float_as_uint(x);
  auto b = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// ((a << 8) + b) << 8 + c for signed digit sums, in unsigned arithmetic (the
// intermediate values may be negative; the result fits in int32).
__device__ inline int combine3(int a, int b, int c) {
  uint32_t t = ((uint32_t)a << 8) + (uint32_t)b;
  asm("" : "+v"(t));  // keeps two shift-adds (no re-association into 2 shifts + add3)
  return (int)((t << 8) + (uint32_t)c);
}

// Per-wave LDS: the page copy and the exchanges between lane roles.  The weight
// digits of chunk 0 go over the page's spent K codes and K scales, those of
// chunks 1..NCH-1 to areas of their own (same slot placement).
constexpr int kWSlots = 208;  // slots of one chunk's weight digits (the K area of the page)
template <int NCH>
struct WaveLds {
  uint4 page[kSlots];                 // page-head block (slot placement above)
  uint4 wdig[NCH - 1][kWSlots];       // weight digits of chunks 1..NCH-1
  float4 p[4][17];                    // softmax weights of the page, [head][token / 4] (pitch 17)
  float2 hs[4];                       // (alpha, p_max) per head
  float ws[NCH][16];                  // P.V scale per (head, group) and chunk; at the end, sum w z
  int qs[16];                         // sum of q_int per (head, 32-channel slice)
  float sq[4];                        // q scale per head
};

typedef uint32_t u4 __attribute__((ext_vector_type(4)));

struct Stage {  // chunks 64 i + lane of the next page, i = 0..5
  u4 v0, v1, v2, v3, v4, v5;
};

// A page-head block has 256 + 32 NG chunks of 16 bytes (NG groups per head): the
// codes, then 16 NG chunks of K (s, z) and 16 NG of V (s, z).  Chunks past the
// block are not loaded.  NT: non-temporal loads (every block is read by exactly
// one wave, so its lines are not kept for reuse; this raised the read rate from
// 5.3 to 5.8 TB/s on the Qwen3-8B-shaped batch).
template <bool NT>
__device__ inline u4 ld16(const u4* p) {
  if (NT) return __builtin_nontemporal_load(p);
  return *p;
}
template <int NG, bool NT>
__device__ inline void stage_load(Stage& s, const uint8_t* __restrict__ blk, int l) {
  const u4* src = reinterpret_cast<const u4*>(blk) + l;
  s.v0 = ld16<NT>(src);
  s.v1 = ld16<NT>(src + 64);
  s.v2 = ld16<NT>(src + 128);
  s.v3 = ld16<NT>(src + 192);
  if (NG >= 2 || l < 32) s.v4 = ld16<NT>(src + 256);
  if (NG == 4) s.v5 = ld16<NT>(src + 320);
}
template <int NG>
__device__ inline void stage_store(uint4* page, const Stage& s, int l) {
  lane_exchange();  // after every lane's reads of the previous page
  u4* dst = reinterpret_cast<u4*>(page);
  const int a = l + (l >> 3);                  // K codes
  const int v = l ^ (((l >> 4) & 1) << 1);     // V codes
  dst[a] = s.v0;
  dst[72 + a] = s.v1;
  dst[kSlotVCodes + v] = s.v2;
  dst[kSlotVCodes + 64 + v] = s.v3;
  if (NG == 4) {
    dst[kSlotKSz + l] = s.v4;
    dst[kSlotVSz + l + (l >> 4)] = s.v5;
  } else if (NG == 2) {  // chunk 256 + l: K (s, z) for l < 32, V (s, z) chunk l - 32 after
    const int c = l - 32;
    dst[l < 32 ? kSlotKSz + l : kSlotVSz + c + (c >> 4)] = s.v4;
  } else if (l < 32) {   // chunk 256 + l: K (s, z) for l < 16, V (s, z) chunk l - 16
    dst[l < 16 ? kSlotKSz + l : kSlotVSz + l - 16] = s.v4;
  }
  lane_exchange();  // before any lane reads the page
}

struct WaveState {
  long aq[4];           // query digit operand per group (row: head lo>>2, digit lo&3)
  float qs[4];          // sum of q_int over group i of head hi
  float sq;             // q scale of head hi
  float m;              // running max (log2 units), head hi
  float lsum;           // partial sum of p over this lane's tokens, head hi
  float zacc;           // partial sum of w z_v, (head lo>>2, group lo&3)
  float of[8];          // unnormalized o~ of head hi, tile (G, F) at of[2G + F]
};

// FULL: all 64 token slots of the page are read; otherwise only slots in
// [t0, t1) (the partial first or last page of a token range).
// NG groups of 128 / NG channels per head: a group spans 4 / NG of the 32-channel
// slices that the MFMA tiles use, which share its (s, z) and its P.V weights.
// NCH chunks of 4 query heads would share the page (the K-code operands of the
// score MFMAs, the V scales and the V-code operands of the P.V MFMAs formed once,
// everything per head once per chunk); the kernel instantiates NCH = 1 only: 5 to
// 16 query heads per KV head take the wide path (compute_page_wide), whose score
// tiles hold one or two rows per head.
template <bool FULL, bool BF, int NG, int NCH>
__device__ inline void compute_page(WaveState (&st)[NCH], WaveLds<NCH>& L, int t0, int t1, int lo,
                                    int hi) {
  char* pb = reinterpret_cast<char*>(L.page);
  // ---- scores of head hi of every chunk for tokens 4*lo + u ----
  // code dword 2g + (hi>>1) of token 4*lo + u at byte 32u + 8g from the lane base
  const uint32_t* kc = reinterpret_cast<const uint32_t*>(pb + kLdsKCodes + 144 * lo + 4 * (hi >> 1));
  const uint32_t sh4 = 4u * (uint32_t)(hi & 1);
  uint4 ksz[NG];  // (s, z) of tokens 4*lo + (0..3), group i
#pragma unroll
  for (int i = 0; i < NG; ++i) ksz[i] = *reinterpret_cast<const uint4*>(pb + kLdsKSz + 256 * i + 16 * lo);
  float S[NCH][4];
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    float acc[NCH];
    v4i dg[NCH][NG];  // NG < 4: the digit sums of a group's slices accumulate in one MFMA chain
#pragma unroll
    for (int c = 0; c < NCH; ++c) acc[c] = 0.0f;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const uint32_t y = kc[8 * u + 2 * g] >> sh4;  // fields 2(hi&1), 2(hi&1)+1 of each byte
      const uint32_t msk = 0x03030303u;
      const long b = (long)((uint64_t)(y & msk) | ((uint64_t)((y >> 2) & msk) << 32));
#pragma unroll
      for (int c = 0; c < NCH; ++c) {
        if (NG == 4) {
          const v4i d = mfma32(st[c].aq[g], b);
          const int t = combine3(d[0], d[1], d[2]);
          const uint32_t sz = comp(ksz[g], u);
          // s * (acc - z * sum q_int) with s, z read from the packed pair
          float y = (float)t;
          sz_nz_acc<BF>(sz, st[c].qs[g], y);
          if (g == 0) {
            sz_s_mul<BF>(sz, y);
            acc[c] = y;
          } else {
            sz_s_acc<BF>(sz, y, acc[c]);
          }
        } else {
          const int j = g * NG / 4;  // the slice's group
          if (g % (4 / NG) == 0) dg[c][j] = mfma32(st[c].aq[g], b);
          else dg[c][j] = mfma32acc(st[c].aq[g], b, dg[c][j]);
        }
      }
    }
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      if (NG == 2) {  // 64 channels: |digit sums| <= 64 * 128 * 3, the combined sum < 2^31
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const uint32_t sz = comp(ksz[j], u);
          const int t = combine3(dg[c][j][0], dg[c][j][1], dg[c][j][2]);
          float y = (float)t;
          sz_nz_acc<BF>(sz, st[c].qs[j], y);
          if (j == 0) {
            sz_s_mul<BF>(sz, y);
            acc[c] = y;
          } else {
            sz_s_acc<BF>(sz, y, acc[c]);
          }
        }
      } else if (NG == 1) {
        // 128 channels: the combined sum can exceed int32, so the digits are combined
        // in fp32: 256 d_1 + d_2 is exact (< 2^24), and one rounding adds 65536 d_0
        const uint32_t sz = comp(ksz[0], u);
        const float T = fmaf((float)dg[c][0][0], 65536.0f, fmaf((float)dg[c][0][1], 256.0f, (float)dg[c][0][2]));
        float y = T;
        sz_nz_acc<BF>(sz, st[c].qs[0], y);
        sz_s_mul<BF>(sz, y);
        acc[c] = y;
      }
      S[c][u] = acc[c];
    }
  }

  // ---- V scales of the weight layout, shared by the chunks ----
  // lane (head wh = lo>>2, group wg = lo&3); their largest value on this page
  const int wh = lo >> 2, wg = lo & 3;
  constexpr int NE = NG == 1 ? 4 : NG == 2 ? 8 : 16;  // tokens whose weights a lane forms
  uint32_t sz[NE];
  float svmax;
  if (NG == 1) {
    // one group per head: lane (head wh, quarter wg) forms the weights of tokens
    // 16*hi + 4*wg + (0..3), dword wg of the head's k-group hi operand (every lane
    // busy, a quarter of the work per lane of the per-group layout)
    const uint4 vz = *reinterpret_cast<const uint4*>(pb + kLdsVSz + 64 * hi + 16 * wg);
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const int tok = 16 * hi + 4 * wg + b;
      sz[b] = comp(vz, b);
      if (!FULL && (tok < t0 || tok >= t1)) sz[b] = 0u;  // (0, 0): w = 0, z = 0
    }
    // largest V scale of the head on this page (bit patterns of positive scales)
    const uint32_t smax = max3_lo16(max3_lo16(sz[0], sz[1], sz[2]), sz[3], 0u);
    svmax = rows_max_pos(quad_max_pos(BF ? __uint_as_float(smax << 16) : h_lo(smax)));
  } else if (NG == 2) {
    // two groups per head: lane (head wh, group wg & 1, half wg >> 1) forms the
    // weights of tokens 16*hi + 8*(wg >> 1) + (0..7) of its group, dwords
    // 2*(wg >> 1) + (0, 1) of the group's k-group hi operand
    const int gq = wg & 1, hf = wg >> 1;
    uint4 vz[2];
#pragma unroll
    for (int j = 0; j < 2; ++j)
      vz[j] = *reinterpret_cast<const uint4*>(pb + kLdsVSz + 272 * gq + 64 * hi + 16 * (2 * hf + j));
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int tok = 16 * hi + 8 * hf + e;
      sz[e] = comp(vz[e >> 2], e & 3);
      if (!FULL && (tok < t0 || tok >= t1)) sz[e] = 0u;  // (0, 0): w = 0, z = 0
    }
    // largest V scale of the group on this page: this lane's 8 tokens, the other
    // half's lane (wg ^ 2) and the k-groups hi
    const uint32_t smax = max3_lo16(max3_lo16(sz[0], sz[1], sz[2]), max3_lo16(sz[3], sz[4], sz[5]),
                                    max3_lo16(sz[6], sz[7], 0u));
    float sv = BF ? __uint_as_float(smax << 16) : h_lo(smax);
    svmax = rows_max_pos(quad_pair_max_pos(sv));
  } else {
    uint4 vz[4];
#pragma unroll
    for (int j = 0; j < 4; ++j)
      vz[j] = *reinterpret_cast<const uint4*>(pb + kLdsVSz + 272 * wg + 64 * hi + 16 * j);
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      sz[e] = comp(vz[e >> 2], e & 3);
      if (!FULL && (16 * hi + e < t0 || 16 * hi + e >= t1)) sz[e] = 0u;  // (0, 0): w = 0, z = 0
    }
    // largest V scale of the group on this page: scales are positive binary16 or
    // bfloat16, so their bit patterns order like their values (high halves, the
    // zero points, ignored)
    uint32_t m5[6];
#pragma unroll
    for (int e = 0; e < 5; ++e) m5[e] = max3_lo16(sz[3 * e], sz[3 * e + 1], sz[3 * e + 2]);
    m5[5] = sz[15];
    const uint32_t smax = max3_lo16(max3_lo16(m5[0], m5[1], m5[2]), max3_lo16(m5[3], m5[4], m5[5]), 0u);
    svmax = rows_max_pos(BF ? __uint_as_float(smax << 16) : h_lo(smax));
  }

  // ---- per chunk: online softmax of head hi, then the P.V weights w = p * s_v of
  // (head wh, group wg) as three int8 digit operands in the chunk's LDS area ----
  auto valid = [&](int u) { return FULL || (4 * lo + u >= t0 && 4 * lo + u < t1); };
  float alpha[NCH];
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    float mx = -INFINITY;
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (valid(u)) mx = fmaxf(mx, S[c][u]);
    mx = row16_max1(mx) * st[c].sq;  // sq > 0; at least one valid token per page
    const float mn = fmaxf(st[c].m, mx);
    // alpha rescales the head's running sums (1 on the pages where the maximum
    // stays, which is most of them; the multiplies are kept: a wave-uniform skip
    // with a reference maximum that moves lazily needs registers that the
    // 4-waves-per-SIMD budget does not have)
    alpha[c] = ex2(st[c].m - mn);  // m = -inf on the first page -> 0
    const float pmax = ex2(mx - mn);
    float p[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) p[u] = valid(u) ? ex2(fmaf(st[c].sq, S[c][u], -mn)) : 0.0f;
    const float ls = ((p[0] + p[1]) + p[2]) + p[3];  // p >= 0: the sum from 0 without the 0 + p[0]
    st[c].lsum = fmaf(st[c].lsum, alpha[c], ls);
    st[c].m = mn;
    L.p[hi][lo] = make_float4(p[0], p[1], p[2], p[3]);
    L.hs[hi] = make_float2(alpha[c], pmax);  // every lane of the row writes the same value
    lane_exchange();

    char* wbase = c == 0 ? pb : reinterpret_cast<char*>(L.wdig[c == 0 ? 0 : c - 1]);
    const float2 hsw = L.hs[wh];
    const float sig = hsw.y * svmax;  // >= every w of the row on this page
    const float inv = sig > 0.0f ? kWMax * __builtin_amdgcn_rcpf(sig) : 0.0f;
    float zp = 0.0f;
    constexpr int NJ = NE / 4;  // dwords of digits per lane and digit row
    uint32_t aw[kNDig][NJ];
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      // p of tokens 4*(4*hi + q) + (0..3): q = wg (NG 1), 2*(wg>>1) + j (NG 2), j (NG 4)
      const int q = NG == 1 ? wg : NG == 2 ? 2 * (wg >> 1) + j : j;
      const float4 pw = L.p[wh][4 * hi + q];
      uint32_t f[4];
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        const int e = 4 * j + b;
        float w = compf(pw, b);
        sz_s_mul<BF>(sz[e], w);
        // mantissa of rne(w * inv) + 2^23 + 32896 = k + 32896, k in [0, 2^21]:
        // k = 65536 d_0 + 256 d_1 + d_2 with d_2, d_1 = (bytes 0, 1) ^ 0x80, d_0 = byte 2
        f[b] = __float_as_uint(fmaf(w, inv, kMagic + kDigitBias));
        sz_z_acc<BF>(sz[e], w, zp);  // unquantized w: differs from the quantized by <= 2^-22 sig
      }
      const uint32_t t01 = __builtin_amdgcn_perm(f[1], f[0], 0x05010400u) ^ 0x80808080u;  // [f0.0 f1.0 f0.1 f1.1]
      const uint32_t t23 = __builtin_amdgcn_perm(f[3], f[2], 0x05010400u) ^ 0x80808080u;
      const uint32_t h01 = __builtin_amdgcn_perm(f[1], f[0], 0x0c0c0602u);                // [f0.2 f1.2 0 0]
      const uint32_t h23 = __builtin_amdgcn_perm(f[3], f[2], 0x0c0c0602u);
      aw[2][j] = __builtin_amdgcn_perm(t23, t01, 0x05040100u);
      aw[1][j] = __builtin_amdgcn_perm(t23, t01, 0x07060302u);
      aw[0][j] = __builtin_amdgcn_perm(h23, h01, 0x05040100u);
    }
    if (NG == 1) {  // dword wg of the head's k-group hi operand
      L.ws[c][lo] = sig * (1.0f / kWMax);  // equal for the 16 lanes of head wh
      char* wp = wbase + 16 * (w_base(0) + w_slot(wh, hi)) + 4 * wg;
#pragma unroll
      for (int dg = 0; dg < kNDig; ++dg) *reinterpret_cast<uint32_t*>(wp + 16 * dg) = aw[dg][0];
    } else if (NG == 2) {  // dwords 2*(wg>>1) + (0, 1) of group wg & 1
      L.ws[c][lo] = sig * (1.0f / kWMax);  // lanes wg and wg ^ 2: group wg & 1 of head wh
      char* wp = wbase + 16 * (w_base(wg & 1) + w_slot(wh, hi)) + 8 * (wg >> 1);
#pragma unroll
      for (int dg = 0; dg < kNDig; ++dg)
        *reinterpret_cast<uint2*>(wp + 16 * dg) = make_uint2(aw[dg][0], aw[dg][1]);
    } else {  // group wg, rows 3*wh + digit, k-group hi
      L.ws[c][lo] = sig * (1.0f / kWMax);
      char* wp = wbase + 16 * (w_base(wg) + w_slot(wh, hi));
#pragma unroll
      for (int dg = 0; dg < kNDig; ++dg)
        *reinterpret_cast<uint4*>(wp + 16 * dg) = make_uint4(aw[dg][0], aw[dg][1], aw[dg][2], aw[dg][3]);
    }
    st[c].zacc = fmaf(st[c].zacc, hsw.x, zp);
  }

  lane_exchange();
  // ---- P.V on the matrix cores: lane (channel column, head hi), every chunk ----
  // B operand: field 2F + (lo>>3) of each token's byte, taken in place by the mask
  // mk = 3 << 2(lo>>3): columns lo >= 8 hold 4 x code (undone when the state is written)
  const uint32_t mk = 0x03030303u << (2 * (lo >> 3));
  // V codes of quad 8G + (lo&7), tokens 16*hi + (0..15)
  const char* vb = pb + kLdsVCodes + 16 * (4 * (lo & 7) + (hi ^ (((lo >> 2) & 1) << 1)));
  // A operand row (head lo>>2, digit lo&3); the padding digit row reads digit 2
  const int arow = 16 * (w_slot(lo >> 2, hi) + min(lo & 3, 2));
  float4 ws[NCH];
#pragma unroll
  for (int c = 0; c < NCH; ++c) ws[c] = *reinterpret_cast<const float4*>(&L.ws[c][4 * hi]);
#pragma unroll
  for (int G = 0; G < 4; ++G) {
    v4i aop[NCH];
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      const char* wbase = c == 0 ? pb : reinterpret_cast<const char*>(L.wdig[c == 0 ? 0 : c - 1]);
      const uint4 a4 = *reinterpret_cast<const uint4*>(wbase + arow + 16 * w_base(G * NG / 4));
      aop[c] = v4i{(int)a4.x, (int)a4.y, (int)a4.z, (int)a4.w};
    }
    const uint4 x = *reinterpret_cast<const uint4*>(vb + 512 * G);  // quad 8G + (lo&7)
#pragma unroll
    for (int F = 0; F < 2; ++F) {
      const v4i bv = {(int)((x.x >> (4 * F)) & mk), (int)((x.y >> (4 * F)) & mk),
                      (int)((x.z >> (4 * F)) & mk), (int)((x.w >> (4 * F)) & mk)};
#pragma unroll
      for (int c = 0; c < NCH; ++c) {
        const v4i d = mfma64(aop[c], bv);
        const int t = combine3(d[0], d[1], d[2]);
        float& o = st[c].of[2 * G + F];
        o = fmaf((float)t, compf(ws[c], G * NG / 4), o * alpha[c]);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Wide instances (5 to 16 query heads per kv-head).  The scores of all the
// kv-head's query heads come from one set of fp16 MFMAs, so the per-(token, head,
// group) work after them is one scale FMA (two with 8 heads, below); the P.V
// products stay on the int8 MFMAs in chunks of 4 heads (as above).  Up to 8
// heads (RPH = 2 rows per head) the hi and lo halves of q~ are two MFMA rows of
// the head (row lo: head lo>>1, half lo&1), one MFMA per slice and tile, and
// the lane's D registers hold heads 2hi + (i>>1) whose halves add up; from 9
// heads (RPH = 1) a row is a head and the halves are two chained MFMAs.
//
// v_mfma_f32_16x16x32_f16: A row = head lo, k-slots 8*hi + e; B column lo,
// k-slots 8*hi + e; D lane l, register i = (head 4*hi + i, column lo).  A K code
// enters B as a binary16 subnormal: its two bits, masked in place at field j of
// a byte (bits c * 4^j), are the value c * 4^j * 2^-24, exactly.  The A side
// holds q~ * E / 4^j as a hi + lo pair of binary16 values (E a power of two per
// head that puts max|q~| * E in [2^14, 2^15)), so every product is exactly
// q~ * c * E * 2^-24 and a slice's sum is exact up to the fp32 accumulation.
// Token tile u: column lo is token 4*lo + u.  Slice g (32 channels), k-group hi:
// the codes of bytes A = 8g + 2hi and A + 1 of the token (channels 32g + 8hi + f
// and 32g + 8hi + 4 + f for field f), Y = byte A | byte (A + 1) << 16 and
// P_f = Y & (0x00030003 << 2f); B dwords (P_0, P_1, P_2, P_3), so k-slot e is
// field e>>1 of byte A (e even) or A + 1 (e odd).  Two chained MFMAs per slice
// and tile take the hi and the lo halves of q~ against the same B.  The
// zero-point term sum_g s_g z_g Q_g(h) of a tile is one fp32
// MFMA (16x16x4: A row = head, k = group: Q_g E 2^-24; B k = group, column =
// token: s_g z_g, exact in fp32) that seeds the sum of the scaled slices.
//
// Softmax per page: p' = 2^(score - page max + 21 - e), with svmax < 2^e the
// largest V scale of the page, so that every weight s_v p' lies in [0, 2^21]
// and is quantized as it is (no per-(head, group) rescale).  The true weight is
// p' s_v ws, ws = 2^(page max - m - 21 + e), with m a reference maximum per head
// that only moves when a page's maximum exceeds it by more than kSlack (sums
// relative to m then stay below 2^kSlack times their true size; the running
// sums are rescaled only on those pages).

typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef float f4v __attribute__((ext_vector_type(4)));

__device__ inline f4v mfma_h(u4 a, u4 b, f4v c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(h8, a), __builtin_bit_cast(h8, b), c,
                                                0, 0, 0);
}
__device__ inline f4v mfma_f(float a, float b) {
  const f4v z = {0.0f, 0.0f, 0.0f, 0.0f};
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, z, 0, 0, 0);
}
// s * z of a packed (scale, zero) word (exact in fp32), in plain C like every
// operation next to the wide path's MFMAs: the compiler inserts the MFMA
// read/write wait states only around instructions it sees, not inline asm.
template <bool BF>
__device__ inline float sz_prod(uint32_t h) {
  if (BF) return __uint_as_float(h << 16) * __uint_as_float(h & 0xffff0000u);
  return fmaf(__half2float(__ushort_as_half((uint16_t)(h & 0xffffu))),
              __half2float(__ushort_as_half((uint16_t)(h >> 16))), 0.0f);
}

// p' of a page for the chunks' weight lanes: [head][token / 4] float4, pitch 17.
// Up to 12 heads it lies over the page's K area (spent once the scores are done).
template <int NCH>
struct WideLdsX {};
template <>
struct WideLdsX<4> {
  uint4 pqx[16 * 17];
};
template <int NCH>
struct WideLds : WideLdsX<NCH> {
  uint4 page[kSlots];            // page-head block (slot placement above)
  uint4 wdig[NCH][kWSlots];      // weight digits of each chunk
  float wsh[16];                 // per head on this page: P.V scale ws
  float alh[16];                 // per head: rescale factor alpha (pages that move m)
};
template <int NCH>
__device__ inline float4* wide_pq(WideLds<NCH>& L) {
  if constexpr (NCH == 4) return reinterpret_cast<float4*>(L.pqx);
  else return reinterpret_cast<float4*>(L.page);
}

// Score rows: (head, half) pairs at 2 rows per head (RPH 2: row r holds head
// r >> 1), or one row per head (RPH 1: row r holds head (r >> 2) + 4 (r & 3), so
// that D register j of lane (hi, lo) is head hi + 4j and, at 9 to 12 heads, the
// padding heads 12..15 are register 3 of every lane: that register is skipped).
template <int NCH>
struct WideRows {
  static constexpr int RPH = NCH <= 2 ? 2 : 1;  // MFMA rows per head
  static constexpr int HPL = 4 / RPH;           // heads per lane in the score layout
  static constexpr int NJ = NCH == 3 ? 3 : HPL; // of them, those that can be real heads
  __device__ static int row_head(int r) { return RPH == 1 ? (r >> 2) + 4 * (r & 3) : r >> 1; }
  __device__ static int lane_head(int hi, int j) { return RPH == 1 ? hi + 4 * j : HPL * hi + j; }
};
template <int NCH>
struct WideState {
  static constexpr int RPH = WideRows<NCH>::RPH, HPL = WideRows<NCH>::HPL;
  u4 aq[4][3 - RPH]; // score A operands of row lo (head row_head(lo)), slice g, k-group hi:
                     // RPH 1: its hi (0) and lo (1) halves; RPH 2: the half lo&1
  float az;          // zero-point MFMA A operand of row lo, group hi: E 2^-24 sum of q~
  float sq[HPL];     // 2^24 / E of head lane_head(hi, j) (log2 units per accumulated score)
  float m[HPL];      // reference maximum (log2 units) of that head
  float lsum[HPL];   // partial sum of p relative to m over this lane's tokens, that head
  float zacc[NCH];   // partial sum of w z_v of (head 4c + (lo>>2), group lo&3)
  float of[NCH][8];  // unnormalized o~ of head 4c + hi, tile (G, F) at of[c][2G + F]
};

template <bool FULL, bool BF, int NG, int NCH>
__device__ inline void compute_page_wide(WideState<NCH>& st, WideLds<NCH>& L, int t0, int t1, int lo,
                                         int hi) {
  char* pb = reinterpret_cast<char*>(L.page);
  const int l = threadIdx.x & 63;
  __builtin_assume(hi >= 0 && hi < 4);
  __builtin_assume(lo >= 0 && lo < 16);
  auto valid = [&](int u) { return FULL || (4 * lo + u >= t0 && 4 * lo + u < t1); };

  // ---- largest V scale of the page over its valid tokens: lane l < 16 NG reads V
  // (s, z) chunk l (tokens 4(l&15) + b of group l>>4) ----
  int esv;
  {
    uint32_t mloc = 0u;
    if (NG == 4 || l < 16 * NG) {
      const uint4 w = *reinterpret_cast<const uint4*>(pb + kLdsVSz + 16 * (l + (l >> 4)));
      uint32_t x[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
      for (int b = 0; b < 4; ++b)
        if (!FULL && (4 * (l & 15) + b < t0 || 4 * (l & 15) + b >= t1)) x[b] = 0u;
      mloc = max(max(x[0] & 0xffffu, x[1] & 0xffffu), max(x[2] & 0xffffu, x[3] & 0xffffu));
    }
    const float sv = rows_max_pos(row16_max1(BF ? __uint_as_float(mloc << 16) : h_lo(mloc)));
    frexpf(sv, &esv);  // sv < 2^esv
  }
  const float cw = (float)(21 - esv);

  // ---- scores of heads lane_head(hi, j) for tokens 4lo + u ----
  const uint32_t* kc = reinterpret_cast<const uint32_t*>(pb + kLdsKCodes + 144 * lo + 4 * (hi >> 1));
  const uint32_t sel = (hi & 1) ? 0x0C030C02u : 0x0C010C00u;  // bytes 2(hi&1), +1 to the two halves
  constexpr int RPH = WideRows<NCH>::RPH, HPL = WideRows<NCH>::HPL, NJ = WideRows<NCH>::NJ;
  // zero-point terms of the tiles: dz[u] = sum_g Q_g s_g z_g (B: group hi of token 4lo + u)
  f4v dz[4];
  {
    const uint4 kszb = *reinterpret_cast<const uint4*>(pb + kLdsKSz + 256 * (hi < NG ? hi : 0) + 16 * lo);
#pragma unroll
    for (int u = 0; u < 4; ++u) dz[u] = mfma_f(st.az, hi < NG ? sz_prod<BF>(comp(kszb, u)) : 0.0f);
  }
  // slices g (outer) for the four token tiles; a group's slices chain in the MFMA
  // accumulator and its scale is applied after the last one
  float acc[4][HPL];
  f4v d[4];
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    const bool first = (g % (4 / NG)) == 0, lastg = (g + 1) % (4 / NG) == 0;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const uint32_t D = kc[8 * u + 2 * g];
      const uint32_t Y = __builtin_amdgcn_perm(D, D, sel);
      const u4 bk = {Y & 0x00030003u, Y & 0x000C000Cu, Y & 0x00300030u, Y & 0x00C000C0u};
      const f4v zero = {0.0f, 0.0f, 0.0f, 0.0f};
      d[u] = mfma_h(st.aq[g][0], bk, first ? zero : d[u]);
      if (RPH == 1) d[u] = mfma_h(st.aq[g][1], bk, d[u]);
    }
    if (lastg) {  // (s, z) of tokens 4lo + (0..3) of the group
      const uint4 kg = *reinterpret_cast<const uint4*>(pb + kLdsKSz + 256 * (g * NG / 4) + 16 * lo);
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
          const float x = RPH == 1 ? d[u][j] : d[u][2 * j] + d[u][2 * j + 1];
          acc[u][j] = sz_s_fma_c<BF>(comp(kg, u), x, g + 1 == 4 / NG ? -dz[u][RPH * j] : acc[u][j]);
        }
    }
  }

  // ---- online softmax of heads lane_head(hi, j) ----
  float mx[HPL];
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    float x = -INFINITY;
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (valid(u)) x = fmaxf(x, acc[u][j]);
    mx[j] = x;
  }
  // at least one valid token per page
  if (NJ == 4) row16_max4(mx[0], mx[NJ > 1 ? 1 : 0], mx[NJ > 2 ? 2 : 0], mx[NJ > 3 ? 3 : 0]);
  else if (NJ == 3) row16_max3(mx[0], mx[NJ > 1 ? 1 : 0], mx[NJ > 2 ? 2 : 0]);
  else row16_max2(mx[0], mx[NJ > 1 ? 1 : 0]);
  bool need = false;
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    mx[j] *= st.sq[j];
    need = need || !(mx[j] <= st.m[j] + kSlack);
  }
  if (__ballot(need) != 0ull) {  // wave-uniform
    float alpha[HPL];
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const float mn = fmaxf(st.m[j], mx[j]);
      alpha[j] = ex2(st.m[j] - mn);  // m = -inf on the first page -> 0
      st.m[j] = mn;
      st.lsum[j] *= alpha[j];
    }
    // each head's alpha through LDS to the zero-point sums (head 4c + (lo>>2)) and
    // the o~ accumulators (head 4c + hi) of the lane
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int hh = WideRows<NCH>::lane_head(hi, j);
      if (hh < 4 * NCH) L.alh[hh] = alpha[j];  // every lane of the row writes the same value
    }
    lane_exchange();
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      st.zacc[c] *= L.alh[4 * c + (lo >> 2)];
      const float a = L.alh[4 * c + hi];
#pragma unroll
      for (int k = 0; k < 8; ++k) st.of[c][k] *= a;
    }
  }
  float4* pq = wide_pq(L);
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const int hh = WideRows<NCH>::lane_head(hi, j);
    const float c = cw - mx[j];
    const float ws = ex2(mx[j] - st.m[j] - cw);
    float pv[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) pv[u] = valid(u) ? ex2(fmaf(st.sq[j], acc[u][j], c)) : 0.0f;
    const float ls = ((pv[0] + pv[1]) + pv[2]) + pv[3];
    st.lsum[j] = fmaf(ls, ws, st.lsum[j]);
    if (hh < 4 * NCH) {
      pq[hh * 17 + lo] = make_float4(pv[0], pv[1], pv[2], pv[3]);
      L.wsh[hh] = ws;  // every lane of the row writes the same value
    }
  }
  lane_exchange();

  const int wh = lo >> 2, wg = lo & 3;
  // ---- per chunk: the P.V weights w' = s_v p' of (head 4c + wh, group wg) as three
  // int8 digit operands in the chunk's LDS area ----
  constexpr int NE = NG == 1 ? 4 : NG == 2 ? 8 : 16;  // tokens whose weights a lane forms
  uint32_t sz[NE];
  if (NG == 1) {  // lane (head wh, quarter wg): tokens 16*hi + 4*wg + (0..3)
    const uint4 vz = *reinterpret_cast<const uint4*>(pb + kLdsVSz + 64 * hi + 16 * wg);
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const int tok = 16 * hi + 4 * wg + b;
      sz[b] = comp(vz, b);
      if (!FULL && (tok < t0 || tok >= t1)) sz[b] = 0u;
    }
  } else if (NG == 2) {  // lane (head wh, group wg & 1, half wg >> 1): tokens 16*hi + 8*(wg >> 1) + (0..7)
    const int gq = wg & 1, hf = wg >> 1;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const uint4 vz = *reinterpret_cast<const uint4*>(pb + kLdsVSz + 272 * gq + 64 * hi + 16 * (2 * hf + j));
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        const int tok = 16 * hi + 8 * hf + 4 * j + b;
        sz[4 * j + b] = comp(vz, b);
        if (!FULL && (tok < t0 || tok >= t1)) sz[4 * j + b] = 0u;
      }
    }
  } else {  // lane (head wh, group wg): tokens 16*hi + (0..15)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint4 vz = *reinterpret_cast<const uint4*>(pb + kLdsVSz + 272 * wg + 64 * hi + 16 * j);
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        sz[4 * j + b] = comp(vz, b);
        if (!FULL && (16 * hi + 4 * j + b < t0 || 16 * hi + 4 * j + b >= t1)) sz[4 * j + b] = 0u;
      }
    }
  }
  float szp[NE];
#pragma unroll
  for (int e = 0; e < NE; ++e) szp[e] = sz_prod<BF>(sz[e]);
  // the digit bias as a register operand (a literal would split the mixed-precision
  // FMA into a conversion and an FMA)
  float magic = kMagic + kDigitBias;
  asm("" : "+v"(magic));
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    const int hh = 4 * c + wh;
    const float wsv = L.wsh[hh];
    char* wbase = reinterpret_cast<char*>(L.wdig[c]);
    float zp = 0.0f;
    constexpr int NJ = NE / 4;
    uint32_t aw[kNDig][NJ];
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int q = NG == 1 ? wg : NG == 2 ? 2 * (wg >> 1) + j : j;
      const float4 pw = pq[hh * 17 + 4 * hi + q];
      uint32_t f[4];
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        const int e = 4 * j + b;
        // mantissa of rne(w') + 2^23 + 32896 = k + 32896, k in [0, 2^21] (as above)
        f[b] = __float_as_uint(sz_s_fma_asm<BF>(sz[e], compf(pw, b), magic));
        zp = fmaf(szp[e], compf(pw, b), zp);
      }
      const uint32_t t01 = __builtin_amdgcn_perm(f[1], f[0], 0x05010400u) ^ 0x80808080u;
      const uint32_t t23 = __builtin_amdgcn_perm(f[3], f[2], 0x05010400u) ^ 0x80808080u;
      const uint32_t h01 = __builtin_amdgcn_perm(f[1], f[0], 0x0c0c0602u);
      const uint32_t h23 = __builtin_amdgcn_perm(f[3], f[2], 0x0c0c0602u);
      aw[2][j] = __builtin_amdgcn_perm(t23, t01, 0x05040100u);
      aw[1][j] = __builtin_amdgcn_perm(t23, t01, 0x07060302u);
      aw[0][j] = __builtin_amdgcn_perm(h23, h01, 0x05040100u);
    }
    if (NG == 1) {
      char* wp = wbase + 16 * (w_base(0) + w_slot(wh, hi)) + 4 * wg;
#pragma unroll
      for (int dg = 0; dg < kNDig; ++dg) *reinterpret_cast<uint32_t*>(wp + 16 * dg) = aw[dg][0];
    } else if (NG == 2) {
      char* wp = wbase + 16 * (w_base_v(wg & 1) + w_slot(wh, hi)) + 8 * (wg >> 1);
#pragma unroll
      for (int dg = 0; dg < kNDig; ++dg)
        *reinterpret_cast<uint2*>(wp + 16 * dg) = make_uint2(aw[dg][0], aw[dg][1]);
    } else {
      char* wp = wbase + 16 * (w_base_v(wg) + w_slot(wh, hi));
#pragma unroll
      for (int dg = 0; dg < kNDig; ++dg)
        *reinterpret_cast<uint4*>(wp + 16 * dg) = make_uint4(aw[dg][0], aw[dg][1], aw[dg][2], aw[dg][3]);
    }
    st.zacc[c] = fmaf(zp, wsv, st.zacc[c]);
  }

  lane_exchange();
  // ---- P.V on the int8 matrix cores: lane (channel column, head hi), every chunk ----
  const uint32_t mk = 0x03030303u << (2 * (lo >> 3));
  const char* vb = pb + kLdsVCodes + 16 * (4 * (lo & 7) + (hi ^ (((lo >> 2) & 1) << 1)));
  const int arow = 16 * (w_slot(lo >> 2, hi) + min(lo & 3, 2));
  float wsc[NCH];
#pragma unroll
  for (int c = 0; c < NCH; ++c) wsc[c] = L.wsh[4 * c + hi];
#pragma unroll
  for (int G = 0; G < 4; ++G) {
    v4i aop[NCH];
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      const uint4 a4 = *reinterpret_cast<const uint4*>(reinterpret_cast<const char*>(L.wdig[c]) + arow +
                                                       16 * w_base(G * NG / 4));
      aop[c] = v4i{(int)a4.x, (int)a4.y, (int)a4.z, (int)a4.w};
    }
    const uint4 x = *reinterpret_cast<const uint4*>(vb + 512 * G);
#pragma unroll
    for (int F = 0; F < 2; ++F) {
      const v4i bv = {(int)((x.x >> (4 * F)) & mk), (int)((x.y >> (4 * F)) & mk),
                      (int)((x.z >> (4 * F)) & mk), (int)((x.w >> (4 * F)) & mk)};
#pragma unroll
      for (int c = 0; c < NCH; ++c) {
        const v4i d = mfma64(aop[c], bv);
        const int t = combine3(d[0], d[1], d[2]);
        st.of[c][2 * G + F] = fmaf((float)t, wsc[c], st.of[c][2 * G + F]);
      }
    }
  }
}

// The INT2 token range of a sequence in page terms: pages [first, first + npg)
// of its block-table row; token slots [t0, 64) of the range's first page and
// [0, t1) of its last page are in the range (t0 = 0, t1 = 64 when aligned).
struct TokRange {
  int first, npg, t0, t1;
};
// Tokens [lo, hi) of a sequence.
__device__ inline TokRange tok_range(int lo, int hi) {
  TokRange r;
  r.first = lo / kP;
  r.npg = hi > lo ? (hi + kP - 1) / kP - r.first : 0;
  r.t0 = lo - r.first * kP;
  r.t1 = hi - (r.first + r.npg - 1) * kP;
  return r;
}

// Pages [p0, p1) of the token range R of sequence b (page indices relative to
// R.first), kv-head kvh: each page-head block is staged into `page` and handed to
// compute(full, t0, t1) (full: all 64 token slots; otherwise slots [t0, t1)).
// The wave has done `done0` of its `total` pages before these (issue-priority
// bands).  Without MIXED the range starts at token 0 (R.t0 = 0).
template <bool MIXED, int NG, typename Compute>
__device__ __attribute__((always_inline)) inline void walk_pages(uint4* page, const uint8_t* __restrict__ pages,
                                                                 int Hkv, const int32_t* __restrict__ block_table,
                                                                 int max_pages, int b, TokRange R, int kvh, int p0,
                                                                 int p1, int done0, int total, Compute&& compute) {
  const int l = threadIdx.x;
  const int npg = R.npg;
  const int32_t* __restrict__ bt = block_table + (size_t)b * max_pages + (MIXED ? R.first : 0);
  const uint8_t* __restrict__ base = pages + (size_t)kvh * block_bytes(NG);
  const size_t page_stride = (size_t)Hkv * block_bytes(NG);
  // Block-table entries of the split, 64 pages at a time: lane i holds the entry
  // of page cb + i (a vector load, so that waiting for it never waits on LDS).
  int cb = p0;
  int btv = (p0 + l < p1) ? bt[p0 + l] : 0;
  Stage sg;
  if (p0 < p1) stage_load<NG, true>(sg, base + (size_t)__builtin_amdgcn_readlane(btv, 0) * page_stride, l);
  // pages [p0, pf) are full; page pf (if < p1) is the range's partial last page
  int pf = (p0 < p1 && p1 == npg && R.t1 != kP) ? p1 - 1 : p1;
  int pg = p0;
  if (MIXED && p0 == 0 && p0 < p1 && R.t0 != 0) {  // the range's partial first page
    stage_store<NG>(page, sg, l);
    stage_load<NG, true>(sg, base + (size_t)__builtin_amdgcn_readlane(btv, min(1, p1 - 1)) * page_stride, l);
    compute(std::false_type{}, R.t0, npg == 1 ? R.t1 : kP);
    pg = 1;
    pf = max(pf, 1);  // a one-page range is done
  }
  // Full pages in four bands of the wave's whole page count (done0 pages of it
  // before this piece, total in all): the wave lowers its issue priority at
  // 25 %, 50 % and 75 % of its pages.  Waves sharing a SIMD otherwise issue in age
  // order, and the youngest of them finished up to 1.7x later than the oldest
  // with the same page count; waves that are behind now go first.
  for (int band = 1; band <= 4; ++band) {
    const int lim = (int)(((int64_t)(25 * band) * total + 99) / 100) - done0 + p0;  // band end
    const int e = min(max(lim, pg), pf);
    for (; pg < e; ++pg) {
      stage_store<NG>(page, sg, l);
      const int nx = min(pg + 1, p1 - 1);  // page pg+1 (the last page again at the end)
      if (nx - cb >= 64) {                 // uniform: next 64 entries
        cb += 64;
        btv = (cb + l < p1) ? bt[cb + l] : 0;
      }
      stage_load<NG, true>(sg, base + (size_t)__builtin_amdgcn_readlane(btv, nx - cb) * page_stride, l);
      compute(std::true_type{}, 0, kP);
    }
    if (band < 4 && lim > p0 && lim <= pf) {  // the band ended inside this piece
      if (band == 1) __builtin_amdgcn_s_setprio(2);
      else if (band == 2) __builtin_amdgcn_s_setprio(1);
      else __builtin_amdgcn_s_setprio(0);
    }
  }
  if (pf < p1) {  // the partial last page; the stage holds it
    stage_store<NG>(page, sg, l);
    compute(std::false_type{}, 0, R.t1);
  }

}

// Pages [p0, p1) of the token range R of sequence b, kv-head kvh, one chunk of
// at most 4 query heads: online softmax over the pages and the partial state
// written to slot `piece` of the (sequence, head) rows, whose slots are
// row_stride apart.  `last`: the piece ends the range, so slots piece + 1 ..
// num_splits - 1 are marked empty.
template <bool MIXED, bool BF, int NG, int NCH>
__device__ __attribute__((always_inline)) inline void process_piece(WaveLds<NCH>& L, const uint8_t* __restrict__ pages, int Hkv, int Hq,
                                     const int32_t* __restrict__ block_table, int max_pages, int b,
                                     TokRange R, int kvh, int p0, int p1, int piece,
                                     bool last, int num_splits, int row_stride,
                                     const float* __restrict__ qt,
                                     float* __restrict__ part_o, float* __restrict__ part_ml,
                                     int done0, int total) {
  const int g_heads = Hq / Hkv;
  const int l = threadIdx.x, lo = l & 15, hi = l >> 4;

  WaveState st[NCH];
  // ---- query operands: q_int = rne(q~ * Q / max|q~|), three int8 digits ----
  // Lane (head lo>>2, digit lo&3, k-group hi) holds, for group g, element e of
  // the k-group: channel 32g + 16(hi>>1) + 4(e&3) + 2(hi&1) + (e>>2).  Chunk c
  // holds query heads 4c .. 4c + 3 of the KV head.
#pragma unroll
  for (int chunk = 0; chunk < NCH; ++chunk) {
    WaveState& sc = st[chunk];
    const int h = lo >> 2, dsel = lo & 3;
    const int hloc = 4 * chunk + h;
    float qv[4][8];
    float amax = 0.0f;
#pragma unroll
    for (int g = 0; g < 4; ++g)
#pragma unroll
      for (int e = 0; e < 8; ++e) qv[g][e] = 0.0f;
    if (hloc < g_heads) {
      const float* src = qt + ((size_t)b * Hq + kvh * g_heads + hloc) * kD + 16 * (hi >> 1) + 2 * (hi & 1);
#pragma unroll
      for (int g = 0; g < 4; ++g)
#pragma unroll
        for (int bb = 0; bb < 4; ++bb) {
          const float2 x = *reinterpret_cast<const float2*>(src + 32 * g + 4 * bb);
          qv[g][bb] = x.x;
          qv[g][4 + bb] = x.y;
        }
#pragma unroll
      for (int g = 0; g < 4; ++g)
#pragma unroll
        for (int e = 0; e < 8; ++e) amax = fmaxf(amax, fabsf(qv[g][e]));
    }
    amax = rows_max(amax);  // all 128 channels of the head (k-groups hi)
    const float inv = amax > 0.0f ? kQMax / amax : 0.0f;
    const float sq = amax > 0.0f ? amax * (1.0f / kQMax) : 1.0f;
    int qsum[4];
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      int sum = 0;
      uint32_t w[2] = {0u, 0u};
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int v = (int)rintf(qv[g][e] * inv);
        sum += v;
        // q = 65536 d_0 + 256 d_1 + d_2 with d_2 = q - 256 c1, c1 = (q + 128) >> 8, etc.
        const int c1 = (v + 128) >> 8;
        const int d2 = v - 256 * c1;
        const int d0 = (c1 + 128) >> 8;
        const int d1 = c1 - 256 * d0;
        const int dv = dsel == 0 ? d0 : dsel == 1 ? d1 : dsel == 2 ? d2 : 0;
        w[e >> 2] |= ((uint32_t)dv & 0xffu) << (8 * (e & 3));
      }
      sc.aq[g] = (long)((uint64_t)w[0] | ((uint64_t)w[1] << 32));
      // sum over the group's 32 channels (k-groups hi), exact in int
      sum += __shfl_xor(sum, 16, 64);
      sum += __shfl_xor(sum, 32, 64);
      qsum[g] = sum;
    }
    L.qs[lo] = dsel == 0 ? qsum[0] : dsel == 1 ? qsum[1] : dsel == 2 ? qsum[2] : qsum[3];  // (head h, group dsel)
    L.sq[h] = sq;  // lanes of equal h write equal values
    lane_exchange();
    const int4 q4 = *reinterpret_cast<const int4*>(&L.qs[4 * hi]);
    if (NG == 4) {
      sc.qs[0] = (float)q4.x; sc.qs[1] = (float)q4.y; sc.qs[2] = (float)q4.z; sc.qs[3] = (float)q4.w;
    } else if (NG == 2) {  // sums over the group's slices, in int32 (|sum| < 2^31)
      sc.qs[0] = (float)(q4.x + q4.y); sc.qs[1] = (float)(q4.z + q4.w);
      sc.qs[2] = sc.qs[3] = 0.0f;
    } else {
      sc.qs[0] = (float)(q4.x + q4.y + q4.z + q4.w);
      sc.qs[1] = sc.qs[2] = sc.qs[3] = 0.0f;
    }
    sc.sq = L.sq[hi];
    sc.m = -INFINITY;
    sc.lsum = 0.0f;
    sc.zacc = 0.0f;
#pragma unroll
    for (int k = 0; k < 8; ++k) sc.of[k] = 0.0f;
  }

  walk_pages<MIXED, NG>(L.page, pages, Hkv, block_table, max_pages, b, R, kvh, p0, p1, done0, total,
                        [&](auto full, int t0, int t1) {
                          compute_page<decltype(full)::value, BF, NG, NCH>(st, L, t0, t1, lo, hi);
                        });

  // ---- write the split's partial state, per chunk ----
#pragma unroll
  for (int chunk = 0; chunk < NCH; ++chunk) {
    const WaveState& sc = st[chunk];
    const float ltot = row16_sum(sc.lsum);  // head hi
    float ztot = rows_sum(sc.zacc);         // (head lo>>2, group lo&3)
    if (NG == 1) ztot = quad_sum(ztot);     // the head's quarters: its one group
    if (NG == 2)                            // the group's halves: lanes wg and wg ^ 2
      ztot += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(ztot), 0x4E, 0xF, 0xF, false));
    L.ws[0][lo] = ztot;                     // lanes of equal lo write equal values
    lane_exchange();
    const float4 zh = *reinterpret_cast<const float4*>(&L.ws[0][4 * hi]);
    const int hout = 4 * chunk + hi;        // head of this lane's accumulators
    if (hout >= g_heads) continue;          // padding head
    const size_t row = ((size_t)b * Hq + kvh * g_heads + hout) * (MIXED ? row_stride : num_splits) + piece;
    if (last && lo == 0)  // the range's last piece: the remaining slots hold nothing
      for (int s2 = piece + 1; s2 < num_splits; ++s2) {
        part_ml[(row + s2 - piece) * 2] = -INFINITY;
        part_ml[(row + s2 - piece) * 2 + 1] = 0.0f;
      }
    const bool empty = sc.m == -INFINITY;
    const float cs = lo >= 8 ? 0.25f : 1.0f;  // P.V columns lo >= 8 accumulate 4 x code
#pragma unroll
    for (int G = 0; G < 4; ++G) {
#pragma unroll
      for (int F = 0; F < 2; ++F) {
        const int ch = 32 * G + 4 * (lo & 7) + 2 * F + (lo >> 3);
        part_o[row * kD + ch] = empty ? 0.0f : fmaf(sc.of[2 * G + F], cs, -compf(zh, G * NG / 4));
      }
    }
    if (lo == 0) {
      part_ml[row * 2] = sc.m;
      part_ml[row * 2 + 1] = ltot;
    }
  }
}

// The same for 5 to 16 query heads per kv-head (all of them in one wave: scores
// with one MFMA row per head, P.V in chunks of 4 heads).
template <bool MIXED, bool BF, int NG, int NCH>
__device__ __attribute__((always_inline)) inline void process_piece_wide(
    WideLds<NCH>& L, const uint8_t* __restrict__ pages, int Hkv, int Hq, const int32_t* __restrict__ block_table,
    int max_pages, int b, TokRange R, int kvh, int p0, int p1, int piece, bool last, int num_splits,
    int row_stride, const float* __restrict__ qt, float* __restrict__ part_o, float* __restrict__ part_ml,
    int done0, int total) {
  const int g_heads = Hq / Hkv;
  const int l = threadIdx.x & 63, lo = l & 15, hi = l >> 4;
  const size_t stride = MIXED ? row_stride : num_splits;

  WideState<NCH> st;
  constexpr int RPH = WideRows<NCH>::RPH, HPL = WideRows<NCH>::HPL, NJ = WideRows<NCH>::NJ;
  // ---- query operands of head hq = row_head(lo): lane k-group hi holds channels
  // 32g + 8hi + (0..7) of slice g ----
  {
    const int hq = WideRows<NCH>::row_head(lo);
    float qv[4][8];
    float amax = 0.0f;
#pragma unroll
    for (int g = 0; g < 4; ++g)
#pragma unroll
      for (int e = 0; e < 8; ++e) qv[g][e] = 0.0f;
    if (hq < g_heads) {
      const float* src = qt + ((size_t)b * Hq + kvh * g_heads + hq) * kD + 8 * hi;
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const float4 x0 = *reinterpret_cast<const float4*>(src + 32 * g);
        const float4 x1 = *reinterpret_cast<const float4*>(src + 32 * g + 4);
        qv[g][0] = x0.x; qv[g][1] = x0.y; qv[g][2] = x0.z; qv[g][3] = x0.w;
        qv[g][4] = x1.x; qv[g][5] = x1.y; qv[g][6] = x1.z; qv[g][7] = x1.w;
      }
#pragma unroll
      for (int g = 0; g < 4; ++g)
#pragma unroll
        for (int e = 0; e < 8; ++e) amax = fmaxf(amax, fabsf(qv[g][e]));
    }
    amax = rows_max(amax);  // all 128 channels of the head
    int ex = 0;
    if (amax > 0.0f) frexpf(amax, &ex);  // amax in [2^(ex-1), 2^ex)
    const float E = amax > 0.0f ? ldexpf(1.0f, 15 - ex) : 1.0f;
    const float sqv = amax > 0.0f ? ldexpf(1.0f, 9 + ex) : 1.0f;  // 2^24 / E
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      uint32_t hw[8], lw[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {  // k-slot e: channel 32g + 8hi + (e>>1) + 4(e&1), field e>>1
        const int f = e >> 1;
        const float v = qv[g][f + 4 * (e & 1)] * ldexpf(E, -2 * f);
        const __half h = __float2half_rn(v);
        hw[e] = __half_as_ushort(h);
        lw[e] = __half_as_ushort(__float2half_rn(v - __half2float(h)));
        if (RPH == 2 && (lo & 1)) hw[e] = lw[e];  // the lo-half row of the head
      }
      st.aq[g][0] = u4{hw[0] | (hw[1] << 16), hw[2] | (hw[3] << 16), hw[4] | (hw[5] << 16), hw[6] | (hw[7] << 16)};
      if (RPH == 1)
        st.aq[g][RPH == 1 ? 1 : 0] =
            u4{lw[0] | (lw[1] << 16), lw[2] | (lw[3] << 16), lw[4] | (lw[5] << 16), lw[6] | (lw[7] << 16)};
    }
    // zero-point MFMA operand: the sum of q~ over group hi (slice sums over the k-groups)
    float ps[4];
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      float t = 0.0f;
#pragma unroll
      for (int e = 0; e < 8; ++e) t += qv[g][e];
      ps[g] = rows_sum(t);
    }
    float gsum;
    if (NG == 4) gsum = hi == 0 ? ps[0] : hi == 1 ? ps[1] : hi == 2 ? ps[2] : ps[3];
    else if (NG == 2) gsum = hi == 0 ? ps[0] + ps[1] : hi == 1 ? ps[2] + ps[3] : 0.0f;
    else gsum = hi == 0 ? (ps[0] + ps[1]) + (ps[2] + ps[3]) : 0.0f;
    st.az = RPH == 2 && (lo & 1) ? 0.0f : gsum * E * (1.0f / 16777216.0f);  // one row per head
    float* sqh = reinterpret_cast<float*>(L.page);  // the page is staged after this
    sqh[hq] = sqv;  // lanes of equal hq write equal values
    lane_exchange();
#pragma unroll
    for (int j = 0; j < HPL; ++j) {
      st.sq[j] = sqh[j < NJ ? WideRows<NCH>::lane_head(hi, j) : 0];
      st.m[j] = -INFINITY;
      st.lsum[j] = 0.0f;
    }
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      st.zacc[c] = 0.0f;
#pragma unroll
      for (int k = 0; k < 8; ++k) st.of[c][k] = 0.0f;
    }
  }

  walk_pages<MIXED, NG>(L.page, pages, Hkv, block_table, max_pages, b, R, kvh, p0, p1, done0, total,
                        [&](auto full, int t0, int t1) {
                          compute_page_wide<decltype(full)::value, BF, NG, NCH>(st, L, t0, t1, lo, hi);
                        });

  // ---- the piece's partial state: (m, l) of heads lane_head(hi, j) ----
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const float ltot = row16_sum(st.lsum[j]);
    const int hh = WideRows<NCH>::lane_head(hi, j);
    if (hh < g_heads && lo == 0) {
      const size_t row = ((size_t)b * Hq + kvh * g_heads + hh) * stride + piece;
      part_ml[row * 2] = st.m[j];
      part_ml[row * 2 + 1] = ltot;
      if (last)  // the range's last piece: the remaining slots hold nothing
        for (int s2 = piece + 1; s2 < num_splits; ++s2) {
          part_ml[(row + s2 - piece) * 2] = -INFINITY;
          part_ml[(row + s2 - piece) * 2 + 1] = 0.0f;
        }
    }
  }
  // ---- o~ of head 4c + hi per chunk (sum w z_v per (head, group) through LDS) ----
  float* zx = reinterpret_cast<float*>(L.page);  // the last page is done
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    float ztot = rows_sum(st.zacc[c]);  // (head 4c + (lo>>2), group lo&3)
    if (NG == 1) ztot = quad_sum(ztot);
    if (NG == 2) ztot += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(ztot), 0x4E, 0xF, 0xF, false));
    zx[16 * c + lo] = ztot;  // lanes of equal lo write equal values
  }
  lane_exchange();
  const bool empty = p0 >= p1;
  const float cs = lo >= 8 ? 0.25f : 1.0f;  // P.V columns lo >= 8 accumulate 4 x code
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    const float4 zh = *reinterpret_cast<const float4*>(&zx[16 * c + 4 * hi]);
    const int hout = 4 * c + hi;
    if (hout >= g_heads) continue;  // padding head
    const size_t row = ((size_t)b * Hq + kvh * g_heads + hout) * stride + piece;
#pragma unroll
    for (int G = 0; G < 4; ++G) {
#pragma unroll
      for (int F = 0; F < 2; ++F) {
        const int ch = 32 * G + 4 * (lo & 7) + 2 * F + (lo >> 3);
        part_o[row * kD + ch] = empty ? 0.0f : fmaf(st.of[c][2 * G + F], cs, -compf(zh, G * NG / 4));
      }
    }
  }
}

// LDS of a split wave: one chunk of 4 heads, or the wide layout.
template <int NCH>
using SplitLds = typename std::conditional<NCH == 1, WaveLds<1>, WideLds<NCH>>::type;

// Balanced split (persistent waves over equal page ranges).  The sequences'
// pages are laid end to end, T pages in total; range r covers pages
// [r*pw, (r+1)*pw) with pw = max(ceil(T / n_ranges), ceil(max_pages / (S - 1)),
// kMinRange), so every wave reads the same number of pages and a sequence is cut
// into at most S pieces (piece = r - first range of the sequence).  Each range
// runs one wave per kv-head, which handles all NCH chunks of 4 query heads of
// that kv-head, so every page-head block is read by exactly one wave; the waves
// of a range read the blocks of the same pages at the same time (each page's Hkv
// blocks are contiguous).  With S = 1 each range is one whole sequence.  With
// MIXED a sequence's pages are those of its INT2 history only, and a row's slots
// are row_stride apart (the slots after the S history slots belong to other
// kernels).  Grid: n_ranges * Hkv one-wave workgroups, workgroup u = (range u /
// Hkv, kv-head u % Hkv).  Waves per SIMD: 4 for one chunk (128 VGPRs), 2 for the
// wide instances (their query operands, chunk states and prefetched page; at 3
// waves the prefetched page spills to scratch).
constexpr int kMinRange = 4;
template <int NCH>
struct SplitWaves {
  static constexpr int per_simd = NCH == 1 ? 4 : 2;
};

__device__ inline int wave_sum_i(int x) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) x += __shfl_xor(x, m, 64);
  return x;
}

template <bool MIXED, bool BF, int NG, int NCH>
__global__ __launch_bounds__(64) __attribute__((
    amdgpu_waves_per_eu(SplitWaves<NCH>::per_simd, SplitWaves<NCH>::per_simd))) void split_mfma_kernel(
    const uint8_t* __restrict__ pages, int Hkv, int Hq, const int32_t* __restrict__ block_table,
    int max_pages, const int32_t* __restrict__ seq_lens, int num_splits, int n_ranges, int B,
    const float* __restrict__ qt, float* __restrict__ part_o, float* __restrict__ part_ml,
    int S0, int W, int row_stride) {
  __shared__ SplitLds<NCH> L;
  const int64_t u = blockIdx.x;
  if (u >= (int64_t)n_ranges * Hkv) return;
  const int r = (int)(u / Hkv), kvh = (int)(u % Hkv);
  const int l = threadIdx.x;
  const int stride = MIXED ? row_stride : num_splits;
  // The INT2 tokens of sequence bb: all of them, or with MIXED the history
  // [lo, hi), lo = min(S0, n), hi = max(lo, n - W) (the bf16 sink and recent
  // window are handled elsewhere).  Lengths beyond the block table are clamped.
  auto range_of = [&](int bb) {
    const int len = min(max(seq_lens[bb], 0), max_pages * kP);
    if (!MIXED) return tok_range(0, len);
    const int lo = min(S0, len);
    return tok_range(lo, max(lo, len - W));
  };
  auto run_piece = [&](int bb, TokRange R, int p0, int p1, int piece, bool last, int done0, int total) {
    if constexpr (NCH == 1)
      process_piece<MIXED, BF, NG, NCH>(L, pages, Hkv, Hq, block_table, max_pages, bb, R, kvh, p0, p1, piece,
                                        last, num_splits, stride, qt, part_o, part_ml, done0, total);
    else
      process_piece_wide<MIXED, BF, NG, NCH>(L, pages, Hkv, Hq, block_table, max_pages, bb, R, kvh, p0, p1,
                                             piece, last, num_splits, stride, qt, part_o, part_ml, done0,
                                             total);
  };
  if (num_splits == 1) {  // one range per sequence
    const TokRange R = range_of(r);
    run_piece(r, R, 0, R.npg, 0, true, 0, 1 << 20);
    return;
  }
  // total pages over all sequences
  int64_t T = 0;
  for (int b0 = 0; b0 < B; b0 += 64) {
    const int bb = b0 + l;
    T += __builtin_amdgcn_readfirstlane(wave_sum_i(bb < B ? range_of(bb).npg : 0));
  }
  const int64_t pw = max(max((T + n_ranges - 1) / n_ranges,
                             (int64_t)((max_pages + num_splits - 2) / (num_splits - 1))),
                         (int64_t)kMinRange);
  int64_t x = (int64_t)r * pw;
  const int64_t xe = min(T, x + pw);
  // a sequence with no pages gets empty slots from the (range b mod n_ranges,
  // kv-head 0, chunk 0) wave, for all its heads
  if (kvh == 0)
    for (int bb = r; bb < B; bb += n_ranges)
      if (range_of(bb).npg == 0)
        for (int i = l; i < Hq * num_splits; i += 64) {
          const size_t row = ((size_t)bb * Hq + i / num_splits) * stride + i % num_splits;
          part_ml[row * 2] = -INFINITY;
          part_ml[row * 2 + 1] = 0.0f;
        }
  if (x >= xe) return;
  // the sequence holding page x: pages before sequence b, scanned 64 sequences at a time
  int b = 0, npg_b = 0;
  int64_t before = 0;
  for (int b0 = 0; b0 < B; b0 += 64) {
    const int bb = b0 + l;
    const int np = bb < B ? range_of(bb).npg : 0;
    int incl = np;  // inclusive prefix sum over the lanes
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const int y = __shfl_up(incl, off, 64);
      if (l >= off) incl += y;
    }
    const uint64_t hit =
        __ballot(bb < B && np > 0 && before + (incl - np) <= x && x < before + incl);
    if (hit) {
      const int lane = __ffsll((unsigned long long)hit) - 1;
      b = b0 + lane;
      npg_b = __builtin_amdgcn_readlane(np, lane);
      before += __builtin_amdgcn_readlane(incl - np, lane);
      break;
    }
    before += __builtin_amdgcn_readlane(incl, 63);
  }
  if (npg_b == 0) return;  // not reached: page x < T lies in some sequence
  const int64_t x0 = x;
  __builtin_amdgcn_s_setprio(3);  // lowered in bands as the wave's pages are done
  while (true) {
    const int64_t end = min(xe, before + npg_b);
    const int piece = (int)(r - before / pw);
    run_piece(b, range_of(b), (int)(x - before), (int)(end - before), piece, end == before + npg_b,
              (int)(x - x0), (int)(xe - x0));
    x = end;
    if (x >= xe) break;
    before += npg_b;
    do {  // next sequence with pages
      if (++b >= B) return;  // not reached: pages remain before xe <= T
      npg_b = range_of(b).npg;
    } while (npg_b == 0);
  }
}

// The launches of the NCH-chunk instances for the given quantizer format.
template <int NCH>
void launch_split_nch(const SplitLaunch& a, bool mixed, int meta_bf16, int ng) {
  auto go = [&](auto kernel) {
    hipLaunchKernelGGL(kernel, dim3((unsigned)a.blocks), dim3(64), 0, a.stream, a.pages, a.Hkv, a.Hq,
                       a.block_table, a.max_pages, a.seq_lens, a.num_splits, a.ranges, a.B, a.qt,
                       a.part_o, a.part_ml, a.S0, a.W, a.row_stride);
  };
  auto by_ng = [&](auto mixed_c, auto bf_c) {
    constexpr bool M = decltype(mixed_c)::value, BFV = decltype(bf_c)::value;
    if (ng == 4) go(split_mfma_kernel<M, BFV, 4, NCH>);
    else if (ng == 2) go(split_mfma_kernel<M, BFV, 2, NCH>);
    else go(split_mfma_kernel<M, BFV, 1, NCH>);
  };
  using T = std::true_type;
  using F = std::false_type;
  if (mixed) {
    if (meta_bf16) by_ng(T{}, T{});
    else by_ng(T{}, F{});
  } else {
    if (meta_bf16) by_ng(F{}, T{});
    else by_ng(F{}, F{});
  }
}

}  // namespace

#ifdef OSCAR_SPLIT_TWO_CHUNK_UNIT
void launch_split_two_chunk(const SplitLaunch& a, bool mixed, int meta_bf16, int ng) {
  launch_split_nch<2>(a, mixed, meta_bf16, ng);
}
#else
hipError_t launch_decode_split_mfma(const uint8_t* pages, int Hkv, int B, int Hq,
                                    const int32_t* block_table, int max_pages,
                                    const int32_t* seq_lens, int num_splits, int cus,
                                    const float* qt, float* part_o, float* part_ml,
                                    hipStream_t st, int meta_bf16, int ng,
                                    const MixedSpec* mixed) {
  const int nch = split_chunks(Hq / Hkv);
  // one range per resident group of Hkv waves
  const int64_t ranges =
      num_splits == 1 ? (int64_t)B
                      : std::max<int64_t>(1, (int64_t)split_waves_per_cu(nch) * cus / Hkv);
  const int64_t blocks = ranges * Hkv;
  if (blocks > 0x7fffffffLL) return hipErrorInvalidConfiguration;
  SplitLaunch a;
  a.pages = pages;
  a.Hkv = Hkv;
  a.Hq = Hq;
  a.block_table = block_table;
  a.max_pages = max_pages;
  a.seq_lens = seq_lens;
  a.num_splits = num_splits;
  a.ranges = (int)ranges;
  a.B = B;
  a.qt = qt;
  a.part_o = part_o;
  a.part_ml = part_ml;
  a.S0 = mixed ? mixed->S0 : 0;
  a.W = mixed ? mixed->W : 0;
  a.row_stride = mixed ? mixed->row_stride : num_splits;
  a.blocks = blocks;
  a.stream = st;
  const bool mx = mixed != nullptr;
  if (nch == 1) launch_split_nch<1>(a, mx, meta_bf16, ng);
  else if (nch == 2) launch_split_two_chunk(a, mx, meta_bf16, ng);
  else if (nch == 3) launch_split_nch<3>(a, mx, meta_bf16, ng);
  else launch_split_nch<4>(a, mx, meta_bf16, ng);
  return hipGetLastError();
}
#endif

}  // namespace oscar
