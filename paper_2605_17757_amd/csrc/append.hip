// Cache update: rotate -> clip -> asymmetric INT2 per 32-channel group -> pack.
// (Sec. 4 "KV Cache Update"; App. "Scale Determination and Per-token Clipping
// Details"; Alg. 1 QuantizeAndWrite.)
//
// This file is compiled with -ffp-contract=off: every fp32 step below is one
// IEEE operation (no fused multiply-add), and the rotation is an explicit fp64
// fused multiply-add chain in ascending channel order.  Because each product of
// a bf16 input and an fp32 matrix entry is exact in fp64, that chain equals
// "sum in fp64, ascending, round once to fp32" bit for bit.
//
// Work decomposition: blockIdx.y selects K (0) or V (1); the block stages that
// rotation matrix (64 KB fp32) in LDS once and its waves then take rows (token,
// head), grid-stride.  Lane l computes output channels l and l+64 of the rows.
// A 32-channel group is one half of the wave: channels 0-31 / 64-95 live in lanes
// 0-31, channels 32-63 / 96-127 in lanes 32-63; the group max / min are DPP steps
// inside each row of 16 lanes plus one row-pair swap.  Small appends (a decode
// step) run one row per wave on many short waves; large ones run the bulk kernel
// below (8 rows per wave, persistent blocks).
#include <hip/hip_fp16.h>

#include <algorithm>

#include "internal.h"

namespace oscar {
namespace {

constexpr int kWaves = 4;
constexpr int kMaxClipCands = 32;  // candidate clip ratios per calibration call

__device__ inline float f16_bits_to_f32(uint16_t h) { return __half2float(__ushort_as_half(h)); }

// binary16 with saturation to +-65504 (round to nearest even).
__device__ inline uint16_t f16_sat_bits(float f) {
  f = fminf(fmaxf(f, -65504.0f), 65504.0f);
  return __half_as_ushort(__float2half_rn(f));
}

// A zero point of zero is stored as +0.  This is done on the binary16 bits: the
// compiler may drop an "x + 0.0f" whose result only feeds fmaxf/fminf.
__device__ inline uint16_t plus_zero(uint16_t h) { return (h & 0x7fffu) ? h : (uint16_t)0; }

// max / min over the 32 lanes of a half wave: quad swaps and row rotations by 4
// and 8 (DPP) reduce each row of 16 lanes, the row-pair swap joins rows 2k, 2k+1.
template <bool MAX>
__device__ inline float half_wave_reduce(float x) {
  auto op = [](float a, float b) { return MAX ? fmaxf(a, b) : fminf(a, b); };
  x = op(x, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0xB1, 0xF, 0xF, false)));
  x = op(x, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x4E, 0xF, 0xF, false)));
  x = op(x, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x124, 0xF, 0xF, false)));
  x = op(x, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x128, 0xF, 0xF, false)));
  const uint32_t u = __float_as_uint(x);
  const auto sw = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  return op(__uint_as_float(sw[0]), __uint_as_float(sw[1]));
}
__device__ inline float half_wave_max(float x) { return half_wave_reduce<true>(x); }
__device__ inline float half_wave_min(float x) { return half_wave_reduce<false>(x); }

// bfloat16 with saturation to +-(largest finite) (round to nearest even on the
// binary32 bits; finite inputs).
__device__ inline uint16_t bf16_sat_bits(float f) {
  const uint32_t u = __float_as_uint(f);
  uint16_t h = (uint16_t)((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
  if ((h & 0x7fffu) == 0x7f80u) h = (uint16_t)((h & 0x8000u) | 0x7f7fu);
  return h;
}

using QFmt = QuantFmt;  // storage format of scale and zero, and the clip rule
__device__ inline uint16_t meta_store(const QFmt& q, float f) {
  return q.bf16 ? bf16_sat_bits(f) : f16_sat_bits(f);
}
__device__ inline float meta_load(const QFmt& q, uint16_t h) {
  return q.bf16 ? __uint_as_float((uint32_t)h << 16) : f16_bits_to_f32(h);
}

struct QOut {
  uint32_t code;
  uint16_t s16, z16;
};

// Scale and zero point of a group with (clipped) minimum a and maximum b, as
// stored (s16, z16) and as used for the codes (sf, zf); a group whose stored
// scale is 0 stores s = 1, z = M(-a) and codes 0 (deg).
struct QParams {
  uint16_t s16, z16;
  float sf, zf;
  bool deg;
};
__device__ inline QParams quant_params(float a, float b, const QFmt& fmt) {
  QParams p;
  const float s = __fdiv_rn(__fsub_rn(b, a), 3.0f);
  p.s16 = meta_store(fmt, s);
  p.deg = (p.s16 & 0x7fffu) == 0;
  if (p.deg) {
    p.s16 = fmt.bf16 ? 0x3f80u : 0x3c00u;  // 1.0
    p.z16 = plus_zero(meta_store(fmt, -a));
    p.sf = p.zf = 0.0f;
  } else {
    p.sf = meta_load(fmt, p.s16);
    p.z16 = plus_zero(meta_store(fmt, __fdiv_rn(-a, p.sf)));
    p.zf = meta_load(fmt, p.z16);
  }
  return p;
}
// Code of one clipped channel value y: clamp(round_half_even(y / s + z), 0, 3).
__device__ inline uint32_t quant_code(float y, const QParams& p) {
  if (p.deg) return 0u;
  const float r = rintf(__fadd_rn(__fdiv_rn(y, p.sf), p.zf));
  return (uint32_t)fminf(fmaxf(r, 0.0f), 3.0f);
}

// Quantize one clipped channel value y of a group with minimum a and maximum b.
__device__ inline QOut quantize(float y, float a, float b, const QFmt& fmt) {
  const QParams p = quant_params(a, b, fmt);
  QOut o;
  o.s16 = p.s16;
  o.z16 = p.z16;
  o.code = quant_code(y, p);
  return o;
}

// Token-wise clip threshold (App. "Scale Determination and Per-token Clipping
// Details"): the rho-quantile of |x~| over the row, a_k + f (a_{k+1} - a_k) with
// pos = rho (d - 1), k = floor(pos), f = pos - k, in fp32 steps.  The order
// statistics come from a binary search over the bit patterns of |x~| (positive
// floats order like their bits): the smallest T with #{|x~| <= T} >= k + 1 is a_k.
__device__ inline void quantile_pos(float rho, int& k, float& f) {
  const float pos = __fmul_rn(rho, (float)(kD - 1));
  k = min((int)floorf(pos), kD - 1);
  f = __fsub_rn(pos, (float)k);
}
__device__ inline float lerp_tau(float ak, float ak1, float f) {
  return __fadd_rn(ak, __fmul_rn(f, __fsub_rn(ak1, ak)));
}

// One row over the wave: lane l holds channels l and l + 64.
__device__ inline float token_quantile_wave(float x0, float x1, float rho) {
  const uint32_t u0 = __float_as_uint(x0) & 0x7fffffffu, u1 = __float_as_uint(x1) & 0x7fffffffu;
  int k;
  float f;
  quantile_pos(rho, k, f);
  auto count_le = [&](uint32_t t) {  // wave-uniform
    return __popcll(__ballot(u0 <= t)) + __popcll(__ballot(u1 <= t));
  };
  uint32_t lo = 0, hi = 0x7f800000u;
  while (lo < hi) {
    const uint32_t mid = lo + ((hi - lo) >> 1);
    if (count_le(mid) >= k + 1) hi = mid;
    else lo = mid + 1;
  }
  const float ak = __uint_as_float(lo);
  if (k >= kD - 1) return ak;
  float ak1 = ak;
  if (count_le(lo) < k + 2) {  // a_{k+1} = the smallest value above a_k
    uint32_t m = min(u0 > lo ? u0 : 0xffffffffu, u1 > lo ? u1 : 0xffffffffu);
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) m = min(m, (uint32_t)__shfl_xor((int)m, o, 64));
    ak1 = __uint_as_float(m);
  }
  return lerp_tau(ak, ak1, f);
}

// Two rows, one per wave half: lane l' = l & 31 of half h holds channels
// l' + 32 q of row h.  Both searches run together (31 halvings of the bit range).
__device__ inline float token_quantile_halves(const float (&x)[4], float rho, int half) {
  uint32_t u[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) u[q] = __float_as_uint(x[q]) & 0x7fffffffu;
  int k;
  float f;
  quantile_pos(rho, k, f);
  // counts of the two halves for per-half thresholds t0 (half 0) and t1 (half 1)
  auto counts = [&](uint32_t t0, uint32_t t1, int& c0, int& c1) {
    const uint32_t t = half ? t1 : t0;
    c0 = c1 = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint64_t b = __ballot(u[q] <= t);
      c0 += __popc((uint32_t)b);
      c1 += __popc((uint32_t)(b >> 32));
    }
  };
  uint32_t lo0 = 0, hi0 = 0x7f800000u, lo1 = 0, hi1 = 0x7f800000u;
  for (int it = 0; it < 31; ++it) {
    const uint32_t m0 = lo0 + ((hi0 - lo0) >> 1), m1 = lo1 + ((hi1 - lo1) >> 1);
    int c0, c1;
    counts(m0, m1, c0, c1);
    if (c0 >= k + 1) hi0 = m0; else lo0 = m0 + 1;
    if (c1 >= k + 1) hi1 = m1; else lo1 = m1 + 1;
  }
  const uint32_t lo = half ? lo1 : lo0;
  const float ak = __uint_as_float(lo);
  if (k >= kD - 1) return ak;
  int c0, c1;
  counts(lo0, lo1, c0, c1);
  uint32_t m = 0xffffffffu;
#pragma unroll
  for (int q = 0; q < 4; ++q) m = min(m, u[q] > lo ? u[q] : 0xffffffffu);
#pragma unroll
  for (int o = 16; o >= 1; o >>= 1) m = min(m, (uint32_t)__shfl_xor((int)m, o, 64));  // within the half
  const float ak1 = ((half ? c1 : c0) >= k + 2) ? ak : __uint_as_float(m);
  return lerp_tau(ak, ak1, f);
}

// OR the 2-bit codes of lanes 4j..4j+3 into the byte of quad j (valid in lane 4j).
__device__ inline uint32_t pack_quad(uint32_t code, int lane) {
  uint32_t v = code << (2 * (lane & 3));
  v |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xF, 0xF, false);  // lane ^ 1
  v |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xF, 0xF, false);  // lane ^ 2
  return v;
}

__device__ inline float bf16_to_f32(uint16_t h) { return __uint_as_float(((uint32_t)h) << 16); }

// ---------------------------------------------------------------------------
// prepare: q~ = q R_k (times the logit scale) on the fp32 matrix cores, 16 query
// rows per block.  Wave w computes column tiles 2w and 2w + 1 (16 channels each)
// of the block's rows as 32 chained 16x16x4 MFMAs per tile: step s takes channels
// c = 32k + s in k-slot k, so lane (row lo, k-slot hi) holds q[row][32hi + s] (one
// 64-byte run of the row) and lane (column lo, k-slot hi) R_k[32hi + s][16t + lo]
// (16 lanes read 64 contiguous bytes of a row of R_k).  R_k is read straight from
// L2 (no LDS copy, no barrier); all loads of a wave are issued before its MFMAs.
// D lane (column lo, hi): rows 4hi + i.
// ---------------------------------------------------------------------------
constexpr int kPrepRows = 16;

typedef float prep_f4 __attribute__((ext_vector_type(4)));

__device__ inline void prepare_body(int bx, const uint16_t* __restrict__ q, int rows,
                                    const float* __restrict__ Rk, float qscale,
                                    float* __restrict__ qt, int rph, int Hq, int Hkv) {
  const int t = threadIdx.x, w = t >> 6, lo = t & 15, hi = (t >> 4) & 3;
  int kvh;
  query_row(bx, 0, kPrepRows, rows, Hq, Hkv, rph, kvh);
  if (Rk && rph) Rk += (size_t)kvh * kD * kD;  // the block's rows share a KV head
  int kv_;
  const int arow = query_row(bx, lo, kPrepRows, rows, Hq, Hkv, rph, kv_);
  if (!Rk) {  // R = I (bf16 baseline): a scaled copy, rows 4w + (0..3), lane: 2 channels
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = query_row(bx, 4 * w + i, kPrepRows, rows, Hq, Hkv, rph, kv_);
      if (row < 0) continue;
      const int c = 2 * (t & 63);
      const uint32_t v = *reinterpret_cast<const uint32_t*>(q + (size_t)row * kD + c);
      qt[(size_t)row * kD + c] = bf16_to_f32((uint16_t)(v & 0xffffu)) * qscale;
      qt[(size_t)row * kD + c + 1] = bf16_to_f32((uint16_t)(v >> 16)) * qscale;
    }
    return;
  }
  float a[32];
  if (arow >= 0) {
    const uint4* src = reinterpret_cast<const uint4*>(q + (size_t)arow * kD + 32 * hi);
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const uint4 v = src[k];
      const uint32_t u[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        a[8 * k + 2 * e] = bf16_to_f32((uint16_t)(u[e] & 0xffffu));
        a[8 * k + 2 * e + 1] = bf16_to_f32((uint16_t)(u[e] >> 16));
      }
    }
  } else {
#pragma unroll
    for (int s = 0; s < 32; ++s) a[s] = 0.0f;
  }
  float b[2][32];
#pragma unroll
  for (int tt = 0; tt < 2; ++tt)
#pragma unroll
    for (int s = 0; s < 32; ++s) b[tt][s] = Rk[(size_t)(32 * hi + s) * kD + 16 * (2 * w + tt) + lo];
#pragma unroll
  for (int tt = 0; tt < 2; ++tt) {
    prep_f4 d = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int s = 0; s < 32; ++s) d = __builtin_amdgcn_mfma_f32_16x16x4f32(a[s], b[tt][s], d, 0, 0, 0);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = query_row(bx, 4 * hi + i, kPrepRows, rows, Hq, Hkv, rph, kv_);
      if (row >= 0) qt[(size_t)row * kD + 16 * (2 * w + tt) + lo] = d[i] * qscale;
    }
  }
}

// ---------------------------------------------------------------------------
// Row routing.  A cache-update kernel takes rows (token, kv-head) = row; for each
// row and tensor (is_v) a policy names
//   src(row, is_v)  : the bf16 row to rotate and quantize (nullptr: none),
//   slot(row)       : the pool slot that receives it (< 0: none),
//   copy(row, is_v, l) : bf16 rows to copy into the mixed cache's segment store,
//                     done by lane l for its 4 bytes after src has been read.
// ---------------------------------------------------------------------------
struct PlainRows {  // oscar_kv_append: token i -> slot_mapping[i]
  const uint16_t* k;
  const uint16_t* v;
  const int64_t* slots;
  int n_rows, Hkv;
  __device__ const uint16_t* src(int row, int is_v) const {
    return row < n_rows ? (is_v ? v : k) + (size_t)row * kD : nullptr;
  }
  __device__ int64_t slot(int row) const { return row < n_rows ? slots[row / Hkv] : -1; }
  __device__ void copy(int, int, int) const {}
  // the row's bf16 input (whatever its destination), and its bf16 copy destination
  __device__ const uint16_t* data(int row, int is_v) const { return src(row, is_v); }
  __device__ uint32_t* seg_dst(int, int) const { return nullptr; }
};

// Segment store of the mixed cache: [B][Hkv][K, V][S0 + W][d] bf16; position p
// of a sequence has segment slot p (p < S0) or S0 + (p - S0) mod W (window).
__device__ inline uint32_t* seg_row(uint16_t* seg, int Hkv, int S0, int W, int b, int h,
                                    int is_v, int slot) {
  return reinterpret_cast<uint32_t*>(
      seg + ((((size_t)b * Hkv + h) * 2 + is_v) * (size_t)(S0 + W) + slot) * kD);
}
__device__ inline int seg_slot(int S0, int W, int p) { return p < S0 ? p : S0 + (p - S0) % W; }

// oscar_mixed_append: token i of sequence seq_idx[i] at position pos[i] goes
// where a cache of length seq_lens[b] keeps it: INT2 for the history [lo, hi)
// (pool slot from the block table), bf16 segment slot otherwise; positions
// outside [0, seq_lens[b]) are skipped.
struct PrefillRows {
  const uint16_t* k;
  const uint16_t* v;
  uint16_t* seg;
  const int32_t* seq_idx;
  const int64_t* pos;
  const int32_t* seq_lens;
  const int32_t* block_table;
  int n_rows, Hkv, max_pages, S0, W;
  // -1: skipped, 0: INT2, 1: bf16; b and p of the row's token
  __device__ int route(int row, int& b, int& p) const {
    if (row >= n_rows) return -1;
    const int tok = row / Hkv;
    b = seq_idx[tok];
    const int64_t p64 = pos[tok];
    const int len = min(max(seq_lens[b], 0), max_pages * kP);
    if (p64 < 0 || p64 >= len) return -1;
    p = (int)p64;
    const int lo = min(S0, len), hi = max(lo, len - W);
    return (p >= lo && p < hi) ? 0 : 1;
  }
  __device__ const uint16_t* src(int row, int is_v) const {
    int b, p;
    return route(row, b, p) == 0 ? (is_v ? v : k) + (size_t)row * kD : nullptr;
  }
  __device__ int64_t slot(int row) const {
    int b, p;
    if (route(row, b, p) != 0) return -1;
    return (int64_t)block_table[(size_t)b * max_pages + p / kP] * kP + p % kP;
  }
  __device__ void copy(int row, int is_v, int l) const {
    int b, p;
    if (route(row, b, p) != 1) return;
    const int h = row % Hkv;
    seg_row(seg, Hkv, S0, W, b, h, is_v, seg_slot(S0, W, p))[l] =
        reinterpret_cast<const uint32_t*>((is_v ? v : k) + (size_t)row * kD)[l];
  }
  __device__ const uint16_t* data(int row, int is_v) const {
    return row < n_rows ? (is_v ? v : k) + (size_t)row * kD : nullptr;
  }
  __device__ uint32_t* seg_dst(int row, int is_v) const {
    int b, p;
    if (route(row, b, p) != 1) return nullptr;
    return seg_row(seg, Hkv, S0, W, b, row % Hkv, is_v, seg_slot(S0, W, p));
  }
};

// Decode step over the mixed cache: one new token per sequence b (row =
// b * Hkv + h) at position p = seq_lens[b] - 1 (Alg. 1 DecodeStep):
//   p < S0          -> bf16 sink slot p;
//   p >= S0, W = 0  -> INT2 at position p;
//   otherwise       -> bf16 window slot of p; when p - W >= S0 the token at
//                      p - W, which holds that slot, is first quantized into
//                      INT2 at position p - W (read before the slot is reused).
struct StepRows {
  const uint16_t* k;
  const uint16_t* v;
  uint16_t* seg;
  const int32_t* seq_lens;
  const int32_t* block_table;
  int n_rows, Hkv, max_pages, S0, W;
  __device__ int pos(int row) const {  // -1: no token
    return row < n_rows ? min(max(seq_lens[row / Hkv], 0), max_pages * kP) - 1 : -1;
  }
  // position quantized into INT2 by this step, or -1
  __device__ int qpos(int p) const {
    if (p < S0) return -1;
    if (W == 0) return p;
    return p - W >= S0 ? p - W : -1;
  }
  __device__ const uint16_t* src(int row, int is_v) const {
    const int p = pos(row), qp = qpos(p);
    if (qp < 0) return nullptr;
    if (qp == p) return (is_v ? v : k) + (size_t)row * kD;
    const int b = row / Hkv, h = row % Hkv;
    return reinterpret_cast<const uint16_t*>(seg_row(seg, Hkv, S0, W, b, h, is_v, seg_slot(S0, W, qp)));
  }
  __device__ int64_t slot(int row) const {
    const int qp = qpos(pos(row));
    if (qp < 0) return -1;
    return (int64_t)block_table[(size_t)(row / Hkv) * max_pages + qp / kP] * kP + qp % kP;
  }
  __device__ void copy(int row, int is_v, int l) const {
    const int p = pos(row);
    if (p < 0 || (p >= S0 && W == 0)) return;
    const int b = row / Hkv, h = row % Hkv;
    // same lane and address as the read of a demoted row: ordered after it
    seg_row(seg, Hkv, S0, W, b, h, is_v, seg_slot(S0, W, p))[l] =
        reinterpret_cast<const uint32_t*>((is_v ? v : k) + (size_t)row * kD)[l];
  }
};

// Clip, quantize, pack and write one rotated row (token, head) whose channels l
// and l + 64 are in lane l, to pool slot `slot` (wave-uniform; < 0: the row only
// takes part in the cross-lane steps).
// Group reductions of the one-row-per-wave layout (lane l: channels l, l + 64):
// with 32-channel groups each value's group is a wave half, with 64 its whole
// wave, with 128 both values over the wave.
__device__ inline float wave_max(float x) {
  x = half_wave_max(x);
  const uint32_t u = __float_as_uint(x);
  const auto sw = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1]));
}
__device__ inline float wave_min(float x) {
  x = half_wave_min(x);
  const uint32_t u = __float_as_uint(x);
  const auto sw = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return fminf(__uint_as_float(sw[0]), __uint_as_float(sw[1]));
}
template <bool MAX>
__device__ inline void group_reduce2(float v0, float v1, int ng, float& r0, float& r1) {
  auto op = [](float a, float b) { return MAX ? fmaxf(a, b) : fminf(a, b); };
  auto half = [](float x) { return MAX ? half_wave_max(x) : half_wave_min(x); };
  auto wave = [](float x) { return MAX ? wave_max(x) : wave_min(x); };
  if (ng == 4) {
    r0 = half(v0);
    r1 = half(v1);
  } else if (ng == 2) {
    r0 = wave(v0);
    r1 = wave(v1);
  } else {
    r0 = r1 = wave(op(v0, v1));
  }
}

__device__ inline void store_row(uint8_t* __restrict__ pages, int Hkv, int64_t slot, int row,
                                 int is_v, float clip, const QFmt& fmt, double acc0, double acc1,
                                 int l) {
  const float xt0 = __double2float_rn(acc0);  // channel l
  const float xt1 = __double2float_rn(acc1);  // channel l + 64
  float tau0, tau1;
  if (fmt.quantile) {
    tau0 = tau1 = token_quantile_wave(xt0, xt1, clip);
  } else {
    group_reduce2<true>(fabsf(xt0), fabsf(xt1), fmt.ng, tau0, tau1);
    tau0 = __fmul_rn(clip, tau0);
    tau1 = __fmul_rn(clip, tau1);
  }
  const float y0 = fminf(fmaxf(xt0, -tau0), tau0), y1 = fminf(fmaxf(xt1, -tau1), tau1);
  float a0, a1, b0, b1;
  group_reduce2<false>(y0, y1, fmt.ng, a0, a1);
  group_reduce2<true>(y0, y1, fmt.ng, b0, b1);
  const QOut q0 = quantize(y0, a0, b0, fmt);
  const QOut q1 = quantize(y1, a1, b1, fmt);
  const uint32_t byte0 = pack_quad(q0.code, l);  // quad l/4
  const uint32_t byte1 = pack_quad(q1.code, l);  // quad 16 + l/4
  if (slot < 0) return;                          // uniform across the wave
  const int h = row % Hkv;
  const int64_t page = slot / kP;
  const int t = (int)(slot - page * kP);
  uint8_t* blk = pages + ((size_t)page * Hkv + h) * block_bytes(fmt.ng);
  if ((l & 3) == 0) {
    const int j0 = l >> 2, j1 = 16 + (l >> 2);
    if (is_v) {
      blk[kOffVCodes + j0 * kP + t] = (uint8_t)byte0;
      blk[kOffVCodes + j1 * kP + t] = (uint8_t)byte1;
    } else {
      blk[kOffKCodes + t * (kD / 4) + j0] = (uint8_t)byte0;
      blk[kOffKCodes + t * (kD / 4) + j1] = (uint8_t)byte1;
    }
  }
  // (s, z) of the groups: value 0 of lane l is in group l / 32 (G = 32) or 0,
  // value 1 in group 2 + l / 32 (G = 32), 1 (G = 64) or 0 (G = 128)
  const uint32_t sz_base = is_v ? off_vsz(fmt.ng) : kOffKSz;
  const bool lead = fmt.ng == 4 ? (l & 31) == 0 : l == 0;
  if (lead) {
    const int g0 = fmt.ng == 4 ? l >> 5 : 0;
    const int g1 = fmt.ng == 4 ? 2 + (l >> 5) : fmt.ng == 2 ? 1 : -1;
    *reinterpret_cast<uint32_t*>(blk + sz_base + (g0 * kP + t) * 4) =
        (uint32_t)q0.s16 | ((uint32_t)q0.z16 << 16);
    if (g1 >= 0)
      *reinterpret_cast<uint32_t*>(blk + sz_base + (g1 * kP + t) * 4) =
          (uint32_t)q1.s16 | ((uint32_t)q1.z16 << 16);
  }
}

// Cache update by one block: is_v selects K or V, blocks bx of gx take rows
// grid-stride.  Rs: 64 KB LDS for the matrix, xs: the waves' input rows.
template <int RW, class Rows>
__device__ inline void append_body(float* Rs, double (*xs)[RW][kD], int is_v, int bx, int gx,
                                   uint8_t* __restrict__ pages, int Hkv, const Rows& rows,
                                   int n_rows, const float* __restrict__ Rk,
                                   const float* __restrict__ Rv, float clip_k, float clip_v,
                                   const QFmt& fmt) {
  const float* __restrict__ R = is_v ? Rv : Rk;  // nullptr: identity
  const float clip = is_v ? clip_v : clip_k;
  // rph: the block takes the rows (token, h) of one KV head h, so that it stages
  // that head's matrix; gx is then a multiple of Hkv
  int h = 0;
  if (fmt.rph) {
    h = bx % Hkv;
    bx /= Hkv;
    gx /= Hkv;
    if (R) R += (size_t)h * kD * kD;
  }
  const int n_seq = fmt.rph ? n_rows / Hkv : n_rows;
  auto row_at = [&](int i) { return fmt.rph ? (i < n_seq ? i * Hkv + h : n_rows) : i; };

  if (R) {  // 16 float4 per thread, all loads issued before the stores
    float4 r4[kD * kD / 4 / 256];
#pragma unroll
    for (int i = 0; i < kD * kD / 4 / 256; ++i)
      r4[i] = reinterpret_cast<const float4*>(R)[threadIdx.x + 256 * i];
#pragma unroll
    for (int i = 0; i < kD * kD / 4 / 256; ++i) reinterpret_cast<float4*>(Rs)[threadIdx.x + 256 * i] = r4[i];
  }
  __syncthreads();

  const int w = threadIdx.x >> 6;
  const int l = threadIdx.x & 63;
  const int n_items = (n_seq + RW - 1) / RW;

  // each wave owns xs[w]: no block-level synchronization inside the loop, only
  // fences around the exchange between its lanes
  for (int item = bx * kWaves + w; item < n_items; item += gx * kWaves) {
    lane_exchange();  // the previous item's reads of xs[w] come first
#pragma unroll
    for (int rr = 0; rr < RW; ++rr) {
      const int row = row_at(item * RW + rr);
      double x0 = 0.0, x1 = 0.0;
      const uint16_t* src = rows.src(row, is_v);
      if (src) {
        const uint32_t pair = reinterpret_cast<const uint32_t*>(src)[l];
        x0 = (double)__uint_as_float(pair << 16);
        x1 = (double)__uint_as_float(pair & 0xffff0000u);
      }
      xs[w][rr][2 * l] = x0;
      xs[w][rr][2 * l + 1] = x1;
      rows.copy(row, is_v, l);
    }
    lane_exchange();

    double acc0[RW], acc1[RW];
    if (R) {
#pragma unroll
      for (int rr = 0; rr < RW; ++rr) acc0[rr] = acc1[rr] = 0.0;
#pragma unroll 4
      for (int c = 0; c < kD; ++c) {
        const double r0 = (double)Rs[c * kD + l];
        const double r1 = (double)Rs[c * kD + l + 64];
#pragma unroll
        for (int rr = 0; rr < RW; ++rr) {
          const double xc = xs[w][rr][c];
          acc0[rr] = __fma_rn(xc, r0, acc0[rr]);
          acc1[rr] = __fma_rn(xc, r1, acc1[rr]);
        }
      }
    } else {  // identity: x~ = x
#pragma unroll
      for (int rr = 0; rr < RW; ++rr) {
        acc0[rr] = xs[w][rr][l];
        acc1[rr] = xs[w][rr][l + 64];
      }
    }

#pragma unroll
    for (int rr = 0; rr < RW; ++rr) {
      const int row = row_at(item * RW + rr);
      store_row(pages, Hkv, rows.slot(row), row, is_v, clip, fmt, acc0[rr], acc1[rr], l);
    }
  }
}

// DEF: the default format (binary16 metadata, group-absmax clip, 32-channel
// groups) as compile-time constants, so that its code has no format branches.
__device__ inline QFmt pick(bool def, const QFmt& fmt) { return def ? QFmt{0, 0, 4, 0} : fmt; }

template <int RW, class Rows, bool DEF>
__global__ __launch_bounds__(256) void append_kernel(uint8_t* __restrict__ pages, int Hkv,
                                                     Rows rows, int n_rows,
                                                     const float* __restrict__ Rk,
                                                     const float* __restrict__ Rv, float clip_k,
                                                     float clip_v, QFmt fmt) {
  __shared__ float Rs[kD * kD];
  __shared__ double xs[kWaves][RW][kD];
  append_body<RW>(Rs, xs, blockIdx.y, blockIdx.x, gridDim.x, pages, Hkv, rows, n_rows, Rk, Rv,
                  clip_k, clip_v, pick(DEF, fmt));
}

// Row-pair layout of the bulk cache update: the two halves of a wave hold rows
// 2p and 2p + 1, and lane l' = l & 31 of a half holds channels l' + 32 q
// (q = 0..3), so each group of 32 channels is one half wave as in the per-row
// path.

// store_row for the pair layout: lane l' of the half holds channels l' + 32 q;
// slot is uniform across the half wave.
__device__ inline void store_row4(uint8_t* __restrict__ pages, int Hkv, int64_t slot, int row,
                                  int is_v, float clip, const QFmt& fmt, const double (&acc)[4],
                                  int lp, int half) {
  float xt[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) xt[q] = __double2float_rn(acc[q]);
  // group reductions of the two-rows-per-wave layout (lane l' of a half: channels
  // l' + 32 q of its row): values q of one group over the half
  auto reduce4 = [&](auto op, auto half_red, const float (&v)[4], float (&r)[4]) {
    if (fmt.ng == 4) {
#pragma unroll
      for (int q = 0; q < 4; ++q) r[q] = half_red(v[q]);
    } else if (fmt.ng == 2) {
      r[0] = r[1] = half_red(op(v[0], v[1]));
      r[2] = r[3] = half_red(op(v[2], v[3]));
    } else {
      r[0] = r[1] = r[2] = r[3] = half_red(op(op(v[0], v[1]), op(v[2], v[3])));
    }
  };
  auto fmax_ = [](float a, float b) { return fmaxf(a, b); };
  auto fmin_ = [](float a, float b) { return fminf(a, b); };
  auto hmax = [](float x) { return half_wave_max(x); };
  auto hmin = [](float x) { return half_wave_min(x); };
  float tau[4];
  if (fmt.quantile) {
    const float t = token_quantile_halves(xt, clip, half);
#pragma unroll
    for (int q = 0; q < 4; ++q) tau[q] = t;
  } else {
    float ax[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) ax[q] = fabsf(xt[q]);
    reduce4(fmax_, hmax, ax, tau);
#pragma unroll
    for (int q = 0; q < 4; ++q) tau[q] = __fmul_rn(clip, tau[q]);
  }
  float y[4], ga[4], gb[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) y[q] = fminf(fmaxf(xt[q], -tau[q]), tau[q]);
  reduce4(fmin_, hmin, y, ga);
  reduce4(fmax_, hmax, y, gb);
  QOut qo[4];
  uint32_t byte[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    qo[q] = quantize(y[q], ga[q], gb[q], fmt);  // 32-channel slice q of the row
    byte[q] = pack_quad(qo[q].code, lp);         // quad 8 q + l'/4
  }
  if (slot < 0) return;
  const int h = row % Hkv;
  const int64_t page = slot / kP;
  const int t = (int)(slot - page * kP);
  uint8_t* blk = pages + ((size_t)page * Hkv + h) * block_bytes(fmt.ng);
  if ((lp & 3) == 0) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int j = 8 * q + (lp >> 2);
      if (is_v) blk[kOffVCodes + j * kP + t] = (uint8_t)byte[q];
      else blk[kOffKCodes + t * (kD / 4) + j] = (uint8_t)byte[q];
    }
  }
  if (lp == 0) {  // group g holds the slices q = g (4 / ng) .. (g + 1) (4 / ng) - 1
    const uint32_t sz_base = is_v ? off_vsz(fmt.ng) : kOffKSz;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      if (g >= fmt.ng) break;
      const int q = g * (4 / fmt.ng);
      *reinterpret_cast<uint32_t*>(blk + sz_base + (g * kP + t) * 4) =
          (uint32_t)qo[q].s16 | ((uint32_t)qo[q].z16 << 16);
    }
  }
}

// ---------------------------------------------------------------------------
// Bulk cache update on the fp64 matrix cores (large appends; every format).  A
// wave rotates 16 rows at a time as one 16 x 128 x 128 product of
// v_mfma_f64_16x16x4_f64 steps: step s takes channels 4 s .. 4 s + 3, A = the 16
// rows' bf16 values of those channels (lane l: row l % 16, channel 4 s + l / 16),
// B = rows 4 s .. 4 s + 3 of R (lane l: row 4 s + l / 16), over eight column
// tiles whose column j is channel 8 j + t (tile t).  A step adds its four
// products to the running fp64 sum one after another in channel order (lane
// group l / 16 = position in that order) and the steps run s = 0..31 in turn,
// so each x~ is the fp64 sum of the 128 exact products in ascending channel
// order rounded once to fp32, bit for bit the value of the row-per-lane path.
// Output lane l, register i of tile t holds row l / 16 + 4 i, channel 8 (l % 16)
// + t; the 16 rows go through LDS (fp32) to the layout of the quantizer: lane
// (row, 32-channel slice) for the group-absmax clip (store_slice32), two rows per
// wave (store_row4) for the token-quantile clip.  R is staged once per block
// as fp32 (64 KB) and read as two 16-byte words per lane and step.
// ---------------------------------------------------------------------------
constexpr int kMfmaWaves = 8;
constexpr int kMfmaRows = 16;
constexpr int kStagePitch = 66;   // dwords per staged bf16 row (8-byte reads of 16 rows: all banks)
constexpr int kXtPitch = 132;     // floats per x~ row
constexpr int kAreaWords = kMfmaRows * kXtPitch;  // per wave: staged rows, then x~

typedef double d4v __attribute__((ext_vector_type(4)));

// Clip, quantize and pack the 16 rows of a bulk item under the group-absmax
// clip: lane l takes row l / 4, channels 32 q .. 32 q + 31 (q = l % 4) in x; a
// group of G channels is the G / 32 lanes q of one row with equal q / (G / 32)
// (quad-lane reductions for G = 64, 128).  Same steps and operation order as
// store_row4.
__device__ inline float quad_group_max(float v, int ng) {
  if (ng <= 2) v = fmaxf(v, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xF, 0xF, false)));
  if (ng == 1) v = fmaxf(v, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x4E, 0xF, 0xF, false)));
  return v;
}
__device__ inline float quad_group_min(float v, int ng) {
  if (ng <= 2) v = fminf(v, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xF, 0xF, false)));
  if (ng == 1) v = fminf(v, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x4E, 0xF, 0xF, false)));
  return v;
}

__device__ inline void store_slice32(uint8_t* __restrict__ pages, int Hkv, int64_t slot, int row,
                                     int is_v, float clip, const QFmt& fmt, const float (&x)[32],
                                     int q) {
  float m = 0.0f;
#pragma unroll
  for (int i = 0; i < 32; ++i) m = fmaxf(m, fabsf(x[i]));
  const float tau = __fmul_rn(clip, quad_group_max(m, fmt.ng));
  float y[32];
  float a = INFINITY, b = -INFINITY;
#pragma unroll
  for (int i = 0; i < 32; ++i) {
    y[i] = fminf(fmaxf(x[i], -tau), tau);
    a = fminf(a, y[i]);
    b = fmaxf(b, y[i]);
  }
  a = quad_group_min(a, fmt.ng);
  b = quad_group_max(b, fmt.ng);
  const QParams p = quant_params(a, b, fmt);
  uint32_t w[8];
#pragma unroll
  for (int jb = 0; jb < 8; ++jb) {
    uint32_t byte = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) byte |= quant_code(y[4 * jb + e], p) << (2 * e);
    w[jb] = byte;
  }
  if (slot < 0) return;
  const int h = row % Hkv;
  const int64_t page = slot / kP;
  const int t = (int)(slot - page * kP);
  uint8_t* blk = pages + ((size_t)page * Hkv + h) * block_bytes(fmt.ng);
  if (is_v) {
#pragma unroll
    for (int jb = 0; jb < 8; ++jb) blk[kOffVCodes + (8 * q + jb) * kP + t] = (uint8_t)w[jb];
  } else {
    *reinterpret_cast<uint2*>(blk + kOffKCodes + t * (kD / 4) + 8 * q) =
        make_uint2(w[0] | (w[1] << 8) | (w[2] << 16) | (w[3] << 24),
                   w[4] | (w[5] << 8) | (w[6] << 16) | (w[7] << 24));
  }
  const int per = 4 / fmt.ng;  // slices per group
  if (q % per == 0) {
    const uint32_t sz_base = is_v ? off_vsz(fmt.ng) : kOffKSz;
    *reinterpret_cast<uint32_t*>(blk + sz_base + ((q / per) * kP + t) * 4) =
        (uint32_t)p.s16 | ((uint32_t)p.z16 << 16);
  }
}

// 64-bit value of lane src (any source lane, per-lane index).  The halves are
// moved as 32-bit ints and widened as unsigned (a sign-extended low half would
// set every bit of the high half).
__device__ inline int64_t shfl64(int64_t v, int src) {
  const int lo = __shfl((int)(uint32_t)v, src, 64), hi = __shfl((int)(v >> 32), src, 64);
  return (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}
// 64-bit value of lane `lane` (wave-uniform index), widened the same way.
__device__ inline uint64_t readlane64(uint64_t v, int lane) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, lane);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), lane);
  return ((uint64_t)hi << 32) | lo;
}

template <class Rows, bool DEF>
__global__ __launch_bounds__(512) void append_mfma_kernel(
    uint8_t* __restrict__ pages, int Hkv, Rows rows, int n_rows, const float* __restrict__ Rk,
    const float* __restrict__ Rv, float clip_k, float clip_v, QFmt fmt_arg) {
  const QFmt fmt = pick(DEF, fmt_arg);
  __shared__ float4 Rs4[kD][kD / 4];                        // R[c][j], 64 KB
  __shared__ uint32_t area_all[kMfmaWaves][kAreaWords];     // 66 KB
  const int is_v = blockIdx.y;
  const float* __restrict__ R = is_v ? Rv : Rk;  // nullptr: identity
  const float clip = is_v ? clip_v : clip_k;
  const int t = threadIdx.x;
  int h = 0, bx = blockIdx.x, gx = gridDim.x;
  if (fmt.rph) {  // one KV head's rows per block (gridDim.x is a multiple of Hkv)
    h = bx % Hkv;
    bx /= Hkv;
    gx /= Hkv;
    if (R) R += (size_t)h * kD * kD;
  }
  const int n_seq = fmt.rph ? n_rows / Hkv : n_rows;
  auto row_at = [&](int i) { return fmt.rph ? (i < n_seq ? i * Hkv + h : n_rows) : i; };
  if (R) {  // 8 float4 per thread, loads issued before the stores
    float4 r4[kD * kD / 4 / 512];
#pragma unroll
    for (int i = 0; i < kD * kD / 4 / 512; ++i) r4[i] = reinterpret_cast<const float4*>(R)[t + 512 * i];
#pragma unroll
    for (int i = 0; i < kD * kD / 4 / 512; ++i) (&Rs4[0][0])[t + 512 * i] = r4[i];
  }
  __syncthreads();
  const int w = t >> 6, l = t & 63, half = l >> 5, lp = l & 31;
  const int kq = l >> 4, j = l & 15;
  uint32_t* area = area_all[w];
  float* xt = reinterpret_cast<float*>(area);
  // v_perm selector: the bf16 of channel 4 s + kq (of the 8 bytes read) into the
  // high half of a dword, zeros below: an fp32 with the same value
  const uint32_t asel = 0x01000C0Cu + 0x02020000u * (uint32_t)kq;
  const int n_items = (n_seq + kMfmaRows - 1) / kMfmaRows;
  const int stride = gx * kMfmaWaves;
  // Rows of an item: their bf16 words (lane l: channels 2 l, 2 l + 1 of each
  // row), loaded one item ahead into registers, and their destinations, resolved
  // by lane r % 16 for row r (in parallel: the routing may take several
  // dependent loads).
  uint32_t nxt[kMfmaRows];
  int64_t slot_n = -1;
  uint32_t* seg_n = nullptr;
  auto fetch = [&](int it) {
#pragma unroll
    for (int rr = 0; rr < kMfmaRows; ++rr) {
      const uint16_t* src = rows.data(row_at(it * kMfmaRows + rr), is_v);
      nxt[rr] = src ? reinterpret_cast<const uint32_t*>(src)[l] : 0u;
    }
    const int row = row_at(it * kMfmaRows + (l & 15));
    slot_n = rows.slot(row);
    seg_n = rows.seg_dst(row, is_v);
  };
  int item = bx * kMfmaWaves + w;
  if (item < n_items) fetch(item);
  for (; item < n_items; item += stride) {
    // stage the item's rows (and their bf16 copies, if any), then fetch the next
    const int64_t slot_l = slot_n;
    lane_exchange();  // the previous item's reads of the wave's area come first
#pragma unroll
    for (int rr = 0; rr < kMfmaRows; ++rr) {
      area[rr * kStagePitch + l] = nxt[rr];
      uint32_t* d = reinterpret_cast<uint32_t*>(
          (uintptr_t)readlane64((uint64_t)reinterpret_cast<uintptr_t>(seg_n), rr));
      if (d) d[l] = nxt[rr];
    }
    if (item + stride < n_items) fetch(item + stride);
    lane_exchange();
    if (R) {
      d4v acc[8];
#pragma unroll
      for (int tt = 0; tt < 8; ++tt) acc[tt] = d4v{0.0, 0.0, 0.0, 0.0};
#pragma unroll 2
      for (int s2 = 0; s2 < kD / 4; ++s2) {
        const uint2 xa = *reinterpret_cast<const uint2*>(&area[j * kStagePitch + 2 * s2]);
        const double a = (double)__uint_as_float(__builtin_amdgcn_perm(xa.y, xa.x, asel));
        const float4 r0 = Rs4[4 * s2 + kq][2 * j], r1 = Rs4[4 * s2 + kq][2 * j + 1];
        const float rb[8] = {r0.x, r0.y, r0.z, r0.w, r1.x, r1.y, r1.z, r1.w};
#pragma unroll
        for (int tt = 0; tt < 8; ++tt)
          acc[tt] = __builtin_amdgcn_mfma_f64_16x16x4f64(a, (double)rb[tt], acc[tt], 0, 0, 0);
      }
      // x~ rows to LDS as fp32 (the staged rows are no longer read)
      lane_exchange();
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float* dst = xt + (kq + 4 * i) * kXtPitch + 8 * j;
        *reinterpret_cast<float4*>(dst) =
            make_float4(__double2float_rn(acc[0][i]), __double2float_rn(acc[1][i]),
                        __double2float_rn(acc[2][i]), __double2float_rn(acc[3][i]));
        *reinterpret_cast<float4*>(dst + 4) =
            make_float4(__double2float_rn(acc[4][i]), __double2float_rn(acc[5][i]),
                        __double2float_rn(acc[6][i]), __double2float_rn(acc[7][i]));
      }
    }
    lane_exchange();  // x~ (or the staged rows) before the quantizer's reads
    if (!fmt.quantile) {  // lane l: row l / 4, channels 32 (l % 4) .. + 31
      const int rr = l >> 2, q = l & 3;
      float x[32];
      if (R) {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const float4 v = *reinterpret_cast<const float4*>(xt + rr * kXtPitch + 32 * q + 4 * i);
          x[4 * i] = v.x; x[4 * i + 1] = v.y; x[4 * i + 2] = v.z; x[4 * i + 3] = v.w;
        }
      } else {  // identity: the staged bf16 values
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const uint32_t pr = area[rr * kStagePitch + 16 * q + i];
          x[2 * i] = __uint_as_float(pr << 16);
          x[2 * i + 1] = __uint_as_float(pr & 0xffff0000u);
        }
      }
      const int row = row_at(item * kMfmaRows + rr);
      store_slice32(pages, Hkv, shfl64(slot_l, rr), row, is_v, clip, fmt, x, q);
      continue;
    }
    // token-quantile clip: row pairs, half `half` takes row 2 p + half; lane lp
    // holds channels lp + 32 q
#pragma unroll 1
    for (int p = 0; p < kMfmaRows / 2; ++p) {
      const int rr = 2 * p + half;
      double x4[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int c = lp + 32 * q;
        if (R) {
          x4[q] = (double)xt[rr * kXtPitch + c];
        } else {  // identity: the staged bf16 value
          const uint32_t pr = area[rr * kStagePitch + (c >> 1)];
          x4[q] = (double)__uint_as_float((c & 1) ? (pr & 0xffff0000u) : (pr << 16));
        }
      }
      const int row = row_at(item * kMfmaRows + rr);
      store_row4(pages, Hkv, shfl64(slot_l, rr), row, is_v, clip, fmt, x4, lp, half);
    }
  }
}

__global__ __launch_bounds__(256) void prepare_kernel(const uint16_t* __restrict__ q, int rows,
                                                      const float* __restrict__ Rk, float qscale,
                                                      float* __restrict__ qt, int rph, int Hq,
                                                      int Hkv) {
  prepare_body(blockIdx.x, q, rows, Rk, qscale, qt, rph, Hq, Hkv);
}

// One launch for a decode step's prologue: blockIdx.y 0/1 = K/V cache update
// (append_blocks blocks), 2 = query rotation (prep_blocks blocks).  The two are
// independent; the split kernel that follows needs both.
template <int RW, class Rows, bool DEF>
__global__ __launch_bounds__(256) void prologue_kernel(
    uint8_t* __restrict__ pages, int Hkv, Rows rows, int n_rows, const float* __restrict__ Rk,
    const float* __restrict__ Rv, float clip_k, float clip_v, QFmt fmt_arg, int append_blocks,
    const uint16_t* __restrict__ q, int q_rows, int Hq, float qscale, float* __restrict__ qt,
    int prep_blocks) {
  __shared__ float Rs[kD * kD];
  __shared__ double xs[kWaves][RW][kD];
  if (blockIdx.y < 2) {
    if ((int)blockIdx.x < append_blocks)
      append_body<RW>(Rs, xs, blockIdx.y, blockIdx.x, append_blocks, pages, Hkv, rows, n_rows,
                      Rk, Rv, clip_k, clip_v, pick(DEF, fmt_arg));
  } else if ((int)blockIdx.x < prep_blocks) {
    prepare_body(blockIdx.x, q, q_rows, Rk, qscale, qt, fmt_arg.rph, Hq, Hkv);
  }
}

// ---------------------------------------------------------------------------
// Clip calibration (Alg. 1 CalibrateClip).  The paper leaves the procedure open;
// it is read here as: the candidate ratio whose quantization of the rotated
// calibration rows has the smallest squared error.  A wave takes rows (token,
// head) grid-stride and rotates each exactly as the cache update does (lane l:
// channels l and l + 64); for every candidate it clips and quantizes the row with
// the cache update's steps and adds (x~_c - s (code_c - z))^2 in fp64, s and z
// read back from their stored format, to the lane's sum for that candidate.  The
// clip threshold is formed as in the cache update: ratio x group absmax (the
// group maxima found once per row), or the token quantile a_k + f (a_{k+1} - a_k)
// read from the row's |x~| sorted once per row (bitonic network over the wave).
// At the end the lanes, the waves and then (clip_reduce_kernel) the blocks are
// summed in a fixed order.
// ---------------------------------------------------------------------------
__device__ inline double wave_sum_f64(double x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}

// Ascending sort of the 128 values (element 2 l + s in slot s of lane l).
__device__ inline void wave_sort128(float& v0, float& v1, int l) {
#pragma unroll
  for (int k = 2; k <= kD; k <<= 1) {
#pragma unroll
    for (int j = k >> 1; j >= 2; j >>= 1) {
      const bool lower = ((2 * l) & j) == 0, asc = ((2 * l) & k) == 0;
      const float o0 = __shfl_xor(v0, j >> 1, 64), o1 = __shfl_xor(v1, j >> 1, 64);
      v0 = (lower == asc) ? fminf(v0, o0) : fmaxf(v0, o0);
      v1 = (lower == asc) ? fminf(v1, o1) : fmaxf(v1, o1);
    }
    const bool asc = ((2 * l) & k) == 0;  // j = 1: the lane's own pair
    const float lo = fminf(v0, v1), hi = fmaxf(v0, v1);
    v0 = asc ? lo : hi;
    v1 = asc ? hi : lo;
  }
}
__device__ inline float sorted_at(float v0, float v1, int e) {  // e wave-uniform
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int((e & 1) ? v1 : v0), e >> 1));
}

__global__ __launch_bounds__(256) void clip_err_kernel(const uint16_t* __restrict__ x, int n_rows,
                                                       const float* __restrict__ R,
                                                       const float* __restrict__ cands,
                                                       int n_cands, QFmt fmt, int Hkv,
                                                       double* __restrict__ partial) {
  __shared__ float Rs[kD * kD];
  __shared__ double xs[kWaves][kD];
  __shared__ double werr[kWaves][kMaxClipCands];
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  // rph: the block takes the rows (token, h) of one KV head h and its matrix
  int h = 0, bx = blockIdx.x, gx = gridDim.x;
  if (fmt.rph) {
    h = bx % Hkv;
    bx /= Hkv;
    gx /= Hkv;
    if (R) R += (size_t)h * kD * kD;
  }
  const int n_seq = fmt.rph ? n_rows / Hkv : n_rows;
  if (R) {
    float4 r4[kD * kD / 4 / 256];
#pragma unroll
    for (int i = 0; i < kD * kD / 4 / 256; ++i)
      r4[i] = reinterpret_cast<const float4*>(R)[threadIdx.x + 256 * i];
#pragma unroll
    for (int i = 0; i < kD * kD / 4 / 256; ++i) reinterpret_cast<float4*>(Rs)[threadIdx.x + 256 * i] = r4[i];
  }
  __syncthreads();
  double e[kMaxClipCands];
#pragma unroll
  for (int n = 0; n < kMaxClipCands; ++n) e[n] = 0.0;
  for (int i = bx * kWaves + w; i < n_seq; i += gx * kWaves) {
    const int row = fmt.rph ? i * Hkv + h : i;
    const uint32_t pair = reinterpret_cast<const uint32_t*>(x + (size_t)row * kD)[l];
    lane_exchange();  // the previous row's reads of xs[w] come first
    xs[w][2 * l] = (double)__uint_as_float(pair << 16);
    xs[w][2 * l + 1] = (double)__uint_as_float(pair & 0xffff0000u);
    lane_exchange();
    double acc0 = 0.0, acc1 = 0.0;
    if (R) {
#pragma unroll 4
      for (int c = 0; c < kD; ++c) {
        const double xc = xs[w][c];
        acc0 = __fma_rn(xc, (double)Rs[c * kD + l], acc0);
        acc1 = __fma_rn(xc, (double)Rs[c * kD + l + 64], acc1);
      }
    } else {
      acc0 = xs[w][l];
      acc1 = xs[w][l + 64];
    }
    const float xt0 = __double2float_rn(acc0), xt1 = __double2float_rn(acc1);
    float g0, g1, s0 = 0.0f, s1 = 0.0f;
    if (fmt.quantile) {
      s0 = fabsf(xt0);
      s1 = fabsf(xt1);
      wave_sort128(s0, s1, l);
    } else {
      group_reduce2<true>(fabsf(xt0), fabsf(xt1), fmt.ng, g0, g1);
    }
#pragma clang loop unroll(full)
    for (int n = 0; n < kMaxClipCands; ++n) {
      if (n >= n_cands) continue;
      const float clip = cands[n];
      float tau0, tau1;
      if (fmt.quantile) {
        int k;
        float f;
        quantile_pos(clip, k, f);
        k = __builtin_amdgcn_readfirstlane(k);
        const float ak = sorted_at(s0, s1, k);
        tau0 = tau1 = k >= kD - 1 ? ak : lerp_tau(ak, sorted_at(s0, s1, k + 1), f);
      } else {
        tau0 = __fmul_rn(clip, g0);
        tau1 = __fmul_rn(clip, g1);
      }
      const float y0 = fminf(fmaxf(xt0, -tau0), tau0), y1 = fminf(fmaxf(xt1, -tau1), tau1);
      float a0, a1, b0, b1;
      group_reduce2<false>(y0, y1, fmt.ng, a0, a1);
      group_reduce2<true>(y0, y1, fmt.ng, b0, b1);
      const QOut q0 = quantize(y0, a0, b0, fmt);
      const QOut q1 = quantize(y1, a1, b1, fmt);
      const double d0 = (double)xt0 - (double)meta_load(fmt, q0.s16) *
                                          ((double)q0.code - (double)meta_load(fmt, q0.z16));
      const double d1 = (double)xt1 - (double)meta_load(fmt, q1.s16) *
                                          ((double)q1.code - (double)meta_load(fmt, q1.z16));
      e[n] += d0 * d0 + d1 * d1;
    }
  }
#pragma unroll
  for (int n = 0; n < kMaxClipCands; ++n) {
    if (n >= n_cands) continue;
    const double t = wave_sum_f64(e[n]);
    if (l == 0) werr[w][n] = t;
  }
  __syncthreads();
  if ((int)threadIdx.x < n_cands) {
    const int n = threadIdx.x;
    partial[(size_t)blockIdx.x * n_cands + n] = ((werr[0][n] + werr[1][n]) + werr[2][n]) + werr[3][n];
  }
}

// err[n] = (sum of the blocks' partials) / (n_rows d); best = the candidate of the
// first minimum.  Thread (candidate n, part p) adds blocks p, p + 8, ... in order,
// then the 8 part sums are added in order (a fixed order: deterministic).
constexpr int kClipParts = 8;

__global__ __launch_bounds__(kClipParts * kMaxClipCands) void clip_reduce_kernel(
    const double* __restrict__ partial, int n_blocks, int n_cands,
    const float* __restrict__ cands, double inv_n, double* __restrict__ err,
    float* __restrict__ best) {
  __shared__ double ps[kClipParts][kMaxClipCands];
  __shared__ double es[kMaxClipCands];
  const int n = threadIdx.x % kMaxClipCands, part = threadIdx.x / kMaxClipCands;
  double acc = 0.0;
  if (n < n_cands)
    for (int b = part; b < n_blocks; b += kClipParts) acc += partial[(size_t)b * n_cands + n];
  ps[part][n] = acc;
  __syncthreads();
  if (part == 0 && n < n_cands) {
    double tot = 0.0;
#pragma unroll
    for (int p = 0; p < kClipParts; ++p) tot += ps[p][n];
    es[n] = tot * inv_n;
    err[n] = es[n];
  }
  __syncthreads();
  if (threadIdx.x == 0 && best) {
    int arg = 0;
    for (int i = 1; i < n_cands; ++i)
      if (es[i] < es[arg]) arg = i;
    best[0] = cands[arg];
  }
}

}  // namespace

namespace {
int64_t append_blocks_for(int64_t n_rows, int rw) {
  const int64_t n_items = (n_rows + rw - 1) / rw;
  const int64_t blocks = (n_items + kWaves - 1) / kWaves;
  return blocks > 1024 ? 1024 : blocks;
}
// With one rotation per KV head a block takes one head's rows: a multiple of Hkv
// blocks, each head's share sized for its n_rows / Hkv rows.
int64_t append_blocks_rph(int64_t n_rows, int rw, int64_t Hkv, int rph) {
  if (!rph) return append_blocks_for(n_rows, rw);
  const int64_t n_items = (n_rows / Hkv + rw - 1) / rw;
  int64_t per = (n_items + kWaves - 1) / kWaves;
  per = std::max<int64_t>(1, std::min(per, std::max<int64_t>(1, 1024 / Hkv)));
  return per * Hkv;
}

bool is_default(const QFmt& f) { return f.bf16 == 0 && f.quantile == 0 && f.ng == 4 && f.rph == 0; }

template <class Rows>
hipError_t launch_rows(void* pages, int64_t Hkv, const Rows& rows, int64_t n_rows, const float* Rk,
                       const float* Rv, float clip_k, float clip_v, QFmt fmt, hipStream_t st) {
  const bool def = is_default(fmt);
  if (n_rows <= 4096) {  // one decode step: many short waves
    const dim3 grid((unsigned)append_blocks_rph(n_rows, 1, Hkv, fmt.rph), 2);
    auto go = [&](auto kernel) {
      hipLaunchKernelGGL(kernel, grid, dim3(256), 0, st, static_cast<uint8_t*>(pages), (int)Hkv,
                         rows, (int)n_rows, Rk, Rv, clip_k, clip_v, fmt);
    };
    if (def) go(append_kernel<1, Rows, true>);
    else go(append_kernel<1, Rows, false>);
  } else {  // bulk: one persistent 8-wave block per CU (fp64 MFMA), half of them per tensor
    const int64_t heads = fmt.rph ? Hkv : 1;  // rph: a block per head's share
    const int64_t items = (n_rows / heads + kMfmaRows - 1) / kMfmaRows;
    int64_t nb = (items + kMfmaWaves - 1) / kMfmaWaves;
    const int64_t cap = std::max<int64_t>(1, device_cus() / 2 / heads);
    if (nb > cap) nb = cap;
    nb *= heads;
    auto go = [&](auto kernel) {
      hipLaunchKernelGGL(kernel, dim3((unsigned)nb, 2), dim3(512), 0, st,
                         static_cast<uint8_t*>(pages), (int)Hkv, rows, (int)n_rows, Rk, Rv,
                         clip_k, clip_v, fmt);
    };
    if (def) go(append_mfma_kernel<Rows, true>);
    else go(append_mfma_kernel<Rows, false>);
  }
  return hipGetLastError();
}

template <class Rows>
hipError_t launch_prologue(void* pages, int64_t Hkv, const Rows& rows, int64_t n_rows,
                           const float* Rk, const float* Rv, float clip_k, float clip_v,
                           QFmt fmt, const uint16_t* q, int B, int Hq, float qscale, float* qt,
                           hipStream_t st) {
  const int rw = n_rows <= 4096 ? 1 : 4;
  const int ab = n_rows > 0 ? (int)append_blocks_rph(n_rows, rw, Hkv, fmt.rph) : 0;
  const int pb = query_blocks(B, Hq, (int)Hkv, fmt.rph, kPrepRows);
  const dim3 grid((unsigned)(ab > pb ? ab : pb), 3);
  auto go = [&](auto kernel) {
    hipLaunchKernelGGL(kernel, grid, dim3(256), 0, st, static_cast<uint8_t*>(pages), (int)Hkv,
                       rows, (int)n_rows, Rk, Rv, clip_k, clip_v, fmt, ab, q, B * Hq, Hq, qscale,
                       qt, pb);
  };
  const bool def = is_default(fmt);
  if (rw == 1) {
    if (def) go(prologue_kernel<1, Rows, true>);
    else go(prologue_kernel<1, Rows, false>);
  } else {
    if (def) go(prologue_kernel<4, Rows, true>);
    else go(prologue_kernel<4, Rows, false>);
  }
  return hipGetLastError();
}
}  // namespace

hipError_t launch_append(void* pages, int64_t Hkv, const uint16_t* k, const uint16_t* v,
                         const int64_t* slots, int n_tok, const float* Rk, const float* Rv,
                         float clip_k, float clip_v, QuantFmt fmt, hipStream_t st) {
  const int64_t n_rows = (int64_t)n_tok * Hkv;
  const PlainRows rows{k, v, slots, (int)n_rows, (int)Hkv};
  return launch_rows(pages, Hkv, rows, n_rows, Rk, Rv, clip_k, clip_v, fmt, st);
}

hipError_t launch_mixed_append(void* pages, uint16_t* seg, int64_t Hkv, int S0, int W,
                               const uint16_t* k, const uint16_t* v, const int32_t* seq_idx,
                               const int64_t* pos, int n_tok, const int32_t* seq_lens,
                               const int32_t* block_table, int max_pages, const float* Rk,
                               const float* Rv, float clip_k, float clip_v, QuantFmt fmt,
                               hipStream_t st) {
  const int64_t n_rows = (int64_t)n_tok * Hkv;
  const PrefillRows rows{k, v, seg, seq_idx, pos, seq_lens, block_table, (int)n_rows, (int)Hkv,
                         max_pages, S0, W};
  return launch_rows(pages, Hkv, rows, n_rows, Rk, Rv, clip_k, clip_v, fmt, st);
}

hipError_t launch_decode_prepare(const uint16_t* q, int B, int Hq, const float* Rk,
                                 float qscale, float* qt, hipStream_t st, int rph, int Hkv) {
  const int rows = B * Hq;
  hipLaunchKernelGGL(prepare_kernel, dim3(query_blocks(B, Hq, Hkv, rph, kPrepRows)), dim3(256), 0,
                     st, q, rows, Rk, qscale, qt, rph, Hq, Hkv);
  return hipGetLastError();
}

hipError_t launch_step_prologue(void* pages, int64_t Hkv, const uint16_t* k, const uint16_t* v,
                                const int64_t* slots, int n_tok, const float* Rk,
                                const float* Rv, float clip_k, float clip_v, QuantFmt fmt,
                                const uint16_t* q, int B, int Hq, float qscale, float* qt,
                                hipStream_t st) {
  const int64_t n_rows = (int64_t)n_tok * Hkv;
  const PlainRows rows{k, v, slots, (int)n_rows, (int)Hkv};
  return launch_prologue(pages, Hkv, rows, n_rows, Rk, Rv, clip_k, clip_v, fmt, q, B, Hq, qscale,
                         qt, st);
}

hipError_t launch_mixed_step_prologue(void* pages, uint16_t* seg, int64_t Hkv, int S0, int W,
                                      const uint16_t* k, const uint16_t* v,
                                      const int32_t* seq_lens, const int32_t* block_table,
                                      int max_pages, const float* Rk, const float* Rv,
                                      float clip_k, float clip_v, QuantFmt fmt, const uint16_t* q,
                                      int B, int Hq, float qscale, float* qt, hipStream_t st) {
  const int64_t n_rows = (int64_t)B * Hkv;
  const StepRows rows{k, v, seg, seq_lens, block_table, (int)n_rows, (int)Hkv, max_pages, S0, W};
  return launch_prologue(pages, Hkv, rows, n_rows, Rk, Rv, clip_k, clip_v, fmt, q, B, Hq, qscale,
                         qt, st);
}

hipError_t launch_clip_errors(const uint16_t* x, int64_t n_rows, const float* R,
                              const float* cands, int n_cands, QuantFmt fmt, int Hkv,
                              double* partial, int n_blocks, double* err, float* best,
                              hipStream_t st) {
  hipLaunchKernelGGL(clip_err_kernel, dim3((unsigned)n_blocks), dim3(256), 0, st, x, (int)n_rows, R,
                     cands, n_cands, fmt, Hkv, partial);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(clip_reduce_kernel, dim3(1), dim3(kClipParts * kMaxClipCands), 0, st, partial,
                     n_blocks, n_cands,
                     cands, 1.0 / ((double)n_rows * kD), err, best);
  return hipGetLastError();
}

int clip_blocks(int64_t n_rows, int Hkv, int rph) {
  const int64_t heads = rph ? Hkv : 1;  // rph: blocks per head, times Hkv
  const int64_t items = (n_rows / heads + kWaves - 1) / kWaves;
  const int64_t cap = std::max<int64_t>(1, 4 * (int64_t)device_cus() / heads);
  return (int)(std::max<int64_t>(1, std::min(items, cap)) * heads);
}

}  // namespace oscar
