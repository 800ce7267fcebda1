// bf16 paged-decode baseline: the same paging and split-K / log-sum-exp scheme as
// the INT2 path, over an uncompressed bf16 cache (no rotation, no quantization).
// It exists to compare the INT2 path against plain bf16 decode on the same GPU,
// so it is written to run at the HBM read rate: both contractions are bf16
// matrix-core products with one row per query head.
//
// Page-head block (page p, kv-head h) at element (p*Hkv + h) * 2*P*d, stored in
// the order the decode's matrix-core operands take it, so that every load of the
// decode is one contiguous 1 KB per wave (16 bytes per lane) straight into the
// operand registers:
//   K(t, c) at ((u*4 + kc)*64 + lane)*8 + e,        t = 4 lo + u, c = 32 hi + 8 kc + e
//   V(t, c) at P*d + ((ct*2 + kt)*64 + lane)*8 + e,  t = 16 hi + 8 kt + e, c = 16 ct + lo
// with lane = lo + 16 hi.  The query is scaled by sm_scale*log2 e by the prepare
// kernel (R = I) and the reduce takes R = I.
#include "internal.h"

namespace oscar {
namespace {

constexpr int kAppendWaves = 4;
constexpr int kBlockElems = 2 * kP * kD;  // bf16 elements per page-head block
constexpr float kBfSlack = 10.0f;         // reference-maximum slack (log2 units), as the INT2 path

typedef __bf16 bf8 __attribute__((ext_vector_type(8)));
typedef float f4v __attribute__((ext_vector_type(4)));
typedef uint32_t u4v __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void bf16_append_kernel(uint16_t* __restrict__ pages, int Hkv,
                                                          const uint16_t* __restrict__ k,
                                                          const uint16_t* __restrict__ v,
                                                          const int64_t* __restrict__ slots,
                                                          int n_rows) {
  // one wave per (token, head) row; lane writes channels 2l, 2l+1 of K and of V
  const int row = blockIdx.x * kAppendWaves + (threadIdx.x >> 6);
  const int l = threadIdx.x & 63;
  if (row >= n_rows) return;
  const int tok = row / Hkv, h = row - tok * Hkv;
  const int64_t slot = slots[tok];
  const int64_t page = slot / kP;
  const int t = (int)(slot - page * kP);
  uint16_t* blk = pages + ((size_t)page * Hkv + h) * kBlockElems;
  const uint32_t kk = reinterpret_cast<const uint32_t*>(k + (size_t)row * kD)[l];
  const uint32_t vv = reinterpret_cast<const uint32_t*>(v + (size_t)row * kD)[l];
  // K: channels 2l, 2l+1 are e, e+1 of one 16-byte operand slot (adjacent)
  {
    const int c = 2 * l, u = t & 3, lo = t >> 2, hi = c >> 5, kc = (c >> 3) & 3, e = c & 7;
    *reinterpret_cast<uint32_t*>(blk + ((u * 4 + kc) * 64 + lo + 16 * hi) * 8 + e) = kk;
  }
  // V: token t is element e of the operand slots of channels 2l and 2l+1
  const int hi = t >> 4, kt = (t >> 3) & 1, e = t & 7;
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int c = 2 * l + j, ct = c >> 4, lo = c & 15;
    blk[kP * kD + ((ct * 2 + kt) * 64 + lo + 16 * hi) * 8 + e] = (uint16_t)(j ? vv >> 16 : vv & 0xffffu);
  }
}

__device__ inline f4v mfma_bf(u4v a, u4v b, f4v c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf8, a), __builtin_bit_cast(bf8, b), c,
                                                 0, 0, 0);
}
// round to nearest even bf16 of two floats, packed (lo, hi); and the value back
__device__ inline uint32_t bf16x2(float lo, float hi) {
  const __bf16 a = (__bf16)lo, b = (__bf16)hi;
  return (uint32_t)__builtin_bit_cast(uint16_t, a) | ((uint32_t)__builtin_bit_cast(uint16_t, b) << 16);
}
__device__ inline float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ inline float bf_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
// x = hi + lo as two bf16 values (about 16 significant bits), for 8 values: the
// hi and the lo operand of one MFMA k-group
__device__ inline void split8(const float (&x)[8], u4v& hi, u4v& lo) {
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const uint32_t h = bf16x2(x[2 * j], x[2 * j + 1]);
    hi[j] = h;
    lo[j] = bf16x2(x[2 * j] - bf_lo(h), x[2 * j + 1] - bf_hi(h));
  }
}

__device__ inline float rowmax16(float x) {  // over the 16 lanes of a row
#pragma unroll
  for (int m = 8; m >= 1; m >>= 1) x = fmaxf(x, __shfl_xor(x, m, 64));
  return x;
}
__device__ inline float rowsum16(float x) {
#pragma unroll
  for (int m = 8; m >= 1; m >>= 1) x += __shfl_xor(x, m, 64);
  return x;
}

// One wave per (split, kv-head, sequence): pages [s*pps, (s+1)*pps) of the
// sequence.  MFMA 16x16x32 bf16 lane layout: A row lo, k-slots 8hi + e; B column
// lo, k-slots 8hi + e; D lane l register i = (row 4hi + i, column lo).
//   scores, token tile u: rows = query heads (up to 16), k = channels (k-chunk
//     kc, k-slot (hi, e) <-> channel 32hi + 8kc + e), column lo = token 4lo + u;
//     q in hi + lo bf16 halves, two MFMAs per k-chunk.
//   P.V, channel tile ct: rows = heads, k = tokens (k-chunk kt, k-slot (hi, e)
//     <-> token 16hi + 8kt + e), column lo = channel 16ct + lo; p in hi + lo
//     halves.  The output accumulates in the MFMA accumulators across pages
//     (rescaled only when a page's maximum exceeds the reference by kBfSlack).
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(3, 3))) void bf16_split_kernel(
    const uint16_t* __restrict__ pages, int Hkv, int Hq, const int32_t* __restrict__ block_table,
    int max_pages, const int32_t* __restrict__ seq_lens, int num_splits, int pages_per_split,
    const float* __restrict__ qt, float* __restrict__ part_o, float* __restrict__ part_ml) {
  __shared__ float4 ps[16][17];  // p of the page: [head][token / 4], pitch 17
  __shared__ u4v qa[4][2][64];   // score A operands (k-chunk, hi/lo half, lane): kept in LDS
                                 // so that a page's K and V fit in registers at 3 waves per SIMD
  const int s = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
  const int g = Hq / Hkv;
  const int l = threadIdx.x & 63, lo = l & 15, hi = l >> 4;
  const int len = min(max(seq_lens[b], 0), max_pages * kP);
  const int npg = (len + kP - 1) / kP;
  const int p0 = s * pages_per_split;
  const int p1 = min(npg, p0 + pages_per_split);

  // query operands of head lo: channels 32hi + 8kc + e
  {
    float qv[4][8];
#pragma unroll
    for (int kc = 0; kc < 4; ++kc)
#pragma unroll
      for (int e = 0; e < 8; ++e) qv[kc][e] = 0.0f;
    if (lo < g) {
      const float* src = qt + ((size_t)b * Hq + kvh * g + lo) * kD + 32 * hi;
#pragma unroll
      for (int kc = 0; kc < 4; ++kc) {
        const float4 x0 = *reinterpret_cast<const float4*>(src + 8 * kc);
        const float4 x1 = *reinterpret_cast<const float4*>(src + 8 * kc + 4);
        qv[kc][0] = x0.x; qv[kc][1] = x0.y; qv[kc][2] = x0.z; qv[kc][3] = x0.w;
        qv[kc][4] = x1.x; qv[kc][5] = x1.y; qv[kc][6] = x1.z; qv[kc][7] = x1.w;
      }
    }
#pragma unroll
    for (int kc = 0; kc < 4; ++kc) split8(qv[kc], qa[kc][0][l], qa[kc][1][l]);
  }

  float m[4], lsum[4];
  f4v o[8];
#pragma unroll
  for (int i = 0; i < 4; ++i) { m[i] = -INFINITY; lsum[i] = 0.0f; }
#pragma unroll
  for (int ct = 0; ct < 8; ++ct) o[ct] = f4v{0.0f, 0.0f, 0.0f, 0.0f};
  const int32_t* __restrict__ bt = block_table + (size_t)b * max_pages;

  for (int pg = p0; pg < p1; ++pg) {
    const uint16_t* blk = pages + ((size_t)bt[pg] * Hkv + kvh) * kBlockElems;
    const int ntok = min(kP, len - pg * kP);
    // K of tokens 4lo + u, channels 32hi + 8kc + (0..7)
    const u4v* kb = reinterpret_cast<const u4v*>(blk) + l;
    u4v kr[4][4];
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int kc = 0; kc < 4; ++kc) kr[u][kc] = __builtin_nontemporal_load(kb + (u * 4 + kc) * 64);
    // ---- scores of heads 4hi + i, tokens 4lo + u ----
    f4v d[4];
#pragma unroll
    for (int kc = 0; kc < 4; ++kc) {
      const u4v ah = qa[kc][0][l], al = qa[kc][1][l];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        d[u] = mfma_bf(ah, kr[u][kc], kc == 0 ? f4v{0.0f, 0.0f, 0.0f, 0.0f} : d[u]);
        d[u] = mfma_bf(al, kr[u][kc], d[u]);
      }
    }
    float sc[4][4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const bool ok = 4 * lo + u < ntok;
#pragma unroll
      for (int i = 0; i < 4; ++i) sc[u][i] = ok ? d[u][i] : -INFINITY;
    }
    // V^T of channels 16ct + lo, tokens 16hi + 8kt + (0..7), loaded once K is spent
    // (kept below the score MFMAs: K and V of a whole page do not fit at 3 waves)
    __builtin_amdgcn_sched_barrier(0);
    const u4v* vbp = reinterpret_cast<const u4v*>(blk + kP * kD) + l;
    u4v vr[8][2];
#pragma unroll
    for (int ct = 0; ct < 8; ++ct)
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) vr[ct][kt] = __builtin_nontemporal_load(vbp + (ct * 2 + kt) * 64);
    if (ntok < kP) {  // the partial last page: tokens past the length weigh 0
#pragma unroll
      for (int ct = 0; ct < 8; ++ct)
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int t = 16 * hi + 8 * kt + 2 * j;
            const uint32_t mk = (t < ntok ? 0xffffu : 0u) | (t + 1 < ntok ? 0xffff0000u : 0u);
            vr[ct][kt][j] &= mk;
          }
    }
    // ---- online softmax with a lazily moved reference maximum ----
    float mx[4];
    bool need = false;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      mx[i] = rowmax16(fmaxf(fmaxf(sc[0][i], sc[1][i]), fmaxf(sc[2][i], sc[3][i])));
      need = need || !(mx[i] <= m[i] + kBfSlack);
    }
    if (__ballot(need) != 0ull) {  // wave-uniform
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float mn = fmaxf(m[i], mx[i]);
        const float alpha = __builtin_amdgcn_exp2f(m[i] - mn);  // m = -inf on the first page -> 0
        m[i] = mn;
        lsum[i] *= alpha;
#pragma unroll
        for (int ct = 0; ct < 8; ++ct) o[ct][i] *= alpha;
      }
    }
    lane_exchange();  // after every lane's reads of the previous page's p
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float pv[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        pv[u] = __builtin_amdgcn_exp2f(sc[u][i] - m[i]);  // -inf -> 0
        lsum[i] += pv[u];
      }
      ps[4 * hi + i][lo] = make_float4(pv[0], pv[1], pv[2], pv[3]);
    }
    lane_exchange();
    // ---- P.V: p of head lo, tokens 16hi + 8kt + (0..7) ----
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      const float4 p0v = ps[lo][4 * hi + 2 * kt];
      const float4 p1v = ps[lo][4 * hi + 2 * kt + 1];
      const float pw[8] = {p0v.x, p0v.y, p0v.z, p0v.w, p1v.x, p1v.y, p1v.z, p1v.w};
      u4v ah, al;
      split8(pw, ah, al);
#pragma unroll
      for (int ct = 0; ct < 8; ++ct) {
        o[ct] = mfma_bf(ah, vr[ct][kt], o[ct]);
        o[ct] = mfma_bf(al, vr[ct][kt], o[ct]);
      }
    }
  }

  // ---- the piece's partial state: heads 4hi + i ----
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int h = 4 * hi + i;
    const float ltot = rowsum16(lsum[i]);
    if (h >= g) continue;
    const size_t row = ((size_t)b * Hq + kvh * g + h) * num_splits + s;
    const bool empty = p0 >= p1;
#pragma unroll
    for (int ct = 0; ct < 8; ++ct) part_o[row * kD + 16 * ct + lo] = empty ? 0.0f : o[ct][i];
    if (lo == 0) {
      part_ml[row * 2] = empty ? -INFINITY : m[i];
      part_ml[row * 2 + 1] = empty ? 0.0f : ltot;
    }
  }
}

}  // namespace

hipError_t launch_bf16_append(void* pages, int64_t Hkv, const uint16_t* k, const uint16_t* v,
                              const int64_t* slots, int n_tok, hipStream_t st) {
  const int64_t n_rows = (int64_t)n_tok * Hkv;
  hipLaunchKernelGGL(bf16_append_kernel, dim3((unsigned)((n_rows + kAppendWaves - 1) / kAppendWaves)),
                     dim3(256), 0, st, static_cast<uint16_t*>(pages), (int)Hkv, k, v, slots,
                     (int)n_rows);
  return hipGetLastError();
}

hipError_t launch_bf16_split(const uint16_t* pages, int Hkv, int B, int Hq,
                             const int32_t* block_table, int max_pages, const int32_t* seq_lens,
                             int num_splits, const float* qt, float* part_o, float* part_ml,
                             hipStream_t st) {
  const int pps = (max_pages + num_splits - 1) / num_splits;
  hipLaunchKernelGGL(bf16_split_kernel, dim3(num_splits, Hkv, B), dim3(64), 0, st, pages, Hkv, Hq,
                     block_table, max_pages, seq_lens, num_splits, pps, qt, part_o, part_ml);
  return hipGetLastError();
}

}  // namespace oscar
