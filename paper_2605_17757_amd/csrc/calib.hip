// Offline calibration of the rotations (Sec. 3 "Algorithm Design: Offline
// Calibration and Justification"; App. "Hadamard transform" and "P_K"; Alg. 1
// Calibrate), on the GPU:
//
//   C_Q = (1/Hkv) sum_h (1/(T g)) sum_{i in group h} sum_t q_{t,i}^T q_{t,i}
//                                   -> gram_kernel + gram_reduce_kernel
//   O   = softmax_row(Q K^T / sqrt(d) + M) V per query head   -> attn_kernel
//   C_S = the same GQA average of o^T o (= V^T S^T S V / N)   -> gram kernels on O
//   C   = U diag(lam) U^T, lam descending, each eigenvector's largest-magnitude
//         entry positive                                      -> jacobi_kernel,
//                                                                jacobi_vectors_kernel,
//                                                                eig_finish_kernel
//   R   = U H_Had P_br                                         -> compose_kernel
//
// Equal group sizes make the GQA average the plain mean over all T * Hq rows.
//
// This file is compiled with -ffp-contract=off: the composition's sums are
// separate IEEE multiplies and adds in ascending order, so that for a given U the
// rotation is the same bit pattern as the plain definition evaluated in fp64.
#include <math.h>

#include "internal.h"

namespace oscar {
namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// ---------------------------------------------------------------------------
// Second-moment matrix X^T X of rows X [n][128] (bf16 or fp32) on fp32 MFMAs.
// A block stages 64 rows at a time in LDS as fp32 and accumulates the 10 upper
// 32x32 tiles of the 128x128 result (2 per wave, 5 waves) with
// v_mfma_f32_32x32x2_f32: per step the two rows 2s + h (h = lane / 32) feed
// lane l as A[i = l % 32][k = h] = x[32 ti + i] and B[k = h][j = l % 32] = x[32 tj + j].
// Products of bf16 inputs are exact in fp32; the block's fp32 partial tiles are
// summed in fp64, in block order, by gram_reduce_kernel.
// ---------------------------------------------------------------------------
constexpr int kGramRows = 64;
constexpr int kGramWaves = 5;
constexpr int kGramTiles = 10;
constexpr int kGramPitch = kD + 32;  // floats: rows 2s and 2s + 1 use different bank halves

__device__ inline void gram_tile(int t, int& ti, int& tj) {
  // (0,0) (0,1) (0,2) (0,3) (1,1) (1,2) (1,3) (2,2) (2,3) (3,3)
  ti = t < 4 ? 0 : t < 7 ? 1 : t < 9 ? 2 : 3;
  const int first = ti == 0 ? 0 : ti == 1 ? 4 : ti == 2 ? 7 : 9;
  tj = ti + (t - first);
}

// Row r of X is at element (r / rpt) * tok_stride + (r % rpt) * 128: rpt
// consecutive rows per token (one KV head's query heads), tokens tok_stride apart.
__device__ inline int64_t gram_row(int64_t r, int64_t rpt, int64_t tok_stride) {
  return (r / rpt) * tok_stride + (r % rpt) * kD;
}

template <bool BF16>
__global__ __launch_bounds__(kGramWaves * 64) void gram_kernel(const void* __restrict__ X,
                                                              int64_t n_rows,
                                                              int64_t rows_per_block,
                                                              int64_t rpt, int64_t tok_stride,
                                                              float* __restrict__ partial) {
  __shared__ float xs[kGramRows * kGramPitch];
  const int tid = threadIdx.x, w = tid >> 6, l = tid & 63, h = l >> 5, li = l & 31;
  int ti0, tj0, ti1, tj1;
  gram_tile(2 * w, ti0, tj0);
  gram_tile(2 * w + 1, ti1, tj1);
  f32x16 acc0 = {}, acc1 = {};
  const int64_t r0 = (int64_t)blockIdx.x * rows_per_block;
  const int64_t r1 = min(n_rows, r0 + rows_per_block);
  for (int64_t base = r0; base < r1; base += kGramRows) {
    __syncthreads();
    if (BF16) {  // 64 rows x 16 pieces of 8 bf16
      const uint16_t* x = static_cast<const uint16_t*>(X);
      for (int idx = tid; idx < kGramRows * 16; idx += kGramWaves * 64) {
        const int row = idx >> 4, c8 = idx & 15;
        uint4 u = make_uint4(0, 0, 0, 0);
        if (base + row < r1)
          u = *reinterpret_cast<const uint4*>(x + gram_row(base + row, rpt, tok_stride) + c8 * 8);
        float* dst = xs + row * kGramPitch + c8 * 8;
        const uint32_t wd[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          dst[2 * e] = __uint_as_float(wd[e] << 16);
          dst[2 * e + 1] = __uint_as_float(wd[e] & 0xffff0000u);
        }
      }
    } else {  // 64 rows x 32 float4
      const float* x = static_cast<const float*>(X);
      for (int idx = tid; idx < kGramRows * 32; idx += kGramWaves * 64) {
        const int row = idx >> 5, c4 = idx & 31;
        float4 f = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
        if (base + row < r1)
          f = *reinterpret_cast<const float4*>(x + gram_row(base + row, rpt, tok_stride) + c4 * 4);
        *reinterpret_cast<float4*>(xs + row * kGramPitch + c4 * 4) = f;
      }
    }
    __syncthreads();
#pragma unroll 4
    for (int s = 0; s < kGramRows / 2; ++s) {
      const float* rp = xs + (2 * s + h) * kGramPitch + li;
      const float a0 = rp[32 * ti0], b0 = rp[32 * tj0];
      const float a1 = rp[32 * ti1], b1 = rp[32 * tj1];
      acc0 = __builtin_amdgcn_mfma_f32_32x32x2f32(a0, b0, acc0, 0, 0, 0);
      acc1 = __builtin_amdgcn_mfma_f32_32x32x2f32(a1, b1, acc1, 0, 0, 0);
    }
  }
  // result element of register r: row 8 (r / 4) + 4 h + r % 4, column l % 32
  float* p0 = partial + ((size_t)blockIdx.x * kGramTiles + 2 * w) * 1024;
  float* p1 = p0 + 1024;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int i = 8 * (r >> 2) + 4 * h + (r & 3);
    p0[i * 32 + li] = acc0[r];
    p1[i * 32 + li] = acc1[r];
  }
}

// C[i][j] = C[j][i] = (sum over the blocks' partial tiles, in fp64) * inv_n.  A
// block takes 32 elements; thread (element e, part p) adds blocks p, p + 8, ...
// in order, then part 0 adds the 8 sums in order (a fixed order: deterministic).
constexpr int kRedParts = 8;

__global__ __launch_bounds__(256) void gram_reduce_kernel(const float* __restrict__ partial,
                                                          int n_blocks, double inv_n,
                                                          double* __restrict__ C) {
  __shared__ double sums[kRedParts][32];
  const int el = threadIdx.x & 31, part = threadIdx.x >> 5;
  const int e = blockIdx.x * 32 + el;  // tile * 1024 + element
  double acc = 0.0;
  for (int b = part; b < n_blocks; b += kRedParts)
    acc += (double)partial[((size_t)b * kGramTiles) * 1024 + e];
  sums[part][el] = acc;
  __syncthreads();
  if (part != 0) return;
  double tot = 0.0;
#pragma unroll
  for (int p = 0; p < kRedParts; ++p) tot += sums[p][el];
  const int t = e >> 10, ij = e & 1023;
  int ti, tj;
  gram_tile(t, ti, tj);
  const int i = 32 * ti + (ij >> 5), j = 32 * tj + (ij & 31);
  const double c = tot * inv_n;
  C[i * kD + j] = c;
  C[j * kD + i] = c;
}

// ---------------------------------------------------------------------------
// Calibration attention, O = softmax_row(Q K^T / sqrt(d) + M) V, M causal or 0.
// A block of kCalibAttnWaves (8) waves covers one KV head's key/value tiles for hc
// of its query heads and 32 * 8 / hc queries; wave w takes head (w % hc) and 32
// queries (blocks of 4 waves, two per CU, measured 1.34x slower: each K/V tile then
// serves half as many waves; a double-buffered version that issues the next tile's
// score MFMAs before the current tile's softmax needs more than 256 registers per
// lane and spills: 1.16x slower).
// Per 64-key tile the wave computes S^T = K Q^T (v_mfma_f32_32x32x16_bf16,
// A = K rows from LDS, B = the wave's queries held in registers), so that a lane
// owns one query and 32 of the tile's keys: the row maximum is a lane maximum and
// one cross-half exchange.  Those scores, exponentiated, are already the B
// operand of O^T += V^T P^T, the key order inside an MFMA step being free as long
// as A and B agree; V^T comes from LDS (staged transposed).  P enters the bf16
// MFMA as a sum of two bf16 parts, p = hi + lo (16 significant bits), so that
// the product with the bf16 values is kept to ~2^-17 relative; Q K^T of bf16
// inputs is exact up to the fp32 accumulation.  Online softmax in base 2; the
// running maximum is raised (and O^T, l rescaled) only when a tile's maximum
// exceeds it by more than 8, the result being the same up to rounding; O^T is kept
// in the accumulators and normalized at the end.
// ---------------------------------------------------------------------------
constexpr int kAttnWaves = kCalibAttnWaves;
constexpr int kKPitch = kD + 8;  // bf16: 272-byte K rows (conflict-free 16-byte reads)
constexpr int kVPitch = 64 + 4;  // bf16: 136-byte V^T rows (conflict-free 8-byte reads)

__global__ __launch_bounds__(kAttnWaves * 64) void attn_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k, const uint16_t* __restrict__ v,
    int T, int Hq, int Hkv, int hc, int causal, float scale_log2, int n_qtiles,
    float* __restrict__ out) {
  __shared__ __align__(16) uint16_t Ks[64 * kKPitch];
  __shared__ __align__(16) uint16_t Vt[kD * kVPitch];
  const int tid = threadIdx.x, w = tid >> 6, l = tid & 63, h = l >> 5, li = l & 31;
  const int g = Hq / Hkv;
  const int span = 32 * (kAttnWaves / hc);
  const int qt = n_qtiles - 1 - (int)blockIdx.y;  // longest causal rows first
  const int head = blockIdx.x * hc + (w % hc);
  const int kvh = (blockIdx.x * hc) / g;
  const int qw0 = qt * span + 32 * (w / hc);
  const int qblock_last = min(T - 1, qt * span + span - 1);
  const int n_kt = causal ? qblock_last / 64 + 1 : (T + 63) / 64;
  const bool active = qw0 < T;
  const int wave_kt = causal ? min(T - 1, qw0 + 31) / 64 + 1 : n_kt;
  const int qrow = qw0 + li;

  // the wave's queries: lane l holds q[qrow][16 ks + 8 h + 0..7], ks = 0..7
  bf16x8 qf[8];
#pragma unroll
  for (int ks = 0; ks < 8; ++ks) {
    uint4 u = make_uint4(0, 0, 0, 0);
    if (qrow < T) u = *reinterpret_cast<const uint4*>(q + ((size_t)qrow * Hq + head) * kD + 16 * ks + 8 * h);
    qf[ks] = __builtin_bit_cast(bf16x8, u);
  }

  f32x16 o[4] = {};
  float m = -INFINITY, lsum = 0.0f;

  // tile staging: K as 16-byte pieces (64 rows x 16) spread over the threads; V as
  // items (key pair kp: keys 2 kp, 2 kp + 1; dims 8 dq .. 8 dq + 7), written
  // transposed (key pairs per dword)
  constexpr int kNT = kAttnWaves * 64;
  constexpr int kKPer = 1024 / kNT, kVPer = 512 / kNT;
  uint4 kr[kKPer], vr[kVPer][2];
  auto load_tile = [&](int kt) {
#pragma unroll
    for (int i = 0; i < kKPer; ++i) {
      const int idx = tid + kNT * i, row = idx >> 4, c8 = idx & 15;
      const int key = 64 * kt + row;
      kr[i] = key < T ? *reinterpret_cast<const uint4*>(k + ((size_t)key * Hkv + kvh) * kD + c8 * 8)
                      : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int j = 0; j < kVPer; ++j) {
      const int item = tid + kNT * j, kp = item & 31, dq = item >> 5;
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        const int vkey = 64 * kt + 2 * kp + e;
        vr[j][e] = vkey < T ? *reinterpret_cast<const uint4*>(v + ((size_t)vkey * Hkv + kvh) * kD + dq * 8)
                            : make_uint4(0, 0, 0, 0);
      }
    }
  };
  load_tile(0);

  for (int kt = 0; kt < n_kt; ++kt) {
    __syncthreads();
#pragma unroll
    for (int i = 0; i < kKPer; ++i) {
      const int idx = tid + kNT * i, row = idx >> 4, c8 = idx & 15;
      *reinterpret_cast<uint4*>(Ks + row * kKPitch + c8 * 8) = kr[i];
    }
#pragma unroll
    for (int j = 0; j < kVPer; ++j) {
      const int item = tid + kNT * j, kp = item & 31, dq = item >> 5;
      const uint32_t a[4] = {vr[j][0].x, vr[j][0].y, vr[j][0].z, vr[j][0].w};
      const uint32_t b[4] = {vr[j][1].x, vr[j][1].y, vr[j][1].z, vr[j][1].w};
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        const uint32_t word = __builtin_amdgcn_perm(b[c >> 1], a[c >> 1], (c & 1) ? 0x07060302u : 0x05040100u);
        *reinterpret_cast<uint32_t*>(Vt + (8 * dq + c) * kVPitch + 2 * kp) = word;
      }
    }
    __syncthreads();
    if (kt + 1 < n_kt) load_tile(kt + 1);
    if (!active || kt >= wave_kt) continue;

    // issue priority: high while a wave feeds the matrix cores, low in its softmax,
    // so that a SIMD's other wave fills the gaps
    __builtin_amdgcn_s_setprio(1);
    // S^T: lane holds query qrow, keys 64 kt + 32 kk + 8 (r / 4) + 4 h + r % 4
    // the two 32-key halves as two interleaved MFMA chains; each step's K pieces
    // are read from LDS one step ahead
    f32x16 s[2] = {};
    const uint16_t* kb = Ks + li * kKPitch + 8 * h;
    uint4 ka0 = *reinterpret_cast<const uint4*>(kb);
    uint4 ka1 = *reinterpret_cast<const uint4*>(kb + 32 * kKPitch);
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) {
      uint4 kn0 = ka0, kn1 = ka1;
      if (ks + 1 < 8) {
        kn0 = *reinterpret_cast<const uint4*>(kb + 16 * (ks + 1));
        kn1 = *reinterpret_cast<const uint4*>(kb + 32 * kKPitch + 16 * (ks + 1));
      }
      s[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, ka0), qf[ks], s[0], 0, 0, 0);
      s[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, ka1), qf[ks], s[1], 0, 0, 0);
      ka0 = kn0;
      ka1 = kn1;
    }
    // keep the LDS reads one step ahead of the MFMAs that consume them
    __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
#pragma unroll
    for (int ks = 0; ks < 7; ++ks) {
      __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
      if (ks < 6) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
    __builtin_amdgcn_s_setprio(0);
    const bool edge = (causal && 64 * kt + 63 > qw0) || 64 * kt + 64 > T;
    float mt = -INFINITY;
    if (edge) {  // keys >= limit are masked
      const int limit = causal ? min(T, qrow + 1) : T;
#pragma unroll
      for (int kk = 0; kk < 2; ++kk)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = 64 * kt + 32 * kk + 8 * (r >> 2) + 4 * h + (r & 3);
          s[kk][r] = key < limit ? s[kk][r] : -INFINITY;
        }
    }
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
#pragma unroll
      for (int r = 0; r < 16; ++r) mt = fmaxf(mt, s[kk][r]);
    mt = fmaxf(mt, __shfl_xor(mt, 32, 64)) * scale_log2;  // finite: key 0 is visible to every query
    // The running maximum m (base-2 units) is raised only when a score exceeds it
    // by more than 8, so most tiles skip the rescale; probabilities stay <= 2^8.
    if (__ballot(mt > m + 8.0f)) {
      const float m_new = fmaxf(m, mt);
      const float alpha = __builtin_amdgcn_exp2f(m - m_new);
      m = m_new;
      lsum *= alpha;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[dt][r] *= alpha;
    }
    __builtin_amdgcn_s_setprio(1);
    float tsum = 0.0f;  // the tile's probabilities, added to the running sum once
    // V^T pieces for step (kk, u): dims 32 dt + l % 32, keys 32 kk + 16 u + 4 h + 0..3
    // and + 8; read one step ahead
    auto vload = [&](int kk, int u, uint4 (&va)[4]) {
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) {
        const uint16_t* vp = Vt + (32 * dt + li) * kVPitch + 32 * kk + 16 * u + 4 * h;
        const uint2 v0 = *reinterpret_cast<const uint2*>(vp);
        const uint2 v1 = *reinterpret_cast<const uint2*>(vp + 8);
        va[dt] = make_uint4(v0.x, v0.y, v1.x, v1.y);
      }
    };
    uint4 vcur[4], vnext[4];
    vload(0, 0, vcur);
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int step = 2 * kk + u;
        if (step + 1 < 4) vload((step + 1) >> 1, (step + 1) & 1, vnext);
        uint32_t hw[4], lw[4];
#pragma unroll
        for (int t2 = 0; t2 < 4; ++t2) {
          const float p0 = __builtin_amdgcn_exp2f(fmaf(s[kk][8 * u + 2 * t2], scale_log2, -m));
          const float p1 = __builtin_amdgcn_exp2f(fmaf(s[kk][8 * u + 2 * t2 + 1], scale_log2, -m));
          tsum += p0;
          tsum += p1;
          const bf16x2 hb = {(__bf16)p0, (__bf16)p1};
          hw[t2] = __builtin_bit_cast(uint32_t, hb);
          const bf16x2 lb = {(__bf16)(p0 - __uint_as_float(hw[t2] << 16)),
                             (__bf16)(p1 - __uint_as_float(hw[t2] & 0xffff0000u))};
          lw[t2] = __builtin_bit_cast(uint32_t, lb);
        }
        const bf16x8 phi = __builtin_bit_cast(bf16x8, make_uint4(hw[0], hw[1], hw[2], hw[3]));
        const bf16x8 plo = __builtin_bit_cast(bf16x8, make_uint4(lw[0], lw[1], lw[2], lw[3]));
#pragma unroll
        for (int dt = 0; dt < 4; ++dt)
          o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, vcur[dt]), phi, o[dt], 0, 0, 0);
#pragma unroll
        for (int dt = 0; dt < 4; ++dt)
          o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, vcur[dt]), plo, o[dt], 0, 0, 0);
#pragma unroll
        for (int dt = 0; dt < 4; ++dt) vcur[dt] = vnext[dt];
      }
    lsum += tsum;
    __builtin_amdgcn_s_setprio(0);
  }

  if (!active || qrow >= T) return;
  const float ltot = lsum + __shfl_xor(lsum, 32, 64);
  const float inv = 1.0f / ltot;
  float* orow = out + ((size_t)qrow * Hq + head) * kD;
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int r4 = 0; r4 < 4; ++r4) {
      const int dim = 32 * dt + 8 * r4 + 4 * h;
      *reinterpret_cast<float4*>(orow + dim) =
          make_float4(o[dt][4 * r4] * inv, o[dt][4 * r4 + 1] * inv, o[dt][4 * r4 + 2] * inv,
                      o[dt][4 * r4 + 3] * inv);
    }
}

// ---------------------------------------------------------------------------
// Symmetric eigen-decomposition by cyclic Jacobi (round-robin ordering), fp64.
// One block of 16 waves per matrix keeps the whole matrix in LDS (130 KB, both
// triangles: plain row-major addressing for the block updates).  A sweep is 127
// rounds of 64 disjoint pairs (p, q) (circle method: in round r the pairs are
// (127, r) and ((r + k) mod 127, (r - k) mod 127), k = 1..63), so every
// off-diagonal entry is visited once per sweep.  For each pair the rotation
// J (J_pp = J_qq = c, J_pq = s, J_qp = -s) with tau = (a_qq - a_pp) / (2 a_pq),
// t = sign(tau) / (|tau| + sqrt(1 + tau^2)), c = 1 / sqrt(1 + t^2), s = t c
// zeroes a_pq (Golub and Van Loan, symmetric Schur decomposition); the round
// applies A <- J^T A J as independent 2x2 block updates.  A pair is skipped when
// |a_pq| <= 1e-15 sqrt(|a_pp a_qq|); the sweeps stop when a sweep skips every
// pair (info = sweeps run, or -1 if max_sweeps did not converge).  The rounds' (c, s) are recorded; jacobi_vectors_kernel multiplies them
// into the eigenvectors afterwards (the vectors do not fit in LDS next to A).
// ---------------------------------------------------------------------------
constexpr int kJacRounds = kD - 1;
constexpr int kJacPairs = kD / 2;
constexpr int kJacPitch = kD + 2;  // doubles: rows of the LDS copy, 8 bytes of padding
constexpr int kJacBlocks = kJacPairs * (kJacPairs + 1) / 2;  // 2x2 blocks with k1 <= k2
constexpr double kJacTol = 1e-15;

__device__ inline void round_pair(int r, int kk, int& p, int& q) {
  int a, b;
  if (kk == 0) {
    a = kD - 1;
    b = r;
  } else {
    a = (r + kk) % kJacRounds;
    b = (r - kk + kJacRounds) % kJacRounds;
  }
  p = min(a, b);
  q = max(a, b);
}

constexpr int kJacThreads = 1024;  // 16 waves: the round's 2080 block updates, ~2 per thread
constexpr int kJacPerThread = (kJacBlocks + kJacThreads - 1) / kJacThreads;

__global__ __launch_bounds__(kJacThreads) void jacobi_kernel(const double* __restrict__ C, int max_sweeps,
                                                     double* __restrict__ diag,
                                                     double2* __restrict__ rot,
                                                     int* __restrict__ n_rounds,
                                                     int* __restrict__ info) {
  __shared__ double A[kD * kJacPitch];  // both triangles (130 KB)
  __shared__ double2 cs[kJacPairs];
  __shared__ int pp[kJacPairs], qq[kJacPairs];
  __shared__ int rotated;
  const int mtx = blockIdx.x, tid = threadIdx.x;
  const double* Cm = C + (size_t)mtx * kD * kD;
  for (int e = tid; e < kD * kD; e += kJacThreads) {
    const int i = e >> 7, j = e & (kD - 1);
    A[i * kJacPitch + j] = Cm[e];
  }
  // this thread's 2x2 blocks (k1 <= k2), fixed for every round
  int bk1[kJacPerThread], bk2[kJacPerThread];
#pragma unroll
  for (int n = 0; n < kJacPerThread; ++n) {
    const int b = tid + kJacThreads * n;
    int k1 = 0, rem = b;
    while (k1 < kJacPairs && rem >= kJacPairs - k1) {
      rem -= kJacPairs - k1;
      ++k1;
    }
    bk1[n] = b < kJacBlocks ? k1 : -1;
    bk2[n] = k1 + rem;
  }
  double2* rm = rot + (size_t)mtx * max_sweeps * kJacRounds * kJacPairs;
  int sweeps = 0, converged = 0;
  for (int sw = 0; sw < max_sweeps; ++sw) {
    __syncthreads();
    if (tid == 0) rotated = 0;
    for (int r = 0; r < kJacRounds; ++r) {
      __syncthreads();
      if (tid < kJacPairs) {
        int p, q;
        round_pair(r, tid, p, q);
        const double app = A[p * kJacPitch + p], aqq = A[q * kJacPitch + q];
        const double apq = A[p * kJacPitch + q];
        double c = 1.0, s = 0.0;
        if (apq != 0.0 && fabs(apq) > kJacTol * sqrt(fabs(app * aqq))) {
          const double tau = (aqq - app) / (2.0 * apq);
          const double t = (tau >= 0.0 ? 1.0 : -1.0) / (fabs(tau) + sqrt(1.0 + tau * tau));
          c = 1.0 / sqrt(1.0 + t * t);
          s = t * c;
          rotated = 1;
        }
        cs[tid] = make_double2(c, s);
        pp[tid] = p;
        qq[tid] = q;
        rm[((size_t)sw * kJacRounds + r) * kJacPairs + tid] = make_double2(c, s);
      }
      __syncthreads();
#pragma unroll
      for (int n = 0; n < kJacPerThread; ++n) {
        const int k1 = bk1[n], k2 = bk2[n];
        if (k1 < 0) continue;
        const double2 c1 = cs[k1], c2 = cs[k2];
        if (c1.y == 0.0 && c2.y == 0.0) continue;
        const int p1 = pp[k1], q1 = qq[k1], p2 = pp[k2], q2 = qq[k2];
        if (k1 == k2) {
          const double app = A[p1 * kJacPitch + p1], aqq = A[q1 * kJacPitch + q1];
          const double apq = A[p1 * kJacPitch + q1];
          const double c = c1.x, s = c1.y;
          // J^T M J with M symmetric; the off-diagonal entry is zero by construction
          const double t00 = c * app - s * apq, t01 = c * apq - s * aqq;
          const double t10 = s * app + c * apq, t11 = s * apq + c * aqq;
          A[p1 * kJacPitch + p1] = t00 * c - t01 * s;
          A[q1 * kJacPitch + q1] = t10 * s + t11 * c;
          A[p1 * kJacPitch + q1] = 0.0;
          A[q1 * kJacPitch + p1] = 0.0;
        } else {  // rows (p1, q1) x columns (p2, q2), mirrored to the transposed block
          const double m00 = A[p1 * kJacPitch + p2], m01 = A[p1 * kJacPitch + q2];
          const double m10 = A[q1 * kJacPitch + p2], m11 = A[q1 * kJacPitch + q2];
          const double t00 = c1.x * m00 - c1.y * m10, t01 = c1.x * m01 - c1.y * m11;
          const double t10 = c1.y * m00 + c1.x * m10, t11 = c1.y * m01 + c1.x * m11;
          const double n00 = t00 * c2.x - t01 * c2.y, n01 = t00 * c2.y + t01 * c2.x;
          const double n10 = t10 * c2.x - t11 * c2.y, n11 = t10 * c2.y + t11 * c2.x;
          A[p1 * kJacPitch + p2] = n00;
          A[p1 * kJacPitch + q2] = n01;
          A[q1 * kJacPitch + p2] = n10;
          A[q1 * kJacPitch + q2] = n11;
          A[p2 * kJacPitch + p1] = n00;
          A[q2 * kJacPitch + p1] = n01;
          A[p2 * kJacPitch + q1] = n10;
          A[q2 * kJacPitch + q1] = n11;
        }
      }
    }
    __syncthreads();
    if (!rotated) {  // a sweep without rotations: converged (its identity rounds are not kept)
      converged = 1;
      break;
    }
    sweeps = sw + 1;
  }
  __syncthreads();
  for (int i = tid; i < kD; i += kJacThreads) diag[(size_t)mtx * kD + i] = A[i * kJacPitch + i];
  if (tid == 0) {
    n_rounds[mtx] = sweeps * kJacRounds;
    info[mtx] = converged ? sweeps + 1 : -1;
  }
}

// V = J_1 J_2 ... J_R: each row of V evolves on its own (v <- v J), so one wave
// per row applies the recorded rounds to its row in LDS; lane k rotates pair k.
// The rounds' (c, s) are loaded 8 rounds ahead.
constexpr int kVecWaves = 4;
constexpr int kVecAhead = 8;

__global__ __launch_bounds__(kVecWaves * 64) void jacobi_vectors_kernel(
    const double2* __restrict__ rot, const int* __restrict__ n_rounds, int max_sweeps,
    int n_mats, double* __restrict__ V) {
  __shared__ double vr[kVecWaves][kD];
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  const int grow = blockIdx.x * kVecWaves + w;  // matrix * 128 + row
  if (grow >= n_mats * kD) return;            // whole wave
  const int mtx = grow / kD, row = grow % kD;
  vr[w][l] = l == row ? 1.0 : 0.0;
  vr[w][l + 64] = l + 64 == row ? 1.0 : 0.0;
  const int R = n_rounds[mtx];
  const double2* rm = rot + (size_t)mtx * max_sweeps * kJacRounds * kJacPairs;
  double2 buf[kVecAhead];
#pragma unroll
  for (int i = 0; i < kVecAhead; ++i) buf[i] = i < R ? rm[(size_t)i * kJacPairs + l] : make_double2(1.0, 0.0);
  for (int t0 = 0; t0 < R; t0 += kVecAhead) {
#pragma unroll
    for (int i = 0; i < kVecAhead; ++i) {
      const int t = t0 + i;
      if (t < R) {
        int p, q;
        round_pair(t % kJacRounds, l, p, q);
        const double2 c = buf[i];
        __builtin_amdgcn_wave_barrier();
        lane_exchange();
        const double vp = vr[w][p], vq = vr[w][q];
        vr[w][p] = c.x * vp - c.y * vq;
        vr[w][q] = c.y * vp + c.x * vq;
        __builtin_amdgcn_wave_barrier();
        lane_exchange();
        const int tn = t + kVecAhead;
        buf[i] = tn < R ? rm[(size_t)tn * kJacPairs + l] : make_double2(1.0, 0.0);
      }
    }
  }
  __builtin_amdgcn_wave_barrier();
  lane_exchange();
  double* vo = V + ((size_t)mtx * kD + row) * kD;
  vo[l] = vr[w][l];
  vo[l + 64] = vr[w][l + 64];
}

// Sort the eigenpairs by descending eigenvalue (ties: lower index first) and fix
// each eigenvector's sign so that its largest-magnitude entry (the first such)
// is positive.  One block of 128 threads per matrix; thread i moves column i.
__global__ __launch_bounds__(kD) void eig_finish_kernel(const double* __restrict__ diag,
                                                        const double* __restrict__ V,
                                                        double* __restrict__ lam,
                                                        double* __restrict__ U) {
  __shared__ double ls[kD];
  const int mtx = blockIdx.x, i = threadIdx.x;
  const double li = diag[(size_t)mtx * kD + i];
  ls[i] = li;
  __syncthreads();
  int rank = 0;
  for (int j = 0; j < kD; ++j) {
    const double lj = ls[j];
    rank += (lj > li || (lj == li && j < i)) ? 1 : 0;
  }
  lam[(size_t)mtx * kD + rank] = li;
  const double* Vm = V + (size_t)mtx * kD * kD;
  double best = -1.0, sgn = 1.0;
  for (int r = 0; r < kD; ++r) {
    const double x = Vm[r * kD + i];
    if (fabs(x) > best) {
      best = fabs(x);
      sgn = x < 0.0 ? -1.0 : 1.0;
    }
  }
  double* Um = U + (size_t)mtx * kD * kD;
  for (int r = 0; r < kD; ++r) Um[r * kD + rank] = sgn * Vm[r * kD + i];
}

// R = U H_Had P_br: R[i][j] = sum_c U[i][c] H[c][bitrev(j)] (P_br moves column k
// to bitrev(k); bit reversal is its own inverse), summed in ascending c with
// H[c][k] = (-1)^popcount(c & k) h, h = 1 divided by sqrt 2 seven times (the
// Sylvester recursion's normalization).  One thread per entry.
__global__ __launch_bounds__(256) void compose_kernel(const double* __restrict__ U,
                                                      double* __restrict__ R64,
                                                      float* __restrict__ R32) {
  const int mtx = blockIdx.y;
  const int e = blockIdx.x * 256 + threadIdx.x;
  const int i = e >> 7, j = e & (kD - 1);
  const int k = (int)(__brev((unsigned)j) >> 25);  // 7-bit reversal
  double hmag = 1.0;
  for (int lev = 1; lev < kD; lev <<= 1) hmag = hmag / sqrt(2.0);
  const double* Ui = U + ((size_t)mtx * kD + i) * kD;
  double acc = 0.0;
  for (int c = 0; c < kD; ++c) {
    const double hc = (__popc((unsigned)(c & k)) & 1) ? -hmag : hmag;
    acc = acc + Ui[c] * hc;
  }
  if (R64) R64[((size_t)mtx * kD + i) * kD + j] = acc;
  if (R32) R32[((size_t)mtx * kD + i) * kD + j] = (float)acc;
}

}  // namespace

// ---------------------------------------------------------------------------
// Launchers
// ---------------------------------------------------------------------------

int64_t gram_blocks(int64_t n_rows) {
  int64_t nb = (n_rows + kGramRows - 1) / kGramRows;
  const int64_t cap = 2 * (int64_t)device_cus();
  return nb < 1 ? 1 : nb > cap ? cap : nb;
}

size_t gram_partial_bytes(int64_t n_rows) {
  return (size_t)gram_blocks(n_rows) * kGramTiles * 1024 * sizeof(float);
}

hipError_t launch_gram(const void* X, int x_bf16, int64_t n_rows, double inv_n, float* partial,
                       double* C, hipStream_t st, int64_t rpt, int64_t tok_stride) {
  const int64_t nb = gram_blocks(n_rows);
  int64_t per = (n_rows + nb - 1) / nb;
  per = (per + kGramRows - 1) / kGramRows * kGramRows;
  if (x_bf16)
    hipLaunchKernelGGL(gram_kernel<true>, dim3((unsigned)nb), dim3(kGramWaves * 64), 0, st, X,
                       n_rows, per, rpt, tok_stride, partial);
  else
    hipLaunchKernelGGL(gram_kernel<false>, dim3((unsigned)nb), dim3(kGramWaves * 64), 0, st, X,
                       n_rows, per, rpt, tok_stride, partial);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(gram_reduce_kernel, dim3(kGramTiles * 1024 / 32), dim3(256), 0, st,
                     partial, (int)nb, inv_n, C);
  return hipGetLastError();
}

hipError_t launch_calib_attn(const uint16_t* q, const uint16_t* k, const uint16_t* v, int T,
                             int Hq, int Hkv, int causal, float* out, hipStream_t st) {
  const int g = Hq / Hkv;
  const int hc = g % 4 == 0 ? 4 : g % 2 == 0 ? 2 : 1;
  const int span = 32 * (kAttnWaves / hc);
  const int n_qtiles = (T + span - 1) / span;
  const float scale_log2 = (float)(1.4426950408889634 / sqrt((double)kD));
  hipLaunchKernelGGL(attn_kernel, dim3((unsigned)(Hq / hc), (unsigned)n_qtiles),
                     dim3(kAttnWaves * 64), 0, st, q, k, v, T, Hq, Hkv, hc, causal, scale_log2,
                     n_qtiles, out);
  return hipGetLastError();
}

size_t eig_rot_bytes(int n_mats, int max_sweeps) {
  return (size_t)n_mats * max_sweeps * kJacRounds * kJacPairs * sizeof(double2);
}

hipError_t launch_eig(const double* C, int n_mats, int max_sweeps, double* diag, double2* rot,
                      int* n_rounds, double* V, double* lam, double* U, int* info,
                      hipStream_t st) {
  hipLaunchKernelGGL(jacobi_kernel, dim3((unsigned)n_mats), dim3(kJacThreads), 0, st, C, max_sweeps,
                     diag, rot, n_rounds, info);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(jacobi_vectors_kernel, dim3((unsigned)((n_mats * kD + kVecWaves - 1) / kVecWaves)),
                     dim3(kVecWaves * 64), 0, st, rot, n_rounds, max_sweeps, n_mats, V);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(eig_finish_kernel, dim3((unsigned)n_mats), dim3(kD), 0, st, diag, V, lam, U);
  return hipGetLastError();
}

hipError_t launch_compose(const double* U, int n_mats, double* R64, float* R32, hipStream_t st) {
  hipLaunchKernelGGL(compose_kernel, dim3(kD * kD / 256, (unsigned)n_mats), dim3(256), 0, st, U,
                     R64, R32);
  return hipGetLastError();
}

}  // namespace oscar
