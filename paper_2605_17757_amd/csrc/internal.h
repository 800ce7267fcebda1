// Internal declarations shared by the liboscar host entry points and kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace oscar {

// Supported geometry: head dim 128, 64 token slots per page, groups of 32, 64 or
// 128 channels (ng = 128 / G = 4, 2 or 1 groups per head).
constexpr int kD = 128;
constexpr int kP = 64;
constexpr int kG = 32;                             // the default group size
constexpr int kCodeBytes = kP * kD / 4;            // one code region of a page-head block
constexpr int kOffKCodes = 0;
constexpr int kOffVCodes = kCodeBytes;             // 2048
constexpr int kOffKSz = 2 * kCodeBytes;            // 4096
// one (scale, zero) region, the V one's offset and the block size for ng groups
__host__ __device__ constexpr int sz_bytes(int ng) { return ng * kP * 4; }
__host__ __device__ constexpr int off_vsz(int ng) { return kOffKSz + sz_bytes(ng); }
__host__ __device__ constexpr int block_bytes(int ng) { return 2 * kCodeBytes + 2 * sz_bytes(ng); }
constexpr int kMaxGroupHeads = 16;                 // query heads per kv-head

// Lanes of one wave hand values to each other through LDS.  The hardware runs a
// wave's LDS operations in order, so no instruction is needed, but to the compiler
// each lane is a thread of its own: without a wavefront-scope fence between the
// writes and the reads it may move a lane's read of another lane's value above
// that lane's write.
__device__ inline void lane_exchange() { __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront"); }

// Split kernel geometry: a wave handles all query heads of its kv-head in chunks
// of 4, and the number of chunks sets its registers, hence the waves per CU.
inline int split_chunks(int heads_per_kv) { return (heads_per_kv + 3) / 4; }
inline int split_waves_per_cu(int nch) { return nch == 1 ? 16 : 8; }

// Workspace carving for decode (byte offsets, 256-aligned).
struct DecodeWs {
  size_t qt_off, po_off, pml_off, total;
};
inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }
inline DecodeWs decode_ws(int64_t B, int64_t Hq, int64_t S) {
  DecodeWs w;
  w.qt_off = 0;
  w.po_off = align256(w.qt_off + (size_t)(B * Hq) * kD * sizeof(float));
  w.pml_off = align256(w.po_off + (size_t)(B * Hq * S) * kD * sizeof(float));
  w.total = align256(w.pml_off + (size_t)(B * Hq * S) * 2 * sizeof(float));
  return w;
}

// Mixed-precision cache (bf16 sink [0, S0), INT2 history, bf16 window of W):
// the decode rows have row_stride = num_splits + 1 partial-state slots, the last
// one for the bf16 tokens.
struct MixedSpec {
  int S0, W, row_stride;
};

// Quantizer format (oscar_layout clip_mode / meta_dtype): scale and zero stored
// as bfloat16 instead of binary16; the token-wise quantile clip threshold
// instead of ratio x group absmax.
struct QuantFmt {
  int bf16;
  int quantile;
  int ng;   // groups per head (128 / G)
  int rph;  // one rotation matrix per KV head ([Hkv][128][128]) instead of one shared
};

// Query rows (b, head) = b * Hq + head, taken n per block: block bx takes rows
// bx * n + r in the natural order, or (rph) the rows of one KV head per block,
// kvh = bx % Hkv, local rows (bx / Hkv) * n + r enumerating (b, head in the KV
// head's group).  Returns the row, or -1 past the end.
__device__ inline int query_row(int bx, int r, int n, int rows, int Hq, int Hkv, int rph,
                                int& kvh) {
  if (!rph) {
    kvh = 0;
    const int idx = bx * n + r;
    return idx < rows ? idx : -1;
  }
  const int g = Hq / Hkv;
  kvh = bx % Hkv;
  const int idx = (bx / Hkv) * n + r;
  return idx < (rows / Hq) * g ? (idx / g) * Hq + kvh * g + idx % g : -1;
}
// Blocks of n query rows: natural order, or (rph) per KV head.
inline int query_blocks(int B, int Hq, int Hkv, int rph, int n) {
  return rph ? Hkv * ((B * (Hq / Hkv) + n - 1) / n) : (B * Hq + n - 1) / n;
}

// Kernel launchers (each returns the hipError_t of its launch).
// Rk or Rv nullptr: identity rotation.
hipError_t launch_append(void* pages, int64_t Hkv, const uint16_t* k, const uint16_t* v,
                         const int64_t* slots, int n_tok, const float* Rk, const float* Rv,
                         float clip_k, float clip_v, QuantFmt fmt, hipStream_t st);

hipError_t launch_decode_prepare(const uint16_t* q, int B, int Hq, const float* Rk,
                                 float qscale, float* qt, hipStream_t st, int rph = 0,
                                 int Hkv = 1);
// Cache update of n_tok tokens and query rotation in one launch (decode step prologue).
hipError_t launch_step_prologue(void* pages, int64_t Hkv, const uint16_t* k, const uint16_t* v,
                                const int64_t* slots, int n_tok, const float* Rk,
                                const float* Rv, float clip_k, float clip_v, QuantFmt fmt,
                                const uint16_t* q, int B, int Hq, float qscale, float* qt,
                                hipStream_t st);
// Mixed cache: prompt tokens routed to INT2 or the bf16 segment store by their
// position in a cache of length seq_lens[b].
hipError_t launch_mixed_append(void* pages, uint16_t* seg, int64_t Hkv, int S0, int W,
                               const uint16_t* k, const uint16_t* v, const int32_t* seq_idx,
                               const int64_t* pos, int n_tok, const int32_t* seq_lens,
                               const int32_t* block_table, int max_pages, const float* Rk,
                               const float* Rv, float clip_k, float clip_v, QuantFmt fmt,
                               hipStream_t st);
// Mixed cache decode-step prologue: one new token per sequence (sink, window with
// demotion of the oldest window token, or INT2) and the query rotation.
hipError_t launch_mixed_step_prologue(void* pages, uint16_t* seg, int64_t Hkv, int S0, int W,
                                      const uint16_t* k, const uint16_t* v,
                                      const int32_t* seq_lens, const int32_t* block_table,
                                      int max_pages, const float* Rk, const float* Rv,
                                      float clip_k, float clip_v, QuantFmt fmt, const uint16_t* q,
                                      int B, int Hq, float qscale, float* qt, hipStream_t st);
// Partial softmax state of the bf16 tokens (sink and window) of every (sequence,
// head) row, in the original basis, into slot num_splits of rows of num_splits + 1.
hipError_t launch_seg_partial(const uint16_t* seg, int Hkv, int S0, int W, int B, int Hq,
                              const int32_t* seq_lens, int max_pages, const uint16_t* q,
                              float qscale, int num_splits, float* part_o, float* part_ml,
                              hipStream_t st);
// mixed == nullptr: every token of a sequence is INT2 (rows of num_splits slots).
// meta_bf16: scale and zero stored as bfloat16; ng: groups per head.
hipError_t launch_decode_split(const uint8_t* pages, int Hkv, int B, int Hq,
                               const int32_t* block_table, int max_pages,
                               const int32_t* seq_lens, int num_splits, const float* qt,
                               float* part_o, float* part_ml, hipStream_t st, int meta_bf16,
                               int ng, const MixedSpec* mixed = nullptr);
// Balanced split kernel: split_waves_per_cu(chunks) * cus resident waves share
// the pages equally; a (sequence, head) row gets at most num_splits partial states.
hipError_t launch_decode_split_mfma(const uint8_t* pages, int Hkv, int B, int Hq,
                                    const int32_t* block_table, int max_pages,
                                    const int32_t* seq_lens, int num_splits, int cus,
                                    const float* qt, float* part_o, float* part_ml,
                                    hipStream_t st, int meta_bf16, int ng,
                                    const MixedSpec* mixed);
// One launch of the split kernel: its arguments and grid (blocks one-wave groups).
struct SplitLaunch {
  const uint8_t* pages;
  int Hkv, Hq;
  const int32_t* block_table;
  int max_pages;
  const int32_t* seq_lens;
  int num_splits, ranges, B;
  const float* qt;
  float* part_o;
  float* part_ml;
  int S0, W, row_stride;
  int64_t blocks;
  hipStream_t stream;
};
// The instances for 5 to 8 query heads per kv-head, compiled in a unit of their own
// (decode_mfma_wide2.hip) with another instruction scheduler.
void launch_split_two_chunk(const SplitLaunch& a, bool mixed, int meta_bf16, int ng);
int device_cus();  // compute units of the current device (cached)
// mixed != nullptr: rows of num_splits + 1 slots, the last one in the original
// basis (added after the back-rotation).
hipError_t launch_decode_reduce(int B, int Hq, int num_splits, const float* part_o,
                                const float* part_ml, const float* Rv, void* out, int out_f32,
                                hipStream_t st, const MixedSpec* mixed = nullptr, int rph = 0,
                                int Hkv = 1);

hipError_t launch_bf16_append(void* pages, int64_t Hkv, const uint16_t* k, const uint16_t* v,
                              const int64_t* slots, int n_tok, hipStream_t st);
hipError_t launch_bf16_split(const uint16_t* pages, int Hkv, int B, int Hq,
                             const int32_t* block_table, int max_pages,
                             const int32_t* seq_lens, int num_splits, const float* qt,
                             float* part_o, float* part_ml, hipStream_t st);

// Offline calibration.
// Waves per block of the calibration attention kernel (32 queries each); a block
// covers 32 * kCalibAttnWaves / hc queries of hc query heads.
constexpr int kCalibAttnWaves = 8;
// Second moment C = (X^T X) * inv_n of rows X [n_rows][128] (bf16 or fp32), fp64
// [128][128]; partial: gram_partial_bytes(n_rows) bytes of scratch.
size_t gram_partial_bytes(int64_t n_rows);
// Row r of X at element (r / rpt) * tok_stride + (r % rpt) * 128 (rpt = 1,
// tok_stride = 128: consecutive rows).
hipError_t launch_gram(const void* X, int x_bf16, int64_t n_rows, double inv_n, float* partial,
                       double* C, hipStream_t st, int64_t rpt = 1, int64_t tok_stride = kD);
// O[t][i] = softmax(q_{t,i} K_h^T / sqrt(d) + M) V_h (fp32 [T][Hq][128]).
hipError_t launch_calib_attn(const uint16_t* q, const uint16_t* k, const uint16_t* v, int T,
                             int Hq, int Hkv, int causal, float* out, hipStream_t st);
// Symmetric eigen-decomposition of n_mats matrices [128][128] (fp64): lam
// descending, U columns sign-fixed; scratch diag [n][128], rot eig_rot_bytes,
// n_rounds [n], V [n][128][128]; info [n] = sweeps run or -1.
size_t eig_rot_bytes(int n_mats, int max_sweeps);
hipError_t launch_eig(const double* C, int n_mats, int max_sweeps, double* diag, double2* rot,
                      int* n_rounds, double* V, double* lam, double* U, int* info,
                      hipStream_t st);
// R = U H_Had P_br for n_mats matrices (either output may be nullptr).
hipError_t launch_compose(const double* U, int n_mats, double* R64, float* R32, hipStream_t st);
// Mean squared quantization error of the rotated rows for each candidate clip
// ratio (n_cands <= 32) and the first minimizing candidate; partial: n_blocks x
// n_cands doubles, n_blocks = clip_blocks(n_rows).
// Rows x [n_rows / Hkv][Hkv][128]; with fmt.rph, R is [Hkv][128][128].
int clip_blocks(int64_t n_rows, int Hkv, int rph);
hipError_t launch_clip_errors(const uint16_t* x, int64_t n_rows, const float* R,
                              const float* cands, int n_cands, QuantFmt fmt, int Hkv,
                              double* partial, int n_blocks, double* err, float* best,
                              hipStream_t st);

}  // namespace oscar
