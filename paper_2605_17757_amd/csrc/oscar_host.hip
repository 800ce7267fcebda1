// liboscar C ABI: argument validation, workspace carving and kernel launches.
// Every entry point validates all host arguments before launching anything.
#include <math.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <atomic>
#include <mutex>
#include <vector>

#include "../../include/oscar.h"
#include "internal.h"

using namespace oscar;

namespace oscar {

int device_cus() {
  static std::atomic<int> cached{0};
  int v = cached.load(std::memory_order_relaxed);
  if (v > 0) return v;
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) == hipSuccess &&
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
      cus > 0)
    v = cus;
  else
    v = 256;
  cached.store(v, std::memory_order_relaxed);
  return v;
}

}  // namespace oscar

namespace {

constexpr float kLog2e = 1.4426950408889634f;

int check_layout(const oscar_layout* L) {
  if (!L) return OSCAR_ERR_INVALID_ARG;
  if (L->head_dim <= 0 || L->num_kv_heads <= 0 || L->page_size <= 0 || L->group_size <= 0 ||
      L->num_pages <= 0)
    return OSCAR_ERR_INVALID_ARG;
  if (L->head_dim % L->group_size != 0 || L->head_dim % 4 != 0) return OSCAR_ERR_INVALID_ARG;
  if (L->clip_mode != OSCAR_CLIP_GROUP_ABSMAX && L->clip_mode != OSCAR_CLIP_TOKEN_QUANTILE)
    return OSCAR_ERR_INVALID_ARG;
  if (L->meta_dtype != OSCAR_META_F16 && L->meta_dtype != OSCAR_META_BF16) return OSCAR_ERR_INVALID_ARG;
  if (L->rot_per_head != 0 && L->rot_per_head != 1) return OSCAR_ERR_INVALID_ARG;
  if (L->head_dim != kD || L->page_size != kP ||
      (L->group_size != 32 && L->group_size != 64 && L->group_size != 128))
    return OSCAR_ERR_UNSUPPORTED;
  if (L->num_kv_heads > 65535) return OSCAR_ERR_UNSUPPORTED;
  return OSCAR_OK;
}

bool clip_ok(float c) { return isfinite(c) && c > 0.0f && c <= 1.0f; }

int hip_status(hipError_t e) { return e == hipSuccess ? OSCAR_OK : OSCAR_ERR_HIP; }

// ---------------------------------------------------------------------------
// OSCAR_DEBUG (environment variable, read at every call; set and not "0"): the
// entry points that take device-resident indices synchronize the stream, copy
// the indices to host memory and check them before launching anything:
//   seq_lens[b] in [0, max_pages_per_seq * page_size], the block-table entries
//   of the pages a sequence uses (ceil(seq_lens[b] / page_size)) in
//   [0, num_pages), slots below num_pages * page_size (negative slots are
//   skipped by the cache update), seq_idx in [0, B).
// An index out of range returns OSCAR_ERR_INVALID_ARG with nothing launched; a
// failed copy (e.g. a host pointer) returns OSCAR_ERR_HIP.
// ---------------------------------------------------------------------------
bool debug_on() {
  const char* e = getenv("OSCAR_DEBUG");
  return e && e[0] && strcmp(e, "0") != 0;
}

template <class T>
int copy_to_host(std::vector<T>& h, const T* d, int64_t n) {
  h.resize((size_t)n);
  if (n == 0) return OSCAR_OK;
  return hip_status(hipMemcpy(h.data(), d, (size_t)n * sizeof(T), hipMemcpyDeviceToHost));
}

// Any of the index arrays may be null (not part of the call).
int debug_check(const oscar_layout* L, void* stream, int32_t B, const int32_t* block_table,
                int32_t max_pages_per_seq, const int32_t* seq_lens, const int64_t* slots,
                int64_t n_slots, const int32_t* seq_idx, int64_t n_idx) {
  if (!debug_on()) return OSCAR_OK;
  int st = hip_status(hipStreamSynchronize(static_cast<hipStream_t>(stream)));
  if (st) return st;
  const int64_t P = L->page_size;
  if (seq_lens) {
    std::vector<int32_t> lens, bt;
    if ((st = copy_to_host(lens, seq_lens, B))) return st;
    if (block_table && (st = copy_to_host(bt, block_table, (int64_t)B * max_pages_per_seq)))
      return st;
    for (int32_t b = 0; b < B; ++b) {
      const int64_t len = lens[(size_t)b];
      if (len < 0 || len > (int64_t)max_pages_per_seq * P) return OSCAR_ERR_INVALID_ARG;
      if (!block_table) continue;
      for (int64_t i = 0; i < (len + P - 1) / P; ++i) {
        const int32_t pg = bt[(size_t)b * max_pages_per_seq + (size_t)i];
        if (pg < 0 || pg >= L->num_pages) return OSCAR_ERR_INVALID_ARG;
      }
    }
  }
  if (slots) {
    std::vector<int64_t> sl;
    if ((st = copy_to_host(sl, slots, n_slots))) return st;
    for (int64_t s : sl)
      if (s >= L->num_pages * P) return OSCAR_ERR_INVALID_ARG;
  }
  if (seq_idx) {
    std::vector<int32_t> si;
    if ((st = copy_to_host(si, seq_idx, n_idx))) return st;
    for (int32_t x : si)
      if (x < 0 || x >= B) return OSCAR_ERR_INVALID_ARG;
  }
  return OSCAR_OK;
}

int check_decode_common(const oscar_layout* L, int32_t B, int32_t Hq, int32_t num_splits) {
  int st = check_layout(L);
  if (st) return st;
  if (B < 1 || Hq < 1 || num_splits < 1) return OSCAR_ERR_INVALID_ARG;
  if (Hq % L->num_kv_heads != 0) return OSCAR_ERR_INVALID_ARG;
  if (Hq / L->num_kv_heads > kMaxGroupHeads) return OSCAR_ERR_UNSUPPORTED;
  if (B > 65535) return OSCAR_ERR_UNSUPPORTED;
  return OSCAR_OK;
}

// Split count for num_splits == 0: >= 1, or -status for an invalid layout, or 0
// for an invalid max_pages_per_seq.
int32_t resolve_default_splits(const oscar_layout* L, int32_t B, int32_t Hq,
                               int32_t max_pages_per_seq) {
  const int ls = check_layout(L);
  if (ls) return -ls;
  if (max_pages_per_seq < 1) return 0;
  int64_t max_len = (int64_t)max_pages_per_seq * L->page_size;
  if (max_len > 0x7fffffffLL) max_len = 0x7fffffffLL;
  return oscar_default_num_splits(L, B, Hq, (int32_t)max_len);
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

QuantFmt quant_fmt(const oscar_layout* L) {
  return QuantFmt{L->meta_dtype == OSCAR_META_BF16 ? 1 : 0,
                  L->clip_mode == OSCAR_CLIP_TOKEN_QUANTILE ? 1 : 0, kD / L->group_size,
                  L->rot_per_head};
}
int meta_bf16(const oscar_layout* L) { return L->meta_dtype == OSCAR_META_BF16 ? 1 : 0; }
int groups(const oscar_layout* L) { return kD / L->group_size; }

// Mixed cache: sink and window sizes (and B, for the segment store size).
bool seg_ok(int32_t B, int32_t S0, int32_t W) {
  return B >= 1 && B <= 65535 && S0 >= 0 && W >= 0 && (int64_t)S0 + W <= 65536;
}
size_t seg_bytes(const oscar_layout* L, int32_t B, int32_t S0, int32_t W) {
  return (size_t)B * (size_t)L->num_kv_heads * 2 * (size_t)(S0 + W) * (size_t)L->head_dim * 2;
}

}  // namespace

extern "C" {

const char* oscar_status_string(int status) {
  switch (status) {
    case OSCAR_OK: return "OSCAR_OK";
    case OSCAR_ERR_INVALID_ARG: return "OSCAR_ERR_INVALID_ARG";
    case OSCAR_ERR_UNSUPPORTED: return "OSCAR_ERR_UNSUPPORTED";
    case OSCAR_ERR_WORKSPACE_TOO_SMALL: return "OSCAR_ERR_WORKSPACE_TOO_SMALL";
    case OSCAR_ERR_HIP: return "OSCAR_ERR_HIP";
    default: return "OSCAR_ERR_UNKNOWN";
  }
}

int oscar_layout_check(const oscar_layout* L) { return check_layout(L); }

size_t oscar_page_bytes(const oscar_layout* L) {
  if (check_layout(L) == OSCAR_ERR_INVALID_ARG) return 0;
  const size_t d = (size_t)L->head_dim, P = (size_t)L->page_size, G = (size_t)L->group_size;
  return (size_t)L->num_kv_heads * (2 * P * (d / 4) + 2 * (d / G) * P * 4);
}

size_t oscar_pool_bytes(const oscar_layout* L) {
  const size_t pb = oscar_page_bytes(L);
  return pb ? pb * (size_t)L->num_pages : 0;
}

size_t oscar_decode_workspace_bytes(const oscar_layout* L, int32_t B, int32_t Hq,
                                    int32_t num_splits) {
  if (check_decode_common(L, B, Hq, num_splits) != OSCAR_OK) return 0;
  return decode_ws(B, Hq, num_splits).total;
}

int32_t oscar_default_num_splits(const oscar_layout* L, int32_t B, int32_t Hq,
                                 int32_t max_seq_len) {
  if (check_layout(L) != OSCAR_OK || B < 1 || Hq < 1 || max_seq_len < 1) return 1;
  const int64_t pages = (max_seq_len + L->page_size - 1) / L->page_size;
  if (pages < 4) return 1;
  // The split kernel gives each of its resident waves (8 to 16 per CU, by the
  // query heads per kv-head) an equal share of all pages (ranges of >= 4 pages);
  // a (sequence, head) row is cut into at most num_splits pieces.  Assuming
  // sequences average half the longest, the range is ~B * Hkv * pages / 2 /
  // waves pages; allow one more piece than the longest sequence needs at that
  // range.
  const int chunks = (Hq % L->num_kv_heads == 0) ? split_chunks(Hq / L->num_kv_heads) : 1;
  const int64_t ranges = std::max<int64_t>(
      1, (int64_t)split_waves_per_cu(chunks) * device_cus() / L->num_kv_heads);
  int64_t range = ((int64_t)B * pages / 2 + ranges - 1) / ranges;
  if (range < 4) range = 4;
  int64_t s = (pages + range - 1) / range + 1;
  if (s > pages / 2) s = pages / 2;  // at least two pages per piece on average
  if (s < 2) s = 2;
  return (int32_t)s;
}

int oscar_kv_append(const oscar_layout* L, void* pages, const void* k_new, const void* v_new,
                    const int64_t* slot_mapping, int32_t n_tok, const float* R_k,
                    const float* R_v, float clip_k, float clip_v, void* stream) {
  int st = check_layout(L);
  if (st) return st;
  if (n_tok < 0 || !clip_ok(clip_k) || !clip_ok(clip_v)) return OSCAR_ERR_INVALID_ARG;
  if (n_tok == 0) return OSCAR_OK;
  if (!pages || !k_new || !v_new || !slot_mapping) return OSCAR_ERR_INVALID_ARG;
  if (!aligned(k_new, 4) || !aligned(v_new, 4) || !aligned(R_k, 16) || !aligned(R_v, 16) ||
      !aligned(pages, 16) || !aligned(slot_mapping, 8))
    return OSCAR_ERR_INVALID_ARG;
  if ((int64_t)n_tok * L->num_kv_heads > 0x7fffffffLL) return OSCAR_ERR_UNSUPPORTED;
  st = debug_check(L, stream, 0, nullptr, 0, nullptr, slot_mapping, n_tok, nullptr, 0);
  if (st) return st;
  return hip_status(launch_append(pages, L->num_kv_heads, static_cast<const uint16_t*>(k_new),
                                  static_cast<const uint16_t*>(v_new), slot_mapping, n_tok, R_k,
                                  R_v, clip_k, clip_v, quant_fmt(L),
                                  static_cast<hipStream_t>(stream)));
}

int oscar_decode_prepare(const oscar_layout* L, const void* q, int32_t B, int32_t Hq,
                         const float* R_k, float sm_scale, int32_t num_splits, void* workspace,
                         size_t workspace_bytes, void* stream) {
  int st = check_decode_common(L, B, Hq, num_splits);
  if (st) return st;
  if (!q || !workspace || !isfinite(sm_scale)) return OSCAR_ERR_INVALID_ARG;
  if (!aligned(workspace, 256) || !aligned(q, 4)) return OSCAR_ERR_INVALID_ARG;
  const DecodeWs ws = decode_ws(B, Hq, num_splits);
  if (workspace_bytes < ws.total) return OSCAR_ERR_WORKSPACE_TOO_SMALL;
  float* qt = reinterpret_cast<float*>(static_cast<uint8_t*>(workspace) + ws.qt_off);
  return hip_status(launch_decode_prepare(static_cast<const uint16_t*>(q), B, Hq, R_k,
                                          sm_scale * kLog2e, qt,
                                          static_cast<hipStream_t>(stream), L->rot_per_head,
                                          L->num_kv_heads));
}

int oscar_decode_split(const oscar_layout* L, const void* pages, int32_t B, int32_t Hq,
                       const int32_t* block_table, int32_t max_pages_per_seq,
                       const int32_t* seq_lens, int32_t num_splits, void* workspace,
                       size_t workspace_bytes, void* stream) {
  int st = check_decode_common(L, B, Hq, num_splits);
  if (st) return st;
  if (!pages || !block_table || !seq_lens || !workspace || max_pages_per_seq < 1)
    return OSCAR_ERR_INVALID_ARG;
  if (!aligned(workspace, 256) || !aligned(pages, 16)) return OSCAR_ERR_INVALID_ARG;
  const DecodeWs ws = decode_ws(B, Hq, num_splits);
  if (workspace_bytes < ws.total) return OSCAR_ERR_WORKSPACE_TOO_SMALL;
  st = debug_check(L, stream, B, block_table, max_pages_per_seq, seq_lens, nullptr, 0, nullptr, 0);
  if (st) return st;
  uint8_t* base = static_cast<uint8_t*>(workspace);
  return hip_status(launch_decode_split(
      static_cast<const uint8_t*>(pages), L->num_kv_heads, B, Hq, block_table, max_pages_per_seq,
      seq_lens, num_splits, reinterpret_cast<const float*>(base + ws.qt_off),
      reinterpret_cast<float*>(base + ws.po_off), reinterpret_cast<float*>(base + ws.pml_off),
      static_cast<hipStream_t>(stream), meta_bf16(L), groups(L)));
}

int oscar_decode_reduce(const oscar_layout* L, int32_t B, int32_t Hq, const float* R_v,
                        int32_t num_splits, void* workspace, size_t workspace_bytes, void* out,
                        oscar_dtype out_dtype, void* stream) {
  int st = check_decode_common(L, B, Hq, num_splits);
  if (st) return st;
  if (!workspace || !out) return OSCAR_ERR_INVALID_ARG;
  if (out_dtype != OSCAR_OUT_BF16 && out_dtype != OSCAR_OUT_F32) return OSCAR_ERR_INVALID_ARG;
  if (!aligned(workspace, 256) || !aligned(out, out_dtype == OSCAR_OUT_F32 ? 4 : 2))
    return OSCAR_ERR_INVALID_ARG;
  const DecodeWs ws = decode_ws(B, Hq, num_splits);
  if (workspace_bytes < ws.total) return OSCAR_ERR_WORKSPACE_TOO_SMALL;
  uint8_t* base = static_cast<uint8_t*>(workspace);
  return hip_status(launch_decode_reduce(B, Hq, num_splits,
                                         reinterpret_cast<const float*>(base + ws.po_off),
                                         reinterpret_cast<const float*>(base + ws.pml_off), R_v,
                                         out, out_dtype == OSCAR_OUT_F32 ? 1 : 0,
                                         static_cast<hipStream_t>(stream), nullptr,
                                         L->rot_per_head, L->num_kv_heads));
}

}  // extern "C"

namespace {

// Host-argument checks of oscar_decode_attn (all three stages), with num_splits
// == 0 resolved to the default; the workspace is checked separately.
int check_decode_attn(const oscar_layout* L, const void* pages, const void* q, int32_t B,
                      int32_t Hq, const int32_t* block_table, int32_t max_pages_per_seq,
                      const int32_t* seq_lens, float sm_scale, int32_t* num_splits,
                      const void* out, oscar_dtype out_dtype) {
  if (*num_splits < 0) return OSCAR_ERR_INVALID_ARG;
  if (*num_splits == 0) {
    *num_splits = resolve_default_splits(L, B, Hq, max_pages_per_seq);
    if (*num_splits < 1) return *num_splits == 0 ? OSCAR_ERR_INVALID_ARG : -*num_splits;
  }
  int st = check_decode_common(L, B, Hq, *num_splits);
  if (st) return st;
  if (!pages || !q || !block_table || !seq_lens || !out || max_pages_per_seq < 1 ||
      !isfinite(sm_scale))
    return OSCAR_ERR_INVALID_ARG;
  if (out_dtype != OSCAR_OUT_BF16 && out_dtype != OSCAR_OUT_F32) return OSCAR_ERR_INVALID_ARG;
  if (!aligned(pages, 16) || !aligned(q, 4) || !aligned(out, out_dtype == OSCAR_OUT_F32 ? 4 : 2))
    return OSCAR_ERR_INVALID_ARG;
  return OSCAR_OK;
}

}  // namespace

extern "C" {

int oscar_decode_attn(const oscar_layout* L, const void* pages, const void* q, int32_t B,
                      int32_t Hq, const int32_t* block_table, int32_t max_pages_per_seq,
                      const int32_t* seq_lens, const float* R_k, const float* R_v,
                      float sm_scale, int32_t num_splits, void* workspace,
                      size_t workspace_bytes, void* out, oscar_dtype out_dtype, void* stream) {
  // validate every argument of all three stages before launching any of them
  int st = check_decode_attn(L, pages, q, B, Hq, block_table, max_pages_per_seq, seq_lens,
                             sm_scale, &num_splits, out, out_dtype);
  if (st) return st;
  if (!workspace || !aligned(workspace, 256)) return OSCAR_ERR_INVALID_ARG;
  if (workspace_bytes < decode_ws(B, Hq, num_splits).total) return OSCAR_ERR_WORKSPACE_TOO_SMALL;
  st = debug_check(L, stream, B, block_table, max_pages_per_seq, seq_lens, nullptr, 0, nullptr, 0);
  if (st) return st;
  st = oscar_decode_prepare(L, q, B, Hq, R_k, sm_scale, num_splits, workspace, workspace_bytes,
                            stream);
  if (st) return st;
  st = oscar_decode_split(L, pages, B, Hq, block_table, max_pages_per_seq, seq_lens, num_splits,
                          workspace, workspace_bytes, stream);
  if (st) return st;
  return oscar_decode_reduce(L, B, Hq, R_v, num_splits, workspace, workspace_bytes, out,
                             out_dtype, stream);
}

int oscar_decode_step(const oscar_layout* L, void* pages, const void* k_new, const void* v_new,
                      const int64_t* slot_mapping, int32_t n_new, float clip_k, float clip_v,
                      const void* q, int32_t B, int32_t Hq, const int32_t* block_table,
                      int32_t max_pages_per_seq, const int32_t* seq_lens, const float* R_k,
                      const float* R_v, float sm_scale, int32_t num_splits, void* workspace,
                      size_t workspace_bytes, void* out, oscar_dtype out_dtype, void* stream) {
  // append arguments (as oscar_kv_append)
  int st = check_layout(L);
  if (st) return st;
  if (n_new < 0 || !clip_ok(clip_k) || !clip_ok(clip_v)) return OSCAR_ERR_INVALID_ARG;
  if (n_new > 0) {
    if (!k_new || !v_new || !slot_mapping) return OSCAR_ERR_INVALID_ARG;
    if (!aligned(k_new, 4) || !aligned(v_new, 4) || !aligned(slot_mapping, 8))
      return OSCAR_ERR_INVALID_ARG;
    if ((int64_t)n_new * L->num_kv_heads > 0x7fffffffLL) return OSCAR_ERR_UNSUPPORTED;
  }
  // decode arguments (as oscar_decode_attn)
  if (num_splits < 0) return OSCAR_ERR_INVALID_ARG;
  if (num_splits == 0) {
    num_splits = resolve_default_splits(L, B, Hq, max_pages_per_seq);
    if (num_splits < 1) return num_splits == 0 ? OSCAR_ERR_INVALID_ARG : -num_splits;
  }
  st = check_decode_common(L, B, Hq, num_splits);
  if (st) return st;
  if (!pages || !q || !block_table || !seq_lens || !workspace || !out ||
      max_pages_per_seq < 1 || !isfinite(sm_scale))
    return OSCAR_ERR_INVALID_ARG;
  if (out_dtype != OSCAR_OUT_BF16 && out_dtype != OSCAR_OUT_F32) return OSCAR_ERR_INVALID_ARG;
  if (!aligned(workspace, 256) || !aligned(pages, 16) || !aligned(q, 4) || !aligned(R_k, 16) ||
      !aligned(R_v, 16) || !aligned(out, out_dtype == OSCAR_OUT_F32 ? 4 : 2))
    return OSCAR_ERR_INVALID_ARG;
  const DecodeWs ws = decode_ws(B, Hq, num_splits);
  if (workspace_bytes < ws.total) return OSCAR_ERR_WORKSPACE_TOO_SMALL;
  st = debug_check(L, stream, B, block_table, max_pages_per_seq, seq_lens,
                   n_new > 0 ? slot_mapping : nullptr, n_new, nullptr, 0);
  if (st) return st;
  hipStream_t hs = static_cast<hipStream_t>(stream);
  uint8_t* base = static_cast<uint8_t*>(workspace);
  float* qt = reinterpret_cast<float*>(base + ws.qt_off);
  st = hip_status(launch_step_prologue(pages, L->num_kv_heads,
                                       static_cast<const uint16_t*>(k_new),
                                       static_cast<const uint16_t*>(v_new), slot_mapping, n_new,
                                       R_k, R_v, clip_k, clip_v, quant_fmt(L),
                                       static_cast<const uint16_t*>(q), B, Hq, sm_scale * kLog2e,
                                       qt, hs));
  if (st) return st;
  st = hip_status(launch_decode_split(
      static_cast<const uint8_t*>(pages), L->num_kv_heads, B, Hq, block_table, max_pages_per_seq,
      seq_lens, num_splits, qt, reinterpret_cast<float*>(base + ws.po_off),
      reinterpret_cast<float*>(base + ws.pml_off), hs, meta_bf16(L), groups(L)));
  if (st) return st;
  return hip_status(launch_decode_reduce(B, Hq, num_splits,
                                         reinterpret_cast<const float*>(base + ws.po_off),
                                         reinterpret_cast<const float*>(base + ws.pml_off), R_v,
                                         out, out_dtype == OSCAR_OUT_F32 ? 1 : 0, hs, nullptr,
                                         L->rot_per_head, L->num_kv_heads));
}

// ---------------------------------------------------------------------------
// mixed-precision cache
// ---------------------------------------------------------------------------

size_t oscar_seg_bytes(const oscar_layout* L, int32_t B, int32_t S0, int32_t W) {
  if (check_layout(L) != OSCAR_OK || !seg_ok(B, S0, W)) return 0;
  return seg_bytes(L, B, S0, W);
}

size_t oscar_mixed_workspace_bytes(const oscar_layout* L, int32_t B, int32_t Hq,
                                   int32_t num_splits) {
  if (check_decode_common(L, B, Hq, num_splits) != OSCAR_OK) return 0;
  return decode_ws(B, Hq, (int64_t)num_splits + 1).total;
}

int oscar_mixed_append(const oscar_layout* L, void* pages, void* seg, int32_t B, int32_t S0,
                       int32_t W, const void* k, const void* v, const int32_t* seq_idx,
                       const int64_t* pos, int32_t n_tok, const int32_t* block_table,
                       int32_t max_pages_per_seq, const int32_t* seq_lens, const float* R_k,
                       const float* R_v, float clip_k, float clip_v, void* stream) {
  int st = check_layout(L);
  if (st) return st;
  if (n_tok < 0 || B < 1 || !seg_ok(B, S0, W) || !clip_ok(clip_k) || !clip_ok(clip_v) ||
      max_pages_per_seq < 1)
    return OSCAR_ERR_INVALID_ARG;
  if (n_tok == 0) return OSCAR_OK;
  if (!pages || !k || !v || !seq_idx || !pos || !block_table || !seq_lens ||
      (S0 + W > 0 && !seg))
    return OSCAR_ERR_INVALID_ARG;
  if (!aligned(k, 4) || !aligned(v, 4) || !aligned(R_k, 16) || !aligned(R_v, 16) ||
      !aligned(pages, 16) || !aligned(pos, 8) || !aligned(seg, 16))
    return OSCAR_ERR_INVALID_ARG;
  if ((int64_t)n_tok * L->num_kv_heads > 0x7fffffffLL ||
      (int64_t)max_pages_per_seq * L->page_size > 0x7fffffffLL)
    return OSCAR_ERR_UNSUPPORTED;
  st = debug_check(L, stream, B, block_table, max_pages_per_seq, seq_lens, nullptr, 0, seq_idx,
                   n_tok);
  if (st) return st;
  return hip_status(launch_mixed_append(
      pages, static_cast<uint16_t*>(seg), L->num_kv_heads, S0, W, static_cast<const uint16_t*>(k),
      static_cast<const uint16_t*>(v), seq_idx, pos, n_tok, seq_lens, block_table,
      max_pages_per_seq, R_k, R_v, clip_k, clip_v, quant_fmt(L), static_cast<hipStream_t>(stream)));
}

namespace {

// Validation shared by the two mixed decode entry points; resolves num_splits.
int check_mixed_decode(const oscar_layout* L, const void* pages, const void* seg, int32_t S0,
                       int32_t W, const void* q, int32_t B, int32_t Hq,
                       const int32_t* block_table, int32_t max_pages_per_seq,
                       const int32_t* seq_lens, const float* R_k, const float* R_v,
                       float sm_scale, int32_t* num_splits, void* workspace,
                       size_t workspace_bytes, void* out, oscar_dtype out_dtype) {
  if (*num_splits < 0) return OSCAR_ERR_INVALID_ARG;
  if (*num_splits == 0) {
    const int32_t s = resolve_default_splits(L, B, Hq, max_pages_per_seq);
    if (s < 1) return s == 0 ? OSCAR_ERR_INVALID_ARG : -s;
    *num_splits = s;
  }
  int st = check_decode_common(L, B, Hq, *num_splits);
  if (st) return st;
  if (*num_splits > 0x3fffffff || !seg_ok(B, S0, W)) return OSCAR_ERR_INVALID_ARG;
  if (!pages || !q || !block_table || !seq_lens || !workspace || !out ||
      max_pages_per_seq < 1 || !isfinite(sm_scale) || (S0 + W > 0 && !seg))
    return OSCAR_ERR_INVALID_ARG;
  if ((int64_t)max_pages_per_seq * L->page_size > 0x7fffffffLL) return OSCAR_ERR_UNSUPPORTED;
  if (out_dtype != OSCAR_OUT_BF16 && out_dtype != OSCAR_OUT_F32) return OSCAR_ERR_INVALID_ARG;
  if (!aligned(workspace, 256) || !aligned(pages, 16) || !aligned(q, 4) || !aligned(R_k, 16) ||
      !aligned(R_v, 16) || !aligned(seg, 16) ||
      !aligned(out, out_dtype == OSCAR_OUT_F32 ? 4 : 2))
    return OSCAR_ERR_INVALID_ARG;
  if (workspace_bytes < decode_ws(B, Hq, (int64_t)*num_splits + 1).total)
    return OSCAR_ERR_WORKSPACE_TOO_SMALL;
  return OSCAR_OK;
}

// split (history), bf16 partial and merge of a mixed decode; qt already in the workspace
int launch_mixed_rest(const oscar_layout* L, const void* pages, const void* seg, int32_t S0,
                      int32_t W, const void* q, int32_t B, int32_t Hq, const int32_t* block_table,
                      int32_t max_pages_per_seq, const int32_t* seq_lens, const float* R_v,
                      float sm_scale, int32_t num_splits, void* workspace, void* out,
                      oscar_dtype out_dtype, hipStream_t hs) {
  const DecodeWs ws = decode_ws(B, Hq, (int64_t)num_splits + 1);
  uint8_t* base = static_cast<uint8_t*>(workspace);
  float* po = reinterpret_cast<float*>(base + ws.po_off);
  float* pml = reinterpret_cast<float*>(base + ws.pml_off);
  const MixedSpec mx{S0, W, num_splits + 1};
  int st = hip_status(launch_decode_split(static_cast<const uint8_t*>(pages), L->num_kv_heads, B,
                                          Hq, block_table, max_pages_per_seq, seq_lens,
                                          num_splits, reinterpret_cast<const float*>(base + ws.qt_off),
                                          po, pml, hs, meta_bf16(L), groups(L), &mx));
  if (st) return st;
  st = hip_status(launch_seg_partial(static_cast<const uint16_t*>(seg), L->num_kv_heads, S0, W, B,
                                     Hq, seq_lens, max_pages_per_seq,
                                     static_cast<const uint16_t*>(q), sm_scale * kLog2e,
                                     num_splits, po, pml, hs));
  if (st) return st;
  return hip_status(launch_decode_reduce(B, Hq, num_splits, po, pml, R_v, out,
                                         out_dtype == OSCAR_OUT_F32 ? 1 : 0, hs, &mx,
                                         L->rot_per_head, L->num_kv_heads));
}

}  // namespace

int oscar_decode_attn_mixed(const oscar_layout* L, const void* pages, const void* seg,
                            int32_t S0, int32_t W, const void* q, int32_t B, int32_t Hq,
                            const int32_t* block_table, int32_t max_pages_per_seq,
                            const int32_t* seq_lens, const float* R_k, const float* R_v,
                            float sm_scale, int32_t num_splits, void* workspace,
                            size_t workspace_bytes, void* out, oscar_dtype out_dtype,
                            void* stream) {
  int st = check_mixed_decode(L, pages, seg, S0, W, q, B, Hq, block_table, max_pages_per_seq,
                              seq_lens, R_k, R_v, sm_scale, &num_splits, workspace,
                              workspace_bytes, out, out_dtype);
  if (st) return st;
  st = debug_check(L, stream, B, block_table, max_pages_per_seq, seq_lens, nullptr, 0, nullptr, 0);
  if (st) return st;
  hipStream_t hs = static_cast<hipStream_t>(stream);
  const DecodeWs ws = decode_ws(B, Hq, (int64_t)num_splits + 1);
  float* qt = reinterpret_cast<float*>(static_cast<uint8_t*>(workspace) + ws.qt_off);
  st = hip_status(launch_decode_prepare(static_cast<const uint16_t*>(q), B, Hq, R_k,
                                        sm_scale * kLog2e, qt, hs,
                                        L->rot_per_head, L->num_kv_heads));
  if (st) return st;
  return launch_mixed_rest(L, pages, seg, S0, W, q, B, Hq, block_table, max_pages_per_seq,
                           seq_lens, R_v, sm_scale, num_splits, workspace, out, out_dtype, hs);
}

int oscar_decode_step_mixed(const oscar_layout* L, void* pages, void* seg, int32_t S0,
                            int32_t W, const void* k_new, const void* v_new, float clip_k,
                            float clip_v, const void* q, int32_t B, int32_t Hq,
                            const int32_t* block_table, int32_t max_pages_per_seq,
                            const int32_t* seq_lens, const float* R_k, const float* R_v,
                            float sm_scale, int32_t num_splits, void* workspace,
                            size_t workspace_bytes, void* out, oscar_dtype out_dtype,
                            void* stream) {
  int st = check_mixed_decode(L, pages, seg, S0, W, q, B, Hq, block_table, max_pages_per_seq,
                              seq_lens, R_k, R_v, sm_scale, &num_splits, workspace,
                              workspace_bytes, out, out_dtype);
  if (st) return st;
  st = debug_check(L, stream, B, block_table, max_pages_per_seq, seq_lens, nullptr, 0, nullptr, 0);
  if (st) return st;
  if (!k_new || !v_new || !clip_ok(clip_k) || !clip_ok(clip_v)) return OSCAR_ERR_INVALID_ARG;
  if (!aligned(k_new, 4) || !aligned(v_new, 4)) return OSCAR_ERR_INVALID_ARG;
  if ((int64_t)B * L->num_kv_heads > 0x7fffffffLL) return OSCAR_ERR_UNSUPPORTED;
  hipStream_t hs = static_cast<hipStream_t>(stream);
  const DecodeWs ws = decode_ws(B, Hq, (int64_t)num_splits + 1);
  float* qt = reinterpret_cast<float*>(static_cast<uint8_t*>(workspace) + ws.qt_off);
  st = hip_status(launch_mixed_step_prologue(
      pages, static_cast<uint16_t*>(seg), L->num_kv_heads, S0, W,
      static_cast<const uint16_t*>(k_new), static_cast<const uint16_t*>(v_new), seq_lens,
      block_table, max_pages_per_seq, R_k, R_v, clip_k, clip_v, quant_fmt(L),
      static_cast<const uint16_t*>(q), B, Hq, sm_scale * kLog2e, qt, hs));
  if (st) return st;
  return launch_mixed_rest(L, pages, seg, S0, W, q, B, Hq, block_table, max_pages_per_seq,
                           seq_lens, R_v, sm_scale, num_splits, workspace, out, out_dtype, hs);
}

// ---------------------------------------------------------------------------
// bf16 baseline
// ---------------------------------------------------------------------------

size_t oscar_bf16_page_bytes(const oscar_layout* L) {
  if (check_layout(L) == OSCAR_ERR_INVALID_ARG) return 0;
  return (size_t)L->num_kv_heads * 2 * (size_t)L->page_size * (size_t)L->head_dim * 2;
}

int oscar_bf16_kv_append(const oscar_layout* L, void* pages, const void* k_new,
                         const void* v_new, const int64_t* slot_mapping, int32_t n_tok,
                         void* stream) {
  int st = check_layout(L);
  if (st) return st;
  if (n_tok < 0) return OSCAR_ERR_INVALID_ARG;
  if (n_tok == 0) return OSCAR_OK;
  if (!pages || !k_new || !v_new || !slot_mapping) return OSCAR_ERR_INVALID_ARG;
  if (!aligned(pages, 16) || !aligned(k_new, 4) || !aligned(v_new, 4)) return OSCAR_ERR_INVALID_ARG;
  st = debug_check(L, stream, 0, nullptr, 0, nullptr, slot_mapping, n_tok, nullptr, 0);
  if (st) return st;
  return hip_status(launch_bf16_append(pages, L->num_kv_heads,
                                       static_cast<const uint16_t*>(k_new),
                                       static_cast<const uint16_t*>(v_new), slot_mapping, n_tok,
                                       static_cast<hipStream_t>(stream)));
}

size_t oscar_bf16_decode_workspace_bytes(const oscar_layout* L, int32_t B, int32_t Hq,
                                         int32_t num_splits) {
  return oscar_decode_workspace_bytes(L, B, Hq, num_splits);
}

int oscar_bf16_decode_attn(const oscar_layout* L, const void* pages, const void* q, int32_t B,
                           int32_t Hq, const int32_t* block_table, int32_t max_pages_per_seq,
                           const int32_t* seq_lens, float sm_scale, int32_t num_splits,
                           void* workspace, size_t workspace_bytes, void* out,
                           oscar_dtype out_dtype, void* stream) {
  if (num_splits < 0) return OSCAR_ERR_INVALID_ARG;
  if (num_splits == 0) {
    num_splits = resolve_default_splits(L, B, Hq, max_pages_per_seq);
    if (num_splits < 1) return num_splits == 0 ? OSCAR_ERR_INVALID_ARG : -num_splits;
  }
  int st = check_decode_common(L, B, Hq, num_splits);
  if (st) return st;
  if (!pages || !q || !block_table || !seq_lens || !workspace || !out || max_pages_per_seq < 1 ||
      !isfinite(sm_scale))
    return OSCAR_ERR_INVALID_ARG;
  if (out_dtype != OSCAR_OUT_BF16 && out_dtype != OSCAR_OUT_F32) return OSCAR_ERR_INVALID_ARG;
  if (!aligned(workspace, 256) || !aligned(pages, 16) || !aligned(q, 4) ||
      !aligned(out, out_dtype == OSCAR_OUT_F32 ? 4 : 2))
    return OSCAR_ERR_INVALID_ARG;
  const DecodeWs ws = decode_ws(B, Hq, num_splits);
  if (workspace_bytes < ws.total) return OSCAR_ERR_WORKSPACE_TOO_SMALL;
  st = debug_check(L, stream, B, block_table, max_pages_per_seq, seq_lens, nullptr, 0, nullptr, 0);
  if (st) return st;
  uint8_t* base = static_cast<uint8_t*>(workspace);
  float* qt = reinterpret_cast<float*>(base + ws.qt_off);
  float* po = reinterpret_cast<float*>(base + ws.po_off);
  float* pml = reinterpret_cast<float*>(base + ws.pml_off);
  hipStream_t s = static_cast<hipStream_t>(stream);
  // q scaled by sm_scale*log2 e, no rotation (R = I); reduce with R = I
  st = hip_status(launch_decode_prepare(static_cast<const uint16_t*>(q), B, Hq, nullptr,
                                        sm_scale * kLog2e, qt, s));
  if (st) return st;
  st = hip_status(launch_bf16_split(static_cast<const uint16_t*>(pages), L->num_kv_heads, B, Hq,
                                    block_table, max_pages_per_seq, seq_lens, num_splits, qt, po,
                                    pml, s));
  if (st) return st;
  return hip_status(launch_decode_reduce(B, Hq, num_splits, po, pml, nullptr, out,
                                         out_dtype == OSCAR_OUT_F32 ? 1 : 0, s));
}

}  // extern "C"

// ---------------------------------------------------------------------------
// Offline calibration
// ---------------------------------------------------------------------------

namespace {

constexpr int kCalibMaxSweeps = OSCAR_CALIB_MAX_SWEEPS;

int check_calib(int64_t T, int32_t Hq, int32_t Hkv) {
  if (T < 1 || Hkv < 1 || Hq < Hkv || Hq % Hkv != 0) return OSCAR_ERR_INVALID_ARG;
  const int64_t g = Hq / Hkv;
  const int64_t hc = g % 4 == 0 ? 4 : g % 2 == 0 ? 2 : 1;
  const int64_t span = 32 * kCalibAttnWaves / hc;
  if ((T + span - 1) / span > 65535 || Hq / hc > 65535) return OSCAR_ERR_UNSUPPORTED;
  return OSCAR_OK;
}

struct CalibWs {
  size_t o_off, part_off, total;
};
CalibWs calib_ws(int64_t T, int32_t Hq) {
  CalibWs w;
  w.o_off = 0;
  w.part_off = align256((size_t)T * Hq * kD * sizeof(float));
  w.total = align256(w.part_off + gram_partial_bytes(T * Hq));
  return w;
}

struct RotWs {
  size_t diag_off, rot_off, rounds_off, v_off, info_off, total;
};
RotWs rot_ws(int32_t n) {
  RotWs w;
  w.diag_off = 0;
  w.rot_off = align256(w.diag_off + (size_t)n * kD * sizeof(double));
  w.rounds_off = align256(w.rot_off + eig_rot_bytes(n, kCalibMaxSweeps));
  w.v_off = align256(w.rounds_off + (size_t)n * sizeof(int));
  w.info_off = align256(w.v_off + (size_t)n * kD * kD * sizeof(double));
  w.total = align256(w.info_off + (size_t)n * sizeof(int));
  return w;
}

size_t clip_ws_bytes(int64_t n_rows, int32_t Hkv, int32_t n_cands) {
  // enough partials for either block schedule (shared or per-head rotation)
  const int nb = std::max(clip_blocks(n_rows, Hkv, 0), clip_blocks(n_rows, Hkv, 1));
  return align256((size_t)nb * n_cands * sizeof(double));
}

bool cands_shape_ok(int32_t n_cands) { return n_cands >= 1 && n_cands <= OSCAR_CALIB_MAX_CANDS; }

struct LayerWs {
  size_t c_off, calib_off, rot_off, lam_off, u_off, clip_off, err_off, info_off, total;
};
// nm = 2 (C_Q, C_S) shared, or 2 Hkv with one rotation per KV head.
LayerWs layer_ws(int64_t T, int32_t Hq, int32_t Hkv, int32_t n_cands, int32_t nm) {
  LayerWs w;
  w.c_off = 0;
  w.calib_off = align256((size_t)nm * kD * kD * sizeof(double));
  w.rot_off = align256(w.calib_off + calib_ws(T, Hq).total);
  w.lam_off = align256(w.rot_off + rot_ws(nm).total);
  w.u_off = align256(w.lam_off + (size_t)nm * kD * sizeof(double));
  w.clip_off = align256(w.u_off + (size_t)nm * kD * kD * sizeof(double));
  w.err_off = align256(w.clip_off + clip_ws_bytes(T * Hkv, Hkv, n_cands));
  w.info_off = align256(w.err_off + 2 * (size_t)n_cands * sizeof(double));
  w.total = align256(w.info_off + (size_t)nm * sizeof(int));
  return w;
}

// C_Q over all query heads (Hkv_mats = 1), or one per KV head over its g query
// heads (Hkv_mats = Hkv: C + h d^2 for head h).
int query_cov_impl(const void* q, int64_t T, int32_t Hq, int32_t Hkv, int32_t Hkv_mats,
                   double* C, char* ws, hipStream_t st) {
  const CalibWs w = calib_ws(T, Hq);
  const int64_t g = Hq / Hkv_mats;  // query heads per matrix
  for (int h = 0; h < Hkv_mats; ++h) {
    const uint16_t* x = static_cast<const uint16_t*>(q) + (size_t)h * g * kD;
    const int rc = hip_status(launch_gram(x, 1, T * g, 1.0 / ((double)T * g),
                                          reinterpret_cast<float*>(ws + w.part_off),
                                          C + (size_t)h * kD * kD, st, g, (int64_t)Hq * kD));
    if (rc) return rc;
  }
  (void)Hkv;
  return OSCAR_OK;
}

int score_cov_impl(const void* q, const void* k, const void* v, int64_t T, int32_t Hq,
                   int32_t Hkv, int32_t Hkv_mats, int32_t causal, double* C, char* ws,
                   hipStream_t st) {
  const CalibWs w = calib_ws(T, Hq);
  float* O = reinterpret_cast<float*>(ws + w.o_off);
  hipError_t e = launch_calib_attn(static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k),
                                   static_cast<const uint16_t*>(v), (int)T, Hq, Hkv, causal ? 1 : 0,
                                   O, st);
  if (e != hipSuccess) return OSCAR_ERR_HIP;
  const int64_t g = Hq / Hkv_mats;
  for (int h = 0; h < Hkv_mats; ++h) {
    const int rc = hip_status(launch_gram(O + (size_t)h * g * kD, 0, T * g, 1.0 / ((double)T * g),
                                          reinterpret_cast<float*>(ws + w.part_off),
                                          C + (size_t)h * kD * kD, st, g, (int64_t)Hq * kD));
    if (rc) return rc;
  }
  return OSCAR_OK;
}

int rotation_impl(const double* C, int32_t n, double* lam, double* U, double* R64, float* R32,
                  int32_t* info, char* ws, hipStream_t st) {
  const RotWs w = rot_ws(n);
  int* inf = info ? info : reinterpret_cast<int*>(ws + w.info_off);
  hipError_t e = launch_eig(C, n, kCalibMaxSweeps, reinterpret_cast<double*>(ws + w.diag_off),
                            reinterpret_cast<double2*>(ws + w.rot_off),
                            reinterpret_cast<int*>(ws + w.rounds_off),
                            reinterpret_cast<double*>(ws + w.v_off), lam, U, inf, st);
  if (e != hipSuccess) return OSCAR_ERR_HIP;
  return hip_status(launch_compose(U, n, R64, R32, st));
}

bool cands_values_ok(const float* cands, int32_t n) {
  // candidate ratios live on the device; only their count is checked here
  return cands != nullptr && n >= 1;
}

}  // namespace

extern "C" {

size_t oscar_calib_workspace_bytes(int64_t T, int32_t Hq, int32_t Hkv) {
  if (check_calib(T, Hq, Hkv) != OSCAR_OK) return 0;
  return calib_ws(T, Hq).total;
}

int oscar_calib_query_cov(const void* q, int64_t T, int32_t Hq, int32_t Hkv, double* C,
                          void* workspace, size_t workspace_bytes, void* stream) {
  int st = check_calib(T, Hq, Hkv);
  if (st) return st;
  if (!q || !C || !workspace || !aligned(q, 16) || !aligned(C, 8) || !aligned(workspace, 256))
    return OSCAR_ERR_INVALID_ARG;
  if (workspace_bytes < calib_ws(T, Hq).total) return OSCAR_ERR_WORKSPACE_TOO_SMALL;
  return query_cov_impl(q, T, Hq, Hkv, 1, C, static_cast<char*>(workspace),
                        static_cast<hipStream_t>(stream));
}

int oscar_calib_attn(const void* q, const void* k, const void* v, int64_t T, int32_t Hq,
                     int32_t Hkv, int32_t causal, float* out, void* stream) {
  int st = check_calib(T, Hq, Hkv);
  if (st) return st;
  if (!q || !k || !v || !out || !aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) ||
      !aligned(out, 16))
    return OSCAR_ERR_INVALID_ARG;
  return hip_status(launch_calib_attn(static_cast<const uint16_t*>(q),
                                      static_cast<const uint16_t*>(k),
                                      static_cast<const uint16_t*>(v), (int)T, Hq, Hkv,
                                      causal ? 1 : 0, out, static_cast<hipStream_t>(stream)));
}

int oscar_calib_score_cov(const void* q, const void* k, const void* v, int64_t T, int32_t Hq,
                          int32_t Hkv, int32_t causal, double* C, void* workspace,
                          size_t workspace_bytes, void* stream) {
  int st = check_calib(T, Hq, Hkv);
  if (st) return st;
  if (!q || !k || !v || !C || !workspace || !aligned(q, 16) || !aligned(k, 16) ||
      !aligned(v, 16) || !aligned(C, 8) || !aligned(workspace, 256))
    return OSCAR_ERR_INVALID_ARG;
  if (workspace_bytes < calib_ws(T, Hq).total) return OSCAR_ERR_WORKSPACE_TOO_SMALL;
  return score_cov_impl(q, k, v, T, Hq, Hkv, 1, causal, C, static_cast<char*>(workspace),
                        static_cast<hipStream_t>(stream));
}

size_t oscar_calib_rotation_workspace_bytes(int32_t n_mats) {
  if (n_mats < 1 || n_mats > 65535) return 0;
  return rot_ws(n_mats).total;
}

int oscar_calib_rotation(const double* C, int32_t n_mats, double* lam, double* U, double* R64,
                         float* R32, int32_t* info, void* workspace, size_t workspace_bytes,
                         void* stream) {
  if (n_mats < 1 || !C || !lam || !U || !workspace) return OSCAR_ERR_INVALID_ARG;
  if (n_mats > 65535) return OSCAR_ERR_UNSUPPORTED;
  if (!aligned(C, 8) || !aligned(lam, 8) || !aligned(U, 8) || !aligned(R64, 8) ||
      !aligned(R32, 4) || !aligned(info, 4) || !aligned(workspace, 256))
    return OSCAR_ERR_INVALID_ARG;
  if (workspace_bytes < rot_ws(n_mats).total) return OSCAR_ERR_WORKSPACE_TOO_SMALL;
  return rotation_impl(C, n_mats, lam, U, R64, R32, info, static_cast<char*>(workspace),
                       static_cast<hipStream_t>(stream));
}

size_t oscar_calib_clip_workspace_bytes(int64_t n_tok, int32_t Hkv, int32_t n_cands) {
  if (n_tok < 1 || Hkv < 1 || !cands_shape_ok(n_cands)) return 0;
  if (n_tok * Hkv > 0x7fffffffLL) return 0;
  return clip_ws_bytes(n_tok * Hkv, Hkv, n_cands);
}

int oscar_calib_clip(const oscar_layout* L, const void* x, int64_t n_tok, const float* R,
                     const float* cands, int32_t n_cands, double* err, float* best,
                     void* workspace, size_t workspace_bytes, void* stream) {
  int st = check_layout(L);
  if (st) return st;
  if (n_tok < 1 || !x || !err || !workspace || !cands_values_ok(cands, n_cands))
    return OSCAR_ERR_INVALID_ARG;
  if (!cands_shape_ok(n_cands)) return OSCAR_ERR_UNSUPPORTED;
  if (n_tok * L->num_kv_heads > 0x7fffffffLL) return OSCAR_ERR_UNSUPPORTED;
  if (!aligned(x, 4) || !aligned(R, 16) || !aligned(cands, 4) || !aligned(err, 8) ||
      !aligned(best, 4) || !aligned(workspace, 256))
    return OSCAR_ERR_INVALID_ARG;
  const int64_t rows = n_tok * L->num_kv_heads;
  if (workspace_bytes < clip_ws_bytes(rows, L->num_kv_heads, n_cands))
    return OSCAR_ERR_WORKSPACE_TOO_SMALL;
  return hip_status(launch_clip_errors(static_cast<const uint16_t*>(x), rows, R, cands, n_cands,
                                       quant_fmt(L), L->num_kv_heads,
                                       static_cast<double*>(workspace),
                                       clip_blocks(rows, L->num_kv_heads, L->rot_per_head), err,
                                       best, static_cast<hipStream_t>(stream)));
}

size_t oscar_calibrate_layer_workspace_bytes(const oscar_layout* L, int64_t T, int32_t Hq,
                                             int32_t n_cands) {
  if (check_layout(L) != OSCAR_OK) return 0;
  const int32_t Hkv = L->num_kv_heads;
  if (check_calib(T, Hq, Hkv) != OSCAR_OK || !cands_shape_ok(n_cands)) return 0;
  if (T * Hkv > 0x7fffffffLL) return 0;
  return layer_ws(T, Hq, Hkv, n_cands, L->rot_per_head ? 2 * Hkv : 2).total;
}

int oscar_calibrate_layer(const oscar_layout* L, const void* q, const void* k, const void* v,
                          int64_t T, int32_t Hq, int32_t causal, const float* cands,
                          int32_t n_cands, float* R_k, float* R_v, float* clip, double* lam,
                          int32_t* info, void* workspace, size_t workspace_bytes,
                          void* stream) {
  int st = check_layout(L);
  if (st) return st;
  const int32_t Hkv = L->num_kv_heads;
  st = check_calib(T, Hq, Hkv);
  if (st) return st;
  if (!q || !k || !v || !R_k || !R_v || !clip || !workspace || !cands_values_ok(cands, n_cands))
    return OSCAR_ERR_INVALID_ARG;
  if (!cands_shape_ok(n_cands)) return OSCAR_ERR_UNSUPPORTED;
  if (T * Hkv > 0x7fffffffLL) return OSCAR_ERR_UNSUPPORTED;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(R_k, 16) ||
      !aligned(R_v, 16) || !aligned(clip, 4) || !aligned(lam, 8) || !aligned(info, 4) ||
      !aligned(cands, 4) || !aligned(workspace, 256))
    return OSCAR_ERR_INVALID_ARG;
  const int32_t hm = L->rot_per_head ? Hkv : 1;  // matrices per tensor
  const LayerWs w = layer_ws(T, Hq, Hkv, n_cands, 2 * hm);
  if (workspace_bytes < w.total) return OSCAR_ERR_WORKSPACE_TOO_SMALL;
  char* ws = static_cast<char*>(workspace);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const size_t dd = (size_t)kD * kD;
  double* C = reinterpret_cast<double*>(ws + w.c_off);  // [2][hm][d][d]: C_Q, C_S
  double* lm = lam ? lam : reinterpret_cast<double*>(ws + w.lam_off);
  double* U = reinterpret_cast<double*>(ws + w.u_off);
  int32_t* inf = info ? info : reinterpret_cast<int32_t*>(ws + w.info_off);
  double* err = reinterpret_cast<double*>(ws + w.err_off);
  char* cw = ws + w.calib_off;
  if ((st = query_cov_impl(q, T, Hq, Hkv, hm, C, cw, s))) return st;
  if ((st = score_cov_impl(q, k, v, T, Hq, Hkv, hm, causal, C + hm * dd, cw, s))) return st;
  // R_k and R_v are adjacent only through the caller's pointers: compose each
  if ((st = rotation_impl(C, 2 * hm, lm, U, nullptr, nullptr, inf, ws + w.rot_off, s))) return st;
  if (launch_compose(U, hm, nullptr, R_k, s) != hipSuccess) return OSCAR_ERR_HIP;
  if (launch_compose(U + hm * dd, hm, nullptr, R_v, s) != hipSuccess) return OSCAR_ERR_HIP;
  const QuantFmt fmt = quant_fmt(L);
  const int64_t rows = T * Hkv;
  const int nb = clip_blocks(rows, Hkv, L->rot_per_head);
  double* part = reinterpret_cast<double*>(ws + w.clip_off);
  if (launch_clip_errors(static_cast<const uint16_t*>(k), rows, R_k, cands, n_cands, fmt, Hkv, part,
                         nb, err, clip, s) != hipSuccess)
    return OSCAR_ERR_HIP;
  if (launch_clip_errors(static_cast<const uint16_t*>(v), rows, R_v, cands, n_cands, fmt, Hkv, part,
                         nb, err + n_cands, clip + 1, s) != hipSuccess)
    return OSCAR_ERR_HIP;
  return OSCAR_OK;
}

}  // extern "C"

// ---------------------------------------------------------------------------
// decode attention without a caller workspace
// ---------------------------------------------------------------------------

namespace {

// The decode workspace (q~ and the partial states) of oscar_decode_attn_noalloc,
// for callers that cannot allocate: one copy per GPU, held until the process
// ends.  In host code `scratch` is only the symbol's name; its device address is
// looked up with hipGetSymbolAddress once per device (scratch_address) and only
// that address is handed to the kernels.
static __device__ __align__(256) uint8_t scratch[OSCAR_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 256;
std::mutex g_scratch_mu;
void* g_scratch_addr[kMaxDevices];

// Device address of the current device's scratch array.
int scratch_address(void** addr) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return OSCAR_ERR_HIP;
  if (dev < 0 || dev >= kMaxDevices) return OSCAR_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_addr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return OSCAR_ERR_HIP;
    g_scratch_addr[dev] = p;
  }
  *addr = g_scratch_addr[dev];
  return OSCAR_OK;
}

}  // namespace

extern "C" {

int oscar_decode_attn_noalloc(const oscar_layout* L, const void* pages, const void* q, int32_t B,
                              int32_t Hq, const int32_t* block_table, int32_t max_pages_per_seq,
                              const int32_t* seq_lens, const float* R_k, const float* R_v,
                              float sm_scale, int32_t num_splits, void* out,
                              oscar_dtype out_dtype, void* stream) {
  int st = check_decode_attn(L, pages, q, B, Hq, block_table, max_pages_per_seq, seq_lens,
                             sm_scale, &num_splits, out, out_dtype);
  if (st) return st;
  if (decode_ws(B, Hq, num_splits).total > OSCAR_NOALLOC_SCRATCH_BYTES)
    return OSCAR_ERR_WORKSPACE_TOO_SMALL;
  void* ws = nullptr;
  if ((st = scratch_address(&ws))) return st;
  return oscar_decode_attn(L, pages, q, B, Hq, block_table, max_pages_per_seq, seq_lens, R_k, R_v,
                           sm_scale, num_splits, ws, OSCAR_NOALLOC_SCRATCH_BYTES, out, out_dtype,
                           stream);
}

}  // extern "C"
