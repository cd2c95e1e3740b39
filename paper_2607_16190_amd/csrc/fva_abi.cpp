// C ABI of libfva.so: argument validation, workspace sizing and launch
// sequencing. Every check runs on the host before anything is launched.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "../../include/fva.h"
#include "fva_geometry.h"
#include "fva_internal.h"

namespace {

bool tiling_ok(const fva_tiling* t) {
  return t && t->T > 0 && t->H > 0 && t->W > 0 && t->bt > 0 && t->bh > 0 && t->bw > 0;
}

// Shape checks shared by route and attn; returns FVA_OK or the error.
fva_status check_shape(const fva_qkv_desc* d, const fva_tiling* t, int* nb_out) {
  if (!d || !t) return FVA_ERR_INVALID_ARG;
  if (!tiling_ok(t)) return FVA_ERR_SHAPE;
  if (d->batch < 0 || d->heads < 0 || d->tokens <= 0) return FVA_ERR_SHAPE;
  const int64_t n = (int64_t)t->T * t->H * t->W;
  if (n != (int64_t)d->tokens) return FVA_ERR_SHAPE;
  if (d->head_dim != fva::kHeadDim) return FVA_ERR_UNSUPPORTED;
  const int64_t vol = (int64_t)t->bt * t->bh * t->bw;
  if (vol != 64 && vol != 128) return FVA_ERR_UNSUPPORTED;
  const fva::Geometry g = fva::make_geometry(t->T, t->H, t->W, t->bt, t->bh, t->bw);
  if (g.nb > fva::kMaxBlocks) return FVA_ERR_UNSUPPORTED;
  // Strides are in elements; every token row must start on a 16-byte boundary.
  if (d->stride_n < d->head_dim || d->stride_h < 0 || d->stride_b < 0) return FVA_ERR_SHAPE;
  if (d->stride_n % 8 != 0 || d->stride_h % 8 != 0 || d->stride_b % 8 != 0) return FVA_ERR_SHAPE;
  // Kernels address a head with 32-bit byte offsets.
  if ((int64_t)d->tokens * d->stride_n * 2 >= ((int64_t)1 << 31)) return FVA_ERR_UNSUPPORTED;
  *nb_out = g.nb;
  return FVA_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Largest grid extent of the curve order: curve indices stay below 8^8.
constexpr int kMaxCurveExtent = 256;

fva_status check_curve_grid(int32_t T, int32_t H, int32_t W) {
  if (T <= 0 || H <= 0 || W <= 0) return FVA_ERR_SHAPE;
  if (T > kMaxCurveExtent || H > kMaxCurveExtent || W > kMaxCurveExtent) return FVA_ERR_UNSUPPORTED;
  return FVA_OK;
}

// Scheduling bits, the trace bit and a forced chunk size in bits 8..23.
constexpr uint32_t kAttnFlags = 7u | (0xFFFFu << 8);

// Attention indexes its work items -- batch * heads * nb query blocks plus
// the chunk items of split rows (at most 2048 with the automatic chunk size,
// at most 2^28 under FVA_SPLIT_BLOCKS) -- and their trace records with 32-bit
// integers.
bool attn_items_fit(const fva_qkv_desc* d, int nb, uint32_t flags) {
  const int64_t chunks = (flags & 1u) ? 0 : (((flags >> 8) & 0xFFFFu) ? ((int64_t)1 << 28) : 2048);
  return (int64_t)d->batch * d->heads * nb + chunks <= (int64_t)INT32_MAX;
}

}  // namespace

extern "C" {

int32_t fva_num_blocks(const fva_tiling* tiling) {
  if (!tiling_ok(tiling)) return -1;
  const int64_t nb = (int64_t)((tiling->T + tiling->bt - 1) / tiling->bt) * ((tiling->H + tiling->bh - 1) / tiling->bh) *
                     ((tiling->W + tiling->bw - 1) / tiling->bw);
  return nb > INT32_MAX ? -1 : (int32_t)nb;
}

fva_status fva_route_workspace_size(const fva_qkv_desc* desc, const fva_tiling* tiling, size_t* bytes) {
  if (!bytes) return FVA_ERR_INVALID_ARG;
  int nb = 0;
  const fva_status s = check_shape(desc, tiling, &nb);
  if (s != FVA_OK) return s;
  *bytes = fva::route_workspace_bytes(desc->batch, desc->heads, nb);
  return FVA_OK;
}

fva_status fva_attn_workspace_size(const fva_qkv_desc* desc, const fva_tiling* tiling, uint32_t flags, size_t* bytes) {
  if (!bytes) return FVA_ERR_INVALID_ARG;
  if (flags & ~kAttnFlags) return FVA_ERR_INVALID_ARG;
  int nb = 0;
  const fva_status s = check_shape(desc, tiling, &nb);
  if (s != FVA_OK) return s;
  if (!attn_items_fit(desc, nb, flags)) return FVA_ERR_UNSUPPORTED;
  const fva::Geometry g = fva::make_geometry(tiling->T, tiling->H, tiling->W, tiling->bt, tiling->bh, tiling->bw);
  *bytes = fva::attn_workspace_bytes(desc->batch, desc->heads, g, flags);
  return FVA_OK;
}

int64_t fva_trace_words(const fva_qkv_desc* desc, const fva_tiling* tiling) {
  int nb = 0;
  if (check_shape(desc, tiling, &nb) != FVA_OK || !attn_items_fit(desc, nb, 0u)) return -1;
  return fva::attn_trace_words(desc->batch, desc->heads, nb);
}

}  // extern "C"

namespace {

fva_status route_common(const void* Q, const void* K, const fva_qkv_desc* desc, double p, int32_t k_min,
                        const fva_tiling* tiling, uint8_t* block_mask, int32_t* counts, int32_t* kv_idx,
                        const int32_t* rank_of, int32_t n_ranks, double n1, double n2, int32_t* rank_extra,
                        void* workspace, size_t workspace_bytes, void* stream) {
  if (!Q || !K || !block_mask || !counts) return FVA_ERR_INVALID_ARG;
  if (std::isnan(p) || p < 0.0 || p > 1.0 || k_min < 0) return FVA_ERR_INVALID_ARG;
  int nb = 0;
  const fva_status s = check_shape(desc, tiling, &nb);
  if (s != FVA_OK) return s;
  if (!aligned16(Q) || !aligned16(K)) return FVA_ERR_INVALID_ARG;
  if ((int64_t)desc->batch * desc->heads > 65535) return FVA_ERR_UNSUPPORTED;  // pool grid's y extent
  const size_t need = rank_of ? fva::route_sasa_workspace_bytes(desc->batch, desc->heads, nb)
                              : fva::route_workspace_bytes(desc->batch, desc->heads, nb);
  if (!workspace || workspace_bytes < need || (reinterpret_cast<uintptr_t>(workspace) & 255u)) return FVA_ERR_WORKSPACE;
  fva::RouteArgs a;
  a.Q = Q;
  a.K = K;
  a.batch = desc->batch;
  a.heads = desc->heads;
  a.tokens = desc->tokens;
  a.stride_b = desc->stride_b;
  a.stride_h = desc->stride_h;
  a.stride_n = desc->stride_n;
  a.T = tiling->T;
  a.H = tiling->H;
  a.W = tiling->W;
  a.bt = tiling->bt;
  a.bh = tiling->bh;
  a.bw = tiling->bw;
  a.p = p;
  a.k_min = k_min;
  a.mask = block_mask;
  a.counts = counts;
  a.kv_idx = kv_idx;
  a.rank_of = rank_of;
  a.n_ranks = n_ranks;
  a.n1 = n1;
  a.n2 = n2;
  a.rank_extra = rank_extra;
  a.workspace = workspace;
  a.stream = reinterpret_cast<hipStream_t>(stream);
  return fva::launch_route(a) == hipSuccess ? FVA_OK : FVA_ERR_HIP;
}

}  // namespace

extern "C" {

fva_status fva_route(const void* Q, const void* K, const fva_qkv_desc* desc, double p, int32_t k_min,
                     const fva_tiling* tiling, uint8_t* block_mask, int32_t* counts, int32_t* kv_idx, void* workspace,
                     size_t workspace_bytes, void* stream) {
  return route_common(Q, K, desc, p, k_min, tiling, block_mask, counts, kv_idx, nullptr, 0, 0.0, 0.0, nullptr,
                      workspace, workspace_bytes, stream);
}

fva_status fva_route_sasa_workspace_size(const fva_qkv_desc* desc, const fva_tiling* tiling, size_t* bytes) {
  if (!bytes) return FVA_ERR_INVALID_ARG;
  int nb = 0;
  const fva_status s = check_shape(desc, tiling, &nb);
  if (s != FVA_OK) return s;
  *bytes = fva::route_sasa_workspace_bytes(desc->batch, desc->heads, nb);
  return FVA_OK;
}

fva_status fva_route_sasa(const void* Q, const void* K, const fva_qkv_desc* desc, double p, int32_t k_min,
                          const fva_tiling* tiling, const int32_t* rank_of, int32_t n_ranks, double n1, double n2,
                          uint8_t* block_mask, int32_t* counts, int32_t* kv_idx, int32_t* rank_extra, void* workspace,
                          size_t workspace_bytes, void* stream) {
  if (!rank_of || (reinterpret_cast<uintptr_t>(rank_of) & 3u)) return FVA_ERR_INVALID_ARG;
  if (rank_extra && (reinterpret_cast<uintptr_t>(rank_extra) & 3u)) return FVA_ERR_INVALID_ARG;
  if (n_ranks < 1 || n_ranks > 1024) return FVA_ERR_INVALID_ARG;
  if (!(n1 >= 0.0 && n1 <= 1.0) || !(n2 >= 0.0 && n2 <= 1.0)) return FVA_ERR_INVALID_ARG;
  return route_common(Q, K, desc, p, k_min, tiling, block_mask, counts, kv_idx, rank_of, n_ranks, n1, n2, rank_extra,
                      workspace, workspace_bytes, stream);
}

}  // extern "C"

namespace {

// fva_attn and fva_attn_fp8v: V is bf16 rows, or (V8 != null) E4M3 tiles with
// their exponents.
fva_status attn_common(const void* Q, const void* K, const void* V, const uint8_t* V8, const int32_t* v_exp,
                       const fva_qkv_desc* desc, const fva_tiling* tiling, const uint8_t* block_mask,
                       const int32_t* counts, const int32_t* kv_idx, float softmax_scale, uint32_t flags, void* O,
                       void* workspace, size_t workspace_bytes, void* trace, void* stream) {
  if (!Q || !K || !O) return FVA_ERR_INVALID_ARG;
  if (!V && !V8) return FVA_ERR_INVALID_ARG;
  if (V8 && (!v_exp || (reinterpret_cast<uintptr_t>(v_exp) & 3u))) return FVA_ERR_INVALID_ARG;
  if (flags & ~kAttnFlags) return FVA_ERR_INVALID_ARG;
  if ((counts == nullptr) != (kv_idx == nullptr)) return FVA_ERR_INVALID_ARG;
  if (!counts && !block_mask) return FVA_ERR_INVALID_ARG;
  if ((flags & FVA_TRACE) && !trace) return FVA_ERR_INVALID_ARG;
  if (std::isnan(softmax_scale) || std::isinf(softmax_scale)) return FVA_ERR_INVALID_ARG;
  int nb = 0;
  const fva_status s = check_shape(desc, tiling, &nb);
  if (s != FVA_OK) return s;
  if (!attn_items_fit(desc, nb, flags)) return FVA_ERR_UNSUPPORTED;
  if (!aligned16(Q) || !aligned16(K) || !aligned16(O)) return FVA_ERR_INVALID_ARG;
  if (V && !aligned16(V)) return FVA_ERR_INVALID_ARG;
  if (V8 && !aligned16(V8)) return FVA_ERR_INVALID_ARG;
  const fva::Geometry g = fva::make_geometry(tiling->T, tiling->H, tiling->W, tiling->bt, tiling->bh, tiling->bw);
  const size_t need = fva::attn_workspace_bytes(desc->batch, desc->heads, g, flags);
  if (!workspace || workspace_bytes < need || (reinterpret_cast<uintptr_t>(workspace) & 255u)) return FVA_ERR_WORKSPACE;
  fva::AttnArgs a;
  a.Q = Q;
  a.K = K;
  a.V = V;
  a.V8 = V8;
  a.vexp = v_exp;
  a.O = O;
  a.batch = desc->batch;
  a.heads = desc->heads;
  a.tokens = desc->tokens;
  a.stride_b = desc->stride_b;
  a.stride_h = desc->stride_h;
  a.stride_n = desc->stride_n;
  a.T = tiling->T;
  a.H = tiling->H;
  a.W = tiling->W;
  a.bt = tiling->bt;
  a.bh = tiling->bh;
  a.bw = tiling->bw;
  a.mask = block_mask;
  a.counts = counts;
  a.kv_idx = kv_idx;
  a.scale = softmax_scale > 0.f ? softmax_scale : 1.0f / std::sqrt(128.0f);
  a.flags = flags;
  a.trace = reinterpret_cast<int64_t*>(trace);
  a.workspace = workspace;
  a.stream = reinterpret_cast<hipStream_t>(stream);
  return fva::launch_attn(a) == hipSuccess ? FVA_OK : FVA_ERR_HIP;
}

}  // namespace

extern "C" {

fva_status fva_attn(const void* Q, const void* K, const void* V, const fva_qkv_desc* desc, const fva_tiling* tiling,
                    const uint8_t* block_mask, const int32_t* counts, const int32_t* kv_idx, float softmax_scale,
                    uint32_t flags, void* O, void* workspace, size_t workspace_bytes, void* trace, void* stream) {
  if (!V) return FVA_ERR_INVALID_ARG;
  return attn_common(Q, K, V, nullptr, nullptr, desc, tiling, block_mask, counts, kv_idx, softmax_scale, flags, O,
                     workspace, workspace_bytes, trace, stream);
}

fva_status fva_attn_noalloc(const void* Q, const void* K, const void* V, const fva_qkv_desc* desc,
                            const fva_tiling* tiling, const int32_t* counts, const int32_t* kv_idx,
                            float softmax_scale, uint32_t flags, void* O, void* trace, void* stream) {
  if (!Q || !K || !V || !O || !counts || !kv_idx) return FVA_ERR_INVALID_ARG;
  if (flags & ~FVA_TRACE) return FVA_ERR_INVALID_ARG;  // persistent scheduler, automatic chunks only
  if ((flags & FVA_TRACE) && !trace) return FVA_ERR_INVALID_ARG;
  if (std::isnan(softmax_scale) || std::isinf(softmax_scale)) return FVA_ERR_INVALID_ARG;
  int nb = 0;
  const fva_status s = check_shape(desc, tiling, &nb);
  if (s != FVA_OK) return s;
  if (!attn_items_fit(desc, nb, 1u)) return FVA_ERR_UNSUPPORTED;
  if (!aligned16(Q) || !aligned16(K) || !aligned16(V) || !aligned16(O)) return FVA_ERR_INVALID_ARG;
  const fva::Geometry g = fva::make_geometry(tiling->T, tiling->H, tiling->W, tiling->bt, tiling->bh, tiling->bw);
  if (fva::attn_noalloc_bytes(desc->batch, desc->heads, g) > fva::attn_noalloc_capacity()) return FVA_ERR_SCRATCH;
  fva::AttnArgs a;
  a.Q = Q;
  a.K = K;
  a.V = V;
  a.V8 = nullptr;
  a.vexp = nullptr;
  a.O = O;
  a.batch = desc->batch;
  a.heads = desc->heads;
  a.tokens = desc->tokens;
  a.stride_b = desc->stride_b;
  a.stride_h = desc->stride_h;
  a.stride_n = desc->stride_n;
  a.T = tiling->T;
  a.H = tiling->H;
  a.W = tiling->W;
  a.bt = tiling->bt;
  a.bh = tiling->bh;
  a.bw = tiling->bw;
  a.mask = nullptr;
  a.counts = counts;
  a.kv_idx = kv_idx;
  a.scale = softmax_scale > 0.f ? softmax_scale : 1.0f / std::sqrt(128.0f);
  a.flags = flags;
  a.trace = reinterpret_cast<int64_t*>(trace);
  a.workspace = nullptr;  // the library's static scratch
  a.stream = reinterpret_cast<hipStream_t>(stream);
  return fva::launch_attn_noalloc(a) == hipSuccess ? FVA_OK : FVA_ERR_HIP;
}

fva_status fva_v8_size(const fva_qkv_desc* desc, const fva_tiling* tiling, size_t* bytes) {
  if (!bytes) return FVA_ERR_INVALID_ARG;
  int nb = 0;
  const fva_status s = check_shape(desc, tiling, &nb);
  if (s != FVA_OK) return s;
  *bytes = (size_t)desc->batch * desc->heads * nb * fva::kV8TileBytes;
  return FVA_OK;
}

fva_status fva_quantize_v_workspace_size(const fva_qkv_desc* desc, const fva_tiling* tiling, size_t* bytes) {
  if (!bytes) return FVA_ERR_INVALID_ARG;
  int nb = 0;
  const fva_status s = check_shape(desc, tiling, &nb);
  if (s != FVA_OK) return s;
  *bytes = fva::quantize_v_workspace_bytes(desc->batch, desc->heads);
  return FVA_OK;
}

fva_status fva_quantize_v(const void* V, const fva_qkv_desc* desc, const fva_tiling* tiling, uint8_t* V8,
                          int32_t* v_exp, void* workspace, size_t workspace_bytes, void* stream) {
  if (!V || !V8 || !v_exp) return FVA_ERR_INVALID_ARG;
  int nb = 0;
  const fva_status s = check_shape(desc, tiling, &nb);
  if (s != FVA_OK) return s;
  if (!aligned16(V) || !aligned16(V8) || (reinterpret_cast<uintptr_t>(v_exp) & 3u)) return FVA_ERR_INVALID_ARG;
  if ((int64_t)desc->batch * desc->heads > 65535) return FVA_ERR_UNSUPPORTED;
  const size_t need = fva::quantize_v_workspace_bytes(desc->batch, desc->heads);
  if (!workspace || workspace_bytes < need || (reinterpret_cast<uintptr_t>(workspace) & 255u)) return FVA_ERR_WORKSPACE;
  fva::QuantizeArgs a;
  a.V = V;
  a.batch = desc->batch;
  a.heads = desc->heads;
  a.tokens = desc->tokens;
  a.stride_b = desc->stride_b;
  a.stride_h = desc->stride_h;
  a.stride_n = desc->stride_n;
  a.T = tiling->T;
  a.H = tiling->H;
  a.W = tiling->W;
  a.bt = tiling->bt;
  a.bh = tiling->bh;
  a.bw = tiling->bw;
  a.V8 = V8;
  a.vexp = v_exp;
  a.workspace = workspace;
  a.stream = reinterpret_cast<hipStream_t>(stream);
  return fva::launch_quantize_v(a) == hipSuccess ? FVA_OK : FVA_ERR_HIP;
}

fva_status fva_attn_fp8v(const void* Q, const void* K, const uint8_t* V8, const int32_t* v_exp,
                         const fva_qkv_desc* desc, const fva_tiling* tiling, const uint8_t* block_mask,
                         const int32_t* counts, const int32_t* kv_idx, float softmax_scale, uint32_t flags, void* O,
                         void* workspace, size_t workspace_bytes, void* trace, void* stream) {
  if (!V8 || !v_exp) return FVA_ERR_INVALID_ARG;
  return attn_common(Q, K, nullptr, V8, v_exp, desc, tiling, block_mask, counts, kv_idx, softmax_scale, flags, O,
                     workspace, workspace_bytes, trace, stream);
}

fva_status fva_curve_workspace_size(int32_t T, int32_t H, int32_t W, size_t* bytes) {
  if (!bytes) return FVA_ERR_INVALID_ARG;
  const fva_status s = check_curve_grid(T, H, W);
  if (s != FVA_OK) return s;
  *bytes = fva::curve_workspace_bytes(T, H, W);
  return FVA_OK;
}

fva_status fva_curve_order(int32_t T, int32_t H, int32_t W, int32_t* perm, void* workspace, size_t workspace_bytes,
                           void* stream) {
  if (!perm) return FVA_ERR_INVALID_ARG;
  const fva_status s = check_curve_grid(T, H, W);
  if (s != FVA_OK) return s;
  const size_t need = fva::curve_workspace_bytes(T, H, W);
  if (!workspace || workspace_bytes < need || (reinterpret_cast<uintptr_t>(workspace) & 255u)) return FVA_ERR_WORKSPACE;
  return fva::launch_curve_order(T, H, W, perm, workspace, reinterpret_cast<hipStream_t>(stream)) == hipSuccess
             ? FVA_OK
             : FVA_ERR_HIP;
}

fva_status fva_permute_tokens(const void* src, void* dst, const fva_qkv_desc* desc, const int32_t* perm,
                              int32_t direction, void* stream) {
  if (!src || !dst || !desc || !perm) return FVA_ERR_INVALID_ARG;
  if (direction != FVA_TO_CURVE && direction != FVA_FROM_CURVE) return FVA_ERR_INVALID_ARG;
  if (src == dst) return FVA_ERR_INVALID_ARG;
  if (!aligned16(src) || !aligned16(dst)) return FVA_ERR_INVALID_ARG;
  const fva_qkv_desc* d = desc;
  if (d->batch < 0 || d->heads < 0 || d->tokens <= 0) return FVA_ERR_SHAPE;
  if (d->head_dim != fva::kHeadDim) return FVA_ERR_UNSUPPORTED;
  if (d->stride_n < d->head_dim || d->stride_h < 0 || d->stride_b < 0) return FVA_ERR_SHAPE;
  if (d->stride_n % 8 != 0 || d->stride_h % 8 != 0 || d->stride_b % 8 != 0) return FVA_ERR_SHAPE;
  if ((int64_t)d->batch * d->heads > 65535) return FVA_ERR_UNSUPPORTED;
  return fva::launch_permute_rows(src, dst, d->batch, d->heads, d->tokens, d->stride_b, d->stride_h, d->stride_n, perm,
                                  direction, reinterpret_cast<hipStream_t>(stream)) == hipSuccess
             ? FVA_OK
             : FVA_ERR_HIP;
}

const char* fva_status_string(fva_status status) {
  switch (status) {
    case FVA_OK: return "ok";
    case FVA_ERR_INVALID_ARG: return "invalid argument";
    case FVA_ERR_SHAPE: return "shape mismatch";
    case FVA_ERR_UNSUPPORTED: return "unsupported shape (head_dim must be 128, tile volume 64 or 128, nb <= 1024, curve grid extents <= 256)";
    case FVA_ERR_WORKSPACE: return "workspace missing, misaligned or too small";
    case FVA_ERR_HIP: return "HIP launch failed";
    case FVA_ERR_SCRATCH: return "shape needs more scratch than the library's static device scratch holds (fva_attn_noalloc)";
  }
  return "unknown status";
}

}  // extern "C"
