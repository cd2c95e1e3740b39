// Internal launch interface between the C ABI layer and the HIP kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "fva_geometry.h"

namespace fva {

struct RouteArgs {
  const void* Q;
  const void* K;
  int batch, heads, tokens;
  int64_t stride_b, stride_h, stride_n;
  int T, H, W, bt, bh, bw;
  double p;
  int k_min;
  uint8_t* mask;
  int32_t* counts;
  int32_t* kv_idx;  // may be null
  // slack-aware augmentation (null rank_of: plain routing)
  const int32_t* rank_of = nullptr;  // [batch * heads] rank of every head (device)
  int n_ranks = 0;
  double n1 = 0.0, n2 = 0.0;
  int32_t* rank_extra = nullptr;  // [n_ranks] extra blocks per row of each rank (device) or null
  int32_t* extra_head = nullptr;  // [batch * heads] workspace tail
  void* row_cuts = nullptr;       // [batch * heads * nb] last kept block of each routed row (augmentation)
  void* workspace;
  hipStream_t stream;
};

struct AttnArgs {
  const void* Q;
  const void* K;
  const void* V;
  void* O;
  int batch, heads, tokens;
  int64_t stride_b, stride_h, stride_n;
  int T, H, W, bt, bh, bw;
  const uint8_t* V8;      // E4M3 V tiles (FP8 variant) or null
  const int32_t* vexp;    // per-channel exponents of V8 (FP8 variant)
  const uint8_t* mask;
  const int32_t* counts;  // null: rebuilt from mask in the workspace
  const int32_t* kv_idx;  // null together with counts
  float scale;
  uint32_t flags;
  int64_t* trace;  // null unless tracing
  void* workspace;
  hipStream_t stream;
  bool lean = false;  // workspace laid out without list copies and chunk items
};

struct QuantizeArgs {
  const void* V;
  int batch, heads, tokens;
  int64_t stride_b, stride_h, stride_n;
  int T, H, W, bt, bh, bw;
  uint8_t* V8;
  int32_t* vexp;
  void* workspace;
  hipStream_t stream;
};

size_t route_workspace_bytes(int batch, int heads, int nb);
size_t route_sasa_workspace_bytes(int batch, int heads, int nb);
size_t attn_workspace_bytes(int batch, int heads, const Geometry& g, uint32_t flags);
int64_t attn_trace_words(int batch, int heads, int nb);

hipError_t launch_route(const RouteArgs& a);
hipError_t launch_attn(const AttnArgs& a);

// Allocation-free attention: scratch bytes a shape needs, the capacity of
// the library's static device scratch, and the launch (persistent scheduler,
// caller's counts and kept lists, no split rows) on that scratch.
size_t attn_noalloc_bytes(int batch, int heads, const Geometry& g);
size_t attn_noalloc_capacity();
hipError_t launch_attn_noalloc(const AttnArgs& a);

// E4M3 V quantisation for the FP8 attention variant (fp8_kernels.hip).
size_t quantize_v_workspace_bytes(int batch, int heads);
hipError_t launch_quantize_v(const QuantizeArgs& a);

// Hilbert-curve token order and row permutation (curve_kernels.hip).
size_t curve_workspace_bytes(int T, int H, int W);
hipError_t launch_curve_order(int T, int H, int W, int32_t* perm, void* workspace, hipStream_t stream);
hipError_t launch_permute_rows(const void* src, void* dst, int batch, int heads, int tokens, int64_t sb, int64_t sh,
                               int64_t sn, const int32_t* perm, int direction, hipStream_t stream);

}  // namespace fva
