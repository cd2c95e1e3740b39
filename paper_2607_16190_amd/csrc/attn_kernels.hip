// Block-sparse attention over the retained blocks on gfx950 (§2.1, §3.1).
//
// Work item = one (b, h, query block i). A 256-thread workgroup owns an item;
// each of its four waves owns 32 query rows (packed real tokens of block i).
// For every kept key block j (ascending ids from kv_idx) the workgroup stages
// K_j and V_j^T in LDS, then every wave computes
//     S^T = K_j Q_i^T             (bf16 MFMA 16x16x32, fp32 accumulation)
//     online softmax per query row (exp2 with the scale folded in)
//     O^T += V_j^T P^T            (bf16 MFMA 16x16x32)
// Working on S^T and O^T keeps every query row in one lane column, so the row
// statistics, the P operand and the O rescale never leave the lane group.
// The K rows are placed in LDS in an interleaved order so that the fp32
// accumulator of S^T, converted to bf16, is directly the B operand of the PV
// product (8 consecutive keys per lane) without any register shuffle.
//
// Scheduling: a persistent grid pulls items from a list ordered by descending
// kept-block count (longest-processing-time first) through one atomic
// counter; FVA_SCHED_NAIVE launches the same item body once per item in
// head-major order.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fva_common.h"
#include "fva_geometry.h"
#include "fva_internal.h"

namespace fva {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x8 __attribute__((ext_vector_type(8)));

constexpr int kAttnThreads = 256;
constexpr int kLdsStride = 136;  // bf16 per LDS row: 128 + 8 padding (272 B) keeps MFMA reads conflict-free
constexpr int kTileElems = 128 * kLdsStride;
constexpr size_t kAttnLds = 2 * kTileElems * sizeof(uint16_t);

struct AttnParams {
  const uint16_t* Q;
  const uint16_t* K;
  const uint16_t* V;
  uint16_t* O;
  int heads;
  int64_t sb, sh, sn;
  Geometry g;
  const int32_t* counts;
  const int32_t* kv_idx;
  float c2;  // softmax scale * log2(e)
  int64_t* trace;
};

// LDS row of key kap: keys 32kg + 8g + e (e < 8) land on rows
// 32kg + 16*(e/4) + 4g + e%4, i.e. the S^T accumulator of lane group g in
// tiles 2kg and 2kg+1 holds keys 32kg + 8g .. 32kg + 8g + 7 in order.
__device__ __forceinline__ int k_lds_row(int kap) {
  const int kg = kap >> 5;
  const int g = (kap >> 3) & 3;
  const int e = kap & 7;
  return (kg << 5) | ((e >> 2) << 4) | (g << 2) | (e & 3);
}

__device__ __forceinline__ uint32_t hw_location() {
  uint32_t hw, xcc;
  asm volatile("s_getreg_b32 %0, hwreg(HW_REG_HW_ID)" : "=s"(hw));
  asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(xcc));
  return ((xcc & 0xffu) << 16) | (hw & 0xffffu);
}

__device__ __forceinline__ void load_kv_regs(const AttnParams& P, int64_t base, int j, uint4 (&kr)[8],
                                             uint4 (&vr)[8]) {
  const BlockBox bj = block_box(P.g, j);
#pragma unroll
  for (int u = 0; u < 8; ++u) {
    const int it = threadIdx.x + kAttnThreads * u;
    const int kap = it >> 4;
    const int cc = it & 15;
    if (kap < bj.n) {
      const int64_t off = base + (int64_t)box_token(P.g, bj, kap) * P.sn + cc * 8;
      kr[u] = *reinterpret_cast<const uint4*>(P.K + off);
      vr[u] = *reinterpret_cast<const uint4*>(P.V + off);
    } else {
      kr[u] = make_uint4(0, 0, 0, 0);
      vr[u] = make_uint4(0, 0, 0, 0);
    }
  }
}

__device__ __forceinline__ void store_kv_lds(uint16_t* __restrict__ Ks, uint16_t* __restrict__ Vt,
                                             const uint4 (&kr)[8], const uint4 (&vr)[8]) {
#pragma unroll
  for (int u = 0; u < 8; ++u) {
    const int it = threadIdx.x + kAttnThreads * u;
    const int kap = it >> 4;
    const int cc = it & 15;
    *reinterpret_cast<uint4*>(Ks + k_lds_row(kap) * kLdsStride + cc * 8) = kr[u];
    const uint32_t w[4] = {vr[u].x, vr[u].y, vr[u].z, vr[u].w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      Vt[(cc * 8 + 2 * e) * kLdsStride + kap] = (uint16_t)(w[e] & 0xffffu);
      Vt[(cc * 8 + 2 * e + 1) * kLdsStride + kap] = (uint16_t)(w[e] >> 16);
    }
  }
}

__device__ __forceinline__ bf16x8 to_bf16x8(f32x4 a, f32x4 b) {
  const f32x8 v = __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
  return __builtin_convertvector(v, bf16x8);
}

__device__ void process_item(const AttnParams& P, int item, uint16_t* __restrict__ lds) {
  uint16_t* Ks = lds;
  uint16_t* Vt = lds + kTileElems;
  const int nb = P.g.nb;
  const int bh = item / nb;
  const int i = item - bh * nb;
  const int b = bh / P.heads;
  const int h = bh - b * P.heads;
  const int64_t base = (int64_t)b * P.sb + (int64_t)h * P.sh;
  const BlockBox bi = block_box(P.g, i);
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int g4 = lane >> 4;
  const int l16 = lane & 15;
  const int row0 = wave * 32;
  const bool active = row0 < bi.n;

  // Q_i^T as the B operand: lane holds query row l16 of each 16-row tile,
  // head dims 32ks + 8g4 .. +7.
  bf16x8 qf[2][4];
  int qtok[2];
#pragma unroll
  for (int nt = 0; nt < 2; ++nt) {
    const int row = row0 + 16 * nt + l16;
    qtok[nt] = row < bi.n ? box_token(P.g, bi, row) : -1;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      if (qtok[nt] >= 0) {
        qf[nt][ks] = *reinterpret_cast<const bf16x8*>(P.Q + base + (int64_t)qtok[nt] * P.sn + 32 * ks + 8 * g4);
      } else {
        qf[nt][ks] = bf16x8{};
      }
    }
  }

  f32x4 o[8][2];
#pragma unroll
  for (int mt = 0; mt < 8; ++mt)
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) o[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
  float mrow[2] = {-1.0e30f, -1.0e30f};
  float lrow[2] = {0.f, 0.f};

  // counts and kv_idx come from the caller: clamp so a bad list cannot
  // address outside the tensors.
  const int cnt = min(max(P.counts[item], 0), nb);
  const int32_t* kvl = P.kv_idx + (int64_t)item * nb;
  uint4 kr[8], vr[8];
  int jn = cnt > 0 ? min(max(kvl[0], 0), nb - 1) : 0;
  if (cnt > 0) load_kv_regs(P, base, jn, kr, vr);

  for (int c = 0; c < cnt; ++c) {
    const int nj = block_box(P.g, jn).n;
    __syncthreads();
    store_kv_lds(Ks, Vt, kr, vr);
    __syncthreads();
    if (c + 1 < cnt) {
      jn = min(max(kvl[c + 1], 0), nb - 1);
      load_kv_regs(P, base, jn, kr, vr);
    }
    if (!active) continue;
    const int ngroups = (nj + 31) >> 5;

    // S^T = K Q^T over the key tiles that hold real keys.
    f32x4 s[8][2];
#pragma unroll
    for (int mt = 0; mt < 8; ++mt) {
      if (mt < 2 * ngroups) {
        s[mt][0] = f32x4{0.f, 0.f, 0.f, 0.f};
        s[mt][1] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
          const bf16x8 a = *reinterpret_cast<const bf16x8*>(Ks + (mt * 16 + l16) * kLdsStride + 32 * ks + 8 * g4);
          s[mt][0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, qf[0][ks], s[mt][0], 0, 0, 0);
          s[mt][1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, qf[1][ks], s[mt][1], 0, 0, 0);
        }
      }
    }

    // Online softmax; key of accumulator (mt, r) in lane group g4 is
    // 32*(mt/2) + 8*g4 + 4*(mt%2) + r.
    float mx[2] = {-INFINITY, -INFINITY};
#pragma unroll
    for (int mt = 0; mt < 8; ++mt) {
      if (mt < 2 * ngroups) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int kap = 32 * (mt >> 1) + 8 * g4 + 4 * (mt & 1) + r;
#pragma unroll
          for (int nt = 0; nt < 2; ++nt) {
            const float v = kap < nj ? s[mt][nt][r] : -INFINITY;
            s[mt][nt][r] = v;
            mx[nt] = fmaxf(mx[nt], v);
          }
        }
      }
    }
    float alpha[2], negmc[2];
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
      mx[nt] = fmaxf(mx[nt], __shfl_xor(mx[nt], 16));
      mx[nt] = fmaxf(mx[nt], __shfl_xor(mx[nt], 32));
      const float mnew = fmaxf(mrow[nt], mx[nt]);
      alpha[nt] = exp2f((mrow[nt] - mnew) * P.c2);
      mrow[nt] = mnew;
      negmc[nt] = -mnew * P.c2;
    }
    float rs[2] = {0.f, 0.f};
#pragma unroll
    for (int mt = 0; mt < 8; ++mt) {
      if (mt < 2 * ngroups) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
#pragma unroll
          for (int nt = 0; nt < 2; ++nt) {
            const float pv = exp2f(fmaf(s[mt][nt][r], P.c2, negmc[nt]));
            s[mt][nt][r] = pv;
            rs[nt] += pv;
          }
        }
      }
    }
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
      rs[nt] += __shfl_xor(rs[nt], 16);
      rs[nt] += __shfl_xor(rs[nt], 32);
      lrow[nt] = lrow[nt] * alpha[nt] + rs[nt];
    }
#pragma unroll
    for (int mt = 0; mt < 8; ++mt)
#pragma unroll
      for (int nt = 0; nt < 2; ++nt) o[mt][nt] *= alpha[nt];

    // O^T += V^T P^T, 32 keys per MFMA.
#pragma unroll
    for (int kg = 0; kg < 4; ++kg) {
      if (kg < ngroups) {
        const bf16x8 p0 = to_bf16x8(s[2 * kg][0], s[2 * kg + 1][0]);
        const bf16x8 p1 = to_bf16x8(s[2 * kg][1], s[2 * kg + 1][1]);
#pragma unroll
        for (int mt = 0; mt < 8; ++mt) {
          const bf16x8 a = *reinterpret_cast<const bf16x8*>(Vt + (mt * 16 + l16) * kLdsStride + 32 * kg + 8 * g4);
          o[mt][0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, p0, o[mt][0], 0, 0, 0);
          o[mt][1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, p1, o[mt][1], 0, 0, 0);
        }
      }
    }
  }

  // Epilogue: O^T accumulator (mt, r) of lane (g4, l16) is head dim
  // 16mt + 4g4 + r of query row 16nt + l16.
  if (active) {
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
      if (qtok[nt] >= 0) {
        const float inv = lrow[nt] > 0.f ? 1.0f / lrow[nt] : 0.f;
        uint16_t* orow = P.O + base + (int64_t)qtok[nt] * P.sn + 4 * g4;
#pragma unroll
        for (int mt = 0; mt < 8; ++mt) {
          const f32x4 v = o[mt][nt] * inv;
          *reinterpret_cast<bf16x4*>(orow + 16 * mt) = __builtin_convertvector(v, bf16x4);
        }
      }
    }
  }
}

__device__ __forceinline__ void trace_item(const AttnParams& P, int item, int64_t t0) {
  if (P.trace && threadIdx.x == 0) {
    const int64_t t1 = (int64_t)wall_clock64();
    int64_t* tr = P.trace + (int64_t)item * 4;
    tr[0] = t0;
    tr[1] = t1;
    tr[2] = (int64_t)hw_location();
    tr[3] = (int64_t)blockIdx.x;
  }
}

__global__ __launch_bounds__(kAttnThreads, 1) void attn_naive_kernel(AttnParams P) {
  extern __shared__ __align__(16) uint16_t lds[];
  const int64_t t0 = (int64_t)wall_clock64();
  process_item(P, blockIdx.x, lds);
  if (P.trace) {
    __syncthreads();
    trace_item(P, blockIdx.x, t0);
  }
}

__global__ __launch_bounds__(kAttnThreads, 1) void attn_persistent_kernel(AttnParams P, const int32_t* __restrict__ items,
                                                                          int n_items, int32_t* __restrict__ counter) {
  extern __shared__ __align__(16) uint16_t lds[];
  __shared__ int next;
  for (;;) {
    __syncthreads();
    if (threadIdx.x == 0) next = atomicAdd(counter, 1);
    __syncthreads();
    const int slot = next;
    if (slot >= n_items) break;
    const int item = items[slot];
    const int64_t t0 = (int64_t)wall_clock64();
    process_item(P, item, lds);
    if (P.trace) {
      __syncthreads();
      trace_item(P, item, t0);
    }
  }
}

// Longest-processing-time order: items sorted by kept-block count, largest
// first (counting sort in one workgroup); also resets the queue counter.
__global__ __launch_bounds__(1024) void plan_kernel(const int32_t* __restrict__ counts, int n_items, int nb,
                                                   int32_t* __restrict__ items, int32_t* __restrict__ counter) {
  __shared__ int hist[kMaxBlocks + 1];
  for (int c = threadIdx.x; c <= nb; c += blockDim.x) hist[c] = 0;
  __syncthreads();
  for (int r = threadIdx.x; r < n_items; r += blockDim.x) {
    int c = counts[r];
    c = c < 0 ? 0 : (c > nb ? nb : c);
    atomicAdd(&hist[c], 1);
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int run = 0;
    for (int c = nb; c >= 0; --c) {
      const int n = hist[c];
      hist[c] = run;
      run += n;
    }
    *counter = 0;
  }
  __syncthreads();
  for (int r = threadIdx.x; r < n_items; r += blockDim.x) {
    int c = counts[r];
    c = c < 0 ? 0 : (c > nb ? nb : c);
    items[atomicAdd(&hist[c], 1)] = r;
  }
}

// counts and ascending kept-block lists from a block mask, one wave per row.
__global__ __launch_bounds__(256) void compact_kernel(const uint8_t* __restrict__ mask, int n_rows, int nb,
                                                     int32_t* __restrict__ counts, int32_t* __restrict__ kv_idx) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= n_rows) return;
  const uint8_t* mr = mask + (int64_t)row * nb;
  int32_t* kr = kv_idx + (int64_t)row * nb;
  int base = 0;
  for (int j0 = 0; j0 < nb; j0 += 64) {
    const int j = j0 + lane;
    const bool kept = j < nb && mr[j] != 0;
    const uint64_t bal = __ballot(kept);
    if (kept) kr[base + lanes_below(bal)] = j;
    base += __popcll(bal);
  }
  if (lane == 0) counts[row] = base;
}

struct DeviceInfo {
  int cus = 0;
  int per_cu = 0;
};

hipError_t device_info(DeviceInfo& info) {
  static DeviceInfo cache[64];
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  if (cache[dev].cus == 0) {
    DeviceInfo d;
    e = hipDeviceGetAttribute(&d.cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
    for (const void* fn : {reinterpret_cast<const void*>(&attn_naive_kernel),
                           reinterpret_cast<const void*>(&attn_persistent_kernel)}) {
      e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)kAttnLds);
      if (e != hipSuccess) return e;
    }
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&d.per_cu, reinterpret_cast<const void*>(&attn_persistent_kernel),
                                                     kAttnThreads, kAttnLds);
    if (e != hipSuccess) return e;
    if (d.per_cu < 1) d.per_cu = 1;
    cache[dev] = d;
  }
  info = cache[dev];
  return hipSuccess;
}

}  // namespace

size_t attn_workspace_bytes(int batch, int heads, int nb) {
  auto al = [](size_t x) { return (x + 255) & ~(size_t)255; };
  const size_t rows = (size_t)batch * heads * nb;
  return al(rows * 4) + al(rows * nb * 4) + al(rows * 4) + al(4);
}

hipError_t launch_attn(const AttnArgs& a) {
  (void)hipGetLastError();  // drop an error left by an unrelated earlier HIP call
  const Geometry g = make_geometry(a.T, a.H, a.W, a.bt, a.bh, a.bw);
  const int n_items = a.batch * a.heads * g.nb;
  if (n_items == 0) return hipSuccess;
  auto al = [](size_t x) { return (x + 255) & ~(size_t)255; };
  char* ws = reinterpret_cast<char*>(a.workspace);
  int32_t* ws_counts = reinterpret_cast<int32_t*>(ws);
  int32_t* ws_kv = reinterpret_cast<int32_t*>(ws + al((size_t)n_items * 4));
  int32_t* items = reinterpret_cast<int32_t*>(ws + al((size_t)n_items * 4) + al((size_t)n_items * g.nb * 4));
  int32_t* counter = items + (al((size_t)n_items * 4) / 4);

  DeviceInfo info;
  hipError_t e = device_info(info);
  if (e != hipSuccess) return e;

  const int32_t* counts = a.counts;
  const int32_t* kv_idx = a.kv_idx;
  if (!counts) {
    hipLaunchKernelGGL(compact_kernel, dim3((n_items + 3) / 4), dim3(256), 0, a.stream, a.mask, n_items, g.nb,
                       ws_counts, ws_kv);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    counts = ws_counts;
    kv_idx = ws_kv;
  }

  AttnParams P;
  P.Q = reinterpret_cast<const uint16_t*>(a.Q);
  P.K = reinterpret_cast<const uint16_t*>(a.K);
  P.V = reinterpret_cast<const uint16_t*>(a.V);
  P.O = reinterpret_cast<uint16_t*>(a.O);
  P.heads = a.heads;
  P.sb = a.stride_b;
  P.sh = a.stride_h;
  P.sn = a.stride_n;
  P.g = g;
  P.counts = counts;
  P.kv_idx = kv_idx;
  P.c2 = a.scale * 1.4426950408889634f;
  P.trace = (a.flags & 2u) ? a.trace : nullptr;

  if (a.flags & 1u) {
    hipLaunchKernelGGL(attn_naive_kernel, dim3(n_items), dim3(kAttnThreads), kAttnLds, a.stream, P);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(plan_kernel, dim3(1), dim3(1024), 0, a.stream, counts, n_items, g.nb, items, counter);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  int grid = info.cus * info.per_cu;
  if (grid > n_items) grid = n_items;
  hipLaunchKernelGGL(attn_persistent_kernel, dim3(grid), dim3(kAttnThreads), kAttnLds, a.stream, P, items, n_items,
                     counter);
  return hipGetLastError();
}

}  // namespace fva
