// V quantisation for the FP8 attention variant (gfx950).
//
// §3.4 quantises V on the GPU before attention on every step. Here every
// (batch, head, channel d) gets a power-of-two scale 2^e_d,
//     e_d = max(-127, min{e : amax_d * 2^-e <= 448}),
// amax_d = max |V[., d]| over the head's tokens, and every element is
// rounded to OCP E4M3 (round to nearest even): code = E4M3(V * 2^-e_d). The
// scaling is exact, so the codes are exactly the format's rounding of V / 2^e_d.
//
// Output layout (one 16 KB tile per block, the attention kernel's PV operand
// order): V8[b][h][j] is 128 rows (channel d) x 128 bytes (key position p);
// byte (d, p) is the code of channel d of the block's packed real key
//     kap(p) = 64 hb + 32 (t / 2) + 8 g + 4 (t % 2) + r,
//     p = 32 g + 16 hb + 4 t + r  (g, t in 0..3; hb in 0..1; r in 0..3),
// and 0 for positions past the block's real keys. Lane group g of the
// attention kernel holds the E4M3 probabilities of its S^T accumulators in
// exactly this order (byte 16 hb + 4 t + r of its 32-byte fp8 MFMA operand),
// and reads bytes 32 g .. 32 g + 31 of each channel row as the V^T operand,
// so the two meet without any shuffle.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fva_common.h"
#include "fva_geometry.h"
#include "fva_internal.h"

namespace fva {
namespace {

__device__ __forceinline__ int v8_key_of_pos(int p) {
  const int g = p >> 5, hb = (p >> 4) & 1, t = (p >> 2) & 3, r = p & 3;
  return 64 * hb + 32 * (t >> 1) + 8 * g + 4 * (t & 1) + r;
}

__global__ void v8_clear_kernel(uint32_t* __restrict__ amax, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) amax[i] = 0u;
}

// amax over tokens for every (b, h, d): 16 lanes per 256-byte row, 16 rows
// per step, 256 rows per workgroup, one atomic max per channel and workgroup
// (non-negative floats order like their bit patterns).
__global__ __launch_bounds__(256) void v8_amax_kernel(const uint16_t* __restrict__ V, int heads, int tokens,
                                                      int64_t sb, int64_t sh, int64_t sn,
                                                      uint32_t* __restrict__ amax) {
  __shared__ float red[16][128];
  const int bh = blockIdx.y;
  const int b = bh / heads;
  const int h = bh - b * heads;
  const uint16_t* Vh = V + (int64_t)b * sb + (int64_t)h * sh;
  const int c = threadIdx.x & 15;
  const int rg = threadIdx.x >> 4;
  float m[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) m[e] = 0.f;
  const int r0 = blockIdx.x * 256;
#pragma unroll 4
  for (int s = 0; s < 16; ++s) {
    const int r = r0 + 16 * s + rg;
    if (r < tokens) {
      const uint4 v = *reinterpret_cast<const uint4*>(Vh + (int64_t)r * sn + 8 * c);
      const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        m[2 * e] = fmaxf(m[2 * e], fabsf(bf16_lo(w[e])));
        m[2 * e + 1] = fmaxf(m[2 * e + 1], fabsf(bf16_hi(w[e])));
      }
    }
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) red[rg][8 * c + e] = m[e];
  __syncthreads();
  if (threadIdx.x < 128) {
    float mx = 0.f;
#pragma unroll
    for (int g = 0; g < 16; ++g) mx = fmaxf(mx, red[g][threadIdx.x]);
    atomicMax(&amax[(int64_t)bh * 128 + threadIdx.x], __float_as_uint(mx));
  }
}

// e_d from amax_d: amax = 1.f * 2^(E - 127) with biased exponent E and
// fraction f; amax * 2^-e <= 448 = 1.75 * 2^8 first holds at
// e = E - 135 when 1.f <= 1.75, at e = E - 134 otherwise. Zero and
// subnormal amax (and anything below) give the floor -127.
__device__ __forceinline__ int v8_exponent(uint32_t amax_bits) {
  const int E = (int)((amax_bits >> 23) & 255u);
  const uint32_t f = amax_bits & 0x7FFFFFu;
  const int e = E - 135 + (f > 0x600000u ? 1 : 0);
  return E == 0 ? -127 : (e < -127 ? -127 : e);
}

// One workgroup per (b, h, block j): stage the block's real key rows (bf16,
// packed order) in LDS, then thread t writes channel d = t / 2, key
// positions 64 (t % 2) .. +63 of the tile. Workgroups of block 0 also write
// the head's exponents.
__global__ __launch_bounds__(256) void v8_quantize_kernel(const uint16_t* __restrict__ V, int heads, int64_t sb,
                                                          int64_t sh, int64_t sn, Geometry g,
                                                          const uint32_t* __restrict__ amax,
                                                          uint8_t* __restrict__ V8, int32_t* __restrict__ vexp) {
  __shared__ __align__(16) uint16_t rows[128][128];
  const int j = blockIdx.x;
  const int bh = blockIdx.y;
  const int b = bh / heads;
  const int h = bh - b * heads;
  const uint16_t* Vh = V + (int64_t)b * sb + (int64_t)h * sh;
  const BlockBox box = block_box(g, j);
  const int c = threadIdx.x & 15;
#pragma unroll
  for (int s = 0; s < 8; ++s) {
    const int kap = 16 * s + (threadIdx.x >> 4);
    uint4 v = make_uint4(0, 0, 0, 0);
    if (kap < box.n) v = *reinterpret_cast<const uint4*>(Vh + (int64_t)box_token(g, box, kap) * sn + 8 * c);
    *reinterpret_cast<uint4*>(&rows[kap][8 * c]) = v;
  }
  const int d = threadIdx.x >> 1;
  const int e = v8_exponent(amax[(int64_t)bh * 128 + d]);
  if (j == 0 && (threadIdx.x & 1) == 0) vexp[(int64_t)bh * 128 + d] = e;
  // 2^-e as a float: e in [-127, 120] keeps the biased exponent in [7, 254]
  const float inv = __uint_as_float((uint32_t)(127 - e) << 23);
  __syncthreads();
  const int p0 = 64 * (threadIdx.x & 1);
  uint32_t out[16];
#pragma unroll
  for (int q = 0; q < 16; ++q) {
    float x[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const uint16_t bits = rows[v8_key_of_pos(p0 + 4 * q + r)][d];
      x[r] = __uint_as_float((uint32_t)bits << 16) * inv;
    }
    int w = __builtin_amdgcn_cvt_pk_fp8_f32(x[0], x[1], 0, false);
    w = __builtin_amdgcn_cvt_pk_fp8_f32(x[2], x[3], w, true);
    out[q] = (uint32_t)w;
  }
  uint8_t* dst = V8 + ((int64_t)bh * g.nb + j) * kV8TileBytes + d * 128 + p0;
#pragma unroll
  for (int q = 0; q < 4; ++q)
    *reinterpret_cast<uint4*>(dst + 16 * q) = make_uint4(out[4 * q], out[4 * q + 1], out[4 * q + 2], out[4 * q + 3]);
}

}  // namespace

size_t quantize_v_workspace_bytes(int batch, int heads) {
  return (((size_t)batch * heads * 128 * 4) + 255) & ~(size_t)255;
}

hipError_t launch_quantize_v(const QuantizeArgs& a) {
  (void)hipGetLastError();
  const Geometry g = make_geometry(a.T, a.H, a.W, a.bt, a.bh, a.bw);
  const int nbh = a.batch * a.heads;
  if (nbh == 0) return hipSuccess;
  uint32_t* amax = static_cast<uint32_t*>(a.workspace);
  const int n = nbh * 128;
  const uint16_t* V = static_cast<const uint16_t*>(a.V);
  v8_clear_kernel<<<(n + 255) / 256, 256, 0, a.stream>>>(amax, n);
  v8_amax_kernel<<<dim3((a.tokens + 255) / 256, nbh), 256, 0, a.stream>>>(V, a.heads, a.tokens, a.stride_b, a.stride_h,
                                                                        a.stride_n, amax);
  v8_quantize_kernel<<<dim3(g.nb, nbh), 256, 0, a.stream>>>(V, a.heads, a.stride_b, a.stride_h, a.stride_n, g, amax,
                                                           a.V8, a.vexp);
  return hipGetLastError();
}

}  // namespace fva
