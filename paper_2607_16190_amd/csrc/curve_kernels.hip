// Hilbert-curve token order and row permutation (gfx950).
//
// §3.1 (routing frontend) reorders blocks along a Hilbert curve so that
// tokens close in the latent video fall into nearby blocks at every scale.
// Here the tokens of the T x H x W grid are ranked along J. Skilling's 3D
// Hilbert curve ("Programming the Hilbert curve", AIP Conf. Proc. 707, 2004)
// on the cube of side 2^k >= max(T, H, W), with (t, y, x) as the curve's
// axes 0, 1, 2 (axis 0 the most significant bit of each 3-bit digit).
// Cutting the ranked sequence into runs of B tokens gives blocks that are all
// full except the last; the routing and attention kernels then run unchanged
// on the permuted rows with the one-dimensional tiling {1, 1, N, 1, 1, B}.
//
// The rank of a token is the number of grid points with a smaller curve
// index. Curve indices are below 8^k <= 2^24, so the build marks every
// grid point's index in a bitmap of 8^k bits, takes an exclusive prefix sum
// of the bitmap's word popcounts, and ranks each token from its word's
// prefix plus the set bits below its own. Everything is exact integer work.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fva_internal.h"

namespace fva {
namespace {

constexpr int kScanThreads = 1024;
constexpr int kRowsPerThread = 4;

// Skilling's transform: coordinates -> transposed index -> interleaved index.
__host__ __device__ inline uint32_t curve_index(uint32_t a0, uint32_t a1, uint32_t a2, int bits) {
  if (bits == 0) return 0u;
  uint32_t X[3] = {a0, a1, a2};
  const uint32_t top = 1u << (bits - 1);
  // Inverse undo, top level first: a set bit on axis i inverts the lower
  // bits of axis 0, a clear one exchanges the lower bits of axes 0 and i.
  for (uint32_t q = top; q > 1u; q >>= 1) {
    const uint32_t low = q - 1u;
#pragma unroll
    for (int i = 0; i < 3; ++i) {
      if (X[i] & q) {
        X[0] ^= low;
      } else {
        const uint32_t s = (X[0] ^ X[i]) & low;
        X[0] ^= s;
        X[i] ^= s;
      }
    }
  }
  // Gray encode.
  X[1] ^= X[0];
  X[2] ^= X[1];
  uint32_t fix = 0u;
  for (uint32_t q = top; q > 1u; q >>= 1)
    if (X[2] & q) fix ^= q - 1u;
  X[0] ^= fix;
  X[1] ^= fix;
  X[2] ^= fix;
  uint32_t h = 0u;
  for (int b = bits - 1; b >= 0; --b)
    h = (h << 3) | (((X[0] >> b) & 1u) << 2) | (((X[1] >> b) & 1u) << 1) | ((X[2] >> b) & 1u);
  return h;
}

__global__ void curve_clear_kernel(uint32_t* __restrict__ bitmap, int words) {
  for (int w = blockIdx.x * blockDim.x + threadIdx.x; w < words; w += gridDim.x * blockDim.x) bitmap[w] = 0u;
}

__global__ void curve_mark_kernel(int T, int H, int W, int bits, uint32_t* __restrict__ keys,
                                  uint32_t* __restrict__ bitmap) {
  const int n = blockIdx.x * blockDim.x + threadIdx.x;
  const int HW = H * W;
  if (n >= T * HW) return;
  const int t = n / HW;
  const int rem = n - t * HW;
  const int y = rem / W;
  const int x = rem - y * W;
  const uint32_t key = curve_index((uint32_t)t, (uint32_t)y, (uint32_t)x, bits);
  keys[n] = key;
  atomicOr(&bitmap[key >> 5], 1u << (key & 31u));
}

// Exclusive prefix of the word popcounts, one workgroup walking the bitmap
// in tiles of kScanThreads words.
__global__ __launch_bounds__(kScanThreads) void curve_scan_kernel(const uint32_t* __restrict__ bitmap,
                                                                  int32_t* __restrict__ prefix, int words) {
  __shared__ int wave_sum[kScanThreads / 64];
  __shared__ int carry_s;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  if (threadIdx.x == 0) carry_s = 0;
  __syncthreads();
  for (int base = 0; base < words; base += kScanThreads) {
    const int w = base + threadIdx.x;
    const int c = w < words ? __popc(bitmap[w]) : 0;
    int incl = c;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const int o = __shfl_up(incl, d, 64);
      if (lane >= d) incl += o;
    }
    if (lane == 63) wave_sum[wave] = incl;
    __syncthreads();
    int before = 0, total = 0;
    for (int v = 0; v < kScanThreads / 64; ++v) {
      const int s = wave_sum[v];
      before += v < wave ? s : 0;
      total += s;
    }
    const int carry = carry_s;
    if (w < words) prefix[w] = carry + before + incl - c;
    __syncthreads();  // every thread has read wave_sum and carry_s
    if (threadIdx.x == 0) carry_s = carry + total;
    __syncthreads();
  }
}

__global__ void curve_rank_kernel(int N, const uint32_t* __restrict__ keys, const uint32_t* __restrict__ bitmap,
                                  const int32_t* __restrict__ prefix, int32_t* __restrict__ perm) {
  const int n = blockIdx.x * blockDim.x + threadIdx.x;
  if (n >= N) return;
  const uint32_t key = keys[n];
  const uint32_t w = key >> 5;
  const uint32_t below = bitmap[w] & ((1u << (key & 31u)) - 1u);
  perm[prefix[w] + __popc(below)] = n;
}

// Row permutation of a [batch, heads, tokens, 128] bf16 tensor: 16 lanes
// move one 256-byte row as 16-byte pieces; each thread moves kRowsPerThread
// rows, all loads issued before the stores. TO_CURVE gathers
// dst[r] = src[perm[r]], FROM_CURVE scatters dst[perm[r]] = src[r]; a perm
// entry outside [0, tokens) zeroes the gathered row or drops the scattered one.
__global__ __launch_bounds__(256) void permute_rows_kernel(const uint16_t* __restrict__ src,
                                                           uint16_t* __restrict__ dst, int heads, int tokens,
                                                           int64_t sb, int64_t sh, int64_t sn,
                                                           const int32_t* __restrict__ perm, int direction) {
  const int bh = blockIdx.y;
  const int b = bh / heads;
  const int h = bh - b * heads;
  const int64_t base = (int64_t)b * sb + (int64_t)h * sh + (threadIdx.x & 15) * 8;
  const int r0 = blockIdx.x * (16 * kRowsPerThread) + (threadIdx.x >> 4);
  uint4 v[kRowsPerThread];
  int to[kRowsPerThread];
#pragma unroll
  for (int u = 0; u < kRowsPerThread; ++u) {
    const int r = r0 + 16 * u;
    int from = -1;
    to[u] = -1;
    if (r < tokens) {
      const int p = perm[r];
      const bool ok = p >= 0 && p < tokens;
      from = direction == 0 ? (ok ? p : -1) : r;
      to[u] = direction == 0 ? r : (ok ? p : -1);
    }
    v[u] = from >= 0 ? *reinterpret_cast<const uint4*>(src + base + (int64_t)from * sn) : make_uint4(0, 0, 0, 0);
  }
#pragma unroll
  for (int u = 0; u < kRowsPerThread; ++u)
    if (to[u] >= 0) *reinterpret_cast<uint4*>(dst + base + (int64_t)to[u] * sn) = v[u];
}

size_t al256(size_t x) { return (x + 255) & ~(size_t)255; }

int bits_for(int T, int H, int W) {
  int m = T > H ? T : H;
  m = m > W ? m : W;
  int k = 0;
  while ((1 << k) < m) ++k;
  return k;
}

int bitmap_words(int bits) {
  const int64_t cells = (int64_t)1 << (3 * bits);
  return (int)(cells >= 32 ? cells / 32 : 1);
}

}  // namespace

size_t curve_workspace_bytes(int T, int H, int W) {
  const int words = bitmap_words(bits_for(T, H, W));
  const int64_t N = (int64_t)T * H * W;
  return al256((size_t)words * 4) * 2 + al256((size_t)N * 4);
}

hipError_t launch_curve_order(int T, int H, int W, int32_t* perm, void* workspace, hipStream_t stream) {
  const int bits = bits_for(T, H, W);
  const int words = bitmap_words(bits);
  const int N = T * H * W;
  unsigned char* p = static_cast<unsigned char*>(workspace);
  uint32_t* bitmap = reinterpret_cast<uint32_t*>(p);
  int32_t* prefix = reinterpret_cast<int32_t*>(p + al256((size_t)words * 4));
  uint32_t* keys = reinterpret_cast<uint32_t*>(p + 2 * al256((size_t)words * 4));
  const int clear_blocks = (words + 255) / 256 < 1024 ? (words + 255) / 256 : 1024;
  curve_clear_kernel<<<clear_blocks, 256, 0, stream>>>(bitmap, words);
  curve_mark_kernel<<<(N + 255) / 256, 256, 0, stream>>>(T, H, W, bits, keys, bitmap);
  curve_scan_kernel<<<1, kScanThreads, 0, stream>>>(bitmap, prefix, words);
  curve_rank_kernel<<<(N + 255) / 256, 256, 0, stream>>>(N, keys, bitmap, prefix, perm);
  return hipGetLastError();
}

hipError_t launch_permute_rows(const void* src, void* dst, int batch, int heads, int tokens, int64_t sb, int64_t sh,
                               int64_t sn, const int32_t* perm, int direction, hipStream_t stream) {
  if (batch * heads == 0) return hipSuccess;
  const dim3 grid((tokens + 16 * kRowsPerThread - 1) / (16 * kRowsPerThread), batch * heads);
  permute_rows_kernel<<<grid, 256, 0, stream>>>(static_cast<const uint16_t*>(src), static_cast<uint16_t*>(dst), heads,
                                                tokens, sb, sh, sn, perm, direction);
  return hipGetLastError();
}

}  // namespace fva
